// Vision-encoder side of the partial recompute on gfx950: one Qwen2.5-VL-style vision
// block over the patches of the recomputed merged tokens (Sec. 4.1: tokens that are not
// reused are recomputed by the visual encoder), with the reused patches' keys and values
// taken from the encoder's per-layer cache.
//
// Rows: the recomputed patches of item b are slots b Np + j, j < n_recompute[b] m^2,
// slot j being patch sub-position j mod m^2 of merged token recompute_idx[j / m^2]
// (patch rows token-major).  Kernels per call:
//
//   k_vit_gather_norm  one workgroup per slot: the patch row of x, RMSNorm (g1) as the
//                      bf16 operand of the QKV GEMM; the item's row count.
//   QKV GEMM           the weight-streaming split-K GEMM (fp32 partials).
//   k_vit_red_qkv      per slot: partial sums + bias; q rotated at the patch position
//                      (bf16, compact), raw k and v into the cache at the patch row.
//   k_vit_attn         one workgroup per (window, query chunk, head) or, with full
//                      attention, per (query chunk, head): the chunk's queries against the
//                      window's (the frame's) keys in blocks of 64, keys rotated on load,
//                      online softmax in fp32 on the vector ALUs.
//   O GEMM, k_vit_red_o       + bias + residual -> h1 (fp32) and bf16(RMSNorm(h1) g2).
//   gate/up GEMM, k_vit_red_gu   + biases, SiLU(g) u -> bf16.
//   down GEMM, k_vit_red_down    + bias + h1 -> the slot's output row of y (bf16).
//
// The 2-D rotary angle of dim pair i (i < hd/2) of a patch at (row, col) is
// row * f_i for i < hd/4 and col * f_(i - hd/4) otherwise, f_k = theta^(-2k / (hd/2));
// cos and sin are formed in fp64 and rounded to fp32.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "fc_internal.h"

namespace fc {
namespace {

constexpr int kVitThreads = 256;
constexpr int kVitMaxPos = 128;      // patch-grid side limit (rotary tables in LDS)
constexpr int kVitMaxHd = 128;
constexpr int kVitMaxD = 2048;       // hidden size limit of the QKV reduction's LDS row
constexpr int kVitQ = 64;            // queries per attention workgroup
constexpr int kVitK = 64;            // keys per staged block

__device__ __forceinline__ float bf2f_v(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }
__device__ __forceinline__ uint16_t f2bf_v(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

struct VitGeo {
  int N, m, mm, Np, gh, gw, d, H, hd, win;
};

// slot j of an item -> patch row (idx: the item's token ids)
__device__ __forceinline__ int slot_patch(const int32_t *idx, const VitGeo &g, int b, int j) {
  const int t = min(max(idx[(long)b * g.N + j / g.mm], 0), g.N - 1);
  return t * g.mm + j % g.mm;
}
__device__ __forceinline__ void patch_pos(const VitGeo &g, int p, int &pr, int &pc) {
  const int t = p / g.mm, sub = p - t * g.mm;
  pr = (t / g.gw) * g.m + sub / g.m;
  pc = (t % g.gw) * g.m + sub % g.m;
}
__device__ __forceinline__ int n_rows(const int32_t *nrec, const VitGeo &g, int b) {
  return min(max(nrec[b], 0), g.N) * g.mm;
}

__device__ float block_sum(float v, float *red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) s += red[i];
  __syncthreads();
  return s;
}

// --------------------------------------------------------------------- gather + norm
__global__ __launch_bounds__(kVitThreads) void k_vit_gather_norm(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ g1,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, VitGeo g, float eps,
    uint16_t *__restrict__ hb, int32_t *__restrict__ rows_out) {
  __shared__ float red[kVitThreads / 64];
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j == 0 && threadIdx.x == 0) rows_out[b] = n_rows(nrec, g, b);
  if (j >= n_rows(nrec, g, b)) return;
  const uint16_t *xr = x + ((long)b * g.Np + slot_patch(idx, g, b, j)) * g.d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < g.d; c += blockDim.x) {
    const float v = bf2f_v(xr[c]);
    ss = fmaf(v, v, ss);
  }
  const float inv = 1.f / sqrtf(block_sum(ss, red) / (float)g.d + eps);
  for (int c = threadIdx.x; c < g.d; c += blockDim.x)
    hb[s * g.d + c] = f2bf_v(bf2f_v(xr[c]) * inv * bf2f_v(g1[c]));
}

// ------------------------------------------------------------------- QKV reduction
__global__ __launch_bounds__(kVitThreads) void k_vit_red_qkv(
    const float *__restrict__ part, int splits, const uint16_t *__restrict__ bias,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, VitGeo g, double theta,
    uint16_t *__restrict__ q, uint16_t *__restrict__ kc, uint16_t *__restrict__ vc) {
  __shared__ float row[3 * kVitMaxD];
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const int p = slot_patch(idx, g, b, j);
  const int nc = 3 * g.d;
  const long rows = (long)gridDim.x;
  for (int c = threadIdx.x; c < nc; c += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < splits; ++sp) v += part[((long)sp * rows + s) * nc + c];
    row[c] = v + bf2f_v(bias[c]);
  }
  __syncthreads();
  int pr, pc;
  patch_pos(g, p, pr, pc);
  const int half = g.hd / 2, quarter = g.hd / 4;
  for (int c = threadIdx.x; c < g.d; c += blockDim.x) {
    const int hd_i = c % g.hd;
    const int i = hd_i % half;                                  // rotary pair
    const int fk = i < quarter ? i : i - quarter;
    const double ang = (double)(i < quarter ? pr : pc) * pow(theta, -2.0 * fk / (double)half);
    const float cs = (float)cos(ang), sn = (float)sin(ang);
    const float xv = row[c];
    const float partner = hd_i < half ? -row[c + half] : row[c - half];
    q[s * g.d + c] = f2bf_v(xv * cs + partner * sn);
    const long kv = ((long)b * g.Np + p) * g.d + c;
    kc[kv] = f2bf_v(row[g.d + c]);
    vc[kv] = f2bf_v(row[2 * g.d + c]);
  }
}

// ------------------------------------------------------------------------ attention
// Key k of a workgroup's key set: the window's patches (token-major within the window)
// or, with full attention, patch k of the frame.
__device__ __forceinline__ int key_patch(const VitGeo &g, int w, int k) {
  if (g.win <= 0) return k;
  const int wpr = (g.gw + g.win - 1) / g.win;
  const int wi = w / wpr, wj = w - wi * wpr;
  const int I0 = wi * g.win, J0 = wj * g.win;
  const int wcols = min(g.win, g.gw - J0);
  const int tk = k / g.mm, sub = k - tk * g.mm;
  const int I = I0 + tk / wcols, J = J0 + tk % wcols;
  return (I * g.gw + J) * g.mm + sub;
}
__device__ __forceinline__ int window_keys(const VitGeo &g, int w) {
  if (g.win <= 0) return g.Np;
  const int wpr = (g.gw + g.win - 1) / g.win;
  const int wi = w / wpr, wj = w - wi * wpr;
  return min(g.win, g.gh - wi * g.win) * min(g.win, g.gw - wj * g.win) * g.mm;
}
__device__ __forceinline__ int window_of(const VitGeo &g, int p) {
  if (g.win <= 0) return 0;
  const int t = p / g.mm;
  const int wpr = (g.gw + g.win - 1) / g.win;
  return (t / g.gw) / g.win * wpr + (t % g.gw) / g.win;
}

// Grid: x = window * chunks_per_window + chunk, y = head, z = item.  Each workgroup takes
// the chunk-th group of up to 64 recomputed slots of its window (slot order).
__global__ __launch_bounds__(kVitThreads) void k_vit_attn(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ kc,
    const uint16_t *__restrict__ vc, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ nrec, VitGeo g, double theta, int chunks,
    uint16_t *__restrict__ out) {
  __shared__ float Qs[kVitQ][kVitMaxHd + 1];
  __shared__ float Ks[kVitK][kVitMaxHd + 1];
  __shared__ float Vs[kVitK][kVitMaxHd + 1];
  __shared__ float Ps[kVitQ][kVitK + 1];
  __shared__ float2 rtab[kVitMaxPos][kVitMaxHd / 4];
  __shared__ int qslot[kVitQ];
  __shared__ int nq_s;
  const int w = blockIdx.x / chunks, chunk = blockIdx.x - w * chunks;
  const int h = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x;
  const int half = g.hd / 2, quarter = g.hd / 4;
  const int nrow = n_rows(nrec, g, b);
  // the chunk's queries: recomputed slots of window w (in slot order), the chunk-th 64
  // of them; found by all threads in rounds of 256 slots with a ballot prefix count
  __shared__ int wcnt[kVitThreads / 64];
  const int lo = chunk * kVitQ, hi = lo + kVitQ;
  int seen = 0;
  for (int j0 = 0; j0 < nrow && seen < hi; j0 += blockDim.x) {
    const int j = j0 + t;
    const bool in = j < nrow && window_of(g, slot_patch(idx, g, b, j)) == w;
    const unsigned long long bal = __ballot(in);
    const int lane = t & 63, wv = t >> 6;
    if (lane == 0) wcnt[wv] = __popcll(bal);
    __syncthreads();
    int before = 0, total = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
      if (i < wv) before += wcnt[i];
      total += wcnt[i];
    }
    const int pos = seen + before + __popcll(bal & ((1ull << lane) - 1ull));
    if (in && pos >= lo && pos < hi) qslot[pos - lo] = j;
    seen += total;
    __syncthreads();
  }
  if (t == 0) nq_s = min(max(seen - lo, 0), kVitQ);
  // rotary table: position x frequency (positions up to the grid's patch side)
  const int npos = max(g.gh, g.gw) * g.m;
  for (int e = t; e < npos * quarter; e += blockDim.x) {
    const int ps = e / quarter, fk = e - ps * quarter;
    const double ang = (double)ps * pow(theta, -2.0 * fk / (double)half);
    rtab[ps][fk] = make_float2((float)cos(ang), (float)sin(ang));
  }
  __syncthreads();
  const int nq = nq_s;
  if (nq == 0) return;
  for (int e = t; e < nq * g.hd; e += blockDim.x) {
    const int qi = e / g.hd, c = e - qi * g.hd;
    Qs[qi][c] = bf2f_v(q[((long)b * g.Np + qslot[qi]) * g.d + h * g.hd + c]);
  }
  // four threads per query: scores of keys k = 4 r + l, output dims d = l, l + 4, ...
  const int qi = t >> 2, l = t & 3;
  const bool qa = qi < nq;
  float mrun = -INFINITY, lsum = 0.f;
  float acc[kVitMaxHd / 4];
#pragma unroll
  for (int e = 0; e < kVitMaxHd / 4; ++e) acc[e] = 0.f;
  const float scale = 1.f / sqrtf((float)g.hd);
  const int nk = window_keys(g, w);
  for (int k0 = 0; k0 < nk; k0 += kVitK) {
    const int kn = min(kVitK, nk - k0);
    __syncthreads();                          // previous block's Ks, Vs, Ps are consumed
    for (int e = t; e < kn * g.hd; e += blockDim.x) {
      const int ki = e / g.hd, c = e - ki * g.hd;
      const int p = key_patch(g, w, k0 + ki);
      const long base = (((long)b * g.Np + p) * g.H + h) * g.hd;
      int pr, pc;
      patch_pos(g, p, pr, pc);
      const int i = c % half;
      const float2 cs = rtab[i < quarter ? pr : pc][i < quarter ? i : i - quarter];
      const float xv = bf2f_v(kc[base + c]);
      const float partner = c < half ? -bf2f_v(kc[base + c + half]) : bf2f_v(kc[base + c - half]);
      Ks[ki][c] = xv * cs.x + partner * cs.y;
      Vs[ki][c] = bf2f_v(vc[base + c]);
    }
    __syncthreads();
    float bmax = -INFINITY;
    if (qa) {
      for (int ki = l; ki < kn; ki += 4) {
        float sdot = 0.f;
        for (int c = 0; c < g.hd; ++c) sdot = fmaf(Qs[qi][c], Ks[ki][c], sdot);
        sdot *= scale;
        Ps[qi][ki] = sdot;
        bmax = fmaxf(bmax, sdot);
      }
    }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 1));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 2));
    const float mnew = fmaxf(mrun, bmax);
    const float corr = (mrun == -INFINITY) ? 0.f : expf(mrun - mnew);
    float psum = 0.f;
    if (qa) {
      for (int ki = l; ki < kn; ki += 4) {
        const float pv = expf(Ps[qi][ki] - mnew);
        Ps[qi][ki] = pv;
        psum += pv;
      }
    }
    psum += __shfl_xor(psum, 1);
    psum += __shfl_xor(psum, 2);
    lsum = lsum * corr + psum;
    mrun = mnew;
    __syncthreads();                          // every probability of the block is written
    if (qa) {
#pragma unroll
      for (int e = 0; e < kVitMaxHd / 4; ++e) {
        const int c = e * 4 + l;
        if (c >= g.hd) break;
        float a = acc[e] * corr;
        for (int ki = 0; ki < kn; ++ki) a = fmaf(Ps[qi][ki], Vs[ki][c], a);
        acc[e] = a;
      }
    }
  }
  if (qa) {
    const float inv = 1.f / lsum;
    uint16_t *o = out + ((long)b * g.Np + qslot[qi]) * g.d + h * g.hd;
#pragma unroll
    for (int e = 0; e < kVitMaxHd / 4; ++e)
      if (e * 4 + l < g.hd) o[e * 4 + l] = f2bf_v(acc[e] * inv);
  }
}

// --------------------------------------------------------------- O / MLP reductions
__global__ __launch_bounds__(kVitThreads) void k_vit_red_o(
    const float *__restrict__ part, int splits, const uint16_t *__restrict__ bias,
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ g2,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, VitGeo g, float eps,
    float *__restrict__ h1, uint16_t *__restrict__ hb) {
  __shared__ float red[kVitThreads / 64];
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const uint16_t *xr = x + ((long)b * g.Np + slot_patch(idx, g, b, j)) * g.d;
  const long rows = (long)gridDim.x;
  float ss = 0.f;
  for (int c = threadIdx.x; c < g.d; c += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < splits; ++sp) v += part[((long)sp * rows + s) * g.d + c];
    const float hv = bf2f_v(xr[c]) + (v + bf2f_v(bias[c]));
    h1[s * g.d + c] = hv;
    ss = fmaf(hv, hv, ss);
  }
  const float inv = 1.f / sqrtf(block_sum(ss, red) / (float)g.d + eps);
  for (int c = threadIdx.x; c < g.d; c += blockDim.x)
    hb[s * g.d + c] = f2bf_v(h1[s * g.d + c] * inv * bf2f_v(g2[c]));
}

__global__ __launch_bounds__(kVitThreads) void k_vit_red_gu(
    const float *__restrict__ part, int splits, const uint16_t *__restrict__ bias, int f,
    const int32_t *__restrict__ nrec, VitGeo g, uint16_t *__restrict__ act) {
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const long rows = (long)gridDim.x;
  for (int c = threadIdx.x; c < f; c += blockDim.x) {
    float gv = 0.f, uv = 0.f;
    for (int sp = 0; sp < splits; ++sp) {
      gv += part[((long)sp * rows + s) * 2 * f + c];
      uv += part[((long)sp * rows + s) * 2 * f + f + c];
    }
    gv += bf2f_v(bias[c]);
    uv += bf2f_v(bias[f + c]);
    act[s * f + c] = f2bf_v(gv / (1.f + expf(-gv)) * uv);
  }
}

__global__ __launch_bounds__(kVitThreads) void k_vit_red_down(
    const float *__restrict__ part, int splits, const uint16_t *__restrict__ bias,
    const float *__restrict__ h1, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ nrec, VitGeo g, uint16_t *__restrict__ y) {
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  uint16_t *yr = y + ((long)b * g.Np + slot_patch(idx, g, b, j)) * g.d;
  const long rows = (long)gridDim.x;
  for (int c = threadIdx.x; c < g.d; c += blockDim.x) {
    float v = 0.f;
    for (int sp = 0; sp < splits; ++sp) v += part[((long)sp * rows + s) * g.d + c];
    yr[c] = f2bf_v(h1[s * g.d + c] + (v + bf2f_v(bias[c])));
  }
}

// --------------------------------------------------------------------- patch merger
// One workgroup per (item, recomputed token): the token's merge^2 patch rows, each
// RMS-normalised with its own 1/rms, side by side as the token's bf16 GEMM row.
__global__ __launch_bounds__(kVitThreads) void k_merge_norm(
    const uint16_t *__restrict__ y, const uint16_t *__restrict__ gain,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, int N, int mm, int d,
    float eps, uint16_t *__restrict__ hb) {
  __shared__ float red[kVitThreads / 64];
  const long s = blockIdx.x;
  const int b = (int)(s / N), j = (int)(s - (long)b * N);
  if (j >= min(max(nrec[b], 0), N)) return;
  const int t = min(max(idx[s], 0), N - 1);
  for (int a = 0; a < mm; ++a) {
    const uint16_t *yr = y + (((long)b * N + t) * mm + a) * d;
    float ss = 0.f;
    for (int c = threadIdx.x; c < d; c += blockDim.x) {
      const float v = bf2f_v(yr[c]);
      ss = fmaf(v, v, ss);
    }
    const float inv = 1.f / sqrtf(block_sum(ss, red) / (float)d + eps);
    uint16_t *o = hb + (s * mm + a) * d;
    for (int c = threadIdx.x; c < d; c += blockDim.x) o[c] = f2bf_v(bf2f_v(yr[c]) * inv * bf2f_v(gain[c]));
  }
}

// split-K sums + bias, then exact GELU (x Phi(x)), bf16
__global__ __launch_bounds__(kVitThreads) void k_merge_red_gelu(
    const float *__restrict__ part, int splits, const uint16_t *__restrict__ bias,
    const int32_t *__restrict__ nrec, int N, int hidden, uint16_t *__restrict__ act) {
  const long s = blockIdx.x;
  const int b = (int)(s / N), j = (int)(s - (long)b * N);
  if (j >= min(max(nrec[b], 0), N)) return;
  const long rows = (long)gridDim.x;
  for (int c = threadIdx.x; c < hidden; c += blockDim.x) {
    float v = bf2f_v(bias[c]);
    for (int sp = 0; sp < splits; ++sp) v += part[((long)sp * rows + s) * hidden + c];
    act[s * hidden + c] = f2bf_v(0.5f * v * (1.f + erff(v * 0.70710678118654752f)));
  }
}

// split-K sums + bias into the token's output row
__global__ __launch_bounds__(kVitThreads) void k_merge_red_out(
    const float *__restrict__ part, int splits, const uint16_t *__restrict__ bias,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, int N, int d_out,
    uint16_t *__restrict__ x_out) {
  const long s = blockIdx.x;
  const int b = (int)(s / N), j = (int)(s - (long)b * N);
  if (j >= min(max(nrec[b], 0), N)) return;
  const int t = min(max(idx[s], 0), N - 1);
  const long rows = (long)gridDim.x;
  uint16_t *o = x_out + ((long)b * N + t) * d_out;
  for (int c = threadIdx.x; c < d_out; c += blockDim.x) {
    float v = bf2f_v(bias[c]);
    for (int sp = 0; sp < splits; ++sp) v += part[((long)sp * rows + s) * d_out + c];
    o[c] = f2bf_v(v);
  }
}

}  // namespace

fc_status launch_vit_block(fc_ctx *ctx, const fc_vit_desc &L, const fc_vit_cache &c,
                           const uint16_t *x, const int32_t *idx, const int32_t *nrec,
                           uint16_t *y, int B, hipStream_t st) {
  VitGeo g;
  g.N = c.grid_h * c.grid_w;
  g.m = c.merge;
  g.mm = c.merge * c.merge;
  g.Np = g.N * g.mm;
  g.gh = c.grid_h;
  g.gw = c.grid_w;
  g.d = L.d_model;
  g.H = L.n_heads;
  g.hd = L.head_dim;
  g.win = c.window;
  const long slots = (long)B * g.Np;
  const int f = L.d_ffn;
  int splits = 1;
  fc_status rc;
  {
    ProfScope ps(ctx, st, "fc_vit_gather_norm");
    hipLaunchKernelGGL(k_vit_gather_norm, dim3((unsigned)slots), dim3(kVitThreads), 0, st, x, L.g1,
                       idx, nrec, g, L.rms_eps, ctx->hb, ctx->vit_rows);
    FC_LAUNCH_OK(st, "k_vit_gather_norm");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_qkv", ctx->hb, L.w_qkv, g.d, 3 * g.d, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_qkv");
    hipLaunchKernelGGL(k_vit_red_qkv, dim3((unsigned)slots), dim3(kVitThreads), 0, st,
                       (const float *)ctx->part, splits, L.b_qkv, idx, nrec, g, L.rope_theta,
                       ctx->qbuf, c.k, c.v);
    FC_LAUNCH_OK(st, "k_vit_red_qkv");
  }
  {
    // query chunks of 64 per window (full attention: one window of every patch)
    const int nwin = c.window > 0 ? ((g.gh + c.window - 1) / c.window) * ((g.gw + c.window - 1) / c.window) : 1;
    const int wkeys = c.window > 0 ? std::min(c.window, g.gh) * std::min(c.window, g.gw) * g.mm : g.Np;
    const int chunks = (wkeys + kVitQ - 1) / kVitQ;
    ProfScope ps(ctx, st, "fc_vit_attn");
    hipLaunchKernelGGL(k_vit_attn, dim3((unsigned)(nwin * chunks), (unsigned)g.H, (unsigned)B),
                       dim3(kVitThreads), 0, st, (const uint16_t *)ctx->qbuf, (const uint16_t *)c.k,
                       (const uint16_t *)c.v, idx, nrec, g, L.rope_theta, chunks, ctx->attn);
    FC_LAUNCH_OK(st, "k_vit_attn");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_o", ctx->attn, L.w_o, g.d, g.d, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_o");
    hipLaunchKernelGGL(k_vit_red_o, dim3((unsigned)slots), dim3(kVitThreads), 0, st,
                       (const float *)ctx->part, splits, L.b_o, x, L.g2, idx, nrec, g, L.rms_eps,
                       ctx->h1, ctx->hb);
    FC_LAUNCH_OK(st, "k_vit_red_o");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_gateup", ctx->hb, L.w_gate_up, g.d, 2 * f, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_gu");
    hipLaunchKernelGGL(k_vit_red_gu, dim3((unsigned)slots), dim3(kVitThreads), 0, st,
                       (const float *)ctx->part, splits, L.b_gate_up, f, nrec, g, ctx->act);
    FC_LAUNCH_OK(st, "k_vit_red_gu");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_down", ctx->act, L.w_down, f, g.d, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_down");
    hipLaunchKernelGGL(k_vit_red_down, dim3((unsigned)slots), dim3(kVitThreads), 0, st,
                       (const float *)ctx->part, splits, L.b_down, (const float *)ctx->h1, idx,
                       nrec, g, y);
    FC_LAUNCH_OK(st, "k_vit_red_down");
  }
  return FC_OK;
}

fc_status launch_vit_cache_update(fc_ctx *ctx, const fc_vit_desc &L, const fc_vit_cache &c,
                                  const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                                  const uint8_t *reuse, int B, hipStream_t st) {
  // a merged token's patch rows are contiguous: the token-level remap with rows of
  // m^2 patches (one frame slot, whose in-place overwrite stages the old rows)
  const int mm = c.merge * c.merge;
  fc_layer_desc ld{};
  ld.d_model = mm * L.d_model;
  ld.n_heads = mm * L.n_heads;
  ld.n_kv_heads = mm * L.n_heads;
  ld.head_dim = L.head_dim;
  fc_kv_cache kv{};
  kv.k = c.k;
  kv.v = c.v;
  kv.text_tokens = 0;
  kv.frame_tokens = c.grid_h * c.grid_w;
  kv.window = 1;
  kv.head = 0;
  return launch_cache_update(ctx, ld, kv, y_prev, y_cur, shift, reuse, c.grid_w, B, st);
}

fc_status launch_vit_merger(fc_ctx *ctx, const fc_merger_desc &M, const uint16_t *y,
                            const int32_t *idx, const int32_t *nrec, uint16_t *x_out, int N,
                            int B, hipStream_t st) {
  const int mm = M.merge * M.merge;
  const int hidden = mm * M.d_model;
  const long slots = (long)B * N;
  uint16_t *hb = ctx->act;                                   // normalised token rows
  uint16_t *act = ctx->act + slots * hidden;                 // GELU outputs
  int splits = 1;
  fc_status rc;
  {
    ProfScope ps(ctx, st, "fc_merge_norm");
    hipLaunchKernelGGL(k_merge_norm, dim3((unsigned)slots), dim3(kVitThreads), 0, st, y, M.g, idx,
                       nrec, N, mm, M.d_model, M.rms_eps, hb);
    FC_LAUNCH_OK(st, "k_merge_norm");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_merge_gemm1", hb, M.w1, hidden, hidden, N, nrec,
                           ctx->part, B, &splits)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_merge_red_gelu");
    hipLaunchKernelGGL(k_merge_red_gelu, dim3((unsigned)slots), dim3(kVitThreads), 0, st,
                       (const float *)ctx->part, splits, M.b1, nrec, N, hidden, act);
    FC_LAUNCH_OK(st, "k_merge_red_gelu");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_merge_gemm2", act, M.w2, hidden, M.d_out, N, nrec,
                           ctx->part, B, &splits)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_merge_red_out");
    hipLaunchKernelGGL(k_merge_red_out, dim3((unsigned)slots), dim3(kVitThreads), 0, st,
                       (const float *)ctx->part, splits, M.b2, idx, nrec, N, M.d_out, x_out);
    FC_LAUNCH_OK(st, "k_merge_red_out");
  }
  return FC_OK;
}

}  // namespace fc
