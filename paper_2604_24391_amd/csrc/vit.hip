// Vision-encoder side of the partial recompute on gfx950: one Qwen2.5-VL-style vision
// block over the patches of the recomputed merged tokens (Sec. 4.1: a token that is not
// reused goes through the vision encoder again), with the reused patches' keys and values
// taken from the encoder's per-layer cache.
//
// Rows: the recomputed patches of item b are slots b Np + j, j < n_recompute[b] m^2,
// slot j being patch sub-position j mod m^2 of merged token recompute_idx[j / m^2]
// (patch rows token-major).  Kernels per call:
//
//   k_vit_gather_norm  one workgroup per slot: the patch row of x, RMSNorm (g1) as the
//                      bf16 operand of the QKV GEMM; the item's row count; the rotary table.
//   QKV GEMM           the weight-streaming split-K GEMM (fp32 partials).
//   k_vit_red_qkv      per (slot, column chunk): partial sums + bias; q rotated at the patch
//                      position (bf16, compact), raw k and v into the cache at the patch row.
//   k_vit_attn         one workgroup per (window, query chunk, head) or, with full
//                      attention, per (query chunk, head): the chunk's queries against the
//                      window's (the frame's) keys in blocks of 64, keys rotated on load,
//                      S^T = K Q^T and O^T = V^T P^T on bf16 MFMAs, online softmax in fp32.
//   O GEMM, k_vit_red_o       + bias + residual -> h1 (fp32), bf16(h1 g2) and the row's
//                             sum of squares by column chunk.
//   gate/up GEMM, k_vit_red_gu   times 1/rms(h1), + biases, SiLU(g) u -> bf16.
//   down GEMM, k_vit_red_down    + bias + h1 -> the slot's output row of y (bf16).
//
// The 2-D rotary angle of dim pair i (i < hd/2) of a patch at (row, col) is
// row * f_i for i < hd/4 and col * f_(i - hd/4) otherwise, f_k = theta^(-2k / (hd/2));
// cos and sin are formed in fp64 and rounded to fp32, once per call, into a table by
// position and frequency (filled by the gather kernel's first workgroups).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "fc_internal.h"

namespace fc {
namespace {

constexpr int kVitThreads = 256;
constexpr int kVitMaxPos = 128;      // patch-grid side limit (rows of the rotary table)
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
// position of item b's slot j among the rows packed across items (the many-row GEMM's
// row order: item b's rows follow those of items 0 .. b - 1)
__device__ __forceinline__ int packed_row(const int32_t *nrec, const VitGeo &g, int b, int j) {
  int p = j;
  for (int i = 0; i < b; ++i) p += n_rows(nrec, g, i);
  return p;
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

// Split-K sums of columns c .. c + 3 of row s (partials [split][rows][nc]): all SPL
// 16-byte loads issued first (indices past the last split re-read it), then summed in
// split order with the extra ones masked out.
// Sum over the splits of the float4 at p0 + sp stride, in split order, loads issued in
// groups of up to 4 (a group past the last split is skipped; `splits` is uniform).
template <int SPL>
__device__ __forceinline__ float4 sum_splits4(const float *__restrict__ p0, long stride, int splits) {
  constexpr int G = SPL < 4 ? SPL : 4;
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int g0 = 0; g0 < SPL; g0 += G) {
    if (g0 > 0 && g0 >= splits) break;
    float4 u[G];
#pragma unroll
    for (int i = 0; i < G; ++i)
      u[i] = *reinterpret_cast<const float4 *>(p0 + (long)min(g0 + i, splits - 1) * stride);
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const bool in = g0 + i < splits;
      a.x += in ? u[i].x : 0.f;
      a.y += in ? u[i].y : 0.f;
      a.z += in ? u[i].z : 0.f;
      a.w += in ? u[i].w : 0.f;
    }
  }
  return a;
}
template <int SPL>
__device__ __forceinline__ float4 sum_parts4(const float *__restrict__ part, int splits, long rows,
                                             long s, int nc, int c) {
  return sum_splits4<SPL>(part + s * nc + c, rows * nc, splits);
}
// The split-K sums a reduction reads: [split][rows][nc] rows (tiled = 0), or, from the
// many-row GEMM, [split][V][ceil(nc / 256)] tiles of [256 packed rows][256 columns] with
// the split count on the device (V: 256-row tiles of the packed rows).
struct PartIn {
  const float *part;
  int splits;          // split count (an upper bound when dsp is set)
  const int *dsp;      // device split count, or null
  int tiled;           // 1: tile layout
};
template <int SPL>
__device__ __forceinline__ float4 part_sum(const PartIn &P, int splits, long rows, long s, int prow,
                                           int V, int nc, int c) {
  if (!P.tiled) return sum_parts4<SPL>(P.part, splits, rows, s, nc, c);
  const int ntn = (nc + 255) >> 8;
  const float *p0 = P.part + ((long)((prow >> 8) * ntn + (c >> 8)) << 16) + ((prow & 255) << 8) + (c & 255);
  return sum_splits4<SPL>(p0, (long)V * ntn << 16, splits);
}

__device__ __forceinline__ float4 bf4(const uint16_t *p) {
  const uint2 u = *reinterpret_cast<const uint2 *>(p);
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}
__device__ __forceinline__ void st_bf4(uint16_t *p, float a, float b, float c, float d) {
  *reinterpret_cast<uint2 *>(p) = make_uint2(f2bf_v(a) | ((uint32_t)f2bf_v(b) << 16),
                                             f2bf_v(c) | ((uint32_t)f2bf_v(d) << 16));
}

__device__ __forceinline__ void ld_bf8(const uint16_t *p, float *v) {
  const uint4 u = *reinterpret_cast<const uint4 *>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(w[i] << 16);
    v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
  }
}
__device__ __forceinline__ void st_bf8(uint16_t *p, const float *v) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = f2bf_v(v[2 * i]) | ((uint32_t)f2bf_v(v[2 * i + 1]) << 16);
  *reinterpret_cast<uint4 *>(p) = make_uint4(w[0], w[1], w[2], w[3]);
}

// RMSNorm of one bf16 row of d <= 2048 (a multiple of 8) times a gain, by a whole
// workgroup in one pass: thread t holds columns 8 t .. 8 t + 7.
__device__ __forceinline__ void norm_row(const uint16_t *xr, const uint16_t *gain, int d, float eps,
                                         uint16_t *dst, float *red) {
  const int c = 8 * threadIdx.x;
  float v[8];
  float ss = 0.f;
  if (c < d) {
    ld_bf8(xr + c, v);
#pragma unroll
    for (int i = 0; i < 8; ++i) ss = fmaf(v[i], v[i], ss);
  }
  const float inv = 1.f / sqrtf(block_sum(ss, red) / (float)d + eps);
  if (c < d) {
    float gn[8];
    ld_bf8(gain + c, gn);
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = v[i] * inv * gn[i];
    st_bf8(dst + c, v);
  }
}

// --------------------------------------------------------------------- gather + norm
// One workgroup per slot: the patch row of x, RMSNorm (g1) as the bf16 GEMM operand; the
// item's row count.  The first workgroups also fill the rotary table (cos, sin of
// position ps times frequency fk at [ps][fk], fp64 angles), read after the QKV GEMM.
__global__ __launch_bounds__(kVitThreads) void k_vit_gather_norm(
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ g1,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, VitGeo g, float eps,
    double theta, uint16_t *__restrict__ hb, int32_t *__restrict__ rows_out,
    float2 *__restrict__ rope) {
  __shared__ float red[kVitThreads / 64];
  const long s = blockIdx.x;
  const int e = (int)s * kVitThreads + threadIdx.x;
  const int npos = max(g.gh, g.gw) * g.m;
  if (e < npos * 32) {
    const int ps = e / 32, fk = e - ps * 32;
    if (fk < g.hd / 4) {
      const double ang = (double)ps * pow(theta, -2.0 * fk / (double)(g.hd / 2));
      rope[e] = make_float2((float)cos(ang), (float)sin(ang));
    }
  }
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j == 0 && threadIdx.x == 0) rows_out[b] = n_rows(nrec, g, b);
  if (j >= n_rows(nrec, g, b)) return;
  norm_row(x + ((long)b * g.Np + slot_patch(idx, g, b, j)) * g.d, g1, g.d, eps, hb + s * g.d, red);
}

// ------------------------------------------------------------------- QKV reduction
// Grid (slot, 1024-column chunk of the 3 d q | k | v columns), 4 columns per thread:
// split-K sums + bias; q rotated at the patch position (its partner columns, half a head
// away, summed by the same thread), raw k and v into the cache at the patch row.
template <int SPL>
__global__ __launch_bounds__(kVitThreads) void k_vit_red_qkv(
    PartIn P, const uint16_t *__restrict__ bias,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, VitGeo g,
    const float2 *__restrict__ rope, uint16_t *__restrict__ q, uint16_t *__restrict__ kc,
    uint16_t *__restrict__ vc) {
  const int splits = P.dsp ? *P.dsp : P.splits;
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const int prow = packed_row(nrec, g, b, j);
  const int V = (packed_row(nrec, g, (int)(gridDim.x / g.Np), 0) + 255) >> 8;
  const int d = g.d, nc = 3 * d;
  const int c = 4 * (blockIdx.y * kVitThreads + threadIdx.x);
  if (c >= nc) return;
  const long rows = (long)gridDim.x;
  const int p = slot_patch(idx, g, b, j);
  float4 v = part_sum<SPL>(P, splits, rows, s, prow, V, nc, c);
  const float4 bb = bf4(bias + c);
  v = make_float4(v.x + bb.x, v.y + bb.y, v.z + bb.z, v.w + bb.w);
  if (c >= d) {
    const long kvrow = ((long)b * g.Np + p) * d;
    st_bf4((c < 2 * d ? kc + kvrow + (c - d) : vc + kvrow + (c - 2 * d)), v.x, v.y, v.z, v.w);
    return;
  }
  const int half = g.hd / 2, quarter = g.hd / 4;
  const int hd_i = c % g.hd;
  const int pcol = hd_i < half ? c + half : c - half;          // 4 partner columns
  float4 pv = part_sum<SPL>(P, splits, rows, s, prow, V, nc, pcol);
  const float4 pb = bf4(bias + pcol);
  const float sg = hd_i < half ? -1.f : 1.f;
  const float pp[4] = {sg * (pv.x + pb.x), sg * (pv.y + pb.y), sg * (pv.z + pb.z), sg * (pv.w + pb.w)};
  const float xv[4] = {v.x, v.y, v.z, v.w};
  int pr, pc;
  patch_pos(g, p, pr, pc);
  float o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int pair = (hd_i + i) % half;
    const float2 cs = rope[(pair < quarter ? pr : pc) * 32 + (pair < quarter ? pair : pair - quarter)];
    o[i] = xv[i] * cs.x + pp[i] * cs.y;
  }
  st_bf4(q + s * d + c, o[0], o[1], o[2], o[3]);
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

// The chunk-th group of up to 64 recomputed slots of window w (slot order), found by all
// threads in rounds of 256 slots with a ballot prefix count; returns how many there are.
__device__ int window_queries(const int32_t *idx, const VitGeo &g, int b, int w, int chunk,
                              int nrow, int *qslot, int *wcnt, int *nq_s) {
  const int t = threadIdx.x;
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
  if (t == 0) *nq_s = min(max(seen - lo, 0), kVitQ);
  __syncthreads();
  return *nq_s;
}

typedef __bf16 vbf16x8 __attribute__((ext_vector_type(8)));
typedef float vf32x4 __attribute__((ext_vector_type(4)));

// Grid: x = window * chunks_per_window + chunk, y = head, z = item; 4 waves of 16
// queries.  Per key block of 64 the workgroup stages the keys (rotated at their patch
// position, head dims zero-padded to HDP) row-major and the values transposed in LDS,
// two blocks in flight: the next block's loads are issued before this block's MFMAs.
// Each wave computes S^T = K Q^T with 16x16x32 bf16 MFMAs, so a lane's accumulators
// all belong to one query (keys 4 (lane / 16) + e of each 16-key tile) and the online
// softmax needs two cross-lane steps; P then feeds O^T = V^T P^T straight from the
// registers, the values being read from LDS in the same key order.
template <int HDP, bool PIPE>
__global__ __launch_bounds__(kVitThreads) void k_vit_attn(
    const uint16_t *__restrict__ q, const uint16_t *__restrict__ kc,
    const uint16_t *__restrict__ vc, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ nrec, VitGeo g, const float2 *__restrict__ rope, int chunks,
    uint16_t *__restrict__ out) {
  constexpr int KP = HDP + 8;          // key row pitch (bf16)
  constexpr int VP = kVitK + 8;        // transposed value row pitch (bf16)
  constexpr int NB = PIPE ? 2 : 1;     // key blocks in flight
  __shared__ __attribute__((aligned(16))) uint16_t Ks[NB][kVitK * KP];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[NB][HDP * VP];
  __shared__ int qslot[kVitQ];
  __shared__ int wcnt[kVitThreads / 64];
  __shared__ int nq_s;
  const int w = blockIdx.x / chunks, chunk = blockIdx.x - w * chunks;
  const int h = blockIdx.y, b = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, wv = t >> 6, l16 = lane & 15, gq = lane >> 4;
  const int hd = g.hd, half = hd / 2, quarter = hd / 4;
  const int nq = window_queries(idx, g, b, w, chunk, n_rows(nrec, g, b), qslot, wcnt, &nq_s);
  if (nq == 0) return;
  // padded head dims stay zero for the whole kernel
  for (int e = t; e < kVitK * (HDP - hd); e += blockDim.x) {
    const int r = e / (HDP - hd);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) Ks[nb][r * KP + hd + (e - r * (HDP - hd))] = 0;
  }
  for (int e = t; e < (HDP - hd) * VP; e += blockDim.x)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) Vt[nb][hd * VP + e] = 0;
  // this lane's query (column l16 of the wave's 16) as the B operand, dims 32 s + 8 gq..
  const int qi = wv * 16 + l16;
  const bool qv = qi < nq;
  const bool wact = wv * 16 < nq;
  vbf16x8 qf[HDP / 32];
#pragma unroll
  for (int s = 0; s < HDP / 32; ++s) {
    const int c0 = 32 * s + 8 * gq;
    uint4 raw = make_uint4(0, 0, 0, 0);
    if (qv && c0 < hd)
      raw = *reinterpret_cast<const uint4 *>(q + ((long)b * g.Np + qslot[qi]) * g.d + h * hd + c0);
    qf[s] = __builtin_bit_cast(vbf16x8, raw);
  }
  vf32x4 o[HDP / 16];
#pragma unroll
  for (int i = 0; i < HDP / 16; ++i) o[i] = vf32x4{0.f, 0.f, 0.f, 0.f};
  float mrun = -INFINITY, lpart = 0.f;
  const float scale = 1.f / sqrtf((float)hd);
  const int nk = window_keys(g, w);
  const int cpr = hd / 8;                                  // 8-dim chunks per row
  // Staging of a key block: task e (< 64 cpr) is key e / cpr, dims 8 (e % cpr) ..; the
  // raw loads of block k + 1 are issued into registers before block k's MFMAs and go
  // to the other LDS buffer (rotated) after them.
  constexpr int TASKS = (kVitK * (HDP / 8) + kVitThreads - 1) / kVitThreads;
  uint4 rk[TASKS], rp[TASKS], rv[TASKS];
  int rpatch[TASKS];
  auto load_block = [&](int k0) {
    const int kn = min(kVitK, nk - k0);
#pragma unroll
    for (int i = 0; i < TASKS; ++i) {
      const int e = t + i * kVitThreads;
      const int ki = e / cpr, c0 = (e - ki * cpr) * 8;
      rpatch[i] = -1;
      if (e < kVitK * cpr && ki < kn) {
        const int p = key_patch(g, w, k0 + ki);
        const long base = (((long)b * g.Np + p) * g.H + h) * hd;
        rk[i] = *reinterpret_cast<const uint4 *>(kc + base + c0);
        rp[i] = *reinterpret_cast<const uint4 *>(kc + base + (c0 < half ? c0 + half : c0 - half));
        rv[i] = *reinterpret_cast<const uint4 *>(vc + base + c0);
        rpatch[i] = p;
      }
    }
  };
  auto store_block = [&](int buf) {
#pragma unroll
    for (int i = 0; i < TASKS; ++i) {
      const int e = t + i * kVitThreads;
      if (e >= kVitK * cpr) continue;
      const int ki = e / cpr, c0 = (e - ki * cpr) * 8;
      uint16_t kr[8], vr[8];
      if (rpatch[i] >= 0) {
        const uint16_t *xs = reinterpret_cast<const uint16_t *>(&rk[i]);
        const uint16_t *ps = reinterpret_cast<const uint16_t *>(&rp[i]);
        const uint16_t *vs = reinterpret_cast<const uint16_t *>(&rv[i]);
        int pr, pc;
        patch_pos(g, rpatch[i], pr, pc);
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int c = c0 + q, pair = c % half;
          const float2 cs = rope[(pair < quarter ? pr : pc) * 32 + (pair < quarter ? pair : pair - quarter)];
          const float partner = c < half ? -bf2f_v(ps[q]) : bf2f_v(ps[q]);
          kr[q] = f2bf_v(bf2f_v(xs[q]) * cs.x + partner * cs.y);
          vr[q] = vs[q];
        }
      } else {
#pragma unroll
        for (int q = 0; q < 8; ++q) kr[q] = vr[q] = 0;
      }
      *reinterpret_cast<uint4 *>(Ks[buf] + ki * KP + c0) = *reinterpret_cast<const uint4 *>(kr);
#pragma unroll
      for (int q = 0; q < 8; ++q) Vt[buf][(c0 + q) * VP + ki] = vr[q];
    }
  };
  // one key block from LDS buffer buf (kn valid keys): S^T, the online softmax, O^T
  auto compute = [&](int buf, int kn) {
    vf32x4 sa[4];
#pragma unroll
    for (int kt = 0; kt < 4; ++kt) {
      sa[kt] = vf32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < HDP / 32; ++s) {
        const vbf16x8 ka = *reinterpret_cast<const vbf16x8 *>(Ks[buf] + (16 * kt + l16) * KP + 32 * s + 8 * gq);
        sa[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ka, qf[s], sa[kt], 0, 0, 0);
      }
    }
    float bmax = -INFINITY;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = (16 * kt + 4 * gq + e < kn) ? sa[kt][e] * scale : -INFINITY;
        sa[kt][e] = v;
        bmax = fmaxf(bmax, v);
      }
    bmax = fmaxf(bmax, __shfl_xor(bmax, 16));
    bmax = fmaxf(bmax, __shfl_xor(bmax, 32));
    const float mnew = fmaxf(mrun, bmax);                  // finite: kn >= 1
    const float corr = mrun == -INFINITY ? 0.f : __expf(mrun - mnew);
    float psum = 0.f;
#pragma unroll
    for (int kt = 0; kt < 4; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float pv = __expf(sa[kt][e] - mnew);
        sa[kt][e] = pv;
        psum += pv;
      }
    lpart = lpart * corr + psum;
    mrun = mnew;
#pragma unroll
    for (int i = 0; i < HDP / 16; ++i) o[i] *= corr;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      vbf16x8 pb;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        pb[e] = (__bf16)sa[2 * ks][e];
        pb[4 + e] = (__bf16)sa[2 * ks + 1][e];
      }
#pragma unroll
      for (int dt = 0; dt < HDP / 16; ++dt) {
        const uint16_t *vrow = Vt[buf] + (16 * dt + l16) * VP + 32 * ks + 4 * gq;
        const uint2 lo = *reinterpret_cast<const uint2 *>(vrow);
        const uint2 hi = *reinterpret_cast<const uint2 *>(vrow + 16);
        const vbf16x8 va = __builtin_bit_cast(vbf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, o[dt], 0, 0, 0);
      }
    }
  };
  const int nblk = (nk + kVitK - 1) / kVitK;
  if (PIPE) {
    load_block(0);
    store_block(0);
    for (int kb = 0; kb < nblk; ++kb) {
      const int k0 = kb * kVitK, buf = kb & 1;
      // block kb is in buffer buf; every reader of the other buffer (block kb - 1) is done
      __syncthreads();
      if (kb + 1 < nblk) load_block(k0 + kVitK);
      if (wact) compute(buf, min(kVitK, nk - k0));
      if (kb + 1 < nblk) store_block(buf ^ 1);
    }
  } else {
    for (int kb = 0; kb < nblk; ++kb) {
      const int k0 = kb * kVitK;
      __syncthreads();                                   // the previous block is consumed
      load_block(k0);
      store_block(0);
      __syncthreads();
      if (wact) compute(0, min(kVitK, nk - k0));
    }
  }
  if (!wact) return;
  float ltot = lpart + __shfl_xor(lpart, 16);
  ltot += __shfl_xor(ltot, 32);
  if (!qv) return;
  const float inv = 1.f / ltot;
  uint16_t *orow = out + ((long)b * g.Np + qslot[qi]) * g.d + h * hd;
#pragma unroll
  for (int dt = 0; dt < HDP / 16; ++dt) {
    const int c0 = 16 * dt + 4 * gq;
    if (c0 >= hd) continue;
    uint16_t v4[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) v4[e] = f2bf_v(o[dt][e] * inv);
    *reinterpret_cast<uint2 *>(orow + c0) = *reinterpret_cast<const uint2 *>(v4);
  }
}


// --------------------------------------------------------------- O / MLP reductions
// Grid (slot, 1024-column chunk), 4 columns per thread.  O: split-K sums + bias +
// residual -> h1 (fp32) and bf16(h1 g2), the MLP operand without its 1/rms, which the
// gate/up reduction applies to the (linear) GEMM sums; the chunk's sum of squares of h1
// goes to ssq[slot][chunk].
template <int SPL>
__global__ __launch_bounds__(kVitThreads) void k_vit_red_o(
    PartIn P, const uint16_t *__restrict__ bias,
    const uint16_t *__restrict__ x, const uint16_t *__restrict__ g2,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, VitGeo g,
    float *__restrict__ h1, uint16_t *__restrict__ hb, float *__restrict__ ssq) {
  const int splits = P.dsp ? *P.dsp : P.splits;
  __shared__ float red[kVitThreads / 64];
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const int prow = packed_row(nrec, g, b, j);
  const int V = (packed_row(nrec, g, (int)(gridDim.x / g.Np), 0) + 255) >> 8;
  const int c = 4 * (blockIdx.y * kVitThreads + threadIdx.x);
  const long rows = (long)gridDim.x;
  float ss = 0.f;
  if (c < g.d) {
    const uint16_t *xr = x + ((long)b * g.Np + slot_patch(idx, g, b, j)) * g.d;
    const float4 v = part_sum<SPL>(P, splits, rows, s, prow, V, g.d, c);
    const float4 bb = bf4(bias + c), xv = bf4(xr + c), gn = bf4(g2 + c);
    const float4 h = make_float4(xv.x + (v.x + bb.x), xv.y + (v.y + bb.y), xv.z + (v.z + bb.z),
                                 xv.w + (v.w + bb.w));
    *reinterpret_cast<float4 *>(h1 + s * g.d + c) = h;
    st_bf4(hb + s * g.d + c, h.x * gn.x, h.y * gn.y, h.z * gn.z, h.w * gn.w);
    ss = h.x * h.x + h.y * h.y + h.z * h.z + h.w * h.w;
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) ssq[s * gridDim.y + blockIdx.y] = ss;
}

// gate/up: 1/rms of h1 (from the O reduction's chunk sums) times the split-K sums, +
// biases, SiLU(g) u -> bf16
template <int SPL>
__global__ __launch_bounds__(kVitThreads) void k_vit_red_gu(
    PartIn P, const uint16_t *__restrict__ bias, int f,
    const int32_t *__restrict__ nrec, VitGeo g, const float *__restrict__ ssq, int nch, float eps,
    uint16_t *__restrict__ act) {
  const int splits = P.dsp ? *P.dsp : P.splits;
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const int prow = packed_row(nrec, g, b, j);
  const int V = (packed_row(nrec, g, (int)(gridDim.x / g.Np), 0) + 255) >> 8;
  const int c = 4 * (blockIdx.y * kVitThreads + threadIdx.x);
  if (c >= f) return;
  float sq = 0.f;
  for (int i = 0; i < nch; ++i) sq += ssq[s * nch + i];
  const float inv = 1.f / sqrtf(sq / (float)g.d + eps);
  const long rows = (long)gridDim.x;
  const float4 gs = part_sum<SPL>(P, splits, rows, s, prow, V, 2 * f, c);
  const float4 us = part_sum<SPL>(P, splits, rows, s, prow, V, 2 * f, f + c);
  const float4 gb = bf4(bias + c), ub = bf4(bias + f + c);
  const float g0 = gs.x * inv + gb.x, g1 = gs.y * inv + gb.y, g2 = gs.z * inv + gb.z,
              g3 = gs.w * inv + gb.w;
  st_bf4(act + s * f + c, g0 / (1.f + expf(-g0)) * (us.x * inv + ub.x),
         g1 / (1.f + expf(-g1)) * (us.y * inv + ub.y), g2 / (1.f + expf(-g2)) * (us.z * inv + ub.z),
         g3 / (1.f + expf(-g3)) * (us.w * inv + ub.w));
}

// down: split-K sums + bias + h1 -> the slot's output row of y (bf16)
template <int SPL>
__global__ __launch_bounds__(kVitThreads) void k_vit_red_down(
    PartIn P, const uint16_t *__restrict__ bias,
    const float *__restrict__ h1, const int32_t *__restrict__ idx,
    const int32_t *__restrict__ nrec, VitGeo g, uint16_t *__restrict__ y) {
  const int splits = P.dsp ? *P.dsp : P.splits;
  const long s = blockIdx.x;
  const int b = (int)(s / g.Np), j = (int)(s - (long)b * g.Np);
  if (j >= n_rows(nrec, g, b)) return;
  const int prow = packed_row(nrec, g, b, j);
  const int V = (packed_row(nrec, g, (int)(gridDim.x / g.Np), 0) + 255) >> 8;
  const int c = 4 * (blockIdx.y * kVitThreads + threadIdx.x);
  if (c >= g.d) return;
  uint16_t *yr = y + ((long)b * g.Np + slot_patch(idx, g, b, j)) * g.d;
  const long rows = (long)gridDim.x;
  const float4 v = part_sum<SPL>(P, splits, rows, s, prow, V, g.d, c);
  const float4 bb = bf4(bias + c);
  const float4 h = *reinterpret_cast<const float4 *>(h1 + s * g.d + c);
  st_bf4(yr + c, h.x + (v.x + bb.x), h.y + (v.y + bb.y), h.z + (v.z + bb.z), h.w + (v.w + bb.w));
}

// --------------------------------------------------------------------- patch merger
// Grid (item x recomputed token, patch): the patch row RMS-normalised, written at its
// place in the token's concatenated row (hidden = merge^2 d).
__global__ __launch_bounds__(kVitThreads) void k_merge_norm(
    const uint16_t *__restrict__ y, const uint16_t *__restrict__ gain,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, int N, int mm, int d,
    float eps, uint16_t *__restrict__ hb) {
  __shared__ float red[kVitThreads / 64];
  const long s = blockIdx.x;
  const int a = blockIdx.y;
  const int b = (int)(s / N), j = (int)(s - (long)b * N);
  if (j >= min(max(nrec[b], 0), N)) return;
  const int t = min(max(idx[s], 0), N - 1);
  norm_row(y + (((long)b * N + t) * mm + a) * d, gain, d, eps, hb + (s * mm + a) * d, red);
}

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.f + erff(v * 0.70710678118654752f));
}
// Grid (slot, 1024-column chunk): split-K sums + bias, exact GELU (x Phi(x)), bf16
template <int SPL>
__global__ __launch_bounds__(kVitThreads) void k_merge_red_gelu(
    PartIn P, const uint16_t *__restrict__ bias,
    const int32_t *__restrict__ nrec, int N, int hidden, uint16_t *__restrict__ act) {
  const int splits = P.dsp ? *P.dsp : P.splits;
  const long s = blockIdx.x;
  const int b = (int)(s / N), j = (int)(s - (long)b * N);
  if (j >= min(max(nrec[b], 0), N)) return;
  const int c = 4 * (blockIdx.y * kVitThreads + threadIdx.x);
  if (c >= hidden) return;
  const float4 v = part_sum<SPL>(P, splits, (long)gridDim.x, s, 0, 0, hidden, c);
  const float4 bb = bf4(bias + c);
  st_bf4(act + s * hidden + c, gelu_erf(bb.x + v.x), gelu_erf(bb.y + v.y), gelu_erf(bb.z + v.z),
         gelu_erf(bb.w + v.w));
}

// Grid (slot, 1024-column chunk): split-K sums + bias into the token's output row
template <int SPL>
__global__ __launch_bounds__(kVitThreads) void k_merge_red_out(
    PartIn P, const uint16_t *__restrict__ bias,
    const int32_t *__restrict__ idx, const int32_t *__restrict__ nrec, int N, int d_out,
    uint16_t *__restrict__ x_out) {
  const int splits = P.dsp ? *P.dsp : P.splits;
  const long s = blockIdx.x;
  const int b = (int)(s / N), j = (int)(s - (long)b * N);
  if (j >= min(max(nrec[b], 0), N)) return;
  const int c = 4 * (blockIdx.y * kVitThreads + threadIdx.x);
  if (c >= d_out) return;
  const int t = min(max(idx[s], 0), N - 1);
  const float4 v = part_sum<SPL>(P, splits, (long)gridDim.x, s, 0, 0, d_out, c);
  const float4 bb = bf4(bias + c);
  st_bf4(x_out + ((long)b * N + t) * d_out + c, bb.x + v.x, bb.y + v.y, bb.z + v.z, bb.w + v.w);
}

}  // namespace

// A reduction kernel instantiated for the smallest power of two >= the split count
#define FC_VIT_RED(kern, grid, ...)                                                     \
  do {                                                                                  \
    if (splits <= 1) hipLaunchKernelGGL(kern<1>, grid, dim3(kVitThreads), 0, st, __VA_ARGS__);      \
    else if (splits <= 2) hipLaunchKernelGGL(kern<2>, grid, dim3(kVitThreads), 0, st, __VA_ARGS__); \
    else if (splits <= 4) hipLaunchKernelGGL(kern<4>, grid, dim3(kVitThreads), 0, st, __VA_ARGS__); \
    else if (splits <= 8) hipLaunchKernelGGL(kern<8>, grid, dim3(kVitThreads), 0, st, __VA_ARGS__); \
    else hipLaunchKernelGGL(kern<16>, grid, dim3(kVitThreads), 0, st, __VA_ARGS__);                 \
  } while (0)

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
  int splits = 1, tiles = 0;
  const int *dsp = nullptr;
  int *ks_dev = ctx->vit_rows + ctx->caps.max_batch;
  fc_status rc;
  const dim3 red_d((unsigned)slots, (unsigned)((g.d + 1023) / 1024));
  const int nch = (g.d + 1023) / 1024;
  {
    ProfScope ps(ctx, st, "fc_vit_gather_norm");
    hipLaunchKernelGGL(k_vit_gather_norm, dim3((unsigned)slots), dim3(kVitThreads), 0, st, x, L.g1,
                       idx, nrec, g, L.rms_eps, L.rope_theta, ctx->hb, ctx->vit_rows,
                       ctx->vit_rope);
    FC_LAUNCH_OK(st, "k_vit_gather_norm");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_qkv", ctx->hb, L.w_qkv, g.d, 3 * g.d, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits, ks_dev, &dsp, &tiles)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_qkv");
    const dim3 grid((unsigned)slots, (unsigned)((3 * g.d + 1023) / 1024));
    FC_VIT_RED(k_vit_red_qkv, grid, PartIn{ctx->part, splits, dsp, tiles}, L.b_qkv, idx, nrec, g,
               (const float2 *)ctx->vit_rope, ctx->qbuf, c.k, c.v);
    FC_LAUNCH_OK(st, "k_vit_red_qkv");
  }
  {
    // query chunks of 64 per window (full attention: one window of every patch)
    const int nwin = c.window > 0 ? ((g.gh + c.window - 1) / c.window) * ((g.gw + c.window - 1) / c.window) : 1;
    const int wkeys = c.window > 0 ? std::min(c.window, g.gh) * std::min(c.window, g.gw) * g.mm : g.Np;
    const int chunks = (wkeys + kVitQ - 1) / kVitQ;
    const dim3 grid((unsigned)(nwin * chunks), (unsigned)g.H, (unsigned)B);
    const uint16_t *qb = ctx->qbuf, *kb = c.k, *vb = c.v;
    const float2 *rp = ctx->vit_rope;
    ProfScope ps(ctx, st, "fc_vit_attn");
    // more than one key block per workgroup: two blocks in flight
    const bool pipe = wkeys > kVitK;
#define FC_VIT_ATTN(HDP)                                                                      \
  do {                                                                                        \
    if (pipe)                                                                                 \
      hipLaunchKernelGGL((k_vit_attn<HDP, true>), grid, dim3(kVitThreads), 0, st, qb, kb, vb, idx, nrec, g, rp, chunks, ctx->attn); \
    else                                                                                      \
      hipLaunchKernelGGL((k_vit_attn<HDP, false>), grid, dim3(kVitThreads), 0, st, qb, kb, vb, idx, nrec, g, rp, chunks, ctx->attn); \
  } while (0)
    if (g.hd <= 32) FC_VIT_ATTN(32);
    else if (g.hd <= 64) FC_VIT_ATTN(64);
    else if (g.hd <= 96) FC_VIT_ATTN(96);
    else FC_VIT_ATTN(128);
#undef FC_VIT_ATTN
    FC_LAUNCH_OK(st, "k_vit_attn");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_o", ctx->attn, L.w_o, g.d, g.d, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits, ks_dev, &dsp, &tiles)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_o");
    FC_VIT_RED(k_vit_red_o, red_d, PartIn{ctx->part, splits, dsp, tiles}, L.b_o, x, L.g2, idx, nrec, g,
               ctx->h1, ctx->hb, ctx->ssq);
    FC_LAUNCH_OK(st, "k_vit_red_o");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_gateup", ctx->hb, L.w_gate_up, g.d, 2 * f, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits, ks_dev, &dsp, &tiles)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_gu");
    const dim3 grid((unsigned)slots, (unsigned)((f + 1023) / 1024));
    FC_VIT_RED(k_vit_red_gu, grid, PartIn{ctx->part, splits, dsp, tiles}, L.b_gate_up, f, nrec, g,
               (const float *)ctx->ssq, nch, L.rms_eps, ctx->act);
    FC_LAUNCH_OK(st, "k_vit_red_gu");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_vit_gemm_down", ctx->act, L.w_down, f, g.d, g.Np,
                           ctx->vit_rows, ctx->part, B, &splits, ks_dev, &dsp, &tiles)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_vit_red_down");
    FC_VIT_RED(k_vit_red_down, red_d, PartIn{ctx->part, splits, dsp, tiles}, L.b_down,
               (const float *)ctx->h1, idx, nrec, g, y);
    FC_LAUNCH_OK(st, "k_vit_red_down");
  }
  return FC_OK;
}

fc_status launch_vit_cache_update(fc_ctx *ctx, const fc_vit_desc &L, const fc_vit_cache &c,
                                  const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                                  const uint8_t *reuse, int B, hipStream_t st) {
  // a merged token's patch rows are contiguous: the token-level remap with rows of
  // m^2 patches, from a separate previous-frame cache, or in place in the one frame
  // slot (whose overwrite stages the old rows)
  const int mm = c.merge * c.merge;
  if (c.k_prev)
    return launch_remap_copy(ctx, c.k_prev, c.v_prev, c.k, c.v, y_prev, y_cur,
                             c.grid_h * c.grid_w, mm * L.d_model, mm * L.d_model, c.grid_w,
                             shift, reuse, B, st);
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
  int splits = 1, tiles = 0;
  const int *dsp = nullptr;
  fc_status rc;
  {
    ProfScope ps(ctx, st, "fc_merge_norm");
    hipLaunchKernelGGL(k_merge_norm, dim3((unsigned)slots, (unsigned)mm), dim3(kVitThreads), 0, st,
                       y, M.g, idx, nrec, N, mm, M.d_model, M.rms_eps, hb);
    FC_LAUNCH_OK(st, "k_merge_norm");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_merge_gemm1", hb, M.w1, hidden, hidden, N, nrec,
                           ctx->part, B, &splits, nullptr, &dsp, &tiles)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_merge_red_gelu");
    const dim3 grid((unsigned)slots, (unsigned)((hidden + 1023) / 1024));
    FC_VIT_RED(k_merge_red_gelu, grid, PartIn{ctx->part, splits, dsp, tiles}, M.b1, nrec, N, hidden,
               act);
    FC_LAUNCH_OK(st, "k_merge_red_gelu");
  }
  if ((rc = run_plain_gemm(ctx, st, "fc_merge_gemm2", act, M.w2, hidden, M.d_out, N, nrec,
                           ctx->part, B, &splits, nullptr, &dsp, &tiles)) != FC_OK)
    return rc;
  {
    ProfScope ps(ctx, st, "fc_merge_red_out");
    const dim3 grid((unsigned)slots, (unsigned)((M.d_out + 1023) / 1024));
    FC_VIT_RED(k_merge_red_out, grid, PartIn{ctx->part, splits, dsp, tiles}, M.b2, idx, nrec, N,
               M.d_out, x_out);
    FC_LAUNCH_OK(st, "k_merge_red_out");
  }
  return FC_OK;
}

}  // namespace fc
