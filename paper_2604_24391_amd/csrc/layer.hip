// Partial-recompute decoder layer and token-cache remap on gfx950.
//
// Rows of the layer are "slots": slot r = b * N + j holds the j-th recomputed
// token of batch item b, j < n_recompute[b] (read on the device, so no host
// sync); grids are sized for N rows per item and surplus tiles exit.
//
//   k_gemm      bf16 MFMA (v_mfma_f32_32x32x16_bf16) GEMM  C = A W^T, W row-major
//               [out][in] like torch.nn.Linear.  128x128x32 tiles, 4 waves of
//               64x64, LDS double buffer.  A rows are gathered through the
//               recompute ids inside the tile load (optionally scaled by an
//               RMSNorm gain and converted from float32).  Either writes float32
//               split-K partial sums, or (SwiGLU mode) interleaves gate and up
//               rows in one tile and applies SiLU(g) * u in the epilogue.
//   k_epi_qkv   sums the split-K partials, applies 1/rms(x) and the q/k/v bias,
//               stores q (pre-RoPE) and scatters raw k and v into the current
//               frame's cache rows.
//   k_attn      attention of the gathered queries over the whole cache, GQA
//               (one wave per query head of a KV group), RoPE applied to q and to
//               each key block as it is staged in LDS, causal by position, float32
//               online softmax in the transposed form S^T = K Q^T so that a lane
//               owns one query column.  Optional split over key blocks.
//   k_attn_combine  merges split-KV partials.
//   k_epi_o     residual add, h1 in float32, 1/rms(h1) for the MLP norm.
//   k_epi_down  residual add, bf16 output scattered into the output cache.
//   k_cache_update  copies cached K/V/output rows of each reused token from its
//               aligned source token.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "fc_internal.h"

namespace fc {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) {
  // round to nearest even (inputs are finite)
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

struct alignas(16) U16x8 {
  uint16_t v[8];
};

// Device-side counts and ids come from fc_select; clamp them so that a caller
// passing anything else can never make a kernel leave its buffers.
__device__ __forceinline__ int n_valid(const int32_t *nrec, int b, int N) {
  return min(max(nrec[b], 0), N);
}
__device__ __forceinline__ int tok_of(const int32_t *idx, long slot, int N) {
  return min(max(idx[slot], 0), N - 1);
}

// ------------------------------------------------------------------------------- GEMM
constexpr int BM = kGemmBM, BN = kGemmBN, BK = kGemmBK;
constexpr int LDA = BK + 8;  // LDS row stride in bf16 (16-B pad)

struct GemmArgs {
  const void *A;             // activations; bf16 or float32
  int a_f32;                 // 1: A is float32
  int gather;                // 1: A row of slot (b, j) is b*N + idx[b*N + j]; 0: the slot itself
  const uint16_t *gain;      // [K] multiplied into A (RMSNorm gain), or null
  const uint16_t *W0;        // weights [rows][K]
  const uint16_t *W1;        // SwiGLU: up weights (W0 = gate)
  int swiglu;
  int K, Nout;               // reduction length, output columns
  int kchunk, splits;
  int N;                     // slots per batch item
  const int32_t *idx, *nrec;
  int m_tiles, n_tiles;
  float *C;                  // [split][B*N][Nout] partial sums (non-SwiGLU)
  uint16_t *act;             // [B*N][Nout] SwiGLU output
  const float *row_scale;    // [B*N] 1/rms applied to gate and up (SwiGLU)
};

// Workgroup id -> tile id so that each XCD (workgroups are dealt round-robin over
// the 8 XCDs) works on a contiguous range of tiles, M fastest: the M tiles that
// share a weight tile then run on the same XCD and share its L2.
__device__ __forceinline__ int xcd_tile(int w, int total) {
  const int per = total / 8;
  if (w >= per * 8) return w;
  return (w & 7) * per + (w >> 3);
}

__global__ __launch_bounds__(256) void k_gemm(GemmArgs a) {
  __shared__ __bf16 As[2][BM * LDA];
  __shared__ __bf16 Bs[2][BN * LDA];
  const int total = a.m_tiles * a.n_tiles * a.splits;
  const int tile = xcd_tile(blockIdx.x, total);
  const int mt = tile % a.m_tiles;
  const int nt = (tile / a.m_tiles) % a.n_tiles;
  const int sp = tile / (a.m_tiles * a.n_tiles);
  const int tpb = (a.N + BM - 1) / BM;
  const int b = mt / tpb;
  const int row0 = (mt % tpb) * BM;
  const int nvalid = min(BM, n_valid(a.nrec, b, a.N) - row0);
  if (nvalid <= 0) return;
  const int k0 = sp * a.kchunk;
  const int k1 = min(a.K, k0 + a.kchunk);
  if (k0 >= k1) return;
  const int nk = (k1 - k0) / BK;

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, hi = lane >> 5;

  // per-thread load assignments: 2 chunks of 8 elements for A and for B
  const void *a_src[2];
  const uint16_t *b_src[2];
  int a_row[2], a_kc[2], b_row[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = t + 256 * i;
    a_row[i] = c >> 2;
    a_kc[i] = (c & 3) * 8;
    b_row[i] = c >> 2;
    const int r = a_row[i];
    a_src[i] = nullptr;
    if (r < nvalid) {
      const int slot_j = row0 + r;
      const long src_row = a.gather ? (long)b * a.N + tok_of(a.idx, (long)b * a.N + slot_j, a.N)
                                    : (long)b * a.N + slot_j;
      if (a.a_f32)
        a_src[i] = (const float *)a.A + src_row * a.K;
      else
        a_src[i] = (const uint16_t *)a.A + src_row * a.K;
    }
    const int br = b_row[i];
    const uint16_t *wp = nullptr;
    if (a.swiglu) {
      const int n = nt * (BN / 2) + (br & 63);
      if (n < a.Nout) wp = (br < 64 ? a.W0 : a.W1) + (long)n * a.K;
    } else {
      const int n = nt * BN + br;
      if (n < a.Nout) wp = a.W0 + (long)n * a.K;
    }
    b_src[i] = wp;
  }

  U16x8 ra[2], rb[2];
  auto load_tile = [&](int kk) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int kbase = kk + a_kc[i];
      if (a_src[i]) {
        if (a.a_f32) {
          const float *p = (const float *)a_src[i] + kbase;
          const float4 x0 = *reinterpret_cast<const float4 *>(p);
          const float4 x1 = *reinterpret_cast<const float4 *>(p + 4);
          float v[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
          if (a.gain) {
            const U16x8 gg = *reinterpret_cast<const U16x8 *>(a.gain + kbase);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] *= bf2f(gg.v[e]);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) ra[i].v[e] = f2bf(v[e]);
        } else {
          ra[i] = *reinterpret_cast<const U16x8 *>((const uint16_t *)a_src[i] + kbase);
          if (a.gain) {
            const U16x8 gg = *reinterpret_cast<const U16x8 *>(a.gain + kbase);
#pragma unroll
            for (int e = 0; e < 8; ++e) ra[i].v[e] = f2bf(bf2f(ra[i].v[e]) * bf2f(gg.v[e]));
          }
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) ra[i].v[e] = 0;
      }
      if (b_src[i]) {
        rb[i] = *reinterpret_cast<const U16x8 *>(b_src[i] + kk + a_kc[i]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) rb[i].v[e] = 0;
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *reinterpret_cast<U16x8 *>(&As[buf][a_row[i] * LDA + a_kc[i]]) = ra[i];
      *reinterpret_cast<U16x8 *>(&Bs[buf][b_row[i] * LDA + a_kc[i]]) = rb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // rows of this wave's two 32-row blocks that hold valid slots
  const bool act0 = wm * 64 < nvalid, act1 = wm * 64 + 32 < nvalid;
  // LDS rows of this wave's two B blocks
  const int brow0 = a.swiglu ? wn * 32 : wn * 64;
  const int brow1 = a.swiglu ? 64 + wn * 32 : wn * 64 + 32;

  load_tile(k0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tile(k0 + (kt + 1) * BK);
    if (act0) {
#pragma unroll
      for (int ks = 0; ks < BK / 16; ++ks) {
        const int ko = ks * 16 + hi * 8;
        const bf16x8 b0 = *reinterpret_cast<const bf16x8 *>(&Bs[buf][(brow0 + l32) * LDA + ko]);
        const bf16x8 b1 = *reinterpret_cast<const bf16x8 *>(&Bs[buf][(brow1 + l32) * LDA + ko]);
        const bf16x8 a0 = *reinterpret_cast<const bf16x8 *>(&As[buf][(wm * 64 + l32) * LDA + ko]);
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
        if (act1) {
          const bf16x8 a1 =
              *reinterpret_cast<const bf16x8 *>(&As[buf][(wm * 64 + 32 + l32) * LDA + ko]);
          acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
          acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
        }
      }
    }
    if (kt + 1 < nk) store_tile(buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds column l32 and rows (e/4)*8 + hi*4 + e%4 of each 32x32 block
  const long slot_base = (long)b * a.N + row0;
  if (a.swiglu) {
    const int col = nt * (BN / 2) + wn * 32 + l32;
    if (col >= a.Nout) return;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int r = wm * 64 + i * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
        if (r < nvalid) {
          const float s = a.row_scale[slot_base + r];
          const float gv = acc[i][0][e] * s, uv = acc[i][1][e] * s;
          const float y = gv / (1.f + __expf(-gv)) * uv;
          a.act[(slot_base + r) * a.Nout + col] = f2bf(y);
        }
      }
    }
  } else {
    const long plane = (long)(a.m_tiles / ((a.N + BM - 1) / BM)) * a.N;  // B*N rows
    float *Cs = a.C + (long)sp * plane * a.Nout;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = nt * BN + wn * 64 + j * 32 + l32;
      if (col >= a.Nout) continue;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int r = wm * 64 + i * 32 + (e >> 2) * 8 + hi * 4 + (e & 3);
          if (r < nvalid) Cs[(slot_base + r) * a.Nout + col] = acc[i][j][e];
        }
      }
    }
  }
}

// ------------------------------------------------------------------------------- epilogues
__device__ float block_sum256(float v, float *red) {
  const int t = threadIdx.x;
  red[t] = v;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if (t < s) red[t] += red[t + s];
    __syncthreads();
  }
  const float r = red[0];
  __syncthreads();
  return r;
}

struct EpiArgs {
  int N, d, nh, nkv, hd;
  int splits, ncols;
  float eps;
  const int32_t *idx, *nrec;
  const float *part;           // [split][B*N][ncols]
  const uint16_t *x;           // [B][N][d] layer input (bf16)
  const uint16_t *bias;        // [qkv]
  uint16_t *q;                 // [B*N][nh*hd]
  uint16_t *kc, *vc;           // cache [B][S][nkv][hd]
  int S, cur_row0;             // rows of the current frame start at T + cur_slot * N
  float *h1;                   // [B*N][d]
  float *inv2;                 // [B*N]
  uint16_t *y;                 // [B][N][d]
};

__device__ __forceinline__ float sum_splits(const EpiArgs &e, long slot, int c, long plane) {
  float v = 0.f;
  for (int s = 0; s < e.splits; ++s) v += e.part[(long)s * plane * e.ncols + slot * e.ncols + c];
  return v;
}

__global__ __launch_bounds__(256) void k_epi_qkv(EpiArgs e, int B) {
  __shared__ float red[256];
  const int slot = blockIdx.x;
  const int b = slot / e.N, j = slot - b * e.N;
  if (j >= n_valid(e.nrec, b, e.N)) return;
  const int tok = tok_of(e.idx, slot, e.N);
  const uint16_t *xr = e.x + ((long)b * e.N + tok) * e.d;
  float ss = 0.f;
  for (int c = threadIdx.x; c < e.d; c += 256) {
    const float v = bf2f(xr[c]);
    ss += v * v;
  }
  ss = block_sum256(ss, red);
  const float inv = 1.f / sqrtf(ss / (float)e.d + e.eps);
  const long plane = (long)B * e.N;
  const int qw = e.nh * e.hd, kw = e.nkv * e.hd;
  const long crow = (long)b * e.S + e.cur_row0 + tok;
  for (int c = threadIdx.x; c < e.ncols; c += 256) {
    const float v = sum_splits(e, slot, c, plane) * inv + bf2f(e.bias[c]);
    if (c < qw)
      e.q[(long)slot * qw + c] = f2bf(v);
    else if (c < qw + kw)
      e.kc[crow * kw + (c - qw)] = f2bf(v);
    else
      e.vc[crow * kw + (c - qw - kw)] = f2bf(v);
  }
}

__global__ __launch_bounds__(256) void k_epi_o(EpiArgs e, int B) {
  __shared__ float red[256];
  const int slot = blockIdx.x;
  const int b = slot / e.N, j = slot - b * e.N;
  if (j >= n_valid(e.nrec, b, e.N)) return;
  const int tok = tok_of(e.idx, slot, e.N);
  const uint16_t *xr = e.x + ((long)b * e.N + tok) * e.d;
  const long plane = (long)B * e.N;
  float ss = 0.f;
  for (int c = threadIdx.x; c < e.d; c += 256) {
    const float v = bf2f(xr[c]) + sum_splits(e, slot, c, plane);
    e.h1[(long)slot * e.d + c] = v;
    ss += v * v;
  }
  ss = block_sum256(ss, red);
  if (threadIdx.x == 0) e.inv2[slot] = 1.f / sqrtf(ss / (float)e.d + e.eps);
}

__global__ __launch_bounds__(256) void k_epi_down(EpiArgs e, int B) {
  const int slot = blockIdx.x;
  const int b = slot / e.N, j = slot - b * e.N;
  if (j >= n_valid(e.nrec, b, e.N)) return;
  const int tok = tok_of(e.idx, slot, e.N);
  const long plane = (long)B * e.N;
  uint16_t *yr = e.y + ((long)b * e.N + tok) * e.d;
  for (int c = threadIdx.x; c < e.d; c += 256)
    yr[c] = f2bf(e.h1[(long)slot * e.d + c] + sum_splits(e, slot, c, plane));
}

// ------------------------------------------------------------------------------- attention
struct AttnArgs {
  const uint16_t *q;          // [B*N][nh*HD] pre-RoPE
  const uint16_t *kc, *vc;    // [B][S][nkv][HD]
  const float2 *rope;         // [S][HD/2] (cos, sin)
  const int32_t *idx, *nrec;
  int N, nh, nkv, S, T, W, head;
  int splits, kb_per_split;
  float scale_log2;
  uint16_t *out;              // [B*N][nh*HD] (splits == 1)
  float *po;                  // [split][B*N][nh][HD] unnormalised partial output
  float *pm, *pl;             // [split][B*N][nh] running max (log2 units) and sum
};

__device__ __forceinline__ int key_pos(int row, int T, int N, int W, int head) {
  if (row < T) return row;
  const int r = row - T;
  const int p = r / N, i = r - p * N;
  int lg = p - head;
  if (lg < 0) lg += W;
  return T + lg * N + i;
}

template <int HD, int G>
__global__ __launch_bounds__(G * 64) void k_attn(AttnArgs a) {
  constexpr int NS = HD / 16;   // k-steps of the QK^T product
  constexpr int NHB = HD / 32;  // 32-row blocks of the output
  __shared__ __bf16 Ks[32 * (HD + 8)];
  __shared__ __bf16 Vt[HD * 40];
  __shared__ int kpos[32];

  const int tiles_per_b = (a.N + 31) / 32;
  const int b = blockIdx.x / tiles_per_b;
  const int j0 = (blockIdx.x % tiles_per_b) * 32;
  const int n = n_valid(a.nrec, b, a.N);
  if (j0 >= n) return;
  const int g = blockIdx.y;
  const int sp = blockIdx.z;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const int h = g * G + w;

  const int j = j0 + l32;
  const bool qvalid = j < n;
  const long slot = (long)b * a.N + (qvalid ? j : j0);
  const int tok = tok_of(a.idx, slot, a.N);
  const int qpos = a.T + (a.W - 1) * a.N + tok;

  // Q fragments (B operand of S^T = K Q^T): lane holds q[16 s + 8 hi + e]
  float qf[NS][8];
  {
    const uint16_t *qr = a.q + slot * (long)(a.nh * HD) + h * HD;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const U16x8 v = *reinterpret_cast<const U16x8 *>(qr + 16 * s + 8 * hi);
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[s][e] = bf2f(v.v[e]);
    }
    // rotate-half RoPE: dims d and d + HD/2 sit in steps s and s + NS/2 of this lane
    const float2 *rp = a.rope + (long)qpos * (HD / 2);
#pragma unroll
    for (int s = 0; s < NS / 2; ++s)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float2 cs = rp[16 * s + 8 * hi + e];
        const float x1 = qf[s][e], x2 = qf[s + NS / 2][e];
        qf[s][e] = x1 * cs.x - x2 * cs.y;
        qf[s + NS / 2][e] = x2 * cs.x + x1 * cs.y;
      }
  }
  bf16x8 qb[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s)
#pragma unroll
    for (int e = 0; e < 8; ++e) qb[s][e] = (__bf16)qf[s][e];

  f32x16 o[NHB];
#pragma unroll
  for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
    for (int e = 0; e < 16; ++e) o[hb][e] = 0.f;
  float m_run = -INFINITY, l_run = 0.f;

  const int nkb = (a.S + 31) / 32;
  const int kb0 = sp * a.kb_per_split;
  const int kb1 = min(nkb, kb0 + a.kb_per_split);
  const long kvbase = (long)b * a.S * a.nkv * HD + (long)g * HD;
  const long kvrow = (long)a.nkv * HD;

  for (int kb = kb0; kb < kb1; ++kb) {
    __syncthreads();
    // stage 32 keys (rotated) and values (transposed) of kv head g
    for (int task = t; task < 32 * (HD / 16); task += G * 64) {
      const int key = task / (HD / 16), c = task - key * (HD / 16);
      const int row = kb * 32 + key;
      U16x8 k1, k2, v1, v2;
      if (row < a.S) {
        const int pos = key_pos(row, a.T, a.N, a.W, a.head);
        if (c == 0) kpos[key] = pos;
        const uint16_t *kp = a.kc + kvbase + row * kvrow;
        const uint16_t *vp = a.vc + kvbase + row * kvrow;
        k1 = *reinterpret_cast<const U16x8 *>(kp + 8 * c);
        k2 = *reinterpret_cast<const U16x8 *>(kp + HD / 2 + 8 * c);
        v1 = *reinterpret_cast<const U16x8 *>(vp + 8 * c);
        v2 = *reinterpret_cast<const U16x8 *>(vp + HD / 2 + 8 * c);
        const float2 *rp = a.rope + (long)pos * (HD / 2) + 8 * c;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float2 cs = rp[e];
          const float x1 = bf2f(k1.v[e]), x2 = bf2f(k2.v[e]);
          k1.v[e] = f2bf(x1 * cs.x - x2 * cs.y);
          k2.v[e] = f2bf(x2 * cs.x + x1 * cs.y);
        }
      } else {
        if (c == 0) kpos[key] = 0x7fffffff;
#pragma unroll
        for (int e = 0; e < 8; ++e) k1.v[e] = k2.v[e] = v1.v[e] = v2.v[e] = 0;
      }
      *reinterpret_cast<U16x8 *>(&Ks[key * (HD + 8) + 8 * c]) = k1;
      *reinterpret_cast<U16x8 *>(&Ks[key * (HD + 8) + HD / 2 + 8 * c]) = k2;
      uint16_t *vt = reinterpret_cast<uint16_t *>(Vt);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        vt[(8 * c + e) * 40 + key] = v1.v[e];
        vt[(HD / 2 + 8 * c + e) * 40 + key] = v2.v[e];
      }
    }
    __syncthreads();

    // S^T block: rows = 32 keys, columns = 32 queries
    f32x16 st;
#pragma unroll
    for (int e = 0; e < 16; ++e) st[e] = 0.f;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(&Ks[l32 * (HD + 8) + 16 * s + 8 * hi]);
      st = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qb[s], st, 0, 0, 0);
    }
    float mloc = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = (e >> 2) * 8 + hi * 4 + (e & 3);
      const float v = (kpos[key] <= qpos) ? st[e] * a.scale_log2 : -INFINITY;
      st[e] = v;
      mloc = fmaxf(mloc, v);
    }
    mloc = fmaxf(mloc, __shfl_xor(mloc, 32));
    const float m_new = fmaxf(m_run, mloc);
    const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
    const float corr = exp2f(m_run - m_use);
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      st[e] = exp2f(st[e] - m_use);
      psum += st[e];
    }
    l_run = l_run * corr + psum;
    m_run = m_new;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[hb][e] *= corr;
    // O^T += V^T P^T; k index (8 hi + i) of step s2 <-> key 16 s2 + 8 (i/4) + 4 hi + i%4,
    // which is exactly accumulator element 8 s2 + i of S^T in this lane.
    const uint16_t *vt = reinterpret_cast<const uint16_t *>(Vt);
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8 pb;
#pragma unroll
      for (int i = 0; i < 8; ++i) pb[i] = (__bf16)st[8 * s2 + i];
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) {
        const uint16_t *vr = vt + (hb * 32 + l32) * 40 + 16 * s2 + 4 * hi;
        const uint2 lo = *reinterpret_cast<const uint2 *>(vr);
        const uint2 hi8 = *reinterpret_cast<const uint2 *>(vr + 8);
        bf16x8 va;
        const uint32_t w4[4] = {lo.x, lo.y, hi8.x, hi8.y};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          va[2 * i] = __builtin_bit_cast(__bf16, (uint16_t)(w4[i] & 0xFFFF));
          va[2 * i + 1] = __builtin_bit_cast(__bf16, (uint16_t)(w4[i] >> 16));
        }
        o[hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[hb], 0, 0, 0);
      }
    }
  }

  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!qvalid) return;
  if (a.splits == 1) {
    uint16_t *orow = a.out + slot * (long)(a.nh * HD) + h * HD;
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        orow[hb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3)] = f2bf(o[hb][e] * inv);
  } else {
    const long plane = (long)gridDim.x / tiles_per_b * a.N;  // B*N
    const long pr = ((long)sp * plane + slot) * a.nh + h;
    float *orow = a.po + pr * HD;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int e = 0; e < 16; ++e) orow[hb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3)] = o[hb][e];
    if (hi == 0) {
      a.pm[pr] = m_run;
      a.pl[pr] = l_tot;
    }
  }
}

__global__ __launch_bounds__(128) void k_attn_combine(AttnArgs a, int HD, int B) {
  const long slot = blockIdx.x;
  const int b = (int)(slot / a.N), j = (int)(slot - (long)b * a.N);
  if (j >= n_valid(a.nrec, b, a.N)) return;
  const int h = blockIdx.y;
  const long plane = (long)B * a.N;
  float mx = -INFINITY;
  for (int s = 0; s < a.splits; ++s) mx = fmaxf(mx, a.pm[((long)s * plane + slot) * a.nh + h]);
  const float mu = (mx == -INFINITY) ? 0.f : mx;
  float l = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const long pr = ((long)s * plane + slot) * a.nh + h;
    l += a.pl[pr] * exp2f(a.pm[pr] - mu);
  }
  const float inv = l > 0.f ? 1.f / l : 0.f;
  for (int d = threadIdx.x; d < HD; d += blockDim.x) {
    float v = 0.f;
    for (int s = 0; s < a.splits; ++s) {
      const long pr = ((long)s * plane + slot) * a.nh + h;
      v += a.po[pr * HD + d] * exp2f(a.pm[pr] - mu);
    }
    a.out[slot * (long)(a.nh * HD) + h * HD + d] = f2bf(v * inv);
  }
}

// ------------------------------------------------------------------------------- rope table
__global__ void k_rope_table(float2 *tab, int S, int half, int hd, double theta) {
  const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= (long)S * half) return;
  const int pos = (int)(e / half), i = (int)(e - (long)pos * half);
  const double inv = pow(theta, -(2.0 * i) / (double)hd);
  double s, c;
  sincos((double)pos * inv, &s, &c);
  tab[e] = make_float2((float)c, (float)s);
}

// ------------------------------------------------------------------------------- cache update
__global__ void k_copy16(const uint4 *__restrict__ src, uint4 *__restrict__ dst, long n16) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n16) dst[i] = src[i];
}

struct CacheArgs {
  uint16_t *kc, *vc;             // [B][S][kvw]
  const uint16_t *ksrc, *vsrc;   // previous-frame rows: cache rows, or the staging copy
  long src_bstride;              // elements between batch items in ksrc / vsrc
  long src_row0;                 // first previous-frame row in ksrc / vsrc (per item)
  const uint16_t *y_prev;
  uint16_t *y_cur;
  const int32_t *shift;
  const uint8_t *reuse;
  int N, S, kvw, d, gw, gh, cur_row0;
};

__global__ __launch_bounds__(256) void k_cache_update(CacheArgs c) {
  const int b = blockIdx.y;
  const int tok = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (tok >= c.N) return;
  if (!c.reuse[(long)b * c.N + tok]) return;
  const int I = tok / c.gw, J = tok - I * c.gw;
  const int si = I + c.shift[b * 2], sj = J + c.shift[b * 2 + 1];
  if (si < 0 || si >= c.gh || sj < 0 || sj >= c.gw) return;  // never for a valid mask
  const int src = si * c.gw + sj;
  const long drow = (long)b * c.S + c.cur_row0 + tok;
  const long srow = (long)b * c.src_bstride / c.kvw + c.src_row0 + src;
  const uint4 *ks = reinterpret_cast<const uint4 *>(c.ksrc + srow * c.kvw);
  const uint4 *vs = reinterpret_cast<const uint4 *>(c.vsrc + srow * c.kvw);
  uint4 *kd = reinterpret_cast<uint4 *>(c.kc + drow * c.kvw);
  uint4 *vd = reinterpret_cast<uint4 *>(c.vc + drow * c.kvw);
  for (int e = lane; e < c.kvw / 8; e += 64) {
    kd[e] = ks[e];
    vd[e] = vs[e];
  }
  const uint4 *ys = reinterpret_cast<const uint4 *>(c.y_prev + ((long)b * c.N + src) * c.d);
  uint4 *yd = reinterpret_cast<uint4 *>(c.y_cur + ((long)b * c.N + tok) * c.d);
  for (int e = lane; e < c.d / 8; e += 64) yd[e] = ys[e];
}

int pick_splits(int tiles, int K, int want_wgs, long rows, int ncols, size_t cap_elems) {
  int s = std::max(1, std::min(kMaxSplits, (want_wgs + tiles - 1) / tiles));
  s = std::min(s, std::max(1, K / (4 * BK)));
  while (s > 1 && (size_t)s * rows * ncols > cap_elems) --s;
  return s;
}

fc_status run_gemm(fc_ctx *ctx, hipStream_t st, const char *name, GemmArgs g, int B) {
  g.m_tiles = B * ((g.N + BM - 1) / BM);
  if (g.swiglu)
    g.n_tiles = (g.Nout + BN / 2 - 1) / (BN / 2);
  else
    g.n_tiles = (g.Nout + BN - 1) / BN;
  // split-K chunk, a multiple of BK
  const int kc = ((g.K + g.splits - 1) / g.splits + BK - 1) / BK * BK;
  g.kchunk = kc;
  g.splits = (g.K + kc - 1) / kc;
  const int total = g.m_tiles * g.n_tiles * g.splits;
  ProfScope ps(ctx, st, name);
  hipLaunchKernelGGL(k_gemm, dim3(total), dim3(256), 0, st, g);
  FC_HIP_TRY(hipGetLastError());
  return FC_OK;
}

}  // namespace

fc_status launch_layer(fc_ctx *ctx, const fc_layer_desc &L, const fc_kv_cache &kv,
                       const uint16_t *x_cur, const int32_t *idx, const int32_t *nrec,
                       uint16_t *y_cur, int B, hipStream_t st) {
  const int N = kv.frame_tokens, d = L.d_model, nh = L.n_heads, nkv = L.n_kv_heads,
            hd = L.head_dim, ffn = L.d_ffn;
  const int S = kv.text_tokens + kv.window * N;
  const int qkv = (nh + 2 * nkv) * hd;
  const long rows = (long)B * N;
  const int cur_slot = (kv.head + kv.window - 1) % kv.window;
  const int cur_row0 = kv.text_tokens + cur_slot * N;

  // RoPE table for (hd, theta) over the cache length (rebuilt only when they change)
  if (ctx->rope_hd != hd || ctx->rope_theta != L.rope_theta || ctx->rope_seq < S) {
    const int seq = ctx->caps.max_seq;
    const long n = (long)seq * (hd / 2);
    ProfScope ps(ctx, st, "fc_rope_table");
    hipLaunchKernelGGL(k_rope_table, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                       ctx->rope, seq, hd / 2, hd, L.rope_theta);
    FC_HIP_TRY(hipGetLastError());
    ctx->rope_hd = hd;
    ctx->rope_theta = L.rope_theta;
    ctx->rope_seq = seq;
  }

  const int mt = B * ((N + BM - 1) / BM);
  const int want = 2 * std::max(ctx->num_cus, 1);

  // 1. gathered RMSNorm (gain in the tile load, 1/rms in the epilogue) + QKV
  GemmArgs g{};
  g.A = x_cur;
  g.a_f32 = 0;
  g.gather = 1;
  g.gain = L.g_attn;
  g.W0 = L.w_qkv;
  g.K = d;
  g.Nout = qkv;
  g.N = N;
  g.idx = idx;
  g.nrec = nrec;
  g.C = ctx->part;
  g.splits = pick_splits(mt * ((qkv + BN - 1) / BN), d, want, rows, qkv, ctx->part_elems);
  const int s_qkv = g.splits;
  fc_status rc = run_gemm(ctx, st, "fc_gemm_qkv", g, B);
  if (rc != FC_OK) return rc;
  {
    // the GEMM may have rounded the split count; recompute what it used
    const int kc = ((d + s_qkv - 1) / s_qkv + BK - 1) / BK * BK;
    EpiArgs e{};
    e.N = N; e.d = d; e.nh = nh; e.nkv = nkv; e.hd = hd;
    e.splits = (d + kc - 1) / kc;
    e.ncols = qkv;
    e.eps = L.rms_eps;
    e.idx = idx; e.nrec = nrec;
    e.part = ctx->part;
    e.x = x_cur;
    e.bias = L.b_qkv;
    e.q = ctx->qbuf;
    e.kc = kv.k; e.vc = kv.v;
    e.S = S; e.cur_row0 = cur_row0;
    ProfScope ps(ctx, st, "fc_epi_qkv");
    hipLaunchKernelGGL(k_epi_qkv, dim3((unsigned)rows), dim3(256), 0, st, e, B);
    FC_HIP_TRY(hipGetLastError());
  }

  // 2. attention over the whole cache
  {
    AttnArgs a{};
    a.q = ctx->qbuf;
    a.kc = kv.k; a.vc = kv.v;
    a.rope = ctx->rope;
    a.idx = idx; a.nrec = nrec;
    a.N = N; a.nh = nh; a.nkv = nkv; a.S = S;
    a.T = kv.text_tokens; a.W = kv.window; a.head = kv.head;
    a.scale_log2 = (float)(1.0 / std::sqrt((double)hd) * 1.4426950408889634);
    a.out = ctx->attn;
    const int tiles = B * ((N + 31) / 32);
    const int nkb = (S + 31) / 32;
    int splits = std::max(1, std::min(kMaxSplits, (2 * std::max(ctx->num_cus, 1)) / (tiles * nkv)));
    splits = std::min(splits, std::max(1, nkb / 4));
    const size_t need = (size_t)splits * rows * nh * (hd + 2);
    while (splits > 1 && need > ctx->part_elems) --splits;
    a.kb_per_split = (nkb + splits - 1) / splits;
    a.splits = (nkb + a.kb_per_split - 1) / a.kb_per_split;
    a.po = ctx->part;
    a.pm = ctx->part + (size_t)a.splits * rows * nh * hd;
    a.pl = a.pm + (size_t)a.splits * rows * nh;
    const int G = nh / nkv;
    dim3 grid(tiles, nkv, a.splits);
    {
      ProfScope ps(ctx, st, "fc_attn");
      if (hd == 128 && G == 7)
        hipLaunchKernelGGL((k_attn<128, 7>), grid, dim3(7 * 64), 0, st, a);
      else if (hd == 128 && G == 1)
        hipLaunchKernelGGL((k_attn<128, 1>), grid, dim3(64), 0, st, a);
      else if (hd == 64 && G == 1)
        hipLaunchKernelGGL((k_attn<64, 1>), grid, dim3(64), 0, st, a);
      else if (hd == 64 && G == 2)
        hipLaunchKernelGGL((k_attn<64, 2>), grid, dim3(128), 0, st, a);
      else if (hd == 128 && G == 4)
        hipLaunchKernelGGL((k_attn<128, 4>), grid, dim3(256), 0, st, a);
      else
        return fail(FC_ERR_UNSUPPORTED, "attention: head_dim %d with %d query heads per kv head", hd, G);
      FC_HIP_TRY(hipGetLastError());
    }
    if (a.splits > 1) {
      ProfScope ps(ctx, st, "fc_attn_combine");
      hipLaunchKernelGGL(k_attn_combine, dim3((unsigned)rows, nh), dim3(128), 0, st, a, hd, B);
      FC_HIP_TRY(hipGetLastError());
    }
  }

  // 3. O projection + residual -> h1 (float32), 1/rms(h1)
  {
    GemmArgs go{};
    go.A = ctx->attn;
    go.gather = 0;
    go.W0 = L.w_o;
    go.K = nh * hd;
    go.Nout = d;
    go.N = N;
    go.idx = idx; go.nrec = nrec;
    go.C = ctx->part;
    go.splits = pick_splits(mt * ((d + BN - 1) / BN), nh * hd, want, rows, d, ctx->part_elems);
    const int s0 = go.splits;
    rc = run_gemm(ctx, st, "fc_gemm_o", go, B);
    if (rc != FC_OK) return rc;
    const int kc = ((nh * hd + s0 - 1) / s0 + BK - 1) / BK * BK;
    EpiArgs e{};
    e.N = N; e.d = d;
    e.splits = (nh * hd + kc - 1) / kc;
    e.ncols = d;
    e.eps = L.rms_eps;
    e.idx = idx; e.nrec = nrec;
    e.part = ctx->part;
    e.x = x_cur;
    e.h1 = ctx->h1;
    e.inv2 = ctx->inv2;
    ProfScope ps(ctx, st, "fc_epi_o");
    hipLaunchKernelGGL(k_epi_o, dim3((unsigned)rows), dim3(256), 0, st, e, B);
    FC_HIP_TRY(hipGetLastError());
  }

  // 4. gate/up with the MLP RMSNorm folded in, SiLU(g) * u -> act (bf16)
  {
    GemmArgs gu{};
    gu.A = ctx->h1;
    gu.a_f32 = 1;
    gu.gather = 0;
    gu.gain = L.g_mlp;
    gu.W0 = L.w_gate;
    gu.W1 = L.w_up;
    gu.swiglu = 1;
    gu.K = d;
    gu.Nout = ffn;
    gu.N = N;
    gu.idx = idx; gu.nrec = nrec;
    gu.act = ctx->act;
    gu.row_scale = ctx->inv2;
    gu.splits = 1;
    rc = run_gemm(ctx, st, "fc_gemm_gateup", gu, B);
    if (rc != FC_OK) return rc;
  }

  // 5. down projection + residual, scattered into the output cache
  {
    GemmArgs gd{};
    gd.A = ctx->act;
    gd.gather = 0;
    gd.W0 = L.w_down;
    gd.K = ffn;
    gd.Nout = d;
    gd.N = N;
    gd.idx = idx; gd.nrec = nrec;
    gd.C = ctx->part;
    gd.splits = pick_splits(mt * ((d + BN - 1) / BN), ffn, want, rows, d, ctx->part_elems);
    const int s0 = gd.splits;
    rc = run_gemm(ctx, st, "fc_gemm_down", gd, B);
    if (rc != FC_OK) return rc;
    const int kc = ((ffn + s0 - 1) / s0 + BK - 1) / BK * BK;
    EpiArgs e{};
    e.N = N; e.d = d;
    e.splits = (ffn + kc - 1) / kc;
    e.ncols = d;
    e.idx = idx; e.nrec = nrec;
    e.part = ctx->part;
    e.h1 = ctx->h1;
    e.y = y_cur;
    ProfScope ps(ctx, st, "fc_epi_down");
    hipLaunchKernelGGL(k_epi_down, dim3((unsigned)rows), dim3(256), 0, st, e, B);
    FC_HIP_TRY(hipGetLastError());
  }
  return FC_OK;
}

fc_status launch_cache_update(fc_ctx *ctx, const fc_layer_desc &L, const fc_kv_cache &kv,
                              const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                              const uint8_t *reuse, int grid_w, int B, hipStream_t st) {
  const int N = kv.frame_tokens;
  const int S = kv.text_tokens + kv.window * N;
  const int kvw = L.n_kv_heads * L.head_dim;
  const int cur_slot = (kv.head + kv.window - 1) % kv.window;
  const int prev_slot = kv.window > 1 ? (kv.head + kv.window - 2) % kv.window : cur_slot;
  CacheArgs c{};
  c.kc = kv.k;
  c.vc = kv.v;
  c.y_prev = y_prev;
  c.y_cur = y_cur;
  c.shift = shift;
  c.reuse = reuse;
  c.N = N;
  c.S = S;
  c.kvw = kvw;
  c.d = L.d_model;
  c.gw = grid_w;
  c.gh = N / grid_w;
  c.cur_row0 = kv.text_tokens + cur_slot * N;
  if (kv.window == 1) {
    // the current frame overwrites the previous one in place: stage the old rows
    const long per = (long)N * kvw;
    for (int b = 0; b < B; ++b) {
      ProfScope ps(ctx, st, "fc_cache_stage");
      const long n16 = per / 8;
      const uint16_t *ks = kv.k + ((long)b * S + c.cur_row0) * kvw;
      const uint16_t *vs = kv.v + ((long)b * S + c.cur_row0) * kvw;
      hipLaunchKernelGGL(k_copy16, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, st,
                         reinterpret_cast<const uint4 *>(ks),
                         reinterpret_cast<uint4 *>(ctx->stage + (long)b * 2 * per), n16);
      hipLaunchKernelGGL(k_copy16, dim3((unsigned)((n16 + 255) / 256)), dim3(256), 0, st,
                         reinterpret_cast<const uint4 *>(vs),
                         reinterpret_cast<uint4 *>(ctx->stage + (long)b * 2 * per + per), n16);
      FC_HIP_TRY(hipGetLastError());
    }
    c.ksrc = ctx->stage;
    c.vsrc = ctx->stage + per;
    c.src_bstride = 2 * per;
    c.src_row0 = 0;
  } else {
    c.ksrc = kv.k;
    c.vsrc = kv.v;
    c.src_bstride = (long)S * kvw;
    c.src_row0 = kv.text_tokens + prev_slot * N;
  }
  ProfScope ps(ctx, st, "fc_cache_update");
  hipLaunchKernelGGL(k_cache_update, dim3((N + 3) / 4, B), dim3(256), 0, st, c);
  FC_HIP_TRY(hipGetLastError());
  return FC_OK;
}

}  // namespace fc
