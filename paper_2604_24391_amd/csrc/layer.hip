// Partial-recompute decoder layer and token-cache remap on gfx950.
//
// Rows of the layer are "slots": slot r = b * N + j holds the j-th recomputed
// token of batch item b, j < n_recompute[b] (read on the device, so no host
// sync); grids are sized for N rows per item and surplus tiles exit.
//
//   k_wgemm     weight-streaming bf16 MFMA GEMM (v_mfma_f32_16x16x32_bf16) over the
//               slots, C = A W^T with W row-major [out][in] like torch.nn.Linear;
//               split-K float32 partials, or (SwiGLU) SiLU(g) * u in the epilogue.
//               The QKV projection gathers the recomputed tokens' rows of x by id and
//               multiplies x g (the attention RMSNorm gain) on its A fragments.
//   k_red_qkv   sums the QKV partials, scales by the token's 1/rms, adds the bias,
//               stores rotated q and scatters raw k and v into the current frame's
//               cache rows.
//   k_attn      attention of the gathered queries over the whole cache, GQA
//               (one wave per query head of a KV group), RoPE applied to q and to
//               each key block as it is staged in LDS, causal by position, float32
//               online softmax in the transposed form S^T = K Q^T so that a lane
//               owns one query column.  Optional split over key blocks.
//   k_attn_combine  merges split-KV partials.
//   k_red_o     residual add -> h1 (float32), the SwiGLU operand bf16(h1 * g_mlp)
//               and per-chunk sums of squares of h1 for the MLP RMSNorm.
//   k_red_down  residual add, bf16 output rows scattered into the output cache.
//   k_cache_update  copies cached K/V/output rows of each reused token from its
//               aligned source token.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

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
// Null counts and ids (the trailing-text rows) mean every token of the region, in order.
__device__ __forceinline__ int n_valid(const int32_t *nrec, int b, int N) {
  return nrec ? min(max(nrec[b], 0), N) : N;
}
__device__ __forceinline__ int tok_of(const int32_t *idx, long slot, int N) {
  return idx ? min(max(idx[slot], 0), N - 1) : (int)(slot % N);
}

// RoPE position of rotary frequency pair k for the token at sequence position seqpos
// (its index in the current step's prompt, which also decides causality).  1-D RoPE:
// seqpos itself.  Multimodal RoPE (Qwen2.5-VL): pairs [0, s1) rotate by the temporal,
// [s1, s2) by the row and [s2, hd/2) by the column position; a text token has all three
// equal to its index, the token (I, J) of the frame with logical index l has
// (st, st + I, st + J) with st = T + l span, span = max(grid rows, grid columns), each
// frame taking span positions after the one before it.
// Text after the frames continues from the last frame's span: its three positions are
// T + W span + (its index past the frames).
struct MRope {
  int on, T, N, W, gw, span, s1, s2;
};
__device__ __forceinline__ int rope_pos(const MRope &m, int seqpos, int k) {
  if (!m.on || seqpos < m.T) return seqpos;
  if (seqpos >= m.T + m.W * m.N) return seqpos - m.W * m.N + m.W * m.span;
  const int r = seqpos - m.T, l = r / m.N, tok = r - l * m.N;
  const int st = m.T + l * m.span;
  if (k < m.s1) return st;
  const int I = tok / m.gw;
  return k < m.s2 ? st + I : st + (tok - I * m.gw);
}

// ------------------------------------------------------------------------------- GEMM
// Weight-streaming GEMM over the gathered rows, C[rows][cols] = A[rows][K] W[cols][K]^T
// with W row-major [out][in] like torch.nn.Linear.  With a few hundred gathered rows
// the layer is bound by streaming the weights, and every CU must also re-read the
// whole activation tile for its columns, so the kernel is shaped by the per-CU load
// path:
//   * output columns are dealt in 16-column blocks evenly over all CUs (SwiGLU: the gate
//     block and the up block of the same columns form a pair); the QKV, O and down
//     projections add a K split so that the column groups times the splits cover the
//     chip once, each split's activation K-slice staying in one XCD's L2;
//   * a K step stages 64 K values of every operand row -- one full 128-B line per row,
//     8 rows per 1 KB DMA instruction (half lines double the request count) -- into LDS
//     by global_load_lds.  Rows are unpadded, their 16-B chunks XOR-swizzled by
//     (row >> 1) & 7, which keeps the fragment reads free of bank conflicts;
//   * waves 4-7 only issue those DMAs.  A DMA instruction holds its wave at issue, so a
//     wave that also multiplied would leave its matrix core idle meanwhile;
//   * waves 0-3 run v_mfma_f32_16x16x32_bf16 on the staged operands, wave w owning the
//     16-row blocks w, w + 4, ...  Every wave runs the full block grid without a branch
//     per MFMA: blocks past the valid rows and absent weight blocks multiply stale LDS
//     into accumulators that are never stored;
//   * PD stages rotate with one LDS barrier per K step: after barrier k the loaders
//     refill the stage of step k - 1 with step k + PD - 1.
// Split-K partial sums go to a float32 buffer [split][rows][cols] that the k_red_*
// kernels reduce; the SwiGLU mode applies the MLP RMSNorm and SiLU(g) * u in its own
// epilogue.
enum { G_QKV = 0, G_O = 1, G_GU = 2, G_DOWN = 3, G_PLAIN = 4 };   // PLAIN: fp32 sums only (k_mgemm)
constexpr int KS = kGemmBK;                 // 64 K values per step
constexpr int RB = KS * 2;                  // bytes per staged operand row
constexpr int MT = 256;                     // rows per M tile
constexpr int kLdsBytes = 158 * 1024;       // operand stages
constexpr int kGainSteps = 2 * MT * 4 / (KS * 2);   // K steps of gain the QKV LDS slice holds

struct WArgs {
  const uint16_t *A;              // bf16 activations: one row per slot, or (gather) x [B][N][K]
  int gather;                     // QKV: A rows are the layer input's rows at the token ids
  const uint16_t *gain;           // QKV: attention RMSNorm gain, applied along K to A
  const uint16_t *W0, *W1;        // weights [cols][K]; SwiGLU: gate, up
  int K, Nout, N;                 // N = token slots per batch item
  int nb, ncg, splits, ksteps;    // 16-col blocks, column groups, K splits, K steps per split
  int tpb;                        // M tiles per batch item
  const int32_t *idx, *nrec;
  float *part;                    // [split][B*N][Nout]
  long rows;                      // B*N
  uint16_t *act;                  // SwiGLU output [B*N][Nout]
  const float *ssq;               // SwiGLU: [B*N][ss_parts] partial sums of squares of h1
  int ss_parts;
  float eps;
};

// Workgroup id -> tile id so that each XCD (workgroups are dealt round-robin over
// the 8 XCDs) works on a contiguous range of tiles.
__device__ __forceinline__ int xcd_tile(int w, int total) {
  const int per = total / 8;
  if (w >= per * 8) return w;
  return (w & 7) * per + (w >> 3);
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t lds_addr(const void *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void *)p;
}
// LDS DMA of 16 B per lane to lds + 16 * lane (lds must be wave-uniform).  M0 is
// reserved to the compiler, so the asm restores it.
__device__ __forceinline__ void dma16(const void *gp, uint32_t lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gp), "s"(l)
      : "memory");
}
// The same for data read once (streamed weights): the non-temporal hint keeps such
// lines from displacing the re-read activation rows in L2.
__device__ __forceinline__ void dma16_nt(const void *gp, uint32_t lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "global_load_lds_dwordx4 %1, off nt\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(gp), "s"(l)
      : "memory");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt holds at most 63 outstanding loads");
  __builtin_amdgcn_s_waitcnt(0x3F70 | (N & 0xF) | ((N >> 4) << 14));
}
// wait until at most n (wave-uniform, < 64) of this wave's loads are outstanding
__device__ __forceinline__ void wait_vm_rt(int n) {
  switch (n) {
#define FC_W1(x) case x: wait_vm<x>(); break;
#define FC_W8(x) FC_W1(x) FC_W1(x + 1) FC_W1(x + 2) FC_W1(x + 3) FC_W1(x + 4) FC_W1(x + 5) FC_W1(x + 6) FC_W1(x + 7)
    FC_W8(0) FC_W8(8) FC_W8(16) FC_W8(24) FC_W8(32) FC_W8(40) FC_W8(48) FC_W8(56)
#undef FC_W8
#undef FC_W1
    default: wait_vm<0>(); break;
  }
}
// Workgroup barrier that orders LDS accesses only: global loads in flight stay in
// flight across it (the full fence of __syncthreads would drain them).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}
__device__ __forceinline__ int swz8(int row) { return (row >> 1) & 7; }

template <int MODE>
struct WTraits {
  // 16-column blocks a column group may hold: 1184 SwiGLU pairs over 256 groups is
  // 4.625; the Qwen QKV (288 blocks) and O/down (224 blocks) split into 32 groups of 9
  // and 7
  static constexpr int NBLK = MODE == G_GU ? 5 : (MODE == G_QKV ? 9 : 7);
  static constexpr int NBW = (MODE == G_GU ? 2 : 1) * NBLK;   // staged weight blocks
};
template <int MODE, int MBW>
struct WStage {
  static constexpr int ABLK = 4 * MBW;                        // 16-row activation blocks
  static constexpr int AROWS = ABLK * 16;
  static constexpr int BYTES = (AROWS + WTraits<MODE>::NBW * 16) * RB;
  static constexpr int PD = (kLdsBytes / BYTES) > 6 ? 6 : (kLdsBytes / BYTES);
  static constexpr int MAXI = (ABLK * 2 + WTraits<MODE>::NBW * 2 + 3) / 4;  // DMAs per loader
  static_assert(PD >= 3, "at least three stages");
  static_assert((PD - 2) * MAXI < 64, "vmcnt holds at most 63 outstanding loads");
};

// One (M tile, column group, K split) with MBW 16-row blocks per MFMA wave.
template <int MODE, int MBW>
__device__ __forceinline__ void wgemm_tile(const WArgs &a, unsigned char *lds, float *rowinv,
                                           int b, int row0, int nvalid, int cg, int sp, int nk) {
  using T = WTraits<MODE>;
  using S = WStage<MODE, MBW>;
  constexpr int PD = S::PD, NBLK = T::NBLK, NBW = T::NBW, MAXI = S::MAXI;
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int cb0 = (int)((long)cg * a.nb / a.ncg);
  const int nblk = (int)((long)(cg + 1) * a.nb / a.ncg) - cb0;
  const int nbm = (nvalid + 15) >> 4;
  const long k0 = (long)sp * a.ksteps * KS;
  const long slot0 = (long)b * a.N + row0;

  if (w >= 4) {
    // ----------------------------------------------------------------- loader waves
    // Instruction j of a step stages 8 rows: j < nA the activation rows 8j.., then
    // two per present weight block.  Loader q issues j = q, q + 4, ...
    const int q = w - 4;
    const int nA = nbm * 2;
    const int npres = MODE == G_GU ? 2 * nblk : nblk;
    const int ntot = nA + npres * 2;
    const int rsub = lane >> 3, ch = lane & 7;
    const uint16_t *gp[MAXI];
    uint32_t lo[MAXI];
    bool wt[MAXI];
    int L = 0;
#pragma unroll
    for (int i = 0; i < MAXI; ++i) {
      const int j = min(q + 4 * i, ntot - 1);
      L += (q + 4 * i < ntot);
      wt[i] = j >= nA;
      if (j < nA) {
        const int r = j * 8 + rsub;                            // tile row
        const int rr = r < nvalid ? r : nvalid - 1;            // clamp: never stored
        const long arow = a.gather ? (long)b * a.N + tok_of(a.idx, slot0 + rr, a.N) : slot0 + rr;
        gp[i] = a.A + arow * a.K + k0 + ((ch ^ swz8(r)) * 8);
        lo[i] = j * 1024;
      } else {
        const int jw = j - nA, pb = jw >> 1;                   // present weight block pb
        int blk, col0;
        const uint16_t *M = a.W0;
        if (MODE == G_GU && pb >= nblk) {
          blk = NBLK + pb - nblk;
          col0 = (cb0 + pb - nblk) * 16;
          M = a.W1;
        } else {
          blk = pb;
          col0 = (cb0 + pb) * 16;
        }
        const int r = blk * 16 + (jw & 1) * 8 + rsub;         // row of the weight region
        gp[i] = M + (long)(col0 + (r & 15)) * a.K + k0 + ((ch ^ swz8(r)) * 8);
        lo[i] = S::AROWS * RB + (blk * 2 + (jw & 1)) * 1024;
      }
    }
    const uint32_t lbase = lds_addr(lds);
    auto issue = [&](int kt, int stg) {
      const int kk = kt * KS;
      const uint32_t st = lbase + stg * S::BYTES;
#pragma unroll
      for (int i = 0; i < MAXI; ++i) {
        if (i < L) {
          if (wt[i]) dma16_nt(gp[i] + kk, st + lo[i]);
          else dma16(gp[i] + kk, st + lo[i]);
        }
      }
    };
    for (int u = 0; u < PD - 1 && u < nk; ++u) issue(u, u);
    for (int k = 0; k < nk; ++k) {
      wait_vm_rt(min(nk - 1 - k, PD - 2) * L);                 // this wave's share of step k
      lds_barrier();                                           // barrier k: step k staged
      const int nxt = k + PD - 1;
      if (nxt < nk) issue(nxt, nxt % PD);                      // the stage of step k - 1
    }
    lds_barrier();                                             // barrier nk: LDS is free
    return;
  }

  // -------------------------------------------------------------------- MFMA waves
  if (MODE == G_GU) {
    // 1/rms of each row from the per-chunk sums of squares of h1, while the first
    // stages are in flight (these waves have no loads of their own outstanding)
    for (int r = t; r < MT; r += 256) {
      float v = 0.f;
      if (r < nvalid)
        for (int c = 0; c < a.ss_parts; ++c) v += a.ssq[(slot0 + r) * a.ss_parts + c];
      rowinv[r] = 1.f / sqrtf(v / (float)a.K + a.eps);
    }
  }
  const int l16 = lane & 15, g = lane >> 4;
  f32x4 acc[MBW][NBW];
#pragma unroll
  for (int i = 0; i < MBW; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // QKV multiplies x g: the attention RMSNorm gain of this split's K range is staged in
  // LDS before barrier 0 (at most kGainSteps K steps, checked at launch); 1/rms scales
  // the summed rows in k_red_qkv
  const __bf16 *gsl = reinterpret_cast<const __bf16 *>(rowinv);
  if (MODE == G_QKV) {
    for (int e = t; e < nk * KS / 8; e += 256)
      reinterpret_cast<uint4 *>(rowinv)[e] = *reinterpret_cast<const uint4 *>(a.gain + k0 + 8 * e);
  }
  // fragment (row l16, K sub-step s): 16-B chunk 4 s + g of the row, at its swizzled slot;
  // A and B use the same K order, so the products are those of the plain K order
  const uint32_t rowoff = l16 * RB;
  const int sw = swz8(l16);
  for (int k = 0; k < nk; ++k) {
    lds_barrier();                                             // barrier k: step k staged
    const unsigned char *st = lds + (k % PD) * S::BYTES;
    bf16x8 fa[2][MBW], fb[2][NBW];
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const uint32_t slot = (uint32_t)(((4 * s + g) ^ sw) << 4);
#pragma unroll
      for (int i = 0; i < MBW; ++i)
        fa[s][i] = *reinterpret_cast<const bf16x8 *>(st + (w + 4 * i) * 16 * RB + rowoff + slot);
#pragma unroll
      for (int j = 0; j < NBW; ++j)
        fb[s][j] = *reinterpret_cast<const bf16x8 *>(st + (S::AROWS + j * 16) * RB + rowoff + slot);
    }
    if (MODE == G_QKV) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        const bf16x8 gc = *reinterpret_cast<const bf16x8 *>(gsl + k * KS + (4 * s + g) * 8);
#pragma unroll
        for (int i = 0; i < MBW; ++i)
#pragma unroll
          for (int e = 0; e < 8; ++e) fa[s][i][e] = (__bf16)((float)fa[s][i][e] * (float)gc[e]);
      }
    }
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int j = 0; j < NBW; ++j)
#pragma unroll
        for (int i = 0; i < MBW; ++i)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[s][i], fb[s][j], acc[i][j], 0, 0, 0);
  }

  lds_barrier();                                               // barrier nk: LDS is free

  // Epilogue: each 16-row block goes through a wave-private LDS tile so that the global
  // stores are whole 16-B chunks of contiguous row segments (a lane's accumulators hold
  // one column of 4 rows).  The row pitch is 16 B past a multiple of 64 B, which spreads
  // the 4 row groups of a tile write over distinct banks.
  // lane holds column l16 and rows 4 g + e of each 16-row block
  constexpr int ESZ = MODE == G_GU ? 2 : 4;                    // bytes per output value
  constexpr int PITCH = NBLK * 16 * ESZ + (MODE == G_GU ? 48 : 16);
  static_assert(4 * 16 * PITCH <= kLdsBytes, "epilogue tiles fit in LDS");
  unsigned char *tile = lds + w * 16 * PITCH;
  const int nch = nblk * 16 * ESZ / 16;                        // 16-B chunks per row segment
#pragma unroll
  for (int i = 0; i < MBW; ++i) {
    const int blk = w + 4 * i;
    if (blk >= nbm) continue;
#pragma unroll
    for (int j = 0; j < NBLK; ++j) {
      if (j >= nblk) continue;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = 4 * g + e;
        if (MODE == G_GU) {
          const float sc = rowinv[min(blk * 16 + r, MT - 1)];
          const float gv = acc[i][j][e] * sc;
          const float uv = acc[i][NBLK + j][e] * sc;
          *reinterpret_cast<uint16_t *>(tile + r * PITCH + (j * 16 + l16) * 2) =
              f2bf(gv / (1.f + __expf(-gv)) * uv);
        } else {
          *reinterpret_cast<float *>(tile + r * PITCH + (j * 16 + l16) * 4) = acc[i][j][e];
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
    const int rows_here = min(16, nvalid - blk * 16);
    for (int c = lane; c < rows_here * nch; c += 64) {
      const int r = c / nch, x = c - r * nch;
      const uint4 v = *reinterpret_cast<const uint4 *>(tile + r * PITCH + x * 16);
      const long grow = slot0 + blk * 16 + r;
      if (MODE == G_GU)
        *reinterpret_cast<uint4 *>(a.act + grow * a.Nout + cb0 * 16 + x * 8) = v;
      else
        *reinterpret_cast<uint4 *>(a.part + ((long)sp * a.rows + grow) * a.Nout + cb0 * 16 + x * 4) = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront", "local");
  }
}

template <int MODE>
__global__ __launch_bounds__(512) void k_wgemm(WArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  // SwiGLU: 1/rms per row; QKV: the attention RMSNorm gain of the split's K range
  __shared__ __attribute__((aligned(16))) float rowinv[2 * MT];
  // split fastest: with 8 splits every split's workgroups share one XCD and its L2
  const int bid = blockIdx.x;
  const int sp = bid % a.splits;
  const int rest = bid / a.splits;
  const int cg = rest % a.ncg;
  const int mt = rest / a.ncg;
  const int b = mt / a.tpb;
  const int row0 = (mt % a.tpb) * MT;
  const int nvalid = min(MT, n_valid(a.nrec, b, a.N) - row0);
  const int nk = min(a.ksteps, a.K / KS - sp * a.ksteps);
  if (nvalid <= 0 || nk <= 0) return;
  switch ((((nvalid + 15) >> 4) + 3) >> 2) {
    case 1: wgemm_tile<MODE, 1>(a, lds, rowinv, b, row0, nvalid, cg, sp, nk); break;
    case 2: wgemm_tile<MODE, 2>(a, lds, rowinv, b, row0, nvalid, cg, sp, nk); break;
    case 3: wgemm_tile<MODE, 3>(a, lds, rowinv, b, row0, nvalid, cg, sp, nk); break;
    default: wgemm_tile<MODE, 4>(a, lds, rowinv, b, row0, nvalid, cg, sp, nk); break;
  }
}

// ------------------------------------------------------------------------------- reductions
// One workgroup per (row, 1024-column chunk); each thread sums the split-K partials of
// 4 columns with float4 loads and applies the epilogue of its projection.
struct RedArgs {
  int N, d, splits, ncols, qw, kw, S, cur_row0;
  int hd, qpos0;                  // head dim; prompt position of current-frame token 0
  const float2 *rope;             // [S][hd/2] (cos, sin)
  MRope mr;                       // RoPE positions (1-D or multimodal)
  long rows;
  float eps;
  const int32_t *idx, *nrec;
  const float *part;              // [split][B*N][ncols]
  const uint16_t *x;              // [B][N][d] layer input
  const uint16_t *bias;           // [ncols] (QKV)
  const uint16_t *gain;           // [d] MLP RMSNorm gain (O reduction)
  uint16_t *q, *kc, *vc;          // QKV outputs
  const int32_t *smap;            // slot map of the K/V rows (null: rows in place)
  float *h1;                      // [B*N][d]
  uint16_t *hb;                   // [B*N][d] bf16(h1 * g_mlp), the SwiGLU operand
  float *ssq;                     // [B*N][chunks] sums of squares of h1 per 1024 columns
  uint16_t *y;                    // [B][N][d]
};

// Sum of the split-K partials of 4 columns, in split order.  SPL is the split count
// rounded up to a power of two: every load is issued before the first add (splits past
// the last re-read it and are not added), so the sum costs one memory round trip.
template <int SPL>
__device__ __forceinline__ float4 sum_parts(const RedArgs &r, long slot, int c) {
  const float *p = r.part + slot * r.ncols + c;
  const long stride = r.rows * r.ncols;
  float4 u[SPL];
#pragma unroll
  for (int s = 0; s < SPL; ++s)
    u[s] = *reinterpret_cast<const float4 *>(p + min(s, r.splits - 1) * stride);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int s = 0; s < SPL; ++s) {
    const bool in = s < r.splits;
    v.x += in ? u[s].x : 0.f;
    v.y += in ? u[s].y : 0.f;
    v.z += in ? u[s].z : 0.f;
    v.w += in ? u[s].w : 0.f;
  }
  return v;
}

// Sum over a 256-thread workgroup: a butterfly within each wave, then the four wave
// sums in a fixed order (every thread gets the same bits).
__device__ float block_sum256(float v, float *red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  const int t = threadIdx.x;
  if ((t & 63) == 0) red[t >> 6] = v;
  __syncthreads();
  const float res = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return res;
}

// Large-M path: one workgroup per slot, the gathered token's row of x, normalised and
// scaled by the attention RMSNorm gain, as the QKV GEMM's bf16 operand.
__global__ __launch_bounds__(256) void k_gather_norm(const uint16_t *__restrict__ x,
                                                     const uint16_t *__restrict__ gain,
                                                     const int32_t *__restrict__ idx,
                                                     const int32_t *__restrict__ nrec, int N,
                                                     int d, float eps, uint16_t *__restrict__ xs) {
  __shared__ float red[256];
  const long slot = blockIdx.x;
  const int b = (int)(slot / N), j = (int)(slot - (long)b * N);
  if (j >= n_valid(nrec, b, N)) return;
  const int tok = tok_of(idx, slot, N);
  const uint16_t *xr = x + ((long)b * N + tok) * d;
  // the row is read once and held in registers (d <= 8192: at most 4 chunks a thread)
  constexpr int kIt = 4;
  U16x8 v[kIt];
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < kIt; ++it) {
    const int c = (it * 256 + threadIdx.x) * 8;
    if (c < d) {
      v[it] = *reinterpret_cast<const U16x8 *>(xr + c);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float f = bf2f(v[it].v[e]);
        ss = fmaf(f, f, ss);
      }
    }
  }
  ss = block_sum256(ss, red);
  const float inv = 1.f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int it = 0; it < kIt; ++it) {
    const int c = (it * 256 + threadIdx.x) * 8;
    if (c < d) {
      const U16x8 g = *reinterpret_cast<const U16x8 *>(gain + c);
      U16x8 o;
#pragma unroll
      for (int e = 0; e < 8; ++e) o.v[e] = f2bf(bf2f(v[it].v[e]) * inv * bf2f(g.v[e]));
      *reinterpret_cast<U16x8 *>(xs + slot * d + c) = o;
    }
  }
}

// One workgroup per (slot, 1024 columns): split-K sum of (x g) W^T, scaled by the
// token's 1/rms (from its row of x, read once per workgroup), plus the bias.  Queries
// are rotated (rotate-half RoPE at the token's prompt position) in float32 before
// their single rounding to bf16; a 1024-column block always holds whole heads, so
// the partner dim of the rotation comes from LDS.  K and V rows go raw into the cache.
template <int SPL>
__global__ __launch_bounds__(256) void k_red_qkv(RedArgs r) {
  __shared__ float qs[1024];
  const long slot = blockIdx.x;
  const int b = (int)(slot / r.N), j = (int)(slot - (long)b * r.N);
  if (j >= n_valid(r.nrec, b, r.N)) return;
  const int c0 = blockIdx.y * 1024;
  const int c = c0 + threadIdx.x * 4;
  const int tok = tok_of(r.idx, slot, r.N);
  const bool incol = c < r.ncols;
  const bool rot = c < r.qw;                      // query columns are rotated
  const int half = r.hd / 2;
  // Every load that depends only on the token goes out before the first use, so the
  // workgroup waits one memory round trip instead of three: the split partials and
  // the bias of the thread's 4 columns, its chunks of the input row (for 1/rms; d <=
  // 8192: at most 4 chunks of 8 a thread) and the rotary pairs of its query dims.
  // Threads past the columns or the row read an in-range element and never use it.
  const float *pp = r.part + slot * r.ncols + (incol ? c : 0);
  const long stride = r.rows * r.ncols;
  float4 u[SPL];
#pragma unroll
  for (int s = 0; s < SPL; ++s)
    u[s] = *reinterpret_cast<const float4 *>(pp + min(s, r.splits - 1) * stride);
  const uint2 bb = *reinterpret_cast<const uint2 *>(r.bias + (incol ? c : 0));
  const uint16_t *xr = r.x + ((long)b * r.N + tok) * r.d;
  U16x8 xv[4];
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int cx = (it * 256 + threadIdx.x) * 8;
    xv[it] = *reinterpret_cast<const U16x8 *>(xr + (cx < r.d ? cx : 0));
  }
  float2 cs[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int k = ((c + e) % r.hd) % half;       // rotary frequency pair
    cs[e] = r.rope[rot ? (long)rope_pos(r.mr, r.qpos0 + tok, k) * half + k : 0L];
  }
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int s = 0; s < SPL; ++s) {
    const bool in = s < r.splits;
    v.x += in ? u[s].x : 0.f;
    v.y += in ? u[s].y : 0.f;
    v.z += in ? u[s].z : 0.f;
    v.w += in ? u[s].w : 0.f;
  }
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    if ((it * 256 + (int)threadIdx.x) * 8 < r.d) {
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(bf2f(xv[it].v[e]), bf2f(xv[it].v[e]), ss);
    }
  }
  const float inv = 1.f / sqrtf(block_sum256(ss, qs) / (float)r.d + r.eps);
  float vv[4] = {0.f, 0.f, 0.f, 0.f};
  if (incol) {
    const float bias[4] = {__uint_as_float(bb.x << 16), __uint_as_float(bb.x & 0xFFFF0000u),
                           __uint_as_float(bb.y << 16), __uint_as_float(bb.y & 0xFFFF0000u)};
    vv[0] = v.x; vv[1] = v.y; vv[2] = v.z; vv[3] = v.w;
#pragma unroll
    for (int e = 0; e < 4; ++e) vv[e] = fmaf(vv[e], inv, bias[e]);
  }
  if (c0 < r.qw) {   // uniform: the block's query columns are rotated
    *reinterpret_cast<float4 *>(&qs[threadIdx.x * 4]) = make_float4(vv[0], vv[1], vv[2], vv[3]);
    __syncthreads();
    if (rot) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int d = (c + e) % r.hd;                 // dim within the head
        const int lc = threadIdx.x * 4 + e;           // column within the block
        vv[e] = d < half ? vv[e] * cs[e].x - qs[lc + half] * cs[e].y
                         : vv[e] * cs[e].x + qs[lc - half] * cs[e].y;
      }
    }
  }
  if (!incol) return;
  uint16_t o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = f2bf(vv[e]);
  uint16_t *dst;
  if (c < r.qw)
    dst = r.q + slot * r.qw + c;
  else if (c < r.qw + r.kw)
    dst = r.kc + ((long)b * r.S + pool_row(r.smap, b, r.S, r.cur_row0 + tok)) * r.kw + (c - r.qw);
  else
    dst = r.vc + ((long)b * r.S + pool_row(r.smap, b, r.S, r.cur_row0 + tok)) * r.kw +
          (c - r.qw - r.kw);
  *reinterpret_cast<uint2 *>(dst) = make_uint2(o[0] | ((uint32_t)o[1] << 16), o[2] | ((uint32_t)o[3] << 16));
}

template <int SPL>
__global__ __launch_bounds__(256) void k_red_o(RedArgs r) {
  __shared__ float red[256];
  const long slot = blockIdx.x;
  const int b = (int)(slot / r.N), j = (int)(slot - (long)b * r.N);
  if (j >= n_valid(r.nrec, b, r.N)) return;
  const int c = blockIdx.y * 1024 + threadIdx.x * 4;
  const int tok = tok_of(r.idx, slot, r.N);
  float ss = 0.f;
  if (c < r.d) {
    const float4 v = sum_parts<SPL>(r, slot, c);
    const uint2 xb = *reinterpret_cast<const uint2 *>(r.x + ((long)b * r.N + tok) * r.d + c);
    float4 h;
    h.x = v.x + __uint_as_float(xb.x << 16);
    h.y = v.y + __uint_as_float(xb.x & 0xFFFF0000u);
    h.z = v.z + __uint_as_float(xb.y << 16);
    h.w = v.w + __uint_as_float(xb.y & 0xFFFF0000u);
    *reinterpret_cast<float4 *>(r.h1 + slot * r.d + c) = h;
    // the SwiGLU operand carries the MLP RMSNorm gain; 1/rms is applied to its sums
    const uint2 gb = *reinterpret_cast<const uint2 *>(r.gain + c);
    const uint16_t b0 = f2bf(h.x * __uint_as_float(gb.x << 16));
    const uint16_t b1 = f2bf(h.y * __uint_as_float(gb.x & 0xFFFF0000u));
    const uint16_t b2 = f2bf(h.z * __uint_as_float(gb.y << 16));
    const uint16_t b3 = f2bf(h.w * __uint_as_float(gb.y & 0xFFFF0000u));
    *reinterpret_cast<uint2 *>(r.hb + slot * r.d + c) =
        make_uint2(b0 | ((uint32_t)b1 << 16), b2 | ((uint32_t)b3 << 16));
    ss = h.x * h.x + h.y * h.y + h.z * h.z + h.w * h.w;
  }
  ss = block_sum256(ss, red);
  if (threadIdx.x == 0) r.ssq[slot * gridDim.y + blockIdx.y] = ss;
}

template <int SPL>
__global__ __launch_bounds__(256) void k_red_down(RedArgs r) {
  const long slot = blockIdx.x;
  const int b = (int)(slot / r.N), j = (int)(slot - (long)b * r.N);
  if (j >= n_valid(r.nrec, b, r.N)) return;
  const int c = blockIdx.y * 1024 + threadIdx.x * 4;
  if (c >= r.d) return;
  const int tok = tok_of(r.idx, slot, r.N);
  const float4 v = sum_parts<SPL>(r, slot, c);
  const float4 h = *reinterpret_cast<const float4 *>(r.h1 + slot * r.d + c);
  *reinterpret_cast<uint2 *>(r.y + ((long)b * r.N + tok) * r.d + c) =
      make_uint2(f2bf(h.x + v.x) | ((uint32_t)f2bf(h.y + v.y) << 16),
                 f2bf(h.z + v.z) | ((uint32_t)f2bf(h.w + v.w) << 16));
}

// ------------------------------------------------------------------------------- large-M GEMM
// For thousands of gathered rows (many batch items) the projections are compute bound
// and a square tile pays: each workgroup owns a 256 x 256 output tile and streams
// K in steps of 64 through two LDS stages (A rows, then the 256 staged weight rows,
// each one 128-B line with 16-B chunks XOR-swizzled by (row >> 1) & 7).
//   * eight waves, two per SIMD, each owning 128 x 64 of the tile as 4 x 2 blocks of
//     v_mfma_f32_32x32x16_bf16; the per-CU load rate grows with the number of waves
//     issuing, and a wave waiting at a DMA issue leaves its SIMD to the other wave;
//   * every wave issues an eighth of the next step's DMAs as soon as the step's barrier
//     frees their stage, and reads the fragments of sub-step s + 1 before the MFMAs of
//     sub-step s;
//   * the epilogue is fused and goes through LDS 32 rows at a time, so that every
//     global access is a 16-B (or 8-B) piece of a row: QKV adds the bias, rotates the
//     queries and scatters raw k and v into the cache; O adds the residual and writes
//     h1, the SwiGLU operand and per-256-column sums of squares; SwiGLU stages gate
//     and up rows of the same 32 columns per wave and writes SiLU(g) * u; down adds h1
//     and scatters the output rows.
// Tiles are ordered so that the workgroups resident on one XCD at a time cover 4 M
// tiles x 8 N tiles, which keeps their operand slabs in that XCD's L2; only the tiles
// of the packed rows are mapped, evenly over the XCDs.
constexpr int MB = 256;                     // tile rows and staged weight rows
constexpr int kMStage = 2 * MB * RB;        // 64 KB per stage
constexpr int kMSsqCols = 256;              // columns per sum-of-squares partial
constexpr int kMEpPitch = MB + 4;           // floats per row of the epilogue tile
constexpr int kMMaxItems = 1024;            // batch items the packed row map holds

struct MArgs {
  const uint16_t *A;              // bf16 activations, one row per slot
  const uint16_t *W0, *W1;        // weights [cols][K]; SwiGLU: gate, up
  int K, Nout, N;                 // Nout: output columns; N: token slots per item
  int B, mtiles, ntn;             // items, M tiles (over the packed rows), N tiles
  int ss_parts;                   // O writes / SwiGLU reads this many partials per row
  uint16_t *act;                  // SwiGLU output [B*N][Nout]
  int cus;                        // workgroup slots: one resident workgroup per CU
  int part_units;                 // 256 x 256 fp32 tiles the partial buffer holds
  float *part;                    // K-range partial tiles of the split tail
  float *out;                     // G_PLAIN output: [ks][V][ntn] tiles of 256 x 256 fp32
  int *ks_out;                    // G_PLAIN: the K-range part count ks, written by workgroup 0
  RedArgs r;                      // epilogue operands (as the reductions use them)
};

// G_PLAIN: when the tiles fill at most half the CUs, every tile runs as ks K-range parts
// (at most kPlainMaxParts, at least 4 K steps each), written as separate sums that the
// consumer adds.
constexpr int kPlainMaxParts = 8;
__host__ __device__ inline int plain_split(int tiles, int cus, int nk) {
  int ks = 1;
  if (tiles > 0 && 2 * tiles <= cus) {
    ks = cus / tiles;
    ks = ks < kPlainMaxParts ? ks : kPlainMaxParts;
    ks = ks < nk / 4 ? ks : nk / 4;
    ks = ks > 1 ? ks : 1;
  }
  return ks;
}

// With one workgroup per CU, tiles run in rounds of `cus`.  When there are few rounds
// and the last is at most half full, its `tail` tiles run as `ks` parts over K ranges
// each (written as fp32 partial tiles, summed in part order by k_mtail), so the round
// takes about 1/ks of a tile's time; tiles [0, F) run whole.  (Over many rounds the
// tiles' uneven durations already blur the last round, and the partial round trip
// would cost more than it saves.)  Host and device take the same decision.
__host__ __device__ inline void mtail_split(int total, int cus, int part_units, int nk, int &F,
                                            int &tail, int &ks) {
  tail = cus > 0 ? total % cus : 0;
  ks = 1;
  if (tail > 0 && 2 * tail <= cus && total < 8 * cus) {
    ks = cus / tail;
    ks = ks < 4 ? ks : 4;
    ks = ks < nk / 4 ? ks : nk / 4;              // at least 4 K steps per part
    while (ks > 1 && tail * ks > part_units) --ks;
  }
  if (ks < 2) {
    tail = 0;
    ks = 1;
  }
  F = total - tail;
}

// Tile order over the V valid M tiles (known on the device only): each XCD takes a
// contiguous range of tiles, walked in groups of 4 M tiles, N tile by N tile, so the
// workgroups resident on one XCD share 4 activation slabs and about 8 weight slabs.
constexpr int kMGroupM = 4;
__device__ __forceinline__ void mtile_of(int V, int ntn, int bid, int &mt, int &nt) {
  const int L = xcd_tile(bid, V * ntn);
  const int grp = L / (kMGroupM * ntn);
  const int base = grp * kMGroupM;
  const int gsz = min(kMGroupM, V - base);
  const int li = L - grp * kMGroupM * ntn;
  nt = li / gsz;
  mt = base + (li - nt * gsz);
}

__device__ __forceinline__ uint2 pack_bf16x4(float a, float b, float c, float d) {
  return make_uint2(f2bf(a) | ((uint32_t)f2bf(b) << 16), f2bf(c) | ((uint32_t)f2bf(d) << 16));
}
__device__ __forceinline__ float4 unpack_bf16x4(uint2 u) {
  return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                     __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}

// The gathered rows of all items, packed: packed row p is slot b * N + (p - pre[b]) of
// the item b with pre[b] <= p < pre[b + 1] (pre = exclusive prefix sums of the
// recompute counts), so only the last tile of the whole batch is partly empty.
__device__ __forceinline__ long packed_slot(const int *pre, int B, int N, int p, int &b) {
  int lo = 0, hi = B - 1;                       // largest b with pre[b] <= p
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (pre[mid] <= p) lo = mid; else hi = mid - 1;
  }
  b = lo;
  return (long)lo * N + (p - pre[lo]);
}

// Exclusive prefix sums of the recompute counts into pre[0..B] (wave 0; the caller
// synchronises): each lane sums a run of items, then the runs are scanned.
__device__ __forceinline__ void mg_prefix(const MArgs &a, int *pre) {
  const int lane = threadIdx.x & 63;
  const int per = (a.B + 63) / 64, i0 = lane * per;
  int run = 0;
  for (int i = i0; i < min(i0 + per, a.B); ++i) run += n_valid(a.r.nrec, i, a.N);
  int inc = run;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(inc, o);
    if (lane >= o) inc += v;
  }
  int acc_run = inc - run;
  for (int i = i0; i < min(i0 + per, a.B); ++i) {
    pre[i] = acc_run;
    acc_run += n_valid(a.r.nrec, i, a.N);
  }
  if (lane == 63) pre[a.B] = inc;
}

// Epilogue of 8 tile rows, rows(it) for it = 0..7, by one wave: trow(it) holds the row's
// 256 accumulated columns (SwiGLU: the 128 products), lane l handles columns
// 4 l .. 4 l + 3.  The rows' slots, token ids and residual inputs are loaded for all 8
// rows first, so their memory latencies overlap instead of adding up row by row.
template <int MODE, typename RowOf, typename TrowOf>
__device__ __forceinline__ void mg_epi_rows8(const MArgs &a, const int *pre, RowOf rows,
                                             TrowOf trow, int row0, int nvalid, int col0, int nt) {
  const RedArgs &r = a.r;
  const int lane = threadIdx.x & 63;
  constexpr int TN = MODE == G_GU ? MB / 2 : MB;
  const int c4 = lane * 4;                                   // column within the tile
  const int col = col0 + c4;
  const bool cv = col < a.Nout && c4 < TN;
  bool rv[8];
  int bi[8], tok[8];
  long slot[8];
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    rv[it] = rows(it) < nvalid;
    bi[it] = 0;
    slot[it] = rv[it] ? packed_slot(pre, a.B, a.N, row0 + rows(it), bi[it]) : 0;
    tok[it] = (MODE != G_GU && MODE != G_PLAIN && rv[it]) ? tok_of(r.idx, slot[it], a.N) : 0;
  }
  // residual inputs: x rows for O, h1 rows for down
  uint2 xin[MODE == G_O ? 8 : 1];
  float4 hin[MODE == G_DOWN ? 8 : 1];
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    if (MODE == G_O)
      xin[it] = (rv[it] && cv) ? *reinterpret_cast<const uint2 *>(
                                     r.x + ((long)bi[it] * a.N + tok[it]) * r.d + col)
                               : make_uint2(0, 0);
    if (MODE == G_DOWN)
      hin[it] = (rv[it] && cv) ? *reinterpret_cast<const float4 *>(r.h1 + slot[it] * r.d + col)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
  }
#pragma unroll
  for (int it = 0; it < 8; ++it) {
    const float *tr = trow(it);
    if (MODE == G_GU) {
      if (rv[it] && cv) {
        const float4 v = *reinterpret_cast<const float4 *>(tr + c4);
        *reinterpret_cast<uint2 *>(a.act + slot[it] * a.Nout + col) = pack_bf16x4(v.x, v.y, v.z, v.w);
      }
      continue;
    }
    const float4 v = *reinterpret_cast<const float4 *>(tr + c4);
    if (MODE == G_QKV) {
      if (!rv[it] || !cv) continue;
      const float4 bs = unpack_bf16x4(*reinterpret_cast<const uint2 *>(r.bias + col));
      float o[4] = {v.x + bs.x, v.y + bs.y, v.z + bs.z, v.w + bs.w};
      uint16_t *dst;
      if (col < r.qw) {
        // rotate-half RoPE: the partner dims are half a head away in the same row
        const int half = r.hd / 2, dim = col % r.hd;
        const int pc4 = dim < half ? c4 + half : c4 - half;
        const float4 pv = *reinterpret_cast<const float4 *>(tr + pc4);
        const float4 pb = unpack_bf16x4(*reinterpret_cast<const uint2 *>(r.bias + col0 + pc4));
        const float p[4] = {pv.x + pb.x, pv.y + pb.y, pv.z + pb.z, pv.w + pb.w};
        // four consecutive pairs share one M-RoPE section (sections are multiples of 8)
        const float2 *rp = r.rope + (long)rope_pos(r.mr, r.qpos0 + tok[it], dim % half) * half + dim % half;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float2 cs = rp[q];
          o[q] = dim < half ? o[q] * cs.x - p[q] * cs.y : o[q] * cs.x + p[q] * cs.y;
        }
        dst = r.q + slot[it] * r.qw + col;
      } else {
        const long crow = (long)bi[it] * r.S + pool_row(r.smap, bi[it], r.S, r.cur_row0 + tok[it]);
        dst = col < r.qw + r.kw ? r.kc + crow * r.kw + (col - r.qw)
                                : r.vc + crow * r.kw + (col - r.qw - r.kw);
      }
      *reinterpret_cast<uint2 *>(dst) = pack_bf16x4(o[0], o[1], o[2], o[3]);
    } else if (MODE == G_O) {
      float ss = 0.f;
      if (rv[it] && cv) {
        const float4 xv = unpack_bf16x4(xin[it]);
        const float4 hv = make_float4(v.x + xv.x, v.y + xv.y, v.z + xv.z, v.w + xv.w);
        *reinterpret_cast<float4 *>(r.h1 + slot[it] * r.d + col) = hv;
        const float4 gn = unpack_bf16x4(*reinterpret_cast<const uint2 *>(r.gain + col));
        *reinterpret_cast<uint2 *>(r.hb + slot[it] * r.d + col) =
            pack_bf16x4(hv.x * gn.x, hv.y * gn.y, hv.z * gn.z, hv.w * gn.w);
        ss = hv.x * hv.x + hv.y * hv.y + hv.z * hv.z + hv.w * hv.w;
      }
      // the row's 256 columns are this wave's 64 lanes
#pragma unroll
      for (int m = 32; m > 0; m >>= 1) ss += __shfl_xor(ss, m);
      if (rv[it] && lane == 0 && nt < a.ss_parts) r.ssq[slot[it] * a.ss_parts + nt] = ss;
    } else {
      if (!rv[it] || !cv) continue;
      const float4 hv = hin[it];
      *reinterpret_cast<uint2 *>(r.y + ((long)bi[it] * a.N + tok[it]) * r.d + col) =
          pack_bf16x4(hv.x + v.x, hv.y + v.y, hv.z + v.z, hv.w + v.w);
    }
  }
}

// 1/rms of tile row `row` from the O epilogue's partial sums of squares of h1
__device__ __forceinline__ float mg_rowinv(const MArgs &a, const int *pre, int row0, int row,
                                           int nvalid) {
  float v = 0.f;
  if (row < nvalid) {
    int ib;
    const long sl = packed_slot(pre, a.B, a.N, row0 + row, ib);
    for (int c = 0; c < a.ss_parts; ++c) v += a.r.ssq[sl * a.ss_parts + c];
  }
  return 1.f / sqrtf(v / (float)a.K + a.r.eps);
}

template <int MODE>
__global__ __launch_bounds__(512) void k_mgemm(MArgs a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[2 * kMStage];
  __shared__ float rowinv[MB];
  __shared__ int pre[kMMaxItems + 1];
  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  if (w == 0) mg_prefix(a, pre);
  __syncthreads();
  // the grid covers every slot; only the tiles of the packed rows run, the tail
  // tiles as K-range parts
  const int V = (pre[a.B] + MB - 1) / MB;
  const int nk = a.K / KS;
  const int bid = blockIdx.x;
  int split = 0;
  int mt, nt, kb = 0, ke = nk, unit = -1;
  if (MODE == G_PLAIN) {
    // every tile as ks K-range parts, part p of tile i at workgroup p V ntn + i
    const int T = V * a.ntn;
    const int ks = plain_split(T, a.cus, nk);
    if (bid == 0 && t == 0) *a.ks_out = ks;
    if (bid >= T * ks) return;
    split = bid / T;
    mtile_of(V, a.ntn, bid - split * T, mt, nt);
    kb = split * nk / ks;
    ke = (split + 1) * nk / ks;
  } else {
    int F, tail, ks;
    mtail_split(V * a.ntn, a.cus, a.part_units, nk, F, tail, ks);
    if (bid >= F + tail * ks) return;
    if (bid < F) {
      mtile_of(V, a.ntn, bid, mt, nt);
    } else {
      const int u = bid - F, ti = u % tail, kp = u / tail;
      mtile_of(V, a.ntn, F + ti, mt, nt);
      kb = kp * nk / ks;
      ke = (kp + 1) * nk / ks;
      unit = ti * ks + kp;
    }
  }
  const int row0 = mt * MB;
  const int nvalid = min(MB, pre[a.B] - row0);
  const int wm = w & 1, wn = w >> 1;
  const int l32 = lane & 31, h = lane >> 5;
  // output columns of this tile: SwiGLU stages 32 gate + 32 up rows per wave column
  constexpr int TN = MODE == G_GU ? MB / 2 : MB;
  const int col0 = nt * TN;

  // DMA instruction j of a step (this wave issues j = w + 8 i) stages 8 rows:
  // j < 32 the activation rows 8 j .., else the staged weight rows 8 (j - 32) ..
  const int rsub = lane >> 3, ch = lane & 7;
  const uint16_t *gp[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int j = w + 8 * i;
    const int r = (j & 31) * 8 + rsub;                         // row within its operand
    const int cs = (ch ^ swz8(r)) * 8;
    if (j < 32) {
      const int rr = r < nvalid ? r : nvalid - 1;              // clamp: never stored
      int ib;
      gp[i] = a.A + packed_slot(pre, a.B, a.N, row0 + rr, ib) * a.K + cs;
    } else {
      const uint16_t *M = a.W0;
      int col;
      if (MODE == G_GU) {
        col = col0 + (r >> 6) * 32 + (r & 31);
        if (r & 32) M = a.W1;
      } else {
        col = col0 + r;
      }
      col = min(col, a.Nout - 1);                              // clamp: never stored
      gp[i] = M + (long)col * a.K + cs;
    }
  }
  const uint32_t lbase = lds_addr(lds);
  auto issue = [&](int kt) {
    const int kk = kt * KS;
    const uint32_t st = lbase + (kt & 1) * kMStage;
#pragma unroll
    for (int i = 0; i < 8; ++i) dma16(gp[i] + kk, st + (w + 8 * i) * 1024);
  };

  if (MODE == G_GU && t < MB && unit < 0) rowinv[t] = mg_rowinv(a, pre, row0, t, nvalid);

  f32x16 acc[4][2];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  // fragment of block i, sub-step s: row l32 of the block, 16-B chunk 2 s + h
  const int sw = swz8(l32);
  const uint32_t aoff = (uint32_t)((wm * 128 + l32) * RB);
  const uint32_t boff = (uint32_t)((MB + wn * 64 + l32) * RB);
  auto rd = [&](const unsigned char *st, int s, bf16x8 (&fa)[4], bf16x8 (&fb)[2]) {
    const uint32_t slot = (uint32_t)(((2 * s + h) ^ sw) << 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) fa[i] = *reinterpret_cast<const bf16x8 *>(st + aoff + i * 32 * RB + slot);
#pragma unroll
    for (int j = 0; j < 2; ++j) fb[j] = *reinterpret_cast<const bf16x8 *>(st + boff + j * 32 * RB + slot);
  };

  // The next step's DMAs go into the stage of step k - 1 as soon as the barrier frees
  // it: waves 0-3 before their first MFMA, waves 4-7 (the other wave of each SIMD) one
  // sub-step later, so that each SIMD always has a wave issuing MFMAs.
  const bool early = w < 4;
  issue(kb);
  for (int k = kb; k < ke; ++k) {
    wait_vm<0>();                                              // this wave's share of step k
    lds_barrier();                                             // all of step k; step k - 1 read
    const unsigned char *st = lds + (k & 1) * kMStage;
    const bool more = k + 1 < ke;
    if (more && early) issue(k + 1);
    bf16x8 fa[2][4], fb[2][2];
    rd(st, 0, fa[0], fb[0]);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      if (s == 1 && more && !early) issue(k + 1);
      if (s < 3) rd(st, s + 1, fa[(s + 1) & 1], fb[(s + 1) & 1]);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[s & 1][i], fb[s & 1][j], acc[i][j], 0, 0, 0);
    }
  }
  lds_barrier();                                               // the stages are free

  if (MODE == G_PLAIN) {
    // the raw K-range sums straight from the accumulators, tile-contiguous: part `split`
    // of tile (mt, nt) is the [256 packed rows][256 columns] block at
    // ((split V + mt) ntn + nt) 256^2, V the valid M tiles (rows past the packed rows are
    // not stored)
    float *ob = a.out + (((long)split * V + mt) * a.ntn + nt) * (MB * MB);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int rr = wm * 128 + i * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
        if (rr >= nvalid) continue;
#pragma unroll
        for (int j = 0; j < 2; ++j) ob[rr * MB + wn * 64 + j * 32 + l32] = acc[i][j][e];
      }
    return;
  }
  if (unit >= 0) {
    // a part of a tail tile: the raw fp32 accumulators, [256 rows][256 staged columns]
    float *pt = a.part + (long)unit * (MB * MB);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int rr = wm * 128 + i * 32 + (e >> 2) * 8 + h * 4 + (e & 3);
          pt[rr * MB + wn * 64 + j * 32 + l32] = acc[i][j][e];
        }
    return;
  }

  // ---------------------------------------------------------------- fused epilogue
  // Per 32-row block i: the waves put their accumulators into an LDS tile ([2][32]
  // rows of 256 floats; SwiGLU: the 128 products), then each wave handles whole
  // rows, one 4-column piece per lane.  A lane's accumulator element e of block
  // (i, j) is column l32 of row 8 (e / 4) + 4 h + e % 4.
  float *T = reinterpret_cast<float *>(lds);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int rr = (e >> 2) * 8 + h * 4 + (e & 3);
      float *trow = T + (wm * 32 + rr) * kMEpPitch;
      if (MODE == G_GU) {
        const float sc = rowinv[wm * 128 + i * 32 + rr];
        const float gv = acc[i][0][e] * sc, uv = acc[i][1][e] * sc;
        trow[wn * 32 + l32] = gv / (1.f + __expf(-gv)) * uv;
      } else {
        trow[wn * 64 + l32] = acc[i][0][e];
        trow[wn * 64 + 32 + l32] = acc[i][1][e];
      }
    }
    lds_barrier();
    // 64 rows (two per wave-row half) x 64 four-column pieces: wave w takes epilogue rows
    // er = w + 8 it (0..63), tile rows 128 (er / 32) + 32 i + er % 32
    mg_epi_rows8<MODE>(
        a, pre, [&](int it) { const int er = w + 8 * it; return (er >> 5) * 128 + i * 32 + (er & 31); },
        [&](int it) { return T + (w + 8 * it) * kMEpPitch; }, row0, nvalid, col0, nt);
    lds_barrier();                                             // the tile is free again
  }
}

// The tail tiles of a large-M GEMM: the ks K-range partial tiles are summed in part
// order and go through the same epilogue as a whole tile.  Workgroup 4 q + i handles
// tail tile q, rows i * 32 .. and 128 + i * 32 .. (the rows of epilogue block i).
template <int MODE>
__global__ __launch_bounds__(512) void k_mtail(MArgs a) {
  __shared__ __attribute__((aligned(16))) float S[64 * kMEpPitch];
  __shared__ __attribute__((aligned(16))) float P[MODE == G_GU ? 64 * kMEpPitch : 4];
  __shared__ float rowinv[64];
  __shared__ int pre[kMMaxItems + 1];
  const int t = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  if (w == 0) mg_prefix(a, pre);
  __syncthreads();
  const int V = (pre[a.B] + MB - 1) / MB;
  const int nk = a.K / KS;
  int F, tail, ks;
  mtail_split(V * a.ntn, a.cus, a.part_units, nk, F, tail, ks);
  const int q = blockIdx.x >> 2, i = blockIdx.x & 3;
  if (q >= tail) return;
  int mt, nt;
  mtile_of(V, a.ntn, F + q, mt, nt);
  const int row0 = mt * MB;
  const int nvalid = min(MB, pre[a.B] - row0);
  constexpr int TN = MODE == G_GU ? MB / 2 : MB;
  const int col0 = nt * TN;
  // thread t sums row er = t / 8, columns 32 (t % 8) .. + 32, over the parts in order
  {
    const int er = t >> 3, row = (er >> 5) * 128 + i * 32 + (er & 31);
    const float *p0 = a.part + (long)q * ks * (MB * MB) + (long)row * MB + (t & 7) * 32;
    float4 sum[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) sum[c] = *reinterpret_cast<const float4 *>(p0 + 4 * c);
    for (int kp = 1; kp < ks; ++kp) {
      const float *pk = p0 + (long)kp * (MB * MB);
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        const float4 v = *reinterpret_cast<const float4 *>(pk + 4 * c);
        sum[c] = make_float4(sum[c].x + v.x, sum[c].y + v.y, sum[c].z + v.z, sum[c].w + v.w);
      }
    }
#pragma unroll
    for (int c = 0; c < 8; ++c)
      *reinterpret_cast<float4 *>(&S[er * kMEpPitch + (t & 7) * 32 + 4 * c]) = sum[c];
    if (MODE == G_GU && t < 64) {
      const int r2 = (t >> 5) * 128 + i * 32 + (t & 31);
      rowinv[t] = mg_rowinv(a, pre, row0, r2, nvalid);
    }
  }
  __syncthreads();
  const float *T = S;
  if (MODE == G_GU) {
    // product c of a row: gate at staged column 64 (c / 32) + c % 32, up 32 further
    for (int e = t; e < 64 * (MB / 2); e += 512) {
      const int er = e >> 7, c = e & 127;
      const float sc = rowinv[er];
      const float gv = S[er * kMEpPitch + (c >> 5) * 64 + (c & 31)] * sc;
      const float uv = S[er * kMEpPitch + (c >> 5) * 64 + 32 + (c & 31)] * sc;
      P[er * kMEpPitch + c] = gv / (1.f + __expf(-gv)) * uv;
    }
    __syncthreads();
    T = P;
  }
  mg_epi_rows8<MODE>(
      a, pre, [&](int it) { const int er = w + 8 * it; return (er >> 5) * 128 + i * 32 + (er & 31); },
      [&](int it) { return T + (w + 8 * it) * kMEpPitch; }, row0, nvalid, col0, nt);
}

// ------------------------------------------------------------------------------- attention
struct AttnArgs {
  const uint16_t *q;          // [B*N][nh*HD], rotated at the query's position
  const uint16_t *kc, *vc;    // [B][S][nkv][HD]
  const int32_t *smap;        // slot map of the K/V rows (null: rows in place)
  const float2 *rope;         // [S][HD/2] (cos, sin)
  const int32_t *idx, *nrec;
  int N, nh, nkv, S, T, W, head;
  int fN;                     // tokens per frame (N: query tokens of the region)
  int cur_lo, qpos0;          // first cache row and prompt index of the query region
  int frames_end;             // T + W fN: text after the frames starts here
  MRope mr;                   // RoPE positions of the keys (1-D or multimodal)
  int splits, kb_per_split;
  int tiles;                  // B * ceil(N / 32) query tiles
  float scale_log2;
  uint16_t *out;              // [B*N][nh*HD] (splits == 1)
  float *po;                  // [split][B*N][nh][HD] unnormalised partial output
  float *pm, *pl;             // [split][B*N][nh] running max (log2 units) and sum
};

__device__ __forceinline__ int key_pos(int row, int T, int N, int W, int head) {
  if (row < T || row >= T + W * N) return row;     // text before and after the frames
  const int r = row - T;
  const int p = r / N, i = r - p * N;
  int lg = p - head;
  if (lg < 0) lg += W;
  return T + lg * N + i;
}


// Raw data of one staging task of a 32-key block (the same task count for keys and
// values): two 8-dim key chunks, the (cos, sin) pairs of those dims at the key's
// position when the keys are rotated on load, the position itself (INT_MAX past the
// end of the cache), and 4 dims of 4 consecutive values.
struct KVRaw {
  u32x4 k1, k2;
  u32x4 cs[4];
  u32x2 v[4];
  int pos;
};

// The raw loads are inline asm and their waits explicit: the compiler would otherwise
// copy the pipelined registers right after issue and wait on every block's loads.
// These loads read only the cache and the RoPE table, which no kernel of the layer
// writes while attention runs.
__device__ __forceinline__ u32x4 kv_load16(const void *p) {
  u32x4 r;
  asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(p));
  return r;
}
__device__ __forceinline__ u32x2 kv_load8(const void *p) {
  u32x2 r;
  asm volatile("global_load_dwordx2 %0, %1, off" : "=v"(r) : "v"(p));
  return r;
}
// The same from a wave-uniform base (scalar registers) plus a 32-bit byte offset per
// lane, which spares the 64-bit address arithmetic per load.
__device__ __forceinline__ const unsigned char *uniform_ptr(const void *p) {
  const uint64_t u = (uint64_t)(uintptr_t)p;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return reinterpret_cast<const unsigned char *>((uintptr_t)(((uint64_t)hi << 32) | lo));
}
__device__ __forceinline__ u32x4 kv_load16s(const unsigned char *base, uint32_t off) {
  u32x4 r;
  asm volatile("global_load_dwordx4 %0, %1, %2" : "=v"(r) : "v"(off), "s"(base));
  return r;
}
__device__ __forceinline__ u32x2 kv_load8s(const unsigned char *base, uint32_t off) {
  u32x2 r;
  asm volatile("global_load_dwordx2 %0, %1, %2" : "=v"(r) : "v"(off), "s"(base));
  return r;
}
template <typename T>
__device__ __forceinline__ void kv_anchor(T &r) { asm volatile("" : "+v"(r)); }
__device__ __forceinline__ float lo_f(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float hi_f(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
__device__ __forceinline__ uint16_t bf16_bits(float f) {
  return __builtin_bit_cast(uint16_t, (__bf16)f);   // round to nearest even
}

// Rotated keys sit in LDS as unpadded rows of HD bf16; 16-B chunk q of key r is
// stored at chunk q ^ kswz(r), which spreads both the MFMA reads (16 keys, one
// chunk) and the staging writes (2 or 4 keys, all chunks) over all banks.
template <int HD>
__device__ __forceinline__ int kswz(int key) {
  return HD == 128 ? (((key & 1) << 3) | ((key >> 1) & 7)) : ((key >> 1) & 7);
}
// Values sit as [key / 4][HD / 32][32][4 keys]: the 4 consecutive keys of one dim
// form one 8-B word (half an MFMA A fragment), and dim h of group h / 32 is at
// slot (h + h / 32) % 32 of its group, so the staging writes (dims 4 apart across
// lanes) and the fragment reads (32 consecutive dims) both hit distinct banks.
template <int HD>
__device__ __forceinline__ int vq_word(int kg, int hd) {
  return (kg * (HD / 32) + (hd >> 5)) * 32 + (((hd & 31) + (hd >> 5)) & 31);
}

// Attention of one 32-query tile of kv head g over key blocks [kb0, kb1) of the cache.
// Wave w < G handles query head g*G + w; the queries arrive rotated.  The waves past
// them only move data: they fetch the raw K/V rows, rotate the keys (unless the keys
// come rotated) and stage both into one of two LDS buffers (keys rotated, values
// interleaved), with the raw loads of block kb + 2 in flight while block kb is
// multiplied, so the cache latency is paid once per split and the staging ALU work
// runs beside the MFMAs.
constexpr int kAttnStageWaves = 4;
// Slot-mapped caches: the pool rows of a workgroup's key range are staged in LDS (at
// most this many rows per key split); only the four-staging-wave variants take a map.
constexpr int kAttnMapRows = 4096;
template <int HD, int G, bool ROT, int QB, int SW>
__global__ __launch_bounds__((G + SW) * 64) void k_attn(AttnArgs a) {
  constexpr int NS = HD / 16;   // k-steps of the QK^T product
  constexpr int NHB = HD / 32;  // 32-row blocks of the output
  constexpr int NL = SW * 64;   // staging threads
  constexpr int CPK = HD / 16;  // key staging tasks per key
  constexpr int TASKS = 32 * CPK;
  constexpr int TPT = (TASKS + NL - 1) / NL;   // staging tasks per thread
  constexpr int QR = 32 * QB;   // query rows of a tile: QB blocks of 32 per query wave
  constexpr int QLD = HD + 8;   // padded LDS row of the rotated queries
  static_assert(TASKS % 64 == 0, "staging tasks fill whole waves");
  static_assert(TASKS == 8 * (HD / 4), "key and value tasks pair up");
  static_assert(TPT == 1 || TPT * NL == TASKS, "tasks divide over the staging threads");
  static_assert(QB == 1 || QB == 2, "one or two query blocks per wave");
  __shared__ __attribute__((aligned(16))) __bf16 Qs[G][QR * QLD];
  __shared__ __attribute__((aligned(16))) __bf16 Ks[2][32 * HD];
  __shared__ __attribute__((aligned(16))) uint2 Vq[2][8 * HD];
  __shared__ int kpos[2][32];
  __shared__ int rmap[SW > 1 ? kAttnMapRows : 1];

  // 1-D grid; the query tiles of one (kv head, key split) are consecutive logical
  // tiles, which xcd_tile places on one XCD, so each XCD's L2 holds only its own
  // share of the cache
  const int tiles = a.tiles;
  const int lt = xcd_tile(blockIdx.x, (int)gridDim.x);
  const int g = (lt / tiles) % a.nkv;
  const int sp = lt / (tiles * a.nkv);
  const int tiles_per_b = (a.N + QR - 1) / QR;
  // an item's tiles are dispatched last first: later tiles see more of the current
  // frame's keys (fewer skipped blocks), so the longest workgroups start first and the
  // short ones fill the last round
  const int b = (lt % tiles) / tiles_per_b;
  const int qt = b * tiles_per_b + (tiles_per_b - 1 - (lt % tiles) % tiles_per_b);
  const int j0 = (qt % tiles_per_b) * QR;
  const int n = n_valid(a.nrec, b, a.N);
  if (j0 >= n) return;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  // waves below G multiply (one query head each); the waves past them fetch, rotate
  // and stage the next key block meanwhile, so loads and staging overlap the MFMAs
  const bool qwave = w < G;
  const int tl = t - G * 64;          // staging thread index (staging waves only)
  const int h = g * G + (qwave ? w : 0);

  const int nkb = (a.S + 31) / 32;
  const int kb0 = sp * a.kb_per_split;
  const int kb1 = min(nkb, kb0 + a.kb_per_split);
  const long kvbase = (long)b * a.S * a.nkv * HD + (long)g * HD;
  const long kvrow = (long)a.nkv * HD;
  // only the current frame's keys can lie after a query; other blocks skip the mask
  // (the query region: the current frame's slot, or the text after the frames)
  const int cur_lo = a.cur_lo, cur_hi = cur_lo + a.N;

  auto needs_mask = [&](int kb) {
    const int r0 = kb * 32, r1 = r0 + 32;
    return r1 > a.S || (r1 > cur_lo && r0 < cur_hi) || r1 > a.frames_end;
  };
  // Key blocks of the current frame's slot past the tile's last query: every key in
  // them comes after every query of the tile, so they add exactly nothing to the
  // softmax and are skipped.  Loop index i runs over the other blocks of the split.
  __shared__ int tile_tok_max;
  if (w == 0) {
    int v = -1;
    if (lane < QR && j0 + lane < n) v = tok_of(a.idx, (long)b * a.N + j0 + lane, a.N);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o));
    if (lane == 0) tile_tok_max = v;
  }
  // slot-mapped caches: the pool row of every row of the split's key range
  const bool mapped = SW > 1 && a.smap != nullptr;
  const int m0 = kb0 * 32;
  const int m1 = min(kb1 * 32, a.S);          // rows [m0, m1) are staged
  if (mapped) {
    for (int r = t; r < m1 - m0; r += blockDim.x) rmap[r] = pool_row(a.smap, b, a.S, m0 + r);
  }
  __syncthreads();
  int s0 = (cur_lo + tile_tok_max + 1 + 31) / 32, s1 = min(cur_hi, a.S) / 32;
  s0 = max(s0, kb0);
  s1 = min(s1, kb1);
  if (s1 < s0) s1 = s0;
  const int nb = (kb1 - kb0) - (s1 - s0);
  // block of loop index i (clamped to the last); a split with no block left (nb = 0)
  // still prefetches one block of its own range, never multiplied
  auto blk = [&](int i) {
    i = max(min(i, nb - 1), 0);
    const int k = kb0 + i;
    return min(min(k >= s0 ? k + (s1 - s0) : k, kb1 - 1), nkb - 1);
  };

  if (!qwave) {
    // ------------------------------------------------------------ staging waves
    // Fetch, (rotate and) stage block kb + 1 while block kb is multiplied.  Everything
    // that does not depend on the block is computed once here: task i of a thread is
    //   keys:   dims [8c, 8c + 8) and [HD/2 + 8c, HD/2 + 8c + 8) of key `key`;
    //   values: dims [4l, 4l + 4) of keys 4kg .. 4kg + 3,
    // so per block only the row offset of the block is added.
    // Byte offsets of a task's loads from the first row of a full block: key row
    // `key`, dims 8c..; value rows 4kg + r, dims 4l..
    bool act[TPT];
    int key[TPT], c[TPT], kg[TPT], lq[TPT], kofs1[TPT], kofs2[TPT], vofs[TPT][4];
    uint32_t koff[TPT], voff[TPT][4];
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      act[i] = tl + i * NL < TASKS;
      const int tk = act[i] ? tl + i * NL : 0;
      key[i] = tk / CPK;
      c[i] = tk - key[i] * CPK;
      kg[i] = tk / (HD / 4);
      lq[i] = tk - kg[i] * (HD / 4);
      const int ksw = kswz<HD>(key[i]);
      kofs1[i] = key[i] * HD + 8 * (c[i] ^ ksw);
      kofs2[i] = key[i] * HD + 8 * ((c[i] + HD / 16) ^ ksw);
#pragma unroll
      for (int q = 0; q < 4; ++q) vofs[i][q] = vq_word<HD>(kg[i], 4 * lq[i] + q);
      koff[i] = (uint32_t)(key[i] * kvrow * 2 + 16 * c[i]);
#pragma unroll
      for (int r = 0; r < 4; ++r) voff[i][r] = (uint32_t)((4 * kg[i] + r) * kvrow * 2 + 8 * lq[i]);
    }
    const int S = a.S;

    // raw loads of block kb (the pipeline runs ahead onto the last block again: those
    // loads are never multiplied)
    auto fetch = [&](int kb, KVRaw (&R)[TPT]) {
      const int rb = kb * 32;                          // first row of the block (uniform)
      // positions: rows of one region (text, or one frame slot of the ring) share the
      // shift from row to position
      int delta = 0;
      bool uniform_pos = rb + 32 <= a.T || rb >= a.frames_end;
      if (!uniform_pos && rb >= a.T) {
        const int p0 = (rb - a.T) / a.fN, p1 = (min(rb + 31, S - 1) - a.T) / a.fN;
        if (p0 == p1) {
          int lg = p0 - a.head;
          if (lg < 0) lg += a.W;
          delta = (lg - p0) * a.fN;
          uniform_pos = true;
        }
      }
      // the block's first K and V rows as scalar bases; rows past the end of the cache
      // read its last row (lim, relative to the block) again and are never multiplied
      const int lim = S - 1 - rb;
      const uint32_t lim_off = (uint32_t)(lim * kvrow * 2);
      // (slot-mapped: the item's first row as base, each row's pool row as offset)
      const unsigned char *kblk = uniform_ptr(a.kc + kvbase + (mapped ? 0L : (long)rb * kvrow));
      const unsigned char *vblk = uniform_ptr(a.vc + kvbase + (mapped ? 0L : (long)rb * kvrow));
#pragma unroll
      for (int i = 0; i < TPT; ++i) {
        const int row0 = rb + key[i];
        const int row = min(row0, S - 1);
        const int pos = uniform_pos ? row + delta : key_pos(row, a.T, a.fN, a.W, a.head);
        R[i].pos = row0 < S ? pos : 0x7fffffff;
        const uint32_t ko = mapped ? (uint32_t)(rmap[min(row, m1 - 1) - m0] * kvrow * 2 + 16 * c[i])
                                   : (key[i] <= lim ? koff[i] : lim_off + 16 * c[i]);
        R[i].k1 = kv_load16s(kblk, ko);
        R[i].k2 = kv_load16s(kblk, ko + HD);
        if (ROT) {
          const float2 *rp = a.rope + (long)rope_pos(a.mr, pos, 8 * c[i]) * (HD / 2) + 8 * c[i];
#pragma unroll
          for (int q = 0; q < 4; ++q) R[i].cs[q] = kv_load16(rp + 2 * q);
        }
        // every asm load is unconditional (no register set chosen at run time)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t vo =
              mapped ? (uint32_t)(rmap[min(rb + 4 * kg[i] + r, m1 - 1) - m0] * kvrow * 2 + 8 * lq[i])
                     : (4 * kg[i] + r <= lim ? voff[i][r] : lim_off + 8 * lq[i]);
          R[i].v[r] = kv_load8s(vblk, vo);
        }
      }
    };
    // the loads of R are complete once only the other set's loads (issued after R's)
    // may still be in flight
    auto settle = [&](KVRaw (&R)[TPT]) {
      constexpr int kLater = (ROT ? 10 : 6) * TPT;
      static_assert(kLater < 64, "vmcnt holds at most 63 outstanding loads");
      __builtin_amdgcn_s_waitcnt(0x3F70 | (kLater & 0xF) | ((kLater >> 4) << 14));
#pragma unroll
      for (int i = 0; i < TPT; ++i) {
        kv_anchor(R[i].k1); kv_anchor(R[i].k2);
        if (ROT) {
#pragma unroll
          for (int q = 0; q < 4; ++q) kv_anchor(R[i].cs[q]);
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) kv_anchor(R[i].v[r]);
      }
    };
    // rotate-half RoPE of the keys (unless they come rotated) into Ks[buf]; values
    // interleaved into Vq[buf]: word q of a task holds dim 4l + q of its 4 keys
    auto stage = [&](const KVRaw (&R)[TPT], int buf) {
      __bf16 *kr = &Ks[buf][0];
#pragma unroll
      for (int i = 0; i < TPT; ++i) {
        if (!act[i]) continue;
        if (ROT) {
          U16x8 k1, k2;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const u32x4 q = R[i].cs[e >> 1];
            const float cs = __uint_as_float(q[(e & 1) * 2]), sn = __uint_as_float(q[(e & 1) * 2 + 1]);
            const uint32_t w1 = R[i].k1[e >> 1], w2 = R[i].k2[e >> 1];
            const float x1 = (e & 1) ? hi_f(w1) : lo_f(w1), x2 = (e & 1) ? hi_f(w2) : lo_f(w2);
            k1.v[e] = bf16_bits(x1 * cs - x2 * sn);
            k2.v[e] = bf16_bits(x2 * cs + x1 * sn);
          }
          *reinterpret_cast<U16x8 *>(kr + kofs1[i]) = k1;
          *reinterpret_cast<U16x8 *>(kr + kofs2[i]) = k2;
        } else {
          *reinterpret_cast<u32x4 *>(kr + kofs1[i]) = R[i].k1;
          *reinterpret_cast<u32x4 *>(kr + kofs2[i]) = R[i].k2;
        }
        if (c[i] == 0) kpos[buf][key[i]] = R[i].pos;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          // low (q even) or high (q odd) bf16 halves of word q / 2 of the 4 rows
          const uint32_t sel = (q & 1) ? 0x07060302u : 0x05040100u;
          const uint32_t x = __builtin_amdgcn_perm(R[i].v[1][q >> 1], R[i].v[0][q >> 1], sel);
          const uint32_t y = __builtin_amdgcn_perm(R[i].v[3][q >> 1], R[i].v[2][q >> 1], sel);
          Vq[buf][vofs[i][q]] = make_uint2(x, y);
        }
      }
    };

    // two register sets with fixed roles (an asm load must never write a register set
    // chosen at run time: the compiler would copy it before it lands)
    KVRaw ra[TPT], rb[TPT];
    fetch(blk(0), ra);
    fetch(blk(1), rb);
    settle(ra);
    stage(ra, 0);
    lds_barrier();
    for (int i = 0; i < nb; i += 2) {
      fetch(blk(i + 2), ra);
      settle(rb);
      stage(rb, 1);
      lds_barrier();
      fetch(blk(i + 3), rb);
      settle(ra);
      stage(ra, 0);
      lds_barrier();
    }
    // nothing may be left in flight when the wave ends
    __builtin_amdgcn_s_waitcnt(0x3F70);
    return;
  }

  // ------------------------------------------------------------ query waves
  // query block qb of this wave: queries j0 + 32 qb + l32
  bool qvalid[QB];
  long slot[QB];
  int qpos[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int j = j0 + 32 * qb + l32;
    qvalid[qb] = j < n;
    slot[qb] = (long)b * a.N + (qvalid[qb] ? j : j0);
    qpos[qb] = a.qpos0 + tok_of(a.idx, slot[qb], a.N);
  }
  f32x16 o[QB][NHB];
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m_run[qb] = -INFINITY;
    l_run[qb] = 0.f;
#pragma unroll
    for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
      for (int e = 0; e < 16; ++e) o[qb][hb][e] = 0.f;
  }
  // S^T = K Q^T for the 32 keys of buffer buf, each key fragment serving every query
  // block (independent accumulation chains)
  auto qk = [&](int buf, f32x16 (&st)[QB]) {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int e = 0; e < 16; ++e) st[qb][e] = 0.f;
    const int ksw = kswz<HD>(l32);
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bf16x8 ka = *reinterpret_cast<const bf16x8 *>(&Ks[buf][l32 * HD + 8 * ((2 * s + hi) ^ ksw)]);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const bf16x8 qv = *reinterpret_cast<const bf16x8 *>(&Qs[w][(32 * qb + l32) * QLD + 16 * s + 8 * hi]);
        st[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qv, st[qb], 0, 0, 0);
      }
    }
  };
  // online softmax of the scores of buffer buf, then O^T += V^T P^T, each value
  // fragment serving every query block
  auto softmax_pv = [&](f32x16 (&st)[QB], int buf, bool masked) {
    bf16x8 pb[QB][2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      // raw scores here; the scale (> 0, in log2 units) enters the maximum once and each
      // exponent through one fused multiply-add
      float mloc = -INFINITY;
      if (masked) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = (e >> 2) * 8 + hi * 4 + (e & 3);
          st[qb][e] = (kpos[buf][key] <= qpos[qb]) ? st[qb][e] : -INFINITY;
          mloc = fmaxf(mloc, st[qb][e]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) mloc = fmaxf(mloc, st[qb][e]);
      }
      mloc = fmaxf(mloc, __shfl_xor(mloc, 32)) * a.scale_log2;
      // The reference maximum moves only when a score exceeds it by more than 2^8 (in
      // log2 units): below that the probabilities stay under 256, which fp32 sums and
      // bf16 products hold with the same relative precision, and the rescale of the
      // output sums is skipped.  The final division uses the same reference.
      const bool grow = mloc > m_run[qb] + 8.f;
      if (__ballot(grow)) {
        const float corr = grow ? __builtin_amdgcn_exp2f(m_run[qb] - mloc) : 1.f;
        l_run[qb] *= corr;
#pragma unroll
        for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
          for (int e = 0; e < 16; ++e) o[qb][hb][e] *= corr;
        if (grow) m_run[qb] = mloc;
      }
      const float m_use = (m_run[qb] == -INFINITY) ? 0.f : m_run[qb];
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        st[qb][e] = __builtin_amdgcn_exp2f(fmaf(st[qb][e], a.scale_log2, -m_use));
        psum += st[qb][e];
      }
      l_run[qb] += psum;
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int i = 0; i < 8; ++i) pb[qb][s2][i] = (__bf16)st[qb][8 * s2 + i];
    }
    // k index (8 hi + i) of step s2 <-> key 16 s2 + 8 (i/4) + 4 hi + i%4, which is
    // accumulator element 8 s2 + i of S^T in this lane; its 4-key halves are words
    // of key groups 4 s2 + hi and 4 s2 + 2 + hi
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb) {
        const int hd = hb * 32 + l32;
        const uint2 v0 = Vq[buf][vq_word<HD>(4 * s2 + hi, hd)];
        const uint2 v1 = Vq[buf][vq_word<HD>(4 * s2 + 2 + hi, hd)];
        const bf16x8 va = __builtin_bit_cast(bf16x8, u32x4{v0.x, v0.y, v1.x, v1.y});
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          o[qb][hb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[qb][s2], o[qb][hb], 0, 0, 0);
      }
    }
  };
  {
    // Q fragments (B operand of S^T = K Q^T; lane holds q[16 s + 8 hi + e]): the tile's
    // rotated query rows (the G heads of kv group g are contiguous in a row) are staged
    // through LDS with whole-line loads while the first key blocks are in flight
    constexpr int QT = G * 64;                        // query-wave threads
    constexpr int QCH = G * HD / 8;                   // 16-B chunks of one query row
    constexpr int QIT = (QR * QCH + QT - 1) / QT;     // chunks per thread
    uint4 qv[QIT];
#pragma unroll
    for (int i = 0; i < QIT; ++i) {
      const int c = min(t + i * QT, QR * QCH - 1);
      const int r = c / QCH, x = c - r * QCH;
      const long sl = (long)b * a.N + (j0 + r < n ? j0 + r : j0);
      qv[i] = *reinterpret_cast<const uint4 *>(a.q + sl * (a.nh * HD) + (long)g * G * HD + 8 * x);
    }
#pragma unroll
    for (int i = 0; i < QIT; ++i) {
      const int c = t + i * QT;
      if (c < QR * QCH) {
        const int r = c / QCH, x = c - r * QCH;
        *reinterpret_cast<uint4 *>(&Qs[(8 * x) / HD][r * QLD + (8 * x) % HD]) = qv[i];
      }
    }
  }
  lds_barrier();
  for (int i = 0; i < nb; i += 2) {
    f32x16 st[QB];
    qk(0, st);
    softmax_pv(st, 0, needs_mask(blk(i)));                         // buffer 0: index i
    lds_barrier();
    if (i + 1 < nb) {                                              // buffer 1: index i + 1
      qk(1, st);
      softmax_pv(st, 1, needs_mask(blk(i + 1)));
    }
    lds_barrier();
  }

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
    if (a.splits == 1) {
      if (!qvalid[qb]) continue;
      uint16_t *orow = a.out + slot[qb] * (long)(a.nh * HD) + h * HD;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
        for (int e = 0; e < 16; ++e)
          orow[hb * 32 + (e >> 2) * 8 + hi * 4 + (e & 3)] = f2bf(o[qb][hb][e] * inv);
    } else if (QB == 1) {
      // partials of this (split, tile, head) in accumulator order: 16-B group i of
      // lane L at ((i * 64) + L) * 16 B, so each wave store is 1 KB contiguous; the
      // running max and sum per query follow as [split][tile][head][32].  (Two-block
      // tiles are launched with one split only.)
      const long blk = ((long)sp * tiles + qt) * a.nh + h;
      float4 *po = reinterpret_cast<float4 *>(a.po) + blk * (NHB * 4 * 64);
#pragma unroll
      for (int hb = 0; hb < NHB; ++hb)
#pragma unroll
        for (int eg = 0; eg < 4; ++eg)
          po[(hb * 4 + eg) * 64 + lane] = make_float4(o[qb][hb][4 * eg], o[qb][hb][4 * eg + 1],
                                                      o[qb][hb][4 * eg + 2], o[qb][hb][4 * eg + 3]);
      if (hi == 0) {
        a.pm[blk * 32 + l32] = m_run[qb];
        a.pl[blk * 32 + l32] = l_tot;
      }
    }
  }
}

// Rotate-half RoPE of every cached key at its position in the current step, raw
// cache -> rotated copy (same rounding as when the attention kernel rotates on load).
// For many query tiles per item this replaces one rotation per (key, tile) by one per
// key.  One thread per 8-dim pair of chunks (dims 8c.. and hd/2 + 8c..) of a key row.
// Slot-mapped caches (smap): keys are read from their pool rows and written in row
// order, and the values are gathered into vr in row order too, so that the attention
// kernel reads both without the map.
__global__ __launch_bounds__(256) void k_rot_keys(const uint16_t *__restrict__ kc,
                                                  const float2 *__restrict__ rope,
                                                  uint16_t *__restrict__ kr, int S, int nkv,
                                                  int hd, int T, int N, int W, int head,
                                                  MRope mr, const int32_t *__restrict__ smap,
                                                  const uint16_t *__restrict__ vc,
                                                  uint16_t *__restrict__ vr) {
  const int cpr = hd / 16;                              // chunk pairs per head row
  const long task = (long)blockIdx.x * 256 + threadIdx.x;
  const int b = blockIdx.y;
  if (task >= (long)S * nkv * cpr) return;
  const int c = (int)(task % cpr);
  const long rh = task / cpr;                           // row * nkv + kv head
  const int row = (int)(rh / nkv);
  const int pos = key_pos(row, T, N, W, head);
  const long off = ((long)b * S * nkv + rh) * hd + 8 * c;
  const long src = smap ? ((long)b * S + pool_row(smap, b, S, row)) * nkv * hd +
                              (rh - (long)row * nkv) * hd + 8 * c
                        : off;
  const U16x8 x1 = *reinterpret_cast<const U16x8 *>(kc + src);
  const U16x8 x2 = *reinterpret_cast<const U16x8 *>(kc + src + hd / 2);
  if (vr) {
    *reinterpret_cast<U16x8 *>(vr + off) = *reinterpret_cast<const U16x8 *>(vc + src);
    *reinterpret_cast<U16x8 *>(vr + off + hd / 2) = *reinterpret_cast<const U16x8 *>(vc + src + hd / 2);
  }
  const float2 *rp = rope + (long)rope_pos(mr, pos, 8 * c) * (hd / 2) + 8 * c;
  U16x8 y1, y2;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float2 cs = rp[e];
    const float a1 = bf2f(x1.v[e]), a2 = bf2f(x2.v[e]);
    y1.v[e] = bf16_bits(a1 * cs.x - a2 * cs.y);
    y2.v[e] = bf16_bits(a2 * cs.x + a1 * cs.y);
  }
  *reinterpret_cast<U16x8 *>(kr + off) = y1;
  *reinterpret_cast<U16x8 *>(kr + off + hd / 2) = y2;
}

// Merges the split-KV partials of one (32-query tile, head): each split's sum is
// rescaled by 2^(m_s - max m) and the total divided by the rescaled denominators.
// The partials are read in the attention kernel's accumulator order and the bf16
// result is transposed through LDS so that every query row is written contiguously.
constexpr int kMaxAttnSplits = 8;
template <int HD>
__global__ __launch_bounds__(HD * 8) void k_attn_combine(AttnArgs a) {
  constexpr int NG = HD / 8;                       // 16-B groups per lane
  constexpr int NT = NG * 64;                      // one thread per 16-B group
  __shared__ float wt[kMaxAttnSplits][32];
  __shared__ __attribute__((aligned(16))) uint16_t ob[32][HD + 8];
  const int nh = a.nh, tiles = a.tiles;
  const int qt = blockIdx.x / nh, h = blockIdx.x - qt * nh;
  const int tiles_per_b = (a.N + 31) / 32;
  const int b = qt / tiles_per_b, j0 = (qt % tiles_per_b) * 32;
  const int n = n_valid(a.nrec, b, a.N);
  if (j0 >= n) return;
  const int t = threadIdx.x, splits = a.splits;
  // every split's group of this thread in flight at once
  const float4 *po = reinterpret_cast<const float4 *>(a.po);
  float4 p[kMaxAttnSplits];
#pragma unroll
  for (int s = 0; s < kMaxAttnSplits; ++s)
    p[s] = po[(((long)min(s, splits - 1) * tiles + qt) * nh + h) * NT + t];
  if (t < 32) {
    float m[kMaxAttnSplits], l[kMaxAttnSplits];
    float mx = -INFINITY;
#pragma unroll
    for (int s = 0; s < kMaxAttnSplits; ++s) {
      const long blk = ((long)min(s, splits - 1) * tiles + qt) * nh + h;
      m[s] = s < splits ? a.pm[blk * 32 + t] : -INFINITY;
      l[s] = s < splits ? a.pl[blk * 32 + t] : 0.f;
      mx = fmaxf(mx, m[s]);
    }
    const float mu = (mx == -INFINITY) ? 0.f : mx;
    float tot = 0.f;
#pragma unroll
    for (int s = 0; s < kMaxAttnSplits; ++s) {
      m[s] = s < splits ? exp2f(m[s] - mu) : 0.f;
      tot += l[s] * m[s];
    }
    const float inv = tot > 0.f ? 1.f / tot : 0.f;
#pragma unroll
    for (int s = 0; s < kMaxAttnSplits; ++s) wt[s][t] = m[s] * inv;
  }
  __syncthreads();
  {
    const int grp = t >> 6, lane = t & 63, q = lane & 31, hi = lane >> 5;
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int s = 0; s < kMaxAttnSplits; ++s) {
      const float ws = wt[s][q];   // zero for s >= splits
      v.x += p[s].x * ws; v.y += p[s].y * ws; v.z += p[s].z * ws; v.w += p[s].w * ws;
    }
    // group grp = hb * 4 + eg holds dims hb * 32 + eg * 8 + hi * 4 + 0..3
    const int d = (grp >> 2) * 32 + (grp & 3) * 8 + hi * 4;
    ushort4 r;
    r.x = f2bf(v.x); r.y = f2bf(v.y); r.z = f2bf(v.z); r.w = f2bf(v.w);
    *reinterpret_cast<ushort4 *>(&ob[q][d]) = r;
  }
  __syncthreads();
  if (t < 32 * (HD / 8)) {
    const int q = t / (HD / 8), x = t - q * (HD / 8);
    if (j0 + q < n)
      *reinterpret_cast<uint4 *>(a.out + ((long)b * a.N + j0 + q) * (long)(nh * HD) + h * HD + 8 * x) =
          *reinterpret_cast<const uint4 *>(&ob[q][8 * x]);
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
  int kv_copy;                   // 0: K/V rows are not moved (slot-mapped caches)
  int y_copy;                    // 0: output rows are not moved
};

// Chunks of 16 B the remap moves per reused token.
__host__ __device__ inline int cache_chunks(const CacheArgs &c) {
  return (c.kv_copy ? 2 * (c.kvw / 8) : 0) + (c.y_copy ? c.d / 8 : 0);
}

// One thread per 16-B chunk of a reused token's K row, V row and output row, so that
// every copy of the remap is in flight at once.
__device__ __forceinline__ void cache_copy(const CacheArgs &c) {
  const int b = blockIdx.y;
  const int kc = c.kv_copy ? c.kvw / 8 : 0, cpt = cache_chunks(c);   // chunks per token
  const long e = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const int tok = (int)(e / cpt);
  if (tok >= c.N) return;
  if (!c.reuse[(long)b * c.N + tok]) return;
  const int q = (int)(e - (long)tok * cpt);
  const int I = tok / c.gw, J = tok - I * c.gw;
  const int si = I + c.shift[b * 2], sj = J + c.shift[b * 2 + 1];
  if (si < 0 || si >= c.gh || sj < 0 || sj >= c.gw) return;  // never for a valid mask
  const int src = si * c.gw + sj;
  if (q < 2 * kc) {
    const long drow = (long)b * c.S + c.cur_row0 + tok;
    const long srow = (long)b * c.src_bstride / c.kvw + c.src_row0 + src;
    const bool isk = q < kc;
    const uint4 *s4 = reinterpret_cast<const uint4 *>((isk ? c.ksrc : c.vsrc) + srow * c.kvw);
    uint4 *d4 = reinterpret_cast<uint4 *>((isk ? c.kc : c.vc) + drow * c.kvw);
    const int x = isk ? q : q - kc;
    d4[x] = s4[x];
  } else {
    const int x = q - 2 * kc;
    const uint4 *ys = reinterpret_cast<const uint4 *>(c.y_prev + ((long)b * c.N + src) * c.d);
    uint4 *yd = reinterpret_cast<uint4 *>(c.y_cur + ((long)b * c.N + tok) * c.d);
    yd[x] = ys[x];
  }
}

__global__ __launch_bounds__(256) void k_cache_update(CacheArgs c) { cache_copy(c); }

// The remap of up to kCacheLayers layers' caches in one launch (blockIdx.z = layer);
// each layer's rows move exactly as in k_cache_update.
constexpr int kCacheLayers = 32;
struct CacheLayers {
  CacheArgs c;                                   // shared sizes; pointers of layer 0
  uint16_t *kc[kCacheLayers], *vc[kCacheLayers];
  const uint16_t *yp[kCacheLayers];
  uint16_t *yc[kCacheLayers];
};
__global__ __launch_bounds__(256) void k_cache_update_layers(CacheLayers m) {
  CacheArgs c = m.c;
  const int l = blockIdx.z;
  c.kc = m.kc[l];
  c.vc = m.vc[l];
  c.ksrc = m.kc[l];
  c.vsrc = m.vc[l];
  c.y_prev = m.yp[l];
  c.y_cur = m.yc[l];
  cache_copy(c);
}

// Column groups and K splits of a weight-streaming GEMM: columns in 16-wide blocks,
// at most NBLK blocks per group, and enough (group, split) pairs to cover the CUs
// about once; every split keeps at least 4 K steps and the partial sums fit.
template <int MODE>
fc_status run_wgemm(fc_ctx *ctx, hipStream_t st, const char *name, WArgs &g, int B) {
  if (g.K % KS || g.Nout % 16)
    return fail(FC_ERR_SHAPE, "%s: K %d must be a multiple of %d and N %d of 16", name, g.K, KS, g.Nout);
  const int cus = std::max(ctx->num_cus, 1);
  const int nblk = WTraits<MODE>::NBLK;
  g.nb = g.Nout / 16;
  g.tpb = (g.N + MT - 1) / MT;
  const int ksteps = g.K / KS;
  int splits = 1;
  if (MODE == G_GU) {
    g.ncg = std::max((g.nb + nblk - 1) / nblk, std::min(cus, g.nb));
  } else {
    g.ncg = (g.nb + nblk - 1) / nblk;
    splits = std::max(1, std::min(kMaxSplits, cus / g.ncg));
    splits = std::min(splits, std::max(1, ksteps / 4));
    while (splits > 1 && (size_t)splits * g.rows * g.Nout > ctx->part_elems) --splits;
  }
  if (MODE == G_QKV && (ksteps + splits - 1) / splits > kGainSteps) {
    // the gain slice of a split's K range must fit in LDS
    splits = (ksteps + kGainSteps - 1) / kGainSteps;
    if (splits > kMaxSplits || (size_t)splits * g.rows * g.Nout > ctx->part_elems)
      return fail(FC_ERR_UNSUPPORTED, "%s: K %d needs more than %d splits", name, g.K, kMaxSplits);
  }
  g.ksteps = (ksteps + splits - 1) / splits;
  g.splits = (ksteps + g.ksteps - 1) / g.ksteps;
  if (MODE != G_GU && (size_t)g.splits * g.rows * g.Nout > ctx->part_elems)
    return fail(FC_ERR_CAPACITY, "%s: partial sums exceed the workspace", name);
  const long total = (long)B * g.tpb * g.ncg * g.splits;
  ProfScope ps(ctx, st, name);
  hipLaunchKernelGGL(k_wgemm<MODE>, dim3((unsigned)total), dim3(512), 0, st, g);
  FC_LAUNCH_OK(st, "k_wgemm");
  return FC_OK;
}

// rot: keys rotated on load (32-query tiles, four staging waves); otherwise keys come
// rotated and, with one key split, each query wave takes two 32-query blocks (one
// staging wave), so a staged key block feeds twice the MFMAs
template <int HD, int G>
void launch_attn(hipStream_t st, AttnArgs a, bool rot, int nkv) {
  if (rot) {
    hipLaunchKernelGGL((k_attn<HD, G, true, 1, kAttnStageWaves>), dim3(a.tiles * nkv * a.splits),
                       dim3((G + kAttnStageWaves) * 64), 0, st, a);
  } else if (a.splits > 1) {
    hipLaunchKernelGGL((k_attn<HD, G, false, 1, kAttnStageWaves>), dim3(a.tiles * nkv * a.splits),
                       dim3((G + kAttnStageWaves) * 64), 0, st, a);
  } else {
    const int tiles_per_b = (a.N + 63) / 64;
    a.tiles = (a.tiles / ((a.N + 31) / 32)) * tiles_per_b;      // B * tiles of 64 queries
    hipLaunchKernelGGL((k_attn<HD, G, false, 2, 1>), dim3(a.tiles * nkv), dim3((G + 1) * 64), 0,
                       st, a);
  }
}

// Tiles of the large-M GEMM: 256 packed rows, 256 output columns (SwiGLU: 128 output
// columns, staged as gate and up rows); tiles past the packed rows exit.
template <int MODE>
fc_status run_mgemm(fc_ctx *ctx, hipStream_t st, const char *name, MArgs &g, int B) {
  if (g.K % KS || g.Nout % 16)
    return fail(FC_ERR_SHAPE, "%s: K %d must be a multiple of %d and N %d of 16", name, g.K, KS, g.Nout);
  if (B > kMMaxItems) return fail(FC_ERR_CAPACITY, "%s: more than %d batch items", name, kMMaxItems);
  g.B = B;
  g.mtiles = (int)(((long)B * g.N + MB - 1) / MB);      // packed rows need at most these
  const int tn = MODE == G_GU ? MB / 2 : MB;
  g.ntn = (g.Nout + tn - 1) / tn;
  g.cus = std::max(ctx->num_cus, 1);
  if (!g.part) {
    g.part = ctx->part;
    g.part_units = (int)std::min<size_t>(ctx->part_elems / ((size_t)MB * MB), 1 << 20);
  }
  // whole tiles plus the extra parts of a split tail (fewer than one round)
  const long total = (long)g.mtiles * g.ntn + g.cus;
  if (total > INT32_MAX) return fail(FC_ERR_CAPACITY, "%s: too many tiles", name);
  ProfScope ps(ctx, st, name);
  hipLaunchKernelGGL(k_mgemm<MODE>, dim3((unsigned)total), dim3(512), 0, st, g);
  FC_LAUNCH_OK(st, "k_mgemm");
  // a split tail has at most cus / 2 tiles, 4 workgroups each
  hipLaunchKernelGGL(k_mtail<MODE>, dim3((unsigned)(2 * g.cus)), dim3(512), 0, st, g);
  FC_LAUNCH_OK(st, "k_mtail");
  return FC_OK;
}

}  // namespace

namespace {
template <int SPL>
void launch_red(int which, dim3 grid, hipStream_t st, const RedArgs &r) {
  if (which == 0) hipLaunchKernelGGL(k_red_qkv<SPL>, grid, dim3(256), 0, st, r);
  else if (which == 1) hipLaunchKernelGGL(k_red_o<SPL>, grid, dim3(256), 0, st, r);
  else hipLaunchKernelGGL(k_red_down<SPL>, grid, dim3(256), 0, st, r);
}
// which: 0 QKV, 1 O, 2 down
void run_red(int which, dim3 grid, hipStream_t st, const RedArgs &r) {
  if (r.splits <= 1) launch_red<1>(which, grid, st, r);
  else if (r.splits <= 2) launch_red<2>(which, grid, st, r);
  else if (r.splits <= 4) launch_red<4>(which, grid, st, r);
  else if (r.splits <= 8) launch_red<8>(which, grid, st, r);
  else launch_red<16>(which, grid, st, r);
}
}  // namespace

fc_status launch_layer(fc_ctx *ctx, const fc_layer_desc &L, const fc_kv_cache &kv,
                       const uint16_t *x_cur, const int32_t *idx, const int32_t *nrec,
                       uint16_t *y_cur, int B, hipStream_t st, bool trail) {
  // The rows a call recomputes form its region: the current frame's recomputed tokens
  // (ids and counts from the selection), or every text token after the frames (trail:
  // null ids and counts, the region's tokens in order).  N below is the region's token
  // count; FN the frame's.
  const int FN = kv.frame_tokens, d = L.d_model, nh = L.n_heads, nkv = L.n_kv_heads,
            hd = L.head_dim, ffn = L.d_ffn;
  const int frames_end = kv.text_tokens + kv.window * FN;
  const int S = frames_end + kv.trail_tokens;
  const int N = trail ? kv.trail_tokens : FN;
  const int qkv = (nh + 2 * nkv) * hd;
  const long rows = (long)B * N;
  const int cur_slot = (kv.head + kv.window - 1) % kv.window;
  const int cur_row0 = trail ? frames_end : kv.text_tokens + cur_slot * FN;
  const int qpos0 = trail ? frames_end : kv.text_tokens + (kv.window - 1) * FN;
  if (trail) idx = nrec = nullptr;
  const int want = std::max(ctx->num_cus, 1);
  // thousands of gathered rows (several batch items of large frames) make the
  // projections compute bound: square MFMA tiles with fused epilogues instead of the
  // weight-streaming kernels and their split-K reductions
  const bool big = !trail && rows >= kBigRows && (hd == 64 || hd == 128) && B <= kMMaxItems;

  // RoPE table for (hd, theta) over the cache length (rebuilt only when they change)
  if (ctx->rope_hd != hd || ctx->rope_theta != L.rope_theta || ctx->rope_seq < S) {
    const int seq = ctx->caps.max_seq;
    const long n = (long)seq * (hd / 2);
    ProfScope ps(ctx, st, "fc_rope_table");
    hipLaunchKernelGGL(k_rope_table, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st,
                       ctx->rope, seq, hd / 2, hd, L.rope_theta);
    FC_LAUNCH_OK(st, "k_rope_table");
    ctx->rope_hd = hd;
    ctx->rope_theta = L.rope_theta;
    ctx->rope_seq = seq;
  }

  RedArgs r{};
  r.N = N; r.d = d; r.S = S; r.cur_row0 = cur_row0; r.rows = rows; r.eps = L.rms_eps;
  r.idx = idx; r.nrec = nrec; r.part = ctx->part; r.x = x_cur;
  r.qw = nh * hd; r.kw = nkv * hd;
  r.hd = hd; r.qpos0 = qpos0; r.rope = ctx->rope;
  MRope mr{};
  if (kv.mrope_section[0] + kv.mrope_section[1] + kv.mrope_section[2] > 0) {
    const int gh = FN / kv.grid_w;
    mr = MRope{1, kv.text_tokens, FN, kv.window, kv.grid_w, std::max(gh, kv.grid_w),
               kv.mrope_section[0], kv.mrope_section[0] + kv.mrope_section[1]};
  }
  r.mr = mr;
  fc_status rc;

  // 1. QKV of the recomputed rows.  Large-M path: gather + RMSNorm of the rows, then a
  //    GEMM whose epilogue adds the bias, rotates q and scatters raw k, v into the
  //    current frame's cache rows.  Few-row path: the GEMM gathers the rows of x by
  //    token id itself and multiplies x g; the reduction scales by 1/rms, adds the bias,
  //    stores rotated q and scatters raw k, v
  {
    r.ncols = qkv;
    r.bias = L.b_qkv; r.q = ctx->qbuf; r.kc = kv.k; r.vc = kv.v; r.smap = kv.slot_map;
    if (big) {
      {
        ProfScope ps(ctx, st, "fc_gather_norm");
        hipLaunchKernelGGL(k_gather_norm, dim3((unsigned)rows), dim3(256), 0, st, x_cur, L.g_attn,
                           idx, nrec, N, d, L.rms_eps, ctx->hb);
        FC_LAUNCH_OK(st, "k_gather_norm");
      }
      MArgs g{};
      g.A = ctx->hb; g.W0 = L.w_qkv;
      g.K = d; g.Nout = qkv; g.N = N; g.r = r;
      if ((rc = run_mgemm<G_QKV>(ctx, st, "fc_mgemm_qkv", g, B)) != FC_OK) return rc;
    } else {
      WArgs g{};
      g.A = x_cur; g.gather = 1; g.gain = L.g_attn; g.W0 = L.w_qkv;
      g.K = d; g.Nout = qkv; g.N = N; g.idx = idx; g.nrec = nrec;
      g.part = ctx->part; g.rows = rows; g.eps = L.rms_eps;
      if ((rc = run_wgemm<G_QKV>(ctx, st, "fc_gemm_qkv", g, B)) != FC_OK) return rc;
      r.splits = g.splits;
      ProfScope ps(ctx, st, "fc_red_qkv");
      run_red(0, dim3((unsigned)rows, (qkv + 1023) / 1024), st, r);
      FC_LAUNCH_OK(st, "k_red_qkv");
    }
  }

  // 2. attention over the whole cache
  {
    AttnArgs a{};
    a.q = ctx->qbuf;
    a.kc = kv.k; a.vc = kv.v; a.smap = kv.slot_map;
    a.rope = ctx->rope;
    a.mr = mr;
    a.idx = idx; a.nrec = nrec;
    a.N = N; a.nh = nh; a.nkv = nkv; a.S = S;
    a.T = kv.text_tokens; a.W = kv.window; a.head = kv.head;
    a.fN = FN; a.cur_lo = cur_row0; a.qpos0 = qpos0; a.frames_end = frames_end;
    a.scale_log2 = (float)(1.0 / std::sqrt((double)hd) * 1.4426950408889634);
    a.out = ctx->attn;
    const int tiles = B * ((N + 31) / 32);
    const int nkb = (S + 31) / 32;
    int splits = std::max(1, std::min(kMaxAttnSplits, (2 * want) / (tiles * nkv)));
    splits = std::min(splits, std::max(1, nkb / 4));
    const size_t prow = (size_t)tiles * 32;           // query rows padded to whole tiles
    // with many query tiles per item, every cached key is rotated once into a copy
    // instead of once per (key, tile) inside the attention kernel
    const long kvw = (long)nkv * hd;
    const bool prerot = big && ctx->krot && (size_t)B * S * kvw <= ctx->krot_elems;
    // a slot map read by the attention kernel itself: at most kAttnMapRows rows per split
    const bool map_in_attn = kv.slot_map && !prerot;
    const int min_splits = map_in_attn ? (nkb * 32 + kAttnMapRows - 1) / kAttnMapRows : 1;
    splits = std::max(splits, min_splits);
    while (splits > min_splits && (size_t)splits * prow * nh * (hd + 2) > ctx->part_elems) --splits;
    if (splits > kMaxAttnSplits || (splits > 1 && (size_t)splits * prow * nh * (hd + 2) > ctx->part_elems))
      return fail(FC_ERR_UNSUPPORTED, "attention: a slot-mapped cache of %d rows needs %d key "
                  "splits, more than the workspace holds", S, splits);
    a.kb_per_split = (nkb + splits - 1) / splits;
    a.splits = (nkb + a.kb_per_split - 1) / a.kb_per_split;
    a.po = ctx->part;
    a.pm = ctx->part + (size_t)a.splits * prow * nh * hd;
    a.pl = a.pm + (size_t)a.splits * prow * nh;
    const int G = nh / nkv;
    a.tiles = tiles;
    if (prerot) {
      // slot-mapped: the values are gathered into row order beside the rotated keys
      uint16_t *vr = nullptr;
      if (kv.slot_map) {
        if (!ctx->vlog) {
          hipError_t e = hipMalloc(reinterpret_cast<void **>(&ctx->vlog),
                                   ctx->krot_elems * sizeof(uint16_t));
          if (e != hipSuccess) {
            ctx->vlog = nullptr;
            return fail(FC_ERR_HIP, "hipMalloc(slot-mapped values, %zu bytes): %s",
                        ctx->krot_elems * sizeof(uint16_t), hipGetErrorString(e));
          }
          ctx->vlog_elems = ctx->krot_elems;
        }
        vr = ctx->vlog;
      }
      ProfScope ps(ctx, st, "fc_rot_keys");
      const long tasks = (long)S * nkv * (hd / 16);
      hipLaunchKernelGGL(k_rot_keys, dim3((unsigned)((tasks + 255) / 256), B), dim3(256), 0, st,
                         kv.k, ctx->rope, ctx->krot, S, nkv, hd, kv.text_tokens, FN, kv.window,
                         kv.head, mr, kv.slot_map, kv.v, vr);
      FC_LAUNCH_OK(st, "k_rot_keys");
      a.kc = ctx->krot;
      if (vr) {
        a.vc = vr;
        a.smap = nullptr;
      }
    }
    {
      ProfScope ps(ctx, st, "fc_attn");
      if (hd == 128 && G == 7)
        launch_attn<128, 7>(st, a, !prerot, nkv);
      else if (hd == 128 && G == 1)
        launch_attn<128, 1>(st, a, !prerot, nkv);
      else if (hd == 64 && G == 1)
        launch_attn<64, 1>(st, a, !prerot, nkv);
      else if (hd == 64 && G == 2)
        launch_attn<64, 2>(st, a, !prerot, nkv);
      else if (hd == 128 && G == 4)
        launch_attn<128, 4>(st, a, !prerot, nkv);
      else
        return fail(FC_ERR_UNSUPPORTED, "attention: head_dim %d with %d query heads per kv head", hd, G);
      FC_LAUNCH_OK(st, "k_attn");
    }
    if (a.splits > 1) {
      ProfScope ps(ctx, st, "fc_attn_combine");
      if (hd == 128)
        hipLaunchKernelGGL(k_attn_combine<128>, dim3((unsigned)(tiles * nh)), dim3(1024), 0, st, a);
      else
        hipLaunchKernelGGL(k_attn_combine<64>, dim3((unsigned)(tiles * nh)), dim3(512), 0, st, a);
      FC_LAUNCH_OK(st, "k_attn_combine");
    }
  }

  // 3. O projection; reduction adds the residual -> h1 (float32) and its bf16 copy
  r.ncols = d; r.h1 = ctx->h1; r.hb = ctx->hb; r.ssq = ctx->ssq; r.gain = L.g_mlp; r.y = y_cur;
  // sums of squares of h1 per row: per 1024 columns from the O reduction, per 256
  // columns from the large-M epilogue
  const int ss_parts = big ? (d + kMSsqCols - 1) / kMSsqCols : (d + 1023) / 1024;
  if (big) {
    MArgs g{};
    g.A = ctx->attn; g.W0 = L.w_o;
    g.K = nh * hd; g.Nout = d; g.N = N; g.ss_parts = ss_parts; g.r = r;
    if ((rc = run_mgemm<G_O>(ctx, st, "fc_mgemm_o", g, B)) != FC_OK) return rc;
  } else {
    WArgs g{};
    g.A = ctx->attn; g.W0 = L.w_o;
    g.K = nh * hd; g.Nout = d; g.N = N; g.idx = idx; g.nrec = nrec;
    g.part = ctx->part; g.rows = rows;
    if ((rc = run_wgemm<G_O>(ctx, st, "fc_gemm_o", g, B)) != FC_OK) return rc;
    r.splits = g.splits;
    ProfScope ps(ctx, st, "fc_red_o");
    run_red(1, dim3((unsigned)rows, (d + 1023) / 1024), st, r);
    FC_LAUNCH_OK(st, "k_red_o");
  }

  // 4. gate/up on bf16(h1 * g_mlp); 1/rms from the sums of squares is applied to both
  //    sums, then SiLU(g) * u -> act (bf16)
  if (big) {
    MArgs g{};
    g.A = ctx->hb; g.W0 = L.w_gate; g.W1 = L.w_up;
    g.K = d; g.Nout = ffn; g.N = N; g.ss_parts = ss_parts; g.act = ctx->act; g.r = r;
    if ((rc = run_mgemm<G_GU>(ctx, st, "fc_mgemm_gateup", g, B)) != FC_OK) return rc;
  } else {
    WArgs g{};
    g.A = ctx->hb; g.W0 = L.w_gate; g.W1 = L.w_up;
    g.K = d; g.Nout = ffn; g.N = N; g.idx = idx; g.nrec = nrec;
    g.rows = rows; g.act = ctx->act; g.eps = L.rms_eps;
    g.ssq = ctx->ssq; g.ss_parts = ss_parts;
    if ((rc = run_wgemm<G_GU>(ctx, st, "fc_gemm_gateup", g, B)) != FC_OK) return rc;
  }

  // 5. down projection; adds h1 and scatters bf16 rows into the output cache
  if (big) {
    MArgs g{};
    g.A = ctx->act; g.W0 = L.w_down;
    g.K = ffn; g.Nout = d; g.N = N; g.r = r;
    if ((rc = run_mgemm<G_DOWN>(ctx, st, "fc_mgemm_down", g, B)) != FC_OK) return rc;
  } else {
    WArgs g{};
    g.A = ctx->act; g.W0 = L.w_down;
    g.K = ffn; g.Nout = d; g.N = N; g.idx = idx; g.nrec = nrec;
    g.part = ctx->part; g.rows = rows;
    if ((rc = run_wgemm<G_DOWN>(ctx, st, "fc_gemm_down", g, B)) != FC_OK) return rc;
    r.splits = g.splits;
    ProfScope ps(ctx, st, "fc_red_down");
    run_red(2, dim3((unsigned)rows, (d + 1023) / 1024), st, r);
    FC_LAUNCH_OK(st, "k_red_down");
  }
  return FC_OK;
}

fc_status run_plain_gemm(fc_ctx *ctx, hipStream_t st, const char *name, const uint16_t *A,
                         const uint16_t *W, int K, int Nout, int N, const int32_t *nrec,
                         float *part, int B, int *splits, int *dsplits, const int **dsplits_used,
                         int *tiles) {
  *dsplits_used = nullptr;
  // many rows: the 256 x 256-tile GEMM, each tile as up to 8 K-range parts whose sums go
  // to part as 256 x 256 tiles over the packed rows; the part count is decided on the
  // device (it depends on the row counts there) and written to *dsplits for the consumer
  const long mtiles = ((long)B * N + MB - 1) / MB, ntn = (Nout + MB - 1) / MB;
  const int cus = std::max(ctx->num_cus, 1);
  // the most tiles any row count can store: V ntn ks(V) over V <= mtiles
  long most = 0;
  for (long V = 1; V <= mtiles && V * ntn <= INT32_MAX; ++V)
    most = std::max(most, V * ntn * plain_split((int)(V * ntn), cus, K / KS));
  *tiles = 0;
  if (dsplits && (long)B * N >= kPlainBigRows && B <= kMMaxItems && K % KS == 0 &&
      Nout % 16 == 0 && most > 0 && (size_t)most * MB * MB <= ctx->part_elems) {
    MArgs m{};
    m.A = A; m.W0 = W;
    m.K = K; m.Nout = Nout; m.N = N; m.B = B;
    m.r.nrec = nrec;
    m.out = part;
    m.ks_out = dsplits;
    m.mtiles = (int)(((long)B * N + MB - 1) / MB);
    m.ntn = (Nout + MB - 1) / MB;
    m.cus = cus;
    const long total = (long)m.mtiles * m.ntn * kPlainMaxParts;
    if (total > INT32_MAX) return fail(FC_ERR_CAPACITY, "%s: too many tiles", name);
    ProfScope ps(ctx, st, name);
    hipLaunchKernelGGL(k_mgemm<G_PLAIN>, dim3((unsigned)total), dim3(512), 0, st, m);
    FC_LAUNCH_OK(st, "k_mgemm");
    *splits = kPlainMaxParts;
    *dsplits_used = dsplits;
    *tiles = 1;
    return FC_OK;
  }
  WArgs g{};
  g.A = A; g.W0 = W;
  g.K = K; g.Nout = Nout; g.N = N; g.nrec = nrec;
  g.part = part; g.rows = (long)B * N;
  fc_status rc = run_wgemm<G_O>(ctx, st, name, g, B);
  *splits = g.splits;
  return rc;
}

fc_status launch_cache_update(fc_ctx *ctx, const fc_layer_desc &L, const fc_kv_cache &kv,
                              const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                              const uint8_t *reuse, int grid_w, int B, hipStream_t st) {
  const int N = kv.frame_tokens;
  const int S = kv.text_tokens + kv.window * N + kv.trail_tokens;
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
  c.kv_copy = 1;
  c.y_copy = y_prev != nullptr;
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
      FC_LAUNCH_OK(st, "k_copy16");
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
  const long chunks = (long)N * cache_chunks(c);
  hipLaunchKernelGGL(k_cache_update, dim3((unsigned)((chunks + 255) / 256), B), dim3(256), 0, st, c);
  FC_LAUNCH_OK(st, "k_cache_update");
  return FC_OK;
}

fc_status launch_remap_copy(fc_ctx *ctx, const uint16_t *ksrc, const uint16_t *vsrc, uint16_t *kdst,
                            uint16_t *vdst, const uint16_t *y_prev, uint16_t *y_cur, int N, int kvw,
                            int d, int grid_w, const int32_t *shift, const uint8_t *reuse, int B,
                            hipStream_t st) {
  CacheArgs c{};
  c.kc = kdst;
  c.vc = vdst;
  c.ksrc = ksrc;
  c.vsrc = vsrc;
  c.src_bstride = (long)N * kvw;
  c.src_row0 = 0;
  c.y_prev = y_prev;
  c.y_cur = y_cur;
  c.shift = shift;
  c.reuse = reuse;
  c.N = N;
  c.S = N;
  c.kvw = kvw;
  c.d = d;
  c.gw = grid_w;
  c.gh = N / grid_w;
  c.cur_row0 = 0;
  c.kv_copy = 1;
  c.y_copy = y_prev != nullptr;
  ProfScope ps(ctx, st, "fc_cache_update");
  const long chunks = (long)N * cache_chunks(c);
  hipLaunchKernelGGL(k_cache_update, dim3((unsigned)((chunks + 255) / 256), B), dim3(256), 0, st, c);
  FC_LAUNCH_OK(st, "k_cache_update");
  return FC_OK;
}

fc_status launch_cache_update_layers(fc_ctx *ctx, const fc_layer_desc &L, int n_layers,
                                     const fc_kv_cache *kvs, const uint16_t *const *y_prev,
                                     uint16_t *const *y_cur, const int32_t *shift,
                                     const uint8_t *reuse, int grid_w, int B, hipStream_t st) {
  const fc_kv_cache &kv = kvs[0];
  const bool ycopy = y_prev != nullptr;
  if (kv.slot_map) {
    // one map for all layers: the reused rows are shared, no K/V byte moves
    fc_status s = launch_slot_remap(ctx, kv, shift, reuse, grid_w, B, st);
    if (s != FC_OK || !ycopy) return s;
  } else if (kv.window == 1) {
    // in-place overwrite of the only frame slot: the per-layer path stages the old rows
    for (int l = 0; l < n_layers; ++l) {
      fc_status s = launch_cache_update(ctx, L, kvs[l], ycopy ? y_prev[l] : nullptr,
                                        ycopy ? y_cur[l] : nullptr, shift, reuse, grid_w, B, st);
      if (s != FC_OK) return s;
    }
    return FC_OK;
  }
  const int N = kv.frame_tokens;
  const int S = kv.text_tokens + kv.window * N + kv.trail_tokens;
  const int kvw = L.n_kv_heads * L.head_dim;
  const int cur_slot = (kv.head + kv.window - 1) % kv.window;
  const int prev_slot = (kv.head + kv.window - 2) % kv.window;
  CacheLayers m{};
  CacheArgs &c = m.c;
  c.shift = shift;
  c.reuse = reuse;
  c.N = N;
  c.S = S;
  c.kvw = kvw;
  c.d = L.d_model;
  c.gw = grid_w;
  c.gh = N / grid_w;
  c.cur_row0 = kv.text_tokens + cur_slot * N;
  c.src_bstride = (long)S * kvw;
  c.src_row0 = kv.text_tokens + prev_slot * N;
  c.kv_copy = kv.slot_map == nullptr;
  c.y_copy = ycopy;
  ProfScope ps(ctx, st, "fc_cache_update");
  const long chunks = (long)N * cache_chunks(c);
  for (int l0 = 0; l0 < n_layers; l0 += kCacheLayers) {
    const int nl = std::min(kCacheLayers, n_layers - l0);
    for (int i = 0; i < nl; ++i) {
      m.kc[i] = kvs[l0 + i].k;
      m.vc[i] = kvs[l0 + i].v;
      m.yp[i] = ycopy ? y_prev[l0 + i] : nullptr;
      m.yc[i] = ycopy ? y_cur[l0 + i] : nullptr;
    }
    hipLaunchKernelGGL(k_cache_update_layers, dim3((unsigned)((chunks + 255) / 256), B, nl),
                       dim3(256), 0, st, m);
    FC_LAUNCH_OK(st, "k_cache_update_layers");
  }
  return FC_OK;
}

}  // namespace fc
