// Frequency-guided cacheable-token selection on gfx950 (FreqCache Sec. 4.1-4.4,
// Algorithm 1).  Four kernels:
//
//   k_spectra  one workgroup per strip of up to 16 patches (14 rows x 224 px) of
//              one frame.  Coalesced float4 loads of R, G, B rows, float64 luma
//              staged in LDS, then per patch: the 14x14 DFT amplitude (Eq. 3-2)
//              with real/even folding in float32, the patch mean, and for the
//              current frame the orthonormal DCT-II high-pass energy (Eqs. 3-4,
//              3-5) in float64, as the patch energy minus that of the removed
//              3 x 3 low block (the transform is orthonormal).
//   k_grid     one workgroup per frame pair: token-grid mean-luma maps, their
//              2-D DFTs (float64), global amplitude similarity (Eq. 3-3) and the
//              migration gate, spectral entropy and the reuse budget (Eqs. 3-6,
//              4-4), phase correlation and its peak (Eq. 4-1), token energies and
//              their mean / std / refresh threshold (Eq. 4-3).
//   k_patchsim per patch: the products of its amplitude spectrum with that of the
//              same patch of its token's aligned source token (Eqs. 3-3, 4-2).
//   k_topk     one workgroup per frame pair: alignment mask and token similarity,
//              refresh mask, candidate set, ascending-energy top-K with ties to the
//              lower id (radix select of the energy bits), reuse mask and
//              ballot/prefix-sum compaction of the recomputed ids.
//
// The transforms are direct (no FFT library): a 14-point DFT folded on its
// even/odd symmetry costs 84 real FMAs per row and 168 per complex column, and
// the work is bound by reading the frames from HBM anyway.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "fc_internal.h"

namespace fc {
namespace {

constexpr int P = kPatch;      // 14
constexpr int PW = 16;         // patches per k_spectra workgroup
constexpr int NB = kBins;      // 100 unique amplitude bins

__constant__ float c_cos14[P];       // cos(2 pi j / 14)
__constant__ float c_sin14[P];       // sin(2 pi j / 14)
__constant__ double c_dct14[P * P];  // orthonormal DCT-II, C[k][x]

// Unique-bin index of amplitude A(u, v) for v in 0..7 (see the layout note in
// k_spectra); returns -1 for a duplicate bin.
__device__ __forceinline__ int bin_of(int u, int v) {
  if (v == 0) return u <= 7 ? u : -1;
  if (v == 7) return u <= 7 ? 8 + u : -1;
  return 16 + (v - 1) * P + u;
}

// Multiplicity of a unique bin in the full 196-bin spectrum.
__device__ __forceinline__ double bin_weight(int bin) {
  return (bin == 0 || bin == 7 || bin == 8 || bin == 15) ? 1.0 : 2.0;
}

// Amplitudes of a frame batch are stored per 16-patch chunk of a patch row,
// [b][chunk][bin][16], chunk = pi * ncx + pj / 16 with ncx = ceil(Gpw / 16): one
// k_spectra workgroup writes its whole 6.4 KB block with full-line stores (a bin-major
// layout cost it 64-B pieces).  The previous and the current frames have separate
// buffers, so the current frame's spectra can be carried to the next step.
__device__ __forceinline__ size_t amp_chunk(int b, int pi, int cx, int Gph, int ncx) {
  return ((size_t)b * Gph * ncx + (size_t)pi * ncx + cx) * NB * 16;
}

// ------------------------------------------------------------------------------- k_spectra
// Grid: x = 16-patch chunk of a patch row, y = patch row, z = item and frame: z = 2 b + f
// (f = 0 prev, 1 cur), or z = b for the current frame only (nf = 1, the previous
// frame's spectra carried).  Outputs per frame f:
//   amp_f[amp_chunk(b, pi, chunk) + bin * 16 + slot]  float32 amplitude, unique bins:
//       bins 0..7   = (u = 0..7,  v = 0),  bins 8..15 = (u = 0..7, v = 7),
//       bins 16..99 = (u = 0..13, v = 1..6)   (the rest follow from A(u,v) = A(-u,-v));
//   pmean_f[b * Np + patch]       float64 mean luma;
//   penergy[b * Np + patch]       float64 high-pass DCT energy (current frame only).
__global__ __launch_bounds__(256) void k_spectra(const float *__restrict__ prev,
                                                 const float *__restrict__ cur, int H, int W,
                                                 int Gph, int Gpw, int nf, FrameSpectra sp_prev,
                                                 FrameSpectra sp_cur,
                                                 double *__restrict__ penergy) {
  const int f = nf == 1 ? 1 : (int)(blockIdx.z & 1);
  const int b = nf == 1 ? (int)blockIdx.z : (int)(blockIdx.z >> 1);
  const int pi = blockIdx.y;
  const int j0 = blockIdx.x * PW;
  const int pw = min(PW, Gpw - j0);
  const int Np = Gph * Gpw;
  const int t = threadIdx.x;
  const float *frame = f ? cur : prev;
  float *__restrict__ amp = f ? sp_cur.amp : sp_prev.amp;
  double *__restrict__ pmean = f ? sp_cur.pmean : sp_prev.pmean;

  const int ncx = (Gpw + PW - 1) / PW;
  float4 *ablk = reinterpret_cast<float4 *>(amp + amp_chunk(b, pi, blockIdx.x, Gph, ncx));
  if (frame == nullptr) {  // no previous frame: an all-zero frame
    for (int e = t; e < NB * PW / 4; e += blockDim.x) ablk[e] = make_float4(0.f, 0.f, 0.f, 0.f);
    if (t < pw) pmean[(size_t)b * Np + pi * Gpw + j0 + t] = 0.0;
    return;
  }

  // LDS: the luma tile, then (after every row has been read into registers) the
  // row-stage results in the same space.  The luma tile is [patch][row][15] doubles:
  // the row-stage thread of (patch, row) is thread 14 patch + row, so a 15-double
  // row pitch puts the 32 lanes of a half-wave on 64 distinct banks.  The row DFTs
  // have a 120-float2 patch pitch for the same reason in the column stage.
  constexpr int YP = P + 1;                 // luma row pitch (doubles)
  constexpr int RP = 120;                   // row-DFT patch pitch (float2), 112 used
  struct RowStage {
    float2 row[PW][RP];        // row DFTs [patch][row * 8 + v], v = 0..7
    double r3[PW][3][P];       // row DCTs, k < 3
    double ss[PW][P];          // per-row sums of squares of the luma
    double rs[PW][P];          // per-row luma sums
    double col[PW][3];         // low-block energies: sum over u < 3 of D(u, k)^2
  };
  constexpr int kTileBytes = PW * P * YP * (int)sizeof(double);
  constexpr int kLdsBytes = kTileBytes > (int)sizeof(RowStage) ? kTileBytes : (int)sizeof(RowStage);
  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  double *sY = reinterpret_cast<double *>(lds);
  RowStage &rsg = *reinterpret_cast<RowStage *>(lds);
  float2(*sRow)[RP] = rsg.row;
  double(*sR)[3][P] = rsg.r3;
  double(*sSs)[P] = rsg.ss;
  double(*sRs)[P] = rsg.rs;
  double(*sCol)[3] = rsg.col;

  // ---- 14 rows x (pw*14) px of R, G, B per strip, luma in float64 (BT.601)
  const int cw = pw * P;
  const size_t plane = (size_t)H * W;
  const bool vec = (W & 3) == 0 && (cw & 3) == 0;
  const int q4 = cw >> 2;
  constexpr int kIt = (P * PW * P / 4 + 255) / 256;     // float4 positions per thread
  auto strip_base = [&](int pi) {
    return frame + (size_t)b * 3 * plane + (size_t)(pi * P) * W + j0 * P;
  };
  auto load = [&](int pi, float4 (&r)[kIt], float4 (&g)[kIt], float4 (&bl)[kIt]) {
    const float *base = strip_base(pi);
#pragma unroll
    for (int i = 0; i < kIt; ++i) {
      const int e = min(t + 256 * i, P * q4 - 1);
      const int y = e / q4, q = e - y * q4;
      const float *rp = base + (size_t)y * W + 4 * q;
      r[i] = *reinterpret_cast<const float4 *>(rp);
      g[i] = *reinterpret_cast<const float4 *>(rp + plane);
      bl[i] = *reinterpret_cast<const float4 *>(rp + 2 * plane);
    }
  };
  auto luma = [&](int pi, const float4 (&r)[kIt], const float4 (&g)[kIt], const float4 (&bl)[kIt]) {
    if (vec) {
#pragma unroll
      for (int i = 0; i < kIt; ++i) {
        const int e = t + 256 * i;
        if (e < P * q4) {
          const int y = e / q4, q = e - y * q4;
          const float rr[4] = {r[i].x, r[i].y, r[i].z, r[i].w};
          const float gg[4] = {g[i].x, g[i].y, g[i].z, g[i].w};
          const float bb[4] = {bl[i].x, bl[i].y, bl[i].z, bl[i].w};
          int pp = (4 * q) / P, xx = 4 * q - pp * P;
#pragma unroll
          for (int c = 0; c < 4; ++c) {
            sY[(pp * P + y) * YP + xx] = 0.299 * (double)rr[c] + 0.587 * (double)gg[c] + 0.114 * (double)bb[c];
            if (++xx == P) { xx = 0; ++pp; }
          }
        }
      }
    } else {
      const float *base = strip_base(pi);
      for (int e = t; e < P * cw; e += blockDim.x) {
        int y = e / cw, x = e - y * cw;
        const float *rp = base + (size_t)y * W + x;
        const int pp = x / P;
        sY[(pp * P + y) * YP + (x - pp * P)] =
            0.299 * (double)rp[0] + 0.587 * (double)rp[plane] + 0.114 * (double)rp[2 * plane];
      }
    }
  };
  float4 ra[kIt], ga[kIt], ba[kIt];
  if (vec) load(pi, ra, ga, ba);
  luma(pi, ra, ga, ba);
  __syncthreads();

  // ---- row stage: one thread per (patch, row)
  const bool rowt = t < pw * P;
  const int p = rowt ? t / P : 0, y = rowt ? t - p * P : 0;
  double v[P];
#pragma unroll
  for (int x = 0; x < P; ++x) v[x] = rowt ? sY[(p * P + y) * YP + x] : 0.0;
  __syncthreads();   // the tile is dead from here on: its space holds the row stage
  if (rowt) {
    double rs = 0.0;
#pragma unroll
    for (int x = 0; x < P; ++x) rs += v[x];
    sRs[p][y] = rs;
    // DFT along x (float32), outputs v = 0..7; x and 14 - x folded.
    float pf[P];
#pragma unroll
    for (int x = 0; x < P; ++x) pf[x] = (float)v[x];
    float ev[7], od[7];
#pragma unroll
    for (int x = 1; x < 7; ++x) {
      ev[x] = pf[x] + pf[P - x];
      od[x] = pf[x] - pf[P - x];
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      float re = pf[0] + ((k & 1) ? -pf[7] : pf[7]);
      float im = 0.f;
#pragma unroll
      for (int x = 1; x < 7; ++x) {
        re = fmaf(ev[x], c_cos14[(k * x) % P], re);
        im = fmaf(-od[x], c_sin14[(k * x) % P], im);
      }
      sRow[p][y * 8 + k] = make_float2(re, im);
    }
    if (f == 1) {
      // The orthonormal DCT preserves energy (Parseval), so the high-pass energy is
      // sum p^2 minus the energy of the removed low block (u < 3 and v < 3): only the
      // row DCT coefficients k < 3 are needed (float64; C[k][13 - x] = (-1)^k C[k][x]).
      double s7[7], d7[7], ss = 0.0;
#pragma unroll
      for (int x = 0; x < 7; ++x) {
        s7[x] = v[x] + v[P - 1 - x];
        d7[x] = v[x] - v[P - 1 - x];
      }
#pragma unroll
      for (int x = 0; x < P; ++x) ss = fma(v[x], v[x], ss);
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        double r = 0.0;
#pragma unroll
        for (int x = 0; x < 7; ++x) r = fma(c_dct14[k * P + x], (k & 1) ? d7[x] : s7[x], r);
        sR[p][k][y] = r;
      }
      sSs[p][y] = ss;
    }
  }
  __syncthreads();

  // ---- column stage
  // the row DFTs are read into registers first: their LDS then holds the amplitudes,
  // which leave in [bin][patch] rows (one contiguous 16-patch segment per bin)
  const bool colt = t < pw * 8;
  float2 z[P];
#pragma unroll
  for (int y = 0; y < P; ++y) z[y] = colt ? sRow[t >> 3][y * 8 + (t & 7)] : make_float2(0.f, 0.f);
  __syncthreads();
  float(*sAmp)[PW] = reinterpret_cast<float(*)[PW]>(&rsg.row[0][0][0]);
  static_assert(sizeof(float) * NB * PW <= sizeof(RowStage::row), "amplitudes fit in the row DFTs");
  if (colt) {
    // DFT along y of column v (complex), all 14 u; y and 14 - y folded.
    const int p = t >> 3, k = t & 7;
    float2 s[7], d[7];
#pragma unroll
    for (int y = 1; y < 7; ++y) {
      s[y] = make_float2(z[y].x + z[P - y].x, z[y].y + z[P - y].y);
      d[y] = make_float2(z[y].x - z[P - y].x, z[y].y - z[P - y].y);
    }
    const float2 be = make_float2(z[0].x + z[7].x, z[0].y + z[7].y);
    const float2 bo = make_float2(z[0].x - z[7].x, z[0].y - z[7].y);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      float2 A = (u & 1) ? bo : be;
      float2 Bv = make_float2(0.f, 0.f);
#pragma unroll
      for (int y = 1; y < 7; ++y) {
        const float c = c_cos14[(u * y) % P], sn = c_sin14[(u * y) % P];
        A.x = fmaf(s[y].x, c, A.x);
        A.y = fmaf(s[y].y, c, A.y);
        Bv.x = fmaf(d[y].x, sn, Bv.x);
        Bv.y = fmaf(d[y].y, sn, Bv.y);
      }
      // X(u) = A - i B, X(14 - u) = A + i B
      const float r1 = A.x + Bv.y, i1 = A.y - Bv.x;
      int bin = bin_of(u, k);
      if (bin >= 0) sAmp[bin][p] = sqrtf(r1 * r1 + i1 * i1);
      if (u >= 1 && u <= 6) {
        const float r2 = A.x - Bv.y, i2 = A.y + Bv.x;
        bin = bin_of(P - u, k);
        if (bin >= 0) sAmp[bin][p] = sqrtf(r2 * r2 + i2 * i2);
      }
    }
  } else if (f == 1 && t >= 128 && t < 128 + pw * 3) {
    // DCT along y of the row coefficients k < 3, rows u < 3: the removed low block.
    const int p = (t - 128) / 3, k = (t - 128) % 3;
    double r[P];
#pragma unroll
    for (int y = 0; y < P; ++y) r[y] = sR[p][k][y];
    double s7[7], d7[7];
#pragma unroll
    for (int y = 0; y < 7; ++y) {
      s7[y] = r[y] + r[P - 1 - y];
      d7[y] = r[y] - r[P - 1 - y];
    }
    double acc = 0.0;
#pragma unroll
    for (int u = 0; u < 3; ++u) {
      double dd = 0.0;
#pragma unroll
      for (int y = 0; y < 7; ++y) dd = fma(c_dct14[u * P + y], (u & 1) ? d7[y] : s7[y], dd);
      acc = fma(dd, dd, acc);
    }
    sCol[p][k] = acc;
  }
  __syncthreads();

  {
    // the block in LDS is already [bin][16]; slots past pw are never read
    const float4 *src = reinterpret_cast<const float4 *>(&sAmp[0][0]);
    for (int e = t; e < NB * PW / 4; e += blockDim.x) ablk[e] = src[e];
  }
  if (t < pw) {
    const int patch = pi * Gpw + j0 + t;
    double sum = 0.0;
#pragma unroll
    for (int y = 0; y < P; ++y) sum += sRs[t][y];
    pmean[(size_t)b * Np + patch] = sum / (double)(P * P);
    if (f == 1) {
      double e = 0.0;
#pragma unroll
      for (int y = 0; y < P; ++y) e += sSs[t][y];
      e -= sCol[t][0] + sCol[t][1] + sCol[t][2];
      penergy[(size_t)b * Np + patch] = fmax(e, 0.0);
    }
  }
}

// ------------------------------------------------------------------------------- helpers
// The value that lane (lane ^ O) of the wave holds, moved without the LDS: DPP lane
// permutes inside rows of 16 lanes (quad permutes for 1 and 2, row rotations for 4
// and 8) and the gfx950 row-swap instructions for 16 and 32 (with both operands the
// same register, each swap returns the even rows' and the odd rows' values).
template <int O>
__device__ __forceinline__ uint32_t xor_lane(uint32_t x) {
  const int lane = threadIdx.x & 63;
  if constexpr (O == 1) {
    return __builtin_amdgcn_update_dpp(0u, x, 0xB1, 0xF, 0xF, false);   // quad_perm [1,0,3,2]
  } else if constexpr (O == 2) {
    return __builtin_amdgcn_update_dpp(0u, x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  } else if constexpr (O == 4) {
    const uint32_t r4 = __builtin_amdgcn_update_dpp(0u, x, 0x124, 0xF, 0xF, false);   // row_ror:4
    const uint32_t r12 = __builtin_amdgcn_update_dpp(0u, x, 0x12C, 0xF, 0xF, false);  // row_ror:12
    return (lane & 4) ? r4 : r12;
  } else if constexpr (O == 8) {
    return __builtin_amdgcn_update_dpp(0u, x, 0x128, 0xF, 0xF, false);  // row_ror:8
  } else if constexpr (O == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
    return (lane & 16) ? r[0] : r[1];
  } else {
    static_assert(O == 32, "lane distance 1 .. 32");
    const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
    return (lane & 32) ? r[0] : r[1];
  }
}
template <int O>
__device__ __forceinline__ double xor_lane_d(double x) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(x);
  const uint32_t lo = xor_lane<O>((uint32_t)u), hi = xor_lane<O>((uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}
__device__ __forceinline__ double xor_lane_d(double x, int o) {
  switch (o) {
    case 1: return xor_lane_d<1>(x);
    case 2: return xor_lane_d<2>(x);
    case 4: return xor_lane_d<4>(x);
    case 8: return xor_lane_d<8>(x);
    case 16: return xor_lane_d<16>(x);
    default: return xor_lane_d<32>(x);
  }
}
__device__ __forceinline__ int xor_lane_i(int x, int o) {
  switch (o) {
    case 1: return (int)xor_lane<1>((uint32_t)x);
    case 2: return (int)xor_lane<2>((uint32_t)x);
    case 4: return (int)xor_lane<4>((uint32_t)x);
    case 8: return (int)xor_lane<8>((uint32_t)x);
    case 16: return (int)xor_lane<16>((uint32_t)x);
    default: return (int)xor_lane<32>((uint32_t)x);
  }
}
__device__ __forceinline__ double first_lane_d(double x) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(x);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)u);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(u >> 32));
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// Inclusive prefix sum over the 64 lanes of a wave: DPP shifts inside each row of 16
// lanes, then each row adds the totals of the rows before it.
__device__ __forceinline__ int wave_inclusive_scan(int x) {
  const int lane = threadIdx.x & 63;
  x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x111, 0xF, 0xF, true);   // row_shr:1
  x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x112, 0xF, 0xF, true);   // row_shr:2
  x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x114, 0xF, 0xF, true);   // row_shr:4
  x += (int)__builtin_amdgcn_update_dpp(0u, (uint32_t)x, 0x118, 0xF, 0xF, true);   // row_shr:8
  const int r0 = __builtin_amdgcn_readlane(x, 15), r1 = __builtin_amdgcn_readlane(x, 31),
            r2 = __builtin_amdgcn_readlane(x, 47);
  const int row = lane >> 4;
  return x + (row > 0 ? r0 : 0) + (row > 1 ? r1 : 0) + (row > 2 ? r2 : 0);
}

// Deterministic workgroup reductions of K values at once: a fixed butterfly inside each
// wave, the per-wave partials through LDS, then the same fixed butterfly over them in
// every wave, so every thread gets the results after one barrier pair.  scratch holds
// NW * K doubles.  MAXK: value k < MAXK is a maximum, the others sums.
template <int NW, int K, int MAXK>
__device__ void block_reduce(double (&v)[K], double *scratch) {
  static_assert(NW <= 64 && (NW & (NW - 1)) == 0, "power-of-two wave count");
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1)
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const double u = xor_lane_d(v[k], o);
      v[k] = k < MAXK ? fmax(v[k], u) : v[k] + u;
    }
  __syncthreads();
  if (lane == 0)
#pragma unroll
    for (int k = 0; k < K; ++k) scratch[w * K + k] = v[k];
  __syncthreads();
  double x[K];
#pragma unroll
  for (int k = 0; k < K; ++k)
    x[k] = lane < NW ? scratch[lane * K + k] : (k < MAXK ? -INFINITY : 0.0);
#pragma unroll
  for (int o = NW / 2; o > 0; o >>= 1)
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const double u = xor_lane_d(x[k], o);
      x[k] = k < MAXK ? fmax(x[k], u) : x[k] + u;
    }
#pragma unroll
  for (int k = 0; k < K; ++k) v[k] = first_lane_d(x[k]);
}

// One direct DFT pass over an [Gh][Gw] complex grid in LDS, one output per thread:
// along x (rows) out[y][v] = sum_x in[y][x] w^(v x), or along y (columns)
// out[u][x] = sum_y in[y][x] w^(u y); w = tw[1], tw[k] = exp(-2 pi i k / G) (conj for
// the inverse).  The twiddle index advances by v (or u) modulo G per term.
template <bool ROWS, bool INV>
__device__ __forceinline__ double2 dft_pass(const double2 *in, const double2 *tw, int e, int Gh,
                                            int Gw) {
  const int y = e / Gw, x0 = e - y * Gw;
  const int G = ROWS ? Gw : Gh;
  const int f = ROWS ? x0 : y;             // output frequency
  double re = 0.0, im = 0.0;
  int k = 0;
#pragma unroll 4
  for (int i = 0; i < G; ++i) {
    const double2 a = ROWS ? in[y * Gw + i] : in[i * Gw + x0];
    const double2 w = tw[k];
    const double wy = INV ? -w.y : w.y;
    re = fma(a.x, w.x, fma(-a.y, wy, re));
    im = fma(a.x, wy, fma(a.y, w.x, im));
    k += f;
    if (k >= G) k -= G;
  }
  return make_double2(re, im);
}

// Radix-2 FFT of every row (AXIS 0, length Gw) or column (AXIS 1, length Gh) of an
// [Gh][Gw] complex grid in LDS, in place in Y after a bit-reversed copy from X:
// out[f] = sum_i in[i] w^(f i), w = exp(-2 pi i / G) (conjugate for INV).  The whole
// workgroup takes part; tw[k] = exp(-2 pi i k / G) for the transformed axis.
template <int AXIS, bool INV>
__device__ void fft_axis(const double2 *X, double2 *Y, const double2 *tw, int Gh, int Gw) {
  const int G = AXIS == 0 ? Gw : Gh, L = AXIS == 0 ? Gh : Gw;
  const int lg = __ffs(G) - 1;
  const int M = Gh * Gw, nt = blockDim.x;
  auto at = [&](int line, int i) { return AXIS == 0 ? line * Gw + i : i * Gw + line; };
  for (int e = threadIdx.x; e < M; e += nt) {
    const int line = AXIS == 0 ? e / Gw : e % Gw, i = AXIS == 0 ? e % Gw : e / Gw;
    const int r = lg ? (int)(__brev((unsigned)i) >> (32 - lg)) : 0;
    Y[at(line, r)] = X[e];
  }
  __syncthreads();
  for (int sgl = 1; sgl <= lg; ++sgl) {
    const int half = 1 << (sgl - 1);
    for (int bt = threadIdx.x; bt < L * (G / 2); bt += nt) {
      // rows: lanes along a row; columns: lanes across columns (consecutive addresses)
      const int line = AXIS == 0 ? bt / (G / 2) : bt % L;
      const int j = AXIS == 0 ? bt - line * (G / 2) : bt / L;
      const int pos = j & (half - 1), i0 = ((j >> (sgl - 1)) << sgl) + pos, i1 = i0 + half;
      double2 w = tw[pos << (lg - sgl)];
      if (INV) w.y = -w.y;
      const double2 a = Y[at(line, i0)], c = Y[at(line, i1)];
      const double2 bw = make_double2(c.x * w.x - c.y * w.y, c.x * w.y + c.y * w.x);
      Y[at(line, i0)] = make_double2(a.x + bw.x, a.y + bw.y);
      Y[at(line, i1)] = make_double2(a.x - bw.x, a.y - bw.y);
    }
    __syncthreads();
  }
}

// 2-D transform of the grid in X (result in X, Z is scratch): FFTs for power-of-two
// sides, direct passes otherwise.  Ends with a barrier; every thread may read X.
template <bool INV>
__device__ void dft2(double2 *X, double2 *Z, const double2 *twh, const double2 *tww, int Gh,
                     int Gw) {
  const int M = Gh * Gw, t = threadIdx.x;
  if ((Gh & (Gh - 1)) == 0 && (Gw & (Gw - 1)) == 0) {
    fft_axis<0, INV>(X, Z, tww, Gh, Gw);
    fft_axis<1, INV>(Z, X, twh, Gh, Gw);
  } else {
    if (t < M) Z[t] = dft_pass<true, INV>(X, tww, t, Gh, Gw);
    __syncthreads();
    double2 r = make_double2(0.0, 0.0);
    if (t < M) r = dft_pass<false, INV>(Z, twh, t, Gh, Gw);
    __syncthreads();
    if (t < M) X[t] = r;
    __syncthreads();
  }
}

// 2-D FFT of a power-of-two [Gh][Gw] complex grid (both sides <= 64) with every line
// inside one wave: a row (then a column) sits in consecutive lanes and its radix-2
// decimation-in-frequency butterflies exchange values by lane shuffles, so the whole
// transform needs two barriers.  X holds the input and receives the result in natural
// order; T (>= Gw * (Gh + 1) elements) holds the row-transformed grid transposed,
// with a padded pitch.  out[u][v] = sum_y sum_x in[y][x] w_h^(u y) w_w^(v x),
// w = exp(-2 pi i / G) (conjugate for INV); tw*[k] = exp(-2 pi i k / G).
template <int G, bool INV>
__device__ __forceinline__ double2 fft_lanes(double2 x, int i, const double2 *tw) {
  constexpr int LG = G == 1 ? 0 : __builtin_ctz(G);
  // the twiddle of every stage is loaded up front (one LDS round trip)
  double2 w[LG > 0 ? LG : 1];
#pragma unroll
  for (int st = 0; st < LG; ++st) {
    const int h = G >> (st + 1);
    w[st] = tw[(i & (h - 1)) * (G / (2 * h))];
    if (INV) w[st].y = -w[st].y;
  }
#pragma unroll
  for (int st = 0; st < LG; ++st) {
    const int h = G >> (st + 1);
    const double px = xor_lane_d(x.x, h), py = xor_lane_d(x.y, h);
    // upper half of a butterfly: (a - b) w, a = partner; lower half: a + b
    const bool up = i & h;
    const double dx = px - x.x, dy = py - x.y;
    const double ux = dx * w[st].x - dy * w[st].y, uy = dx * w[st].y + dy * w[st].x;
    x = up ? make_double2(ux, uy) : make_double2(x.x + px, x.y + py);
  }
  return x;                                  // lane i holds frequency bitrev(i)
}
template <int G, bool INV>
__device__ __forceinline__ double2 fft_lanes_rt(double2 x, int i, int g, const double2 *tw) {
  switch (g) {
    case 64: return fft_lanes<64, INV>(x, i, tw);
    case 32: return fft_lanes<32, INV>(x, i, tw);
    case 16: return fft_lanes<16, INV>(x, i, tw);
    case 8: return fft_lanes<8, INV>(x, i, tw);
    case 4: return fft_lanes<4, INV>(x, i, tw);
    case 2: return fft_lanes<2, INV>(x, i, tw);
    default: return x;
  }
}
template <bool INV>
__device__ void fft2_wave(double2 *X, double2 *T, const double2 *twh, const double2 *tww, int Gh,
                          int Gw) {
  const int t = threadIdx.x, M = Gh * Gw, TP = Gh + 1;
  const int lw = __ffs(Gw) - 1, lh = __ffs(Gh) - 1;
  if (t < M) {
    const int row = t >> lw, col = t & (Gw - 1);
    const double2 r = fft_lanes_rt<0, INV>(X[t], col, Gw, tww);
    const int v = lw ? (int)(__brev((unsigned)col) >> (32 - lw)) : 0;
    T[v * TP + row] = r;
  }
  __syncthreads();
  if (t < M) {
    const int v = t >> lh, y = t & (Gh - 1);
    const double2 r = fft_lanes_rt<0, INV>(T[v * TP + y], y, Gh, twh);
    const int u = lh ? (int)(__brev((unsigned)y) >> (32 - lh)) : 0;
    X[u * Gw + v] = r;
  }
  __syncthreads();
}

// Two independent grids through the same transform in one pass: every stage issues the
// lane exchanges of both before either butterfly, so the two shuffle chains overlap.
// Each grid gets exactly the operations of fft_lanes (same results bit for bit).
template <int G, bool INV>
__device__ __forceinline__ void fft_lanes2(double2 &x, double2 &y, int i, const double2 *tw) {
  constexpr int LG = G == 1 ? 0 : __builtin_ctz(G);
  double2 w[LG > 0 ? LG : 1];
#pragma unroll
  for (int st = 0; st < LG; ++st) {
    const int h = G >> (st + 1);
    w[st] = tw[(i & (h - 1)) * (G / (2 * h))];
    if (INV) w[st].y = -w[st].y;
  }
#pragma unroll
  for (int st = 0; st < LG; ++st) {
    const int h = G >> (st + 1);
    const double px = xor_lane_d(x.x, h), py = xor_lane_d(x.y, h);
    const double qx = xor_lane_d(y.x, h), qy = xor_lane_d(y.y, h);
    const bool up = i & h;
    const double dx = px - x.x, dy = py - x.y;
    const double ux = dx * w[st].x - dy * w[st].y, uy = dx * w[st].y + dy * w[st].x;
    x = up ? make_double2(ux, uy) : make_double2(x.x + px, x.y + py);
    const double ex = qx - y.x, ey = qy - y.y;
    const double vx = ex * w[st].x - ey * w[st].y, vy = ex * w[st].y + ey * w[st].x;
    y = up ? make_double2(vx, vy) : make_double2(y.x + qx, y.y + qy);
  }
}
template <bool INV>
__device__ __forceinline__ void fft_lanes2_rt(double2 &x, double2 &y, int i, int g, const double2 *tw) {
  switch (g) {
    case 64: fft_lanes2<64, INV>(x, y, i, tw); break;
    case 32: fft_lanes2<32, INV>(x, y, i, tw); break;
    case 16: fft_lanes2<16, INV>(x, y, i, tw); break;
    case 8: fft_lanes2<8, INV>(x, y, i, tw); break;
    case 4: fft_lanes2<4, INV>(x, y, i, tw); break;
    case 2: fft_lanes2<2, INV>(x, y, i, tw); break;
    default: break;
  }
}
// fft2_wave on two grids X and Y at once; T and U are their transposed scratch grids.
template <bool INV>
__device__ void fft2_wave2(double2 *X, double2 *Y, double2 *T, double2 *U, const double2 *twh,
                           const double2 *tww, int Gh, int Gw) {
  const int t = threadIdx.x, M = Gh * Gw, TP = Gh + 1;
  const int lw = __ffs(Gw) - 1, lh = __ffs(Gh) - 1;
  if (t < M) {
    const int row = t >> lw, col = t & (Gw - 1);
    double2 a = X[t], c = Y[t];
    fft_lanes2_rt<INV>(a, c, col, Gw, tww);
    const int v = lw ? (int)(__brev((unsigned)col) >> (32 - lw)) : 0;
    T[v * TP + row] = a;
    U[v * TP + row] = c;
  }
  __syncthreads();
  if (t < M) {
    const int v = t >> lh, y = t & (Gh - 1);
    double2 a = T[v * TP + y], c = U[v * TP + y];
    fft_lanes2_rt<INV>(a, c, y, Gh, twh);
    const int u = lh ? (int)(__brev((unsigned)y) >> (32 - lh)) : 0;
    X[u * Gw + v] = a;
    Y[u * Gw + v] = c;
  }
  __syncthreads();
}

struct GridParams {
  int Gph, Gpw, m;
  double tau_mig, lambda_, alpha_min, alpha_max, alpha_fixed;
  int adaptive, entropy_norm;
  int no_align;                 // ablation "w/o Module I": shift (0, 0)
};

// ------------------------------------------------------------------------------- k_grid
// One workgroup of 1024 threads per frame pair, one thread per grid point (M <= 1024).
// LDS: four complex grids (two maps, two transposed scratch grids) and the twiddles
// of both axes.
constexpr int kGridThreads = 1024;
__global__ __launch_bounds__(kGridThreads) void k_grid(const double *__restrict__ pmean_prev,
                                                       const double *__restrict__ pmean_cur,
                                                       const double *__restrict__ penergy,
                                                       GridParams g, double *__restrict__ energy,
                                                       int32_t *__restrict__ shift,
                                                       double *__restrict__ scalars,
                                                       int32_t *__restrict__ counts) {
  constexpr int NW = kGridThreads / 64;
  __shared__ double2 A[kMaxTokens], Bg[kMaxTokens], C[kMaxTokens + 64], C2[kMaxTokens + 64];
  __shared__ double2 twh[kMaxTokens], tww[kMaxTokens];
  __shared__ double red[NW * 7 + 7];
  __shared__ double bestv[NW];
  __shared__ int besti[NW];
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int m = g.m;
  const int Gh = g.Gph / m, Gw = g.Gpw / m, M = Gh * Gw;
  const int Np = g.Gph * g.Gpw;
  const bool act = t < M;
  const int I = t / Gw, J = t - I * Gw;
  const bool wave_fft = (Gh & (Gh - 1)) == 0 && (Gw & (Gw - 1)) == 0 && Gh <= 64 && Gw <= 64;

  if (t < Gh) {
    double s, c;
    sincospi(2.0 * t / Gh, &s, &c);
    twh[t] = make_double2(c, -s);
  }
  if (t < Gw) {
    double s, c;
    sincospi(2.0 * t / Gw, &s, &c);
    tww[t] = make_double2(c, -s);
  }
  // token-grid mean luma of both frames (A: current, Bg: previous) and token energy
  const double inv_mm = 1.0 / (double)(m * m);
  double gc = 0.0, gp = 0.0, et = 0.0;
  if (act) {
    for (int a2 = 0; a2 < m; ++a2)
      for (int c2 = 0; c2 < m; ++c2) {
        const int p = (m * I + a2) * g.Gpw + m * J + c2;
        gc += pmean_cur[(size_t)b * Np + p];
        gp += pmean_prev[(size_t)b * Np + p];
        et += penergy[(size_t)b * Np + p];
      }
    A[t] = make_double2(gc * inv_mm, 0.0);
    Bg[t] = make_double2(gp * inv_mm, 0.0);
    if (et < 1e-8 * (double)(m * m)) et = 0.0;
    energy[(size_t)b * M + t] = et;
  }
  __syncthreads();
  // forward 2-D transforms of both maps, each on its own (a zero map must give an
  // exactly zero spectrum: the Sim_freq of Eq. 3-3 is defined as 0 there)
  if (wave_fft) {
    fft2_wave2<false>(A, Bg, C, C2, twh, tww, Gh, Gw);
  } else {
    dft2<false>(A, C, twh, tww, Gh, Gw);
    dft2<false>(Bg, C, twh, tww, Gh, Gw);
  }
  double pc = 0.0, pp = 0.0, cp = 0.0, mag = 0.0;
  if (act) {
    const double2 Fc = A[t], Fp = Bg[t];
    pc = Fc.x * Fc.x + Fc.y * Fc.y;                       // |F_t|^2
    pp = Fp.x * Fp.x + Fp.y * Fp.y;                       // |F_{t-1}|^2
    cp = sqrt(pc) * sqrt(pp);                             // |F_t| |F_{t-1}|
    // cross power X = F_{t-1} conj(F_t), kept in Bg for the inverse transform
    const double xr = Fp.x * Fc.x + Fp.y * Fc.y;
    const double xi = Fp.y * Fc.x - Fp.x * Fc.y;
    mag = sqrt(xr * xr + xi * xi);
    Bg[t] = make_double2(xr, xi);
  }

  // ---- Eq. 3-3 on the global spectra, Eq. 3-6 entropy of the current frame, the
  //      largest cross-power magnitude, token-energy mean and spread (Eq. 4-3)
  // one reduction: the entropy of P = pc / nc is ln nc - (sum pc ln pc) / nc, and the
  // energy spread comes from the sums of e and e^2
  double r1[7] = {mag, cp, pc, pp, act ? et : 0.0, act ? et * et : 0.0,
                  (act && pc > 0.0) ? pc * log(pc) : 0.0};
  block_reduce<NW, 7, 1>(r1, red);
  const double mx = r1[0], dot = r1[1], nc = r1[2], np_ = r1[3];
  const double mu = r1[4] / (double)M;
  const double ent = nc > 0.0 ? log(nc) - r1[6] / nc : 0.0;
  const double ev = fmax(r1[5] - r1[4] * mu, 0.0);

  // ---- Eq. 4-1: normalised cross-power, inverse transform (real part), first maximum
  if (act) {
    const double2 x = Bg[t];
    Bg[t] = (mx > 0.0 && mag > 1e-9 * mx) ? make_double2(x.x / mag, x.y / mag) : make_double2(0.0, 0.0);
  }
  __syncthreads();
  if (wave_fft)
    fft2_wave<true>(Bg, C, twh, tww, Gh, Gw);
  else
    dft2<true>(Bg, C, twh, tww, Gh, Gw);
  const double re = act ? Bg[t].x / (double)M : -INFINITY;
  // first maximum in row-major order: (value, index) max with the lower index on ties
  double bv = re;
  int bi = act ? t : 0x7fffffff;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const double v2 = xor_lane_d(bv, o);
    const int i2 = xor_lane_i(bi, o);
    if (v2 > bv || (v2 == bv && i2 < bi)) {
      bv = v2;
      bi = i2;
    }
  }
  if ((t & 63) == 0) {
    bestv[t >> 6] = bv;
    besti[t >> 6] = bi;
  }
  __syncthreads();

  if (t == 0) {
    double v = bestv[0];
    int kmax = besti[0];
    for (int i = 1; i < NW; ++i)
      if (bestv[i] > v || (bestv[i] == v && besti[i] < kmax)) {
        v = bestv[i];
        kmax = besti[i];
      }
    const double sim = (nc > 0.0 && np_ > 0.0) ? dot / (sqrt(nc) * sqrt(np_)) : 0.0;
    double psi = 0.0;
    if (nc > 0.0) psi = ent;
    if (g.entropy_norm) psi = (M > 1) ? psi / log((double)M) : 0.0;
    const double alpha =
        g.adaptive ? g.alpha_min + (g.alpha_max - g.alpha_min) * exp(-psi) : g.alpha_fixed;
    const int k_reuse = (int)floor(alpha * (double)M);
    const double sd = sqrt(ev / (double)M);
    const int ki = kmax / Gw, kj = kmax - ki * Gw;
    shift[b * 2 + 0] = g.no_align ? 0 : (ki <= Gh / 2 ? ki : ki - Gh);
    shift[b * 2 + 1] = g.no_align ? 0 : (kj <= Gw / 2 ? kj : kj - Gw);
    double *sc = scalars + (size_t)b * FC_NSCALARS;
    sc[FC_SCALAR_SIM_FREQ] = sim;
    sc[FC_SCALAR_PSI] = psi;
    sc[FC_SCALAR_ALPHA] = alpha;
    sc[FC_SCALAR_MU] = mu;
    sc[FC_SCALAR_SIGMA] = sd;
    sc[FC_SCALAR_THR] = mu + g.lambda_ * sd;
    int32_t *cn = counts + (size_t)b * FC_NCOUNTS;
    cn[FC_COUNT_K_REUSE] = k_reuse;
    cn[FC_COUNT_FLUSHED] = (sim < g.tau_mig) ? 1 : 0;
  }
}

// ------------------------------------------------------------------------------- k_patchsim
// Per current-frame patch, the weighted dot product of its amplitude spectrum with that
// of the patch at the same place in its token's aligned source token (previous frame),
// and both squared norms; the token cosine (Eq. 3-3 on the concatenated spectra) is
// their sum over the token's m*m patches.  Grid (ceil(Np / 64), B); the 4 waves of a
// workgroup split the 100 bins for the same 64 patches, so loads of one bin are 64
// consecutive patches.  Output pdot[(b * 3 + {dot, n_cur, n_src}) * Np + patch].
constexpr int kSimBinsPerWave = NB / 4;
__global__ __launch_bounds__(256) void k_patchsim(const float *__restrict__ amp_prev,
                                                  const float *__restrict__ amp_cur, int Gph, int Gpw,
                                                  int m, const int32_t *__restrict__ shift,
                                                  double *__restrict__ pdot) {
  __shared__ double part[3][4][64];
  const int b = blockIdx.y;
  const int Np = Gph * Gpw;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int p = blockIdx.x * 64 + lane;
  const int pc = min(p, Np - 1);
  const int pi = pc / Gpw, pj = pc - pi * Gpw;
  const int Gh = Gph / m, Gw = Gpw / m;
  const int di = shift[b * 2 + 0], dj = shift[b * 2 + 1];
  const int si = pi / m + di, sj = pj / m + dj;
  const bool al = si >= 0 && si < Gh && sj >= 0 && sj < Gw;
  const int spi = al ? pi + m * di : pi, spj = al ? pj + m * dj : pj;
  const int ncx = (Gpw + PW - 1) / PW;
  const float *ac = amp_cur + amp_chunk(b, pi, pj / PW, Gph, ncx) + (pj % PW);
  const float *ap = amp_prev + amp_chunk(b, spi, spj / PW, Gph, ncx) + (spj % PW);
  float x[kSimBinsPerWave], y[kSimBinsPerWave];
#pragma unroll
  for (int i = 0; i < kSimBinsPerWave; ++i) {
    const int bin = w * kSimBinsPerWave + i;
    x[i] = ac[bin * PW];
    y[i] = ap[bin * PW];
  }
  double dot = 0.0, n1 = 0.0, n2 = 0.0;
#pragma unroll
  for (int i = 0; i < kSimBinsPerWave; ++i) {
    const double wt = bin_weight(w * kSimBinsPerWave + i);
    const double xv = x[i], yv = y[i];
    dot = fma(wt * xv, yv, dot);
    n1 = fma(wt * xv, xv, n1);
    n2 = fma(wt * yv, yv, n2);
  }
  part[0][w][lane] = dot;
  part[1][w][lane] = n1;
  part[2][w][lane] = n2;
  __syncthreads();
  if (w == 0 && p < Np) {
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      double s = part[c][0][lane];
#pragma unroll
      for (int i = 1; i < 4; ++i) s += part[c][i][lane];
      pdot[((size_t)b * 3 + c) * Np + p] = s;
    }
  }
}

// ------------------------------------------------------------------------------- k_topk
// One workgroup per frame pair, one thread per token (M <= 1024):
//   * alignment (Eq. 4-2) and the token's spectral cosine from its patches' products;
//   * refresh mask (Eq. 4-3) and candidates (Alg. 1);
//   * the K_final candidates of smallest (energy, id) by an exact radix select of the
//     64-bit energy keys (non-negative doubles order like their bit patterns), eight
//     8-bit digits from the top, each from an LDS histogram; ties on the energy go to
//     the lower ids;
//   * reuse mask and ballot/prefix compaction of the recomputed ids (ascending).
__global__ __launch_bounds__(kMaxTokens) void k_topk(const double *__restrict__ energy,
                                                     const double *__restrict__ pdot,
                                                     const int32_t *__restrict__ shift,
                                                     const double *__restrict__ scalars,
                                                     int32_t *__restrict__ counts, double tau_sim,
                                                     int no_refresh, int Gph, int Gpw, int m,
                                                     float *__restrict__ sim,
                                                     uint8_t *__restrict__ reuse,
                                                     int32_t *__restrict__ ridx,
                                                     int32_t *__restrict__ nrec,
                                                     uint8_t *__restrict__ flags) {
  constexpr int NW = kMaxTokens / 64;
  __shared__ int hist[256];
  __shared__ int wcnt[NW];
  __shared__ int sel_digit, sel_rem, sel_cnt;
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6;
  const int Gh = Gph / m, Gw = Gpw / m, M = Gh * Gw, Np = Gph * Gpw;
  const bool act = t < M;
  const double thr = scalars[(size_t)b * FC_NSCALARS + FC_SCALAR_THR];
  const int k_reuse = counts[(size_t)b * FC_NCOUNTS + FC_COUNT_K_REUSE];
  const int flushed = counts[(size_t)b * FC_NCOUNTS + FC_COUNT_FLUSHED];

  bool cand = false;
  unsigned long long key = ~0ull;
  if (act) {
    const int I = t / Gw, J = t - I * Gw;
    const int si = I + shift[b * 2 + 0], sj = J + shift[b * 2 + 1];
    const bool al = si >= 0 && si < Gh && sj >= 0 && sj < Gw;
    // the cosine in float64; the similarity floor is applied to it before the
    // exported value is rounded to float32
    double cs = 0.0;
    if (al) {
      double dot = 0.0, n1 = 0.0, n2 = 0.0;
      for (int a2 = 0; a2 < m; ++a2)
        for (int c2 = 0; c2 < m; ++c2) {
          const int p = (m * I + a2) * Gpw + m * J + c2;
          dot += pdot[((size_t)b * 3 + 0) * Np + p];
          n1 += pdot[((size_t)b * 3 + 1) * Np + p];
          n2 += pdot[((size_t)b * 3 + 2) * Np + p];
        }
      if (n1 == 0.0 && n2 == 0.0)
        cs = 1.0;
      else if (n1 == 0.0 || n2 == 0.0)
        cs = 0.0;
      else
        cs = dot / (sqrt(n1) * sqrt(n2));
    }
    sim[(size_t)b * M + t] = (float)cs;
    const double e = energy[(size_t)b * M + t];
    const bool fr = !no_refresh && e > thr;
    cand = al && !fr && cs >= tau_sim;
    if (flags) flags[(size_t)b * M + t] = (al ? FC_FLAG_ALIGNED : 0) | (fr ? FC_FLAG_FRESH : 0) |
                                          (cand ? FC_FLAG_CAND : 0);
    if (cand) key = (unsigned long long)__double_as_longlong(e);
  }
  // candidate count
  unsigned long long bal = __ballot(cand);
  if (lane == 0) wcnt[wv] = __popcll(bal);
  __syncthreads();
  int k_cand = 0;
#pragma unroll
  for (int i = 0; i < NW; ++i) k_cand += wcnt[i];
  const int k_final = flushed ? 0 : min(k_reuse, k_cand);

  // radix select of the k_final-th smallest key among the candidates
  unsigned long long kth = 0, pmask = 0;
  int rem = k_final;                      // how many to take at or below the prefix
  if (k_final > 0) {
    for (int pass = 0; pass < 8; ++pass) {
      const int sh = 56 - 8 * pass;
      __syncthreads();
      if (t < 256) hist[t] = 0;
      __syncthreads();
      if (cand && (key & pmask) == kth) atomicAdd(&hist[(key >> sh) & 255], 1);
      __syncthreads();
      if (wv == 0) {
        // lane holds bins 4 lane .. 4 lane + 3; inclusive scan over the wave
        const int h0 = hist[4 * lane], h1 = hist[4 * lane + 1], h2 = hist[4 * lane + 2],
                  h3 = hist[4 * lane + 3];
        const int tot = h0 + h1 + h2 + h3;
        const int inc = wave_inclusive_scan(tot);
        const int exc = inc - tot;
        if (exc < rem && inc >= rem) {     // exactly one lane holds the crossing
          int c = exc, d = 4 * lane, n = h3;
          if (c + h0 >= rem) { d = 4 * lane; n = h0; }
          else if ((c += h0) + h1 >= rem) { d = 4 * lane + 1; n = h1; }
          else if ((c += h1) + h2 >= rem) { d = 4 * lane + 2; n = h2; }
          else { c += h2; d = 4 * lane + 3; }
          sel_digit = d;
          sel_rem = rem - c;
          sel_cnt = n;
        }
      }
      __syncthreads();
      kth |= (unsigned long long)sel_digit << sh;
      pmask |= 255ull << sh;
      rem = sel_rem;
      // every candidate in the chosen bin is taken: the keys need no more digits
      if (sel_cnt == rem) break;
    }
  }
  // reuse: every candidate below the selected key prefix, and the lowest-id `rem` of
  // those at the prefix (all of them when the select stopped early)
  const bool eq = cand && k_final > 0 && (key & pmask) == kth;
  bal = __ballot(eq);
  __syncthreads();
  if (lane == 0) wcnt[wv] = __popcll(bal);
  __syncthreads();
  int eq_before = __popcll(bal & ((1ull << lane) - 1ull));
  for (int i = 0; i < wv; ++i) eq_before += wcnt[i];
  const bool use = cand && k_final > 0 && ((key & pmask) < kth || (eq && eq_before < rem));

  // compaction of recomputed ids (ascending)
  const bool keep = act && !use;
  bal = __ballot(keep);
  const int before = __popcll(bal & ((1ull << lane) - 1ull));
  __syncthreads();
  if (lane == 0) wcnt[wv] = __popcll(bal);
  __syncthreads();
  int off = 0;
  for (int i = 0; i < wv; ++i) off += wcnt[i];
  if (act) {
    reuse[(size_t)b * M + t] = use ? 1 : 0;
    ridx[(size_t)b * M + t] = -1;
  }
  __syncthreads();
  if (keep) ridx[(size_t)b * M + off + before] = t;
  if (t == 0) {
    nrec[b] = M - k_final;
    counts[(size_t)b * FC_NCOUNTS + FC_COUNT_K_CAND] = k_cand;
    counts[(size_t)b * FC_NCOUNTS + FC_COUNT_K_FINAL] = k_final;
  }
}

}  // namespace

fc_status upload_select_tables() {
  float cs[P], sn[P];
  double dct[P * P];
  for (int j = 0; j < P; ++j) {
    cs[j] = (float)std::cos(2.0 * M_PI * j / P);
    sn[j] = (float)std::sin(2.0 * M_PI * j / P);
  }
  for (int k = 0; k < P; ++k)
    for (int x = 0; x < P; ++x)
      dct[k * P + x] = (k == 0 ? std::sqrt(1.0 / P) : std::sqrt(2.0 / P)) *
                       std::cos(M_PI * (2 * x + 1) * k / (2.0 * P));
  FC_HIP_TRY(hipMemcpyToSymbol(HIP_SYMBOL(c_cos14), cs, sizeof(cs)));
  FC_HIP_TRY(hipMemcpyToSymbol(HIP_SYMBOL(c_sin14), sn, sizeof(sn)));
  FC_HIP_TRY(hipMemcpyToSymbol(HIP_SYMBOL(c_dct14), dct, sizeof(dct)));
  return FC_OK;
}

fc_status launch_select(fc_ctx *ctx, const SelectWs &ws, const fc_select_params &prm,
                        const float *prev, const float *cur, int B, int H, int W,
                        const fc_select_out &out, hipStream_t st, bool carried) {
  const int m = prm.merge;
  const int Gph = H / P, Gpw = W / P;
  {
    ProfScope ps(ctx, st, "fc_spectra");
    const int nf = carried ? 1 : 2;
    dim3 grid((Gpw + PW - 1) / PW, Gph, nf * B);
    hipLaunchKernelGGL(k_spectra, grid, dim3(256), 0, st, prev, cur, H, W, Gph, Gpw, nf, ws.prev,
                       ws.cur, ws.penergy);
    FC_LAUNCH_OK(st, "k_spectra");
  }
  {
    ProfScope ps(ctx, st, "fc_grid");
    GridParams g{Gph, Gpw, m, prm.tau_mig, prm.lambda_, prm.alpha_min, prm.alpha_max,
                 prm.alpha_fixed, prm.adaptive, prm.entropy_norm, prm.no_align};
    hipLaunchKernelGGL(k_grid, dim3(B), dim3(kGridThreads), 0, st, ws.prev.pmean, ws.cur.pmean,
                       ws.penergy, g,
                       out.energy, out.shift, out.scalars, out.counts);
    FC_LAUNCH_OK(st, "k_grid");
  }
  if (prm.align_pixel) {
    // Module I at pixel resolution: the token shift of k_grid is replaced
    fc_status s = prm.align_rotation
                      ? launch_pixel_pc_rot(ctx, ws.pix, prev, cur, B, H, W, nullptr, nullptr,
                                            out.shift, P * m, prm.no_align != 0, st)
                      : launch_pixel_pc(ctx, ws.pix, prev, cur, B, H, W, nullptr, nullptr, nullptr,
                                        out.shift, P * m, prm.no_align != 0, st);
    if (s != FC_OK) return s;
  }
  {
    ProfScope ps(ctx, st, "fc_patchsim");
    dim3 grid((Gph * Gpw + 63) / 64, B);
    hipLaunchKernelGGL(k_patchsim, grid, dim3(256), 0, st, ws.prev.amp, ws.cur.amp, Gph, Gpw, m,
                       out.shift, ws.pdot);
    FC_LAUNCH_OK(st, "k_patchsim");
  }
  {
    ProfScope ps(ctx, st, "fc_topk");
    hipLaunchKernelGGL(k_topk, dim3(B), dim3(kMaxTokens), 0, st, out.energy, ws.pdot, out.shift,
                       out.scalars, out.counts, prm.tau_sim, prm.no_refresh, Gph, Gpw, m, out.sim,
                       out.reuse_mask, out.recompute_idx, out.n_recompute, out.flags);
    FC_LAUNCH_OK(st, "k_topk");
  }
  return FC_OK;
}

// ------------------------------------------------------------------------------ no-alloc path
// Workspace of fc_select_noalloc: a static device array, so that the call needs no
// allocation.  Every GPU the library runs on holds its own copy until the process ends.
// In host code the array's name is only a host-side handle; the device address of
// each GPU's copy comes from hipGetSymbolAddress (once per device, with that device
// current) and only that address is passed to kernels.  No part needs clearing: every
// element a kernel reads was written earlier in the same call.
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_noalloc_mu;
unsigned char *g_noalloc_ptr[kMaxDevices];   // per-device address of `scratch`
bool g_noalloc_ready[kMaxDevices];

// One-time set-up on the current device: architecture check, the scratch array's device
// address, and the transform tables (constant memory of this device).
fc_status noalloc_setup(int dev, unsigned char **ptr) {
  std::lock_guard<std::mutex> lk(g_noalloc_mu);
  if (!g_noalloc_ready[dev]) {
    hipDeviceProp_t prop;
    FC_HIP_TRY(hipGetDeviceProperties(&prop, dev));
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
      return fail(FC_ERR_UNSUPPORTED, "fc_select_noalloc: device %d is %s, the library targets gfx950",
                  dev, prop.gcnArchName);
    void *p = nullptr;
    FC_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (p == nullptr) return fail(FC_ERR_HIP, "fc_select_noalloc: no device address for the scratch");
    fc_status s = upload_select_tables();
    if (s != FC_OK) return s;
    g_noalloc_ptr[dev] = static_cast<unsigned char *>(p);
    g_noalloc_ready[dev] = true;
  }
  *ptr = g_noalloc_ptr[dev];
  return FC_OK;
}
}  // namespace

size_t noalloc_scratch_bytes() { return kNoAllocScratchBytes; }

fc_status launch_select_noalloc(const fc_select_params &prm, const float *prev,
                                const float *cur, int B, int H, int W,
                                const fc_select_out &out, hipStream_t st) {
  const SelectWsBytes sb = select_ws_bytes(B, H, W);
  const size_t need =
      sb.total + (prm.align_pixel ? pix_ws_bytes(B, H, W, prm.align_rotation != 0) : 0);
  if (need > kNoAllocScratchBytes)
    return fail(FC_ERR_CAPACITY, "fc_select_noalloc: %zu bytes of scratch needed, %zu available",
                need, kNoAllocScratchBytes);
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0)
    return fail(FC_ERR_NO_DEVICE, "fc_select_noalloc: no current HIP device (%s)",
                e != hipSuccess ? hipGetErrorString(e) : "none");
  if (dev >= kMaxDevices)
    return fail(FC_ERR_UNSUPPORTED, "fc_select_noalloc: device %d >= %d", dev, kMaxDevices);
  unsigned char *base = nullptr;
  fc_status s = noalloc_setup(dev, &base);
  if (s != FC_OK) return s;
  SelectWs ws;
  ws.prev = spectra_at(base, B, H, W);
  ws.cur = spectra_at(base + sb.spectra, B, H, W);
  ws.penergy = reinterpret_cast<double *>(base + 2 * sb.spectra);
  ws.pdot = reinterpret_cast<double *>(base + 2 * sb.spectra + sb.penergy);
  if (prm.align_pixel) ws.pix = pix_ws_at(base + sb.total, B, H, W, prm.align_rotation != 0);
  return launch_select(nullptr, ws, prm, prev, cur, B, H, W, out, st);
}

}  // namespace fc
