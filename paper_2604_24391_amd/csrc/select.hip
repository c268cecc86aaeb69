// Frequency-guided cacheable-token selection on gfx950 (FreqCache Sec. 4.1-4.4,
// Algorithm 1).  Four kernels:
//
//   k_spectra  one workgroup per strip of up to 16 patches (14 rows x 224 px) of
//              one frame.  Coalesced float4 loads of R, G, B rows, float64 luma
//              staged in LDS, then per patch: the 14x14 DFT amplitude (Eq. 3-2)
//              with real/even folding in float32, the patch mean, and for the
//              current frame the orthonormal DCT-II high-pass energy (Eqs. 3-4,
//              3-5) in float64.
//   k_grid     one workgroup per frame pair: token-grid mean-luma maps, their
//              2-D DFTs (float64), global amplitude similarity (Eq. 3-3) and the
//              migration gate, spectral entropy and the reuse budget (Eqs. 3-6,
//              4-4), phase correlation and its peak (Eq. 4-1), token energies and
//              their mean / std / refresh threshold (Eq. 4-3).
//   k_tokensim one thread per token: the alignment mask (Eq. 4-2) and the cosine
//              of the token's amplitude spectrum with that of its aligned source
//              token in the previous frame.
//   k_topk     one workgroup per frame pair: refresh mask, candidate set,
//              ascending-energy top-K with ties to the lower id (bitonic sort of
//              (energy bits, id) pairs in LDS), reuse mask and ballot/prefix-sum
//              compaction of the recomputed ids.
//
// The transforms are direct (no FFT library): a 14-point DFT folded on its
// even/odd symmetry costs 84 real FMAs per row and 168 per complex column, and
// the work is bound by reading the frames from HBM anyway.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>

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

// ------------------------------------------------------------------------------- k_spectra
// Grid: x = 16-patch chunk of a patch row, y = patch row, z = 2 * b + frame (0 prev,
// 1 cur).  Outputs (workspace):
//   amp[((b*2 + f) * NB + bin) * Np + patch]  float32 amplitude, unique bins:
//       bins 0..7   = (u = 0..7,  v = 0),  bins 8..15 = (u = 0..7, v = 7),
//       bins 16..99 = (u = 0..13, v = 1..6)   (the rest follow from A(u,v) = A(-u,-v));
//   pmean[(b*2 + f) * Np + patch]  float64 mean luma;
//   penergy[b * Np + patch]        float64 high-pass DCT energy (current frame only).
__global__ __launch_bounds__(256) void k_spectra(const float *__restrict__ prev,
                                                 const float *__restrict__ cur, int H, int W,
                                                 int Gph, int Gpw, float *__restrict__ amp,
                                                 double *__restrict__ pmean,
                                                 double *__restrict__ penergy) {
  const int f = blockIdx.z & 1;
  const int b = blockIdx.z >> 1;
  const int pi = blockIdx.y;
  const int j0 = blockIdx.x * PW;
  const int pw = min(PW, Gpw - j0);
  const int Np = Gph * Gpw;
  const int t = threadIdx.x;
  const float *frame = f ? cur : prev;

  if (frame == nullptr) {  // no previous frame: an all-zero frame
    for (int e = t; e < pw * NB; e += blockDim.x) {
      int p = e % pw, bin = e / pw;
      amp[((size_t)(b * 2 + f) * NB + bin) * Np + pi * Gpw + j0 + p] = 0.f;
    }
    if (t < pw) pmean[(size_t)(b * 2 + f) * Np + pi * Gpw + j0 + t] = 0.0;
    return;
  }

  __shared__ double sY[P][PW * P + 1];
  __shared__ float2 sRow[PW][P][8];
  __shared__ double sR[PW][3][P];
  __shared__ double sHp[PW][P];
  __shared__ double sRs[PW][P];
  __shared__ double sCol[PW][3];

  // ---- load 14 rows x (pw*14) px of R, G, B; luma in float64 (BT.601)
  const int cw = pw * P;
  const size_t plane = (size_t)H * W;
  const float *base = frame + (size_t)b * 3 * plane + (size_t)(pi * P) * W + j0 * P;
  if ((W & 3) == 0 && (cw & 3) == 0) {
    const int q4 = cw >> 2;
    for (int e = t; e < P * q4; e += blockDim.x) {
      int y = e / q4, q = e - y * q4;
      const float *rp = base + (size_t)y * W + 4 * q;
      float4 r = *reinterpret_cast<const float4 *>(rp);
      float4 g = *reinterpret_cast<const float4 *>(rp + plane);
      float4 bl = *reinterpret_cast<const float4 *>(rp + 2 * plane);
      sY[y][4 * q + 0] = 0.299 * (double)r.x + 0.587 * (double)g.x + 0.114 * (double)bl.x;
      sY[y][4 * q + 1] = 0.299 * (double)r.y + 0.587 * (double)g.y + 0.114 * (double)bl.y;
      sY[y][4 * q + 2] = 0.299 * (double)r.z + 0.587 * (double)g.z + 0.114 * (double)bl.z;
      sY[y][4 * q + 3] = 0.299 * (double)r.w + 0.587 * (double)g.w + 0.114 * (double)bl.w;
    }
  } else {
    for (int e = t; e < P * cw; e += blockDim.x) {
      int y = e / cw, x = e - y * cw;
      const float *rp = base + (size_t)y * W + x;
      sY[y][x] = 0.299 * (double)rp[0] + 0.587 * (double)rp[plane] + 0.114 * (double)rp[2 * plane];
    }
  }
  __syncthreads();

  // ---- row stage: one thread per (patch, row)
  if (t < pw * P) {
    const int p = t / P, y = t - p * P;
    double v[P];
#pragma unroll
    for (int x = 0; x < P; ++x) v[x] = sY[y][p * P + x];
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
      sRow[p][y][k] = make_float2(re, im);
    }
    if (f == 1) {
      // DCT-II along x (float64): C[k][13 - x] = (-1)^k C[k][x].
      double s7[7], d7[7];
#pragma unroll
      for (int x = 0; x < 7; ++x) {
        s7[x] = v[x] + v[P - 1 - x];
        d7[x] = v[x] - v[P - 1 - x];
      }
      double hp = 0.0;
#pragma unroll
      for (int k = 0; k < P; ++k) {
        double r = 0.0;
#pragma unroll
        for (int x = 0; x < 7; ++x) r = fma(c_dct14[k * P + x], (k & 1) ? d7[x] : s7[x], r);
        if (k < 3)
          sR[p][k][y] = r;
        else
          hp = fma(r, r, hp);  // columns v >= 3 keep every u: Parseval along y
      }
      sHp[p][y] = hp;
    }
  }
  __syncthreads();

  // ---- column stage
  if (t < pw * 8) {
    // DFT along y of column v (complex), all 14 u; y and 14 - y folded.
    const int p = t >> 3, k = t & 7;
    float2 z[P];
#pragma unroll
    for (int y = 0; y < P; ++y) z[y] = sRow[p][y][k];
    float2 s[7], d[7];
#pragma unroll
    for (int y = 1; y < 7; ++y) {
      s[y] = make_float2(z[y].x + z[P - y].x, z[y].y + z[P - y].y);
      d[y] = make_float2(z[y].x - z[P - y].x, z[y].y - z[P - y].y);
    }
    const float2 be = make_float2(z[0].x + z[7].x, z[0].y + z[7].y);
    const float2 bo = make_float2(z[0].x - z[7].x, z[0].y - z[7].y);
    const size_t obase = ((size_t)(b * 2 + f) * NB) * Np + pi * Gpw + j0 + p;
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
      if (bin >= 0) amp[obase + (size_t)bin * Np] = sqrtf(r1 * r1 + i1 * i1);
      if (u >= 1 && u <= 6) {
        const float r2 = A.x - Bv.y, i2 = A.y + Bv.x;
        bin = bin_of(P - u, k);
        if (bin >= 0) amp[obase + (size_t)bin * Np] = sqrtf(r2 * r2 + i2 * i2);
      }
    }
  } else if (f == 1 && t >= 128 && t < 128 + pw * 3) {
    // DCT along y of columns v < 3, rows u >= 3 only (the kept part of the block).
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
    for (int u = 3; u < P; ++u) {
      double dd = 0.0;
#pragma unroll
      for (int y = 0; y < 7; ++y) dd = fma(c_dct14[u * P + y], (u & 1) ? d7[y] : s7[y], dd);
      acc = fma(dd, dd, acc);
    }
    sCol[p][k] = acc;
  }
  __syncthreads();

  if (t < pw) {
    const int patch = pi * Gpw + j0 + t;
    double sum = 0.0;
#pragma unroll
    for (int y = 0; y < P; ++y) sum += sRs[t][y];
    pmean[(size_t)(b * 2 + f) * Np + patch] = sum / (double)(P * P);
    if (f == 1) {
      double e = 0.0;
#pragma unroll
      for (int y = 0; y < P; ++y) e += sHp[t][y];
      e += sCol[t][0] + sCol[t][1] + sCol[t][2];
      penergy[(size_t)b * Np + patch] = e;
    }
  }
}

// ------------------------------------------------------------------------------- helpers
template <typename T, typename Op>
__device__ T block_reduce(T v, T *scratch, Op op) {
  // Fixed-order tree over the workgroup (deterministic).
  const int t = threadIdx.x;
  scratch[t] = v;
  __syncthreads();
  for (int s = blockDim.x >> 1; s > 0; s >>= 1) {
    if (t < s) scratch[t] = op(scratch[t], scratch[t + s]);
    __syncthreads();
  }
  T r = scratch[0];
  __syncthreads();
  return r;
}

struct Add {
  __device__ double operator()(double a, double b) const { return a + b; }
};
struct Max {
  __device__ double operator()(double a, double b) const { return a > b ? a : b; }
};

// 2-D DFT of an [Gh][Gw] complex grid in LDS by two direct passes:
// out[u][v] = sum_y sum_x in[y][x] w_h^(u y) w_w^(v x), w = exp(sign 2 pi i / G).
__device__ void dft2_lds(const double2 *in, double2 *tmp, double2 *out, const double2 *twh,
                         const double2 *tww, int Gh, int Gw) {
  const int M = Gh * Gw;
  for (int e = threadIdx.x; e < M; e += blockDim.x) {
    const int y = e / Gw, v = e - y * Gw;
    double re = 0.0, im = 0.0;
    for (int x = 0; x < Gw; ++x) {
      const double2 a = in[y * Gw + x];
      const double2 w = tww[(v * x) % Gw];
      re += a.x * w.x - a.y * w.y;
      im += a.x * w.y + a.y * w.x;
    }
    tmp[e] = make_double2(re, im);
  }
  __syncthreads();
  for (int e = threadIdx.x; e < M; e += blockDim.x) {
    const int u = e / Gw, v = e - u * Gw;
    double re = 0.0, im = 0.0;
    for (int y = 0; y < Gh; ++y) {
      const double2 a = tmp[y * Gw + v];
      const double2 w = twh[(u * y) % Gh];
      re += a.x * w.x - a.y * w.y;
      im += a.x * w.y + a.y * w.x;
    }
    out[e] = make_double2(re, im);
  }
  __syncthreads();
}

struct GridParams {
  int Gph, Gpw, m;
  double tau_mig, lambda_, alpha_min, alpha_max, alpha_fixed;
  int adaptive, entropy_norm;
};

// ------------------------------------------------------------------------------- k_grid
// One workgroup (256 threads) per frame pair.  Dynamic LDS: 3 complex grids of
// M = Gh * Gw <= 1024 doubles2 plus twiddles.
__global__ __launch_bounds__(256) void k_grid(const double *__restrict__ pmean,
                                              const double *__restrict__ penergy, GridParams g,
                                              double *__restrict__ energy,
                                              int32_t *__restrict__ shift,
                                              double *__restrict__ scalars,
                                              int32_t *__restrict__ counts) {
  extern __shared__ double2 dyn[];
  __shared__ double red[256];
  __shared__ int redi[256];
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const int m = g.m;
  const int Gh = g.Gph / m, Gw = g.Gpw / m, M = Gh * Gw;
  const int Np = g.Gph * g.Gpw;
  double2 *X1 = dyn, *X2 = dyn + M, *X3 = dyn + 2 * M;
  double2 *twh = dyn + 3 * M, *tww = twh + Gh;

  for (int k = t; k < Gh; k += blockDim.x) {
    double s, c;
    sincospi(2.0 * k / Gh, &s, &c);
    twh[k] = make_double2(c, -s);
  }
  for (int k = t; k < Gw; k += blockDim.x) {
    double s, c;
    sincospi(2.0 * k / Gw, &s, &c);
    tww[k] = make_double2(c, -s);
  }
  const double inv_mm = 1.0 / (double)(m * m);

  // token-grid mean luma maps and their spectra: F_t -> X3, F_{t-1} -> X1
  for (int f = 1; f >= 0; --f) {
    for (int e = t; e < M; e += blockDim.x) {
      const int I = e / Gw, J = e - I * Gw;
      double s = 0.0;
      for (int a = 0; a < m; ++a)
        for (int c = 0; c < m; ++c)
          s += pmean[(size_t)(b * 2 + f) * Np + (m * I + a) * g.Gpw + m * J + c];
      X1[e] = make_double2(s * inv_mm, 0.0);
    }
    __syncthreads();
    dft2_lds(X1, X2, f ? X3 : X1, twh, tww, Gh, Gw);
  }
  double2 *Fc = X3, *Fp = X1;

  // ---- Eq. 3-3 on the global spectra, Eq. 3-6 entropy of the current frame
  double dot = 0.0, nc = 0.0, np_ = 0.0, mx = 0.0;
  for (int e = t; e < M; e += blockDim.x) {
    const double ac = sqrt(Fc[e].x * Fc[e].x + Fc[e].y * Fc[e].y);
    const double ap = sqrt(Fp[e].x * Fp[e].x + Fp[e].y * Fp[e].y);
    dot += ac * ap;
    nc += ac * ac;
    np_ += ap * ap;
    // cross power X = F_{t-1} conj(F_t)
    const double xr = Fp[e].x * Fc[e].x + Fp[e].y * Fc[e].y;
    const double xi = Fp[e].y * Fc[e].x - Fp[e].x * Fc[e].y;
    const double mag = sqrt(xr * xr + xi * xi);
    X2[e] = make_double2(xr, xi);
    mx = mag > mx ? mag : mx;
  }
  dot = block_reduce(dot, red, Add());
  nc = block_reduce(nc, red, Add());
  np_ = block_reduce(np_, red, Add());
  mx = block_reduce(mx, red, Max());
  double ent = 0.0;
  for (int e = t; e < M; e += blockDim.x) {
    const double p2 = Fc[e].x * Fc[e].x + Fc[e].y * Fc[e].y;
    if (nc > 0.0) {
      const double pr = p2 / nc;
      if (pr > 0.0) ent -= pr * log(pr);
    }
  }
  ent = block_reduce(ent, red, Add());

  // ---- Eq. 4-1: normalised cross-power, inverse transform, first maximum
  for (int e = t; e < M; e += blockDim.x) {
    const double2 x = X2[e];
    const double mag = sqrt(x.x * x.x + x.y * x.y);
    X2[e] = (mx > 0.0 && mag > 1e-9 * mx) ? make_double2(x.x / mag, x.y / mag) : make_double2(0.0, 0.0);
  }
  __syncthreads();
  // inverse: conjugate twiddles.  Row pass X2 -> X3 (F_t is no longer needed),
  // column pass keeps only the real part.
  for (int e = t; e < M; e += blockDim.x) {
    const int y = e / Gw, v = e - y * Gw;
    double re = 0.0, im = 0.0;
    for (int x = 0; x < Gw; ++x) {
      const double2 a = X2[y * Gw + x];
      const double2 w = tww[(v * x) % Gw];  // conj: (w.x, -w.y)
      re += a.x * w.x + a.y * w.y;
      im += a.y * w.x - a.x * w.y;
    }
    X3[e] = make_double2(re, im);
  }
  __syncthreads();
  double best = -INFINITY;
  int besti = 0x7fffffff;
  for (int e = t; e < M; e += blockDim.x) {
    const int u = e / Gw, v = e - u * Gw;
    double re = 0.0;
    for (int y = 0; y < Gh; ++y) {
      const double2 a = X3[y * Gw + v];
      const double2 w = twh[(u * y) % Gh];
      re += a.x * w.x + a.y * w.y;
    }
    re /= (double)M;
    if (re > best) {  // strided visit in increasing index: keeps the first maximum
      best = re;
      besti = e;
    }
  }
  red[t] = best;
  redi[t] = besti;
  __syncthreads();
  for (int s = blockDim.x >> 1; s > 0; s >>= 1) {
    if (t < s) {
      const double v2 = red[t + s];
      const int i2 = redi[t + s];
      if (v2 > red[t] || (v2 == red[t] && i2 < redi[t])) {
        red[t] = v2;
        redi[t] = i2;
      }
    }
    __syncthreads();
  }
  const int kmax = redi[0];
  __syncthreads();

  // ---- token energies (Eq. 3-5 summed over the m*m patches), Eq. 4-3 statistics
  const double snap = 1e-8 * (double)(m * m);
  double es = 0.0;
  for (int e = t; e < M; e += blockDim.x) {
    const int I = e / Gw, J = e - I * Gw;
    double s = 0.0;
    for (int a = 0; a < m; ++a)
      for (int c = 0; c < m; ++c) s += penergy[(size_t)b * Np + (m * I + a) * g.Gpw + m * J + c];
    if (s < snap) s = 0.0;
    energy[(size_t)b * M + e] = s;
    es += s;
  }
  es = block_reduce(es, red, Add());
  const double mu = es / (double)M;
  __syncthreads();  // energy[] written by this block; re-read below by the same threads
  double ev = 0.0;
  for (int e = t; e < M; e += blockDim.x) {
    const double d = energy[(size_t)b * M + e] - mu;
    ev += d * d;
  }
  ev = block_reduce(ev, red, Add());

  if (t == 0) {
    const double sim = (nc > 0.0 && np_ > 0.0) ? dot / (sqrt(nc) * sqrt(np_)) : 0.0;
    double psi = 0.0;
    if (nc > 0.0) psi = ent;
    if (g.entropy_norm) psi = (M > 1) ? psi / log((double)M) : 0.0;
    const double alpha =
        g.adaptive ? g.alpha_min + (g.alpha_max - g.alpha_min) * exp(-psi) : g.alpha_fixed;
    const int k_reuse = (int)floor(alpha * (double)M);
    const double sd = sqrt(ev / (double)M);
    const int ki = kmax / Gw, kj = kmax - ki * Gw;
    shift[b * 2 + 0] = ki <= Gh / 2 ? ki : ki - Gh;
    shift[b * 2 + 1] = kj <= Gw / 2 ? kj : kj - Gw;
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

// ------------------------------------------------------------------------------- k_tokensim
__global__ __launch_bounds__(256) void k_tokensim(const float *__restrict__ amp, int Gph,
                                                  int Gpw, int m, const int32_t *__restrict__ shift,
                                                  float *__restrict__ sim,
                                                  uint8_t *__restrict__ aligned) {
  const int b = blockIdx.y;
  const int Gh = Gph / m, Gw = Gpw / m, M = Gh * Gw;
  const int tok = blockIdx.x * blockDim.x + threadIdx.x;
  if (tok >= M) return;
  const int Np = Gph * Gpw;
  const int I = tok / Gw, J = tok - I * Gw;
  const int si = I + shift[b * 2 + 0], sj = J + shift[b * 2 + 1];
  const bool al = si >= 0 && si < Gh && sj >= 0 && sj < Gw;
  aligned[(size_t)b * M + tok] = al ? 1 : 0;
  float out = 0.f;
  if (al) {
    const float *ac = amp + (size_t)(b * 2 + 1) * NB * Np;
    const float *ap = amp + (size_t)(b * 2 + 0) * NB * Np;
    double dot = 0.0, n1 = 0.0, n2 = 0.0;
    for (int a = 0; a < m; ++a)
      for (int c = 0; c < m; ++c) {
        const int pc = (m * I + a) * Gpw + m * J + c;
        const int ps = (m * si + a) * Gpw + m * sj + c;
        for (int bin = 0; bin < NB; ++bin) {
          const double w = bin_weight(bin);
          const double x = ac[(size_t)bin * Np + pc];
          const double y = ap[(size_t)bin * Np + ps];
          dot = fma(w * x, y, dot);
          n1 = fma(w * x, x, n1);
          n2 = fma(w * y, y, n2);
        }
      }
    if (n1 == 0.0 && n2 == 0.0)
      out = 1.f;
    else if (n1 == 0.0 || n2 == 0.0)
      out = 0.f;
    else
      out = (float)(dot / (sqrt(n1) * sqrt(n2)));
  }
  sim[(size_t)b * M + tok] = out;
}

// ------------------------------------------------------------------------------- k_topk
__global__ __launch_bounds__(1024) void k_topk(const double *__restrict__ energy,
                                               const float *__restrict__ sim,
                                               const uint8_t *__restrict__ aligned,
                                               const double *__restrict__ scalars,
                                               int32_t *__restrict__ counts, double tau_sim, int M,
                                               uint8_t *__restrict__ reuse,
                                               int32_t *__restrict__ ridx,
                                               int32_t *__restrict__ nrec,
                                               uint8_t *__restrict__ flags) {
  __shared__ unsigned long long key[kMaxTokens];
  __shared__ int kid[kMaxTokens];
  __shared__ uint8_t rm[kMaxTokens];
  __shared__ int wsum[kMaxTokens / 64];
  __shared__ int ccount[kMaxTokens / 64];
  const int b = blockIdx.x;
  const int t = threadIdx.x;
  const double thr = scalars[(size_t)b * FC_NSCALARS + FC_SCALAR_THR];
  const int k_reuse = counts[(size_t)b * FC_NCOUNTS + FC_COUNT_K_REUSE];
  const int flushed = counts[(size_t)b * FC_NCOUNTS + FC_COUNT_FLUSHED];
  int npow = 1;
  while (npow < M) npow <<= 1;

  bool cand = false;
  if (t < M) {
    const double e = energy[(size_t)b * M + t];
    const bool fr = e > thr;
    const bool al = aligned[(size_t)b * M + t] != 0;
    cand = al && !fr && ((double)sim[(size_t)b * M + t] >= tau_sim);
    if (flags) flags[(size_t)b * M + t] = (al ? FC_FLAG_ALIGNED : 0) | (fr ? FC_FLAG_FRESH : 0) |
                                          (cand ? FC_FLAG_CAND : 0);
    key[t] = cand ? (unsigned long long)__double_as_longlong(e) : ~0ull;
    kid[t] = t;
    rm[t] = 0;
  } else if (t < npow) {
    key[t] = ~0ull;
    kid[t] = 0x7fffffff;
  }
  // candidate count
  const unsigned long long bal = __ballot(cand);
  const int lane = t & 63, wv = t >> 6;
  if (lane == 0) ccount[wv] = __popcll(bal);
  __syncthreads();
  int k_cand = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) k_cand += ccount[i];

  // bitonic sort ascending on (key, id)
  for (int k = 2; k <= npow; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int ixj = t ^ j;
      if (t < npow && ixj > t) {
        const bool up = (t & k) == 0;
        const unsigned long long ka = key[t], kb = key[ixj];
        const int ia = kid[t], ib = kid[ixj];
        const bool gt = ka > kb || (ka == kb && ia > ib);
        if (gt == up) {
          key[t] = kb;
          key[ixj] = ka;
          kid[t] = ib;
          kid[ixj] = ia;
        }
      }
      __syncthreads();
    }
  }
  const int k_final = flushed ? 0 : min(k_reuse, k_cand);
  if (t < k_final) rm[kid[t]] = 1;
  __syncthreads();

  // compaction of recomputed ids (ascending)
  const bool keep = (t < M) && rm[t] == 0;
  const unsigned long long kb = __ballot(keep);
  const int before = __popcll(kb & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[wv] = __popcll(kb);
  __syncthreads();
  int off = 0;
  for (int i = 0; i < wv; ++i) off += wsum[i];
  if (t < M) {
    reuse[(size_t)b * M + t] = rm[t];
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

fc_status launch_select(fc_ctx *ctx, const fc_select_params &prm, const float *prev,
                        const float *cur, int B, int H, int W, const fc_select_out &out,
                        hipStream_t st) {
  const int m = prm.merge;
  const int Gph = H / P, Gpw = W / P;
  const int Gh = Gph / m, Gw = Gpw / m, M = Gh * Gw;
  {
    ProfScope ps(ctx, st, "fc_spectra");
    dim3 grid((Gpw + PW - 1) / PW, Gph, 2 * B);
    hipLaunchKernelGGL(k_spectra, grid, dim3(256), 0, st, prev, cur, H, W, Gph, Gpw, ctx->amp,
                       ctx->pmean, ctx->penergy);
    FC_HIP_TRY(hipGetLastError());
  }
  {
    ProfScope ps(ctx, st, "fc_grid");
    GridParams g{Gph, Gpw, m, prm.tau_mig, prm.lambda_, prm.alpha_min, prm.alpha_max,
                 prm.alpha_fixed, prm.adaptive, prm.entropy_norm};
    const size_t lds = (size_t)(3 * M + Gh + Gw) * sizeof(double2);
    hipLaunchKernelGGL(k_grid, dim3(B), dim3(256), lds, st, ctx->pmean, ctx->penergy, g,
                       out.energy, out.shift, out.scalars, out.counts);
    FC_HIP_TRY(hipGetLastError());
  }
  {
    ProfScope ps(ctx, st, "fc_tokensim");
    dim3 grid((M + 255) / 256, B);
    hipLaunchKernelGGL(k_tokensim, grid, dim3(256), 0, st, ctx->amp, Gph, Gpw, m, out.shift,
                       out.sim, ctx->aligned);
    FC_HIP_TRY(hipGetLastError());
  }
  {
    ProfScope ps(ctx, st, "fc_topk");
    hipLaunchKernelGGL(k_topk, dim3(B), dim3(1024), 0, st, out.energy, out.sim, ctx->aligned,
                       out.scalars, out.counts, prm.tau_sim, M, out.reuse_mask,
                       out.recompute_idx, out.n_recompute, out.flags);
    FC_HIP_TRY(hipGetLastError());
  }
  return FC_OK;
}

}  // namespace fc
