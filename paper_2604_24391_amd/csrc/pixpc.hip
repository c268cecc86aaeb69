// Pixel-resolution phase correlation on gfx950: Eq. 4-1 with the feature maps taken as
// the frames' full-resolution BT.601 luma, the integer peak refined per axis by a
// three-point parabola, and (for the selection) the displacement rounded to whole tokens.
// A variant of Module I (Sec. 4.1) for frames whose motion is not a whole number of
// tokens; the token-grid reading stays the default.
//
// The frames are real, so only columns 0..W/2 of each row spectrum are kept (the rest
// is their conjugate mirror).  Five kernels per call, all float64 like the oracle's
// decision:
//
//   k_pc_rows      one workgroup per (image row, pair): luma of both frames, their
//                  length-W FFTs in LDS, the two half-row spectra.
//   k_pc_cols<1>   one workgroup per (strip of CW columns, pair): column FFTs of both
//                  half-spectra, cross power X = F_{t-1} conj(F_t) in place, the
//                  strip's largest |X|.
//   k_pc_cols<0>   same strips: X / |X| under the guard |X| > 1e-9 max|X| (else 0),
//                  inverse column FFTs.
//   k_pc_rows_inv  one workgroup per (row, pair): the Hermitian row completed from its
//                  half, inverse FFT, real part / (H W) = the response surface, and the
//                  row's first maximum.
//   k_pc_peak      one workgroup per pair: first maximum over the rows (row-major ties
//                  to the lower index), signed wrap, parabolic refinement with circular
//                  neighbours, the token shift.
//
// The FFTs are self-sorting (Stockham) mixed-radix transforms of length n = 7 2^k:
// one radix-7 stage, then radix-4 stages and at most one radix-2 stage, each stage a
// pass over LDS between two buffers.  Twiddles come from one table per workgroup
// (sincospi of the exact rational angle m / n).  Sizes: H and W of the form 7 2^k with
// 2 <= 2^k <= 128 (14 ... 896).
//
// Rotation (Fourier-Mellin, launch_pixel_pc_rot): the forward column pass also writes
// the high-pass weighted magnitude spectra of both frames; k_lp_sample resamples them
// on a log-polar grid (H angles over [0, pi), min(H, W) / 2 radii); the same correlation
// kernels on those maps give the rotation from the peak's angular coordinate;
// k_derotate rotates the current frame's luma back about the centre; a last
// correlation gives the displacement of the image centre.
#include <hip/hip_runtime.h>

#include <cmath>

#include "fc_internal.h"

namespace fc {
namespace {

constexpr int kPcThreads = 256;
constexpr int kPcMaxN = 896;

__device__ __forceinline__ double2 cmul(double2 a, double2 b) {
  return make_double2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ double2 cadd(double2 a, double2 b) { return make_double2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ double2 csub(double2 a, double2 b) { return make_double2(a.x - b.x, a.y - b.y); }

// Twiddle table of a length-n transform in LDS: tw[m] = e^{-2 pi i m / n}, m < n, from
// sincospi of the exact rational angle.  Every stage's twiddle and the radix-7 roots are
// entries of it (the inverse transform takes their conjugates).
__device__ void make_twiddles(double2 *tw, int n) {
  for (int m = threadIdx.x; m < n; m += blockDim.x) {
    double s, c;
    sincospi(2.0 * (double)m / (double)n, &s, &c);
    tw[m] = make_double2(c, -s);
  }
}

template <bool INV>
__device__ __forceinline__ double2 tw_at(const double2 *tw, int m) {
  const double2 w = tw[m];
  return INV ? make_double2(w.x, -w.y) : w;
}

// In-register DFT of R points: V[q] = sum_r v[r] e^{-+2 pi i r q / R} (- forward).
// w7: the seventh roots of unity of the transform's direction (radix 7 only).
template <int R, bool INV>
__device__ __forceinline__ void dft_reg(double2 (&v)[R], const double2 *w7);

template <>
__device__ __forceinline__ void dft_reg<2, false>(double2 (&v)[2], const double2 *) {
  const double2 a = v[0], b = v[1];
  v[0] = cadd(a, b);
  v[1] = csub(a, b);
}
template <>
__device__ __forceinline__ void dft_reg<2, true>(double2 (&v)[2], const double2 *) {
  const double2 a = v[0], b = v[1];
  v[0] = cadd(a, b);
  v[1] = csub(a, b);
}

template <bool INV>
__device__ __forceinline__ void dft4(double2 (&v)[4]) {
  const double2 s02 = cadd(v[0], v[2]), d02 = csub(v[0], v[2]);
  const double2 s13 = cadd(v[1], v[3]), d13 = csub(v[1], v[3]);
  // -i (v1 - v3) forward, +i (v1 - v3) inverse
  const double2 jd13 = INV ? make_double2(-d13.y, d13.x) : make_double2(d13.y, -d13.x);
  v[0] = cadd(s02, s13);
  v[1] = cadd(d02, jd13);
  v[2] = csub(s02, s13);
  v[3] = csub(d02, jd13);
}
template <>
__device__ __forceinline__ void dft_reg<4, false>(double2 (&v)[4], const double2 *) { dft4<false>(v); }
template <>
__device__ __forceinline__ void dft_reg<4, true>(double2 (&v)[4], const double2 *) { dft4<true>(v); }

template <bool INV>
__device__ __forceinline__ void dft7(double2 (&v)[7], const double2 *w7) {
  double2 out[7];
#pragma unroll
  for (int q = 0; q < 7; ++q) {
    double2 acc = v[0];
#pragma unroll
    for (int r = 1; r < 7; ++r) acc = cadd(acc, cmul(v[r], w7[(r * q) % 7]));
    out[q] = acc;
  }
#pragma unroll
  for (int q = 0; q < 7; ++q) v[q] = out[q];
}
template <>
__device__ __forceinline__ void dft_reg<7, false>(double2 (&v)[7], const double2 *w7) { dft7<false>(v, w7); }
template <>
__device__ __forceinline__ void dft_reg<7, true>(double2 (&v)[7], const double2 *w7) { dft7<true>(v, w7); }

// One Stockham stage of radix R over nseq sequences of length n (pitch n) in LDS:
// it combines R sub-transforms of length ns into ones of length ns R.  The twiddle of
// element r of butterfly j is e^{-+2 pi i r k / (ns R)}, k = j mod ns, which is
// tw[r k n / (ns R)].
template <int R, bool INV>
__device__ __forceinline__ void stage(const double2 *__restrict__ d0, double2 *__restrict__ d1,
                                      const double2 *__restrict__ tw, int n, int nseq, int ns) {
  const int per = n / R;
  const int step = n / (ns * R);
  double2 w7[7];
  if (R == 7) {
#pragma unroll
    for (int k = 0; k < 7; ++k) w7[k] = tw_at<INV>(tw, k * (n / 7));
  }
  for (int it = threadIdx.x; it < nseq * per; it += blockDim.x) {
    const int s = it / per, j = it - s * per;
    const double2 *src = d0 + (long)s * n;
    double2 *dst = d1 + (long)s * n;
    const int k = j % ns;
    double2 v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
      v[r] = src[j + r * per];
      if (r > 0 && k > 0) v[r] = cmul(v[r], tw_at<INV>(tw, r * k * step));
    }
    dft_reg<R, INV>(v, w7);
    const int o = (j / ns) * ns * R + k;
#pragma unroll
    for (int q = 0; q < R; ++q) dst[o + q * ns] = v[q];
  }
}

// Batched FFT of nseq length-n sequences (n = 7 2^k) held in a; b is scratch of the same
// size, tw the table of make_twiddles(n).  Returns the buffer that holds the result.
// INV: the inverse transform, unnormalised.
template <bool INV>
__device__ double2 *fft_lds(double2 *a, double2 *b, const double2 *tw, int n, int nseq) {
  int ns = 1;
  stage<7, INV>(a, b, tw, n, nseq, ns);
  __syncthreads();
  ns = 7;
  double2 *x = b, *y = a;
  int rest = n / 7;
  while (rest >= 4) {
    stage<4, INV>(x, y, tw, n, nseq, ns);
    __syncthreads();
    ns *= 4;
    rest /= 4;
    double2 *t = x;
    x = y;
    y = t;
  }
  if (rest == 2) {
    stage<2, INV>(x, y, tw, n, nseq, ns);
    __syncthreads();
    double2 *t = x;
    x = y;
    y = t;
  }
  return x;
}

__device__ __forceinline__ double luma_at(const float *frame, size_t plane, size_t off) {
  return 0.299 * (double)frame[off] + 0.587 * (double)frame[plane + off] +
         0.114 * (double)frame[2 * plane + off];
}

// ------------------------------------------------------------------------- k_pc_rows
// The two frames' rows are transformed as two separate sequences (not packed into one
// complex sequence): packing leaks rounding noise of one frame's spectrum into the
// other's, which dominates when a frame is (nearly) zero.
// Each side of a pair is a real map ([B][H][W] float64) or a frame's luma ([B][3][H][W]
// float32 RGB), or all zero when both are null.
struct PcIn {
  const float *rgb_prev, *rgb_cur;
  const double *map_prev, *map_cur;
};

__device__ __forceinline__ double pc_input(const float *rgb, const double *map, int b, int H, int W,
                                           int y, int x) {
  const size_t plane = (size_t)H * W, off = (size_t)y * W + x;
  if (map) return map[(size_t)b * plane + off];
  if (rgb) return luma_at(rgb + (size_t)b * 3 * plane, plane, off);
  return 0.0;
}

__global__ __launch_bounds__(kPcThreads) void k_pc_rows(PcIn in, int H, int W, PixWs ws) {
  __shared__ double2 buf[2][2 * kPcMaxN];
  __shared__ double2 tw[kPcMaxN];
  const int y = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  const int hw = W / 2 + 1;
  make_twiddles(tw, W);
  for (int x = t; x < W; x += blockDim.x) {
    buf[0][x] = make_double2(pc_input(in.rgb_prev, in.map_prev, b, H, W, y, x), 0.0);
    buf[0][W + x] = make_double2(pc_input(in.rgb_cur, in.map_cur, b, H, W, y, x), 0.0);
  }
  __syncthreads();
  const double2 *Z = fft_lds<false>(buf[0], buf[1], tw, W, 2);
  double2 *sa = ws.sa + ((size_t)b * H + y) * hw;
  double2 *sb = ws.sb + ((size_t)b * H + y) * hw;
  for (int k = t; k < hw; k += blockDim.x) {
    sa[k] = Z[k];
    sb[k] = Z[W + k];
  }
}

// ------------------------------------------------------------------------- k_pc_cols
// Column strips: CW adjacent half-spectrum columns per workgroup, for H <= MAXH.
// FWD with mag: also the high-pass weighted magnitudes of both spectra,
// mag[b][side][ky][kx] = (1 - X)(2 - X) |F|, X = cos(pi f_y) cos(pi f_x) (f the signed
// frequency in cycles per sample).
template <int MAXH, int CW, bool FWD>
__global__ __launch_bounds__(kPcThreads) void k_pc_cols(int H, int W, PixWs ws, double *mag) {
  constexpr int NS = FWD ? 2 * CW : CW;
  __shared__ double2 buf[2][NS * MAXH];
  __shared__ double2 tw[MAXH];
  __shared__ double red[kPcThreads / 64];
  const int b = blockIdx.y, t = threadIdx.x;
  make_twiddles(tw, H);
  const int hw = W / 2 + 1;
  const int c0 = blockIdx.x * CW;
  const int cw = min(CW, hw - c0);
  double2 *sa = ws.sa + (size_t)b * H * hw;
  const double2 *sb = ws.sb + (size_t)b * H * hw;
  if (FWD) {
    for (int e = t; e < NS * H; e += blockDim.x) {
      const int s = e / H, y = e - s * H;
      const int c = s < CW ? s : s - CW;
      double2 v = make_double2(0.0, 0.0);
      if (c < cw) v = (s < CW ? sa : sb)[(size_t)y * hw + c0 + c];
      buf[0][s * H + y] = v;
    }
    __syncthreads();
    double2 *F = fft_lds<false>(buf[0], buf[1], tw, H, NS);
    double mx = 0.0;
    for (int e = t; e < cw * H; e += blockDim.x) {
      const int c = e / H, ky = e - c * H;
      const double2 f1 = F[c * H + ky], f2 = F[(CW + c) * H + ky];
      if (mag) {
        const int kx = c0 + c;
        const double fy = (double)(2 * ky < H ? ky : ky - H) / (double)H;
        const double fx = (double)(2 * kx < W ? kx : kx - W) / (double)W;
        const double X = cospi(fy) * cospi(fx);
        const double hp = (1.0 - X) * (2.0 - X);
        const size_t o = ((size_t)b * 2 * H + ky) * hw + kx;
        mag[o] = hp * sqrt(f1.x * f1.x + f1.y * f1.y);
        mag[o + (size_t)H * hw] = hp * sqrt(f2.x * f2.x + f2.y * f2.y);
      }
      const double xr = f1.x * f2.x + f1.y * f2.y;
      const double xi = f1.y * f2.x - f1.x * f2.y;
      sa[(size_t)ky * hw + c0 + c] = make_double2(xr, xi);
      mx = fmax(mx, sqrt(xr * xr + xi * xi));
    }
    for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o));
    if ((t & 63) == 0) red[t >> 6] = mx;
    __syncthreads();
    if (t == 0) {
      double m = red[0];
      for (int i = 1; i < kPcThreads / 64; ++i) m = fmax(m, red[i]);
      ws.bmax[(size_t)b * gridDim.x + blockIdx.x] = m;
    }
  } else {
    if (t < 64) {
      double m = 0.0;
      for (int i = t; i < (int)gridDim.x; i += 64) m = fmax(m, ws.bmax[(size_t)b * gridDim.x + i]);
      for (int o = 32; o > 0; o >>= 1) m = fmax(m, __shfl_xor(m, o));
      if (t == 0) red[0] = m;
    }
    __syncthreads();
    const double gmax = red[0];
    for (int e = t; e < NS * H; e += blockDim.x) {
      const int c = e / H, y = e - c * H;
      double2 v = make_double2(0.0, 0.0);
      if (c < cw) {
        const double2 x = sa[(size_t)y * hw + c0 + c];
        const double mag = sqrt(x.x * x.x + x.y * x.y);
        if (gmax > 0.0 && mag > 1e-9 * gmax) v = make_double2(x.x / mag, x.y / mag);
      }
      buf[0][c * H + y] = v;
    }
    __syncthreads();
    const double2 *G = fft_lds<true>(buf[0], buf[1], tw, H, NS);
    for (int e = t; e < cw * H; e += blockDim.x) {
      const int c = e / H, y = e - c * H;
      sa[(size_t)y * hw + c0 + c] = G[c * H + y];
    }
  }
}

// --------------------------------------------------------------------- k_pc_rows_inv
__global__ __launch_bounds__(kPcThreads) void k_pc_rows_inv(int H, int W, PixWs ws,
                                                            double *__restrict__ resp) {
  __shared__ double2 buf[2][kPcMaxN];
  __shared__ double2 tw[kPcMaxN];
  __shared__ double bv[kPcThreads / 64];
  __shared__ int bi[kPcThreads / 64];
  const int y = blockIdx.x, b = blockIdx.y, t = threadIdx.x;
  const int hw = W / 2 + 1;
  make_twiddles(tw, W);
  const double2 *g = ws.sa + ((size_t)b * H + y) * hw;
  for (int k = t; k < W; k += blockDim.x) {
    double2 v;
    if (k < hw) {
      v = g[k];
    } else {
      const double2 m = g[W - k];
      v = make_double2(m.x, -m.y);
    }
    buf[0][k] = v;
  }
  __syncthreads();
  const double2 *R = fft_lds<true>(buf[0], buf[1], tw, W, 1);
  const double hwn = (double)H * (double)W;
  double best = -INFINITY;
  int arg = 0x7fffffff;
  double *row = resp + ((size_t)b * H + y) * W;
  for (int x = t; x < W; x += blockDim.x) {
    const double r = R[x].x / hwn;
    row[x] = r;
    if (r > best) {  // ascending x per thread: the first maximum
      best = r;
      arg = x;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const double v2 = __shfl_xor(best, o);
    const int i2 = __shfl_xor(arg, o);
    if (v2 > best || (v2 == best && i2 < arg)) {
      best = v2;
      arg = i2;
    }
  }
  if ((t & 63) == 0) {
    bv[t >> 6] = best;
    bi[t >> 6] = arg;
  }
  __syncthreads();
  if (t == 0) {
    double v = bv[0];
    int a = bi[0];
    for (int i = 1; i < kPcThreads / 64; ++i)
      if (bv[i] > v || (bv[i] == v && bi[i] < a)) {
        v = bv[i];
        a = bi[i];
      }
    ws.rowmax[(size_t)b * H + y] = v;
    ws.rowarg[(size_t)b * H + y] = a;
  }
}

// ------------------------------------------------------------------------- k_pc_peak
__device__ __forceinline__ double parabolic(double a, double c0, double c) {
  const double den = a - 2.0 * c0 + c;
  return den >= 0.0 ? 0.0 : (a - c) / (2.0 * den);
}

__device__ __forceinline__ int token_round(double d, int tp) {
  const double q = fabs(d) / (double)tp;
  const int k = (int)floor(q + 0.5);
  return d >= 0.0 ? k : -k;
}

__global__ __launch_bounds__(kPcThreads) void k_pc_peak(int H, int W, PixWs ws,
                                                        const double *__restrict__ resp,
                                                        double *__restrict__ shift_px,
                                                        int32_t *__restrict__ peak,
                                                        int32_t *__restrict__ tok_shift, int tp,
                                                        int zero_shift) {
  __shared__ double bv[kPcThreads / 64];
  __shared__ long bi[kPcThreads / 64];
  const int b = blockIdx.x, t = threadIdx.x;
  double best = -INFINITY;
  long arg = 0x7fffffffffffffffL;
  for (int y = t; y < H; y += blockDim.x) {
    const double v = ws.rowmax[(size_t)b * H + y];
    const long i = (long)y * W + ws.rowarg[(size_t)b * H + y];
    if (v > best || (v == best && i < arg)) {
      best = v;
      arg = i;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const double v2 = __shfl_xor(best, o);
    const long i2 = __shfl_xor(arg, o);
    if (v2 > best || (v2 == best && i2 < arg)) {
      best = v2;
      arg = i2;
    }
  }
  if ((t & 63) == 0) {
    bv[t >> 6] = best;
    bi[t >> 6] = arg;
  }
  __syncthreads();
  if (t != 0) return;
  double v = bv[0];
  long a = bi[0];
  for (int i = 1; i < kPcThreads / 64; ++i)
    if (bv[i] > v || (bv[i] == v && bi[i] < a)) {
      v = bv[i];
      a = bi[i];
    }
  const int ki = (int)(a / W), kj = (int)(a - (long)ki * W);
  const int pi = ki <= H / 2 ? ki : ki - H;
  const int pj = kj <= W / 2 ? kj : kj - W;
  const double *r = resp + (size_t)b * H * W;
  const double c0 = r[(size_t)ki * W + kj];
  const double di = pi + parabolic(r[(size_t)((ki - 1 + H) % H) * W + kj], c0,
                                   r[(size_t)((ki + 1) % H) * W + kj]);
  const double dj = pj + parabolic(r[(size_t)ki * W + (kj - 1 + W) % W], c0,
                                   r[(size_t)ki * W + (kj + 1) % W]);
  if (shift_px) {
    shift_px[2 * b] = di;
    shift_px[2 * b + 1] = dj;
  }
  if (peak) {
    peak[2 * b] = pi;
    peak[2 * b + 1] = pj;
  }
  if (tok_shift) {
    tok_shift[2 * b] = zero_shift ? 0 : token_round(di, tp);
    tok_shift[2 * b + 1] = zero_shift ? 0 : token_round(dj, tp);
  }
}

template <int MAXH, int CW>
void launch_cols(int H, int W, int B, const PixWs &ws, double *mag, bool fwd_only, hipStream_t st) {
  const int hw = W / 2 + 1;
  const dim3 grid((unsigned)((hw + CW - 1) / CW), (unsigned)B);
  hipLaunchKernelGGL((k_pc_cols<MAXH, CW, true>), grid, dim3(kPcThreads), 0, st, H, W, ws, mag);
  if (!fwd_only)
    hipLaunchKernelGGL((k_pc_cols<MAXH, CW, false>), grid, dim3(kPcThreads), 0, st, H, W, ws,
                       (double *)nullptr);
}

// ----------------------------------------------------------------- rotation (log-polar)
// Log-polar samples of both frames' weighted magnitude spectra: angle i pi / NT, radius
// R^(j / NR), R = min(H, W) / 2 - 1, bilinear over the half-plane kx in [0, W/2] (a point
// with kx outside it is read at its mirror -k: the magnitudes of real frames are centrally
// symmetric).  lp[side][b][i][j] (side 0: previous frame), so each side is a batch of
// NT x NR maps.
__device__ __forceinline__ double mag_at(const double *m, int H, int W, int ky, int kx) {
  const int hw = W / 2 + 1;
  kx %= W;
  if (kx < 0) kx += W;
  ky %= H;
  if (ky < 0) ky += H;
  if (kx >= hw) {            // the mirror -k
    kx = W - kx;
    ky = ky == 0 ? 0 : H - ky;
  }
  return m[(size_t)ky * hw + kx];
}

__global__ __launch_bounds__(kPcThreads) void k_lp_sample(const double *__restrict__ mag, int H,
                                                          int W, int NT, int NR,
                                                          double *__restrict__ lp) {
  const int i = blockIdx.x, b = blockIdx.y;
  const int hw = W / 2 + 1;
  const double R = (double)min(H, W) / 2.0 - 1.0;
  double sn, cs;
  sincospi((double)i / (double)NT, &sn, &cs);
  for (int e = threadIdx.x; e < 2 * NR; e += blockDim.x) {
    const int side = e / NR, j = e - side * NR;
    const double r = pow(R, (double)j / (double)NR);
    const double fy = r * sn, fx = r * cs;
    const double y0 = floor(fy), x0 = floor(fx);
    const double wy = fy - y0, wx = fx - x0;
    const int iy = (int)y0, ix = (int)x0;
    const double *m = mag + ((size_t)b * 2 + side) * H * hw;
    const double v = (1.0 - wy) * (1.0 - wx) * mag_at(m, H, W, iy, ix) +
                     (1.0 - wy) * wx * mag_at(m, H, W, iy, ix + 1) +
                     wy * (1.0 - wx) * mag_at(m, H, W, iy + 1, ix) +
                     wy * wx * mag_at(m, H, W, iy + 1, ix + 1);
    lp[(((size_t)side * gridDim.y + b) * NT + i) * NR + j] = v;
  }
}

// The current frame's luma rotated back by the estimated angle, a = -dtheta pi / NT
// (dtheta: the angular coordinate of the log-polar correlation peak):
// yrot(q) = Y(R(a)(q - c) + c), bilinear, 0 outside the frame.
__global__ __launch_bounds__(kPcThreads) void k_derotate(const float *__restrict__ cur, int H,
                                                         int W, const double *__restrict__ dth,
                                                         int NT, double *__restrict__ yrot,
                                                         double *__restrict__ angle) {
  const int y = blockIdx.x, b = blockIdx.y;
  const double a = -dth[2 * b] * M_PI / (double)NT;
  if (angle && y == 0 && threadIdx.x == 0) angle[b] = a;
  double sa, ca;
  sincos(a, &sa, &ca);
  const double cy = (H - 1) / 2.0, cx = (W - 1) / 2.0;
  const size_t plane = (size_t)H * W;
  const float *fr = cur + (size_t)b * 3 * plane;
  for (int x = threadIdx.x; x < W; x += blockDim.x) {
    const double qy = y - cy, qx = x - cx;
    const double sy = qx * sa + qy * ca + cy, sx = qx * ca - qy * sa + cx;
    const double y0 = floor(sy), x0 = floor(sx);
    const double wy = sy - y0, wx = sx - x0;
    const int iy = (int)y0, ix = (int)x0;
    double v = 0.0;
    for (int u = 0; u < 2; ++u)
      for (int w2 = 0; w2 < 2; ++w2) {
        const int yy = iy + u, xx = ix + w2;
        if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;
        const double wgt = (u ? wy : 1.0 - wy) * (w2 ? wx : 1.0 - wx);
        v += wgt * luma_at(fr, plane, (size_t)yy * W + xx);
      }
    yrot[(size_t)b * plane + (size_t)y * W + x] = v;
  }
}

}  // namespace

bool pix_size_ok(int n) {
  if (n < 14 || n > kPcMaxN || n % 7) return false;
  const int p = n / 7;
  return (p & (p - 1)) == 0;
}

bool pix_rot_size_ok(int H, int W) {
  return pix_size_ok(H) && pix_size_ok(W) && pix_size_ok(std::min(H, W) / 2);
}

namespace {
// Workspace parts in order: sa, sb, rowmax, rowarg, bmax, shift_px, then with rotation
// mag [B][2][H][W/2 + 1], lp [2][B][H][min(H, W) / 2], yrot [B][H][W].
template <typename F>
void pix_parts(long B, long H, long W, bool rot, F &&take) {
  const long hw = W / 2 + 1;
  const long ncb = (hw + 1) / 2;             // strips of the narrowest kind (CW = 2)
  take(0, (size_t)B * H * hw * sizeof(double2));
  take(1, (size_t)B * H * hw * sizeof(double2));
  take(2, (size_t)B * H * sizeof(double));
  take(3, (size_t)B * H * sizeof(int));
  take(4, (size_t)B * ncb * sizeof(double));
  take(5, (size_t)B * 2 * sizeof(double));
  if (rot) {
    take(6, (size_t)B * 2 * H * hw * sizeof(double));
    take(7, (size_t)B * 2 * H * (std::min(H, W) / 2) * sizeof(double));
    take(8, (size_t)B * H * W * sizeof(double));
  }
}
size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
}  // namespace

size_t pix_ws_bytes(long B, long H, long W, bool rot) {
  size_t n = 0;
  pix_parts(B, H, W, rot, [&](int, size_t bytes) { n += al256(bytes); });
  return n;
}

PixWs pix_ws_at(void *base, long B, long H, long W, bool rot) {
  unsigned char *p = static_cast<unsigned char *>(base);
  PixWs ws;
  pix_parts(B, H, W, rot, [&](int part, size_t bytes) {
    switch (part) {
      case 0: ws.sa = reinterpret_cast<double2 *>(p); break;
      case 1: ws.sb = reinterpret_cast<double2 *>(p); break;
      case 2: ws.rowmax = reinterpret_cast<double *>(p); break;
      case 3: ws.rowarg = reinterpret_cast<int *>(p); break;
      case 4: ws.bmax = reinterpret_cast<double *>(p); break;
      case 5: ws.shift_px = reinterpret_cast<double *>(p); break;
      case 6: ws.mag = reinterpret_cast<double *>(p); break;
      case 7: ws.lp = reinterpret_cast<double *>(p); break;
      case 8: ws.yrot = reinterpret_cast<double *>(p); break;
    }
    p += al256(bytes);
  });
  return ws;
}

namespace {
// One phase correlation of B pairs of H x W inputs.  mag_only: the row transforms and
// the forward column pass only, with the weighted magnitudes written to ws.mag.
fc_status pc_run(fc_ctx *ctx, const PixWs &ws, PcIn in, int B, int H, int W, bool mag_only,
                 double *shift_px, int32_t *peak, double *resp, int32_t *tok_shift, int tp,
                 bool zero_shift, hipStream_t st) {
  // the response surface goes to the caller's buffer or over the current-frame
  // half-spectra, which the forward column pass has consumed by then
  double *r = resp ? resp : reinterpret_cast<double *>(ws.sb);
  {
    ProfScope ps(ctx, st, "fc_pc_rows");
    hipLaunchKernelGGL(k_pc_rows, dim3((unsigned)H, (unsigned)B), dim3(kPcThreads), 0, st, in, H,
                       W, ws);
    FC_LAUNCH_OK(st, "k_pc_rows");
  }
  {
    ProfScope ps(ctx, st, "fc_pc_cols");
    double *mag = mag_only ? ws.mag : nullptr;
    if (H <= 224)
      launch_cols<224, 8>(H, W, B, ws, mag, mag_only, st);
    else if (H <= 448)
      launch_cols<448, 4>(H, W, B, ws, mag, mag_only, st);
    else
      launch_cols<896, 2>(H, W, B, ws, mag, mag_only, st);
    FC_LAUNCH_OK(st, "k_pc_cols");
  }
  if (mag_only) return FC_OK;
  {
    ProfScope ps(ctx, st, "fc_pc_rows_inv");
    hipLaunchKernelGGL(k_pc_rows_inv, dim3((unsigned)H, (unsigned)B), dim3(kPcThreads), 0, st, H,
                       W, ws, r);
    FC_LAUNCH_OK(st, "k_pc_rows_inv");
  }
  {
    ProfScope ps(ctx, st, "fc_pc_peak");
    hipLaunchKernelGGL(k_pc_peak, dim3((unsigned)B), dim3(kPcThreads), 0, st, H, W, ws,
                       (const double *)r, shift_px ? shift_px : ws.shift_px, peak, tok_shift, tp,
                       zero_shift ? 1 : 0);
    FC_LAUNCH_OK(st, "k_pc_peak");
  }
  return FC_OK;
}
}  // namespace

fc_status launch_pixel_pc(fc_ctx *ctx, const PixWs &ws, const float *prev, const float *cur,
                          int B, int H, int W, double *shift_px, int32_t *peak, double *resp,
                          int32_t *tok_shift, int tp, bool zero_shift, hipStream_t st) {
  if (!pix_size_ok(H) || !pix_size_ok(W))
    return fail(FC_ERR_UNSUPPORTED, "pixel phase correlation: H=%d, W=%d must be 7 * 2^k, 14..%d",
                H, W, kPcMaxN);
  return pc_run(ctx, ws, PcIn{prev, cur, nullptr, nullptr}, B, H, W, false, shift_px, peak, resp,
                tok_shift, tp, zero_shift, st);
}

fc_status launch_pixel_pc_rot(fc_ctx *ctx, const PixWs &ws, const float *prev, const float *cur,
                              int B, int H, int W, double *angle, double *shift_px,
                              int32_t *tok_shift, int tp, bool zero_shift, hipStream_t st) {
  if (!pix_rot_size_ok(H, W) || !ws.mag)
    return fail(FC_ERR_UNSUPPORTED, "rotation phase correlation: H=%d, W=%d must be 7 * 2^k with "
                "min(H, W) >= 28", H, W);
  const int NT = H, NR = std::min(H, W) / 2;
  fc_status s;
  // 1. weighted magnitude spectra of both frames
  if ((s = pc_run(ctx, ws, PcIn{prev, cur, nullptr, nullptr}, B, H, W, true, nullptr, nullptr,
                  nullptr, nullptr, 1, false, st)) != FC_OK)
    return s;
  // 2. their log-polar samples, correlated: the angular offset of the peak
  {
    ProfScope ps(ctx, st, "fc_lp_sample");
    hipLaunchKernelGGL(k_lp_sample, dim3((unsigned)NT, (unsigned)B), dim3(kPcThreads), 0, st,
                       (const double *)ws.mag, H, W, NT, NR, ws.lp);
    FC_LAUNCH_OK(st, "k_lp_sample");
  }
  if ((s = pc_run(ctx, ws, PcIn{nullptr, nullptr, ws.lp, ws.lp + (size_t)B * NT * NR}, B, NT, NR,
                  false, ws.shift_px, nullptr, nullptr, nullptr, 1, false, st)) != FC_OK)
    return s;
  // 3. the current frame rotated back, then the displacement of the image centre
  {
    ProfScope ps(ctx, st, "fc_derotate");
    hipLaunchKernelGGL(k_derotate, dim3((unsigned)H, (unsigned)B), dim3(kPcThreads), 0, st, cur, H,
                       W, (const double *)ws.shift_px, NT, ws.yrot, angle);
    FC_LAUNCH_OK(st, "k_derotate");
  }
  return pc_run(ctx, ws, PcIn{prev, nullptr, nullptr, ws.yrot}, B, H, W, false, shift_px, nullptr,
                nullptr, tok_shift, tp, zero_shift, st);
}

}  // namespace fc
