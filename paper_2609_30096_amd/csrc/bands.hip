// Frequency-band decomposition of the calibration disagreement: the guided
// difference d = p_S - p_L (Eqs. 1, 4) on the C x F x H x W latent, read
// straight from the two models' patch-token velocities, is transformed with
// orthonormal DFTs (spatially over (H, W) per (c, f) slice, temporally over F
// per (c, h, w) series) and its energy split into low / mid / high bands of
// the normalised frequency nu = 2|k'|/n (k' the signed frequency index):
// low nu < 1/3, mid nu < 2/3, high otherwise, the spatial nu being the radius
// over (H, W).  Band membership is decided in integer arithmetic.
//
// Passes (all on the caller's stream):
//   band_tables   twiddles exp(-2 pi i m / n) for the three axes (fp64 -> fp32)
//   band_row      per latent row: Y[h, k_w] = sum_w d[h, w] tw_W[k_w w]
//   band_col      per (slice, 32 columns): X[k_h, k_w] = sum_h Y[h, k_w] tw_H[k_h h],
//                 |X|^2 / (H W) accumulated per band (fp64), one partial per block
//   band_temporal per (c, h, w): the F-point DFT, |X|^2 / F per band, partials
//   band_finish   partials summed in a fixed order -> 6 energies (and scores)
// The work is a few GFLOP per call against multi-second denoiser steps, so the
// kernels favour simplicity over peak throughput; all reads of the velocities
// are 16 B contiguous (the 2x2 patch of one channel) or coalesced.
#include <math.h>

#include "common.h"
#include "kernels.h"

namespace track {

namespace {

constexpr int BAND_THREADS = 256;
constexpr int BAND_COLS = 32;     // spatial columns per band_col block
constexpr int BAND_MAX_W = 1024;  // row kernel LDS bound
constexpr int BAND_MAX_H = 256;   // column kernel LDS bound
constexpr int BAND_MAX_F = 64;    // temporal kernel LDS bound

inline unsigned blocks_for(int64_t n, int64_t per) { return (unsigned)((n + per - 1) / per); }
inline size_t align_256(size_t v) { return (v + 255) & ~(size_t)255; }

struct BandShape {
  int C, F, H, W, pt, ph, pw;
  int Hp, Wp, P;
};

// Offset of latent element (c, f, h, w) in the patch-token layout [L][P].
__device__ __forceinline__ int64_t tok_offset(const BandShape& s, int c, int f, int h, int w) {
  const int64_t l = ((int64_t)(f / s.pt) * s.Hp + h / s.ph) * s.Wp + w / s.pw;
  const int e = ((c * s.pt + f % s.pt) * s.ph + h % s.ph) * s.pw + w % s.pw;
  return l * s.P + e;
}

// Guided difference p_S - p_L at token-layout offset o (Eq. 1 per model).
__device__ __forceinline__ float guided_diff(const float* __restrict__ vL, const float* __restrict__ vS, int64_t n,
                                             int B, float w, int64_t o) {
  const float cL = vL[o], cS = vS[o];
  if (B == 2) {
    const float pL = fmaf(w, cL - vL[n + o], vL[n + o]);
    const float pS = fmaf(w, cS - vS[n + o], vS[n + o]);
    return pS - pL;
  }
  return cS - cL;
}

// |k'| of frequency index k on an axis of length n.
__device__ __forceinline__ int64_t fold(int k, int n) { return k <= n / 2 ? k : n - k; }

__device__ __forceinline__ int axis_band(int k, int n) {
  const int64_t a = fold(k, n);
  return 6 * a < n ? 0 : (3 * a < n ? 1 : 2);
}

// nu^2 / 4 * H^2 W^2 = a_h^2 W^2 + a_w^2 H^2 against (1/3)^2 and (2/3)^2.
__device__ __forceinline__ int spatial_band(int kh, int kw, int H, int W) {
  const int64_t ah = fold(kh, H), aw = fold(kw, W);
  const int64_t s = ah * ah * W * W + aw * aw * H * H;
  const int64_t hw2 = (int64_t)H * H * W * W;
  return 36 * s < hw2 ? 0 : (9 * s < hw2 ? 1 : 2);
}

// Block-wide sum of three doubles per thread; thread 0 writes them to out[0..2].
__device__ __forceinline__ void block_sum3(double a0, double a1, double a2, double* __restrict__ out) {
  __shared__ double red[3][BAND_THREADS / 64];
  a0 = wave_sum_d(a0);
  a1 = wave_sum_d(a1);
  a2 = wave_sum_d(a2);
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][wv] = a0;
    red[1][wv] = a1;
    red[2][wv] = a2;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int b = 0; b < 3; ++b) {
      double acc = 0.0;
      for (int i = 0; i < BAND_THREADS / 64; ++i) acc += red[b][i];
      out[b] = acc;
    }
  }
}

__global__ void band_tables_kernel(int W, int H, int F, float2* __restrict__ tw) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= W + H + F) return;
  const int n = i < W ? W : (i < W + H ? H : F);
  const int m = i < W ? i : (i < W + H ? i - W : i - W - H);
  double sn, cs;
  sincospi(2.0 * m / n, &sn, &cs);
  tw[i] = make_float2((float)cs, (float)-sn);
}

__global__ __launch_bounds__(BAND_THREADS) void band_row_kernel(BandShape s, int B, float w, const float* __restrict__ vL,
                                                               const float* __restrict__ vS, int64_t n,
                                                               const float2* __restrict__ twW, float2* __restrict__ Y) {
  __shared__ float drow[BAND_MAX_W];
  __shared__ float2 tw[BAND_MAX_W];
  const int h = blockIdx.x;
  const int sl = blockIdx.y;  // slice c * F + f
  const int c = sl / s.F, f = sl % s.F;
  for (int x = threadIdx.x; x < s.W; x += BAND_THREADS) {
    drow[x] = guided_diff(vL, vS, n, B, w, tok_offset(s, c, f, h, x));
    tw[x] = twW[x];
  }
  __syncthreads();
  float2* yrow = Y + ((int64_t)sl * s.H + h) * s.W;
  for (int kw = threadIdx.x; kw < s.W; kw += BAND_THREADS) {
    float re = 0.0f, im = 0.0f;
    int m = 0;  // kw * x mod W
    for (int x = 0; x < s.W; ++x) {
      const float2 t = tw[m];
      re = fmaf(drow[x], t.x, re);
      im = fmaf(drow[x], t.y, im);
      m += kw;
      if (m >= s.W) m -= s.W;
    }
    yrow[kw] = make_float2(re, im);
  }
}

__global__ __launch_bounds__(BAND_THREADS) void band_col_kernel(BandShape s, const float2* __restrict__ Y,
                                                               const float2* __restrict__ twH,
                                                               double* __restrict__ part) {
  __shared__ float2 ytile[BAND_MAX_H][BAND_COLS];
  __shared__ float2 tw[BAND_MAX_H];
  const int sl = blockIdx.y;
  const int kw0 = blockIdx.x * BAND_COLS;
  for (int i = threadIdx.x; i < s.H * BAND_COLS; i += BAND_THREADS) {
    const int h = i / BAND_COLS, j = i % BAND_COLS;
    ytile[h][j] = kw0 + j < s.W ? Y[((int64_t)sl * s.H + h) * s.W + kw0 + j] : make_float2(0.0f, 0.0f);
  }
  for (int i = threadIdx.x; i < s.H; i += BAND_THREADS) tw[i] = twH[i];
  __syncthreads();
  const double norm = 1.0 / ((double)s.H * s.W);
  double acc[3] = {0.0, 0.0, 0.0};
  for (int i = threadIdx.x; i < s.H * BAND_COLS; i += BAND_THREADS) {
    const int kh = i / BAND_COLS, j = i % BAND_COLS;
    const int kw = kw0 + j;
    if (kw >= s.W) continue;
    float re = 0.0f, im = 0.0f;
    int m = 0;  // kh * h mod H
    for (int h = 0; h < s.H; ++h) {
      const float2 y = ytile[h][j], t = tw[m];
      re = fmaf(y.x, t.x, fmaf(-y.y, t.y, re));
      im = fmaf(y.x, t.y, fmaf(y.y, t.x, im));
      m += kh;
      if (m >= s.H) m -= s.H;
    }
    const double e = ((double)re * re + (double)im * im) * norm;
    const int b = spatial_band(kh, kw, s.H, s.W);
    acc[0] += b == 0 ? e : 0.0;
    acc[1] += b == 1 ? e : 0.0;
    acc[2] += b == 2 ? e : 0.0;
  }
  block_sum3(acc[0], acc[1], acc[2], part + 3 * ((int64_t)blockIdx.y * gridDim.x + blockIdx.x));
}

// One thread per (c, h, w) series, numbered in the token order of one frame
// group so that neighbouring threads read neighbouring floats.
__global__ __launch_bounds__(BAND_THREADS) void band_temporal_kernel(BandShape s, int B, float w,
                                                                    const float* __restrict__ vL,
                                                                    const float* __restrict__ vS, int64_t n,
                                                                    const float2* __restrict__ twF,
                                                                    double* __restrict__ part) {
  __shared__ float ser[BAND_MAX_F][BAND_THREADS];
  __shared__ float2 tw[BAND_MAX_F];
  for (int i = threadIdx.x; i < s.F; i += BAND_THREADS) tw[i] = twF[i];
  const int64_t i = (int64_t)blockIdx.x * BAND_THREADS + threadIdx.x;
  const int Q = s.C * s.ph * s.pw;
  const int64_t total = (int64_t)s.Hp * s.Wp * Q;
  const bool live = i < total;
  int c = 0, h = 0, x = 0;
  if (live) {
    const int64_t lp = i / Q;
    const int e = (int)(i % Q);
    const int iw = e % s.pw, ih = (e / s.pw) % s.ph;
    c = e / (s.ph * s.pw);
    h = (int)(lp / s.Wp) * s.ph + ih;
    x = (int)(lp % s.Wp) * s.pw + iw;
    for (int f = 0; f < s.F; ++f) ser[f][threadIdx.x] = guided_diff(vL, vS, n, B, w, tok_offset(s, c, f, h, x));
  }
  __syncthreads();
  double acc[3] = {0.0, 0.0, 0.0};
  if (live) {
    const double norm = 1.0 / s.F;
    for (int kf = 0; kf < s.F; ++kf) {
      float re = 0.0f, im = 0.0f;
      int m = 0;  // kf * f mod F
      for (int f = 0; f < s.F; ++f) {
        const float d = ser[f][threadIdx.x];
        const float2 t = tw[m];
        re = fmaf(d, t.x, re);
        im = fmaf(d, t.y, im);
        m += kf;
        if (m >= s.F) m -= s.F;
      }
      const double e = ((double)re * re + (double)im * im) * norm;
      const int b = axis_band(kf, s.F);
      acc[0] += b == 0 ? e : 0.0;
      acc[1] += b == 1 ? e : 0.0;
      acc[2] += b == 2 ? e : 0.0;
    }
  }
  block_sum3(acc[0], acc[1], acc[2], part + 3 * (int64_t)blockIdx.x);
}

// Sums the partials in a fixed order.  energy[0..2] spatial, [3..5] temporal.
// With step partials (pairs (sum d^2, sum p_L^2) of the calibration step
// kernel) it also writes score[b] = sqrt(energy[b]) / max(||p_L||, eps).
__global__ __launch_bounds__(BAND_THREADS) void band_finish_kernel(int ns, const double* __restrict__ part_s, int nt,
                                                                  const double* __restrict__ part_t, int nstep,
                                                                  const double* __restrict__ step_part, double eps,
                                                                  double* __restrict__ energy,
                                                                  double* __restrict__ score) {
  __shared__ double tot[7];
  for (int q = 0; q < 7; ++q) {
    const double* p = q < 3 ? part_s + q : (q < 6 ? part_t + (q - 3) : step_part + 1);
    const int cnt = q < 3 ? ns : (q < 6 ? nt : nstep);
    const int stride = q < 6 ? 3 : 2;
    double a = 0.0;
    if (q < 6 || step_part)
      for (int i = threadIdx.x; i < cnt; i += BAND_THREADS) a += p[(int64_t)i * stride];
    __shared__ double red[BAND_THREADS / 64];
    a = wave_sum_d(a);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = a;
    __syncthreads();
    if (threadIdx.x == 0) {
      double s = 0.0;
      for (int i = 0; i < BAND_THREADS / 64; ++i) s += red[i];
      tot[q] = s;
    }
    __syncthreads();
  }
  if (threadIdx.x < 6) {
    energy[threadIdx.x] = tot[threadIdx.x];
    if (step_part && score) {
      const double dn = sqrt(tot[6]);
      score[threadIdx.x] = sqrt(tot[threadIdx.x]) / (dn > eps ? dn : eps);
    }
  }
}

struct BandLayout {
  size_t Y, tw, part_s, part_t, energy, total;
  int col_blocks, ns, nt;
};

BandLayout band_layout(const BandShape& s) {
  BandLayout b{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align_256(off + bytes);
    return o;
  };
  b.col_blocks = (s.W + BAND_COLS - 1) / BAND_COLS;
  b.ns = b.col_blocks * s.C * s.F;
  b.nt = (int)(((int64_t)s.Hp * s.Wp * s.C * s.ph * s.pw + BAND_THREADS - 1) / BAND_THREADS);
  b.Y = take((size_t)s.C * s.F * s.H * s.W * sizeof(float2));
  b.tw = take((size_t)(s.W + s.H + s.F) * sizeof(float2));
  b.part_s = take((size_t)b.ns * 3 * 8);
  b.part_t = take((size_t)b.nt * 3 * 8);
  b.energy = take(6 * 8);
  b.total = off;
  return b;
}

BandShape make_shape(int C, int F, int H, int W, int pt, int ph, int pw) {
  BandShape s{C, F, H, W, pt, ph, pw, H / ph, W / pw, C * pt * ph * pw};
  return s;
}

}  // namespace

track_status band_check(int C, int F, int H, int W, int pt, int ph, int pw) {
  if (C < 1 || F < 1 || H < 1 || W < 1 || pt < 1 || ph < 1 || pw < 1)
    return fail(TRACK_E_SHAPE, "bands: bad latent %dx%dx%dx%d or patch %dx%dx%d", C, F, H, W, pt, ph, pw);
  if (F % pt || H % ph || W % pw) return fail(TRACK_E_SHAPE, "bands: latent not divisible by the patch");
  if (W > BAND_MAX_W || H > BAND_MAX_H || F > BAND_MAX_F)
    return fail(TRACK_E_UNSUPPORTED, "bands: supports W <= %d, H <= %d, F <= %d (got %d, %d, %d)", BAND_MAX_W,
                BAND_MAX_H, BAND_MAX_F, W, H, F);
  if ((int64_t)C * F * H * W > ((int64_t)1 << 31)) return fail(TRACK_E_UNSUPPORTED, "bands: latent too large");
  return TRACK_OK;
}

size_t band_workspace_bytes(int C, int F, int H, int W, int pt, int ph, int pw) {
  return band_layout(make_shape(C, F, H, W, pt, ph, pw)).total;
}

size_t band_energy_offset(int C, int F, int H, int W, int pt, int ph, int pw) {
  return band_layout(make_shape(C, F, H, W, pt, ph, pw)).energy;
}

track_status band_scores(int C, int F, int H, int W, int pt, int ph, int pw, int B, float w, const float* vel_L,
                         const float* vel_S, const double* step_partial, int64_t n_step_partials, double eps, void* ws,
                         double* energy_dev, double* score_dev, hipStream_t st) {
  {
    const track_status c = band_check(C, F, H, W, pt, ph, pw);
    if (c != TRACK_OK) return c;
  }
  if (B != 1 && B != 2) return fail(TRACK_E_INVALID, "bands: batch must be 1 or 2");
  if (!vel_L || !vel_S || !ws) return fail(TRACK_E_INVALID, "bands: null pointer");
  const BandShape s = make_shape(C, F, H, W, pt, ph, pw);
  const BandLayout L = band_layout(s);
  uint8_t* base = (uint8_t*)ws;
  float2* Y = (float2*)(base + L.Y);
  float2* tw = (float2*)(base + L.tw);
  double* part_s = (double*)(base + L.part_s);
  double* part_t = (double*)(base + L.part_t);
  double* energy = energy_dev ? energy_dev : (double*)(base + L.energy);
  const int64_t n = (int64_t)C * F * H * W;  // floats per branch
  ProfScope prof(TRACK_PROF_STEP, st);
  band_tables_kernel<<<blocks_for(W + H + F, 256), 256, 0, st>>>(W, H, F, tw);
  TRACK_LAUNCH_CHECK();
  band_row_kernel<<<dim3(H, C * F), BAND_THREADS, 0, st>>>(s, B, w, vel_L, vel_S, n, tw, Y);
  TRACK_LAUNCH_CHECK();
  band_col_kernel<<<dim3(L.col_blocks, C * F), BAND_THREADS, 0, st>>>(s, Y, tw + W, part_s);
  TRACK_LAUNCH_CHECK();
  band_temporal_kernel<<<L.nt, BAND_THREADS, 0, st>>>(s, B, w, vel_L, vel_S, n, tw + W + H, part_t);
  TRACK_LAUNCH_CHECK();
  band_finish_kernel<<<1, BAND_THREADS, 0, st>>>(L.ns, part_s, L.nt, part_t, (int)n_step_partials, step_partial, eps,
                                                energy, score_dev);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

}  // namespace track
