// Memory-bound kernels of the denoiser step: layout changes at the boundary,
// timestep features and modulation, LayerNorm with adaLN modulation,
// RMSNorm with 3D RoPE, the V transpose feeding the attention kernel, and the
// fused guidance + Euler (+ disagreement) step.  All stream rows with 8- or
// 16-byte vector accesses; reductions use a fixed order (no atomics), so
// every result is bit-reproducible.
#include <math.h>

#include <type_traits>

#include <mutex>

#include "common.h"
#include "kernels.h"

namespace track {

static inline unsigned cdiv(int64_t a, int64_t b) { return (unsigned)((a + b - 1) / b); }

// ------------------------------------------------------------------ patchify / unpatchify
// Token l = (f' H' + h') W' + w', entry e = ((c pt + i_t) ph + i_h) pw + i_w.
__device__ __forceinline__ int64_t latent_index(int64_t l, int e, int C, int F, int H, int W, int pt, int ph, int pw) {
  const int Hp = H / ph, Wp = W / pw;
  const int wq = (int)(l % Wp);
  const int hq = (int)((l / Wp) % Hp);
  const int fq = (int)(l / ((int64_t)Wp * Hp));
  const int iw = e % pw;
  const int ih = (e / pw) % ph;
  const int it = (e / (pw * ph)) % pt;
  const int c = e / (pw * ph * pt);
  return (((int64_t)c * F + (fq * pt + it)) * H + (hq * ph + ih)) * W + (wq * pw + iw);
}

__global__ void patchify_kernel(const float* __restrict__ x, float* __restrict__ tok, int64_t n, int P, int C, int F,
                                int H, int W, int pt, int ph, int pw) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  tok[i] = x[latent_index(i / P, (int)(i % P), C, F, H, W, pt, ph, pw)];
}

__global__ void unpatchify_kernel(const float* __restrict__ tok, float* __restrict__ x, int64_t n, int C, int F, int H,
                                  int W, int pt, int ph, int pw) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  // invert latent_index for output element i
  const int w = (int)(i % W);
  const int h = (int)((i / W) % H);
  const int f = (int)((i / ((int64_t)W * H)) % F);
  const int c = (int)(i / ((int64_t)W * H * F));
  const int Hp = H / ph, Wp = W / pw;
  const int64_t l = ((int64_t)(f / pt) * Hp + h / ph) * Wp + w / pw;
  const int e = ((c * pt + f % pt) * ph + h % ph) * pw + w % pw;
  x[i] = tok[l * ((int64_t)C * pt * ph * pw) + e];
}

track_status patchify(const float* x, float* tok, int C, int F, int H, int W, int pt, int ph, int pw, hipStream_t s) {
  const int64_t n = (int64_t)C * F * H * W;
  patchify_kernel<<<cdiv(n, 256), 256, 0, s>>>(x, tok, n, C * pt * ph * pw, C, F, H, W, pt, ph, pw);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

track_status unpatchify(const float* tok, float* x, int C, int F, int H, int W, int pt, int ph, int pw, hipStream_t s) {
  const int64_t n = (int64_t)C * F * H * W;
  unpatchify_kernel<<<cdiv(n, 256), 256, 0, s>>>(tok, x, n, C, F, H, W, pt, ph, pw);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

__global__ void to_bf16_kernel(const float* __restrict__ src, bf16_t* __restrict__ dst, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = f2bf(src[i]);
}

track_status to_bf16(const float* src, bf16_t* dst, int64_t n, hipStream_t s) {
  to_bf16_kernel<<<cdiv(n, 256), 256, 0, s>>>(src, dst, n);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ timestep features and modulation
// [cos(t w_j), sin(t w_j)], w_j = 10000^(-j/half), evaluated in float64.
__global__ void sinusoid_kernel(double t, int half, float* out) {
  for (int j = threadIdx.x; j < half; j += blockDim.x) {
    const double w = pow(10000.0, -(double)j / (double)half);
    const double a = t * w;
    out[j] = (float)cos(a);
    out[half + j] = (float)sin(a);
  }
}

track_status sinusoid(double t, int dim, float* out, hipStream_t s) {
  sinusoid_kernel<<<1, 256, 0, s>>>(t, dim / 2, out);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// One wave per output row; y = act(W x + b), optionally y_silu = silu(y).
template <typename T>
__global__ __launch_bounds__(256) void gemv_kernel(int N, int K, const T* __restrict__ W, const T* __restrict__ b,
                                                   const float* __restrict__ x, float* __restrict__ y,
                                                   float* __restrict__ y_silu, int post_silu) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  const T* row = W + (int64_t)n * K;
  float acc = 0.0f;
  if constexpr (sizeof(T) == 2) {
    for (int k0 = lane * 8; k0 < K; k0 += 512) {
      const u32x4 v = *(const u32x4*)(row + k0);
      const f32x4 x0 = *(const f32x4*)(x + k0);
      const f32x4 x1 = *(const f32x4*)(x + k0 + 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        acc = fmaf(__uint_as_float(v[j] << 16), j < 2 ? x0[2 * j] : x1[2 * j - 4], acc);
        acc = fmaf(__uint_as_float(v[j] & 0xffff0000u), j < 2 ? x0[2 * j + 1] : x1[2 * j - 3], acc);
      }
    }
  } else {
    for (int k = lane; k < K; k += 64) acc = fmaf(ldf(row + k), x[k], acc);
  }
  acc = wave_sum(acc);
  if (lane == 0) {
    float v = acc + ldf(b + n);
    if (post_silu) v = silu(v);
    y[n] = v;
    if (y_silu) y_silu[n] = silu(v);
  }
}

track_status gemv(int dtype, int N, int K, const void* W, const void* b, const float* x, float* y, float* y_silu,
                  int post_silu, hipStream_t s) {
  if (dtype == TRACK_DTYPE_BF16) {
    if (K % 8) return fail(TRACK_E_UNSUPPORTED, "gemv: K %% 8 != 0");
    gemv_kernel<bf16_t><<<cdiv(N, 4), 256, 0, s>>>(N, K, (const bf16_t*)W, (const bf16_t*)b, x, y, y_silu, post_silu);
  } else {
    gemv_kernel<float><<<cdiv(N, 4), 256, 0, s>>>(N, K, (const float*)W, (const float*)b, x, y, y_silu, post_silu);
  }
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

template <typename T>
__global__ void mod_tables_kernel(int blocks, int n6, const float* __restrict__ m, const T* __restrict__ Tb,
                                  int64_t stride, float* __restrict__ mods) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)blocks * n6) return;
  const int blk = (int)(i / n6), j = (int)(i % n6);
  mods[i] = m[j] + ldf(Tb + blk * stride + j);
}

track_status mod_tables(int dtype, int blocks, int d, const float* m, const void* Tbase, int64_t stride_elems,
                        float* mods, hipStream_t s) {
  const int64_t n = (int64_t)blocks * 6 * d;
  if (n == 0) return TRACK_OK;
  if (dtype == TRACK_DTYPE_BF16)
    mod_tables_kernel<bf16_t><<<cdiv(n, 256), 256, 0, s>>>(blocks, 6 * d, m, (const bf16_t*)Tbase, stride_elems, mods);
  else
    mod_tables_kernel<float><<<cdiv(n, 256), 256, 0, s>>>(blocks, 6 * d, m, (const float*)Tbase, stride_elems, mods);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

template <typename T>
__global__ void head_mod_kernel(int d, const float* __restrict__ e, const T* __restrict__ Tt, float* __restrict__ out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < 2 * d) out[i] = ldf(Tt + i) + e[i % d];
}

track_status head_mod(int dtype, int d, const float* e, const void* T, float* out, hipStream_t s) {
  if (dtype == TRACK_DTYPE_BF16)
    head_mod_kernel<bf16_t><<<cdiv(2 * d, 256), 256, 0, s>>>(d, e, (const bf16_t*)T, out);
  else
    head_mod_kernel<float><<<cdiv(2 * d, 256), 256, 0, s>>>(d, e, (const float*)T, out);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ RoPE tables
// Sections of one head: frame n0 = dh - 4 (dh / 6), height and width n1 = n2 = 2 (dh / 6).
__host__ __device__ __forceinline__ void rope_widths(int dh, int n[3]) {
  n[1] = n[2] = 2 * (dh / 6);
  n[0] = dh - 2 * n[1];
}

__global__ void rope_tables_kernel(int dh, int E0, int E1, int E2, float* cos_t, float* sin_t) {
  int n[3];
  rope_widths(dh, n);
  const int E[3] = {E0, E1, E2};
  int off = 0;
  for (int a = 0; a < 3; ++a) {
    const int half = n[a] / 2;
    for (int i = threadIdx.x; i < E[a] * half; i += blockDim.x) {
      const int pos = i / half, p = i % half;
      const double ang = (double)pos * pow(10000.0, -2.0 * (double)p / (double)n[a]);
      cos_t[off + i] = (float)cos(ang);
      sin_t[off + i] = (float)sin(ang);
    }
    off += E[a] * half;
  }
}

track_status rope_tables(int head_dim, Grid3 g, float* cos_t, float* sin_t, hipStream_t s) {
  rope_tables_kernel<<<1, 256, 0, s>>>(head_dim, g.f, g.h, g.w, cos_t, sin_t);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ LayerNorm + adaLN modulation
// One wave per row; the row is held in registers as NC float4 chunks per
// lane (NC chosen per width at launch, so short rows keep occupancy high).
constexpr int NORM_MAXC = 32;  // widths up to 64 * 4 * 32 = 8192

template <typename T>
__device__ __forceinline__ void store4(T* p, float a, float b, float c, float d) {
  if constexpr (sizeof(T) == 2) {
    u32x2 v;
    v[0] = pack_bf2(a, b);
    v[1] = pack_bf2(c, d);
    *(u32x2*)p = v;
  } else {
    *(f32x4*)p = f32x4{a, b, c, d};
  }
}

// Rows are spread over WPR waves (1, or 4 = the whole 256-thread workgroup):
// thread t of a row owns float4 chunks t, t + 64 WPR, ...  A workgroup-wide
// row kernel takes RPB rows at once, so each thread keeps more loads in
// flight.  Row sums are a wave reduction, then (WPR 4) the four waves'
// partials added in wave order through LDS, the same order in every thread.
template <int WPR, int RPB>
__device__ __forceinline__ void row_sums(float (&v)[RPB], float* red /* [RPB][4] */) {
#pragma unroll
  for (int r = 0; r < RPB; ++r) v[r] = wave_sum(v[r]);
  if constexpr (WPR > 1) {
    if ((threadIdx.x & 63) == 0) {
#pragma unroll
      for (int r = 0; r < RPB; ++r) red[4 * r + (threadIdx.x >> 6)] = v[r];
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < RPB; ++r) v[r] = (red[4 * r] + red[4 * r + 1]) + (red[4 * r + 2] + red[4 * r + 3]);
  }
}

// First row of this wave (WPR 1) or workgroup (WPR 4).
template <int WPR, int RPB>
__device__ __forceinline__ int64_t norm_row0() {
  return WPR == 1 ? ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * RPB : (int64_t)blockIdx.x * RPB;
}

template <typename T, int NC, int WPR, int RPB>
__global__ __launch_bounds__(256) void layernorm_kernel(int64_t rows, int d, const float* __restrict__ x,
                                                        const float* __restrict__ scale,
                                                        const float* __restrict__ shift, T* __restrict__ y) {
  static_assert((WPR == 1 && RPB == 1) || WPR == 4, "one wave per row, or a workgroup per RPB rows");
  __shared__ float red[2][4 * RPB];
  constexpr int CS = 64 * WPR;  // chunk stride between a thread's chunks
  const int t = WPR == 1 ? (threadIdx.x & 63) : threadIdx.x;
  const int64_t row0 = norm_row0<WPR, RPB>();
  if (row0 >= rows) return;  // wave-uniform (WPR 1), or the whole workgroup
  const int nc = d >> 2;     // float4 chunks in a row
  f32x4 v[RPB][NC];
  float sum[RPB];
#pragma unroll
  for (int r = 0; r < RPB; ++r) {
    sum[r] = 0.0f;
    if (row0 + r < rows) {  // workgroup-uniform
      const float* xr = x + (row0 + r) * d;
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int ch = t + CS * i;
        if (ch < nc) {
          v[r][i] = *(const f32x4*)(xr + 4 * ch);
          sum[r] += (v[r][i][0] + v[r][i][1]) + (v[r][i][2] + v[r][i][3]);
        }
      }
    }
  }
  row_sums<WPR, RPB>(sum, red[0]);
  float sq[RPB];
#pragma unroll
  for (int r = 0; r < RPB; ++r) {
    const float mean = sum[r] / (float)d;
    sq[r] = 0.0f;
    if (row0 + r < rows) {
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int ch = t + CS * i;
        if (ch < nc) {
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            v[r][i][j] -= mean;
            sq[r] = fmaf(v[r][i][j], v[r][i][j], sq[r]);
          }
        }
      }
    }
  }
  row_sums<WPR, RPB>(sq, red[1]);
#pragma unroll
  for (int r = 0; r < RPB; ++r) {
    if (row0 + r >= rows) break;
    const float rstd = 1.0f / sqrtf(sq[r] / (float)d + 1e-6f);
    T* yr = y + (row0 + r) * d;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int ch = t + CS * i;
      if (ch < nc) {
        f32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = v[r][i][j] * rstd;
        if (scale) {
          const f32x4 sc = *(const f32x4*)(scale + 4 * ch);
          const f32x4 sh = *(const f32x4*)(shift + 4 * ch);
#pragma unroll
          for (int j = 0; j < 4; ++j) o[j] = fmaf(o[j], 1.0f + sc[j], sh[j]);
        }
        store4(yr + 4 * ch, o[0], o[1], o[2], o[3]);
      }
    }
  }
}

// Smallest compiled chunk count covering `need` float4 chunks per lane.
template <template <int> class Launch>
static void dispatch_chunks(int need) {
  if (need <= 1) Launch<1>::run();
  else if (need <= 2) Launch<2>::run();
  else if (need <= 3) Launch<3>::run();
  else if (need <= 4) Launch<4>::run();
  else if (need <= 6) Launch<6>::run();
  else if (need <= 8) Launch<8>::run();
  else if (need <= 12) Launch<12>::run();
  else if (need <= 16) Launch<16>::run();
  else if (need <= 20) Launch<20>::run();
  else if (need <= 24) Launch<24>::run();
  else Launch<NORM_MAXC>::run();
}

struct LnArgs {
  int dtype;
  int64_t rows;
  int d;
  const float *x, *scale, *shift;
  void* y;
  hipStream_t s;
};
static thread_local LnArgs g_ln;

template <int WPR, int RPB>
struct LnLaunchW {
  template <int NC>
  struct L {
    static void run() {
      const LnArgs& a = g_ln;
      const unsigned grid = (unsigned)(WPR == 1 ? (a.rows + 3) / 4 : (a.rows + RPB - 1) / RPB);
      if (a.dtype == TRACK_DTYPE_BF16)
        layernorm_kernel<bf16_t, NC, WPR, RPB>
            <<<grid, 256, 0, a.s>>>(a.rows, a.d, a.x, a.scale, a.shift, (bf16_t*)a.y);
      else
        layernorm_kernel<float, NC, WPR, RPB><<<grid, 256, 0, a.s>>>(a.rows, a.d, a.x, a.scale, a.shift, (float*)a.y);
    }
  };
};

// Rows wider than this are split over a whole workgroup: a wave alone would
// keep too few bytes of its row in flight.  LayerNorm takes one row per
// workgroup (two float32 rows cost it occupancy), RMSNorm two (its bfloat16
// rows are half the registers).
constexpr int NORM_WIDE = 2048;

track_status layernorm(int dtype, int64_t rows, int d, const float* x, const float* scale, const float* shift, void* y,
                       hipStream_t s) {
  if (d % 4 || d > 256 * NORM_MAXC) return fail(TRACK_E_UNSUPPORTED, "layernorm: width %d unsupported", d);
  if ((scale == nullptr) != (shift == nullptr)) return fail(TRACK_E_INVALID, "layernorm: scale and shift go together");
  if (rows <= 0) return TRACK_OK;
  ProfScope prof(TRACK_PROF_NORM, s);
  g_ln = LnArgs{dtype, rows, d, x, scale, shift, y, s};
  if (d > NORM_WIDE)
    dispatch_chunks<LnLaunchW<4, 1>::L>((d / 4 + 255) / 256);
  else
    dispatch_chunks<LnLaunchW<1, 1>::L>((d / 4 + 63) / 64);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ RMSNorm + 3D RoPE
// Rows are segments of width d = heads * dh at column col0 of rows of stride
// ld, spread over threads as in the LayerNorm kernel in chunks of E elements
// (8 bfloat16 or 4 float32 values: 16-byte accesses); each is normalised by
// its RMS over d, scaled by g, then (if cos_t) each pair (2i, 2i+1) of a
// head is rotated by its section's angle.
template <typename T, int E>
struct RawOf;
template <>
struct RawOf<bf16_t, 8> {
  typedef u32x4 type;
};
template <>
struct RawOf<bf16_t, 4> {
  typedef u32x2 type;
};
template <>
struct RawOf<float, 4> {
  typedef f32x4 type;
};

template <typename T, int E>
__device__ __forceinline__ void unpack_raw(const typename RawOf<T, E>::type& r, float (&f)[E]) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int k = 0; k < E / 2; ++k) {
      f[2 * k] = __uint_as_float(r[k] << 16);
      f[2 * k + 1] = __uint_as_float(r[k] & 0xffff0000u);
    }
  } else {
#pragma unroll
    for (int k = 0; k < E; ++k) f[k] = r[k];
  }
}

template <typename T, int E>
__device__ __forceinline__ typename RawOf<T, E>::type pack_raw(const float (&f)[E]) {
  typename RawOf<T, E>::type r;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int k = 0; k < E / 2; ++k) r[k] = pack_bf2(f[2 * k], f[2 * k + 1]);
  } else {
#pragma unroll
    for (int k = 0; k < E; ++k) r[k] = f[k];
  }
  return r;
}

// With g2, every row holds two adjacent segments (columns col0 .. col0 + d
// with gain g, then col0 + d .. col0 + 2d with gain g2: q and k of the QKV
// rows), treated as 2 rows virtual rows, q then k of each row in turn.
// qscale multiplies the first (or only) segment before its rounding: the
// forward writes q in the attention kernel's log2 units this way.
template <typename T, int E, int NC, int WPR, int RPB>
__global__ __launch_bounds__(256) void rmsnorm_rope_kernel(int64_t rows, int d, int dh, T* __restrict__ buf,
                                                           int64_t ld, int64_t col0, const T* __restrict__ g,
                                                           const T* __restrict__ g2,
                                                           const float* __restrict__ cos_t,
                                                           const float* __restrict__ sin_t, int Gf, int Gh, int Gw,
                                                           int64_t L, float qscale) {
  static_assert(WPR == 1 || WPR == 4, "RPB rows per wave, or per workgroup");
  typedef typename RawOf<T, E>::type Raw;
  __shared__ float red[4 * RPB];
  constexpr int CS = 64 * WPR;  // chunk stride between a thread's chunks
  const int t = WPR == 1 ? (threadIdx.x & 63) : threadIdx.x;
  const int64_t row0 = norm_row0<WPR, RPB>();
  if (row0 >= rows) return;  // wave-uniform (WPR 1), or the whole workgroup
  const int nc = d / E;
  // Rows stay in registers between the two passes in their storage type
  // (bfloat16 rows packed: half the registers, more waves in flight).
  Raw v[RPB][NC];
  float sq[RPB];
#pragma unroll
  for (int r = 0; r < RPB; ++r) {
    sq[r] = 0.0f;
    if (row0 + r < rows) {  // workgroup-uniform
      const int64_t vr = row0 + r;
      const T* xr = g2 ? buf + (vr >> 1) * ld + col0 + (vr & 1) * d : buf + vr * ld + col0;
#pragma unroll
      for (int i = 0; i < NC; ++i) {
        const int ch = t + CS * i;
        if (ch < nc) {
          v[r][i] = *(const Raw*)(xr + E * ch);
          float f[E];
          unpack_raw<T, E>(v[r][i], f);
#pragma unroll
          for (int j = 0; j < E; ++j) sq[r] = fmaf(f[j], f[j], sq[r]);
        }
      }
    }
  }
  row_sums<WPR, RPB>(sq, red);
  int n[3];
  rope_widths(dh, n);
  const int h0 = n[0] / 2, h1 = n[1] / 2, h2 = n[2] / 2;
  const int off1 = Gf * h0, off2 = off1 + Gh * h1;
  // When dh divides the E CS elements between a thread's chunks, its E
  // elements sit at the same offset of their head in every chunk, so its
  // rotation angles are loaded once per row instead of once per chunk.
  const bool lane_fixed = cos_t && ((E * CS) % dh) == 0;
#pragma unroll
  for (int r = 0; r < RPB; ++r) {
    const int64_t vrow = row0 + r;
    if (vrow >= rows) break;
    const int64_t row = g2 ? vrow >> 1 : vrow;
    const int seg = g2 ? (int)(vrow & 1) : 0;
    const T* gs = seg ? g2 : g;
    const float rstd = (1.0f / sqrtf(sq[r] / (float)d + 1e-6f)) * (seg ? 1.0f : qscale);
    int pos[3] = {0, 0, 0};
    if (cos_t) {
      const int64_t l = row % L;
      pos[2] = (int)(l % Gw);
      pos[1] = (int)((l / Gw) % Gh);
      pos[0] = (int)(l / ((int64_t)Gw * Gh));
    }
    auto table_index = [&](int p) {  // p: pair index within the head
      if (p < h0) return pos[0] * h0 + p;
      if (p < h0 + h1) return off1 + pos[1] * h1 + (p - h0);
      return off2 + pos[2] * h2 + (p - h0 - h1);
    };
    float cf[E / 2], sf[E / 2];
#pragma unroll
    for (int pr = 0; pr < E / 2; ++pr) {
      cf[pr] = 1.0f;
      sf[pr] = 0.0f;
    }
    if (lane_fixed) {
#pragma unroll
      for (int pr = 0; pr < E / 2; ++pr) {
        const int idx = table_index(((E * t) % dh) / 2 + pr);
        cf[pr] = cos_t[idx];
        sf[pr] = sin_t[idx];
      }
    }
    T* xr = buf + row * ld + col0 + (int64_t)seg * d;
#pragma unroll
    for (int i = 0; i < NC; ++i) {
      const int ch = t + CS * i;
      if (ch < nc) {
        float gv[E], o[E];
        unpack_raw<T, E>(*(const Raw*)(gs + E * ch), gv);
        unpack_raw<T, E>(v[r][i], o);
#pragma unroll
        for (int j = 0; j < E; ++j) o[j] = o[j] * rstd * gv[j];
        if (cos_t) {
#pragma unroll
          for (int pr = 0; pr < E / 2; ++pr) {
            float c = cf[pr], s = sf[pr];
            if (!lane_fixed) {
              const int idx = table_index(((E * ch) % dh) / 2 + pr);
              c = cos_t[idx];
              s = sin_t[idx];
            }
            const float a = o[2 * pr], b = o[2 * pr + 1];
            o[2 * pr] = a * c - b * s;
            o[2 * pr + 1] = a * s + b * c;
          }
        }
        *(Raw*)(xr + E * ch) = pack_raw<T, E>(o);
      }
    }
  }
}

struct RmsArgs {
  int dtype;
  int64_t rows;
  int heads, head_dim;
  void* buf;
  int64_t ld, col0;
  const void *g, *g2;
  const float *cos_t, *sin_t;
  Grid3 grid;
  int64_t L;
  hipStream_t s;
  float qscale;
};
static thread_local RmsArgs g_rms;

template <int E, int WPR, int RPB>
struct RmsLaunchW {
  template <int NC>
  struct L {
    static void run() {
      const RmsArgs& a = g_rms;
      const int64_t vrows = a.g2 ? 2 * a.rows : a.rows;
      const unsigned grid = (unsigned)(WPR == 1 ? (vrows + 4 * RPB - 1) / (4 * RPB) : (vrows + RPB - 1) / RPB);
      const int d = a.heads * a.head_dim;
      if constexpr (E == 8) {
        rmsnorm_rope_kernel<bf16_t, 8, NC, WPR, RPB><<<grid, 256, 0, a.s>>>(
            vrows, d, a.head_dim, (bf16_t*)a.buf, a.ld, a.col0, (const bf16_t*)a.g, (const bf16_t*)a.g2, a.cos_t,
            a.sin_t, a.grid.f, a.grid.h, a.grid.w, a.L, a.qscale);
      } else {
        if (a.dtype == TRACK_DTYPE_BF16)
          rmsnorm_rope_kernel<bf16_t, 4, NC, WPR, RPB><<<grid, 256, 0, a.s>>>(
              vrows, d, a.head_dim, (bf16_t*)a.buf, a.ld, a.col0, (const bf16_t*)a.g, (const bf16_t*)a.g2, a.cos_t,
              a.sin_t, a.grid.f, a.grid.h, a.grid.w, a.L, a.qscale);
        else
          rmsnorm_rope_kernel<float, 4, NC, WPR, RPB><<<grid, 256, 0, a.s>>>(
              vrows, d, a.head_dim, (float*)a.buf, a.ld, a.col0, (const float*)a.g, (const float*)a.g2, a.cos_t,
              a.sin_t, a.grid.f, a.grid.h, a.grid.w, a.L, a.qscale);
      }
    }
  };
};

track_status rmsnorm_rope(int dtype, int64_t rows, int heads, int head_dim, void* buf, int64_t ld, int64_t col0,
                          const void* g, const void* g2, const float* cos_t, const float* sin_t, Grid3 grid, int64_t L,
                          hipStream_t s, float qscale) {
  const int d = heads * head_dim;
  if (g2 && ld < col0 + 2 * (int64_t)d) return fail(TRACK_E_SHAPE, "rmsnorm_rope: two segments need ld >= col0 + 2d");
  if (head_dim % 4 || d > 256 * NORM_MAXC) return fail(TRACK_E_UNSUPPORTED, "rmsnorm_rope: width %d unsupported", d);
  if (cos_t && (int64_t)grid.f * grid.h * grid.w != L) return fail(TRACK_E_SHAPE, "rmsnorm_rope: grid != L");
  if (rows <= 0) return TRACK_OK;
  ProfScope prof(TRACK_PROF_NORM, s);
  g_rms = RmsArgs{dtype, rows, heads, head_dim, buf, ld, col0, g, g2, cos_t, sin_t, grid, L > 0 ? L : 1, s, qscale};
  // bfloat16 rows move in 16-byte chunks of 8 elements when the width allows
  // (a chunk must not straddle two heads: head_dim % 8 == 0)
  const bool wide_chunks = dtype == TRACK_DTYPE_BF16 && head_dim % 8 == 0 &&
                           ((uintptr_t)buf & 15) == 0 && ((uintptr_t)g & 15) == 0 && (!g2 || ((uintptr_t)g2 & 15) == 0) &&
                           ld % 8 == 0 && col0 % 8 == 0;
  if (wide_chunks) {
    if (d > NORM_WIDE)
      dispatch_chunks<RmsLaunchW<8, 4, 2>::L>((d / 8 + 255) / 256);
    else
      dispatch_chunks<RmsLaunchW<8, 1, 1>::L>((d / 8 + 63) / 64);
  } else if (d > NORM_WIDE) {
    dispatch_chunks<RmsLaunchW<4, 4, 2>::L>((d / 4 + 255) / 256);
  } else {
    dispatch_chunks<RmsLaunchW<4, 1, 1>::L>((d / 4 + 63) / 64);
  }
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ zero columns
__global__ __launch_bounds__(256) void zero_cols_kernel(bf16_t* __restrict__ p, int64_t rows, int64_t ld, int64_t c0,
                                                        int64_t nc) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= rows * nc) return;
  const int64_t r = i / nc, c = i - r * nc;
  p[r * ld + c0 + c] = bf16_t(0);
}

track_status zero_cols_bf16(void* p, int64_t rows, int64_t ld, int64_t c0, int64_t c1, hipStream_t s) {
  if (rows <= 0 || c1 <= c0) return TRACK_OK;
  if (!p || c0 < 0 || c1 > ld) return fail(TRACK_E_INVALID, "zero_cols: bad range");
  const int64_t n = rows * (c1 - c0);
  zero_cols_kernel<<<(unsigned)((n + 255) / 256), 256, 0, s>>>((bf16_t*)p, rows, ld, c0, c1 - c0);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ V transpose
// Tile of 64 keys x 32 channels through LDS; coalesced on both sides.
template <typename T>
__global__ __launch_bounds__(256) void v_transpose_kernel(int H, int dh, int64_t Lk, const T* __restrict__ src,
                                                          int64_t ld, int64_t col0, T* __restrict__ vt, int64_t ldv) {
  __shared__ T tile[64][33];
  const int64_t key0 = (int64_t)blockIdx.x * 64;
  const int cblocks = dh / 32;
  const int h = blockIdx.y / cblocks;
  const int c0 = (blockIdx.y % cblocks) * 32;
  const int b = blockIdx.z;
  const int tid = threadIdx.x;
  // read: 64 keys x 32 channels, thread -> (key = tid / 4 + 64 j / 4 ..)
  for (int i = tid; i < 64 * 32; i += 256) {
    const int kr = i / 32, cc = i % 32;
    const int64_t key = key0 + kr;
    T v = T(0);
    if (key < Lk) v = src[((int64_t)b * Lk + key) * ld + col0 + (int64_t)h * dh + c0 + cc];
    tile[kr][cc] = v;
  }
  __syncthreads();
  for (int i = tid; i < 64 * 32; i += 256) {
    const int cc = i / 64, kr = i % 64;
    const int64_t key = key0 + kr;
    if (key < ldv) vt[(((int64_t)b * H + h) * dh + c0 + cc) * ldv + key] = tile[kr][cc];
  }
}

track_status v_transpose(int dtype, int B, int H, int head_dim, int64_t Lk, const void* src, int64_t ld, int64_t col0,
                         void* vt, int64_t ldv, hipStream_t s) {
  if (head_dim % 32) return fail(TRACK_E_UNSUPPORTED, "v_transpose: head_dim %% 32 != 0");
  if (ldv < Lk) return fail(TRACK_E_SHAPE, "v_transpose: ldv < Lk");
  dim3 grid(cdiv(ldv, 64), H * (head_dim / 32), B);
  if (dtype == TRACK_DTYPE_BF16)
    v_transpose_kernel<bf16_t><<<grid, 256, 0, s>>>(H, head_dim, Lk, (const bf16_t*)src, ld, col0, (bf16_t*)vt, ldv);
  else
    v_transpose_kernel<float><<<grid, 256, 0, s>>>(H, head_dim, Lk, (const float*)src, ld, col0, (float*)vt, ldv);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ------------------------------------------------------------------ guidance + Euler (+ disagreement)
// Guided prediction of Eq. 1 from token-layout velocities: entries [0, n)
// are the conditional branch, [n, 2n) the unconditional one.  The same
// expression serves sampling and calibration so their updates are
// bit-identical.
__device__ __forceinline__ float guided(const float c, const float u, int B, float w) {
  return B == 2 ? fmaf(w, c - u, u) : c;
}

constexpr int STEP_THREADS = 256;
constexpr int STEP_MAX_BLOCKS = 1024;

int64_t step_partial_count(int64_t n) {
  int64_t nb = (n / 4 + STEP_THREADS - 1) / STEP_THREADS;
  if (nb > STEP_MAX_BLOCKS) nb = STEP_MAX_BLOCKS;
  return nb < 1 ? 1 : nb;
}

template <bool CALIB>
__global__ __launch_bounds__(STEP_THREADS) void step_kernel(int64_t n4, int B, float w, float dsigma,
                                                            const f32x4* __restrict__ vL, const f32x4* __restrict__ vS,
                                                            f32x4* __restrict__ x, double* __restrict__ partial) {
  double num = 0.0, den = 0.0;
  for (int64_t i = (int64_t)blockIdx.x * STEP_THREADS + threadIdx.x; i < n4; i += (int64_t)gridDim.x * STEP_THREADS) {
    const f32x4 cL = vL[i];
    const f32x4 uL = B == 2 ? vL[n4 + i] : cL;
    f32x4 xv = x[i];
    f32x4 pL;
#pragma unroll
    for (int j = 0; j < 4; ++j) pL[j] = guided(cL[j], uL[j], B, w);
    if constexpr (CALIB) {
      const f32x4 cS = vS[i];
      const f32x4 uS = B == 2 ? vS[n4 + i] : cS;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float pS = guided(cS[j], uS[j], B, w);
        const double df = (double)pS - (double)pL[j];
        num = fma(df, df, num);
        den = fma((double)pL[j], (double)pL[j], den);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) xv[j] = fmaf(dsigma, pL[j], xv[j]);
    x[i] = xv;
  }
  if constexpr (CALIB) {
    __shared__ double red[2][STEP_THREADS / 64];
    num = wave_sum_d(num);
    den = wave_sum_d(den);
    const int wv = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      red[0][wv] = num;
      red[1][wv] = den;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      double a = 0.0, b = 0.0;
      for (int i = 0; i < STEP_THREADS / 64; ++i) {
        a += red[0][i];
        b += red[1][i];
      }
      partial[2 * blockIdx.x] = a;
      partial[2 * blockIdx.x + 1] = b;
    }
  }
}

// r = sqrt(sum num) / max(sqrt(sum den), eps), partials summed in a fixed order.
__global__ __launch_bounds__(256) void disagreement_kernel(int nb, const double* __restrict__ partial, double eps,
                                                           double* __restrict__ r_out) {
  __shared__ double red[2][4];
  double a = 0.0, b = 0.0;
  for (int i = threadIdx.x; i < nb; i += 256) {
    a += partial[2 * i];
    b += partial[2 * i + 1];
  }
  a = wave_sum_d(a);
  b = wave_sum_d(b);
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = a;
    red[1][threadIdx.x >> 6] = b;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const double num = (red[0][0] + red[0][1]) + (red[0][2] + red[0][3]);
    const double den = (red[1][0] + red[1][1]) + (red[1][2] + red[1][3]);
    const double dn = sqrt(den);
    r_out[0] = sqrt(num) / (dn > eps ? dn : eps);
  }
}

track_status step(int64_t n, int B, float w, float dsigma, const float* vel_L, const float* vel_S, float* x,
                  double* partial, double eps, double* r_out, hipStream_t s) {
  if (n <= 0 || n % 4) return fail(TRACK_E_SHAPE, "step: n must be a positive multiple of 4");
  if (B != 1 && B != 2) return fail(TRACK_E_INVALID, "step: batch must be 1 or 2");
  if (!vel_L || !x) return fail(TRACK_E_INVALID, "step: null pointer");
  if (vel_S && (!partial || !r_out)) return fail(TRACK_E_INVALID, "step: calibration needs partial and r_out");
  ProfScope prof(TRACK_PROF_STEP, s);
  const int64_t nb = step_partial_count(n);
  if (vel_S) {
    step_kernel<true><<<(unsigned)nb, STEP_THREADS, 0, s>>>(n / 4, B, w, dsigma, (const f32x4*)vel_L,
                                                            (const f32x4*)vel_S, (f32x4*)x, partial);
    TRACK_LAUNCH_CHECK();
    disagreement_kernel<<<1, 256, 0, s>>>((int)nb, partial, eps, r_out);
  } else {
    step_kernel<false><<<(unsigned)nb, STEP_THREADS, 0, s>>>(n / 4, B, w, dsigma, (const f32x4*)vel_L, nullptr,
                                                             (f32x4*)x, nullptr);
  }
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ---------------------------------------------------------------- HBM streaming reference kernels
// Plain streams over a buffer, the practical ceiling the memory-bound kernels
// are measured against: each thread moves 4 consecutive 16-byte vectors of a
// 16 KB block chunk (loads first, then stores), whole chunks only.
constexpr int HBM_VEC_PER_THREAD = 4;
constexpr int64_t HBM_CHUNK = 256 * HBM_VEC_PER_THREAD * 16;

// src may equal dst (an in-place pass: each thread stores only what it loaded).
__global__ __launch_bounds__(256) void hbm_copy_kernel(const u32x4* src, u32x4* dst) {
  const int64_t base = (int64_t)blockIdx.x * (256 * HBM_VEC_PER_THREAD) + threadIdx.x;
  u32x4 v[HBM_VEC_PER_THREAD];
#pragma unroll
  for (int i = 0; i < HBM_VEC_PER_THREAD; ++i) v[i] = src[base + 256 * i];
#pragma unroll
  for (int i = 0; i < HBM_VEC_PER_THREAD; ++i) dst[base + 256 * i] = v[i];
}

// Reads every byte; the xor of the words reaches memory only if it equals a
// value a caller would have to plant, so the loads cannot be dropped.
__global__ __launch_bounds__(256) void hbm_read_kernel(const u32x4* __restrict__ src, uint32_t* __restrict__ sink,
                                                       uint32_t key) {
  const int64_t base = (int64_t)blockIdx.x * (256 * HBM_VEC_PER_THREAD) + threadIdx.x;
  uint32_t acc = 0;
#pragma unroll
  for (int i = 0; i < HBM_VEC_PER_THREAD; ++i) {
    const u32x4 v = src[base + 256 * i];
    acc ^= (v[0] ^ v[1]) ^ (v[2] ^ v[3]);
  }
  if (acc == key) sink[0] = acc;
}

__global__ __launch_bounds__(256) void hbm_write_kernel(u32x4* __restrict__ dst, uint32_t value) {
  const int64_t base = (int64_t)blockIdx.x * (256 * HBM_VEC_PER_THREAD) + threadIdx.x;
  const u32x4 v = {value, value, value, value};
#pragma unroll
  for (int i = 0; i < HBM_VEC_PER_THREAD; ++i) dst[base + 256 * i] = v;
}

track_status hbm_stream(int kind, const void* src, void* dst, int64_t bytes, hipStream_t s) {
  if (bytes <= 0 || bytes % HBM_CHUNK) return fail(TRACK_E_SHAPE, "hbm_stream: bytes must be a positive multiple of %lld",
                                                    (long long)HBM_CHUNK);
  if (bytes / HBM_CHUNK > INT32_MAX) return fail(TRACK_E_SHAPE, "hbm_stream: buffer too large");
  if (((uintptr_t)src & 15) || ((uintptr_t)dst & 15)) return fail(TRACK_E_INVALID, "hbm_stream: 16-byte alignment needed");
  const unsigned grid = (unsigned)(bytes / HBM_CHUNK);
  ProfScope prof(TRACK_PROF_OTHER, s);
  switch (kind) {
    case 0:
      if (!src || !dst) return fail(TRACK_E_INVALID, "hbm_stream: null pointer");
      hbm_copy_kernel<<<grid, 256, 0, s>>>((const u32x4*)src, (u32x4*)dst);
      break;
    case 1:
      if (!src || !dst) return fail(TRACK_E_INVALID, "hbm_stream: null pointer");
      hbm_read_kernel<<<grid, 256, 0, s>>>((const u32x4*)src, (uint32_t*)dst, 0x9e3779b9u);
      break;
    case 2:
      if (!dst) return fail(TRACK_E_INVALID, "hbm_stream: null pointer");
      hbm_write_kernel<<<grid, 256, 0, s>>>((u32x4*)dst, 0x3f800000u);
      break;
    default:
      return fail(TRACK_E_INVALID, "hbm_stream: bad kind %d", kind);
  }
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

// ---------------------------------------------------------------- step without caller scratch
// The calibration step's per-block partial sums in a file-scope device array
// instead of a caller workspace, for callers that cannot allocate.  Every
// block writes its own pair before disagreement_kernel reads them on the same
// stream, so nothing in it needs clearing; calls that overlap on one GPU
// share the array and race.
constexpr int STEP_STATIC_DOUBLES = 2 * STEP_MAX_BLOCKS;
static __device__ __align__(256) double step_scratch[STEP_STATIC_DOUBLES];

static std::mutex g_step_scratch_mu;
static double* g_step_scratch_ptr[64] = {nullptr};

// The device address of this GPU's copy of step_scratch, looked up once per
// device (the array's name is a host-side stand-in, not a device address).
static track_status step_scratch_ptr(double** out) {
  int dev = 0;
  TRACK_HIP(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(TRACK_E_DEVICE, "step (static scratch): device index %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_step_scratch_mu);
  if (!g_step_scratch_ptr[dev]) {
    void* p = nullptr;
    TRACK_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(step_scratch)));
    if (!p) return fail(TRACK_E_DEVICE, "step (static scratch): no device address for the scratch array");
    g_step_scratch_ptr[dev] = (double*)p;
  }
  *out = g_step_scratch_ptr[dev];
  return TRACK_OK;
}

track_status step_static(int64_t n, int B, float w, float dsigma, const float* vel_L, const float* vel_S, float* x,
                         double eps, double* r_out, hipStream_t s) {
  if (step_partial_count(n > 0 ? n : 4) * 2 > STEP_STATIC_DOUBLES)
    return fail(TRACK_E_UNSUPPORTED, "step (static scratch): %lld partial sums exceed the %d the scratch holds",
                (long long)(step_partial_count(n) * 2), STEP_STATIC_DOUBLES);
  if (vel_S && !r_out) return fail(TRACK_E_INVALID, "step (static scratch): calibration needs r_out");
  double* partial = nullptr;
  if (vel_S) {
    const track_status st = step_scratch_ptr(&partial);
    if (st != TRACK_OK) return st;
  }
  return step(n, B, w, dsigma, vel_L, vel_S, x, partial, eps, r_out, s);
}

// UniPC step (see UniPCStep): m = x - sigma p, then the corrector (x^c from
// the previous step's corrected sample and the stored data predictions) and
// the predictor, written in place: x <- x_next, x_last <- x^c, m_out <- m.
// The calibration variant also accumulates the Eq. 4 partials and advances
// with the large model's p, like step_kernel.
struct UniPCArgs {
  float sigma;
  float cx, c_m0, c_h0, c_h1, c_new;
  float px, p_m, p_h0, p_h1;
  int corr, nh_c, nh_p;
};

template <bool CALIB>
__global__ __launch_bounds__(STEP_THREADS) void unipc_kernel(int64_t n4, int B, float w, UniPCArgs a,
                                                             const f32x4* __restrict__ vL,
                                                             const f32x4* __restrict__ vS, f32x4* __restrict__ x,
                                                             f32x4* __restrict__ xlast, const f32x4* __restrict__ H0,
                                                             const f32x4* __restrict__ H1,
                                                             const f32x4* __restrict__ H2,
                                                             f32x4* __restrict__ mout, double* __restrict__ partial) {
  double num = 0.0, den = 0.0;
  const bool need_h0 = a.corr || a.nh_p > 0;
  const bool need_h1 = (a.corr && a.nh_c > 0) || a.nh_p > 1;
  const bool need_h2 = a.corr && a.nh_c > 1;
  for (int64_t i = (int64_t)blockIdx.x * STEP_THREADS + threadIdx.x; i < n4; i += (int64_t)gridDim.x * STEP_THREADS) {
    const f32x4 cL = vL[i];
    const f32x4 uL = B == 2 ? vL[n4 + i] : cL;
    const f32x4 xv = x[i];
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    const f32x4 h0 = need_h0 ? H0[i] : z;
    const f32x4 h1 = need_h1 ? H1[i] : z;
    const f32x4 h2 = need_h2 ? H2[i] : z;
    const f32x4 xl = a.corr ? xlast[i] : z;
    f32x4 pL, m, xc, xn;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      pL[j] = guided(cL[j], uL[j], B, w);
      m[j] = fmaf(-a.sigma, pL[j], xv[j]);
    }
    if constexpr (CALIB) {
      const f32x4 cS = vS[i];
      const f32x4 uS = B == 2 ? vS[n4 + i] : cS;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float pS = guided(cS[j], uS[j], B, w);
        const double df = (double)pS - (double)pL[j];
        num = fma(df, df, num);
        den = fma((double)pL[j], (double)pL[j], den);
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float c = xv[j];
      if (a.corr) {
        c = fmaf(a.c_new, m[j], fmaf(a.c_m0, h0[j], a.cx * xl[j]));
        if (a.nh_c > 0) c = fmaf(a.c_h0, h1[j], c);
        if (a.nh_c > 1) c = fmaf(a.c_h1, h2[j], c);
      }
      float nx = fmaf(a.p_m, m[j], a.px * c);
      if (a.nh_p > 0) nx = fmaf(a.p_h0, h0[j], nx);
      if (a.nh_p > 1) nx = fmaf(a.p_h1, h1[j], nx);
      xc[j] = c;
      xn[j] = nx;
    }
    x[i] = xn;
    xlast[i] = xc;
    mout[i] = m;
  }
  if constexpr (CALIB) {
    __shared__ double red[2][STEP_THREADS / 64];
    num = wave_sum_d(num);
    den = wave_sum_d(den);
    const int wv = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0) {
      red[0][wv] = num;
      red[1][wv] = den;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      double s0 = 0.0, s1 = 0.0;
      for (int k = 0; k < STEP_THREADS / 64; ++k) {
        s0 += red[0][k];
        s1 += red[1][k];
      }
      partial[2 * blockIdx.x] = s0;
      partial[2 * blockIdx.x + 1] = s1;
    }
  }
}

track_status unipc_step(int64_t n, int B, float w, float sigma, const UniPCStep& c, const float* vel_L,
                        const float* vel_S, float* x, float* x_last, const float* h0, const float* h1,
                        const float* h2, float* m_out, double* partial, double eps, double* r_out, hipStream_t s) {
  if (n <= 0 || n % 4) return fail(TRACK_E_SHAPE, "unipc_step: n must be a positive multiple of 4");
  if (B != 1 && B != 2) return fail(TRACK_E_INVALID, "unipc_step: batch must be 1 or 2");
  if (!vel_L || !x || !x_last || !m_out) return fail(TRACK_E_INVALID, "unipc_step: null pointer");
  if (c.nh_c < 0 || c.nh_c > 2 || c.nh_p < 0 || c.nh_p > 2) return fail(TRACK_E_INVALID, "unipc_step: bad history count");
  if (((c.corr || c.nh_p > 0) && !h0) || (((c.corr && c.nh_c > 0) || c.nh_p > 1) && !h1) ||
      (c.corr && c.nh_c > 1 && !h2))
    return fail(TRACK_E_INVALID, "unipc_step: a history buffer the step reads is NULL");
  if (vel_S && (!partial || !r_out)) return fail(TRACK_E_INVALID, "unipc_step: calibration needs partial and r_out");
  UniPCArgs a;
  a.sigma = sigma;
  a.cx = (float)c.cx;
  a.c_m0 = (float)c.c_m0;
  a.c_h0 = (float)c.c_h[0];
  a.c_h1 = (float)c.c_h[1];
  a.c_new = (float)c.c_new;
  a.px = (float)c.px;
  a.p_m = (float)c.p_m;
  a.p_h0 = (float)c.p_h[0];
  a.p_h1 = (float)c.p_h[1];
  a.corr = c.corr;
  a.nh_c = c.nh_c;
  a.nh_p = c.nh_p;
  ProfScope prof(TRACK_PROF_STEP, s);
  const int64_t nb = step_partial_count(n);
  const f32x4 *H0 = (const f32x4*)h0, *H1 = (const f32x4*)h1, *H2 = (const f32x4*)h2;
  if (vel_S) {
    unipc_kernel<true><<<(unsigned)nb, STEP_THREADS, 0, s>>>(n / 4, B, w, a, (const f32x4*)vel_L,
                                                             (const f32x4*)vel_S, (f32x4*)x, (f32x4*)x_last, H0, H1,
                                                             H2, (f32x4*)m_out, partial);
    TRACK_LAUNCH_CHECK();
    disagreement_kernel<<<1, 256, 0, s>>>((int)nb, partial, eps, r_out);
  } else {
    unipc_kernel<false><<<(unsigned)nb, STEP_THREADS, 0, s>>>(n / 4, B, w, a, (const f32x4*)vel_L, nullptr,
                                                              (f32x4*)x, (f32x4*)x_last, H0, H1, H2,
                                                              (f32x4*)m_out, nullptr);
  }
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

__global__ void guide_unpatchify_kernel(const float* __restrict__ vel, int B, float w, float* __restrict__ out,
                                        int64_t n, int C, int F, int H, int W, int pt, int ph, int pw) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int wq = (int)(i % W);
  const int hq = (int)((i / W) % H);
  const int fq = (int)((i / ((int64_t)W * H)) % F);
  const int c = (int)(i / ((int64_t)W * H * F));
  const int Hp = H / ph, Wp = W / pw;
  const int64_t l = ((int64_t)(fq / pt) * Hp + hq / ph) * Wp + wq / pw;
  const int e = ((c * pt + fq % pt) * ph + hq % ph) * pw + wq % pw;
  const int64_t t = l * ((int64_t)C * pt * ph * pw) + e;
  const float cv = vel[t];
  out[i] = guided(cv, B == 2 ? vel[n + t] : cv, B, w);
}

track_status guide_unpatchify(const float* vel, int B, float w, float* out, int C, int F, int H, int W, int pt, int ph,
                              int pw, hipStream_t s) {
  const int64_t n = (int64_t)C * F * H * W;
  ProfScope prof(TRACK_PROF_STEP, s);
  guide_unpatchify_kernel<<<cdiv(n, 256), 256, 0, s>>>(vel, B, w, out, n, C, F, H, W, pt, ph, pw);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

}  // namespace track
