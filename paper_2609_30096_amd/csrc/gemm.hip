// Projection GEMMs of the denoiser: out = epilogue(A W^T + b).
//
// A is the activation matrix [M tokens, K] and W a linear weight [N, K]
// (both K-contiguous).  The bfloat16 kernel runs on CDNA4 matrix cores
// (v_mfma_f32_32x32x16_bf16) with the weight tile as the MFMA "A" operand and
// the token tile as the "B" operand, so each lane's accumulators hold one
// token and runs of four consecutive output features; the epilogue then
// writes 8- or 16-byte vectors.  Epilogues fuse the bias, the tanh GELU of
// the MLP, and the adaLN gate with the float32 residual update.
#include <cstdlib>

#include "common.h"
#include "kernels.h"

namespace track {

struct EpiArgs {
  const void* bias;   // [N], weight dtype
  const float* gate;  // [N] float32 (gated residual only)
  void* out;          // output or residual
  int64_t ldo;
};

// ------------------------------------------------------------------ epilogues
template <int EPI, typename T>
__device__ __forceinline__ void epi_store4(const EpiArgs& e, int64_t m, int n, float v0, float v1, float v2,
                                           float v3) {
  const T* b = (const T*)e.bias + n;
  v0 += ldf(b + 0);
  v1 += ldf(b + 1);
  v2 += ldf(b + 2);
  v3 += ldf(b + 3);
  if constexpr (EPI == TRACK_EPI_BIAS || EPI == TRACK_EPI_BIAS_GELU) {
    if constexpr (EPI == TRACK_EPI_BIAS_GELU) {
      v0 = gelu_tanh(v0); v1 = gelu_tanh(v1); v2 = gelu_tanh(v2); v3 = gelu_tanh(v3);
    }
    T* o = (T*)e.out + m * e.ldo + n;
    if constexpr (sizeof(T) == 2) {
      u32x2 pk;
      pk[0] = pack_bf2(v0, v1);
      pk[1] = pack_bf2(v2, v3);
      *(u32x2*)o = pk;
    } else {
      *(f32x4*)o = f32x4{v0, v1, v2, v3};
    }
  } else if constexpr (EPI == TRACK_EPI_GATE_RESID || EPI == TRACK_EPI_RESID) {
    float* o = (float*)e.out + m * e.ldo + n;
    f32x4 x = *(f32x4*)o;
    if constexpr (EPI == TRACK_EPI_GATE_RESID) {
      const f32x4 g = *(const f32x4*)(e.gate + n);
      x[0] = fmaf(g[0], v0, x[0]); x[1] = fmaf(g[1], v1, x[1]);
      x[2] = fmaf(g[2], v2, x[2]); x[3] = fmaf(g[3], v3, x[3]);
    } else {
      x[0] += v0; x[1] += v1; x[2] += v2; x[3] += v3;
    }
    *(f32x4*)o = x;
  } else {  // TRACK_EPI_BIAS_F32
    float* o = (float*)e.out + m * e.ldo + n;
    *(f32x4*)o = f32x4{v0, v1, v2, v3};
  }
}

template <int EPI, typename T>
__device__ __forceinline__ void epi_store1(const EpiArgs& e, int64_t m, int n, float v) {
  v += ldf((const T*)e.bias + n);
  if constexpr (EPI == TRACK_EPI_BIAS || EPI == TRACK_EPI_BIAS_GELU) {
    if constexpr (EPI == TRACK_EPI_BIAS_GELU) v = gelu_tanh(v);
    stf((T*)e.out + m * e.ldo + n, v);
  } else if constexpr (EPI == TRACK_EPI_GATE_RESID) {
    float* o = (float*)e.out + m * e.ldo + n;
    *o = fmaf(e.gate[n], v, *o);
  } else if constexpr (EPI == TRACK_EPI_RESID) {
    float* o = (float*)e.out + m * e.ldo + n;
    *o += v;
  } else {
    ((float*)e.out)[m * e.ldo + n] = v;
  }
}

// ------------------------------------------------------------------ bf16 MFMA kernel
// Block tile BM tokens x BN features x 64 (K); four waves in a 2 x 2 grid,
// each owning (BM/2) x (BN/2) as 32 x 32 MFMA blocks.  Tiles are staged
// through LDS, double buffered, rows of 64 bf16 (128 B) with the 16-byte
// chunk index XOR-swizzled by (row & 7) so that the 32-row fragment reads
// are bank-conflict free.  Global loads of the next K-slab are issued before
// the MFMAs of the current one.
template <int BM, int BN, int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(const bf16_t* __restrict__ A, int64_t lda,
                                                        const bf16_t* __restrict__ W, int64_t M, int N, int K,
                                                        EpiArgs e) {
  constexpr int BK = 64;
  constexpr int WM = BM / 2, WN = BN / 2;
  constexpr int TI = WM / 32, FI = WN / 32;
  constexpr int AC = BM / 32;  // 16-byte chunks per thread for the A tile (BM * 8 / 256)
  constexpr int WC = BN / 32;
  constexpr int TILE_BYTES = (BM + BN) * 128;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * TILE_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // tile order: XCD-aware remap, then bands of 8 M-tiles swept across N
  const int num_tm = (int)((M + BM - 1) / BM);
  const int num_tn = N / BN;
  const int pid = xcd_remap(blockIdx.x, gridDim.x);
  constexpr int G = 8;
  const int band = pid / (G * num_tn);
  const int first_tm = band * G;
  const int gsz = min(num_tm - first_tm, G);
  const int in_band = pid - band * G * num_tn;
  const int tm = first_tm + in_band % gsz;
  const int tn = in_band / gsz;
  const int64_t m0 = (int64_t)tm * BM;
  const int n0 = tn * BN;

  // staging: thread handles chunk column c = tid & 7 of rows (tid >> 3) + 32 i
  const int c = tid & 7;
  const int r0 = tid >> 3;
  const bf16_t* a_ptr[AC];
#pragma unroll
  for (int i = 0; i < AC; ++i) {
    int64_t row = m0 + r0 + 32 * i;
    if (row > M - 1) row = M - 1;
    a_ptr[i] = A + row * lda + c * 8;
  }
  const bf16_t* w_ptr = W + (int64_t)(n0 + r0) * K + c * 8;

  u32x4 ra[AC], rw[WC];
  auto load_global = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int i = 0; i < AC; ++i) ra[i] = *(const u32x4*)(a_ptr[i] + k0);
#pragma unroll
    for (int i = 0; i < WC; ++i) rw[i] = *(const u32x4*)(w_ptr + (int64_t)32 * i * K + k0);
  };
  auto store_lds = [&](int buf) {
    uint8_t* base = smem + buf * TILE_BYTES;
#pragma unroll
    for (int i = 0; i < AC; ++i) {
      const int row = r0 + 32 * i;
      *(u32x4*)(base + row * 128 + ((c ^ (row & 7)) << 4)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < WC; ++i) {
      const int row = r0 + 32 * i;
      *(u32x4*)(base + (BM + row) * 128 + ((c ^ (row & 7)) << 4)) = rw[i];
    }
  };

  f32x16 acc[FI][TI];
#pragma unroll
  for (int fi = 0; fi < FI; ++fi)
#pragma unroll
    for (int ti = 0; ti < TI; ++ti)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[fi][ti][r] = 0.0f;

  const int KT = K / BK;
  load_global(0);
  store_lds(0);
  __syncthreads();

  const int frow = lane & 31;
  const int fhalf = lane >> 5;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) load_global(kt + 1);
    const uint8_t* base = smem + cur * TILE_BYTES;
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int ch = kk * 2 + fhalf;
      bf16x8 fw[FI], fa[TI];
#pragma unroll
      for (int fi = 0; fi < FI; ++fi) {
        const int row = wn * WN + fi * 32 + frow;
        fw[fi] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + (BM + row) * 128 + ((ch ^ (row & 7)) << 4)));
      }
#pragma unroll
      for (int ti = 0; ti < TI; ++ti) {
        const int row = wm * WM + ti * 32 + frow;
        fa[ti] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + row * 128 + ((ch ^ (row & 7)) << 4)));
      }
#pragma unroll
      for (int fi = 0; fi < FI; ++fi)
#pragma unroll
        for (int ti = 0; ti < TI; ++ti)
          acc[fi][ti] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[fi], fa[ti], acc[fi][ti], 0, 0, 0);
    }
    if (kt + 1 < KT) store_lds(cur ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds token (lane & 31) and features 8g + 4 (lane >> 5) + {0..3}
#pragma unroll
  for (int ti = 0; ti < TI; ++ti) {
    const int64_t m = m0 + wm * WM + ti * 32 + frow;
    if (m >= M) continue;
#pragma unroll
    for (int fi = 0; fi < FI; ++fi)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * WN + fi * 32 + 8 * g + 4 * fhalf;
        epi_store4<EPI, bf16_t>(e, m, n, acc[fi][ti][4 * g + 0], acc[fi][ti][4 * g + 1], acc[fi][ti][4 * g + 2],
                                acc[fi][ti][4 * g + 3]);
      }
  }
}

// ------------------------------------------------------------------ float32 kernel
// Plain LDS-tiled FMA GEMM (64 x 64 tile, K-slab 16, 4 x 4 outputs per
// thread) for the float32 parity path; any M, N, K.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ A, int64_t lda,
                                                       const float* __restrict__ W, int64_t M, int N, int K,
                                                       EpiArgs e) {
  __shared__ float As[16][65];
  __shared__ float Ws[16][65];
  const int tid = threadIdx.x;
  const int tx = tid & 15, ty = tid >> 4;
  const int64_t m0 = (int64_t)blockIdx.y * 64;
  const int n0 = blockIdx.x * 64;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int idx = tid + 256 * i;  // 0..1023 over a 64 x 16 tile
      const int row = idx >> 4, kk = idx & 15;
      const int64_t gm = m0 + row;
      const int gn = n0 + row;
      const int gk = k0 + kk;
      As[kk][row] = (gm < M && gk < K) ? A[gm * lda + gk] : 0.0f;
      Ws[kk][row] = (gn < N && gk < K) ? W[(int64_t)gn * K + gk] : 0.0f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        w[i] = Ws[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      if (n < N) epi_store1<EPI, float>(e, m, n, acc[i][j]);
    }
  }
}

// ------------------------------------------------------------------ launchers
template <int BM, int BN>
static void launch_bf16_cfg(int epi, const bf16_t* A, int64_t lda, const bf16_t* W, int64_t M, int N, int K,
                            const EpiArgs& e, hipStream_t s) {
  const int tiles = (int)((M + BM - 1) / BM) * (N / BN);
  dim3 grid(tiles), block(256);
  switch (epi) {
    case TRACK_EPI_BIAS: gemm_bf16_kernel<BM, BN, TRACK_EPI_BIAS><<<grid, block, 0, s>>>(A, lda, W, M, N, K, e); break;
    case TRACK_EPI_BIAS_GELU: gemm_bf16_kernel<BM, BN, TRACK_EPI_BIAS_GELU><<<grid, block, 0, s>>>(A, lda, W, M, N, K, e); break;
    case TRACK_EPI_GATE_RESID: gemm_bf16_kernel<BM, BN, TRACK_EPI_GATE_RESID><<<grid, block, 0, s>>>(A, lda, W, M, N, K, e); break;
    case TRACK_EPI_RESID: gemm_bf16_kernel<BM, BN, TRACK_EPI_RESID><<<grid, block, 0, s>>>(A, lda, W, M, N, K, e); break;
    default: gemm_bf16_kernel<BM, BN, TRACK_EPI_BIAS_F32><<<grid, block, 0, s>>>(A, lda, W, M, N, K, e); break;
  }
}

// Tile override for tuning runs (TRACK_GEMM_CFG): 0 automatic, 1 256x256,
// 2 128x128, 3 256x128; shapes the forced tile does not divide use the
// automatic choice.
static int gemm_config() {
  static const int cfg = [] {
    const char* v = getenv("TRACK_GEMM_CFG");
    const int c = v ? atoi(v) : 0;
    return (c >= 0 && c <= 3) ? c : 0;
  }();
  return cfg;
}

track_status linear(int dtype, int epi, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* W,
                    const void* bias, const float* gate, void* out, int64_t ldo, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0) return fail(TRACK_E_SHAPE, "linear: empty shape M=%lld N=%lld K=%lld", (long long)M, (long long)N, (long long)K);
  if (!A || !W || !bias || !out) return fail(TRACK_E_INVALID, "linear: null pointer");
  if (epi < 0 || epi > TRACK_EPI_BIAS_F32) return fail(TRACK_E_INVALID, "linear: bad epilogue %d", epi);
  if (epi == TRACK_EPI_GATE_RESID && !gate) return fail(TRACK_E_INVALID, "linear: gated residual needs gate");
  if (lda < K || ldo < N) return fail(TRACK_E_SHAPE, "linear: leading dimension too small");
  if (N > (1 << 30) || K > (1 << 30)) return fail(TRACK_E_SHAPE, "linear: N or K too large");
  EpiArgs e{bias, gate, out, ldo};
  ProfScope prof(TRACK_PROF_GEMM, s);
  if (dtype == TRACK_DTYPE_F32) {
    dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64)), block(256);
    const float* a = (const float*)A;
    const float* w = (const float*)W;
    switch (epi) {
      case TRACK_EPI_BIAS: gemm_f32_kernel<TRACK_EPI_BIAS><<<grid, block, 0, s>>>(a, lda, w, M, (int)N, (int)K, e); break;
      case TRACK_EPI_BIAS_GELU: gemm_f32_kernel<TRACK_EPI_BIAS_GELU><<<grid, block, 0, s>>>(a, lda, w, M, (int)N, (int)K, e); break;
      case TRACK_EPI_GATE_RESID: gemm_f32_kernel<TRACK_EPI_GATE_RESID><<<grid, block, 0, s>>>(a, lda, w, M, (int)N, (int)K, e); break;
      case TRACK_EPI_RESID: gemm_f32_kernel<TRACK_EPI_RESID><<<grid, block, 0, s>>>(a, lda, w, M, (int)N, (int)K, e); break;
      default: gemm_f32_kernel<TRACK_EPI_BIAS_F32><<<grid, block, 0, s>>>(a, lda, w, M, (int)N, (int)K, e); break;
    }
    TRACK_LAUNCH_CHECK();
    return TRACK_OK;
  }
  if (dtype != TRACK_DTYPE_BF16) return fail(TRACK_E_INVALID, "linear: bad dtype %d", dtype);
  if (K % 64 || N % 64) return fail(TRACK_E_UNSUPPORTED, "linear: bf16 path needs N, K multiples of 64 (N=%lld K=%lld)", (long long)N, (long long)K);
  if (lda % 8 || ldo % 4 || ((uintptr_t)A & 15) || ((uintptr_t)W & 15) || ((uintptr_t)out & 15) ||
      ((uintptr_t)bias & 7) || (gate && ((uintptr_t)gate & 15)))
    return fail(TRACK_E_INVALID, "linear: bf16 path needs 16-byte aligned rows");
  const bf16_t* a = (const bf16_t*)A;
  const bf16_t* w = (const bf16_t*)W;
  const int n = (int)N, k = (int)K;
  const int64_t big = ((M + 255) / 256) * (N / 256);
  const int force = gemm_config();
  if (force == 1 && N % 256 == 0)
    launch_bf16_cfg<256, 256>(epi, a, lda, w, M, n, k, e, s);
  else if (force == 2 && N % 128 == 0)
    launch_bf16_cfg<128, 128>(epi, a, lda, w, M, n, k, e, s);
  else if (force == 3 && N % 128 == 0)
    launch_bf16_cfg<256, 128>(epi, a, lda, w, M, n, k, e, s);
  else if (N % 256 == 0 && big >= 512)
    launch_bf16_cfg<256, 256>(epi, a, lda, w, M, n, k, e, s);
  else if (N % 128 == 0)
    launch_bf16_cfg<128, 128>(epi, a, lda, w, M, n, k, e, s);
  else
    launch_bf16_cfg<128, 64>(epi, a, lda, w, M, n, k, e, s);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

}  // namespace track
