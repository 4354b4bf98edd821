// Shared device helpers for the gfx950 kernels: bfloat16 storage, MFMA
// vector types, element access overloads and launch bookkeeping.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "track.h"

typedef uint16_t bf16_t;  // bfloat16 bits in memory

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }

// Round to nearest even (the hardware conversion on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(bf16_t, b);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two floats to packed bf16 (round to nearest even) in one conversion.
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  const bf16x2_t v = __builtin_convertvector(f32x2{lo, hi}, bf16x2_t);
  return __builtin_bit_cast(uint32_t, v);
}

// Scalar load/store overloads so element-wise kernels are written once for
// float32 and bfloat16 activations.
__device__ __forceinline__ float ldf(const float* p) { return *p; }
__device__ __forceinline__ float ldf(const bf16_t* p) { return bf2f(*p); }
__device__ __forceinline__ void stf(float* p, float v) { *p = v; }
__device__ __forceinline__ void stf(bf16_t* p, float v) { *p = f2bf(v); }

// tanh-form GELU, 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x + 0.044715 x^3),
// evaluated through the identity 0.5 (1 + tanh(u)) = 1 / (1 + exp(-2u)):
// exp(-2u) = exp2(x (k1 + k2 x^2)) with k1 = -2 sqrt(2/pi) log2(e) and
// k2 = 0.044715 k1, then one reciprocal; saturates to x and to -0 for finite
// x without NaNs.
__device__ __forceinline__ float gelu_tanh(float x) {
  constexpr float k1 = -2.302208198f;
  constexpr float k2 = -0.1029432396f;
  const float e = __builtin_amdgcn_exp2f(x * fmaf(k2, x * x, k1));
  return x * __builtin_amdgcn_rcpf(1.0f + e);
}

__device__ __forceinline__ float silu(float x) { return x / (1.0f + expf(-x)); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Workgroup id remapped so that the workgroups the dispatcher places on one
// XCD (ids congruent mod 8) receive a contiguous range of logical tiles; the
// mapping is a bijection for any grid size.
__device__ __forceinline__ int xcd_remap(int pid, int nwg) {
  const int q = nwg >> 3, rem = nwg & 7;
  const int x = pid & 7;
  const int start = x * q + (x < rem ? x : rem);
  return start + (pid >> 3);
}

// ---------------------------------------------------------------- host side
namespace track {

// Set the thread-local error message and return the status.
track_status fail(track_status s, const char* fmt, ...);

// Profiling of kernel classes (see track_profile_*).
struct ProfScope {
  int kind;
  hipStream_t stream;
  int slot;
  ProfScope(int kind, hipStream_t stream);
  ~ProfScope();
};

}  // namespace track

#define TRACK_HIP(call)                                                                     \
  do {                                                                                      \
    hipError_t e_ = (call);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return ::track::fail(TRACK_E_DEVICE, "%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), \
                           __FILE__, __LINE__);                                             \
  } while (0)

#define TRACK_LAUNCH_CHECK()                                                                \
  do {                                                                                      \
    hipError_t e_ = hipGetLastError();                                                      \
    if (e_ != hipSuccess)                                                                   \
      return ::track::fail(TRACK_E_DEVICE, "kernel launch failed: %s (%s:%d)",              \
                           hipGetErrorString(e_), __FILE__, __LINE__);                      \
  } while (0)
