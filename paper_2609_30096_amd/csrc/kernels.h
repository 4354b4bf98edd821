// Host-side launchers of the denoiser kernels (all asynchronous on `s`).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <vector>

#include "common.h"
#include "track.h"

namespace track {

// gemm.hip
track_status linear(int dtype, int epi, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* W,
                    const void* bias, const float* gate, void* out, int64_t ldo, hipStream_t s);
// A W^T + bias (bfloat16) written transposed per batch of L rows:
// vt[((m / L) * N + n) * ldv + m % L].
track_status linear_vt(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* W, const void* bias,
                       int64_t L, void* vt, int64_t ldv, hipStream_t s);
// Compute units of the current device (cached per device; 256 if the query fails).
int device_cus();
// Zeroes columns [c0, c1) of a rows x ld bfloat16 matrix.
track_status zero_cols_bf16(void* p, int64_t rows, int64_t ld, int64_t c0, int64_t c1, hipStream_t s);

// attention.hip
// q_log2: (bfloat16 only) q already holds q log2(e) / sqrt(head_dim), as
// rmsnorm_rope writes it with qscale = attn_log2_scale(head_dim)
track_status attention(int dtype, int B, int H, int head_dim, int64_t Lq, int64_t Lk, const void* q, int64_t ldq,
                       const void* k, int64_t ldk, const void* vt, int64_t ldv, void* out, int64_t ldo,
                       hipStream_t s, int prof_kind, bool q_log2 = false);
// The softmax scale in log2 units, log2(e) / sqrt(head_dim).
float attn_log2_scale(int head_dim);

// elementwise.hip
struct Grid3 {
  int f, h, w;
};
track_status patchify(const float* x, float* tok, int C, int F, int H, int W, int pt, int ph, int pw, hipStream_t s);
track_status unpatchify(const float* tok, float* x, int C, int F, int H, int W, int pt, int ph, int pw,
                        hipStream_t s);
track_status to_bf16(const float* src, bf16_t* dst, int64_t n, hipStream_t s);
track_status sinusoid(double t, int dim, float* out, hipStream_t s);
// y[n] = act(sum_k W[n, k] x[k] + b[n]) with act = SiLU if post_silu else identity;
// if y_silu != NULL it also receives SiLU(y).
track_status gemv(int dtype, int N, int K, const void* W, const void* b, const float* x, float* y, float* y_silu,
                  int post_silu, hipStream_t s);
// mods[blk, 6, d] = m[6, d] + T_blk[6, d]; T_blk at Tbase + blk * stride_elems (weight dtype)
track_status mod_tables(int dtype, int blocks, int d, const float* m, const void* Tbase, int64_t stride_elems,
                        float* mods, hipStream_t s);
// out[2, d] = T[2, d] + e[d]
track_status head_mod(int dtype, int d, const float* e, const void* T, float* out, hipStream_t s);
// cos/sin tables in float64 cast to float32: for axis a with section width n_a
// and extent E_a, table[a][pos][i] for i < n_a / 2.
track_status rope_tables(int head_dim, Grid3 g, float* cos_t, float* sin_t, hipStream_t s);
track_status layernorm(int dtype, int64_t rows, int d, const float* x, const float* scale, const float* shift, void* y,
                       hipStream_t s);
// g2 != nullptr: two adjacent segments per row (col0 with gain g, col0 + d with g2) in one launch.
// qscale multiplies the first segment's output (before its one rounding).
track_status rmsnorm_rope(int dtype, int64_t rows, int heads, int head_dim, void* buf, int64_t ld, int64_t col0,
                          const void* g, const void* g2, const float* cos_t, const float* sin_t, Grid3 grid, int64_t L,
                          hipStream_t s, float qscale = 1.0f);
// vt[(b*H + h)*head_dim + c][key] = src[(b*Lk + key)*ld + col0 + h*head_dim + c]; zeros for Lk <= key < ldv
track_status v_transpose(int dtype, int B, int H, int head_dim, int64_t Lk, const void* src, int64_t ld, int64_t col0,
                         void* vt, int64_t ldv, hipStream_t s);
// Step kernels (see track_op_step).
int64_t step_partial_count(int64_t n);
track_status step(int64_t n, int B, float w, float dsigma, const float* vel_L, const float* vel_S, float* x,
                  double* partial, double eps, double* r_out, hipStream_t s);
// plain copy (0), read (1) or write (2) stream over `bytes` (multiple of 16 KiB)
track_status hbm_stream(int kind, const void* src, void* dst, int64_t bytes, hipStream_t s);
// independent 32x32x16 bf16 MFMA chains on every CU from caller operands (64 KiB)
track_status mfma_stream(const void* operands, int64_t iters, float* sink, int64_t* flop, hipStream_t s);
// step() with the calibration partials in a static device array (no caller scratch)
track_status step_static(int64_t n, int B, float w, float dsigma, const float* vel_L, const float* vel_S, float* x,
                         double eps, double* r_out, hipStream_t s);
// UniPC: per-step weights of the fused corrector + predictor (sched.cpp) and
// the kernel applying them (elementwise.hip); see track_unipc_coefficients.
struct UniPCStep {
  int corr = 0, nh_c = 0, nh_p = 0;
  double cx = 0.0, c_m0 = 0.0, c_h[2] = {0.0, 0.0}, c_new = 0.0;
  double px = 0.0, p_m = 0.0, p_h[2] = {0.0, 0.0};
};
std::vector<UniPCStep> unipc_plan(const std::vector<double>& sig, int order);
track_status unipc_step(int64_t n, int B, float w, float sigma, const UniPCStep& c, const float* vel_L,
                        const float* vel_S, float* x, float* x_last, const float* h0, const float* h1,
                        const float* h2, float* m_out, double* partial, double eps, double* r_out, hipStream_t s);
// Guided prediction scattered to C x F x H x W (track_dit_forward's output).
track_status guide_unpatchify(const float* vel, int B, float w, float* out, int C, int F, int H, int W, int pt, int ph,
                              int pw, hipStream_t s);

// bands.hip: frequency-band energies of the guided difference p_S - p_L of
// two token-layout velocity buffers (C x F x H x W latent, patch pt x ph x pw).
track_status band_check(int C, int F, int H, int W, int pt, int ph, int pw);
size_t band_workspace_bytes(int C, int F, int H, int W, int pt, int ph, int pw);
// byte offset in the band workspace of the slot that receives the energies
// when energy_dev is NULL
size_t band_energy_offset(int C, int F, int H, int W, int pt, int ph, int pw);
// energy_dev (or, if NULL, a slot in ws) receives 6 energies: spatial low,
// mid, high, temporal low, mid, high.  With step_partial (the calibration step
// kernel's (sum d^2, sum p_L^2) pairs) score_dev receives the 6 band scores.
track_status band_scores(int C, int F, int H, int W, int pt, int ph, int pw, int B, float w, const float* vel_L,
                         const float* vel_S, const double* step_partial, int64_t n_step_partials, double eps, void* ws,
                         double* energy_dev, double* score_dev, hipStream_t s);

}  // namespace track
