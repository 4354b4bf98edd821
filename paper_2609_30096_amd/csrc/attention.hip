// Non-causal attention softmax(q k^T / sqrt(dh)) v for the DiT's 3D
// self-attention and text cross-attention.
//
// bfloat16 path (dh = 128): a flash-style kernel on CDNA4 matrix cores.  Each
// wave owns QG groups of 32 queries.  Per 64-key tile it forms the transposed
// logits S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (K tile from LDS as the
// MFMA "A" operand, the wave's Q fragments held in registers as "B"), so each
// lane's accumulators belong to a single query: the running max and sum of
// the online softmax stay per lane and only the max is exchanged between the
// two half-waves.  The probabilities are packed to bf16 in place and used as
// the "B" operand of O^T += V^T P^T, with V^T read from LDS; V arrives
// pre-transposed ([dh, keys]) so those reads are contiguous.  K and V^T tiles
// are double buffered in LDS with XOR swizzles that keep the 32-row fragment
// reads conflict free; the next tile's global loads are issued before the
// current tile's MFMAs.
#include <math.h>

#include <cstdlib>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace track {

constexpr int ATT_D = 128;
constexpr float ATT_TAU = 8.0f;  // log2 headroom before the running max is moved (lazy rescale)

// Max of a value and the value held by the lane 32 positions away.
__device__ __forceinline__ float halfwave_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}

__device__ __forceinline__ float halfwave_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// NW waves of 32 queries each; BKV keys per LDS tile (a multiple of 32).
// KIND (0 self, 1 cross) only separates the two uses in profiler output.
// PRIO: 0 none; 1 waves of the first half of the workgroup run at raised
// priority, so the two waves sharing a SIMD drift out of phase (one issues
// MFMAs while the other runs the softmax); 2 priority raised while a wave
// issues its MFMA blocks.
template <int NW, int BKV, int KIND, int PRIO>
__global__ __launch_bounds__(NW * 64) void flash_attn_bf16_kernel(const bf16_t* __restrict__ q, int64_t ldq,
                                                                  const bf16_t* __restrict__ k, int64_t ldk,
                                                                  const bf16_t* __restrict__ vt, int64_t ldv,
                                                                  bf16_t* __restrict__ out, int64_t ldo, int H,
                                                                  int Lq, int Lk, float scale_log2) {
  constexpr int D = ATT_D;
  constexpr int NT = NW * 64;
  constexpr int BQ = 32 * NW;
  constexpr int NSB = BKV / 32;         // 32-key sub-blocks per tile
  constexpr int K_BYTES = BKV * D * 2;  // [BKV keys][128] bf16, 256-byte rows
  constexpr int VROW = BKV * 2;         // V^T rows: [128 d][BKV keys] bf16
  constexpr int V_BYTES = D * VROW;
  constexpr int BUF = K_BYTES + V_BYTES;
  constexpr int KCPT = BKV * 16 / NT;   // 16-byte K chunks per thread per tile
  constexpr int VCH = BKV / 8;          // 16-byte chunks (units) per V^T row
  constexpr int VCPT = D * VCH / NT;
  static_assert(KCPT >= 1 && VCPT >= 1, "tile too small for the workgroup");
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * BUF];
  // 16-byte unit swizzle of V^T rows: any 8 consecutive rows get distinct
  // units, and rows r, r + 8 (same bank half at 128-byte rows) differ too, so
  // fragment reads are conflict free for 8 or 16 lanes per LDS cycle.
  auto vswz = [](int row) { return ((row & 7) ^ ((row >> 3) & 1)) & (VCH - 1); };

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int jq = lane & 31;
  const int hf = lane >> 5;
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  const int q0 = blockIdx.x * BQ + wave * 32;

  if constexpr (PRIO == 1) {
    if (wave < NW / 2) __builtin_amdgcn_s_setprio(1);
  }
  const bf16_t* kbase = k + (int64_t)b * Lk * ldk + (int64_t)h * D;
  const bf16_t* vbase = vt + ((int64_t)b * H + h) * D * ldv;

  // this wave's query fragments (B operand of S^T = K Q^T)
  bf16x8 qf[D / 16];
  {
    const int qi = min(q0 + jq, Lq - 1);
    const bf16_t* qp = q + (int64_t)b * Lq * ldq + (int64_t)h * D + (int64_t)qi * ldq + hf * 8;
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) qf[kc] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + kc * 16));
  }

  u32x4 rk[KCPT], rv[VCPT];
  auto load_global = [&](int key0) {
    const bf16_t* kp = kbase + (int64_t)key0 * ldk;
    const bool clamp = key0 + BKV > Lk;
#pragma unroll
    for (int i = 0; i < KCPT; ++i) {
      const int idx = tid + NT * i;
      int r = idx >> 4;
      if (clamp) r = min(r, Lk - 1 - key0);
      rk[i] = *(const u32x4*)(kp + (int64_t)r * ldk + (idx & 15) * 8);
    }
    const bool vclamp = key0 + BKV > ldv;  // keep V^T reads inside the row; those keys are masked
#pragma unroll
    for (int i = 0; i < VCPT; ++i) {
      const int idx = tid + NT * i;
      int col = key0 + (idx % VCH) * 8;
      if (vclamp) col = min(col, (int)ldv - 8);
      rv[i] = *(const u32x4*)(vbase + (int64_t)(idx / VCH) * ldv + col);
    }
  };
  auto store_lds = [&](int buf) {
    uint8_t* kb = smem + buf * BUF;
    uint8_t* vb = kb + K_BYTES;
#pragma unroll
    for (int i = 0; i < KCPT; ++i) {
      const int idx = tid + NT * i;
      const int krow = idx >> 4, kch = idx & 15;
      *(u32x4*)(kb + krow * 256 + ((kch ^ (krow & 15)) << 4)) = rk[i];
    }
#pragma unroll
    for (int i = 0; i < VCPT; ++i) {
      // global chunk j = keys 8j..8j+7.  Within each 16-key group c, 16-byte
      // unit 2c holds keys {0-3, 8-11} and unit 2c+1 keys {4-7, 12-15}: the
      // two runs one half-wave needs for a P V operand sit side by side.
      const int idx = tid + NT * i;
      const int vrow = idx / VCH, j = idx % VCH;
      const int sw = vswz(vrow);
      uint8_t* rowp = vb + vrow * VROW + (j & 1) * 8;
      *(u32x2*)(rowp + (((j & ~1) ^ sw) << 4)) = u32x2{rv[i][0], rv[i][1]};
      *(u32x2*)(rowp + ((((j & ~1) + 1) ^ sw) << 4)) = u32x2{rv[i][2], rv[i][3]};
    }
  };

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m_i = -INFINITY, l_i = 0.0f;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  const int ntiles = (Lk + BKV - 1) / BKV;

  // One tile: S^T for its NSB 32-key blocks (independent MFMA chains over the
  // head dimension), one online-softmax update, then O^T += V^T P^T.
  // MASK: keys at or past Lk get -inf logits (last tile only).
  auto tile = [&](int t, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int cur = t & 1;
    const int key0 = t * BKV;
    if (t + 1 < ntiles) load_global(key0 + BKV);
    const uint8_t* kb = smem + cur * BUF;
    const uint8_t* vb = kb + K_BYTES;

    // lane holds query jq and keys 32 sb + 8 (r/4) + 4 hf + r%4
    if constexpr (PRIO == 2) __builtin_amdgcn_s_setprio(1);
    f32x16 s[NSB];
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[sb][r] = 0.0f;
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
#pragma unroll
      for (int sb = 0; sb < NSB; ++sb) {
        const int row = sb * 32 + jq;
        const int ch = kc * 2 + hf;
        const bf16x8 kf = __builtin_bit_cast(bf16x8, *(const u32x4*)(kb + row * 256 + ((ch ^ (row & 15)) << 4)));
        s[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[kc], s[sb], 0, 0, 0);
      }
    }

    if constexpr (PRIO == 2) __builtin_amdgcn_s_setprio(0);
    float mx = -INFINITY;
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        if constexpr (MASK) {
          if (key0 + 32 * sb + 8 * (r >> 2) + 4 * hf + (r & 3) >= Lk) s[sb][r] = -INFINITY;
        }
        mx = fmaxf(mx, s[sb][r]);
      }
    const float mt = halfwave_max(mx) * scale_log2;
    // move the running max only when it grows by more than ATT_TAU (wave-uniform branch)
    if (__ballot(mt > m_i + ATT_TAU)) {
      const float mn = fmaxf(m_i, mt);
      const float alpha = __builtin_amdgcn_exp2f(m_i - mn);
      m_i = mn;
      l_i *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
    }
    const float nm = -m_i;
    // P as B operands: chunk c of 16 keys = keys 16c + 4 hf + {0..3} then 16c + 8 + 4 hf + {0..3}
    bf16x8 pf[2 * NSB];
#pragma unroll
    for (int c = 0; c < 2 * NSB; ++c) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float p0 = __builtin_amdgcn_exp2f(fmaf(s[c >> 1][(c & 1) * 8 + 2 * e], scale_log2, nm));
        const float p1 = __builtin_amdgcn_exp2f(fmaf(s[c >> 1][(c & 1) * 8 + 2 * e + 1], scale_log2, nm));
        const bf16x2 pb = __builtin_convertvector(f32x2{p0, p1}, bf16x2);
        // the row sum is taken over the rounded probabilities that enter P V
        l_i = __builtin_amdgcn_fdot2_f32_bf16(pb, ones2, l_i, false);
        w[e] = __builtin_bit_cast(uint32_t, pb);
      }
      pf[c] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    }
    if constexpr (PRIO == 2) __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int row = db * 32 + jq;
      const int sw = vswz(row);
#pragma unroll
      for (int c = 0; c < 2 * NSB; ++c) {
        const bf16x8 vf = __builtin_bit_cast(bf16x8, *(const u32x4*)(vb + row * VROW + (((2 * c + hf) ^ sw) << 4)));
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[c], o[db], 0, 0, 0);
      }
    }

    if constexpr (PRIO == 2) __builtin_amdgcn_s_setprio(0);
    if (t + 1 < ntiles) store_lds(cur ^ 1);
    __syncthreads();
  };

  load_global(0);
  store_lds(0);
  __syncthreads();
  for (int t = 0; t < ntiles - 1; ++t) tile(t, std::false_type{});
  if (Lk % BKV) tile(ntiles - 1, std::true_type{});
  else tile(ntiles - 1, std::false_type{});

  // normalise and store: lane holds query jq, channels 32 db + 8 (r/4) + 4 hf + r%4
  const float inv = 1.0f / halfwave_sum(l_i);
  const int qi = q0 + jq;
  if (qi < Lq) {
    bf16_t* op = out + (int64_t)b * Lq * ldo + (int64_t)h * D + (int64_t)qi * ldo;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int c0 = db * 32 + 8 * rg + 4 * hf;
        u32x2 pk;
        pk[0] = pack_bf2(o[db][4 * rg + 0] * inv, o[db][4 * rg + 1] * inv);
        pk[1] = pack_bf2(o[db][4 * rg + 2] * inv, o[db][4 * rg + 3] * inv);
        *(u32x2*)(op + c0) = pk;
      }
  }
}

// float32 path: one thread per query, online softmax over all keys.
template <int D>
__global__ __launch_bounds__(64) void attn_f32_kernel(const float* __restrict__ q, int64_t ldq,
                                                      const float* __restrict__ k, int64_t ldk,
                                                      const float* __restrict__ vt, int64_t ldv,
                                                      float* __restrict__ out, int64_t ldo, int H, int64_t Lq,
                                                      int64_t Lk, float scale) {
  const int64_t qi = (int64_t)blockIdx.x * 64 + threadIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  if (qi >= Lq) return;
  float qv[D], o[D];
  const float* qp = q + ((int64_t)b * Lq + qi) * ldq + (int64_t)h * D;
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qv[c] = qp[c];
    o[c] = 0.0f;
  }
  const float* kb = k + (int64_t)b * Lk * ldk + (int64_t)h * D;
  const float* vb = vt + ((int64_t)b * H + h) * D * ldv;
  float m = -INFINITY, l = 0.0f;
  for (int64_t j = 0; j < Lk; ++j) {
    float sdot = 0.0f;
#pragma unroll
    for (int c = 0; c < D; ++c) sdot = fmaf(qv[c], kb[j * ldk + c], sdot);
    sdot *= scale;
    const float mnew = fmaxf(m, sdot);
    const float a = expf(m - mnew);
    const float p = expf(sdot - mnew);
    l = l * a + p;
#pragma unroll
    for (int c = 0; c < D; ++c) o[c] = fmaf(p, vb[(int64_t)c * ldv + j], o[c] * a);
    m = mnew;
  }
  float* op = out + ((int64_t)b * Lq + qi) * ldo + (int64_t)h * D;
  const float inv = 1.0f / l;
#pragma unroll
  for (int c = 0; c < D; ++c) op[c] = o[c] * inv;
}

// Key-tile length of the bf16 kernel: 0 = 64 keys (default), 1 = 128 keys.
// TRACK_ATTN_CFG overrides the default (for tuning runs).
static int attn_config() {
  static const int cfg = [] {
    const char* e = getenv("TRACK_ATTN_CFG");
    const int v = e ? atoi(e) : 0;
    return (v == 0 || v == 1) ? v : 0;
  }();
  return cfg;
}

// Wave-priority scheme of the bf16 kernel (see the PRIO template parameter);
// TRACK_ATTN_PRIO overrides the default for tuning runs.
static int attn_prio() {
  static const int p = [] {
    const char* e = getenv("TRACK_ATTN_PRIO");
    const int v = e ? atoi(e) : 0;
    return (v >= 0 && v <= 2) ? v : 0;
  }();
  return p;
}

track_status attention(int dtype, int B, int H, int head_dim, int64_t Lq, int64_t Lk, const void* q, int64_t ldq,
                       const void* k, int64_t ldk, const void* vt, int64_t ldv, void* out, int64_t ldo,
                       hipStream_t s, int prof_kind) {
  if (B < 1 || H < 1 || Lq < 0 || Lk < 1) return fail(TRACK_E_SHAPE, "attention: bad sizes B=%d H=%d Lq=%lld Lk=%lld", B, H, (long long)Lq, (long long)Lk);
  if (!q || !k || !vt || !out) return fail(TRACK_E_INVALID, "attention: null pointer");
  const int64_t width = (int64_t)H * head_dim;
  if (ldq < width || ldk < width || ldo < width || ldv < Lk) return fail(TRACK_E_SHAPE, "attention: leading dimension too small");
  if (Lq == 0) return TRACK_OK;
  ProfScope prof(prof_kind, s);
  if (dtype == TRACK_DTYPE_BF16) {
    if (head_dim != ATT_D) return fail(TRACK_E_UNSUPPORTED, "attention: bf16 path needs head_dim 128 (got %d)", head_dim);
    if (ldv % 8) return fail(TRACK_E_SHAPE, "attention: bf16 path needs ldv %% 8 == 0");
    if (ldq % 8 || ldk % 8 || ldo % 4 || ((uintptr_t)q & 15) || ((uintptr_t)k & 15) || ((uintptr_t)vt & 15) ||
        ((uintptr_t)out & 7))
      return fail(TRACK_E_INVALID, "attention: bf16 path needs 16-byte aligned rows");
    if (Lq > INT32_MAX / 2 || Lk > INT32_MAX / 2) return fail(TRACK_E_SHAPE, "attention: sequence too long");
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)head_dim));
    const int cross = prof_kind == TRACK_PROF_ATTN_CROSS;
    const int cfg = attn_config();
    constexpr int NW = 8;
    const int BQ = 32 * NW;
    const int bkv = cfg == 0 ? 64 : 128;
    dim3 grid((unsigned)((Lq + BQ - 1) / BQ), H, B);
    const bf16_t *qq = (const bf16_t*)q, *kk = (const bf16_t*)k, *vv = (const bf16_t*)vt;
    bf16_t* oo = (bf16_t*)out;
#define TRACK_FA(BKV_, KIND_, PRIO_)                                                                        \
  flash_attn_bf16_kernel<NW, BKV_, KIND_, PRIO_><<<grid, NW * 64, 0, s>>>(qq, ldq, kk, ldk, vv, ldv, oo, ldo, H, \
                                                                         (int)Lq, (int)Lk, scale_log2)
    const int prio = attn_prio();
    if (bkv == 64) {
      if (prio == 1) { if (cross) TRACK_FA(64, 1, 1); else TRACK_FA(64, 0, 1); }
      else if (prio == 2) { if (cross) TRACK_FA(64, 1, 2); else TRACK_FA(64, 0, 2); }
      else { if (cross) TRACK_FA(64, 1, 0); else TRACK_FA(64, 0, 0); }
    } else {
      if (cross) TRACK_FA(128, 1, 0); else TRACK_FA(128, 0, 0);
    }
#undef TRACK_FA
    TRACK_LAUNCH_CHECK();
    return TRACK_OK;
  }
  if (dtype != TRACK_DTYPE_F32) return fail(TRACK_E_INVALID, "attention: bad dtype %d", dtype);
  dim3 grid((unsigned)((Lq + 63) / 64), H, B);
  const float scale = (float)(1.0 / sqrt((double)head_dim));
#define TRACK_ATT_F32(DH)                                                                                     \
  attn_f32_kernel<DH><<<grid, 64, 0, s>>>((const float*)q, ldq, (const float*)k, ldk, (const float*)vt, ldv, \
                                          (float*)out, ldo, H, Lq, Lk, scale)
  switch (head_dim) {
    case 32: TRACK_ATT_F32(32); break;
    case 64: TRACK_ATT_F32(64); break;
    case 128: TRACK_ATT_F32(128); break;
    default: return fail(TRACK_E_UNSUPPORTED, "attention: float32 path supports head_dim 32, 64, 128 (got %d)", head_dim);
  }
#undef TRACK_ATT_F32
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

}  // namespace track
