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
constexpr int ATT_BKV = 64;
constexpr float ATT_TAU = 8.0f;  // log2 headroom before the running max is moved (lazy rescale)

// KIND (0 self, 1 cross) only separates the two uses in profiler output.
template <int QG, int NW, int KIND>
__global__ __launch_bounds__(NW * 64) void flash_attn_bf16_kernel(const bf16_t* __restrict__ q, int64_t ldq,
                                                                  const bf16_t* __restrict__ k, int64_t ldk,
                                                                  const bf16_t* __restrict__ vt, int64_t ldv,
                                                                  bf16_t* __restrict__ out, int64_t ldo, int H,
                                                                  int Lq, int Lk, float scale_log2) {
  constexpr int D = ATT_D, BKV = ATT_BKV;
  constexpr int NT = NW * 64;
  constexpr int BQ = 32 * QG * NW;
  constexpr int K_BYTES = BKV * D * 2;  // [64 keys][128] bf16, 256-byte rows
  constexpr int V_BYTES = D * BKV * 2;  // [128 d][64 keys] bf16, 128-byte rows
  constexpr int BUF = K_BYTES + V_BYTES;
  constexpr int CPT = 1024 / NT;        // 16-byte chunks per thread per tile (each of K and V^T)
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * BUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int jq = lane & 31;
  const int hf = lane >> 5;
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  const int q0 = blockIdx.x * BQ + wave * 32 * QG;

  const bf16_t* qbase = q + (int64_t)b * Lq * ldq + (int64_t)h * D;
  const bf16_t* kbase = k + (int64_t)b * Lk * ldk + (int64_t)h * D;
  const bf16_t* vbase = vt + ((int64_t)b * H + h) * D * ldv;

  // this wave's query fragments (B operand of S^T = K Q^T)
  bf16x8 qf[QG][D / 16];
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    const int qi = min(q0 + g * 32 + jq, Lq - 1);
    const bf16_t* qp = qbase + (int64_t)qi * ldq + hf * 8;
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) qf[g][kc] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + kc * 16));
  }

  // staging offsets (elements) of this thread's chunks
  int koff[CPT], voff[CPT], krow_[CPT];
#pragma unroll
  for (int i = 0; i < CPT; ++i) {
    const int idx = tid + NT * i;
    krow_[i] = idx >> 4;
    koff[i] = (idx & 15) * 8;
    voff[i] = (idx >> 3) * (int)ldv + (idx & 7) * 8;
  }
  u32x4 rk[CPT], rv[CPT];
  auto load_global = [&](int key0) {
    const bf16_t* kp = kbase + (int64_t)key0 * ldk;
    const bool clamp = key0 + BKV > Lk;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      int r = krow_[i];
      if (clamp) r = min(r, Lk - 1 - key0);
      rk[i] = *(const u32x4*)(kp + (int64_t)r * ldk + koff[i]);
      rv[i] = *(const u32x4*)(vbase + key0 + voff[i]);
    }
  };
  auto store_lds = [&](int buf) {
    uint8_t* kb = smem + buf * BUF;
    uint8_t* vb = kb + K_BYTES;
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      const int idx = tid + NT * i;
      const int krow = idx >> 4, kch = idx & 15;
      *(u32x4*)(kb + krow * 256 + ((kch ^ (krow & 15)) << 4)) = rk[i];
      const int vrow = idx >> 3, vch = idx & 7;
      const int sw = vrow & 15;
      *(u32x2*)(vb + vrow * 128 + (((2 * vch) ^ sw) << 3)) = u32x2{rv[i][0], rv[i][1]};
      *(u32x2*)(vb + vrow * 128 + (((2 * vch + 1) ^ sw) << 3)) = u32x2{rv[i][2], rv[i][3]};
    }
  };

  f32x16 o[QG][D / 32];
#pragma unroll
  for (int g = 0; g < QG; ++g)
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[g][db][r] = 0.0f;
  float m_i[QG], l_i[QG];
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    m_i[g] = -INFINITY;
    l_i[g] = 0.0f;
  }
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 ones2 = {(__bf16)1.0f, (__bf16)1.0f};

  const int ntiles = (Lk + BKV - 1) / BKV;

  // One 64-key tile.  MASK: keys at or past Lk get -inf logits (last tile only).
  auto tile = [&](int t, auto mask_tag) {
    constexpr bool MASK = decltype(mask_tag)::value;
    const int cur = t & 1;
    const int key0 = t * BKV;
    if (t + 1 < ntiles) load_global(key0 + BKV);
    const uint8_t* kb = smem + cur * BUF;
    const uint8_t* vb = kb + K_BYTES;

    f32x16 s[QG][2];
#pragma unroll
    for (int g = 0; g < QG; ++g)
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[g][kb2][r] = 0.0f;
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2) {
        const int row = kb2 * 32 + jq;
        const int ch = kc * 2 + hf;
        const bf16x8 kf = __builtin_bit_cast(bf16x8, *(const u32x4*)(kb + row * 256 + ((ch ^ (row & 15)) << 4)));
#pragma unroll
        for (int g = 0; g < QG; ++g) s[g][kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[g][kc], s[g][kb2], 0, 0, 0);
      }
    }

    // online softmax: lane holds query jq and keys 8 (r/4) + 4 hf + r%4 of each 32-key block
    bf16x8 pf[QG][4];
#pragma unroll
    for (int g = 0; g < QG; ++g) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if constexpr (MASK) {
            const int key = key0 + kb2 * 32 + 8 * (r >> 2) + 4 * hf + (r & 3);
            if (key >= Lk) s[g][kb2][r] = -INFINITY;
          }
          mx = fmaxf(mx, s[g][kb2][r]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mt = mx * scale_log2;
      // move the running max only when it grows by more than ATT_TAU (wave-uniform branch)
      if (__ballot(mt > m_i[g] + ATT_TAU)) {
        const float mn = fmaxf(m_i[g], mt);
        const float alpha = __builtin_amdgcn_exp2f(m_i[g] - mn);
        m_i[g] = mn;
        l_i[g] *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) o[g][db][r] *= alpha;
      }
      const float nm = -m_i[g];
      float lsum = 0.0f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        uint32_t w[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float p0 = __builtin_amdgcn_exp2f(fmaf(s[g][c >> 1][(c & 1) * 8 + 2 * e], scale_log2, nm));
          const float p1 = __builtin_amdgcn_exp2f(fmaf(s[g][c >> 1][(c & 1) * 8 + 2 * e + 1], scale_log2, nm));
          const bf16x2 pb = __builtin_convertvector(f32x2{p0, p1}, bf16x2);
          // the row sum is taken over the rounded probabilities that enter P V
          lsum = __builtin_amdgcn_fdot2_f32_bf16(pb, ones2, lsum, false);
          w[e] = __builtin_bit_cast(uint32_t, pb);
        }
        pf[g][c] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
      }
      l_i[g] += lsum;
    }

    // O^T += V^T P^T over 4 chunks of 16 keys: keys 16c + 4 hf + {0..3} and 16c + 8 + 4 hf + {0..3}
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const int row = db * 32 + jq;
      const int sw = row & 15;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const u32x2 lo = *(const u32x2*)(vb + row * 128 + (((4 * c + hf) ^ sw) << 3));
        const u32x2 hi = *(const u32x2*)(vb + row * 128 + (((4 * c + 2 + hf) ^ sw) << 3));
        const bf16x8 vf = __builtin_bit_cast(bf16x8, u32x4{lo[0], lo[1], hi[0], hi[1]});
#pragma unroll
        for (int g = 0; g < QG; ++g) o[g][db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[g][c], o[g][db], 0, 0, 0);
      }
    }

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
  bf16_t* obase = out + (int64_t)b * Lq * ldo + (int64_t)h * D;
#pragma unroll
  for (int g = 0; g < QG; ++g) {
    const float l = l_i[g] + __shfl_xor(l_i[g], 32, 64);
    const float inv = 1.0f / l;
    const int qi = q0 + g * 32 + jq;
    if (qi >= Lq) continue;
    bf16_t* op = obase + (int64_t)qi * ldo;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int rg = 0; rg < 4; ++rg) {
        const int c0 = db * 32 + 8 * rg + 4 * hf;
        u32x2 pk;
        pk[0] = pack_bf2(o[g][db][4 * rg + 0] * inv, o[g][db][4 * rg + 1] * inv);
        pk[1] = pack_bf2(o[g][db][4 * rg + 2] * inv, o[g][db][4 * rg + 3] * inv);
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

// Work shape of the bf16 kernel: 0 = 2 query groups x 4 waves, 1 = 1 x 8, 2 = 1 x 4.
// TRACK_ATTN_CFG overrides the default (for tuning runs).
static int attn_config() {
  static const int cfg = [] {
    const char* e = getenv("TRACK_ATTN_CFG");
    const int v = e ? atoi(e) : 1;
    return (v >= 0 && v <= 2) ? v : 1;
  }();
  return cfg;
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
    const int64_t need = (Lk + ATT_BKV - 1) / ATT_BKV * ATT_BKV;
    if (ldv < need || ldv % 8) return fail(TRACK_E_SHAPE, "attention: bf16 path needs ldv >= Lk rounded up to 64 and ldv %% 8 == 0");
    if (ldq % 8 || ldk % 8 || ldo % 4 || ((uintptr_t)q & 15) || ((uintptr_t)k & 15) || ((uintptr_t)vt & 15) ||
        ((uintptr_t)out & 7))
      return fail(TRACK_E_INVALID, "attention: bf16 path needs 16-byte aligned rows");
    if (Lq > INT32_MAX / 2 || Lk > INT32_MAX / 2) return fail(TRACK_E_SHAPE, "attention: sequence too long");
    const float scale_log2 = (float)(1.4426950408889634 / sqrt((double)head_dim));
    const int cross = prof_kind == TRACK_PROF_ATTN_CROSS;
    const int cfg = attn_config();
    const int qg = cfg == 0 ? 2 : 1, nw = cfg == 1 ? 8 : 4;
    const int BQ = 32 * qg * nw;
    dim3 grid((unsigned)((Lq + BQ - 1) / BQ), H, B);
    const bf16_t *qq = (const bf16_t*)q, *kk = (const bf16_t*)k, *vv = (const bf16_t*)vt;
    bf16_t* oo = (bf16_t*)out;
#define TRACK_FA(QG_, NW_, KIND_)                                                                                \
  flash_attn_bf16_kernel<QG_, NW_, KIND_><<<grid, NW_ * 64, 0, s>>>(qq, ldq, kk, ldk, vv, ldv, oo, ldo, H, (int)Lq, \
                                                                   (int)Lk, scale_log2)
    if (cfg == 0) { if (cross) TRACK_FA(2, 4, 1); else TRACK_FA(2, 4, 0); }
    else if (cfg == 1) { if (cross) TRACK_FA(1, 8, 1); else TRACK_FA(1, 8, 0); }
    else { if (cross) TRACK_FA(1, 4, 1); else TRACK_FA(1, 4, 0); }
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
