// Non-causal attention softmax(q k^T / sqrt(dh)) v for the DiT's 3D
// self-attention and text cross-attention.
//
// bfloat16 path (dh = 128): a flash-style kernel on CDNA4 matrix cores.  A
// workgroup of 8 waves owns 256 queries, 32 per wave.  Per 64-key tile each
// wave forms the transposed logits S^T = K Q^T with v_mfma_f32_32x32x16_bf16
// (K tile from LDS as the MFMA "A" operand, the wave's Q fragments held in
// registers as "B"), so each lane's accumulators belong to a single query: the
// running max of the online softmax stays per lane and only the max is
// exchanged between the two half-waves.  The reference max moves only when a
// tile's max exceeds it by more than ATT_TAU (log2 units), which bounds every
// probability by 2^ATT_TAU and spares most rescales of O; while a row's max
// stays within [ATT_MLO, ATT_TAU] the reference is 0.  With QLOG2 q arrives
// multiplied by the softmax scale log2(e) / sqrt(dh) (the forward's RMSNorm
// writes it so, inside its one rounding): the logits leave the MFMAs in log2
// units and a row with reference 0 takes each probability as the plain exp2
// of its logit, with no per-element scale or shift.  Without QLOG2 each
// probability is exp2 of one FMA (logit times scale, minus the reference).
// The probabilities are packed to bf16 and used as the "B" operand of
// O^T += V^T P^T, with V^T read from LDS; V arrives pre-transposed
// ([dh, keys]).  The softmax
// denominators are sums of those same bf16 probabilities, formed on the
// matrix cores too: a 16x16x32 MFMA per 16-key chunk with a 0/1 selector as
// "A" (v_dot2 row sums would wait for the other wave's MFMAs; the MFMA
// keeps the softmax to instructions that run beside them).
#include <math.h>

#include <algorithm>
#include <cstdlib>

#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace track {

constexpr int ATT_D = 128;
// log2 headroom before the reference max is moved (lazy rescale): probabilities
// stay below 2^64, which bf16 P and the float32 sums of up to 2^31 keys carry
constexpr float ATT_TAU = 64.0f;
constexpr float ATT_MLO = -64.0f;  // below this row max the reference leaves 0

// Max of a value and the value held by the lane 32 positions away.
__device__ __forceinline__ float halfwave_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  const float a = __uint_as_float(r[0]), b = __uint_as_float(r[1]);
  return a > b ? a : b;
}

// K and V^T tiles travel from global memory straight into LDS
// (buffer_load ... lds, 16 bytes per lane) through a ring of two slots, with
// no register staging and no LDS store instructions.  Per tile the K source
// is a buffer resource starting at the tile's first key, so keys past Lk read
// as zero; V^T columns are addressed through the vector offset (row and
// column together), so the resource's range check covers every V^T read.
// A DMA copy lands lane-contiguously, so every layout choice is made on the
// source side: each lane picks the 16-byte chunk that belongs at its LDS
// position.  The XOR swizzles keep the 32-row fragment reads conflict free:
// K rows are 256 bytes (unit u of row r at u ^ (r & 15)); V^T rows are 128
// bytes, and any 8 consecutive rows, as well as rows r and r + 8, get
// distinct units.  Each lane's fragment offsets are computed once; the tile
// loop is unrolled by two so the slot offset is an instruction immediate.
// To make each half-wave's P operand cover 8 consecutive keys (one contiguous
// 16-byte V^T chunk), the K tile's rows are a permutation of its keys: within
// every 16 keys, LDS rows 4..7 hold keys 8..11 and rows 8..11 hold keys
// 4..7.  Softmax and P V are indifferent to the order of keys as long as K
// and V agree, and the row a logit came from is mapped back to its key only
// for tail masking.
__device__ __forceinline__ int key_of_row(int row) {
  const int a = (row >> 2) & 3;
  return (row & ~15) | ((((a & 1) << 1) | (a >> 1)) << 2) | (row & 3);
}

typedef __attribute__((address_space(3))) void* att_lds_ptr_t;

template <int N>
__device__ __forceinline__ void att_wait_vmcnt() {
  // s_waitcnt vmcnt(N) (gfx9 encoding), expcnt and lgkmcnt not waited on
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

constexpr int ATT_NW = 8, ATT_BKV = 64, ATT_NSB = 2;
constexpr int ATT_BQ = 32 * ATT_NW;                 // queries per workgroup
constexpr int ATT_K_BYTES = ATT_BKV * ATT_D * 2;    // K tile, 16 KB
constexpr int ATT_VROW = ATT_BKV * 2;               // V^T tile row, 128 bytes
constexpr int ATT_V_BYTES = ATT_D * ATT_VROW;       // V^T tile, 16 KB
constexpr int ATT_SLOT = ATT_K_BYTES + ATT_V_BYTES;  // one ring slot, 32 KB
constexpr int ATT_VCH = ATT_BKV / 8;
// key sequences of at most this many 64-key tiles (an even number) take the item-loop kernel
constexpr int ATT_ITEMS_MAX_TILES = 32;

__device__ __forceinline__ int att_vswz(int row) { return ((row & 7) ^ ((row >> 3) & 1)) & (ATT_VCH - 1); }

// One 64-key tile for one wave's 32 queries: S^T = K Q^T from the slot's K
// tile, the online-softmax update (lazy rescale), and O^T += V^T P^T from the
// slot's V^T tile.  kfo / vfo are the lane's fragment offsets within a tile;
// with MASK, keys at or past Lk get probability zero.
typedef float att_f32x4 __attribute__((ext_vector_type(4)));
// Selector for the row sums: as the A operand of v_mfma_f32_16x16x32_bf16
// (lane l supplies row l % 16, k-block l / 16) it is 1 in row 0 for k-blocks 0
// and 2 and in row 1 for k-blocks 1 and 3; with a P operand of the 32x32x16
// layout as B (lane l: query l % 32, keys 8 (l / 32) .. + 7 of a 16-key chunk)
// the product holds in row 0, column n the sum over the chunk for query n and
// in row 1 that for query n + 16.
__device__ __forceinline__ bf16x8 att_sum_selector(int lane) {
  const int m = lane & 15, kb = lane >> 4;
  const float v = ((m == 0 && (kb & 1) == 0) || (m == 1 && (kb & 1) == 1)) ? 1.0f : 0.0f;
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)v;
  return r;
}
// The row sum of the lane's query (l % 32) from the accumulated selector products.
__device__ __forceinline__ float att_row_sum(att_f32x4 ls, int lane) {
  const int q = lane & 31;
  const float a = __shfl(ls[0], q & 15), b = __shfl(ls[1], q & 15);
  return q < 16 ? a : b;
}

template <bool MASK, bool QLOG2>
__device__ __forceinline__ void att_tile(const uint8_t* kb, const bf16x8 (&qf)[ATT_D / 16],
                                         const uint32_t (&kfo)[ATT_D / 16], const uint32_t (&vfo)[2 * ATT_NSB],
                                         f32x16 (&o)[ATT_D / 32], float& m_i, float& thr, bool& zref, att_f32x4& lsum,
                                         const bf16x8& sel, int key0, int Lk, int hf, float scale_log2) {
  constexpr int D = ATT_D, NSB = ATT_NSB;
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const uint8_t* vb = kb + ATT_K_BYTES;
  f32x16 s[NSB];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
    for (int r = 0; r < 16; ++r) s[sb][r] = 0.0f;
  auto kfrag = [&](int kc, int sb) {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)(kb + sb * 8192 + kfo[kc]));
  };
  bf16x8 kf[2][NSB];
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb) kf[0][sb] = kfrag(0, sb);
#pragma unroll
  for (int kc = 0; kc < D / 16; ++kc) {
    if (kc + 1 < D / 16) {
#pragma unroll
      for (int sb = 0; sb < NSB; ++sb) kf[(kc + 1) & 1][sb] = kfrag(kc + 1, sb);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int sb = 0; sb < NSB; ++sb)
      s[sb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kc & 1][sb], qf[kc], s[sb], 0, 0, 0);
  }
  float mx = -INFINITY;
#pragma unroll
  for (int sb = 0; sb < NSB; ++sb)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (MASK) {
        if (key0 + key_of_row(32 * sb + 8 * (r >> 2) + 4 * hf + (r & 3)) >= Lk) s[sb][r] = -INFINITY;
      }
      mx = fmaxf(mx, s[sb][r]);
    }
  const float mt = QLOG2 ? halfwave_max(mx) : halfwave_max(mx) * scale_log2;
  if (__ballot(mt > thr)) {
    float mn = fmaxf(m_i, mt);
    if (mn >= ATT_MLO && mn <= ATT_TAU) mn = 0.0f;
    const float alpha = __builtin_amdgcn_exp2f(m_i - mn);
    m_i = mn;
    thr = mn + ATT_TAU;
    zref = !__ballot(mn != 0.0f);
    const float alpha_hi = __shfl_down(alpha, 16);  // lane n holds the sums of queries n and n + 16
    lsum[0] *= alpha;
    lsum[1] *= alpha_hi;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] *= alpha;
  }
  // probabilities exp2(s - m) (QLOG2; the shift only where some row of the
  // wave has a nonzero reference, a wave-uniform branch), or exp2(s c - m)
  const float nm = -m_i;
  bf16x8 pf[2 * NSB];
  auto probs = [&](auto shift_tag) {
#pragma unroll
    for (int c = 0; c < 2 * NSB; ++c) {
      uint32_t w[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float x0 = s[c >> 1][(c & 1) * 8 + 2 * e], x1 = s[c >> 1][(c & 1) * 8 + 2 * e + 1];
        if constexpr (!QLOG2) {
          x0 = fmaf(x0, scale_log2, nm);
          x1 = fmaf(x1, scale_log2, nm);
        } else if constexpr (decltype(shift_tag)::value) {
          x0 += nm;
          x1 += nm;
        }
        const bf16x2 pb = __builtin_convertvector(f32x2{__builtin_amdgcn_exp2f(x0), __builtin_amdgcn_exp2f(x1)}, bf16x2);
        w[e] = __builtin_bit_cast(uint32_t, pb);
      }
      pf[c] = __builtin_bit_cast(bf16x8, u32x4{w[0], w[1], w[2], w[3]});
    }
  };
  if (QLOG2 && zref) probs(std::false_type{});
  else probs(std::true_type{});
#pragma unroll
  for (int c = 0; c < 2 * NSB; ++c) lsum = __builtin_amdgcn_mfma_f32_16x16x32_bf16(sel, pf[c], lsum, 0, 0, 0);
  auto vfrag = [&](int db, int c) {
    return __builtin_bit_cast(bf16x8, *(const u32x4*)(vb + db * 4096 + vfo[c]));
  };
  bf16x8 vf[2][2 * NSB];
#pragma unroll
  for (int c = 0; c < 2 * NSB; ++c) vf[0][c] = vfrag(0, c);
#pragma unroll
  for (int db = 0; db < D / 32; ++db) {
    if (db + 1 < D / 32) {
#pragma unroll
      for (int c = 0; c < 2 * NSB; ++c) vf[(db + 1) & 1][c] = vfrag(db + 1, c);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c = 0; c < 2 * NSB; ++c)
      o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf[db & 1][c], pf[c], o[db], 0, 0, 0);
  }
}

template <int KIND, bool QLOG2>
__global__ __launch_bounds__(512) void flash_attn_bf16_kernel(const bf16_t* __restrict__ q, int64_t ldq,
                                                      const bf16_t* __restrict__ k, int64_t ldk,
                                                      const bf16_t* __restrict__ vt, int64_t ldv,
                                                      bf16_t* __restrict__ out, int64_t ldo, int H,
                                                      int Lq, int Lk, float scale_log2) {
  constexpr int BKV = ATT_BKV, NSB = ATT_NSB, D = ATT_D, BQ = ATT_BQ;
  constexpr int K_BYTES = ATT_K_BYTES, VROW = ATT_VROW, SLOT = ATT_SLOT;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * SLOT];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int jq = lane & 31;
  const int hf = lane >> 5;
  const int h = blockIdx.y;
  const int b = blockIdx.z;
  const int q0 = blockIdx.x * BQ + wave * 32;

  const bf16_t* kbase = k + (int64_t)b * Lk * ldk + (int64_t)h * D;
  const bf16_t* vbase = vt + ((int64_t)b * H + h) * D * ldv;

  bf16x8 qf[D / 16];
  {
    const int qi = min(q0 + jq, Lq - 1);
    const bf16_t* qp = q + (int64_t)b * Lq * ldq + (int64_t)h * D + (int64_t)qi * ldq + hf * 8;
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) qf[kc] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qp + kc * 16));
  }
  // copy i (0, 1) of this wave fills its 1 KB block 2 wave + i of the K (or
  // V^T) region; per-lane byte offsets within the tile's rows
  uint32_t koffg[2], voffg[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = 8 * wave + 4 * i + (lane >> 4);
    koffg[i] = (uint32_t)((key_of_row(row) * ldk + ((lane & 15) ^ (row & 15)) * 8) * 2);
    const int vr = 16 * wave + 8 * i + (lane >> 3);
    voffg[i] = (uint32_t)((vr * ldv + ((lane & 7) ^ att_vswz(vr)) * 8) * 2);
  }
  const int ntiles = (Lk + BKV - 1) / BKV;
  // V^T of this (batch, head): D rows of ldv keys
  // (the host keeps D * ldv * 2 and Lk * ldk * 2 below 2^32, the size field's range)
  const __amdgpu_buffer_rsrc_t rsV =
      __builtin_amdgcn_make_buffer_rsrc((void*)vbase, (short)0, (int)(uint32_t)(D * ldv * 2), 0x00020000);
  // tile t (past the end: the last tile again) into slot S
  auto issue = [&](int t, auto slot_tag) {
    constexpr int S = decltype(slot_tag)::value;
    const int tt = min(t, ntiles - 1);
    const int key0 = tt * BKV;
    // K rows key0 .. Lk - 1 of this head; rows past Lk read as zero
    const __amdgpu_buffer_rsrc_t rsK = __builtin_amdgcn_make_buffer_rsrc((void*)(kbase + (int64_t)key0 * ldk), (short)0,
                                                                         (int)(uint32_t)((Lk - key0) * ldk * 2), 0x00020000);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsK, (att_lds_ptr_t)(smem + S * SLOT + wave * 2048 + i * 1024), 16, koffg[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsV, (att_lds_ptr_t)(smem + S * SLOT + K_BYTES + wave * 2048 + i * 1024), 16,
                                               voffg[i] + (uint32_t)(key0 * 2), 0, 0, 0);
  };

  // per-lane LDS fragment offsets (slot and 32-row block are immediates)
  uint32_t kfo[D / 16], vfo[2 * NSB];
#pragma unroll
  for (int kc = 0; kc < D / 16; ++kc) kfo[kc] = jq * 256 + (((kc * 2 + hf) ^ (jq & 15)) << 4);
#pragma unroll
  for (int c = 0; c < 2 * NSB; ++c) vfo[c] = jq * VROW + (((2 * c + hf) ^ att_vswz(jq)) << 4);

  f32x16 o[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
  float m_i = -INFINITY, thr = -INFINITY;  // reference max, and the tile max that moves it
  bool zref = false;                         // every row of the wave has reference 0
  att_f32x4 lsum = {0.0f, 0.0f, 0.0f, 0.0f};
  const bf16x8 sel = att_sum_selector(lane);

  auto subtile = [&](auto slot_tag, int key0, auto mask_tag) {
    constexpr int S = decltype(slot_tag)::value;
    att_tile<decltype(mask_tag)::value, QLOG2>(smem + S * SLOT, qf, kfo, vfo, o, m_i, thr, zref, lsum, sel, key0, Lk, hf,
                                               scale_log2);
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  // tile t in slot S: copy tile t + 1 into the other slot (every wave is past
  // tile t - 1, its last reader), compute, wait for the copy, barrier
  auto tile = [&](int t, auto slot_tag, auto mask_tag) {
    constexpr int S = decltype(slot_tag)::value;
    issue(t + 1, std::integral_constant<int, 1 - S>{});
    subtile(slot_tag, t * BKV, mask_tag);
    att_wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt((15 << 0) | (3 << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
  };

  issue(0, S0{});
  att_wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  const int last = ntiles - 1;
  int t = 0;
  for (; t + 1 < last; t += 2) {
    tile(t, S0{}, std::false_type{});
    tile(t + 1, S1{}, std::false_type{});
  }
  if (t < last) {  // one unmasked tile left (in slot 0)
    tile(t, S0{}, std::false_type{});
    ++t;
  }
  // the last tile, in slot t & 1
  if (Lk % BKV) {
    if (t & 1) tile(t, S1{}, std::true_type{});
    else tile(t, S0{}, std::true_type{});
  } else {
    if (t & 1) tile(t, S1{}, std::false_type{});
    else tile(t, S0{}, std::false_type{});
  }
  att_wait_vmcnt<0>();

  const float inv = 1.0f / att_row_sum(lsum, lane);
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

// Attention over a short key sequence (text cross-attention: Lk = 512, 8
// tiles).  With one workgroup per (query block, head, batch) as above, each
// workgroup would pay its Q load, the first tile's copy and its output stores
// for only 8 tiles.  Here one workgroup per CU walks the work items
// it = (b H + h) nqb + qb, taking p, p + G, p + 2G, ...; the K / V^T copy
// ring runs on from one item's last tile into the next item's first, and each
// wave copies the Q rows of its next item into LDS (buffer_load ... lds, rows
// past Lq read as zero) while the current item runs, so an item starts with 8
// LDS reads instead of a global load.  Every wave reads back only the Q rows
// that it copied itself, so those copies need no barrier.  ntiles must be
// even: a tile's ring slot is then its index within the item modulo 2.
template <int KIND, bool QLOG2>
__global__ __launch_bounds__(512) void flash_attn_items_kernel(const bf16_t* __restrict__ q, int64_t ldq,
                                                               const bf16_t* __restrict__ k, int64_t ldk,
                                                               const bf16_t* __restrict__ vt, int64_t ldv,
                                                               bf16_t* __restrict__ out, int64_t ldo, int H, int Lq,
                                                               int Lk, float scale_log2, int nitems) {
  constexpr int BKV = ATT_BKV, NSB = ATT_NSB, D = ATT_D, BQ = ATT_BQ;
  constexpr int K_BYTES = ATT_K_BYTES, VROW = ATT_VROW, SLOT = ATT_SLOT;
  constexpr int QROW = D * 2;  // 256-byte Q rows in LDS
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * SLOT + BQ * QROW];
  uint8_t* const qs = smem + 2 * SLOT;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int jq = lane & 31;
  const int hf = lane >> 5;
  const int nqb = (Lq + BQ - 1) / BQ;
  const int ntiles = (Lk + BKV - 1) / BKV;
  const int G = gridDim.x;
  // item -> (query block, head, batch); the divisions run on the vector ALU,
  // readfirstlane returns the (wave-uniform) results to scalar registers so the
  // buffer resources built from them stay scalar
  auto split = [&](int it, int& qb, int& h, int& b) {
    const int bh = __builtin_amdgcn_readfirstlane(it / nqb);
    qb = __builtin_amdgcn_readfirstlane(it - bh * nqb);
    b = __builtin_amdgcn_readfirstlane(bh / H);
    h = __builtin_amdgcn_readfirstlane(bh - b * H);
  };

  uint32_t koffg[2], voffg[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = 8 * wave + 4 * i + (lane >> 4);
    koffg[i] = (uint32_t)((key_of_row(row) * ldk + ((lane & 15) ^ (row & 15)) * 8) * 2);
    const int vr = 16 * wave + 8 * i + (lane >> 3);
    voffg[i] = (uint32_t)((vr * ldv + ((lane & 7) ^ att_vswz(vr)) * 8) * 2);
  }
  uint32_t kfo[D / 16], vfo[2 * NSB];
#pragma unroll
  for (int kc = 0; kc < D / 16; ++kc) kfo[kc] = jq * 256 + (((kc * 2 + hf) ^ (jq & 15)) << 4);
#pragma unroll
  for (int c = 0; c < 2 * NSB; ++c) vfo[c] = jq * VROW + (((2 * c + hf) ^ att_vswz(jq)) << 4);

  // K / V^T tile t of item it into slot S (no copy past the last item)
  auto issue = [&](int it, int t, auto slot_tag) {
    constexpr int S = decltype(slot_tag)::value;
    if (it >= nitems) return;
    int qb, h, b;
    split(it, qb, h, b);
    const int key0 = t * BKV;
    const __amdgpu_buffer_rsrc_t rsK =
        __builtin_amdgcn_make_buffer_rsrc((void*)(k + ((int64_t)b * Lk + key0) * ldk + (int64_t)h * D), (short)0,
                                          (int)(uint32_t)((Lk - key0) * ldk * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsV = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(vt + ((int64_t)b * H + h) * D * ldv), (short)0, (int)(uint32_t)(D * ldv * 2), 0x00020000);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsK, (att_lds_ptr_t)(smem + S * SLOT + wave * 2048 + i * 1024), 16,
                                               koffg[i], 0, 0, 0);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsV, (att_lds_ptr_t)(smem + S * SLOT + K_BYTES + wave * 2048 + i * 1024),
                                               16, voffg[i] + (uint32_t)(key0 * 2), 0, 0, 0);
  };
  // this wave's 32 Q rows of item it into LDS (rows past Lq read as zero)
  auto issue_q = [&](int it) {
    if (it >= nitems) return;
    int qb, h, b;
    split(it, qb, h, b);
    const int r0 = qb * BQ + wave * 32;
    const int nrows = __builtin_amdgcn_readfirstlane(max(0, min(32, Lq - r0)));  // (clamped on the vector ALU)
    const __amdgpu_buffer_rsrc_t rsQ =
        __builtin_amdgcn_make_buffer_rsrc((void*)(q + ((int64_t)b * Lq + r0) * ldq + (int64_t)h * D), (short)0,
                                          (int)(uint32_t)(nrows * ldq * 2), 0x00020000);
    // copy i (0..7) fills LDS rows 4 i .. 4 i + 3 of the wave's 32 (1 KB);
    // unit u of row r sits at u ^ (r & 15).  The lane index is made opaque so
    // that these offsets are formed here, not kept live across the tiles.
    int ln = lane;
    asm volatile("" : "+v"(ln));
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = 4 * i + (ln >> 4);
      const uint32_t off = (uint32_t)((r * ldq + ((ln & 15) ^ (r & 15)) * 8) * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsQ, (att_lds_ptr_t)(qs + wave * 32 * QROW + i * 1024), 16, off, 0, 0, 0);
    }
  };
  bf16x8 qf[D / 16];
  auto read_q = [&]() {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc)
      // the same row / unit layout as a K tile: kfo doubles as the offset
      qf[kc] = __builtin_bit_cast(bf16x8, *(const u32x4*)(qs + wave * 32 * QROW + kfo[kc]));
    __builtin_amdgcn_s_waitcnt((15 << 0) | (3 << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0): Q buffer free again
  };

  f32x16 o[D / 32];
  float m_i, thr;
  bool zref;
  att_f32x4 lsum;
  const bf16x8 sel = att_sum_selector(lane);
  auto reset = [&]() {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
    m_i = -INFINITY;
    thr = -INFINITY;
    zref = false;
    lsum = att_f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  // tile t of item it in slot S, the copy of the tile after it in flight
  auto tile = [&](int it, int t, auto slot_tag, auto mask_tag) {
    constexpr int S = decltype(slot_tag)::value;
    if (t + 1 < ntiles) issue(it, t + 1, std::integral_constant<int, 1 - S>{});
    else issue(it + G, 0, std::integral_constant<int, 1 - S>{});
    att_tile<decltype(mask_tag)::value, QLOG2>(smem + S * SLOT, qf, kfo, vfo, o, m_i, thr, zref, lsum, sel, t * BKV, Lk, hf,
                                               scale_log2);
    att_wait_vmcnt<0>();
    __builtin_amdgcn_s_waitcnt((15 << 0) | (3 << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
  };

  int it = blockIdx.x;
  issue_q(it);
  issue(it, 0, S0{});
  att_wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
  for (; it < nitems; it += G) {
    read_q();
    issue_q(it + G);
    reset();
    int t = 0;
    for (; t + 2 < ntiles; t += 2) {
      tile(it, t, S0{}, std::false_type{});
      tile(it, t + 1, S1{}, std::false_type{});
    }
    tile(it, t, S0{}, std::false_type{});
    if (Lk % BKV) tile(it, t + 1, S1{}, std::true_type{});
    else tile(it, t + 1, S1{}, std::false_type{});

    int qb, h, b;
    split(it, qb, h, b);
    const float inv = 1.0f / att_row_sum(lsum, lane);
    const int qi = qb * BQ + wave * 32 + jq;
    if (qi < Lq) {
      bf16_t* op = out + ((int64_t)b * Lq + qi) * ldo + (int64_t)h * D;
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
  att_wait_vmcnt<0>();
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

float attn_log2_scale(int head_dim) { return (float)(1.4426950408889634 / sqrt((double)head_dim)); }

track_status attention(int dtype, int B, int H, int head_dim, int64_t Lq, int64_t Lk, const void* q, int64_t ldq,
                       const void* k, int64_t ldk, const void* vt, int64_t ldv, void* out, int64_t ldo,
                       hipStream_t s, int prof_kind, bool q_log2) {
  if (B < 1 || H < 1 || Lq < 0 || Lk < 1) return fail(TRACK_E_SHAPE, "attention: bad sizes B=%d H=%d Lq=%lld Lk=%lld", B, H, (long long)Lq, (long long)Lk);
  if (!q || !k || !vt || !out) return fail(TRACK_E_INVALID, "attention: null pointer");
  const int64_t width = (int64_t)H * head_dim;
  if (ldq < width || ldk < width || ldo < width || ldv < Lk) return fail(TRACK_E_SHAPE, "attention: leading dimension too small");
  if (q_log2 && dtype != TRACK_DTYPE_BF16) return fail(TRACK_E_INVALID, "attention: pre-scaled q is a bf16-path input");
  if (Lq == 0) return TRACK_OK;
  ProfScope prof(prof_kind, s);
  if (dtype == TRACK_DTYPE_BF16) {
    if (head_dim != ATT_D) return fail(TRACK_E_UNSUPPORTED, "attention: bf16 path needs head_dim 128 (got %d)", head_dim);
    if (ldv % 8) return fail(TRACK_E_SHAPE, "attention: bf16 path needs ldv %% 8 == 0");
    if (ldq % 8 || ldk % 8 || ldo % 4 || ((uintptr_t)q & 15) || ((uintptr_t)k & 15) || ((uintptr_t)vt & 15) ||
        ((uintptr_t)out & 7))
      return fail(TRACK_E_INVALID, "attention: bf16 path needs 16-byte aligned rows");
    if (Lq > INT32_MAX / 2 || Lk > INT32_MAX / 2) return fail(TRACK_E_SHAPE, "attention: sequence too long");
    // the K and V^T copies address one head through 32-bit buffer offsets
    if (Lk * ldk * 2 > (int64_t)UINT32_MAX || (int64_t)ATT_D * ldv * 2 > (int64_t)UINT32_MAX)
      return fail(TRACK_E_SHAPE, "attention: K or V^T of one head spans more than 4 GiB");
    const float scale_log2 = attn_log2_scale(head_dim);
    const int cross = prof_kind == TRACK_PROF_ATTN_CROSS;
    dim3 grid((unsigned)((Lq + 255) / 256), H, B);
    const bf16_t *qq = (const bf16_t*)q, *kk = (const bf16_t*)k, *vv = (const bf16_t*)vt;
    bf16_t* oo = (bf16_t*)out;
    const int64_t ntiles = (Lk + ATT_BKV - 1) / ATT_BKV;
    // TRACK_ATTN_ITEMS=0 keeps short sequences on the per-block kernel (both
    // give identical bits; the tests compare them)
    const char* items_env = getenv("TRACK_ATTN_ITEMS");
    const bool items_ok = !(items_env && items_env[0] == '0');
    if (items_ok && ntiles % 2 == 0 && ntiles <= ATT_ITEMS_MAX_TILES) {
      // short key sequence: one workgroup per CU over all (query block, head, batch) items
      const int64_t nitems = (int64_t)grid.x * H * B;
      if (nitems > INT32_MAX) return fail(TRACK_E_SHAPE, "attention: too many query blocks");
      const int g = (int)std::min<int64_t>(nitems, device_cus());
#define TRACK_ATT_ITEMS(KIND, QL)                                                                               \
  flash_attn_items_kernel<KIND, QL><<<g, 512, 0, s>>>(qq, ldq, kk, ldk, vv, ldv, oo, ldo, H, (int)Lq, (int)Lk, \
                                                      scale_log2, (int)nitems)
      if (cross) {
        if (q_log2) TRACK_ATT_ITEMS(1, true);
        else TRACK_ATT_ITEMS(1, false);
      } else {
        if (q_log2) TRACK_ATT_ITEMS(0, true);
        else TRACK_ATT_ITEMS(0, false);
      }
#undef TRACK_ATT_ITEMS
    } else {
#define TRACK_ATT_BLOCKS(KIND, QL) \
  flash_attn_bf16_kernel<KIND, QL><<<grid, 512, 0, s>>>(qq, ldq, kk, ldk, vv, ldv, oo, ldo, H, (int)Lq, (int)Lk, scale_log2)
      if (cross) {
        if (q_log2) TRACK_ATT_BLOCKS(1, true);
        else TRACK_ATT_BLOCKS(1, false);
      } else {
        if (q_log2) TRACK_ATT_BLOCKS(0, true);
        else TRACK_ATT_BLOCKS(0, false);
      }
#undef TRACK_ATT_BLOCKS
    }
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
