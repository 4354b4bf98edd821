// Projection GEMMs of the denoiser: out = epilogue(A W^T + b).
//
// A is the activation matrix [M tokens, K] and W a linear weight [N, K]
// (both K-contiguous).  The bfloat16 kernel runs on CDNA4 matrix cores
// (v_mfma_f32_32x32x16_bf16) with the weight tile as the MFMA "A" operand and
// the token tile as the "B" operand, so each lane's accumulators hold one
// token and runs of four consecutive output features; the epilogue then
// writes 8- or 16-byte vectors.  Epilogues fuse the bias, the tanh GELU of
// the MLP, and the adaLN gate with the float32 residual update; one variant
// stores the output transposed per batch (V^T for attention) through LDS.
#include <cstdlib>

#include "common.h"
#include "kernels.h"

namespace track {

struct EpiArgs {
  const void* bias;   // [N], weight dtype
  const float* gate;  // [N] float32 (gated residual only)
  void* out;          // output or residual
  int64_t ldo;
  // transposed output (EPI_BIAS_VT): column n of row m goes to
  // vt[((m / L) * N + n) * ldv + m % L], m counted from m_off
  void* vt = nullptr;
  int64_t ldv = 0, L = 1, m_off = 0;
  int nv = 0;  // N
};

// Persistent-kernel epilogue that writes the output transposed per batch
// (V^T for attention); internal to the library (linear_vt), not an ABI
// epilogue code.
constexpr int EPI_BIAS_VT = 16;

// ------------------------------------------------------------------ epilogues
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

// Epilogue of an MFMA tile: lane holds token m_base + 32 ti and features
// n_base + 32 fi + 8 g + {0..3}.  The lane's bias values are loaded (packed
// bf16) before any store, and the output pointer is declared unaliased, so
// the loads are not serialised behind the stores.
template <int EPI, int FI, int TI>
__device__ __forceinline__ void epilogue(const EpiArgs& e, const f32x16 (&acc)[FI][TI], int64_t M, int64_t m_base,
                                         int n_base) {
  const bf16_t* __restrict__ bias_p = (const bf16_t*)e.bias;
  const float* __restrict__ gate_p = e.gate;
#pragma unroll
  for (int fi = 0; fi < FI; ++fi) {
    u32x2 bias[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) bias[g] = *(const u32x2*)(bias_p + n_base + fi * 32 + 8 * g);
#pragma unroll
    for (int ti = 0; ti < TI; ++ti) {
      const int64_t m = m_base + ti * 32;
      if (m >= M) continue;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n_base + fi * 32 + 8 * g;
        const u32x2 bv = bias[g];
        float v[4];
        v[0] = acc[fi][ti][4 * g + 0] + __uint_as_float(bv[0] << 16);
        v[1] = acc[fi][ti][4 * g + 1] + __uint_as_float(bv[0] & 0xffff0000u);
        v[2] = acc[fi][ti][4 * g + 2] + __uint_as_float(bv[1] << 16);
        v[3] = acc[fi][ti][4 * g + 3] + __uint_as_float(bv[1] & 0xffff0000u);
        if constexpr (EPI == TRACK_EPI_BIAS || EPI == TRACK_EPI_BIAS_GELU) {
          if constexpr (EPI == TRACK_EPI_BIAS_GELU) {
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = gelu_tanh(v[j]);
          }
          u32x2 pk;
          pk[0] = pack_bf2(v[0], v[1]);
          pk[1] = pack_bf2(v[2], v[3]);
          bf16_t* __restrict__ o = (bf16_t*)e.out + m * e.ldo + n;
          *(u32x2*)o = pk;
        } else if constexpr (EPI == TRACK_EPI_GATE_RESID || EPI == TRACK_EPI_RESID) {
          float* __restrict__ o = (float*)e.out + m * e.ldo + n;
          f32x4 x = *(f32x4*)o;
          if constexpr (EPI == TRACK_EPI_GATE_RESID) {
            const f32x4 gt = *(const f32x4*)(gate_p + n);
#pragma unroll
            for (int j = 0; j < 4; ++j) x[j] = fmaf(gt[j], v[j], x[j]);
          } else {
#pragma unroll
            for (int j = 0; j < 4; ++j) x[j] += v[j];
          }
          *(f32x4*)o = x;
        } else {
          float* __restrict__ o = (float*)e.out + m * e.ldo + n;
          *(f32x4*)o = f32x4{v[0], v[1], v[2], v[3]};
        }
      }
    }
  }
}

// ------------------------------------------------------------------ bf16 MFMA kernel
// 16-byte chunk swizzle of a 128-byte LDS row: 8 consecutive rows get
// distinct chunks, and rows r and r + 8 differ as well, so 32-row fragment
// reads are conflict free whether LDS serves 8 or 16 lanes per cycle.
__device__ __forceinline__ int lds_swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// Block tile BM tokens x BN features x 64 (K); four waves in a 2 x 2 grid,
// each owning (BM/2) x (BN/2) as 32 x 32 MFMA blocks.  Tiles are staged
// through LDS, double buffered, rows of 64 bf16 (128 B) with the 16-byte
// chunk index XOR-swizzled (lds_swz) so that the 32-row fragment reads are
// bank-conflict free.  Global loads of the next K-slab are issued before
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
      *(u32x4*)(base + row * 128 + ((c ^ lds_swz(row)) << 4)) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < WC; ++i) {
      const int row = r0 + 32 * i;
      *(u32x4*)(base + (BM + row) * 128 + ((c ^ lds_swz(row)) << 4)) = rw[i];
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
        fw[fi] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + (BM + row) * 128 + ((ch ^ lds_swz(row)) << 4)));
      }
#pragma unroll
      for (int ti = 0; ti < TI; ++ti) {
        const int row = wm * WM + ti * 32 + frow;
        fa[ti] = __builtin_bit_cast(bf16x8, *(const u32x4*)(base + row * 128 + ((ch ^ lds_swz(row)) << 4)));
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
  epilogue<EPI, FI, TI>(e, acc, M, m0 + wm * WM + frow, n0 + wn * WN + 4 * fhalf);
}

// ------------------------------------------------------------------ persistent bf16 MFMA kernel
// One workgroup per CU loops over the 256 x 256 output tiles p, p + G, p + 2G,
// ... (p the XCD-remapped block index, G the grid), so the copy pipeline runs
// on from one tile into the next and a tile's epilogue overlaps the loads of
// the next tile's first slab.
//
// K-slabs of 64 (128-byte rows) travel global -> LDS through a 2-slot ring
// with buffer_load ... lds (16 bytes per lane, lane-contiguous in LDS); a
// buffer resource per tile makes rows past M read as zero.  A slab's barrier
// sits before its last 16-deep step: by then every wave holds that step's
// fragments and the next slab has landed, so the last step's MFMAs run while
// the next slab's first fragments are read, and the slot just released is
// refilled.  The 16 loads a wave issues for slab g + 1 go out one per two
// MFMAs during the last step of slab g - 1 and the first step of slab g, in
// program order (sched_barrier), so the load unit never holds a wave's MFMA
// stream for long and each slab has two steps to land; the fragments of the
// next step are read one per MFMA the same way.  LDS rows carry a 32-byte-granular XOR
// swizzle applied on the global side: lane pairs keep contiguous 32-byte
// pieces of a row, which the load path coalesces better than a 16-byte
// permutation, at the cost of 2-way bank conflicts on fragment reads.
__device__ __forceinline__ int lds_swz32(int row) { return ((row & 7) ^ ((row >> 3) & 1)) & ~1; }

typedef __attribute__((address_space(3))) void* lds_ptr_t;

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  // s_waitcnt with vmcnt = N (gfx9 encoding: low 4 bits and bits 15:14),
  // expcnt and lgkmcnt left at their maxima (no wait)
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt((15 << 0) | (3 << 14) | (7 << 4) | (0 << 8)); }

// Epilogue of a tile with bfloat16 output (bias, bias + GELU).  Every bias
// value is loaded before the first store (a load issued after a store would
// wait for it), and lanes l and l + 32, which hold features +0..3 and +4..7
// of the same token, trade halves with permlane32_swap so that each lane
// stores 16 contiguous bytes.
template <int EPI, int FI, int TI>
__device__ __forceinline__ void epilogue_bf16(const EpiArgs& e, const f32x16 (&acc)[FI][TI], int64_t M,
                                              int64_t m_base, int n_base, int fhalf) {
  const bf16_t* __restrict__ bias_p = (const bf16_t*)e.bias;
  u32x2 bias[FI][4];
#pragma unroll
  for (int fi = 0; fi < FI; ++fi)
#pragma unroll
    for (int g = 0; g < 4; ++g) bias[fi][g] = *(const u32x2*)(bias_p + n_base + fi * 32 + 8 * g);
  // Token blocks outermost: the two 32-feature blocks that share a token
  // row's 128-byte line are stored back to back, so the L2 holds whole lines
  // when it writes them back (feature blocks outermost left lines half
  // written long enough to be evicted and written twice: 20% more HBM writes).
#pragma unroll
  for (int ti = 0; ti < TI; ++ti) {
#pragma unroll
    for (int fi = 0; fi < FI; ++fi) {
      const int64_t m = m_base + ti * 32;
      u32x2 pk[4];
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2 bv = bias[fi][g];
        float v[4];
        v[0] = acc[fi][ti][4 * g + 0] + __uint_as_float(bv[0] << 16);
        v[1] = acc[fi][ti][4 * g + 1] + __uint_as_float(bv[0] & 0xffff0000u);
        v[2] = acc[fi][ti][4 * g + 2] + __uint_as_float(bv[1] << 16);
        v[3] = acc[fi][ti][4 * g + 3] + __uint_as_float(bv[1] & 0xffff0000u);
        if constexpr (EPI == TRACK_EPI_BIAS_GELU) {
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = gelu_tanh(v[j]);
        }
        pk[g][0] = pack_bf2(v[0], v[1]);
        pk[g][1] = pack_bf2(v[2], v[3]);
      }
      bf16_t* __restrict__ orow = (bf16_t*)e.out + m * e.ldo + n_base - 4 * fhalf + fi * 32;
#pragma unroll
      for (int gp = 0; gp < 2; ++gp) {
        // lanes < 32 keep group 2gp (own +0..3, partner's +4..7), lanes >= 32
        // group 2gp + 1 (partner's +0..3, own +4..7)
        const auto s0 = __builtin_amdgcn_permlane32_swap(pk[2 * gp][0], pk[2 * gp + 1][0], false, false);
        const auto s1 = __builtin_amdgcn_permlane32_swap(pk[2 * gp][1], pk[2 * gp + 1][1], false, false);
        const u32x4 q = {s0[0], s1[0], s0[1], s1[1]};
        if (m < M) *(u32x4*)(orow + 8 * (2 * gp + fhalf)) = q;
      }
    }
  }
}

// Epilogue of a tile with float32 output (gated residual, residual, plain).
// The bias, gate and residual values of feature block fi + 1 are loaded
// before the stores of block fi are issued, so no load waits behind a store
// of the same tile.
template <int EPI, int FI, int TI>
__device__ __forceinline__ void epilogue_f32(const EpiArgs& e, const f32x16 (&acc)[FI][TI], int64_t M,
                                             int64_t m_base, int n_base) {
  constexpr bool RES = EPI == TRACK_EPI_GATE_RESID || EPI == TRACK_EPI_RESID;
  constexpr bool GATE = EPI == TRACK_EPI_GATE_RESID;
  const bf16_t* __restrict__ bias_p = (const bf16_t*)e.bias;
  float* __restrict__ out = (float*)e.out;
  struct Block {
    u32x2 bias[4];
    f32x4 gate[4];
    f32x4 x[TI][4];
  };
  auto load = [&](int fi, Block& bl) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      bl.bias[g] = *(const u32x2*)(bias_p + n_base + fi * 32 + 8 * g);
      if constexpr (GATE) bl.gate[g] = *(const f32x4*)(e.gate + n_base + fi * 32 + 8 * g);
    }
    if constexpr (RES) {
#pragma unroll
      for (int ti = 0; ti < TI; ++ti) {
        const int64_t m = m_base + ti * 32;
#pragma unroll
        for (int g = 0; g < 4; ++g)
          bl.x[ti][g] = m < M ? *(const f32x4*)(out + m * e.ldo + n_base + fi * 32 + 8 * g) : f32x4{0, 0, 0, 0};
      }
    }
  };
  Block bl[2];
  load(0, bl[0]);
#pragma unroll
  for (int fi = 0; fi < FI; ++fi) {
    if (fi + 1 < FI) load(fi + 1, bl[(fi + 1) & 1]);
    __builtin_amdgcn_sched_barrier(0);  // keep those loads ahead of this block's stores
    const Block& c = bl[fi & 1];
#pragma unroll
    for (int ti = 0; ti < TI; ++ti) {
      const int64_t m = m_base + ti * 32;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2 bv = c.bias[g];
        f32x4 v;
        v[0] = acc[fi][ti][4 * g + 0] + __uint_as_float(bv[0] << 16);
        v[1] = acc[fi][ti][4 * g + 1] + __uint_as_float(bv[0] & 0xffff0000u);
        v[2] = acc[fi][ti][4 * g + 2] + __uint_as_float(bv[1] << 16);
        v[3] = acc[fi][ti][4 * g + 3] + __uint_as_float(bv[1] & 0xffff0000u);
        if constexpr (GATE) {
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = fmaf(c.gate[g][j], v[j], c.x[ti][g][j]);
        } else if constexpr (RES) {
#pragma unroll
          for (int j = 0; j < 4; ++j) v[j] = c.x[ti][g][j] + v[j];
        }
        if (m < M) *(f32x4*)(out + m * e.ldo + n_base + fi * 32 + 8 * g) = v;
      }
    }
  }
}

// Epilogue of the transposed-output GEMM: out^T per batch.
// Each wave stages one 32-feature block of its 128 x 128 sub-tile at a time
// ([feature][128 tokens] bf16, 8 KB of LDS beside the copy ring), then reads
// back rows of 8 consecutive tokens and stores them as 16-byte vectors.
// Requires L % 8 == 0, so that 8 tokens starting at a multiple of 8 share a
// batch, L >= 128 and ldv % 8 == 0.
template <int FI, int TI>
__device__ __forceinline__ void epilogue_vt(const EpiArgs& e, const f32x16 (&acc)[FI][TI], int64_t M, int64_t tok0,
                                            int feat0, int jq, int fhalf, uint8_t* stage) {
  // lane-derived offsets are recomputed here rather than hoisted out of the
  // tile loop (kept live across the main loop they would spill)
  int lane = jq + 32 * fhalf;
  asm volatile("" : "+v"(lane));
  jq = lane & 31;
  fhalf = lane >> 5;
  const bf16_t* __restrict__ bias_p = (const bf16_t*)e.bias + feat0 + 4 * fhalf;
  // batch and position of the wave's first token; its 128 tokens cross at
  // most one batch boundary (L >= 128)
  const int64_t mg0 = e.m_off + tok0;
  const int64_t b0 = mg0 / e.L;
  const int64_t l0 = mg0 - b0 * e.L;
  bf16_t* __restrict__ vt = (bf16_t*)e.vt;
  u32x2 bias[2][4];
#pragma unroll
  for (int g = 0; g < 4; ++g) bias[0][g] = *(const u32x2*)(bias_p + 8 * g);
#pragma unroll
  for (int fi = 0; fi < FI; ++fi) {
    // the next block's bias is loaded before this block's stores
    if (fi + 1 < FI) {
#pragma unroll
      for (int g = 0; g < 4; ++g) bias[(fi + 1) & 1][g] = *(const u32x2*)(bias_p + (fi + 1) * 32 + 8 * g);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int ti = 0; ti < TI; ++ti)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const u32x2 bv = bias[fi & 1][g];
#pragma unroll
        for (int j = 0; j < 4; j += 2) {
          const float b_lo = __uint_as_float(bv[j / 2] << 16), b_hi = __uint_as_float(bv[j / 2] & 0xffff0000u);
          const uint32_t h = pack_bf2(acc[fi][ti][4 * g + j] + b_lo, acc[fi][ti][4 * g + j + 1] + b_hi);
          uint8_t* p = stage + (8 * g + 4 * fhalf + j) * 256 + (ti * 32 + jq) * 2;
          *(uint16_t*)p = (uint16_t)(h & 0xffffu);
          *(uint16_t*)(p + 256) = (uint16_t)(h >> 16);
        }
      }
    // 32 rows x 16 chunks of 8 tokens; LDS operations of a wave complete in order
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int id = i * 64 + lane;
      const int row = id >> 4, ch = id & 15;
      const u32x4 v = *(const u32x4*)(stage + row * 256 + ch * 16);
      if (tok0 + ch * 8 < M) {
        int64_t l = l0 + ch * 8, b = b0;
        if (l >= e.L) {
          l -= e.L;
          ++b;
        }
        const int n = feat0 + fi * 32 + row;
        *(u32x4*)(vt + (b * e.nv + n) * e.ldv + l) = v;
      }
    }
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void gemm_bf16_persist_kernel(const bf16_t* __restrict__ A, int64_t lda,
                                                                const bf16_t* __restrict__ W, int64_t M, int N,
                                                                int K, EpiArgs e, int ntiles, int GB) {
  constexpr int BM = 256, BN = 256, BK = 64, NWV = 4;
  constexpr int WM = 128, WN = 128, TI = 4, FI = 4;
  constexpr int ROWB = BK * 2, CPR = ROWB / 16;      // 128-byte LDS rows, 8 chunks
  constexpr int STAGE_BYTES = (BM + BN) * ROWB;       // 64 KB per slot
  constexpr int LOADS = (BM + BN) * ROWB / (NWV * 64 * 16);  // 16 per wave per slab
  constexpr int ROWS_PER_LOAD = 1024 / ROWB;          // 8 rows per wave-wide load
  constexpr int ALOADS = BM / ROWS_PER_LOAD / NWV;    // 8 of them cover A
  constexpr int KS = BK / 16;                         // 16-deep MFMA steps per slab
  constexpr int DPM = 2;                              // MFMAs per DMA load
  static_assert(LOADS * DPM <= KS * 16, "the loads fit in the slab");
  // the copy ring, then (transposed epilogue only) 8 KB of staging per wave
  __shared__ __attribute__((aligned(1024))) uint8_t smem[2 * STAGE_BYTES + (EPI == EPI_BIAS_VT ? NWV * 8192 : 0)];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int num_tm = (int)((M + BM - 1) / BM), num_tn = N / BN;
  const int G = gridDim.x;
  const int p = xcd_remap(blockIdx.x, G);
  // tile order: bands of GB M-tiles swept across N
  auto tile_mn = [&](int T, int64_t& m0, int& n0) {
    const int band = T / (GB * num_tn);
    const int first_tm = band * GB;
    const int gsz = min(num_tm - first_tm, GB);
    const int in_band = T - band * GB * num_tn;
    m0 = (int64_t)(first_tm + in_band % gsz) * BM;
    n0 = (in_band / gsz) * BN;
  };

  // Load i of a wave covers rows rb(i) .. rb(i) + 7 of the A tile (i < ALOADS)
  // or of the W tile: lane -> row rb(i) + lane / 8, fetching the global
  // chunk that the swizzle puts at LDS chunk lane % 8.  rb(i) is a multiple
  // of 8 whose bit 3 is the wave's, so the swizzle is the same for every load.
  const int lrow = lane / CPR;
  const int lcol = ((lane % CPR) ^ lds_swz32(wave * ROWS_PER_LOAD + lrow)) * 8;
  const uint32_t voffA = (uint32_t)((lrow * lda + lcol) * 2);
  const uint32_t voffW = (uint32_t)((lrow * (int64_t)K + lcol) * 2);
  auto rb = [&](int i) { return (i < ALOADS ? i : i - ALOADS) * NWV * ROWS_PER_LOAD + wave * ROWS_PER_LOAD; };
  __amdgpu_buffer_rsrc_t rsA, rsW;
  auto set_src = [&](int T) {
    int64_t m0;
    int n0;
    tile_mn(T, m0, n0);
    // the host keeps (M - m0) * lda * 2 below 2^31
    rsA = __builtin_amdgcn_make_buffer_rsrc((void*)(A + m0 * lda), (short)0, (int)((M - m0) * lda * 2), 0x00020000);
    rsW = __builtin_amdgcn_make_buffer_rsrc((void*)(W + (int64_t)n0 * K), (short)0, (int)((int64_t)BN * K * 2), 0x00020000);
  };
  const int KT = K / BK;
  int ld_T = p, ld_kt = 0, ld_slot = 0;
  set_src(p);
  // The A row of a load is part of its vector offset and only the slab's
  // column offset (less than a row) is scalar, so a row past M lies beyond
  // the resource's size whatever the scalar part, and an in-range row's
  // address stays inside that row.
  auto issue_one = [&](int i) {
    lds_ptr_t d = (lds_ptr_t)(smem + ld_slot * STAGE_BYTES + (i < ALOADS ? 0 : BM * ROWB) + rb(i) * ROWB);
    if (i < ALOADS)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsA, d, 16, voffA + (uint32_t)(rb(i) * lda * 2), ld_kt * BK * 2, 0, 0);
    else
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsW, d, 16, voffW, (int)((rb(i) * (int64_t)K + ld_kt * BK) * 2), 0, 0);
  };
  // After the last slab of the last tile the loads keep re-fetching that tile
  // (in bounds, into a slot nobody reads again).
  auto advance_ld = [&]() {
    ld_slot ^= 1;
    if (++ld_kt == KT) {
      ld_kt = 0;
      if (ld_T + G < ntiles) {
        ld_T += G;
        set_src(ld_T);
      }
    }
  };
  f32x16 acc[FI][TI];
#pragma unroll
  for (int fi = 0; fi < FI; ++fi)
#pragma unroll
    for (int ti = 0; ti < TI; ++ti)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[fi][ti][r] = 0.0f;

  const int frow = lane & 31, fhalf = lane >> 5;
  // fragment idx of 16-deep step kk: 0..3 the W rows (MFMA A operand),
  // 4..7 the token rows (B operand)
  auto read_frag = [&](const uint8_t* base, int kk, int idx) -> bf16x8 {
    const int ch = kk * 2 + fhalf;
    const int row = idx < FI ? BM + wn * WN + idx * 32 + frow : wm * WM + (idx - FI) * 32 + frow;
    return __builtin_bit_cast(bf16x8, *(const u32x4*)(base + row * ROWB + ((ch ^ lds_swz32(row)) << 4)));
  };
  bf16x8 fw[2][FI], fa[2][TI];
  // MFMAs of 16-deep step kk (fragments in buffer kk & 1); with rd, before
  // MFMA j < 8 fragment j of step nk of the slab at nbase is read into the
  // other buffer; with lo >= 0, DMA loads lo .. lo + 7 follow every second
  // MFMA.
  auto step = [&](int kk, const uint8_t* nbase, int nk, int lo, bool rd) {
    const bf16x8* w_ = fw[kk & 1];
    const bf16x8* a_ = fa[kk & 1];
    bf16x8* nw = fw[(kk + 1) & 1];
    bf16x8* na = fa[(kk + 1) & 1];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      if (rd && j < FI + TI) {
        if (j < FI) nw[j] = read_frag(nbase, nk, j);
        else na[j - FI] = read_frag(nbase, nk, j);
      }
      acc[j / TI][j % TI] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(w_[j / TI], a_[j % TI], acc[j / TI][j % TI], 0, 0, 0);
      if (lo >= 0 && j % DPM == 0) issue_one(lo + j / DPM);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  static_assert(KS == 4 && LOADS == 16 && DPM == 2, "the slab schedule below assumes 4 steps and 16 loads");

  // prologue: slab 0, then the first half of slab 1's loads and slab 0's
  // first fragments
#pragma unroll
  for (int i = 0; i < LOADS; ++i) issue_one(i);
  advance_ld();
  wait_vmcnt<0>();
  __builtin_amdgcn_s_barrier();
#pragma unroll
  for (int i = 0; i < LOADS / 2; ++i) issue_one(i);
#pragma unroll
  for (int f = 0; f < FI + TI; ++f) {
    if (f < FI) fw[0][f] = read_frag(smem, 0, f);
    else fa[0][f - FI] = read_frag(smem, 0, f);
  }

  const int my_tiles = (ntiles - p + G - 1) / G;
  int slot = 0;
  // slab body; rd: read the next slab's first fragments during the last
  // step (not at a tile's last slab, where they would stay live through the
  // epilogue and push it into spilling)
  auto slab = [&](bool rd) {
    const uint8_t* base = smem + slot * STAGE_BYTES;
    const uint8_t* nbase = smem + (slot ^ 1) * STAGE_BYTES;
    step(0, base, 1, LOADS / 2, true);  // second half of slab g + 1's loads
    advance_ld();
    step(1, base, 2, -1, true);
    step(2, base, 3, -1, true);
    // slab g + 1 has landed for this wave (and, at a tile's first slab, the
    // previous epilogue's stores are complete); after the barrier for every
    // wave, and every wave holds its step-3 fragments of slab g
    wait_vmcnt<0>();
    wait_lgkm0();
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    step(3, nbase, 0, 0, rd);  // first half of slab g + 2's loads, into slab g's slot
    slot ^= 1;
  };
  for (int t = 0; t < my_tiles; ++t) {
    for (int kt = 0; kt + 1 < KT; ++kt) slab(true);
    slab(false);
    int64_t cm0;
    int cn0;
    tile_mn(p + t * G, cm0, cn0);
    if constexpr (EPI == EPI_BIAS_VT) {
      epilogue_vt<FI, TI>(e, acc, M, cm0 + wm * WM, cn0 + wn * WN, frow, fhalf, smem + 2 * STAGE_BYTES + wave * 8192);
    } else if constexpr (EPI == TRACK_EPI_BIAS || EPI == TRACK_EPI_BIAS_GELU)
      epilogue_bf16<EPI, FI, TI>(e, acc, M, cm0 + wm * WM + frow, cn0 + wn * WN + 4 * fhalf, fhalf);
    else
      epilogue_f32<EPI, FI, TI>(e, acc, M, cm0 + wm * WM + frow, cn0 + wn * WN + 4 * fhalf);
#pragma unroll
    for (int fi = 0; fi < FI; ++fi)
#pragma unroll
      for (int ti = 0; ti < TI; ++ti)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[fi][ti][r] = 0.0f;
    // the next tile's first fragments (its first slab landed before the
    // last barrier)
    const uint8_t* nb = smem + slot * STAGE_BYTES;
#pragma unroll
    for (int f = 0; f < FI + TI; ++f) {
      if (f < FI) fw[0][f] = read_frag(nb, 0, f);
      else fa[0][f - FI] = read_frag(nb, 0, f);
    }
  }
  // the last copies must land before the workgroup's LDS is released
  wait_vmcnt<0>();
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

// Kernel override for tuning and test runs (TRACK_GEMM_CFG, read at every
// call): 0 automatic, 1 256x256, 2 128x128, 3 256x128 (register-staged
// kernel), 4 the persistent kernel for every shape it supports (N % 256 == 0)
// whatever the tile count; shapes the forced kernel does not take use the
// automatic choice.
static int gemm_config() {
  const char* v = getenv("TRACK_GEMM_CFG");
  const int c = v ? atoi(v) : 0;
  return (c >= 0 && c <= 4) ? c : 0;
}

// Compute units of the current device (the persistent grid size).
int device_cus() {
  static int cus[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cus[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev] = n;
  }
  return cus[dev];
}

// The persistent kernel addresses A through a buffer resource whose size
// field is 32 bits; M is cut into row blocks of at most 2^31 - 1 bytes of A.
static void launch_bf16_persist(int epi, const bf16_t* A, int64_t lda, const bf16_t* W, int64_t M, int N, int K,
                                const EpiArgs& e, int out_elem, hipStream_t s) {
  const int64_t max_rows = ((((int64_t)1 << 31) - 1) / (lda * 2)) / 256 * 256;
  const int cus = device_cus();
  // Height of the bands of M-tiles swept across N (the order in which the
  // CUs take tiles, so what the L2 caches share): measured over the Wan
  // projection shapes, 4 suits long K (5120 and up), 16 wide N at short K,
  // 8 the rest; the order changes no result.
  const int gb = K >= 4096 ? 4 : (N >= 8192 ? 16 : 8);
  for (int64_t r0 = 0; r0 < M; r0 += max_rows) {
    const int64_t rows = M - r0 < max_rows ? M - r0 : max_rows;
    EpiArgs ec = e;
    ec.out = (uint8_t*)e.out + r0 * e.ldo * out_elem;
    ec.m_off = e.m_off + r0;
    const bf16_t* a = A + r0 * lda;
    const int ntiles = (int)((rows + 255) / 256) * (N / 256);
    dim3 grid(ntiles < cus ? ntiles : cus), block(256);
#define TRACK_PK(E) gemm_bf16_persist_kernel<E><<<grid, block, 0, s>>>(a, lda, W, rows, N, K, ec, ntiles, gb)
    switch (epi) {
      case TRACK_EPI_BIAS: TRACK_PK(TRACK_EPI_BIAS); break;
      case TRACK_EPI_BIAS_GELU: TRACK_PK(TRACK_EPI_BIAS_GELU); break;
      case TRACK_EPI_GATE_RESID: TRACK_PK(TRACK_EPI_GATE_RESID); break;
      case TRACK_EPI_RESID: TRACK_PK(TRACK_EPI_RESID); break;
      case EPI_BIAS_VT: TRACK_PK(EPI_BIAS_VT); break;
      default: TRACK_PK(TRACK_EPI_BIAS_F32); break;
    }
#undef TRACK_PK
  }
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
  const int out_elem = (epi == TRACK_EPI_BIAS || epi == TRACK_EPI_BIAS_GELU) ? 2 : 4;
  if (force == 1 && N % 256 == 0)
    launch_bf16_cfg<256, 256>(epi, a, lda, w, M, n, k, e, s);
  else if (force == 2 && N % 128 == 0)
    launch_bf16_cfg<128, 128>(epi, a, lda, w, M, n, k, e, s);
  else if (force == 3 && N % 128 == 0)
    launch_bf16_cfg<256, 128>(epi, a, lda, w, M, n, k, e, s);
  // the persistent kernel for at least two tiles per CU, or, with a long K
  // (the 14B-width text K/V projection: 160 tiles, K 5120, 0.11 against
  // 0.17 ms), at least half a tile per CU
  else if (N % 256 == 0 && (big >= 512 || (big >= 128 && K >= 4096) || force == 4) && lda < ((int64_t)1 << 22))
    launch_bf16_persist(epi, a, lda, w, M, n, k, e, out_elem, s);
  else if (N % 128 == 0)
    launch_bf16_cfg<128, 128>(epi, a, lda, w, M, n, k, e, s);
  else
    launch_bf16_cfg<128, 64>(epi, a, lda, w, M, n, k, e, s);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

track_status linear_vt(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda, const void* W, const void* bias,
                       int64_t L, void* vt, int64_t ldv, hipStream_t s) {
  if (M <= 0 || N <= 0 || K <= 0 || L <= 0) return fail(TRACK_E_SHAPE, "linear_vt: empty shape");
  if (!A || !W || !bias || !vt) return fail(TRACK_E_INVALID, "linear_vt: null pointer");
  if (lda < K || ldv < L) return fail(TRACK_E_SHAPE, "linear_vt: leading dimension too small");
  if (N % 256 || K % 64 || L % 8 || L < 128 || M % L || ldv % 8 || lda % 8 || lda >= ((int64_t)1 << 22) ||
      N > (1 << 30) || K > (1 << 30))
    return fail(TRACK_E_UNSUPPORTED, "linear_vt: needs N %% 256 == 0, K %% 64 == 0, L, ldv, lda %% 8 == 0, L >= 128, "
                "M %% L == 0 (N=%lld K=%lld L=%lld M=%lld)", (long long)N, (long long)K, (long long)L, (long long)M);
  if (((uintptr_t)A & 15) || ((uintptr_t)W & 15) || ((uintptr_t)vt & 15) || ((uintptr_t)bias & 7))
    return fail(TRACK_E_INVALID, "linear_vt: needs 16-byte aligned buffers");
  EpiArgs e{bias, nullptr, nullptr, 0};
  e.vt = vt;
  e.ldv = ldv;
  e.L = L;
  e.m_off = 0;
  e.nv = (int)N;
  ProfScope prof(TRACK_PROF_GEMM, s);
  launch_bf16_persist(EPI_BIAS_VT, (const bf16_t*)A, lda, (const bf16_t*)W, M, (int)N, (int)K, e, 2, s);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}


// ------------------------------------------------------------------ matrix-core stream
// The sustained matrix-core rate, the ceiling the MFMA-bound kernels are
// measured against besides the published peak: one 4-wave workgroup per CU,
// each wave issuing 8 independent v_mfma_f32_32x32x16_bf16 chains per loop
// iteration from operands it loaded once (four A and two B fragments, caller
// data).  The chip's clock under matrix work depends on how many operand bits
// toggle, so the caller picks data like that of the kernel it compares.
constexpr int MFMA_STREAM_CHAINS = 8;
constexpr int64_t MFMA_STREAM_VECS = 4096;  // 16-byte operand vectors read

__global__ __launch_bounds__(256) void mfma_stream_kernel(const bf16x8* __restrict__ ops, float* __restrict__ sink,
                                                          int iters) {
  const int g = blockIdx.x * 256 + threadIdx.x;
  bf16x8 a[4], b[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) a[i] = ops[(g * 3 + i * 131) & (MFMA_STREAM_VECS - 1)];
#pragma unroll
  for (int i = 0; i < 2; ++i) b[i] = ops[(g * 5 + i * 977 + 7) & (MFMA_STREAM_VECS - 1)];
  f32x16 c[MFMA_STREAM_CHAINS];
#pragma unroll
  for (int j = 0; j < MFMA_STREAM_CHAINS; ++j) c[j] = f32x16{};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < MFMA_STREAM_CHAINS; ++j)
      c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[j & 3], b[(j >> 2) ^ (j & 1)], c[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < MFMA_STREAM_CHAINS; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += c[j][e];
  // reaches memory only for a value a caller would have to plant, so the
  // chains cannot be dropped
  if (s == 0x1.5p-99f) sink[0] = s;
}

track_status mfma_stream(const void* operands, int64_t iters, float* sink, int64_t* flop, hipStream_t s) {
  if (!operands || !sink || !flop) return fail(TRACK_E_INVALID, "mfma_stream: null pointer");
  if (iters <= 0 || iters > INT32_MAX) return fail(TRACK_E_SHAPE, "mfma_stream: iters must be in [1, 2^31)");
  if ((uintptr_t)operands & 15) return fail(TRACK_E_INVALID, "mfma_stream: 16-byte alignment needed");
  const int cus = device_cus();
  *flop = (int64_t)cus * 4 * iters * MFMA_STREAM_CHAINS * (2 * 32 * 32 * 16);
  ProfScope prof(TRACK_PROF_OTHER, s);
  mfma_stream_kernel<<<cus, 256, 0, s>>>((const bf16x8*)operands, sink, (int)iters);
  TRACK_LAUNCH_CHECK();
  return TRACK_OK;
}

}  // namespace track
