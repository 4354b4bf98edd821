// Weight table, workspace layout and the denoiser forward pass.
//
// The forward is the Wan-2.1-style video DiT: patch embedding, sinusoidal
// timestep MLP with a shared adaLN modulation plus per-block offsets, text
// MLP, and per block a modulated self-attention sub-block with RMS-normed,
// 3D-rotary q/k, a text cross-attention sub-block and a modulated GELU MLP,
// followed by a modulated output head.  Every step is one of this library's
// kernels, launched in order on a single stream.
#include "model.h"

#include <deque>
#include <map>
#include <mutex>

namespace track {

// Tensor order of the weight buffer (see track.h).
enum GlobalTensor { T_PATCH_W, T_PATCH_B, T_TIME_W1, T_TIME_B1, T_TIME_W2, T_TIME_B2, T_MOD_W, T_MOD_B,
                    T_TEXT_W1, T_TEXT_B1, T_TEXT_W2, T_TEXT_B2, T_NGLOBAL };
enum BlockTensor { B_MOD, B_QKV_W, B_QKV_B, B_NORM_Q, B_NORM_K, B_O_W, B_O_B, B_CQ_W, B_CQ_B, B_CKV_W, B_CKV_B,
                   B_NORM_CQ, B_NORM_CK, B_CO_W, B_CO_B, B_FFN1_W, B_FFN1_B, B_FFN2_W, B_FFN2_B, B_NBLOCK };
enum HeadTensor { H_MOD, H_W, H_B, H_NHEAD };

static const char* kGlobalNames[T_NGLOBAL] = {"patch.w", "patch.b", "time.w1", "time.b1", "time.w2", "time.b2",
                                              "mod.w",   "mod.b",   "text.w1", "text.b1", "text.w2", "text.b2"};
static const char* kBlockNames[B_NBLOCK] = {"mod",    "qkv.w",   "qkv.b",   "norm_q", "norm_k", "o.w",    "o.b",
                                            "cq.w",   "cq.b",    "ckv.w",   "ckv.b",  "norm_cq", "norm_ck", "co.w",
                                            "co.b",   "ffn1.w",  "ffn1.b",  "ffn2.w", "ffn2.b"};
static const char* kHeadNames[H_NHEAD] = {"head.mod", "head.w", "head.b"};

track_status check_config(const track_dit_config& c) {
  if (c.blocks < 0 || c.dim <= 0 || c.heads <= 0 || c.head_dim <= 0 || c.ffn_dim <= 0 || c.in_ch <= 0 ||
      c.patch_t <= 0 || c.patch_h <= 0 || c.patch_w <= 0 || c.text_dim <= 0 || c.freq_dim <= 0)
    return fail(TRACK_E_INVALID, "config: sizes must be positive");
  if (c.dtype != TRACK_DTYPE_F32 && c.dtype != TRACK_DTYPE_BF16) return fail(TRACK_E_INVALID, "config: bad dtype %d", c.dtype);
  if (c.heads * c.head_dim != c.dim) return fail(TRACK_E_INVALID, "config: dim != heads * head_dim");
  if (c.head_dim % 4 || c.freq_dim % 8) return fail(TRACK_E_INVALID, "config: head_dim %% 4 and freq_dim %% 8 must be 0");
  const int P = c.in_ch * c.patch_t * c.patch_h * c.patch_w;
  if (P % 4 || c.dim > 8192) return fail(TRACK_E_UNSUPPORTED, "config: patch elements %% 4 != 0 or dim > 8192");
  if (c.dtype == TRACK_DTYPE_BF16) {
    if (c.head_dim != 128) return fail(TRACK_E_UNSUPPORTED, "config: bf16 path needs head_dim 128");
    if (c.dim % 64 || c.ffn_dim % 64 || c.text_dim % 64 || P % 64)
      return fail(TRACK_E_UNSUPPORTED, "config: bf16 path needs dim, ffn_dim, text_dim and patch elements to be multiples of 64");
  } else {
    if (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 128)
      return fail(TRACK_E_UNSUPPORTED, "config: float32 path supports head_dim 32, 64, 128");
  }
  return TRACK_OK;
}

const std::vector<std::string>& tensor_names(int blocks) {
  static std::mutex mu;
  static std::map<int, std::vector<std::string>> tables;
  std::lock_guard<std::mutex> lock(mu);
  auto it = tables.find(blocks);
  if (it != tables.end()) return it->second;
  std::vector<std::string> v;
  for (int i = 0; i < T_NGLOBAL; ++i) v.push_back(kGlobalNames[i]);
  for (int b = 0; b < blocks; ++b)
    for (int i = 0; i < B_NBLOCK; ++i) v.push_back("blk" + std::to_string(b) + "." + kBlockNames[i]);
  for (int i = 0; i < H_NHEAD; ++i) v.push_back(kHeadNames[i]);
  return tables.emplace(blocks, std::move(v)).first->second;
}

std::vector<TensorSpec> tensor_specs(const track_dit_config& c, size_t* total) {
  const int64_t d = c.dim, f = c.ffn_dim, P = (int64_t)c.in_ch * c.patch_t * c.patch_h * c.patch_w;
  const auto& names = tensor_names(c.blocks);
  std::vector<TensorSpec> s;
  auto add = [&](int64_t r, int64_t cols) {
    TensorSpec t;
    t.name = names[s.size()];
    t.ndim = cols > 0 ? 2 : 1;
    t.shape[0] = r;
    t.shape[1] = cols > 0 ? cols : 0;
    t.offset = 0;
    s.push_back(t);
  };
  add(d, P); add(d, 0); add(d, c.freq_dim); add(d, 0); add(d, d); add(d, 0); add(6 * d, d); add(6 * d, 0);
  add(d, c.text_dim); add(d, 0); add(d, d); add(d, 0);
  for (int b = 0; b < c.blocks; ++b) {
    add(6, d);
    add(3 * d, d); add(3 * d, 0); add(d, 0); add(d, 0);
    add(d, d); add(d, 0);
    add(d, d); add(d, 0); add(2 * d, d); add(2 * d, 0); add(d, 0); add(d, 0);
    add(d, d); add(d, 0);
    add(f, d); add(f, 0); add(d, f); add(d, 0);
  }
  add(2, d); add(P, d); add(P, 0);
  size_t off = 0;
  const size_t es = dtype_size(c.dtype);
  for (auto& t : s) {
    t.offset = off;
    const size_t n = (size_t)t.shape[0] * (t.ndim == 2 ? (size_t)t.shape[1] : 1);
    off = align256(off + n * es);
  }
  if (total) *total = off;
  return s;
}

static inline const void* wptr(const Model& m, int index) { return m.w + m.specs[index].offset; }
static inline const void* gW(const Model& m, GlobalTensor t) { return wptr(m, t); }
static inline const void* bW(const Model& m, int blk, BlockTensor t) { return wptr(m, T_NGLOBAL + blk * B_NBLOCK + t); }
static inline const void* hW(const Model& m, HeadTensor t) { return wptr(m, T_NGLOBAL + m.cfg.blocks * B_NBLOCK + t); }

track_status check_shape(const Model& m, const track_latent_shape& s) {
  const auto& c = m.cfg;
  if (s.channels != c.in_ch) return fail(TRACK_E_SHAPE, "latent channels %d != model in_ch %d", s.channels, c.in_ch);
  if (s.frames <= 0 || s.height <= 0 || s.width <= 0 || s.text_len <= 0) return fail(TRACK_E_SHAPE, "latent: sizes must be positive");
  if (s.frames % c.patch_t || s.height % c.patch_h || s.width % c.patch_w)
    return fail(TRACK_E_SHAPE, "latent %dx%dx%d not divisible by patch %dx%dx%d", s.frames, s.height, s.width, c.patch_t,
                c.patch_h, c.patch_w);
  return TRACK_OK;
}

WsLayout ws_layout(const Model& m, const track_latent_shape& s, int B) {
  const auto& c = m.cfg;
  WsLayout w{};
  const size_t es = dtype_size(c.dtype);
  w.grid = Grid3{s.frames / c.patch_t, s.height / c.patch_h, s.width / c.patch_w};
  w.L = (int64_t)w.grid.f * w.grid.h * w.grid.w;
  w.Lpad = round_up(w.L, 64);
  w.Lc = s.text_len;
  w.Lcpad = round_up(w.Lc, 64);
  w.P = (int64_t)c.in_ch * c.patch_t * c.patch_h * c.patch_w;
  const int64_t d = c.dim;
  const int ds = 2 * (c.head_dim / 6), df = c.head_dim - 2 * ds;
  w.rope_len = w.grid.f * (df / 2) + (w.grid.h + w.grid.w) * (ds / 2);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off = align256(off + bytes);
    return o;
  };
  w.sin = take(c.freq_dim * 4);
  w.h = take(d * 4);
  w.e = take(d * 4);
  w.se = take(d * 4);
  w.m = take(6 * d * 4);
  w.mods = take((size_t)c.blocks * 6 * d * 4);
  w.hmod = take(2 * d * 4);
  w.rope_cos = take((size_t)w.rope_len * 4);
  w.rope_sin = take((size_t)w.rope_len * 4);
  w.ctx = take((size_t)B * w.Lc * c.text_dim * es);
  w.th = take((size_t)B * w.Lc * d * es);
  w.temb = take((size_t)B * w.Lc * d * es);
  w.kvc = take((size_t)B * w.Lc * 2 * d * es);
  w.vct = take((size_t)B * c.heads * c.head_dim * w.Lcpad * es);
  w.tok = take((size_t)w.L * w.P * es);
  w.X = take((size_t)B * w.L * d * 4);
  w.Y = take((size_t)B * w.L * d * es);
  w.QKV = take((size_t)B * w.L * 3 * d * es);
  w.Vt = take((size_t)B * c.heads * c.head_dim * w.Lpad * es);
  w.AO = take((size_t)B * w.L * d * es);
  w.Hf = take((size_t)B * w.L * c.ffn_dim * es);
  w.vel = take((size_t)B * w.L * w.P * 4);
  w.xtok = take((size_t)w.L * w.P * 4);
  w.partial = take((size_t)step_partial_count(w.L * w.P) * 2 * 8);
  w.r = take((size_t)R_CAPACITY * 8);
  // band decomposition scratch (calibration only); none for latents the band
  // kernels do not support
  w.band = take(band_check(c.in_ch, s.frames, s.height, s.width, c.patch_t, c.patch_h, c.patch_w) == TRACK_OK
                    ? band_workspace_bytes(c.in_ch, s.frames, s.height, s.width, c.patch_t, c.patch_h, c.patch_w)
                    : 0);
  w.rband = take((size_t)R_CAPACITY * 6 * 8);
  // multistep scheduler state: the last corrected sample and a ring of four
  // data predictions
  w.sched = take((size_t)5 * w.L * w.P * 4);
  w.total = off;
  return w;
}

#define TRY(expr)                       \
  do {                                  \
    track_status st_ = (expr);          \
    if (st_ != TRACK_OK) return st_;    \
  } while (0)

track_status forward(const Model& m, const track_latent_shape& s, int B, const float* x_tok, double t,
                     const void* const* ctx, float* vel, hipStream_t st) {
  const auto& c = m.cfg;
  const int dt = c.dtype;
  const size_t es = dtype_size(dt);
  const WsLayout w = ws_layout(m, s, B);
  if (!m.ws || m.ws_bytes < w.total) return fail(TRACK_E_NOMEM, "workspace of %zu bytes needed, %zu attached", w.total, m.ws_bytes);
  const int64_t d = c.dim, L = w.L, Lc = w.Lc, P = w.P, H = c.heads, dh = c.head_dim;
  const int64_t rows = B * L;
  float* sinb = wsp<float>(m, w.sin);
  float* hb = wsp<float>(m, w.h);
  float* eb = wsp<float>(m, w.e);
  float* seb = wsp<float>(m, w.se);
  float* mb = wsp<float>(m, w.m);
  float* mods = wsp<float>(m, w.mods);
  float* hmod = wsp<float>(m, w.hmod);
  float* rcos = wsp<float>(m, w.rope_cos);
  float* rsin = wsp<float>(m, w.rope_sin);
  uint8_t* ctxb = wsp<uint8_t>(m, w.ctx);
  void* th = wsp<void>(m, w.th);
  void* temb = wsp<void>(m, w.temb);
  uint8_t* kvc = wsp<uint8_t>(m, w.kvc);
  void* vct = wsp<void>(m, w.vct);
  float* X = wsp<float>(m, w.X);
  void* Y = wsp<void>(m, w.Y);
  uint8_t* QKV = wsp<uint8_t>(m, w.QKV);
  void* Vt = wsp<void>(m, w.Vt);
  void* AO = wsp<void>(m, w.AO);
  void* Hf = wsp<void>(m, w.Hf);

  {
    ProfScope prof(TRACK_PROF_OTHER, st);
    // timestep features -> e, m = Wm silu(e) + bm, per-block modulation tables
    TRY(sinusoid(t, c.freq_dim, sinb, st));
    TRY(gemv(dt, (int)d, c.freq_dim, gW(m, T_TIME_W1), gW(m, T_TIME_B1), sinb, hb, nullptr, 1, st));
    TRY(gemv(dt, (int)d, (int)d, gW(m, T_TIME_W2), gW(m, T_TIME_B2), hb, eb, seb, 0, st));
    TRY(gemv(dt, (int)(6 * d), (int)d, gW(m, T_MOD_W), gW(m, T_MOD_B), seb, mb, nullptr, 0, st));
    const int64_t blk_stride = c.blocks > 1 ? (int64_t)(m.specs[T_NGLOBAL + B_NBLOCK].offset - m.specs[T_NGLOBAL].offset) / (int64_t)es : 0;
    if (c.blocks > 0) TRY(mod_tables(dt, c.blocks, (int)d, mb, bW(m, 0, B_MOD), blk_stride, mods, st));
    TRY(head_mod(dt, (int)d, eb, hW(m, H_MOD), hmod, st));
    TRY(rope_tables(c.head_dim, w.grid, rcos, rsin, st));
    // text context of each branch, contiguous
    const size_t cbytes = (size_t)Lc * c.text_dim * es;
    for (int b = 0; b < B; ++b) TRACK_HIP(hipMemcpyAsync(ctxb + b * cbytes, ctx[b], cbytes, hipMemcpyDeviceToDevice, st));
  }
  TRY(linear(dt, TRACK_EPI_BIAS_GELU, B * Lc, d, c.text_dim, ctxb, c.text_dim, gW(m, T_TEXT_W1), gW(m, T_TEXT_B1), nullptr, th, d, st));
  TRY(linear(dt, TRACK_EPI_BIAS, B * Lc, d, d, th, d, gW(m, T_TEXT_W2), gW(m, T_TEXT_B2), nullptr, temb, d, st));

  // patch embedding (identical for every branch)
  const void* tokA = x_tok;
  if (dt == TRACK_DTYPE_BF16) {
    ProfScope prof(TRACK_PROF_OTHER, st);
    TRY(to_bf16(x_tok, wsp<bf16_t>(m, w.tok), L * P, st));
    tokA = wsp<void>(m, w.tok);
  }
  TRY(linear(dt, TRACK_EPI_BIAS_F32, L, d, P, tokA, P, gW(m, T_PATCH_W), gW(m, T_PATCH_B), nullptr, X, d, st));
  for (int b = 1; b < B; ++b) TRACK_HIP(hipMemcpyAsync(X + b * L * d, X, (size_t)L * d * 4, hipMemcpyDeviceToDevice, st));

  // bfloat16, whole 8-token groups, at least 128 tokens and a width the
  // 256-wide tiles divide: the V projection writes V^T for attention straight
  // from its epilogue, so V^T's padding columns [L, Lpad) are zeroed once
  // here (nothing else writes them during the forward)
  const bool vt_epi = dt == TRACK_DTYPE_BF16 && L % 8 == 0 && L >= 128 && d % 256 == 0 && d < ((int64_t)1 << 22);
  // bfloat16: the q RMSNorms write q times the softmax scale log2(e) / sqrt(dh)
  // (folded into their one rounding), the input the attention kernel takes
  const bool q_log2 = dt == TRACK_DTYPE_BF16;
  const float qscale = q_log2 ? attn_log2_scale((int)dh) : 1.0f;
  if (vt_epi) {
    ProfScope prof(TRACK_PROF_NORM, st);
    TRY(zero_cols_bf16(Vt, B * d, w.Lpad, L, w.Lpad, st));
  }
  for (int blk = 0; blk < c.blocks; ++blk) {
    const float* md = mods + (int64_t)blk * 6 * d;
    const float *sh1 = md, *sc1 = md + d, *g1 = md + 2 * d, *sh2 = md + 3 * d, *sc2 = md + 4 * d, *g2 = md + 5 * d;
    // self-attention sub-block
    TRY(layernorm(dt, rows, (int)d, X, sc1, sh1, Y, st));
    if (vt_epi) {
      // q and k to QKV (columns 0 .. 2d), v straight to V^T
      TRY(linear(dt, TRACK_EPI_BIAS, rows, 2 * d, d, Y, d, bW(m, blk, B_QKV_W), bW(m, blk, B_QKV_B), nullptr, QKV, 3 * d,
                 st));
      TRY(linear_vt(rows, d, d, Y, d, (const uint8_t*)bW(m, blk, B_QKV_W) + 2 * d * d * es,
                    (const uint8_t*)bW(m, blk, B_QKV_B) + 2 * d * es, L, Vt, w.Lpad, st));
    } else {
      TRY(linear(dt, TRACK_EPI_BIAS, rows, 3 * d, d, Y, d, bW(m, blk, B_QKV_W), bW(m, blk, B_QKV_B), nullptr, QKV, 3 * d, st));
      ProfScope prof(TRACK_PROF_NORM, st);
      TRY(v_transpose(dt, B, (int)H, (int)dh, L, QKV, 3 * d, 2 * d, Vt, w.Lpad, st));
    }
    // q and k of each row in one pass
    TRY(rmsnorm_rope(dt, rows, (int)H, (int)dh, QKV, 3 * d, 0, bW(m, blk, B_NORM_Q), bW(m, blk, B_NORM_K), rcos, rsin,
                     w.grid, L, st, qscale));
    TRY(attention(dt, B, (int)H, (int)dh, L, L, QKV, 3 * d, QKV + d * es, 3 * d, Vt, w.Lpad, AO, d, st, TRACK_PROF_ATTN_SELF,
                  q_log2));
    TRY(linear(dt, TRACK_EPI_GATE_RESID, rows, d, d, AO, d, bW(m, blk, B_O_W), bW(m, blk, B_O_B), g1, X, d, st));
    // cross-attention sub-block
    TRY(layernorm(dt, rows, (int)d, X, nullptr, nullptr, Y, st));
    TRY(linear(dt, TRACK_EPI_BIAS, rows, d, d, Y, d, bW(m, blk, B_CQ_W), bW(m, blk, B_CQ_B), nullptr, QKV, d, st));
    TRY(rmsnorm_rope(dt, rows, (int)H, (int)dh, QKV, d, 0, bW(m, blk, B_NORM_CQ), nullptr, nullptr, nullptr, w.grid, L,
                     st, qscale));
    TRY(linear(dt, TRACK_EPI_BIAS, B * Lc, 2 * d, d, temb, d, bW(m, blk, B_CKV_W), bW(m, blk, B_CKV_B), nullptr, kvc, 2 * d, st));
    TRY(rmsnorm_rope(dt, B * Lc, (int)H, (int)dh, kvc, 2 * d, 0, bW(m, blk, B_NORM_CK), nullptr, nullptr, nullptr, w.grid,
                     Lc, st));
    {
      ProfScope prof(TRACK_PROF_NORM, st);
      TRY(v_transpose(dt, B, (int)H, (int)dh, Lc, kvc, 2 * d, d, vct, w.Lcpad, st));
    }
    TRY(attention(dt, B, (int)H, (int)dh, L, Lc, QKV, d, kvc, 2 * d, vct, w.Lcpad, AO, d, st, TRACK_PROF_ATTN_CROSS,
                  q_log2));
    TRY(linear(dt, TRACK_EPI_RESID, rows, d, d, AO, d, bW(m, blk, B_CO_W), bW(m, blk, B_CO_B), nullptr, X, d, st));
    // MLP sub-block
    TRY(layernorm(dt, rows, (int)d, X, sc2, sh2, Y, st));
    TRY(linear(dt, TRACK_EPI_BIAS_GELU, rows, c.ffn_dim, d, Y, d, bW(m, blk, B_FFN1_W), bW(m, blk, B_FFN1_B), nullptr, Hf, c.ffn_dim, st));
    TRY(linear(dt, TRACK_EPI_GATE_RESID, rows, d, c.ffn_dim, Hf, c.ffn_dim, bW(m, blk, B_FFN2_W), bW(m, blk, B_FFN2_B), g2, X, d, st));
  }
  // head
  TRY(layernorm(dt, rows, (int)d, X, hmod + d, hmod, Y, st));
  TRY(linear(dt, TRACK_EPI_BIAS_F32, rows, P, d, Y, d, hW(m, H_W), hW(m, H_B), nullptr, vel, P, st));
  return TRACK_OK;
}

}  // namespace track
