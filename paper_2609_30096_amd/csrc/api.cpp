// C ABI of the TRACK hot path: argument checking, error reporting, the
// sampler loops (guided prediction, reference-trajectory calibration, routed
// sampling), top-K routing and kernel-class profiling.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <numeric>
#include <string>
#include <vector>

#include "model.h"

struct track_model_t {
  track::Model m;
};

namespace track {

static thread_local std::string g_error;

track_status fail(track_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return s;
}

// ---------------------------------------------------------------- progress
static std::mutex g_progress_mu;
static track_progress_fn g_progress_fn = nullptr;
static void* g_progress_user = nullptr;

// After a completed step: synchronise and report, if a callback is set.
static track_status report_progress(hipStream_t s, int sample, int step, int steps) {
  track_progress_fn fn;
  void* user;
  {
    std::lock_guard<std::mutex> lock(g_progress_mu);
    fn = g_progress_fn;
    user = g_progress_user;
  }
  if (!fn) return TRACK_OK;
  TRACK_HIP(hipStreamSynchronize(s));
  fn(user, sample, step, steps);
  return TRACK_OK;
}

// ---------------------------------------------------------------- profiling
struct ProfState {
  std::mutex mu;
  int32_t mask = 0;  // bit k enables kernel class k
  std::vector<hipEvent_t> pool;                 // free events
  std::vector<std::pair<hipEvent_t, hipEvent_t>> open[TRACK_PROF_KINDS];
};
static ProfState g_prof;

static hipEvent_t prof_event() {
  if (!g_prof.pool.empty()) {
    hipEvent_t e = g_prof.pool.back();
    g_prof.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

ProfScope::ProfScope(int kind_, hipStream_t stream_) : kind(kind_), stream(stream_), slot(-1) {
  std::lock_guard<std::mutex> lock(g_prof.mu);
  if (kind < 0 || kind >= TRACK_PROF_KINDS || !(g_prof.mask & (1 << kind))) return;
  hipEvent_t a = prof_event(), b = prof_event();
  if (!a || !b) return;
  if (hipEventRecord(a, stream) != hipSuccess) return;
  g_prof.open[kind].push_back({a, b});
  slot = (int)g_prof.open[kind].size() - 1;
}

ProfScope::~ProfScope() {
  if (slot < 0) return;
  std::lock_guard<std::mutex> lock(g_prof.mu);
  if (slot < (int)g_prof.open[kind].size()) (void)hipEventRecord(g_prof.open[kind][slot].second, stream);
}

}  // namespace track

using namespace track;

#define TRY(expr)                    \
  do {                               \
    track_status st_ = (expr);       \
    if (st_ != TRACK_OK) return st_; \
  } while (0)

extern "C" {

const char* track_last_error(void) { return g_error.c_str(); }

track_status track_set_progress(track_progress_fn fn, void* user) {
  std::lock_guard<std::mutex> lock(g_progress_mu);
  g_progress_fn = fn;
  g_progress_user = user;
  return TRACK_OK;
}

// ---------------------------------------------------------------- weights
int32_t track_weight_count(const track_dit_config* cfg) {
  if (!cfg || check_config(*cfg) != TRACK_OK) return -1;
  return (int32_t)tensor_names(cfg->blocks).size();
}

size_t track_weights_bytes(const track_dit_config* cfg) {
  if (!cfg || check_config(*cfg) != TRACK_OK) return 0;
  size_t total = 0;
  tensor_specs(*cfg, &total);
  return total;
}

track_status track_weight_info(const track_dit_config* cfg, int32_t index, const char** name, int32_t* ndim,
                               int64_t shape[2], size_t* offset_bytes) {
  if (!cfg) return fail(TRACK_E_INVALID, "weight_info: null config");
  TRY(check_config(*cfg));
  const auto specs = tensor_specs(*cfg, nullptr);
  if (index < 0 || index >= (int32_t)specs.size()) return fail(TRACK_E_INVALID, "weight_info: index %d out of range", index);
  const auto& t = specs[index];
  if (name) *name = tensor_names(cfg->blocks)[index].c_str();
  if (ndim) *ndim = t.ndim;
  if (shape) {
    shape[0] = t.shape[0];
    shape[1] = t.shape[1];
  }
  if (offset_bytes) *offset_bytes = t.offset;
  return TRACK_OK;
}

// ---------------------------------------------------------------- models
track_status track_model_create(const track_dit_config* cfg, const void* dev_weights, size_t bytes, track_model* out) {
  if (!cfg || !dev_weights || !out) return fail(TRACK_E_INVALID, "model_create: null argument");
  TRY(check_config(*cfg));
  if ((uintptr_t)dev_weights & 255) return fail(TRACK_E_INVALID, "model_create: weights must be 256-byte aligned");
  size_t total = 0;
  auto specs = tensor_specs(*cfg, &total);
  if (bytes < total) return fail(TRACK_E_SHAPE, "model_create: weight buffer %zu bytes, need %zu", bytes, total);
  auto* h = new (std::nothrow) track_model_t;
  if (!h) return fail(TRACK_E_NOMEM, "model_create: out of host memory");
  h->m.cfg = *cfg;
  h->m.w = (const uint8_t*)dev_weights;
  h->m.wbytes = bytes;
  h->m.specs = std::move(specs);
  *out = h;
  return TRACK_OK;
}

void track_model_destroy(track_model m) { delete m; }

size_t track_workspace_bytes(track_model m, const track_latent_shape* shape, int32_t batch) {
  if (!m || !shape || (batch != 1 && batch != 2)) return 0;
  if (check_shape(m->m, *shape) != TRACK_OK) return 0;
  return ws_layout(m->m, *shape, batch).total;
}

track_status track_model_set_workspace(track_model m, void* dev_ws, size_t bytes) {
  if (!m) return fail(TRACK_E_INVALID, "set_workspace: null model");
  if (dev_ws && ((uintptr_t)dev_ws & 255)) return fail(TRACK_E_INVALID, "set_workspace: workspace must be 256-byte aligned");
  m->m.ws = (uint8_t*)dev_ws;
  m->m.ws_bytes = dev_ws ? bytes : 0;
  return TRACK_OK;
}

// ---------------------------------------------------------------- helpers
static track_status need_ws(const Model& m, const track_latent_shape& s, int B) {
  const size_t need = ws_layout(m, s, B).total;
  if (!m.ws || m.ws_bytes < need)
    return fail(TRACK_E_NOMEM, "workspace of %zu bytes needed for this shape and batch %d, %zu attached", need, B, m.ws_bytes);
  return TRACK_OK;
}

static track_status check_pair(const Model& L, const Model& S) {
  const auto &a = L.cfg, &b = S.cfg;
  if (a.in_ch != b.in_ch || a.patch_t != b.patch_t || a.patch_h != b.patch_h || a.patch_w != b.patch_w ||
      a.text_dim != b.text_dim || a.dtype != b.dtype)
    return fail(TRACK_E_INCOMPATIBLE, "models do not share latent channels, patch, text width and dtype");
  return TRACK_OK;
}

static track_status check_sampler(const track_sampler_config* sc) {
  if (!sc) return fail(TRACK_E_INVALID, "null sampler config");
  if (sc->steps < 1) return fail(TRACK_E_INVALID, "sampler: steps must be >= 1");
  if (!(sc->shift > 0.0)) return fail(TRACK_E_INVALID, "sampler: shift must be > 0");
  if (!(sc->eps > 0.0)) return fail(TRACK_E_INVALID, "sampler: eps must be > 0");
  if (sc->use_cfg != 0 && sc->use_cfg != 1) return fail(TRACK_E_INVALID, "sampler: use_cfg must be 0 or 1");
  if (sc->solver != TRACK_SOLVER_EULER && sc->solver != TRACK_SOLVER_UNIPC)
    return fail(TRACK_E_INVALID, "sampler: unknown solver %d", sc->solver);
  if (sc->solver == TRACK_SOLVER_UNIPC && (sc->order < 1 || sc->order > 3))
    return fail(TRACK_E_INVALID, "sampler: UniPC order %d outside 1..3", sc->order);
  return TRACK_OK;
}

// sigma_i = s u / (1 + (s - 1) u), u = 1 - i / N, in float64.
static std::vector<double> sigma_table(int N, double shift) {
  std::vector<double> sig(N + 1);
  for (int i = 0; i <= N; ++i) {
    const double u = 1.0 - (double)i / (double)N;
    sig[i] = shift * u / (1.0 + (shift - 1.0) * u);
  }
  return sig;
}

// The scheduler update S of Eq. 2 along one trajectory whose state lives in
// the workspace of model `owner` (the Euler step, or UniPC with its history).
struct Scheduler {
  int solver = TRACK_SOLVER_EULER;
  std::vector<double> sig;
  std::vector<UniPCStep> plan;
  float* xlast = nullptr;
  float* ring[4] = {nullptr, nullptr, nullptr, nullptr};
  int64_t n = 0;

  Scheduler(const Model& owner, const WsLayout& wl, const track_sampler_config& sc) {
    solver = sc.solver;
    sig = sigma_table(sc.steps, sc.shift);
    n = wl.L * wl.P;
    if (solver == TRACK_SOLVER_UNIPC) {
      plan = unipc_plan(sig, sc.order);
      float* base = wsp<float>(owner, wl.sched);
      xlast = base;
      for (int k = 0; k < 4; ++k) ring[k] = base + (size_t)(k + 1) * n;
    }
  }
  // Advances x (token layout) from sigma_i to sigma_{i+1} with the guided
  // velocity of vel_L; with vel_S also writes the Eq. 4 score to r_out.
  track_status advance(int i, int B, float w, const float* vel_L, const float* vel_S, float* x, double* partial,
                       double eps, double* r_out, hipStream_t s) const {
    if (solver == TRACK_SOLVER_EULER)
      return step(n, B, w, (float)(sig[i + 1] - sig[i]), vel_L, vel_S, x, partial, eps, r_out, s);
    const float* h0 = i >= 1 ? ring[(i - 1) & 3] : nullptr;
    const float* h1 = i >= 2 ? ring[(i - 2) & 3] : nullptr;
    const float* h2 = i >= 3 ? ring[(i - 3) & 3] : nullptr;
    return unipc_step(n, B, w, (float)sig[i], plan[i], vel_L, vel_S, x, xlast, h0, h1, h2, ring[i & 3], partial, eps,
                      r_out, s);
  }
};

// ---------------------------------------------------------------- the four calls
track_status track_dit_forward(track_model mh, const track_latent_shape* shape, const float* x_t, double t,
                               const void* cond, const void* uncond, float guidance_scale, float* p_out,
                               void* stream) {
  if (!mh || !shape || !x_t || !cond || !p_out) return fail(TRACK_E_INVALID, "dit_forward: null argument");
  const Model& m = mh->m;
  TRY(check_shape(m, *shape));
  if (!isfinite(t) || !isfinite(guidance_scale)) return fail(TRACK_E_INVALID, "dit_forward: t and guidance must be finite");
  const int B = uncond ? 2 : 1;
  TRY(need_ws(m, *shape, B));
  hipStream_t s = (hipStream_t)stream;
  const WsLayout w = ws_layout(m, *shape, B);
  const auto& c = m.cfg;
  float* xtok = wsp<float>(m, w.xtok);
  float* vel = wsp<float>(m, w.vel);
  {
    ProfScope prof(TRACK_PROF_OTHER, s);
    TRY(patchify(x_t, xtok, c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w, s));
  }
  const void* ctx[2] = {cond, uncond};
  TRY(forward(m, *shape, B, xtok, t, ctx, vel, s));
  TRY(guide_unpatchify(vel, B, guidance_scale, p_out, c.in_ch, shape->frames, shape->height, shape->width, c.patch_t,
                       c.patch_h, c.patch_w, s));
  return TRACK_OK;
}

static track_status calibrate_impl(track_model lh, track_model sh, const track_latent_shape* shape, int32_t M,
                                   const float* const* x_T, const void* const* cond, const void* uncond,
                                   const track_sampler_config* scfg, double* r_out, double* q_out, double* band_r_out,
                                   double* band_q_out, bool bands, float* const* x0_out, void* stream) {
  if (!lh || !sh || !shape || !x_T || !cond) return fail(TRACK_E_INVALID, "calibrate: null argument");
  TRY(check_sampler(scfg));
  if (M < 1) return fail(TRACK_E_INVALID, "calibrate: M must be >= 1");
  if (scfg->use_cfg && !uncond) return fail(TRACK_E_INVALID, "calibrate: guidance needs the negative-prompt embedding");
  const Model& L = lh->m;
  const Model& S = sh->m;
  TRY(check_pair(L, S));
  TRY(check_shape(L, *shape));
  TRY(check_shape(S, *shape));
  const auto& c = L.cfg;
  if (bands) TRY(band_check(c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w));
  const int N = scfg->steps;
  if (N > R_CAPACITY) return fail(TRACK_E_UNSUPPORTED, "calibrate: at most %d steps", R_CAPACITY);
  for (int j = 0; j < M; ++j)
    if (!x_T[j] || !cond[j]) return fail(TRACK_E_INVALID, "calibrate: null latent or conditioning for sample %d", j);
  const int B = scfg->use_cfg ? 2 : 1;
  TRY(need_ws(L, *shape, B));
  TRY(need_ws(S, *shape, B));
  if (L.ws == S.ws) return fail(TRACK_E_INVALID, "calibrate: the two models need separate workspaces");
  hipStream_t s = (hipStream_t)stream;
  const WsLayout wl = ws_layout(L, *shape, B);
  const WsLayout wsm = ws_layout(S, *shape, B);
  float* xtok = wsp<float>(L, wl.xtok);
  float* velL = wsp<float>(L, wl.vel);
  float* velS = wsp<float>(S, wsm.vel);
  double* partial = wsp<double>(L, wl.partial);
  double* rdev = wsp<double>(L, wl.r);
  double* rbdev = wsp<double>(L, wl.rband);
  const int64_t nstep = step_partial_count(wl.L * wl.P);
  const Scheduler sched(L, wl, *scfg);
  const std::vector<double>& sig = sched.sig;
  const float w = (float)scfg->guidance;
  std::vector<double> r((size_t)M * N, 0.0), rb(bands ? (size_t)M * N * 6 : 0, 0.0);
  for (int j = 0; j < M; ++j) {
    const void* ctx[2] = {cond[j], uncond};
    {
      ProfScope prof(TRACK_PROF_OTHER, s);
      TRY(patchify(x_T[j], xtok, c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w, s));
    }
    for (int k = 0; k < N; ++k) {
      const double t = 1000.0 * sig[k];
      TRY(forward(L, *shape, B, xtok, t, ctx, velL, s));
      TRY(forward(S, *shape, B, xtok, t, ctx, velS, s));
      // the band kernels read the velocities, which the update leaves intact
      TRY(sched.advance(k, B, w, velL, velS, xtok, partial, scfg->eps, rdev + k, s));
      if (bands)
        TRY(band_scores(c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w, B, w,
                        velL, velS, partial, nstep, scfg->eps, wsp<uint8_t>(L, wl.band), nullptr, rbdev + 6 * k, s));
      TRY(report_progress(s, j, k, N));
    }
    if (x0_out && x0_out[j]) {
      ProfScope prof(TRACK_PROF_OTHER, s);
      TRY(unpatchify(xtok, x0_out[j], c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w, s));
    }
    TRACK_HIP(hipMemcpyAsync(r.data() + (size_t)j * N, rdev, (size_t)N * sizeof(double), hipMemcpyDeviceToHost, s));
    if (bands)
      TRACK_HIP(hipMemcpyAsync(rb.data() + (size_t)j * N * 6, rbdev, (size_t)N * 6 * sizeof(double),
                               hipMemcpyDeviceToHost, s));
    TRACK_HIP(hipStreamSynchronize(s));
  }
  if (r_out) std::copy(r.begin(), r.end(), r_out);
  if (q_out) {
    for (int k = 0; k < N; ++k) {
      double acc = 0.0;
      for (int j = 0; j < M; ++j) acc += r[(size_t)j * N + k];
      q_out[k] = acc / (double)M;
    }
  }
  if (bands && band_r_out) std::copy(rb.begin(), rb.end(), band_r_out);
  if (bands && band_q_out) {
    for (int k = 0; k < N; ++k)
      for (int b = 0; b < 6; ++b) {
        double acc = 0.0;
        for (int j = 0; j < M; ++j) acc += rb[((size_t)j * N + k) * 6 + b];
        band_q_out[(size_t)k * 6 + b] = acc / (double)M;
      }
  }
  return TRACK_OK;
}

track_status track_calibrate(track_model lh, track_model sh, const track_latent_shape* shape, int32_t M,
                             const float* const* x_T, const void* const* cond, const void* uncond,
                             const track_sampler_config* scfg, double* r_out, double* q_out, float* const* x0_out,
                             void* stream) {
  return calibrate_impl(lh, sh, shape, M, x_T, cond, uncond, scfg, r_out, q_out, nullptr, nullptr, false, x0_out,
                        stream);
}

track_status track_calibrate_bands(track_model lh, track_model sh, const track_latent_shape* shape, int32_t M,
                                   const float* const* x_T, const void* const* cond, const void* uncond,
                                   const track_sampler_config* scfg, double* r_out, double* q_out,
                                   double* band_r_out, double* band_q_out, float* const* x0_out, void* stream) {
  return calibrate_impl(lh, sh, shape, M, x_T, cond, uncond, scfg, r_out, q_out, band_r_out, band_q_out, true, x0_out,
                        stream);
}

size_t track_band_workspace_bytes(const track_latent_shape* shape, int32_t patch_t, int32_t patch_h, int32_t patch_w) {
  if (!shape) return 0;
  if (band_check(shape->channels, shape->frames, shape->height, shape->width, patch_t, patch_h, patch_w) != TRACK_OK)
    return 0;
  return band_workspace_bytes(shape->channels, shape->frames, shape->height, shape->width, patch_t, patch_h, patch_w);
}

track_status track_op_band_energy(const track_latent_shape* shape, int32_t patch_t, int32_t patch_h, int32_t patch_w,
                                  int32_t batch, float guidance, const float* vel_large, const float* vel_small,
                                  void* workspace, size_t workspace_bytes, double* energy_out, void* stream) {
  if (!shape || !vel_large || !vel_small || !workspace || !energy_out)
    return fail(TRACK_E_INVALID, "op_band_energy: null argument");
  TRY(band_check(shape->channels, shape->frames, shape->height, shape->width, patch_t, patch_h, patch_w));
  const size_t need =
      band_workspace_bytes(shape->channels, shape->frames, shape->height, shape->width, patch_t, patch_h, patch_w);
  if (workspace_bytes < need) return fail(TRACK_E_NOMEM, "op_band_energy: workspace of %zu bytes needed", need);
  if ((uintptr_t)workspace & 255) return fail(TRACK_E_INVALID, "op_band_energy: workspace must be 256-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  const double* energy = (const double*)((const uint8_t*)workspace +
                                         band_energy_offset(shape->channels, shape->frames, shape->height,
                                                            shape->width, patch_t, patch_h, patch_w));
  TRY(band_scores(shape->channels, shape->frames, shape->height, shape->width, patch_t, patch_h, patch_w, batch,
                  guidance, vel_large, vel_small, nullptr, 0, 1.0, workspace, nullptr, nullptr, s));
  TRACK_HIP(hipMemcpyAsync(energy_out, energy, 6 * sizeof(double), hipMemcpyDeviceToHost, s));
  TRACK_HIP(hipStreamSynchronize(s));
  return TRACK_OK;
}

track_status track_route_policy(const double* q, int32_t N, int32_t K, int32_t* small_idx) {
  if (!q || N < 1) return fail(TRACK_E_INVALID, "route_policy: need q and N >= 1");
  if (K < 0 || K > N) return fail(TRACK_E_INVALID, "route_policy: K=%d outside [0, N=%d]", K, N);
  if (K > 0 && !small_idx) return fail(TRACK_E_INVALID, "route_policy: null output");
  for (int i = 0; i < N; ++i)
    if (isnan(q[i])) return fail(TRACK_E_INVALID, "route_policy: q[%d] is NaN", i);
  std::vector<int32_t> order(N);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return q[a] < q[b]; });
  std::sort(order.begin(), order.begin() + K);
  std::copy(order.begin(), order.begin() + K, small_idx);
  return TRACK_OK;
}

track_status track_route_threshold(const double* q, int32_t N, double C0, int32_t* small_idx, int32_t* K_out) {
  if (!q || N < 1) return fail(TRACK_E_INVALID, "route_threshold: need q and N >= 1");
  if (!small_idx || !K_out) return fail(TRACK_E_INVALID, "route_threshold: null output");
  if (isnan(C0)) return fail(TRACK_E_INVALID, "route_threshold: C0 is NaN");
  for (int i = 0; i < N; ++i)
    if (isnan(q[i])) return fail(TRACK_E_INVALID, "route_threshold: q[%d] is NaN", i);
  int32_t n = 0;
  for (int32_t k = 0; k < N; ++k)
    if (q[k] * q[k] < C0) small_idx[n++] = k;  // beta_k = 1 iff W_k < C_0 (Eq. 7)
  *K_out = n;
  return TRACK_OK;
}

namespace {
// SplitMix64 (Steele, Lea and Flood, 2014): Weyl increment, then two
// xor-shift-multiply rounds and a final xor-shift.
uint64_t splitmix64_next(uint64_t& state) {
  state += 0x9E3779B97F4A7C15ull;
  uint64_t z = state;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
}  // namespace

track_status track_route_baseline(int32_t kind, int32_t N, int32_t K, uint64_t seed, int32_t* small_idx) {
  if (N < 1) return fail(TRACK_E_INVALID, "route_baseline: N=%d < 1", N);
  if (K < 0 || K > N) return fail(TRACK_E_INVALID, "route_baseline: K=%d outside [0, N=%d]", K, N);
  if (K > 0 && !small_idx) return fail(TRACK_E_INVALID, "route_baseline: null output");
  switch (kind) {
    case TRACK_POLICY_FIRST_K:
      for (int32_t i = 0; i < K; ++i) small_idx[i] = i;
      return TRACK_OK;
    case TRACK_POLICY_LAST_K:
      for (int32_t i = 0; i < K; ++i) small_idx[i] = N - K + i;
      return TRACK_OK;
    case TRACK_POLICY_RANDOM_K: {
      std::vector<uint64_t> key(N);
      uint64_t state = seed;
      for (int32_t k = 0; k < N; ++k) key[k] = splitmix64_next(state);
      std::vector<int32_t> order(N);
      std::iota(order.begin(), order.end(), 0);
      std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return key[a] < key[b]; });
      std::sort(order.begin(), order.begin() + K);
      std::copy(order.begin(), order.begin() + K, small_idx);
      return TRACK_OK;
    }
    default:
      return fail(TRACK_E_INVALID, "route_baseline: unknown policy kind %d", kind);
  }
}

track_status track_sample(track_model lh, track_model sh, const uint8_t* use_small, const track_latent_shape* shape,
                          const track_sampler_config* scfg, const float* x_T, const void* cond, const void* uncond,
                          float* x0_out, void* stream) {
  if (!lh || !use_small || !shape || !x_T || !cond || !x0_out) return fail(TRACK_E_INVALID, "sample: null argument");
  TRY(check_sampler(scfg));
  if (scfg->use_cfg && !uncond) return fail(TRACK_E_INVALID, "sample: guidance needs the negative-prompt embedding");
  const int N = scfg->steps;
  bool any_small = false;
  for (int i = 0; i < N; ++i) any_small |= use_small[i] != 0;
  if (any_small && !sh) return fail(TRACK_E_INVALID, "sample: policy routes steps to a null small model");
  const Model& L = lh->m;
  TRY(check_shape(L, *shape));
  const int B = scfg->use_cfg ? 2 : 1;
  TRY(need_ws(L, *shape, B));
  if (any_small) {
    TRY(check_pair(L, sh->m));
    TRY(check_shape(sh->m, *shape));
    TRY(need_ws(sh->m, *shape, B));
  }
  hipStream_t s = (hipStream_t)stream;
  const WsLayout wl = ws_layout(L, *shape, B);
  const auto& c = L.cfg;
  float* xtok = wsp<float>(L, wl.xtok);
  const Scheduler sched(L, wl, *scfg);
  const std::vector<double>& sig = sched.sig;
  const float w = (float)scfg->guidance;
  const void* ctx[2] = {cond, uncond};
  {
    ProfScope prof(TRACK_PROF_OTHER, s);
    TRY(patchify(x_T, xtok, c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w, s));
  }
  for (int i = 0; i < N; ++i) {
    const Model& m = use_small[i] ? sh->m : L;
    float* vel = wsp<float>(m, ws_layout(m, *shape, B).vel);
    TRY(forward(m, *shape, B, xtok, 1000.0 * sig[i], ctx, vel, s));
    // UniPC's history is one sequence whichever model produced each entry
    TRY(sched.advance(i, B, w, vel, nullptr, xtok, nullptr, 0.0, nullptr, s));
    TRY(report_progress(s, -1, i, N));
  }
  {
    ProfScope prof(TRACK_PROF_OTHER, s);
    TRY(unpatchify(xtok, x0_out, c.in_ch, shape->frames, shape->height, shape->width, c.patch_t, c.patch_h, c.patch_w, s));
  }
  return TRACK_OK;
}

// ---------------------------------------------------------------- component entry points
track_status track_unipc_coefficients(int32_t N, double shift, int32_t order, int32_t step_index, double* coef) {
  if (!coef) return fail(TRACK_E_INVALID, "unipc_coefficients: null output");
  if (N < 1 || !(shift > 0.0)) return fail(TRACK_E_INVALID, "unipc_coefficients: need N >= 1 and shift > 0");
  if (order < 1 || order > 3) return fail(TRACK_E_INVALID, "unipc_coefficients: order %d outside 1..3", order);
  if (step_index < 0 || step_index >= N) return fail(TRACK_E_INVALID, "unipc_coefficients: step %d outside [0, N)", step_index);
  const UniPCStep c = unipc_plan(sigma_table(N, shift), order)[step_index];
  const double v[12] = {c.cx, c.c_m0, c.c_h[0], c.c_h[1], c.c_new, (double)c.corr, (double)c.nh_c,
                        c.px, c.p_m,  c.p_h[0], c.p_h[1], (double)c.nh_p};
  std::copy(v, v + 12, coef);
  return TRACK_OK;
}

track_status track_op_unipc_step(int64_t n, int32_t batch, float guidance, float sigma, const double* coef,
                                 const float* vel_L, const float* vel_S, float* x, float* x_last, const float* h0,
                                 const float* h1, const float* h2, float* m_out, double* partial, double eps,
                                 double* r_out, void* stream) {
  if (!coef) return fail(TRACK_E_INVALID, "op_unipc_step: null coefficients");
  UniPCStep c;
  c.cx = coef[0];
  c.c_m0 = coef[1];
  c.c_h[0] = coef[2];
  c.c_h[1] = coef[3];
  c.c_new = coef[4];
  c.corr = coef[5] != 0.0;
  c.nh_c = (int)coef[6];
  c.px = coef[7];
  c.p_m = coef[8];
  c.p_h[0] = coef[9];
  c.p_h[1] = coef[10];
  c.nh_p = (int)coef[11];
  return unipc_step(n, batch, guidance, sigma, c, vel_L, vel_S, x, x_last, h0, h1, h2, m_out, partial, eps, r_out,
                    (hipStream_t)stream);
}


track_status track_op_linear(int32_t dtype, int32_t epilogue, int64_t M, int64_t N, int64_t K, const void* A,
                             int64_t lda, const void* W, const void* bias, const float* gate, void* out, int64_t ldo,
                             void* stream) {
  return linear(dtype, epilogue, M, N, K, A, lda, W, bias, gate, out, ldo, (hipStream_t)stream);
}

track_status track_op_linear_vt(int32_t dtype, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                                const void* W, const void* bias, int64_t L, void* vt, int64_t ldv, void* stream) {
  if (dtype != TRACK_DTYPE_BF16) return fail(TRACK_E_UNSUPPORTED, "linear_vt: bfloat16 only");
  return linear_vt(M, N, K, A, lda, W, bias, L, vt, ldv, (hipStream_t)stream);
}

track_status track_op_attention(int32_t dtype, int32_t B, int32_t H, int32_t head_dim, int64_t Lq, int64_t Lk,
                                const void* q, int64_t ldq, const void* k, int64_t ldk, const void* vt, int64_t ldv,
                                void* out, int64_t ldo, void* stream) {
  return attention(dtype, B, H, head_dim, Lq, Lk, q, ldq, k, ldk, vt, ldv, out, ldo, (hipStream_t)stream,
                   TRACK_PROF_ATTN_SELF);
}

track_status track_op_attention_log2q(int32_t dtype, int32_t B, int32_t H, int32_t head_dim, int64_t Lq, int64_t Lk,
                                      const void* q, int64_t ldq, const void* k, int64_t ldk, const void* vt,
                                      int64_t ldv, void* out, int64_t ldo, void* stream) {
  return attention(dtype, B, H, head_dim, Lq, Lk, q, ldq, k, ldk, vt, ldv, out, ldo, (hipStream_t)stream,
                   TRACK_PROF_ATTN_SELF, true);
}

track_status track_op_layernorm(int32_t dtype, int64_t rows, int32_t d, const float* x, const float* scale,
                                const float* shift, void* y, void* stream) {
  if (!x || !y) return fail(TRACK_E_INVALID, "layernorm: null pointer");
  if (dtype != TRACK_DTYPE_F32 && dtype != TRACK_DTYPE_BF16) return fail(TRACK_E_INVALID, "layernorm: bad dtype");
  if (d < 1) return fail(TRACK_E_SHAPE, "layernorm: width %d", (int)d);
  return layernorm(dtype, rows, d, x, scale, shift, y, (hipStream_t)stream);
}

int64_t track_rope_table_len(int32_t head_dim, const int32_t* grid) {
  if (!grid || head_dim < 4 || grid[0] < 1 || grid[1] < 1 || grid[2] < 1) return -1;
  const int ds = 2 * (head_dim / 6), df = head_dim - 2 * ds;
  return (int64_t)grid[0] * (df / 2) + (int64_t)(grid[1] + grid[2]) * (ds / 2);
}

static track_status op_rmsnorm_rope(int32_t dtype, int64_t rows, int32_t heads, int32_t head_dim, void* buf,
                                    int64_t ld, int64_t col0, const void* g, const void* g2, const int32_t* grid,
                                    float* rope_ws, void* stream) {
  if (!buf || !g) return fail(TRACK_E_INVALID, "rmsnorm_rope: null pointer");
  if (dtype != TRACK_DTYPE_F32 && dtype != TRACK_DTYPE_BF16) return fail(TRACK_E_INVALID, "rmsnorm_rope: bad dtype");
  const int64_t width = (int64_t)heads * head_dim * (g2 ? 2 : 1);
  if (heads < 1 || head_dim < 4 || col0 < 0 || ld < col0 + width) return fail(TRACK_E_SHAPE, "rmsnorm_rope: bad shape");
  hipStream_t s = (hipStream_t)stream;
  if (!grid) return rmsnorm_rope(dtype, rows, heads, head_dim, buf, ld, col0, g, g2, nullptr, nullptr, Grid3{1, 1, 1}, 1, s);
  const int64_t len = track_rope_table_len(head_dim, grid);
  if (len < 0) return fail(TRACK_E_SHAPE, "rmsnorm_rope: bad grid");
  if (!rope_ws) return fail(TRACK_E_INVALID, "rmsnorm_rope: RoPE needs rope_ws");
  const Grid3 g3{grid[0], grid[1], grid[2]};
  TRY(rope_tables(head_dim, g3, rope_ws, rope_ws + len, s));
  return rmsnorm_rope(dtype, rows, heads, head_dim, buf, ld, col0, g, g2, rope_ws, rope_ws + len, g3,
                      (int64_t)g3.f * g3.h * g3.w, s);
}

track_status track_op_rmsnorm_rope(int32_t dtype, int64_t rows, int32_t heads, int32_t head_dim, void* buf, int64_t ld,
                                   int64_t col0, const void* g, const int32_t* grid, float* rope_ws, void* stream) {
  return op_rmsnorm_rope(dtype, rows, heads, head_dim, buf, ld, col0, g, nullptr, grid, rope_ws, stream);
}

track_status track_op_rmsnorm_rope_qk(int32_t dtype, int64_t rows, int32_t heads, int32_t head_dim, void* buf,
                                      int64_t ld, int64_t col0, const void* g_q, const void* g_k, const int32_t* grid,
                                      float* rope_ws, void* stream) {
  if (!g_k) return fail(TRACK_E_INVALID, "rmsnorm_rope_qk: null pointer");
  return op_rmsnorm_rope(dtype, rows, heads, head_dim, buf, ld, col0, g_q, g_k, grid, rope_ws, stream);
}

int64_t track_step_partial_count(int64_t n) { return step_partial_count(n); }

track_status track_op_step(int64_t n, int32_t B, float guidance, float dsigma, const float* vel_L, const float* vel_S,
                           float* x, double* partial, double eps, double* r_out, void* stream) {
  return step(n, B, guidance, dsigma, vel_L, vel_S, x, partial, eps, r_out, (hipStream_t)stream);
}

track_status track_hbm_stream(int32_t kind, const void* src, void* dst, int64_t bytes, void* stream) {
  return hbm_stream(kind, src, dst, bytes, (hipStream_t)stream);
}

track_status track_mfma_stream(const void* operands, int64_t iters, float* sink, int64_t* flop, void* stream) {
  return mfma_stream(operands, iters, sink, flop, (hipStream_t)stream);
}

track_status track_op_step_noalloc(int64_t n, int32_t B, float guidance, float dsigma, const float* vel_L,
                                   const float* vel_S, float* x, double eps, double* r_out, void* stream) {
  return step_static(n, B, guidance, dsigma, vel_L, vel_S, x, eps, r_out, (hipStream_t)stream);
}

// ---------------------------------------------------------------- profiling
track_status track_profile_enable(int32_t kind_mask) {
  std::lock_guard<std::mutex> lock(g_prof.mu);
  g_prof.mask = kind_mask & ((1 << TRACK_PROF_KINDS) - 1);
  return TRACK_OK;
}

track_status track_profile_reset(void) {
  TRACK_HIP(hipDeviceSynchronize());
  std::lock_guard<std::mutex> lock(g_prof.mu);
  for (auto& v : g_prof.open) {
    for (auto& p : v) {
      g_prof.pool.push_back(p.first);
      g_prof.pool.push_back(p.second);
    }
    v.clear();
  }
  return TRACK_OK;
}

track_status track_profile_read(int32_t kind, int64_t* launches, double* total_ms) {
  if (kind < 0 || kind >= TRACK_PROF_KINDS) return fail(TRACK_E_INVALID, "profile_read: bad kind");
  TRACK_HIP(hipDeviceSynchronize());
  std::lock_guard<std::mutex> lock(g_prof.mu);
  double tot = 0.0;
  for (auto& p : g_prof.open[kind]) {
    float ms = 0.0f;
    TRACK_HIP(hipEventElapsedTime(&ms, p.first, p.second));
    tot += ms;
  }
  if (launches) *launches = (int64_t)g_prof.open[kind].size();
  if (total_ms) *total_ms = tot;
  return TRACK_OK;
}

}  // extern "C"
