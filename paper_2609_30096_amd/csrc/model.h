// Host-side model description: weight table, workspace layout and the
// denoiser forward as a kernel sequence on one stream.
#pragma once

#include <string>
#include <vector>

#include "kernels.h"

namespace track {

struct TensorSpec {
  std::string name;
  int ndim;
  int64_t shape[2];
  size_t offset;  // bytes
};

// Validate a config; returns TRACK_OK or sets the error.
track_status check_config(const track_dit_config& c);
// Ordered tensor list with 256-byte aligned offsets; total bytes in *total.
std::vector<TensorSpec> tensor_specs(const track_dit_config& c, size_t* total);
// Stable storage for the names of a config with `blocks` blocks.
const std::vector<std::string>& tensor_names(int blocks);

inline size_t dtype_size(int dtype) { return dtype == TRACK_DTYPE_BF16 ? 2 : 4; }
inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }
inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Byte offsets of the workspace regions for one latent shape and batch.
struct WsLayout {
  size_t sin, h, e, se, m, mods, hmod, rope_cos, rope_sin;
  size_t ctx, th, temb, kvc, vct, tok;
  size_t X, Y, QKV, Vt, AO, Hf, vel, xtok, partial, r, band, rband, sched;
  size_t total;
  int64_t L, Lpad, Lc, Lcpad, P;
  Grid3 grid;
  int rope_len;  // floats per cos (or sin) table
};

constexpr int R_CAPACITY = 4096;  // disagreement scores buffered on the device per sample

struct Model {
  track_dit_config cfg;
  const uint8_t* w = nullptr;
  size_t wbytes = 0;
  std::vector<TensorSpec> specs;
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
};

track_status check_shape(const Model& m, const track_latent_shape& s);
WsLayout ws_layout(const Model& m, const track_latent_shape& s, int B);

// f(x_tok, t, ctx_b) for b < B; vel [B, L, P] float32 in token layout.
// x_tok [L, P] float32.  Uses m's workspace.
track_status forward(const Model& m, const track_latent_shape& s, int B, const float* x_tok, double t,
                     const void* const* ctx, float* vel, hipStream_t stream);

// Pointer into m's workspace.
template <typename T>
inline T* wsp(const Model& m, size_t off) {
  return (T*)(m.ws + off);
}

}  // namespace track
