"""Python binding of libtrack.so (the C ABI declared in include/track.h).

Argument marshalling only: every step of the denoiser, the sampler loops and
the routing run inside the library.  torch provides device memory and the
current stream.  The library must have been built (``__graft_entry__.build()``
or ``python -m paper_2609_30096_amd.build``); without it every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import synth

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtrack.so")
_lib = None

OK, E_INVALID, E_SHAPE, E_INCOMPATIBLE, E_DEVICE, E_NOMEM, E_UNSUPPORTED = range(7)
DTYPE_F32, DTYPE_BF16 = 0, 1
EPI_BIAS, EPI_BIAS_GELU, EPI_GATE_RESID, EPI_RESID, EPI_BIAS_F32 = range(5)
PROF_ATTN_SELF, PROF_ATTN_CROSS, PROF_GEMM, PROF_NORM, PROF_STEP, PROF_OTHER = range(6)

EXPORTS = [
    "track_weight_count", "track_weights_bytes", "track_weight_info", "track_model_create", "track_model_destroy",
    "track_workspace_bytes", "track_model_set_workspace", "track_dit_forward", "track_calibrate",
    "track_calibrate_bands", "track_band_workspace_bytes", "track_op_band_energy",
    "track_route_policy", "track_route_threshold", "track_route_baseline", "track_sample", "track_last_error",
    "track_op_linear", "track_op_linear_vt", "track_op_attention", "track_op_attention_log2q",
    "track_op_layernorm", "track_rope_table_len", "track_op_rmsnorm_rope", "track_op_rmsnorm_rope_qk", "track_step_partial_count",
    "track_op_step", "track_op_step_noalloc", "track_hbm_stream", "track_mfma_stream", "track_unipc_coefficients", "track_op_unipc_step", "track_profile_enable", "track_profile_reset", "track_profile_read", "track_set_progress",
]


class TrackError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"[track status {status}] {msg}")
        self.status = status


class DitConfigC(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "blocks", "dim", "heads", "head_dim", "ffn_dim", "in_ch", "patch_t", "patch_h", "patch_w",
        "text_dim", "freq_dim", "dtype")]


class LatentShapeC(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("channels", "frames", "height", "width", "text_len")]


class SamplerConfigC(ctypes.Structure):
    _fields_ = [("steps", ctypes.c_int32), ("use_cfg", ctypes.c_int32), ("shift", ctypes.c_double),
                ("guidance", ctypes.c_double), ("eps", ctypes.c_double), ("solver", ctypes.c_int32),
                ("order", ctypes.c_int32)]


SOLVERS = {"euler": 0, "unipc": 1}


_vp, _i32, _i64, _f32, _f64, _sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float,
                                    ctypes.c_double, ctypes.c_size_t)
PROGRESS_FN = ctypes.CFUNCTYPE(None, ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32)
_progress_ref = None


def _declare(L):
    P = ctypes.POINTER
    sig = {
        "track_weight_count": (_i32, [P(DitConfigC)]),
        "track_weights_bytes": (_sz, [P(DitConfigC)]),
        "track_weight_info": (_i32, [P(DitConfigC), _i32, P(ctypes.c_char_p), P(_i32), P(_i64), P(_sz)]),
        "track_model_create": (_i32, [P(DitConfigC), _vp, _sz, P(_vp)]),
        "track_model_destroy": (None, [_vp]),
        "track_workspace_bytes": (_sz, [_vp, P(LatentShapeC), _i32]),
        "track_model_set_workspace": (_i32, [_vp, _vp, _sz]),
        "track_dit_forward": (_i32, [_vp, P(LatentShapeC), _vp, _f64, _vp, _vp, _f32, _vp, _vp]),
        "track_calibrate": (_i32, [_vp, _vp, P(LatentShapeC), _i32, P(_vp), P(_vp), _vp, P(SamplerConfigC),
                                   P(_f64), P(_f64), P(_vp), _vp]),
        "track_calibrate_bands": (_i32, [_vp, _vp, P(LatentShapeC), _i32, P(_vp), P(_vp), _vp, P(SamplerConfigC),
                                         P(_f64), P(_f64), P(_f64), P(_f64), P(_vp), _vp]),
        "track_band_workspace_bytes": (_sz, [P(LatentShapeC), _i32, _i32, _i32]),
        "track_op_band_energy": (_i32, [P(LatentShapeC), _i32, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _sz, P(_f64),
                                        _vp]),
        "track_route_policy": (_i32, [P(_f64), _i32, _i32, P(_i32)]),
        "track_route_threshold": (_i32, [P(_f64), _i32, _f64, P(_i32), P(_i32)]),
        "track_route_baseline": (_i32, [_i32, _i32, _i32, ctypes.c_uint64, P(_i32)]),
        "track_sample": (_i32, [_vp, _vp, P(ctypes.c_uint8), P(LatentShapeC), P(SamplerConfigC), _vp, _vp, _vp,
                                _vp, _vp]),
        "track_last_error": (ctypes.c_char_p, []),
        "track_op_linear": (_i32, [_i32, _i32, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _vp, _vp, _i64, _vp]),
        "track_op_linear_vt": (_i32, [_i32, _i64, _i64, _i64, _vp, _i64, _vp, _vp, _i64, _vp, _i64, _vp]),
        "track_op_attention": (_i32, [_i32, _i32, _i32, _i32, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _i64, _vp,
                                      _i64, _vp]),
        "track_op_attention_log2q": (_i32, [_i32, _i32, _i32, _i32, _i64, _i64, _vp, _i64, _vp, _i64, _vp, _i64, _vp,
                                      _i64, _vp]),
        "track_op_layernorm": (_i32, [_i32, _i64, _i32, _vp, _vp, _vp, _vp, _vp]),
        "track_rope_table_len": (_i64, [_i32, P(_i32)]),
        "track_op_rmsnorm_rope": (_i32, [_i32, _i64, _i32, _i32, _vp, _i64, _i64, _vp, P(_i32), _vp, _vp]),
        "track_op_rmsnorm_rope_qk": (_i32, [_i32, _i64, _i32, _i32, _vp, _i64, _i64, _vp, _vp, P(_i32), _vp, _vp]),
        "track_step_partial_count": (_i64, [_i64]),
        "track_op_step": (_i32, [_i64, _i32, _f32, _f32, _vp, _vp, _vp, _vp, _f64, _vp, _vp]),
        "track_op_step_noalloc": (_i32, [_i64, _i32, _f32, _f32, _vp, _vp, _vp, _f64, _vp, _vp]),
        "track_unipc_coefficients": (_i32, [_i32, _f64, _i32, _i32, P(_f64)]),
        "track_op_unipc_step": (_i32, [_i64, _i32, _f32, _f32, P(_f64), _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                       _f64, _vp, _vp]),
        "track_hbm_stream": (_i32, [_i32, _vp, _vp, _i64, _vp]),
        "track_mfma_stream": (_i32, [_vp, _i64, _vp, ctypes.POINTER(ctypes.c_int64), _vp]),
        "track_profile_enable": (_i32, [_i32]),
        "track_profile_reset": (_i32, []),
        "track_profile_read": (_i32, [_i32, P(_i64), P(_f64)]),
        "track_set_progress": (_i32, [PROGRESS_FN, _vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args


def lib():
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with `python -m paper_2609_30096_amd.build`")
        L = ctypes.CDLL(_LIB_PATH)
        _declare(L)
        _lib = L
    return _lib


def _check(status: int):
    if status != OK:
        raise TrackError(status, lib().track_last_error().decode())


def _torch():
    import torch
    return torch


def _stream():
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ptr(t) -> ctypes.c_void_p:
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


def dtype_code(dtype: str) -> int:
    return DTYPE_BF16 if dtype == synth.BF16 else DTYPE_F32


def torch_dtype(dtype: str):
    torch = _torch()
    return torch.bfloat16 if dtype == synth.BF16 else torch.float32


def config_c(cfg: synth.DiTConfig) -> DitConfigC:
    pt, ph, pw = cfg.patch
    return DitConfigC(cfg.blocks, cfg.dim, cfg.heads, cfg.head_dim, cfg.ffn_dim, cfg.in_ch, pt, ph, pw,
                      cfg.text_dim, cfg.freq_dim, dtype_code(cfg.dtype))


def shape_c(shape: synth.LatentShape) -> LatentShapeC:
    return LatentShapeC(shape.channels, shape.frames, shape.height, shape.width, shape.text_len)


def sampler_c(scfg: synth.SamplerConfig) -> SamplerConfigC:
    return SamplerConfigC(scfg.steps, 1 if scfg.use_cfg else 0, scfg.shift, scfg.guidance, scfg.eps,
                          SOLVERS[scfg.solver], scfg.order)


# ---------------------------------------------------------------- weights and models
def weight_table(cfg: synth.DiTConfig) -> Tuple[List[Tuple[str, Tuple[int, ...], int]], int]:
    """[(name, shape, byte offset)] in buffer order, and the buffer size."""
    L = lib()
    c = config_c(cfg)
    n = L.track_weight_count(ctypes.byref(c))
    if n < 0:
        raise TrackError(E_INVALID, "invalid config: " + L.track_last_error().decode())
    out = []
    for i in range(n):
        name = ctypes.c_char_p()
        nd = _i32()
        shp = (_i64 * 2)()
        off = _sz()
        _check(L.track_weight_info(ctypes.byref(c), i, ctypes.byref(name), ctypes.byref(nd), shp, ctypes.byref(off)))
        out.append((name.value.decode(), tuple(shp[:nd.value]), off.value))
    return out, L.track_weights_bytes(ctypes.byref(c))


def pack_weights(cfg: synth.DiTConfig, params: Dict[str, np.ndarray], device="cuda"):
    """Device weight buffer (uint8 tensor) holding ``params`` in the library's layout."""
    torch = _torch()
    table, total = weight_table(cfg)
    buf = torch.empty(total, dtype=torch.uint8, device=device)
    tdt = torch_dtype(cfg.dtype)
    es = 2 if cfg.dtype == synth.BF16 else 4
    for name, shape, off in table:
        a = params[name]
        if tuple(a.shape) != shape:
            raise ValueError(f"{name}: shape {a.shape} != {shape}")
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device).to(tdt).reshape(-1)
        buf[off:off + t.numel() * es].view(tdt).copy_(t)
    return buf


def gen_weights_on_device(cfg: synth.DiTConfig, model_seed: int, device="cuda", threads: int = 16):
    """pack_weights of the seeded recipe; drawn on host threads chunk by chunk, one block at a time."""
    import concurrent.futures as cf
    torch = _torch()
    table, total = weight_table(cfg)
    specs = synth.param_specs(cfg)
    for i, (name, _, _) in enumerate(table):
        if specs[i][0] != name:
            raise ValueError(f"tensor order mismatch at {i}: {specs[i][0]} vs {name}")
    buf = torch.empty(total, dtype=torch.uint8, device=device)
    tdt = torch_dtype(cfg.dtype)
    es = 2 if cfg.dtype == synth.BF16 else 4
    # groups of tensors generated together: the globals, each block, the head
    groups, cur, prefix = [], [], None
    for i, (name, _, _) in enumerate(table):
        p = name.split(".")[0] if name.startswith("blk") else ("head" if name.startswith("head") else "global")
        if p != prefix and cur:
            groups.append(cur)
            cur = []
        prefix = p
        cur.append(i)
    groups.append(cur)
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        for g in groups:
            arrs = synth.gen_param_set(cfg, model_seed, g, ex, round_to_dtype=False)
            for i in g:
                name, shape, off = table[i]
                # float32 -> bf16 rounds to nearest even on the device
                t = torch.from_numpy(arrs[name]).reshape(-1).to(device).to(tdt)
                buf[off:off + t.numel() * es].view(tdt).copy_(t)
    return buf


class Model:
    """A model handle over a device weight buffer, with a torch-allocated workspace."""

    def __init__(self, cfg: synth.DiTConfig, weights):
        self.cfg = cfg
        self.weights = weights
        self._c = config_c(cfg)
        h = _vp()
        _check(lib().track_model_create(ctypes.byref(self._c), _ptr(weights), weights.numel(), ctypes.byref(h)))
        self.handle = h
        self.workspace = None

    def workspace_bytes(self, shape: synth.LatentShape, batch: int) -> int:
        n = lib().track_workspace_bytes(self.handle, ctypes.byref(shape_c(shape)), batch)
        if n == 0:
            raise TrackError(E_SHAPE, f"latent shape {shape} is invalid for this model")
        return n

    def ensure_workspace(self, shape: synth.LatentShape, batch: int):
        need = self.workspace_bytes(shape, batch)
        if self.workspace is None or self.workspace.numel() < need:
            torch = _torch()
            self.workspace = None
            self.workspace = torch.empty(need, dtype=torch.uint8, device=self.weights.device)
            _check(lib().track_model_set_workspace(self.handle, _ptr(self.workspace), need))

    def close(self):
        if getattr(self, "handle", None):
            lib().track_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- the four calls
def dit_forward(model: Model, shape: synth.LatentShape, x_t, t: float, cond, uncond=None, guidance: float = 1.0):
    """Guided prediction p(x_t, t) (Eq. 1); x_t: device [C, F, H, W] float32."""
    torch = _torch()
    model.ensure_workspace(shape, 2 if uncond is not None else 1)
    out = torch.empty_like(x_t)
    _check(lib().track_dit_forward(model.handle, ctypes.byref(shape_c(shape)), _ptr(x_t), float(t), _ptr(cond),
                                   _ptr(uncond), float(guidance), _ptr(out), _stream()))
    return out


def calibrate(large: Model, small: Model, shape: synth.LatentShape, x_T: Sequence, conds: Sequence, uncond,
              scfg: synth.SamplerConfig, return_x0: bool = False, bands: bool = False):
    """Reference-trajectory calibration; returns (r [M, N], q [N]) as float64 numpy arrays.

    With bands, also the band scores (rb [M, N, 6], qb [N, 6]: spatial low,
    mid, high, temporal low, mid, high).  With return_x0, also the list of
    each sample's all-large endpoint (device tensors), last.
    """
    torch = _torch()
    B = 2 if scfg.use_cfg else 1
    large.ensure_workspace(shape, B)
    small.ensure_workspace(shape, B)
    M, N = len(x_T), scfg.steps
    xs = (_vp * M)(*[t.data_ptr() for t in x_T])
    cs = (_vp * M)(*[t.data_ptr() for t in conds])
    r = np.zeros((M, N), dtype=np.float64)
    q = np.zeros(N, dtype=np.float64)
    sc = sampler_c(scfg)
    x0 = [torch.empty_like(t) for t in x_T] if return_x0 else None
    x0p = (_vp * M)(*[t.data_ptr() for t in x0]) if return_x0 else None
    if bands:
        rb = np.zeros((M, N, 6), dtype=np.float64)
        qb = np.zeros((N, 6), dtype=np.float64)
        _check(lib().track_calibrate_bands(large.handle, small.handle, ctypes.byref(shape_c(shape)), M, xs, cs,
                                           _ptr(uncond), ctypes.byref(sc), r.ctypes.data_as(ctypes.POINTER(_f64)),
                                           q.ctypes.data_as(ctypes.POINTER(_f64)),
                                           rb.ctypes.data_as(ctypes.POINTER(_f64)),
                                           qb.ctypes.data_as(ctypes.POINTER(_f64)), x0p, _stream()))
        out = (r, q, rb, qb)
    else:
        _check(lib().track_calibrate(large.handle, small.handle, ctypes.byref(shape_c(shape)), M, xs, cs,
                                     _ptr(uncond), ctypes.byref(sc), r.ctypes.data_as(ctypes.POINTER(_f64)),
                                     q.ctypes.data_as(ctypes.POINTER(_f64)), x0p, _stream()))
        out = (r, q)
    return out + (x0,) if return_x0 else out


def route_policy(q, K: int) -> np.ndarray:
    """Indices of the K lowest scores, ascending (ties to the lower index)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    out = np.zeros(max(K, 1), dtype=np.int32)
    _check(lib().track_route_policy(q.ctypes.data_as(ctypes.POINTER(_f64)), len(q), int(K),
                                    out.ctypes.data_as(ctypes.POINTER(_i32))))
    return out[:K].copy()


def route_threshold(q, C0: float) -> np.ndarray:
    """Steps with q_k^2 < C0 (Eqs. 6-7, C_0 form), ascending."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    out = np.zeros(len(q), dtype=np.int32)
    n = _i32(0)
    _check(lib().track_route_threshold(q.ctypes.data_as(ctypes.POINTER(_f64)), len(q), float(C0),
                                       out.ctypes.data_as(ctypes.POINTER(_i32)), ctypes.byref(n)))
    return out[:n.value].copy()


POLICY_FIRST_K, POLICY_LAST_K, POLICY_RANDOM_K = 0, 1, 2


def route_baseline(kind: int, N: int, K: int, seed: int = 0) -> np.ndarray:
    """Equal-budget baseline policy (First-K, Last-K, Random-K): K step indices, ascending."""
    out = np.zeros(max(K, 1), dtype=np.int32)
    _check(lib().track_route_baseline(int(kind), int(N), int(K), int(seed) & (2**64 - 1),
                                      out.ctypes.data_as(ctypes.POINTER(_i32))))
    return out[:K].copy()


def sample(large: Model, small: Optional[Model], use_small, shape: synth.LatentShape, scfg: synth.SamplerConfig,
           x_T, cond, uncond=None, out=None):
    """Routed sampling (Eq. 3); returns x_0 as a device tensor [C, F, H, W] (in `out` if given,
    which may be x_T itself)."""
    torch = _torch()
    B = 2 if scfg.use_cfg else 1
    large.ensure_workspace(shape, B)
    if small is not None:
        small.ensure_workspace(shape, B)
    pol = np.ascontiguousarray(np.asarray(use_small, dtype=bool).astype(np.uint8))
    if pol.shape != (scfg.steps,):
        raise ValueError("use_small must have one entry per step")
    out = torch.empty_like(x_T) if out is None else out
    sc = sampler_c(scfg)
    _check(lib().track_sample(large.handle, None if small is None else small.handle,
                              pol.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), ctypes.byref(shape_c(shape)),
                              ctypes.byref(sc), _ptr(x_T), _ptr(cond), _ptr(uncond), _ptr(out), _stream()))
    return out


# ---------------------------------------------------------------- component entry points
def op_linear(dtype: int, epilogue: int, A, W, bias, out, gate=None, M=None, N=None, K=None, lda=None, ldo=None):
    M = A.shape[0] if M is None else M
    K = W.shape[1] if K is None else K
    N = W.shape[0] if N is None else N
    lda = A.stride(0) if lda is None else lda
    ldo = out.stride(0) if ldo is None else ldo
    _check(lib().track_op_linear(dtype, epilogue, M, N, K, _ptr(A), lda, _ptr(W), _ptr(bias), _ptr(gate), _ptr(out),
                                 ldo, _stream()))


def op_linear_vt(A, W, bias, L: int, vt, ldv: int, dtype: int = DTYPE_BF16):
    """A W^T + bias written transposed per batch of L rows into vt (the V^T layout of op_attention)."""
    M, K = A.shape
    N = W.shape[0]
    _check(lib().track_op_linear_vt(dtype, M, N, K, _ptr(A), A.stride(0), _ptr(W), _ptr(bias), L, _ptr(vt), ldv,
                                    _stream()))


def op_attention(dtype: int, B: int, H: int, head_dim: int, Lq: int, Lk: int, q, ldq: int, k, ldk: int, vt, ldv: int,
                 out, ldo: int, q_log2: bool = False):
    """q_log2: q is given times log2(e) / sqrt(head_dim) (track_op_attention_log2q)."""
    fn = lib().track_op_attention_log2q if q_log2 else lib().track_op_attention
    _check(fn(dtype, B, H, head_dim, Lq, Lk, _ptr(q), ldq, _ptr(k), ldk, _ptr(vt), ldv, _ptr(out), ldo, _stream()))


def op_layernorm(dtype: int, x, y, scale=None, shift=None):
    rows, d = x.shape
    _check(lib().track_op_layernorm(dtype, rows, d, _ptr(x), _ptr(scale), _ptr(shift), _ptr(y), _stream()))


def op_rmsnorm_rope(dtype: int, buf, heads: int, head_dim: int, g, col0: int = 0, grid=None, rows=None, ld=None):
    torch = _torch()
    rows = buf.shape[0] if rows is None else rows
    ld = buf.stride(0) if ld is None else ld
    ws = None
    gp = None
    if grid is not None:
        gp = (_i32 * 3)(*grid)
        n = lib().track_rope_table_len(head_dim, gp)
        ws = torch.empty(2 * n, dtype=torch.float32, device=buf.device)
    _check(lib().track_op_rmsnorm_rope(dtype, rows, heads, head_dim, _ptr(buf), ld, col0, _ptr(g), gp, _ptr(ws),
                                       _stream()))


def op_rmsnorm_rope_qk(dtype: int, buf, heads: int, head_dim: int, g_q, g_k, col0: int = 0, grid=None, rows=None,
                       ld=None):
    """op_rmsnorm_rope on the two adjacent segments (q with g_q, then k with g_k) of every row, one launch."""
    torch = _torch()
    rows = buf.shape[0] if rows is None else rows
    ld = buf.stride(0) if ld is None else ld
    ws = None
    gp = None
    if grid is not None:
        gp = (_i32 * 3)(*grid)
        n = lib().track_rope_table_len(head_dim, gp)
        ws = torch.empty(2 * n, dtype=torch.float32, device=buf.device)
    _check(lib().track_op_rmsnorm_rope_qk(dtype, rows, heads, head_dim, _ptr(buf), ld, col0, _ptr(g_q), _ptr(g_k), gp,
                                          _ptr(ws), _stream()))


def step_partial_count(n: int) -> int:
    return lib().track_step_partial_count(n)


def op_step(n: int, B: int, guidance: float, dsigma: float, vel_L, x, vel_S=None, partial=None, eps: float = 1e-8,
            r_out=None):
    _check(lib().track_op_step(n, B, float(guidance), float(dsigma), _ptr(vel_L), _ptr(vel_S), _ptr(x),
                               _ptr(partial), float(eps), _ptr(r_out), _stream()))


def op_step_noalloc(n: int, B: int, guidance: float, dsigma: float, vel_L, x, vel_S=None, eps: float = 1e-8,
                    r_out=None):
    """op_step with the calibration partials in the library's static device scratch (allocates nothing)."""
    _check(lib().track_op_step_noalloc(n, B, float(guidance), float(dsigma), _ptr(vel_L), _ptr(vel_S), _ptr(x),
                                       float(eps), _ptr(r_out), _stream()))


def unipc_coefficients(N: int, shift: float, order: int, step: int) -> np.ndarray:
    """The 12 weights of step `step` of the fused UniPC update (see include/track.h)."""
    out = np.zeros(12, dtype=np.float64)
    _check(lib().track_unipc_coefficients(int(N), float(shift), int(order), int(step),
                                          out.ctypes.data_as(ctypes.POINTER(_f64))))
    return out


def op_unipc_step(n: int, B: int, guidance: float, sigma: float, coef, vel_L, x, x_last, m_out, h0=None, h1=None,
                  h2=None, vel_S=None, partial=None, eps: float = 1e-8, r_out=None):
    coef = np.ascontiguousarray(coef, dtype=np.float64)
    _check(lib().track_op_unipc_step(int(n), int(B), float(guidance), float(sigma),
                                     coef.ctypes.data_as(ctypes.POINTER(_f64)), _ptr(vel_L), _ptr(vel_S), _ptr(x),
                                     _ptr(x_last), _ptr(h0), _ptr(h1), _ptr(h2), _ptr(m_out), _ptr(partial),
                                     float(eps), _ptr(r_out), _stream()))


def band_workspace_bytes(shape: synth.LatentShape, patch=(1, 2, 2)) -> int:
    return int(lib().track_band_workspace_bytes(ctypes.byref(shape_c(shape)), *patch))


def op_band_energy(shape: synth.LatentShape, B: int, guidance: float, vel_L, vel_S, workspace, patch=(1, 2, 2)):
    """Six band energies of the guided difference of two token-layout velocity buffers (synchronous)."""
    out = np.zeros(6, dtype=np.float64)
    nbytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().track_op_band_energy(ctypes.byref(shape_c(shape)), *patch, int(B), float(guidance), _ptr(vel_L),
                                      _ptr(vel_S), _ptr(workspace), nbytes, out.ctypes.data_as(ctypes.POINTER(_f64)),
                                      _stream()))
    return out


def set_progress(fn=None):
    """Call fn(sample, step, steps) after each completed step of calibrate/sample (None: off)."""
    global _progress_ref
    if fn is None:
        _check(lib().track_set_progress(PROGRESS_FN(), None))
        _progress_ref = None
        return
    cb = PROGRESS_FN(lambda user, j, k, n: fn(j, k, n))
    _check(lib().track_set_progress(cb, None))
    _progress_ref = cb


HBM_COPY, HBM_READ, HBM_WRITE = 0, 1, 2


def hbm_stream(kind: int, src, dst, nbytes: int):
    """Plain copy / read / write stream over nbytes (the HBM reference kernels)."""
    _check(lib().track_hbm_stream(int(kind), _ptr(src), _ptr(dst), int(nbytes), _stream()))


def mfma_stream(operands, iters: int, sink) -> int:
    """Independent bf16 MFMA chains on every CU from 64 KiB of operands (the
    sustained matrix-core reference); returns the launch's FLOP count."""
    flop = ctypes.c_int64(0)
    _check(lib().track_mfma_stream(_ptr(operands), int(iters), _ptr(sink), ctypes.byref(flop), _stream()))
    return int(flop.value)


# ---------------------------------------------------------------- profiling
def profile_enable(kinds=(PROF_ATTN_SELF, PROF_ATTN_CROSS, PROF_GEMM, PROF_NORM, PROF_STEP, PROF_OTHER)):
    """Bracket launches of the given kernel classes with HIP events (empty: off)."""
    mask = 0
    for k in kinds:
        mask |= 1 << k
    _check(lib().track_profile_enable(mask))


def profile_reset():
    _check(lib().track_profile_reset())


def profile_read(kind: int) -> Tuple[int, float]:
    n = _i64()
    ms = _f64()
    _check(lib().track_profile_read(kind, ctypes.byref(n), ctypes.byref(ms)))
    return n.value, ms.value
