"""Seeded synthetic inputs shared by the GPU path's callers and by the tests.

This module holds the workload recipe only: model shapes, the parameter list
(names, shapes, initial scales), the sampler settings, and a per-tensor keyed
random generator.  It contains none of the method's arithmetic; the denoiser,
guidance, scheduler, disagreement score and routing all live elsewhere.

Random numbers are drawn with numpy's PCG64, keyed per tensor as
``SeedSequence([seed, tensor_index, chunk])`` so that any one tensor (for
example a single transformer block at full width) can be regenerated without
drawing the rest.  Weights are ``N(0, 1) * scale`` in float32; a bfloat16
model uses the round-to-nearest-even bfloat16 values of those float32 draws.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

CHUNK = 1 << 22  # elements per independently keyed chunk of a tensor

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class DiTConfig:
    """Shape of a Wan-2.1-style video DiT denoiser."""
    blocks: int
    dim: int
    heads: int
    head_dim: int
    ffn_dim: int
    in_ch: int = 16
    patch: Tuple[int, int, int] = (1, 2, 2)
    text_dim: int = 4096
    freq_dim: int = 256
    dtype: str = BF16
    head_scale: float = 1.0  # extra factor on the output projection's weights

    @property
    def patch_elems(self) -> int:
        pt, ph, pw = self.patch
        return self.in_ch * pt * ph * pw

    def n_params(self) -> int:
        return sum(int(np.prod(s)) for _, s, _ in param_specs(self))


@dataclasses.dataclass(frozen=True)
class LatentShape:
    """Latent video C x F x H x W and the text context length."""
    channels: int
    frames: int
    height: int
    width: int
    text_len: int

    def tokens(self, patch) -> int:
        pt, ph, pw = patch
        return (self.frames // pt) * (self.height // ph) * (self.width // pw)

    @property
    def numel(self) -> int:
        return self.channels * self.frames * self.height * self.width


@dataclasses.dataclass(frozen=True)
class SamplerConfig:
    """Flow-matching sampler with classifier-free guidance.

    solver: "euler" (first-order step) or "unipc" (multistep predictor-corrector
    of the given order, 1 to 3) on the same shifted sigma table.
    """
    steps: int
    shift: float
    guidance: float
    use_cfg: bool = True
    eps: float = 1e-8
    solver: str = "euler"
    order: int = 2


# --------------------------------------------------------------------------
# Workload presets.  Sizes follow the Wan 2.1 family shapes the benchmarks use.
# --------------------------------------------------------------------------
TINY_LARGE = DiTConfig(blocks=4, dim=128, heads=4, head_dim=32, ffn_dim=512,
                       text_dim=128, dtype=F32, head_scale=0.1)
TINY_SMALL = dataclasses.replace(TINY_LARGE, blocks=2)
TINY_LATENT = LatentShape(16, 4, 8, 8, 16)
TINY_SAMPLER = SamplerConfig(steps=8, shift=3.0, guidance=5.0)

WAN_1_3B = DiTConfig(blocks=30, dim=1536, heads=12, head_dim=128, ffn_dim=8960)
WAN_14B = DiTConfig(blocks=40, dim=5120, heads=40, head_dim=128, ffn_dim=13824)
WAN_LATENT = LatentShape(16, 21, 60, 104, 512)      # 81 x 480 x 832 video
WAN_LATENT_LONG = LatentShape(16, 21, 90, 160, 512)  # 81 x 720 x 1280 video
WAN_SAMPLER = SamplerConfig(steps=50, shift=5.0, guidance=5.0)
DISTILLED_SAMPLER = SamplerConfig(steps=4, shift=5.0, guidance=1.0, use_cfg=False)
WAN_UNIPC_SAMPLER = SamplerConfig(steps=50, shift=5.0, guidance=5.0, solver="unipc", order=2)

# Seed scheme: model weights by model seed; per-sample tensors by a seed and
# a sample index.
SEED_LARGE = 1
SEED_SMALL = 2
SEED_LATENT = 100
SEED_COND = 200
SEED_UNCOND = 300
HELD_OUT = 999


def param_specs(cfg: DiTConfig) -> List[Tuple[str, Tuple[int, ...], float]]:
    """Ordered parameter list: (name, shape, init scale).

    Scale 0.0 marks a normalisation gain, initialised to ones.  Linear layers
    store their weight as [out_features, in_features].
    """
    d, f, P = cfg.dim, cfg.ffn_dim, cfg.patch_elems
    w = 0.02
    s: List[Tuple[str, Tuple[int, ...], float]] = [
        ("patch.w", (d, P), w), ("patch.b", (d,), w),
        ("time.w1", (d, cfg.freq_dim), w), ("time.b1", (d,), w),
        ("time.w2", (d, d), w), ("time.b2", (d,), w),
        ("mod.w", (6 * d, d), w), ("mod.b", (6 * d,), w),
        ("text.w1", (d, cfg.text_dim), w), ("text.b1", (d,), w),
        ("text.w2", (d, d), w), ("text.b2", (d,), w),
    ]
    for b in range(cfg.blocks):
        p = f"blk{b}."
        s += [
            (p + "mod", (6, d), w),
            (p + "qkv.w", (3 * d, d), w), (p + "qkv.b", (3 * d,), w),
            (p + "norm_q", (d,), 0.0), (p + "norm_k", (d,), 0.0),
            (p + "o.w", (d, d), w), (p + "o.b", (d,), w),
            (p + "cq.w", (d, d), w), (p + "cq.b", (d,), w),
            (p + "ckv.w", (2 * d, d), w), (p + "ckv.b", (2 * d,), w),
            (p + "norm_cq", (d,), 0.0), (p + "norm_ck", (d,), 0.0),
            (p + "co.w", (d, d), w), (p + "co.b", (d,), w),
            (p + "ffn1.w", (f, d), w), (p + "ffn1.b", (f,), w),
            (p + "ffn2.w", (d, f), w), (p + "ffn2.b", (d,), w),
        ]
    s += [("head.mod", (2, d), w), ("head.w", (P, d), w * cfg.head_scale),
          ("head.b", (P,), w)]
    return s


def _normal_f32(seed_key, n: int) -> np.ndarray:
    """n standard normals, drawn in independently keyed chunks."""
    out = np.empty(n, dtype=np.float32)
    for c0 in range(0, n, CHUNK):
        c1 = min(n, c0 + CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(seed_key) + [c0 // CHUNK])))
        out[c0:c1] = g.standard_normal(c1 - c0, dtype=np.float32)
    return out


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even); returns float32.

    Finite inputs only (the recipe draws no infinities or NaNs).
    """
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def gen_param(cfg: DiTConfig, model_seed: int, index: int, round_to_dtype: bool = True) -> np.ndarray:
    """Regenerate parameter ``index`` of ``param_specs(cfg)`` as float32."""
    name, shape, scale = param_specs(cfg)[index]
    n = int(np.prod(shape))
    if scale == 0.0:
        a = np.ones(n, dtype=np.float32)
    else:
        a = _normal_f32((model_seed, index), n) * np.float32(scale)
    a = a.reshape(shape)
    if round_to_dtype and cfg.dtype == BF16:
        a = bf16_round(a)
    return a


def gen_param_set(cfg: DiTConfig, model_seed: int, indices, pool, round_to_dtype: bool = True) -> Dict[str, np.ndarray]:
    """The parameters ``indices`` of ``param_specs(cfg)``, each equal to ``gen_param``'s, drawn chunk by chunk
    on the thread pool ``pool`` (an ``Executor``)."""
    specs = param_specs(cfg)
    out: Dict[str, np.ndarray] = {}
    jobs = []

    def fill(dst, key, c0, c1, scale):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(list(key) + [c0 // CHUNK])))
        g.standard_normal(c1 - c0, dtype=np.float32, out=dst[c0:c1])
        dst[c0:c1] *= np.float32(scale)
        if round_to_dtype and cfg.dtype == BF16:
            dst[c0:c1] = bf16_round(dst[c0:c1])

    for i in indices:
        name, shape, scale = specs[i]
        n = int(np.prod(shape))
        a = np.empty(n, dtype=np.float32)
        out[name] = a.reshape(shape)
        if scale == 0.0:
            a[:] = 1.0
            continue
        for c0 in range(0, n, CHUNK):
            jobs.append(pool.submit(fill, a, (model_seed, i), c0, min(n, c0 + CHUNK), scale))
    for j in jobs:
        j.result()
    return out


def gen_params(cfg: DiTConfig, model_seed: int, round_to_dtype: bool = True) -> Dict[str, np.ndarray]:
    """All parameters of a model as a name -> float32 array dict."""
    return {name: gen_param(cfg, model_seed, i, round_to_dtype)
            for i, (name, _, _) in enumerate(param_specs(cfg))}


def gen_latent(shape: LatentShape, sample: int) -> np.ndarray:
    """Initial noise x_T ~ N(0, 1), float32, C x F x H x W."""
    a = _normal_f32((SEED_LATENT, sample), shape.numel)
    return a.reshape(shape.channels, shape.frames, shape.height, shape.width)


def gen_text(shape: LatentShape, text_dim: int, sample: int, dtype: str = F32) -> np.ndarray:
    """Conditioning text embedding ~ N(0, 1), [text_len, text_dim] float32."""
    a = _normal_f32((SEED_COND, sample), shape.text_len * text_dim).reshape(shape.text_len, text_dim)
    return bf16_round(a) if dtype == BF16 else a


def gen_null_text(shape: LatentShape, text_dim: int, dtype: str = F32) -> np.ndarray:
    """Null (negative-prompt) embedding ~ N(0, 1), shared by every sample."""
    a = _normal_f32((SEED_UNCOND,), shape.text_len * text_dim).reshape(shape.text_len, text_dim)
    return bf16_round(a) if dtype == BF16 else a


def gen_normal(key, shape, scale: float = 1.0) -> np.ndarray:
    """Generic keyed N(0, scale^2) float32 tensor (for kernel-level tests)."""
    n = int(np.prod(shape))
    return (_normal_f32(tuple(key), n) * np.float32(scale)).reshape(shape)
