"""Helpers shared by the GPU parity tests: seeded inputs on host and device,
error metrics, and the float64 oracle calls they are compared against."""
import sys

import numpy as np

from paper_2609_30096_amd import synth


def say(msg):
    """Print and flush, so a failing GPU step names its case."""
    print(msg, flush=True)
    sys.stdout.flush()


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def normal(key, shape, scale=1.0, bf16=False):
    a = synth.gen_normal(key, shape, scale)
    return synth.bf16_round(a) if bf16 else a


def dev(a, dtype="f32"):
    """numpy float32 -> device tensor of float32 or bfloat16 (exact for bf16-rounded input)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()
    return t.to(torch.bfloat16) if dtype == synth.BF16 else t


def host(t):
    import torch
    return t.float().cpu().numpy() if t.dtype != torch.float32 else t.cpu().numpy()


def vt_layout(v, B, L, H, dh, ldv):
    """[B*L, H*dh] -> transposed [B, H, dh, ldv] with zeros past L (float32 numpy)."""
    out = np.zeros((B, H, dh, ldv), np.float32)
    vv = v.reshape(B, L, H, dh)
    out[..., :L] = vv.transpose(0, 2, 3, 1)
    return out
