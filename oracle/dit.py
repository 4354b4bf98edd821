"""Oracle video DiT denoiser f_m(x_t, t, c), float64, numpy.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper treats each denoiser as a black box f_m(x_t, t, c) with
x_t in R^{C x F x H x W} (Preliminaries, "Video diffusion sampling") and
requires the large and small models of a pair to share latent, output shape,
conditioning and prediction target ("Compatible model pairs").  It does not
define the network.  This file states the network the benchmarks run: a
Wan-2.1-style DiT, written from that published design:

  tokens   : non-overlapping (pt, ph, pw) patches of x, token order (f, h, w),
             entries ordered (c, i_t, i_h, i_w); X = U Wp^T + bp
  time     : s = [cos(t w_j), sin(t w_j)], w_j = 10000^(-j/128);
             e = W2 silu(W1 s + b1) + b2;  m = Wm silu(e) + bm in R^{6 x d}
  text     : C = W2 gelu(W1 ctx + b1) + b2
  block    : (sh1, sc1, g1, sh2, sc2, g2) = m + T_b
             X += g1 * SelfAttn(LN(X)(1 + sc1) + sh1)
             X += CrossAttn(LN(X), C)
             X += g2 * MLP(LN(X)(1 + sc2) + sh2)
  head     : (sh, sc) = T_h + e;  out = (LN(X)(1 + sc) + sh) Wh^T + bh
  self-attn: q, k = RMSNorm over d of the projections, then 3D RoPE per head
  cross    : q = RMSNorm(Y Wq^T + b), k = RMSNorm(C Wk^T + b), v = C Wv^T + b

LN has no affine and eps 1e-6; RMSNorm has eps 1e-6 and a gain; GELU is the
tanh form.  Every array is float64.  Parameters come as a name -> array dict
whose names and shapes are the recipe's parameter list.
"""
from __future__ import annotations

import numpy as np

LN_EPS = 1e-6
RMS_EPS = 1e-6
ROPE_THETA = 10000.0
FREQ_THETA = 10000.0


# ---------------------------------------------------------------- sub-operations
def layer_norm(x):
    """(x - mean) / sqrt(var + eps) over the last axis; biased variance, no affine."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + LN_EPS)


def rms_norm(x, g):
    """x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt((x * x).mean(axis=-1, keepdims=True) + RMS_EPS) * g


def gelu_tanh(x):
    """0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))."""
    return 0.5 * x * (1.0 + np.tanh(np.sqrt(2.0 / np.pi) * (x + 0.044715 * x ** 3)))


def silu(x):
    """x * sigmoid(x)."""
    return x / (1.0 + np.exp(-x))


def linear(x, w, b):
    """x W^T + b, with W stored [out, in]."""
    return x @ np.asarray(w, np.float64).T + np.asarray(b, np.float64)


def sinusoid(t, dim=256):
    """Timestep features [cos(t w_j) for j < dim/2] ++ [sin(t w_j)], w_j = 10000^(-j/(dim/2))."""
    half = dim // 2
    w = FREQ_THETA ** (-np.arange(half, dtype=np.float64) / half)
    a = float(t) * w
    return np.concatenate([np.cos(a), np.sin(a)])


def rope_sections(head_dim):
    """Widths of the (frame, height, width) rotary sections of one head."""
    ds = 2 * (head_dim // 6)
    return head_dim - 2 * ds, ds, ds


def rope_angles(pos, n):
    """Angles pos * theta^(-2i/n) for the n/2 pairs of a section of width n; [len(pos), n/2]."""
    i = np.arange(n // 2, dtype=np.float64)
    return np.asarray(pos, np.float64)[:, None] * ROPE_THETA ** (-2.0 * i / n)[None, :]


def token_grid(frames, height, width):
    """(f, h, w) position of every token in token order (f-major, then h, then w)."""
    f, h, w = np.meshgrid(np.arange(frames), np.arange(height), np.arange(width), indexing="ij")
    return f.reshape(-1), h.reshape(-1), w.reshape(-1)


def rope3d(x, grid):
    """Rotate pairs (x[2i], x[2i+1]) of each head by the angle of its section's axis.

    x: [L, heads, head_dim]; grid: (frames, height, width) of the token grid.
    Pair i of the frame section turns by f * theta^(-2i/n_f), of the height
    section by h * theta^(-2i/n_h), of the width section by w * theta^(-2i/n_w).
    """
    L, H, dh = x.shape
    pos = token_grid(*grid)
    out = np.empty_like(x)
    start = 0
    for axis, n in enumerate(rope_sections(dh)):
        ang = rope_angles(pos[axis], n)                 # [L, n/2]
        c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
        a = x[:, :, start:start + n:2]
        b = x[:, :, start + 1:start + n:2]
        out[:, :, start:start + n:2] = a * c - b * s
        out[:, :, start + 1:start + n:2] = a * s + b * c
        start += n
    return out


def attention(q, k, v, q_chunk=None):
    """softmax(q k^T / sqrt(head_dim)) v per head; q: [Lq, H, dh], k, v: [Lk, H, dh].

    Query rows are independent, so q_chunk only bounds memory; it does not
    change any row's arithmetic.
    """
    Lq, H, dh = q.shape
    out = np.empty((Lq, H, v.shape[2]), dtype=np.float64)
    step = Lq if q_chunk is None else q_chunk
    scale = 1.0 / np.sqrt(dh)
    for h in range(H):
        kh, vh = k[:, h, :], v[:, h, :]
        for r0 in range(0, Lq, step):
            s = (q[r0:r0 + step, h, :] @ kh.T) * scale
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[r0:r0 + step, h, :] = p @ vh
    return out


def patchify(x, patch):
    """C x F x H x W -> [L, C*pt*ph*pw]; token (f, h, w) f-major, entry (c, i_t, i_h, i_w)."""
    C, F, H, W = x.shape
    pt, ph, pw = patch
    y = x.reshape(C, F // pt, pt, H // ph, ph, W // pw, pw)
    y = y.transpose(1, 3, 5, 0, 2, 4, 6)
    return y.reshape((F // pt) * (H // ph) * (W // pw), C * pt * ph * pw)


def unpatchify(u, channels, frames, height, width, patch):
    """Inverse of patchify."""
    pt, ph, pw = patch
    y = u.reshape(frames // pt, height // ph, width // pw, channels, pt, ph, pw)
    y = y.transpose(3, 0, 4, 1, 5, 2, 6)
    return y.reshape(channels, frames, height, width)


# ---------------------------------------------------------------- the network
def _p(params, name):
    return np.asarray(params[name], dtype=np.float64)


def time_embedding(params, cfg, t):
    """e (time embedding, [d]) and m (shared modulation, [6, d]) for timestep t."""
    s = sinusoid(t, cfg.freq_dim)
    e = linear(silu(linear(s, _p(params, "time.w1"), _p(params, "time.b1"))),
               _p(params, "time.w2"), _p(params, "time.b2"))
    m = linear(silu(e), _p(params, "mod.w"), _p(params, "mod.b"))
    return e, m.reshape(6, cfg.dim)


def text_embedding(params, ctx):
    """C = W2 gelu(W1 ctx + b1) + b2; ctx: [Lc, text_dim]."""
    h = gelu_tanh(linear(np.asarray(ctx, np.float64), _p(params, "text.w1"), _p(params, "text.b1")))
    return linear(h, _p(params, "text.w2"), _p(params, "text.b2"))


def block(params, cfg, b, X, ctx_emb, m, grid, q_chunk=None):
    """One transformer block applied to X [L, d] with text embedding ctx_emb [Lc, d]."""
    d, H, dh = cfg.dim, cfg.heads, cfg.head_dim
    p = f"blk{b}."
    sh1, sc1, g1, sh2, sc2, g2 = m + _p(params, p + "mod")
    L = X.shape[0]

    # self-attention sub-block
    Y = layer_norm(X) * (1.0 + sc1) + sh1
    qkv = linear(Y, _p(params, p + "qkv.w"), _p(params, p + "qkv.b"))
    q = rms_norm(qkv[:, :d], _p(params, p + "norm_q"))
    k = rms_norm(qkv[:, d:2 * d], _p(params, p + "norm_k"))
    v = qkv[:, 2 * d:]
    q = rope3d(q.reshape(L, H, dh), grid)
    k = rope3d(k.reshape(L, H, dh), grid)
    a = attention(q, k, v.reshape(L, H, dh), q_chunk).reshape(L, d)
    X = X + g1 * linear(a, _p(params, p + "o.w"), _p(params, p + "o.b"))

    # cross-attention sub-block (no modulation, no RoPE)
    Y = layer_norm(X)
    qc = rms_norm(linear(Y, _p(params, p + "cq.w"), _p(params, p + "cq.b")), _p(params, p + "norm_cq"))
    kv = linear(ctx_emb, _p(params, p + "ckv.w"), _p(params, p + "ckv.b"))
    kc = rms_norm(kv[:, :d], _p(params, p + "norm_ck"))
    vc = kv[:, d:]
    Lc = ctx_emb.shape[0]
    a = attention(qc.reshape(L, H, dh), kc.reshape(Lc, H, dh), vc.reshape(Lc, H, dh), q_chunk).reshape(L, d)
    X = X + linear(a, _p(params, p + "co.w"), _p(params, p + "co.b"))

    # MLP sub-block
    Y = layer_norm(X) * (1.0 + sc2) + sh2
    h = gelu_tanh(linear(Y, _p(params, p + "ffn1.w"), _p(params, p + "ffn1.b")))
    X = X + g2 * linear(h, _p(params, p + "ffn2.w"), _p(params, p + "ffn2.b"))
    return X


def head(params, X, e):
    """Modulated output projection: (LN(X)(1 + sc) + sh) Wh^T + bh."""
    sh, sc = _p(params, "head.mod") + e
    return linear(layer_norm(X) * (1.0 + sc) + sh, _p(params, "head.w"), _p(params, "head.b"))


def dit_forward(params, cfg, x, t, ctx, q_chunk=None):
    """Denoiser output f(x, t, ctx) in R^{C x F x H x W}.

    x: latent [C, F, H, W]; t: model timestep (scalar); ctx: text embedding
    [Lc, text_dim].
    """
    x = np.asarray(x, np.float64)
    C, F, H, W = x.shape
    pt, ph, pw = cfg.patch
    grid = (F // pt, H // ph, W // pw)
    X = linear(patchify(x, cfg.patch), _p(params, "patch.w"), _p(params, "patch.b"))
    e, m = time_embedding(params, cfg, t)
    ctx_emb = text_embedding(params, ctx)
    for b in range(cfg.blocks):
        X = block(params, cfg, b, X, ctx_emb, m, grid, q_chunk)
    return unpatchify(head(params, X, e), C, F, H, W, cfg.patch)
