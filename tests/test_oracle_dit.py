"""Pin of the oracle denoiser's composition against an independent torch.nn.functional build.

The paper does not define the denoiser network; the block layout is a reading
of the Wan 2.1 design.  This test restates that reading with library routines
(conv3d patch embedding, layer_norm, rms_norm, scaled_dot_product_attention,
complex-multiplication RoPE, einops for unpatchify) in float64 and requires the
oracle to match it, so an index, transpose or sign slip in the oracle's own
plumbing fails here.
"""
import dataclasses

import numpy as np
import torch
import torch.nn.functional as F
from einops import rearrange

from oracle import dit
from paper_2609_30096_amd import synth


def _torch_forward(params, cfg, x, t, ctx):
    P = {k: torch.from_numpy(np.asarray(v, np.float64)) for k, v in params.items()}
    d, H, dh = cfg.dim, cfg.heads, cfg.head_dim
    pt, ph, pw = cfg.patch
    xt = torch.from_numpy(np.asarray(x, np.float64))
    C, Fr, Hh, Ww = xt.shape
    g = (Fr // pt, Hh // ph, Ww // pw)
    wconv = P["patch.w"].reshape(d, C, pt, ph, pw)
    X = F.conv3d(xt[None], wconv, P["patch.b"], stride=cfg.patch)[0]          # [d, f, h, w]
    X = rearrange(X, "d f h w -> (f h w) d")
    L = X.shape[0]

    half = cfg.freq_dim // 2
    freqs = torch.pow(torch.tensor(10000.0, dtype=torch.float64), -torch.arange(half, dtype=torch.float64) / half)
    ang = t * freqs
    s = torch.cat([torch.cos(ang), torch.sin(ang)])
    e = F.linear(F.silu(F.linear(s, P["time.w1"], P["time.b1"])), P["time.w2"], P["time.b2"])
    m = F.linear(F.silu(e), P["mod.w"], P["mod.b"]).reshape(6, d)
    ctx_t = torch.from_numpy(np.asarray(ctx, np.float64))
    Cemb = F.linear(F.gelu(F.linear(ctx_t, P["text.w1"], P["text.b1"]), approximate="tanh"),
                    P["text.w2"], P["text.b2"])

    # rotary phases per token and per pair, as complex numbers
    df = dh - 4 * (dh // 6)
    dsec = 2 * (dh // 6)
    pos = torch.stack(torch.meshgrid(*[torch.arange(n, dtype=torch.float64) for n in g], indexing="ij"), -1).reshape(-1, 3)
    phase = []
    for axis, n in enumerate((df, dsec, dsec)):
        inv = 1.0 / torch.pow(torch.tensor(10000.0, dtype=torch.float64), torch.arange(0, n, 2, dtype=torch.float64) / n)
        phase.append(torch.outer(pos[:, axis], inv))
    rot = torch.polar(torch.ones(L, dh // 2, dtype=torch.float64), torch.cat(phase, 1))   # [L, dh/2]

    def rope(z):  # z [L, H, dh]
        zc = torch.view_as_complex(z.reshape(L, H, dh // 2, 2).contiguous())
        return torch.view_as_real(zc * rot[:, None, :]).reshape(L, H, dh)

    def attn(q, k, v):  # [Lq, H, dh]
        o = F.scaled_dot_product_attention(q.permute(1, 0, 2), k.permute(1, 0, 2), v.permute(1, 0, 2))
        return o.permute(1, 0, 2).reshape(q.shape[0], -1)

    ln = lambda z: F.layer_norm(z, (d,), eps=1e-6)
    for b in range(cfg.blocks):
        p = f"blk{b}."
        mod = m + P[p + "mod"]
        Y = ln(X) * (1 + mod[1]) + mod[0]
        Wq, Wk, Wv = P[p + "qkv.w"].split(d)
        bq, bk, bv = P[p + "qkv.b"].split(d)
        q = F.rms_norm(F.linear(Y, Wq, bq), (d,), P[p + "norm_q"], eps=1e-6).reshape(L, H, dh)
        k = F.rms_norm(F.linear(Y, Wk, bk), (d,), P[p + "norm_k"], eps=1e-6).reshape(L, H, dh)
        v = F.linear(Y, Wv, bv).reshape(L, H, dh)
        X = X + mod[2] * F.linear(attn(rope(q), rope(k), v), P[p + "o.w"], P[p + "o.b"])
        Y = ln(X)
        q = F.rms_norm(F.linear(Y, P[p + "cq.w"], P[p + "cq.b"]), (d,), P[p + "norm_cq"], eps=1e-6)
        Wck, Wcv = P[p + "ckv.w"].split(d)
        bck, bcv = P[p + "ckv.b"].split(d)
        k = F.rms_norm(F.linear(Cemb, Wck, bck), (d,), P[p + "norm_ck"], eps=1e-6)
        v = F.linear(Cemb, Wcv, bcv)
        Lc = Cemb.shape[0]
        X = X + F.linear(attn(q.reshape(L, H, dh), k.reshape(Lc, H, dh), v.reshape(Lc, H, dh)),
                         P[p + "co.w"], P[p + "co.b"])
        Y = ln(X) * (1 + mod[4]) + mod[3]
        X = X + mod[5] * F.linear(F.gelu(F.linear(Y, P[p + "ffn1.w"], P[p + "ffn1.b"]), approximate="tanh"),
                                  P[p + "ffn2.w"], P[p + "ffn2.b"])
    hm = P["head.mod"] + e
    out = F.linear(ln(X) * (1 + hm[1]) + hm[0], P["head.w"], P["head.b"])
    out = rearrange(out, "(f h w) (c a b q) -> c (f a) (h b) (w q)", f=g[0], h=g[1], w=g[2],
                    c=C, a=pt, b=ph, q=pw)
    return out.numpy()


def _tiny(**kw):
    return dataclasses.replace(synth.TINY_LARGE, **kw)


def test_dit_forward_matches_torch_build():
    cfg = _tiny(blocks=2)
    params = synth.gen_params(cfg, 7)
    shape = synth.TINY_LATENT
    x = synth.gen_latent(shape, 0)
    ctx = synth.gen_text(shape, cfg.text_dim, 0)
    t = 954.5454545
    out = dit.dit_forward(params, cfg, x, t, ctx)
    ref = _torch_forward(params, cfg, x, t, ctx)
    assert out.shape == x.shape
    rel = np.linalg.norm(out - ref) / np.linalg.norm(ref)
    assert rel < 1e-12, rel


def test_dit_forward_matches_torch_build_wan_head_dim():
    # head_dim 128 (the Wan sections 44/42/42) and a non-square grid
    cfg = _tiny(blocks=1, dim=256, heads=2, head_dim=128, ffn_dim=384, text_dim=64)
    params = synth.gen_params(cfg, 11)
    shape = synth.LatentShape(16, 3, 6, 10, 7)
    x = synth.gen_latent(shape, 1)
    ctx = synth.gen_text(shape, cfg.text_dim, 1)
    out = dit.dit_forward(params, cfg, x, 321.0, ctx)
    ref = _torch_forward(params, cfg, x, 321.0, ctx)
    rel = np.linalg.norm(out - ref) / np.linalg.norm(ref)
    assert rel < 1e-12, rel


def test_scaled_head_scales_output():
    # scaling the output projection (weight and bias) by (1 + a) scales f by (1 + a)
    cfg = _tiny(blocks=1)
    params = synth.gen_params(cfg, 3)
    scaled = dict(params)
    scaled["head.w"] = params["head.w"].astype(np.float64) * 1.25
    scaled["head.b"] = params["head.b"].astype(np.float64) * 1.25
    x = synth.gen_latent(synth.TINY_LATENT, 0)
    ctx = synth.gen_text(synth.TINY_LATENT, cfg.text_dim, 0)
    a = dit.dit_forward(params, cfg, x, 500.0, ctx)
    b = dit.dit_forward(scaled, cfg, x, 500.0, ctx)
    np.testing.assert_allclose(b, 1.25 * a, rtol=1e-12, atol=1e-15)


def test_q_chunk_does_not_change_result():
    cfg = _tiny(blocks=1)
    params = synth.gen_params(cfg, 3)
    x = synth.gen_latent(synth.TINY_LATENT, 2)
    ctx = synth.gen_text(synth.TINY_LATENT, cfg.text_dim, 2)
    np.testing.assert_allclose(dit.dit_forward(params, cfg, x, 10.0, ctx),
                               dit.dit_forward(params, cfg, x, 10.0, ctx, q_chunk=16), rtol=1e-13, atol=1e-15)
