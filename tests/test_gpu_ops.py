"""GPU parity of each kernel against the float64 oracle, through the C ABI.

Small cases span several tiles with ragged tails; the full-size cases run the
Wan-2.1-1.3B step's shapes (65520 token rows, the launch configuration of the
benchmark) and check sampled outputs that the oracle computes one by one.
"""
import numpy as np
import pytest

from gpu_helpers import dev, host, normal, rel_l2, say, vt_layout
from oracle import dit, sampler
from paper_2609_30096_amd import synth, track

pytestmark = pytest.mark.gpu

F32, BF16 = synth.F32, synth.BF16
EPIS = [track.EPI_BIAS, track.EPI_BIAS_GELU, track.EPI_GATE_RESID, track.EPI_RESID, track.EPI_BIAS_F32]


@pytest.fixture(autouse=True)
def _free():
    yield
    import torch
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


def _linear_ref(epi, A, W, b, gate, resid):
    y = dit.linear(A, W, b)
    if epi == track.EPI_BIAS_GELU:
        return dit.gelu_tanh(y)
    if epi == track.EPI_GATE_RESID:
        return resid + gate * y
    if epi == track.EPI_RESID:
        return resid + y
    return y


def _run_linear(dtype, epi, A, W, b, gate, resid):
    import torch
    dc = track.dtype_code(dtype)
    M, N = A.shape[0], W.shape[0]
    tA, tW, tb = dev(A, dtype), dev(W, dtype), dev(b, dtype)
    tg = dev(gate) if gate is not None else None
    if epi in (track.EPI_GATE_RESID, track.EPI_RESID):
        out = dev(resid)
    elif epi == track.EPI_BIAS_F32:
        out = torch.empty(M, N, dtype=torch.float32, device="cuda")
    else:
        out = torch.empty(M, N, dtype=track.torch_dtype(dtype), device="cuda")
    track.op_linear(dc, epi, tA, tW, tb, out, gate=tg)
    return host(out)


@pytest.mark.parametrize("dtype", [F32, BF16])
@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("M,N,K", [(300, 256, 192), (1000, 384, 512), (77, 64, 64), (513, 768, 256)])
def test_linear_small(dtype, epi, M, N, K):
    say(f"linear dtype={dtype} epi={epi} M={M} N={N} K={K}")
    bf = dtype == BF16
    A = normal((5000, M, K), (M, K), 1.0, bf)
    W = normal((5001, N, K), (N, K), 0.05, bf)
    b = normal((5002, N), (N,), 0.1, bf)
    gate = normal((5003, N), (N,), 1.0)
    resid = normal((5004, M, N), (M, N), 1.0)
    got = _run_linear(dtype, epi, A, W, b, gate, resid)
    ref = _linear_ref(epi, A, W, b, gate, resid)
    if dtype == F32 or epi in (track.EPI_GATE_RESID, track.EPI_RESID, track.EPI_BIAS_F32):
        tol = 2e-6 if dtype == F32 else 1e-5
    else:
        tol = 4e-3  # bf16 output rounding
    assert rel_l2(got, ref) < tol, rel_l2(got, ref)
    np.testing.assert_allclose(got, ref, rtol=0, atol=8 * tol * (np.abs(ref).max() + 1))


def test_linear_rejects_bad_shapes():
    import torch
    A = torch.zeros(10, 60, dtype=torch.bfloat16, device="cuda")
    W = torch.zeros(64, 60, dtype=torch.bfloat16, device="cuda")
    b = torch.zeros(64, dtype=torch.bfloat16, device="cuda")
    out = torch.zeros(10, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(track.TrackError) as e:
        track.op_linear(track.DTYPE_BF16, track.EPI_BIAS, A, W, b, out)
    assert e.value.status == track.E_UNSUPPORTED
    with pytest.raises(track.TrackError):
        track.op_linear(track.DTYPE_BF16, track.EPI_GATE_RESID, A, W, b, out)  # gate missing


def _q_log2(q, dh, q_log2):
    """(q the kernel takes, q the reference takes).  With q_log2 the kernel takes
    q' = bf16(q log2(e) / sqrt(dh)) (track_op_attention_log2q) and the reference
    q' sqrt(dh) / log2(e) in float64, the exact query that q' stands for."""
    if not q_log2:
        return q, q.astype(np.float64)
    c = np.log2(np.e) / np.sqrt(dh)
    qk = synth.bf16_round((q.astype(np.float64) * c).astype(np.float32))
    return qk, qk.astype(np.float64) / c


def _attn_case(dtype, B, H, dh, Lq, Lk, key, scale=1.0, ldv=None, q_log2=False):
    import torch
    bf = dtype == BF16
    q = normal((key, 1), (B * Lq, H * dh), scale, bf)
    k = normal((key, 2), (B * Lk, H * dh), scale, bf)
    v = normal((key, 3), (B * Lk, H * dh), 1.0, bf)
    q, qr = _q_log2(q, dh, q_log2)
    ldv = (Lk + 63) // 64 * 64 if ldv is None else ldv
    vt = vt_layout(v, B, Lk, H, dh, ldv)
    out = torch.empty(B * Lq, H * dh, dtype=track.torch_dtype(dtype), device="cuda")
    track.op_attention(track.dtype_code(dtype), B, H, dh, Lq, Lk, dev(q, dtype), H * dh, dev(k, dtype), H * dh,
                       dev(vt, dtype), ldv, out, H * dh, q_log2=q_log2)
    got = host(out).reshape(B, Lq, H, dh)
    ref = np.stack([dit.attention(qr.reshape(B, Lq, H, dh)[b],
                                  k.reshape(B, Lk, H, dh)[b].astype(np.float64),
                                  v.reshape(B, Lk, H, dh)[b].astype(np.float64)) for b in range(B)])
    return got, ref


@pytest.mark.parametrize("q_log2", [False, True])
@pytest.mark.parametrize("Lq,Lk", [(300, 300), (300, 77), (64, 64), (1, 5), (257, 1000), (700, 512),
                                   (130, 65), (130, 128), (33, 129), (33, 192)])
def test_attention_bf16(Lq, Lk, q_log2):
    say(f"attention bf16 Lq={Lq} Lk={Lk} q_log2={q_log2}")
    got, ref = _attn_case(BF16, 2, 2, 128, Lq, Lk, 6000 + Lq + Lk, q_log2=q_log2)
    assert rel_l2(got, ref) < 1e-2, rel_l2(got, ref)


@pytest.mark.parametrize("Lk,ldv", [(77, 80), (300, 304), (129, 136), (128, 128)])
def test_attention_bf16_tight_vt_rows(Lk, ldv):
    say(f"attention bf16 Lk={Lk} ldv={ldv}")
    got, ref = _attn_case(BF16, 1, 2, 128, 70, Lk, 6050 + Lk, ldv=ldv)
    assert rel_l2(got, ref) < 1e-2, rel_l2(got, ref)


@pytest.mark.parametrize("q_log2", [False, True])
def test_attention_bf16_large_logits(q_log2):
    say(f"attention bf16 large logits q_log2={q_log2}")
    got, ref = _attn_case(BF16, 1, 2, 128, 200, 333, 6100, scale=3.0, q_log2=q_log2)  # logits ~ N(0, 81)
    assert rel_l2(got, ref) < 2e-2, rel_l2(got, ref)
    assert np.isfinite(got).all()


@pytest.mark.parametrize("q_log2", [False, True])
@pytest.mark.parametrize("growth", [4.0, 60.0])
def test_attention_bf16_rising_logits(growth, q_log2):
    """Keys whose norms grow along the sequence.  With the larger growth the logits climb past several
    multiples of the 64 (log2 units) of headroom, so the reference max moves again and again, tile after
    tile, on both probability paths."""
    say(f"attention bf16 rising logits growth={growth} q_log2={q_log2}")
    import torch
    B, H, dh, Lq, Lk = 1, 2, 128, 150, 1100
    q = normal((6150, 1), (B * Lq, H * dh), 1.0, True)
    q, qr = _q_log2(q, dh, q_log2)
    ramp = (1.0 + growth * np.arange(Lk) / Lk)[:, None]
    k = synth.bf16_round(normal((6150, 2), (B * Lk, H * dh), 1.0, False) * ramp)
    v = normal((6150, 3), (B * Lk, H * dh), 1.0, True)
    ldv = (Lk + 63) // 64 * 64
    vt = vt_layout(v, B, Lk, H, dh, ldv)
    out = torch.empty(B * Lq, H * dh, dtype=torch.bfloat16, device="cuda")
    track.op_attention(track.DTYPE_BF16, B, H, dh, Lq, Lk, dev(q, BF16), H * dh, dev(k, BF16), H * dh,
                       dev(vt, BF16), ldv, out, H * dh, q_log2=q_log2)
    got = host(out).reshape(Lq, H, dh)
    ref = dit.attention(qr.reshape(Lq, H, dh), k.reshape(Lk, H, dh).astype(np.float64),
                        v.reshape(Lk, H, dh).astype(np.float64))
    assert rel_l2(got, ref) < 2e-2, rel_l2(got, ref)
    assert np.isfinite(got).all()


@pytest.mark.parametrize("q_log2", [False, True])
@pytest.mark.parametrize("Lk", [40, 300])
def test_attention_bf16_offset_logits(Lk, q_log2):
    """Every logit near -100 (head 0) or +100 (head 1): outside the window in which the reference max
    stays 0, on both sides."""
    say(f"attention bf16 offset logits Lk={Lk} q_log2={q_log2}")
    import torch
    B, H, dh, Lq = 1, 2, 128, 70
    a = normal((6160, 0), (1, dh), 1.0, False)
    q = np.concatenate([np.repeat(3.0 * a, Lq, 0)] * H, 1) + 0.3 * normal((6160, 1), (Lq, H * dh), 1.0, False)
    kd = normal((6160, 2), (Lk, H * dh), 0.3, False)
    k = np.concatenate([-3.0 * np.repeat(a, Lk, 0), 3.0 * np.repeat(a, Lk, 0)], 1) + kd
    q, k = synth.bf16_round(q), synth.bf16_round(k)
    q, qr = _q_log2(q, dh, q_log2)
    v = normal((6160, 3), (Lk, H * dh), 1.0, True)
    ldv = (Lk + 63) // 64 * 64
    vt = vt_layout(v, B, Lk, H, dh, ldv)
    out = torch.empty(Lq, H * dh, dtype=torch.bfloat16, device="cuda")
    track.op_attention(track.DTYPE_BF16, B, H, dh, Lq, Lk, dev(q, BF16), H * dh, dev(k, BF16), H * dh,
                       dev(vt, BF16), ldv, out, H * dh, q_log2=q_log2)
    got = host(out).reshape(Lq, H, dh)
    ref = dit.attention(qr.reshape(Lq, H, dh), k.reshape(Lk, H, dh).astype(np.float64),
                        v.reshape(Lk, H, dh).astype(np.float64))
    assert np.isfinite(got).all()
    assert rel_l2(got, ref) < 2e-2, rel_l2(got, ref)


@pytest.mark.parametrize("dh", [32, 64, 128])
@pytest.mark.parametrize("Lq,Lk", [(100, 100), (65, 16)])
def test_attention_f32(dh, Lq, Lk):
    say(f"attention f32 dh={dh} Lq={Lq} Lk={Lk}")
    got, ref = _attn_case(F32, 2, 3, dh, Lq, Lk, 6200 + dh + Lk)
    assert rel_l2(got, ref) < 1e-5, rel_l2(got, ref)


def test_attention_errors_and_empty():
    import torch
    z = torch.zeros(64, 128, dtype=torch.bfloat16, device="cuda")
    vt = torch.zeros(128, 64, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(track.TrackError):
        track.op_attention(track.DTYPE_BF16, 1, 1, 128, 64, 0, z, 128, z, 128, vt, 64, z, 128)
    with pytest.raises(track.TrackError):  # ldv not a multiple of 8
        track.op_attention(track.DTYPE_BF16, 1, 1, 128, 64, 36, z, 128, z, 128, vt, 36, z, 128)
    with pytest.raises(track.TrackError):  # ldv below Lk
        track.op_attention(track.DTYPE_BF16, 1, 1, 128, 64, 48, z, 128, z, 128, vt, 40, z, 128)
    with pytest.raises(track.TrackError):  # bf16 needs head_dim 128
        track.op_attention(track.DTYPE_BF16, 1, 2, 64, 64, 64, z, 128, z, 128, vt, 64, z, 128)
    track.op_attention(track.DTYPE_BF16, 1, 1, 128, 0, 64, z, 128, z, 128, vt, 64, z, 128)


@pytest.mark.parametrize("dtype,d", [(F32, 128), (BF16, 1536), (BF16, 5120), (F32, 260), (F32, 2052)])
@pytest.mark.parametrize("modulated", [True, False])
def test_layernorm(dtype, d, modulated):
    say(f"layernorm {dtype} d={d} mod={modulated}")
    import torch
    rows = 333
    x = normal((7000, d), (rows, d), 2.0) + 0.5
    sc = normal((7001, d), (d,), 0.3) if modulated else None
    sh = normal((7002, d), (d,), 0.3) if modulated else None
    y = torch.empty(rows, d, dtype=track.torch_dtype(dtype), device="cuda")
    track.op_layernorm(track.dtype_code(dtype), dev(x), y, dev(sc) if modulated else None,
                       dev(sh) if modulated else None)
    ref = dit.layer_norm(x.astype(np.float64))
    if modulated:
        ref = ref * (1 + sc) + sh
    tol = 1e-6 if dtype == F32 else 4e-3
    assert rel_l2(host(y), ref) < tol


# Widths above 2048 take the kernel that spreads two rows over a workgroup:
# 40 x 128 (the 14B width); 24 x 96 with B = 1 (ragged last chunk, angles
# looked up per chunk, an odd row count).
# bf16 rows move 8 elements at a time when head_dim % 8 == 0 (24 x 96: a ragged
# last chunk on the wide-row kernel), 4 otherwise (10 x 12).
@pytest.mark.parametrize("dtype,heads,dh,B", [(F32, 4, 32, 2), (BF16, 12, 128, 2), (F32, 2, 128, 2),
                                              (BF16, 40, 128, 2), (F32, 24, 96, 1), (BF16, 24, 96, 1),
                                              (BF16, 10, 12, 2)])
def test_rmsnorm_rope(dtype, heads, dh, B):
    say(f"rmsnorm_rope {dtype} heads={heads} dh={dh} B={B}")
    import torch
    grid = (3, 5, 7)
    L = 105
    d = heads * dh
    bf = dtype == BF16
    buf = normal((7100, d), (B * L, 3 * d), 1.5, bf)
    gq = normal((7101, d), (d,), 1.0, bf)
    gk = normal((7102, d), (d,), 1.0, bf)
    t = dev(buf, dtype)
    dc = track.dtype_code(dtype)
    track.op_rmsnorm_rope(dc, t, heads, dh, dev(gq, dtype), col0=0, grid=grid)
    track.op_rmsnorm_rope(dc, t, heads, dh, dev(gk, dtype), col0=d, grid=grid)
    track.op_rmsnorm_rope(dc, t, heads, dh, dev(gk, dtype), col0=2 * d, grid=None)
    got = host(t)
    b64 = buf.astype(np.float64)
    for bb in range(B):
        rows = slice(bb * L, (bb + 1) * L)
        rq = dit.rope3d(dit.rms_norm(b64[rows, :d], gq).reshape(L, heads, dh), grid).reshape(L, d)
        rk = dit.rope3d(dit.rms_norm(b64[rows, d:2 * d], gk).reshape(L, heads, dh), grid).reshape(L, d)
        rv = dit.rms_norm(b64[rows, 2 * d:], gk)
        tol = 1e-6 if dtype == F32 else 5e-3
        assert rel_l2(got[rows, :d], rq) < tol
        assert rel_l2(got[rows, d:2 * d], rk) < tol
        assert rel_l2(got[rows, 2 * d:], rv) < tol
    # the fused q/k launch the forward uses gives the same bits as the two single-segment launches
    t2 = dev(buf, dtype)
    track.op_rmsnorm_rope_qk(dc, t2, heads, dh, dev(gq, dtype), dev(gk, dtype), col0=0, grid=grid)
    track.op_rmsnorm_rope(dc, t2, heads, dh, dev(gk, dtype), col0=2 * d, grid=None)
    assert torch.equal(t2, t)


@pytest.mark.parametrize("B", [1, 2])
def test_step_sample_and_calibration_modes(B):
    say(f"step B={B}")
    import torch
    n = 32760 * 64
    vL = normal((7200, B), (B * n,), 1.0)
    vS = vL + normal((7201, B), (B * n,), 0.1)
    x0 = normal((7202,), (n,), 1.0)
    w, ds = 5.0, -0.0417
    tvL, tvS = dev(vL), dev(vS)
    xa, xb = dev(x0), dev(x0)
    nb = track.step_partial_count(n)
    part = torch.empty(2 * nb, dtype=torch.float64, device="cuda")
    r = torch.zeros(1, dtype=torch.float64, device="cuda")
    track.op_step(n, B, w, ds, tvL, xa)
    track.op_step(n, B, w, ds, tvL, xb, vel_S=tvS, partial=part, eps=1e-8, r_out=r)
    ga, gb = host(xa), host(xb)
    np.testing.assert_array_equal(ga, gb)  # same update in both modes
    c, u = vL[:n].astype(np.float64), vL[n:].astype(np.float64) if B == 2 else None
    pL = sampler.guided(c, u, w) if B == 2 else c
    cS, uS = vS[:n].astype(np.float64), vS[n:].astype(np.float64) if B == 2 else None
    pS = sampler.guided(cS, uS, w) if B == 2 else cS
    ref_x = sampler.euler_step(x0.astype(np.float64), pL, 0.0, np.float64(np.float32(ds)))
    assert np.max(np.abs(ga - ref_x)) < 1e-5
    ref_r = sampler.relative_disagreement(pS, pL, 1e-8)
    assert abs(r.item() - ref_r) < 1e-6 * ref_r


def test_step_self_disagreement_is_exactly_zero():
    import torch
    n = 4096
    v = dev(normal((7300,), (2 * n,), 1.0))
    x = dev(normal((7301,), (n,), 1.0))
    part = torch.empty(2 * track.step_partial_count(n), dtype=torch.float64, device="cuda")
    r = torch.ones(1, dtype=torch.float64, device="cuda")
    track.op_step(n, 2, 5.0, -0.1, v, x, vel_S=v, partial=part, eps=1e-8, r_out=r)
    assert r.item() == 0.0
    z = torch.zeros(2 * n, dtype=torch.float32, device="cuda")
    track.op_step(n, 2, 5.0, -0.1, z, x, vel_S=v, partial=part, eps=1e-8, r_out=r)
    assert r.item() > 1e6  # p_L = 0: the denominator is eps


@pytest.mark.parametrize("order,N,i,B", [(2, 50, 0, 2), (2, 50, 1, 2), (2, 50, 7, 2), (2, 50, 49, 2),
                                         (3, 50, 3, 2), (3, 50, 20, 1), (3, 8, 6, 2), (1, 4, 2, 1)])
def test_unipc_step_full_size_matches_oracle(order, N, i, B):
    """One fused UniPC step on the 16 x 21 x 60 x 104 latent (token layout) from
    seeded state, against the oracle's UniPC step from the same state."""
    from oracle import unipc
    import torch
    say(f"unipc step order={order} N={N} i={i} B={B}")
    n = 32760 * 64
    shift, w = 5.0, 5.0
    key = 7400 + 10 * order + i
    vL = normal((key, 1), (B * n,), 1.0)
    vS = vL + normal((key, 2), (B * n,), 0.1)
    x = normal((key, 3), (n,), 1.0)
    xl = normal((key, 4), (n,), 1.0)
    hs = [normal((key, 5 + k), (n,), 1.0) for k in range(3)]
    sig = sampler.sigmas(N, shift)
    coef = track.unipc_coefficients(N, shift, order, i)
    # oracle from the same state: reach step i's bookkeeping, then install the arrays
    S = unipc.UniPC(sig, order=order)
    for j in range(i):
        S.step(j, np.zeros(1), np.zeros(1))
    if i >= 1:
        S.x_last = xl.astype(np.float64)
        for k in range(1, 4):
            if i - k >= 0:
                S.m[i - k] = hs[k - 1].astype(np.float64)
    c = vL[:n].astype(np.float64)
    pL = sampler.guided(c, vL[n:].astype(np.float64), w) if B == 2 else c
    ref_next = S.step(i, x.astype(np.float64), pL)
    ref_xc = S.x_last
    ref_m = x.astype(np.float64) - np.float64(np.float32(sig[i])) * pL
    tx, txl, tm = dev(x), dev(xl), torch.empty(n, device="cuda")
    th = [dev(h) for h in hs]
    nb = track.step_partial_count(n)
    part = torch.empty(2 * nb, dtype=torch.float64, device="cuda")
    r = torch.zeros(1, dtype=torch.float64, device="cuda")
    track.op_unipc_step(n, B, w, float(np.float32(sig[i])), coef, dev(vL), tx, txl, tm, h0=th[0], h1=th[1], h2=th[2],
                        vel_S=dev(vS), partial=part, eps=1e-8, r_out=r)
    got_next, got_xc, got_m = host(tx), host(txl), host(tm)
    scale = max(1.0, float(np.abs(ref_next).max()))
    say(f"  max |dx_next| {np.abs(got_next - ref_next).max():.2e}, |dx_c| {np.abs(got_xc - ref_xc).max():.2e}")
    assert np.abs(got_m - ref_m).max() < 1e-5 * max(1.0, float(np.abs(ref_m).max()))
    assert np.abs(got_xc - ref_xc).max() < 2e-5 * max(1.0, float(np.abs(ref_xc).max()))
    assert np.abs(got_next - ref_next).max() < 2e-5 * scale
    cS = vS[:n].astype(np.float64)
    pS = sampler.guided(cS, vS[n:].astype(np.float64), w) if B == 2 else cS
    ref_r = sampler.relative_disagreement(pS, pL, 1e-8)
    assert abs(r.item() - ref_r) < 1e-6 * ref_r
    # sample mode (no small model) applies the same update
    tx2, txl2, tm2 = dev(x), dev(xl), torch.empty(n, device="cuda")
    track.op_unipc_step(n, B, w, float(np.float32(sig[i])), coef, dev(vL), tx2, txl2, tm2, h0=th[0], h1=th[1],
                        h2=th[2])
    np.testing.assert_array_equal(host(tx2), got_next)


def test_unipc_step_rejects_missing_history():
    import torch
    n = 1024
    v = torch.zeros(2 * n, device="cuda")
    x, xl, m = torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    coef = track.unipc_coefficients(50, 5.0, 2, 10)  # corrector and predictor read m_{i-1}, m_{i-2}
    with pytest.raises(track.TrackError):
        track.op_unipc_step(n, 2, 5.0, 0.5, coef, v, x, xl, m)


# ------------------------------------------------------------------ full-size sampled checks
def _tiled_rows(key, rows, cols, block, scale, bf):
    """Seeded [block, cols] tile repeated to `rows` rows: device tensor and the host tile."""
    import torch
    tile = normal(key, (block, cols), scale, bf)
    t = dev(tile, BF16 if bf else F32)
    reps = (rows + block - 1) // block
    full = t.repeat(reps, 1)[:rows].contiguous()
    return full, tile


@pytest.mark.parametrize("name,N,K,epi", [("qkv", 4608, 1536, track.EPI_BIAS),
                                          ("ffn1", 8960, 1536, track.EPI_BIAS_GELU),
                                          ("ffn2", 1536, 8960, track.EPI_GATE_RESID),
                                          ("head", 64, 1536, track.EPI_BIAS_F32)])
def test_linear_full_size_sampled(name, N, K, epi):
    say(f"linear full size {name} M=65520 N={N} K={K}")
    import torch
    M = 65520
    A, tileA = _tiled_rows((8000, K), M, K, 4093, 1.0, True)   # 4093: prime, not a tile multiple
    W = normal((8001, N, K), (N, K), 0.02, True)
    b = normal((8002, N), (N,), 0.02, True)
    gate = normal((8003, N), (N,), 1.0)
    tW, tb = dev(W, BF16), dev(b, BF16)
    resid_tile = None
    if epi == track.EPI_GATE_RESID:
        out, resid_tile = _tiled_rows((8004, N), M, N, 3001, 1.0, False)
    elif epi == track.EPI_BIAS_F32:
        out = torch.empty(M, N, dtype=torch.float32, device="cuda")
    else:
        out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    track.op_linear(track.DTYPE_BF16, epi, A, tW, tb, out, gate=dev(gate))
    rng = np.random.default_rng(1)
    rows = np.concatenate([rng.integers(0, M, 24), [0, M - 1, M - 240, M - 17]])
    got = host(out[torch.from_numpy(rows).cuda()])
    Ar = tileA[rows % 4093].astype(np.float64)
    resid = resid_tile[rows % 3001] if resid_tile is not None else None
    ref = _linear_ref(epi, Ar, W, b, gate, resid)
    tol = 1e-5 if epi in (track.EPI_GATE_RESID, track.EPI_BIAS_F32) else 4e-3
    assert rel_l2(got, ref) < tol, rel_l2(got, ref)


def _periodic_linear_case(epi, M, N, K, key):
    """Inputs whose rows repeat with prime periods, and the oracle's full
    output built from one period of each."""
    import torch
    PA, PR = 509, 263
    A, tileA = _tiled_rows((key, 0), M, K, PA, 1.0, True)
    W = normal((key, 1), (N, K), 0.02, True)
    b = normal((key, 2), (N,), 0.02, True)
    gate = normal((key, 3), (N,), 1.0)
    rows = np.arange(M)
    y_tile = dit.linear(tileA.astype(np.float64), W, b)
    resid_tile = None
    if epi in (track.EPI_GATE_RESID, track.EPI_RESID):
        out, resid_tile = _tiled_rows((key, 4), M, N, PR, 1.0, False)
    elif epi == track.EPI_BIAS_F32:
        out = torch.empty(M, N, dtype=torch.float32, device="cuda")
    else:
        out = torch.empty(M, N, dtype=torch.bfloat16, device="cuda")
    track.op_linear(track.DTYPE_BF16, epi, A, dev(W, BF16), dev(b, BF16), out, gate=dev(gate))
    y = y_tile[rows % PA]
    if epi == track.EPI_BIAS_GELU:
        ref = dit.gelu_tanh(y)
    elif epi == track.EPI_GATE_RESID:
        ref = resid_tile[rows % PR] + gate * y
    elif epi == track.EPI_RESID:
        ref = resid_tile[rows % PR] + y
    else:
        ref = y
    return host(out), ref


@pytest.mark.parametrize("epi", EPIS)
@pytest.mark.parametrize("M,N,K", [(65537, 512, 64), (65600, 768, 192)])
def test_linear_persistent_full_output(epi, M, N, K):
    """Shapes with at least 512 tiles of 256 x 256 run the persistent kernel:
    K = 64 starts a new tile at every slab, 65537 rows leave a one-row last
    M-tile, 771 tiles split unevenly over the workgroups.  Every output is
    compared."""
    say(f"linear persistent epi={epi} M={M} N={N} K={K}")
    got, ref = _periodic_linear_case(epi, M, N, K, 8300 + epi)
    tol = 1e-5 if epi in (track.EPI_GATE_RESID, track.EPI_RESID, track.EPI_BIAS_F32) else 4e-3
    assert rel_l2(got, ref) < tol, rel_l2(got, ref)
    np.testing.assert_allclose(got, ref, rtol=0, atol=8 * tol * (np.abs(ref).max() + 1))


@pytest.mark.parametrize("epi", [track.EPI_BIAS, track.EPI_GATE_RESID])
def test_linear_persistent_row_blocks(epi):
    """An A matrix above 2 GiB (140000 x 8192 bf16) is processed in two row
    blocks (the kernel's buffer resource has a 32-bit size field)."""
    M, N, K = 140000, 512, 8192
    say(f"linear persistent row blocks epi={epi} M={M} N={N} K={K}")
    got, ref = _periodic_linear_case(epi, M, N, K, 8400 + epi)
    tol = 1e-5 if epi == track.EPI_GATE_RESID else 4e-3
    assert rel_l2(got, ref) < tol, rel_l2(got, ref)
    np.testing.assert_allclose(got, ref, rtol=0, atol=8 * tol * (np.abs(ref).max() + 1))


@pytest.mark.parametrize("B,L,N,K,ldv", [(2, 1000, 512, 320, 1008), (3, 136, 256, 64, 136),
                                          (2, 32760, 1536, 1536, 32768), (2, 70000, 256, 8192, 70000)])
def test_linear_vt(B, L, N, K, ldv):
    """The V projection written transposed per batch (the V^T layout attention
    reads): ragged 256-row tiles, batches that change inside a wave's 128
    rows (L = 136), the Wan-1.3B shape, and an A above 2 GiB split into row
    blocks (the second block starts inside batch 1).  Every output is compared
    and the padding columns [L, ldv) stay untouched."""
    import torch
    M = B * L
    say(f"linear_vt B={B} L={L} N={N} K={K} ldv={ldv}")
    key = 8500 + L
    PA = 509
    A, tileA = _tiled_rows((key, 0), M, K, PA, 1.0, True)
    W = normal((key, 1), (N, K), 0.02, True)
    b = normal((key, 2), (N,), 0.02, True)
    vt = torch.full((B * N, ldv), 7.0, dtype=torch.bfloat16, device="cuda")
    track.op_linear_vt(A, dev(W, BF16), dev(b, BF16), L, vt, ldv)
    v = host(vt).reshape(B, N, ldv)
    assert np.all(v[:, :, L:] == 7.0)
    got = v[:, :, :L].transpose(0, 2, 1).reshape(M, N)
    ref = dit.linear(tileA.astype(np.float64), W, b)[np.arange(M) % PA]
    assert rel_l2(got, ref) < 4e-3, rel_l2(got, ref)
    np.testing.assert_allclose(got, ref, rtol=0, atol=3.2e-2 * (np.abs(ref).max() + 1))


@pytest.mark.parametrize("q_log2", [False, True])
@pytest.mark.parametrize("Lk", [32760, 512])
def test_attention_full_size_sampled(Lk, q_log2):
    say(f"attention full size Lq=32760 Lk={Lk} q_log2={q_log2}")
    import torch
    B, H, dh, Lq = 2, 12, 128, 32760
    d = H * dh
    q = normal((8100, 1), (B * Lq, d), 1.0, True)
    k = normal((8100, 2), (B * Lk, d), 1.0, True)
    v = normal((8100, 3), (B * Lk, d), 1.0, True)
    q, qr = _q_log2(q, dh, q_log2)
    ldv = (Lk + 63) // 64 * 64
    tv = dev(v, BF16).reshape(B, Lk, H, dh).permute(0, 2, 3, 1)
    vt = torch.zeros(B, H, dh, ldv, dtype=torch.bfloat16, device="cuda")
    vt[..., :Lk] = tv
    out = torch.empty(B * Lq, d, dtype=torch.bfloat16, device="cuda")
    track.op_attention(track.DTYPE_BF16, B, H, dh, Lq, Lk, dev(q, BF16), d, dev(k, BF16), d, vt, ldv, out, d,
                       q_log2=q_log2)
    rng = np.random.default_rng(2)
    rows = np.concatenate([rng.integers(0, Lq, 12), [0, Lq - 1, 32767 - 8]])
    got = host(out).reshape(B, Lq, H, dh)
    for b in range(B):
        qs = qr.reshape(B, Lq, H, dh)[b][rows]
        ref = dit.attention(qs, k.reshape(B, Lk, H, dh)[b].astype(np.float64),
                            v.reshape(B, Lk, H, dh)[b].astype(np.float64))
        assert rel_l2(got[b][rows], ref) < 1e-2, rel_l2(got[b][rows], ref)


@pytest.mark.parametrize("q_log2", [False, True])
@pytest.mark.parametrize("B,H,Lq,Lk", [(2, 3, 700, 512), (1, 2, 5000, 77), (2, 2, 300, 1000), (1, 1, 1, 128),
                                         (1, 2, 300, 2048), (2, 1, 257, 1985), (2, 12, 32760, 512)])
def test_attention_items_kernel_matches_blocks(B, H, Lq, Lk, q_log2):
    """Short key sequences (an even number of at most 32 tiles) run on the item-loop kernel, one workgroup
    per CU walking (query block, head, batch) items.  Tile for tile it computes what the per-block kernel
    does, so the two agree bit for bit; the first case is also checked against the oracle."""
    say(f"attention items vs blocks B={B} H={H} Lq={Lq} Lk={Lk} q_log2={q_log2}")
    import os
    import torch
    dh = 128
    d = H * dh
    key = 8200 + Lq + Lk
    q = normal((key, 1), (B * Lq, d), 1.0, True)
    k = normal((key, 2), (B * Lk, d), 1.0, True)
    v = normal((key, 3), (B * Lk, d), 1.0, True)
    q, qr = _q_log2(q, dh, q_log2)
    ldv = (Lk + 63) // 64 * 64
    vt = torch.zeros(B, H, dh, ldv, dtype=torch.bfloat16, device="cuda")
    vt[..., :Lk] = dev(v, BF16).reshape(B, Lk, H, dh).permute(0, 2, 3, 1)
    qd, kd = dev(q, BF16), dev(k, BF16)
    outs = []
    prev = os.environ.get("TRACK_ATTN_ITEMS")
    try:
        for flag in ("1", "0"):
            os.environ["TRACK_ATTN_ITEMS"] = flag
            out = torch.full((B * Lq, d), float("nan"), dtype=torch.bfloat16, device="cuda")
            track.op_attention(track.DTYPE_BF16, B, H, dh, Lq, Lk, qd, d, kd, d, vt, ldv, out, d, q_log2=q_log2)
            torch.cuda.synchronize()
            outs.append(out)
    finally:
        if prev is None:
            os.environ.pop("TRACK_ATTN_ITEMS", None)
        else:
            os.environ["TRACK_ATTN_ITEMS"] = prev
    assert bool(torch.isfinite(outs[0].float()).all())
    assert torch.equal(outs[0].view(torch.int16), outs[1].view(torch.int16))
    if B * Lq * Lk <= 1400 * 2048:
        got = host(outs[0]).reshape(B, Lq, H, dh)
        ref = np.stack([dit.attention(qr.reshape(B, Lq, H, dh)[b],
                                      k.reshape(B, Lk, H, dh)[b].astype(np.float64),
                                      v.reshape(B, Lk, H, dh)[b].astype(np.float64)) for b in range(B)])
        assert rel_l2(got, ref) < 1e-2, rel_l2(got, ref)


def test_mfma_stream_kernel():
    """The matrix-core stream runs on every CU, reports its FLOP count and leaves the sink alone."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    ops = (torch.randn(32768, device="cuda") * 0.5).to(torch.bfloat16)
    sink = torch.full((4,), 7.0, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    flop = track.mfma_stream(ops, 100, sink)  # warm
    e0.record()
    flop = track.mfma_stream(ops, 20000, sink)
    e1.record()
    torch.cuda.synchronize()
    assert flop == cus * 4 * 20000 * 8 * 32768
    assert bool((sink == 7.0).all())
    tflops = flop / e0.elapsed_time(e1) / 1e9
    print(f"mfma_stream: {tflops:.0f} TFLOP/s on {cus} CUs")
    assert 100.0 < tflops < 2600.0  # a launch that did no work, or more than the chip can, fails


def test_hbm_stream_kernels():
    """The plain copy / read / write streams used as the HBM ceiling move exactly the bytes asked for."""
    import torch
    n = 3 * 16384
    src = torch.randint(0, 255, (n + 64,), dtype=torch.uint8, device="cuda")
    dst = torch.zeros(n + 64, dtype=torch.uint8, device="cuda")
    track.hbm_stream(track.HBM_COPY, src, dst, n)
    assert torch.equal(dst[:n], src[:n]) and int(dst[n:].sum()) == 0
    before = src.clone()
    track.hbm_stream(track.HBM_COPY, src, src, n)  # in place
    assert torch.equal(src, before)
    track.hbm_stream(track.HBM_WRITE, None, dst, n)
    w = dst[:n].view(torch.float32)
    assert bool((w == 1.0).all()) and int(dst[n:].sum()) == 0
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    track.hbm_stream(track.HBM_READ, src, sink, n)
    torch.cuda.synchronize()
    with pytest.raises(track.TrackError):
        track.hbm_stream(track.HBM_COPY, src, dst, 1000)
