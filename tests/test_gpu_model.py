"""GPU parity of the full denoiser step, calibration, routing and routed
sampling against the float64 oracle, through the C ABI; plus the bitwise
determinism claims of the interface."""
import dataclasses

import numpy as np
import pytest

from gpu_helpers import dev, host, rel_l2, say
from structured_pairs import (TIMESTEP_SHIFT_BF16, TIMESTEP_SHIFT_F32, boundary_gaps, score_tolerance,
                              timestep_pair)
from oracle import dit, sampler
from paper_2609_30096_amd import synth, track

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-4   # per-step guided velocity, relative L2, float32 path
TOL_BF16 = 2e-2  # same, bfloat16 path

# bfloat16 test pair: Wan head width (128), two heads, ragged token and text counts
BF_LARGE = synth.DiTConfig(blocks=2, dim=256, heads=2, head_dim=128, ffn_dim=512, text_dim=256)
BF_SMALL = dataclasses.replace(BF_LARGE, blocks=1)
BF_LATENT = synth.LatentShape(16, 3, 10, 14, 7)   # 3 x 5 x 7 = 105 tokens
BF_SAMPLER = synth.SamplerConfig(steps=4, shift=3.0, guidance=5.0)
# 4 x 8 x 8 = 256 tokens: whole 8-token groups, so the V projection writes V^T from its epilogue
BF_LATENT_VT = synth.LatentShape(16, 4, 16, 16, 7)


class Pair:
    """Host parameters (for the oracle) and device models of one config pair."""

    def __init__(self, cfg_L, cfg_S, shape, seed_L=synth.SEED_LARGE, seed_S=synth.SEED_SMALL):
        self.shape = shape
        self.pL = synth.gen_params(cfg_L, seed_L)
        self.pS = synth.gen_params(cfg_S, seed_S)
        self.cL, self.cS = cfg_L, cfg_S
        self.L = track.Model(cfg_L, track.pack_weights(cfg_L, self.pL))
        self.S = track.Model(cfg_S, track.pack_weights(cfg_S, self.pS))
        dt = cfg_L.dtype
        self.dt = dt
        self.x = [synth.gen_latent(shape, j) for j in range(4)]
        self.c = [synth.gen_text(shape, cfg_L.text_dim, j, dt) for j in range(4)]
        self.u = synth.gen_null_text(shape, cfg_L.text_dim, dt)
        self.dx = [dev(a) for a in self.x]
        self.dc = [dev(a, dt) for a in self.c]
        self.du = dev(self.u, dt)


@pytest.fixture(scope="module")
def tiny():
    say("building tiny float32 pair")
    return Pair(synth.TINY_LARGE, synth.TINY_SMALL, synth.TINY_LATENT)


@pytest.fixture(scope="module")
def bfp():
    say("building bf16 pair")
    return Pair(BF_LARGE, BF_SMALL, BF_LATENT)


def _teacher_forced(pair, model_gpu, model_ora, scfg, j, tol):
    sig = sampler.sigmas(scfg.steps, scfg.shift)
    large = (pair.pL, pair.cL)
    _, path = sampler.sample(np.zeros(scfg.steps, bool), large, None, pair.x[j], pair.c[j], pair.u, scfg,
                             return_path=True)
    errs = []
    for k in range(scfg.steps):
        xk = path[k].astype(np.float32)  # both sides get the same float32 latent
        t = 1000.0 * sig[k]
        got = host(track.dit_forward(model_gpu, pair.shape, dev(xk), t, pair.dc[j], pair.du, scfg.guidance))
        ref = sampler.guided_prediction(model_ora, xk.astype(np.float64), t, pair.c[j], pair.u, scfg)
        errs.append(rel_l2(got, ref))
    say(f"  per-step relative L2: {['%.2e' % e for e in errs]}")
    assert max(errs) < tol, errs
    return errs


def test_tiny_f32_teacher_forced_velocity(tiny):
    say("tiny f32 teacher-forced")
    for j in range(2):
        _teacher_forced(tiny, tiny.L, (tiny.pL, tiny.cL), synth.TINY_SAMPLER, j, TOL_F32)
        _teacher_forced(tiny, tiny.S, (tiny.pS, tiny.cS), synth.TINY_SAMPLER, j, TOL_F32)


def test_tiny_f32_unguided_forward(tiny):
    scfg = dataclasses.replace(synth.TINY_SAMPLER, use_cfg=False)
    got = host(track.dit_forward(tiny.L, tiny.shape, tiny.dx[0], 700.0, tiny.dc[0], None, 1.0))
    ref = sampler.guided_prediction((tiny.pL, tiny.cL), tiny.x[0].astype(np.float64), 700.0, tiny.c[0], None, scfg)
    assert rel_l2(got, ref) < TOL_F32


def _routing_agrees(q_gpu, q_ora, K, delta):
    """Top-K routing parity for per-step velocity tolerance delta.

    The device's scores may differ from the oracle's by up to the bound
    score_tolerance(q, delta).  Where the gap between the oracle's K-th and
    (K+1)-th smallest scores exceeds the two steps' summed bounds, the device
    must pick exactly the oracle's steps; otherwise every step on which the
    two picks differ must itself lie within its bound of that boundary."""
    got = set(track.route_policy(q_gpu, K).tolist())
    exp = set(sampler.route_topk(q_ora, K).tolist())
    if got == exp:
        return True
    if K == 0 or K == len(q_ora):
        return False
    tau = score_tolerance(q_ora, delta)
    order = np.argsort(q_ora, kind="stable")
    lo, hi = order[K - 1], order[K]
    if q_ora[hi] - q_ora[lo] > tau[lo] + tau[hi]:
        return False
    for k in got ^ exp:
        if q_ora[k] < q_ora[lo] - tau[k] - tau[lo] or q_ora[k] > q_ora[hi] + tau[k] + tau[hi]:
            return False
    return True


def _routing_parity_all_K(q_gpu, q_ora, delta, label):
    """_routing_agrees for every K, reporting the oracle's boundary gaps against their tolerances.
    Returns the K whose boundary is resolved (gap above tolerance)."""
    resolved = []
    for K, gap, tol in boundary_gaps(q_ora, delta):
        assert _routing_agrees(q_gpu, q_ora, K, delta), (label, K, gap, tol)
        if gap > tol:
            resolved.append(K)
    gaps = boundary_gaps(q_ora, delta)
    worst = max(abs(a - b) / t for a, b, t in zip(q_gpu, q_ora, score_tolerance(q_ora, delta)))
    say(f"  {label}: boundary gap / tolerance for K = 1..{len(q_ora) - 1}: "
        f"{[round(g / t, 2) for _, g, t in gaps]}; resolved K {resolved}; "
        f"max |q_gpu - q_oracle| / tolerance {worst:.3f}")
    return resolved


def test_tiny_f32_calibration_routing_and_sample(tiny):
    say("tiny f32 calibration")
    scfg = synth.TINY_SAMPLER
    large, small = (tiny.pL, tiny.cL), (tiny.pS, tiny.cS)
    r_ora, q_ora = sampler.calibrate(large, small, tiny.x, tiny.c, tiny.u, scfg)
    r, q = track.calibrate(tiny.L, tiny.S, tiny.shape, tiny.dx, tiny.dc, tiny.du, scfg)
    say(f"  q gpu    {np.round(q, 5)}\n  q oracle {np.round(q_ora, 5)}")
    np.testing.assert_allclose(r, r_ora, rtol=1e-3, atol=1e-6)
    np.testing.assert_allclose(q, np.mean(r, axis=0), rtol=1e-15)
    assert _routing_agrees(q, q_ora, 4, TOL_F32)
    idx = track.route_policy(q, 4)
    use_small = sampler.policy_from_indices(8, idx)
    x0 = host(track.sample(tiny.L, tiny.S, use_small, tiny.shape, scfg, tiny.dx[0], tiny.dc[0], tiny.du))
    ref = sampler.sample(use_small, large, small, tiny.x[0], tiny.c[0], tiny.u, scfg)
    err = rel_l2(x0, ref)
    say(f"  routed sample x0 relative L2 vs oracle: {err:.2e}")
    assert err < 1e-3


def test_tiny_f32_calibration_bands(tiny):
    from oracle import bands
    say("tiny f32 calibration with band decomposition")
    scfg = synth.TINY_SAMPLER
    large, small = (tiny.pL, tiny.cL), (tiny.pS, tiny.cS)
    r_o, q_o, rb_o, qb_o = bands.calibrate_bands(large, small, tiny.x, tiny.c, tiny.u, scfg)
    r, q, rb, qb = track.calibrate(tiny.L, tiny.S, tiny.shape, tiny.dx, tiny.dc, tiny.du, scfg, bands=True)
    say(f"  qb gpu\n{np.round(qb, 4)}\n  qb oracle\n{np.round(qb_o, 4)}")
    np.testing.assert_allclose(r, r_o, rtol=1e-3, atol=1e-6)
    np.testing.assert_allclose(rb, rb_o, rtol=2e-3, atol=1e-5 * float(r_o.max()))
    np.testing.assert_allclose(qb, rb.mean(axis=0), rtol=1e-14)
    # each triple's squares sum to r^2 (Parseval) on the device values
    np.testing.assert_allclose((rb[..., :3] ** 2).sum(-1), r ** 2, rtol=2e-5)
    np.testing.assert_allclose((rb[..., 3:] ** 2).sum(-1), r ** 2, rtol=2e-5)
    # the band kernels do not touch the trajectory: r matches plain calibration bit for bit
    r2, q2 = track.calibrate(tiny.L, tiny.S, tiny.shape, tiny.dx, tiny.dc, tiny.du, scfg)
    np.testing.assert_array_equal(r, r2)


def test_tiny_f32_unipc_sample_and_calibration(tiny):
    say("tiny f32 UniPC sampling and calibration")
    large, small = (tiny.pL, tiny.cL), (tiny.pS, tiny.cS)
    for order in (2, 3):
        scfg = dataclasses.replace(synth.TINY_SAMPLER, solver="unipc", order=order)
        pol = np.array([False, True, True, False, True, False, False, True])  # switches both ways
        x0 = host(track.sample(tiny.L, tiny.S, pol, tiny.shape, scfg, tiny.dx[0], tiny.dc[0], tiny.du))
        ref = sampler.sample(pol, large, small, tiny.x[0], tiny.c[0], tiny.u, scfg)
        err = rel_l2(x0, ref)
        say(f"  order {order}: routed UniPC sample x0 relative L2 vs oracle: {err:.2e}")
        assert err < 1e-3
        r, q, x0c = track.calibrate(tiny.L, tiny.S, tiny.shape, tiny.dx[:2], tiny.dc[:2], tiny.du, scfg,
                                    return_x0=True)
        r_o, q_o = sampler.calibrate(large, small, tiny.x[:2], tiny.c[:2], tiny.u, scfg)
        np.testing.assert_allclose(r, r_o, rtol=1e-3, atol=1e-6)
        # K = 0 reproduces the calibration's all-large UniPC trajectory bit for bit
        import torch
        xs = track.sample(tiny.L, tiny.S, np.zeros(8, bool), tiny.shape, scfg, tiny.dx[1], tiny.dc[1], tiny.du)
        assert torch.equal(xs, x0c[1])
    # UniPC differs from Euler on the same policy (the scheduler really changed)
    e = host(track.sample(tiny.L, tiny.S, pol, tiny.shape, synth.TINY_SAMPLER, tiny.dx[0], tiny.dc[0], tiny.du))
    assert rel_l2(e, x0) > 1e-3


def test_tiny_f32_unipc_history_survives_switches(tiny):
    # two handles over the same weights: any policy must give the all-large
    # result bit for bit, which fails if a switch resets the scheduler history
    import torch
    scfg = dataclasses.replace(synth.TINY_SAMPLER, solver="unipc", order=3)
    L2 = track.Model(tiny.cL, tiny.L.weights)
    ref = track.sample(tiny.L, None, np.zeros(8, bool), tiny.shape, scfg, tiny.dx[2], tiny.dc[2], tiny.du)
    for pol in [np.arange(8) % 2 == 1, np.arange(8) >= 4]:
        got = track.sample(tiny.L, L2, pol, tiny.shape, scfg, tiny.dx[2], tiny.dc[2], tiny.du)
        assert torch.equal(got, ref)


def test_tiny_f32_determinism_claims(tiny):
    say("tiny f32 determinism")
    import torch
    scfg = dataclasses.replace(synth.TINY_SAMPLER, steps=5)
    a = track.dit_forward(tiny.L, tiny.shape, tiny.dx[1], 321.0, tiny.dc[1], tiny.du, 5.0)
    b = track.dit_forward(tiny.L, tiny.shape, tiny.dx[1], 321.0, tiny.dc[1], tiny.du, 5.0)
    assert torch.equal(a, b)
    # self-disagreement is exactly zero (a second handle over the same weights)
    L2 = track.Model(tiny.cL, tiny.L.weights)
    r, q, x0 = track.calibrate(tiny.L, L2, tiny.shape, tiny.dx[:2], tiny.dc[:2], tiny.du, scfg, return_x0=True)
    assert np.all(r == 0.0)
    # K = 0 reproduces the calibration's all-large trajectory bit for bit
    for j in range(2):
        xs = track.sample(tiny.L, tiny.S, np.zeros(5, bool), tiny.shape, scfg, tiny.dx[j], tiny.dc[j], tiny.du)
        assert torch.equal(xs, x0[j])
    # K = N reproduces the all-small trajectory
    xa = track.sample(tiny.L, tiny.S, np.ones(5, bool), tiny.shape, scfg, tiny.dx[0], tiny.dc[0], tiny.du)
    xb = track.sample(tiny.S, None, np.zeros(5, bool), tiny.shape, scfg, tiny.dx[0], tiny.dc[0], tiny.du)
    assert torch.equal(xa, xb)
    # sample may run in place (x_T and x_0 alias) and gives the same bits
    xin = tiny.dx[0].clone()
    out = track.sample(tiny.L, tiny.S, np.zeros(5, bool), tiny.shape, scfg, xin, tiny.dc[0], tiny.du, out=xin)
    assert out.data_ptr() == xin.data_ptr()
    assert torch.equal(xin, x0[0])


def _bitwise_claims(L, S, cfg, shape, dx, dc, du, scfg, label):
    """The determinism guarantees of the interface on one model pair, for one sampler:
    repeated forwards give equal bits; a model's disagreement with a second handle over its own
    weights is exactly 0; K = 0 reproduces the calibration's all-large trajectory bit for bit;
    K = N reproduces the all-small trajectory; and with the second handle as the small model every
    policy reproduces the all-large trajectory (a switch changes nothing but the model, so each prefix
    before a small step is the all-large prefix and the scheduler state survives the switch)."""
    import torch
    N = scfg.steps
    for unc in (du, None):
        a = track.dit_forward(L, shape, dx[0], 777.0, dc[0], unc, scfg.guidance)
        b = track.dit_forward(L, shape, dx[0], 777.0, dc[0], unc, scfg.guidance)
        assert torch.equal(a, b), label
    L2 = track.Model(cfg, L.weights)
    r, q, x0 = track.calibrate(L, L2, shape, dx[:2], dc[:2], du, scfg, return_x0=True)
    assert np.all(r == 0.0), (label, r)
    for j in range(2):
        xs = track.sample(L, S, np.zeros(N, bool), shape, scfg, dx[j], dc[j], du)
        assert torch.equal(xs, x0[j]), (label, "K = 0", j)
    xa = track.sample(L, S, np.ones(N, bool), shape, scfg, dx[0], dc[0], du)
    xb = track.sample(S, None, np.zeros(N, bool), shape, scfg, dx[0], dc[0], du)
    assert torch.equal(xa, xb), (label, "K = N")
    for pol in (np.arange(N) % 2 == 1, np.arange(N) >= N // 2, np.arange(N) == N - 1):
        got = track.sample(L, L2, pol, shape, scfg, dx[0], dc[0], du)
        assert torch.equal(got, x0[0]), (label, "switch to a second handle", pol)
    # a genuinely different small model does change the result
    xr = track.sample(L, S, np.arange(N) == N - 1, shape, scfg, dx[0], dc[0], du)
    assert not torch.equal(xr, x0[0])
    say(f"  {label}: bitwise claims hold")


def test_bf16_determinism_claims():
    """The bf16 pair on 256 tokens (V^T from the projection epilogue), with the automatic kernel
    choice and with the projections forced onto the persistent GEMM kernel, Euler and UniPC-2."""
    import os
    say("bf16 determinism")
    pair = Pair(BF_LARGE, BF_SMALL, BF_LATENT_VT)
    for forced in ("0", "4"):
        os.environ["TRACK_GEMM_CFG"] = forced
        try:
            for scfg in (BF_SAMPLER, dataclasses.replace(BF_SAMPLER, solver="unipc", order=2)):
                _bitwise_claims(pair.L, pair.S, pair.cL, pair.shape, pair.dx, pair.dc, pair.du, scfg,
                                f"bf16 pair, {scfg.solver}, TRACK_GEMM_CFG={forced}")
        finally:
            os.environ.pop("TRACK_GEMM_CFG", None)


def test_bf16_determinism_claims_wan_width_full_size():
    """One Wan-1.3B-width block (d = 1536) as the large model and a second one-block model as the
    small one, on the full 16 x 21 x 60 x 104 latent with CFG: the step's own kernels (persistent
    GEMMs, V^T epilogue, the flash attention over 32760 keys, the wide norms)."""
    say("bf16 determinism, Wan width, full size")
    cfg = dataclasses.replace(synth.WAN_1_3B, blocks=1)
    shape = synth.WAN_LATENT
    L = track.Model(cfg, track.gen_weights_on_device(cfg, synth.SEED_SMALL))
    S = track.Model(cfg, track.gen_weights_on_device(cfg, synth.SEED_LARGE))
    dx = [dev(synth.gen_latent(shape, j)) for j in range(2)]
    dc = [dev(synth.gen_text(shape, cfg.text_dim, j, synth.BF16), synth.BF16) for j in range(2)]
    du = dev(synth.gen_null_text(shape, cfg.text_dim, synth.BF16), synth.BF16)
    base = synth.SamplerConfig(steps=4, shift=5.0, guidance=5.0)
    for scfg in (base, dataclasses.replace(base, solver="unipc", order=2)):
        _bitwise_claims(L, S, cfg, shape, dx, dc, du, scfg, f"Wan width, {scfg.solver}")


def test_tiny_nested_pair_calibration(tiny):
    """Structured pair: the small model is the large model's first two blocks with the large model's
    own weights (shared embeddings and head), so the disagreement is what the dropped blocks add."""
    say("tiny nested pair")
    cS = dataclasses.replace(tiny.cL, blocks=2)
    pS = {k: v for k, v in tiny.pL.items() if not k.startswith("blk") or int(k[3:].split(".")[0]) < 2}
    S = track.Model(cS, track.pack_weights(cS, pS))
    scfg = dataclasses.replace(synth.TINY_SAMPLER, steps=4)
    r, q = track.calibrate(tiny.L, S, tiny.shape, tiny.dx[:2], tiny.dc[:2], tiny.du, scfg)
    r_ora, q_ora = sampler.calibrate((tiny.pL, tiny.cL), (pS, cS), tiny.x[:2], tiny.c[:2], tiny.u, scfg)
    say(f"  q gpu    {np.round(q, 5)}\n  q oracle {np.round(q_ora, 5)}")
    assert np.all(r > 0) and np.all(np.isfinite(r))
    np.testing.assert_allclose(r, r_ora, rtol=1e-3, atol=1e-6)


def test_tiny_perturbed_pair_is_linear_in_delta(tiny):
    """Structured pair: S = L + delta N(0,1) on every weight.  For small delta the disagreement is
    first order in delta (r(2 delta) = 2 r(delta) up to O(delta^2)), and each matches the oracle."""
    say("tiny perturbed pair")
    scfg = dataclasses.replace(synth.TINY_SAMPLER, steps=3)
    rs = []
    for delta in (1e-4, 2e-4):
        pS = {k: v + delta * synth.gen_normal((9100, i), v.shape).astype(v.dtype)
              for i, (k, v) in enumerate(sorted(tiny.pL.items()))}
        S = track.Model(tiny.cL, track.pack_weights(tiny.cL, pS))
        r, _ = track.calibrate(tiny.L, S, tiny.shape, tiny.dx[:1], tiny.dc[:1], tiny.du, scfg)
        r_ora, _ = sampler.calibrate((tiny.pL, tiny.cL), (pS, tiny.cL), tiny.x[:1], tiny.c[:1], tiny.u, scfg)
        np.testing.assert_allclose(r, r_ora, rtol=2e-2, atol=1e-7)
        rs.append(r)
    say(f"  r(delta) {rs[0]}, r(2 delta) {rs[1]}")
    np.testing.assert_allclose(rs[1], 2 * rs[0], rtol=2e-2)


def test_tiny_scaled_head_pair_r_is_exact(tiny):
    # S = L with the output projection doubled: p_S = 2 p_L exactly, so r = 1 exactly
    scaled = dict(tiny.pL)
    scaled["head.w"] = tiny.pL["head.w"] * 2
    scaled["head.b"] = tiny.pL["head.b"] * 2
    S2 = track.Model(tiny.cL, track.pack_weights(tiny.cL, scaled))
    scfg = dataclasses.replace(synth.TINY_SAMPLER, steps=3)
    r, q = track.calibrate(tiny.L, S2, tiny.shape, tiny.dx[:1], tiny.dc[:1], tiny.du, scfg)
    assert np.all(r == 1.0), r


SAMPLER8 = synth.SamplerConfig(steps=8, shift=3.0, guidance=5.0)


def _timestep_pair_routing(cfg, shape, alpha, delta, label):
    """Calibration and top-K routing of a large model against its timestep-offset copy, whose
    disagreement varies strongly from step to step; the routing must equal the oracle's wherever a
    boundary gap exceeds the score tolerance, and the boundaries routed below must be resolved."""
    pL = synth.gen_params(cfg, synth.SEED_LARGE)
    pS = timestep_pair(cfg, pL, alpha)
    L = track.Model(cfg, track.pack_weights(cfg, pL))
    S = track.Model(cfg, track.pack_weights(cfg, pS))
    M = 4
    xs = [synth.gen_latent(shape, j) for j in range(M)]
    cs = [synth.gen_text(shape, cfg.text_dim, j, cfg.dtype) for j in range(M)]
    u = synth.gen_null_text(shape, cfg.text_dim, cfg.dtype)
    r_ora, q_ora = sampler.calibrate((pL, cfg), (pS, cfg), xs, cs, u, SAMPLER8)
    r, q = track.calibrate(L, S, shape, [dev(a) for a in xs], [dev(a, cfg.dtype) for a in cs], dev(u, cfg.dtype),
                           SAMPLER8)
    say(f"  {label}: q gpu    {np.round(q, 5)}\n  {label}: q oracle {np.round(q_ora, 5)}")
    resolved = _routing_parity_all_K(q, q_ora, delta, label)
    return q, q_ora, resolved


def test_tiny_f32_timestep_pair_routing():
    q, q_ora, resolved = _timestep_pair_routing(synth.TINY_LARGE, synth.TINY_LATENT, TIMESTEP_SHIFT_F32, TOL_F32,
                                                "f32 timestep pair")
    assert resolved == list(range(1, 8))
    np.testing.assert_array_equal(track.route_policy(q, 4), sampler.route_topk(q_ora, 4))


def test_bf16_timestep_pair_routing():
    q, q_ora, resolved = _timestep_pair_routing(BF_LARGE, BF_LATENT, TIMESTEP_SHIFT_BF16, TOL_BF16,
                                                "bf16 timestep pair")
    assert 2 in resolved and 4 in resolved
    for K in (2, 4):
        np.testing.assert_array_equal(track.route_policy(q, K), sampler.route_topk(q_ora, K))


def test_bf16_teacher_forced_velocity(bfp):
    say("bf16 teacher-forced")
    _teacher_forced(bfp, bfp.L, (bfp.pL, bfp.cL), BF_SAMPLER, 0, TOL_BF16)
    _teacher_forced(bfp, bfp.S, (bfp.pS, bfp.cS), BF_SAMPLER, 1, TOL_BF16)


def test_bf16_teacher_forced_velocity_vt_epilogue():
    """The same pair on a latent whose token count takes the transposed-V projection path."""
    say("bf16 teacher-forced, V^T from the projection epilogue")
    pair = Pair(BF_LARGE, BF_SMALL, BF_LATENT_VT)
    _teacher_forced(pair, pair.L, (pair.pL, pair.cL), BF_SAMPLER, 0, TOL_BF16)


def test_bf16_calibration_and_routing(bfp):
    say("bf16 calibration")
    large, small = (bfp.pL, bfp.cL), (bfp.pS, bfp.cS)
    r_ora, q_ora = sampler.calibrate(large, small, bfp.x[:2], bfp.c[:2], bfp.u, BF_SAMPLER)
    r, q = track.calibrate(bfp.L, bfp.S, bfp.shape, bfp.dx[:2], bfp.dc[:2], bfp.du, BF_SAMPLER)
    say(f"  r gpu    {np.round(r, 4)}\n  r oracle {np.round(r_ora, 4)}")
    np.testing.assert_allclose(r, r_ora, rtol=3e-2, atol=3e-2)
    assert _routing_agrees(q, q_ora, 2, TOL_BF16)


def test_bf16_unguided_sample_matches_oracle(bfp):
    scfg = dataclasses.replace(BF_SAMPLER, use_cfg=False)
    pol = np.array([False, True, True, False])
    x0 = host(track.sample(bfp.L, bfp.S, pol, bfp.shape, scfg, bfp.dx[0], bfp.dc[0], None))
    ref = sampler.sample(pol, (bfp.pL, bfp.cL), (bfp.pS, bfp.cS), bfp.x[0], bfp.c[0], None, scfg)
    err = rel_l2(x0, ref)
    say(f"  bf16 routed sample x0 relative L2 vs oracle: {err:.2e}")
    assert err < 2e-2


def _one_block_full_size_sampled(base_cfg, seed, label, shape=synth.WAN_LATENT, cfg_guided=True):
    """One block of the given width on a full-size latent (81 x 480 x 832: 32760 tokens, CFG batch 2;
    81 x 720 x 1280 unguided: 75600 tokens, batch 1): the benchmark's kernels at their real shapes;
    the oracle evaluates sampled tokens."""
    say(f"{label} one block, full size")
    cfg = dataclasses.replace(base_cfg, blocks=1)
    params = synth.gen_params(cfg, seed)
    model = track.Model(cfg, track.pack_weights(cfg, params))
    x = synth.gen_latent(shape, 0)
    cond = synth.gen_text(shape, cfg.text_dim, 0, synth.BF16)
    unc = synth.gen_null_text(shape, cfg.text_dim, synth.BF16)
    t = 1000.0 * sampler.sigmas(50, 5.0)[10]
    if cfg_guided:
        got = host(track.dit_forward(model, shape, dev(x), t, dev(cond, synth.BF16), dev(unc, synth.BF16), 5.0))
    else:
        got = host(track.dit_forward(model, shape, dev(x), t, dev(cond, synth.BF16)))
    del model
    assert np.isfinite(got).all()
    say("  forward done; oracle on sampled tokens")
    # oracle on sampled tokens
    d, H, dh = cfg.dim, cfg.heads, cfg.head_dim
    P = {k: np.asarray(v, np.float64) for k, v in params.items()}
    del params
    pt, ph, pw = cfg.patch
    grid = (shape.frames // pt, shape.height // ph, shape.width // pw)
    L = grid[0] * grid[1] * grid[2]
    U = dit.patchify(x.astype(np.float64), cfg.patch)
    X0 = dit.linear(U, P["patch.w"], P["patch.b"])
    e, m = dit.time_embedding(P, cfg, t)
    rng = np.random.default_rng(3)
    toks = np.unique(np.concatenate([rng.integers(0, L, 14), [0, L - 1]]))
    # self-attention does not see the text: its keys, values and sampled queries serve both branches
    sh1, sc1, g1, sh2, sc2, g2 = m + P["blk0.mod"]
    Y = dit.layer_norm(X0) * (1 + sc1) + sh1
    qkv_k = dit.linear(Y, P["blk0.qkv.w"][d:], P["blk0.qkv.b"][d:])              # K and V, all tokens
    k = dit.rope3d(dit.rms_norm(qkv_k[:, :d], P["blk0.norm_k"]).reshape(L, H, dh), grid)
    v = qkv_k[:, d:].reshape(L, H, dh)
    del qkv_k
    q_all = dit.rms_norm(dit.linear(Y[toks], P["blk0.qkv.w"][:d], P["blk0.qkv.b"][:d]), P["blk0.norm_q"])
    del Y
    # RoPE of the sampled query rows: rotate a full-size array holding only those rows
    qfull = np.zeros((L, H, dh))
    qfull[toks] = q_all.reshape(-1, H, dh)
    q = dit.rope3d(qfull, grid)[toks]
    del qfull
    say("  oracle keys and values done")
    a = dit.attention(q, k, v).reshape(-1, d)
    X1 = X0[toks] + g1 * dit.linear(a, P["blk0.o.w"], P["blk0.o.b"])
    outs = []
    for ctx in ((cond, unc) if cfg_guided else (cond,)):
        C = dit.text_embedding(P, ctx)
        Yc = dit.layer_norm(X1)
        qc = dit.rms_norm(dit.linear(Yc, P["blk0.cq.w"], P["blk0.cq.b"]), P["blk0.norm_cq"])
        kv = dit.linear(C, P["blk0.ckv.w"], P["blk0.ckv.b"])
        kc = dit.rms_norm(kv[:, :d], P["blk0.norm_ck"])
        ac = dit.attention(qc.reshape(-1, H, dh), kc.reshape(-1, H, dh), kv[:, d:].reshape(-1, H, dh)).reshape(-1, d)
        X = X1 + dit.linear(ac, P["blk0.co.w"], P["blk0.co.b"])
        Y2 = dit.layer_norm(X) * (1 + sc2) + sh2
        X = X + g2 * dit.linear(dit.gelu_tanh(dit.linear(Y2, P["blk0.ffn1.w"], P["blk0.ffn1.b"])),
                                P["blk0.ffn2.w"], P["blk0.ffn2.b"])
        outs.append(dit.head(P, X, e))                                            # [n, 64] token layout
    ref_tok = sampler.guided(outs[0], outs[1], 5.0) if cfg_guided else outs[0]
    got_tok = dit.patchify(got.astype(np.float64), cfg.patch)[toks]
    err = rel_l2(got_tok, ref_tok)
    say(f"  width {d}, {len(toks)} of {L} tokens: sampled-token velocity relative L2 {err:.4e}")
    assert err < TOL_BF16


def test_wan13b_one_block_full_size_sampled():
    _one_block_full_size_sampled(synth.WAN_1_3B, synth.SEED_SMALL, "wan 1.3B")


def test_wan14b_one_block_full_size_sampled():
    """The 14B width (5120) takes the workgroup-per-row norm kernels and the largest GEMMs."""
    _one_block_full_size_sampled(synth.WAN_14B, synth.SEED_LARGE, "wan 14B")


def test_wan13b_one_block_full_size_long_unguided_sampled():
    """The step-distilled workload: 75600 tokens, no CFG (batch 1), ragged query tiles in attention."""
    _one_block_full_size_sampled(synth.WAN_1_3B, synth.SEED_SMALL, "wan 1.3B long", synth.WAN_LATENT_LONG, False)
