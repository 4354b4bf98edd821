"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function that include/track.h declares, and its host-only calls (weight
table, routing, argument validation) behave as documented."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import sampler
from paper_2609_30096_amd import synth, track

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "track.h")


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(track_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    return track.lib()


def test_library_exports_every_declared_function(L):
    names = header_functions()
    assert len(names) >= 20
    for n in names:
        assert hasattr(L, n), f"{n} declared in track.h but not exported"
    assert sorted(track.EXPORTS) == names


def test_weight_table_matches_recipe(L):
    for cfg in (synth.TINY_LARGE, synth.WAN_1_3B, synth.WAN_14B):
        table, total = track.weight_table(cfg)
        specs = synth.param_specs(cfg)
        assert [t[0] for t in table] == [s[0] for s in specs]
        assert [t[1] for t in table] == [s[1] for s in specs]
        es = 2 if cfg.dtype == synth.BF16 else 4
        end = 0
        for name, shape, off in table:
            assert off % 256 == 0 and off >= end
            end = off + int(np.prod(shape)) * es
        assert total >= end and total - end < 256
    # parameter counts of the Wan-shaped presets
    assert abs(synth.WAN_14B.n_params() - 14.28e9) < 0.02e9
    assert abs(synth.WAN_1_3B.n_params() - 1.42e9) < 0.02e9


def test_invalid_configs_rejected(L):
    bad = [
        dict(heads=3),                       # dim != heads * head_dim
        dict(dtype="bf16"),                  # bf16 with head_dim 32
    ]
    import dataclasses
    for kw in bad:
        cfg = dataclasses.replace(synth.TINY_LARGE, **kw)
        c = track.config_c(cfg)
        assert L.track_weight_count(ctypes.byref(c)) < 0
        assert L.track_weights_bytes(ctypes.byref(c)) == 0
        assert len(L.track_last_error()) > 0


def test_model_create_argument_checks(L):
    c = track.config_c(synth.TINY_LARGE)
    h = ctypes.c_void_p()
    assert L.track_model_create(ctypes.byref(c), None, 1 << 20, ctypes.byref(h)) == track.E_INVALID
    # misaligned pointer (never dereferenced on the host)
    assert L.track_model_create(ctypes.byref(c), ctypes.c_void_p(0x1001), 1 << 30, ctypes.byref(h)) == track.E_INVALID
    # buffer too small
    assert L.track_model_create(ctypes.byref(c), ctypes.c_void_p(0x100000), 16, ctypes.byref(h)) == track.E_SHAPE
    # a valid view (no device access happens at creation)
    total = L.track_weights_bytes(ctypes.byref(c))
    assert L.track_model_create(ctypes.byref(c), ctypes.c_void_p(0x100000), total, ctypes.byref(h)) == track.OK
    shp = track.shape_c(synth.TINY_LATENT)
    assert L.track_workspace_bytes(h, ctypes.byref(shp), 2) > L.track_workspace_bytes(h, ctypes.byref(shp), 1) > 0
    assert L.track_workspace_bytes(h, ctypes.byref(shp), 3) == 0
    bad = track.shape_c(synth.LatentShape(16, 4, 7, 8, 16))  # height not divisible by the patch
    assert L.track_workspace_bytes(h, ctypes.byref(bad), 2) == 0
    bad = track.shape_c(synth.LatentShape(8, 4, 8, 8, 16))  # channel mismatch
    assert L.track_workspace_bytes(h, ctypes.byref(bad), 2) == 0
    # calls that need a workspace fail cleanly without one
    x = ctypes.c_void_p(0x200000)
    assert L.track_dit_forward(h, ctypes.byref(shp), x, 500.0, x, x, 5.0, x, None) == track.E_NOMEM
    L.track_model_destroy(h)
    L.track_model_destroy(None)


def test_route_policy_golden_and_bruteforce(L):
    for line in open(os.path.join(ROOT, "tests", "golden", "topk_cases.txt")):
        if not line.strip() or line[0] == "#":
            continue
        k, q, exp = [p.split() for p in line.split("|")]
        got = track.route_policy([float(v) for v in q], int(k[0]))
        assert list(got) == [int(v) for v in exp]
    rng = np.random.default_rng(5)
    for _ in range(50):
        q = rng.random(12)
        q[rng.integers(0, 12, 3)] = q[0]  # force ties
        for K in range(13):
            np.testing.assert_array_equal(track.route_policy(q, K), sampler.route_topk(q, K))


def test_route_policy_errors(L):
    q = np.array([0.3, 0.1, 0.2])
    with pytest.raises(track.TrackError) as e:
        track.route_policy(q, 4)
    assert e.value.status == track.E_INVALID
    with pytest.raises(track.TrackError):
        track.route_policy(q, -1)
    with pytest.raises(track.TrackError):
        track.route_policy(np.array([0.1, np.nan]), 1)
    assert len(track.route_policy(q, 0)) == 0


def test_route_threshold_matches_oracle(L):
    rng = np.random.default_rng(7)
    for _ in range(40):
        N = int(rng.integers(1, 60))
        q = rng.uniform(0.0, 2.0, N)
        q[rng.integers(0, N, max(1, N // 4))] = q[0]  # ties, and W_k == C_0 below
        for C0 in (0.0, float(q[0] ** 2), float(np.median(q) ** 2), 5.0, -1.0):
            np.testing.assert_array_equal(track.route_threshold(q, C0), sampler.route_threshold(q, C0))
    with pytest.raises(track.TrackError):
        track.route_threshold(np.array([0.1, np.nan]), 1.0)
    with pytest.raises(track.TrackError):
        track.route_threshold(np.array([0.1]), float("nan"))


def test_route_baselines_match_oracle(L):
    rng = np.random.default_rng(8)
    for N, K in [(1, 0), (1, 1), (50, 25), (50, 30), (4, 2), (35, 17)]:
        np.testing.assert_array_equal(track.route_baseline(track.POLICY_FIRST_K, N, K), sampler.first_k(N, K))
        np.testing.assert_array_equal(track.route_baseline(track.POLICY_LAST_K, N, K), sampler.last_k(N, K))
        for seed in [0, 1, 2**63 + 5, 2**64 - 1] + [int(v) for v in rng.integers(0, 2**62, 20)]:
            np.testing.assert_array_equal(track.route_baseline(track.POLICY_RANDOM_K, N, K, seed),
                                          sampler.random_k(N, K, seed))
    for bad in [(3, 1, 4), (3, 1, -1), (7, 5, 2), (0, 0, 0)]:
        kind, N, K = bad
        with pytest.raises(track.TrackError):
            track.route_baseline(kind, N, K)


def test_calibrate_and_sample_argument_checks(L):
    cL = track.config_c(synth.TINY_LARGE)
    cS = track.config_c(synth.dataclasses.replace(synth.TINY_SMALL, text_dim=64))
    hL, hS = ctypes.c_void_p(), ctypes.c_void_p()
    assert L.track_model_create(ctypes.byref(cL), ctypes.c_void_p(0x100000), 1 << 40, ctypes.byref(hL)) == 0
    assert L.track_model_create(ctypes.byref(cS), ctypes.c_void_p(0x100000), 1 << 40, ctypes.byref(hS)) == 0
    shp = track.shape_c(synth.TINY_LATENT)
    sc = track.sampler_c(synth.TINY_SAMPLER)
    ptr = ctypes.c_void_p(0x300000)
    xs = (ctypes.c_void_p * 1)(ptr)
    st = L.track_calibrate(hL, hS, ctypes.byref(shp), 1, xs, xs, ptr, ctypes.byref(sc), None, None, None, None)
    assert st == track.E_INCOMPATIBLE
    st = L.track_calibrate(hL, hL, ctypes.byref(shp), 0, xs, xs, ptr, ctypes.byref(sc), None, None, None, None)
    assert st == track.E_INVALID
    bad = track.SamplerConfigC(0, 1, 3.0, 5.0, 1e-8)
    st = L.track_calibrate(hL, hL, ctypes.byref(shp), 1, xs, xs, ptr, ctypes.byref(bad), None, None, None, None)
    assert st == track.E_INVALID
    pol = (ctypes.c_uint8 * 8)(*([0] * 7 + [1]))
    st = L.track_sample(hL, None, pol, ctypes.byref(shp), ctypes.byref(sc), ptr, ptr, ptr, ptr, None)
    assert st == track.E_INVALID  # routes a step to a missing small model
    noguid = track.SamplerConfigC(8, 1, 3.0, 5.0, 1e-8)
    st = L.track_sample(hL, None, (ctypes.c_uint8 * 8)(), ctypes.byref(shp), ctypes.byref(noguid), ptr, ptr, None,
                        ptr, None)
    assert st == track.E_INVALID  # guidance without the negative prompt
    # scheduler choice: unknown solver, UniPC order outside 1..3
    for solver, order in [(2, 2), (-1, 2), (1, 0), (1, 4)]:
        bad = track.SamplerConfigC(8, 1, 3.0, 5.0, 1e-8, solver, order)
        st = L.track_sample(hL, None, (ctypes.c_uint8 * 8)(), ctypes.byref(shp), ctypes.byref(bad), ptr, ptr, ptr,
                            ptr, None)
        assert st == track.E_INVALID, (solver, order)
        st = L.track_calibrate(hL, hL, ctypes.byref(shp), 1, xs, xs, ptr, ctypes.byref(bad), None, None, None, None)
        assert st == track.E_INVALID, (solver, order)
    # band decomposition: latent beyond the kernels' bounds
    big = track.LatentShapeC(16, 4, 8, 2048, 16)
    st = L.track_calibrate_bands(hL, hL, ctypes.byref(big), 1, xs, xs, ptr, ctypes.byref(sc), None, None, None, None,
                                 None, None)
    assert st in (track.E_UNSUPPORTED, track.E_SHAPE)
    L.track_model_destroy(hL)
    L.track_model_destroy(hS)


def test_step_partial_count(L):
    assert L.track_step_partial_count(4) == 1
    assert L.track_step_partial_count(32760 * 64) == 1024
    assert L.track_rope_table_len(128, (ctypes.c_int32 * 3)(21, 30, 52)) == 21 * 22 + (30 + 52) * 21


def _oracle_unipc_weights(N, shift, order, i):
    """The fused-step weights of step i, read off the oracle's UniPC step by
    feeding basis vectors (the step is linear in its inputs)."""
    from oracle import unipc
    sig = sampler.sigmas(N, shift)
    S = unipc.UniPC(sig, order=order)
    rng = np.random.default_rng(1)
    for j in range(i):  # reach step i's state (history length, previous order)
        S.step(j, rng.standard_normal(6), rng.standard_normal(6))
    e = np.eye(6)
    if i >= 1:
        S.x_last = e[0]
        for k in range(1, 4):
            if i - k >= 0:
                S.m[i - k] = e[k]
    x_next = S.step(i, e[4], e[5])
    xc = S.x_last
    corr = i >= 1
    if corr:
        px = x_next[0] / xc[0]
        w = [xc[0], xc[1], xc[2], xc[3], xc[4], 1.0]
    else:
        px = None
        w = [0.0, 0.0, 0.0, 0.0, 0.0, 0.0]
    if corr:
        p_m = -(x_next[5] - px * xc[5]) / sig[i]
    else:
        p_m = -x_next[5] / sig[i]
        px = x_next[4] - p_m
    p_h0 = x_next[1] - px * xc[1]
    p_h1 = x_next[2] - px * xc[2]
    return np.array(w[:5]), px, p_m, p_h0, p_h1


def test_unipc_plan_matches_oracle(L):
    for N, shift in [(1, 1.0), (2, 3.0), (3, 5.0), (5, 3.0), (8, 3.0), (50, 5.0), (12, 1.0)]:
        for order in (1, 2, 3):
            for i in range(N):
                c = track.unipc_coefficients(N, shift, order, i)
                w, px, p_m, p_h0, p_h1 = _oracle_unipc_weights(N, shift, order, i)
                assert c[5] == (1.0 if i >= 1 else 0.0)
                got_c = np.array([c[0], c[1], c[2], c[3], c[4]])
                np.testing.assert_allclose(got_c, w, rtol=1e-10, atol=1e-12, err_msg=f"N={N} s={shift} q={order} i={i}")
                np.testing.assert_allclose([c[7], c[8], c[9], c[10]], [px, p_m, p_h0, p_h1], rtol=1e-10, atol=1e-12,
                                           err_msg=f"N={N} s={shift} q={order} i={i}")
                # the history counts say which terms exist
                assert (c[6] >= 1) == (abs(c[2]) > 0) and (c[6] >= 2) == (abs(c[3]) > 0)
                assert (c[11] >= 1) == (abs(c[9]) > 0) and (c[11] >= 2) == (abs(c[10]) > 0)


def test_unipc_coefficient_errors(L):
    with pytest.raises(track.TrackError):
        track.unipc_coefficients(5, 3.0, 4, 0)
    with pytest.raises(track.TrackError):
        track.unipc_coefficients(5, 3.0, 2, 5)
    with pytest.raises(track.TrackError):
        track.unipc_coefficients(0, 3.0, 2, 0)
    with pytest.raises(track.TrackError):
        track.unipc_coefficients(5, -1.0, 2, 0)


def test_attention_rejects_heads_beyond_4gib(L):
    """The bf16 kernel addresses one head's K and V^T through buffer resources
    with a 32-bit size field; larger heads are refused before any launch
    (profiling is off, so nothing touches a device)."""
    p = ctypes.c_void_p(1 << 20)  # aligned stand-in; never dereferenced
    E = track.DTYPE_BF16
    # K of one batch: Lk * ldk * 2 bytes = 150000 * 15360 * 2 > 4 GiB
    st = L.track_op_attention(E, 1, 40, 128, 64, 150000, p, 15360, p, 15360, p, 150016, p, 5120, None)
    assert st == track.E_SHAPE
    # V^T of one head: 128 * ldv * 2 bytes > 4 GiB
    st = L.track_op_attention(E, 1, 1, 128, 64, 64, p, 128, p, 128, p, 1 << 24, p, 128, None)
    assert st == track.E_SHAPE
    assert b"4 GiB" in L.track_last_error()


def test_norm_width_checks(L):
    """Widths the norm kernels do not cover are refused before any launch."""
    p = ctypes.c_void_p(1 << 20)  # aligned stand-in; never dereferenced
    F, E = track.DTYPE_F32, track.DTYPE_BF16
    assert L.track_op_layernorm(F, 10, 0, p, None, None, p, None) == track.E_SHAPE
    assert L.track_op_layernorm(F, 10, 6, p, None, None, p, None) == track.E_UNSUPPORTED
    assert L.track_op_layernorm(E, 10, 8196, p, None, None, p, None) == track.E_UNSUPPORTED
    assert L.track_op_layernorm(E, 10, 64, None, None, None, p, None) == track.E_INVALID
    assert L.track_op_layernorm(E, 10, 64, p, p, None, p, None) == track.E_INVALID  # scale without shift
    assert L.track_op_rmsnorm_rope(E, 10, 4, 6, p, 24, 0, p, None, None, None) == track.E_UNSUPPORTED
    assert L.track_op_rmsnorm_rope(E, 10, 66, 128, p, 66 * 128, 0, p, None, None, None) == track.E_UNSUPPORTED
    assert L.track_op_rmsnorm_rope(E, 10, 4, 128, p, 256, 0, p, None, None, None) == track.E_SHAPE  # ld < d


def test_linear_vt_argument_checks(L):
    """Shapes the transposed-output projection does not cover are refused before any launch."""
    p = ctypes.c_void_p(1 << 20)  # aligned stand-in; never dereferenced
    E, F = track.DTYPE_BF16, track.DTYPE_F32
    ok = dict(M=2 * 1000, N=512, K=320, lda=320, L=1000, ldv=1008)

    def call(dtype=E, **kw):
        a = dict(ok, **kw)
        return L.track_op_linear_vt(dtype, a["M"], a["N"], a["K"], p, a["lda"], p, p, a["L"], p, a["ldv"], None)

    assert call(F) == track.E_UNSUPPORTED
    assert call(N=384) == track.E_UNSUPPORTED          # N % 256
    assert call(L=120, M=240, ldv=120) == track.E_UNSUPPORTED  # L < 128
    assert call(L=1004, M=2008, ldv=1008) == track.E_UNSUPPORTED  # L % 8
    assert call(M=2001) == track.E_UNSUPPORTED          # M % L
    assert call(ldv=996) == track.E_SHAPE               # ldv < L
    assert call(lda=256) == track.E_SHAPE               # lda < K
    assert call(M=0) == track.E_SHAPE
    assert L.track_op_linear_vt(E, 2000, 512, 320, None, 320, p, p, 1000, p, 1008, None) == track.E_INVALID


def test_attention_log2q_is_bf16_only(L):
    """q given in log2 units is a bfloat16-path input: the float32 path refuses it before any launch."""
    p = ctypes.c_void_p(1 << 20)  # aligned stand-in; never dereferenced
    st = L.track_op_attention_log2q(track.DTYPE_F32, 1, 2, 64, 10, 10, p, 128, p, 128, p, 16, p, 128, None)
    assert st == track.E_INVALID


def test_mfma_stream_argument_checks(L):
    """The matrix-core stream refuses null pointers, misaligned operands and iteration counts out of range
    before any launch, and leaves the FLOP count untouched then."""
    p = ctypes.c_void_p(1 << 20)  # aligned stand-in; never dereferenced
    flop = ctypes.c_int64(-7)
    assert L.track_mfma_stream(p, 0, p, ctypes.byref(flop), None) == track.E_SHAPE
    assert L.track_mfma_stream(p, 1 << 31, p, ctypes.byref(flop), None) == track.E_SHAPE
    assert L.track_mfma_stream(ctypes.c_void_p((1 << 20) + 8), 1, p, ctypes.byref(flop), None) == track.E_INVALID
    assert L.track_mfma_stream(None, 1, p, ctypes.byref(flop), None) == track.E_INVALID
    assert L.track_mfma_stream(p, 1, None, ctypes.byref(flop), None) == track.E_INVALID
    assert L.track_mfma_stream(p, 1, p, None, None) == track.E_INVALID
    assert flop.value == -7


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """No CPU fallback: without the built library every entry point raises."""
    monkeypatch.setattr(track, "_lib", None)
    monkeypatch.setattr(track, "_LIB_PATH", str(tmp_path / "libtrack.so"))
    with pytest.raises(RuntimeError, match="missing"):
        track.lib()
    with pytest.raises(RuntimeError, match="missing"):
        track.route_policy(np.zeros(4), 2)


def test_failed_host_calls_leave_outputs_untouched(L):
    """A call that fails writes nothing: the output buffers keep their sentinel."""
    q = np.array([0.3, 0.1, 0.2])
    qp = q.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
    out = np.full(4, -7, dtype=np.int32)
    op = out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    assert L.track_route_policy(qp, 3, 4, op) == track.E_INVALID           # K > N
    assert np.all(out == -7)
    qn = np.array([0.1, np.nan, 0.2])
    assert L.track_route_policy(qn.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), 3, 1, op) != track.OK
    assert np.all(out == -7)
    kout = ctypes.c_int32(-7)
    assert L.track_route_threshold(qn.ctypes.data_as(ctypes.POINTER(ctypes.c_double)), 3, 0.5, op,
                                   ctypes.byref(kout)) != track.OK
    assert np.all(out == -7) and kout.value == -7
    assert L.track_route_baseline(7, 3, 1, 0, op) == track.E_INVALID       # unknown policy kind
    assert np.all(out == -7)
    coef = np.full(12, -7.0)
    assert L.track_unipc_coefficients(8, 5.0, 4, 0, coef.ctypes.data_as(ctypes.POINTER(ctypes.c_double))) != track.OK
    assert np.all(coef == -7.0)
