"""Teacher-forced parity of the benchmarked Wan-shaped models at their full depth.

The bfloat16 denoisers the benchmark times have 30 blocks of width 1536
(Wan-2.1-1.3B-shaped) and 40 blocks of width 5120 (Wan-2.1-14B-shaped).  Here
both run at that full depth and width, with the full 512 x 4096 text context,
on a reduced 16 x 4 x 16 x 16 latent (256 tokens: whole 8-token groups, so
the V projection writes V^T from its epilogue), and their guided velocity
(Eq. 1, w = 5) and conditional velocity are compared with the float64
oracle on the same float32 latent.  Each case runs twice on the device: with
the automatic kernel choice, and with every projection whose width the
256-wide tiles divide forced onto the persistent GEMM kernel that the
full-size step uses (at 512 rows the automatic choice takes the
register-staged kernel).

The oracle evaluates the network block by block through ``oracle.dit``,
with each block's parameters regenerated from the seeded recipe just before
it is needed (the whole 14B-shaped parameter set in float64 would not fit
comfortably in host memory), and every block is uploaded into the device
weight buffer from the same host arrays.  Latents follow the flow-matching
interpolant x = (1 - sigma) z_data + sigma z_noise of two seeded normal
fields at the sigma of the step, so the timestep embedding and the latent
statistics match the point of the trajectory.
"""
import concurrent.futures as cf
import os
import time

import numpy as np
import pytest

from gpu_helpers import dev, host, rel_l2, say
from oracle import dit, sampler
from paper_2609_30096_amd import synth, track

pytestmark = pytest.mark.gpu

TOL_BF16 = 2e-2
DEPTH_LATENT = synth.LatentShape(16, 4, 16, 16, 512)    # grid 4 x 8 x 8 = 256 tokens
GUIDANCE = 5.0


def _latent(sigma, key):
    z_data = synth.gen_normal((key, 0), (16, 4, 16, 16))
    z_noise = synth.gen_normal((key, 1), (16, 4, 16, 16))
    return ((1.0 - sigma) * z_data.astype(np.float64) + sigma * z_noise).astype(np.float32)


def oracle_and_weights(cfg, seed, sigma_steps, label, device="cuda"):
    """The float64 oracle's velocities per (latent, branch) and the device weight buffer, built block by block."""
    shape = DEPTH_LATENT
    sig = sampler.sigmas(50, 5.0)
    ts = [1000.0 * sig[k] for k in sigma_steps]
    xs = [_latent(sig[k], 7100 + k) for k in sigma_steps]
    cond = synth.gen_text(shape, cfg.text_dim, 0, synth.BF16)
    unc = synth.gen_null_text(shape, cfg.text_dim, synth.BF16)
    specs = synth.param_specs(cfg)
    table, total = track.weight_table(cfg)
    assert [n for n, _, _ in table] == [n for n, _, _ in specs]
    import torch
    buf = torch.empty(total, dtype=torch.uint8, device=device)
    bf = torch.bfloat16

    def upload(params):
        for i, (name, shp, off) in enumerate(table):
            if name in params:
                t = torch.from_numpy(params[name]).reshape(-1).to(device).to(bf)
                buf[off:off + 2 * t.numel()].view(bf).copy_(t)

    pt, ph, pw = cfg.patch
    grid = (shape.frames // pt, shape.height // ph, shape.width // pw)
    t_start = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=min(16, len(os.sched_getaffinity(0)))) as pool:
        nb = cfg.blocks
        glob = [i for i, (n, _, _) in enumerate(specs) if not n.startswith("blk")]
        G = synth.gen_param_set(cfg, seed, glob, pool)
        upload(G)
        P = {k: v.astype(np.float64) for k, v in G.items()}
        del G
        # oracle state per (latent, branch): residual stream X, shared modulation m and time embedding e
        X0 = [dit.linear(dit.patchify(x.astype(np.float64), cfg.patch), P["patch.w"], P["patch.b"]) for x in xs]
        tm = [dit.time_embedding(P, cfg, t) for t in ts]
        ctx = [dit.text_embedding(P, cond), dit.text_embedding(P, unc)]
        X = {(i, br): X0[i].copy() for i in range(len(xs)) for br in range(2)}
        f64 = {}
        for b in range(nb):
            idx = [i for i, (n, _, _) in enumerate(specs) if n.startswith(f"blk{b}.")]
            Pb = synth.gen_param_set(cfg, seed, idx, pool)
            upload(Pb)
            for name, a in Pb.items():   # float64 copies in reused buffers
                key = name.split(".", 1)[1]
                if key not in f64:
                    f64[key] = np.empty(a.shape, np.float64)
                np.copyto(f64[key], a)
            view = {f"blk{b}.{k}": v for k, v in f64.items()}
            for (i, br), Xs in X.items():
                X[(i, br)] = dit.block(view, cfg, b, Xs, ctx[br], tm[i][1], grid)
            if b % 5 == 4 or b == nb - 1:
                say(f"  {label}: oracle through block {b + 1}/{nb} ({time.perf_counter() - t_start:.0f} s)")
        del f64
    ref = {}
    for (i, br), Xs in X.items():
        out = dit.head(P, Xs, tm[i][0])
        ref[(i, br)] = dit.unpatchify(out, shape.channels, shape.frames, shape.height, shape.width, cfg.patch)
    return buf, ref, xs, ts, cond, unc


def _full_depth(cfg, seed, sigma_steps, label):
    import torch
    shape = DEPTH_LATENT
    buf, ref, xs, ts, cond, unc = oracle_and_weights(cfg, seed, sigma_steps, label)
    nb = cfg.blocks
    model = track.Model(cfg, buf)
    dc, du = dev(cond, synth.BF16), dev(unc, synth.BF16)
    worst = 0.0
    for forced in ("0", "4"):
        prev = os.environ.get("TRACK_GEMM_CFG")
        os.environ["TRACK_GEMM_CFG"] = forced
        try:
            for i, (x, t) in enumerate(zip(xs, ts)):
                dx = dev(x)
                got_g = host(track.dit_forward(model, shape, dx, t, dc, du, GUIDANCE))
                got_c = host(track.dit_forward(model, shape, dx, t, dc))
                e_g = rel_l2(got_g, sampler.guided(ref[(i, 0)], ref[(i, 1)], GUIDANCE))
                e_c = rel_l2(got_c, ref[(i, 0)])
                kern = "persistent GEMMs" if forced == "4" else "automatic kernels"
                say(f"  {label}, {nb} blocks, t = {t:.1f} ({kern}): guided relative L2 {e_g:.3e}, "
                    f"unguided {e_c:.3e}")
                worst = max(worst, e_g, e_c)
        finally:
            if prev is None:
                os.environ.pop("TRACK_GEMM_CFG", None)
            else:
                os.environ["TRACK_GEMM_CFG"] = prev
    model.close()
    del buf
    torch.cuda.empty_cache()
    assert worst < TOL_BF16, worst


@pytest.mark.timeout(900)
def test_wan13b_full_depth_teacher_forced():
    """30 blocks x 1536: sigma = 1 (the first step of the 50-step, shift-5 schedule) and mid-trajectory."""
    say("wan 1.3B full depth")
    _full_depth(synth.WAN_1_3B, synth.SEED_SMALL, [0, 25], "wan 1.3B")


@pytest.mark.timeout(900)
def test_wan14b_full_depth_teacher_forced():
    """40 blocks x 5120 at a mid-trajectory sigma."""
    say("wan 14B full depth")
    _full_depth(synth.WAN_14B, synth.SEED_LARGE, [25], "wan 14B")
