"""Per-kernel timing of the denoiser step at the Wan-2.1 shapes, through the C ABI.

    python -m paper_2609_30096_amd.kernel_bench [--model 1.3b|14b] [--tokens 32760] [--iters N] [--only NAME]
                                                [--reference] [--cold] [--power SECONDS]

Each kernel is launched on torch's current stream and timed with HIP events
around `iters` back-to-back launches (after one warm launch).  Reports
algorithmic TFLOP/s (2MNK per GEMM, 4 B H Lq Lk dh per attention) or GB/s
(algorithmic bytes read + written) and the fraction of the MI355X peak
(bf16 dense MFMA 2.5 PFLOP/s, HBM 8 TB/s).  The library's plain streaming
kernels (copy, read and write of 1 GiB: hbm_copy_1GiB, hbm_read_1GiB,
hbm_write_1GiB; hbm_copy_inplace_1GiB for in-place kernels) are the practical ceiling for the memory-bound kernels and
the reference for scaling rocprofv3's FETCH_SIZE / WRITE_SIZE counters;
the library's MFMA stream (mfma_stream: independent bf16 32x32x16 chains on
every CU, on random operands; mfma_stream_zeros on zeros) is the sustained
matrix-core ceiling for the MFMA-bound ones;
torch's device copy (copy_1GiB) is kept for comparison.  Inputs are seeded random
tensors; only timing is measured here (parity lives in tests/).  --cold also
times each memory-bound kernel one launch at a time after a 1 GiB write has
flushed the caches (median), since the step kernels' inputs (< 256 MB) are
otherwise served partly from the Infinity Cache.  --power reads the socket power
and graphics clock (amd-smi) while each kernel runs back to back: the
MFMA-bound kernels run at the board's power limit and below the 2.4 GHz of the
peak figures.

attn_self and attn_cross take q as the forward's RMSNorm writes it, times
log2(e) / sqrt(dh) (track_op_attention_log2q); attn_self_q_unscaled times the
same kernel on unscaled q (track_op_attention, one FMA per probability).

--reference adds, for context only, the vendor libraries at the same shapes:
hipBLASLt through torch.nn.functional.linear (bias epilogue only) for the four
projection GEMMs, and torch's scaled_dot_product_attention (flash and
memory-efficient backends) for the self-attention.  The library never calls
either; they are a yardstick for the hand-written kernels.
"""
from __future__ import annotations

import argparse
import json
import sys

PEAK_TFLOPS = 2500.0
PEAK_GBS = 8000.0


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--model", choices=["1.3b", "14b"], default="1.3b")
    ap.add_argument("--tokens", type=int, default=32760)
    ap.add_argument("--batch", type=int, default=2)
    ap.add_argument("--iters", type=int, default=10)
    ap.add_argument("--only", default=None, help="comma-separated kernel names")
    ap.add_argument("--reference", action="store_true", help="also time vendor-library equivalents (context)")
    ap.add_argument("--cold", action="store_true",
                    help="also time memory-bound kernels one launch at a time after evicting the caches")
    ap.add_argument("--power", type=float, default=0.0, metavar="SECONDS",
                    help="also run each kernel back to back for SECONDS while amd-smi samples the socket power "
                         "and graphics clock (median of the samples after the first two)")
    a = ap.parse_args()

    import torch

    from . import synth, track

    torch.manual_seed(0)
    cfg = synth.WAN_1_3B if a.model == "1.3b" else synth.WAN_14B
    B, L, Lc = a.batch, a.tokens, 512
    d, H, dh, f = cfg.dim, cfg.heads, cfg.head_dim, cfg.ffn_dim
    M = B * L
    Lpad = (L + 63) // 64 * 64
    bf = torch.bfloat16
    dev = "cuda"
    BF = track.DTYPE_BF16

    def rnd(*shape, dtype=bf, scale=1.0):
        return (torch.randn(*shape, device=dev, dtype=torch.float32) * scale).to(dtype)

    qkv = rnd(M, 3 * d)
    vt = torch.zeros(B, H, dh, Lpad, device=dev, dtype=bf)
    vt[..., :L] = rnd(B, H, dh, L)
    kvc = rnd(B * Lc, 2 * d)
    vct = rnd(B, H, dh, Lc)
    ao = torch.empty(M, d, device=dev, dtype=bf)
    y = rnd(M, d)
    X = rnd(M, d, dtype=torch.float32)
    hid = rnd(M, f)
    gate = rnd(d, dtype=torch.float32)
    sc = rnd(d, dtype=torch.float32, scale=0.1)
    sh = rnd(d, dtype=torch.float32, scale=0.1)
    g = rnd(d, scale=0.1) + 1
    W = {n: rnd(N, K, scale=0.02) for n, N, K in [("qkv", 3 * d, d), ("o", d, d), ("ffn1", f, d), ("ffn2", d, f),
                                                 ("kv", 2 * d, d)]}
    bias = {n: rnd(W[n].shape[0], scale=0.02) for n in W}
    outs = {"qkv": torch.empty(M, 3 * d, device=dev, dtype=bf), "ffn1": torch.empty(M, f, device=dev, dtype=bf),
            "kv": torch.empty(B * Lc, 2 * d, device=dev, dtype=bf), "cq": torch.empty(M, d, device=dev, dtype=bf)}
    n_step = L * 64
    vel = rnd(B * n_step, dtype=torch.float32)
    velS = rnd(B * n_step, dtype=torch.float32)
    xl = rnd(n_step, dtype=torch.float32)
    part = torch.empty(2 * track.step_partial_count(n_step), device=dev, dtype=torch.float64)
    rout = torch.empty(1, device=dev, dtype=torch.float64)
    cp_src = torch.empty(1 << 30, device=dev, dtype=torch.uint8).fill_(1)
    cp_dst = torch.empty_like(cp_src)
    sink = torch.zeros(4, device=dev, dtype=torch.int32)
    temb = rnd(B * Lc, d)

    k_self = qkv[:, d:]
    # q as the forward's RMSNorm writes it, times log2(e) / sqrt(dh) (track_op_attention_log2q)
    q_l2 = (qkv[:, :d].float() * (1.4426950408889634 / dh ** 0.5)).to(bf).contiguous()
    cases = {
        # name: (launch, flops, bytes)
        "attn_self": (lambda: track.op_attention(BF, B, H, dh, L, L, q_l2, d, k_self, 3 * d, vt, Lpad, ao, d,
                                                 q_log2=True),
                      4 * B * H * L * L * dh, None),
        "attn_cross": (lambda: track.op_attention(BF, B, H, dh, L, Lc, q_l2, d, kvc, 2 * d, vct, Lc, ao, d,
                                                  q_log2=True),
                       4 * B * H * L * Lc * dh, None),
        # the same with q unscaled (track_op_attention: one FMA per probability)
        "attn_self_q_unscaled": (lambda: track.op_attention(BF, B, H, dh, L, L, qkv, 3 * d, k_self, 3 * d, vt, Lpad,
                                                            ao, d),
                                 4 * B * H * L * L * dh, None),
        "gemm_qkv": (lambda: track.op_linear(BF, track.EPI_BIAS, y, W["qkv"], bias["qkv"], outs["qkv"]),
                     2 * M * 3 * d * d, None),
        # the forward's split of the QKV projection: q, k to the row-major buffer, v transposed to V^T
        "gemm_qk": (lambda: track.op_linear(BF, track.EPI_BIAS, y, W["qkv"][:2 * d], bias["qkv"][:2 * d], outs["qkv"],
                                            N=2 * d), 2 * M * 2 * d * d, None),
        "gemm_v_vt": (lambda: track.op_linear_vt(y, W["qkv"][2 * d:], bias["qkv"][2 * d:], L, vt, Lpad),
                      2 * M * d * d, None),
        "gemm_o_gate_resid": (lambda: track.op_linear(BF, track.EPI_GATE_RESID, y, W["o"], bias["o"], X, gate=gate),
                              2 * M * d * d, None),
        "gemm_cross_q": (lambda: track.op_linear(BF, track.EPI_BIAS, y, W["o"], bias["o"], outs["cq"]),
                         2 * M * d * d, None),
        "gemm_ffn1_gelu": (lambda: track.op_linear(BF, track.EPI_BIAS_GELU, y, W["ffn1"], bias["ffn1"], outs["ffn1"]),
                           2 * M * f * d, None),
        "gemm_ffn2_gate_resid": (lambda: track.op_linear(BF, track.EPI_GATE_RESID, hid, W["ffn2"], bias["ffn2"], X,
                                                         gate=gate), 2 * M * d * f, None),
        "gemm_text_kv": (lambda: track.op_linear(BF, track.EPI_BIAS, temb, W["kv"], bias["kv"], outs["kv"]),
                         2 * B * Lc * 2 * d * d, None),
        "layernorm_mod": (lambda: track.op_layernorm(BF, X, y, sc, sh), None, M * d * (4 + 2)),
        "rmsnorm_rope_q": (lambda: track.op_rmsnorm_rope(BF, qkv, H, dh, g, col0=0, grid=(21, 30, 52) if L == 32760
                                                         else (21, 45, 80), rows=M), None, M * d * (2 + 2)),
        "step_sample": (lambda: track.op_step(n_step, B, 5.0, -0.02, vel, xl), None, n_step * (4 * B + 8)),
        "step_calibrate": (lambda: track.op_step(n_step, B, 5.0, -0.02, vel, xl, vel_S=velS, partial=part,
                                                 r_out=rout), None, n_step * (8 * B + 8)),
        "rmsnorm_rope_qk": (lambda: track.op_rmsnorm_rope_qk(BF, qkv, H, dh, g, g, col0=0,
                                                             grid=(21, 30, 52) if L == 32760 else (21, 45, 80), rows=M),
                            None, 2 * M * d * (2 + 2)),
        # the practical HBM ceiling: the library's plain streaming kernels over 1 GiB
        "hbm_copy_1GiB": (lambda: track.hbm_stream(track.HBM_COPY, cp_src, cp_dst, 1 << 30), None, 2 * (1 << 30)),
        "hbm_copy_inplace_1GiB": (lambda: track.hbm_stream(track.HBM_COPY, cp_src, cp_src, 1 << 30), None, 2 * (1 << 30)),
        "hbm_read_1GiB": (lambda: track.hbm_stream(track.HBM_READ, cp_src, sink, 1 << 30), None, 1 << 30),
        "hbm_write_1GiB": (lambda: track.hbm_stream(track.HBM_WRITE, None, cp_dst, 1 << 30), None, 1 << 30),
        "copy_1GiB": (lambda: cp_dst.copy_(cp_src), None, 2 * (1 << 30)),
    }
    # the sustained matrix-core ceiling: the library's MFMA stream on every CU,
    # on normal random bf16 operands like the kernels' inputs, and on zeros
    # (the clock under matrix work depends on the operand bits)
    mf_iters = 500000
    mf_flop = torch.cuda.get_device_properties(0).multi_processor_count * 4 * mf_iters * 8 * (2 * 32 * 32 * 16)
    mf_ops = rnd(32768)
    mf_zero = torch.zeros(32768, device=dev, dtype=bf)
    cases["mfma_stream"] = (lambda: track.mfma_stream(mf_ops, mf_iters, sink), mf_flop, None)
    cases["mfma_stream_zeros"] = (lambda: track.mfma_stream(mf_zero, mf_iters, sink), mf_flop, None)
    if L == 32760:
        # band decomposition of the calibration difference on the 16 x 21 x 60 x 104
        # latent (synchronous op: includes the 48-byte copy of the result)
        bshape = synth.LatentShape(16, 21, 60, 104, Lc)
        bws = torch.empty(track.band_workspace_bytes(bshape), device=dev, dtype=torch.uint8)
        # both passes read both models' branches; the row pass writes and the
        # column pass reads the complex intermediate
        cases["band_energy"] = (lambda: track.op_band_energy(bshape, B, 5.0, vel, velS, bws), None,
                                2 * (2 * B * n_step * 4) + 2 * n_step * 8)
    # a mid-trajectory order-2 UniPC step (corrector with one history term,
    # predictor with one): reads x, x_last, two stored predictions and the
    # velocities, writes x, x_last and the new prediction
    ucoef = track.unipc_coefficients(50, 5.0, 2, 10)
    xlast = rnd(n_step, dtype=torch.float32)
    hist = [rnd(n_step, dtype=torch.float32) for _ in range(2)]
    mout = torch.empty(n_step, device=dev, dtype=torch.float32)
    cases["unipc_step_sample"] = (lambda: track.op_unipc_step(n_step, B, 5.0, 0.5, ucoef, vel, xl, xlast, mout,
                                                              h0=hist[0], h1=hist[1]), None,
                                  n_step * (4 * B + 4 * 4 + 3 * 4))
    cases["unipc_step_calibrate"] = (lambda: track.op_unipc_step(n_step, B, 5.0, 0.5, ucoef, vel, xl, xlast, mout,
                                                                 h0=hist[0], h1=hist[1], vel_S=velS, partial=part,
                                                                 r_out=rout), None,
                                     n_step * (8 * B + 4 * 4 + 3 * 4))
    only = set(a.only.split(",")) if a.only else None
    results = []
    for name, (fn, flops, nbytes) in cases.items():
        if only and name not in only:
            continue
        print(f"[kernel_bench] {name}", file=sys.stderr, flush=True)
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(a.iters):
            fn()
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / a.iters
        r = {"kernel": name, "model": a.model, "tokens": L, "batch": B, "ms": round(ms, 4)}
        if flops:
            r["tflops"] = round(flops / ms / 1e9, 1)
            r["frac_peak"] = round(flops / ms / 1e9 / PEAK_TFLOPS, 4)
        else:
            r["gbs"] = round(nbytes / ms / 1e6, 1)
            r["frac_peak"] = round(nbytes / ms / 1e6 / PEAK_GBS, 4)
            if a.cold:
                ms_cold = _time_cold(torch, fn, max(5, a.iters))
                r["ms_cold"] = round(ms_cold, 4)
                r["gbs_cold"] = round(nbytes / ms_cold / 1e6, 1)
        if a.power > 0:
            r.update(_power(torch, fn, a.power))
        results.append(r)
        print(json.dumps(r), flush=True)
    if a.reference:
        results += _reference(a, torch, B, L, cfg)
    return results


def _time(torch, fn, iters):
    fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(iters):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / iters


def _power(torch, fn, seconds):
    """Socket power (W) and graphics clock (MHz) read by `amd-smi metric -p -c` about once a second
    while fn runs back to back; the first two samples (ramp-up) are dropped."""
    import subprocess
    import threading
    import time

    samples, stop = [], []

    def sample():
        while not stop:
            try:
                out = subprocess.run(["amd-smi", "metric", "-p", "-c", "--json"], capture_output=True, text=True,
                                     timeout=10).stdout
                g = json.loads(out)
                g = g["gpu_data"][0] if isinstance(g, dict) else g[0]
                samples.append((float(g["power"]["socket_power"]["value"]), float(g["clock"]["gfx_0"]["clk"]["value"])))
            except (OSError, ValueError, KeyError, IndexError, TypeError, subprocess.SubprocessError):
                pass
            time.sleep(0.7)

    th = threading.Thread(target=sample)
    th.start()
    t0 = time.time()
    while time.time() - t0 < seconds:
        for _ in range(5):
            fn()
        torch.cuda.synchronize()
    stop.append(True)
    th.join()
    kept = samples[2:]
    if not kept:
        return {"power_samples": 0}
    pw = sorted(x[0] for x in kept)
    ck = sorted(x[1] for x in kept)
    return {"power_samples": len(kept), "socket_power_w": pw[len(pw) // 2], "gfx_clock_mhz": ck[len(ck) // 2]}


_FLUSH = []


def _time_cold(torch, fn, reps):
    """Median time of single launches, each after 1 GiB of writes has evicted
    the L2 caches and the 256 MB Infinity Cache (so the inputs come from HBM)."""
    if not _FLUSH:
        _FLUSH.append(torch.empty(1 << 28, device="cuda", dtype=torch.float32))
    times = []
    for _ in range(reps):
        _FLUSH[0].fill_(1.0)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    times.sort()
    return times[len(times) // 2]


def _reference(a, torch, B, L, cfg):
    """Vendor-library timings at the step shapes (context, not used by the library)."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    d, H, dh, f = cfg.dim, cfg.heads, cfg.head_dim, cfg.ffn_dim
    M = B * L
    bf = torch.bfloat16
    out = []
    for name, N, K in [("ref_linear_qkv", 3 * d, d), ("ref_linear_o", d, d), ("ref_linear_ffn1", f, d),
                       ("ref_linear_ffn2", d, f)]:
        x = torch.randn(M, K, device="cuda", dtype=bf)
        w = torch.randn(N, K, device="cuda", dtype=bf) * 0.02
        bias = torch.randn(N, device="cuda", dtype=bf) * 0.02
        ms = _time(torch, lambda: torch.nn.functional.linear(x, w, bias), a.iters)
        r = {"kernel": name, "library": "hipBLASLt (torch linear)", "model": a.model, "ms": round(ms, 4),
             "tflops": round(2 * M * N * K / ms / 1e9, 1)}
        out.append(r)
        print(json.dumps(r), flush=True)
        del x, w, bias
    q = torch.randn(B, H, L, dh, device="cuda", dtype=bf)
    k = torch.randn_like(q)
    v = torch.randn_like(q)
    for be in (SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION):
        with sdpa_kernel([be]):
            ms = _time(torch, lambda: torch.nn.functional.scaled_dot_product_attention(q, k, v), max(1, a.iters // 3))
        r = {"kernel": "ref_sdpa_self", "library": f"torch sdpa {be.name}", "model": a.model, "ms": round(ms, 4),
             "tflops": round(4 * B * H * L * L * dh / ms / 1e9, 1)}
        out.append(r)
        print(json.dumps(r), flush=True)
    return out


if __name__ == "__main__":
    main()
