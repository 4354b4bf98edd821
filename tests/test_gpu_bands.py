"""GPU parity of the band-decomposition kernels (csrc/bands.hip) against the
oracle's numpy FFTs (oracle/bands.py), through the C ABI's component op."""
import math

import numpy as np
import pytest

from oracle import bands, dit
from paper_2609_30096_amd import synth

from gpu_helpers import dev, normal, say

pytestmark = pytest.mark.gpu


def _guided(v, B, w):
    return v[1] + w * (v[0] - v[1]) if B == 2 else v[0]


@pytest.mark.parametrize("C,F,H,W,patch,B", [
    (4, 5, 12, 20, (1, 2, 2), 2),
    (3, 7, 6, 10, (1, 2, 2), 1),
    (2, 6, 8, 8, (2, 2, 2), 2),
    (1, 1, 2, 2, (1, 2, 2), 2),
    (2, 3, 34, 38, (1, 2, 2), 2),      # W > 32: two column blocks, the second ragged
    (16, 21, 60, 104, (1, 2, 2), 2),   # the Wan 81 x 480 x 832 latent
])
def test_band_energy_matches_oracle(C, F, H, W, patch, B):
    import torch
    from paper_2609_30096_amd import track
    say(f"band energy C={C} F={F} H={H} W={W} patch={patch} B={B}")
    shape = synth.LatentShape(C, F, H, W, 16)
    L = shape.tokens(patch)
    P = C * math.prod(patch)
    key = 7000 + C + F + H + W + B
    vL = normal((key, 1), (B, L, P))
    vS = vL + 0.3 * normal((key, 2), (B, L, P))
    w = 5.0
    ws = torch.empty(track.band_workspace_bytes(shape, patch), dtype=torch.uint8, device="cuda")
    got = track.op_band_energy(shape, B, w, dev(vL), dev(vS), ws, patch)
    d_tok = _guided(vS.astype(np.float64), B, w) - _guided(vL.astype(np.float64), B, w)
    sp, tp = bands.band_energies(dit.unpatchify(d_tok, C, F, H, W, patch))
    ref = np.concatenate([sp, tp])
    tot = float(sp.sum())
    say(f"  got {np.round(got, 3)}\n  ref {np.round(ref, 3)}")
    assert np.all(np.abs(got - ref) <= 2e-5 * tot + 2e-5 * np.abs(ref)), (got, ref)
    # Parseval on the device: both triples sum to ||d||^2
    assert got[:3].sum() == pytest.approx(tot, rel=1e-5)
    assert got[3:].sum() == pytest.approx(tot, rel=1e-5)
    # a second call on the same workspace gives the same bits
    again = track.op_band_energy(shape, B, w, dev(vL), dev(vS), ws, patch)
    np.testing.assert_array_equal(got, again)


def test_band_energy_argument_checks():
    import torch
    from paper_2609_30096_amd import track
    shape = synth.LatentShape(2, 3, 4, 4, 16)
    v = torch.zeros(2 * 2 * 3 * 4 * 4, device="cuda")
    ws = torch.empty(track.band_workspace_bytes(shape), dtype=torch.uint8, device="cuda")
    with pytest.raises(track.TrackError):  # workspace too small
        track.op_band_energy(shape, 2, 1.0, v, v, ws[:256])
    with pytest.raises(track.TrackError):  # batch 3
        track.op_band_energy(shape, 3, 1.0, v, v, ws)
    with pytest.raises(track.TrackError):  # latent not divisible by the patch
        track.op_band_energy(synth.LatentShape(2, 3, 5, 4, 16), 2, 1.0, v, v, ws)
    assert track.band_workspace_bytes(synth.LatentShape(2, 3, 300, 4, 16)) == 0  # H beyond the kernels' bound
