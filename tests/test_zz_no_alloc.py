"""track_op_step_noalloc: the calibration step with its partial sums in the
library's static device scratch, against track_op_step with a caller
workspace, through the C ABI.  Two calls in a row, the second on a smaller
latent, both bit for bit (the same kernels in the same order)."""
import numpy as np
import pytest

from gpu_helpers import normal, say
from paper_2609_30096_amd import track

pytestmark = pytest.mark.gpu


def _pair_of_runs(n, B, w, dsigma, key):
    import torch
    vL = torch.from_numpy(normal((key, 0), (B * n,))).cuda()
    vS = torch.from_numpy(normal((key, 1), (B * n,))).cuda()
    x0 = torch.from_numpy(normal((key, 2), (n,))).cuda()
    # with a caller workspace
    xa = x0.clone()
    part = torch.empty(2 * track.step_partial_count(n), dtype=torch.float64, device="cuda")
    ra = torch.zeros(1, dtype=torch.float64, device="cuda")
    track.op_step(n, B, w, dsigma, vL, xa, vel_S=vS, partial=part, r_out=ra)
    # without one
    xb = x0.clone()
    rb = torch.full((1,), -1.0, dtype=torch.float64, device="cuda")
    track.op_step_noalloc(n, B, w, dsigma, vL, xb, vel_S=vS, r_out=rb)
    # sample mode (no partials) as well
    xc, xd = x0.clone(), x0.clone()
    track.op_step(n, B, w, dsigma, vL, xc)
    track.op_step_noalloc(n, B, w, dsigma, vL, xd)
    torch.cuda.synchronize()
    return ra.item(), rb.item(), torch.equal(xa, xb), torch.equal(xc, xd), torch.equal(xa, xc)


def test_step_noalloc_matches_workspace_step_twice():
    # 16 x 21 x 60 x 104 latent (CFG batch 2, the full partial count), then a smaller ragged one
    for n, B in ((16 * 21 * 60 * 104, 2), (16 * 3 * 10 * 14, 1)):
        say(f"step_noalloc n={n} B={B}")
        ra, rb, same_x, same_x_sample, same_update = _pair_of_runs(n, B, 5.0, -0.0371, 8800 + B)
        assert ra == rb, (n, B, ra, rb)
        assert np.isfinite(ra) and ra > 0
        assert same_x and same_x_sample and same_update


def test_step_noalloc_rejects_missing_r_out():
    import torch
    v = torch.zeros(8, device="cuda")
    x = torch.zeros(4, device="cuda")
    with pytest.raises(track.TrackError):
        track.op_step_noalloc(4, 2, 5.0, -0.1, v, x, vel_S=v, r_out=None)
