"""Oracle: a plain, slow, float64 CPU statement of what the GPU path computes.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or
calls this package; only the tests, the smoke check and the benchmark's CPU
baseline leg do.  It shares no code with the GPU path: it takes plain numpy
arrays (parameters, latents, text embeddings) and returns numpy arrays.

Modules
  dit      -- the video DiT denoiser f_m(x, t, c) that every denoising step
              evaluates (patchify, adaLN blocks with 3D-RoPE self-attention,
              text cross-attention and a GELU MLP, modulated head).
  sampler  -- classifier-free guidance (Eq. 1), the flow-matching Euler
              scheduler (Eq. 2), routed sampling (Eq. 3), reference-trajectory
              calibration (Sec. 3.2.1), relative disagreement (Eq. 4), the mean
              score (Eq. 5), the box LP and its threshold solution (Eqs. 6-7),
              top-K routing (Sec. 3.2.3) and the equal-budget baselines.
  unipc    -- the UniPC multistep scheduler (Eq. 2 with a history h_i): the
              predictor/corrector weights and the step, in the data-prediction
              form on the flow-matching sigma table.
  bands    -- the spatial and temporal frequency-band split of the disagreement
              (Sec. "Frequency Analysis") with orthonormal DFTs.

Pins (tests/test_oracle_*.py, run without a GPU) tie every function here to
something other than itself: textbook or library routines (torch.nn.functional
in float64, conv3d for patch embedding, complex multiplication for RoPE), closed
forms (the shifted sigma table, Euler on constant and point-mass velocity
fields), invariants and brute force on tiny inputs.

Parity unpinned: the denoiser's architecture is not defined by the paper (it
only names the Wan 2.1 / Cosmos families).  The block layout here is a reading
of the Wan 2.1 design; its composition is pinned against an independent
torch.nn.functional build of the same reading, not against values the paper
prints (it prints none).
"""
