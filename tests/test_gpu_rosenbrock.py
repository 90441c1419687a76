"""MicroAdam through the library on the paper's Fig. 1 problem (the 2-D
Rosenbrock function from (-1/2, 1)): one 2-element tensor in a Top-K block of
16 with density 1/2, so one coordinate is kept per step.  Every step is
checked against the oracle started from the same parameters and gradient."""
import numpy as np
import pytest
import torch

import oracle
from paper_2405_15593_amd import MICROADAM_F32, MicroAdam, make_config
from paper_2405_15593_amd import rosenbrock as rb

pytestmark = pytest.mark.gpu


def test_rosenbrock_trajectory_matches_oracle():
    print("[rosenbrock] 400 steps, library vs oracle", flush=True)
    lr, window, steps = 1e-2, 10, 400
    p = torch.tensor(rb.START, dtype=torch.float32, device="cuda")
    opt = MicroAdam([p], make_config(density=0.5, window=window, ef_bucket=16, topk_block=16, lr=lr,
                                     window_value_dtype=MICROADAM_F32))
    st = oracle.default().tensor(2, block=16, bucket=16, density=0.5, window=window, value_bf16=False)
    moved = 0
    for t in range(1, steps + 1):
        g = rb.gradient(p)
        before = p.cpu().numpy().copy()
        opt.step([g])
        got = p.cpu().numpy()
        ref = before.copy()
        st.step(ref, g.cpu().numpy().astype(np.float32), t, lr)
        assert np.all(np.abs(got.astype(np.float64) - ref) <= 1e-5 * np.maximum(np.abs(ref), lr)), (t, got, ref)
        moved += int(np.any(got != before))
    opt.close()
    assert moved > steps // 2


def test_rosenbrock_summary_runs():
    traj = rb.run_microadam(200, 1e-2)
    s = rb.summary(traj, rb.run_adam(200, 1e-2))
    assert traj.shape == (201, 2) and np.all(np.isfinite(traj))
    assert s["path_length"] > 0
