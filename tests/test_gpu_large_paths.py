"""Blocks above 4096 elements take two routes through the select: the
threshold and apply passes (microadam_step, whose handle holds the per-block
threshold records) and the multi-wave select that holds a whole block
(microadam_step_noalloc, which allocates nothing and so keeps no records).
Both must give the same bits: parameters and the whole state buffer (codes,
bucket pairs, window rows and segment tables) after every step."""
import math

import pytest
import torch

import paper_2405_15593_amd as ma
from paper_2405_15593_amd import workloads as wl

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("grad_dist,steps", [("student_t2_snapped64", 24), ("student_t4", 6)])
def test_threshold_route_matches_multiwave_select(grad_dist, steps):
    """The flat workload's block shape: B_d = 65536, k = 3277, m = 20, B_q =
    128, two full blocks and a 12,032-element tail (whole sub-blocks empty);
    Student-t(2) snapped to 64 magnitudes puts tie groups at the threshold
    (24 steps: the window wraps), Student-t(4) does not."""
    dev = torch.device("cuda")
    numels = [65536 * 2 + 12032]
    cfg = ma.make_config(density=0.05, window=20, ef_bucket=128, topk_block=65536, lr=1e-4)
    bf = torch.bfloat16
    params_a = [wl.draw(n, "normal", 0.02, 3 + j, dev, bf) for j, n in enumerate(numels)]
    params_b = [p.clone() for p in params_a]
    opt = ma.MicroAdam(params_a, cfg)
    nbytes = ma.microadam_state_bytes(cfg, numels)
    raw = torch.zeros(nbytes + 256, dtype=torch.uint8, device=dev)
    off = (-raw.data_ptr()) % 256
    state_b = raw[off:off + nbytes]
    stream = torch.cuda.current_stream().cuda_stream
    for t in range(1, steps + 1):
        print(f"[large-paths] {grad_dist} step {t}", flush=True)
        grads = [wl.draw(n, grad_dist, 1e-3, wl.grad_seed(t, j, 9), dev, bf) for j, n in enumerate(numels)]
        opt.step(grads)
        assert opt.step_kernels == 4  # threshold, apply, multi-wave for the blocks left, update
        ma.microadam_step_noalloc(cfg, numels, ma.MICROADAM_BF16, ma.MICROADAM_BF16, state_b.data_ptr(), nbytes,
                                  t, [p.data_ptr() for p in params_b], [g.data_ptr() for g in grads], math.nan,
                                  stream)
        torch.cuda.synchronize()
        assert torch.equal(opt.state_view, state_b), f"state buffers differ after step {t}"
        for a, b in zip(params_a, params_b):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"params differ after step {t}"
    opt.close()


def test_many_unsettled_blocks_through_the_list():
    """A constant gradient over 301 blocks of 8192 (and a ragged tail): every
    key ties, so the threshold pass settles no full block and the multi-wave
    select works through a list longer than its 256 workgroups (two rounds
    per workgroup).  The result matches the multi-wave select run over every
    block, bit for bit, at each of 3 steps."""
    dev = torch.device("cuda")
    numels = [8192 * 301 + 5000]
    cfg = ma.make_config(density=0.02, window=3, ef_bucket=64, topk_block=8192, lr=1e-4)
    bf = torch.bfloat16
    params_a = [wl.draw(n, "normal", 0.02, 11 + j, dev, bf) for j, n in enumerate(numels)]
    params_b = [p.clone() for p in params_a]
    opt = ma.MicroAdam(params_a, cfg)
    nbytes = ma.microadam_state_bytes(cfg, numels)
    raw = torch.zeros(nbytes + 256, dtype=torch.uint8, device=dev)
    off = (-raw.data_ptr()) % 256
    state_b = raw[off:off + nbytes]
    stream = torch.cuda.current_stream().cuda_stream
    for t in range(1, 4):
        print(f"[large-paths] constant gradient, 301 blocks, step {t}", flush=True)
        grads = [wl.draw(n, "constant", 0.25, wl.grad_seed(t, j, 9), dev, bf) for j, n in enumerate(numels)]
        opt.step(grads)
        assert opt.step_kernels == 4
        ma.microadam_step_noalloc(cfg, numels, ma.MICROADAM_BF16, ma.MICROADAM_BF16, state_b.data_ptr(), nbytes,
                                  t, [p.data_ptr() for p in params_b], [g.data_ptr() for g in grads], math.nan,
                                  stream)
        torch.cuda.synchronize()
        assert torch.equal(opt.state_view, state_b), f"state buffers differ after step {t}"
        for a, b in zip(params_a, params_b):
            assert torch.equal(a.view(torch.int16), b.view(torch.int16)), f"params differ after step {t}"
    opt.close()
