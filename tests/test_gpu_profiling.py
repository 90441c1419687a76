"""Kernel timers of the library: per-step durations and the totals that
bench.py reads once after its timed steps."""
import pytest
import torch

pytestmark = pytest.mark.gpu


def test_kernel_times_total_over_the_event_ring():
    import paper_2405_15593_amd as ma
    from paper_2405_15593_amd import workloads as wl
    dev = torch.device("cuda:0")
    w = wl.WORKLOADS["flat1m_f32"]
    params = wl.init_params(w, dev)
    opt = ma.MicroAdam(params, ma.make_config(density=w.density, window=w.window, ef_bucket=w.bucket,
                                              topk_block=w.block, lr=w.lr))
    try:
        for s in range(1, 4):  # unprofiled steps count in no total
            opt.step(wl.grads_for_step(w, s, dev))
        grads = wl.grads_for_step(w, 4, dev)
        opt.set_profiling(True)
        for _ in range(6):  # more steps than the ring holds
            opt.step(grads)
        last = opt.kernel_times()
        sel, upd, n = opt.kernel_times_total()
        assert n == 6
        assert sel > 0 and upd > 0
        assert last[0] <= sel and last[1] <= upd
        assert opt.kernel_times_total() == (0.0, 0.0, 0)  # the totals restart
        opt.step(grads)
        opt.set_profiling(True)  # switching on again starts a new total
        opt.step(grads)
        assert opt.kernel_times_total()[2] == 1
        opt.set_profiling(False)
        opt.step(grads)
        assert opt.kernel_times_total()[2] == 0
        assert opt.t == 3 + 6 + 3
    finally:
        opt.close()
