"""microadam_step_noalloc (the entry point for callers that cannot allocate)
against microadam_init + microadam_step on the same inputs: two calls in a
row on one GPU, the second with a smaller tensor list, then one with blocks
above 4096 elements; parameters and the whole state buffer bit for bit."""
import math

import pytest
import torch

import paper_2405_15593_amd as ma
from paper_2405_15593_amd import workloads as wl

pytestmark = pytest.mark.gpu

DT = {torch.float32: ma.MICROADAM_F32, torch.bfloat16: ma.MICROADAM_BF16}


def _run_both(numels, steps, dtype, **cfg_kw):
    dev = torch.device("cuda")
    cfg = ma.make_config(**cfg_kw)
    params_a = [wl.draw(n, "normal", 0.02, 11 + j, dev, dtype) for j, n in enumerate(numels)]
    params_b = [p.clone() for p in params_a]
    params_0 = [p.clone() for p in params_a]
    opt = ma.MicroAdam(params_a, cfg)
    nbytes = ma.microadam_state_bytes(cfg, numels)
    raw = torch.zeros(nbytes + 256, dtype=torch.uint8, device=dev)  # step 1 starts from zeros
    off = (-raw.data_ptr()) % 256
    state_b = raw[off:off + nbytes]
    stream = torch.cuda.current_stream().cuda_stream
    for t in range(1, steps + 1):
        grads = [wl.draw(n, "student_t4", 1e-3, wl.grad_seed(t, j, 5), dev, dtype) for j, n in enumerate(numels)]
        opt.step(grads)
        ma.microadam_step_noalloc(cfg, numels, DT[dtype], DT[dtype], state_b.data_ptr(), nbytes, t,
                                  [p.data_ptr() for p in params_b], [g.data_ptr() for g in grads],
                                  math.nan, stream)
    torch.cuda.synchronize()
    for j, (a, b) in enumerate(zip(params_a, params_b)):
        assert torch.equal(a.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                           b.view(torch.int16 if dtype == torch.bfloat16 else torch.int32)), f"params differ, tensor {j}"
    assert torch.equal(opt.state_view, state_b), "state buffers differ"
    assert sum(int((a.float() != b.float()).sum()) for a, b in zip(params_a, params_0)) > 0, "nothing changed"
    opt.close()


def test_noalloc_matches_step_two_calls():
    print("[noalloc] call 1: 3 tensors, 3 steps, bf16", flush=True)
    _run_both([4096 * 3 + 100, 777, 5000], 3, torch.bfloat16, window=3)
    print("[noalloc] call 2: a smaller list, 2 steps, float32", flush=True)
    _run_both([3000, 17], 2, torch.float32, window=2)
    print("[noalloc] call 3: blocks of 8192, 2 steps", flush=True)
    _run_both([8192 + 100], 2, torch.float32, window=2, topk_block=8192)


def test_noalloc_rejects_too_many_tensors():
    cfg = ma.make_config()
    with pytest.raises(ma.MicroAdamError) as e:
        ma.microadam_step_noalloc(cfg, [16] * 4097, ma.MICROADAM_F32, ma.MICROADAM_F32, 256, 1 << 30, 1,
                                  [256] * 4097, [256] * 4097)
    assert e.value.code == ma.MICROADAM_ERR_UNSUPPORTED
