"""Non-finite gradients: NaN and +-inf in some Top-K blocks of one tensor.

The method leaves them undefined (every step of Algorithm 1 assumes finite
values), so the library promises only this: a block whose gradient holds a
NaN or an infinity gets unspecified parameters and state, and every other
block, of that tensor or of another, is computed exactly as if the
non-finite values were not there.  Blocks are independent in the step (with
buckets inside blocks), so each clean block and the second tensor must match,
bit for bit, a run on the same inputs with the non-finite values replaced by
zeros.  Both select kernels are covered: B_d = 4096 and B_d = 65536."""
import pytest

import paper_2405_15593_amd as ma

pytestmark = pytest.mark.gpu


def _run(numels, block, density, window, grads, steps, bucket):
    import torch
    dev = torch.device("cuda:0")
    gen = torch.Generator(device="cpu").manual_seed(5)
    params = [(torch.randn(n, generator=gen) * 0.02).to(dev, torch.bfloat16) for n in numels]
    cfg = ma.make_config(density=density, window=window, ef_bucket=bucket, topk_block=block, lr=1e-3)
    opt = ma.MicroAdam(params, cfg)
    for t in range(steps):
        opt.step([g[t % len(g)] for g in grads])
    torch.cuda.synchronize()
    moments = [opt.debug_moments(j) for j in range(len(numels))]
    out = [p.clone() for p in params], moments
    opt.close()
    return out


@pytest.mark.parametrize("block,bucket,density,window", [(4096, 64, 0.01, 3), (65536, 128, 0.05, 4)],
                         ids=["block4096", "block65536"])
def test_nonfinite_blocks_are_isolated(block, bucket, density, window):
    import torch
    dev = torch.device("cuda:0")
    na = block * 5 + 1000          # five full blocks and a ragged one
    nb = block + 333
    gen = torch.Generator(device="cpu").manual_seed(11)
    bad_blocks = [1, 3]            # blocks of tensor A that get NaN / inf
    ga, ga_clean, gb = [], [], []
    for s in range(2):
        a = torch.randn(na, generator=gen) * 1e-3
        clean = a.clone()
        # block 1: NaNs, one of them the largest-index element; block 3: +-inf
        a[block + 7] = float("nan")
        a[2 * block - 1] = float("nan")
        a[3 * block + 100] = float("inf")
        a[3 * block + 101] = float("-inf")
        clean[block + 7] = clean[2 * block - 1] = clean[3 * block + 100] = clean[3 * block + 101] = 0.0
        ga.append(a.to(dev, torch.bfloat16))
        ga_clean.append(clean.to(dev, torch.bfloat16))
        gb.append((torch.randn(nb, generator=gen) * 1e-3).to(dev, torch.bfloat16))
    print(f"[nonfinite] block={block} numels={[na, nb]} bad blocks {bad_blocks}", flush=True)
    steps = window + 2
    (p_bad, m_bad) = _run([na, nb], block, density, window, [ga, gb], steps, bucket)
    print("[nonfinite] run with NaN/inf done", flush=True)
    (p_ok, m_ok) = _run([na, nb], block, density, window, [ga_clean, gb], steps, bucket)
    print("[nonfinite] clean run done", flush=True)
    # the second tensor: bit-identical parameters and moments
    assert torch.equal(p_bad[1].view(torch.int16), p_ok[1].view(torch.int16))
    for x, y in zip(m_bad[1], m_ok[1]):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))
    # tensor A: every block other than the bad ones bit-identical
    good = torch.ones(na, dtype=torch.bool, device=dev)
    for q in bad_blocks:
        good[q * block:(q + 1) * block] = False
    assert torch.equal(p_bad[0][good].view(torch.int16), p_ok[0][good].view(torch.int16))
    for x, y in zip(m_bad[0], m_ok[0]):
        assert torch.equal(x[good].view(torch.int32), y[good].view(torch.int32))
