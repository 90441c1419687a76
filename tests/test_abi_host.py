"""Host-side checks of libmicroadam that need no GPU: the library loads and
exports every symbol its header declares, the state-size planner matches the
paper's byte model, and invalid configurations are rejected before any
device work."""
import math
import os
import re

import pytest

import paper_2405_15593_amd as ma

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "microadam.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(ma.LIBRARY):
        from paper_2405_15593_amd import _build
        _build.build()
    return ma.load()


def test_exports_every_declared_symbol(lib):
    decl = re.findall(r"^\S[^;(]*?\b(microadam_\w+)\s*\(", open(HEADER).read(), re.M)
    assert set(decl) == set(ma.EXPORTS), sorted(set(decl) ^ set(ma.EXPORTS))
    for name in decl:
        assert hasattr(lib, name), name


def llama7b_numels():
    from paper_2405_15593_amd.workloads import WORKLOADS
    return WORKLOADS["llama2_7b_bf16"].numels


def test_state_bytes_llama2_7b(lib):
    """0.5 B/param of EF (Section 3.2), 8 B per bucket of 64 for (delta, Delta),
    and m rows of 41 entries per 4096-block at 4 B each; no tails here."""
    numels = llama7b_numels()
    d = sum(numels)
    assert d == 6_738_415_616
    cfg = ma.make_config()
    got = ma.microadam_state_bytes(cfg, numels)
    blocks = d // 4096
    assert all(n % 4096 == 0 for n in numels)
    # a window record (10 rows of 41 four-byte entries, 1640 B) is padded to
    # whole 128-byte lines: 1664 B
    want_payload = d // 2 + 8 * (d // 64) + 1664 * blocks
    # each of the 3 planes is padded to 256 bytes
    assert want_payload <= got <= want_payload + 3 * 256
    # the paper's 0.5d + 4mk with a global k = ceil(d/100) (Section 3.2)
    paper = 0.5 * d + 4 * 10 * math.ceil(d / 100)
    ours_without_stats = d // 2 + 10 * 41 * 4 * blocks
    assert abs(ours_without_stats / paper - 1) < 2e-3   # 41/4096 vs 1/100
    assert round(got / 2 ** 30, 3) == 6.472


def test_state_bytes_tails_and_f32(lib):
    cfg = ma.make_config(density=0.01, window=3, ef_bucket=16, topk_block=256,
                         window_value_dtype=ma.MICROADAM_F32)
    n = 1001            # 3 full blocks of 256 (k 3) and a tail of 233 (k 3)
    pad = lambda x: -(-x // 256) * 256
    # every block owns a full-size record in each plane: 128 B of codes,
    # 16 (delta, Delta) pairs and 3 rows of k_full = 3 eight-byte entries
    # (72 B, padded to one 128-byte line)
    per_block = (128, 16 * 8, 128)
    got = ma.microadam_state_bytes(cfg, [n])
    assert got == sum(pad(4 * x) for x in per_block)
    # a second tensor of 10 elements adds one block (k 1, padded to k_full)
    got2 = ma.microadam_state_bytes(cfg, [n, 10])
    assert got2 == sum(pad(5 * x) for x in per_block)


def test_state_bytes_8bit_codes(lib):
    cfg = ma.make_config(density=0.01, window=3, ef_bucket=16, topk_block=256, ef_bits=8,
                         ef_rounding=ma.MICROADAM_ROUND_RANDOMIZED, seed=7)
    n = 1001            # 4 blocks of 256 (k 3): one code byte per element
    pad = lambda x: -(-x // 256) * 256
    per_block = (256, 16 * 8, 128)
    assert ma.microadam_state_bytes(cfg, [n]) == sum(pad(4 * x) for x in per_block)


def test_state_bytes_buckets_spanning_blocks(lib):
    cfg = ma.make_config(density=0.01, window=3, ef_bucket=100000, topk_block=4096)
    numels = [4096 * 30 + 1000, 250000]   # 31 and 62 blocks; 2 and 3 buckets
    pad = lambda x: -(-x // 256) * 256
    blocks, buckets = 31 + 62, 2 + 3
    rec = -(-3 * 41 * 4 // 128) * 128    # 3 rows of 41 four-byte entries, whole lines
    # 4-bit codes, two tables of (delta, Delta) pairs, per-block partials, window
    want = pad(blocks * 2048) + pad(2 * buckets * 8) + pad(blocks * 16) + pad(blocks * rec)
    assert ma.microadam_state_bytes(cfg, numels) == want


def test_state_bytes_large_blocks(lib):
    """Blocks above 4096 elements (the flat 1.5e9 workload's B_d = 65536,
    k = 3277, m = 20, B_q = 128): each window record holds the m rows and an
    m x 64 table of uint32 segment starts (one per 1024-element quarter),
    padded to whole 128-byte lines."""
    cfg = ma.make_config(density=0.05, window=20, ef_bucket=128, topk_block=65536)
    n = 65536 * 2 + 12032          # two full blocks and a tail of 12032 (k 602)
    pad = lambda x: -(-x // 256) * 256
    rec = -(-(20 * 3277 * 4 + 20 * 64 * 4) // 128) * 128
    per_block = (65536 // 2, (65536 // 128) * 8, rec)
    got = ma.microadam_state_bytes(cfg, [n])
    assert got == sum(pad(3 * x) for x in per_block)


def test_state_bytes_large_blocks_spanning_buckets(lib):
    """Buckets of 20,000 over blocks of 8192: codes, two tables of bucket
    pairs, per-block partials, and window records holding the m rows and the
    m x 8 segment table."""
    cfg = ma.make_config(density=0.02, window=3, ef_bucket=20000, topk_block=8192)
    numels = [8192 * 3 + 700, 20000]            # 4 and 3 blocks; 2 and 1 buckets
    pad = lambda x: -(-x // 256) * 256
    blocks, buckets = 7, 3
    rec = -(-(3 * 164 * 4 + 3 * 8 * 4) // 128) * 128   # k = ceil(0.02 * 8192) = 164
    want = pad(blocks * 4096) + pad(2 * buckets * 8) + pad(blocks * 16) + pad(blocks * rec)
    assert ma.microadam_state_bytes(cfg, numels) == want


def test_state_bytes_large_blocks_8bit(lib):
    """8-bit codes with B_d = 8192: one code byte per element, and the
    record's segment table of m x 8 uint32 behind the rows."""
    cfg = ma.make_config(density=0.01, window=3, ef_bucket=64, topk_block=8192, ef_bits=8,
                         ef_rounding=ma.MICROADAM_ROUND_RANDOMIZED, seed=11)
    n = 8192 * 2 + 500
    pad = lambda x: -(-x // 256) * 256
    rec = -(-(3 * 82 * 4 + 3 * 8 * 4) // 128) * 128   # k = ceil(0.01 * 8192) = 82
    per_block = (8192, (8192 // 64) * 8, rec)
    assert ma.microadam_state_bytes(cfg, [n]) == sum(pad(3 * x) for x in per_block)


BAD = [
    (dict(density=0.0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(density=1.5), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(density=math.nan), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(beta1=1.0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(beta2=-0.1), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(eps=-1.0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(eps=0.0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(fused=2), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(lr=math.inf), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(weight_decay=-1.0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(window=0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(window=65), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(ef_bits=6), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(ef_bits=0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(ef_rounding=2), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(ef_bucket=1000, topk_block=4096), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(ef_bucket=48), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(ef_bucket=1), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(topk_block=4000, ef_bucket=64), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(topk_block=131072), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(topk_block=0), ma.MICROADAM_ERR_INVALID_ARG),
    (dict(topk_block=8, ef_bucket=8), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(topk_block=1048, ef_bucket=8), ma.MICROADAM_ERR_UNSUPPORTED),
    (dict(window_value_dtype=7), ma.MICROADAM_ERR_INVALID_ARG),
]


@pytest.mark.parametrize("kw,code", BAD, ids=[str(b[0]) for b in BAD])
def test_invalid_config_rejected(lib, kw, code):
    cfg = ma.make_config(**kw)
    with pytest.raises(ma.MicroAdamError) as e:
        ma.microadam_state_bytes(cfg, [4096])
    assert e.value.code == code
    # init validates the same way before touching the device
    with pytest.raises(ma.MicroAdamError) as e:
        ma.microadam_init(cfg, [4096], ma.MICROADAM_BF16, ma.MICROADAM_BF16, 256, 1 << 20)
    assert e.value.code == code


def test_invalid_tensor_lists(lib):
    cfg = ma.make_config()
    for numels in ([], [0], [10, -3]):
        with pytest.raises(ma.MicroAdamError) as e:
            ma.microadam_state_bytes(cfg, numels)
        assert e.value.code == ma.MICROADAM_ERR_INVALID_ARG


def test_init_argument_checks_before_device_work(lib):
    cfg = ma.make_config()
    need = ma.microadam_state_bytes(cfg, [4096])
    cases = [
        ((cfg, [4096], 5, ma.MICROADAM_BF16, 256, need), ma.MICROADAM_ERR_INVALID_ARG),
        ((cfg, [4096], ma.MICROADAM_BF16, ma.MICROADAM_BF16, 0, need), ma.MICROADAM_ERR_INVALID_ARG),
        ((cfg, [4096], ma.MICROADAM_BF16, ma.MICROADAM_BF16, 258, need), ma.MICROADAM_ERR_INVALID_ARG),
        ((cfg, [4096], ma.MICROADAM_BF16, ma.MICROADAM_BF16, 256, need - 1), ma.MICROADAM_ERR_STATE_SIZE),
    ]
    for args, code in cases:
        with pytest.raises(ma.MicroAdamError) as e:
            ma.microadam_init(*args)
        assert e.value.code == code, (args, e.value)


def test_null_handle_calls(lib):
    for f, args in [(ma.microadam_get_step, (0,)), (ma.microadam_set_step, (0, 1)),
                    (ma.microadam_tensor_layout, (0, 0)), (ma.microadam_debug_moments, (0, 0, 1, 1)),
                    (ma.microadam_step, (0, [1], [1])), (ma.microadam_set_profiling, (0, True)),
                    (ma.microadam_kernel_times, (0,)), (ma.microadam_kernel_times_total, (0,))]:
        with pytest.raises(ma.MicroAdamError) as e:
            f(*args)
        assert e.value.code == ma.MICROADAM_ERR_INVALID_ARG
    ma.microadam_destroy(0)   # NULL is accepted
    assert ma.microadam_error_string(ma.MICROADAM_ERR_SHAPE) == "tensor list differs from init"
