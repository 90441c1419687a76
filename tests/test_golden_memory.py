"""The paper's printed optimizer-state sizes for the Llama-2-7B parameter
count (Section 3.2, Appendix D), recomputed from the stated byte model:
4-bit error feedback (0.5 B/param) plus m rows of k int16 indices and
bf16 values (4 B per entry).  No GPU needed."""
import json
import math
import os

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "memory_llama2_7b.json")


def test_printed_memory_model():
    g = json.load(open(GOLDEN))
    d, m = g["d"], g["window_m"]
    k = math.ceil(d / 100)
    gib = 2 ** 30
    p = g["printed_GiB"]
    assert round(8 * d / gib, 2) == p["AdamW_fp32_8d"]
    assert round(4 * d / gib, 2) == p["AdamW_bf16_4d"]
    assert round(2 * d / gib, 2) == p["AdamW_8bit_2d"]
    assert round((0.5 * d + 4 * m * k) / gib, 2) == p["MicroAdam_0.5d_plus_4mk"]
    # window length at which MicroAdam's state equals 8-bit Adam's: 0.5d + 4mk = 2d
    assert abs((2 * d - 0.5 * d) / (4 * d / 100) - g["m_max_vs_8bit"]) < 1e-9
