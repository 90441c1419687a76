"""Plants plausible mistakes in a copy of the oracle source (on the CPU) and
requires the pins to catch each one.  This is how the pins are shown to be
strong enough: a dropped term, a wrong sign, a wrong index or exponent, a
reversed tie rule or the wrong rounding mode must all fail some pin."""
import os
import subprocess

import pytest

import oracle
import oracle_pins

# (label, text in microadam_oracle.c, replacement)
MUTANTS = [
    ("exponent r off by one", "pow(beta, (double)(t - s))", "pow(beta, (double)(t - s + 1))"),
    ("bias correction dropped", "const double scale = (1.0 - beta) / (1.0 - pow(beta, (double)t));",
     "const double scale = (1.0 - beta);"),
    ("bias correction over the window only",
     "const double scale = (1.0 - beta) / (1.0 - pow(beta, (double)t));",
     "const double scale = (1.0 - beta) / (1.0 - pow(beta, (double)(t < m ? t : m)));"),
    ("one row too many", "int64_t first = t - m + 1;", "int64_t first = t - m;"),
    ("row pointer off by one", "const int64_t row = (t - 1) % m;", "const int64_t row = t % m;"),
    ("higher index wins ties", "return (i < j) ? -1 : (i > j);", "return (i > j) ? -1 : (i < j);"),
    ("signed instead of |a|", "float ai = fabsf(g_sort_vals[i]), aj = fabsf(g_sort_vals[j]);",
     "float ai = g_sort_vals[i], aj = g_sort_vals[j];"),
    ("kept entries not zeroed", "for (int64_t j = 0; j < k; ++j) ab[chosen[j]] = 0.0f;", ""),
    ("round half up", "float r = nearbyintf(y);", "float r = floorf(y + 0.5f);"),
    ("truncating quantizer", "float r = nearbyintf(y);", "float r = floorf(y);"),
    ("decode sign", "return scaled + lo;", "return scaled - lo;"),
    ("decode level 16", "const float levels = (float)((1 << c->ef_bits) - 1);",
     "const float levels = (float)(1 << c->ef_bits);"),
    ("min and max swapped", "if (a[i - lo] < mn) mn = a[i - lo];", "if (a[i - lo] > mn) mn = a[i - lo];"),
    ("update sign", "(double)theta[i] * decay - lr * upd", "(double)theta[i] * decay + lr * upd"),
    ("eps inside sqrt", "mh[i - lo] / (c->eps + sqrt(vh[i - lo]))", "mh[i - lo] / sqrt(c->eps + vh[i - lo])"),
    ("second moment not squared", "(squared ? v * v : v)", "(squared ? v : v)"),
    ("decay sign", "1.0 - lr * c->weight_decay", "1.0 + lr * c->weight_decay"),
    ("bf16 keeps 9 bits", "int q = e - 8;", "int q = e - 9;"),
    ("accumulator ignores EF",
     "a[i - lo] = grad[i] + dequantize(get_code(ef, i, c->ef_bits), delta[b], Delta[b], levels);",
     "a[i - lo] = grad[i];"),
    ("nibbles swapped", "return (i & 1) ? (unsigned)(byte >> 4) : (unsigned)(byte & 0x0F);",
     "return (i & 1) ? (unsigned)(byte & 0x0F) : (unsigned)(byte >> 4);"),
    ("beta1 for both moments", "adam_stats(c, t, c->beta2, 1,", "adam_stats(c, t, c->beta1, 1,"),
    ("k rounds down", "double x = ceil(density * (double)s - 1e-9);", "double x = floor(density * (double)s);"),
    ("philox multiplier", "(uint64_t)0xD2511F53u * x0", "(uint64_t)0xD2511F55u * x0"),
    ("philox key bump", "k0 += 0x9E3779B9u;", "k0 += 0x9E3779BBu;"),
    ("philox nine rounds", "round < 10", "round < 9"),
    ("xi from the low bits", "return out[i & 3] >> 8;", "return out[i & 3] & 0xFFFFFFu;"),
    ("xi ignores the step", "(uint32_t)j, (uint32_t)t}", "(uint32_t)j, 0u}"),
    ("randomized rounds to nearest", "float r = fy + ((w24 + fr >= (1u << 24)) ? 1.0f : 0.0f);",
     "float r = nearbyintf(y);"),
    ("randomized rounds up", "float r = fy + ((w24 + fr >= (1u << 24)) ? 1.0f : 0.0f);",
     "float r = fy + (f > 0.0f ? 1.0f : 0.0f);"),
    ("randomized ignores the fraction", "(w24 + fr >= (1u << 24))", "(w24 >= (1u << 23))"),
    ("8-bit codes read as nibbles", "if (bits == 8) return ef[i];", "if (bits == 8) return ef[i] & 0x0F;"),
    ("param_bf16 ignored", "theta[i] = c->param_bf16 ? round_to_bf16(nt) : (float)nt;", "theta[i] = (float)nt;"),
    ("theta rounded through binary32", "theta[i] = c->param_bf16 ? round_to_bf16(nt) : (float)nt;",
     "theta[i] = c->param_bf16 ? round_to_bf16((double)(float)nt) : (float)nt;"),
    ("decode bucket relative to the block", "const int64_t b = i / c->bucket;",
     "const int64_t b = (i / c->block) * ((c->block + c->bucket - 1) / c->bucket) + (i % c->block) / c->bucket;"),
    ("buckets restart at each block", "int64_t b1 = b0 + c->bucket;",
     "int64_t b1 = b0 + c->bucket; if ((b1 - 1) / c->block != b0 / c->block) b1 = (b0 / c->block + 1) * c->block;"),
]


@pytest.mark.parametrize("label,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, label, old, new):
    src = open(oracle.SOURCE).read()
    assert src.count(old) == 1, f"mutation anchor not unique/present: {old!r}"
    mutated = tmp_path / "mutant.c"
    mutated.write_text(src.replace(old, new))
    lib = oracle.build(str(mutated), str(tmp_path / "libmutant.so"))
    o = oracle.Oracle(lib)
    caught = []
    for check in oracle_pins.ALL_CHECKS:
        try:
            check(o)
        except (AssertionError, ValueError, IndexError):
            caught.append(check.__name__)
    assert caught, f"no pin catches mutant '{label}'"
