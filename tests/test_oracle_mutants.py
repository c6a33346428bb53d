"""Plant plausible mistakes in a copy of the oracle and check the pins catch each.

Each mutant is a one-spot textual edit of ``oracle/oracle.c`` (a dropped
term, a wrong sign, a transposed operand, a flipped comparison, a wrong
rounding rule), compiled into a temporary library.  The pin suite of
tests/pins.py must fail on every one of them; otherwise the pins would not
be able to tell a broken oracle from a correct one.  Everything runs on the
CPU; the real oracle is never modified.
"""
import os
import shutil

import pytest

import oracle
import pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "oracle.c")

MUTANTS = {
    "softmax_drops_max_shift": (
        "y[i] = exp(load_elem(row, dtype, i) - m) / d;",
        "y[i] = exp(load_elem(row, dtype, i)) / d;"),
    "softmax_wrong_sign": (
        "y[i] = exp(load_elem(row, dtype, i) - m) / d;",
        "y[i] = exp(m - load_elem(row, dtype, i)) / d;"),
    "normalizer_drops_first_term": (
        "for (int64_t j = 0; j < V; ++j) d += exp(load_elem(row, dtype, j) - m);",
        "for (int64_t j = 1; j < V; ++j) d += exp(load_elem(row, dtype, j) - m);"),
    "max_skips_last_element": (
        "for (int64_t k = 0; k < V; ++k) {\n        double v = load_elem(row, dtype, k);",
        "for (int64_t k = 0; k + 1 < V; ++k) {\n        double v = load_elem(row, dtype, k);"),
    "combine_takes_min": (
        "double M = mi > mj ? mi : mj;",
        "double M = mi < mj ? mi : mj;"),
    "combine_transposed_scale": (
        "*d_out = di * exp(mi - M) + dj * exp(mj - M);",
        "*d_out = di * exp(mj - M) + dj * exp(mi - M);"),
    "combine_no_identity_guard": (
        "if (M == -INFINITY) {\n        *m_out = -INFINITY;\n        *d_out = 0.0;",
        "if (M == -INFINITY && 0) {\n        *m_out = -INFINITY;\n        *d_out = 0.0;"),
    "online_uses_new_element_weight_zero": (
        "orc_md_combine(m, d, xj, 1.0, &m, &d);\n    }\n    *m_out = m;",
        "orc_md_combine(m, d, xj, 0.5, &m, &d);\n    }\n    *m_out = m;"),
    "topk_ties_to_higher_index": (
        "return (p->i > q->i) - (p->i < q->i);",
        "return (p->i < q->i) - (p->i > q->i);"),
    "topk_ascending": (
        "if (p->x > q->x) return -1;\n        if (p->x < q->x) return 1;",
        "if (p->x > q->x) return 1;\n        if (p->x < q->x) return -1;"),
    "topk_value_off_by_one": (
        "z[r * K + k] = buf[k].i;\n                v[r * K + k] = exp(buf[k].x - m) / d;",
        "z[r * K + k] = buf[k].i;\n                v[r * K + k] = exp(buf[k + (k + 1 < K)].x - m) / d;"),
    "select_ties_to_higher_index": (
        "return ia < ib;          /* equal values",
        "return ia > ib;          /* equal values"),
    "select_skips_last_element": (
        "for (int64_t j = 0; j < V; ++j) {\n                double xj = load_elem(row, dtype, j);\n                if (prev_i",
        "for (int64_t j = 0; j + 1 < V; ++j) {\n                double xj = load_elem(row, dtype, j);\n                if (prev_i"),
    "bf16_widen_reads_wrong_type": (
        "out[i] = load_elem(bits, ORC_BF16, i);",
        "out[i] = load_elem(bits, ORC_F32, i / 2);"),
    "bf16_round_half_away": (
        "double r = rint(a / q) * q;",
        "double r = round(a / q) * q;"),
    "bf16_round_truncates": (
        "double r = rint(a / q) * q;",
        "double r = floor(a / q) * q;"),
    "bf16_subnormal_spacing": (
        "if (ex < -126) ex = -126;",
        "if (ex < -127) ex = -127;"),
    "proj_transposed_weight_index": (
        "acc += load_elem(hr, hdtype, k) * load_elem(wr, wdtype, k);",
        "acc += load_elem(hr, hdtype, k) * load_elem(row_ptr(w, wdtype, H, k % V), wdtype, v % H);"),
    "proj_skips_last_term": (
        "for (int64_t k = 0; k < H; ++k) acc += load_elem(hr, hdtype, k)",
        "for (int64_t k = 0; k + 1 < H; ++k) acc += load_elem(hr, hdtype, k)"),
    "proj_squares_hidden": (
        "acc += load_elem(hr, hdtype, k) * load_elem(wr, wdtype, k);",
        "acc += load_elem(hr, hdtype, k) * load_elem(hr, hdtype, k);"),
    "bf16_widening_wrong_shift": (
        "uint32_t bits = (uint32_t)((const uint16_t*)row)[i] << 16;",
        "uint32_t bits = (uint32_t)((const uint16_t*)row)[i] << 15;"),
}


def _first_failure(orc):
    for check in pins.ALL:
        try:
            check(orc)
        except AssertionError:
            return check.__name__
    return None


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site for {name} not unique or missing"
    src = tmp_path / "oracle.c"
    src.write_text(text.replace(old, new))
    lib = oracle.build(str(src), str(tmp_path / "liboracle_mutant.so"))
    caught = _first_failure(oracle.load(lib))
    assert caught is not None, f"no pin caught mutant {name}"


def test_widening_pin_catches_wrong_shift(tmp_path):
    """The bfloat16 widening pin on its own catches a widening off by one bit
    position (the expected values of every bfloat16 GPU check go through it)."""
    old, new = MUTANTS["bf16_widening_wrong_shift"]
    text = open(SRC).read()
    src = tmp_path / "oracle.c"
    src.write_text(text.replace(old, new))
    lib = oracle.build(str(src), str(tmp_path / "liboracle_mutant.so"))
    with pytest.raises(AssertionError):
        pins.check_bf16_widening(oracle.load(lib))
