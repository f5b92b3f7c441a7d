"""Planted mistakes in a copy of the oracle must each fail at least one pin.

Every mutant is a textual edit of ``oracle/kvx_oracle.c`` compiled into a
temporary library on the CPU; the pins of ``oracle_pins.py`` run against it.
A mutant that passes every pin would mean the pins cannot see that class of
mistake.
"""
import os
import shutil
import subprocess

import pytest

from oracle import oracle as O
from tests import oracle_pins as P

MUTANTS = {
    "derotate_sign": ("rope_apply(s->xk, s->xr, Ds, -(double)k, s->ths);",
                      "rope_apply(s->xk, s->xr, Ds, (double)k, s->ths);"),
    "derotate_uses_target_pos": ("rope_apply(s->xk, s->xr, Ds, -(double)k, s->ths);",
                                 "rope_apply(s->xk, s->xr, Ds, -(double)t, s->ths);"),
    "rerotate_sign": ("Dt, (double)t, s->tht);", "Dt, -(double)t, s->tht);"),
    "rerotate_off_by_one": ("Dt, (double)t, s->tht);", "Dt, (double)(t + 1), s->tht);"),
    "rotation_sign": ("y[i] = x0 * c - x1 * s;", "y[i] = x0 * c + x1 * s;"),
    "pairing_interleaved": ("double x0 = x[i], x1 = x[i + h];",
                            "double x0 = x[2 * i], x1 = x[2 * i + 1];"),
    "freq_exponent": ("-2.0 * (double)i / (double)m->head_dim",
                      "-(double)i / (double)m->head_dim"),
    "w_transposed": ("wl + o * din + i", "wl + i * dout + o"),
    "bias_dropped": ("if (p->b_k) ak += (double)p->b_k[(int64_t)l * dout + o];", ""),
    "pool_weight_ignored": ("double w = p->tgt_tokens ? (double)p->weight[e] : 1.0;",
                            "double w = 1.0;"),
    "mix_layer_ignored": ("p->layer_map[(int64_t)l * p->mix + j]",
                          "p->layer_map[(int64_t)l * p->mix]"),
    "feature_order_head_major": ("int64_t col = ((int64_t)j * Hs + h) * Ds;",
                                 "int64_t col = ((int64_t)h * p->mix + j) * Ds;"),
    "v_rotated": ("s->zv[col + d] += w * s->xv[d];", "s->zv[col + d] += w * s->xr[d];"),
    "context_ignored": ("(((ls * B + b) * Hs + h)", "(((ls * B + 0) * Hs + h)"),
    "inv_freq_index_2i": ("if (m->inv_freq) return m->inv_freq[i];",
                          "if (m->inv_freq) return m->inv_freq[(2 * i) % (m->head_dim / 2)];"),
    "inv_freq_as_revolutions": ("if (m->inv_freq) return m->inv_freq[i];",
                                "if (m->inv_freq) return m->inv_freq[i] * 6.283185307179586;"),
    "inv_freq_ignored": ("if (m->inv_freq) return m->inv_freq[i];", ""),
    "inv_freq_needs_base": ("return m->inv_freq != NULL || m->rope_base > 0.0;",
                            "return m->rope_base > 0.0;"),
    "span_last_dropped": ("e1 = p->row_ptr[row0 + t + 1];",
                          "e1 = p->row_ptr[row0 + t + 1] - (p->row_ptr[row0 + t + 1] > e0 + 1);"),
}


@pytest.fixture(scope="module")
def mutant_dir(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    return tmp_path_factory.mktemp("oracle_mutants")


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, mutant_dir):
    old, new = MUTANTS[name]
    src = open(O.SRC).read()
    assert src.count(old) >= 1, f"mutation anchor for {name} not found"
    d = mutant_dir / name
    d.mkdir()
    shutil.copy(os.path.join(os.path.dirname(O.SRC), "kvx_oracle.h"), d / "kvx_oracle.h")
    (d / "kvx_oracle.c").write_text(src.replace(old, new))
    lib = O.build(str(d / "libmut.so"), str(d / "kvx_oracle.c"))
    failed = []
    for pin in P.ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} passed every pin"
