"""CPU tests of the oracle: its pins, its argument checks, and a check that
each pin set catches plausible mistakes planted in a copy of the oracle."""
from __future__ import annotations

import os
import re
import subprocess
import sys

import numpy as np
import pytest

import oracle
from paper_2609_38981_amd import workloads as W
from tests import oracle_pins as pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    oracle.build(force=False)
    return oracle._load()


@pytest.mark.parametrize("pin", pins.ALL_PINS, ids=lambda f: f.__name__)
def test_pin(lib, pin):
    pin(lib)


# ---------------------------------------------------------------------------
# argument checks
# ---------------------------------------------------------------------------
def _tiny_args():
    call = W.config1()
    kp, vp = call.std_pool()
    return dict(q_bits=call.q_bits(), cu_q_lens=call.cu_q_lens, context_lens=call.context_lens,
                page_table=call.page_table, k_pool_bits=kp, v_pool_bits=vp), call


def test_rejects_query_longer_than_context():
    a, call = _tiny_args()
    ctx = a["context_lens"].copy()
    ctx[1] = 7  # s = 8 > n = 7
    a["context_lens"] = ctx
    with pytest.raises(ValueError):
        oracle.paged_attention(**a, num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16)


def test_rejects_page_out_of_range():
    a, call = _tiny_args()
    pt = a["page_table"].copy()
    pt[0, 0] = call.num_pages
    a["page_table"] = pt
    with pytest.raises(ValueError):
        oracle.paged_attention(**a, num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16)


def test_rejects_empty_query():
    a, call = _tiny_args()
    a["cu_q_lens"] = np.array([0, 0, 9], np.int32)
    with pytest.raises(ValueError):
        oracle.paged_attention(**a, num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16)


def test_row_selection_and_threads():
    a, call = _tiny_args()
    full = oracle.paged_attention(**a, num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16,
                                  threads=1)
    part = oracle.paged_attention(**a, num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16,
                                  rows=[0, 5], threads=3)
    assert np.array_equal(part[[0, 5]], full[[0, 5]])
    assert np.isnan(part[1]).all()
    assert np.isfinite(full).all()  # the NaN-poisoned slots were never read


def test_empty_batch():
    sh = W.TINY
    out = oracle.paged_attention(np.zeros((0, 4, 64), np.uint16), np.zeros(1, np.int32),
                                 np.zeros(0, np.int32), np.zeros((0, 1), np.int32),
                                 np.zeros((1, 2, 16, 64), np.uint16), np.zeros((1, 2, 16, 64), np.uint16),
                                 num_q_heads=4, num_kv_heads=2, head_dim=64, page_size=16)
    assert out.shape == (0, 4, 64)


def test_linear_rejects_bad_sizes():
    a = np.zeros((2, 8), np.uint16)
    b = np.zeros((3, 8), np.uint16)
    with pytest.raises(ValueError):
        oracle.linear(a, b, k=9)  # k beyond the row stride
    assert oracle.linear(a[:0], b).shape == (0, 3)


# ---------------------------------------------------------------------------
# planted mistakes: every mutant must fail at least one pin
# ---------------------------------------------------------------------------
MUTANTS = {
    "dropped_scale": ("score[j] = J->scale * acc;", "score[j] = acc;"),
    "sign_error": ("score[j] = J->scale * acc;", "score[j] = -J->scale * acc;"),
    "position_convention": ("const int p = n - s + i;", "const int p = i;"),
    "position_off_by_one": ("const int p = n - s + i;", "const int p = n - s + i - (i > 0);"),
    "gqa_interleaved": ("const int g = h / group;", "const int g = h % J->hkv;"),
    "page_index_swapped": ("const int64_t page = pt[j / P];\n      const uint16_t *krow",
                           "const int64_t page = pt[j % P];\n      const uint16_t *krow"),
    "slot_transposed": ("((page * J->hkv + g) * P) + (j % P)) * (int64_t)D;\n      double acc",
                        "((page * J->hkv + g) * P) + (P - 1 - j % P)) * (int64_t)D;\n      double acc"),
    "unnormalised": ("w[j] /= denom;", "w[j] /= 1.0;"),
    "value_from_key_pool": ("J->v_pool + (((page", "J->k_pool + (((page"),
    "drops_last_key": ("for (int j = lo; j <= p; ++j) {\n      const int64_t page = pt[j / P];\n      const uint16_t *vrow",
                       "for (int j = lo; j < p; ++j) {\n      const int64_t page = pt[j / P];\n      const uint16_t *vrow"),
    "window_off_by_one": ("p - J->window + 1 > 0) ? p - J->window + 1 : 0;",
                          "p - J->window > 0) ? p - J->window : 0;"),
    "window_ignored": ("const int lo = (J->window > 0 &&", "const int lo = (J->window < 0 &&"),
    "lse_log2": ("J->lse[t * J->hq + h] = mx + log(denom);", "J->lse[t * J->hq + h] = mx + log2(denom);"),
    "lse_no_max": ("J->lse[t * J->hq + h] = mx + log(denom);", "J->lse[t * J->hq + h] = log(denom);"),
    "lse_sign": ("J->lse[t * J->hq + h] = mx + log(denom);", "J->lse[t * J->hq + h] = mx - log(denom);"),
    "window_from_n": ("p - J->window + 1 > 0) ? p - J->window + 1 : 0;",
                      "n - J->window + 1 > 0) ? n - J->window + 1 : 0;"),
    # linear layer
    "linear_transposed_weights": ("acc += bf16_to_double(arow[k]) * bf16_to_double(brow[k]);",
                                  "acc += bf16_to_double(arow[k]) * bf16_to_double(J->b[(int64_t)(k % J->N) * J->ldb + n % J->K]);"),
    "linear_drops_last_k": ("for (int k = 0; k < J->K; ++k)", "for (int k = 0; k < J->K - 1; ++k)"),
    "linear_ignores_stride": ("const uint16_t *arow = J->a + m * J->lda;",
                              "const uint16_t *arow = J->a + m * J->K;"),
    "linear_previous_row": ("const uint16_t *arow = J->a + m * J->lda;",
                            "const uint16_t *arow = J->a + (m > 0 ? m - 1 : 0) * J->lda;"),
    "linear_sign": ("acc += bf16_to_double(arow[k]) * bf16_to_double(brow[k]);",
                    "acc -= bf16_to_double(arow[k]) * bf16_to_double(brow[k]);"),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    src = open(os.path.join(os.path.dirname(oracle.__file__), "vd_oracle.c")).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, "mutation anchor not found or not unique: %r" % old
    mut = tmp_path / ("mut_%s.c" % name)
    mut.write_text(src.replace(old, new))
    so = tmp_path / ("mut_%s.so" % name)
    subprocess.run(["gcc", "-O1", "-std=c11", "-fPIC", "-shared", "-pthread", str(mut), "-o",
                    str(so), "-lm"], check=True)
    env = dict(os.environ, PYTHONPATH=ROOT + os.pathsep + os.environ.get("PYTHONPATH", ""))
    res = subprocess.run([sys.executable, "-m", "tests.oracle_pins", str(so)], cwd=ROOT, env=env,
                         capture_output=True, text=True, timeout=300)
    caught = [ln for ln in res.stdout.splitlines() if ln.startswith("CAUGHT")]
    crashed = res.returncode != 0
    assert caught or crashed, "no pin caught the planted mistake %s" % name
