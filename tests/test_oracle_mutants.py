"""Plants plausible mistakes in copies of the oracle's C source and checks that
the pins catch every one of them (the mistakes live only in temporary copies
built on the CPU; the committed oracle is untouched)."""
import os
import subprocess

import pytest

import oracle
from tests import test_oracle_pins as pins

MUTANTS = {
    "page_slot_swapped": ("int32_t page = bt[j / jb->s];\n    int32_t slot = j % jb->s;",
                          "int32_t page = bt[j % jb->s];\n    int32_t slot = j / jb->s;"),
    "kv_head_modulo": ("const int32_t kvh = h / group;", "const int32_t kvh = h % jb->hkv;"),
    "scale_dropped": ("scores[j] = dot * jb->scale;", "scores[j] = dot;"),
    "exp_sign_flipped": ("scores[j] = exp(scores[j] - m);", "scores[j] = exp(m - scores[j]);"),
    "not_normalised": ("for (int32_t e = 0; e < jb->d; ++e) o[e] /= l;", ""),
    "last_value_dropped": ("for (int32_t j = 0; j < nvis; ++j) {\n        const uint16_t *v",
                           "for (int32_t j = 0; j < nvis - 1; ++j) {\n        const uint16_t *v"),
    "pool_layout_transposed": ("(((size_t)page * jb->hkv + kvh) * jb->s + slot) * jb->d",
                               "(((size_t)page * jb->s + slot) * jb->hkv + kvh) * jb->d"),
    "query_head_is_kv_head": ("jb->q + ((size_t)row * jb->hq + h) * jb->d",
                              "jb->q + ((size_t)row * jb->hq + kvh) * jb->d"),
    "dot_term_dropped": ("for (int32_t e = 0; e < jb->d; ++e)\n            dot +=",
                         "for (int32_t e = 1; e < jb->d; ++e)\n            dot +="),
    "bf16_widening_wrong": ("uint32_t w = (uint32_t)bits << 16;", "uint32_t w = (uint32_t)bits << 15;"),
}


def _checks():
    yield lambda: pins.test_worked_example_fixture()
    yield lambda: pins.test_single_visible_key_returns_its_value_exactly()
    yield lambda: pins.test_zero_query_gives_mean_of_visible_values()
    for shape in pins.SHAPES:
        yield lambda shape=shape: pins.test_oracle_matches_library_sdpa_and_bruteforce(*shape)


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    src = open(oracle._SRC).read()
    old, new = MUTANTS[name]
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    c = tmp_path / "mutant.c"
    so = tmp_path / "libmutant.so"
    c.write_text(src.replace(old, new))
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                           "-pthread", "-o", str(so), str(c), "-lm"])
    caught = []
    with oracle.use_library(str(so)):
        for check in _checks():
            try:
                check()
            except (AssertionError, ValueError) as e:
                caught.append(repr(e)[:80])
                break
    assert caught, f"no pin caught the planted mistake {name}"


def test_unmutated_copy_passes_every_check(tmp_path):
    so = tmp_path / "libcopy.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fPIC", "-shared",
                           "-pthread", "-o", str(so), oracle._SRC, "-lm"])
    with oracle.use_library(str(so)):
        for check in _checks():
            check()
