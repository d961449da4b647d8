"""Plants plausible mistakes in copies of the oracle's launch simulation and
checks that the hand-computed launch pins catch every one of them (the
mistakes live only in temporary copies; the committed oracle is untouched)."""
import importlib.util
import os

import pytest

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle", "estimator.py")

# (new lens, prefix lens, hkv, group, CUs) -> (kernel path, load-imbalance factor),
# each worked out by hand in tests/test_estimator.py
PINS = [(([64], [0], 1, 1, 2), (1, 1 / 0.9)),
        (([128], [0], 1, 1, 1), (0, 1.0)),
        (([192], [0], 1, 1, 2), (0, 4 / 3)),
        (([32], [4064], 1, 1, 4), (1, 1.0)),
        (([4096], [0], 8, 4, 64), (0, 1.0)),
        (([141], [3000], 2, 1, 3), (0, 99 * 3 / 294)),
        (([130], [576], 1, 1, 6), (1, 11 * 6 / 54))]

MUTANTS = {
    "no_tie_window": ("window = 0.05 * total / len(work)", "window = 0.0"),
    "tie_ignores_cu_count": ("key=lambda e: (count[e[2]], e[1], e[2])", "key=lambda e: (e[1], e[2])"),
    "lone_factor_dropped": ("(0.9 if per_cu == 2 and count[c] == 1 else 1.0)", "1.0"),
    "key_tiles_off_by_one": ("return (r + min(q * bm + bm, n) + 63) // 64", "return (r + min(q * bm + bm, n)) // 64"),
    "never_paired": ("paired = npairs >= slots and rounds * slots * 20 <= npairs * 21", "paired = False"),
}


def _load(path):
    spec = importlib.util.spec_from_file_location("estimator_copy", path)
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _failures(mod):
    bad = []
    for args, (path, kappa) in PINS:
        got = mod.prefill_launch(*args)
        if got[0] != path or abs(got[1] - kappa) > 1e-12 * kappa:
            bad.append(args)
    return bad


def test_unmutated_copy_passes_every_pin(tmp_path):
    p = tmp_path / "estimator.py"
    p.write_text(open(SRC).read())
    assert _failures(_load(str(p))) == []


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_catch_planted_mistake(name, tmp_path):
    old, new = MUTANTS[name]
    text = open(SRC).read()
    assert text.count(old) == 1, f"mutation site of {name} not found once"
    p = tmp_path / "estimator.py"
    p.write_text(text.replace(old, new))
    assert _failures(_load(str(p))), f"no pin catches {name}"
