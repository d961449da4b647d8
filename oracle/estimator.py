"""CPU oracle of the contention-tolerant estimator (test infrastructure).

Only ``tests/`` use this module; the library neither imports nor links it.
Plain numpy, written from the paper's Sec. 3.3 and Sec. 3.4:

* solo-run latency models, Eq. (1) for prefill and Eq. (2) for decode, with
  coefficients fitted to measured calls by least squares of the relative
  error (each sample's equation divided by its measured time);
* the contention guard: per cell of a grid over (prefill new tokens, prefill
  reused tokens, decode batch size, decode reused tokens in total, prefill
  partition size) the maximum decode slowdown observed; token counts in
  powers-of-4 cells, batch sizes in powers-of-2 cells;
* the number of prefill layers launched next to a decode iteration,
  N_PL = ceil(T_d * N_T / T_P) (Sec. 3.4), clamped to [1, N_T].
"""
from __future__ import annotations

import math
from typing import Dict, Iterable, Tuple

import numpy as np


def prefill_features(new_lens, prefix_lens) -> np.ndarray:
    """Eq. (1) terms: sum n^2, sum n r, sum n, 1."""
    n = np.asarray(new_lens, dtype=np.float64)
    r = np.asarray(prefix_lens, dtype=np.float64)
    return np.array([np.sum(n * n), np.sum(n * r), np.sum(n), 1.0])


def decode_features(seq_lens) -> np.ndarray:
    """Eq. (2) terms: sum r, bs, 1, with r = L - 1 reused tokens per sequence."""
    L = np.asarray(seq_lens, dtype=np.float64)
    return np.array([np.sum(L - 1.0), float(len(L)), 1.0])


def fit_relative(features: np.ndarray, times: np.ndarray) -> np.ndarray:
    """argmin_theta sum_j ((x_j . theta - t_j) / t_j)^2 (numpy's least squares
    on the rows x_j / t_j against 1; a term no sample exercises gets 0)."""
    X = np.asarray(features, dtype=np.float64)
    t = np.asarray(times, dtype=np.float64)
    A = X / t[:, None]
    theta = np.zeros(X.shape[1])
    used = np.any(A != 0.0, axis=0)
    sol, *_ = np.linalg.lstsq(A[:, used], np.ones(len(t)), rcond=None)
    theta[used] = sol
    return theta


def cell(x: int, base: int) -> int:
    """Smallest k with base^k >= x (0 for x <= 1)."""
    k, v = 0, 1
    while v < x:
        v *= base
        k += 1
    return k


def guard_cell(prefill_new, prefill_reused, decode_batch, decode_reused, prefill_cus) -> Tuple:
    return (int(prefill_cus), cell(prefill_new, 4), cell(prefill_reused, 4), cell(decode_batch, 2),
            cell(decode_reused, 4))


def guard_build(samples: Iterable[Tuple[Tuple, float]]) -> Dict[Tuple, float]:
    """samples: ((prefill_new, prefill_reused, decode_batch, decode_reused,
    prefill_cus), slowdown) -> {cell: maximum slowdown}."""
    cells: Dict[Tuple, float] = {}
    for key, s in samples:
        c = guard_cell(*key)
        cells[c] = max(cells.get(c, s), s)
    return cells


def guard_lookup(cells: Dict[Tuple, float], key) -> float:
    c = guard_cell(*key)
    if c in cells:
        return cells[c]
    same = [v for k, v in cells.items() if k[0] == c[0]]
    if same:
        return max(same)
    return max(cells.values()) if cells else 1.0


def prefill_layers(t_decode_ms: float, t_prefill_ms: float, n_layers: int) -> int:
    return int(min(max(math.ceil(t_decode_ms * n_layers / t_prefill_ms), 1), n_layers))
