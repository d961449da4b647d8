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
  N_PL = ceil(T_d * N_T / T_P) (Sec. 3.4), clamped to [1, N_T];
* the launch-imbalance factor that scales Eq. (1)'s terms for a single
  attention call (not from the paper: it restates the library's documented
  prefill launch rules and simulates the dispatch of the work-groups).
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


def prefill_launch(new_lens, prefix_lens, hkv: int, group: int, cus: int) -> Tuple[int, float]:
    """Kernel path (0: 8-wave, 1: 4-wave) and load-imbalance factor of a prefill
    call on `cus` CUs, as the library launches it with a split workspace.

    Launch rules: heads = hkv * ceil(group / 4); 64-position query blocks, one
    work-group per CU, unless their pairs (ceil(ceil(n/64) / 2) per sequence,
    times heads) number fewer than the CUs: then 32-position blocks, two per
    CU.  Blocks are paired (block nqb-1-i with block i) when the pairs fill
    whole rounds of the slots (pairs >= slots and rounds * slots * 20 <=
    pairs * 21); otherwise single blocks, heaviest first.  With 32-position
    blocks, the key-range split: units = sum ceil(n/32) * heads, max_nt = key
    tiles of the heaviest block; k = min(8, max(2, ceil(2 cus / units))) if
    units < cus, else 3 if units < 2 cus and max_nt >= 96, else no split;
    pieces of pt = max(4, ceil(max_nt / k)) tiles, at most 8 per block (a block
    of nt tiles has min(8, ceil(nt / pt)) pieces, piece p covering tiles
    [p nt / np, (p+1) nt / np)).  Block q of a sequence (n, r) reads
    ceil((r + min(q bm + bm, n)) / 64) key tiles.

    Dispatch: grid x fastest, then the sequence; grid x enumerates pairs (or
    blocks) times heads (times pieces, piece fastest, for the split).  Each
    work-group goes to a slot that frees no later than the earliest free time
    plus a window of 5% of the mean work-group's work, and among those to the
    CU that holds the fewest work-groups so far (then the lower slot index on
    its CU, then the lower CU): work-groups that differ by a tile or two finish
    together in practice, and the next ones spread over the CUs that freed.
    The slot stays busy for the work-group's work in tiles.  A CU that holds
    one work-group of a two-per-CU launch takes its work / 0.9.  Factor = max
    CU time (the sum of its work-groups' work) * cus / total work."""
    ng = (group + 3) // 4
    heads = hkv * ng
    lens = list(zip([int(n) for n in new_lens], [int(r) for r in prefix_lens]))
    max_n = max(n for n, _ in lens)

    def n_pairs(bm):
        return sum(((n + bm - 1) // bm + 1) // 2 for n, _ in lens) * heads

    if n_pairs(64) < cus:
        path, bm, per_cu = 1, 32, 2
    else:
        path, bm, per_cu = 0, 64, 1
    slots = per_cu * cus
    npairs = n_pairs(bm)
    rounds = (npairs + slots - 1) // slots
    paired = npairs >= slots and rounds * slots * 20 <= npairs * 21
    max_qb = (max_n + bm - 1) // bm
    pieces, pt = 1, 0
    if path == 1:
        units = sum((n + 31) // 32 for n, _ in lens) * heads
        max_nt = max((r + n + 63) // 64 for n, r in lens if n > 0)
        k = 1
        if units < cus:
            k = min(8, max(2, (2 * cus + units - 1) // units))
        elif units < 2 * cus and max_nt >= 96:
            k = 3
        if k > 1:
            pt = max(4, (max_nt + k - 1) // k)
            pieces = min(8, max(1, (max_nt + pt - 1) // pt))
    work = []
    for n, r in lens:
        nqb = (n + bm - 1) // bm

        def tiles(q):
            return (r + min(q * bm + bm, n) + 63) // 64

        if pieces > 1:
            for x in range(max_qb * heads * pieces):
                unit, piece = divmod(x, pieces)
                pair = unit // heads
                if pair >= nqb:
                    continue
                nt = tiles(nqb - 1 - pair)
                np_ = min(pieces, max(1, (nt + pt - 1) // pt))
                if piece < np_:
                    work.append((piece + 1) * nt // np_ - piece * nt // np_)
        else:
            gx = ((max_qb + 1) // 2 if paired else max_qb) * heads
            for x in range(gx):
                pair = x // heads
                last = nqb - 1 - pair
                if pair >= ((nqb + 1) // 2 if paired else nqb):
                    continue
                work.append(tiles(last) + (tiles(pair) if paired and pair != last else 0))
    total = float(sum(work))
    if total <= 0:
        return path, 1.0
    window = 0.05 * total / len(work)
    free = [[0.0, k, c] for k in range(per_cu) for c in range(cus)]
    load = [0.0] * cus
    count = [0] * cus
    for w in work:
        t0 = min(e[0] for e in free)
        s = min((e for e in free if e[0] <= t0 + window), key=lambda e: (count[e[2]], e[1], e[2]))
        load[s[2]] += w
        count[s[2]] += 1
        s[0] += w
    t_max = max(load[c] / (0.9 if per_cu == 2 and count[c] == 1 else 1.0) for c in range(cus))
    return path, t_max * cus / total


def prefill_features_launch(new_lens, prefix_lens, hkv: int, group: int, cus: int) -> Tuple[int, np.ndarray]:
    """Model index (0: 8-wave path, 2: 4-wave path) and Eq. (1) terms with the
    n^2, n r and n terms multiplied by the launch-imbalance factor."""
    path, kappa = prefill_launch(new_lens, prefix_lens, hkv, group, cus)
    x = prefill_features(new_lens, prefix_lens)
    x[:3] *= kappa
    return (0 if path == 0 else 2), x
