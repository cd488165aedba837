"""Comparison of the GPU path's results with the oracle's (test infrastructure).

TEST INFRASTRUCTURE: imported only by the tests, the smoke check and the
benchmark's CPU-baseline leg.

Agreement required (the parity bars of this path):
  * budgets: a head's block count may differ from the oracle's only where the
    cumulative-mass crossing of gamma is ambiguous, i.e. a count c is
    accepted when the oracle's sorted cumulative share satisfies
    P[c-1] >= gamma - window and (c == 1 or P[c-2] < gamma + window)
    (window 1e-4, shares computed in float64 from the oracle's fp32 masses).
  * block lists: per (head, block row) the symmetric difference between the
    GPU's list (as a set) and the oracle's selection at the GPU's count may
    hold only blocks whose oracle log-score lies within `window` of the
    oracle's K-th largest log-score (1e-4 in the log domain = 1e-4 relative
    in A); the GPU lists blocks from the highest score down.
  * attention: max |dO| <= 2e-2 and mean |dO| <= 2e-3 against the oracle's
    attention on the GPU's own lists.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

WINDOW = 1e-4
ATTN_MAX_ABS = 2e-2
ATTN_MEAN_ABS = 2e-3


class ParityError(AssertionError):
    pass


@dataclass
class Report:
    ambiguous_heads: list = field(default_factory=list)
    ambiguous_rows: int = 0
    ambiguous_blocks: int = 0
    rows_checked: int = 0
    max_abs: float = 0.0
    mean_abs: float = 0.0
    notes: list = field(default_factory=list)


def accepted_counts(cum_row: np.ndarray, gamma: float, min_budget_tokens: int, block_size: int,
                    window: float = WINDOW) -> set:
    """All block counts consistent with the budget rule under a `window` perturbation."""
    nk = cum_row.shape[0]
    p = cum_row.astype(np.float64)
    floor_blocks = -(-int(min_budget_tokens) // block_size)
    ok = set()
    if gamma >= 1.0:
        pre = {nk}
    else:
        pre = set()
        for c in range(1, nk + 1):
            reach = p[c - 1] >= gamma - window or c == nk
            before = c == 1 or p[c - 2] < gamma + window
            if reach and before:
                pre.add(c)
    for c in pre:
        ok.add(min(nk, max(c, floor_blocks)))
    return ok


def check_counts(gpu_counts, oracle_counts, oracle_cums, gamma, min_budget_tokens, block_size,
                 report: Report, window: float = WINDOW):
    gpu_counts = np.asarray(gpu_counts)
    for i, c in enumerate(gpu_counts.tolist()):
        if c == int(oracle_counts[i]):
            continue
        acc = accepted_counts(oracle_cums[i], gamma, min_budget_tokens, block_size, window)
        if c not in acc:
            raise ParityError(f"head {i}: GPU budget {c} blocks, oracle {int(oracle_counts[i])}, "
                              f"accepted {sorted(acc)}")
        report.ambiguous_heads.append(i)


def check_lists(gpu_count, gpu_index, logA, counts_used, num_q_heads, rows=None,
                report: Report | None = None, window: float = WINDOW,
                rank_order: bool = True, row_ratio: bool = False) -> Report:
    """Verify GPU lists against the oracle's shared scores `logA` [G, Mq, Nk].

    Lists are compared as sets; with `rank_order` they must also be listed
    from the highest score down (the library's documented order).
    `counts_used`: the per-head budget the GPU used (already validated);
    `row_ratio`: the per-row-ratio reading of Eq. 3 sets each row's count.
    """
    from oracle.proxyattn_oracle import row_budget
    report = report or Report()
    g_count, mq, nk = logA.shape
    gsize = num_q_heads // g_count
    gpu_count = np.asarray(gpu_count)
    gpu_index = np.asarray(gpu_index)
    row_list = range(mq) if rows is None else sorted(set(int(r) for r in rows))
    for g in range(g_count):
        for m in row_list:
            sc = logA[g, m, :m + 1].astype(np.float64)
            order = np.lexsort((np.arange(m + 1), -sc))
            for i in range(g * gsize, (g + 1) * gsize):
                kk = row_budget(counts_used[i], m, nk, row_ratio)
                if int(gpu_count[i, m]) != kk:
                    raise ParityError(f"head {i} row {m}: count {int(gpu_count[i, m])} != {kk}")
                lst_raw = gpu_index[i, m, :kk]
                lst = np.sort(lst_raw)
                if kk > 1 and np.any(np.diff(lst) <= 0):
                    raise ParityError(f"head {i} row {m}: list repeats a block: {lst_raw}")
                if kk and (lst.min() < 0 or lst.max() > m):
                    raise ParityError(f"head {i} row {m}: index out of range: {lst}")
                if np.any(gpu_index[i, m, kk:] != -1):
                    raise ParityError(f"head {i} row {m}: padding is not -1")
                ref = np.sort(order[:kk])
                report.rows_checked += 1
                if rank_order and kk > 1:
                    # listed from the highest score down (up to near-ties)
                    drop = np.diff(sc[lst_raw])
                    if np.any(drop > window):
                        raise ParityError(f"head {i} row {m}: list not in score order: "
                                          f"{lst_raw} scores {sc[lst_raw]}")
                if np.array_equal(lst, ref):
                    continue
                theta = sc[order[kk - 1]]
                diff = np.setxor1d(lst, ref)
                bad = diff[np.abs(sc[diff] - theta) > window]
                if bad.size:
                    raise ParityError(
                        f"head {i} row {m}: blocks {bad.tolist()} differ from the oracle with "
                        f"scores {sc[bad].tolist()} vs threshold {theta}")
                report.ambiguous_rows += 1
                report.ambiguous_blocks += int(diff.size)
    return report


def check_attention(gpu_out, oracle_out, report: Report | None = None, rows=None,
                    max_abs: float = ATTN_MAX_ABS, mean_abs: float = ATTN_MEAN_ABS) -> Report:
    report = report or Report()
    a = np.asarray(gpu_out, dtype=np.float64)
    b = np.asarray(oracle_out, dtype=np.float64)
    if rows is not None:
        a, b = a[rows], b[rows]
    if not np.all(np.isfinite(a)):
        raise ParityError("GPU attention output holds non-finite values")
    err = np.abs(a - b)
    report.max_abs = float(err.max()) if err.size else 0.0
    report.mean_abs = float(err.mean()) if err.size else 0.0
    if report.max_abs > max_abs or report.mean_abs > mean_abs:
        raise ParityError(f"attention max|dO|={report.max_abs:.3e} (<= {max_abs}), "
                          f"mean|dO|={report.mean_abs:.3e} (<= {mean_abs})")
    return report
