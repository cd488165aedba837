"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: a closed
form, a brute-force enumeration, a float64 full-matrix computation through a
library softmax, or a special case that reduces to a textbook routine.  The
paper prints no worked example, so whole-pipeline parity with the paper's own
numbers is unpinned; these pins cover every stage.
"""
import itertools
import math

import numpy as np
import pytest
from scipy.special import log_softmax, softmax

from oracle import proxyattn_oracle as O

RNG = np.random.default_rng(1234)


def _qkv(n, hq, hkv, d, scale=1.0, seed=0, bf16=False):
    rng = np.random.default_rng(seed)
    q = (scale * rng.standard_normal((n, hq, d))).astype(np.float32)
    k = rng.standard_normal((n, hkv, d)).astype(np.float32)
    v = rng.standard_normal((n, hkv, d)).astype(np.float32)
    if bf16:
        q, k, v = O.round_to_bf16(q), O.round_to_bf16(k), O.round_to_bf16(v)
    return q, k, v


def _dense_causal_f64(q, k, v, scale):
    """Textbook causal softmax attention on full N x N matrices, float64."""
    n, hq, d = q.shape
    rep = hq // k.shape[1]
    out = np.zeros((n, hq, d))
    for i in range(hq):
        s = scale * q[:, i, :].astype(np.float64) @ k[:, i // rep, :].astype(np.float64).T
        s[np.triu_indices(n, 1)] = -np.inf
        out[:, i, :] = softmax(s, axis=1) @ v[:, i // rep, :].astype(np.float64)
    return out


# ---------------------------------------------------------------- bf16 rounding
def test_round_to_bf16_table():
    # hand-checked values: exact, round down, round up, tie to even (both ways)
    x = np.array([1.0, 1.0 + 2 ** -9, 1.0 + 3 * 2 ** -9, 1.0 + 2 ** -8 + 2 ** -9,
                  -2.5, 3.0e38], dtype=np.float32)
    want = np.array([1.0, 1.0, 1.0 + 2 ** -7, 1.0 + 2 ** -7, -2.5, 2.9910598e38],
                    dtype=np.float32)
    got = O.round_to_bf16(x)
    assert np.array_equal(got[:5], want[:5])
    # largest finite values round into the bf16 grid (mantissa of 7 bits)
    assert got[5].view(np.uint32) & 0xFFFF == 0


def test_round_to_bf16_matches_nearest_grid_point():
    x = RNG.standard_normal(20000).astype(np.float32) * 10
    r = O.round_to_bf16(x).astype(np.float64)
    # neighbours on the bf16 grid: spacing 2^(e-7)
    e = np.floor(np.log2(np.abs(x.astype(np.float64))))
    ulp = 2.0 ** (e - 7)
    assert np.all(np.abs(r - x) <= ulp / 2 + 1e-30)


# ---------------------------------------------------------------- pooling, Eq. 2
def test_pool_group_of_one_is_identity():
    q, k, _ = _qkv(64, 4, 2, 16, bf16=True)
    qg, kg = O.pool_proxy_heads(q, k, num_groups=4, stride=1, dtype="bf16")
    for i in range(4):
        assert np.array_equal(qg[i], q[:, i, :])
        assert np.array_equal(kg[i], k[:, i // 2, :])


def test_pool_hand_example():
    # two query heads share one KV head; values chosen so the mean is exact
    q = np.zeros((8, 2, 2), np.float32)
    q[:, 0, :] = [[1, 2]] * 8
    q[:, 1, :] = [[3, -6]] * 8
    q[4, 1, :] = [5, 0]
    k = np.arange(16, dtype=np.float32).reshape(8, 1, 2)
    qg, kg = O.pool_proxy_heads(q, k, num_groups=1, stride=4, dtype="fp32")
    assert qg.shape == (1, 2, 2)
    assert np.array_equal(qg[0], [[2, -2], [3, 1]])          # tokens 0 and 4
    assert np.array_equal(kg[0], [[0, 1], [8, 9]])           # mean of the same key twice


def test_pool_identical_heads_is_identity():
    q, k, _ = _qkv(40, 1, 1, 8, bf16=True)
    q8 = np.repeat(q, 8, axis=1)
    k2 = np.repeat(k, 2, axis=1)
    qg, kg = O.pool_proxy_heads(q8, k2, num_groups=1, stride=2, dtype="bf16")
    assert np.array_equal(qg[0], q[::2, 0])
    assert np.array_equal(kg[0], k[::2, 0])


def test_pool_keys_follow_kv_head_of_each_query_head():
    # G not aligned with KV heads: group {q0,q1,q2} -> kv heads {0,0,1} (rep 2)
    q, k, _ = _qkv(12, 6, 3, 4)
    qg, kg = O.pool_proxy_heads(q, k, num_groups=2, stride=1, dtype="fp32")
    ref = (k[:, 0] + k[:, 0] + k[:, 1]) / 3
    assert np.allclose(kg[0], ref, rtol=1e-6, atol=1e-6)


# ------------------------------------------------------- proxy score, Eq. 1
def _brute_logscore(qg, kg, n, b, s, scale):
    """Full strided N'xN' log-softmax (scipy, float64), then block max by loops."""
    g_count, npr, d = qg.shape
    bp = b // s
    mq = -(-n // b)
    out = np.full((g_count, mq, mq), -np.inf)
    for g in range(g_count):
        sm = scale * qg[g].astype(np.float64) @ kg[g].astype(np.float64).T
        sm[np.triu_indices(npr, 1)] = -np.inf
        ls = log_softmax(sm, axis=1)
        for t in range(npr):
            for u in range(t + 1):
                m, nn = t // bp, u // bp
                out[g, m, nn] = max(out[g, m, nn], ls[t, u])
    return out


@pytest.mark.parametrize("n,b,s", [(256, 32, 4), (200, 32, 4), (128, 16, 1), (96, 32, 2)])
def test_logscore_matches_brute_force(n, b, s):
    q, k, _ = _qkv(n, 4, 2, 16, bf16=True, seed=n)
    qg, kg = O.pool_proxy_heads(q, k, 2, s, "bf16")
    sc = 1 / math.sqrt(16)
    got, lse = O.proxy_block_logscore(qg, kg, n, b, s, sc)
    ref = _brute_logscore(qg, kg, n, b, s, sc)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(got))
    assert np.max(np.abs(got[fin] - ref[fin])) < 2e-5


def test_logscore_zero_queries_closed_form():
    # Q = 0: every causal strided key gets 1/(t'+1); the block max comes from
    # the block's first row: logA[m, n] = -log(m*b'+1) for every n <= m.
    n, b, s = 512, 64, 4
    q = np.zeros((n, 2, 8), np.float32)
    _, k, _ = _qkv(n, 2, 1, 8)
    qg, kg = O.pool_proxy_heads(q, k, 1, s, "fp32")
    got, _ = O.proxy_block_logscore(qg, kg, n, b, s, 0.3)
    bp = b // s
    for m in range(n // b):
        assert np.allclose(got[0, m, :m + 1], -math.log(m * bp + 1), rtol=0, atol=1e-5)
        assert np.all(np.isneginf(got[0, m, m + 1:]))


def test_group_per_head_equals_per_head_estimation():
    # G = Hq: the proxy of head i is head i itself (exactly), so Eq. 1 reduces
    # to per-head block estimation on the head's own strided Q and K.
    n, b, s = 192, 32, 2
    q, k, _ = _qkv(n, 4, 2, 16, bf16=True, seed=7)
    qg, kg = O.pool_proxy_heads(q, k, 4, s, "bf16")
    got, _ = O.proxy_block_logscore(qg, kg, n, b, s, 0.25)
    for i in range(4):
        own = _brute_logscore(q[::s, i][None], k[::s, i // 2][None], n, b, s, 0.25)[0]
        fin = np.isfinite(own)
        assert np.max(np.abs(got[i][fin] - own[fin])) < 2e-5


def test_logscore_stride_one_equals_unstrided_definition():
    n, b = 64, 16
    q, k, _ = _qkv(n, 2, 2, 8, seed=3)
    qg, kg = O.pool_proxy_heads(q, k, 2, 1, "fp32")
    got, lse = O.proxy_block_logscore(qg, kg, n, b, 1, 0.5)
    for g in range(2):
        sm = 0.5 * q[:, g].astype(np.float64) @ k[:, g].astype(np.float64).T
        sm[np.triu_indices(n, 1)] = -np.inf
        p = softmax(sm, axis=1)
        A = np.zeros((n // b, n // b))
        for m in range(n // b):
            for nn in range(m + 1):
                A[m, nn] = p[m * b:(m + 1) * b, nn * b:(nn + 1) * b].max()
        assert np.allclose(np.exp(got[g])[np.tril_indices(n // b)], A[np.tril_indices(n // b)],
                           rtol=5e-5, atol=0)


# ------------------------------------------------------ Alg. 1: last-block mass
def test_mass_rows_sum_to_row_count():
    q, k, _ = _qkv(300, 4, 2, 16, seed=5)
    mass = O.lastblock_mass(q, k, 64, 0.25)
    assert mass.shape == (4, 5)
    assert np.allclose(mass.sum(axis=1), 64, rtol=1e-5)
    mass_small = O.lastblock_mass(q[:40], k[:40], 64, 0.25)       # N < b
    assert np.allclose(mass_small.sum(axis=1), 40, rtol=1e-5)


def test_mass_zero_queries_closed_form():
    # Q = 0: row t spreads 1/(t+1) over keys 0..t, so block n collects
    # sum_t |{u in n : u <= t}| / (t+1) over the last block's rows.
    n, b = 320, 64
    q = np.zeros((n, 1, 8), np.float32)
    _, k, _ = _qkv(n, 1, 1, 8)
    mass = O.lastblock_mass(q, k, b, 0.1)
    want = np.zeros(n // b)
    for t in range(n - b, n):
        for nn in range(n // b):
            want[nn] += max(0, min(t, (nn + 1) * b - 1) - nn * b + 1) / (t + 1)
    assert np.allclose(mass[0], want, rtol=1e-5)


def test_mass_matches_float64_softmax():
    n, b = 250, 64
    q, k, _ = _qkv(n, 2, 1, 16, seed=9, bf16=True)
    mass = O.lastblock_mass(q, k, b, 0.25)
    rows = np.arange(n - b, n)
    for i in range(2):
        s = 0.25 * q[rows, i].astype(np.float64) @ k[:, 0].astype(np.float64).T
        s[np.arange(n)[None, :] > rows[:, None]] = -np.inf
        p = softmax(s, axis=1).sum(axis=0)
        want = [p[j * b:(j + 1) * b].sum() for j in range(-(-n // b))]
        assert np.allclose(mass[i], want, rtol=1e-4, atol=1e-6)


# ------------------------------------------------------ Alg. 1: budget
def _brute_budget(mass_row, gamma):
    """Fewest blocks (any subset) whose share reaches gamma, by enumeration."""
    a = mass_row.astype(np.float64) / mass_row.astype(np.float64).sum()
    nk = len(a)
    for size in range(1, nk + 1):
        if any(sum(a[list(c)]) >= gamma for c in itertools.combinations(range(nk), size)):
            return size
    return nk


@pytest.mark.parametrize("seed", range(12))
def test_budget_matches_subset_enumeration(seed):
    rng = np.random.default_rng(seed)
    nk = int(rng.integers(2, 11))
    mass = rng.gamma(0.5, size=(1, nk)).astype(np.float32) + 1e-3
    for gamma in (0.5, 0.8, 0.9, 0.95):
        counts, cums = O.budget_counts(mass, gamma, 0, 64)
        want = _brute_budget(mass[0], gamma)
        p = cums[0].astype(np.float64)
        # skip draws whose crossing sits within fp32 rounding of gamma
        if np.any(np.abs(p - gamma) < 1e-5):
            continue
        assert counts[0] == want


def test_budget_monotone_in_gamma_and_limits():
    rng = np.random.default_rng(3)
    mass = rng.gamma(0.3, size=(6, 40)).astype(np.float32)
    prev = None
    for gamma in np.linspace(0.05, 0.999, 25):
        c, _ = O.budget_counts(mass, gamma, 0, 128)
        if prev is not None:
            assert np.all(c >= prev)
        prev = c
    full, _ = O.budget_counts(mass, 1.0, 0, 128)
    assert np.all(full == 40)
    floor, _ = O.budget_counts(mass, 0.05, 2048, 128)
    assert np.all(floor >= 16)
    cap, _ = O.budget_counts(mass, 0.05, 10 ** 9, 128)
    assert np.all(cap == 40)


def test_budget_dominant_sink_is_one_block():
    n, b, d = 512, 64, 16
    q, k, _ = _qkv(n, 2, 1, d, seed=2)
    # key 0 aligned with every query: logit +40 for every row
    q[:, :, 0] = 10.0
    k[0, 0, :] = 0
    k[0, 0, 0] = 16.0
    mass = O.lastblock_mass(q, k, b, 1 / math.sqrt(d))
    counts, _ = O.budget_counts(mass, 0.95, 0, b)
    assert np.all(counts == 1)


# ------------------------------------------------------ Eq. 3: selection
def _brute_topk(scores, kk):
    best, best_set = -np.inf, None
    for c in itertools.combinations(range(len(scores)), kk):     # lexicographic order
        s = float(np.sum(np.exp(scores[list(c)].astype(np.float64))))
        if s > best * (1 + 1e-12):
            best, best_set = s, c
    return np.array(best_set)


def test_select_matches_subset_enumeration():
    rng = np.random.default_rng(11)
    mq = 9
    logA = np.full((1, mq, mq), -np.inf, np.float32)
    for m in range(mq):
        logA[0, m, :m + 1] = -rng.exponential(3.0, m + 1).astype(np.float32)
    counts = np.array([1, 3, 5, 9], np.int32)
    bc, bi = O.select_blocks(logA, counts, 4)
    for i in range(4):
        for m in range(mq):
            kk = min(counts[i], m + 1)
            assert bc[i, m] == kk
            assert np.array_equal(bi[i, m, :kk], _brute_topk(logA[0, m, :m + 1], kk))
            assert np.all(bi[i, m, kk:] == -1)


def test_select_ties_go_to_lower_index_and_lists_nest():
    mq = 6
    logA = np.full((1, mq, mq), -np.inf, np.float32)
    for m in range(mq):
        logA[0, m, :m + 1] = -1.0                     # all tied (the Q = 0 case)
    counts = np.array([2, 4], np.int32)
    bc, bi = O.select_blocks(logA, counts, 2)
    for m in range(mq):
        assert np.array_equal(bi[0, m, :bc[0, m]], np.arange(min(2, m + 1)))
        assert np.array_equal(bi[1, m, :bc[1, m]], np.arange(min(4, m + 1)))
        assert set(bi[0, m, :bc[0, m]]) <= set(bi[1, m, :bc[1, m]])


def test_row_ratio_reading_matches_rational_definition_and_enumeration():
    """Per-row-ratio reading of Eq. 3: K = ceil(b_i (m+1)) with b_i = count/Nk,
    checked with exact rationals, and the lists against subset enumeration."""
    from fractions import Fraction
    rng = np.random.default_rng(12)
    mq = 9
    logA = np.full((1, mq, mq), -np.inf, np.float32)
    for m in range(mq):
        logA[0, m, :m + 1] = -rng.exponential(3.0, m + 1).astype(np.float32)
    counts = np.array([1, 2, 4, 7, 9], np.int32)
    bc, bi = O.select_blocks(logA, counts, 5, row_ratio=True)
    for i, c in enumerate(counts):
        for m in range(mq):
            r = Fraction(int(c), mq) * (m + 1)
            kk = -((-r.numerator) // r.denominator)        # ceil of the rational
            assert bc[i, m] == kk == O.row_budget(c, m, mq, True)
            assert 1 <= kk <= min(int(c), m + 1)
            assert np.array_equal(bi[i, m, :kk], _brute_topk(logA[0, m, :m + 1], kk))
            assert np.all(bi[i, m, kk:] == -1)
        # the last row keeps the head's whole budget, as in the constant reading
        assert bc[i, mq - 1] == c
    # a full budget keeps every causal block in both readings
    full, _ = O.select_blocks(logA, np.array([mq], np.int32), 1, row_ratio=True)
    assert np.array_equal(full[0], np.arange(1, mq + 1))


def test_static_topk_gives_every_head_of_a_group_the_same_lists():
    rng = np.random.default_rng(13)
    mq = 7
    logA = np.full((2, mq, mq), -np.inf, np.float32)
    for g in range(2):
        for m in range(mq):
            logA[g, m, :m + 1] = rng.standard_normal(m + 1).astype(np.float32)
    bc, bi = O.select_blocks(logA, np.full(6, 3, np.int32), 6)
    for i in (1, 2):
        assert np.array_equal(bi[i], bi[0]) and np.array_equal(bi[3 + i], bi[3])
    assert np.array_equal(bc[0], np.minimum(3, np.arange(1, mq + 1)))


# ------------------------------------------------------ attention
@pytest.mark.parametrize("n,b", [(256, 64), (200, 64), (50, 64)])
def test_full_lists_reproduce_dense_causal_attention(n, b):
    q, k, v = _qkv(n, 4, 2, 16, seed=n, bf16=True)
    bc, bi = O.full_causal_lists(n, 4, b)
    out, lse = O.block_sparse_attention(q, k, v, bc, bi, b, 0.25)
    ref = _dense_causal_f64(q, k, v, 0.25)
    assert np.max(np.abs(out - ref)) < 2e-5
    # lse against float64 logsumexp
    s = 0.25 * q[:, 0].astype(np.float64) @ k[:, 0].astype(np.float64).T
    s[np.triu_indices(n, 1)] = -np.inf
    ref_lse = np.log(np.exp(s - s.max(1, keepdims=True)).sum(1)) + s.max(1)
    assert np.max(np.abs(lse[0] - ref_lse)) < 2e-5


def test_constant_values_give_constant_output_for_any_mask():
    n, b = 256, 32
    q, k, _ = _qkv(n, 2, 1, 8, seed=4)
    v = np.full((n, 1, 8), 0.75, np.float32)
    rng = np.random.default_rng(0)
    mq = n // b
    bc = np.zeros((2, mq), np.int32)
    bi = np.full((2, mq, mq), -1, np.int32)
    for i in range(2):
        for m in range(mq):
            kk = int(rng.integers(1, m + 2))
            bi[i, m, :kk] = np.sort(rng.choice(m + 1, kk, replace=False))
            bc[i, m] = kk
    out, _ = O.block_sparse_attention(q, k, v, bc, bi, b, 0.35)
    assert np.allclose(out, 0.75, atol=1e-6)


def test_diagonal_only_lists_are_local_block_attention():
    n, b = 192, 64
    q, k, v = _qkv(n, 2, 2, 8, seed=6)
    mq = n // b
    bc = np.ones((2, mq), np.int32)
    bi = np.full((2, mq, mq), -1, np.int32)
    for m in range(mq):
        bi[:, m, 0] = m
    out, _ = O.block_sparse_attention(q, k, v, bc, bi, b, 0.35)
    for m in range(mq):
        sl = slice(m * b, (m + 1) * b)
        ref = _dense_causal_f64(q[sl], k[sl], v[sl], 0.35)
        assert np.max(np.abs(out[sl] - ref)) < 2e-5


def test_pipeline_full_budget_equals_dense_attention():
    n, b, s = 512, 64, 4
    q, k, v = _qkv(n, 8, 2, 16, seed=8, bf16=True)
    res = O.proxyattn_prefill(q, k, v, num_groups=2, block_size=b, stride=s, gamma=1.0,
                              dtype="bf16")
    assert np.all(res["counts"] == n // b)
    ref = _dense_causal_f64(q, k, v, 0.25)
    assert np.max(np.abs(res["out"] - ref)) < 2e-5


def test_pipeline_sampled_rows_equal_full_run():
    n, b, s = 384, 64, 4
    q, k, v = _qkv(n, 4, 2, 16, seed=10, bf16=True)
    full = O.proxyattn_prefill(q, k, v, num_groups=2, block_size=b, stride=s, gamma=0.8)
    rows = [0, 5, 130, 200, n - 1]
    part = O.proxyattn_prefill(q, k, v, num_groups=2, block_size=b, stride=s, gamma=0.8,
                               query_rows=rows)
    # same math on fewer rows; BLAS blocking may move the last bit
    assert np.allclose(full["out"][rows], part["out"][rows], rtol=0, atol=1e-6)
    for m in sorted(set(r // b for r in rows)):
        assert np.array_equal(full["block_index"][:, m], part["block_index"][:, m])


# ------------------------------------------------------ head-similarity diagnostics (Eq. 4)
def test_head_overlap_closed_forms():
    """Q = 0 gives uniform attention 1/(t+1): Score = k/(t+1) everywhere; with
    n sink tokens removed the top-k are tokens n..n+k-1 (the zeros rank last),
    and renormalising scales every remaining token to 1/(t+1-n)."""
    n, t, topk = 64, 40, 9
    q = np.zeros((n, 4, 8), np.float32)
    k = np.random.default_rng(3).standard_normal((n, 2, 8)).astype(np.float32)
    s = O.head_overlap(q, k, t, topk, 0.3)
    assert np.allclose(s, topk / (t + 1), atol=1e-6)
    s = O.head_overlap(q, k, t, topk, 0.3, sink_tokens=4)
    assert np.allclose(s, topk / (t + 1), atol=1e-6)
    s = O.head_overlap(q, k, t, topk, 0.3, sink_tokens=4, renormalize=True)
    assert np.allclose(s, topk / (t + 1 - 4), atol=1e-6)
    # k beyond the visible tokens: every head's whole mass
    assert np.allclose(O.head_overlap(q, k, t, 10 * n, 0.3), 1.0, atol=1e-6)


def test_head_overlap_identical_heads_and_column_dominance():
    rng = np.random.default_rng(4)
    n, t, topk = 200, 150, 20
    base = rng.standard_normal((n, 1, 16)).astype(np.float32)
    q_same = np.repeat(base, 4, axis=1)
    k = rng.standard_normal((n, 1, 16)).astype(np.float32)
    s = O.head_overlap(q_same, k, t, topk, 0.5)
    assert np.allclose(s, s[0, 0], atol=1e-6)              # every entry = the common top-k mass
    q = rng.standard_normal((n, 6, 16)).astype(np.float32)
    k2 = rng.standard_normal((n, 2, 16)).astype(np.float32)
    s = O.head_overlap(q, k2, t, topk, 0.5)
    a = O.token_attention(q, k2, t, 0.5).astype(np.float64)
    for i in range(6):
        # a head's own top-k holds the most of its mass of any k tokens ...
        assert np.all(s[i, i] >= s[:, i] - 1e-6)
        # ... which is the sum of its k largest probabilities (brute force)
        assert abs(s[i, i] - np.sort(a[i])[::-1][:topk].sum()) < 1e-6


def test_shared_ranking_curves_reduce_to_own_ranking_for_identical_heads():
    rng = np.random.default_rng(5)
    n, t = 128, 127
    q = np.repeat(rng.standard_normal((n, 1, 8)).astype(np.float32), 3, axis=1)
    k = rng.standard_normal((n, 1, 8)).astype(np.float32)
    shared, own = O.shared_ranking_curves(q, k, t, 0.4, [1, 8, 64, 128])
    assert np.allclose(shared, own, atol=1e-9)
    assert np.allclose(own[:, -1], 1.0, atol=1e-6)
    q2 = rng.standard_normal((n, 3, 8)).astype(np.float32)
    shared, own = O.shared_ranking_curves(q2, k, t, 0.4, [1, 8, 64, 128])
    assert np.all(shared <= own + 1e-12)                  # the own ranking is optimal


# ------------------------------------------------------ GQA head mapping and softmax scale
# References below come from torch's scaled_dot_product_attention in float64
# with enable_gqa=True: the library repeats each KV head over its
# Hq/Hkv consecutive query heads itself, and takes the scale as an argument.
# Every case has Hq/Hkv = 2 or 3 with distinct KV heads, nonzero queries and
# a scale other than 1/sqrt(d), so reading KV head i % Hkv instead of
# i // (Hq/Hkv), or dropping the scale, fails each of them (both mutations
# were applied to a copy of the oracle and made every one of these fail).
def _sdpa_f64(q, k, v, scale, causal):
    """q [Hq, Tq, d], k [Hkv, Tk, d], v [Hkv, Tk, e] -> [Hq, Tq, e], float64."""
    import torch
    import torch.nn.functional as F
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x, dtype=np.float64))[None]
    o = F.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=causal, scale=float(scale),
                                       enable_gqa=True)
    return o[0].numpy()


def _sdpa_token_probs(q, k, t, scale):
    """Probabilities of query token t over keys 0..t for every head: SDPA
    with V = the identity, so the output rows are the softmax rows."""
    hkv = k.shape[1]
    eye = np.broadcast_to(np.eye(t + 1), (hkv, t + 1, t + 1))
    return _sdpa_f64(q[t:t + 1].transpose(1, 0, 2), k[:t + 1].transpose(1, 0, 2), eye, scale,
                     causal=False)[:, 0, :]


@pytest.mark.parametrize("hq,hkv,t", [(6, 2, 37), (4, 2, 1), (6, 3, 59)])
def test_token_attention_gqa_and_scale_match_sdpa(hq, hkv, t):
    q, k, _ = _qkv(60, hq, hkv, 16, scale=1.5, seed=21)
    scale = 0.37                                      # 1/sqrt(16) = 0.25
    got = O.token_attention(q, k, t, scale)
    want = _sdpa_token_probs(q, k, t, scale)
    assert got.shape == want.shape == (hq, t + 1)
    assert np.allclose(got, want, rtol=2e-5, atol=1e-7)


@pytest.mark.parametrize("sink,renorm", [(0, False), (3, False), (3, True)])
def test_head_overlap_matches_brute_force_topk_sums_of_sdpa(sink, renorm):
    """Eq. 4 by brute force on the float64 reference probabilities: for each
    head i the k tokens with the largest probability, then every head's mass
    on them (after the sink removal and renormalisation the call asks for)."""
    hq, hkv, n, t, topk = 6, 2, 120, 97, 11
    q, k, _ = _qkv(n, hq, hkv, 16, scale=1.5, seed=22)
    scale = 0.31
    a = _sdpa_token_probs(q, k, t, scale)
    a[:, :sink] = 0.0
    if renorm:
        a = a / a.sum(axis=1, keepdims=True)
    want = np.empty((hq, hq))
    for i in range(hq):
        order = sorted(range(t + 1), key=lambda u: (-a[i, u], u))
        # the ranking is not decided by rounding: the k-th and (k+1)-th
        # probabilities are far apart compared to fp32's error
        assert a[i, order[topk - 1]] - a[i, order[topk]] > 1e-5
        want[i] = a[:, order[:topk]].sum(axis=1)
    got = O.head_overlap(q, k, t, topk, scale, sink_tokens=sink, renormalize=renorm)
    assert np.allclose(got, want, rtol=1e-5, atol=1e-7)


@pytest.mark.parametrize("n,b,hq,hkv", [(200, 32, 4, 2), (256, 64, 6, 2), (100, 64, 6, 3)])
def test_lastblock_mass_gqa_and_scale_match_sdpa(n, b, hq, hkv):
    """Alg. 1, first two steps: causal SDPA over the whole sequence with V =
    the key-block indicator (V[u, n] = 1 when key u lies in block n) gives,
    for every query row, its attention mass per key block; the mass is the
    sum of those rows over the last min(b, N) query tokens."""
    q, k, _ = _qkv(n, hq, hkv, 16, scale=1.5, seed=23)
    scale = 0.41
    nk = -(-n // b)
    ind = np.zeros((n, nk))
    ind[np.arange(n), np.arange(n) // b] = 1.0
    per_row = _sdpa_f64(q.transpose(1, 0, 2), k.transpose(1, 0, 2),
                        np.broadcast_to(ind, (hkv, n, nk)), scale, causal=True)
    want = per_row[:, max(0, n - b):, :].sum(axis=1)
    got = O.lastblock_mass(q, k, b, scale)
    assert np.allclose(got, want, rtol=2e-5, atol=2e-6)
