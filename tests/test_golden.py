"""The oracle against the hand-derived fixtures in tests/golden/.

The paper prints no worked example, so each fixture is a small case whose
expected values follow by hand from the paper's definitions (or a closed
form); every file states the passage it follows and the derivation.  None of
the stored values comes from the oracle or from the GPU path.
"""
import json
import math
import os

import numpy as np
import pytest

from oracle import proxyattn_oracle as O

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name), encoding="utf-8") as fh:
        fx = json.load(fh)
    assert fx["cite"] and fx["derivation"]
    return fx


def test_every_fixture_is_checked():
    names = sorted(f for f in os.listdir(GOLDEN) if f.endswith(".json"))
    assert names == ["budget_alg1.json", "logscore_eq1_zero_queries.json",
                     "overlap_eq4_uniform.json", "pool_eq2_two_heads.json",
                     "select_eq3_ties.json"]


def test_pool_eq2_two_heads():
    fx = _load("pool_eq2_two_heads.json")
    kt = np.asarray(fx["k_tokens"], np.float32)
    n = kt.shape[0]
    q = np.zeros((n, 2, 2), np.float32)
    q[:, 0, :] = fx["q_head0"]
    q[:, 1, :] = fx["q_head1"]
    q[4, 1, :] = fx["q_head1_token4"]
    k = kt.reshape(n, 1, 2)
    qg, kg = O.pool_proxy_heads(q, k, num_groups=fx["num_groups"], stride=fx["stride"],
                                dtype=fx["dtype"])
    assert np.array_equal(qg[0], np.asarray(fx["expected_qg"], np.float32))
    assert np.array_equal(kg[0], np.asarray(fx["expected_kg"], np.float32))


@pytest.mark.parametrize("case", range(6))
def test_budget_alg1(case):
    fx = _load("budget_alg1.json")
    c = fx["cases"][case]
    mass = np.asarray([fx["mass"]], np.float32)
    counts, _ = O.budget_counts(mass, c["gamma"], c["min_budget_tokens"], fx["block_size"])
    assert int(counts[0]) == c["expected_count"]


def test_select_eq3_ties():
    fx = _load("select_eq3_ties.json")
    rows = fx["log_scores"]
    mq = len(rows)
    logA = np.full((1, mq, mq), -np.inf, np.float32)
    for m, row in enumerate(rows):
        for n, v in enumerate(row):
            if v is not None:
                logA[0, m, n] = v
    counts = np.asarray(fx["counts"], np.int32)
    bc, bi = O.select_blocks(logA, counts, num_q_heads=len(counts))
    for i, want_rows in enumerate(fx["expected_sets"]):
        for m, want in enumerate(want_rows):
            got = bi[i, m, :bc[i, m]]
            assert sorted(got.tolist()) == want, (i, m, got)
            assert np.all(bi[i, m, bc[i, m]:] == -1)


def test_logscore_eq1_zero_queries():
    fx = _load("logscore_eq1_zero_queries.json")
    n, b, s, d = fx["seq_len"], fx["block_size"], fx["stride"], fx["head_dim"]
    rng = np.random.default_rng(3)
    q = np.zeros((n, 1, d), np.float32)
    k = rng.standard_normal((n, 1, d)).astype(np.float32)
    qg, kg = O.pool_proxy_heads(q, k, num_groups=1, stride=s, dtype="fp32")
    logA, _ = O.proxy_block_logscore(qg, kg, n, b, s, 1.0 / math.sqrt(d))
    want = fx["expected_logA"]
    for m, row in enumerate(want):
        for col, v in enumerate(row):
            if v is None:
                assert logA[0, m, col] == -np.inf
            else:
                assert abs(float(logA[0, m, col]) - v) <= fx["tolerance"], (m, col)


@pytest.mark.parametrize("case", range(4))
def test_overlap_eq4_uniform(case):
    fx = _load("overlap_eq4_uniform.json")
    c = fx["cases"][case]
    rng = np.random.default_rng(5)
    n, hq, hkv, d = fx["seq_len"], fx["num_q_heads"], fx["num_kv_heads"], fx["head_dim"]
    q = np.zeros((n, hq, d), np.float32)
    k = rng.standard_normal((n, hkv, d)).astype(np.float32)
    score = O.head_overlap(q, k, fx["query_token"], c["topk"], 1.0 / math.sqrt(d),
                           sink_tokens=c["sink_tokens"], renormalize=c["renormalize"])
    assert score.shape == (hq, hq)
    assert np.max(np.abs(score - c["expected"])) <= fx["tolerance"]
