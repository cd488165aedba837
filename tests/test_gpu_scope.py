"""GPU parity at the sizes and settings the benchmark times (Sec. 4.3's
speed setting, the sparsity band of Table 8, the proxy-head settings of
Sec. 4.1): every configuration that is timed is also checked against the
oracle here, in the launch configuration the benchmark uses (the K/V copy
prepared once, then the blocked attention calls).

Bars as in test_gpu_parity.py: pooled heads bit-exact, |dlogA| <= 2e-4,
last-block masses within 1e-4 of the row total, budgets and lists identical
up to the 1e-4 threshold window, attention max|dO| <= 2e-2 and
mean|dO| <= 2e-3 (and |dlse| <= 4e-3) on the oracle's attention over the
GPU's own lists.  What each test checks in full and what on sampled rows is
stated in its docstring; sampled rows are seeded (12345) and always include
the last row.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import check as C
from oracle import proxyattn_oracle as O
from paper_2509_24745_amd.synth import WORKLOADS

pytestmark = pytest.mark.gpu

LOGA_TOL = 2e-4
MASS_RTOL = 1e-4
LSE_TOL = 4e-3


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util as U
    return U


def _sample_rows(n: int, per_head: int) -> np.ndarray:
    rng = np.random.default_rng(12345)
    return np.unique(np.concatenate([rng.integers(0, n, per_head), [n - 1]]))


class Path:
    """One layer on the GPU through the C ABI: estimate once, then any number
    of selections, each followed by the blocked sparse attention on the K/V
    copy prepared once (the benchmark's sequence of calls)."""

    def __init__(self, U, wl, q, k, v):
        from paper_2509_24745_amd import proxyattn as pa
        self.pa, self.U, self.wl = pa, U, wl
        self.prob = prob = U.problem_of(wl)
        self.q, self.k, self.v = q, k, v
        self.qd, self.kd, self.vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
        self.bufs = bufs = pa.Buffers(prob)
        self.kvb = torch.empty(pa.proxyattn_kv_blocked_size(prob), dtype=torch.uint8,
                               device="cuda")
        self.qws = torch.empty(pa.proxyattn_blocked_workspace_size(prob), dtype=torch.uint8,
                               device="cuda")
        pa.proxyattn_estimate(prob, self.qd, self.kd, bufs.logscore, bufs.mass, bufs.workspace)
        pa.proxyattn_prepare_kv(prob, self.kd, self.vd, self.kvb)
        torch.cuda.synchronize()
        self.qg, self.kg = U.pooled_from_workspace(prob, bufs.workspace)
        self.logA = U.to_host(bufs.logscore)
        self.mass = U.to_host(bufs.mass)

    def budget(self, gamma, beta=0):
        self.pa.proxyattn_budget(self.prob, self.bufs.mass, gamma, beta, self.bufs.head_count)
        torch.cuda.synchronize()
        return self.U.to_host(self.bufs.head_count)

    def select(self, mode, head_count=None):
        hc = self.bufs.head_count if head_count is None else torch.from_numpy(
            np.ascontiguousarray(head_count, dtype=np.int32)).cuda()
        self.pa.proxyattn_select_topk(self.prob, self.bufs.logscore, hc, mode,
                                      self.bufs.block_count, self.bufs.block_index)
        torch.cuda.synchronize()
        return self.U.to_host(self.bufs.block_count), self.U.to_host(self.bufs.block_index)

    def attend(self, rows=None):
        b = self.bufs
        self.pa.proxyattn_block_sparse_prefill_blocked(self.prob, self.qd, self.kvb,
                                                       b.block_count, b.block_index, b.out,
                                                       b.lse, self.qws)
        torch.cuda.synchronize()
        if rows is None:
            return self.U.to_host(b.out), self.U.to_host(b.lse)
        r = torch.from_numpy(rows).cuda()
        return self.U.to_host(b.out[r]), self.U.to_host(b.lse[:, r])


def _check_estimate(path, oa, omass, est_rows=None):
    wl = path.wl
    qg, kg = O.pool_proxy_heads(path.q, path.k, wl.num_proxy_groups, wl.stride, wl.dtype)
    assert np.array_equal(path.qg, qg) and np.array_equal(path.kg, kg), "pooled heads differ"
    ga, ob = path.logA, oa
    if est_rows is not None:
        ga, ob = ga[:, est_rows], ob[:, est_rows]
    assert np.array_equal(np.isneginf(ga), np.isneginf(ob)), "-inf pattern differs"
    fin = np.isfinite(ob)
    dla = float(np.max(np.abs(ga[fin] - ob[fin])))
    assert dla <= LOGA_TOL, f"max |dlogA| = {dla}"
    dm = float(np.max(np.abs(path.mass - omass))) / min(wl.block_size, wl.seq_len)
    assert dm <= MASS_RTOL, f"max |dmass|/rows = {dm}"
    return dla, dm


def _check_attention(path, bc, bi, rows, rep):
    wl = path.wl
    out, lse = path.attend(rows)
    ref, ref_lse = O.block_sparse_attention(path.q, path.k, path.v, bc, bi, wl.block_size,
                                            O.default_scale(wl.head_dim), query_rows=rows)
    if rows is not None:
        ref, ref_lse = ref[rows], ref_lse[:, rows]
    C.check_attention(out, ref, rep)
    dl = float(np.abs(lse - ref_lse).max())
    assert dl <= LSE_TOL, f"max |dlse| = {dl}"
    return dl


def _sparsity(bc, wl):
    mq = wl.num_blocks
    return 1.0 - bc.sum() / (wl.num_q_heads * mq * (mq + 1) / 2)


@pytest.mark.parametrize("sigma", [0.1, 0.3, 0.6])
def test_128k_gamma_sigma_grid(sigma):
    """The 128K Llama-3-8B-shaped layer at every point of its threshold x head
    deviation grid (gamma in {0.90, 0.95, 0.99}, sigma in {0.1, 0.3, 0.6}):
    pooled heads, every block score and last-block mass, every head's budget
    and every block row's list in full; attention on 64 sampled query rows.
    At sigma = 0.3 also the budget variants (the per-row-ratio reading of
    Eq. 3 and a static Top-K on the same scores) and ascending lists."""
    U = _gpu()
    pa_ = __import__("paper_2509_24745_amd.proxyattn", fromlist=["x"])
    wl = WORKLOADS["llama3_8b_n131072"].replace(noise=sigma)
    print(f"\n[128K grid] sigma={sigma}", flush=True)
    q, k, v = U.inputs(wl)
    path = Path(U, wl, q, k, v)
    sc = O.default_scale(wl.head_dim)
    qg, kg = O.pool_proxy_heads(q, k, wl.num_proxy_groups, wl.stride, wl.dtype)
    oa, _ = O.proxy_block_logscore(qg, kg, wl.seq_len, wl.block_size, wl.stride, sc)
    omass = O.lastblock_mass(q, k, wl.block_size, sc)
    dla, dm = _check_estimate(path, oa, omass)
    rows = _sample_rows(wl.seq_len, 64)
    for gamma in (0.90, 0.95, 0.99):
        rep = C.Report()
        counts = path.budget(gamma)
        ocounts, cums = O.budget_counts(omass, gamma, 0, wl.block_size)
        C.check_counts(counts, ocounts, cums, gamma, 0, wl.block_size, rep)
        bc, bi = path.select(pa_.TOPK_CONSTANT)
        C.check_lists(bc, bi, oa, counts, wl.num_q_heads, report=rep)
        dl = _check_attention(path, bc, bi, rows, rep)
        print(f"  gamma={gamma}: sparsity={_sparsity(bc, wl):.3f} |dlogA|={dla:.2e} "
              f"|dmass|/rows={dm:.2e} max|dO|={rep.max_abs:.2e} mean|dO|={rep.mean_abs:.2e} "
              f"|dlse|={dl:.2e} ambiguous heads={len(rep.ambiguous_heads)} "
              f"rows={rep.ambiguous_rows} of {rep.rows_checked}", flush=True)
    if sigma != 0.3:
        return
    counts = path.budget(0.95)
    # ascending lists: the same sets as the rank-order lists, sorted
    bc_r, bi_r = path.select(pa_.TOPK_CONSTANT)
    bc_a, bi_a = path.select(pa_.TOPK_CONSTANT | pa_.LIST_ASCENDING)
    assert np.array_equal(bc_a, bc_r)
    big = np.iinfo(np.int32).max
    want = np.sort(np.where(bi_r >= 0, bi_r, big), axis=-1)
    want[want == big] = -1
    assert np.array_equal(bi_a, want), "ascending lists are not the sorted rank-order lists"
    # per-row-ratio reading of Eq. 3 on the GPU's budgets
    rep = C.Report()
    bc, bi = path.select(pa_.TOPK_ROW_RATIO)
    C.check_lists(bc, bi, oa, counts, wl.num_q_heads, report=rep, row_ratio=True)
    _check_attention(path, bc, bi, rows, rep)
    print(f"  row ratio: sparsity={_sparsity(bc, wl):.3f} max|dO|={rep.max_abs:.2e} "
          f"ambiguous rows={rep.ambiguous_rows}", flush=True)
    # static Top-K: every head the mean dynamic budget
    static = np.full(wl.num_q_heads, int(round(counts.mean())), np.int32)
    rep = C.Report()
    bc, bi = path.select(pa_.TOPK_CONSTANT, static)
    C.check_lists(bc, bi, oa, static, wl.num_q_heads, report=rep)
    _check_attention(path, bc, bi, rows, rep)
    print(f"  static top-{static[0]}: sparsity={_sparsity(bc, wl):.3f} max|dO|={rep.max_abs:.2e} "
          f"ambiguous rows={rep.ambiguous_rows}", flush=True)


@pytest.mark.parametrize("groups,beta", [(1, 0), (2, 0), (4, 0), (7, 0), (7, 2048)])
def test_64k_qwen_proxy_groups(groups, beta):
    """The 64K Qwen2.5-7B-shaped layer (28 query heads on 4 KV heads,
    heterogeneous heads) at 1, 2, 4 and 7 proxy groups with no minimum
    budget, and at 7 groups with the paper's 2048-token minimum budget (Sec.
    4.1): every score, budget and list in full; attention on 128 sampled
    query rows."""
    U = _gpu()
    pa_ = __import__("paper_2509_24745_amd.proxyattn", fromlist=["x"])
    wl = WORKLOADS["qwen25_7b_n65536"].replace(num_proxy_groups=groups, min_budget_tokens=beta)
    print(f"\n[64K qwen] G={groups} beta={beta}", flush=True)
    q, k, v = U.inputs(wl)
    path = Path(U, wl, q, k, v)
    sc = O.default_scale(wl.head_dim)
    qg, kg = O.pool_proxy_heads(q, k, groups, wl.stride, wl.dtype)
    oa, _ = O.proxy_block_logscore(qg, kg, wl.seq_len, wl.block_size, wl.stride, sc)
    omass = O.lastblock_mass(q, k, wl.block_size, sc)
    dla, dm = _check_estimate(path, oa, omass)
    rep = C.Report()
    counts = path.budget(wl.gamma, beta)
    ocounts, cums = O.budget_counts(omass, wl.gamma, beta, wl.block_size)
    C.check_counts(counts, ocounts, cums, wl.gamma, beta, wl.block_size, rep)
    bc, bi = path.select(pa_.TOPK_CONSTANT)
    C.check_lists(bc, bi, oa, counts, wl.num_q_heads, report=rep)
    dl = _check_attention(path, bc, bi, _sample_rows(wl.seq_len, 128), rep)
    print(f"  sparsity={_sparsity(bc, wl):.3f} |dlogA|={dla:.2e} |dmass|/rows={dm:.2e} "
          f"max|dO|={rep.max_abs:.2e} mean|dO|={rep.mean_abs:.2e} |dlse|={dl:.2e} "
          f"ambiguous heads={len(rep.ambiguous_heads)} rows={rep.ambiguous_rows} "
          f"of {rep.rows_checked}", flush=True)


def test_32k_llama_full_attention():
    """The 32K Llama-3-8B-shaped layer in full: every score, mass, budget and
    list, and the attention output and lse of every query row of every
    head."""
    U = _gpu()
    pa_ = __import__("paper_2509_24745_amd.proxyattn", fromlist=["x"])
    wl = WORKLOADS["llama3_8b_n32768"]
    q, k, v = U.inputs(wl)
    path = Path(U, wl, q, k, v)
    orc = O.proxyattn_prefill(q, k, None, num_groups=wl.num_proxy_groups,
                              block_size=wl.block_size, stride=wl.stride, gamma=wl.gamma)
    dla, dm = _check_estimate(path, orc["logA"], orc["mass"])
    rep = C.Report()
    counts = path.budget(wl.gamma)
    C.check_counts(counts, orc["counts"], orc["cums"], wl.gamma, 0, wl.block_size, rep)
    bc, bi = path.select(pa_.TOPK_CONSTANT)
    C.check_lists(bc, bi, orc["logA"], counts, wl.num_q_heads, report=rep)
    dl = _check_attention(path, bc, bi, None, rep)
    print(f"\n[32K full] sparsity={_sparsity(bc, wl):.3f} |dlogA|={dla:.2e} "
          f"|dmass|/rows={dm:.2e} max|dO|={rep.max_abs:.2e} mean|dO|={rep.mean_abs:.2e} "
          f"|dlse|={dl:.2e} ambiguous rows={rep.ambiguous_rows} of {rep.rows_checked}",
          flush=True)
