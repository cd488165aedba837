"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bars (the parity tolerances, see oracle/check.py):
  * pooled proxy heads: bit-exact (both sides sum in fp32 in ascending head
    order, multiply by fl32(1/|G|), round to nearest-even);
  * block log-scores: same -inf pattern, |dlogA| <= LOGA_TOL.  Both sides
    compute in fp32; the GPU accumulates d products in a different order
    (MFMA) and works in base 2, so scores differ by a few fp32 ulps of the
    logits (|S| <~ 40 here -> ~1e-5); LOGA_TOL = 2e-4 leaves margin while
    staying below the 1e-4-relative selection window's scale of concern
    only through check_lists, which judges the lists on oracle scores;
  * last-block masses: relative 1e-4 of the row total (fp32 sums of up to
    N terms in different orders);
  * budgets and lists: identical sets except threshold-ambiguous cases
    (window 1e-4), which are counted and reported; lists run from the
    highest score down;
  * attention: max|dO| <= 2e-2, mean|dO| <= 2e-3 against the oracle's
    attention on the GPU's own lists;
  * lse (no stated bar; derived): bf16 problems normalise with the sum
    of the bf16-rounded probabilities the PV product consumes, each within
    2^-8 relative of the exact value, so |dlse| <= ln(1 + 2^-8) = 3.9e-3
    (reached when one key dominates a row); LSE_TOL = 4e-3.
"""
import dataclasses
import math

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import check as C
from oracle import proxyattn_oracle as O
from paper_2509_24745_amd.synth import WORKLOADS, Structure, Workload

pytestmark = pytest.mark.gpu

LOGA_TOL = 2e-4
MASS_RTOL = 1e-4
LSE_TOL = 4e-3


def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util as U
    return U


LLAMA = WORKLOADS["llama3_8b_n32768"]
QWEN = WORKLOADS["qwen25_7b_n65536"]

CASES = {
    "gqa8x2_n2048_fp32": WORKLOADS["gqa8x2_n2048_fp32"],
    "llama_n4096": LLAMA.replace(seq_len=4096),
    "llama_n4173_ragged": LLAMA.replace(seq_len=4173),
    "bf16_d64_b64_s2_n3000": Workload(name="t", seq_len=3000, num_q_heads=8, num_kv_heads=2,
                                      head_dim=64, block_size=64, num_proxy_groups=2, stride=2,
                                      dtype="bf16", gamma=0.9, structure=Structure(rank=8)),
    "llama_s1_n2048": LLAMA.replace(seq_len=2048, stride=1),
    "llama_s2_n2048": LLAMA.replace(seq_len=2048, stride=2),
    "llama_g1_n4096": LLAMA.replace(seq_len=4096, num_proxy_groups=1),
    "llama_g32_n2048": LLAMA.replace(seq_len=2048, num_proxy_groups=32),
    "qwen_g7_n8192": QWEN.replace(seq_len=8192, num_proxy_groups=7),
    "llama_n100_single_partial_block": LLAMA.replace(seq_len=100),
    # the first block of every sorted mass already exceeds gamma: one block
    # per head, so every row keeps only its top-ranked block
    "llama_gamma_tiny_n2048": LLAMA.replace(seq_len=2048, gamma=1e-6),
    "fp32_d128_b128_n1000": LLAMA.replace(seq_len=1000, dtype="fp32", num_q_heads=8,
                                          num_kv_heads=2, num_proxy_groups=2),
    # the remaining compiled (dtype, d, b) instantiations; b = 64 with d = 128
    # is the two-wave workgroup at one wave per SIMD
    "bf16_d128_b64_s4_n3100": LLAMA.replace(seq_len=3100, block_size=64, num_q_heads=16,
                                            num_kv_heads=4, num_proxy_groups=2),
    "bf16_d64_b128_n2600": Workload(name="t", seq_len=2600, num_q_heads=12, num_kv_heads=3,
                                    head_dim=64, block_size=128, num_proxy_groups=3, stride=4,
                                    dtype="bf16", gamma=0.95, structure=Structure(rank=8)),
    "fp32_d64_b128_s2_n1500": Workload(name="t", seq_len=1500, num_q_heads=4, num_kv_heads=4,
                                       head_dim=64, block_size=128, num_proxy_groups=1, stride=2,
                                       dtype="fp32", gamma=0.9, structure=Structure(rank=8)),
    "fp32_d128_b64_n700": LLAMA.replace(seq_len=700, dtype="fp32", block_size=64, num_q_heads=4,
                                        num_kv_heads=1, num_proxy_groups=4),
}


def _oracle(wl, q, k, v=None, scale=None):
    return O.proxyattn_prefill(q, k, v, num_groups=wl.num_proxy_groups, block_size=wl.block_size,
                               stride=wl.stride, gamma=wl.gamma,
                               min_budget_tokens=wl.min_budget_tokens, scale=scale, dtype=wl.dtype)


def _compare(wl, q, k, v, gpu, orc, attn_rows=None, scale=None):
    rep = C.Report()
    # pooled heads: bit-exact
    assert np.array_equal(gpu["qg"], orc["qg"]), "pooled queries differ"
    assert np.array_equal(gpu["kg"], orc["kg"]), "pooled keys differ"
    # block log-scores
    ga, oa = gpu["logA"], orc["logA"]
    assert np.array_equal(np.isneginf(ga), np.isneginf(oa)), "-inf pattern differs"
    fin = np.isfinite(oa)
    assert np.all(np.isfinite(ga[fin]))
    dla = float(np.max(np.abs(ga[fin] - oa[fin]))) if fin.any() else 0.0
    assert dla <= LOGA_TOL, f"max |dlogA| = {dla}"
    # masses
    rows = min(wl.block_size, wl.seq_len)
    dm = float(np.max(np.abs(gpu["mass"] - orc["mass"]))) / rows
    assert dm <= MASS_RTOL, f"max |dmass|/rows = {dm}"
    # budgets and lists
    C.check_counts(gpu["counts"], orc["counts"], orc["cums"], wl.gamma, wl.min_budget_tokens,
                   wl.block_size, rep)
    C.check_lists(gpu["block_count"], gpu["block_index"], oa, gpu["counts"], wl.num_q_heads,
                  report=rep)
    # attention on the GPU's lists
    if v is not None:
        sc = O.default_scale(wl.head_dim) if scale is None else scale
        ref_out, ref_lse = O.block_sparse_attention(q, k, v, gpu["block_count"], gpu["block_index"],
                                                    wl.block_size, sc, query_rows=attn_rows)
        sel = slice(None) if attn_rows is None else np.asarray(attn_rows)
        C.check_attention(gpu["out"][sel], ref_out[sel], rep)
        dl = np.abs(gpu["lse"][:, sel] - ref_lse[:, sel])
        assert float(dl.max()) <= LSE_TOL, f"max |dlse| = {float(dl.max())}"
    print(f"\n[{wl.name} N={wl.seq_len}] |dlogA|={dla:.2e} |dmass|/rows={dm:.2e} "
          f"max|dO|={rep.max_abs:.2e} mean|dO|={rep.mean_abs:.2e} "
          f"ambiguous heads={len(rep.ambiguous_heads)} rows={rep.ambiguous_rows} "
          f"blocks={rep.ambiguous_blocks} of {rep.rows_checked} rows", flush=True)
    return rep


@pytest.mark.parametrize("case", list(CASES))
def test_pipeline_matches_oracle(case):
    U = _gpu()
    wl = CASES[case]
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    gpu = U.run_path(prob, q, k, v, wl.gamma, wl.min_budget_tokens)
    orc = _oracle(wl, q, k)
    _compare(wl, q, k, v, gpu, orc)


def _random_workload(seed: int) -> Workload:
    """A seeded draw from the supported shapes: dtype, d, b, stride, GQA
    ratio, proxy groups (a divisor of Hq), N from 1 to 2600 (partial and
    single blocks included), gamma, minimum budget and input structure."""
    rng = np.random.default_rng(1000 + seed)
    dtype = "fp32" if rng.random() < 0.25 else "bf16"
    d = int(rng.choice([64, 128]))
    b = int(rng.choice([64, 128]))
    stride = int(rng.choice([1, 2, 4]))
    hkv = int(rng.choice([1, 2, 3, 4]))
    rep = int(rng.choice([r for r in (1, 2, 3, 4, 7) if hkv * r <= 16]))
    hq = hkv * rep
    groups = int(rng.choice([g for g in range(1, hq + 1) if hq % g == 0]))
    n = int(rng.integers(1, 2601))
    return Workload(name=f"rand{seed}", seq_len=n, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                    block_size=b, num_proxy_groups=groups, stride=stride, dtype=dtype,
                    gamma=float(rng.uniform(0.8, 0.99)),
                    min_budget_tokens=int(rng.choice([0, 0, 2 * b])),
                    structure=Structure(rank=int(rng.choice([4, 8, 16])),
                                        noise=float(rng.uniform(0.1, 0.6)),
                                        hetero=bool(rng.random() < 0.3)), seed=seed)


@pytest.mark.parametrize("seed", range(8))
def test_random_shapes_match_oracle(seed):
    U = _gpu()
    wl = _random_workload(seed)
    print(f"\n[random {seed}] {wl}", flush=True)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    gpu = U.run_path(prob, q, k, v, wl.gamma, wl.min_budget_tokens)
    orc = _oracle(wl, q, k)
    _compare(wl, q, k, v, gpu, orc)


@pytest.mark.parametrize("scale", [0.06, 0.15])
def test_caller_softmax_scale(scale):
    """A softmax scale in the problem (instead of 1/sqrt(d)) reaches every
    stage: block scores, last-block masses and the attention."""
    U = _gpu()
    wl = LLAMA.replace(seq_len=2600, num_q_heads=8, num_kv_heads=2, num_proxy_groups=2)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl, softmax_scale=scale)
    gpu = U.run_path(prob, q, k, v, wl.gamma, wl.min_budget_tokens)
    orc = _oracle(wl, q, k, scale=scale)
    _compare(wl, q, k, v, gpu, orc, scale=scale)


def test_all_zero_queries_give_exact_ties_to_lower_blocks():
    """Q = 0: every proxy score is 0, so within a block row every causal key
    block pools to the same value (the largest probability of a block's
    rows is 1/(t'+1) of its first row, whichever key block).  The scores must
    tie exactly, and every list must then be the lowest block indices
    [0, 1, ..., K-1] (ties go to the lower index); attention as the oracle."""
    U = _gpu()
    wl = LLAMA.replace(seq_len=2048 + 40, num_q_heads=8, num_kv_heads=2, num_proxy_groups=2)
    _, k, v = U.inputs(wl)
    q = np.zeros((wl.seq_len, wl.num_q_heads, wl.head_dim), np.float32)
    prob = U.problem_of(wl)
    gpu = U.run_path(prob, q, k, v, wl.gamma)
    la = gpu["logA"]
    mq = la.shape[1]
    for m in range(mq):
        row = la[:, m, :m + 1]
        assert np.all(row == row[:, :1]), f"block row {m}: scores do not tie exactly"
        assert np.all(np.isneginf(la[:, m, m + 1:]))
    for i in range(wl.num_q_heads):
        for m in range(mq):
            c = int(gpu["block_count"][i, m])
            assert c == min(int(gpu["counts"][i]), m + 1)
            assert np.array_equal(gpu["block_index"][i, m, :c], np.arange(c)), (i, m)
    orc = _oracle(wl, q, k)
    _compare(wl, q, k, v, gpu, orc)


@pytest.mark.parametrize("n", [1, 2, 3, 5, 17, 127, 128, 129, 255])
def test_tiny_sequences(n):
    """N below the stride (one strided token), below, at and just above one
    block, and a ragged second block: the whole path against the oracle."""
    U = _gpu()
    wl = LLAMA.replace(seq_len=n, num_q_heads=8, num_kv_heads=2, num_proxy_groups=2)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    gpu = U.run_path(prob, q, k, v, wl.gamma)
    orc = _oracle(wl, q, k)
    _compare(wl, q, k, v, gpu, orc)


def test_min_budget_and_full_budget():
    U = _gpu()
    wl = LLAMA.replace(seq_len=4096, min_budget_tokens=2048)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    gpu = U.run_path(prob, q, k, v, wl.gamma, wl.min_budget_tokens)
    assert np.all(gpu["counts"] >= 16)
    _compare(wl, q, k, v, gpu, _oracle(wl, q, k))
    # gamma = 1: every head keeps every causal block; the attention on those
    # (score-ordered) lists matches the dense kernel to rounding, and the
    # sparse kernel on ascending full lists reproduces it bit for bit
    full = U.run_path(prob, q, k, v, 1.0)
    mq = prob.num_blocks
    assert np.all(full["counts"] == mq)
    assert np.all(full["block_count"] == np.arange(1, mq + 1)[None, :])
    for i in range(wl.num_q_heads):
        for m in range(mq):
            assert np.array_equal(np.sort(full["block_index"][i, m, :m + 1]), np.arange(m + 1))
    dense_out, dense_lse = U.run_attention(prob, q, k, v, dense=True)
    rep = C.check_attention(full["out"], dense_out)
    assert float(np.max(np.abs(full["lse"] - dense_lse))) <= LSE_TOL
    fbc, fbi = O.full_causal_lists(wl.seq_len, wl.num_q_heads, wl.block_size)
    asc_out, asc_lse = U.run_attention(prob, q, k, v, fbc, fbi)
    assert np.array_equal(asc_out, dense_out)
    assert np.array_equal(asc_lse, dense_lse)


def test_attention_random_lists_and_dense():
    U = _gpu()
    for wl in (LLAMA.replace(seq_len=3000), CASES["gqa8x2_n2048_fp32"],
               CASES["bf16_d64_b64_s2_n3000"]):
        q, k, v = U.inputs(wl)
        prob = U.problem_of(wl)
        rng = np.random.default_rng(5)
        mq = prob.num_blocks
        bc = np.zeros((wl.num_q_heads, mq), np.int32)
        bi = np.full((wl.num_q_heads, mq, mq), -1, np.int32)
        for i in range(wl.num_q_heads):
            for m in range(mq):
                kk = int(rng.integers(1, m + 2))
                bi[i, m, :kk] = np.sort(rng.choice(m + 1, kk, replace=False))
                bc[i, m] = kk
        out, lse = U.run_attention(prob, q, k, v, bc, bi)
        sc = O.default_scale(wl.head_dim)
        ref, ref_lse = O.block_sparse_attention(q, k, v, bc, bi, wl.block_size, sc)
        rep = C.check_attention(out, ref)
        assert float(np.max(np.abs(lse - ref_lse))) <= LSE_TOL
        fbc, fbi = O.full_causal_lists(wl.seq_len, wl.num_q_heads, wl.block_size)
        dout, dlse = U.run_attention(prob, q, k, v, dense=True)
        dref, dref_lse = O.block_sparse_attention(q, k, v, fbc, fbi, wl.block_size, sc)
        rep2 = C.check_attention(dout, dref)
        print(f"\n[{wl.name} {wl.dtype}] random lists max|dO|={rep.max_abs:.2e} "
              f"mean={rep.mean_abs:.2e}; dense max|dO|={rep2.max_abs:.2e} "
              f"mean={rep2.mean_abs:.2e}", flush=True)


def test_select_budget_on_oracle_scores_is_exact():
    """Fed the oracle's own scores and masses, the GPU selection reproduces the
    oracle's budgets and lists (ambiguous cumulative crossings aside)."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = QWEN.replace(seq_len=8192, num_proxy_groups=2)
    q, k, _ = U.inputs(wl)
    orc = _oracle(wl, q, k)
    prob = U.problem_of(wl)
    bufs = pa.Buffers(prob)
    logA = torch.from_numpy(orc["logA"]).cuda()
    mass = torch.from_numpy(orc["mass"]).cuda()
    pa.proxyattn_select_budget(prob, logA, mass, wl.gamma, 0, bufs.head_count, bufs.block_count,
                               bufs.block_index)
    torch.cuda.synchronize()
    counts = bufs.head_count.cpu().numpy()
    rep = C.Report()
    C.check_counts(counts, orc["counts"], orc["cums"], wl.gamma, 0, wl.block_size, rep)
    C.check_lists(bufs.block_count.cpu().numpy(), bufs.block_index.cpu().numpy(), orc["logA"],
                  counts, wl.num_q_heads, report=rep)
    assert rep.ambiguous_rows == 0 or len(rep.ambiguous_heads) > 0
    if not rep.ambiguous_heads:
        # same sets as the oracle's (which lists them ascending)
        got = bufs.block_index.cpu().numpy()
        got_sorted = np.where(got >= 0, got, np.iinfo(np.int32).max)
        got_sorted = np.sort(got_sorted, axis=-1)
        got_sorted[got_sorted == np.iinfo(np.int32).max] = -1
        assert np.array_equal(got_sorted, orc["block_index"])


def test_head_major_strided_layout():
    """Q/K/V/O given head-major ([H][N][d]) through the stride fields."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = LLAMA.replace(seq_len=2048, num_q_heads=8, num_kv_heads=2, num_proxy_groups=2)
    q, k, v = U.inputs(wl)
    n, d = wl.seq_len, wl.head_dim
    prob = U.problem_of(wl, q_tok_stride=d, q_head_stride=n * d, kv_tok_stride=d,
                        kv_head_stride=n * d, o_tok_stride=d, o_head_stride=n * d)
    qh = U.to_dev(np.ascontiguousarray(q.transpose(1, 0, 2)), prob)
    kh = U.to_dev(np.ascontiguousarray(k.transpose(1, 0, 2)), prob)
    vh = U.to_dev(np.ascontiguousarray(v.transpose(1, 0, 2)), prob)
    bufs = pa.prefill(prob, qh, kh, vh, wl.gamma)
    out_hm = torch.empty((wl.num_q_heads, n, d), dtype=prob.torch_dtype, device="cuda")
    pa.proxyattn_block_sparse_prefill(prob, qh, kh, vh, bufs.block_count, bufs.block_index,
                                      out_hm, None, bufs.workspace)
    torch.cuda.synchronize()
    ref = U.run_path(U.problem_of(wl), q, k, v, wl.gamma)
    assert np.array_equal(bufs.block_index.cpu().numpy(), ref["block_index"])
    assert np.array_equal(U.to_host(out_hm).transpose(1, 0, 2), ref["out"])


def test_deterministic_across_runs_and_streams():
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = LLAMA.replace(seq_len=4096)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    qd, kd, vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
    outs = []
    s2 = torch.cuda.Stream()
    for stream in (None, None, s2):
        with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
            b = pa.prefill(prob, qd, kd, vd, wl.gamma)
        torch.cuda.synchronize()
        outs.append([t.cpu() for t in (b.logscore, b.mass, b.head_count, b.block_index, b.out,
                                       b.lse)])
    for later in outs[1:]:
        for a, b in zip(outs[0], later):
            assert torch.equal(a, b)


@pytest.mark.parametrize("wl", [LLAMA.replace(seq_len=4096 + 77), QWEN.replace(seq_len=3000)],
                         ids=["llama_n4173", "qwen_n3000"])
def test_work_orders_give_identical_output(wl):
    """Every work order and chunk size must hand each (head, block row) item to
    exactly one workgroup, which computes it alone: sparse and dense outputs
    and lse are then bitwise those of the default order (ragged N, GQA 4 and
    7, chunk sizes that do not divide the block rows)."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    qd, kd, vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
    b = pa.prefill(prob, qd, kd, vd, wl.gamma)
    torch.cuda.synchronize()

    def run(p, dense):
        out = torch.full_like(b.out, float("nan"))
        lse = torch.full_like(b.lse, float("nan"))
        if dense:
            pa.proxyattn_dense_prefill(p, qd, kd, vd, out, lse, b.workspace)
        else:
            pa.proxyattn_block_sparse_prefill(p, qd, kd, vd, b.block_count, b.block_index,
                                              out, lse, b.workspace)
        torch.cuda.synchronize()
        return out.cpu(), lse.cpu()

    ref = {dense: run(prob, dense) for dense in (False, True)}
    for order, rows in ((1, 1), (2, 1), (2, 3), (3, 1), (3, 4), (3, 7), (0, 5)):
        p = dataclasses.replace(prob, attn_order=order, attn_chunk_rows=rows)
        for dense in (False, True):
            out, lse = run(p, dense)
            assert torch.equal(out, ref[dense][0]), (order, rows, dense)
            assert torch.equal(lse, ref[dense][1]), (order, rows, dense)


def _list_status(bc, bi):
    """What proxyattn_check_lists reports, row by row in NumPy."""
    hq, mq = bc.shape
    st = np.zeros((hq, mq), np.int32)
    for i in range(hq):
        for m in range(mq):
            c = int(bc[i, m])
            f = 0 if 1 <= c <= m + 1 else 1
            ent = bi[i, m, :min(max(c, 0), mq)]
            inside = ent[(ent >= 0) & (ent <= m)]
            if inside.size != ent.size:
                f |= 2
            if np.unique(inside).size != inside.size:
                f |= 4
            st[i, m] = f
    return st


def test_check_lists_flags_every_malformed_row():
    """Selected lists are clean; caller lists with planted faults (counts out
    of range, entries out of the causal range, repeated blocks, padding
    beyond the count that must not be read) are flagged exactly."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = LLAMA.replace(seq_len=40 * 64 + 17, block_size=64, num_q_heads=8, num_kv_heads=2,
                       num_proxy_groups=2)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    gpu = U.run_path(prob, q, k, v, wl.gamma)
    hq, mq = gpu["block_count"].shape

    def run(bc, bi):
        st = torch.full((hq, mq), -7, dtype=torch.int32, device="cuda")
        pa.proxyattn_check_lists(prob, torch.from_numpy(bc).cuda(), torch.from_numpy(bi).cuda(),
                                 st)
        torch.cuda.synchronize()
        return st.cpu().numpy()

    bc, bi = gpu["block_count"].copy(), gpu["block_index"].copy()
    assert not run(bc, bi).any(), "selected lists flagged"
    rng = np.random.default_rng(7)
    bc2, bi2 = bc.copy(), bi.copy()
    for _ in range(60):
        i, m = int(rng.integers(hq)), int(rng.integers(mq))
        kind = int(rng.integers(5))
        c = min(max(int(bc2[i, m]), 0), mq)   # entries the check examines
        if kind == 0:
            bc2[i, m] = int(rng.choice([0, -3, m + 2, mq + 5]))
        elif kind == 1 and c >= 1:
            bi2[i, m, int(rng.integers(c))] = int(rng.choice([-1, m + 1, mq + 9]))
        elif kind == 2 and c >= 2:
            a, b = rng.choice(c, 2, replace=False)
            bi2[i, m, b] = bi2[i, m, a]
        elif kind == 3:
            bi2[i, m, c:] = 0          # junk past the count: not read
        elif kind == 4 and 1 <= c <= m:
            bc2[i, m] = c + 1          # one more entry: the -1 padding
    want = _list_status(bc2, bi2)
    got = run(bc2, bi2)
    assert want.any()
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]


def test_check_lists_at_the_largest_size():
    """8192 blocks (the LDS bitmap's full width): full causal lists are clean;
    planted faults in the last rows are flagged."""
    _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    mq, b = 8192, 64
    prob = pa.Problem(seq_len=mq * b, num_q_heads=1, num_kv_heads=1, head_dim=64, block_size=b,
                      num_proxy_groups=1, stride=4, dtype="bf16")
    bc = np.arange(1, mq + 1, dtype=np.int32)[None, :]
    bi = np.full((1, mq, mq), -1, dtype=np.int32)
    tri = np.tril_indices(mq)
    bi[0][tri] = tri[1]
    bi[0, mq - 1, mq - 1] = mq - 2      # duplicate in the last row
    bi[0, 5000, 17] = 5001               # beyond the causal range
    bc[0, 6000] = 0                      # empty list
    st = torch.full((1, mq), -7, dtype=torch.int32, device="cuda")
    pa.proxyattn_check_lists(prob, torch.from_numpy(bc).cuda(), torch.from_numpy(bi).cuda(), st)
    torch.cuda.synchronize()
    got = st.cpu().numpy()[0]
    want = np.zeros(mq, np.int32)
    want[mq - 1], want[5000], want[6000] = 4, 2, 1
    assert np.array_equal(got, want), np.argwhere(got != want)[:5]


def test_empty_problem_is_a_noop():
    _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    prob = pa.Problem(seq_len=0, num_q_heads=4, num_kv_heads=1, head_dim=64, block_size=64,
                      num_proxy_groups=1)
    assert pa.proxyattn_workspace_size(prob) == 0
    pa.proxyattn_estimate(prob, None, None, None, None, None)
    pa.proxyattn_dense_prefill(prob, None, None, None, None, None, None)


def test_budget_and_topk_calls_and_budget_variants():
    """proxyattn_budget + proxyattn_select_topk (constant reading) reproduce
    proxyattn_select_budget bit for bit; the per-row-ratio reading and a
    static Top-K match the oracle's selection; out-of-range counts clamp."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = LLAMA.replace(seq_len=8192 + 77)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    mq = prob.num_blocks
    ref = U.run_path(prob, q, k, None, wl.gamma)
    qd, kd = U.to_dev(q, prob), U.to_dev(k, prob)
    bufs = pa.Buffers(prob)
    pa.proxyattn_estimate(prob, qd, kd, bufs.logscore, bufs.mass, bufs.workspace)
    pa.proxyattn_budget(prob, bufs.mass, wl.gamma, 0, bufs.head_count)
    pa.proxyattn_select_topk(prob, bufs.logscore, bufs.head_count, pa.TOPK_CONSTANT,
                             bufs.block_count, bufs.block_index)
    torch.cuda.synchronize()
    assert np.array_equal(U.to_host(bufs.head_count), ref["counts"])
    assert np.array_equal(U.to_host(bufs.block_count), ref["block_count"])
    assert np.array_equal(U.to_host(bufs.block_index), ref["block_index"])
    orc = _oracle(wl, q, k)
    oa = orc["logA"]
    # per-row-ratio reading on the GPU's budgets
    pa.proxyattn_select_topk(prob, bufs.logscore, bufs.head_count, pa.TOPK_ROW_RATIO,
                             bufs.block_count, bufs.block_index)
    torch.cuda.synchronize()
    counts = U.to_host(bufs.head_count)
    rep = C.check_lists(U.to_host(bufs.block_count), U.to_host(bufs.block_index), oa, counts,
                        wl.num_q_heads, row_ratio=True)
    # static Top-K: one count for every head, and clamping of caller counts
    static = np.full(wl.num_q_heads, 9, np.int32)
    static[0], static[1] = -5, mq + 10
    hc = torch.from_numpy(static).cuda()
    pa.proxyattn_select_topk(prob, bufs.logscore, hc, pa.TOPK_CONSTANT, bufs.block_count,
                             bufs.block_index)
    torch.cuda.synchronize()
    used = np.clip(static, 0, mq)
    bc = U.to_host(bufs.block_count)
    assert np.all(bc[0] == 0) and np.array_equal(bc[1], np.arange(1, mq + 1))
    C.check_lists(bc, U.to_host(bufs.block_index), oa, used, wl.num_q_heads, report=rep)
    print(f"\n[budget variants] ambiguous rows {rep.ambiguous_rows} of {rep.rows_checked}",
          flush=True)


@pytest.mark.parametrize("n,hq,hkv,g,b", [
    (8192, 32, 8, 4, 128),    # Nk = 64, the largest one-launch case
    (4173, 32, 8, 4, 128),    # ragged
    (100, 32, 8, 4, 128),     # Nk = 1
    (129, 8, 2, 2, 128),      # Nk = 2
    (4096, 28, 4, 7, 64),     # b = 64, Nk = 64, 4 heads per group
    (3000, 28, 4, 1, 64),     # one group of 28 heads (7 per wave)
    (8193, 32, 8, 4, 128),    # Nk = 65: two blocks per lane
    (16384, 32, 8, 4, 128),   # Nk = 128
    (12000, 28, 4, 2, 128),   # Nk = 94, 14 heads per group
    (8192, 28, 4, 7, 64),     # b = 64, Nk = 128
    (16385, 32, 8, 4, 128),   # Nk = 129: the two launches, for the same checks
])
def test_one_launch_selection_matches_two(n, hq, hkv, g, b):
    """With at most 128 key blocks proxyattn_select_budget derives the budgets
    inside the selection launch; its counts and lists equal, bit for bit,
    those of proxyattn_budget followed by proxyattn_select_topk (constant
    reading, two launches), on seeded random masses and scores with exact
    ties, zero masses, gamma from 0.3 to 1 and a minimum budget."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    prob = pa.Problem(seq_len=n, num_q_heads=hq, num_kv_heads=hkv, head_dim=128, block_size=b,
                      num_proxy_groups=g, stride=4, dtype="bf16")
    mq = prob.num_blocks
    rng = np.random.default_rng(n * 31 + hq + b)
    logA = rng.standard_normal((g, mq, mq)).astype(np.float32)
    logA[:, :, ::3] = np.round(logA[:, :, ::3] * 2) / 2            # ties among scores
    mass = rng.exponential(1.0, (hq, mq)).astype(np.float32)
    mass[::3, 1::2] = 0.0                                           # zero masses
    mass[1::4] = np.round(mass[1::4] * 4) / 4                       # ties among masses
    mass[2] = 0.0
    mass[2, 0] = 1.0                                                # one block holds it all
    la, md = torch.from_numpy(logA).cuda(), torch.from_numpy(mass).cuda()
    for gamma, min_tok in [(0.3, 0), (0.9, 0), (0.95, 3 * b), (0.999, 0), (1.0, 0)]:
        one = pa.Buffers(prob)
        two = pa.Buffers(prob)
        for x in (one, two):
            x.head_count.fill_(-7)
            x.block_count.fill_(-7)
            x.block_index.fill_(-7)
        pa.proxyattn_select_budget(prob, la, md, gamma, min_tok, one.head_count, one.block_count,
                                   one.block_index)
        pa.proxyattn_budget(prob, md, gamma, min_tok, two.head_count)
        pa.proxyattn_select_topk(prob, la, two.head_count, pa.TOPK_CONSTANT, two.block_count,
                                 two.block_index)
        torch.cuda.synchronize()
        assert torch.equal(one.head_count, two.head_count), (gamma, min_tok)
        assert torch.equal(one.block_count, two.block_count), (gamma, min_tok)
        assert torch.equal(one.block_index, two.block_index), (gamma, min_tok)
        hc = U.to_host(one.head_count)
        assert hc.min() >= max(1, min(mq, -(-min_tok // b))) and hc.max() <= mq
        if gamma == 1.0:
            assert np.all(hc == mq)
    print(f"\n[one-launch selection N={n} Nk={mq} G={g}] counts and lists identical", flush=True)


# The diagnostic's top-k sets can differ from the oracle's only at probability
# near-ties (both compute in fp32, in different orders); a swapped token
# moves one score by at most one probability, which stays far below this.
OVERLAP_TOL = 2e-3


@pytest.mark.parametrize("case,t,topk,sink,renorm", [
    ("gqa8x2_n2048_fp32", 2047, 256, 0, False),
    ("gqa8x2_n2048_fp32", 1000, 64, 4, True),
    ("llama_n4173_ragged", 4172, 1024, 0, False),
    ("llama_n4173_ragged", 4172, 1024, 4, False),
    ("llama_n4173_ragged", 3000, 512, 4, True),
    ("llama_n100_single_partial_block", 99, 1000, 0, False),
])
def test_head_overlap_matches_oracle(case, t, topk, sink, renorm):
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = CASES[case]
    q, k, _ = U.inputs(wl)
    prob = U.problem_of(wl)
    bufs = pa.Buffers(prob)
    scores = torch.empty((wl.num_q_heads, wl.num_q_heads), dtype=torch.float32, device="cuda")
    pa.proxyattn_head_overlap(prob, U.to_dev(q, prob), U.to_dev(k, prob), t, topk, sink, renorm,
                              scores, bufs.workspace)
    torch.cuda.synchronize()
    got = U.to_host(scores)
    ref = O.head_overlap(q, k, t, topk, O.default_scale(wl.head_dim), sink_tokens=sink,
                         renormalize=renorm)
    err = float(np.max(np.abs(got - ref)))
    assert err <= OVERLAP_TOL, f"max |dScore| = {err}"
    # own top-k holds the most of a head's mass (up to rounding)
    assert np.all(np.diag(got)[None, :] >= got - 1e-5)
    print(f"\n[overlap {case} t={t} k={topk} sink={sink} renorm={renorm}] max|dScore|={err:.2e}",
          flush=True)


def test_whole_step_replays_from_a_hip_graph():
    """estimate -> select_budget -> block_sparse_prefill captured once into a
    HIP graph (the library issues no memsets, allocations or syncs) and
    replayed three times, with eager work and synchronisations between the
    replays: every replay reproduces the eager results bit for bit."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = LLAMA.replace(seq_len=4096 + 33)
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    qd, kd, vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
    bufs = pa.Buffers(prob)

    def step():
        pa.proxyattn_estimate(prob, qd, kd, bufs.logscore, bufs.mass, bufs.workspace)
        pa.proxyattn_select_budget(prob, bufs.logscore, bufs.mass, wl.gamma, 0, bufs.head_count,
                                   bufs.block_count, bufs.block_index)
        pa.proxyattn_block_sparse_prefill(prob, qd, kd, vd, bufs.block_count, bufs.block_index,
                                          bufs.out, bufs.lse, bufs.workspace)

    names = ("logscore", "mass", "head_count", "block_count", "block_index", "out", "lse")
    step()
    torch.cuda.synchronize()
    ref = {n: getattr(bufs, n).clone() for n in names}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for n in names:                       # eager work between the replays
            getattr(bufs, n).zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            assert torch.equal(getattr(bufs, n), ref[n]), f"replay {rep}: {n} differs"


def _sampled_rows_check(wl, nsample: int, pre: dict | None = None, pool=None):
    """The whole path at full size, in the benchmark's launch configuration:
    pooled heads bit-exact, every head's last-block mass and budget, and the
    proxy scores, lists and attention of seeded sampled query rows (always
    including the last row) and their block rows.  `pre`: the layer's inputs
    and the oracle's pooled heads, block scores of those block rows and
    masses, prepared ahead (tests/pregen.py); computed here when absent.
    `pool`: the preparing processes, which then also run the oracle's
    attention of the sampled rows, split over groups of KV heads."""
    U = _gpu()
    from tests import pregen
    rows = pregen.sample_rows(wl.seq_len, nsample)
    if pre is None:
        q, k, v = U.inputs(wl)
    else:
        q, k, v = pre["q"], pre["k"], pre["v"]
    gpu = U.run_path(U.problem_of(wl), q, k, v, wl.gamma, rows=rows)
    check_sampled_rows(wl, rows, q, k, v, gpu, pre, pool)


def check_sampled_rows(wl, rows, q, k, v, gpu: dict, pre: dict | None = None, pool=None):
    """Check the path's results `gpu` on inputs q, k, v (host arrays) against
    the oracle: pooled heads, every head's mass and budget, the scores and
    lists of the block rows of `rows`, and the attention of `rows` (gpu's
    out and lse hold those rows only).  `pre` and `pool` as in
    _sampled_rows_check."""
    brows = np.unique(np.asarray(rows) // wl.block_size)
    sc = O.default_scale(wl.head_dim)
    if pre is None:
        qg, kg = O.pool_proxy_heads(q, k, wl.num_proxy_groups, wl.stride, wl.dtype)
        oa, _ = O.proxy_block_logscore(qg, kg, wl.seq_len, wl.block_size, wl.stride, sc,
                                       rows=brows)
        mass = O.lastblock_mass(q, k, wl.block_size, sc)
    else:
        qg, kg, oa, mass = pre["qg"], pre["kg"], pre["logA"], pre["mass"]
    assert np.array_equal(gpu["qg"], qg) and np.array_equal(gpu["kg"], kg), "pooled heads differ"
    ga = gpu["logA"][:, brows]
    ob = oa[:, brows]
    assert np.array_equal(np.isneginf(ga), np.isneginf(ob)), "-inf pattern differs"
    fin = np.isfinite(ob)
    dla = float(np.max(np.abs(ga[fin] - ob[fin])))
    assert dla <= LOGA_TOL, f"max |dlogA| = {dla}"
    dm = float(np.max(np.abs(gpu["mass"] - mass))) / wl.block_size
    assert dm <= MASS_RTOL, f"max |dmass|/rows = {dm}"
    counts, cums = O.budget_counts(mass, wl.gamma, wl.min_budget_tokens, wl.block_size)
    rep = C.Report()
    C.check_counts(gpu["counts"], counts, cums, wl.gamma, wl.min_budget_tokens, wl.block_size, rep)
    C.check_lists(gpu["block_count"], gpu["block_index"], oa, gpu["counts"], wl.num_q_heads,
                  rows=brows, report=rep)
    if pool is None:
        ref_out, ref_lse = O.block_sparse_attention(q, k, v, gpu["block_count"],
                                                    gpu["block_index"], wl.block_size, sc,
                                                    query_rows=rows)
        ref_out, ref_lse = ref_out[rows], ref_lse[:, rows]
    else:
        ref_out, ref_lse = pool.attention(wl.seed, wl.block_size, wl.num_q_heads,
                                          wl.num_kv_heads, rows, gpu["block_count"],
                                          gpu["block_index"])
        pool.release(wl.seed)
    C.check_attention(gpu["out"], ref_out, rep)
    dl = float(np.abs(gpu["lse"] - ref_lse).max())
    assert dl <= LSE_TOL, f"max |dlse| = {dl}"
    print(f"\n[{wl.name} seed {wl.seed}] |dlogA|={dla:.2e} |dmass|/rows={dm:.2e} "
          f"max|dO|={rep.max_abs:.2e} mean|dO|={rep.mean_abs:.2e} |dlse|={dl:.2e} "
          f"ambiguous heads={len(rep.ambiguous_heads)} rows={rep.ambiguous_rows} "
          f"of {rep.rows_checked}", flush=True)


@pytest.mark.parametrize("layer", [0, 7, 15, 23, 31])
def test_256k_layer_sampled_rows(layer):
    """Five layers spread over the 32-layer 256K stack (layer l is drawn with
    seed l): every head's last-block mass and budget, and the scores, lists
    and attention of 512 sampled query rows per head (the same rows for every
    head) and of their block rows."""
    from tests import pregen
    wl = WORKLOADS["llama3_8b_n262144"].replace(seed=layer)
    print(f"\n[256K layer {layer}]", flush=True)
    pg = pregen.active()
    _sampled_rows_check(wl, 512, pg.get(layer) if pg is not None else None, pg)


def test_maximum_size_sampled_rows():
    """The largest problem the library accepts: 8192 blocks of 128 tokens
    (N = 1,048,576), with 4 query heads on one KV head and d = 64 to keep
    the oracle's share small; 16 sampled query rows."""
    wl = LLAMA.replace(seq_len=8192 * 128, num_q_heads=4, num_kv_heads=1, head_dim=64,
                       num_proxy_groups=1, name="llama_shaped_n1048576_h4")
    _sampled_rows_check(wl, 16)


# The full-size 32K, 64K and 128K layers are checked in test_gpu_scope.py.


@pytest.mark.parametrize("case", ["llama_n4173_ragged", "qwen_g7_n8192", "gqa8x2_n2048_fp32"])
def test_ascending_lists_match_oracle(case):
    """PROXYATTN_LIST_ASCENDING: the same sets as the rank-order lists, listed
    by ascending block index, which is the oracle's own list order (Eq. 3);
    where no threshold ambiguity arises the lists equal the oracle's bit for
    bit.  Constant and per-row-ratio readings; attention on the ascending
    lists against the oracle."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = CASES[case]
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    qd, kd, vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
    bufs = pa.Buffers(prob)
    pa.proxyattn_estimate(prob, qd, kd, bufs.logscore, bufs.mass, bufs.workspace)
    pa.proxyattn_budget(prob, bufs.mass, wl.gamma, 0, bufs.head_count)
    torch.cuda.synchronize()
    counts = U.to_host(bufs.head_count)
    orc = _oracle(wl, q, k)
    for row_ratio in (False, True):
        mode = (pa.TOPK_ROW_RATIO if row_ratio else pa.TOPK_CONSTANT) | pa.LIST_ASCENDING
        pa.proxyattn_select_topk(prob, bufs.logscore, bufs.head_count, mode, bufs.block_count,
                                 bufs.block_index)
        torch.cuda.synchronize()
        bc, bi = U.to_host(bufs.block_count), U.to_host(bufs.block_index)
        for i in range(wl.num_q_heads):
            for m in range(prob.num_blocks):
                c = int(bc[i, m])
                assert np.all(np.diff(bi[i, m, :c]) > 0), (i, m, bi[i, m, :c])
        rep = C.check_lists(bc, bi, orc["logA"], counts, wl.num_q_heads, rank_order=False,
                            row_ratio=row_ratio)
        obc, obi = O.select_blocks(orc["logA"], counts, wl.num_q_heads, row_ratio=row_ratio)
        if rep.ambiguous_rows == 0:
            assert np.array_equal(bc, obc) and np.array_equal(bi, obi)
        out, lse = U.run_attention(prob, q, k, v, bc, bi)
        ref, ref_lse = O.block_sparse_attention(q, k, v, bc, bi, wl.block_size,
                                                O.default_scale(wl.head_dim))
        arep = C.check_attention(out, ref)
        assert float(np.max(np.abs(lse - ref_lse))) <= LSE_TOL
        print(f"\n[ascending {case} row_ratio={row_ratio}] ambiguous rows {rep.ambiguous_rows} "
              f"of {rep.rows_checked}; max|dO|={arep.max_abs:.2e}", flush=True)


@pytest.mark.parametrize("case", ["llama_n4173_ragged", "gqa8x2_n2048_fp32",
                                  "bf16_d64_b64_s2_n3000", "fp32_d128_b64_n700",
                                  "bf16_d128_b64_s4_n3100"])
def test_blocked_calls_match_unblocked(case):
    """proxyattn_prepare_kv once, then the _blocked sparse and dense calls
    (twice each, sharing one small workspace, so the work-queue counters are
    reset between launches): output and lse bitwise those of the calls that
    re-block K/V themselves."""
    U = _gpu()
    from paper_2509_24745_amd import proxyattn as pa
    wl = CASES[case]
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    qd, kd, vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
    b = pa.prefill(prob, qd, kd, vd, wl.gamma)
    dense_out, dense_lse = torch.empty_like(b.out), torch.empty_like(b.lse)
    pa.proxyattn_dense_prefill(prob, qd, kd, vd, dense_out, dense_lse, b.workspace)
    kvb = torch.empty(pa.proxyattn_kv_blocked_size(prob), dtype=torch.uint8, device="cuda")
    qws = torch.empty(pa.proxyattn_blocked_workspace_size(prob), dtype=torch.uint8, device="cuda")
    pa.proxyattn_prepare_kv(prob, kd, vd, kvb)
    for rep in range(2):
        out, lse = torch.full_like(b.out, float("nan")), torch.full_like(b.lse, float("nan"))
        pa.proxyattn_block_sparse_prefill_blocked(prob, qd, kvb, b.block_count, b.block_index,
                                                  out, lse, qws)
        torch.cuda.synchronize()
        assert torch.equal(out, b.out) and torch.equal(lse, b.lse), f"sparse, call {rep}"
        out.fill_(float("nan"))
        lse.fill_(float("nan"))
        pa.proxyattn_dense_prefill_blocked(prob, qd, kvb, out, lse, qws)
        torch.cuda.synchronize()
        assert torch.equal(out, dense_out) and torch.equal(lse, dense_lse), f"dense, call {rep}"
