"""Head sharding, shown on one GPU.  With one proxy group per KV head
(G = Hkv), the query heads of a set of KV heads need nothing from the other
heads: pooling, block scores, masses, budgets, lists and attention of those
heads follow from their own slices of Q, K and V.  A layer is split into P
parts, each part runs the path alone on its slices (as one of P GPUs would),
and its results are compared with the same heads of the whole layer."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import check as C
from oracle import proxyattn_oracle as O
from paper_2509_24745_amd.synth import WORKLOADS
from tests.test_gpu_parity import LOGA_TOL, MASS_RTOL, _gpu

pytestmark = pytest.mark.gpu

LLAMA = WORKLOADS["llama3_8b_n32768"]


@pytest.mark.parametrize("parts", [2, 8])
def test_head_shards_reproduce_the_whole_layer(parts):
    """Pooled heads bit for bit; block scores and masses to the parity bars
    (the estimation kernels split their key loops by problem size, so row
    normalisers are summed in another order); budgets and lists equal up to
    threshold ties, judged on the whole layer's scores; and the attention of
    every head, run on the whole layer's lists, bit for bit."""
    U = _gpu()
    wl = LLAMA.replace(seq_len=16384 + 77, num_proxy_groups=LLAMA.num_kv_heads)
    q, k, v = U.inputs(wl)
    full = U.run_path(U.problem_of(wl), q, k, v, wl.gamma)
    rq, rk, rg = wl.num_q_heads // parts, wl.num_kv_heads // parts, wl.num_proxy_groups // parts
    for s in range(parts):
        hs, ks, gs = slice(s * rq, (s + 1) * rq), slice(s * rk, (s + 1) * rk), slice(s * rg, (s + 1) * rg)
        ws = wl.replace(num_q_heads=rq, num_kv_heads=rk, num_proxy_groups=rg)
        qs, kk, vs = (np.ascontiguousarray(x) for x in (q[:, hs], k[:, ks], v[:, ks]))
        part = U.run_path(U.problem_of(ws), qs, kk, vs, wl.gamma)
        assert np.array_equal(part["qg"], full["qg"][gs]), f"part {s}: pooled queries differ"
        assert np.array_equal(part["kg"], full["kg"][gs]), f"part {s}: pooled keys differ"
        fa, pa_ = full["logA"][gs], part["logA"]
        assert np.array_equal(np.isneginf(fa), np.isneginf(pa_))
        fin = np.isfinite(fa)
        dla = float(np.max(np.abs(fa[fin] - pa_[fin])))
        assert dla <= LOGA_TOL, f"part {s}: max |dlogA| = {dla}"
        dm = float(np.max(np.abs(full["mass"][hs] - part["mass"]))) / wl.block_size
        assert dm <= MASS_RTOL, f"part {s}: max |dmass|/rows = {dm}"
        rep = C.Report()
        counts, cums = O.budget_counts(full["mass"][hs], wl.gamma, 0, wl.block_size)
        C.check_counts(part["counts"], counts, cums, wl.gamma, 0, wl.block_size, rep)
        C.check_lists(part["block_count"], part["block_index"], fa, part["counts"], rq, report=rep)
        # attention on the whole layer's lists of these heads: the same items
        # of the same kernel, so the same bits
        lists = (np.ascontiguousarray(full["block_count"][hs]),
                 np.ascontiguousarray(full["block_index"][hs]))
        again = U.run_path(U.problem_of(ws), qs, kk, vs, wl.gamma, lists=lists)
        assert np.array_equal(again["out"], full["out"][:, hs]), f"part {s}: outputs differ"
        assert np.array_equal(again["lse"], full["lse"][hs]), f"part {s}: lse differs"
        same = int(np.sum(part["block_count"] == full["block_count"][hs]))
        print(f"\n[{parts} parts, part {s}] |dlogA|={dla:.2e} |dmass|/rows={dm:.2e} "
              f"ambiguous heads={len(rep.ambiguous_heads)} rows={rep.ambiguous_rows}; "
              f"equal row counts {same}/{part['block_count'].size}", flush=True)
