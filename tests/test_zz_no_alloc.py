"""The entry point that allocates nothing, against the blocked sparse call
that takes a workspace: through the C ABI (ctypes, raw device pointers),
two calls in a row on one GPU, the second on a smaller problem, each bitwise
equal to proxyattn_block_sparse_prefill_blocked on the same inputs.  The
library keeps the scratch array's contents between calls, so the second
call also shows that the work-queue counters are cleared before use."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2509_24745_amd.synth import WORKLOADS

pytestmark = pytest.mark.gpu


def _run(U, pa, wl):
    q, k, v = U.inputs(wl)
    prob = U.problem_of(wl)
    qd, kd, vd = U.to_dev(q, prob), U.to_dev(k, prob), U.to_dev(v, prob)
    b = pa.prefill(prob, qd, kd, vd, wl.gamma)
    kvb = torch.empty(pa.proxyattn_kv_blocked_size(prob), dtype=torch.uint8, device="cuda")
    qws = torch.empty(pa.proxyattn_blocked_workspace_size(prob), dtype=torch.uint8, device="cuda")
    pa.proxyattn_prepare_kv(prob, kd, vd, kvb)
    ref_out, ref_lse = torch.empty_like(b.out), torch.empty_like(b.lse)
    pa.proxyattn_block_sparse_prefill_blocked(prob, qd, kvb, b.block_count, b.block_index,
                                              ref_out, ref_lse, qws)
    out = torch.full_like(b.out, float("nan"))
    lse = torch.full_like(b.lse, float("nan"))
    torch.cuda.synchronize()
    p = prob.c_struct()
    stream = torch.cuda.current_stream().cuda_stream
    rc = pa.lib().proxyattn_block_sparse_prefill_blocked_noalloc(
        ctypes.byref(p), qd.data_ptr(), kvb.data_ptr(), kvb.numel(), b.block_count.data_ptr(),
        b.block_index.data_ptr(), out.data_ptr(), lse.data_ptr(), stream)
    assert rc == pa.E_OK, pa.lib().proxyattn_last_error()
    torch.cuda.synchronize()
    assert torch.equal(out, ref_out), f"{wl.name}: output differs"
    assert torch.equal(lse, ref_lse), f"{wl.name}: lse differs"
    # the results are the sparse path's (lists from the selection step)
    assert torch.equal(out, b.out)


def test_noalloc_matches_workspace_call_twice_second_smaller():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from tests import gpu_util as U
    from paper_2509_24745_amd import proxyattn as pa
    llama = WORKLOADS["llama3_8b_n32768"]
    _run(U, pa, llama.replace(seq_len=8192 + 77, name="llama_n8269"))
    _run(U, pa, llama.replace(seq_len=2048 + 5, num_q_heads=8, num_kv_heads=2,
                              num_proxy_groups=2, name="llama_n2053_h8"))


def test_noalloc_rejects_bad_arguments_before_launch():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2509_24745_amd import proxyattn as pa
    from tests import gpu_util as U
    prob = U.problem_of(WORKLOADS["llama3_8b_n32768"].replace(seq_len=4096))
    p = prob.c_struct()
    fake = 1 << 20
    kvb = pa.proxyattn_kv_blocked_size(prob)
    f = pa.lib().proxyattn_block_sparse_prefill_blocked_noalloc
    assert f(ctypes.byref(p), fake, fake, kvb - 1, fake, fake, fake, None, None) == pa.E_WORKSPACE
    assert f(ctypes.byref(p), fake, fake, kvb, None, fake, fake, None, None) == pa.E_INVALID
    assert f(ctypes.byref(p), fake, fake + 4, kvb, fake, fake, fake, None, None) == pa.E_INVALID
    p0 = U.problem_of(WORKLOADS["llama3_8b_n32768"].replace(seq_len=0)).c_struct()
    assert f(ctypes.byref(p0), None, None, 0, None, None, None, None, None) == pa.E_OK
