"""The C-ABI library on the host: it loads, exports every function the header
declares, its problem struct matches the C compiler's layout, and argument
validation rejects bad calls before anything reaches a GPU (these calls
return before any HIP call, so they run without a GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "proxyattn.h")

pa = pytest.importorskip("paper_2509_24745_amd.proxyattn")


def _lib():
    if not os.path.exists(pa.LIB_PATH):
        pytest.skip("libproxyattn.so not built")
    return pa.lib()


def test_header_functions_are_all_exported():
    text = open(HEADER).read()
    declared = set(re.findall(r"^\s*(?:int|const char\*)\s+(proxyattn_\w+)\s*\(", text, re.M))
    assert declared == set(pa.EXPORTS)
    lib = _lib()
    for name in declared:
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", pa.LIB_PATH], capture_output=True,
                         text=True).stdout
    for name in declared:
        assert re.search(rf"\bT {name}$", out, re.M), f"{name} not exported"


def test_struct_layout_matches_c_compiler(tmp_path):
    fields = [f[0] for f in pa.proxyattn_problem._fields_]
    src = tmp_path / "layout.c"
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "proxyattn.h"', 'int main(void){',
             'printf("%zu\\n", sizeof(proxyattn_problem));']
    lines += [f'printf("%zu\\n", offsetof(proxyattn_problem, {f}));' for f in fields]
    lines += ['return 0;}']
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)], check=True)
    vals = [int(x) for x in subprocess.run([str(exe)], capture_output=True, text=True).stdout.split()]
    assert vals[0] == ctypes.sizeof(pa.proxyattn_problem)
    for f, off in zip(fields, vals[1:]):
        assert getattr(pa.proxyattn_problem, f).offset == off, f


def _prob(**kw):
    base = dict(seq_len=4096, num_q_heads=32, num_kv_heads=8, head_dim=128, block_size=128,
                num_proxy_groups=4, stride=4, dtype="bf16")
    base.update(kw)
    return pa.Problem(**base)


def test_version_and_error_strings():
    lib = _lib()
    assert lib.proxyattn_version().decode().count(".") == 2
    for code in range(5):
        assert lib.proxyattn_error_string(code)
    assert lib.proxyattn_error_string(77) == b"unknown error"


@pytest.mark.parametrize("kw,code", [
    (dict(seq_len=-1), pa.E_INVALID),
    (dict(num_q_heads=0), pa.E_INVALID),
    (dict(num_q_heads=30), pa.E_UNSUPPORTED),        # 30 % 8 != 0
    (dict(num_proxy_groups=3), pa.E_UNSUPPORTED),    # 32 % 3 != 0
    (dict(head_dim=96), pa.E_UNSUPPORTED),
    (dict(block_size=256), pa.E_UNSUPPORTED),
    (dict(stride=8), pa.E_UNSUPPORTED),
    (dict(block_size=64, stride=4, head_dim=64), None),  # b/s = 16 is fine
    (dict(dtype="fp16"), pa.E_UNSUPPORTED),
    (dict(seq_len=8193 * 128), pa.E_UNSUPPORTED),   # more than 8192 blocks
    (dict(q_tok_stride=4100), pa.E_UNSUPPORTED),    # rows not 16-byte aligned
    (dict(num_q_heads=4104, num_kv_heads=8, num_proxy_groups=8), pa.E_UNSUPPORTED),  # > 4096
    (dict(num_q_heads=4096, num_kv_heads=8, num_proxy_groups=8), None),
])
def test_problem_validation(kw, code):
    _lib()
    prob = _prob(**kw)
    if code is None:
        assert pa.proxyattn_workspace_size(prob) > 0
        return
    with pytest.raises(pa.ProxyAttnError) as ei:
        pa.proxyattn_workspace_size(prob)
    assert ei.value.code == code


@pytest.mark.parametrize("order,rows,ok", [
    (0, 0, True), (1, 1, True), (2, 2, True), (3, 8192, True), (0, 7, True), (3, 0, True),
    (4, 4, False), (-1, 4, False), (3, -4, False), (3, 8193, False), (2**31 - 1, 4, False),
    (3, -2**31, False),
])
def test_work_order_fields_are_validated(order, rows, ok):
    """The attention work-order fields of the problem descriptor reach kernel
    index arithmetic: values outside the documented ranges fail every call
    with E_INVALID before anything is enqueued."""
    _lib()
    prob = _prob(attn_order=order, attn_chunk_rows=rows)
    if ok:
        assert pa.proxyattn_workspace_size(prob) > 0
        return
    with pytest.raises(pa.ProxyAttnError) as ei:
        pa.proxyattn_workspace_size(prob)
    assert ei.value.code == pa.E_INVALID
    assert "attn_" in str(ei.value)


def test_library_reads_no_environment(monkeypatch):
    """Settings once read from the environment are descriptor fields now: the
    old variables, even malformed, change nothing."""
    _lib()
    want = pa.proxyattn_workspace_size(_prob())
    monkeypatch.setenv("PROXYATTN_ATTN_ORDER", "7x")
    monkeypatch.setenv("PROXYATTN_ATTN_CHUNK_ROWS", "-1")
    assert pa.proxyattn_workspace_size(_prob()) == want


def test_bad_struct_size_and_null_problem():
    lib = _lib()
    p = _prob().c_struct()
    p.struct_size = 12
    n = ctypes.c_size_t(0)
    assert lib.proxyattn_workspace_size(ctypes.byref(p), ctypes.byref(n)) == pa.E_INVALID
    assert lib.proxyattn_workspace_size(None, ctypes.byref(n)) == pa.E_INVALID


def _key_chunks(n, hq, g, b, s):
    """The library's rule for splitting the estimation kernels' key loops:
    halve the mass kernels' 2048-key chunk (not below one block), and the
    block-scoring chunk of 32-key tiles (a multiple of 4, not below 4, at most
    128), while a launch has fewer than 1024 workgroups.  Returns (mass chunk, mass
    chunks, tiles per scoring chunk, scoring chunks of the longest row)."""
    npr = -(-n // s)
    mc = 2048
    while mc > b and hq * -(-n // mc) < 1024:
        mc //= 2
    nrb, nt = -(-npr // 128), -(-npr // 32)

    def groups(kc):
        return g * sum((min(x * 128 + 127, npr - 1) // 32) // kc + 1 for x in range(nrb))

    kc = max(4, min(-(-nt // 4) * 4, 128))
    while kc > 4 and groups(kc) < 1024:
        kc = max(4, -(-(kc // 2) // 4) * 4)
    return mc, -(-n // mc), kc, max(1, -(-nt // kc))


def test_key_chunk_rule():
    # long sequences: 2048-key mass chunks, scoring chunks of 128 tiles
    assert _key_chunks(131072, 32, 4, 128, 4) == (2048, 64, 128, 8)
    assert _key_chunks(262144, 32, 4, 128, 4) == (2048, 128, 128, 16)
    # short ones split until the launches reach 1024 workgroups (or the floor)
    assert _key_chunks(32768, 32, 4, 128, 4) == (1024, 32, 32, 8)
    assert _key_chunks(8192, 32, 4, 128, 4) == (256, 32, 4, 16)
    assert _key_chunks(2048, 32, 4, 128, 4) == (128, 16, 4, 4)


RBM_MAX_BYTES = 512 << 20


def _rbm_pairs(n, g, b, s):
    """The library's band groups of the per-(row, key block) maxima:
    consecutive bands of 128 strided rows (128 / b' block rows each), grown
    greedily while the group's lower-triangular block pairs over all proxy
    groups fit 512 MiB.  Returns (groups, largest group's pairs)."""
    npr, mq, bp = -(-n // s), -(-n // b), b // s
    nb, rpb = -(-npr // 128), 128 // bp
    cap = RBM_MAX_BYTES // (g * bp * 4)

    def pairs(x0, x1):
        m0, m1 = x0 * rpb, min(x1 * rpb, mq)
        return m1 * (m1 + 1) // 2 - m0 * (m0 + 1) // 2

    groups, mx, x0 = 0, 0, 0
    while x0 < nb:
        x1 = x0 + 1
        while x1 < nb and pairs(x0, x1 + 1) <= cap:
            x1 += 1
        mx = max(mx, pairs(x0, x1))
        groups += 1
        x0 = x1
    return groups, mx


def test_rbm_band_groups():
    """One group up to 128K with 4 proxy groups (the region is the whole
    lower triangle, 268 MB); longer problems split into groups whose region
    stays within 512 MiB."""
    assert _rbm_pairs(131072, 4, 128, 4) == (1, 1024 * 1025 // 2)
    g256, p256 = _rbm_pairs(262144, 4, 128, 4)
    assert g256 >= 2 and 4 * p256 * 32 * 4 <= RBM_MAX_BYTES
    g1m, p1m = _rbm_pairs(8192 * 128, 4, 128, 4)
    assert g1m > 8 and 4 * p1m * 32 * 4 <= RBM_MAX_BYTES
    g1, p1 = _rbm_pairs(8192 * 128, 1, 128, 1)       # b' = 128
    assert 1 * p1 * 128 * 4 <= RBM_MAX_BYTES


@pytest.mark.parametrize("n,hq,hkv,g,b,s", [
    (32768, 32, 8, 4, 128, 4), (262144, 32, 8, 4, 128, 4), (8192 * 128, 8, 2, 2, 128, 4),
    (8192 * 128, 8, 2, 1, 128, 1), (8192, 32, 8, 4, 128, 4), (131072, 32, 8, 4, 128, 4),
    (65536, 28, 4, 2, 128, 4), (3000, 8, 2, 2, 64, 2), (777, 4, 4, 1, 64, 1)])
def test_workspace_size_formula(n, hq, hkv, g, b, s):
    _lib()
    prob = _prob(seq_len=n, num_q_heads=hq, num_kv_heads=hkv, num_proxy_groups=g,
                 block_size=b, stride=s)
    assert pa.proxyattn_workspace_size(prob) == _expected_ws(n, hq, hkv, g, b, s)


def _expected_ws(n, hq, hkv, g, b, s, d=128):
    """The workspace regions as the header states them, each rounded up to
    256 bytes; the head-overlap diagnostic's region reuses the K/V copy's."""
    npr, mq, bp = -(-n // s), -(-n // b), b // s
    _, _, _, est_nc = _key_chunks(n, hq, g, b, s)
    regions = [g * npr * d * 2, g * npr * d * 2, g * est_nc * npr * 8,
               g * _rbm_pairs(n, g, b, s)[1] * bp * 4, hq * b * mq * 8, hq * b * 4,
               hkv * mq * 2 * d * b * 2, 8 * 32 * 4]
    end = sum(-(-r // 256) * 256 for r in regions)
    kvb = sum(-(-r // 256) * 256 for r in regions[:6])
    diag_end = kvb + -(-(hq * n * 4) // 256) * 256 + -(-(hq * 8) // 256) * 256
    return max(end, diag_end)


def test_workspace_size_at_the_largest_problem():
    """8192 blocks: the per-(row, block) maxima are produced and reduced one
    group of row bands at a time, so their region stays within 512 MiB
    (the whole lower triangle would be 4.3 GB per proxy group with b' = 32
    and 17 GB with s = 1)."""
    _lib()
    mq = 8192
    for g, s, bp in ((1, 4, 32), (4, 4, 32), (1, 1, 128)):
        prob = _prob(seq_len=mq * 128, num_q_heads=32, num_kv_heads=8, num_proxy_groups=g,
                     stride=s)
        ws = pa.proxyattn_workspace_size(prob)
        whole = g * (mq * (mq + 1) // 2) * bp * 4
        assert whole > 4e9
        groups, pairs = _rbm_pairs(mq * 128, g, 128, s)
        assert groups > 1 and g * pairs * bp * 4 <= RBM_MAX_BYTES
        assert ws == _expected_ws(mq * 128, 32, 8, g, 128, s)
        assert ws < _expected_ws(mq * 128, 32, 8, g, 128, s) - g * pairs * bp * 4 + whole


def test_workspace_size_of_empty_problem():
    _lib()
    assert pa.proxyattn_workspace_size(_prob(seq_len=0)) == 0


def test_calls_reject_bad_arguments_before_launch():
    lib = _lib()
    prob = _prob()
    p = prob.c_struct()
    fake = 1 << 20                       # aligned, never dereferenced: calls fail first
    ws = pa.proxyattn_workspace_size(prob)
    # null tensor
    assert lib.proxyattn_estimate(ctypes.byref(p), None, fake, fake, fake, fake, ws, None) \
        == pa.E_INVALID
    # misaligned tensor
    assert lib.proxyattn_estimate(ctypes.byref(p), fake + 2, fake, fake, fake, fake, ws, None) \
        == pa.E_INVALID
    # workspace too small
    assert lib.proxyattn_estimate(ctypes.byref(p), fake, fake, fake, fake, fake, ws - 1, None) \
        == pa.E_WORKSPACE
    # gamma outside (0, 1], negative minimum budget
    for gamma, beta in ((0.0, 0), (1.5, 0), (float("nan"), 0), (0.9, -1)):
        assert lib.proxyattn_select_budget(ctypes.byref(p), fake, fake, gamma, beta, fake, fake,
                                           fake, None) == pa.E_INVALID
    assert b"gamma" in lib.proxyattn_last_error() or b"min_budget" in lib.proxyattn_last_error()
    for gamma, beta in ((0.0, 0), (1.5, 0), (float("nan"), 0), (0.9, -1)):
        assert lib.proxyattn_budget(ctypes.byref(p), fake, gamma, beta, fake, None) == pa.E_INVALID
    assert lib.proxyattn_budget(ctypes.byref(p), fake, 0.9, 0, None, None) == pa.E_INVALID
    # list check: null or misaligned pointers
    assert lib.proxyattn_check_lists(ctypes.byref(p), fake, fake, None, None) == pa.E_INVALID
    assert lib.proxyattn_check_lists(ctypes.byref(p), None, fake, fake, None) == pa.E_INVALID
    assert lib.proxyattn_check_lists(ctypes.byref(p), fake, fake + 4, fake, None) == pa.E_INVALID
    # unknown top-k mode, missing counts
    for mode in (-1, 4, 7):
        assert lib.proxyattn_select_topk(ctypes.byref(p), fake, fake, mode, fake, fake, None) \
            == pa.E_INVALID
    assert b"mode" in lib.proxyattn_last_error()
    assert lib.proxyattn_select_topk(ctypes.byref(p), fake, None, pa.TOPK_CONSTANT, fake, fake,
                                     None) == pa.E_INVALID
    # head-overlap diagnostic: token, k, sinks, renormalize flag, output
    n = prob.seq_len
    for t, kk, sink, rn in ((-1, 8, 0, 0), (n, 8, 0, 0), (5, 0, 0, 0), (5, 8, 6, 0), (5, 8, -1, 0),
                            (5, 8, 0, 2)):
        assert lib.proxyattn_head_overlap(ctypes.byref(p), fake, fake, t, kk, sink, rn, fake, fake,
                                          ws, None) == pa.E_INVALID
    assert lib.proxyattn_head_overlap(ctypes.byref(p), fake, fake, 5, 8, 0, 0, None, fake, ws,
                                      None) == pa.E_INVALID
    assert lib.proxyattn_head_overlap(ctypes.byref(p), fake, fake, 5, 8, 0, 0, fake, fake, ws - 1,
                                      None) == pa.E_WORKSPACE
    # prefill without lists
    assert lib.proxyattn_block_sparse_prefill(ctypes.byref(p), fake, fake, fake, None, fake, fake,
                                              None, fake, ws, None) == pa.E_INVALID
    # blocked K/V copy: missing, misaligned, too small; blocked calls' workspace
    kvb = pa.proxyattn_kv_blocked_size(prob)
    qws = pa.proxyattn_blocked_workspace_size(prob)
    assert lib.proxyattn_prepare_kv(ctypes.byref(p), fake, fake, None, kvb, None) == pa.E_INVALID
    assert lib.proxyattn_prepare_kv(ctypes.byref(p), fake, fake, fake + 8, kvb, None) \
        == pa.E_INVALID
    assert lib.proxyattn_prepare_kv(ctypes.byref(p), fake, fake, fake, kvb - 1, None) \
        == pa.E_WORKSPACE
    assert lib.proxyattn_prepare_kv(ctypes.byref(p), None, fake, fake, kvb, None) == pa.E_INVALID
    assert lib.proxyattn_block_sparse_prefill_blocked(ctypes.byref(p), fake, fake, kvb - 1, fake,
                                                      fake, fake, None, fake, qws, None) \
        == pa.E_WORKSPACE
    assert lib.proxyattn_block_sparse_prefill_blocked(ctypes.byref(p), fake, fake, kvb, fake,
                                                      fake, fake, None, fake, qws - 1, None) \
        == pa.E_WORKSPACE
    assert lib.proxyattn_block_sparse_prefill_blocked(ctypes.byref(p), fake, fake, kvb, None,
                                                      fake, fake, None, fake, qws, None) \
        == pa.E_INVALID
    assert lib.proxyattn_dense_prefill_blocked(ctypes.byref(p), fake, fake, kvb, fake, None, None,
                                               qws, None) == pa.E_INVALID
    # empty problem: valid no-op, nothing touched
    p0 = _prob(seq_len=0).c_struct()
    assert lib.proxyattn_estimate(ctypes.byref(p0), None, None, None, None, None, 0, None) == 0
    assert lib.proxyattn_budget(ctypes.byref(p0), None, 0.9, 0, None, None) == 0
    assert lib.proxyattn_select_topk(ctypes.byref(p0), None, None, pa.TOPK_ROW_RATIO, None, None,
                                     None) == 0
    assert lib.proxyattn_dense_prefill(ctypes.byref(p0), None, None, None, None, None, None, 0,
                                       None) == 0
    assert lib.proxyattn_prepare_kv(ctypes.byref(p0), None, None, None, 0, None) == 0
    assert lib.proxyattn_dense_prefill_blocked(ctypes.byref(p0), None, None, 0, None, None, None,
                                               0, None) == 0


@pytest.mark.parametrize("n,hkv,d,b,dtype,esz", [(131072, 8, 128, 128, "bf16", 2),
                                                  (2048, 2, 64, 64, "fp32", 4),
                                                  (1000, 8, 128, 128, "bf16", 2)])
def test_blocked_sizes(n, hkv, d, b, dtype, esz):
    """The blocked K/V copy holds every KV head's keys and values in whole
    blocks (the ragged last block padded); the blocked calls' workspace is
    the kernel's eight 128-byte work-queue lines."""
    _lib()
    prob = _prob(seq_len=n, num_kv_heads=hkv, num_q_heads=4 * hkv, num_proxy_groups=hkv,
                 head_dim=d, block_size=b, dtype=dtype)
    assert pa.proxyattn_kv_blocked_size(prob) == hkv * -(-n // b) * 2 * b * d * esz
    assert pa.proxyattn_blocked_workspace_size(prob) == 8 * 128
    assert pa.proxyattn_kv_blocked_size(_prob(seq_len=0)) == 0
    assert pa.proxyattn_blocked_workspace_size(_prob(seq_len=0)) == 0


def test_binding_rejects_tensors_smaller_than_the_problem():
    """The library sees raw pointers only; the binding checks torch arguments
    against the problem before any call (CPU tensors: nothing is launched).
    Arguments before the one under test are raw pointers (ints), which the
    binding passes through unchecked."""
    import torch
    _lib()
    prob = _prob(seq_len=1000)
    n, hq, hkv, d = prob.seq_len, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    mq = prob.num_blocks
    bf = torch.bfloat16
    fake = 1 << 20
    q = torch.zeros(n, hq, d, dtype=bf)
    small_k = torch.zeros(n // 2, hkv, d, dtype=bf)
    scores = torch.zeros(prob.num_proxy_groups, mq, mq)
    mass = torch.zeros(hq, mq)
    with pytest.raises(pa.ProxyAttnError, match="k: .* touches"):
        pa.proxyattn_estimate(prob, fake, small_k, scores, mass, None)
    with pytest.raises(pa.ProxyAttnError, match="dtype"):
        pa.proxyattn_estimate(prob, q.float(), fake, scores, mass, None)
    bi64 = torch.zeros(hq, mq, mq, dtype=torch.int64)
    with pytest.raises(pa.ProxyAttnError, match="block_index: dtype"):
        pa.proxyattn_block_sparse_prefill(prob, fake, fake, fake, fake, bi64, fake, None, None)
    # a view offset into a larger buffer counts only what lies past its start
    big = torch.zeros(2 * n * hq * d, dtype=bf)
    tail_view = big[n * hq * d + 1:]
    with pytest.raises(pa.ProxyAttnError, match="out: .* touches"):
        pa.proxyattn_dense_prefill(prob, fake, fake, fake, tail_view, None, None)


def test_binding_rejects_host_and_strided_tensors():
    """A host tensor's address must never reach a kernel, and every array
    other than Q, K, V and O is read as packed: full-size CPU tensors and
    non-contiguous views are rejected before anything is launched."""
    import torch
    _lib()
    prob = _prob(seq_len=1000)
    n, hq, hkv, d = prob.seq_len, prob.num_q_heads, prob.num_kv_heads, prob.head_dim
    mq, g = prob.num_blocks, prob.num_proxy_groups
    fake = 1 << 20
    i32 = torch.int32
    q = torch.zeros(n, hq, d, dtype=torch.bfloat16)
    with pytest.raises(pa.ProxyAttnError, match="q: tensor on cpu"):
        pa.proxyattn_estimate(prob, q, fake, fake, fake, fake)
    with pytest.raises(pa.ProxyAttnError, match="head_count: tensor on cpu"):
        pa.proxyattn_select_topk(prob, fake, torch.zeros(hq, dtype=i32), 0, fake, fake)
    with pytest.raises(pa.ProxyAttnError, match="block_index: tensor on cpu"):
        pa.proxyattn_block_sparse_prefill(prob, fake, fake, fake, fake,
                                          torch.zeros(hq, mq, mq, dtype=i32), fake, None, fake)
    with pytest.raises(pa.ProxyAttnError, match="workspace: tensor on cpu"):
        pa.proxyattn_dense_prefill(prob, fake, fake, fake, fake, None,
                                   torch.zeros(64, dtype=torch.uint8))
    # strided views of packed arrays: a transposed score matrix, every other
    # row of a list array, a column of a status matrix
    scores_t = torch.zeros(g, mq, mq).transpose(1, 2)
    with pytest.raises(pa.ProxyAttnError, match="block_logscore: not contiguous"):
        pa.proxyattn_select_topk(prob, scores_t, fake, 0, fake, fake)
    bc_every_other = torch.zeros(hq, 2 * mq, dtype=i32)[:, ::2]
    with pytest.raises(pa.ProxyAttnError, match="block_count: not contiguous"):
        pa.proxyattn_check_lists(prob, bc_every_other, fake, fake)
    mass_t = torch.zeros(mq, hq).t()
    with pytest.raises(pa.ProxyAttnError, match="lastblk_mass: not contiguous"):
        pa.proxyattn_budget(prob, mass_t, 0.9, 0, fake)
