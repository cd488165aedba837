"""Python binding of libproxyattn.so (argument marshalling only).

The functions here carry the C ABI's names and arguments (see
include/proxyattn.h).  Tensors are torch tensors on the GPU; only their
device pointers and the current HIP stream cross the boundary.  Every step
of the path runs in the library's HIP kernels: there is no fallback, and the
module raises ImportError when the library has not been built.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

import torch  # loaded first: the library then binds to torch's HIP runtime

_HERE = os.path.dirname(os.path.abspath(__file__))
# PROXYATTN_LIBRARY selects another build of the library (the sanitized host
# build for the boundary tests); by default the one next to this file
LIB_PATH = os.environ.get("PROXYATTN_LIBRARY") or os.path.join(_HERE, "libproxyattn.so")

BF16 = 0
F32 = 1

E_OK, E_INVALID, E_UNSUPPORTED, E_WORKSPACE, E_HIP = 0, 1, 2, 3, 4
TOPK_CONSTANT, TOPK_ROW_RATIO, LIST_ASCENDING = 0, 1, 2
LIST_BAD_COUNT, LIST_BAD_INDEX, LIST_DUPLICATE = 1, 2, 4


class proxyattn_problem(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("seq_len", ctypes.c_int32),
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_size", ctypes.c_int32),
        ("num_proxy_groups", ctypes.c_int32),
        ("stride", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("softmax_scale", ctypes.c_float),
        ("q_tok_stride", ctypes.c_int64),
        ("q_head_stride", ctypes.c_int64),
        ("kv_tok_stride", ctypes.c_int64),
        ("kv_head_stride", ctypes.c_int64),
        ("o_tok_stride", ctypes.c_int64),
        ("o_head_stride", ctypes.c_int64),
        ("attn_order", ctypes.c_int32),
        ("attn_chunk_rows", ctypes.c_int32),
    ]


_SIGS = {
    "proxyattn_workspace_size": [ctypes.c_void_p, ctypes.c_void_p],
    "proxyattn_workspace_layout": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "proxyattn_estimate": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_select_budget": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float,
                                ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p],
    "proxyattn_budget": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_float, ctypes.c_int32,
                         ctypes.c_void_p, ctypes.c_void_p],
    "proxyattn_select_topk": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
    "proxyattn_head_overlap": [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                               ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                               ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_check_lists": [ctypes.c_void_p] * 5,
    "proxyattn_block_sparse_prefill": [ctypes.c_void_p] * 9 + [ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_dense_prefill": [ctypes.c_void_p] * 7 + [ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_kv_blocked_size": [ctypes.c_void_p, ctypes.c_void_p],
    "proxyattn_prepare_kv": [ctypes.c_void_p] * 4 + [ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_blocked_workspace_size": [ctypes.c_void_p, ctypes.c_void_p],
    "proxyattn_block_sparse_prefill_blocked": [ctypes.c_void_p] * 3 + [ctypes.c_size_t]
                                              + [ctypes.c_void_p] * 5
                                              + [ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_dense_prefill_blocked": [ctypes.c_void_p] * 3 + [ctypes.c_size_t]
                                       + [ctypes.c_void_p] * 3 + [ctypes.c_size_t, ctypes.c_void_p],
    "proxyattn_block_sparse_prefill_blocked_noalloc": [ctypes.c_void_p] * 3 + [ctypes.c_size_t]
                                                      + [ctypes.c_void_p] * 5,
    "proxyattn_error_string": [ctypes.c_int],
    "proxyattn_last_error": [],
    "proxyattn_version": [],
}
EXPORTS = tuple(_SIGS)


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with `python -m paper_2509_24745_amd.build`")
    lib = ctypes.CDLL(path)
    for name, args in _SIGS.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name in ("proxyattn_error_string", "proxyattn_last_error",
                                                 "proxyattn_version") else ctypes.c_int
    return lib


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        _lib = load_library()
    return _lib


class ProxyAttnError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


def _check(rc: int):
    if rc != E_OK:
        L = lib()
        raise ProxyAttnError(rc, f"{L.proxyattn_error_string(rc).decode()}: "
                                 f"{L.proxyattn_last_error().decode()}")


@dataclass(frozen=True)
class Problem:
    """Host-side problem description (mirrors proxyattn_problem)."""

    seq_len: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    num_proxy_groups: int
    stride: int = 4
    dtype: str = "bf16"
    softmax_scale: float = 0.0
    q_tok_stride: int = 0
    q_head_stride: int = 0
    kv_tok_stride: int = 0
    kv_head_stride: int = 0
    o_tok_stride: int = 0
    o_head_stride: int = 0
    attn_order: int = 0        # 0 by kernel and size; 1 plain, 2 row chunks, 3 KV-head-major chunks then short rows
    attn_chunk_rows: int = 0   # 0 by size

    @property
    def num_blocks(self) -> int:
        return -(-self.seq_len // self.block_size)

    @property
    def scale(self) -> float:
        return self.softmax_scale if self.softmax_scale > 0 else 1.0 / math.sqrt(self.head_dim)

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == "bf16" else torch.float32

    def c_struct(self) -> proxyattn_problem:
        p = proxyattn_problem()
        p.struct_size = ctypes.sizeof(proxyattn_problem)
        p.seq_len = self.seq_len
        p.num_q_heads = self.num_q_heads
        p.num_kv_heads = self.num_kv_heads
        p.head_dim = self.head_dim
        p.block_size = self.block_size
        p.num_proxy_groups = self.num_proxy_groups
        p.stride = self.stride
        p.dtype = BF16 if self.dtype == "bf16" else (F32 if self.dtype == "fp32" else 99)
        p.softmax_scale = self.softmax_scale
        p.q_tok_stride, p.q_head_stride = self.q_tok_stride, self.q_head_stride
        p.kv_tok_stride, p.kv_head_stride = self.kv_tok_stride, self.kv_head_stride
        p.o_tok_stride, p.o_head_stride = self.o_tok_stride, self.o_head_stride
        p.attn_order, p.attn_chunk_rows = self.attn_order, self.attn_chunk_rows
        return p


def _ptr(x) -> int | None:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _nbytes(x) -> int:
    return x.numel() * x.element_size()


def _stream(stream) -> int | None:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def proxyattn_workspace_size(prob: Problem) -> int:
    n = ctypes.c_size_t(0)
    p = prob.c_struct()
    _check(lib().proxyattn_workspace_size(ctypes.byref(p), ctypes.byref(n)))
    return n.value


def proxyattn_kv_blocked_size(prob: Problem) -> int:
    n = ctypes.c_size_t(0)
    p = prob.c_struct()
    _check(lib().proxyattn_kv_blocked_size(ctypes.byref(p), ctypes.byref(n)))
    return n.value


def proxyattn_blocked_workspace_size(prob: Problem) -> int:
    n = ctypes.c_size_t(0)
    p = prob.c_struct()
    _check(lib().proxyattn_blocked_workspace_size(ctypes.byref(p), ctypes.byref(n)))
    return n.value


def proxyattn_workspace_layout(prob: Problem):
    a, b = ctypes.c_size_t(0), ctypes.c_size_t(0)
    p = prob.c_struct()
    _check(lib().proxyattn_workspace_layout(ctypes.byref(p), ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


# Checks of torch arguments: the library receives raw pointers and cannot see
# the allocations, so a tensor smaller than the problem would be read or
# written out of bounds, and a host tensor's address would reach a kernel as
# if it were device memory.  Each check needs the number of elements the call
# touches from the tensor's data pointer (ints are raw pointers and are passed
# through unchecked).  Q, K, V and O may be strided views (the problem carries
# their strides); every other array is read as packed, so it must be
# contiguous.
def _need(x, n_elems: int, name: str, dtype=None, contiguous: bool = True):
    if x is None or isinstance(x, int) or n_elems <= 0:
        return
    if dtype is not None and x.dtype != dtype:
        raise ProxyAttnError(E_INVALID, f"{name}: dtype {x.dtype}, the problem needs {dtype}")
    avail = x.untyped_storage().nbytes() // x.element_size() - x.storage_offset()
    if avail < n_elems:
        raise ProxyAttnError(E_INVALID, f"{name}: {avail} elements from its data pointer, the "
                                        f"problem touches {n_elems}")
    if contiguous and not x.is_contiguous():
        raise ProxyAttnError(E_INVALID, f"{name}: not contiguous (read as a packed array)")
    if not x.is_cuda:
        raise ProxyAttnError(E_INVALID, f"{name}: tensor on {x.device}, the library needs "
                                        f"device memory of the current GPU")
    if x.device.index != torch.cuda.current_device():
        raise ProxyAttnError(E_INVALID, f"{name}: tensor on {x.device}, the current device is "
                                        f"cuda:{torch.cuda.current_device()}")


def _need_ws(workspace, n_bytes: int, name: str = "workspace"):
    """A workspace of at least n_bytes on the current GPU (sizes are checked
    again by the library against what the problem needs)."""
    if workspace is None or isinstance(workspace, int):
        return
    _need(workspace, 1, name)
    if workspace.numel() * workspace.element_size() < n_bytes:
        raise ProxyAttnError(E_WORKSPACE, f"{name}: {workspace.numel() * workspace.element_size()}"
                                          f" bytes, the problem needs {n_bytes}")


def _span(n, heads, d, tok_stride, head_stride):
    tok = tok_stride or heads * d
    head = head_stride or d
    return (n - 1) * tok + (heads - 1) * head + d if n > 0 else 0


def _need_q(prob: Problem, q, name="q"):
    _need(q, _span(prob.seq_len, prob.num_q_heads, prob.head_dim, prob.q_tok_stride,
                   prob.q_head_stride), name, prob.torch_dtype, contiguous=False)


def _need_kv(prob: Problem, x, name):
    _need(x, _span(prob.seq_len, prob.num_kv_heads, prob.head_dim, prob.kv_tok_stride,
                   prob.kv_head_stride), name, prob.torch_dtype, contiguous=False)


def _need_out(prob: Problem, out):
    _need(out, _span(prob.seq_len, prob.num_q_heads, prob.head_dim, prob.o_tok_stride,
                     prob.o_head_stride), "out", prob.torch_dtype, contiguous=False)


def _need_scores(prob: Problem, block_logscore):
    mq = prob.num_blocks
    _need(block_logscore, prob.num_proxy_groups * mq * mq, "block_logscore", torch.float32)


def _need_lists(prob: Problem, block_count, block_index):
    mq = prob.num_blocks
    _need(block_count, prob.num_q_heads * mq, "block_count", torch.int32)
    _need(block_index, prob.num_q_heads * mq * mq, "block_index", torch.int32)


def proxyattn_estimate(prob: Problem, q, k, block_logscore, lastblk_mass, workspace, stream=None):
    _need_q(prob, q)
    _need_kv(prob, k, "k")
    _need_scores(prob, block_logscore)
    _need(lastblk_mass, prob.num_q_heads * prob.num_blocks, "lastblk_mass", torch.float32)
    _need_ws(workspace, 0)
    p = prob.c_struct()
    _check(lib().proxyattn_estimate(ctypes.byref(p), _ptr(q), _ptr(k), _ptr(block_logscore),
                                    _ptr(lastblk_mass), _ptr(workspace), _nbytes(workspace)
                                    if workspace is not None else 0, _stream(stream)))


def proxyattn_select_budget(prob: Problem, block_logscore, lastblk_mass, gamma: float,
                            min_budget_tokens: int, head_count, block_count, block_index,
                            stream=None):
    _need_scores(prob, block_logscore)
    _need(lastblk_mass, prob.num_q_heads * prob.num_blocks, "lastblk_mass", torch.float32)
    _need(head_count, prob.num_q_heads, "head_count", torch.int32)
    _need_lists(prob, block_count, block_index)
    p = prob.c_struct()
    _check(lib().proxyattn_select_budget(ctypes.byref(p), _ptr(block_logscore), _ptr(lastblk_mass),
                                         float(gamma), int(min_budget_tokens), _ptr(head_count),
                                         _ptr(block_count), _ptr(block_index), _stream(stream)))


def proxyattn_budget(prob: Problem, lastblk_mass, gamma: float, min_budget_tokens: int, head_count,
                     stream=None):
    _need(lastblk_mass, prob.num_q_heads * prob.num_blocks, "lastblk_mass", torch.float32)
    _need(head_count, prob.num_q_heads, "head_count", torch.int32)
    p = prob.c_struct()
    _check(lib().proxyattn_budget(ctypes.byref(p), _ptr(lastblk_mass), float(gamma),
                                  int(min_budget_tokens), _ptr(head_count), _stream(stream)))


def proxyattn_select_topk(prob: Problem, block_logscore, head_count, mode: int, block_count,
                          block_index, stream=None):
    _need_scores(prob, block_logscore)
    _need(head_count, prob.num_q_heads, "head_count", torch.int32)
    _need_lists(prob, block_count, block_index)
    p = prob.c_struct()
    _check(lib().proxyattn_select_topk(ctypes.byref(p), _ptr(block_logscore), _ptr(head_count),
                                       int(mode), _ptr(block_count), _ptr(block_index),
                                       _stream(stream)))


def proxyattn_head_overlap(prob: Problem, q, k, query_token: int, topk: int, sink_tokens: int,
                           renormalize: bool, scores, workspace, stream=None):
    _need_q(prob, q)
    _need_kv(prob, k, "k")
    _need(scores, prob.num_q_heads * prob.num_q_heads, "scores", torch.float32)
    _need_ws(workspace, 0)
    p = prob.c_struct()
    _check(lib().proxyattn_head_overlap(ctypes.byref(p), _ptr(q), _ptr(k), int(query_token),
                                        int(topk), int(sink_tokens), int(bool(renormalize)),
                                        _ptr(scores), _ptr(workspace),
                                        _nbytes(workspace) if workspace is not None else 0,
                                        _stream(stream)))


def proxyattn_check_lists(prob: Problem, block_count, block_index, status, stream=None):
    _need_lists(prob, block_count, block_index)
    _need(status, prob.num_q_heads * prob.num_blocks, "status", torch.int32)
    p = prob.c_struct()
    _check(lib().proxyattn_check_lists(ctypes.byref(p), _ptr(block_count), _ptr(block_index),
                                       _ptr(status), _stream(stream)))


def proxyattn_block_sparse_prefill(prob: Problem, q, k, v, block_count, block_index, out, lse,
                                   workspace, stream=None):
    _need_q(prob, q)
    _need_kv(prob, k, "k")
    _need_kv(prob, v, "v")
    _need_lists(prob, block_count, block_index)
    _need_out(prob, out)
    _need(lse, prob.num_q_heads * prob.seq_len, "lse", torch.float32)
    _need_ws(workspace, 0)
    p = prob.c_struct()
    _check(lib().proxyattn_block_sparse_prefill(
        ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(block_count), _ptr(block_index),
        _ptr(out), _ptr(lse), _ptr(workspace),
        _nbytes(workspace) if workspace is not None else 0, _stream(stream)))


def proxyattn_dense_prefill(prob: Problem, q, k, v, out, lse, workspace, stream=None):
    _need_q(prob, q)
    _need_kv(prob, k, "k")
    _need_kv(prob, v, "v")
    _need_out(prob, out)
    _need(lse, prob.num_q_heads * prob.seq_len, "lse", torch.float32)
    _need_ws(workspace, 0)
    p = prob.c_struct()
    _check(lib().proxyattn_dense_prefill(
        ctypes.byref(p), _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(workspace),
        _nbytes(workspace) if workspace is not None else 0, _stream(stream)))


def _need_kvb(prob: Problem, kv_blocked):
    if kv_blocked is None or isinstance(kv_blocked, int):
        return
    _need_ws(kv_blocked, proxyattn_kv_blocked_size(prob), "kv_blocked")


def proxyattn_prepare_kv(prob: Problem, k, v, kv_blocked, stream=None):
    _need_kv(prob, k, "k")
    _need_kv(prob, v, "v")
    _need_kvb(prob, kv_blocked)
    p = prob.c_struct()
    _check(lib().proxyattn_prepare_kv(ctypes.byref(p), _ptr(k), _ptr(v), _ptr(kv_blocked),
                                      _nbytes(kv_blocked) if kv_blocked is not None else 0,
                                      _stream(stream)))


def proxyattn_block_sparse_prefill_blocked(prob: Problem, q, kv_blocked, block_count, block_index,
                                           out, lse, workspace, stream=None):
    _need_q(prob, q)
    _need_kvb(prob, kv_blocked)
    _need_lists(prob, block_count, block_index)
    _need_out(prob, out)
    _need(lse, prob.num_q_heads * prob.seq_len, "lse", torch.float32)
    _need_ws(workspace, 0)
    p = prob.c_struct()
    _check(lib().proxyattn_block_sparse_prefill_blocked(
        ctypes.byref(p), _ptr(q), _ptr(kv_blocked),
        _nbytes(kv_blocked) if kv_blocked is not None else 0, _ptr(block_count),
        _ptr(block_index), _ptr(out), _ptr(lse), _ptr(workspace),
        _nbytes(workspace) if workspace is not None else 0, _stream(stream)))


def proxyattn_block_sparse_prefill_blocked_noalloc(prob: Problem, q, kv_blocked, block_count,
                                                   block_index, out, lse, stream=None):
    _need_q(prob, q)
    _need_kvb(prob, kv_blocked)
    _need_lists(prob, block_count, block_index)
    _need_out(prob, out)
    _need(lse, prob.num_q_heads * prob.seq_len, "lse", torch.float32)
    p = prob.c_struct()
    _check(lib().proxyattn_block_sparse_prefill_blocked_noalloc(
        ctypes.byref(p), _ptr(q), _ptr(kv_blocked),
        _nbytes(kv_blocked) if kv_blocked is not None else 0, _ptr(block_count),
        _ptr(block_index), _ptr(out), _ptr(lse), _stream(stream)))


def proxyattn_dense_prefill_blocked(prob: Problem, q, kv_blocked, out, lse, workspace,
                                    stream=None):
    _need_q(prob, q)
    _need_kvb(prob, kv_blocked)
    _need_out(prob, out)
    _need(lse, prob.num_q_heads * prob.seq_len, "lse", torch.float32)
    _need_ws(workspace, 0)
    p = prob.c_struct()
    _check(lib().proxyattn_dense_prefill_blocked(
        ctypes.byref(p), _ptr(q), _ptr(kv_blocked),
        _nbytes(kv_blocked) if kv_blocked is not None else 0, _ptr(out), _ptr(lse),
        _ptr(workspace), _nbytes(workspace) if workspace is not None else 0, _stream(stream)))


def proxyattn_version() -> str:
    return lib().proxyattn_version().decode()


class Buffers:
    """Device buffers for one problem (allocation through torch only)."""

    def __init__(self, prob: Problem, device="cuda"):
        g, mq, hq = prob.num_proxy_groups, prob.num_blocks, prob.num_q_heads
        n, d = prob.seq_len, prob.head_dim
        f32, i32 = torch.float32, torch.int32
        self.prob = prob
        self.workspace = torch.empty(max(proxyattn_workspace_size(prob), 16), dtype=torch.uint8,
                                     device=device)
        self.logscore = torch.empty((g, mq, mq), dtype=f32, device=device)
        self.mass = torch.empty((hq, mq), dtype=f32, device=device)
        self.head_count = torch.empty(hq, dtype=i32, device=device)
        self.block_count = torch.empty((hq, mq), dtype=i32, device=device)
        self.block_index = torch.empty((hq, mq, mq), dtype=i32, device=device)
        self.out = torch.empty((n, hq, d), dtype=prob.torch_dtype, device=device)
        self.lse = torch.empty((hq, n), dtype=f32, device=device)


def prefill(prob: Problem, q, k, v, gamma: float, min_budget_tokens: int = 0,
            bufs: Buffers | None = None, stream=None) -> Buffers:
    """Run the three steps (estimate, select_budget, block_sparse_prefill)."""
    bufs = bufs or Buffers(prob, q.device)
    proxyattn_estimate(prob, q, k, bufs.logscore, bufs.mass, bufs.workspace, stream)
    proxyattn_select_budget(prob, bufs.logscore, bufs.mass, gamma, min_budget_tokens,
                            bufs.head_count, bufs.block_count, bufs.block_index, stream)
    proxyattn_block_sparse_prefill(prob, q, k, v, bufs.block_count, bufs.block_index, bufs.out,
                                   bufs.lse, bufs.workspace, stream)
    return bufs
