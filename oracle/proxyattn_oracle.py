"""CPU oracle for ProxyAttn's prefill path (test infrastructure only).

TEST INFRASTRUCTURE.  Only the test suite, the package's smoke check and the
CPU-baseline leg of the benchmark may import or run this module.  The product
path (the HIP library and its Python binding) never calls it, and it shares no
code with that path.

Plain, slow NumPy, written step by step from the paper "ProxyAttn: Guided
Sparse Attention via Representative Heads" (arXiv 2509.24745):

  pool_proxy_heads       Sec. 3.1, Eq. 2 (head average pooling) and the
                         strided qk-pair dropping described after it
  proxy_block_logscore   Sec. 3.1, Eq. 1: maxpool(softmax(Q^g K^g^T / sqrt d)),
                         kept in the log domain
  lastblock_mass         Alg. 1, first two steps (last-block softmax, block
                         average pooling)
  budget_counts          Alg. 1, last two steps (normalise, sort, smallest
                         prefix reaching gamma)
  select_blocks          Sec. 3.2, Eq. 3 (per-head Top-K over the shared score)
  block_sparse_attention Sec. 3.2, closing paragraph: causal attention over the
                         selected blocks only
  head_overlap           Eq. 4 (the overlap scores of the sink-token analysis)
                         and the Sec. 2.2 overlap measure it generalises
  shared_ranking_curves  Sec. 2.2: cumulative attention of every head along
                         the ranking by the head-mean attention and along its
                         own ranking

Arithmetic is fp32 (numpy float32), the precision the GPU kernels make their
selection decisions in.  Inputs are fp32 arrays; bf16 problems pass values
that are exactly bf16 (upcast losslessly).

Readings of passages the paper leaves open:
  * pooling: fp32 sum over the group's heads in ascending head order, times
    fl32(1/|G|), rounded to nearest-even bf16 for bf16 problems.  The key of
    query head i is the key of its KV head, so for GQA the pooled key is the
    mean over the group's query heads of their KV heads' keys.  Groups are
    contiguous runs of |G| = Hq/G query heads.
  * stride s keeps tokens t with t mod s == 0 on both the query and the key
    axis; the proxy softmax runs over the kept causal keys, scale 1/sqrt(d).
  * the budget uses each head's own Q and K at full resolution, the last
    min(b, N) query tokens, causal.
  * "avgpool" sums the last-block probabilities over the rows and over the
    keys of each key block: with b keys in every block, mean and sum differ
    by one factor that the normalisation cancels; a partial last key block
    (N not a multiple of b) keeps its sum, the probability it receives.
  * sort is descending; the budget is k*+1 blocks where k* is the first
    0-based prefix index whose cumulative mass reaches gamma (N_k if none,
    and N_k whenever gamma >= 1), then raised to ceil(min_budget/b) and
    capped at N_k.
  * every block row m of head i keeps min(count_i, m+1) blocks: the highest
    shared scores among the causal blocks 0..m, ties to the lower index.
  * attention renormalises over the selected keys (standard block-sparse).
  * ragged N (not a multiple of b): the last block is partial; block counts
    are ceil(N/b), strided length ceil(N/s).
"""
from __future__ import annotations

import math

import numpy as np

F32 = np.float32


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 to the nearest bf16 value, ties to even (result in fp32)."""
    bits = np.ascontiguousarray(x, dtype=F32).view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    bits = (bits + lsb + np.uint32(0x7FFF)) & np.uint32(0xFFFF0000)
    return bits.view(F32)


def default_scale(head_dim: int) -> float:
    return 1.0 / math.sqrt(head_dim)


def num_blocks(n: int, b: int) -> int:
    return -(-n // b)


# --------------------------------------------------------------------------
# Sec. 3.1, Eq. 2 + strided dropping
# --------------------------------------------------------------------------
def pool_proxy_heads(q: np.ndarray, k: np.ndarray, num_groups: int, stride: int,
                     dtype: str = "bf16"):
    """Proxy queries and keys, one per group, on the strided tokens.

    q: [N, Hq, d], k: [N, Hkv, d]  ->  qg, kg: [G, ceil(N/s), d] (fp32 arrays;
    for dtype "bf16" every value is a bf16 value).
    """
    n, hq, d = q.shape
    hkv = k.shape[1]
    assert hq % hkv == 0 and hq % num_groups == 0
    rep = hq // hkv                      # query heads per KV head
    gsize = hq // num_groups             # |G|
    qs = q[::stride].astype(F32)         # keep t = s*t'
    ks = k[::stride].astype(F32)
    inv = F32(1.0) / F32(gsize)
    npr = qs.shape[0]
    qg = np.empty((num_groups, npr, d), dtype=F32)
    kg = np.empty((num_groups, npr, d), dtype=F32)
    for g in range(num_groups):
        acc_q = np.zeros((npr, d), dtype=F32)
        acc_k = np.zeros((npr, d), dtype=F32)
        for i in range(g * gsize, (g + 1) * gsize):
            acc_q = acc_q + qs[:, i, :]
            acc_k = acc_k + ks[:, i // rep, :]
        qg[g] = acc_q * inv
        kg[g] = acc_k * inv
    if dtype == "bf16":
        qg, kg = round_to_bf16(qg), round_to_bf16(kg)
    return qg, kg


# --------------------------------------------------------------------------
# Sec. 3.1, Eq. 1 (log domain)
# --------------------------------------------------------------------------
def proxy_block_logscore(qg: np.ndarray, kg: np.ndarray, seq_len: int, block_size: int,
                         stride: int, scale: float, rows=None):
    """log of maxpool(softmax(c * Q^g K^g^T)) over b x b token blocks.

    The softmax of strided row t' runs over the strided keys u' <= t'.  The
    max-pool of block (m, n) is over its strided rows and keys (u' <= t').
    Returns (logA [G, Mq, Nk] with -inf for n > m, L [G, N'] row log-sum-exp).
    ``rows``: optional iterable of block rows m to compute (others stay -inf).
    """
    g_count, npr, d = qg.shape
    bp = block_size // stride                         # strided rows per block
    mq = num_blocks(seq_len, block_size)
    logA = np.full((g_count, mq, mq), -np.inf, dtype=F32)
    lse = np.full((g_count, npr), np.nan, dtype=F32)
    sc = F32(scale)
    row_list = range(mq) if rows is None else sorted(set(int(r) for r in rows))
    for g in range(g_count):
        for m in row_list:
            r0, r1 = m * bp, min((m + 1) * bp, npr)
            if r0 >= r1:
                continue
            s = sc * (qg[g, r0:r1] @ kg[g, :r1].T)     # [rows, keys u' < r1]
            t_idx = np.arange(r0, r1)[:, None]
            u_idx = np.arange(r1)[None, :]
            s = np.where(u_idx <= t_idx, s, F32(-np.inf))
            mx = s.max(axis=1, keepdims=True)
            row_lse = mx[:, 0] + np.log(np.exp(s - mx).sum(axis=1, dtype=F32))
            lse[g, r0:r1] = row_lse
            z = s - row_lse[:, None]                    # log softmax
            for n in range(m + 1):
                c0, c1 = n * bp, min((n + 1) * bp, r1)
                logA[g, m, n] = z[:, c0:c1].max()
    return logA, lse


# --------------------------------------------------------------------------
# Alg. 1, steps 1-2
# --------------------------------------------------------------------------
def lastblock_mass(q: np.ndarray, k: np.ndarray, block_size: int, scale: float):
    """Per head, block-pooled causal attention mass of the last query block.

    Rows are the last min(b, N) query tokens, keys all u <= t at full
    resolution, each head with its own KV head.  Returns mass [Hq, Nk]
    (fp32); each row sums to the number of rows.
    """
    n, hq, d = q.shape
    hkv = k.shape[1]
    rep = hq // hkv
    nk = num_blocks(n, block_size)
    rows = np.arange(max(0, n - block_size), n)
    sc = F32(scale)
    mass = np.zeros((hq, nk), dtype=F32)
    pad = nk * block_size - n
    for i in range(hq):
        s = sc * (q[rows, i, :].astype(F32) @ k[:, i // rep, :].astype(F32).T)   # [rows, N]
        s = np.where(np.arange(n)[None, :] <= rows[:, None], s, F32(-np.inf))
        mx = s.max(axis=1, keepdims=True)
        e = np.exp(s - mx)
        p = e / e.sum(axis=1, keepdims=True, dtype=F32)
        p = np.concatenate([p, np.zeros((p.shape[0], pad), dtype=F32)], axis=1)
        mass[i] = p.reshape(p.shape[0], nk, block_size).sum(axis=(0, 2), dtype=F32)
    return mass


# --------------------------------------------------------------------------
# Alg. 1, steps 3-4
# --------------------------------------------------------------------------
def budget_counts(mass: np.ndarray, gamma: float, min_budget_tokens: int, block_size: int):
    """Per-head block budget: the fewest top blocks whose share reaches gamma.

    Returns (count [Hq] int32, cumulative [Hq, Nk] fp32 sorted prefix sums).
    """
    hq, nk = mass.shape
    floor_blocks = -(-int(min_budget_tokens) // block_size)
    counts = np.empty(hq, dtype=np.int32)
    cums = np.empty((hq, nk), dtype=F32)
    g32 = F32(gamma)
    for i in range(hq):
        a = mass[i].astype(F32) / mass[i].astype(F32).sum(dtype=F32)
        a_sorted = -np.sort(-a)
        cum = np.cumsum(a_sorted, dtype=F32)
        cums[i] = cum
        hit = np.nonzero(cum >= g32)[0]
        # gamma >= 1 asks for all the mass: the full budget, whatever fp32
        # rounding does to the last prefix sums
        k_star = int(hit[0]) if (hit.size and gamma < 1.0) else nk - 1
        counts[i] = min(nk, max(k_star + 1, floor_blocks))
    return counts, cums


# --------------------------------------------------------------------------
# Sec. 3.2, Eq. 3
# --------------------------------------------------------------------------
def row_budget(count: int, m: int, nk: int, row_ratio: bool = False) -> int:
    """Eq. 3's K = b_i N for block row m, with b_i = count / Nk.

    Constant reading (N = Nk, the block-level sequence length): count blocks,
    capped at the row's m+1 causal blocks.  Per-row-ratio reading (N = m+1):
    ceil(b_i (m+1)) blocks, the same fraction of every row.
    """
    count = min(max(int(count), 0), nk)
    if not row_ratio:
        return min(count, m + 1)
    return min(-(-count * (m + 1) // nk), m + 1)


def select_blocks(logA: np.ndarray, counts: np.ndarray, num_q_heads: int, rows=None,
                  row_ratio: bool = False):
    """Per head i and block row m: the row_budget(count_i, m) causal blocks
    with the highest shared score of the head's group (ties -> lower index),
    listed in ascending order (Eq. 3).

    Returns (block_count [Hq, Mq] int32, block_index [Hq, Mq, Nk] int32, -1 pad).
    """
    g_count, mq, nk = logA.shape
    gsize = num_q_heads // g_count
    block_count = np.zeros((num_q_heads, mq), dtype=np.int32)
    block_index = np.full((num_q_heads, mq, nk), -1, dtype=np.int32)
    row_list = range(mq) if rows is None else sorted(set(int(r) for r in rows))
    for g in range(g_count):
        for m in row_list:
            cand = np.arange(m + 1)
            order = np.lexsort((cand, -logA[g, m, :m + 1]))   # score desc, index asc
            for i in range(g * gsize, (g + 1) * gsize):
                kk = row_budget(counts[i], m, nk, row_ratio)
                block_index[i, m, :kk] = np.sort(order[:kk])
                block_count[i, m] = kk
    return block_count, block_index


# --------------------------------------------------------------------------
# Block-sparse causal attention over the selected blocks
# --------------------------------------------------------------------------
def block_sparse_attention(q, k, v, block_count, block_index, block_size: int, scale: float,
                           query_rows=None):
    """O[t, i] = softmax over the selected causal keys of c*<q, k>, times V.

    Returns (out [N, Hq, d] fp32, lse [Hq, N] fp32).  ``query_rows``:
    optional sorted token indices to compute (others stay NaN).
    """
    n, hq, d = q.shape
    hkv = k.shape[1]
    rep = hq // hkv
    mq = num_blocks(n, block_size)
    out = np.full((n, hq, d), np.nan, dtype=F32)
    lse = np.full((hq, n), np.nan, dtype=F32)
    sc = F32(scale)
    if query_rows is None:
        rows_by_block = {m: np.arange(m * block_size, min((m + 1) * block_size, n)) for m in range(mq)}
    else:
        qr = np.asarray(sorted(set(int(t) for t in query_rows)), dtype=np.int64)
        rows_by_block = {}
        for m in np.unique(qr // block_size):
            rows_by_block[int(m)] = qr[qr // block_size == m]
    for i in range(hq):
        kh, vh = k[:, i // rep, :].astype(F32), v[:, i // rep, :].astype(F32)
        for m, trow in rows_by_block.items():
            blocks = block_index[i, m, :block_count[i, m]]
            keys = np.concatenate([np.arange(bn * block_size, min((bn + 1) * block_size, n))
                                   for bn in blocks])
            s = sc * (q[trow, i, :].astype(F32) @ kh[keys].T)
            s = np.where(keys[None, :] <= trow[:, None], s, F32(-np.inf))
            mx = s.max(axis=1, keepdims=True)
            e = np.exp(s - mx)
            den = e.sum(axis=1, keepdims=True, dtype=F32)
            out[trow, i, :] = (e / den) @ vh[keys]
            lse[i, trow] = mx[:, 0] + np.log(den[:, 0])
    return out, lse


def full_causal_lists(seq_len: int, num_q_heads: int, block_size: int):
    """Every causal block in every row: the lists a full budget produces."""
    mq = num_blocks(seq_len, block_size)
    block_count = np.tile(np.arange(1, mq + 1, dtype=np.int32), (num_q_heads, 1))
    block_index = np.full((num_q_heads, mq, mq), -1, dtype=np.int32)
    for m in range(mq):
        block_index[:, m, :m + 1] = np.arange(m + 1, dtype=np.int32)
    return block_count, block_index


# --------------------------------------------------------------------------
# The whole path
# --------------------------------------------------------------------------
def proxyattn_prefill(q, k, v, *, num_groups: int, block_size: int, stride: int, gamma: float,
                      min_budget_tokens: int = 0, scale: float | None = None,
                      dtype: str = "bf16", est_rows=None, query_rows=None):
    """Run estimation -> budget -> selection -> block-sparse attention.

    ``est_rows``: block rows for which to compute scores and lists (default
    all); ``query_rows``: token rows for which to compute attention (default
    all; their block rows are added to ``est_rows``).
    """
    n, hq, d = q.shape
    sc = default_scale(d) if scale is None or scale <= 0 else scale
    if query_rows is not None:
        qb = set(int(t) // block_size for t in query_rows)
        est_rows = sorted(qb if est_rows is None else (set(est_rows) | qb))
    qg, kg = pool_proxy_heads(q, k, num_groups, stride, dtype)
    logA, proxy_lse = proxy_block_logscore(qg, kg, n, block_size, stride, sc, rows=est_rows)
    mass = lastblock_mass(q, k, block_size, sc)
    counts, cums = budget_counts(mass, gamma, min_budget_tokens, block_size)
    block_count, block_index = select_blocks(logA, counts, hq, rows=est_rows)
    if v is not None:
        out, lse = block_sparse_attention(q, k, v, block_count, block_index, block_size, sc,
                                          query_rows=query_rows)
    else:
        out, lse = None, None
    return dict(qg=qg, kg=kg, logA=logA, proxy_lse=proxy_lse, mass=mass, counts=counts,
                cums=cums, block_count=block_count, block_index=block_index, out=out, lse=lse,
                scale=sc)


# --------------------------------------------------------------------------
# Head-similarity diagnostics (Sec. 2.2 and the sink-token analysis, Eq. 4)
# --------------------------------------------------------------------------
def token_attention(q: np.ndarray, k: np.ndarray, t: int, scale: float) -> np.ndarray:
    """Causal attention probabilities of query token t for every head at full
    resolution: A [Hq, t+1] (fp32), head i against its KV head's keys."""
    hq = q.shape[1]
    rep = hq // k.shape[1]
    a = np.empty((hq, t + 1), dtype=F32)
    for i in range(hq):
        s = F32(scale) * (k[:t + 1, i // rep] @ q[t, i])
        e = np.exp(s - s.max())
        a[i] = e / e.sum(dtype=F32)
    return a


def head_overlap(q: np.ndarray, k: np.ndarray, t: int, topk: int, scale: float,
                 sink_tokens: int = 0, renormalize: bool = False) -> np.ndarray:
    """Eq. 4: Score[i, j] = the attention head j gives to the top-k tokens of
    head i (query token t; ties between equal scores go to the lower token).

    ``sink_tokens``: the attention to the first n tokens is removed first
    (set to zero); ``renormalize``: each head's remaining attention is then
    rescaled to sum 1 (a head with nothing left stays all zero).
    Returns Score [Hq, Hq] fp32 (sums taken in float64).
    """
    a = token_attention(q, k, t, scale)
    if sink_tokens:
        a[:, :sink_tokens] = 0.0
    if renormalize:
        tot = a.sum(axis=1, dtype=F32, keepdims=True)
        a = np.where(tot > 0, a / np.where(tot > 0, tot, F32(1)), F32(0)).astype(F32)
    hq, n1 = a.shape
    kk = min(int(topk), n1)
    tokens = np.arange(n1)
    score = np.empty((hq, hq), dtype=F32)
    for i in range(hq):
        top = np.lexsort((tokens, -a[i]))[:kk]           # score desc, token asc
        for j in range(hq):
            score[i, j] = a[j, top].sum(dtype=np.float64)
    return score


def shared_ranking_curves(q: np.ndarray, k: np.ndarray, t: int, scale: float, points):
    """Sec. 2.2: rank the tokens by their mean attention over the heads; for
    every head, the cumulative attention of the first p tokens of that shared
    ranking and of the head's own ranking, for p in ``points``.
    Returns (shared [Hq, P], own [Hq, P]) in float64."""
    a = token_attention(q, k, t, scale).astype(np.float64)
    hq, n1 = a.shape
    tokens = np.arange(n1)
    shared_order = np.lexsort((tokens, -a.mean(axis=0)))
    pts = [min(int(p), n1) for p in points]
    shared = np.empty((hq, len(pts)))
    own = np.empty((hq, len(pts)))
    for i in range(hq):
        cs = np.cumsum(a[i, shared_order])
        co = np.cumsum(np.sort(a[i])[::-1])
        shared[i] = [cs[p - 1] if p else 0.0 for p in pts]
        own[i] = [co[p - 1] if p else 0.0 for p in pts]
    return shared, own
