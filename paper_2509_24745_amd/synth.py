"""Seeded synthetic Q/K/V for one long-context prefill attention layer.

This module only draws inputs. It holds none of ProxyAttn's arithmetic (no
pooling, scoring, budgeting, selection or attention), so both the HIP path
and the CPU oracle may consume what it produces.

The paper measures speed on Q/K/V cached from real long-context prompts
(Sec. 4.3); those activations and the model weights are not available, so
these inputs stand in for them.  They are built to carry the structure the
method relies on (Sec. 2.2): heads of one key group attend to largely the
same tokens, heads differ in how sparse they are, a sink token at position 0,
a recency window, and a handful of strongly attended far-away key blocks.

Construction, per KV head h (all draws from one numpy PCG64 stream, in the
fixed order documented in ``generate``):

* shared content ``x_t = Z_t B_h``: ``Z`` is a rank-``rank`` Gaussian AR(1)
  process along the sequence with correlation length ``corr_len`` tokens and
  unit marginal variance, ``B_h`` an ``rank x d`` N(0, 1/rank) basis.  Because
  ``Z`` varies smoothly, keys near the query and keys in far regions whose
  latent happens to align with the query's receive high logits; this gives
  block-level (not token-level) sparsity.
* per-head deviation ``sigma * y^i_t``: an independent process of the same
  law for every query head and every KV head.  ``sigma`` sets how far a head's
  pattern departs from its group's (head similarity).
* iid token noise of std ``iid_noise`` on Q and K.
* sink: key 0 gets a logit bonus ``sink_logit`` for every query of the group.
* hot blocks: ``hot_blocks`` key blocks drawn from [1, Nk) get a logit bonus
  ``hot_logit`` for every query of the group.
* per-head temperature: query head i is scaled by ``temp_i`` drawn
  log-uniformly from ``[1/temp_spread, temp_spread]`` (heads differ in
  sparsity).  ``hetero`` instead alternates flat heads (x0.1) and sharp
  local-plus-sink heads inside every KV group.
* V is iid N(0, 1).

``content_logit`` is the standard deviation of the shared-content logit
between two distant tokens, c * <q, k>; the query scale is derived from it.

Values are produced in fp32 and, for bf16 workloads, rounded to nearest-even
bf16 once, so the GPU and the oracle see identical bits.
"""
from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import numpy as np
from scipy.signal import lfilter


@dataclass(frozen=True)
class Structure:
    """Structure constants of the synthetic attention workload."""

    rank: int = 16
    noise: float = 0.3          # sigma: per-head deviation, relative to shared
    corr_len: float = 1024.0    # tokens; correlation length of the latent
    content_logit: float = 3.1  # std of c*<q,k> between distant tokens
    iid_noise: float = 0.1      # iid token noise on Q and K (relative)
    sink_logit: float = 6.0     # logit bonus of key 0
    hot_blocks: int = 4         # strongly attended key blocks per KV head
    hot_logit: float = 4.0      # logit bonus of keys in hot blocks
    temp_spread: float = 1.5    # per-head query temperature spread
    hetero: bool = False        # alternate flat / sharp heads in every group


@dataclass(frozen=True)
class Workload:
    """One attention layer's shape, the method's hyper-parameters and inputs."""

    name: str
    seq_len: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    num_proxy_groups: int
    stride: int = 4
    dtype: str = "bf16"         # "bf16" or "fp32"
    gamma: float = 0.95
    min_budget_tokens: int = 0
    seed: int = 0
    structure: Structure = Structure()

    def replace(self, **kw) -> "Workload":
        s_kw = {k: kw.pop(k) for k in list(kw) if k in Structure.__dataclass_fields__}
        wl = dataclasses.replace(self, **kw)
        if s_kw:
            wl = dataclasses.replace(wl, structure=dataclasses.replace(wl.structure, **s_kw))
        return wl

    @property
    def num_blocks(self) -> int:
        return -(-self.seq_len // self.block_size)


# Named workloads.  Shapes follow the layers of the models the paper uses
# (Llama-3.1-8B: 32 query / 8 KV heads, Qwen2.5-7B: 28 / 4, head dim 128),
# stride 4 as in the paper's main setting.
WORKLOADS = {
    # small fp32 GQA layer: parity at sizes the oracle finishes in seconds
    "gqa8x2_n2048_fp32": Workload(
        name="gqa8x2_n2048_fp32", seq_len=2048, num_q_heads=8, num_kv_heads=2,
        head_dim=64, block_size=64, num_proxy_groups=2, stride=4, dtype="fp32",
        gamma=0.9, seed=0, structure=Structure(rank=8, noise=0.3, hot_blocks=0)),
    # Llama-3-8B-shaped layer at 32K
    "llama3_8b_n32768": Workload(
        name="llama3_8b_n32768", seq_len=32768, num_q_heads=32, num_kv_heads=8,
        head_dim=128, block_size=128, num_proxy_groups=4, stride=4, dtype="bf16",
        gamma=0.95, seed=0, structure=Structure(rank=16, noise=0.3)),
    # Llama-3-8B-shaped layer at 128K (the timed workload)
    "llama3_8b_n131072": Workload(
        name="llama3_8b_n131072", seq_len=131072, num_q_heads=32, num_kv_heads=8,
        head_dim=128, block_size=128, num_proxy_groups=4, stride=4, dtype="bf16",
        gamma=0.95, seed=0, structure=Structure(rank=16, noise=0.3)),
    # Qwen2.5-7B-shaped layer at 64K with heterogeneous heads
    "qwen25_7b_n65536": Workload(
        name="qwen25_7b_n65536", seq_len=65536, num_q_heads=28, num_kv_heads=4,
        head_dim=128, block_size=128, num_proxy_groups=2, stride=4, dtype="bf16",
        gamma=0.95, seed=0, structure=Structure(rank=16, noise=0.3, hetero=True)),
    # one layer of a 32-layer Llama-3-8B-shaped stack at 256K (layer l: seed l)
    "llama3_8b_n262144": Workload(
        name="llama3_8b_n262144", seq_len=262144, num_q_heads=32, num_kv_heads=8,
        head_dim=128, block_size=128, num_proxy_groups=4, stride=4, dtype="bf16",
        gamma=0.95, seed=0, structure=Structure(rank=16, noise=0.3)),
}


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even), kept as fp32.

    Works in place on a float32 C-contiguous input."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    flat = b.reshape(-1)
    step = 1 << 22
    tmp = np.empty(min(step, flat.size), dtype=np.uint32)
    for s0 in range(0, flat.size, step):
        seg = flat[s0:s0 + step]
        t = tmp[:seg.size]
        np.right_shift(seg, 16, out=t)
        np.bitwise_and(t, 1, out=t)
        t += np.uint32(0x7FFF)
        seg += t
        seg &= np.uint32(0xFFFF0000)
    return x


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are exactly bf16 (as uint16)."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (b >> 16).astype(np.uint16)


def _ar1(rng: np.random.Generator, n: int, rank: int, corr_len: float) -> np.ndarray:
    """Unit-variance Gaussian AR(1) process, shape (n, rank), along axis 0."""
    rho = math.exp(-1.0 / max(corr_len, 1e-6))
    xi = rng.standard_normal((n, rank), dtype=np.float32)
    z0 = rng.standard_normal((1, rank), dtype=np.float32)
    c = math.sqrt(max(1.0 - rho * rho, 0.0))
    z = lfilter([c], [1.0, -rho], xi, axis=0, zi=(rho * z0)).__getitem__(0)
    return z.astype(np.float32)


def _orthonormal_pair(rng: np.random.Generator, d: int):
    """Two random orthonormal directions and the projector onto their complement."""
    a = rng.standard_normal((d, 2))
    qm, _ = np.linalg.qr(a)
    e, f = qm[:, 0], qm[:, 1]
    proj = np.eye(d) - np.outer(e, e) - np.outer(f, f)
    return e.astype(np.float32), f.astype(np.float32), proj.astype(np.float32)


def head_temperatures(wl: Workload, rng: np.random.Generator) -> np.ndarray:
    st = wl.structure
    if st.hetero:
        return np.where(np.arange(wl.num_q_heads) % 2 == 0, 0.1, 2.0).astype(np.float32)
    lo, hi = -math.log(st.temp_spread), math.log(st.temp_spread)
    return np.exp(rng.uniform(lo, hi, wl.num_q_heads)).astype(np.float32)


def generate(wl: Workload, with_v: bool = True) -> dict:
    """Draw Q [N,Hq,d], K [N,Hkv,d], V [N,Hkv,d] as fp32 arrays.

    For bf16 workloads every value is exactly representable in bf16.

    The sink and hot-block directions (e_h, f_h) are orthonormal and the
    content and noise of the group are projected onto their complement, so
    c*<q,k> gains exactly temp_i*sink_logit at key 0 and temp_i*hot_logit at
    keys of hot blocks, and nothing elsewhere.

    Draw order: head temperatures; then per KV head h: e_h/f_h, shared
    latent and basis, the KV head's deviation latent and basis, hot-block
    indices, then for each query head of the group its deviation latent and
    basis; then iid Q noise, iid K noise, then V.
    """
    st = wl.structure
    n, hq, hkv, d = wl.seq_len, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    r = hq // hkv
    rng = np.random.Generator(np.random.PCG64(wl.seed))
    temps = head_temperatures(wl, rng)

    sq1 = np.float32(math.sqrt(1.0 + st.noise ** 2))
    sig = np.float32(st.noise)
    # distant-token std of (1/sqrt d) <x_t, x_u> is about sqrt(d/rank) for a
    # rank-`rank` content of unit per-coordinate variance
    q_scale = st.content_logit * math.sqrt(st.rank / d)
    sqrt_d = np.float32(math.sqrt(d))
    q = np.empty((n, hq, d), dtype=np.float32)
    k = np.empty((n, hkv, d), dtype=np.float32)
    nk = wl.num_blocks
    projs = []

    def basis():
        return (rng.standard_normal((st.rank, d), dtype=np.float32)
                / np.float32(math.sqrt(st.rank)))

    for h in range(hkv):
        e, f, proj = _orthonormal_pair(rng, d)
        projs.append(proj)
        x = _ar1(rng, n, st.rank, st.corr_len) @ (basis() @ proj)
        dev = _ar1(rng, n, st.rank, st.corr_len) @ (basis() @ proj)
        kh = (x + sig * dev) / sq1
        if st.hot_blocks > 0 and nk > 1:
            hot = rng.choice(np.arange(1, nk), size=min(st.hot_blocks, nk - 1), replace=False)
        else:
            hot = np.zeros(0, dtype=np.int64)
        kh[0] += sqrt_d * e
        for blk in hot:
            lo_t, hi_t = int(blk) * wl.block_size, min((int(blk) + 1) * wl.block_size, n)
            kh[lo_t:hi_t] += sqrt_d * f
        k[:, h, :] = kh
        for j in range(r):
            i = h * r + j
            dq = _ar1(rng, n, st.rank, st.corr_len) @ (basis() @ proj)
            t_i = float(temps[i])
            sink_gain = 3.0 if (st.hetero and i % 2 == 1) else 1.0
            qi = (x + sig * dq) * np.float32(q_scale * t_i / float(sq1))
            qi += np.float32(t_i * sink_gain * st.sink_logit) * e
            if hot.size:
                qi += np.float32(t_i * st.hot_logit) * f
            q[:, i, :] = qi
    if st.iid_noise > 0:
        for h in range(hkv):
            pq = rng.standard_normal((n, r, d), dtype=np.float32) @ projs[h]
            q[:, h * r:(h + 1) * r, :] += (np.float32(st.iid_noise * q_scale)
                                           * temps[h * r:(h + 1) * r, None]) * pq
        for h in range(hkv):
            k[:, h, :] += np.float32(st.iid_noise) * (
                rng.standard_normal((n, d), dtype=np.float32) @ projs[h])
    v = rng.standard_normal((n, hkv, d), dtype=np.float32) if with_v else None
    if wl.dtype == "bf16":
        q, k = round_bf16(q), round_bf16(k)
        v = round_bf16(v) if v is not None else None
    out = {"q": q, "k": k, "temps": temps}
    if v is not None:
        out["v"] = v
    return out
