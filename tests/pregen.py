"""Background preparation of the 256K stack layers for the GPU tests, and the
oracle's sampled-row attention on them split over head groups.

Drawing a 256K layer and running the oracle's estimation stages on it take
about a minute each on the host; the GPU tests of five layers would spend
most of their time waiting for them.  When those tests are selected, the
test session starts one spawned process per layer before anything touches
the GPU (see conftest.py).  Each process draws its layer and computes what
the oracle fixes before the GPU runs: the pooled proxy heads, the block
scores of the sampled query rows' block rows and every head's last-block
mass.  Arrays travel through .npy files.  These processes import numpy, the
input generator and the oracle only; the attention of the sampled rows, which
needs the GPU's lists, runs after the GPU in the same processes, one job per
group of heads (the oracle computes each head alone, so a group of query
heads with its KV heads is a smaller problem of the same kind).
"""
from __future__ import annotations

import os
import shutil
import tempfile

import numpy as np

WORKLOAD = "llama3_8b_n262144"
SAMPLE_SEED = 12345


def sample_rows(n: int, per_head: int) -> np.ndarray:
    rng = np.random.default_rng(SAMPLE_SEED)
    return np.unique(np.concatenate([rng.integers(0, n, per_head), [n - 1]]))


def layer_job(job):
    """Spawned worker: draw layer `seed`, run the oracle's estimation stages,
    store everything under `outdir`; returns {name: path}."""
    wname, seed, per_head, outdir, threads = job
    from threadpoolctl import threadpool_limits
    from oracle import proxyattn_oracle as O
    from paper_2509_24745_amd.synth import WORKLOADS, generate, to_bf16_bits
    wl = WORKLOADS[wname].replace(seed=seed)
    paths = {}

    def put(name, arr):
        path = os.path.join(outdir, f"layer{seed}_{name}.npy")
        np.save(path, arr)
        paths[name] = path

    with threadpool_limits(threads):
        g = generate(wl)
        q, k = g["q"], g["k"]
        for x in ("q", "k", "v"):
            put(x, to_bf16_bits(g[x]))
        del g
        sc = O.default_scale(wl.head_dim)
        rows = sample_rows(wl.seq_len, per_head)
        brows = np.unique(rows // wl.block_size)
        qg, kg = O.pool_proxy_heads(q, k, wl.num_proxy_groups, wl.stride, wl.dtype)
        put("qg", qg)
        put("kg", kg)
        oa, _ = O.proxy_block_logscore(qg, kg, wl.seq_len, wl.block_size, wl.stride, sc,
                                       rows=brows)
        put("logA", oa)
        put("mass", O.lastblock_mass(q, k, wl.block_size, sc))
    return paths


def attn_job(job):
    """Spawned worker: the oracle's block-sparse attention of `rows` for query
    heads [h0, h1) of layer `seed` (whose inputs `layer_job` stored), on the
    given lists of those heads (block rows `brows` only)."""
    wname, seed, outdir, h0, h1, rows, brows, bc_rows, bi_rows, threads = job
    from threadpoolctl import threadpool_limits
    from oracle import proxyattn_oracle as O
    from paper_2509_24745_amd.synth import WORKLOADS
    wl = WORKLOADS[wname].replace(seed=seed)
    rep = wl.num_q_heads // wl.num_kv_heads
    assert h0 % rep == 0 and h1 % rep == 0

    def load(x):
        a = np.load(os.path.join(outdir, f"layer{seed}_{x}.npy"), mmap_mode="r")
        return a

    q = load("q")[:, h0:h1]
    k = load("k")[:, h0 // rep:h1 // rep]
    v = load("v")[:, h0 // rep:h1 // rep]
    widen = lambda a: (np.asarray(a).astype(np.uint32) << 16).view(np.float32)
    q, k, v = widen(q), widen(k), widen(v)
    mq = wl.num_blocks
    bc = np.zeros((h1 - h0, mq), np.int32)
    bi = np.full((h1 - h0, mq, mq), -1, np.int32)
    bc[:, brows] = bc_rows
    bi[:, brows] = bi_rows
    with threadpool_limits(threads):
        out, lse = O.block_sparse_attention(q, k, v, bc, bi, wl.block_size,
                                            O.default_scale(wl.head_dim), query_rows=rows)
    return out[rows], lse[:, rows]


class Pregen:
    def __init__(self, seeds, per_head: int, wname: str = WORKLOAD):
        import multiprocessing as mp
        self.per_head = per_head
        root = "/dev/shm" if os.path.isdir("/dev/shm") else None
        if root:
            st = os.statvfs(root)
            if st.f_bavail * st.f_frsize < len(seeds) * 3 * 2**30:
                root = None
        self.dir = tempfile.mkdtemp(prefix="proxyattn_layers_", dir=root)
        self.wname = wname
        workers = max(1, len(seeds))
        self.workers = workers
        threads = max(1, min(16, os.cpu_count() or 1) // workers)
        self.threads = threads
        self.pool = mp.get_context("spawn").Pool(workers)
        self.pending = {s: self.pool.apply_async(layer_job,
                                                 ((wname, s, per_head, self.dir, threads),))
                        for s in seeds}

    def get(self, seed: int, timeout: float = 900.0) -> dict:
        """The layer's arrays (inputs as fp32 with bf16 values).  The input
        files stay until release(seed), for attention()."""
        paths = self.pending.pop(seed).get(timeout)
        out = {}
        for name, path in paths.items():
            a = np.load(path)
            if name in ("q", "k", "v"):        # bf16 bits -> the same values in fp32
                a = (a.astype(np.uint32) << 16).view(np.float32)
            else:
                os.remove(path)
            out[name] = a
        return out

    def attention(self, seed: int, block_size: int, num_q_heads: int, num_kv_heads: int, rows,
                  bc, bi, timeout: float = 900.0):
        """The oracle's attention of `rows` on lists (bc [Hq, Mq], bi [Hq, Mq, Nk]),
        computed by the worker processes in groups of whole KV heads; returns
        (out [len(rows), Hq, d], lse [Hq, len(rows)])."""
        rep = num_q_heads // num_kv_heads
        rows = np.asarray(rows)
        brows = np.unique(rows // block_size)
        groups = max(1, min(self.workers, num_kv_heads))
        while num_kv_heads % groups:
            groups -= 1
        per = num_q_heads // groups
        threads = max(1, min(16, os.cpu_count() or 1) // groups)
        jobs = []
        for j in range(groups):
            h0, h1 = j * per, (j + 1) * per
            assert h0 % rep == 0
            jobs.append(self.pool.apply_async(attn_job, ((
                self.wname, seed, self.dir, h0, h1, rows, brows,
                np.ascontiguousarray(bc[h0:h1][:, brows]),
                np.ascontiguousarray(bi[h0:h1][:, brows]), threads),)))
        parts = [jb.get(timeout) for jb in jobs]
        out = np.concatenate([p[0] for p in parts], axis=1)
        lse = np.concatenate([p[1] for p in parts], axis=0)
        return out, lse

    def release(self, seed: int):
        for x in ("q", "k", "v"):
            try:
                os.remove(os.path.join(self.dir, f"layer{seed}_{x}.npy"))
            except OSError:
                pass

    def close(self):
        self.pool.terminate()
        self.pool.join()
        shutil.rmtree(self.dir, ignore_errors=True)


_ACTIVE: Pregen | None = None


def start(seeds, per_head: int):
    global _ACTIVE
    _ACTIVE = Pregen(seeds, per_head)


def active() -> Pregen | None:
    return _ACTIVE


def stop():
    global _ACTIVE
    if _ACTIVE is not None:
        _ACTIVE.close()
        _ACTIVE = None
