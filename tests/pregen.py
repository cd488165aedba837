"""Background preparation of the 256K stack layers for the GPU tests.

Drawing a 256K layer and running the oracle's estimation stages on it take
about a minute each on the host; the GPU tests of five layers would spend
most of their time waiting for them.  When those tests are selected, the
test session starts one spawned process per layer before anything touches
the GPU (see conftest.py).  Each process draws its layer and computes what
the oracle fixes before the GPU runs: the pooled proxy heads, the block
scores of the sampled query rows' block rows and every head's last-block
mass.  Arrays travel through .npy files.  These processes import numpy, the
input generator and the oracle only; the attention of the sampled rows, which
needs the GPU's lists, stays in the test.
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
        workers = max(1, len(seeds))
        threads = max(1, min(16, os.cpu_count() or 1) // workers)
        self.pool = mp.get_context("spawn").Pool(workers)
        self.pending = {s: self.pool.apply_async(layer_job,
                                                 ((wname, s, per_head, self.dir, threads),))
                        for s in seeds}

    def get(self, seed: int, timeout: float = 900.0) -> dict:
        """The layer's arrays (inputs as fp32 with bf16 values)."""
        paths = self.pending.pop(seed).get(timeout)
        out = {}
        for name, path in paths.items():
            a = np.load(path)
            if name in ("q", "k", "v"):        # bf16 bits -> the same values in fp32
                a = (a.astype(np.uint32) << 16).view(np.float32)
            out[name] = a
            os.remove(path)
        return out

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
