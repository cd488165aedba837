"""The seeded input generator: determinism, shapes, exact bf16 values, and
that its structure knobs move what they are meant to move."""
import math

import numpy as np

from paper_2509_24745_amd.synth import WORKLOADS, Workload, Structure, generate, round_bf16


def _small(**kw):
    base = Workload(name="t", seq_len=1024, num_q_heads=8, num_kv_heads=2, head_dim=64,
                    block_size=64, num_proxy_groups=2, stride=4, dtype="bf16", seed=3,
                    structure=Structure(rank=8))
    return base.replace(**kw)


def test_deterministic_per_seed_and_shapes():
    wl = _small()
    a, b = generate(wl), generate(wl)
    for key in ("q", "k", "v"):
        assert np.array_equal(a[key], b[key])
    c = generate(wl.replace(seed=4))
    assert not np.array_equal(a["q"], c["q"])
    assert a["q"].shape == (1024, 8, 64) and a["k"].shape == (1024, 2, 64)
    assert a["v"].shape == (1024, 2, 64) and a["q"].dtype == np.float32


def test_bf16_workloads_hold_exact_bf16_values():
    g = generate(_small())
    for key in ("q", "k", "v"):
        assert np.all(g[key].view(np.uint32) & 0xFFFF == 0)
    f = generate(_small(dtype="fp32"))
    assert np.any(f["q"].view(np.uint32) & 0xFFFF != 0)


def test_round_bf16_in_place_variant_matches_formula():
    x = np.random.default_rng(0).standard_normal(10000).astype(np.float32)
    b = x.copy().view(np.uint32)
    want = ((b + ((b >> 16) & 1) + 0x7FFF) & 0xFFFF0000).view(np.float32)
    assert np.array_equal(round_bf16(x.copy()), want)


def test_sink_bonus_is_exact():
    # sink/hot directions are orthogonal to content: c*<q_t, k_0> - c*<q_t, k_0 without sink>
    wl = _small(dtype="fp32", hot_blocks=0, iid_noise=0.0)
    g = generate(wl)
    q, k = g["q"].astype(np.float64), g["k"].astype(np.float64)
    g0 = generate(wl.replace(sink_logit=0.0))
    q0, k0 = g0["q"].astype(np.float64), g0["k"].astype(np.float64)
    c = 1 / math.sqrt(64)
    bonus = c * np.einsum("td,d->t", q[:, 0], k[0, 0]) - c * np.einsum("td,d->t", q0[:, 0], k0[0, 0])
    assert np.allclose(bonus, g["temps"][0] * wl.structure.sink_logit, rtol=1e-4, atol=1e-3)


def test_noise_knob_lowers_head_similarity():
    # correlation of two query heads of one group falls as sigma grows
    def corr(sig):
        g = generate(_small(dtype="fp32", noise=sig, iid_noise=0.0, sink_logit=0.0,
                            hot_blocks=0))
        a, b = g["q"][:, 0].ravel(), g["q"][:, 1].ravel()
        return np.corrcoef(a, b)[0, 1]
    c1, c3, c6 = corr(0.1), corr(0.3), corr(0.6)
    assert c1 > c3 > c6


def test_named_workloads_are_consistent():
    for wl in WORKLOADS.values():
        assert wl.num_q_heads % wl.num_kv_heads == 0
        assert wl.num_q_heads % wl.num_proxy_groups == 0
        assert wl.block_size % wl.stride == 0


def test_head_similarity_follows_the_deviation_knob():
    """Eq. 4 overlap on the generator's heads: the mean overlap between
    different heads falls as the per-head deviation sigma grows, with and
    without the sink tokens (renormalised), the premise of proxy heads."""
    from oracle import proxyattn_oracle as O
    base = WORKLOADS["llama3_8b_n32768"].replace(seq_len=8192)
    means = []
    for sigma in (0.1, 0.3, 0.6):
        wl = base.replace(noise=sigma)
        g = generate(wl, with_v=False)
        row = []
        for sink, renorm in ((0, False), (4, True)):
            s = O.head_overlap(g["q"], g["k"], wl.seq_len - 1, 1024, O.default_scale(wl.head_dim),
                               sink_tokens=sink, renormalize=renorm).astype(np.float64)
            off = s[~np.eye(s.shape[0], dtype=bool)]
            row.append(off.mean())
        means.append(row)
    means = np.array(means)
    assert np.all(np.diff(means, axis=0) < 0), means
    assert means[0, 0] > 0.5, means
