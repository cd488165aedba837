"""GPU parity of the decoder prefill around the path (bench.DecoderPrefill):
every layer's attention runs on the inputs its own projections produced
(structured inputs plus the scaled, rotated projections of the previous
layer's hidden state), so each layer is checked against the oracle on the
Q, K and V that layer actually fed to the path.  Bars as in
test_gpu_parity.py."""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import check as C
from oracle import proxyattn_oracle as O
from paper_2509_24745_amd.synth import WORKLOADS
from tests.test_gpu_parity import LSE_TOL, _compare, _gpu, _oracle, check_sampled_rows

pytestmark = pytest.mark.gpu

LLAMA = WORKLOADS["llama3_8b_n32768"]


def _capture(U, dec, rows=None):
    """A layer hook that fetches the layer's attention inputs and results;
    with `rows`, only those query rows of out and lse."""
    got = {}

    def hook(l):
        torch.cuda.synchronize()
        b = dec.bufs
        res = {x: U.to_host(getattr(dec, x)) for x in ("q", "k", "v")}
        res["qg"], res["kg"] = U.pooled_from_workspace(dec.prob, b.workspace)
        res.update(logA=U.to_host(b.logscore), mass=U.to_host(b.mass),
                   counts=U.to_host(b.head_count), block_count=U.to_host(b.block_count),
                   block_index=U.to_host(b.block_index))
        if rows is None:
            res.update(out=U.to_host(b.out), lse=U.to_host(b.lse))
        else:
            r = torch.from_numpy(np.asarray(rows, dtype=np.int64)).cuda()
            res.update(out=U.to_host(b.out[r]), lse=U.to_host(b.lse[:, r]))
        got[l] = res

    return got, hook


def test_decoder_layers_match_oracle():
    """Three layers at a ragged length (4173 tokens, Llama-shaped heads, a
    narrow hidden size): with the sparse path, every stage of every layer
    against the oracle on that layer's composed inputs; with the dense
    kernel, every layer's attention against the oracle's causal attention.
    The two prefills start from the same hidden state and differ after the
    first layer."""
    U = _gpu()
    from bench import DecoderPrefill
    wl = LLAMA.replace(seq_len=4173)
    prob = U.problem_of(wl)
    layers = 3
    host = [U.inputs(wl.replace(seed=l)) for l in range(layers)]
    structured = [tuple(U.to_dev(a, prob) for a in h) for h in host]
    dec = DecoderPrefill(wl, structured, hidden=1024, inter=2048)
    x0 = dec.embed()
    got, hook = _capture(U, dec)
    xs, _ = dec.forward(x0, dense=False, hook=hook)
    for l in range(layers):
        g = got[l]
        # the projections reach the attention: its inputs are not the structure alone
        assert not np.array_equal(g["q"], host[l][0])
        assert not np.array_equal(g["k"], host[l][1])
        assert not np.array_equal(g["v"], host[l][2])
        print(f"\n[decoder layer {l}, sparse path]", flush=True)
        _compare(wl, g["q"], g["k"], g["v"], g, _oracle(wl, g["q"], g["k"]))
    gotd, hookd = _capture(U, dec)
    xd, _ = dec.forward(x0, dense=True, hook=hookd)
    fbc, fbi = O.full_causal_lists(wl.seq_len, wl.num_q_heads, wl.block_size)
    sc = O.default_scale(wl.head_dim)
    for l in range(layers):
        g = gotd[l]
        ref, ref_lse = O.block_sparse_attention(g["q"], g["k"], g["v"], fbc, fbi, wl.block_size,
                                                sc)
        rep = C.check_attention(g["out"], ref)
        dl = float(np.abs(g["lse"] - ref_lse).max())
        assert dl <= LSE_TOL, f"layer {l}: max |dlse| = {dl}"
        print(f"[decoder layer {l}, dense] max|dO|={rep.max_abs:.2e} mean|dO|={rep.mean_abs:.2e} "
              f"|dlse|={dl:.2e}", flush=True)
    assert np.array_equal(gotd[0]["q"], got[0]["q"])          # same first-layer inputs
    assert not np.array_equal(gotd[1]["q"], got[1]["q"])      # then the attention differs
    torch.cuda.synchronize()
    assert torch.isfinite(xs.float()).all() and torch.isfinite(xd.float()).all()


def test_decoder_128k_second_layer_sampled_rows():
    """The benchmark's decoder at the 128K Llama-3-8B shape (hidden 4096,
    intermediate 14336), two layers sharing one structured draw: the second
    layer, whose inputs carry the first layer's attention output through the
    output projection, MLP and next projections, checked on 256 sampled query
    rows (pooled heads, every head's mass and budget, the scores and lists of
    their block rows, their attention)."""
    U = _gpu()
    from bench import DecoderPrefill
    from tests import pregen
    wl = WORKLOADS["llama3_8b_n131072"]
    prob = U.problem_of(wl)
    s = tuple(U.to_dev(a, prob) for a in U.inputs(wl))
    dec = DecoderPrefill(wl, [s, s])
    rows = pregen.sample_rows(wl.seq_len, 256)
    got, hook = _capture(U, dec, rows)

    def only_second(l):
        if l == 1:
            hook(l)

    dec.forward(dec.embed(), dense=False, hook=only_second)
    g = got[1]
    print("\n[128K decoder, layer 1]", flush=True)
    check_sampled_rows(wl, rows, g["q"], g["k"], g["v"], g)
