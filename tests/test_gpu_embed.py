"""Bit-exact checks of the token gather and of the embedding-gradient indices, and of the bf16
compute copy of the weights."""
import numpy as np
import pytest

import datagen
from gpu_common import log, shape_of, to_device

pytestmark = pytest.mark.gpu


REDUCED = dict(n_blocks=1, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ffn=512, vocab=1000)


@pytest.mark.parametrize("wname", ["small-reduced", "ragged", "16384-tokens", "32768-tokens", "few-ids", "small"])
def test_gather_and_indices_bit_exact(wname):
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = {
        "small": datagen.SMALL.with_(n_blocks=1),  # the gather and indices do not depend on depth
        "small-reduced": datagen.SMALL.with_(seq_len=96, micro_batch=2, **REDUCED),
        "ragged": datagen.SMALL.with_(seq_len=93, micro_batch=3, **REDUCED),  # 279 positions
        # several 1024-key chunks of the radix sort, and twice the 16384 positions of the former rank sort
        "16384-tokens": datagen.SMALL.with_(seq_len=2048, micro_batch=8, **dict(REDUCED, vocab=32000)),
        "32768-tokens": datagen.SMALL.with_(seq_len=4096, micro_batch=8, **dict(REDUCED, vocab=32000)),
        # 50 ids over 16384 positions: long runs of equal keys across chunks (the sort's stability)
        "few-ids": datagen.SMALL.with_(seq_len=2048, micro_batch=8, **dict(REDUCED, vocab=50)),
    }[wname]
    log(f"gather/indices {wname}")
    dev = torch.device("cuda:0")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inp = datagen.step_inputs(w, 0)
    d = to_device(inp, w, dev)
    st.forward(0, 0, tokens=d["tokens"], y_out=torch.empty_like(d["dy"]))
    st.backward(0, dy=d["dy"])
    torch.cuda.synchronize()
    E_bits = datagen.bf16_bits(p0["embed"]).reshape(w.vocab, w.d_model)
    w0 = st.view("w0.embed").view(torch.int16).cpu().numpy().view(np.uint16).reshape(w.vocab, w.d_model)
    assert np.array_equal(w0, E_bits)
    x0 = st.view("act0.x0").view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1, w.d_model)
    assert np.array_equal(x0, E_bits[inp["tokens"].reshape(-1)])
    ids, counts = st.embed_indices(0)
    ref_ids, ref_counts = np.unique(inp["tokens"].reshape(-1), return_counts=True)
    assert np.array_equal(ids, ref_ids) and np.array_equal(counts, ref_counts)
    # rows of tokens that did not occur have an exactly zero gradient
    g = st.view("grad0.embed").cpu().numpy().reshape(w.vocab, w.d_model)
    absent = np.setdiff1d(np.arange(w.vocab), ref_ids)
    assert np.all(g[absent] == 0.0)
    assert np.all(np.any(g[ref_ids] != 0.0, axis=1))
    st.close()


def test_invalid_token_ids_are_not_read():
    """Token ids outside [0, vocab) embed as zero rows and reach no embedding-gradient row, also
    ids whose key would alias a valid token under a plain 32-bit shift (2^18 + 5 -> 5)."""
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = datagen.SMALL.with_(n_blocks=1, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ffn=512,
                            vocab=1000, seq_len=96, micro_batch=2)
    log("invalid token ids")
    dev = torch.device("cuda:0")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inp = datagen.step_inputs(w, 0)
    tok = inp["tokens"].copy()
    tok[tok == 5] = 6
    bad = [(0, 3, -1), (0, 50, w.vocab), (1, 7, (1 << 18) + 5), (1, 95, 2**31 - 1), (1, 0, -(2**31))]
    for b, p, v in bad:
        tok[b, p] = v
    inp["tokens"] = tok
    d = to_device(inp, w, dev)
    st.forward(0, 0, tokens=d["tokens"], y_out=torch.empty_like(d["dy"]))
    st.backward(0, dy=d["dy"])
    torch.cuda.synchronize()
    flat = tok.reshape(-1)
    valid = (flat >= 0) & (flat < w.vocab)
    E_bits = datagen.bf16_bits(p0["embed"]).reshape(w.vocab, w.d_model)
    x0 = st.view("act0.x0").view(torch.int16).cpu().numpy().view(np.uint16).reshape(-1, w.d_model)
    assert np.array_equal(x0[valid], E_bits[flat[valid]])
    assert np.all(x0[~valid] == 0)
    ids, counts = st.embed_indices(0)
    ref_ids, ref_counts = np.unique(flat[valid], return_counts=True)
    assert np.array_equal(ids, ref_ids) and np.array_equal(counts, ref_counts)
    g = st.view("grad0.embed").cpu().numpy().reshape(w.vocab, w.d_model)
    assert np.all(g[5] == 0.0)
    absent = np.setdiff1d(np.arange(w.vocab), ref_ids)
    assert np.all(g[absent] == 0.0)
    st.close()


def test_invalid_targets_are_ignored():
    """A target outside [0, vocab) adds zero loss; the mean still divides by every position.  The
    expected loss is the cross-entropy of the oracle's fp64 logits over the valid positions."""
    import torch
    import oracle
    from paper_2606_30634_amd.stage import Stage
    w = datagen.TINY.with_(n_blocks=1)
    log("invalid targets")
    dev = torch.device("cuda:0")
    st = Stage(shape_of(w), "cuda:0")
    p0 = datagen.init_params(w)
    st.load_master(p0)
    inp = datagen.step_inputs(w, 0)
    tg = inp["targets"].copy()
    bad = [(0, 3, -1), (1, 10, w.vocab), (1, 63, (1 << 20) + 2)]
    for b, p, v in bad:
        tg[b, p] = v
    flat = tg.reshape(-1)
    valid = (flat >= 0) & (flat < w.vocab)
    safe = dict(inp)
    safe["targets"] = np.where(valid.reshape(tg.shape), tg, 0).astype(np.int32)
    out, _ = oracle.model.stage_forward(p0, safe, w)
    logits = out["logits"].reshape(-1, w.vocab)
    mx = logits.max(axis=1, keepdims=True)
    lse = (mx + np.log(np.exp(logits - mx).sum(axis=1, keepdims=True)))[:, 0]
    rows = lse - logits[np.arange(len(flat)), np.where(valid, flat, 0)]
    expect = float(np.sum(rows[valid]) / len(flat))
    inp["targets"] = tg
    d = to_device(inp, w, dev)
    loss = torch.zeros(1, device=dev)
    st.forward(0, 0, tokens=d["tokens"], targets=d["targets"], loss=loss)
    st.backward(0)
    torch.cuda.synchronize()
    got = float(loss.item())
    log(f"  loss {got:.8f} expected {expect:.8f}")
    assert abs(got - expect) <= 1e-5 * abs(expect)
    assert bool(torch.isfinite(st.view("grad0.embed")).all())
    st.close()
