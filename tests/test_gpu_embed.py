"""Bit-exact checks of the token gather and of the embedding-gradient indices, and of the bf16
compute copy of the weights."""
import numpy as np
import pytest

import datagen
from gpu_common import log, shape_of, to_device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("wname", ["small-reduced", "small"])
def test_gather_and_indices_bit_exact(wname):
    import torch
    from paper_2606_30634_amd.stage import Stage
    w = datagen.SMALL if wname == "small" else datagen.SMALL.with_(
        n_blocks=1, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, d_ffn=512, vocab=1000,
        seq_len=96, micro_batch=2)
    if wname == "small":
        w = w.with_(n_blocks=1)  # the gather and indices do not depend on depth
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
