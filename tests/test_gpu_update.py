"""GPU parity of the fused delayed-update kernel (delayed_update_flat) against the oracle's
elementwise rule, including ragged lengths, bf16 gradients, EF on/off and the full 1e9-element
workload on sampled slices."""
import numpy as np
import pytest

import datagen
from gpu_common import log, rel
from oracle.update import HParams, flat_update

pytestmark = pytest.mark.gpu


def _hp(lam, clip=0.0):
    from paper_2606_30634_amd.stage import hparams
    return hparams(lr=1e-3, ef_lambda=lam, clip_norm=clip), HParams(lr=1e-3, ef_lambda=lam, clip_norm=clip)


@pytest.mark.parametrize("g_bf16", [False, True])
@pytest.mark.parametrize("lam", [0.0, 1.0, 0.5])
@pytest.mark.parametrize("shadow", ["bf16", "f32", None])
def test_flat_update_matches_oracle(g_bf16, lam, shadow):
    import torch
    from paper_2606_30634_amd import binding as B
    n = 1_000_003  # not a multiple of 4: exercises the ragged tail
    dev = torch.device("cuda:0")
    hpg, hpo = _hp(lam)
    x0 = datagen.normal(11, "x", n, 0.02)
    x = torch.from_numpy(x0).to(dev)
    m = torch.zeros(n, device=dev)
    v = torch.zeros(n, device=dev)
    up = torch.zeros(n, device=dev)
    sh = None if shadow is None else torch.zeros(n, device=dev, dtype=torch.bfloat16 if shadow == "bf16" else torch.float32)
    xo, mo, vo, uo = x0.astype(np.float64), np.zeros(n), np.zeros(n), np.zeros(n)
    stream = torch.cuda.current_stream().cuda_stream
    for t in range(6):
        gv = datagen.normal(11, "g", n, 1e-3, step=t)
        if g_bf16:
            gv = datagen.bf16_values(gv)
        gd = torch.from_numpy(gv).to(dev)
        if g_bf16:
            gd = gd.to(torch.bfloat16)
        B.delayed_update_flat(n, x.data_ptr(), gd.data_ptr(), g_bf16, m.data_ptr(), v.data_ptr(),
                              up.data_ptr(), None if sh is None else sh.data_ptr(), shadow == "bf16", t,
                              hpg, None, stream)
        xo, mo, vo, uo = flat_update(xo, gv.astype(np.float64), mo, vo, uo, t, hpo)
    torch.cuda.synchronize()
    xg = x.cpu().numpy()
    assert rel(xg, xo) < 1e-6, rel(xg, xo)
    assert rel(m.cpu().numpy(), mo) < 1e-5
    assert rel(v.cpu().numpy(), vo) < 1e-5
    if lam:
        assert rel(up.cpu().numpy(), uo) < 1e-5
    if shadow == "bf16":
        assert np.array_equal(sh.view(torch.int16).cpu().numpy().view(np.uint16), datagen.bf16_bits(xg))
    elif shadow == "f32":
        assert np.array_equal(sh.cpu().numpy(), xg)


def test_update_workload_1e9_sampled_slices():
    """The update-only workload: 1.0e9 fp32 elements, bf16 gradients, EF, 50 iterations; 16 random
    slices of 65536 elements re-derived by the oracle from the regenerated inputs."""
    import torch
    from paper_2606_30634_amd import binding as B
    n, seed, steps = datagen.UPDATE_N, datagen.UPDATE_SEED, datagen.UPDATE_STEPS
    dev = torch.device("cuda:0")
    log("update-1e9: generating inputs")
    x = torch.from_numpy(datagen.normal_flat(seed, "x", n, 0.02)).to(dev)
    g = torch.from_numpy(datagen.bf16_bits(datagen.normal_flat(seed, "g", n, 1e-3)).view(np.int16)).to(dev).view(torch.bfloat16)
    m = torch.zeros(n, device=dev)
    v = torch.zeros(n, device=dev)
    up = torch.zeros(n, device=dev)
    sh = torch.empty(n, device=dev, dtype=torch.bfloat16)
    hpg, hpo = _hp(1.0)
    stream = torch.cuda.current_stream().cuda_stream
    log("update-1e9: 50 iterations")
    for t in range(steps):
        B.delayed_update_flat(n, x.data_ptr(), g.data_ptr(), True, m.data_ptr(), v.data_ptr(), up.data_ptr(),
                              sh.data_ptr(), True, t, hpg, None, stream)
    torch.cuda.synchronize()
    rng = np.random.default_rng(123)
    cnt = 65536
    worst = 0.0
    for s in rng.integers(0, n - cnt, size=16):
        s = int(s)
        xo = datagen.normal_flat_slice(seed, "x", n, s, cnt, 0.02).astype(np.float64)
        gv = datagen.bf16_values(datagen.normal_flat_slice(seed, "g", n, s, cnt, 1e-3)).astype(np.float64)
        mo, vo, uo = np.zeros(cnt), np.zeros(cnt), np.zeros(cnt)
        for t in range(steps):
            xo, mo, vo, uo = flat_update(xo, gv, mo, vo, uo, t, hpo)
        xg = x[s:s + cnt].cpu().numpy()
        e = max(rel(xg, xo), rel(m[s:s + cnt].cpu().numpy(), mo), rel(v[s:s + cnt].cpu().numpy(), vo),
                rel(up[s:s + cnt].cpu().numpy(), uo))
        worst = max(worst, e)
        assert np.array_equal(sh[s:s + cnt].view(torch.int16).cpu().numpy().view(np.uint16), datagen.bf16_bits(xg))
    log(f"update-1e9: worst sampled rel err {worst:.3e}")
    assert worst < 1e-5
