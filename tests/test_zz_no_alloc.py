"""The no-alloc variant of the flat gradient norm (grad_norm_flat_noalloc: partial sums in the
library's static per-GPU array) against the workspace entry point (grad_norm_flat), through the C
ABI: two calls in a row, the second on a smaller input, bit for bit (the same kernels, grid and
summation order); the non-finite flag; both against the float64 norm at 1e-6."""
import numpy as np
import pytest

import datagen

pytestmark = pytest.mark.gpu


def _run_pair(B, torch, g, bf16, clip, stream):
    dev = g.device
    n = g.numel()
    ws_bytes = B.grad_norm_flat_workspace_bytes()
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    out_ws = torch.full((2,), -1.0, device=dev)
    out_na = torch.full((2,), -2.0, device=dev)
    fl_ws = torch.full((1,), 7, dtype=torch.int32, device=dev)
    fl_na = torch.full((1,), 9, dtype=torch.int32, device=dev)
    B.grad_norm_flat(n, g.data_ptr(), bf16, clip, out_ws.data_ptr(), fl_ws.data_ptr(), ws.data_ptr(), ws_bytes, stream)
    B.grad_norm_flat_noalloc(n, g.data_ptr(), bf16, clip, out_na.data_ptr(), fl_na.data_ptr(), stream)
    torch.cuda.synchronize()
    return out_ws.cpu().numpy(), out_na.cpu().numpy(), int(fl_ws.item()), int(fl_na.item())


@pytest.mark.parametrize("bf16", [False, True])
def test_noalloc_norm_matches_workspace_entry_point(bf16):
    import torch
    from paper_2606_30634_amd import binding as B
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    dt = torch.bfloat16 if bf16 else torch.float32
    for n, clip in ((5_000_011, 1.0), (70_003, 0.0)):      # the second call smaller, clipping off
        g = torch.from_numpy(datagen.normal(31, "g", n, 1e-3)).to(dev).to(dt)
        ref = float(np.linalg.norm(g.float().cpu().numpy().astype(np.float64)))
        ws, na, f_ws, f_na = _run_pair(B, torch, g, bf16, clip, stream)
        print(f"n={n} bf16={bf16}: workspace {ws}, noalloc {na}, float64 {ref:.9g}", flush=True)
        assert np.array_equal(ws, na), (ws, na)
        assert f_ws == 0 and f_na == 0
        assert abs(float(na[0]) - ref) <= 1e-6 * ref
        c = min(1.0, clip / (ref + 1e-6)) if clip > 0 else 1.0
        assert abs(float(na[1]) - c) <= 1e-6 * c
    # a non-finite element sets the flag and leaves the clip coefficient at 1
    g = torch.from_numpy(datagen.normal(31, "g", 9_001, 1e-3)).to(dev).to(dt)
    g[4321] = float("inf")
    ws, na, f_ws, f_na = _run_pair(B, torch, g, bf16, 1.0, stream)
    assert f_ws == 1 and f_na == 1 and na[1] == 1.0 and not np.isfinite(na[0])
