"""Error paths of the C ABI on a live stage: call order (STAGE_ESTATE), arena size
(STAGE_ENOSPACE), bad arguments (STAGE_EINVAL)."""
import numpy as np
import pytest

import datagen
from gpu_common import shape_of, to_device

pytestmark = pytest.mark.gpu

W = datagen.MID.with_(n_blocks=1, d_model=128, n_heads=2, n_kv_heads=2, head_dim=64, d_ffn=256,
                      seq_len=64, micro_batch=1, max_inflight=2)


def test_call_order_errors():
    import torch
    from paper_2606_30634_amd import binding as B
    from paper_2606_30634_amd.stage import Stage, hparams
    dev = torch.device("cuda:0")
    st = Stage(shape_of(W), "cuda:0")
    st.load_master(datagen.init_params(W))
    d = to_device(datagen.step_inputs(W, 0), W, dev)
    hp = hparams()
    with pytest.raises(B.StageError) as e:
        st.backward(0, dy=d["dy"])                       # no forward yet
    assert e.value.code == B.STAGE_ESTATE
    with pytest.raises(B.StageError) as e:
        st.forward(0, 1, x_in=d["x_in"])                 # weights of step 1 not resident
    assert e.value.code == B.STAGE_ESTATE
    with pytest.raises(B.StageError) as e:
        st.update(1, hp)                                 # t must start at 0
    assert e.value.code == B.STAGE_ESTATE
    st.forward(0, 0, x_in=d["x_in"])
    with pytest.raises(B.StageError) as e:
        st.forward(0, 0, x_in=d["x_in"])                 # slot busy
    assert e.value.code == B.STAGE_ESTATE
    st.backward(0, dy=d["dy"])
    st.update(0, hp)                                     # t = 0: no gradient consumed yet
    st.forward(1, 1, x_in=d["x_in"])
    with pytest.raises(B.StageError) as e:
        st.update(1, hparams(delay=0, ef_lambda=0.0))    # delay 0 needs g_1: its backward is pending
    assert e.value.code == B.STAGE_ESTATE
    st.backward(1, dy=d["dy"])
    st.update(1, hp)                                     # consumes g_0
    st.update(2, hp)                                     # consumes g_1
    with pytest.raises(B.StageError) as e:
        st.update(3, hp)                                 # g_2 was never computed
    assert e.value.code == B.STAGE_ESTATE
    with pytest.raises(B.StageError) as e:
        st.set_update_overlap(3)                         # modes 0, 1, 2
    assert e.value.code == B.STAGE_EINVAL
    torch.cuda.synchronize()
    st.close()


def test_arena_and_argument_errors():
    import torch
    from paper_2606_30634_amd import binding as B
    sh = shape_of(W)
    need = B.stage_required_bytes(sh)
    buf = torch.empty(need, dtype=torch.uint8, device="cuda:0")
    with pytest.raises(B.StageError) as e:
        B.stage_init(sh, buf.data_ptr(), need - 256, torch.cuda.current_stream().cuda_stream)
    assert e.value.code == B.STAGE_ENOSPACE
    with pytest.raises(B.StageError) as e:
        B.stage_init(sh, buf.data_ptr() + 16, need, torch.cuda.current_stream().cuda_stream)
    assert e.value.code == B.STAGE_EINVAL
