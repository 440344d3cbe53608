"""Thin PyTorch-memory wrapper over the C ABI: allocates the arena as a torch uint8 tensor on the
device, passes torch's current HIP stream, and exposes named arena regions as torch views.
No arithmetic happens here; every step runs in the library's kernels."""
from __future__ import annotations

import ctypes as C
from typing import Dict, Optional

import torch

from . import binding as B

_TORCH_DT = {B.DT_F32: torch.float32, B.DT_BF16: torch.bfloat16, B.DT_I32: torch.int32}
_ESZ = {B.DT_F32: 4, B.DT_BF16: 2, B.DT_I32: 4}


def make_shape(n_blocks, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab, first_stage,
               last_stage, tie_embedding, seq_len, micro_batch, max_inflight=1, bf16=True,
               rms_eps=1e-5, rope_theta=10000.0, muon=False, max_delay=1, adan=False) -> B.StageShape:
    if muon and adan:
        raise ValueError("a stage holds the Muon workspace or the Adan state, not both")
    return B.StageShape(n_blocks, d_model, n_heads, n_kv_heads, head_dim, d_ffn, vocab,
                        int(first_stage), int(last_stage), int(tie_embedding), seq_len, micro_batch,
                        max_inflight, 1 if bf16 else 0, rms_eps, rope_theta, 1 if muon else (2 if adan else 0),
                        max_delay)


def hparams(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, clip_norm=1.0,
            ef_lambda=1.0, delay=1, optimizer="adamw", momentum=0.95, update_rms=0.2,
            ns_steps=5, predict="none", nadam_psi=0.004, beta3=0.99) -> B.UpdateHParams:
    opt = {"adamw": 0, "muon": 1, "lion": 2, "nadam": 3, "adan": 4}[optimizer]
    pred = {"none": 0, "updated": 1}[predict]
    return B.UpdateHParams(lr, beta1, beta2, eps, weight_decay, clip_norm, ef_lambda, delay, opt,
                           momentum, update_rms, ns_steps, pred, nadam_psi, beta3)


class Stage:
    """One pipeline stage resident on a device."""

    def __init__(self, shape: B.StageShape, device: str = "cuda:0", stream: Optional[torch.cuda.Stream] = None):
        self.shape = shape
        self.device = torch.device(device)
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        nbytes = B.stage_required_bytes(shape)
        if nbytes == 0:
            raise B.StageError("stage_required_bytes", B.STAGE_EINVAL, B.last_error())
        self.nbytes = nbytes
        self.arena = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.arena.data_ptr()
        self.base = (base + 255) // 256 * 256
        self._off0 = self.base - base
        self.handle = B.stage_init(shape, self.base, nbytes, self.stream.cuda_stream)
        self.tensors: Dict[str, tuple] = {}
        for i in range(B.stage_num_tensors(self.handle)):
            name, ptr, numel, dt = B.stage_tensor(self.handle, i)
            self.tensors[name] = (ptr, numel, dt)

    def view(self, name: str) -> torch.Tensor:
        """Flat torch view of a named arena region (shares memory with the stage)."""
        ptr, numel, dt = self.tensors[name]
        off = ptr - self.arena.data_ptr()
        return self.arena[off: off + numel * _ESZ[dt]].view(_TORCH_DT[dt])

    def param_names(self):
        return [n for n in self.tensors if "." not in n or n.startswith("blk") and n.count(".") == 1]

    def load_master(self, params: Dict[str, "object"]) -> None:
        """Write fp32 master weights (numpy or torch, by name) and refresh both compute versions."""
        for name, arr in params.items():
            t = torch.as_tensor(arr, dtype=torch.float32).reshape(-1)
            self.view(name).copy_(t.to(self.device))
        B.stage_sync_weights(self.handle)

    def forward(self, slot: int, step: int, tokens=None, x_in=None, targets=None, y_out=None, loss=None):
        p = lambda t: None if t is None else t.data_ptr()
        B.stage_forward(self.handle, slot, step, p(tokens), p(x_in), p(targets), p(y_out), p(loss))

    def backward(self, slot: int, dy=None, dx_out=None, microbatches_per_step: int = 1):
        p = lambda t: None if t is None else t.data_ptr()
        B.stage_backward(self.handle, slot, p(dy), p(dx_out), microbatches_per_step)

    def update(self, t: int, hp: B.UpdateHParams):
        B.delayed_update(self.handle, t, hp)

    def resume(self, next_t: int, delay: int = 1):
        """Continue a run at iteration next_t from the state written through the views."""
        B.stage_resume(self.handle, next_t, delay)

    def set_update_overlap(self, mode: int):
        """Overlap mode 1: the stage stream waits for an update only where the delay needs it; 2: also
        the update's elementwise pass deferred in chunks beside the attention backwards (state views
        after join_update()); 0: off."""
        B.stage_set_update_overlap(self.handle, int(mode))

    def join_update(self):
        """The stage stream waits for every update issued so far."""
        B.stage_join_update(self.handle)

    def embed_indices(self, slot: int):
        T = self.shape.seq_len * self.shape.micro_batch
        ids = torch.empty(T, dtype=torch.int32, device=self.device)
        counts = torch.empty(T, dtype=torch.int32, device=self.device)
        nu = torch.empty(1, dtype=torch.int32, device=self.device)
        B.stage_embed_indices(self.handle, slot, ids.data_ptr(), counts.data_ptr(), nu.data_ptr())
        torch.cuda.synchronize(self.device)
        n = int(nu.item())
        return ids[:n].cpu().numpy(), counts[:n].cpu().numpy()

    def grad_norm(self, which: int) -> float:
        out = torch.empty(1, dtype=torch.float32, device=self.device)
        B.stage_grad_norm(self.handle, which, out.data_ptr())
        return float(out.item())

    def close(self):
        if getattr(self, "handle", None):
            B.stage_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
