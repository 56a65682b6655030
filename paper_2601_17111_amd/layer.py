"""One MoE expert layer on one GPU with P virtual devices: owns the device
buffers and runs the four library calls in order. Allocation and call
sequencing only; all arithmetic happens in the library's kernels."""

from __future__ import annotations

from typing import Optional

from . import binding as B


class LLEPLayer:
    """Buffers and calls for one layer shape.

    ids [T, K] int32, gates [T, K] float32, x [T, D] (bf16 or f32) are device
    tensors; w_gate_up / w_down are the packed weights (llep_pack_weights).
    """

    def __init__(self, T: int, K: int, E: int, P: int, D: int, F: int, capacity: int,
                 dtype, device="cuda", min_chunk: int = 1, lam: float = 0.0,
                 mode: str = "llep"):
        import torch
        self.T, self.K, self.E, self.P, self.D, self.F = T, K, E, P, D, F
        self.dtype = dtype
        self.device = device
        self.params = B.make_params(T, K, E, P, capacity, min_chunk, lam, mode)
        self.bufs = B.PlanBuffers(self.params, device)
        R = T * K
        self.x_perm = torch.empty((max(R, 1), D), dtype=dtype, device=device)
        self.out_perm = torch.empty((max(R, 1), D), dtype=dtype, device=device)
        self.gate_perm = torch.empty(max(R, 1), dtype=torch.float32, device=device)
        self.row_pair = torch.empty(max(R, 1), dtype=torch.int32, device=device)
        self.pair_row = torch.empty(max(R, 1), dtype=torch.int32, device=device)
        self.y = torch.empty((T, D), dtype=dtype, device=device)
        code = B.LLEP_BF16 if dtype == torch.bfloat16 else B.LLEP_F32
        nbytes = B.llep_grouped_ffn_workspace_bytes(self.params, F, code)
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)

    def set_mode(self, mode: str):
        self.params.mode = B.LLEP_MODE_EP if mode == "ep" else B.LLEP_MODE_LLEP

    def plan(self, ids, stream=None):
        B.llep_plan(self.params, ids, self.bufs, stream)

    def permute(self, ids, gates, x, stream=None):
        B.llep_permute(self.params, self.bufs, ids, gates, x, self.x_perm, self.gate_perm,
                       self.row_pair, self.pair_row, stream)

    def ffn(self, w_gate_up, w_down, device: int = -1, stream=None):
        B.llep_grouped_ffn(self.params, self.bufs, device, self.x_perm, w_gate_up, w_down,
                           self.out_perm, self.workspace, stream)

    def combine(self, gates, stream=None):
        B.llep_combine(self.params, self.out_perm, self.pair_row, gates, self.y, stream)

    def forward(self, ids, gates, x, w_gate_up, w_down, device: Optional[int] = -1,
                stream=None):
        """plan -> permute -> grouped FFN (one device's groups, or all with -1)
        -> combine. Returns y (valid for every token only when device == -1)."""
        self.plan(ids, stream)
        self.permute(ids, gates, x, stream)
        self.ffn(w_gate_up, w_down, -1 if device is None else device, stream)
        self.combine(gates, stream)
        return self.y
