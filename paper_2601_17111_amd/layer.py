"""One MoE expert layer on one GPU with P virtual devices: owns the device
buffers and runs the four library calls in order. Allocation and call
sequencing only; all arithmetic happens in the library's kernels."""

from __future__ import annotations

from typing import List, Optional, Sequence

from . import binding as B


def m_local_bytes(groups: Sequence[Sequence[int]], P: int, D: int, F: int,
                  elem_bytes: int) -> List[int]:
    """Peak-memory model of each device's share (Sec. 3.2, Eq. 4) from a
    plan's group table: for every group (device, expert, row_start, n) its
    n x D token rows, the expert's three D x F SwiGLU matrices and its n x F
    intermediate, in bytes of `elem_bytes` per element."""
    out = [0] * P
    for g in groups:
        d, n = int(g[0]), int(g[3])
        out[d] += (n * (D + F) + 3 * D * F) * elem_bytes
    return out


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

    def ffn(self, w_gate_up, w_down, device: int = -1, stream=None, save_gate_up=False):
        """save_gate_up: keep g and u (self.gate_up) so that backward() does
        not recompute them."""
        if save_gate_up:
            if getattr(self, "gate_up", None) is None:
                import torch
                self.gate_up = torch.empty((max(self.T * self.K, 1), 2 * self.F),
                                           dtype=self.dtype, device=self.device)
            B.llep_grouped_ffn_train(self.params, self.bufs, device, self.x_perm, w_gate_up,
                                     w_down, self.out_perm, self.gate_up, self.workspace, stream)
            self.gate_up_device = device
        else:
            B.llep_grouped_ffn(self.params, self.bufs, device, self.x_perm, w_gate_up, w_down,
                               self.out_perm, self.workspace, stream)
            self.gate_up_device = None

    def combine(self, gates, stream=None):
        B.llep_combine(self.params, self.out_perm, self.pair_row, gates, self.y, stream)

    def forward(self, ids, gates, x, w_gate_up, w_down, device: Optional[int] = -1,
                stream=None, save_gate_up=False):
        """plan -> permute -> grouped FFN (one device's groups, or all with -1)
        -> combine. Returns y (valid for every token only when device == -1).
        save_gate_up: training forward (g and u kept for backward())."""
        self.plan(ids, stream)
        self.permute(ids, gates, x, stream)
        self.ffn(w_gate_up, w_down, -1 if device is None else device, stream, save_gate_up)
        self.combine(gates, stream)
        return self.y

    def _saved_covers(self, device: int) -> bool:
        saved = getattr(self, "gate_up_device", None)
        return saved is not None and (saved == -1 or saved == device)

    def backward(self, dy, gates, w_gate_up, w_gate_up_t, w_down_t, device: int = -1,
                 stream=None):
        """Backward of forward() (bf16 or f32), reusing its plan, permutation and expert
        outputs: combine backward -> grouped FFN backward (one device's groups,
        or all with -1) -> the pairs' input gradients summed per token. Uses
        the g and u of a forward with save_gate_up (same device range), else
        recomputes them.

        Returns (dx [T, D], d_gates [T, K] float32, dw_gate, dw_up [E, D, F],
        dw_down [E, F, D] float32). dx and d_gates cover every token only when
        device == -1; the weight gradients are the device's partials, or with
        -1 the totals after the gradient return (experts without rows: zero).
        """
        import torch
        if not hasattr(self, "d_out_perm"):
            R = max(self.T * self.K, 1)
            dev, E, D, F = self.device, self.E, self.D, self.F
            self.d_out_perm = torch.empty((R, D), dtype=self.dtype, device=dev)
            self.dx_perm = torch.empty((R, D), dtype=self.dtype, device=dev)
            self.d_gates = torch.empty((self.T, self.K), dtype=torch.float32, device=dev)
            self.dx = torch.empty((self.T, D), dtype=self.dtype, device=dev)
            self.dw_gate = torch.empty((E, D, F), dtype=torch.float32, device=dev)
            self.dw_up = torch.empty((E, D, F), dtype=torch.float32, device=dev)
            self.dw_down = torch.empty((E, F, D), dtype=torch.float32, device=dev)
            code = B.LLEP_BF16 if self.dtype == torch.bfloat16 else B.LLEP_F32
            nbytes = B.llep_grouped_ffn_backward_workspace_bytes(self.params, D, F, code)
            self.bwd_workspace = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        for w in (self.dw_gate, self.dw_up, self.dw_down):
            w.zero_()
        B.llep_combine_backward(self.params, self.out_perm, self.pair_row, gates, dy,
                                self.d_out_perm, self.d_gates, stream)
        B.llep_grouped_ffn_backward(self.params, self.bufs, device, self.x_perm, self.d_out_perm,
                                    w_gate_up, w_gate_up_t, w_down_t, self.dx_perm, self.dw_gate,
                                    self.dw_up, self.dw_down, self.bwd_workspace, stream,
                                    self.gate_up if self._saved_covers(device) else None)
        B.llep_combine(self.params, self.dx_perm, self.pair_row, None, self.dx, stream)
        return self.dx, self.d_gates, self.dw_gate, self.dw_up, self.dw_down
