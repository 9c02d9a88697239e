"""Sparse drop-in for ``torch.nn.Linear`` (with a fused activation) on decode
steps: the pruned weight is encoded once and every call is one ``usp_spmm_ex``
(product, bias, activation and residual add in one kernel launch).

``torch.ops.usp.sparse_linear`` is the custom operator; ``SparseLinear`` is the
module around it. Inputs are fp16 CUDA (HIP) tensors whose last dimension is
``in_features``; leading dimensions are flattened into the token count N.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from . import usp


@torch.library.custom_op("usp::sparse_linear", mutates_args=("workspace",))
def sparse_linear(x: torch.Tensor, handle: int, out_features: int, bias: Optional[torch.Tensor],
                  residual: Optional[torch.Tensor], activation: int,
                  workspace: Optional[torch.Tensor]) -> torch.Tensor:
    """act(x @ W^T + bias) + residual for the encoded W behind ``handle``; x is
    [N, in_features], residual [N, out_features]. The workspace (zero-filled
    once) is left zero again by every call."""
    y = torch.empty((x.shape[0], out_features), dtype=torch.float16, device=x.device)
    usp.usp_spmm_ex(handle, x, y, workspace, bias, residual, activation)
    return y


@sparse_linear.register_fake
def _(x, handle, out_features, bias, residual, activation, workspace):
    return x.new_empty((x.shape[0], out_features))


class SparseLinear(torch.nn.Module):
    """``act(x W^T + b) (+ residual)`` with W pruned by ``mask`` (kept where nonzero).

    weight: [out_features, in_features] tensor (converted to fp16); mask: array or
    tensor of the same shape; bias: [out_features] or None; activation: one of
    "none", "relu", "gelu_tanh", "silu"."""

    def __init__(self, weight: torch.Tensor, mask, bias: Optional[torch.Tensor] = None,
                 activation: str = "none", device: Optional[int] = None):
        super().__init__()
        if activation not in usp.ACTIVATIONS:
            raise ValueError(f"activation must be one of {sorted(usp.ACTIVATIONS)}")
        dev = torch.cuda.current_device() if device is None else int(device)
        w = weight.detach().to(torch.float16).cpu().contiguous().numpy().view(np.uint16)
        m = mask.detach().cpu().numpy() if isinstance(mask, torch.Tensor) else np.asarray(mask)
        m = np.ascontiguousarray(m != 0, dtype=np.uint8)
        if m.shape != w.shape:
            raise ValueError("mask must have the weight's shape")
        self.matrix = usp.SparseMatrix(w, m, dev)
        self.out_features, self.in_features = w.shape
        self.activation = activation
        self.register_buffer(
            "bias", None if bias is None else bias.detach().to(device=f"cuda:{dev}", dtype=torch.float16).contiguous())
        self._ws: Optional[torch.Tensor] = None  # one workspace for every N, grown when a call needs more

    @classmethod
    def from_linear(cls, linear: torch.nn.Linear, mask, activation: str = "none") -> "SparseLinear":
        dev = linear.weight.device.index if linear.weight.is_cuda else None
        return cls(linear.weight, mask, linear.bias, activation, dev)

    def workspace(self, N: int) -> Optional[torch.Tensor]:
        """A zero-filled workspace of at least usp_workspace_size(N) bytes. Every
        completed call leaves a workspace ready for the next call with any N, so
        one buffer serves all token counts; it is replaced (zero-filled again) only
        when a token count needs more bytes than it has."""
        need = self.matrix.workspace_size(N)
        if need == 0:
            return self._ws
        if self._ws is None or self._ws.numel() < need:
            self._ws = self.matrix.make_workspace(N)
        return self._ws

    def forward(self, x: torch.Tensor, residual: Optional[torch.Tensor] = None) -> torch.Tensor:
        lead = x.shape[:-1]
        x2 = x.reshape(-1, self.in_features)
        if x2.dtype != torch.float16 or not x2.is_contiguous():
            x2 = x2.to(torch.float16).contiguous()
        N = x2.shape[0]
        r2 = None
        if residual is not None:
            r2 = residual.reshape(N, self.out_features)
            if r2.dtype != torch.float16 or not r2.is_contiguous():
                r2 = r2.to(torch.float16).contiguous()
        y = torch.ops.usp.sparse_linear(x2, self.matrix.handle, self.out_features, self.bias, r2,
                                        usp.ACTIVATIONS[self.activation], self.workspace(N))
        return y.reshape(*lead, self.out_features)

    def extra_repr(self) -> str:
        return (f"in_features={self.in_features}, out_features={self.out_features}, "
                f"nnz={self.matrix.nnz}, bias={self.bias is not None}, activation={self.activation}")
