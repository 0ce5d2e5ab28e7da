"""torch.library registration of the W8A8 linear, and a drop-in module.

The fused op replaces the bf16 linear at a diffusion transformer's linear layers with
the surrounding runtime unchanged (Section 3, "Integration"). Registered as custom ops
with fake (meta) implementations, the calls stay inside one graph under torch.compile
instead of breaking it at an opaque Python call:

  torch.ops.w8a8.linear(x, wq, w_scale, bias, act, col_mul) -> y bf16 [..., N]
  torch.ops.w8a8.quantize_act(x, act, col_mul)             -> (xq int8, x_scale fp32)
  torch.ops.w8a8.gemm(xq, x_scale, wq, w_scale, bias)      -> y bf16 [M, N]

The ops are inference-only (no autograd formula): the integer codes have no useful
gradient. The real implementations are the HIP library's entry points; the fake ones
only compute output shapes and dtypes.
"""
from __future__ import annotations

from typing import Optional

import torch

from . import ACTS, gemm, linear, quantize_act, quantize_weight

_ACT_NAMES = {v: k for k, v in ACTS.items()}


@torch.library.custom_op("w8a8::linear", mutates_args=())
def linear_op(x: torch.Tensor, wq: torch.Tensor, w_scale: torch.Tensor,
              bias: Optional[torch.Tensor], act: int,
              col_mul: Optional[torch.Tensor]) -> torch.Tensor:
    return linear(x, wq, w_scale, bias, act=_ACT_NAMES[act], col_mul=col_mul)


@linear_op.register_fake
def _linear_fake(x, wq, w_scale, bias, act, col_mul):
    torch._check(x.shape[-1] == wq.shape[1], lambda: "K mismatch")
    return x.new_empty((*x.shape[:-1], wq.shape[0]), dtype=torch.bfloat16)


@torch.library.custom_op("w8a8::quantize_act", mutates_args=())
def quantize_act_op(x: torch.Tensor, act: int,
                    col_mul: Optional[torch.Tensor]) -> tuple[torch.Tensor, torch.Tensor]:
    return quantize_act(x, act=_ACT_NAMES[act], col_mul=col_mul)


@quantize_act_op.register_fake
def _quantize_act_fake(x, act, col_mul):
    return (x.new_empty(x.shape, dtype=torch.int8),
            x.new_empty((x.shape[0],), dtype=torch.float32))


@torch.library.custom_op("w8a8::gemm", mutates_args=())
def gemm_op(xq: torch.Tensor, x_scale: torch.Tensor, wq: torch.Tensor,
            w_scale: torch.Tensor, bias: Optional[torch.Tensor]) -> torch.Tensor:
    return gemm(xq, x_scale, wq, w_scale, bias)


@gemm_op.register_fake
def _gemm_fake(xq, x_scale, wq, w_scale, bias):
    torch._check(xq.shape[1] == wq.shape[1], lambda: "K mismatch")
    return xq.new_empty((xq.shape[0], wq.shape[0]), dtype=torch.bfloat16)


class W8A8Linear(torch.nn.Module):
    """Inference replacement for a bf16 nn.Linear: per-channel int8 weights (quantized
    once, here), per-token int8 activations and the fused int8 GEMM + dequantization
    epilogue on every call. With `smooth` (SmoothQuant factors s [K]) the weights are
    quantized as W * s and the activations multiplied by 1/s inside the quantizer; with
    act="gelu" the module consumes the pre-activation of a GELU MLP."""

    def __init__(self, wq: torch.Tensor, w_scale: torch.Tensor,
                 bias: Optional[torch.Tensor] = None, *, act: str = "none",
                 smooth_inv: Optional[torch.Tensor] = None):
        super().__init__()
        self.register_buffer("wq", wq)
        self.register_buffer("w_scale", w_scale)
        self.register_buffer("bias", bias)
        self.register_buffer("smooth_inv", smooth_inv)
        self.act = ACTS[act]
        self.in_features = wq.shape[1]
        self.out_features = wq.shape[0]

    @classmethod
    def from_linear(cls, lin: torch.nn.Linear, *, act: str = "none",
                    smooth: Optional[torch.Tensor] = None,
                    smooth_inv: Optional[torch.Tensor] = None) -> "W8A8Linear":
        if (smooth is None) != (smooth_inv is None):
            raise ValueError("pass both smooth and smooth_inv, or neither")
        w = lin.weight.detach().to(torch.bfloat16).contiguous()
        wq, sw = quantize_weight(w, col_mul=smooth)
        b = None if lin.bias is None else lin.bias.detach().to(torch.bfloat16).contiguous()
        return cls(wq, sw, b, act=act, smooth_inv=smooth_inv)

    def forward(self, x: torch.Tensor) -> torch.Tensor:
        return torch.ops.w8a8.linear(x, self.wq, self.w_scale, self.bias, self.act,
                                     self.smooth_inv)

    def extra_repr(self) -> str:
        return (f"in_features={self.in_features}, out_features={self.out_features}, "
                f"act={_ACT_NAMES[self.act]}, smoothed={self.smooth_inv is not None}")
