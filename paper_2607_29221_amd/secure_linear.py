"""Pi_Sec-Linear on one GPU (Section 5 protocol box): a floating-point linear
layer evaluated through the masked ring product. This module orders C-ABI
calls and allocates buffers; every arithmetic step is a libmosaic kernel.

Init W (once per weight matrix W, N x K fp32):
  1. signs d in {-1, +1}^K from the Philox sign stream, R = H diag(d) / sqrt(b)
     (block-diagonal with Sylvester blocks of length b when K is not a power
     of two: K = 28672 uses seven blocks of 4096);
  2. rotate every weight row, W~ = W R^T, and quantise each row to q_w
     (int8 weights: q_w = 127) with scale s_w = max |row| / q_w;
  3. Init W of Pi_Sec-Approx-MatMul on the integer codes.
Online (activations A, M x K fp32, one row per token):
  1. rotate every token, A~ = A R^T (the protocol box's R X in the row-major layout), and
     quantise each token to q_x with scale s_x;
  2. Init X, mask, server product and unmask of Pi_Sec-Approx-MatMul;
  3. dequantise in the unmask epilogue: Y = s_x[m] s_w[n] Y^[m, n], plus
     the optional bias b[n].

The activation window q_x is the largest value for which no inner product of
the noisy codes can leave the signed ring range: with |E| <= bound,
K (q_w + bound) (q_x + bound) <= 2^31 - 1 (the window condition of the
"Straw-man solution" paragraph, with the LWE error added to both operands).
"""
from __future__ import annotations

from typing import Optional

import torch

from . import mosaic as m
from . import protocol as gp

MAX_BLOCK = 32768


def rotation_block(K: int) -> int:
    """Largest power of two <= 32768 dividing K (the Sylvester block length)."""
    b = 1
    while b * 2 <= MAX_BLOCK and K % (b * 2) == 0:
        b *= 2
    if b < 16:
        raise ValueError(f"K = {K} has no power-of-two block >= 16")
    return b


def activation_window(K: int, q_w: int, bound: int) -> int:
    lim = (2 ** 31 - 1) // (K * (q_w + bound))
    q_x = lim - bound
    if q_x < 1:
        raise ValueError(f"no activation window for K = {K}, q_w = {q_w}")
    return int(q_x)


class SecureLinear:
    """One linear layer y = x W^T + b through Pi_Sec-Linear (b optional, N
    floats, added in the unmask epilogue)."""

    def __init__(self, W: torch.Tensor, params, seed: int, weight_id: int, q_w: int = 127,
                 keep_weight_codes: bool = False, bias: Optional[torch.Tensor] = None):
        if W.dtype != torch.float32 or W.dim() != 2:
            raise ValueError("W must be a 2-D float32 tensor (N x K)")
        if bias is not None and (bias.dtype != torch.float32 or bias.shape != (W.shape[0],)
                                 or not bias.is_contiguous()):
            raise ValueError("bias must be a contiguous float32 vector of N entries")
        self.bias = bias
        dev = W.device
        self.N, self.K = W.shape
        self.block = rotation_block(self.K)
        self.q_w = q_w
        bound = params.noise.bound if params.noise.kind != "zero" else 0
        self.q_x = activation_window(self.K, q_w, bound)
        self.signs = torch.empty(self.K, dtype=torch.int8, device=dev)
        m.mosaic_sample_signs(m.rng(seed, gp.STREAM_SIGNS, weight_id, m.DIST_ZERO), self.K, self.signs)
        Wr = torch.empty_like(W)
        m.mosaic_hadamard_rotate(W, Wr, block=self.block, signs=self.signs)
        codes = torch.empty((self.N, self.K), dtype=torch.int32, device=dev)
        self.s_w = torch.empty(self.N, dtype=torch.float32, device=dev)
        m.mosaic_quantize_rows(Wr, q_w, q=codes, scale=self.s_w)
        del Wr
        self.w = gp.MaskedWeight(codes, params, seed, weight_id)
        self.weight_codes: Optional[torch.Tensor] = codes if keep_weight_codes else None
        del codes
        self.last_codes: Optional[torch.Tensor] = None
        self.last_scales: Optional[torch.Tensor] = None
        self.last_buf: Optional[gp.CallBuffers] = None
        self.fused = True                   # fused input pass when the shape allows
        # When set to a list, each call appends (phase, event) pairs recorded
        # on the current stream at the phase boundaries: "begin", "init_x",
        # "input" (rotation, quantisation, mask), "server", "unmask".
        self.phase_events: Optional[list] = None

    def _mark(self, phase: str) -> None:
        if self.phase_events is not None:
            ev = torch.cuda.Event(enable_timing=True)
            ev.record()
            self.phase_events.append((phase, ev))

    def quantize_activations(self, x: torch.Tensor):
        """Rotated, quantised activations: (codes int32 M x K, scales M)."""
        M = x.shape[0]
        xr = torch.empty_like(x)
        m.mosaic_hadamard_rotate(x, xr, block=self.block, signs=self.signs)
        codes = torch.empty((M, self.K), dtype=torch.int32, device=x.device)
        s_x = torch.empty(M, dtype=torch.float32, device=x.device)
        m.mosaic_quantize_rows(xr, self.q_x, q=codes, scale=s_x)
        return codes, s_x

    def __call__(self, x: torch.Tensor, call_id: int, keep_codes: bool = False) -> torch.Tensor:
        """Online phase. The rotation, quantisation and mask run as one fused
        pass (mosaic_rotate_quantize_mask) unless the codes are to be kept or
        the shape is outside what the fused kernel takes, in which case the
        three passes run in sequence; both give the same bits."""
        if x.dtype != torch.float32 or x.dim() != 2 or x.shape[1] != self.K or not x.is_contiguous():
            raise ValueError("x must be a contiguous float32 tensor (M x K)")
        M = x.shape[0]
        buf = gp.alloc_call(self.w, M, x.device)
        self._mark("begin")
        gp.init_x(self.w, M, call_id, buf)
        self._mark("init_x")
        codes = None
        done = False
        if self.fused and not keep_codes:
            s_x = torch.empty(M, dtype=torch.float32, device=x.device)
            try:
                m.mosaic_rotate_quantize_mask(x, self.q_x, buf.A_masked, block=self.block, signs=self.signs,
                                              u=buf.UK[:, : self.K],
                                              noise=gp._noise_rng(self.w.params, self.w.seed, gp.STREAM_EX, call_id),
                                              scale=s_x)
                done = True
            except m.MosaicError as err:
                if err.status != m.STATUS_UNSUPPORTED:
                    raise
        if not done:
            codes, s_x = self.quantize_activations(x)
            gp.mask(self.w, codes, call_id, buf)
        self._mark("input")
        gp.server(self.w, M, buf)
        self._mark("server")
        y = torch.empty((M, self.N), dtype=torch.float32, device=x.device)
        gp.unmask(self.w, M, buf, y_f32=y, s_rows=s_x, s_cols=self.s_w, bias=self.bias)
        self._mark("unmask")
        if keep_codes:
            self.last_codes, self.last_scales, self.last_buf = codes, s_x, buf
        return y
