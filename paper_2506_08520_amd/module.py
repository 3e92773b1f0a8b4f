"""PyTorch-ROCm modules around the window-attention block of libnystra.

``NystraWindowAttention`` is a drop-in replacement for the (shifted-)window
multi-head self-attention of SwinIR / Uformer-style restoration models (the
W-MSA / SW-MSA module of Sec. 1): feature map in, feature map out, with the
QKV projection, window partition, attention, head merge, output projection
and window reverse all in HIP kernels (``nystra_block_forward``).  PnP-Nystra
is training-free, so the modules are inference-only: their outputs carry no
autograd history.

``SwinTransformerBlock`` is the transformer block those models stack
(LayerNorm, window attention, residual, LayerNorm, MLP, residual), with the
window attention replaced; LayerNorm and the MLP are plain torch layers.
Relative-position bias and the shifted-window mask are not applied: Eqs.
(1)-(8) have neither.
"""
import torch
from torch import nn

from . import binding as B


class NystraWindowAttention(nn.Module):
    """Window attention on x [B, H, W, C] (channels last, contiguous).

    Weights follow the ``y = x W`` convention of the C ABI: ``w_qkv`` [C, 3C]
    (Q, K, V column blocks, head j taking columns j d_h .. (j+1) d_h - 1 of
    each), ``w_proj`` [C, C].  ``attention`` is "nystrom" (PnP-Nystra with
    ``m`` landmarks and ``iters`` pseudo-inverse iterations) or "exact"."""

    def __init__(self, dim, heads, window, shift=0, m=16, iters=6, attention="nystrom",
                 landmark_mode=B.LM_POOL2D, dtype=torch.float32, device="cuda"):
        super().__init__()
        if dim % heads != 0:
            raise ValueError("heads must divide dim")
        if attention not in ("nystrom", "exact"):
            raise ValueError(attention)
        self.dim, self.heads, self.window, self.shift = dim, heads, window, shift
        self.m, self.iters, self.attention = m, iters, attention
        self.opts = B.make_opts(pinv_iters=iters, landmark_mode=landmark_mode)
        kw = dict(dtype=dtype, device=device)
        self.w_qkv = nn.Parameter(torch.empty(dim, 3 * dim, **kw), requires_grad=False)
        self.b_qkv = nn.Parameter(torch.zeros(3 * dim, **kw), requires_grad=False)
        self.w_proj = nn.Parameter(torch.empty(dim, dim, **kw), requires_grad=False)
        self.b_proj = nn.Parameter(torch.zeros(dim, **kw), requires_grad=False)
        self._ws = None
        self._packed, self._packed_key = None, None

    @classmethod
    def from_linear(cls, qkv, proj, heads, window, shift=0, **kw):
        """From the nn.Linear layers of an existing model (weight [out, in])."""
        dim = proj.in_features
        mod = cls(dim, heads, window, shift, dtype=qkv.weight.dtype,
                  device=qkv.weight.device, **kw)
        with torch.no_grad():
            mod.w_qkv.copy_(qkv.weight.t())
            mod.w_proj.copy_(proj.weight.t())
            if qkv.bias is not None:
                mod.b_qkv.copy_(qkv.bias)
            if proj.bias is not None:
                mod.b_proj.copy_(proj.bias)
        return mod

    def _workspace(self, x):
        shape = B.BlockShape(*x.shape[:3], self.dim, self.heads, self.window, self.shift)
        att = B.BLOCK_NYSTROM if self.attention == "nystrom" else B.BLOCK_EXACT
        code = B.F32 if x.dtype == torch.float32 else B.BF16
        need = B.nystra_block_workspace_size(shape, self.m, code, self.opts, att)
        if self._ws is None or self._ws.numel() < need or self._ws.device != x.device:
            self._ws = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
        return self._ws, att

    def _packed_weights(self):
        """The GEMMs' packed image of w_qkv and w_proj, packed again only when
        either weight changed (new storage, or an in-place update, which
        advances the tensor's version counter)."""
        key = tuple((t.data_ptr(), t._version, t.dtype) for t in (self.w_qkv, self.w_proj))
        if key != self._packed_key:
            self._packed = B.nystra_block_pack_weights(self.w_qkv, self.w_proj)
            self._packed_key = key
        return self._packed

    @torch.no_grad()
    def forward(self, x):
        if x.dim() != 4 or x.shape[-1] != self.dim:
            raise ValueError(f"expected [B, H, W, {self.dim}]")
        x = x.contiguous()
        ws, att = self._workspace(x)
        return B.nystra_block_forward(x, self.w_qkv, self.b_qkv, self.w_proj, self.b_proj,
                                      self.heads, self.window, shift=self.shift, m=self.m,
                                      opts=self.opts, attention=att, workspace=ws,
                                      packed=self._packed_weights())


class SwinTransformerBlock(nn.Module):
    """x + attn(norm1(x)), then + mlp(norm2(.)), on x [B, H, W, C]."""

    def __init__(self, dim, heads, window, shift=0, mlp_ratio=2.0, m=16, iters=6,
                 attention="nystrom", dtype=torch.float32, device="cuda"):
        super().__init__()
        kw = dict(dtype=dtype, device=device)
        self.norm1 = nn.LayerNorm(dim, **kw)
        self.attn = NystraWindowAttention(dim, heads, window, shift, m, iters, attention,
                                          dtype=dtype, device=device)
        self.norm2 = nn.LayerNorm(dim, **kw)
        hidden = int(dim * mlp_ratio)
        self.mlp = nn.Sequential(nn.Linear(dim, hidden, **kw), nn.GELU(),
                                 nn.Linear(hidden, dim, **kw))

    @torch.no_grad()
    def forward(self, x):
        x = x + self.attn(self.norm1(x))
        return x + self.mlp(self.norm2(x))
