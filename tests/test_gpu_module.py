"""GPU parity of the nn.Module wrappers: NystraWindowAttention built from
nn.Linear layers, and a SwinIR-shaped transformer block around it, against
float64 compositions of the block oracle with numpy LayerNorm / GELU / MLP."""
import numpy as np
import pytest
from scipy.special import erf

from oracle import block as OB
from helpers import to_host

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def t2n(t):
    return t.detach().double().cpu().numpy()


def linear_pair(C, seed):
    g = torch.Generator().manual_seed(seed)
    qkv, proj = torch.nn.Linear(C, 3 * C), torch.nn.Linear(C, C)
    with torch.no_grad():
        for lin in (qkv, proj):
            lin.weight.copy_(torch.randn(lin.weight.shape, generator=g) / C ** 0.5)
            lin.bias.copy_(0.02 * torch.randn(lin.bias.shape, generator=g))
    return qkv.cuda(), proj.cuda()


@pytest.mark.parametrize("attention", ["nystrom", "exact"])
def test_window_attention_from_linear(attention):
    from paper_2506_08520_amd.module import NystraWindowAttention
    C, heads, w, s = 96, 3, 8, 4
    qkv, proj = linear_pair(C, 11)
    mod = NystraWindowAttention.from_linear(qkv, proj, heads, w, s, m=16, attention=attention)
    x = torch.randn(2, 16, 24, C, generator=torch.Generator().manual_seed(12)).cuda()
    y = to_host(mod(x))
    ref = OB.block_forward(t2n(x), t2n(qkv.weight).T, t2n(qkv.bias), t2n(proj.weight).T,
                           t2n(proj.bias), heads=heads, window=w, shift=s, m=16,
                           attention=attention)
    assert np.abs(y - ref).max() <= 1e-4


def test_window_attention_repacks_after_weight_update():
    """The module packs its projection weights once and reuses the image; an
    in-place update of a weight (or new weights) is packed again."""
    from paper_2506_08520_amd.module import NystraWindowAttention
    C, heads, w, s = 96, 3, 8, 4
    qkv, proj = linear_pair(C, 31)
    mod = NystraWindowAttention.from_linear(qkv, proj, heads, w, s, m=16)
    x = torch.randn(1, 16, 16, C, generator=torch.Generator().manual_seed(32)).cuda()
    y0 = mod(x)
    image = mod._packed
    assert image is not None
    assert torch.equal(mod(x), y0) and mod._packed is image    # reused, not repacked
    qkv2, proj2 = linear_pair(C, 33)
    with torch.no_grad():
        mod.w_qkv.copy_(qkv2.weight.t())
        mod.w_proj.copy_(proj2.weight.t())
    y = to_host(mod(x))
    ref = OB.block_forward(t2n(x), t2n(qkv2.weight).T, t2n(qkv.bias), t2n(proj2.weight).T,
                           t2n(proj.bias), heads=heads, window=w, shift=s, m=16)
    assert np.abs(y - ref).max() <= 1e-4


def layer_norm(x, g, b, eps=1e-5):
    mu = x.mean(-1, keepdims=True)
    var = ((x - mu) ** 2).mean(-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def test_swin_transformer_block():
    from paper_2506_08520_amd.module import SwinTransformerBlock
    torch.manual_seed(3)
    C, heads, w, s = 180, 6, 8, 4
    blk = SwinTransformerBlock(C, heads, w, s, m=16)
    with torch.no_grad():
        blk.attn.w_qkv.copy_(torch.randn(C, 3 * C) / C ** 0.5)
        blk.attn.b_qkv.copy_(0.02 * torch.randn(3 * C))
        blk.attn.w_proj.copy_(torch.randn(C, C) / C ** 0.5)
        blk.attn.b_proj.copy_(0.02 * torch.randn(C))
        for ln in (blk.norm1, blk.norm2):
            ln.weight.copy_(1 + 0.1 * torch.randn(C))
            ln.bias.copy_(0.1 * torch.randn(C))
    x = torch.randn(1, 32, 32, C).cuda()
    y = to_host(blk(x))
    xn = t2n(x)
    a = blk.attn
    h = xn + OB.block_forward(layer_norm(xn, t2n(blk.norm1.weight), t2n(blk.norm1.bias)),
                              t2n(a.w_qkv), t2n(a.b_qkv), t2n(a.w_proj), t2n(a.b_proj),
                              heads=heads, window=w, shift=s, m=16)
    l1, l2 = blk.mlp[0], blk.mlp[2]
    u = layer_norm(h, t2n(blk.norm2.weight), t2n(blk.norm2.bias)) @ t2n(l1.weight).T + t2n(l1.bias)
    u = 0.5 * u * (1 + erf(u / np.sqrt(2)))
    ref = h + u @ t2n(l2.weight).T + t2n(l2.bias)
    assert np.abs(y - ref).max() <= 1e-4


def test_module_rejects_bad_input():
    from paper_2506_08520_amd.module import NystraWindowAttention
    mod = NystraWindowAttention(96, 3, 8)
    with pytest.raises(ValueError):
        mod(torch.zeros(1, 16, 16, 48, device="cuda"))
    with pytest.raises(ValueError):
        NystraWindowAttention(96, 5, 8)
