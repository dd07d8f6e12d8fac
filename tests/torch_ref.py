"""Independent float64 forward of the SwiGLU decoder with PyTorch library ops.

Used only to pin the oracle's model forward and its MLP steering.  It shares
nothing with the oracle: attention is
``torch.nn.functional.scaled_dot_product_attention`` with a causal mask, RoPE
is a complex rotation (``torch.polar``), the MLP uses
``torch.nn.functional.silu``, the steering LayerNorm is
``torch.nn.functional.layer_norm``, and the matrix products are ``torch``
matmuls.
"""
import numpy as np
import torch
import torch.nn.functional as F

import sd2_inputs as si


def _t(a, dtype):
    if dtype == "bf16":
        return torch.from_numpy(si.bf16_to_f32(a)).double()
    return torch.from_numpy(a).double()


def rope_complex(x, pos, theta):
    """x [..., T, hd]; pairs (i, i + hd/2) rotated by pos * theta^(-2i/hd)."""
    hd = x.shape[-1]
    half = hd // 2
    freqs = theta ** (-torch.arange(half, dtype=torch.float64) * 2.0 / hd)
    ang = pos.double()[:, None] * freqs[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)
    z = torch.complex(x[..., :half], x[..., half:]) * rot
    return torch.cat([z.real, z.imag], dim=-1)


def tap_blocks(L):
    """Decoder blocks (counted from 1) whose outputs feed W_hml, in the order high, middle, low."""
    return [L - 2, L // 2, 3]


def forward(dm, w, dtype, toks, add=None, ubias=None, taps=False, obias=None, cond=None):
    """Causal forward of a whole sequence; returns (final-norm hidden [T][d], logits [T][V]).

    ubias: up-projection biases added before the gating product, [L][F] for every row or
    [T][L][F] per row.  obias: a bias added to every layer's MLP output, [d] or [T][d] per row.
    cond: the conditional MLP bias, a dict with vf [L*R][d], vg [L*R][d_V], u [L*F][R] (model
    dtype), rank R, per-row steering vectors g [T][d_V] and a per-row mask on [T] (rows without
    a bias): layer l adds U_l SiLU(V_l [f; g]) to the up projection, V_l = [V_l^f V_l^g]
    concatenated and f the layer's input row.  taps=True also returns the residual stream after
    the tap blocks, [T][3][d]."""
    T = len(toks)
    d, H, Hkv, hd = dm.d_model, dm.n_heads, dm.n_kv_heads, dm.head_dim
    toks_t = torch.as_tensor(np.asarray(toks, dtype=np.int64))
    x = _t(w["embed"], dtype)[toks_t]
    if add is not None:
        x = x + torch.as_tensor(add, dtype=torch.float64)
    pos = torch.arange(T)
    ub = None if ubias is None else torch.as_tensor(np.asarray(ubias), dtype=torch.float64)
    outs = []

    def norm(v, g):
        return v * torch.rsqrt(v.pow(2).mean(-1, keepdim=True) + dm.rms_eps) * _t(g, dtype)

    for li, layer in enumerate(w["layers"]):
        an, wq, wk, wv, wo, fn, wg, wu, wd = layer
        cb = None
        if cond is not None:
            R, Fd = cond["rank"], dm.d_ff
            V = torch.cat([_t(cond["vf"], dtype)[li * R:(li + 1) * R], _t(cond["vg"], dtype)[li * R:(li + 1) * R]], dim=1)
            fg = torch.cat([x, torch.as_tensor(np.asarray(cond["g"]), dtype=torch.float64)], dim=1)
            cb = F.silu(fg @ V.T) @ _t(cond["u"], dtype)[li * Fd:(li + 1) * Fd].T
            cb = cb * torch.as_tensor(np.asarray(cond["on"], dtype=np.float64))[:, None]
        n = norm(x, an)
        q = (n @ _t(wq, dtype).T).view(T, H, hd).transpose(0, 1)
        k = (n @ _t(wk, dtype).T).view(T, Hkv, hd).transpose(0, 1)
        v = (n @ _t(wv, dtype).T).view(T, Hkv, hd).transpose(0, 1)
        q = rope_complex(q, pos, dm.rope_theta)
        k = rope_complex(k, pos, dm.rope_theta)
        k = k.repeat_interleave(H // Hkv, dim=0)
        v = v.repeat_interleave(H // Hkv, dim=0)
        o = F.scaled_dot_product_attention(q[None], k[None], v[None], is_causal=True)[0]
        x = x + o.transpose(0, 1).reshape(T, H * hd) @ _t(wo, dtype).T
        n2 = norm(x, fn)
        up = n2 @ _t(wu, dtype).T
        if ub is not None:
            up = up + (ub[li] if ub.dim() == 2 else ub[:, li, :])
        if cb is not None:
            up = up + cb
        x = x + (F.silu(n2 @ _t(wg, dtype).T) * up) @ _t(wd, dtype).T
        if obias is not None:
            x = x + torch.as_tensor(np.asarray(obias), dtype=torch.float64)
        outs.append(x)
    hF = norm(x, w["final_norm"])
    logits = (hF @ _t(w["lm_head"], dtype).T).numpy()
    if not taps:
        return hF.numpy(), logits
    tp = torch.stack([outs[blk - 1] for blk in tap_blocks(len(w["layers"]))], dim=1)
    return hF.numpy(), logits, tp.numpy()


def mlp_steer(z, mlp, dtype, n_layers, d_ff):
    """Biases from z = [h; m; l]: W_s LayerNorm(W_hml z), per-layer up-projection biases [L][F]
    (form 1) or the one bias after every MLP [d_D] (form 2)."""
    zt = torch.as_tensor(np.asarray(z, dtype=np.float64)).reshape(-1)
    g = _t(mlp["w_hml"], dtype) @ zt
    g = F.layer_norm(g, (g.shape[0],), weight=_t(mlp["ln_gain"], dtype), bias=_t(mlp["ln_bias"], dtype),
                     eps=mlp["ln_eps"])
    out = _t(mlp["w_s"], dtype) @ g
    return (out.reshape(n_layers, d_ff) if int(mlp.get("form", 1)) == 1 else out).numpy()


def steer_g(z, mlp, dtype):
    """g = LayerNorm(W_hml z) for z = [h; m; l]."""
    zt = torch.as_tensor(np.asarray(z, dtype=np.float64)).reshape(-1)
    g = _t(mlp["w_hml"], dtype) @ zt
    return F.layer_norm(g, (g.shape[0],), weight=_t(mlp["ln_gain"], dtype), bias=_t(mlp["ln_bias"], dtype),
                        eps=mlp["ln_eps"]).numpy()
