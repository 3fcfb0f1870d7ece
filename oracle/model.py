"""Decoder-only language-model loss and its gradient, in float64 (oracle).

The paper measures on decoder-only causal LMs (GPT-style and Llama/Qwen-style
models, sections 5.1, 6 and 7); its loss is the mean next-token cross-entropy
of such a model (padding labels are ignored, section 7.1), and the
finite-difference HVP needs only gradients of that loss (section 3.1).  The
architecture details the paper leaves open are fixed as follows:

GPT-2 family   token embedding + learned positions; pre-LN blocks
               x += Wo . attn(LN1 x) + bo ;  x += W2 . gelu_tanh(W1 LN2 x + b1) + b2;
               causal multi-head attention with scale 1/sqrt(dh) and biases on
               QKV/O; final LayerNorm; LM head tied to the token embedding.
Llama family   token embedding; blocks
               x += Wo . attn(rope(Wq h), rope(Wk h), Wv h), h = RMS1 x;
               x += Wd . (silu(Wg h') * (Wu h')), h' = RMS2 x;
               grouped-query attention (head i uses KV head i // (H / Hkv)),
               rotate-half RoPE; final RMSNorm; untied LM head; no biases.

LayerNorm eps and RMSNorm eps are taken from the config (1e-5), LayerNorm
variance is the biased one.  The loss is the mean over the B*(S-1) next-token
targets, or over those whose label is not -100 when labels are given.  Everything is float64 numpy; the reverse pass is written by hand.

Flat parameter layout (one vector, per-layer blocks contiguous, which is the
layer partition of the block-diagonal test in section 6):

GPT-2:  wte[V,d] wpe[S_max,d] | per layer: ln1.g ln1.b wqkv[3d,d] bqkv[3d]
        wo[d,d] bo[d] ln2.g ln2.b w1[F,d] b1[F] w2[d,F] b2[d] | lnf.g lnf.b
Llama:  embed[V,d] | per layer: norm1.g wqkv[(H+2Hkv)dh,d] wo[d,H dh]
        norm2.g wgu[2F,d] (gate rows, then up rows) wd[d,F] | normf.g head[V,d]
"""
from __future__ import annotations

from dataclasses import dataclass, field
import math

import numpy as np

GPT2 = "gpt2"
LLAMA = "llama"

MATRIX, GAIN, BIAS = 0, 1, 2


@dataclass
class ModelConfig:
    family: str
    n_layers: int
    d_model: int
    n_heads: int
    d_ff: int
    vocab: int
    max_seq: int
    n_kv_heads: int = 0
    norm_eps: float = 1e-5
    rope_base: float = 10000.0
    bf16: bool = False

    def __post_init__(self):
        if self.n_kv_heads == 0:
            self.n_kv_heads = self.n_heads
        assert self.d_model % self.n_heads == 0
        assert self.n_heads % self.n_kv_heads == 0

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_heads


@dataclass
class Entry:
    name: str
    offset: int
    shape: tuple
    kind: int
    layer: int

    @property
    def numel(self) -> int:
        return int(np.prod(self.shape))


def layout(cfg: ModelConfig) -> list[Entry]:
    d, F, V = cfg.d_model, cfg.d_ff, cfg.vocab
    dh, H, Hkv = cfg.head_dim, cfg.n_heads, cfg.n_kv_heads
    out: list[Entry] = []
    off = 0

    def add(name, shape, kind, layer):
        nonlocal off
        e = Entry(name, off, tuple(shape), kind, layer)
        out.append(e)
        off += e.numel

    if cfg.family == GPT2:
        add("wte", (V, d), MATRIX, -1)
        add("wpe", (cfg.max_seq, d), MATRIX, -1)
        for l in range(cfg.n_layers):
            p = f"h{l}."
            add(p + "ln1.g", (d,), GAIN, l)
            add(p + "ln1.b", (d,), BIAS, l)
            add(p + "wqkv", (3 * d, d), MATRIX, l)
            add(p + "bqkv", (3 * d,), BIAS, l)
            add(p + "wo", (d, d), MATRIX, l)
            add(p + "bo", (d,), BIAS, l)
            add(p + "ln2.g", (d,), GAIN, l)
            add(p + "ln2.b", (d,), BIAS, l)
            add(p + "w1", (F, d), MATRIX, l)
            add(p + "b1", (F,), BIAS, l)
            add(p + "w2", (d, F), MATRIX, l)
            add(p + "b2", (d,), BIAS, l)
        add("lnf.g", (d,), GAIN, -1)
        add("lnf.b", (d,), BIAS, -1)
    elif cfg.family == LLAMA:
        add("embed", (V, d), MATRIX, -1)
        for l in range(cfg.n_layers):
            p = f"h{l}."
            add(p + "norm1.g", (d,), GAIN, l)
            add(p + "wqkv", ((H + 2 * Hkv) * dh, d), MATRIX, l)
            add(p + "wo", (d, H * dh), MATRIX, l)
            add(p + "norm2.g", (d,), GAIN, l)
            add(p + "wgu", (2 * F, d), MATRIX, l)
            add(p + "wd", (d, F), MATRIX, l)
        add("normf.g", (d,), GAIN, -1)
        add("head", (V, d), MATRIX, -1)
    else:
        raise ValueError(cfg.family)
    return out


def num_params(cfg: ModelConfig) -> int:
    lay = layout(cfg)
    return lay[-1].offset + lay[-1].numel


def init_ranges(cfg: ModelConfig):
    """(offset, numel, kind) list for ``synth.init_params``."""
    return [(e.offset, e.numel, e.kind) for e in layout(cfg)]


def unflatten(cfg: ModelConfig, theta: np.ndarray) -> dict:
    return {e.name: theta[e.offset:e.offset + e.numel].reshape(e.shape) for e in layout(cfg)}


# ----------------------------------------------------------------------------
# elementwise pieces
# ----------------------------------------------------------------------------
_K_GELU = math.sqrt(2.0 / math.pi)
_A_GELU = 0.044715


def gelu_tanh(u):
    return 0.5 * u * (1.0 + np.tanh(_K_GELU * (u + _A_GELU * u ** 3)))


def gelu_tanh_grad(u):
    t = np.tanh(_K_GELU * (u + _A_GELU * u ** 3))
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * _K_GELU * (1.0 + 3.0 * _A_GELU * u * u)


def sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def layernorm_fwd(x, g, b, eps):
    mu = x.mean(-1, keepdims=True)
    xc = x - mu
    r = 1.0 / np.sqrt((xc * xc).mean(-1, keepdims=True) + eps)
    xh = xc * r
    return xh * g + b, (xh, r)


def layernorm_bwd(dy, g, cache):
    xh, r = cache
    dxh = dy * g
    dx = r * (dxh - dxh.mean(-1, keepdims=True) - xh * (dxh * xh).mean(-1, keepdims=True))
    dg = (dy * xh).reshape(-1, xh.shape[-1]).sum(0)
    db = dy.reshape(-1, xh.shape[-1]).sum(0)
    return dx, dg, db


def rmsnorm_fwd(x, g, eps):
    r = 1.0 / np.sqrt((x * x).mean(-1, keepdims=True) + eps)
    xh = x * r
    return xh * g, (xh, r)


def rmsnorm_bwd(dy, g, cache):
    xh, r = cache
    dxh = dy * g
    dx = r * (dxh - xh * (dxh * xh).mean(-1, keepdims=True))
    dg = (dy * xh).reshape(-1, xh.shape[-1]).sum(0)
    return dx, dg


def rope_tables(S, dh, base):
    half = dh // 2
    inv = base ** (-np.arange(half, dtype=np.float64) * 2.0 / dh)
    ang = np.arange(S, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def rope_apply(x, cos, sin, inverse=False):
    """Rotate-half RoPE on x[..., S, dh]; ``inverse`` applies the transpose."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    s = -sin if inverse else sin
    return np.concatenate([x1 * cos - x2 * s, x2 * cos + x1 * s], axis=-1)


# ----------------------------------------------------------------------------
# loss and gradient
# ----------------------------------------------------------------------------
def _attention_fwd(cfg, q, k, v):
    """q [B,H,S,dh], k/v [B,Hkv,S,dh] -> o [B,H,S,dh] and cache."""
    B, H, S, dh = q.shape
    G = H // cfg.n_kv_heads
    ke = np.repeat(k, G, axis=1)
    ve = np.repeat(v, G, axis=1)
    scale = 1.0 / math.sqrt(dh)
    s = np.matmul(q, ke.transpose(0, 1, 3, 2)) * scale
    mask = np.triu(np.ones((S, S), dtype=bool), 1)
    s = np.where(mask, -np.inf, s)
    s = s - s.max(-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(-1, keepdims=True)
    o = np.matmul(p, ve)
    return o, (q, ke, ve, p, scale, G)


def _attention_bwd(cfg, do, cache):
    q, ke, ve, p, scale, G = cache
    dp = np.matmul(do, ve.transpose(0, 1, 3, 2))
    dve = np.matmul(p.transpose(0, 1, 3, 2), do)
    ds = p * (dp - (p * dp).sum(-1, keepdims=True))
    dq = np.matmul(ds, ke) * scale
    dke = np.matmul(ds.transpose(0, 1, 3, 2), q) * scale
    B, H, S, dh = q.shape
    Hkv = H // G
    dk = dke.reshape(B, Hkv, G, S, dh).sum(2)
    dv = dve.reshape(B, Hkv, G, S, dh).sum(2)
    return dq, dk, dv


IGNORE = -100   # label of positions that carry no target (padding, prompt)


def loss_and_grad(cfg: ModelConfig, theta: np.ndarray, tokens: np.ndarray,
                  want_grad: bool = True, labels=None):
    """Mean next-token cross-entropy L(theta) and its gradient (float64).

    ``theta`` is the flat parameter vector (any float dtype; used in float64),
    ``tokens`` int [B, S].  The logits at position t predict the label at
    position t + 1: without ``labels`` that is tokens[:, t + 1]; with
    ``labels`` (int [B, S], aligned with the tokens as in section 7.1, where
    padding positions carry the label -100) it is labels[:, t + 1], and
    positions whose label is -100 are left out of the mean.  The mean is over
    the remaining targets (zero loss and gradient when there are none).
    Returns (L, grad) with grad float64 of length P.
    """
    theta = np.asarray(theta, dtype=np.float64)
    W = unflatten(cfg, theta)
    tok = np.asarray(tokens, dtype=np.int64)
    B, S = tok.shape
    d, H, Hkv, dh, F = cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_ff
    eps = cfg.norm_eps
    gpt2 = cfg.family == GPT2

    # ---- forward -----------------------------------------------------------
    if gpt2:
        x = W["wte"][tok] + W["wpe"][:S][None, :, :]
    else:
        x = W["embed"][tok].copy()
        cos, sin = rope_tables(S, dh, cfg.rope_base)
    caches = []
    for l in range(cfg.n_layers):
        p = f"h{l}."
        c = {}
        if gpt2:
            a, c["n1"] = layernorm_fwd(x, W[p + "ln1.g"], W[p + "ln1.b"], eps)
            qkv = a @ W[p + "wqkv"].T + W[p + "bqkv"]
        else:
            a, c["n1"] = rmsnorm_fwd(x, W[p + "norm1.g"], eps)
            qkv = a @ W[p + "wqkv"].T
        c["a"] = a
        q = qkv[..., :H * dh].reshape(B, S, H, dh).transpose(0, 2, 1, 3)
        k = qkv[..., H * dh:(H + Hkv) * dh].reshape(B, S, Hkv, dh).transpose(0, 2, 1, 3)
        v = qkv[..., (H + Hkv) * dh:].reshape(B, S, Hkv, dh).transpose(0, 2, 1, 3)
        if not gpt2:
            q = rope_apply(q, cos, sin)
            k = rope_apply(k, cos, sin)
        o, c["attn"] = _attention_fwd(cfg, q, k, v)
        of = o.transpose(0, 2, 1, 3).reshape(B, S, H * dh)
        c["o"] = of
        y = of @ W[p + "wo"].T
        if gpt2:
            y = y + W[p + "bo"]
        x = x + y
        if gpt2:
            b2, c["n2"] = layernorm_fwd(x, W[p + "ln2.g"], W[p + "ln2.b"], eps)
            u = b2 @ W[p + "w1"].T + W[p + "b1"]
            z = gelu_tanh(u)
            c["u"] = u
        else:
            b2, c["n2"] = rmsnorm_fwd(x, W[p + "norm2.g"], eps)
            gu = b2 @ W[p + "wgu"].T
            gt, up = gu[..., :F], gu[..., F:]
            sg = sigmoid(gt)
            z = gt * sg * up
            c["gt"], c["up"], c["sg"] = gt, up, sg
        c["b"] = b2
        c["z"] = z
        if gpt2:
            x = x + z @ W[p + "w2"].T + W[p + "b2"]
        else:
            x = x + z @ W[p + "wd"].T
        caches.append(c)
    if gpt2:
        f, cf = layernorm_fwd(x, W["lnf.g"], W["lnf.b"], eps)
        wh = W["wte"]
    else:
        f, cf = rmsnorm_fwd(x, W["normf.g"], eps)
        wh = W["head"]
    logits = f @ wh.T                       # [B, S, V]
    zl = logits[:, :-1, :]
    raw = tok[:, 1:] if labels is None else np.asarray(labels, dtype=np.int64)[:, 1:]
    valid = raw != IGNORE
    tgt = np.where(valid, raw, 0)
    zmax = zl.max(-1, keepdims=True)
    ez = np.exp(zl - zmax)
    sez = ez.sum(-1, keepdims=True)
    lse = np.log(sez) + zmax
    N = int(valid.sum())
    picked = np.take_along_axis(zl, tgt[..., None], axis=-1)
    loss = float(((lse - picked)[..., 0] * valid).sum() / N) if N else 0.0
    if not want_grad:
        return loss, None

    # ---- reverse pass ------------------------------------------------------
    g = {e.name: np.zeros(e.shape) for e in layout(cfg)}
    dz = ez / sez
    np.put_along_axis(dz, tgt[..., None], np.take_along_axis(dz, tgt[..., None], -1) - 1.0, -1)
    dz *= valid[..., None]
    dz /= max(N, 1)
    dlogits = np.zeros_like(logits)
    dlogits[:, :-1, :] = dz
    dl2 = dlogits.reshape(-1, cfg.vocab)
    f2 = f.reshape(-1, d)
    if gpt2:
        g["wte"] += dl2.T @ f2
    else:
        g["head"] += dl2.T @ f2
    df = dlogits @ wh
    if gpt2:
        dx, g["lnf.g"], g["lnf.b"] = layernorm_bwd(df, W["lnf.g"], cf)
    else:
        dx, g["normf.g"] = rmsnorm_bwd(df, W["normf.g"], cf)

    for l in reversed(range(cfg.n_layers)):
        p = f"h{l}."
        c = caches[l]
        # MLP
        dy = dx
        dy2 = dy.reshape(-1, d)
        z2 = c["z"].reshape(B * S, -1)
        if gpt2:
            g[p + "w2"] += dy2.T @ z2
            g[p + "b2"] += dy2.sum(0)
            dzz = dy @ W[p + "w2"]
            du = dzz * gelu_tanh_grad(c["u"])
            du2 = du.reshape(-1, F)
            g[p + "w1"] += du2.T @ c["b"].reshape(-1, d)
            g[p + "b1"] += du2.sum(0)
            db2 = du @ W[p + "w1"]
            dxn, g[p + "ln2.g"], g[p + "ln2.b"] = layernorm_bwd(db2, W[p + "ln2.g"], c["n2"])
        else:
            g[p + "wd"] += dy2.T @ z2
            dzz = dy @ W[p + "wd"]
            gt, up, sg = c["gt"], c["up"], c["sg"]
            dgt = dzz * up * sg * (1.0 + gt * (1.0 - sg))
            dup = dzz * gt * sg
            dgu = np.concatenate([dgt, dup], axis=-1)
            g[p + "wgu"] += dgu.reshape(-1, 2 * F).T @ c["b"].reshape(-1, d)
            db2 = dgu @ W[p + "wgu"]
            dxn, g[p + "norm2.g"] = rmsnorm_bwd(db2, W[p + "norm2.g"], c["n2"])
        dx = dx + dxn
        # attention
        dy = dx
        dy2 = dy.reshape(-1, d)
        g[p + "wo"] += dy2.T @ c["o"].reshape(-1, H * dh)
        if gpt2:
            g[p + "bo"] += dy2.sum(0)
        do = (dy @ W[p + "wo"]).reshape(B, S, H, dh).transpose(0, 2, 1, 3)
        dq, dk, dv = _attention_bwd(cfg, do, c["attn"])
        if not gpt2:
            dq = rope_apply(dq, cos, sin, inverse=True)
            dk = rope_apply(dk, cos, sin, inverse=True)
        dqkv = np.concatenate([
            dq.transpose(0, 2, 1, 3).reshape(B, S, H * dh),
            dk.transpose(0, 2, 1, 3).reshape(B, S, Hkv * dh),
            dv.transpose(0, 2, 1, 3).reshape(B, S, Hkv * dh)], axis=-1)
        dqkv2 = dqkv.reshape(B * S, -1)
        g[p + "wqkv"] += dqkv2.T @ c["a"].reshape(-1, d)
        if gpt2:
            g[p + "bqkv"] += dqkv2.sum(0)
        da = dqkv @ W[p + "wqkv"]
        if gpt2:
            dxn, g[p + "ln1.g"], g[p + "ln1.b"] = layernorm_bwd(da, W[p + "ln1.g"], c["n1"])
        else:
            dxn, g[p + "norm1.g"] = rmsnorm_bwd(da, W[p + "norm1.g"], c["n1"])
        dx = dx + dxn

    # embeddings
    if gpt2:
        np.add.at(g["wte"], tok.reshape(-1), dx.reshape(-1, d))
        g["wpe"][:S] += dx.sum(0)
    else:
        np.add.at(g["embed"], tok.reshape(-1), dx.reshape(-1, d))

    grad = np.concatenate([g[e.name].reshape(-1) for e in layout(cfg)])
    return loss, grad


def loss(cfg: ModelConfig, theta, tokens, labels=None) -> float:
    return loss_and_grad(cfg, theta, tokens, want_grad=False, labels=labels)[0]


def num_targets(tokens, labels=None) -> int:
    """Number of targets the mean loss is taken over."""
    tok = np.asarray(tokens)
    if labels is None:
        return tok.shape[0] * (tok.shape[1] - 1)
    return int((np.asarray(labels)[:, 1:] != IGNORE).sum())
