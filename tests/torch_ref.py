"""An independent float64 PyTorch (CPU, autograd) statement of the same LM loss.

Used only to pin the oracle: it shares no code with ``oracle.model`` (its own
parameter slicing, its own attention / norms), and its exact Hessian-vector
product comes from double backward rather than from finite differences.
"""
import math

import torch


def _slices(cfg):
    d, F, V, H, Hkv = cfg["d_model"], cfg["d_ff"], cfg["vocab"], cfg["n_heads"], cfg["n_kv_heads"]
    dh = d // H
    shapes = []
    if cfg["family"] == "gpt2":
        shapes += [("wte", (V, d)), ("wpe", (cfg["max_seq"], d))]
        for l in range(cfg["n_layers"]):
            shapes += [(f"{l}.g1", (d,)), (f"{l}.b1", (d,)), (f"{l}.wqkv", (3 * d, d)),
                       (f"{l}.bqkv", (3 * d,)), (f"{l}.wo", (d, d)), (f"{l}.bo", (d,)),
                       (f"{l}.g2", (d,)), (f"{l}.b2", (d,)), (f"{l}.w1", (F, d)),
                       (f"{l}.bf1", (F,)), (f"{l}.w2", (d, F)), (f"{l}.bf2", (d,))]
        shapes += [("gf", (d,)), ("bf", (d,))]
    else:
        shapes += [("emb", (V, d))]
        for l in range(cfg["n_layers"]):
            shapes += [(f"{l}.g1", (d,)), (f"{l}.wqkv", ((H + 2 * Hkv) * dh, d)),
                       (f"{l}.wo", (d, H * dh)), (f"{l}.g2", (d,)),
                       (f"{l}.wgu", (2 * F, d)), (f"{l}.wd", (d, F))]
        shapes += [("gf", (d,)), ("head", (V, d))]
    return shapes


def num_params(cfg):
    return sum(math.prod(s) for _, s in _slices(cfg))


def _params(cfg, flat):
    out, off = {}, 0
    for name, shape in _slices(cfg):
        n = math.prod(shape)
        out[name] = flat[off:off + n].view(shape)
        off += n
    return out


def _ln(x, g, b, eps):
    return torch.nn.functional.layer_norm(x, (x.shape[-1],), g, b, eps)


def _rms(x, g, eps):
    return x * torch.rsqrt((x * x).mean(-1, keepdim=True) + eps) * g


def _rope(x, base):
    S, dh = x.shape[-2], x.shape[-1]
    half = dh // 2
    inv = base ** (-torch.arange(half, dtype=torch.float64) * 2 / dh)
    ang = torch.arange(S, dtype=torch.float64)[:, None] * inv[None, :]
    c, s = torch.cos(ang), torch.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return torch.cat([x1 * c - x2 * s, x2 * c + x1 * s], -1)


def loss(cfg, flat, tokens, labels=None):
    W = _params(cfg, flat)
    tok = torch.as_tensor(tokens, dtype=torch.long)
    B, S = tok.shape
    d, H, Hkv, F = cfg["d_model"], cfg["n_heads"], cfg["n_kv_heads"], cfg["d_ff"]
    dh = d // H
    eps = 1e-5
    gpt2 = cfg["family"] == "gpt2"
    x = W["wte"][tok] + W["wpe"][:S] if gpt2 else W["emb"][tok]
    mask = torch.ones(S, S, dtype=torch.bool).triu(1)
    for l in range(cfg["n_layers"]):
        a = _ln(x, W[f"{l}.g1"], W[f"{l}.b1"], eps) if gpt2 else _rms(x, W[f"{l}.g1"], eps)
        qkv = a @ W[f"{l}.wqkv"].T
        if gpt2:
            qkv = qkv + W[f"{l}.bqkv"]
        q, k, v = torch.split(qkv, [H * dh, Hkv * dh, Hkv * dh], -1)
        q = q.view(B, S, H, dh).transpose(1, 2)
        k = k.view(B, S, Hkv, dh).transpose(1, 2)
        v = v.view(B, S, Hkv, dh).transpose(1, 2)
        if not gpt2:
            q, k = _rope(q, cfg["rope_base"]), _rope(k, cfg["rope_base"])
        k = k.repeat_interleave(H // Hkv, 1)
        v = v.repeat_interleave(H // Hkv, 1)
        sc = (q @ k.transpose(-1, -2)) / math.sqrt(dh)
        sc = sc.masked_fill(mask, float("-inf"))
        o = torch.softmax(sc, -1) @ v
        o = o.transpose(1, 2).reshape(B, S, H * dh)
        y = o @ W[f"{l}.wo"].T
        if gpt2:
            y = y + W[f"{l}.bo"]
        x = x + y
        if gpt2:
            h = _ln(x, W[f"{l}.g2"], W[f"{l}.b2"], eps)
            u = h @ W[f"{l}.w1"].T + W[f"{l}.bf1"]
            x = x + torch.nn.functional.gelu(u, approximate="tanh") @ W[f"{l}.w2"].T + W[f"{l}.bf2"]
        else:
            h = _rms(x, W[f"{l}.g2"], eps)
            gt, up = torch.split(h @ W[f"{l}.wgu"].T, [F, F], -1)
            x = x + (torch.nn.functional.silu(gt) * up) @ W[f"{l}.wd"].T
    if gpt2:
        f = _ln(x, W["gf"], W["bf"], eps)
        logits = f @ W["wte"].T
    else:
        f = _rms(x, W["gf"], eps)
        logits = f @ W["head"].T
    # torch's ignore_index=-100 drops those targets from the mean
    tgt = tok if labels is None else torch.as_tensor(labels, dtype=torch.long)
    return torch.nn.functional.cross_entropy(
        logits[:, :-1].reshape(-1, cfg["vocab"]), tgt[:, 1:].reshape(-1), ignore_index=-100)


def grad(cfg, theta, tokens, labels=None):
    t = torch.tensor(theta, dtype=torch.float64, requires_grad=True)
    (g,) = torch.autograd.grad(loss(cfg, t, tokens, labels), t)
    return g.numpy()


def exact_hvp(cfg, theta, v, tokens, labels=None):
    t = torch.tensor(theta, dtype=torch.float64, requires_grad=True)
    vv = torch.tensor(v, dtype=torch.float64)
    (g,) = torch.autograd.grad(loss(cfg, t, tokens, labels), t, create_graph=True)
    (hv,) = torch.autograd.grad(g @ vv, t)
    return hv.numpy()
