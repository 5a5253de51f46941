"""Plain numpy definition of one adapter fine-tuning step of a Qwen3-shaped
decoder (test infrastructure only).

Paper passages followed (arXiv 2609.28568):
  * section "The clinical stage": a frozen Qwen3-0.6B base adapted with
    low-rank adaptation (rank 16, scaling 32), rank-stabilised, i.e. the
    adapter's contribution is scaled by alpha / sqrt(rank); the loss is taken
    on answer tokens only; only the adapter parameters train;
  * section "Optimisation and precision": AdamW with bias correction, the
    decay term inside the learning-rate product, step count starting at 1.

The paper names the base model without describing it. Its shape here is the
public Qwen3-0.6B configuration, as the benchmark configuration states it:
pre-RMSNorm decoder layers; grouped-query attention (16 query heads, 8
key/value heads, head dimension 128) with an RMSNorm over the head dimension
on every query and key head before the rotary embedding (theta 1e6); a gated
MLP down(silu(gate(x)) * up(x)) of width 3072; a final RMSNorm; the token
table tied to the LM head; no biases.

Readings where neither the paper nor that configuration fixes the detail
(each also listed in the design notes):
  RMSNorm y = x / sqrt(mean(x^2) + eps) * w with eps 1e-6; rotary embedding in
  the split-half convention (dimension i pairs with i + hd/2, frequency
  theta^(-2i/hd)); attention scale 1/sqrt(hd), causal, query head h reading
  key/value head h // (H / H_kv); adapters y = x W^T + s (x A^T) B^T with
  A [r, in], B [out, r], s = alpha / sqrt(r); the loss is the mean over the
  unmasked positions (the last half of every sequence, as the benchmark
  configuration states it); the adapter AdamW takes the one AdamW recipe the
  paper states (its optimisation section: betas (0.9, 0.95), eps 1e-8, decay
  0.1 on two-dimensional tensors, which every adapter tensor is, global-norm
  clip 1.0), since the clinical stage names AdamW without other values; the
  rate (2e-4) is the one free choice.

All arithmetic happens in the dtype of the parameters passed in.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# Projections of a layer, their input and output widths as functions of the
# config, in the order the paper's seven-projection adapter set lists them.
PROJECTIONS = ("q", "k", "v", "o", "gate", "up", "down")


@dataclass
class Qwen3Config:
    n_layer: int
    d_model: int
    n_head: int
    n_kv_head: int
    head_dim: int
    d_ff: int
    vocab: int
    max_seq_len: int
    rope_theta: float = 1e6
    rms_eps: float = 1e-6
    lora_rank: int = 16
    lora_alpha: float = 32.0
    lora_targets: tuple = ("q", "k", "v", "o")
    loss_from: float = 0.5      # loss on positions t >= loss_from * T of each sequence
    lr: float = 2e-4
    beta1: float = 0.9
    beta2: float = 0.95
    adam_eps: float = 1e-8
    weight_decay: float = 0.1
    grad_clip: float = 1.0      # global-norm clip of the adapter gradients

    @classmethod
    def from_dict(cls, d: dict) -> "Qwen3Config":
        names = cls.__dataclass_fields__.keys()
        kw = {k: v for k, v in d.items() if k in names}
        if "lora_targets" in kw:
            kw["lora_targets"] = tuple(kw["lora_targets"])
        return cls(**kw)

    @property
    def lora_scale(self) -> float:
        """Rank-stabilised scaling alpha / sqrt(rank) ("The clinical stage")."""
        return self.lora_alpha / math.sqrt(self.lora_rank)


# ----------------------------------------------------------------------------
# Parameter bookkeeping
# ----------------------------------------------------------------------------

def proj_dims(cfg: Qwen3Config, name: str) -> tuple:
    """(in, out) widths of a layer projection; weights are stored [out, in]."""
    C, qd, kvd, F = cfg.d_model, cfg.n_head * cfg.head_dim, cfg.n_kv_head * cfg.head_dim, cfg.d_ff
    return {"q": (C, qd), "k": (C, kvd), "v": (C, kvd), "o": (qd, C),
            "gate": (C, F), "up": (C, F), "down": (F, C)}[name]


def base_shapes(cfg: Qwen3Config) -> dict:
    """Frozen base parameters, stacked over layers."""
    L, C, hd = cfg.n_layer, cfg.d_model, cfg.head_dim
    s = {"embed": (cfg.vocab, C), "in_norm": (L, C), "q_norm": (L, hd), "k_norm": (L, hd),
         "post_norm": (L, C), "final_norm": (C,)}
    for p in PROJECTIONS:
        i, o = proj_dims(cfg, p)
        s[p] = (L, o, i)
    return s


def lora_shapes(cfg: Qwen3Config) -> dict:
    """Adapter parameters A [L, r, in] and B [L, out, r] of every target."""
    L, r = cfg.n_layer, cfg.lora_rank
    s = {}
    for p in cfg.lora_targets:
        i, o = proj_dims(cfg, p)
        s[p + "_A"] = (L, r, i)
        s[p + "_B"] = (L, o, r)
    return s


def lora_param_count(cfg: Qwen3Config) -> int:
    """Trainable parameters: L * r * sum over targets of (in + out)."""
    return sum(int(np.prod(v)) for v in lora_shapes(cfg).values())


# ----------------------------------------------------------------------------
# Forward and backward pieces
# ----------------------------------------------------------------------------

def rmsnorm_forward(x, w, eps):
    """y = x / sqrt(mean(x^2) + eps) * w over the last axis; returns (y, rstd)."""
    rstd = 1.0 / np.sqrt((x * x).mean(axis=-1, keepdims=True) + x.dtype.type(eps))
    return x * rstd * w, rstd[..., 0]


def rmsnorm_backward(dy, x, rstd, w):
    """Gradient of rmsnorm_forward with respect to x (the gain is frozen):
    dx = rstd (g - xhat mean(g xhat)), g = dy w, xhat = x rstd."""
    r = rstd[..., None]
    xhat = x * r
    g = dy * w
    return r * (g - xhat * (g * xhat).mean(axis=-1, keepdims=True))


def rope_tables(T: int, hd: int, theta: float, dtype):
    """cos and sin [T, hd/2] of angle t * theta^(-2i/hd), computed in fp64."""
    inv = theta ** (-np.arange(0, hd, 2, dtype=np.float64) / hd)
    ang = np.arange(T, dtype=np.float64)[:, None] * inv[None, :]
    return np.cos(ang).astype(dtype), np.sin(ang).astype(dtype)


def rope_forward(x, cos, sin):
    """Rotate pairs (i, i + hd/2) of x [..., T, hd] by the position's angle."""
    h = x.shape[-1] // 2
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * cos - x2 * sin, x2 * cos + x1 * sin], axis=-1)


def rope_backward(dy, cos, sin):
    """The transposed rotation (rope_forward is orthogonal)."""
    h = dy.shape[-1] // 2
    d1, d2 = dy[..., :h], dy[..., h:]
    return np.concatenate([d1 * cos + d2 * sin, d2 * cos - d1 * sin], axis=-1)


def lora_linear_forward(x, W, A, B, s):
    """y = x W^T (+ s (x A^T) B^T when the projection is adapted); returns (y, u = x A^T)."""
    y = x @ W.T
    if A is None:
        return y, None
    u = x @ A.T
    return y + x.dtype.type(s) * (u @ B.T), u


def lora_linear_backward(dy, x, u, W, A, B, s):
    """Gradients of lora_linear_forward: dx, and dA, dB for an adapted one.

    dx = dy W + s (dy B) A;  dA = s (dy B)^T x;  dB = s dy^T u."""
    dx = dy @ W
    if A is None:
        return dx, None, None
    sc = x.dtype.type(s)
    du = sc * (dy @ B)
    dx = dx + du @ A
    xf = x.reshape(-1, x.shape[-1])
    dA = du.reshape(-1, du.shape[-1]).T @ xf
    dB = sc * (dy.reshape(-1, dy.shape[-1]).T @ u.reshape(-1, u.shape[-1]))
    return dx, dA, dB


def silu(x):
    return x / (1.0 + np.exp(-x))


def swiglu_forward(g, u):
    """m = silu(g) * u."""
    return silu(g) * u


def swiglu_backward(dm, g, u):
    """(dg, du) of swiglu_forward: silu'(g) = sig(g) (1 + g (1 - sig(g)))."""
    sig = 1.0 / (1.0 + np.exp(-g))
    return dm * u * sig * (1.0 + g * (1.0 - sig)), dm * g * sig


def gqa_attention_forward(q, k, v):
    """Causal grouped-query attention. q [B,H,T,hd], k and v [B,Hkv,T,hd];
    query head h reads key/value head h // (H/Hkv). Returns (out [B,H,T,hd],
    P [B,H,T,T])."""
    H, Hkv = q.shape[1], k.shape[1]
    grp = H // Hkv
    ke, ve = np.repeat(k, grp, axis=1), np.repeat(v, grp, axis=1)
    T, hd = q.shape[2], q.shape[3]
    s = (q @ ke.transpose(0, 1, 3, 2)) * q.dtype.type(1.0 / math.sqrt(hd))
    s = np.where(np.triu(np.ones((T, T), dtype=bool), k=1), -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=-1, keepdims=True)
    return p @ ve, p


def gqa_attention_backward(dout, q, k, v, p):
    """Gradients of gqa_attention_forward; a key/value head collects the
    gradients of its group of query heads."""
    B, H, T, hd = q.shape
    Hkv = k.shape[1]
    grp = H // Hkv
    ke, ve = np.repeat(k, grp, axis=1), np.repeat(v, grp, axis=1)
    scale = q.dtype.type(1.0 / math.sqrt(hd))
    dve = p.transpose(0, 1, 3, 2) @ dout
    dp = dout @ ve.transpose(0, 1, 3, 2)
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
    dq = (ds @ ke) * scale
    dke = (ds.transpose(0, 1, 3, 2) @ q) * scale
    dk = dke.reshape(B, Hkv, grp, T, hd).sum(axis=2)
    dv = dve.reshape(B, Hkv, grp, T, hd).sum(axis=2)
    return dq, dk, dv


def loss_mask(T: int, loss_from: float) -> np.ndarray:
    """Positions whose next-token loss counts: t >= floor(loss_from * T)."""
    return np.arange(T) >= int(math.floor(loss_from * T))


def masked_cross_entropy(logits, targets, mask):
    """Per-position losses lse(logits) - logits[target] on masked positions
    (0 elsewhere), their mean over the n masked positions, and dlogits =
    (softmax - onehot) / n on masked rows, 0 on the others."""
    m = logits.max(axis=-1, keepdims=True)
    e = np.exp(logits - m)
    ssum = e.sum(axis=-1, keepdims=True)
    lse = (m + np.log(ssum))[..., 0]
    tl = np.take_along_axis(logits, targets[..., None], axis=-1)[..., 0]
    mk = np.broadcast_to(mask, targets.shape)
    n = int(mk.sum())
    losses = np.where(mk, lse - tl, 0.0).astype(logits.dtype)
    d = e / ssum
    np.put_along_axis(d, targets[..., None], np.take_along_axis(d, targets[..., None], axis=-1) - 1.0, axis=-1)
    d = np.where(mk[..., None], d, 0.0).astype(logits.dtype) / logits.dtype.type(n)
    return losses, losses.sum() / logits.dtype.type(n), d


# ----------------------------------------------------------------------------
# The step
# ----------------------------------------------------------------------------

def _split(x, heads):
    B, T, D = x.shape
    return x.reshape(B, T, heads, D // heads).transpose(0, 2, 1, 3)


def _merge(x):
    B, H, T, hd = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, T, H * hd)


def _lora(lora, name, l):
    if lora is None or (name + "_A") not in lora:
        return None, None
    return lora[name + "_A"][l], lora[name + "_B"][l]


def forward(base: dict, lora: dict, ids, targets, cfg: Qwen3Config) -> dict:
    """Forward pass and masked loss ("The clinical stage"); returns a cache
    with every intermediate the backward needs, plus 'loss' and 'losses'."""
    dt = base["embed"].dtype.type
    B, T = ids.shape
    H, Hkv, hd = cfg.n_head, cfg.n_kv_head, cfg.head_dim
    s = cfg.lora_scale
    cos, sin = rope_tables(T, hd, cfg.rope_theta, base["embed"].dtype)
    x = base["embed"][ids]
    cache = {"x0": x, "cos": cos, "sin": sin, "layers": []}
    for l in range(cfg.n_layer):
        c = {"x_in": x}
        h, c["r1"] = rmsnorm_forward(x, base["in_norm"][l], cfg.rms_eps)
        c["h"] = h
        proj = {}
        for p in ("q", "k", "v"):
            A, Bm = _lora(lora, p, l)
            proj[p], c["u_" + p] = lora_linear_forward(h, base[p][l], A, Bm, s)
        q = _split(proj["q"], H)
        k = _split(proj["k"], Hkv)
        v = _split(proj["v"], Hkv)
        qn, c["rq"] = rmsnorm_forward(q, base["q_norm"][l], cfg.rms_eps)
        kn, c["rk"] = rmsnorm_forward(k, base["k_norm"][l], cfg.rms_eps)
        c.update(q=q, k=k, v=v)
        qr, kr = rope_forward(qn, cos, sin), rope_forward(kn, cos, sin)
        att, c["p"] = gqa_attention_forward(qr, kr, v)
        c.update(qr=qr, kr=kr)
        a = _merge(att)
        c["a"] = a
        A, Bm = _lora(lora, "o", l)
        o, c["u_o"] = lora_linear_forward(a, base["o"][l], A, Bm, s)
        xm = x + o
        c["x_mid"] = xm
        h2, c["r2"] = rmsnorm_forward(xm, base["post_norm"][l], cfg.rms_eps)
        c["h2"] = h2
        A, Bm = _lora(lora, "gate", l)
        gt, c["u_gate"] = lora_linear_forward(h2, base["gate"][l], A, Bm, s)
        A, Bm = _lora(lora, "up", l)
        up, c["u_up"] = lora_linear_forward(h2, base["up"][l], A, Bm, s)
        mm = swiglu_forward(gt, up)
        c.update(gate=gt, up=up, m=mm)
        A, Bm = _lora(lora, "down", l)
        dn, c["u_down"] = lora_linear_forward(mm, base["down"][l], A, Bm, s)
        x = xm + dn
        cache["layers"].append(c)
    cache["x_final"] = x
    xf, cache["rf"] = rmsnorm_forward(x, base["final_norm"], cfg.rms_eps)
    cache["xf"] = xf
    logits = xf @ base["embed"].T
    mask = loss_mask(T, cfg.loss_from)
    losses, loss, dlogits = masked_cross_entropy(logits, targets, mask)
    cache.update(logits=logits, losses=losses, loss=dt(loss), dlogits=dlogits, ids=ids)
    return cache


def backward(base: dict, lora: dict, cache: dict, cfg: Qwen3Config) -> dict:
    """Gradients of the masked mean loss with respect to every adapter
    parameter (the base stays frozen, so only its input gradients flow).
    Also returns 'dx0', the gradient at the embedding output."""
    H, Hkv = cfg.n_head, cfg.n_kv_head
    s = cfg.lora_scale
    grads = {k: np.zeros(v, dtype=base["embed"].dtype) for k, v in lora_shapes(cfg).items()} if lora else {}
    cos, sin = cache["cos"], cache["sin"]
    dxf = cache["dlogits"] @ base["embed"]
    dx = rmsnorm_backward(dxf, cache["x_final"], cache["rf"], base["final_norm"])
    for l in reversed(range(cfg.n_layer)):
        c = cache["layers"][l]

        def lin_back(dy, xin, name):
            A, Bm = _lora(lora, name, l)
            dxi, dA, dB = lora_linear_backward(dy, xin, c["u_" + name], base[name][l], A, Bm, s)
            if dA is not None:
                grads[name + "_A"][l] += dA
                grads[name + "_B"][l] += dB
            return dxi

        # MLP
        dm = lin_back(dx, c["m"], "down")
        dg, du = swiglu_backward(dm, c["gate"], c["up"])
        dh2 = lin_back(dg, c["h2"], "gate") + lin_back(du, c["h2"], "up")
        dxm = dx + rmsnorm_backward(dh2, c["x_mid"], c["r2"], base["post_norm"][l])
        # attention
        da = lin_back(dxm, c["a"], "o")
        dqr, dkr, dv = gqa_attention_backward(_split(da, H), c["qr"], c["kr"], c["v"], c["p"])
        dqn, dkn = rope_backward(dqr, cos, sin), rope_backward(dkr, cos, sin)
        dq = rmsnorm_backward(dqn, c["q"], c["rq"], base["q_norm"][l])
        dk = rmsnorm_backward(dkn, c["k"], c["rk"], base["k_norm"][l])
        dh = (lin_back(_merge(dq), c["h"], "q") + lin_back(_merge(dk), c["h"], "k")
              + lin_back(_merge(dv), c["h"], "v"))
        dx = dxm + rmsnorm_backward(dh, c["x_in"], c["r1"], base["in_norm"][l])
    grads["dx0"] = dx
    return grads


def adamw_step(lora: dict, grads: dict, m: dict, v: dict, step: int, cfg: Qwen3Config) -> None:
    """In-place AdamW on the adapter parameters, step counted from 0
    ("Optimisation and precision": bias correction with t = step + 1, decay
    inside the learning-rate product)."""
    t = step + 1
    dt = next(iter(lora.values())).dtype.type
    b1, b2 = dt(cfg.beta1), dt(cfg.beta2)
    bc1, bc2 = dt(1.0 - cfg.beta1 ** t), dt(1.0 - cfg.beta2 ** t)
    for k in lora:
        g = grads[k]
        m[k] = b1 * m[k] + (1 - b1) * g
        v[k] = b2 * v[k] + (1 - b2) * g * g
        upd = (m[k] / bc1) / (np.sqrt(v[k] / bc2) + dt(cfg.adam_eps)) + dt(cfg.weight_decay) * lora[k]
        lora[k] -= dt(cfg.lr) * upd


def train_step(base: dict, lora: dict, m: dict, v: dict, step: int, ids, targets, cfg: Qwen3Config):
    """One adapter step: forward and masked loss, adapter gradients, global-norm
    clipping of those gradients to grad_clip, AdamW. Returns (loss, norm
    before clipping)."""
    from .gpt2 import clip_coefficient, global_norm
    cache = forward(base, lora, ids, targets, cfg)
    grads = backward(base, lora, cache, cfg)
    grads.pop("dx0")
    norm = global_norm(grads)
    coef = clip_coefficient(norm, cfg.grad_clip)
    dt = next(iter(lora.values())).dtype.type
    adamw_step(lora, {k: g * dt(coef) for k, g in grads.items()}, m, v, step, cfg)
    return cache["loss"], norm
