"""Plain numpy definition of one GPT-2 training step (test infrastructure only).

Paper passages followed (arXiv 2609.28568):
  * section "Model" and Figure 1: pre-LayerNorm decoder blocks with residual
    connections around attention and the MLP (768 -> 3072, GELU, 3072 -> 768),
    learned positions, token table tied to the LM head, vocabulary padded to a
    multiple of 128 while the softmax covers only the real tokens, so padding
    rows get no probability and no gradient;
  * section "Optimisation and precision": AdamW with betas (0.9, 0.95),
    epsilon 1e-8, weight decay 0.1 on two-dimensional weights only, global-norm
    clipping to 1.0, linear warmup then cosine decay of the learning rate;
  * section "Batch geometry": gradient accumulation over micro-batches.

Readings where the paper is silent (each also listed in the design notes):
  LayerNorm eps 1e-5 with the biased variance; GELU in its tanh form; attention
  scale 1/sqrt(head_dim), causal, no dropout; Q|K|V packed in that order with
  head h on channels [h*hd, (h+1)*hd); weights stored [out, in]; the loss is
  the mean over all tokens, and under accumulation the optimiser gradient is
  the gradient of the mean over all micro-batches; clip coefficient
  c = clip/n when n > clip else 1; bias-corrected AdamW with the decay term
  inside the learning-rate product, step count starting at 1.

All arithmetic happens in the dtype of the parameters passed in.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

# Parameter kinds in the order of the flat buffer.
KINDS = ("wte", "wpe", "ln1w", "ln1b", "qkvw", "qkvb", "attprojw", "attprojb",
         "ln2w", "ln2b", "fcw", "fcb", "fcprojw", "fcprojb", "lnfw", "lnfb")
# Two-dimensional weights receive weight decay ("Optimisation and precision").
DECAYED = frozenset({"wte", "wpe", "qkvw", "attprojw", "fcw", "fcprojw"})


@dataclass
class Config:
    n_layer: int
    n_head: int
    d_model: int
    d_ff: int
    vocab: int
    vocab_padded: int
    max_seq_len: int
    ln_eps: float = 1e-5
    lr_max: float = 6e-4
    lr_min: float = 0.0
    warmup_steps: int = 700
    total_steps: int = 18865
    beta1: float = 0.9
    beta2: float = 0.95
    adam_eps: float = 1e-8
    weight_decay: float = 0.1
    grad_clip: float = 1.0

    @classmethod
    def from_dict(cls, d: dict) -> "Config":
        names = cls.__dataclass_fields__.keys()
        return cls(**{k: v for k, v in d.items() if k in names})


# ----------------------------------------------------------------------------
# Parameter bookkeeping
# ----------------------------------------------------------------------------

def param_shapes(cfg: Config) -> dict:
    """Shapes of the parameter kinds, stacked over layers, weights [out, in]."""
    L, C, F = cfg.n_layer, cfg.d_model, cfg.d_ff
    return {
        "wte": (cfg.vocab_padded, C), "wpe": (cfg.max_seq_len, C),
        "ln1w": (L, C), "ln1b": (L, C), "qkvw": (L, 3 * C, C), "qkvb": (L, 3 * C),
        "attprojw": (L, C, C), "attprojb": (L, C), "ln2w": (L, C), "ln2b": (L, C),
        "fcw": (L, F, C), "fcb": (L, F), "fcprojw": (L, C, F), "fcprojb": (L, C),
        "lnfw": (C,), "lnfb": (C,),
    }


def param_count(cfg: Config, padded: bool = True) -> int:
    """Number of scalar parameters; with padded=False the token table counts
    only the real vocabulary (the figure the paper prints)."""
    n = sum(int(np.prod(s)) for s in param_shapes(cfg).values())
    if not padded:
        n -= (cfg.vocab_padded - cfg.vocab) * cfg.d_model
    return n


def tensor_names(cfg: Config) -> list:
    """Names of the individual parameter tensors, one per layer slice."""
    per_layer = ("ln_1.weight", "ln_1.bias", "attn.c_attn.weight", "attn.c_attn.bias",
                 "attn.c_proj.weight", "attn.c_proj.bias", "ln_2.weight", "ln_2.bias",
                 "mlp.c_fc.weight", "mlp.c_fc.bias", "mlp.c_proj.weight", "mlp.c_proj.bias")
    names = ["wte", "wpe"]
    for l in range(cfg.n_layer):
        names += [f"h.{l}.{n}" for n in per_layer]
    return names + ["ln_f.weight", "ln_f.bias"]


# ----------------------------------------------------------------------------
# Forward pieces
# ----------------------------------------------------------------------------

def embed_forward(wte, wpe, ids):
    """Token embedding plus learned position (Figure 1): x[b,t] = wte[id] + wpe[t]."""
    T = ids.shape[1]
    return wte[ids] + wpe[np.arange(T)][None, :, :]


def layernorm_forward(x, w, b, eps):
    """y = (x - mean) / sqrt(var + eps) * w + b over the last axis, biased var."""
    mean = x.mean(axis=-1, keepdims=True)
    xc = x - mean
    var = (xc * xc).mean(axis=-1, keepdims=True)
    rstd = 1.0 / np.sqrt(var + x.dtype.type(eps))
    y = xc * rstd * w + b
    return y, mean[..., 0], rstd[..., 0]


def layernorm_backward(dy, x, mean, rstd, w):
    """Gradients of layernorm_forward with respect to x, w and b."""
    xhat = (x - mean[..., None]) * rstd[..., None]
    g = dy * w
    C = x.shape[-1]
    gm = g.sum(axis=-1, keepdims=True) / C
    gxm = (g * xhat).sum(axis=-1, keepdims=True) / C
    dx = rstd[..., None] * (g - gm - xhat * gxm)
    axes = tuple(range(x.ndim - 1))
    dw = (dy * xhat).sum(axis=axes)
    db = dy.sum(axis=axes)
    return dx, dw, db


_GELU_K = math.sqrt(2.0 / math.pi)
_GELU_A = 0.044715


def gelu_forward(u):
    """GELU, tanh form: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    t = np.tanh(u.dtype.type(_GELU_K) * (u + u.dtype.type(_GELU_A) * u ** 3))
    return 0.5 * u * (1.0 + t)


def gelu_backward(u, dg):
    """d/du of gelu_forward times the upstream gradient."""
    k, a = u.dtype.type(_GELU_K), u.dtype.type(_GELU_A)
    t = np.tanh(k * (u + a * u ** 3))
    dt = (1.0 - t * t) * k * (1.0 + 3.0 * a * u * u)
    return dg * (0.5 * (1.0 + t) + 0.5 * u * dt)


def _split_heads(x, n_head):
    B, T, C = x.shape
    return x.reshape(B, T, n_head, C // n_head).transpose(0, 2, 1, 3)


def _merge_heads(x):
    B, H, T, hd = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, T, H * hd)


def attention_forward(qkv, n_head):
    """Causal multi-head self-attention on packed q|k|v [B,T,3C].

    S = q k^T / sqrt(hd) with keys j > i excluded, P = softmax over keys,
    out = P v with heads concatenated. Returns (out [B,T,C], P [B,H,T,T])."""
    C = qkv.shape[-1] // 3
    q, k, v = (_split_heads(qkv[..., i * C:(i + 1) * C], n_head) for i in range(3))
    hd = C // n_head
    T = qkv.shape[1]
    s = (q @ k.transpose(0, 1, 3, 2)) * qkv.dtype.type(1.0 / math.sqrt(hd))
    mask = np.triu(np.ones((T, T), dtype=bool), k=1)
    s = np.where(mask, -np.inf, s)
    s = s - s.max(axis=-1, keepdims=True)
    e = np.exp(s)
    p = e / e.sum(axis=-1, keepdims=True)
    return _merge_heads(p @ v), p


def attention_backward(dout, qkv, p, n_head):
    """Gradient of attention_forward with respect to the packed q|k|v."""
    C = qkv.shape[-1] // 3
    q, k, v = (_split_heads(qkv[..., i * C:(i + 1) * C], n_head) for i in range(3))
    hd = C // n_head
    scale = qkv.dtype.type(1.0 / math.sqrt(hd))
    do = _split_heads(dout, n_head)
    dv = p.transpose(0, 1, 3, 2) @ do
    dp = do @ v.transpose(0, 1, 3, 2)
    ds = p * (dp - (dp * p).sum(axis=-1, keepdims=True))
    dq = (ds @ k) * scale
    dk = (ds.transpose(0, 1, 3, 2) @ q) * scale
    return np.concatenate([_merge_heads(dq), _merge_heads(dk), _merge_heads(dv)], axis=-1)


def cross_entropy(logits, targets, vocab, grad_scale):
    """Softmax cross-entropy over the first ``vocab`` columns only.

    Returns per-token losses lse(real logits) - logit[target], and dlogits =
    (softmax - onehot) * grad_scale on the real columns and exactly zero on the
    padding columns."""
    N = logits.shape[0]
    real = logits[:, :vocab]
    mx = real.max(axis=-1, keepdims=True)
    e = np.exp(real - mx)
    ssum = e.sum(axis=-1, keepdims=True)
    lse = mx[:, 0] + np.log(ssum[:, 0])
    losses = lse - real[np.arange(N), targets]
    dlogits = np.zeros_like(logits)
    dlogits[:, :vocab] = e / ssum
    dlogits[np.arange(N), targets] -= 1.0
    dlogits *= logits.dtype.type(grad_scale)
    return losses, dlogits


# ----------------------------------------------------------------------------
# Whole model
# ----------------------------------------------------------------------------

def block_forward(x, p, l, cfg: Config):
    """One pre-LN block: x + attn(LN1(x)), then + MLP(LN2(.)). Returns the
    output and the values the backward pass needs."""
    c = {"x_in": x}
    h1, c["ln1_mean"], c["ln1_rstd"] = layernorm_forward(x, p["ln1w"][l], p["ln1b"][l], cfg.ln_eps)
    c["ln1"] = h1
    qkv = h1 @ p["qkvw"][l].T + p["qkvb"][l]
    c["qkv"] = qkv
    att, c["probs"] = attention_forward(qkv, cfg.n_head)
    c["att"] = att
    x2 = x + (att @ p["attprojw"][l].T + p["attprojb"][l])
    c["x_mid"] = x2
    h2, c["ln2_mean"], c["ln2_rstd"] = layernorm_forward(x2, p["ln2w"][l], p["ln2b"][l], cfg.ln_eps)
    c["ln2"] = h2
    u = h2 @ p["fcw"][l].T + p["fcb"][l]
    c["fc"] = u
    g = gelu_forward(u)
    c["gelu"] = g
    x3 = x2 + (g @ p["fcprojw"][l].T + p["fcprojb"][l])
    c["x_out"] = x3
    return x3, c


def block_backward(dx3, c, p, l, cfg: Config, grads: dict):
    """Backward of block_forward; adds parameter gradients of layer l into
    ``grads`` and returns the gradient with respect to the block input."""
    dm = dx3
    grads["fcprojw"][l] += dm.reshape(-1, dm.shape[-1]).T @ c["gelu"].reshape(-1, c["gelu"].shape[-1])
    grads["fcprojb"][l] += dm.reshape(-1, dm.shape[-1]).sum(axis=0)
    dg = dm @ p["fcprojw"][l]
    du = gelu_backward(c["fc"], dg)
    grads["fcw"][l] += du.reshape(-1, du.shape[-1]).T @ c["ln2"].reshape(-1, c["ln2"].shape[-1])
    grads["fcb"][l] += du.reshape(-1, du.shape[-1]).sum(axis=0)
    dh2 = du @ p["fcw"][l]
    dx2, dw, db = layernorm_backward(dh2, c["x_mid"], c["ln2_mean"], c["ln2_rstd"], p["ln2w"][l])
    grads["ln2w"][l] += dw
    grads["ln2b"][l] += db
    dx2 = dx2 + dx3
    da = dx2
    grads["attprojw"][l] += da.reshape(-1, da.shape[-1]).T @ c["att"].reshape(-1, c["att"].shape[-1])
    grads["attprojb"][l] += da.reshape(-1, da.shape[-1]).sum(axis=0)
    datt = da @ p["attprojw"][l]
    dqkv = attention_backward(datt, c["qkv"], c["probs"], cfg.n_head)
    grads["qkvw"][l] += dqkv.reshape(-1, dqkv.shape[-1]).T @ c["ln1"].reshape(-1, c["ln1"].shape[-1])
    grads["qkvb"][l] += dqkv.reshape(-1, dqkv.shape[-1]).sum(axis=0)
    dh1 = dqkv @ p["qkvw"][l]
    dx, dw, db = layernorm_backward(dh1, c["x_in"], c["ln1_mean"], c["ln1_rstd"], p["ln1w"][l])
    grads["ln1w"][l] += dw
    grads["ln1b"][l] += db
    return dx + dx2


def forward(params, ids, targets, cfg: Config, grad_scale=None):
    """Forward pass: embedding, L blocks, final LN, tied LM head over all
    padded columns, cross-entropy over the real vocabulary.

    Returns a cache dict holding 'loss' (mean over all tokens), 'losses'
    [B,T], 'logits', 'dlogits' (scaled by grad_scale, default 1/(B*T)) and the
    per-layer activations."""
    B, T = ids.shape
    if grad_scale is None:
        grad_scale = 1.0 / (B * T)
    cache = {"ids": ids, "layers": []}
    x = embed_forward(params["wte"], params["wpe"], ids)
    cache["x0"] = x
    for l in range(cfg.n_layer):
        x, c = block_forward(x, params, l, cfg)
        cache["layers"].append(c)
    hf, cache["lnf_mean"], cache["lnf_rstd"] = layernorm_forward(
        x, params["lnfw"], params["lnfb"], cfg.ln_eps)
    cache["x_final"] = x
    cache["lnf"] = hf
    logits = hf.reshape(B * T, -1) @ params["wte"].T
    cache["logits"] = logits
    if targets is not None:
        losses, dlogits = cross_entropy(logits, targets.reshape(-1), cfg.vocab, grad_scale)
        cache["losses"] = losses.reshape(B, T)
        cache["loss"] = losses.mean()
        cache["dlogits"] = dlogits
    return cache


def zero_grads(params):
    return {k: np.zeros_like(v) for k, v in params.items()}


def backward(params, cache, cfg: Config, grads=None):
    """Backward pass from the cached dlogits; accumulates into ``grads``
    (fresh zeros when None). The token table receives both the LM-head term
    and the embedding scatter (tied weights)."""
    if grads is None:
        grads = zero_grads(params)
    ids = cache["ids"]
    B, T = ids.shape
    dlogits = cache["dlogits"]
    hf = cache["lnf"].reshape(B * T, -1)
    grads["wte"] += dlogits.T @ hf
    dhf = (dlogits @ params["wte"]).reshape(B, T, -1)
    dx, dw, db = layernorm_backward(dhf, cache["x_final"], cache["lnf_mean"],
                                    cache["lnf_rstd"], params["lnfw"])
    grads["lnfw"] += dw
    grads["lnfb"] += db
    for l in reversed(range(cfg.n_layer)):
        dx = block_backward(dx, cache["layers"][l], params, l, cfg, grads)
    np.add.at(grads["wte"], ids.reshape(-1), dx.reshape(B * T, -1))
    grads["wpe"][:T] += dx.sum(axis=0)
    return grads


# ----------------------------------------------------------------------------
# Optimiser
# ----------------------------------------------------------------------------

def global_norm(grads):
    """Euclidean norm over every gradient element of every tensor."""
    return math.sqrt(sum(float(np.sum(np.asarray(g, np.float64) ** 2)) for g in grads.values()))


def clip_coefficient(norm, clip):
    """Global-norm clipping to ``clip``: scale gradients by clip/norm when the
    norm exceeds it, otherwise leave them alone."""
    return clip / norm if norm > clip else 1.0


def lr_at(cfg: Config, step: int) -> float:
    """Linear warmup over warmup_steps to lr_max, then cosine decay from lr_max
    to lr_min across the remaining steps (0-based step index)."""
    if step < cfg.warmup_steps:
        return cfg.lr_max * (step + 1) / cfg.warmup_steps
    frac = (step - cfg.warmup_steps) / (cfg.total_steps - cfg.warmup_steps)
    frac = min(max(frac, 0.0), 1.0)
    return cfg.lr_min + 0.5 * (1.0 + math.cos(math.pi * frac)) * (cfg.lr_max - cfg.lr_min)


def adamw_update(params, grads, m, v, step, lr, cfg: Config, coef=1.0):
    """Decoupled-weight-decay Adam with bias correction, applied in place.

    For each element: g' = coef*g; m = b1 m + (1-b1) g'; v = b2 v + (1-b2) g'^2;
    p -= lr * (m/(1-b1^t) / (sqrt(v/(1-b2^t)) + eps) + wd * p), with t = step+1
    and wd = weight_decay for two-dimensional weights, else 0."""
    t = step + 1
    for k in params:
        dt = params[k].dtype.type
        g = grads[k] * dt(coef)
        m[k] = dt(cfg.beta1) * m[k] + dt(1.0 - cfg.beta1) * g
        v[k] = dt(cfg.beta2) * v[k] + dt(1.0 - cfg.beta2) * g * g
        mhat = m[k] / dt(1.0 - cfg.beta1 ** t)
        vhat = v[k] / dt(1.0 - cfg.beta2 ** t)
        wd = cfg.weight_decay if k in DECAYED else 0.0
        params[k] = params[k] - dt(lr) * (mhat / (np.sqrt(vhat) + dt(cfg.adam_eps)) + dt(wd) * params[k])
    return params, m, v


def train_step(params, m, v, step, micro_batches, cfg: Config):
    """One optimiser step over a list of (ids, targets) micro-batches.

    The gradient is that of the mean loss over all micro-batch tokens; it is
    clipped to the global norm, then AdamW runs with the scheduled rate.
    Returns (mean of micro-batch losses, grad norm before clipping, lr)."""
    grads = zero_grads(params)
    n = len(micro_batches)
    losses = []
    for ids, tgt in micro_batches:
        B, T = ids.shape
        cache = forward(params, ids, tgt, cfg, grad_scale=1.0 / (B * T * n))
        losses.append(float(cache["loss"]))
        backward(params, cache, cfg, grads)
        del cache
    norm = global_norm(grads)
    coef = clip_coefficient(norm, cfg.grad_clip)
    lr = lr_at(cfg, step)
    adamw_update(params, grads, m, v, step, lr, cfg, coef)
    return sum(losses) / n, norm, lr
