"""Seeded synthetic inputs for the GPT-2 training step.

This module is the only code shared by the CPU oracle side (tests, the CPU
baseline) and the HIP side (binding, bench): it draws random numbers and
describes workload shapes. It performs none of the training step's arithmetic.

Streams: numpy PCG64 via ``default_rng([seed, k])`` with k = 0 for weights,
1 for token ids, 2 for upstream gradients / activations; the default seed is
1337, the run seed the paper states in its optimisation section.

Workload shapes follow the paper's model description (section "Model": 12
blocks, 12 heads, 768 channels, context 1024, vocabulary 50,257 padded to
50,304) plus small and single-block variants used as parity cases.
"""
from __future__ import annotations

import numpy as np

SEED = 1337
STREAM_WEIGHTS, STREAM_TOKENS, STREAM_GRADS = 0, 1, 2

# Shapes: n_layer, n_head, d_model, d_ff, vocab, vocab_padded, max_seq_len, B, T.
WORKLOADS = {
    # two-layer model used by the oracle pins and the small parity cases
    "tiny": dict(n_layer=2, n_head=4, d_model=64, d_ff=256, vocab=512,
                 vocab_padded=512, max_seq_len=32, B=2, T=32, grad_accum=1,
                 token_dist="uniform"),
    # one GPT-2 124M block in isolation (B=16, T=1024)
    "block124m": dict(n_layer=1, n_head=12, d_model=768, d_ff=3072, vocab=50257,
                      vocab_padded=50304, max_seq_len=1024, B=16, T=1024,
                      grad_accum=1, token_dist="zipf"),
    # the full GPT-2 124M micro-batch step (B=16, T=1024)
    "gpt2_124m": dict(n_layer=12, n_head=12, d_model=768, d_ff=3072, vocab=50257,
                      vocab_padded=50304, max_seq_len=1024, B=16, T=1024,
                      grad_accum=1, token_dist="zipf"),
    # gradient accumulation to 524,288 tokens per optimizer step
    "gpt2_124m_accum32": dict(n_layer=12, n_head=12, d_model=768, d_ff=3072,
                              vocab=50257, vocab_padded=50304, max_seq_len=1024,
                              B=16, T=1024, grad_accum=32, token_dist="zipf"),
}

# Optimiser hyper-parameters as the paper states them (section "Optimisation
# and precision"); lr_min is the floor of the accumulation workload's schedule.
OPTIM = dict(lr_max=6e-4, lr_min=6e-5, warmup_steps=700, total_steps=18865,
             beta1=0.9, beta2=0.95, adam_eps=1e-8, weight_decay=0.1, grad_clip=1.0,
             ln_eps=1e-5)


def rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([seed, stream])


def uniform_ids(g: np.random.Generator, shape, vocab: int) -> np.ndarray:
    return g.integers(0, vocab, size=shape, dtype=np.int64).astype(np.int32)


def zipf_ids(g: np.random.Generator, shape, vocab: int, s: float = 1.1) -> np.ndarray:
    """Zipf(s) over ranks 1..vocab mapped to id = rank - 1, by inverse CDF on
    the finite support."""
    ranks = np.arange(1, vocab + 1, dtype=np.float64)
    w = ranks ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    u = g.random(size=shape)
    ids = np.searchsorted(cdf, u, side="right")
    return np.minimum(ids, vocab - 1).astype(np.int32)


def token_batch(w: dict, seed: int = SEED, micro: int = 0):
    """Draw [B, T+1] ids; inputs are the first T, targets the last T.

    ``micro`` selects the micro-batch inside the token stream (each micro-batch
    is drawn from its own child stream so that micro-batches are independent
    of how many were drawn before)."""
    g = np.random.default_rng([seed, STREAM_TOKENS, micro])
    shape = (w["B"], w["T"] + 1)
    if w.get("token_dist", "uniform") == "zipf":
        ids = zipf_ids(g, shape, w["vocab"])
    else:
        ids = uniform_ids(g, shape, w["vocab"])
    return np.ascontiguousarray(ids[:, :-1]), np.ascontiguousarray(ids[:, 1:])


def init_params(w: dict, seed: int = SEED) -> dict:
    """Initial fp32 weights, drawn in a fixed order.

    2-D weights ~ N(0, 0.02); the two projections that write into the residual
    stream (attention output and MLP output) use 0.02/sqrt(2L); biases 0;
    LayerNorm gain 1 and shift 0; padding rows of the token table are 0.
    Shapes are stacked over layers and stored [out, in]."""
    g = rng(seed, STREAM_WEIGHTS)
    L, C, F = w["n_layer"], w["d_model"], w["d_ff"]
    V, Vp, Tm = w["vocab"], w["vocab_padded"], w["max_seq_len"]
    std, rstd = 0.02, 0.02 / np.sqrt(2.0 * L)

    def normal(shape, s):
        return (g.standard_normal(size=shape, dtype=np.float32) * np.float32(s)).astype(np.float32)

    wte = np.zeros((Vp, C), np.float32)
    wte[:V] = normal((V, C), std)
    p = {
        "wte": wte,
        "wpe": normal((Tm, C), std),
        "ln1w": np.ones((L, C), np.float32),
        "ln1b": np.zeros((L, C), np.float32),
        "qkvw": normal((L, 3 * C, C), std),
        "qkvb": np.zeros((L, 3 * C), np.float32),
        "attprojw": normal((L, C, C), rstd),
        "attprojb": np.zeros((L, C), np.float32),
        "ln2w": np.ones((L, C), np.float32),
        "ln2b": np.zeros((L, C), np.float32),
        "fcw": normal((L, F, C), std),
        "fcb": np.zeros((L, F), np.float32),
        "fcprojw": normal((L, C, F), rstd),
        "fcprojb": np.zeros((L, C), np.float32),
        "lnfw": np.ones((C,), np.float32),
        "lnfb": np.zeros((C,), np.float32),
    }
    return p


def perturb_params(p: dict, seed: int, scale: float = 0.05) -> dict:
    """Add small noise to the biases and LayerNorm parameters so that tests
    exercise them away from their trivial initial values."""
    g = rng(seed, 7)
    q = {k: v.copy() for k, v in p.items()}
    for k in ("ln1w", "ln1b", "qkvb", "attprojb", "ln2w", "ln2b", "fcb",
              "fcprojb", "lnfw", "lnfb"):
        q[k] = (q[k] + g.standard_normal(size=q[k].shape).astype(np.float32)
                * np.float32(scale)).astype(np.float32)
    return q


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16-representable value (ties to
    even), returned as fp32, so both sides receive identical inputs."""
    a = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (a >> 16) & 1
    r = ((a + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32)


def block_inputs(w: dict, seed: int = SEED):
    """Single-block workload: x ~ N(0,1) rounded to bf16 [B*T, C], upstream
    gradient ~ N(0, 1e-3) (standard deviation) rounded to bf16."""
    g = rng(seed, STREAM_GRADS)
    BT, C = w["B"] * w["T"], w["d_model"]
    x = round_to_bf16(g.standard_normal(size=(BT, C), dtype=np.float32))
    dy = round_to_bf16(g.standard_normal(size=(BT, C), dtype=np.float32) * np.float32(1e-3))
    return x, dy


# ---------------------------------------------------------------------------
# Qwen3-shaped adapter step (section "The clinical stage")
# ---------------------------------------------------------------------------

# The paper's base model is Qwen3 at 0.6 billion parameters; its shape is the
# public configuration of that model. The benchmark geometry is four
# sequences of 2048 tokens, adapters on the attention projections q, k, v, o.
QWEN3_WORKLOADS = {
    # two layers, several GEMM and attention tiles, a ragged sequence tail
    "qwen3_tiny": dict(n_layer=2, d_model=256, n_head=4, n_kv_head=2, head_dim=128, d_ff=512, vocab=1024,
                       max_seq_len=128, B=2, T=96, lora_rank=16, lora_alpha=32.0,
                       lora_targets=("q", "k", "v", "o", "gate", "up", "down"), loss_from=0.5,
                       token_dist="zipf"),
    "qwen3_06b_lora": dict(n_layer=28, d_model=1024, n_head=16, n_kv_head=8, head_dim=128, d_ff=3072,
                           vocab=151936, max_seq_len=2048, B=4, T=2048, lora_rank=16, lora_alpha=32.0,
                           lora_targets=("q", "k", "v", "o"), loss_from=0.5, token_dist="zipf"),
}

# Adapter optimiser: the clinical stage names AdamW without values, so the one
# AdamW recipe the paper states (section "Optimisation and precision": betas
# 0.9/0.95, eps 1e-8, decay 0.1 on two-dimensional tensors, which every
# adapter tensor is, global-norm clip 1.0) applies; the rate is the one free
# choice.
QWEN3_OPTIM = dict(lr=2e-4, beta1=0.9, beta2=0.95, adam_eps=1e-8, weight_decay=0.1, grad_clip=1.0,
                   rms_eps=1e-6, rope_theta=1e6)


def _qwen3_dims(w: dict) -> dict:
    C, F = w["d_model"], w["d_ff"]
    qd, kvd = w["n_head"] * w["head_dim"], w["n_kv_head"] * w["head_dim"]
    return {"q": (C, qd), "k": (C, kvd), "v": (C, kvd), "o": (qd, C), "gate": (C, F), "up": (C, F),
            "down": (F, C)}


def init_qwen3(w: dict, seed: int = SEED, std: float = 0.02, b_std: float = 0.0, norm_jitter: float = 0.0):
    """Frozen base parameters (bf16-representable fp32) and fp32 adapters,
    drawn in a fixed order, named per projection as [out, in] stacked over
    layers: matrices ~ N(0, std); RMSNorm gains 1 (+ N(0, norm_jitter));
    adapter A ~ N(0, std) [L, r, in]; adapter B ~ N(0, b_std) [L, out, r]
    (zero by default, the usual adapter initialisation)."""
    g = rng(seed, STREAM_WEIGHTS)
    L, C, V, hd, r = w["n_layer"], w["d_model"], w["vocab"], w["head_dim"], w["lora_rank"]
    dims = _qwen3_dims(w)

    def normal(shape, s):
        return (g.standard_normal(size=shape, dtype=np.float32) * np.float32(s)).astype(np.float32)

    def gain(shape):
        return (np.ones(shape, np.float32) + normal(shape, norm_jitter)).astype(np.float32)

    base = {"embed": normal((V, C), std), "in_norm": gain((L, C)), "q_norm": gain((L, hd)),
            "k_norm": gain((L, hd)), "post_norm": gain((L, C)), "final_norm": gain((C,))}
    for p in ("q", "k", "v", "o", "gate", "up", "down"):
        i, o = dims[p]
        base[p] = normal((L, o, i), std)
    base = {k: round_to_bf16(v) for k, v in base.items()}
    lora = {}
    for p in w["lora_targets"]:
        i, o = dims[p]
        lora[p + "_A"] = normal((L, r, i), std)
        lora[p + "_B"] = normal((L, o, r), b_std) if b_std > 0 else np.zeros((L, o, r), np.float32)
    return base, lora
