"""Pins for the Qwen3-shaped adapter-step oracle (CPU only).

Each check ties the oracle to something other than itself: the paper's
printed adapter count, closed forms, an independent fp64 implementation on
torch library primitives with autograd gradients, and central finite
differences.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import qwen3 as q3

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "paper_figures.json")

QWEN3_06B = dict(n_layer=28, d_model=1024, n_head=16, n_kv_head=8, head_dim=128, d_ff=3072, vocab=151936,
                 max_seq_len=2048)
TINY = dict(n_layer=2, d_model=32, n_head=4, n_kv_head=2, head_dim=8, d_ff=48, vocab=50, max_seq_len=16,
            rope_theta=100.0, lora_rank=4, lora_alpha=8.0, lora_targets=q3.PROJECTIONS, loss_from=0.5)


def _params(cfg, seed, b_scale=0.05, dtype=np.float64):
    rng = np.random.default_rng(seed)
    base = {k: (rng.standard_normal(s) * 0.2).astype(dtype) for k, s in q3.base_shapes(cfg).items()}
    for k in ("in_norm", "q_norm", "k_norm", "post_norm", "final_norm"):
        base[k] = (1.0 + 0.1 * rng.standard_normal(q3.base_shapes(cfg)[k])).astype(dtype)
    lora = {}
    for k, s in q3.lora_shapes(cfg).items():
        scale = 0.2 if k.endswith("_A") else b_scale
        lora[k] = (rng.standard_normal(s) * scale).astype(dtype)
    return base, lora


def _batch(cfg, B, T, seed):
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, cfg.vocab, size=(B, T + 1))
    return ids[:, :-1].copy(), ids[:, 1:].copy()


def test_adapter_counts_match_the_paper_and_the_config():
    figures = json.load(open(GOLDEN))
    cfg7 = q3.Qwen3Config.from_dict(dict(QWEN3_06B, lora_targets=q3.PROJECTIONS))
    # seven projections per layer, rank 16 ("The clinical stage")
    assert (figures["clinical_lora_rank"], figures["clinical_lora_alpha"]) == (16, 32)
    assert q3.lora_param_count(cfg7) == figures["clinical_trainable_params"] == 10_092_544
    cfg4 = q3.Qwen3Config.from_dict(QWEN3_06B)
    assert q3.lora_param_count(cfg4) == 28 * 16 * (3072 + 2048 + 2048 + 3072) == 4_587_520
    assert cfg7.lora_scale == 32.0 / math.sqrt(16) == 8.0


def test_rope_is_a_rotation_depending_on_relative_position():
    rng = np.random.default_rng(1)
    T, hd = 20, 16
    cos, sin = q3.rope_tables(T, hd, 1e4, np.float64)
    x = rng.standard_normal((T, hd))
    y = q3.rope_forward(x, cos, sin)
    np.testing.assert_allclose(np.linalg.norm(y, axis=-1), np.linalg.norm(x, axis=-1), rtol=1e-12)
    # <R(m) a, R(n) b> depends only on m - n
    a, b = rng.standard_normal(hd), rng.standard_normal(hd)
    ra = q3.rope_forward(np.broadcast_to(a, (T, hd)), cos, sin)
    rb = q3.rope_forward(np.broadcast_to(b, (T, hd)), cos, sin)
    d1 = ra[7] @ rb[3]
    d2 = ra[15] @ rb[11]
    assert abs(d1 - d2) < 1e-10
    # position 0 is the identity, and the backward is the inverse rotation
    np.testing.assert_allclose(y[0], x[0], rtol=0, atol=0)
    np.testing.assert_allclose(q3.rope_backward(y, cos, sin), x, atol=1e-12)


def test_zero_B_adapters_leave_the_base_model_unchanged():
    cfg = q3.Qwen3Config.from_dict(TINY)
    base, lora = _params(cfg, 3)
    for k in lora:
        if k.endswith("_B"):
            lora[k][:] = 0.0
    ids, tgt = _batch(cfg, 2, 12, 4)
    with_ad = q3.forward(base, lora, ids, tgt, cfg)
    without = q3.forward(base, None, ids, tgt, cfg)
    assert with_ad["loss"] == without["loss"]
    g = q3.backward(base, lora, with_ad, cfg)
    # dA = s (dy B)^T x vanishes with B = 0; dB does not
    for k in g:
        if k.endswith("_A"):
            assert np.all(g[k] == 0.0)
    assert any(np.abs(g[k]).max() > 0 for k in g if k.endswith("_B"))


def _torch_reference(base, lora, ids, tgt, cfg):
    """Independent fp64 model on torch primitives; returns (loss, grads)."""
    t = {k: torch.tensor(v, dtype=torch.float64) for k, v in base.items()}
    tl = {k: torch.tensor(v, dtype=torch.float64, requires_grad=True) for k, v in lora.items()}
    s = cfg.lora_alpha / math.sqrt(cfg.lora_rank)
    B, T = ids.shape
    H, Hkv, hd = cfg.n_head, cfg.n_kv_head, cfg.head_dim
    pos = torch.arange(T, dtype=torch.float64)
    inv = cfg.rope_theta ** (-torch.arange(0, hd, 2, dtype=torch.float64) / hd)
    ang = pos[:, None] * inv[None, :]
    rot = torch.polar(torch.ones_like(ang), ang)          # e^{i angle}, [T, hd/2]

    def rope(x):                                           # pairs (i, i + hd/2) as complex numbers
        c = torch.complex(x[..., : hd // 2], x[..., hd // 2:]) * rot
        return torch.cat([c.real, c.imag], dim=-1)

    def lin(x, name, l):
        y = x @ t[name][l].T
        if name + "_A" in tl:
            y = y + s * ((x @ tl[name + "_A"][l].T) @ tl[name + "_B"][l].T)
        return y

    x = t["embed"][torch.tensor(ids)]
    for l in range(cfg.n_layer):
        h = F.rms_norm(x, (cfg.d_model,), t["in_norm"][l], eps=cfg.rms_eps)
        qh = lin(h, "q", l).view(B, T, H, hd).transpose(1, 2)
        kh = lin(h, "k", l).view(B, T, Hkv, hd).transpose(1, 2)
        vh = lin(h, "v", l).view(B, T, Hkv, hd).transpose(1, 2)
        qh = rope(F.rms_norm(qh, (hd,), t["q_norm"][l], eps=cfg.rms_eps))
        kh = rope(F.rms_norm(kh, (hd,), t["k_norm"][l], eps=cfg.rms_eps))
        a = F.scaled_dot_product_attention(qh, kh, vh, is_causal=True, enable_gqa=True)
        x = x + lin(a.transpose(1, 2).reshape(B, T, H * hd), "o", l)
        h2 = F.rms_norm(x, (cfg.d_model,), t["post_norm"][l], eps=cfg.rms_eps)
        x = x + lin(F.silu(lin(h2, "gate", l)) * lin(h2, "up", l), "down", l)
    xf = F.rms_norm(x, (cfg.d_model,), t["final_norm"], eps=cfg.rms_eps)
    logits = xf @ t["embed"].T
    target = torch.tensor(tgt).clone()
    target[:, : int(math.floor(cfg.loss_from * T))] = -100
    loss = F.cross_entropy(logits.reshape(-1, cfg.vocab), target.reshape(-1), ignore_index=-100)
    loss.backward()
    return loss.item(), {k: v.grad.numpy() for k, v in tl.items()}


@pytest.mark.parametrize("targets", [q3.PROJECTIONS, ("q", "k", "v", "o")])
def test_loss_and_adapter_gradients_match_torch_autograd(targets):
    cfg = q3.Qwen3Config.from_dict(dict(TINY, lora_targets=targets))
    base, lora = _params(cfg, 5)
    ids, tgt = _batch(cfg, 2, 12, 6)
    c = q3.forward(base, lora, ids, tgt, cfg)
    g = q3.backward(base, lora, c, cfg)
    ref_loss, ref_g = _torch_reference(base, lora, ids, tgt, cfg)
    assert abs(c["loss"] - ref_loss) <= 1e-10 * abs(ref_loss)
    for k in lora:
        err = np.linalg.norm(g[k] - ref_g[k]) / np.linalg.norm(ref_g[k])
        assert err < 1e-10, (k, err)


def test_adapter_gradients_match_central_differences():
    cfg = q3.Qwen3Config.from_dict(TINY)
    base, lora = _params(cfg, 7)
    ids, tgt = _batch(cfg, 2, 10, 8)
    g = q3.backward(base, lora, q3.forward(base, lora, ids, tgt, cfg), cfg)
    rng = np.random.default_rng(9)
    h = 1e-5
    for k in lora:
        for _ in range(4):
            idx = tuple(rng.integers(0, n) for n in lora[k].shape)
            old = lora[k][idx]
            lora[k][idx] = old + h
            lp = q3.forward(base, lora, ids, tgt, cfg)["loss"]
            lora[k][idx] = old - h
            lm = q3.forward(base, lora, ids, tgt, cfg)["loss"]
            lora[k][idx] = old
            fd = (lp - lm) / (2 * h)
            assert abs(fd - g[k][idx]) <= 1e-6 * max(1e-3, abs(fd)), (k, idx, fd, g[k][idx])


def test_loss_counts_only_the_last_half_of_each_sequence():
    cfg = q3.Qwen3Config.from_dict(TINY)
    base, lora = _params(cfg, 11)
    ids, tgt = _batch(cfg, 2, 12, 12)
    c = q3.forward(base, lora, ids, tgt, cfg)
    assert np.all(c["losses"][:, :6] == 0.0) and np.all(c["losses"][:, 6:] > 0.0)
    assert np.all(c["dlogits"][:, :6] == 0.0)
    # changing a target in the unmasked half changes nothing
    tgt2 = tgt.copy()
    tgt2[:, :6] = (tgt2[:, :6] + 1) % cfg.vocab
    assert q3.forward(base, lora, ids, tgt2, cfg)["loss"] == c["loss"]
    # every masked dlogits row sums to zero
    np.testing.assert_allclose(c["dlogits"][:, 6:].sum(axis=-1), 0.0, atol=1e-15)


def test_adapter_adamw_first_step_closed_form():
    cfg = q3.Qwen3Config.from_dict(dict(TINY, lr=1e-3))
    lora = {"q_A": np.array([[1.0, -2.0]])}
    grads = {"q_A": np.array([[0.5, -0.25]])}
    m = {"q_A": np.zeros((1, 2))}
    v = {"q_A": np.zeros((1, 2))}
    q3.adamw_step(lora, grads, m, v, 0, cfg)
    # step 1: m_hat = g, v_hat = g^2, so the update is lr * (g / (|g| + eps)
    # + decay * p), the decay 0.1 of the paper's optimisation section
    assert cfg.weight_decay == 0.1
    expect = np.array([[1.0 - 1e-3 * (0.5 / (0.5 + 1e-8) + 0.1 * 1.0),
                        -2.0 + 1e-3 * (0.25 / (0.25 + 1e-8) + 0.1 * 2.0)]])
    np.testing.assert_allclose(lora["q_A"], expect, rtol=0, atol=1e-15)


@pytest.mark.parametrize("clip", [1e-3, 1e9])
def test_train_step_clips_then_takes_the_closed_form_first_step(clip):
    """First step from zero moments: m_hat = c g and v_hat = (c g)^2, so every
    adapter element moves by lr (c g / (|c g| + eps) + decay p) with
    c = clip / ||g|| when the norm over all adapter elements exceeds the clip,
    else c = 1."""
    cfg = q3.Qwen3Config.from_dict(dict(TINY, grad_clip=clip, lr=1e-3))
    base, lora = _params(cfg, 13)
    ids, tgt = _batch(cfg, 2, 10, 14)
    g = q3.backward(base, lora, q3.forward(base, lora, ids, tgt, cfg), cfg)
    g.pop("dx0")
    norm = np.linalg.norm(np.concatenate([g[k].ravel() for k in sorted(g)]))
    c = clip / norm if norm > clip else 1.0
    assert (c < 1.0) == (clip < 1.0)
    before = {k: v.copy() for k, v in lora.items()}
    m = {k: np.zeros_like(v) for k, v in lora.items()}
    v = {k: np.zeros_like(x) for k, x in lora.items()}
    loss, got_norm = q3.train_step(base, lora, m, v, 0, ids, tgt, cfg)
    assert abs(got_norm - norm) <= 1e-12 * norm
    for k in lora:
        step = 1e-3 * (c * g[k] / (np.abs(c * g[k]) + 1e-8) + cfg.weight_decay * before[k])
        np.testing.assert_allclose(before[k] - lora[k], step, rtol=1e-9, atol=1e-15)


def test_adapter_adamw_hand_steps():
    """Three steps against hand arithmetic with betas (0.9, 0.999): from t=2 on
    the moments' history matters, so wrong or swapped betas or a wrong bias
    correction change the result."""
    gold = json.load(open(os.path.join(os.path.dirname(GOLDEN), "adamw_adapter_hand.json")))
    cfg = q3.Qwen3Config.from_dict(dict(TINY, lr=gold["lr"], beta1=gold["beta1"], beta2=gold["beta2"],
                                        adam_eps=gold["eps"], weight_decay=0.0))
    lora = {"q_A": np.array([[gold["p0"]]])}
    m = {"q_A": np.zeros((1, 1))}
    v = {"q_A": np.zeros((1, 1))}
    for step, (g, want) in enumerate(zip(gold["grads"], gold["p_after"])):
        q3.adamw_step(lora, {"q_A": np.array([[g]])}, m, v, step, cfg)
        assert abs(float(lora["q_A"][0, 0]) - want) <= 1e-15, (step, float(lora["q_A"][0, 0]), want)


@pytest.mark.parametrize("betas,wd", [((0.9, 0.999), 0.0), ((0.9, 0.95), 0.0), ((0.8, 0.99), 0.1)])
def test_adapter_adamw_matches_torch_over_steps(betas, wd):
    """Five steps of the oracle's AdamW against torch.optim.AdamW in fp64
    (decoupled decay, bias correction), with gradients that change sign."""
    cfg = q3.Qwen3Config.from_dict(dict(TINY, lr=3e-3, beta1=betas[0], beta2=betas[1], adam_eps=1e-8,
                                        weight_decay=wd))
    rng = np.random.default_rng(21)
    lora = {"q_A": rng.standard_normal((3, 5)), "o_B": rng.standard_normal((4, 2))}
    tp = {k: torch.tensor(x.copy(), requires_grad=True) for k, x in lora.items()}
    opt = torch.optim.AdamW(list(tp.values()), lr=3e-3, betas=betas, eps=1e-8, weight_decay=wd, foreach=False)
    m = {k: np.zeros_like(x) for k, x in lora.items()}
    v = {k: np.zeros_like(x) for k, x in lora.items()}
    for step in range(5):
        grads = {k: rng.standard_normal(x.shape) * (0.5 + step) for k, x in lora.items()}
        for k in lora:
            tp[k].grad = torch.tensor(grads[k])
        opt.step()
        q3.adamw_step(lora, grads, m, v, step, cfg)
        for k in lora:
            np.testing.assert_allclose(lora[k], tp[k].detach().numpy(), rtol=1e-13, atol=1e-15)
