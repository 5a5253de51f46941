"""GPU checks of the alternative kernel arrangements (gpt2_set_fusion).

The fused residual-and-pre-norm kernel (mode 1) is gated the way the paper
gates its own (section "Speed", table of levers): its residual sums must equal
the composed addition (mode 2: an addition kernel, then the LayerNorm)
exactly, and so, since the normalisation reads those sums, must everything
after them. Both also meet the oracle's tolerances."""
import numpy as np
import pytest

import oracle
from paper_2609_28568_amd import synth
from tests.util import LOSS_ATOL, REL_L2, oracle_config, rel_l2, workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = {
    "tiny_ragged": dict(vocab=500, vocab_padded=512, B=3, T=29, max_seq_len=32),
    "wide_c384": dict(n_layer=2, n_head=6, d_model=384, d_ff=1536, vocab=1000, vocab_padded=1024,
                      max_seq_len=160, B=2, T=150),
}
PER_LAYER = ("residual", "ln1", "ln1_mean", "ln1_rstd", "qkv", "att", "att_lse", "x_mid", "ln2", "ln2_mean",
             "ln2_rstd", "fc", "gelu")


def _run(w, p, ids, tgt, mode):
    from paper_2609_28568_amd import binding
    m = binding.GPT2(binding.make_config(w, synth.OPTIM))
    m.set_params(p)
    m.set_fusion("residual_norm", mode)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    acts = {}
    for name in PER_LAYER:
        n_l = w["n_layer"] + (1 if name == "residual" else 0)
        acts[name] = [m.activation(name, l).clone() for l in range(n_l)]
    for name in ("lnf", "lnf_mean", "lnf_rstd", "losses"):
        acts[name] = [m.activation(name).clone()]
    loss = m.loss()
    m.backward()
    g = m.to_dict("grads")
    m.close()
    return acts, loss, g


def _case(name, **over):
    w = workload("tiny", **dict(CASES[name], **over)) if name in CASES else workload(name, **over)
    p = synth.perturb_params(synth.init_params(w, seed=101), seed=102)
    ids, tgt = synth.token_batch(w, seed=103)
    return w, p, ids, tgt


@pytest.mark.parametrize("case", list(CASES))
def test_fused_residual_norm_is_bit_identical_to_composed(case):
    w, p, ids, tgt = _case(case)
    fused, loss_f, g_f = _run(w, p, ids, tgt, 1)
    comp, loss_c, g_c = _run(w, p, ids, tgt, 2)
    for name in fused:
        for l, (a, b) in enumerate(zip(fused[name], comp[name])):
            assert torch.equal(a, b), (name, l)
    assert loss_f == loss_c


@pytest.mark.parametrize("mode", [1, 2])
@pytest.mark.parametrize("case", list(CASES))
def test_fused_residual_norm_meets_the_oracle(case, mode):
    w, p, ids, tgt = _case(case)
    _, loss, g = _run(w, p, ids, tgt, mode)
    ocfg = oracle_config(w)
    cache = oracle.forward(p, ids, tgt, ocfg)
    ref = oracle.backward(p, cache, ocfg)
    assert abs(loss - float(cache["loss"])) < LOSS_ATOL
    for k in oracle.KINDS:
        assert rel_l2(g[k], ref[k]) < REL_L2, k


def test_fused_residual_norm_bit_identical_at_full_size():
    """The gate at GPT-2 124M, B=16, T=1024, in the benchmark's launch
    configuration: every saved activation of all 12 blocks."""
    w = workload("gpt2_124m")
    p = synth.init_params(w)
    ids, tgt = synth.token_batch(w)
    from paper_2609_28568_amd import binding
    m = binding.GPT2(binding.make_config(w, synth.OPTIM))
    m.set_params(p)
    out = {}
    for mode in (1, 2):
        m.set_fusion("residual_norm", mode)
        m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
        loss = m.loss()
        h = {}
        for name in PER_LAYER:
            n_l = w["n_layer"] + (1 if name == "residual" else 0)
            h[name] = [m.activation(name, l).clone() for l in range(n_l)]
        h["lnf"] = [m.activation("lnf").clone()]
        h["losses"] = [m.activation("losses").clone()]
        out[mode] = (loss, h)
    m.close()
    assert out[1][0] == out[2][0]
    for name, xs in out[1][1].items():
        for l, (a, b) in enumerate(zip(xs, out[2][1][name])):
            assert torch.equal(a, b), (name, l)


def _head_ce_run(w, p, ids, tgt, mode):
    from paper_2609_28568_amd import binding
    m = binding.GPT2(binding.make_config(w, synth.OPTIM))
    m.set_params(p)
    m.set_fusion("head_ce", mode)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    loss = m.loss()
    losses = m.activation("losses").clone()
    dlogits = m.activation("logits").clone()
    m.backward()
    g = m.to_dict("grads")
    ev_losses = torch.zeros_like(losses)
    ev = m.evaluate(torch.from_numpy(ids), torch.from_numpy(tgt), ev_losses)
    m.close()
    return dict(loss=loss, losses=losses, dlogits=dlogits, grads=g, ev=ev, ev_losses=ev_losses)


@pytest.mark.parametrize("case", list(CASES) + ["single_token"])
def test_two_pass_head_cross_entropy_meets_the_oracle(case):
    """Head + cross-entropy without stored logits (mode 1): loss, per-token
    losses and all gradients against the oracle; padding columns of dlogits
    exactly 0; the forward-only evaluation gives the training forward's
    per-token losses bit for bit."""
    if case == "single_token":
        w = workload("tiny", B=5, T=1)
        p = synth.perturb_params(synth.init_params(w, seed=101), seed=102)
        ids, tgt = synth.token_batch(w, seed=103)
    else:
        w, p, ids, tgt = _case(case)
    r = _head_ce_run(w, p, ids, tgt, 1)
    ocfg = oracle_config(w)
    cache = oracle.forward(p, ids, tgt, ocfg)
    ref = oracle.backward(p, cache, ocfg)
    assert abs(r["loss"] - float(cache["loss"])) < LOSS_ATOL
    got = r["losses"].cpu().numpy()
    assert np.max(np.abs(got - cache["losses"].ravel())) < 5 * LOSS_ATOL
    assert rel_l2(got, cache["losses"].ravel()) < REL_L2
    Vp, V = w["vocab_padded"], w["vocab"]
    dl = r["dlogits"].view(-1, Vp)
    assert int(torch.count_nonzero(dl[:, V:]).item()) == 0
    assert rel_l2(dl.float().cpu().numpy(), cache["dlogits"]) < REL_L2
    for k in oracle.KINDS:
        assert rel_l2(r["grads"][k], ref[k]) < REL_L2, k
    assert torch.equal(r["ev_losses"], r["losses"])
    assert r["ev"] == r["loss"]


def test_two_pass_head_cross_entropy_full_size():
    """GPT-2 124M, the benchmark's batch: the two arrangements' losses,
    dlogits and gradients agree (the second works from fp32 logits, the first
    from bf16 ones), and the padding columns are exactly 0."""
    w = workload("gpt2_124m")
    p = synth.init_params(w)
    ids, tgt = synth.token_batch(w)
    a = _head_ce_run(w, p, ids, tgt, 0)
    b = _head_ce_run(w, p, ids, tgt, 1)
    V, Vp = w["vocab"], w["vocab_padded"]
    assert abs(a["loss"] - b["loss"]) < 1e-3
    assert float((a["losses"] - b["losses"]).abs().max()) < 2e-2
    dla, dlb = a["dlogits"].view(-1, Vp), b["dlogits"].view(-1, Vp)
    assert int(torch.count_nonzero(dlb[:, V:]).item()) == 0
    e = float(torch.linalg.norm((dla.float() - dlb.float())) / torch.linalg.norm(dla.float()))
    print(f"head_ce full size: dlogits rel_l2 {e:.2e}, loss {a['loss']:.5f} vs {b['loss']:.5f}")
    assert e < 1e-2
    for k in oracle.KINDS:
        assert rel_l2(b["grads"][k], a["grads"][k]) < 1e-2, k
    assert torch.equal(b["ev_losses"], b["losses"])
