"""GPU checks of the C-ABI boundary calls: the seeded initialisation against
the oracle's counter-based draw, per-position losses handed out by gpt2_loss,
and ids outside the vocabulary reported as a malformed request."""
import numpy as np
import pytest

import oracle
from oracle import init as oinit
from paper_2609_28568_amd import synth
from tests.util import LOSS_ATOL, oracle_config, workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _model(w, seed=None):
    from paper_2609_28568_amd import binding
    return binding.GPT2(binding.make_config(w, synth.OPTIM), seed=seed)


def _ulps32(a, b):
    """Distance in fp32 units in the last place (same-sign values)."""
    ia = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    ib = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    return np.abs(ia - ib)


def test_seeded_init_matches_oracle_small():
    """Every element of a small model (padded vocabulary) against the
    oracle's draw: Philox is integer work, so only the final fp64 transform
    and rounding can differ, by at most one fp32 unit in the last place."""
    w = workload("tiny", vocab=500, vocab_padded=512)
    ocfg = oracle_config(w)
    ref = oinit.seeded_params(ocfg, seed=1337)
    m = _model(w, seed=1337)
    got = m.to_dict("params")
    for k in oracle.KINDS:
        assert got[k].shape == ref[k].shape, k
        assert np.all(np.sign(got[k]) == np.sign(ref[k])), k
        assert _ulps32(got[k], ref[k]).max() <= 1, k
    assert np.all(got["wte"][500:] == 0.0)
    flat_bf16 = m.flat_bf16().float().cpu().numpy()
    flat = m.flat("params").cpu().numpy()
    assert np.array_equal(flat_bf16, synth.round_to_bf16(flat))
    assert not m.flat("m").any().item() and not m.flat("v").any().item()
    # a different seed gives different weights
    m2 = _model(w, seed=1338)
    assert not np.array_equal(m2.to_dict("params")["qkvw"], got["qkvw"])
    m.close()
    m2.close()


def test_seeded_init_full_size():
    """GPT-2 124M: exact zeros and ones over the whole buffer, 2^20 sampled
    elements against the oracle's draw, and the moments of every drawn kind."""
    w = workload("gpt2_124m")
    ocfg = oracle_config(w)
    m = _model(w, seed=1337)
    got = m.to_dict("params")
    L = w["n_layer"]
    for k in ("ln1b", "ln2b", "lnfb", "qkvb", "attprojb", "fcb", "fcprojb"):
        assert np.all(got[k] == 0.0), k
    for k in ("ln1w", "ln2w", "lnfw"):
        assert np.all(got[k] == 1.0), k
    assert np.all(got["wte"][w["vocab"]:] == 0.0)
    for k, std in (("wte", 0.02), ("wpe", 0.02), ("qkvw", 0.02), ("fcw", 0.02),
                   ("attprojw", 0.02 / np.sqrt(2 * L)), ("fcprojw", 0.02 / np.sqrt(2 * L))):
        x = (got[k][: w["vocab"]] if k == "wte" else got[k]).astype(np.float64).ravel()
        assert abs(x.mean()) < 5 * std / np.sqrt(x.size), k
        assert abs(x.std() / std - 1.0) < 5 * np.sqrt(0.5 / x.size), k
    flat = m.flat("params").cpu().numpy()
    idx = np.random.default_rng(3).integers(0, flat.size, 1 << 20)
    ref = oinit.seeded_values_at(ocfg, 1337, idx)
    assert _ulps32(flat[idx], ref).max() <= 1
    m.close()


def test_seeded_init_trains_like_caller_filled_weights():
    """A seeded model and a model given the same weights by the caller take
    bit-identical training steps."""
    w = workload("tiny", vocab=500, vocab_padded=512)
    ids, tgt = synth.token_batch(w, seed=5)
    a = _model(w, seed=99)
    b = _model(w)
    b.set_params(a.to_dict("params"))
    for m in (a, b):
        m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
        m.backward()
        m.adamw_step(0)
    torch.cuda.synchronize()
    assert torch.equal(a.flat("params"), b.flat("params"))
    assert a.loss() == b.loss()
    a.close()
    b.close()


def test_loss_hands_out_per_position_losses():
    w = workload("tiny", vocab=500, vocab_padded=512, B=3, T=29, max_seq_len=32)
    p = synth.perturb_params(synth.init_params(w, seed=51), seed=52)
    ids, tgt = synth.token_batch(w, seed=53)
    m = _model(w)
    m.set_params(p)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    tl = torch.full((w["B"] * w["T"],), -1.0, device="cuda")
    loss = m.loss(tl)
    got = tl.cpu().numpy()
    assert np.array_equal(got, m.activation("losses").cpu().numpy())
    cache = oracle.forward(p, ids, tgt, oracle_config(w))
    assert np.max(np.abs(got - cache["losses"].ravel())) < 0.05
    assert abs(loss - float(cache["loss"])) < LOSS_ATOL
    m.close()


@pytest.mark.parametrize("where", ["inputs", "targets", "both"])
def test_out_of_range_ids_are_reported_at_loss(where):
    """Ids outside [0, vocab) are a malformed request: nothing is read out of
    bounds, the loss call reports INVALID_ARG (the loss still written), and
    the next forward with valid ids reports nothing."""
    from paper_2609_28568_amd import binding
    w = workload("tiny", vocab=500, vocab_padded=512)
    ids, tgt = synth.token_batch(w, seed=61)
    bad_ids, bad_tgt = ids.copy(), tgt.copy()
    if where in ("inputs", "both"):
        bad_ids[0, 3] = w["vocab"]          # a padding row: still inside the table
        bad_ids[1, 0] = -7
    if where in ("targets", "both"):
        bad_tgt[1, 5] = 10 ** 6
    m = _model(w, seed=1)
    m.forward(torch.from_numpy(bad_ids), torch.from_numpy(bad_tgt))
    with pytest.raises(binding.LibError) as e:
        m.loss()
    assert e.value.status == binding.GPT2_ERR_INVALID_ARG
    msg = str(e.value)
    assert "outside [0, vocab)" in msg
    assert ("inputs" in msg) == (where in ("inputs", "both"))
    assert ("targets" in msg) == (where in ("targets", "both"))
    m.backward()   # the malformed step still runs to completion on the device
    torch.cuda.synchronize()
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    assert np.isfinite(m.loss())
    # the forward-only evaluation reports the same way
    with pytest.raises(binding.LibError):
        m.evaluate(torch.from_numpy(bad_ids), torch.from_numpy(bad_tgt))
    m.evaluate(torch.from_numpy(ids), torch.from_numpy(tgt))
    m.close()


def test_init_mode_is_validated():
    import ctypes
    from paper_2609_28568_amd import binding
    w = workload("tiny")
    cfg = binding.make_config(w, synth.OPTIM)
    s = binding.query_sizes(cfg)
    bufs = [torch.empty(int(n), dtype=torch.uint8, device="cuda")
            for n in (s.params_f32, s.grads_f32, s.adam_m, s.adam_v, s.params_bf16, s.activations, s.workspace)]
    b = binding.Buffers(*(t.data_ptr() for t in bufs))
    h = ctypes.c_void_p()
    st = binding.lib().gpt2_init(ctypes.byref(cfg), ctypes.byref(b), None, 0, 2, ctypes.byref(h))
    assert st == binding.GPT2_ERR_INVALID_ARG
    assert b"init_mode" in binding.lib().gpt2_last_error(None)
