"""The allocation-free optimizer entry point (gpt2_adamw_step_noalloc, whose
scratch is the library's static device array) against gpt2_adamw_step on
twin models: identical parameters, moments, bf16 copy, norm and rate, over
two calls in a row, the second on a smaller model."""
import numpy as np
import pytest

from paper_2609_28568_amd import synth
from tests.util import workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _pair(w, seed):
    from paper_2609_28568_amd import binding
    cfg = binding.make_config(w, dict(synth.OPTIM, warmup_steps=2, lr_max=1e-3))
    a, b = binding.GPT2(cfg, seed=seed), binding.GPT2(cfg, seed=seed)
    return a, b


def _step_both(w, seed, steps):
    a, b = _pair(w, seed)
    for step in range(steps):
        ids, tgt = synth.token_batch(w, seed=seed + step)
        for m in (a, b):
            m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
            m.backward()
        # the token-table scatter adds with atomics in no fixed order: both
        # optimizers get the same gradient bits
        b.flat("grads").copy_(a.flat("grads"))
        outs = []
        for m, noalloc in ((a, False), (b, True)):
            norm = torch.full((1,), -1.0, device="cuda")
            lr = m.adamw_step(step, norm, noalloc=noalloc)
            outs.append((lr, float(norm.item())))
        assert outs[0] == outs[1], (step, outs)
    torch.cuda.synchronize()
    for which in ("params", "m", "v"):
        assert torch.equal(a.flat(which), b.flat(which)), which
    assert torch.equal(a.flat_bf16(), b.flat_bf16())
    # the step did move the weights
    assert not np.array_equal(a.to_dict("params")["qkvw"], synth.init_params(w)["qkvw"])
    a.close()
    b.close()


def test_noalloc_adamw_matches_workspace_adamw_two_calls():
    # first a larger model, then a smaller one on the same GPU's array
    _step_both(workload("tiny", n_layer=2, d_model=256, n_head=4, d_ff=1024, vocab=1000, vocab_padded=1024,
                        max_seq_len=64, B=2, T=64), seed=81, steps=2)
    _step_both(workload("tiny", vocab=500, vocab_padded=512), seed=91, steps=2)
