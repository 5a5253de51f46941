"""The SwiGLU of the Qwen3-shaped adapter step inside the GEMM epilogues
(qwen3_set_fusion mode 1, the default: the gate|up projection writes the
pre-activation and silu(gate) up, the down projection's input gradient writes
the gate and up gradients) against the separate SwiGLU kernels (mode 0).
Both arrangements round the same values to bf16 and share the per-element
arithmetic, so the loss, every position's loss, every adapter gradient and
the adapters after one AdamW step must agree bit for bit. Each case fixes
which direction is fused: a projection with an adapter keeps the separate
kernel. Parity of the default arrangement with the oracle is in
test_gpu_qwen3.py and test_gpu_qwen3_fullsize.py."""
import numpy as np
import pytest

from paper_2609_28568_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = {
    # no MLP adapter: both directions fused; one 64-row tile minus a tail
    "qkvo": dict(lora_targets=("q", "k", "v", "o"), B=4, T=48),
    # gate|up adapted (forward kept separate), down not (backward fused);
    # four query heads per key/value head, rows past several tiles
    "gate_up_adapted": dict(n_head=8, n_kv_head=2, d_model=384, d_ff=640, vocab=640, max_seq_len=256, B=2,
                            T=160, loss_from=0.25, lora_rank=8, lora_alpha=16.0,
                            lora_targets=("q", "k", "v", "gate", "up")),
    # down adapted (backward kept separate), gate|up not (forward fused)
    "down_adapted": dict(lora_targets=("o", "down"), B=2, T=96),
}


def _run(w, base, lora, ids, tgt, mode):
    from paper_2609_28568_amd import qwen3_binding as qb
    m = qb.Qwen3(qb.make_config(w, synth.QWEN3_OPTIM))
    m.set_fusion("swiglu", mode)
    m.set_base(base)
    m.set_lora(lora)
    tl = torch.zeros(w["B"] * w["T"], device="cuda")
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    loss = m.loss(tl)
    m.backward()
    grads = m.flat("lora_grads").clone()
    m.adamw_step(0)
    after = m.flat("lora_f32").clone()
    torch.cuda.synchronize()
    m.close()
    return loss, tl, grads, after


def _compare(w, seed):
    base, lora = synth.init_qwen3(w, seed=seed, b_std=0.02, norm_jitter=0.1)
    ids, tgt = synth.token_batch(w, seed=seed + 1)
    fused = _run(w, base, lora, ids, tgt, 1)
    sep = _run(w, base, lora, ids, tgt, 0)
    assert fused[0] == sep[0]
    for name, a, b in zip(("per-position losses", "adapter gradients", "adapters after AdamW"), fused[1:], sep[1:]):
        assert torch.equal(a, b), name
    assert float(fused[2].abs().sum()) > 0.0   # the gradients are not trivially zero
    return fused


@pytest.mark.parametrize("case", list(CASES))
def test_fused_swiglu_is_bit_identical_to_separate_kernels(case):
    w = dict(synth.QWEN3_WORKLOADS["qwen3_tiny"])
    w.update(CASES[case])
    print(f"qwen3 fusion case {case}: {w}", flush=True)
    _compare(w, seed=71)


def test_fused_swiglu_bit_identical_at_full_size():
    """The benchmark's configuration (28 layers, SwiGLU 3072, B = 4,
    T = 2048, rank-16 q/k/v/o adapters): both directions fused."""
    w = dict(synth.QWEN3_WORKLOADS["qwen3_06b_lora"])
    print(f"qwen3 fusion full size: {w}", flush=True)
    loss, tl, grads, _ = _compare(w, seed=81)
    mf = int(np.floor(w["loss_from"] * w["T"]))
    tl = tl.view(w["B"], w["T"]).cpu().numpy()
    assert np.all(tl[:, :mf] == 0.0) and np.all(tl[:, mf:] > 0.0)
    assert np.isfinite(loss)
