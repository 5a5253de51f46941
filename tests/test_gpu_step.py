"""GPU parity of the whole training step against the CPU oracle, on small
models the oracle runs in seconds: loss, per-token losses, saved activations,
all parameter gradients, the optimizer update and exact index handling."""
import numpy as np
import pytest

import oracle
from paper_2609_28568_amd import synth
from tests.util import LOSS_ATOL, REL_L2, oracle_config, rel_l2, workload

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _model(w, optim=None):
    from paper_2609_28568_amd import binding
    o = dict(synth.OPTIM)
    o.update(optim or {})
    return binding.GPT2(binding.make_config(w, o))


def _np(t):
    return t.float().cpu().numpy()


def _oracle_acts(cache, name, l):
    if name == "residual":
        L = len(cache["layers"])
        if l == 0:
            return cache["x0"]
        return cache["x_final"] if l == L else cache["layers"][l - 1]["x_out"]
    if name in ("lnf", "logits"):
        return cache[name]
    return cache["layers"][l][name]


# small shapes: several GEMM/attention tiles, ragged sequence and vocabulary tails
CASES = {
    "tiny": dict(),
    "tiny_ragged": dict(vocab=500, vocab_padded=512, B=3, T=29, max_seq_len=32),
    "wide_hd64": dict(n_layer=2, n_head=4, d_model=256, d_ff=1024, vocab=1000, vocab_padded=1024,
                      max_seq_len=160, B=2, T=150),
    # widths that are multiples of 192 with 300 token rows: the input
    # gradients run on the eight-wave 256-row tiles, the second row tile
    # ragged
    "wide_c384": dict(n_layer=2, n_head=6, d_model=384, d_ff=1536, vocab=1000, vocab_padded=1024,
                      max_seq_len=160, B=2, T=150),
    # degenerate: one-token sequences (attention over a single key, 5 rows in
    # every product, token contractions far shorter than one k-tile)
    "single_token": dict(B=5, T=1),
    # the 124M model's block widths (12 layers, 768 wide) on 2 x 64 tokens:
    # the grouped weight-gradient launch has the 124M step's 2,304 tiles, so
    # its last half round (the MLP-down weight gradients of layers 8-11) takes
    # the token contraction split in two, checked here element by element
    "blocks124m_short": dict(n_layer=12, n_head=12, d_model=768, d_ff=3072, vocab=512, vocab_padded=512,
                             max_seq_len=64, B=2, T=64),
}


@pytest.fixture(scope="module", params=list(CASES))
def step_case(request):
    w = workload("tiny", **CASES[request.param])
    params = synth.perturb_params(synth.init_params(w, seed=21), seed=22)
    ids, tgt = synth.token_batch(w, seed=23)
    ocfg = oracle_config(w)
    cache = oracle.forward(params, ids, tgt, ocfg)
    grads = oracle.backward(params, cache, ocfg)
    m = _model(w)
    m.set_params(params)
    tids, ttgt = torch.from_numpy(ids), torch.from_numpy(tgt)
    # forward without targets keeps the logits for inspection
    m.forward(tids, None)
    logits = _np(m.activation("logits"))
    m.forward(tids, ttgt)
    acts = {}
    for name in ("residual", "ln1", "qkv", "att", "x_mid", "ln2", "fc", "gelu"):
        n_l = w["n_layer"] + (1 if name == "residual" else 0)
        acts[name] = [_np(m.activation(name, l)) for l in range(n_l)]
    acts["lnf"] = [_np(m.activation("lnf"))]
    loss = m.loss()
    losses = _np(m.activation("losses"))
    m.backward(accumulate=False)
    g = m.to_dict("grads")
    torch.cuda.synchronize()
    yield dict(w=w, params=params, ids=ids, tgt=tgt, cache=cache, grads=grads, m=m, logits=logits,
               acts=acts, loss=loss, losses=losses, gpu_grads=g)
    m.close()


def test_loss(step_case):
    c = step_case
    print("loss gpu", c["loss"], "oracle", float(c["cache"]["loss"]))
    assert abs(c["loss"] - float(c["cache"]["loss"])) < LOSS_ATOL
    assert np.max(np.abs(c["losses"] - c["cache"]["losses"].ravel())) < 5 * LOSS_ATOL


def test_activations(step_case):
    c = step_case
    for name, per_layer in c["acts"].items():
        for l, a in enumerate(per_layer):
            ref = _oracle_acts(c["cache"], name, l).reshape(a.shape)
            e = rel_l2(a, ref)
            print(f"{name}[{l}] rel_l2 {e:.2e}")
            assert e < REL_L2, (name, l, e)
    e = rel_l2(c["logits"], c["cache"]["logits"])
    print(f"logits rel_l2 {e:.2e}")
    assert e < REL_L2


@pytest.mark.parametrize("kind", oracle.KINDS)
def test_gradients(step_case, kind):
    c = step_case
    got, ref = c["gpu_grads"][kind], c["grads"][kind]
    if kind == "wpe":
        T = c["ids"].shape[1]
        assert np.all(got[T:] == 0.0)
    # per tensor: each layer slice of a stacked kind is one of the 148 tensors
    slices = [(got, ref)] if got.ndim <= 1 or kind in ("wte", "wpe") else list(zip(got, ref))
    for i, (a, b) in enumerate(slices):
        e = rel_l2(a, b)
        print(f"{kind}[{i}] rel_l2 {e:.2e}")
        assert e < REL_L2, (kind, i, e)


def test_padding_rows_and_columns_exactly_zero(step_case):
    c = step_case
    V = c["w"]["vocab"]
    assert np.all(c["gpu_grads"]["wte"][V:] == 0.0)
    dl = _np(c["m"].activation("logits")).reshape(-1, c["w"]["vocab_padded"])
    assert np.all(dl[:, V:] == 0.0)


def test_embedding_backward_rows_touched_exactly():
    """The embedding backward in isolation: the set of token-table rows with a
    nonzero gradient is exactly the set of input ids, each row equals the sum
    of its positions' gradients, and the position table gets the batch sum."""
    w = workload("tiny", vocab=500, vocab_padded=512, B=3, T=29)
    m = _model(w)
    m.set_params(synth.init_params(w))
    ids, _ = synth.token_batch(w, seed=51)
    g = np.random.default_rng(52)
    dx = synth.round_to_bf16(g.standard_normal((ids.size, w["d_model"])).astype(np.float32) + 3.0)
    tdx = torch.from_numpy(dx).to("cuda").to(torch.bfloat16)
    m.embedding_backward(torch.from_numpy(ids), tdx)
    got = m.to_dict("grads")
    rows = set(np.where(np.any(got["wte"] != 0.0, axis=1))[0].tolist())
    assert rows == set(np.unique(ids).tolist())
    ref = np.zeros_like(got["wte"], dtype=np.float64)
    np.add.at(ref, ids.ravel(), dx.astype(np.float64))
    assert np.max(np.abs(got["wte"] - ref)) < 1e-4
    refp = dx.reshape(w["B"], w["T"], -1).astype(np.float64).sum(0)
    assert np.max(np.abs(got["wpe"][: w["T"]] - refp)) < 1e-4
    assert np.all(got["wpe"][w["T"]:] == 0.0)
    m.close()


def test_embedding_reproduces_ids_exactly():
    """Encode each id in two channels of its token-table row; the embedding
    output must give back every id exactly."""
    w = workload("tiny", vocab=500, vocab_padded=512, B=3, T=29)
    p = synth.init_params(w, seed=5)
    p["wpe"][:] = 0.0
    p["wte"][:] = 0.0
    k = np.arange(w["vocab"])
    p["wte"][: w["vocab"], 0] = k // 256
    p["wte"][: w["vocab"], 1] = k % 256
    ids, _ = synth.token_batch(w, seed=6)
    m = _model(w)
    m.set_params(p)
    m.forward(torch.from_numpy(ids), None)
    x = _np(m.activation("residual", 0)).reshape(-1, w["d_model"])
    got = (x[:, 0] * 256 + x[:, 1]).astype(np.int64)
    assert np.array_equal(got, ids.ravel().astype(np.int64))
    m.close()


def test_per_token_losses_at_their_positions():
    """Per-token losses must line up with the oracle's position by position
    (the target gather is exact): a shuffled comparison would fail."""
    w = workload("tiny", vocab=500, vocab_padded=512, B=3, T=29)
    p = synth.init_params(w, seed=8)
    ids, tgt = synth.token_batch(w, seed=9)
    cache = oracle.forward(p, ids, tgt, oracle_config(w))
    m = _model(w)
    m.set_params(p)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    got = _np(m.activation("losses"))
    ref = cache["losses"].ravel()
    assert np.max(np.abs(got - ref)) < 0.05
    assert np.argmax(got) == np.argmax(ref) or abs(got[np.argmax(ref)] - ref.max()) < 0.05
    m.close()


@pytest.mark.parametrize("case", list(CASES))
def test_evaluate_equals_the_training_forward(case):
    """The forward-only evaluation runs the training forward's kernels (the
    head and cross-entropy as the two-pass arrangement's statistics pass): its
    per-token losses equal a training forward's in that arrangement bit for
    bit, are within tolerance of the oracle and of the default arrangement's,
    and it leaves no state to backward from."""
    w = workload("tiny", **CASES[case])
    p = synth.perturb_params(synth.init_params(w, seed=41), seed=42)
    ids, tgt = synth.token_batch(w, seed=43)
    m = _model(w)
    m.set_params(p)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    ref0 = _np(m.activation("losses")).copy()
    m.set_fusion("head_ce", 1)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    loss = m.loss()
    ref = _np(m.activation("losses")).copy()
    tl = torch.zeros(w["B"] * w["T"], device="cuda")
    ev = m.evaluate(torch.from_numpy(ids), torch.from_numpy(tgt), tl)
    got = tl.cpu().numpy()
    assert np.array_equal(got, ref)
    assert ev == loss
    assert np.max(np.abs(got - ref0)) < LOSS_ATOL
    cache = oracle.forward(p, ids, tgt, oracle_config(w))
    assert abs(ev - float(cache["loss"])) < LOSS_ATOL
    assert np.max(np.abs(got - cache["losses"].ravel())) < 5 * LOSS_ATOL
    from paper_2609_28568_amd import binding
    with pytest.raises(binding.LibError):
        m.backward()
    m.close()


def test_zero_table_loss_is_ln_vocab():
    w = workload("tiny", vocab=500, vocab_padded=512)
    p = synth.init_params(w)
    p["wte"][:] = 0.0
    ids, tgt = synth.token_batch(w)
    m = _model(w)
    m.set_params(p)
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    assert abs(m.loss() - np.log(500)) < 1e-5
    m.close()


def test_adamw_matches_oracle_on_oracle_gradients():
    """Feed the oracle's gradients into the gradient buffer and run two
    optimizer steps; parameters, moments and the bf16 copy must follow the
    oracle's AdamW with clipping."""
    w = workload("tiny")
    ocfg = oracle_config(w, warmup_steps=1, lr_max=6e-4)
    p = synth.perturb_params(synth.init_params(w, seed=31), seed=32)
    m = _model(w, dict(warmup_steps=1, lr_max=6e-4, lr_min=6e-5))
    m.set_params(p)
    ref_p = {k: v.astype(np.float64) for k, v in p.items()}
    ref_m = {k: np.zeros_like(v) for k, v in ref_p.items()}
    ref_v = {k: np.zeros_like(v) for k, v in ref_p.items()}
    g = np.random.default_rng(33)
    for step, gscale in enumerate((3.0, 0.05)):   # first clipped, second not
        ids, tgt = synth.token_batch(w, seed=34 + step)
        m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
        m.backward()
        grads = {k: (g.standard_normal(v.shape) * gscale / np.sqrt(v.size)).astype(np.float32)
                 for k, v in p.items()}
        grads["wte"][w["vocab"]:] = 0.0
        flat = np.zeros(m.n_params, np.float32)
        for k, (off, shape) in m.kinds.items():
            flat[off:off + grads[k].size] = grads[k].ravel()
        m.flat("grads").copy_(torch.from_numpy(flat))
        norm_out = torch.zeros(1, device="cuda")
        lr = m.adamw_step(step, norm_out)
        norm = oracle.global_norm(grads)
        assert abs(float(norm_out.item()) - norm) < 1e-5 * norm
        coef = oracle.clip_coefficient(norm, 1.0)
        assert abs(lr - oracle.lr_at(ocfg, step)) < 1e-12 + 1e-6 * lr
        oracle.adamw_update(ref_p, {k: v.astype(np.float64) for k, v in grads.items()}, ref_m, ref_v,
                            step, oracle.lr_at(ocfg, step), ocfg, coef)
        got = m.to_dict("params")
        for k in oracle.KINDS:
            d_ref = ref_p[k] - p[k]
            d_got = got[k].astype(np.float64) - p[k]
            e = rel_l2(d_got, d_ref) if np.any(d_ref) else float(np.max(np.abs(d_got)))
            assert e < 1e-3, (step, k, e)
        gm = m.to_dict("m")
        for k in oracle.KINDS:
            assert rel_l2(gm[k], ref_m[k]) < 1e-5 or not np.any(ref_m[k])
    bf = m.flat_bf16().float().cpu().numpy()
    fp = m.flat("params").cpu().numpy()
    assert np.max(np.abs(bf - fp) / np.maximum(np.abs(fp), 1e-30)) <= 2.0 ** -8
    m.close()


def test_gradient_accumulation_matches_one_big_batch():
    """Two micro-steps with accumulate give the oracle's gradient of the mean
    over both micro-batches."""
    w = workload("tiny", grad_accum=2)
    p = synth.perturb_params(synth.init_params(w, seed=41), seed=42)
    ocfg = oracle_config(w)
    mb = [synth.token_batch(w, seed=43, micro=i) for i in range(2)]
    ref = oracle.zero_grads(p)
    losses = []
    for ids, tgt in mb:
        c = oracle.forward(p, ids, tgt, ocfg, grad_scale=1.0 / (ids.size * 2))
        losses.append(float(c["loss"]))
        oracle.backward(p, c, ocfg, ref)
    m = _model(w)
    m.set_params(p)
    got_losses = []
    for i, (ids, tgt) in enumerate(mb):
        m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
        got_losses.append(m.loss())
        m.backward(accumulate=i > 0)
    g = m.to_dict("grads")
    for a, b in zip(got_losses, losses):
        assert abs(a - b) < LOSS_ATOL
    for k in oracle.KINDS:
        assert rel_l2(g[k], ref[k]) < REL_L2, k
    m.close()


def test_call_order_errors():
    from paper_2609_28568_amd import binding
    w = workload("tiny")
    m = _model(w)
    m.set_params(synth.init_params(w))
    with pytest.raises(binding.LibError) as e:
        m.backward()
    assert e.value.status == binding.GPT2_ERR_STATE
    with pytest.raises(binding.LibError) as e:
        m.adamw_step(0)
    assert e.value.status == binding.GPT2_ERR_STATE
    ids, tgt = synth.token_batch(w)
    m.forward(torch.from_numpy(ids), None)
    with pytest.raises(binding.LibError):
        m.backward()
    m.forward(torch.from_numpy(ids), torch.from_numpy(tgt))
    with pytest.raises(binding.LibError):
        m.backward(accumulate=True)
    m.backward()
    m.adamw_step(0)
    m.close()


def test_bf16_copy_rounds_to_nearest_even_exactly():
    """The bf16 weight copy is the round-to-nearest-even image of the fp32
    master, bit for bit: exact ties both ways, values just beside a tie,
    subnormals, the largest finite values (which round to infinity) and
    infinities."""
    w = workload("tiny")
    m = _model(w)
    n = m.n_params
    g = np.random.default_rng(77)
    hi = g.integers(0, 1 << 16, n, dtype=np.uint32) << 16
    lo = g.choice(np.array([0x8000, 0x7FFF, 0x8001, 0x0000, 0xFFFF], np.uint32), n)
    bits = hi | lo
    bits[:13] = [0x00008000, 0x00018000, 0x7F7F8000, 0x7F7FFFFF, 0xFF7F7FFF, 0x7F800000, 0xFF800000,
                 0x00000001, 0x807FFFFF, 0x3F808000, 0x3F818000, 0xBF808000, 0x3F80FFFF]
    nan = ((bits & 0x7F800000) == 0x7F800000) & ((bits & 0x007FFFFF) != 0)
    bits[nan] = 0
    vals = bits.view(np.float32)
    m.flat("params").copy_(torch.from_numpy(vals.copy()))
    assert m.L.gpt2_sync_weights(m.handle) == 0
    torch.cuda.synchronize()
    got = m.flat_bf16().view(torch.int16).cpu().numpy().view(np.uint16)
    want = (synth.round_to_bf16(vals).view(np.uint32) >> 16).astype(np.uint16)
    assert np.array_equal(got, want), np.flatnonzero(got != want)[:8]
    m.close()
