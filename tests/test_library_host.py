"""Host-side checks of the HIP library: it loads without a GPU, exports every
function the header declares, validates configs, and lays parameters out the
way the oracle names and counts them."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle
from paper_2609_28568_amd import binding, synth
from tests.util import oracle_config, workload

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "gpt2.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gpt2_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_function():
    L = binding.lib()
    names = header_functions()
    assert len(names) >= 18
    for n in names:
        assert hasattr(L, n), n


@pytest.mark.parametrize("name", ["tiny", "block124m", "gpt2_124m"])
def test_layout_matches_oracle(name):
    w = workload(name)
    cfg = binding.make_config(w, synth.OPTIM)
    ocfg = oracle_config(w)
    sizes = binding.query_sizes(cfg)
    assert sizes.n_params == oracle.param_count(ocfg)
    table = binding.tensor_table(cfg)
    assert [t[0] for t in table] == oracle.tensor_names(ocfg)
    kinds = binding.kind_table(cfg)
    shapes = oracle.param_shapes(ocfg)
    off = 0
    for k in oracle.KINDS:
        assert kinds[k] == (off, shapes[k]), k
        off += int(np.prod(shapes[k]))
    for n, _, shape, decay in table:
        assert decay == (len(shape) == 2), n


def test_paper_parameter_count_through_the_abi():
    cfg = binding.make_config(workload("gpt2_124m"), synth.OPTIM)
    table = binding.tensor_table(cfg)
    assert len(table) == 148
    n = sum(int(np.prod(s)) for _, _, s, _ in table)
    assert n - (50304 - 50257) * 768 == 124439808


@pytest.mark.parametrize("over", [
    dict(n_head=5), dict(d_model=96, n_head=2), dict(vocab_padded=500), dict(vocab=600),
    dict(T=64, max_seq_len=32), dict(B=0), dict(d_ff=100), dict(vocab_padded=70000, vocab=512),
    # 42,496 tokens x 50,304 padded vocabulary: the logits exceed 32-bit offsets
    dict(B=83, T=512, max_seq_len=512, vocab=50257, vocab_padded=50304),
])
def test_invalid_configs_are_rejected(over):
    w = workload("tiny", **over)
    cfg = binding.make_config(w, synth.OPTIM)
    s = binding.Sizes()
    assert binding.lib().gpt2_query_sizes(ctypes.byref(cfg), ctypes.byref(s)) == binding.GPT2_ERR_INVALID_ARG
    assert binding.lib().gpt2_last_error(None)


def test_null_arguments_are_rejected():
    L = binding.lib()
    assert L.gpt2_query_sizes(None, None) == binding.GPT2_ERR_INVALID_ARG
    assert L.gpt2_forward(None, None, None) == binding.GPT2_ERR_INVALID_ARG
    assert L.gpt2_backward(None, 0) == binding.GPT2_ERR_INVALID_ARG


@pytest.mark.parametrize("step", [0, 1, 350, 699, 700, 701, 5000, 18864, 18865, 30000])
def test_schedule_matches_oracle(step):
    w = workload("gpt2_124m")
    cfg = binding.make_config(w, synth.OPTIM)
    got = binding.lib().gpt2_lr_at(ctypes.byref(cfg), step)
    want = oracle.lr_at(oracle_config(w), step)
    assert math.isclose(got, want, rel_tol=1e-6, abs_tol=1e-12)
