"""Host-side checks of the adapter-step part of the HIP library: it exports
every function include/qwen3.h declares, validates configs, and its adapter
layout holds exactly the oracle's adapter parameters once padding is removed."""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import qwen3 as q3
from paper_2609_28568_amd import binding, qwen3_binding as qb, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions():
    text = open(os.path.join(ROOT, "include", "qwen3.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(qwen3_[a-z_0-9]+)\s*\(", text)))


def _cfg(name="qwen3_tiny", **over):
    w = dict(synth.QWEN3_WORKLOADS[name])
    w.update(over)
    return w, qb.make_config(w, synth.QWEN3_OPTIM)


def test_library_exports_every_declared_function():
    names = header_functions()
    assert len(names) == 14
    L = qb.lib()
    for n in names:
        assert hasattr(L, n), n


def test_config_struct_matches_the_header_field_order():
    text = open(os.path.join(ROOT, "include", "qwen3.h")).read()
    body = re.search(r"typedef struct qwen3_config \{(.*?)\} qwen3_config;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = []
    for decl in body.split(";"):
        decl = decl.strip()
        if decl:
            fields += [f.strip() for f in decl.split(None, 1)[1].split(",")]
    assert fields == [f for f, _ in qb.Qwen3Config._fields_]


@pytest.mark.parametrize("name,targets", [("qwen3_tiny", q3.PROJECTIONS), ("qwen3_tiny", ("q", "k", "v", "o")),
                                          ("qwen3_06b_lora", ("q", "k", "v", "o")),
                                          ("qwen3_06b_lora", q3.PROJECTIONS)])
def test_adapter_layout_round_trips_the_oracle_parameters(name, targets):
    w, cfg = _cfg(name, lora_targets=targets)
    if name == "qwen3_06b_lora":
        w = dict(w, n_layer=2)   # shapes per layer are what matter; keeps the host arrays small
        cfg = qb.make_config(w, synth.QWEN3_OPTIM)
    ocfg = q3.Qwen3Config.from_dict(w)
    table = {n: s for n, _, s in qb.tensor_table(cfg, 1)}
    rng = np.random.default_rng(5)
    lora = {k: rng.standard_normal(s).astype(np.float32) for k, s in q3.lora_shapes(ocfg).items()}
    packed = qb.pack_lora(lora, table, cfg.lora_rank)
    assert {k: v.shape for k, v in packed.items()} == table
    # every oracle element appears once; the rest is zero padding
    assert sum(int(np.count_nonzero(v)) for v in packed.values()) == q3.lora_param_count(ocfg)
    back = qb.unpack_lora(packed, targets, cfg.lora_rank, qb.out_widths(cfg))
    assert set(back) == set(lora)
    for k in lora:
        assert np.array_equal(back[k], lora[k]), k
    # offsets are contiguous in the header's group order
    off = 0
    for n, o, s in qb.tensor_table(cfg, 1):
        assert o == off, n
        off += int(np.prod(s))


def test_paper_and_benchmark_adapter_counts_through_the_abi():
    for targets, count in ((q3.PROJECTIONS, 10_092_544), (("q", "k", "v", "o"), 4_587_520)):
        w, cfg = _cfg("qwen3_06b_lora", lora_targets=targets)
        table = {n: s for n, _, s in qb.tensor_table(cfg, 1)}
        # real (unpadded) adapter elements: rank-r slices of every projection
        r, L = cfg.lora_rank, cfg.n_layer
        real = 0
        for g, ts in qb._GROUP_TARGETS.items():
            if g + "_A" in table:
                real += L * r * (len(ts) * table[g + "_A"][2] + table[g + "_B"][1])
        assert real == count


def test_base_layout_matches_the_oracle_shapes():
    w, cfg = _cfg()
    ocfg = q3.Qwen3Config.from_dict(w)
    shapes = q3.base_shapes(ocfg)
    base = {k: np.zeros(s, np.float32) for k, s in shapes.items()}
    packed = qb.pack_base(base)
    off = 0
    for n, o, s in qb.tensor_table(cfg, 0):
        assert packed[n].shape == s, n
        assert o == off
        off += int(np.prod(s))
    assert off == sum(int(np.prod(s)) for k, s in shapes.items()) 


@pytest.mark.parametrize("over", [
    dict(head_dim=64), dict(n_kv_head=3), dict(d_model=192), dict(d_ff=200), dict(vocab=1000),
    dict(B=1, T=96), dict(T=200), dict(lora_rank=0), dict(lora_rank=33), dict(lora_targets=()),
    dict(loss_from=1.0), dict(loss_from=-0.1), dict(d_model=4096, n_head=32, n_kv_head=8),
    # 8192 tokens x a 524,288-entry vocabulary: the logits exceed 32-bit offsets
    dict(vocab=524288, B=4, T=2048, max_seq_len=2048),
])
def test_invalid_configs_are_rejected(over):
    w = dict(synth.QWEN3_WORKLOADS["qwen3_tiny"])
    w.update(over)
    cfg = qb.make_config(w, synth.QWEN3_OPTIM)
    s = qb.Qwen3Sizes()
    assert qb.lib().qwen3_query_sizes(ctypes.byref(cfg), ctypes.byref(s)) == binding.GPT2_ERR_INVALID_ARG
    assert qb.lib().qwen3_last_error(None)


def test_partial_groups_are_refused_by_the_binding():
    w = dict(synth.QWEN3_WORKLOADS["qwen3_tiny"], lora_targets=("q", "v"))
    with pytest.raises(ValueError):
        qb.make_config(w, synth.QWEN3_OPTIM)


def test_null_arguments_are_rejected():
    L = qb.lib()
    assert L.qwen3_query_sizes(None, None) == binding.GPT2_ERR_INVALID_ARG
    assert L.qwen3_forward(None, None, None) == binding.GPT2_ERR_INVALID_ARG
    assert L.qwen3_backward(None) == binding.GPT2_ERR_INVALID_ARG
    assert L.qwen3_set_fusion(None, 0, 1) == binding.GPT2_ERR_INVALID_ARG
    assert L.qwen3_adamw_step(None, 0, None) == binding.GPT2_ERR_INVALID_ARG
    w, cfg = _cfg()
    assert L.qwen3_init(ctypes.byref(cfg), None, None, None) == binding.GPT2_ERR_INVALID_ARG
    name = ctypes.create_string_buffer(64)
    assert L.qwen3_tensor_info(ctypes.byref(cfg), 2, 0, name, None, None, None) == binding.GPT2_ERR_INVALID_ARG
    assert L.qwen3_tensor_info(ctypes.byref(cfg), 1, 99, name, None, None, None) == binding.GPT2_ERR_INVALID_ARG
