"""Pins for the oracle's seeded initialisation (CPU only): the counter-based
generator against its published known-answer values, the normal transform
against the normal distribution, and the initialised parameters against the
paper's initialisation rule (section "Model")."""
import json
import os

import numpy as np
import pytest
from scipy import stats

import oracle
from oracle import init as oinit
from paper_2609_28568_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox4x32_10_kat.json")


def test_philox_known_answers():
    for case in json.load(open(GOLDEN))["cases"]:
        ctr = np.array([[int(x, 16) for x in case["counter"]]], np.uint32)
        key = tuple(int(x, 16) for x in case["key"])
        got = oinit.philox4x32_10(ctr, key)[0]
        assert [f"{int(v):08x}" for v in got] == case["out"], case


def test_philox_counters_are_independent_of_batching():
    """The draw of element i depends on i and the seed only."""
    a = oinit.normals(1000, 64, seed=5)
    b = oinit.normals_at(np.arange(1000, 1064, dtype=np.uint64)[::-1], seed=5)[::-1]
    assert np.array_equal(a, b)
    assert not np.array_equal(a, oinit.normals(1000, 64, seed=6))


def test_box_muller_gives_standard_normals():
    z = oinit.normals(0, 1 << 20, seed=1337)
    n = z.size
    assert abs(z.mean()) < 5.0 / np.sqrt(n)
    assert abs(z.var() - 1.0) < 5.0 * np.sqrt(2.0 / n)
    assert abs(stats.skew(z)) < 5.0 * np.sqrt(6.0 / n)
    assert stats.kstest(z, "norm").pvalue > 1e-4
    # element pairs are uncorrelated
    assert abs(np.corrcoef(z[:-1], z[1:])[0, 1]) < 5.0 / np.sqrt(n)


def test_seeded_params_follow_the_initialisation_rule():
    w = dict(synth.WORKLOADS["tiny"], vocab=500, vocab_padded=512)
    cfg = oracle.Config.from_dict({**w, **synth.OPTIM})
    p = oinit.seeded_params(cfg, seed=1337)
    L = cfg.n_layer
    assert set(p) == set(oracle.KINDS)
    for k, shape in oracle.param_shapes(cfg).items():
        assert p[k].shape == shape and p[k].dtype == np.float32, k
    for k in ("ln1b", "ln2b", "lnfb", "qkvb", "attprojb", "fcb", "fcprojb"):
        assert np.all(p[k] == 0.0), k
    for k in ("ln1w", "ln2w", "lnfw"):
        assert np.all(p[k] == 1.0), k
    assert np.all(p["wte"][cfg.vocab:] == 0.0)
    for k, std in (("wte", 0.02), ("wpe", 0.02), ("qkvw", 0.02), ("fcw", 0.02),
                   ("attprojw", 0.02 / np.sqrt(2 * L)), ("fcprojw", 0.02 / np.sqrt(2 * L))):
        x = p[k][: cfg.vocab] if k == "wte" else p[k]
        x = x.astype(np.float64).ravel()
        n = x.size
        assert abs(x.mean()) < 5 * std / np.sqrt(n), k
        assert abs(x.std() / std - 1.0) < 5 * np.sqrt(0.5 / n), k


def test_seeded_values_at_matches_whole_draw():
    w = dict(synth.WORKLOADS["tiny"], vocab=500, vocab_padded=512)
    cfg = oracle.Config.from_dict({**w, **synth.OPTIM})
    p = oinit.seeded_params(cfg, seed=7)
    flat = np.concatenate([p[k].ravel() for k in oracle.KINDS])
    idx = np.random.default_rng(0).integers(0, flat.size, 5000)
    assert np.array_equal(oinit.seeded_values_at(cfg, 7, idx), flat[idx])
