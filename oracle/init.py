"""Seeded initial weights of the GPT-2 step, drawn from a counter-based
generator (test infrastructure only).

The library can initialise its weights on the device from a seed instead of
receiving them from the caller. Random numbers drawn on the device cannot be
passed in as inputs, so both sides implement the same counter-based
generator from its published definition, and this module is the oracle's
side:

  * Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
    easy as 1, 2, 3", SC 2011): a 128-bit counter and a 64-bit key go
    through ten rounds, each two 32x32->64-bit products with the multipliers
    0xD2511F53 and 0xCD9E8D57 whose high halves are XORed with the other
    counter words and the key; the key is bumped by the Weyl constants
    0x9E3779B9 and 0xBB67AE85 between rounds;
  * the Box-Muller transform (Box and Muller, 1958) of the first two output
    words, as u1 = (x0 + 1/2) / 2^32 and u2 = (x1 + 1/2) / 2^32:
    z = sqrt(-2 ln u1) cos(2 pi u2), in float64.

Element i of the flat parameter buffer (the layout of the library's ABI:
kinds in order, each stacked over layers) takes counter (i mod 2^32,
i div 2^32, 0, 0) and key (seed mod 2^32, seed div 2^32).

What each tensor gets follows section "Model" (normal initialisation with
standard deviation 0.02; projections that write into the residual stream
scaled by 1/sqrt(2L)) and the readings of the oracle's header: every 2-D
weight including both embedding tables N(0, 0.02), the attention and MLP
output projections N(0, 0.02/sqrt(2L)), biases 0, LayerNorm gains 1 and
shifts 0, and the padding rows of the token table exactly 0.
"""
from __future__ import annotations

import numpy as np

from .gpt2 import Config, KINDS, param_shapes

_M0, _M1 = 0xD2511F53, 0xCD9E8D57
_W0, _W1 = 0x9E3779B9, 0xBB67AE85
_MASK = 0xFFFFFFFF


def philox4x32_10(ctr, key):
    """Philox4x32 with 10 rounds. ctr: uint32 array [..., 4]; key: two
    uint32. Returns uint32 [..., 4]."""
    c = [np.asarray(ctr[..., j], np.uint64) for j in range(4)]
    k0, k1 = np.uint64(int(key[0]) & _MASK), np.uint64(int(key[1]) & _MASK)
    m0, m1, mask = np.uint64(_M0), np.uint64(_M1), np.uint64(_MASK)
    for r in range(10):
        if r > 0:
            k0 = np.uint64((int(k0) + _W0) & _MASK)
            k1 = np.uint64((int(k1) + _W1) & _MASK)
        p0 = m0 * c[0]   # exact: both factors < 2^32
        p1 = m1 * c[2]
        hi0, lo0 = p0 >> np.uint64(32), p0 & mask
        hi1, lo1 = p1 >> np.uint64(32), p1 & mask
        c = [hi1 ^ c[1] ^ k0, lo1, hi0 ^ c[3] ^ k1, lo0]
    return np.stack([x.astype(np.uint32) for x in c], axis=-1)


def normals(first: int, count: int, seed: int) -> np.ndarray:
    """Standard normal deviates of flat elements first .. first+count-1."""
    return normals_at(np.arange(first, first + count, dtype=np.uint64), seed)


def normals_at(i, seed: int) -> np.ndarray:
    """Standard normal deviates of the flat elements with indices i."""
    i = np.asarray(i, np.uint64)
    ctr = np.zeros(i.shape + (4,), np.uint32)
    ctr[..., 0] = (i & np.uint64(_MASK)).astype(np.uint32)
    ctr[..., 1] = (i >> np.uint64(32)).astype(np.uint32)
    x = philox4x32_10(ctr, (seed & _MASK, (seed >> 32) & _MASK))
    u1 = (x[..., 0].astype(np.float64) + 0.5) / 4294967296.0
    u2 = (x[..., 1].astype(np.float64) + 0.5) / 4294967296.0
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)


# standard deviation of each kind, as a function of the layer count; None:
# constant fill
def _kind_rule(kind: str, n_layer: int):
    std, rstd = 0.02, 0.02 / np.sqrt(2.0 * n_layer)
    rules = {"wte": std, "wpe": std, "qkvw": std, "fcw": std, "attprojw": rstd, "fcprojw": rstd}
    if kind in rules:
        return rules[kind], None
    return None, 1.0 if kind in ("ln1w", "ln2w", "lnfw") else 0.0


def seeded_params(cfg: Config, seed: int) -> dict:
    """Initial fp32 parameters {kind: array} as the device initialisation
    draws them (each element rounded once from its float64 value)."""
    shapes = param_shapes(cfg)
    out, off = {}, 0
    for k in KINDS:
        n = int(np.prod(shapes[k]))
        std, fill = _kind_rule(k, cfg.n_layer)
        if std is None:
            a = np.full(n, fill, np.float32)
        else:
            a = (normals(off, n, seed) * std).astype(np.float32)
        a = a.reshape(shapes[k])
        if k == "wte":
            a[cfg.vocab:] = 0.0
        out[k] = a
        off += n
    return out


def seeded_values_at(cfg: Config, seed: int, flat_index) -> np.ndarray:
    """The fp32 values seeded_params gives the flat elements with the given
    indices, without drawing the rest of the buffer."""
    shapes = param_shapes(cfg)
    idx = np.asarray(flat_index, np.int64)
    out = np.empty(idx.shape, np.float32)
    off = 0
    for k in KINDS:
        n = int(np.prod(shapes[k]))
        sel = (idx >= off) & (idx < off + n)
        if sel.any():
            std, fill = _kind_rule(k, cfg.n_layer)
            if std is None:
                out[sel] = fill
            else:
                out[sel] = (normals_at(idx[sel].astype(np.uint64), seed) * std).astype(np.float32)
            if k == "wte":
                out[sel & (idx >= off + cfg.vocab * cfg.d_model)] = 0.0
        off += n
    return out
