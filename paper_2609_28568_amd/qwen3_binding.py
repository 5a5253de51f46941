"""ctypes binding of the Qwen3-shaped adapter step (include/qwen3.h) in
libgpt2_mi355x.so.

Argument marshalling only: torch supplies the device buffers and the stream,
every step runs in the library's HIP kernels. Also maps the per-projection
tensors of the oracle's parameter dictionaries to the library's packed
layouts (q|k|v and gate|up stacked, adapter ranks zero-padded) and back.
"""
from __future__ import annotations

import ctypes

import numpy as np

from .binding import LibError, lib as _lib_gpt2

RP = 64   # padded adapter rank of the library
# kernel classes of the timing probes (QWEN3_K_* in include/qwen3.h)
FUSION = dict(swiglu=0)
KCLASS = dict(gemm_fwd=0, gemm_dx=1, gemm_adapter=2, attn_fwd=3, attn_bwd=4, norm=5, cross_entropy=6, optimizer=7,
              other=8)
GROUPS = {"qkv": 1, "o": 2, "gate_up": 4, "down": 8}
_GROUP_TARGETS = {"qkv": ("q", "k", "v"), "o": ("o",), "gate_up": ("gate", "up"), "down": ("down",)}


class Qwen3Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layer", "d_model", "n_head", "n_kv_head", "head_dim", "d_ff",
                                              "vocab", "max_seq_len", "B", "T")] + [
        ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float), ("lora_rank", ctypes.c_int32),
        ("lora_alpha", ctypes.c_float), ("lora_groups", ctypes.c_int32), ("loss_from", ctypes.c_float),
        ("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("adam_eps", ctypes.c_float),
        ("weight_decay", ctypes.c_float), ("grad_clip", ctypes.c_float)]


_BUFS = ("base_bf16", "lora_f32", "lora_grads", "adam_m", "adam_v", "lora_bf16", "activations", "workspace")


class Qwen3Sizes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in _BUFS]


class Qwen3Buffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in _BUFS]


_lib = None


def lib():
    """The shared library with the qwen3_* prototypes declared."""
    global _lib
    if _lib is not None:
        return _lib
    L = _lib_gpt2()
    P, I32, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_float
    protos = {
        "qwen3_query_sizes": (I32, [ctypes.POINTER(Qwen3Config), ctypes.POINTER(Qwen3Sizes)]),
        "qwen3_tensor_info": (I32, [ctypes.POINTER(Qwen3Config), I32, I32, ctypes.c_char_p,
                                    ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(I32), ctypes.POINTER(I32)]),
        "qwen3_init": (I32, [ctypes.POINTER(Qwen3Config), ctypes.POINTER(Qwen3Buffers), P, ctypes.POINTER(P)]),
        "qwen3_sync_weights": (I32, [P]),
        "qwen3_forward": (I32, [P, P, P]),
        "qwen3_backward": (I32, [P]),
        "qwen3_adamw_step": (I32, [P, ctypes.c_int64, P]),
        "qwen3_loss": (I32, [P, ctypes.POINTER(F32), P]),
        "qwen3_set_fusion": (I32, [P, I32, I32]),
        "qwen3_destroy": (None, [P]),
        "qwen3_last_error": (ctypes.c_char_p, [P]),
        "qwen3_probe_enable": (I32, [P, ctypes.c_uint32]),
        "qwen3_probe_reset": (I32, [P]),
        "qwen3_probe_read": (I32, [P, I32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64),
                                   ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in protos.items():
        f = getattr(L, name)
        f.restype, f.argtypes = res, args
    _lib = L
    return L


def make_config(w: dict, optim: dict | None = None) -> Qwen3Config:
    """Library config from a workload dict and optimiser settings (the
    oracle's field names); adapter targets become whole groups."""
    src = dict(w)
    src.update(optim or {})
    c = Qwen3Config()
    for f, _ in Qwen3Config._fields_:
        if f != "lora_groups" and f in src:
            setattr(c, f, src[f])
    targets = tuple(src.get("lora_targets", ("q", "k", "v", "o")))
    groups = 0
    for g, ts in _GROUP_TARGETS.items():
        present = [t in targets for t in ts]
        if any(present):
            if not all(present):
                raise ValueError(f"adapter targets must cover the whole group {ts}")
            groups |= GROUPS[g]
    c.lora_groups = groups
    return c


def out_widths(cfg: Qwen3Config) -> dict:
    qd, kvd = cfg.n_head * cfg.head_dim, cfg.n_kv_head * cfg.head_dim
    return {"q": qd, "k": kvd, "v": kvd, "o": cfg.d_model, "gate": cfg.d_ff, "up": cfg.d_ff, "down": cfg.d_model}


def targets_of(cfg: Qwen3Config) -> tuple:
    return tuple(t for g, ts in _GROUP_TARGETS.items() if cfg.lora_groups & GROUPS[g] for t in ts)


def _check(status, handle=None):
    if status != 0:
        msg = lib().qwen3_last_error(handle)
        raise LibError(status, msg.decode() if msg else "")


def query_sizes(cfg: Qwen3Config) -> Qwen3Sizes:
    s = Qwen3Sizes()
    _check(lib().qwen3_query_sizes(ctypes.byref(cfg), ctypes.byref(s)))
    return s


def tensor_table(cfg: Qwen3Config, which: int):
    """[(name, offset, shape)] of the base (0) or adapter (1) layout."""
    out, i = [], 0
    name = ctypes.create_string_buffer(64)
    off = ctypes.c_size_t()
    shape = (ctypes.c_int32 * 3)()
    nd = ctypes.c_int32()
    while lib().qwen3_tensor_info(ctypes.byref(cfg), which, i, name, ctypes.byref(off), shape, ctypes.byref(nd)) == 0:
        out.append((name.value.decode(), off.value, tuple(shape[k] for k in range(nd.value))))
        i += 1
    return out


def pack_base(base: dict) -> dict:
    """The library's base tensors from the oracle's: q|k|v and gate|up stacked."""
    p = dict(base)
    p["qkv"] = np.concatenate([base["q"], base["k"], base["v"]], axis=1)
    p["gate_up"] = np.concatenate([base["gate"], base["up"]], axis=1)
    return p


def pack_lora(lora: dict, shapes: dict, r: int) -> dict:
    """Padded group tensors (name -> array of the library's shape) from the
    oracle's per-projection A [L, r, in] and B [L, out, r]."""
    out = {}
    for g, ts in _GROUP_TARGETS.items():
        if g + "_A" not in shapes:
            continue
        A = np.zeros(shapes[g + "_A"], dtype=np.float32)
        B = np.zeros(shapes[g + "_B"], dtype=np.float32)
        row = 0
        for j, t in enumerate(ts):
            A[:, j * RP:j * RP + r, :] = lora[t + "_A"]
            o = lora[t + "_B"].shape[1]
            B[:, row:row + o, :r] = lora[t + "_B"]
            row += o
        out[g + "_A"], out[g + "_B"] = A, B
    return out


def unpack_lora(packed: dict, targets, r: int, out_widths: dict) -> dict:
    """The oracle's per-projection tensors from the library's padded groups."""
    res = {}
    for g, ts in _GROUP_TARGETS.items():
        if g + "_A" not in packed:
            continue
        row = 0
        for j, t in enumerate(ts):
            o = out_widths[t]
            res[t + "_A"] = packed[g + "_A"][:, j * RP:j * RP + r, :]
            res[t + "_B"] = packed[g + "_B"][:, row:row + o, :r]
            row += o
    return {k: v for k, v in res.items() if k[:-2] in targets}


class Qwen3:
    """One model instance on a torch-owned set of device buffers."""

    def __init__(self, cfg: Qwen3Config, device="cuda"):
        import torch
        self.torch = torch
        self.cfg = cfg
        sizes = query_sizes(cfg)
        self.bufs = {n: torch.zeros(getattr(sizes, n), dtype=torch.uint8, device=device) for n in _BUFS}
        self.base_table = {n: (o, s) for n, o, s in tensor_table(cfg, 0)}
        self.lora_table = {n: (o, s) for n, o, s in tensor_table(cfg, 1)}
        self.n_lora = sum(int(np.prod(s)) for _, s in self.lora_table.values())
        self.stream = torch.cuda.current_stream(device)
        b = Qwen3Buffers(**{n: t.data_ptr() for n, t in self.bufs.items()})
        self.h = ctypes.c_void_p()
        _check(lib().qwen3_init(ctypes.byref(cfg), ctypes.byref(b), ctypes.c_void_p(self.stream.cuda_stream),
                                ctypes.byref(self.h)))

    def close(self):
        if self.h:
            lib().qwen3_destroy(self.h)
            self.h = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _view(self, buf, dtype, table, name):
        torch = self.torch
        off, shape = table[name]
        esz = 2 if dtype == torch.bfloat16 else 4
        n = int(np.prod(shape))
        return self.bufs[buf][off * esz:(off + n) * esz].view(dtype).view(*shape)

    def set_base(self, base: dict):
        """Copy the oracle's base parameters (rounded to bf16) to the device."""
        torch = self.torch
        p = pack_base(base)
        for name in self.base_table:
            v = self._view("base_bf16", torch.bfloat16, self.base_table, name)
            v.copy_(torch.from_numpy(np.ascontiguousarray(p[name], dtype=np.float32)).to(torch.bfloat16))

    def set_lora(self, lora: dict):
        """Copy the oracle's adapter parameters (fp32) and refresh their bf16 copy."""
        self.set_packed("lora_f32", lora)
        _check(lib().qwen3_sync_weights(self.h), self.h)

    def packed(self, which="lora_f32") -> dict:
        """Group tensors of an adapter-layout buffer (lora_f32, lora_grads,
        adam_m, adam_v: fp32; lora_bf16: bf16), copied to the host as fp32."""
        torch = self.torch
        torch.cuda.synchronize()
        dt = torch.bfloat16 if which == "lora_bf16" else torch.float32
        return {n: self._view(which, dt, self.lora_table, n).float().cpu().numpy() for n in self.lora_table}

    def adapters(self, which="lora_f32") -> dict:
        """Per-projection tensors of an adapter-layout buffer, oracle names."""
        return unpack_lora(self.packed(which), targets_of(self.cfg), self.cfg.lora_rank, out_widths(self.cfg))

    def flat(self, which="lora_grads"):
        """An fp32 adapter-layout buffer as one flat device tensor."""
        return self.bufs[which][:self.n_lora * 4].view(self.torch.float32)

    def set_packed(self, which: str, per_projection: dict):
        """Write per-projection fp32 tensors (oracle names) into an fp32
        adapter-layout buffer, padding zero."""
        torch = self.torch
        shapes = {n: s for n, (_, s) in self.lora_table.items()}
        for name, arr in pack_lora(per_projection, shapes, self.cfg.lora_rank).items():
            self._view(which, torch.float32, self.lora_table, name).copy_(torch.from_numpy(arr))


    def forward(self, ids, targets=None):
        torch = self.torch
        self._ids = ids.to(torch.int32).cuda().contiguous()
        self._tgt = None if targets is None else targets.to(torch.int32).cuda().contiguous()
        _check(lib().qwen3_forward(self.h, ctypes.c_void_p(self._ids.data_ptr()),
                                   ctypes.c_void_p(self._tgt.data_ptr() if self._tgt is not None else 0)), self.h)

    def backward(self):
        _check(lib().qwen3_backward(self.h), self.h)

    def adamw_step(self, step: int, norm_out=None):
        ptr = ctypes.c_void_p(norm_out.data_ptr() if norm_out is not None else 0)
        _check(lib().qwen3_adamw_step(self.h, step, ptr), self.h)

    def loss(self, token_losses=None) -> float:
        v = ctypes.c_float()
        ptr = ctypes.c_void_p(token_losses.data_ptr() if token_losses is not None else 0)
        _check(lib().qwen3_loss(self.h, ctypes.byref(v), ptr), self.h)
        return v.value

    # ---- probes -------------------------------------------------------------
    def set_fusion(self, fusion: str, mode: int):
        """Select an alternative kernel arrangement (qwen3_set_fusion)."""
        _check(lib().qwen3_set_fusion(self.h, FUSION[fusion], int(mode)), self.h)

    def probe_enable(self, classes):
        mask = 0
        for c in classes:
            mask |= 1 << KCLASS[c]
        _check(lib().qwen3_probe_enable(self.h, mask), self.h)

    def probe_reset(self):
        _check(lib().qwen3_probe_reset(self.h), self.h)

    def probe_read(self, cls: str) -> dict:
        ms, fl, by = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
        n = ctypes.c_int64()
        _check(lib().qwen3_probe_read(self.h, KCLASS[cls], ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl),
                                      ctypes.byref(by)), self.h)
        return {"ms": ms.value, "launches": n.value, "flops": fl.value, "bytes": by.value}
