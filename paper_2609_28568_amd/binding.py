"""ctypes binding of libgpt2_mi355x.so: the C ABI declared in include/gpt2.h.

Argument marshalling only: torch supplies device buffers and the stream, every
step of the training step runs in the library's HIP kernels. The library must
be built (``paper_2609_28568_amd.build``); loading fails loudly otherwise.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgpt2_mi355x.so")

GPT2_OK, GPT2_ERR_INVALID_ARG, GPT2_ERR_STATE, GPT2_ERR_DEVICE = 0, 1, 2, 3

ACT = dict(residual=0, ln1=1, ln1_mean=2, ln1_rstd=3, qkv=4, att=5, att_lse=6, x_mid=7,
           ln2=8, ln2_mean=9, ln2_rstd=10, fc=11, gelu=12, lnf=13, lnf_mean=14, lnf_rstd=15,
           logits=16, losses=17)
FUSION = dict(residual_norm=0, head_ce=1)
KCLASS = dict(gemm_fwd=0, gemm_fwd_gelu=1, gemm_dx=2, gemm_dx_gelu=3, gemm_dw=4, attn_fwd=5,
              attn_bwd=6, layernorm=7, cross_entropy=8, optimizer=9, other=10, gemm_dw_grouped=11)

# parameter kinds of the flat buffer, in order, with the per-layer tensor
# name each stacked kind is made of
KINDS = ("wte", "wpe", "ln1w", "ln1b", "qkvw", "qkvb", "attprojw", "attprojb",
         "ln2w", "ln2b", "fcw", "fcb", "fcprojw", "fcprojb", "lnfw", "lnfb")
_LAYER_NAME = {"ln1w": "ln_1.weight", "ln1b": "ln_1.bias", "qkvw": "attn.c_attn.weight",
               "qkvb": "attn.c_attn.bias", "attprojw": "attn.c_proj.weight",
               "attprojb": "attn.c_proj.bias", "ln2w": "ln_2.weight", "ln2b": "ln_2.bias",
               "fcw": "mlp.c_fc.weight", "fcb": "mlp.c_fc.bias", "fcprojw": "mlp.c_proj.weight",
               "fcprojb": "mlp.c_proj.bias"}


class Config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("n_layer", "n_head", "d_model", "d_ff", "vocab",
                                              "vocab_padded", "max_seq_len", "B", "T", "grad_accum")] + [
        ("ln_eps", ctypes.c_float), ("lr_max", ctypes.c_float), ("lr_min", ctypes.c_float),
        ("warmup_steps", ctypes.c_int32), ("total_steps", ctypes.c_int32),
        ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("adam_eps", ctypes.c_float),
        ("weight_decay", ctypes.c_float), ("grad_clip", ctypes.c_float)]


class Sizes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in ("params_f32", "grads_f32", "adam_m", "adam_v",
                                               "params_bf16", "activations", "workspace", "n_params")]


class Buffers(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("params_f32", "grads_f32", "adam_m", "adam_v",
                                               "params_bf16", "activations", "workspace")]


_lib = None


def lib():
    """Load the library once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_28568_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, F32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float
    cfgp = ctypes.POINTER(Config)
    sig = {
        "gpt2_query_sizes": (I32, [cfgp, ctypes.POINTER(Sizes)]),
        "gpt2_num_tensors": (I32, [cfgp]),
        "gpt2_tensor_info": (I32, [cfgp, I32, ctypes.c_char_p, ctypes.POINTER(ctypes.c_size_t),
                                   ctypes.POINTER(I32), ctypes.POINTER(I32), ctypes.POINTER(I32)]),
        "gpt2_init": (I32, [cfgp, ctypes.POINTER(Buffers), P, ctypes.c_uint64, I32, ctypes.POINTER(P)]),
        "gpt2_sync_weights": (I32, [P]),
        "gpt2_forward": (I32, [P, P, P]),
        "gpt2_backward": (I32, [P, I32]),
        "gpt2_adamw_step": (I32, [P, I64, ctypes.POINTER(F32), P]),
        "gpt2_adamw_step_noalloc": (I32, [P, I64, ctypes.POINTER(F32), P]),
        "gpt2_loss": (I32, [P, ctypes.POINTER(F32), P]),
        "gpt2_evaluate": (I32, [P, P, P, ctypes.POINTER(F32), P]),
        "gpt2_lr_at": (F32, [cfgp, I64]),
        "gpt2_destroy": (None, [P]),
        "gpt2_last_error": (ctypes.c_char_p, [P]),
        "gpt2_activation_info": (I32, [P, I32, I32, ctypes.POINTER(ctypes.c_size_t),
                                       ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(I32)]),
        "gpt2_block_forward": (I32, [P, I32, P, P]),
        "gpt2_block_backward": (I32, [P, I32, P, P, I32]),
        "gpt2_embedding_backward": (I32, [P, P, P, I32]),
        "gpt2_set_fusion": (I32, [P, I32, I32]),
        "gpt2_probe_enable": (I32, [P, ctypes.c_uint32]),
        "gpt2_probe_reset": (I32, [P]),
        "gpt2_probe_read": (I32, [P, I32, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(I64),
                                  ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


def make_config(w: dict, optim: dict | None = None) -> Config:
    """Config from a workload dict (shapes) and optimiser settings."""
    o = dict(lr_max=6e-4, lr_min=0.0, warmup_steps=700, total_steps=18865, beta1=0.9, beta2=0.95,
             adam_eps=1e-8, weight_decay=0.1, grad_clip=1.0, ln_eps=1e-5)
    if optim:
        o.update(optim)
    c = Config()
    for k in ("n_layer", "n_head", "d_model", "d_ff", "vocab", "vocab_padded", "max_seq_len", "B", "T"):
        setattr(c, k, int(w[k]))
    c.grad_accum = int(w.get("grad_accum", 1))
    for k in ("ln_eps", "lr_max", "lr_min", "beta1", "beta2", "adam_eps", "weight_decay", "grad_clip"):
        setattr(c, k, float(o[k]))
    c.warmup_steps = int(o["warmup_steps"])
    c.total_steps = int(o["total_steps"])
    return c


class LibError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"status {status}: {msg}")
        self.status = status


def _check(status, handle=None):
    if status != GPT2_OK:
        msg = lib().gpt2_last_error(handle)
        raise LibError(status, msg.decode() if msg else "")


def query_sizes(cfg: Config) -> Sizes:
    s = Sizes()
    _check(lib().gpt2_query_sizes(ctypes.byref(cfg), ctypes.byref(s)))
    return s


def tensor_table(cfg: Config):
    """[(name, element offset, shape, decay)] for every parameter tensor."""
    L = lib()
    out = []
    name = ctypes.create_string_buffer(64)
    off = ctypes.c_size_t()
    shape = (ctypes.c_int32 * 2)()
    nd, dec = ctypes.c_int32(), ctypes.c_int32()
    for i in range(L.gpt2_num_tensors(ctypes.byref(cfg))):
        _check(L.gpt2_tensor_info(ctypes.byref(cfg), i, name, ctypes.byref(off), shape,
                                  ctypes.byref(nd), ctypes.byref(dec)))
        out.append((name.value.decode(), off.value, tuple(shape[:nd.value]), bool(dec.value)))
    return out


def kind_table(cfg: Config):
    """{kind: (element offset, shape stacked over layers)} from the tensor table."""
    tt = {n: (o, s) for n, o, s, _ in tensor_table(cfg)}
    L = cfg.n_layer
    kinds = {"wte": tt["wte"], "wpe": tt["wpe"], "lnfw": tt["ln_f.weight"], "lnfb": tt["ln_f.bias"]}
    for k, n in _LAYER_NAME.items():
        off, shape = tt[f"h.0.{n}"]
        kinds[k] = (off, (L,) + shape)
    return kinds


class GPT2:
    """One model over torch-allocated device buffers on the current stream.

    seed=None: the weights start at zero until set_params fills them
    (init_mode 0); seed=int: the library draws them on the device from that
    seed (init_mode 1) and clears the Adam moments."""

    def __init__(self, cfg: Config, device="cuda", seed=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.L = lib()
        self.sizes = query_sizes(cfg)
        self.device = torch.device(device)
        s = self.sizes
        alloc = lambda n: torch.empty(max(int(n), 256), dtype=torch.uint8, device=self.device)
        self.params_f32 = alloc(s.params_f32)
        self.grads_f32 = alloc(s.grads_f32)
        self.adam_m = torch.zeros(max(int(s.adam_m), 256), dtype=torch.uint8, device=self.device)
        self.adam_v = torch.zeros(max(int(s.adam_v), 256), dtype=torch.uint8, device=self.device)
        self.params_bf16 = alloc(s.params_bf16)
        self.activations = alloc(s.activations)
        self.workspace = alloc(s.workspace)
        self.params_f32.zero_()
        self.kinds = kind_table(cfg)
        self.n_params = int(s.n_params)
        self.stream = torch.cuda.current_stream(self.device)
        b = Buffers(*(t.data_ptr() for t in (self.params_f32, self.grads_f32, self.adam_m, self.adam_v,
                                              self.params_bf16, self.activations, self.workspace)))
        self.handle = ctypes.c_void_p()
        _check(self.L.gpt2_init(ctypes.byref(cfg), ctypes.byref(b), ctypes.c_void_p(self.stream.cuda_stream),
                                0 if seed is None else int(seed), 0 if seed is None else 1,
                                ctypes.byref(self.handle)))

    def close(self):
        if self.handle:
            self.torch.cuda.synchronize(self.device)
            self.L.gpt2_destroy(self.handle)
            self.handle = ctypes.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- parameters and state ------------------------------------------
    def flat(self, which="params"):
        buf = {"params": self.params_f32, "grads": self.grads_f32, "m": self.adam_m,
               "v": self.adam_v}[which]
        return buf[: self.n_params * 4].view(self.torch.float32)

    def flat_bf16(self):
        return self.params_bf16[: self.n_params * 2].view(self.torch.bfloat16)

    def set_params(self, params: dict):
        """Copy a {kind: array} dict into the fp32 master weights and refresh
        the bf16 copy; Adam moments are reset to zero."""
        host = np.zeros(self.n_params, np.float32)
        for k, (off, shape) in self.kinds.items():
            a = np.asarray(params[k], np.float32)
            assert a.shape == shape, (k, a.shape, shape)
            host[off:off + a.size] = a.ravel()
        self.flat("params").copy_(self.torch.from_numpy(host))
        self.adam_m.zero_()
        self.adam_v.zero_()
        _check(self.L.gpt2_sync_weights(self.handle), self.handle)

    def to_dict(self, which="params") -> dict:
        host = self.flat(which).cpu().numpy()
        return {k: host[off:off + int(np.prod(shape))].reshape(shape).copy()
                for k, (off, shape) in self.kinds.items()}

    # ---- the training step ------------------------------------------------
    def forward(self, ids, targets=None):
        self._ids = ids.to(self.device, self.torch.int32).contiguous()
        self._tgt = None if targets is None else targets.to(self.device, self.torch.int32).contiguous()
        _check(self.L.gpt2_forward(self.handle, ctypes.c_void_p(self._ids.data_ptr()),
                                   ctypes.c_void_p(self._tgt.data_ptr() if self._tgt is not None else 0)),
               self.handle)

    def backward(self, accumulate=False):
        _check(self.L.gpt2_backward(self.handle, int(bool(accumulate))), self.handle)

    def adamw_step(self, step: int, norm_out=None, noalloc=False):
        """Clip + AdamW; noalloc=True takes the entry point whose scratch is
        the library's static device array instead of the workspace."""
        lr = ctypes.c_float()
        ptr = ctypes.c_void_p(norm_out.data_ptr()) if norm_out is not None else ctypes.c_void_p(0)
        fn = self.L.gpt2_adamw_step_noalloc if noalloc else self.L.gpt2_adamw_step
        _check(fn(self.handle, int(step), ctypes.byref(lr), ptr), self.handle)
        return lr.value

    def loss(self, token_losses=None) -> float:
        """Mean loss of the last forward with targets; optionally fills a
        device fp32 [B*T] tensor with the per-position losses."""
        out = ctypes.c_float()
        tl = ctypes.c_void_p(token_losses.data_ptr()) if token_losses is not None else ctypes.c_void_p(0)
        _check(self.L.gpt2_loss(self.handle, ctypes.byref(out), tl), self.handle)
        return out.value

    def evaluate(self, ids, targets, token_losses=None) -> float:
        """Forward-only loss of held-out tokens (no activations kept, no
        dlogits); optionally fills a device fp32 [B*T] tensor of per-token
        losses."""
        ids = ids.to(self.device, self.torch.int32).contiguous()
        tgt = targets.to(self.device, self.torch.int32).contiguous()
        out = ctypes.c_float()
        tl = ctypes.c_void_p(token_losses.data_ptr()) if token_losses is not None else ctypes.c_void_p(0)
        _check(self.L.gpt2_evaluate(self.handle, ctypes.c_void_p(ids.data_ptr()), ctypes.c_void_p(tgt.data_ptr()),
                                    ctypes.byref(out), tl), self.handle)
        return out.value

    def lr_at(self, step: int) -> float:
        return self.L.gpt2_lr_at(ctypes.byref(self.cfg), int(step))

    def block_forward(self, layer, x_in, x_out=None):
        _check(self.L.gpt2_block_forward(self.handle, layer, ctypes.c_void_p(x_in.data_ptr()),
                                         ctypes.c_void_p(x_out.data_ptr() if x_out is not None else 0)),
               self.handle)

    def block_backward(self, layer, dx_out, dx_in=None, accumulate=False):
        _check(self.L.gpt2_block_backward(self.handle, layer, ctypes.c_void_p(dx_out.data_ptr()),
                                          ctypes.c_void_p(dx_in.data_ptr() if dx_in is not None else 0),
                                          int(bool(accumulate))), self.handle)

    def embedding_backward(self, ids, dx, accumulate=False):
        self._eids = ids.to(self.device, self.torch.int32).contiguous()
        _check(self.L.gpt2_embedding_backward(self.handle, ctypes.c_void_p(self._eids.data_ptr()),
                                              ctypes.c_void_p(dx.data_ptr()), int(bool(accumulate))),
               self.handle)

    def activation(self, name: str, layer: int = 0):
        """Torch view of a saved forward tensor in the activations buffer."""
        off, n, dt = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_int32()
        _check(self.L.gpt2_activation_info(self.handle, ACT[name], layer, ctypes.byref(off), ctypes.byref(n),
                                           ctypes.byref(dt)), self.handle)
        tdt, es = {0: (self.torch.float32, 4), 1: (self.torch.bfloat16, 2), 2: (self.torch.int32, 4)}[dt.value]
        return self.activations[off.value: off.value + n.value * es].view(tdt)

    def set_fusion(self, fusion: str, mode: int):
        """Select an alternative kernel arrangement (gpt2_set_fusion)."""
        _check(self.L.gpt2_set_fusion(self.handle, FUSION[fusion], int(mode)), self.handle)

    # ---- probes -------------------------------------------------------------
    def probe_enable(self, classes):
        mask = 0
        for c in classes:
            mask |= 1 << KCLASS[c]
        _check(self.L.gpt2_probe_enable(self.handle, mask), self.handle)

    def probe_reset(self):
        _check(self.L.gpt2_probe_reset(self.handle), self.handle)

    def probe_read(self, cls: str):
        ms, n = ctypes.c_double(), ctypes.c_int64()
        fl, by = ctypes.c_double(), ctypes.c_double()
        _check(self.L.gpt2_probe_read(self.handle, KCLASS[cls], ctypes.byref(ms), ctypes.byref(n),
                                      ctypes.byref(fl), ctypes.byref(by)), self.handle)
        return dict(ms=ms.value, launches=n.value, flops=fl.value, bytes=by.value)
