"""Thin ctypes binding of libfal.so (the C ABI in include/fal.h).

Everything here is argument marshalling: flattening parameter dicts into the
library's layout, device buffers owned by PyTorch, and status checking.  All
computation of the training step happens in the library's HIP kernels.  If
libfal.so is missing the import of :func:`lib` raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, byref, c_char_p, c_double, c_float, c_int32, c_int64, c_size_t, c_void_p

import numpy as np

from .config import Config
from .synth import BLOCK_NAMES, GLOBAL_NAMES

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfal.so")

FAL_OK, FAL_ERR_INVALID_ARG, FAL_ERR_UNSUPPORTED, FAL_ERR_WORKSPACE, FAL_ERR_HIP, FAL_ERR_STATE = range(6)

# Order of the FAL_P_* and FAL_B_* enums in include/fal.h.
GLOBAL_TENSORS = GLOBAL_NAMES
BLOCK_TENSORS = BLOCK_NAMES

ABI_FUNCTIONS = (
    "fal_validate_config", "fal_param_layout", "fal_workspace_bytes", "fal_init", "fal_destroy",
    "fal_block_fwd", "fal_block_bwd", "fal_model_step", "fal_stack_step", "fal_residual_out",
    "fal_profile_enable", "fal_profile_read", "fal_status_string", "fal_last_error", "fal_adamw_step",
    "fal_model_forward", "fal_stack_forward", "fal_adamw_step_noalloc",
)
PROF_GEMM, PROF_ATTN_FWD, PROF_ATTN_BWD, PROF_NORM, PROF_CE, PROF_EMBED, PROF_BIAS, PROF_OPTIM = range(8)
PROF_NAMES = {PROF_GEMM: "gemm", PROF_ATTN_FWD: "attn_fwd", PROF_ATTN_BWD: "attn_bwd", PROF_NORM: "norm",
              PROF_CE: "cross_entropy", PROF_EMBED: "embedding", PROF_BIAS: "bias_grad", PROF_OPTIM: "optimizer"}

# AdamW settings of the paper's training setups (appendix: lr 1e-4, weight
# decay 0.001, clip-grad-norm 1) with the usual beta and eps defaults.
ADAMW_PAPER = {"lr": 1e-4, "beta1": 0.9, "beta2": 0.999, "eps": 1e-8, "weight_decay": 1e-3,
               "max_grad_norm": 1.0}


class fal_config_t(ctypes.Structure):
    _fields_ = [
        ("n_layer", c_int32), ("d_model", c_int32), ("n_head", c_int32), ("head_dim", c_int32),
        ("d_ff", c_int32), ("vocab", c_int32), ("seq_len", c_int32), ("batch", c_int32),
        ("arch", c_int32), ("dtype", c_int32), ("sched", c_int32), ("ln_eps", c_float),
        ("gelu_tanh", c_int32), ("has_embed_head", c_int32), ("fal_block1_mode", c_int32),
        ("bidirectional", c_int32), ("n_kv_head", c_int32),
    ]


class fal_adamw_t(ctypes.Structure):
    _fields_ = [("lr", c_float), ("beta1", c_float), ("beta2", c_float), ("eps", c_float),
                ("weight_decay", c_float), ("max_grad_norm", c_float)]


def adamw_params(**hp) -> fal_adamw_t:
    v = dict(ADAMW_PAPER)
    v.update(hp)
    return fal_adamw_t(**{k: float(v[k]) for k in ADAMW_PAPER})


class FalError(RuntimeError):
    def __init__(self, status, msg=""):
        self.status = status
        super().__init__(f"libfal status {status}: {msg}")


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise FalError(-1, f"{LIB_PATH} is not built (python -m paper_2510_14614_amd.build)")
        L = ctypes.CDLL(LIB_PATH)
        cfgp = POINTER(fal_config_t)
        L.fal_validate_config.argtypes = [cfgp]
        L.fal_param_layout.argtypes = [cfgp, POINTER(c_int64), POINTER(c_int64), POINTER(c_int64),
                                       POINTER(c_int64), POINTER(c_int64)]
        L.fal_workspace_bytes.argtypes = [cfgp, POINTER(c_size_t)]
        L.fal_init.argtypes = [cfgp, c_void_p, c_size_t, c_void_p, c_void_p, POINTER(c_void_p)]
        L.fal_destroy.argtypes = [c_void_p]
        L.fal_block_fwd.argtypes = [c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_block_bwd.argtypes = [c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                    c_void_p, c_void_p, c_void_p]
        L.fal_model_step.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_stack_step.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_model_forward.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_stack_forward.argtypes = [c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_residual_out.argtypes = [c_void_p, POINTER(c_void_p)]
        L.fal_profile_enable.argtypes = [c_void_p, c_int32]
        L.fal_profile_read.argtypes = [c_void_p, c_int32, POINTER(c_int64), POINTER(c_double),
                                       POINTER(c_double), POINTER(c_double)]
        L.fal_adamw_step.argtypes = [c_void_p, POINTER(fal_adamw_t), c_int64, c_int64, c_void_p, c_void_p,
                                     c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_adamw_step_noalloc.argtypes = [POINTER(fal_adamw_t), c_int64, c_int64, c_int32, c_void_p, c_void_p,
                                             c_void_p, c_void_p, c_void_p, c_void_p, c_void_p]
        L.fal_status_string.argtypes = [c_int32]
        L.fal_status_string.restype = c_char_p
        L.fal_last_error.argtypes = [c_void_p]
        L.fal_last_error.restype = c_char_p
        for name in ABI_FUNCTIONS:
            if name not in ("fal_status_string", "fal_last_error"):
                getattr(L, name).restype = c_int32
        _LIB = L
    return _LIB


def to_c(cfg: Config) -> fal_config_t:
    return fal_config_t(cfg.n_layer, cfg.d_model, cfg.n_head, cfg.head_dim, cfg.d_ff, cfg.vocab,
                        cfg.seq_len, cfg.batch, cfg.arch, cfg.dtype, cfg.sched, cfg.ln_eps,
                        cfg.gelu_tanh, cfg.has_embed_head, cfg.fal_block1_mode, cfg.bidirectional,
                        cfg.n_kv_head)


def _check(status, ctx=None):
    if status != FAL_OK:
        L = lib()
        msg = L.fal_last_error(ctx).decode() if ctx else ""
        name = L.fal_status_string(status).decode()
        raise FalError(status, f"{name}: {msg}")


def validate_config(cfg: Config) -> int:
    c = to_c(cfg)
    return lib().fal_validate_config(byref(c))


def param_layout(cfg: Config) -> dict:
    c = to_c(cfg)
    g = (c_int64 * 4)()
    b = (c_int64 * 14)()
    base, stride, total = c_int64(), c_int64(), c_int64()
    _check(lib().fal_param_layout(byref(c), g, b, byref(base), byref(stride), byref(total)))
    return {"global": list(g), "block": list(b), "block_base": base.value,
            "block_stride": stride.value, "total": total.value}


def workspace_bytes(cfg: Config) -> int:
    c = to_c(cfg)
    n = c_size_t()
    _check(lib().fal_workspace_bytes(byref(c), byref(n)))
    return n.value


def flatten_params(cfg: Config, gparams: dict, blocks: list, layout: dict | None = None) -> np.ndarray:
    """Host float32 flat buffer in the library's parameter layout."""
    lay = layout or param_layout(cfg)
    flat = np.zeros(lay["total"], dtype=np.float32)
    if cfg.has_embed_head:
        for k, name in enumerate(GLOBAL_TENSORS):
            a = np.asarray(gparams[name], dtype=np.float32).reshape(-1)
            flat[lay["global"][k]:lay["global"][k] + a.size] = a
    for i, blk in enumerate(blocks):
        base = lay["block_base"] + i * lay["block_stride"]
        for k, name in enumerate(BLOCK_TENSORS):
            a = np.asarray(blk[name], dtype=np.float32).reshape(-1)
            o = base + lay["block"][k]
            flat[o:o + a.size] = a
    return flat


def unflatten(cfg: Config, flat: np.ndarray, gshapes: dict, bshapes: dict, layout: dict | None = None):
    """Inverse of flatten_params for a host float32 buffer (gradients)."""
    lay = layout or param_layout(cfg)
    g = {}
    if cfg.has_embed_head:
        for k, name in enumerate(GLOBAL_TENSORS):
            n = int(np.prod(gshapes[name]))
            g[name] = flat[lay["global"][k]:lay["global"][k] + n].reshape(gshapes[name]).copy()
    blocks = []
    for i in range(cfg.n_layer):
        base = lay["block_base"] + i * lay["block_stride"]
        d = {}
        for k, name in enumerate(BLOCK_TENSORS):
            n = int(np.prod(bshapes[name]))
            o = base + lay["block"][k]
            d[name] = flat[o:o + n].reshape(bshapes[name]).copy()
        blocks.append(d)
    return g, blocks


def adamw_step_noalloc(hp: fal_adamw_t, step: int, n: int, dtype: int, master, params, grads, m, v,
                       grad_norm=None, stream=None):
    """fal_adamw_step_noalloc on torch device tensors (no context, no
    allocation): one AdamW update of n elements on `stream` (a torch stream;
    None: the current stream)."""
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    ptr = lambda t: c_void_p(t.data_ptr()) if t is not None else None  # noqa: E731
    st = lib().fal_adamw_step_noalloc(byref(hp), step, n, dtype, ptr(master), ptr(params), ptr(grads), ptr(m), ptr(v),
                                      ptr(grad_norm), c_void_p(s.cuda_stream))
    if st != FAL_OK:
        L = lib()
        raise FalError(st, f"{L.fal_status_string(st).decode()}: {L.fal_last_error(None).decode()}")


class Fal:
    """A libfal context with PyTorch-owned device buffers on the current GPU."""

    def __init__(self, cfg: Config, stream_main=None, stream_aux=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.layout = param_layout(cfg)
        self.ws_bytes = workspace_bytes(cfg)
        dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        self._ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=dev)
        ptr = self._ws.data_ptr()
        self.ws_ptr = (ptr + 255) // 256 * 256
        self.stream_main = stream_main if stream_main is not None else torch.cuda.current_stream(dev)
        self.stream_aux = stream_aux if stream_aux is not None else torch.cuda.Stream(dev)
        self.pdtype = torch.bfloat16 if cfg.dtype == 1 else torch.float32
        self.params = torch.zeros(self.layout["total"], dtype=self.pdtype, device=dev)
        self.grads = torch.zeros(self.layout["total"], dtype=torch.float32, device=dev)
        self.loss = torch.zeros(1, dtype=torch.float32, device=dev)
        c = to_c(cfg)
        self._ccfg = c
        ctx = c_void_p()
        _check(lib().fal_init(byref(c), c_void_p(self.ws_ptr), self.ws_bytes,
                              c_void_p(self.stream_main.cuda_stream), c_void_p(self.stream_aux.cuda_stream),
                              byref(ctx)))
        self.ctx = ctx

    def close(self):
        if getattr(self, "ctx", None):
            lib().fal_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -------------------------------------------------------------- params --
    def load_params(self, gparams: dict, blocks: list):
        flat = flatten_params(self.cfg, gparams, blocks, self.layout)
        t = self.torch.from_numpy(flat).to(self.pdtype)
        self.params.copy_(t.to(self.device))

    def block_param_ptr(self, i: int) -> int:
        es = self.params.element_size()
        return self.params.data_ptr() + (self.layout["block_base"] + i * self.layout["block_stride"]) * es

    def block_grad_ptr(self, i: int) -> int:
        return self.grads.data_ptr() + (self.layout["block_base"] + i * self.layout["block_stride"]) * 4

    def grads_numpy(self):
        from .synth import block_shapes, global_shapes
        flat = self.grads.detach().cpu().numpy()
        return unflatten(self.cfg, flat, global_shapes(self.cfg), block_shapes(self.cfg), self.layout)

    # ---------------------------------------------------------------- calls --
    def model_step(self, tokens, logits=None):
        """tokens: int32 device tensor [B, T+1]; logits: optional fp32 device
        tensor [B*T, V].  Returns the loss tensor (device, shape [1])."""
        assert tokens.dtype == self.torch.int32 and tokens.is_cuda and tokens.is_contiguous()
        lp = c_void_p(logits.data_ptr()) if logits is not None else None
        _check(lib().fal_model_step(self.ctx, c_void_p(self.params.data_ptr()), c_void_p(tokens.data_ptr()),
                                    c_void_p(self.loss.data_ptr()), lp, c_void_p(self.grads.data_ptr())),
               self.ctx)
        return self.loss

    def model_forward(self, tokens, logits=None, loss=True):
        """Forward only (no gradients).  Returns the loss tensor (device [1])
        when loss is True, else None."""
        assert tokens.dtype == self.torch.int32 and tokens.is_cuda and tokens.is_contiguous()
        lp = c_void_p(logits.data_ptr()) if logits is not None else None
        _check(lib().fal_model_forward(self.ctx, c_void_p(self.params.data_ptr()), c_void_p(tokens.data_ptr()),
                                       c_void_p(self.loss.data_ptr()) if loss else None, lp), self.ctx)
        return self.loss if loss else None

    def stack_forward(self, x_in, x_out=None):
        _check(lib().fal_stack_forward(self.ctx, c_void_p(self.params.data_ptr()), c_void_p(x_in.data_ptr()),
                                       c_void_p(x_out.data_ptr()) if x_out is not None else None), self.ctx)

    def stack_step(self, x_in, dy, dx_in=None):
        _check(lib().fal_stack_step(self.ctx, c_void_p(self.params.data_ptr()), c_void_p(x_in.data_ptr()),
                                    c_void_p(dy.data_ptr()), c_void_p(self.loss.data_ptr()),
                                    c_void_p(self.grads.data_ptr()),
                                    c_void_p(dx_in.data_ptr()) if dx_in is not None else None), self.ctx)
        return self.loss

    def block_fwd(self, layer, x_in, x_out, first):
        _check(lib().fal_block_fwd(self.ctx, layer, c_void_p(self.block_param_ptr(layer)),
                                   c_void_p(x_in.data_ptr()), c_void_p(x_out.data_ptr()),
                                   c_void_p(first.data_ptr()) if first is not None else None), self.ctx)

    def block_bwd(self, layer, x_in, first, dx_out, dx_in, dfirst):
        _check(lib().fal_block_bwd(self.ctx, layer, c_void_p(self.block_param_ptr(layer)),
                                   c_void_p(x_in.data_ptr()),
                                   c_void_p(first.data_ptr()) if first is not None else None,
                                   c_void_p(dx_out.data_ptr()),
                                   c_void_p(dx_in.data_ptr()),
                                   c_void_p(dfirst.data_ptr()) if dfirst is not None else None,
                                   c_void_p(self.block_grad_ptr(layer))), self.ctx)

    # ----------------------------------------------------------- optimizer --
    def init_optimizer(self):
        """fp32 master weights (copied from the current parameters) and zero
        AdamW moments, all in the flat parameter layout."""
        torch = self.torch
        self.master = self.params.float().clone() if self.cfg.dtype == 1 else self.params
        self.m = torch.zeros_like(self.grads)
        self.v = torch.zeros_like(self.grads)
        self.grad_norm = torch.zeros(1, dtype=torch.float32, device=self.device)
        self.opt_step = 0

    def adamw_step(self, **hp):
        """One AdamW update of every parameter from self.grads (defaults: the
        paper's lr 1e-4, weight decay 0.001, clip 1).  Returns the pre-clip
        gradient norm (device tensor [1])."""
        if getattr(self, "master", None) is None:
            self.init_optimizer()
        self.opt_step += 1
        p = adamw_params(**hp)
        lp = c_void_p(self.params.data_ptr()) if self.cfg.dtype == 1 else None
        _check(lib().fal_adamw_step(self.ctx, byref(p), self.opt_step, self.layout["total"],
                                    c_void_p(self.master.data_ptr()), lp, c_void_p(self.grads.data_ptr()),
                                    c_void_p(self.m.data_ptr()), c_void_p(self.v.data_ptr()),
                                    c_void_p(self.grad_norm.data_ptr())), self.ctx)
        return self.grad_norm

    def train_step(self, tokens, **hp):
        """Forward + backward (fal_model_step) and one AdamW update; returns
        the loss of the batch before the update (device tensor [1])."""
        self.model_step(tokens)
        self.adamw_step(**hp)
        return self.loss

    def profile_enable(self, on: bool = True):
        _check(lib().fal_profile_enable(self.ctx, 1 if on else 0), self.ctx)

    def profile_read(self) -> dict:
        out = {}
        for cls, name in PROF_NAMES.items():
            n, ms, fl, by = c_int64(), c_double(), c_double(), c_double()
            _check(lib().fal_profile_read(self.ctx, cls, byref(n), byref(ms), byref(fl), byref(by)), self.ctx)
            out[name] = {"launches": n.value, "ms": ms.value, "flops": fl.value, "bytes": by.value}
        return out

    def residual_out(self):
        p = c_void_p()
        _check(lib().fal_residual_out(self.ctx, byref(p)))
        return p.value
