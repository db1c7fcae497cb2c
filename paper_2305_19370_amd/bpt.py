"""ctypes binding of libbpt (argument marshalling only).

Every step of the layer runs inside libbpt's HIP kernels. This module only
mirrors the C structs of ``include/libbpt.h``, allocates the caller-owned
buffers with torch (device memory plumbing) and passes raw pointers plus the
current HIP stream. If the library is not built, loading fails loudly; there
is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Tuple

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbpt.so")

BPT_F32, BPT_BF16 = 0, 1
BPT_GELU, BPT_RELU = 0, 1
STATUS = {0: "BPT_OK", 1: "BPT_ERR_INVALID_ARG", 2: "BPT_ERR_UNSUPPORTED", 3: "BPT_ERR_WORKSPACE",
          4: "BPT_ERR_HIP"}

c_i64, c_i32, c_f32, c_sz, c_vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_size_t, ctypes.c_void_p


class Config(ctypes.Structure):
    _fields_ = [("B", c_i64), ("S", c_i64), ("D", c_i64), ("H", c_i64), ("F", c_i64), ("Bq", c_i64),
                ("Bkv", c_i64), ("causal", c_i32), ("dtype", c_i32), ("out_dtype", c_i32),
                ("group_blocks", c_i32), ("ln_eps", c_f32), ("activation", c_i32), ("dropout", c_f32),
                ("dropout_seed", ctypes.c_uint64)]


PARAM_FIELDS = ("ln1_g", "ln1_b", "Wq", "Wk", "Wv", "Wo", "ln2_g", "ln2_b", "W1", "b1", "W2", "b2")
GRAD_FIELDS = ("dln1_g", "dln1_b", "dWq", "dWk", "dWv", "dWo", "dln2_g", "dln2_b", "dW1", "db1", "dW2", "db2")
SAVED_FIELDS = ("qkv", "o", "lse", "h", "mu1", "rstd1", "mu2", "rstd2", "total")


class Params(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in PARAM_FIELDS]


class Grads(ctypes.Structure):
    _fields_ = [(n, c_vp) for n in GRAD_FIELDS]


class SavedLayout(ctypes.Structure):
    _fields_ = [(n, c_sz) for n in SAVED_FIELDS]


class XentConfig(ctypes.Structure):
    _fields_ = [("T", c_i64), ("D", c_i64), ("V", c_i64), ("ldw", c_i64), ("block_rows", c_i64),
                ("dtype", c_i32), ("reserved", c_i32)]


class EmbedConfig(ctypes.Structure):
    _fields_ = [("B", c_i64), ("S", c_i64), ("D", c_i64), ("V", c_i64), ("dtype", c_i32), ("grad_dtype", c_i32)]


class LnConfig(ctypes.Structure):
    _fields_ = [("rows", c_i64), ("D", c_i64), ("eps", c_f32), ("in_dtype", c_i32), ("out_dtype", c_i32),
                ("reserved", c_i32)]


class AdamWConfig(ctypes.Structure):
    _fields_ = [("lr", c_f32), ("beta1", c_f32), ("beta2", c_f32), ("eps", c_f32), ("weight_decay", c_f32),
                ("lowp_dtype", c_i32), ("step", c_i64)]


EXPORTS = ("bpt_validate", "bpt_group_rows", "bpt_saved_bytes", "bpt_saved_layout_of", "bpt_workspace_bytes",
           "bpt_layer_fwd", "bpt_layer_bwd", "bpt_status_string", "bpt_last_error", "bpt_describe",
           "bpt_profile_enable", "bpt_profile_report", "bpt_xent_validate", "bpt_xent_workspace_bytes",
           "bpt_xent_fwd", "bpt_xent_bwd", "bpt_embed_fwd", "bpt_embed_bwd", "bpt_ln_workspace_bytes",
           "bpt_ln_fwd", "bpt_ln_bwd", "bpt_adamw_step", "bpt_bwd_qkv_grad_offset",
           "bpt_layer_fwd_noalloc")

_lib = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libbpt.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with __graft_entry__.build() "
                           "(python -m paper_2305_19370_amd.build)")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    lib.bpt_validate.argtypes = [P(Config)]
    lib.bpt_validate.restype = c_i32
    lib.bpt_group_rows.argtypes = [P(Config)]
    lib.bpt_group_rows.restype = c_i64
    lib.bpt_saved_bytes.argtypes = [P(Config)]
    lib.bpt_saved_bytes.restype = c_sz
    lib.bpt_saved_layout_of.argtypes = [P(Config), P(SavedLayout)]
    lib.bpt_saved_layout_of.restype = c_i32
    lib.bpt_workspace_bytes.argtypes = [P(Config), c_i32]
    lib.bpt_workspace_bytes.restype = c_sz
    lib.bpt_layer_fwd.argtypes = [P(Config), c_vp, P(Params), c_vp, c_vp, c_vp, c_sz, c_vp]
    lib.bpt_layer_fwd.restype = c_i32
    lib.bpt_layer_fwd_noalloc.argtypes = [P(Config), c_vp, P(Params), c_vp, c_vp, c_vp]
    lib.bpt_layer_fwd_noalloc.restype = c_i32
    lib.bpt_layer_bwd.argtypes = [P(Config), c_vp, P(Params), c_vp, c_vp, c_vp, P(Grads), c_vp, c_sz, c_vp]
    lib.bpt_layer_bwd.restype = c_i32
    lib.bpt_bwd_qkv_grad_offset.argtypes = [P(Config), P(c_sz)]
    lib.bpt_bwd_qkv_grad_offset.restype = c_i32
    lib.bpt_status_string.argtypes = [c_i32]
    lib.bpt_status_string.restype = ctypes.c_char_p
    lib.bpt_last_error.argtypes = []
    lib.bpt_last_error.restype = ctypes.c_char_p
    lib.bpt_describe.argtypes = [P(Config), ctypes.c_char_p, c_sz]
    lib.bpt_describe.restype = c_sz
    lib.bpt_profile_enable.argtypes = [c_i32]
    lib.bpt_profile_enable.restype = c_i32
    lib.bpt_profile_report.argtypes = [ctypes.c_char_p, c_sz]
    lib.bpt_profile_report.restype = c_sz
    lib.bpt_xent_validate.argtypes = [P(XentConfig)]
    lib.bpt_xent_validate.restype = c_i32
    lib.bpt_xent_workspace_bytes.argtypes = [P(XentConfig), c_i32]
    lib.bpt_xent_workspace_bytes.restype = c_sz
    lib.bpt_xent_fwd.argtypes = [P(XentConfig), c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    lib.bpt_xent_fwd.restype = c_i32
    lib.bpt_xent_bwd.argtypes = [P(XentConfig), c_vp, c_vp, c_vp, c_vp, c_f32, c_vp, c_vp, c_vp, c_sz, c_vp]
    lib.bpt_xent_bwd.restype = c_i32
    lib.bpt_embed_fwd.argtypes = [P(EmbedConfig), c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.bpt_embed_fwd.restype = c_i32
    lib.bpt_embed_bwd.argtypes = [P(EmbedConfig), c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.bpt_embed_bwd.restype = c_i32
    lib.bpt_ln_workspace_bytes.argtypes = [P(LnConfig)]
    lib.bpt_ln_workspace_bytes.restype = c_sz
    lib.bpt_ln_fwd.argtypes = [P(LnConfig), c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.bpt_ln_fwd.restype = c_i32
    lib.bpt_ln_bwd.argtypes = [P(LnConfig), c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp, c_sz, c_vp]
    lib.bpt_ln_bwd.restype = c_i32
    lib.bpt_adamw_step.argtypes = [P(AdamWConfig), c_i64, c_vp, c_vp, c_vp, c_vp, c_vp, c_vp]
    lib.bpt_adamw_step.restype = c_i32
    _lib = lib
    return lib


class BptError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def _check(status: int) -> None:
    if status != 0:
        raise BptError(status, load().bpt_last_error().decode())


def make_config(B: int, S: int, D: int, H: int, F: int, Bq: int, Bkv: int, causal: bool = True,
                dtype: str = "bf16", out_dtype: Optional[str] = None, group_blocks: int = 0,
                ln_eps: float = 1e-5, activation: str = "gelu", dropout: float = 0.0,
                dropout_seed: int = 0) -> Config:
    dt = {"f32": BPT_F32, "bf16": BPT_BF16}
    act = {"gelu": BPT_GELU, "relu": BPT_RELU}
    return Config(B, S, D, H, F, Bq, Bkv, int(bool(causal)), dt[dtype], dt[out_dtype or dtype],
                  group_blocks, ln_eps, act[activation], dropout, dropout_seed & (2 ** 64 - 1))


def validate(cfg: Config) -> int:
    return load().bpt_validate(ctypes.byref(cfg))


def saved_bytes(cfg: Config) -> int:
    return load().bpt_saved_bytes(ctypes.byref(cfg))


def workspace_bytes(cfg: Config, backward: bool) -> int:
    return load().bpt_workspace_bytes(ctypes.byref(cfg), int(backward))


def group_rows(cfg: Config) -> int:
    return load().bpt_group_rows(ctypes.byref(cfg))


def saved_layout(cfg: Config) -> Dict[str, int]:
    out = SavedLayout()
    _check(load().bpt_saved_layout_of(ctypes.byref(cfg), ctypes.byref(out)))
    return {n: getattr(out, n) for n in SAVED_FIELDS}


def bwd_qkv_grad_offset(cfg: Config) -> int:
    off = c_sz()
    _check(load().bpt_bwd_qkv_grad_offset(ctypes.byref(cfg), ctypes.byref(off)))
    return off.value


def describe(cfg: Config) -> str:
    buf = ctypes.create_string_buffer(1024)
    load().bpt_describe(ctypes.byref(cfg), buf, 1024)
    return buf.value.decode()


def profile_enable(on: bool) -> None:
    _check(load().bpt_profile_enable(int(on)))


def profile_report() -> Dict[str, Dict[str, float]]:
    """Per call-site launch timings recorded since profile_enable(True); call after a
    device synchronisation."""
    import json
    lib = load()
    n = lib.bpt_profile_report(None, 0)
    buf = ctypes.create_string_buffer(n + 1)
    lib.bpt_profile_report(buf, n + 1)
    return json.loads(buf.value.decode())


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def params_struct(params: Dict[str, Optional[torch.Tensor]]) -> Params:
    return Params(*[_ptr(params.get(n)) for n in PARAM_FIELDS])


def layer_fwd(cfg: Config, X: torch.Tensor, params: Dict[str, Optional[torch.Tensor]], Y: torch.Tensor,
              saved: torch.Tensor, workspace: torch.Tensor) -> None:
    p = params_struct(params)
    _check(load().bpt_layer_fwd(ctypes.byref(cfg), X.data_ptr(), ctypes.byref(p), Y.data_ptr(),
                                saved.data_ptr(), workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                _stream()))


NOALLOC_SCRATCH_BYTES = 64 << 20


def layer_fwd_noalloc(cfg: Config, X: torch.Tensor, params: Dict[str, Optional[torch.Tensor]], Y: torch.Tensor,
                      saved: torch.Tensor) -> None:
    """bpt_layer_fwd_noalloc: the forward with the library's static scratch as workspace."""
    p = params_struct(params)
    _check(load().bpt_layer_fwd_noalloc(ctypes.byref(cfg), X.data_ptr(), ctypes.byref(p), Y.data_ptr(),
                                        saved.data_ptr(), _stream()))


def layer_bwd(cfg: Config, X: torch.Tensor, params: Dict[str, Optional[torch.Tensor]], saved: torch.Tensor,
              dY: torch.Tensor, dX: torch.Tensor, grads: Dict[str, Optional[torch.Tensor]],
              workspace: torch.Tensor) -> None:
    p = params_struct(params)
    g = Grads(*[_ptr(grads.get(n)) for n in GRAD_FIELDS])
    _check(load().bpt_layer_bwd(ctypes.byref(cfg), X.data_ptr(), ctypes.byref(p), saved.data_ptr(),
                                dY.data_ptr(), dX.data_ptr(), ctypes.byref(g), workspace.data_ptr(),
                                workspace.numel() * workspace.element_size(), _stream()))


_TORCH_DT = {BPT_F32: torch.float32, BPT_BF16: torch.bfloat16}


class Layer:
    """One BPT layer: owns nothing but the buffers it allocates through torch."""

    def __init__(self, cfg: Config, device: str = "cuda"):
        _check(validate(cfg))
        self.cfg, self.device = cfg, device
        self.out_dtype = _TORCH_DT[cfg.out_dtype]

    def _bytes(self, n: int) -> torch.Tensor:
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.device)

    def forward(self, X: torch.Tensor, params: Dict[str, Optional[torch.Tensor]],
                workspace: Optional[torch.Tensor] = None) -> Tuple[torch.Tensor, torch.Tensor]:
        Y = torch.empty(X.shape, dtype=self.out_dtype, device=self.device)
        saved = self._bytes(saved_bytes(self.cfg))
        ws = workspace if workspace is not None else self._bytes(workspace_bytes(self.cfg, False))
        layer_fwd(self.cfg, X, params, Y, saved, ws)
        return Y, saved

    def backward(self, X: torch.Tensor, params: Dict[str, Optional[torch.Tensor]], saved: torch.Tensor,
                 dY: torch.Tensor, want: Optional[Tuple[str, ...]] = None,
                 workspace: Optional[torch.Tensor] = None,
                 qkv_grads: bool = False) -> Tuple[torch.Tensor, Dict[str, torch.Tensor]]:
        """dX and the parameter gradients; with qkv_grads, also "dQ", "dK", "dV" [B, S, D]
        (copies of what the backward leaves in its workspace, bpt_bwd_qkv_grad_offset)."""
        D, F = self.cfg.D, self.cfg.F
        shapes = {"dln1_g": (D,), "dln1_b": (D,), "dWq": (D, D), "dWk": (D, D), "dWv": (D, D), "dWo": (D, D),
                  "dln2_g": (D,), "dln2_b": (D,), "dW1": (D, F), "db1": (F,), "dW2": (F, D), "db2": (D,)}
        src = {"dln1_g": "ln1_g", "dln1_b": "ln1_b", "dln2_g": "ln2_g", "dln2_b": "ln2_b", "db1": "b1", "db2": "b2"}
        grads = {}
        for n, shp in shapes.items():
            if want is not None and n not in want:
                continue
            if n in src and params.get(src[n]) is None:
                continue
            grads[n] = torch.empty(shp, dtype=torch.float32, device=self.device)
        dX = torch.empty(X.shape, dtype=self.out_dtype, device=self.device)
        ws = workspace if workspace is not None else self._bytes(workspace_bytes(self.cfg, True))
        layer_bwd(self.cfg, X, params, saved, dY, dX, grads, ws)
        if qkv_grads:
            c = self.cfg
            E = _TORCH_DT[c.dtype]
            Sp = (c.S + 63) // 64 * 64
            off, n = bwd_qkv_grad_offset(c), 3 * c.D * c.B * Sp
            m = ws[off:off + n * (2 if E == torch.bfloat16 else 4)].view(E).view(3, c.D, c.B, Sp)[..., :c.S]
            for i, name in enumerate(("dQ", "dK", "dV")):
                grads[name] = m[i].permute(1, 2, 0).contiguous()
        return dX, grads

    def saved_views(self, saved: torch.Tensor) -> Dict[str, torch.Tensor]:
        """Typed views of the saved activations (see bpt_saved_layout in include/libbpt.h)."""
        c = self.cfg
        lay = saved_layout(c)
        E = _TORCH_DT[c.dtype]
        T, D, Sp = c.B * c.S, c.D, (c.S + 63) // 64 * 64

        def view(name, n, dt, shape):
            off = lay[name]
            nbytes = n * (2 if dt == torch.bfloat16 else 4)
            return saved[off:off + nbytes].view(dt).view(*shape)

        return {
            "qkv": view("qkv", T * 3 * D, E, (T, 3 * D)),
            "o": view("o", T * D, E, (T, D)),
            "lse": view("lse", c.B * c.H * Sp, torch.float32, (c.B, c.H, Sp)),
            "h": view("h", T * D, torch.float32, (T, D)),
            "mu1": view("mu1", T, torch.float32, (T,)),
            "rstd1": view("rstd1", T, torch.float32, (T,)),
            "mu2": view("mu2", T, torch.float32, (T,)),
            "rstd2": view("rstd2", T, torch.float32, (T,)),
        }


# ---------------------------------------------------------------- cross-entropy of an LM head
def make_xent_config(T: int, D: int, V: int, ldw: Optional[int] = None, block_rows: int = 0,
                     dtype: str = "bf16") -> XentConfig:
    dt = {"f32": BPT_F32, "bf16": BPT_BF16}
    return XentConfig(T, D, V, ldw if ldw is not None else (V + 63) // 64 * 64, block_rows, dt[dtype], 0)


def xent_validate(cfg: XentConfig) -> int:
    return load().bpt_xent_validate(ctypes.byref(cfg))


def xent_workspace_bytes(cfg: XentConfig, backward: bool) -> int:
    return load().bpt_xent_workspace_bytes(ctypes.byref(cfg), int(backward))


def xent_fwd(cfg: XentConfig, h: torch.Tensor, W: torch.Tensor, targets: torch.Tensor, loss: torch.Tensor,
             lse: torch.Tensor, workspace: torch.Tensor) -> None:
    _check(load().bpt_xent_fwd(ctypes.byref(cfg), h.data_ptr(), W.data_ptr(), targets.data_ptr(),
                               loss.data_ptr(), lse.data_ptr(), workspace.data_ptr(),
                               workspace.numel() * workspace.element_size(), _stream()))


def xent_bwd(cfg: XentConfig, h: torch.Tensor, W: torch.Tensor, targets: torch.Tensor, lse: torch.Tensor,
             dloss: float, dh: torch.Tensor, dW: Optional[torch.Tensor], workspace: torch.Tensor) -> None:
    _check(load().bpt_xent_bwd(ctypes.byref(cfg), h.data_ptr(), W.data_ptr(), targets.data_ptr(),
                               lse.data_ptr(), float(dloss), dh.data_ptr(), _ptr(dW), workspace.data_ptr(),
                               workspace.numel() * workspace.element_size(), _stream()))


class LMHeadLoss:
    """Cross-entropy of an LM head through libbpt; allocates its buffers with torch."""

    def __init__(self, cfg: XentConfig, device: str = "cuda"):
        _check(xent_validate(cfg))
        self.cfg, self.device = cfg, device

    def _bytes(self, n: int) -> torch.Tensor:
        return torch.empty(max(n, 256), dtype=torch.uint8, device=self.device)

    def forward(self, h: torch.Tensor, W: torch.Tensor, targets: torch.Tensor) -> Tuple[torch.Tensor, torch.Tensor]:
        loss = torch.empty(1, dtype=torch.float32, device=self.device)
        lse = torch.empty(self.cfg.T, dtype=torch.float32, device=self.device)
        xent_fwd(self.cfg, h, W, targets, loss, lse, self._bytes(xent_workspace_bytes(self.cfg, False)))
        return loss, lse

    def backward(self, h: torch.Tensor, W: torch.Tensor, targets: torch.Tensor, lse: torch.Tensor,
                 dloss: float = 1.0, want_dW: bool = True) -> Tuple[torch.Tensor, Optional[torch.Tensor]]:
        dh = torch.empty(h.shape, dtype=h.dtype, device=self.device)
        dW = torch.empty((self.cfg.D, self.cfg.ldw), dtype=torch.float32, device=self.device) if want_dW else None
        xent_bwd(self.cfg, h, W, targets, lse, dloss, dh, dW, self._bytes(xent_workspace_bytes(self.cfg, True)))
        return dh, dW


# ---------------------------------------------------------------- GPT training step pieces
_DT = {"f32": BPT_F32, "bf16": BPT_BF16}


def make_embed_config(B: int, S: int, D: int, V: int, dtype: str = "bf16", grad_dtype: Optional[str] = None):
    return EmbedConfig(B, S, D, V, _DT[dtype], _DT[grad_dtype or dtype])


def embed_fwd(cfg: EmbedConfig, tokens: torch.Tensor, Wte: torch.Tensor, Wpe: Optional[torch.Tensor],
              X: torch.Tensor) -> None:
    _check(load().bpt_embed_fwd(ctypes.byref(cfg), tokens.data_ptr(), Wte.data_ptr(), _ptr(Wpe), X.data_ptr(),
                                _stream()))


def embed_bwd(cfg: EmbedConfig, tokens: torch.Tensor, dX: torch.Tensor, dWte: Optional[torch.Tensor],
              dWpe: Optional[torch.Tensor]) -> None:
    _check(load().bpt_embed_bwd(ctypes.byref(cfg), tokens.data_ptr(), dX.data_ptr(), _ptr(dWte), _ptr(dWpe),
                                _stream()))


def make_ln_config(rows: int, D: int, eps: float = 1e-5, in_dtype: str = "bf16",
                   out_dtype: Optional[str] = None) -> LnConfig:
    return LnConfig(rows, D, eps, _DT[in_dtype], _DT[out_dtype or in_dtype], 0)


def ln_workspace_bytes(cfg: LnConfig) -> int:
    return load().bpt_ln_workspace_bytes(ctypes.byref(cfg))


def ln_fwd(cfg: LnConfig, X: torch.Tensor, g: Optional[torch.Tensor], b: Optional[torch.Tensor], Y: torch.Tensor,
           mean: torch.Tensor, rstd: torch.Tensor) -> None:
    _check(load().bpt_ln_fwd(ctypes.byref(cfg), X.data_ptr(), _ptr(g), _ptr(b), Y.data_ptr(), mean.data_ptr(),
                             rstd.data_ptr(), _stream()))


def ln_bwd(cfg: LnConfig, X: torch.Tensor, g: Optional[torch.Tensor], mean: torch.Tensor, rstd: torch.Tensor,
           dY: torch.Tensor, dX: torch.Tensor, dg: Optional[torch.Tensor], db: Optional[torch.Tensor],
           workspace: torch.Tensor) -> None:
    _check(load().bpt_ln_bwd(ctypes.byref(cfg), X.data_ptr(), _ptr(g), mean.data_ptr(), rstd.data_ptr(),
                             dY.data_ptr(), dX.data_ptr(), _ptr(dg), _ptr(db), workspace.data_ptr(),
                             workspace.numel() * workspace.element_size(), _stream()))


def adamw_step(p: torch.Tensor, g: torch.Tensor, m: torch.Tensor, v: torch.Tensor, step: int, lr: float,
               beta1: float = 0.9, beta2: float = 0.95, eps: float = 1e-8, weight_decay: float = 0.1,
               p_lowp: Optional[torch.Tensor] = None) -> None:
    """One AdamW update of the fp32 tensor p (in place, with its moments m, v); p_lowp,
    if given, receives p rounded to its dtype."""
    lowp = BPT_BF16 if p_lowp is not None and p_lowp.dtype == torch.bfloat16 else BPT_F32
    cfg = AdamWConfig(lr, beta1, beta2, eps, weight_decay, lowp, step)
    _check(load().bpt_adamw_step(ctypes.byref(cfg), p.numel(), p.data_ptr(), g.data_ptr(), m.data_ptr(),
                                 v.data_ptr(), _ptr(p_lowp), _stream()))
