"""An L-layer GPT training step on libbpt (the models of Section 5, Table 1 shapes).

    X_0 = Wte[tokens] + Wpe[positions]        bpt_embed_fwd
    X_{l+1} = BPT layer l (X_l)               bpt_layer_fwd, saving what its backward needs
    h = LN_f(X_L)                             bpt_ln_fwd
    loss = cross-entropy of h Wout            bpt_xent_fwd (blockwise over tokens)

then the backward in reverse through bpt_xent_bwd, bpt_ln_bwd, bpt_layer_bwd per layer
and bpt_embed_bwd, and AdamW (bpt_adamw_step) on fp32 master weights, which also
writes the bf16 copies the kernels read. Every step runs in libbpt's kernels; this
module allocates the buffers (torch) and sequences the calls on the current stream.

Parameters live in two flat fp32 buffers (weight matrices and embeddings, which take
weight decay; LayerNorm gains/shifts and biases, which do not), each with matching
flat gradient and moment buffers, so one optimiser step is two launches. Entries
start on 256-byte boundaries; the gaps stay zero (zero gradient, zero update).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import torch

from . import bpt

LAYER_MATS = ("Wq", "Wk", "Wv", "Wo", "W1", "W2")
LAYER_VECS = ("ln1_g", "ln1_b", "ln2_g", "ln2_b", "b1", "b2")


@dataclasses.dataclass
class GPTShape:
    L: int
    B: int
    S: int
    D: int
    H: int
    F: int
    V: int
    Bq: int = 1024
    Bkv: int = 1024
    dtype: str = "bf16"            # "bf16" (weights, activations) or "f32"
    activation: str = "gelu"
    biases: bool = True            # FFN biases b1, b2
    pos_table: bool = True         # learned position table Wpe
    causal: bool = True
    ln_eps: float = 1e-5
    xent_block_rows: int = 0       # 0 = the library's default
    dropout: float = 0.0           # residual-branch dropout rate of every layer
    dropout_seed: int = 0          # base of the per-layer, per-step mask keys

    @property
    def ldw(self) -> int:
        return (self.V + 63) // 64 * 64

    def n_params(self) -> int:
        per = 4 * self.D * self.D + 2 * self.D * self.F + 4 * self.D + (self.F + self.D if self.biases else 0)
        return (self.L * per + self.V * self.D + (self.S * self.D if self.pos_table else 0)
                + 2 * self.D + self.D * self.V)


class _Flat:
    """One flat group of fp32 parameters with gradient, moments and a low-precision copy."""

    def __init__(self, shapes: List[Tuple[str, Tuple[int, ...]]], device, lowp: Optional[torch.dtype]):
        self.index: Dict[str, Tuple[int, Tuple[int, ...]]] = {}
        off = 0
        for name, shp in shapes:
            self.index[name] = (off, shp)
            off += (math.prod(shp) + 63) // 64 * 64
        self.n = max(off, 64)
        z = lambda dt: torch.zeros(self.n, dtype=dt, device=device)
        self.p, self.g, self.m, self.v = z(torch.float32), z(torch.float32), z(torch.float32), z(torch.float32)
        self.low = z(lowp) if lowp is not None else None

    def view(self, buf: torch.Tensor, name: str) -> torch.Tensor:
        off, shp = self.index[name]
        return buf[off:off + math.prod(shp)].view(shp)


class GPT:
    """Buffers and call sequence of one GPT training step through libbpt."""

    def __init__(self, shape: GPTShape, device: str = "cuda", seed: int = 0, init: bool = True):
        s = self.shape = shape
        self.device = device
        self.tdt = torch.bfloat16 if s.dtype == "bf16" else torch.float32
        lowp = torch.bfloat16 if s.dtype == "bf16" else None
        self.cfg = bpt.make_config(s.B, s.S, s.D, s.H, s.F, s.Bq, s.Bkv, causal=s.causal, dtype=s.dtype,
                                   out_dtype=s.dtype, ln_eps=s.ln_eps, activation=s.activation,
                                   dropout=s.dropout)
        bpt._check(bpt.validate(self.cfg))
        T = s.B * s.S
        self.xcfg = bpt.make_xent_config(T, s.D, s.V, ldw=s.ldw, block_rows=s.xent_block_rows, dtype=s.dtype)
        bpt._check(bpt.xent_validate(self.xcfg))
        self.ecfg = bpt.make_embed_config(s.B, s.S, s.D, s.V, dtype=s.dtype)
        self.lcfg = bpt.make_ln_config(T, s.D, s.ln_eps, in_dtype=s.dtype)

        mats = [("Wte", (s.V, s.D))] + ([("Wpe", (s.S, s.D))] if s.pos_table else []) + [("Wout", (s.D, s.ldw))]
        dims = {"Wq": (s.D, s.D), "Wk": (s.D, s.D), "Wv": (s.D, s.D), "Wo": (s.D, s.D), "W1": (s.D, s.F),
                "W2": (s.F, s.D), "ln1_g": (s.D,), "ln1_b": (s.D,), "ln2_g": (s.D,), "ln2_b": (s.D,),
                "b1": (s.F,), "b2": (s.D,)}
        vecs = [("lnf_g", (s.D,)), ("lnf_b", (s.D,))]
        for l in range(s.L):
            mats += [(f"{l}.{k}", dims[k]) for k in LAYER_MATS]
            vecs += [(f"{l}.{k}", dims[k]) for k in LAYER_VECS if s.biases or k not in ("b1", "b2")]
        self.decay = _Flat(mats, device, lowp)
        self.nodecay = _Flat(vecs, device, None)     # vectors are read in fp32 by the kernels
        self.step_count = 0

        # activations, saved state, workspace
        self.X = [torch.empty((T, s.D), dtype=self.tdt, device=device) for _ in range(s.L + 1)]
        sb = bpt.saved_bytes(self.cfg)
        self.saved = [torch.empty(max(sb, 256), dtype=torch.uint8, device=device) for _ in range(s.L)]
        self.hf = torch.empty((T, s.D), dtype=self.tdt, device=device)
        self.mean = torch.empty(T, dtype=torch.float32, device=device)
        self.rstd = torch.empty(T, dtype=torch.float32, device=device)
        self.loss = torch.empty(1, dtype=torch.float32, device=device)
        self.lse = torch.empty(T, dtype=torch.float32, device=device)
        self.dh = torch.empty((T, s.D), dtype=self.tdt, device=device)
        self.dX = [torch.empty((T, s.D), dtype=self.tdt, device=device) for _ in range(2)]
        ws = max(bpt.workspace_bytes(self.cfg, False), bpt.workspace_bytes(self.cfg, True),
                 bpt.xent_workspace_bytes(self.xcfg, False), bpt.xent_workspace_bytes(self.xcfg, True),
                 bpt.ln_workspace_bytes(self.lcfg), 256)
        self.ws = torch.empty(ws, dtype=torch.uint8, device=device)
        if init:
            self.init_params(seed)

    # ------------------------------------------------------------ parameters
    def _group(self, name: str) -> _Flat:
        return self.decay if name in self.decay.index else self.nodecay

    def master(self, name: str) -> torch.Tensor:
        g = self._group(name)
        return g.view(g.p, name)

    def grad(self, name: str) -> torch.Tensor:
        g = self._group(name)
        return g.view(g.g, name)

    def weight(self, name: str) -> torch.Tensor:
        """The tensor the kernels read: the low-precision copy of a matrix on the bf16
        path, else the fp32 master."""
        g = self._group(name)
        return g.view(g.low, name) if g.low is not None else g.view(g.p, name)

    def names(self) -> List[str]:
        return list(self.decay.index) + list(self.nodecay.index)

    def sync_lowp(self) -> None:
        """Refresh the low-precision copies from the masters (after setting masters by hand)."""
        if self.decay.low is not None:
            self.decay.low.copy_(self.decay.p)

    def init_params(self, seed: int) -> None:
        """GPT-2 style initialisation: N(0, 0.02) matrices and tables, residual
        projections (Wo, W2) scaled by 1/sqrt(2L), gains 1, shifts and biases 0."""
        gen = torch.Generator(device="cpu").manual_seed(seed)
        s = self.shape
        for name in self.decay.index:
            m = self.master(name)
            std = 0.02 / math.sqrt(2 * s.L) if name.endswith((".Wo", ".W2")) else 0.02
            w = torch.randn(m.shape, generator=gen) * std
            if name == "Wout":
                w[:, s.V:] = 0.0
            m.copy_(w)
        for name in self.nodecay.index:
            self.master(name).fill_(1.0 if name.endswith("_g") else 0.0)
        self.sync_lowp()

    def layer_params(self, l: int) -> Dict[str, Optional[torch.Tensor]]:
        p = {k: self.weight(f"{l}.{k}") for k in LAYER_MATS}
        for k in LAYER_VECS:
            n = f"{l}.{k}"
            p[k] = self.master(n) if n in self.nodecay.index else None
        return p

    def layer_grads(self, l: int) -> Dict[str, Optional[torch.Tensor]]:
        out = {}
        for k in LAYER_MATS + LAYER_VECS:
            n = f"{l}.{k}"
            out["d" + k] = self.grad(n) if (n in self.decay.index or n in self.nodecay.index) else None
        return out

    # ------------------------------------------------------------ step
    def _layer_cfg(self, l: int) -> bpt.Config:
        """The layer config with layer l's dropout key for the current step (forward and
        backward of one step use the same key; every layer and step a different one)."""
        if self.shape.dropout > 0.0:
            self.cfg.dropout_seed = (self.shape.dropout_seed + (self.step_count << 20) + l) & (2 ** 64 - 1)
        return self.cfg

    def forward(self, tokens: torch.Tensor, targets: torch.Tensor, saving: bool = True) -> torch.Tensor:
        """Loss (a one-element fp32 tensor) of tokens [B*S] int32 with targets [B*S] int32."""
        s = self.shape
        bpt.embed_fwd(self.ecfg, tokens, self.weight("Wte"), self.weight("Wpe") if s.pos_table else None, self.X[0])
        for l in range(s.L):
            bpt.layer_fwd(self._layer_cfg(l), self.X[l], self.layer_params(l), self.X[l + 1], self.saved[l], self.ws)
        bpt.ln_fwd(self.lcfg, self.X[s.L], self.master("lnf_g"), self.master("lnf_b"), self.hf, self.mean, self.rstd)
        bpt.xent_fwd(self.xcfg, self.hf, self.weight("Wout"), targets, self.loss, self.lse, self.ws)
        return self.loss

    def backward(self, tokens: torch.Tensor, targets: torch.Tensor, dloss: float = 1.0) -> None:
        """Gradients of dloss * loss into the flat gradient buffers (overwritten)."""
        s = self.shape
        bpt.xent_bwd(self.xcfg, self.hf, self.weight("Wout"), targets, self.lse, dloss, self.dh, self.grad("Wout"),
                     self.ws)
        cur, nxt = self.dX
        bpt.ln_bwd(self.lcfg, self.X[s.L], self.master("lnf_g"), self.mean, self.rstd, self.dh, cur,
                   self.grad("lnf_g"), self.grad("lnf_b"), self.ws)
        for l in range(s.L - 1, -1, -1):
            bpt.layer_bwd(self._layer_cfg(l), self.X[l], self.layer_params(l), self.saved[l], cur, nxt, self.layer_grads(l),
                          self.ws)
            cur, nxt = nxt, cur
        bpt.embed_bwd(self.ecfg, tokens, cur, self.grad("Wte"), self.grad("Wpe") if s.pos_table else None)
        self.dX0 = cur

    def optimizer_step(self, lr: float, weight_decay: float = 0.1, beta1: float = 0.9, beta2: float = 0.95,
                       eps: float = 1e-8) -> None:
        self.step_count += 1
        for grp, wd in ((self.decay, weight_decay), (self.nodecay, 0.0)):
            bpt.adamw_step(grp.p, grp.g, grp.m, grp.v, self.step_count, lr, beta1, beta2, eps, wd, p_lowp=grp.low)

    def train_step(self, tokens: torch.Tensor, targets: torch.Tensor, lr: float, **opt) -> torch.Tensor:
        loss = self.forward(tokens, targets)
        self.backward(tokens, targets)
        self.optimizer_step(lr, **opt)
        return loss


def cosine_lr(step: int, max_lr: float = 2e-4, warmup: int = 0, total: int = 1, min_lr: float = 0.0) -> float:
    """Cosine learning-rate decay (Section 5's schedule, peak 2e-4), host-side."""
    if step < warmup:
        return max_lr * (step + 1) / warmup
    t = min(1.0, (step - warmup) / max(1, total - warmup))
    return min_lr + 0.5 * (max_lr - min_lr) * (1.0 + math.cos(math.pi * t))
