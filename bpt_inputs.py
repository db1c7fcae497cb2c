"""Seeded synthetic inputs for one Blockwise Parallel Transformer layer.

This module holds the workload shapes and the random draws only. It contains
none of the layer's arithmetic, so both the CPU oracle (``oracle/``) and the
HIP path (``paper_2305_19370_amd``) can take their inputs from it without
sharing any computation.

Draw recipe (one CPU ``torch.Generator`` per call, seeded; fp32 standard-normal
draws in this fixed order, each scaled by its std and then rounded once to the
workload's storage dtype with round-to-nearest-even):

    X, Wq, Wk, Wv, Wo, W1, W2, dY            (always)
    ln1_g, ln1_b, ln2_g, ln2_b               (only when ``affine=True``)
    b1, b2                                   (only when ``biases=True``)

``init="small"``: X and every weight ~ N(0, 0.02^2) (the fp32 parity workload).
``init="unit"``:  X ~ N(0, 1); every weight, W2 included, ~ N(0, 1/D).
dY ~ N(0, 1) in both. LayerNorm gamma = 1 and beta = 0 unless ``affine=True``
(then gamma ~ 1 + N(0, 0.1^2), beta ~ N(0, 0.1^2)); FFN biases are absent
unless ``biases=True`` (then ~ N(0, 0.1^2)).

The long-context workloads stand in for the paper's training data (web text
for the GPT-shaped layers, offline RL trajectories for the RL-shaped one):
only the tensor shapes matter for cost, so the values are synthetic.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int
    S: int
    D: int
    H: int
    F: int
    causal: bool
    Bq: int
    Bkv: int
    dtype: str          # "f32" or "bf16": storage/compute type of X, weights, dY
    init: str           # "small" or "unit"
    note: str = ""

    @property
    def dh(self) -> int:
        return self.D // self.H

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# Shapes of the paper's model family (GPT-style layers; d_model, heads and
# head width as in its model-size table; the RL shape follows its trajectory
# experiment: 32 trajectories x 1000 steps x 3 tokens).
WORKLOADS: Dict[str, Workload] = {
    w.name: w
    for w in [
        Workload("fp32_s512_d256", 1, 512, 256, 4, 1024, True, 128, 128, "f32", "small",
                 "single layer, fp32 parity workload"),
        Workload("bf16_1b_s4096", 2, 4096, 2048, 16, 8192, True, 512, 512, "bf16", "unit",
                 "GPT 1B-shaped layer"),
        Workload("bf16_7b_s32768", 1, 32768, 4096, 32, 16384, True, 1024, 1024, "bf16", "unit",
                 "GPT 7B-shaped layer, long context"),
        Workload("bf16_13b_s65536", 1, 65536, 5120, 40, 20480, True, 2048, 2048, "bf16", "unit",
                 "GPT 13B-shaped layer, long context (S swept 8K..64K)"),
        Workload("bf16_rl_s96000", 4, 96000, 1024, 8, 4096, True, 1024, 1024, "bf16", "unit",
                 "RL trajectories: 32 x 1000 x (return, state, action)"),
        Workload("bf16_dh64_nc_s32768", 1, 32768, 2048, 32, 8192, False, 1024, 1024, "bf16", "unit",
                 "1B-width layer with heads of 64, without the causal mask, long context (parity case)"),
    ]
}

# The 13B-shaped layer's sequence-length sweep (linear memory in S): same shape and
# blocks at shorter sequences.
SWEEP_S = (8192, 16384, 32768, 65536)


def sweep_workload(S: int) -> Workload:
    base = WORKLOADS["bf16_13b_s65536"]
    return base.with_(S=S, name=f"bf16_13b_s{S}", note=f"GPT 13B-shaped layer at S={S} (sweep)")


def workload(name: str) -> Workload:
    """A named workload: one of WORKLOADS, or bf16_13b_s<S> for a length of the sweep."""
    if name in WORKLOADS:
        return WORKLOADS[name]
    if name.startswith("bf16_13b_s") and name[len("bf16_13b_s"):].isdigit():
        return sweep_workload(int(name[len("bf16_13b_s"):]))
    raise KeyError(name)


TENSOR_ORDER = ("X", "Wq", "Wk", "Wv", "Wo", "W1", "W2", "dY")


def torch_dtype(dtype: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[dtype]


def make_inputs(w: Workload, seed: int = 0, affine: bool = False, biases: bool = False,
                dY: bool = True) -> Dict[str, Optional[torch.Tensor]]:
    """Return CPU tensors in ``w.dtype`` (vectors: fp32) drawn per the recipe above."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    B, S, D, F = w.B, w.S, w.D, w.F
    if w.init == "small":
        sx, sw = 0.02, 0.02
    elif w.init == "unit":
        sx, sw = 1.0, D ** -0.5
    else:
        raise ValueError(f"unknown init {w.init!r}")
    shapes = {
        "X": ((B, S, D), sx), "Wq": ((D, D), sw), "Wk": ((D, D), sw), "Wv": ((D, D), sw),
        "Wo": ((D, D), sw), "W1": ((D, F), sw), "W2": ((F, D), sw), "dY": ((B, S, D), 1.0),
    }
    dt = torch_dtype(w.dtype)
    out: Dict[str, Optional[torch.Tensor]] = {}
    for name in TENSOR_ORDER:
        shape, std = shapes[name]
        if name == "dY" and not dY:
            out[name] = None
            continue
        t = torch.randn(shape, generator=g, dtype=torch.float32)
        if std != 1.0:
            t.mul_(std)
        out[name] = t.to(dt)
    for name in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
        out[name] = None
    if affine:
        for name in ("ln1_g", "ln1_b", "ln2_g", "ln2_b"):
            t = torch.randn((D,), generator=g, dtype=torch.float32) * 0.1
            out[name] = t + 1.0 if name.endswith("_g") else t
    out["b1"] = None
    out["b2"] = None
    if biases:
        out["b1"] = torch.randn((F,), generator=g, dtype=torch.float32) * 0.1
        out["b2"] = torch.randn((D,), generator=g, dtype=torch.float32) * 0.1
    return out


def small_workload(dtype: str = "f32", B: int = 1, S: int = 250, D: int = 256, H: int = 2,
                   F: int = 512, causal: bool = True, Bq: int = 128, Bkv: int = 128,
                   init: Optional[str] = None) -> Workload:
    """A reduced-shape workload for parity tests (ragged S by default)."""
    return Workload(f"small_{dtype}_B{B}_S{S}_D{D}_H{H}_F{F}_{'c' if causal else 'nc'}",
                    B, S, D, H, F, causal, Bq, Bkv, dtype,
                    init or ("small" if dtype == "f32" else "unit"))


# ---------------------------------------------------------------- LM-head cross-entropy inputs
def make_xent_inputs(T: int, D: int, V: int, ldw: int, dtype: str = "bf16", seed: int = 0,
                     logit_std: float = 2.0) -> Dict[str, torch.Tensor]:
    """Inputs of the LM-head cross-entropy, CPU tensors: h [T, D] ~ N(0, 1) (a final
    LayerNorm's output), W [D, ldw] ~ N(0, logit_std^2 / D) in its first V columns and
    zero in the padding columns (so logits have std ~logit_std), targets [T] int32
    uniform over [0, V). One CPU generator, draws in the order h, W, targets; h and W
    rounded once to the storage dtype."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    dt = torch_dtype(dtype)
    h = torch.randn((T, D), generator=g, dtype=torch.float32).to(dt)
    W = torch.zeros((D, ldw), dtype=torch.float32)
    W[:, :V] = torch.randn((D, V), generator=g, dtype=torch.float32) * (logit_std / D ** 0.5)
    targets = torch.randint(0, V, (T,), generator=g, dtype=torch.int32)
    return {"h": h, "W": W.to(dt), "targets": targets}


def make_gpt_inputs(L: int, B: int, S: int, D: int, F: int, V: int, ldw: int, dtype: str = "f32", seed: int = 0,
                    pos_table: bool = True, biases: bool = True) -> Dict[str, torch.Tensor]:
    """Parameters, tokens and targets of an L-layer GPT, CPU tensors keyed by parameter
    name ("Wte", "Wpe", "Wout", "lnf_g", "lnf_b", "<l>.<name>" per layer, "tokens",
    "targets"). One CPU generator, draws in the order Wte ~ N(0, 1) [V, D],
    Wpe ~ N(0, 0.5^2) [S, D], Wout ~ N(0, 4/D) [D, V] (zero padding columns up to ldw),
    then per layer Wq, Wk, Wv, Wo, W1, W2 ~ N(0, 1/D_in), ln1_g, ln2_g ~ 1 + N(0, 0.1^2),
    ln1_b, ln2_b, b1, b2 ~ N(0, 0.1^2), then lnf_g ~ 1 + N(0, 0.1^2), lnf_b ~ N(0, 0.1^2),
    tokens and targets uniform over [0, V) as int32 [B*S]. Matrices and tables are
    rounded once to the dtype; vectors stay fp32."""
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    dt = torch_dtype(dtype)
    rn = lambda *s: torch.randn(s, generator=g, dtype=torch.float32)
    out: Dict[str, torch.Tensor] = {"Wte": rn(V, D).to(dt)}
    if pos_table:
        out["Wpe"] = (rn(S, D) * 0.5).to(dt)
    Wout = torch.zeros((D, ldw), dtype=torch.float32)
    Wout[:, :V] = rn(D, V) * (2.0 / D ** 0.5)
    out["Wout"] = Wout.to(dt)
    for l in range(L):
        for name, (r, c) in (("Wq", (D, D)), ("Wk", (D, D)), ("Wv", (D, D)), ("Wo", (D, D)), ("W1", (D, F)),
                             ("W2", (F, D))):
            out[f"{l}.{name}"] = (rn(r, c) * r ** -0.5).to(dt)
        for name, n in (("ln1_g", D), ("ln1_b", D), ("ln2_g", D), ("ln2_b", D), ("b1", F), ("b2", D)):
            if name in ("b1", "b2") and not biases:
                continue
            t = rn(n) * 0.1
            out[f"{l}.{name}"] = t + 1.0 if name.endswith("_g") else t
    out["lnf_g"] = rn(D) * 0.1 + 1.0
    out["lnf_b"] = rn(D) * 0.1
    out["tokens"] = torch.randint(0, V, (B * S,), generator=g, dtype=torch.int32)
    out["targets"] = torch.randint(0, V, (B * S,), generator=g, dtype=torch.int32)
    return out
