"""The five synthetic workloads, shaped like the paper's 60M model.

Section 3 "Model and training": d_model 512 = 8 heads x d_head 64, 16 layers,
training length 1024, bf16 autocast, seed 42; Section 4.5 ("Length extrapolation") evaluates at 4x length
(T = 4096) with RoPE and the offsets unchanged.  The run matrix sweeps
W in {6, 8, 10, 12} (Section 3 "Run matrix").  Inputs are i.i.d. N(0,1)
(paper_2606_28560_amd.inputs); layers are independent calls with their own seeded
inputs, run one after another on one stream.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

from . import inputs, schedules


@dataclass(frozen=True)
class LayerCall:
    layer: int
    W: int
    base_name: str
    base: Tuple[int, ...]
    alpha: np.float32


@dataclass
class Workload:
    name: str
    case: int              # seed-stream id of this workload's inputs
    B: int
    H: int
    T: int
    D: int
    dtype: str             # "fp32" or "bf16"
    backward: bool
    calls: List[LayerCall] = field(default_factory=list)

    @property
    def queries_heads(self) -> int:
        return self.B * self.H * self.T


def _calls(Ws, bases, alphas):
    out = []
    for W in Ws:
        for bname, base in bases:
            for l, a in enumerate(alphas):
                out.append(LayerCall(l, W, bname, tuple(base), np.float32(a)))
    return out


def all_workloads():
    fib = ("fib15", schedules.FIB15)
    pow2 = ("pow2_11", schedules.POW2_11)
    learned = schedules.alpha_from_theta(inputs.thetas(16, case=5))
    return [
        Workload("single_layer_fp32_T128", 1, 1, 2, 128, 32, "fp32", True,
                 _calls([8], [fib], [1.0])),
        Workload("layer_60m_fixed_T1024", 2, 8, 8, 1024, 64, "bf16", True,
                 _calls([8], [fib], [1.0])),
        Workload("stagger16_T1024", 3, 16, 8, 1024, 64, "bf16", True,
                 _calls([6, 8, 10, 12], [fib], schedules.alpha_linear_stagger(16))),
        Workload("extrap_coprime16_T4096", 4, 4, 8, 4096, 64, "bf16", False,
                 _calls([8], [fib], schedules.alpha_coprime_stagger(16))),
        Workload("pow2_fib_learned16_T1024", 5, 32, 8, 1024, 64, "bf16", True,
                 _calls([10], [pow2, fib], learned)),
    ]


def workload(name_or_index):
    wl = all_workloads()
    if isinstance(name_or_index, int):
        return wl[name_or_index]
    for w in wl:
        if w.name == name_or_index:
            return w
    raise KeyError(name_or_index)


def layer_inputs(wl: Workload, call_index: int, names=("q", "k", "v", "dO")):
    """CPU torch tensors for one layer call of a workload."""
    return inputs.attention_inputs(wl.B, wl.H, wl.T, wl.D, wl.dtype, wl.case, call_index, names)
