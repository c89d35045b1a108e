"""Seeded synthetic inputs and the named Dyad workloads.

This module draws random tensors and names shapes; it holds none of the Dyad
arithmetic, so both the GPU path's tests and the CPU oracle can consume the
same bytes from it.

Recipe (stands in for the paper's BabyLM-pretrained OPT/Pythia feed-forward
activations, which are not used): numpy ``default_rng`` with one seed per
tensor, values drawn in float32 and rounded once to the compute dtype with
round-to-nearest-even (torch's CPU conversion).  X ~ N(0, 1), W1, W2 ~ N(0, 0.02),
bias ~ N(0, 0.02) (zero for the tiny fp32 case), dZ ~ N(0, 1), H_in ~ N(0, 1).
The GPU side uploads these exact bits; the oracle widens them to float64.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

SEEDS = {"X": 1001, "W1": 1002, "W2": 1003, "bias": 1004, "dZ": 1005, "H_in": 1006}
W_STD = 0.02

DTYPES = {"f32": torch.float32, "bf16": torch.bfloat16}


def _normal(seed: int, shape, std: float) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(std))


def draw(name: str, shape, std: float, dtype: str, seed_offset: int = 0) -> torch.Tensor:
    """One seeded tensor, drawn in fp32 and rounded (RNE) to ``dtype``, on the CPU."""
    a = _normal(SEEDS[name] + seed_offset, shape, std)
    return torch.from_numpy(a).to(DTYPES[dtype])


@dataclass
class LayerInputs:
    """CPU tensors in the compute dtype for one Dyad layer of shape n_in -> n_out."""
    n_in: int
    n_out: int
    n_dyad: int
    M: int
    dtype: str
    X: torch.Tensor
    W1: torch.Tensor
    W2: torch.Tensor
    bias: torch.Tensor | None
    dZ: torch.Tensor
    H_in: torch.Tensor

    def f64(self, name: str) -> np.ndarray | None:
        t = getattr(self, name)
        return None if t is None else t.to(torch.float64).numpy()


def layer_inputs(n_in: int, n_out: int, n_dyad: int, M: int, dtype: str = "bf16",
                 bias: str = "normal", seed_offset: int = 0) -> LayerInputs:
    """Inputs for one layer; ``bias`` is "normal", "zero" or "none"."""
    bo, bi = -(-n_out // n_dyad), -(-n_in // n_dyad)   # widths zero-padded up to n_dyad blocks
    X = draw("X", (M, n_in), 1.0, dtype, seed_offset)
    W1 = draw("W1", (n_dyad, bo, bi), W_STD, dtype, seed_offset)
    W2 = draw("W2", (n_dyad, bo, bi), W_STD, dtype, seed_offset)
    if bias == "normal":
        b = draw("bias", (n_out,), W_STD, dtype, seed_offset)
    elif bias == "zero":
        b = torch.zeros((n_out,), dtype=DTYPES[dtype])
    else:
        b = None
    dZ = draw("dZ", (M, n_out), 1.0, dtype, seed_offset)
    H_in = draw("H_in", (M, n_in), 1.0, dtype, seed_offset)
    return LayerInputs(n_in, n_out, n_dyad, M, dtype, X, W1, W2, b, dZ, H_in)


@dataclass
class Workload:
    """A named feed-forward shape: fc1 d->ffn (GELU after it), fc2 ffn->d."""
    name: str
    d: int
    ffn: int
    n_dyad: int
    M: int
    dtype: str = "bf16"
    variants: tuple = ("IT", "OT", "DT")
    note: str = ""
    layers: list = field(default_factory=list)

    def __post_init__(self):
        if not self.layers:
            self.layers = [("fc1", self.d, self.ffn), ("fc2", self.ffn, self.d)]

    def flops_per_pass(self, n_in: int, n_out: int) -> float:
        """Algorithmic FLOPs of one pass (fwd, dX or dW) of one layer: 4 M n_in n_out / n_dyad."""
        return 4.0 * self.M * n_in * n_out / self.n_dyad


TINY = Workload("tiny_it_f32", d=64, ffn=256, n_dyad=4, M=128, dtype="f32",
                variants=("IT", "OT", "DT"),
                note="n_in=64, n_out=256, n_dyad=4, M=128, fp32, bias 0",
                layers=[("layer", 64, 256)])
OPT125M = Workload("opt125m_ff", d=768, ffn=3072, n_dyad=4, M=16384,
                   note="OPT-125m FF: fc1 768->3072 (+GELU), fc2 3072->768, n_dyad=4, M=8x2048")
OPT350M = Workload("opt350m_ff", d=1024, ffn=4096, n_dyad=4, M=16384,
                   note="OPT-350m FF: fc1 1024->4096 (+GELU), fc2 4096->1024, n_dyad=4, M=8x2048")


def sweep(d: int, n_dyad: int) -> Workload:
    """Width/block sweep point: ffn = 4d, M = 16384."""
    return Workload(f"sweep_d{d}_D{n_dyad}", d=d, ffn=4 * d, n_dyad=n_dyad, M=16384,
                    note=f"sweep d={d}, ffn={4 * d}, n_dyad={n_dyad}")


SWEEP = [sweep(d, D) for d in (1024, 2048, 4096, 8192) for D in (2, 4, 8, 16)]


def wide(M: int) -> Workload:
    """Wide FF pair 8192 -> 32768 -> 8192, n_dyad=16, M tokens (16 and 256: decode-sized)."""
    return Workload(f"wide_M{M}", d=8192, ffn=32768, n_dyad=16, M=M,
                    note=f"wide FF 8192->32768->8192, n_dyad=16, M={M}")


WIDE = [wide(M) for M in (16, 256, 32768)]


# Widths that n_dyad does not divide (zero-padded blocks): OPT-125m's feed-forward
# at n_dyad 3, 5 and 6 (blocks of 256/1024, 154/615 and 128/512)
PADDED = [Workload(f"opt125m_ff_D{D}", d=768, ffn=3072, n_dyad=D, M=16384,
                   note=f"OPT-125m FF at n_dyad={D}" + ("" if 768 % D == 0 else " (zero-padded blocks)"))
          for D in (3, 5, 6)]
