"""Seeded synthetic workloads shaped like the paper's models.

This module only draws inputs: shapes, seeds and value distributions. It holds
none of the update, threshold or rounding arithmetic, and both the GPU path and
the CPU oracle consume what it returns.

Distributions (a stand-in for the missing trained models and datasets):
  A  = -exp(U[0, 2.5])                   per head (Mamba-2) or per (channel, n)
  dt = softplus(N(0, 1) - 4)             per (batch, head)
  B, C, x, D ~ N(0, 1)
  initial state h0 ~ N(0, 1) * sigma, sigma = 0.07 * exp(U[-1, 1]) per head,
  stored with torch's own round-to-nearest casts (fp16, bf16); E4M3 codes are
  cast from N(0, 112^2) clamped to +-448, with a per-group scale U[1e-4, 1e-3].
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    name: str
    family: str            # "mamba1" or "mamba2"
    batch: int
    nheads: int            # Mamba-1: d_inner
    headdim: int           # Mamba-1: 1
    dstate: int
    ngroups: int
    layers: int
    steps: int
    formats: tuple
    rules: tuple = ("rtn", "sr", "weyl")
    dither_block: int = 16
    scale_group: int = 0   # E4M3 entries per scale; 0 = one head
    int_group: int = 16    # INT8 / INT4 block: 16 (Mamba), the state dimension (hybrids)
    notes: str = ""
    extra: dict = field(default_factory=dict)

    @property
    def entries_per_layer(self) -> int:
        return self.batch * self.nheads * self.headdim * self.dstate

    @property
    def a_per_state(self) -> int:
        return 1 if self.family == "mamba1" else 0


# The five workloads of the measurement plan. Dither block: 16 for the pure
# Mamba shapes, the state dimension for the hybrid shapes (Section 2, "Low-
# precision storage").
WORKLOADS = {
    "m1_small": Workload("m1_small", "mamba1", 1, 1536, 1, 16, 1, 1, 64, ("fp16",),
                         notes="Mamba-1 state update, batch 1, d_inner 1536, d_state 16"),
    "m2_ssd_b8": Workload("m2_ssd_b8", "mamba2", 8, 80, 64, 128, 1, 1, 256, ("bf16",),
                          notes="Mamba-2 SSD decode, batch 8, 80 heads of 64x128"),
    "m2_b64_fp8": Workload("m2_b64_fp8", "mamba2", 64, 128, 64, 128, 8, 1, 512, ("e4m3",),
                           dither_block=128,
                           notes="Mamba-2 decode, batch 64, 128 heads, 8 groups, E4M3 per-head scale"),
    "m1_long": Workload("m1_long", "mamba1", 16, 5120, 1, 16, 1, 64, 4096, ("fp16",),
                        notes="long-horizon Mamba-1 shape, batch 16, 64 layers, d_inner 5120"),
    "hybrid_m2_stack": Workload("hybrid_m2_stack", "mamba2", 256, 128, 64, 128, 8, 48, 1024,
                                ("bf16", "e4m3"), rules=("weyl", "sr", "rtn"), dither_block=128,
                                int_group=128,
                                notes="hybrid-style Mamba-2 stack, batch 256, 48 SSM layers, "
                                      "128 heads of 64x128, 8 groups"),
}


def _gen(seed: int, device="cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed) & 0x7FFFFFFFFFFFFFFF)
    return g


def scale_group_of(w: "Workload", fmt: str) -> int:
    """Entries per scale of a scaled format on a workload (0 = one head)."""
    if fmt in ("int8", "int4"):
        return w.int_group
    return w.scale_group if fmt == "e4m3" else 0


def splitmix64(*words: int) -> int:
    """Combine integers into one 63-bit seed (SplitMix64 finalizer, Steele et al.)."""
    z = 0x243F6A8885A308D3
    for w in words:
        z = (z + (int(w) & 0xFFFFFFFFFFFFFFFF) + 0x9E3779B97F4A7C15) & 0xFFFFFFFFFFFFFFFF
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & 0xFFFFFFFFFFFFFFFF
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & 0xFFFFFFFFFFFFFFFF
        z ^= z >> 31
    return z & 0x7FFFFFFFFFFFFFFF


def layer_params(family: str, nheads: int, dstate: int, seed: int, device="cpu"):
    """A and D of one layer (fixed across steps)."""
    g = _gen(splitmix64(seed, 1), device)
    shape = (nheads, dstate) if family == "mamba1" else (nheads,)
    A = -torch.exp(torch.rand(shape, generator=g, device=device, dtype=torch.float32) * 2.5)
    D = torch.randn((nheads,), generator=g, device=device, dtype=torch.float32)
    return A.contiguous(), D.contiguous()


def layer_params_trained_memory(family: str, nheads: int, dstate: int, seed: int, device="cpu"):
    """A and D with a trained model's spread of memories: with E[dt] = 0.029, 80 % of
    the decay rates give tau = 1 / (1 - exp(A E[dt])) below about 35 steps
    (A = -exp(U[0, 2.5])) and 20 % give tau from about 100 to 1900 steps
    (A = -exp(U[-4, -1.1])), close to the 13-23 % with tau >= 100 and up to 5 %
    with tau >= 1000 measured on trained models (Section 2)."""
    g = _gen(splitmix64(seed, 4), device)
    shape = (nheads, dstate) if family == "mamba1" else (nheads,)
    short = torch.rand(shape, generator=g, device=device, dtype=torch.float32) * 2.5
    long_ = torch.rand(shape, generator=g, device=device, dtype=torch.float32) * 2.9 - 4.0
    pick = torch.rand(shape, generator=g, device=device, dtype=torch.float32) < 0.2
    A = -torch.exp(torch.where(pick, long_, short))
    D = torch.randn((nheads,), generator=g, device=device, dtype=torch.float32)
    return A.contiguous(), D.contiguous()


def step_inputs(batch: int, nheads: int, headdim: int, dstate: int, ngroups: int, seed: int,
                device="cpu"):
    """x, dt, B, C of one (layer, step)."""
    g = _gen(splitmix64(seed, 2), device)
    x = torch.randn((batch, nheads, headdim), generator=g, device=device, dtype=torch.float32)
    dt_raw = torch.randn((batch, nheads), generator=g, device=device, dtype=torch.float32) - 4.0
    dt = torch.nn.functional.softplus(dt_raw)
    B = torch.randn((batch, ngroups, dstate), generator=g, device=device, dtype=torch.float32)
    C = torch.randn((batch, ngroups, dstate), generator=g, device=device, dtype=torch.float32)
    return x.contiguous(), dt.contiguous(), B.contiguous(), C.contiguous()


_TORCH_DTYPE = {"fp16": torch.float16, "bf16": torch.bfloat16, "fp32": torch.float32}
CODE_TORCH_DTYPE = {"fp16": torch.int16, "bf16": torch.int16, "e4m3": torch.uint8,
                    "fp32": torch.int32, "int8": torch.uint8, "int4": torch.uint8}
INT_QMAX = {"int8": 127, "int4": 7}


def initial_state(fmt: str, batch: int, nheads: int, headdim: int, dstate: int, seed: int,
                  group: int = 0, device="cpu"):
    """Stored codes [batch, nheads, headdim, dstate] (and E4M3 / INT group scales).

    Codes are returned as integer tensors (int16 / uint8 / int32 bit patterns);
    INT4 packs two entries per byte, [batch, nheads, headdim, dstate / 2].
    """
    g = _gen(splitmix64(seed, 3), device)
    shape = (batch, nheads, headdim, dstate)
    if fmt in INT_QMAX:
        # a Gaussian state at the scale's resolution: integers k ~ N(0, (qmax/3)^2)
        # clamped to +-qmax, scales U[1e-3, 1e-2] per group
        qmax = INT_QMAX[fmt]
        head = headdim * dstate
        group = head if group == 0 else group
        k = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * (qmax / 3.0)
        k = k.round_().clamp_(-qmax, qmax).to(torch.int32)
        u = (k & (0xFF if fmt == "int8" else 0xF)).to(torch.uint8)
        if fmt == "int4":
            u = (u[..., 0::2] | (u[..., 1::2] << 4)).to(torch.uint8)
        n_groups = batch * nheads * head // group
        scale = (torch.rand((n_groups,), generator=g, device=device, dtype=torch.float32)
                 * 9e-3 + 1e-3)
        return u.contiguous(), scale.contiguous()
    if fmt == "e4m3":
        head = headdim * dstate
        group = head if group == 0 else group
        q = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * 112.0
        q = q.clamp_(-448.0, 448.0)
        codes = q.to(torch.float8_e4m3fn).view(torch.uint8).contiguous()
        n_groups = batch * nheads * head // group
        scale = (torch.rand((n_groups,), generator=g, device=device, dtype=torch.float32)
                 * 9e-4 + 1e-4)
        return codes, scale.contiguous()
    sigma = 0.07 * torch.exp(torch.rand((1, nheads, 1, 1), generator=g, device=device,
                                        dtype=torch.float32) * 2.0 - 1.0)
    h0 = torch.randn(shape, generator=g, device=device, dtype=torch.float32) * sigma
    codes = h0.to(_TORCH_DTYPE[fmt]).view(CODE_TORCH_DTYPE[fmt]).contiguous()
    return codes, None


def to_numpy_codes(fmt: str, codes: torch.Tensor) -> np.ndarray:
    """Host copy of codes with the oracle's unsigned dtypes."""
    a = codes.detach().cpu().numpy()
    if fmt in ("fp16", "bf16"):
        return a.view(np.uint16)
    if fmt == "fp32":
        return a.view(np.uint32)
    return a.view(np.uint8)
