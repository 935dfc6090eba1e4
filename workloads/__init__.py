"""Seeded synthetic inputs for the fused attention forward+backward pass.

This module is shared by the HIP path's tests/bench and by the CPU oracle's
tests. It holds the workload table and the random-number recipe only: no step
of the attention arithmetic lives here. Rounding the generated float32 values
to bfloat16 is input quantisation (the values the GPU is handed), done with
integer round-to-nearest-even on the bit pattern.

The paper's own workloads are synthetic arrays of shape B x N x D with the
heads folded into B (Paper II, "Backward Pass and Fused Forward+Backward";
Paper I, "Validation against M_fwd", Table tab:paper1-dram). The table below
adds a head axis ([B, H, n, d], d fastest) and the sizes, value distributions
and masks of the five attention workloads this library is measured on.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Dict, Optional, Sequence

import numpy as np

__all__ = ["Workload", "WORKLOADS", "Inputs", "generate", "to_torch", "f32_to_bf16_bits",
           "bf16_bits_to_f32", "round_to_bf16", "causal_pairs", "alg_flops",
           "alg_bytes", "DecodeWorkload", "DECODE_WORKLOADS", "DecodeInputs", "generate_decode",
           "decode_to_torch", "decode_bytes"]


@dataclass(frozen=True)
class Workload:
    """One attention workload: shape, element type, mask and distributions.

    sigma_* are standard deviations (N(0, 4) has sigma 2; N(0, 0.1^2) has 0.1).
    """
    name: str
    B: int
    H: int
    n: int
    d: int
    dtype: str          # "f32" or "bf16"
    causal: bool
    sigma_qk: float
    sigma_v: float
    sigma_do: float
    seed: int

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def heads(self) -> int:
        return self.B * self.H

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


# The five measured workloads. Seeds are fixed per workload.
WORKLOADS: Dict[str, Workload] = {w.name: w for w in [
    Workload("h1_n128_d32_f32", 1, 1, 128, 32, "f32", False, 1.0, 1.0, 1.0, 1),
    Workload("b4h8_n1024_d64_f32", 4, 8, 1024, 64, "f32", False, 1.0, 1.0, 1.0, 2),
    Workload("b8h16_n4096_d64_bf16_causal", 8, 16, 4096, 64, "bf16", True, 1.0, 1.0, 0.1, 3),
    Workload("b2h32_n16384_d128_bf16_causal", 2, 32, 16384, 128, "bf16", True, 1.0, 1.0, 0.1, 4),
    Workload("b16h32_n2048_d128_bf16_peaked", 16, 32, 2048, 128, "bf16", False, 2.0, 1.0, 1.0, 5),
]}


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); return uint16 bits.

    Inputs are finite normal samples, so NaN/Inf handling is not needed.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to float32."""
    return (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 value, returned as float32."""
    return bf16_bits_to_f32(f32_to_bf16_bits(x))


@dataclass
class Inputs:
    """Q, K, V, dO of one workload as float32 [B, H, n, d] arrays.

    For bf16 workloads the float32 values are exactly the bfloat16 values
    handed to the GPU, and ``bits`` holds their uint16 patterns.
    """
    workload: Workload
    q: np.ndarray
    k: np.ndarray
    v: np.ndarray
    do: np.ndarray
    bits: Optional[Dict[str, np.ndarray]] = None

    def tensors(self):
        return {"q": self.q, "k": self.k, "v": self.v, "do": self.do}


def generate(w: Workload, *, n: Optional[int] = None, B: Optional[int] = None,
             H: Optional[int] = None, seed: Optional[int] = None) -> Inputs:
    """Draw Q, K, V, dO for workload ``w`` (optionally overriding sizes/seed).

    One PCG64 stream per tensor, spawned from SeedSequence(seed) in the order
    Q, K, V, dO; each tensor is standard_normal(float32) * sigma, then rounded
    to bfloat16 for bf16 workloads.
    """
    B = w.B if B is None else B
    H = w.H if H is None else H
    n = w.n if n is None else n
    seed = w.seed if seed is None else seed
    shape = (B, H, n, w.d)
    streams = np.random.SeedSequence(seed).spawn(4)
    sig = {"q": w.sigma_qk, "k": w.sigma_qk, "v": w.sigma_v, "do": w.sigma_do}
    out = {}
    bits = {} if w.dtype == "bf16" else None
    for name, ss in zip(("q", "k", "v", "do"), streams):
        g = np.random.Generator(np.random.PCG64(ss))
        x = g.standard_normal(shape, dtype=np.float32)
        if sig[name] != 1.0:
            x *= np.float32(sig[name])
        if bits is not None:
            b = f32_to_bf16_bits(x)
            bits[name] = b
            x = bf16_bits_to_f32(b)
        out[name] = x
    return Inputs(w, out["q"], out["k"], out["v"], out["do"], bits)


def to_torch(inp: Inputs, device="cuda") -> Dict[str, "object"]:
    """Copy the inputs to torch tensors on ``device`` in the workload's type
    (bfloat16 from the stored bit patterns, or float32)."""
    import torch
    out = {}
    for name in ("q", "k", "v", "do"):
        if inp.workload.dtype == "bf16":
            out[name] = torch.from_numpy(inp.bits[name].view(np.int16)).to(device).view(torch.bfloat16)
        else:
            out[name] = torch.from_numpy(getattr(inp, name)).to(device)
    return out


def causal_pairs(n: int, causal: bool) -> int:
    """Number of (query, key) pairs that take part: n^2, or n(n+1)/2 with the
    top-left-aligned causal mask (key j <= query i)."""
    return n * (n + 1) // 2 if causal else n * n


def alg_flops(B: int, H: int, n: int, d: int, causal: bool, fwd_only: bool = False) -> int:
    """Algorithmic flop count: each of the forward's two products (Q K^T, P V)
    and the backward's five (S recompute, dP, dV, dQ, dK) counted once, two
    flops per multiply-add: 4*d per pair forward, 14*d per pair fwd+bwd."""
    per_pair = 4 * d if fwd_only else 14 * d
    return per_pair * causal_pairs(n, causal) * B * H


def alg_bytes(B: int, H: int, n: int, d: int, elem_bytes: int, fwd_only: bool = False) -> int:
    """Minimum HBM bytes of one call: every input read once, every output
    written once. fwd+bwd reads Q, K, V, dO and writes O, dQ, dK, dV (8 n*d
    elements) plus L (n fp32); the forward alone reads Q, K, V and writes O and
    L. Internal row vectors (D) are not counted."""
    if fwd_only:
        return B * H * (4 * n * d * elem_bytes + 4 * n)
    return B * H * (8 * n * d * elem_bytes + 4 * n)


# ----------------------------------------------------------------- decode --
@dataclass(frozen=True)
class DecodeWorkload:
    """One decode step: B sequences, Hq query heads over Hkv cache heads
    (Hq / Hkv query heads per cache head), ``n`` tokens already cached per
    sequence (or, with ``ragged``, between n/2 and n), a cache of capacity
    n_cap rows, head dimension d. The new token's key and value are appended
    at row len_b before it attends."""
    name: str
    B: int
    Hq: int
    Hkv: int
    n: int
    n_cap: int
    d: int
    dtype: str
    ragged: bool
    sigma_qk: float
    seed: int

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


# Decode workloads: a GQA serving batch (8 query heads per cache head), a long
# single-sequence context, a ragged batch, and the paper's sizes (B = 2, one
# head, d = 64; the paper runs them in float32) at its largest cache length.
DECODE_WORKLOADS: Dict[str, DecodeWorkload] = {w.name: w for w in [
    DecodeWorkload("dec_b16_hq64_hkv8_n8192_d128_bf16", 16, 64, 8, 8192, 8193, 128, "bf16", False, 1.0, 11),
    DecodeWorkload("dec_b1_hq64_hkv8_n131072_d128_bf16", 1, 64, 8, 131072, 131073, 128, "bf16", False, 1.0, 12),
    DecodeWorkload("dec_b32_hq32_hkv8_n4096_d128_bf16_ragged", 32, 32, 8, 4096, 4097, 128, "bf16", True, 1.0, 13),
    DecodeWorkload("dec_b2_h1_n1048576_d64_bf16", 2, 1, 1, 1048576, 1048577, 64, "bf16", False, 1.0, 14),
]}


@dataclass
class DecodeInputs:
    """q [B, Hq, d]; caches [B, Hkv, n_cap, d] (rows past a sequence's length
    hold random values the step must ignore); k_new, v_new [B, Hkv, d]; lens
    [B] int32 (tokens cached before the step). float32 arrays hold exactly
    the values handed to the GPU; ``bits`` their bfloat16 patterns."""
    workload: DecodeWorkload
    q: np.ndarray
    k_cache: np.ndarray
    v_cache: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray
    lens: np.ndarray
    bits: Optional[Dict[str, np.ndarray]] = None


def generate_decode(w: DecodeWorkload, *, n: Optional[int] = None, B: Optional[int] = None,
                    seed: Optional[int] = None) -> DecodeInputs:
    """Draw one decode step's inputs: one PCG64 stream per array, spawned from
    SeedSequence(seed) in the order q, k_cache, v_cache, k_new, v_new, lens;
    standard normal (q and keys times sigma_qk), bfloat16-rounded for bf16."""
    B = w.B if B is None else B
    n = w.n if n is None else n
    n_cap = max(w.n_cap, n + 1)
    seed = w.seed if seed is None else seed
    shapes = {"q": (B, w.Hq, w.d), "k_cache": (B, w.Hkv, n_cap, w.d), "v_cache": (B, w.Hkv, n_cap, w.d),
              "k_new": (B, w.Hkv, w.d), "v_new": (B, w.Hkv, w.d)}
    sig = {"q": w.sigma_qk, "k_cache": w.sigma_qk, "k_new": w.sigma_qk, "v_cache": 1.0, "v_new": 1.0}
    streams = np.random.SeedSequence(seed).spawn(6)
    out, bits = {}, ({} if w.dtype == "bf16" else None)
    for (name, shape), ss in zip(shapes.items(), streams[:5]):
        x = np.random.Generator(np.random.PCG64(ss)).standard_normal(shape, dtype=np.float32)
        if sig[name] != 1.0:
            x *= np.float32(sig[name])
        if bits is not None:
            bb = f32_to_bf16_bits(x)
            bits[name] = bb
            x = bf16_bits_to_f32(bb)
        out[name] = x
    g = np.random.Generator(np.random.PCG64(streams[5]))
    lens = g.integers(max(n // 2, 0), n + 1, size=B).astype(np.int32) if w.ragged else \
        np.full(B, n, dtype=np.int32)
    return DecodeInputs(w, out["q"], out["k_cache"], out["v_cache"], out["k_new"], out["v_new"], lens, bits)


def decode_to_torch(inp: DecodeInputs, device="cuda") -> Dict[str, "object"]:
    import torch
    out = {}
    for name in ("q", "k_cache", "v_cache", "k_new", "v_new"):
        if inp.workload.dtype == "bf16":
            out[name] = torch.from_numpy(inp.bits[name].view(np.int16)).to(device).view(torch.bfloat16)
        else:
            out[name] = torch.from_numpy(getattr(inp, name)).to(device)
    out["lens"] = torch.from_numpy(inp.lens).to(device)
    return out


def decode_bytes(lens, Hq: int, Hkv: int, d: int, elem_bytes: int, append: bool = True) -> int:
    """Minimum HBM bytes of one decode step: every cached key and value row
    the step attends to read once (the appended row written once), q read and
    O written once, L written (float32)."""
    B = len(lens)
    rows = sum(int(x) for x in lens)
    kv = 2 * Hkv * d * elem_bytes * rows
    new = 2 * 2 * B * Hkv * d * elem_bytes if append else 0     # k_new/v_new read, cache row written
    return kv + new + 2 * B * Hq * d * elem_bytes + 4 * B * Hq
