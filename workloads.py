"""Seeded synthetic inputs for the FP8 linear-layer workloads.

This module only draws random numbers and lays them out.  It holds none of
the layer's arithmetic (no FP8 encoding, no scaling, no GEMM), so both the
CPU oracle and the HIP path can be fed from it without sharing any of the
method.  Every tensor is drawn from its own stream,

    numpy.random.default_rng(SeedSequence([seed, cfg, unit, role, mb, step]))

as float32 values, and then, where a workload says bf16, rounded to bfloat16
with round-to-nearest-even on the float32 bit pattern.  bf16 tensors are
carried as uint16 bit patterns so that nothing downstream re-rounds them.

Distributions (standard deviation, not variance, after the N(mean, sigma)
notation the workloads use):
  * activations  X  ~ N(0, 1)
  * weights      W  ~ N(0, 0.02)
  * grads        dY ~ N(0, 0.01)
  * outlier activations: N(0, 1) with round(0.001 * K) input channels (columns
    of X, chosen by the same stream) multiplied by 300
  * log-normal gradients: sign * exp(sigma * z), z ~ N(0, 1), fair random sign
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

ROLE_X, ROLE_W, ROLE_DY = 0, 1, 2


def rng_for(seed: int, cfg: int, unit: int, role: int, mb: int = 0, step: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg, unit, role, mb, step]))


def _bf16_chunk(u: np.ndarray, out: np.ndarray) -> None:
    # u: uint32 bits.  (u + 0x7FFF + lsb) >> 16 cannot wrap in 32 bits for a
    # non-NaN pattern (the largest, -inf = 0xFF800000, stays far below 2^32);
    # NaN patterns are replaced afterwards.
    r = (u >> np.uint32(16)) & np.uint32(1)
    r += u
    r += np.uint32(0x7FFF)
    r >>= np.uint32(16)
    nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    if nan.any():
        r[nan] = (u[nan] >> np.uint32(16)) | np.uint32(0x40)
    out[...] = r.astype(np.uint16)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (RNE on the bit pattern); returns uint16 bits.

    NaN inputs keep a quiet-NaN pattern; infinities pass through.  Large
    tensors are converted in chunks on a thread pool (NumPy releases the GIL),
    which bounds the temporaries to a few chunks."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.reshape(-1).view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    chunk = 1 << 22
    if u.size <= chunk:
        _bf16_chunk(u, out)
    else:
        from concurrent.futures import ThreadPoolExecutor
        import os
        n = max(1, min(16, len(os.sched_getaffinity(0))))
        with ThreadPoolExecutor(max_workers=n) as ex:
            list(ex.map(lambda o: _bf16_chunk(u[o:o + chunk], out[o:o + chunk]), range(0, u.size, chunk)))
    return out.reshape(x.shape)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Tensor:
    """A host tensor as the layer sees it: float32 data, or bf16 bits."""
    data: np.ndarray          # float32 [rows, cols] or uint16 [rows, cols]
    dtype: str                # "f32" or "bf16"

    @property
    def shape(self) -> Tuple[int, int]:
        return tuple(self.data.shape)

    def as_f32(self) -> np.ndarray:
        return self.data if self.dtype == "f32" else bf16_bits_to_f32(self.data)


def normal(rng: np.random.Generator, shape, sigma: float, dtype: str) -> Tensor:
    x = (rng.standard_normal(size=shape, dtype=np.float32) * np.float32(sigma)).astype(np.float32)
    return Tensor(f32_to_bf16_bits(x), "bf16") if dtype == "bf16" else Tensor(x, "f32")


def outlier_activations(rng: np.random.Generator, rows: int, cols: int, frac: float, mult: float,
                        dtype: str) -> Tensor:
    x = rng.standard_normal(size=(rows, cols), dtype=np.float32)
    n_out = int(round(frac * cols))
    ch = rng.choice(cols, size=n_out, replace=False) if n_out else np.zeros(0, dtype=np.int64)
    x[:, ch] *= np.float32(mult)
    return Tensor(f32_to_bf16_bits(x), "bf16") if dtype == "bf16" else Tensor(x, "f32")


def lognormal_signed(rng: np.random.Generator, shape, sigma: float, dtype: str) -> Tensor:
    z = rng.standard_normal(size=shape, dtype=np.float32)
    s = np.where(rng.random(size=shape, dtype=np.float32) < 0.5, np.float32(-1), np.float32(1))
    x = (s * np.exp(np.float32(sigma) * z)).astype(np.float32)
    return Tensor(f32_to_bf16_bits(x), "bf16") if dtype == "bf16" else Tensor(x, "f32")


# --------------------------------------------------------------------------------------------
# Workload shapes.  A linear is (name, K in-features, N out-features); W is [N, K].
# --------------------------------------------------------------------------------------------

@dataclasses.dataclass(frozen=True)
class Linear:
    name: str
    k_in: int
    n_out: int


@dataclasses.dataclass(frozen=True)
class Workload:
    key: str
    cfg: int
    linears: Tuple[Linear, ...]
    tokens: int               # tokens per microbatch
    microbatches: int
    history: int
    margin: int
    in_dtype: str             # dtype of X, dY and the master W
    steps: int = 1
    description: str = ""

    def flat_grad_elems(self) -> int:
        return sum(l.n_out * l.k_in for l in self.linears)

    def grad_offsets(self) -> List[int]:
        offs, o = [], 0
        for l in self.linears:
            offs.append(o)
            o += l.n_out * l.k_in
        return offs

    def gemm_flops_per_pass(self) -> int:
        """FLOPs of fwd + dI + dW (2*M*N*K each) for one microbatch through every linear."""
        return sum(3 * 2 * self.tokens * l.n_out * l.k_in for l in self.linears)


LLAMA3_8B = (Linear("qkv", 4096, 6144), Linear("o_proj", 4096, 4096),
             Linear("gate_up", 4096, 2 * 14336), Linear("down", 14336, 4096))
LLAMA3_70B = (Linear("qkv", 8192, 10240), Linear("o_proj", 8192, 8192),
              Linear("gate_up", 8192, 2 * 28672), Linear("down", 28672, 8192))

WORKLOADS: Dict[str, Workload] = {
    "single_linear_128x256x256": Workload(
        "single_linear_128x256x256", 0, (Linear("fc", 256, 256),), tokens=128, microbatches=2,
        history=4, margin=0, in_dtype="f32",
        description="one FP8 linear, 2 microbatches of 128 tokens, K=N=256, fp32 inputs"),
    "llama3_8b_stage_4096tok": Workload(
        "llama3_8b_stage_4096tok", 1, LLAMA3_8B, tokens=4096, microbatches=1, history=1024, margin=0,
        in_dtype="bf16",
        description="Llama-3-8B-shaped stage layer (QKV, O, gate+up, down), 4096 tokens, bf16"),
    "llama3_8b_zb_8x2048": Workload(
        "llama3_8b_zb_8x2048", 2, LLAMA3_8B, tokens=2048, microbatches=8, history=16, margin=0,
        in_dtype="bf16", steps=2,
        description="zero-bubble-style schedule, 8 microbatches of 2048 tokens, 2 optimizer steps"),
    "outlier_8192cube": Workload(
        "outlier_8192cube", 3, (Linear("fc", 8192, 8192),), tokens=8192, microbatches=1, history=1024,
        margin=1, in_dtype="f32", steps=3,
        description="outlier stress 8192^3, 0.1% channels x300, log-normal(2) grads, margin 1"),
    "llama3_70b_stage_8192tok": Workload(
        "llama3_70b_stage_8192tok", 4, LLAMA3_70B, tokens=8192, microbatches=1, history=1024, margin=0,
        in_dtype="bf16",
        description="Llama-3-70B-shaped stage layer, 8192 tokens, bf16"),
}


def layer_inputs(w: Workload, unit: int, seed: int = 0, mb: int = 0, step: int = 0,
                 tokens: int | None = None, outliers: bool | None = None) -> Dict[str, Tensor]:
    """X [tokens, K], dY [tokens, N] for one (linear, microbatch, step)."""
    lin = w.linears[unit]
    t = w.tokens if tokens is None else tokens
    use_outliers = (w.cfg == 3) if outliers is None else outliers
    rx = rng_for(seed, w.cfg, unit, ROLE_X, mb, step)
    rd = rng_for(seed, w.cfg, unit, ROLE_DY, mb, step)
    if use_outliers:
        x = outlier_activations(rx, t, lin.k_in, 0.001, 300.0, w.in_dtype)
        dy = lognormal_signed(rd, (t, lin.n_out), 2.0, w.in_dtype)
    else:
        x = normal(rx, (t, lin.k_in), 1.0, w.in_dtype)
        dy = normal(rd, (t, lin.n_out), 0.01, w.in_dtype)
    return {"x": x, "dy": dy}


def layer_weight(w: Workload, unit: int, seed: int = 0) -> Tensor:
    lin = w.linears[unit]
    return normal(rng_for(seed, w.cfg, unit, ROLE_W), (lin.n_out, lin.k_in), 0.02, w.in_dtype)
