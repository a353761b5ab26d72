"""Seeded synthetic inputs for the exact non-causal attention path.

This module is shared by the HIP path's tests and benchmark and by the fp64
oracle's tests. It holds no attention arithmetic: it only draws i.i.d. normal
tensors, encodes them as bfloat16 bit patterns, and picks sampled rows.

Workloads (Sec. II-A, II-E, V-E and VI-A of the paper): one GPU's share of a
DeepSpeed-Ulysses head-sharded attention, i.e. the full patch-token sequence N
for H local heads. The token counts are patch grids: 32x32, 128x128, 256x256,
368x512 (= 92 channels x 2,048 patches, the paper's 188K Multi-Ch-ViT run) and
1024x1024 (the paper's 1M-token runs). Head dims 64 (ViT-Base/Large) and 128
(ViT-5B) come from Table I.

The ERA5 activations the paper trains on are not available; dense attention's
run time does not depend on the values, so i.i.d. normal data stands in for
them. The 16,384-token ViT-block workload (id 2) scales head 0's Q and K by 8 so that its softmax rows are close
to one-hot (logit standard deviation about 64), which stresses the running
max and the bf16 rounding of P.

Recipe: numpy Generator(PCG64(seed)); draw Q, K, V, dO in that order, each
standard_normal((B,H,N,d), float32); multiply by sigma (and by 8 for the id-2 workload's
head 0 in Q and K; both multipliers are powers of two, so exact); round to
bfloat16 with round-to-nearest-even.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    B: int
    H: int
    N: int
    d: int
    backward: bool
    sigma: float
    seed: int
    stress_head0_qk: float  # multiplier on head 0's Q and K (1.0 = none)
    check: str  # "full" or "sampled"
    grid: tuple

    @property
    def scale(self) -> float:
        """Softmax scale 1/sqrt(d), rounded to fp32 (the value both sides use)."""
        return float(np.float32(1.0 / math.sqrt(self.d)))

    @property
    def shape(self):
        return (self.B, self.H, self.N, self.d)

    def counted_flops(self) -> dict:
        """FlashAttention flop convention: fwd 4*B*H*N^2*d, bwd 2.5x fwd."""
        fwd = 4.0 * self.B * self.H * self.N * self.N * self.d
        bwd = 10.0 * self.B * self.H * self.N * self.N * self.d if self.backward else 0.0
        return {"fwd": fwd, "bwd": bwd, "total": fwd + bwd}


WORKLOADS = {
    1: Workload(1, "single_head_fwd_N1024_d64", 1, 1, 1024, 64, False, 1.0, 1001, 1.0, "full", (32, 32)),
    2: Workload(2, "vit_block_fwdbwd_B2_H16_N16384_d64", 2, 16, 16384, 64, True, 1.0, 1002, 8.0, "full",
                (128, 128)),
    3: Workload(3, "ulysses_shard_fwdbwd_H4_N65536_d128", 1, 4, 65536, 128, True, 1.0, 1003, 1.0, "sampled",
                (256, 256)),
    4: Workload(4, "paper_scale_fwdbwd_H2_N188416_d128", 1, 2, 188416, 128, True, 1.0, 1004, 1.0, "sampled",
                (368, 512)),
    5: Workload(5, "one_million_token_fwd_N1048576_d64", 1, 1, 1048576, 64, False, 0.5, 1005, 1.0, "sampled",
                (1024, 1024)),
}

N_SAMPLED_ROWS = 256


def float32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns as uint16. Inputs must be finite."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    bias = ((u >> np.uint64(16)) & np.uint64(1)) + np.uint64(0x7FFF)
    return ((u + bias) >> np.uint64(16)).astype(np.uint16)


def bf16_bits_to_float32(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns to fp32 (used to build test
    inputs with prescribed structure, e.g. repeated keys)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def random_bf16(rng: np.random.Generator, shape, sigma: float = 1.0) -> np.ndarray:
    return float32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(sigma))


def make_inputs(w: Workload, with_dout: bool | None = None) -> dict:
    """Seeded bf16 bit arrays q, k, v (and dout when the workload has a
    backward pass), each uint16 of shape (B, H, N, d)."""
    if with_dout is None:
        with_dout = w.backward
    rng = np.random.Generator(np.random.PCG64(w.seed))
    names = ["q", "k", "v"] + (["dout"] if with_dout else [])
    out = {}
    for name in names:
        x = rng.standard_normal(w.shape, dtype=np.float32)
        if w.sigma != 1.0:
            x *= np.float32(w.sigma)
        if name in ("q", "k") and w.stress_head0_qk != 1.0:
            x[:, 0] *= np.float32(w.stress_head0_qk)
        out[name] = float32_to_bf16_bits(x)
        del x
    return out


def make_small_inputs(B, H, N, d, seed, sigma=1.0, with_dout=True) -> dict:
    """Seeded bf16 inputs of an arbitrary (B, H, N, d) shape for small parity
    cases (ragged tails, tiny N, odd head counts)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    names = ["q", "k", "v"] + (["dout"] if with_dout else [])
    return {n: random_bf16(rng, (B, H, N, d), sigma) for n in names}


def sampled_query_rows(w: Workload, count: int = N_SAMPLED_ROWS) -> np.ndarray:
    """Distinct flat (b, h, i) indices of sampled query rows, sorted; returns
    an int64 array of shape (count, 3)."""
    rng = np.random.Generator(np.random.PCG64(w.seed + 1))
    flat = np.sort(rng.choice(w.B * w.H * w.N, size=count, replace=False))
    return np.stack(np.unravel_index(flat, (w.B, w.H, w.N)), axis=1).astype(np.int64)


def sampled_key_rows(w: Workload, count: int = N_SAMPLED_ROWS) -> np.ndarray:
    """Distinct flat (b, h, j) indices of sampled key rows (for dK, dV)."""
    rng = np.random.Generator(np.random.PCG64(w.seed + 2))
    flat = np.sort(rng.choice(w.B * w.H * w.N, size=count, replace=False))
    return np.stack(np.unravel_index(flat, (w.B, w.H, w.N)), axis=1).astype(np.int64)


def fingerprint(bits: np.ndarray) -> str:
    """Short content hash of a bit array, to detect generator drift between
    the machine that wrote a stored expected value and the one reading it."""
    import hashlib

    return hashlib.sha256(np.ascontiguousarray(bits).tobytes()).hexdigest()[:16]


def make_aggregation_inputs(M, H, C, d, seed, with_dout=True) -> dict:
    """Seeded bf16 inputs of the channel aggregation: q (H, d), k and v
    (M, H, C, d), and dout (M, H, d). Draw order q, k, v, dout."""
    rng = np.random.Generator(np.random.PCG64(seed))
    out = {"q": random_bf16(rng, (H, d)), "k": random_bf16(rng, (M, H, C, d)), "v": random_bf16(rng, (M, H, C, d))}
    if with_dout:
        out["dout"] = random_bf16(rng, (M, H, d))
    return out
