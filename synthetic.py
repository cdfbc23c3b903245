"""Seeded synthetic Q/K/V for video-DiT-shaped attention layers.

This module is shared by the tests, the benchmark and the smoke check. It only draws random
inputs: it holds none of the attention method's arithmetic (no RoPE, no quantizer, no softmax).

The captured Wan2.2 / LongCat activations the paper measures on are not available, so inputs
are synthetic with the paper's workload shapes (d = 128; tens of thousands of tokens flattened
from a frames x rows x cols latent grid) and the structure the method targets: channel offsets
and a few outlier channels in Q/K, spatially smooth low-frequency structure shared by
neighbouring tokens, and a value offset that drifts smoothly with the frame index.

Every tensor of every (batch, head) comes from its own Philox stream keyed by
(seed, workload, call, tensor, batch, head), so any head can be regenerated on its own.
Values are formed in fp64/fp32 and rounded to bf16 (nearest even) last; the result is returned
as uint16 bf16 bit patterns.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

D = 128


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    grid: tuple  # (frames, rows, cols)
    structured: bool  # sinusoidal field + outliers (video-DiT-like) vs plain N(0,1)

    @property
    def N(self) -> int:
        F, Ht, Wd = self.grid
        return F * Ht * Wd


WORKLOADS = {
    # tiny: 4x16x16 grid, plain N(0,1) tokens with a K channel offset and a frame-smooth V offset
    "tiny": Workload("tiny", 1, 2, (4, 16, 16), False),
    # small video-DiT layer: 21x39x40 latent grid (N = 32760), 12 heads
    "dit_small": Workload("dit_small", 1, 12, (21, 39, 40), True),
    # large video-DiT layer: 21x60x60 latent grid (N = 75600), 40 heads
    "dit_large": Workload("dit_large", 1, 40, (21, 60, 60), True),
    # 40 heads on the 21x39x40 grid (the 4-bit study shape)
    "dit_small_h40": Workload("dit_small_h40", 1, 40, (21, 39, 40), True),
}
_WID = {"tiny": 1, "dit_small": 2, "dit_large": 3, "dit_small_h40": 5}
_TID = {"q": 0, "k": 1, "v": 2}


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.array(x, dtype=np.float32, copy=True, order="C").view(np.uint32)
    lsb = (u >> 16) & np.uint32(1)
    u += np.uint32(0x7FFF)  # finite inputs only: no uint32 overflow below the NaN range
    u += lsb
    u >>= 16
    return u.astype(np.uint16)


def bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _rng(seed: int, wid: int, call: int, tensor: int, b: int, h: int, salt: int = 0) -> np.random.Generator:
    key = np.random.SeedSequence([int(seed), wid, call, tensor, b, h, salt]).generate_state(2, dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def _grid_coords(grid):
    F, Ht, Wd = grid
    n = np.arange(F * Ht * Wd)
    return n // (Ht * Wd), (n // Wd) % Ht, n % Wd


def _base_head(w: Workload, seed: int, tensor: str, b: int, h: int) -> np.ndarray:
    """Pre-rounding fp32 values of one (tensor, batch, head) at call 0 (the shared base field)."""
    F, Ht, Wd = w.grid
    N = w.N
    wid, tid = _WID[w.name], _TID[tensor]
    rng = _rng(seed, wid, 0, tid, b, h)
    f, y, x = _grid_coords(w.grid)
    if w.structured:
        # Sum of 4 low-frequency 3D sinusoids per channel:
        #   field[n, c] = sum_m A[m, c] sin(2 pi (kt f/F + kh y/Ht + kw x/Wd) + phi[m, c])
        # written as [sin g_m, cos g_m] @ [A cos phi; A sin phi] (angle-addition identity).
        G = np.empty((N, 8), np.float64)
        for m in range(4):
            while True:
                kap = rng.integers(0, 3, size=3)
                if kap.any():
                    break
            g = 2.0 * np.pi * (kap[0] * f / F + kap[1] * y / Ht + kap[2] * x / Wd)
            G[:, m], G[:, 4 + m] = np.sin(g), np.cos(g)
        A = rng.normal(0.0, 0.5, size=(4, D))
        phi = rng.uniform(0.0, 2.0 * np.pi, size=(4, D))
        W = np.concatenate([A * np.cos(phi), A * np.sin(phi)], axis=0)
        X = (G @ W).astype(np.float32)
        X += 0.5 * rng.standard_normal((N, D), dtype=np.float32)
    else:
        X = rng.standard_normal((N, D), dtype=np.float32)
    if tensor == "k":
        X += rng.normal(0.0, 3.0, size=D).astype(np.float32)[None, :]
    elif tensor == "v":
        a = rng.normal(0.0, 1.0, size=D)
        bb = rng.normal(0.0, 1.0, size=D)
        frame = np.cos(np.pi * np.arange(F) / max(F - 1, 1))
        X += (a[None, :] + bb[None, :] * frame[f][:, None]).astype(np.float32)
    elif tensor == "q" and w.structured:
        X += rng.normal(0.0, 1.0, size=D).astype(np.float32)[None, :]
    if w.structured:
        # 1% of the channels (ceil(0.01 * 128) = 2) of this tensor are outliers, scaled x10
        ch = rng.choice(D, size=math.ceil(0.01 * D), replace=False)
        X[:, ch] *= 10.0
    return X


def _noise(w: Workload, seed: int, call: int, tensor: str, b: int, h: int) -> np.ndarray:
    rng = _rng(seed, _WID[w.name], call, _TID[tensor], b, h, salt=1)
    return rng.standard_normal((w.N, D), dtype=np.float32)


def make_qkv(name: str, seed: int = 0, call: int = 0, drift: float = 0.0, heads=None,
             token_outliers: bool = False):
    """Q, K, V as uint16 bf16 bits [B, H, N, 128] for a named workload.

    call / drift: X_call = bf16(X_base + drift * eps_call) with eps_call a fresh N(0,1) draw per
    call (the 'same layer, next denoising step' drift); call 0 with drift 0 is the base field.
    heads: optional list of flat head indices to generate (others are left zero).
    token_outliers: additionally scale 0.5% of the V tokens x10 (token-outlier stress field).
    """
    w = WORKLOADS[name]
    out = [np.zeros((w.B, w.H, w.N, D), np.uint16) for _ in range(3)]
    sel = range(w.B * w.H) if heads is None else heads

    def one(job):
        bh, t, tensor = job
        b, h = divmod(int(bh), w.H)
        X = _base_head(w, seed, tensor, b, h)
        if drift and call:
            X = X + np.float32(drift) * _noise(w, seed, call, tensor, b, h)
        if token_outliers and tensor == "v":
            rng = _rng(seed, _WID[w.name], call, 3, b, h, salt=2)
            tok = rng.choice(w.N, size=max(1, int(0.005 * w.N)), replace=False)
            X = X.copy()
            X[tok] *= 10.0
        out[t][b, h] = bf16_bits(X)

    _run([(bh, t, tensor) for bh in sel for t, tensor in enumerate(("q", "k", "v"))], one)
    return tuple(out)


def _run(jobs, fn):
    """Independent per-(tensor, head) jobs on a small thread pool (numpy releases the GIL)."""
    workers = max(1, min(16, len(os.sched_getaffinity(0)), len(jobs)))
    with ThreadPoolExecutor(workers) as ex:
        list(ex.map(fn, jobs))


def make_interpolated(name: str, step: int, steps: int = 8, seeds=(0, 1), heads=None):
    """Denoising-loop slice: X_t = bf16((1 - t/(steps-1)) Xa + t/(steps-1) Xb), fields from two seeds."""
    w = WORKLOADS[name]
    lam = np.float32(step / (steps - 1))
    out = [np.zeros((w.B, w.H, w.N, D), np.uint16) for _ in range(3)]
    sel = range(w.B * w.H) if heads is None else heads

    def one(job):
        bh, t, tensor = job
        b, h = divmod(int(bh), w.H)
        Xa = _base_head(w, seeds[0], tensor, b, h)
        Xb = _base_head(w, seeds[1], tensor, b, h)
        out[t][b, h] = bf16_bits((np.float32(1) - lam) * Xa + lam * Xb)

    _run([(bh, t, tensor) for bh in sel for t, tensor in enumerate(("q", "k", "v"))], one)
    return tuple(out)


def random_perm(N: int, seed: int, B: int = 1, H: int = 1) -> np.ndarray:
    """A seeded random permutation per (batch, head), int32 [B, H, N] (for gather tests)."""
    out = np.empty((B, H, N), np.int32)
    for b in range(B):
        for h in range(H):
            out[b, h] = _rng(seed, 99, 0, 9, b, h).permutation(N).astype(np.int32)
    return out
