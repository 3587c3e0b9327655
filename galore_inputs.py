"""Seeded synthetic inputs for the GaLore 2 hot path (harness side).

Holds none of the method's arithmetic: it only draws planted-spectrum gradients,
weights and optimizer states with the shapes, spectra and storage precisions of
the Llama-shaped workloads, and rounds them to their storage dtype.  The same
stored bits feed both the HIP library and the CPU oracle.

Gradient recipe:  G = U diag(s) V^T + noise * N(0, 1), with U (m x d) and
V (n x d), d = min(m, n), Haar-distributed orthonormal columns (QR of a Gaussian
matrix with the columns multiplied by sign(diag(R)), Mezzadri 2007), then
rounded to fp32 or to bf16 (round-to-nearest-even).

The paper trains on C4 with Llama models (shapes of its Llama-7B table:
hidden 4096, intermediate 11008, 32 layers); no real gradients are available
here, so these planted-spectrum matrices stand in for them.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, List, Tuple

import numpy as np

# --------------------------------------------------------------------------
# spectra (s_i for i = 0 .. d-1)
# --------------------------------------------------------------------------


def spectrum_geometric_cut(d: int, scale: float = 10.0, ratio: float = 0.85, cut: int = 64) -> np.ndarray:
    i = np.arange(d, dtype=np.float64)
    s = scale * ratio ** i
    s[cut:] = 0.0
    return s


def spectrum_geometric(d: int, ratio: float = 0.9) -> np.ndarray:
    return ratio ** np.arange(d, dtype=np.float64)


def spectrum_power(d: int, exponent: float) -> np.ndarray:
    return (np.arange(d, dtype=np.float64) + 1.0) ** (-exponent)


def spectrum_gapped(base: np.ndarray, r: int) -> np.ndarray:
    """Keep s_i for i < r and zero the rest: a spectrum with a clean gap at r."""
    s = base.copy()
    s[r:] = 0.0
    return s


# --------------------------------------------------------------------------
# workload presets
# --------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    groups: Tuple[Tuple[str, int, int, int], ...]   # (label, m, n, count)
    spectrum: Callable[[int], np.ndarray]
    noise: float
    dtype: str                                       # "f32" | "bf16"
    r: int
    p: int
    q: int
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    lr: float = 1e-3
    alpha: float = 0.25


def _layers(layers: int, h: int, f: int):
    return (("qkvo", h, h, 4 * layers), ("gate_up", h, f, 2 * layers), ("down", f, h, layers))


WORKLOADS = {
    "single-256x688": Workload("single-256x688", (("single", 256, 688, 1),),
                               lambda d: spectrum_geometric_cut(d), 1e-3, "f32", 32, 8, 2),
    "llama-60m": Workload("llama-60m", _layers(8, 512, 1376), lambda d: spectrum_geometric(d, 0.9),
                          1e-4, "f32", 128, 8, 2),
    "llama-350m": Workload("llama-350m", _layers(24, 1024, 2736), lambda d: spectrum_power(d, 1.0),
                           1e-4, "f32", 256, 16, 2),
    "llama-1b": Workload("llama-1b", _layers(24, 2048, 5461), lambda d: spectrum_power(d, 0.8),
                         1e-4, "bf16", 512, 16, 2),
    "llama-7b": Workload("llama-7b", _layers(32, 4096, 11008), lambda d: spectrum_power(d, 0.7),
                         1e-4, "bf16", 1024, 32, 2),
}

# --------------------------------------------------------------------------
# storage rounding
# --------------------------------------------------------------------------


def bf16_bits_from_f32(x: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest-even) and return the 16-bit patterns (uint16)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def f32_from_bf16_bits(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# --------------------------------------------------------------------------
# host (numpy) generators
# --------------------------------------------------------------------------


def haar_columns(rng: np.random.Generator, rows: int, cols: int) -> np.ndarray:
    """rows x cols with orthonormal columns, Haar distributed (Mezzadri 2007)."""
    z = rng.standard_normal((rows, cols))
    qm, rm = np.linalg.qr(z)
    d = np.sign(np.diag(rm))
    d[d == 0] = 1.0
    return qm * d


def planted_gradient(m: int, n: int, spectrum: np.ndarray, noise: float, seed: int,
                     rank: int | None = None) -> np.ndarray:
    """fp64 m x n matrix U diag(s) V^T + noise N(0,1) (not yet rounded).

    ``spectrum`` has min(m, n) entries; ``rank`` (optional) limits the planted
    part to its first ``rank`` directions (for exact-recovery cases).
    """
    rng = np.random.default_rng(seed)
    d = min(m, n)
    kk = d if rank is None else rank
    U = haar_columns(rng, m, kk)
    V = haar_columns(rng, n, kk)
    G = (U * spectrum[:kk]) @ V.T
    if noise:
        G = G + noise * rng.standard_normal((m, n))
    return G


@dataclasses.dataclass
class Stored:
    """A matrix as stored for the library (``data``: fp32 array or bf16 uint16
    bits) plus its exact fp64 value for the oracle."""
    data: np.ndarray
    dtype: str
    exact: np.ndarray


def store(x: np.ndarray, dtype: str) -> Stored:
    if dtype == "f32":
        d = np.ascontiguousarray(x, dtype=np.float32)
        return Stored(d, "f32", d.astype(np.float64))
    if dtype == "bf16":
        b = bf16_bits_from_f32(np.asarray(x, dtype=np.float32))
        return Stored(b, "bf16", f32_from_bf16_bits(b).astype(np.float64))
    raise ValueError(dtype)


def weights(m: int, n: int, seed: int, std: float = 0.02) -> np.ndarray:
    return (std * np.random.default_rng(seed).standard_normal((m, n))).astype(np.float32)


def lowrank_state(rows: int, cols: int, seed: int, scale: float = 1e-3) -> Tuple[np.ndarray, ...]:
    """(R, M, V) fp32 arrays resembling a running low-rank Adam state."""
    rng = np.random.default_rng(seed)
    R = (scale * rng.standard_normal((rows, cols))).astype(np.float32)
    M = (0.5 * scale * rng.standard_normal((rows, cols))).astype(np.float32)
    V = ((scale * rng.standard_normal((rows, cols))) ** 2).astype(np.float32)
    return R, M, V


def gradient_seed(workload_index: int, matrix_id: int) -> int:
    return 1000 * workload_index + matrix_id


def sketch_seed(update_index: int) -> int:
    return 20250429 + update_index


# --------------------------------------------------------------------------
# device (torch) generator for the full-size throughput workload
# --------------------------------------------------------------------------


def torch_planted_group(m: int, n: int, count: int, spectrum: np.ndarray, noise: float, seed: int,
                        dtype: str, device: str = "cuda"):
    """``count`` m x n planted-spectrum gradients on ``device``.

    One Haar pair (U, V) per shape group; each matrix applies an independent
    random signed permutation to the rows and to the columns of U diag(s) V^T
    (which keeps the Haar law of the singular vectors and the exact spectrum)
    and adds its own noise.  Returns a (count, m, n) tensor in fp32 or bf16.
    """
    import torch

    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    d = min(m, n)

    def haar(rows, cols):
        z = torch.randn(rows, cols, generator=gen, device=device, dtype=torch.float32)
        qm, rm = torch.linalg.qr(z)
        sgn = torch.sign(torch.diagonal(rm))
        sgn[sgn == 0] = 1
        return qm * sgn

    U = haar(m, d)
    V = haar(n, d)
    s = torch.as_tensor(spectrum[:d], dtype=torch.float32, device=device)
    base = (U * s) @ V.T.contiguous()
    del U, V
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    out = torch.empty((count, m, n), dtype=tdt, device=device)
    for i in range(count):
        pr = torch.randperm(m, generator=gen, device=device)
        pc = torch.randperm(n, generator=gen, device=device)
        sr = torch.randint(0, 2, (m, 1), generator=gen, device=device).float() * 2 - 1
        sc = torch.randint(0, 2, (1, n), generator=gen, device=device).float() * 2 - 1
        g = base.index_select(0, pr).index_select(1, pc) * sr * sc
        if noise:
            g.add_(torch.randn(m, n, generator=gen, device=device), alpha=noise)
        out[i].copy_(g)
        del g
    return out


def group_list(w: Workload) -> List[Tuple[str, int, int, int]]:
    return list(w.groups)
