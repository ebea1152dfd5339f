"""Seeded generators for the five synthetic workloads.

Every generator uses numpy's ``Generator(PCG64)`` through ``default_rng`` with
the seeds stated below, draws in float64 and then casts.  Casts are
round-to-nearest-even: fp16 through numpy, bf16 by rounding the float32 bit
pattern (returned as ``uint16`` bit patterns, since numpy has no bf16 dtype).

Workloads (the paper's attribution pipeline, section "Attribution Pipelines",
and its scaling study shapes; the values are synthetic):

* ``tiny``    one 64->64 module, 256 examples x 32 tokens, fp32, k=16.
* ``gpt2``    12 layers x (qkv 768->2304, out 768->768, up 768->3072,
              down 3072->768), T=512, bf16, g scaled by 1e-2, k=16.
* ``llama1b`` 16 layers x (q,k,v,o 2048->2048, gate,up 2048->8192,
              down 8192->2048), T=2048 with lengths uniform in [256, 2048],
              a ~ Student-t(4), g ~ N(0,1)*1e-2, bf16, k=16.
* ``precond`` low-rank-plus-noise rows G = Z F^T + 0.1 E (rank 64), fp16.
* ``store``   unit-length fp16 rows (uniform directions) plus queries with
              planted near-duplicates of known rows.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "ModuleShape", "Workload", "TINY", "GPT2", "LLAMA1B", "workload",
    "to_bf16_bits", "projection_pair", "module_example", "module_queries",
    "tiny_inputs", "example_lengths", "lowrank_factor", "lowrank_rows",
    "lowrank_queries", "unit_rows", "planted_queries", "nan_pad",
]


# ----------------------------------------------------------------------------
# casts (data layout only)
# ----------------------------------------------------------------------------
def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float values to bf16 (round-to-nearest-even), as uint16 bits."""
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    rounding = ((u >> 16) & 1) + 0x7FFF
    out = ((u + rounding) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        out[nan] = 0x7FC0
    return out.reshape(f.shape)


# ----------------------------------------------------------------------------
# workload shapes
# ----------------------------------------------------------------------------
@dataclasses.dataclass(frozen=True)
class ModuleShape:
    name: str
    d_in: int
    d_out: int


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    modules: Tuple[ModuleShape, ...]
    n_examples: int
    T: int
    k: int
    dtype: str            # "f32" or "bf16" for a/g/R/S
    g_scale: float
    a_law: str            # "normal" or "student_t4"
    n_queries: int
    topk: int

    @property
    def D(self) -> int:
        return len(self.modules) * self.k * self.k

    def out_col(self, m: int) -> int:
        return m * self.k * self.k

    def elems_per_token(self) -> int:
        return sum(md.d_in + md.d_out for md in self.modules)


def _gpt2_modules() -> Tuple[ModuleShape, ...]:
    mods: List[ModuleShape] = []
    for layer in range(12):
        mods += [ModuleShape(f"h{layer}.attn.qkv", 768, 2304),
                 ModuleShape(f"h{layer}.attn.out", 768, 768),
                 ModuleShape(f"h{layer}.mlp.up", 768, 3072),
                 ModuleShape(f"h{layer}.mlp.down", 3072, 768)]
    return tuple(mods)


def _llama1b_modules() -> Tuple[ModuleShape, ...]:
    mods: List[ModuleShape] = []
    for layer in range(16):
        for nm in ("q", "k", "v", "o"):
            mods.append(ModuleShape(f"l{layer}.attn.{nm}", 2048, 2048))
        mods += [ModuleShape(f"l{layer}.mlp.gate", 2048, 8192),
                 ModuleShape(f"l{layer}.mlp.up", 2048, 8192),
                 ModuleShape(f"l{layer}.mlp.down", 8192, 2048)]
    return tuple(mods)


TINY = Workload("tiny", (ModuleShape("linear", 64, 64),), 256, 32, 16, "f32",
                1.0, "normal", 8, 5)
GPT2 = Workload("gpt2", _gpt2_modules(), 4096, 512, 16, "bf16", 1e-2,
                "normal", 64, 10)
LLAMA1B = Workload("llama1b", _llama1b_modules(), 16384, 2048, 16, "bf16",
                   1e-2, "student_t4", 0, 0)


def workload(name: str) -> Workload:
    return {"tiny": TINY, "gpt2": GPT2, "llama1b": LLAMA1B}[name]


def _cast(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return x.astype(np.float32)
    if dtype == "bf16":
        return to_bf16_bits(x)
    if dtype == "f16":
        return x.astype(np.float16)
    raise ValueError(dtype)


# ----------------------------------------------------------------------------
# projection matrices and per-token inputs
# ----------------------------------------------------------------------------
def projection_pair(wl: Workload, m: int) -> Tuple[np.ndarray, np.ndarray]:
    """(R [d_out, k], S [d_in, k]) for module m, i.i.d. N(0, 1/k).

    Tiny uses ``default_rng(1)``; multi-module workloads ``default_rng([1, m])``.
    R is drawn first, then S.
    """
    md = wl.modules[m]
    rng = np.random.default_rng(1) if wl.name == "tiny" else np.random.default_rng([1, m])
    scale = 1.0 / np.sqrt(wl.k)
    R = rng.standard_normal((md.d_out, wl.k)) * scale
    S = rng.standard_normal((md.d_in, wl.k)) * scale
    return _cast(R, wl.dtype), _cast(S, wl.dtype)


def _draw_a(rng: np.random.Generator, shape, law: str) -> np.ndarray:
    if law == "normal":
        return rng.standard_normal(shape)
    if law == "student_t4":
        return rng.standard_t(4.0, size=shape)
    raise ValueError(law)


def module_example(wl: Workload, m: int, i: int, T: Optional[int] = None,
                   seed: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """(a [T, d_in], g [T, d_out]) of example i for module m.

    Drawn from ``default_rng([seed, m, i])``: a first, then g (times g_scale).
    Training examples use seed 0, queries seed 2.
    """
    md = wl.modules[m]
    T = wl.T if T is None else T
    rng = np.random.default_rng([seed, m, i])
    a = _draw_a(rng, (T, md.d_in), wl.a_law)
    g = rng.standard_normal((T, md.d_out)) * wl.g_scale
    return _cast(a, wl.dtype), _cast(g, wl.dtype)


def module_queries(wl: Workload, m: int, q: int, T: Optional[int] = None):
    return module_example(wl, m, q, T=T, seed=2)


def tiny_inputs():
    """The tiny workload exactly: returns dict with a, g, R, S, aq, gq (fp32)."""
    rng0 = np.random.default_rng(0)
    a = rng0.standard_normal((256, 32, 64)).astype(np.float32)
    g = rng0.standard_normal((256, 32, 64)).astype(np.float32)
    R, S = projection_pair(TINY, 0)
    rng2 = np.random.default_rng(2)
    aq = rng2.standard_normal((8, 32, 64)).astype(np.float32)
    gq = rng2.standard_normal((8, 32, 64)).astype(np.float32)
    return dict(a=a, g=g, R=R, S=S, aq=aq, gq=gq)


def example_lengths(n: int, lo: int = 256, hi: int = 2048, seed: int = 4) -> np.ndarray:
    """Per-example valid-token counts, uniform integers in [lo, hi]."""
    return np.random.default_rng(seed).integers(lo, hi + 1, n).astype(np.int32)


def nan_pad(x: np.ndarray, length: int) -> np.ndarray:
    """Copy of a [T, d] token array with rows >= length set to NaN (padding)."""
    y = np.array(x, copy=True)
    if y.dtype == np.uint16:
        y[length:] = 0x7FC0
    else:
        y[length:] = np.nan
    return y


# ----------------------------------------------------------------------------
# preconditioner and store workloads
# ----------------------------------------------------------------------------
def lowrank_factor(D: int = 8192, rank: int = 64, seed: int = 3) -> np.ndarray:
    """F [D, rank] ~ N(0, 1) from ``default_rng(seed)``."""
    return np.random.default_rng(seed).standard_normal((D, rank))


def lowrank_rows(start: int, stop: int, D: int = 8192, rank: int = 64,
                 seed: int = 3, chunk: int = 65536, noise: float = 0.1,
                 F: Optional[np.ndarray] = None) -> np.ndarray:
    """Rows [start, stop) of G = Z F^T + noise * E, cast to fp16.

    Row block c (rows [c*chunk, (c+1)*chunk)) draws Z [chunk, rank] then
    E [chunk, D] from ``default_rng([seed, c])``, so any prefix of a longer
    store equals the shorter store.
    """
    if F is None:
        F = lowrank_factor(D, rank, seed)
    out = np.empty((stop - start, D), dtype=np.float16)
    c0, c1 = start // chunk, (stop - 1) // chunk if stop > start else start // chunk - 1
    for c in range(c0, c1 + 1):
        rng = np.random.default_rng([seed, c])
        Z = rng.standard_normal((chunk, rank))
        lo, hi = max(start, c * chunk), min(stop, (c + 1) * chunk)
        # Only rows [lo, hi) of this block are needed; E is drawn row-major so
        # the draw of the block must still be complete up to row hi.
        nrow = hi - c * chunk
        E = rng.standard_normal((nrow, D))
        blk = Z[lo - c * chunk:nrow] @ F.T + noise * E[lo - c * chunk:]
        out[lo - start:hi - start] = blk.astype(np.float16)
    return out


def lowrank_queries(n: int, D: int = 8192, rank: int = 64, seed: int = 5,
                    F: Optional[np.ndarray] = None, factor_seed: int = 3) -> np.ndarray:
    """Query rows drawn like the store (same factor F), from ``default_rng([seed, 0])``."""
    if F is None:
        F = lowrank_factor(D, rank, factor_seed)
    return lowrank_rows(0, n, D=D, rank=rank, seed=seed, F=F)


def unit_rows(n: int, D: int, seed: int, dtype=np.float16) -> np.ndarray:
    """n rows drawn uniformly on the unit sphere of R^D (Gaussian direction), cast.

    This is the distribution a whitened, unit-normalised store approaches.
    """
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((n, D))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    return x.astype(dtype)


def planted_queries(store_rows: np.ndarray, targets: Sequence[int], n_queries: int,
                    cos: float = 0.9, seed: int = 4, dtype=np.float16) -> np.ndarray:
    """Queries whose first len(targets) rows are near-duplicates of store rows.

    Query p < len(targets) is cos * g_hat + sqrt(1 - cos^2) * u with g_hat the
    target row scaled to unit length and u a random unit vector orthogonal to
    it; the remaining queries are uniform random unit vectors.
    ``store_rows`` holds the target rows (already in the store's dtype).
    """
    D = store_rows.shape[1]
    rng = np.random.default_rng([seed, 1])
    out = np.empty((n_queries, D), dtype=np.float64)
    for p, j in enumerate(targets):
        gh = store_rows[p].astype(np.float64)
        gh /= np.linalg.norm(gh)
        u = rng.standard_normal(D)
        u -= (u @ gh) * gh
        u /= np.linalg.norm(u)
        out[p] = cos * gh + np.sqrt(1.0 - cos * cos) * u
    rest = rng.standard_normal((n_queries - len(targets), D))
    rest /= np.linalg.norm(rest, axis=1, keepdims=True)
    out[len(targets):] = rest
    return out.astype(dtype)
