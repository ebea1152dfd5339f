"""Plain, slow, fp64 CPU oracle of the gradient-attribution hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product package imports or calls
this module; it exists so that tests, the smoke check and the bench's CPU
baseline can compare the HIP library against the method's definition.  It
shares no code with the HIP path: inputs come from the ``synth`` generators.

Everything is computed in float64 from the exact values of the (fp32, bf16
or fp16) inputs.  Each function cites the passage of the paper it follows:

* the double-sided per-module random projection of linear-layer gradients
  (Figure 1 caption; Appendix B, paragraph "Gradients"), with the compressed
  gradient P_i = sum_t (R^T g_t)(S^T a_t)^T, optionally of the gradient
  normalised by a factored (Adafactor) second moment (Figure 1 caption);
* unit normalisation ("grad-cosine", section "Attribution Pipelines" and the
  method-family table), the empirical-Fisher / autocorrelation
  preconditioner ("Flat (full) autocorrelation" in the method-family table;
  the TrackStar description in "Attribution Pipelines") and its diagonal;
* exact top-k lookup of the most influential training items (section
  "Attribution Pipelines": every gradient store supports exact top-k).

Readings taken where the paper is silent are listed in the repository's
design notes; the ones that change a result are repeated at each function.
Parity status: every function here is pinned by the tests in
``tests/test_oracle_pins.py``.
"""
from __future__ import annotations

from typing import Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "as_f64", "bf16_bits_to_f64", "to_f16", "project_explicit", "project",
    "project_tokens", "factored_second_moment", "project_normalized", "project_concat", "unit_normalize",
    "accumulate_diag", "accumulate_full", "kfac_factors", "finalize_diag", "finalize_full",
    "precond_apply", "scores", "score_topk", "merge_topk", "PAD_SCORE", "PAD_INDEX",
]

PAD_SCORE = -np.inf
PAD_INDEX = -1


# ----------------------------------------------------------------------------
# exact decoding of the stored input formats
# ----------------------------------------------------------------------------
def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) to float64: the bf16 value is the top half
    of an IEEE float32."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return u.view(np.float32).astype(np.float64)


def as_f64(x: np.ndarray) -> np.ndarray:
    """Exact float64 value of an fp32 / fp16 array or of bf16 uint16 bits."""
    x = np.asarray(x)
    if x.dtype == np.uint16:
        return bf16_bits_to_f64(x)
    return x.astype(np.float64)


def to_f16(x: np.ndarray) -> np.ndarray:
    """Round to fp16 with round-to-nearest-even (numpy's cast)."""
    return np.asarray(x, dtype=np.float64).astype(np.float16)


# ----------------------------------------------------------------------------
# (1) per-example double-sided random projection
# ----------------------------------------------------------------------------
def _lengths(n: int, T: int, length: Optional[Sequence[int]]) -> np.ndarray:
    if length is None:
        return np.full(n, T, dtype=np.int64)
    L = np.asarray(length, dtype=np.int64)
    if L.shape != (n,) or (L < 0).any() or (L > T).any():
        raise ValueError("length must hold n values in [0, T]")
    return L


def project_explicit(a: np.ndarray, g: np.ndarray, R: np.ndarray, S: np.ndarray,
                     length: Optional[Sequence[int]] = None) -> np.ndarray:
    """Compressed gradient of one linear module from the explicit gradient.

    For example i the weight gradient of a linear layer y = W x summed over
    its valid tokens is G_i = sum_{t < len_i} g_t a_t^T (d_out x d_in); the
    double-sided projection (Figure 1 caption; Appendix B "Gradients")
    compresses it to P_i = R^T G_i S (k x k).  Row i of the result is P_i
    flattened row-major, entry [r * k + c] = P_i[r, c]: r indexes R's columns
    (the output side), c indexes S's columns (the input side).

    a: [n, T, d_in], g: [n, T, d_out], R: [d_out, k], S: [d_in, k].
    Tokens t >= len_i are never read (they may hold NaN padding).
    Returns float64 [n, k*k].
    """
    n, T, _ = a.shape
    L = _lengths(n, T, length)
    Rf, Sf = as_f64(R), as_f64(S)
    k = Rf.shape[1]
    out = np.zeros((n, k * k))
    for i in range(n):
        ai = as_f64(a[i, :L[i]])
        gi = as_f64(g[i, :L[i]])
        G = gi.T @ ai                      # d_out x d_in, the full gradient
        out[i] = (Rf.T @ G @ Sf).reshape(-1)
    return out


def project(a: np.ndarray, g: np.ndarray, R: np.ndarray, S: np.ndarray,
            length: Optional[Sequence[int]] = None) -> np.ndarray:
    """Same quantity as ``project_explicit`` without forming G_i.

    P_i = sum_t (R^T g_t)(S^T a_t)^T = (g_i R)^T (a_i S) with g_i, a_i the
    valid-token rows: the factored form the method exists to exploit
    (Figure 1 caption; Appendix B "Gradients").  Float64 [n, k*k].
    """
    n, T, _ = a.shape
    L = _lengths(n, T, length)
    Rf, Sf = as_f64(R), as_f64(S)
    k = Rf.shape[1]
    out = np.zeros((n, k * k))
    for i in range(n):
        gt = as_f64(g[i, :L[i]]) @ Rf         # len x k, R^T g_t per token
        at = as_f64(a[i, :L[i]]) @ Sf         # len x k, S^T a_t per token
        out[i] = (gt.T @ at).reshape(-1)
    return out


def project_tokens(a: np.ndarray, g: np.ndarray, R: np.ndarray, S: np.ndarray,
                   length: Optional[Sequence[int]] = None) -> np.ndarray:
    """Per-token compressed gradients (Figure 1 caption: attribution scores
    are per-token or per-sequence): for token t of example i the k x k block
    (R^T g_t)(S^T a_t)^T, flattened like ``project_explicit``; the
    per-example projection is their sum over valid tokens.  Float64
    [n, T, k*k], rows of tokens t >= len_i zero (never read)."""
    n, T, _ = a.shape
    L = _lengths(n, T, length)
    Rf, Sf = as_f64(R), as_f64(S)
    k = Rf.shape[1]
    out = np.zeros((n, T, k * k))
    for i in range(n):
        for t in range(L[i]):
            out[i, t] = np.outer(Rf.T @ as_f64(g[i, t]), Sf.T @ as_f64(a[i, t])).reshape(-1)
    return out


def factored_second_moment(v_out: np.ndarray, v_in: np.ndarray) -> np.ndarray:
    """Factored (Adafactor) second-moment estimate of a d_out x d_in weight:
    V = v_out v_in^T / sum(v_out), from its row factor v_out and column
    factor v_in (Figure 1 caption: Adafactor second moments as a
    normalisation option).  Non-positive factors are read as 0.  Float64."""
    r = np.maximum(np.asarray(v_out, dtype=np.float64), 0.0)
    c = np.maximum(np.asarray(v_in, dtype=np.float64), 0.0)
    tot = r.sum()
    return np.outer(r, c) / tot if tot > 0 else np.zeros((r.size, c.size))


def project_normalized(a: np.ndarray, g: np.ndarray, R: np.ndarray, S: np.ndarray,
                       v_out: np.ndarray, v_in: np.ndarray,
                       length: Optional[Sequence[int]] = None) -> np.ndarray:
    """Projection of the optimizer-normalised gradient (Figure 1 caption:
    normalisation by Adafactor second moments, before projection; used by
    TrackStar, section "Attribution Pipelines").

    For example i: G_i = sum_{t < len_i} g_t a_t^T, then the elementwise
    normalised gradient N_i = G_i / sqrt(V) with V the factored second moment
    (``factored_second_moment``), 0 wherever V is 0 (reading: no epsilon),
    then P_i = R^T N_i S, flattened as in ``project_explicit``.
    Float64 [n, k*k].
    """
    n, T, _ = a.shape
    L = _lengths(n, T, length)
    Rf, Sf = as_f64(R), as_f64(S)
    k = Rf.shape[1]
    V = factored_second_moment(v_out, v_in)
    inv = np.zeros_like(V)
    pos = V > 0
    inv[pos] = 1.0 / np.sqrt(V[pos])
    out = np.zeros((n, k * k))
    for i in range(n):
        G = as_f64(g[i, :L[i]]).T @ as_f64(a[i, :L[i]])
        out[i] = (Rf.T @ (G * inv) @ Sf).reshape(-1)
    return out


def project_concat(per_module: Sequence[np.ndarray]) -> np.ndarray:
    """Concatenate per-module k*k blocks in module order into one row per
    example (the per-module layout of the gradient store, section
    "Attribution Pipelines": stores are indexed by module)."""
    return np.concatenate([np.asarray(p, dtype=np.float64) for p in per_module], axis=1)


# ----------------------------------------------------------------------------
# (2) normalisation and preconditioning
# ----------------------------------------------------------------------------
def unit_normalize(X: np.ndarray) -> np.ndarray:
    """Scale every row to unit Euclidean length ("grad-cosine": identity
    Hessian plus unit normalisation).  The norm is taken over the whole
    concatenated row; a zero row stays zero (no epsilon)."""
    X = as_f64(X)
    nrm = np.sqrt((X * X).sum(axis=1, keepdims=True))
    out = np.zeros_like(X)
    nz = nrm[:, 0] > 0
    out[nz] = X[nz] / nrm[nz]
    return out


def accumulate_diag(X: np.ndarray) -> np.ndarray:
    """Column sums of squares h_j = sum_i x_ij^2: the diagonal of the
    second-moment matrix G^T G of the store, unscaled."""
    X = as_f64(X)
    return (X * X).sum(axis=0)


def accumulate_full(X: np.ndarray) -> np.ndarray:
    """H = G^T G over the rows of X, unscaled, full symmetric (the flat
    autocorrelation / empirical Fisher of the method-family table)."""
    X = as_f64(X)
    return X.T @ X


def kfac_factors(a: np.ndarray, g: np.ndarray,
                 length: Optional[Sequence[int]] = None) -> Tuple[np.ndarray, np.ndarray]:
    """K-FAC factors of one linear module over the valid tokens of a batch
    (Figure 1 caption: K-FAC among the Hessian approximations; the factors
    are the input and output-gradient second moments whose Kronecker product
    approximates the module's Fisher): A = sum_i sum_{t < len_i} a_t a_t^T
    (d_in x d_in) and Gamma = sum g_t g_t^T (d_out x d_out), unscaled.
    a: [n, T, d_in], g: [n, T, d_out]; padding is never read.  Float64."""
    n, T, _ = a.shape
    L = _lengths(n, T, length)
    A = np.zeros((a.shape[-1], a.shape[-1]))
    Gm = np.zeros((g.shape[-1], g.shape[-1]))
    for i in range(n):
        ai = as_f64(a[i, :L[i]])
        gi = as_f64(g[i, :L[i]])
        A += ai.T @ ai
        Gm += gi.T @ gi
    return A, Gm


def finalize_diag(h: np.ndarray, n_rows: int) -> np.ndarray:
    """Diagonal preconditioner m_j = (h_j / N)^{-1/2}; a coordinate with zero
    second moment maps to 0 so that it contributes nothing to any score."""
    hn = np.asarray(h, dtype=np.float64) / float(n_rows)
    m = np.zeros_like(hn)
    pos = hn > 0
    m[pos] = 1.0 / np.sqrt(hn[pos])
    return m


def finalize_full(H: np.ndarray, n_rows: int) -> Tuple[np.ndarray, np.ndarray]:
    """Inverse square root of the normalised second moment Hn = H / N.

    Hn is symmetrised, eigendecomposed in float64 (Hn = V diag(lam) V^T) and
    M = V diag(lam^{-1/2}) V^T is returned with the eigenvalues.  Eigenvalues
    at or below lam_max * D * eps64 are treated as zero (pseudo-inverse
    square root), so M stays finite on a rank-deficient store.
    """
    H = np.asarray(H, dtype=np.float64) / float(n_rows)
    H = 0.5 * (H + H.T)
    lam, V = np.linalg.eigh(H)
    D = H.shape[0]
    floor = max(lam.max(), 0.0) * D * np.finfo(np.float64).eps
    f = np.zeros_like(lam)
    keep = lam > floor
    f[keep] = 1.0 / np.sqrt(lam[keep])
    M = (V * f) @ V.T
    return 0.5 * (M + M.T), lam


def precond_apply(X: np.ndarray, mode: str, M: Optional[np.ndarray] = None,
                  unit_norm: bool = True) -> np.ndarray:
    """Precondition then (optionally) unit-normalise rows, in float64.

    Order: precondition -> unit-normalise; the caller casts to the store
    dtype.  mode "none": y = x; "diag": y = m * x (elementwise);
    "full": y = M x for each row (M symmetric), i.e. Y = X M^T.
    """
    X = as_f64(X)
    if mode == "none":
        Y = X.copy()
    elif mode == "diag":
        Y = X * np.asarray(M, dtype=np.float64)[None, :]
    elif mode == "full":
        Y = X @ np.asarray(M, dtype=np.float64).T
    else:
        raise ValueError(mode)
    return unit_normalize(Y) if unit_norm else Y


# ----------------------------------------------------------------------------
# (3) scoring and exact top-k
# ----------------------------------------------------------------------------
def scores(Q: np.ndarray, G: np.ndarray) -> np.ndarray:
    """All query x store inner products s_qj = <q, g_j> in float64 (the
    cosine when both sides are unit rows)."""
    return as_f64(Q) @ as_f64(G).T


def _select(sc: np.ndarray, idx: np.ndarray, k: int) -> Tuple[np.ndarray, np.ndarray]:
    """The k best of one query's candidates ordered by (score desc, index
    asc).  NaN and -inf scores are never selected (reading: a candidate
    with no finite lower bound ranks below every slot's padding value, so
    it cannot be told apart from an empty slot); +inf ranks first.  Missing
    slots are (-inf, -1)."""
    ok = ~np.isnan(sc) & ~np.isneginf(sc)
    sc, idx = sc[ok], idx[ok]
    order = np.lexsort((idx, -sc))        # primary -score, secondary index
    sc, idx = sc[order][:k], idx[order][:k]
    out_s = np.full(k, PAD_SCORE)
    out_i = np.full(k, PAD_INDEX, dtype=np.int64)
    out_s[:len(sc)] = sc
    out_i[:len(idx)] = idx
    return out_s, out_i


def score_topk(Q: np.ndarray, G: np.ndarray, k: int, index_base: int = 0
               ) -> Tuple[np.ndarray, np.ndarray]:
    """Exact top-k of every query over the store (the store lookup of section
    "Attribution Pipelines"): scores (float64 [nq, k]) and store indices
    (int64 [nq, k], offset by index_base), ordered by (score desc, index
    asc)."""
    S = scores(Q, G)
    nq, ng = S.shape
    idx = np.arange(ng, dtype=np.int64) + index_base
    outs = np.full((nq, k), PAD_SCORE)
    outi = np.full((nq, k), PAD_INDEX, dtype=np.int64)
    for q in range(nq):
        outs[q], outi[q] = _select(S[q], idx, k)
    return outs, outi


def merge_topk(s1: np.ndarray, i1: np.ndarray, s2: np.ndarray, i2: np.ndarray,
               k: int) -> Tuple[np.ndarray, np.ndarray]:
    """Top-k of the union of two candidate lists per query (padding entries
    with index -1 are dropped first).  Merging the lists of consecutive store
    chunks gives the top-k of the whole store."""
    nq = s1.shape[0]
    outs = np.full((nq, k), PAD_SCORE)
    outi = np.full((nq, k), PAD_INDEX, dtype=np.int64)
    for q in range(nq):
        sc = np.concatenate([s1[q], s2[q]]).astype(np.float64)
        ix = np.concatenate([i1[q], i2[q]]).astype(np.int64)
        keep = ix >= 0
        outs[q], outi[q] = _select(sc[keep], ix[keep], k)
    return outs, outi
