"""Host finalize of the second-moment preconditioner: M = (H / N)^{-1/2}.

Fitting the preconditioner is a step of its own, run once per store between
accumulation and application (TrackStar's Fisher fitting in section
"Attribution Pipelines"; the flat autocorrelation of the method-family
table).  It is the only step of the path that is not a GPU kernel: the
accumulated H (fp32, upper triangle, from ``attr_precond_accumulate``) is
copied to the host, symmetrised and eigendecomposed in fp64 with LAPACK
(numpy's ``eigh``), and M goes back to the device in fp32 for
``attr_precond_apply``.

Readings: H is the unscaled sum over the N accumulated rows, so it is divided
by N here; no damping; eigenvalues at or below lam_max * D * eps64 are
treated as zero (pseudo-inverse square root), so M stays finite on a
rank-deficient store; a coordinate with zero diagonal second moment gets a
zero scale.
"""
from __future__ import annotations

import numpy as np
import torch

__all__ = ["finalize_diag", "finalize_full"]


def finalize_diag(h: torch.Tensor, n_rows: int) -> torch.Tensor:
    """m = (h / N)^{-1/2}, 0 where h is 0; h: fp32 [D] on the device."""
    if h.dim() != 1 or h.dtype != torch.float32:
        raise ValueError("h must be an fp32 vector [D]")
    if n_rows <= 0:
        raise ValueError("n_rows must be positive")
    hn = h.detach().double().cpu().numpy() / float(n_rows)
    m = np.zeros_like(hn)
    pos = hn > 0
    m[pos] = 1.0 / np.sqrt(hn[pos])
    return torch.from_numpy(m.astype(np.float32)).to(h.device)


def finalize_full(H: torch.Tensor, n_rows: int, return_eigenvalues: bool = False):
    """M = (H / N)^{-1/2} from the upper triangle of H (fp32 [D, D] on the
    device): symmetrised, eigendecomposed in fp64 (LAPACK syevd through
    numpy), eigenvalues at or below lam_max * D * eps64 dropped.  Returns M
    (fp32 [D, D], same device), and the eigenvalues of H / N (fp64, host,
    ascending) when return_eigenvalues is set."""
    if H.dim() != 2 or H.shape[0] != H.shape[1] or H.dtype != torch.float32:
        raise ValueError("H must be a square fp32 matrix [D, D]")
    if n_rows <= 0:
        raise ValueError("n_rows must be positive")
    Hu = np.triu(H.detach().cpu().numpy().astype(np.float64))
    Hs = (Hu + np.triu(Hu, 1).T) / float(n_rows)
    lam, V = np.linalg.eigh(Hs)
    floor = max(lam.max(), 0.0) * Hs.shape[0] * np.finfo(np.float64).eps
    f = np.where(lam > floor, 1.0 / np.sqrt(np.maximum(lam, floor)), 0.0)
    M = (V * f) @ V.T
    M = 0.5 * (M + M.T)
    Mt = torch.from_numpy(M.astype(np.float32)).to(H.device)
    return (Mt, lam) if return_eigenvalues else Mt
