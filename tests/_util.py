"""Helpers shared by the GPU tests: host arrays <-> device tensors, error metrics."""
import sys

import numpy as np
import torch


def say(*args):
    """Print and flush, so that a GPU run names its case before each step."""
    print(*args, flush=True)
    sys.stdout.flush()


def dev(x: np.ndarray, device="cuda") -> torch.Tensor:
    """Upload a synth array: uint16 arrays are bf16 bit patterns."""
    x = np.ascontiguousarray(x)
    if x.dtype == np.uint16:
        return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(x).to(device)


def host(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def row_rel_l2(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per-row ||got - ref|| / ||ref|| (0/0 counts as 0)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    num = np.linalg.norm(got - ref, axis=1)
    den = np.linalg.norm(ref, axis=1)
    out = np.where(den > 0, num / np.where(den > 0, den, 1.0), num)
    return out


def check_topk(got_s, got_i, ref_scores, k, index_base=0, tol=1e-3):
    """Top-k parity against the oracle's full fp64 score matrix.

    (a) every returned score is within tol of the oracle's score of the
        returned index and of the oracle's score at that rank;
    (b) every oracle item scoring above s_{k+1} + tol is returned;
    (c) the index at rank r equals the oracle's wherever the oracle scores
        are separated from both neighbours by more than tol;
    (d) returned indices are unique and scores non-increasing.
    """
    got_s = np.asarray(got_s, dtype=np.float64)
    got_i = np.asarray(got_i, dtype=np.int64)
    nq, ng = ref_scores.shape
    for q in range(nq):
        ref = ref_scores[q]
        order = np.lexsort((np.arange(ng), -ref))
        rs = ref[order]
        kk = min(k, ng)
        valid = got_i[q] >= 0
        assert valid.sum() == kk, (q, valid.sum(), kk)
        assert (got_i[q, kk:] == -1).all() and np.isneginf(got_s[q, kk:]).all()
        gi = got_i[q, :kk] - index_base
        gs = got_s[q, :kk]
        assert len(set(gi.tolist())) == kk, "duplicate indices"
        assert (np.diff(gs) <= 0).all(), "scores not sorted"
        assert (gi >= 0).all() and (gi < ng).all()
        assert np.abs(gs - ref[gi]).max() <= tol, (q, np.abs(gs - ref[gi]).max())
        assert np.abs(gs - rs[:kk]).max() <= tol
        s_next = rs[kk] if ng > kk else -np.inf
        must = order[:kk][rs[:kk] > s_next + tol]
        assert set(must.tolist()) <= set(gi.tolist()), (q, "missing a clear winner")
        for r in range(kk):
            left = rs[r - 1] - rs[r] if r > 0 else np.inf
            right = rs[r] - rs[r + 1] if r + 1 < ng else np.inf
            if left > tol and right > tol:
                assert gi[r] == order[r], (q, r, gi[r], order[r])


def check_topk_from_lists(got_s, got_i, ref_s, ref_i, returned_scores, k, tol=1e-3):
    """The checks of check_topk from the oracle's top-(k + 1) list instead of
    the full score matrix (for stores too large to score whole on the host).

    ref_s / ref_i: [nq, k + 1] the oracle's best k + 1 (score desc, index
    asc); returned_scores: [nq, k] the oracle's scores of the returned
    indices.  (a) returned scores within tol of the oracle's score of the
    returned index and of the oracle's score at that rank; (b) every oracle
    item scoring above s_{k+1} + tol is returned; (c) indices equal the
    oracle's wherever the oracle's scores are separated from both neighbours
    by more than tol; (d) indices unique and valid, scores non-increasing."""
    got_s = np.asarray(got_s, dtype=np.float64)
    got_i = np.asarray(got_i, dtype=np.int64)
    for q in range(got_s.shape[0]):
        rs, ri = ref_s[q], ref_i[q]
        gs, gi = got_s[q], got_i[q]
        assert (gi >= 0).all() and len(set(gi.tolist())) == k, "invalid or duplicate indices"
        assert (np.diff(gs) <= 0).all(), "scores not sorted"
        assert np.abs(gs - returned_scores[q]).max() <= tol, (q, np.abs(gs - returned_scores[q]).max())
        assert np.abs(gs - rs[:k]).max() <= tol, (q, np.abs(gs - rs[:k]).max())
        must = ri[:k][rs[:k] > rs[k] + tol]
        assert set(must.tolist()) <= set(gi.tolist()), (q, "missing a clear winner")
        for r in range(k):
            left = rs[r - 1] - rs[r] if r > 0 else np.inf
            right = rs[r] - rs[r + 1]
            if left > tol and right > tol:
                assert gi[r] == ri[r], (q, r, gi[r], ri[r])
