"""Parity at the full workload sizes, in the launch configurations the bench
times: outputs the oracle can recompute one by one (entries of H, rows of the
applied preconditioner, the scores of returned top-k entries) and properties
that hold at any size (planted near-duplicates rank first, no row of a large
random sample beats the k-th returned score).

Inputs are drawn on the device by torch's seeded generator (16-65 GB would
take minutes to draw and upload from the host); the oracle reads the same
values back, never an output of the HIP path.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_11660_amd as P
from tests._util import host, row_rel_l2, say

pytestmark = pytest.mark.gpu

D = 8192


def _lowrank_store(n, seed=3):
    """Low-rank-plus-noise fp16 rows (rank-64 factor, 0.1 noise), the
    preconditioner workload's distribution."""
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    F = torch.randn((D, 64), generator=gen, device="cuda")
    X = torch.empty((n, D), dtype=torch.float16, device="cuda")
    for i in range(0, n, 65536):
        m = min(65536, n - i)
        Z = torch.randn((m, 64), generator=gen, device="cuda")
        X[i:i + m] = (Z @ F.T + 0.1 * torch.randn((m, D), generator=gen, device="cuda")).half()
    return X


def _unit_store(n, seed):
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)
    G = torch.empty((n, D), dtype=torch.float16, device="cuda")
    for i in range(0, n, 65536):
        m = min(65536, n - i)
        c = torch.randn((m, D), generator=gen, device="cuda")
        G[i:i + m] = (c / c.norm(dim=1, keepdim=True)).half()
    return G


def test_syrk_full_config_sampled_entries():
    """H += X^T X over the 10^6 x 8192 store (four chunks of 250,000 rows);
    78 upper-triangle entries recomputed in fp64 from the same columns."""
    n = 1_000_000
    say(f"case: syrk full size n={n} D={D}")
    X = _lowrank_store(n)
    H = torch.zeros((D, D), dtype=torch.float32, device="cuda")
    P.attr_precond_accumulate(X, P.PRECOND_FULL, H)
    torch.cuda.synchronize()
    cols = np.sort(np.random.default_rng(7).choice(D, 12, replace=False))
    cols[0], cols[-1] = 0, D - 1                      # first and last tile edges
    Xc = host(X[:, torch.from_numpy(cols).cuda()]).astype(np.float64)
    ref = Xc.T @ Xc
    Hh = host(H)
    iu = np.triu_indices(len(cols))
    got = Hh[cols[iu[0]], cols[iu[1]]].astype(np.float64)
    err = np.abs(got - ref[iu]).max() / np.abs(ref).max()
    say("sampled H max rel err", err)
    assert err <= 1e-5
    assert np.isfinite(Hh[np.triu_indices(D)]).all()
    del X, H
    torch.cuda.empty_cache()


def test_full_apply_full_config_sampled_rows():
    """y = M x with unit norm over 10^6 x 8192 rows (fp16 out); 24 rows, the
    first and last included, against the fp64 oracle."""
    n = 1_000_000
    say(f"case: full apply full size n={n} D={D}")
    X = _lowrank_store(n, seed=5)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(11)
    B = torch.randn((D, D), generator=gen, device="cuda") / D ** 0.5
    M = (B @ B.T + torch.eye(D, device="cuda")).contiguous()
    del B
    Y = torch.empty_like(X)
    P.attr_precond_apply(X, P.PRECOND_FULL, M, True, Y)
    torch.cuda.synchronize()
    rows = np.r_[0, np.sort(np.random.default_rng(8).choice(n, 22, replace=False)), n - 1]
    ridx = torch.from_numpy(rows).cuda()
    ref = O.precond_apply(host(X[ridx]), "full", host(M).astype(np.float64), unit_norm=True)
    err = row_rel_l2(host(Y[ridx]), ref)
    say("sampled rows max rel-L2", err.max())
    assert err.max() <= 2e-3
    del X, Y, M
    torch.cuda.empty_cache()


def _check_scan(G, Q, ts, ti, qs, k, n_sample, tol=1e-3):
    """For queries qs: returned scores equal fp64 recomputations, are sorted
    and unique, and no row of a random sample that was not returned scores
    above the k-th + tol."""
    n = G.shape[0]
    sample_idx = np.random.default_rng(9).choice(n, n_sample, replace=False)
    Gs = host(G[torch.from_numpy(sample_idx).cuda()]).astype(np.float64)
    for q in qs:
        idx = host(ti[q])
        assert (idx >= 0).all() and len(set(idx.tolist())) == k
        s = host(ts[q]).astype(np.float64)
        assert (np.diff(s) <= 0).all()
        qv = host(Q[q]).astype(np.float64)
        rec = host(G[torch.from_numpy(idx).cuda()]).astype(np.float64) @ qv
        assert np.abs(rec - s).max() <= tol, (q, np.abs(rec - s).max())
        others = ~np.isin(sample_idx, idx)           # sampled rows not returned
        assert (Gs[others] @ qv).max() <= s[-1] + tol, q


@pytest.mark.parametrize("nq", [1024, 16, 64])
def test_store_scan_full_config(nq):
    """4M x 8192 unit fp16 store (65.5 GB), top-100: Q = 1024 runs the GEMM
    plan, Q = 16 and 64 the streaming plan (with its prefix bound).  16 planted near-duplicates (cosine 0.9)
    of known rows must rank first; sampled queries pass _check_scan."""
    n, k = 4_000_000, 100
    say(f"case: store scan full size n={n} nq={nq} k={k}")
    G = _unit_store(n, seed=21)
    targets = np.random.default_rng(4).choice(n, 16, replace=False)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(22)
    q = torch.randn((nq, D), generator=gen, device="cuda")
    q = q / q.norm(dim=1, keepdim=True)
    g = G[torch.from_numpy(targets).cuda()].float()
    g = g / g.norm(dim=1, keepdim=True)
    u = q[:16] - (q[:16] * g).sum(1, keepdim=True) * g
    u = u / u.norm(dim=1, keepdim=True)
    q[:16] = 0.9 * g + (1 - 0.81) ** 0.5 * u
    Q = q.half().contiguous()
    ts = torch.empty((nq, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((nq, k), dtype=torch.int64, device="cuda")
    P.attr_score_topk(Q, G, k, ts, ti)
    torch.cuda.synchronize()
    assert (host(ti)[:16, 0] == targets).all()
    assert np.abs(host(ts)[:16, 0] - 0.9).max() <= 2e-3
    _check_scan(G, Q, ts, ti, [0, 5, nq // 2, nq - 1], k, 200_000)
    del G
    torch.cuda.empty_cache()
