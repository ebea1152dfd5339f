"""Operands whose row stride exceeds their width (views into wider buffers
whose extra columns hold NaN) on the entry points that take a stride: the
GEMM-plan and streaming-plan store scans (Q and G), the FULL accumulate
(X), the FULL and DIAG applies (X in, Y out: the padding of Y stays
untouched), the DIAG accumulate and the projection (every module's a and g
rows).  A kernel that read or wrote past a
row's width would turn results into NaN or overwrite the sentinel."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_11660_amd as P
import synth
from tests._util import check_topk, dev, host, row_rel_l2, say

pytestmark = pytest.mark.gpu


def _wide(x: np.ndarray, pad: int) -> torch.Tensor:
    """Device view of x inside a buffer pad columns wider, padding NaN."""
    n, d = x.shape
    buf = np.full((n, d + pad), np.nan, dtype=x.dtype)
    buf[:, :d] = x
    return dev(buf)[:, :d]


def _wide_any(x: np.ndarray, pad: int) -> torch.Tensor:
    """_wide for fp32 arrays and for bf16 bit patterns (uint16: NaN 0x7fc0)."""
    if x.dtype == np.uint16:
        n, d = x.shape
        buf = np.full((n, d + pad), 0x7FC0, dtype=np.uint16)
        buf[:, :d] = x
        return dev(buf)[:, :d]
    return _wide(x, pad)


def _topk(Q, G, k):
    ts = torch.full((Q.shape[0], k), 5.0, dtype=torch.float32, device="cuda")
    ti = torch.full((Q.shape[0], k), 7, dtype=torch.int64, device="cuda")
    P.attr_score_topk(Q, G, k, ts, ti)
    torch.cuda.synchronize()
    return host(ts), host(ti)


@pytest.mark.parametrize("nq,ng,D,k,qpad,gpad,dt", [(300, 9000, 256, 10, 64, 192, np.float16),
                                                    (128, 5000, 192, 20, 8, 72, np.float16),
                                                    (40, 9000, 256, 10, 64, 128, np.float16),
                                                    (40, 9000, 96, 10, 4, 36, np.float32)])
def test_scan_strided(nq, ng, D, k, qpad, gpad, dt):
    """GEMM plan (300 queries: 256 x 256 tiles; 128: the ring) and the
    streaming plan (40 queries, fp16 and fp32) on strided Q and G."""
    say(f"case: strided scan nq={nq} ng={ng} D={D} k={k} pads {qpad},{gpad} {dt.__name__}")
    Q = synth.unit_rows(nq, D, seed=51, dtype=dt)
    G = synth.unit_rows(ng, D, seed=52, dtype=dt)
    Qd, Gd = _wide(Q, qpad), _wide(G, gpad)
    assert Qd.stride(0) == D + qpad and Gd.stride(0) == D + gpad
    ts, ti = _topk(Qd, Gd, k)
    check_topk(ts, ti, O.scores(Q, G), k)


@pytest.mark.parametrize("n,D,pad,bf16", [(5000, 320, 64, False), (700, 256, 8, False),
                                          (3000, 320, 32, True)])
def test_full_accumulate_strided(n, D, pad, bf16):
    """X with row stride D + pad (a ragged last column tile at D = 320), fp16
    and bf16."""
    say(f"case: strided syrk n={n} D={D} pad={pad} bf16={bf16}")
    Xf = np.random.default_rng(n).standard_normal((n, D)) * 2
    X = synth.to_bf16_bits(Xf) if bf16 else Xf.astype(np.float16)
    H = torch.zeros((D, D), dtype=torch.float32, device="cuda")
    P.attr_precond_accumulate(_wide_any(X, pad), P.PRECOND_FULL, H)
    torch.cuda.synchronize()
    ref = O.accumulate_full(X)
    iu = np.triu_indices(D)
    got = host(H)
    err = np.abs(got[iu] - ref[iu]).max() / np.abs(ref).max()
    say("max rel err", err)
    assert np.isfinite(got[iu]).all() and err <= 1e-5


@pytest.mark.parametrize("mode", ["full", "diag"])
def test_apply_strided(mode):
    """X in and Y out both strided; Y's padding keeps its sentinel."""
    n, D, xpad, ypad = 777, 320, 64, 128
    say(f"case: strided apply {mode} n={n} D={D}")
    rng = np.random.default_rng(8)
    X = (rng.standard_normal((n, D)) * 3).astype(np.float16)
    if mode == "full":
        B = rng.standard_normal((D, D)) / np.sqrt(D)
        M = (B @ B.T + 0.5 * np.eye(D)).astype(np.float32)
    else:
        M = (rng.random(D) + 0.5).astype(np.float32)
    Ybuf = torch.full((n, D + ypad), 12345.0, dtype=torch.float32, device="cuda")
    Y = Ybuf[:, :D]
    P.attr_precond_apply(_wide(X, xpad), P.PRECOND_FULL if mode == "full" else P.PRECOND_DIAG,
                         dev(M), True, Y)
    torch.cuda.synchronize()
    ref = O.precond_apply(X, mode, M.astype(np.float64), unit_norm=True)
    err = row_rel_l2(host(Y), ref)
    say("max row rel-L2", err.max())
    assert err.max() <= 1e-5
    assert (host(Ybuf)[:, D:] == 12345.0).all(), "padding of Y was written"


def test_diag_accumulate_strided():
    n, D, pad = 3001, 512, 64
    say(f"case: strided diag accumulate n={n} D={D}")
    X = (np.random.default_rng(9).standard_normal((n, D))).astype(np.float16)
    h = torch.zeros(D, dtype=torch.float32, device="cuda")
    P.attr_precond_accumulate(_wide(X, pad), P.PRECOND_DIAG, h)
    torch.cuda.synchronize()
    ref = O.accumulate_diag(X)
    rel = np.abs(host(h) - ref) / ref
    say("max rel err", rel.max())
    assert rel.max() <= 1e-6


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_project_strided(dtype):
    """Projection with every module's a and g rows as views of wider buffers
    (NaN in the extra columns), two 256-token chunks per example."""
    n, T, k = 5, 300, 16
    shapes = [(64, 192), (128, 64)]
    say(f"case: strided projection {dtype} n={n} T={T} k={k}")
    rng = np.random.default_rng(77)
    cast = synth.to_bf16_bits if dtype == "bf16" else (lambda v: v.astype(np.float32))
    host_mods, mods = [], []
    for m, (d_in, d_out) in enumerate(shapes):
        a = cast(rng.standard_normal((n * T, d_in)))
        g = cast(rng.standard_normal((n * T, d_out)) * 1e-2)
        R = cast(rng.standard_normal((d_out, k)) / np.sqrt(k))
        S = cast(rng.standard_normal((d_in, k)) / np.sqrt(k))
        host_mods.append((a, g, R, S))
        mods.append(P.Module(_wide_any(a, 64), _wide_any(g, 32), dev(R), dev(S), out_col=m * k * k))
    D = len(shapes) * k * k
    out = torch.full((n, D), -7.0, dtype=torch.float32, device="cuda")
    P.attr_project(mods, k, n, T, out)
    torch.cuda.synchronize()
    ref = O.project_concat([O.project(a.reshape(n, T, -1), g.reshape(n, T, -1), R, S)
                            for (a, g, R, S) in host_mods])
    got = host(out)
    err = row_rel_l2(got, ref)
    say("max row rel-L2", err.max())
    assert np.isfinite(got).all()
    assert err.max() <= (1e-4 if dtype == "bf16" else 1e-5)
