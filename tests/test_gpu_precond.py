"""GPU parity of attr_precond_apply / attr_precond_accumulate against the oracle."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_11660_amd as P
import synth
from tests._util import dev, host, row_rel_l2, say

pytestmark = pytest.mark.gpu


def _f16_ulp_close(got16, ref64, ulps=1.0):
    """|got - ref| <= ulps * ulp_f16(ref) + tiny, elementwise (ref rounded once)."""
    ref = np.asarray(ref64, dtype=np.float64)
    spacing = np.spacing(np.abs(ref).astype(np.float16)).astype(np.float64)
    return np.abs(got16.astype(np.float64) - ref) <= ulps * spacing + 1e-12


@pytest.mark.parametrize("D", [256, 12288, 28672, 40000])
def test_unit_normalise_fp32_to_fp16(D):
    say(f"case: apply NONE+unit fp32->fp16 D={D}")
    rng = np.random.default_rng(D)
    X = (rng.standard_normal((37, D)) * rng.uniform(0.01, 100, size=(37, 1))).astype(np.float32)
    X[5] = 0.0
    Y = torch.empty((37, D), dtype=torch.float16, device="cuda")
    P.attr_precond_apply(dev(X), P.PRECOND_NONE, None, True, Y)
    torch.cuda.synchronize()
    got = host(Y)
    ref = O.precond_apply(X, "none", None, unit_norm=True)
    assert (got[5] == 0).all()
    assert _f16_ulp_close(got, ref, 1.0).all()
    err = row_rel_l2(got, ref)
    say("max row rel-L2", err.max())
    assert err.max() <= 2e-2


def test_diag_apply_fp16_inplace_and_fp32_out():
    say("case: apply DIAG+unit fp16 in place, and fp16->fp32")
    D = 8192
    rng = np.random.default_rng(3)
    X = (rng.standard_normal((64, D)) * 3).astype(np.float16)
    m = rng.uniform(0.1, 10, size=D).astype(np.float32)
    m[7] = 0.0
    Xd = dev(X)
    Y32 = torch.empty((64, D), dtype=torch.float32, device="cuda")
    P.attr_precond_apply(Xd, P.PRECOND_DIAG, dev(m), True, Y32)
    P.attr_precond_apply(Xd, P.PRECOND_DIAG, dev(m), True, Xd)        # in place
    torch.cuda.synchronize()
    ref = O.precond_apply(X, "diag", m, unit_norm=True)
    err32 = row_rel_l2(host(Y32), ref)
    say("fp32 out max row rel-L2", err32.max())
    assert err32.max() <= 1e-5
    assert _f16_ulp_close(host(Xd), ref, 1.0).all()
    # no normalisation: plain scaling
    Y2 = torch.empty((64, D), dtype=torch.float32, device="cuda")
    P.attr_precond_apply(dev(X), P.PRECOND_DIAG, dev(m), False, Y2)
    torch.cuda.synchronize()
    np.testing.assert_allclose(host(Y2), O.precond_apply(X, "diag", m, unit_norm=False), rtol=1e-6)


@pytest.mark.parametrize("D", [8192, 1000])
def test_diag_apply_many_rows(D):
    """4500 rows take the row-walk kernel (1024 workgroups, 4 or 5 rows each,
    next row prefetched): fp16 in place, fp16 -> fp32, unnormalised; a
    zero row and a zero scale column."""
    say(f"case: apply DIAG many rows D={D}")
    n = 4500
    rng = np.random.default_rng(D + 1)
    X = (rng.standard_normal((n, D)) * rng.uniform(0.1, 5, size=(n, 1))).astype(np.float16)
    X[4499] = 0
    m = rng.uniform(0.1, 10, size=D).astype(np.float32)
    m[3] = 0.0
    Xd, md = dev(X), dev(m)
    Y32 = torch.empty((n, D), dtype=torch.float32, device="cuda")
    Yu = torch.empty((n, D), dtype=torch.float32, device="cuda")
    P.attr_precond_apply(Xd, P.PRECOND_DIAG, md, True, Y32)
    P.attr_precond_apply(Xd, P.PRECOND_DIAG, md, False, Yu)
    P.attr_precond_apply(Xd, P.PRECOND_DIAG, md, True, Xd)          # in place, last
    torch.cuda.synchronize()
    ref = O.precond_apply(X, "diag", m, unit_norm=True)
    err32 = row_rel_l2(host(Y32), ref)
    say("fp32 out max row rel-L2", err32.max())
    assert err32.max() <= 1e-5
    assert (host(Y32)[4499] == 0).all() and (host(Xd)[4499] == 0).all()
    assert _f16_ulp_close(host(Xd), ref, 1.0).all()
    np.testing.assert_allclose(host(Yu), O.precond_apply(X, "diag", m, unit_norm=False), rtol=1e-6)


@pytest.mark.parametrize("dtype", ["f16", "f32"])
def test_diag_accumulate(dtype):
    say(f"case: accumulate DIAG {dtype}")
    n, D = 5003, 8192
    X = synth.lowrank_rows(0, n, D=D, rank=16, chunk=4096)
    if dtype == "f32":
        X = X.astype(np.float32)
    H = torch.zeros(D, dtype=torch.float32, device="cuda")
    Xd = dev(X)
    P.attr_precond_accumulate(Xd[:3000], P.PRECOND_DIAG, H)
    P.attr_precond_accumulate(Xd[3000:], P.PRECOND_DIAG, H)     # additive across calls
    torch.cuda.synchronize()
    ref = O.accumulate_diag(X)
    rel = np.abs(host(H) - ref) / ref
    say("max rel err", rel.max())
    assert rel.max() <= 1e-6
