"""The Python binding rejects tensors that do not match the sizes it would
pass to the library (which sees only pointers), before any library call.
CPU tensors suffice: every check here runs before the device check."""
import pytest
import torch

import paper_2606_11660_amd as P


def _mods(n=2, T=4, d_in=64, d_out=128, k=16, dtype=torch.bfloat16):
    a = torch.zeros((n * T, d_in), dtype=dtype)
    g = torch.zeros((n * T, d_out), dtype=dtype)
    R = torch.zeros((d_out, k), dtype=dtype)
    S = torch.zeros((d_in, k), dtype=dtype)
    return [P.Module(a, g, R, S, 0)]


def _out(n=2, w=256):
    return torch.zeros((n, w), dtype=torch.float32)


def test_project_valid_call_stops_at_the_device_check():
    with pytest.raises(ValueError, match="same GPU"):
        P.attr_project(_mods(), 16, 2, 4, _out())


def test_project_too_few_output_rows():
    with pytest.raises(ValueError, match="rows, the call writes"):
        P.attr_project(_mods(), 16, 3, 4, _out(n=2))


def test_project_output_too_narrow():
    with pytest.raises(ValueError, match="exceed out's width"):
        P.attr_project(_mods(), 16, 2, 4, _out(w=255))
    m = _mods()
    m[0].out_col = 16
    with pytest.raises(ValueError, match="exceed out's width"):
        P.attr_project(m, 16, 2, 4, _out())


def test_project_too_few_token_rows():
    with pytest.raises(ValueError, match="need 12"):
        P.attr_project(_mods(n=2, T=4), 16, 3, 4, _out(n=3))


def test_project_mixed_dtypes():
    m = _mods()
    m[0].R = m[0].R.float()
    with pytest.raises(ValueError, match="R is torch.float32"):
        P.attr_project(m, 16, 2, 4, _out())
    m = _mods() + _mods(dtype=torch.float32)
    m[1].out_col = 256
    with pytest.raises(ValueError, match="module 1: a is torch.float32"):
        P.attr_project(m, 16, 2, 4, _out(w=512))


def test_project_projection_shapes():
    m = _mods()
    m[0].R = torch.zeros((64, 16), dtype=torch.bfloat16)      # [d_in, k] instead of [d_out, k]
    with pytest.raises(ValueError, match="R must be"):
        P.attr_project(m, 16, 2, 4, _out())
    with pytest.raises(ValueError, match="R must be"):
        P.attr_project(_mods(), 32, 2, 4, _out(w=1024))       # k disagrees with R and S


def test_project_offsets_and_lengths():
    with pytest.raises(ValueError, match="row_offset"):
        P.attr_project(_mods(), 16, 2, 4, _out(), row_offset=torch.zeros(1, dtype=torch.int64))
    with pytest.raises(ValueError, match="row_offset"):
        P.attr_project(_mods(), 16, 2, 4, _out(), row_offset=torch.zeros(2, dtype=torch.int32))
    with pytest.raises(ValueError, match="length"):
        P.attr_project(_mods(), 16, 2, 4, _out(), length=torch.zeros(2, dtype=torch.int64))


def test_project_tokens_checks_modules_too():
    m = _mods()
    m[0].S = torch.zeros((64, 8), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="S "):
        P.attr_project_tokens(m, 16, 2, 4, torch.zeros((8, 256)))


def test_accumulate_shapes():
    X = torch.zeros((10, 64), dtype=torch.float16)
    with pytest.raises(ValueError, match=r"shape \[64\]"):
        P.attr_precond_accumulate(X, P.PRECOND_DIAG, torch.zeros(63))
    with pytest.raises(ValueError, match=r"shape \[64, 64\]"):
        P.attr_precond_accumulate(X, P.PRECOND_FULL, torch.zeros(64))
    with pytest.raises(ValueError, match=r"shape \[64, 64\]"):
        P.attr_precond_accumulate(X, P.PRECOND_FULL, torch.zeros((64, 64), dtype=torch.float64))
    with pytest.raises(ValueError, match="DIAG or PRECOND_FULL"):
        P.attr_precond_accumulate(X, P.PRECOND_NONE, torch.zeros(64))


def test_apply_shapes():
    X = torch.zeros((10, 64), dtype=torch.float16)
    Y = torch.zeros((10, 64), dtype=torch.float16)
    with pytest.raises(ValueError, match=r"shape \[64\]"):
        P.attr_precond_apply(X, P.PRECOND_DIAG, torch.zeros((64, 64)), True, Y)
    with pytest.raises(ValueError, match=r"shape \[64, 64\]"):
        P.attr_precond_apply(X, P.PRECOND_FULL, torch.zeros(64), True, Y)
    with pytest.raises(ValueError, match="must be None"):
        P.attr_precond_apply(X, P.PRECOND_NONE, torch.zeros(64), True, Y)
    with pytest.raises(ValueError, match="shapes differ"):
        P.attr_precond_apply(X, P.PRECOND_NONE, None, True, Y[:9])


def test_score_output_shapes():
    Q = torch.zeros((4, 64), dtype=torch.float16)
    G = torch.zeros((100, 64), dtype=torch.float16)
    ts, ti = torch.zeros((4, 5)), torch.zeros((4, 5), dtype=torch.int64)
    with pytest.raises(ValueError, match=r"must be \[4, 6\]"):
        P.attr_score_topk(Q, G, 6, ts, ti)
    with pytest.raises(ValueError, match=r"must be \[4, 5\]"):
        P.attr_score_topk(Q, G, 5, ts, ti[:3])
    with pytest.raises(ValueError, match="same GPU"):
        P.attr_score_topk(Q, G, 5, ts, ti)


def test_finalize_lives_outside_the_binding():
    # the host eigendecomposition is its own module, not part of the marshalling layer
    assert not hasattr(P, "finalize_full") and not hasattr(P, "finalize_diag")
    from paper_2606_11660_amd import finalize as F
    import numpy as np
    H = torch.tensor([[4.0, 0.0], [0.0, 1.0]])
    M = F.finalize_full(H, 1)
    np.testing.assert_allclose(M.numpy(), [[0.5, 0.0], [0.0, 1.0]], rtol=1e-7)
    m = F.finalize_diag(torch.tensor([4.0, 0.0, 9.0]), 1)
    np.testing.assert_allclose(m.numpy(), [0.5, 0.0, 1.0 / 3.0], rtol=1e-7)
    with pytest.raises(ValueError):
        F.finalize_full(torch.zeros(3), 1)
