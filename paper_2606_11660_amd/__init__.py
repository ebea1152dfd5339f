"""Python binding of libattr, the MI355X gradient-attribution hot path.

Thin ctypes marshalling over the C ABI declared in ``include/attr.h``: the
functions below carry the same names as the C entry points, take torch
tensors that already live on the GPU, and pass their device pointers, sizes
and the current HIP stream through unchanged.  Every arithmetic step runs in
the library's HIP kernels; PyTorch only provides device memory and streams.
The library must have been built (``python -m paper_2606_11660_amd.build``);
importing this package without it raises, there is no fallback path.

Every wrapper checks the tensors it is given against the sizes it passes
(shapes, dtypes, devices) and raises ``ValueError`` before calling the
library, which sees only pointers.  The one host step of the method, turning
the accumulated second moment into H^{-1/2}, lives in ``finalize``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Iterable, List, Optional, Sequence, Tuple

import torch

__all__ = [
    "AttrError", "ATTR_F32", "ATTR_BF16", "ATTR_F16", "PRECOND_NONE", "PRECOND_DIAG",
    "PRECOND_FULL", "Module", "lib", "lib_path", "attr_project", "attr_project_noalloc",
    "attr_project_tokens",
    "attr_precond_accumulate",
    "attr_precond_apply", "attr_score_topk", "attr_project_workspace_size",
    "attr_precond_accumulate_workspace_size", "attr_precond_apply_workspace_size",
    "attr_score_topk_workspace_size", "Workspace", "attr_probe_read", "attr_probe_mfma",
]

_PKG = os.path.dirname(os.path.abspath(__file__))
# ATTR_LIBRARY selects another build of the same library (the host-sanitizer
# build of the CPU tests); by default the in-tree libattr.so.
_LIB_PATH = os.environ.get("ATTR_LIBRARY") or os.path.join(_PKG, "libattr.so")

ATTR_F32, ATTR_BF16, ATTR_F16 = 0, 1, 2
PRECOND_NONE, PRECOND_DIAG, PRECOND_FULL = 0, 1, 2
_STATUS = {0: "ATTR_OK", 1: "ATTR_ERR_INVALID_ARG", 2: "ATTR_ERR_UNSUPPORTED",
           3: "ATTR_ERR_ALIGNMENT", 4: "ATTR_ERR_WORKSPACE", 5: "ATTR_ERR_DEVICE"}
_TORCH_DTYPE = {torch.float32: ATTR_F32, torch.bfloat16: ATTR_BF16, torch.float16: ATTR_F16}


class AttrError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{_STATUS.get(status, status)}: {message}")
        self.status = status
        self.message = message


class _CModule(ctypes.Structure):
    _fields_ = [("a", ctypes.c_void_p), ("g", ctypes.c_void_p), ("R", ctypes.c_void_p),
                ("S", ctypes.c_void_p), ("lda", ctypes.c_int64), ("ldg", ctypes.c_int64),
                ("d_in", ctypes.c_int64), ("d_out", ctypes.c_int64), ("out_col", ctypes.c_int64),
                ("v_out", ctypes.c_void_p), ("v_in", ctypes.c_void_p)]


_lib = None


def lib_path() -> str:
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    """Load libattr.so (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2606_11660_amd.build`")
    L = ctypes.CDLL(_LIB_PATH)
    i64, i32, vp, sz = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t
    L.attr_last_error.restype = ctypes.c_char_p
    L.attr_status_string.restype = ctypes.c_char_p
    L.attr_status_string.argtypes = [ctypes.c_int]
    L.attr_abi_version.restype = ctypes.c_int
    L.attr_project_workspace_size.restype = sz
    L.attr_project_workspace_size.argtypes = [ctypes.POINTER(_CModule), i32, ctypes.c_int, i64, i64, i32]
    L.attr_project.restype = ctypes.c_int
    L.attr_project.argtypes = [ctypes.POINTER(_CModule), i32, ctypes.c_int, i32, i64, i64, vp, vp,
                               vp, i64, vp, sz, vp]
    L.attr_project_tokens.restype = ctypes.c_int
    L.attr_project_tokens.argtypes = [ctypes.POINTER(_CModule), i32, ctypes.c_int, i32, i64, i64, vp,
                                      vp, vp, i64, i64, vp, sz, vp]
    L.attr_project_noalloc.restype = ctypes.c_int
    L.attr_project_noalloc.argtypes = [ctypes.POINTER(_CModule), i32, ctypes.c_int, i32, i64, i64,
                                       vp, vp, vp, i64, vp]
    L.attr_precond_accumulate_workspace_size.restype = sz
    L.attr_precond_accumulate_workspace_size.argtypes = [i64, i64, ctypes.c_int, ctypes.c_int]
    L.attr_precond_accumulate.restype = ctypes.c_int
    L.attr_precond_accumulate.argtypes = [vp, ctypes.c_int, i64, i64, i64, ctypes.c_int, vp, vp, sz, vp]
    L.attr_precond_apply_workspace_size.restype = sz
    L.attr_precond_apply_workspace_size.argtypes = [i64, i64, ctypes.c_int]
    L.attr_precond_apply.restype = ctypes.c_int
    L.attr_precond_apply.argtypes = [vp, ctypes.c_int, i64, i64, i64, ctypes.c_int, vp, i32, vp,
                                     ctypes.c_int, i64, vp, sz, vp]
    L.attr_probe_read.restype = ctypes.c_int
    L.attr_probe_read.argtypes = [vp, sz, vp, vp]
    L.attr_probe_mfma.restype = ctypes.c_int
    L.attr_probe_mfma.argtypes = [i64, vp, vp]
    L.attr_score_topk_workspace_size.restype = sz
    L.attr_score_topk_workspace_size.argtypes = [i64, i64, i64, i32]
    L.attr_score_topk.restype = ctypes.c_int
    L.attr_score_topk.argtypes = [vp, i64, i64, vp, i64, i64, ctypes.c_int, i64, i32, i64, i32, vp,
                                  vp, vp, sz, vp]
    _lib = L
    return L


def _check(status: int) -> None:
    if status != 0:
        raise AttrError(status, lib().attr_last_error().decode(errors="replace"))


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dtype(t: torch.Tensor) -> int:
    if t.dtype not in _TORCH_DTYPE:
        raise TypeError(f"unsupported dtype {t.dtype}")
    return _TORCH_DTYPE[t.dtype]


def _rows(t: torch.Tensor) -> Tuple[int, int, int]:
    """(rows, width, row stride) of a tensor whose last dim is contiguous."""
    if t.dim() < 2 or t.stride(-1) != 1:
        raise ValueError("expected a tensor with a contiguous last dimension")
    width, ld = t.shape[-1], t.stride(-2)
    rows = 1
    for d in range(t.dim() - 1):
        rows *= t.shape[d]
    for d in range(t.dim() - 2):
        if t.stride(d) != t.stride(d + 1) * t.shape[d + 1]:
            raise ValueError("leading dimensions must be packed")
    return rows, width, ld


def _same_gpu(*tensors: Optional[torch.Tensor]) -> None:
    """Every given tensor lives on one GPU (the library takes raw pointers)."""
    ts = [t for t in tensors if t is not None]
    if not ts:
        return
    d = ts[0].device
    for t in ts:
        if t.device.type != "cuda" or t.device != d:
            raise ValueError("every tensor must live on the same GPU device")


def _vector(t: Optional[torch.Tensor], n: int, dtype, name: str) -> None:
    """t is None or a contiguous `dtype` tensor with at least n elements."""
    if t is None:
        return
    if t.dtype != dtype or not t.is_contiguous() or t.numel() < n:
        raise ValueError(f"{name} must be a contiguous {dtype} tensor of at least {n} elements")


def _torch_stream(stream):
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream))


class Workspace:
    """Grow-only device scratch buffer handed to the library calls.

    A workspace serves one stream at a time: calls that may overlap on
    different streams need workspaces of their own (the default workspace is
    kept per device and stream).  Every use records its stream on the
    buffer, so a buffer replaced by a larger one is not handed out again by
    torch's allocator before the work queued on those streams has finished.
    """

    def __init__(self, device=None):
        self.device = torch.device(device or "cuda")
        self.buf: Optional[torch.Tensor] = None

    def get(self, nbytes: int, stream=None) -> Tuple[Optional[int], int]:
        if nbytes == 0:
            return None, 0
        if self.buf is None or self.buf.numel() < nbytes:
            self.buf = torch.empty(int(nbytes), dtype=torch.uint8, device=self.device)
        self.buf.record_stream(_torch_stream(stream))
        return self.buf.data_ptr(), self.buf.numel()


_default_ws: Dict[Tuple[str, int], Workspace] = {}


def _ws(ws: Optional[Workspace], device, stream=None) -> Workspace:
    if ws is not None:
        return ws
    key = (str(device), _stream(stream))
    if key not in _default_ws:
        _default_ws[key] = Workspace(device)
    return _default_ws[key]


# ----------------------------------------------------------------------------
# (1) projection
# ----------------------------------------------------------------------------
class Module:
    """One linear module's inputs for ``attr_project``.

    a: [..., d_in] activations, g: [..., d_out] output gradients (token rows,
    last dim contiguous); R: [d_out, k], S: [d_in, k] contiguous, same dtype
    as a and g; out_col: first column of the module's k*k block in the output
    row.  v_out [d_out] and v_in [d_in] (fp32, optional, both or neither): the
    factored (Adafactor) second moment that normalises the gradient before
    projection.
    """

    def __init__(self, a: torch.Tensor, g: torch.Tensor, R: torch.Tensor, S: torch.Tensor,
                 out_col: int, v_out: Optional[torch.Tensor] = None,
                 v_in: Optional[torch.Tensor] = None):
        self.a, self.g, self.R, self.S, self.out_col = a, g, R, S, int(out_col)
        self.v_out, self.v_in = v_out, v_in

    def tensors(self):
        return (self.a, self.g, self.R, self.S, self.v_out, self.v_in)

    def c(self) -> _CModule:
        _, d_in, lda = _rows(self.a)
        _, d_out, ldg = _rows(self.g)
        if not (self.R.is_contiguous() and self.S.is_contiguous()):
            raise ValueError("R and S must be contiguous")
        for v, n, name in ((self.v_out, d_out, "v_out"), (self.v_in, d_in, "v_in")):
            if v is not None and (v.dtype != torch.float32 or not v.is_contiguous() or v.numel() != n):
                raise ValueError(f"{name} must be a contiguous fp32 vector of {n} elements")
        return _CModule(self.a.data_ptr(), self.g.data_ptr(), self.R.data_ptr(), self.S.data_ptr(),
                        lda, ldg, d_in, d_out, self.out_col, _ptr(self.v_out), _ptr(self.v_in))


def _cmods(mods: Sequence[Module]):
    arr = (_CModule * len(mods))(*[m.c() for m in mods])
    return arr


def _check_modules(mods: Sequence[Module], k: int, n_examples: int, T: int,
                   row_offset: Optional[torch.Tensor], length: Optional[torch.Tensor],
                   out: torch.Tensor, out_rows_needed: int) -> int:
    """Validate a projection call's tensors against its sizes; returns the
    input dtype code."""
    if not mods:
        raise ValueError("need at least one module")
    dt = mods[0].a.dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise ValueError("token rows must be fp32 or bf16")
    if out.dtype != torch.float32 or out.dim() != 2 or out.stride(1) != 1:
        raise ValueError("out must be fp32 [rows, ldo] with contiguous rows")
    if out.shape[0] < out_rows_needed:
        raise ValueError(f"out has {out.shape[0]} rows, the call writes {out_rows_needed}")
    if n_examples < 0 or T < 1:
        raise ValueError("n_examples must be >= 0 and T >= 1")
    _vector(row_offset, n_examples, torch.int64, "row_offset")
    _vector(length, n_examples, torch.int32, "length")
    for j, m in enumerate(mods):
        for name, t in (("a", m.a), ("g", m.g), ("R", m.R), ("S", m.S)):
            if t.dtype != dt:
                raise ValueError(f"module {j}: {name} is {t.dtype}, module 0's a is {dt}")
        na, d_in, _ = _rows(m.a)
        ng, d_out, _ = _rows(m.g)
        if tuple(m.R.shape) != (d_out, k) or tuple(m.S.shape) != (d_in, k):
            raise ValueError(f"module {j}: R must be [{d_out}, {k}] and S [{d_in}, {k}]")
        if m.out_col < 0 or m.out_col + k * k > out.shape[1]:
            raise ValueError(f"module {j}: columns [{m.out_col}, {m.out_col + k * k}) exceed "
                             f"out's width {out.shape[1]}")
        if row_offset is None and min(na, ng) < n_examples * T:
            raise ValueError(f"module {j}: a/g hold {min(na, ng)} rows, {n_examples} examples "
                             f"of {T} tokens need {n_examples * T}")
    _same_gpu(out, row_offset, length, *[t for m in mods for t in m.tensors()])
    return _dtype(mods[0].a)


def attr_project_workspace_size(mods: Sequence[Module], in_dtype: int, n_examples: int, T: int,
                                k: int) -> int:
    return int(lib().attr_project_workspace_size(_cmods(mods), len(mods), in_dtype, n_examples, T, k))


def attr_project(mods: Sequence[Module], k: int, n_examples: int, T: int,
                 out: torch.Tensor, row_offset: Optional[torch.Tensor] = None,
                 length: Optional[torch.Tensor] = None, ws: Optional[Workspace] = None,
                 stream=None) -> torch.Tensor:
    """P_{i,m} = sum_{t < len_i} (R^T g_t)(S^T a_t)^T into out[i, out_col:out_col+k*k].

    Without row_offset, example i's tokens are rows i*T .. i*T + T - 1 of every
    a and g; with it (int64 [n_examples], device) they start at row_offset[i]
    and the caller keeps every valid token inside a and g (device values
    cannot be checked here).  length: int32 [n_examples] on the device,
    clamped to [0, T] by the library."""
    in_dtype = _check_modules(mods, k, n_examples, T, row_offset, length, out, n_examples)
    cm = _cmods(mods)
    L = lib()
    need = L.attr_project_workspace_size(cm, len(mods), in_dtype, n_examples, T, k)
    wsp, wsn = _ws(ws, out.device, stream).get(need, stream)
    _check(L.attr_project(cm, len(mods), in_dtype, k, n_examples, T, _ptr(row_offset), _ptr(length),
                          out.data_ptr(), out.stride(0), wsp, wsn, _stream(stream)))
    return out


def attr_project_noalloc(mods: Sequence[Module], k: int, n_examples: int, T: int,
                         out: torch.Tensor, row_offset: Optional[torch.Tensor] = None,
                         length: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """attr_project without a workspace: the library's static per-GPU scratch
    (ATTR_PROJECT_NOALLOC_SCRATCH bytes) serves as workspace, so this call
    allocates nothing (usable under graph capture).  Calls that overlap on one
    GPU share that scratch and must be ordered by the caller."""
    in_dtype = _check_modules(mods, k, n_examples, T, row_offset, length, out, n_examples)
    _check(lib().attr_project_noalloc(_cmods(mods), len(mods), in_dtype, k, n_examples, T,
                                      _ptr(row_offset), _ptr(length), out.data_ptr(),
                                      out.stride(0), _stream(stream)))
    return out


def attr_project_tokens(mods: Sequence[Module], k: int, n_examples: int, T: int,
                        out: torch.Tensor, row_offset: Optional[torch.Tensor] = None,
                        length: Optional[torch.Tensor] = None, ws: Optional[Workspace] = None,
                        stream=None) -> torch.Tensor:
    """Per-token blocks (R^T g_t)(S^T a_t)^T into out[token row, out_col:out_col+k*k];
    rows at or past out.shape[0] are not written."""
    in_dtype = _check_modules(mods, k, n_examples, T, row_offset, length, out, 0)
    cm = _cmods(mods)
    L = lib()
    need = L.attr_project_workspace_size(cm, len(mods), in_dtype, n_examples, T, k)
    wsp, wsn = _ws(ws, out.device, stream).get(need, stream)
    _check(L.attr_project_tokens(cm, len(mods), in_dtype, k, n_examples, T, _ptr(row_offset),
                                 _ptr(length), out.data_ptr(), out.stride(0), out.shape[0], wsp, wsn,
                                 _stream(stream)))
    return out


# ----------------------------------------------------------------------------
# (2) preconditioning
# ----------------------------------------------------------------------------
def _check_precond_matrix(t: Optional[torch.Tensor], mode: int, D: int, name: str) -> None:
    """DIAG: fp32 [D]; FULL: fp32 [D, D], contiguous."""
    if mode == PRECOND_NONE:
        if t is not None:
            raise ValueError(f"{name} must be None without a preconditioner")
        return
    want = (D,) if mode == PRECOND_DIAG else (D, D) if mode == PRECOND_FULL else None
    if want is None:
        raise ValueError(f"unknown preconditioner mode {mode}")
    if t is None or t.dtype != torch.float32 or not t.is_contiguous() or tuple(t.shape) != want:
        raise ValueError(f"{name} must be a contiguous fp32 tensor of shape {list(want)}")


def attr_precond_accumulate_workspace_size(n_rows: int, D: int, x_dtype: int, mode: int) -> int:
    return int(lib().attr_precond_accumulate_workspace_size(n_rows, D, x_dtype, mode))


def attr_precond_accumulate(X: torch.Tensor, mode: int, H: torch.Tensor,
                            ws: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """H += diag(X^T X) (DIAG, H [D]) or the upper triangle of X^T X (FULL, H [D, D])."""
    n, D, ldx = _rows(X)
    xd = _dtype(X)
    if mode not in (PRECOND_DIAG, PRECOND_FULL):
        raise ValueError("attr_precond_accumulate takes PRECOND_DIAG or PRECOND_FULL")
    _check_precond_matrix(H, mode, D, "H")
    _same_gpu(X, H)
    L = lib()
    need = L.attr_precond_accumulate_workspace_size(n, D, xd, mode)
    wsp, wsn = _ws(ws, X.device, stream).get(need, stream)
    _check(L.attr_precond_accumulate(X.data_ptr(), xd, n, D, ldx, mode, H.data_ptr(), wsp, wsn,
                                     _stream(stream)))
    return H


def attr_precond_apply_workspace_size(n_rows: int, D: int, mode: int) -> int:
    return int(lib().attr_precond_apply_workspace_size(n_rows, D, mode))


def attr_precond_apply(X: torch.Tensor, mode: int, M: Optional[torch.Tensor], unit_normalize: bool,
                       Y: torch.Tensor, ws: Optional[Workspace] = None, stream=None) -> torch.Tensor:
    """Y = unit_normalise(precondition(X)) cast to Y's dtype."""
    n, D, ldx = _rows(X)
    ny, Dy, ldy = _rows(Y)
    if (ny, Dy) != (n, D):
        raise ValueError("X and Y shapes differ")
    _check_precond_matrix(M, mode, D, "M")
    _same_gpu(X, Y, M)
    L = lib()
    need = L.attr_precond_apply_workspace_size(n, D, mode)
    wsp, wsn = _ws(ws, X.device, stream).get(need, stream)
    _check(L.attr_precond_apply(X.data_ptr(), _dtype(X), n, D, ldx, mode, _ptr(M),
                                1 if unit_normalize else 0, Y.data_ptr(), _dtype(Y), ldy, wsp, wsn,
                                _stream(stream)))
    return Y


# ----------------------------------------------------------------------------
# (3) scoring
# ----------------------------------------------------------------------------
def attr_score_topk_workspace_size(n_q: int, n_g: int, D: int, k: int) -> int:
    return int(lib().attr_score_topk_workspace_size(n_q, n_g, D, k))


def attr_score_topk(Q: torch.Tensor, G: torch.Tensor, k: int, top_score: torch.Tensor,
                    top_index: torch.Tensor, index_base: int = 0, merge: bool = False,
                    ws: Optional[Workspace] = None, stream=None) -> Tuple[torch.Tensor, torch.Tensor]:
    """Exact top-k of <Q_q, G_j> per query, merged with top_* when merge is set."""
    nq, D, ldq = _rows(Q)
    ng, Dg, ldg = _rows(G)
    if Dg != D:
        raise ValueError("Q and G widths differ")
    if Q.dtype != G.dtype:
        raise ValueError("Q and G dtypes differ")
    if top_score.dtype != torch.float32 or top_index.dtype != torch.int64:
        raise ValueError("top_score must be fp32 and top_index int64")
    if not (top_score.is_contiguous() and top_index.is_contiguous()):
        raise ValueError("top_score / top_index must be contiguous")
    if tuple(top_score.shape) != (nq, k) or tuple(top_index.shape) != (nq, k):
        raise ValueError(f"top_score and top_index must be [{nq}, {k}]")
    _same_gpu(Q, G, top_score, top_index)
    L = lib()
    need = L.attr_score_topk_workspace_size(nq, ng, D, k)
    wsp, wsn = _ws(ws, Q.device, stream).get(need, stream)
    _check(L.attr_score_topk(Q.data_ptr(), nq, ldq, G.data_ptr(), ng, ldg, _dtype(Q), D, k,
                             index_base, 1 if merge else 0, top_score.data_ptr(),
                             top_index.data_ptr(), wsp, wsn, _stream(stream)))
    return top_score, top_index


# ----------------------------------------------------------------------------
# calibration (measured peaks; not part of the method)
# ----------------------------------------------------------------------------
def attr_probe_read(x: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """One streaming read of every byte of x (HBM read-bandwidth probe)."""
    if not x.is_contiguous():
        raise ValueError("x must be contiguous")
    _same_gpu(x, sink)
    _check(lib().attr_probe_read(x.data_ptr(), x.numel() * x.element_size(), sink.data_ptr(),
                                 _stream(stream)))


def attr_probe_mfma(n_mfma: int, sink: torch.Tensor, stream=None) -> int:
    """n_mfma fp16 16x16x32 MFMAs per wave on 2048 waves; returns the flops."""
    _same_gpu(sink)
    _check(lib().attr_probe_mfma(n_mfma, sink.data_ptr(), _stream(stream)))
    return 2 * 16 * 16 * 32 * n_mfma * 2048
