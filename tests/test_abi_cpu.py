"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function declared in include/attr.h and
reject bad arguments on the host with the documented status before any
device work is enqueued.  Only calls that fail validation are made here, so
no kernel is ever launched.
"""
import ctypes
import os
import re

import pytest

import paper_2606_11660_amd as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

OK, INVALID, UNSUPPORTED, ALIGN, WORKSPACE, DEVICE = 0, 1, 2, 3, 4, 5
FAKE = 1 << 40          # 16-byte aligned fake device address, never dereferenced


@pytest.fixture(scope="module")
def L():
    return P.lib()


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "attr.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"\b(attr_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_exports_every_declared_symbol(L):
    names = _declared_functions()
    assert len(names) >= 11
    for n in names:
        assert hasattr(L, n), n


def test_version_and_status_strings(L):
    assert L.attr_abi_version() == 3
    assert L.attr_status_string(0) == b"ATTR_OK"
    assert L.attr_status_string(4) == b"ATTR_ERR_WORKSPACE"
    assert L.attr_last_error() == b""


def _mod(d_in=64, d_out=64, lda=None, ldg=None, out_col=0, a=FAKE, g=FAKE, R=FAKE, S=FAKE,
         v_out=None, v_in=None):
    return P._CModule(a, g, R, S, lda or d_in, ldg or d_out, d_in, d_out, out_col, v_out, v_in)


def _project(L, mods, dtype=P.ATTR_BF16, k=16, n=4, T=32, out=FAKE, ldo=256, ws=None, wsb=0):
    arr = (P._CModule * len(mods))(*mods)
    return L.attr_project(arr, len(mods), dtype, k, n, T, None, None, out, ldo, ws, wsb, None)


def test_project_validation(L):
    assert _project(L, [_mod()], k=24) == UNSUPPORTED
    assert _project(L, [_mod()], dtype=P.ATTR_F16) == UNSUPPORTED
    assert b"in_dtype" in L.attr_last_error()
    assert _project(L, [_mod(d_in=96)]) == ALIGN                   # not a multiple of 64 (bf16)
    assert _project(L, [_mod(d_in=96)], dtype=P.ATTR_F32) != ALIGN   # fine for fp32 (32)
    assert _project(L, [_mod(d_in=48)], dtype=P.ATTR_F32) == ALIGN
    assert _project(L, [_mod(a=0)]) == INVALID
    assert _project(L, [_mod(a=FAKE + 2)]) == ALIGN
    assert _project(L, [_mod(lda=32)]) == INVALID
    assert _project(L, [_mod(lda=68)]) == ALIGN
    assert _project(L, [_mod(out_col=1)]) == INVALID               # 1 + 256 > ldo
    assert _project(L, [_mod(), _mod(out_col=128)], ldo=512) == INVALID   # overlapping blocks
    assert _project(L, [_mod()], n=-1) == INVALID
    assert _project(L, [_mod()], T=0) == INVALID
    assert _project(L, [_mod()], out=0) == INVALID
    assert _project(L, [_mod()], ldo=100) == INVALID
    assert _project(L, [_mod(v_out=FAKE)]) == INVALID                # normalisation factors: both or neither
    assert _project(L, [_mod(v_in=FAKE)]) == INVALID
    assert _project(L, [_mod(v_out=FAKE + 2, v_in=FAKE)]) == ALIGN
    # all arguments valid, no workspace: rejected before any launch
    assert _project(L, [_mod()], ws=None, wsb=0) == WORKSPACE
    need = L.attr_project_workspace_size((P._CModule * 1)(_mod()), 1, P.ATTR_BF16, 4, 32, 16)
    assert need > 0
    assert _project(L, [_mod()], ws=FAKE, wsb=need - 1) == WORKSPACE
    assert _project(L, [_mod()], ws=FAKE + 16, wsb=need) == ALIGN   # workspace not 256-aligned
    # zero examples: valid no-op that touches nothing
    assert _project(L, [_mod()], n=0) == OK
    # per-token variant: same checks, plus the output row count
    tok = lambda n_rows, out=FAKE: L.attr_project_tokens((P._CModule * 1)(_mod()), 1, P.ATTR_BF16, 16,
                                                          4, 32, None, None, out, 256, n_rows, None, 0, None)
    assert tok(-1) == INVALID
    assert tok(128, out=0) == INVALID
    assert tok(128) == WORKSPACE


def test_project_workspace_size_grows_with_batch(L):
    mods = (P._CModule * 2)(_mod(768, 2304), _mod(3072, 768, out_col=256))
    s1 = L.attr_project_workspace_size(mods, 2, P.ATTR_BF16, 8, 512, 16)
    s2 = L.attr_project_workspace_size(mods, 2, P.ATTR_BF16, 16, 512, 16)
    assert 0 < s1 < s2
    assert L.attr_project_workspace_size(mods, 2, P.ATTR_BF16, 8, 512, 24) == 0


def test_accumulate_and_apply_validation(L):
    acc = L.attr_precond_accumulate
    H = FAKE + (1 << 30)
    assert acc(FAKE, P.ATTR_F16, 10, 64, 64, 7, H, None, 0, None) == UNSUPPORTED
    assert acc(FAKE, P.ATTR_F16, -1, 64, 64, P.PRECOND_DIAG, H, None, 0, None) == INVALID
    assert acc(FAKE, P.ATTR_F16, 10, 60, 64, P.PRECOND_DIAG, H, None, 0, None) == ALIGN
    assert acc(FAKE, P.ATTR_F16, 10, 64, 32, P.PRECOND_DIAG, H, None, 0, None) == INVALID
    assert acc(FAKE, P.ATTR_F16, 10, 64, 64, P.PRECOND_DIAG, 0, None, 0, None) == INVALID
    assert acc(FAKE, P.ATTR_F16, 10, 64, 64, P.PRECOND_DIAG, H, None, 0, None) == WORKSPACE
    assert acc(FAKE, P.ATTR_F16, 10, 64, 64, P.PRECOND_DIAG, FAKE + 64, None, 0, None) == INVALID  # H inside X
    assert acc(FAKE, P.ATTR_F16, 0, 64, 64, P.PRECOND_DIAG, H, None, 0, None) == OK
    app = L.attr_precond_apply
    Y = FAKE + (1 << 30)
    assert app(FAKE, P.ATTR_BF16, 4, 64, 64, P.PRECOND_NONE, None, 1, Y, P.ATTR_F16, 64, None, 0, None) == UNSUPPORTED
    assert app(FAKE, P.ATTR_F32, 4, 64, 64, P.PRECOND_DIAG, None, 1, Y, P.ATTR_F16, 64, None, 0, None) == INVALID
    assert app(FAKE, P.ATTR_F32, 4, 64, 64, P.PRECOND_NONE, FAKE, 1, Y, P.ATTR_F16, 64, None, 0, None) == INVALID
    assert app(FAKE, P.ATTR_F32, 4, 64, 64, P.PRECOND_NONE, None, 1, FAKE + 8 * 64, P.ATTR_F16, 64, None, 0, None) == INVALID
    assert app(FAKE, P.ATTR_F32, 4, 12, 64, P.PRECOND_NONE, None, 1, Y, P.ATTR_F16, 64, None, 0, None) == ALIGN
    assert app(FAKE, P.ATTR_F32, 0, 64, 64, P.PRECOND_NONE, None, 1, Y, P.ATTR_F16, 64, None, 0, None) == OK


def test_error_message_is_thread_local_and_cleared(L):
    _project(L, [_mod()], k=24)
    assert L.attr_last_error() != b""
    assert _project(L, [_mod()], n=0) == OK
    assert L.attr_last_error() == b""


def test_score_validation(L):
    sc = L.attr_score_topk
    G = FAKE + (1 << 32)
    TS, TI = FAKE + (2 << 32), FAKE + (3 << 32)
    args = dict(Q=FAKE, nq=4, ldq=128, G=G, ng=100, ldg=128, dt=P.ATTR_F16, D=128, k=10,
                base=0, merge=0, ts=TS, ti=TI, ws=None, wsb=0)

    def call(**kw):
        a = dict(args, **kw)
        return sc(a["Q"], a["nq"], a["ldq"], a["G"], a["ng"], a["ldg"], a["dt"], a["D"], a["k"],
                  a["base"], a["merge"], a["ts"], a["ti"], a["ws"], a["wsb"], None)
    assert call(dt=P.ATTR_BF16) == UNSUPPORTED
    assert call(k=0) == UNSUPPORTED and call(k=129) == UNSUPPORTED
    assert call(D=96) == ALIGN                       # fp16 needs multiples of 64
    assert call(D=96, dt=P.ATTR_F32, ldq=96, ldg=96) == WORKSPACE   # fp32: multiples of 32 are fine
    assert call(ldq=64) == INVALID
    assert call(nq=-1) == INVALID
    assert call(merge=2) == INVALID
    assert call(base=-5) == INVALID
    assert call(ts=FAKE + 256) == INVALID            # output inside Q
    assert call(ti=TS + 16) == INVALID               # outputs overlap
    assert call(G=0) == INVALID
    assert call() == WORKSPACE
    need = L.attr_score_topk_workspace_size(4, 100, 128, 10)
    assert need > 0
    assert call(ws=FAKE + (4 << 32) + 16, wsb=need) == ALIGN
    assert call(nq=0) == OK
    assert call(ng=0, merge=1) == OK


def test_full_mode_validation(L):
    acc, app = L.attr_precond_accumulate, L.attr_precond_apply
    H = FAKE + (1 << 34)
    Y = FAKE + (1 << 35)
    assert acc(FAKE, P.ATTR_F32, 100, 256, 256, P.PRECOND_FULL, H, None, 0, None) == UNSUPPORTED
    assert acc(FAKE, P.ATTR_F16, 100, 200, 200, P.PRECOND_FULL, H, None, 0, None) == ALIGN
    assert acc(FAKE, P.ATTR_F16, 100, 256, 256, P.PRECOND_FULL, FAKE + 4096, None, 0, None) == INVALID
    assert acc(FAKE, P.ATTR_F16, 100, 256, 256, P.PRECOND_FULL, H, None, 0, None) == WORKSPACE
    need = L.attr_precond_accumulate_workspace_size(100, 256, P.ATTR_F16, P.PRECOND_FULL)
    assert need > 256 * 256 * 8
    assert app(FAKE, P.ATTR_F32, 4, 256, 256, P.PRECOND_FULL, H, 1, Y, P.ATTR_F16, 256, None, 0, None) == UNSUPPORTED
    assert app(FAKE, P.ATTR_F16, 4, 256, 256, P.PRECOND_FULL, None, 1, Y, P.ATTR_F16, 256, None, 0, None) == INVALID
    assert app(FAKE, P.ATTR_F16, 4, 256, 256, P.PRECOND_FULL, H, 1, FAKE, P.ATTR_F16, 256, None, 0, None) == INVALID
    assert app(FAKE, P.ATTR_F16, 4, 256, 256, P.PRECOND_FULL, H, 1, Y, P.ATTR_F16, 256, None, 0, None) == WORKSPACE
    assert L.attr_precond_apply_workspace_size(4, 256, P.PRECOND_FULL) >= 2 * 256 * 256 * 2
    assert L.attr_precond_apply_workspace_size(4, 256, P.PRECOND_DIAG) == 0


def test_build_flags_unprotected_lds_dma_loads():
    """The build rejects device code where a VALU instruction writes a
    descriptor SGPR of an inline-asm direct-to-LDS load fewer than five wait
    states before it (the compiler does not protect loads inside asm)."""
    from paper_2606_11660_amd.build import lds_dma_hazards
    bad = "\n".join(["_Zkern:", "\tv_readfirstlane_b32 s6, v38", "\tv_add_u32_e32 v5, v1, v2",
                     "\tbuffer_load_dwordx4 v5, s[4:7], 0 offen offset:0 lds"])
    good = "\n".join(["_Zkern:", "\tv_readfirstlane_b32 s6, v38", "\ts_nop 4",
                      "\tbuffer_load_dwordx4 v5, s[4:7], 0 offen offset:0 lds"])
    other = "\n".join(["_Zkern:", "\tv_readfirstlane_b32 s9, v38",
                       "\tbuffer_load_dwordx4 v5, s[4:7], 0 offen offset:0 lds"])
    assert len(lds_dma_hazards(bad)) == 1
    assert lds_dma_hazards(good) == []
    assert lds_dma_hazards(other) == []


LOAD = "\tbuffer_load_dwordx4 v5, s[4:7], 0 offen offset:0 lds"


def _asm(*lines):
    return "\n".join(["_Zkern:", *lines])


def test_lds_dma_hazards_vop3b_sgpr_destinations():
    """SGPR outputs in the second operand of VOP3b forms (carry-out of
    v_add_co_u32, v_mad_u64_u32, v_div_scale) count as writes; an SGPR a
    VALU instruction only reads does not, nor does a carry into VCC."""
    from paper_2606_11660_amd.build import lds_dma_hazards
    for w in ("\tv_add_co_u32_e64 v1, s[6:7], v2, v3", "\tv_addc_co_u32_e64 v1, s[4:5], v2, v3, vcc",
              "\tv_mad_u64_u32 v[2:3], s[6:7], v4, v5, v[6:7]",
              "\tv_div_scale_f32 v1, s[4:5], v2, v2, v3", "\tv_cmp_lt_i64_e64 s[6:7], v[0:1], v[2:3]"):
        assert len(lds_dma_hazards(_asm(w, "\ts_nop 3", LOAD))) == 1, w
        assert lds_dma_hazards(_asm(w, "\ts_nop 4", LOAD)) == [], w
    for r in ("\tv_add_u32_e32 v1, s4, v2", "\tv_mov_b32_e32 v1, s7",
              "\tv_add_co_u32_e32 v1, vcc, s4, v2", "\tv_cndmask_b32_e64 v1, v2, v3, s[6:7]"):
        assert lds_dma_hazards(_asm(r, LOAD)) == [], r


def test_lds_dma_hazards_follow_branches_and_back_edges():
    """Wait states are counted along every path into the load: a write at
    the bottom of a loop reaches a load at the top through the back-edge; a
    write before a forward branch reaches the branch target; an unconditional
    branch or s_endpgm ends fall-through; enough wait states on every path
    pass."""
    from paper_2606_11660_amd.build import lds_dma_hazards
    loop = _asm("\ts_mov_b32 s10, 0", "\ts_nop 7", ".LBB0_1:", LOAD, "\ts_add_u32 s10, s10, 1",
                "\tv_readfirstlane_b32 s5, v9", "\ts_cmp_lg_u32 s10, 8", "\ts_cbranch_scc1 .LBB0_1",
                "\ts_endpgm")
    assert len(lds_dma_hazards(loop)) == 1
    safe_loop = loop.replace("\ts_cmp_lg_u32", "\ts_nop 4\n\ts_cmp_lg_u32")
    assert lds_dma_hazards(safe_loop) == []
    fwd = _asm("\tv_readfirstlane_b32 s6, v1", "\ts_cbranch_scc0 .LBB0_2", "\ts_nop 7",
               "\ts_nop 7", ".LBB0_2:", LOAD, "\ts_endpgm")
    assert len(lds_dma_hazards(fwd)) == 1
    assert lds_dma_hazards(fwd.replace("\ts_cbranch_scc0", "\ts_nop 4\n\ts_cbranch_scc0")) == []
    dead = _asm("\tv_readfirstlane_b32 s6, v1", "\ts_branch .LBB0_3", ".LBB0_4:", LOAD,
                "\ts_endpgm", ".LBB0_3:", "\ts_nop 7", "\ts_nop 7", "\ts_branch .LBB0_4")
    assert lds_dma_hazards(dead) == []
    fall = _asm("\tv_readfirstlane_b32 s6, v1", "\ts_endpgm", ".LBB0_5:", LOAD)
    assert lds_dma_hazards(fall) == []


def test_lds_dma_hazards_m0_write():
    """The load reads its LDS address from M0: an M0 write needs one wait
    state before it."""
    from paper_2606_11660_amd.build import lds_dma_hazards
    set_m0 = [";;#ASMSTART", "\ts_mov_b32 m0, s8"]
    assert len(lds_dma_hazards(_asm(*set_m0, ";;#ASMEND", LOAD))) == 1
    assert lds_dma_hazards(_asm(*set_m0, "\ts_nop 0", ";;#ASMEND", LOAD)) == []


def test_lds_dma_hazards_compiler_m0_write():
    """M0 belongs to the asm that sets it for the loads: a compiler-generated
    M0 write (outside the asm blocks) in a function with direct-to-LDS loads
    is refused; the same write in a function without them is not."""
    from paper_2606_11660_amd.build import lds_dma_hazards
    own = _asm(";;#ASMSTART", "\ts_mov_b32 m0, s8", "\ts_nop 0", ";;#ASMEND", "\ts_nop 7", LOAD)
    assert lds_dma_hazards(own) == []
    comp = _asm("\ts_movk_i32 m0, 0x100", "\ts_nop 7", "\ts_nop 7", LOAD)
    assert len(lds_dma_hazards(comp)) == 1
    other = "\n".join(["_Zother:", "\ts_mov_b32 m0, -1", "\ts_endpgm"]) + "\n" + _asm("\ts_nop 7", LOAD)
    assert lds_dma_hazards(other) == []


def test_asm_valu_write_before_mfma_read():
    """An inline-asm VALU write (the sign flips of MFMA fragments) needs two
    wait states before an MFMA reads the VGPR; other MFMAs, s_nop and
    unrelated VGPRs do not trip it; a label or branch inside the window is
    refused (the scan does not follow control flow)."""
    from paper_2606_11660_amd.build import asm_valu_mfma_hazards
    flip = [";;#ASMSTART", "\tv_xor_b32 v5, 0x80008000, v5", ";;#ASMEND"]
    mf = "\tv_mfma_f32_16x16x32_f16 a[0:3], v[8:11], v[4:7], a[0:3]"
    assert len(asm_valu_mfma_hazards(_asm(*flip, mf))) == 1
    assert len(asm_valu_mfma_hazards(_asm(*flip, "\ts_nop 0", mf))) == 1
    assert asm_valu_mfma_hazards(_asm(*flip, "\ts_nop 1", mf)) == []
    other = "\tv_mfma_f32_16x16x32_f16 a[4:7], v[8:11], v[12:15], a[4:7]"
    assert len(asm_valu_mfma_hazards(_asm(*flip, other, mf))) == 1
    assert asm_valu_mfma_hazards(_asm(*flip, other, other, mf)) == []
    assert len(asm_valu_mfma_hazards(_asm(*flip, ".LBB0_1:", "\ts_nop 7", mf))) == 1
    # the same write by compiler-generated code is the compiler's to protect
    assert asm_valu_mfma_hazards(_asm("\tv_xor_b32_e32 v5, 0x80008000, v5", mf)) == []


def test_built_device_code_passes_the_hazard_scan():
    """Every device assembly file of the last build passes the scan (the
    build itself refuses to link otherwise); the scan sees the loads."""
    import glob
    from paper_2606_11660_amd.build import lds_dma_hazards
    files = glob.glob(os.path.join(ROOT, "paper_2606_11660_amd", "_build", "*.s"))
    if not files:
        pytest.skip("no device assembly: build first")
    from paper_2606_11660_amd.build import asm_valu_mfma_hazards
    n_loads = n_flips = 0
    for f in files:
        asm = open(f).read()
        n_loads += sum(1 for l in asm.splitlines() if "buffer_load_dword" in l and " lds" in l)
        n_flips += sum(1 for l in asm.splitlines() if l.strip().startswith("v_xor_b32 v"))
        assert lds_dma_hazards(asm) == [], f
        assert asm_valu_mfma_hazards(asm) == [], f
    assert n_loads > 0 and n_flips > 0


def test_syrk_plan_slices_fit_their_buffer_range(tmp_path):
    """Compile the host-only SYRK planner with g++ and check its arithmetic
    over row counts, widths and strides up to the accepted maximum (65536):
    no K-slice spans more than 2^31 bytes, chunks cover the rows, the
    workspace query covers every stride's plan, and the last stage holding
    rows starts inside its slice's descriptor range."""
    import shutil
    import subprocess
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = tmp_path / "syrk_plan_check"
    src = os.path.join(ROOT, "tests", "native", "syrk_plan_check.cpp")
    csrc = os.path.join(ROOT, "paper_2606_11660_amd", "csrc")
    subprocess.run([gxx, "-std=c++17", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                    f"-I{csrc}", f"-I{os.path.join(ROOT, 'include')}", src, "-o", str(exe)],
                   check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.startswith("ok")


def test_project_noalloc_validation_and_scratch_limit(L):
    """The allocation-free projection validates like attr_project, and a call
    whose workspace would exceed the static scratch (64 MiB) is rejected with
    ATTR_ERR_WORKSPACE before any device call."""
    def call(mods, n=4, T=32, k=16, dtype=P.ATTR_BF16, ldo=256):
        arr = (P._CModule * len(mods))(*mods)
        return L.attr_project_noalloc(arr, len(mods), dtype, k, n, T, None, None, FAKE, ldo, None)
    assert call([_mod()], k=24) == UNSUPPORTED
    assert call([_mod(d_in=96)]) == ALIGN
    assert call([_mod(out_col=1)]) == INVALID
    assert call([_mod()], n=0) == OK                                    # nothing to do
    # one 64x64 module at k = 64: 16 KiB of partials per example; 5000 examples need 78 MiB
    need = L.attr_project_workspace_size((P._CModule * 1)(_mod()), 1, P.ATTR_BF16, 5000, 32, 64)
    assert need > (64 << 20)
    assert call([_mod()], n=5000, k=64, ldo=4096) == WORKSPACE
    assert b"static buffer" in L.attr_last_error()
