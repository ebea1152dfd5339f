"""GPU parity of attr_project against the fp64 oracle (same seeded inputs).

Bar: per-row relative L2 error <= 1e-5 for fp32 inputs and <= 2e-2 for
bf16 inputs.  The bf16 path multiplies exact bf16 values and accumulates in
fp32, so its error is also checked against a 1e-4 design bound.
"""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_11660_amd as P
import synth
from tests._util import dev, host, row_rel_l2, say

pytestmark = pytest.mark.gpu

BF16_TOL, F32_TOL, BF16_DESIGN = 2e-2, 1e-5, 1e-4


def _run_project(mods_host, k, n, T, length=None, row_offset=None, dtype="bf16", ldo=None,
                 extra_cols=0, nan_pad=True):
    """mods_host: list of (a [n*T or rows, d_in], g, R, S) numpy arrays."""
    D = len(mods_host) * k * k
    ldo = ldo or D + extra_cols
    out = torch.full((n, ldo), -7.0, dtype=torch.float32, device="cuda")
    mods = []
    for m, (a, g, R, S) in enumerate(mods_host):
        mods.append(P.Module(dev(a), dev(g), dev(R), dev(S), out_col=m * k * k))
    L = None if length is None else torch.from_numpy(np.asarray(length, dtype=np.int32)).cuda()
    ro = None if row_offset is None else torch.from_numpy(np.asarray(row_offset, dtype=np.int64)).cuda()
    P.attr_project(mods, k, n, T, out, row_offset=ro, length=L)
    torch.cuda.synchronize()
    return host(out)


def _oracle(mods_host, k, n, T, length=None, row_offset=None):
    blocks = []
    for (a, g, R, S) in mods_host:
        if row_offset is None:
            a3 = a.reshape(n, T, -1)
            g3 = g.reshape(n, T, -1)
        else:
            a3 = np.stack([a[row_offset[i]:row_offset[i] + T] for i in range(n)])
            g3 = np.stack([g[row_offset[i]:row_offset[i] + T] for i in range(n)])
        blocks.append(O.project(a3, g3, R, S, length=length))
    return O.project_concat(blocks)


def test_tiny_fp32_parity():
    say("case: tiny fp32 k=16 n=256 T=32")
    x = synth.tiny_inputs()
    a = x["a"].reshape(-1, 64)
    g = x["g"].reshape(-1, 64)
    got = _run_project([(a, g, x["R"], x["S"])], 16, 256, 32, dtype="f32")
    ref = O.project(x["a"], x["g"], x["R"], x["S"])
    err = row_rel_l2(got, ref)
    say("tiny max row rel-L2", err.max())
    assert err.max() <= F32_TOL


def _random_modules(shapes, n, T, k, dtype, seed, lengths=None):
    rng = np.random.default_rng(seed)
    out = []
    for (d_in, d_out) in shapes:
        a = rng.standard_normal((n * T, d_in))
        g = rng.standard_normal((n * T, d_out)) * 1e-2
        R = rng.standard_normal((d_out, k)) / np.sqrt(k)
        S = rng.standard_normal((d_in, k)) / np.sqrt(k)
        if dtype == "bf16":
            cast = synth.to_bf16_bits
        else:
            cast = lambda v: v.astype(np.float32)
        a, g, R, S = cast(a), cast(g), cast(R), cast(S)
        if lengths is not None:
            for i, L in enumerate(lengths):
                a[i * T:(i + 1) * T] = synth.nan_pad(a[i * T:(i + 1) * T], L)
                g[i * T:(i + 1) * T] = synth.nan_pad(g[i * T:(i + 1) * T], L)
        out.append((a, g, R, S))
    return out


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k", [16, 32, 64])
def test_ragged_lengths_nan_padding(dtype, k):
    n, T = 7, 300                     # T spans two 256-token chunks, not a multiple of 16
    lengths = [0, 1, 17, 255, 256, 257, 300]
    shapes = [(64, 192), (128, 64), (64, 128)]
    say(f"case: ragged dtype={dtype} k={k} n={n} T={T}")
    mods = _random_modules(shapes, n, T, k, dtype, seed=100 + k, lengths=lengths)
    got = _run_project(mods, k, n, T, length=lengths, dtype=dtype)
    ref = _oracle(mods, k, n, T, length=lengths)
    assert np.isfinite(got).all()
    assert (got[0] == 0).all()        # len 0 -> zero row
    err = row_rel_l2(got, ref)
    say("max row rel-L2", err.max())
    assert err.max() <= (BF16_DESIGN if dtype == "bf16" else F32_TOL)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k", [16, 32, 64])
def test_shared_inputs_grouped(dtype, k):
    """Modules reading the same input rows (same a tensor, stride and width)
    are projected in groups that read a once: three modules share one a
    (q/k/v-like), two another (gate/up-like), four a third (a group of three,
    or of two at k = 64, plus the rest), one is alone; the members are
    interleaved in the module list; ragged lengths with NaN padding.  Parity
    with the oracle per module, and bitwise equality with the same call on
    unshared copies of every a."""
    n, T = 5, 300
    lengths = [1, 255, 256, 300, 77]
    spec = [(0, 64, 192), (1, 128, 64), (2, 64, 64), (0, 64, 128), (3, 192, 64),
            (2, 64, 128), (1, 128, 192), (0, 64, 64), (2, 64, 64), (2, 64, 192)]
    say(f"case: shared inputs dtype={dtype} k={k}")
    rng = np.random.default_rng(300 + k)
    cast = synth.to_bf16_bits if dtype == "bf16" else (lambda v: v.astype(np.float32))

    def padded(x):
        for i, L in enumerate(lengths):
            x[i * T:(i + 1) * T] = synth.nan_pad(x[i * T:(i + 1) * T], L)
        return x

    a_host = {}
    for aid, d_in, _ in spec:
        if aid not in a_host:
            a_host[aid] = padded(cast(rng.standard_normal((n * T, d_in))))
    mods_host = []
    for aid, d_in, d_out in spec:
        g = padded(cast(rng.standard_normal((n * T, d_out)) * 1e-2))
        R = cast(rng.standard_normal((d_out, k)) / np.sqrt(k))
        S = cast(rng.standard_normal((d_in, k)) / np.sqrt(k))
        mods_host.append((a_host[aid], g, R, S))
    a_dev = {aid: dev(a) for aid, a in a_host.items()}
    out = torch.full((n, len(spec) * k * k), -7.0, dtype=torch.float32, device="cuda")
    mods = [P.Module(a_dev[aid], dev(g), dev(R), dev(S), out_col=m * k * k)
            for m, ((aid, _, _), (_, g, R, S)) in enumerate(zip(spec, mods_host))]
    L = torch.from_numpy(np.asarray(lengths, dtype=np.int32)).cuda()
    P.attr_project(mods, k, n, T, out, length=L)
    torch.cuda.synchronize()
    shared = host(out)
    separate = _run_project(mods_host, k, n, T, length=lengths, dtype=dtype)
    assert np.isfinite(shared).all()
    assert np.array_equal(shared, separate)
    err = row_rel_l2(shared, _oracle(mods_host, k, n, T, length=lengths))
    say("max row rel-L2", err.max())
    assert err.max() <= (BF16_DESIGN if dtype == "bf16" else F32_TOL)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k", [16, 32, 64])
def test_optimizer_state_normalisation(dtype, k):
    """Gradients normalised by a factored (Adafactor) second moment before
    projection, next to a module without normalisation in the same call;
    factors include a zero and a negative entry (their rows/columns drop
    out); ragged lengths with NaN padding.  bf16: the scaled R/S are
    rounded to bf16 once more, so the bar is the bf16 tolerance."""
    n, T = 4, 300
    lengths = [1, 300, 128, 257]
    shapes = [(64, 192), (128, 64), (64, 128)]
    say(f"case: optimizer-state normalisation dtype={dtype} k={k}")
    mods_host = _random_modules(shapes, n, T, k, dtype, seed=400 + k, lengths=lengths)
    rng = np.random.default_rng(500 + k)
    facs = []
    for m, (d_in, d_out) in enumerate(shapes):
        if m == 1:
            facs.append(None)
            continue
        vo = rng.uniform(0.05, 3.0, d_out).astype(np.float32)
        vi = rng.uniform(0.05, 3.0, d_in).astype(np.float32)
        vo[3], vo[7], vi[5] = 0.0, -2.0, 0.0
        facs.append((vo, vi))
    out = torch.full((n, len(shapes) * k * k), -7.0, dtype=torch.float32, device="cuda")
    mods = []
    for m, ((a, g, R, S), f) in enumerate(zip(mods_host, facs)):
        vo, vi = (None, None) if f is None else (dev(f[0]), dev(f[1]))
        mods.append(P.Module(dev(a), dev(g), dev(R), dev(S), out_col=m * k * k, v_out=vo, v_in=vi))
    P.attr_project(mods, k, n, T, out, length=torch.from_numpy(np.asarray(lengths, dtype=np.int32)).cuda())
    torch.cuda.synchronize()
    got = host(out)
    blocks = []
    for (a, g, R, S), f in zip(mods_host, facs):
        a3, g3 = a.reshape(n, T, -1), g.reshape(n, T, -1)
        blocks.append(O.project(a3, g3, R, S, length=lengths) if f is None else
                      O.project_normalized(a3, g3, R, S, f[0], f[1], length=lengths))
    ref = O.project_concat(blocks)
    assert np.isfinite(got).all()
    err = row_rel_l2(got, ref)
    say("max row rel-L2", err.max())
    assert err.max() <= (BF16_TOL if dtype == "bf16" else F32_TOL)


def test_optimizer_state_factors_both_or_neither():
    a = torch.zeros((4, 64), dtype=torch.float32, device="cuda")
    g = torch.zeros((4, 64), dtype=torch.float32, device="cuda")
    R = torch.zeros((64, 16), dtype=torch.float32, device="cuda")
    S = torch.zeros((64, 16), dtype=torch.float32, device="cuda")
    out = torch.zeros((1, 256), dtype=torch.float32, device="cuda")
    m = P.Module(a, g, R, S, 0, v_out=torch.ones(64, device="cuda"), v_in=None)
    with pytest.raises(P.AttrError):
        P.attr_project([m], 16, 1, 4, out)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k", [16, 32, 64])
@pytest.mark.parametrize("packed", [False, True])
def test_per_token_blocks(dtype, k, packed):
    """attr_project_tokens: every valid token's k x k block at the token's
    own row (padded layout, or packed back to back through row_offset);
    padded tokens' rows and columns outside the blocks untouched; two modules
    share their input rows (grouped path); the token rows of an example sum
    to attr_project's row."""
    n, T = 3, 300
    lengths = [1, 300, 77]
    shapes = [(64, 192), (128, 64), (64, 128)]
    say(f"case: per-token blocks dtype={dtype} k={k} packed={packed}")
    mods_host = _random_modules(shapes, n, T, k, dtype, seed=600 + k, lengths=lengths)
    a0 = mods_host[0][0]
    mods_host[2] = (a0, mods_host[2][1], mods_host[2][2], mods_host[2][3])   # shares module 0's a
    D = len(shapes) * k * k
    if packed:
        offs = np.concatenate([[0], np.cumsum(lengths)[:-1]]).astype(np.int64)
        rows = int(sum(lengths))
        def pack(x):
            return np.concatenate([x[i * T:i * T + lengths[i]] for i in range(n)])
        dev_mods_src = [(pack(a), pack(g), R, S) for a, g, R, S in mods_host]
        ro = torch.from_numpy(offs).cuda()
    else:
        rows = n * T
        dev_mods_src = mods_host
        ro = None
    a_dev = {}
    mods = []
    for m, (a, g, R, S) in enumerate(dev_mods_src):
        key = id(mods_host[m][0])
        if key not in a_dev:
            a_dev[key] = dev(a)
        mods.append(P.Module(a_dev[key], dev(g), dev(R), dev(S), out_col=m * k * k))
    L = torch.from_numpy(np.asarray(lengths, dtype=np.int32)).cuda()
    out = torch.full((rows, D + 5), -7.0, dtype=torch.float32, device="cuda")
    P.attr_project_tokens(mods, k, n, T, out, row_offset=ro, length=L)
    ex = torch.empty((n, D), dtype=torch.float32, device="cuda")
    P.attr_project(mods, k, n, T, ex, row_offset=ro, length=L)
    torch.cuda.synchronize()
    got = host(out)
    ref = O.project_concat([O.project_tokens(a.reshape(n, T, -1), g.reshape(n, T, -1), R, S,
                                             length=lengths).reshape(n * T, -1)
                            for a, g, R, S in mods_host]).reshape(n, T, D)
    tol = BF16_DESIGN if dtype == "bf16" else F32_TOL
    assert (got[:, D:] == -7.0).all()
    for i in range(n):
        r0 = int(offs[i]) if packed else i * T
        blk = got[r0:r0 + lengths[i], :D]
        err = row_rel_l2(blk, ref[i, :lengths[i]])
        assert err.max() <= tol, (i, err.max())
        if not packed:
            assert (got[r0 + lengths[i]:r0 + T] == -7.0).all()
        np.testing.assert_allclose(blk.astype(np.float64).sum(0), host(ex)[i], rtol=1e-4,
                                   atol=1e-4 * np.abs(host(ex)[i]).max())


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("k", [16, 32])
def test_per_token_blocks_normalised(dtype, k):
    """Per-token blocks of optimizer-normalised gradients: each valid token's
    block equals the oracle's normalised projection of a one-token example
    (the definition, G_t = g_t a_t^T divided elementwise by sqrt(V)); a
    module without factors in the same call; padded tokens' rows untouched."""
    n, T = 3, 200
    lengths = [200, 1, 45]
    shapes = [(64, 192), (128, 64)]
    say(f"case: per-token normalised dtype={dtype} k={k}")
    mods_host = _random_modules(shapes, n, T, k, dtype, seed=700 + k, lengths=lengths)
    rng = np.random.default_rng(800 + k)
    vo = rng.uniform(0.05, 3.0, shapes[0][1]).astype(np.float32)
    vi = rng.uniform(0.05, 3.0, shapes[0][0]).astype(np.float32)
    vo[2], vi[9] = 0.0, -1.0
    D = len(shapes) * k * k
    mods = [P.Module(dev(a), dev(g), dev(R), dev(S), out_col=m * k * k,
                     v_out=dev(vo) if m == 0 else None, v_in=dev(vi) if m == 0 else None)
            for m, (a, g, R, S) in enumerate(mods_host)]
    out = torch.full((n * T, D), -7.0, dtype=torch.float32, device="cuda")
    P.attr_project_tokens(mods, k, n, T, out, length=torch.from_numpy(np.asarray(lengths, dtype=np.int32)).cuda())
    torch.cuda.synchronize()
    got = host(out)
    tok_len = [1 if t < lengths[i] else 0 for i in range(n) for t in range(T)]
    blocks = []
    for m, (a, g, R, S) in enumerate(mods_host):
        a1, g1 = a.reshape(n * T, 1, -1), g.reshape(n * T, 1, -1)
        blocks.append(O.project_normalized(a1, g1, R, S, vo, vi, length=tok_len) if m == 0 else
                      O.project(a1, g1, R, S, length=tok_len))
    ref = O.project_concat(blocks).reshape(n, T, D)
    # bf16: the scaled R/S are rounded to bf16 once more (as in attr_project)
    tol = BF16_TOL if dtype == "bf16" else F32_TOL
    for i in range(n):
        blk = got[i * T:i * T + lengths[i]]
        err = row_rel_l2(blk, ref[i, :lengths[i]])
        say(f"example {i}: max row rel-L2 {err.max():.2e}")
        assert err.max() <= tol, (i, err.max())
        assert (got[i * T + lengths[i]:(i + 1) * T] == -7.0).all()


def test_untouched_columns_and_row_offset():
    n, T, k = 5, 40, 16
    say("case: row_offset packed layout, extra output columns")
    shapes = [(192, 64), (64, 128)]
    lengths = [40, 3, 0, 33, 16]
    # packed rows: example i starts at row_offset[i]; rows between are garbage
    row_offset = [0, 50, 60, 61, 120]
    rows = 200
    rng = np.random.default_rng(7)
    mods = []
    for (d_in, d_out) in shapes:
        a = synth.to_bf16_bits(rng.standard_normal((rows, d_in)))
        g = synth.to_bf16_bits(rng.standard_normal((rows, d_out)))
        R = synth.to_bf16_bits(rng.standard_normal((d_out, k)) / 4)
        S = synth.to_bf16_bits(rng.standard_normal((d_in, k)) / 4)
        mods.append((a, g, R, S))
    got = _run_project(mods, k, n, T, length=lengths, row_offset=row_offset, extra_cols=24)
    ref = _oracle(mods, k, n, T, length=lengths, row_offset=row_offset)
    err = row_rel_l2(got[:, :2 * k * k], ref)
    say("max row rel-L2", err.max())
    assert err.max() <= BF16_DESIGN
    assert (got[:, 2 * k * k:] == -7.0).all()


def test_gpt2_shaped_two_examples():
    wl = synth.GPT2
    n, T, k = 2, wl.T, wl.k
    say("case: gpt2 48 modules n=2 T=512")
    mods, blocks = [], []
    for m in range(len(wl.modules)):
        R, S = synth.projection_pair(wl, m)
        a = np.concatenate([synth.module_example(wl, m, i)[0] for i in range(n)])
        g = np.concatenate([synth.module_example(wl, m, i)[1] for i in range(n)])
        mods.append((a, g, R, S))
    got = _run_project(mods, k, n, T)
    ref = _oracle(mods, k, n, T)
    err = row_rel_l2(got, ref)
    say("gpt2 max row rel-L2", err.max())
    assert err.max() <= BF16_DESIGN


def test_llama1b_shaped_lengths():
    wl = synth.LLAMA1B
    n, T, k = 3, wl.T, wl.k
    lengths = synth.example_lengths(wl.n_examples)[:n]
    say(f"case: 1B-shaped modules q/gate/down n=3 T=2048 lengths={list(lengths)}")
    picks = [0, 4, 6]                  # q (2048->2048), gate (2048->8192), down (8192->2048)
    mods = []
    for m in picks:
        R, S = synth.projection_pair(wl, m)
        a = np.concatenate([synth.nan_pad(synth.module_example(wl, m, i)[0], lengths[i]) for i in range(n)])
        g = np.concatenate([synth.nan_pad(synth.module_example(wl, m, i)[1], lengths[i]) for i in range(n)])
        mods.append((a, g, R, S))
    got = _run_project(mods, k, n, T, length=lengths)
    ref = _oracle(mods, k, n, T, length=lengths)
    err = row_rel_l2(got, ref)
    say("1B max row rel-L2", err.max())
    assert err.max() <= BF16_DESIGN


def test_deterministic_bitwise():
    n, T, k = 9, 520, 16
    say("case: determinism")
    mods = _random_modules([(256, 512), (512, 256)], n, T, k, "bf16", seed=5)
    a = _run_project(mods, k, n, T)
    b = _run_project(mods, k, n, T)
    assert np.array_equal(a, b)


def test_zero_examples_is_noop():
    k = 16
    mods = _random_modules([(64, 64)], 1, 16, k, "bf16", seed=6)
    out = torch.full((1, 256), 3.0, device="cuda")
    m = [P.Module(dev(mods[0][0]), dev(mods[0][1]), dev(mods[0][2]), dev(mods[0][3]), 0)]
    P.attr_project(m, k, 0, 16, out)
    torch.cuda.synchronize()
    assert (host(out) == 3.0).all()


def test_bench_launch_full_batch_sampled():
    """The bench's launch: 64 GPT-2 examples x 48 modules x 512 tokens in one
    call (9.7 GB of bf16 inputs); examples 0, 31 and 63 hold the seeded synth
    inputs and are checked row by row against the oracle."""
    wl = synth.GPT2
    n, T, k = 64, wl.T, wl.k
    sampled = [0, 31, 63]
    say("case: gpt2 full batch n=64 (bench launch), sampled rows", sampled)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(1234)
    mods, host_mods = [], []
    for m, md in enumerate(wl.modules):
        a = torch.randn((n * T, md.d_in), generator=gen, device="cuda").to(torch.bfloat16)
        g = (torch.randn((n * T, md.d_out), generator=gen, device="cuda") * 1e-2).to(torch.bfloat16)
        R, S = synth.projection_pair(wl, m)
        ha, hg = [], []
        for i in sampled:
            ai, gi = synth.module_example(wl, m, i)
            a[i * T:(i + 1) * T] = dev(ai)
            g[i * T:(i + 1) * T] = dev(gi)
            ha.append(ai)
            hg.append(gi)
        mods.append(P.Module(a, g, dev(R), dev(S), m * k * k))
        host_mods.append((np.stack(ha), np.stack(hg), R, S))
    out = torch.empty((n, wl.D), dtype=torch.float32, device="cuda")
    P.attr_project(mods, k, n, T, out)
    torch.cuda.synchronize()
    got = host(out)[sampled]
    ref = O.project_concat([O.project(a, g, R, S) for (a, g, R, S) in host_mods])
    err = row_rel_l2(got, ref)
    say("full-batch sampled max row rel-L2", err.max())
    assert err.max() <= BF16_DESIGN
    assert np.isfinite(host(out)).all()


def test_llama1b_bench_launch_sampled():
    """The bench's 1B-shaped launch: 16 examples with ragged lengths packed
    back to back (row_offset / length; 21900 tokens x 112 modules, 33 GB of
    bf16 inputs) in one call; examples 0, 7 and 15 are recomputed by the
    oracle from the same device values (read back, exact bf16 -> fp32)."""
    wl = synth.LLAMA1B
    B, T, k = 16, wl.T, wl.k
    lengths = synth.example_lengths(wl.n_examples)[:B]
    offs = np.concatenate([[0], np.cumsum(lengths.astype(np.int64))[:-1]])
    tot = int(lengths.sum())
    say("case: 1B bench launch B=16 packed, tokens", tot)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(77)
    mods, RS = [], []
    for m, md in enumerate(wl.modules):
        a = torch.randn((tot, md.d_in), generator=gen, device="cuda", dtype=torch.bfloat16)
        g = (torch.randn((tot, md.d_out), generator=gen, device="cuda") * 1e-2).to(torch.bfloat16)
        R, S = synth.projection_pair(wl, m)
        mods.append(P.Module(a, g, dev(R), dev(S), m * k * k))
        RS.append((R, S))
    out = torch.empty((B, wl.D), dtype=torch.float32, device="cuda")
    P.attr_project(mods, k, B, T, out, row_offset=torch.from_numpy(offs).cuda(),
                   length=torch.from_numpy(lengths.astype(np.int32)).cuda())
    torch.cuda.synchronize()
    got = host(out)
    assert np.isfinite(got).all()
    for i in (0, 7, 15):
        r0, n_i = int(offs[i]), int(lengths[i])
        blocks = []
        for M, (R, S) in zip(mods, RS):
            a = M.a[r0:r0 + n_i].float().cpu().numpy()[None]
            g = M.g[r0:r0 + n_i].float().cpu().numpy()[None]
            blocks.append(O.project(a, g, R, S))
        err = row_rel_l2(got[i:i + 1], O.project_concat(blocks))
        say(f"example {i} (length {n_i}) row rel-L2", err[0])
        assert err[0] <= BF16_DESIGN
    del mods, out
    torch.cuda.empty_cache()
