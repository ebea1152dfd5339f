"""Pins of the CPU oracle against what the method and the mathematics fix.

Each test checks the oracle against something other than itself: hand-worked
fixtures, brute force over tokens / pairs on tiny inputs, special cases that
reduce to a known matrix, closed forms (Johnson-Lindenstrauss expectation,
Marchenko-Pastur edges) and invariants.  A plausible mistake in the oracle
(dropped term, wrong sign or index, transposed operand, wrong flatten order,
wrong tie order) fails at least one of them.
"""
import json
import math
import os

import numpy as np
import pytest

import oracle as O
import synth


def _load(golden_dir, name):
    with open(os.path.join(golden_dir, name)) as f:
        d = json.load(f)

    def conv(v):
        if isinstance(v, list):
            return [conv(x) for x in v]
        if isinstance(v, str):
            return float(v)
        return v
    return {k: (conv(v) if k != "source" else v) for k, v in d.items()}


# ----------------------------------------------------------------------------
# projection
# ----------------------------------------------------------------------------
def test_projection_golden_hand_worked(golden_dir):
    d = _load(golden_dir, "projection_k2.json")
    a = np.array(d["a"], dtype=np.float32)[None]
    g = np.array(d["g"], dtype=np.float32)[None]
    R = np.array(d["R"], dtype=np.float32)
    S = np.array(d["S"], dtype=np.float32)
    for fn in (O.project_explicit, O.project):
        P = fn(a, g, R, S, length=[d["length"]])
        np.testing.assert_array_equal(P[0], np.array(d["P_flat"], dtype=np.float64))


def test_concat_golden_module_and_flatten_order(golden_dir):
    # Two modules, two examples, ragged lengths: the store row is module A's
    # k x k block then module B's, each flattened with R's index first.  A
    # module-order, axis or flatten mistake in the concatenation fails here.
    d = _load(golden_dir, "concat_two_modules.json")
    blocks = []
    for m in ("A", "B"):
        a = np.array(d[m + "_a"], dtype=np.float32)
        g = np.array(d[m + "_g"], dtype=np.float32)
        R = np.array(d[m + "_R"], dtype=np.float32)
        S = np.array(d[m + "_S"], dtype=np.float32)
        blocks.append(O.project(a, g, R, S, length=d[m + "_length"]))
    rows = O.project_concat(blocks)
    assert rows.shape == (2, 8)
    np.testing.assert_array_equal(rows, np.array(d["rows"], dtype=np.float64))


def _brute_gradient(a, g, L):
    """Per-example weight gradient summed over tokens by explicit loops over
    tokens and matrix entries (no matrix product)."""
    d_out, d_in = g.shape[1], a.shape[1]
    G = np.zeros((d_out, d_in))
    for t in range(L):
        for r in range(d_out):
            for c in range(d_in):
                G[r, c] += float(g[t, r]) * float(a[t, c])
    return G


def test_identity_projection_reproduces_full_gradient():
    # k = d_in = d_out with R = S = I: P_i is the full per-example gradient.
    rng = np.random.default_rng(11)
    d, T, n = 8, 5, 3
    a = rng.standard_normal((n, T, d)).astype(np.float32)
    g = rng.standard_normal((n, T, d)).astype(np.float32)
    eye = np.eye(d, dtype=np.float32)
    L = [5, 3, 0]
    for fn in (O.project_explicit, O.project):
        P = fn(a, g, eye, eye, length=L)
        for i in range(n):
            np.testing.assert_allclose(P[i].reshape(d, d), _brute_gradient(a[i], g[i], L[i]),
                                       rtol=1e-12, atol=1e-12)


def test_identity_projection_k64_tiny_shape():
    # The tiny workload's module is 64 -> 64, so k = 64 with identities
    # reproduces its exact gradient; checked against a per-token outer sum.
    rng = np.random.default_rng(12)
    a = rng.standard_normal((2, 32, 64)).astype(np.float32)
    g = rng.standard_normal((2, 32, 64)).astype(np.float32)
    eye = np.eye(64, dtype=np.float32)
    P = O.project(a, g, eye, eye)
    for i in range(2):
        G = sum(np.outer(g[i, t].astype(np.float64), a[i, t].astype(np.float64)) for t in range(32))
        np.testing.assert_allclose(P[i].reshape(64, 64), G, rtol=1e-12, atol=1e-10)


def test_selection_projection_picks_entries():
    # R = I[:, r_idx], S = I[:, c_idx]  =>  P[r, c] = G[r_idx[r], c_idx[c]].
    rng = np.random.default_rng(13)
    d_in, d_out, T, k = 24, 20, 7, 16
    a = rng.standard_normal((1, T, d_in)).astype(np.float32)
    g = rng.standard_normal((1, T, d_out)).astype(np.float32)
    r_idx = rng.permutation(d_out)[:k]
    c_idx = rng.permutation(d_in)[:k]
    R = np.eye(d_out, dtype=np.float32)[:, r_idx]
    S = np.eye(d_in, dtype=np.float32)[:, c_idx]
    G = _brute_gradient(a[0], g[0], T)
    want = G[np.ix_(r_idx, c_idx)]
    for fn in (O.project_explicit, O.project):
        np.testing.assert_allclose(fn(a, g, R, S)[0].reshape(k, k), want, rtol=1e-12, atol=1e-12)


def test_tiny_factored_equals_explicit():
    x = synth.tiny_inputs()
    P1 = O.project_explicit(x["a"][:32], x["g"][:32], x["R"], x["S"])
    P2 = O.project(x["a"][:32], x["g"][:32], x["R"], x["S"])
    assert np.max(np.abs(P1 - P2)) <= 1e-12 * np.max(np.abs(P1))


def test_projection_bilinear_additive_and_padding_invariant():
    rng = np.random.default_rng(14)
    n, T, d_in, d_out, k = 2, 9, 32, 48, 16
    a = rng.standard_normal((n, T, d_in)).astype(np.float32)
    g = rng.standard_normal((n, T, d_out)).astype(np.float32)
    R = rng.standard_normal((d_out, k)).astype(np.float32)
    S = rng.standard_normal((d_in, k)).astype(np.float32)
    P = O.project(a, g, R, S)
    # bilinearity in (a, g)
    P2 = O.project(a * np.float32(2.0), g * np.float32(-0.5), R, S)
    np.testing.assert_allclose(P2, -1.0 * P, rtol=1e-12, atol=1e-12)
    # token additivity: P(len 9) = P(first 4 tokens) + P(last 5 tokens)
    Pa = O.project(a[:, :4], g[:, :4], R, S)
    Pb = O.project(a[:, 4:], g[:, 4:], R, S)
    np.testing.assert_allclose(Pa + Pb, P, rtol=1e-10, atol=1e-10)
    # length L equals the first L tokens; NaN padding beyond L changes nothing
    L = [4, 7]
    an = np.stack([synth.nan_pad(a[i], L[i]) for i in range(n)])
    gn = np.stack([synth.nan_pad(g[i], L[i]) for i in range(n)])
    Pl = O.project(an, gn, R, S, length=L)
    for i in range(n):
        ref = O.project(a[i:i + 1, :L[i]], g[i:i + 1, :L[i]], R, S)[0]
        np.testing.assert_array_equal(Pl[i], ref)
    assert np.isfinite(O.project_explicit(an, gn, R, S, length=L)).all()


# ----------------------------------------------------------------------------
# optimizer-state (factored second moment) normalisation before projection
# ----------------------------------------------------------------------------
def _small_module(seed, n=3, T=6, d_in=24, d_out=40, k=16):
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((n, T, d_in))
    g = rng.standard_normal((n, T, d_out))
    R = rng.standard_normal((d_out, k))
    S = rng.standard_normal((d_in, k))
    return rng, a, g, R, S


def test_project_tokens_rank_one_blocks_summing_to_the_example():
    """Per-token blocks: each k x k block has rank one (its singular values
    past the first vanish), a token's block equals the example projection of
    that token alone, the valid blocks sum to the per-example projection,
    and padded tokens give zero rows."""
    rng, a, g, R, S = _small_module(35)
    L = [6, 2, 0]
    an = np.stack([synth.nan_pad(a[i], L[i]) for i in range(3)])
    gn = np.stack([synth.nan_pad(g[i], L[i]) for i in range(3)])
    Pt = O.project_tokens(an, gn, R, S, length=L)
    k = R.shape[1]
    sv = np.linalg.svd(Pt[0, 3].reshape(k, k), compute_uv=False)
    assert sv[1] <= 1e-12 * sv[0]
    np.testing.assert_allclose(Pt[1, 1], O.project(a[1:2, 1:2], g[1:2, 1:2], R, S)[0], rtol=1e-12)
    np.testing.assert_allclose(Pt.sum(axis=1), O.project(an, gn, R, S, length=L), rtol=1e-10, atol=1e-12)
    assert (Pt[1, 2:] == 0).all() and (Pt[2] == 0).all()


def test_factored_second_moment_rebuilds_rank_one_from_sums():
    """Adafactor's factored estimate, built from the row sums and column sums
    of a non-negative rank-one matrix W = r c^T, is W itself (row sums r_i
    sum(c), column sums c_j sum(r)); a dropped or wrong normaliser fails."""
    rng = np.random.default_rng(41)
    r, c = rng.uniform(0.1, 2.0, 7), rng.uniform(0.1, 2.0, 5)
    W = np.outer(r, c)
    V = O.factored_second_moment(W.sum(axis=1), W.sum(axis=0))
    np.testing.assert_allclose(V, W, rtol=1e-13)


def test_factored_second_moment_worked_case():
    """v_out = (1, 3), v_in = (2, 0, -1): non-positive factors read as 0,
    V = v_out v_in^T / 4 = [[0.5, 0, 0], [1.5, 0, 0]] by hand; all-zero row
    factors give V = 0."""
    V = O.factored_second_moment(np.array([1.0, 3.0]), np.array([2.0, 0.0, -1.0]))
    np.testing.assert_array_equal(V, np.array([[0.5, 0.0, 0.0], [1.5, 0.0, 0.0]]))
    assert not O.factored_second_moment(np.zeros(3), np.ones(2)).any()


def test_to_f16_rounding_fixed_by_ieee754():
    """Binary16 rounding to nearest, ties to even (IEEE 754): 2049 and 2051
    are ties between representable neighbours 2 apart; 65520 is the tie
    between the largest finite value 65504 and the overflow threshold, so it
    rounds to infinity; 2^-24 is the smallest subnormal and 2^-25 ties to 0."""
    x = np.array([2049.0, 2051.0, 65519.0, 65520.0, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26, -2049.0])
    with np.errstate(over="ignore"):
        got = O.to_f16(x).astype(np.float64)
    want = np.array([2048.0, 2052.0, 65504.0, np.inf, 2.0 ** -24, 0.0, 2.0 ** -24, -2048.0])
    np.testing.assert_array_equal(got, want)


def test_normalized_uniform_factors_scale_plain_projection():
    """v_out = alpha 1, v_in = beta 1: V = beta / d_out everywhere, so the
    normalised projection is sqrt(d_out / beta) times the plain one."""
    _, a, g, R, S = _small_module(31)
    d_out = g.shape[-1]
    Pn = O.project_normalized(a, g, R, S, np.full(d_out, 3.0), np.full(a.shape[-1], 0.25))
    np.testing.assert_allclose(Pn, math.sqrt(d_out / 0.25) * O.project(a, g, R, S), rtol=1e-12)


def test_normalized_matching_rank_one_moment_gives_sign_matrix():
    """One token, g = u, a = w, and factors u^2, w^2: the normalised
    gradient is sqrt(sum u^2) sign(u) sign(w)^T, so P = sqrt(sum u^2)
    (R^T sign u)(S^T sign w)^T."""
    rng, _, _, R, S = _small_module(32)
    u = rng.standard_normal(R.shape[0])
    w = rng.standard_normal(S.shape[0])
    P = O.project_normalized(w[None, None, :], u[None, None, :], R, S, u ** 2, w ** 2)
    ref = math.sqrt((u ** 2).sum()) * np.outer(R.T @ np.sign(u), S.T @ np.sign(w))
    np.testing.assert_allclose(P[0], ref.reshape(-1), rtol=1e-10)


def test_normalized_invariances_and_zero_factors():
    """Scaling v_out leaves V unchanged; scaling v_in by mu scales P by
    mu^-1/2; a zero factor makes the result independent of that gradient row
    (output side) or column (input side)."""
    rng, a, g, R, S = _small_module(33)
    vo = rng.uniform(0.5, 2.0, g.shape[-1])
    vi = rng.uniform(0.5, 2.0, a.shape[-1])
    P = O.project_normalized(a, g, R, S, vo, vi)
    np.testing.assert_allclose(O.project_normalized(a, g, R, S, 7.0 * vo, vi), P, rtol=1e-12)
    np.testing.assert_allclose(O.project_normalized(a, g, R, S, vo, 4.0 * vi), P / 2.0, rtol=1e-12)
    vo0, vi0 = vo.copy(), vi.copy()
    vo0[5], vi0[3] = 0.0, -1.0
    g2, a2 = g.copy(), a.copy()
    g2[..., 5] = rng.standard_normal(g2[..., 5].shape)
    a2[..., 3] = rng.standard_normal(a2[..., 3].shape)
    np.testing.assert_allclose(O.project_normalized(a2, g2, R, S, vo0, vi0),
                               O.project_normalized(a, g, R, S, vo0, vi0), rtol=1e-12, atol=1e-12)


def test_bf16_decoding_exact():
    vals = np.array([1.0, -2.5, 3.140625, 0.0, 65280.0, 1e-2], dtype=np.float32)
    bits = synth.to_bf16_bits(vals)
    back = O.bf16_bits_to_f64(bits)
    np.testing.assert_array_equal(back[:5], vals[:5].astype(np.float64))
    # 1e-2 rounds to the nearest bf16 (8 significant bits): |err| <= 2^-8 relative
    assert abs(back[5] - 1e-2) <= 1e-2 * 2.0 ** -8


def test_projection_jl_expectation():
    # Under R, S with i.i.d. N(0, 1/k) entries, E[R R^T] = I and E[S S^T] = I,
    # so E <P_i, P_j> = <G_i, G_j>_F (unbiased inner products, the reason the
    # projection preserves scores in expectation).  Mean over 400 draws, 5 sigma.
    rng = np.random.default_rng(15)
    T, d_in, d_out, k = 6, 12, 10, 16
    a = rng.standard_normal((2, T, d_in)).astype(np.float32)
    g = rng.standard_normal((2, T, d_out)).astype(np.float32)
    Gi = _brute_gradient(a[0], g[0], T)
    Gj = _brute_gradient(a[1], g[1], T)
    target = float((Gi * Gj).sum())
    samples = []
    for s in range(400):
        r = np.random.default_rng([77, s])
        R = (r.standard_normal((d_out, k)) / math.sqrt(k)).astype(np.float32)
        S = (r.standard_normal((d_in, k)) / math.sqrt(k)).astype(np.float32)
        P = O.project(a, g, R, S)
        samples.append(float(P[0] @ P[1]))
    samples = np.array(samples)
    se = samples.std(ddof=1) / math.sqrt(len(samples))
    assert abs(samples.mean() - target) < 5 * se


# ----------------------------------------------------------------------------
# normalisation and preconditioning
# ----------------------------------------------------------------------------
def test_normalisation_golden_and_invariants(golden_dir):
    d = _load(golden_dir, "precond_small.json")
    np.testing.assert_allclose(O.unit_normalize(np.array(d["norm_in"])), np.array(d["norm_out"]),
                               rtol=0, atol=1e-15)
    X = np.random.default_rng(16).standard_normal((50, 33)) * 7.0
    Y = O.unit_normalize(X)
    assert np.allclose(np.linalg.norm(Y, axis=1), 1.0, atol=1e-14)
    # direction preserved: every row is a positive multiple of the input row
    ratio = Y / X
    assert np.allclose(ratio, ratio[:, :1], rtol=1e-12) and (ratio > 0).all()


def test_diag_finalize_golden(golden_dir):
    d = _load(golden_dir, "precond_small.json")
    m = O.finalize_diag(np.array(d["diag_h"], dtype=np.float64), d["diag_n"])
    np.testing.assert_allclose(m, np.array(d["diag_m"]), rtol=0, atol=1e-15)


def test_full_finalize_golden(golden_dir):
    d = _load(golden_dir, "precond_small.json")
    M, lam = O.finalize_full(np.array(d["full_H"], dtype=np.float64), d["full_n"])
    np.testing.assert_allclose(M, np.array(d["full_M"]), rtol=0, atol=1e-14)
    np.testing.assert_allclose(np.sort(lam), [1.0, 3.0], atol=1e-14)


def test_accumulate_brute_force():
    rng = np.random.default_rng(17)
    X = rng.standard_normal((37, 9)).astype(np.float16)
    h = O.accumulate_diag(X)
    H = O.accumulate_full(X)
    Hb = np.zeros((9, 9))
    for i in range(37):
        for p in range(9):
            for q in range(9):
                Hb[p, q] += float(X[i, p]) * float(X[i, q])
    np.testing.assert_allclose(H, Hb, rtol=1e-13, atol=1e-12)
    np.testing.assert_allclose(h, np.diag(Hb), rtol=1e-13)
    assert np.array_equal(H, H.T)
    assert np.linalg.eigvalsh(H).min() > -1e-9


def test_kfac_factors_brute_force_and_single_token_kronecker():
    """K-FAC factors: per-token outer products summed by brute force over the
    valid tokens (padding ignored); and with a single token the Kronecker
    product Gamma (x) A equals vec(G) vec(G)^T for G = g a^T, row-major vec
    (the factorisation is exact for one rank-one gradient)."""
    rng = np.random.default_rng(34)
    n, T, d_in, d_out = 3, 5, 6, 4
    a = rng.standard_normal((n, T, d_in))
    g = rng.standard_normal((n, T, d_out))
    L = [5, 2, 0]
    an = np.stack([synth.nan_pad(a[i], L[i]) for i in range(n)])
    gn = np.stack([synth.nan_pad(g[i], L[i]) for i in range(n)])
    A, Gm = O.kfac_factors(an, gn, length=L)
    Ab = np.zeros((d_in, d_in))
    Gb = np.zeros((d_out, d_out))
    for i in range(n):
        for t in range(L[i]):
            for p in range(d_in):
                for q in range(d_in):
                    Ab[p, q] += a[i, t, p] * a[i, t, q]
            for p in range(d_out):
                for q in range(d_out):
                    Gb[p, q] += g[i, t, p] * g[i, t, q]
    np.testing.assert_allclose(A, Ab, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(Gm, Gb, rtol=1e-12, atol=1e-12)
    A1, G1 = O.kfac_factors(a[:1, :1], g[:1, :1])
    G = np.outer(g[0, 0], a[0, 0])
    np.testing.assert_allclose(np.kron(G1, A1), np.outer(G.reshape(-1), G.reshape(-1)), rtol=1e-12)


def test_diag_whitening_unit_second_moment():
    # After the diagonal preconditioner every coordinate has mean square 1.
    rng = np.random.default_rng(18)
    X = rng.standard_normal((400, 20)) * rng.uniform(0.1, 30, size=20)
    X[:, 3] = 0.0                     # a dead coordinate stays at zero
    m = O.finalize_diag(O.accumulate_diag(X), X.shape[0])
    Y = O.precond_apply(X, "diag", m, unit_norm=False)
    ms = (Y * Y).mean(axis=0)
    np.testing.assert_allclose(np.delete(ms, 3), 1.0, rtol=1e-12)
    assert ms[3] == 0.0


def test_full_finalize_identities():
    rng = np.random.default_rng(19)
    X = rng.standard_normal((300, 24)) @ rng.standard_normal((24, 24))
    N = X.shape[0]
    H = O.accumulate_full(X)
    M, _ = O.finalize_full(H, N)
    Hn = H / N
    np.testing.assert_allclose(M @ Hn @ M, np.eye(24), atol=1e-8)
    np.testing.assert_allclose(M @ M, np.linalg.inv(Hn), rtol=1e-7, atol=1e-8)
    # end to end: the second moment of the whitened rows is N * I
    Y = O.precond_apply(X, "full", M, unit_norm=False)
    np.testing.assert_allclose(Y.T @ Y, N * np.eye(24), atol=1e-7 * N)


def test_full_finalize_rank_deficient_is_pseudo_inverse():
    rng = np.random.default_rng(20)
    B = rng.standard_normal((200, 5))
    X = B @ rng.standard_normal((5, 12))      # rank 5 in R^12
    M, lam = O.finalize_full(O.accumulate_full(X), 200)
    assert np.isfinite(M).all()
    # M^2 is the Moore-Penrose pseudo-inverse of Hn
    np.testing.assert_allclose(M @ M, np.linalg.pinv(X.T @ X / 200, rcond=1e-10), rtol=1e-6, atol=1e-8)


def test_lowrank_spectrum_marchenko_pastur():
    # G = Z F^T + 0.1 E: the D - r noise eigenvalues of G^T G / N fill the
    # Marchenko-Pastur bulk 0.01 (1 +- sqrt((D - r)/N))^2 and the r signal
    # eigenvalues sit near those of F F^T.  Scaled-down (D=256, r=8, N=8192).
    D, r, N = 256, 8, 8192
    F = synth.lowrank_factor(D, r, seed=3)
    X = synth.lowrank_rows(0, N, D=D, rank=r, seed=3, chunk=4096, F=F)
    lam = np.sort(np.linalg.eigvalsh(O.accumulate_full(X) / N))
    noise = lam[:D - r]
    ratio = (D - r) / N
    lo, hi = 0.01 * (1 - math.sqrt(ratio)) ** 2, 0.01 * (1 + math.sqrt(ratio)) ** 2
    assert abs(noise.min() - lo) / lo < 0.05 and abs(noise.max() - hi) / hi < 0.05
    sig = lam[D - r:]
    ff = np.sort(np.linalg.eigvalsh(F.T @ F))
    np.testing.assert_allclose(sig, ff, rtol=0.1)


# ----------------------------------------------------------------------------
# scoring and top-k
# ----------------------------------------------------------------------------
def test_topk_golden(golden_dir):
    d = _load(golden_dir, "topk_order.json")
    Q, G = np.array(d["Q"]), np.array(d["G"])
    s, i = O.score_topk(Q, G, 3)
    np.testing.assert_array_equal(s[0], d["k3_scores"])
    np.testing.assert_array_equal(i[0], d["k3_index"])
    s, i = O.score_topk(Q, G, 6)
    np.testing.assert_array_equal(s[0], d["k6_scores"])
    np.testing.assert_array_equal(i[0], d["k6_index"])


def test_topk_brute_force_all_pairs():
    rng = np.random.default_rng(21)
    nq, ng, D, k = 8, 256, 12, 5
    Q = rng.integers(-3, 4, (nq, D)).astype(np.float16)    # small integers: many exact ties
    G = rng.integers(-3, 4, (ng, D)).astype(np.float16)
    s, idx = O.score_topk(Q, G, k, index_base=1000)
    for q in range(nq):
        pairs = []
        for j in range(ng):
            v = sum(float(Q[q, e]) * float(G[j, e]) for e in range(D))
            pairs.append((v, j))
        # selection by repeated extraction of the best remaining (max score,
        # then smallest index)
        chosen = []
        remaining = list(pairs)
        for _ in range(k):
            best = max(remaining, key=lambda p: (p[0], -p[1]))
            chosen.append(best)
            remaining.remove(best)
        assert [c[0] for c in chosen] == list(s[q])
        assert [c[1] + 1000 for c in chosen] == list(idx[q])


def test_self_cosine_and_symmetry():
    x = synth.tiny_inputs()
    P = O.project(x["a"], x["g"], x["R"], x["S"])
    U = O.unit_normalize(P)
    Sm = O.scores(U, U)
    np.testing.assert_allclose(np.diag(Sm), 1.0, atol=1e-12)
    np.testing.assert_allclose(Sm, Sm.T, atol=0)
    assert (np.abs(Sm) <= 1 + 1e-12).all()
    s, idx = O.score_topk(U[:8], U, 5)
    assert (idx[:, 0] == np.arange(8)).all()


def test_merge_equals_single_pass_and_is_associative():
    rng = np.random.default_rng(22)
    Q = rng.standard_normal((6, 16))
    G = rng.standard_normal((500, 16))
    G[100] = G[7]                     # an exact tie across chunks
    k = 9
    ref_s, ref_i = O.score_topk(Q, G, k)
    s, i = O.score_topk(Q, G[:0], k)
    assert (i == -1).all() and np.isneginf(s).all()
    for lo in range(0, 500, 130):
        hi = min(500, lo + 130)
        cs, ci = O.score_topk(Q, G[lo:hi], k, index_base=lo)
        s, i = O.merge_topk(s, i, cs, ci, k)
    np.testing.assert_array_equal(s, ref_s)
    np.testing.assert_array_equal(i, ref_i)


def test_fewer_candidates_than_k_and_nan():
    Q = np.array([[1.0, 0.0]])
    G = np.array([[np.nan, 0.0], [2.0, 0.0]])
    s, i = O.score_topk(Q, G, 4)
    assert list(i[0]) == [1, -1, -1, -1]
    assert s[0, 0] == 2.0 and np.isneginf(s[0, 1:]).all()


def test_infinite_scores_selection_rule():
    # +inf ranks first (ties by index); -inf and NaN are never selected and
    # leave (-inf, -1) padding, so a selected entry is always finite or +inf.
    Q = np.array([[1.0, 1.0]])
    G = np.array([[np.inf, 0.0], [1.0, 0.0], [-np.inf, 0.0], [np.nan, 0.0],
                  [np.inf, 1.0], [-np.inf, 5.0], [0.5, 0.0]])
    s, i = O.score_topk(Q, G, 6)
    assert list(i[0]) == [0, 4, 1, 6, -1, -1]
    assert list(s[0][:4]) == [np.inf, np.inf, 1.0, 0.5]
    assert np.isneginf(s[0, 4:]).all()
    # merging keeps the rule: a list holding only -inf candidates adds nothing
    s2, i2 = O.merge_topk(s, i, np.array([[-np.inf, 2.0]]), np.array([[9, 10]]), 6)
    assert list(i2[0]) == [0, 4, 10, 1, 6, -1]
