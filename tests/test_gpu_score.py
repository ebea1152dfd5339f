"""GPU parity of attr_score_topk (and the tiny end-to-end pipeline) against
the fp64 oracle: scores within 1e-3, indices exact wherever the score gaps
exceed 1e-3, ties ordered by index, padding (-inf, -1)."""
import numpy as np
import pytest
import torch

import oracle as O
import paper_2606_11660_amd as P
import synth
from tests._util import check_topk, dev, host, say

pytestmark = pytest.mark.gpu


def _topk(Q, G, k, index_base=0, merge=False, prev=None):
    nq = Q.shape[0]
    if prev is None:
        ts = torch.full((nq, k), 5.0, dtype=torch.float32, device="cuda")
        ti = torch.full((nq, k), 7, dtype=torch.int64, device="cuda")
    else:
        ts, ti = prev
    P.attr_score_topk(Q, G, k, ts, ti, index_base=index_base, merge=merge)
    torch.cuda.synchronize()
    return ts, ti


def test_tiny_pipeline_end_to_end():
    """Tiny workload: project (fp32) -> unit-normalise -> score 8 queries -> top-5."""
    say("case: tiny end-to-end")
    x = synth.tiny_inputs()
    k = 16

    def rows(a, g, n):
        out = torch.empty((n, k * k), dtype=torch.float32, device="cuda")
        m = [P.Module(dev(a.reshape(-1, 64)), dev(g.reshape(-1, 64)), dev(x["R"]), dev(x["S"]), 0)]
        P.attr_project(m, k, n, 32, out)
        y = torch.empty_like(out)
        P.attr_precond_apply(out, P.PRECOND_NONE, None, True, y)
        return y

    G = rows(x["a"], x["g"], 256)
    Q = rows(x["aq"], x["gq"], 8)
    ts, ti = _topk(Q, G, 5)
    Gr = O.unit_normalize(O.project(x["a"], x["g"], x["R"], x["S"]))
    Qr = O.unit_normalize(O.project(x["aq"], x["gq"], x["R"], x["S"]))
    check_topk(host(ts), host(ti), O.scores(Qr, Gr), 5)
    rs, ri = O.score_topk(Qr, Gr, 5)
    assert np.abs(host(ts) - rs).max() <= 1e-5


def test_on_the_fly_scoring_without_a_store():
    """On-the-fly scoring (training gradients scored against the queries as
    they are produced, no store kept): per batch of 16 examples, project ->
    unit-normalise to fp16 -> score with the running top-k merged; after four
    batches the lists match the oracle's top-k over all 64 examples."""
    say("case: on-the-fly scoring")
    rng = np.random.default_rng(81)
    k_proj, T, B, nb, nq, k = 16, 64, 16, 4, 12, 8
    shapes = [(64, 128), (128, 64), (64, 64)]
    D = len(shapes) * k_proj * k_proj
    RS = [(synth.to_bf16_bits(rng.standard_normal((d_out, k_proj)) / 4),
           synth.to_bf16_bits(rng.standard_normal((d_in, k_proj)) / 4)) for d_in, d_out in shapes]

    def batch(nex):
        return [(synth.to_bf16_bits(rng.standard_normal((nex * T, d_in))),
                 synth.to_bf16_bits(rng.standard_normal((nex * T, d_out)) * 1e-2)) for d_in, d_out in shapes]

    def rows_fp16(ag):
        out = torch.empty((ag[0][0].shape[0] // T, D), dtype=torch.float32, device="cuda")
        mods = [P.Module(dev(a), dev(g), dev(R), dev(S), m * k_proj * k_proj)
                for m, ((a, g), (R, S)) in enumerate(zip(ag, RS))]
        P.attr_project(mods, k_proj, out.shape[0], T, out)
        y = torch.empty(out.shape, dtype=torch.float16, device="cuda")
        P.attr_precond_apply(out, P.PRECOND_NONE, None, True, y)
        return y

    def oracle_rows(ag):
        blocks = [O.project(a.reshape(-1, T, a.shape[1]), g.reshape(-1, T, g.shape[1]), R, S)
                  for (a, g), (R, S) in zip(ag, RS)]
        return O.to_f16(O.unit_normalize(O.project_concat(blocks)))

    qb = batch(nq)
    Qd = rows_fp16(qb)
    ts = torch.empty((nq, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((nq, k), dtype=torch.int64, device="cuda")
    train = []
    for b in range(nb):
        tb = batch(B)
        train.append(tb)
        P.attr_score_topk(Qd, rows_fp16(tb), k, ts, ti, index_base=b * B, merge=b > 0)
    torch.cuda.synchronize()
    Gr = np.concatenate([oracle_rows(tb) for tb in train])
    check_topk(host(ts), host(ti), O.scores(oracle_rows(qb), Gr), k)


def test_per_token_attribution():
    """Per-token attribution: the training batch's per-token compressed
    gradients (attr_project_tokens, packed valid tokens), unit-normalised to
    fp16, scored against per-sequence queries; the top tokens per query
    match the oracle's top-k over all valid tokens."""
    say("case: per-token attribution")
    rng = np.random.default_rng(82)
    k_proj, T, nq, k = 16, 96, 6, 10
    lengths = [96, 40, 73, 1]
    n = len(lengths)
    shapes = [(64, 128), (128, 64)]
    D = len(shapes) * k_proj * k_proj
    RS = [(synth.to_bf16_bits(rng.standard_normal((d_out, k_proj)) / 4),
           synth.to_bf16_bits(rng.standard_normal((d_in, k_proj)) / 4)) for d_in, d_out in shapes]
    ag = [(synth.to_bf16_bits(rng.standard_normal((n, T, d_in))),
           synth.to_bf16_bits(rng.standard_normal((n, T, d_out)))) for d_in, d_out in shapes]
    offs = np.concatenate([[0], np.cumsum(lengths)[:-1]]).astype(np.int64)
    tot = int(sum(lengths))
    mods = []
    for m, ((a, g), (R, S)) in enumerate(zip(ag, RS)):
        a_pk = np.concatenate([a[i, :lengths[i]] for i in range(n)])
        g_pk = np.concatenate([g[i, :lengths[i]] for i in range(n)])
        mods.append(P.Module(dev(a_pk), dev(g_pk), dev(R), dev(S), m * k_proj * k_proj))
    rows = torch.empty((tot, D), dtype=torch.float32, device="cuda")
    P.attr_project_tokens(mods, k_proj, n, T, rows, row_offset=torch.from_numpy(offs).cuda(),
                          length=torch.from_numpy(np.asarray(lengths, dtype=np.int32)).cuda())
    G16 = torch.empty((tot, D), dtype=torch.float16, device="cuda")
    P.attr_precond_apply(rows, P.PRECOND_NONE, None, True, G16)
    Q = synth.unit_rows(nq, D, seed=83)
    ts, ti = _topk(dev(Q), G16, k)
    blocks = [O.project_tokens(a, g, R, S, length=lengths) for (a, g), (R, S) in zip(ag, RS)]
    tok = O.project_concat([b.reshape(n * T, -1) for b in blocks]).reshape(n, T, D)
    Gr = O.to_f16(O.unit_normalize(np.concatenate([tok[i, :lengths[i]] for i in range(n)])))
    check_topk(host(ts), host(ti), O.scores(Q, Gr), k)


@pytest.mark.parametrize("k", [1, 10, 100])
def test_random_unit_rows_f16(k):
    nq, ng, D = 70, 1000, 128            # two query blocks, ragged store tile
    say(f"case: random fp16 nq={nq} ng={ng} D={D} k={k}")
    Q = synth.unit_rows(nq, D, seed=11)
    G = synth.unit_rows(ng, D, seed=12)
    ts, ti = _topk(dev(Q), dev(G), k, index_base=1000)
    check_topk(host(ts), host(ti), O.scores(Q, G), k, index_base=1000)


def test_exact_ties_index_order_and_self_cosine():
    say("case: duplicates / ties")
    D = 64
    base = synth.unit_rows(40, D, seed=13)
    G = np.concatenate([base, base[:10], base[5:15]])     # rows 40..59 duplicate rows 0..14
    Q = base[:12]
    ts, ti = _topk(dev(Q), dev(G), 3)
    ref_s, ref_i = O.score_topk(Q, G, 3)
    gi = host(ti)
    # the top entries are exact duplicates of the query: equal scores, index ascending
    np.testing.assert_array_equal(gi, ref_i)
    assert np.abs(host(ts) - ref_s).max() <= 1e-3
    assert np.abs(host(ts)[:, 0] - 1.0).max() <= 2e-3      # self-cosine


def test_symmetric_scores_f32():
    say("case: Q == G symmetric, fp32")
    X = synth.unit_rows(96, 256, seed=14, dtype=np.float32)
    ts, ti = _topk(dev(X), dev(X), 96)
    S = np.full((96, 96), np.nan)
    for q in range(96):
        S[q, host(ti)[q]] = host(ts)[q]
    np.testing.assert_allclose(S, S.T, atol=1e-6)
    np.testing.assert_allclose(np.diag(S), 1.0, atol=1e-5)


def test_merge_chunks_equals_single_call():
    say("case: merge chunks")
    nq, ng, D, k = 33, 3000, 192, 20
    Q = synth.unit_rows(nq, D, seed=15)
    G = synth.unit_rows(ng, D, seed=16)
    G[2500] = G[100]                   # tie across chunks
    Qd, Gd = dev(Q), dev(G)
    s1, i1 = _topk(Qd, Gd, k)
    ts = torch.empty((nq, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((nq, k), dtype=torch.int64, device="cuda")
    P.attr_score_topk(Qd, Gd[:0], k, ts, ti, merge=False)     # empty store -> padding
    torch.cuda.synchronize()
    assert (host(ti) == -1).all() and np.isneginf(host(ts)).all()
    for lo in range(0, ng, 700):
        hi = min(ng, lo + 700)
        P.attr_score_topk(Qd, Gd[lo:hi], k, ts, ti, index_base=lo, merge=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(ti), host(i1))
    np.testing.assert_array_equal(host(ts), host(s1))
    check_topk(host(ts), host(ti), O.scores(Q, G), k)


@pytest.mark.parametrize("k", [10, 128])
def test_merge_small_batches_like_the_bench(k):
    """The bench's pattern: 64-row batches scored and merged into the running
    list (split-K plan with at most 256 rows: fused select and merge), with
    NaN and duplicate rows; equals one call over the whole store."""
    say(f"case: merge 64-row batches k={k}")
    nq, ng, D = 64, 640, 12288
    Q = synth.unit_rows(nq, D, seed=51)
    G = synth.unit_rows(ng, D, seed=52)
    G[600] = G[5]                          # tie across batches
    Q[3] = G[5]
    G[70] = np.nan                         # never selected
    Qd, Gd = dev(Q), dev(G)
    ts = torch.empty((nq, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((nq, k), dtype=torch.int64, device="cuda")
    for b in range(0, ng, 64):
        P.attr_score_topk(Qd, Gd[b:b + 64], k, ts, ti, index_base=b, merge=b > 0)
    torch.cuda.synchronize()
    ref = O.scores(Q, G)
    ref[:, 70] = -np.inf
    gi = host(ti)
    assert not (gi == 70).any()
    check_topk(host(ts), gi, ref, k)
    assert gi[3, 0] == 5 and gi[3, 1] == 600


@pytest.mark.parametrize("nq,ng,D,k,dt,chunk", [(70, 3001, 1024, 100, np.float16, 1000),
                                                (20, 5000, 2048, 10, np.float32, 5000),
                                                (64, 4096, 12288, 128, np.float16, 4096),
                                                (5, 300, 1024, 33, np.float16, 300),
                                                (64, 20000, 2048, 100, np.float16, 12000),
                                                (30, 17000, 1024, 10, np.float32, 17000)])
def test_split_plan_select(nq, ng, D, k, dt, chunk):
    """Small stores (split-K partial slices, one selection workgroup per
    query and part of at most 8192 rows, part lists merged when there are
    several): ragged query blocks and row counts, a NaN row, an exact tie
    across chunks, chunks merged into the running list."""
    say(f"case: split plan nq={nq} ng={ng} D={D} k={k} {dt.__name__} chunk={chunk}")
    Q = synth.unit_rows(nq, D, seed=61, dtype=dt)
    G = synth.unit_rows(ng, D, seed=62, dtype=dt)
    G[ng - 2] = G[7]
    Q[1] = G[7]
    G[ng // 2] = np.nan
    Qd, Gd = dev(Q), dev(G)
    ts = torch.empty((nq, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((nq, k), dtype=torch.int64, device="cuda")
    for lo in range(0, ng, chunk):
        P.attr_score_topk(Qd, Gd[lo:lo + chunk], k, ts, ti, index_base=lo, merge=lo > 0)
    torch.cuda.synchronize()
    ref = O.scores(Q, G)
    ref[:, ng // 2] = -np.inf
    gi = host(ti)
    assert not (gi == ng // 2).any()
    check_topk(host(ts), gi, ref, k)
    assert gi[1, 0] == 7 and gi[1, 1] == ng - 2


def test_split_plan_all_ties_fallback():
    """Every row equal to every query: 2033 or more rows reach the k-th best
    16-row segment maximum at k = 128, past the gather capacity, so the list
    comes from k rounds of arg-max; merged with a second call on the same
    rows (all ties again), the lowest indices win."""
    nq, ng, D, k = 3, 3000, 2048, 128
    say("case: split plan, all ties")
    row = synth.unit_rows(1, D, seed=63)
    Gd = dev(np.repeat(row, ng, axis=0))
    Qd = dev(np.repeat(row, nq, axis=0))
    ts = torch.empty((nq, k), dtype=torch.float32, device="cuda")
    ti = torch.empty((nq, k), dtype=torch.int64, device="cuda")
    P.attr_score_topk(Qd, Gd, k, ts, ti, index_base=5000)
    P.attr_score_topk(Qd, Gd, k, ts, ti, index_base=10, merge=True)
    torch.cuda.synchronize()
    assert (host(ti) == np.arange(k)[None, :] + 10).all()
    sc = host(ts)
    assert (sc == sc[:, :1]).all() and np.abs(sc - 1.0).max() <= 1e-3


def test_fewer_rows_than_k():
    say("case: n_g < k")
    Q = synth.unit_rows(5, 64, seed=17)
    G = synth.unit_rows(7, 64, seed=18)
    ts, ti = _topk(dev(Q), dev(G), 12)
    check_topk(host(ts), host(ti), O.scores(Q, G), 12)


def test_planted_near_duplicates():
    say("case: planted near-duplicates D=8192")
    ng, D, nq = 20000, 8192, 64
    G = synth.unit_rows(ng, D, seed=19)
    targets = np.random.default_rng(4).choice(ng, 16, replace=False)
    Q = synth.planted_queries(G[targets], targets, nq)
    ts, ti = _topk(dev(Q), dev(G), 100)
    gi, gs = host(ti), host(ts)
    assert (gi[:16, 0] == targets).all()
    assert np.abs(gs[:16, 0] - 0.9).max() <= 2e-3
    check_topk(gs, gi, O.scores(Q, G), 100)


def test_gpt2_store_scan():
    """GPT-2-shaped scoring: 64 queries x 4096 store rows x 12288 dims, top-10."""
    say("case: gpt2 store scan")
    Q = synth.unit_rows(64, 12288, seed=21)
    G = synth.unit_rows(4096, 12288, seed=22)
    ts, ti = _topk(dev(Q), dev(G), 10)
    check_topk(host(ts), host(ti), O.scores(Q, G), 10)


@pytest.mark.parametrize("nq,ng,D,k,dt", [(100, 9000, 256, 100, np.float16),
                                          (40, 40001, 128, 10, np.float16),
                                          (70, 33000, 96, 5, np.float32),
                                          (17, 70000, 64, 128, np.float16),
                                          (50, 30000, 256, 32, np.float16),
                                          (50, 30000, 256, 33, np.float16),
                                          (9, 30000, 64, 64, np.float32),
                                          (12, 50000, 128, 100, np.float16),
                                          (16, 20000, 256, 65, np.float16),
                                          (32, 30000, 128, 128, np.float16),
                                          (20, 30000, 64, 128, np.float32)])
def test_streaming_plan(nq, ng, D, k, dt):
    """Shapes large enough for the streaming (LDS-ring) plan: ragged query
    blocks, ragged partitions and tiles, duplicate rows, fp32 and fp16."""
    say(f"case: streaming nq={nq} ng={ng} D={D} k={k} {dt.__name__}")
    Q = synth.unit_rows(nq, D, seed=31, dtype=dt)
    G = synth.unit_rows(ng, D, seed=32, dtype=dt)
    G[ng - 5] = G[3]                       # exact tie far apart
    Q[0] = G[3]
    ts, ti = _topk(dev(Q), dev(G), k, index_base=7)
    check_topk(host(ts), host(ti), O.scores(Q, G), k, index_base=7)
    assert host(ti)[0, 0] == 3 + 7 and host(ti)[0, 1] == ng - 5 + 7


@pytest.mark.parametrize("nq,k,D,dt", [(64, 100, 64, np.float16), (20, 64, 128, np.float16),
                                       (64, 16, 256, np.float16), (24, 65, 64, np.float32)])
def test_streaming_plan_with_bound(nq, k, D, dt):
    """Stores of 262144 rows or more with n_q * k >= 1024 take a lower bound
    on each query's k-th best score from the first 16384 rows before the
    scan: random unit rows, ragged last partition."""
    ng = 300001
    say(f"case: streaming with bound nq={nq} ng={ng} D={D} k={k} {dt.__name__}")
    Q = synth.unit_rows(nq, D, seed=41, dtype=dt)
    G = synth.unit_rows(ng, D, seed=42, dtype=dt)
    ts, ti = _topk(dev(Q), dev(G), k, index_base=3)
    check_topk(host(ts), host(ti), O.scores(Q, G), k, index_base=3)


@pytest.mark.parametrize("nq,ng,D,k,n_pinf,dt", [
    (8, 200, 256, 10, 3, np.float16),        # split-K, one selection wave per query
    (40, 3001, 1024, 50, 3, np.float16),     # split-K, several parts + merge
    (100, 9000, 256, 100, 3, np.float16),    # streaming
    (20, 9000, 128, 10, 3, np.float32),      # streaming, fp32
    (64, 300001, 64, 100, 3, np.float16),    # streaming with the prefix bound
    (120, 300001, 64, 9, 12, np.float16),    # bound itself +inf: only +inf rows enter
    (130, 5000, 256, 10, 3, np.float16),     # GEMM plan
    (200, 300000, 64, 2, 3, np.float16),     # GEMM plan, running bound +inf after chunk 0
])
def test_infinite_and_nan_store_rows(nq, ng, D, k, n_pinf, dt):
    """Store rows scoring +inf rank first, by index; rows scoring -inf or
    NaN are never selected (the oracle's selection rule), on every plan."""
    say(f"case: +-inf / NaN rows nq={nq} ng={ng} D={D} k={k} n_pinf={n_pinf} {dt.__name__}")
    Q = synth.unit_rows(nq, D, seed=71, dtype=dt)
    Q[:, 0] = np.abs(Q[:, 0]) + dt(0.05)         # every query positive on column 0
    G = synth.unit_rows(ng, D, seed=72, dtype=dt)
    rng = np.random.default_rng(73)
    # +inf rows in distinct 64-row segments of the first 16384 rows (and one
    # late row), -inf and NaN rows spread over the store
    pinf = sorted(set((rng.choice(min(ng, 16384) // 64, n_pinf - 1, replace=False) * 64 + 7).tolist())
                  | {ng - 3})
    rest = np.setdiff1d(np.arange(ng), pinf)
    ninf = rng.choice(rest, 4, replace=False)
    nan = rng.choice(np.setdiff1d(rest, ninf), 3, replace=False)
    G[pinf, 0] = np.inf
    G[ninf, 0] = -np.inf
    G[nan, 1] = np.nan
    ts, ti = _topk(dev(Q), dev(G), k, index_base=5)
    got_s, got_i = host(ts), host(ti)
    finite = np.ones(ng, dtype=bool)
    finite[pinf] = finite[ninf] = finite[nan] = False
    Gf = G.copy()
    Gf[~finite] = 0
    sc = O.scores(Q, Gf)
    sc[:, ~finite] = -1e30                       # never among a finite top-k
    ref_s, ref_i = O.score_topk(Q, G, k, index_base=5)
    npos = min(k, len(pinf))
    # the +inf rows: exact scores and index order
    np.testing.assert_array_equal(got_i[:, :npos], ref_i[:, :npos])
    assert np.isposinf(got_s[:, :npos]).all() and np.isposinf(ref_s[:, :npos]).all()
    # the rest: the top (k - npos) of the finite rows, by the usual gap rule
    if k > npos:
        check_topk(got_s[:, npos:], got_i[:, npos:], sc, k - npos, index_base=5)
    bad = set((np.concatenate([ninf, nan]) + 5).tolist())
    assert not (set(got_i.ravel().tolist()) & bad)


def test_merge_fallback_all_ties():
    """Every store row equal and the query equal to it: all scores tie, each
    partition list holds its first k rows, and nearly every list entry ranks
    at or above the k-th best list head, which overflows the merge's
    gather-and-sort buffer; the k-round arg-max fallback must still return
    rows 0..k-1 in index order."""
    nq, ng, D, k = 4, 40000, 64, 100
    say("case: merge fallback, all rows tie")
    row = synth.unit_rows(1, D, seed=45)
    G = np.repeat(row, ng, axis=0)
    Q = np.repeat(row, nq, axis=0)
    ts, ti = _topk(dev(Q), dev(G), k, index_base=11)
    assert (host(ti) == np.arange(k)[None, :] + 11).all()
    s = host(ts)
    assert (s == s[:, :1]).all() and np.abs(s - 1.0).max() <= 1e-3


def test_streaming_bound_ties_at_the_bound():
    """Query 0 equals store row A, copied into 16 distinct 64-row segments of
    the 16384-row prefix (plus the original in the first) and 40 times beyond
    it: the 16th largest segment maximum, the bound, is exactly A's score,
    and the top 16 are the lowest-index copies, every one scoring exactly the
    bound (a strict comparison against the bound itself would drop them)."""
    nq, ng, D, k = 64, 300000, 64, 16
    say("case: streaming bound with ties at the bound")
    G = synth.unit_rows(ng, D, seed=43)
    A = G[7].copy()
    pre = [64 * s + (13 * s) % 64 for s in range(0, 256, 16)]
    post = list(range(20000, 290000, 6750))[:40]
    for r in pre + post:
        G[r] = A
    Q = synth.unit_rows(nq, D, seed=44)
    Q[0] = A
    ts, ti = _topk(dev(Q), dev(G), k)
    want = sorted(set(pre + [7]))[:k]
    assert host(ti)[0].tolist() == want
    s0 = host(ts)[0]
    assert (s0 == s0[0]).all() and abs(s0[0] - 1.0) <= 1e-3
    check_topk(host(ts)[1:], host(ti)[1:], O.scores(Q[1:], G), k)


# ---------------------------------------------------------------------------
# GEMM plan (fp16, n_q >= 128, n_g >= 4096): chunked score matrix + exact
# per-chunk selection
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("nq,ng,D,k", [(130, 5000, 256, 10), (300, 9000, 256, 100),
                                       (257, 4100, 64, 128), (128, 5000, 256, 10),
                                       (128, 4097, 128, 5), (384, 6000, 192, 50),
                                       (128, 530000, 64, 100)])
def test_gemm_plan(nq, ng, D, k):
    """256 x 256 tiles (130 queries) and 128-query x 256-row ring tiles (128,
    257, 300, 384 queries): ragged query tiles, ragged row tiles whose last
    workgroup has waves without rows (4097 = 16 x 256 + 1: one row in wave 0;
    5000 = 19 x 256 + 136: 8 rows in wave 2, none in wave 3), one and three
    stages (D = 64, 192: fewer stages than ring slots), three chunks of at
    most 262144 rows with the running bound (530000 rows); a tie far apart, a
    NaN row that must never be selected."""
    say(f"case: gemm plan nq={nq} ng={ng} D={D} k={k}")
    Q = synth.unit_rows(nq, D, seed=41)
    G = synth.unit_rows(ng, D, seed=42)
    G[ng - 5] = G[3]
    Q[0] = G[3]
    G[17] = np.nan
    ts, ti = _topk(dev(Q), dev(G), k, index_base=11)
    ref = O.scores(Q, G)
    ref[:, 17] = -np.inf                  # NaN is never selected
    gi = host(ti)
    assert not (gi == 17 + 11).any()
    check_topk(host(ts), gi, ref, k, index_base=11)
    assert gi[0, 0] == 3 + 11 and gi[0, 1] == ng - 5 + 11


def test_gemm_plan_several_chunks():
    """8192 queries make 8192-row chunks: a 20000-row store is three chunks
    (the last ragged); sampled queries are checked against the oracle, and
    the result equals two merged calls."""
    say("case: gemm plan, three chunks")
    nq, ng, D, k = 8192, 20000, 64, 16
    Q = synth.unit_rows(nq, D, seed=43)
    G = synth.unit_rows(ng, D, seed=44)
    G[19990] = G[5]                       # tie across chunks
    Q[7] = G[5]
    Qd, Gd = dev(Q), dev(G)
    ts, ti = _topk(Qd, Gd, k)
    sample = np.r_[0:8, 4000:4008, nq - 8:nq]
    check_topk(host(ts)[sample], host(ti)[sample], O.scores(Q[sample], G), k)
    assert host(ti)[7, 0] == 5 and host(ti)[7, 1] == 19990
    ts2 = torch.empty_like(ts)
    ti2 = torch.empty_like(ti)
    P.attr_score_topk(Qd, Gd[:9000], k, ts2, ti2)
    P.attr_score_topk(Qd, Gd[9000:], k, ts2, ti2, index_base=9000, merge=True)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(ti2), host(ti))
    np.testing.assert_array_equal(host(ts2), host(ts))


def test_gemm_plan_all_ties():
    """Every score equal: more than 2048 rows pass any threshold, so the
    exact arg-max selection runs; ties resolve to the lowest indices."""
    say("case: gemm plan, all scores tied")
    nq, ng, D, k = 128, 5000, 64, 20
    row = synth.unit_rows(1, D, seed=45)
    G = np.repeat(row, ng, axis=0)
    Q = synth.unit_rows(nq, D, seed=46)
    ts, ti = _topk(dev(Q), dev(G), k)
    np.testing.assert_array_equal(host(ti), np.tile(np.arange(k), (nq, 1)))
    ref = O.scores(Q, G[:1])
    assert np.abs(host(ts) - ref).max() <= 1e-3


def test_gemm_plan_misleading_sample():
    """Rows at the sampled positions (every 4th of 8192) score 0, the others
    1: the sampled threshold passes 8192 rows, so the exact fallback must
    return the first k rows scoring 1."""
    say("case: gemm plan, sample-adversarial store")
    nq, ng, D, k = 128, 8192, 64, 100
    e0 = np.zeros(D, dtype=np.float16); e0[0] = 1
    e1 = np.zeros(D, dtype=np.float16); e1[1] = 1
    G = np.where((np.arange(ng) % 4 == 0)[:, None], e1, e0).astype(np.float16)
    Q = np.tile(e0, (nq, 1))
    ts, ti = _topk(dev(Q), dev(G), k)
    want = np.flatnonzero(np.arange(ng) % 4 != 0)[:k]
    np.testing.assert_array_equal(host(ti), np.tile(want, (nq, 1)))
    assert (host(ts) == 1.0).all()


def _banded_store(ng, D, chunk, weights, seed):
    """Rows r of chunk c: weights[c] * e0 + sqrt(1 - weights[c]^2) * (random
    unit direction orthogonal to e0), fp16."""
    R = synth.unit_rows(ng, D, seed=seed).astype(np.float64)
    R[:, 0] = 0
    R /= np.linalg.norm(R, axis=1, keepdims=True)
    w = np.asarray(weights, dtype=np.float64)[np.arange(ng) // chunk]
    G = w[:, None] * np.eye(1, D)[0] + np.sqrt(1 - w ** 2)[:, None] * R
    return G.astype(np.float16)


@pytest.mark.parametrize("order", ["rising", "falling"])
def test_gemm_plan_running_bound(order):
    """8192 queries make 8192-row chunks.  Rising: every row of a later chunk
    beats the bound of the earlier ones (more than 2048 candidates: the
    sampled threshold above the bound is used).  Falling: nothing after the
    first chunk beats it (empty chunk lists, segments not written) except one
    planted copy of a query in the last chunk, which must rank first."""
    say(f"case: gemm plan running bound, {order} store")
    nq, D, k, chunk = 8192, 64, 100, 8192
    ng = 3 * chunk - 100
    w = [0.1, 0.5, 0.9] if order == "rising" else [0.9, 0.5, 0.1]
    G = _banded_store(ng, D, chunk, w, seed=61)
    Q = synth.unit_rows(nq, D, seed=62).astype(np.float64)
    Q[:, 0] = 0
    Q = 0.8 * np.eye(1, D)[0] + 0.6 * Q / np.linalg.norm(Q, axis=1, keepdims=True)
    Q = Q.astype(np.float16)
    if order == "falling":
        G[ng - 7] = Q[5]
    ts, ti = _topk(dev(Q), dev(G), k)
    sample = np.r_[0:6, 4000:4004, nq - 6:nq]
    check_topk(host(ts)[sample], host(ti)[sample], O.scores(Q[sample], G), k)
    if order == "rising":
        assert (host(ti)[sample] >= 2 * chunk).all()
    else:
        assert host(ti)[5, 0] == ng - 7
        assert (host(ti)[sample][:, 1:] < chunk).all()


@pytest.mark.parametrize("ragged", [False, True])
def test_bench_two_stream_step_matches_one_stream(ragged):
    """The bench step pipelines over two streams (projection of batch i + 1
    while batch i is normalised and scored; two fp32 row buffers ordered by
    events).  Every call is deterministic, so the store rows and the running
    top-k after 5 pipelined steps equal, bitwise, the same calls issued one
    after another on one stream.  ragged: the steps cycle over two packed
    batches of ragged lengths (row_offset / length), as the headline does."""
    import bench
    say(f"case: two-stream bench step vs one stream, 5 steps, ragged={ragged}")
    rng = np.random.default_rng(91)
    k, B, T, steps, topk = 16, 8, 96, 5, 7
    shapes = [(64, 192), (128, 64), (64, 128)]
    D = len(shapes) * k * k
    mods = []
    for m, (d_in, d_out) in enumerate(shapes):
        a = torch.from_numpy(synth.to_bf16_bits(rng.standard_normal((B * T, d_in))).view(np.int16)).view(torch.bfloat16).cuda()
        g = torch.from_numpy(synth.to_bf16_bits(rng.standard_normal((B * T, d_out))).view(np.int16)).view(torch.bfloat16).cuda()
        R = torch.from_numpy(synth.to_bf16_bits(rng.standard_normal((d_out, k)) / 4).view(np.int16)).view(torch.bfloat16).cuda()
        S = torch.from_numpy(synth.to_bf16_bits(rng.standard_normal((d_in, k)) / 4).view(np.int16)).view(torch.bfloat16).cuda()
        mods.append(P.Module(a, g, R, S, m * k * k))
    Qrows = torch.from_numpy(rng.standard_normal((6, D)).astype(np.float16)).cuda()
    batches = None
    if ragged:
        batches = []
        for lens in ([96, 0, 17, 64, 95, 1, 33, 80], [5, 96, 96, 96, 2, 60, 0, 70]):
            offs = np.concatenate([[0], np.cumsum(lens)[:-1]])
            batches.append((torch.from_numpy(offs.astype(np.int64)).cuda(),
                            torch.from_numpy(np.asarray(lens, dtype=np.int32)).cuda()))
    results = []
    for two in (True, False):
        s1 = torch.cuda.Stream()
        s2 = torch.cuda.Stream() if two else s1
        store = torch.full((steps * B, D), float("nan"), dtype=torch.float16, device="cuda")
        rows = [torch.empty((B, D), dtype=torch.float32, device="cuda") for _ in range(2)]
        top_s = torch.empty((6, topk), dtype=torch.float32, device="cuda")
        top_i = torch.empty((6, topk), dtype=torch.int64, device="cuda")
        ws = [P.Workspace("cuda") for _ in range(3)]
        pd, nd = bench._pipeline_events(s2)
        bench.run_pipeline(mods, k, B, T, rows, store, Qrows, topk, top_s, top_i, 0, steps, s1, s2,
                           ws[0], ws[1], ws[2], pd, nd, batches=batches)
        s1.synchronize()
        s2.synchronize()
        results.append((host(store), host(top_s), host(top_i)))
    (st2, ts2, ti2), (st1, ts1, ti1) = results
    assert np.isfinite(st2).all()
    if ragged:   # a zero-length example stores a zero row, never NaN
        assert (st2[1] == 0).all() and (st2[B + 6] == 0).all()
    assert np.array_equal(st2.view(np.uint16), st1.view(np.uint16))
    assert np.array_equal(ts2, ts1) and np.array_equal(ti2, ti1)
    assert (ti2 >= 0).all() and (ti2 < steps * B).all()
