"""Throughput of the attribution hot path on one MI355X.

Headline workload (1B-decoder-shaped gradient store build with on-the-fly
scoring): 16 layers x 7 linear modules (q, k, v, o 2048->2048; gate, up
2048->8192; down 8192->2048), k = 16 per module (28672 dims per row),
per-example lengths uniform in [256, 2048] with the tokens of a batch packed
back to back (padding never stored or read), bf16 token rows resident in
HBM, fp16 store, 64 query rows with the running top-10.  One step is one
batch of 32 examples through the whole path:

  attr_project        (bf16 token rows of 112 modules -> fp32 rows)
  attr_precond_apply  (unit-normalise, cast to the fp16 store slot)
  attr_score_topk     (64 queries x the 32 new rows, merged into the
                       running top-10 of the store built so far)

The steps cycle through eight batches of the length law (examples 0..255),
each packed from the start of one resident token buffer, so the work per
step follows the workload's length distribution.  `value` is examples/s
over the timed steps.  The dominant kernel is the projection; its roofline
entry uses the algorithmic bytes of one call (every valid token's a/g
element once, R/S once, the fp32 output rows) averaged over the timed steps,
over the average call duration measured with HIP events on the projection's
stream.  `rows` reports every other row of the path on its own (each the
median of >= 10 timed calls after >= 3 warm-up calls), `peaks` the HBM read
rate and fp16 matrix-core rate this GPU sustains (calibration kernels), and
`cpu_baseline` the fp64 oracle on a bounded sample of the headline workload
on the host cores, with labelled oracle timings of the other workloads.

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--quick]
       [--no-cpu-baseline] [--profile-row ROW] [--copy-reference]
"""
from __future__ import annotations

import argparse
import json
import os
import platform
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0   # dense fp16 / bf16
BATCH = 32                  # examples per headline step
N_BATCHES = 8               # distinct length vectors the steps cycle through
N_QUERIES, TOPK = 64, 10
PROFILE_REPS = 3            # each --profile-row operation runs this often (the first call is cold)


# ----------------------------------------------------------------------------
# timing helpers
# ----------------------------------------------------------------------------
def _median_ms(fn, stream, reps=10, warmup=3):
    """Median over `reps` calls of fn's duration on `stream` (HIP events
    around each call), after `warmup` untimed calls."""
    import torch
    with torch.cuda.stream(stream):
        for _ in range(warmup):
            fn()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(reps)]
        for a, b in ev:
            a.record(stream)
            fn()
            b.record(stream)
    stream.synchronize()
    return statistics.median(a.elapsed_time(b) for a, b in ev)


def _hbm(bytes_, ms):
    gbps = bytes_ / ms / 1e6
    return {"GBps": gbps, "frac_hbm": gbps / HBM_PEAK_GBPS}


def _mfma(flops, ms):
    tf = flops / ms / 1e9
    return {"TFLOPs": tf, "frac_mfma": tf / MFMA_PEAK_TFLOPS}


# ----------------------------------------------------------------------------
# workload builders (timing buffers: values drawn on the device, seeded)
# ----------------------------------------------------------------------------
def _dev_bf16(a):
    import numpy as np
    import torch
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)


def _llama1b_modules(dev, rows, variant="separate", seed=1):
    """The 112 modules of the 1B-shaped model over `rows` resident token rows
    (bf16, device-filled: a ~ N(0,1), g ~ N(0,1) 1e-2; values do not change
    the work), R and S from the seeded host generator.  variant "separate":
    every module reads its own a; "shared": q/k/v and gate/up of a layer read
    one a each (the model's real sharing); "adafactor": shared, plus a
    factored second moment per module.  Returns (modules, unique row
    elements per token)."""
    import torch
    import paper_2606_11660_amd as P
    import synth
    wl = synth.LLAMA1B
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    mods, by_layer, uniq = [], {}, 0
    for m, md in enumerate(wl.modules):
        layer, kind = md.name.split(".")[0], md.name.split(".")[-1]
        group = {"q": "qkv", "k": "qkv", "v": "qkv", "gate": "gu", "up": "gu"}.get(kind)
        key = (layer, group)
        if variant != "separate" and group and key in by_layer:
            a = by_layer[key]
        else:
            a = torch.randn((rows, md.d_in), generator=gen, device=dev, dtype=torch.bfloat16)
            uniq += md.d_in
            if group:
                by_layer[key] = a
        g = torch.randn((rows, md.d_out), generator=gen, device=dev, dtype=torch.bfloat16)
        g.mul_(wl.g_scale)
        uniq += md.d_out
        R, S = synth.projection_pair(wl, m)
        vo = vi = None
        if variant == "adafactor":
            vo = torch.rand(md.d_out, generator=gen, device=dev) + 0.5
            vi = torch.rand(md.d_in, generator=gen, device=dev) + 0.5
        mods.append(P.Module(a, g, _dev_bf16(R).to(dev), _dev_bf16(S).to(dev), m * wl.k * wl.k,
                             v_out=vo, v_in=vi))
    return mods, uniq


def _llama1b_batches(dev, B=BATCH, n_batches=N_BATCHES):
    """Length vectors of examples [b B, (b + 1) B) of the length law, each
    packed from row 0: (list of (row_offset, length) device tensors, list of
    valid-token totals, rows of the resident buffer)."""
    import numpy as np
    import torch
    import synth
    L = synth.example_lengths(synth.LLAMA1B.n_examples)
    out, tokens = [], []
    for b in range(n_batches):
        lb = L[b * B:(b + 1) * B].astype(np.int64)
        offs = np.concatenate([[0], np.cumsum(lb)[:-1]])
        out.append((torch.from_numpy(offs.astype(np.int64)).to(dev),
                    torch.from_numpy(lb.astype(np.int32)).to(dev)))
        tokens.append(int(lb.sum()))
    return out, tokens, max(tokens)


def _gpt2_modules(dev, B=64):
    import torch
    import paper_2606_11660_amd as P
    import synth
    wl = synth.GPT2
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    mods = []
    for m, md in enumerate(wl.modules):
        a = torch.randn((B * wl.T, md.d_in), generator=gen, device=dev, dtype=torch.bfloat16)
        g = torch.randn((B * wl.T, md.d_out), generator=gen, device=dev, dtype=torch.bfloat16)
        g.mul_(wl.g_scale)
        R, S = synth.projection_pair(wl, m)
        mods.append(P.Module(a, g, _dev_bf16(R).to(dev), _dev_bf16(S).to(dev), m * wl.k * wl.k))
    return mods


def _rs_bytes(wl):
    return sum((md.d_in + md.d_out) * wl.k * 2 for md in wl.modules)


def _lowrank_store(dev, N, D=8192, seed=3):
    """G = Z F^T + 0.1 E (rank 64) as fp16 rows, drawn on the device."""
    import torch
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    F = torch.randn((D, 64), generator=gen, device=dev)
    X = torch.empty((N, D), dtype=torch.float16, device=dev)
    for i in range(0, N, 65536):
        n = min(65536, N - i)
        Z = torch.randn((n, 64), generator=gen, device=dev)
        X[i:i + n] = (Z @ F.T + 0.1 * torch.randn((n, D), generator=gen, device=dev)).half()
    return X


def _unit_store(dev, N, D, seed):
    import torch
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    G = torch.empty((N, D), dtype=torch.float16, device=dev)
    for i in range(0, N, 65536):
        c = torch.randn((min(65536, N - i), D), generator=gen, device=dev)
        G[i:i + c.shape[0]] = (c / c.norm(dim=1, keepdim=True)).half()
    return G


# ----------------------------------------------------------------------------
# the pipelined step
# ----------------------------------------------------------------------------
def _pipeline_events(stream2):
    """Events ordering the two row buffers of run_pipeline (both start free)."""
    import torch
    proj_done = [torch.cuda.Event() for _ in range(2)]
    norm_done = [torch.cuda.Event() for _ in range(2)]
    for e in norm_done:
        e.record(stream2)
    return proj_done, norm_done


def run_pipeline(mods, k, B, T, rows, store, Qrows, topk, top_s, top_i, i0, n, stream, stream2,
                 ws_p, ws_a, ws_s, proj_done, norm_done, ev=None, batches=None):
    """Steps i0 .. i0 + n - 1 of the store build: projection of the batch (on
    `stream`) -> unit norm into store slot i (on `stream2`) -> top-k merge of
    the slot against the queries (on `stream2`; step 0 starts the lists).
    Two fp32 row buffers let the projection of batch i + 1 run while batch i
    is normalised and scored: the projection into buffer b waits for the norm
    that last read b, the norm waits for its projection.  batches (optional):
    (row_offset, length) device tensors per batch, step i taking batch
    i % len(batches).  ev[i - i0] (optional) brackets step i's projection on
    `stream`."""
    import paper_2606_11660_amd as P
    n_slots = store.shape[0] // B
    for i in range(i0, i0 + n):
        b = i % 2
        slot_i = i % n_slots
        slot = store[slot_i * B:(slot_i + 1) * B]
        ro, ln = batches[i % len(batches)] if batches else (None, None)
        stream.wait_event(norm_done[b])
        if ev is not None:
            ev[i - i0][0].record(stream)
        P.attr_project(mods, k, B, T, rows[b], row_offset=ro, length=ln, ws=ws_p, stream=stream)
        if ev is not None:
            ev[i - i0][1].record(stream)
        proj_done[b].record(stream)
        stream2.wait_event(proj_done[b])
        P.attr_precond_apply(rows[b], P.PRECOND_NONE, None, True, slot, ws=ws_a, stream=stream2)
        norm_done[b].record(stream2)
        P.attr_score_topk(Qrows, slot, topk, top_s, top_i, index_base=slot_i * B, merge=i > 0,
                          ws=ws_s, stream=stream2)


# ----------------------------------------------------------------------------
# rows of the path on their own
# ----------------------------------------------------------------------------
def _row_tiny(dev, stream):
    """cfg tiny end to end: project 256 + 8 examples (fp32, one 64->64
    module, 32 tokens, k = 16), unit-normalise both, score 8 queries, top-5."""
    import numpy as np
    import torch
    import paper_2606_11660_amd as P
    import synth
    x = synth.tiny_inputs()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    G_in = P.Module(t(x["a"].reshape(-1, 64)), t(x["g"].reshape(-1, 64)), t(x["R"]), t(x["S"]), 0)
    Q_in = P.Module(t(x["aq"].reshape(-1, 64)), t(x["gq"].reshape(-1, 64)), t(x["R"]), t(x["S"]), 0)
    raw_g = torch.empty((256, 256), dtype=torch.float32, device=dev)
    raw_q = torch.empty((8, 256), dtype=torch.float32, device=dev)
    G, Q = torch.empty_like(raw_g), torch.empty_like(raw_q)
    ts = torch.empty((8, 5), dtype=torch.float32, device=dev)
    ti = torch.empty((8, 5), dtype=torch.int64, device=dev)
    ws = P.Workspace(dev)

    def run():
        P.attr_project([G_in], 16, 256, 32, raw_g, ws=ws, stream=stream)
        P.attr_precond_apply(raw_g, P.PRECOND_NONE, None, True, G, ws=ws, stream=stream)
        P.attr_project([Q_in], 16, 8, 32, raw_q, ws=ws, stream=stream)
        P.attr_precond_apply(raw_q, P.PRECOND_NONE, None, True, Q, ws=ws, stream=stream)
        P.attr_score_topk(Q, G, 5, ts, ti, ws=ws, stream=stream)
    ms = _median_ms(run, stream, reps=20, warmup=5)
    return {"workload": "tiny: one 64->64 module, 256 + 8 examples x 32 tokens fp32, k=16, "
                        "unit norm, 8 queries top-5 (5 library calls)",
            "latency_us": ms * 1e3, "examples_per_s": 264 / (ms * 1e-3)}


def _row_gpt2(dev, stream):
    """GPT-2-shaped rows: the 64-example projection call (48 modules x 512
    tokens) and the full scan of a 4096-row store (64 queries, top-10)."""
    import torch
    import paper_2606_11660_amd as P
    import synth
    wl = synth.GPT2
    B = 64
    mods = _gpt2_modules(dev, B)
    rows = torch.empty((B, wl.D), dtype=torch.float32, device=dev)
    ws = P.Workspace(dev)
    ms = _median_ms(lambda: P.attr_project(mods, wl.k, B, wl.T, rows, ws=ws, stream=stream), stream)
    byts = B * wl.T * wl.elems_per_token() * 2 + _rs_bytes(wl) + B * wl.D * 4
    tok_rows = torch.empty((B * wl.T, wl.D), dtype=torch.float32, device=dev)
    ms_tok = _median_ms(lambda: P.attr_project_tokens(mods, wl.k, B, wl.T, tok_rows, ws=ws,
                                                      stream=stream), stream)
    tok_bytes = B * wl.T * wl.elems_per_token() * 2 + _rs_bytes(wl) + B * wl.T * wl.D * 4
    del tok_rows, mods
    G = _unit_store(dev, 4096, wl.D, seed=11)
    Q = _unit_store(dev, wl.n_queries, wl.D, seed=12)
    ts = torch.empty((wl.n_queries, wl.topk), dtype=torch.float32, device=dev)
    ti = torch.empty((wl.n_queries, wl.topk), dtype=torch.int64, device=dev)
    ms_scan = _median_ms(lambda: P.attr_score_topk(Q, G, wl.topk, ts, ti, ws=ws, stream=stream),
                         stream)
    scan_bytes = (4096 + wl.n_queries) * wl.D * 2
    del G, Q
    torch.cuda.empty_cache()
    return {
        "projection": {"workload": "64 examples x 48 modules x 512 tokens, bf16, k=16", "ms": ms,
                       "examples_per_s": B / (ms * 1e-3), "bytes": byts, **_hbm(byts, ms)},
        "per_token_projection": {"workload": "the same batch, 32768 token rows x 12288 fp32 written",
                                 "ms": ms_tok, "bytes": tok_bytes, **_hbm(tok_bytes, ms_tok)},
        "store_scan_4096": {"workload": "64 queries x 4096 unit rows x 12288 fp16, top-10",
                            "ms": ms_scan, "pairs_per_s": wl.n_queries * 4096 / (ms_scan * 1e-3),
                            **_hbm(scan_bytes, ms_scan)},
    }


def _row_llama1b_variants(dev, stream):
    """1B-shaped projection of batch 0 (32 examples, 43190 tokens) with the
    model's real input sharing (q/k/v and gate/up read one a each: 0.870 of
    the separate bytes) and with Adafactor normalisation on top; the rate
    counts the unique bytes read."""
    import torch
    import paper_2606_11660_amd as P
    import synth
    wl = synth.LLAMA1B
    batches, tokens, rows_max = _llama1b_batches(dev, n_batches=1)
    out = {}
    for variant in ("shared", "adafactor"):
        mods, uniq = _llama1b_modules(dev, rows_max, variant)
        rows = torch.empty((BATCH, wl.D), dtype=torch.float32, device=dev)
        ws = P.Workspace(dev)
        ro, ln = batches[0]
        ms = _median_ms(lambda: P.attr_project(mods, wl.k, BATCH, wl.T, rows, row_offset=ro,
                                               length=ln, ws=ws, stream=stream), stream)
        byts = tokens[0] * uniq * 2 + _rs_bytes(wl) + BATCH * wl.D * 4
        out[variant] = {"ms": ms, "examples_per_s": BATCH / (ms * 1e-3), "bytes": byts,
                        **_hbm(byts, ms)}
        del mods, rows
        torch.cuda.empty_cache()
    out["workload"] = (f"batch of {BATCH} 1B-shaped examples ({tokens[0]} tokens packed), 112 "
                       "modules; shared: q/k/v and gate/up share their input rows")
    return out


def _row_kfac(dev, stream):
    """K-FAC factors of one 1B-shaped layer over 16 examples' valid tokens
    (21900, packed): A for the four distinct inputs, Gamma for the seven
    outputs, each a FULL accumulate of bf16 token rows."""
    import torch
    import paper_2606_11660_amd as P
    import synth
    lengths = synth.example_lengths(synth.LLAMA1B.n_examples)[:16]
    tot = int(lengths.sum())
    gen = torch.Generator(device=dev)
    gen.manual_seed(6)
    widths = [2048, 2048, 2048, 8192] + [2048] * 5 + [8192, 8192]
    rows = [torch.randn((tot, d), generator=gen, device=dev, dtype=torch.bfloat16) for d in widths]
    Hs = {d: torch.zeros((d, d), dtype=torch.float32, device=dev) for d in set(widths)}
    ws = P.Workspace(dev)

    def run():
        for X in rows:
            P.attr_precond_accumulate(X, P.PRECOND_FULL, Hs[X.shape[1]], ws=ws, stream=stream)
    ms = _median_ms(run, stream)
    fl = sum(tot * d * (d + 1) for d in widths)
    del rows, Hs
    torch.cuda.empty_cache()
    return {"workload": f"one 1B-shaped layer, 11 factors over {tot} tokens", "ms": ms,
            **_mfma(fl, ms), "flops": "sum over factors of tokens*d*(d+1)"}


def _row_precond(dev, stream):
    """Preconditioner rows on the 10^6 x 8192 low-rank-plus-noise store:
    DIAG accumulate, FULL accumulate (SYRK), the host finalize of H (fp64
    eigendecomposition at D = 8192, one run), DIAG apply + unit norm, FULL
    apply + unit norm with the finalized M."""
    import torch
    import paper_2606_11660_amd as P
    from paper_2606_11660_amd import finalize as F
    N, D = 1_000_000, 8192
    X = _lowrank_store(dev, N, D)
    torch.cuda.synchronize()
    xb = N * D * 2
    out = {"workload": "10^6 x 8192 fp16 rows G = Z F^T + 0.1 E (rank 64)"}
    ws = P.Workspace(dev)
    h = torch.zeros(D, dtype=torch.float32, device=dev)
    ms = _median_ms(lambda: P.attr_precond_accumulate(X, P.PRECOND_DIAG, h, ws=ws, stream=stream),
                    stream)
    out["diag_accumulate"] = {"ms": ms, **_hbm(xb, ms)}
    H = torch.zeros((D, D), dtype=torch.float32, device=dev)
    ms = _median_ms(lambda: P.attr_precond_accumulate(X, P.PRECOND_FULL, H, ws=ws, stream=stream),
                    stream)
    out["syrk"] = {"ms": ms, **_mfma(N * D * (D + 1), ms), "flops": "N*D*(D+1)"}
    H.zero_()
    P.attr_precond_accumulate(X, P.PRECOND_FULL, H, ws=ws, stream=stream)
    stream.synchronize()
    t0 = time.perf_counter()
    M, lam = F.finalize_full(H, N, return_eigenvalues=True)
    torch.cuda.synchronize()
    out["finalize_host"] = {"s": time.perf_counter() - t0, "runs": 1,
                            "what": "H (268 MB) to host, fp64 symmetrise + LAPACK eigh at D=8192, "
                                    "M = V diag(lam^-1/2) V^T, M to device",
                            "kappa": float(lam[-1] / lam[lam > 0][0]),
                            "threads": _blas_threads()}
    h.zero_()
    P.attr_precond_accumulate(X, P.PRECOND_DIAG, h, ws=ws, stream=stream)
    stream.synchronize()
    m = F.finalize_diag(h, N)
    Y = torch.empty_like(X)
    ms = _median_ms(lambda: P.attr_precond_apply(X, P.PRECOND_DIAG, m, True, Y, ws=ws,
                                                 stream=stream), stream)
    out["diag_apply_unit"] = {"ms": ms, **_hbm(2 * xb, ms)}
    ms = _median_ms(lambda: P.attr_precond_apply(X, P.PRECOND_FULL, M, True, Y, ws=ws,
                                                 stream=stream), stream)
    out["full_apply_unit"] = {"ms": ms, **_mfma(2.0 * N * D * D, ms),
                              "flops": "2*N*D^2 algorithmic (the hi/lo split executes it twice)"}
    del X, Y, H, M, ws
    torch.cuda.empty_cache()
    return out


def _row_store_scan(dev, stream, qs=(16, 64, 128, 200, 256, 1024)):
    """4M x 8192 fp16 unit store (65.5 GB), top-100, Q sweep; 16 planted
    near-duplicates (cosine 0.9) of known rows must rank first."""
    import torch
    import paper_2606_11660_amd as P
    NS, D = 4_000_000, 8192
    G = _unit_store(dev, NS, D, seed=7)
    gen = torch.Generator(device=dev)
    gen.manual_seed(8)
    tg = torch.Generator()
    tg.manual_seed(4)
    targets = torch.randperm(NS, generator=tg)[:16].to(dev)
    ws = P.Workspace(dev)
    out = {"workload": "4,000,000 x 8192 fp16 unit rows, top-100"}
    for nq in qs:
        with torch.cuda.stream(stream):
            q = torch.randn((nq, D), generator=gen, device=dev)
            q = q / q.norm(dim=1, keepdim=True)
            g = G[targets].float()
            g = g / g.norm(dim=1, keepdim=True)
            u = q[:16] - (q[:16] * g).sum(1, keepdim=True) * g
            u = u / u.norm(dim=1, keepdim=True)
            q[:16] = 0.9 * g + (1 - 0.81) ** 0.5 * u
            Q = q.half().contiguous()
        stream.synchronize()
        ts = torch.empty((nq, 100), dtype=torch.float32, device=dev)
        ti = torch.empty((nq, 100), dtype=torch.int64, device=dev)
        ms = _median_ms(lambda: P.attr_score_topk(Q, G, 100, ts, ti, ws=ws, stream=stream), stream)
        ok = bool((ti[:16, 0] == targets).all().item())
        plan = ("streaming" if nq < 128 else
                "gemm 128x256 ring" if 1 <= nq % 256 <= 128 and nq <= 384 else "gemm 256x256")
        out[str(nq)] = {"plan": plan, "ms": ms,
                        "pairs_per_s": nq * NS / (ms * 1e-3), **_hbm(NS * D * 2, ms),
                        **_mfma(2.0 * nq * NS * D, ms), "planted_rank1": ok}
    del G, ws
    torch.cuda.empty_cache()
    return out


def _peaks(dev, stream):
    """Measured peaks: one streaming read of 8 GiB (median of 10) and 2048
    waves of register-only fp16 MFMAs (median of 10)."""
    import torch
    import paper_2606_11660_amd as P
    x = torch.ones(8 << 30, dtype=torch.uint8, device=dev)
    sink = torch.zeros(4, dtype=torch.float32, device=dev)
    ms_r = _median_ms(lambda: P.attr_probe_read(x, sink, stream=stream), stream)
    del x
    torch.cuda.empty_cache()
    n = 1 << 16
    flops = 2 * 16 * 16 * 32 * n * 2048
    ms_m = _median_ms(lambda: P.attr_probe_mfma(n, sink, stream=stream), stream)
    return {"hbm_read_GBps": (8 << 30) / ms_r / 1e6, "mfma_f16_TFLOPs": flops / ms_m / 1e9,
            "method": "attr_probe_read over 8 GiB; attr_probe_mfma, 65536 MFMA 16x16x32 f16 per "
                      "wave on 2048 waves; medians of 10"}


# ----------------------------------------------------------------------------
# CPU baseline: the fp64 oracle on the host cores
# ----------------------------------------------------------------------------
def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([int(d.get("num_threads", 1)) for d in threadpool_info()] or [1])
    except Exception:
        return len(os.sched_getaffinity(0))


def _host_info():
    model = platform.processor() or "?"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    ram = None
    try:
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                ram = round(int(line.split()[1]) / 2 ** 20, 1)
                break
    except OSError:
        pass
    blas = "?"
    try:
        from threadpoolctl import threadpool_info
        blas = ", ".join(f"{d.get('internal_api')} {d.get('version')} ({d.get('num_threads')} threads)"
                         for d in threadpool_info())
    except Exception:
        pass
    return {"cpu_model": model, "ram_GiB": ram, "blas": blas,
            "affinity_cpus": len(os.sched_getaffinity(0))}


def _cpu_baseline(min_seconds: float = 12.0):
    """The fp64 oracle, as written, on the host: 2 examples of the headline
    workload (lengths 1216 and 1373 from the length law's tail, 112 modules,
    bf16) projected, unit-normalised and scored against 64 queries (top-10),
    repeated until min_seconds are timed; then single labelled runs of the
    oracle on samples of the preconditioner and store-scan workloads.  The
    token values are synthetic pools reused across modules of one width (the
    oracle's work does not depend on them)."""
    import numpy as np
    import oracle as O
    import synth
    wl = synth.LLAMA1B
    rng = np.random.default_rng(9)
    lengths = [int(x) for x in synth.example_lengths(wl.n_examples)[-2:]]
    widths = sorted({md.d_in for md in wl.modules} | {md.d_out for md in wl.modules})
    pool = {d: synth.to_bf16_bits(rng.standard_normal((max(lengths), d), dtype=np.float32))
            for d in widths}
    pairs = [synth.projection_pair(wl, m) for m in range(len(wl.modules))]
    qrows = synth.unit_rows(N_QUERIES, wl.D, seed=21)
    done, passes = 0, 0
    t0 = time.perf_counter()
    while True:
        rows = []
        for L in lengths:
            blocks = [O.project(pool[md.d_in][None, :L], pool[md.d_out][None, :L], *pairs[m])
                      for m, md in enumerate(wl.modules)]
            rows.append(O.project_concat(blocks)[0])
        U = O.to_f16(O.unit_normalize(np.stack(rows)))
        O.score_topk(qrows, U, TOPK)
        done += len(lengths)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    res = {"value": done / dt, "unit": "examples/s", "cores": _blas_threads(), "kind": "oracle",
           "sample": f"{len(lengths)} 1B-shaped examples ({sum(lengths)} tokens, 112 modules, bf16) "
                     f"through the fp64 oracle {passes} times: project, unit-normalise, score "
                     f"against {N_QUERIES} queries top-{TOPK}; {dt:.1f} s timed",
           **_host_info()}
    # labelled single runs on the other workloads' samples
    D = 8192
    X = (rng.standard_normal((8192, D), dtype=np.float32)).astype(np.float16)
    t = time.perf_counter()
    O.accumulate_full(X)
    syrk_s = time.perf_counter() - t
    M = np.eye(D) + 1e-3 * rng.standard_normal((D, D))
    t = time.perf_counter()
    O.precond_apply(X[:2048], "full", M, unit_norm=True)
    apply_s = time.perf_counter() - t
    Q = synth.unit_rows(64, D, seed=22)
    t = time.perf_counter()
    O.score_topk(Q, X[:32768], 100)
    scan_s = time.perf_counter() - t
    res["other_workloads"] = {
        "syrk_8192_rows_s": syrk_s,
        "syrk_10e6_rows_extrapolated_s": syrk_s * 1e6 / 8192,
        "full_apply_2048_rows_s": apply_s,
        "full_apply_rows_per_s": 2048 / apply_s,
        "score_64q_x_8192_rows_top100_s": scan_s,
        "score_pairs_per_s": 64 * 8192 / scan_s,
        "note": "single runs of the oracle on 8192 x 8192 fp16 rows (SYRK; its 10^6-row figure is "
                "extrapolated linearly), 2048 rows (FULL apply + unit norm) and 64 queries x 8192 "
                "rows (scores + top-100); the fp64 eigendecomposition is the finalize row",
    }
    return res


# ----------------------------------------------------------------------------
# counter runs
# ----------------------------------------------------------------------------
def _profile_row(row, dev):
    """One row of the path on its own, for rocprofv3 counter runs, each
    operation PROFILE_REPS times: `llama1b` the headline projection call
    (batch 0: 32 examples, 43190 tokens, separate inputs), `gpt2` the
    64-example GPT-2-shaped call, `gpt2_tok` its per-token variant, `syrk` a 500000 x 8192 accumulate (one full
    launch), `full_apply` 131072 rows, `scan16` / `scan128` / `scan1024` a
    1M x 8192 store with top-100, `diag_acc` / `diag_apply` 10^6 x 8192."""
    import torch
    import paper_2606_11660_amd as P
    import synth
    stream = torch.cuda.current_stream()
    if row == "llama1b":
        wl = synth.LLAMA1B
        batches, tokens, rows_max = _llama1b_batches(dev, n_batches=1)
        mods, _ = _llama1b_modules(dev, rows_max)
        rows = torch.empty((BATCH, wl.D), dtype=torch.float32, device=dev)
        for _ in range(PROFILE_REPS):
            P.attr_project(mods, wl.k, BATCH, wl.T, rows, row_offset=batches[0][0],
                           length=batches[0][1])
    elif row in ("gpt2", "gpt2_tok"):
        wl = synth.GPT2
        mods = _gpt2_modules(dev, 64)
        if row == "gpt2":
            rows = torch.empty((64, wl.D), dtype=torch.float32, device=dev)
            for _ in range(PROFILE_REPS):
                P.attr_project(mods, wl.k, 64, wl.T, rows)
        else:
            rows = torch.empty((64 * wl.T, wl.D), dtype=torch.float32, device=dev)
            for _ in range(PROFILE_REPS):
                P.attr_project_tokens(mods, wl.k, 64, wl.T, rows)
    elif row in ("diag_acc", "diag_apply"):
        X = _unit_store(dev, 1_000_000, 8192, seed=3)
        if row == "diag_acc":
            h = torch.zeros(8192, dtype=torch.float32, device=dev)
            for _ in range(PROFILE_REPS):
                P.attr_precond_accumulate(X, P.PRECOND_DIAG, h)
        else:
            m = torch.rand(8192, device=dev) + 0.5
            Y = torch.empty_like(X)
            for _ in range(PROFILE_REPS):
                P.attr_precond_apply(X, P.PRECOND_DIAG, m, True, Y)
    elif row in ("syrk", "full_apply"):
        D = 8192
        X = _lowrank_store(dev, 500_000 if row == "syrk" else 131072, D)
        if row == "syrk":
            H = torch.zeros((D, D), dtype=torch.float32, device=dev)
            for _ in range(PROFILE_REPS):
                P.attr_precond_accumulate(X, P.PRECOND_FULL, H)
        else:
            gen = torch.Generator(device=dev)
            gen.manual_seed(5)
            B = torch.randn((D, D), generator=gen, device=dev) / D ** 0.5
            M = (B @ B.T + torch.eye(D, device=dev)).contiguous()
            Y = torch.empty_like(X)
            for _ in range(PROFILE_REPS):
                P.attr_precond_apply(X, P.PRECOND_FULL, M, True, Y)
    elif row.startswith("scan"):
        nq = int(row[4:])
        G = _unit_store(dev, 1_000_000, 8192, seed=7)
        Q = _unit_store(dev, nq, 8192, seed=8)
        ts = torch.empty((nq, 100), dtype=torch.float32, device=dev)
        ti = torch.empty((nq, 100), dtype=torch.int64, device=dev)
        for _ in range(PROFILE_REPS):
            P.attr_score_topk(Q, G, 100, ts, ti)
    elif row == "kfac":
        print(json.dumps({"profile_row": row, "result": _row_kfac(dev, stream)}))
        return
    torch.cuda.synchronize()
    print(json.dumps({"profile_row": row}))


def _copy_reference(dev):
    """A plain device copy of 1 GiB, five times: the reference kernel whose
    FETCH_SIZE / WRITE_SIZE counters calibrate the traffic figures."""
    import torch
    x = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    x.fill_(1)
    torch.cuda.synchronize()
    for _ in range(5):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_reference_bytes": 1 << 30, "copies": 5}))


def _measured_traffic():
    """HBM bytes per headline attr_project call from the committed rocprofv3
    counter summary (FETCH_SIZE and WRITE_SIZE runs scaled by the copy-kernel
    calibration), or None when the projection source has changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "project_llama1b_traffic.txt")
    src = os.path.join(ROOT, "paper_2606_11660_amd", "csrc", "project.hip")
    try:
        fields = dict(line.split(": ", 1) for line in open(path).read().splitlines() if ": " in line)
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
        if fields.get("source_sha256_16", "").strip() != digest:
            return None
        return int(fields["traffic_bytes_per_call"])
    except (OSError, KeyError, ValueError):
        return None


# ----------------------------------------------------------------------------
def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--quick", action="store_true", help="headline only (no other rows, no peaks)")
    ap.add_argument("--copy-reference", action="store_true",
                    help="only run the 1 GiB copy used to calibrate traffic counters")
    ap.add_argument("--profile-row", choices=["llama1b", "gpt2", "gpt2_tok", "syrk", "full_apply", "scan16",
                                              "scan128", "scan1024", "diag_acc", "diag_apply",
                                              "kfac"],
                    help="only run one row of the path, for counter runs")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(examples and store rows would shard across GPUs, with a top-k merge of "
              "the per-GPU lists). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import paper_2606_11660_amd as P
    import synth

    wl = synth.LLAMA1B
    k, T, B, D = wl.k, wl.T, BATCH, wl.D
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_reference:
        _copy_reference(dev)
        return
    if args.profile_row:
        _profile_row(args.profile_row, dev)
        return
    stream = torch.cuda.Stream(device=dev)
    stream2 = torch.cuda.Stream(device=dev)

    # ---------------- setup (not timed) ----------------
    batches, tokens, rows_max = _llama1b_batches(dev)
    mods, elems = _llama1b_modules(dev, rows_max, "separate")
    n_store = max(args.steps, 1) * B
    store = torch.empty((n_store, D), dtype=torch.float16, device=dev)
    rows32 = [torch.empty((B, D), dtype=torch.float32, device=dev) for _ in range(2)]
    Qrows = torch.empty((N_QUERIES, D), dtype=torch.float16, device=dev)
    top_s = torch.empty((N_QUERIES, TOPK), dtype=torch.float32, device=dev)
    top_i = torch.empty((N_QUERIES, TOPK), dtype=torch.int64, device=dev)
    ws_p, ws_a, ws_s = P.Workspace(dev), P.Workspace(dev), P.Workspace(dev)
    with torch.cuda.stream(stream):
        # query rows: the processed rows of batches 0 and 1
        for b in range(2):
            P.attr_project(mods, k, B, T, rows32[0], row_offset=batches[b][0], length=batches[b][1],
                           ws=ws_p, stream=stream)
            P.attr_precond_apply(rows32[0], P.PRECOND_NONE, None, True, Qrows[b * B:(b + 1) * B],
                                 ws=ws_a, stream=stream)
    stream.synchronize()
    proj_done, norm_done = _pipeline_events(stream2)

    def steps(i0, n, ev=None):
        run_pipeline(mods, k, B, T, rows32, store, Qrows, TOPK, top_s, top_i, i0, n, stream,
                     stream2, ws_p, ws_a, ws_s, proj_done, norm_done, ev, batches)

    steps(0, args.warmup)
    stream.synchronize()
    stream2.synchronize()
    torch.cuda.synchronize()

    # ---------------- timed region ----------------
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    # the timed steps fill store slots 0 .. steps - 1 and restart the merge
    steps(0, args.steps, ev)
    stream.synchronize()
    stream2.synchronize()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    proj_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    # algorithmic bytes of the timed calls: valid tokens' a/g rows once, R/S
    # once, fp32 rows out
    call_bytes = [tokens[i % len(batches)] * elems * 2 + _rs_bytes(wl) + B * D * 4
                  for i in range(args.steps)]
    proj_bytes = float(np.mean(call_bytes))
    achieved = proj_bytes / (proj_ms * 1e-3) / 1e9
    scan_ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    with torch.cuda.stream(stream):
        P.attr_score_topk(Qrows, store, TOPK, top_s, top_i, ws=ws_s, stream=stream)
        scan_ev[0].record(stream)
        P.attr_score_topk(Qrows, store, TOPK, top_s, top_i, ws=ws_s, stream=stream)
        scan_ev[1].record(stream)
    stream.synchronize()

    result = {
        "metric": "projected per-example grads/sec; score pairs/sec + HBM GB/s on store scan",
        "value": args.steps * B / elapsed,
        "unit": "examples/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded device fill of the token rows; R, S and lengths from the "
                "seeded host generators)",
        "config": {"workload": "1B-decoder-shaped gradient store build: 16 layers x (q,k,v,o "
                               "2048->2048, gate/up 2048->8192, down 8192->2048), lengths uniform "
                               "in [256, 2048] packed (padding never read), k=16, D=28672, batch "
                               "32 per step cycling over examples 0..255, fp16 store, 64 queries "
                               "top-10 merged per step",
                   "global_batch": B, "seq_len": T, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": _measured_traffic(),
                     "kernel": "attr_project call: project_pack_kernel (x5) + project_main_kernel"
                               "<bf16,k=16> + project_reduce_kernel",
                     "bytes_per_launch": proj_bytes, "ms_per_launch": proj_ms,
                     "tokens_per_launch": float(np.mean([tokens[i % len(batches)]
                                                         for i in range(args.steps)]))},
        "store_scan": {"queries": N_QUERIES, "rows": n_store, "D": D, "k": TOPK,
                       "ms": scan_ev[0].elapsed_time(scan_ev[1])},
    }
    del mods, store, rows32
    torch.cuda.empty_cache()
    if not args.quick:
        rows = {}
        for name, fn in (("peaks", _peaks), ("tiny", _row_tiny), ("gpt2", _row_gpt2),
                         ("llama1b_variants", _row_llama1b_variants), ("kfac", _row_kfac),
                         ("precond", _row_precond), ("store_scan_4M", _row_store_scan)):
            try:
                rows[name] = fn(dev, stream)
            except Exception as exc:  # report, keep the headline line
                rows[name] = {"error": repr(exc)}
            torch.cuda.empty_cache()
        pk = rows.get("peaks", {})
        if "hbm_read_GBps" in pk:
            result["roofline"]["frac_of_measured_peak"] = achieved / pk["hbm_read_GBps"]
            result["roofline"]["measured_peak"] = pk["hbm_read_GBps"]
        result["rows"] = rows
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = _cpu_baseline()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
