"""Throughput of the attribution hot path on one MI355X.

Workload (GPT-2-shaped gradient store build + on-the-fly scoring): 12 layers
x 4 linear modules (qkv 768->2304, out 768->768, up 768->3072, down
3072->768), 512 tokens per example, k = 16 per module (12288 dims per row),
fp16 store, 64 query rows with top-10.  One step is one batch of 64
examples through the whole path:

  attr_project        (bf16 token rows resident in HBM -> fp32 rows)
  attr_precond_apply  (unit-normalise, cast to the fp16 store slot)
  attr_score_topk     (64 queries x the 64 new rows, merged into the
                       running top-10 of the store built so far)

`value` is examples/s over the timed steps.  The dominant kernel is the
projection; its roofline entry uses the algorithmic bytes of one call
(every a/g element once, R/S once, the fp32 output row) over the average
call duration measured with HIP events on the bench stream.  After the timed
steps the finished store is scanned once more (64 queries x 4096 rows) and
reported under `store_scan`.  `cpu_baseline` times the fp64 oracle on a
sample of examples on the host cores.

Usage: python bench.py [--gpus 1] [--steps 64] [--warmup 3]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MFMA_PEAK_TFLOPS = 2500.0   # dense fp16 / bf16
BATCH = 64
PROFILE_REPS = 3  # each --profile-row operation runs this often (the first call is cold)


def _cpu_baseline(n_sample: int = 6, min_seconds: float = 12.0):
    """Time the fp64 oracle on GPT-2-shaped examples on the host: project all
    48 modules, unit-normalise, score against the 64 queries.  n_sample
    examples are generated once (not timed) and passed through the oracle
    repeatedly until min_seconds of CPU work have been timed."""
    import numpy as np
    import oracle as O
    import synth
    wl = synth.GPT2
    pairs = [synth.projection_pair(wl, m) for m in range(len(wl.modules))]
    ex = [[synth.module_example(wl, m, i) for m in range(len(wl.modules))] for i in range(n_sample)]
    qrows = synth.unit_rows(wl.n_queries, wl.D, seed=21)
    try:
        from threadpoolctl import threadpool_info
        cores = max([int(d.get("num_threads", 1)) for d in threadpool_info()] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    done, passes = 0, 0
    t0 = time.perf_counter()
    while True:
        rows = []
        for i in range(n_sample):
            blocks = [O.project(ex[i][m][0][None], ex[i][m][1][None], pairs[m][0], pairs[m][1])
                      for m in range(len(wl.modules))]
            rows.append(O.project_concat(blocks)[0])
        U = O.to_f16(O.unit_normalize(np.stack(rows)))
        O.score_topk(qrows, U, wl.topk)
        done += n_sample
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds:
            break
    return {"value": done / dt, "unit": "examples/s", "cores": cores, "kind": "oracle",
            "sample": f"{n_sample} seeded GPT-2-shaped examples (48 modules x 512 tokens, bf16) "
                      f"through the fp64 oracle {passes} times: project, unit-normalise, score "
                      f"against 64 queries; {dt:.1f} s timed"}



def _measured_traffic(key="traffic_bytes_per_call"):
    """HBM bytes per attr_project call (or, with key
    "per_token_traffic_bytes_per_call", per attr_project_tokens call) from the
    committed rocprofv3 counter summary (FETCH_SIZE and WRITE_SIZE runs,
    scaled by the copy-kernel calibration), or None when the projection
    source has changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "project_gpt2_traffic.txt")
    src = os.path.join(ROOT, "paper_2606_11660_amd", "csrc", "project.hip")
    try:
        fields = dict(line.split(": ", 1) for line in open(path).read().splitlines() if ": " in line)
        digest = hashlib.sha256(open(src, "rb").read()).hexdigest()[:16]
        if fields.get("source_sha256_16", "").strip() != digest:
            return None
        return int(fields[key])
    except (OSError, KeyError, ValueError):
        return None


def _pipeline_events(stream2):
    """Events ordering the two row buffers of run_pipeline (both start free)."""
    import torch
    proj_done = [torch.cuda.Event() for _ in range(2)]
    norm_done = [torch.cuda.Event() for _ in range(2)]
    for e in norm_done:
        e.record(stream2)
    return proj_done, norm_done


def run_pipeline(mods, k, B, T, rows, store, Qrows, topk, top_s, top_i, i0, n, stream, stream2,
                 ws_p, ws_a, ws_s, proj_done, norm_done, ev=None):
    """Steps i0 .. i0 + n - 1 of the store build: projection of the batch (on
    `stream`) -> unit norm into store slot i (on `stream2`) -> top-k merge of
    the slot against the queries (on `stream2`; step 0 starts the lists).
    Two fp32 row buffers let the projection of batch i + 1 run while batch i
    is normalised and scored: the projection into buffer b waits for the norm
    that last read b, the norm waits for its projection.  ev[i - i0] (optional)
    brackets step i's projection on `stream`."""
    import paper_2606_11660_amd as P
    n_slots = store.shape[0] // B
    for i in range(i0, i0 + n):
        b = i % 2
        slot_i = i % n_slots
        slot = store[slot_i * B:(slot_i + 1) * B]
        stream.wait_event(norm_done[b])
        if ev is not None:
            ev[i - i0][0].record(stream)
        P.attr_project(mods, k, B, T, rows[b], ws=ws_p, stream=stream)
        if ev is not None:
            ev[i - i0][1].record(stream)
        proj_done[b].record(stream)
        stream2.wait_event(proj_done[b])
        P.attr_precond_apply(rows[b], P.PRECOND_NONE, None, True, slot, ws=ws_a, stream=stream2)
        norm_done[b].record(stream2)
        P.attr_score_topk(Qrows, slot, topk, top_s, top_i, index_base=slot_i * B, merge=i > 0,
                          ws=ws_s, stream=stream2)


def _timeit(fn, stream, reps):
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    with torch.cuda.stream(stream):
        fn()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
    stream.synchronize()
    return e0.elapsed_time(e1) / reps


def _llama1b_projection(stream, dev):
    """Projection of the 1B-shaped model (16 layers x q,k,v,o 2048->2048,
    gate/up 2048->8192, down 8192->2048; k = 16, row of 28672): a resident
    batch of 16 examples with ragged lengths (uniform in [256, 2048], seed 4),
    tokens packed back to back (row_offset / length).  Algorithmic bytes are
    the valid tokens' a/g rows, R/S once and the fp32 rows.  The second
    variant points q/k/v at one input tensor and gate/up at another (the
    model's real sharing): its unique bytes are 0.870 of the first, and the
    rate is reported over those unique bytes.  The third adds optimizer-state
    normalisation (factored second moments per module) to the second."""
    import numpy as np
    import torch
    import paper_2606_11660_amd as P
    import synth

    wl = synth.LLAMA1B
    k, B, T = wl.k, 16, wl.T
    lengths = synth.example_lengths(wl.n_examples)[:B]
    tot = int(lengths.sum())
    offs = np.concatenate([[0], np.cumsum(lengths.astype(np.int64))[:-1]])
    off_t = torch.from_numpy(offs.astype(np.int64)).to(dev)
    len_t = torch.from_numpy(lengths.astype(np.int32)).to(dev)
    gen = torch.Generator(device=dev)
    gen.manual_seed(1)
    sep, shared, normed, by_layer = [], [], [], {}
    for m, md in enumerate(wl.modules):
        layer, kind = md.name.split(".")[0], md.name.split(".")[-1]
        a = torch.randn((tot, md.d_in), generator=gen, device=dev, dtype=torch.bfloat16)
        g = torch.randn((tot, md.d_out), generator=gen, device=dev, dtype=torch.bfloat16)
        R, S = synth.projection_pair(wl, m)
        Rt = torch.from_numpy(R.view(np.int16)).view(torch.bfloat16).to(dev)
        St = torch.from_numpy(S.view(np.int16)).view(torch.bfloat16).to(dev)
        sep.append(P.Module(a, g, Rt, St, m * k * k))
        group = {"q": "qkv", "k": "qkv", "v": "qkv", "gate": "gu", "up": "gu"}.get(kind)
        a_sh = by_layer.setdefault((layer, group), a) if group else a
        shared.append(P.Module(a_sh, g, Rt, St, m * k * k))
        vo = torch.rand(md.d_out, generator=gen, device=dev) + 0.5
        vi = torch.rand(md.d_in, generator=gen, device=dev) + 0.5
        normed.append(P.Module(a_sh, g, Rt, St, m * k * k, v_out=vo, v_in=vi))
    rows = torch.empty((B, wl.D), dtype=torch.float32, device=dev)
    ws = P.Workspace(dev)
    elems = sum(md.d_in + md.d_out for md in wl.modules)
    uniq = sum(md.d_out + (md.d_in if md.name.split(".")[-1] in ("q", "gate", "o", "down") else 0)
               for md in wl.modules)
    rs = sum((md.d_in + md.d_out) * k * 2 for md in wl.modules)
    out = {"modules": len(wl.modules), "batch": B, "valid_tokens": tot,
           "lengths": "uniform integers in [256, 2048], seed 4, first 16", "D": wl.D}
    for name, mods, e in (("separate_inputs", sep, elems), ("shared_qkv_gateup_inputs", shared, uniq),
                          ("shared_inputs_adafactor_normalised", normed, uniq)):
        ms = _timeit(lambda: P.attr_project(mods, k, B, T, rows, row_offset=off_t, length=len_t,
                                            ws=ws, stream=stream), stream, 5)
        byts = tot * e * 2 + rs + B * wl.D * 4
        out[name] = {"ms": ms, "examples_per_s": B / (ms * 1e-3), "bytes": byts,
                     "GBps": byts / ms / 1e6, "frac_hbm": byts / ms / 1e6 / HBM_PEAK_GBPS}
    del sep, shared, normed, by_layer, rows
    torch.cuda.empty_cache()
    return out


def _kfac_factors_1b_layer(stream, dev):
    """K-FAC factors of one 1B-shaped layer over a 16-example batch's valid
    tokens (21900, packed): A for the layer's four distinct inputs (q/k/v
    share one, gate/up another; 3 x 2048 + 8192 wide) and Gamma for its
    seven outputs (5 x 2048 + 2 x 8192), each a FULL accumulate on the
    packed bf16 token rows.  Algorithmic flops N d (d + 1) per factor."""
    import numpy as np
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
    ms = _timeit(run, stream, 3)
    fl = sum(tot * d * (d + 1) for d in widths)
    del rows, Hs
    torch.cuda.empty_cache()
    return {"tokens": tot, "factors": len(widths), "widths": widths, "ms": ms,
            "TFLOPs": fl / ms / 1e9, "frac_mfma": fl / ms / 1e9 / MFMA_PEAK_TFLOPS,
            "flops": "sum over factors of tokens*d*(d+1), upper triangles incl. diagonal"}


def _other_rows(stream, dev):
    """Timings of the 1B-shaped projection, of the preconditioner rows on the
    10^6 x 8192 low-rank-plus-noise store and of the 4M-row store scan (Q
    sweep: Q <= 64 runs the streaming plan, HBM-bound; Q >= 128 the GEMM plan,
    MFMA-bound), each against its roofline."""
    import torch
    import paper_2606_11660_amd as P
    out = {"projection_llama1b_shaped": _llama1b_projection(stream, dev),
           "kfac_factors_1b_layer": _kfac_factors_1b_layer(stream, dev)}
    N, D = 1_000_000, 8192
    gen = torch.Generator(device=dev)
    gen.manual_seed(3)
    with torch.cuda.stream(stream):
        F = torch.randn((D, 64), generator=gen, device=dev)
        X = torch.empty((N, D), dtype=torch.float16, device=dev)
        for i in range(0, N, 65536):
            n = min(65536, N - i)
            Z = torch.randn((n, 64), generator=gen, device=dev)
            X[i:i + n] = (Z @ F.T + 0.1 * torch.randn((n, D), generator=gen, device=dev)).half()
        del F, Z
    stream.synchronize()
    xb = N * D * 2
    h = torch.zeros(D, dtype=torch.float32, device=dev)
    ms = _timeit(lambda: P.attr_precond_accumulate(X, P.PRECOND_DIAG, h, stream=stream), stream, 3)
    out["diag_accumulate"] = {"shape": [N, D], "ms": ms, "GBps": xb / ms / 1e6,
                              "frac_hbm": xb / ms / 1e6 / HBM_PEAK_GBPS}
    H = torch.zeros((D, D), dtype=torch.float32, device=dev)
    ms = _timeit(lambda: P.attr_precond_accumulate(X, P.PRECOND_FULL, H, stream=stream), stream, 2)
    fl = N * D * (D + 1)
    out["syrk"] = {"shape": [N, D], "ms": ms, "TFLOPs": fl / ms / 1e9,
                   "frac_mfma": fl / ms / 1e9 / MFMA_PEAK_TFLOPS,
                   "flops": "N*D*(D+1), upper triangle incl. diagonal"}
    m = torch.rand(D, generator=gen, device=dev) + 0.5
    Y = torch.empty_like(X)
    ms = _timeit(lambda: P.attr_precond_apply(X, P.PRECOND_DIAG, m, True, Y, stream=stream), stream, 3)
    out["diag_apply_unit"] = {"shape": [N, D], "ms": ms, "GBps": 2 * xb / ms / 1e6,
                              "frac_hbm": 2 * xb / ms / 1e6 / HBM_PEAK_GBPS}
    B = torch.randn((D, D), generator=gen, device=dev) / D ** 0.5
    M = (B @ B.T + torch.eye(D, device=dev)).contiguous()
    del B
    ms = _timeit(lambda: P.attr_precond_apply(X, P.PRECOND_FULL, M, True, Y, stream=stream), stream, 2)
    fl = 2.0 * N * D * D
    out["full_apply_unit"] = {"shape": [N, D], "ms": ms, "TFLOPs": fl / ms / 1e9,
                              "frac_mfma": fl / ms / 1e9 / MFMA_PEAK_TFLOPS,
                              "flops": "2*N*D^2 algorithmic (the hi/lo split executes it twice)"}
    del X, Y, H, M
    torch.cuda.empty_cache()

    # store scan: 4M unit rows x 8192 fp16 (65.5 GB), planted near-duplicates
    NS = 4_000_000
    G = torch.empty((NS, D), dtype=torch.float16, device=dev)
    with torch.cuda.stream(stream):
        for i in range(0, NS, 65536):
            n = min(65536, NS - i)
            c = torch.randn((n, D), generator=gen, device=dev)
            G[i:i + n] = (c / c.norm(dim=1, keepdim=True)).half()
        del c
    stream.synchronize()
    tg = torch.Generator()
    tg.manual_seed(4)
    targets = torch.randperm(NS, generator=tg)[:16].to(dev)
    scan = {}
    for nq in (16, 64, 256, 1024):
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
        ms = _timeit(lambda: P.attr_score_topk(Q, G, 100, ts, ti, stream=stream), stream, 1)
        ok = bool((ti[:16, 0] == targets).all().item())
        scan[str(nq)] = {"plan": "streaming" if nq < 128 else "gemm",
                         "ms": ms, "pairs_per_s": nq * NS / (ms * 1e-3),
                         "GBps": NS * D * 2 / ms / 1e6,
                         "frac_hbm": NS * D * 2 / ms / 1e6 / HBM_PEAK_GBPS,
                         "TFLOPs": 2.0 * nq * NS * D / ms / 1e9,
                         "frac_mfma": 2.0 * nq * NS * D / ms / 1e9 / MFMA_PEAK_TFLOPS,
                         "planted_rank1": ok}
    out["store_scan_4M_x_8192_top100"] = scan
    del G
    torch.cuda.empty_cache()
    return out


def _profile_row(row, dev):
    """One row of the path on its own, sized for counter runs (rocprofv3
    --pmc): `syrk` on a 500000 x 8192 low-rank-plus-noise store (one full
    accumulate launch), `full_apply` on 131072 rows of it, `scan16` / `scan1024` on a 1M x 8192 unit fp16 store with top-100,
    `diag_acc` / `diag_apply` (DIAG accumulate, DIAG apply + unit norm) on a
    10^6 x 8192 fp16 store, each run PROFILE_REPS times; `llama1b` the
    1B-shaped projection row (timed, printed as JSON)."""
    import torch
    import paper_2606_11660_amd as P
    if row in ("llama1b", "kfac"):
        stream = torch.cuda.Stream(device=dev)
        fn = _llama1b_projection if row == "llama1b" else _kfac_factors_1b_layer
        print(json.dumps({"profile_row": row, "result": fn(stream, dev)}))
        return
    D = 8192
    gen = torch.Generator(device=dev)
    gen.manual_seed(3)
    if row in ("diag_acc", "diag_apply"):
        N = 1_000_000
        X = torch.empty((N, D), dtype=torch.float16, device=dev)
        for i in range(0, N, 65536):
            n = min(65536, N - i)
            X[i:i + n] = torch.randn((n, D), generator=gen, device=dev).half()
        if row == "diag_acc":
            h = torch.zeros(D, dtype=torch.float32, device=dev)
            for _ in range(PROFILE_REPS):
                P.attr_precond_accumulate(X, P.PRECOND_DIAG, h)
        else:
            m = torch.rand(D, generator=gen, device=dev) + 0.5
            Y = torch.empty_like(X)
            for _ in range(PROFILE_REPS):
                P.attr_precond_apply(X, P.PRECOND_DIAG, m, True, Y)
    elif row in ("syrk", "full_apply"):
        N = 500_000 if row == "syrk" else 131072
        F = torch.randn((D, 64), generator=gen, device=dev)
        X = torch.empty((N, D), dtype=torch.float16, device=dev)
        for i in range(0, N, 65536):
            n = min(65536, N - i)
            Z = torch.randn((n, 64), generator=gen, device=dev)
            X[i:i + n] = (Z @ F.T + 0.1 * torch.randn((n, D), generator=gen, device=dev)).half()
        del F, Z
        if row == "syrk":
            H = torch.zeros((D, D), dtype=torch.float32, device=dev)
            for _ in range(PROFILE_REPS):
                P.attr_precond_accumulate(X, P.PRECOND_FULL, H)
        else:
            B = torch.randn((D, D), generator=gen, device=dev) / D ** 0.5
            M = (B @ B.T + torch.eye(D, device=dev)).contiguous()
            Y = torch.empty_like(X)
            for _ in range(PROFILE_REPS):
                P.attr_precond_apply(X, P.PRECOND_FULL, M, True, Y)
    else:
        N, nq = 1_000_000, int(row[4:])
        G = torch.empty((N, D), dtype=torch.float16, device=dev)
        for i in range(0, N, 65536):
            c = torch.randn((min(65536, N - i), D), generator=gen, device=dev)
            G[i:i + c.shape[0]] = (c / c.norm(dim=1, keepdim=True)).half()
        q = torch.randn((nq, D), generator=gen, device=dev)
        Q = (q / q.norm(dim=1, keepdim=True)).half()
        ts = torch.empty((nq, 100), dtype=torch.float32, device=dev)
        ti = torch.empty((nq, 100), dtype=torch.int64, device=dev)
        for _ in range(PROFILE_REPS):
            P.attr_score_topk(Q, G, 100, ts, ti)
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--quick", action="store_true", help="skip the preconditioner / store-scan rows")
    ap.add_argument("--copy-reference", action="store_true",
                    help="only run the 1 GiB copy used to calibrate traffic counters")
    ap.add_argument("--profile-row", choices=["syrk", "full_apply", "scan16", "scan1024", "diag_acc", "kfac",
                                              "diag_apply", "llama1b"],
                    help="only run one row of the path once, for counter runs")
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

    wl = synth.GPT2
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

    # ---------------- setup (not timed) ----------------
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    mods = []
    for m, md in enumerate(wl.modules):
        a = torch.empty((B * T, md.d_in), dtype=torch.bfloat16, device=dev)
        g = torch.empty((B * T, md.d_out), dtype=torch.bfloat16, device=dev)
        a.copy_(torch.randn(a.shape, generator=gen, device=dev))
        g.copy_(torch.randn(g.shape, generator=gen, device=dev) * wl.g_scale)
        R, S = synth.projection_pair(wl, m)
        Rt = torch.from_numpy(R.view(np.int16)).view(torch.bfloat16).to(dev)
        St = torch.from_numpy(S.view(np.int16)).view(torch.bfloat16).to(dev)
        mods.append(P.Module(a, g, Rt, St, m * k * k))
    n_store = max(args.steps, 1) * B
    store = torch.empty((n_store, D), dtype=torch.float16, device=dev)
    rows32 = torch.empty((B, D), dtype=torch.float32, device=dev)
    rows32b = [rows32, torch.empty((B, D), dtype=torch.float32, device=dev)]
    stream2 = torch.cuda.Stream(device=dev)
    Qrows = torch.empty((wl.n_queries, D), dtype=torch.float16, device=dev)
    top_s = torch.empty((wl.n_queries, wl.topk), dtype=torch.float32, device=dev)
    top_i = torch.empty((wl.n_queries, wl.topk), dtype=torch.int64, device=dev)
    ws_p, ws_a, ws_s = P.Workspace(dev), P.Workspace(dev), P.Workspace(dev)
    with torch.cuda.stream(stream):
        # query rows: the processed rows of the first batch
        P.attr_project(mods, k, B, T, rows32, ws=ws_p, stream=stream)
        P.attr_precond_apply(rows32, P.PRECOND_NONE, None, True, Qrows[:B], ws=ws_a, stream=stream)
    stream.synchronize()

    proj_done, norm_done = _pipeline_events(stream2)

    def steps(i0, n, ev=None):
        run_pipeline(mods, k, B, T, rows32b, store, Qrows, wl.topk, top_s, top_i, i0, n,
                     stream, stream2, ws_p, ws_a, ws_s, proj_done, norm_done, ev)

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

    # ---------------- full store scan (reported separately) ----------------
    scan_ev = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
    with torch.cuda.stream(stream):
        P.attr_score_topk(Qrows, store, wl.topk, top_s, top_i, ws=ws_s, stream=stream)
        scan_ev[0].record(stream)
        reps = 10
        for _ in range(reps):
            P.attr_score_topk(Qrows, store, wl.topk, top_s, top_i, ws=ws_s, stream=stream)
        scan_ev[1].record(stream)
    stream.synchronize()
    scan_ms = scan_ev[0].elapsed_time(scan_ev[1]) / reps
    scan_bytes = n_store * D * 2 + wl.n_queries * D * 2

    # ---------------- per-token blocks of the same batch (reported separately) ----------------
    tok_rows = torch.empty((B * T, D), dtype=torch.float32, device=dev)
    tok_ms = _timeit(lambda: P.attr_project_tokens(mods, k, B, T, tok_rows, ws=ws_p, stream=stream),
                     stream, 5)
    del tok_rows
    tok_bytes = B * T * wl.elems_per_token() * 2 + B * T * D * 4 + sum(
        (md.d_in + md.d_out) * k * 2 for md in wl.modules)

    # algorithmic bytes of one projection call: a/g rows once, R/S once, fp32 rows out
    per_example = T * wl.elems_per_token() * 2 + D * 4
    rs_bytes = sum((md.d_in + md.d_out) * k * 2 for md in wl.modules)
    proj_bytes = B * per_example + rs_bytes
    achieved = proj_bytes / (proj_ms * 1e-3) / 1e9

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
        "data": "synthetic (seeded device fill; R, S from the seeded host generator)",
        "config": {"workload": "gpt2-shaped store build: 12 layers x (qkv 768->2304, out 768->768, "
                               "up 768->3072, down 3072->768), T=512, k=16, D=12288, "
                               "batch 64 per step, fp16 store, 64 queries top-10 merged per step",
                   "global_batch": B, "seq_len": T, "parallelism": "single GPU"},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBPS, "traffic": _measured_traffic(),
                     "kernel": "attr_project call: 2 x project_pack_kernel + project_main_kernel"
                               "<bf16,k=16> + project_reduce_kernel",
                     "bytes_per_launch": proj_bytes, "ms_per_launch": proj_ms},
        "store_scan": {"queries": wl.n_queries, "rows": n_store, "D": D, "k": wl.topk,
                       "ms": scan_ms, "pairs_per_s": wl.n_queries * n_store / (scan_ms * 1e-3),
                       "GBps": scan_bytes / (scan_ms * 1e-3) / 1e9},
        "per_token_projection": {"tokens": B * T, "ms": tok_ms, "bytes": tok_bytes,
                                 "GBps": tok_bytes / tok_ms / 1e6,
                                 "frac_hbm": tok_bytes / tok_ms / 1e6 / HBM_PEAK_GBPS,
                                 "traffic": _measured_traffic("per_token_traffic_bytes_per_call")},
    }
    del mods, store, rows32, rows32b
    torch.cuda.empty_cache()
    if not args.quick:
        try:
            result["other_rows"] = _other_rows(stream, dev)
        except Exception as exc:  # report, keep the headline line
            result["other_rows"] = {"error": repr(exc)}
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = _cpu_baseline()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
