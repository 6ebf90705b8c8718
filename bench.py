#!/usr/bin/env python3
"""Benchmark of the ResKV hot path on one MI355X.

Workload (default): batched decode, bf16, 32 layers x (32 query / 8 KV heads,
head_dim 128), batch 32, every sequence a 32768-token prefill compressed to a
2048-slot budget per KV head, residual split per (layer, KV head) drawn from
{0, 64, 128, 256, 512}, per-query gate thresholds tau ~ N(0, 0.5), 256 decode
steps that each append one token per (sequence, KV head).

One timed step = the whole job on one batch: reskv_build_cache for all 32
layers (from prefill K/V resident in HBM), then 256 decode steps, each of
which runs reskv_decode_attn for all 32 layers with that step's token
appended inside the call.
value = decode tokens (batch x layers x decode steps) / step time, i.e. the
decode rate of the whole job with its construction included (the metric
label says so); decode_tokens_per_s beside it is the decode phase alone.

Also reported: decode-only throughput and HBM GB/s, construction GB/s,
construction with the validation proxy choosing r and with AdaKV's
cross-head allocation (ms per layer, untimed in the job), the roofline of
the decode kernels (algorithmic bytes per call / average call time from HIP
events on the launch stream), and the fp64 oracle's throughput on the host
cores over a bounded sample of the same job. After the main job its
buffers are freed and two more workloads are measured (per_config): the
long-context construction workload (B 4, 128K context, 8 layers, budget
1024 = 768 + 256, window 64: construction GB/s and TFLOP/s against the
MFMA roofline, decode GB/s) and the ragged GQA-7 workload (B 64, 28 q / 4
KV heads, contexts 4K-64K, budgets 256-1024, 28 layers: decode GB/s
against the HBM roofline, construction time).

    python bench.py [--gpus 1] [--steps K] [--warmup W]
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=2, help="index of the synthetic workload (2 = batched decode)")
    ap.add_argument("--decode-steps", type=int, default=None, help="override decode steps per job (testing only)")
    ap.add_argument("--layers", type=int, default=None, help="override layer count (testing only)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--eager-decode", action="store_true",
                    help="issue the decode calls one by one instead of replaying them as one HIP graph")
    ap.add_argument("--cpu-budget-s", type=float, default=25.0)
    ap.add_argument("--mode", choices=["job", "decode", "proxy"], default="job",
                    help="job: the timed whole job (default); decode: build once, then only decode calls "
                         "(for rocprofv3 counter runs), preceded by one 256 MiB plain copy used to calibrate "
                         "the byte counters; proxy: only construction with the validation proxy, every layer")
    ap.add_argument("--proxy-layers", type=int, default=2,
                    help="layers built with the validation proxy after the timed job (0: skip)")
    ap.add_argument("--slot-cap", type=int, default=None,
                    help="slots allocated per (sequence, KV head) cache (default: budget + decode steps)")
    ap.add_argument("--adakv-layers", type=int, default=2,
                    help="layers built with AdaKV's cross-head allocation after the timed job (0: skip)")
    ap.add_argument("--per-config", default="3,4",
                    help="other workloads measured after the main job, comma-separated indices "
                         "(3 = long-context construction, 4 = ragged GQA-7; empty: none)")
    ap.add_argument("--per-config-reps", type=int, default=2, help="timed constructions per layer of those workloads")
    return ap.parse_args()


def decode_call_bytes(B, Hq, Hkv, d, elem, r, main_len):
    """Algorithmic HBM bytes of one decode call with its fused append: every
    live K and V slot once (the appended token included), the residual
    log-counts, the queries, the fp32 outputs, and the appended token's K/V
    read from its staging buffer."""
    slots = int((r + main_len).sum())
    return (slots * 2 * d * elem + 4 * int(r.sum()) + B * Hq * d * elem + B * Hq * d * 4
            + B * Hkv * 2 * d * elem)


def build_call_bytes(wl, elem, res):
    """Algorithmic bytes of one construction call: prefill K and V read once,
    window queries, the written cache rows, log-counts and main indices."""
    B, Hkv, d = wl.batch, wl.hkv, wl.d
    kv = sum(2 * wl.ctx[b] * d * elem * Hkv for b in range(B))
    q = B * wl.hq * wl.window * d * elem
    out = 0
    for b in range(B):
        for h in range(Hkv):
            r = int(res[b][h])
            m = min(wl.budget[b] - r, wl.ctx[b])
            out += (r + m) * 2 * d * elem + 4 * r + 4 * m
    return kv + q + out


def source_hash(*paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


# Committed rocprofv3 summaries per workload (profiles/<name>.json).
PROFILES = {2: {"decode": "decode_head_batched_decode_traffic", "construction": "construction_batched_decode_counters"},
            3: {"construction": "construction_long_context_counters"},
            4: {"decode": "decode_head_ragged_gqa7_traffic"}}


def traffic_from_profile(src_hash, name=PROFILES[2]["decode"]):
    """Measured / algorithmic HBM bytes of the decode calls profiled with
    rocprofv3 counters, if that measurement was taken on the current decode
    source."""
    path = os.path.join(ROOT, "profiles", name + ".json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("decode_source_sha256_16") != src_hash:
        return None
    num, den = rec.get("bytes_per_call"), rec.get("algorithmic_bytes_per_call")
    return num / den if num and den else None


def construction_mfma_from_profile(src_hash, name=PROFILES[2]["construction"]):
    """MFMA use of the construction's MFMA kernels from the committed
    rocprofv3 counters (kernel time, busy percent, executed and algorithmic
    TFLOP/s, and algorithmic flops over the 2.5 PF/s peak), if the
    measurement was taken on the current construction source."""
    rec = counters_from_profile(name, src_hash)
    return rec["summary"] if rec is not None else None


# Validation proxy settings of App. B.3: grid of budget fractions, 8 of the 32
# window rows of every query head held out (96 fit / 32 validation queries at
# G = 4), relative margin 0.01.
PROXY_GRID = (0.0, 0.05, 0.10, 0.15, 0.20)
PROXY_VAL_ROWS = 8
PROXY_DELTA = 0.01


def proxy_runs(rk, torch, wl, shape, layers, caches, n_layers, dev):
    """Construction with the validation proxy for the first n_layers layers:
    one untimed call, then every layer once between events on the launch
    stream. Returns ms per layer and the chosen residual counts."""
    import numpy as np
    S = wl.max_ctx
    params = rk.BuildParams(S, wl.window, wl.window, wl.lloyd_iters, 0)
    xp = rk.make_proxy(PROXY_GRID, PROXY_VAL_ROWS, PROXY_DELTA)
    gate = rk.make_gate(tau_scalar=0.25, alpha=wl.alpha, g_min=wl.g_min, beta=wl.beta)
    nws = max(rk.reskv_build_proxy_workspace_size(shape, params, xp, layers[l]["seq_len"], layers[l]["budget"])
              for l in range(n_layers))
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def call(l):
        x, c = layers[l], caches[l]
        rk.reskv_build_cache_proxy(shape, params, xp, gate, x["K"], x["V"], x["seq_len"], x["q_obs"], x["budget"],
                                   c["kc"], c["vc"], c["logc"], c["main_idx"], c["res_len"], c["main_len"], ws)

    call(0)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for l in range(n_layers):
        call(l)
    e1.record(stream)
    torch.cuda.synchronize()
    chosen = np.concatenate([caches[l]["res_len"].cpu().numpy() for l in range(n_layers)])
    counts = [int(np.floor(f * wl.budget[0] + 0.5)) for f in PROXY_GRID]
    return dict(ms_per_layer=e0.elapsed_time(e1) / n_layers, layers_timed=n_layers,
                workspace_bytes=nws, grid_counts=counts,
                chosen_count_heads={str(r): int((chosen == r).sum()) for r in counts})


# AdaKV's safeguard coefficient (App. B.2.2).
ADAKV_SAFEGUARD = 0.2


def adakv_runs(rk, torch, wl, shape, layers, caches, res_layers, n_layers, dev):
    """Construction with AdaKV's cross-head allocation for the first n_layers
    layers (slot capacity of the decode caches): one untimed call, then every
    layer once between events on the launch stream. Returns ms per layer and
    the spread of the allocated main lengths."""
    import numpy as np
    S = wl.max_ctx
    params = rk.BuildParams(S, wl.window, wl.window, wl.lloyd_iters, 0)
    nws = max(rk.reskv_build_adakv_workspace_size(shape, params, ADAKV_SAFEGUARD, wl.steps, layers[l]["seq_len"],
                                                  layers[l]["budget"], res_layers[l].reshape(-1))
              for l in range(n_layers))
    ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def call(l):
        x, c = layers[l], caches[l]
        rk.reskv_build_cache_adakv(shape, params, ADAKV_SAFEGUARD, wl.steps, x["K"], x["V"], x["seq_len"], x["q_obs"],
                                   x["budget"], res_layers[l].reshape(-1), c["kc"], c["vc"], c["logc"],
                                   c["main_idx"], c["res_len"], c["main_len"], ws)

    call(0)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for l in range(n_layers):
        call(l)
    e1.record(stream)
    torch.cuda.synchronize()
    ml = np.concatenate([caches[l]["main_len"].cpu().numpy() for l in range(n_layers)])
    return dict(ms_per_layer=e0.elapsed_time(e1) / n_layers, layers_timed=n_layers, safeguard=ADAKV_SAFEGUARD,
                main_len_min=int(ml.min()), main_len_mean=float(ml.mean()), main_len_max=int(ml.max()))


def cpu_baseline(wl, x0, q0, tau0, res_layers, budget_s):
    """Time the fp64 oracle on a bounded sample of the job on the host and
    extrapolate to the whole job: construction of one (sequence, KV head)
    for each residual count that layer 0 of sequence 0 uses (scores +
    selection, then Lloyd, whose cost grows with r), and a few decode
    layer-steps for every query head of every sequence. Heads of other
    layers are priced at the measured head with their r (linear in r between
    measured counts); the sample stops taking heads once `budget_s` of
    construction has been spent."""
    import numpy as np
    from oracle import reskv_oracle as orc
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max(int(i.get("num_threads", 1)) for i in threadpool_info()) if threadpool_info() else 1
    except Exception:
        blas_threads = None
    cores = len(os.sched_getaffinity(0))
    B, Hkv, G, d = wl.batch, wl.hkv, wl.group, wl.d
    s = wl.ctx[0]
    r_row = res_layers[0][0]
    picks = {}
    for h in sorted(range(Hkv), key=lambda j: r_row[j]):
        picks.setdefault(int(r_row[h]), h)
    t_build = {}
    spent = 0.0
    for r, h in sorted(picks.items()):
        if spent > budget_s:
            break
        m = wl.budget[0] - r
        K = x0["K"][0, h, :s].float().cpu().numpy().astype(np.float64)
        V = x0["V"][0, h, :s].float().cpu().numpy().astype(np.float64)
        Qw = x0["q_obs"][0, h * G:(h + 1) * G].float().cpu().numpy().astype(np.float64)
        t0 = time.perf_counter()
        n = orc.scored_length(s, m, wl.window)
        raw = orc.window_raw_scores(K, Qw)
        sc = orc.pool5(raw[:n])
        main, ev, seeds = orc.select_main(sc, s, m, wl.window, r)
        if r > 0:
            a, mu, _ = orc.lloyd(K[ev], K[seeds], wl.lloyd_iters)
            orc.residual_entries(K[ev], V[ev], a, mu, r, d)
        t_build[r] = time.perf_counter() - t0
        spent += t_build[r]
    rs = np.array(sorted(t_build))
    ts = np.array([t_build[r] for r in rs])

    def head_cost(r):
        if len(rs) == 1:
            return ts[0] * max(r, 1) / max(rs[0], 1)
        return float(np.interp(r, rs, ts, left=None, right=None)) if r <= rs[-1] else \
            ts[-1] + (r - rs[-1]) * (ts[-1] - ts[-2]) / (rs[-1] - rs[-2])

    # decode: a few layer-steps, every (sequence, query head), on caches of
    # the decode shape (main rows from the prefill, residual rows from means)
    rng = np.random.default_rng(0)
    r = int(np.median(r_row))
    m = wl.budget[0] - r
    n_main = m + wl.steps // 2
    kc = x0["K"][:, :, :n_main + r].float().cpu().numpy().astype(np.float64)
    vc = x0["V"][:, :, :n_main + r].float().cpu().numpy().astype(np.float64)
    logc = np.log(rng.integers(1, 100, size=(B, Hkv, max(r, 1))).astype(np.float64))
    res_len = np.full((B, Hkv), r)
    main_len = np.full((B, Hkv), n_main)
    q = q0.float().cpu().numpy().astype(np.float64)
    tau = tau0.cpu().numpy().astype(np.float64)
    n_dec = 4
    t0 = time.perf_counter()
    for _ in range(n_dec):
        orc.decode(q, kc, vc, logc, res_len, main_len, tau, wl.alpha, wl.g_min, wl.beta)
    t_dec = (time.perf_counter() - t0) / n_dec
    # extrapolate to one job
    job = sum(head_cost(int(res_layers[l][b][hh])) for l in range(wl.layers) for b in range(B) for hh in range(Hkv))
    job += t_dec * wl.layers * wl.steps
    tokens = B * wl.layers * wl.steps
    built = ", ".join(f"r={r}: {t_build[r]:.2f}s" for r in rs)
    return dict(value=tokens / job, unit="tokens/s", cores=cores, blas_threads=blas_threads, kind="oracle",
                sample=(f"fp64 numpy oracle on the host: construction (scores, selection, Lloyd, summaries) of "
                        f"{len(rs)} (sequence, KV head) pairs of layer 0, one per residual count ({built}; "
                        f"context {s}), and {n_dec} decode layer-steps for all {B}x{wl.hq} query heads "
                        f"({t_dec:.2f}s each); extrapolated to the whole job ({job:.0f}s) with each head priced "
                        f"at the measured head of its r"),
                seconds_measured=spent + t_dec * n_dec)


def build_call_flops(wl, res):
    """Algorithmic flops of one construction call: the window logits once
    (2 d per visible (window row, key) pair, causal inside the window, every
    query head of the group) and T Lloyd assignments of 2 |E| r' d each
    (the method's products; the split-bf16 centres' second MFMA pass is not
    counted)."""
    B, Hkv, G, d, w, T = wl.batch, wl.hkv, wl.group, wl.d, wl.window, wl.lloyd_iters
    score = lloyd = 0.0
    for b in range(B):
        s = wl.ctx[b]
        pairs = w * (s - w) + w * (w + 1) // 2
        for h in range(Hkv):
            r = int(res[b][h])
            m = wl.budget[b] - r
            score += G * pairs * 2 * d
            if s > m:
                nE = s - m
                lloyd += T * 2 * nE * min(r, nE) * d
    return score, lloyd


def counters_from_profile(name, src_hash):
    """A committed rocprofv3 counter summary (profiles/<name>.json), if it was
    taken on the current construction source."""
    path = os.path.join(ROOT, "profiles", name + ".json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("build_source_sha256_16") != src_hash:
        return None
    return rec


def progress(msg):
    """One line on stderr per finished phase (the JSON result goes to stdout)."""
    print(f"bench: {msg}", file=sys.stderr, flush=True)


def per_config_run(rk, torch, np, synth, idx, dev, reps, ragged):
    """Construction and decode of another workload, after the main job's
    buffers are freed. Every layer is generated into one reused prefill
    buffer, built once untimed and then `reps` times between events on the
    launch stream (inputs resident in HBM); then every decode call of the
    workload runs once as a warm-up, the cache lengths are reset to the built
    ones, and the whole decode phase is captured as one HIP graph and
    replayed between events. Returns the measurements."""
    wl = synth.workload(idx)
    L, B, Hq, Hkv, d = wl.layers, wl.batch, wl.hq, wl.hkv, wl.d
    elem = 2 if wl.dtype == "bf16" else 4
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    C, Rcap, S = wl.slot_cap, wl.res_cap, wl.max_ctx
    shape = rk.make_shape(B, Hq, Hkv, d, wl.dtype, C, Rcap)
    params = rk.BuildParams(S, wl.window, wl.window, wl.lloyd_iters)
    seq = np.asarray(wl.ctx, np.int32)
    bud = np.asarray(wl.budget, np.int32)
    res_layers = [np.asarray(wl.res[l], np.int32) for l in range(L)]
    nws = max(rk.reskv_build_workspace_size(shape, params, seq, bud, res_layers[l].reshape(-1)) for l in range(L))
    build_ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    buf = dict(K=torch.empty((B, Hkv, S, d), dtype=tdt, device=dev),
               V=torch.empty((B, Hkv, S, d), dtype=tdt, device=dev))
    stream = torch.cuda.current_stream()
    caches, dec_in, built_len = [], [], []
    build_ms = 0.0
    for l in range(L):
        x = synth.gen_layer_device(wl, l, dev, out=buf)
        c = dict(kc=torch.empty((B, Hkv, C, d), dtype=tdt, device=dev),
                 vc=torch.empty((B, Hkv, C, d), dtype=tdt, device=dev),
                 logc=torch.empty((B, Hkv, Rcap), device=dev),
                 main_idx=torch.empty((B, Hkv, C), dtype=torch.int32, device=dev),
                 res_len=torch.empty((B * Hkv,), dtype=torch.int32, device=dev),
                 main_len=torch.empty((B * Hkv,), dtype=torch.int32, device=dev))

        def build():
            rk.reskv_build_cache(shape, params, buf["K"], buf["V"], seq, x["q_obs"], bud, res_layers[l].reshape(-1),
                                 c["kc"], c["vc"], c["logc"], c["main_idx"], c["res_len"], c["main_len"], build_ws)

        build()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            build()
        e1.record(stream)
        torch.cuda.synchronize()
        build_ms += e0.elapsed_time(e1) / reps
        if l == 0 or l == L - 1:
            progress(f"{wl.name}: layer {l} built")
        caches.append(c)
        built_len.append(c["main_len"].clone())
        dec_in.append(dict(q=x["q_dec"], kn=x["k_new"], vn=x["v_new"], tau=x["tau"]))
        del x
    del buf
    dec_ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, d), device=dev)
    gates = [[rk.make_gate(tau=dec_in[l]["tau"][t], alpha=wl.alpha, g_min=wl.g_min, beta=wl.beta)
              for t in range(wl.steps)] for l in range(L)]

    rag_ws = None
    if ragged:
        rag_ws = torch.empty(rk.reskv_decode_ragged_workspace_size(shape), dtype=torch.uint8, device=dev)

    def calls_on(st, rag):
        prep = rk.prepare_decode_attn_ragged if rag else rk.prepare_decode_attn
        ws = rag_ws if rag else dec_ws
        return [[prep(shape, gates[l][t], dec_in[l]["q"][t], caches[l]["kc"], caches[l]["vc"], caches[l]["logc"],
                      caches[l]["res_len"], caches[l]["main_len"], out, ws, k_new=dec_in[l]["kn"][t],
                      v_new=dec_in[l]["vn"][t], stream=st)
                 for l in range(L)] for t in range(wl.steps)]

    def timed_decode(rag):
        """Warm-up pass, lengths reset, then the whole decode phase captured
        as one HIP graph and replayed between events; the appends must have
        grown every head by the number of steps."""
        for step in calls_on(stream, rag):
            for call in step:
                call()
        torch.cuda.synchronize()
        for l in range(L):
            caches[l]["main_len"].copy_(built_len[l])
        torch.cuda.synchronize()
        cap = torch.cuda.Stream()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            for step in calls_on(cap, rag):
                for call in step:
                    call()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
        ended = np.concatenate([c["main_len"].cpu().numpy() for c in caches])
        started = np.concatenate([x.cpu().numpy() for x in built_len])
        assert (ended == started + wl.steps).all(), "decode appends missing"
        del g
        return e0.elapsed_time(e1)

    # the per-head schedule (reskv_decode_attn), then for ragged batches the
    # balanced-range one (reskv_decode_attn_ragged) beside it, each from the
    # built lengths
    dec_ms = timed_decode(False)
    rag_ms = timed_decode(True) if ragged else None
    progress(f"{wl.name}: decode phase timed")
    dec_bytes = 0
    for l in range(L):
        r = res_layers[l].astype(np.int64)
        m0 = np.minimum(np.asarray(wl.budget)[:, None] - r, np.asarray(wl.ctx)[:, None])
        for t in range(wl.steps):
            dec_bytes += decode_call_bytes(B, Hq, Hkv, d, elem, r, np.minimum(m0 + t + 1, C - r))
    calls = L * wl.steps
    b_bytes = sum(build_call_bytes(wl, elem, res_layers[l]) for l in range(L))
    f_score = f_lloyd = 0.0
    for l in range(L):
        fs, fl = build_call_flops(wl, res_layers[l])
        f_score += fs
        f_lloyd += fl
    dec_gbs = dec_bytes / (dec_ms * 1e-3) / 1e9
    b_tflops = (f_score + f_lloyd) / (build_ms * 1e-3) / 1e12
    del caches, dec_in, built_len, build_ws, dec_ws, rag_ws
    torch.cuda.empty_cache()
    return wl, dict(
        workload=workload_text(wl, L, what="construction of all layers + all decode steps, timed apart"),
        layers=L, decode_steps=wl.steps,
        build_ms_per_layer=build_ms / L, build_gbs=b_bytes / (build_ms * 1e-3) / 1e9,
        build_bytes_per_layer=b_bytes / L, build_tflop_per_layer=(f_score + f_lloyd) / L / 1e12,
        build_roofline={"bound": "mfma" if (f_score + f_lloyd) / 2.5e15 > b_bytes / 8e12 else "hbm",
                        "achieved": b_tflops, "peak": 2500.0, "unit": "TFLOP/s", "frac": b_tflops / 2500.0,
                        "hbm_gbs": b_bytes / (build_ms * 1e-3) / 1e9,
                        "floor_ms_per_layer": max((f_score + f_lloyd) / 2.5e15, b_bytes / 8e12) * 1e3 / L},
        decode_us_per_call=dec_ms * 1e3 / calls, decode_bytes_per_call=dec_bytes / calls, decode_gbs=dec_gbs,
        decode_tokens_per_s=B * L * wl.steps / (dec_ms * 1e-3),
        decode_roofline={"bound": "hbm", "achieved": dec_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": dec_gbs / HBM_PEAK_GBS, "calls_timed": calls,
                         "kernel": ("reskv_decode_attn (decode_head: one block per (sequence, KV head), append "
                                    "fused)" if B * Hkv >= 256 else "reskv_decode_attn (decode_split + "
                                    "decode_combine, append fused)")},
        decode_us_per_call_ragged_schedule=(rag_ms * 1e3 / calls if rag_ms is not None else None),
        decode_launch="hip_graph")


def workload_text(wl, L, what="step = construction of all layers + all decode steps"):
    """What one timed step covers, with the workload's sizes."""
    import numpy as np
    ctx = (f"context {wl.ctx[0]}" if min(wl.ctx) == max(wl.ctx)
           else f"contexts {min(wl.ctx)}-{max(wl.ctx)} (ragged)")
    bud = (f"budget {wl.budget[0]}" if min(wl.budget) == max(wl.budget)
           else f"budgets {sorted(set(int(b) for b in wl.budget))}")
    rs = sorted(set(int(x) for x in np.unique(wl.res[:L])))
    rtxt = f"residual r per (layer, head) in {{{','.join(map(str, rs))}}}" if len(rs) <= 6 else \
        f"residual r per (layer, head) from {rs[0]} to {rs[-1]}"
    return (f"{wl.name}: {L} layers x (Hq {wl.hq} / Hkv {wl.hkv}, head_dim {wl.d}), batch {wl.batch}, {ctx} -> "
            f"{bud} per KV head, {rtxt}, {wl.steps} decode steps with appends; {what}")


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py measures one GPU: the ResKV hot path here is built and timed on a "
                                   "single MI355X and has no multi-GPU mode (every (sequence, KV head) is "
                                   "independent, so sharding by sequence or KV head needs no communication)",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2607_29591_amd import reskv as rk
    from paper_2607_29591_amd import synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    rk.lib()  # fail loudly if the HIP library is missing
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.workload(args.workload)
    if args.decode_steps is not None:
        wl.steps = args.decode_steps
    if args.layers is not None:
        wl.layers = args.layers
        wl.res = wl.res[:args.layers]
    L, B, Hq, Hkv, d = wl.layers, wl.batch, wl.hq, wl.hkv, wl.d
    elem = 2 if wl.dtype == "bf16" else 4
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    C, Rcap, S = max(wl.slot_cap, args.slot_cap or 0), wl.res_cap, wl.max_ctx
    shape = rk.make_shape(B, Hq, Hkv, d, wl.dtype, C, Rcap)
    params = rk.BuildParams(S, wl.window, wl.window, wl.lloyd_iters)

    t_setup = time.perf_counter()
    layers = []
    for l in range(L):
        x = synth.gen_layer_device(wl, l, dev)
        layers.append(x)
        if l == 0 or l == L - 1 or args.mode == "decode":
            progress(f"input of layer {l} generated")
    q_stage = torch.stack([x["q_dec"] for x in layers])      # [L, steps, B, Hq, d]
    kn_stage = torch.stack([x["k_new"] for x in layers])
    vn_stage = torch.stack([x["v_new"] for x in layers])
    tau_stage = torch.stack([x["tau"] for x in layers])       # [L, steps, B, Hq]
    for x in layers:
        del x["q_dec"], x["k_new"], x["v_new"], x["tau"]
    caches = []
    for l in range(L):
        caches.append(dict(kc=torch.empty((B, Hkv, C, d), dtype=tdt, device=dev),
                           vc=torch.empty((B, Hkv, C, d), dtype=tdt, device=dev),
                           logc=torch.empty((B, Hkv, Rcap), device=dev),
                           main_idx=torch.empty((B, Hkv, C), dtype=torch.int32, device=dev),
                           res_len=torch.empty((B * Hkv,), dtype=torch.int32, device=dev),
                           main_len=torch.empty((B * Hkv,), dtype=torch.int32, device=dev)))
    res_layers = [np.asarray(wl.res[l], np.int32) for l in range(L)]
    nws = max(rk.reskv_build_workspace_size(shape, params, layers[l]["seq_len"], layers[l]["budget"],
                                            res_layers[l].reshape(-1)) for l in range(L))
    build_ws = torch.empty(nws, dtype=torch.uint8, device=dev)
    dec_ws = torch.empty(rk.reskv_decode_workspace_size(shape), dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, d), device=dev)
    gates = [[rk.make_gate(tau=tau_stage[l, t], alpha=wl.alpha, g_min=wl.g_min, beta=wl.beta)
              for t in range(wl.steps)] for l in range(L)]
    torch.cuda.synchronize()
    t_setup = time.perf_counter() - t_setup

    stream = torch.cuda.current_stream()
    # every decode call of a job, with its arguments marshalled once: the
    # timed loop only issues the launches
    dec_calls = [[rk.prepare_decode_attn(shape, gates[l][t], q_stage[l, t], caches[l]["kc"], caches[l]["vc"],
                                         caches[l]["logc"], caches[l]["res_len"], caches[l]["main_len"], out,
                                         dec_ws, k_new=kn_stage[l, t], v_new=vn_stage[l, t], stream=stream)
                  for l in range(L)] for t in range(wl.steps)]

    dec_graph = None

    def job(record):
        eb0 = torch.cuda.Event(enable_timing=True)
        eb1 = torch.cuda.Event(enable_timing=True)
        eb0.record(stream)
        for l in range(L):
            x, c = layers[l], caches[l]
            rk.reskv_build_cache(shape, params, x["K"], x["V"], x["seq_len"], x["q_obs"], x["budget"],
                                 res_layers[l].reshape(-1), c["kc"], c["vc"], c["logc"], c["main_idx"],
                                 c["res_len"], c["main_len"], build_ws)
        eb1.record(stream)
        if dec_graph is not None:
            dec_graph.replay()
        else:
            for calls in dec_calls:
                for call in calls:  # this step's token is appended inside each decode call
                    call()
        ed = torch.cuda.Event(enable_timing=True)
        ed.record(stream)
        return eb0, eb1, ed

    def capture_decode():
        """All decode calls of a job as one HIP graph (the library enqueues
        kernel launches only), captured on a stream of its own after the
        kernels have run once eagerly."""
        cap = torch.cuda.Stream()
        calls = [[rk.prepare_decode_attn(shape, gates[l][t], q_stage[l, t], caches[l]["kc"], caches[l]["vc"],
                                         caches[l]["logc"], caches[l]["res_len"], caches[l]["main_len"], out,
                                         dec_ws, k_new=kn_stage[l, t], v_new=vn_stage[l, t], stream=cap)
                  for l in range(L)] for t in range(wl.steps)]
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            for step in calls:
                for call in step:
                    call()
        torch.cuda.synchronize()
        return g

    if args.mode == "proxy":
        pr = proxy_runs(rk, torch, wl, shape, layers, caches, L, dev)
        print(json.dumps({"mode": "proxy", "layers": L, **pr}), flush=True)
        return

    if args.mode == "decode":
        src = torch.empty(256 << 20, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        dst.copy_(src)                      # plain copy kernel: 256 MiB read + 256 MiB written
        torch.cuda.synchronize()
        for l in range(L):
            x, c = layers[l], caches[l]
            rk.reskv_build_cache(shape, params, x["K"], x["V"], x["seq_len"], x["q_obs"], x["budget"],
                                 res_layers[l].reshape(-1), c["kc"], c["vc"], c["logc"], c["main_idx"],
                                 c["res_len"], c["main_len"], build_ws)
            torch.cuda.synchronize()
            progress(f"layer {l} built")
        for t in range(args.steps):
            for l in range(L):
                c = caches[l]
                rk.reskv_decode_attn(shape, gates[l][t], q_stage[l, t], c["kc"], c["vc"], c["logc"],
                                     c["res_len"], c["main_len"], out, dec_ws, k_new=kn_stage[l, t],
                                     v_new=vn_stage[l, t])
        torch.cuda.synchronize()
        per_call = []
        for l in range(L):
            r0 = res_layers[l].astype(np.int64)
            m0 = np.minimum(np.asarray(wl.budget)[:, None] - r0, np.asarray(wl.ctx)[:, None])
            for t in range(args.steps):
                per_call.append(decode_call_bytes(B, Hq, Hkv, d, elem, r0, np.minimum(m0 + t + 1, C - r0)))
        print(json.dumps({"mode": "decode", "layers": L, "steps": args.steps,
                          "algorithmic_bytes_per_call": float(np.mean(per_call)),
                          "copy_bytes_each_way": 256 << 20}), flush=True)
        return

    progress(f"setup done ({t_setup:.1f} s)")
    for _ in range(args.warmup):
        job(False)
    progress("warm-up jobs done")
    decode_launch = "eager"
    if not args.eager_decode:
        if args.warmup == 0:
            for call in dec_calls[0]:  # every decode kernel runs once before the capture
                call()
        torch.cuda.synchronize()
        try:
            dec_graph = capture_decode()
            decode_launch = "hip_graph"
        except Exception as exc:  # keep the eager calls
            dec_graph = None
            decode_launch = f"eager (graph capture failed: {exc})"
    torch.cuda.synchronize()
    phase = []
    t0 = time.perf_counter()
    for _ in range(args.steps):
        phase.append(job(True))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1000 / args.steps
    progress(f"{args.steps} timed jobs done ({ms_per_step:.1f} ms each)")
    graph_check = None
    if dec_graph is not None:
        # the replayed job's last output against the same job issued call by call
        out_graph = out.clone()
        dec_graph = None
        job(False)
        torch.cuda.synchronize()
        graph_check = "bitwise equal to eager calls" if torch.equal(out, out_graph) else "MISMATCH with eager calls"
    build_ms = sum(a.elapsed_time(b) for a, b, _ in phase) / args.steps
    decode_ms = sum(b.elapsed_time(c) for _, b, c in phase) / args.steps
    # spread over the timed jobs: per-job decode time and whole-job GPU time
    dec_job_ms = [b.elapsed_time(c) for _, b, c in phase]
    job_ms = [a.elapsed_time(c) for a, _, c in phase]

    # algorithmic bytes
    build_bytes = sum(build_call_bytes(wl, elem, res_layers[l]) for l in range(L))
    dec_bytes_job = 0
    for l in range(L):
        r = res_layers[l].astype(np.int64)
        m0 = np.minimum(np.asarray(wl.budget)[:, None] - r, np.asarray(wl.ctx)[:, None])
        for t in range(wl.steps):
            ml = np.minimum(m0 + t + 1, C - r)
            dec_bytes_job += decode_call_bytes(B, Hq, Hkv, d, elem, r, ml)
    tokens = B * L * wl.steps
    # decode roofline: the decode phase of every timed job is bracketed by
    # events on the stream the calls are launched on; every launch in it is
    # one decode_head, back to back
    calls = L * wl.steps
    avg_ms = decode_ms / calls
    avg_bytes = dec_bytes_job / calls
    achieved = avg_bytes / (avg_ms * 1e-3) / 1e9
    src = source_hash("paper_2607_29591_amd/csrc/decode.hip", "paper_2607_29591_amd/csrc/common.h")
    traffic_ratio = traffic_from_profile(src)
    # counter bytes of the profiled calls, scaled to this job's average call
    traffic = traffic_ratio * avg_bytes if traffic_ratio is not None else None
    cmfma = construction_mfma_from_profile(
        source_hash("paper_2607_29591_amd/csrc/build.hip", "paper_2607_29591_amd/csrc/common.h"))

    result = {
        "metric": ("decode attn tokens/s (batch x layers), whole job: construction of every layer from the "
                   "prefill plus every decode step"),
        "value": tokens / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded; LLM-shaped keys with outlier channels and heavy tokens)",
        "config": {"workload": workload_text(wl, L), "global_batch": B, "seq_len": int(max(wl.ctx)), "layers": L,
                   "decode_steps": wl.steps, "budget": int(max(wl.budget)), "parallelism": "single GPU"},
        "decode_tokens_per_s": tokens / (decode_ms * 1e-3),
        "decode_ms_per_job": decode_ms,
        "decode_gbs": dec_bytes_job / (decode_ms * 1e-3) / 1e9,
        "build_ms_per_layer": build_ms / L,
        "build_gbs": build_bytes / (build_ms * 1e-3) / 1e9,
        "construction_mfma": cmfma,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": ("reskv_decode_attn (one launch per layer-step: decode_head, one block per "
                                "(sequence, KV head), append fused)" if B * Hkv >= 256 and (elem == 2 or d == 64) else
                                "reskv_decode_attn (per layer-step: decode_split over 256-slot blocks with the "
                                "append fused, decode_combine with the gate)"),
                     "bytes_per_call": avg_bytes, "us_per_call": avg_ms * 1e3,
                     "us_per_call_range": [min(dec_job_ms) / calls * 1e3, max(dec_job_ms) / calls * 1e3],
                     "calls_timed": calls * args.steps},
        "job_ms_range": [min(job_ms), max(job_ms)],
        "setup_s": t_setup,
        "decode_launch": decode_launch,
        "decode_graph_check": graph_check,
    }
    if args.proxy_layers > 0:
        # after the timed jobs: construction with the validation proxy choosing r
        result["proxy_build"] = proxy_runs(rk, torch, wl, shape, layers, caches, min(args.proxy_layers, L), dev)
    if args.adakv_layers > 0:
        result["adakv_build"] = adakv_runs(rk, torch, wl, shape, layers, caches, res_layers,
                                           min(args.adakv_layers, L), dev)
    progress("proxy and AdaKV constructions done")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, layers[0], q_stage[0, 0], tau_stage[0, 0], res_layers,
                                              args.cpu_budget_s)
        progress("oracle baseline done")
    others = [int(v) for v in args.per_config.split(",") if v.strip() != ""]
    if others:
        # the main job's buffers go before the other workloads are generated
        del layers, caches, q_stage, kn_stage, vn_stage, tau_stage, dec_calls, build_ws, dec_ws, gates
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        bsrc = source_hash("paper_2607_29591_amd/csrc/build.hip", "paper_2607_29591_amd/csrc/common.h")
        per = {}
        dsrc = source_hash("paper_2607_29591_amd/csrc/decode.hip", "paper_2607_29591_amd/csrc/common.h")
        for idx in others:
            # the ragged GQA-7 batch (budgets and contexts differ per sequence)
            # also decodes with the balanced-range schedule, reported beside
            wl_i, rec = per_config_run(rk, torch, np, synth, idx, dev, args.per_config_reps, ragged=idx == 4)
            names = PROFILES.get(idx, {})
            if "construction" in names:
                rec["construction_mfma"] = construction_mfma_from_profile(bsrc, names["construction"])
            if "decode" in names:
                ratio = traffic_from_profile(dsrc, names["decode"])
                rec["decode_roofline"]["traffic"] = (ratio * rec["decode_bytes_per_call"]
                                                     if ratio is not None else None)
            per[wl_i.name] = rec
        result["per_config"] = per
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
