#!/usr/bin/env python3
"""Throughput of TransX candidate scoring on one MI355X.

One step = one score_candidates call over the whole batch: every request's
serving-event tokens and candidates run through the decoder (self-attention,
cross-attention onto the request's cached behavior K/V, FFN) and the linear
head. The caches are built (untimed) before the timed region; inputs are
resident in HBM when it starts. Prints one JSON line.

  python bench.py [--steps K] [--warmup W] [--workload headline]
  python bench.py --l-local 10        # local-global sparse cross-attention
                                      # (last 10 cached tokens + pooled token)
  python bench.py --actions 3         # k-action softmax decoder head
  python bench.py --events 8          # event-sliced decoding (seq2seq training
                                      # forward): B/8 users x 8 serving events,
                                      # each against its own prefix of the cache

The JSON carries the roofline of the dominant kernel, whose per-launch time
comes from HIP events the library records around its launches on the stream
during the timed steps (tx_profile_*: a few untimed steps with every launch
bracketed pick that kernel and give the per-class table first), the minimum,
median and maximum of the timed steps' own times, and the fp64 CPU oracle's
own throughput on a bounded sample. The per-class table ("kernels") gives
every kernel class's average launch time in those untimed steps, its
algorithmic TFLOP/s and GB/s, and the fraction of the roof that bounds it
(above the ridge of the dtype's arithmetic peak over 8 TB/s: bf16 MFMA, or
the fp32 vector ALUs for fp32 models; HBM below).
"""
from __future__ import annotations

import argparse
import dataclasses
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP32_TFLOPS = 157.3    # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

METRIC = "candidate scores/sec + % bf16 MFMA peak, B=256 L=4096 C=512 on 1 MI355X"


def cross_keys(m, L: int) -> int:
    """Keys each decoder query attends to: the whole cache, or the
    local-global sparse set (last l_local tokens, plus the pooled token)."""
    if m.l_local <= 0:
        return L
    return min(L, m.l_local) + (1 if m.global_pool else 0)


def score_work(wl):
    """Algorithmic flops and bytes of one score call: the contractions the
    decoder must do once the cache exists (QKV/O/cross-Q/cross-O/FFN GEMMs,
    self- and cross-attention, head) and the bytes it must move (cached K/V
    read once, tokens in, scores out, weights once). In the last decoder layer
    serving rows only supply their self-attention keys and values."""
    m = wl.model
    d, F = m.d_model, m.d_ffn
    es = 2 if m.dtype == "bf16" else 4
    f_gemm = f_cross = f_self = 0.0
    for L, S, C in zip(wl.L, wl.S, wl.C):
        N = S + C
        for layer in range(m.n_dec_layers):
            last = layer == m.n_dec_layers - 1
            rows = C if last else N
            f_gemm += (12 * d * d + 4 * d * F) * rows + (4 * d * d * S if last else 0)
            f_cross += 4.0 * cross_keys(m, L) * d * rows
            f_self += (0 if last else 2.0 * d * S * (S + 1)) + 4.0 * d * C * (S + 1)
        f_gemm += 2 * d * C * max(1, m.n_actions)
    kv = sum(m.n_dec_layers * 2 * cross_keys(m, L) * d for L in wl.L) * es
    tok = sum(S + C for S, C in zip(wl.S, wl.C)) * d * es
    wts = m.n_dec_layers * (12 * d * d + 2 * d * F) * es
    return {"flop": f_gemm + f_cross + f_self, "flop_gemm": f_gemm, "flop_cross": f_cross, "flop_self": f_self,
            "bytes": float(kv + tok + 4 * sum(wl.C) + wts), "bytes_kv": float(kv)}


def cpu_baseline(wl, weights, n_req: int):
    """The fp64 oracle's score phase on the first n_req requests, wall clock on
    the host's cores. Its cross-attention cache is seeded N(0,1) data of the
    right shape (the phase's cost does not depend on the values)."""
    import numpy as np
    from oracle import oracle as O
    from paper_2607_28940_amd import inputs as I
    O.build()
    orc = O.Oracle(wl.model, weights)
    m = wl.model
    n_scores = 0
    elapsed = 0.0
    for r in range(n_req):
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([I.SEED_X, wl.cfg_id, 7, r])))
        nk = cross_keys(m, wl.L[r])
        Kx = rng.standard_normal((m.n_dec_layers, nk, m.d_model))
        Vx = rng.standard_normal((m.n_dec_layers, nk, m.d_model))
        Xs = I.request_tokens(wl, r, I.STREAM_SERVING)
        Xc = I.request_tokens(wl, r, I.STREAM_CANDIDATES)
        t0 = time.perf_counter()
        orc.score(Kx, Vx, Xs, Xc)
        elapsed += time.perf_counter() - t0
        n_scores += len(Xc)
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": n_scores / elapsed, "unit": "scores/s", "cores": cores, "kind": "oracle",
            "sample": f"score phase of the fp64 oracle on {n_req} request(s) of the workload "
                      f"({n_scores} scores, {elapsed:.1f} s), cache contents seeded N(0,1)"}


KERNEL_SOURCES = {"cross_attention": "attention.hip", "self_attention": "attention.hip", "gemm": "gemm.hip",
                  "layernorm": "rowops.hip", "scatter": "rowops.hip", "causal_attention": "attention.hip"}


def kernel_source_sha(kernel_class: str):
    import hashlib
    for key, fn in KERNEL_SOURCES.items():
        if key in kernel_class:
            path = os.path.join(ROOT, "paper_2607_28940_amd", "csrc", fn)
            return hashlib.sha256(open(path, "rb").read()).hexdigest()
    return None


def measured_traffic(path: str, kernel_class: str):
    """HBM bytes per launch of `kernel_class` from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary, or None when there is none or the
    kernel's source has changed since the counters were taken."""
    try:
        rec = json.load(open(path)).get(kernel_class)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_sha256") != kernel_source_sha(kernel_class):
        return None
    return rec.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="headline", choices=["headline", "uniform", "ragged", "tiny", "append"])
    ap.add_argument("--l-local", type=int, default=0,
                    help="local-global sparse cross-attention window (0: dense cross-attention, the headline)")
    ap.add_argument("--no-global-token", action="store_true",
                    help="with --l-local: no attention-pooled global token")
    ap.add_argument("--events", type=int, default=0,
                    help="T > 0: B/T users with T serving events each, decoded against prefixes L(t+1)/T")
    ap.add_argument("--actions", type=int, default=0,
                    help="k >= 2: softmax decoder head over k action tokens (0: the scalar logit head)")
    ap.add_argument("--cpu-requests", type=int, default=None,
                    help="requests in the oracle's timed sample (default: about 10 s of CPU work)")
    ap.add_argument("--append", action="store_true",
                    help="workload 'append': each timed step first appends the workload's n_append events to "
                         "every user's cache (through the causal encoder, in place), then scores")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="time without per-launch events")
    ap.add_argument("--profile-steps", type=int, default=3,
                    help="untimed steps with every launch bracketed by events (per-class table)")
    ap.add_argument("--traffic-json", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="HBM bytes per launch from rocprofv3 counters (optional)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="run one plain 1 GiB device copy first (reference for counter scaling)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the serving path shards by request with no exchange between GPUs, "
              "and this build runs on a single MI355X. Use --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    from paper_2607_28940_amd import inputs as I
    from paper_2607_28940_amd import transx as T

    assert torch.cuda.is_available(), "bench.py needs a ROCm GPU"
    torch.cuda.set_device(0)
    wl = I.workload(args.workload)
    if args.l_local > 0:
        wl = dataclasses.replace(wl, model=dataclasses.replace(wl.model, l_local=args.l_local,
                                                               global_pool=not args.no_global_token))
    if args.actions:
        wl = dataclasses.replace(wl, model=dataclasses.replace(wl.model, n_actions=args.actions))
    m = wl.model
    t_setup = time.time()
    weights = I.make_weights(m)
    model = T.Model(m, weights)
    # caches of the users (every request, or B/T users with T events each)
    n_users = max(1, wl.B // args.events) if args.events else wl.B
    users = list(range(n_users))
    if args.append and (wl.n_append <= 0 or args.events):
        print("--append needs a workload with appended events (--workload append) and no --events", file=sys.stderr)
        sys.exit(2)
    extra = 0 if args.no_profile else args.profile_steps  # untimed profiled steps
    grow = wl.n_append * (args.warmup + extra + args.steps) if args.append else 0  # tokens appended per user
    n_pages = sum((wl.L[u] + grow + 63) // 64 for u in users)
    cache = T.KVCache(model, n_pages=n_pages, max_requests=n_users, max_tokens=max(wl.L) + grow)
    # build every user's cache (untimed), a few at a time
    chunk = max(1, (1 << 19) // max(1, max(wl.L)))
    build_ms = 0.0
    for a in range(0, n_users, chunk):
        ids = list(range(a, min(n_users, a + chunk)))
        Xb = T.to_device(I.packed_tokens(wl, I.STREAM_BEHAVIOR, ids, threads=16), m)
        b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        b0.record()
        cache.build(ids, Xb, I.offsets([wl.L[r] for r in ids]), ws_limit=8 << 30)
        b1.record()
        torch.cuda.synchronize()
        build_ms += b0.elapsed_time(b1)
        del Xb
    build_tokens = sum(wl.L[u] for u in users)
    xs = T.to_device(I.packed_tokens(wl, I.STREAM_SERVING, threads=16), m)
    xc = T.to_device(I.packed_tokens(wl, I.STREAM_CANDIDATES, threads=16), m)
    so, co = I.offsets(wl.S), I.offsets(wl.C)
    ids = list(range(wl.B))
    prefix = None
    if args.events:
        # serving event e = t of user u = e // T, decoded against the first
        # L (t + 1) / T cached tokens; the work model counts those prefixes
        ids = [min(e // args.events, n_users - 1) for e in range(wl.B)]
        prefix = [max(1, wl.L[ids[e]] * (e % args.events + 1) // args.events) for e in range(wl.B)]
        wl = dataclasses.replace(wl, L=prefix)

    if args.append:
        xe = T.to_device(I.packed_tokens(wl, I.STREAM_EVENTS, users, threads=16), m)
        eo = I.offsets([wl.n_append] * n_users)

    def step():
        if args.append:
            cache.append(users, xe, eo, ws_limit=8 << 30)
        if prefix is None:
            cache.score(ids, xs, so, xc, co, out=out)
        else:
            cache.score_events(ids, prefix, xs, so, xc, co, out=out)
    out = torch.empty((int(co[-1]), m.n_actions) if m.n_actions else int(co[-1]), dtype=torch.float32,
                      device="cuda")
    torch.cuda.synchronize()
    print(f"# setup {time.time() - t_setup:.1f} s: {n_users} caches built", file=sys.stderr, flush=True)

    if args.calib_copy:
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    prof_all, dom = {}, None
    if not args.no_profile:
        # per-class launch times from untimed profiled steps; the timed steps
        # then bracket only the dominant class's launches with event pairs
        T.profile_enable(True)
        for _ in range(args.profile_steps):
            step()
        torch.cuda.synchronize()
        prof_all = T.profile_read()
        dom = max(prof_all, key=lambda k: prof_all[k]["ms"])
        T.profile_enable(True)
        T.profile_select([dom])
    # one event between consecutive steps: the whole timed region and every
    # step's own time (its distribution goes into the JSON line)
    stream = torch.cuda.current_stream()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for k in range(args.steps):
        step()
        evs[k + 1].record(stream)
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    step_ms = sorted(evs[k].elapsed_time(evs[k + 1]) for k in range(args.steps))
    prof = {}
    if not args.no_profile:
        prof = T.profile_read()
        T.profile_enable(False)
    assert bool(torch.isfinite(out).all()), "non-finite scores"

    if args.append:  # cached length grows by n_append per step; the work model takes the timed average
        avg_len = [L + wl.n_append * (args.warmup + extra + (args.steps + 1) / 2) for L in wl.L]
        work = score_work(dataclasses.replace(wl, L=[int(round(x)) for x in avg_len]))
    else:
        work = score_work(wl)
    n_scores = int(co[-1])
    value = n_scores / (ms / 1e3)
    tflops = work["flop"] / (ms / 1e3) / 1e12
    peak = PEAK_BF16_TFLOPS if m.dtype == "bf16" else PEAK_FP32_TFLOPS

    ridge = peak * 1e12 / (PEAK_HBM_GBS * 1e9)  # flop per byte where the two roofs meet
    arith = "mfma" if m.dtype == "bf16" else "alu"  # fp32 models run on the vector ALUs
    kernels = {}
    for name, p in prof_all.items():
        avg = p["ms"] / p["launches"]
        tf = p["flops"] / (p["ms"] / 1e3) / 1e12 if p["flops"] else None
        gbs = p["bytes"] / (p["ms"] / 1e3) / 1e9
        on_mfma = bool(p["flops"]) and p["flops"] / max(p["bytes"], 1) > ridge
        kernels[name] = {"avg_ms": round(avg, 5), "launches_per_step": p["launches"] / args.profile_steps,
                         "share": round(p["ms"] / (ms * args.profile_steps), 4),
                         "tflops": round(tf, 2) if tf is not None else None, "gbs": round(gbs, 1),
                         "bound": arith if on_mfma else "hbm",
                         "frac": round(tf / peak if on_mfma else gbs / PEAK_HBM_GBS, 4)}
    roofline = None
    if prof.get(dom, {}).get("launches"):
        p = prof[dom]
        avg_s = p["ms"] / p["launches"] / 1e3
        fl_launch, by_launch = p["flops"] / p["launches"], p["bytes"] / p["launches"]
        mfma = fl_launch > 0 and fl_launch / max(by_launch, 1) > ridge
        # the counters were taken on the default headline run: other
        # workloads and modes launch the same kernel on other shapes
        default_run = (args.workload == "headline" and not args.append and not args.events and not args.actions
                       and not args.l_local)
        traffic = measured_traffic(args.traffic_json, dom) if default_run else None
        if mfma:
            ach = fl_launch / avg_s / 1e12
            roofline = {"kernel": dom, "bound": arith, "achieved": round(ach, 2), "peak": peak, "unit": "TFLOP/s",
                        "frac": round(ach / peak, 4), "traffic": traffic,
                        "per_launch": {"flop": fl_launch, "bytes": by_launch, "avg_ms": round(avg_s * 1e3, 5)}}
        else:
            ach = by_launch / avg_s / 1e9
            roofline = {"kernel": dom, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                        "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4), "traffic": traffic,
                        "per_launch": {"flop": fl_launch, "bytes": by_launch, "avg_ms": round(avg_s * 1e3, 5)}}

    cpu = None
    if not args.no_cpu_baseline:
        n_cpu = args.cpu_requests or (32 if m.l_local > 0 else 10)  # ~10 s of the oracle on 16 cores
        cpu = cpu_baseline(wl, weights, min(n_cpu, wl.B))

    sparse = m.l_local > 0
    if sparse:
        mode = f"local-global sparse cross-attention (last {m.l_local} cached tokens" + \
               (" + pooled global token)" if m.global_pool else ")")
    else:
        mode = "dense cross-attention over every cached token"
    head = f"softmax over {m.n_actions} action tokens" if m.n_actions else "scalar logit head"
    append_info = None
    if args.append:
        # the append's launches, from the untimed steps that bracket every
        # launch (the timed steps bracket only the dominant class's)
        enc = {k: v for k, v in prof_all.items() if k.startswith("encode.")}
        app_ms = sum(v["ms"] for v in enc.values()) / args.profile_steps if enc else None
        append_info = {"events_per_step": wl.n_append * n_users,
                       "append_ms_per_step": round(app_ms, 4) if app_ms is not None else None,
                       "events_per_s": round(wl.n_append * n_users / (app_ms / 1e3), 1) if app_ms else None}
    if args.append:
        metric = (f"candidate scores/sec with incremental append: {n_users} users, {wl.n_append} events appended "
                  f"per user (causal encoder against the cached prefix, in place) then scored, {mode}, "
                  f"{head} on 1 MI355X")
    elif args.events:
        metric = (f"candidate scores/sec, event-sliced decoding (seq2seq training forward): {n_users} users x "
                  f"{args.events} serving events of the {args.workload} shape, each against its own cache prefix, "
                  f"with {mode} and {head} on 1 MI355X")
    elif sparse or m.n_actions or args.workload != "headline":
        metric = f"candidate scores/sec, {args.workload} with {mode} and {head} on 1 MI355X"
    else:
        metric = METRIC
    line = {
        "metric": metric,
        "value": round(value, 1), "unit": "scores/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "step_ms": {"min": round(step_ms[0], 4), "median": round(float(np.median(step_ms)), 4),
                    "max": round(step_ms[-1], 4)},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": m.dtype, "data": "synthetic (seeded N(0,1) tokens, N(0,0.02) weights)",
        "config": {"workload": f"{args.workload}: B={wl.B} L={'ragged' if len(set(wl.L)) > 1 else wl.L[0]} "
                               f"S={'ragged' if len(set(wl.S)) > 1 else wl.S[0]} "
                               f"C={'ragged' if len(set(wl.C)) > 1 else wl.C[0]} d={m.d_model} H={m.n_heads} "
                               f"F={m.d_ffn} n_enc={m.n_enc_layers} n_dec={m.n_dec_layers} page=64",
                   "global_batch": wl.B, "scores_per_step": n_scores, "cross_attention": mode,
                   "head": head,
                   "events": ({"users": n_users, "per_user": args.events,
                               "prefixes": "L (t + 1) / T"} if args.events else None),
                   "append": append_info,
                   "build": {"tokens": build_tokens, "ms": round(build_ms, 2),
                             "tokens_per_s": round(build_tokens / (build_ms / 1e3), 1) if build_ms > 0 else None,
                             "note": "kv_cache_build of every cache before the timed steps (untimed in value)"}},
        "mfma_frac_of_peak": round(tflops / peak, 4),
        "achieved_tflops": round(tflops, 2),
        "algorithmic": {"flop_per_step": work["flop"], "bytes_per_step": work["bytes"]},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
