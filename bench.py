"""Benchmark: candidate scores/s of one batched rank call on one MI355X.

One step = one upr_rank_candidates call over the whole workload (every layer's
LayerNorm, Q/K/V projection, candidate cross-attention over the cached
history, output projection, FFN, and the score head), with inputs and the
cache already resident in HBM.  The cache comes from one prior
upr_encode_user call, timed separately.

Prints one JSON line.  Besides the contract fields it carries:
  roofline      - the dominant kernel: algorithmic work per launch / its mean
                  duration (HIP events on the call's stream, from a second,
                  profiled pass over the same steps), against MI355X's peak;
  cpu_baseline  - the CPU oracle ranking a bounded sample of the same
                  workload on this host's cores;
  path_mfma_frac, p10/p50/p90 of the timed steps, p50/p90 single-user latency
  (eager calls, and the same calls replayed from HIP graphs), encode time,
  per-kernel times.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synth import WORKLOADS, make_workload  # noqa: E402

PEAK_MFMA_TFLOPS = 2500.0     # MI355X dense bf16 / fp16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def kernel_work(inp):
    """Algorithmic FLOPs per launch of each rank kernel, and bytes for the
    memory-bound ones (one launch = one layer's pass over all candidates)."""
    d, F, H = inp.d, inp.F, inp.H
    R = int(inp.cand_offsets[-1] - inp.cand_offsets[0])
    n = inp.hist_lens
    k = inp.cand_lens
    es = 2 if inp.dtype == "bf16" else 4
    attn_pairs = int(np.sum(k * (n + 1)))
    # (gemm_o and gemm_down also apply the LayerNorm that follows them, and
    # the last gemm_down the score head, when a row fits their tile: d <= 512;
    # their figure stays the projection FLOPs)
    return {
        "rank.gemm_qkv": ("mfma", 2.0 * R * 3 * d * d),
        "rank.gemm_o": ("mfma", 2.0 * R * d * d),
        "rank.gemm_up": ("mfma", 2.0 * R * F * d),
        "rank.gemm_down": ("mfma", 2.0 * R * d * F),
        # the layer's tail in one launch: O projection (with its residual
        # update and LN2), FFN up and down, the hidden rows kept on chip
        "rank.oproj_ffn": ("mfma", 2.0 * R * d * d + 4.0 * R * d * F),
        # q.k and p.v over the history plus the candidate's own key
        "rank.attn": ("mfma", 4.0 * d * attn_pairs),
        # read the fp32 residual, write the normalised row
        "rank.ln1": ("hbm", R * d * (4.0 + es)),
        "rank.ln2": ("hbm", R * d * (4.0 + es)),
        "rank.score_head": ("hbm", R * d * 4.0 + R * 4.0),
        # read the tokens, write the normalised row (and, for fp32 models,
        # the fp32 residual: bf16 models' first O projection reads the tokens)
        "rank.init_ln1": ("hbm", R * d * (es + es) if inp.dtype == "bf16" else R * d * (es + 4.0 + es)),
    }


# Counter-measured HBM traffic per launch (profiles/traffic.json, written from
# two rocprofv3 --pmc passes per workload, scaled by a plain-copy
# calibration).  A record only applies to its own workload and while every
# source its kernel is built from is unchanged.
TRAFFIC_KEYS = {"rank.attn": "attn", "rank.gemm_qkv": "gemm_qkv", "rank.gemm_o": "gemm_o",
                "rank.oproj_ffn": "oproj_ffn"}


def _traffic_record(kernel, workload):
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))[workload][TRAFFIC_KEYS[kernel]]
        h = hashlib.sha1()
        for src in rec["sources"]:
            h.update(open(os.path.join(ROOT, src), "rb").read())
    except (OSError, KeyError, ValueError, TypeError):
        return None
    return rec if h.hexdigest()[:12] == rec["source_sha1"] else None


def measured_traffic(kernel, workload):
    rec = _traffic_record(kernel, workload)
    return None if rec is None else round(rec["hbm_read_bytes"] + rec["hbm_write_bytes"])


def traffic_provenance(kernel, workload):
    rec = _traffic_record(kernel, workload)
    return (f"profiles/traffic.json[{workload}][{TRAFFIC_KEYS[kernel]}]: rocprofv3 --pmc FETCH_SIZE "
            f"and WRITE_SIZE passes over {', '.join(rec['sources'])} (sha1 {rec['source_sha1']}), "
            f"each scaled by the same counter's reading for a plain device copy "
            f"(x{1 / rec['fetch_factor']:.3f} and x{1 / rec['write_factor']:.3f}); "
            f"replayed while those sources are unchanged")


def path_flops(inp):
    d, F, L = inp.d, inp.F, inp.L
    R = float(inp.cand_offsets[-1] - inp.cand_offsets[0])
    pairs = float(np.sum(inp.cand_lens * (inp.hist_lens + 1)))
    return L * (R * (8 * d * d + 4 * d * F) + 4 * d * pairs) + 2 * d * R


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, budget_s=12.0, single_users=2):
    """Oracle rank on a bounded sample of users (its cache from oracle.encode,
    untimed: encoding is the step before ranking), with the BLAS pool as it
    comes; then single-threaded on `single_users` of those users,
    extrapolated to the whole workload."""
    import oracle
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        blas = ",".join(sorted({i.get("internal_api", "?") for i in threadpool_info()}))
    except Exception:
        threadpool_limits = None
        threads, blas = os.cpu_count() or 1, "unknown"
    done_users, cands, t_rank, caches = [], 0, 0.0, {}
    order = np.argsort(-inp.cand_lens, kind="stable")        # typical users first
    order = order[len(order) // 2:].tolist() + order[: len(order) // 2].tolist()
    for u in order:
        cache = oracle.encode(inp.weights, inp.d, inp.H, inp.L, inp.F, inp.hist_emb,
                              inp.hist_offsets, users=[u])
        if len(caches) < single_users:
            caches[int(u)] = cache
        t0 = time.perf_counter()
        oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                    inp.cand_emb, inp.cand_offsets, users=[u])
        t_rank += time.perf_counter() - t0
        done_users.append(int(u))
        cands += int(inp.cand_lens[u])
        if t_rank >= budget_s:
            break
    out = {"value": cands / t_rank, "unit": "candidate scores/s", "cores": int(threads),
           "kind": "oracle", "cpu": cpu_model(), "blas": blas,
           "sample": f"oracle.rank (numpy float64, BLAS {blas}) over {len(done_users)} of "
                     f"{inp.U} users ({cands} candidates), {t_rank:.1f} s"}
    if threadpool_limits is not None and caches:
        c1, t1 = 0, 0.0
        with threadpool_limits(limits=1):
            for u, cache in caches.items():
                t0 = time.perf_counter()
                oracle.rank(inp.weights, inp.d, inp.H, inp.L, inp.F, cache, inp.hist_offsets,
                            inp.cand_emb, inp.cand_offsets, users=[u])
                t1 += time.perf_counter() - t0
                c1 += int(inp.cand_lens[u])
        total = float(inp.cand_offsets[-1] - inp.cand_offsets[0])
        out["single_thread"] = {
            "value": c1 / t1, "unit": "candidate scores/s", "cores": 1,
            "sample": f"{len(caches)} users ({c1} candidates), {t1:.1f} s",
            "extrapolated_workload_s": round(t1 * total / c1, 1)}
    return out


def actions_topk(args, inp, model, kv, hs, cs, C, Kc, ev, stream):
    """The serving step after scoring (paper Sec. 3, L0 + L1 deployment): the
    same forward pass with C = 3 per-action heads (hidden d/2), sigmoid
    probabilities, utility, and each user's top 1000 by utility.  One step =
    one upr_rank_actions over every candidate + one upr_topk_by_utility."""
    import torch
    from paper_2606_00422_amd import upr
    from synth import DEFAULT_UTILITY, make_heads
    n_act, hidden, K = len(DEFAULT_UTILITY), inp.d // 2, 1000
    heads = upr.Heads(model, n_act, hidden, make_heads(inp.d, n_act, hidden, dtype=inp.dtype,
                                                       seed=args.seed))
    U = inp.U
    probs = torch.empty((max(Kc, 1), n_act), dtype=torch.float32, device="cuda")
    util = torch.empty(max(Kc, 1), dtype=torch.float32, device="cuda")
    rows = torch.empty((max(U, 1), K), dtype=torch.int32, device="cuda")
    vals = torch.empty((max(U, 1), K), dtype=torch.float32, device="cuda")
    ws = model.workspace(upr.upr_rank_actions_workspace_bytes(model.handle, heads.handle, hs, cs))
    uw = np.asarray(DEFAULT_UTILITY, dtype=np.float32)

    def step():
        upr.upr_rank_actions(model.handle, heads.handle, kv, hs, C.data_ptr(), cs, uw,
                             probs.data_ptr(), util.data_ptr(), ws.data_ptr(), ws.numel(), stream)
        upr.upr_topk_by_utility(util.data_ptr(), cs, K, rows.data_ptr(), vals.data_ptr(), stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    assert bool(torch.isfinite(probs[:Kc]).all()), "non-finite action probabilities"
    upr.upr_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = upr.upr_profile_read()
    upr.upr_profile_enable(False)
    heads.close()
    extra = {k: round(v[1] / v[0], 5) for k, v in prof.items()
             if k in ("rank.lnf", "rank.heads_hidden", "rank.heads_out", "topk")}
    return {"ms_per_step": round(ms, 4), "candidates_per_s": round(Kc / (ms * 1e-3), 1),
            "n_actions": n_act, "head_hidden": hidden, "K": K,
            "utility_weights": list(DEFAULT_UTILITY), "extra_kernels_avg_ms": extra}


def mxfp8_rank(args, inp, kv, hs, cs, C, Kc, ev, stream, work):
    """The fp8 projection variant (paper Sec. 3, FP8 quantization; NEXT-3):
    the same rank call on a UPR_BF16_MXFP8 model of the same weights, reusing
    the cache (encode is unchanged).  Reported beside the headline, never as
    it: the headline workload is bf16."""
    import torch
    from paper_2606_00422_amd import upr
    cfg = upr.make_config(inp.d, inp.H, inp.L, inp.F, "bf16_mxfp8")
    model = upr.Model(cfg, inp.weights)
    scores = torch.empty(max(Kc, 1), dtype=torch.float32, device="cuda")
    ws = model.workspace(upr.upr_rank_workspace_bytes(model.handle, hs, cs))

    def step():
        upr.upr_rank_candidates(model.handle, kv, hs, C.data_ptr(), cs, scores.data_ptr(),
                                ws.data_ptr(), ws.numel(), stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = ev(), ev()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    assert bool(torch.isfinite(scores[:Kc]).all()), "non-finite fp8 scores"
    upr.upr_profile_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    prof = upr.upr_profile_read()
    upr.upr_profile_enable(False)
    model.close()
    kernels = {}
    for name, (launches, total) in sorted(prof.items()):
        avg = total / launches
        entry = {"launches_per_step": launches / args.steps, "avg_ms": round(avg, 5)}
        if name in work and work[name][0] == "mfma":
            entry["tflops"] = round(work[name][1] / (avg * 1e-3) / 1e12, 2)
        kernels[name] = entry
    return {"ms_per_step": round(ms, 4), "candidates_per_s": round(Kc / (ms * 1e-3), 1),
            "projections": "MXFP8 (E4M3, E8M0 scale per 32), peak 5.0 PFLOP/s dense fp8",
            "kernels": kernels}


def encode_flops(inp):
    """Algorithmic FLOPs of one upr_encode_user over the workload's histories:
    every layer's Q/K/V projection (the cache), and for all but the last
    layer the causal attention (q.k and p.v over the n(n+1)/2 visible
    pairs), the output projection and the FFN; the last layer stops once its
    keys and values are in the cache."""
    d, F, L = inp.d, inp.F, inp.L
    n = inp.hist_lens.astype(np.float64)
    per_layer_qkv = 6.0 * d * d * n.sum()
    per_layer_rest = (2.0 * d * d + 4.0 * d * F) * n.sum() + 2.0 * d * np.sum(n * (n + 1))
    return L * per_layer_qkv + (L - 1) * per_layer_rest


def dominant_roofline(prof, work, workload):
    dom = max((n for n in prof if n in work), key=lambda n: prof[n][1])
    bound, amount = work[dom]
    avg_s = prof[dom][1] / prof[dom][0] * 1e-3
    traffic = measured_traffic(dom, workload)
    if bound == "mfma":
        achieved = amount / avg_s / 1e12
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(achieved, 2),
                "peak": PEAK_MFMA_TFLOPS, "unit": "TFLOP/s",
                "frac": round(achieved / PEAK_MFMA_TFLOPS, 4), "traffic": traffic}
    else:
        achieved = amount / avg_s / 1e9
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(achieved, 1),
                "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": traffic}
    roof["work_per_launch"] = amount
    roof["avg_launch_ms"] = round(avg_s * 1e3, 5)
    roof["traffic_from"] = (traffic_provenance(dom, workload) if traffic is not None else
                            "null: no counter record for this kernel source and workload")
    return roof


def measure(name, args, full):
    """One workload: encode once (timed), then `args.steps` timed rank steps,
    then the same steps again with per-kernel HIP events.  `full` adds the
    single-user latency passes and the variant measurements."""
    import torch
    from paper_2606_00422_amd import upr

    inp = make_workload(name, seed=args.seed)
    cfg = upr.make_config(inp.d, inp.H, inp.L, inp.F, inp.dtype)
    model = upr.Model(cfg, inp.weights)
    tdt = torch.bfloat16 if inp.dtype == "bf16" else torch.float32
    X = torch.from_numpy(inp.hist_emb).cuda().to(tdt)
    C = torch.from_numpy(inp.cand_emb).cuda().to(tdt)
    hoff = np.ascontiguousarray(inp.hist_offsets, np.int32)
    coff = np.ascontiguousarray(inp.cand_offsets, np.int32)
    hoff_d = torch.from_numpy(hoff).cuda()
    coff_d = torch.from_numpy(coff).cuda()
    T, Kc = int(hoff[-1]), int(coff[-1])
    cache = model.new_cache(max(T, 1))
    scores = torch.empty(max(Kc, 1), dtype=torch.float32, device="cuda")
    hs, cs = upr.segments(hoff, hoff_d), upr.segments(coff, coff_d)
    ws = model.workspace(max(upr.upr_encode_workspace_bytes(model.handle, hs),
                             upr.upr_rank_workspace_bytes(model.handle, hs, cs)))
    stream = upr.current_stream()
    kv = upr.upr_kv_cache(cache.data_ptr(), cache.shape[3])

    def encode():
        upr.upr_encode_user(model.handle, X.data_ptr(), hs, kv, ws.data_ptr(), ws.numel(), stream)

    flush = torch.empty(512 << 20, dtype=torch.uint8, device="cuda") if args.flush_mall else None

    def rank(h=hs, c=cs, st=None):
        if flush is not None and st is None:
            flush.fill_(1)
        upr.upr_rank_candidates(model.handle, kv, h, C.data_ptr(), c, scores.data_ptr(),
                                ws.data_ptr(), ws.numel(), stream if st is None else st)

    ev = lambda: torch.cuda.Event(enable_timing=True)
    encode()
    torch.cuda.synchronize()
    enc = []
    for _ in range(3):
        e0, e1 = ev(), ev()
        e0.record()
        encode()
        e1.record()
        torch.cuda.synchronize()
        enc.append(e0.elapsed_time(e1))
    encode_ms = float(np.median(enc))

    for _ in range(args.warmup):
        rank()
    torch.cuda.synchronize()
    # timed region: one event between consecutive steps (no per-kernel events)
    evs = [ev() for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for i in range(args.steps):
        rank()
        evs[i + 1].record()
    torch.cuda.synchronize()
    ms = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    assert bool(torch.isfinite(scores[:Kc]).all()), f"{name}: non-finite scores"

    # profiled pass over the same steps: per-kernel HIP events on the stream
    upr.upr_profile_enable(True)
    for _ in range(args.steps):
        rank()
    torch.cuda.synchronize()
    prof = upr.upr_profile_read()
    upr.upr_profile_enable(False)

    work = kernel_work(inp)
    kernels = {}
    for kname, (launches, total) in sorted(prof.items()):
        avg = total / launches
        entry = {"launches_per_step": launches / args.steps, "avg_ms": round(avg, 5)}
        if kname in work:
            bound, amount = work[kname]
            if bound == "mfma":
                entry["tflops"] = round(amount / (avg * 1e-3) / 1e12, 2)
            else:
                entry["gbs"] = round(amount / (avg * 1e-3) / 1e9, 1)
        kernels[kname] = entry
    flops = path_flops(inp)
    eflops = encode_flops(inp)
    res = {
        "ms_per_step": round(ms, 4),
        "value": round(Kc / (ms * 1e-3), 1),
        "unit": "candidate scores/s",
        "config": {"workload": name, "users": inp.U, "flush_mall": bool(args.flush_mall),
                   "history_rows": T, "candidate_rows": Kc, "d_model": inp.d,
                   "heads": inp.H, "layers": inp.L, "d_ff": inp.F},
        "path_tflops": round(flops / (ms * 1e-3) / 1e12, 2),
        "path_mfma_frac": round(flops / (ms * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4),
        "step_ms": {"p10": round(float(np.percentile(per_step, 10)), 4),
                    "p50": round(float(np.percentile(per_step, 50)), 4),
                    "p90": round(float(np.percentile(per_step, 90)), 4)},
        "roofline": dominant_roofline(prof, work, name),
        "encode_ms": round(encode_ms, 3),
        "encode_roofline": {"bound": "mfma", "flops": eflops,
                            "achieved": round(eflops / (encode_ms * 1e-3) / 1e12, 2),
                            "peak": PEAK_MFMA_TFLOPS, "unit": "TFLOP/s",
                            "frac": round(eflops / (encode_ms * 1e-3) / 1e12 / PEAK_MFMA_TFLOPS, 4)},
        "kernels": kernels,
    }
    if not full:
        model.close()
        return res, inp

    # single-user calls (sub-range of the packed buffers), per-call latency
    lat = []
    for _ in range(args.user_reps):
        for u in range(inp.U):
            h1 = upr.segments(np.ascontiguousarray(hoff[u:u + 2]), hoff_d[u:u + 2])
            c1 = upr.segments(np.ascontiguousarray(coff[u:u + 2]), coff_d[u:u + 2])
            a, b = ev(), ev()
            a.record()
            rank(h1, c1)
            b.record()
            torch.cuda.synchronize()
            lat.append(a.elapsed_time(b))
    lat = np.array(lat) if lat else np.array([np.nan])

    # the same single-user calls captured once each into a HIP graph and
    # replayed; every replay is checked bit for bit against the eager result
    # (the user's scores are overwritten with NaN between replays)
    glat = []
    for u in range(inp.U if args.user_reps > 0 else 0):
        h1 = upr.segments(np.ascontiguousarray(hoff[u:u + 2]), hoff_d[u:u + 2])
        c1 = upr.segments(np.ascontiguousarray(coff[u:u + 2]), coff_d[u:u + 2])
        sl = slice(int(coff[u]), int(coff[u + 1]))
        rank(h1, c1)
        torch.cuda.synchronize()
        ref = scores[sl].clone()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            rank(h1, c1, upr.current_stream())
        for _ in range(args.user_reps):
            scores[sl].fill_(float("nan"))
            a, b = ev(), ev()
            a.record()
            g.replay()
            b.record()
            torch.cuda.synchronize()
            glat.append(a.elapsed_time(b))
            assert torch.equal(scores[sl], ref), f"graph replay of user {u} differs from eager"
        del g
    glat = np.array(glat) if glat else np.array([np.nan])

    def pct(v, q):          # null when the pass was skipped (JSON has no NaN)
        return None if np.all(np.isnan(v)) else round(float(np.nanpercentile(v, q)), 4)

    res["user_latency_ms"] = {"p50": pct(lat, 50), "p90": pct(lat, 90),
                              "calls": int(np.sum(~np.isnan(lat)))}
    res["user_latency_graph_ms"] = {"p50": pct(glat, 50), "p90": pct(glat, 90),
                                    "replays": int(np.sum(~np.isnan(glat)))}
    if not args.no_actions:
        res["actions_topk"] = actions_topk(args, inp, model, kv, hs, cs, C, Kc, ev, stream)
    if not args.no_mxfp8 and inp.dtype == "bf16" and inp.d % 256 == 0 and inp.F % 128 == 0:
        res["mxfp8"] = mxfp8_rank(args, inp, kv, hs, cs, C, Kc, ev, stream, work)
    model.close()
    return res, inp


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="u64_n1024_k2000", choices=sorted(WORKLOADS))
    ap.add_argument("--others", default="u16_n256_k1000,ragged_u64,u8_n8192_k4096",
                    help="comma-separated workloads measured after the headline, reported in "
                         "the same line under 'workloads' ('' for none)")
    ap.add_argument("--user-reps", type=int, default=3, help="reps of the per-user latency pass")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-actions", action="store_true",
                    help="skip the per-action heads + utility top-K measurement")
    ap.add_argument("--no-mxfp8", action="store_true",
                    help="skip the fp8-projection variant's measurement")
    ap.add_argument("--flush-mall", action="store_true",
                    help="write a 512 MiB scratch buffer before every rank step (evicts the "
                         "256 MB MALL; for counter runs, not for the headline number)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): this path has no "
              "multi-GPU mode; per-GPU work is independent by user.", file=sys.stderr)
        sys.exit(2)

    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    print(f"[bench] {args.workload}: {args.steps} steps after {args.warmup} warmup",
          file=sys.stderr, flush=True)
    head, inp = measure(args.workload, args, full=True)
    others = {}
    for name in [w for w in args.others.split(",") if w and w != args.workload]:
        print(f"[bench] {name}", file=sys.stderr, flush=True)
        torch.cuda.empty_cache()
        res, _ = measure(name, args, full=False)
        others[name] = res
    out = {
        "metric": "candidate scores/sec (1 GPU)",
        "value": head.pop("value"),
        "unit": head.pop("unit"),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16+fp16" if inp.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": head.pop("config"),
        "roofline": head.pop("roofline"),
    }
    out.update(head)
    out["workloads"] = others
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(inp)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
