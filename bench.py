"""Benchmark of the expert-choice MoE layer on one MI355X.

A step is one pass of the whole layer over one batch: routing (router GEMM +
softmax, column top-k), gather, SwiGLU expert grouped GEMMs, combine, and the
full backward (gate gradient, grouped dgrad/wgrad GEMMs, router backward).
Default workload: 8 sequences x 2048 tokens, d = 2048, 64 experts of hidden
1024, per-sequence capacity c(t) = 12 - 8t (mask ratio t ~ U(0,1)), bf16
storage, forward + backward.  Prints ONE JSON line on stdout.

    python bench.py [--steps K] [--warmup W]
                    [--workload train|train_shared|static|timestep|fine|decode|tiny]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sqlite3
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "EC-MoE layer tokens/s fwd and fwd+bwd; grouped-GEMM MFMA util % and route GB/s"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
GEMM_STAGES = {"gemm_w13_swiglu", "gemm_w2", "gemm_dA_swiglu_bwd", "gemm_dW2", "gemm_dXe",
               "gemm_dW13", "router_dx", "router_dwg", "shared_w13_swiglu", "shared_w2",
               "shared_dA_swiglu_bwd", "shared_dW2", "shared_dX", "shared_dW13"}


# kernel-symbol stage tags of the grouped GEMMs (gemm_dma_kernel's last template argument)
GEMM_TAGS = {"gemm_w13_swiglu": 1, "gemm_w2": 2, "gemm_dA_swiglu_bwd": 3, "gemm_dXe": 4,
             "gemm_dW2": 5, "gemm_dW13": 6, "router_dx": 7, "router_dwg": 8,
             "shared_w13_swiglu": 9, "shared_w2": 10, "shared_dA_swiglu_bwd": 11, "shared_dX": 12,
             "shared_dW2": 13, "shared_dW13": 14}
CSRC = "paper_2604_01622_amd/csrc/"
# the sources each stage's kernels are built from (a record of counters stays valid
# while their code is unchanged)
STAGE_SOURCES = {"router": ["router.hip"], "topk": ["topk.hip"],
                 "combine": ["movement.hip"], "bwd_combine": ["movement.hip"],
                 "router_dz": ["movement.hip"], "router_dwg_reduce": ["gemm.hip"]}
SIMD_NUM = 256 * 4   # MI355X: 256 CUs of 4 SIMDs
CALIB_BYTES = 1 << 30   # plain elementwise copy used to scale the byte counters
FLUSH_BYTES = 512 << 20  # cold-cache steps: twice the 256 MiB last-level (MALL) cache


def sources_hash(stage="gemm"):
    """Hash of the code of a stage's sources and the shared header (comments and
    whitespace removed), so that stored counters stay valid across comment-only edits."""
    h = hashlib.sha256()
    for f in [CSRC + x for x in STAGE_SOURCES.get(stage, ["gemm.hip"])] + [CSRC + "ec_common.h"]:
        with open(os.path.join(ROOT, f), encoding="utf-8") as fh:
            src = fh.read()
        src = re.sub(r"/\*.*?\*/", " ", src, flags=re.S)
        src = re.sub(r"//[^\n]*", " ", src)
        h.update(" ".join(src.split()).encode())
    return h.hexdigest()[:16]


def stage_of_kernel(name):
    """Stage of a kernel from its name: a gemm_dma_kernel instantiation by its
    stage-tag template argument (the eleventh: BM, BN, WGM, WGN, KSTEP, STAGES, A_KC,
    B_KC, EPI, OUT_F32, TAG, OPT), the other kernels by their names."""
    m = re.search(r"gemm_dma_kernel<([^>]*)>", name)
    if not m:
        for key, st in (("router_softmax", "router"), ("topk_col_kernel", "topk"),
                        ("topk_kernel", "topk"), ("router_dz_kernel", "router_dz"),
                        ("splitk_reduce_kernel", "router_dwg_reduce")):
            if key in name:
                return st
        c = re.search(r"combine_kernel<[^>]*,\s*(true|false)>", name)
        if c:
            return "bwd_combine" if c.group(1) == "true" else "combine"
        return None
    args = [a.strip() for a in m.group(1).split(",")]
    if len(args) < 11 or not args[10].isdigit():
        return None
    tag = int(args[10])
    return next((k for k, v in GEMM_TAGS.items() if v == tag), None)


def pmc_per_dispatch(db, counter):
    """{kernel name: [value per dispatch]} for one counter of a rocprofv3 --pmc database:
    the sum over the counter's instances, except GRBM counters (one per XCD), whose
    maximum is the dispatch's value (as in rocprof's derived metrics)."""
    c = sqlite3.connect(db)
    out = {}
    agg = "max" if counter.startswith("GRBM") else "sum"
    for name, did, v in c.execute(
            f"select name, dispatch_id, {agg}(counter_value) from pmc_events where counter_name = ? "
            "group by name, dispatch_id order by dispatch_id", (counter,)):
        out.setdefault(name, []).append(v)
    return out


def counters_from(dbs, workload):
    """Per-stage medians of the counters in rocprofv3 --pmc databases (each run with
    --kernel-trace, so that the durations under counting come along), with the MFMA
    utilisation SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE x SIMDs) and the clock
    GRBM_GUI_ACTIVE / duration."""
    import statistics as stat
    per = {}
    for db in dbs:
        c = sqlite3.connect(db)
        names = [r[0] for r in c.execute("select distinct counter_name from pmc_events")]
        for cn in names:
            for name, vals in pmc_per_dispatch(db, cn).items():
                st = stage_of_kernel(name)
                if st:
                    per.setdefault(st, {}).setdefault(cn, []).extend(vals)
        try:
            for name, dur in c.execute("select name, duration from kernels"):
                st = stage_of_kernel(name)
                if st:
                    per.setdefault(st, {}).setdefault("duration_ns", []).append(dur)
        except sqlite3.OperationalError:
            pass
    out = {}
    for st, d in per.items():
        rec = {k: stat.median(v) for k, v in d.items()}
        if "SQ_VALU_MFMA_BUSY_CYCLES" in rec and rec.get("GRBM_GUI_ACTIVE"):
            rec["mfma_busy_frac"] = rec["SQ_VALU_MFMA_BUSY_CYCLES"] / (rec["GRBM_GUI_ACTIVE"] * SIMD_NUM)
        if rec.get("GRBM_GUI_ACTIVE") and rec.get("duration_ns"):
            rec["clock_ghz"] = rec["GRBM_GUI_ACTIVE"] / rec["duration_ns"]
        rec["sources_sha256_16"] = sources_hash(st)
        rec["workload"] = workload
        out[st] = rec
    return out


def traffic_from(fetch_db, write_db, workload):
    """Turns two --pmc runs of this benchmark (FETCH_SIZE, WRITE_SIZE) into per-launch HBM
    bytes of every GEMM stage, scaled by what the counters read for the calibration copy."""
    fetch = pmc_per_dispatch(fetch_db, "FETCH_SIZE")
    write = pmc_per_dispatch(write_db, "WRITE_SIZE")
    def calib(d):
        vals = [v for n, vs in d.items() if "neg" in n.lower() for v in vs]
        if not vals:
            raise SystemExit("calibration copy not found in the counter database")
        return CALIB_BYTES / (sum(vals) / len(vals) * 1024.0)
    f_fetch, f_write = calib(fetch), calib(write)
    recs = {}
    for name, vals in fetch.items():
        st = stage_of_kernel(name)
        if st is None or name not in write:
            continue
        if st in recs and recs[st]["dispatches"] >= len(vals):
            continue   # another instantiation of the stage ran more often
        fb = sum(vals) / len(vals) * 1024.0 * f_fetch
        wb = sum(write[name]) / len(write[name]) * 1024.0 * f_write
        recs[st] = {"stage": st, "kernel": name, "fetch_bytes": fb, "write_bytes": wb,
                    "traffic_bytes": fb + wb, "fetch_scale": f_fetch, "write_scale": f_write,
                    "dispatches": len(vals), "sources_sha256_16": sources_hash(st),
                    "workload": workload}
    return recs


def _rocm_version():
    """ROCm release of the runtime, from the installation's version file (None if absent)."""
    for path in ("/opt/rocm/.info/version", "/opt/rocm/.info/version-dev"):
        try:
            with open(path) as f:
                return f.read().strip()
        except OSError:
            pass
    return None


def WORKLOADS(synth):
    return {"train": synth.TRAIN_BF16, "train_shared": synth.TRAIN_SHARED_BF16,
            "static": synth.STATIC_BF16, "timestep": synth.TIMESTEP_BF16,
            "fine": synth.FINE_BF16, "decode": synth.DECODE_BF16, "tiny": synth.TINY_F32}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def stage_work(name, N, d, E, h, K, esz, EP, save_h, splits, hs=0):
    """(algorithmic flops, algorithmic HBM bytes) of one launch of a stage (hs: hidden width
    of the shared experts)."""
    P = E * K
    s = esz
    parts = (h + 63) // 64 if esz == 4 else (h + 127) // 128  # gate-gradient partials per row
    table = {
        "router": (2 * N * d * E, N * d * s + E * d * s + 2 * N * E * 4),
        "topk": (0, 2 * E * N * 4 + P * 4),
        "gather": (0, P * 4 + 2 * P * d * s),
        "gemm_w13_swiglu": (4 * P * d * h, P * d * s + 2 * E * h * d * s + P * h * s + P * 4
                            + (2 * P * h * s if save_h else 0)),
        "gemm_w2": (2 * P * d * h, P * h * s + E * d * h * s + P * d * s),
        "combine": (0, E * N * 4 + P * d * s + N * d * s),
        "bwd_gather": (0, P * 4 + 2 * P * d * s),
        "gemm_dA_swiglu_bwd": (2 * P * d * h, P * d * s + E * d * h * s + 4 * P * h * s
                               + P * parts * 4 + 2 * P * 4),
        "gemm_dW2": (2 * P * d * h, P * d * s + P * h * s + E * d * h * s),
        "gemm_dXe": (4 * P * d * h, 2 * P * h * s + 2 * E * h * d * s + P * d * s),
        "gemm_dW13": (4 * P * d * h, 2 * P * h * s + P * d * s + 2 * E * h * d * s),
        "router_dz": (0, 3 * N * E * 4 + P * parts * 4 + N * EP * 2),
        "router_dx": (2 * N * EP * d, N * EP * 2 + E * d * s + N * d * s),
        "bwd_combine": (0, E * N * 4 + P * d * s + 2 * N * d * s),
        "router_dwg": (2 * N * EP * d, N * EP * 2 + N * d * s + 2 * splits * E * d * 4),
        "shared_w13_swiglu": (4 * N * d * hs, N * d * s + 2 * hs * d * s + 3 * N * hs * s),
        "shared_w2": (2 * N * d * hs, N * hs * s + hs * d * s + 2 * N * d * s),
        "shared_dA_swiglu_bwd": (2 * N * d * hs, N * d * s + hs * d * s + 4 * N * hs * s),
        "shared_dW2": (2 * N * d * hs, N * d * s + N * hs * s + hs * d * s),
        "shared_dX": (4 * N * d * hs, 2 * N * hs * s + 2 * hs * d * s + 2 * N * d * s),
        "shared_dW13": (4 * N * d * hs, 2 * N * hs * s + N * d * s + 2 * hs * d * s),
    }
    return table[name]


def cpu_baseline(inp, caps, inv_tau, backward, budget_s=10.0):
    """The float64 oracle on a bounded sample: whole routing groups (sequences), one at a
    time in order, until the budget is spent; each group is routed on its own, exactly as
    in the layer (routing never crosses a group)."""
    from oracle import ec_ref as ref
    affinity = len(os.sched_getaffinity(0))
    try:
        from threadpoolctl import threadpool_info
        pools = [i for i in threadpool_info() if i.get("user_api") == "blas"] or threadpool_info()
        blas_threads = max([i.get("num_threads", 1) for i in pools] or [1])
        blas = ", ".join(sorted({str(i.get("internal_api", "?")) for i in pools})) or None
    except Exception:  # pragma: no cover
        blas_threads, blas = affinity, None
    wl = inp.wl
    off = wl.group_offsets
    tokens, dt, groups = 0, 0.0, 0
    for g in range(wl.n_groups):
        lo, hi = int(off[g]), int(off[g + 1])
        X = inp.X[lo:hi]
        t0 = time.perf_counter()
        fw = ref.forward_ref(X, inp.Wg, inp.W1, inp.W3, inp.W2, [0, hi - lo], [int(caps[g])],
                             inv_tau, shared=inp.shared)
        if backward:
            ref.backward_ref(X, inp.Wg, inp.W1, inp.W3, inp.W2, inp.dY[lo:hi], [0, hi - lo],
                             [int(caps[g])], inv_tau, sel_token=fw["sel_token"],
                             shared=inp.shared)
        dt += time.perf_counter() - t0
        tokens += hi - lo
        groups += 1
        if dt >= budget_s:
            break
    return {"value": tokens / dt, "unit": "tokens/s", "cores": int(blas_threads), "kind": "oracle",
            "affinity_cpus": affinity, "blas": blas,
            "sample": f"routing groups 0..{groups - 1} of {wl.n_groups} ({tokens} tokens, all "
                      f"{wl.n_experts} experts), {'fwd+bwd' if backward else 'fwd'}, numpy float64, "
                      f"{dt:.1f} s",
            "seconds": dt}


def run_tc(a):
    """Token choice (the comparison policy, forward) on a workload's inputs, and expert
    choice on the same inputs with the same number of token-expert pairs (c = top_k)."""
    import torch
    import paper_2604_01622_amd as ec
    from paper_2604_01622_amd import binding, synth

    wl = WORKLOADS(synth)[a.workload]
    torch.cuda.set_device(0)
    log(f"[bench] drawing {wl.name}")
    inp = synth.draw(wl, with_dy=False)
    inv_tau = wl.inv_temperatures[0]
    if a.router_skew > 0:
        scale = np.exp(np.random.default_rng(99).normal(0.0, a.router_skew, (wl.n_experts, 1)))
        w = inp.Wg.view(np.uint16).astype(np.uint32) << 16 if wl.dtype == "bf16" else None
        wf = w.view(np.float32) if w is not None else inp.Wg
        inp.Wg[:] = (synth.f32_to_bf16_bits((wf * scale).astype(np.float32)) if wl.dtype == "bf16"
                     else (wf * scale).astype(np.float32))

    def dev(x):
        if x.dtype == np.uint16:
            return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(x).cuda()

    X, Wg, W1, W3, W2 = (dev(x) for x in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2))
    shared = None if inp.shared is None else tuple(dev(w) for w in inp.shared)
    N, d, E, h = wl.n_tokens, wl.d_model, wl.n_experts, wl.d_ff
    L = np.asarray(wl.group_lengths)
    caps = ec.tc_capacity(L, E, a.top_k, a.cf)
    tc = ec.TcLayer(X, Wg, W1, W3, W2, wl.group_offsets, caps, a.top_k, inv_tau, shared)
    ec_caps = ec.capacity(L, E, c=float(a.top_k))
    ecl = ec.Layer(X, Wg, W1, W3, W2, wl.group_offsets, ec_caps, inv_tau, training=False,
                   shared=shared)

    def timed(fn, events=None):
        for _ in range(a.warmup):
            fn()
        torch.cuda.synchronize()
        # uninstrumented steps for the time, then instrumented ones for the stages
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(a.steps):
            fn()
        s1.record()
        torch.cuda.synchronize()
        ms = s0.elapsed_time(s1) / a.steps
        evs = [binding.StageEvents(len(binding.FORWARD_STAGES)) for _ in range(a.steps)]
        for i in range(a.steps):
            evs[i].arm()
            fn()
        binding.StageEvents.disarm()
        torch.cuda.synchronize()
        st = {n: float(np.mean(col)) for n, col in
              zip(binding.FORWARD_STAGES, zip(*[e.durations_ms() for e in evs]))}
        return ms, st

    log(f"[bench] token choice top-{a.top_k}, cf {a.cf}")
    ms_tc, st_tc = timed(tc.forward)
    rows = tc.rows.cpu().numpy().astype(np.int64)
    loads = np.diff(rows)
    R = int(rows[-1])
    log("[bench] expert choice, same pairs")
    ms_ec, st_ec = timed(ecl.forward)
    Kec = int(np.sum(ec_caps))
    shards = loads.reshape(8, -1).sum(axis=1) if E % 8 == 0 else None
    esz = 2 if wl.dtype == "bf16" else 4

    def gemm_stats(st, pairs):
        out = {}
        for n, fl in (("gemm_w13_swiglu", 4 * pairs * d * h), ("gemm_w2", 2 * pairs * d * h)):
            out[n] = {"ms": round(st[n], 4), "tflops": round(fl / (st[n] * 1e-3) / 1e12, 1)}
        for n in ("router", "topk", "gather", "combine"):
            out[n] = {"ms": round(st[n], 4)}
        return out

    out = {"metric": METRIC, "value": round(N / (ms_tc * 1e-3), 1), "unit": "tokens/s",
           "n_gpus": 1, "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_tc, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
           "data": "synthetic (seeded normal inputs and random-init weights)",
           "config": {"workload": f"{wl.name}_tc_top{a.top_k}_cf{a.cf:g}_skew{a.router_skew:g}",
                      "pass": "fwd",
                      "routing": "token choice", "top_k": a.top_k, "capacity_factor": a.cf,
                      "tokens": N, "d_model": d, "experts": E, "d_ff": h,
                      "cap_per_group": [int(x) for x in caps]},
           "stages": gemm_stats(st_tc, R),
           "token_choice": {"pairs_kept": R, "pairs_chosen": a.top_k * N,
                            "dropped_fraction": round(1 - R / (a.top_k * N), 5),
                            "load_max_over_mean": round(float(loads.max() / loads.mean()), 4),
                            "load_min": int(loads.min()), "load_max": int(loads.max()),
                            "ep8_shard_max_over_mean": (None if shards is None else
                                                        round(float(shards.max() / shards.mean()), 4))},
           "expert_choice_same_pairs": {"tokens_per_s": round(N / (ms_ec * 1e-3), 1),
                                        "ms": round(ms_ec, 4), "pairs": E * Kec,
                                        "load_max_over_mean": 1.0,
                                        "stages": gemm_stats(st_ec, E * Kec)}}
    print(json.dumps(out), flush=True)


def vendor_gemm(E, M, d, h, warmup, steps, backward):
    """torch.matmul (hipBLASLt) on the expert products' batched shapes, every
    operand contiguous and row-major, seeded normal bf16 values: a reference for
    the library's grouped GEMMs (same FLOPs, no gather, no fused epilogue)."""
    import torch
    shapes = {"gemm_w13_swiglu": (M, d, 2 * h), "gemm_w2": (M, h, d)}
    if backward:
        shapes.update({"gemm_dA_swiglu_bwd": (M, d, h), "gemm_dXe": (M, 2 * h, d),
                       "gemm_dW2": (d, M, h), "gemm_dW13": (2 * h, M, d)})
    gen = torch.Generator(device="cuda").manual_seed(0)
    res = {}
    for name, (m, k, n) in shapes.items():
        A = torch.randn(E, m, k, device="cuda", generator=gen).to(torch.bfloat16)
        B = (torch.randn(E, k, n, device="cuda", generator=gen) * 0.02).to(torch.bfloat16)
        C = torch.empty(E, m, n, device="cuda", dtype=torch.bfloat16)
        for _ in range(warmup):
            torch.matmul(A, B, out=C)
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(steps):
            torch.matmul(A, B, out=C)
        ev1.record()
        torch.cuda.synchronize()
        t = ev0.elapsed_time(ev1) / steps
        fl = 2.0 * E * m * k * n
        res[name] = {"ms": round(t, 4), "tflops": round(fl / (t * 1e-3) / 1e12, 1),
                     "shape": f"{E} x ({m} x {k}) @ ({k} x {n})"}
        del A, B, C
    torch.cuda.empty_cache()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="train",
                    choices=["train", "train_shared", "static", "timestep", "fine", "decode",
                             "tiny"])
    ap.add_argument("--routing", default="ec", choices=["ec", "tc"],
                    help="tc: the token-choice comparison policy (forward), beside expert choice "
                         "with the same number of token-expert pairs")
    ap.add_argument("--top-k", type=int, default=8, help="token choice: experts per token")
    ap.add_argument("--cf", type=float, default=1.0,
                    help="token choice: capacity factor (<= 0: dropless)")
    ap.add_argument("--router-skew", type=float, default=0.0,
                    help="token choice: scale router rows by exp(N(0, s)) (uneven expert loads)")
    ap.add_argument("--mask-ratio", type=float, default=None,
                    help="every sequence's mask ratio t (workloads with c(t) = 12 - 8t capacities): "
                         "the capacity, and so the expert work, of one point of the schedule")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-forward-only", action="store_true")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip timing the step as a replayed HIP graph")
    ap.add_argument("--no-cold", action="store_true",
                    help="skip the cold-cache steps (a 512 MiB buffer overwritten before each)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="run one plain 1 GiB elementwise copy first (scales --pmc byte counters)")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="also time torch.matmul (hipBLASLt) on the same batched expert-product "
                         "shapes, as a reference for the grouped GEMM figures")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_DB", "WRITE_DB"),
                    help="write profiles/traffic_<stage>.json from two --pmc runs and exit")
    ap.add_argument("--counters-from", nargs="+", metavar="PMC_DB",
                    help="write profiles/counters_<workload>.json (per-stage medians, MFMA "
                         "utilisation, clock) from --pmc --kernel-trace runs and exit")
    a = ap.parse_args()
    if a.counters_from:
        recs = counters_from(a.counters_from, a.workload)
        with open(os.path.join(ROOT, "profiles", f"counters_{a.workload}.json"), "w") as f:
            json.dump(recs, f, indent=1, sort_keys=True)
        for st, r in sorted(recs.items()):
            mf = r.get("mfma_busy_frac")
            print(f"{st:22s} mfma_busy {'-' if mf is None else f'{100 * mf:5.1f}%'} clock "
                  f"{r.get('clock_ghz', float('nan')):.2f} GHz  duration "
                  f"{r.get('duration_ns', float('nan')) / 1e3:8.1f} us")
        return
    if a.routing == "tc" and not a.traffic_from:
        if a.gpus != 1:
            print(f"bench.py runs on exactly one GPU; --gpus {a.gpus} is not supported",
                  file=sys.stderr)
            sys.exit(2)
        return run_tc(a)
    if a.traffic_from:
        recs = traffic_from(a.traffic_from[0], a.traffic_from[1], a.workload)
        for st, r in recs.items():
            with open(os.path.join(ROOT, "profiles", f"traffic_{st}.json"), "w") as f:
                json.dump(r, f, indent=1)
            print(f"{st}: fetch {r['fetch_bytes'] / 1e9:.3f} GB write {r['write_bytes'] / 1e9:.3f} GB "
                  f"per launch")
        return
    if a.gpus != 1:
        print(f"bench.py runs on exactly one GPU; --gpus {a.gpus} is not supported (the layer's "
              "multi-GPU sharding is described, not implemented)", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2604_01622_amd as ec
    from paper_2604_01622_amd import binding, synth

    wl = WORKLOADS(synth)[a.workload]
    if a.mask_ratio is not None and not (wl.time_dependent and 0.0 <= a.mask_ratio <= 1.0):
        print(f"--mask-ratio needs a workload with c(t) capacities and t in [0, 1] "
              f"(got {a.workload}, {a.mask_ratio})", file=sys.stderr)
        sys.exit(2)
    backward = a.workload in ("train", "train_shared")
    inv_tau = wl.inv_temperatures[0]
    torch.cuda.set_device(0)
    log(f"[bench] drawing {wl.name}")
    inp = synth.draw(wl, with_dy=backward)
    L = np.asarray(wl.group_lengths)
    if a.mask_ratio is not None:
        inp.t = np.full_like(inp.t, a.mask_ratio)
    if wl.time_dependent:
        caps = ec.capacity(L, wl.n_experts, t=inp.t, c_min=wl.c_min, c_max=wl.c_max)
    else:
        caps = ec.capacity(L, wl.n_experts, c=wl.capacity_factor)

    def dev(x):
        if x.dtype == np.uint16:
            return torch.from_numpy(x.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(x).cuda()

    X, Wg, W1, W3, W2 = (dev(x) for x in (inp.X, inp.Wg, inp.W1, inp.W3, inp.W2))
    dY = dev(inp.dY) if backward else None
    shared = None if inp.shared is None else tuple(dev(w) for w in inp.shared)
    hs = wl.d_shared
    layer = ec.Layer(X, Wg, W1, W3, W2, wl.group_offsets, caps, inv_tau, training=backward,
                     shared=shared)
    N, d, E, h, K = wl.n_tokens, wl.d_model, wl.n_experts, wl.d_ff, layer.P.K
    esz = 2 if wl.dtype == "bf16" else 4
    EP = (E + 63) // 64 * 64
    splits = max(1, min((512 + (d + 127) // 128 - 1) // ((d + 127) // 128), (N + 255) // 256))

    def step():
        layer.forward()
        if backward:
            layer.backward(dY)

    if a.calibration_copy:
        src = torch.ones(CALIB_BYTES // 2, dtype=torch.bfloat16, device="cuda")
        dst = torch.empty_like(src)
        torch.neg(src, out=dst)   # reads and writes CALIB_BYTES
        torch.cuda.synchronize()
        del src, dst

    log(f"[bench] warmup {a.warmup}")
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # The timed steps run uninstrumented: each stage event the library records is
    # a command of its own on the stream (several microseconds apiece), so the
    # per-stage durations come from a second pass of the same number of steps.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    log(f"[bench] timing {a.steps} steps")
    torch.cuda.synchronize()
    start.record()
    for _ in range(a.steps):
        step()
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / a.steps
    value = N / (ms * 1e-3)

    fwd_ev = [binding.StageEvents(len(binding.FORWARD_STAGES)) for _ in range(a.steps)]
    bwd_ev = [binding.StageEvents(len(binding.BACKWARD_STAGES)) for _ in range(a.steps)]
    log(f"[bench] {a.steps} steps with stage events")
    s_start, s_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s_start.record()
    for i in range(a.steps):
        fwd_ev[i].arm()
        layer.forward()
        if backward:
            bwd_ev[i].arm()
            layer.backward(dY)
    binding.StageEvents.disarm()
    s_end.record()
    torch.cuda.synchronize()
    ms_instrumented = s_start.elapsed_time(s_end) / a.steps

    stage_ms, stage_med = {}, {}
    for n, col in zip(binding.FORWARD_STAGES, zip(*[e.durations_ms() for e in fwd_ev])):
        stage_ms[n], stage_med[n] = float(np.mean(col)), float(np.median(col))
    if backward:
        for n, col in zip(binding.BACKWARD_STAGES, zip(*[e.durations_ms() for e in bwd_ev])):
            stage_ms[n], stage_med[n] = float(np.mean(col)), float(np.median(col))
    if not hs:   # the shared-expert stages are empty
        stage_ms = {n: t for n, t in stage_ms.items() if not n.startswith("shared_")}
    stages = {}
    for n, t in stage_ms.items():
        fl, by = stage_work(n, N, d, E, h, K, esz, EP, backward, splits, hs)
        st = {"ms": round(t, 4), "ms_median": round(stage_med[n], 4)}
        if t < 0.010:   # an empty stage (bf16: the gather happens inside the W1/W3 product)
            stages[n] = st
            continue
        if n in GEMM_STAGES:
            t = max(t, 1e-6)
            st["tflops"] = round(fl / (t * 1e-3) / 1e12, 1)
            st["mfma_frac"] = round(fl / (t * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)
        else:
            t = max(t, 1e-6)
            st["gbs"] = round(by / (t * 1e-3) / 1e9, 1)
            st["hbm_frac"] = round(by / (t * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
        stages[n] = st
    # routing as one stage: the router GEMM + softmax and the column top-k together
    r_ms = stage_ms["router"] + stage_ms["topk"]
    r_by = sum(stage_work(n, N, d, E, h, K, esz, EP, backward, splits, hs)[1]
               for n in ("router", "topk"))
    route = {"ms": round(r_ms, 4), "bytes": r_by, "gbs": round(r_by / (r_ms * 1e-3) / 1e9, 1),
             "hbm_frac": round(r_by / (r_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
    dom = max(stage_ms, key=stage_ms.get)
    fl, by = stage_work(dom, N, d, E, h, K, esz, EP, backward, splits, hs)
    t_dom = stage_ms[dom] * 1e-3
    traffic = None
    tf = os.path.join(ROOT, "profiles", f"traffic_{dom}.json")
    if os.path.exists(tf):
        with open(tf) as f:
            rec = json.load(f)
        if rec.get("sources_sha256_16") == sources_hash(dom) and rec.get("workload") == a.workload:
            traffic = round(rec["traffic_bytes"])
    if dom in GEMM_STAGES:
        peak = PEAK_BF16_TFLOPS if esz == 2 else PEAK_F32_TFLOPS
        roof = {"kernel": dom, "bound": "mfma", "achieved": round(fl / t_dom / 1e12, 1),
                "peak": peak, "unit": "TFLOP/s", "frac": round(fl / t_dom / 1e12 / peak, 4),
                "traffic": traffic, "work_per_launch": fl, "avg_launch_ms": round(stage_ms[dom], 4)}
    else:
        roof = {"kernel": dom, "bound": "hbm", "achieved": round(by / t_dom / 1e9, 1),
                "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(by / t_dom / 1e9 / PEAK_HBM_GBS, 4),
                "traffic": traffic, "work_per_launch": by, "avg_launch_ms": round(stage_ms[dom], 4)}
    gemm_fl = sum(stage_work(n, N, d, E, h, K, esz, EP, backward, splits, hs)[0]
                  for n in stage_ms if n.startswith("gemm_") or n.startswith("shared_"))
    gemm_ms = sum(stage_ms[n] for n in stage_ms if n.startswith("gemm_") or n.startswith("shared_"))

    out = {"metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1,
           "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 4),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": wl.dtype, "data": "synthetic (seeded normal inputs and random-init weights)",
           "config": {"workload": wl.name, "pass": "fwd+bwd" if backward else "fwd",
                      "tokens": N, "groups": wl.n_groups, "d_model": d, "experts": E,
                      "d_ff": h, "shared_hidden": hs, "k_per_group": [int(x) for x in caps],
                      "K_tot": K},
           "stages": stages, "route": route, "ms_per_step_with_stage_events": round(ms_instrumented, 4),
           "roofline": roof,
           "grouped_gemm": {"tflops": round(gemm_fl / (gemm_ms * 1e-3) / 1e12, 1),
                            "mfma_frac": round(gemm_fl / (gemm_ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4)}}

    if a.mask_ratio is not None:
        out["config"]["mask_ratio"] = a.mask_ratio
    # token drop statistic (Appendix D) of this batch, from the routing the step made
    if backward:
        slot = binding.saved_views(layer.saved, layer.P)["slot"]
    else:
        slot = ec.route(X, Wg, wl.group_offsets, caps, inv_tau, d_ff=h)[3]
    _, dropped = ec.token_coverage(slot, wl.group_offsets, caps, d_model=d, d_ff=h)
    n_drop = int(dropped.sum().item())
    out["token_drop"] = {"dropped_tokens": n_drop, "fraction": round(n_drop / N, 5),
                         "per_group": [int(v) for v in dropped.cpu().tolist()]}

    if backward and not a.no_forward_only:
        # forward alone, inference mode (no saved activations), same inputs
        inf = ec.Layer(X, Wg, W1, W3, W2, wl.group_offsets, caps, inv_tau, training=False,
                       shared=shared)
        for _ in range(a.warmup):
            inf.forward()
        torch.cuda.synchronize()
        start.record()
        for _ in range(a.steps):
            inf.forward()
        end.record()
        torch.cuda.synchronize()
        fms = start.elapsed_time(end) / a.steps
        out["forward_only"] = {"tokens_per_s": round(N / (fms * 1e-3), 1), "ms": round(fms, 4)}
        del inf

    if not a.no_graph:
        # the same step captured once in a HIP graph and replayed (launch overhead gone)
        try:
            side = torch.cuda.Stream()
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(side):
                step()
            torch.cuda.current_stream().wait_stream(side)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step()
            for _ in range(a.warmup):
                g.replay()
            torch.cuda.synchronize()
            start.record()
            for _ in range(a.steps):
                g.replay()
            end.record()
            torch.cuda.synchronize()
            gms = start.elapsed_time(end) / a.steps
            out["graph_replay"] = {"ms": round(gms, 4), "tokens_per_s": round(N / (gms * 1e-3), 1)}
            del g
        except Exception as exc:   # report, do not fail the benchmark line
            out["graph_replay"] = {"error": str(exc)[:200]}

    if not a.no_cold:
        # cold caches: overwrite a buffer twice the size of the MALL before every
        # step (outside the timed events), then the step alone; median over steps
        log("[bench] cold-cache steps")
        flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda")
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(a.steps)]
        for i in range(a.steps):
            flush.fill_(float(i))
            evs[i][0].record()
            step()
            evs[i][1].record()
        torch.cuda.synchronize()
        cms = float(np.median([s0.elapsed_time(s1) for s0, s1 in evs]))
        out["cold_cache"] = {"ms_median": round(cms, 4), "tokens_per_s": round(N / (cms * 1e-3), 1),
                             "flush_bytes": FLUSH_BYTES}
        del flush

    if a.vendor_gemm and esz == 2:
        out["vendor_gemm"] = vendor_gemm(E, K, d, h, a.warmup, a.steps, backward)

    props = torch.cuda.get_device_properties(0)
    out["env"] = {"device": props.name, "gfx": getattr(props, "gcnArchName", None),
                  "hip": torch.version.hip, "torch": torch.__version__,
                  "rocm": _rocm_version()}

    if not a.no_cpu_baseline:
        log("[bench] cpu baseline (oracle on a sample)")
        out["cpu_baseline"] = cpu_baseline(inp, caps, inv_tau, backward)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
