#!/usr/bin/env python3
"""Benchmark of the PLD+ drafting step (find -> rank -> emit -> verify) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config C] [--verify greedy|sample]
                    [--temperature T] [--mode auto|fused|split] [--split S] [--warm]
                    [--no-cpu-baseline] [--copy-probe]
    python bench.py --loop TASK        # the generation loop, once per ranking
    python bench.py --probe            # bandwidth ceilings of the access patterns

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM.  The default workload is config 2 (batch 8, context
4096, n-grams 3..1 longest first, hidden 4096 bf16, K = 10, fp32 logits over
32000 ids); --config picks another (1-5 scale the workload up, 6 and 7 are the
paper's attention-MAX and thresholded hidden-state settings at its input
sizes); --verify sample verifies by sampling at --temperature (default 1)
instead of the argmax.  To keep the caches honest the
inputs exist in several copies at distinct addresses and consecutive steps
rotate through them, so every step reads from HBM rather than from the 256 MB
last-level cache.  W untimed steps run first, then exactly K steps are timed
between two device synchronisations; HIP events on the launch stream time the
dominant kernel inside that region, on every eighth step (--event-every).  One JSON line goes to stdout.

The CPU oracle (test infrastructure) is timed on the host on the same inputs
as a reported baseline, unless --no-cpu-baseline.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "draft+verify step latency (us) per batch; ranking-kernel HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
MALL_BYTES = 256 << 20         # last-level (Infinity) cache
SEG = 128                      # HBM fetch granule of gathered data (a 128-byte line)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--config", type=int, default=2, choices=[1, 2, 3, 4, 5, 6, 7])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="CPU work the oracle baseline is given (whole steps, at least one)")
    p.add_argument("--warm", action="store_true",
                   help="one copy of the inputs, so steps re-read what the last-level cache holds "
                        "(labelled warm in the output); the default rotates cold copies")
    p.add_argument("--copy-probe", action="store_true",
                   help="after the timed region, copy 1 GiB three times (counter calibration)")
    p.add_argument("--event-every", type=int, default=8,
                   help="bracket the dominant call with timing events on every N-th timed step")
    p.add_argument("--split", type=int, default=0,
                   help="blocks per sequence of the one-call drafting (default: from the "
                        "first step's candidate counts)")
    p.add_argument("--mode", choices=["auto", "fused", "split"], default="auto",
                   help="drafting: one-launch call (fused), separate calls (split), or auto")
    p.add_argument("--verify", choices=["greedy", "sample"], default="greedy",
                   help="verification: argmax (greedy) or sampling at --temperature")
    p.add_argument("--temperature", type=float, default=1.0)
    p.add_argument("--probe", action="store_true",
                   help="instead of the step benchmark, run bench_probe (the read-bandwidth "
                        "ceilings of the kernels' access patterns, from HBM) and print its lines")
    p.add_argument("--loop", default=None,
                   help="instead of the step benchmark, run the generation loop on a decoding "
                        "task (synth.DECODE_TASKS) with each ranking and report the loop step "
                        "latency and the average acceptance length")
    return p.parse_args()


def algorithmic_bytes(cfg, lens, cand_count, draft_len, cand_pos, elt_logits, fused,
                      sample=False):
    """What each kernel must move per step (never the dense work it avoids)."""
    import numpy as np
    B, K = cfg.B, cfg.K
    C = cand_count.astype(np.int64)
    out = {}
    out["find"] = int(lens.astype(np.int64).sum() * 4 + C.sum() * 4)
    if cfg.rank in ("attn", "both"):
        # distinct 128-byte lines of each attention row that hold a key j-1
        segs = 0
        for b in range(B):
            keys = cand_pos[b, :C[b]].astype(np.int64) - 1
            segs += len(np.unique((keys * 4) // SEG))
        out["score_attn"] = int(segs * cfg.R * SEG + C.sum() * 4)
        out["select_attn"] = B * 8 * 2 + B * 8
    if cfg.rank in ("hidden", "both"):
        out["score_hidden"] = int(((C + (C > 0)) * cfg.d * 2).sum() + C.sum() * 4)
        out["select"] = B * 8 * 2 + B * 8
    out["emit"] = int(B * K * 4 * 2)
    rows = draft_len.astype(np.int64) + 1
    if sample:
        # statistics: the logits rows i <= L once, one (max, mass) pair per segment
        # written; finish: the pairs and the draws read, the tokens written (the
        # re-read of one segment per row is the method's choice, not counted)
        nseg = max(1, -(-(cfg.V * elt_logits // 16) // 512))
        out["verify_sample_stats"] = int((rows * cfg.V * elt_logits).sum() + rows.sum() * nseg * 8)
        out["verify_sample_finish"] = int(rows.sum() * (nseg * 8 + 4) + B * K * 4 + B * (K + 1) * 4)
    else:
        out["verify_argmax"] = int((rows * cfg.V * elt_logits).sum())
        out["verify_accept"] = int((rows * 8 * 2).sum() + B * K * 4 + B * (K + 1) * 4)
    if fused:   # one launch does find, rank, select and emit
        out["draft"] = sum(out.pop(k) for k in ("find", "score_hidden", "score_attn", "select",
                                                "select_attn", "emit") if k in out)
    return out


# kernels behind each timed call (names as rocprofv3 reports them)
KERNELS = {"draft": "pld::draft_", "find": "pld::find_", "score_hidden": "pld::rank_hidden_kernel",
           "score_attn": "pld::rank_attn_kernel", "select": "pld::rank_finish_kernel",
           "select_attn": "pld::rank_finish_kernel", "emit": "pld::emit_kernel",
           "verify_argmax": "pld::verify_argmax_kernel", "verify_accept": "pld::verify_accept_kernel",
           "verify_sample_stats": "pld::sample_stats_kernel",
           "verify_sample_finish": "pld::sample_finish_kernel"}


class TimingEvents:
    """HIP events for timing only, created with hipEventDisableSystemFence: a
    default event's system-scope release writes back and invalidates the
    caches at every record, which both slows the following kernel and adds
    microseconds to the bracketed interval."""
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n):
        import ctypes
        self.ct = ctypes
        lib = ctypes.CDLL("libamdhip64.so")
        lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
        lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
        lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                            ctypes.c_void_p]
        lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
        for f in ("hipEventCreateWithFlags", "hipEventRecord", "hipEventElapsedTime",
                  "hipEventDestroy"):
            getattr(lib, f).restype = ctypes.c_int
        self.lib = lib
        self.ev = []
        for _ in range(2 * n):
            e = ctypes.c_void_p()
            rc = lib.hipEventCreateWithFlags(ctypes.byref(e), self.DISABLE_SYSTEM_FENCE)
            if rc != 0:
                raise RuntimeError(f"hipEventCreateWithFlags failed ({rc})")
            self.ev.append(e)

    def record(self, i, stream):
        rc = self.lib.hipEventRecord(self.ev[i], self.ct.c_void_p(stream.cuda_stream))
        if rc != 0:
            raise RuntimeError(f"hipEventRecord failed ({rc})")

    def elapsed_ms(self, i, j):
        ms = self.ct.c_float()
        rc = self.lib.hipEventElapsedTime(self.ct.byref(ms), self.ev[i], self.ev[j])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return ms.value

    def close(self):
        for e in self.ev:
            self.lib.hipEventDestroy(e)
        self.ev = []


def measured_traffic(workload, call):
    """HBM bytes per launch of the call's kernel from the committed counter runs
    (profiles/traffic.json), or None when the kernel sources changed since."""
    import glob
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    h = hashlib.sha256()
    for fn in sorted(glob.glob(os.path.join(ROOT, "paper_2412_01447_amd", "csrc", "*"))):
        h.update(os.path.basename(fn).encode())
        with open(fn, "rb") as f:
            h.update(f.read())
    if h.hexdigest() != table.get("sources_sha256"):
        return None
    rows = table.get("workloads", {}).get(workload, {})
    hits = [v for k, v in rows.items() if k.startswith(KERNELS.get(call, "?"))]
    return sum(hits) if hits else None


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU (--gpus 1): the step shards by sequence with no "
              "exchange between GPUs, so more GPUs only scale the batch.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import synth
    from paper_2412_01447_amd.step import DraftStep

    if args.probe:
        import subprocess
        exe = os.path.join(ROOT, "bench_probe")
        if not os.path.exists(exe):
            sys.exit(f"{exe} is missing: build it with `python -c 'import __graft_entry__ as g; "
                     "g.build()'`")
        sys.exit(subprocess.run([exe]).returncode)
    if args.loop:
        return run_loop(args)
    cfg = synth.CONFIGS[args.config]
    dev = torch.device("cuda:0")
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    log(f"[bench] config {args.config}: {cfg.name}")
    t0 = time.time()
    w = synth.make_workload(cfg, dev, structured=True)
    toks, lens = w["tokens"], w["lens"]
    draft_i, dlen_i = synth.intended_drafts(w["metas"], cfg.K)
    z = synth.logits_for(w, draft_i, dlen_i)
    bf16 = cfg.logits == "bf16"
    elt = 2 if bf16 else 4
    log(f"[bench] inputs generated in {time.time() - t0:.1f}s")

    def dev_logits(a):
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if bf16 else a).to(dev)
        return t.view(torch.bfloat16) if bf16 else t

    base = dict(tokens=torch.from_numpy(toks).to(dev), lens=torch.from_numpy(lens).to(dev),
                logits=dev_logits(z), hidden=w["hidden"],
                attn=torch.from_numpy(w["attn"]).to(dev) if w["attn"] is not None else None)
    step = DraftStep(cfg.B, cfg.T, cfg.K, device=dev, mode=args.mode)
    fused = step.uses_fused(base["hidden"], base["attn"])
    sample = args.verify == "sample"
    if sample:
        step.set_sampling(args.temperature, cfg.V, bf16,
                          uniforms=torch.from_numpy(synth.make_uniforms(cfg.B, cfg.K, cfg.seed)).to(dev))

    from paper_2412_01447_amd import PLD_AGG_MAX, PLD_AGG_SUM
    rank_args = dict(ngram=cfg.ngram, agg=PLD_AGG_MAX if cfg.agg == "max" else PLD_AGG_SUM,
                     threshold=cfg.theta)

    def run(s):
        step.run(s["tokens"], s["lens"], s["logits"], hidden=s["hidden"], attn=s["attn"],
                 **rank_args)

    # one step to learn the data-dependent byte counts (and, for the one-call
    # drafting, how many blocks should share a sequence)
    run(base)
    torch.cuda.synchronize()
    nbytes = algorithmic_bytes(cfg, lens, step.cand_count.cpu().numpy(),
                               step.draft_len.cpu().numpy(), step.cand_pos.cpu().numpy(), elt,
                               fused, sample=sample)
    step_bytes = sum(nbytes.values())
    dominant = max(nbytes, key=nbytes.get)
    # input copies at distinct addresses: the steps of one rotation touch at
    # least twice the last-level cache
    copies = 1 if args.warm else int(min(64, max(2, math.ceil(2 * MALL_BYTES / max(step_bytes, 1)))))
    sets = [base]
    for _ in range(copies - 1):
        sets.append({k: (v.clone() if v is not None else None) for k, v in base.items()})
    torch.cuda.synchronize()
    log(f"[bench] step bytes {step_bytes / 1e6:.2f} MB {json.dumps(nbytes)}; "
        f"dominant {dominant}; {copies} input copies")
    # every step as prepared calls (arguments marshalled once, one kernel each)
    stream = torch.cuda.current_stream()

    def make_plans():
        return [step.plan(s_["tokens"], s_["lens"], s_["logits"], hidden=s_["hidden"],
                          attn=s_["attn"], stream=stream, **rank_args) for s_ in sets]

    if fused:
        # blocks per sequence for the one-call drafting, from the first step's
        # candidate counts (or as given)
        if args.split:
            step.set_split(args.split)
        else:
            step.tune_split(step.cand_count.cpu().numpy(), hidden=base["hidden"] is not None)
        log(f"[bench] drafting with {step.draft_split} block(s) per sequence")
    plans = make_plans()
    names = [n for n, _ in plans[0]]
    assert set(names) == set(nbytes), (names, list(nbytes))
    # the dominant call is bracketed by events on every `event_every`-th timed
    # step: an event pair adds its own dispatches to the step, so sampling keeps
    # the step time close to the unbracketed one
    timed = [k for k in range(args.steps) if k % args.event_every == 0]
    ev = TimingEvents(len(timed))

    for k in range(args.warmup):
        for _, call in plans[k % copies]:
            call()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(args.steps):
        e = k // args.event_every if k % args.event_every == 0 else -1
        for name, call in plans[k % copies]:
            if name == dominant and e >= 0:
                ev.record(2 * e, stream)
                call()
                ev.record(2 * e + 1, stream)
            else:
                call()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed * 1e3 / args.steps
    dom_each = [ev.elapsed_ms(2 * e, 2 * e + 1) for e in range(len(timed))]
    dom_ms = sum(dom_each) / len(dom_each)
    ev.close()
    import numpy as np
    pct = {f"p{q}_us": round(float(np.percentile(dom_each, q)) * 1e3, 2) for q in (10, 50, 90)}

    roofline = None
    if dom_ms:
        achieved = nbytes[dominant] / (dom_ms * 1e-3) / 1e9
        roofline = {"bound": "hbm", "kernel": dominant, "achieved": round(achieved, 1),
                    "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "traffic": measured_traffic(cfg.name, dominant),
                    "bytes_per_launch": nbytes[dominant],
                    "avg_us": round(dom_ms * 1e3, 2), **pct, "launches_timed": len(timed)}
        log(f"[bench] {dominant}: {dom_ms * 1e3:.2f} us avg, {achieved:.1f} GB/s")

    if args.copy_probe:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy probe: 3 x 1 GiB device copies done")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(cfg, w, z, bf16, args.cpu_seconds, log,
                           (args.temperature, synth.make_uniforms(cfg.B, cfg.K, cfg.seed))
                           if sample else None)

    line = {
        "metric": METRIC, "value": round(ms_per_step * 1e3, 2), "unit": "us", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "batch": cfg.B, "context": cfg.T, "vocab": cfg.V,
                   "ngram": list(cfg.ngram), "ranking": cfg.rank, "hidden_dim": cfg.d,
                   "attn_rows": cfg.R, "attn_aggregation": cfg.agg, "threshold": cfg.theta,
                   "K": cfg.K, "logits": cfg.logits,
                   "inputs": "hidden bf16, attention f32, tokens int32",
                   "drafting": (f"one call, {step.draft_split} block(s) per sequence" if fused
                                else "separate calls"),
                   "verification": (f"sampling at temperature {args.temperature}" if sample
                                    else "greedy"),
                   "input_copies": copies,
                   "cache": "warm: one copy of the inputs" if args.warm else
                            "cold: copies rotated past the last-level cache",
                   **({"attn_bytes_dense": int(cfg.B) * cfg.R * cfg.T * 4}
                      if cfg.rank in ("attn", "both") else {}),
                   "step_bytes": step_bytes},
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)


LOOP_METRIC = "draft+verify+commit loop step latency (us); average acceptance length"


def run_loop(args):
    """The generation loop (draft -> verify -> commit) on a synthetic decoding task,
    once per ranking: PLD+ with hidden states (Eq. 2), prompt lookup's first match of
    the longest n-gram up to 3, and prompt lookup's longest matching prefix up to 64.
    The stand-in model's logits depend only on the lengths, so they are produced
    before each step and the events bracket the library's calls alone."""
    import numpy as np
    import torch

    import synth
    from paper_2412_01447_amd.step import DraftStep
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    task = synth.DECODE_TASKS[args.loop]
    dev = torch.device("cuda:0")
    w = synth.make_decode_task(task, device=dev)
    target, start = w["target"], w["start"]
    B, T = target.shape
    rankings = [("pld_plus_hidden", dict(hidden=w["hidden"], ngram=(1, 1))),
                ("pld_first_ngram3", dict(prefix_match=3, ngram=(1, 3))),
                ("pld_longest_prefix64", dict(prefix_match=64, ngram=(1, 1)))]
    results = {}
    for name, kw in rankings:
        for rep in range(2):        # the first pass warms up
            toks = np.where(np.arange(T)[None, :] < start[:, None], target, -1).astype(np.int32)
            td = torch.from_numpy(toks).to(dev)
            ld = torch.from_numpy(start.copy()).to(dev)
            limit = torch.full((B,), T, dtype=torch.int32, device=dev)
            stats = torch.zeros((B, 2), dtype=torch.int64, device=dev)
            step = DraftStep(B, T, task.K, device=dev)
            model = synth.TargetModel(target, task.K, task.V, task.seed, device=dev)
            stream = torch.cuda.current_stream()
            z = model.logits(ld)       # the one logits buffer, patched in place per step
            if "hidden" in kw:         # blocks per sequence from the prompt's candidate counts
                step.make_draft(td, ld, **kw)
                if args.split:
                    step.set_split(args.split)
                else:
                    step.tune_split(step.cand_count.cpu().numpy(), hidden=True)
            ops = [c for _, c in step.plan(td, ld, z, commit=(limit, stats), stream=stream, **kw)]
            ev = TimingEvents(4 * (T - int(start.min())) + 8)
            n = 0
            while True:
                if n % 4 == 0 and bool((ld >= limit).all()):
                    break
                model.logits(ld)
                ev.record(2 * n, stream)
                for call in ops:
                    call()
                ev.record(2 * n + 1, stream)
                n += 1
            torch.cuda.synchronize()
            us = [ev.elapsed_ms(2 * i, 2 * i + 1) * 1e3 for i in range(n)]
            ev.close()
            s = stats.cpu().numpy()
            assert np.array_equal(td.cpu().numpy(), target), "the loop must end on the targets"
        steps = int(s[:, 1].sum())
        results[name] = {"avg_accept_len": round(float(s[:, 0].sum()) / max(steps, 1), 4),
                         "loop_steps": n, "drafting": [c for c, _ in step.plan(
                             td, ld, z, stream=stream, **kw)][:-2],
                         "blocks_per_seq": step.draft_split,
                         "us_per_step": round(float(np.mean(us)), 2),
                         "us_per_step_p50": round(float(np.median(us)), 2),
                         "tokens_generated": int(s[:, 0].sum())}
        log(f"[loop] {name}: {n} steps, {results[name]['avg_accept_len']} tokens per step, "
            f"{results[name]['us_per_step']} us per step")
    first = results["pld_plus_hidden"]
    line = {"metric": LOOP_METRIC, "value": first["us_per_step"], "unit": "us", "n_gpus": 1,
            "higher_is_better": False, "vs_baseline": None, "dtype": "f32", "data": "synthetic",
            "config": {"workload": task.name, "batch": B, "context": T,
                       "generated": int(T - start.min()), "vocab": task.V, "K": task.K,
                       "hidden_dim": task.d, "model": "stand-in: greedy output = target"},
            "rankings": results}
    print(json.dumps(line), flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(cfg, w, z, bf16, seconds, log, sampling=None):
    """The oracle's whole step on the host, on the same inputs: single-threaded
    (the reported value, with a per-operation breakdown), then the same oracle
    calls spread over sequences on a pool of threads (the C oracle releases the
    interpreter lock, so sequences run in parallel; the oracle itself is
    unchanged)."""
    import numpy as np
    import torch
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    toks, lens = w["tokens"], w["lens"]
    cp, cc, nu = oracle.find(toks, lens, *cfg.ngram)
    hb = None
    if w["hidden"] is not None:
        # the rows the step reads (H[T-2] and H[j-1]); the others stay zero pages
        B, T, d = w["hidden"].shape
        hb = np.zeros((B, T, d), np.uint16)
        for b in range(B):
            rows = sorted({int(lens[b]) - 2} | {int(j) - 1 for j in cp[b, :cc[b]]})
            idx = torch.tensor(rows, device=w["hidden"].device)
            hb[b, rows] = w["hidden"][b].index_select(0, idx).view(torch.int16).cpu().numpy() \
                .view(np.uint16)
    attn = w["attn"]
    agg = oracle.AGG_MAX if cfg.agg == "max" else oracle.AGG_SUM
    ops = {"find": 0.0, "rank": 0.0, "emit": 0.0, "verify": 0.0}

    def one(sl=slice(None), timing=None):
        t = time.perf_counter
        t0 = t()
        p, c, n = oracle.find(toks[sl], lens[sl], *cfg.ngram)
        t1 = t()
        if attn is not None:
            _, best, _ = oracle.rank_attn(attn[sl], lens[sl], p, c, agg, cfg.theta)
        if hb is not None:
            _, best, _ = oracle.rank_hidden(hb[sl], lens[sl], p, c, cfg.theta)
        t2 = t()
        dr, dl = oracle.emit(toks[sl], lens[sl], best, cfg.K)
        t3 = t()
        if sampling is not None:
            oracle.verify_sample(z[sl], dr, dl, sampling[0], sampling[1][sl], bf16=bf16)
        else:
            oracle.verify(z[sl], dr, dl, bf16=bf16)
        t4 = t()
        if timing is not None:
            for k, a_, b_ in (("find", t0, t1), ("rank", t1, t2), ("emit", t2, t3),
                              ("verify", t3, t4)):
                timing[k] += b_ - a_

    n = 0
    t0 = time.perf_counter()
    while True:
        one(timing=ops)
        n += 1
        if time.perf_counter() - t0 >= seconds:
            break
    dt = (time.perf_counter() - t0) / n
    log(f"[bench] cpu oracle: {n} whole steps, {dt * 1e3:.2f} ms per step")
    out = {"value": round(dt * 1e6, 1), "unit": "us", "cores": 1, "kind": "oracle",
           "sample": f"{n} whole steps of the same workload (all {cfg.B} sequences), "
                     f"single-threaded C oracle in fp64",
           "per_op_us": {k: round(v / n * 1e6, 1) for k, v in ops.items()},
           "cpu_model": cpu_model()}
    threads = min(cfg.B, 16, os.cpu_count() or 1)
    if threads > 1:
        parts = [slice(i, i + 1) for i in range(cfg.B)]
        with ThreadPoolExecutor(threads) as pool:
            m = 0
            t0 = time.perf_counter()
            while True:
                list(pool.map(lambda sl: one(sl), parts))
                m += 1
                if time.perf_counter() - t0 >= seconds / 2:
                    break
            dtp = (time.perf_counter() - t0) / m
        out["parallel"] = {"value": round(dtp * 1e6, 1), "unit": "us", "threads": threads,
                           "sample": f"{m} whole steps, one sequence per task"}
        log(f"[bench] cpu oracle on {threads} threads: {dtp * 1e3:.2f} ms per step")
    return out


if __name__ == "__main__":
    main()
