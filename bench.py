#!/usr/bin/env python3
"""Benchmark of the PLD+ drafting step (find -> rank -> emit -> verify) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config C] [--verify greedy|sample]
                    [--temperature T] [--mode auto|fused|split|split_sep] [--split S] [--warm]
                    [--no-cpu-baseline] [--no-gate] [--copy-probe]
    python bench.py --loop TASK        # the generation loop, once per ranking
    python bench.py --probe            # bandwidth ceilings of the access patterns

A step is one pass of the whole hot path over one batch of synthetic input
already resident in HBM.  The default workload is config 4, the largest one
(batch 64, context 16384, vocabulary 128256, hidden 8192 bf16 and 64 attention
rows per sequence, both rankings, K = 16, bf16 logits); --config picks another
(1-5 scale the workload up, 6 and 7 are the paper's attention-MAX and
thresholded hidden-state settings at its input sizes); --verify sample
verifies by sampling at --temperature (default 1) instead of the argmax.  To
keep the caches honest the inputs exist in several copies at distinct
addresses and consecutive steps rotate through them, so every step reads from
HBM rather than from the 256 MB last-level cache.  W untimed steps run first,
then exactly K steps are timed between two device synchronisations; HIP
events on the launch stream bracket the ranking kernel, the attention
scoring (when the step ranks by both artifacts in launches of their own) and
the verification argmax, each on one step in eight, in turn (--event-every).
`roofline` is the ranking kernel's (both scorings in one launch when the step
ranks by both artifacts, else the hidden-state scoring when there is one, else
the attention scoring, else the one-call drafting); `rooflines_other` holds
the others.  With --gate (the default) the other two of the three largest
workloads (configs 3, 4, 5) are measured as well, in the same run, and their
ranking and verification fractions of peak are reported under `gate` (configs
3 and 5 both as their steps run -- the one-call drafting -- and with the
separate calls, where the ranking kernel is a launch of its own; config 4 also
with its two scorings in launches of their own).  One JSON
line goes to stdout.

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
    p.add_argument("--config", type=int, default=4, choices=[1, 2, 3, 4, 5, 6, 7])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=10.0,
                   help="CPU work the oracle baseline is given (whole steps, at least one)")
    p.add_argument("--warm", action="store_true",
                   help="one copy of the inputs, so steps re-read what the last-level cache holds "
                        "(labelled warm in the output); the default rotates cold copies")
    p.add_argument("--copy-probe", action="store_true",
                   help="after the timed region, copy 1 GiB three times (counter calibration)")
    p.add_argument("--event-every", type=int, default=8,
                   help="bracket each timed call (ranking, attention scoring, verification "
                        "argmax) with timing events on one step in N, in turn")
    p.add_argument("--gate", action=argparse.BooleanOptionalAction, default=True,
                   help="also measure the ranking and verification kernels of the three "
                        "largest workloads (configs 3, 4, 5) in the same run (default on)")
    p.add_argument("--gate-steps", type=int, default=200,
                   help="timed steps of each extra workload of --gate")
    p.add_argument("--split", type=int, default=0,
                   help="blocks per sequence of the one-call drafting (default: from the "
                        "first step's candidate counts)")
    p.add_argument("--mode", choices=["auto", "fused", "split", "split_sep"], default="auto",
                   help="drafting: one-launch call (fused), separate calls (split; with both "
                        "artifacts the two scorings share a launch), separate calls with each "
                        "scoring in a launch of its own (split_sep), or auto")
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
    if cfg.rank in ("hidden", "both"):
        out["score_hidden"] = int(((C + (C > 0)) * cfg.d * 2).sum() + C.sum() * 4)
    # the selection (key slots read and zeroed, per ranking) and the draft
    # (tokens read and written, lengths and choices written)
    nrank = 2 if cfg.rank == "both" else 1
    out["select_draft"] = int(nrank * B * 16 * 8 * 2 + B * K * 4 * 2 + nrank * B * 8 + B * 4)
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
        out["draft"] = sum(out.pop(k) for k in ("find", "score_hidden", "score_attn",
                                                "select_draft") if k in out)
    return out


# kernels behind each timed call (names as rocprofv3 reports them)
KERNELS = {"draft": "pld::draft_", "find": "pld::find_", "score_hidden": "pld::rank_hidden_kernel",
           "score_both": "pld::rank_both_kernel",
           "score_attn": "pld::rank_attn_kernel", "select_draft": "pld::select_draft_kernel",
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


def sources_sha256():
    import glob
    import hashlib
    h = hashlib.sha256()
    for fn in sorted(glob.glob(os.path.join(ROOT, "paper_2412_01447_amd", "csrc", "*"))):
        h.update(os.path.basename(fn).encode())
        with open(fn, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload, call):
    """HBM bytes per launch of the call's kernel from the committed counter runs
    (profiles/traffic.json), or None when the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    if sources_sha256() != table.get("sources_sha256"):
        return None
    rows = table.get("workloads", {}).get(workload, {})
    hits = [v for k, v in rows.items() if k.startswith(KERNELS.get(call, "?"))]
    return sum(hits) if hits else None


def drafting_label(m):
    """How a measured step drafted."""
    if m["fused"]:
        return f"one call, {m['draft_split']} block(s) per sequence"
    if "score_both" in m["calls"]:
        return "separate calls, both scorings in one launch"
    return "separate calls"


def ranking_call(names):
    """The call that holds the ranking kernel (Eq. 2 / Eq. 3): the hidden-state
    scoring when the step has one, else the attention scoring, else the one-call
    drafting (whose launch finds, ranks and selects)."""
    for n in ("score_both", "score_hidden", "score_attn", "draft"):
        if n in names:
            return n
    return None


def measure(cfg, args, log, mode=None, steps=None, warmup=None, cpu=False, cold=True):
    """One workload: inputs resident in HBM (rotated cold copies), W warm-up steps,
    then exactly K timed steps between two device synchronisations; HIP events on
    the launch stream bracket the ranking call, the verification argmax (or the
    sampling statistics) and, with two rankings, the attention scoring, each on
    every `event_every`-th step in turn.  Returns the step time, the byte counts
    and each bracketed call's timings; the CPU oracle's baseline when `cpu`."""
    import numpy as np
    import torch

    import synth
    from paper_2412_01447_amd import PLD_AGG_MAX, PLD_AGG_SUM
    from paper_2412_01447_amd.step import DraftStep
    mode = mode or args.mode
    steps = args.steps if steps is None else steps
    warmup = args.warmup if warmup is None else warmup
    dev = torch.device("cuda:0")
    t0 = time.time()
    w = synth.make_workload(cfg, dev, structured=True)
    toks, lens = w["tokens"], w["lens"]
    draft_i, dlen_i = synth.intended_drafts(w["metas"], cfg.K)
    z = synth.logits_for(w, draft_i, dlen_i)
    bf16 = cfg.logits == "bf16"
    elt = 2 if bf16 else 4
    log(f"[bench] {cfg.name}: inputs generated in {time.time() - t0:.1f}s")

    def dev_logits(a):
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16) if bf16 else a).to(dev)
        return t.view(torch.bfloat16) if bf16 else t

    base = dict(tokens=torch.from_numpy(toks).to(dev), lens=torch.from_numpy(lens).to(dev),
                logits=dev_logits(z), hidden=w["hidden"],
                attn=torch.from_numpy(w["attn"]).to(dev) if w["attn"] is not None else None)
    step = DraftStep(cfg.B, cfg.T, cfg.K, device=dev, mode="split" if mode == "split_sep" else mode,
                     rank_both=mode != "split_sep")
    fused = step.uses_fused(base["hidden"], base["attn"])
    sample = args.verify == "sample"
    if sample:
        step.set_sampling(args.temperature, cfg.V, bf16,
                          uniforms=torch.from_numpy(synth.make_uniforms(cfg.B, cfg.K, cfg.seed)).to(dev))
    rank_args = dict(ngram=cfg.ngram, agg=PLD_AGG_MAX if cfg.agg == "max" else PLD_AGG_SUM,
                     threshold=cfg.theta)

    # one step to learn the data-dependent byte counts (and, for the one-call
    # drafting, how many blocks should share a sequence)
    step.run(base["tokens"], base["lens"], base["logits"], hidden=base["hidden"],
             attn=base["attn"], **rank_args)
    torch.cuda.synchronize()
    nbytes = algorithmic_bytes(cfg, lens, step.cand_count.cpu().numpy(),
                               step.draft_len.cpu().numpy(), step.cand_pos.cpu().numpy(), elt,
                               fused, sample=sample)
    step_bytes = sum(nbytes.values())
    # input copies at distinct addresses: the steps of one rotation touch at
    # least twice the last-level cache
    copies = 1 if not cold else int(min(64, max(2, math.ceil(2 * MALL_BYTES /
                                                              max(step_bytes, 1)))))
    sets = [base]
    for _ in range(copies - 1):
        sets.append({k: (v.clone() if v is not None else None) for k, v in base.items()})
    torch.cuda.synchronize()
    log(f"[bench] step bytes {step_bytes / 1e6:.2f} MB {json.dumps(nbytes)}; {copies} input copies")
    stream = torch.cuda.current_stream()
    if fused:
        # blocks per sequence for the one-call drafting, from the first step's
        # candidate counts (or as given)
        if args.split:
            step.set_split(args.split)
        else:
            step.tune_split(step.cand_count.cpu().numpy(), hidden=base["hidden"] is not None)
        log(f"[bench] drafting with {step.draft_split} block(s) per sequence")
    # every step as prepared calls (arguments marshalled once, one kernel each)
    plans = [step.plan(s_["tokens"], s_["lens"], s_["logits"], hidden=s_["hidden"],
                       attn=s_["attn"], stream=stream, **rank_args) for s_ in sets]
    names = [n for n, _ in plans[0]]
    if "score_both" in names:   # both scorings in one launch
        nbytes["score_both"] = nbytes.pop("score_hidden") + nbytes.pop("score_attn")
    assert set(names) == set(nbytes), (names, list(nbytes))
    rank = ranking_call(names)
    timed = [rank] + [n for n in ("score_attn",) if n in names and n != rank] + \
            ["verify_sample_stats" if sample else "verify_argmax"]
    E = args.event_every
    assert len(timed) <= E
    slots = [(k, timed[k % E]) for k in range(steps) if k % E < len(timed)]
    ev = TimingEvents(len(slots))
    which = {k: (i, name) for i, (k, name) in enumerate(slots)}

    for k in range(warmup):
        for _, call in plans[k % copies]:
            call()
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for k in range(steps):
        i, target = which.get(k, (-1, None))
        for name, call in plans[k % copies]:
            if name == target:
                ev.record(2 * i, stream)
                call()
                ev.record(2 * i + 1, stream)
            else:
                call()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t_start
    per_call = {}
    for i, (k, name) in enumerate(slots):
        per_call.setdefault(name, []).append(ev.elapsed_ms(2 * i, 2 * i + 1))
    ev.close()
    calls = {}
    for name, ms in per_call.items():
        avg = sum(ms) / len(ms)
        ach = nbytes[name] / (avg * 1e-3) / 1e9
        calls[name] = {"kernel": KERNELS[name], "achieved": round(ach, 1),
                       "frac": round(ach / HBM_PEAK_GBS, 4), "bytes_per_launch": nbytes[name],
                       "avg_us": round(avg * 1e3, 2),
                       **{f"p{q}_us": round(float(np.percentile(ms, q)) * 1e3, 2)
                          for q in (10, 50, 90)},
                       "launches_timed": len(ms)}
        log(f"[bench] {name}: {avg * 1e3:.2f} us avg, {ach:.1f} GB/s "
            f"({ach / HBM_PEAK_GBS:.3f} of peak)")
    out = {"cfg": cfg, "step": step, "fused": fused, "sample": sample, "copies": copies,
           "nbytes": nbytes, "step_bytes": step_bytes, "us_per_step": elapsed * 1e6 / steps,
           "calls": calls, "rank": rank, "w": w, "z": z, "bf16": bf16,
           "draft_split": step.draft_split}
    if cpu:
        out["cpu"] = cpu_baseline(cfg, w, z, bf16, args.cpu_seconds, log,
                                  (args.temperature, synth.make_uniforms(cfg.B, cfg.K, cfg.seed))
                                  if sample else None)
    del sets, plans, base
    return out


def roofline_of(cfg, call, rec):
    """The roofline object of one bracketed call."""
    return {"bound": "hbm", "kernel": call, "achieved": rec["achieved"], "peak": HBM_PEAK_GBS,
            "unit": "GB/s", "frac": rec["frac"], "traffic": measured_traffic(cfg.name, call),
            **{k: rec[k] for k in ("bytes_per_launch", "avg_us", "p10_us", "p50_us", "p90_us",
                                   "launches_timed")}}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU (--gpus 1): the step shards by sequence with no "
              "exchange between GPUs, so more GPUs only scale the batch.", file=sys.stderr)
        sys.exit(2)
    import torch

    import synth

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
    log = lambda *a: print(*a, file=sys.stderr, flush=True)
    log(f"[bench] config {args.config}: {cfg.name}")
    m = measure(cfg, args, log, cpu=not args.no_cpu_baseline, cold=not args.warm)
    step, fused, sample = m["step"], m["fused"], m["sample"]
    rank = m["rank"]
    roofline = roofline_of(cfg, rank, m["calls"][rank]) if rank in m["calls"] else None
    others = {n: roofline_of(cfg, n, r) for n, r in m["calls"].items() if n != rank}

    if args.copy_probe:
        dev = torch.device("cuda:0")
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("[bench] copy probe: 3 x 1 GiB device copies done")

    gate = None
    if args.gate and not args.warm:
        # the other two of the three largest workloads, measured in the same run
        # (their own step configuration, fewer steps, no CPU baseline): the
        # fractions of peak of their ranking and verification kernels.  Their
        # steps draft with the one-call drafting, whose launch also finds the
        # occurrences and is followed by its finishing launch; each is also
        # run with the separate calls, where the ranking kernel is timed alone.
        m.pop("w"), m.pop("z"), m.pop("step")
        torch.cuda.empty_cache()
        gate = {}
        runs = [(3, None), (3, "split"), (4, None), (4, "split_sep"), (5, None), (5, "split")]
        for cid, mode in runs:
            if cid == args.config and mode is None:
                g = m
            else:
                g = measure(synth.CONFIGS[cid], args, log, mode=mode, steps=args.gate_steps,
                            warmup=args.warmup)
            suffix = {"split": "_separate_calls", "split_sep": "_separate_rankings"}
            gate[f"config{cid}" + suffix.get(mode, "")] = {
                "workload": synth.CONFIGS[cid].name, "us_per_step": round(g["us_per_step"], 2),
                "drafting": drafting_label(g),
                **{n: {"avg_us": r["avg_us"], "p50_us": r["p50_us"], "GBps": r["achieved"],
                       "frac": r["frac"], "bytes": r["bytes_per_launch"]}
                   for n, r in g["calls"].items()}}
            if g is not m:
                del g
                torch.cuda.empty_cache()

    line = {
        "metric": METRIC, "value": round(m["us_per_step"], 2), "unit": "us", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(m["us_per_step"] / 1e3, 5),
        "higher_is_better": False, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": cfg.name, "batch": cfg.B, "context": cfg.T, "vocab": cfg.V,
                   "ngram": list(cfg.ngram), "ranking": cfg.rank, "hidden_dim": cfg.d,
                   "attn_rows": cfg.R, "attn_aggregation": cfg.agg, "threshold": cfg.theta,
                   "K": cfg.K, "logits": cfg.logits,
                   "inputs": "hidden bf16, attention f32, tokens int32",
                   "drafting": drafting_label(m),
                   "verification": (f"sampling at temperature {args.temperature}" if sample
                                    else "greedy"),
                   "input_copies": m["copies"],
                   "cache": "warm: one copy of the inputs" if args.warm else
                            "cold: copies rotated past the last-level cache",
                   **({"attn_bytes_dense": int(cfg.B) * cfg.R * cfg.T * 4}
                      if cfg.rank in ("attn", "both") else {}),
                   "step_bytes": m["step_bytes"]},
        "roofline": roofline,
        "rooflines_other": others,
        "cpu_baseline": m.get("cpu"),
    }
    if gate is not None:
        line["gate"] = gate
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
    try:
        affinity = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        affinity = None
    out = {"value": round(dt * 1e6, 1), "unit": "us", "cores": 1, "kind": "oracle",
           "host_cores": os.cpu_count(), "host_cores_usable": affinity,
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
