"""Calls on several streams at once.

Three callers, each with its own buffers, workspaces and stream, run whole
steps from host threads of their own at the same time: the one-call drafting
with one block per sequence, the one-call drafting with split positions on a
long context, and the separate calls with both rankings.  Every step must give
exactly what the same step gives when it runs alone: the library keeps no
device state between calls besides the caller's workspaces (the
allocation-free call's array aside, which this does not use), and its host
caches are locked.
"""
import threading

import numpy as np
import pytest
import torch

import synth
from gpu_helpers import say
from paper_2412_01447_amd.step import DraftStep

pytestmark = pytest.mark.gpu


def _case(B, T, V, d, R, K, mode, split, seed):
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(seed)
    toks, lens, _ = synth.make_tokens(B, T, V, s=1.1, plant_frac=0.3, span=(8, 32), seed=seed)
    hidden = synth.f32_to_bf16_bits(rng.standard_normal((B, T, d), dtype=np.float32))
    attn = rng.random((B, R, T), dtype=np.float32) if R else None
    logits = rng.standard_normal((B, K + 1, V), dtype=np.float32)
    step = DraftStep(B, T, K, device=dev, mode=mode, keep_scores=True)
    if split:
        step.set_split(split)
    args = dict(tokens=torch.from_numpy(toks).to(dev), lens=torch.from_numpy(lens).to(dev),
                logits=torch.from_numpy(logits).to(dev),
                hidden=torch.from_numpy(hidden.view(np.int16)).to(dev).view(torch.bfloat16),
                attn=torch.from_numpy(attn).to(dev) if attn is not None else None,
                ngram=(1, 2))
    return step, args


def test_steps_on_three_streams_from_three_threads():
    cases = [_case(4, 2048, 64, 512, 0, 8, "fused", 1, 31),
             _case(2, 20000, 200, 256, 0, 16, "fused", 8, 32),
             _case(3, 3000, 80, 128, 6, 8, "split", 0, 33)]
    say("streams: reference runs")
    refs = []
    for step, args in cases:
        step.run(**args)
        torch.cuda.synchronize()
        refs.append(step.host())
        assert refs[-1]["cand_count"].sum() > 0
    errors = []
    rounds = 25

    def worker(i):
        step, args = cases[i]
        s = torch.cuda.Stream()
        try:
            for r in range(rounds):
                with torch.cuda.stream(s):
                    step.run(**args, stream=s)
                s.synchronize()
                got = step.host()
                for name, want in refs[i].items():
                    if name in ("cand_pos", "scores", "scores_attn"):
                        # the listed prefix of each row (entries past the count are unspecified)
                        same = all(np.array_equal(got[name][b, :n].view(np.uint32),
                                                  want[b, :n].view(np.uint32))
                                   for b, n in enumerate(refs[i]["cand_count"]))
                    else:
                        same = np.array_equal(got[name], want)
                    if not same:
                        errors.append(f"caller {i} round {r}: {name} differs")
                        return
        except Exception as e:   # reported by the main thread
            errors.append(f"caller {i}: {e!r}")

    say("streams: three callers at once,", rounds, "rounds each")
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(cases))]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
