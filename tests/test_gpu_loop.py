"""GPU parity of the steps either side of the drafting path: prompt lookup's
selection (pld_select_prefix) and the commit (pld_commit), then the whole
generation loop (draft -> verify -> commit) run in lockstep with an oracle loop
on a synthetic decoding task, every step compared.

Greedy verification against the stand-in target model reproduces the target
sequences whatever the drafts, so every loop must end with them; the drafts
decide only how many steps it takes (the paper's average acceptance length).
"""
import math

import numpy as np
import pytest
import torch

import golden_cases
import oracle
import paper_2412_01447_amd as pld
import synth
from gpu_helpers import RTOL, d_f32, d_i32, dev, say
from paper_2412_01447_amd.step import DraftStep, decode_loop

pytestmark = pytest.mark.gpu


def gpu_select_prefix(toks, lens, cp, cc, max_match):
    B, cap = cp.shape
    scores = torch.full((B, cap), -7.0, device=dev())
    bp = torch.full((B,), -7, dtype=torch.int32, device=dev())
    bs = torch.zeros(B, device=dev())
    pld.pld_select_prefix(d_i32(toks), d_i32(lens), d_i32(cp), d_i32(cc), bp, bs, max_match,
                          scores=scores)
    torch.cuda.synchronize()
    return scores.cpu().numpy(), bp.cpu().numpy(), bs.cpu().numpy()


def check_prefix(g, r, cc, what):
    gs, gb, gbs = g
    rs, rb, rbs = r
    for b in range(len(rb)):
        n = int(cc[b]) if 0 <= cc[b] <= rs.shape[1] else 0
        a, e = gs[b, :n], rs[b, :n].astype(np.float32)
        assert np.array_equal(np.isnan(a), np.isnan(e)), f"{what} b={b}: NaN pattern"
        assert np.array_equal(a[~np.isnan(a)], e[~np.isnan(e)]), f"{what} b={b}: lengths"
    assert np.array_equal(gb, rb), f"{what}: best_pos {gb} vs {rb}"
    assert np.array_equal(gbs, rbs.astype(np.float32)), f"{what}: best_score"


@pytest.mark.parametrize("B,T,V,nmin,nmax,seed", [(4, 300, 3, 1, 1, 0), (6, 2000, 5, 1, 3, 1),
                                                  (3, 9000, 40, 1, 4, 2), (2, 70000, 2, 2, 2, 3)])
def test_select_prefix_parity(B, T, V, nmin, nmax, seed):
    """Random rows over small vocabularies (many long matches, several 16-token
    rounds), planted long copies, ragged and invalid lengths, every cap."""
    say("select_prefix", B, T, V, nmin, nmax, seed)
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, V, size=(B, T)).astype(np.int32)
    lens = rng.integers(T // 2, T + 1, size=B).astype(np.int32)
    lens[0] = T
    Tq = int(lens[0])
    for src in (100, 5):                    # long copies of the query's context
        ln = min(300, src + 1, Tq - 1 - src)
        if ln > 0:
            toks[0, src - ln + 1:src + 1] = toks[0, Tq - ln:Tq]
    if B > 2:
        lens[2] = 1                          # too short: no choice
    cp, cc, _ = oracle.find(toks, lens, nmin, nmax)
    for mm in (1, 3, 15, 16, 17, 64, 1024):
        r = oracle.select_prefix(toks, lens, cp, cc, mm)
        check_prefix(gpu_select_prefix(toks, lens, cp, cc, mm), r, cc, f"max_match {mm}")


def test_select_prefix_arbitrary_positions_and_fig3():
    """Candidates outside [0, T-2] score NaN and are never chosen; counts past
    cap count as 0; the Fig. 3 fixture gives prompt lookup's choice, f's span."""
    say("select_prefix positions")
    rng = np.random.default_rng(9)
    toks = rng.integers(0, 3, size=(3, 64)).astype(np.int32)
    lens = np.array([64, 40, 64], np.int32)
    cp = np.array([[-3, 0, 5, 62, 63, 64, 10], [39, 38, 0, 1, 2, 100, -1], [1, 2, 3, 4, 5, 6, 7]],
                  np.int32)
    cc = np.array([7, 6, 9], np.int32)
    r = oracle.select_prefix(toks, lens, cp, cc, 8)
    check_prefix(gpu_select_prefix(toks, lens, cp, cc, 8), r, cc, "positions")
    fx, ft, fl, _, _ = golden_cases.load("fig3_newline.json")
    e = fx["expected"]["pld_prefix"]
    fcp, fcc, _ = oracle.find(ft, fl, 1, 1)
    for cap_m in (8, 3, 1):
        gs, gb, gbs = gpu_select_prefix(ft, fl, fcp, fcc, cap_m)
        assert list(gs[0, :fcc[0]]) == e[f"match_len_max{cap_m}"] and gb[0] == e[f"best_pos_max{cap_m}"]


def test_commit_parity():
    """Appends under limits and row capacity, invalid lengths and counts left
    alone, counters accumulated over two calls; every byte of the rows checked."""
    say("commit")
    rng = np.random.default_rng(4)
    B, stride, K = 9, 50, 6
    toks = rng.integers(0, 100, size=(B, stride)).astype(np.int32)
    lens = np.array([0, 10, 49, 50, 45, -1, 51, 20, 30], np.int32)
    out = rng.integers(1000, 2000, size=(B, K + 1)).astype(np.int32)
    cnt = np.array([7, 3, 7, 2, 7, 3, 2, 0, 8], np.int32)
    limit = np.array([50, 12, 50, 50, 48, 50, 50, 50, 50], np.int32)
    stats0 = rng.integers(0, 9, size=(B, 2)).astype(np.int64)
    td, ld = d_i32(toks), d_i32(lens)
    sd = torch.from_numpy(stats0.copy()).to(dev())
    want_t, want_l, want_s = toks, lens, stats0
    for call in range(2):
        pld.pld_commit(td, ld, d_i32(out), d_i32(cnt), limit=d_i32(limit), stats=sd)
        want_t, want_l, want_s = oracle.commit(want_t, want_l, out, cnt, limit=limit,
                                               stats=want_s)
        torch.cuda.synchronize()
        assert np.array_equal(td.cpu().numpy(), want_t), f"call {call}: tokens"
        assert np.array_equal(ld.cpu().numpy(), want_l), f"call {call}: lens"
        assert np.array_equal(sd.cpu().numpy(), want_s), f"call {call}: stats"
    # no limit, no counters
    td, ld = d_i32(toks), d_i32(lens)
    pld.pld_commit(td, ld, d_i32(out), d_i32(cnt))
    t2, l2, _ = oracle.commit(toks, lens, out, cnt)
    torch.cuda.synchronize()
    assert np.array_equal(td.cpu().numpy(), t2) and np.array_equal(ld.cpu().numpy(), l2)


def test_accept_commit_parity():
    """pld_accept_commit equals pld_verify_accept followed by pld_commit, and the
    oracle's verification and commit: accepted lengths, emitted tokens, rows,
    lengths and counters, over two steps, with invalid draft lengths, limits that
    cut the append and invalid sequence lengths; the workspace ends at zero."""
    say("accept + commit")
    rng = np.random.default_rng(11)
    B, K, V, stride = 9, 6, 50, 40
    Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
    agree = np.array([6, 0, 2, 6, 3, 6, 1, 6, 4])
    for b in range(B):
        draft[b, :agree[b]] = Z[b, :agree[b]].argmax(axis=1)
    dlen = np.array([6, 0, 3, 6, -1, 7, 6, 2, 6], np.int32)
    toks = rng.integers(0, 100, size=(B, stride)).astype(np.int32)
    lens = np.array([10, 38, 40, 0, 5, 12, -1, 39, 20], np.int32)
    limit = np.array([40, 40, 40, 3, 40, 40, 40, 40, 25], np.int32)
    stats0 = rng.integers(0, 9, size=(B, 2)).astype(np.int64)
    zd, dr, dl, lim = d_f32(Z), d_i32(draft), d_i32(dlen), d_i32(limit)
    i32 = dict(dtype=torch.int32, device=dev())
    runs = {}
    for fused in (False, True):
        ws = torch.zeros(pld.pld_workspace_bytes(B, K), dtype=torch.uint8, device=dev())
        td, ld = d_i32(toks), d_i32(lens)
        sd = torch.from_numpy(stats0.copy()).to(dev())
        acc, out, cnt = (torch.full((B,), -7, **i32), torch.full((B, K + 1), -7, **i32),
                         torch.full((B,), -7, **i32))
        for _ in range(2):
            pld.pld_verify_argmax(zd, dl, ws)
            if fused:
                pld.pld_accept_commit(dr, dl, acc, out, cnt, td, ld, ws, limit=lim, stats=sd)
            else:
                pld.pld_verify_accept(dr, dl, acc, out, cnt, ws)
                pld.pld_commit(td, ld, out, cnt, limit=lim, stats=sd)
            torch.cuda.synchronize()
            assert int(torch.count_nonzero(ws).item()) == 0
        runs[fused] = [t.cpu().numpy() for t in (acc, out, cnt, td, ld, sd)]
    for x, y in zip(runs[False], runs[True]):
        assert np.array_equal(x, y)
    ra, ro, rc, _ = oracle.verify(Z, draft, dlen)
    wt, wl, ws_ = toks, lens, stats0
    for _ in range(2):
        wt, wl, ws_ = oracle.commit(wt, wl, ro, rc, limit=limit, stats=ws_)
    acc, out, cnt, t, l, s_ = runs[True]
    assert np.array_equal(acc, ra) and np.array_equal(out, ro) and np.array_equal(cnt, rc)
    assert np.array_equal(t, wt) and np.array_equal(l, wl) and np.array_equal(s_, ws_)


# ------------------------------------------------------------- the loop
LOOPS = [("b1_t1024_copy60_k10", "hidden", None, (1, 1)),
         ("b1_t1024_copy60_k10", "prefix", 3, (1, 3)),
         ("b1_t1024_copy60_k10", "prefix", 64, (1, 1)),
         ("b8_t4096_copy50_k16", "hidden", None, (1, 1)),
         ("b8_t4096_copy50_k16", "prefix", 3, (1, 3)),
         ("b1_t1024_sections_edit10_k10", "hidden", None, (1, 1)),
         ("b1_t1024_sections_edit10_k10", "prefix", 3, (1, 3)),
         ("b8_t4096_sections_edit10_k16", "hidden", None, (1, 1)),
         ("b8_t4096_sections_edit10_k16", "prefix", 64, (1, 1))]


@pytest.mark.parametrize("task_name,ranking,max_match,ngram", LOOPS,
                         ids=[f"{t}_{r}{m or ''}" for t, r, m, _ in LOOPS])
def test_decode_loop_lockstep(task_name, ranking, max_match, ngram):
    """draft -> verify -> commit on the device, the same loop with the oracle on
    the host, compared after every step: candidates, choice (a near-tie flip of
    the cosine is adopted by the oracle and counted), draft, acceptance, the
    committed rows, lengths and counters.  Both end on the target sequences."""
    task = synth.DECODE_TASKS[task_name]
    say("decode loop", task_name, ranking, max_match, ngram)
    w = synth.make_decode_task(task, device=dev())
    target, start = w["target"], w["start"]
    B, T = target.shape
    hidden = w["hidden"] if ranking == "hidden" else None
    hbits = (hidden.view(torch.int16).cpu().numpy().view(np.uint16)
             if hidden is not None else None)
    model = synth.TargetModel(target, task.K, task.V, task.seed, device=dev())
    base = model.base.cpu().numpy()

    toks = np.where(np.arange(T)[None, :] < start[:, None], target, -1).astype(np.int32)
    td, ld = d_i32(toks), d_i32(start)
    limit = d_i32(np.full(B, T, np.int32))
    stats = torch.zeros((B, 2), dtype=torch.int64, device=dev())
    step = DraftStep(B, T, task.K, device=dev(), keep_scores=True)
    ref = dict(x=toks.copy(), T=start.copy(), stats=np.zeros((B, 2), np.int64), flips=0)

    def oracle_step(i):
        x, Tn = ref["x"], ref["T"]
        cp, cc, nu = oracle.find(x, Tn, *ngram)
        g = step.host()
        assert np.array_equal(g["cand_count"], cc), f"step {i}: counts"
        if ranking == "hidden":
            sc, bp, bs = oracle.rank_hidden(hbits, Tn, cp, cc)
        else:
            sc, bp, bs = oracle.select_prefix(x, Tn, cp, cc, max_match)
        for b in range(B):
            if g["best_pos"][b] != bp[b]:
                assert ranking == "hidden", f"step {i} b={b}: prefix choice differs"
                slots = {int(cp[b, c]): c for c in range(cc[b])}
                s_g = sc[b, slots[int(g["best_pos"][b])]]
                assert abs(bs[b] - s_g) < RTOL * abs(bs[b]), f"step {i} b={b}: not a near tie"
                bp[b] = g["best_pos"][b]
                ref["flips"] += 1
        dr, dl = oracle.emit(x, Tn, bp, task.K)
        assert np.array_equal(g["draft"], dr) and np.array_equal(g["draft_len"], dl), \
            f"step {i}: draft"
        z = base.copy()
        pos = np.minimum(Tn[:, None] + np.arange(task.K + 1)[None, :], T - 1)
        tgt = np.take_along_axis(target, pos, axis=1)
        for b in range(B):
            z[b, np.arange(task.K + 1), tgt[b]] += np.float32(model.boost)
        acc, out, cnt, _ = oracle.verify(z, dr, dl)
        assert np.array_equal(g["accept_len"], acc) and np.array_equal(g["out_count"], cnt), \
            f"step {i}: acceptance"
        assert np.array_equal(g["out_tokens"], out), f"step {i}: out_tokens"
        ref["x"], ref["T"], ref["stats"] = oracle.commit(x, Tn, out, cnt,
                                                         limit=np.full(B, T, np.int32),
                                                         stats=ref["stats"])
        assert np.array_equal(ld.cpu().numpy(), ref["T"]), f"step {i}: lens"
        assert np.array_equal(td.cpu().numpy(), ref["x"]), f"step {i}: tokens"
        assert np.array_equal(stats.cpu().numpy(), ref["stats"]), f"step {i}: stats"

    n = decode_loop(step, td, ld, limit, lambda st, lens: model.logits(lens), hidden=hidden,
                    ngram=ngram, prefix_match=max_match, stats=stats, check_every=1,
                    on_step=oracle_step)
    assert np.array_equal(td.cpu().numpy(), target), "the loop must end on the targets"
    s = stats.cpu().numpy()
    assert (s[:, 0] == T - start).all()
    say(f"  {n} steps, average acceptance length {s[:, 0].sum() / s[:, 1].sum():.3f}, "
        f"near-tie flips {ref['flips']}")
