"""Helpers for the GPU parity tests: device transfer, stage runners, comparisons.

The comparison rules (the parity bar):
* candidate positions, counts, n used, chosen candidate, draft tokens and
  lengths, accepted lengths and emitted tokens: bit-exact;
* similarity / attention scores: |s_gpu - s_ref| <= 1e-3 |s_ref| + 1e-6 (fp32
  accumulation of bf16 / fp32 inputs against the oracle's fp64);
* a chosen candidate that differs from the oracle's is a "near-tie flip" and
  is counted, not failed, only when the oracle's scores of the two choices
  differ by less than 1e-3 relative; every stage after a flip is then checked
  on the oracle's own inputs.
"""
import math
import sys

import numpy as np
import torch

import oracle
import paper_2412_01447_amd as pld

RTOL = 1e-3
ATOL = 1e-6


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def dev():
    return torch.device("cuda:0")


def d_i32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev())


def d_f32(a):
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(dev())


def d_bf16(bits):
    t = torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16))
    return t.to(dev()).view(torch.bfloat16)


def h_bits(t):
    """bf16 device/host tensor -> uint16 numpy bits."""
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def workspace(B, K):
    return torch.zeros(pld.pld_workspace_bytes(B, K), dtype=torch.uint8, device=dev())


def draft_workspace(B, S):
    """The one-call drafting's workspace (None for one block per sequence)."""
    n = pld.pld_draft_workspace_bytes(B, S)
    return torch.zeros(n, dtype=torch.uint8, device=dev()) if n else None


def draft_keys_zero(ws, B):
    """The key slots (the first B*128 bytes) are left zero by every call."""
    return ws is None or int(torch.count_nonzero(ws[:B * 128]).item()) == 0


def scratch(B, tok_stride, fill=0x5A):
    """Find scratch, deliberately filled with garbage: its contents must not matter."""
    n = pld.pld_find_scratch_bytes(B, tok_stride)
    return torch.full((n,), fill, dtype=torch.uint8, device=dev()) if n else None


def assert_ws_zero(ws):
    torch.cuda.synchronize()
    nz = int(torch.count_nonzero(ws).item())
    assert nz == 0, f"workspace not returned to zero ({nz} bytes set)"


# ------------------------------------------------------------------ stages
def gpu_find(tokens, lens, nmin, nmax, cap=None, scr=None):
    B, stride = tokens.shape
    cap = stride if cap is None else cap
    t, l = d_i32(tokens), d_i32(lens)
    cp = torch.full((B, cap), -1, dtype=torch.int32, device=dev())
    cc = torch.full((B,), -7, dtype=torch.int32, device=dev())
    nu = torch.full((B,), -7, dtype=torch.int32, device=dev())
    scr = scratch(B, stride) if scr is None else scr
    pld.pld_find_candidates(t, l, nmin, nmax, cp, cc, nu, scr)
    torch.cuda.synchronize()
    return cp.cpu().numpy(), cc.cpu().numpy(), nu.cpu().numpy()


def check_find(g, r, what=""):
    gp, gc, gn = g
    rp, rc, rn = r
    assert np.array_equal(gc, rc), f"{what} cand_count {gc} vs {rc}"
    assert np.array_equal(gn, rn), f"{what} ngram_used {gn} vs {rn}"
    for b in range(len(rc)):
        assert np.array_equal(gp[b, :rc[b]], rp[b, :rc[b]]), f"{what} cand_pos of sequence {b}"


def gpu_rank_hidden(hidden_dev, lens, cp, cc, threshold=-math.inf, ws=None):
    B = hidden_dev.shape[0]
    cap = cp.shape[1]
    bp = torch.full((B,), -7, dtype=torch.int32, device=dev())
    bs = torch.zeros(B, dtype=torch.float32, device=dev())
    sc = torch.full((B, cap), 12345.0, dtype=torch.float32, device=dev())
    ws = workspace(B, 1) if ws is None else ws
    pld.pld_rank_hidden(hidden_dev, d_i32(lens), d_i32(cp), d_i32(cc), bp, bs, ws,
                        threshold=threshold, scores=sc)
    torch.cuda.synchronize()
    assert_ws_zero(ws)
    return sc.cpu().numpy(), bp.cpu().numpy(), bs.cpu().numpy()


def gpu_rank_attn(attn_dev, lens, cp, cc, agg, threshold=-math.inf, ws=None):
    B = attn_dev.shape[0]
    cap = cp.shape[1]
    bp = torch.full((B,), -7, dtype=torch.int32, device=dev())
    bs = torch.zeros(B, dtype=torch.float32, device=dev())
    sc = torch.full((B, cap), 12345.0, dtype=torch.float32, device=dev())
    ws = workspace(B, 1) if ws is None else ws
    pld.pld_rank_attn(attn_dev, d_i32(lens), d_i32(cp), d_i32(cc), bp, bs, ws, agg=agg,
                      threshold=threshold, scores=sc)
    torch.cuda.synchronize()
    assert_ws_zero(ws)
    return sc.cpu().numpy(), bp.cpu().numpy(), bs.cpu().numpy()


def check_scores(gsc, rsc, cc, what=""):
    for b in range(len(cc)):
        n = max(0, min(int(cc[b]), rsc.shape[1]))
        g, r = gsc[b, :n].astype(np.float64), rsc[b, :n]
        nan_r = np.isnan(r)
        assert np.array_equal(np.isnan(g), nan_r), f"{what} NaN pattern of sequence {b}"
        err = np.abs(g[~nan_r] - r[~nan_r])
        lim = RTOL * np.abs(r[~nan_r]) + ATOL
        bad = np.nonzero(err > lim)[0]
        assert len(bad) == 0, (f"{what} score of sequence {b}, slot {bad[0]}: "
                               f"{g[~nan_r][bad[0]]} vs {r[~nan_r][bad[0]]}")


def check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, what="", threshold=-math.inf):
    """Bit-exact chosen candidate, or a counted near-tie flip.  Returns #flips."""
    flips = 0
    for b in range(len(rbp)):
        if gbp[b] == rbp[b]:
            if rbp[b] < 0:
                assert gbs[b] == -math.inf, f"{what} best_score of empty sequence {b}"
            else:
                assert abs(gbs[b] - rbs[b]) <= RTOL * abs(rbs[b]) + ATOL, (
                    f"{what} best_score {gbs[b]} vs {rbs[b]} (sequence {b})")
            continue
        # a flip is legitimate only between two eligible near-equal candidates
        n = int(cc[b])
        slots = {int(cp[b, c]): c for c in range(n)}
        assert gbp[b] in slots and rbp[b] >= 0, (
            f"{what} best_pos {gbp[b]} vs {rbp[b]} (sequence {b}) is not a near tie")
        s_g = rsc[b, slots[int(gbp[b])]]
        assert s_g > threshold and abs(rbs[b] - s_g) < RTOL * abs(rbs[b]), (
            f"{what} best_pos {gbp[b]} vs {rbp[b]} (sequence {b}): oracle scores "
            f"{s_g} vs {rbs[b]} are not a near tie")
        flips += 1
    return flips


def gpu_emit(tokens, lens, best_pos, K):
    B = tokens.shape[0]
    dr = torch.full((B, K), -7, dtype=torch.int32, device=dev())
    dl = torch.full((B,), -7, dtype=torch.int32, device=dev())
    pld.pld_emit_draft(d_i32(tokens), d_i32(lens), d_i32(best_pos), K, dr, dl)
    torch.cuda.synchronize()
    return dr.cpu().numpy(), dl.cpu().numpy()


def gpu_verify(logits_dev, draft, draft_len, ws=None):
    B, K1, V = logits_dev.shape
    acc = torch.full((B,), -7, dtype=torch.int32, device=dev())
    out = torch.full((B, K1), -7, dtype=torch.int32, device=dev())
    cnt = torch.full((B,), -7, dtype=torch.int32, device=dev())
    ws = workspace(B, K1 - 1) if ws is None else ws
    pld.pld_verify_greedy(logits_dev, d_i32(draft), d_i32(draft_len), acc, out, cnt, ws)
    torch.cuda.synchronize()
    assert_ws_zero(ws)
    return acc.cpu().numpy(), out.cpu().numpy(), cnt.cpu().numpy()


def check_verify(g, r, what=""):
    ga, go, gc = g
    ra, ro, rc = r[:3]
    assert np.array_equal(ga, ra), f"{what} accept_len {ga} vs {ra}"
    assert np.array_equal(gc, rc), f"{what} out_count {gc} vs {rc}"
    assert np.array_equal(go, ro), f"{what} out_tokens differ"


def sparse_hidden_rows(hidden_dev, lens, cp, cc):
    """Host copy holding only the rows the oracle reads (H[T-2] and H[j-1]); the
    rest stays as untouched zero pages."""
    B, n_rows, d = hidden_dev.shape
    host = np.zeros((B, n_rows, d), np.uint16)
    for b in range(B):
        T = int(lens[b])
        rows = set()
        if 2 <= T and T - 2 < n_rows:
            rows.add(T - 2)
        n = int(cc[b])
        if 0 <= n <= cp.shape[1]:
            rows.update(int(j) - 1 for j in cp[b, :n] if 1 <= j <= T - 2)
        if rows:
            idx = torch.tensor(sorted(rows), dtype=torch.long, device=hidden_dev.device)
            host[b, idx.cpu().numpy()] = h_bits(hidden_dev[b].index_select(0, idx))
    return host
