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


def random_plan(seed, iters):
    """Seed and case count of a seeded random-shape test: the defaults, unless
    PLD_RANDOM_SEED_OFFSET (added to the seed) or PLD_RANDOM_ITERS_SCALE (a
    factor on the count) ask for a wider sweep of new shapes."""
    import os
    off = int(os.environ.get("PLD_RANDOM_SEED_OFFSET", "0"))
    scale = float(os.environ.get("PLD_RANDOM_ITERS_SCALE", "1"))
    return np.random.default_rng(seed + off), max(1, int(round(iters * scale)))


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


def sample_workspace(B, K, V, bf16):
    n = pld.pld_verify_sample_workspace_bytes(B, K, V, pld.PLD_BF16 if bf16 else pld.PLD_F32)
    return torch.zeros(n, dtype=torch.uint8, device=dev())


def gpu_verify_sample(logits_dev, draft, draft_len, temperature, uniforms, ws=None):
    """pld_verify_sample; returns (accept_len, out_tokens, out_count, row_sample) and checks
    that the shared leading part of the workspace is zero again."""
    B, K1, V = logits_dev.shape
    bf16 = logits_dev.dtype == torch.bfloat16
    acc = torch.full((B,), -7, dtype=torch.int32, device=dev())
    out = torch.full((B, K1), -7, dtype=torch.int32, device=dev())
    cnt = torch.full((B,), -7, dtype=torch.int32, device=dev())
    rows = torch.full((B, K1), -7, dtype=torch.int32, device=dev())
    ws = sample_workspace(B, K1 - 1, V, bf16) if ws is None else ws
    u = uniforms if torch.is_tensor(uniforms) else d_f32(uniforms)
    pld.pld_verify_sample(logits_dev, d_i32(draft), d_i32(draft_len), temperature, u, acc, out,
                          cnt, ws, row_sample=rows)
    torch.cuda.synchronize()
    assert_ws_zero(ws[:pld.pld_workspace_bytes(B, K1 - 1)])
    return acc.cpu().numpy(), out.cpu().numpy(), cnt.cpu().numpy(), rows.cpu().numpy()


SAMPLE_EPS = 1e-5   # fp32 mass sums vs the fp64 oracle: tolerance on the target, relative to S


def sample_window_ok(z, temperature, u, y, eps=SAMPLE_EPS):
    """Is y the inverse-CDF sample of softmax(z / temperature) at u for a target
    within eps * S of u * S (fp64 masses)?  z: one row as float64."""
    m = z.max()
    if m == -np.inf:
        return y == 0
    if not 0 <= y < len(z):
        return False
    p = np.exp((z - m) / temperature)
    c = np.cumsum(p)
    S = c[-1]
    u = min(max(float(u), 0.0), float(np.nextafter(np.float32(1), np.float32(0))))
    if u != u:
        u = 0.0
    t = u * S
    before = c[y - 1] if y > 0 else 0.0
    return bool(p[y] > 0 and c[y] > t - eps * S and before <= t + eps * S)


def check_sample(z_rows, temperature, uniforms, draft, draft_len, g, r, what="",
                 max_flip_frac=0.02):
    """GPU sampling verification against the oracle's.  Rows past the draft and
    invalid lengths must match exactly; each sampled row must equal the oracle's
    token or be one that a target within SAMPLE_EPS * S would give (a flip, from
    fp32 vs fp64 mass sums, counted); acceptance and outputs must follow exactly
    from the GPU's own samples.  z_rows(b, i) -> float64 row.  Returns flips."""
    ga, go, gc, gy = g
    ra, ro, rc, ry = r
    B, K1 = gy.shape
    K = K1 - 1
    flips = rows = 0
    for b in range(B):
        L = int(draft_len[b])
        if L < 0 or L > K:
            assert (ga[b], gc[b]) == (-1, 0) and (go[b] == -1).all() and (gy[b] == -1).all(), \
                f"{what} b={b}: invalid length"
            continue
        assert (gy[b, L + 1:] == -1).all(), f"{what} b={b}: rows past the draft"
        for i in range(L + 1):
            rows += 1
            if gy[b, i] != ry[b, i]:
                flips += 1
                assert sample_window_ok(z_rows(b, i), temperature, uniforms[b, i], int(gy[b, i])), \
                    f"{what} b={b} i={i}: GPU {gy[b, i]} vs oracle {ry[b, i]} is no rounding flip"
        a = 0
        while a < L and gy[b, a] == draft[b, a]:
            a += 1
        want = np.full(K1, -1, np.int32)
        want[:a] = draft[b, :a]
        want[a] = gy[b, a]
        assert ga[b] == a and gc[b] == a + 1, f"{what} b={b}: accept {ga[b]} vs {a}"
        assert np.array_equal(go[b], want), f"{what} b={b}: out_tokens"
    assert flips <= max(3, max_flip_frac * rows), f"{what}: {flips} of {rows} rows flipped"
    if flips:
        print(f"  {what}: {flips} of {rows} sampled rows differ from the oracle within the "
              f"rounding window", flush=True)
    return flips


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
