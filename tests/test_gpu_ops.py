"""GPU parity of each call of the C ABI against the CPU oracle, on small and
edge-case inputs (several tiles, ragged tails, empty and invalid cases).

Every case prints its name before touching the GPU.  Inputs are seeded; the
oracle sees the same bytes as the kernels; comparisons follow gpu_helpers.
"""
import math

import numpy as np
import pytest
import torch

import golden_cases
import oracle
import paper_2412_01447_amd as pld
import synth
from gpu_helpers import (check_best, check_find, check_scores, check_verify, d_bf16, d_f32,
                         draft_keys_zero, draft_workspace, random_plan,
                         d_i32, dev, gpu_emit, gpu_find, gpu_rank_attn, gpu_rank_hidden,
                         gpu_verify, say, scratch, workspace, assert_ws_zero)

pytestmark = pytest.mark.gpu


# ----------------------------------------------------------------- golden
def _pad8(H):
    """The library takes d % 8 == 0; zero columns leave every dot product and norm unchanged."""
    d = H.shape[-1]
    return np.concatenate([H, np.zeros(H.shape[:-1] + ((-d) % 8,), np.float32)], axis=-1)


def test_golden_fig1_on_gpu():
    say("golden fig1")
    fx, toks, lens, H, A = golden_cases.load("fig1_overview.json")
    H = _pad8(H)
    ex = fx["expected"]
    cp, cc, nu = gpu_find(toks, lens, 1, 1)
    assert list(cp[0, :cc[0]]) == ex["cand_pos"] and nu[0] == 1
    bits = synth.f32_to_bf16_bits(H)
    sc, bp, bs = gpu_rank_hidden(d_bf16(bits), lens, cp, cc)
    np.testing.assert_allclose(sc[0, :2], ex["hidden_scores"], rtol=1e-6, atol=1e-7)
    assert bp[0] == ex["hidden_best_pos"]
    for agg, key in ((pld.PLD_AGG_SUM, "attn_sum"), (pld.PLD_AGG_MAX, "attn_max")):
        sc, bp, bs = gpu_rank_attn(d_f32(A), lens, cp, cc, agg)
        assert list(sc[0, :2]) == ex[key + "_scores"] and bp[0] == ex[key + "_best_pos"]
    for K in (3, 12):
        dr, dl = gpu_emit(toks, lens, np.array([10], np.int32), K)
        assert list(dr[0]) == ex[f"draft_K{K}"] and dl[0] == ex[f"draft_len_K{K}"]
    for vc in fx["verify_cases"]:
        Z, dr, dl = golden_cases.verify_case(vc)
        e = vc["expected"]
        for z in (d_f32(Z), d_bf16(synth.f32_to_bf16_bits(Z))):
            acc, out, cnt = gpu_verify(z, dr, dl)
            assert acc[0] == e["accept_len"] and list(out[0]) == e["out_tokens"], vc["name"]
            assert cnt[0] == e["out_count"], vc["name"]


def test_golden_fig3_on_gpu():
    say("golden fig3")
    fx, toks, lens, H, _ = golden_cases.load("fig3_newline.json")
    bits = synth.f32_to_bf16_bits(_pad8(H))
    for key, (a, b) in (("n1", (1, 1)), ("n1to3", (1, 3)), ("n1to4", (1, 4)), ("n5to6", (5, 6)),
                        ("n7to8", (7, 8))):
        e = fx["expected"][key]
        cp, cc, nu = gpu_find(toks, lens, a, b)
        assert list(cp[0, :cc[0]]) == e["cand_pos"] and nu[0] == e["ngram_used"], key
        sc, bp, bs = gpu_rank_hidden(d_bf16(bits), lens, cp, cc)
        assert bp[0] == e["best_pos"], key


# ------------------------------------------------------------------- find
FIND_CASES = [
    # (B, tok_stride, V, n_min, n_max, seed)
    (16, 1, 2, 1, 1, 0), (16, 5, 2, 1, 2, 1), (16, 64, 3, 1, 3, 2), (16, 700, 5, 1, 4, 3),
    (12, 4096, 50, 1, 3, 4), (8, 8192, 7, 2, 5, 5), (8, 8192, 1, 1, 8, 6),
    (6, 8193, 4, 1, 1, 7), (5, 12000, 30, 1, 3, 12), (6, 16384, 2, 1, 4, 13),
    (4, 16384, 1, 1, 1, 14), (4, 16385, 3, 1, 2, 15),
    (5, 20000, 3, 1, 3, 8), (4, 70000, 1000, 1, 2, 9),
    (3, 131072, 2, 8, 8, 10), (3, 50000, 1, 1, 1, 11),
    # 256 tiles: each compaction block sums the tile counts; 257 and more: the scan launch
    (3, 524288, 3, 1, 3, 16), (3, 524289, 3, 1, 3, 17), (4, 2000003, 2, 1, 8, 18),
    (3, 1048576, 5000, 1, 2, 19),
]


@pytest.mark.parametrize("case", FIND_CASES, ids=[f"B{c[0]}_S{c[1]}_V{c[2]}_n{c[3]}-{c[4]}"
                                                  for c in FIND_CASES])
def test_find_parity(case):
    B, stride, V, nmin, nmax, seed = case
    say("find", case)
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, V, size=(B, stride)).astype(np.int32)
    lens = rng.integers(1, stride + 1, size=B).astype(np.int32)
    lens[0] = stride                               # full length
    if B > 2:
        lens[1] = 0                                # invalid: too short
        lens[2] = stride + 1                       # invalid: too long
    if B > 3:
        lens[3] = min(stride, 3)
    ref = oracle.find(toks, lens, nmin, nmax)
    check_find(gpu_find(toks, lens, nmin, nmax), ref, str(case))
    # a larger cap leaves the same prefix
    check_find(gpu_find(toks, lens, nmin, nmax, cap=stride + 37), ref, str(case) + " cap")


@pytest.mark.parametrize("stride", [8192, 16384, 20000])
def test_find_lane31_hits(stride):
    """Sparse hits at positions 31 mod 64 (plus lane 63 once): a 64-position
    ballot with bit 31 set and the upper half otherwise empty must not widen
    into the upper lanes.  Both the one-block path and the tiled path, and the
    one-call drafting with one block and with split positions."""
    say("find lane 31", stride)
    B = 2
    toks = (np.arange(B * stride, dtype=np.int64).reshape(B, stride) % 1000003 + 10).astype(np.int32)
    lens = np.array([stride, stride - 5], np.int32)
    for b in range(B):
        T = lens[b]
        toks[b, T - 1] = 7
        toks[b, 31:T - 1:64] = 7
        toks[b, 63] = 7
    ref = oracle.find(toks, lens, 1, 1)
    assert ref[1][0] > 100
    check_find(gpu_find(toks, lens, 1, 1), ref, f"lane31 {stride}")
    if True:
        i32 = dict(dtype=torch.int32, device="cuda")
        K = 4
        A = synth.make_attn(B, 3, stride, lens, seed=5)
        for split in ((1, 5) if stride <= pld.DRAFT_MAX_TOK_STRIDE else (3, 40)):
            o = [torch.full((B, stride), -1, **i32), torch.zeros(B, **i32), torch.zeros(B, **i32),
                 torch.zeros(B, **i32), torch.zeros(B, dtype=torch.float32, device="cuda"),
                 torch.zeros((B, K), **i32), torch.zeros(B, **i32)]
            pld.pld_draft_attn(d_i32(toks), d_i32(lens), 1, 1, d_f32(A), K, *o,
                               blocks_per_seq=split, workspace=draft_workspace(B, split))
            torch.cuda.synchronize()
            check_find((o[0].cpu().numpy(), o[1].cpu().numpy(), o[2].cpu().numpy()), ref,
                       f"lane31 draft split {split}")


def test_find_random_shapes():
    """Seeded random shapes of the candidate search alone -- ragged lengths (1 to
    the stride), strides on both sides of the one-block and tiled limits and up to
    131072, n-gram ranges up to 8, small vocabularies (dense hits) and periodic
    rows (every position a long match) -- against the oracle's occurrence lists,
    counts and n used, bit for bit."""
    rng, n_cases = random_plan(31, 40)
    for it in range(n_cases):
        B = int(rng.integers(1, 13))
        stride = int(rng.choice([1, 2, 63, 64, 65, 4095, 8191, 8192, 8193, 16383, 16384,
                                 16385, 20000, 65536, 131072]))
        while B * stride > 1 << 20:
            B = max(1, B // 2)
        V = int(rng.choice([1, 2, 3, 17, 1000]))
        nmin = int(rng.integers(1, 5))
        nmax = int(rng.integers(nmin, 9))
        what = f"case {it}: B{B} S{stride} V{V} n{nmin}-{nmax}"
        say("find random", what)
        if rng.integers(0, 4) == 0:   # periodic rows
            period = int(rng.integers(1, 6))
            toks = np.tile((np.arange(stride) % period).astype(np.int32), (B, 1))
        else:
            toks = rng.integers(0, V, size=(B, stride)).astype(np.int32)
        lens = rng.integers(1, stride + 1, size=B).astype(np.int32)
        lens[0] = stride
        check_find(gpu_find(toks, lens, nmin, nmax), oracle.find(toks, lens, nmin, nmax), what)


def test_find_and_emit_at_the_largest_stride():
    """tok_stride = 2^30, the largest the calls accept (positions are int32): two
    sequences, 2^31 tokens (8 GiB) in all, occurrences planted at the start, the
    middle and the end of each row, so the tiled search (524288 tiles per row,
    offsets from the scan launch) and the draft of the last occurrence, which
    reaches the context end, run at the far end of the index ranges.  Only the
    listed prefix of the outputs is copied back."""
    import torch
    S = 1 << 30
    say("find at the largest stride", S)
    toks = np.zeros((2, S), np.int32)
    lens = np.array([S, S - 11], np.int32)
    # sequence 0: the query 2-gram (5, 7) ends at 1, 2^29 + 3 and T - 3; lone 7s elsewhere
    for j in (1, (1 << 29) + 3, S - 3, S - 1):
        toks[0, j - 1], toks[0, j] = 5, 7
    toks[0, [100, S - 100]] = 7
    # sequence 1: the last token 9 follows a 0, as do its earlier copies
    T1 = int(lens[1])
    toks[1, [12345, 1 << 28, T1 - 20, T1 - 1]] = 9
    cp_ref, cc_ref, nu_ref = oracle.find(toks, lens, 1, 2)
    assert list(cc_ref) == [3, 3] and list(nu_ref) == [2, 2]
    K = 8
    best = np.array([cp_ref[0, 2], cp_ref[1, 2]], np.int32)   # the last occurrence of each
    dr_ref, dl_ref = oracle.emit(toks, lens, best, K)
    say("oracle done; copying the tokens")
    t = torch.from_numpy(toks).to(dev())
    del toks
    l = d_i32(lens)
    cp = torch.full((2, S), -1, dtype=torch.int32, device=dev())
    cc = torch.full((2,), -7, dtype=torch.int32, device=dev())
    nu = torch.full((2,), -7, dtype=torch.int32, device=dev())
    pld.pld_find_candidates(t, l, 1, 2, cp, cc, nu, scratch(2, S))
    dr = torch.full((2, K), -7, dtype=torch.int32, device=dev())
    dl = torch.full((2,), -7, dtype=torch.int32, device=dev())
    pld.pld_emit_draft(t, l, d_i32(best), K, dr, dl)
    torch.cuda.synchronize()
    assert list(cc.cpu().numpy()) == [3, 3] and list(nu.cpu().numpy()) == [2, 2]
    assert np.array_equal(cp[:, :3].cpu().numpy(), cp_ref[:, :3])
    assert np.array_equal(dr.cpu().numpy(), dr_ref) and np.array_equal(dl.cpu().numpy(), dl_ref)
    assert list(dl_ref) == [2, 8]


@pytest.mark.parametrize("stride", [8192, 16384])
def test_find_group_and_wave_borders(stride):
    """The one-block search takes 64 positions per compare mask and a run of
    groups per wave (8 groups of 64 for rows up to 8192 tokens, 16 up to
    16384): occurrences of 1- to 8-grams planted so that their windows end on
    either side of every group border of the first waves and of every wave
    border, with the length ending inside, on and past a group; the find call
    and the one-call drafting with one block against the oracle, bit for bit."""
    say("find group/wave borders", stride)
    rng = np.random.default_rng(stride)
    per_wave = stride // 16
    B = 4
    toks = rng.integers(1000, 30000, size=(B, stride)).astype(np.int32)
    lens = np.array([stride, stride - 1, stride - 63, stride - 64 - 17], np.int32)
    ends = set()
    for g in range(1, 3 * per_wave // 64):
        ends.update((64 * g - 1, 64 * g))
    for w in range(1, 16):
        ends.update((w * per_wave - 1, w * per_wave, w * per_wave + 7))
    for b in range(B):
        T = int(lens[b])
        q = toks[b, T - 8:T].copy()
        for e in sorted(ends):
            if 8 <= e <= T - 9:
                n = 1 + (e % 8)                  # a window of n tokens ending at e
                toks[b, e - n + 1:e + 1] = q[8 - n:]
    for nmin, nmax in ((1, 1), (1, 8), (3, 5), (8, 8)):
        ref = oracle.find(toks, lens, nmin, nmax)
        check_find(gpu_find(toks, lens, nmin, nmax), ref, f"borders {stride} n{nmin}-{nmax}")
        if stride <= pld.DRAFT_MAX_TOK_STRIDE:
            i32 = dict(dtype=torch.int32, device="cuda")
            K = 4
            A = synth.make_attn(B, 2, stride, lens, seed=3)
            o = [torch.full((B, stride), -1, **i32), torch.zeros(B, **i32), torch.zeros(B, **i32),
                 torch.zeros(B, **i32), torch.zeros(B, dtype=torch.float32, device="cuda"),
                 torch.zeros((B, K), **i32), torch.zeros(B, **i32)]
            pld.pld_draft_attn(d_i32(toks), d_i32(lens), nmin, nmax, d_f32(A), K, *o,
                               blocks_per_seq=1, workspace=draft_workspace(B, 1))
            torch.cuda.synchronize()
            check_find((o[0].cpu().numpy(), o[1].cpu().numpy(), o[2].cpu().numpy()), ref,
                       f"borders draft {stride} n{nmin}-{nmax}")


def test_find_planted_ngrams_multi_tile():
    """Long sequences with planted n-gram repeats crossing tile borders."""
    say("find planted multi-tile")
    rng = np.random.default_rng(42)
    B, stride = 3, 40000
    toks = rng.integers(0, 30000, size=(B, stride)).astype(np.int32)
    lens = np.array([40000, 39999, 12345], np.int32)
    for b in range(B):
        T = lens[b]
        q = toks[b, T - 5:T].copy()
        for p in (2046, 2047, 2048, 4095, 10000, T - 7):   # around tile borders of 2048
            toks[b, p - 4:p + 1] = q
    for nmin, nmax in ((1, 5), (1, 8), (3, 3), (6, 8)):
        check_find(gpu_find(toks, lens, nmin, nmax), oracle.find(toks, lens, nmin, nmax))


# ------------------------------------------------------------- rank hidden
def _hidden_case(B, T, d, V, seed, nmin=1, nmax=1, plants=(), row_pad=0):
    rng = np.random.default_rng(seed)
    toks = rng.integers(0, V, size=(B, T)).astype(np.int32)
    lens = rng.integers(3, T + 1, size=B).astype(np.int32)
    lens[0] = T
    H = rng.standard_normal((B, T, d + row_pad)).astype(np.float32)
    for (b, dst, src) in plants:
        H[b, dst] = H[b, src]
    bits = synth.f32_to_bf16_bits(H)
    cp, cc, nu = oracle.find(toks, lens, nmin, nmax)
    return toks, lens, bits, cp, cc


@pytest.mark.parametrize("d", [8, 40, 512, 520, 4096, 5120, 8192, 16384])
def test_rank_hidden_parity(d):
    say("rank_hidden d", d)
    B, T = 6, 300
    toks, lens, bits, cp, cc = _hidden_case(B, T, d, 12, d)
    rsc, rbp, rbs = oracle.rank_hidden(bits, lens, cp, cc)
    gsc, gbp, gbs = gpu_rank_hidden(d_bf16(bits), lens, cp, cc)
    check_scores(gsc, rsc, cc, f"d={d}")
    flips = check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, f"d={d}")
    say("near-tie flips", flips)


def test_rank_at_the_largest_batch_and_width():
    """B = PLD_MAX_BATCH sequences with hidden rows of the largest width
    (PLD_MAX_HIDDEN): every ranking block holds the per-sequence prefix of all
    4096 lists and a 32 KB query row in LDS at once.  Short rows over a
    3-token vocabulary give 0 to 5 occurrences per sequence, empty lists
    included; both rankings and both in one launch, against the oracle."""
    B, T, d, R = pld.PLD_MAX_BATCH, 8, pld.PLD_MAX_HIDDEN, 5
    say("rank at the largest batch and width", B, d)
    rng = np.random.default_rng(4096)
    toks = rng.integers(0, 3, size=(B, T)).astype(np.int32)
    lens = rng.integers(1, T + 1, size=B).astype(np.int32)
    bits = synth.f32_to_bf16_bits(rng.standard_normal((B, T, d), dtype=np.float32))
    attn = rng.random((B, R, T), dtype=np.float32)
    cp, cc, nu = oracle.find(toks, lens, 1, 1)
    assert (cc == 0).any() and cc.max() >= 5
    hd, ad = d_bf16(bits), d_f32(attn)
    rsc, rbp, rbs = oracle.rank_hidden(bits, lens, cp, cc)
    gsc, gbp, gbs = gpu_rank_hidden(hd, lens, cp, cc)
    check_scores(gsc, rsc, cc, "largest batch and width")
    flips = check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, "largest batch and width")
    asc, abp, abs_ = oracle.rank_attn(attn, lens, cp, cc, oracle.AGG_SUM)
    gasc, gabp, gabs = gpu_rank_attn(ad, lens, cp, cc, pld.PLD_AGG_SUM)
    check_scores(gasc, asc, cc, "largest batch, attention")
    flips += check_best(gabp, gabs, asc, abp, abs_, cp, cc, "largest batch, attention")
    # both scorings in one launch: the same scores bit for bit, the same keys
    wh, wa = workspace(B, 1), workspace(B, 1)
    sh = torch.zeros((B, T), dtype=torch.float32, device=dev())
    sa = torch.zeros((B, T), dtype=torch.float32, device=dev())
    dl, dcp, dcc = d_i32(lens), d_i32(cp), d_i32(cc)
    pld.pld_score_both(hd, ad, dl, dcp, dcc, wh, wa, agg=pld.PLD_AGG_SUM, scores_h=sh, scores_a=sa)
    bp = torch.full((2, B), -7, dtype=torch.int32, device=dev())
    bs = torch.zeros((2, B), dtype=torch.float32, device=dev())
    pld.pld_select_best(B, bp[0], bs[0], wh)
    pld.pld_select_best(B, bp[1], bs[1], wa)
    torch.cuda.synchronize()
    assert_ws_zero(wh)
    assert_ws_zero(wa)
    both_h, both_a = sh.cpu().numpy(), sa.cpu().numpy()
    for b in range(B):
        n = int(cc[b])
        assert np.array_equal(both_h[b, :n].view(np.uint32), gsc[b, :n].view(np.uint32)), b
        assert np.array_equal(both_a[b, :n].view(np.uint32), gasc[b, :n].view(np.uint32)), b
    assert np.array_equal(bp[0].cpu().numpy(), gbp) and np.array_equal(bp[1].cpu().numpy(), gabp)
    say("near-tie flips", flips)


def test_rank_hidden_strided_rows_and_threshold():
    say("rank_hidden strided")
    B, T, d, pad = 4, 200, 256, 24
    toks, lens, bits, cp, cc = _hidden_case(B, T, d, 9, 3, row_pad=pad)
    hd = d_bf16(bits)[:, :, :d]                    # row stride d + pad
    assert hd.stride(1) == d + pad
    rsc, rbp, rbs = oracle.rank_hidden(np.ascontiguousarray(bits[:, :, :d]), lens, cp, cc)
    gsc, gbp, gbs = gpu_rank_hidden(hd, lens, cp, cc)
    check_scores(gsc, rsc, cc, "strided")
    check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, "strided")
    for th in (0.0, 0.05, float(np.nanmax(rsc[0, :cc[0]])), 2.0):
        rsc2, rbp2, rbs2 = oracle.rank_hidden(np.ascontiguousarray(bits[:, :, :d]), lens, cp, cc,
                                              threshold=th)
        gsc2, gbp2, gbs2 = gpu_rank_hidden(hd, lens, cp, cc, threshold=th)
        check_best(gbp2, gbs2, rsc2, rbp2, rbs2, cp, cc, f"threshold {th}", threshold=th)


def test_rank_hidden_exact_ties_and_planted_copy():
    """Identical and power-of-two-scaled rows tie bit-exactly on the GPU (the later j
    wins); a copy of the query row scores exactly 1."""
    say("rank_hidden ties")
    T, d = 64, 1024
    rng = np.random.default_rng(5)
    H = rng.standard_normal((2, T, d)).astype(np.float32)
    H[0, 9] = H[0, 19]
    H[0, 39] = 4.0 * H[0, 19]
    H[0, T - 2] = H[0, 19] + 0.05 * rng.standard_normal(d).astype(np.float32)
    H[1, 30] = H[1, T - 2]
    bits = synth.f32_to_bf16_bits(H)
    lens = np.array([T, T], np.int32)
    cp = np.full((2, T), -1, np.int32)
    cp[0, :4] = [10, 20, 40, 50]
    cp[1, :3] = [5, 31, 60]
    cc = np.array([4, 3], np.int32)
    gsc, gbp, gbs = gpu_rank_hidden(d_bf16(bits), lens, cp, cc)
    assert gsc[0, 0] == gsc[0, 1] == gsc[0, 2]
    assert gbp[0] == 40
    assert gsc[1, 1] == 1.0 and gbp[1] == 31 and gbs[1] == 1.0
    # the same row in another slot and another block gives the same bits
    cp2 = np.full((2, T), -1, np.int32)
    cp2[0, :3] = [40, 20, 10]
    gsc2, _, _ = gpu_rank_hidden(d_bf16(bits), lens, cp2, np.array([3, 0], np.int32))
    assert gsc2[0, 0] == gsc[0, 2] and gsc2[0, 2] == gsc[0, 0]


def test_rank_hidden_invalid_inputs():
    """Out-of-range candidates score NaN, bad counts count as zero, unusable
    sequences have no best; nothing outside the buffers is read."""
    say("rank_hidden invalid")
    B, T, d = 5, 40, 64
    rng = np.random.default_rng(8)
    bits = synth.f32_to_bf16_bits(rng.standard_normal((B, T, d)).astype(np.float32))
    lens = np.array([40, 1, 41, 40, 40], np.int32)    # seq 1 too short, seq 2 row T-2 = 39 ok
    lens[2] = 42                                       # T-2 = 40 >= n_rows: unusable
    cp = np.full((B, T), -1, np.int32)
    cp[0, :5] = [0, 1, 38, 39, 100]
    cp[1, :1] = [1]
    cp[2, :2] = [3, 4]
    cp[3, :2] = [5, 6]
    cp[4, :1] = [7]
    cc = np.array([5, 1, 2, T + 1, -3], np.int32)       # seq 3 count > cap, seq 4 negative
    rsc, rbp, rbs = oracle.rank_hidden(bits, lens, cp, cc)
    gsc, gbp, gbs = gpu_rank_hidden(d_bf16(bits), lens, cp, cc)
    check_scores(gsc, rsc, np.array([5, 1, 2, 0, 0]), "invalid")
    assert list(gbp) == list(rbp) and list(gbp[1:]) == [-1, -1, -1, -1]
    assert math.isnan(gsc[0, 0]) and math.isnan(gsc[0, 3]) and math.isnan(gsc[0, 4])


def test_rank_hidden_many_sequences_and_empty():
    """A batch where most sequences have no candidate and one has thousands."""
    say("rank_hidden skewed batch")
    B, T, d = 40, 4000, 128
    rng = np.random.default_rng(11)
    toks = rng.integers(0, 100000, size=(B, T)).astype(np.int32)
    toks[7] = rng.integers(0, 2, size=T)
    lens = np.full(B, T, np.int32)
    H = synth.f32_to_bf16_bits(rng.standard_normal((B, T, d)).astype(np.float32))
    cp, cc, nu = oracle.find(toks, lens, 1, 1)
    assert cc[7] > 1000 and (cc == 0).sum() > 20
    rsc, rbp, rbs = oracle.rank_hidden(H, lens, cp, cc)
    gsc, gbp, gbs = gpu_rank_hidden(d_bf16(H), lens, cp, cc)
    check_scores(gsc, rsc, cc, "skewed")
    check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, "skewed")


# --------------------------------------------------------------- rank attn
@pytest.mark.parametrize("R,agg", [(1, 0), (7, 0), (40, 0), (64, 1), (9, 1)])
def test_rank_attn_parity(R, agg):
    say("rank_attn", R, agg)
    B, T = 7, 900
    rng = np.random.default_rng(R * 10 + agg)
    toks = rng.integers(0, 15, size=(B, T)).astype(np.int32)
    lens = rng.integers(2, T + 1, size=B).astype(np.int32)
    lens[0] = T
    lens[1] = 1
    A = synth.make_attn(B, R, T, lens, seed=R)
    cp, cc, nu = oracle.find(toks, lens, 1, 1)
    rsc, rbp, rbs = oracle.rank_attn(A, lens, cp, cc, agg)
    gsc, gbp, gbs = gpu_rank_attn(d_f32(A), lens, cp, cc, agg)
    check_scores(gsc, rsc, cc, f"attn R={R}")
    check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, f"attn R={R}")


def test_rank_random_shapes():
    """Seeded random shapes of the separate ranking calls against the oracle --
    hidden (bf16, d from 8 to 8192, padded rows) and attention (SUM or MAX over 1 to
    70 rows, padded keys), ragged lengths, dense or sparse candidates, thresholds --
    scores within the stated tolerance, the choice bit for bit or a counted near tie."""
    rng, n_cases = random_plan(57, 30)
    flips = 0
    for it in range(n_cases):
        B = int(rng.integers(1, 9))
        T = int(rng.choice([2, 3, 70, 1000, 5000]))
        V = int(rng.choice([1, 3, 40, 5000]))
        hidden = bool(rng.integers(0, 2))
        th = float(rng.choice([-math.inf, 0.0, 0.2]))
        toks = rng.integers(0, V, size=(B, T)).astype(np.int32)
        lens = rng.integers(1, T + 1, size=B).astype(np.int32)
        lens[0] = T
        cp, cc, _ = oracle.find(toks, lens, 1, 1)
        if hidden:
            d = int(rng.choice([8, 64, 520, 4096, 8192]))
            while B * T * d > 2e7 and d > 8:
                d = {8192: 520, 4096: 520, 520: 64, 64: 8}[d]
            pad = int(rng.choice([0, 8]))
            what = f"case {it}: hidden B{B} T{T} V{V} d{d} pad{pad} th{th}"
            say("rank random", what)
            H = rng.standard_normal((B, T, d + pad)).astype(np.float32)
            bits = synth.f32_to_bf16_bits(H)
            rsc, rbp, rbs = oracle.rank_hidden(bits[:, :, :d], lens, cp, cc, threshold=th)
            gsc, gbp, gbs = gpu_rank_hidden(d_bf16(bits)[:, :, :d], lens, cp, cc, threshold=th)
        else:
            R = int(rng.integers(1, 71))
            agg = int(rng.integers(0, 2))
            pad = int(rng.choice([0, 5]))
            what = f"case {it}: attn B{B} T{T} V{V} R{R} agg{agg} pad{pad} th{th}"
            say("rank random", what)
            A = rng.random((B, R, T + pad)).astype(np.float32)
            A /= A.sum(axis=2, keepdims=True)
            rsc, rbp, rbs = oracle.rank_attn(A[:, :, :T], lens, cp, cc, agg, threshold=th)
            gsc, gbp, gbs = gpu_rank_attn(d_f32(A)[:, :, :T], lens, cp, cc, agg, threshold=th)
        check_scores(gsc, rsc, cc, what)
        flips += check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, what, threshold=th)
    say("rank random: near-tie flips", flips)


def test_score_both_equals_separate_calls():
    """pld_score_both against pld_score_hidden + pld_score_attn on the same
    candidate lists, over seeded random shapes (d on each hidden path: 8, 520,
    4096, 8192; 1 to 70 attention rows, SUM or MAX; ragged and empty sequences;
    each ranking's own threshold): scores and choices bit for bit, both
    workspaces left zero, and the choices against the oracle."""
    rng, n_cases = random_plan(83, 16)
    flips = 0
    for it in range(n_cases):
        B = int(rng.choice([1, 3, 8, 64]))
        T = int(rng.choice([2, 70, 1000, 3000]))
        V = int(rng.choice([3, 40, 5000]))
        d = int(rng.choice([8, 520, 4096, 8192]))
        while B * T * d > 2e7 and d > 8:
            d = {8192: 4096, 4096: 520, 520: 8}[d]
        R = int(rng.integers(1, 71))
        agg = int(rng.integers(0, 2))
        th_h = float(rng.choice([-math.inf, 0.0, 2.0]))
        th_a = float(rng.choice([-math.inf, 0.001, 2.0]))
        what = f"case {it}: B{B} T{T} V{V} d{d} R{R} agg{agg} th{th_h}/{th_a}"
        say("score both", what)
        toks = rng.integers(0, V, size=(B, T)).astype(np.int32)
        lens = rng.integers(1, T + 1, size=B).astype(np.int32)
        lens[0] = T
        if B > 2:
            lens[1] = 1                               # no candidates
        cp, cc, _ = oracle.find(toks, lens, 1, 1)
        bits = synth.f32_to_bf16_bits(rng.standard_normal((B, T, d)).astype(np.float32))
        A = rng.random((B, R, T)).astype(np.float32)
        A /= A.sum(axis=2, keepdims=True)
        hd, ad, ld, cpd, ccd = d_bf16(bits), d_f32(A), d_i32(lens), d_i32(cp), d_i32(cc)
        out = {}
        for how in ("separate", "both"):
            ws = [workspace(B, 1), workspace(B, 1)]
            sc = [torch.full(cp.shape, 12345.0, dtype=torch.float32, device=dev()) for _ in ws]
            if how == "separate":
                pld.pld_score_hidden(hd, ld, cpd, ccd, ws[0], threshold=th_h, scores=sc[0])
                pld.pld_score_attn(ad, ld, cpd, ccd, ws[1], agg=agg, threshold=th_a,
                                   scores=sc[1])
            else:
                pld.pld_score_both(hd, ad, ld, cpd, ccd, ws[0], ws[1], agg=agg,
                                   threshold_h=th_h, threshold_a=th_a, scores_h=sc[0],
                                   scores_a=sc[1])
            res = []
            for w_, s_ in zip(ws, sc):
                bp = torch.full((B,), -7, dtype=torch.int32, device=dev())
                bs = torch.zeros(B, dtype=torch.float32, device=dev())
                pld.pld_select_best(B, bp, bs, w_)
                res.append((s_.cpu().numpy(), bp.cpu().numpy(), bs.cpu().numpy()))
            torch.cuda.synchronize()
            for w_ in ws:
                assert_ws_zero(w_)
            out[how] = res
        for (a_sc, a_bp, a_bs), (b_sc, b_bp, b_bs) in zip(out["separate"], out["both"]):
            assert np.array_equal(a_sc, b_sc, equal_nan=True), what
            assert np.array_equal(a_bp, b_bp) and np.array_equal(a_bs, b_bs), what
        ref_h = oracle.rank_hidden(bits, lens, cp, cc, threshold=th_h)
        ref_a = oracle.rank_attn(A, lens, cp, cc, agg, threshold=th_a)
        for (g_sc, g_bp, g_bs), (r_sc, r_bp, r_bs), name in zip(out["both"], (ref_h, ref_a),
                                                               ("hidden", "attn")):
            check_scores(g_sc, r_sc, cc, what + " " + name)
            flips += check_best(g_bp, g_bs, r_sc, r_bp, r_bs, cp, cc, what + " " + name,
                                threshold=th_h if name == "hidden" else th_a)
        del hd, ad
        torch.cuda.empty_cache()
    say("score both: near-tie flips", flips)


def test_rank_attn_strided_keys_and_ties():
    say("rank_attn strided/ties")
    B, R, T, pad = 3, 5, 120, 13
    A = np.zeros((B, R, T + pad), np.float32)
    A[0, :, 9] = 0.25        # j = 10
    A[0, :, 49] = 0.25       # j = 50 ties with j = 10 -> 50 wins
    A[1, 2, 70] = 1.0
    A[2, :, 5] = 0.5
    lens = np.array([T, T, T], np.int32)
    cp = np.full((B, T), -1, np.int32)
    cp[0, :3] = [10, 30, 50]
    cp[1, :3] = [10, 71, 119]          # 119 > T-2: unusable
    cp[2, :2] = [6, 7]
    cc = np.array([3, 3, 2], np.int32)
    ad = d_f32(A)[:, :, :T]
    for agg in (0, 1):
        rsc, rbp, rbs = oracle.rank_attn(np.ascontiguousarray(A[:, :, :T]), lens, cp, cc, agg)
        gsc, gbp, gbs = gpu_rank_attn(ad, lens, cp, cc, agg)
        check_scores(gsc, rsc, cc)
        assert list(gbp) == list(rbp) == [50, 71, 6]


# ------------------------------------------------------------------- emit
def test_emit_parity():
    say("emit")
    rng = np.random.default_rng(3)
    B, stride = 64, 50
    toks = rng.integers(0, 1000, size=(B, stride)).astype(np.int32)
    lens = rng.integers(0, stride + 2, size=B).astype(np.int32)
    best = np.array([rng.integers(-2, stride + 1) for _ in range(B)], np.int32)
    best[:4] = [-1, 0, 48, 49]
    lens[:4] = [50, 50, 50, 50]
    for K in (1, 5, 16, 64):
        rd, rl = oracle.emit(toks, lens, best, K)
        gd, gl = gpu_emit(toks, lens, best, K)
        assert np.array_equal(gd, rd) and np.array_equal(gl, rl), K


# ------------------------------------------------- selection + draft, one launch
def _order_key(score, j):
    """The ranking key (orderable fp32 score << 32 | j) written on the host."""
    u = int(np.array([score], np.float32).view(np.uint32)[0])
    if u == 0x80000000:
        u = 0
    o = (~u & 0xffffffff) if u & 0x80000000 else (u | 0x80000000)
    return (o << 32) | (int(j) & 0xffffffff)


def _key_slots(rng, B, stride, empty_every):
    """Random key slots [B][16]: some sequences with no key at all, equal scores at
    different positions, signed zeros, positions past the context."""
    keys = np.zeros((B, 16), np.uint64)
    for b in range(B):
        if b % empty_every == 0:
            continue
        for k in range(16):
            if rng.random() < 0.3:
                continue
            s = float(rng.choice([rng.normal(), 0.5, -0.0, 0.0, -2.0]))
            j = int(rng.integers(1, stride + 3))
            keys[b, k] = _order_key(s, j)
    return keys


def _decode(keys):
    """best_pos / best_score of each sequence from its slots, decoded on the host."""
    best = keys.max(axis=1)
    pos = np.where(best == 0, -1, (best & np.uint64(0xffffffff)).astype(np.int64)).astype(np.int32)
    o = (best >> np.uint64(32)).astype(np.uint32)
    u = np.where(o & 0x80000000, o & 0x7fffffff, ~o).astype(np.uint32)
    sc = np.where(best == 0, -np.inf, u.view(np.float32)).astype(np.float32)
    return pos, sc


@pytest.mark.parametrize("K", [1, 16, 70])
def test_select_draft_parity(K):
    """pld_select_draft: the choice from the key slots and the draft equal the
    host-decoded keys and the oracle's emit, with and without a second ranking's
    keys, and both workspaces are left zero; the same outputs as pld_select_best
    followed by pld_emit_draft, bit for bit."""
    say("select_draft", K)
    rng = np.random.default_rng(100 + K)
    B, stride = 70, 90
    toks = rng.integers(0, 500, size=(B, stride)).astype(np.int32)
    lens = rng.integers(1, stride + 1, size=B).astype(np.int32)
    lens[:5] = [0, -3, stride + 1, 1, 2]          # invalid lengths, then the shortest
    keys = _key_slots(rng, B, stride, 7)
    aux = _key_slots(rng, B, stride, 5)
    want_pos, want_sc = _decode(keys)
    aux_pos, aux_sc = _decode(aux)
    rd, rl = oracle.emit(toks, lens, want_pos, K)
    td, ld = d_i32(toks), d_i32(lens)
    for with_aux in (False, True):
        ws = workspace(B, K)
        ws[:B * 128] = torch.from_numpy(keys.view(np.uint8).reshape(-1)).to(dev())
        ws2 = workspace(B, K) if with_aux else None
        if with_aux:
            ws2[:B * 128] = torch.from_numpy(aux.view(np.uint8).reshape(-1)).to(dev())
        bp = torch.full((B,), -7, dtype=torch.int32, device=dev())
        bs = torch.zeros(B, dtype=torch.float32, device=dev())
        dr = torch.full((B, K), -7, dtype=torch.int32, device=dev())
        dl = torch.full((B,), -7, dtype=torch.int32, device=dev())
        abp = torch.full((B,), -7, dtype=torch.int32, device=dev())
        abs_ = torch.zeros(B, dtype=torch.float32, device=dev())
        pld.pld_select_draft(td, ld, K, bp, bs, dr, dl, ws, aux_workspace=ws2,
                             aux_best_pos=abp if with_aux else None,
                             aux_best_score=abs_ if with_aux else None)
        torch.cuda.synchronize()
        assert np.array_equal(bp.cpu().numpy(), want_pos)
        assert np.array_equal(bs.cpu().numpy().view(np.uint32), want_sc.view(np.uint32))
        assert np.array_equal(dr.cpu().numpy(), rd) and np.array_equal(dl.cpu().numpy(), rl)
        assert_ws_zero(ws)
        if with_aux:
            assert np.array_equal(abp.cpu().numpy(), aux_pos)
            assert np.array_equal(abs_.cpu().numpy().view(np.uint32), aux_sc.view(np.uint32))
            assert_ws_zero(ws2)
        else:
            assert (abp == -7).all()
    # the two separate calls from the same slots
    ws = workspace(B, K)
    ws[:B * 128] = torch.from_numpy(keys.view(np.uint8).reshape(-1)).to(dev())
    bp = torch.full((B,), -7, dtype=torch.int32, device=dev())
    bs = torch.zeros(B, dtype=torch.float32, device=dev())
    pld.pld_select_best(B, bp, bs, ws)
    dr = torch.full((B, K), -7, dtype=torch.int32, device=dev())
    dl = torch.full((B,), -7, dtype=torch.int32, device=dev())
    pld.pld_emit_draft(td, ld, bp, K, dr, dl)
    torch.cuda.synchronize()
    assert np.array_equal(bp.cpu().numpy(), want_pos)
    assert np.array_equal(dr.cpu().numpy(), rd) and np.array_equal(dl.cpu().numpy(), rl)


# ----------------------------------------------------------------- verify
VERIFY_CASES = [
    # (B, K, V, bf16, integer_valued, seed)
    (3, 4, 1, False, False, 0), (5, 6, 7, False, True, 1), (5, 6, 7, True, True, 2),
    (4, 10, 1001, False, False, 3), (4, 10, 1001, True, True, 4), (2, 3, 1000003, False, False, 5),
    (8, 10, 32000, False, False, 6), (6, 16, 128256, True, False, 7), (3, 32, 128256, False, True, 8),
]


@pytest.mark.parametrize("case", VERIFY_CASES, ids=[f"B{c[0]}_K{c[1]}_V{c[2]}_{'bf16' if c[3] else 'f32'}"
                                                    for c in VERIFY_CASES])
def test_verify_parity(case):
    B, K, V, bf16, integer, seed = case
    say("verify", case)
    rng = np.random.default_rng(seed)
    if integer:
        Z = rng.integers(-3, 4, size=(B, K + 1, V)).astype(np.float32)
        Z[rng.random(Z.shape) < 0.3] *= -1.0        # signed zeros
    else:
        Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    L = rng.integers(0, K + 1, size=B).astype(np.int32)
    draft = np.full((B, K), -1, np.int32)
    for b in range(B):
        draft[b, :L[b]] = rng.integers(0, V, size=L[b])
        p = rng.integers(0, L[b] + 1)
        for i in range(p):
            Z[b, i, draft[b, i]] = 10.0            # accepted prefix
    if B > 2:
        L[2] = K + 1                                # invalid draft length
    zbits = synth.f32_to_bf16_bits(Z) if bf16 else Z
    ref = oracle.verify(zbits, draft, L, bf16=bf16)
    zd = d_bf16(zbits) if bf16 else d_f32(Z)
    check_verify(gpu_verify(zd, draft, L), ref, str(case))


@pytest.mark.parametrize("bf16", [False, True])
def test_verify_at_the_largest_draft(bf16):
    """K + 1 = 65535 rows per sequence, the most the argmax launch's second grid
    dimension holds: a full acceptance (K + 1 tokens), a first mismatch deep in
    the rows, a draft accepted to its length, and an empty draft, against the
    oracle; the workspace is left zero."""
    B, K, V = 4, 65534, 5
    say("verify at the largest draft", K, "bf16" if bf16 else "f32")
    rng = np.random.default_rng(65534)
    Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
    L = np.array([K, K, 40000, 0], np.int32)
    for b, upto in ((0, K), (1, 50000), (2, 40000)):
        Z[b, np.arange(upto), draft[b, :upto]] = 10.0
    Z[1, 50000, draft[1, 50000]] = -10.0          # a sure mismatch at row 50000
    zbits = synth.f32_to_bf16_bits(Z) if bf16 else Z
    ref = oracle.verify(zbits, draft, L, bf16=bf16)
    assert list(ref[0]) == [K, 50000, 40000, 0] and ref[2][0] == K + 1
    got = gpu_verify(d_bf16(zbits) if bf16 else d_f32(Z), draft, L)
    check_verify(got, ref, f"K={K}")


def test_verify_random_shapes():
    """Seeded random shapes of greedy verification -- f32 and bf16 logits, integer
    rows with ties and signed zeros, draft lengths from -1 to K+1, planted accepted
    prefixes -- the one-call greedy verification, its halves and the acceptance fused
    with the commit, each against the oracle (accepted lengths and tokens bit for bit,
    the rows, lengths and counters of the commit too)."""
    rng, n_cases = random_plan(77, 40)
    i32 = dict(dtype=torch.int32, device="cuda")
    for it in range(n_cases):
        B = int(rng.integers(1, 17))
        K = int(rng.integers(1, 41))
        V = int(rng.choice([1, 3, 7, 1000, 32000, 50001]))
        bf16 = bool(rng.integers(0, 2))
        integer = bool(rng.integers(0, 2))
        what = f"case {it}: B{B} K{K} V{V} {'bf16' if bf16 else 'f32'} {'int' if integer else 'normal'}"
        say("verify random", what)
        if integer:
            Z = rng.integers(-2, 3, size=(B, K + 1, V)).astype(np.float32)
            Z[rng.random(Z.shape) < 0.3] *= -1.0
        else:
            Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
        L = rng.integers(-1, K + 2, size=B).astype(np.int32)
        draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
        for b in range(B):
            for i in range(int(rng.integers(0, K + 1))):
                Z[b, i, draft[b, i]] = 10.0
        zbits = synth.f32_to_bf16_bits(Z) if bf16 else Z
        ref = oracle.verify(zbits, draft, L, bf16=bf16)
        zd = d_bf16(zbits) if bf16 else d_f32(Z)
        check_verify(gpu_verify(zd, draft, L), ref, what)
        # the halves, then the acceptance fused with the commit
        ws = workspace(B, K)
        acc, out, cnt = (torch.full((B,), -7, **i32), torch.full((B, K + 1), -7, **i32),
                         torch.full((B,), -7, **i32))
        stride = int(rng.integers(1, 3 * (K + 1) + 2))
        toks = rng.integers(0, 100, size=(B, stride)).astype(np.int32)
        lens = rng.integers(-1, stride + 2, size=B).astype(np.int32)
        limit = rng.integers(0, stride + 1, size=B).astype(np.int32)
        td, ld = d_i32(toks), d_i32(lens)
        pld.pld_verify_argmax(zd, d_i32(L), ws)
        pld.pld_accept_commit(d_i32(draft), d_i32(L), acc, out, cnt, td, ld, ws, limit=d_i32(limit))
        torch.cuda.synchronize()
        assert int(torch.count_nonzero(ws).item()) == 0, what
        check_verify((acc.cpu().numpy(), out.cpu().numpy(), cnt.cpu().numpy()), ref, what)
        wt, wl, _ = oracle.commit(toks, lens, ref[1], ref[2], limit=limit)
        assert np.array_equal(td.cpu().numpy(), wt) and np.array_equal(ld.cpu().numpy(), wl), what


def test_verify_misaligned_row_views():
    """Rows that start off a 16-byte boundary (a view into a padded buffer)."""
    say("verify misaligned")
    rng = np.random.default_rng(9)
    B, K, V = 3, 5, 3001
    Z = rng.standard_normal((B, K + 1, V + 3)).astype(np.float32)
    draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
    L = np.array([5, 2, 0], np.int32)
    for off in (1, 2, 3):
        view = np.ascontiguousarray(Z[:, :, off:off + V])
        ref = oracle.verify(view, draft, L)
        zd = d_f32(Z)[:, :, off:off + V]
        check_verify(gpu_verify(zd, draft, L), ref, f"offset {off}")
        zb = synth.f32_to_bf16_bits(Z)
        refb = oracle.verify(np.ascontiguousarray(zb[:, :, off:off + V]), draft, L, bf16=True)
        check_verify(gpu_verify(d_bf16(zb)[:, :, off:off + V], draft, L), refb, f"bf16 offset {off}")


def test_verify_all_equal_rows_and_negative_infinity():
    say("verify degenerate rows")
    B, K, V = 2, 3, 777
    Z = np.full((B, K + 1, V), -np.inf, np.float32)
    Z[1] = 0.0
    Z[1, :, ::2] = -0.0
    draft = np.array([[0, 0, 0], [0, 0, 5]], np.int32)
    L = np.array([3, 3], np.int32)
    ref = oracle.verify(Z, draft, L)
    assert list(ref[0]) == [3, 2]
    check_verify(gpu_verify(d_f32(Z), draft, L), ref, "degenerate")


@pytest.mark.parametrize("B,K,V,bf16", [(200, 16, 5000, False), (1, 16, 128256, True),
                                         (3, 70, 32000, False)])
def test_verify_one_launch_repeated_calls(B, K, V, bf16):
    """Greedy verification on one workspace over calls in a row with changing
    draft lengths, invalid ones included, at 1 to over a hundred blocks per
    row: every call against the oracle and the workspace zero after each."""
    say("verify one launch", B, K, V, bf16)
    rng = np.random.default_rng(B * 1000 + K)
    ws = workspace(B, K)
    Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
    for b in range(B):   # accepted prefixes of every length
        for i in range(int(rng.integers(0, K + 1))):
            Z[b, i, draft[b, i]] = 10.0
    zbits = synth.f32_to_bf16_bits(Z) if bf16 else Z
    zd = d_bf16(zbits) if bf16 else d_f32(Z)
    for call in range(4):
        L = rng.integers(0, K + 1, size=B).astype(np.int32)
        if call == 1:
            L[:] = K
        if call == 2:
            L[0] = -1
            L[-1] = K + 1 if B > 1 else 0
        if call == 3:
            L[:] = 0
        ref = oracle.verify(zbits, draft, L, bf16=bf16)
        check_verify(gpu_verify(zd, draft, L, ws=ws), ref, f"call {call}")


def test_workspace_shared_across_calls_and_determinism():
    """One workspace serves every call in turn and is zero after each; repeated
    calls give bit-identical results."""
    say("shared workspace")
    cfg = synth.Config("t", 4, 3000, 500, 1.1, 0.3, (8, 32), (1, 2), 256, "hidden", 0, 8, "f32", 21)
    toks, lens, metas = synth.make_tokens(cfg)
    ws = workspace(cfg.B, cfg.K)
    H = synth.make_hidden(cfg.B, cfg.T, cfg.d, cfg.seed, device="cuda")
    runs = []
    for _ in range(3):
        cp, cc, nu = gpu_find(toks, lens, 1, 2)
        sc, bp, bs = gpu_rank_hidden(H, lens, cp, cc, ws=ws)
        runs.append((cp.copy(), cc.copy(), sc.copy(), bp.copy(), bs.copy()))
    for r in runs[1:]:
        for x, y in zip(r, runs[0]):
            assert np.array_equal(x, y, equal_nan=True)


# ------------------------------------------------------- one-call drafting
DRAFT_CASES = [
    # (B, tok_stride, V, n_min, n_max, d, R, K, seed)
    (9, 1, 3, 1, 1, 64, 0, 4, 0), (9, 50, 3, 1, 3, 64, 0, 4, 1), (12, 700, 6, 1, 4, 520, 0, 9, 2),
    (8, 4096, 40, 1, 3, 4096, 0, 10, 3), (5, 8192, 2, 2, 5, 128, 0, 16, 4),
    (9, 300, 4, 1, 2, 0, 7, 6, 5), (6, 8192, 20, 1, 1, 0, 40, 16, 6), (4, 5000, 1, 1, 3, 0, 3, 8, 7),
    # long contexts (split positions only) and a stride that is not a multiple of 4
    (3, 20000, 30, 1, 3, 256, 0, 8, 8), (3, 40000, 5, 1, 1, 0, 5, 8, 9),
    (4, 20001, 3, 2, 4, 64, 0, 5, 10),
    # more occurrences in one sequence than one compaction window (16384) holds
    (2, 40000, 1, 1, 1, 0, 3, 5, 11), (2, 36000, 2, 1, 1, 64, 0, 5, 12),
]
DRAFT_SPLITS = [1, 3, 64, 1000]


@pytest.mark.parametrize("split", DRAFT_SPLITS)
@pytest.mark.parametrize("case", DRAFT_CASES, ids=[f"B{c[0]}_S{c[1]}_V{c[2]}_n{c[3]}-{c[4]}_"
                                                   f"{'d' + str(c[5]) if c[5] else 'R' + str(c[6])}"
                                                   for c in DRAFT_CASES])
def test_draft_fused_parity(case, split):
    """The one-call drafting equals the oracle's find, rank and emit, and its
    scores are bit-identical to the separate ranking call, for any number of
    blocks per sequence the call accepts (and an error for those it rejects)."""
    B, stride, V, nmin, nmax, d, R, K, seed = case
    say("draft fused", case, "split", split)
    rng = np.random.default_rng(100 + seed)
    toks = rng.integers(0, V, size=(B, stride)).astype(np.int32)
    lens = rng.integers(1, stride + 1, size=B).astype(np.int32)
    lens[0] = stride
    if B > 2:
        lens[1] = 0
        lens[2] = stride + 1
    part = -(-(-(-stride // split)) // 8) * 8           # positions per block, split > 1
    accepted = (stride <= pld.DRAFT_MAX_TOK_STRIDE) if split == 1 else part <= pld.DRAFT_MAX_PART
    ref_find = oracle.find(toks, lens, nmin, nmax)
    cp, cc, nu = ref_find
    i32 = dict(dtype=torch.int32, device="cuda")
    ws = draft_workspace(B, split)
    o = dict(cand_pos=torch.full((B, stride), -1, **i32), cand_count=torch.zeros(B, **i32),
             ngram_used=torch.zeros(B, **i32), best_pos=torch.zeros(B, **i32),
             best_score=torch.zeros(B, dtype=torch.float32, device="cuda"),
             draft=torch.zeros((B, K), **i32), draft_len=torch.zeros(B, **i32),
             scores=torch.full((B, stride), 777.0, dtype=torch.float32, device="cuda"))
    for th in (-math.inf, 0.0):
        if d:
            bits = synth.f32_to_bf16_bits(rng.standard_normal((B, stride, d)).astype(np.float32))
            hd = d_bf16(bits)
            call = lambda: pld.pld_draft_hidden(
                d_i32(toks), d_i32(lens), nmin, nmax, hd, K, o["cand_pos"], o["cand_count"],
                o["ngram_used"], o["best_pos"], o["best_score"], o["draft"], o["draft_len"],
                threshold=th, scores=o["scores"], blocks_per_seq=split, workspace=ws)
            if not accepted:
                with pytest.raises(pld.PLDError):
                    call()
                return
            ref = oracle.rank_hidden(bits, lens, cp, cc, threshold=th)
            call()
            split_ref = gpu_rank_hidden(hd, lens, cp, cc, threshold=th)
        else:
            A = synth.make_attn(B, R, stride, lens, seed=seed)
            call = lambda: pld.pld_draft_attn(
                d_i32(toks), d_i32(lens), nmin, nmax, d_f32(A), K, o["cand_pos"], o["cand_count"],
                o["ngram_used"], o["best_pos"], o["best_score"], o["draft"], o["draft_len"],
                threshold=th, scores=o["scores"], blocks_per_seq=split, workspace=ws)
            if not accepted:
                with pytest.raises(pld.PLDError):
                    call()
                return
            ref = oracle.rank_attn(A, lens, cp, cc, oracle.AGG_SUM, threshold=th)
            call()
            split_ref = gpu_rank_attn(d_f32(A), lens, cp, cc, pld.PLD_AGG_SUM, threshold=th)
        torch.cuda.synchronize()
        g = {k: v.cpu().numpy() for k, v in o.items()}
        assert draft_keys_zero(ws, B)
        check_find((g["cand_pos"], g["cand_count"], g["ngram_used"]), ref_find, str(case))
        rsc, rbp, rbs = ref
        check_scores(g["scores"], rsc, cc, str(case))
        flips = check_best(g["best_pos"], g["best_score"], rsc, rbp, rbs, cp, cc, str(case),
                           threshold=th)
        for b in range(B):          # same bits as the separate ranking call
            n = cc[b]
            assert np.array_equal(g["scores"][b, :n], split_ref[0][b, :n], equal_nan=True)
        assert np.array_equal(g["best_pos"], split_ref[1])
        rd, rl = oracle.emit(toks, lens, g["best_pos"] if flips else rbp, K)
        assert np.array_equal(g["draft"], rd) and np.array_equal(g["draft_len"], rl)


@pytest.mark.parametrize("split", [64, 57, 240, 241, 1000])
def test_draft_finish_read_ahead_limits(split):
    """All-equal tokens make every position an occurrence.  4096 positions in
    64 parts of 64 entries fill the finishing kernel's read-ahead exactly, as
    do 240 parts (of 24; the most it covers); 57 parts of 72 hold more than it
    reads per part, and 241 or 1000 parts are more than it covers: these take
    the windowed compaction."""
    test_draft_fused_parity((2, 4096, 1, 1, 1, 64, 0, 6, 13), split)


def test_autotune_split_keeps_the_results():
    """DraftStep.autotune_split times a few blocks-per-sequence choices (8-wave
    blocks for small grids, 4-wave blocks for large ones) and keeps one; the
    drafting outputs are the same bits under every choice and equal the
    oracle's."""
    from paper_2412_01447_amd.step import DraftStep
    say("autotune split")
    B, stride, V, d, K = 3, 20000, 40, 64, 8
    rng = np.random.default_rng(77)
    toks = rng.integers(0, V, size=(B, stride)).astype(np.int32)
    lens = np.array([stride, stride - 3, 777], np.int32)
    bits = synth.f32_to_bf16_bits(rng.standard_normal((B, stride, d)).astype(np.float32))
    td, ld, hd = d_i32(toks), d_i32(lens), d_bf16(bits)
    step = DraftStep(B, stride, K, device="cuda", mode="fused")
    step.set_split(step.min_split())
    outs = []
    for S in (step.min_split(), 64, 200, 1000):   # 4-wave blocks where B*S > 512
        step.set_split(S)
        step.draft_fused(td, ld, hidden=hd)
        torch.cuda.synchronize()
        outs.append([t.clone() for t in (step.cand_pos, step.cand_count, step.best_pos,
                                         step.best_score, step.draft, step.draft_len)])
    chosen = step.autotune_split(lambda i: step.draft_fused(td, ld, hidden=hd),
                                 step.cand_count.cpu().numpy(), hidden=True, reps=2, trials=1)
    assert step.min_split() <= chosen <= pld.PLD_MAX_DRAFT_SPLIT and step.draft_split == chosen
    step.draft_fused(td, ld, hidden=hd)
    torch.cuda.synchronize()
    outs.append([t.clone() for t in (step.cand_pos, step.cand_count, step.best_pos,
                                     step.best_score, step.draft, step.draft_len)])
    cc = outs[0][1].cpu().numpy()
    for o in outs[1:]:
        assert np.array_equal(o[1].cpu().numpy(), cc)
        for b in range(B):
            assert torch.equal(o[0][b, :cc[b]], outs[0][0][b, :cc[b]])
        for x, y in zip(o[2:], outs[0][2:]):
            assert torch.equal(x, y)
    cp, rc, _ = oracle.find(toks, lens, 1, 1)
    assert np.array_equal(cc, rc)
    rsc, rbp, rbs = oracle.rank_hidden(bits, lens, cp, rc)
    flips = check_best(outs[0][2].cpu().numpy(), outs[0][3].cpu().numpy(), rsc, rbp, rbs, cp, rc,
                       "autotune")
    rd, rl = oracle.emit(toks, lens, outs[0][2].cpu().numpy() if flips else rbp, K)
    assert np.array_equal(outs[0][4].cpu().numpy(), rd)
    assert np.array_equal(outs[0][5].cpu().numpy(), rl)


def test_draft_random_shapes():
    """Seeded random shapes of the one-call drafting -- hidden (bf16, d up to 4096) and
    attention (SUM or MAX over up to 69 rows), n-gram ranges, thresholds, every kind of
    split (one block, few, the finishing kernel's read-ahead limits, more) -- against
    the oracle's occurrence lists and draft and, bit for bit, the separate ranking
    calls' scores and choices."""
    rng, n_cases = random_plan(2024, 60)
    i32 = dict(dtype=torch.int32, device="cuda")
    for it in range(n_cases):
        B = int(rng.integers(1, 9))
        stride = int(rng.choice([17, 300, 1024, 4096, 8192, 8200, 12000, 16384, 30000]))
        V = int(rng.choice([1, 2, 5, 50, 1000]))
        nmin = int(rng.integers(1, 4))
        nmax = int(rng.integers(nmin, 6))
        hidden = bool(rng.integers(0, 2))
        d = int(rng.choice([8, 64, 520, 4096])) if hidden else 0
        while hidden and B * stride * d > 4e7 and d > 8:
            d = {4096: 520, 520: 64, 64: 8}[d]
        R = 0 if hidden else int(rng.integers(1, 70))
        K = int(rng.integers(1, 40))
        th = float(rng.choice([-math.inf, 0.0, 0.3]))
        lo = 1 if stride <= pld.DRAFT_MAX_TOK_STRIDE else -(-stride // pld.DRAFT_MAX_PART)
        S = int(rng.choice([lo, max(2, lo), max(3, lo), 64, 240, 241, 600, 1024]))
        toks = rng.integers(0, V, size=(B, stride)).astype(np.int32)
        lens = rng.integers(1, stride + 1, size=B).astype(np.int32)
        lens[0] = stride
        what = f"case {it}: B{B} S{stride} V{V} n{nmin}-{nmax} d{d} R{R} K{K} th{th} split{S}"
        say("draft random", what)
        cp, cc, nu = oracle.find(toks, lens, nmin, nmax)
        ws = draft_workspace(B, S)
        o = [torch.full((B, stride), -1, **i32), torch.zeros(B, **i32), torch.zeros(B, **i32),
             torch.zeros(B, **i32), torch.zeros(B, dtype=torch.float32, device="cuda"),
             torch.zeros((B, K), **i32), torch.zeros(B, **i32)]
        sc = torch.full((B, stride), 777.0, dtype=torch.float32, device="cuda")
        if hidden:
            bits = synth.f32_to_bf16_bits(rng.standard_normal((B, stride, d)).astype(np.float32))
            hd = d_bf16(bits)
            pld.pld_draft_hidden(d_i32(toks), d_i32(lens), nmin, nmax, hd, K, *o, threshold=th,
                                 scores=sc, blocks_per_seq=S, workspace=ws)
            ref = gpu_rank_hidden(hd, lens, cp, cc, threshold=th)
        else:
            A = synth.make_attn(B, R, stride, lens, seed=it)
            agg = int(rng.integers(0, 2))
            pld.pld_draft_attn(d_i32(toks), d_i32(lens), nmin, nmax, d_f32(A), K, *o, agg=agg,
                               threshold=th, scores=sc, blocks_per_seq=S, workspace=ws)
            ref = gpu_rank_attn(d_f32(A), lens, cp, cc, agg, threshold=th)
        torch.cuda.synchronize()
        g = [t.cpu().numpy() for t in o]
        check_find((g[0], g[1], g[2]), (cp, cc, nu), what)
        gs = sc.cpu().numpy()
        for b in range(B):
            assert np.array_equal(gs[b, :cc[b]], ref[0][b, :cc[b]], equal_nan=True), what
        assert np.array_equal(g[3], ref[1]), what
        rd, rl = oracle.emit(toks, lens, g[3], K)
        assert np.array_equal(g[5], rd) and np.array_equal(g[6], rl), what
        if ws is not None:
            assert draft_keys_zero(ws, B), what


# ------------------------------------------------ halves and graph replays
def test_halves_equal_combined_calls():
    """score + select == rank, verify_argmax + verify_accept == verify_greedy, bit for bit."""
    say("halves")
    from paper_2412_01447_amd.step import DraftStep
    cfg = synth.Config("t", 6, 12000, 300, 1.1, 0.3, (8, 32), (1, 2), 256, "both", 9, 8, "f32", 31)
    w = synth.make_workload(cfg, "cuda", structured=False)
    toks, lens = d_i32(w["tokens"]), d_i32(w["lens"])
    attn = d_f32(w["attn"])
    dr, dl = synth.intended_drafts(w["metas"], cfg.K)
    z = d_f32(synth.logits_for(w, dr, dl))
    a = DraftStep(cfg.B, cfg.T, cfg.K, device="cuda", keep_scores=True, mode="split")
    b = DraftStep(cfg.B, cfg.T, cfg.K, device="cuda", keep_scores=True, mode="split")
    a.run(toks, lens, z, hidden=w["hidden"], attn=attn, ngram=cfg.ngram)
    b.find(toks, lens, *cfg.ngram)
    b.score_attn(attn, lens)
    b.select(into_best=False)
    b.score_hidden(w["hidden"], lens)
    b.select()
    b.emit(toks, lens)
    b.verify_argmax(z)
    b.verify_accept()
    torch.cuda.synchronize()
    ha, hb = a.host(), b.host()
    for k in ha:
        assert np.array_equal(ha[k], hb[k], equal_nan=True), k
    assert int(torch.count_nonzero(b.workspace).item()) == 0
    assert int(torch.count_nonzero(a.workspace).item()) == 0
    assert int(torch.count_nonzero(a.workspace_aux).item()) == 0


@pytest.mark.parametrize("mode", ["fused", "split", "both"])
def test_graph_replays_match_eager(mode):
    """The step captured in a HIP graph gives the eager result on every replay,
    with eager work and synchronisations between the replays ("both": the two
    artifacts ranked side by side, both scorings in one launch)."""
    say("graph replay", mode)
    from paper_2412_01447_amd.step import DraftStep
    both = mode == "both"
    cfg = synth.Config("t", 5, 6000, 400, 1.1, 0.3, (8, 32), (1, 3), 512,
                       "both" if both else "hidden", 9 if both else 0, 10, "f32", 41)
    w = synth.make_workload(cfg, "cuda", structured=True)
    toks, lens = d_i32(w["tokens"]), d_i32(w["lens"])
    attn = d_f32(w["attn"]) if both else None
    dr, dl = synth.intended_drafts(w["metas"], cfg.K)
    z = d_f32(synth.logits_for(w, dr, dl))
    smode = "split" if both else mode
    eager = DraftStep(cfg.B, cfg.T, cfg.K, device="cuda", keep_scores=True, mode=smode)
    eager.run(toks, lens, z, hidden=w["hidden"], attn=attn, ngram=cfg.ngram)
    torch.cuda.synchronize()
    want = eager.host()
    st = DraftStep(cfg.B, cfg.T, cfg.K, device="cuda", keep_scores=True, mode=smode)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        st.run(toks, lens, z, hidden=w["hidden"], attn=attn, ngram=cfg.ngram)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        st.run(toks, lens, z, hidden=w["hidden"], attn=attn, ngram=cfg.ngram)
    for rep in range(4):
        scribble = [st.cand_count, st.best_pos, st.draft, st.out_tokens]
        for t in scribble + ([st.best_pos_attn] if both else []):
            t.fill_(-9)   # scribble, replay
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = st.host()
        for k in want:
            assert np.array_equal(got[k], want[k], equal_nan=True), (rep, k)
        assert int(torch.count_nonzero(st.workspace).item()) == 0
        assert int(torch.count_nonzero(st.workspace_aux).item()) == 0
        eager.run(toks, lens, z, hidden=w["hidden"], attn=attn, ngram=cfg.ngram)
        torch.cuda.synchronize()


def test_graph_replays_sampling_and_loop_steps():
    """Sampling verification, and a whole loop step (draft, verify, commit, which
    moves the state forward), captured in HIP graphs: every replay matches the
    same calls made eagerly, with eager work between the replays."""
    say("graph replay: sampling and loop steps")
    from paper_2412_01447_amd.step import DraftStep
    cfg = synth.Config("t", 4, 3000, 300, 1.1, 0.4, (8, 32), (1, 2), 256, "hidden", 0, 8, "f32", 43)
    w = synth.make_workload(cfg, "cuda", structured=True)
    dr, dl = synth.intended_drafts(w["metas"], cfg.K)
    z = d_f32(synth.logits_for(w, dr, dl))
    U = d_f32(synth.make_uniforms(cfg.B, cfg.K, 43))

    def fresh():
        st = DraftStep(cfg.B, cfg.T + 64, cfg.K, device="cuda", keep_scores=True)
        st.set_sampling(0.7, 300, False, uniforms=U)
        toks = torch.full((cfg.B, cfg.T + 64), -1, dtype=torch.int32, device="cuda")
        toks[:, :cfg.T] = d_i32(w["tokens"])
        hid = torch.zeros((cfg.B, cfg.T + 64, 256), dtype=torch.bfloat16, device="cuda")
        hid[:, :cfg.T] = w["hidden"]
        return st, toks, d_i32(w["lens"]), hid, torch.zeros((cfg.B, 2), dtype=torch.int64,
                                                           device="cuda")

    def one_step(st, toks, lens, hid, stats):
        st.run(toks, lens, z, hidden=hid, ngram=cfg.ngram)
        st.commit(toks, lens, stats=stats)

    eager = fresh()
    cap = fresh()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):          # warm-up outside the capture, then restore the state
        one_step(*cap)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    cap = fresh()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        one_step(*cap)
    for rep in range(4):
        one_step(*eager)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        a, b = eager[0].host(), cap[0].host()
        for k in a:
            assert np.array_equal(a[k], b[k], equal_nan=True), (rep, k)
        for i in (1, 2, 4):
            assert torch.equal(eager[i], cap[i]), (rep, i)
        assert torch.equal(eager[0].row_sample, cap[0].row_sample), rep
        ws = cap[0].workspace[:pld.pld_workspace_bytes(cfg.B, cfg.K)]
        assert int(torch.count_nonzero(ws).item()) == 0
    assert int(cap[2].sum()) > int(d_i32(w["lens"]).sum())   # the replays moved forward


def test_verify_aligned_rows_with_tail():
    """16-byte aligned rows (the persistent kernel) whose width is not a whole
    number of vectors: the last elements of each row are taken one by one."""
    say("verify aligned rows with tail")
    rng = np.random.default_rng(12)
    for dt, V, pad in (("f32", 1001, 3), ("f32", 4094, 2), ("bf16", 8191, 1), ("bf16", 3001, 7)):
        B, K = 5, 7
        Z = rng.standard_normal((B, K + 1, V + pad)).astype(np.float32)
        Z[:, :, V - 1] = 50.0           # the maximum sits in the tail
        Z[1, :, V - 2] = 50.0           # a tie between the last vector's end and the tail
        draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
        draft[0, :3] = V - 1
        L = np.array([7, 3, 0, 7, 5], np.int32)
        view = np.ascontiguousarray(Z[:, :, :V])
        if dt == "f32":
            ref = oracle.verify(view, draft, L)
            got = gpu_verify(d_f32(Z)[:, :, :V], draft, L)
        else:
            bits = synth.f32_to_bf16_bits(Z)
            ref = oracle.verify(np.ascontiguousarray(bits[:, :, :V]), draft, L, bf16=True)
            got = gpu_verify(d_bf16(bits)[:, :, :V], draft, L)
        check_verify(got, ref, f"{dt} V={V}")
