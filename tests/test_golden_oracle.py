"""The oracle reproduces the hand-derived fixtures of tests/golden/ (CPU only).

The fixtures restate the worked scenarios the paper describes in words (Fig. 1
caption: the 'to' example; Fig. 3 caption: the newline example in code editing)
with small integer hidden states, so every expected value is a closed form.
"""
import math

import numpy as np

import brute
import golden_cases
import oracle
import synth


def test_fig1_overview_oracle():
    fx, toks, lens, H, A = golden_cases.load("fig1_overview.json")
    ex = fx["expected"]
    assert int(lens[0]) == ex["T"]
    cp, cc, nu = oracle.find(toks, lens, 1, 1)
    assert list(cp[0, :cc[0]]) == ex["cand_pos"] and nu[0] == ex["ngram_used"]
    bits = synth.f32_to_bf16_bits(H)
    sc, bp, bs = oracle.rank_hidden(bits, lens, cp, cc)
    np.testing.assert_allclose(sc[0, :cc[0]], ex["hidden_scores"], rtol=1e-15, atol=0)
    assert bp[0] == ex["hidden_best_pos"]
    for agg, key in ((oracle.AGG_SUM, "attn_sum"), (oracle.AGG_MAX, "attn_max")):
        sc, bp, bs = oracle.rank_attn(A, lens, cp, cc, agg)
        assert list(sc[0, :cc[0]]) == ex[key + "_scores"]
        assert bp[0] == ex[key + "_best_pos"]
    for K in (3, 12):
        dr, dl = oracle.emit(toks, lens, np.array([ex["hidden_best_pos"]], np.int32), K)
        assert list(dr[0]) == ex[f"draft_K{K}"] and dl[0] == ex[f"draft_len_K{K}"]


def test_fig1_verify_cases_oracle_and_brute():
    fx, *_ = golden_cases.load("fig1_overview.json")
    for vc in fx["verify_cases"]:
        Z, dr, dl = golden_cases.verify_case(vc)
        acc, out, cnt, ra = oracle.verify(Z, dr, dl)
        e = vc["expected"]
        assert acc[0] == e["accept_len"], vc["name"]
        assert list(out[0]) == e["out_tokens"], vc["name"]
        assert cnt[0] == e["out_count"], vc["name"]
        assert list(ra[0]) == e["row_argmax"], vc["name"]
        a, toks, _ = brute.verify(Z[0], list(dr[0, :dl[0]]))
        assert a == e["accept_len"] and toks == e["out_tokens"][:a + 1]
        acc, out, cnt, ra = oracle.verify(synth.f32_to_bf16_bits(Z), dr, dl, bf16=True)
        assert acc[0] == e["accept_len"] and list(out[0]) == e["out_tokens"]


def test_fig3_newline_oracle():
    fx, toks, lens, H, _ = golden_cases.load("fig3_newline.json")
    ex = fx["expected"]
    bits = synth.f32_to_bf16_bits(H)
    for key, (nmin, nmax) in (("n1", (1, 1)), ("n1to3", (1, 3)), ("n1to4", (1, 4)),
                              ("n5to6", (5, 6)), ("n7to8", (7, 8))):
        e = ex[key]
        cp, cc, nu = oracle.find(toks, lens, nmin, nmax)
        assert list(cp[0, :cc[0]]) == e["cand_pos"], key
        assert nu[0] == e["ngram_used"], key
        sc, bp, bs = oracle.rank_hidden(bits, lens, cp, cc)
        assert bp[0] == e["best_pos"], key
        if "hidden_scores" in e:
            np.testing.assert_allclose(sc[0, :cc[0]], e["hidden_scores"], rtol=1e-15)
        if "draft_len_K4" in e:
            dr, dl = oracle.emit(toks, lens, bp, 4)
            assert dl[0] == e["draft_len_K4"], key
            if "draft_K4" in e:
                assert list(dr[0, :4]) == e["draft_K4"], key
    assert math.isclose(ex["n1"]["hidden_scores"][2], 6 / math.sqrt(42), rel_tol=1e-16)
    # prompt lookup's selection on the same occurrences: the span of f
    e = ex["pld_prefix"]
    cp, cc, _ = oracle.find(toks, lens, 1, 1)
    assert list(cp[0, :cc[0]]) == e["cand_pos"]
    for cap_m in (8, 3, 1):
        sc, bp, bs = oracle.select_prefix(toks, lens, cp, cc, cap_m)
        assert list(sc[0, :cc[0]]) == e[f"match_len_max{cap_m}"], cap_m
        assert bp[0] == e[f"best_pos_max{cap_m}"] and bs[0] == max(e[f"match_len_max{cap_m}"])
    dr, dl = oracle.emit(toks, lens, oracle.select_prefix(toks, lens, cp, cc, 8)[1], 4)
    assert list(dr[0]) == e["draft_K4_max8"]
