"""The pins have teeth: plausible slips planted in a copy of the oracle are caught.

Each mutant is a one-line textual change to oracle/pld_oracle.c (a shifted
artifact row, the query taken at the last token, a reversed tie rule, ...),
compiled with gcc into a temporary library.  A compact run of the same pins
as test_oracle_pins.py / test_golden_oracle.py must fail on every mutant and
pass on the unmodified source.  CPU only; the mistakes live in the oracle.
"""
import os
import subprocess

import math

import numpy as np
import pytest

import brute
import golden_cases
import oracle
import synth

SRC = os.path.join(os.path.dirname(oracle.__file__), "pld_oracle.c")

MUTANTS = {
    "artifact row j instead of j-1": ("const uint16_t *h = Hb + (j - 1) * h_row_stride;",
                                      "const uint16_t *h = Hb + j * h_row_stride;"),
    "query row T-1 instead of T-2": ("seq_ok ? Hb + (T - 2) * h_row_stride : Hb;",
                                     "seq_ok ? Hb + (T - 1) * h_row_stride : Hb;"),
    "tie goes to the earliest position": ("(v == bs && pos[c] > bj)", "(v == bs && pos[c] < bj)"),
    "verify takes the last maximum": ("if (v == 0 || z > best) {", "if (v == 0 || z >= best) {"),
    "shortest n-gram first": ("for (int n = ngram_max; n >= ngram_min; --n) {",
                              "for (int n = ngram_min; n <= ngram_max; ++n) {"),
    "last token counted as its own occurrence": ("for (int64_t j = lo; j <= T - 2; ++j) {",
                                                 "for (int64_t j = lo; j <= T - 1; ++j) {"),
    "draft truncation off by one": ("L = T - 1 - j;", "L = T - j;"),
    "attention key j instead of j-1": ("a_row_stride + (j - 1)];", "a_row_stride + j];"),
    "norm without the square": ("hh += hv * hv;", "hh += hv;"),
    "accept counts one past the mismatch": ("a = i;\n            break;", "a = i + 1;\n            break;"),
    "threshold taken as >=": ("!(v > threshold)", "!(v >= threshold)"),
    "sample boundary taken as >=": ("if (c > t) {", "if (c >= t) {"),
    "sampling temperature ignored": ("p[v] = exp((p[v] - m) / temperature);",
                                     "p[v] = exp(p[v] - m);"),
    "sampling uses the previous row's uniform": (
        "double u = (double)uniforms[(int64_t)b * u_stride + i];",
        "double u = (double)uniforms[(int64_t)b * u_stride + (i > 0 ? i - 1 : 0)];"),
    "prefix tie goes to the latest position": ("(s == bs && j < bj)", "(s == bs && j > bj)"),
    "prefix match compared one token early": ("x[j - m] == x[T - 1 - m]", "x[j - m] == x[T - 2 - m]"),
    "commit ignores the limit": ("if (limit && limit[b] < cap_b) cap_b = limit[b];",
                                 "if (limit && limit[b] < 0) cap_b = limit[b];"),
    "commit counts a step with nothing appended": ("stats[2 * b + 1] += (m > 0) ? 1 : 0;",
                                                   "stats[2 * b + 1] += 1;"),
}


def _pins_pass():
    """A compact run of the pins; True when every check holds."""
    try:
        # golden fixtures
        fx, toks, lens, H, A = golden_cases.load("fig1_overview.json")
        ex = fx["expected"]
        cp, cc, nu = oracle.find(toks, lens, 1, 1)
        if list(cp[0, :cc[0]]) != ex["cand_pos"]:
            return False
        bits = synth.f32_to_bf16_bits(H)
        sc, bp, bs = oracle.rank_hidden(bits, lens, cp, cc)
        if bp[0] != ex["hidden_best_pos"] or not np.allclose(sc[0, :2], ex["hidden_scores"]):
            return False
        sc, bp, bs = oracle.rank_attn(A, lens, cp, cc, oracle.AGG_SUM)
        if bp[0] != ex["attn_sum_best_pos"]:
            return False
        # the token row padded with a sentinel past T, so that a slip that reads
        # beyond the sequence sees a defined value; the length is compared too
        padded = np.full((toks.shape[0], toks.shape[1] + 16), 424242, np.int32)
        padded[:, :toks.shape[1]] = toks
        for K in (3, 12):
            for tk in (toks, padded):
                dr, dl = oracle.emit(tk, lens, np.array([10], np.int32), K)
                want = ex[f"draft_K{K}"]
                if list(dr[0]) != want or dl[0] != sum(1 for t in want if t != -1):
                    return False
        for vc in fx["verify_cases"]:
            Z, dr, dl = golden_cases.verify_case(vc)
            acc, out, cnt, ra = oracle.verify(Z, dr, dl)
            if acc[0] != vc["expected"]["accept_len"] or list(out[0]) != vc["expected"]["out_tokens"]:
                return False
        fx, toks, lens, H, _ = golden_cases.load("fig3_newline.json")
        for key, (a, b) in (("n1", (1, 1)), ("n1to4", (1, 4)), ("n7to8", (7, 8))):
            cp, cc, nu = oracle.find(toks, lens, a, b)
            if list(cp[0, :cc[0]]) != fx["expected"][key]["cand_pos"]:
                return False
        # brute force on random tiny inputs
        rng = np.random.default_rng(0)
        for _ in range(60):
            T = int(rng.integers(2, 30))
            x = rng.integers(0, 3, size=(1, T)).astype(np.int32)
            cp, cc, nu = oracle.find(x, np.array([T], np.int32), 1, 3)
            P, n = brute.find(x[0], T, 1, 3)
            if list(cp[0, :cc[0]]) != P or nu[0] != n:
                return False
        # identical rows tie -> the most recent occurrence
        Hr = rng.standard_normal((12, 8)).astype(np.float32)
        Hr[2] = Hr[6]
        Hr[10] = Hr[6] + np.float32(0.01)
        cpos = np.full((1, 12), -1, np.int32)
        cpos[0, :2] = [3, 7]
        _, bp, bs = oracle.rank_hidden(synth.f32_to_bf16_bits(Hr)[None], np.array([12], np.int32),
                                       cpos, np.array([2], np.int32))
        if bp[0] != 7:
            return False
        # threshold: the top score itself is not eligible
        sc, bp, bs = oracle.rank_hidden(synth.f32_to_bf16_bits(Hr)[None],
                                        np.array([12], np.int32), cpos, np.array([2], np.int32),
                                        threshold=float(bs[0]))
        if bp[0] != -1:
            return False
        # sampling verification: closed forms, the strict boundary, brute force
        for a_, b_, tau in ((3.0, 1.0, 1.0), (3.0, 1.0, 0.5)):
            z = np.array([[[math.log(a_), math.log(b_)], [0.0, 0.0]]], np.float32)
            p0 = a_ ** (1 / tau) / (a_ ** (1 / tau) + b_ ** (1 / tau))
            for u, want in ((p0 * 0.999, 0), (p0 * 1.001, 1)):
                _, _, _, rows = oracle.verify_sample(z, np.full((1, 1), -1, np.int32),
                                                     np.array([0], np.int32), tau,
                                                     np.array([[u, 0.0]], np.float32))
                if rows[0, 0] != want:
                    return False
        _, _, _, rows = oracle.verify_sample(np.zeros((1, 2, 2), np.float32),
                                             np.full((1, 1), -1, np.int32),
                                             np.array([0], np.int32), 1.0,
                                             np.array([[0.5, 0.0]], np.float32))
        if rows[0, 0] != 1:
            return False
        for _ in range(40):
            K, V = 3, 5
            Zs = rng.standard_normal((K + 1, V)).astype(np.float32)
            us = rng.random(K + 1).astype(np.float32)
            dr = rng.integers(0, V, K).astype(np.int32)
            acc, out, cnt, rows = oracle.verify_sample(Zs[None], dr[None],
                                                       np.array([K], np.int32), 1.0, us[None])
            a_, toks, y = brute.verify_sample(Zs, list(dr), 1.0, us)
            if list(rows[0]) != y or acc[0] != a_:
                return False
        # prompt lookup's selection: the Fig. 3 fixture, brute force
        fx, toks, lens, _, _ = golden_cases.load("fig3_newline.json")
        e = fx["expected"]["pld_prefix"]
        cp, cc, _ = oracle.find(toks, lens, 1, 1)
        for cap_m in (8, 3):
            sc, bp, _ = oracle.select_prefix(toks, lens, cp, cc, cap_m)
            if list(sc[0, :cc[0]]) != e[f"match_len_max{cap_m}"] or bp[0] != e[f"best_pos_max{cap_m}"]:
                return False
        for _ in range(40):
            T = int(rng.integers(2, 40))
            x = rng.integers(0, 2, size=(1, T)).astype(np.int32)
            cp, cc, _ = oracle.find(x, np.array([T], np.int32), 1, 1)
            sc, bp, bs = oracle.select_prefix(x, np.array([T], np.int32), cp, cc, 6)
            want, wj, ws = brute.select_prefix(x[0], T, list(cp[0, :cc[0]]), 6)
            if [int(v) for v in sc[0, :cc[0]]] != want or bp[0] != wj:
                return False
        # commit: list appends under a limit, the counters
        for _ in range(40):
            stride, K = 12, 3
            x = rng.integers(0, 5, size=(2, stride)).astype(np.int32)
            T0 = rng.integers(0, stride + 1, size=2).astype(np.int32)
            out = rng.integers(5, 9, size=(2, K + 1)).astype(np.int32)
            n = rng.integers(0, K + 2, size=2).astype(np.int32)
            lim = rng.integers(0, stride + 1, size=2).astype(np.int32)
            t2, l2, s2 = oracle.commit(x, T0, out, n, limit=lim)
            for b in range(2):
                wx, wT, m = brute.commit(x[b], int(T0[b]), out[b], int(n[b]), int(lim[b]))
                if list(t2[b]) != wx[:stride] or l2[b] != wT or list(s2[b]) != [m, int(m > 0)]:
                    return False
        return True
    except Exception:
        return False


def _with_lib(path):
    saved = oracle._lib
    oracle._lib = oracle.load_library(path)
    try:
        return _pins_pass()
    finally:
        oracle._lib = saved


def _build(src_text, tmp_path, name):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"lib{name}.so"
    c.write_text(src_text)
    subprocess.run(["gcc", "-std=c11", "-O2", "-fPIC", "-shared", "-ffp-contract=off",
                    str(c), "-o", str(so), "-lm"], check=True)
    return str(so)


def test_unmodified_oracle_passes(tmp_path):
    assert _with_lib(_build(open(SRC).read(), tmp_path, "orig"))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_is_caught(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site not unique: {old!r}"
    so = _build(src.replace(old, new), tmp_path, "mutant")
    assert not _with_lib(so), f"pins did not catch: {name}"
