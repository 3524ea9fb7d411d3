"""The boundary from plain C.

tests/c_step (C99, the HIP runtime's C API, no C++ and no torch) runs find ->
rank by hidden states and by attention -> emit -> greedy verification through
libpld on a stream of its own, with device buffers it allocates itself.  Its
outputs must match the oracle stage by stage: bit-exact lists, choices, drafts
and acceptance, scores within the tolerance, near-tie flips counted.
"""
import os
import subprocess

import numpy as np
import pytest

import oracle
import synth
from gpu_helpers import check_best, check_find, check_scores, check_verify, say

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
EXE = os.path.join(ROOT, "tests", "c_step")


def _save(d, name, a):
    np.ascontiguousarray(a).tofile(os.path.join(d, name))


def _load(d, name, dtype, shape):
    a = np.fromfile(os.path.join(d, name), dtype=dtype)
    assert a.size == int(np.prod(shape)), f"{name}: {a.size} values"
    return a.reshape(shape)


def test_c_program_runs_the_step(tmp_path):
    assert os.path.exists(EXE), "tests/c_step is not built: run __graft_entry__.build()"
    B, S, D, R, K, V = 4, 600, 192, 5, 6, 300
    nmin, nmax = 1, 2
    rng = np.random.default_rng(2024)
    tokens = rng.integers(0, 12, size=(B, S)).astype(np.int32)
    # a full row, a ragged one, one too short for any occurrence, a short one
    lens = np.array([600, 257, 1, 37], np.int32)
    hidden = synth.f32_to_bf16_bits(rng.standard_normal((B, S, D)).astype(np.float32))
    attn = rng.random((B, R, S)).astype(np.float32)
    cp, cc, nu = oracle.find(tokens, lens, nmin, nmax)
    assert cc[0] >= 2 and cc[2] == 0
    # an exact tie in sequence 0: the rows before its last two occurrences
    # equal the query row, so both score 1 and the later one must win
    T0 = int(lens[0])
    for c in (int(cc[0]) - 1, int(cc[0]) - 2):
        hidden[0, cp[0, c] - 1] = hidden[0, T0 - 2]
    sh, bh, bsh = oracle.rank_hidden(hidden, lens, cp, cc)
    assert bh[0] == cp[0, cc[0] - 1]
    dr, dl = oracle.emit(tokens, lens, bh, K)
    Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    for b in range(B):
        for i in range(min(int(dl[b]), 4)):        # a planted accepted prefix of up to 4 tokens
            Z[b, i, dr[b, i]] += 8.0
    d = str(tmp_path)
    _save(d, "tokens.i32", tokens)
    _save(d, "lens.i32", lens)
    _save(d, "hidden.u16", hidden)
    _save(d, "attn.f32", attn)
    _save(d, "logits.f32", Z)
    say("c_step", d, B, S, D, R, K, V)
    r = subprocess.run([EXE, d, str(B), str(S), str(nmin), str(nmax), str(D), str(R), str(K),
                        str(V)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, f"c_step failed ({r.returncode}): {r.stdout}{r.stderr}"

    g = {n: _load(d, f"{n}.i32", np.int32, shp) for n, shp in (
        ("cand_pos", (B, S)), ("cand_count", (B,)), ("ngram_used", (B,)), ("best_h", (B,)),
        ("best_a", (B,)), ("draft", (B, K)), ("draft_len", (B,)), ("accept_len", (B,)),
        ("out_tokens", (B, K + 1)), ("out_count", (B,)))}
    for n, shp in (("scores_h", (B, S)), ("bscore_h", (B,)), ("scores_a", (B, S)),
                   ("bscore_a", (B,))):
        g[n] = _load(d, f"{n}.f32", np.float32, shp)

    check_find((g["cand_pos"], g["cand_count"], g["ngram_used"]), (cp, cc, nu), "c_step")
    check_scores(g["scores_h"], sh, cc, "c_step hidden")
    flips = check_best(g["best_h"], g["bscore_h"], sh, bh, bsh, cp, cc, "c_step hidden")
    assert g["best_h"][0] == bh[0], "the exact tie goes to the later occurrence"
    sa, ba, bsa = oracle.rank_attn(attn, lens, cp, cc)
    check_scores(g["scores_a"], sa, cc, "c_step attention")
    flips += check_best(g["best_a"], g["bscore_a"], sa, ba, bsa, cp, cc, "c_step attention")
    # the later stages on the GPU's own choice and draft
    rdr, rdl = oracle.emit(tokens, lens, g["best_h"], K)
    assert np.array_equal(g["draft"], rdr) and np.array_equal(g["draft_len"], rdl)
    check_verify((g["accept_len"], g["out_tokens"], g["out_count"]),
                 oracle.verify(Z, g["draft"], g["draft_len"]), "c_step verify")
    assert (g["accept_len"][g["draft_len"] > 0] > 0).any(), "no planted prefix was accepted"
    ws = np.fromfile(os.path.join(d, "workspace.u8"), dtype=np.uint8)
    assert not ws.any(), "the workspace is left zero"
    say("c_step: near-tie flips", flips)
