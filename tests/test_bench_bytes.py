"""The algorithmic bytes the bench divides by kernel time, on inputs small
enough to count by hand: what each kernel must move per step, written out
from the definitions (candidate rows plus the query row for Eq. 2, distinct
128-byte lines of each attention row for Eq. 3, rows i <= L of the logits),
never the dense work a kernel avoids."""
import numpy as np

import bench
import synth


def _cfg(rank, B=2, d=8, R=3, K=2, V=10, logits="f32"):
    return synth.Config("t", B, 64, V, 1.1, 0.0, (1, 1), (1, 1), d, rank, R, K, logits, 0)


def test_hidden_and_greedy_bytes():
    cfg = _cfg("hidden")
    lens = np.array([64, 50], np.int32)
    cc = np.array([3, 0], np.int32)
    cp = np.full((2, 64), -1, np.int32)
    cp[0, :3] = [5, 9, 40]
    dlen = np.array([2, 0], np.int32)
    got = bench.algorithmic_bytes(cfg, lens, cc, dlen, cp, 4, fused=False)
    # find: both token rows up to their lengths, plus the three positions written
    assert got["find"] == (64 + 50) * 4 + 3 * 4
    # Eq. 2: three candidate rows and the query row of d = 8 bf16, plus the positions
    # read; the empty sequence reads no query row
    assert got["score_hidden"] == (3 + 1) * 8 * 2 + 3 * 4
    # greedy verification: rows 0..L of V fp32 logits per sequence
    assert got["verify_argmax"] == (3 + 1) * 10 * 4
    assert "score_attn" not in got
    # the one-launch drafting counts find, ranking and selection together
    fused = bench.algorithmic_bytes(cfg, lens, cc, dlen, cp, 4, fused=True)
    assert fused["draft"] == got["find"] + got["score_hidden"] + got["select_draft"]
    assert fused["verify_argmax"] == got["verify_argmax"]


def test_attention_counts_distinct_lines():
    cfg = _cfg("attn", R=3)
    lens = np.array([64, 64], np.int32)
    cc = np.array([4, 1], np.int32)
    cp = np.full((2, 64), -1, np.int32)
    # keys j-1: 0, 1, 31 share the first 128-byte line (32 fp32 keys); 32 starts the next
    cp[0, :4] = [1, 2, 32, 33]
    cp[1, :1] = [60]          # key 59: one line
    dlen = np.array([2, 2], np.int32)
    got = bench.algorithmic_bytes(cfg, lens, cc, dlen, cp, 4, fused=False)
    assert got["score_attn"] == (2 + 1) * 3 * 128 + 5 * 4
    both = bench.algorithmic_bytes(_cfg("both", R=3), lens, cc, dlen, cp, 4, fused=False)
    assert both["score_attn"] == got["score_attn"]
    assert both["score_hidden"] == (4 + 1 + 1 + 1) * 8 * 2 + 5 * 4


def test_sampling_bytes():
    cfg = _cfg("hidden", V=5000)
    lens = np.array([64, 64], np.int32)
    cc = np.array([1, 1], np.int32)
    cp = np.full((2, 64), -1, np.int32)
    cp[:, 0] = 7
    dlen = np.array([2, 1], np.int32)
    got = bench.algorithmic_bytes(cfg, lens, cc, dlen, cp, 4, fused=False, sample=True)
    # 5000 fp32 = 1250 vectors of 16 bytes: 3 segments of 512 vectors per row
    rows = 3 + 2
    assert got["verify_sample_stats"] == rows * 5000 * 4 + rows * 3 * 8
    assert got["verify_sample_finish"] == rows * (3 * 8 + 4) + 2 * 2 * 4 + 2 * 3 * 4
    assert "verify_argmax" not in got
