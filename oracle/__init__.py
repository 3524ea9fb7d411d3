"""CPU oracle for the PLD+ drafting step -- TEST INFRASTRUCTURE ONLY.

Only the test-suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never does, and the
oracle imports nothing from it.

The arithmetic lives in ``pld_oracle.c`` (plain scalar C, IEEE double, built by
gcc); this module only marshals numpy arrays into it.  Each wrapper names the
passage of the paper (arXiv 2412.01447) whose definition the C function writes
out:

* :func:`find`         -- occurrence set P, Eq. 1 (Sec. 4.2), n-gram longest-first
* :func:`rank_hidden`  -- cosine ranking of H[j-1] against H[T-2], Eq. 2 (Sec. 4.2.2)
* :func:`rank_attn`    -- aggregated attention ranking, Eq. 3 (Sec. 4.2.1, Sec. 7.1)
* :func:`emit`         -- draft span x[j*+1 .. j*+K], Sec. 4.3
* :func:`verify`       -- greedy acceptance of the longest matching prefix, Sec. 3, 4.4
* :func:`verify_sample` -- the same acceptance on tokens drawn from softmax(Z / tau)
* :func:`select_prefix` -- prompt lookup's selection: longest matching prefix, earliest
  (Sec. 2, Fig. 3 caption), the baseline PLD+ replaces
* :func:`commit`       -- the emitted tokens appended to the sequences (the generation loop)

All inputs are host numpy arrays; bf16 data is passed as its uint16 bit pattern.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libpld_oracle.so")
_lib = None

AGG_SUM = 0
AGG_MAX = 1
DT_F32 = 0
DT_BF16 = 1

_i32p = ctypes.POINTER(ctypes.c_int32)
_f64p = ctypes.POINTER(ctypes.c_double)
_vp = ctypes.c_void_p
_i64 = ctypes.c_int64
_int = ctypes.c_int


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b
        _b.build()
    _lib = load_library(_LIB_PATH)
    return _lib


def load_library(path):
    """Open a build of pld_oracle.c and declare its signatures."""
    lib = ctypes.CDLL(path)
    lib.pld_ref_find.argtypes = [_vp, _i64, _vp, _int, _int, _int, _vp, _i64, _vp, _vp]
    lib.pld_ref_rank_hidden.argtypes = [_vp, _i64, _i64, _int, _i64, _vp, _vp, _i64, _vp, _int,
                                        ctypes.c_double, _vp, _vp, _vp, _vp]
    lib.pld_ref_rank_attn.argtypes = [_vp, _i64, _i64, _int, _i64, _int, _vp, _vp, _i64, _vp,
                                      _int, ctypes.c_double, _vp, _vp, _vp, _vp]
    lib.pld_ref_emit.argtypes = [_vp, _i64, _vp, _vp, _int, _int, _vp, _vp]
    lib.pld_ref_verify.argtypes = [_vp, _int, _i64, _i64, _int, _int, _vp, _vp, _int, _vp, _vp,
                                   _vp, _vp]
    lib.pld_ref_verify_sample.argtypes = [_vp, _int, _i64, _i64, _int, _int, _vp, _vp, _int,
                                          ctypes.c_double, _vp, _i64, _vp, _vp, _vp, _vp]
    lib.pld_ref_select_prefix.argtypes = [_vp, _i64, _vp, _vp, _i64, _vp, _int, _int, _vp, _vp,
                                          _vp]
    lib.pld_ref_commit.argtypes = [_vp, _i64, _vp, _vp, _vp, _vp, _int, _int, _vp]
    for f in (lib.pld_ref_find, lib.pld_ref_rank_hidden, lib.pld_ref_rank_attn,
              lib.pld_ref_emit, lib.pld_ref_verify, lib.pld_ref_verify_sample,
              lib.pld_ref_select_prefix, lib.pld_ref_commit):
        f.restype = _int
    return lib


def _p(a):
    return a.ctypes.data_as(_vp) if a is not None else None


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"oracle {name}: invalid arguments")


def find(tokens, lens, ngram_min=1, ngram_max=1, cap=None):
    """Occurrence set (Eq. 1), longest n first.

    tokens: int32 [B, tok_stride]; lens: int32 [B].
    Returns (cand_pos [B, cap] int32 with -1 past the count, cand_count [B], ngram_used [B]).
    """
    tokens = _c(tokens, np.int32)
    lens = _c(lens, np.int32)
    B, stride = tokens.shape
    cap = stride if cap is None else cap
    cand_pos = np.full((B, cap), -1, np.int32)
    cnt = np.zeros(B, np.int32)
    used = np.zeros(B, np.int32)
    rc = _load().pld_ref_find(_p(tokens), stride, _p(lens), B, ngram_min, ngram_max,
                              _p(cand_pos), cap, _p(cnt), _p(used))
    _check(rc, "find")
    return cand_pos, cnt, used


def rank_hidden(hidden_bits, lens, cand_pos, cand_count, threshold=-np.inf):
    """Cosine ranking (Eq. 2).  hidden_bits: uint16 [B, n_rows, d] (bf16 bits).

    Returns (scores [B, cap] float64, best_pos [B] int32, best_score [B] float64).
    """
    h = _c(hidden_bits, np.uint16)
    B, n_rows, d = h.shape
    lens = _c(lens, np.int32)
    cand_pos = _c(cand_pos, np.int32)
    cand_count = _c(cand_count, np.int32)
    cap = cand_pos.shape[1]
    scores = np.full((B, cap), np.nan)
    best = np.zeros(B, np.int32)
    bscore = np.zeros(B)
    work = np.zeros(max(cap, 1))
    rc = _load().pld_ref_rank_hidden(_p(h), n_rows * d, d, d, n_rows, _p(lens), _p(cand_pos),
                                     cap, _p(cand_count), B, float(threshold), _p(scores),
                                     _p(best), _p(bscore), _p(work))
    _check(rc, "rank_hidden")
    return scores, best, bscore


def rank_attn(attn, lens, cand_pos, cand_count, agg=AGG_SUM, threshold=-np.inf):
    """Attention ranking (Eq. 3 / head aggregation).  attn: float32 [B, R, n_keys].

    Returns (scores [B, cap] float64, best_pos [B] int32, best_score [B] float64).
    """
    a = _c(attn, np.float32)
    B, R, n_keys = a.shape
    lens = _c(lens, np.int32)
    cand_pos = _c(cand_pos, np.int32)
    cand_count = _c(cand_count, np.int32)
    cap = cand_pos.shape[1]
    scores = np.full((B, cap), np.nan)
    best = np.zeros(B, np.int32)
    bscore = np.zeros(B)
    work = np.zeros(max(cap, 1))
    rc = _load().pld_ref_rank_attn(_p(a), R * n_keys, n_keys, R, n_keys, int(agg), _p(lens),
                                   _p(cand_pos), cap, _p(cand_count), B, float(threshold),
                                   _p(scores), _p(best), _p(bscore), _p(work))
    _check(rc, "rank_attn")
    return scores, best, bscore


def emit(tokens, lens, best_pos, K):
    """Draft span (Sec. 4.3).  Returns (draft [B, K] int32 padded with -1, draft_len [B])."""
    tokens = _c(tokens, np.int32)
    lens = _c(lens, np.int32)
    best_pos = _c(best_pos, np.int32)
    B, stride = tokens.shape
    draft = np.zeros((B, K), np.int32)
    dlen = np.zeros(B, np.int32)
    rc = _load().pld_ref_emit(_p(tokens), stride, _p(lens), _p(best_pos), B, K, _p(draft),
                              _p(dlen))
    _check(rc, "emit")
    return draft, dlen


def verify(logits, draft, draft_len, bf16=False):
    """Greedy verification (Sec. 3, 4.4).

    logits: float32 [B, K+1, V], or uint16 bf16 bits when ``bf16``.
    Returns (accept_len [B], out_tokens [B, K+1], out_count [B], row_argmax [B, K+1]).
    """
    z = _c(logits, np.uint16 if bf16 else np.float32)
    B, K1, V = z.shape
    K = K1 - 1
    draft = _c(draft, np.int32)
    draft_len = _c(draft_len, np.int32)
    assert draft.shape == (B, K)
    acc = np.zeros(B, np.int32)
    out = np.zeros((B, K1), np.int32)
    cnt = np.zeros(B, np.int32)
    rowarg = np.zeros((B, K1), np.int32)
    rc = _load().pld_ref_verify(_p(z), DT_BF16 if bf16 else DT_F32, K1 * V, V, V, K, _p(draft),
                                _p(draft_len), B, _p(acc), _p(out), _p(cnt), _p(rowarg))
    _check(rc, "verify")
    return acc, out, cnt, rowarg


def select_prefix(tokens, lens, cand_pos, cand_count, max_match):
    """Prompt lookup's selection (Sec. 2, Fig. 3 caption): the candidate whose
    preceding tokens match the query's for the longest run (up to max_match),
    the earliest among equals.  Returns (scores [B, cap] float64 match lengths,
    NaN for out-of-range candidates; best_pos [B]; best_score [B])."""
    tokens = _c(tokens, np.int32)
    lens = _c(lens, np.int32)
    cand_pos = _c(cand_pos, np.int32)
    cand_count = _c(cand_count, np.int32)
    B, stride = tokens.shape
    cap = cand_pos.shape[1]
    scores = np.zeros((B, cap), np.float64)
    bp = np.zeros(B, np.int32)
    bs = np.zeros(B, np.float64)
    rc = _load().pld_ref_select_prefix(_p(tokens), stride, _p(lens), _p(cand_pos), cap,
                                       _p(cand_count), B, int(max_match), _p(scores), _p(bp),
                                       _p(bs))
    _check(rc, "select_prefix")
    return scores, bp, bs


def commit(tokens, lens, out_tokens, out_count, limit=None, stats=None):
    """The generation loop's append: out_tokens[b][:out_count[b]] joins sequence b
    (capped at limit[b] and the row's capacity), lens advance, stats [B, 2] int64
    (emitted tokens, steps) accumulate.  Works in place on copies and returns
    (tokens, lens, stats)."""
    tokens = np.array(tokens, np.int32, order="C")
    lens = np.array(lens, np.int32)
    out_tokens = _c(out_tokens, np.int32)
    out_count = _c(out_count, np.int32)
    B, stride = tokens.shape
    K = out_tokens.shape[1] - 1
    lim = None if limit is None else _c(limit, np.int32)
    st = np.zeros((B, 2), np.int64) if stats is None else np.array(stats, np.int64)
    rc = _load().pld_ref_commit(_p(tokens), stride, _p(lens), _p(lim), _p(out_tokens),
                                _p(out_count), B, K, _p(st))
    _check(rc, "commit")
    return tokens, lens, st


def verify_sample(logits, draft, draft_len, temperature, uniforms, bf16=False):
    """Sampling verification (Sec. 4.4 with a temperature; Sec. 5 samples at T = 1).

    Row i's token is the inverse CDF of softmax(Z[b][i] / temperature) at the
    caller's uniform draw uniforms[b][i] in [0, 1); acceptance keeps the draft
    up to the first mismatch with these samples.
    logits: float32 [B, K+1, V], or uint16 bf16 bits when ``bf16``; uniforms:
    float32 [B, K+1].  Returns (accept_len [B], out_tokens [B, K+1],
    out_count [B], row_sample [B, K+1]).
    """
    z = _c(logits, np.uint16 if bf16 else np.float32)
    B, K1, V = z.shape
    K = K1 - 1
    draft = _c(draft, np.int32)
    draft_len = _c(draft_len, np.int32)
    u = _c(uniforms, np.float32)
    assert draft.shape == (B, K) and u.shape == (B, K1)
    acc = np.zeros(B, np.int32)
    out = np.zeros((B, K1), np.int32)
    cnt = np.zeros(B, np.int32)
    rows = np.zeros((B, K1), np.int32)
    rc = _load().pld_ref_verify_sample(_p(z), DT_BF16 if bf16 else DT_F32, K1 * V, V, V, K,
                                       _p(draft), _p(draft_len), B, float(temperature), _p(u), K1,
                                       _p(acc), _p(out), _p(cnt), _p(rows))
    _check(rc, "verify_sample")
    return acc, out, cnt, rows


def step_hidden(tokens, lens, hidden_bits, logits, K, ngram_min=1, ngram_max=1,
                threshold=-np.inf, bf16_logits=False):
    """The whole drafting step with hidden-state ranking, chained stage by stage."""
    cp, cc, nu = find(tokens, lens, ngram_min, ngram_max)
    sc, bp, bs = rank_hidden(hidden_bits, lens, cp, cc, threshold)
    dr, dl = emit(tokens, lens, bp, K)
    acc, out, cnt, ra = verify(logits, dr, dl, bf16=bf16_logits)
    return dict(cand_pos=cp, cand_count=cc, ngram_used=nu, scores=sc, best_pos=bp,
                best_score=bs, draft=dr, draft_len=dl, accept_len=acc, out_tokens=out,
                out_count=cnt, row_argmax=ra)
