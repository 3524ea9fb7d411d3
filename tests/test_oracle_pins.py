"""Pins of the CPU oracle against things other than itself (CPU only).

Each group ties one oracle function to the paper's definition (arXiv 2412.01447)
through brute force on tiny inputs (tests/brute.py, a second reading written
with slicing and library reductions), closed forms, special cases and
invariants, chosen so that a plausible slip in the oracle -- a shifted row
index, the query row taken at T-1, a reversed tie rule, a dropped bound --
fails at least one of them.
"""
import math

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

import brute
import oracle
import synth


def _bits(a):
    return synth.f32_to_bf16_bits(np.asarray(a, np.float32))


# --------------------------------------------------------------------- find
@st.composite
def token_batches(draw):
    B = draw(st.integers(1, 4))
    stride = draw(st.integers(1, 48))
    V = draw(st.integers(1, 5))
    toks = np.array(draw(st.lists(st.lists(st.integers(0, V - 1), min_size=stride,
                                            max_size=stride), min_size=B, max_size=B)),
                    np.int32)
    lens = np.array(draw(st.lists(st.integers(0, stride + 1), min_size=B, max_size=B)),
                    np.int32)
    n_min = draw(st.integers(1, 4))
    n_max = draw(st.integers(n_min, 5))
    return toks, lens, n_min, n_max


@settings(max_examples=400, deadline=None)
@given(token_batches())
def test_find_matches_brute_force(case):
    """Eq. 1 with longest-first n-grams: the oracle equals the slicing reading."""
    toks, lens, n_min, n_max = case
    cp, cc, nu = oracle.find(toks, lens, n_min, n_max)
    stride = toks.shape[1]
    for b in range(len(lens)):
        T = int(lens[b])
        if T < 1 or T > stride:
            assert cc[b] == 0 and nu[b] == -1
            continue
        P, n = brute.find(toks[b], T, n_min, n_max)
        assert nu[b] == n
        assert list(cp[b, :cc[b]]) == P
        assert np.all(cp[b, cc[b]:] == -1)          # slots past the count untouched


@settings(max_examples=200, deadline=None)
@given(token_batches())
def test_find_unigram_is_flatnonzero(case):
    """n = 1 reduces to numpy.flatnonzero(x[:T-1] == x[T-1]) without j = 0."""
    toks, lens, _, _ = case
    cp, cc, nu = oracle.find(toks, lens, 1, 1)
    for b in range(len(lens)):
        T = int(lens[b])
        if 1 <= T <= toks.shape[1]:
            P = brute.find_unigram_numpy(toks[b], T)
            assert list(cp[b, :cc[b]]) == P
            assert nu[b] == (1 if P else 0)


@settings(max_examples=200, deadline=None)
@given(token_batches())
def test_find_invariants(case):
    """Every candidate's window equals the query n-gram, order is strictly ascending,
    every longer n has no occurrence, and j stays in [max(n-1,1), T-2]."""
    toks, lens, n_min, n_max = case
    cp, cc, nu = oracle.find(toks, lens, n_min, n_max)
    for b in range(len(lens)):
        T, n, P = int(lens[b]), int(nu[b]), cp[b, :cc[b]]
        if n <= 0:
            assert cc[b] == 0
            continue
        x = toks[b]
        assert np.all(np.diff(P) > 0)
        for j in P:
            assert max(n - 1, 1) <= j <= T - 2
            assert np.array_equal(x[j - n + 1:j + 1], x[T - n:T])
        for m in range(n + 1, n_max + 1):
            q = x[T - m:T] if T >= m else None
            assert q is None or not any(np.array_equal(x[j - m + 1:j + 1], q)
                                        for j in range(max(m - 1, 1), T - 1))


def test_find_degenerate_lengths():
    toks = np.array([[5, 5, 5, 5]], np.int32)
    for T, want in [(0, ([], -1)), (1, ([], 0)), (2, ([], 0)), (3, ([1], 1)), (4, ([1, 2], 1)),
                    (5, ([], -1))]:
        cp, cc, nu = oracle.find(toks, np.array([T], np.int32), 1, 1)
        assert (list(cp[0, :cc[0]]), int(nu[0])) == want, T
    # a query longer than the context has no occurrence; T = n+1 allows exactly j = n-1 >= 1
    cp, cc, nu = oracle.find(np.array([[1, 2, 1, 2]], np.int32), np.array([4], np.int32), 2, 2)
    assert list(cp[0, :cc[0]]) == [1] and nu[0] == 2


# -------------------------------------------------------------- rank hidden
def _rank_h(H, T, P, threshold=-math.inf):
    B = 1
    bits = _bits(H)[None]
    cp = np.array([P + [-1] * (H.shape[0] - len(P))], np.int32)
    return oracle.rank_hidden(bits, np.array([T], np.int32), cp,
                              np.array([len(P)], np.int32), threshold)


@pytest.mark.parametrize("seed", range(6))
def test_rank_hidden_is_cosine_of_previous_rows(seed):
    """Eq. 2: s_j = cos(H[j-1], H[T-2]); compared with numpy dot products and with
    torch.nn.functional.cosine_similarity in float64."""
    rng = np.random.default_rng(seed)
    T, d = 40, 24
    H = rng.standard_normal((T, d)).astype(np.float32)
    Hq = synth.bf16_bits_to_f32(_bits(H)).astype(np.float64)
    P = sorted(rng.choice(np.arange(1, T - 1), size=9, replace=False).tolist())
    sc, bp, bs = _rank_h(H, T, P)
    ref = [brute.cosine(Hq[j - 1], Hq[T - 2]) for j in P]
    np.testing.assert_allclose(sc[0, :len(P)], ref, rtol=1e-12, atol=1e-15)
    tref = torch.nn.functional.cosine_similarity(torch.from_numpy(Hq[[j - 1 for j in P]]),
                                                 torch.from_numpy(Hq[T - 2])[None], dim=1)
    np.testing.assert_allclose(sc[0, :len(P)], tref.numpy(), rtol=1e-12, atol=1e-15)
    j, s = brute.select(ref, P)
    assert bp[0] == j and math.isclose(bs[0], s, rel_tol=1e-12)


def test_rank_hidden_planted_copy_scores_exactly_one():
    """A bitwise copy of the query row before one occurrence gives cos = 1 exactly."""
    rng = np.random.default_rng(7)
    T, d = 30, 64
    H = rng.standard_normal((T, d)).astype(np.float32)
    H[11] = H[T - 2]                               # row before j = 12
    sc, bp, bs = _rank_h(H, T, [4, 12, 20])
    assert bs[0] == 1.0 and bp[0] == 12 and sc[0, 1] == 1.0


def test_rank_hidden_ties_go_to_most_recent():
    """Identical rows and a power-of-two-scaled row tie exactly; the latest j wins."""
    rng = np.random.default_rng(3)
    T, d = 32, 16
    H = rng.standard_normal((T, d)).astype(np.float32)
    H[4] = H[9]
    H[19] = 4.0 * H[9]
    # make these three the best: align them with the query
    H[T - 2] = H[9] + 0.01 * rng.standard_normal(d).astype(np.float32)
    sc, bp, bs = _rank_h(H, T, [5, 10, 20, 25])
    assert sc[0, 0] == sc[0, 1] == sc[0, 2]
    assert bp[0] == 20
    sc, bp, bs = _rank_h(H, T, [5, 10, 25])
    assert bp[0] == 10


def test_rank_hidden_threshold_and_empty():
    """App. B threshold: only s > theta is eligible; nothing eligible gives -1."""
    rng = np.random.default_rng(5)
    T, d = 20, 8
    H = rng.standard_normal((T, d)).astype(np.float32)
    P = [2, 7, 13]
    sc, bp, bs = _rank_h(H, T, P)
    top = np.max(sc[0, :3])
    sc2, bp2, bs2 = _rank_h(H, T, P, threshold=top)
    assert bp2[0] == -1 and bs2[0] == -math.inf
    mid = np.sort(sc[0, :3])[1]
    _, bp3, _ = _rank_h(H, T, P, threshold=mid)
    assert bp3[0] == bp[0]
    _, bp4, bs4 = _rank_h(H, T, [])
    assert bp4[0] == -1 and bs4[0] == -math.inf


def test_rank_hidden_zero_rows_and_out_of_range():
    """The eps clamp gives 0 for a zero row; out-of-range candidates score NaN and never win."""
    T, d = 10, 8
    H = np.zeros((T, d), np.float32)
    H[T - 2] = 1.0
    H[3] = -1.0
    sc, bp, bs = _rank_h(H, T, [1, 4, 9, 0])
    assert sc[0, 0] == 0.0 and sc[0, 1] == -1.0
    assert math.isnan(sc[0, 2]) and math.isnan(sc[0, 3])
    assert bp[0] == 1


# ---------------------------------------------------------------- rank attn
def _rank_a(A, T, P, agg, threshold=-math.inf):
    R, n = A.shape
    cp = np.array([P + [-1] * (n - len(P))], np.int32)
    return oracle.rank_attn(A[None].astype(np.float32), np.array([T], np.int32), cp,
                            np.array([len(P)], np.int32), agg, threshold)


def test_rank_attn_one_hot_and_lookup():
    """One-hot rows give a known winner; R = 1 SUM is a lookup of key j-1."""
    T = 16
    A = np.zeros((3, T), np.float32)
    A[0, 6] = 1.0
    A[1, 6] = 1.0
    A[2, 11] = 1.0
    sc, bp, _ = _rank_a(A, T, [3, 7, 12], oracle.AGG_SUM)
    assert list(sc[0, :3]) == [0.0, 2.0, 1.0] and bp[0] == 7
    sc, bp, _ = _rank_a(A, T, [3, 7, 12], oracle.AGG_MAX)
    assert list(sc[0, :3]) == [0.0, 1.0, 1.0] and bp[0] == 12     # tie -> most recent
    rng = np.random.default_rng(1)
    A1 = rng.random((1, T)).astype(np.float32)
    sc, _, _ = _rank_a(A1, T, [1, 5, 14], oracle.AGG_SUM)
    assert list(sc[0, :3]) == [float(A1[0, 0]), float(A1[0, 4]), float(A1[0, 13])]


@pytest.mark.parametrize("agg", [oracle.AGG_SUM, oracle.AGG_MAX])
def test_rank_attn_matches_numpy(agg):
    rng = np.random.default_rng(11)
    B, R, T = 3, 7, 50
    A = rng.random((B, R, T)).astype(np.float32)
    lens = np.array([50, 33, 2], np.int32)
    P = [[1, 5, 9, 48], [2, 31], [1]]
    cap = T
    cp = np.full((B, cap), -1, np.int32)
    for b, p in enumerate(P):
        cp[b, :len(p)] = p
    cc = np.array([len(p) for p in P], np.int32)
    sc, bp, bs = oracle.rank_attn(A, lens, cp, cc, agg)
    for b in range(B):
        for c, j in enumerate(P[b]):
            if j > lens[b] - 2:
                assert math.isnan(sc[b, c])
                continue
            col = A[b, :, j - 1].astype(np.float64)
            want = col.sum() if agg == oracle.AGG_SUM else col.max()
            assert math.isclose(sc[b, c], want, rel_tol=1e-15)
    assert bp[2] == -1


def test_generator_attention_rows_sum_to_one():
    """Sanity of the Dirichlet-like generator: SUM over all keys of R rows is R."""
    lens = np.array([64, 40], np.int32)
    A = synth.make_attn(2, 5, 64, lens, seed=0)
    np.testing.assert_allclose(A.astype(np.float64).sum(axis=2), 1.0, rtol=1e-6)
    assert np.all(A[1, :, 39:] == 0)


# --------------------------------------------------------------------- emit
@settings(max_examples=200, deadline=None)
@given(st.integers(1, 40), st.integers(1, 12), st.integers(-2, 45), st.integers(0, 3))
def test_emit_is_contiguous_span(T, K, j, pad):
    """Sec. 4.3: draft = x[j*+1 .. j*+L], L = min(K, T-1-j*), no draft for j* = -1."""
    stride = T + pad
    x = np.arange(100, 100 + stride, dtype=np.int32)[None]
    dr, dl = oracle.emit(x, np.array([T], np.int32), np.array([j], np.int32), K)
    want = brute.emit(x[0], T, j, K)
    assert dl[0] == len(want)
    assert list(dr[0, :dl[0]]) == want
    assert np.all(dr[0, dl[0]:] == -1)
    if 0 <= j <= T - 2:
        assert dl[0] == min(K, T - 1 - j) >= 1


# ------------------------------------------------------------------- verify
@settings(max_examples=300, deadline=None)
@given(st.integers(1, 6), st.integers(1, 9), st.data())
def test_verify_matches_numpy_argmax(K, V, data):
    """Greedy acceptance: numpy.argmax (first maximum) per row, longest matching prefix.
    Small integer logits make ties common; -0/+0 appear through negation of 0."""
    vals = data.draw(st.lists(st.lists(st.integers(-2, 2), min_size=V, max_size=V),
                              min_size=K + 1, max_size=K + 1))
    Z = np.array(vals, np.float32)
    neg = data.draw(st.lists(st.booleans(), min_size=V, max_size=V))
    Z[:, np.array(neg)] *= -1.0                          # turns some 0 into -0
    L = data.draw(st.integers(0, K))
    draft = np.full(K, -1, np.int32)
    draft[:L] = data.draw(st.lists(st.integers(0, V - 1), min_size=L, max_size=L))
    acc, out, cnt, ra = oracle.verify(Z[None], draft[None], np.array([L], np.int32))
    a, toks, y = brute.verify(Z, list(draft[:L]))
    assert acc[0] == a and cnt[0] == a + 1
    assert list(out[0, :a + 1]) == toks and np.all(out[0, a + 1:] == -1)
    assert list(ra[0, :L + 1]) == y and np.all(ra[0, L + 1:] == -1)
    # invariants: 0 <= a <= L <= K, out[:a] == draft[:a], out[i] == argmax Z[i] for i <= a
    assert 0 <= acc[0] <= L <= K
    assert np.array_equal(out[0, :a], draft[:a])
    assert all(out[0, i] == y[i] for i in range(a + 1))


def test_verify_bf16_ties_and_signed_zero():
    """bf16 logits widen exactly; equal maxima and -0/+0 resolve to the lowest id."""
    Z = np.array([[[-1.0, 0.5, 0.5, 0.25], [-0.0, 0.0, -3.0, -0.0]]], np.float32)
    bits = synth.f32_to_bf16_bits(Z)
    for z, bf in ((Z, False), (bits, True)):
        acc, out, cnt, ra = oracle.verify(z, np.array([[2]], np.int32),
                                          np.array([1], np.int32), bf16=bf)
        assert list(ra[0]) == [1, 0] and acc[0] == 0 and list(out[0]) == [1, -1]
        assert cnt[0] == 1


def test_verify_one_hot_known_accepts():
    """One-hot logits planted on the first p draft tokens accept exactly p tokens."""
    K, V = 6, 20
    draft = np.array([[3, 4, 5, 6, 7, 8]], np.int32)
    for p in range(K + 1):
        Z = np.zeros((1, K + 1, V), np.float32)
        for i in range(K + 1):
            Z[0, i, draft[0, i] if (i < p and i < K) else 19] = 1.0
        acc, out, cnt, _ = oracle.verify(Z, draft, np.array([K], np.int32))
        assert acc[0] == p
        assert cnt[0] == p + 1
        want = list(draft[0, :p]) + [19]
        assert list(out[0, :p + 1]) == want
    # full acceptance emits K+1 tokens; a short draft (L < K) emits L+1
    Z = np.zeros((1, K + 1, V), np.float32)
    for i in range(K):
        Z[0, i, draft[0, i]] = 1
    Z[0, K, 0] = 1
    acc, out, cnt, _ = oracle.verify(Z, draft, np.array([K], np.int32))
    assert cnt[0] == K + 1 and out[0, K] == 0
    acc, out, cnt, _ = oracle.verify(Z, draft, np.array([2], np.int32))
    assert acc[0] == 2 and cnt[0] == 3 and out[0, 2] == int(np.argmax(Z[0, 2]))


def test_verify_bad_draft_len():
    Z = np.zeros((2, 3, 4), np.float32)
    acc, out, cnt, _ = oracle.verify(Z, np.zeros((2, 2), np.int32), np.array([-1, 3], np.int32))
    assert list(acc) == [-1, -1] and list(cnt) == [0, 0] and np.all(out == -1)


# ------------------------------------------------------- the chained step
def test_structured_step_finds_planted_source():
    """On generated data with the structured hidden variant, the planted source of the
    last token is the unique cosine winner, and the draft is what follows it."""
    cfg = synth.Config("t", 3, 256, 50, 1.1, 0.3, (4, 12), (1, 1), 32, "hidden", 0, 5, "f32", 9)
    toks, lens, metas = synth.make_tokens(cfg)
    H = synth.make_hidden(cfg.B, cfg.T, cfg.d, cfg.seed,
                          plants=synth.structured_hidden_plants(lens, metas))
    bits = H.view(torch.int16).numpy().view(np.uint16)
    cp, cc, nu = oracle.find(toks, lens)
    sc, bp, bs = oracle.rank_hidden(bits, lens, cp, cc)
    for b in range(cfg.B):
        assert bp[b] == metas[b].query_src_end and bs[b] == 1.0
    dr, dl = oracle.emit(toks, lens, bp, cfg.K)
    want, wn = synth.intended_drafts(metas, cfg.K)
    assert np.array_equal(dr, want) and np.array_equal(dl, wn)


# ------------------------------------------------------- sampling verification
def _sample1(z, tau, u):
    """One row through a K = 1 call with an empty draft (L = 0): row 0 is sampled."""
    Z = np.stack([np.asarray(z, np.float32), np.zeros(len(z), np.float32)])[None]
    acc, out, cnt, rows = oracle.verify_sample(Z, np.full((1, 1), -1, np.int32),
                                               np.array([0], np.int32), tau,
                                               np.array([[u, 0.0]], np.float32))
    assert acc[0] == 0 and cnt[0] == 1 and out[0, 0] == rows[0, 0]
    return int(rows[0, 0])


def test_sample_two_tokens_closed_form():
    """softmax of [log a, log b] / tau puts a^(1/tau) / (a^(1/tau) + b^(1/tau)) on token 0."""
    for a, b, tau in ((3.0, 1.0, 1.0), (1.0, 4.0, 1.0), (3.0, 1.0, 0.5), (2.0, 5.0, 2.0)):
        z = [math.log(a), math.log(b)]
        p0 = a ** (1 / tau) / (a ** (1 / tau) + b ** (1 / tau))
        assert _sample1(z, tau, p0 * 0.999) == 0
        assert _sample1(z, tau, min(p0 * 1.001, 0.9999)) == 1


def test_sample_exact_boundary_and_zero_mass():
    """The cumulative mass must exceed u * S strictly; tokens without mass are
    never drawn; u is clamped to [0, 1); a row with no mass gives token 0."""
    assert _sample1([0.0, 0.0], 1.0, 0.5) == 1               # t lands exactly on the boundary
    assert _sample1([0.0, 0.0, 0.0, 0.0], 1.0, 0.25) == 1
    z = [-math.inf, 0.0, -math.inf, 0.0, -math.inf]
    assert _sample1(z, 1.0, 0.0) == 1
    assert _sample1(z, 1.0, 0.4999) == 1
    assert _sample1(z, 1.0, 0.5) == 3
    assert _sample1(z, 1.0, 0.9999) == 3
    assert _sample1(z, 1.0, 1.5) == 3                        # clamped below 1
    assert _sample1(z, 1.0, -0.3) == 1                       # clamped to 0
    assert _sample1([-math.inf] * 4, 1.0, 0.7) == 0


def test_sample_small_temperature_is_argmax():
    """As tau -> 0 the distribution concentrates on the first maximum."""
    z = [0.3, 1.7, -0.4, 1.6, 1.7]
    for u in (0.0, 0.3, 0.49, 0.999):
        assert _sample1(z, 1e-3, u) in (1, 4)
    assert _sample1(z, 1e-3, 0.0) == 1 and _sample1(z, 1e-3, 0.3) == 1
    assert _sample1(z, 1e-3, 0.999) == 4                     # the two maxima share the mass


def test_sample_distribution_matches_softmax():
    """The inverse CDF maps uniform draws to softmax(z / tau): token frequencies
    over a regular grid of u equal the probabilities to within the grid step."""
    z = np.array([0.2, -1.0, 1.5, 0.0, 0.7, -3.0], np.float32)
    for tau in (1.0, 0.6):
        p = np.exp((z.astype(np.float64) - z.max()) / tau)
        p /= p.sum()
        n = 4000
        grid = (np.arange(n) + 0.5) / n
        Z = np.broadcast_to(z, (n, 2, 6)).copy()
        U = np.stack([grid, np.zeros(n)], axis=1).astype(np.float32)
        acc, out, cnt, rows = oracle.verify_sample(Z, np.full((n, 1), -1, np.int32),
                                                   np.zeros(n, np.int32), tau, U)
        freq = np.bincount(rows[:, 0], minlength=6) / n
        assert np.allclose(freq, p, atol=1.5 / n)


@settings(max_examples=300, deadline=None)
@given(st.integers(1, 6), st.integers(1, 9), st.sampled_from([0.5, 1.0, 2.0]), st.data())
def test_verify_sample_matches_brute(K, V, tau, data):
    """Random small logits (ties, -inf entries) and uniforms: the oracle's samples
    and acceptance equal numpy's cumsum / searchsorted reading."""
    vals = data.draw(st.lists(st.lists(st.sampled_from([-2.0, -1.0, 0.0, 0.5, 1.0, 3.0, -math.inf]),
                                       min_size=V, max_size=V), min_size=K + 1, max_size=K + 1))
    Z = np.array(vals, np.float32)
    u = np.array(data.draw(st.lists(st.sampled_from([0.0, 0.1, 0.25, 0.5, 0.73, 0.999, 1.0]),
                                    min_size=K + 1, max_size=K + 1)), np.float32)
    L = data.draw(st.integers(0, K))
    draft = np.full(K, -1, np.int32)
    draft[:L] = data.draw(st.lists(st.integers(0, V - 1), min_size=L, max_size=L))
    acc, out, cnt, rows = oracle.verify_sample(Z[None], draft[None], np.array([L], np.int32),
                                               tau, u[None])
    a, toks, y = brute.verify_sample(Z, list(draft[:L]), tau, u)
    assert acc[0] == a and cnt[0] == a + 1
    assert list(out[0, :a + 1]) == toks and np.all(out[0, a + 1:] == -1)
    assert list(rows[0, :L + 1]) == y and np.all(rows[0, L + 1:] == -1)
    assert np.array_equal(out[0, :a], draft[:a])


def test_verify_sample_acceptance_and_bad_lengths():
    """Drafts equal to the samples are accepted whole (K+1 tokens out); a draft
    differing at i keeps i tokens; bad lengths give -1 / 0 as in greedy."""
    rng = np.random.default_rng(5)
    B, K, V = 3, 4, 7
    Z = rng.standard_normal((B, K + 1, V)).astype(np.float32)
    U = rng.random((B, K + 1)).astype(np.float32)
    _, _, _, rows = oracle.verify_sample(Z, np.zeros((B, K), np.int32), np.full(B, K, np.int32),
                                         1.0, U)
    draft = rows[:, :K].copy()
    draft[1, 2] = (draft[1, 2] + 1) % V
    lens = np.array([K, K, 9], np.int32)
    acc, out, cnt, r2 = oracle.verify_sample(Z, draft, lens, 1.0, U)
    assert acc[0] == K and cnt[0] == K + 1 and list(out[0]) == list(rows[0])
    assert acc[1] == 2 and list(out[1, :3]) == [draft[1, 0], draft[1, 1], rows[1, 2]]
    assert acc[2] == -1 and cnt[2] == 0 and np.all(out[2] == -1)


# ------------------------------------------------------- prefix selection
@settings(max_examples=300, deadline=None)
@given(token_batches(), st.integers(1, 9), st.data())
def test_select_prefix_matches_brute(batch, max_match, data):
    """Prompt lookup's selection (Sec. 2, Fig. 3 caption) on random small token
    rows, over the oracle's own occurrence lists and over arbitrary (also
    out-of-range) candidate positions: match lengths, the longest-then-earliest
    choice and its score equal the commonprefix reading."""
    toks, lens, n_min, n_max = batch
    B, stride = toks.shape
    cp, cc, _ = oracle.find(toks, lens, n_min, n_max)
    extra = data.draw(st.lists(st.integers(-2, stride + 1), min_size=1, max_size=6))
    for pos_lists in ([list(cp[b, :cc[b]]) for b in range(B)], [extra] * B):
        cap = max(1, max(len(p) for p in pos_lists))
        pos = np.full((B, cap), -1, np.int32)
        cnt = np.zeros(B, np.int32)
        for b, p in enumerate(pos_lists):
            pos[b, :len(p)] = p
            cnt[b] = len(p)
        sc, bp, bs = oracle.select_prefix(toks, lens, pos, cnt, max_match)
        for b in range(B):
            T = int(lens[b])
            if not 2 <= T <= stride:
                assert bp[b] == -1 and bs[b] == -math.inf
                continue
            want, wj, ws = brute.select_prefix(toks[b], T, pos_lists[b], max_match)
            got = [None if math.isnan(v) else int(v) for v in sc[b, :cnt[b]]]
            assert got == want and bp[b] == wj and bs[b] == ws


def test_select_prefix_invariants():
    """Every n-gram occurrence matches at least n tokens back; capping at the n
    used makes every candidate tie, so the earliest (cand_pos[0]) wins, which is
    prompt lookup's first match."""
    rng = np.random.default_rng(3)
    toks = rng.integers(0, 4, size=(6, 200)).astype(np.int32)
    lens = np.array([200, 150, 2, 1, 77, 199], np.int32)
    cp, cc, nu = oracle.find(toks, lens, 1, 4)
    sc, bp, bs = oracle.select_prefix(toks, lens, cp, cc, 64)
    for b in range(6):
        if cc[b] == 0:
            assert bp[b] == -1
            continue
        assert (sc[b, :cc[b]] >= nu[b]).all()
        assert bs[b] == sc[b, :cc[b]].max()
        first_best = cp[b, int(np.argmax(sc[b, :cc[b]]))]   # argmax: the first, i.e. earliest
        assert bp[b] == first_best
    _, bp_n, bs_n = oracle.select_prefix(toks, lens, cp, cc, 1)
    for b in range(6):
        assert bp_n[b] == (cp[b, 0] if cc[b] else -1)


# ------------------------------------------------------------------ commit
@settings(max_examples=300, deadline=None)
@given(st.data())
def test_commit_matches_brute(data):
    """The append of the generation loop: list concatenation, capped by the
    limit and the row, lengths and the (emitted, steps) counters."""
    B = data.draw(st.integers(1, 4))
    stride = data.draw(st.integers(1, 20))
    K = data.draw(st.integers(1, 5))
    toks = np.array(data.draw(st.lists(st.lists(st.integers(0, 9), min_size=stride,
                                                max_size=stride), min_size=B, max_size=B)),
                    np.int32)
    lens = np.array(data.draw(st.lists(st.integers(-1, stride + 1), min_size=B, max_size=B)),
                    np.int32)
    out = np.array(data.draw(st.lists(st.lists(st.integers(10, 19), min_size=K + 1,
                                               max_size=K + 1), min_size=B, max_size=B)),
                   np.int32)
    cnt = np.array(data.draw(st.lists(st.integers(-1, K + 2), min_size=B, max_size=B)), np.int32)
    limit = np.array(data.draw(st.lists(st.integers(0, stride + 3), min_size=B, max_size=B)),
                     np.int32) if data.draw(st.booleans()) else None
    stats0 = np.array(data.draw(st.lists(st.lists(st.integers(0, 50), min_size=2, max_size=2),
                                         min_size=B, max_size=B)), np.int64)
    t2, l2, s2 = oracle.commit(toks, lens, out, cnt, limit=limit, stats=stats0)
    for b in range(B):
        cap = stride if limit is None else min(int(limit[b]), stride)
        n = int(cnt[b]) if 0 <= cnt[b] <= K + 1 else -1
        want_x, want_T, m = brute.commit(toks[b], int(lens[b]), out[b], n, cap)
        assert list(t2[b]) == want_x[:stride] and l2[b] == want_T
        assert list(s2[b]) == [stats0[b, 0] + m, stats0[b, 1] + (m > 0)]
