"""A second, independent reading of the drafting step for tiny inputs.

Written with Python slicing and numpy / torch library reductions instead of the
oracle's index loops, so that a mistake in the oracle (a dropped term, a
shifted index, a reversed tie rule) shows up as a disagreement.  Only for
inputs small enough for pure Python.  Cites the paper (arXiv 2412.01447).
"""
import math

import numpy as np


def find(x, T, n_min=1, n_max=1):
    """Eq. 1 with n-gram queries tried longest first: compare list slices."""
    x = [int(v) for v in x[:T]]
    if T < 1:
        return [], -1
    for n in range(n_max, n_min - 1, -1):
        if T < n + 1:
            continue
        q = x[T - n:T]
        P = [j for j in range(1, T - 1) if j - n + 1 >= 0 and x[j - n + 1:j + 1] == q]
        if P:
            return P, n
    return [], 0


def find_unigram_numpy(x, T):
    """n = 1 reduces to numpy.flatnonzero over x[:T-1] == x[T-1], dropping j = 0."""
    x = np.asarray(x[:T])
    P = np.flatnonzero(x[:T - 1] == x[T - 1])
    return [int(j) for j in P if j >= 1]


def cosine(h, q):
    """Eq. 2's cos_sim with the eps = 1e-8 clamp, via numpy dot products in float64."""
    h = np.asarray(h, np.float64)
    q = np.asarray(q, np.float64)
    return float(np.dot(h, q) / math.sqrt(max(np.dot(h, h) * np.dot(q, q), 1e-16)))


def select(scores, pos, threshold=-math.inf):
    """argmax over (score, position): highest score, then the most recent position."""
    best = None
    for s, j in sorted(zip(scores, pos), key=lambda t: (t[0], t[1])):
        if s > threshold:
            best = (s, j)
    return (-1, -math.inf) if best is None else (best[1], best[0])


def emit(x, T, j, K):
    """Sec. 4.3: the K tokens after x[j], cut at the end of the context."""
    if j < 0 or j > T - 2:
        return []
    return [int(v) for v in x[j + 1:T][:K]]


def verify(Z, draft):
    """Greedy acceptance: numpy.argmax (first maximum) per row, keep the matching prefix."""
    L = len(draft)
    y = [int(np.argmax(np.asarray(Z[i], np.float64))) for i in range(L + 1)]
    a = 0
    while a < L and y[a] == draft[a]:
        a += 1
    return a, list(draft[:a]) + [y[a]], y


def sample_row(z, temperature, u):
    """Inverse CDF of softmax(z / temperature) at u, with numpy's cumsum and
    searchsorted (the first index whose cumulative mass exceeds u * total)."""
    z = np.asarray(z, np.float64)
    m = z.max()
    if m == -np.inf:
        return 0
    p = np.exp((z - m) / temperature)
    c = np.cumsum(p)
    u = min(max(float(u), 0.0), float(np.nextafter(np.float32(1), np.float32(0))))
    v = int(np.searchsorted(c, u * c[-1], side="right"))
    if v >= len(z):
        v = int(np.flatnonzero(p > 0)[-1])
    return v


def verify_sample(Z, draft, temperature, u):
    """Sampling verification: the sampled token of every row, then the prefix
    of the draft that agrees with them."""
    L = len(draft)
    y = [sample_row(Z[i], temperature, u[i]) for i in range(L + 1)]
    a = 0
    while a < L and y[a] == draft[a]:
        a += 1
    return a, list(draft[:a]) + [y[a]], y


def select_prefix(x, T, pos, max_match):
    """Prompt lookup's selection: the match length of a candidate is the common
    prefix of the reversed context ending at j and the reversed context ending at
    T-1 (os.path.commonprefix on lists), capped; the best is the longest, the
    earliest among equals (min over (-length, j))."""
    import os.path
    back_q = list(x[:T])[::-1]
    lens_ = []
    for j in pos:
        if not 0 <= j <= T - 2:
            lens_.append(None)
            continue
        m = len(os.path.commonprefix([list(x[:j + 1])[::-1], back_q]))
        lens_.append(min(m, max_match))
    ok = [(-m, j) for m, j in zip(lens_, pos) if m is not None]
    if not ok:
        return lens_, -1, -math.inf
    m, j = min(ok)
    return lens_, j, float(-m)


def commit(x, T, out, n, cap):
    """Append with Python lists: the first min(n, cap - T) of out join x[:T]."""
    if T < 0 or T > cap or n < 0 or n > len(out):
        return list(x), T, 0
    keep = list(x[:T]) + list(out[:n])[:cap - T]
    m = len(keep) - T
    return keep + list(x[len(keep):]), len(keep), m
