"""Seeded synthetic inputs for the PLD+ drafting step.

This module is shared by the oracle side (tests, CPU baseline) and the GPU side
(tests, bench).  It holds none of the method's arithmetic: no matching, no
ranking, no argmax.  It only draws inputs shaped like the paper's input-guided
workloads (arXiv 2412.01447, Sec. 5.1: outputs that copy spans of their input):

* tokens  -- finite Zipf(s) ids over a vocabulary of V; the last quarter of each
  sequence plays the generated text and a stated fraction of it is covered by
  spans copied from the first three quarters (the "prompt").  One span always
  ends at the last token, so the query has a planted source; its position is
  returned in the metadata.
* hidden  -- one layer of hidden states, N(0,1) rounded to bf16 (round to
  nearest even, done by torch).  Optionally the row before the planted source
  is made a bitwise copy of the query row (the "structured" variant), so that
  the planted source is the unique cosine winner.
* attn    -- one query row of attention per (sequence, head): Dirichlet(0.3)
  weights over the visible keys 0..T-2 (normalised Gamma draws in double, cast
  to fp32), zero for keys >= T-1.  The structured variant adds one unit of
  mass at the key before the planted source and renormalises.
* logits  -- N(0,1) verification logits [B][K+1][V]; for a random prefix of
  length p ~ U{0..K} the caller-given draft tokens get +boost (the draft is an
  input here; the generator never computes one).
* uniforms -- the draws of sampling verification, U[0, 1) fp32 [B][K+1].
* decoding tasks (DECODE_TASKS) -- for the multi-step loop: target sequences
  (the token generator's output, whose last quarter is the continuation to
  generate; or sectioned documents copied with edits), hidden states that embed each
  position's last few tokens (a decaying window), and a stand-in target model
  whose greedy choice at every position is the target token, so that greedy
  decoding reproduces the target whatever the drafts.

Seeds are numpy SeedSequence([seed, b, stream]) per sequence and stream, so a
sequence can be regenerated alone.
"""
from __future__ import annotations

import dataclasses

import numpy as np

STREAM_TOKENS = 1
STREAM_PLANT = 2
STREAM_ATTN = 3
STREAM_LOGITS = 4
STREAM_HIDDEN = 5
STREAM_UNIFORMS = 6
STREAM_CONTEXT = 7
STREAM_MODEL = 8
STREAM_EDIT = 9
STREAM_SECTIONS = 10


@dataclasses.dataclass(frozen=True)
class Config:
    """One workload of the drafting step (all sequences of one batch share T)."""
    name: str
    B: int
    T: int
    V: int
    zipf_s: float
    plant_frac: float
    span: tuple
    ngram: tuple          # (n_min, n_max), tried longest first
    d: int                # hidden width (0: no hidden ranking in the step)
    rank: str             # "hidden", "attn" or "both"
    R: int                # attention rows per sequence (0: no attention ranking)
    K: int
    logits: str           # "f32" or "bf16"
    seed: int
    query_count_max: int = 0   # >0: choose a query token with at most this many hits
    agg: str = "sum"           # attention aggregation over the R rows: "sum" or "max"
    theta: float = float("-inf")   # ranking threshold: only scores > theta are eligible


# The workloads the drafting step is measured on.  Config 1 matches the
# paper's input sizes (a few hundred words, Table of input lengths in App. B);
# the others scale batch, context, vocabulary and hidden width up.
CONFIGS = {
    1: Config("b1_t1024_v32000_d4096_hidden_k10", 1, 1024, 32000, 1.1, 0.40, (8, 32), (1, 1),
              4096, "hidden", 0, 10, "f32", 0),
    2: Config("b8_t4096_v32000_d4096_hidden_n3to1_k10", 8, 4096, 32000, 1.1, 0.30, (8, 64),
              (1, 3), 4096, "hidden", 0, 10, "f32", 1),
    3: Config("b32_t8192_v32000_attn_sum_r40_k16", 32, 8192, 32000, 1.1, 0.25, (8, 64), (1, 1),
              5120, "attn", 40, 16, "f32", 2),
    4: Config("b64_t16384_v128256_d8192_hidden_attn_r64_k16_bf16", 64, 16384, 128256, 1.05, 0.20,
              (16, 128), (1, 1), 8192, "both", 64, 16, "bf16", 3),
    5: Config("b4_t131072_v128256_d4096_hidden_k32", 4, 131072, 128256, 1.05, 0.15, (16, 128),
              (1, 1), 4096, "hidden", 0, 32, "f32", 4, query_count_max=4000),
    # The paper's own two settings at its input sizes: PLD+(a) takes the MAX over
    # the top-50 induction heads across layers with K = 70 (Eq. 3, Sec. 5.5 and the
    # head-count table of App. B), PLD+(h) the cosine ranking with theta = 0, the
    # best threshold of App. B.  The last token is a frequent one (up to 64
    # occurrences), so that ranking and threshold have candidates to act on.
    6: Config("b1_t1024_v32000_attn_max_r50_k70", 1, 1024, 32000, 1.1, 0.40, (8, 32), (1, 1),
              0, "attn", 50, 70, "f32", 5, query_count_max=64, agg="max"),
    7: Config("b1_t1024_v32000_d4096_hidden_theta0_k10", 1, 1024, 32000, 1.1, 0.40, (8, 32),
              (1, 1), 4096, "hidden", 0, 10, "f32", 6, query_count_max=64, theta=0.0),
}


def rng_for(seed: int, b: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([int(seed), int(b), int(stream)]))


def zipf_cdf(V: int, s: float) -> np.ndarray:
    k = np.arange(1, V + 1, dtype=np.float64)
    w = k ** (-s)
    c = np.cumsum(w)
    return c / c[-1]


def zipf_tokens(rng: np.random.Generator, n: int, cdf: np.ndarray) -> np.ndarray:
    """Finite Zipf draw by inverse CDF; token id = rank - 1."""
    u = rng.random(n)
    t = np.searchsorted(cdf, u, side="right")
    return np.minimum(t, len(cdf) - 1).astype(np.int32)


@dataclasses.dataclass
class SeqMeta:
    spans: list            # (dst_start, src_start, length) of every planted copy
    query_src_end: int     # position of the planted source of the last token
    intended: np.ndarray   # the tokens that follow the planted source (up to 64)


def make_sequence(T: int, V: int, s: float, plant_frac: float, span: tuple, seed: int, b: int,
                  query_count_max: int = 0, margin: int = 64, cdf=None):
    """One token sequence of length T with planted copies (see module doc)."""
    cdf = zipf_cdf(V, s) if cdf is None else cdf
    x = zipf_tokens(rng_for(seed, b, STREAM_TOKENS), T, cdf)
    rng = rng_for(seed, b, STREAM_PLANT)
    lo, hi = span
    g0 = T - T // 4                      # start of the "generated" region
    spans = []
    if T < 8 or g0 < 2:
        return x, SeqMeta(spans, -1, np.zeros(0, np.int32))
    hi = max(lo, min(hi, T // 4, g0 // 2))
    lo = min(lo, hi)
    lf = int(rng.integers(lo, hi + 1))   # the span that ends at the last token
    margin = max(0, min(margin, g0 - lf - 1))
    # fill the rest of the generated region with non-overlapping copies
    target = int(round(plant_frac * (T - g0)))
    covered = lf
    taken = np.zeros(T, bool)
    taken[T - lf - 1:] = True            # keep one gap before the forced span
    attempts = 0
    while covered < target and attempts < 20000:
        attempts += 1
        ln = int(rng.integers(lo, hi + 1))
        if g0 + ln > T - lf - 1:
            break
        dst = int(rng.integers(g0, T - lf - ln))
        if taken[max(dst - 1, 0):dst + ln + 1].any():
            continue
        src = int(rng.integers(0, g0 - ln + 1))
        x[dst:dst + ln] = x[src:src + ln]
        taken[dst:dst + ln] = True
        spans.append((dst, src, ln))
        covered += ln
    # the forced span: its source must leave `margin` tokens after it in the prompt
    src_hi = g0 - lf - margin            # inclusive upper bound of the source start
    if query_count_max > 0:
        prefix = x[:T - lf]
        counts = np.bincount(prefix, minlength=V)
        ok = np.nonzero(counts + lf <= query_count_max)[0]
        # most frequent token whose final count stays within the bound and that
        # occurs at a usable source end
        order = ok[np.argsort(-counts[ok], kind="stable")]
        src = -1
        for tok in order[:64]:
            ends = np.nonzero(x[:src_hi + lf] == tok)[0]
            ends = ends[(ends >= lf - 1) & (ends - lf + 1 <= src_hi)]
            if len(ends):
                src = int(ends[rng.integers(0, len(ends))]) - lf + 1
                break
        if src < 0:
            src = int(rng.integers(0, src_hi + 1))
    else:
        src = int(rng.integers(0, src_hi + 1))
    x[T - lf:] = x[src:src + lf]
    spans.append((T - lf, src, lf))
    src_end = src + lf - 1
    intended = x[src_end + 1:min(src_end + 1 + 64, T - 1)].copy()
    return x, SeqMeta(spans, src_end, intended)


def make_tokens(cfg_or_B, T=None, V=None, s=1.1, plant_frac=0.3, span=(8, 32), seed=0,
                lens=None, tok_stride=None, query_count_max=0):
    """Token batch [B][tok_stride] int32 (padded with -1 past each length), lens, metas.

    Either pass a Config, or B, T, V, ... explicitly.  `lens` may give ragged
    per-sequence lengths (each <= tok_stride).
    """
    if isinstance(cfg_or_B, Config):
        c = cfg_or_B
        B, T, V, s, plant_frac, span, seed = c.B, c.T, c.V, c.zipf_s, c.plant_frac, c.span, c.seed
        query_count_max = c.query_count_max
    else:
        B = cfg_or_B
    lens = np.full(B, T, np.int32) if lens is None else np.asarray(lens, np.int32)
    stride = int(tok_stride or max(int(lens.max()), 1))
    toks = np.full((B, stride), -1, np.int32)
    cdf = zipf_cdf(V, s)
    metas = []
    for b in range(B):
        Tb = int(lens[b])
        x, m = make_sequence(Tb, V, s, plant_frac, span, seed, b, query_count_max, cdf=cdf)
        toks[b, :Tb] = x
        metas.append(m)
    return toks, lens, metas


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (round to nearest even, by torch) and return the bits."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    return (bits.astype(np.uint32) << 16).view(np.float32)


def make_hidden(B: int, T: int, d: int, seed: int, device="cpu", plants=()):
    """Hidden states of one layer, [B][T][d] bf16 torch tensor on `device`.

    Drawn with torch's generator for that device (so values depend on the device
    type), N(0,1) in fp32 then rounded to bf16.  `plants` = ((b, dst_row,
    src_row), ...) makes row dst a bitwise copy of row src.
    """
    import torch
    g = torch.Generator(device=device)
    out = torch.empty((B, T, d), dtype=torch.bfloat16, device=device)
    for b in range(B):
        g.manual_seed(int(np.random.SeedSequence([seed, b, STREAM_HIDDEN]).generate_state(1)[0]))
        out[b].copy_(torch.randn((T, d), generator=g, device=device, dtype=torch.float32))
    for (b, dst, src) in plants:
        out[b, dst].copy_(out[b, src])
    return out


def structured_hidden_plants(lens, metas):
    """Copy the query row T-2 into the row before the planted source."""
    plants = []
    for b, m in enumerate(metas):
        T = int(lens[b])
        if m.query_src_end >= 1 and T >= 3 and m.query_src_end - 1 != T - 2:
            plants.append((b, m.query_src_end - 1, T - 2))
    return tuple(plants)


def make_attn(B: int, R: int, n_keys: int, lens, seed: int, alpha: float = 0.3, metas=None):
    """Attention of query row T-2 over keys, [B][R][n_keys] fp32 (see module doc)."""
    out = np.zeros((B, R, n_keys), np.float32)
    for b in range(B):
        T = int(lens[b])
        vis = max(0, min(T - 1, n_keys))          # keys 0..T-2
        if vis == 0:
            continue
        rng = rng_for(seed, b, STREAM_ATTN)
        g = rng.gamma(alpha, 1.0, size=(R, vis))
        if metas is not None and metas[b].query_src_end >= 1:
            k = metas[b].query_src_end - 1
            if k < vis:
                g[:, k] += g.sum(axis=1)          # one unit of mass after normalising
        g /= g.sum(axis=1, keepdims=True)
        out[b, :, :vis] = g.astype(np.float32)
    return out


def make_logits(B: int, K: int, V: int, seed: int, draft, draft_len, boost: float = 5.0,
                bf16: bool = False):
    """Verification logits [B][K+1][V]: N(0,1) plus +boost on a random prefix of the draft.

    Returns fp32 values, or bf16 bits (uint16) when `bf16`.  Also returns the
    planted prefix length p per sequence.
    """
    draft = np.asarray(draft)
    draft_len = np.asarray(draft_len)
    z = np.empty((B, K + 1, V), np.float32)
    p = np.zeros(B, np.int32)
    for b in range(B):
        rng = rng_for(seed, b, STREAM_LOGITS)
        z[b] = rng.standard_normal((K + 1, V), dtype=np.float32)
        p[b] = int(rng.integers(0, K + 1))
        n = min(int(p[b]), int(draft_len[b]), draft.shape[1] if draft.ndim == 2 else 0)
        for i in range(n):
            t = int(draft[b, i])
            if 0 <= t < V:
                z[b, i, t] += np.float32(boost)
    if bf16:
        return f32_to_bf16_bits(z), p
    return z, p


def make_uniforms(B: int, K: int, seed: int) -> np.ndarray:
    """The draws of sampling verification: fp32 [B][K+1], uniform on [0, 1)."""
    return np.stack([rng_for(seed, b, STREAM_UNIFORMS).random(K + 1, dtype=np.float32)
                     for b in range(B)])


def intended_drafts(metas, K):
    """The K tokens after each planted source, padded with -1 (generator metadata)."""
    B = len(metas)
    d = np.full((B, K), -1, np.int32)
    n = np.zeros(B, np.int32)
    for b, m in enumerate(metas):
        k = min(K, len(m.intended))
        d[b, :k] = m.intended[:k]
        n[b] = k
    return d, n


def to_device_bf16(bits, device):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits, np.uint16).view(np.int16))
    return t.to(device).view(torch.bfloat16)


def make_workload(cfg: Config, device, structured: bool = True, plant_draft=None):
    """All inputs of one configuration.

    tokens/lens (host int32), hidden (device bf16 [B][T][d] or None), attn
    (host fp32 [B][R][T] or None).  Logits are made by `logits_for(w, draft,
    draft_len)` once the draft to plant is known; with `plant_draft` given
    here (a (draft, draft_len) pair) they are made at once.
    """
    toks, lens, metas = make_tokens(cfg)
    w = dict(cfg=cfg, tokens=toks, lens=lens, metas=metas, hidden=None, attn=None, logits=None)
    if cfg.rank in ("hidden", "both"):
        plants = structured_hidden_plants(lens, metas) if structured else ()
        w["hidden"] = make_hidden(cfg.B, cfg.T, cfg.d, cfg.seed, device=device, plants=plants)
    if cfg.rank in ("attn", "both"):
        w["attn"] = make_attn(cfg.B, cfg.R, cfg.T, lens, cfg.seed,
                              metas=metas if structured else None)
    if plant_draft is not None:
        w["logits"] = logits_for(w, *plant_draft)
    return w


def logits_for(w, draft, draft_len):
    c = w["cfg"]
    z, _ = make_logits(c.B, c.K, c.V, c.seed, draft, draft_len, bf16=(c.logits == "bf16"))
    return z


# ------------------------------------------------------------ decoding tasks
@dataclasses.dataclass(frozen=True)
class DecodeTask:
    """A multi-step decoding run: B target sequences of length T whose last
    quarter is generated step by step, starting from the first three quarters
    (the prompt); a stated fraction of the generated part copies spans of the
    prompt (input-guided generation, Sec. 5.1), or, for a sectioned task
    (header > 0), the prompt is a run of sections and the generated part an
    edited copy of consecutive ones (span then gives the body lengths)."""
    name: str
    B: int
    T: int
    V: int
    zipf_s: float
    plant_frac: float
    span: tuple
    d: int
    K: int
    seed: int
    window: int = 4       # hidden state of position p: decaying sum over x[p-window+1 .. p]
    decay: float = 0.5
    noise: float = 0.25
    edit_rate: float = 0.0   # sectioned tasks: chance that a copied token is replaced
    header: int = 0          # > 0: a sectioned task (make_sections) with a header this long


DECODE_TASKS = {
    # the paper's input sizes (App. B) with a highly overlapping output, K = 10
    "b1_t1024_copy60_k10": DecodeTask("b1_t1024_copy60_k10", 1, 1024, 32000, 1.1, 0.6, (8, 64),
                                      4096, 10, 21),
    # a batch of eight, longer contexts, K = 16
    "b8_t4096_copy50_k16": DecodeTask("b8_t4096_copy50_k16", 8, 4096, 32000, 1.1, 0.5, (8, 64),
                                      4096, 16, 22),
    # Sectioned documents copied with edits, the situation of the Fig. 3
    # caption.  The input is a run of sections that all start with the same
    # 8-token header (as functions or lines of code start alike) followed by
    # 24-56 Zipf tokens; the output copies consecutive sections from a random
    # one, one copied token in ten replaced (an edit).  The hidden states carry
    # a decaying window of the last 32 tokens.  After an edit, the drafter has
    # to find its place again: the last tokens, often header tokens, occur in
    # every section, and prompt lookup takes the earliest of the equally long
    # matches, while the hidden state still resembles the one at the true source.
    "b1_t1024_sections_edit10_k10": DecodeTask("b1_t1024_sections_edit10_k10", 1, 1024, 32000,
                                               1.1, 0.0, (24, 56), 4096, 10, 23, window=32,
                                               decay=0.85, edit_rate=0.1, header=8),
    "b8_t4096_sections_edit10_k16": DecodeTask("b8_t4096_sections_edit10_k16", 8, 4096, 32000,
                                               1.1, 0.0, (24, 56), 4096, 16, 24, window=32,
                                               decay=0.85, edit_rate=0.1, header=8),
}


def make_sections(task: "DecodeTask") -> np.ndarray:
    """Targets [B][T] of a sectioned task: the first T - T/4 tokens are sections
    (the header, then a body of task.span[0]..task.span[1] Zipf tokens); the last
    T/4 copy consecutive sections from a random one, with each copied token
    replaced by a fresh Zipf token with probability task.edit_rate."""
    cdf = zipf_cdf(task.V, task.zipf_s)
    T = task.T
    P = T - T // 4
    out = np.zeros((task.B, T), np.int32)
    for b in range(task.B):
        rng = rng_for(task.seed, b, STREAM_SECTIONS)
        header = zipf_tokens(rng, task.header, cdf)
        starts, x = [], []
        while len(x) < P:
            starts.append(len(x))
            body = int(rng.integers(task.span[0], task.span[1] + 1))
            x.extend(header.tolist())
            x.extend(zipf_tokens(rng, body, cdf).tolist())
        x = x[:P]
        edit = rng_for(task.seed, b, STREAM_EDIT)
        src = starts[int(rng.integers(0, max(1, len(starts) - 8)))]
        gen = []
        while len(gen) < T - P:
            t = x[src % P]
            if edit.random() < task.edit_rate:
                t = int(zipf_tokens(edit, 1, cdf)[0])
            gen.append(t)
            src += 1
        out[b] = np.array(x + gen, np.int32)
    return out


def make_context_hidden(tokens: np.ndarray, d: int, seed: int, window: int = 4,
                        decay: float = 0.5, noise: float = 0.25, device="cpu"):
    """Hidden states [B][T][d] bf16 for the loop: H[p] = sum_k decay^k E[x[p-k]]
    (k < window, p-k >= 0) plus N(0, noise^2), E a Gaussian table over token ids
    (hashed to 4096 rows).  Positions whose last few tokens agree get similar
    rows, the property the paper's hidden-state ranking relies on (Sec. 4.2.2)."""
    import torch
    B, T = tokens.shape
    g = torch.Generator(device=device)
    g.manual_seed(int(np.random.SeedSequence([seed, 0, STREAM_CONTEXT]).generate_state(1)[0]))
    E = torch.randn((4096, d), generator=g, device=device)
    ids = torch.from_numpy(np.where(tokens >= 0, tokens, 0) % 4096).to(device).long()
    out = torch.empty((B, T, d), dtype=torch.bfloat16, device=device)
    for b in range(B):
        h = torch.zeros((T, d), device=device)
        for k in range(window):
            h[k:] += (decay ** k) * E[ids[b, :T - k]]
        h += noise * torch.randn((T, d), generator=g, device=device)
        out[b] = h.to(torch.bfloat16)
    return out


def make_decode_task(task: DecodeTask, device="cpu"):
    """Targets (host int32 [B][T]), the prompt length per sequence (host int32),
    and the loop's hidden states (device bf16 [B][T][d])."""
    if task.header > 0:
        toks, metas = make_sections(task), None
    else:
        toks, lens, metas = make_tokens(task.B, task.T, task.V, task.zipf_s, task.plant_frac,
                                        task.span, task.seed)
    start = np.full(task.B, task.T - task.T // 4, np.int32)
    hidden = make_context_hidden(toks, task.d, task.seed, task.window, task.decay, task.noise,
                                 device)
    return dict(task=task, target=toks, start=start, hidden=hidden, metas=metas)


class TargetModel:
    """Stand-in for the target model's forward pass over context + draft (the
    forward pass itself is outside the drafting step).  Row i of its logits is
    the distribution at position lens[b] + i: N(0, 1) noise, fixed per run,
    with +boost at the target token of that position, so that its greedy
    continuation of any prefix of the target is the target.  The logits buffer
    is patched in place between calls rather than rebuilt."""

    def __init__(self, target, K: int, V: int, seed: int, device="cpu", boost: float = 10.0):
        import torch
        self.device = device
        self.target = torch.as_tensor(target, device=device).long()
        B, self.T = self.target.shape
        g = torch.Generator(device=device)
        g.manual_seed(int(np.random.SeedSequence([seed, 0, STREAM_MODEL]).generate_state(1)[0]))
        self.base = torch.randn((B, K + 1, V), generator=g, device=device)
        self.buf = self.base.clone()
        self.boost = float(boost)
        self.prev = None
        self.offs = torch.arange(K + 1, device=device)

    def target_tokens(self, lens):
        import torch
        pos = (torch.as_tensor(lens, device=self.device).long()[:, None] + self.offs)
        return self.target.gather(1, pos.clamp(max=self.T - 1))

    def logits(self, lens):
        """The logits for the drafts of sequences at lengths `lens` (device)."""
        if self.prev is not None:
            self.buf.scatter_(2, self.prev, self.base.gather(2, self.prev))
        tok = self.target_tokens(lens)[:, :, None]
        self.buf.scatter_(2, tok, self.base.gather(2, tok) + self.boost)
        self.prev = tok
        return self.buf
