"""PLD+ drafting step on AMD Instinct MI355X (gfx950): Python binding of libpld.so.

The calls carry the names and argument order of the C ABI in include/pld.h and
only marshal arguments: every step runs in the HIP kernels of libpld.so.  Pass
device tensors (torch is used for device memory and streams only); each call
enqueues on ``stream`` (default: torch's current stream) and returns without
synchronising.  A non-zero status from the library raises :class:`PLDError`.

Method: arXiv 2412.01447 -- occurrences of the last token (Eq. 1), ranked by
hidden-state cosine (Eq. 2) or aggregated attention (Eq. 3), the K tokens after
the best occurrence as the draft (Sec. 4.3), greedy verification (Sec. 3, 4.4).
"""
import ctypes
import os

__all__ = [
    "PLDError", "PLD_F32", "PLD_BF16", "PLD_AGG_SUM", "PLD_AGG_MAX", "library_path",
    "pld_version", "pld_status_string", "pld_workspace_bytes", "pld_find_scratch_bytes",
    "pld_find_candidates",
    "pld_rank_hidden", "pld_rank_attn", "pld_emit_draft", "pld_verify_greedy",
    "pld_verify_greedy_noalloc", "NOALLOC_MAX_KEYS",
    "pld_draft_hidden", "pld_draft_attn", "pld_draft_workspace_bytes", "DRAFT_MAX_TOK_STRIDE",
    "DRAFT_MAX_PART", "pld_score_hidden", "pld_score_both",
    "pld_score_attn", "pld_select_best", "pld_select_draft", "pld_verify_argmax",
    "pld_verify_accept",
    "pld_verify_sample", "pld_verify_sample_workspace_bytes", "pld_verify_sample_stats",
    "pld_verify_sample_finish", "PLD_MAX_SAMPLE_ROWS", "pld_select_prefix", "pld_commit", "pld_accept_commit",
    "PLD_MAX_MATCH",
]

PLD_OK, PLD_ERR_INVALID, PLD_ERR_ALIGN, PLD_ERR_WORKSPACE, PLD_ERR_LAUNCH, PLD_ERR_SCRATCH = range(6)
NOALLOC_MAX_KEYS = 65536        # pld_verify_greedy_noalloc: B*(K+1) limit
PLD_F32, PLD_BF16 = 0, 1
PLD_AGG_SUM, PLD_AGG_MAX = 0, 1
PLD_MAX_NGRAM, PLD_MAX_HIDDEN, PLD_MAX_BATCH, PLD_MAX_DRAFT_SPLIT = 8, 16384, 4096, 1024
PLD_MAX_SAMPLE_ROWS = 16384
PLD_MAX_MATCH = 1024
DRAFT_MAX_TOK_STRIDE = 8192     # one-call drafting, one block per sequence (S = 1)
DRAFT_MAX_PART = 8192           # one-call drafting, S > 1: positions per block

_HERE = os.path.dirname(os.path.abspath(__file__))
library_path = os.path.join(_HERE, "libpld.so")
_lib = None

_vp, _i64, _int, _sz, _f32 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_size_t,
                              ctypes.c_float)

_SIGNATURES = {
    "pld_version": ([], _int),
    "pld_status_string": ([_int], ctypes.c_char_p),
    "pld_workspace_bytes": ([_int, _int], _sz),
    "pld_draft_workspace_bytes": ([_int, _int], _sz),
    "pld_verify_sample_workspace_bytes": ([_int, _int, _int, _int], _sz),
    "pld_find_scratch_bytes": ([_int, _i64], _sz),
    "pld_find_candidates": ([_vp, _i64, _vp, _int, _int, _int, _vp, _i64, _vp, _vp, _vp, _sz, _vp],
                            _int),
    "pld_rank_hidden": ([_vp, _i64, _i64, _i64, _int, _vp, _vp, _i64, _vp, _int, _f32, _vp, _vp,
                         _vp, _vp, _sz, _vp], _int),
    "pld_rank_attn": ([_vp, _i64, _i64, _i64, _int, _int, _vp, _vp, _i64, _vp, _int, _f32, _vp,
                       _vp, _vp, _vp, _sz, _vp], _int),
    "pld_emit_draft": ([_vp, _i64, _vp, _vp, _int, _int, _vp, _vp, _vp], _int),
    "pld_verify_greedy": ([_vp, _int, _i64, _i64, _int, _int, _vp, _vp, _int, _vp, _vp, _vp, _vp,
                           _sz, _vp], _int),
    "pld_verify_greedy_noalloc": ([_vp, _int, _i64, _i64, _int, _int, _vp, _vp, _int, _vp, _vp,
                                   _vp, _vp], _int),
    "pld_score_hidden": ([_vp, _i64, _i64, _i64, _int, _vp, _vp, _i64, _vp, _int, _f32, _vp, _vp,
                          _sz, _vp], _int),
    "pld_score_attn": ([_vp, _i64, _i64, _i64, _int, _int, _vp, _vp, _i64, _vp, _int, _f32, _vp,
                        _vp, _sz, _vp], _int),
    "pld_score_both": ([_vp, _i64, _i64, _i64, _int, _vp, _i64, _i64, _i64, _int, _int, _vp, _vp,
                        _i64, _vp, _int, _f32, _f32, _vp, _vp, _vp, _sz, _vp, _sz, _vp], _int),
    "pld_select_best": ([_int, _vp, _vp, _vp, _sz, _vp], _int),
    "pld_select_draft": ([_vp, _i64, _vp, _int, _int, _vp, _vp, _vp, _vp, _vp, _sz, _vp, _sz, _vp,
                          _vp, _vp], _int),
    "pld_verify_argmax": ([_vp, _int, _i64, _i64, _int, _int, _vp, _int, _vp, _sz, _vp], _int),
    "pld_verify_accept": ([_vp, _vp, _int, _int, _vp, _vp, _vp, _vp, _sz, _vp], _int),
    "pld_verify_sample": ([_vp, _int, _i64, _i64, _int, _int, _vp, _vp, _int, ctypes.c_double, _vp,
                           _i64, _vp, _vp, _vp, _vp, _vp, _sz, _vp], _int),
    "pld_verify_sample_stats": ([_vp, _int, _i64, _i64, _int, _int, _vp, _int, ctypes.c_double,
                                 _vp, _sz, _vp], _int),
    "pld_verify_sample_finish": ([_vp, _int, _i64, _i64, _int, _int, _vp, _vp, _int,
                                  ctypes.c_double, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _sz, _vp],
                                 _int),
    "pld_select_prefix": ([_vp, _i64, _vp, _vp, _i64, _vp, _int, _int, _vp, _vp, _vp, _vp], _int),
    "pld_commit": ([_vp, _i64, _vp, _vp, _vp, _vp, _int, _int, _vp, _vp], _int),
    "pld_accept_commit": ([_vp, _vp, _int, _int, _vp, _vp, _vp, _vp, _i64, _vp, _vp, _vp, _vp,
                           _sz, _vp], _int),
    "pld_draft_hidden": ([_vp, _i64, _vp, _int, _int, _int, _vp, _i64, _i64, _i64, _int, _f32, _int,
                          _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _int, _vp, _sz, _vp],
                         _int),
    "pld_draft_attn": ([_vp, _i64, _vp, _int, _int, _int, _vp, _i64, _i64, _i64, _int, _int, _f32,
                        _int, _vp, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _int, _vp, _sz, _vp],
                       _int),
}


class PLDError(RuntimeError):
    def __init__(self, name, status):
        super().__init__(f"{name}: {_load().pld_status_string(status).decode()} (status {status})")
        self.status = status


def _load():
    """Open libpld.so; fail loudly when it has not been built (no fallback exists)."""
    global _lib
    if _lib is None:
        if not os.path.exists(library_path):
            raise ImportError(f"{library_path} is missing: build it with "
                              "`python -c 'import __graft_entry__ as g; g.build()'`")
        lib = ctypes.CDLL(library_path)
        for name, (args, res) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.argtypes = args
            fn.restype = res
        _lib = lib
    return _lib


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _need(t, dtype, name, dims):
    if t.dtype != dtype or t.dim() != dims or not t.is_cuda:
        raise TypeError(f"{name}: expected a {dims}-d {dtype} device tensor, got "
                        f"{tuple(t.shape)} {t.dtype} on {t.device}")
    if t.stride(-1) != 1:
        raise TypeError(f"{name}: the last dimension must be contiguous")


def _call(name, *args):
    rc = getattr(_load(), name)(*args)
    if rc != PLD_OK:
        raise PLDError(name, rc)


class Prepared:
    """One library call with its arguments marshalled once.  Calling it only
    enqueues the kernels (the lowest-overhead way to issue a step from Python);
    the tensors it points to must stay alive and in place."""
    __slots__ = ("name", "fn", "args")

    def __init__(self, name, args):
        self.name = name
        self.fn = getattr(_load(), name)
        conv = []
        for a, t in zip(args, self.fn.argtypes):
            conv.append(a if isinstance(a, (ctypes.c_void_p,)) or a is None else t(a))
        self.args = tuple(conv)

    def __call__(self):
        rc = self.fn(*self.args)
        if rc != PLD_OK:
            raise PLDError(self.name, rc)


def _run(name, args, prepare):
    if prepare:
        return Prepared(name, args)
    _call(name, *args)


def pld_version():
    return _load().pld_version()


def pld_status_string(status):
    return _load().pld_status_string(status).decode()


def pld_workspace_bytes(B, K):
    return int(_load().pld_workspace_bytes(B, K))


def pld_draft_workspace_bytes(B, blocks_per_seq):
    return int(_load().pld_draft_workspace_bytes(B, blocks_per_seq))


def pld_verify_sample_workspace_bytes(B, K, V, dtype):
    return int(_load().pld_verify_sample_workspace_bytes(B, K, V, dtype))


def pld_find_scratch_bytes(B, tok_stride):
    return int(_load().pld_find_scratch_bytes(B, tok_stride))


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def pld_find_candidates(tokens, lens, ngram_min, ngram_max, cand_pos, cand_count, ngram_used,
                        scratch=None, stream=None, prepare=False):
    """tokens int32 [B][tok_stride]; writes cand_pos [B][cap], cand_count [B], ngram_used [B]."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    B = tokens.shape[0]
    return _run("pld_find_candidates", (_ptr(tokens), tokens.stride(0), _ptr(lens), B, ngram_min,
          ngram_max, _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), _ptr(ngram_used),
          _ptr(scratch), _nbytes(scratch), _stream(stream),), prepare)


def pld_rank_hidden(hidden, lens, cand_pos, cand_count, best_pos, best_score, workspace,
                    threshold=float("-inf"), scores=None, stream=None, prepare=False):
    """hidden bf16 [B][n_rows][d]; writes best_pos [B], best_score [B] and optionally scores."""
    import torch
    _need(hidden, torch.bfloat16, "hidden", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    B, n_rows, d = hidden.shape
    return _run("pld_rank_hidden", (_ptr(hidden), hidden.stride(0), hidden.stride(1), n_rows, d,
          _ptr(lens), _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), B, float(threshold),
          _ptr(scores), _ptr(best_pos), _ptr(best_score), _ptr(workspace),
          _nbytes(workspace), _stream(stream),), prepare)


def pld_rank_attn(attn, lens, cand_pos, cand_count, best_pos, best_score, workspace,
                  agg=PLD_AGG_SUM, threshold=float("-inf"), scores=None, stream=None, prepare=False):
    """attn fp32 [B][R][n_keys] (query row T-2 per selected head); agg SUM or MAX."""
    import torch
    _need(attn, torch.float32, "attn", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    B, R, n_keys = attn.shape
    return _run("pld_rank_attn", (_ptr(attn), attn.stride(0), attn.stride(1), n_keys, R, int(agg),
          _ptr(lens), _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), B, float(threshold),
          _ptr(scores), _ptr(best_pos), _ptr(best_score), _ptr(workspace),
          _nbytes(workspace), _stream(stream),), prepare)


def pld_emit_draft(tokens, lens, best_pos, K, draft, draft_len, stream=None, prepare=False):
    """Writes draft [B][K] (padded with -1) and draft_len [B]."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    _need(draft, torch.int32, "draft", 2)
    if draft.shape[1] != K or draft.stride(0) != K:
        raise TypeError("draft must be a contiguous [B][K] tensor")
    return _run("pld_emit_draft", (_ptr(tokens), tokens.stride(0), _ptr(lens), _ptr(best_pos),
          tokens.shape[0], K, _ptr(draft), _ptr(draft_len), _stream(stream),), prepare)


def pld_verify_greedy(logits, draft, draft_len, accept_len, out_tokens, out_count, workspace,
                      stream=None, prepare=False):
    """logits fp32 or bf16 [B][K+1][V]; writes accept_len [B], out_tokens [B][K+1], out_count [B]."""
    import torch
    if logits.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("logits must be float32 or bfloat16")
    _need(logits, logits.dtype, "logits", 3)
    B, K1, V = logits.shape
    K = K1 - 1
    if draft.shape != (B, K) or draft.stride(0) != K:
        raise TypeError("draft must be a contiguous [B][K] tensor")
    if out_tokens.shape != (B, K1) or out_tokens.stride(0) != K1:
        raise TypeError("out_tokens must be a contiguous [B][K+1] tensor")
    dtype = PLD_F32 if logits.dtype == torch.float32 else PLD_BF16
    return _run("pld_verify_greedy", (_ptr(logits), dtype, logits.stride(0), logits.stride(1), V, K,
          _ptr(draft), _ptr(draft_len), B, _ptr(accept_len), _ptr(out_tokens), _ptr(out_count),
          _ptr(workspace), _nbytes(workspace), _stream(stream),), prepare)


def pld_verify_greedy_noalloc(logits, draft, draft_len, accept_len, out_tokens, out_count,
                              stream=None, prepare=False):
    """pld_verify_greedy without a workspace: the row maxima live in the library's static
    per-GPU array (B*(K+1) <= NOALLOC_MAX_KEYS); calls on one GPU must not overlap."""
    import torch
    if logits.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("logits must be float32 or bfloat16")
    _need(logits, logits.dtype, "logits", 3)
    B, K1, V = logits.shape
    K = K1 - 1
    if draft.shape != (B, K) or draft.stride(0) != K:
        raise TypeError("draft must be a contiguous [B][K] tensor")
    if out_tokens.shape != (B, K1) or out_tokens.stride(0) != K1:
        raise TypeError("out_tokens must be a contiguous [B][K+1] tensor")
    dtype = PLD_F32 if logits.dtype == torch.float32 else PLD_BF16
    return _run("pld_verify_greedy_noalloc", (_ptr(logits), dtype, logits.stride(0),
          logits.stride(1), V, K, _ptr(draft), _ptr(draft_len), B, _ptr(accept_len),
          _ptr(out_tokens), _ptr(out_count), _stream(stream),), prepare)


def pld_verify_sample(logits, draft, draft_len, temperature, uniforms, accept_len, out_tokens,
                      out_count, workspace, row_sample=None, stream=None, prepare=False):
    """Sampling verification: y_i drawn from softmax(logits / temperature) at uniforms [B][>=K+1]
    (fp32); outputs as pld_verify_greedy, plus the per-row samples when row_sample is given."""
    B, K, V, dtype = _sample_shapes(logits, draft, uniforms, out_tokens, row_sample)
    return _run("pld_verify_sample", (_ptr(logits), dtype, logits.stride(0), logits.stride(1), V, K,
          _ptr(draft), _ptr(draft_len), B, float(temperature), _ptr(uniforms), uniforms.stride(0),
          _ptr(accept_len), _ptr(out_tokens), _ptr(out_count), _ptr(row_sample), _ptr(workspace),
          _nbytes(workspace), _stream(stream),), prepare)


def pld_select_prefix(tokens, lens, cand_pos, cand_count, best_pos, best_score, max_match,
                      scores=None, stream=None, prepare=False):
    """Prompt lookup's selection over the occurrence lists: longest matching prefix (up to
    max_match tokens), earliest among equals; writes best_pos [B], best_score [B]."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    return _run("pld_select_prefix", (_ptr(tokens), tokens.stride(0), _ptr(lens), _ptr(cand_pos),
          cand_pos.stride(0), _ptr(cand_count), tokens.shape[0], int(max_match), _ptr(scores),
          _ptr(best_pos), _ptr(best_score), _stream(stream),), prepare)


def pld_commit(tokens, lens, out_tokens, out_count, limit=None, stats=None, stream=None,
               prepare=False):
    """Appends out_tokens[b][:out_count[b]] to tokens[b] (up to limit[b]), advances lens and
    adds (emitted, steps) to stats [B][2] int64 when given."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    B, K1 = out_tokens.shape
    if out_tokens.stride(0) != K1:
        raise TypeError("out_tokens must be a contiguous [B][K+1] tensor")
    if stats is not None and (stats.dtype != torch.int64 or tuple(stats.shape) != (B, 2)
                              or not stats.is_contiguous()):
        raise TypeError("stats must be a contiguous int64 [B][2] tensor")
    return _run("pld_commit", (_ptr(tokens), tokens.stride(0), _ptr(lens), _ptr(limit),
          _ptr(out_tokens), _ptr(out_count), B, K1 - 1, _ptr(stats), _stream(stream),), prepare)


def pld_accept_commit(draft, draft_len, accept_len, out_tokens, out_count, tokens, lens, workspace,
                      limit=None, stats=None, stream=None, prepare=False):
    """pld_verify_accept then pld_commit in one launch: the accepted length and emitted
    tokens from the row maxima in the workspace, appended to tokens[b] (up to limit[b]),
    lens advanced, (emitted, steps) added to stats [B][2] int64 when given."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    B, K = draft.shape
    if draft.stride(0) != K or out_tokens.shape != (B, K + 1) or out_tokens.stride(0) != K + 1:
        raise TypeError("draft [B][K] and out_tokens [B][K+1] must be contiguous")
    if stats is not None and (stats.dtype != torch.int64 or tuple(stats.shape) != (B, 2)
                              or not stats.is_contiguous()):
        raise TypeError("stats must be a contiguous int64 [B][2] tensor")
    return _run("pld_accept_commit", (
        _ptr(draft), _ptr(draft_len), B, K, _ptr(accept_len), _ptr(out_tokens), _ptr(out_count),
        _ptr(tokens), tokens.stride(0), _ptr(lens), _ptr(limit), _ptr(stats), _ptr(workspace),
        _nbytes(workspace), _stream(stream),), prepare)


def pld_draft_hidden(tokens, lens, ngram_min, ngram_max, hidden, K, cand_pos, cand_count,
                     ngram_used, best_pos, best_score, draft, draft_len, threshold=float("-inf"),
                     scores=None, blocks_per_seq=1, workspace=None, stream=None, prepare=False):
    """find + hidden-state ranking + emit in one call (blocks_per_seq 1: tok_stride <= 8192;
    more: a workspace of pld_draft_workspace_bytes(B, blocks_per_seq) bytes)."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    _need(hidden, torch.bfloat16, "hidden", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    if draft.shape[1] != K or draft.stride(0) != K:
        raise TypeError("draft must be a contiguous [B][K] tensor")
    B, n_rows, d = hidden.shape
    return _run("pld_draft_hidden", (
        _ptr(tokens), tokens.stride(0), _ptr(lens), tokens.shape[0], ngram_min, ngram_max,
        _ptr(hidden), hidden.stride(0), hidden.stride(1), n_rows, d, float(threshold), K,
        _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), _ptr(ngram_used), _ptr(scores),
        _ptr(best_pos), _ptr(best_score), _ptr(draft), _ptr(draft_len), int(blocks_per_seq),
        _ptr(workspace), _nbytes(workspace), _stream(stream)), prepare)


def pld_draft_attn(tokens, lens, ngram_min, ngram_max, attn, K, cand_pos, cand_count, ngram_used,
                   best_pos, best_score, draft, draft_len, agg=PLD_AGG_SUM,
                   threshold=float("-inf"), scores=None, blocks_per_seq=1, workspace=None,
                   stream=None, prepare=False):
    """find + attention ranking + emit in one call (blocks_per_seq 1: tok_stride <= 8192;
    more: a workspace of pld_draft_workspace_bytes(B, blocks_per_seq) bytes)."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    _need(attn, torch.float32, "attn", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    if draft.shape[1] != K or draft.stride(0) != K:
        raise TypeError("draft must be a contiguous [B][K] tensor")
    B, R, n_keys = attn.shape
    return _run("pld_draft_attn", (
        _ptr(tokens), tokens.stride(0), _ptr(lens), tokens.shape[0], ngram_min, ngram_max,
        _ptr(attn), attn.stride(0), attn.stride(1), n_keys, R, int(agg), float(threshold), K,
        _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), _ptr(ngram_used), _ptr(scores),
        _ptr(best_pos), _ptr(best_score), _ptr(draft), _ptr(draft_len), int(blocks_per_seq),
        _ptr(workspace), _nbytes(workspace), _stream(stream)), prepare)


def pld_score_hidden(hidden, lens, cand_pos, cand_count, workspace, threshold=float("-inf"),
                     scores=None, stream=None, prepare=False):
    """Scoring half of pld_rank_hidden: per-sequence best keys into the workspace."""
    import torch
    _need(hidden, torch.bfloat16, "hidden", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    B, n_rows, d = hidden.shape
    return _run("pld_score_hidden", (_ptr(hidden), hidden.stride(0), hidden.stride(1), n_rows, d,
          _ptr(lens), _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), B, float(threshold),
          _ptr(scores), _ptr(workspace), _nbytes(workspace), _stream(stream),), prepare)


def pld_score_attn(attn, lens, cand_pos, cand_count, workspace, agg=PLD_AGG_SUM,
                   threshold=float("-inf"), scores=None, stream=None, prepare=False):
    """Scoring half of pld_rank_attn."""
    import torch
    _need(attn, torch.float32, "attn", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    B, R, n_keys = attn.shape
    return _run("pld_score_attn", (_ptr(attn), attn.stride(0), attn.stride(1), n_keys, R, int(agg),
          _ptr(lens), _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), B, float(threshold),
          _ptr(scores), _ptr(workspace), _nbytes(workspace), _stream(stream),), prepare)


def pld_score_both(hidden, attn, lens, cand_pos, cand_count, workspace_h, workspace_a,
                   agg=PLD_AGG_SUM, threshold_h=float("-inf"), threshold_a=float("-inf"),
                   scores_h=None, scores_a=None, stream=None, prepare=False):
    """pld_score_hidden and pld_score_attn of the same occurrences in one launch."""
    import torch
    _need(hidden, torch.bfloat16, "hidden", 3)
    _need(attn, torch.float32, "attn", 3)
    _need(cand_pos, torch.int32, "cand_pos", 2)
    B, n_rows, d = hidden.shape
    _, R, n_keys = attn.shape
    return _run("pld_score_both", (
        _ptr(hidden), hidden.stride(0), hidden.stride(1), n_rows, d,
        _ptr(attn), attn.stride(0), attn.stride(1), n_keys, R, int(agg),
        _ptr(lens), _ptr(cand_pos), cand_pos.stride(0), _ptr(cand_count), B,
        float(threshold_h), float(threshold_a), _ptr(scores_h), _ptr(scores_a),
        _ptr(workspace_h), _nbytes(workspace_h), _ptr(workspace_a), _nbytes(workspace_a),
        _stream(stream)), prepare)


def pld_select_best(B, best_pos, best_score, workspace, stream=None, prepare=False):
    """Selection half of the ranking calls: keys -> best_pos / best_score."""
    return _run("pld_select_best", (B, _ptr(best_pos), _ptr(best_score), _ptr(workspace),
          _nbytes(workspace), _stream(stream),), prepare)


def pld_select_draft(tokens, lens, K, best_pos, best_score, draft, draft_len, workspace,
                     aux_workspace=None, aux_best_pos=None, aux_best_score=None, stream=None,
                     prepare=False):
    """Selection and draft in one launch: keys in `workspace` -> best_pos / best_score and
    draft [B][K] / draft_len [B]; a second ranking's keys in `aux_workspace` (optional) ->
    aux_best_pos / aux_best_score."""
    import torch
    _need(tokens, torch.int32, "tokens", 2)
    _need(draft, torch.int32, "draft", 2)
    if draft.shape[1] != K or draft.stride(0) != K:
        raise TypeError("draft must be a contiguous [B][K] tensor")
    return _run("pld_select_draft", (_ptr(tokens), tokens.stride(0), _ptr(lens), tokens.shape[0],
          K, _ptr(best_pos), _ptr(best_score), _ptr(draft), _ptr(draft_len), _ptr(workspace),
          _nbytes(workspace), _ptr(aux_workspace), _nbytes(aux_workspace), _ptr(aux_best_pos),
          _ptr(aux_best_score), _stream(stream),), prepare)


def pld_verify_argmax(logits, draft_len, workspace, stream=None, prepare=False):
    """Row maxima of the K+1 logits rows (rows past each draft skipped) into the workspace."""
    import torch
    if logits.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("logits must be float32 or bfloat16")
    _need(logits, logits.dtype, "logits", 3)
    B, K1, V = logits.shape
    dtype = PLD_F32 if logits.dtype == torch.float32 else PLD_BF16
    return _run("pld_verify_argmax", (_ptr(logits), dtype, logits.stride(0), logits.stride(1), V, K1 - 1,
          _ptr(draft_len), B, _ptr(workspace), _nbytes(workspace), _stream(stream),), prepare)


def _sample_shapes(logits, draft, uniforms, out_tokens, row_sample):
    import torch
    if logits.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("logits must be float32 or bfloat16")
    _need(logits, logits.dtype, "logits", 3)
    B, K1, V = logits.shape
    if draft is not None and (draft.shape != (B, K1 - 1) or draft.stride(0) != K1 - 1):
        raise TypeError("draft must be a contiguous [B][K] tensor")
    if uniforms is not None:
        _need(uniforms, torch.float32, "uniforms", 2)
        if uniforms.shape[0] != B or uniforms.shape[1] < K1:
            raise TypeError("uniforms must be [B][>=K+1]")
    if out_tokens is not None and (out_tokens.shape != (B, K1) or out_tokens.stride(0) != K1):
        raise TypeError("out_tokens must be a contiguous [B][K+1] tensor")
    if row_sample is not None and (row_sample.shape != (B, K1) or row_sample.stride(0) != K1):
        raise TypeError("row_sample must be a contiguous [B][K+1] tensor")
    return B, K1 - 1, V, PLD_F32 if logits.dtype == torch.float32 else PLD_BF16


def pld_verify_sample_stats(logits, draft_len, temperature, workspace, stream=None,
                            prepare=False):
    """Streaming half of sampling verification: per-segment (max, mass) of the rows
    i <= draft_len into the workspace."""
    B, K, V, dtype = _sample_shapes(logits, None, None, None, None)
    return _run("pld_verify_sample_stats", (_ptr(logits), dtype, logits.stride(0),
          logits.stride(1), V, K, _ptr(draft_len), B, float(temperature), _ptr(workspace),
          _nbytes(workspace), _stream(stream),), prepare)


def pld_verify_sample_finish(logits, draft, draft_len, temperature, uniforms, accept_len,
                             out_tokens, out_count, workspace, row_sample=None, stream=None,
                             prepare=False):
    """Second half: the sampled tokens from the statistics, then the acceptance."""
    B, K, V, dtype = _sample_shapes(logits, draft, uniforms, out_tokens, row_sample)
    return _run("pld_verify_sample_finish", (_ptr(logits), dtype, logits.stride(0),
          logits.stride(1), V, K, _ptr(draft), _ptr(draft_len), B, float(temperature),
          _ptr(uniforms), uniforms.stride(0), _ptr(accept_len), _ptr(out_tokens), _ptr(out_count),
          _ptr(row_sample), _ptr(workspace), _nbytes(workspace), _stream(stream),), prepare)


def pld_verify_accept(draft, draft_len, accept_len, out_tokens, out_count, workspace,
                      stream=None, prepare=False):
    """Accepted length and emitted tokens from the row maxima in the workspace."""
    B, K = draft.shape
    if draft.stride(0) != K or out_tokens.shape != (B, K + 1) or out_tokens.stride(0) != K + 1:
        raise TypeError("draft [B][K] and out_tokens [B][K+1] must be contiguous")
    return _run("pld_verify_accept", (_ptr(draft), _ptr(draft_len), B, K, _ptr(accept_len),
          _ptr(out_tokens), _ptr(out_count), _ptr(workspace), _nbytes(workspace),
          _stream(stream),), prepare)
