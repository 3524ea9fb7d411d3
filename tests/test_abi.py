"""The C ABI library loads, exports what include/pld.h declares, and validates
arguments on the host (CPU only; no kernel is ever launched here).

Every error-path call below carries at least one argument the host check
rejects, so it returns before any HIP call.  Those calls use placeholder
pointers, so they run only where no GPU is visible; on a machine with a GPU the same
paths are exercised with real device buffers by the GPU tests.
"""
import ctypes
import math
import os
import re
import subprocess

import pytest

import paper_2412_01447_amd as pld

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pld.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pld_\w+)\s*\(", text)))


def _no_gpu():
    import torch
    return torch.cuda.device_count() == 0


def test_header_declares_the_five_calls():
    names = _declared()
    for n in ("pld_find_candidates", "pld_rank_hidden", "pld_rank_attn", "pld_emit_draft",
              "pld_verify_greedy", "pld_workspace_bytes", "pld_status_string", "pld_version"):
        assert n in names


def test_library_exports_every_declared_symbol():
    assert os.path.exists(pld.library_path), "libpld.so not built"
    out = subprocess.run(["nm", "-D", "--defined-only", pld.library_path], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (pld_\w+)$", out, flags=re.M))
    missing = [n for n in _declared() if n not in exported]
    assert not missing, missing
    lib = pld._load()
    for n in _declared():
        assert hasattr(lib, n)
        assert hasattr(pld, n), f"binding lacks {n}"


def test_header_compiles_as_c_and_cpp(tmp_path):
    """include/pld.h is self-contained: it compiles alone as strict C99 and as C++17."""
    inc = os.path.join(ROOT, "include")
    src = tmp_path / "use.c"
    src.write_text('#include "pld.h"\nint main(void) { return pld_version() == PLD_ABI_VERSION ? 0 : 1; }\n')
    for cc, std in (("gcc", "-std=c99"), ("g++", "-std=c++17")):
        r = subprocess.run([cc, std, "-Wall", "-Wextra", "-pedantic", "-Werror", "-fsyntax-only",
                            "-x", "c" if cc == "gcc" else "c++", "-I", inc, str(src)],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_status_strings_and_version():
    m = re.search(r"#define PLD_ABI_VERSION (\d+)", open(HEADER).read())
    assert m and pld.pld_version() == int(m.group(1))
    assert pld.pld_status_string(0) == "ok"
    assert "workspace" in pld.pld_status_string(3)
    assert pld.pld_status_string(99) == "unknown status"


def test_workspace_and_scratch_bytes():
    assert pld.pld_workspace_bytes(0, 4) == 0
    assert pld.pld_workspace_bytes(1, 0) == 0
    a = pld.pld_workspace_bytes(8, 10)
    assert a > 0 and a % 256 == 0
    assert pld.pld_workspace_bytes(64, 32) >= pld.pld_workspace_bytes(64, 16)
    assert pld.pld_workspace_bytes(64, 16) >= 64 * 17 * 8      # verify keys: B*(K+1) u64
    assert pld.pld_workspace_bytes(4096, 1) >= 4096 * 8        # ranking keys: B u64
    assert pld.pld_workspace_bytes(1, 2**31 - 1) == 8 << 31     # K + 1 counted without overflow
    assert pld.pld_verify_sample_workspace_bytes(1, 2**31 - 1, 10, pld.PLD_F32) > 8 << 31
    # find: no scratch up to 16384 tokens (one block per sequence), per-tile counts beyond
    assert pld.pld_find_scratch_bytes(8, 8192) == 0
    assert pld.pld_find_scratch_bytes(8, 16384) == 0
    assert pld.pld_find_scratch_bytes(8, 16385) >= 8 * 9 * 8 * 4
    assert pld.pld_find_scratch_bytes(4, 131072) >= 4 * 64 * 8 * 4
    assert pld.pld_find_scratch_bytes(0, 9000) == 0
    # past 256 tiles (524288 tokens) also a per-tile offset and each sequence's (n, count)
    assert pld.pld_find_scratch_bytes(2, 256 * 2048) == 2 * 256 * 8 * 4
    assert pld.pld_find_scratch_bytes(2, 256 * 2048 + 1) >= 2 * 257 * (8 + 1) * 4 + 2 * 2 * 4
    assert pld.pld_find_scratch_bytes(3, 1 << 30) >= 3 * (1 << 19) * (8 + 1) * 4 + 3 * 2 * 4
    assert pld.pld_find_scratch_bytes(3, (1 << 30) + 1) == 0
    # one-call drafting: none for one block per sequence; key slots, per-block
    # counts and per-block per-n counts for split positions
    assert pld.pld_draft_workspace_bytes(8, 1) == 0
    assert pld.pld_draft_workspace_bytes(8, 37) >= 8 * 16 * 8 + 8 * 37 * 4 + 8 * 37 * 8 * 4
    assert pld.pld_draft_workspace_bytes(8, 1024) > pld.pld_draft_workspace_bytes(8, 37)
    assert pld.pld_draft_workspace_bytes(8, 1025) == 0
    assert pld.pld_draft_workspace_bytes(0, 4) == 0
    # sampling verification: the shared part, then (max, mass) per 512-vector
    # segment of each of the B*(K+1) rows
    f32, bf16 = pld.PLD_F32, pld.PLD_BF16
    assert pld.pld_verify_sample_workspace_bytes(8, 10, 32000, f32) >= \
        pld.pld_workspace_bytes(8, 10) + 8 * 11 * 16 * 8
    assert pld.pld_verify_sample_workspace_bytes(64, 16, 128256, bf16) >= \
        pld.pld_workspace_bytes(64, 16) + 64 * 17 * 32 * 8
    assert pld.pld_verify_sample_workspace_bytes(1, 1, 1, f32) > pld.pld_workspace_bytes(1, 1)
    assert pld.pld_verify_sample_workspace_bytes(0, 1, 5, f32) == 0
    assert pld.pld_verify_sample_workspace_bytes(1, 1, 5, 7) == 0


P = ctypes.c_void_p
F = P(0x1000)            # placeholder pointer, never dereferenced (host check fails first)
MIS = P(0x1002)          # misaligned placeholder
NULL = None
INF = float("-inf")


@pytest.mark.skipif(not _no_gpu(), reason="placeholder pointers are only used where no GPU is visible")
def test_host_validation_error_codes():
    lib = pld._load()
    E_INV, E_AL, E_WS = pld.PLD_ERR_INVALID, pld.PLD_ERR_ALIGN, pld.PLD_ERR_WORKSPACE
    # find: NULLs, B, n range, cap, tok_stride
    f = lib.pld_find_candidates
    assert f(NULL, 16, F, 1, 1, 1, F, 16, F, F, F, 1 << 20, NULL) == E_INV
    assert f(F, 16, F, 0, 1, 1, F, 16, F, F, F, 1 << 20, NULL) == E_INV
    assert f(F, 16, F, 1, 0, 1, F, 16, F, F, F, 1 << 20, NULL) == E_INV
    assert f(F, 16, F, 1, 2, 1, F, 16, F, F, F, 1 << 20, NULL) == E_INV
    assert f(F, 16, F, 1, 1, 9, F, 16, F, F, F, 1 << 20, NULL) == E_INV
    assert f(F, 16, F, 1, 1, 1, F, 15, F, F, F, 1 << 20, NULL) == E_INV
    assert f(F, 0, F, 1, 1, 1, F, 16, F, F, F, 1 << 20, NULL) == E_INV
    # the multi-tile path needs a scratch buffer of the documented size
    big = 1 << 15
    assert f(F, big, F, 2, 1, 1, F, big, F, F, NULL, 0, NULL) == E_WS
    assert f(F, big, F, 2, 1, 1, F, big, F, F, F, 16, NULL) == E_WS
    # rank hidden
    h = lib.pld_rank_hidden
    ok = dict()
    assert h(NULL, 64, 8, 8, 8, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert h(F, 64, 8, 8, 8, F, F, 8, F, 0, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert h(F, 64, 8, 8, 8, F, F, 8, F, 4097, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert h(F, 64, 8, 8, 12, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV   # d%8
    assert h(F, 64, 8, 8, 16392, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert h(F, 64, 8, 8, 8, F, F, 8, F, 1, math.nan, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert h(F, 64, 8, 0, 8, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert h(MIS, 64, 8, 8, 8, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_AL
    assert h(F, 64, 12, 8, 8, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_AL
    assert h(F, 64, 8, 8, 8, F, F, 8, F, 1, INF, NULL, F, F, NULL, 1 << 20, NULL) == E_WS
    assert h(F, 64, 8, 8, 8, F, F, 8, F, 1, INF, NULL, F, F, F, 7, NULL) == E_WS
    # rank attn
    a = lib.pld_rank_attn
    assert a(F, 64, 8, 8, 0, 0, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert a(F, 64, 8, 8, 1, 2, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert a(F, 64, 8, 0, 1, 0, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    assert a(MIS, 64, 8, 8, 1, 0, F, F, 8, F, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_AL
    assert a(F, 64, 8, 8, 1, 0, F, F, 8, NULL, 1, INF, NULL, F, F, F, 1 << 20, NULL) == E_INV
    # both scorings in one launch: each half's checks, then distinct workspaces
    sb = lib.pld_score_both
    W2 = P(0x2000)

    def both(hidden=F, hr=8, d=8, attn=F, R=1, agg=0, ws_a=W2, ws_a_bytes=1 << 20):
        return sb(hidden, 64, hr, 8, d, attn, 64, 8, 8, R, agg, F, F, 8, F, 1, INF, INF,
                  NULL, NULL, F, 1 << 20, ws_a, ws_a_bytes, NULL)
    assert both(hidden=NULL) == E_INV
    assert both(d=12) == E_INV
    assert both(hidden=MIS) == E_AL
    assert both(hr=12) == E_AL
    assert both(R=0) == E_INV
    assert both(agg=2) == E_INV
    assert both(attn=MIS) == E_AL
    assert both(ws_a=NULL) == E_WS
    assert both(ws_a_bytes=7) == E_WS
    assert both(ws_a=F) == E_WS                                           # same buffer
    assert both(ws_a=P(0x1000 + 127)) == E_WS                             # keys overlap (B = 1)
    assert both(ws_a=P(0x1000 - 127)) == E_WS
    # emit
    e = lib.pld_emit_draft
    assert e(F, 8, F, F, 1, 0, F, F, NULL) == E_INV
    assert e(F, 8, F, F, 0, 4, F, F, NULL) == E_INV
    assert e(F, 8, F, NULL, 1, 4, F, F, NULL) == E_INV
    # selection + draft in one launch
    sd = lib.pld_select_draft
    assert sd(NULL, 8, F, 1, 4, F, F, F, F, F, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_INV
    assert sd(F, 8, F, 0, 4, F, F, F, F, F, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_INV
    assert sd(F, 8, F, 4097, 4, F, F, F, F, F, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_INV
    assert sd(F, 8, F, 1, 0, F, F, F, F, F, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_INV
    assert sd(F, 0, F, 1, 4, F, F, F, F, F, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_INV
    assert sd(F, 8, F, 1, 4, F, F, F, NULL, F, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_INV
    assert sd(F, 8, F, 1, 4, F, F, F, F, F, 1 << 20, P(0x2000), 1 << 20, NULL, F, NULL) == E_INV
    assert sd(F, 8, F, 1, 4, F, F, F, F, NULL, 1 << 20, NULL, 0, NULL, NULL, NULL) == E_WS
    assert sd(F, 8, F, 1, 4, F, F, F, F, F, 8, NULL, 0, NULL, NULL, NULL) == E_WS
    assert sd(F, 8, F, 1, 4, F, F, F, F, F, 1 << 20, P(0x2000), 8, F, F, NULL) == E_WS
    assert sd(F, 8, F, 1, 4, F, F, F, F, F, 1 << 20, F, 1 << 20, F, F, NULL) == E_WS   # same buffer
    assert sd(F, 8, F, 1, 4, F, F, F, F, F, 1 << 20, P(0x1000 + 64), 1 << 20, F, F, NULL) == E_WS
    # the allocation-free verification: host checks come before any device set-up
    na = lib.pld_verify_greedy_noalloc
    assert na(F, 0, 40, 10, 10, 3, NULL, F, 1, F, F, F, NULL) == E_INV
    assert na(F, 2, 40, 10, 10, 3, F, F, 1, F, F, F, NULL) == E_INV                # dtype
    assert na(F, 0, 39, 10, 10, 3, F, F, 1, F, F, F, NULL) == E_INV                # seq stride
    assert na(MIS, 0, 40, 10, 10, 3, F, F, 1, F, F, F, NULL) == E_AL
    E_SC = pld.PLD_ERR_SCRATCH
    assert na(F, 0, 17 * 10, 10, 10, 16, F, F, 3856, F, F, F, NULL) == E_SC   # 65552 keys
    assert na(F, 0, 40001 * 2, 2, 2, 40000, F, F, 2, F, F, F, NULL) == E_SC   # 80002 keys
    # verify
    v = lib.pld_verify_greedy
    assert v(F, 2, 40, 10, 10, 3, F, F, 1, F, F, F, F, 1 << 20, NULL) == E_INV   # dtype
    assert v(F, 0, 40, 10, 10, 0, F, F, 1, F, F, F, F, 1 << 20, NULL) == E_INV   # K
    assert v(F, 0, 40, 10, 0, 3, F, F, 1, F, F, F, F, 1 << 20, NULL) == E_INV    # V
    assert v(F, 0, 40, 9, 10, 3, F, F, 1, F, F, F, F, 1 << 20, NULL) == E_INV    # row stride
    assert v(F, 0, 39, 10, 10, 3, F, F, 1, F, F, F, F, 1 << 20, NULL) == E_INV   # seq stride
    assert v(MIS, 0, 40, 10, 10, 3, F, F, 1, F, F, F, F, 1 << 20, NULL) == E_AL  # fp32 alignment
    assert v(F, 0, 40, 10, 10, 3, F, F, 1, F, F, F, F, 8, NULL) == E_WS
    # K + 1 rows must fit the launch's second grid dimension (65535), also at the int limit
    for k in (65535, 2**31 - 1):
        assert v(F, 0, (k + 1) * 10, 10, 10, k, F, F, 1, F, F, F, F, 1 << 40, NULL) == E_INV, k
    assert v(F, 0, 40, 10, 10, 3, F, F, 1, F, F, F, NULL, 1 << 20, NULL) == E_WS


@pytest.mark.skipif(not _no_gpu(), reason="placeholder pointers are only used where no GPU is visible")
def test_draft_host_validation():
    """The one-call drafting's own checks: blocks per sequence, the slice
    width for split positions, the context limit of one block per sequence,
    and the workspace of split positions."""
    lib = pld._load()
    E_INV, E_WS = pld.PLD_ERR_INVALID, pld.PLD_ERR_WORKSPACE
    d = lib.pld_draft_attn

    def call(tok_stride, S, ws=F, ws_bytes=1 << 24, K=4, cap=None):
        cap = tok_stride if cap is None else cap
        return d(F, tok_stride, F, 2, 1, 1, F, 8 * tok_stride, tok_stride, tok_stride, 8, 0, INF,
                 K, F, cap, F, F, NULL, F, F, F, F, S, ws, ws_bytes, NULL)

    assert call(8193, 1) == E_INV                  # one block per sequence: <= 8192 tokens
    assert call(20000, 2) == E_INV                 # slices of 10000 positions > 8192
    assert call(100, 0) == E_INV
    assert call(100, 1025) == E_INV
    assert call(100, 3, ws=NULL, ws_bytes=0) == E_WS
    assert call(20000, 3, ws_bytes=pld.pld_draft_workspace_bytes(2, 3) - 1) == E_WS
    assert call(100, 3, K=0) == E_INV
    assert call(100, 3, cap=99) == E_INV


def test_verify_sample_host_validation():
    """Checks made before any launch: temperature, uniforms and their stride,
    workspace size, and the checks shared with pld_verify_greedy."""
    lib = pld._load()
    E_INV, E_AL, E_WS = pld.PLD_ERR_INVALID, pld.PLD_ERR_ALIGN, pld.PLD_ERR_WORKSPACE
    B, K, V = 2, 3, 1000
    need = pld.pld_verify_sample_workspace_bytes(B, K, V, pld.PLD_F32)

    def call(tau=1.0, u=F, u_stride=K + 1, ws_bytes=need, V=V, dtype=pld.PLD_F32, K=K):
        return lib.pld_verify_sample(F, dtype, (K + 1) * V, V, V, K, F, F, B, tau, u, u_stride,
                                     F, F, F, NULL, F, ws_bytes, NULL)

    for tau in (0.0, -2.0, math.inf, -math.inf, math.nan, 1e-45):
        assert call(tau=tau) == E_INV, tau
    assert call(u=NULL) == E_INV
    assert call(u_stride=K) == E_INV
    assert call(u=MIS) == E_AL
    assert call(ws_bytes=need - 1) == E_WS
    assert call(ws_bytes=pld.pld_workspace_bytes(B, K)) == E_WS
    assert call(V=0) == E_INV
    assert call(dtype=5) == E_INV
    assert call(K=0) == E_INV
    assert call(K=pld.PLD_MAX_SAMPLE_ROWS, u_stride=pld.PLD_MAX_SAMPLE_ROWS + 1,
                ws_bytes=1 << 40) == E_INV
    assert call(K=2**31 - 1, u_stride=2**31, ws_bytes=1 << 62) == E_INV
    # the two halves check the same things
    st = lib.pld_verify_sample_stats
    assert st(F, pld.PLD_F32, (K + 1) * V, V, V, K, F, B, 0.0, F, need, NULL) == E_INV
    assert st(F, pld.PLD_F32, (K + 1) * V, V, V, K, F, B, 1.0, F, need - 1, NULL) == E_WS
    fin = lib.pld_verify_sample_finish
    assert fin(F, pld.PLD_F32, (K + 1) * V, V, V, K, F, F, B, 1.0, F, K, F, F, F, NULL, F, need,
               NULL) == E_INV
    assert fin(F, pld.PLD_F32, (K + 1) * V, V, V, K, F, F, B, 1.0, MIS, K + 1, F, F, F, NULL, F,
               need, NULL) == E_AL


def test_prefix_and_commit_host_validation():
    """Host-side checks of prompt lookup's selection and the commit."""
    lib = pld._load()
    E_INV = pld.PLD_ERR_INVALID
    sp = lib.pld_select_prefix
    assert sp(NULL, 100, F, F, 100, F, 2, 4, NULL, F, F, NULL) == E_INV
    assert sp(F, 100, F, F, 100, F, 0, 4, NULL, F, F, NULL) == E_INV
    assert sp(F, 100, F, F, 0, F, 2, 4, NULL, F, F, NULL) == E_INV
    assert sp(F, 100, F, F, 100, F, 2, 0, NULL, F, F, NULL) == E_INV
    assert sp(F, 100, F, F, 100, F, 2, pld.PLD_MAX_MATCH + 1, NULL, F, F, NULL) == E_INV
    cm = lib.pld_commit
    assert cm(NULL, 100, F, NULL, F, F, 2, 4, NULL, NULL) == E_INV
    assert cm(F, 100, F, NULL, F, F, 0, 4, NULL, NULL) == E_INV
    assert cm(F, 100, F, NULL, F, F, 2, 0, NULL, NULL) == E_INV
    assert cm(F, 0, F, NULL, F, F, 2, 4, NULL, NULL) == E_INV
    assert cm(F, 100, F, NULL, F, F, 65536, 4, NULL, NULL) == E_INV
    assert cm(F, 100, F, NULL, F, F, 2, 65535, NULL, NULL) == E_INV
    assert cm(F, 100, F, NULL, F, F, 2, 2**31 - 1, NULL, NULL) == E_INV
    # the acceptance with the commit: the union of the two calls' checks
    ac = lib.pld_accept_commit
    ws_n = pld.pld_workspace_bytes(2, 4)
    ok = (F, F, 2, 4, F, F, F, F, 100, F, NULL, NULL, F, ws_n, NULL)
    for k in (0, 1, 4, 5, 6, 7, 9):      # required pointers
        args = list(ok)
        args[k] = NULL
        assert ac(*args) == E_INV, k
    assert ac(*(ok[:2] + (0,) + ok[3:])) == E_INV                  # B
    assert ac(*(ok[:3] + (0,) + ok[4:])) == E_INV                  # K
    assert ac(*(ok[:8] + (0,) + ok[9:])) == E_INV                  # tok_stride
    assert ac(*(ok[:12] + (NULL,) + ok[13:])) == pld.PLD_ERR_WORKSPACE
    assert ac(*(ok[:13] + (ws_n - 1,) + ok[14:])) == pld.PLD_ERR_WORKSPACE


def test_split_rule():
    """DraftStep.tune_split, the one-call drafting's blocks per sequence: one block
    for short contexts with short lists; for hidden-state ranking about 32 rows per
    block of the longest list and at least 512 blocks in all; for attention about
    32 gathers per block; at least 64 positions per block, and never fewer blocks
    than the stride needs (8192 positions at most per block)."""
    from paper_2412_01447_amd.step import DraftStep
    s = DraftStep(8, 4096, 10, device="cpu")
    assert s.tune_split([2, 32], hidden=True) == 1
    assert s.tune_split([33], hidden=True) == 64          # 512 // 8
    assert s.tune_split([480, 3], hidden=True) == 64
    assert s.tune_split([3000], hidden=True) == 64        # ceil(3000/32) capped at 4096/64
    assert s.tune_split([256], hidden=False) == 1
    assert s.tune_split([257], hidden=False) == 9         # ceil(257/32)
    big = DraftStep(4, 131072, 32, device="cpu")
    assert big.tune_split([3298, 10, 0, 5], hidden=True) == 128   # 512 // 4 > ceil(3298/32)
    assert big.tune_split([8000], hidden=True) == 250             # ceil(8000/32)
    assert big.tune_split([10], hidden=False) == 16               # 131072 / 8192 positions
    one = DraftStep(1, 1024, 10, device="cpu")
    assert one.tune_split([32], hidden=True) == 1
    assert one.tune_split([42], hidden=True) == 16                # 1024 / 64 positions
    assert one.tune_split([100], hidden=True) == 16               # 1024 / 64 positions
    att = DraftStep(32, 8192, 16, device="cpu")
    assert att.tune_split([1181, 7], hidden=False) == 37
