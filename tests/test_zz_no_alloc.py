"""The allocation-free verification call against the workspace one.

pld_verify_greedy_noalloc keeps the row maxima in the library's static per-GPU
array instead of a caller's workspace.  Called through the C ABI (ctypes, no
binding wrapper), two calls in a row -- the second with a smaller batch, K and
vocabulary, so that anything the first call left in the shared array would
show -- must give exactly what pld_verify_greedy gives on the same inputs (and
what the oracle gives); a third call beyond the array's size must be refused
with PLD_ERR_SCRATCH and touch nothing.
"""
import ctypes

import numpy as np
import pytest
import torch

import oracle
import paper_2412_01447_amd as pld
import synth
from gpu_helpers import d_bf16, d_f32, d_i32, dev, gpu_verify, say

pytestmark = pytest.mark.gpu


def _noalloc(z, draft, dlen):
    """The C entry point called directly: outputs as numpy, and the status."""
    B, K1, V = z.shape
    acc = torch.full((B,), -7, dtype=torch.int32, device=dev())
    out = torch.full((B, K1), -7, dtype=torch.int32, device=dev())
    cnt = torch.full((B,), -7, dtype=torch.int32, device=dev())
    dr, dl = d_i32(draft), d_i32(dlen)
    dtype = pld.PLD_BF16 if z.dtype == torch.bfloat16 else pld.PLD_F32
    P = lambda t: ctypes.c_void_p(t.data_ptr())
    rc = pld._load().pld_verify_greedy_noalloc(
        P(z), dtype, z.stride(0), z.stride(1), V, K1 - 1, P(dr), P(dl), B, P(acc), P(out), P(cnt),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    torch.cuda.synchronize()
    return rc, (acc.cpu().numpy(), out.cpu().numpy(), cnt.cpu().numpy())


def _case(B, K, V, bf16, seed):
    rng = np.random.default_rng(seed)
    draft = rng.integers(0, V, size=(B, K)).astype(np.int32)
    dlen = rng.integers(0, K + 1, size=B).astype(np.int32)
    dlen[0] = K
    dlen[1] = -1                        # an invalid length: accept -1, nothing emitted
    z, _ = synth.make_logits(B, K, V, seed, draft, dlen.clip(0), bf16=bf16)
    zd = d_bf16(z) if bf16 else d_f32(z)
    return z, zd, draft, dlen


@pytest.mark.parametrize("first,second", [((64, 16, 128256, True), (5, 3, 1001, False)),
                                          ((8, 10, 32000, False), (3, 1, 7, True))])
def test_noalloc_matches_workspace_call(first, second):
    say("noalloc", first, second)
    for i, (B, K, V, bf16) in enumerate((first, second)):
        z, zd, draft, dlen = _case(B, K, V, bf16, 500 + i)
        rc, got = _noalloc(zd, draft, dlen)
        assert rc == pld.PLD_OK, pld.pld_status_string(rc)
        want = gpu_verify(zd, draft, dlen)           # the workspace call
        for g, w in zip(got, want):
            assert np.array_equal(g, w)
        ref = oracle.verify(z, draft, dlen, bf16=bf16)
        for g, r in zip(got, ref[:3]):
            assert np.array_equal(g, r)
        say("  call", i, "accept", got[0].tolist()[:12])


def test_noalloc_refuses_beyond_the_array():
    say("noalloc oversize")
    B, K, V = 4096, 16, 8               # 69632 keys > 65536
    zd = torch.zeros((B, K + 1, V), dtype=torch.float32, device=dev())
    draft = np.zeros((B, K), np.int32)
    dlen = np.zeros(B, np.int32)
    rc, got = _noalloc(zd, draft, dlen)
    assert rc == pld.PLD_ERR_SCRATCH
    assert (got[0] == -7).all() and (got[1] == -7).all() and (got[2] == -7).all()
