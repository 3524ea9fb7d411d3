"""GPU parity of the whole drafting step on the five synthetic workloads, at full
size, in the launch configuration the benchmark times (DraftStep, one stream).

For each workload the oracle runs first on the same inputs (hidden rows it
needs are copied back from the device), its draft plants the accepted prefixes
in the verification logits, then the GPU step runs and every stage is compared:
positions / counts / n / draft / accept lengths / emitted tokens bit-exactly,
scores within 1e-3 relative, near-tie flips counted.  Both the structured
variant (the planted source of the last token is the cosine winner) and the
plain random variant are run.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2412_01447_amd as pld
import synth
from gpu_helpers import (check_best, check_find, check_scores, check_verify, d_bf16, d_f32,
                         d_i32, draft_keys_zero, gpu_emit, gpu_verify, say, sparse_hidden_rows)
from paper_2412_01447_amd.step import DraftStep

pytestmark = pytest.mark.gpu

# mode: "split" separate calls (with both artifacts, the two scorings in one launch);
# "split_sep" the same with the two scorings in launches of their own; "fused" the
# one-call drafting with blocks per sequence
# from the candidate counts, as the benchmark tunes it; "fused1" one block per
# sequence; "fused8" positions split over 8 blocks per sequence.  The one-call
# drafting takes one artifact: on the workload with both it runs on the hidden
# states alone.
CASES = [(1, True, "fused"), (1, False, "split"), (2, True, "fused"), (2, False, "fused"),
         (2, True, "split"), (2, True, "fused8"), (3, True, "fused"), (3, False, "split"),
         (3, False, "fused"), (3, False, "fused1"), (4, True, "split"), (4, False, "split"), (4, False, "split_sep"),
         (4, True, "fused"), (5, True, "split"),
         (5, False, "split"), (5, True, "fused"), (5, False, "fused"),
         (6, True, "fused"), (6, False, "fused"), (6, False, "split"), (6, True, "fused8"),
         (7, True, "fused"), (7, False, "fused"), (7, False, "split"), (7, False, "fused8")]


@pytest.mark.parametrize("cid,structured,mode", CASES,
                         ids=[f"cfg{c}_{'structured' if s else 'random'}_{m}" for c, s, m in CASES])
def test_config_step_parity(cid, structured, mode):
    cfg = synth.CONFIGS[cid]
    say("config", cid, cfg.name, "structured" if structured else "random", mode)
    dev = torch.device("cuda:0")
    w = synth.make_workload(cfg, dev, structured=structured)
    toks, lens = w["tokens"], w["lens"]
    if mode.startswith("fused") and w["hidden"] is not None:
        w["attn"] = None
    # ---- oracle, stage by stage
    cp, cc, nu = oracle.find(toks, lens, *cfg.ngram)
    ref = {}
    agg = oracle.AGG_MAX if cfg.agg == "max" else oracle.AGG_SUM
    if w["hidden"] is not None:
        hb = sparse_hidden_rows(w["hidden"], lens, cp, cc)
        ref["h"] = oracle.rank_hidden(hb, lens, cp, cc, cfg.theta)
        del hb
    if w["attn"] is not None:
        ref["a"] = oracle.rank_attn(w["attn"], lens, cp, cc, agg, cfg.theta)
    drafter = ref["h"] if "h" in ref else ref["a"]
    rdraft, rdl = oracle.emit(toks, lens, drafter[1], cfg.K)
    z = synth.logits_for(w, rdraft, rdl)
    bf16 = cfg.logits == "bf16"
    rver = oracle.verify(z, rdraft, rdl, bf16=bf16)
    say("  oracle: counts", cc.tolist()[:8], "n", sorted(set(nu.tolist())), "accept",
        rver[0].tolist()[:16])
    # ---- GPU step, as the benchmark launches it
    step = DraftStep(cfg.B, cfg.T, cfg.K, device=dev, keep_scores=True,
                     mode="fused" if mode.startswith("fused") else "split",
                     rank_both=mode != "split_sep")
    if mode == "fused":     # blocks per sequence from the candidate counts, as the bench does
        say("  blocks per sequence:", step.tune_split(cc, hidden=w["hidden"] is not None))
    elif mode == "fused8":
        step.set_split(8)
    zd = d_bf16(z) if bf16 else d_f32(z)
    attn_d = d_f32(w["attn"]) if w["attn"] is not None else None
    td, ld = d_i32(toks), d_i32(lens)
    step.run(td, ld, zd, hidden=w["hidden"], attn=attn_d, ngram=cfg.ngram,
             agg=pld.PLD_AGG_MAX if cfg.agg == "max" else pld.PLD_AGG_SUM, threshold=cfg.theta)
    torch.cuda.synchronize()
    g = step.host()
    assert int(torch.count_nonzero(step.workspace).item()) == 0
    assert int(torch.count_nonzero(step.workspace_aux).item()) == 0
    assert draft_keys_zero(step.draft_ws, cfg.B)
    check_find((g["cand_pos"], g["cand_count"], g["ngram_used"]), (cp, cc, nu), cfg.name)
    flips = 0
    if "h" in ref:
        rsc, rbp, rbs = ref["h"]
        check_scores(g["scores"], rsc, cc, cfg.name + " hidden")
        flips += check_best(g["best_pos"], g["best_score"], rsc, rbp, rbs, cp, cc, cfg.name,
                            threshold=cfg.theta)
    if "a" in ref:
        rsc, rbp, rbs = ref["a"]
        check_scores(g["scores_attn"], rsc, cc, cfg.name + " attn")
        gbp = g["best_pos_attn"] if "h" in ref else g["best_pos"]
        gbs = g["best_score_attn"] if "h" in ref else g["best_score"]
        flips += check_best(gbp, gbs, rsc, rbp, rbs, cp, cc, cfg.name + " attn",
                            threshold=cfg.theta)
    say("  near-tie flips:", flips)
    if structured and "h" in ref:
        srcs = np.array([m.query_src_end for m in w["metas"]])
        assert np.array_equal(g["best_pos"], srcs) and np.all(g["best_score"] == 1.0)
    if flips == 0:
        # chained outputs equal the oracle's chain
        assert np.array_equal(g["draft"], rdraft) and np.array_equal(g["draft_len"], rdl)
        check_verify((g["accept_len"], g["out_tokens"], g["out_count"]), rver, cfg.name)
    else:
        # after a flip, the later stages are checked on the oracle's own inputs
        gd, gl = gpu_emit(toks, lens, drafter[1], cfg.K)
        assert np.array_equal(gd, rdraft) and np.array_equal(gl, rdl)
        check_verify(gpu_verify(zd, rdraft, rdl), rver, cfg.name)
    # accepted lengths cover a range (the planted prefixes work)
    say("  accept lengths:", np.bincount(rver[0], minlength=cfg.K + 1).tolist())
    del step, w, zd
    torch.cuda.empty_cache()


@pytest.mark.parametrize("cid", [1, 2, 3, 4, 5, 6])
def test_config_verify_sample(cid):
    """Sampling verification at temperature 1 (the paper's sampling setting) at
    each workload's full logits shape, issued as the benchmark issues it (the
    prepared statistics and finishing calls), against the oracle on every
    row: rounding flips counted and window-checked, acceptance exact."""
    from gpu_helpers import check_sample
    cfg = synth.CONFIGS[cid]
    say("config sample", cid, cfg.name)
    dev = torch.device("cuda:0")
    toks, lens, metas = synth.make_tokens(cfg)
    draft, dlen = synth.intended_drafts(metas, cfg.K)
    bf16 = cfg.logits == "bf16"
    z, _ = synth.make_logits(cfg.B, cfg.K, cfg.V, cfg.seed, draft, dlen, bf16=bf16)
    U = synth.make_uniforms(cfg.B, cfg.K, cfg.seed)
    ref = oracle.verify_sample(z, draft, dlen, 1.0, U, bf16=bf16)
    step = DraftStep(cfg.B, cfg.T, cfg.K, device=dev)
    step.set_sampling(1.0, cfg.V, bf16, uniforms=d_f32(U))
    step.draft.copy_(d_i32(draft))
    step.draft_len.copy_(d_i32(dlen))
    zd = d_bf16(z) if bf16 else d_f32(z)
    ops = dict(step.plan(d_i32(toks), d_i32(lens), zd, hidden=None, attn=None))
    ops["verify_sample_stats"]()
    ops["verify_sample_finish"]()
    torch.cuda.synchronize()
    assert int(torch.count_nonzero(step.workspace[:pld.pld_workspace_bytes(cfg.B, cfg.K)])) == 0
    got = (step.accept_len.cpu().numpy(), step.out_tokens.cpu().numpy(),
           step.out_count.cpu().numpy(), step.row_sample.cpu().numpy())

    def z_rows(b, i):
        r = synth.bf16_bits_to_f32(z[b, i]) if bf16 else z[b, i]
        return np.asarray(r, np.float64)

    flips = check_sample(z_rows, 1.0, U, draft, dlen, got, ref, cfg.name, max_flip_frac=0.01)
    say("  sampled-row flips:", flips, " accept lengths:",
        np.bincount(got[0][got[0] >= 0], minlength=cfg.K + 1).tolist())
    del step, zd
    torch.cuda.empty_cache()
