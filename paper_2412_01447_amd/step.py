"""One drafting step (find -> rank -> emit -> verify) over preallocated device buffers.

A convenience over the five calls of the binding: it owns the output and
workspace tensors for a batch shape and enqueues the calls on one stream with
no host synchronisation (arXiv 2412.01447, Sec. 4: retrieval Eq. 1, ranking
Eq. 2 / Eq. 3, draft Sec. 4.3, greedy verification Sec. 4.4, or sampling
verification at a temperature once set_sampling() is called).
"""
import torch

from . import (DRAFT_MAX_PART, DRAFT_MAX_TOK_STRIDE, PLD_AGG_SUM, PLD_BF16, PLD_F32,
               PLD_MAX_DRAFT_SPLIT, pld_accept_commit, pld_commit, pld_draft_attn, pld_draft_hidden,
               pld_draft_workspace_bytes, pld_emit_draft, pld_find_candidates,
               pld_find_scratch_bytes, pld_rank_attn, pld_rank_hidden, pld_score_attn,
               pld_score_both, pld_score_hidden, pld_select_best, pld_select_draft, pld_select_prefix,
               pld_verify_accept,
               pld_verify_argmax, pld_verify_greedy, pld_verify_sample, pld_verify_sample_finish,
               pld_verify_sample_stats, pld_verify_sample_workspace_bytes, pld_workspace_bytes)


class DraftStep:
    """mode: "split" runs the separate calls (find, rank, emit), "fused" the one-call
    drafting (one ranking artifact), "auto" the one-call drafting when there is one
    ranking artifact and the separate calls otherwise.  draft_split is the one-call
    drafting's blocks per sequence (1: one block owns a sequence, tok_stride <= 8192).
    rank_both: with both artifacts, the two scorings share one launch (pld_score_both)
    instead of two (the same scores and choices)."""

    def __init__(self, B, tok_stride, K, device="cuda", cap=None, keep_scores=False, mode="auto",
                 draft_split=1, rank_both=True):
        if mode not in ("auto", "fused", "split"):
            raise ValueError(mode)
        self.B, self.tok_stride, self.K, self.mode = B, tok_stride, K, mode
        # with both artifacts, both scorings in one launch (pld_score_both)
        self.rank_both = bool(rank_both)
        cap = tok_stride if cap is None else cap
        self.device = device
        i32 = dict(dtype=torch.int32, device=device)
        self.cand_pos = torch.full((B, cap), -1, **i32)
        self.cand_count = torch.zeros(B, **i32)
        self.ngram_used = torch.zeros(B, **i32)
        self.best_pos = torch.zeros(B, **i32)
        self.best_score = torch.zeros(B, dtype=torch.float32, device=device)
        self.best_pos_attn = torch.zeros(B, **i32)
        self.best_score_attn = torch.zeros(B, dtype=torch.float32, device=device)
        self.scores = torch.zeros((B, cap), dtype=torch.float32, device=device) if keep_scores else None
        self.scores_attn = (torch.zeros((B, cap), dtype=torch.float32, device=device)
                            if keep_scores else None)
        self.draft = torch.zeros((B, K), **i32)
        self.draft_len = torch.zeros(B, **i32)
        self.accept_len = torch.zeros(B, **i32)
        self.out_tokens = torch.zeros((B, K + 1), **i32)
        self.out_count = torch.zeros(B, **i32)
        # ranking / verification keys: zero once here, left zero by every call
        self.workspace = torch.zeros(pld_workspace_bytes(B, K), dtype=torch.uint8, device=device)
        # the attention ranking's keys when both artifacts rank the same occurrences
        self.workspace_aux = torch.zeros(pld_workspace_bytes(B, K), dtype=torch.uint8,
                                         device=device)
        nscratch = pld_find_scratch_bytes(B, tok_stride)
        self.scratch = (torch.empty(nscratch, dtype=torch.uint8, device=device)
                        if nscratch else None)
        # the one-call drafting's own workspace (key slots left zero, counts rewritten)
        self.draft_ws = None
        self.set_split(max(int(draft_split), self.min_split()))
        # sampling verification (set_sampling): temperature, the draws, the per-row tokens
        self.temperature = None
        self.uniforms = None
        self.row_sample = None

    def set_sampling(self, temperature, V, bf16, uniforms=None):
        """Verify by sampling at `temperature` (None: greedy again).  `uniforms` is a
        device fp32 [B][K+1] tensor of draws the caller refreshes before each step
        (default: a buffer of zeros, self.uniforms, to be filled in place); the
        workspace grows to what the sampling calls need for vocabulary V."""
        if temperature is None:
            self.temperature = None
            return
        need = pld_verify_sample_workspace_bytes(self.B, self.K, V, PLD_BF16 if bf16 else PLD_F32)
        if self.workspace.numel() < need:
            self.workspace = torch.zeros(need, dtype=torch.uint8, device=self.device)
        if uniforms is None:
            uniforms = torch.zeros((self.B, self.K + 1), dtype=torch.float32, device=self.device)
        self.uniforms = uniforms
        self.row_sample = torch.full((self.B, self.K + 1), -1, dtype=torch.int32,
                                     device=self.device)
        self.temperature = float(temperature)

    def min_split(self):
        """The fewest blocks per sequence the one-call drafting accepts."""
        if self.tok_stride <= DRAFT_MAX_TOK_STRIDE:
            return 1
        return max(2, -(-self.tok_stride // DRAFT_MAX_PART))

    def set_split(self, S):
        S = int(S)
        if not self.min_split() <= S <= PLD_MAX_DRAFT_SPLIT:
            raise ValueError(f"blocks per sequence {S} out of range")
        self.draft_split = S
        need = pld_draft_workspace_bytes(self.B, S) if S > 1 else 0
        if need and (self.draft_ws is None or self.draft_ws.numel() < need):
            self.draft_ws = torch.zeros(need, dtype=torch.uint8, device=self.device)
        return S

    def find(self, tokens, lens, ngram_min=1, ngram_max=1, stream=None):
        pld_find_candidates(tokens, lens, ngram_min, ngram_max, self.cand_pos, self.cand_count,
                            self.ngram_used, self.scratch, stream=stream)

    def rank_hidden(self, hidden, lens, threshold=float("-inf"), stream=None):
        pld_rank_hidden(hidden, lens, self.cand_pos, self.cand_count, self.best_pos,
                        self.best_score, self.workspace, threshold=threshold, scores=self.scores,
                        stream=stream)

    def rank_attn(self, attn, lens, agg=PLD_AGG_SUM, threshold=float("-inf"), into_best=True,
                  stream=None):
        bp = self.best_pos if into_best else self.best_pos_attn
        bs = self.best_score if into_best else self.best_score_attn
        pld_rank_attn(attn, lens, self.cand_pos, self.cand_count, bp, bs, self.workspace, agg=agg,
                      threshold=threshold, scores=self.scores_attn, stream=stream)

    def select_prefix(self, tokens, lens, max_match, stream=None):
        """Prompt lookup's choice among the occurrences (the PLD baseline)."""
        pld_select_prefix(tokens, lens, self.cand_pos, self.cand_count, self.best_pos,
                          self.best_score, max_match, scores=self.scores, stream=stream)

    def commit(self, tokens, lens, limit=None, stats=None, stream=None):
        """Appends the verified tokens to the sequences and advances lens (in place)."""
        pld_commit(tokens, lens, self.out_tokens, self.out_count, limit=limit, stats=stats,
                   stream=stream)

    def emit(self, tokens, lens, stream=None):
        pld_emit_draft(tokens, lens, self.best_pos, self.K, self.draft, self.draft_len,
                       stream=stream)

    def verify(self, logits, stream=None):
        if self.temperature is not None:
            pld_verify_sample(logits, self.draft, self.draft_len, self.temperature, self.uniforms,
                              self.accept_len, self.out_tokens, self.out_count, self.workspace,
                              row_sample=self.row_sample, stream=stream)
            return
        pld_verify_greedy(logits, self.draft, self.draft_len, self.accept_len, self.out_tokens,
                          self.out_count, self.workspace, stream=stream)

    # the halves of the ranking and verification calls (same results, one kernel each)
    def score_hidden(self, hidden, lens, threshold=float("-inf"), stream=None):
        pld_score_hidden(hidden, lens, self.cand_pos, self.cand_count, self.workspace,
                         threshold=threshold, scores=self.scores, stream=stream)

    def score_attn(self, attn, lens, agg=PLD_AGG_SUM, threshold=float("-inf"), stream=None):
        pld_score_attn(attn, lens, self.cand_pos, self.cand_count, self.workspace, agg=agg,
                       threshold=threshold, scores=self.scores_attn, stream=stream)

    def select(self, into_best=True, stream=None):
        bp = self.best_pos if into_best else self.best_pos_attn
        bs = self.best_score if into_best else self.best_score_attn
        pld_select_best(self.B, bp, bs, self.workspace, stream=stream)

    def verify_argmax(self, logits, stream=None):
        pld_verify_argmax(logits, self.draft_len, self.workspace, stream=stream)

    def verify_accept(self, stream=None):
        pld_verify_accept(self.draft, self.draft_len, self.accept_len, self.out_tokens,
                          self.out_count, self.workspace, stream=stream)

    def uses_fused(self, hidden, attn):
        one = (hidden is None) != (attn is None)
        if self.mode == "fused":
            if not one:
                raise ValueError("the one-call drafting takes one ranking artifact")
            return True
        return self.mode == "auto" and one

    def tune_split(self, cand_count, hidden=True):
        """Blocks per sequence for the one-call drafting from observed candidate
        counts (e.g. the previous step's).  Short contexts with short lists keep
        one block per sequence (one launch): up to 32 hidden rows or 256
        attention gathers in the longest list (past 32 rows of 8 KB, spreading
        them over more CUs repays the finishing launch).  Otherwise, for
        hidden-state ranking, about 32 rows per block of the longest list and at
        least 512 blocks in all (the library gives grids of up to 512 blocks 8
        waves each, two per CU); for attention ranking, about 32 gathers per
        block; and at least 64 positions per block."""
        import math
        mx = int(max(int(c) for c in cand_count)) if len(cand_count) else 0
        small = 32 if hidden else 256
        if self.tok_stride <= DRAFT_MAX_TOK_STRIDE and mx <= small:
            return self.set_split(1)
        if hidden:
            S = max(math.ceil(mx / 32), 512 // self.B)
        else:
            S = math.ceil(mx / 32)
        S = min(S, math.ceil(self.tok_stride / 64))
        S = max(2, self.min_split(), S)
        return self.set_split(min(PLD_MAX_DRAFT_SPLIT, S))

    def autotune_split(self, call, cand_count, hidden=True, factors=(0.5, 1.0, 2.0), reps=16,
                       trials=2):
        """Blocks per sequence for the one-call drafting, measured.  The candidates
        are tune_split's choice for these counts (its split form when that is one
        block) scaled by `factors`, plus one block per sequence where the stride
        allows it.  `call(i)` issues the i-th call to time -- the drafting call, or
        a whole step around it (a caller can rotate inputs through i); each
        candidate gets one warm-up call and `trials` runs of `reps` calls between
        two events, and the one with the lowest mean of its best run stays set.
        The outputs of the drafting do not depend on the choice, only its time."""
        import math
        mx = int(max(int(c) for c in cand_count)) if len(cand_count) else 0
        base = self.tune_split(cand_count, hidden)
        if base == 1:
            base = max(2, math.ceil(mx / 32))
        cands = {min(PLD_MAX_DRAFT_SPLIT, max(2, self.min_split(), round(base * f)))
                 for f in factors}
        if self.min_split() == 1:
            cands.add(1)
        best = None
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        for S in sorted(cands):
            self.set_split(S)
            call(0)
            t = float("inf")
            for _ in range(trials):
                e0.record()
                for i in range(reps):
                    call(i)
                e1.record()
                e1.synchronize()
                t = min(t, e0.elapsed_time(e1) / reps)
            if best is None or t < best[0]:
                best = (t, S)
        return self.set_split(best[1])

    def draft_fused(self, tokens, lens, hidden=None, attn=None, ngram=(1, 1), agg=PLD_AGG_SUM,
                    threshold=float("-inf"), stream=None):
        """find + rank + emit with the one-launch call."""
        if hidden is not None:
            pld_draft_hidden(tokens, lens, ngram[0], ngram[1], hidden, self.K, self.cand_pos,
                             self.cand_count, self.ngram_used, self.best_pos, self.best_score,
                             self.draft, self.draft_len, threshold=threshold, scores=self.scores,
                             blocks_per_seq=self.draft_split, workspace=self.draft_ws,
                             stream=stream)
        else:
            pld_draft_attn(tokens, lens, ngram[0], ngram[1], attn, self.K, self.cand_pos,
                           self.cand_count, self.ngram_used, self.best_pos, self.best_score,
                           self.draft, self.draft_len, agg=agg, threshold=threshold,
                           scores=self.scores_attn, blocks_per_seq=self.draft_split,
                           workspace=self.draft_ws, stream=stream)

    def make_draft(self, tokens, lens, hidden=None, attn=None, ngram=(1, 1), agg=PLD_AGG_SUM,
                   threshold=float("-inf"), prefix_match=None, stream=None):
        """The drafting half of a step.  With prefix_match set, prompt lookup's selection
        (longest matching prefix up to that many tokens) replaces the artifact ranking.
        With both artifacts, the hidden-state ranking drafts and the attention ranking
        is written to best_pos_attn / best_score_attn."""
        if prefix_match is not None:
            self.find(tokens, lens, *ngram, stream=stream)
            self.select_prefix(tokens, lens, prefix_match, stream=stream)
            self.emit(tokens, lens, stream=stream)
            return
        if self.uses_fused(hidden, attn):
            self.draft_fused(tokens, lens, hidden, attn, ngram, agg, threshold, stream=stream)
            return
        # (unprepared: each call is issued as the list is built)
        self._split_drafting(tokens, lens, hidden, attn, ngram, agg, threshold,
                             dict(stream=stream, prepare=False))

    def _split_drafting(self, tokens, lens, hidden, attn, ngram, agg, threshold, P):
        """The separate calls of the drafting half: find, the scoring of each artifact,
        then the selection and the draft in one launch (with both artifacts the
        attention ranking's keys go to the second workspace and its choice to
        best_pos_attn / best_score_attn; with rank_both the two scorings are one launch)."""
        both = hidden is not None and attn is not None
        ops = [("find", pld_find_candidates(tokens, lens, ngram[0], ngram[1], self.cand_pos,
                                            self.cand_count, self.ngram_used, self.scratch, **P))]
        if both and self.rank_both:
            ops.append(("score_both", pld_score_both(
                hidden, attn, lens, self.cand_pos, self.cand_count, self.workspace,
                self.workspace_aux, agg=agg, threshold_h=threshold, threshold_a=threshold,
                scores_h=self.scores, scores_a=self.scores_attn, **P)))
        else:
            if attn is not None:
                ops.append(("score_attn", pld_score_attn(
                    attn, lens, self.cand_pos, self.cand_count,
                    self.workspace_aux if both else self.workspace, agg=agg,
                    threshold=threshold, scores=self.scores_attn, **P)))
            if hidden is not None:
                ops.append(("score_hidden", pld_score_hidden(
                    hidden, lens, self.cand_pos, self.cand_count, self.workspace,
                    threshold=threshold, scores=self.scores, **P)))
        ops.append(("select_draft", pld_select_draft(
            tokens, lens, self.K, self.best_pos, self.best_score, self.draft, self.draft_len,
            self.workspace, aux_workspace=self.workspace_aux if both else None,
            aux_best_pos=self.best_pos_attn if both else None,
            aux_best_score=self.best_score_attn if both else None, **P)))
        return ops

    def run(self, tokens, lens, logits, hidden=None, attn=None, ngram=(1, 1), agg=PLD_AGG_SUM,
            threshold=float("-inf"), prefix_match=None, stream=None):
        """The whole step: drafting, then verification of the drafts against `logits`."""
        self.make_draft(tokens, lens, hidden, attn, ngram, agg, threshold, prefix_match,
                        stream=stream)
        self.verify(logits, stream=stream)

    def plan(self, tokens, lens, logits, hidden=None, attn=None, ngram=(1, 1), agg=PLD_AGG_SUM,
             threshold=float("-inf"), prefix_match=None, commit=None, stream=None):
        """The step as an ordered list of (name, prepared call), one kernel per entry
        except "find" on long contexts (two): the same work as run(), with every
        argument marshalled once so that issuing a step costs only the launches.
        commit=(limit, stats) adds the commit of the generation loop (with greedy
        verification, fused into the acceptance's launch: pld_accept_commit)."""
        P = dict(stream=stream, prepare=True)
        if prefix_match is not None:
            ops = [("find", pld_find_candidates(tokens, lens, ngram[0], ngram[1], self.cand_pos,
                                                self.cand_count, self.ngram_used, self.scratch,
                                                **P)),
                   ("select_prefix", pld_select_prefix(tokens, lens, self.cand_pos,
                                                       self.cand_count, self.best_pos,
                                                       self.best_score, prefix_match,
                                                       scores=self.scores, **P)),
                   ("emit", pld_emit_draft(tokens, lens, self.best_pos, self.K, self.draft,
                                           self.draft_len, **P))]
        elif self.uses_fused(hidden, attn):
            if hidden is not None:
                d = pld_draft_hidden(tokens, lens, ngram[0], ngram[1], hidden, self.K,
                                     self.cand_pos, self.cand_count, self.ngram_used,
                                     self.best_pos, self.best_score, self.draft, self.draft_len,
                                     threshold=threshold, scores=self.scores,
                                     blocks_per_seq=self.draft_split, workspace=self.draft_ws,
                                     **P)
            else:
                d = pld_draft_attn(tokens, lens, ngram[0], ngram[1], attn, self.K, self.cand_pos,
                                   self.cand_count, self.ngram_used, self.best_pos,
                                   self.best_score, self.draft, self.draft_len, agg=agg,
                                   threshold=threshold, scores=self.scores_attn,
                                   blocks_per_seq=self.draft_split, workspace=self.draft_ws,
                                   **P)
            ops = [("draft", d)]
        else:
            ops = self._split_drafting(tokens, lens, hidden, attn, ngram, agg, threshold, P)
        if self.temperature is not None:
            ops.append(("verify_sample_stats", pld_verify_sample_stats(
                logits, self.draft_len, self.temperature, self.workspace, **P)))
            ops.append(("verify_sample_finish", pld_verify_sample_finish(
                logits, self.draft, self.draft_len, self.temperature, self.uniforms,
                self.accept_len, self.out_tokens, self.out_count, self.workspace,
                row_sample=self.row_sample, **P)))
        else:
            ops.append(("verify_argmax", pld_verify_argmax(logits, self.draft_len,
                                                           self.workspace, **P)))
            ops.append(("verify_accept", pld_verify_accept(self.draft, self.draft_len,
                                                           self.accept_len, self.out_tokens,
                                                           self.out_count, self.workspace, **P)))
        if commit is not None:
            limit, stats = commit
            if ops[-1][0] == "verify_accept":   # the acceptance and the commit in one launch
                ops[-1] = ("verify_accept_commit", pld_accept_commit(
                    self.draft, self.draft_len, self.accept_len, self.out_tokens, self.out_count,
                    tokens, lens, self.workspace, limit=limit, stats=stats, **P))
            else:
                ops.append(("commit", pld_commit(tokens, lens, self.out_tokens, self.out_count,
                                                 limit=limit, stats=stats, **P)))
        return ops

    def host(self):
        """Copies every output to host numpy arrays (synchronises)."""
        names = ["cand_pos", "cand_count", "ngram_used", "best_pos", "best_score",
                 "best_pos_attn", "best_score_attn", "draft", "draft_len", "accept_len",
                 "out_tokens", "out_count"]
        out = {n: getattr(self, n).cpu().numpy() for n in names}
        if self.scores is not None:
            out["scores"] = self.scores.cpu().numpy()
            out["scores_attn"] = self.scores_attn.cpu().numpy()
        return out


def decode_loop(step, tokens, lens, limit, model, hidden=None, attn=None, ngram=(1, 1),
                agg=PLD_AGG_SUM, threshold=float("-inf"), prefix_match=None, stats=None,
                max_steps=1 << 20, check_every=4, stream=None, on_step=None):
    """The generation loop around the drafting step, on the device: draft, verify
    against `model(step, lens)` (the target model's logits over context + draft),
    commit the emitted tokens; until every sequence has reached `limit` (checked
    on the host every `check_every` steps) or `max_steps`.  `tokens` [B][stride]
    and `lens` [B] are updated in place; `stats` (int64 [B][2], optional)
    accumulates (emitted tokens, steps) per sequence, whose ratio is the paper's
    average acceptance length.  `on_step(i)` runs after each commit (tests use it
    to compare every step).  Returns the number of steps run."""
    for i in range(max_steps):
        if i % check_every == 0 and bool((lens >= limit).all()):
            return i
        step.make_draft(tokens, lens, hidden, attn, ngram, agg, threshold, prefix_match,
                        stream=stream)
        step.verify(model(step, lens), stream=stream)
        step.commit(tokens, lens, limit=limit, stats=stats, stream=stream)
        if on_step is not None:
            on_step(i)
    return max_steps
