/*
 * c_step.c -- one drafting step through libpld from plain C99: no C++, no
 * torch, only the HIP runtime's C API for device memory and a stream.  The
 * boundary's five calls run in order on the program's own stream:
 * pld_find_candidates (n-grams NMAX down to NMIN, Eq. 1), pld_rank_hidden
 * (Eq. 2) and pld_rank_attn (Eq. 3, SUM over the R rows) of the same
 * occurrences, pld_emit_draft from the hidden-state choice (Sec. 4.3) and
 * pld_verify_greedy (Sec. 3, Sec. 4.4).
 *
 *   c_step DIR B STRIDE NMIN NMAX D R K V
 *
 * Inputs, raw little-endian files in DIR:
 *   tokens.i32 [B][STRIDE], lens.i32 [B], hidden.u16 [B][STRIDE][D] (bf16
 *   bits), attn.f32 [B][R][STRIDE], logits.f32 [B][K+1][V].
 * Outputs, written to DIR in the same form:
 *   cand_pos.i32 [B][STRIDE], cand_count.i32, ngram_used.i32,
 *   scores_h.f32 [B][STRIDE], best_h.i32, bscore_h.f32,
 *   scores_a.f32 [B][STRIDE], best_a.i32, bscore_a.f32,
 *   draft.i32 [B][K], draft_len.i32, accept_len.i32, out_tokens.i32 [B][K+1],
 *   out_count.i32.
 * Exit status 0 on success; otherwise the failing step is printed.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pld.h"

static const char *g_dir;

static int hip_ok(hipError_t e, const char *what) {
    if (e == hipSuccess) return 1;
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 0;
}

static int pld_ok(int rc, const char *what) {
    if (rc == PLD_OK) return 1;
    fprintf(stderr, "%s: %s\n", what, pld_status_string(rc));
    return 0;
}

/* A device buffer of n bytes holding the file DIR/name (which must have n bytes). */
static void *dev_input(const char *name, size_t n) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", g_dir, name);
    FILE *f = fopen(path, "rb");
    if (!f) {
        fprintf(stderr, "cannot open %s\n", path);
        return NULL;
    }
    void *h = malloc(n ? n : 1);
    const size_t got = h ? fread(h, 1, n, f) : 0;
    const int extra = fgetc(f) != EOF;
    fclose(f);
    if (!h || got != n || extra) {
        fprintf(stderr, "%s: expected %zu bytes\n", path, n);
        free(h);
        return NULL;
    }
    void *d = NULL;
    if (!hip_ok(hipMalloc(&d, n ? n : 1), "hipMalloc") ||
        !hip_ok(hipMemcpy(d, h, n, hipMemcpyHostToDevice), "hipMemcpy to device")) {
        free(h);
        return NULL;
    }
    free(h);
    return d;
}

/* A device buffer of n bytes, every byte set to `fill`. */
static void *dev_output(size_t n, int fill) {
    void *d = NULL;
    if (!hip_ok(hipMalloc(&d, n ? n : 1), "hipMalloc")) return NULL;
    if (!hip_ok(hipMemset(d, fill, n ? n : 1), "hipMemset")) return NULL;
    return d;
}

/* Copies n bytes of the device buffer d to the file DIR/name. */
static int save(const char *name, const void *d, size_t n) {
    char path[4096];
    snprintf(path, sizeof path, "%s/%s", g_dir, name);
    void *h = malloc(n ? n : 1);
    if (!h || !hip_ok(hipMemcpy(h, d, n, hipMemcpyDeviceToHost), "hipMemcpy to host")) {
        free(h);
        return 0;
    }
    FILE *f = fopen(path, "wb");
    const int ok = f && fwrite(h, 1, n, f) == n;
    if (f) fclose(f);
    free(h);
    if (!ok) fprintf(stderr, "cannot write %s\n", path);
    return ok;
}

int main(int argc, char **argv) {
    if (argc != 10) {
        fprintf(stderr, "usage: c_step DIR B STRIDE NMIN NMAX D R K V\n");
        return 2;
    }
    g_dir = argv[1];
    const int B = atoi(argv[2]);
    const int64_t S = atoll(argv[3]);
    const int nmin = atoi(argv[4]), nmax = atoi(argv[5]);
    const int D = atoi(argv[6]), R = atoi(argv[7]), K = atoi(argv[8]), V = atoi(argv[9]);
    if (B < 1 || S < 1 || D < 1 || R < 1 || K < 1 || V < 1) {
        fprintf(stderr, "sizes must be positive\n");
        return 2;
    }
    const size_t b = (size_t)B, s = (size_t)S;

    int32_t *tokens = dev_input("tokens.i32", b * s * 4);
    int32_t *lens = dev_input("lens.i32", b * 4);
    uint16_t *hidden = dev_input("hidden.u16", b * s * (size_t)D * 2);
    float *attn = dev_input("attn.f32", b * (size_t)R * s * 4);
    float *logits = dev_input("logits.f32", b * (size_t)(K + 1) * (size_t)V * 4);
    if (!tokens || !lens || !hidden || !attn || !logits) return 1;

    int32_t *cand_pos = dev_output(b * s * 4, 0xff), *cand_count = dev_output(b * 4, 0xff);
    int32_t *ngram_used = dev_output(b * 4, 0xff);
    float *scores_h = dev_output(b * s * 4, 0), *scores_a = dev_output(b * s * 4, 0);
    int32_t *best_h = dev_output(b * 4, 0xff), *best_a = dev_output(b * 4, 0xff);
    float *bscore_h = dev_output(b * 4, 0), *bscore_a = dev_output(b * 4, 0);
    int32_t *draft = dev_output(b * (size_t)K * 4, 0xff), *draft_len = dev_output(b * 4, 0xff);
    int32_t *accept_len = dev_output(b * 4, 0xff), *out_count = dev_output(b * 4, 0xff);
    int32_t *out_tokens = dev_output(b * (size_t)(K + 1) * 4, 0xff);
    /* the workspace starts zero and every call leaves it zero, so the calls
     * below share one (one after another on one stream) */
    const size_t ws_bytes = pld_workspace_bytes(B, K);
    const size_t scr_bytes = pld_find_scratch_bytes(B, S);
    void *ws = dev_output(ws_bytes, 0), *scr = dev_output(scr_bytes, 0);
    if (!cand_pos || !cand_count || !ngram_used || !scores_h || !scores_a || !best_h || !best_a ||
        !bscore_h || !bscore_a || !draft || !draft_len || !accept_len || !out_count ||
        !out_tokens || !ws || !scr || ws_bytes == 0)
        return 1;

    hipStream_t st;
    if (!hip_ok(hipStreamCreate(&st), "hipStreamCreate")) return 1;
    if (!pld_ok(pld_find_candidates(tokens, S, lens, B, nmin, nmax, cand_pos, S, cand_count,
                                    ngram_used, scr, scr_bytes, st),
                "pld_find_candidates") ||
        !pld_ok(pld_rank_hidden(hidden, S * D, D, S, D, lens, cand_pos, S, cand_count, B,
                                -INFINITY, scores_h, best_h, bscore_h, ws, ws_bytes, st),
                "pld_rank_hidden") ||
        !pld_ok(pld_rank_attn(attn, (int64_t)R * S, S, S, R, PLD_AGG_SUM, lens, cand_pos, S,
                              cand_count, B, -INFINITY, scores_a, best_a, bscore_a, ws,
                              ws_bytes, st),
                "pld_rank_attn") ||
        !pld_ok(pld_emit_draft(tokens, S, lens, best_h, B, K, draft, draft_len, st),
                "pld_emit_draft") ||
        !pld_ok(pld_verify_greedy(logits, PLD_F32, (int64_t)(K + 1) * V, V, V, K, draft,
                                  draft_len, B, accept_len, out_tokens, out_count, ws, ws_bytes,
                                  st),
                "pld_verify_greedy"))
        return 1;
    if (!hip_ok(hipStreamSynchronize(st), "hipStreamSynchronize")) return 1;

    const int saved = save("cand_pos.i32", cand_pos, b * s * 4) &&
                      save("cand_count.i32", cand_count, b * 4) &&
                      save("ngram_used.i32", ngram_used, b * 4) &&
                      save("scores_h.f32", scores_h, b * s * 4) &&
                      save("best_h.i32", best_h, b * 4) && save("bscore_h.f32", bscore_h, b * 4) &&
                      save("scores_a.f32", scores_a, b * s * 4) &&
                      save("best_a.i32", best_a, b * 4) && save("bscore_a.f32", bscore_a, b * 4) &&
                      save("draft.i32", draft, b * (size_t)K * 4) &&
                      save("draft_len.i32", draft_len, b * 4) &&
                      save("accept_len.i32", accept_len, b * 4) &&
                      save("out_tokens.i32", out_tokens, b * (size_t)(K + 1) * 4) &&
                      save("out_count.i32", out_count, b * 4) && save("workspace.u8", ws, ws_bytes);
    if (!saved) return 1;
    hipStreamDestroy(st);
    printf("c_step: ok\n");
    return 0;
}
