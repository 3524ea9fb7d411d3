// pld_sample.hip -- sampling verification (arXiv 2412.01447, Sec. 3 and Sec.
// 4.4 with a temperature tau; the paper's sampling experiments use tau = 1).
//
// y_i is drawn from softmax(Z[b][i] / tau) by inversion at a caller-supplied
// uniform u: the first v whose cumulative mass exceeds u times the row's
// total.  One streaming pass writes, per 512-vector segment of a row, the
// segment maximum and the segment's mass relative to it; a finishing kernel
// (one wave per row, up to 16 rows per block) combines the segment masses,
// finds the segment the target falls in, re-reads only that segment (1/nseg of
// the row) to find the token, and runs the acceptance on the row tokens.
#include <float.h>
#include <math.h>

#include "pld.h"
#include "pld_device.h"
#include "pld_verify.h"

namespace pld {

// -------------------------------------------------------------- sampling
// Mass of one element relative to a maximum m: 2^((z - m) * k) with
// k = log2(e) / tau, i.e. exp((z - m) / tau).  The subtraction comes first so
// that the exponent's rounding error scales with z - m, not with m.  The
// finishing kernel recomputes the masses of one segment with the segment's own
// maximum, so it gets bit-for-bit the values the statistics pass summed.
__device__ __forceinline__ float rel_mass(float z, float m, float k) {
    return __builtin_amdgcn_exp2f((z - m) * k);
}

constexpr int kSegVecs = kWave * kVerifyUnroll;   // 16-byte vectors per segment

struct SampleArgs {
    const void *logits;
    int64_t ls, lr;
    int V, K, B;
    int S;          // statistics blocks per row
    int nseg_max;   // segment slots per row in `stats`
    float k;        // log2(e) / tau
    const float *uniforms;
    int64_t u_stride;
    const int32_t *draft;
    const int32_t *draft_len;
    int32_t *accept_len;
    int32_t *out_tokens;
    int32_t *out_count;
    int32_t *row_sample;   // [B][K+1] or null
    float2 *stats;         // [B][K+1][nseg_max]: (segment maximum, mass relative to it)
    int parts;             // finishing blocks per sequence (rows split between them)
    int32_t *tickets;      // [B], zero on entry and exit: the parts that are done
    int32_t *tokens;       // [B][K+1]: the parts' tokens, handed to the last part
};

__host__ __device__ __forceinline__ int seg_count(int nvec) {
    return nvec > 0 ? (nvec + kSegVecs - 1) / kSegVecs : 1;
}

// One wave per segment: lane l takes vectors l, l+64, ..., l+448 of it (each
// load instruction reads 1 KB contiguous), plus one head element (segment 0)
// and one tail element (last segment).  Rows past the draft are not read.
template <int kBf16>
__global__ __launch_bounds__(kVerifyThreads) void sample_stats_kernel(SampleArgs a) {
    using E = Elem<kBf16>;
    using T = typename E::T;
    constexpr int P = E::kPerVec;
    constexpr uint32_t kNegInf2 = kBf16 ? 0xff80ff80u : 0xff800000u;   // -inf in every element
    const int i = blockIdx.y, b = blockIdx.z;
    const int L = a.draft_len[b];
    if (L < 0 || L > a.K || i > L) return;
    const RowView<T, P> rv = row_view<T, P>(a.logits, a.ls, a.lr, b, i, a.V);
    const int nseg = seg_count(rv.nvec);
    const int lane = lane_id();
    float2 *st = a.stats + ((int64_t)b * (a.K + 1) + i) * a.nseg_max;
    const int step = a.S * kVerifyWaves;
    for (int g = blockIdx.x * kVerifyWaves + (int)threadIdx.x / kWave; g < nseg; g += step) {
        const int64_t v_base = (int64_t)g * kSegVecs + lane;
        uint4 r[kVerifyUnroll];
#pragma unroll
        for (int u = 0; u < kVerifyUnroll; ++u) {
            const int64_t vi = v_base + (int64_t)u * kWave;
            r[u] = make_uint4(kNegInf2, kNegInf2, kNegInf2, kNegInf2);
            if (vi < rv.nvec) r[u] = ld_stream(rv.vec + vi);
        }
        const float zh = (g == 0 && lane < rv.head) ? E::get(rv.row, lane) : -INFINITY;
        const float zt =
            (g == nseg - 1 && rv.body_end + lane < a.V) ? E::get(rv.row, rv.body_end + lane)
                                                        : -INFINITY;
        float z[kVerifyUnroll][P];
        float m = fmaxf(zh, zt);
#pragma unroll
        for (int u = 0; u < kVerifyUnroll; ++u) {
            E::unpack(r[u], z[u]);
#pragma unroll
            for (int e = 0; e < P; ++e) m = fmaxf(m, z[u][e]);
        }
        const float M = wave_max_f32(m);
        float mass = 0.f;
        if (M > -INFINITY) {   // wave-uniform; an all -inf segment has no mass
            mass = rel_mass(zh, M, a.k) + rel_mass(zt, M, a.k);
#pragma unroll
            for (int u = 0; u < kVerifyUnroll; ++u)
#pragma unroll
                for (int e = 0; e < P; ++e) mass += rel_mass(z[u][e], M, a.k);
            mass = wave_sum_f32(mass);
        }
        if (lane == 0) st[g] = make_float2(M, mass);
    }
}

// Mass of segment g rescaled to the row maximum M (0 for a segment of -inf).
__device__ __forceinline__ float seg_weight(float2 st, float M, float k) {
    return st.x > -INFINITY ? st.y * rel_mass(st.x, M, k) : 0.f;
}

// The rows' tokens and the acceptance.  A sequence's K+1 rows are split over
// ceil((K+1)/16) blocks (parts) of at most 16 waves, so that every row is in
// the first round of its block's waves; a wave takes a row i <= L:
//  1. the row maximum M over the segment maxima, the segment masses rescaled
//     to M and their inclusive scan (64 segments per round, rounds chained in
//     one fixed order, so the last cumulative value is the total S bit for
//     bit), the target t = u * S and the first segment whose cumulative mass
//     exceeds t;
//  2. that segment re-read (lane l takes its vectors l, l+64, ..., coalesced)
//     with the masses recomputed exactly as the statistics pass computed them,
//     and scanned in index order: head elements, then vector rounds 0..7
//     (lanes in order within a round), then tail elements;
//  3. the first element whose cumulative mass exceeds the target, found by a
//     ballot and a walk through one vector's elements.
// Where rounding leaves no crossing, the last element with mass is taken, so
// the token always has nonzero fp32 probability.  With one part the tokens go
// to LDS and, after a barrier, one wave runs the acceptance.  With several,
// each token goes to the workspace by an atomic exchange whose return is
// waited for, each part then counts itself done with one atomic add on the
// sequence's counter, and the part that brings it to the number of parts
// reads the tokens back by atomics, returns the counter to zero and runs the
// acceptance: the tokens travel through atomics only, so no part writes back
// or invalidates a cache.
constexpr int kFinishWaves = 16;
constexpr int kFinishMaxRows = PLD_MAX_SAMPLE_ROWS;   // K+1 limit (the row tokens live in LDS)

// A row's first loads -- the statistics of its first 64 segments (one per
// lane) and its uniform draw -- issued ahead of the work that needs them.
struct RowInputs {
    float2 s0;
    float u;
};

template <int kBf16>
__device__ __forceinline__ int row_segments(const SampleArgs &a, int b, int i) {
    using E = Elem<kBf16>;
    return seg_count(row_view<typename E::T, E::kPerVec>(a.logits, a.ls, a.lr, b, i, a.V).nvec);
}

template <int kBf16>
__device__ __forceinline__ RowInputs load_row_inputs(const SampleArgs &a, int b, int i) {
    const int nseg = row_segments<kBf16>(a, b, i);
    const int lane = lane_id();
    const float2 *st = a.stats + ((int64_t)b * (a.K + 1) + i) * a.nseg_max;
    RowInputs in;
    in.s0 = make_float2(-INFINITY, 0.f);
    if (lane < nseg) in.s0 = st[lane];
    in.u = a.uniforms[(int64_t)b * a.u_stride + i];
    return in;
}

template <int kBf16>
__device__ __forceinline__ int sample_row(const SampleArgs &a, int b, int i, const RowInputs &in) {
    using E = Elem<kBf16>;
    using T = typename E::T;
    constexpr int P = E::kPerVec;
    constexpr uint32_t kNegInf2 = kBf16 ? 0xff80ff80u : 0xff800000u;
    const int lane = lane_id();
    const int64_t slot = (int64_t)b * (a.K + 1) + i;
    const RowView<T, P> rv = row_view<T, P>(a.logits, a.ls, a.lr, b, i, a.V);
    const int nseg = seg_count(rv.nvec);
    const float2 *st = a.stats + slot * a.nseg_max;
    const float k = a.k;
    auto seg_stat = [&](int g) {   // by value (a select between two addresses would need a stack slot)
        float2 v = make_float2(-INFINITY, 0.f);
        if (g < nseg) v = st[g];
        return v;
    };
    auto readf = [](float v, int l) {
        return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
    };

    // 1. The segment the target falls in.
    float M = wave_max_f32(in.s0.x);
    for (int g0 = kWave; g0 < nseg; g0 += kWave) M = fmaxf(M, wave_max_f32(seg_stat(g0 + lane).x));
    if (!(M > -INFINITY)) return 0;   // a row of -inf only: token 0
    float u = in.u;
    if (!(u >= 0.f)) u = 0.f;                   // also NaN
    if (u >= 1.f) u = 0x1.fffffep-1f;           // the largest float below 1
    int gc = -1, glast = 0;
    float r_loc = INFINITY, mc = M;
    // Rounds of 64 segments, inclusive scans chained through `carry` in one
    // fixed order: the total is the last cumulative value bit for bit, so
    // t = u * total < total is crossed.  One round (nseg <= 64) scans once.
    float tot = 0.f;
    if (nseg > kWave)
        for (int g0 = 0; g0 < nseg; g0 += kWave) {
            const float2 sg = g0 == 0 ? in.s0 : seg_stat(g0 + lane);
            const float W = tot + wave_incl_scan_f32(seg_weight(sg, M, k));
            tot = readf(W, kWave - 1);
        }
    float carry = 0.f;
    for (int g0 = 0; g0 < nseg && gc < 0; g0 += kWave) {
        const float2 sg = g0 == 0 ? in.s0 : seg_stat(g0 + lane);
        const float wg = seg_weight(sg, M, k);
        const float W = carry + wave_incl_scan_f32(wg);
        if (nseg <= kWave) tot = readf(W, kWave - 1);
        const float t = u * tot;
        const uint64_t cross = __ballot(W > t && wg > 0.f);
        const uint64_t pos = __ballot(wg > 0.f);
        if (pos) glast = g0 + 63 - __clzll((long long)pos);
        if (cross) {
            const int f = __ffsll((unsigned long long)cross) - 1;
            const float before = f > 0 ? readf(W, f - 1) : carry;
            gc = g0 + f;
            mc = readf(sg.x, f);
            // the target inside the segment, in units of the segment's own maximum
            r_loc = fmaxf(t - before, 0.f) / rel_mass(mc, M, k);
        }
        carry = readf(W, kWave - 1);
    }
    if (gc < 0) {   // rounding left no crossing: the last element with mass of the last such segment
        gc = glast;
        mc = st[gc].x;
        r_loc = INFINITY;
    }

    // 2. The segment re-read: lane l takes vectors l, l+64, ..., l+448 of it
    // (each load instruction reads 1 KB contiguous), plus one head element
    // (first segment) and one tail element (last segment), with the masses
    // recomputed exactly as the statistics pass computed them.
    const int64_t vb = (int64_t)gc * kSegVecs + lane;
    uint4 r[kVerifyUnroll];
#pragma unroll
    for (int q = 0; q < kVerifyUnroll; ++q) {
        const int64_t vi = vb + (int64_t)q * kWave;
        r[q] = make_uint4(kNegInf2, kNegInf2, kNegInf2, kNegInf2);
        if (vi < rv.nvec) r[q] = rv.vec[vi];
    }
    const float zh = (gc == 0 && lane < rv.head) ? E::get(rv.row, lane) : -INFINITY;
    const float zt =
        (gc == nseg - 1 && rv.body_end + lane < a.V) ? E::get(rv.row, rv.body_end + lane) : -INFINITY;
    const float ph = rel_mass(zh, mc, k), pt = rel_mass(zt, mc, k);
    float sv[kVerifyUnroll];
#pragma unroll
    for (int q = 0; q < kVerifyUnroll; ++q) {
        float z[P];
        E::unpack(r[q], z);
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < P; ++e) acc += rel_mass(z[e], mc, k);
        sv[q] = acc;
    }

    // 3. Rounds in index order -- head elements, vector rounds 0..7 (lanes in
    // order within a round), tail elements -- each an inclusive scan chained
    // through `run`, the cumulative mass before the round.  The first crossing
    // element is found by a ballot and a walk through one vector's elements.
    float run = 0.f;
    auto round_cross = [&](float x, int &f, float &before) {
        const float W = run + wave_incl_scan_f32(x);
        const uint64_t cr = __ballot(W > r_loc && x > 0.f);
        if (cr) {
            f = __ffsll((unsigned long long)cr) - 1;
            before = f > 0 ? readf(W, f - 1) : run;
        }
        run = readf(W, kWave - 1);
        return cr != 0;
    };
    // The element of vector round q, lane f (its vector rq), whose cumulative
    // mass first exceeds rr (the last one with mass when rounding leaves none):
    // uniform values only.
    auto walk = [&](const uint4 &rq, int q, int f, float rr) {
        uint4 v;
        v.x = __builtin_amdgcn_readlane(rq.x, f);
        v.y = __builtin_amdgcn_readlane(rq.y, f);
        v.z = __builtin_amdgcn_readlane(rq.z, f);
        v.w = __builtin_amdgcn_readlane(rq.w, f);
        float z[P];
        E::unpack(v, z);
        int pick = -1, last = -1;
        float c = 0.f;
#pragma unroll
        for (int e = 0; e < P; ++e) {
            const float pe = rel_mass(z[e], mc, k);
            c += pe;
            if (pe > 0.f) last = e;
            if (pick < 0 && c > rr) pick = e;
        }
        const int e = pick >= 0 ? pick : last;
        return (int)(rv.head + ((int64_t)gc * kSegVecs + (int64_t)q * kWave + f) * P + e);
    };
    // (Loops without early exits, so that they unroll and r[], sv[] stay in
    // registers.)
    int f, y = -1;
    float before;
    if (round_cross(ph, f, before)) y = f;   // a head element (segment 0)
#pragma unroll
    for (int q = 0; q < kVerifyUnroll; ++q)
        if (y < 0 && round_cross(sv[q], f, before))
            y = walk(r[q], q, f, fmaxf(r_loc - before, 0.f));
    if (y < 0 && round_cross(pt, f, before)) y = (int)(rv.body_end + f);
    if (y >= 0) return y;
    // No crossing (rounding, or the fallback above): the last element with mass.
    uint64_t c = __ballot(pt > 0.f);
    if (c) return (int)(rv.body_end + 63 - __clzll((long long)c));
#pragma unroll
    for (int q = kVerifyUnroll - 1; q >= 0; --q) {
        c = __ballot(sv[q] > 0.f);
        if (y < 0 && c) y = walk(r[q], q, 63 - __clzll((long long)c), INFINITY);
    }
    if (y >= 0) return y;
    c = __ballot(ph > 0.f);
    return c ? 63 - __clzll((long long)c) : (int)(gc == 0 ? 0 : rv.head + (int64_t)gc * kSegVecs * P);
}

template <int kBf16>
__global__ __launch_bounds__(kFinishWaves *kWave) void sample_finish_kernel(SampleArgs a) {
    extern __shared__ int32_t s_y[];   // [K+1]
    __shared__ int s_last;
    const int part = blockIdx.x, b = blockIdx.y, K = a.K;
    const int w = (int)threadIdx.x / kWave, lane = lane_id();
    const int nw = (int)blockDim.x / kWave;   // rows of this part per round
    // This part's rows: [r0, r1), with the parts taking consecutive runs of at
    // most 16 rows, so that every row of the sequence is in its first round.
    const int per = (K + 1 + a.parts - 1) / a.parts;
    const int r0 = part * per, r1 = min(r0 + per, K + 1);
    // The first row's inputs and (wave 0) the draft are requested together with
    // the length: every row's statistics and draws exist whatever the length.
    RowInputs next{};
    if (r0 + w < r1) next = load_row_inputs<kBf16>(a, b, r0 + w);
    const int32_t *dr = a.draft + (int64_t)b * K;
    const int32_t d0 = (w == 0 && lane < K) ? dr[lane] : -1;
    const int L = a.draft_len[b];
    const bool ok = L >= 0 && L <= K;   // block-uniform
    int32_t *rs = a.row_sample ? a.row_sample + (int64_t)b * (K + 1) : nullptr;
    int32_t *tok = a.tokens + (int64_t)b * (K + 1);
    if (ok) {
        for (int i = r0 + w; i < r1 && i <= L; i += nw) {
            const RowInputs in = next;
            if (i + nw < r1 && i + nw <= L) next = load_row_inputs<kBf16>(a, b, i + nw);
            const int y = sample_row<kBf16>(a, b, i, in);
            if (lane == 0) {
                if (a.parts == 1) {
                    s_y[i] = y;
                } else {
                    // handed over by an atomic, whose return is waited for: the
                    // exchange is complete before this part counts itself done
                    const int prev = atomicExch(tok + i, y);
                    asm volatile("" ::"v"(prev));   // the returned value must arrive here
                    __builtin_amdgcn_s_waitcnt(0);
                }
                if (rs) rs[i] = y;
            }
        }
    }
    if (rs)
        for (int i = max(r0, ok ? L + 1 : 0) + (int)threadIdx.x; i < r1; i += (int)blockDim.x)
            rs[i] = -1;
    if (a.parts > 1) {
        // The last part to finish runs the acceptance.  The tokens travel by
        // atomics only (no cache maintenance): every part's exchanges have
        // completed before its count, and the last part reads them after its
        // own count, with atomics as well.
        __syncthreads();
        if (threadIdx.x == 0) {
            const int done = atomicAdd(a.tickets + b, 1);
            s_last = done == a.parts - 1;
            if (s_last) atomicExch(a.tickets + b, 0);   // zero again for the next call
        }
        __syncthreads();
        if (!s_last) return;   // block-uniform
        if (ok)
            for (int i = (int)threadIdx.x; i <= L; i += (int)blockDim.x) s_y[i] = atomicAdd(tok + i, 0);
    }
    __syncthreads();
    if (w == 0) {
        auto lds_token = [&](int r) { return (ok && r <= L) ? s_y[r] : -1; };
        // lane l asks for r = l first (d0), then r = l + 64, ... (loaded then)
        auto draft_token = [&](int r) { return r < kWave ? d0 : (r < K ? dr[r] : -1); };
        accept_wave(K, L, lds_token, draft_token, a.out_tokens + (int64_t)b * (K + 1),
                    a.accept_len + b, a.out_count + b);
    }
}

static int sample_nseg_max(int V, int dtype) {
    return seg_count(V / (dtype == PLD_F32 ? 4 : 8));   // a row has at most V / P whole vectors
}
static size_t sample_stats_bytes(int B, int K, int V, int dtype) {
    return align_up((size_t)B * ((size_t)K + 1) * (size_t)sample_nseg_max(V, dtype) * sizeof(float2),
                    256);
}
// [the shared zero-invariant part | statistics | tickets (zero-invariant) | tokens]
static size_t sample_ws_bytes(int B, int K, int V, int dtype) {
    return common_ws_bytes(B, K) + sample_stats_bytes(B, K, V, dtype) +
           align_up((size_t)B * sizeof(int32_t), 256) +
           align_up((size_t)B * ((size_t)K + 1) * sizeof(int32_t), 256);
}

// The sampling calls' arguments: those of prep_verify plus the temperature,
// the draws and the statistics region of the workspace.  k = log2(e) / tau.
static int prep_sample(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                       int V, int K, const int32_t *draft_len, int B, double temperature,
                       void *workspace, size_t workspace_bytes, SampleArgs &a) {
    VerifyArgs va;
    int rc = prep_verify(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B, workspace,
                         workspace_bytes, va);
    if (rc != PLD_OK) return rc;
    if (!(temperature > 0.0) || !(temperature <= DBL_MAX)) return PLD_ERR_INVALID;
    const double kd = 1.4426950408889634 / temperature;
    if (!(kd <= FLT_MAX)) return PLD_ERR_INVALID;
    if (K > kFinishMaxRows - 1) return PLD_ERR_INVALID;
    if (workspace_bytes < sample_ws_bytes(B, K, V, dtype)) return PLD_ERR_WORKSPACE;
    a = SampleArgs{};
    a.logits = logits;
    a.ls = l_seq_stride;
    a.lr = l_row_stride;
    a.V = V;
    a.K = K;
    a.B = B;
    a.nseg_max = sample_nseg_max(V, dtype);
    a.k = (float)kd;
    a.draft_len = draft_len;
    char *ws = static_cast<char *>(workspace);
    a.stats = reinterpret_cast<float2 *>(ws + common_ws_bytes(B, K));
    a.tickets = reinterpret_cast<int32_t *>(ws + common_ws_bytes(B, K) +
                                            sample_stats_bytes(B, K, V, dtype));
    a.tokens = a.tickets + align_up((size_t)B * sizeof(int32_t), 256) / sizeof(int32_t);
    // finishing parts: every row of a sequence in the first round of a part's waves
    a.parts = (K + 1 + kFinishWaves - 1) / kFinishWaves;
    // Statistics blocks per row: about PLD_VERIFY_TARGET_BLOCKS in all, and
    // no more waves per row than the row has segments.
    const int64_t rows = (int64_t)B * (K + 1);
    int64_t S = (PLD_VERIFY_TARGET_BLOCKS + rows - 1) / rows;
    const int64_t smax = (a.nseg_max + kVerifyWaves - 1) / kVerifyWaves;
    if (S > smax) S = smax;
    if (S < 1) S = 1;
    a.S = (int)S;
    return PLD_OK;
}

static int prep_finish(SampleArgs &a, const int32_t *draft, const float *uniforms,
                       int64_t u_stride, int32_t *accept_len, int32_t *out_tokens,
                       int32_t *out_count, int32_t *row_sample) {
    if (!draft || !uniforms || !accept_len || !out_tokens || !out_count) return PLD_ERR_INVALID;
    if (u_stride < (int64_t)a.K + 1) return PLD_ERR_INVALID;
    if ((uintptr_t)uniforms % sizeof(float)) return PLD_ERR_ALIGN;
    a.draft = draft;
    a.uniforms = uniforms;
    a.u_stride = u_stride;
    a.accept_len = accept_len;
    a.out_tokens = out_tokens;
    a.out_count = out_count;
    a.row_sample = row_sample;
    return PLD_OK;
}

static void launch_stats(const SampleArgs &a, int dtype, hipStream_t s) {
    const dim3 grid((unsigned)a.S, (unsigned)(a.K + 1), (unsigned)a.B);
    if (dtype == PLD_F32)
        hipLaunchKernelGGL(sample_stats_kernel<0>, grid, dim3(kVerifyThreads), 0, s, a);
    else
        hipLaunchKernelGGL(sample_stats_kernel<1>, grid, dim3(kVerifyThreads), 0, s, a);
}

static void launch_finish(const SampleArgs &a, int dtype, hipStream_t s) {
    const size_t lds = (size_t)(a.K + 1) * sizeof(int32_t);
    const int per = (a.K + 1 + a.parts - 1) / a.parts;   // <= kFinishWaves
    const dim3 grid((unsigned)a.parts, (unsigned)a.B), block((unsigned)(kWave * per));
    if (dtype == PLD_F32)
        hipLaunchKernelGGL(sample_finish_kernel<0>, grid, block, lds, s, a);
    else
        hipLaunchKernelGGL(sample_finish_kernel<1>, grid, block, lds, s, a);
}

}  // namespace pld

using namespace pld;

extern "C" int pld_verify_sample_stats(const void *logits, int dtype, int64_t l_seq_stride,
                                       int64_t l_row_stride, int V, int K,
                                       const int32_t *draft_len, int B, double temperature,
                                       void *workspace, size_t workspace_bytes, void *stream) {
    SampleArgs a;
    const int rc = prep_sample(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B,
                               temperature, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    launch_stats(a, dtype, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_verify_sample_finish(const void *logits, int dtype, int64_t l_seq_stride,
                                        int64_t l_row_stride, int V, int K, const int32_t *draft,
                                        const int32_t *draft_len, int B, double temperature,
                                        const float *uniforms, int64_t u_stride,
                                        int32_t *accept_len, int32_t *out_tokens,
                                        int32_t *out_count, int32_t *row_sample, void *workspace,
                                        size_t workspace_bytes, void *stream) {
    SampleArgs a;
    int rc = prep_sample(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B,
                         temperature, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    rc = prep_finish(a, draft, uniforms, u_stride, accept_len, out_tokens, out_count, row_sample);
    if (rc != PLD_OK) return rc;
    launch_finish(a, dtype, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_verify_sample(const void *logits, int dtype, int64_t l_seq_stride,
                                 int64_t l_row_stride, int V, int K, const int32_t *draft,
                                 const int32_t *draft_len, int B, double temperature,
                                 const float *uniforms, int64_t u_stride, int32_t *accept_len,
                                 int32_t *out_tokens, int32_t *out_count, int32_t *row_sample,
                                 void *workspace, size_t workspace_bytes, void *stream) {
    SampleArgs a;
    int rc = prep_sample(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B,
                         temperature, workspace, workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    rc = prep_finish(a, draft, uniforms, u_stride, accept_len, out_tokens, out_count, row_sample);
    if (rc != PLD_OK) return rc;
    launch_stats(a, dtype, (hipStream_t)stream);
    launch_finish(a, dtype, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" size_t pld_verify_sample_workspace_bytes(int B, int K, int V, int dtype) {
    if (B < 1 || K < 1 || V < 1 || (dtype != PLD_F32 && dtype != PLD_BF16)) return 0;
    return sample_ws_bytes(B, K, V, dtype);
}
