// pld_verify.hip -- greedy verification (arXiv 2412.01447, Sec. 3 "greedy
// acceptance" and Sec. 4.4) and draft emission (Sec. 4.3).
//
// Verification: y_i = argmax_v Z[b][i][v] for the rows i <= L = draft_len[b]
// (lowest v among equal maxima, -0 == +0), then the accepted length is the
// first i < L with y_i != draft[b][i] (else L), and the step emits the
// accepted draft prefix followed by y_a.
//
// The argmax is a streaming read of the logits, so the kernel is shaped for
// HBM: every row is split across S blocks (S picked on the host so that a few
// thousand blocks are in flight), each thread issues 16-byte loads (4 fp32 or
// 8 bf16) unrolled eight deep, keeps the first maximum of its own elements,
// and the wave / block reduce the 64-bit key (orderable(value) << 32 |
// ~index), whose maximum is the highest value with the lowest index.  A block
// folds its key into the row's workspace slot with one 64-bit atomic max.
// A small acceptance kernel, launched right after on the same stream (the
// kernel boundary orders the two), reads the row keys back with one thread
// per sequence, computes the accepted length, writes the outputs and returns
// the slots to zero.  Rows i > L are never read.
//
// Sampling verification (Sec. 3 and Sec. 4.4 with a temperature tau): y_i is
// drawn from softmax(Z[b][i] / tau) by inversion at a caller-supplied uniform
// u: the first v whose cumulative mass exceeds u times the row's total.  One
// streaming pass writes, per 512-vector segment of a row, the segment maximum
// and the segment's mass relative to it; a finishing kernel (one block per
// sequence, one wave per row) combines the segment masses, finds the segment
// the target falls in, re-reads only that segment (1/nseg of the row) to find
// the token, and runs the acceptance on the tokens from LDS.
#include <float.h>
#include <math.h>

#include "pld.h"
#include "pld_device.h"

namespace pld {

// Launch tunables (compile-time; -D overrides serve tuning builds only).
#ifndef PLD_VERIFY_UNROLL
#define PLD_VERIFY_UNROLL 8          // 16-byte loads in flight per thread
#endif
#ifndef PLD_VERIFY_TARGET_BLOCKS
#define PLD_VERIFY_TARGET_BLOCKS 2048    // split-row kernel: blocks to aim for
#endif

constexpr int kVerifyThreads = 256;
constexpr int kVerifyWaves = kVerifyThreads / kWave;
constexpr int kVerifyUnroll = PLD_VERIFY_UNROLL;

struct VerifyArgs {
    const void *logits;
    int64_t ls, lr;
    int V, K, B;
    int S;         // blocks per row (general kernel)
    int chunk;     // 16-byte vectors per block (the last block of a row takes the rest)
    const int32_t *draft;
    const int32_t *draft_len;
    int32_t *accept_len;
    int32_t *out_tokens;
    int32_t *out_count;
    uint64_t *keys;      // [B][K+1], zero on entry
};

template <int kBf16>
struct Elem;
template <>
struct Elem<0> {
    using T = float;
    static constexpr int kPerVec = 4;
    __device__ static float get(const float *p, int64_t i) { return p[i]; }
    __device__ static void unpack(const uint4 &v, float (&o)[4]) {
        o[0] = __uint_as_float(v.x);
        o[1] = __uint_as_float(v.y);
        o[2] = __uint_as_float(v.z);
        o[3] = __uint_as_float(v.w);
    }
};
template <>
struct Elem<1> {
    using T = uint16_t;
    static constexpr int kPerVec = 8;
    __device__ static float get(const uint16_t *p, int64_t i) {
        return __uint_as_float(((uint32_t)p[i]) << 16);
    }
    __device__ static void unpack(const uint4 &v, float (&o)[8]) {
        o[0] = bf16_lo(v.x);
        o[1] = bf16_hi(v.x);
        o[2] = bf16_lo(v.y);
        o[3] = bf16_hi(v.y);
        o[4] = bf16_lo(v.z);
        o[5] = bf16_hi(v.z);
        o[6] = bf16_lo(v.w);
        o[7] = bf16_hi(v.w);
    }
};

// A logits row as [head | 16-byte vectors | tail]: the head takes the
// elements before the first 16-byte boundary, the tail those after the last
// whole vector; both are read one element at a time.
template <typename T, int P>
struct RowView {
    const T *row;
    const uint4 *vec;   // the body's vectors
    int head;           // elements before the body
    int nvec;           // vectors in the body
    int64_t body_end;   // first element of the tail
};
template <typename T, int P>
__device__ __forceinline__ RowView<T, P> row_view(const void *logits, int64_t ls, int64_t lr,
                                                  int b, int i, int V) {
    RowView<T, P> r;
    r.row = reinterpret_cast<const T *>(logits) + (int64_t)b * ls + (int64_t)i * lr;
    const int mis = (int)(((uintptr_t)r.row & 15) / sizeof(T));
    r.head = mis ? (P - mis) : 0;
    if (r.head > V) r.head = V;
    r.nvec = (V - r.head) / P;
    r.body_end = r.head + (int64_t)r.nvec * P;
    r.vec = reinterpret_cast<const uint4 *>(r.row + r.head);
    return r;
}

template <int kBf16>
__global__ __launch_bounds__(kVerifyThreads) void verify_argmax_kernel(VerifyArgs a) {
    using E = Elem<kBf16>;
    using T = typename E::T;
    constexpr int P = E::kPerVec;
    __shared__ uint64_t s_key[kVerifyWaves];
    const int split = blockIdx.x, i = blockIdx.y, b = blockIdx.z;

    const RowView<T, P> rv = row_view<T, P>(a.logits, a.ls, a.lr, b, i, a.V);
    const T *row = rv.row;
    const int head = rv.head, nvec = rv.nvec;
    const int64_t body_end = rv.body_end;
    const int v0 = min(split * a.chunk, nvec);
    const int v1 = (split == a.S - 1) ? nvec : min(v0 + a.chunk, nvec);
    const uint4 *vec = rv.vec;
    const int64_t my_v = v0 + threadIdx.x;

    // The first batch of this thread's vectors is requested together with the
    // draft length (every row of the buffer exists, so the loads are in
    // bounds); a row past the draft then returns without reading further.
    uint4 r[kVerifyUnroll];
#pragma unroll
    for (int u = 0; u < kVerifyUnroll; ++u) {
        const int64_t vi = my_v + (int64_t)u * kVerifyThreads;
        if (vi < v1) r[u] = ld_stream(vec + vi);
    }
    const int L = a.draft_len[b];
    if (L < 0 || L > a.K || i > L) return;   // rows past the draft are not used

    // Each thread keeps the first maximum of its own elements, which it visits
    // in increasing index order: a later element replaces the best only when
    // strictly greater (so an equal value, or -0 after +0, never does).  The
    // index starts at the thread's first element, so a thread whose elements
    // are all -inf still reports its first one.
    constexpr uint32_t kNone = 0xffffffffu;
    float best = -INFINITY;
    uint32_t bi = kNone;
    const bool has_head = split == 0 && (int)threadIdx.x < head;
    const bool has_tail = split == a.S - 1 && body_end + threadIdx.x < a.V;
    if (has_head) bi = threadIdx.x;
    else if (my_v < v1) bi = (uint32_t)(head + my_v * P);
    else if (has_tail) bi = (uint32_t)(body_end + threadIdx.x);
    if (has_head) {
        const float f = E::get(row, threadIdx.x);
        if (f > best) best = f;
    }
    for (int64_t vb = my_v; vb < v1; vb += (int64_t)kVerifyThreads * kVerifyUnroll) {
        if (vb != my_v) {
#pragma unroll
            for (int u = 0; u < kVerifyUnroll; ++u) {
                const int64_t vi = vb + (int64_t)u * kVerifyThreads;
                if (vi < v1) r[u] = ld_stream(vec + vi);
            }
        }
#pragma unroll
        for (int u = 0; u < kVerifyUnroll; ++u) {
            const int64_t vi = vb + (int64_t)u * kVerifyThreads;
            if (vi < v1) {
                float f[P];
                E::unpack(r[u], f);
                const uint32_t base = (uint32_t)(head + vi * P);
#pragma unroll
                for (int e = 0; e < P; ++e) {
                    if (f[e] > best) {
                        best = f[e];
                        bi = base + e;
                    }
                }
            }
        }
    }
    if (has_tail) {
        const int64_t e = body_end + threadIdx.x;
        const float f = E::get(row, e);
        if (f > best) {
            best = f;
            bi = (uint32_t)e;
        }
    }
    uint64_t key = (bi == kNone) ? 0ull : argmax_key(best, bi);
    key = wave_max_u64(key);
    const int w = threadIdx.x / kWave;
    if (lane_id() == 0) s_key[w] = key;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint64_t k = s_key[0];
#pragma unroll
        for (int t = 1; t < kVerifyWaves; ++t) k = s_key[t] > k ? s_key[t] : k;
        if (k)
            atomicMax((unsigned long long *)&a.keys[(int64_t)b * (a.K + 1) + i],
                      (unsigned long long)k);
    }
}

// Acceptance of one sequence by one wave, one lane per row: the first
// mismatch by a ballot, then the emitted tokens (Sec. 4.4).  `row_token(r)`
// gives y_r for r <= K (its value past L is not used); it is called for every
// r <= K of a round before the draft entries are compared.  `draft_token(r)`
// gives draft[r] for r < K and -1 for r = K; lane l asks for r = l, l+64, ...
template <class RowToken, class DraftToken>
__device__ __forceinline__ void accept_wave(int K, int L, RowToken row_token,
                                            DraftToken draft_token, int32_t *out,
                                            int32_t *accept_len, int32_t *out_count) {
    const int lane = lane_id();
    const bool ok = (L >= 0 && L <= K);   // wave-uniform
    int acc = ok ? L : -1;  // accepted length: first mismatch, else L
    int32_t y_acc = -1;     // the model's token at position acc
    bool found = !ok;
    for (int base = 0; base <= K; base += kWave) {
        const int r = base + lane;
        const int32_t d = draft_token(r);
        const int32_t y = row_token(r);
        const bool mism = !found && (r < L) && (y != d);
        const uint64_t mk = __ballot(mism);
        if (!found && mk) {
            const int f = __ffsll((unsigned long long)mk) - 1;
            acc = base + f;
            y_acc = __shfl(y, f);
            found = true;
        }
        if (!found && L >= base && L < base + kWave) y_acc = __shfl(y, L - base);
    }
    for (int r = lane; r <= K; r += kWave)
        out[r] = !ok ? -1 : (r < acc ? draft_token(r) : (r == acc ? y_acc : -1));
    if (lane == 0) {
        *accept_len = acc;
        *out_count = ok ? acc + 1 : 0;
    }
}

// One wave per sequence: y_i from the row keys, which are returned to zero.
// Every slot exists whatever the length, and the argmax never writes a slot
// past the draft, so those are zero already and zeroing all K+1 is the same.
__global__ __launch_bounds__(256) void verify_accept_kernel(VerifyArgs a) {
    const int b = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
    if (b >= a.B) return;   // wave-uniform
    const int K = a.K;
    uint64_t *slot = a.keys + (int64_t)b * (K + 1);
    const int L = a.draft_len[b];
    auto key_token = [&](int r) {
        const uint64_t k = (r <= K) ? slot[r] : 0ull;
        if (r <= K) slot[r] = 0;
        return (int32_t)argmax_key_index(k);
    };
    const int32_t *dr = a.draft + (int64_t)b * K;
    auto draft_token = [&](int r) { return r < K ? dr[r] : -1; };
    accept_wave(K, L, key_token, draft_token, a.out_tokens + (int64_t)b * (K + 1), a.accept_len + b,
                a.out_count + b);
}

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

// The rows' tokens and the acceptance, one block per sequence of
// min(16, K+1) waves.  A wave takes a row i <= L (then i + waves, ...):
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
// the token always has nonzero fp32 probability.  The tokens go to LDS; after
// a barrier one wave runs the acceptance.
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
    const int b = blockIdx.x, K = a.K;
    const int w = (int)threadIdx.x / kWave, lane = lane_id();
    const int nw = (int)blockDim.x / kWave;   // min(16, K+1) waves
    // The first row's inputs and (wave 0) the draft are requested together with
    // the length: every row's statistics and draws exist whatever the length.
    RowInputs next{};
    if (w <= K) next = load_row_inputs<kBf16>(a, b, w);
    const int32_t *dr = a.draft + (int64_t)b * K;
    const int32_t d0 = (w == 0 && lane < K) ? dr[lane] : -1;
    const int L = a.draft_len[b];
    const bool ok = L >= 0 && L <= K;   // block-uniform
    int32_t *rs = a.row_sample ? a.row_sample + (int64_t)b * (K + 1) : nullptr;
    if (ok) {
        for (int i = w; i <= L; i += nw) {
            const RowInputs in = next;
            if (i + nw <= L) next = load_row_inputs<kBf16>(a, b, i + nw);
            const int y = sample_row<kBf16>(a, b, i, in);
            if (lane == 0) {
                s_y[i] = y;
                if (rs) rs[i] = y;
            }
        }
    }
    if (rs)
        for (int i = (ok ? L + 1 : 0) + (int)threadIdx.x; i <= K; i += (int)blockDim.x) rs[i] = -1;
    __syncthreads();
    if (w == 0) {
        auto lds_token = [&](int r) { return (ok && r <= L) ? s_y[r] : -1; };
        // lane l asks for r = l first (d0), then r = l + 64, ... (loaded then)
        auto draft_token = [&](int r) { return r < kWave ? d0 : (r < K ? dr[r] : -1); };
        accept_wave(K, L, lds_token, draft_token, a.out_tokens + (int64_t)b * (K + 1),
                    a.accept_len + b, a.out_count + b);
    }
}

// ------------------------------------------------------------------ emit
// draft[b][i] = x[j*+1+i] for i < L = min(K, T-1-j*), -1 after (Sec. 4.3).
__global__ __launch_bounds__(256) void emit_kernel(const int32_t *tokens, int64_t tok_stride,
                                                   const int32_t *lens, const int32_t *best_pos,
                                                   int B, int K, int32_t *draft,
                                                   int32_t *draft_len) {
    const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (g >= (int64_t)B * K) return;
    const int b = (int)(g / K), i = (int)(g % K);
    const int64_t T = lens[b];
    const int64_t j = best_pos[b];
    int64_t L = 0;
    if (T >= 1 && T <= tok_stride && j >= 0 && j <= T - 2) L = min((int64_t)K, T - 1 - j);
    draft[g] = (i < L) ? tokens[(int64_t)b * tok_stride + j + 1 + i] : -1;
    if (i == 0) draft_len[b] = (int32_t)L;
}

// ---------------------------------------------------------------- commit
// The step after verification: the emitted tokens join the sequence.  One
// wave per sequence: m = min(out_count, cap - T) tokens appended at x[T..],
// lens advanced, the (emitted, steps) counters added to.
__global__ __launch_bounds__(256) void commit_kernel(int32_t *tokens, int64_t tok_stride,
                                                     int32_t *lens, const int32_t *limit,
                                                     const int32_t *out_tokens,
                                                     const int32_t *out_count, int B, int K,
                                                     int64_t *stats) {
    const int b = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
    const int lane = lane_id();
    if (b >= B) return;   // wave-uniform
    int64_t cap = tok_stride;
    if (limit && limit[b] < cap) cap = limit[b];
    const int64_t T = lens[b];
    const int64_t n = out_count[b];
    if (T < 0 || T > cap || n < 0 || n > K + 1) return;
    const int64_t m = min(n, cap - T);
    for (int64_t i = lane; i < m; i += kWave)
        tokens[(int64_t)b * tok_stride + T + i] = out_tokens[(int64_t)b * (K + 1) + i];
    if (lane == 0) {
        lens[b] = (int32_t)(T + m);
        if (stats) {
            stats[2 * b] += m;
            stats[2 * b + 1] += m > 0 ? 1 : 0;
        }
    }
}

static int prep_verify(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                       int V, int K, const int32_t *draft_len, int B, void *workspace,
                       size_t workspace_bytes, VerifyArgs &a) {
    if (!logits || !draft_len) return PLD_ERR_INVALID;
    if (B < 1 || K < 1 || V < 1 || (dtype != PLD_F32 && dtype != PLD_BF16)) return PLD_ERR_INVALID;
    if (B > 65535 || K + 1 > 65535) return PLD_ERR_INVALID;       // grid y / z limits
    if (l_row_stride < V || l_seq_stride < (int64_t)(K + 1) * l_row_stride) return PLD_ERR_INVALID;
    const size_t esz = dtype == PLD_F32 ? 4 : 2;
    if ((uintptr_t)logits % esz) return PLD_ERR_ALIGN;
    if (!workspace || workspace_bytes < verify_ws_bytes(B, K)) return PLD_ERR_WORKSPACE;
    // Blocks per row: enough for ~2048 blocks in flight, but each block keeps
    // at least two 16-byte vectors per thread.
    const int64_t rows = (int64_t)B * (K + 1);
    const int64_t nvec = (int64_t)V * esz / 16;
    int64_t S = (PLD_VERIFY_TARGET_BLOCKS + rows - 1) / rows;
    const int64_t smax = nvec / (2 * kVerifyThreads);
    if (S > smax) S = smax;
    if (S < 1) S = 1;
    a = VerifyArgs{};
    a.logits = logits;
    a.ls = l_seq_stride;
    a.lr = l_row_stride;
    a.V = V;
    a.K = K;
    a.B = B;
    a.S = (int)S;
    a.chunk = (int)((nvec + S - 1) / S);
    a.draft_len = draft_len;
    a.keys = (uint64_t *)workspace;
    return PLD_OK;
}

static void launch_argmax(const VerifyArgs &a, int dtype, hipStream_t s) {
    dim3 grid((unsigned)a.S, (unsigned)(a.K + 1), (unsigned)a.B);
    if (dtype == PLD_F32)
        hipLaunchKernelGGL(verify_argmax_kernel<0>, grid, dim3(kVerifyThreads), 0, s, a);
    else
        hipLaunchKernelGGL(verify_argmax_kernel<1>, grid, dim3(kVerifyThreads), 0, s, a);
}

static void launch_accept(const VerifyArgs &a, hipStream_t s) {
    hipLaunchKernelGGL(verify_accept_kernel, dim3((a.B + 3) / 4), dim3(256), 0, s, a);
}

// The ranking and verification calls share the leading, zero-invariant part
// of a workspace; the sampling statistics come after it.
static size_t common_ws_bytes(int B, int K) {
    const size_t r = rank_ws_bytes(B);
    const size_t v = verify_ws_bytes(B, K);
    return r > v ? r : v;
}
static int sample_nseg_max(int V, int dtype) {
    return seg_count(V / (dtype == PLD_F32 ? 4 : 8));   // a row has at most V / P whole vectors
}
static size_t sample_ws_bytes(int B, int K, int V, int dtype) {
    return common_ws_bytes(B, K) +
           align_up((size_t)B * (size_t)(K + 1) * (size_t)sample_nseg_max(V, dtype) * sizeof(float2),
                    256);
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
    if (K + 1 > kFinishMaxRows) return PLD_ERR_INVALID;
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
    a.stats = reinterpret_cast<float2 *>(static_cast<char *>(workspace) + common_ws_bytes(B, K));
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
    const dim3 block((unsigned)(kWave * (a.K + 1 < kFinishWaves ? a.K + 1 : kFinishWaves)));
    if (dtype == PLD_F32)
        hipLaunchKernelGGL(sample_finish_kernel<0>, dim3((unsigned)a.B), block, lds, s, a);
    else
        hipLaunchKernelGGL(sample_finish_kernel<1>, dim3((unsigned)a.B), block, lds, s, a);
}

}  // namespace pld

using namespace pld;

extern "C" int pld_verify_argmax(const void *logits, int dtype, int64_t l_seq_stride,
                                 int64_t l_row_stride, int V, int K, const int32_t *draft_len,
                                 int B, void *workspace, size_t workspace_bytes, void *stream) {
    VerifyArgs a;
    int rc = prep_verify(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B, workspace,
                         workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    launch_argmax(a, dtype, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_verify_accept(const int32_t *draft, const int32_t *draft_len, int B, int K,
                                 int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                                 void *workspace, size_t workspace_bytes, void *stream) {
    if (!draft || !draft_len || !accept_len || !out_tokens || !out_count) return PLD_ERR_INVALID;
    if (B < 1 || K < 1 || B > 65535 || K + 1 > 65535) return PLD_ERR_INVALID;
    if (!workspace || workspace_bytes < verify_ws_bytes(B, K)) return PLD_ERR_WORKSPACE;
    VerifyArgs a{};
    a.K = K;
    a.B = B;
    a.draft = draft;
    a.draft_len = draft_len;
    a.accept_len = accept_len;
    a.out_tokens = out_tokens;
    a.out_count = out_count;
    a.keys = (uint64_t *)workspace;
    launch_accept(a, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_verify_greedy(const void *logits, int dtype, int64_t l_seq_stride,
                                 int64_t l_row_stride, int V, int K, const int32_t *draft,
                                 const int32_t *draft_len, int B, int32_t *accept_len,
                                 int32_t *out_tokens, int32_t *out_count, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    if (!draft || !accept_len || !out_tokens || !out_count) return PLD_ERR_INVALID;
    VerifyArgs a;
    int rc = prep_verify(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B, workspace,
                         workspace_bytes, a);
    if (rc != PLD_OK) return rc;
    a.draft = draft;
    a.accept_len = accept_len;
    a.out_tokens = out_tokens;
    a.out_count = out_count;
    launch_argmax(a, dtype, (hipStream_t)stream);
    launch_accept(a, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

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

extern "C" int pld_emit_draft(const int32_t *tokens, int64_t tok_stride, const int32_t *lens,
                              const int32_t *best_pos, int B, int K, int32_t *draft,
                              int32_t *draft_len, void *stream) {
    if (!tokens || !lens || !best_pos || !draft || !draft_len) return PLD_ERR_INVALID;
    if (B < 1 || K < 1 || tok_stride < 1) return PLD_ERR_INVALID;
    const int64_t n = (int64_t)B * K;
    const int64_t blocks = (n + 255) / 256;
    if (blocks > 0x7fffffff) return PLD_ERR_INVALID;
    hipLaunchKernelGGL(emit_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       tokens, tok_stride, lens, best_pos, B, K, draft, draft_len);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_commit(int32_t *tokens, int64_t tok_stride, int32_t *lens,
                          const int32_t *limit, const int32_t *out_tokens,
                          const int32_t *out_count, int B, int K, int64_t *stats, void *stream) {
    if (!tokens || !lens || !out_tokens || !out_count) return PLD_ERR_INVALID;
    if (B < 1 || K < 1 || tok_stride < 1 || tok_stride > kMaxTokStride) return PLD_ERR_INVALID;
    hipLaunchKernelGGL(commit_kernel, dim3((unsigned)((B + 3) / 4)), dim3(256), 0,
                       (hipStream_t)stream, tokens, tok_stride, lens, limit, out_tokens,
                       out_count, B, K, stats);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_version(void) { return 100; }

extern "C" const char *pld_status_string(int status) {
    switch (status) {
    case PLD_OK: return "ok";
    case PLD_ERR_INVALID: return "invalid argument";
    case PLD_ERR_ALIGN: return "misaligned pointer or stride";
    case PLD_ERR_WORKSPACE: return "workspace missing or too small";
    case PLD_ERR_LAUNCH: return "kernel launch failed";
    default: return "unknown status";
    }
}

extern "C" size_t pld_workspace_bytes(int B, int K) {
    if (B < 1 || K < 1) return 0;
    return common_ws_bytes(B, K);
}
