// pld_match.h -- device pieces of the occurrence search (Eq. 1 of arXiv
// 2412.01447 with longest-first n-gram queries), shared by the find kernels
// and the fused drafting kernel.
#pragma once

#include "pld_device.h"

namespace pld {

// Copies x[lo, hi) of one sequence into s[0, hi-lo) (block-wide).  With a
// 16-byte aligned start and a multiple of four tokens, 16-byte loads carry
// four tokens each.  A thread requests up to eight loads before its first
// store; indices past the end are clamped to the last element, for the loads
// and the stores alike (a repeated store of the same value), so there is no
// branch for the compiler to sink the loads into.
__device__ __forceinline__ void stage_tokens(const int32_t *x, int64_t lo, int64_t hi, int32_t *s) {
    const int n = (int)(hi - lo);
    constexpr int U = 8;
    const int32_t *src = x + lo;
    if ((((uintptr_t)src | (uintptr_t)s) & 15) == 0 && (n & 3) == 0) {
        const uint4 *sv = reinterpret_cast<const uint4 *>(src);
        uint4 *dv = reinterpret_cast<uint4 *>(s);
        const int nv = n >> 2;
        for (int i0 = threadIdx.x; i0 < nv; i0 += blockDim.x * U) {
            uint4 v[U];
#pragma unroll
            for (int u = 0; u < U; ++u) v[u] = sv[min(i0 + u * (int)blockDim.x, nv - 1)];
#pragma unroll
            for (int u = 0; u < U; ++u) dv[min(i0 + u * (int)blockDim.x, nv - 1)] = v[u];
        }
        return;
    }
    for (int i0 = threadIdx.x; i0 < n; i0 += blockDim.x * U) {
        int32_t v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = src[min(i0 + u * (int)blockDim.x, n - 1)];
#pragma unroll
        for (int u = 0; u < U; ++u) s[min(i0 + u * (int)blockDim.x, n - 1)] = v[u];
    }
}

// The query read backwards: q.v[k] = x[T-1-k] for k < nmax (0 beyond T).
struct Query {
    int32_t v[kMaxNgram];
};

// Reads the query from x (T >= 1 tokens, global memory or LDS) with
// unconditional, clamped loads.
__device__ __forceinline__ Query load_query(const int32_t *x, int64_t T, int nmax) {
    Query q;
    int32_t t[kMaxNgram];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) t[k] = x[T - 1 - k >= 0 ? T - 1 - k : 0];
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) q.v[k] = (k < nmax && T - 1 - k >= 0) ? t[k] : 0;
    return q;
}

// A lane takes 8 consecutive positions base .. base+7 (base a multiple of 8)
// and reads the 16 tokens x[base-8 .. base+7] from LDS with four aligned
// 16-byte loads; every comparison is then a register compare, with no
// branch: one wave covers 512 positions per pass.
constexpr int kLanePos = 8;

__device__ __forceinline__ uint32_t clamp8(int64_t v) {
    return v < 0 ? 0u : (v > 8 ? 8u : (uint32_t)v);
}

// lane_hits: byte k (k < nmax) of the result has bit j set iff position
// p = base + j is an occurrence of the (k+1)-gram query (Eq. 1):
// 1 <= p <= T-2 and x[p-i] == x[T-1-i] for every i <= k.  Levels >= nmax are
// zero.  `s` holds x[s0 ...] with base - s0 a multiple of 4 and at least 8,
// or s0 == 0 (then the window loads below index 0 are clamped and their
// tokens only meet positions p - i < 0, which are masked out).
// p - i >= 0 with p <= T-2 implies T-1-i >= 1, so q.v[i] is a real token.
__device__ __forceinline__ uint64_t lane_hits(const int32_t *s, int64_t s0, int64_t T,
                                              int64_t base, const Query &q, int nmax) {
    // a wave whose first position is past T-2 has nothing to compare (the
    // lanes' bases grow with the lane, so this is the same test for all)
    if (base - (int64_t)kLanePos * lane_id() > T - 2) return 0ull;
    const int i0 = (int)(base - s0) - 8;
    int32_t w[16];
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const int idx = i0 + 4 * c;
        const uint4 v = *reinterpret_cast<const uint4 *>(s + (idx < 0 ? 0 : idx));
        w[4 * c] = (int32_t)v.x;
        w[4 * c + 1] = (int32_t)v.y;
        w[4 * c + 2] = (int32_t)v.z;
        w[4 * c + 3] = (int32_t)v.w;
    }
    // positions in [1, T-2]
    uint32_t m = ((0xffu << clamp8(1 - base)) & 0xffu) & ((1u << clamp8(T - 1 - base)) - 1u);
    uint64_t out = 0;
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k) {
        if (k >= nmax) break;   // uniform
        uint32_t e = 0;
#pragma unroll
        for (int j = 0; j < kLanePos; ++j) e |= (w[8 + j - k] == q.v[k] ? 1u : 0u) << j;
        m &= e & ((0xffu << clamp8(k - base)) & 0xffu);   // p - k >= 0
        out |= (uint64_t)m << (8 * k);
    }
    return out;
}

// ------------------------------------------------------------- block search
// Writes the positions p0 + l of the set bits l of the wave-uniform mask m to
// out[run ...] (and out2[run ...] when given) in ascending order; returns run
// plus the number of bits.  The mask becomes the execution mask of the
// stores; an entry's byte offset fits in 32 bits (fewer than 2^30 positions
// per row).
__device__ __forceinline__ int emit_group(uint64_t m, int p0, int32_t *out, int32_t *out2,
                                          int run) {
    if (__builtin_amdgcn_inverse_ballot_w64(m)) {
        const uint32_t below = __builtin_amdgcn_mbcnt_hi(
            (uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        const uint32_t off = ((uint32_t)run + below) << 2;
        const int32_t p = p0 + lane_id();
        *reinterpret_cast<int32_t *>(reinterpret_cast<char *>(out) + off) = p;
        if (out2) *reinterpret_cast<int32_t *>(reinterpret_cast<char *>(out2) + off) = p;
    }
    return run + (int)__popcll(m);
}

// Occurrence search of a whole row by one block of kW waves (Eq. 1 with
// n-gram queries tried longest first).  The row is in LDS: s_x[p] = x[p] for
// p < kW * G * 64 (tokens past the length do no harm: positions past T-2 are
// masked).  Wave w takes the positions [w * G * 64, (w + 1) * G * 64) in
// groups of 64, one position per lane, and keeps one 64-bit mask per group:
// level 0 is one vector compare of the tokens against x[T-1] (and, in each
// group of the wave whose positions reach past T-2, one more against the
// position); level k keeps the bits whose x[p-k] equals x[T-1-k], all groups
// of a level at once, while any bit is left.  On the single CU that searches
// a sequence the pass costs a few instructions per 64 positions and level.  Returns n (0: no occurrence)
// and the count; with n > 0 the occurrences are written in ascending order
// to out (and out2 when given).  s_lvl: kW x kMaxNgram ints of LDS.  Call
// with T in [1, kW * G * 64], from the whole block.
template <int kW, int G>
__device__ __forceinline__ int block_search(const int32_t *s_x, int64_t T, int nmin, int nmax,
                                            int (*s_lvl)[kMaxNgram], int32_t *out, int32_t *out2,
                                            int &total) {
    const int w = __builtin_amdgcn_readfirstlane((int)threadIdx.x / kWave);
    const int lane = lane_id();
    const int w0 = w * G * kWave;
    const int hi = (int)T - 2;             // occurrences lie in [1, T-2]
    const int pl = w0 + lane;              // the lane's position in group 0
    const bool some = w0 <= hi;            // uniform: the wave has positions to test
    // level 0
    uint64_t m0[G];
#pragma unroll
    for (int i = 0; i < G; ++i) m0[i] = 0ull;
    if (some) {
        const int32_t q0 = s_x[T - 1];
        int32_t t[G];
#pragma unroll
        for (int i = 0; i < G; ++i) t[i] = s_x[pl + i * kWave];
        if (w0 + G * kWave - 1 <= hi) {    // every position of the wave is below T-1
#pragma unroll
            for (int i = 0; i < G; ++i) m0[i] = __ballot(t[i] == q0);
        } else {
#pragma unroll
            for (int i = 0; i < G; ++i) m0[i] = __ballot(t[i] == q0) & __ballot(pl <= hi - i * kWave);
        }
        if (w == 0) m0[0] &= ~1ull;        // position 0 is never an occurrence
    }
    // The masks of level `upto` (at most nmax - 1) from level 0, level by
    // level; `count(k, c)` gets each level's count.  A non-empty level k-1
    // holds a position p <= T-2 with p >= k-1, so x[T-1-k] exists.
    auto levels = [&](uint64_t (&m)[G], int upto, auto count) {
        for (int k = 1; k <= upto; ++k) {
            uint64_t any = 0ull;
#pragma unroll
            for (int i = 0; i < G; ++i) any |= m[i];
            if (!any) break;   // uniform
            const int32_t qk = s_x[T - 1 - k];
            int32_t t[G];
#pragma unroll
            for (int i = 0; i < G; ++i) t[i] = s_x[max(pl + i * kWave - k, 0)];
#pragma unroll
            for (int i = 0; i < G; ++i) m[i] &= __ballot(t[i] == qk);
            if (w == 0) m[0] &= ~0ull << k;   // x[p-k] exists only from p = k on
            int c = 0;
#pragma unroll
            for (int i = 0; i < G; ++i) c += (int)__popcll(m[i]);
            count(k, c);
        }
    };
    {
        int c0 = 0;
#pragma unroll
        for (int i = 0; i < G; ++i) c0 += (int)__popcll(m0[i]);
        if (lane == 0) {
            s_lvl[w][0] = c0;
#pragma unroll
            for (int k = 1; k < kMaxNgram; ++k) s_lvl[w][k] = 0;
        }
        if (nmax > 1 && some) {   // uniform
            uint64_t m[G];
#pragma unroll
            for (int i = 0; i < G; ++i) m[i] = m0[i];
            levels(m, nmax - 1, [&](int k, int c) {
                if (lane == 0) s_lvl[w][k] = c;
            });
        }
    }
    __syncthreads();
    // the longest n with an occurrence, and this wave's offset in the list:
    // lane i < kW holds wave i's count of the level
    int n_used = 0, run = 0;
    total = 0;
    for (int n = nmax; n >= nmin; --n) {
        const int c = lane < kW ? s_lvl[lane][n - 1] : 0;
        int t;
        const int ex = wave_excl_scan(c, t);
        if (t > 0) {   // uniform
            n_used = n;
            total = t;
            run = __builtin_amdgcn_readlane(ex, w);
            break;
        }
    }
    if (n_used > 0 && some) {   // uniform; ascending: wave, then group, then lane
        if (n_used > 1) levels(m0, n_used - 1, [](int, int) {});
#pragma unroll
        for (int i = 0; i < G; ++i) run = emit_group(m0[i], w0 + i * kWave, out, out2, run);
    }
    return n_used;
}

__device__ __forceinline__ uint32_t level_bits(uint64_t hits, int n) {
    return (uint32_t)(hits >> (8 * (n - 1))) & 0xffu;
}

// Adds the popcount of every level byte of `hits` to cnt[k], k < nmax.
__device__ __forceinline__ void count_levels(uint64_t hits, int nmax, int (&cnt)[kMaxNgram]) {
#pragma unroll
    for (int k = 0; k < kMaxNgram; ++k)
        if (k < nmax) cnt[k] += __popc((uint32_t)(hits >> (8 * k)) & 0xffu);
}

// Writes the positions base + j of the set bits j of `bits` to out[run ...]
// (and out2[run ...] when given) in ascending order across the wave's lanes;
// returns run plus the wave's number of bits.
__device__ __forceinline__ int64_t emit_bits(uint32_t bits, int64_t base, int32_t *out,
                                             int32_t *out2, int64_t run) {
    if (__ballot(bits != 0u) == 0ull) return run;   // nothing in this wave
    int total;
    int64_t o = run + wave_excl_scan(__popc(bits), total);
    while (bits) {
        const int j = __ffs(bits) - 1;
        bits &= bits - 1u;
        out[o] = (int32_t)(base + j);
        if (out2) out2[o] = (int32_t)(base + j);
        ++o;
    }
    return run + total;
}

}  // namespace pld
