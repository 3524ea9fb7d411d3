// pld_device.h -- device helpers shared by the PLD+ kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>

#if defined(__HIP_DEVICE_COMPILE__) && !defined(__gfx950__)
#error "this library is written for gfx950 (MI355X) only"
#endif

namespace pld {

constexpr int kWave = 64;
constexpr int kMaxNgram = 8;                   // equals PLD_MAX_NGRAM
constexpr int64_t kMaxTokStride = 1ll << 30;   // positions are stored as int32

// Tiling of the occurrence search.
constexpr int kFindTile = 2048;          // positions per block, multi-block find
constexpr int kFindWavesTiled = 4;       // 256 threads, 512 positions per wave
constexpr int kFindWavesFused = 16;      // 1024 threads, one block per sequence
constexpr int kFindFusedMax = kFindWavesFused * 512;  // tok_stride <= 8192: fused path
#ifndef PLD_FIND_FUSED_PASSES
#define PLD_FIND_FUSED_PASSES 2
#endif
constexpr int kFindFusedPasses = PLD_FIND_FUSED_PASSES;   // one-block search: tok_stride <= 16384

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Whether the byte ranges [p, p + np) and [q, q + nq) share a byte.
inline bool ranges_overlap(const void *p, size_t np, const void *q, size_t nq) {
    const uintptr_t a = (uintptr_t)p, b = (uintptr_t)q;
    return a < b + nq && b < a + np;
}

// Blocks of `kernel` that fit on the current device at once (CUs x resident
// blocks per CU): the grid of the persistent kernels, whose equal contiguous
// work ranges then finish in a single round.  Cached per device, kernel and
// dynamic LDS size.
inline int resident_blocks(const void *kernel, int threads, size_t dyn_lds) {
    struct Entry {
        int dev;
        const void *k;
        size_t lds;
        int blocks;
    };
    static std::mutex mu;
    static Entry cache[64];
    static int used = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) dev = 0;
    {
        std::lock_guard<std::mutex> g(mu);
        for (int i = 0; i < used; ++i)
            if (cache[i].dev == dev && cache[i].k == kernel && cache[i].lds == dyn_lds)
                return cache[i].blocks;
    }
    int cus = 0, per = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus < 1)
        cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, dyn_lds) != hipSuccess ||
        per < 1)
        per = 1;
    const int blocks = cus * per;
    std::lock_guard<std::mutex> g(mu);
    if (used < 64) cache[used++] = Entry{dev, kernel, dyn_lds, blocks};
    return blocks;
}

// Tiles per sequence up to which each compaction block sums the per-tile
// counts itself (a few KB per block); past it a scan launch gives every tile
// its offset, so the work grows with the tiles, not with their square.
constexpr int kFindScanTiles = 256;

// Scratch of the multi-block find: per-tile occurrence counts of every n;
// past kFindScanTiles tiles also the per-tile offsets of the chosen n and
// each sequence's (n, count).
inline size_t find_scratch_bytes(int B, int64_t tok_stride) {
    if (tok_stride <= kFindFusedPasses * kFindFusedMax) return 0;   // the one-block search
    const int64_t ntiles = (tok_stride + kFindTile - 1) / kFindTile;
    size_t bytes = align_up((size_t)B * (size_t)ntiles * 8 * sizeof(int32_t), 256);
    if (ntiles > kFindScanTiles)
        bytes += align_up((size_t)B * (size_t)ntiles * sizeof(int32_t), 256) +
                 align_up((size_t)B * 2 * sizeof(int32_t), 256);
    return bytes;
}
// Workspace of the ranking and verification calls: 64-bit keys that must be
// zero when a call starts and that the call leaves zero.  The ranking keys of
// a sequence are spread over kKeySlots slots (a block folds into slot
// blockIdx % kKeySlots), so that few atomics ever queue on one address.
constexpr int kKeySlots = 16;
inline size_t rank_ws_bytes(int B) {
    return align_up((size_t)B * kKeySlots * sizeof(uint64_t), 256);
}
inline size_t verify_ws_bytes(int B, int K) {
    return align_up((size_t)B * ((size_t)K + 1) * sizeof(uint64_t), 256);
}

// ---------------------------------------------------------------- keys
// Order-preserving map of a float to uint32 (larger float -> larger key);
// -0 is folded into +0 first so that the two compare equal.
__device__ __forceinline__ uint32_t ord_f32(float f) {
    uint32_t u = __float_as_uint(f);
    if (u == 0x80000000u) u = 0u;
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float unord_f32(uint32_t o) {
    uint32_t u = (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o;
    return __uint_as_float(u);
}

// Ranking key: highest score first, then the most recent position (j >= 1,
// so 0 means "no eligible candidate").
__device__ __forceinline__ uint64_t rank_key(float s, int32_t j) {
    return ((uint64_t)ord_f32(s) << 32) | (uint32_t)j;
}
// Argmax key over a vocabulary row: highest value first, then the lowest id.
__device__ __forceinline__ uint64_t argmax_key(float v, uint32_t idx) {
    return ((uint64_t)ord_f32(v) << 32) | (uint64_t)(0xffffffffu - idx);
}
__device__ __forceinline__ uint32_t argmax_key_index(uint64_t k) {
    return 0xffffffffu - (uint32_t)(k & 0xffffffffu);
}

// ------------------------------------------------------- wave reductions
__device__ __forceinline__ int lane_id() { return (int)__lane_id(); }

// Wave reductions use DPP lane moves -- quad permutes, the half-row and row
// mirrors, and the row broadcasts of lanes 15 and 31 -- a few cycles each,
// where a shuffle goes through the LDS crossbar.  The total lands in lane 63
// and is read back as a scalar, so every lane gets the same bits, and the
// association depends only on the lane layout, never on the data.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ int dpp_move(int v) {   // lanes the move does not reach get 0
    return __builtin_amdgcn_update_dpp(0, v, kCtrl, kRowMask, 0xf, false);
}
constexpr int kDppQuadSwap1 = 0xb1;   // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4e;   // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;
constexpr int kDppMirror = 0x140;
constexpr int kDppBcast15 = 0x142;    // lane 15 of a row into the next row (rows 1, 3)
constexpr int kDppBcast31 = 0x143;    // lane 31 into rows 2 and 3
constexpr int kDppShr1 = 0x111;       // row_shr:1 (+1, +3, +7 likewise)

__device__ __forceinline__ int wave_sum_i32(int v) {
    v += dpp_move<kDppQuadSwap1, 0xf>(v);
    v += dpp_move<kDppQuadSwap2, 0xf>(v);
    v += dpp_move<kDppHalfMirror, 0xf>(v);
    v += dpp_move<kDppMirror, 0xf>(v);
    v += dpp_move<kDppBcast15, 0xa>(v);
    v += dpp_move<kDppBcast31, 0xc>(v);
    return __builtin_amdgcn_readlane(v, 63);
}

// Maximum over the lanes of non-negative values (a move's unreached lanes
// read 0, which no lane's value is below).
__device__ __forceinline__ int wave_max_nonneg_i32(int v) {
    v = max(v, dpp_move<kDppQuadSwap1, 0xf>(v));
    v = max(v, dpp_move<kDppQuadSwap2, 0xf>(v));
    v = max(v, dpp_move<kDppHalfMirror, 0xf>(v));
    v = max(v, dpp_move<kDppMirror, 0xf>(v));
    v = max(v, dpp_move<kDppBcast15, 0xa>(v));
    v = max(v, dpp_move<kDppBcast31, 0xc>(v));
    return __builtin_amdgcn_readlane(v, 63);
}

__device__ __forceinline__ float wave_sum_f32(float v) {
    v += __int_as_float(dpp_move<kDppQuadSwap1, 0xf>(__float_as_int(v)));
    v += __int_as_float(dpp_move<kDppQuadSwap2, 0xf>(__float_as_int(v)));
    v += __int_as_float(dpp_move<kDppHalfMirror, 0xf>(__float_as_int(v)));
    v += __int_as_float(dpp_move<kDppMirror, 0xf>(__float_as_int(v)));
    v += __int_as_float(dpp_move<kDppBcast15, 0xa>(__float_as_int(v)));
    v += __int_as_float(dpp_move<kDppBcast31, 0xc>(__float_as_int(v)));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint64_t dpp_max_step(uint64_t v) {
    const uint32_t lo = (uint32_t)dpp_move<kCtrl, kRowMask>((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)dpp_move<kCtrl, kRowMask>((int)(uint32_t)(v >> 32));
    const uint64_t o = ((uint64_t)hi << 32) | lo;
    return o > v ? o : v;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
    v = dpp_max_step<kDppQuadSwap1, 0xf>(v);
    v = dpp_max_step<kDppQuadSwap2, 0xf>(v);
    v = dpp_max_step<kDppHalfMirror, 0xf>(v);
    v = dpp_max_step<kDppMirror, 0xf>(v);
    v = dpp_max_step<kDppBcast15, 0xa>(v);
    v = dpp_max_step<kDppBcast31, 0xc>(v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

// A DPP move whose unreached lanes get `fill` (the identity of the caller's
// operation) instead of 0.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_move_f(float v, float fill) {
    return __int_as_float(__builtin_amdgcn_update_dpp(__float_as_int(fill), __float_as_int(v),
                                                      kCtrl, kRowMask, 0xf, false));
}

__device__ __forceinline__ float wave_max_f32(float v) {
    v = fmaxf(v, dpp_move_f<kDppQuadSwap1, 0xf>(v, -INFINITY));
    v = fmaxf(v, dpp_move_f<kDppQuadSwap2, 0xf>(v, -INFINITY));
    v = fmaxf(v, dpp_move_f<kDppHalfMirror, 0xf>(v, -INFINITY));
    v = fmaxf(v, dpp_move_f<kDppMirror, 0xf>(v, -INFINITY));
    v = fmaxf(v, dpp_move_f<kDppBcast15, 0xa>(v, -INFINITY));
    v = fmaxf(v, dpp_move_f<kDppBcast31, 0xc>(v, -INFINITY));
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 63));
}

// Inclusive prefix sum of floats over the lanes, in a fixed association.
__device__ __forceinline__ float wave_incl_scan_f32(float x) {
    x += dpp_move_f<kDppShr1, 0xf>(x, 0.f);
    x += dpp_move_f<kDppShr1 + 1, 0xf>(x, 0.f);
    x += dpp_move_f<kDppShr1 + 3, 0xf>(x, 0.f);
    x += dpp_move_f<kDppShr1 + 7, 0xf>(x, 0.f);
    x += dpp_move_f<kDppBcast15, 0xa>(x, 0.f);
    x += dpp_move_f<kDppBcast31, 0xc>(x, 0.f);
    return x;
}

// Exclusive prefix sum over the lanes (shifts by 1, 2, 4, 8 within each row
// of 16, then the row broadcasts); `total` gets the wave's sum.
__device__ __forceinline__ int wave_excl_scan(int v, int &total) {
    int x = v;
    x += dpp_move<kDppShr1, 0xf>(x);
    x += dpp_move<kDppShr1 + 1, 0xf>(x);
    x += dpp_move<kDppShr1 + 3, 0xf>(x);
    x += dpp_move<kDppShr1 + 7, 0xf>(x);
    x += dpp_move<kDppBcast15, 0xa>(x);
    x += dpp_move<kDppBcast31, 0xc>(x);
    total = __builtin_amdgcn_readlane(x, 63);
    return x - v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    int l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

// Loads of data read exactly once per call (logits rows, candidate hidden
// rows): the nontemporal hint streams them past the caches, which measurably
// raises the HBM read rate on gfx950.  (The attention gathers are not in this
// class: nearby candidates share 128-byte lines of weights.)
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const uint4 *p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Copies n 16-byte chunks from global memory straight into LDS (block-wide)
// with global_load_lds_dwordx4: no registers are held, the copy runs while the
// block does other work, and it is complete after the block's next
// `s_waitcnt vmcnt(0)` + barrier.  Lane l of a wave lands at the wave's LDS
// base + 16 l, so the chunks land in order.
__device__ __forceinline__ void copy_to_lds(const uint4 *g, uint4 *lds, int n) {
    const int lane = threadIdx.x & (kWave - 1);
    for (int i0 = (int)(threadIdx.x - lane); i0 < n; i0 += (int)blockDim.x) {
        if (i0 + lane < n)
            __builtin_amdgcn_global_load_lds(
                (const void *)(g + i0 + lane),
                (__attribute__((address_space(3))) void *)(lds + i0), 16, 0, 0);
    }
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// ------------------------------------------------------- cosine pieces
// Dot products and squared norms of bf16 rows against the bf16 query row in
// LDS, with the gfx950 bf16 dot instruction (v_dot2c_f32_bf16: two bf16
// products added to an fp32 accumulator).  Lane l owns the 8-element chunks
// l, l+64, l+128, ... of a row, in that order; pair p of a chunk accumulates
// into acc[p]; the four accumulators are added as (a0+a1)+(a2+a3) and then
// summed across the wave by a butterfly.  The order depends only on d, so a
// row gives the same bits whichever slot, wave, block or kernel scores it,
// and a row equal to the query gives a dot product equal to both norms.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                           __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ __forceinline__ void accum_chunk(const uint4 &h, const uint4 &q, float (&ad)[4],
                                            float (&an)[4]) {
    ad[0] = dot2(h.x, q.x, ad[0]);
    ad[1] = dot2(h.y, q.y, ad[1]);
    ad[2] = dot2(h.z, q.z, ad[2]);
    ad[3] = dot2(h.w, q.w, ad[3]);
    an[0] = dot2(h.x, h.x, an[0]);
    an[1] = dot2(h.y, h.y, an[1]);
    an[2] = dot2(h.z, h.z, an[2]);
    an[3] = dot2(h.w, h.w, an[3]);
}

__device__ __forceinline__ void finish_row(const float (&ad)[4], const float (&an)[4], float &dot,
                                           float &nrm) {
    dot = wave_sum_f32((ad[0] + ad[1]) + (ad[2] + ad[3]));
    nrm = wave_sum_f32((an[0] + an[1]) + (an[2] + an[3]));
}

// One row of any width: up to 16 chunks per lane requested at once.  `row`
// is either the LDS copy of the query (kStream false) or a candidate row in
// HBM read once (kStream true).
template <bool kStream>
__device__ __forceinline__ void row_dot(const uint4 *row, const uint4 *q, int nch, float &dot,
                                        float &nrm) {
    constexpr int U = 16;
    const int lane = lane_id();
    float ad[4] = {0.f, 0.f, 0.f, 0.f}, an[4] = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = lane; c0 < nch; c0 += kWave * U) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ch = c0 + u * kWave;
            if (ch < nch) v[u] = kStream ? ld_stream(row + ch) : row[ch];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ch = c0 + u * kWave;
            if (ch < nch) accum_chunk(v[u], q[ch], ad, an);
        }
    }
    finish_row(ad, an, dot, nrm);
}

// The query row's squared norm from its LDS copy, in row_dot's order (lane l:
// chunks l, l+64, ..., pair p into acc[p]) with one chunk in hand at a time,
// so that it costs few registers; the same bits as row_dot(q, q).
__device__ __forceinline__ float query_norm(const uint4 *q, int nch) {
    float ad[4] = {0.f, 0.f, 0.f, 0.f}, an[4] = {0.f, 0.f, 0.f, 0.f};
    for (int ch = lane_id(); ch < nch; ch += kWave) {
        const uint4 v = q[ch];
        accum_chunk(v, v, ad, an);
    }
    float dot, nrm;
    finish_row(ad, an, dot, nrm);
    return nrm;
}

// G rows of width nch <= 64 * (16 / G) chunks, all their loads requested at
// once; a row whose pointer is null is skipped (its results are 0).
template <int G>
__device__ __forceinline__ void rows_dot(const uint4 *const (&rows)[G], const uint4 *q, int nch,
                                         float (&dot)[G], float (&nrm)[G]) {
    constexpr int U = 16 / G;
    const int lane = lane_id();
    uint4 v[G][U];
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int ch = lane + u * kWave;
            if (rows[g] && ch < nch) v[g][u] = ld_stream(rows[g] + ch);
        }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
        float ad[4] = {0.f, 0.f, 0.f, 0.f}, an[4] = {0.f, 0.f, 0.f, 0.f};
        if (rows[g]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int ch = lane + u * kWave;
                if (ch < nch) accum_chunk(v[g][u], q[ch], ad, an);
            }
        }
        finish_row(ad, an, dot[g], nrm[g]);
    }
}

// Rows streamed through a two-deep pipeline of pieces.  A piece is 64 kU
// chunks of 8 bf16 (kU 16-byte loads per lane, lane l taking chunks l, l+64,
// ... of the piece; 4 KB for kU = 4); a row is kPieces pieces.  The callers
// split a row in two (kPieces = 2: kU = 4 for d = 4096, 8 for d = 8192), the
// fastest of the piece sizes measured for both widths.
// The wave keeps the loads of the next piece in flight while it reduces the
// current one, so its memory queue never drains between rows the way a
// load-all-then-wait round does.  The accumulation order is row_dot's (lane l
// visits its chunks l, l+64, l+128, ... in order, pair p of a chunk into
// acc[p]), so a row gives the same bits here as through row_dot / rows_dot.
// `row(k)` gives the k-th row (k < n) of this wave, or null for an unusable
// one (its results are reported as not valid); `done(k, valid, dot, nrm)` runs
// in every lane when row k is complete, in order of k.
template <int kPieces, int kU, class RowPtr, class Done>
__device__ __forceinline__ void stream_rows(int n, RowPtr row, const uint4 *q, Done done) {
    constexpr int kPiece = kU * kWave;    // chunks per piece (kU 16-byte loads per lane)
    const int lane = lane_id();
    const int total = n * kPieces;
    uint4 buf[2][kU];
    float ad[4] = {0.f, 0.f, 0.f, 0.f}, an[4] = {0.f, 0.f, 0.f, 0.f};
    auto issue = [&](int slot, int pc) {
        const uint4 *r = row(pc / kPieces);
        if (r) {
            const uint4 *src = r + (pc % kPieces) * kPiece + lane;
#pragma unroll
            for (int u = 0; u < kU; ++u) buf[slot][u] = ld_stream(src + u * kWave);
        }
    };
    auto consume = [&](int slot, int pc) {
        const int k = pc / kPieces, p = pc % kPieces;
        const bool ok = row(k) != nullptr;
        if (p == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) ad[i] = an[i] = 0.f;
        }
        if (ok) {
            const uint4 *qq = q + p * kPiece + lane;
#pragma unroll
            for (int u = 0; u < kU; ++u) accum_chunk(buf[slot][u], qq[u * kWave], ad, an);
        }
        if (p == kPieces - 1) {
            float dot, nrm;
            finish_row(ad, an, dot, nrm);
            done(k, ok, dot, nrm);
        }
    };
    if (total > 0) issue(0, 0);
    if (total > 1) issue(1, 1);
    for (int pc = 0; pc < total; pc += 2) {
        consume(0, pc);
        if (pc + 2 < total) issue(0, pc + 2);
        if (pc + 1 < total) {
            consume(1, pc + 1);
            if (pc + 3 < total) issue(1, pc + 3);
        }
    }
}

// Aggregated attention of one candidate (Eq. 3 / Sec. 7.1), gathered by a
// group of kGatherLanes consecutive lanes: lane t of the group reads the
// weights A[r][j-1] of rows r = t, t+8, t+16, ... (col = &A[0][j-1], rows ar
// apart), up to 8 of them requested at once, and sums them in that order in
// fp32 (or takes their maximum); the group's eight partials are then combined
// by DPP moves inside the group (lane xor 1, xor 2, then the half-row mirror),
// which leaves the same bits in every lane of the group.  A candidate's R loads
// are thus one trip to memory for R <= 64.  Plain (cached) loads: candidates
// a few positions apart read the same 128-byte lines, and a line kept in L2
// serves the second one.  Call with the whole wave converged; `active` masks
// the loads of lanes without a candidate.
constexpr int kGatherLanes = 8;
__device__ __forceinline__ float attn_gather_group(const float *col, int64_t ar, int R, bool sum,
                                                   bool active) {
    const int t = lane_id() & (kGatherLanes - 1);
    const float none = sum ? 0.f : -INFINITY;
    float acc = none;
    for (int r0 = 0; r0 < R; r0 += 8 * kGatherLanes) {
        float v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int r = r0 + u * kGatherLanes + t;
            v[u] = (active && r < R) ? col[(int64_t)r * ar] : none;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = sum ? acc + v[u] : fmaxf(acc, v[u]);
    }
    const float x1 = dpp_move_f<kDppQuadSwap1, 0xf>(acc, none);
    acc = sum ? acc + x1 : fmaxf(acc, x1);
    const float x2 = dpp_move_f<kDppQuadSwap2, 0xf>(acc, none);
    acc = sum ? acc + x2 : fmaxf(acc, x2);
    const float x4 = dpp_move_f<kDppHalfMirror, 0xf>(acc, none);
    return sum ? acc + x4 : fmaxf(acc, x4);
}

// The choice j* of a sequence from its best ranking key (0: no eligible
// candidate) and its draft (Sec. 4.3): L = min(K, T-1-j*) when the length is
// valid and 0 <= j* <= T-2, else 0; draft[i] = x[j*+1+i] for i < L, -1 after.
// One wave; `x` is the sequence's token row (global memory or its LDS copy),
// the outputs point at the sequence's own entries.
__device__ __forceinline__ void write_choice_draft(uint64_t best, int64_t T, bool tok_ok,
                                                   const int32_t *x, int K, int32_t *best_pos,
                                                   float *best_score, int32_t *draft,
                                                   int32_t *draft_len) {
    const int lane = lane_id();
    const int32_t bp = best ? (int32_t)(uint32_t)(best & 0xffffffffu) : -1;
    if (lane == 0) {
        *best_pos = bp;
        *best_score = best ? unord_f32((uint32_t)(best >> 32)) : -INFINITY;
    }
    int64_t L = 0;
    if (tok_ok && bp >= 0 && (int64_t)bp <= T - 2) L = min((int64_t)K, T - 1 - bp);
    for (int i = lane; i < K; i += kWave) draft[i] = (i < L) ? x[bp + 1 + i] : -1;
    if (lane == 0) *draft_len = (int32_t)L;
}

// Eq. 2's cosine from the dot product and the two squared norms; the clamp
// is the usual eps = 1e-8 guard (eps^2 on the product of squared norms).
__device__ __forceinline__ float cosine(float dot, float hh, float qq) {
    return dot / sqrtf(fmaxf(hh * qq, 1e-16f));
}

}  // namespace pld
