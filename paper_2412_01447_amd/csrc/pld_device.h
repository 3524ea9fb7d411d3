// pld_device.h -- device helpers shared by the PLD+ kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Scratch of the multi-block find: per-tile occurrence counts of every n.
inline size_t find_scratch_bytes(int B, int64_t tok_stride) {
    if (tok_stride <= kFindFusedMax) return 0;
    const int64_t ntiles = (tok_stride + kFindTile - 1) / kFindTile;
    return align_up((size_t)B * (size_t)ntiles * 8 * sizeof(int32_t), 256);
}
// Workspace of the ranking and verification calls: 64-bit keys that must be
// zero when a call starts and that the call leaves zero.
inline size_t rank_ws_bytes(int B) { return align_up((size_t)B * sizeof(uint64_t), 256); }
inline size_t verify_ws_bytes(int B, int K) {
    return align_up((size_t)B * (size_t)(K + 1) * sizeof(uint64_t), 256);
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

__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int m) {
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    lo = (uint32_t)__shfl_xor((int)lo, m);
    hi = (uint32_t)__shfl_xor((int)hi, m);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
        uint64_t o = shfl_xor_u64(v, m);
        v = o > v ? o : v;
    }
    return v;
}

// Butterfly sum: every lane ends with the same, bit-identical total, and the
// association depends only on the lane layout, never on the data.
__device__ __forceinline__ float wave_sum_f32(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
    return v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
    int l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

}  // namespace pld
