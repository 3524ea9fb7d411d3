// pld_verify.h -- pieces shared by greedy verification (pld_verify.hip) and
// sampling verification (pld_sample.hip): the logits row layout, the element
// types, the acceptance of one sequence by one wave (Sec. 4.4) and the host
// checks of the logits arguments.
#pragma once

#include <stddef.h>
#include <stdint.h>

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

#ifndef PLD_ARGMAX_UNROLL
#define PLD_ARGMAX_UNROLL 11         // 16-byte loads per thread per batch of the argmax
#endif

constexpr int kVerifyThreads = 256;
constexpr int kVerifyWaves = kVerifyThreads / kWave;
constexpr int kVerifyUnroll = PLD_VERIFY_UNROLL;   // sampling statistics (its segment size)
constexpr int kArgmaxUnroll = PLD_ARGMAX_UNROLL;

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

// The largest of n values by the NaN-propagating maximum (three inputs per
// instruction on gfx950; -0 < +0, which only decides which zero is kept).
template <int n>
__device__ __forceinline__ float vmax_of(const float (&f)[n]) {
    float m = f[0];
#pragma unroll
    for (int e = 1; e < n; ++e) m = __builtin_elementwise_maximum(m, f[e]);
    return m;
}

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
    __device__ static float vmax(const uint4 &v) {
        float o[4];
        unpack(v, o);
        return vmax_of(o);
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
    __device__ static float vmax(const uint4 &v) {
        float o[8];
        unpack(v, o);
        return vmax_of(o);
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

// The accepted length a (-1 for an invalid draft length) and the model's
// token y_a, the same in every lane of the wave.
struct Accepted {
    int acc;
    int32_t y;
};

// Acceptance of one sequence by one wave, one lane per row: the first
// mismatch by a ballot, then the emitted tokens (Sec. 4.4).  `row_token(r)`
// gives y_r for r <= K (its value past L is not used); it is called for every
// r <= K of a round before the draft entries are compared.  `draft_token(r)`
// gives draft[r] for r < K and -1 for r = K; lane l asks for r = l, l+64, ...
template <class RowToken, class DraftToken>
__device__ __forceinline__ Accepted accept_wave(int K, int L, RowToken row_token,
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
    return Accepted{acc, y_acc};
}

// The ranking and verification calls share the leading, zero-invariant part
// of a workspace; the sampling statistics come after it.
inline size_t common_ws_bytes(int B, int K) {
    const size_t r = rank_ws_bytes(B);
    const size_t v = verify_ws_bytes(B, K);
    return r > v ? r : v;
}
// Host checks shared by the verification calls (logits, strides, lengths,
// the key region of the workspace) and the argmax launch shape.
int prep_verify(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride, int V,
                int K, const int32_t *draft_len, int B, void *workspace, size_t workspace_bytes,
                VerifyArgs &a);

}  // namespace pld
