// pld_verify.hip -- greedy verification (arXiv 2412.01447, Sec. 3 "greedy
// acceptance" and Sec. 4.4) and draft emission (Sec. 4.3).
//
// Verification: y_i = argmax_v Z[b][i][v] for the rows i <= L = draft_len[b]
// (lowest v among equal maxima, -0 == +0), then the accepted length is the
// first i < L with y_i != draft[b][i] (else L), and the step emits the
// accepted draft prefix followed by y_a.
//
// The argmax is a streaming read of the logits, so the kernel is shaped for
// HBM: every row is split across S blocks (picked on the host: as many per
// row as are resident together when each block's share then fits one batch
// of loads, otherwise about PLD_VERIFY_TARGET_BLOCKS blocks in all), each
// thread issues 16-byte loads (4 fp32 or 8 bf16) in batches of
// PLD_ARGMAX_UNROLL, keeps the first maximum of its own elements, and the
// wave / block reduce the 64-bit key (orderable(value) << 32 | ~index), whose
// maximum is the highest value with the lowest index.  A block folds its key
// into the row's workspace slot with one 64-bit atomic max.  A small
// acceptance kernel, launched right after on the same stream (the kernel
// boundary orders the two), reads the row keys back with one wave per
// sequence (a lane per row), computes the accepted length, writes the outputs
// and returns the slots to zero.  Rows i > L never reach a slot: a block requests its
// first batch of loads before the draft length arrives (the latency of that
// read is then hidden) and returns once it sees that its row is past the
// draft, so every row of the buffer must be readable, and rows past a short
// draft are read in part or in full.
//
// Also here: the commit of the generation loop and the library-wide calls
// (version, status strings, workspace sizes).  Sampling verification is in
// pld_sample.hip; the pieces both use are in pld_verify.h.
#include <math.h>

#include <mutex>

#include "pld.h"
#include "pld_device.h"
#include "pld_verify.h"

namespace pld {

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
    uint4 r[kArgmaxUnroll];
#pragma unroll
    for (int u = 0; u < kArgmaxUnroll; ++u) {
        const int64_t vi = my_v + (int64_t)u * kVerifyThreads;
        if (vi < v1) r[u] = ld_stream(vec + vi);
    }
    const int L = a.draft_len[b];
    if (L < 0 || L > a.K || i > L) return;   // rows past the draft are not used

    // Each thread keeps the first maximum of its own elements, which it visits
    // in increasing index order: a later element replaces the best only when
    // strictly greater (so an equal value, or -0 after +0, never does).  The
    // index starts at the thread's first element, so a thread whose elements
    // are all -inf still reports its first one.  The body is taken a 16-byte
    // vector at a time: the vector's maximum (three values per maximum
    // instruction) decides whether the vector replaces the kept one, and the
    // first element equal to the kept maximum is found once, at the end --
    // the same element as a scan of every element, with a third of its
    // vector instructions (bf16 rows are compute-heavy enough to notice).
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
    float vbest = -INFINITY;
    uint4 bvec = make_uint4(0u, 0u, 0u, 0u);
    int bvi = -1;
    for (int64_t vb = my_v; vb < v1; vb += (int64_t)kVerifyThreads * kArgmaxUnroll) {
        if (vb != my_v) {
#pragma unroll
            for (int u = 0; u < kArgmaxUnroll; ++u) {
                const int64_t vi = vb + (int64_t)u * kVerifyThreads;
                if (vi < v1) r[u] = ld_stream(vec + vi);
            }
        }
#pragma unroll
        for (int u = 0; u < kArgmaxUnroll; ++u) {
            const int64_t vi = vb + (int64_t)u * kVerifyThreads;
            if (vi < v1) {
                const float m = E::vmax(r[u]);
                if (m > vbest) {
                    vbest = m;
                    bvec = r[u];
                    bvi = (int)vi;
                }
            }
        }
    }
    if (bvi >= 0 && vbest > best) {
        float f[P];
        E::unpack(bvec, f);
        int e0 = P - 1;
#pragma unroll
        for (int e = P - 1; e >= 0; --e)
            if (f[e] == vbest) e0 = e;
        best = vbest;
        bi = (uint32_t)(head + (int64_t)bvi * P + e0);
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

// The acceptance of sequence b by one wave: y_i from the row keys, which are
// returned to zero.  Every slot exists whatever the length, and the argmax
// never writes a slot past the draft, so those are zero already and zeroing
// all K+1 is the same.
__device__ __forceinline__ Accepted accept_from_keys(const VerifyArgs &a, int b) {
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
    return accept_wave(K, L, key_token, draft_token, a.out_tokens + (int64_t)b * (K + 1),
                       a.accept_len + b, a.out_count + b);
}

// One wave per sequence: the acceptance after the argmax launch.
__global__ __launch_bounds__(256) void verify_accept_kernel(VerifyArgs a) {
    const int b = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
    if (b >= a.B) return;   // wave-uniform
    accept_from_keys(a, b);
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

struct CommitArgs {
    int32_t *tokens;
    int64_t tok_stride;
    int32_t *lens;
    const int32_t *limit;
    int64_t *stats;
};

// The acceptance and then the commit of sequence b by the same wave
// (pld_accept_commit): the outputs of verify_accept_kernel followed by
// commit_kernel, with the committed tokens taken from the draft and y_a
// directly instead of being read back from out_tokens.
__global__ __launch_bounds__(256) void accept_commit_kernel(VerifyArgs a, CommitArgs c) {
    const int b = (int)((blockIdx.x * (int64_t)blockDim.x + threadIdx.x) / kWave);
    const int lane = lane_id();
    if (b >= a.B) return;   // wave-uniform
    const Accepted r = accept_from_keys(a, b);
    int64_t cap = c.tok_stride;
    if (c.limit && c.limit[b] < cap) cap = c.limit[b];
    const int64_t T = c.lens[b];
    const int64_t n = r.acc >= 0 ? r.acc + 1 : 0;   // out_count
    if (T < 0 || T > cap) return;
    const int64_t m = min(n, cap - T);
    const int32_t *dr = a.draft + (int64_t)b * a.K;
    for (int64_t i = lane; i < m; i += kWave)
        c.tokens[(int64_t)b * c.tok_stride + T + i] = i < r.acc ? dr[i] : r.y;
    if (lane == 0) {
        c.lens[b] = (int32_t)(T + m);
        if (c.stats) {
            c.stats[2 * b] += m;
            c.stats[2 * b + 1] += m > 0 ? 1 : 0;
        }
    }
}

// The checks of the logits arguments (everything but the workspace).
static int check_verify(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                        int V, int K, const int32_t *draft_len, int B) {
    if (!logits || !draft_len) return PLD_ERR_INVALID;
    if (B < 1 || K < 1 || V < 1 || (dtype != PLD_F32 && dtype != PLD_BF16)) return PLD_ERR_INVALID;
    if (B > 65535 || K > 65534) return PLD_ERR_INVALID;           // grid y / z limits
    if (l_row_stride < V || l_seq_stride < (int64_t)(K + 1) * l_row_stride) return PLD_ERR_INVALID;
    const size_t esz = dtype == PLD_F32 ? 4 : 2;
    if ((uintptr_t)logits % esz) return PLD_ERR_ALIGN;
    return PLD_OK;
}

int prep_verify(const void *logits, int dtype, int64_t l_seq_stride, int64_t l_row_stride,
                int V, int K, const int32_t *draft_len, int B, void *workspace,
                size_t workspace_bytes, VerifyArgs &a) {
    const int rc = check_verify(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B);
    if (rc != PLD_OK) return rc;
    const size_t esz = dtype == PLD_F32 ? 4 : 2;
    if (!workspace || workspace_bytes < verify_ws_bytes(B, K)) return PLD_ERR_WORKSPACE;
    // Blocks per row.  When every block can take its share of a row in one
    // batch of loads with the whole grid resident at once, as many blocks per
    // row as fit on the GPU together (a grid a little larger than what is
    // resident would run its last blocks in a second round, one whole block
    // duration later); otherwise, for rows that need several batches per
    // thread anyway, about PLD_VERIFY_TARGET_BLOCKS blocks in all.  Each
    // block keeps at least two 16-byte vectors per thread.
    const int64_t rows = (int64_t)B * (K + 1);
    const int64_t nvec = (int64_t)V * esz / 16;
    const void *kern = dtype == PLD_F32
        ? reinterpret_cast<const void *>(&verify_argmax_kernel<0>)
        : reinterpret_cast<const void *>(&verify_argmax_kernel<1>);
    const int64_t fit = resident_blocks(kern, kVerifyThreads, 0) / rows;
    int64_t S = (PLD_VERIFY_TARGET_BLOCKS + rows - 1) / rows;
    if (fit >= 1 && (nvec + fit - 1) / fit <= (int64_t)kArgmaxUnroll * kVerifyThreads) S = fit;
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

// ------------------------------------------------ allocation-free variant
// pld_verify_greedy_noalloc keeps the row keys in this file-scope device
// array instead of a caller's workspace.  Each GPU holds its own copy, at its
// own address, which the host learns once per device from
// hipGetSymbolAddress; in host code the array's name is only a stand-in and
// is never passed to a kernel.  Every call on a GPU shares that GPU's array.
constexpr int kStaticKeys = 65536;                  // B*(K+1) limit: 512 KiB per GPU
static __device__ __align__(256) uint64_t scratch[kStaticKeys];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static uint64_t *g_scratch_addr[kMaxDevices] = {};

// The device address of `scratch` on the current device (looked up on the
// first call made with that device current, then kept).
static int scratch_address(uint64_t **out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PLD_ERR_LAUNCH;
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PLD_ERR_LAUNCH;
        g_scratch_addr[dev] = reinterpret_cast<uint64_t *>(p);
    }
    *out = g_scratch_addr[dev];
    return PLD_OK;
}

// The keys the argmax folds into must start at zero: a fill kernel (rather
// than a memset node) clears the n slots this call uses.
__global__ __launch_bounds__(256) void clear_keys_kernel(uint64_t *keys, int n) {
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i < n) keys[i] = 0;
}

}  // namespace pld

using namespace pld;

extern "C" int pld_verify_greedy_noalloc(const void *logits, int dtype, int64_t l_seq_stride,
                                         int64_t l_row_stride, int V, int K, const int32_t *draft,
                                         const int32_t *draft_len, int B, int32_t *accept_len,
                                         int32_t *out_tokens, int32_t *out_count, void *stream) {
    if (!draft || !accept_len || !out_tokens || !out_count) return PLD_ERR_INVALID;
    int rc = check_verify(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B);
    if (rc != PLD_OK) return rc;
    if ((int64_t)B * ((int64_t)K + 1) > kStaticKeys) return PLD_ERR_SCRATCH;
    uint64_t *keys = nullptr;
    rc = scratch_address(&keys);
    if (rc != PLD_OK) return rc;
    VerifyArgs a;
    rc = prep_verify(logits, dtype, l_seq_stride, l_row_stride, V, K, draft_len, B, keys,
                     (size_t)kStaticKeys * sizeof(uint64_t), a);
    if (rc != PLD_OK) return rc;
    a.draft = draft;
    a.accept_len = accept_len;
    a.out_tokens = out_tokens;
    a.out_count = out_count;
    const int n = B * (K + 1);
    hipLaunchKernelGGL(clear_keys_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       (hipStream_t)stream, keys, n);
    launch_argmax(a, dtype, (hipStream_t)stream);
    launch_accept(a, (hipStream_t)stream);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

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
    if (B < 1 || K < 1 || B > 65535 || K > 65534) return PLD_ERR_INVALID;
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

extern "C" int pld_accept_commit(const int32_t *draft, const int32_t *draft_len, int B, int K,
                                 int32_t *accept_len, int32_t *out_tokens, int32_t *out_count,
                                 int32_t *tokens, int64_t tok_stride, int32_t *lens,
                                 const int32_t *limit, int64_t *stats, void *workspace,
                                 size_t workspace_bytes, void *stream) {
    if (!draft || !draft_len || !accept_len || !out_tokens || !out_count || !tokens || !lens)
        return PLD_ERR_INVALID;
    if (B < 1 || K < 1 || B > 65535 || K > 65534) return PLD_ERR_INVALID;
    if (tok_stride < 1 || tok_stride > kMaxTokStride) return PLD_ERR_INVALID;
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
    const CommitArgs c{tokens, tok_stride, lens, limit, stats};
    hipLaunchKernelGGL(accept_commit_kernel, dim3((unsigned)((B + 3) / 4)), dim3(256), 0,
                       (hipStream_t)stream, a, c);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_commit(int32_t *tokens, int64_t tok_stride, int32_t *lens,
                          const int32_t *limit, const int32_t *out_tokens,
                          const int32_t *out_count, int B, int K, int64_t *stats, void *stream) {
    if (!tokens || !lens || !out_tokens || !out_count) return PLD_ERR_INVALID;
    if (B < 1 || B > 65535 || K < 1 || K > 65534) return PLD_ERR_INVALID;
    if (tok_stride < 1 || tok_stride > kMaxTokStride) return PLD_ERR_INVALID;
    hipLaunchKernelGGL(commit_kernel, dim3((unsigned)((B + 3) / 4)), dim3(256), 0,
                       (hipStream_t)stream, tokens, tok_stride, lens, limit, out_tokens,
                       out_count, B, K, stats);
    return hipGetLastError() == hipSuccess ? PLD_OK : PLD_ERR_LAUNCH;
}

extern "C" int pld_version(void) { return PLD_ABI_VERSION; }

extern "C" const char *pld_status_string(int status) {
    switch (status) {
    case PLD_OK: return "ok";
    case PLD_ERR_INVALID: return "invalid argument";
    case PLD_ERR_ALIGN: return "misaligned pointer or stride";
    case PLD_ERR_WORKSPACE: return "workspace missing or too small";
    case PLD_ERR_LAUNCH: return "kernel launch failed";
    case PLD_ERR_SCRATCH: return "sizes exceed the static scratch of the allocation-free call";
    default: return "unknown status";
    }
}

extern "C" size_t pld_workspace_bytes(int B, int K) {
    if (B < 1 || K < 1) return 0;
    return common_ws_bytes(B, K);
}
