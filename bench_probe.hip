// bench_probe.hip -- read-bandwidth ceilings of the access patterns the
// drafting step's kernels use, measured from HBM on this GPU (a companion of
// bench.py: `python bench.py --probe` runs it; the kernels of the library are
// not involved).  Every pattern rotates through inputs larger than the 256 MB
// last-level cache, so no repetition is served from it.  One JSON line per
// pattern on stdout; times are means over batches of back-to-back launches.
//
//   stream   block-contiguous 16-byte loads over 1 GiB (8 per thread in flight);
//            stream_279mb / stream_68mb the same at the verification logits sizes
//   rows8k   random 8 KB rows, 106 MB per launch (the hidden rows of the b4 x
//            131072 workload), 2 rows of 8 loads per wave in flight
//   rows16k  random 16 KB rows, 380 MB per launch (the b64 x 16384 workload)
//   columns  one 4-byte value from each of 64 rows 64 KB apart per lane, for
//            285 random columns of each of 64 sequences (the attention gathers
//            of the b64 workload); bytes counted as distinct 128-byte lines
//   gather_b32_tripsN  the attention gathers of the b32 x 8192 workload (~10 MB
//            of distinct lines) behind N = 1, 2 or 3 dependent trips to memory
//   strideS  4M 4-byte reads S bytes apart (S = 32 .. 512), consecutive lanes
//            on consecutive addresses: the time per read shows the granule the
//            memory system fetches for scattered 4-byte loads
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#define CK(x)                                                                            \
    do {                                                                                 \
        hipError_t e_ = (x);                                                             \
        if (e_ != hipSuccess) {                                                          \
            std::fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
            std::exit(1);                                                                \
        }                                                                                \
    } while (0)

typedef unsigned v4u __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(256) void stream_kernel(const v4u *p, size_t per_block, v4u *sink) {
    const v4u *b = p + (size_t)blockIdx.x * per_block;
    v4u acc = {0, 0, 0, 0};
    for (size_t i = threadIdx.x; i < per_block; i += 256 * 8) {
        v4u v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(b + i + (size_t)u * 256);
#pragma unroll
        for (int u = 0; u < 8; ++u) acc ^= v[u];
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

template <int G, int U>
__global__ __launch_bounds__(256) void rows_kernel(const v4u *buf, int row_vecs, const int *idx,
                                                   int m, v4u *sink) {
    const int lane = threadIdx.x & 63;
    const int wave = (int)((blockIdx.x * blockDim.x + threadIdx.x) >> 6);
    const int nw = (int)((gridDim.x * blockDim.x) >> 6);
    v4u acc = {0, 0, 0, 0};
    for (int r0 = wave * G; r0 < m; r0 += nw * G) {
        v4u v[G][U];
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const v4u *row = buf + (size_t)idx[min(r0 + g, m - 1)] * row_vecs;
#pragma unroll
            for (int u = 0; u < U; ++u) v[g][u] = __builtin_nontemporal_load(row + lane + u * 64);
        }
#pragma unroll
        for (int g = 0; g < G; ++g)
#pragma unroll
            for (int u = 0; u < U; ++u) acc ^= v[g][u];
    }
    if ((acc.x ^ acc.y ^ acc.z ^ acc.w) == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

__global__ __launch_bounds__(256) void columns_kernel(const float *buf, int R, int N,
                                                      const int *col, int C, int S, float *sink) {
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i >= S * C) return;
    const float *p = buf + (size_t)(i / C) * R * N + col[i];
    float acc = 0.f;
    for (int r0 = 0; r0 < R; r0 += 32) {
        float v[32];
#pragma unroll
        for (int u = 0; u < 32; ++u) v[u] = __builtin_nontemporal_load(p + (size_t)(r0 + u) * N);
#pragma unroll
        for (int u = 0; u < 32; ++u) acc += v[u];
    }
    if (acc == 12345.f) sink[i] = acc;
}

// The attention gathers of the b32 x 8192 workload (40 rows of 8192 keys per
// sequence, ~80 candidate columns each, ~10 MB of distinct 128-byte lines),
// with kTrips dependent trips to memory in the launch: 1 -- the columns are
// computed in registers; 2 -- read from a list first (the positions); 3 -- a
// per-sequence count read before the list (the counts, then the positions).
// A group of 8 lanes per column, lane t reading rows t, t+8, ... as the
// ranking kernels do.  The launch time against the bytes gives the fastest a
// single launch of this dependency structure can read them.
__device__ __forceinline__ int hashed_column(int s, int k, int N) {
    unsigned h = (unsigned)(s * 131071 + k * 8191 + 12345) * 2654435761u;
    return (int)((h >> 7) % (unsigned)(N - 1));
}

template <int kTrips>
__global__ __launch_bounds__(256) void gather_kernel(const float *buf, int R, int N, const int *col,
                                                     const int *count, int C, int S, float *sink) {
    const int g = (int)((blockIdx.x * blockDim.x + threadIdx.x) >> 3);
    const int t = threadIdx.x & 7;
    if (g >= S * C) return;
    const int s = g / C, k = g % C;
    int c;
    if constexpr (kTrips == 1) {
        c = hashed_column(s, k, N);
    } else if constexpr (kTrips == 2) {
        c = col[g];
    } else {
        const int n = count[s];
        c = k < n ? col[g] : 0;
    }
    const float *p = buf + (size_t)s * R * N + c;
    float v[8], acc = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        const int r = t + 8 * u;
        v[u] = r < R ? p[(size_t)r * N] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
    if (acc == 12345.f) sink[g] = acc;
}

__global__ __launch_bounds__(256) void strided_kernel(const float *p, size_t stride, float *sink) {
    const size_t n = (size_t)gridDim.x * blockDim.x;
    const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + ((size_t)u * n + i) * stride);
    float acc = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u) acc += v[u];
    if (acc == 12345.f) sink[i] = acc;
}

template <class Launch>
static double time_us(Launch launch, int nvariants) {
    hipEvent_t e0, e1;
    CK(hipEventCreate(&e0));
    CK(hipEventCreate(&e1));
    for (int r = 0; r < nvariants; ++r) launch(r);   // warm-up over every variant
    CK(hipDeviceSynchronize());
    // back-to-back launches between two events: each launch's dispatch overlaps
    // the previous kernel, so the mean approaches the kernel's own duration
    const int batches = 3, reps = 16;
    float total = 0.f;
    for (int t = 0; t < batches; ++t) {
        CK(hipEventRecord(e0, 0));
        for (int r = 0; r < reps; ++r) launch((r * 3 + 1 + t) % nvariants);
        CK(hipEventRecord(e1, 0));
        CK(hipEventSynchronize(e1));
        float ms;
        CK(hipEventElapsedTime(&ms, e0, e1));
        total += ms;
    }
    CK(hipEventDestroy(e0));
    CK(hipEventDestroy(e1));
    return total / (batches * reps) * 1e3;
}

static void report(const char *pattern, double bytes, double us) {
    std::printf("{\"pattern\": \"%s\", \"bytes\": %.0f, \"us\": %.2f, \"GBps\": %.1f, "
                "\"frac_of_8TBps\": %.4f}\n",
                pattern, bytes, us, bytes / (us * 1e-6) / 1e9, bytes / (us * 1e-6) / 8e12);
    std::fflush(stdout);
}

int main() {
    int cus = 0;
    CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
    const size_t buf_bytes = (size_t)8 << 30;
    v4u *buf;
    CK(hipMalloc(&buf, buf_bytes));
    CK(hipMemset(buf, 1, buf_bytes));
    v4u *sink;
    CK(hipMalloc(&sink, (size_t)1 << 24));

    // stream: 1 GiB per launch at 8 rotating offsets; then the same at the
    // logits sizes of the verification kernels (279 MB: b64 x 17 rows x 128256
    // bf16; 68 MB: b32 x 17 x 32000 fp32 and b4 x 33 x 128256 bf16), where the
    // launch's ramp-up and drain weigh more
    for (const size_t chunk : {(size_t)1 << 30, (size_t)279 << 20, (size_t)68 << 20}) {
        const size_t per = chunk / 16 / ((size_t)cus * 8) / 2048 * 2048;   // whole rounds
        const double us = time_us([&](int r) {
            hipLaunchKernelGGL(stream_kernel, dim3(cus * 8), dim3(256), 0, 0,
                               buf + (size_t)r * (((size_t)1 << 30) / 16), per, sink);
        }, 8);
        report(chunk == ((size_t)1 << 30) ? "stream" : chunk == ((size_t)279 << 20) ? "stream_279mb"
                                                                                  : "stream_68mb",
               (double)per * 16 * cus * 8, us);
    }
    std::mt19937_64 rng(7);
    const int nsets = 8;
    int *didx;
    CK(hipMalloc(&didx, (size_t)nsets * 65536 * sizeof(int)));
    for (int rb : {8192, 16384}) {   // random rows, 8 index sets
        const size_t nrows = buf_bytes / rb;
        const int m = (int)(((rb == 8192 ? (size_t)106 : (size_t)380) << 20) / rb);
        std::vector<int> h((size_t)nsets * m);
        for (auto &v : h) v = (int)(rng() % nrows);
        CK(hipMemcpy(didx, h.data(), h.size() * sizeof(int), hipMemcpyHostToDevice));
        const double us = time_us([&](int r) {
            if (rb == 8192)
                hipLaunchKernelGGL((rows_kernel<2, 8>), dim3(cus * 4), dim3(256), 0, 0, buf, rb / 16,
                                   didx + (size_t)r * m, m, sink);
            else
                hipLaunchKernelGGL((rows_kernel<1, 16>), dim3(cus * 8), dim3(256), 0, 0, buf, rb / 16,
                                   didx + (size_t)r * m, m, sink);
        }, nsets);
        report(rb == 8192 ? "rows8k" : "rows16k", (double)m * rb, us);
    }
    {   // scattered columns over 4 copies of [64][64][16384] fp32 (1 GiB)
        const int S = 64, R = 64, N = 16384, C = 285;
        const size_t n = (size_t)S * R * N;
        std::vector<int> h((size_t)nsets * S * C);
        size_t lines = 0;
        for (int t = 0; t < nsets; ++t)
            for (int s = 0; s < S; ++s) {
                int *c = h.data() + ((size_t)t * S + s) * C;
                for (int k = 0; k < C; ++k) c[k] = (int)(rng() % (N - 1));
                std::sort(c, c + C);
                int last = -1;
                for (int k = 0; k < C; ++k)
                    if (c[k] / 32 != last) {
                        lines += t == 0;
                        last = c[k] / 32;
                    }
            }
        CK(hipMemcpy(didx, h.data(), h.size() * sizeof(int), hipMemcpyHostToDevice));
        const float *fb = reinterpret_cast<const float *>(buf);
        const double us = time_us([&](int r) {
            hipLaunchKernelGGL(columns_kernel, dim3((S * C + 255) / 256), dim3(256), 0, 0,
                               fb + (size_t)(r % 4) * n, R, N, didx + (size_t)r * S * C, C, S,
                               reinterpret_cast<float *>(sink));
        }, nsets);
        report("columns", (double)lines * R * 128, us);
    }
    {   // the b32 x 8192 attention gathers: 1, 2 and 3 dependent trips per launch
        const int S = 32, R = 40, N = 8192, C = 80;
        const size_t n = (size_t)S * R * N;   // 42 MB per copy; 8 copies rotate past the LLC
        std::vector<int> h((size_t)S * C), cnt(S, C);
        size_t lines = 0;
        for (int s = 0; s < S; ++s) {
            std::vector<int> lk;
            for (int k = 0; k < C; ++k) {
                const unsigned hh = (unsigned)(s * 131071 + k * 8191 + 12345) * 2654435761u;
                h[(size_t)s * C + k] = (int)((hh >> 7) % (unsigned)(N - 1));
                lk.push_back(h[(size_t)s * C + k] / 32);
            }
            std::sort(lk.begin(), lk.end());
            lines += (size_t)(std::unique(lk.begin(), lk.end()) - lk.begin());
        }
        int *dcnt;
        CK(hipMalloc(&dcnt, S * sizeof(int)));
        CK(hipMemcpy(didx, h.data(), h.size() * sizeof(int), hipMemcpyHostToDevice));
        CK(hipMemcpy(dcnt, cnt.data(), S * sizeof(int), hipMemcpyHostToDevice));
        const float *fb = reinterpret_cast<const float *>(buf);
        const unsigned blocks = (unsigned)((S * C * 8 + 255) / 256);
        for (int trips = 1; trips <= 3; ++trips) {
            const double us = time_us([&](int r) {
                const float *src = fb + (size_t)r * n;
                float *sk = reinterpret_cast<float *>(sink);
                if (trips == 1)
                    hipLaunchKernelGGL(gather_kernel<1>, dim3(blocks), dim3(256), 0, 0, src, R, N,
                                       didx, dcnt, C, S, sk);
                else if (trips == 2)
                    hipLaunchKernelGGL(gather_kernel<2>, dim3(blocks), dim3(256), 0, 0, src, R, N,
                                       didx, dcnt, C, S, sk);
                else
                    hipLaunchKernelGGL(gather_kernel<3>, dim3(blocks), dim3(256), 0, 0, src, R, N,
                                       didx, dcnt, C, S, sk);
            }, 8);
            char name[32];
            std::snprintf(name, sizeof(name), "gather_b32_trips%d", trips);
            report(name, (double)lines * R * 128, us);
        }
        CK(hipFree(dcnt));
    }
    for (int stride : {32, 64, 128, 256, 512}) {   // 4M reads, spans of 128 MB to 2 GB
        const size_t reads = (size_t)1 << 22, threads = reads / 8;
        const size_t span = reads * stride;
        const int variants = (int)std::min<size_t>(4, buf_bytes / span);
        const float *fb = reinterpret_cast<const float *>(buf);
        const double us = time_us([&](int r) {
            hipLaunchKernelGGL(strided_kernel, dim3((unsigned)(threads / 256)), dim3(256), 0, 0,
                               fb + (size_t)r * (span / 4), (size_t)stride / 4,
                               reinterpret_cast<float *>(sink));
        }, variants);
        char name[32];
        std::snprintf(name, sizeof(name), "stride%d", stride);
        std::printf("{\"pattern\": \"%s\", \"reads\": %zu, \"us\": %.2f, \"ns_per_read\": %.4f, "
                    "\"GBps_if_64B\": %.1f, \"GBps_if_128B\": %.1f}\n",
                    name, reads, us, us * 1e3 / reads, reads * 64.0 / (us * 1e-6) / 1e9,
                    reads * 128.0 / (us * 1e-6) / 1e9);
        std::fflush(stdout);
    }
    CK(hipFree(didx));
    CK(hipFree(sink));
    CK(hipFree(buf));
    return 0;
}
