// stream_ceiling.hip -- measures the data-movement ceiling of this GPU for the
// access patterns of the optimizer steps, with no arithmetic:
//   mix (pattern "step8", the default): per element read 8 B (4 B weight, 2 B
//         gradient, 1 B + 1 B codes) and write 6 B back in place (weight, two
//         codes): the fused 8-bit step's traffic;
//   mix (pattern "step8_copy"): the same plus 2 B written to a separate array (the
//         bf16 weight copy): 8 B read, 8 B written;
//   mix (pattern "adamw32"): read 4 B weight, 2 B gradient, 4 B + 4 B moments and
//         write weight and moments back: 14 B read, 12 B written (the fp32-state step);
//   read: read 2 B per element (the bf16 gradient): the sum of squares' traffic.
// Same layout as the steps (separate arrays, 16-byte vector accesses).  The step8
// mix is timed in two shapes and the faster one is reported: one granule per thread
// per workgroup iteration over contiguous per-workgroup ranges, and wave tiles of 32
// elements per lane (a lane's granules 64 apart, as the step kernel lays them out)
// handed to the waves in turn.  The other two patterns are timed as wave tiles of 16
// and 32 elements per lane.  Prints one JSON line.
// Usage: stream_ceiling [n] [reps] [step8 | step8_copy | adamw32]
//
// Placement mode: stream_ceiling n reps step8|adamw32 sets K allocates K sets of
// the pattern's arrays, each array its own hipMalloc and all sets alive at once,
// and times the pattern (wave tiles of 32 elements per lane, 3 workgroups per CU)
// on each set, then on each set again.  Sets that differ only in where the
// allocator placed them show how much the rate depends on physical placement.
// Prints one JSON line per pass over the sets.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#define CK(x)                                                                       \
    do {                                                                            \
        hipError_t e_ = (x);                                                        \
        if (e_ != hipSuccess) {                                                     \
            fprintf(stderr, "%s: %s\n", #x, hipGetErrorString(e_));                 \
            return 1;                                                               \
        }                                                                           \
    } while (0)

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int64_t kIter = 2048;  // elements per workgroup iteration: 8 per thread

__device__ inline void range(int64_t iters, int64_t* b, int64_t* e)
{
    const int64_t per = iters / gridDim.x, rem = iters % gridDim.x, i = blockIdx.x;
    *b = i * per + (i < rem ? i : rem);
    *e = *b + per + (i < rem ? 1 : 0);
}

// Trivial integer work that changes every word the probes store.  A word stored
// unchanged lets the compiler (the pointers are restrict) drop it from the store and
// the load, which would leave partial lines and fewer bytes than the steps move.
__device__ inline void xor_words(uint4& x, const uint4& k)
{
    x.x ^= k.x | 1u;
    x.y ^= k.y | 1u;
    x.z ^= k.z | 1u;
    x.w ^= k.w | 1u;
}

__device__ inline void mix_words(uint4& w0, uint4& w1, uint2& m, uint2& v, const uint4& g)
{
    xor_words(w0, g);
    xor_words(w1, make_uint4(g.y, g.z, g.w, g.x));
    m.x ^= g.x | 1u;
    m.y ^= g.z | 1u;
    v.x ^= g.y | 1u;
    v.y ^= g.w | 1u;
}

// Elements [0, iters * 2048): granule gi (8 elements) is w[2gi..2gi+1], g[gi],
// m[gi], v[gi]; every access is inside its array.
__global__ __launch_bounds__(kThreads) void k_mix(uint4* __restrict__ w, const uint4* __restrict__ g,
                                                 uint2* __restrict__ m, uint2* __restrict__ v,
                                                 int64_t iters)
{
    int64_t b, e;
    range(iters, &b, &e);
    const int t = threadIdx.x;
    for (int64_t it = b; it < e; ++it) {
        const int64_t gi = it * kThreads + t;  // granule of 8 elements
        uint4 w0 = w[2 * gi], w1 = w[2 * gi + 1];
        const uint4 gg = g[gi];
        uint2 mm = m[gi], vv = v[gi];
        // every stored word changes, so no load or store can be narrowed
        mix_words(w0, w1, mm, vv, gg);
        w[2 * gi] = w0;
        w[2 * gi + 1] = w1;
        m[gi] = mm;
        v[gi] = vv;
    }
}

// Wave tiles: tile t covers granules [256 t, 256 (t + 1)); granule j of lane l is
// 256 t + l + 64 j (j = 0..3).  Tiles go to the waves in turn.  Every access is
// inside its array: the largest granule index is 256 * tiles - 1 = n / 8 - 1.
__global__ __launch_bounds__(kThreads) void k_mix_tiles(uint4* __restrict__ w,
                                                       const uint4* __restrict__ g,
                                                       uint2* __restrict__ m,
                                                       uint2* __restrict__ v, int64_t tiles)
{
    constexpr int G = 4;  // granules per lane: 32 elements
    const int lane = threadIdx.x & 63;
    const int64_t waves = int64_t(gridDim.x) * 4;
    for (int64_t t = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6); t < tiles; t += waves) {
        uint4 a[G], b[G], c[G];
        uint2 mm[G], vv[G];
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int64_t gi = t * (64 * G) + lane + 64 * j;
            a[j] = w[2 * gi];
            b[j] = w[2 * gi + 1];
            c[j] = g[gi];
            mm[j] = m[gi];
            vv[j] = v[gi];
        }
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int64_t gi = t * (64 * G) + lane + 64 * j;
            mix_words(a[j], b[j], mm[j], vv[j], c[j]);
            w[2 * gi] = a[j];
            w[2 * gi + 1] = b[j];
            m[gi] = mm[j];
            v[gi] = vv[j];
        }
    }
}

enum Pattern { kStep8 = 0, kStep8Copy = 1, kAdamW32 = 2 };

// Wave tiles of G granules per lane for the other two patterns, laid out as in
// k_mix_tiles: granule j of lane l in tile t is 64 G t + l + 64 j, and every stored
// vector differs from the one loaded, so no store can be dropped.  Every access is
// inside its array: the largest granule index is 64 G * tiles - 1 = n / 8 - 1.
// step8_copy: w[2gi..2gi+1], g[gi], m2[gi], v2[gi] read and written back (g read
// only), c[gi] written.  adamw32: w, m4, v4 [2gi..2gi+1] and g[gi] read, w, m4, v4
// written back.
template <int P, int G>
__global__ __launch_bounds__(kThreads) void k_pattern_tiles(uint4* __restrict__ w,
                                                           const uint4* __restrict__ g,
                                                           uint2* __restrict__ m2,
                                                           uint2* __restrict__ v2,
                                                           uint4* __restrict__ m4,
                                                           uint4* __restrict__ v4,
                                                           uint4* __restrict__ c, int64_t tiles)
{
    const int lane = threadIdx.x & 63;
    const int64_t waves = int64_t(gridDim.x) * 4;
    for (int64_t t = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6); t < tiles; t += waves) {
        uint4 a[G], b[G], gg[G], ma[G], mb[G], va[G], vb[G];
        uint2 mm[G], vv[G];
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int64_t gi = t * (64 * G) + lane + 64 * j;
            a[j] = w[2 * gi];
            b[j] = w[2 * gi + 1];
            gg[j] = g[gi];
            if (P == kAdamW32) {
                ma[j] = m4[2 * gi];
                mb[j] = m4[2 * gi + 1];
                va[j] = v4[2 * gi];
                vb[j] = v4[2 * gi + 1];
            } else {
                mm[j] = m2[gi];
                vv[j] = v2[gi];
            }
        }
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int64_t gi = t * (64 * G) + lane + 64 * j;
            if (P == kAdamW32) {
                xor_words(a[j], gg[j]);
                xor_words(b[j], gg[j]);
                xor_words(ma[j], gg[j]);
                xor_words(mb[j], gg[j]);
                xor_words(va[j], gg[j]);
                xor_words(vb[j], gg[j]);
                m4[2 * gi] = ma[j];
                m4[2 * gi + 1] = mb[j];
                v4[2 * gi] = va[j];
                v4[2 * gi + 1] = vb[j];
            } else {
                mix_words(a[j], b[j], mm[j], vv[j], gg[j]);
                m2[gi] = mm[j];
                v2[gi] = vv[j];
            }
            w[2 * gi] = a[j];
            w[2 * gi + 1] = b[j];
            if (P == kStep8Copy)
                c[gi] = make_uint4(a[j].x ^ b[j].w, a[j].y ^ b[j].z, a[j].z ^ b[j].y, a[j].w ^ b[j].x);
        }
    }
}

template <int P, int G>
float time_pattern(int grid, int reps, uint4* w, const uint4* g, uint2* m2, uint2* v2, uint4* m4,
                   uint4* v4, uint4* c, int64_t n, hipEvent_t a, hipEvent_t b)
{
    const int64_t tiles = n / (8 * 64 * G);
    k_pattern_tiles<P, G><<<grid, kThreads>>>(w, g, m2, v2, m4, v4, c, tiles);  // warm
    if (hipGetLastError() != hipSuccess || hipEventRecord(a) != hipSuccess)
        return -1.f;
    for (int r = 0; r < reps; ++r)
        k_pattern_tiles<P, G><<<grid, kThreads>>>(w, g, m2, v2, m4, v4, c, tiles);
    float ms;
    if (hipEventRecord(b) != hipSuccess || hipEventSynchronize(b) != hipSuccess ||
        hipEventElapsedTime(&ms, a, b) != hipSuccess)
        return -1.f;
    return ms / reps;
}

__global__ __launch_bounds__(kThreads) void k_read(const u32x4* __restrict__ g, int64_t iters,
                                                  uint32_t* __restrict__ sink)
{
    int64_t b, e;
    range(iters, &b, &e);
    const int t = threadIdx.x;
    uint32_t acc = 0;
    for (int64_t it = b; it < e; ++it) {
        const u32x4 x = __builtin_nontemporal_load(&g[it * kThreads + t]);
        acc ^= x.x ^ x.y ^ x.z ^ x.w;
    }
    if (acc == 0x9E3779B9u)  // practically never true; keeps the loads
        sink[0] = acc;
}

// One set of a pattern's arrays (step8: w, g, m, v; adamw32: w, g, m4, v4).
struct ArraySet {
    uint4 *w = nullptr, *g = nullptr, *m4 = nullptr, *v4 = nullptr;
    uint2 *m = nullptr, *v = nullptr;
};

int run_sets(int64_t n, int reps, int pattern, const char* pname, int K)
{
    int cus;
    CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
    std::vector<ArraySet> sets(K);
    for (ArraySet& s : sets) {
        CK(hipMalloc(&s.w, n * 4));
        CK(hipMalloc(&s.g, n * 2));
        CK(hipMemset(s.w, 1, n * 4));
        CK(hipMemset(s.g, 2, n * 2));
        if (pattern == kAdamW32) {
            CK(hipMalloc(&s.m4, n * 4));
            CK(hipMalloc(&s.v4, n * 4));
            CK(hipMemset(s.m4, 3, n * 4));
            CK(hipMemset(s.v4, 4, n * 4));
        } else {
            CK(hipMalloc(&s.m, n));
            CK(hipMalloc(&s.v, n));
            CK(hipMemset(s.m, 3, n));
            CK(hipMemset(s.v, 4, n));
        }
    }
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    const int grid = 3 * cus;
    const int64_t tiles = n / 2048;  // n is a multiple of 2048
    const double per_elem = pattern == kStep8 ? 14.0 : 26.0;
    for (int pass = 0; pass < 2; ++pass) {
        printf("{\"n\": %lld, \"pattern\": \"%s\", \"pass\": %d, \"sets\": [", (long long)n,
               pname, pass);
        for (int k = 0; k < K; ++k) {
            const ArraySet& s = sets[k];
            float ms;
            if (pattern == kStep8) {
                k_mix_tiles<<<grid, kThreads>>>(s.w, s.g, s.m, s.v, tiles);  // warm
                CK(hipGetLastError());
                CK(hipEventRecord(a));
                for (int r = 0; r < reps; ++r)
                    k_mix_tiles<<<grid, kThreads>>>(s.w, s.g, s.m, s.v, tiles);
                CK(hipEventRecord(b));
                CK(hipEventSynchronize(b));
                CK(hipEventElapsedTime(&ms, a, b));
                ms /= reps;
            } else {
                ms = time_pattern<kAdamW32, 4>(grid, reps, s.w, s.g, nullptr, nullptr, s.m4, s.v4,
                                               nullptr, n, a, b);
                if (ms < 0.f) {
                    fprintf(stderr, "pattern kernel launch or timing failed\n");
                    return 1;
                }
            }
            printf("%s{\"set\": %d, \"ms\": %.4f, \"gbps\": %.1f}", k ? ", " : "", k, ms,
                   double(n) * per_elem / ms / 1e6);
        }
        printf("]}\n");
        fflush(stdout);
    }
    for (ArraySet& s : sets)
        for (void* p : {(void*)s.w, (void*)s.g, (void*)s.m, (void*)s.v, (void*)s.m4, (void*)s.v4})
            if (p)
                CK(hipFree(p));
    return 0;
}

int main(int argc, char** argv)
{
    const int64_t n_req = argc > 1 ? atoll(argv[1]) : 3085844480LL;
    const int reps = argc > 2 ? atoi(argv[2]) : 3;
    const char* pname = argc > 3 ? argv[3] : "step8";
    const int pattern = !strcmp(pname, "step8")        ? kStep8
                        : !strcmp(pname, "step8_copy") ? kStep8Copy
                        : !strcmp(pname, "adamw32")    ? kAdamW32
                                                       : -1;
    const int64_t iters = n_req / kIter;
    const int64_t n = iters * kIter;  // a multiple of 2048: whole tiles for G = 2 and 4
    if (iters < 1 || reps < 1 || pattern < 0) {
        fprintf(stderr, "need n >= %lld, reps >= 1 and pattern step8, step8_copy or adamw32\n",
                (long long)kIter);
        return 2;
    }
    if (argc > 4) {
        const int K = argc > 5 && !strcmp(argv[4], "sets") ? atoi(argv[5]) : 0;
        if (K < 1 || K > 64 || pattern == kStep8Copy) {
            fprintf(stderr, "placement mode: stream_ceiling n reps step8|adamw32 sets K "
                            "(1 <= K <= 64)\n");
            return 2;
        }
        return run_sets(n, reps, pattern, pname, K);
    }
    int cus;
    CK(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, 0));
    uint4 *w, *g, *m4 = nullptr, *v4 = nullptr, *c = nullptr;
    uint2 *m = nullptr, *v = nullptr;
    uint32_t* sink;
    CK(hipMalloc(&w, n * 4));
    CK(hipMalloc(&g, n * 2));
    CK(hipMalloc(&sink, 4));
    CK(hipMemset(w, 1, n * 4));
    CK(hipMemset(g, 2, n * 2));
    if (pattern == kAdamW32) {
        CK(hipMalloc(&m4, n * 4));
        CK(hipMalloc(&v4, n * 4));
        CK(hipMemset(m4, 3, n * 4));
        CK(hipMemset(v4, 4, n * 4));
    } else {
        CK(hipMalloc(&m, n));
        CK(hipMalloc(&v, n));
        CK(hipMemset(m, 3, n));
        CK(hipMemset(v, 4, n));
    }
    if (pattern == kStep8Copy) {
        CK(hipMalloc(&c, n * 2));
        CK(hipMemset(c, 5, n * 2));
    }
    hipEvent_t a, b;
    CK(hipEventCreate(&a));
    CK(hipEventCreate(&b));
    float best_mix = 1e30f, best_read = 1e30f;
    for (int per_cu : {2, 4, 8}) {
        const int grid = cus * per_cu;
        float ms;
        if (pattern == kStep8) {
            k_mix<<<grid, kThreads>>>(w, g, m, v, iters);  // warm
            CK(hipGetLastError());
            CK(hipEventRecord(a));
            for (int r = 0; r < reps; ++r)
                k_mix<<<grid, kThreads>>>(w, g, m, v, iters);
            CK(hipEventRecord(b));
            CK(hipEventSynchronize(b));
            CK(hipEventElapsedTime(&ms, a, b));
            if (ms / reps < best_mix)
                best_mix = ms / reps;
        }
        k_read<<<grid, kThreads>>>(reinterpret_cast<const u32x4*>(g), iters, sink);  // warm
        CK(hipGetLastError());
        CK(hipEventRecord(a));
        for (int r = 0; r < reps; ++r)
            k_read<<<grid, kThreads>>>(reinterpret_cast<const u32x4*>(g), iters, sink);
        CK(hipEventRecord(b));
        CK(hipEventSynchronize(b));
        CK(hipEventElapsedTime(&ms, a, b));
        if (ms / reps < best_read)
            best_read = ms / reps;
    }
    for (int per_cu : {1, 2, 3}) {
        if (pattern == kStep8)
            break;
        const int grid = cus * per_cu;
        const float t2 = pattern == kStep8Copy
                             ? time_pattern<kStep8Copy, 2>(grid, reps, w, g, m, v, m4, v4, c, n, a, b)
                             : time_pattern<kAdamW32, 2>(grid, reps, w, g, m, v, m4, v4, c, n, a, b);
        const float t4 = pattern == kStep8Copy
                             ? time_pattern<kStep8Copy, 4>(grid, reps, w, g, m, v, m4, v4, c, n, a, b)
                             : time_pattern<kAdamW32, 4>(grid, reps, w, g, m, v, m4, v4, c, n, a, b);
        if (t2 < 0.f || t4 < 0.f) {
            fprintf(stderr, "pattern kernel launch or timing failed\n");
            return 1;
        }
        fprintf(stderr, "%s: %d workgroups per CU: %.4f ms (16 per lane), %.4f ms (32 per lane)\n",
                pname, per_cu, t2, t4);
        best_mix = fminf(best_mix, fminf(t2, t4));
    }
    // wave tiles of 2048 elements: n is a multiple of kIter = 2048
    for (int per_cu : {1, 2, 3}) {
        if (pattern != kStep8)
            break;
        const int grid = cus * per_cu;
        const int64_t tiles = n / 2048;
        k_mix_tiles<<<grid, kThreads>>>(w, g, m, v, tiles);  // warm
        CK(hipGetLastError());
        CK(hipEventRecord(a));
        for (int r = 0; r < reps; ++r)
            k_mix_tiles<<<grid, kThreads>>>(w, g, m, v, tiles);
        CK(hipEventRecord(b));
        CK(hipEventSynchronize(b));
        float ms;
        CK(hipEventElapsedTime(&ms, a, b));
        if (ms / reps < best_mix)
            best_mix = ms / reps;
    }
    CK(hipDeviceSynchronize());
    // an iteration of k_read reads 256 x 16 B: 2048 bf16 gradient elements
    const double per_elem = pattern == kStep8 ? 14.0 : pattern == kStep8Copy ? 16.0 : 26.0;
    const double mix_bytes = double(n) * per_elem, read_bytes = double(n) * 2.0;
    printf("{\"n\": %lld, \"pattern\": \"%s\", \"mix_bytes\": %.0f, \"mix_ms\": %.4f, "
           "\"mix_gbps\": %.1f, \"read_bytes\": %.0f, \"read_ms\": %.4f, \"read_gbps\": %.1f}\n",
           (long long)n, pname, mix_bytes, best_mix, mix_bytes / best_mix / 1e6, read_bytes,
           best_read, read_bytes / best_read / 1e6);
    CK(hipFree(w));
    CK(hipFree(g));
    for (void* p : {(void*)m, (void*)v, (void*)m4, (void*)v4, (void*)c})
        if (p)
            CK(hipFree(p));
    CK(hipFree(sink));
    return 0;
}
