// mix_probe.hip -- a measurement tool for bench.py, not part of the optimizer.
//
// Moves exactly the fused 8-bit step's bytes over the step's own arrays, with no
// arithmetic: per element it reads the 4-byte weight, the gradient and the two
// 1-byte codes and writes the weight and both codes back in place.  Every stored
// word changes (XOR with a mask taken from the gradient, never zero), so no load
// or store can be narrowed; XOR-ing twice restores the arrays.  The geometry is
// the step kernel's at 32 elements per lane: 2048-element wave spans handed to the
// waves in turn, granule j of lane l at elements 8 * (l + 64 j) of the span, one
// 16-byte load or store per weight half and gradient word, 8 bytes per code
// array.  A span that runs past its tensor's end moves its elements one by one.
// Timing it beside the step shows what the memory system gives this byte pattern
// at the placement the step's arrays actually have.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

struct ProbeTensor {
    uint32_t* w;
    const void* g;
    uint8_t* mq;
    uint8_t* vq;
    int64_t numel;
    int64_t pad[3];
};
static_assert(sizeof(ProbeTensor) == 64, "one 64-byte line per tensor");

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

template <typename T>
__device__ inline __attribute__((address_space(1))) T* gp(T* p)
{
    return (__attribute__((address_space(1))) T*)p;
}

__device__ inline int find_tensor(const int64_t* prefix, int n, int64_t u)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (prefix[mid] <= u)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

constexpr int kSpan = 2048;

// GB: gradient bytes per element (2 or 4).
template <int GB>
__global__ __launch_bounds__(256) void k_mix_same(const int64_t* __restrict__ prefix,
                                                  const ProbeTensor* __restrict__ desc, int K,
                                                  int64_t n_units)
{
    const int lane = threadIdx.x & 63;
    const int64_t workers = int64_t(gridDim.x) * 4;
    const int64_t me = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
    int k = me < n_units ? find_tensor(prefix, K, me) : 0;
    for (int64_t u = me; u < n_units; u += workers) {
        while (u >= prefix[k + 1])
            ++k;
        const ProbeTensor d = desc[k];
        const int64_t e0 = (u - prefix[k]) * kSpan;
        if (d.numel - e0 >= kSpan) {
            u32x4 a[4], b[4], c[4][GB / 2];
            u32x2 m[4], v[4];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t ei = e0 + 8 * (lane + 64 * j);
                a[j] = *gp(reinterpret_cast<u32x4*>(d.w + ei));
                b[j] = *gp(reinterpret_cast<u32x4*>(d.w + ei + 4));
#pragma unroll
                for (int q = 0; q < GB / 2; ++q)
                    c[j][q] = __builtin_nontemporal_load(
                        gp(reinterpret_cast<const u32x4*>(static_cast<const uint8_t*>(d.g) +
                                                          ei * GB) + q));
                m[j] = *gp(reinterpret_cast<u32x2*>(d.mq + ei));
                v[j] = *gp(reinterpret_cast<u32x2*>(d.vq + ei));
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int64_t ei = e0 + 8 * (lane + 64 * j);
                u32x4 g = c[j][0];
                if constexpr (GB == 4)
                    g ^= c[j][1];  // uses the second gradient word, so its load stays
                g |= 1u;
                a[j] ^= g;
                b[j] ^= g.yzwx;
                m[j] ^= g.xz;
                v[j] ^= g.yw;
                *gp(reinterpret_cast<u32x4*>(d.w + ei)) = a[j];
                *gp(reinterpret_cast<u32x4*>(d.w + ei + 4)) = b[j];
                *gp(reinterpret_cast<u32x2*>(d.mq + ei)) = m[j];
                *gp(reinterpret_cast<u32x2*>(d.vq + ei)) = v[j];
            }
        } else {
            for (int64_t e = e0 + lane; e < d.numel; e += 64) {
                const uint32_t g =
                    GB == 2 ? uint32_t(gp(static_cast<const uint16_t*>(d.g))[e]) | 1u
                            : gp(static_cast<const uint32_t*>(d.g))[e] | 1u;
                gp(d.w)[e] ^= g;
                gp(d.mq)[e] ^= uint8_t(g);
                gp(d.vq)[e] ^= uint8_t(g);
            }
        }
    }
}

}  // namespace

extern "C" {

// prefix: device int64[K + 1], the span prefix (ceil(numel / 2048) per tensor);
// desc: device ProbeTensor[K].  grid: workgroups of 256 threads.
int ltp_mix_same_arrays(const int64_t* prefix, const void* desc, int K, int64_t n_units,
                        int grad_bytes, int grid, void* stream)
{
    if (K < 1 || n_units < 1 || grid < 1 || (grad_bytes != 2 && grad_bytes != 4))
        return 1;
    const auto* d = static_cast<const ProbeTensor*>(desc);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (grad_bytes == 2)
        k_mix_same<2><<<grid, 256, 0, st>>>(prefix, d, K, n_units);
    else
        k_mix_same<4><<<grid, 256, 0, st>>>(prefix, d, K, n_units);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
