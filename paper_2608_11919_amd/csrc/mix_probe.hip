// mix_probe.hip -- a measurement tool for bench.py, not part of the optimizer.
//
// Moves exactly a fused step's bytes over the step's own arrays, with no
// arithmetic: per element it reads the 4-byte weight, the gradient and the two
// moment states (1-byte codes for the 8-bit step, 4-byte floats for the
// fp32-state step) and writes the weight and both states back in place.  Every stored
// word changes (XOR with a mask taken from the gradient, never zero), so no load
// or store can be narrowed; XOR-ing twice restores the arrays.  The geometry is
// the step kernel's at 32 elements per lane: 2048-element wave spans handed to the
// waves in turn, granule j of lane l at elements 8 * (l + 64 j) of the span, one
// 16-byte load or store per weight half and gradient word, 8 bytes per code
// array or two 16-byte words per fp32 state array.  A span that runs past its tensor's end moves its elements one by one.
// Timing it beside the step shows what the memory system gives this byte pattern
// at the placement the step's arrays actually have.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

struct ProbeTensor {
    uint32_t* w;
    const void* g;
    uint8_t* mq;  // the first moment's state (codes, or fp32 values)
    uint8_t* vq;  // the second moment's state
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

// One lane's 8 elements of a state array of SB bytes per element.
template <int SB>
struct StateWords {
    u32x4 q[SB == 4 ? 2 : 1];  // SB = 1 uses the low half of q[0]
};

template <int SB>
__device__ inline void load_state(const uint8_t* base, int64_t ei, StateWords<SB>& s)
{
    if constexpr (SB == 1) {
        const u32x2 v = *gp(reinterpret_cast<const u32x2*>(base + ei));
        s.q[0] = u32x4{v.x, v.y, 0u, 0u};
    } else {
        s.q[0] = *gp(reinterpret_cast<const u32x4*>(base + 4 * ei));
        s.q[1] = *gp(reinterpret_cast<const u32x4*>(base + 4 * ei) + 1);
    }
}

template <int SB>
__device__ inline void store_state(uint8_t* base, int64_t ei, const StateWords<SB>& s)
{
    if constexpr (SB == 1) {
        *gp(reinterpret_cast<u32x2*>(base + ei)) = s.q[0].xy;
    } else {
        *gp(reinterpret_cast<u32x4*>(base + 4 * ei)) = s.q[0];
        *gp(reinterpret_cast<u32x4*>(base + 4 * ei) + 1) = s.q[1];
    }
}

// GB: gradient bytes per element (2 or 4); SB: state bytes per element (1 or 4).
template <int GB, int SB>
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
            StateWords<SB> m[4], v[4];
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
                load_state<SB>(d.mq, ei, m[j]);
                load_state<SB>(d.vq, ei, v[j]);
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
#pragma unroll
                for (int q = 0; q < (SB == 4 ? 2 : 1); ++q) {
                    m[j].q[q] ^= q ? g.zwxy : g;
                    v[j].q[q] ^= q ? g.wxyz : g.yzwx;
                }
                *gp(reinterpret_cast<u32x4*>(d.w + ei)) = a[j];
                *gp(reinterpret_cast<u32x4*>(d.w + ei + 4)) = b[j];
                store_state<SB>(d.mq, ei, m[j]);
                store_state<SB>(d.vq, ei, v[j]);
            }
        } else {
            for (int64_t e = e0 + lane; e < d.numel; e += 64) {
                const uint32_t g =
                    GB == 2 ? uint32_t(gp(static_cast<const uint16_t*>(d.g))[e]) | 1u
                            : gp(static_cast<const uint32_t*>(d.g))[e] | 1u;
                gp(d.w)[e] ^= g;
                if constexpr (SB == 1) {
                    gp(d.mq)[e] ^= uint8_t(g);
                    gp(d.vq)[e] ^= uint8_t(g);
                } else {
                    gp(reinterpret_cast<uint32_t*>(d.mq))[e] ^= g;
                    gp(reinterpret_cast<uint32_t*>(d.vq))[e] ^= g;
                }
            }
        }
    }
}

}  // namespace

extern "C" {

// prefix: device int64[K + 1], the span prefix (ceil(numel / 2048) per tensor);
// desc: device ProbeTensor[K]; state_bytes: 1 (8-bit codes) or 4 (fp32 moments).
// grid: workgroups of 256 threads.
int ltp_mix_same_arrays(const int64_t* prefix, const void* desc, int K, int64_t n_units,
                        int grad_bytes, int state_bytes, int grid, void* stream)
{
    if (K < 1 || n_units < 1 || grid < 1 || (grad_bytes != 2 && grad_bytes != 4) ||
        (state_bytes != 1 && state_bytes != 4))
        return 1;
    const auto* d = static_cast<const ProbeTensor*>(desc);
    hipStream_t st = static_cast<hipStream_t>(stream);
    if (grad_bytes == 2 && state_bytes == 1)
        k_mix_same<2, 1><<<grid, 256, 0, st>>>(prefix, d, K, n_units);
    else if (grad_bytes == 4 && state_bytes == 1)
        k_mix_same<4, 1><<<grid, 256, 0, st>>>(prefix, d, K, n_units);
    else if (grad_bytes == 2)
        k_mix_same<2, 4><<<grid, 256, 0, st>>>(prefix, d, K, n_units);
    else
        k_mix_same<4, 4><<<grid, 256, 0, st>>>(prefix, d, K, n_units);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}

}  // extern "C"
