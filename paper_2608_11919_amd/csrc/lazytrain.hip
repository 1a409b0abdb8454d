// lazytrain.hip -- gfx950 kernels and C ABI of the Hybrid 8-bit optimizer step
// (LazyTrain, Sec. 3.5: fast gradient clipping coupled with block-wise 8-bit
// AdamW states; App. C: AdamW hyperparameters, max grad norm, non-finite skip).
//
// Kernels (all HBM-bound streaming, no MFMA: there is no contraction):
//   k_sqnorm_chunks  one fp64 sum of squares per 8192-element gradient chunk;
//                    16-byte loads, wave64 butterfly, 4-wave combine in LDS.
//   k_sqnorm_finish  per-tensor fixed-order combine of the chunk sums.
//   k_sqnorm_total   list-order global sum and the non-finite status.
//   k_clip_coef      fp32(sqrt(S)) (fp64 root, then fp32) and the clip coefficient.
//   k_adamw8_step    fused dequantize -> AdamW -> block absmax -> requantize,
//                    with the linear or the dynamic code map and an optional
//                    bf16 copy of the updated weights.
//   k_adamw32_step   the same update with fp32 moments (the hybrid operator's
//                    non-8-bit part).
//   k_bf16_on_skip   bf16 copies of unchanged weights after a skipped step.
// Host side: the C ABI, descriptor uploads through a pinned staging ring, and
// the layer-streamed step (a ring of device slots on three streams).
// The reduction order and the fp32 operation order are fixed (see
// include/lazytrain.h, which also names the steps a1..a11 and f1..f4 used in
// the section titles below); every kernel's result is independent of its grid.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <initializer_list>
#include <chrono>
#include <map>
#include <mutex>
#include <string>
#include <unordered_map>
#include <vector>

#include "lazytrain.h"

namespace {

constexpr int kThreads = 256;  // 4 wave64s per workgroup
constexpr int kChunk = 8192;   // sum-of-squares chunk: 256 lanes x 4 granules x 8 elements
constexpr int kGranule = 8;    // elements per lane per 16-byte bf16 load

// ------------------------------------------------------------------ errors

thread_local std::string g_last_error;

lt_err fail(lt_err code, const std::string& msg)
{
    g_last_error = msg;
    return code;
}

#define LT_HIP(call)                                                                    \
    do {                                                                                \
        hipError_t e_ = (call);                                                         \
        if (e_ != hipSuccess)                                                           \
            return fail(LT_ERR_HIP, std::string(#call) + ": " + hipGetErrorString(e_)); \
    } while (0)

// ------------------------------------------------------------- descriptors

// Device-side view of one tensor of the step.
struct StepTensor {
    float* w;
    const void* g;
    int8_t* mq;
    float* ma;
    uint8_t* vq;
    float* va;
    int64_t numel;
    uint16_t* wb;  // bf16 copy of the updated weights, or null
};
static_assert(sizeof(StepTensor) == 64, "descriptor is one 64-byte line");

struct StepScalars {
    float beta1, beta2, eps, c1, c2, decay, step_size, rbc2;
    const uint8_t* state;  // the caller's step state, or null: step_size and rbc2 as given
    double lr;             // for step_size from the step state's table
};

constexpr size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Every workspace starts with kTagBytes that hold the tag of the descriptors it
// holds (see put_descriptors); the descriptors follow.
constexpr size_t kTagBytes = 64;

// Sum-of-squares workspace: [tag][chunk_prefix K+1][ptr K][numel K] | [partials C][S_k K]
struct SqLayout {
    size_t prefix, ptrs, numels, header_bytes, partials, sk, total;
};

SqLayout sq_layout(int K, int64_t C)
{
    SqLayout l;
    l.prefix = kTagBytes;
    l.ptrs = l.prefix + round_up(sizeof(int64_t) * (K + 1), 64);
    l.numels = l.ptrs + round_up(sizeof(uint64_t) * K, 64);
    l.header_bytes = l.numels + round_up(sizeof(int64_t) * K, 64);
    l.partials = round_up(l.header_bytes, 256);
    l.sk = l.partials + round_up(sizeof(double) * C, 256);
    l.total = l.sk + round_up(sizeof(double) * K, 256);
    return l;
}

// Step workspace: [tag][tile_prefix K+1][StepTensor K]
struct StepLayout {
    size_t prefix, desc, total;
};

StepLayout step_layout(int K)
{
    StepLayout l;
    l.prefix = kTagBytes;
    l.desc = l.prefix + round_up(sizeof(int64_t) * (K + 1), 64);
    l.total = round_up(l.desc + sizeof(StepTensor) * K, 256);
    return l;
}

// ---------------------------------------------------- descriptor uploads
//
// A list call builds its descriptors on the host as an image of the head of its
// workspace.  The library remembers, per workspace address, the image it last
// copied there; when a call's image is the same, nothing is copied, so a caller
// that repeats a step over the same tensors stages nothing on the host after the
// first call, and those calls can be captured into a HIP graph.
//
// Each copy writes a new 64-bit tag into the workspace's first word, and the
// kernels receive the tag by value: a kernel whose workspace does not hold its
// tag (the caller wrote into the workspace, or freed it and the address came back
// for another use) returns before it reads a descriptor, instead of following
// stale pointers.  lt_workspace_release makes the library forget a workspace.
//
// Images are staged in pinned host slots.  A slot is reused once the copy out of
// it has run (checked without waiting); when the next slot is still in use, the
// ring grows by one slot rather than wait, so no call waits on the host.

struct WsGuard {
    const uint64_t* at;  // the workspace's tag word
    uint64_t tag;        // the tag of the descriptors this launch expects
};

struct StagingSlot {
    void* host = nullptr;
    size_t cap = 0;
    hipEvent_t done = nullptr;
    bool pending = false;
};

// What a workspace holds: the image last copied into it, its tag, and an event
// behind that copy on the stream that made it.
struct CachedImage {
    std::vector<uint8_t> image;
    uint64_t tag = 0;
    hipEvent_t copied = nullptr;
    hipStream_t stream = nullptr;
};

constexpr int kMaxDevices = 64;

struct DeviceState {
    std::mutex mu;
    std::vector<StagingSlot> slots;
    size_t next = 0;
    int cu_count = 0;
    std::map<std::pair<const void*, size_t>, int> occupancy;  // workgroups per CU, by kernel and LDS
    std::unordered_map<const void*, CachedImage> cache;        // by workspace address
    std::vector<hipEvent_t> spare_events;
    std::vector<void*> retired;  // staging buffers outgrown; freed never (a free may synchronize)
};

DeviceState g_dev[kMaxDevices];
std::atomic<int> g_max_workgroups{0};
std::atomic<uint64_t> g_tag_counter{0};

lt_err current_device(int* dev)
{
    LT_HIP(hipGetDevice(dev));
    if (*dev < 0 || *dev >= kMaxDevices)
        return fail(LT_ERR_HIP, "device index out of range");
    return LT_OK;
}

uint64_t mix64(uint64_t z)
{
    z += 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// A tag no earlier copy of this process wrote, and unlikely to be found in
// memory by accident (never 0).
uint64_t fresh_tag()
{
    static const uint64_t salt =
        mix64(uint64_t(reinterpret_cast<uintptr_t>(&g_tag_counter)) ^
              uint64_t(std::chrono::steady_clock::now().time_since_epoch().count()));
    const uint64_t t = mix64(salt ^ g_tag_counter.fetch_add(1));
    return t ? t : 1;
}

lt_err stream_capturing(hipStream_t st, bool* capturing)
{
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    LT_HIP(hipStreamIsCapturing(st, &cs));
    *capturing = cs != hipStreamCaptureStatusNone;
    return LT_OK;
}

// Copies n bytes from host memory to device address dst on stream st through a
// pinned staging slot (ds.mu held).  A slot is reused once its copy has run,
// checked without waiting; when the next one is still in flight the ring grows by
// a slot, so the call never waits for the device.
lt_err stage_copy_locked(DeviceState& ds, const void* src, size_t n, void* dst, hipStream_t st)
{
    if (ds.slots.empty())
        ds.slots.resize(8);
    if (ds.next >= ds.slots.size())
        ds.next = 0;
    {
        StagingSlot& s = ds.slots[ds.next];
        if (s.pending) {
            const hipError_t q = hipEventQuery(s.done);
            if (q == hipSuccess)
                s.pending = false;
            else if (q == hipErrorNotReady)
                ds.slots.insert(ds.slots.begin() + ptrdiff_t(ds.next), StagingSlot{});  // grow
            else
                return fail(LT_ERR_HIP, std::string("hipEventQuery: ") + hipGetErrorString(q));
        }
    }
    StagingSlot& s = ds.slots[ds.next];
    ds.next += 1;
    if (!s.done)
        LT_HIP(hipEventCreateWithFlags(&s.done, hipEventDisableTiming));
    if (s.cap < n) {
        if (s.host)
            ds.retired.push_back(s.host);
        s.host = nullptr;
        s.cap = 0;
        const size_t cap = round_up(std::max(n, size_t(4096)), 4096);
        LT_HIP(hipHostMalloc(&s.host, cap, hipHostMallocDefault));
        s.cap = cap;
    }
    std::memcpy(s.host, src, n);
    LT_HIP(hipMemcpyAsync(dst, s.host, n, hipMemcpyHostToDevice, st));
    LT_HIP(hipEventRecord(s.done, st));
    s.pending = true;
    return LT_OK;
}

// Makes the workspace `ws` hold `image` (the bytes of its head; the first
// kTagBytes are the tag slot, filled here) before the work enqueued next on `st`
// reads it, and returns the guard that work's kernels check.
lt_err put_descriptors(std::vector<uint8_t>& image, void* ws, hipStream_t st, WsGuard* guard)
{
    int dev;
    if (lt_err e = current_device(&dev))
        return e;
    bool capturing;
    if (lt_err e = stream_capturing(st, &capturing))
        return e;
    DeviceState& ds = g_dev[dev];
    std::lock_guard<std::mutex> lock(ds.mu);
    CachedImage& c = ds.cache[ws];
    guard->at = static_cast<const uint64_t*>(ws);
    const size_t n = image.size();
    if (c.tag != 0 && c.image.size() == n &&
        std::memcmp(c.image.data() + kTagBytes, image.data() + kTagBytes, n - kTagBytes) == 0) {
        // Already in place.  Work on another stream waits for the copy; under
        // capture the copy must have completed before capture began (the header
        // says so), since a graph cannot wait on work outside it.
        if (!capturing && st != c.stream)
            LT_HIP(hipStreamWaitEvent(st, c.copied, 0));
        guard->tag = c.tag;
        return LT_OK;
    }
    if (capturing)
        return fail(LT_ERR_INVALID_ARG,
                    "the descriptors of this tensor list are not in the workspace: make one "
                    "uncaptured call with this workspace and list, and let it complete, before "
                    "capturing");
    const uint64_t tag = fresh_tag();
    std::memcpy(image.data(), &tag, sizeof(tag));
    if (lt_err e = stage_copy_locked(ds, image.data(), n, ws, st))
        return e;

    if (!c.copied) {
        if (!ds.spare_events.empty()) {
            c.copied = ds.spare_events.back();
            ds.spare_events.pop_back();
        } else {
            LT_HIP(hipEventCreateWithFlags(&c.copied, hipEventDisableTiming));
        }
    }
    LT_HIP(hipEventRecord(c.copied, st));
    c.image = image;
    c.tag = tag;
    c.stream = st;
    guard->tag = tag;
    return LT_OK;
}

lt_err compute_units(int* cus)
{
    int dev;
    if (lt_err e = current_device(&dev))
        return e;
    DeviceState& ds = g_dev[dev];
    {
        std::lock_guard<std::mutex> lock(ds.mu);
        if (ds.cu_count > 0) {
            *cus = ds.cu_count;
            return LT_OK;
        }
    }
    int n = 0;
    LT_HIP(hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev));
    std::lock_guard<std::mutex> lock(ds.mu);
    ds.cu_count = n > 0 ? n : 1;
    *cus = ds.cu_count;
    return LT_OK;
}

// Persistent grid: enough workgroups to fill every CU at the kernel's
// occupancy (with `lds` bytes of dynamic LDS per workgroup), never more than
// there are work units.  The occupancy of each kernel is queried once per device.
template <typename Kernel>
lt_err grid_size(Kernel kernel, int64_t units, int* grid, size_t lds = 0)
{
    int cus, dev;
    if (lt_err e = compute_units(&cus))
        return e;
    if (lt_err e = current_device(&dev))
        return e;
    const auto key = std::make_pair(reinterpret_cast<const void*>(kernel), lds);
    int per_cu = 0;
    {
        std::lock_guard<std::mutex> lock(g_dev[dev].mu);
        auto it = g_dev[dev].occupancy.find(key);
        if (it != g_dev[dev].occupancy.end())
            per_cu = it->second;
    }
    if (per_cu <= 0) {
        LT_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, lds));
        per_cu = std::max(per_cu, 1);
        std::lock_guard<std::mutex> lock(g_dev[dev].mu);
        g_dev[dev].occupancy[key] = per_cu;
    }
    int64_t g = int64_t(cus) * std::max(per_cu, 1);
    int cap = g_max_workgroups.load();
    if (cap > 0)
        g = std::min<int64_t>(g, cap);
    g = std::min<int64_t>(g, units);
    *grid = int(std::max<int64_t>(g, 1));
    return LT_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// True when a nullable list of n pointers holds a non-null entry.
template <typename T>
bool any_set(T* const* list, int n)
{
    if (!list)
        return false;
    for (int k = 0; k < n; ++k)
        if (list[k])
            return true;
    return false;
}

// ============================================================== device code

__device__ inline int64_t i64min(int64_t a, int64_t b) { return a < b ? a : b; }
__device__ inline int64_t i64max(int64_t a, int64_t b) { return a > b ? a : b; }

__device__ inline float bf16_lo(uint32_t d) { return __uint_as_float(d << 16); }
__device__ inline float bf16_hi(uint32_t d) { return __uint_as_float(d & 0xFFFF0000u); }

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Every tensor lives in device (global) memory, but the kernels read its address
// from a descriptor, so the compiler cannot tell and would emit flat memory
// instructions.  Those count against the LDS/scalar counter as well as the
// vector-memory one, so each wait for a shuffle or a scalar load would also wait
// for every load and store the wave has in flight.  Tensor data is therefore
// accessed through global address-space pointers (global_load/global_store),
// as the compiler's vector types (HIP's uint4/float4 classes take no such pointer).
template <typename T>
__device__ inline __attribute__((address_space(1))) T* gp(T* p)
{
    return (__attribute__((address_space(1))) T*)p;
}

// 16-byte load that asks the memory system not to keep the line (streaming).
__device__ inline uint4 load16_stream(const void* p)
{
    const u32x4 v = __builtin_nontemporal_load(gp(static_cast<const u32x4*>(p)));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ inline uint4 load16(const void* p)
{
    const u32x4 v = *gp(static_cast<const u32x4*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ inline void store16(void* p, uint4 q) { *gp(static_cast<u32x4*>(p)) = u32x4{q.x, q.y, q.z, q.w}; }

__device__ inline void store16f(float* p, float a, float b, float c, float d)
{
    *gp(reinterpret_cast<f32x4*>(p)) = f32x4{a, b, c, d};
}

__device__ inline uint2 load8(const void* p)
{
    const u32x2 v = *gp(static_cast<const u32x2*>(p));
    return make_uint2(v.x, v.y);
}

__device__ inline void store8(void* p, uint32_t lo, uint32_t hi) { *gp(static_cast<u32x2*>(p)) = u32x2{lo, hi}; }

// Raw bits of one gradient element (bf16: 16 bits, fp32: 32 bits).
__device__ inline uint32_t grad_bits(const uint16_t* p) { return *gp(p); }
__device__ inline uint32_t grad_bits(const float* p) { return __float_as_uint(*gp(p)); }

// Packed 16-byte words holding the 8 gradients of one granule: bf16 needs one
// word, fp32 two.  Unpacking is exact (bf16 is the top half of an fp32).
template <typename GT>
struct GradWords {
    static constexpr int N = sizeof(GT) / 2;
    uint4 q[N];
};

template <typename GT>
__device__ inline void unpack8(const GradWords<GT>& r, float (&x)[8])
{
    if constexpr (sizeof(GT) == 2) {
        const uint4 v = r.q[0];
        x[0] = bf16_lo(v.x); x[1] = bf16_hi(v.x);
        x[2] = bf16_lo(v.y); x[3] = bf16_hi(v.y);
        x[4] = bf16_lo(v.z); x[5] = bf16_hi(v.z);
        x[6] = bf16_lo(v.w); x[7] = bf16_hi(v.w);
    } else {
        x[0] = __uint_as_float(r.q[0].x); x[1] = __uint_as_float(r.q[0].y);
        x[2] = __uint_as_float(r.q[0].z); x[3] = __uint_as_float(r.q[0].w);
        x[4] = __uint_as_float(r.q[1].x); x[5] = __uint_as_float(r.q[1].y);
        x[6] = __uint_as_float(r.q[1].z); x[7] = __uint_as_float(r.q[1].w);
    }
}

// Loads the granule of 8 gradients at p of which the first nv exist; the
// others read as +0.  STREAM selects non-temporal loads for full granules.
template <bool STREAM, typename GT>
__device__ inline void load_grads(const GT* p, int nv, GradWords<GT>& r)
{
    if (nv >= kGranule) {
#pragma unroll
        for (int q = 0; q < GradWords<GT>::N; ++q)
            r.q[q] = STREAM ? load16_stream(reinterpret_cast<const uint4*>(p) + q)
                            : load16(reinterpret_cast<const uint4*>(p) + q);
        return;
    }
    uint32_t b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
        b[e] = e < nv ? grad_bits(p + e) : 0u;
    if constexpr (sizeof(GT) == 2) {
        r.q[0] = make_uint4(b[0] | (b[1] << 16), b[2] | (b[3] << 16), b[4] | (b[5] << 16),
                            b[6] | (b[7] << 16));
    } else {
        r.q[0] = make_uint4(b[0], b[1], b[2], b[3]);
        r.q[1] = make_uint4(b[4], b[5], b[6], b[7]);
    }
}

// Index of the tensor that holds work unit u: the last k with prefix[k] <= u.
__device__ inline int find_tensor(const int64_t* __restrict__ prefix, int n_tensors, int64_t u)
{
    int lo = 0, hi = n_tensors - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (prefix[mid] <= u)
            lo = mid;
        else
            hi = mid - 1;
    }
    return lo;
}

// True when the workspace holds the descriptors this launch was given the tag of.
__device__ inline bool guard_ok(const WsGuard& g) { return *g.at == g.tag; }

// With a caller's step state: the step applied is t = applied + 1, its step size
// fp32(lr / (1 - beta1^t)) by an fp64 division of the table's fp64 1 - beta1^t
// (the host's expression and rounding), its rbc2 the table's.  False when the
// state lets no step apply (stopped, or its table does not reach t).
__device__ inline bool resolve_step(StepScalars& s)
{
    if (!s.state)
        return true;
    const auto* h = reinterpret_cast<const lt_step_state*>(s.state);
    const int64_t a = h->applied;
    if (h->stopped != 0 || a < 0 || a >= h->table_len)
        return false;
    const lt_step_table_entry e =
        reinterpret_cast<const lt_step_table_entry*>(s.state + sizeof(lt_step_state))[a];
    s.step_size = float(s.lr / e.one_minus_beta1_t);
    s.rbc2 = e.rbc2;
    return true;
}

// ------------------------------------------------------- a1: chunk sums

// One lane's share of a chunk: granules lane + 256*r, r = 0..3.
template <typename GT>
struct ChunkLane {
    GradWords<GT> r[4];
};

template <typename GT>
__device__ inline void load_chunk_lane(const uint64_t* __restrict__ ptrs,
                                       const int64_t* __restrict__ numels, int k, int64_t local,
                                       int lane, ChunkLane<GT>& out)
{
    const int64_t n_in = i64min(kChunk, numels[k] - local * kChunk);
    const GT* base = reinterpret_cast<const GT*>(ptrs[k]) + local * kChunk;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int j0 = kGranule * (lane + kThreads * r);
        load_grads<true>(base + j0, int(i64min(i64max(n_in - j0, 0), kGranule)), out.r[r]);
    }
}

// Lane sum of one chunk in the fixed order.  The square of an fp32 value is
// exact in fp64, so fma(x, x, a) is the single rounding of a + x*x; positions
// past the end read as 0 and leave the non-negative sum unchanged.
template <typename GT>
__device__ inline double lane_sum(const ChunkLane<GT>& c)
{
    double a = 0.0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        float x[8];
        unpack8(c.r[r], x);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const double xd = double(x[e]);
            a = __builtin_fma(xd, xd, a);
        }
    }
    return a;
}

// Chunks per iteration: their loads are all issued first, then the wave sums,
// one barrier and the partials.  Two measured best among 1-8 with and without a
// next-iteration prefetch and with grid-strided iterations (all within ~5%).
constexpr int kSqChunksPerIter = 2;

// Each iteration takes U consecutive chunks.
template <typename GT>
__global__ __launch_bounds__(kThreads) void k_sqnorm_chunks(WsGuard guard,
                                                            const int64_t* __restrict__ chunk_prefix,
                                                            const uint64_t* __restrict__ ptrs,
                                                            const int64_t* __restrict__ numels,
                                                            int n_tensors, int64_t n_chunks,
                                                            double* __restrict__ partials)
{
    constexpr int U = kSqChunksPerIter;
    __shared__ double wave_sum[2][U][4];
    if (!guard_ok(guard))
        return;
    const int lane = threadIdx.x;
    const int wave = lane >> 6;
    const int64_t n_iter = (n_chunks + U - 1) / U;
    // A contiguous, balanced range of iterations per workgroup: for this
    // read-only pass it measured 5% faster than handing iterations out in turn
    // (the opposite of the step kernels).
    int64_t i_begin, i_end;
    {
        const int64_t G = gridDim.x, b = blockIdx.x;
        const int64_t per = n_iter / G, rem = n_iter % G;
        i_begin = b * per + (b < rem ? b : rem);
        i_end = i_begin + per + (b < rem ? 1 : 0);
    }
    if (i_begin >= i_end)
        return;
    int k = find_tensor(chunk_prefix, n_tensors, i_begin * U);
    int buf = 0;
    for (int64_t it = i_begin; it < i_end; ++it, buf ^= 1) {
        ChunkLane<GT> cur[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t c = it * U + u;
            if (c < n_chunks) {
                while (c >= chunk_prefix[k + 1])
                    ++k;
                load_chunk_lane(ptrs, numels, k, c - chunk_prefix[k], lane, cur[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            double a = lane_sum(cur[u]);
            // 64-lane halving tree as a butterfly: lane i adds lane i^o; for
            // i < o that is a_i + a_(i+o), and addition is commutative.
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1)
                a = a + __shfl_xor(a, o, 64);
            if ((lane & 63) == 0)
                wave_sum[buf][u][wave] = a;
        }
        __syncthreads();
        if (lane < U) {
            const int64_t c = it * U + lane;
            if (c < n_chunks)
                partials[c] = (wave_sum[buf][lane][0] + wave_sum[buf][lane][2]) +
                              (wave_sum[buf][lane][1] + wave_sum[buf][lane][3]);
        }
        // The other buffer is written next; this one again only after the next
        // barrier, which the reading lanes reach after their reads.
    }
}

// ------------------------------------------------- a2: fixed-order finish

__global__ __launch_bounds__(kThreads) void k_sqnorm_finish(WsGuard guard,
                                                            const int64_t* __restrict__ chunk_prefix,
                                                            const double* __restrict__ partials,
                                                            double* __restrict__ sk)
{
    __shared__ double acc[kThreads];
    if (!guard_ok(guard))
        return;
    constexpr int U = 8;  // loads in flight per accumulator; the additions stay in order
    const int k = blockIdx.x;
    const int t = threadIdx.x;
    const int64_t c0 = chunk_prefix[k];
    const int64_t nc = chunk_prefix[k + 1] - c0;
    double b = 0.0;  // accumulator t takes chunks c = t (mod 256), ascending
    int64_t c = t;
    for (; c + (U - 1) * kThreads < nc; c += U * kThreads) {
        double p[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            p[u] = partials[c0 + c + u * kThreads];
#pragma unroll
        for (int u = 0; u < U; ++u)
            b = b + p[u];
    }
    for (; c < nc; c += kThreads)
        b = b + partials[c0 + c];
    acc[t] = b;
    __syncthreads();
    if (t < 128) {
        b = b + acc[t + 128];
        acc[t] = b;
    }
    __syncthreads();
    if (t < 64) {
        b = b + acc[t + 64];
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1)
            b = b + __shfl_xor(b, o, 64);
        if (t == 0)
            sk[k] = b;
    }
}

// A workspace that does not hold this launch's descriptors (see guard_ok) gives
// S = NaN and LT_STATUS_BAD_WORKSPACE, which every step then skips on.
__global__ __launch_bounds__(256) void k_sqnorm_total(WsGuard guard, const double* __restrict__ sk,
                                                      int n_tensors,
                                                      double* __restrict__ sk_out,
                                                      double* __restrict__ sq_total,
                                                      int32_t* __restrict__ status)
{
    __shared__ double batch[1024];
    if (!guard_ok(guard)) {
        if (threadIdx.x == 0) {
            *sq_total = __builtin_nan("");
            *status = LT_STATUS_BAD_WORKSPACE;
        }
        return;
    }
    double S = 0.0;  // kept by thread 0: the list-order sum
    for (int k0 = 0; k0 < n_tensors; k0 += 1024) {
        const int n = min(1024, n_tensors - k0);
        for (int i = threadIdx.x; i < n; i += 256) {
            const double v = sk[k0 + i];
            batch[i] = v;
            if (sk_out)
                sk_out[k0 + i] = v;
        }
        __syncthreads();
        if (threadIdx.x == 0)
            for (int i = 0; i < n; ++i)
                S = S + batch[i];
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        *sq_total = S;
        *status = isfinite(S) ? LT_STATUS_OK : LT_STATUS_NONFINITE;
    }
}

// ------------------------------------------------------ a3: clip coefficient

// Spacing of fp32 values just above (up) and just below (down) a positive
// finite fp32 f, as doubles.
__device__ inline void fp32_spacing(float f, double* up, double* down)
{
    const uint32_t u = __float_as_uint(f);
    const int biased = int(u >> 23);
    if (biased == 0) {  // subnormal
        *up = *down = 0x1p-149;
        return;
    }
    *up = ldexp(1.0, biased - 127 - 23);
    *down = ((u & 0x7FFFFFu) == 0 && biased > 1) ? *up * 0.5 : *up;
}

// The fp32 value nearest sqrt(S) (ties to even) for any double S >= 0.  An
// approximate square root is corrected against the exact squares of the two
// neighbouring fp32 midpoints: a midpoint has at most 25 significant bits, so
// its square is exact in fp64.
__device__ float sqrt_fp32_single_rounding(double S)
{
    float f = float(sqrt(S));
    if (!(S > 0.0) || !isfinite(f))
        return f;  // 0, NaN, +inf, and overflow to +inf (the exact result rounds there too)
    for (int i = 0; i < 4; ++i) {
        double up, down;
        fp32_spacing(f, &up, &down);
        const double hi = double(f) + 0.5 * up;
        const double lo = double(f) - 0.5 * down;
        const bool odd = (__float_as_uint(f) & 1u) != 0;
        if (S > hi * hi || (S == hi * hi && odd))
            f = __uint_as_float(__float_as_uint(f) + 1u);
        else if (__float_as_uint(f) != 0u && (S < lo * lo || (S == lo * lo && odd)))
            f = __uint_as_float(__float_as_uint(f) - 1u);  // +0 has no smaller neighbour >= 0
        else
            break;
    }
    return f;
}

// The norm is defined as fp32(sqrt(S)) with the fp64 square root correctly
// rounded first: two roundings.  They differ from one rounding only when the
// fp64 root lands exactly on an fp32 midpoint m; then the conversion ties to
// even.  The fp64 root is m exactly when m - u/2 < sqrt(S) < m + u/2 (u the fp64
// ulp of m; sqrt(S) is never itself an fp64 midpoint), i.e. when
// -m*u < S - m*m <= m*u: m*m is exact (25-bit m), S - m*m is exact (Sterbenz:
// S is within a factor of two of m*m), m*u is exact, and the u*u/4 terms of the
// squares lie far below the spacing of S - m*m.
__device__ float norm_from_sum_of_squares(double S)
{
    const float f = sqrt_fp32_single_rounding(S);
    if (!(S > 0.0) || !isfinite(f))
        return f;
    double up, down;
    fp32_spacing(f, &up, &down);
    const uint32_t fb = __float_as_uint(f);
    for (int side = 0; side < 2; ++side) {
        const double m = side == 0 ? double(f) + 0.5 * up : double(f) - 0.5 * down;
        if (!(m > 0.0))
            continue;
        const int e = int((__double_as_longlong(m) >> 52) & 0x7FF) - 1023;
        const double u = ldexp(1.0, e - 52);
        const double d = S - m * m;
        if (d > -m * u && d <= m * u) {
            const uint32_t lo = side == 0 ? fb : fb - 1u;  // fp32 neighbours lo, lo + 1 of m
            return __uint_as_float((lo & 1u) ? lo + 1u : lo);
        }
    }
    return f;
}

// status (may be null): OK or NONFINITE from S, unless it holds another value
// (a library error), which it keeps.
__global__ __launch_bounds__(64) void k_clip_coef(const double* __restrict__ sq_total, float max_norm,
                                                  float* __restrict__ total_norm,
                                                  float* __restrict__ coef,
                                                  int32_t* __restrict__ status)
{
    if (threadIdx.x != 0)
        return;
    const double S = *sq_total;
    const float norm = norm_from_sum_of_squares(S);
    const float c = max_norm / (norm + 1e-6f);
    if (total_norm)
        *total_norm = norm;
    *coef = fminf(1.0f, c);
    if (status) {
        const int32_t old = *status;
        if (old == LT_STATUS_OK || old == LT_STATUS_NONFINITE)
            *status = isfinite(S) ? LT_STATUS_OK : LT_STATUS_NONFINITE;
    }
}

// ------------------------------------------------------ a4-a10: fused step
//
// Geometry.  A lane owns E consecutive-granule slots (granule j of lane l is
// elements 8*(l + 64*j) .. +7 of its wave's span), so each load instruction of
// a wave covers one contiguous 1-2 KB run.  E = 32 (16 with the dynamic map for
// B <= 4096), except that B = 1024 and every B <= 512 take 16.  When a
// block is no longer than a wave's span, a wave owns whole blocks and the block
// absmax is a wave reduction; otherwise B / (64 E) <= 4 waves of a workgroup
// share a block and combine their maxima in LDS.
//
// Blocks of B <= 512 elements are at most one row of the span (64 granules), so
// one lane's granules fall in G different blocks and a span holds 64 E / B of
// them.  Their per-block scalars (stored scales, code steps, new maxima,
// reciprocals) are computed once per block, block t of the span in lane t, and
// each lane fetches the values of its granules' blocks by lane permutes; the G
// rows of per-granule maxima are reduced over their blocks' lanes together, by
// recursive halving.  A lane thus does the per-block work of one block for 16
// elements rather than for every 8.  Measured on the 3B-class step against one
// granule per lane: 4-6% faster with the linear map and 3-5% with the dynamic map
// at B = 64..512, which brings them within 1-3% (linear) and 1% (dynamic) of
// B = 2048.  32 elements per lane gained nothing with the linear map: at about
// 190 VGPRs it runs two waves per SIMD.

// 32 elements per lane amortizes the per-block work (scales, maxima, the sqrt
// ballot) over long contiguous runs; measured on the 3B-class step it beats 16
// and 8 per lane.  The lane's granules are loaded and updated in kStepPhases
// phases (when its granule count divides evenly), which bounds the registers the
// loads occupy: about 160 VGPRs, three waves per SIMD, against about 210 and two
// waves with every load issued first.  One, two and four phases time within 0.5%
// of each other; four is the fastest of them.
constexpr int kStepElemsPerLane = 32;
// With the dynamic code map the per-element work adds LDS table reads, whose
// latency more waves hide better: 16 elements per lane (about 126 VGPRs, four
// waves per SIMD) measured 5% faster than 32 and 1% faster than 8 on the
// 3B-class step.  Block sizes whose block would then span more than the four
// waves of a workgroup keep 32.
constexpr int kStepElemsDynamic = 16;
// Blocks of 512 elements or fewer (several blocks per wave span).
constexpr int kStepElemsSmall = 16;
constexpr int kStepPhases = 4;

// Elements per lane at most, by block size and code map.
constexpr int step_elems_max(int B, bool dynamic)
{
    return dynamic && B <= 64 * 4 * kStepElemsDynamic ? kStepElemsDynamic : kStepElemsPerLane;
}

template <int B, bool DYN = false>
struct StepGeom {
    static constexpr int E_MAX = step_elems_max(B, DYN);
    static constexpr bool SMALL = B <= 512;                            // several blocks per span
    static constexpr int E = SMALL ? kStepElemsSmall : (B >= 64 * E_MAX ? E_MAX : B / 64);
    static constexpr int G = E / kGranule;                             // granules per lane
    static constexpr int WAVE_SPAN = 64 * E;                           // elements per wave pass
    static constexpr int W = B > WAVE_SPAN ? B / WAVE_SPAN : 1;        // waves per block
    static constexpr int L = SMALL ? B / kGranule : 64;                // lanes per block in a row
    static constexpr int NB = SMALL ? WAVE_SPAN / B : 1;               // blocks per wave span
    static constexpr int R = 64 / L;                                   // blocks per row
    static constexpr int UNIT = W > 1 ? 4 * WAVE_SPAN : WAVE_SPAN;      // elements per work unit
    static constexpr int PH = G % kStepPhases == 0 ? kStepPhases : 1;   // load phases
    static_assert(W <= 4, "a block spans at most the four waves of one workgroup");
    static_assert(!SMALL || (NB == G * R && NB <= 64 && L >= G), "small-block geometry");
};

// Maxima of a lane's G granule rows over the L lanes of each row's block (L a
// power of two >= G, groups of L consecutive lanes), by recursive halving: at
// each of log2(G) levels, with partner lane ^ o, a lane keeps one half of its
// remaining rows (the upper half when its bit o is set), sends the other half and
// takes the partner's maxima of the half it kept; then plain exchanges finish the
// reduction over the group.  The lane ends with the maximum of one row over its
// whole group, the row whose binary digits are the lane's bits L/2, L/4, ...
// (halving_lane below gives a lane for each row).  max is exact and order-free,
// so the result is the block maximum however the exchanges pair up.
template <int G, int L>
__device__ inline float halving_max(const float (&p)[G], int lane)
{
    constexpr int LG = G == 4 ? 2 : (G == 2 ? 1 : 0);
    static_assert((1 << LG) == G && L >= G, "halving over a power of two of rows");
    float x[G];
#pragma unroll
    for (int j = 0; j < G; ++j)
        x[j] = p[j];
#pragma unroll
    for (int h = 0; h < LG; ++h) {
        const int c = G >> h, o = L >> (h + 1);
        const bool hi = (lane & o) != 0;
#pragma unroll
        for (int i = 0; i < c / 2; ++i) {
            const float keep = hi ? x[c / 2 + i] : x[i];
            const float send = hi ? x[i] : x[c / 2 + i];
            x[i] = fmaxf(keep, __shfl_xor(send, o, 64));
        }
    }
#pragma unroll
    for (int o = L >> (LG + 1); o >= 1; o >>= 1)
        x[0] = fmaxf(x[0], __shfl_xor(x[0], o, 64));
    return x[0];
}

// The lane of a group of L that ends halving_max<G, L> holding row j's maximum
// (the first such lane; the bits below L >> log2(G) are free).
template <int G, int L>
__device__ inline int halving_lane(int j)
{
    constexpr int LG = G == 4 ? 2 : (G == 2 ? 1 : 0);
    int lane = 0;
#pragma unroll
    for (int h = 0; h < LG; ++h)
        if ((j >> (LG - 1 - h)) & 1)
            lane |= L >> (h + 1);
    return lane;
}

__device__ inline float wave_max_xor(float x, int width)
{
    for (int o = width >> 1; o >= 1; o >>= 1)
        x = fmaxf(x, __shfl_xor(x, o, 64));
    return x;
}

// a / 127 and a / 255, correctly rounded, for every fp32 a: the product with
// the rounded reciprocal, corrected once by its fma residual; zero, infinite
// and NaN inputs take the plain product.  A CPU test checks all 2^32 inputs.
template <int D>
__device__ inline float div_by_const(float a)
{
    constexpr float c = D == 127 ? 0x1.020408p-7f : 0x1.010102p-8f;  // RN(1/D)
    const float q = a * c;
    const float r = __builtin_fmaf(-q, float(D), a);
    const float q1 = __builtin_fmaf(r, c, q);
    return __builtin_amdgcn_classf(a, 0x267) ? q : q1;  // 0x267: +-0, +-inf, NaN
}

// Correctly rounded sqrt of an fp32 v that is 0, >= 2^-96, infinite or NaN:
// the hardware estimate corrected by the signs of the fma residuals of its two
// neighbours.  This is the sequence the compiler emits for sqrtf once the
// scaling it applies to inputs below 2^-96 is not needed.
__device__ inline float sqrt_rn_unscaled(float v)
{
    const float s = __builtin_amdgcn_sqrtf(v);
    const float dn = __uint_as_float(__float_as_uint(s) - 1u);
    const float up = __uint_as_float(__float_as_uint(s) + 1u);
    const float r_dn = __builtin_fmaf(-dn, s, v);
    const float r_up = __builtin_fmaf(-up, s, v);
    float t = r_dn <= 0.0f ? dn : s;
    t = r_up > 0.0f ? up : t;
    return t;
}

// The inputs of one granule (8 consecutive elements of a tensor), as loaded.
template <typename GT>
struct StepIn {
    uint4 w[2];
    GradWords<GT> g;
    uint2 m, v;
};

// The gradients are read once and never written back, so their loads carry the
// streaming (non-temporal) hint: measured 0.4% faster on the whole 3B-class step
// (16 alternating rounds).  Loads of data that the step writes back keep the
// default policy: streaming those costs 4% in a probe of the same byte mix.
template <typename GT>
__device__ inline void load_step_full(const StepTensor& d, int64_t ei, StepIn<GT>& in)
{
    load_grads<true>(static_cast<const GT*>(d.g) + ei, kGranule, in.g);
    in.w[0] = load16(d.w + ei);
    in.w[1] = load16(d.w + ei + 4);
    in.m = load8(d.mq + ei);
    in.v = load8(d.vq + ei);
}

// Ragged granule: the first nv (0..8) elements exist, the others read as 0.
template <typename GT>
__device__ inline void load_step_ragged(const StepTensor& d, int64_t ei, int nv, StepIn<GT>& in)
{
    load_grads<true>(static_cast<const GT*>(d.g) + ei, nv, in.g);
    uint32_t wb[8], mb[8], vb[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const bool ok = e < nv;
        wb[e] = ok ? __float_as_uint(gp(d.w)[ei + e]) : 0u;
        mb[e] = ok ? uint32_t(uint8_t(gp(d.mq)[ei + e])) : 0u;
        vb[e] = ok ? uint32_t(gp(d.vq)[ei + e]) : 0u;
    }
    in.w[0] = make_uint4(wb[0], wb[1], wb[2], wb[3]);
    in.w[1] = make_uint4(wb[4], wb[5], wb[6], wb[7]);
    in.m = make_uint2(mb[0] | (mb[1] << 8) | (mb[2] << 16) | (mb[3] << 24),
                      mb[4] | (mb[5] << 8) | (mb[6] << 16) | (mb[7] << 24));
    in.v = make_uint2(vb[0] | (vb[1] << 8) | (vb[2] << 16) | (vb[3] << 24),
                      vb[4] | (vb[5] << 8) | (vb[6] << 16) | (vb[7] << 24));
}

// bf16 copy of eight updated weights (nv of them exist): round to nearest even,
// by the hardware's packed conversion.
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ inline uint32_t bf16_pair(float lo, float hi)
{
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

__device__ inline void store_bf16x8(uint16_t* p, int nv, const float (&w)[8])
{
    const uint4 q = make_uint4(bf16_pair(w[0], w[1]), bf16_pair(w[2], w[3]),
                               bf16_pair(w[4], w[5]), bf16_pair(w[6], w[7]));
    if (nv >= kGranule) {
        store16(p, q);
        return;
    }
    const uint32_t word[4] = {q.x, q.y, q.z, q.w};
    for (int e = 0; e < nv; ++e)
        gp(p)[e] = uint16_t(word[e >> 1] >> (16 * (e & 1)));
}

// Packs four codes held as exact small integers (as floats) into one word.
// q must lie in [0, 255] (m codes arrive offset by +128).
__device__ inline uint32_t pack4(float q0, float q1, float q2, float q3)
{
    uint32_t w = __builtin_amdgcn_cvt_pk_u8_f32(q0, 0, 0u);
    w = __builtin_amdgcn_cvt_pk_u8_f32(q1, 1, w);
    w = __builtin_amdgcn_cvt_pk_u8_f32(q2, 2, w);
    return __builtin_amdgcn_cvt_pk_u8_f32(q3, 3, w);
}

// ------------------------------------------- f2: dynamic code map tables
//
// Sign-magnitude dynamic tree codes (Dettmers et al., block-wise 8-bit
// optimizers): a code's magnitude bits are leading zeros z (the decade
// 10^-z), an indicator one and p fraction bits f, with magnitude
// fp32((0.1 + 0.9 * ((f + 1) / 2^p)) * 10^-z) computed in fp64 in that order;
// the first moment has a sign bit (set for m < 0) and 7 magnitude bits
// (1e-6 .. 1), the second 8 magnitude bits (1e-7 .. 1).  Encoding picks the
// magnitude nearest to the normalized value a by fp32 distance (ties to the
// smaller code).
//
// The kernel encodes with one LDS read and one integer add.  The fp32
// pattern's exponent and top 7 mantissa bits (pattern >> 16) index a bucket.
// No bucket holds two decision points of the map (the builder checks it), so
// inside bucket i the answer is the nearest code c_i at the bucket's lower end
// up to some pattern, and c_i + 1 above it.  The bucket's entry is
// (c_i << 16) + (0xFFFF - l_i), l_i the low 16 bits of the last pattern that
// still takes c_i: adding the pattern's low 16 bits carries into the code
// exactly when they exceed l_i.  Patterns below the first bucket take code 0;
// patterns above the last bucket (only NaN and negative values reach them)
// take the sentinel entry 0: code 0.  Decoding reads one of 256 signed (or
// unsigned) magnitudes per byte.  All tables are built at compile time and
// copied to LDS by each workgroup.
namespace dyn {

constexpr double kPow10[8] = {1.0, 1e-1, 1e-2, 1e-3, 1e-4, 1e-5, 1e-6, 1e-7};

constexpr float magnitude(int c, int bits)
{
    if (c == 0)
        return 0.0f;
    int p = 0;
    while ((c >> (p + 1)) != 0)
        ++p;
    const int zeros = bits - 1 - p;
    const int f = c - (1 << p);
    return float((0.1 + 0.9 * (double(f + 1) / double(1 << p))) * kPow10[zeros]);
}

// Buckets: (pattern >> 16) - base.  Bucket 0 starts at 2^-21 (signed) or 2^-25
// (unsigned), below half the smallest nonzero magnitude; bucket `top` starts
// at 1.0 (normalized values never exceed 1 + 2^-23); bucket top + 1 is the
// sentinel.
constexpr int kBaseM = (127 - 21) << 7, kTopM = (127 << 7) - kBaseM;
constexpr int kBaseV = (127 - 25) << 7, kTopV = (127 << 7) - kBaseV;

struct Tables {
    float dm[256];               // decoding: +-magnitude of every m byte (0x80 is -0)
    float dv[256];               // decoding: magnitude of every v byte
    uint32_t em[kTopM + 2];      // bucket entries: (code << 16) + 0xFFFF - last low half
    uint32_t ev[kTopV + 2];
    float tm[128];               // signed magnitudes (building only)
    float tv[256];               // unsigned magnitudes (building only)
    uint32_t one_decision_per_bucket;  // checked at compile time
};

constexpr float from_bits(uint32_t u) { return __builtin_bit_cast(float, u); }

// The rule between neighbours: code c + 1 beats c when its fp32 distance is smaller.
constexpr bool next_wins(const float* t, int n, int c, float a)
{
    return c + 1 < n && (t[c + 1] - a) < (a - t[c]);
}

// Nearest magnitude to a >= 0 among t[0..n): the largest c with t[c] <= a by
// binary search (t rises strictly, t[0] = 0), then that code or the next.
constexpr int nearest(const float* t, int n, float a)
{
    int lo = 0, hi = n - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (t[mid] <= a)
            lo = mid;
        else
            hi = mid - 1;
    }
    return next_wins(t, n, lo, a) ? lo + 1 : lo;
}

// A bucket's entry; *ok is cleared when the bucket holds two decision points.
constexpr uint32_t bucket_entry(const float* t, int n, int bucket_hi16, uint32_t* ok)
{
    const uint32_t p0 = uint32_t(bucket_hi16) << 16;
    const int c = nearest(t, n, from_bits(p0));
    if (nearest(t, n, from_bits(p0 | 0xFFFFu)) > c + 1)
        *ok = 0;
    if (!next_wins(t, n, c, from_bits(p0 | 0xFFFFu)))
        return uint32_t(c) << 16;
    // the first low half where c + 1 wins (the rule is monotone in a), in (0, 0xFFFF]
    uint32_t a = 1, b = 0xFFFF;
    while (a < b) {
        const uint32_t mid = (a + b) / 2;
        if (next_wins(t, n, c, from_bits(p0 | mid)))
            b = mid;
        else
            a = mid + 1;
    }
    return (uint32_t(c) << 16) + (0xFFFFu - (a - 1));
}

constexpr Tables make_tables()
{
    Tables x{};
    for (int c = 0; c < 128; ++c)
        x.tm[c] = magnitude(c, 7);
    for (int c = 0; c < 256; ++c)
        x.tv[c] = magnitude(c, 8);
    for (int b = 0; b < 256; ++b) {
        x.dm[b] = (b & 0x80) ? -x.tm[b & 0x7F] : x.tm[b & 0x7F];
        x.dv[b] = x.tv[b];
    }
    x.one_decision_per_bucket = 1;
    for (int i = 0; i <= kTopM; ++i)
        x.em[i] = bucket_entry(x.tm, 128, kBaseM + i, &x.one_decision_per_bucket);
    for (int i = 0; i <= kTopV; ++i)
        x.ev[i] = bucket_entry(x.tv, 256, kBaseV + i, &x.one_decision_per_bucket);
    x.em[kTopM + 1] = 0;  // sentinel: code 0
    x.ev[kTopV + 1] = 0;
    return x;
}

constexpr Tables kTablesHost = make_tables();
static_assert(kTablesHost.one_decision_per_bucket, "a bucket holds two decision points");
// the first bucket must take code 0 throughout (smaller patterns are clamped into it)
static_assert(kTablesHost.em[0] == 0 && kTablesHost.ev[0] == 0, "first bucket");

// What the kernels read, copied to LDS (the building tables stay out).
struct LdsTables {
    float dm[256];
    float dv[256];
    uint32_t em[kTopM + 2];
    uint32_t ev[kTopV + 2];
};

constexpr LdsTables lds_tables()
{
    LdsTables y{};
    for (int i = 0; i < 256; ++i) {
        y.dm[i] = kTablesHost.dm[i];
        y.dv[i] = kTablesHost.dv[i];
    }
    for (int i = 0; i < kTopM + 2; ++i)
        y.em[i] = kTablesHost.em[i];
    for (int i = 0; i < kTopV + 2; ++i)
        y.ev[i] = kTablesHost.ev[i];
    return y;
}

__constant__ const LdsTables kTables = lds_tables();

// Code of the normalized magnitude a (>= 0; NaN and negative values give 0).
template <int BASE, int TOP>
__device__ inline uint32_t encode(const uint32_t* entries, float a)
{
    const uint32_t bits = __float_as_uint(a);
    int i = int(bits >> 16) - BASE;
    i = i < 0 ? 0 : (i > TOP + 1 ? TOP + 1 : i);
    return (entries[i] + (bits & 0xFFFFu)) >> 16;
}

}  // namespace dyn

constexpr int kMapLinear = 0, kMapDynamic = 1;

// WB: some tensor of the launch asks for the bf16 weight copy (a separate
// instantiation keeps the copy's code out of the launches that do not).
// MAP: the code map of both moments, kMapLinear or kMapDynamic.
template <typename GT, int B, bool WB, int MAP>
__global__ __launch_bounds__(kThreads) void k_adamw8_step(WsGuard guard,
                                                          const int64_t* __restrict__ unit_prefix,
                                                          const StepTensor* __restrict__ desc,
                                                          int n_tensors, int64_t n_units,
                                                          StepScalars s,
                                                          const float* __restrict__ coef_ptr,
                                                          const int32_t* __restrict__ status_ptr)
{
    using Geo = StepGeom<B, MAP == kMapDynamic>;
    constexpr int E = Geo::E, G = Geo::G, W = Geo::W, L = Geo::L, UNIT = Geo::UNIT, PH = Geo::PH;
    constexpr bool SMALL = Geo::SMALL;
    constexpr int NB = Geo::NB, R = Geo::R;
    __shared__ float red[2][2][4];  // [buffer][m, v][wave], used when W > 1

    if (!guard_ok(guard))
        return;  // the workspace does not hold this launch's descriptors
    if (status_ptr && *status_ptr != LT_STATUS_OK)
        return;  // skipped step: nothing is written
    if (!resolve_step(s))
        return;  // the step state lets no step apply
    const float coef = coef_ptr ? *coef_ptr : 1.0f;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    // Dynamic map: the workgroup copies the code tables into LDS once.
    __shared__ __align__(16) uint8_t dyn_lds[MAP == kMapDynamic ? sizeof(dyn::LdsTables) : 16];
    const dyn::LdsTables& tab = *reinterpret_cast<const dyn::LdsTables*>(dyn_lds);
    if constexpr (MAP == kMapDynamic) {
        static_assert(sizeof(dyn::LdsTables) % 4 == 0, "tables copy in words");
        const auto* src = reinterpret_cast<const uint32_t*>(&dyn::kTables);
        auto* dst = reinterpret_cast<uint32_t*>(dyn_lds);
        for (int i = threadIdx.x; i < int(sizeof(dyn::LdsTables) / 4); i += kThreads)
            dst[i] = src[i];
        __syncthreads();
    }

    // Work units: wave spans (W == 1, each wave on its own) or workgroup spans,
    // handed to the workers in turn, so that at any moment the chip streams one
    // contiguous region of every array.  Measured on the 3B-class step: 2%
    // faster than one contiguous range of units per worker.
    const int64_t workers = W > 1 ? int64_t(gridDim.x) : int64_t(gridDim.x) * 4;
    const int64_t me = W > 1 ? int64_t(blockIdx.x) : int64_t(blockIdx.x) * 4 + wave;
    // Offset of this wave's span inside a unit.
    const int64_t span0 = W > 1 ? int64_t(wave) * Geo::WAVE_SPAN : 0;
    int k = me < n_units ? find_tensor(unit_prefix, n_tensors, me) : 0;
    int buf = 0;
    for (int64_t u = me; u < n_units; u += workers, buf ^= 1) {
        while (u >= unit_prefix[k + 1])
            ++k;
        const StepTensor d = desc[k];
        const int64_t e_unit = (u - unit_prefix[k]) * UNIT;
        const int64_t e0 = e_unit + span0;          // first element of this wave's span
        const int64_t n_span = d.numel - e0;        // elements left from e0 (may be <= 0)
        const bool full = n_span >= Geo::WAVE_SPAN;  // wave-uniform

        // Stored scales: of the wave's block (B >= 1024), or of block `lane` of
        // the span (B <= 512; lanes past the span's blocks, or past the tensor's
        // end, hold zero).
        float a_m, a_v;
        {
            const int64_t o = SMALL ? int64_t(B) * lane : 0;
            const bool exists = (!SMALL || lane < NB) && n_span > o;
            const int64_t blk = (e0 + o) / B;
            a_m = exists ? gp(d.ma)[blk] : 0.0f;
            a_v = exists ? gp(d.va)[blk] : 0.0f;
        }
        // The dequantization factors: the code steps A/127 and A/255 (linear map)
        // or the scales themselves (dynamic map).
        const float f_m = MAP == kMapLinear ? div_by_const<127>(a_m) : a_m;
        const float f_v = MAP == kMapLinear ? div_by_const<255>(a_v) : a_v;
        // Block of the span that granule row j of this lane falls in (B <= 512).
        auto block_of = [&](int j) { return j * R + lane / L; };

        // The lane's granules go through load -> moments -> sqrt/divide -> weight
        // store in PH phases, which bounds the registers the loads occupy.  m1 and
        // v1 of every granule stay for the block's requantization.  Elements past
        // the end read as zero gradient and zero codes, so they produce
        // m1 = v1 = 0 (or NaN from a non-finite stored scale) and leave the block
        // maxima unchanged.
        float m1[E], v1[E];
        float amax_m = 0.0f, amax_v = 0.0f;  // over the lane's elements (B >= 1024)
        float rmax_m[G], rmax_v[G];          // per granule row (B <= 512)
#pragma unroll
        for (int j = 0; j < G; ++j)
            rmax_m[j] = rmax_v[j] = 0.0f;
#pragma unroll
        for (int ph = 0; ph < PH; ++ph) {
            constexpr int GP = G / PH;
            StepIn<GT> in[GP];
            if (full) {
#pragma unroll
                for (int jj = 0; jj < GP; ++jj)
                    load_step_full(d, e0 + kGranule * (lane + 64 * (ph * GP + jj)), in[jj]);
            } else {
#pragma unroll
                for (int jj = 0; jj < GP; ++jj) {
                    const int64_t o = kGranule * (lane + 64 * (ph * GP + jj));
                    load_step_ragged(d, e0 + o, int(i64min(i64max(n_span - o, 0), kGranule)),
                                     in[jj]);
                }
            }
#pragma unroll
            for (int jj = 0; jj < GP; ++jj) {
                const int j = ph * GP + jj;
                float g[8];
                unpack8(in[jj].g, g);
                const float fm = SMALL ? __shfl(f_m, block_of(j), 64) : f_m;
                const float fv = SMALL ? __shfl(f_v, block_of(j), 64) : f_v;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const uint32_t mw = e < 4 ? in[jj].m.x : in[jj].m.y;
                    const uint32_t vw = e < 4 ? in[jj].v.x : in[jj].v.y;
                    float m0, v0;
                    if constexpr (MAP == kMapLinear) {
                        m0 = float(int8_t(mw >> (8 * (e & 3)))) * fm;
                        v0 = float((vw >> (8 * (e & 3))) & 0xFFu) * fv;
                    } else {
                        m0 = tab.dm[(mw >> (8 * (e & 3))) & 0xFFu] * fm;
                        v0 = tab.dv[(vw >> (8 * (e & 3))) & 0xFFu] * fv;
                    }
                    const float gc = g[e] * coef;
                    m1[8 * j + e] = __builtin_fmaf(s.beta1, m0, s.c1 * gc);
                    v1[8 * j + e] = __builtin_fmaf(s.beta2, v0, s.c2 * (gc * gc));
                }
            }
            // sqrt: the short correction sequence is exact unless some v1 of the
            // wave (in this phase) lies in (0, 2^-96); then every lane takes the
            // full sqrtf.
            uint32_t vmin = 0xFFFFFFFFu;
#pragma unroll
            for (int e = ph * 8 * GP; e < (ph + 1) * 8 * GP; ++e)
                vmin = min(vmin, __float_as_uint(v1[e]) - 1u);  // 0 wraps to the top
            const bool scaled = __builtin_amdgcn_ballot_w64(vmin < 0x0F800000u - 1u) != 0;
#pragma unroll
            for (int jj = 0; jj < GP; ++jj) {
                const int j = ph * GP + jj;
                float w[8];
                w[0] = __uint_as_float(in[jj].w[0].x); w[1] = __uint_as_float(in[jj].w[0].y);
                w[2] = __uint_as_float(in[jj].w[0].z); w[3] = __uint_as_float(in[jj].w[0].w);
                w[4] = __uint_as_float(in[jj].w[1].x); w[5] = __uint_as_float(in[jj].w[1].y);
                w[6] = __uint_as_float(in[jj].w[1].z); w[7] = __uint_as_float(in[jj].w[1].w);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float m = m1[8 * j + e], v = v1[8 * j + e];
                    const float root = scaled ? sqrtf(v) : sqrt_rn_unscaled(v);
                    const float den = __builtin_fmaf(root, s.rbc2, s.eps);
                    w[e] = __builtin_fmaf(-s.step_size, m / den, w[e] * s.decay);
                    if constexpr (SMALL) {
                        rmax_m[j] = fmaxf(rmax_m[j], fabsf(m));
                        rmax_v[j] = fmaxf(rmax_v[j], v);
                    } else {
                        amax_m = fmaxf(amax_m, fabsf(m));
                        amax_v = fmaxf(amax_v, v);
                    }
                }
                const int64_t ei = e0 + kGranule * (lane + 64 * j);
                if (full) {
                    store16f(d.w + ei, w[0], w[1], w[2], w[3]);
                    store16f(d.w + ei + 4, w[4], w[5], w[6], w[7]);
                } else {
                    const int nv =
                        int(i64min(i64max(n_span - kGranule * (lane + 64 * j), 0), kGranule));
                    for (int e = 0; e < nv; ++e)
                        gp(d.w)[ei + e] = w[e];
                }
                if (WB && d.wb) {
                    const int nv = full ? kGranule
                                        : int(i64min(i64max(n_span - kGranule * (lane + 64 * j), 0),
                                                     kGranule));
                    store_bf16x8(d.wb + ei, nv, w);
                }
            }
        }

        // Block absmax (max is exact and order-free).  B <= 512: lane t < NB
        // ends with block t's maxima.
        if constexpr (SMALL) {
            const int src = (lane % R) * L + halving_lane<G, L>(lane / R);
            amax_m = __shfl(halving_max<G, L>(rmax_m, lane), src, 64);
            amax_v = __shfl(halving_max<G, L>(rmax_v, lane), src, 64);
        } else {
            amax_m = wave_max_xor(amax_m, L);
            amax_v = wave_max_xor(amax_v, L);
        }
        if constexpr (W > 1) {
            if (lane == 0) {
                red[buf][0][wave] = amax_m;
                red[buf][1][wave] = amax_v;
            }
            __syncthreads();
            const int first = (wave / W) * W;
            amax_m = red[buf][0][first];
            amax_v = red[buf][1][first];
#pragma unroll
            for (int i = 1; i < W; ++i) {
                amax_m = fmaxf(amax_m, red[buf][0][first + i]);
                amax_v = fmaxf(amax_v, red[buf][1][first + i]);
            }
        }
        const float inv_m = (MAP == kMapLinear ? 127.0f : 1.0f) / amax_m;
        const float inv_v = (MAP == kMapLinear ? 255.0f : 1.0f) / amax_v;
        const bool ok_m = isfinite(amax_m) && isfinite(inv_m);
        const bool ok_v = isfinite(amax_v) && isfinite(inv_v);
        // B <= 512: which of the span's blocks (bit t: block t) requantize
        const uint64_t okm_blocks = SMALL ? __builtin_amdgcn_ballot_w64(ok_m) : 0;
        const uint64_t okv_blocks = SMALL ? __builtin_amdgcn_ballot_w64(ok_v) : 0;

#pragma unroll
        for (int j = 0; j < G; ++j) {
            // this granule's block: its reciprocals and whether it requantizes
            const float jinv_m = SMALL ? __shfl(inv_m, block_of(j), 64) : inv_m;
            const float jinv_v = SMALL ? __shfl(inv_v, block_of(j), 64) : inv_v;
            const bool jok_m = SMALL ? ((okm_blocks >> block_of(j)) & 1u) != 0 : ok_m;
            const bool jok_v = SMALL ? ((okv_blocks >> block_of(j)) & 1u) != 0 : ok_v;
            uint32_t pm0, pm1, pv0, pv1;
            if constexpr (MAP == kMapLinear) {
                float qm[8], qv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    // clamp, then shift m codes by +128 (exact) so both pack as unsigned bytes
                    qm[e] = fminf(fmaxf(rintf(m1[8 * j + e] * jinv_m), -127.0f), 127.0f) + 128.0f;
                    qv[e] = fminf(fmaxf(rintf(v1[8 * j + e] * jinv_v), 0.0f), 255.0f);
                }
                // m: undo the offset on all four bytes at once (two's complement int8)
                pm0 = pack4(qm[0], qm[1], qm[2], qm[3]) ^ 0x80808080u;
                pm1 = pack4(qm[4], qm[5], qm[6], qm[7]) ^ 0x80808080u;
                pv0 = pack4(qv[0], qv[1], qv[2], qv[3]);
                pv1 = pack4(qv[4], qv[5], qv[6], qv[7]);
            } else {
                uint32_t bm[8], bv[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float m = m1[8 * j + e];
                    const uint32_t c = dyn::encode<dyn::kBaseM, dyn::kTopM>(tab.em,
                                                                           fabsf(m) * jinv_m);
                    bm[e] = c | (m < 0.0f ? 0x80u : 0u);
                    bv[e] = dyn::encode<dyn::kBaseV, dyn::kTopV>(tab.ev, v1[8 * j + e] * jinv_v);
                }
                pm0 = bm[0] | (bm[1] << 8) | (bm[2] << 16) | (bm[3] << 24);
                pm1 = bm[4] | (bm[5] << 8) | (bm[6] << 16) | (bm[7] << 24);
                pv0 = bv[0] | (bv[1] << 8) | (bv[2] << 16) | (bv[3] << 24);
                pv1 = bv[4] | (bv[5] << 8) | (bv[6] << 16) | (bv[7] << 24);
            }
            if (!jok_m)
                pm0 = pm1 = 0u;
            if (!jok_v)
                pv0 = pv1 = 0u;
            const int64_t ei = e0 + kGranule * (lane + 64 * j);
            if (full) {
                store8(d.mq + ei, pm0, pm1);
                store8(d.vq + ei, pv0, pv1);
            } else {
                const int nv = int(i64min(i64max(n_span - kGranule * (lane + 64 * j), 0), kGranule));
                for (int e = 0; e < nv; ++e) {
                    const uint32_t wm = e < 4 ? pm0 : pm1, wv = e < 4 ? pv0 : pv1;
                    gp(d.mq)[ei + e] = int8_t((wm >> (8 * (e & 3))) & 0xFFu);
                    gp(d.vq)[ei + e] = uint8_t((wv >> (8 * (e & 3))) & 0xFFu);
                }
            }
        }
        // The scales: lane t writes block t's (B <= 512), else the first lane of
        // the block's first wave.
        {
            const int64_t o = SMALL ? int64_t(B) * lane : 0;
            const bool first_lane = SMALL ? lane < NB : lane == 0;
            const bool first_wave = W > 1 ? (wave % W) == 0 : true;
            if (first_lane && first_wave && n_span > o) {
                const int64_t blk = (e0 + o) / B;
                gp(d.ma)[blk] = ok_m ? amax_m : 0.0f;
                gp(d.va)[blk] = ok_v ? amax_v : 0.0f;
            }
        }
    }
}

// ---------------------------------------- a4-a10: any block size (generic)
//
// Block sizes outside the set above (any multiple of 64 up to 65536, besides
// the powers of two up to 8192) take this kernel.  It computes exactly what
// k_adamw8_step computes, in a simpler shape: a workgroup owns one block at a
// time and thread t takes the block's granules t, t + 256, ...  Pass 1 updates the
// moments and the weights and finds the block maxima; pass 2 requantizes.  The
// moments m1 and v1 reach pass 2 through LDS when the block's 8 B per element
// fit (STASH, B <= kGenericStashMax); otherwise pass 2 reads the block's
// gradients and old codes again and repeats pass 1's moment operations, which
// give the same bits (4 B per element more traffic with bf16 gradients).  Only
// the thread that wrote a stash entry reads it.
constexpr int kGenericStashMax = 8192;

// The moments of one granule from its loaded inputs (linear map: step_m, step_v;
// dynamic map: the tables and the stored absmax).  Both passes call this.
template <typename GT, int MAP>
__device__ inline void granule_moments(const StepIn<GT>& in, float step_m, float step_v, float a_m,
                                       float a_v, float coef, const StepScalars& s,
                                       const dyn::LdsTables& tab, float (&m1)[8], float (&v1)[8])
{
    float g[8];
    unpack8(in.g, g);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        const uint32_t mw = e < 4 ? in.m.x : in.m.y;
        const uint32_t vw = e < 4 ? in.v.x : in.v.y;
        float m0, v0;
        if constexpr (MAP == kMapLinear) {
            m0 = float(int8_t(mw >> (8 * (e & 3)))) * step_m;
            v0 = float((vw >> (8 * (e & 3))) & 0xFFu) * step_v;
        } else {
            m0 = tab.dm[(mw >> (8 * (e & 3))) & 0xFFu] * a_m;
            v0 = tab.dv[(vw >> (8 * (e & 3))) & 0xFFu] * a_v;
        }
        const float gc = g[e] * coef;
        m1[e] = __builtin_fmaf(s.beta1, m0, s.c1 * gc);
        v1[e] = __builtin_fmaf(s.beta2, v0, s.c2 * (gc * gc));
    }
}

template <typename GT>
__device__ inline void load_granule(const StepTensor& d, int64_t ei, int nv, StepIn<GT>& in)
{
    if (nv >= kGranule)
        load_step_full(d, ei, in);
    else
        load_step_ragged(d, ei, nv, in);
}

template <typename GT, bool WB, int MAP, bool STASH>
__global__ __launch_bounds__(kThreads) void k_adamw8_generic(WsGuard guard,
                                                             const int64_t* __restrict__ unit_prefix,
                                                             const StepTensor* __restrict__ desc,
                                                             int n_tensors, int64_t n_units, int B,
                                                             StepScalars s,
                                                             const float* __restrict__ coef_ptr,
                                                             const int32_t* __restrict__ status_ptr)
{
    extern __shared__ float stash[];  // STASH: m1 at [0, B), v1 at [B, 2B)
    __shared__ float red[2][2][4];    // [buffer][m, v][wave]
    __shared__ __align__(16) uint8_t dyn_lds[MAP == kMapDynamic ? sizeof(dyn::LdsTables) : 16];
    const dyn::LdsTables& tab = *reinterpret_cast<const dyn::LdsTables*>(dyn_lds);

    if (!guard_ok(guard))
        return;  // the workspace does not hold this launch's descriptors
    if (status_ptr && *status_ptr != LT_STATUS_OK)
        return;  // skipped step: nothing is written
    if (!resolve_step(s))
        return;  // the step state lets no step apply
    const float coef = coef_ptr ? *coef_ptr : 1.0f;
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    if constexpr (MAP == kMapDynamic) {
        const auto* src = reinterpret_cast<const uint32_t*>(&dyn::kTables);
        auto* dst = reinterpret_cast<uint32_t*>(dyn_lds);
        for (int i = t; i < int(sizeof(dyn::LdsTables) / 4); i += kThreads)
            dst[i] = src[i];
        __syncthreads();
    }

    int k = int64_t(blockIdx.x) < n_units ? find_tensor(unit_prefix, n_tensors, blockIdx.x) : 0;
    int buf = 0;
    for (int64_t u = blockIdx.x; u < n_units; u += gridDim.x, buf ^= 1) {
        while (u >= unit_prefix[k + 1])
            ++k;
        const StepTensor d = desc[k];
        const int64_t blk = u - unit_prefix[k];
        const int64_t e0 = blk * B;
        const int len = int(i64min(B, d.numel - e0));  // >= 1
        const int n_gran = (len + kGranule - 1) / kGranule;
        const float a_m = gp(d.ma)[blk], a_v = gp(d.va)[blk];
        const float step_m = MAP == kMapLinear ? a_m / 127.0f : 0.0f;
        const float step_v = MAP == kMapLinear ? a_v / 255.0f : 0.0f;

        // pass 1: moments, weights, block maxima
        float amax_m = 0.0f, amax_v = 0.0f;
        for (int gi = t; gi < n_gran; gi += kThreads) {
            const int o = kGranule * gi;
            const int nv = min(kGranule, len - o);
            StepIn<GT> in;
            load_granule(d, e0 + o, nv, in);
            float m1[8], v1[8], w[8];
            granule_moments<GT, MAP>(in, step_m, step_v, a_m, a_v, coef, s, tab, m1, v1);
            w[0] = __uint_as_float(in.w[0].x); w[1] = __uint_as_float(in.w[0].y);
            w[2] = __uint_as_float(in.w[0].z); w[3] = __uint_as_float(in.w[0].w);
            w[4] = __uint_as_float(in.w[1].x); w[5] = __uint_as_float(in.w[1].y);
            w[6] = __uint_as_float(in.w[1].z); w[7] = __uint_as_float(in.w[1].w);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float den = __builtin_fmaf(sqrtf(v1[e]), s.rbc2, s.eps);
                w[e] = __builtin_fmaf(-s.step_size, m1[e] / den, w[e] * s.decay);
                amax_m = fmaxf(amax_m, fabsf(m1[e]));
                amax_v = fmaxf(amax_v, v1[e]);
                if constexpr (STASH) {
                    stash[o + e] = m1[e];
                    stash[B + o + e] = v1[e];
                }
            }
            if (nv >= kGranule) {
                store16f(d.w + e0 + o, w[0], w[1], w[2], w[3]);
                store16f(d.w + e0 + o + 4, w[4], w[5], w[6], w[7]);
            } else {
                for (int e = 0; e < nv; ++e)
                    gp(d.w)[e0 + o + e] = w[e];
            }
            if (WB && d.wb)
                store_bf16x8(d.wb + e0 + o, nv, w);
        }
        amax_m = wave_max_xor(amax_m, 64);
        amax_v = wave_max_xor(amax_v, 64);
        if (lane == 0) {
            red[buf][0][wave] = amax_m;
            red[buf][1][wave] = amax_v;
        }
        __syncthreads();  // also orders this buffer's reads before its next write, two blocks on
        amax_m = fmaxf(fmaxf(red[buf][0][0], red[buf][0][1]), fmaxf(red[buf][0][2], red[buf][0][3]));
        amax_v = fmaxf(fmaxf(red[buf][1][0], red[buf][1][1]), fmaxf(red[buf][1][2], red[buf][1][3]));
        const float inv_m = (MAP == kMapLinear ? 127.0f : 1.0f) / amax_m;
        const float inv_v = (MAP == kMapLinear ? 255.0f : 1.0f) / amax_v;
        const bool ok_m = isfinite(amax_m) && isfinite(inv_m);
        const bool ok_v = isfinite(amax_v) && isfinite(inv_v);

        // pass 2: requantize
        for (int gi = t; gi < n_gran; gi += kThreads) {
            const int o = kGranule * gi;
            const int nv = min(kGranule, len - o);
            float m1[8], v1[8];
            if constexpr (STASH) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    m1[e] = stash[o + e];
                    v1[e] = stash[B + o + e];
                }
            } else {
                StepIn<GT> in;
                load_granule(d, e0 + o, nv, in);
                granule_moments<GT, MAP>(in, step_m, step_v, a_m, a_v, coef, s, tab, m1, v1);
            }
            uint32_t bm[8], bv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                if constexpr (MAP == kMapLinear) {
                    bm[e] = uint32_t(int32_t(fminf(fmaxf(rintf(m1[e] * inv_m), -127.0f), 127.0f))) & 0xFFu;
                    bv[e] = uint32_t(fminf(fmaxf(rintf(v1[e] * inv_v), 0.0f), 255.0f));
                } else {
                    bm[e] = dyn::encode<dyn::kBaseM, dyn::kTopM>(tab.em, fabsf(m1[e]) * inv_m) |
                            (m1[e] < 0.0f ? 0x80u : 0u);
                    bv[e] = dyn::encode<dyn::kBaseV, dyn::kTopV>(tab.ev, v1[e] * inv_v);
                }
                if (!ok_m)
                    bm[e] = 0u;
                if (!ok_v)
                    bv[e] = 0u;
            }
            const int64_t ei = e0 + o;
            if (nv >= kGranule) {
                store8(d.mq + ei, bm[0] | (bm[1] << 8) | (bm[2] << 16) | (bm[3] << 24),
                       bm[4] | (bm[5] << 8) | (bm[6] << 16) | (bm[7] << 24));
                store8(d.vq + ei, bv[0] | (bv[1] << 8) | (bv[2] << 16) | (bv[3] << 24),
                       bv[4] | (bv[5] << 8) | (bv[6] << 16) | (bv[7] << 24));
            } else {
                for (int e = 0; e < nv; ++e) {
                    gp(d.mq)[ei + e] = int8_t(bm[e]);
                    gp(d.vq)[ei + e] = uint8_t(bv[e]);
                }
            }
        }
        if (t == 0) {
            gp(d.ma)[blk] = ok_m ? amax_m : 0.0f;
            gp(d.va)[blk] = ok_v ? amax_v : 0.0f;
        }
    }
}

// ------------------------------------------ f1: fp32-state fused AdamW
//
// The part of the hybrid operator that keeps fp32 moments (the role DeepSpeed
// CPUAdam plays for most parameters in the paper's run): the same per-element
// arithmetic as the 8-bit step with m0, v0 read from and m1, v1 written to fp32
// arrays, 26 B/param with bf16 gradients.  A wave owns spans of 64 x 16
// elements; there is no cross-lane work.

struct Fp32Tensor {
    float* w;
    const void* g;
    float* m;
    float* v;
    int64_t numel;
    uint16_t* wb;  // bf16 copy of the updated weights, or null
    int64_t pad_[2];
};
static_assert(sizeof(Fp32Tensor) == 64, "descriptor is one 64-byte line");

// 32 elements per lane (224-230 VGPRs, 2 waves per SIMD): measured on the 3B-class
// model with fp32 states, 1.2% faster than 16 per lane (4 waves) and 2.7% faster
// than 8 per lane (8 waves), bitwise identical.
constexpr int kFp32ElemsPerLane = 32;

__device__ inline void load8f(const float* p, int nv, float (&x)[8])
{
    if (nv >= kGranule) {
        const uint4 a = load16(p), b = load16(p + 4);
        x[0] = __uint_as_float(a.x); x[1] = __uint_as_float(a.y);
        x[2] = __uint_as_float(a.z); x[3] = __uint_as_float(a.w);
        x[4] = __uint_as_float(b.x); x[5] = __uint_as_float(b.y);
        x[6] = __uint_as_float(b.z); x[7] = __uint_as_float(b.w);
        return;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e)
        x[e] = e < nv ? gp(p)[e] : 0.0f;
}

__device__ inline void store8f(float* p, int nv, const float (&x)[8])
{
    if (nv >= kGranule) {
        store16f(p, x[0], x[1], x[2], x[3]);
        store16f(p + 4, x[4], x[5], x[6], x[7]);
        return;
    }
    for (int e = 0; e < nv; ++e)
        gp(p)[e] = x[e];
}

template <typename GT, bool WB>
__global__ __launch_bounds__(kThreads) void k_adamw32_step(WsGuard guard,
                                                           const int64_t* __restrict__ unit_prefix,
                                                           const Fp32Tensor* __restrict__ desc,
                                                           int n_tensors, int64_t n_units,
                                                           StepScalars s,
                                                           const float* __restrict__ coef_ptr,
                                                           const int32_t* __restrict__ status_ptr)
{
    constexpr int E = kFp32ElemsPerLane, G = E / kGranule, SPAN = 64 * E;
    if (!guard_ok(guard))
        return;  // the workspace does not hold this launch's descriptors
    if (status_ptr && *status_ptr != LT_STATUS_OK)
        return;  // skipped step: nothing is written
    if (!resolve_step(s))
        return;  // the step state lets no step apply
    const float coef = coef_ptr ? *coef_ptr : 1.0f;
    const int lane = threadIdx.x & 63;
    // Units go to the waves in turn, as in the 8-bit step.
    const int64_t workers = int64_t(gridDim.x) * 4;
    const int64_t me = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6);
    int k = me < n_units ? find_tensor(unit_prefix, n_tensors, me) : 0;
    for (int64_t u = me; u < n_units; u += workers) {
        while (u >= unit_prefix[k + 1])
            ++k;
        const Fp32Tensor d = desc[k];
        const int64_t e0 = (u - unit_prefix[k]) * SPAN;
        const int64_t n_span = d.numel - e0;
        float w[E], g[E], m[E], v[E];
        int nv[G];
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int64_t o = kGranule * (lane + 64 * j);
            nv[j] = int(i64min(i64max(n_span - o, 0), kGranule));
            const int64_t ei = e0 + o;
            GradWords<GT> gw;
            load_grads<true>(static_cast<const GT*>(d.g) + ei, nv[j], gw);
            float gg[8], ww[8], mm[8], vv[8];
            unpack8(gw, gg);
            load8f(d.w + ei, nv[j], ww);
            load8f(d.m + ei, nv[j], mm);
            load8f(d.v + ei, nv[j], vv);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                w[8 * j + e] = ww[e];
                g[8 * j + e] = gg[e];
                m[8 * j + e] = mm[e];
                v[8 * j + e] = vv[e];
            }
        }
        uint32_t vmin = 0xFFFFFFFFu;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float gc = g[e] * coef;
            m[e] = __builtin_fmaf(s.beta1, m[e], s.c1 * gc);
            v[e] = __builtin_fmaf(s.beta2, v[e], s.c2 * (gc * gc));
            vmin = min(vmin, __float_as_uint(v[e]) - 1u);
        }
        const bool scaled = __builtin_amdgcn_ballot_w64(vmin < 0x0F800000u - 1u) != 0;
#pragma unroll
        for (int e = 0; e < E; ++e) {
            const float root = scaled ? sqrtf(v[e]) : sqrt_rn_unscaled(v[e]);
            const float den = __builtin_fmaf(root, s.rbc2, s.eps);
            w[e] = __builtin_fmaf(-s.step_size, m[e] / den, w[e] * s.decay);
        }
#pragma unroll
        for (int j = 0; j < G; ++j) {
            const int64_t ei = e0 + kGranule * (lane + 64 * j);
            float ww[8], mm[8], vv[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                ww[e] = w[8 * j + e];
                mm[e] = m[8 * j + e];
                vv[e] = v[8 * j + e];
            }
            store8f(d.w + ei, nv[j], ww);
            store8f(d.m + ei, nv[j], mm);
            store8f(d.v + ei, nv[j], vv);
            if (WB && d.wb)
                store_bf16x8(d.wb + ei, nv[j], ww);
        }
    }
}

// -------------------------------------- f3: bf16 copy after a skipped step
//
// A skipped step (non-finite gradient) leaves the weights unchanged; tensors
// with a bf16 copy get it refreshed from them, so that after every call the
// copy is bf16(weights).  The kernel exits at once when the step was not
// skipped.  Units and their prefix are those of the step launch it follows.
template <typename Desc>
__global__ __launch_bounds__(kThreads) void k_bf16_on_skip(WsGuard guard,
                                                           const int64_t* __restrict__ unit_prefix,
                                                           const Desc* __restrict__ desc,
                                                           int n_tensors, int64_t n_units,
                                                           int64_t unit_elems,
                                                           const int32_t* __restrict__ status_ptr)
{
    if (!guard_ok(guard) || *status_ptr == LT_STATUS_OK)
        return;
    const int lane = threadIdx.x & 63;
    const int64_t waves = int64_t(gridDim.x) * 4;
    for (int64_t u = int64_t(blockIdx.x) * 4 + (threadIdx.x >> 6); u < n_units; u += waves) {
        const int k = find_tensor(unit_prefix, n_tensors, u);
        const Desc d = desc[k];
        if (!d.wb)
            continue;
        const int64_t e0 = (u - unit_prefix[k]) * unit_elems;
        const int64_t e1 = i64min(e0 + unit_elems, d.numel);
        for (int64_t ei = e0 + kGranule * lane; ei < e1; ei += 64 * kGranule) {
            const int nv = int(i64min(e1 - ei, kGranule));
            float w[8];
            load8f(d.w + ei, nv, w);
            store_bf16x8(d.wb + ei, nv, w);
        }
    }
}

template <typename Desc>
lt_err launch_bf16_on_skip(const WsGuard& guard, const int64_t* unit_prefix, const Desc* desc,
                           int n_tensors, int64_t n_units, int64_t unit_elems,
                           const int32_t* status, hipStream_t st)
{
    if (n_units == 0)
        return LT_OK;
    const int grid = int(std::min<int64_t>((n_units + 3) / 4, 1024));
    k_bf16_on_skip<Desc><<<grid, kThreads, 0, st>>>(guard, unit_prefix, desc, n_tensors, n_units,
                                                    unit_elems, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

// ================================================================ host side

template <typename GT, int B>
lt_err launch_step_b(const WsGuard& guard, const int64_t* prefix, const StepTensor* desc, int K,
                     int64_t units, const StepScalars& s, const float* coef,
                     const int32_t* status, bool wb, int map, hipStream_t stream)
{
    // One workgroup takes four units at a time when each wave works alone.
    const int64_t wg_units = (map == kMapDynamic ? StepGeom<B, true>::W : StepGeom<B, false>::W) > 1
                                 ? units
                                 : (units + 3) / 4;
    auto* kernel = map == kMapDynamic
                       ? (wb ? k_adamw8_step<GT, B, true, kMapDynamic>
                             : k_adamw8_step<GT, B, false, kMapDynamic>)
                       : (wb ? k_adamw8_step<GT, B, true, kMapLinear>
                             : k_adamw8_step<GT, B, false, kMapLinear>);
    int grid;
    if (lt_err e = grid_size(kernel, wg_units, &grid))
        return e;
    kernel<<<grid, kThreads, 0, stream>>>(guard, prefix, desc, K, units, s, coef, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

// The generic step kernel: one work unit per block.
template <typename GT, bool WB, int MAP>
lt_err launch_generic_map(const WsGuard& guard, int B, const int64_t* prefix,
                          const StepTensor* desc, int K, int64_t units, const StepScalars& s,
                          const float* coef, const int32_t* status, hipStream_t stream)
{
    const bool stash = B <= kGenericStashMax;
    const size_t lds = stash ? size_t(B) * 2 * sizeof(float) : 0;
    auto* kernel = stash ? k_adamw8_generic<GT, WB, MAP, true> : k_adamw8_generic<GT, WB, MAP, false>;
    int grid;
    if (lt_err e = grid_size(kernel, units, &grid, lds))
        return e;
    kernel<<<grid, kThreads, lds, stream>>>(guard, prefix, desc, K, units, B, s, coef, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

template <typename GT>
lt_err launch_generic(const WsGuard& guard, int B, const int64_t* prefix, const StepTensor* desc,
                      int K, int64_t units, const StepScalars& s, const float* coef,
                      const int32_t* status, bool wb, int map, hipStream_t stream)
{
    if (map == kMapDynamic)
        return wb ? launch_generic_map<GT, true, kMapDynamic>(guard, B, prefix, desc, K, units, s,
                                                               coef, status, stream)
                  : launch_generic_map<GT, false, kMapDynamic>(guard, B, prefix, desc, K, units,
                                                                s, coef, status, stream);
    return wb ? launch_generic_map<GT, true, kMapLinear>(guard, B, prefix, desc, K, units, s, coef,
                                                          status, stream)
              : launch_generic_map<GT, false, kMapLinear>(guard, B, prefix, desc, K, units, s,
                                                           coef, status, stream);
}

template <typename GT>
lt_err launch_step(const WsGuard& g, int B, const int64_t* prefix, const StepTensor* desc, int K,
                   int64_t tiles, const StepScalars& s, const float* coef, const int32_t* status,
                   bool wb, int map, hipStream_t stream)
{
    switch (B) {
    case 64: return launch_step_b<GT, 64>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 128: return launch_step_b<GT, 128>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 256: return launch_step_b<GT, 256>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 512: return launch_step_b<GT, 512>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 1024: return launch_step_b<GT, 1024>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 2048: return launch_step_b<GT, 2048>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 4096: return launch_step_b<GT, 4096>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    case 8192: return launch_step_b<GT, 8192>(g, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    default: return launch_generic<GT>(g, B, prefix, desc, K, tiles, s, coef, status, wb, map, stream);
    }
}

template <int B>
int64_t geom_unit(int map)
{
    return map == kMapDynamic ? StepGeom<B, true>::UNIT : StepGeom<B, false>::UNIT;
}

// Elements per work unit of the step kernel (StepGeom<B, map>::UNIT; one block
// for the generic kernel).
int64_t step_unit_elems(int B, int map)
{
    switch (B) {
    case 64: return geom_unit<64>(map);
    case 128: return geom_unit<128>(map);
    case 256: return geom_unit<256>(map);
    case 512: return geom_unit<512>(map);
    case 1024: return geom_unit<1024>(map);
    case 2048: return geom_unit<2048>(map);
    case 4096: return geom_unit<4096>(map);
    case 8192: return geom_unit<8192>(map);
    default: return B;
    }
}

int64_t sq_chunks_of(const int64_t* numels, int K)
{
    int64_t C = 0;
    for (int k = 0; k < K; ++k)
        C += (numels[k] + kChunk - 1) / kChunk;
    return C;
}

// A tensor list: n_tensors >= 0 sizes, each >= 0; numels may be NULL only for
// an empty list.  A tensor with no elements contributes nothing: its pointers
// are neither checked nor dereferenced.
bool valid_list(const int64_t* numels, int K)
{
    if (K < 0 || (K > 0 && !numels))
        return false;
    for (int k = 0; k < K; ++k)
        if (numels[k] < 0)
            return false;
    return true;
}

// The host lists of a call: each may be NULL only when the list is empty.
bool lists_given(int K, std::initializer_list<const void*> lists)
{
    if (K == 0)
        return true;
    for (const void* l : lists)
        if (!l)
            return false;
    return true;
}

// eps must be positive after its rounding to fp32 as well: with eps = 0 an element
// whose gradient and stored second moment are both zero divides 0 by 0.
bool valid_hyper(double lr, double beta1, double beta2, double eps, double weight_decay,
                 int64_t step)
{
    return std::isfinite(lr) && lr >= 0.0 && std::isfinite(weight_decay) && weight_decay >= 0.0 &&
           beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0 && std::isfinite(eps) &&
           eps > 0.0 && float(eps) > 0.0f && std::isfinite(float(eps)) && step >= 1;
}

constexpr int kMaxBlockSize = 65536;

bool valid_block_size(int B) { return B >= 64 && B <= kMaxBlockSize && B % 64 == 0; }

// Byte ranges a call reads or writes, for the no-overlap rule: no array the call
// writes may share a byte with any other array of the call (gradients, which are
// only read, may alias one another).
struct ByteRange {
    uintptr_t lo, hi;  // [lo, hi)
    bool written;
};

void add_range(std::vector<ByteRange>& v, const void* p, size_t bytes, bool written)
{
    if (p && bytes)
        v.push_back({reinterpret_cast<uintptr_t>(p), reinterpret_cast<uintptr_t>(p) + bytes, written});
}

// The first pair of ranges that overlap with at least one of them written, as a
// message; empty when there is none.
std::string overlap_error(std::vector<ByteRange> v)
{
    std::sort(v.begin(), v.end(), [](const ByteRange& a, const ByteRange& b) { return a.lo < b.lo; });
    // sweep: the furthest-reaching written range and any range seen so far
    uintptr_t end_any = 0, end_written = 0;
    for (const ByteRange& r : v) {
        if (r.lo < end_written || (r.written && r.lo < end_any))
            return "tensors of one call overlap in memory (at address " +
                   std::to_string(static_cast<unsigned long long>(r.lo)) + ")";
        end_any = std::max(end_any, r.hi);
        if (r.written)
            end_written = std::max(end_written, r.hi);
    }
    return std::string();
}

// The fp32 scalars of one step, each computed in fp64 and rounded once.
StepScalars make_scalars(double lr, double beta1, double beta2, double eps, double weight_decay,
                         int64_t step)
{
    StepScalars s;
    const double t = double(step);
    s.beta1 = float(beta1);
    s.beta2 = float(beta2);
    s.eps = float(eps);
    s.c1 = float(1.0 - beta1);
    s.c2 = float(1.0 - beta2);
    s.decay = float(1.0 - lr * weight_decay);
    s.step_size = float(lr / (1.0 - std::pow(beta1, t)));
    s.rbc2 = float(1.0 / std::sqrt(1.0 - std::pow(beta2, t)));
    s.state = nullptr;
    s.lr = lr;
    return s;
}

// The table entry of step t, by the same expressions as make_scalars.
lt_step_table_entry step_table_entry(double beta1, double beta2, int64_t step)
{
    const double t = double(step);
    lt_step_table_entry e;
    e.one_minus_beta1_t = 1.0 - std::pow(beta1, t);
    e.rbc2 = float(1.0 / std::sqrt(1.0 - std::pow(beta2, t)));
    e.reserved = 0.0f;
    return e;
}

static_assert(sizeof(lt_step_state) == 64 && sizeof(lt_step_table_entry) == 16,
              "step state layout");

// Takes applied, skips, max_skips and stopped from another step state.
__global__ void k_step_state_copy(lt_step_state* __restrict__ dst,
                                  const lt_step_state* __restrict__ src)
{
    if (threadIdx.x != 0)
        return;
    dst->applied = src->applied;
    dst->skips = src->skips;
    dst->max_skips = src->max_skips;
    dst->stopped = src->stopped;
}

__global__ void k_step_state_advance(lt_step_state* __restrict__ h,
                                     const int32_t* __restrict__ status)
{
    if (threadIdx.x != 0 || h->stopped != 0)
        return;
    if (*status == LT_STATUS_OK) {
        if (h->applied >= h->table_len) {
            h->stopped = 2;  // the steps found no table entry and wrote nothing
            return;
        }
        h->applied += 1;
        h->skips = 0;
    } else {
        h->skips += 1;
        if (h->max_skips > 0 && h->skips >= h->max_skips)
            h->stopped = 1;
    }
}

lt_err launch_sq_chunks(const WsGuard& guard, int gdt, const int64_t* prefix, const uint64_t* ptrs,
                        const int64_t* numels, int K, int64_t C, double* partials, hipStream_t st)
{
    if (C == 0)
        return LT_OK;  // no chunks: every tensor of the list is empty
    const int64_t iters = (C + kSqChunksPerIter - 1) / kSqChunksPerIter;
    int grid;
    if (gdt == LT_DTYPE_BF16) {
        if (lt_err e = grid_size(k_sqnorm_chunks<uint16_t>, iters, &grid))
            return e;
        k_sqnorm_chunks<uint16_t><<<grid, kThreads, 0, st>>>(guard, prefix, ptrs, numels, K, C,
                                                             partials);
    } else {
        if (lt_err e = grid_size(k_sqnorm_chunks<float>, iters, &grid))
            return e;
        k_sqnorm_chunks<float><<<grid, kThreads, 0, st>>>(guard, prefix, ptrs, numels, K, C,
                                                          partials);
    }
    LT_HIP(hipGetLastError());
    return LT_OK;
}

// ---------------------------------------------------- a11: layer streaming
//
// Weights, gradients and 8-bit states stay in (pinned) host memory; layers pass
// through a ring of device slots.  Pass 1 copies each layer's gradients in and
// writes its chunk sums at their global indices, so S is bitwise the resident
// sum; the finish, total and clip run once.  Pass 2 copies each layer in, runs
// the fused step on it and copies weights, codes and scales back.  Copies in,
// kernels and copies out run on three streams ordered by per-slot events.

constexpr int kMaxSlots = 16;

struct StreamEvents {
    hipEvent_t in[kMaxSlots], computed[kMaxSlots], freed[kMaxSlots], done;
    bool ready = false;
};

StreamEvents g_stream_events[kMaxDevices];
std::mutex g_stream_mu[kMaxDevices];

size_t align256(size_t x) { return round_up(x, 256); }

// Bytes of one tensor's arrays inside a slot: w, g, m codes, v codes, m and v absmax.
struct SlotTensor {
    size_t w, g, mq, vq, ma, va, wb, end;
};

// Offsets of one tensor's arrays inside a slot; the bf16 weight copy takes room
// only when the call asks for it.
SlotTensor slot_tensor(size_t at, int64_t n, int gbytes, int B, bool bf16_copy)
{
    const int64_t nb = (n + B - 1) / B;
    SlotTensor t;
    t.w = at;
    t.g = t.w + align256(size_t(n) * 4);
    t.mq = t.g + align256(size_t(n) * gbytes);
    t.vq = t.mq + align256(size_t(n));
    t.ma = t.vq + align256(size_t(n));
    t.va = t.ma + align256(size_t(nb) * 4);
    t.wb = t.va + align256(size_t(nb) * 4);
    t.end = t.wb + (bf16_copy ? align256(size_t(n) * 2) : 0);
    return t;
}

struct StreamLayout {
    size_t header = 0;                  // uploaded descriptors
    size_t gprefix = 0;                 // global chunk prefix, K + 1
    std::vector<size_t> sq_prefix, sq_ptrs, sq_numels, st_prefix, st_desc;  // per layer
    size_t partials = 0, sk = 0, slots = 0, slot_bytes = 0, total = 0;
    size_t resident = 0;        // resident gradients (keep_grads), after the slots
    std::vector<size_t> roff;   // per tensor, from `resident`
    int64_t C = 0;
};

// With keep_grads every gradient gets its own region after the slots, and the
// slots hold no gradient.
StreamLayout stream_layout(const int64_t* numels, int K, const int* first, int L, int gbytes, int B,
                           int S, bool bf16_copy, bool keep_grads)
{
    StreamLayout l;
    size_t at = kTagBytes;
    l.gprefix = at;
    at = round_up(at + sizeof(int64_t) * (K + 1), 64);
    for (int i = 0; i < L; ++i) {
        const int Ki = first[i + 1] - first[i];
        l.sq_prefix.push_back(at);
        at = round_up(at + sizeof(int64_t) * (Ki + 1), 64);
        l.sq_ptrs.push_back(at);
        at = round_up(at + sizeof(uint64_t) * Ki, 64);
        l.sq_numels.push_back(at);
        at = round_up(at + sizeof(int64_t) * Ki, 64);
        l.st_prefix.push_back(at);
        at = round_up(at + sizeof(int64_t) * (Ki + 1), 64);
        l.st_desc.push_back(at);
        at = round_up(at + sizeof(StepTensor) * Ki, 64);
    }
    l.header = round_up(at, 256);
    l.C = sq_chunks_of(numels, K);
    l.partials = l.header;
    l.sk = l.partials + align256(sizeof(double) * l.C);
    l.slots = l.sk + align256(sizeof(double) * K);
    size_t biggest = 0;
    for (int i = 0; i < L; ++i) {
        size_t b = 0;
        for (int k = first[i]; k < first[i + 1]; ++k)
            b = slot_tensor(b, numels[k], keep_grads ? 0 : gbytes, B, bf16_copy).end;
        biggest = std::max(biggest, b);
    }
    l.slot_bytes = biggest;
    l.resident = l.slots + l.slot_bytes * size_t(S);
    size_t r = 0;
    for (int k = 0; keep_grads && k < K; ++k) {
        l.roff.push_back(r);
        r += align256(size_t(numels[k]) * gbytes);
    }
    l.total = l.resident + r;
    return l;
}

bool valid_layers(const int* first, int L, int K)
{
    if (!first || L < 1 || first[0] != 0 || first[L] != K)
        return false;
    for (int i = 0; i < L; ++i)
        if (first[i + 1] <= first[i])
            return false;
    return true;
}

// ------------------------------------- the sum of squares without allocation
//
// lt_grad_sqnorm_noalloc keeps what lt_grad_sqnorm keeps in its workspace (the
// descriptors, one fp64 partial per chunk, S_k) in `scratch`, a device array of
// this file that every device the library runs on holds until the process ends.
// Its descriptors are written by k_put_words from kernel arguments, so the call
// needs no staging buffer and no copy from the host, and allocates nothing.  In
// host code `scratch` names a host-side stand-in: the device address comes from
// hipGetSymbolAddress, once per device, and only that address is used.
constexpr size_t kScratchBytes = size_t(16) << 20;  // 16 MiB per device
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

struct ScratchAddress {
    uint8_t* ptr = nullptr;  // this device's copy of `scratch`
    bool ready = false;
};
ScratchAddress g_scratch[kMaxDevices];

// The device address of `scratch` on the current device (looked up on the first
// call on that device, with it current).
lt_err scratch_address(uint8_t** out)
{
    int dev;
    if (lt_err e = current_device(&dev))
        return e;
    std::lock_guard<std::mutex> lock(g_dev[dev].mu);
    ScratchAddress& a = g_scratch[dev];
    if (!a.ready) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(LT_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") +
                                        hipGetErrorString(e));
        a.ptr = static_cast<uint8_t*>(p);
        a.ready = true;
    }
    *out = a.ptr;
    return LT_OK;
}

// One launch writes up to kPutWords consecutive 8-byte words at base + offset.
constexpr int kPutWords = 440;  // 3.5 KB of kernel arguments
struct PutWords {
    uint64_t offset;  // bytes, a multiple of 8
    uint32_t n;
    uint32_t pad;
    uint64_t w[kPutWords];
};

__global__ __launch_bounds__(256) void k_put_words(uint8_t* __restrict__ base, PutWords a)
{
    auto* dst = reinterpret_cast<uint64_t*>(base + a.offset);
    for (uint32_t i = threadIdx.x; i < a.n; i += blockDim.x)
        dst[i] = a.w[i];
}

// Collects runs of consecutive words and launches k_put_words for each full or
// finished run.
struct WordWriter {
    uint8_t* base;
    hipStream_t st;
    PutWords a;
    lt_err put(size_t offset, uint64_t word)
    {
        if (a.n > 0 && (a.n == kPutWords || offset != a.offset + 8 * size_t(a.n)))
            if (lt_err e = flush())
                return e;
        if (a.n == 0)
            a.offset = offset;
        a.w[a.n++] = word;
        return LT_OK;
    }
    lt_err flush()
    {
        if (a.n == 0)
            return LT_OK;
        k_put_words<<<1, 256, 0, st>>>(base, a);
        LT_HIP(hipGetLastError());
        a.n = 0;
        return LT_OK;
    }
};

}  // namespace

// =================================================================== C ABI

extern "C" {

size_t lt_grad_sqnorm_workspace_bytes(const int64_t* numels, int n_tensors)
{
    if (!valid_list(numels, n_tensors))
        return 0;
    return sq_layout(n_tensors, sq_chunks_of(numels, n_tensors)).total;
}

lt_err lt_grad_sqnorm(const void* const* grads, const int64_t* numels, int n_tensors,
                      int grad_dtype, void* workspace, size_t workspace_bytes,
                      double* sq_per_tensor, double* sq_total, int32_t* status, void* stream)
{
    g_last_error.clear();
    if (!valid_list(numels, n_tensors) || !lists_given(n_tensors, {grads}))
        return fail(LT_ERR_INVALID_ARG, "grads/numels must hold n_tensors >= 0 entries with numel >= 0");
    if (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16)
        return fail(LT_ERR_INVALID_ARG, "grad_dtype must be LT_DTYPE_F32 or LT_DTYPE_BF16");
    if (!sq_total || !status)
        return fail(LT_ERR_INVALID_ARG, "sq_total and status must not be NULL");
    if (!aligned(sq_total, 8) || !aligned(status, 4) || (sq_per_tensor && !aligned(sq_per_tensor, 8)))
        return fail(LT_ERR_ALIGNMENT, "scalar outputs must be naturally aligned");
    for (int k = 0; k < n_tensors; ++k) {
        if (numels[k] == 0)
            continue;
        if (!grads[k])
            return fail(LT_ERR_INVALID_ARG, "grads[" + std::to_string(k) + "] is NULL");
        if (!aligned(grads[k], 16))
            return fail(LT_ERR_ALIGNMENT, "grads[" + std::to_string(k) + "] is not 16-byte aligned");
    }
    const int K = n_tensors;
    const int64_t C = sq_chunks_of(numels, K);
    const SqLayout lay = sq_layout(K, C);
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < lay.total)
        return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned and hold " +
                                          std::to_string(lay.total) + " bytes");

    std::vector<uint8_t> header(lay.header_bytes, 0);
    auto* prefix = reinterpret_cast<int64_t*>(header.data() + lay.prefix);
    auto* ptrs = reinterpret_cast<uint64_t*>(header.data() + lay.ptrs);
    auto* ns = reinterpret_cast<int64_t*>(header.data() + lay.numels);
    prefix[0] = 0;
    for (int k = 0; k < K; ++k) {
        prefix[k + 1] = prefix[k] + (numels[k] + kChunk - 1) / kChunk;
        ptrs[k] = reinterpret_cast<uint64_t>(grads[k]);
        ns[k] = numels[k];
    }
    auto* ws = static_cast<uint8_t*>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    WsGuard guard;
    if (lt_err e = put_descriptors(header, ws, st, &guard))
        return e;
    const auto* d_prefix = reinterpret_cast<const int64_t*>(ws + lay.prefix);
    const auto* d_ptrs = reinterpret_cast<const uint64_t*>(ws + lay.ptrs);
    const auto* d_numels = reinterpret_cast<const int64_t*>(ws + lay.numels);
    auto* d_partials = reinterpret_cast<double*>(ws + lay.partials);
    auto* d_sk = reinterpret_cast<double*>(ws + lay.sk);

    if (lt_err e = launch_sq_chunks(guard, grad_dtype, d_prefix, d_ptrs, d_numels, K, C,
                                    d_partials, st))
        return e;
    if (K > 0) {
        k_sqnorm_finish<<<K, kThreads, 0, st>>>(guard, d_prefix, d_partials, d_sk);
        LT_HIP(hipGetLastError());
    }
    k_sqnorm_total<<<1, 256, 0, st>>>(guard, d_sk, K, sq_per_tensor, sq_total, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

lt_err lt_clip_coef(const double* sq_total, float max_norm, float* total_norm, float* coef,
                    int32_t* status, void* stream)
{
    g_last_error.clear();
    if (!sq_total || !coef)
        return fail(LT_ERR_INVALID_ARG, "sq_total and coef must not be NULL");
    if (!(max_norm > 0.0f))
        return fail(LT_ERR_INVALID_ARG, "max_norm must be > 0 (+inf disables clipping)");
    if (!aligned(sq_total, 8) || !aligned(coef, 4) || (total_norm && !aligned(total_norm, 4)) ||
        (status && !aligned(status, 4)))
        return fail(LT_ERR_ALIGNMENT, "scalar arguments must be naturally aligned");
    k_clip_coef<<<1, 64, 0, static_cast<hipStream_t>(stream)>>>(sq_total, max_norm, total_norm,
                                                                 coef, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

lt_err lt_grad_sqnorm_noalloc(const void* const* grads, const int64_t* numels, int n_tensors,
                              int grad_dtype, double* sq_per_tensor, double* sq_total,
                              int32_t* status, void* stream)
{
    g_last_error.clear();
    if (!valid_list(numels, n_tensors) || !lists_given(n_tensors, {grads}))
        return fail(LT_ERR_INVALID_ARG, "grads/numels must hold n_tensors >= 0 entries with numel >= 0");
    if (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16)
        return fail(LT_ERR_INVALID_ARG, "grad_dtype must be LT_DTYPE_F32 or LT_DTYPE_BF16");
    if (!sq_total || !status)
        return fail(LT_ERR_INVALID_ARG, "sq_total and status must not be NULL");
    if (!aligned(sq_total, 8) || !aligned(status, 4) || (sq_per_tensor && !aligned(sq_per_tensor, 8)))
        return fail(LT_ERR_ALIGNMENT, "scalar outputs must be naturally aligned");
    for (int k = 0; k < n_tensors; ++k) {
        if (numels[k] == 0)
            continue;
        if (!grads[k])
            return fail(LT_ERR_INVALID_ARG, "grads[" + std::to_string(k) + "] is NULL");
        if (!aligned(grads[k], 16))
            return fail(LT_ERR_ALIGNMENT, "grads[" + std::to_string(k) + "] is not 16-byte aligned");
    }
    const int K = n_tensors;
    const int64_t C = sq_chunks_of(numels, K);
    const SqLayout lay = sq_layout(K, C);
    if (lay.total > kScratchBytes)
        return fail(LT_ERR_INVALID_ARG,
                    "the list needs " + std::to_string(lay.total) + " bytes of scratch; the "
                    "no-allocation sum of squares holds " + std::to_string(kScratchBytes) +
                    " (about 2 million 8192-element chunks); use lt_grad_sqnorm");
    uint8_t* ws;
    if (lt_err e = scratch_address(&ws))
        return e;
    hipStream_t st = static_cast<hipStream_t>(stream);

    // The descriptors, as lt_grad_sqnorm lays them out, written by kernels.
    const WsGuard guard{reinterpret_cast<const uint64_t*>(ws), fresh_tag()};
    WordWriter out{ws, st, {}};
    if (lt_err e = out.put(0, guard.tag))
        return e;
    int64_t prefix = 0;
    for (int k = 0; k <= K; ++k) {
        if (lt_err e = out.put(lay.prefix + 8 * size_t(k), uint64_t(prefix)))
            return e;
        if (k < K)
            prefix += (numels[k] + kChunk - 1) / kChunk;
    }
    for (int k = 0; k < K; ++k)
        if (lt_err e = out.put(lay.ptrs + 8 * size_t(k), reinterpret_cast<uint64_t>(grads[k])))
            return e;
    for (int k = 0; k < K; ++k)
        if (lt_err e = out.put(lay.numels + 8 * size_t(k), uint64_t(numels[k])))
            return e;
    if (lt_err e = out.flush())
        return e;

    const auto* d_prefix = reinterpret_cast<const int64_t*>(ws + lay.prefix);
    auto* d_partials = reinterpret_cast<double*>(ws + lay.partials);
    auto* d_sk = reinterpret_cast<double*>(ws + lay.sk);
    if (lt_err e = launch_sq_chunks(guard, grad_dtype, d_prefix,
                                    reinterpret_cast<const uint64_t*>(ws + lay.ptrs),
                                    reinterpret_cast<const int64_t*>(ws + lay.numels), K, C,
                                    d_partials, st))
        return e;
    if (K > 0) {
        k_sqnorm_finish<<<K, kThreads, 0, st>>>(guard, d_prefix, d_partials, d_sk);
        LT_HIP(hipGetLastError());
    }
    k_sqnorm_total<<<1, 256, 0, st>>>(guard, d_sk, K, sq_per_tensor, sq_total, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

int64_t lt_grad_chunk_count(const int64_t* numels, int n_tensors)
{
    return valid_list(numels, n_tensors) ? sq_chunks_of(numels, n_tensors) : 0;
}

size_t lt_grad_sqnorm_partials_workspace_bytes(int n_tensors)
{
    return n_tensors < 0 ? 0 : round_up(sq_layout(n_tensors, 0).header_bytes, 256);
}

lt_err lt_grad_sqnorm_partials(const void* const* grads, const int64_t* numels, int n_tensors,
                               int grad_dtype, double* partials, void* workspace,
                               size_t workspace_bytes, void* stream)
{
    g_last_error.clear();
    if (!valid_list(numels, n_tensors) || !lists_given(n_tensors, {grads}))
        return fail(LT_ERR_INVALID_ARG, "grads/numels must hold n_tensors >= 0 entries with numel >= 0");
    if (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16)
        return fail(LT_ERR_INVALID_ARG, "grad_dtype must be LT_DTYPE_F32 or LT_DTYPE_BF16");
    const int64_t n_chunks = sq_chunks_of(numels, n_tensors);
    if (n_chunks == 0)
        return LT_OK;  // nothing to sum: partials is not touched
    if (!partials)
        return fail(LT_ERR_INVALID_ARG, "partials must not be NULL");
    if (!aligned(partials, 8))
        return fail(LT_ERR_ALIGNMENT, "partials must be 8-byte aligned");
    for (int k = 0; k < n_tensors; ++k) {
        if (numels[k] == 0)
            continue;
        if (!grads[k])
            return fail(LT_ERR_INVALID_ARG, "grads[" + std::to_string(k) + "] is NULL");
        if (!aligned(grads[k], 16))
            return fail(LT_ERR_ALIGNMENT, "grads[" + std::to_string(k) + "] is not 16-byte aligned");
    }
    const int K = n_tensors;
    const SqLayout lay = sq_layout(K, 0);
    const size_t need = lt_grad_sqnorm_partials_workspace_bytes(K);
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < need)
        return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned and hold " +
                                          std::to_string(need) + " bytes");
    std::vector<uint8_t> header(lay.header_bytes, 0);
    auto* prefix = reinterpret_cast<int64_t*>(header.data() + lay.prefix);
    auto* ptrs = reinterpret_cast<uint64_t*>(header.data() + lay.ptrs);
    auto* ns = reinterpret_cast<int64_t*>(header.data() + lay.numels);
    prefix[0] = 0;
    for (int k = 0; k < K; ++k) {
        prefix[k + 1] = prefix[k] + (numels[k] + kChunk - 1) / kChunk;
        ptrs[k] = reinterpret_cast<uint64_t>(grads[k]);
        ns[k] = numels[k];
    }
    auto* ws = static_cast<uint8_t*>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    WsGuard guard;
    if (lt_err e = put_descriptors(header, ws, st, &guard))
        return e;
    return launch_sq_chunks(guard, grad_dtype, reinterpret_cast<const int64_t*>(ws + lay.prefix),
                            reinterpret_cast<const uint64_t*>(ws + lay.ptrs),
                            reinterpret_cast<const int64_t*>(ws + lay.numels), K, prefix[K],
                            partials, st);
}

// Finish workspace: [tag][chunk prefix K+1] | [S_k K]
size_t lt_grad_sqnorm_finish_workspace_bytes(int n_tensors)
{
    return n_tensors < 0 ? 0
                         : round_up(kTagBytes + sizeof(int64_t) * (n_tensors + 1), 256) +
                               round_up(sizeof(double) * n_tensors, 256);
}

lt_err lt_grad_sqnorm_finish(const int64_t* numels, int n_tensors, const double* partials,
                             void* workspace, size_t workspace_bytes, double* sq_per_tensor,
                             double* sq_total, int32_t* status, void* stream)
{
    g_last_error.clear();
    if (!valid_list(numels, n_tensors))
        return fail(LT_ERR_INVALID_ARG, "numels must hold n_tensors >= 0 entries >= 0");
    const bool no_chunks = sq_chunks_of(numels, n_tensors) == 0;  // partials is then not read
    if ((!partials && !no_chunks) || !sq_total || !status)
        return fail(LT_ERR_INVALID_ARG, "partials, sq_total and status must not be NULL");
    if (!aligned(partials, 8) || !aligned(sq_total, 8) || !aligned(status, 4) ||
        (sq_per_tensor && !aligned(sq_per_tensor, 8)))
        return fail(LT_ERR_ALIGNMENT, "partials and scalar outputs must be naturally aligned");
    const int K = n_tensors;
    const size_t need = lt_grad_sqnorm_finish_workspace_bytes(K);
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < need)
        return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned and hold " +
                                          std::to_string(need) + " bytes");
    std::vector<uint8_t> image(kTagBytes + sizeof(int64_t) * (K + 1), 0);
    auto* prefix = reinterpret_cast<int64_t*>(image.data() + kTagBytes);
    for (int k = 0; k < K; ++k)
        prefix[k + 1] = prefix[k] + (numels[k] + kChunk - 1) / kChunk;
    auto* ws = static_cast<uint8_t*>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    WsGuard guard;
    if (lt_err e = put_descriptors(image, ws, st, &guard))
        return e;
    auto* d_sk = reinterpret_cast<double*>(ws + round_up(kTagBytes + sizeof(int64_t) * (K + 1), 256));
    if (K > 0) {
        k_sqnorm_finish<<<K, kThreads, 0, st>>>(guard, reinterpret_cast<const int64_t*>(ws + kTagBytes),
                                                partials, d_sk);
        LT_HIP(hipGetLastError());
    }
    k_sqnorm_total<<<1, 256, 0, st>>>(guard, d_sk, K, sq_per_tensor, sq_total, status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

size_t lt_step_workspace_bytes(int n_tensors)
{
    return n_tensors < 0 ? 0 : step_layout(n_tensors).total;
}

lt_err lt_hybrid8bit_adamw_step(float* const* params, const void* const* grads, int grad_dtype,
                                int8_t* const* m_codes, float* const* m_absmax,
                                uint8_t* const* v_codes, float* const* v_absmax,
                                uint16_t* const* params_bf16, const int64_t* numels,
                                int n_tensors, int block_size, int code_map, double lr,
                                double beta1, double beta2, double eps, double weight_decay,
                                int64_t step, const float* coef, const int32_t* status,
                                const void* step_state, void* workspace, size_t workspace_bytes,
                                void* stream)
{
    g_last_error.clear();
    if (!valid_list(numels, n_tensors) ||
        !lists_given(n_tensors, {params, grads, m_codes, m_absmax, v_codes, v_absmax}))
        return fail(LT_ERR_INVALID_ARG, "tensor lists must hold n_tensors >= 0 entries with numel >= 0");
    if (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16)
        return fail(LT_ERR_INVALID_ARG, "grad_dtype must be LT_DTYPE_F32 or LT_DTYPE_BF16");
    if (!valid_block_size(block_size))
        return fail(LT_ERR_INVALID_ARG, "block_size must be a multiple of 64 in [64, 65536]");
    if (code_map != LT_MAP_LINEAR && code_map != LT_MAP_DYNAMIC)
        return fail(LT_ERR_INVALID_ARG, "code_map must be LT_MAP_LINEAR or LT_MAP_DYNAMIC");
    if (!valid_hyper(lr, beta1, beta2, eps, weight_decay, step_state ? 1 : step))
        return fail(LT_ERR_INVALID_ARG, "need finite lr, weight_decay >= 0, finite eps > 0 (also "
                                        "in fp32), 0 <= beta1, beta2 < 1 and step >= 1");
    if ((coef && !aligned(coef, 4)) || (status && !aligned(status, 4)) ||
        (step_state && !aligned(step_state, 16)))
        return fail(LT_ERR_ALIGNMENT, "coef and status must be 4-byte aligned, step_state 16-byte");
    const int K = n_tensors;
    for (int k = 0; k < K; ++k) {
        if (numels[k] == 0)
            continue;
        const std::string at = "[" + std::to_string(k) + "]";
        if (!params[k] || !grads[k] || !m_codes[k] || !m_absmax[k] || !v_codes[k] || !v_absmax[k])
            return fail(LT_ERR_INVALID_ARG, "NULL tensor pointer at index " + at);
        if (!aligned(params[k], 16) || !aligned(grads[k], 16) || !aligned(m_codes[k], 16) ||
            !aligned(v_codes[k], 16))
            return fail(LT_ERR_ALIGNMENT, "params/grads/codes" + at + " must be 16-byte aligned");
        if (!aligned(m_absmax[k], 4) || !aligned(v_absmax[k], 4))
            return fail(LT_ERR_ALIGNMENT, "absmax" + at + " must be 4-byte aligned");
        if (params_bf16 && !aligned(params_bf16[k], 16))
            return fail(LT_ERR_ALIGNMENT, "params_bf16" + at + " must be 16-byte aligned");
    }
    {
        std::vector<ByteRange> r;
        r.reserve(size_t(K) * 7);
        const size_t gbytes = grad_dtype == LT_DTYPE_BF16 ? 2 : 4;
        for (int k = 0; k < K; ++k) {
            const size_t n = size_t(numels[k]), nb = size_t((numels[k] + block_size - 1) / block_size);
            add_range(r, params[k], n * 4, true);
            add_range(r, grads[k], n * gbytes, false);
            add_range(r, m_codes[k], n, true);
            add_range(r, v_codes[k], n, true);
            add_range(r, m_absmax[k], nb * 4, true);
            add_range(r, v_absmax[k], nb * 4, true);
            if (params_bf16)
                add_range(r, params_bf16[k], n * 2, true);
        }
        const std::string e = overlap_error(std::move(r));
        if (!e.empty())
            return fail(LT_ERR_INVALID_ARG, e);
    }
    const StepLayout lay = step_layout(K);
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < lay.total)
        return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned and hold " +
                                          std::to_string(lay.total) + " bytes");

    const int64_t tile = step_unit_elems(block_size, code_map);
    std::vector<uint8_t> host(lay.total, 0);
    auto* prefix = reinterpret_cast<int64_t*>(host.data() + lay.prefix);
    auto* desc = reinterpret_cast<StepTensor*>(host.data() + lay.desc);
    prefix[0] = 0;
    for (int k = 0; k < K; ++k) {
        prefix[k + 1] = prefix[k] + (numels[k] + tile - 1) / tile;
        desc[k] = StepTensor{params[k], grads[k], m_codes[k], m_absmax[k], v_codes[k], v_absmax[k],
                             numels[k], params_bf16 ? params_bf16[k] : nullptr};
    }
    const int64_t tiles = prefix[K];
    if (tiles == 0)
        return LT_OK;  // every tensor is empty

    StepScalars s = make_scalars(lr, beta1, beta2, eps, weight_decay, step_state ? 1 : step);
    s.state = static_cast<const uint8_t*>(step_state);

    auto* ws = static_cast<uint8_t*>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    WsGuard guard;
    if (lt_err e = put_descriptors(host, ws, st, &guard))
        return e;
    const auto* d_prefix = reinterpret_cast<const int64_t*>(ws + lay.prefix);
    const auto* d_desc = reinterpret_cast<const StepTensor*>(ws + lay.desc);
    const bool wb = any_set(params_bf16, K);
    if (lt_err e = grad_dtype == LT_DTYPE_BF16
                       ? launch_step<uint16_t>(guard, block_size, d_prefix, d_desc, K, tiles, s,
                                               coef, status, wb, code_map, st)
                       : launch_step<float>(guard, block_size, d_prefix, d_desc, K, tiles, s,
                                            coef, status, wb, code_map, st))
        return e;
    if (status && wb)
        return launch_bf16_on_skip(guard, d_prefix, d_desc, K, tiles, tile, status, st);
    return LT_OK;
}

size_t lt_streamed_workspace_bytes(const int64_t* numels, int n_tensors, const int* layer_first,
                                   int n_layers, int grad_dtype, int block_size, int ring_slots,
                                   int bf16_copy, int keep_grads)
{
    if (!valid_list(numels, n_tensors) || !valid_layers(layer_first, n_layers, n_tensors) ||
        (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16) ||
        !valid_block_size(block_size) || ring_slots < 2 || ring_slots > kMaxSlots)
        return 0;
    return stream_layout(numels, n_tensors, layer_first, n_layers,
                         grad_dtype == LT_DTYPE_BF16 ? 2 : 4, block_size, ring_slots,
                         bf16_copy != 0, keep_grads != 0)
        .total;
}

lt_err lt_streamed_hybrid8bit_adamw_step(float* const* params, const void* const* grads,
                                         int grad_dtype, int8_t* const* m_codes,
                                         float* const* m_absmax, uint8_t* const* v_codes,
                                         float* const* v_absmax, uint16_t* const* params_bf16,
                                         const int64_t* numels,
                                         int n_tensors, const int* layer_first, int n_layers,
                                         int block_size, int code_map, double lr, double beta1,
                                         double beta2,
                                         double eps, double weight_decay, int64_t step,
                                         float max_norm, int norm_ready, int keep_grads,
                                         int ring_slots, void* workspace,
                                         size_t workspace_bytes, double* sq_total,
                                         float* total_norm, float* coef, int32_t* status,
                                         void* const* layer_events, void* compute_stream,
                                         void* h2d_stream, void* d2h_stream)
{
    g_last_error.clear();
    const int K = n_tensors, L = n_layers, S = ring_slots, B = block_size;
    if (K < 1 || !valid_list(numels, K) ||
        !lists_given(K, {params, grads, m_codes, m_absmax, v_codes, v_absmax}))
        return fail(LT_ERR_INVALID_ARG, "tensor lists must hold n_tensors >= 1 entries with numel >= 0");
    if (!valid_layers(layer_first, L, K))
        return fail(LT_ERR_INVALID_ARG,
                    "layer_first must rise strictly from 0 to n_tensors over n_layers + 1 entries");
    if (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16)
        return fail(LT_ERR_INVALID_ARG, "grad_dtype must be LT_DTYPE_F32 or LT_DTYPE_BF16");
    if (!valid_block_size(B))
        return fail(LT_ERR_INVALID_ARG, "block_size must be a multiple of 64 in [64, 65536]");
    if (code_map != LT_MAP_LINEAR && code_map != LT_MAP_DYNAMIC)
        return fail(LT_ERR_INVALID_ARG, "code_map must be LT_MAP_LINEAR or LT_MAP_DYNAMIC");
    if (!valid_hyper(lr, beta1, beta2, eps, weight_decay, step) || !(max_norm > 0.0f))
        return fail(LT_ERR_INVALID_ARG, "need finite lr, weight_decay >= 0, finite eps > 0 (also "
                                        "in fp32), 0 <= beta1, beta2 < 1, step >= 1 and "
                                        "max_norm > 0");
    if (S < 2 || S > kMaxSlots)
        return fail(LT_ERR_INVALID_ARG, "ring_slots must be in [2, 16]");
    if (!sq_total || !coef || !status)
        return fail(LT_ERR_INVALID_ARG, "sq_total, coef and status must not be NULL");
    if (!aligned(sq_total, 8) || !aligned(coef, 4) || !aligned(status, 4) ||
        (total_norm && !aligned(total_norm, 4)))
        return fail(LT_ERR_ALIGNMENT, "scalar outputs must be naturally aligned");
    for (int k = 0; k < K; ++k)
        if (numels[k] > 0 &&
            (!params[k] || !grads[k] || !m_codes[k] || !m_absmax[k] || !v_codes[k] || !v_absmax[k]))
            return fail(LT_ERR_INVALID_ARG, "NULL host pointer at index " + std::to_string(k));
    const int gbytes = grad_dtype == LT_DTYPE_BF16 ? 2 : 4;
    const bool bf16_copy = params_bf16 != nullptr;
    const bool resident = keep_grads != 0;
    const StreamLayout lay =
        stream_layout(numels, K, layer_first, L, gbytes, B, S, bf16_copy, resident);
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < lay.total)
        return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned and hold " +
                                          std::to_string(lay.total) + " bytes");

    auto* ws = static_cast<uint8_t*>(workspace);
    auto slot_base = [&](int layer) { return ws + lay.slots + lay.slot_bytes * size_t(layer % S); };
    // Where tensor k's gradient sits on the device: its resident region, or the
    // layer's slot (place = the tensor's offsets in that slot).
    auto grad_at = [&](int k, uint8_t* base, const SlotTensor& place) {
        return resident ? ws + lay.resident + lay.roff[k] : base + place.g;
    };
    const int64_t unit = step_unit_elems(B, code_map);

    // Descriptors of every layer, each pointing into the slot the layer will use.
    std::vector<uint8_t> header(lay.header, 0);
    auto* gprefix = reinterpret_cast<int64_t*>(header.data() + lay.gprefix);
    gprefix[0] = 0;
    for (int k = 0; k < K; ++k)
        gprefix[k + 1] = gprefix[k] + (numels[k] + kChunk - 1) / kChunk;
    std::vector<std::vector<SlotTensor>> places(L);
    for (int i = 0; i < L; ++i) {
        auto* sp = reinterpret_cast<int64_t*>(header.data() + lay.sq_prefix[i]);
        auto* pp = reinterpret_cast<uint64_t*>(header.data() + lay.sq_ptrs[i]);
        auto* np = reinterpret_cast<int64_t*>(header.data() + lay.sq_numels[i]);
        auto* up = reinterpret_cast<int64_t*>(header.data() + lay.st_prefix[i]);
        auto* dp = reinterpret_cast<StepTensor*>(header.data() + lay.st_desc[i]);
        uint8_t* base = slot_base(i);
        size_t at = 0;
        sp[0] = 0;
        up[0] = 0;
        for (int k = layer_first[i], j = 0; k < layer_first[i + 1]; ++k, ++j) {
            const SlotTensor t = slot_tensor(at, numels[k], resident ? 0 : gbytes, B, bf16_copy);
            places[i].push_back(t);
            at = t.end;
            sp[j + 1] = sp[j] + (numels[k] + kChunk - 1) / kChunk;
            pp[j] = reinterpret_cast<uint64_t>(grad_at(k, base, t));
            np[j] = numels[k];
            up[j + 1] = up[j] + (numels[k] + unit - 1) / unit;
            dp[j] = StepTensor{reinterpret_cast<float*>(base + t.w), grad_at(k, base, t),
                               reinterpret_cast<int8_t*>(base + t.mq),
                               reinterpret_cast<float*>(base + t.ma),
                               reinterpret_cast<uint8_t*>(base + t.vq),
                               reinterpret_cast<float*>(base + t.va), numels[k],
                               bf16_copy && params_bf16[k]
                                   ? reinterpret_cast<uint16_t*>(base + t.wb)
                                   : nullptr};
        }
    }

    int dev;
    if (lt_err e = current_device(&dev))
        return e;
    std::lock_guard<std::mutex> lock(g_stream_mu[dev]);  // one streamed call per device at a time
    StreamEvents& ev = g_stream_events[dev];
    if (!ev.ready) {
        for (int i = 0; i < kMaxSlots; ++i) {
            LT_HIP(hipEventCreateWithFlags(&ev.in[i], hipEventDisableTiming));
            LT_HIP(hipEventCreateWithFlags(&ev.computed[i], hipEventDisableTiming));
            LT_HIP(hipEventCreateWithFlags(&ev.freed[i], hipEventDisableTiming));
        }
        LT_HIP(hipEventCreateWithFlags(&ev.done, hipEventDisableTiming));
        ev.ready = true;
    }
    hipStream_t cs = static_cast<hipStream_t>(compute_stream);
    hipStream_t hs = static_cast<hipStream_t>(h2d_stream);
    hipStream_t ds = static_cast<hipStream_t>(d2h_stream);
    WsGuard guard;
    if (lt_err e = put_descriptors(header, ws, cs, &guard))
        return e;
    // Copies into a slot may start once the work that last used it is done.
    bool used[kMaxSlots] = {};
    LT_HIP(hipEventRecord(ev.done, cs));  // the descriptors are in place
    LT_HIP(hipStreamWaitEvent(hs, ev.done, 0));
    auto* d_partials = reinterpret_cast<double*>(ws + lay.partials);
    auto* d_sk = reinterpret_cast<double*>(ws + lay.sk);
    const auto H2D = hipMemcpyHostToDevice, D2H = hipMemcpyDeviceToHost;

    // The caller's events, when given: mark(i, m, stream) records event m of layer i.
    auto mark = [&](int i, int m, hipStream_t s) -> lt_err {
        if (layer_events && layer_events[8 * size_t(i) + m])
            LT_HIP(hipEventRecord(static_cast<hipEvent_t>(layer_events[8 * size_t(i) + m]), s));
        return LT_OK;
    };

    // Pass 1: gradients in, chunk sums at their global indices.  Skipped when the
    // caller summed the gradients as they arrived (sq_total and status are given).
    // Resident gradients each have their own region, so their copies wait for no
    // slot and pass 2 does not copy them again.
    for (int i = 0; i < (norm_ready ? 0 : L); ++i) {
        const int sl = i % S;
        if (used[sl] && !resident)
            LT_HIP(hipStreamWaitEvent(hs, ev.freed[sl], 0));
        uint8_t* base = slot_base(i);
        if (lt_err e = mark(i, 0, hs))
            return e;
        for (int k = layer_first[i], j = 0; k < layer_first[i + 1]; ++k, ++j)
            if (numels[k] > 0)
                LT_HIP(hipMemcpyAsync(grad_at(k, base, places[i][j]), grads[k],
                                      size_t(numels[k]) * gbytes, H2D, hs));
        if (lt_err e = mark(i, 1, hs))
            return e;
        LT_HIP(hipEventRecord(ev.in[sl], hs));
        LT_HIP(hipStreamWaitEvent(cs, ev.in[sl], 0));
        const int Ki = layer_first[i + 1] - layer_first[i];
        const int64_t Ci = reinterpret_cast<int64_t*>(header.data() + lay.sq_prefix[i])[Ki];
        if (lt_err e = launch_sq_chunks(
                guard, grad_dtype, reinterpret_cast<const int64_t*>(ws + lay.sq_prefix[i]),
                reinterpret_cast<const uint64_t*>(ws + lay.sq_ptrs[i]),
                reinterpret_cast<const int64_t*>(ws + lay.sq_numels[i]), Ki, Ci,
                d_partials + gprefix[layer_first[i]], cs))
            return e;
        LT_HIP(hipEventRecord(ev.freed[sl], cs));
        used[sl] = used[sl] || !resident;
    }
    if (!norm_ready) {
        const auto* d_gprefix = reinterpret_cast<const int64_t*>(ws + lay.gprefix);
        k_sqnorm_finish<<<K, kThreads, 0, cs>>>(guard, d_gprefix, d_partials, d_sk);
        LT_HIP(hipGetLastError());
        k_sqnorm_total<<<1, 256, 0, cs>>>(guard, d_sk, K, nullptr, sq_total, status);
        LT_HIP(hipGetLastError());
    }
    k_clip_coef<<<1, 64, 0, cs>>>(sq_total, max_norm, total_norm, coef, nullptr);
    LT_HIP(hipGetLastError());

    // Pass 2: layer in, fused step, layer out.
    const StepScalars sc = make_scalars(lr, beta1, beta2, eps, weight_decay, step);
    for (int i = 0; i < L; ++i) {
        const int sl = i % S;
        if (used[sl])
            LT_HIP(hipStreamWaitEvent(hs, ev.freed[sl], 0));
        uint8_t* base = slot_base(i);
        if (lt_err e = mark(i, 2, hs))
            return e;
        for (int k = layer_first[i], j = 0; k < layer_first[i + 1]; ++k, ++j) {
            const SlotTensor& t = places[i][j];
            const size_t n = size_t(numels[k]), nb = size_t((numels[k] + B - 1) / B);
            if (n == 0)
                continue;
            LT_HIP(hipMemcpyAsync(base + t.w, params[k], n * 4, H2D, hs));
            if (!resident || norm_ready)  // resident gradients came in during pass 1
                LT_HIP(hipMemcpyAsync(grad_at(k, base, t), grads[k], n * gbytes, H2D, hs));
            LT_HIP(hipMemcpyAsync(base + t.mq, m_codes[k], n, H2D, hs));
            LT_HIP(hipMemcpyAsync(base + t.vq, v_codes[k], n, H2D, hs));
            LT_HIP(hipMemcpyAsync(base + t.ma, m_absmax[k], nb * 4, H2D, hs));
            LT_HIP(hipMemcpyAsync(base + t.va, v_absmax[k], nb * 4, H2D, hs));
        }
        if (lt_err e = mark(i, 3, hs))
            return e;
        LT_HIP(hipEventRecord(ev.in[sl], hs));
        LT_HIP(hipStreamWaitEvent(cs, ev.in[sl], 0));
        if (lt_err e = mark(i, 6, cs))
            return e;
        const int Ki = layer_first[i + 1] - layer_first[i];
        const auto* up = reinterpret_cast<const int64_t*>(ws + lay.st_prefix[i]);
        const auto* dp = reinterpret_cast<const StepTensor*>(ws + lay.st_desc[i]);
        const int64_t units = reinterpret_cast<int64_t*>(header.data() + lay.st_prefix[i])[Ki];
        const bool wb = any_set(params_bf16 ? params_bf16 + layer_first[i] : nullptr, Ki);
        lt_err e = units == 0 ? LT_OK
                   : grad_dtype == LT_DTYPE_BF16
                       ? launch_step<uint16_t>(guard, B, up, dp, Ki, units, sc, coef, status, wb,
                                               code_map, cs)
                       : launch_step<float>(guard, B, up, dp, Ki, units, sc, coef, status, wb,
                                            code_map, cs);
        if (e)
            return e;
        if (wb)
            if (lt_err e2 = launch_bf16_on_skip(guard, up, dp, Ki, units, unit, status, cs))
                return e2;
        if (lt_err e = mark(i, 7, cs))
            return e;
        LT_HIP(hipEventRecord(ev.computed[sl], cs));
        LT_HIP(hipStreamWaitEvent(ds, ev.computed[sl], 0));
        if (lt_err e = mark(i, 4, ds))
            return e;
        for (int k = layer_first[i], j = 0; k < layer_first[i + 1]; ++k, ++j) {
            const SlotTensor& t = places[i][j];
            const size_t n = size_t(numels[k]), nb = size_t((numels[k] + B - 1) / B);
            if (n == 0)
                continue;
            LT_HIP(hipMemcpyAsync(params[k], base + t.w, n * 4, D2H, ds));
            LT_HIP(hipMemcpyAsync(m_codes[k], base + t.mq, n, D2H, ds));
            LT_HIP(hipMemcpyAsync(v_codes[k], base + t.vq, n, D2H, ds));
            LT_HIP(hipMemcpyAsync(m_absmax[k], base + t.ma, nb * 4, D2H, ds));
            LT_HIP(hipMemcpyAsync(v_absmax[k], base + t.va, nb * 4, D2H, ds));
            if (bf16_copy && params_bf16[k])
                LT_HIP(hipMemcpyAsync(params_bf16[k], base + t.wb, n * 2, D2H, ds));
        }
        if (lt_err e = mark(i, 5, ds))
            return e;
        LT_HIP(hipEventRecord(ev.freed[sl], ds));
        used[sl] = true;
    }
    // The call's work ends on the compute stream once the last copy out is done.
    LT_HIP(hipEventRecord(ev.done, ds));
    LT_HIP(hipStreamWaitEvent(cs, ev.done, 0));
    return LT_OK;
}

// fp32-state workspace: [tag][unit prefix K+1][Fp32Tensor K]
size_t lt_adamw_fp32_workspace_bytes(int n_tensors)
{
    return n_tensors < 0 ? 0 : round_up(kTagBytes + round_up(sizeof(int64_t) * (n_tensors + 1), 64) +
                                            sizeof(Fp32Tensor) * size_t(n_tensors), 256);
}

lt_err lt_adamw_fp32_step(float* const* params, const void* const* grads, int grad_dtype,
                          float* const* exp_avg, float* const* exp_avg_sq,
                          uint16_t* const* params_bf16, const int64_t* numels, int n_tensors, double lr, double beta1, double beta2, double eps,
                          double weight_decay, int64_t step, const float* coef,
                          const int32_t* status, const void* step_state, void* workspace,
                          size_t workspace_bytes, void* stream)
{
    g_last_error.clear();
    const int K = n_tensors;
    if (!valid_list(numels, K) || !lists_given(K, {params, grads, exp_avg, exp_avg_sq}))
        return fail(LT_ERR_INVALID_ARG, "tensor lists must hold n_tensors >= 0 entries with numel >= 0");
    if (grad_dtype != LT_DTYPE_F32 && grad_dtype != LT_DTYPE_BF16)
        return fail(LT_ERR_INVALID_ARG, "grad_dtype must be LT_DTYPE_F32 or LT_DTYPE_BF16");
    if (!valid_hyper(lr, beta1, beta2, eps, weight_decay, step_state ? 1 : step))
        return fail(LT_ERR_INVALID_ARG, "need finite lr, weight_decay >= 0, finite eps > 0 (also "
                                        "in fp32), 0 <= beta1, beta2 < 1 and step >= 1");
    if ((coef && !aligned(coef, 4)) || (status && !aligned(status, 4)) ||
        (step_state && !aligned(step_state, 16)))
        return fail(LT_ERR_ALIGNMENT, "coef and status must be 4-byte aligned, step_state 16-byte");
    for (int k = 0; k < K; ++k) {
        if (numels[k] == 0)
            continue;
        if (!params[k] || !grads[k] || !exp_avg[k] || !exp_avg_sq[k])
            return fail(LT_ERR_INVALID_ARG, "NULL tensor pointer at index " + std::to_string(k));
        if (!aligned(params[k], 16) || !aligned(grads[k], 16) || !aligned(exp_avg[k], 16) ||
            !aligned(exp_avg_sq[k], 16))
            return fail(LT_ERR_ALIGNMENT, "tensor " + std::to_string(k) + " is not 16-byte aligned");
        if (params_bf16 && !aligned(params_bf16[k], 16))
            return fail(LT_ERR_ALIGNMENT,
                        "params_bf16[" + std::to_string(k) + "] must be 16-byte aligned");
    }
    {
        std::vector<ByteRange> r;
        r.reserve(size_t(K) * 5);
        const size_t gbytes = grad_dtype == LT_DTYPE_BF16 ? 2 : 4;
        for (int k = 0; k < K; ++k) {
            const size_t n = size_t(numels[k]);
            add_range(r, params[k], n * 4, true);
            add_range(r, grads[k], n * gbytes, false);
            add_range(r, exp_avg[k], n * 4, true);
            add_range(r, exp_avg_sq[k], n * 4, true);
            if (params_bf16)
                add_range(r, params_bf16[k], n * 2, true);
        }
        const std::string e = overlap_error(std::move(r));
        if (!e.empty())
            return fail(LT_ERR_INVALID_ARG, e);
    }
    const size_t desc_at = kTagBytes + round_up(sizeof(int64_t) * (K + 1), 64);
    const size_t total = lt_adamw_fp32_workspace_bytes(K);
    if (!workspace || !aligned(workspace, 256) || workspace_bytes < total)
        return fail(LT_ERR_WORKSPACE, "workspace must be 256-byte aligned and hold " +
                                          std::to_string(total) + " bytes");
    constexpr int64_t span = 64 * kFp32ElemsPerLane;
    std::vector<uint8_t> host(total, 0);
    auto* prefix = reinterpret_cast<int64_t*>(host.data() + kTagBytes);
    auto* desc = reinterpret_cast<Fp32Tensor*>(host.data() + desc_at);
    prefix[0] = 0;
    for (int k = 0; k < K; ++k) {
        prefix[k + 1] = prefix[k] + (numels[k] + span - 1) / span;
        desc[k] = Fp32Tensor{params[k],  grads[k],
                             exp_avg[k], exp_avg_sq[k],
                             numels[k],  params_bf16 ? params_bf16[k] : nullptr,
                             {0, 0}};
    }
    const int64_t units = prefix[K];
    if (units == 0)
        return LT_OK;  // every tensor is empty
    StepScalars sc = make_scalars(lr, beta1, beta2, eps, weight_decay, step_state ? 1 : step);
    sc.state = static_cast<const uint8_t*>(step_state);
    auto* ws = static_cast<uint8_t*>(workspace);
    hipStream_t st = static_cast<hipStream_t>(stream);
    WsGuard guard;
    if (lt_err e = put_descriptors(host, ws, st, &guard))
        return e;
    const auto* d_prefix = reinterpret_cast<const int64_t*>(ws + kTagBytes);
    const auto* d_desc = reinterpret_cast<const Fp32Tensor*>(ws + desc_at);
    const bool wb = any_set(params_bf16, K);
    auto* kernel = grad_dtype == LT_DTYPE_BF16
                       ? (wb ? k_adamw32_step<uint16_t, true> : k_adamw32_step<uint16_t, false>)
                       : (wb ? k_adamw32_step<float, true> : k_adamw32_step<float, false>);
    int grid;
    if (lt_err e = grid_size(kernel, (units + 3) / 4, &grid))
        return e;
    kernel<<<grid, kThreads, 0, st>>>(guard, d_prefix, d_desc, K, units, sc, coef, status);
    LT_HIP(hipGetLastError());
    if (status && wb)
        return launch_bf16_on_skip(guard, d_prefix, d_desc, K, units, span, status, st);
    return LT_OK;
}

lt_err lt_select_8bit_slice(const int64_t* numels, int n_tensors, double fraction,
                            uint8_t* is_8bit, int64_t* n_8bit_params)
{
    g_last_error.clear();
    if (!valid_list(numels, n_tensors) || !lists_given(n_tensors, {is_8bit}) ||
        !(fraction >= 0.0 && fraction <= 1.0))
        return fail(LT_ERR_INVALID_ARG, "need n_tensors >= 0 numels >= 0, is_8bit and 0 <= fraction <= 1");
    int64_t total = 0;
    for (int k = 0; k < n_tensors; ++k)
        total += numels[k];
    const double target = fraction * double(total);
    std::vector<int> order(n_tensors);
    for (int k = 0; k < n_tensors; ++k)
        order[k] = k;
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return numels[a] > numels[b]; });
    int64_t chosen = 0;
    for (int k = 0; k < n_tensors; ++k)
        is_8bit[k] = 0;
    for (int k : order)
        if (double(chosen + numels[k]) <= target) {
            is_8bit[k] = 1;
            chosen += numels[k];
        }
    if (n_8bit_params)
        *n_8bit_params = chosen;
    return LT_OK;
}

size_t lt_step_state_bytes(int64_t table_len)
{
    return table_len < 1 ? 0 : sizeof(lt_step_state) + sizeof(lt_step_table_entry) * size_t(table_len);
}

lt_err lt_step_table(double beta1, double beta2, int64_t t_first, int64_t count,
                     lt_step_table_entry* out)
{
    g_last_error.clear();
    if (!(beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0) || t_first < 1 ||
        count < 0 || (count > 0 && !out))
        return fail(LT_ERR_INVALID_ARG, "need 0 <= beta1, beta2 < 1, t_first >= 1, count >= 0");
    for (int64_t i = 0; i < count; ++i)
        out[i] = step_table_entry(beta1, beta2, t_first + i);
    return LT_OK;
}

lt_err lt_step_state_init(void* state, size_t bytes, int64_t table_len, double beta1,
                          double beta2, int64_t applied, int32_t skips, int32_t max_skips,
                          const void* from_state, void* stream)
{
    g_last_error.clear();
    if (table_len < 1 || applied < 0 || skips < 0 || max_skips < 0 ||
        !(beta1 >= 0.0 && beta1 < 1.0 && beta2 >= 0.0 && beta2 < 1.0))
        return fail(LT_ERR_INVALID_ARG, "need table_len >= 1, applied, skips, max_skips >= 0 and "
                                        "0 <= beta1, beta2 < 1");
    if (!state || bytes < lt_step_state_bytes(table_len))
        return fail(LT_ERR_WORKSPACE, "the step state must hold " +
                                          std::to_string(lt_step_state_bytes(table_len)) + " bytes");
    if (!aligned(state, 16) || (from_state && !aligned(from_state, 16)))
        return fail(LT_ERR_ALIGNMENT, "step states must be 16-byte aligned");
    std::vector<uint8_t> image(lt_step_state_bytes(table_len), 0);
    auto* h = reinterpret_cast<lt_step_state*>(image.data());
    h->applied = applied;
    h->table_len = table_len;
    h->skips = skips;
    h->max_skips = max_skips;
    h->stopped = 0;
    auto* table = reinterpret_cast<lt_step_table_entry*>(image.data() + sizeof(lt_step_state));
    for (int64_t i = 0; i < table_len; ++i)
        table[i] = step_table_entry(beta1, beta2, i + 1);
    int dev;
    if (lt_err e = current_device(&dev))
        return e;
    hipStream_t st = static_cast<hipStream_t>(stream);
    {
        std::lock_guard<std::mutex> lock(g_dev[dev].mu);
        if (lt_err e = stage_copy_locked(g_dev[dev], image.data(), image.size(), state, st))
            return e;
    }
    if (from_state) {
        k_step_state_copy<<<1, 64, 0, st>>>(static_cast<lt_step_state*>(state),
                                             static_cast<const lt_step_state*>(from_state));
        LT_HIP(hipGetLastError());
    }
    return LT_OK;
}

lt_err lt_step_state_advance(void* state, const int32_t* status, void* stream)
{
    g_last_error.clear();
    if (!state || !status)
        return fail(LT_ERR_INVALID_ARG, "state and status must not be NULL");
    if (!aligned(state, 16) || !aligned(status, 4))
        return fail(LT_ERR_ALIGNMENT, "state must be 16-byte aligned, status 4-byte");
    k_step_state_advance<<<1, 64, 0, static_cast<hipStream_t>(stream)>>>(
        static_cast<lt_step_state*>(state), status);
    LT_HIP(hipGetLastError());
    return LT_OK;
}

lt_err lt_read_status(const int32_t* status, void* stream, int32_t* out)
{
    g_last_error.clear();
    if (!status || !out)
        return fail(LT_ERR_INVALID_ARG, "status and out must not be NULL");
    hipStream_t st = static_cast<hipStream_t>(stream);
    LT_HIP(hipMemcpyAsync(out, status, sizeof(int32_t), hipMemcpyDeviceToHost, st));
    LT_HIP(hipStreamSynchronize(st));
    return LT_OK;
}

lt_err lt_workspace_release(const void* workspace)
{
    g_last_error.clear();
    if (!workspace)
        return LT_OK;
    for (int d = 0; d < kMaxDevices; ++d) {
        DeviceState& ds = g_dev[d];
        std::lock_guard<std::mutex> lock(ds.mu);
        auto it = ds.cache.find(workspace);
        if (it == ds.cache.end())
            continue;
        if (it->second.copied)
            ds.spare_events.push_back(it->second.copied);
        ds.cache.erase(it);
    }
    return LT_OK;
}

lt_err lt_set_max_workgroups(int max_workgroups)
{
    g_last_error.clear();
    if (max_workgroups < 0)
        return fail(LT_ERR_INVALID_ARG, "max_workgroups must be >= 0");
    g_max_workgroups.store(max_workgroups);
    return LT_OK;
}

const char* lt_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
