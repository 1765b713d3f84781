// Ceilings for the rooflines, measured on the GPU that runs the kernels:
// for the render kernel, streaming reads of a buffer (a footprint that one
// XCD's L2 holds, one that the MALL holds, one that only HBM holds) and
// random gathers of 64-byte records over a buffer, the access pattern of the
// cache lookups; the vector-memory data path at saturation, with gathers
// that the vector L1 serves in the lane patterns of the render kernel's
// loads; for cache generation, the rate of independent
// v_mfma_f32_32x32x16_f16 products at two waves per SIMD.  A measurement aid
// for bench.py, built as its own library (libsqn_probe.so); the render
// library does not use it.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Every thread folds what it reads into one word; the store of a value that
// never occurs keeps the loads alive.  U 16-byte loads in flight per lane.
// Cached levels (several passes over the buffer): four loads, 16 workgroups
// per CU striding over the whole buffer.  HBM (one pass over 4 GiB): eight
// loads on a grid of 128 workgroups per CU, 6.0-6.3 TB/s on one MI355X
// against 5.6 TB/s in the cached-level form, and with the non-temporal hint
// (NT: no reuse expected) 6.7-7.1 TB/s.
template <int U, bool NT>
__global__ __launch_bounds__(kThreads) void stream_kernel(const u32x4* __restrict__ buf, uint64_t n16, int passes,
                                                          uint32_t* __restrict__ sink)
{
    uint32_t acc = 0;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kThreads;
    for (int p = 0; p < passes; ++p) {
        uint64_t i = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x;
        for (; i + (U - 1) * stride < n16; i += U * stride) {
            u32x4 v[U];
#pragma unroll
            for (int k = 0; k < U; ++k)
                v[k] = NT ? __builtin_nontemporal_load(&buf[i + k * stride]) : buf[i + k * stride];
#pragma unroll
            for (int k = 0; k < U; ++k)
                acc ^= v[k].x ^ v[k].y ^ v[k].z ^ v[k].w;
        }
        for (; i < n16; i += stride) {
            const u32x4 v = buf[i];
            acc ^= v.x ^ v.y ^ v.z ^ v.w;
        }
    }
    if (acc == 0x9e3779b9u)
        sink[threadIdx.x] = acc;
}

// Four lanes read one 64-byte record (16 bytes each); the record of a
// group of 4 lanes is a hash of its global index scaled to the records in
// the buffer.
__global__ __launch_bounds__(kThreads) void gather_kernel(const uint4* __restrict__ buf, uint32_t n_rec,
                                                          uint64_t n_reads, uint32_t* __restrict__ sink)
{
    uint32_t acc = 0;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kThreads;
    auto piece = [&](uint64_t i) {
        uint64_t z = (i >> 2) * 0x9E3779B97F4A7C15ull;
        z = (z ^ (z >> 31)) * 0xBF58476D1CE4E5B9ull;
        const uint32_t r = static_cast<uint32_t>(((z >> 32) * n_rec) >> 32);
        return 4ull * r + (i & 3);
    };
    uint64_t i = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x;
    // four gathers in flight per lane (stride is a multiple of 4, so a
    // lane keeps its 16-byte piece of each record)
    for (; i + 3 * stride < n_reads; i += 4 * stride) {
        const uint4 a = buf[piece(i)], b = buf[piece(i + stride)], c = buf[piece(i + 2 * stride)],
                    d = buf[piece(i + 3 * stride)];
        acc ^= (a.x ^ a.y ^ a.z ^ a.w) ^ (b.x ^ b.y ^ b.z ^ b.w) ^ (c.x ^ c.y ^ c.z ^ c.w) ^ (d.x ^ d.y ^ d.z ^ d.w);
    }
    for (; i < n_reads; i += stride) {
        const uint4 v = buf[piece(i)];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u)
        sink[threadIdx.x] = acc;
}

// Gathers from a 16 KiB buffer (256 segments of 64 bytes) that stays in
// every CU's vector L1, four independent loads per lane and iteration, so
// the memory data path is all that limits the rate.  A load's segment is a
// hash of the lane (or, with `quads`, of the lane's quad: the four lanes of
// a quad then share a segment) and of the load's number; within the
// segment a lane reads dword (lane % 16) or, with 16-byte loads, piece
// (lane % 4).  Every index stays below 4096 dwords / 1024 pieces.
template <bool WIDE>
__global__ __launch_bounds__(kThreads) void vmem_kernel(const uint32_t* __restrict__ buf, int iters, int quads,
                                                        uint32_t* __restrict__ sink)
{
    const uint32_t lane = threadIdx.x & 63u;
    const uint32_t who = quads ? (lane >> 2) : lane;
    uint32_t h = (blockIdx.x * 0x9E3779B9u) ^ ((threadIdx.x >> 6) * 0x85EBCA6Bu) ^ (who * 0xC2B2AE35u);
    uint32_t acc = 0;
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            h = h * 1664525u + 1013904223u;
            const uint32_t seg = h >> 24;   // 0..255
            if constexpr (WIDE) {
                const uint4 v = reinterpret_cast<const uint4*>(buf)[seg * 4u + (lane & 3u)];
                acc ^= v.x ^ v.y ^ v.z ^ v.w;
            } else {
                acc ^= buf[seg * 16u + (lane & 15u)];
            }
        }
    }
    if (acc == 0x9e3779b9u)
        sink[threadIdx.x] = acc;
}

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

// Eight independent accumulators per wave, operands in registers: nothing
// but the matrix cores limits the rate.
__global__ __launch_bounds__(kThreads, 2) void mfma_kernel(int iters, float* __restrict__ sink)
{
    half8 a, b;
    for (int e = 0; e < 8; ++e) {
        a[e] = static_cast<_Float16>(static_cast<float>(threadIdx.x) * 0.001f + static_cast<float>(e));
        b[e] = static_cast<_Float16>(0.5f * static_cast<float>(e));
    }
    float16v acc[8] = {};
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int m = 0; m < 8; ++m)
            acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[m], 0, 0, 0);
    }
    float s = 0.0f;
    for (int m = 0; m < 8; ++m)
        s += acc[m][0];
    if (s == 1234.5f)
        sink[threadIdx.x] = s;
}

int grid_for(uint64_t items, int per_cu = 16)
{
    int cus = 256;
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const uint64_t want = (items + kThreads - 1) / kThreads;
    const uint64_t cap = static_cast<uint64_t>(cus) * per_cu;
    return static_cast<int>(want < cap ? (want > 0 ? want : 1) : cap);
}

template <typename F>
int time_launch(F launch, float* ms_out)
{
    hipEvent_t e0, e1;
    if (hipEventCreate(&e0) != hipSuccess)
        return 1;
    if (hipEventCreate(&e1) != hipSuccess) {
        (void)hipEventDestroy(e0);
        return 1;
    }
    launch();  // warm the caches and the code
    (void)hipEventRecord(e0, nullptr);
    launch();
    (void)hipEventRecord(e1, nullptr);
    hipError_t e = hipEventSynchronize(e1);
    float ms = 0.0f;
    if (e == hipSuccess)
        e = hipEventElapsedTime(&ms, e0, e1);
    if (e == hipSuccess)
        e = hipGetLastError();
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    *ms_out = ms;
    return e == hipSuccess ? 0 : 1;
}

int probe_stream(uint64_t bytes, int passes, bool nontemporal, float* ms_out)
{
    if (bytes < 16 || bytes % 16 != 0 || passes < 1 || !ms_out)
        return 1;
    void* buf = nullptr;
    uint32_t* sink = nullptr;
    if (hipMalloc(&buf, bytes) != hipSuccess)
        return 1;
    if (hipMalloc(reinterpret_cast<void**>(&sink), kThreads * 4) != hipSuccess) {
        (void)hipFree(buf);
        return 1;
    }
    int rc = hipMemset(buf, 1, bytes) == hipSuccess ? 0 : 1;
    const uint64_t n16 = bytes / 16;
    const u32x4* b = static_cast<const u32x4*>(buf);
    if (rc == 0) {
        if (passes > 1) {
            const int grid = grid_for(n16, 16);
            rc = nontemporal
                     ? time_launch([&] { stream_kernel<4, true><<<grid, kThreads>>>(b, n16, passes, sink); }, ms_out)
                     : time_launch([&] { stream_kernel<4, false><<<grid, kThreads>>>(b, n16, passes, sink); }, ms_out);
        } else {
            const int grid = grid_for(n16, 128);
            rc = nontemporal
                     ? time_launch([&] { stream_kernel<8, true><<<grid, kThreads>>>(b, n16, passes, sink); }, ms_out)
                     : time_launch([&] { stream_kernel<8, false><<<grid, kThreads>>>(b, n16, passes, sink); }, ms_out);
        }
    }
    (void)hipFree(sink);
    (void)hipFree(buf);
    return rc;
}

}  // namespace

extern "C" {

// Read a `bytes` buffer (a multiple of 16) `passes` times; *ms_out is the
// time of one such launch.  Returns 0, or 1 on a HIP error.
int sqn_probe_stream(uint64_t bytes, int passes, float* ms_out)
{
    return probe_stream(bytes, passes, false, ms_out);
}

// The same with non-temporal loads (the streaming rate of a buffer that
// only HBM holds).
int sqn_probe_stream_nt(uint64_t bytes, int passes, float* ms_out)
{
    return probe_stream(bytes, passes, true, ms_out);
}

// n_records random 64-byte records gathered from a `bytes` buffer (a
// multiple of 64, at most 2^32 records); *ms_out is the time of the launch.
int sqn_probe_gather(uint64_t bytes, uint64_t n_records, float* ms_out)
{
    if (bytes < 64 || bytes % 64 != 0 || bytes / 64 > 0xffffffffull || n_records < 1 || !ms_out)
        return 1;
    void* buf = nullptr;
    uint32_t* sink = nullptr;
    if (hipMalloc(&buf, bytes) != hipSuccess)
        return 1;
    if (hipMalloc(reinterpret_cast<void**>(&sink), kThreads * 4) != hipSuccess) {
        (void)hipFree(buf);
        return 1;
    }
    int rc = hipMemset(buf, 1, bytes) == hipSuccess ? 0 : 1;
    const uint32_t n_rec = static_cast<uint32_t>(bytes / 64);
    const uint64_t n_reads = 4 * n_records;
    const int grid = grid_for(n_reads);
    if (rc == 0)
        rc = time_launch([&] { gather_kernel<<<grid, kThreads>>>(static_cast<const uint4*>(buf), n_rec, n_reads, sink); },
                         ms_out);
    (void)hipFree(sink);
    (void)hipFree(buf);
    return rc;
}

// Vector-memory data path at saturation: `iters` x 4 gathers per lane from
// a 16 KiB L1-resident buffer, dword (wide = 0) or 16-byte (wide = 1)
// loads, every lane its own 64-byte segment (quads = 0) or the four lanes of
// a quad sharing one (quads = 1); 32 waves per CU.  *cycles_out is the
// GPU time per wave-level load instruction on one CU, in cycles of
// `clock_ghz`.  Returns 0, or 1 on a HIP error or bad argument.
int sqn_probe_vmem(int wide, int quads, int iters, double clock_ghz, float* cycles_out)
{
    if (iters < 1 || clock_ghz <= 0.0 || !cycles_out || (wide != 0 && wide != 1) || (quads != 0 && quads != 1))
        return 1;
    int cus = 256;
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    constexpr uint64_t kBytes = 16384;
    void* buf = nullptr;
    uint32_t* sink = nullptr;
    if (hipMalloc(&buf, kBytes) != hipSuccess)
        return 1;
    if (hipMalloc(reinterpret_cast<void**>(&sink), kThreads * 4) != hipSuccess) {
        (void)hipFree(buf);
        return 1;
    }
    int rc = hipMemset(buf, 1, kBytes) == hipSuccess ? 0 : 1;
    const int blocks = cus * 8;
    float ms = 0.0f;
    if (rc == 0)
        rc = time_launch(
            [&] {
                if (wide)
                    vmem_kernel<true><<<blocks, kThreads>>>(static_cast<const uint32_t*>(buf), iters, quads, sink);
                else
                    vmem_kernel<false><<<blocks, kThreads>>>(static_cast<const uint32_t*>(buf), iters, quads, sink);
            },
            &ms);
    (void)hipFree(sink);
    (void)hipFree(buf);
    if (rc != 0 || !(ms > 0.0f))
        return 1;
    const double insts_per_cu = static_cast<double>(blocks) * (kThreads / 64) * iters * 4 / cus;
    *cycles_out = static_cast<float>(static_cast<double>(ms) * 1e-3 * clock_ghz * 1e9 / insts_per_cu);
    return 0;
}

// Dense binary16 matrix-core rate: `iters` x 8 products of 32x32x16 per
// wave, two workgroups of 4 waves on each CU, four rounds; *tflops_out in
// TFLOP/s.  Returns 0, or 1 on a HIP error or bad argument.
int sqn_probe_mfma_f16(int iters, float* tflops_out)
{
    if (iters < 1 || !tflops_out)
        return 1;
    int cus = 256;
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    float* sink = nullptr;
    if (hipMalloc(reinterpret_cast<void**>(&sink), kThreads * 4) != hipSuccess)
        return 1;
    const int blocks = cus * 2 * 4;
    float ms = 0.0f;
    const int rc = time_launch([&] { mfma_kernel<<<blocks, kThreads>>>(iters, sink); }, &ms);
    (void)hipFree(sink);
    if (rc != 0 || !(ms > 0.0f))
        return 1;
    const double flops = static_cast<double>(blocks) * (kThreads / 64) * iters * 8 * (32.0 * 32.0 * 16.0 * 2.0);
    *tflops_out = static_cast<float>(flops / (static_cast<double>(ms) * 1e-3) / 1e12);
    return 0;
}

}  // extern "C"
