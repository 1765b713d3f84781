// Memory-level ceilings for the render kernel's roofline, measured on the
// GPU that runs it: streaming reads of a buffer (a footprint that one XCD's
// L2 holds, one that the MALL holds, one that only HBM holds) and random
// gathers of 64-byte records over a buffer, the access pattern of the cache
// lookups.  A measurement aid for bench.py, built as its own library
// (libsqn_probe.so); the render library does not use it.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

constexpr int kThreads = 256;

// Every thread folds what it reads into one word; the store of a value that
// never occurs keeps the loads alive.
__global__ __launch_bounds__(kThreads) void stream_kernel(const uint4* __restrict__ buf, uint64_t n16,
                                                          int passes, uint32_t* __restrict__ sink)
{
    uint32_t acc = 0;
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kThreads;
    for (int p = 0; p < passes; ++p) {
        uint64_t i = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x;
        // four loads in flight per lane
        for (; i + 3 * stride < n16; i += 4 * stride) {
            const uint4 a = buf[i], b = buf[i + stride], c = buf[i + 2 * stride], d = buf[i + 3 * stride];
            acc ^= (a.x ^ a.y ^ a.z ^ a.w) ^ (b.x ^ b.y ^ b.z ^ b.w) ^ (c.x ^ c.y ^ c.z ^ c.w) ^ (d.x ^ d.y ^ d.z ^ d.w);
        }
        for (; i < n16; i += stride) {
            const uint4 v = buf[i];
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

int grid_for(uint64_t items)
{
    int cus = 256;
    int dev = 0;
    if (hipGetDevice(&dev) == hipSuccess)
        (void)hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    const uint64_t want = (items + kThreads - 1) / kThreads;
    const uint64_t cap = static_cast<uint64_t>(cus) * 16;
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

}  // namespace

extern "C" {

// Read a `bytes` buffer (a multiple of 16) `passes` times; *ms_out is the
// time of one such launch.  Returns 0, or 1 on a HIP error.
int sqn_probe_stream(uint64_t bytes, int passes, float* ms_out)
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
    const int grid = grid_for(n16);
    if (rc == 0)
        rc = time_launch([&] { stream_kernel<<<grid, kThreads>>>(static_cast<const uint4*>(buf), n16, passes, sink); },
                         ms_out);
    (void)hipFree(sink);
    (void)hipFree(buf);
    return rc;
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

}  // extern "C"
