// Cache generation on gfx950: the three position networks F_pos^j on their
// plane grids and the direction network F_dir on the direction nodes
// (SqueezeNeRF Sec. 3.2-3.4), written straight into the cache layout the
// renderer reads.
//
// Every layer is a GEMM on the matrix cores, v_mfma_f32_32x32x16_f16, in
// the transposed form  H_out^T = W H_in^T:  the weights are the A operand
// (32 output units x 16 inputs per fragment) and the activations the B
// operand (16 inputs x 32 points), so a wave carries 32 points through the
// whole network without leaving registers.  The accumulator of an M-tile
// holds, in lane l, units 8g + 4(l/32) + q (g, q = 0..3) of point l % 32;
// a K step of the next layer is made of the 8 units g in {2t, 2t + 1} of
// one tile, i.e. the MFMA's k index kappa = 8 (l/32) + e of K step s stands
// for unit 16 s + 8 (e/4) + 4 (l/32) + e % 4.  The weight fragments are laid
// out on the host with that same permutation of the inputs, so the product
// is exact and no activation is shuffled.  Activations are rounded to
// binary16 after bias and ReLU (binary32); accumulation is binary32.
//
// The weights of each layer are staged through LDS in chunks of 4 K steps
// x all M-tiles (32 KiB at 256 units), shared by the waves of a workgroup
// (8 waves, 256 points, for the position networks; 4 waves for the
// direction network); each lane reads its 16-byte fragment with one
// ds_read_b128.
#include <math.h>

#include "sqn_internal.h"

namespace sqn {
namespace {

typedef _Float16 half8 __attribute__((ext_vector_type(8)));
typedef float float16v __attribute__((ext_vector_type(16)));

constexpr int kFrag = 512;          // halves per fragment (64 lanes x 8)
constexpr int kChunkSteps = 4;      // K steps staged per chunk
constexpr double kPi = 3.14159265358979323846;

__device__ __forceinline__ const _Float16* frag_of(const GenNet& net, int l)
{
    return static_cast<const _Float16*>(net.frag[l]);
}

// the unit held by element e of lane-half h in a K step (see the file head)
__device__ __forceinline__ int kmap(int h, int e) { return 8 * (e >> 2) + 4 * h + (e & 3); }

// Stage chunk c of a layer (fragments [c][m][ss][lane][8], `tiles` M-tiles)
// into LDS.
__device__ __forceinline__ void stage_chunk(const _Float16* __restrict__ frag, int tiles, _Float16* wbuf)
{
    const int n16 = tiles * kChunkSteps * kFrag / 8;      // 16-byte pieces
    const uint4* src = reinterpret_cast<const uint4*>(frag);
    uint4* dst = reinterpret_cast<uint4*>(wbuf);
    for (int i = threadIdx.x; i < n16; i += blockDim.x)
        dst[i] = src[i];
}

// One layer: acc[m] = sum over K steps of W-fragment(m, s) x x[s], for
// m < tiles (TMAX compile-time bound) and KS K steps.
template <int TMAX, int KS>
__device__ __forceinline__ void layer(const _Float16* __restrict__ frag, int tiles, const half8 (&x)[KS],
                                      float16v (&acc)[TMAX], _Float16* wbuf)
{
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int m = 0; m < TMAX; ++m)
        acc[m] = float16v{};
#pragma unroll
    for (int c = 0; c < KS / kChunkSteps; ++c) {
        __syncthreads();
        stage_chunk(frag + static_cast<size_t>(c) * tiles * kChunkSteps * kFrag, tiles, wbuf);
        __syncthreads();
#pragma unroll
        for (int ss = 0; ss < kChunkSteps; ++ss) {
#pragma unroll
            for (int m = 0; m < TMAX; ++m) {
                if (m < tiles) {
                    const half8 a = *reinterpret_cast<const half8*>(wbuf + ((m * kChunkSteps + ss) * 64 + lane) * 8);
                    acc[m] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, x[c * kChunkSteps + ss], acc[m], 0, 0, 0);
                }
            }
        }
    }
}

// bias + ReLU, rounded to binary16: the K-step fragments of the next layer
template <int T>
__device__ __forceinline__ void activate(const float16v (&acc)[T], const float* __restrict__ bias,
                                         half8 (&x)[2 * T])
{
    const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
    for (int m = 0; m < T; ++m) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float4 b = *reinterpret_cast<const float4*>(bias + 32 * m + 8 * g + 4 * h);
            const float bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float v = fmaxf(acc[m][4 * g + q] + bv[q], 0.0f);
                x[2 * m + (g >> 1)][4 * (g & 1) + q] = static_cast<_Float16>(v);
            }
        }
    }
}

// ---- double-buffered layers (position networks): while the matrix cores
// work on one chunk of weights from LDS, the next chunk streams from global
// memory straight into the other LDS buffer (global_load_lds, no
// registers), and with a layer's first chunk its 256 biases; one barrier per
// chunk, which also waits for those loads.  The two buffers are separate
// arrays chosen at compile time, so the compiler sees that the reads of one
// do not wait for the loads into the other.  Measured on the 1K cache:
// biases read from global memory in the activation, loads left to sink to
// the end of the chunk and one buffer array indexed at run time each cost
// 4-10%; a deeper pipeline (four buffers, two chunks ahead) was slower.

constexpr int kPosThreads = 512;    // threads per position workgroup (2 waves per SIMD)

// Direct-to-LDS loads of a chunk of TMAX tiles x 4 K steps (32 KiB at 8
// tiles; the host pads every layer of the position networks to TMAX tiles):
// piece i = 512 k + threadIdx.x (16 bytes) lands at buf + 16 i.
template <int TMAX>
__device__ __forceinline__ void load_chunk(const _Float16* __restrict__ frag, _Float16* buf)
{
    const int wave = threadIdx.x >> 6;
#pragma unroll
    for (int k = 0; k < TMAX * 256 / kPosThreads; ++k) {
        const int piece = kPosThreads * k + threadIdx.x;
        __builtin_amdgcn_global_load_lds(reinterpret_cast<const unsigned int*>(frag) + 4 * piece,
                                         reinterpret_cast<unsigned int*>(buf) + 4 * (kPosThreads * k + 64 * wave),
                                         16, 0, 0);
    }
}

// One layer of KS K steps over `tiles` (<= TMAX) M-tiles for NB point
// blocks.  The current chunk is in buffer P0 (loaded and published by the
// last barrier); next_frag is the first chunk of the following layer
// (after the last layer any valid chunk: loaded but never read).
template <int TMAX, int NB, int KS, int P0>
__device__ __forceinline__ void layer_pipe(const _Float16* __restrict__ frag, int tiles,
                                           const half8 (&x)[NB][KS], float16v (&acc)[TMAX][NB], _Float16* buf0,
                                           _Float16* buf1, const _Float16* next_frag, const float* __restrict__ bias,
                                           float* bias_lds)
{
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int m = 0; m < TMAX; ++m)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
            acc[m][nb] = float16v{};
    constexpr int NC = KS / kChunkSteps;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const bool last = c + 1 == NC;
        // chunk c sits in buffer (P0 + c) % 2, known at compile time, so the
        // compiler can tell the loads into the other buffer from the reads
        _Float16* const cur = ((P0 + c) & 1) ? buf1 : buf0;
        _Float16* const other = ((P0 + c) & 1) ? buf0 : buf1;
        load_chunk<TMAX>(last ? next_frag : frag + static_cast<size_t>(c + 1) * TMAX * kChunkSteps * kFrag, other);
        // the layer's 256 biases (1 KiB) follow the same way, by one wave
        if (c == 0 && threadIdx.x < 64)
            __builtin_amdgcn_global_load_lds(reinterpret_cast<const unsigned int*>(bias) + 4 * threadIdx.x,
                                             reinterpret_cast<unsigned int*>(bias_lds), 16, 0, 0);
        // keep the loads at the top of the chunk: issued late they would be
        // waited for at the chunk's barrier
        __builtin_amdgcn_sched_barrier(0);
        const _Float16* wb = cur;
#pragma unroll
        for (int ss = 0; ss < kChunkSteps; ++ss) {
            // fragment reads of the step ahead of its products, so each wait
            // covers several reads; the other wave on the SIMD fills it
            half8 a[TMAX];
#pragma unroll
            for (int m = 0; m < TMAX; ++m)
                a[m] = *reinterpret_cast<const half8*>(wb + ((m * kChunkSteps + ss) * 64 + lane) * 8);
#pragma unroll
            for (int m = 0; m < TMAX; ++m)
                if (m < tiles) {
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        acc[m][nb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[m], x[nb][c * kChunkSteps + ss],
                                                                            acc[m][nb], 0, 0, 0);
                }
            // in halves: four reads, four products (bounds the registers)
            __builtin_amdgcn_sched_group_barrier(0x100, TMAX / 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, TMAX / 2 * NB, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, TMAX / 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, TMAX / 2 * NB, 0);
        }
        __syncthreads();
    }
}

template <int T, int NB>
__device__ __forceinline__ void activate_nb(const float16v (&acc)[T][NB], const float* __restrict__ bias,
                                            half8 (&x)[NB][2 * T])
{
    const int h = (threadIdx.x & 63) >> 5;
#pragma unroll
    for (int m = 0; m < T; ++m)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const float4 b = *reinterpret_cast<const float4*>(bias + 32 * m + 8 * g + 4 * h);
            const float bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float v = fmaxf(acc[m][nb][4 * g + q] + bv[q], 0.0f);
                    x[nb][2 * m + (g >> 1)][4 * (g & 1) + q] = static_cast<_Float16>(v);
                }
        }
}

__device__ __forceinline__ void store_value(void* base, size_t idx, float v, int f16)
{
    if (f16)
        static_cast<_Float16*>(base)[idx] = static_cast<_Float16>(v);
    else
        static_cast<float*>(base)[idx] = v;
}

// Per-axis NeRF encoding tables, binary64 evaluation rounded to binary16:
// tab[axis][i][0] = x_i, [1 + 2k] = sin(2^k pi x_i), [2 + 2k] = cos(2^k pi x_i)
// with x_i = lo + i (hi - lo) / (n_p - 1).
__global__ void encode_axes(GenParams P, _Float16* __restrict__ tab)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    const int axis = blockIdx.y;
    if (i >= P.n_p)
        return;
    const int nc = 1 + 2 * P.pos_freq;
    const double lo = P.bmin[axis], hi = P.bmax[axis];
    const double x = lo + static_cast<double>(i) * ((hi - lo) / static_cast<double>(P.n_p - 1));
    _Float16* row = tab + (static_cast<size_t>(axis) * P.n_p + i) * nc;
    row[0] = static_cast<_Float16>(x);
    for (int k = 0; k < P.pos_freq; ++k) {
        const double y = ldexp(x, k);
        row[1 + 2 * k] = static_cast<_Float16>(sinpi(y));
        row[2 + 2 * k] = static_cast<_Float16>(cospi(y));
    }
}

// Position networks: blockIdx.y = plane j (xy, yz, zx); 256 points of the
// plane's [n_p][n_p] grid per workgroup, row-major, kPosNB blocks of 32 per
// wave (blocks share every weight fragment read from LDS).
constexpr int kPosNB = 1;
constexpr int kPosPoints = kPosThreads / 64 * 32 * kPosNB;

__global__ __launch_bounds__(kPosThreads, 1) void position_kernel(GenParams P, const _Float16* __restrict__ tab)
{
    // two separate arrays, so that loads into one never wait for reads of
    // the other
    __shared__ __align__(16) _Float16 wbuf0[8 * kChunkSteps * kFrag];
    __shared__ __align__(16) _Float16 wbuf1[8 * kChunkSteps * kFrag];
    // layer l's biases sit in bias_lds[l & 1] from its first chunk on
    __shared__ __align__(16) float bias_lds[2][256];
    const int j = blockIdx.y;
    const int lane = threadIdx.x & 63, h = lane >> 5;
    const int64_t n_pts = static_cast<int64_t>(P.n_p) * P.n_p;
    const int64_t base = static_cast<int64_t>(blockIdx.x) * kPosPoints + (threadIdx.x >> 6) * (32 * kPosNB);
    // plane j = (first, second) axes (0,1), (1,2), (2,0)
    const int ax_a = j, ax_b = (j + 1) % 3;
    const int nc = 1 + 2 * P.pos_freq;
    const GenNet& net = P.pos[j];

    // start loading the first layer's weights, then build the input
    // fragments: NeRF order [a, b, sin a, sin b, cos a, cos b, ...] per
    // frequency, zero beyond n_in (64 inputs = 4 K steps)
    load_chunk<8>(frag_of(net, 0), wbuf0);
    int64_t pt[kPosNB];
    half8 x0[kPosNB][4];
#pragma unroll
    for (int nb = 0; nb < kPosNB; ++nb) {
        const int64_t p_raw = base + 32 * nb + (lane & 31);
        pt[nb] = p_raw < n_pts ? p_raw : -1;
        const int64_t p = p_raw < n_pts ? p_raw : n_pts - 1;
        const int ia = static_cast<int>(p / P.n_p), ib = static_cast<int>(p - static_cast<int64_t>(ia) * P.n_p);
        const _Float16* ta = tab + (static_cast<size_t>(ax_a) * P.n_p + ia) * nc;
        const _Float16* tb = tab + (static_cast<size_t>(ax_b) * P.n_p + ib) * nc;
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int f = 16 * s + kmap(h, e);
                _Float16 v = 0;
                if (f < 2) {
                    v = f == 0 ? ta[0] : tb[0];
                } else if (f < P.pos_in) {
                    const int r = f - 2, k = r >> 2, t = r & 3;
                    const _Float16* src = (t & 1) ? tb : ta;
                    v = src[1 + 2 * k + (t >> 1)];
                }
                x0[nb][s][e] = v;
            }
    }
    __syncthreads();

    float16v acc[8][kPosNB];
    half8 x[kPosNB][16];
    const int L = net.n_hidden;
    layer_pipe<8, kPosNB, 4, 0>(frag_of(net, 0), 8, x0, acc, wbuf0, wbuf1, frag_of(net, 1), net.bias[0],
                                bias_lds[0]);
    activate_nb<8, kPosNB>(acc, bias_lds[0], x);
    for (int l = 1; l < L; ++l) {
        layer_pipe<8, kPosNB, 16, 1>(frag_of(net, l), 8, x, acc, wbuf0, wbuf1, frag_of(net, l + 1),
                                     net.bias[l], bias_lds[l & 1]);
        activate_nb<8, kPosNB>(acc, bias_lds[l & 1], x);
    }
    layer_pipe<8, kPosNB, 16, 1>(frag_of(net, L), net.out_tiles, x, acc, wbuf0, wbuf1, frag_of(net, L),
                                 net.bias[L], bias_lds[L & 1]);

    // head: pair slot P = 16 m + 8 gg + 4 h + q sits in rows 32 m + 16 gg +
    // 4 h + q and + 8 of tile m, i.e. accumulator entries 8 gg + q and
    // 8 gg + 4 + q of this lane; slot 0 is (sigma_0, w_sigma), slot 1 + c D + d
    // is (w_c[d], c_0[d]) (Eq. 3)
    const float* hb = bias_lds[L & 1];
    const int D = P.D;
#pragma unroll
    for (int m = 0; m < 8; ++m) {
        if (m >= net.out_tiles)
            break;
#pragma unroll
        for (int gg = 0; gg < 2; ++gg)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int slot = 16 * m + 8 * gg + 4 * h + q;
                const int row = 32 * m + 16 * gg + 4 * h + q;
                const float b0 = hb[row], b1 = hb[row + 8];
#pragma unroll
                for (int nb = 0; nb < kPosNB; ++nb) {
                    if (pt[nb] < 0)
                        continue;
                    const float prod = (acc[m][nb][8 * gg + q] + b0) * (acc[m][nb][8 * gg + 4 + q] + b1);
                    if (slot == 0)
                        store_value(P.sigma_out[j], static_cast<size_t>(pt[nb]), prod, P.sigma_f16);
                    else if (slot <= 3 * D)
                        store_value(P.uvw_out[j], static_cast<size_t>(pt[nb]) * (3 * D) + (slot - 1), prod,
                                    P.uvw_f16);
                }
            }
    }
}

// Direction network on the n_theta x n_phi nodes (theta from +z over
// [0, pi], phi = -pi + b 2 pi / n_phi), 128 nodes per workgroup.
__global__ __launch_bounds__(256, 2) void direction_kernel(GenParams P)
{
    __shared__ __align__(16) _Float16 wbuf[4 * kChunkSteps * kFrag];
    const int lane = threadIdx.x & 63, h = lane >> 5;
    const int64_t n_pts = static_cast<int64_t>(P.n_theta) * P.n_phi;
    const int64_t p_raw = static_cast<int64_t>(blockIdx.x) * 128 + (threadIdx.x >> 6) * 32 + (lane & 31);
    const bool valid = p_raw < n_pts;
    const int64_t p = valid ? p_raw : n_pts - 1;
    const int a = static_cast<int>(p / P.n_phi), b = static_cast<int>(p - static_cast<int64_t>(a) * P.n_phi);
    const double th = static_cast<double>(a) * (kPi / static_cast<double>(P.n_theta - 1));
    const double ph = -kPi + static_cast<double>(b) * (2.0 * kPi / static_cast<double>(P.n_phi));
    const double d[3] = {sin(th) * cos(ph), sin(th) * sin(ph), cos(th)};

    // NeRF order [d, sin(2^0 pi d), cos(2^0 pi d), ...], 3 components each
    half8 x0[4];
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int f = 16 * s + kmap(h, e);
            double v = 0.0;
            if (f < 3) {
                v = d[f];
            } else if (f < P.dir_in) {
                const int r = f - 3, k = r / 6, t = r % 6;
                const double y = ldexp(d[t % 3], k);
                v = t < 3 ? sinpi(y) : cospi(y);
            }
            x0[s][e] = static_cast<_Float16>(v);
        }

    const GenNet& net = P.dir;
    float16v acc[4];
    half8 x[8];
    layer<4, 4>(frag_of(net, 0), 4, x0, acc, wbuf);
    activate<4>(acc, net.bias[0], x);
    for (int l = 1; l < net.n_hidden; ++l) {
        layer<4, 8>(frag_of(net, l), 4, x, acc, wbuf);
        activate<4>(acc, net.bias[l], x);
    }
    layer<4, 8>(frag_of(net, net.n_hidden), 1, x, acc, wbuf);
    if (!valid)
        return;
    const float* hb = net.bias[net.n_hidden];
#pragma unroll
    for (int g = 0; g < 4; ++g)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int row = 8 * g + 4 * h + q;
            if (row < P.D)
                store_value(P.beta_out, static_cast<size_t>(p) * P.D + row, acc[0][4 * g + q] + hb[row], P.beta_f16);
        }
}

}  // namespace

hipError_t launch_generate(const GenParams& p, _Float16* enc_table, hipStream_t stream)
{
    encode_axes<<<dim3((p.n_p + 63) / 64, 3), 64, 0, stream>>>(p, enc_table);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    const int64_t n_pos = static_cast<int64_t>(p.n_p) * p.n_p;
    position_kernel<<<dim3(static_cast<uint32_t>((n_pos + kPosPoints - 1) / kPosPoints), 3), kPosThreads, 0, stream>>>(
        p, enc_table);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    const int64_t n_dir = static_cast<int64_t>(p.n_theta) * p.n_phi;
    direction_kernel<<<dim3(static_cast<uint32_t>((n_dir + 127) / 128)), 256, 0, stream>>>(p);
    return hipGetLastError();
}

}  // namespace sqn
