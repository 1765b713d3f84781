// Internal types shared by the C ABI layer (api.hip) and the render kernels
// (render.hip).  Not part of the public interface.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sqn.h"

namespace sqn {

// Everything one render launch reads, passed by value as the kernel argument.
struct RenderParams {
    // caches (library-owned device memory)
    const void* sigma[3];     // packed (sigma, distance) records of planes xy, yz, zx, four rows
                              // interleaved (prepare.hip)
    const void* uvw[3];       // [n_p][n_p][3D] records
    const void* beta;         // [n_theta][n_phi][D]
    // camera batch and outputs (caller-owned device memory)
    const float* poses;       // [B][3][4]
    float* rgb;               // [B][H][W][3] or null (stats launches)
    float* depth;             // [B][H][W] or null
    uint32_t* stats;          // [B][H][W][4] or null
    // camera
    float fx, fy, cx, cy;
    int32_t width, height, n_views;
    // sampling
    float near_t, far_t, dt;  // dt = (far - near) / N in binary32
    int32_t n_samples;
    int32_t stratified;       // 1: seeded offset inside each bin
    // grid
    float bmin[3], bmax[3];
    float scale[3];           // (n_p - 1) / (bmax - bmin) in binary32
    int32_t n_p, D, n_theta, n_phi;
    int32_t beta_f16;
    double theta_scale;       // (n_theta - 1) / pi: grid coordinate per radian
    double phi_scale;         // n_phi / (2 pi)
    uint32_t rec_bytes;       // bytes of one uvw record (3D values)
    int64_t tau_eps;          // floor(-ln(eps) 2^32), INT64_MAX for eps = 0
    uint64_t seed;
    float inv_dt;             // 1 / dt (conservative box clip and leap indices)
    float leap_k, leap_c;     // leap index fma(t_exit, leap_k, -leap_c): leap_k = (1 - 2^-19) / dt,
                              // leap_c = near leap_k + 2^-19 |near| / dt (binary64, rounded once)
    // launch geometry
    int32_t lanes;            // lanes per ray: 1, 4 or 8
    int32_t skip;             // 1: one lane per ray with empty-space leaps
    float leap_margin;        // texels a leap keeps from its square's edge
    int32_t tiles_x, tiles_y; // workgroup tiles per view
    int32_t n_groups;         // workgroups in the grid
    int32_t block_order;      // 1: blocks of 2 x 2 tiles, each on one XCD, from the centre outwards
    // hybrid launch (one view): a centred rectangle of blocks of 16 x 16
    // pixels marched with four lanes per ray, the other blocks with one
    int32_t hybrid;           // 1: hybrid launch
    int32_t hy_bx, hy_by;     // blocks per image row and column
    int32_t hy_x0, hy_y0;     // first block of the rectangle
    int32_t hy_w, hy_h;       // rectangle size in blocks
    int32_t n_heavy;          // workgroups of the rectangle (four per block), dispatched first
    // linear (Eq. 5) decoder; sigma[j] then holds per-plane partial sums
    int32_t linear;           // 1: Eq. 5, 0: Eq. 4
    float b_sigma;            // density bias
    const float* lin_w;       // [9D + 3][D]: rows c*3D + e of W_c^T, then b_u, b_v, b_w
    int32_t lin_stride;       // LDS floats per ray of the folded weights
    float ndc_near;           // > 0: rays marched in normalized device coordinates
    // Eq. 5: 3-D grid of cells of cell_g^3 nodes, cell_m per axis, holding
    // the capped Chebyshev distance (cells) to the nearest cell that may
    // hold sigma > 0
    const uint8_t* cell_dist;
    int32_t cell_shift, cell_m;   // cell side 2^cell_shift nodes
};

// Launch one render over all views on `stream`; `stats` selects the variant
// that writes per-ray diagnostics.  Shapes have been validated by the
// caller.  Returns the launch status.
hipError_t launch_render(const RenderParams& p, int sigma_dtype, int uvw_dtype,
                         bool stats, hipStream_t stream);

// Cap of the stored Chebyshev distance to the nearest occupied texel.
constexpr int32_t kDistCap = 255;

// Temporary device buffers of the create-time preparation.
struct PrepareWork {
    uint8_t* live;        // [n_p^2] 1 where a texel may give sigma > 0
    uint16_t* f;          // [n_p^2] row distances
    uint16_t* dist;       // [n_p^2] capped Chebyshev distances
    float* maxima;        // [6][n_p] row / column maxima of the partial sums
    float* w_sigma;       // [3 d_sigma] density weights (linear decoder)
    float* cell_max;      // [3][m][m] per-plane cell maxima (linear decoder)
    uint8_t* cell_live;   // [m^3]
    uint16_t* cell_f;     // [m^3] partial distances
    uint16_t* cell_f2;    // [m^3]
    uint2* rows;          // [n_p^2] row-major copy of a linear decoder's plane
};

// Pack sigma plane j (n_p x n_p of sigma_dtype, device memory) into
// `packed` (4-byte records for binary16 sigma, 8-byte for binary32) with the
// capped distance transform.
hipError_t prepare_sigma_plane(const void* sigma, int sigma_dtype, int32_t n_p, void* packed,
                               const PrepareWork& work, hipStream_t stream);

// Linear (Eq. 5) decoder: fold each plane's sigma^j vectors
// ([n_p][n_p][d_sigma] of sigma_dtype) with its block of W_sigma into
// per-texel partial sums, mark the texels whose samples are empty whatever
// the other two planes hold, and write 8-byte records (partial sum, capped
// distance to the nearest texel not so marked) to packed[j].
hipError_t prepare_linear_planes(const void* const sigma[3], int sigma_dtype, int32_t n_p,
                                 int32_t d_sigma, float b_sigma, void* const packed[3],
                                 const PrepareWork& work, hipStream_t stream);

// Cell grid of the linear decoder (after prepare_linear_planes): cells of
// g x g x g nodes (g = 2^shift), m = ceil(n_p / g) per axis; a cell is empty when
// ((M_xy + M_yz) + M_zx) + b_sigma <= 0 with M_j the largest partial sum of
// plane j over the cell's footprint (binary32 addition is monotone), and
// cell_dist[(cx m + cy) m + cz] receives the capped Chebyshev distance in
// cells to the nearest cell not so marked.  work.cell_max holds 3 m^2
// floats, work.cell_live m^3 bytes, work.cell_f / cell_g2 m^3 uint16 each.
hipError_t prepare_linear_cells(const void* const packed[3], int32_t n_p, float b_sigma, int32_t shift,
                                int32_t m, uint8_t* cell_dist, const PrepareWork& work, hipStream_t stream);

// Move the linear decoder's packed planes (row-major after the passes
// above) into the interleaved order the renderer reads, through work.rows.
hipError_t interleave_linear_planes(void* const packed[3], int32_t n_p, const PrepareWork& work,
                                    hipStream_t stream);

// Cell side 2^shift for an n_p grid: the smallest power of two >= 2 that
// leaves at most 128 cells per axis.
constexpr int32_t linear_cell_shift(int32_t n_p)
{
    int32_t s = 1;
    while (((n_p + (1 << s) - 1) >> s) > 128)
        ++s;
    return s;
}
constexpr int32_t linear_cells(int32_t n_p) { return (n_p + (1 << linear_cell_shift(n_p)) - 1) >> linear_cell_shift(n_p); }

// Per-ray LDS floats of the folded Eq. 5 radiance weights: n values padded
// to 4 (mod 8) words so that 16 rays' 16-byte reads spread over the banks.
constexpr int32_t lin_pad(int32_t n)
{
    const int32_t m = (n + 3) / 4 * 4;
    return m % 8 == 0 ? m + 4 : m;
}
// 9D + 3 rows for a compile-time D; 10D + 3 (rows, then beta) otherwise.
constexpr int32_t lin_stride(int32_t D) { return lin_pad(9 * D + 3); }
constexpr int32_t lin_stride_generic(int32_t D) { return lin_pad(10 * D + 3); }

// ---- cache generation (generate.hip) ----------------------------------------

// Most hidden layers a network may have.
constexpr int32_t kMaxHidden = 16;

// One network on the device: per layer (hidden layers, then the head) the
// weights in MFMA fragment order (binary16) and the binary32 biases.
struct GenNet {
    const void* frag[kMaxHidden + 1];
    const float* bias[kMaxHidden + 1];
    int32_t n_hidden;
    int32_t out_tiles;        // 32-row tiles of the head
};

struct GenParams {
    GenNet pos[3];            // F_pos^xy, F_pos^yz, F_pos^zx (256 units)
    GenNet dir;               // F_dir (128 units)
    int32_t n_p, n_theta, n_phi, D;
    int32_t pos_freq, dir_freq, pos_in, dir_in;
    float bmin[3], bmax[3];
    void* sigma_out[3];
    void* uvw_out[3];
    void* beta_out;
    int32_t sigma_f16, uvw_f16, beta_f16;
};

// Encoding tables (3 n_p (1 + 2 pos_freq) binary16 values of scratch in
// enc_table), then the position and direction kernels, on `stream`.
hipError_t launch_generate(const GenParams& p, _Float16* enc_table, hipStream_t stream);

// Workgroup geometry: 256 threads = 4 wave64; with L lanes per ray a wave
// holds 64/L rays laid out as a wave tile of kWaveW(L) x kWaveH(L) pixels
// (8x8, 4x4 or 4x2 for L = 1, 4, 8) and a workgroup covers 2 x 2 wave tiles.
constexpr int kBlockThreads = 256;
constexpr int kWaveW(int L) { return L >= 4 ? 4 : 8; }
constexpr int kWaveH(int L) { return (64 / L) / kWaveW(L); }
constexpr int kTileW(int L) { return 2 * kWaveW(L); }
constexpr int kTileH(int L) { return 2 * kWaveH(L); }

}  // namespace sqn
