// Internal host-side interface between the C-ABI layer and the kernel
// launch tables.  Not installed; the public interface is include/mep.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "mep_kernels.hpp"

namespace mep {

// Row-group geometry of one streaming-kernel instance: G lanes per row
// group, V vectors per lane, B rows per batch, WPE waves per SIMD (the
// register budget is 512 / WPE per lane), AUX the cache-policy bits of the
// matrix loads (0 = default, 2 = non-temporal streaming).  MAP and CUX are
// launch arguments, not part of the instance: MAP hands row blocks to
// workgroups cyclically (0), in contiguous runs (1) or cyclically with the
// positions rotated from one window of blocks to the next (2); CUX is how many of
// each XCD's 32 compute units the grid is sized for (workgroups are dealt to
// the 8 XCDs in turn).  Measured on MI355X, streaming one large matrix from
// 22-26 compute units per XCD beats all 32 (fewer rows in flight at once);
// with two matrices all 32 are faster.
struct Cfg {
    int G, V, B, WPE, AUX, MAP = 0, CUX = 32;
};

constexpr int kXcds = 8;
constexpr int kCusPerXcd = 32;

// Vector path (16-byte loads), ordered by row capacity G * V; among equal
// capacities the preferred shape comes first (measured on MI355X: streaming
// the matrix with non-temporal loads is faster for every shape).
constexpr int kNumVecCfg = 58;
constexpr Cfg kVecCfg[kNumVecCfg] = {
    // rows of 1-8 vectors: 2, 4 or 8 lanes per row, 32, 16 or 8 rows per wave
    // (4-row batches for BICG, whose 8-row batches spill registers in fp64)
    {2, 1, 8, 4, 2},     {2, 1, 8, 4, 0},     {2, 1, 4, 4, 2},
    {4, 1, 8, 4, 2},     {4, 1, 8, 4, 0},     {4, 1, 4, 4, 2},
    {8, 1, 8, 4, 2},     {8, 1, 8, 4, 0},     {8, 1, 4, 4, 2},
    {16, 1, 8, 4, 2},    {16, 1, 8, 4, 2, 0, 24}, {16, 1, 8, 4, 2, 0, 16}, {16, 1, 8, 4, 0},
    {16, 1, 4, 4, 2},
    {64, 1, 8, 4, 2},    {64, 1, 8, 4, 0},
    {64, 2, 4, 4, 2},    {64, 2, 4, 4, 0},    {64, 4, 2, 4, 2},    {64, 4, 2, 4, 0},
    // 512 vectors
    {256, 2, 4, 4, 2},   {256, 2, 4, 4, 0},   {512, 1, 8, 4, 2},
    // 1024 vectors
    {256, 4, 2, 4, 2},   {256, 4, 2, 4, 0},   {512, 2, 8, 2, 2},   {512, 2, 8, 2, 0},
    {512, 2, 8, 2, 2, 0, 24},
    {512, 2, 4, 4, 2},   {1024, 1, 8, 4, 2},
    // 2048 vectors
    {1024, 2, 4, 4, 2},  {1024, 2, 4, 4, 0},  {512, 4, 4, 2, 2},   {512, 4, 4, 2, 0},
    {512, 4, 4, 2, 2, 0, 24},
    // 4096 vectors: a 16384-element fp32 row
    {512, 8, 2, 2, 2, 2, 24}, {512, 8, 2, 2, 2, 0, 24}, {512, 8, 2, 2, 2, 0, 22}, {512, 8, 2, 2, 2}, {512, 8, 2, 2, 2, 1},
    {1024, 4, 2, 4, 2},  {1024, 4, 2, 4, 2, 0, 24}, {512, 8, 1, 4, 2}, {256, 16, 1, 2, 2},
    {512, 8, 2, 2, 0},   {1024, 4, 2, 4, 0},   {512, 8, 1, 4, 0},   {256, 16, 1, 2, 0},
    // 8192 vectors: a 16384-element fp64 row or a 32768-element fp32 row
    {512, 16, 1, 2, 2, 2, 26}, {512, 16, 1, 2, 2, 0, 26}, {512, 16, 1, 2, 2, 0, 24}, {512, 16, 1, 2, 2}, {512, 16, 1, 2, 2, 1},
    {1024, 8, 1, 4, 2},  {256, 32, 1, 1, 2},   {512, 16, 1, 2, 0},  {1024, 8, 1, 4, 0},
    {256, 32, 1, 1, 0}};
// Element-wise path (rows not 16-byte aligned): one element per load, so
// batches are deep (B * V = 8-16 elements per lane) to keep 32-64 bytes per
// lane in flight; short rows get as many lanes as they have elements.
// Ordered by row capacity G * V.
constexpr int kNumScalarCfg = 16;
constexpr Cfg kScalarCfg[kNumScalarCfg] = {
    {8, 1, 16, 4, 2},   {8, 1, 8, 4, 2},    {16, 1, 16, 4, 2},  {16, 1, 8, 4, 2},
    {32, 1, 16, 4, 2},  {32, 1, 8, 4, 2},   {64, 1, 16, 4, 2},  {64, 1, 8, 4, 2},
    {64, 2, 8, 4, 2},   {64, 4, 4, 4, 2},   {64, 4, 2, 4, 2},
    {256, 2, 8, 4, 2},  {256, 4, 4, 4, 2},  {256, 4, 2, 4, 2},
    {1024, 8, 2, 4, 2}, {1024, 8, 1, 4, 2}};

// Rows per batch an instance really uses: two-matrix modes (GESUMMV) hold
// twice the rows in registers, so they take half the batch.
constexpr int batch_of(int B, int mode) { return (mode & F_TWO) ? (B > 1 ? B / 2 : 1) : B; }

// Rough per-lane register need of an instance (vgpr32 = registers per
// loaded vector): two row buffers, the column sums, the register copies of
// the column vectors, the rank-2 row scalars and some fixed overhead.  Instances above the budget of
// their occupancy target are never built or chosen.
constexpr int n_colvecs(int mode) { return ((mode & F_DOT) ? 1 : 0) + ((mode & F_RANK2) ? 2 : 0); }
constexpr bool colvecs_in_lds(Cfg c, int mode, int vgpr32)
{
    return n_colvecs(mode) > 0 && n_colvecs(mode) * c.V * vgpr32 * 4 > (c.WPE <= 2 ? 128 : 64);
}
constexpr int vgpr_estimate(Cfg c, int mode, int vgpr32)
{
    const int mats = (mode & F_TWO) ? 2 : 1;
    const int bufs = 2 * mats * batch_of(c.B, mode) * c.V * vgpr32;
    const int col = (mode & F_COL) ? c.V * vgpr32 : 0;
    const int x = colvecs_in_lds(c, mode, vgpr32) ? 0 : n_colvecs(mode) * c.V * vgpr32;
    // rank-2 update: u1 and u2 of every row of both batches (two registers
    // each for fp64) and the store addressing
    const int u = (mode & F_RANK2) ? 8 * batch_of(c.B, mode) + 8 : 0;
    return bufs + col + x + u + 24;
}
// LDS of the per-lane column-vector slots (the other arrays are small).
constexpr int lds_estimate(Cfg c, int mode, int vgpr32)
{
    const int threads = c.G < 256 ? 256 : c.G;
    return colvecs_in_lds(c, mode, vgpr32) ? n_colvecs(mode) * c.V * threads * vgpr32 * 4 : 0;
}
constexpr bool cfg_fits(Cfg c, int mode, int vgpr32)
{
    return vgpr_estimate(c, mode, vgpr32) <= 512 / c.WPE && lds_estimate(c, mode, vgpr32) <= 144 * 1024;
}

struct Plan {
    bool vec;         // 16-byte vector path
    int vw;           // elements per load
    int cfg;          // index into kVecCfg / kScalarCfg
    Cfg c;
    int threads;      // workgroup size
    int64_t pw;       // columns per panel (equal panels, the last possibly shorter)
    int64_t panels;   // column panels (gridDim.x)
    int64_t nb;       // row workgroups (gridDim.y)
};

// Candidate configurations for an m x n matrix (a pure function of its
// arguments: no device query), the default first.  Returns the count; fills
// idx[] (capacity 16).
int stream_candidates(int esize, bool vec, int mode, int64_t m, int64_t n, int* idx);
// The plan of candidate `variant` (-1: the default, candidate 0).
Plan plan_stream(int esize, bool vec, int mode, int64_t m, int64_t n, int variant);

// Optional timing events for one streaming-kernel launch (both null: none).
struct LaunchEvents {
    hipEvent_t start, stop;
};

template <typename T>
hipError_t launch_stream(const Plan& p, int mode, const StreamArgs<T>& a, hipStream_t s,
                         const LaunchEvents& ev);

template <typename T>
hipError_t launch_colreduce(const T* P, const T* Q, int64_t ldp, int64_t nrows, int64_t ncols,
                            T alpha, T beta, T* out, hipStream_t s, int epi);

template <typename T>
hipError_t launch_fill_zero(T* p, int64_t count, hipStream_t s);

// The per-dtype launch tables (mep_launch_{f32,f64}{,_wide}.hip).
template <>
hipError_t launch_stream<float>(const Plan&, int, const StreamArgs<float>&, hipStream_t, const LaunchEvents&);
template <>
hipError_t launch_stream<double>(const Plan&, int, const StreamArgs<double>&, hipStream_t, const LaunchEvents&);
template <>
hipError_t launch_colreduce<float>(const float*, const float*, int64_t, int64_t, int64_t, float, float,
                                   float*, hipStream_t, int);
template <>
hipError_t launch_colreduce<double>(const double*, const double*, int64_t, int64_t, int64_t, double,
                                    double, double*, hipStream_t, int);
template <>
hipError_t launch_fill_zero<float>(float*, int64_t, hipStream_t);
template <>
hipError_t launch_fill_zero<double>(double*, int64_t, hipStream_t);

// Two-stage sum of n elements (partials in ws, nb = reduce_blocks(n)).
int64_t reduce_blocks(int64_t n, int esize);
template <typename T>
hipError_t launch_reduce_sum(const T* x, int64_t n, T* out, T* partial, int64_t nb, hipStream_t s,
                             const LaunchEvents& ev);
template <typename T>
hipError_t launch_vector_add(const T* a, const T* b, T* c, int64_t n, int variant, hipStream_t s,
                             const LaunchEvents& ev);
template <>
hipError_t launch_reduce_sum<float>(const float*, int64_t, float*, float*, int64_t, hipStream_t,
                                    const LaunchEvents&);
template <>
hipError_t launch_reduce_sum<double>(const double*, int64_t, double*, double*, int64_t, hipStream_t,
                                     const LaunchEvents&);
template <>
hipError_t launch_vector_add<float>(const float*, const float*, float*, int64_t, int, hipStream_t,
                                    const LaunchEvents&);
template <>
hipError_t launch_vector_add<double>(const double*, const double*, double*, int64_t, int, hipStream_t,
                                     const LaunchEvents&);

// Candidate launches of the vector add: 0-1 = rows of 1024-lane workgroups
// through buffer resources on 32 or 24 compute units per XCD (0, the
// default, measured the fastest), 2 = contiguous chunk per workgroup, 3-5 =
// rows with plain non-temporal loads and stores on 32, 24 or 16.
constexpr int kNumVaddVariants = 6;

hipError_t launch_copy16(const void* src, void* dst, size_t bytes, hipStream_t s);
hipError_t launch_flush(void* buf, size_t bytes, uint32_t tag, hipStream_t s);

}  // namespace mep
