// Device kernels of the dense matrix-vector family for gfx950 (MI355X).
//
// One streaming kernel serves every operation.  A "row group" of G lanes
// holds one row of A (or one column panel of it) in registers: lane g owns
// the V vectors of VW elements that start at column (v * G + g) * VW, so each
// load instruction of a row group reads G * VW consecutive elements and the
// whole matrix is read exactly once, front to back.  Rows are processed in
// batches of B per row group; the next batch is loaded while the current one
// is reduced (two register buffers used in turn).
//
// With a row in registers the kernel can, in the same pass,
//   * form the row dot d_i = A_i . x (butterfly shuffles inside a wave, then
//     an LDS exchange across the waves of a row group), and
//   * add s_i * A_i into per-lane column partial sums, where s_i is a given
//     weight w_i (z = A^T w, BICG's s = A^T r) or the dot itself
//     (ATAX: y = A^T (A x)).
// Column partials of a workgroup are written to a workspace row P[b, :];
// a second kernel sums the rows of P in a fixed order (no atomics), which
// makes every result bitwise reproducible.
//
// Matrix rows are read with buffer loads.  When a row group spans whole
// waves (G >= 64) the row is wave-uniform: its buffer resources (one per
// vector slot, base = the slot's first element in the row, size = the valid
// bytes left in the panel) live in scalar registers, every lane needs one
// 32-bit offset, and columns past the end of the row read as zero through
// the resource's range check (which covers the lane offset, not soffset).
// Narrower row groups (G < 64) put several consecutive rows in one wave;
// their resource spans those rows and lanes past the row end are pointed
// out of range explicitly.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mep {

enum : int { F_DOT = 1, F_TWO = 2, F_COL = 4, F_FROMDOT = 8, F_RANK2 = 16, F_STORE = 32 };
enum : int {
    MODE_MV = F_DOT,                         // y = A x (optionally scaled by alpha)
    MODE_AXPBY = F_DOT | F_TWO,              // y = alpha A x + beta B x
    MODE_ATW = F_COL,                        // z = A^T w
    MODE_BICG = F_DOT | F_COL,               // q = A p, s = A^T r
    MODE_ATAX = F_DOT | F_COL | F_FROMDOT,   // y = A^T (A x)
    MODE_GEMV1 = F_COL | F_RANK2 | F_STORE   // Ahat = A + u1 v1^T + u2 v2^T stored, and Ahat^T y
};

template <typename T, int VW>
struct VecOf {
    typedef T type __attribute__((ext_vector_type(VW)));
};

template <typename T>
struct StreamArgs {
    const T* A;        // m x n, row-major
    const T* B;        // second matrix (AXPBY)
    const T* x;        // dot vector, length n (x or p)
    const T* w;        // row weights, length m (ATW, BICG)
    T* rowout;         // per-row result, length m (y, q or ATAX's t; may be null for ATAX)
    T* colpart;        // column partials P[row workgroups][ldp]
    T* dotpart;        // multi-panel: partial dots D[panel][m]
    T* dotpart2;       // multi-panel AXPBY: partial dots of B
    const T* u1;       // rank-2 update (GEMVER): row factors, length m
    const T* u2;
    const T* v1;       // ... and column factors, length n
    const T* v2;
    T* Aout;           // the updated matrix (may equal A)
    T alpha, beta;
    int64_t m, n, ldp;
    int blocked;       // row-block map: 0 cyclic, 1 contiguous runs, 2 rotated cyclic (see k_stream)
    int64_t pw;        // columns per panel (all panels but the last have this width)
    int scale_rows;    // MV: rowout = alpha * dot instead of dot
};

// Cache-policy bits of a buffer store that writes through to memory at
// system scope (sc0 sc1): partial rows that the next kernel reads leave
// nothing dirty in the L2 for the end-of-kernel release to write back.
constexpr int kWriteThrough = 17;

// gfx9-family buffer descriptor, word 3 (raw, untyped 32-bit data).
constexpr int kRsrcWord3 = 0x00020000;
// A lane offset that is past the end of every resource built here.
constexpr uint32_t kOutOfRange = 0x40000000u;
// Shift per round of the rotated row-block map, in blocks (odd, so that the
// position of a workgroup's blocks in each window, and its address bits,
// cycle through every residue).
constexpr int kRotStride = 25;

// Buffer resource for `bytes` bytes at `base`.  Both must be wave-uniform;
// the size is pinned to a scalar register so that the descriptor never ends
// up in vector registers (which would force a per-lane loop around loads).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes)
{
    const int sbytes = __builtin_amdgcn_readfirstlane((int)bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, sbytes,
                                             kRsrcWord3);
}

__device__ __forceinline__ float fma_t(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ __forceinline__ double fma_t(double a, double b, double c) { return __builtin_fma(a, b, c); }

// 4, 8 or 16-byte raw buffer load; out-of-range lanes read zero.
template <typename T, int VW, int AUX>
__device__ __forceinline__ typename VecOf<T, VW>::type
load_buf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff)
{
    typedef typename VecOf<T, VW>::type vec;
    static_assert(sizeof(vec) == 4 || sizeof(vec) == 8 || sizeof(vec) == 16, "load width");
    if constexpr (sizeof(vec) == 16)
        return __builtin_bit_cast(vec, __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, AUX));
    else if constexpr (sizeof(vec) == 8)
        return __builtin_bit_cast(vec, __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, AUX));
    else
        return __builtin_bit_cast(vec, __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, AUX));
}

// 4, 8 or 16-byte raw buffer store; stores of out-of-range lanes are dropped.
template <typename T, int VW, int AUX>
__device__ __forceinline__ void store_buf(typename VecOf<T, VW>::type v, __amdgpu_buffer_rsrc_t r,
                                          uint32_t voff)
{
    typedef typename VecOf<T, VW>::type vec;
    if constexpr (sizeof(vec) == 16) {
        typedef unsigned int u4 __attribute__((ext_vector_type(4)));
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u4, v), r, (int)voff, 0, AUX);
    } else if constexpr (sizeof(vec) == 8) {
        typedef unsigned int u2 __attribute__((ext_vector_type(2)));
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u2, v), r, (int)voff, 0, AUX);
    } else {
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned int, v), r, (int)voff, 0, AUX);
    }
}

template <typename T, int VW>
__device__ __forceinline__ typename VecOf<T, VW>::type load_vec(const T* p)
{
    return *reinterpret_cast<const typename VecOf<T, VW>::type*>(p);
}

template <typename T, int VW>
__device__ __forceinline__ void store_vec(T* p, typename VecOf<T, VW>::type v)
{
    *reinterpret_cast<typename VecOf<T, VW>::type*>(p) = v;
}

// Streaming store: written once, read once by the next kernel.
template <typename T, int VW>
__device__ __forceinline__ void store_vec_nt(T* p, typename VecOf<T, VW>::type v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<typename VecOf<T, VW>::type*>(p));
}

// Workgroup barrier that orders LDS traffic only: outstanding global loads
// (the prefetched batch) stay in flight across it.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Cross-lane moves on 32-bit halves.  DPP controls (GFX9 encoding):
// quad_perm [1,0,3,2] = 0xB1 (lane ^ 1), quad_perm [2,3,0,1] = 0x4E
// (lane ^ 2), row_half_mirror = 0x141 (lane i <-> 7 - i within 8),
// row_mirror = 0x140 (lane i <-> 15 - i within 16).  ds_swizzle in bit-mask
// mode with and = 0x1F, xor = 0x10 (pattern 0x401F) swaps 16-lane halves of
// each 32 lanes.
template <int CTRL>
__device__ __forceinline__ int dpp_i(int v)
{
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, true);
}

template <typename T, typename F>
__device__ __forceinline__ T lanes_apply(T v, F f)
{
    if constexpr (sizeof(T) == 4) {
        return __builtin_bit_cast(T, f(__builtin_bit_cast(int, v)));
    } else {
        static_assert(sizeof(T) == 8, "32 or 64-bit values only");
        const uint64_t u = __builtin_bit_cast(uint64_t, v);
        const int lo = f((int)(uint32_t)u);
        const int hi = f((int)(uint32_t)(u >> 32));
        return __builtin_bit_cast(T, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
    }
}

// Sum over aligned groups of W lanes (W a power of two <= 64).  Each step adds
// a value from a lane of the other half of the current group; floating-point
// addition is commutative, so every lane of a group ends with the
// bitwise-same total, and the order never depends on timing.
template <int W, typename T>
__device__ __forceinline__ T group_sum(T v)
{
    static_assert(W >= 1 && W <= 64 && (W & (W - 1)) == 0, "group width");
    if constexpr (W >= 2)
        v += lanes_apply(v, [](int x) { return dpp_i<0xB1>(x); });
    if constexpr (W >= 4)
        v += lanes_apply(v, [](int x) { return dpp_i<0x4E>(x); });
    if constexpr (W >= 8)
        v += lanes_apply(v, [](int x) { return dpp_i<0x141>(x); });
    if constexpr (W >= 16)
        v += lanes_apply(v, [](int x) { return dpp_i<0x140>(x); });
    if constexpr (W >= 32)
        v += lanes_apply(v, [](int x) { return __builtin_amdgcn_ds_swizzle(x, 0x401F); });
    if constexpr (W >= 64) {
        const T lo = lanes_apply(v, [](int x) { return __builtin_amdgcn_readlane(x, 0); });
        const T hi = lanes_apply(v, [](int x) { return __builtin_amdgcn_readlane(x, 32); });
        v = lo + hi;
    }
    return v;
}

template <int G>
struct Geometry {
    static constexpr int THREADS = G < 256 ? 256 : G;
    static constexpr int RG = THREADS / G;            // row groups per workgroup
    static constexpr int NWAVES = THREADS / 64;
    static constexpr int WPG = G >= 64 ? G / 64 : 1;  // waves per row group
    static constexpr int RPW = G >= 64 ? 1 : 64 / G;  // rows per wave (G < 64)
};

// The streaming kernel.  Grid: x = column panels of a.pw columns (at most
// G * V * VW; the host makes them equal), y = row workgroups (rows handed out
// in blocks of B * RG, block k going to row workgroup k mod gridDim.y).
// Workgroups are dealt to the eight XCDs round-robin by linear id, so with
// the panel as the fast index the pieces of one row are read on different
// XCDs; with the panel as the slow index they all went to one XCD, and the
// panelled shapes streamed 3-22% slower (unequal panels: their short last
// panel also left compute units idle).  Narrow row groups (G < 64) are only
// launched with a single panel.  WPE is the occupancy target (waves per SIMD), which
// sets the register budget per lane to 512 / WPE.
template <typename T, int VW, int G, int V, int B, int WPE, int MODE, int AUX>
__global__ void __launch_bounds__(Geometry<G>::THREADS, WPE)
k_stream(StreamArgs<T> a)
{
    typedef typename VecOf<T, VW>::type vec;
    constexpr int THREADS = Geometry<G>::THREADS;
    constexpr int RG = Geometry<G>::RG;
    constexpr int NWAVES = Geometry<G>::NWAVES;
    constexpr int WPG = Geometry<G>::WPG;
    constexpr int RPW = Geometry<G>::RPW;
    constexpr int PW = G * V * VW;
    constexpr int BR = B * RG;
    constexpr uint32_t ES = sizeof(T);
    constexpr uint32_t VB = VW * ES;          // bytes per vector
    constexpr bool WIDE = G >= 64;            // one row per wave
    constexpr bool DOT = (MODE & F_DOT) != 0;
    constexpr bool TWO = (MODE & F_TWO) != 0;
    constexpr bool COL = (MODE & F_COL) != 0;
    constexpr bool FROMDOT = (MODE & F_FROMDOT) != 0;
    constexpr bool WTS = COL && !FROMDOT;
    constexpr bool RANK2 = (MODE & F_RANK2) != 0;
    constexpr bool STORE = (MODE & F_STORE) != 0;
    // the column vectors each lane keeps (x; or v1 and v2) live in registers
    // when their slices are small against the register budget (512 / WPE per
    // lane), else in per-lane LDS slots
    constexpr int NXV = (DOT ? 1 : 0) + (RANK2 ? 2 : 0);
    constexpr bool XLDS = NXV > 0 && (NXV * V * VB > (WPE <= 2 ? 128u : 64u));
    constexpr int NDOT = TWO ? 2 : 1;

    __shared__ vec xs[XLDS ? NXV * V * THREADS : 1];
    __shared__ T red[2][(G > 64) ? NDOT * B * WPG : 1];
    __shared__ vec cred[(COL && RG > 1) ? NWAVES * G * V : 1];

    const int tid = threadIdx.x;
    const int g = tid % G;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t m = a.m, n = a.n;
    const int m32 = (int)m;  // the host limits m and n to int range
    const int bx = (int)blockIdx.y;  // row workgroup
    const int by = (int)blockIdx.x;  // column panel
    const int64_t col0 = (int64_t)by * a.pw;
    const bool multipanel = gridDim.x > 1;
    const int nbx = gridDim.y;
    // valid bytes of this panel of one row
    const int64_t pcols = (n - col0) < a.pw ? (n - col0) : a.pw;
    const uint32_t pbytes = (uint32_t)(pcols * ES);
    const int64_t rowbytes = n * ES;

    // Row of row group `grp` of this wave in batch j of block blk: first row
    // of the wave is blk * BR + j * RG + wave_first_group.
    const int wgrp0 = WIDE ? wave / WPG : wave * RPW;   // first row group of this wave
    const int sub = WIDE ? 0 : lane / G;                // row of this lane inside the wave

    // lane offsets (bytes) of the V vectors inside the wave's resource
    uint32_t voff[WIDE ? 1 : V];
    if constexpr (WIDE) {
        voff[0] = (uint32_t)g * VB;
    } else {
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int64_t c = (int64_t)(v * G + g) * VW;
            voff[v] = c < n ? (uint32_t)(sub * rowbytes + c * ES) : kOutOfRange;
        }
    }
    // Wide row groups give vector v its own resource (base advanced by
    // v * G * VW elements, size clamped to what is left of the panel), so the
    // range check masks the row end for every vector with one lane offset.
    auto rsrc_v = [&](const T* rowp, uint32_t bytes, int v) __attribute__((always_inline)) {
        if constexpr (WIDE) {
            const int left = (int)bytes - v * G * (int)VB;
            return make_rsrc(rowp + (int64_t)v * G * VW, (uint32_t)(left > 0 ? left : 0));
        } else {
            return make_rsrc(rowp, bytes);
        }
    };
    auto lane_off = [&](int v) __attribute__((always_inline)) -> uint32_t {
        if constexpr (WIDE)
            return voff[0];
        else
            return voff[v];
    };

    const vec zero = (vec)(T)0;

    vec xv[XLDS ? 1 : NXV * V + 1];
    // slot k (0: x or v1, 1: v2) of vector v
    auto colvec = [&](int k, int v) __attribute__((always_inline)) -> vec {
        if constexpr (XLDS)
            return xs[(k * V + v) * THREADS + tid];
        else
            return xv[k * V + v];
    };

    vec acc[COL ? V : 1];
#pragma unroll
    for (int v = 0; v < (COL ? V : 1); ++v)
        acc[v] = zero;
    // Where a lane's row buffers and column sums leave no room for the rest
    // (16 vectors per lane at 2 waves per SIMD), the compiler spilled a few
    // registers to scratch, and each reload waited for every load in flight
    // (the prefetched row included).  The last NACCL column sums of each lane
    // live in LDS there instead; the counts are the smallest that leave these
    // instances without spills (fp32 A^T w 4; fp32 BICG and ATAX 3; fp64 ATAX 3).
    constexpr int NACCL = !(COL && WIDE && RG == 1 && V == 16 && WPE == 2 && !RANK2)
                              ? 0
                              : (DOT ? (FROMDOT || ES == 4 ? 3 : 0) : (ES == 4 ? 4 : 0));
    __shared__ vec accl[NACCL > 0 ? NACCL * THREADS : 1];
    static_assert(sizeof(xs) + sizeof(red) + sizeof(cred) + sizeof(accl) <= 160 * 1024,
                  "LDS of one workgroup above the 160 KiB of a compute unit");
    if constexpr (NACCL > 0) {
#pragma unroll
        for (int k = 0; k < NACCL; ++k)
            accl[k * THREADS + tid] = zero;
    }

    int row_end = m32;  // rows at or past this read as zeros (set before the loop)
    vec ra[B][V], rb[B][V];
    vec sa[TWO ? B : 1][V], sb[TWO ? B : 1][V];
    T wa[WTS ? B : 1], wb[WTS ? B : 1];
    T ua[RANK2 ? 2 * B : 1], ub[RANK2 ? 2 * B : 1];

    auto load_batch = [&](int blk, vec (&buf)[B][V], vec (&bbuf)[TWO ? B : 1][V],
                          T (&wbuf)[WTS ? B : 1], T (&ubuf)[RANK2 ? 2 * B : 1])
                          __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < B; ++j) {
            // first row covered by this wave in batch j, and how many of its rows exist
            const int r0 = blk * BR + j * RG + wgrp0;
            const int left = row_end - r0;
            const int nrows = left < 0 ? 0 : (left < RPW ? left : RPW);
            const uint32_t bytes = WIDE ? (nrows > 0 ? pbytes : 0u) : (uint32_t)(nrows * rowbytes);
            const T* arow = a.A + (int64_t)r0 * n + col0;
#pragma unroll
            for (int v = 0; v < V; ++v)
                buf[j][v] = load_buf<T, VW, AUX>(rsrc_v(arow, bytes, v), lane_off(v), 0);
            if constexpr (TWO) {
                const T* brow = a.B + (int64_t)r0 * n + col0;
#pragma unroll
                for (int v = 0; v < V; ++v)
                    bbuf[j][v] = load_buf<T, VW, AUX>(rsrc_v(brow, bytes, v), lane_off(v), 0);
            }
            if constexpr (WTS) {
                if constexpr (WIDE) {
                    wbuf[j] = nrows > 0 ? a.w[r0] : (T)0;
                } else {
                    const __amdgpu_buffer_rsrc_t wr = make_rsrc(a.w + r0, (uint32_t)(nrows * ES));
                    wbuf[j] = load_buf<T, 1, 0>(wr, (uint32_t)sub * ES, 0)[0];
                }
            }
            if constexpr (RANK2) {
                if constexpr (WIDE) {
                    ubuf[2 * j] = nrows > 0 ? a.u1[r0] : (T)0;
                    ubuf[2 * j + 1] = nrows > 0 ? a.u2[r0] : (T)0;
                } else {
                    const __amdgpu_buffer_rsrc_t r1 = make_rsrc(a.u1 + r0, (uint32_t)(nrows * ES));
                    const __amdgpu_buffer_rsrc_t r2 = make_rsrc(a.u2 + r0, (uint32_t)(nrows * ES));
                    ubuf[2 * j] = load_buf<T, 1, 0>(r1, (uint32_t)sub * ES, 0)[0];
                    ubuf[2 * j + 1] = load_buf<T, 1, 0>(r2, (uint32_t)sub * ES, 0)[0];
                }
            }
        }
    };

    auto process = [&](int blk, int parity, vec (&buf)[B][V], vec (&bbuf)[TWO ? B : 1][V],
                       T (&wbuf)[WTS ? B : 1], T (&ubuf)[RANK2 ? 2 * B : 1])
                       __attribute__((always_inline)) {
        T d[B], d2[TWO ? B : 1];
        // A row past the end of the matrix reads as zeros, yet its dot (0 * x)
        // or its rank-2 update (0 * v1 + 0 * v2) is NaN where that vector
        // holds an infinity, so it must add nothing to the column sums.  Only
        // a block that reaches past the last row (wave-uniform) has such rows.
        const bool tail = blk * BR + BR > row_end;
        // Instances with non-temporal loads (GEMVER's on streamed matrices;
        // the read-only modes use them at every size), row groups of 512
        // lanes or more and batches of up to 4 rows skip such rows in the
        // column sums (one row per wave: a wave-uniform test).  Besides, that
        // branch keeps the column sums in their registers: without it the
        // compiler copied them once per batch, and GEMVER's first pass ran
        // 3-7% slower on streamed matrices (the read-only modes: up to 1.3%).
        // The other ATAX and GEMVER instances zero the rows' weights or
        // elements instead: there the branch cost up to 4% (scalar spills with
        // 8-row batches, shorter rows and GEMVER's cache-resident matrices).
        // In A^T w and BICG such rows have zero weights and zero elements, and
        // add nothing either way.
        constexpr bool SKIP_PAST = WIDE && COL && G >= 512 && B <= 4 && AUX != 0;
        if constexpr (RANK2) {
            // Ahat_i = A_i + u1_i v1 + u2_i v2, in the registers that hold A_i;
            // each slice of v1 and v2 is read once for the whole batch
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const vec v1v = colvec(0, v);
                const vec v2v = colvec(1, v);
#pragma unroll
                for (int j = 0; j < B; ++j)
#pragma unroll
                    for (int e = 0; e < VW; ++e)
                        buf[j][v][e] = fma_t(ubuf[2 * j + 1], v2v[e],
                                             fma_t(ubuf[2 * j], v1v[e], buf[j][v][e]));
                if constexpr (XLDS)
                    __builtin_amdgcn_sched_barrier(0);
            }
            if (!SKIP_PAST && tail) {
                // zero the updated rows past the end (the fence keeps these
                // selects inside the branch, off the path of every other block)
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    const bool in = sub < row_end - (blk * BR + j * RG + wgrp0);
#pragma unroll
                    for (int v = 0; v < V; ++v)
#pragma unroll
                        for (int e = 0; e < VW; ++e)
                            buf[j][v][e] = in ? buf[j][v][e] : (T)0;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if constexpr (STORE) {
#pragma unroll
            for (int j = 0; j < B; ++j) {
                const int r0 = blk * BR + j * RG + wgrp0;
                const int left = row_end - r0;
                const int nrows = left < 0 ? 0 : (left < RPW ? left : RPW);
                const uint32_t bytes = WIDE ? (nrows > 0 ? pbytes : 0u) : (uint32_t)(nrows * rowbytes);
                T* orow = a.Aout + (int64_t)r0 * n + col0;
#pragma unroll
                for (int v = 0; v < V; ++v)
                    store_buf<T, VW, AUX>(buf[j][v], rsrc_v(orow, bytes, v), lane_off(v));
            }
        }
        if constexpr (DOT) {
#pragma unroll
            for (int j = 0; j < B; ++j) {
                T s = 0, s2 = 0;
#pragma unroll
                for (int v = 0; v < V; ++v) {
                    const vec xx = colvec(0, v);
#pragma unroll
                    for (int e = 0; e < VW; ++e) {
                        s = fma_t(buf[j][v][e], xx[e], s);
                        if constexpr (TWO)
                            s2 = fma_t(bbuf[j][v][e], xx[e], s2);
                    }
                    // keep each LDS read of x next to its use: hoisting all of
                    // them would hold the whole slice in registers at once
                    if constexpr (XLDS)
                        __builtin_amdgcn_sched_barrier(0);
                }
                d[j] = s;
                if constexpr (TWO)
                    d2[j] = s2;
            }
            if constexpr (G <= 64) {
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    d[j] = group_sum<G>(d[j]);
                    if constexpr (TWO)
                        d2[j] = group_sum<G>(d2[j]);
                }
            } else {
                static_assert(RG == 1, "a row group wider than a wave spans the whole workgroup");
                const int wig = wave;  // wave index inside the row group
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    d[j] = group_sum<64>(d[j]);
                    if constexpr (TWO)
                        d2[j] = group_sum<64>(d2[j]);
                }
                if (lane == 0) {
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        red[parity][j * WPG + wig] = d[j];
                        if constexpr (TWO)
                            red[parity][(B + j) * WPG + wig] = d2[j];
                    }
                }
                lds_barrier();
                // The table holds NROW rows of WPG wave partials.
                constexpr int NROW = NDOT * B;
                if constexpr (NROW * WPG <= 16 && WPE <= 2) {
                    // small table and a large register budget: every lane adds
                    // each row's partials in wave order
#pragma unroll
                    for (int j = 0; j < B; ++j) {
                        T s = 0, s2 = 0;
#pragma unroll
                        for (int w = 0; w < WPG; ++w) {
                            s += red[parity][j * WPG + w];
                            if constexpr (TWO)
                                s2 += red[parity][(B + j) * WPG + w];
                        }
                        d[j] = s;
                        if constexpr (TWO)
                            d2[j] = s2;
                    }
                } else {
                    // larger tables: lane l of every wave takes entry l (and
                    // l + 64, ...), a butterfly over each aligned group of WPG
                    // lanes adds one row's partials, and the row totals are
                    // read back as wave-uniform values.  One LDS read per lane
                    // instead of NROW * WPG reads and as many live registers,
                    // which made the 8-row batches of 512 and 1024-lane groups
                    // spill.
                    constexpr int NCH = (NROW * WPG + 63) / 64;
                    T part[NCH];
#pragma unroll
                    for (int ch = 0; ch < NCH; ++ch) {
                        const int i = ch * 64 + lane;
                        part[ch] = i < NROW * WPG ? red[parity][i] : (T)0;
                        part[ch] = group_sum<WPG>(part[ch]);
                    }
#pragma unroll
                    for (int k = 0; k < NROW; ++k) {
                        const T tot = lanes_apply(part[k * WPG / 64], [&](int x) {
                            return __builtin_amdgcn_readlane(x, (k * WPG) % 64);
                        });
                        if (k < B)
                            d[k] = tot;
                        else if constexpr (TWO)
                            d2[k - B] = tot;
                    }
                }
            }
            if (g == 0) {
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    const int row = blk * BR + j * RG + tid / G;
                    if (row < m32) {
                        if (multipanel) {
                            a.dotpart[(int64_t)by * m + row] = d[j];
                            if constexpr (TWO)
                                a.dotpart2[(int64_t)by * m + row] = d2[j];
                        } else if constexpr (TWO) {
                            a.rowout[row] = fma_t(a.alpha, d[j], a.beta * d2[j]);
                        } else if (a.rowout != nullptr) {
                            a.rowout[row] = a.scale_rows ? a.alpha * d[j] : d[j];
                        }
                    }
                }
            }
            if (FROMDOT && !SKIP_PAST && tail) {
                // zero the weight of the rows past the end (fenced into the
                // branch like the rank-2 rows above)
#pragma unroll
                for (int j = 0; j < B; ++j) {
                    if (sub >= row_end - (blk * BR + j * RG + wgrp0))
                        d[j] = (T)0;
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if constexpr (COL) {
#pragma unroll
            for (int j = 0; j < B; ++j) {
                if constexpr (SKIP_PAST) {
                    if (blk * BR + j * RG + wgrp0 >= row_end)
                        continue;
                }
                T s;
                if constexpr (FROMDOT)
                    s = d[j];
                else
                    s = wbuf[j];
#pragma unroll
                for (int v = 0; v < V - NACCL; ++v)
#pragma unroll
                    for (int e = 0; e < VW; ++e)
                        acc[v][e] = fma_t(s, buf[j][v][e], acc[v][e]);
                if constexpr (NACCL > 0) {
#pragma unroll
                    for (int k = 0; k < NACCL; ++k) {
                        vec t = accl[k * THREADS + tid];
#pragma unroll
                        for (int e = 0; e < VW; ++e)
                            t[e] = fma_t(s, buf[j][V - NACCL + k][e], t[e]);
                        accl[k * THREADS + tid] = t;
                    }
                }
            }
        }
        (void)parity;
    };

    // Row blocks of this workgroup, one per round r (nbx = gridDim.y):
    // - cyclic (map 0): block bx + r * nbx;
    // - blocked (map 1): one contiguous run of blocks;
    // - rotated (map 2): round r covers the same window of nbx blocks as the
    //   cyclic map, dealt to the workgroups shifted by r * kRotStride, so that
    //   no workgroup, and no XCD, reads the same position of every window; in
    //   the last round some workgroups may get a block past the matrix.
    // The round count is uniform across the workgroup, so the barriers inside
    // are too.  The next block is always prefetched: past the last row of the
    // matrix (or of a blocked run) its resources are empty, so those loads
    // return zeros without touching memory, and such a block adds nothing.
    // The scheduling fences keep each refill after the previous use of its
    // buffer, so no more than two batches are ever live.
    const int nblk = (int)((m + BR - 1) / BR);
    const int map = a.blocked;
    int blk0, bstep, bend;
    if (map == 1) {
        const int per = (nblk + nbx - 1) / nbx;
        blk0 = bx * per;
        bstep = 1;
        bend = blk0 + per < nblk ? blk0 + per : nblk;
    } else {
        blk0 = bx;
        bstep = nbx;
        bend = nblk;
    }
    const int rounds =
        map == 2 ? (nblk + nbx - 1) / nbx : (blk0 < bend ? (bend - blk0 + bstep - 1) / bstep : 0);
    row_end = map == 2 ? m32 : (bend * BR < m32 ? bend * BR : m32);
    auto block_of = [&](int r) __attribute__((always_inline)) -> int {
        if (map == 2) {
            const unsigned un = (unsigned)nbx;
            const int shift = (int)(((unsigned)r % un) * ((unsigned)kRotStride % un) % un);
            const int pos = bx + shift;
            return r * nbx + (pos < nbx ? pos : pos - nbx);
        }
        return blk0 + r * bstep;
    };
    // the first batch goes out before the column vectors: those come from L2
    // (every workgroup reads the same slice), the matrix from HBM
    if (rounds > 0)
        load_batch(block_of(0), ra, sa, wa, ua);
    if constexpr (NXV > 0) {
#pragma unroll
        for (int k = 0; k < NXV; ++k) {
            const T* src = DOT ? a.x : (k == 0 ? a.v1 : a.v2);
            const __amdgpu_buffer_rsrc_t xr = make_rsrc(src + col0, pbytes);
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int64_t c = (int64_t)(v * G + g) * VW;
                vec t = load_buf<T, VW, 0>(xr, c < PW ? (uint32_t)(c * ES) : kOutOfRange, 0);
                if constexpr (XLDS)
                    xs[(k * V + v) * THREADS + tid] = t;
                else
                    xv[k * V + v] = t;
            }
        }
    }

    if (rounds > 0) {
        int r = 0;
        for (;;) {
            load_batch(block_of(r + 1), rb, sb, wb, ub);
            __builtin_amdgcn_sched_barrier(0);
            process(block_of(r), 0, ra, sa, wa, ua);
            __builtin_amdgcn_sched_barrier(0);
            if (++r >= rounds)
                break;
            load_batch(block_of(r + 1), ra, sa, wa, ua);
            __builtin_amdgcn_sched_barrier(0);
            process(block_of(r), 1, rb, sb, wb, ub);
            __builtin_amdgcn_sched_barrier(0);
            if (++r >= rounds)
                break;
        }
    }

    if constexpr (COL) {
        T* out = a.colpart + (int64_t)bx * a.ldp + col0;
        if constexpr (NACCL > 0) {
#pragma unroll
            for (int k = 0; k < NACCL; ++k)
                acc[V - NACCL + k] = accl[k * THREADS + tid];
        }
        if constexpr (RG == 1) {
#pragma unroll
            for (int v = 0; v < V; ++v) {
                const int64_t c = (int64_t)(v * G + g) * VW;
                // fp32: written through (5% off the cache-resident BICG 4096^2
                // step); fp64 keeps non-temporal stores, with which the
                // 16384-wide kernel's registers fit (write-through: 20% slower)
                if (c < pcols) {
                    if constexpr (sizeof(T) == 4)
                        store_buf<T, VW, kWriteThrough>(acc[v], make_rsrc(out, (uint32_t)(pcols * sizeof(T))),
                                                        (uint32_t)(c * sizeof(T)));
                    else
                        store_vec_nt<T, VW>(out + c, acc[v]);
                }
            }
        } else {
            // row groups of one wave first (butterfly over the lane bits above G) ...
#pragma unroll
            for (int v = 0; v < V; ++v)
#pragma unroll
                for (int e = 0; e < VW; ++e) {
                    T t = acc[v][e];
#pragma unroll
                    for (int mask = G; mask < 64; mask <<= 1)
                        t += __shfl_xor(t, mask, 64);
                    acc[v][e] = t;
                }
            if (lane < G) {
#pragma unroll
                for (int v = 0; v < V; ++v)
                    cred[(wave * G + g) * V + v] = acc[v];
            }
            lds_barrier();
            // ... then the waves, in ascending order
            for (int s = tid; s < G * V; s += THREADS) {
                const int gg = s / V, vv = s % V;
                vec t = cred[gg * V + vv];
#pragma unroll
                for (int w = 1; w < NWAVES; ++w)
                    t += cred[(w * G + gg) * V + vv];
                const int64_t c = (int64_t)(vv * G + gg) * VW;
                // written through: 2.3% off a 2^20 x 64 A^T w step
                if (c < pcols)
                    store_buf<T, VW, kWriteThrough>(t, make_rsrc(out, (uint32_t)(pcols * sizeof(T))),
                                                    (uint32_t)(c * sizeof(T)));
            }
        }
    }
}

// Epilogues of the column reduction.
enum : int {
    EPI_SCALE = 0,  // out = alpha * sum(P)            (alpha = 1: the plain sum)
    EPI_TWO = 1,    // out = alpha * sum(P) + beta * sum(Q)
    EPI_ADDVEC = 2  // out = alpha * sum(P) + Q[j]     (Q a vector of ncols)
};

// out[j] = sum_{b < nrows} P[b * ldp + j] for j < ncols, rows summed in a fixed
// order: SL = THREADS / 16 slices of rows (slice s takes rows s, s + SL, ...,
// sixteen of them per step with their loads issued together, missing rows
// read as zero), then the slices by a fixed pairwise tree in LDS; then the
// epilogue EPI.  Narrow outputs use 1024 threads, so that many partial rows
// still take one round of loads.
template <typename T, int VW, int EPI, int THREADS = 256>
__global__ void __launch_bounds__(THREADS)
k_colreduce(const T* __restrict__ P, const T* __restrict__ Q, int64_t ldp, int64_t nrows,
            int64_t ncols, T alpha, T beta, T* __restrict__ out)
{
    constexpr bool TWO = EPI == EPI_TWO;
    typedef typename VecOf<T, VW>::type vec;
    constexpr int CV = 16;
    constexpr int SL = THREADS / CV;
    constexpr int U = 16;
    __shared__ vec rp[SL][CV];
    __shared__ vec rq[TWO ? SL : 1][CV];
    const int tid = threadIdx.x;
    const int cv = tid % CV;
    const int sl = tid / CV;
    const int64_t col = ((int64_t)blockIdx.x * CV + cv) * VW;
    const bool ok = col < ncols;
    const vec zero = (vec)(T)0;
    vec s = zero, s2 = zero;
    if (ok) {
        for (int64_t b0 = sl; b0 < nrows; b0 += (int64_t)U * SL) {
            vec t[U], t2[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int64_t r = b0 + (int64_t)u * SL;
                t[u] = r < nrows ? load_vec<T, VW>(P + r * ldp + col) : zero;
                if constexpr (TWO)
                    t2[u] = r < nrows ? load_vec<T, VW>(Q + r * ldp + col) : zero;
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                s += t[u];
                if constexpr (TWO)
                    s2 += t2[u];
            }
        }
    }
    rp[sl][cv] = s;
    if constexpr (TWO)
        rq[sl][cv] = s2;
    lds_barrier();
#pragma unroll
    for (int stride = SL / 2; stride >= 1; stride >>= 1) {
        if (sl < stride) {
            rp[sl][cv] += rp[sl + stride][cv];
            if constexpr (TWO)
                rq[sl][cv] += rq[sl + stride][cv];
        }
        lds_barrier();
    }
    if (sl == 0 && ok) {
        vec t = rp[0][cv];
        if constexpr (EPI == EPI_TWO) {
            const vec t2 = rq[0][cv];
#pragma unroll
            for (int e = 0; e < VW; ++e)
                t[e] = fma_t(alpha, t[e], beta * t2[e]);
        } else if constexpr (EPI == EPI_ADDVEC) {
            const vec z = load_vec<T, VW>(Q + col);
#pragma unroll
            for (int e = 0; e < VW; ++e)
                t[e] = fma_t(alpha, t[e], z[e]);
        } else {
#pragma unroll
            for (int e = 0; e < VW; ++e)
                t[e] = alpha * t[e];
        }
        store_vec<T, VW>(out + col, t);
    }
}

// Zero-fill of count elements (outputs of empty sums).
template <typename T>
__global__ void __launch_bounds__(256) k_fill_zero(T* __restrict__ p, int64_t count)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count;
         i += (int64_t)gridDim.x * 256)
        p[i] = (T)0;
}

}  // namespace mep
