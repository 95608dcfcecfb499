// Kernels of the two streaming samples of the APP SDK table (Table 3):
// the sum of a vector ("reduction") and the elementwise sum of two vectors
// ("vectoradd").  Kept apart from the matrix kernels so that each family's
// source can be stamped on its own measurements.
#pragma once

#include "mep_kernels.hpp"

namespace mep {

// Sum of a vector, first stage: workgroup b adds the 16-byte vectors of its
// own contiguous chunk (lanes stride by 256 vectors, four loads in flight per
// lane, non-temporal), then its lanes (butterfly) and its four waves
// (ascending) into partial[b].  The trailing n mod VW elements are added by
// the first lanes of workgroup 0.  The order depends only on n and
// gridDim.x, so the result is reproducible; k_colreduce with one column adds
// the partials.
template <typename T, int VW>
__global__ void __launch_bounds__(256)
k_reduce_sum(const T* __restrict__ x, int64_t n, T* __restrict__ partial)
{
    typedef typename VecOf<T, VW>::type vec;
    constexpr int U = 4;
    const vec* xv = reinterpret_cast<const vec*>(x);
    const int64_t nv = n / VW;
    const int64_t chunk = (nv + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = (int64_t)blockIdx.x * chunk;
    const int64_t b1 = b0 + chunk < nv ? b0 + chunk : nv;
    int64_t i = b0 + threadIdx.x;
    vec acc = (vec)(T)0;
    for (; i + (U - 1) * 256 < b1; i += U * 256) {
        vec t[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            t[u] = __builtin_nontemporal_load(xv + i + u * 256);
#pragma unroll
        for (int u = 0; u < U; ++u)
            acc += t[u];
    }
    for (; i < b1; i += 256)
        acc += __builtin_nontemporal_load(xv + i);
    T s = 0;
#pragma unroll
    for (int e = 0; e < VW; ++e)
        s += acc[e];
    if (blockIdx.x == 0 && (int64_t)threadIdx.x < n - nv * VW)
        s += x[nv * VW + threadIdx.x];
    s = group_sum<64>(s);
    __shared__ T red[4];
    if ((threadIdx.x & 63) == 0)
        red[threadIdx.x >> 6] = s;
    lds_barrier();
    if (threadIdx.x == 0)
        partial[blockIdx.x] = ((red[0] + red[1]) + red[2]) + red[3];
}

// c = a + b elementwise: workgroup b handles its own contiguous chunk of
// 16-byte vectors (lanes stride by 256 vectors, four in flight per lane),
// with non-temporal loads and stores; the trailing n mod VW elements by
// workgroup 0.
template <typename T, int VW>
__global__ void __launch_bounds__(256)
k_vector_add(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ c, int64_t n)
{
    typedef typename VecOf<T, VW>::type vec;
    constexpr int U = 4;
    const vec* av = reinterpret_cast<const vec*>(a);
    const vec* bv = reinterpret_cast<const vec*>(b);
    vec* cv = reinterpret_cast<vec*>(c);
    const int64_t nv = n / VW;
    const int64_t chunk = (nv + gridDim.x - 1) / gridDim.x;
    const int64_t b0 = (int64_t)blockIdx.x * chunk;
    const int64_t b1 = b0 + chunk < nv ? b0 + chunk : nv;
    int64_t i = b0 + threadIdx.x;
    for (; i + (U - 1) * 256 < b1; i += U * 256) {
        vec ta[U], tb[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            ta[u] = __builtin_nontemporal_load(av + i + u * 256);
            tb[u] = __builtin_nontemporal_load(bv + i + u * 256);
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            __builtin_nontemporal_store(ta[u] + tb[u], cv + i + u * 256);
    }
    for (; i < b1; i += 256)
        __builtin_nontemporal_store(__builtin_nontemporal_load(av + i) + __builtin_nontemporal_load(bv + i),
                                    cv + i);
    if (blockIdx.x == 0 && (int64_t)threadIdx.x < n - nv * VW) {
        const int64_t k = nv * VW + threadIdx.x;
        c[k] = a[k] + b[k];
    }
}

// c = a + b, row-streamed: the vectors are read as rows of THREADS * V
// 16-byte vectors (64 KiB of each input for 1024 x 4); workgroup w takes rows
// w, w + gridDim.x, ..., so the grid sweeps one contiguous window at a time,
// and the next row of a and b is loaded while the current one is added and
// stored.  Every access is guarded by the vector count; the trailing n mod VW
// elements go to the first lanes of workgroup 0.
template <typename T, int VW, int V, int THREADS>
__global__ void __launch_bounds__(THREADS)
k_vector_add_rows(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ c, int64_t n)
{
    typedef typename VecOf<T, VW>::type vec;
    const vec* av = reinterpret_cast<const vec*>(a);
    const vec* bv = reinterpret_cast<const vec*>(b);
    vec* cv = reinterpret_cast<vec*>(c);
    const int64_t nv = n / VW;
    constexpr int64_t RV = (int64_t)THREADS * V;
    const int64_t rows = (nv + RV - 1) / RV;
    const int tid = threadIdx.x;
    const vec zero = (vec)(T)0;
    vec xa[V], xb[V], ya[V], yb[V];
    auto load = [&](int64_t r, vec (&pa)[V], vec (&pb)[V]) __attribute__((always_inline)) {
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int64_t i = r * RV + (int64_t)v * THREADS + tid;
            pa[v] = i < nv ? __builtin_nontemporal_load(av + i) : zero;
            pb[v] = i < nv ? __builtin_nontemporal_load(bv + i) : zero;
        }
    };
    auto store = [&](int64_t r, vec (&pa)[V], vec (&pb)[V]) __attribute__((always_inline)) {
#pragma unroll
        for (int v = 0; v < V; ++v) {
            const int64_t i = r * RV + (int64_t)v * THREADS + tid;
            if (i < nv)
                __builtin_nontemporal_store(pa[v] + pb[v], cv + i);
        }
    };
    const int64_t step = gridDim.x;
    int64_t r = blockIdx.x;
    if (r < rows)
        load(r, xa, xb);
    while (r < rows) {
        load(r + step, ya, yb);
        store(r, xa, xb);
        r += step;
        if (r >= rows)
            break;
        load(r + step, xa, xb);
        store(r, ya, yb);
        r += step;
    }
    if (blockIdx.x == 0 && (int64_t)tid < n - nv * VW) {
        const int64_t k = nv * VW + tid;
        c[k] = a[k] + b[k];
    }
}

// c = a + b, row-streamed through buffer resources: as k_vector_add_rows
// (rows of THREADS * V vectors of each input, row w, w + gridDim.x, ... per
// workgroup, the next row loaded while the current one is added and stored),
// but every access is a non-temporal buffer load or store through a
// resource whose base is the row's first element and whose size is what is
// left of the vector: one 32-bit offset per lane, the range check drops the
// ragged end, and the prefetch past the last row reads nothing.
template <typename T, int VW, int V, int THREADS>
__global__ void __launch_bounds__(THREADS)
k_vector_add_buf(const T* __restrict__ a, const T* __restrict__ b, T* __restrict__ c, int64_t n)
{
    typedef typename VecOf<T, VW>::type vec;
    constexpr int64_t RE = (int64_t)THREADS * V * VW;  // elements per row
    constexpr uint32_t VB = VW * sizeof(T);
    const int64_t nv = n / VW;
    const int64_t ne = nv * VW;  // elements covered by whole vectors
    const int64_t rows = (ne + RE - 1) / RE;
    const int tid = threadIdx.x;
    vec xa[V], xb[V], ya[V], yb[V];
    auto rsrc = [&](const T* base, int64_t r) __attribute__((always_inline)) {
        const int64_t left = r < rows ? (ne - r * RE) * (int64_t)sizeof(T) : 0;
        return make_rsrc(base + (r < rows ? r * RE : 0),
                         (uint32_t)(left < RE * (int64_t)sizeof(T) ? left : RE * (int64_t)sizeof(T)));
    };
    auto load = [&](int64_t r, vec (&pa)[V], vec (&pb)[V]) __attribute__((always_inline)) {
        const __amdgpu_buffer_rsrc_t ra = rsrc(a, r), rb = rsrc(b, r);
#pragma unroll
        for (int k = 0; k < V; ++k) {
            const uint32_t off = (uint32_t)(k * THREADS + tid) * VB;
            pa[k] = load_buf<T, VW, 2>(ra, off, 0);
            pb[k] = load_buf<T, VW, 2>(rb, off, 0);
        }
    };
    auto store = [&](int64_t r, vec (&pa)[V], vec (&pb)[V]) __attribute__((always_inline)) {
        const __amdgpu_buffer_rsrc_t rc = rsrc(c, r);
#pragma unroll
        for (int k = 0; k < V; ++k)
            store_buf<T, VW, 2>(pa[k] + pb[k], rc, (uint32_t)(k * THREADS + tid) * VB);
    };
    const int64_t step = gridDim.x;
    int64_t r = blockIdx.x;
    if (r < rows)
        load(r, xa, xb);
    while (r < rows) {
        load(r + step, ya, yb);
        store(r, xa, xb);
        r += step;
        if (r >= rows)
            break;
        load(r + step, xa, xb);
        store(r, ya, yb);
        r += step;
    }
    if (blockIdx.x == 0 && (int64_t)tid < n - ne) {
        const int64_t k = ne + tid;
        c[k] = a[k] + b[k];
    }
}

}  // namespace mep
