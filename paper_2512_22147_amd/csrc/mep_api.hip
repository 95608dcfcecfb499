// C-ABI of libmep.so (include/mep.h): argument checks, planning, launch
// sequences of the matrix-vector operations and the minimal-executable-
// program harness (trimmed-mean timing of Eq. 3, functional-equivalence
// check of Eq. 4, candidate selection for Eqs. 4-5).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <mutex>
#include <string>
#include <vector>

#include "mep.h"
#include "mep_internal.hpp"

namespace mep {

// ---------------------------------------------------------------------------
// errors
// ---------------------------------------------------------------------------

static thread_local std::string g_last_error;

static int fail(int code, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

static int hip_fail(hipError_t e, const char* what)
{
    return fail(MEP_EHIP, "%s: %s", what, hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// planning
// ---------------------------------------------------------------------------

constexpr int64_t kMaxDim = int64_t(1) << 30;
constexpr int64_t kMaxRow = int64_t(65535) * 8192;

static int esize_of(int dtype) { return dtype == MEP_F32 ? 4 : (dtype == MEP_F64 ? 8 : 0); }

// The default shape for a row of nv vectors, from candidate sweeps on MI355X
// (every operation, both element types, two machines, rows of 1-8192 vectors,
// matrices of 64 MiB that stay in the 256 MB Infinity Cache across calls and
// of 1 GiB that stream from HBM).  What decides the shape is how much of each
// row group holds data and how many bytes every compute unit keeps in
// flight: the narrowest group that holds the row, except that rows filling
// it (about 7/8 and more) often run faster on the next wider shape.
// Non-temporal loads are the faster default for both matrix sizes (each
// candidate timed after a 1 GiB write that clears the caches: a
// non-temporal shape timed right after a cached-load one inherits its cache
// state and reads 5-17% slower); the cache-resident exceptions are noted
// where they are taken.
static Cfg preferred_shape(int mode, int esize, int64_t m, int64_t n, int64_t nv)
{
    const bool two = (mode & F_TWO) != 0;
    const bool col = (mode & F_COL) != 0;
    const bool mv = mode == MODE_MV;
    const bool atw = mode == MODE_ATW;
    const bool bicg = mode == MODE_BICG;
    const bool atax = (mode & F_FROMDOT) != 0;
    const int64_t mats = two ? 2 : 1;
    const bool stream = mats * m * n * esize > (int64_t(128) << 20);
    // load policy of rows of <= 256 vectors: non-temporal, except for
    // GEMVER's first pass (it also stores Ahat) on a cache-resident matrix
    const int naux = (mode & F_STORE) && !stream ? 0 : 2;
    // rows of <= 8 vectors: as many lanes per row as the row has vectors
    // (2, 4 or 8; a wider group leaves most lanes idle: 2.4-4.3 instead of
    // 5.7-6.6 TB/s for 1 GiB of 12- and 16-element fp32 rows)
    if (nv <= 8) {
        // rows of one vector of a cache-resident matrix: cached loads (3-10%
        // faster for y = A x, A^T w and BICG).  Otherwise BICG takes 4-row
        // batches: its 8-row batches spill registers in fp64 (1 GiB of 4- and
        // 8-vector fp64 rows: 25% faster; fp32 up to 2%)
        const int g = nv <= 2 ? 2 : (nv <= 4 ? 4 : 8);
        if (bicg && (nv > 1 || stream))
            return Cfg{g, 1, 4, 4, 2};
        const int aux1 = nv == 1 && !stream && !atax && !two ? 0 : naux;
        return Cfg{g, 1, 8, 4, aux1};
    }
    // rows of <= 16 vectors: 16 compute units per XCD (512 workgroups) halve
    // the partial rows the single-workgroup column reduce adds (the step is
    // ~4% faster for 2^20 x 64, the streaming kernel ~2% slower); BICG takes
    // 4-row batches (fp64: 8-row batches spill, 5.6 instead of 3.4 TB/s)
    if (nv <= 16)
        return bicg ? Cfg{16, 1, 4, 4, 2} : Cfg{16, 1, 8, 4, naux, 0, 16};
    if (nv <= 64)
        return Cfg{64, 1, 8, 4, naux};
    // 65-128 vectors: 2 vectors per lane.  A^T w and ATAX of streamed rows
    // that fill more than 7/8 of them take 4 with half the rows per batch (a
    // few % faster there; the same shape is 13-15% slower for 80-vector
    // rows), and so does GEMVER's first pass
    if (nv <= 128) {
        if ((mode & F_STORE) || ((atw || atax) && stream && nv > 112))
            return Cfg{64, 4, 2, 4, naux};
        return Cfg{64, 2, 4, 4, 2};
    }
    if (nv <= 256)
        return Cfg{64, 4, 2, 4, naux};
    // the rank-2 update that stores Ahat (GEMVER's first pass), from sweeps
    // with cleared caches: streamed rows of up to 7/8 of 1024 vectors on
    // 256 x 4 x 2 (fp32 rows of 449-512 vectors on 512 x 2 x 8), fuller ones
    // on 512 x 4 x 4 (fp64: 512 x 2 x 8), 1025-2048 vectors on 512 x 4 x 4,
    // 1024 x 4 x 2 beyond; cache-resident (cached loads) 256 x 4 x 2 up to 352
    // vectors, 512 x 2 x 8 up to 1024, then as streamed
    if (mode & F_STORE) {
        const int aux = stream ? 2 : 0;
        if (nv <= 512) {
            if (stream)
                return esize == 8 || nv <= 448 ? Cfg{256, 4, 2, 4, 2} : Cfg{512, 2, 8, 2, 2};
            return nv <= 352 ? Cfg{256, 4, 2, 4, 0} : Cfg{512, 2, 8, 2, 0};
        }
        if (nv <= 1024) {
            if (!stream)
                return Cfg{512, 2, 8, 2, 0};
            if (nv < 896)
                return Cfg{256, 4, 2, 4, 2};
            return esize == 8 ? Cfg{512, 2, 8, 2, 2} : Cfg{512, 4, 4, 2, 2};
        }
        if (nv <= 2048)
            return Cfg{512, 4, 4, 2, aux};
        return Cfg{1024, 4, 2, 4, aux};
    }
    // 257-512 vectors: 512-vector shapes (the 1024-vector ones left a row of
    // 320 vectors 15-30% slower): y = A x and GESUMMV of cache-resident
    // matrices on 256-lane groups, the rest on 512 lanes x 1 vector with
    // 8-row batches.  Rows past 3/4 of the group go to the 1024-vector
    // shapes; cache-resident ATAX and fp32 BICG only past 7/8,
    // fp64 BICG (the most registers per row) never, and streamed fp64 BICG
    // rows up to 3/4 run 2-12% faster on 256 x 2 x 4.
    if (nv <= 512) {
        if (bicg && esize == 8)
            return stream && nv <= 384 ? Cfg{256, 2, 4, 4, 2} : Cfg{512, 1, 8, 4, 2};
        if (!stream && (mv || two))
            return Cfg{256, 2, 4, 4, 2};
        if (nv <= 384 || (nv <= 448 && (bicg || (atax && !stream))))
            return Cfg{512, 1, 8, 4, 2};
        if (atw || bicg || (atax && !stream) || (two && esize == 4))
            return Cfg{512, 2, 8, 2, 2};
        return Cfg{512, 2, 4, 4, 2};
    }
    // 513-1024 vectors: 512 lanes x 2 vectors, 8-row batches; y = A x and
    // GESUMMV of cache-resident matrices on 256 x 4 (10-20% faster).
    // Streamed: A^T w, and the other modes for rows that fill the group 7/8
    // or more, on 24 compute units per XCD (2-4% faster), except BICG (fp32
    // rows past 7/8: 512 x 4 x 4), GESUMMV past 7/8 and y = A x from 7/8 to
    // 15/16 (512 x 4 x 4).
    if (nv <= 1024) {
        if (!stream)
            return mv || two ? Cfg{256, 4, 2, 4, 2} : Cfg{512, 2, 8, 2, 2};
        if (bicg)
            return esize == 4 && nv > 896 ? Cfg{512, 4, 4, 2, 2} : Cfg{512, 2, 8, 2, 2};
        if (nv >= 896 && (two || (mv && nv <= 960)))
            return Cfg{512, 4, 4, 2, 2};
        return atw || nv >= 896 ? Cfg{512, 2, 8, 2, 2, 0, 24} : Cfg{512, 2, 8, 2, 2};
    }
    // 1025-2048 vectors: 512 lanes x 4 vectors, 4-row batches; streamed on 24
    // compute units per XCD (2-7% faster; BICG from 1408 vectors on; A^T w
    // and GESUMMV of full rows on 512 x 8 x 2).  Cache-resident A^T w, and BICG and ATAX
    // above 1664 vectors, read cached (the only place where cached loads are
    // measurably faster).
    if (nv <= 2048) {
        if (!stream) {
            if (mv || two)
                return Cfg{512, 4, 4, 2, 2};
            return Cfg{512, 4, 4, 2, atw || nv > 1664 ? 0 : 2};
        }
        if ((atw || two) && nv > 1920)
            return Cfg{512, 8, 2, 2, 2};
        if (bicg && nv <= 1408)
            return Cfg{512, 4, 4, 2, 2};
        return Cfg{512, 4, 4, 2, 2, 0, 24};
    }
    // Longer rows (4096- and 8192-vector shapes).  Streamed, one matrix:
    // rows of 2049-4096 vectors on 24 compute units per XCD (ATAX rows past
    // 7/8 of the group on 22; BICG only past 11/16), 8192-vector rows past
    // 11/16 on 26, A^T w on 26
    // then 24 (3-7% faster than all 32 wherever the row is longer than 2048
    // vectors).  Two matrices (half the rows per batch, 4096-vector column
    // panels beyond): streamed on 24 up to 4096 vectors, cache-resident on 24
    // past them.  Cache-resident: the column-sum modes read cached; y = A x of
    // rows short of 8192 vectors on 1024 x 8 x 1 at 4 waves per SIMD (4-9%).
    // Rows cut into column panels (past 8192 vectors) use every compute unit.
    const int laux = stream || !col ? 2 : 0;
    const bool panelled = nv > 8192;
    if (two) {
        const int cux = !panelled && (stream ? nv <= 4096 : nv > 4096) ? 24 : kCusPerXcd;
        return Cfg{512, 8, 2, 2, 2, 0, cux};
    }
    if (nv <= 4096) {
        // streamed fp32 rows past 2816 vectors: the rotated block map on 24
        // compute units per XCD.  With the cyclic map each workgroup reads the
        // same position of every window of blocks, and some positions stream
        // slower than others, so a few workgroups end their rows well after
        // the rest; rotating the positions evens them out (1-3% faster for
        // y = A x, A^T w, BICG and ATAX at 12200-16384 columns, up to 7% for
        // ATAX; neutral at 10000 columns, 0.5-1% slower at 8400)
        if (stream && esize == 4 && nv > 2816)
            return Cfg{512, 8, 2, 2, 2, 2, 24};
        const int cux = !stream || (bicg && nv <= 2816) ? kCusPerXcd : (atax && nv > 3584 ? 22 : 24);
        return Cfg{512, 8, 2, 2, laux, 0, cux};
    }
    if (!stream)
        return mv && nv <= 7680 ? Cfg{1024, 8, 1, 4, 2} : Cfg{512, 16, 1, 2, laux};
    // streamed fp64 ATAX rows past 11/16: the rotated map on 26 (1% faster at
    // 16384 columns, 5% at 13000, within 0.5% at 12000 and 14000)
    if (atax && esize == 8 && !panelled && nv > 5632)
        return Cfg{512, 16, 1, 2, 2, 2, 26};
    const int64_t narrow_from = bicg && esize == 8 ? 6656 : 5632;  // fp64 BICG: past 13/16
    const int cux = panelled ? kCusPerXcd : (atw ? (nv <= 5632 ? 26 : 24) : (nv > narrow_from ? 26 : kCusPerXcd));
    return Cfg{512, 16, 1, 2, 2, 0, cux};
}

// The default of the element-wise path: the narrowest row group that holds
// the row, with 16 elements per lane in flight for fp32 and 8 for fp64 (64
// bytes either way).  Measured exceptions (cleared caches before each
// candidate): fp64 rows longer than 128 elements of a streamed matrix, and
// fp64 BICG rows longer than 1024, take 16 (4-22% faster); fp32 rows that
// fill more than 7/8 of a 256- or 1024-lane group take 8, except BICG (2-9%).
static Cfg preferred_scalar_shape(int mode, int esize, int64_t m, int64_t n)
{
    const bool bicg = mode == MODE_BICG;
    const bool stream = ((mode & F_TWO) ? 2 : 1) * m * n * esize > (int64_t(128) << 20);
    int per_lane = esize == 4 ? 16 : 8;
    if (esize == 8 && ((stream && n > 128) || (bicg && n > 1024)))
        per_lane = 16;
    const int64_t cap = n <= 512 ? 512 : (n <= 1024 ? 1024 : 8192);  // G x V of the shapes below
    if (esize == 4 && !bicg && n > 256 && n <= 8192 && 8 * n > 7 * cap)
        per_lane = 8;
    if (n <= 64) {
        const int g = n <= 8 ? 8 : (n <= 16 ? 16 : (n <= 32 ? 32 : 64));
        return Cfg{g, 1, per_lane, 4, 2};
    }
    if (n <= 128)
        return Cfg{64, 2, per_lane / 2, 4, 2};
    if (n <= 256)
        return Cfg{64, 4, per_lane / 4, 4, 2};
    if (n <= 512)
        return Cfg{256, 2, per_lane / 2, 4, 2};
    if (n <= 1024)
        return Cfg{256, 4, per_lane / 4, 4, 2};
    return Cfg{1024, 8, per_lane / 8, 4, 2};
}

static bool same_cfg(const Cfg& a, const Cfg& b)
{
    return a.G == b.G && a.V == b.V && a.B == b.B && a.WPE == b.WPE && a.AUX == b.AUX && a.MAP == b.MAP &&
           a.CUX == b.CUX;
}

int stream_candidates(int esize, bool vec, int mode, int64_t m, int64_t n, int* idx)
{
    const int vw = vec ? 16 / esize : 1;
    const int vgpr32 = vec ? 4 : esize / 4;
    const Cfg* tab = vec ? kVecCfg : kScalarCfg;
    const int nt = vec ? kNumVecCfg : kNumScalarCfg;
    const int64_t nv = (n + vw - 1) / vw;
    int cnt = 0;
    int64_t first_cap = -1;
    // shapes that hold a whole row, narrowest first; much wider ones only idle lanes
    for (int i = 0; i < nt && cnt < 16; ++i) {
        const Cfg c = tab[i];
        const int64_t cap = (int64_t)c.G * c.V;
        if (!cfg_fits(c, mode, vgpr32) || cap < nv)
            continue;
        if (first_cap < 0)
            first_cap = cap;
        if (cap > 4 * first_cap)
            continue;
        idx[cnt++] = i;
    }
    if (cnt == 0) {
        // rows longer than any shape: the widest shapes, over column panels
        int64_t best = 0;
        for (int i = 0; i < nt; ++i)
            if (cfg_fits(tab[i], mode, vgpr32) && tab[i].G >= 64)
                best = std::max<int64_t>(best, (int64_t)tab[i].G * tab[i].V);
        for (int i = 0; i < nt && cnt < 16; ++i)
            if (cfg_fits(tab[i], mode, vgpr32) && tab[i].G >= 64 &&
                (int64_t)tab[i].G * tab[i].V == best)
                idx[cnt++] = i;
    }
    // the measured default goes first; when the capacity window above left it
    // out (or the list was full), it is taken from the whole table, as long
    // as it fits this mode's register and LDS budget
    {
        const Cfg want = vec ? preferred_shape(mode, esize, m, n, nv) : preferred_scalar_shape(mode, esize, m, n);
        int at = -1;
        for (int k = 0; k < cnt && at < 0; ++k)
            if (same_cfg(tab[idx[k]], want))
                at = k;
        if (at < 0) {
            for (int i = 0; i < nt && at < 0; ++i) {
                if (same_cfg(tab[i], want) && cfg_fits(tab[i], mode, vgpr32) && (int64_t)tab[i].G * tab[i].V >= std::min<int64_t>(nv, 8192)) {
                    if (cnt < 16)
                        ++cnt;
                    at = cnt - 1;
                    idx[at] = i;
                }
            }
        }
        if (at > 0) {
            const int keep = idx[at];
            for (int j = at; j > 0; --j)
                idx[j] = idx[j - 1];
            idx[0] = keep;
        }
    }
    return cnt;
}

// The plan of table shape `cfg` for an m x n matrix.
static Plan plan_of(int esize, bool vec, int mode, int64_t m, int64_t n, int cfg)
{
    Plan p;
    p.vec = vec;
    p.vw = vec ? 16 / esize : 1;
    p.cfg = cfg;
    p.c = vec ? kVecCfg[p.cfg] : kScalarCfg[p.cfg];
    p.threads = p.c.G < 256 ? 256 : p.c.G;
    p.pw = (int64_t)p.c.G * p.c.V * p.vw;
    p.panels = std::max<int64_t>(1, (n + p.pw - 1) / p.pw);
    if (p.panels > 1) {
        // panels of equal width (a multiple of the vector width): a short
        // last panel would finish early and leave its compute units idle
        // (8-16% slower for rows of 1.2-2.4 panels)
        const int64_t even = (n + p.panels - 1) / p.panels;
        p.pw = std::min<int64_t>(p.pw, (even + p.vw - 1) / p.vw * p.vw);
        p.panels = (n + p.pw - 1) / p.pw;  // no empty last panel
    }
    const int64_t rows_per_block = (int64_t)batch_of(p.c.B, mode) * (p.threads / p.c.G);
    const int64_t nblk = (m + rows_per_block - 1) / rows_per_block;
    // enough workgroups to fill the shape's CUX compute units per XCD at its occupancy
    const int64_t per_cu = p.threads <= 256 ? 4 : (p.threads == 512 && p.c.WPE >= 4 ? 2 : 1);
    int64_t fill = (int64_t)kXcds * p.c.CUX * per_cu;
    // column sums over several panels: the panels already fill the chip, and
    // every row workgroup adds a partial row of n to the workspace (208
    // partial rows for 268 matrix rows of 10^6 elements would cost as much
    // traffic as the matrix), so the workgroups of a panel share the chip
    if ((mode & F_COL) && p.panels > 1)
        fill = std::max<int64_t>(1, (fill + p.panels - 1) / p.panels);
    p.nb = std::max<int64_t>(1, std::min<int64_t>(nblk, fill));
    return p;
}

Plan plan_stream(int esize, bool vec, int mode, int64_t m, int64_t n, int variant)
{
    int idx[16];
    const int cnt = stream_candidates(esize, vec, mode, m, n, idx);
    const int k = (variant >= 0 && variant < cnt) ? variant : 0;
    return plan_of(esize, vec, mode, m, n, idx[k]);
}

static std::atomic<int> g_variant[8] = {{-1}, {-1}, {-1}, {-1}, {-1}, {-1}, {-1}, {-1}};

static int op_mode(int op)
{
    switch (op) {
    case MEP_OP_MATVEC: return MODE_MV;
    case MEP_OP_MATVEC_T: return MODE_ATW;
    case MEP_OP_BICG: return MODE_BICG;
    case MEP_OP_ATA_X: return MODE_ATAX;
    case MEP_OP_AXPBY_MV: return MODE_AXPBY;
    case MEP_OP_GEMVER: return MODE_GEMV1;
    default: return -1;
    }
}

static size_t align256(size_t b) { return (b + 255) & ~size_t(255); }

// The two vector samples (sum, elementwise add) have no kernel candidates.
static bool is_vector_op(int op) { return op == MEP_OP_REDUCE_SUM || op == MEP_OP_VECTOR_ADD; }

// Workgroups of the sum: one contiguous chunk of >= 8192 vectors each, at
// most 512 (two per compute unit: measured the fastest on MI355X).
int64_t reduce_blocks(int64_t n, int esize)
{
    const int64_t nv = n * esize / 16;
    return std::max<int64_t>(1, std::min<int64_t>((nv + 8191) / 8192, 512));
}

// Workspace pieces of one plan: column partials (nb rows of n), partial dots
// of column panels (panels rows of m, twice for two matrices) and, for the
// two-pass ATAX, the intermediate t.
struct WsLayout {
    size_t colpart, dotpart, dotpart2, tvec, total;
};

static WsLayout layout_for(int mode, const Plan& p, int esize, int64_t m, int64_t n, bool need_t)
{
    WsLayout w{0, 0, 0, 0, 0};
    if (mode & F_COL)
        w.colpart = align256((size_t)p.nb * (size_t)n * esize);
    if ((mode & F_DOT) && p.panels > 1) {
        w.dotpart = align256((size_t)p.panels * (size_t)m * esize);
        if (mode & F_TWO)
            w.dotpart2 = w.dotpart;
    }
    if (need_t)
        w.tvec = align256((size_t)m * esize);
    w.total = w.colpart + w.dotpart + w.dotpart2 + w.tvec;
    return w;
}

static bool vec_ok_n(int esize, int64_t n) { return n % (16 / esize) == 0; }
static bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Largest workspace of any candidate of `mode` on one load path.
static size_t max_layout(int mode, int esize, bool vec, int64_t m, int64_t n)
{
    int idx[16];
    const int cnt = stream_candidates(esize, vec, mode, m, n, idx);
    size_t best = 0;
    for (int k = 0; k < cnt; ++k)
        best = std::max(best, layout_for(mode, plan_of(esize, vec, mode, m, n, idx[k]), esize, m, n, false).total);
    return best;
}

// Two-pass ATAX (rows over column panels): A x over panels into t, then
// A^T t; both passes take the same variant index (each list clipped to its
// default), and the space of the partial dots, t and the column partials is
// held at once.
static size_t two_pass_ata_x_ws(int esize, bool vec, int64_t m, int64_t n)
{
    int i1[16], i2[16];
    const int c1 = stream_candidates(esize, vec, MODE_MV, m, n, i1);
    const int c2 = stream_candidates(esize, vec, MODE_ATW, m, n, i2);
    size_t best = 0;
    for (int k = 0; k < std::max(c1, c2); ++k) {
        const WsLayout l1 = layout_for(MODE_MV, plan_of(esize, vec, MODE_MV, m, n, i1[k < c1 ? k : 0]), esize, m,
                                       n, true);
        const WsLayout l2 = layout_for(MODE_ATW, plan_of(esize, vec, MODE_ATW, m, n, i2[k < c2 ? k : 0]), esize,
                                       m, n, false);
        best = std::max(best, l1.dotpart + l1.tvec + l2.colpart);
    }
    return best;
}

// Largest workspace over both load paths and every candidate shape.  Each
// candidate list is built once (this runs on every operation call).
static size_t ws_bytes_mode(int mode, int esize, int64_t m, int64_t n)
{
    if (m == 0 || n == 0)
        return 0;
    size_t best = 0;
    for (int v = 0; v < 2; ++v) {
        const bool vec = v == 0;
        if (vec && !vec_ok_n(esize, n))
            continue;
        if (mode == MODE_GEMV1) {
            // pass 1 column partials, then (reusing the space) pass 2 partial dots
            best = std::max({best, max_layout(MODE_GEMV1, esize, vec, m, n), max_layout(MODE_MV, esize, vec, m, n)});
        } else if (mode == MODE_ATAX) {
            int idx[16];
            const int cnt = stream_candidates(esize, vec, mode, m, n, idx);
            bool two_pass = false;
            for (int k = 0; k < cnt; ++k) {
                const Plan p = plan_of(esize, vec, mode, m, n, idx[k]);
                if (p.panels > 1)
                    two_pass = true;
                else
                    best = std::max(best, layout_for(mode, p, esize, m, n, false).total);
            }
            if (two_pass)
                best = std::max(best, two_pass_ata_x_ws(esize, vec, m, n));
        } else {
            best = std::max(best, max_layout(mode, esize, vec, m, n));
        }
    }
    return best;
}

// ---------------------------------------------------------------------------
// argument checks (pure host code: nothing here touches the GPU)
// ---------------------------------------------------------------------------

struct Range {
    const void* p;
    size_t bytes;
    const char* name;
};

static int check_sizes(int dtype, int64_t m, int64_t n)
{
    if (esize_of(dtype) == 0)
        return fail(MEP_EINVAL, "dtype %d is neither MEP_F32 nor MEP_F64", dtype);
    if (m < 0 || n < 0)
        return fail(MEP_EINVAL, "negative size m=%lld n=%lld", (long long)m, (long long)n);
    if (m > kMaxDim || n > kMaxDim)
        return fail(MEP_EINVAL, "size above 2^30: m=%lld n=%lld", (long long)m, (long long)n);
    // rows are cut into at most 65535 column panels of >= 8192 elements
    if (n > kMaxRow)
        return fail(MEP_EINVAL, "row length n=%lld above %lld", (long long)n, (long long)kMaxRow);
    return MEP_OK;
}

static int check_ptr(const void* p, int64_t count, int esize, const char* name)
{
    if (count > 0 && p == nullptr)
        return fail(MEP_EINVAL, "%s is NULL but has %lld elements", name, (long long)count);
    if (p != nullptr && !aligned(p, (size_t)esize))
        return fail(MEP_EALIGN, "%s is not aligned to %d bytes", name, esize);
    return MEP_OK;
}

static bool overlap(const Range& a, const Range& b)
{
    if (a.p == nullptr || b.p == nullptr || a.bytes == 0 || b.bytes == 0)
        return false;
    const uintptr_t a0 = (uintptr_t)a.p, a1 = a0 + a.bytes;
    const uintptr_t b0 = (uintptr_t)b.p, b1 = b0 + b.bytes;
    return a0 < b1 && b0 < a1;
}

// outputs must not overlap any other range (inputs, workspace, other outputs)
static int check_overlaps(const Range* outs, int nout, const Range* ins, int nin)
{
    for (int i = 0; i < nout; ++i) {
        for (int j = 0; j < nin; ++j)
            if (overlap(outs[i], ins[j]))
                return fail(MEP_EINVAL, "output %s overlaps %s", outs[i].name, ins[j].name);
        for (int j = i + 1; j < nout; ++j)
            if (overlap(outs[i], outs[j]))
                return fail(MEP_EINVAL, "outputs %s and %s overlap", outs[i].name, outs[j].name);
    }
    return MEP_OK;
}

static int check_ws(void* ws, size_t ws_bytes, size_t need)
{
    if (need == 0)
        return MEP_OK;
    if (ws == nullptr || ws_bytes < need)
        return fail(MEP_EWORKSPACE, "workspace of %zu bytes given, %zu needed", ws == nullptr ? 0 : ws_bytes,
                    need);
    if (!aligned(ws, 256))
        return fail(MEP_EALIGN, "workspace is not aligned to 256 bytes");
    return MEP_OK;
}

// ---------------------------------------------------------------------------
// profiling of the streaming kernel
// ---------------------------------------------------------------------------

struct Prof {
    bool armed = false;
    int cap = 0, used = 0;
    // launch ordinal since arming; launch i is stamped when (i / group) % every == 0
    int64_t seen = 0;
    int group = 1, every = 1;
    std::vector<hipEvent_t> start, stop;
};
static Prof g_prof;

// The event pair for the next streaming launch while profiling is armed.
static LaunchEvents prof_next()
{
    if (!g_prof.armed)
        return LaunchEvents{nullptr, nullptr};
    const int64_t i = g_prof.seen++;
    if ((i / g_prof.group) % g_prof.every == 0 && g_prof.used < g_prof.cap) {
        const LaunchEvents ev{g_prof.start[g_prof.used], g_prof.stop[g_prof.used]};
        ++g_prof.used;
        return ev;
    }
    return LaunchEvents{nullptr, nullptr};
}

template <typename T>
static hipError_t stream_launch(const Plan& p, int mode, const StreamArgs<T>& a, hipStream_t s)
{
    if (p.panels > 65535 || p.nb > 65535)
        return hipErrorInvalidConfiguration;  // beyond the grid limits; sizes are checked first
    return launch_stream<T>(p, mode, a, s, prof_next());
}

static int variant_of(int op) { return g_variant[op].load(std::memory_order_relaxed); }

// ---------------------------------------------------------------------------
// operations
// ---------------------------------------------------------------------------

template <typename T>
static StreamArgs<T> empty_args(int64_t m, int64_t n)
{
    StreamArgs<T> a;
    std::memset(&a, 0, sizeof a);
    a.m = m;
    a.n = n;
    a.ldp = n;
    return a;
}

template <typename T>
static int run_matvec(int64_t m, int64_t n, const T* A, const T* x, T* y, char* ws, hipStream_t s)
{
    hipError_t e = hipSuccess;
    if (m == 0)
        return MEP_OK;
    if (n == 0) {
        e = launch_fill_zero<T>(y, m, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    const bool vec = vec_ok_n(sizeof(T), n) && aligned(A, 16) && aligned(x, 16);
    const Plan p = plan_stream(sizeof(T), vec, MODE_MV, m, n, variant_of(MEP_OP_MATVEC));
    StreamArgs<T> a = empty_args<T>(m, n);
    a.A = A;
    a.x = x;
    if (p.panels == 1) {
        a.rowout = y;
        e = stream_launch<T>(p, MODE_MV, a, s);
    } else {
        a.dotpart = reinterpret_cast<T*>(ws);
        e = stream_launch<T>(p, MODE_MV, a, s);
        if (e == hipSuccess)
            e = launch_colreduce<T>(a.dotpart, nullptr, m, p.panels, m, (T)1, (T)0, y, s, EPI_SCALE);
    }
    return e == hipSuccess ? MEP_OK : hip_fail(e, "matvec launch");
}

template <typename T>
static int run_matvec_t(int64_t m, int64_t n, const T* A, const T* w, T* z, const T* pv, T* q, bool pair,
                        char* ws, hipStream_t s)
{
    hipError_t e = hipSuccess;
    if (n == 0) {
        if (pair && m > 0)
            e = launch_fill_zero<T>(q, m, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    if (m == 0) {
        e = launch_fill_zero<T>(z, n, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    const int mode = pair ? MODE_BICG : MODE_ATW;
    const int op = pair ? MEP_OP_BICG : MEP_OP_MATVEC_T;
    const bool vec = vec_ok_n(sizeof(T), n) && aligned(A, 16) && (!pair || aligned(pv, 16));
    const Plan p = plan_stream(sizeof(T), vec, mode, m, n, variant_of(op));
    const WsLayout l = layout_for(mode, p, sizeof(T), m, n, false);
    StreamArgs<T> a = empty_args<T>(m, n);
    a.A = A;
    a.x = pv;
    a.w = w;
    a.colpart = reinterpret_cast<T*>(ws);
    if (pair) {
        if (p.panels == 1)
            a.rowout = q;
        else
            a.dotpart = reinterpret_cast<T*>(ws + l.colpart);
    }
    e = stream_launch<T>(p, mode, a, s);
    if (e == hipSuccess)
        e = launch_colreduce<T>(a.colpart, nullptr, n, p.nb, n, (T)1, (T)0, z, s, EPI_SCALE);
    if (e == hipSuccess && pair && p.panels > 1)
        e = launch_colreduce<T>(a.dotpart, nullptr, m, p.panels, m, (T)1, (T)0, q, s, EPI_SCALE);
    return e == hipSuccess ? MEP_OK : hip_fail(e, "matvec_t launch");
}

// Workspace bytes the ATAX call with these operands really uses under the
// given variant (mep_workspace_bytes covers every candidate).
static size_t ata_x_used_bytes(int esize, bool vec, int64_t m, int64_t n, int variant)
{
    if (m == 0 || n == 0)
        return 0;
    const Plan p = plan_stream(esize, vec, MODE_ATAX, m, n, variant);
    if (p.panels == 1)
        return layout_for(MODE_ATAX, p, esize, m, n, false).total;
    const Plan p1 = plan_stream(esize, vec, MODE_MV, m, n, variant);
    const Plan p2 = plan_stream(esize, vec, MODE_ATW, m, n, variant);
    const WsLayout l1 = layout_for(MODE_MV, p1, esize, m, n, true);
    return l1.dotpart + l1.tvec + layout_for(MODE_ATW, p2, esize, m, n, false).colpart;
}

template <typename T>
static int run_ata_x(int64_t m, int64_t n, const T* A, const T* x, T* y, T* t, char* ws, hipStream_t s,
                     int variant)
{
    hipError_t e = hipSuccess;
    if (n == 0) {
        if (t != nullptr && m > 0)
            e = launch_fill_zero<T>(t, m, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    if (m == 0) {
        e = launch_fill_zero<T>(y, n, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    const bool vec = vec_ok_n(sizeof(T), n) && aligned(A, 16) && aligned(x, 16);
    const Plan p = plan_stream(sizeof(T), vec, MODE_ATAX, m, n, variant);
    if (p.panels == 1) {
        // one pass: row dot, then the same row scaled by it into the column sums
        StreamArgs<T> a = empty_args<T>(m, n);
        a.A = A;
        a.x = x;
        a.rowout = t;
        a.colpart = reinterpret_cast<T*>(ws);
        e = stream_launch<T>(p, MODE_ATAX, a, s);
        if (e == hipSuccess)
            e = launch_colreduce<T>(a.colpart, nullptr, n, p.nb, n, (T)1, (T)0, y, s, EPI_SCALE);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "ata_x launch");
    }
    // rows too long to keep on chip: t = A x over column panels, then A^T t
    const Plan p1 = plan_stream(sizeof(T), vec, MODE_MV, m, n, variant);
    const Plan p2 = plan_stream(sizeof(T), vec, MODE_ATW, m, n, variant);
    const WsLayout l1 = layout_for(MODE_MV, p1, sizeof(T), m, n, true);
    T* dot = reinterpret_cast<T*>(ws);
    T* tt = t != nullptr ? t : reinterpret_cast<T*>(ws + l1.dotpart);
    T* colpart = reinterpret_cast<T*>(ws + l1.dotpart + l1.tvec);
    StreamArgs<T> a1 = empty_args<T>(m, n);
    a1.A = A;
    a1.x = x;
    a1.dotpart = dot;
    if (p1.panels == 1)
        a1.rowout = tt;
    e = stream_launch<T>(p1, MODE_MV, a1, s);
    if (e == hipSuccess && p1.panels > 1)
        e = launch_colreduce<T>(dot, nullptr, m, p1.panels, m, (T)1, (T)0, tt, s, EPI_SCALE);
    if (e == hipSuccess) {
        StreamArgs<T> a2 = empty_args<T>(m, n);
        a2.A = A;
        a2.w = tt;
        a2.colpart = colpart;
        e = stream_launch<T>(p2, MODE_ATW, a2, s);
        if (e == hipSuccess)
            e = launch_colreduce<T>(colpart, nullptr, n, p2.nb, n, (T)1, (T)0, y, s, EPI_SCALE);
    }
    return e == hipSuccess ? MEP_OK : hip_fail(e, "ata_x launch");
}

template <typename T>
static int run_axpby(int64_t m, int64_t n, T alpha, const T* A, T beta, const T* B, const T* x, T* y,
                     char* ws, hipStream_t s)
{
    hipError_t e = hipSuccess;
    if (m == 0)
        return MEP_OK;
    if (n == 0) {
        e = launch_fill_zero<T>(y, m, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    const bool vec = vec_ok_n(sizeof(T), n) && aligned(A, 16) && aligned(B, 16) && aligned(x, 16);
    const Plan p = plan_stream(sizeof(T), vec, MODE_AXPBY, m, n, variant_of(MEP_OP_AXPBY_MV));
    const WsLayout l = layout_for(MODE_AXPBY, p, sizeof(T), m, n, false);
    StreamArgs<T> a = empty_args<T>(m, n);
    a.A = A;
    a.B = B;
    a.x = x;
    a.alpha = alpha;
    a.beta = beta;
    if (p.panels == 1) {
        a.rowout = y;
        e = stream_launch<T>(p, MODE_AXPBY, a, s);
    } else {
        a.dotpart = reinterpret_cast<T*>(ws);
        a.dotpart2 = reinterpret_cast<T*>(ws + l.dotpart);
        e = stream_launch<T>(p, MODE_AXPBY, a, s);
        if (e == hipSuccess)
            e = launch_colreduce<T>(a.dotpart, a.dotpart2, m, p.panels, m, alpha, beta, y, s, EPI_TWO);
    }
    return e == hipSuccess ? MEP_OK : hip_fail(e, "axpby_mv launch");
}

// ---------------------------------------------------------------------------
// streaming copy (ceiling probe) and cache flush
// ---------------------------------------------------------------------------

// The copy probe streams rows of THREADS * V 16-byte vectors (128 KiB):
// workgroup w takes rows w, w + gridDim.x, ..., with non-temporal buffer
// loads and stores (the resource's range check drops the ragged end), the
// next row loaded while the current one is stored -- the access pattern of
// the matrix kernels' store pass, without the arithmetic.  Scheduling fences
// keep each row's loads ahead of the previous row's stores, as in the
// streaming kernel (1.3% faster than letting the compiler interleave them).
constexpr int kCopyThreads = 1024, kCopyV = 8;

__global__ void __launch_bounds__(kCopyThreads) k_copy16(const void* __restrict__ src, void* __restrict__ dst,
                                                         int64_t count)
{
    typedef float vec __attribute__((ext_vector_type(4)));
    constexpr int64_t RV = (int64_t)kCopyThreads * kCopyV;
    const int64_t rows = (count + RV - 1) / RV;
    const int tid = threadIdx.x;
    vec a[kCopyV], b[kCopyV];
    // one resource per row: base = the row's first vector, size = what is left
    auto rsrc = [&](const void* base, int64_t r) __attribute__((always_inline)) {
        const int64_t left = r < rows ? (count - r * RV) * 16 : 0;
        return make_rsrc(static_cast<const char*>(base) + (r < rows ? r * RV * 16 : 0),
                         (uint32_t)(left < RV * 16 ? left : RV * 16));
    };
    auto load = [&](int64_t r, vec (&v)[kCopyV]) __attribute__((always_inline)) {
        const __amdgpu_buffer_rsrc_t rs = rsrc(src, r);
#pragma unroll
        for (int k = 0; k < kCopyV; ++k)
            v[k] = load_buf<float, 4, 2>(rs, (uint32_t)((k * kCopyThreads + tid) * 16), 0);
    };
    auto store = [&](int64_t r, vec (&v)[kCopyV]) __attribute__((always_inline)) {
        const __amdgpu_buffer_rsrc_t rs = rsrc(dst, r);
#pragma unroll
        for (int k = 0; k < kCopyV; ++k)
            store_buf<float, 4, 2>(v[k], rs, (uint32_t)((k * kCopyThreads + tid) * 16));
    };
    const int64_t step = gridDim.x;
    int64_t r = blockIdx.x;
    if (r < rows)
        load(r, a);
    while (r < rows) {
        load(r + step, b);
        __builtin_amdgcn_sched_barrier(0);
        store(r, a);
        __builtin_amdgcn_sched_barrier(0);
        r += step;
        if (r >= rows)
            break;
        load(r + step, a);
        __builtin_amdgcn_sched_barrier(0);
        store(r, b);
        __builtin_amdgcn_sched_barrier(0);
        r += step;
    }
}

__global__ void __launch_bounds__(256) k_flush16(uint4* __restrict__ dst, int64_t count, uint32_t tag)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256)
        dst[i] = make_uint4(tag, (uint32_t)i, (uint32_t)(i >> 32), tag ^ 0xFFFFFFFFu);
}

hipError_t launch_copy16(const void* src, void* dst, size_t bytes, hipStream_t s)
{
    const int64_t count = (int64_t)(bytes / 16);
    const int64_t rv = (int64_t)kCopyThreads * kCopyV;
    const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((count + rv - 1) / rv, kXcds * kCusPerXcd));
    hipLaunchKernelGGL(k_copy16, dim3((unsigned)blocks), dim3(kCopyThreads), 0, s, src, dst, count);
    return hipGetLastError();
}

hipError_t launch_flush(void* buf, size_t bytes, uint32_t tag, hipStream_t s)
{
    const int64_t count = (int64_t)(bytes / 16);
    if (count == 0)
        return hipSuccess;
    const int64_t blocks = std::min<int64_t>((count + 255) / 256, 256 * 16);
    hipLaunchKernelGGL(k_flush16, dim3((unsigned)blocks), dim3(256), 0, s, (uint4*)buf, count, tag);
    return hipGetLastError();
}

template <typename T>
static int run_gemver(int64_t m, int64_t n, T alpha, T beta, const T* A, T* Ahat, const T* u1, const T* v1,
                      const T* u2, const T* v2, const T* y, const T* z, T* x, T* w, char* ws, hipStream_t s)
{
    hipError_t e = hipSuccess;
    if (n == 0) {
        e = launch_fill_zero<T>(w, m, s);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "fill");
    }
    if (m == 0) {
        // x = beta * (empty sum) + z
        e = launch_colreduce<T>(reinterpret_cast<const T*>(z), z, n, 0, n, beta, (T)0, x, s, EPI_ADDVEC);
        return e == hipSuccess ? MEP_OK : hip_fail(e, "gemver launch");
    }
    // pass 1: Ahat = A + u1 v1^T + u2 v2^T, stored; column partials of Ahat^T y
    const bool vec1 = vec_ok_n(sizeof(T), n) && aligned(A, 16) && aligned(Ahat, 16) && aligned(v1, 16) &&
                      aligned(v2, 16);
    const Plan p1 = plan_stream(sizeof(T), vec1, MODE_GEMV1, m, n, variant_of(MEP_OP_GEMVER));
    StreamArgs<T> a1 = empty_args<T>(m, n);
    a1.A = A;
    a1.Aout = Ahat;
    a1.w = y;
    a1.u1 = u1;
    a1.u2 = u2;
    a1.v1 = v1;
    a1.v2 = v2;
    a1.colpart = reinterpret_cast<T*>(ws);
    e = stream_launch<T>(p1, MODE_GEMV1, a1, s);
    // x = beta * (Ahat^T y) + z
    if (e == hipSuccess)
        e = launch_colreduce<T>(a1.colpart, z, n, p1.nb, n, beta, (T)0, x, s, EPI_ADDVEC);
    // pass 2: w = alpha * Ahat x
    if (e == hipSuccess) {
        const bool vec2 = vec_ok_n(sizeof(T), n) && aligned(Ahat, 16) && aligned(x, 16);
        const Plan p2 = plan_stream(sizeof(T), vec2, MODE_MV, m, n, -1);
        StreamArgs<T> a2 = empty_args<T>(m, n);
        a2.A = Ahat;
        a2.x = x;
        a2.alpha = alpha;
        a2.scale_rows = 1;
        if (p2.panels == 1) {
            a2.rowout = w;
            e = stream_launch<T>(p2, MODE_MV, a2, s);
        } else {
            a2.dotpart = reinterpret_cast<T*>(ws);
            e = stream_launch<T>(p2, MODE_MV, a2, s);
            if (e == hipSuccess)
                e = launch_colreduce<T>(a2.dotpart, nullptr, m, p2.panels, m, alpha, (T)0, w, s, EPI_SCALE);
        }
    }
    return e == hipSuccess ? MEP_OK : hip_fail(e, "gemver launch");
}

}  // namespace mep

using namespace mep;

// ---------------------------------------------------------------------------
// extern "C" entry points
// ---------------------------------------------------------------------------

extern "C" {

const char* mep_last_error(void) { return g_last_error.c_str(); }

const char* mep_version(void) { return "mep 0.1 (gfx950)"; }

size_t mep_workspace_bytes(int op, int dtype, int64_t m, int64_t n)
{
    const int es = esize_of(dtype);
    if (is_vector_op(op)) {
        if (es == 0 || n < 0 || n > kMaxDim || op == MEP_OP_VECTOR_ADD || n == 0)
            return 0;
        return align256((size_t)reduce_blocks(n, es) * es);
    }
    const int mode = op_mode(op);
    if (es == 0 || mode < 0 || m < 0 || n < 0 || m > kMaxDim || n > kMaxDim)
        return 0;
    return ws_bytes_mode(mode, es, m, n);
}

int mep_variant_count(int op, int dtype, int64_t m, int64_t n)
{
    const int es = esize_of(dtype);
    if (is_vector_op(op))
        return (es == 0 || n < 0 || n > kMaxDim) ? 0 : (op == MEP_OP_VECTOR_ADD ? kNumVaddVariants : 1);
    const int mode = op_mode(op);
    if (es == 0 || mode < 0 || m < 0 || n < 0 || m > kMaxDim || n > kMaxDim)
        return 0;
    int idx[16];
    const bool vec = vec_ok_n(es, n);
    return std::max(1, stream_candidates(es, vec, mode, std::max<int64_t>(m, 1), std::max<int64_t>(n, 1), idx));
}

int mep_variant_info(int op, int dtype, int64_t m, int64_t n, int variant, char* buf, size_t buf_len)
{
    const int es = esize_of(dtype);
    if (is_vector_op(op)) {
        const int count = mep_variant_count(op, dtype, m, n);
        if (es == 0 || n < 0 || n > kMaxDim || variant < 0 || variant >= count || buf == nullptr ||
            buf_len == 0)
            return fail(MEP_EINVAL, "bad arguments to mep_variant_info");
        if (op == MEP_OP_REDUCE_SUM)
            snprintf(buf, buf_len, "reduce threads=256 grid=%lld, fixed-order partials",
                     (long long)reduce_blocks(n, es));
        else if (variant < 2)
            snprintf(buf, buf_len, "vector-add buffer rows threads=1024 V=4 cus=%d/%d, 16-byte non-temporal",
                     variant == 0 ? kCusPerXcd : 24, kCusPerXcd);
        else if (variant == 2)
            snprintf(buf, buf_len, "vector-add chunks threads=256, 16-byte non-temporal");
        else
            snprintf(buf, buf_len, "vector-add rows threads=1024 V=4 cus=%d/%d, 16-byte non-temporal",
                     variant == 3 ? kCusPerXcd : (variant == 4 ? 24 : 16), kCusPerXcd);
        return MEP_OK;
    }
    const int mode = op_mode(op);
    if (es == 0 || mode < 0 || m < 1 || n < 1 || m > kMaxDim || n > kMaxRow || buf == nullptr ||
        buf_len == 0)
        return fail(MEP_EINVAL, "bad arguments to mep_variant_info");
    const bool vec = vec_ok_n(es, n);
    int idx[16];
    const int cnt = stream_candidates(es, vec, mode, m, n, idx);
    if (variant < 0 || variant >= cnt)
        return fail(MEP_EINVAL, "variant %d outside 0..%d", variant, cnt - 1);
    const Plan p = plan_stream(es, vec, mode, m, n, variant);
    snprintf(buf, buf_len, "%s G=%d V=%d B=%d WPE=%d %s %s cus=%d/%d threads=%d grid=%lldx%lld",
             vec ? "vec16" : "elem", p.c.G, p.c.V, batch_of(p.c.B, mode), p.c.WPE,
             p.c.AUX ? "nt" : "cached", p.c.MAP == 1 ? "blocked" : (p.c.MAP == 2 ? "rotated" : "cyclic"), p.c.CUX,
             kCusPerXcd, p.threads,
             (long long)p.nb, (long long)p.panels);
    return MEP_OK;
}

int mep_set_variant(int op, int variant)
{
    if (op_mode(op) < 0 && !is_vector_op(op))
        return fail(MEP_EINVAL, "unknown op %d", op);
    g_variant[op].store(variant < 0 ? -1 : variant, std::memory_order_relaxed);
    return MEP_OK;
}

int mep_matvec(int dtype, int64_t m, int64_t n, const void* A, const void* x, void* y, void* ws,
               size_t ws_bytes, mep_stream_t stream)
{
    int rc = check_sizes(dtype, m, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(A, m * n, es, "A")) || (rc = check_ptr(x, n, es, "x")) ||
        (rc = check_ptr(y, m, es, "y")))
        return rc;
    const size_t need = mep_workspace_bytes(MEP_OP_MATVEC, dtype, m, n);
    if ((rc = check_ws(ws, ws_bytes, need)))
        return rc;
    const Range outs[] = {{y, (size_t)m * es, "y"}};
    const Range ins[] = {{A, (size_t)(m * n) * es, "A"}, {x, (size_t)n * es, "x"}, {ws, need, "ws"}};
    if ((rc = check_overlaps(outs, 1, ins, 3)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    if (dtype == MEP_F32)
        return run_matvec<float>(m, n, (const float*)A, (const float*)x, (float*)y, (char*)ws, s);
    return run_matvec<double>(m, n, (const double*)A, (const double*)x, (double*)y, (char*)ws, s);
}

int mep_matvec_t(int dtype, int64_t m, int64_t n, const void* A, const void* w, void* z, const void* p,
                 void* q, void* ws, size_t ws_bytes, mep_stream_t stream)
{
    int rc = check_sizes(dtype, m, n);
    if (rc)
        return rc;
    // the pair is requested by either pointer; each may be NULL only when empty
    const bool pair = p != nullptr || q != nullptr;
    if (pair && ((p == nullptr && n > 0) || (q == nullptr && m > 0)))
        return fail(MEP_EINVAL, "p and q must both be set for the paired product");
    const int es = esize_of(dtype);
    if ((rc = check_ptr(A, m * n, es, "A")) || (rc = check_ptr(w, m, es, "w")) ||
        (rc = check_ptr(z, n, es, "z")))
        return rc;
    if (pair && ((rc = check_ptr(p, n, es, "p")) || (rc = check_ptr(q, m, es, "q"))))
        return rc;
    const size_t need = mep_workspace_bytes(pair ? MEP_OP_BICG : MEP_OP_MATVEC_T, dtype, m, n);
    if ((rc = check_ws(ws, ws_bytes, need)))
        return rc;
    const Range outs[] = {{z, (size_t)n * es, "z"}, {q, pair ? (size_t)m * es : 0, "q"}};
    const Range ins[] = {{A, (size_t)(m * n) * es, "A"},
                         {w, (size_t)m * es, "w"},
                         {p, pair ? (size_t)n * es : 0, "p"},
                         {ws, need, "ws"}};
    if ((rc = check_overlaps(outs, 2, ins, 4)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    if (dtype == MEP_F32)
        return run_matvec_t<float>(m, n, (const float*)A, (const float*)w, (float*)z, (const float*)p,
                                   (float*)q, pair, (char*)ws, s);
    return run_matvec_t<double>(m, n, (const double*)A, (const double*)w, (double*)z, (const double*)p,
                                (double*)q, pair, (char*)ws, s);
}

int mep_ata_x(int dtype, int64_t m, int64_t n, const void* A, const void* x, void* y, void* t, void* ws,
              size_t ws_bytes, mep_stream_t stream)
{
    int rc = check_sizes(dtype, m, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(A, m * n, es, "A")) || (rc = check_ptr(x, n, es, "x")) ||
        (rc = check_ptr(y, n, es, "y")))
        return rc;
    if (t != nullptr && (rc = check_ptr(t, m, es, "t")))
        return rc;
    const size_t need = mep_workspace_bytes(MEP_OP_ATA_X, dtype, m, n);
    if ((rc = check_ws(ws, ws_bytes, need)))
        return rc;
    const Range outs[] = {{y, (size_t)n * es, "y"}, {t, t ? (size_t)m * es : 0, "t"}};
    const Range ins[] = {{A, (size_t)(m * n) * es, "A"}, {x, (size_t)n * es, "x"}, {ws, need, "ws"}};
    if ((rc = check_overlaps(outs, 2, ins, 3)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    const int variant = variant_of(MEP_OP_ATA_X);
    if (dtype == MEP_F32)
        return run_ata_x<float>(m, n, (const float*)A, (const float*)x, (float*)y, (float*)t, (char*)ws, s,
                                variant);
    return run_ata_x<double>(m, n, (const double*)A, (const double*)x, (double*)y, (double*)t, (char*)ws, s,
                             variant);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// scratch of the allocation-free ATAX entry point
// ---------------------------------------------------------------------------

namespace mep {

// Device scratch owned by the library: every GPU that runs the entry point
// holds its own copy for the life of the process.  Host code never uses the
// array's name as an address (on the host it is only a stand-in symbol): it
// takes each device's address once from hipGetSymbolAddress and passes that.
constexpr size_t kNoAllocScratchBytes = MEP_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices] = {};

// Address of `scratch` on device `dev`, looked up on the first call there
// (with that device current) and kept.
static int scratch_on(int dev, void** out)
{
    if (dev < 0 || dev >= kMaxDevices)
        return fail(MEP_EINVAL, "device %d outside 0..%d", dev, kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        int cur = -1;
        hipError_t e = hipGetDevice(&cur);
        if (e == hipSuccess && cur != dev)
            e = hipSetDevice(dev);
        void* ptr = nullptr;
        if (e == hipSuccess)
            e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        const hipError_t back = (cur >= 0 && cur != dev) ? hipSetDevice(cur) : hipSuccess;
        if (e != hipSuccess)
            return hip_fail(e, "scratch address");
        if (back != hipSuccess)
            return hip_fail(back, "restore device");
        if (ptr == nullptr)
            return fail(MEP_EHIP, "scratch address is NULL");
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return MEP_OK;
}

}  // namespace mep

extern "C" {

int mep_ata_x_noalloc(int dtype, int64_t m, int64_t n, const void* A, const void* x, void* y, void* t,
                      mep_stream_t stream)
{
    int rc = check_sizes(dtype, m, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(A, m * n, es, "A")) || (rc = check_ptr(x, n, es, "x")) ||
        (rc = check_ptr(y, n, es, "y")))
        return rc;
    if (t != nullptr && (rc = check_ptr(t, m, es, "t")))
        return rc;
    // one reading of the op's variant sizes the call and plans it, so a
    // concurrent mep_set_variant cannot make the plan outgrow the scratch
    const int variant = variant_of(MEP_OP_ATA_X);
    const bool vec = vec_ok_n(es, n) && aligned(A, 16) && aligned(x, 16);
    const size_t need = ata_x_used_bytes(es, vec, m, n, variant);
    if (need > kNoAllocScratchBytes)
        return fail(MEP_EWORKSPACE, "this call needs %zu bytes of scratch; the allocation-free entry point "
                    "holds %zu (use mep_ata_x with a workspace)", need, kNoAllocScratchBytes);
    const Range outs[] = {{y, (size_t)n * es, "y"}, {t, t ? (size_t)m * es : 0, "t"}};
    const Range ins[] = {{A, (size_t)(m * n) * es, "A"}, {x, (size_t)n * es, "x"}};
    if ((rc = check_overlaps(outs, 2, ins, 2)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    int dev = -1;
    hipError_t e = s != nullptr ? hipStreamGetDevice(s, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess)
        return hip_fail(e, "stream device");
    void* ws = nullptr;
    if ((rc = scratch_on(dev, &ws)))
        return rc;
    if (dtype == MEP_F32)
        return run_ata_x<float>(m, n, (const float*)A, (const float*)x, (float*)y, (float*)t, (char*)ws, s,
                                variant);
    return run_ata_x<double>(m, n, (const double*)A, (const double*)x, (double*)y, (double*)t, (char*)ws, s,
                             variant);
}

int mep_axpby_mv(int dtype, int64_t m, int64_t n, double alpha, const void* A, double beta, const void* B,
                 const void* x, void* y, void* ws, size_t ws_bytes, mep_stream_t stream)
{
    int rc = check_sizes(dtype, m, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(A, m * n, es, "A")) || (rc = check_ptr(B, m * n, es, "B")) ||
        (rc = check_ptr(x, n, es, "x")) || (rc = check_ptr(y, m, es, "y")))
        return rc;
    const size_t need = mep_workspace_bytes(MEP_OP_AXPBY_MV, dtype, m, n);
    if ((rc = check_ws(ws, ws_bytes, need)))
        return rc;
    const Range outs[] = {{y, (size_t)m * es, "y"}};
    const Range ins[] = {{A, (size_t)(m * n) * es, "A"},
                         {B, (size_t)(m * n) * es, "B"},
                         {x, (size_t)n * es, "x"},
                         {ws, need, "ws"}};
    if ((rc = check_overlaps(outs, 1, ins, 4)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    if (dtype == MEP_F32)
        return run_axpby<float>(m, n, (float)alpha, (const float*)A, (float)beta, (const float*)B,
                                (const float*)x, (float*)y, (char*)ws, s);
    return run_axpby<double>(m, n, alpha, (const double*)A, beta, (const double*)B, (const double*)x,
                             (double*)y, (char*)ws, s);
}

int mep_gemver(int dtype, int64_t m, int64_t n, double alpha, double beta, const void* A, void* Ahat,
               const void* u1, const void* v1, const void* u2, const void* v2, const void* y, const void* z,
               void* x, void* w, void* ws, size_t ws_bytes, mep_stream_t stream)
{
    int rc = check_sizes(dtype, m, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(A, m * n, es, "A")) || (rc = check_ptr(Ahat, m * n, es, "Ahat")) ||
        (rc = check_ptr(u1, m, es, "u1")) || (rc = check_ptr(v1, n, es, "v1")) ||
        (rc = check_ptr(u2, m, es, "u2")) || (rc = check_ptr(v2, n, es, "v2")) ||
        (rc = check_ptr(y, m, es, "y")) || (rc = check_ptr(z, n, es, "z")) || (rc = check_ptr(x, n, es, "x")) ||
        (rc = check_ptr(w, m, es, "w")))
        return rc;
    const size_t need = mep_workspace_bytes(MEP_OP_GEMVER, dtype, m, n);
    if ((rc = check_ws(ws, ws_bytes, need)))
        return rc;
    const size_t mat = (size_t)(m * n) * es;
    // Ahat may be A itself (in-place update); otherwise it must not overlap A
    const Range aRange{Ahat == A ? nullptr : A, mat, "A"};
    const Range outs[] = {{Ahat, mat, "Ahat"}, {x, (size_t)n * es, "x"}, {w, (size_t)m * es, "w"}};
    const Range ins[] = {aRange,
                         {u1, (size_t)m * es, "u1"},
                         {v1, (size_t)n * es, "v1"},
                         {u2, (size_t)m * es, "u2"},
                         {v2, (size_t)n * es, "v2"},
                         {y, (size_t)m * es, "y"},
                         {z, (size_t)n * es, "z"},
                         {ws, need, "ws"}};
    if ((rc = check_overlaps(outs, 3, ins, 8)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    if (dtype == MEP_F32)
        return run_gemver<float>(m, n, (float)alpha, (float)beta, (const float*)A, (float*)Ahat, (const float*)u1,
                                 (const float*)v1, (const float*)u2, (const float*)v2, (const float*)y,
                                 (const float*)z, (float*)x, (float*)w, (char*)ws, s);
    return run_gemver<double>(m, n, alpha, beta, (const double*)A, (double*)Ahat, (const double*)u1,
                              (const double*)v1, (const double*)u2, (const double*)v2, (const double*)y,
                              (const double*)z, (double*)x, (double*)w, (char*)ws, s);
}

int mep_reduce_sum(int dtype, int64_t n, const void* x, void* out, void* ws, size_t ws_bytes,
                   mep_stream_t stream)
{
    int rc = check_sizes(dtype, 1, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(x, n, es, "x")) || (rc = check_ptr(out, 1, es, "s")))
        return rc;
    const size_t need = mep_workspace_bytes(MEP_OP_REDUCE_SUM, dtype, 1, n);
    if ((rc = check_ws(ws, ws_bytes, need)))
        return rc;
    const Range outs[] = {{out, (size_t)es, "s"}};
    const Range ins[] = {{x, (size_t)n * es, "x"}, {ws, need, "ws"}};
    if ((rc = check_overlaps(outs, 1, ins, 2)))
        return rc;
    hipStream_t s = (hipStream_t)stream;
    hipError_t e;
    const int64_t nb = reduce_blocks(n, es);
    if (n == 0)
        e = dtype == MEP_F32 ? launch_fill_zero<float>((float*)out, 1, s) : launch_fill_zero<double>((double*)out, 1, s);
    else if (dtype == MEP_F32)
        e = launch_reduce_sum<float>((const float*)x, n, (float*)out, (float*)ws, nb, s, prof_next());
    else
        e = launch_reduce_sum<double>((const double*)x, n, (double*)out, (double*)ws, nb, s, prof_next());
    return e == hipSuccess ? MEP_OK : hip_fail(e, "reduce launch");
}

int mep_vector_add(int dtype, int64_t n, const void* a, const void* b, void* c, mep_stream_t stream)
{
    int rc = check_sizes(dtype, 1, n);
    if (rc)
        return rc;
    const int es = esize_of(dtype);
    if ((rc = check_ptr(a, n, es, "a")) || (rc = check_ptr(b, n, es, "b")) || (rc = check_ptr(c, n, es, "c")))
        return rc;
    const Range outs[] = {{c, (size_t)n * es, "c"}};
    const Range ins[] = {{a, (size_t)n * es, "a"}, {b, (size_t)n * es, "b"}};
    if ((rc = check_overlaps(outs, 1, ins, 2)))
        return rc;
    if (n == 0)
        return MEP_OK;
    hipStream_t s = (hipStream_t)stream;
    const LaunchEvents ev = prof_next();
    const int v = std::max(0, variant_of(MEP_OP_VECTOR_ADD));
    const hipError_t e =
        dtype == MEP_F32 ? launch_vector_add<float>((const float*)a, (const float*)b, (float*)c, n, v, s, ev)
                         : launch_vector_add<double>((const double*)a, (const double*)b, (double*)c, n, v, s, ev);
    return e == hipSuccess ? MEP_OK : hip_fail(e, "vector add launch");
}

int mep_run(const mep_call_t* c)
{
    if (c == nullptr)
        return fail(MEP_EINVAL, "call is NULL");
    switch (c->op) {
    case MEP_OP_MATVEC:
        return mep_matvec(c->dtype, c->m, c->n, c->A, c->in0, c->out0, c->ws, c->ws_bytes, c->stream);
    case MEP_OP_MATVEC_T:
        return mep_matvec_t(c->dtype, c->m, c->n, c->A, c->in0, c->out0, nullptr, nullptr, c->ws,
                            c->ws_bytes, c->stream);
    case MEP_OP_BICG:
        if ((c->in1 == nullptr && c->n > 0) || (c->out1 == nullptr && c->m > 0))
            return fail(MEP_EINVAL, "BICG needs in1 = p and out1 = q");
        return mep_matvec_t(c->dtype, c->m, c->n, c->A, c->in0, c->out0, c->in1, c->out1, c->ws,
                            c->ws_bytes, c->stream);
    case MEP_OP_ATA_X:
        return mep_ata_x(c->dtype, c->m, c->n, c->A, c->in0, c->out0, c->out1, c->ws, c->ws_bytes,
                         c->stream);
    case MEP_OP_AXPBY_MV:
        return mep_axpby_mv(c->dtype, c->m, c->n, c->alpha, c->A, c->beta, c->B, c->in0, c->out0, c->ws,
                            c->ws_bytes, c->stream);
    case MEP_OP_REDUCE_SUM:
        return mep_reduce_sum(c->dtype, c->n, c->in0, c->out0, c->ws, c->ws_bytes, c->stream);
    case MEP_OP_VECTOR_ADD:
        return mep_vector_add(c->dtype, c->n, c->in0, c->in1, c->out0, c->stream);
    case MEP_OP_GEMVER:
        return mep_gemver(c->dtype, c->m, c->n, c->alpha, c->beta, c->A, c->out2, c->in0, c->in1, c->in2,
                          c->in3, c->in4, c->in5, c->out0, c->out1, c->ws, c->ws_bytes, c->stream);
    default:
        return fail(MEP_EINVAL, "unknown op %d", c->op);
    }
}

double mep_trimmed_mean(const double* samples, int R, int k)
{
    if (samples == nullptr || k < 0 || R <= 2 * k)
        return std::numeric_limits<double>::quiet_NaN();
    std::vector<double> v(samples, samples + R);
    std::sort(v.begin(), v.end());
    double sum = 0.0;
    for (int i = k; i < R - k; ++i)
        sum += v[i];
    return sum / (double)(R - 2 * k);
}

int mep_time_trimmed(const mep_call_t* call, int warmup, int R, int k, int inner, int flush, double* mean_ms,
                     double* samples_ms)
{
    if (call == nullptr || mean_ms == nullptr)
        return fail(MEP_EINVAL, "call and mean_ms must be set");
    if (k < 0 || R <= 2 * k)
        return fail(MEP_EBUDGET, "Eq. 3 needs R > 2k >= 0 (R=%d, k=%d)", R, k);
    if (inner < 1 || warmup < 0)
        return fail(MEP_EBUDGET, "inner must be >= 1 and warmup >= 0");
    if (flush && call->flush_buf != nullptr && (!aligned(call->flush_buf, 16) || call->flush_bytes % 16))
        return fail(MEP_EALIGN, "flush buffer must be 16-byte aligned and a multiple of 16 bytes");
    hipStream_t s = (hipStream_t)call->stream;
    for (int i = 0; i < warmup; ++i) {
        const int rc = mep_run(call);
        if (rc)
            return rc;
    }
    std::vector<hipEvent_t> ev(2 * (size_t)R, nullptr);
    int rc = MEP_OK;
    hipError_t e = hipSuccess;
    for (size_t i = 0; i < ev.size() && e == hipSuccess; ++i)
        e = hipEventCreate(&ev[i]);
    for (int r = 0; r < R && e == hipSuccess && rc == MEP_OK; ++r) {
        if (flush && call->flush_buf != nullptr && call->flush_bytes > 0)
            e = launch_flush(call->flush_buf, call->flush_bytes, 0x9E3779B9u + (uint32_t)r, s);
        if (e == hipSuccess)
            e = hipEventRecord(ev[2 * r], s);
        for (int i = 0; i < inner && e == hipSuccess && rc == MEP_OK; ++i)
            rc = mep_run(call);
        if (e == hipSuccess && rc == MEP_OK)
            e = hipEventRecord(ev[2 * r + 1], s);
    }
    if (e == hipSuccess)
        e = hipStreamSynchronize(s);
    std::vector<double> samples((size_t)R, 0.0);
    for (int r = 0; r < R && e == hipSuccess && rc == MEP_OK; ++r) {
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, ev[2 * r], ev[2 * r + 1]);
        samples[r] = (double)ms / inner;
    }
    for (hipEvent_t x : ev)
        if (x != nullptr)
            (void)hipEventDestroy(x);
    if (rc)
        return rc;
    if (e != hipSuccess)
        return hip_fail(e, "timing");
    if (samples_ms != nullptr)
        std::memcpy(samples_ms, samples.data(), sizeof(double) * R);
    *mean_ms = mep_trimmed_mean(samples.data(), R, k);
    return MEP_OK;
}

// The outputs of a call (out0, out1, out2) and their lengths in elements.
struct CallOutputs {
    void* ptr[3];
    int64_t len[3];
};

static CallOutputs call_outputs(const mep_call_t* c)
{
    CallOutputs o{{c->out0, c->out1, c->out2}, {0, 0, 0}};
    switch (c->op) {
    case MEP_OP_MATVEC: o.len[0] = c->m; break;
    case MEP_OP_MATVEC_T: o.len[0] = c->n; break;
    case MEP_OP_BICG: o.len[0] = c->n; o.len[1] = c->out1 ? c->m : 0; break;
    case MEP_OP_ATA_X: o.len[0] = c->n; o.len[1] = c->out1 ? c->m : 0; break;
    case MEP_OP_AXPBY_MV: o.len[0] = c->m; break;
    case MEP_OP_REDUCE_SUM: o.len[0] = 1; break;
    case MEP_OP_VECTOR_ADD: o.len[0] = c->n; break;
    case MEP_OP_GEMVER: o.len[0] = c->n; o.len[1] = c->m; o.len[2] = c->m * c->n; break;
    default: break;
    }
    return o;
}

// Runs the call once and returns its outputs on the host, promoted to fp64,
// one after another in the order out0, out1, out2.
static int run_and_fetch(const mep_call_t* c, std::vector<double>& out)
{
    int rc = mep_run(c);
    if (rc)
        return rc;
    hipError_t e = hipStreamSynchronize((hipStream_t)c->stream);
    if (e != hipSuccess)
        return hip_fail(e, "synchronize");
    const CallOutputs o = call_outputs(c);
    const int es = esize_of(c->dtype);
    const int64_t total = o.len[0] + o.len[1] + o.len[2];
    std::vector<char> raw((size_t)total * es + 1);
    size_t at = 0;
    for (int k = 0; k < 3 && e == hipSuccess; ++k) {
        if (o.len[k] > 0)
            e = hipMemcpy(raw.data() + at, o.ptr[k], (size_t)o.len[k] * es, hipMemcpyDeviceToHost);
        at += (size_t)o.len[k] * es;
    }
    if (e != hipSuccess)
        return hip_fail(e, "copy outputs");
    out.resize((size_t)total);
    for (int64_t i = 0; i < total; ++i)
        out[i] = es == 4 ? (double)((const float*)raw.data())[i] : ((const double*)raw.data())[i];
    return MEP_OK;
}

// The FE metric of mep_check_fe on elements [lo, hi) of two host fp64
// vectors: +inf when either side holds a non-finite value (std::max would
// skip a NaN reference entry and let an all-NaN reference pass).
static double fe_metric(const std::vector<double>& out, const std::vector<double>& ref, size_t lo, size_t hi)
{
    double worst = 0.0, scale = 0.0;
    for (size_t i = lo; i < hi; ++i) {
        if (!std::isfinite(out[i]) || !std::isfinite(ref[i]))
            return std::numeric_limits<double>::infinity();
        scale = std::max(scale, std::fabs(ref[i]));
        worst = std::max(worst, std::fabs(out[i] - ref[i]));
    }
    if (scale == 0.0)
        return worst == 0.0 ? 0.0 : std::numeric_limits<double>::infinity();
    return worst / scale;
}

// Each output of a call is judged on its own scale; the worst one counts.
static double fe_metric_call(const mep_call_t* c, const std::vector<double>& out, const std::vector<double>& ref)
{
    const CallOutputs o = call_outputs(c);
    double worst = 0.0;
    size_t lo = 0;
    for (int k = 0; k < 3; ++k) {
        worst = std::max(worst, fe_metric(out, ref, lo, lo + (size_t)o.len[k]));
        lo += (size_t)o.len[k];
    }
    return worst;
}

// The load path a call really takes (the 16-byte vector path needs the row
// length and the streamed operands' addresses aligned, as each run_* checks),
// and so the candidate list its variant index refers to.
static bool call_vec(const mep_call_t* c)
{
    const int es = esize_of(c->dtype);
    if (es == 0 || !vec_ok_n(es, c->n) || !aligned(c->A, 16))
        return false;
    switch (c->op) {
    case MEP_OP_MATVEC:
    case MEP_OP_ATA_X: return aligned(c->in0, 16);
    case MEP_OP_BICG: return aligned(c->in1, 16);
    case MEP_OP_AXPBY_MV: return aligned(c->B, 16) && aligned(c->in0, 16);
    case MEP_OP_GEMVER: return aligned(c->out2, 16) && aligned(c->in1, 16) && aligned(c->in3, 16);
    default: return true;
    }
}

static int call_variant_count(const mep_call_t* c)
{
    if (is_vector_op(c->op))
        return mep_variant_count(c->op, c->dtype, c->m, c->n);
    const int es = esize_of(c->dtype);
    const int mode = op_mode(c->op);
    if (es == 0 || mode < 0 || c->m < 0 || c->n < 0 || c->m > kMaxDim || c->n > kMaxDim)
        return 0;
    int idx[16];
    return std::max(1, stream_candidates(es, call_vec(c), mode, std::max<int64_t>(c->m, 1),
                                         std::max<int64_t>(c->n, 1), idx));
}

int mep_select_variant(const mep_call_t* call, int warmup, int R, int k, int inner, int flush, double tol,
                       int apply, int* best, mep_candidate_result_t* results, int results_cap)
{
    if (call == nullptr || best == nullptr || (results == nullptr && results_cap > 0) || results_cap < 0)
        return fail(MEP_EINVAL, "bad arguments to mep_select_variant");
    if (op_mode(call->op) < 0 && !is_vector_op(call->op))
        return fail(MEP_EINVAL, "unknown op %d", call->op);
    if (k < 0 || R <= 2 * k || inner < 1 || warmup < 0)
        return fail(MEP_EBUDGET, "Eq. 3 needs R > 2k >= 0, inner >= 1, warmup >= 0");
    if (call->op == MEP_OP_GEMVER && call->out2 == call->A && call->A != nullptr)
        return fail(MEP_EINVAL, "selection needs an out-of-place GEMVER call (each in-place run changes A)");
    const bool have_flush = call->flush_buf != nullptr && call->flush_bytes > 0;
    if (have_flush && (!aligned(call->flush_buf, 16) || call->flush_bytes % 16))
        return fail(MEP_EALIGN, "flush buffer must be 16-byte aligned and a multiple of 16 bytes");
    const int count = call_variant_count(call);
    if (count < 1)
        return fail(MEP_EINVAL, "no candidates for this call");
    const int saved = variant_of(call->op);
    std::vector<double> base, out;
    int rc = MEP_OK;
    int win = -1;
    double win_ms = 0.0;
    // Settling runs of the default before any candidate is timed: the first
    // launches after the operands were allocated (or after an idle gap) read
    // a few % slower, and candidate 0, timed first, took that penalty alone
    // (7% in one selection over 4 GiB, which its per-candidate warm-up did not
    // absorb).  These runs are not timed and count toward no candidate.
    g_variant[call->op].store(0, std::memory_order_relaxed);
    for (int i = 0; i < std::max(8, 2 * warmup) && rc == MEP_OK; ++i)
        rc = mep_run(call);
    for (int v = 0; v < count && rc == MEP_OK; ++v) {
        g_variant[call->op].store(v, std::memory_order_relaxed);
        mep_candidate_result_t r{std::numeric_limits<double>::quiet_NaN(), 0.0, 0};
        // warm timings: no candidate may inherit the previous one's cache
        // state (a non-temporal shape timed right after a cached-load one
        // reads a cache-resident matrix 5-17% slower), so the caches are
        // cleared once before each candidate runs
        if (!flush && have_flush) {
            const hipError_t fe = launch_flush(call->flush_buf, call->flush_bytes, 0x5BD1E995u + (uint32_t)v,
                                               (hipStream_t)call->stream);
            if (fe != hipSuccess) {
                rc = hip_fail(fe, "flush");
                break;
            }
        }
        rc = run_and_fetch(call, v == 0 ? base : out);
        if (rc)
            break;
        // the baseline is held to its own outputs: 0, or +inf when any is not finite
        r.fe_err = fe_metric_call(call, v == 0 ? base : out, base);
        r.fe_pass = r.fe_err <= tol ? 1 : 0;
        if (r.fe_pass) {
            rc = mep_time_trimmed(call, warmup, R, k, inner, flush, &r.mean_ms, nullptr);
            if (rc)
                break;
            if (win < 0 || r.mean_ms < win_ms) {
                win = v;
                win_ms = r.mean_ms;
            }
        }
        if (v < results_cap)
            results[v] = r;
    }
    g_variant[call->op].store(rc == MEP_OK && apply ? win : saved, std::memory_order_relaxed);
    if (rc)
        return rc;
    *best = win;
    return MEP_OK;
}

int mep_check_fe(int dtype, const void* out, const double* ref, int64_t len, double tol, double* err, int* pass)
{
    if (esize_of(dtype) == 0)
        return fail(MEP_EINVAL, "dtype %d is neither MEP_F32 nor MEP_F64", dtype);
    if (len < 0 || err == nullptr || pass == nullptr || (len > 0 && (out == nullptr || ref == nullptr)))
        return fail(MEP_EINVAL, "bad arguments to mep_check_fe");
    double worst = 0.0, scale = 0.0;
    bool finite = true;
    for (int64_t i = 0; i < len; ++i)
        if (!std::isfinite(ref[i]))
            return fail(MEP_EINVAL, "reference element %lld is not finite", (long long)i);
    for (int64_t i = 0; i < len; ++i) {
        const double o = dtype == MEP_F32 ? (double)((const float*)out)[i] : ((const double*)out)[i];
        if (!std::isfinite(o))
            finite = false;
        scale = std::max(scale, std::fabs(ref[i]));
        worst = std::max(worst, std::fabs(o - ref[i]));
    }
    double e;
    if (!finite)
        e = std::numeric_limits<double>::infinity();
    else if (scale == 0.0)
        e = worst == 0.0 ? 0.0 : std::numeric_limits<double>::infinity();
    else
        e = worst / scale;
    *err = e;
    *pass = e <= tol ? 1 : 0;
    return MEP_OK;
}

int mep_profile_begin(int capacity)
{
    return mep_profile_begin_sampled(capacity, 1, 1);
}

int mep_profile_begin_sampled(int capacity, int group, int every)
{
    if (capacity < 1)
        return fail(MEP_EINVAL, "capacity must be >= 1");
    if (group < 1 || every < 1)
        return fail(MEP_EINVAL, "group and every must be >= 1");
    if (g_prof.armed)
        return fail(MEP_EINVAL, "profiling is already armed");
    g_prof.start.assign((size_t)capacity, nullptr);
    g_prof.stop.assign((size_t)capacity, nullptr);
    // no system-scope fence when these events complete: they only time
    // kernels, nothing on the host reads results through them
    for (int i = 0; i < capacity; ++i) {
        hipError_t e = hipEventCreateWithFlags(&g_prof.start[i], hipEventDisableSystemFence);
        if (e == hipSuccess)
            e = hipEventCreateWithFlags(&g_prof.stop[i], hipEventDisableSystemFence);
        if (e != hipSuccess) {
            for (hipEvent_t x : g_prof.start)
                if (x)
                    (void)hipEventDestroy(x);
            for (hipEvent_t x : g_prof.stop)
                if (x)
                    (void)hipEventDestroy(x);
            g_prof.start.clear();
            g_prof.stop.clear();
            return hip_fail(e, "event create");
        }
    }
    g_prof.cap = capacity;
    g_prof.used = 0;
    g_prof.seen = 0;
    g_prof.group = group;
    g_prof.every = every;
    g_prof.armed = true;
    return MEP_OK;
}

int mep_profile_end(double* total_ms, int* launches)
{
    return mep_profile_end_samples(nullptr, 0, total_ms, launches);
}

int mep_profile_end_samples(double* samples_ms, int cap, double* total_ms, int* launches)
{
    if (!g_prof.armed)
        return fail(MEP_EINVAL, "profiling is not armed");
    if (cap < 0 || (samples_ms == nullptr && cap > 0))
        return fail(MEP_EINVAL, "bad sample buffer");
    double tot = 0.0;
    hipError_t e = hipSuccess;
    for (int i = 0; i < g_prof.used && e == hipSuccess; ++i) {
        e = hipEventSynchronize(g_prof.stop[i]);
        float ms = 0.f;
        if (e == hipSuccess)
            e = hipEventElapsedTime(&ms, g_prof.start[i], g_prof.stop[i]);
        tot += ms;
        if (samples_ms != nullptr && i < cap)
            samples_ms[i] = ms;
    }
    const int used = g_prof.used;
    for (hipEvent_t x : g_prof.start)
        (void)hipEventDestroy(x);
    for (hipEvent_t x : g_prof.stop)
        (void)hipEventDestroy(x);
    g_prof = Prof();
    if (e != hipSuccess)
        return hip_fail(e, "profile events");
    if (total_ms)
        *total_ms = tot;
    if (launches)
        *launches = used;
    return MEP_OK;
}

int mep_stream_copy(const void* src, void* dst, size_t bytes, mep_stream_t stream)
{
    if (bytes == 0)
        return MEP_OK;
    if (src == nullptr || dst == nullptr)
        return fail(MEP_EINVAL, "NULL pointer");
    if (!aligned(src, 16) || !aligned(dst, 16) || bytes % 16)
        return fail(MEP_EALIGN, "copy needs 16-byte aligned pointers and a multiple of 16 bytes");
    const Range a{dst, bytes, "dst"}, b{src, bytes, "src"};
    if (overlap(a, b))
        return fail(MEP_EINVAL, "src and dst overlap");
    const hipError_t e = launch_copy16(src, dst, bytes, (hipStream_t)stream);
    return e == hipSuccess ? MEP_OK : hip_fail(e, "copy launch");
}

}  // extern "C"
