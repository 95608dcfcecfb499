/*
 * mep.h -- C-ABI of libmep.so: the dense matrix-vector family on MI355X
 * (gfx950), wrapped in the minimal-executable-program (MEP) harness of
 * "GPU Kernel Optimization Beyond Full Builds: An LLM Framework with Minimal
 * Executable Programs" (arXiv 2512.22147).
 *
 * The paper's benchmark tables (Tables 1-2, Sec. 4.2) name the PolyBench
 * kernels ATAX, BICG and GESUMMV; their computations are the matrix-vector
 * products below.  The harness follows Sec. 3.1-3.2: a fixed problem size,
 * repeated timed runs ranked by the trimmed mean of Eq. 3, and the
 * functional-equivalence (FE) check of Eq. 4.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Matrices are row-major and contiguous: element (i, j) of the m x n
 *   matrix A is A[i * n + j].  Vectors are contiguous.
 * - dtype is MEP_F32 or MEP_F64 (a mep_dtype_t value, passed as an int).
 *   Every vector has that element type and the arithmetic is done in it
 *   (fp32 inputs accumulate in fp32).
 * - Device pointers are plain HIP device addresses (e.g. a torch tensor's
 *   data_ptr()).  Each must be aligned to its element size.  16-byte aligned
 *   matrices whose row length is a multiple of 16 bytes take the 16-byte
 *   vector path; anything else takes the element-wise path.  Both give
 *   results within the same tolerance; each is deterministic.
 * - 0 <= m <= 2^30 and 0 <= n <= 65535 * 8192.  A zero-length vector may be NULL.  An empty sum is
 *   zero: e.g. with n = 0, y = A x is all zeros.
 * - stream is a hipStream_t (NULL = the default stream).  Operations only
 *   enqueue kernels and return: they never synchronize, allocate or issue a
 *   memset, so a caller may capture them into a HIP graph (outside
 *   mep_profile_begin ... mep_profile_end, whose event stamps are not meant
 *   for capture).
 * - ws is a caller-owned device workspace of at least
 *   mep_workspace_bytes(op, dtype, m, n) bytes (may be NULL when that is 0).
 *   Its contents on entry are irrelevant and on exit unspecified.
 * - Ownership: the caller allocates and frees every buffer.  The library
 *   never allocates or frees device memory and keeps no pointer after a call
 *   returns.
 * - Errors: every argument is checked before anything is launched.  A
 *   non-zero MEP_E* code means nothing was launched and nothing written;
 *   mep_last_error() then describes the problem.  Outputs must not overlap
 *   inputs, the workspace or each other.
 * - Results are bitwise reproducible for a given binary, device, shape and
 *   input: every reduction runs in a fixed order and no atomics are used.
 * - NaN and infinities follow IEEE arithmetic on the defining sums: a NaN or
 *   an infinity in an input reaches exactly the outputs whose sums contain
 *   it, as NaN, +inf or -inf (only where finite partial sums overflow can
 *   the summation order decide).  Padding past the end of the matrix adds
 *   nothing, even where 0 * inf would give NaN.
 */
#ifndef MEP_H
#define MEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { MEP_F32 = 0, MEP_F64 = 1 } mep_dtype_t;

enum {
    MEP_OK = 0,
    MEP_EINVAL = 1,      /* bad size, NULL pointer, overlap, bad op/dtype      */
    MEP_EALIGN = 2,      /* pointer not aligned to its element size            */
    MEP_EWORKSPACE = 3,  /* ws_bytes smaller than mep_workspace_bytes(...)     */
    MEP_EHIP = 4,        /* the HIP runtime reported an error on launch        */
    MEP_EBUDGET = 5      /* harness: R <= 2k or another budget violation       */
};

/* Operation codes, used by mep_workspace_bytes() and mep_call_t. */
enum {
    MEP_OP_MATVEC = 0,   /* y = A x                                          */
    MEP_OP_MATVEC_T = 1, /* z = A^T w                                        */
    MEP_OP_BICG = 2,     /* q = A p and s = A^T r, one read of A (BICG)      */
    MEP_OP_ATA_X = 3,    /* y = A^T (A x) (ATAX)                             */
    MEP_OP_AXPBY_MV = 4, /* y = alpha A x + beta B x (GESUMMV)               */
    MEP_OP_REDUCE_SUM = 5, /* s = sum_i x_i ("reduction", Table 3); m = 1    */
    MEP_OP_VECTOR_ADD = 6, /* c = a + b ("vectoradd", Table 3); m = 1        */
    MEP_OP_GEMVER = 7      /* GEMVER (Tables 1-2), see mep_gemver            */
};

typedef void* mep_stream_t; /* hipStream_t */

/*
 * Workspace bytes that op needs for an m x n problem of the given dtype
 * (covers every kernel candidate and both load paths; 0 for bad arguments).
 * No passage of the paper defines this call: it sizes the caller-owned
 * scratch that the MEP statement's "allocate" step provides.
 */
size_t mep_workspace_bytes(int op, int dtype, int64_t m, int64_t n);

/*
 * y = A x (matrix-vector product; the building block of ATAX, BICG and
 * GESUMMV in Tables 1-2).  A: m x n, x: n, y: m.
 */
int mep_matvec(int dtype, int64_t m, int64_t n, const void* A, const void* x, void* y,
               void* ws, size_t ws_bytes, mep_stream_t stream);

/*
 * z = A^T w (transposed product).  A: m x n, w: m, z: n.
 * If p is not NULL, also q = A p (p: n, q: m) in the same single read of A:
 * this pair is the BICG kernel of Tables 1-2 (q = A p, s = A^T r with w = r,
 * z = s).  The pair is requested when p or q is non-NULL; then each of them
 * may be NULL only if its length is zero.
 */
int mep_matvec_t(int dtype, int64_t m, int64_t n, const void* A, const void* w, void* z,
                 const void* p, void* q, void* ws, size_t ws_bytes, mep_stream_t stream);

/*
 * y = A^T (A x): the ATAX kernel of Table 1.  A: m x n, x: n, y: n.
 * t (nullable, length m) receives the intermediate A x.  When a row of A fits
 * on chip (n <= 32768 for fp32, n <= 16384 for fp64, on the vector path) A is
 * read from memory once; otherwise A x is formed first and A is read twice.
 */
int mep_ata_x(int dtype, int64_t m, int64_t n, const void* A, const void* x, void* y,
              void* t, void* ws, size_t ws_bytes, mep_stream_t stream);

/*
 * Allocation-free variant of mep_ata_x, for callers that cannot allocate or
 * bring workspace: code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation.  The same kernels and results as
 * mep_ata_x (bit for bit), with the column partials kept in a scratch array
 * that the library owns on each GPU: MEP_NOALLOC_SCRATCH_BYTES (64 MiB),
 * reserved on a device when the library's code is first loaded there and
 * held until the process ends; its address is looked up on the first call on
 * a device, which must therefore be made outside a graph capture (later calls
 * may be captured and replayed).  The call allocates and frees nothing.  A call whose plan needs
 * more scratch than that (e.g. a row too long to keep on chip, which takes
 * the two-pass path over a huge m) returns MEP_EWORKSPACE and launches
 * nothing.  Every call on one GPU shares that GPU's scratch: calls that may
 * overlap on one GPU (other streams, other host threads) race and must be
 * serialized by the caller.  The device is the stream's (the current
 * device for a NULL stream).  Arguments as for mep_ata_x, without ws.
 */
#define MEP_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int mep_ata_x_noalloc(int dtype, int64_t m, int64_t n, const void* A, const void* x, void* y,
                      void* t, mep_stream_t stream);

/*
 * y = alpha A x + beta B x: the GESUMMV kernel of Tables 1-2.  A, B: m x n,
 * x: n, y: m.  On the fp32 path alpha and beta are rounded to fp32 first.
 */
int mep_axpby_mv(int dtype, int64_t m, int64_t n, double alpha, const void* A, double beta,
                 const void* B, const void* x, void* y, void* ws, size_t ws_bytes,
                 mep_stream_t stream);

/*
 * GEMVER (named in Tables 1-2; the paper gives no definition, this is the BLAS
 * Technical Forum standard's):
 *     Ahat = A + u1 v1^T + u2 v2^T,   x = beta Ahat^T y + z,   w = alpha Ahat x.
 * A, Ahat: m x n; u1, u2, y, w: m; v1, v2, z, x: n.  Ahat may be A itself (the
 * in-place update of the standard); no other overlap is allowed.  Two passes
 * over the matrix: the first reads A, forms and stores Ahat and accumulates
 * Ahat^T y in the same pass; the second reads Ahat for w (it needs the whole
 * x).  On the fp32 path alpha and beta are rounded to fp32.  Workspace:
 * mep_workspace_bytes(MEP_OP_GEMVER, dtype, m, n).
 */
int mep_gemver(int dtype, int64_t m, int64_t n, double alpha, double beta, const void* A, void* Ahat,
               const void* u1, const void* v1, const void* u2, const void* v2, const void* y,
               const void* z, void* x, void* w, void* ws, size_t ws_bytes, mep_stream_t stream);

/*
 * s = sum_{i<n} x_i: the "reduction" sample of the AMD APP SDK table (Table 3,
 * Sec. 4.3).  x: n elements; s: one element of device memory.  Each workgroup
 * adds one contiguous chunk of x into its partial in ws (mep_workspace_bytes(
 * MEP_OP_REDUCE_SUM, dtype, 1, n) bytes), and one more kernel adds the
 * partials in a fixed order: the result is reproducible and no atomics are
 * used.
 * n = 0 gives s = 0.
 */
int mep_reduce_sum(int dtype, int64_t n, const void* x, void* s, void* ws, size_t ws_bytes,
                   mep_stream_t stream);

/*
 * c = a + b elementwise: the "vectoradd" sample of Table 3.  a, b, c: n
 * elements; c must not overlap a or b.  No workspace.
 */
int mep_vector_add(int dtype, int64_t n, const void* a, const void* b, void* c,
                   mep_stream_t stream);

/*
 * One operation, as the MEP harness runs it.  Field use per op:
 *   MATVEC    in0 = x, out0 = y
 *   MATVEC_T  in0 = w, out0 = z
 *   BICG      in0 = r, out0 = s, in1 = p, out1 = q
 *   ATA_X     in0 = x, out0 = y, out1 = t (nullable)
 *   AXPBY_MV  A, B, in0 = x, out0 = y, alpha, beta
 *   REDUCE_SUM  in0 = x, out0 = s (m = 1, n = length)
 *   VECTOR_ADD  in0 = a, in1 = b, out0 = c (m = 1, n = length)
 *   GEMVER    A, in0..in5 = u1, v1, u2, v2, y, z, out0 = x, out1 = w,
 *             out2 = Ahat, alpha, beta
 * flush_buf / flush_bytes: optional device buffer the harness overwrites
 * before every timed sample so that no operand stays in the caches.
 */
typedef struct {
    int op;
    int dtype;
    int64_t m, n;
    const void* A;
    const void* B;
    const void* in0;
    const void* in1;
    void* out0;
    void* out1;
    double alpha, beta;
    void* ws;
    size_t ws_bytes;
    mep_stream_t stream;
    void* flush_buf;
    size_t flush_bytes;
    const void* in2;
    const void* in3;
    const void* in4;
    const void* in5;
    void* out2;
} mep_call_t;

/* Runs one call as described above (the same checks, the same kernels). */
int mep_run(const mep_call_t* call);

/*
 * Trimmed-mean timing of Eq. 3 (Sec. 3.2): `warmup` untimed calls, then R
 * samples; sample r is the elapsed device time (HIP events on call->stream)
 * of `inner` back-to-back calls divided by `inner`, preceded (outside the
 * timed interval) by a cache flush when flush != 0 and call->flush_buf is
 * set.  The samples are sorted, the k lowest and k highest dropped and the
 * remaining R - 2k averaged into *mean_ms.  samples_ms (nullable) receives
 * the R samples in run order.  Requires R > 2k >= 0, inner >= 1, warmup >= 0
 * (MEP_EBUDGET otherwise).  Synchronizes call->stream.  The paper uses R = 30,
 * k = 3 (Sec. 4.1.3).
 */
int mep_time_trimmed(const mep_call_t* call, int warmup, int R, int k, int inner, int flush,
                     double* mean_ms, double* samples_ms);

/*
 * Eq. 3 on host samples: mean of the sorted samples with the k lowest and k
 * highest removed, summed in ascending order.  NaN if R <= 2k or k < 0.
 */
double mep_trimmed_mean(const double* samples, int R, int k);

/*
 * Functional-equivalence check (Eq. 4; the paper asks that outputs agree): compares the
 * host copy `out` (len elements of dtype) with a host fp64 reference.
 * *err = max_i |out_i - ref_i| / max_i |ref_i| (normwise relative error);
 * +inf if any out_i is not finite, or if ref is all zero and out is not.
 * *pass = (*err <= tol).  len = 0 passes with *err = 0.  Every ref_i must be
 * finite (MEP_EINVAL otherwise: a NaN reference would compare as agreeing).
 */
int mep_check_fe(int dtype, const void* out, const double* ref, int64_t len, double tol,
                 double* err, int* pass);

/*
 * Kernel candidates (Sec. 3.2, Eqs. 4-5).  The paper's loop ranks N candidate
 * kernels per round by trimmed-mean time among those that pass FE.  Here the
 * candidates are the library's own hand-written kernel shapes for an
 * operation: mep_variant_count() gives how many there are for an op, dtype
 * and shape (>= 1; 0 on bad arguments), and mep_set_variant(op, v) makes
 * every later call of op use candidate v (-1 restores the default, candidate
 * 0; a v beyond the count of a later shape also means the default).
 * mep_workspace_bytes() already covers every candidate.  The setting is
 * process-wide; it changes speed only, never the checks or the contract.
 * The count and the descriptions assume 16-byte aligned operands (the vector
 * path) whenever the row length allows it; a call with unaligned operands
 * takes the element-wise path, whose list differs.  An index is kept per op
 * only: it means the candidate it named for the shape, dtype and load path
 * it was chosen on, and some other candidate (or the default) elsewhere.
 */
int mep_variant_count(int op, int dtype, int64_t m, int64_t n);
int mep_set_variant(int op, int variant);
/* Writes a short description of candidate `variant` for the shape into buf
 * (at most buf_len bytes, NUL-terminated): lanes per row group, vectors per
 * lane, rows per batch, waves per SIMD, load policy, grid (row workgroups x
 * column panels).  Returns MEP_OK,
 * or MEP_EINVAL for a bad op, dtype, shape or variant. */
int mep_variant_info(int op, int dtype, int64_t m, int64_t n, int variant, char* buf, size_t buf_len);

/*
 * One round of the candidate selection of Sec. 3.2 over the library's own
 * kernels for call->op at call's shape: candidate 0 (the default) is the
 * baseline K^(d).  The default first runs max(8, 2 * warmup) times untimed
 * (the first launches after an allocation or an idle gap read slower, and
 * candidate 0 is timed first); then every candidate n runs once and its
 * outputs are compared
 * with the baseline's by the FE metric of mep_check_fe (Eq. 4, tolerance
 * tol; every output of the call is judged on its own scale, GEMVER's Ahat
 * included, and a non-finite output fails, the baseline's too); each
 * candidate that passes is timed with mep_time_trimmed(warmup, R, k, inner,
 * flush) (Eq. 3); *best receives the argmin of the trimmed means over the
 * passing candidates, the lower index on ties (Eq. 5), or -1 when none
 * passes.  The candidates are those of the load path the call really takes
 * (its operands' alignment decides it, as for any call).  With
 * apply != 0 the winner becomes the op's variant (mep_set_variant), else the
 * previous setting is restored.  results (nullable, results_cap entries)
 * receives, per candidate, the trimmed mean (ms; NaN when not timed), the FE
 * error against the baseline (each output on its own scale, the worse of
 * the two) and the FE verdict.  With flush == 0 and a flush buffer in the
 * call, the caches are cleared once (by writing the buffer) before each
 * candidate runs, so that no candidate's warm timing inherits the cache
 * state another one left behind.  A GEMVER call must be out of place (out2 !=
 * A), else MEP_EINVAL: each in-place run changes A.  Stop rule: the paper
 * iterates until round D or until the gain falls below a threshold (Sec. 3.2,
 * after Eq. 5), each round generating new candidates.  Here the candidate set
 * is fixed, so a second round would only re-find the same argmin: one round
 * is the whole search, and the call takes neither D nor a threshold.
 * Synchronizes call->stream; overwrites the call's outputs.  While it runs,
 * the op's process-wide variant steps through the candidates: a call of the
 * same op from another host thread meanwhile runs whichever candidate is set
 * (each one correct; only its speed differs).
 */
typedef struct {
    double mean_ms;
    double fe_err;
    int fe_pass;
} mep_candidate_result_t;

int mep_select_variant(const mep_call_t* call, int warmup, int R, int k, int inner, int flush,
                       double tol, int apply, int* best, mep_candidate_result_t* results,
                       int results_cap);

/*
 * No passage of the paper defines the calls from here to the end of the
 * file: they are the library's own measurement and diagnostics.
 *
 * Device-time instrumentation of each operation's dominant kernel (the
 * matrix-streaming kernel; the first stage of the sum; the vector add).
 * mep_profile_begin(cap) arms up to cap records; while armed, every operation
 * launches its streaming kernel with a HIP event pair that the launch itself
 * stamps at the kernel's start and end (hipExtLaunchKernel), on the kernel's
 * own stream, so the timing adds no work to the stream.
 * mep_profile_end() synchronizes those events, returns the number of
 * recorded launches and their summed duration, and disarms.  Not thread-safe.
 */
int mep_profile_begin(int capacity);
/* As mep_profile_begin, but stamps only a sample of the launches: counting
 * the streaming-kernel launches from the call on (0, 1, 2, ...), launch i is
 * recorded when (i / group) % every == 0, i.e. the first `group` launches of
 * every `every` groups (group = the launches of one operation, so that
 * GEMVER's two passes stay paired).  Stamping a launch costs host time and a
 * little device time; sampling keeps that out of a timed loop.
 * mep_profile_begin(cap) is mep_profile_begin_sampled(cap, 1, 1).  MEP_EINVAL
 * for capacity, group or every below 1, or when already armed. */
int mep_profile_begin_sampled(int capacity, int group, int every);
int mep_profile_end(double* total_ms, int* launches);
/* As mep_profile_end, but also returns each recorded launch's duration in
 * launch order (up to cap entries; operations with two streaming passes, such
 * as GEMVER, record two launches per call). */
int mep_profile_end_samples(double* samples_ms, int cap, double* total_ms, int* launches);

/*
 * Plain device copy of `bytes` bytes (16-byte non-temporal loads and stores,
 * rows of 64 KiB streamed by up to 256 workgroups): the probe of the
 * read/write-mix ceiling (one byte written per byte read) and of the traffic
 * counters' calibration.  src and dst must be 16-byte aligned, must not
 * overlap, and bytes must be a multiple of 16.
 */
int mep_stream_copy(const void* src, void* dst, size_t bytes, mep_stream_t stream);

/* Description of the last error on the calling thread ("" if none). */
const char* mep_last_error(void);

/* Library version string. */
const char* mep_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MEP_H */
