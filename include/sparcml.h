/*
 * sparcml.h -- C ABI of the MI355X (gfx950) SparCML hot path.
 *
 * Implements the local reduction work of SparCML's sparse allreduce and its
 * two producers (Renggli et al., "SparCML: High-Performance Sparse
 * Communication for Machine Learning", arXiv 1802.08021):
 *
 *   sparcml_topk_sparsify  -- top-k sparsification of dense gradients
 *                             (§2.2 "Structured Sparsification", Alg. 1)
 *   sparcml_topk_bucketed  -- kb of every bucket of coordinates with the
 *                             error feedback of Alg. 1 (§8.4)
 *   sparcml_quantize       -- QSGD stochastic quantization (§2.2, §6)
 *   sparcml_quantize_bucketed -- QSGD in buckets of B entries (§6)
 *   sparcml_sparse_reduce  -- sum of P sparse streams in recursive-doubling
 *                             order with the sparse->dense switch
 *                             (§5.1, §5.3.1, Fig. 2)
 *   sparcml_sparse_reduce_range -- the same over one index range: a node's
 *                             share of the split phase of the large-data
 *                             allreduce (§5.3.2)
 *   sparcml_sparse_reduce_async -- either reduce without waiting (result
 *                             header written on the device)
 *   sparcml_sparse_reduce_async_noalloc -- the same with the library's own
 *                             fixed scratch array, for callers that cannot
 *                             allocate
 *   sparcml_concat         -- gathered shares summed as a concatenation
 *                             (§5.1 case (2), §5.3.2), QSGD parts decoded
 *   sparcml_densify        -- dense representation of one stream (§5.1)
 *   sparcml_validate_streams -- input check: indices strictly ascending
 *                             and in range (§5.1)
 *
 * Conventions shared by every call:
 *   - All data pointers are DEVICE pointers (HBM of the current HIP device),
 *     except the descriptor arrays (sparcml_stream[], pointer tables), which
 *     are HOST memory read during the call.
 *   - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *     Work is enqueued on it in order; sparcml_sparse_reduce(_range)
 *     additionally waits for its own result header (see there); the other
 *     calls return without synchronizing.
 *   - The caller owns every buffer.  The library never allocates, frees or
 *     keeps device memory between calls and has no global mutable state
 *     apart from the thread-local last-error message and timing events.  Scratch memory comes
 *     from the caller's workspace (size from sparcml_workspace_size).
 *     Calls on distinct streams with distinct workspaces may run
 *     concurrently.
 *   - Return value: SPARCML_OK (0) or a negative status.  Argument errors
 *     are detected on the host before any device work is enqueued; on error
 *     the outputs are unspecified.  No exception crosses the ABI.
 *   - Values are finite fp32; NaN/Inf inputs give unspecified results.
 */
#ifndef SPARCML_H
#define SPARCML_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__)
#define SPARCML_API __attribute__((visibility("default")))
#else
#define SPARCML_API
#endif

#define SPARCML_OK 0
#define SPARCML_EINVAL -1     /* bad argument (sizes, P, k, delta, bits, NULL pointers) */
#define SPARCML_ECAPACITY -2  /* output capacity too small for the result */
#define SPARCML_EWORKSPACE -3 /* workspace missing or smaller than required */
#define SPARCML_EUNSORTED -4  /* stream indices not strictly ascending or >= N */
#define SPARCML_EHIP -5       /* a HIP runtime call failed (see sparcml_last_error) */

/* Operation ids for sparcml_workspace_size. */
#define SPARCML_OP_TOPK 1
#define SPARCML_OP_QUANTIZE 2
#define SPARCML_OP_REDUCE 3
#define SPARCML_OP_DENSIFY 4
#define SPARCML_OP_QUANTIZE_BUCKETED 5
#define SPARCML_OP_CONCAT 6
#define SPARCML_OP_VALIDATE 7

/*
 * Sparse stream (§5.1 "Vector Representations" and "Switching to a Dense
 * Format"): a representation flag plus either index/value pairs or a dense
 * array.  Layout is structure-of-arrays.
 *   idx      sparse: nnz uint32 indices, strictly ascending, each < N.
 *   val      qbits == 0: sparse: nnz fp32 values; dense: N fp32 values.
 *   qval     qbits != 0: QSGD codes packed 8/qbits per byte, element j in
 *            byte j/(8/qbits) at bit (j%(8/qbits))*qbits; a code is
 *            (sign << (qbits-1)) | level, level in [0, 2^(qbits-1)-1].
 *   qscale   qbits != 0: device pointer to the stream's fp32 scale.
 *   nnz      number of stored pairs (N for a dense stream).
 *   is_dense representation flag.
 *   qbits    0 (fp32 values) or 2, 4, 8.
 */
typedef struct sparcml_stream {
    uint32_t* idx;
    float* val;
    uint8_t* qval;
    float* qscale;
    uint64_t nnz;
    uint32_t is_dense;
    uint32_t qbits;
} sparcml_stream;

/*
 * Workspace bytes needed by an operation.
 *   op       SPARCML_OP_*.
 *   P        number of ranks (streams / rows).
 *   N        dimension.
 *   max_nnz  TOPK: k; QUANTIZE: largest stream length; REDUCE: largest
 *            input stream nnz; DENSIFY, QUANTIZE_BUCKETED, CONCAT, VALIDATE:
 *            ignored.
 *   delta    REDUCE only (switch threshold as a fraction of N).
 * A workspace sized with max_nnz >= the actual largest nnz is sufficient.
 * Returns SPARCML_OK and *bytes, or SPARCML_EINVAL.
 */
SPARCML_API int sparcml_workspace_size(int op, int P, uint64_t N, uint64_t max_nnz, double delta,
                           size_t* bytes);

/*
 * Top-k sparsification by magnitude, per rank (§2.2 "Structured
 * Sparsification": each node keeps the k largest-magnitude components;
 * Alg. 1: eps = acc - TopK(acc)).
 *   P, N, k    x is P rows of N fp32 (row r at x + r*N), 1 <= N < 2^32,
 *              0 <= k <= N, 1 <= P <= 65535.
 *   out_idx    [P][k] uint32: the selected indices of row r, ascending.
 *   out_val    [P][k] fp32: x[r][out_idx[r][i]] (signed).
 *   residual   NULL, or [P][N] fp32 receiving x with the selected entries
 *              set to +0.0 (the error-feedback update).  May alias x, in
 *              which case only the k selected entries per row are written.
 * Ordering: magnitude = the IEEE bit pattern with the sign cleared; equal
 * magnitudes are taken lowest index first.
 * Errors: EINVAL (P outside [1, 65535], N == 0 or >= 2^32, k > N, NULL x /
 * outputs with k > 0), EWORKSPACE, EHIP.
 */
SPARCML_API int sparcml_topk_sparsify(int P, const float* x, uint64_t N, uint64_t k,
                          uint32_t* out_idx, float* out_val, float* residual,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * Bucketed top-k with error feedback, per rank (§8.4: each group of
 * `bucket` consecutive coordinates sends its kb largest entries and keeps
 * the rest locally; Alg. 1: acc = eps + alpha * grad, eps = acc -
 * TopK(acc)).  acc is formed in fp32 as a product then a sum (two
 * roundings).  Per bucket the min(kb, len) largest magnitudes (key and
 * ties as in sparcml_topk_sparsify), listed in ascending index order, so a
 * rank's output is one sorted sparse stream of K entries,
 *   K = (nb - 1) * kb + min(kb, N - (nb - 1) * bucket), nb = ceil(N / bucket)
 * (sparcml_topk_bucketed_count).
 *   P, N     grad and eps are P rows of N fp32 (row r at r * N), 1 <= P <=
 *            65535, 1 <= N < 2^32.
 *   grad     NULL (acc = eps) or the rows of the new gradient.
 *   eps      in: the accumulated error; out: acc with the selected entries
 *            set to +0.0.
 *   alpha    learning rate (finite).
 *   bucket   a power of two in [64, 4096]; kb in [1, 64].
 *   out_idx, out_val  [P][K]: rank r's entries at r * K.
 * No workspace; does not synchronize.
 * Errors: EINVAL, EHIP.
 */
SPARCML_API int sparcml_topk_bucketed(int P, const float* grad, float* eps, uint64_t N, float alpha,
                          uint64_t bucket, uint64_t kb, uint32_t* out_idx, float* out_val,
                          void* stream);

/* K of sparcml_topk_bucketed (0 for invalid sizes). */
SPARCML_API uint64_t sparcml_topk_bucketed_count(uint64_t N, uint64_t bucket, uint64_t kb);

/*
 * QSGD stochastic quantization of each stream's values (§2.2
 * "Quantization", §6 "Supporting Low-Precision Communication"): scale =
 * the stream's L2 norm (one bucket per stream); s = 2^(bits-1)-1 levels;
 * element v -> level l = floor(|v| s/scale) + [u < frac], u uniform in
 * [0,1), plus a sign bit; the dequantized value is +-l * (scale/s).
 *   P        number of streams, 1 <= P <= 65535.
 *   in       host array of P descriptors; in[r].val holds in[r].nnz fp32
 *            values, nnz <= 2^34 (the counter word j >> 2 below is 32 bits
 *            wide; longer streams would repeat draws); qbits must be 0;
 *            idx/is_dense are not read.
 *   bits     2, 4 or 8.
 *   seed     key of the Philox4x32-10 generator (Salmon et al., SC'11):
 *            element j of stream r uses word (j & 3) of the block at
 *            counter (j >> 2, r, 0, 0), key (seed & 0xffffffff, seed >> 32);
 *            u = (word >> 8) * 2^-24.  Results are deterministic in
 *            (seed, r, j).
 *   out_q    host array of P device pointers; out_q[r] receives
 *            ceil(nnz_r * bits / 8) bytes of packed codes (layout as in
 *            sparcml_stream.qval).
 *   out_scale device array of P fp32 scales.  The L2 norm is accumulated
 *            in fp64 over an adjacent-pair tree (zero-padded to a power of
 *            two) and rounded once to fp32.
 *   out_deq  NULL, or host array of P device pointers (entries may be NULL)
 *            receiving the dequantized fp32 values.
 * Errors: EINVAL, EWORKSPACE, EHIP.
 */
SPARCML_API int sparcml_quantize(int P, const sparcml_stream* in, int bits, uint64_t seed,
                     uint8_t* const* out_q, float* out_scale, float* const* out_deq,
                     void* ws, size_t ws_bytes, void* stream);

/*
 * Root header of an asynchronous reduction, written by the device.
 */
typedef struct sparcml_result {
    uint64_t nnz;      /* root nnz (the range's length if dense) */
    uint32_t is_dense; /* root representation */
    uint32_t reserved; /* 0; nonzero if the reduction could not complete: bit 0, a workgroup of
                          the all-sparse merge path gave up waiting for its predecessors' sizes
                          (never expected); bit 1, streams that do not ascend were met (the merge
                          path, or a sparse root that would not fit out->nnz entries: never
                          written past them).  The outputs are then incomplete */
} sparcml_result;

/*
 * Bucketed QSGD (§6 "Supporting Low-Precision Communication": a stream is
 * split into buckets of B consecutive entries, each quantized on its own
 * with a full-precision scale; the paper uses B in the order of 1024 and
 * applies it to the dense stage of the split-allgather allreduce).  Per
 * bucket exactly as sparcml_quantize per stream: scale = the bucket's L2
 * norm (fp64 adjacent-pair tree over its B entries, zeros past the stream's
 * end, one rounding to fp32), the same levels, codes and random draws
 * (element j of stream r: Philox word j&3 of counter (j>>2, r, 0, 0)).
 * One pass: each value is read once and its code written once.
 *   bucket   B, a power of two in [4, 8192].
 *   out_scale device fp32 array, flat: stream r's ceil(nnz_r / B) scales
 *            (in bucket order) follow those of streams 0..r-1.
 *   Other arguments as for sparcml_quantize.
 *   ws       sparcml_workspace_size(SPARCML_OP_QUANTIZE_BUCKETED, P, ...).
 * Errors: EINVAL (also for a bad bucket), EWORKSPACE, EHIP.
 */
SPARCML_API int sparcml_quantize_bucketed(int P, const sparcml_stream* in, int bits, uint64_t bucket,
                              uint64_t seed, uint8_t* const* out_q, float* out_scale,
                              float* const* out_deq, void* ws, size_t ws_bytes, void* stream);

/*
 * Sparse allreduce of P streams, one GPU's share: the sum of all ranks'
 * contributions, associated as the recursive-doubling rounds of §5.3.1
 * (round t sums adjacent blocks of 2^(t-1) ranks: node g of level t is
 * node 2g plus node 2g+1 of level t-1), with the representation switch of
 * §5.1: a node is dense if a child is dense or |H_L| + |H_R| > thr, where
 * thr = floor(delta * N) (computed in double) and |H| is a sparse child's
 * exact nnz (the union of its leaves' index sets); otherwise it is the
 * sorted union with values summed (fp32) where indices coincide.  Entries
 * whose sum is zero are kept.  A dense node holds the sum at every index
 * (+0.0 where no rank contributes).  For P == 1 the root is the single
 * stream, dense iff its nnz > thr.  For P not a power of two (App. A), with
 * P2 the largest power of two below P, a step in front sums rank P2+i into
 * rank i (i < P - P2; a tree node under the same rule), then recursive
 * doubling runs over the P2 participants.
 *   P        1 <= P <= 256.
 *   streams  host array of P sparse descriptors (is_dense == 0) with the
 *            same qbits (0 = fp32 val, or 2/4/8 = QSGD codes dequantized on
 *            the fly).  Indices strictly ascending and < N (not checked here:
 *            sparcml_validate_streams checks them).
 *   N        1 <= N < 2^32.   delta > 0 (fraction of N).
 *   out      in: out->idx (capacity out->nnz entries, must be >=
 *            min(thr, sum of input nnz), or >= nnz_0 when P == 1 and the
 *            stream stays sparse), out->val (N floats), out->qbits == 0.
 *            out: out->nnz = root nnz (N if dense), out->is_dense; a sparse
 *            root occupies out->idx[0..nnz) / out->val[0..nnz), a dense
 *            root out->val[0..N).
 *   node_nnz   NULL or device uint64[P-1]: union size of every internal
 *              node (N for dense nodes), level order: level-1 nodes first
 *              (g ascending), root last; for P not a power of two the
 *              P - P2 nodes of the step in front come first.
 *   node_dense NULL or device uint8[P-1]: switch decision per node.
 * Synchronization: the call reads back a 16-byte result header from the
 * device and therefore waits for its own work on `stream`.
 * Errors: EINVAL (including P outside [1, 256] or mixed qbits), ECAPACITY (out->nnz
 * below the capacity stated above), EWORKSPACE, EHIP; all but EHIP are
 * detected before any device work is enqueued.  Streams that do not ascend
 * give undefined sums but no write past the outputs: where the device sees
 * them (the all-sparse merge path, or a sparse root that would not fit
 * out->nnz entries) the call returns EUNSORTED.
 */
SPARCML_API int sparcml_sparse_reduce(int P, const sparcml_stream* streams, uint64_t N, double delta,
                          sparcml_stream* out, uint64_t* node_nnz, uint8_t* node_dense,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * One GPU's share of the split phase of the large-data allreduce (§5.3.2,
 * the split-allgather / DSAR scheme): the sum of P streams restricted to
 * the index range [lo, hi) of a vector of N, with the same recursive-
 * doubling association and representation switch as sparcml_sparse_reduce
 * applied to the range as if it were the whole vector: thr =
 * floor(delta * (hi - lo)), a dense node holds hi - lo values.  Each
 * stream is the part of a rank's stream whose indices lie in [lo, hi)
 * (strictly ascending, not checked).  With lo == 0 and hi == N this is
 * sparcml_sparse_reduce.
 *   lo, hi   0 <= lo < hi <= N, N < 2^32.
 *   out      in: as for sparcml_sparse_reduce with hi - lo in place of N
 *            (out->val holds hi - lo floats).
 *            out: a sparse root holds absolute indices (in [lo, hi)); a
 *            dense root holds out->val[i] = sum at index lo + i, i < hi - lo.
 *   node_nnz, node_dense: as for sparcml_sparse_reduce (dense nodes count
 *            hi - lo).
 *   ws       sparcml_workspace_size(SPARCML_OP_REDUCE, P, hi - lo, ...).
 * Errors: as for sparcml_sparse_reduce; EINVAL also for lo >= hi, hi > N,
 * or a stream with more than hi - lo entries.
 */
SPARCML_API int sparcml_sparse_reduce_range(int P, const sparcml_stream* streams, uint64_t N,
                                uint64_t lo, uint64_t hi, double delta, sparcml_stream* out,
                                uint64_t* node_nnz, uint8_t* node_dense, void* ws,
                                size_t ws_bytes, void* stream);

/*
 * sparcml_sparse_reduce_range without any host round trip: the same
 * computation and outputs, but the root header goes to `result` (DEVICE
 * memory, written in stream order) instead of being read back, and the call
 * returns once the work is enqueued.  The passes that write a sparse root
 * are always enqueued and return at once on the device when the root is
 * dense, so the call enqueues the same work whatever the data, never waits,
 * and can be captured in a HIP graph (it issues no memset and no host copy;
 * the descriptor table travels in kernel arguments).  With lo == 0 and
 * hi == N it is sparcml_sparse_reduce.
 *   out      read only: out->idx (capacity out->nnz, as for
 *            sparcml_sparse_reduce) and out->val; out itself is not
 *            written.
 *   result   device pointer to one sparcml_result.
 * Errors: as for sparcml_sparse_reduce_range, EINVAL for a NULL result.
 */
SPARCML_API int sparcml_sparse_reduce_async(int P, const sparcml_stream* streams, uint64_t N, uint64_t lo,
                                uint64_t hi, double delta, const sparcml_stream* out,
                                uint64_t* node_nnz, uint8_t* node_dense, sparcml_result* result,
                                void* ws, size_t ws_bytes, void* stream);

/*
 * sparcml_sparse_reduce_async for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same computation, arguments and outputs, without
 * a workspace argument.  Its scratch memory is a fixed device array of
 * SPARCML_NOALLOC_SCRATCH_BYTES inside the library, which each GPU the
 * library runs on holds until the process ends; the call allocates nothing
 * (no hipMalloc, no hipFree, no allocating library routine).
 *   Limit: a reduce whose workspace (sparcml_workspace_size, OP_REDUCE)
 *   exceeds SPARCML_NOALLOC_SCRATCH_BYTES is rejected with EWORKSPACE
 *   before any device work (16 MiB covers, e.g., every P <= 256 at
 *   N <= 2^31 and P >= 33 at any N < 2^32).
 *   Sharing: every call on one GPU uses that GPU's one array, and the array
 *   keeps the last call's contents (the call initializes what it reads).
 *   Calls that overlap on one GPU (concurrent streams, threads or
 *   processes) race on it; calls in one stream's order do not.
 * Errors: as for sparcml_sparse_reduce_async, EWORKSPACE for sizes above the
 * limit, EHIP if the array's address cannot be obtained.
 */
#define SPARCML_NOALLOC_SCRATCH_BYTES (16u << 20)
SPARCML_API int sparcml_sparse_reduce_async_noalloc(int P, const sparcml_stream* streams, uint64_t N,
                                        uint64_t lo, uint64_t hi, double delta,
                                        const sparcml_stream* out, uint64_t* node_nnz,
                                        uint8_t* node_dense, sparcml_result* result, void* stream);

/*
 * The allgather phase of the split-allgather allreduce (§5.3.2), the local
 * part: the sum of P parts with disjoint index ranges, which is their
 * concatenation (§5.1, case (2)).  Part s covers [bounds[s], bounds[s+1]).
 * The result is dense if a part is dense or the parts hold more than
 * thr = floor(delta * N) entries together (the representation rule of
 * §5.1); a dense result is +0.0 where no part has an entry.  QSGD-coded
 * parts (§6: DSAR's dense stage is sent quantized) are dequantized.
 *   P        1 <= P <= 65535.
 *   parts    host array of P descriptors, all with the same qbits.  Sparse
 *            part: nnz <= its range's length, absolute indices strictly
 *            ascending inside the range (not checked).  Dense part
 *            (is_dense): nnz == its range's length, value i is index
 *            bounds[s] + i.  qbits != 0: codes in qval; qscale holds one
 *            scale (bucket == 0) or ceil(nnz / bucket) scales, entry i of
 *            the part using scale i / bucket.
 *   bounds   host array of P + 1: bounds[0] == 0, bounds[P] == N, not
 *            decreasing (empty ranges allowed).
 *   N, delta 1 <= N < 2^32, delta > 0.
 *   bucket   0 or a power of two in [4, 8192] (read only when qbits != 0).
 *   out      in: out->val (N floats), out->idx (capacity out->nnz entries,
 *            at least the parts' total when the result stays sparse),
 *            out->qbits == 0.  out: out->nnz (N if dense), out->is_dense; a
 *            sparse result is the parts' entries in part order (ascending),
 *            values in fp32.
 *   ws       sparcml_workspace_size(SPARCML_OP_CONCAT, P, ...).
 * The representation is decided on the host from the descriptors; the call
 * does not synchronize.
 * Errors: EINVAL, ECAPACITY, EWORKSPACE, EHIP.
 */
SPARCML_API int sparcml_concat(int P, const sparcml_stream* parts, const uint64_t* bounds, uint64_t N,
                   double delta, uint64_t bucket, sparcml_stream* out, void* ws, size_t ws_bytes,
                   void* stream);

/*
 * Checks what the reduction assumes of its input streams and does not check
 * itself (§5.1 "Vector Representations": a sparse vector is a list of
 * index/value pairs; the merges need each list sorted): every sparse stream's
 * indices strictly ascending (no duplicates) and inside [lo, hi) -- [0, N)
 * for a whole vector.  A read-only pass over the indices.
 *   P        1 <= P <= 65535.
 *   streams  host array of P descriptors; only idx and nnz are read (idx
 *            may be NULL when nnz == 0); dense descriptors are EINVAL.
 *   lo, hi   lo < hi <= 2^32.
 *   ws       sparcml_workspace_size(SPARCML_OP_VALIDATE, P, ...) bytes.
 * Returns SPARCML_OK, or SPARCML_EUNSORTED with the first offending stream
 * and position (lowest stream first) in sparcml_last_error().  Waits for
 * its own work on `stream` (it reads back one 8-byte result).
 * Errors: EINVAL, EWORKSPACE, EHIP.
 */
SPARCML_API int sparcml_validate_streams(int P, const sparcml_stream* streams, uint64_t lo, uint64_t hi,
                             void* ws, size_t ws_bytes, void* stream);

/*
 * Index ranges of a P-way split of [0, N): which coordinates each node
 * reduces in the split phase of the large-data allreduce (§5.3.2), with
 * the rule App. A ("Relaxation of Assumption") gives for N not divisible by
 * P: every node but the last is responsible for floor(N/P) indices, the
 * last for the remaining N - (P-1) floor(N/P).  So bounds[s] = s * floor(N/P)
 * for s < P and bounds[P] = N; node s covers [bounds[s], bounds[s+1]) (empty
 * ranges when N < P).
 *   P        1 <= P <= 65535.   N  1 <= N < 2^32.
 *   bounds   host array of P + 1 uint64 (written).
 * Host only: no device work.  Errors: EINVAL.
 */
SPARCML_API int sparcml_split_bounds(int P, uint64_t N, uint64_t* bounds);

/*
 * Dense representation of one stream (§5.1): dense[j] = value of index j,
 * +0.0 where absent; dequantizes QSGD codes on the fly.  A dense input is
 * copied (or dequantized).  Writes all N floats.  Indices must be strictly
 * ascending and < N (not checked).
 * Errors: EINVAL (NULL pointers, N == 0 or >= 2^32, nnz > N, bad qbits),
 * EHIP.
 */
SPARCML_API int sparcml_densify(const sparcml_stream* in, uint64_t N, float* dense, void* stream);

/*
 * Kernel timing for benchmarks and profiling (off by default; per calling
 * thread).  While enabled, each call records a pair of HIP events on its
 * stream around each of its main kernels; sparcml_timing_read returns the
 * mean duration (ms) over every launch of one kernel group since timing was
 * enabled, waiting for their stop events (so it can be called once after a
 * timed loop without synchronizing inside it).  Groups: SPARCML_TIMER_*.
 * Enabling or disabling forgets earlier records; event pairs are created on
 * first use and kept for reuse by the calling thread.
 * sparcml_timing_read returns EINVAL when the group has no record.
 */
#define SPARCML_TIMER_REDUCE_PASS 0  /* first tile pass of sparse_reduce */
#define SPARCML_TIMER_REDUCE_WRITE 1 /* sparse-output tile pass */
#define SPARCML_TIMER_REDUCE_SLOW 2  /* pass over tiles too full for the first pass */
#define SPARCML_TIMER_QUANT_NORM 3   /* QSGD norm partials */
#define SPARCML_TIMER_QUANT_CODES 4  /* QSGD coding */
#define SPARCML_TIMER_TOPK_SELECT 5  /* top-k radix-select histogram passes */
#define SPARCML_TIMER_TOPK_WRITE 6   /* top-k count, scan and write */
#define SPARCML_TIMER_DENSIFY 7
#define SPARCML_TIMER_CONCAT 8
#define SPARCML_TIMER_TOPK_BUCKETED 9
#define SPARCML_TIMER_REDUCE_MERGE 10 /* small-data reduce: the whole merge tree in one workgroup */
SPARCML_API int sparcml_timing_enable(int on);
SPARCML_API int sparcml_timing_read(int group, float* ms);

/* Static description of a status code. */
SPARCML_API const char* sparcml_strerror(int status);

/* Detail of the last error on the calling thread ("" if none). */
SPARCML_API const char* sparcml_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SPARCML_H */
