/*
 * SparCML reference oracle -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, obviously-correct CPU implementation of what the
 * SparCML hot path computes (Renggli et al., "SparCML: High-Performance
 * Sparse Communication for Machine Learning", arXiv 1802.08021).  Only the
 * test-suite, the smoke check and the CPU-baseline leg of the benchmark may
 * load this library.  It shares no code, header, table or helper with the
 * HIP implementation under paper_1802_08021_amd/.
 *
 * All host pointers.  Return 0 on success, a negative value on bad input.
 */
#ifndef SPARCML_ORACLE_H
#define SPARCML_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11, "Parallel
 * random numbers: as easy as 1, 2, 3"): one block cipher evaluation. */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* Threads for work items that are independent by definition: the nodes of
 * one level of the reduction tree (and of App. A's step in front), the rows
 * of top-k, the streams of quantization.  Each item reads only its own
 * inputs and writes only its own outputs, so every result is the same bits
 * for any count.  Default 1 (plain loops); clamped to [1, 256].  Process-
 * wide; set it before, not during, calls from several threads. */
void orc_set_threads(int n);
int orc_get_threads(void);

/* Sparse allreduce of P sparse streams in recursive-doubling order with the
 * sparse->dense switch (SparCML §5.1 "Switching to a Dense Format" and
 * "Efficient Summation"; §5.3.1 recursive doubling, Fig. 2).
 *   idx[r], val[r], nnz[r]: stream r, indices strictly ascending and < N.
 *   delta: threshold as a fraction of N; thr = floor(delta * N).
 *   out_idx (capacity out_cap entries) / out_val (N floats) receive the root;
 *   *out_dense = 1 when the root is dense (out_val holds all N values).
 *   node_nnz / node_dense (P-1 entries each, may be NULL): per internal tree
 *   node in level order (level 1 groups first, root last), the union size
 *   (N for a dense node) and the switch decision.
 *   P need not be a power of two (App. A): with P2 the largest power of two
 *   <= P, a step in front sums rank P2+i into rank i for i < P-P2 (these
 *   P-P2 nodes come first in node_nnz / node_dense), then recursive
 *   doubling runs over the P2 participants.
 * Returns 0, -1 bad arguments, -2 unsorted / out-of-range input, -3 capacity,
 * -4 out of memory. */
int orc_sparse_reduce(int P, const uint32_t* const* idx, const float* const* val,
                      const uint64_t* nnz, uint64_t N, double delta,
                      uint32_t* out_idx, uint64_t out_cap, float* out_val,
                      uint64_t* out_nnz, int* out_dense,
                      uint64_t* node_nnz, uint8_t* node_dense);

/* Exact top-k by magnitude of each of P dense rows x[r*N .. r*N+N) by a full
 * sort (SparCML §2.2 "Structured Sparsification"; Alg. 1 TopK and the error
 * update).  Key = |x| as the IEEE bit pattern with the sign cleared; equal
 * keys are taken lowest index first.  Output per rank: k indices ascending
 * and the signed values.  residual (may be NULL, may alias x): x with the
 * selected positions set to +0. */
int orc_topk(int P, const float* x, uint64_t N, uint64_t k,
             uint32_t* out_idx, float* out_val, float* residual);

/* Bucketed top-k with the error feedback of Alg. 1 (SparCML §8.4: each
 * group of `bucket` consecutive coordinates sends its kb largest entries;
 * Alg. 1: acc = eps + alpha * grad, eps = acc - TopK(acc)).  grad and eps
 * are P rows of N; grad may be NULL (acc = eps).  Per bucket the min(kb,
 * len) largest magnitudes (key as in orc_topk, lowest index on ties), in
 * ascending index order; rank r's K = sum over buckets of min(kb, len)
 * entries start at out_idx/out_val + r*K.  eps is overwritten with acc, the
 * selected entries set to +0.  kb <= 64. */
int orc_topk_bucketed(int P, const float* grad, float* eps, uint64_t N, float alpha,
                      uint64_t bucket, uint64_t kb, uint32_t* out_idx, float* out_val);

/* QSGD stochastic quantization of each stream (SparCML §2.2 "Quantization",
 * §6; scale = the stream's L2 norm).  bits in {2,4,8}; s = 2^(bits-1)-1
 * levels plus a sign bit; codes packed 8/bits per byte, element j in byte
 * j/(8/bits) at bit (j%(8/bits))*bits.  Random draw for element j of stream
 * r: Philox4x32-10 word (j&3) of counter (j>>2, r, 0, 0), key (seed low,
 * seed high).  out_deq[r] (may be NULL) receives the dequantized values. */
int orc_quantize(int P, const float* const* val, const uint64_t* nnz, int bits,
                 uint64_t seed, uint8_t* const* out_q, float* out_scale,
                 float* const* out_deq);

/* Bucketed QSGD (SparCML §6: each stream split into buckets of B
 * consecutive entries, each quantized with its own scale, the bucket's L2
 * norm).  bucket = B >= 1, or 0 for one bucket per stream (orc_quantize).
 * Scales are flat: stream r's ceil(n_r/B) scales (1 when bucket = 0) follow
 * those of streams 0..r-1.  Random draws as in orc_quantize (by the
 * element's position in its stream). */
int orc_quantize_bucketed(int P, const float* const* val, const uint64_t* nnz, int bits,
                          uint64_t bucket, uint64_t seed, uint8_t* const* out_q,
                          float* out_scale, float* const* out_deq);

/* Dequantize n packed codes with the given scale (inverse of the above). */
int orc_dequantize(const uint8_t* q, float scale, int bits, uint64_t n, float* out);

/* Dequantize n packed codes of one stream quantized in buckets of B (scale
 * of element j: scales[j / B]; bucket = 0: scales[0] for all). */
int orc_dequantize_bucketed(const uint8_t* q, const float* scales, int bits, uint64_t bucket,
                            uint64_t n, float* out);

/* Dense representation of one sparse stream: D = 0, D[idx[i]] = val[i]. */
int orc_densify(const uint32_t* idx, const float* val, uint64_t nnz, uint64_t N,
                float* dense);

#ifdef __cplusplus
}
#endif
#endif
