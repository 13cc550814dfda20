// Internal declarations of the gfx950 SparCML library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sparcml {

// Device copy of one input stream descriptor (48 bytes).
struct StreamDesc {
    const uint32_t* idx;
    const float* val;
    const uint8_t* qval;
    const float* qscale;
    uint64_t nnz;
    uint64_t pad;
};

// Small host->device blobs travel as kernel arguments (no pageable copies).
constexpr int kBlobWords = 768;
struct Blob {
    uint32_t nwords;
    uint32_t words[kBlobWords];
};
hipError_t upload(void* dst, const void* src, size_t bytes, hipStream_t s);

// A reduce's stream descriptors as kernel arguments: whole descriptors (12
// words a stream, up to 64 streams), or 5 words a stream {idx, values or
// codes, nnz} (up to 153 streams) whose level units, for codes, are read
// at scale0 + r; kDescNone: the table was uploaded.
enum DescFmt : uint32_t { kDescNone = 0, kDescFull = 1, kDescValues = 2, kDescCodes = 3 };
struct DescArgs {
    uint32_t nwords;
    uint32_t fmt;
    const float* scale0;
    uint32_t words[kBlobWords];
};

// Optional kernel timing (see sparcml_timing_enable): HIP events recorded
// on the launch stream around the main kernels of each call.
enum TimerSlot {
    kTReducePass = 0,   // first tile pass of sparse_reduce (count or dense)
    kTReduceWrite = 1,  // sparse-output tile pass
    kTReduceSlow = 2,   // deferred-tile pass following the first tile pass
    kTQuantNorm = 3,    // QSGD norm partials
    kTQuantCodes = 4,   // QSGD coding pass
    kTTopkSelect = 5,   // top-k histogram passes
    kTTopkWrite = 6,    // top-k count + scan + write
    kTDensify = 7,
    kTConcat = 8,       // concatenation of disjoint parts
    kTTopkBuckets = 9,  // bucketed top-k with error feedback
    kTReduceMerge = 10, // small-data reduce: the whole merge tree in one workgroup
    kTSlots = 11
};
void timer_begin(int slot, hipStream_t s);
void timer_end(int slot, hipStream_t s);
int timer_enable(int on);
int timer_read(int slot, float* ms);

// Inclusive prefix sum over the 64 lanes of a wave: shifts within rows of
// 16 lanes, then the row broadcasts.
__device__ __forceinline__ uint32_t wave_scan(uint32_t v)
{
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xF, 0xF, true);  // row_shr:1
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xF, 0xF, true);  // row_shr:2
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xF, 0xF, true);  // row_shr:4
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xF, 0xF, true);  // row_shr:8
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xA, 0xF, false); // row_bcast:15
    v += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xC, 0xF, false); // row_bcast:31
    return v;
}

// 16-byte store marked nontemporal (streamed output that is not read back
// soon): it does not displace cached inputs, and measured on gfx950 it
// writes HBM markedly faster than a plain store.
__device__ __forceinline__ void store_nt(float* p, float4 v)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    const f4 x = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p));
}

// 16-byte load marked nontemporal (data streamed through once).
__device__ __forceinline__ float4 load_nt(const float* p)
{
    typedef float f4 __attribute__((ext_vector_type(4)));
    const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(p));
    return make_float4(x.x, x.y, x.z, x.w);
}

// Round x up to a multiple of a (a power of two).
inline size_t align_up(size_t x, size_t a) { return (x + a - 1) & ~(a - 1); }

// Bump allocator over a caller-provided workspace.
struct Carve {
    uint8_t* base;
    size_t used;
    explicit Carve(void* b) : base(static_cast<uint8_t*>(b)), used(0) {}
    template <class T>
    T* take(size_t count) {
        used = align_up(used, 256);
        T* p = reinterpret_cast<T*>(base ? base + used : nullptr);
        used += count * sizeof(T);
        return p;
    }
};

// ---------------------------------------------------------------- reduce
// The reduction covers the index range [lo, lo + N); stream indices lie in it.
struct ReducePlan {
    uint32_t P, L, PK, T, ntiles, nchunks, tiles_per_chunk, qbits;  // PK: rank class 16/32/64/128/256
    uint64_t N, lo, thr, sum_nnz, max_nnz;
    int speculate_dense;
    int small;  // few slots, every node sparse, few entries: the one-workgroup merge tree
    int seg;    // every node sparse, up to 64 slots: the segmented merge tree
    uint32_t nseg;
    uint64_t segw;
};
int reduce_plan(int P, uint64_t N, uint64_t max_nnz, uint64_t sum_nnz, double delta, int qbits,
                ReducePlan* plan, uint64_t lo = 0);
size_t reduce_workspace(const ReducePlan& p);

struct ReduceResult {
    uint64_t nnz;
    uint32_t dense;
    uint32_t pad;
};

// *r = {nnz, dense} on the device, in stream order.
hipError_t set_result_run(ReduceResult* r, uint64_t nnz, uint32_t dense, hipStream_t s);

// Enqueue the whole reduction.  dev_result == NULL: waits for the root
// header and writes it into *res (host).  Otherwise the header goes to
// dev_result (device) and nothing waits: the sparse-output passes are
// enqueued unconditionally and skip themselves on a dense root.
// node_nnz / node_dense receive the level-1 nodes g < nfold and every node
// above level 1 (nfold = P/2 reports all P - 1 nodes).  out_cap: entries
// out_idx holds; a sparse root is never written past it (header bit 1 if
// streams that do not ascend would have done so).
hipError_t reduce_run(const ReducePlan& p, const StreamDesc* host_tab, uint32_t* out_idx,
                      float* out_val, uint64_t* node_nnz, uint8_t* node_dense, void* ws,
                      hipStream_t s, ReduceResult* res, uint32_t nfold, ReduceResult* dev_result,
                      uint64_t out_cap);

// Small-data path: at most 8 slots holding at most thr entries together (so
// every node stays sparse), few enough that one workgroup's merge tree is
// faster than the tile pipeline.
bool merge_small_fits(uint32_t PT, uint64_t sum_nnz, uint64_t thr);
// The whole tree in one launch: root to out_idx / out_val, node sizes (in
// the order of reduce_run), header to hdr and, if not NULL, result.
hipError_t merge_small_run(uint32_t PT, uint32_t L, uint32_t qbits, uint32_t nfold, const StreamDesc* host_tab,
                           uint32_t* out_idx, float* out_val, uint64_t* node_nnz, uint8_t* node_dense,
                           ReduceResult* hdr, ReduceResult* result, hipStream_t s);

// Segmented merge path: at most 64 slots, every node sparse, at most
// kSegMaxEntries entries; the range cut into nseg segments of segw indices
// (merge_seg_shape), each merged by one workgroup.
constexpr uint64_t kSegEntries = 2048;                     // expected entries per segment
constexpr uint32_t kSegMax = 1024;                         // segments at most
constexpr uint64_t kSegMin = 128;                          // segments at least (when the range has as many indices)
constexpr uint64_t kSegMaxEntries = kSegEntries * kSegMax;  // inputs it takes at most
bool merge_seg_fits(uint32_t PT, uint64_t sum_nnz, uint64_t thr);
void merge_seg_shape(uint64_t R, uint64_t sum_nnz, uint32_t* nseg, uint64_t* segw);
// Counters of one segmented merge, zeroed before it (k_partition): node
// union sizes [64], ticket, finished workgroups, error flag, look-back words
// [nseg] (8-byte aligned).
struct SegState {
    uint32_t *node_cnt, *ticket, *done, *err;
    unsigned long long* flags;
};
constexpr uint32_t kSegStateWords = 68;  // words before the look-back words
hipError_t merge_seg_run(uint32_t PT, uint32_t L, uint32_t qbits, uint32_t nfold, const StreamDesc* dev_tab,
                         const uint32_t* off, const SegState& st, uint32_t nseg, uint64_t lo, uint64_t segw,
                         uint64_t N, uint32_t* out_idx, float* out_val, uint64_t* node_nnz, uint8_t* node_dense,
                         ReduceResult* hdr, ReduceResult* result, bool short_units, hipStream_t s);
// Whether segments of this many expected entries merge in short units.
bool merge_seg_short(uint64_t sum_nnz, uint32_t nseg);

// ---------------------------------------------------------------- densify
// dense[i] = the stream's value at index lo + i, i < N (+0.0 where it has none).
hipError_t densify_run(const uint32_t* idx, const float* val, const uint8_t* qval,
                       const float* qscale, uint32_t qbits, uint64_t nnz, uint64_t N,
                       int is_dense, float* dense, hipStream_t s, uint64_t lo = 0);
// out[i] = dequantized code i, i < n.
hipError_t dequant_run(const uint8_t* qval, const float* qscale, uint32_t qbits, uint64_t n,
                       float* out, hipStream_t s);

// ---------------------------------------------------------------- concat
// One part of a concatenation: indices in [lo, lo + len); dense parts hold
// len values.  qscale: one scale, or one per bucket of stored entries.
struct ConcatPart {
    const uint32_t* idx;
    const float* val;
    const uint8_t* qval;
    const float* qscale;
    uint64_t nnz, lo, len;
    int dense;
};
size_t concat_workspace(int P);
// bucket: 0 (one scale per part) or a power of two; dense: the result's
// representation (out_val holds the whole vector).
hipError_t concat_run(int P, const ConcatPart* parts, uint32_t qbits, uint64_t bucket, int dense,
                      uint32_t* out_idx, float* out_val, void* ws, hipStream_t s);

// ---------------------------------------------------------------- top-k
size_t topk_workspace(int P, uint64_t N, uint64_t k);
hipError_t topk_run(int P, const float* x, uint64_t N, uint64_t k, uint32_t* out_idx,
                    float* out_val, float* residual, void* ws, hipStream_t s);

// Bucketed top-k with error feedback: bucket = 64 * 2^j, 64..4096; kb <= 64.
uint64_t topk_buckets_count(uint64_t N, uint64_t bucket, uint64_t kb);
hipError_t topk_buckets_run(int P, const float* grad, float* eps, uint64_t N, float alpha, uint32_t bucket,
                            uint32_t kb, uint32_t* out_idx, float* out_val, hipStream_t s);

// ---------------------------------------------------------------- QSGD
size_t quant_workspace(int P, uint64_t max_n);
hipError_t quant_run(int P, const float* const* vals, const uint64_t* n, int bits, uint64_t seed,
                     uint8_t* const* out_q, float* out_scale, float* const* out_deq, void* ws,
                     hipStream_t s);
// Buckets of `bucket` entries (a power of two, 4..8192); scales flat, stream
// r's ceil(n_r / bucket) scales after those of streams 0..r-1.
size_t quant_buckets_workspace(int P);
hipError_t quant_buckets_run(int P, const float* const* vals, const uint64_t* n, int bits,
                             uint32_t bucket, uint64_t seed, uint8_t* const* out_q, float* out_scale,
                             float* const* out_deq, void* ws, hipStream_t s);

// ---------------------------------------------------------------- validate
// Every stream's indices strictly ascending inside [lo, hi); *bad_stream =
// -1 if so, else the first offending stream and position.  Synchronizes.
size_t validate_workspace(int P);
hipError_t validate_run(int P, const uint32_t* const* idx, const uint64_t* nnz, uint64_t lo, uint64_t hi,
                        void* ws, hipStream_t s, int* bad_stream, uint64_t* bad_pos);

}  // namespace sparcml
