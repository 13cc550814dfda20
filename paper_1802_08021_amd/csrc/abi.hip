// C ABI entry points (declared in include/sparcml.h): argument validation on
// the host, workspace checks, then the device passes.
#include "../../include/sparcml.h"
#include "internal.h"

#include <math.h>
#include <stddef.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <exception>
#include <mutex>
#include <vector>

static_assert(sizeof(sparcml_result) == sizeof(sparcml::ReduceResult) &&
                  offsetof(sparcml_result, nnz) == offsetof(sparcml::ReduceResult, nnz) &&
                  offsetof(sparcml_result, is_dense) == offsetof(sparcml::ReduceResult, dense),
              "the device writes sparcml_result as a ReduceResult");

using namespace sparcml;

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char* where)
{
    return fail(SPARCML_EHIP, "%s: %s", where, hipGetErrorString(e));
}

bool valid_n(uint64_t N) { return N >= 1 && N < (1ull << 32); }
bool valid_bits(uint32_t b) { return b == 2 || b == 4 || b == 8; }
bool is_pow2(int p) { return p >= 1 && (p & (p - 1)) == 0; }

int reduce_validate(int P, const sparcml_stream* streams, uint64_t N, double delta, uint32_t* qbits,
                    uint64_t* max_nnz, uint64_t* sum_nnz)
{
    if (P < 1 || P > 256) return fail(SPARCML_EINVAL, "P must be in [1, 256] (got %d)", P);
    if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
    if (!(delta > 0.0) || isnan(delta)) return fail(SPARCML_EINVAL, "delta must be > 0");
    if (!streams) return fail(SPARCML_EINVAL, "streams is NULL");
    *qbits = streams[0].qbits;
    *max_nnz = 0;
    *sum_nnz = 0;
    for (int r = 0; r < P; ++r) {
        const sparcml_stream& s = streams[r];
        if (s.is_dense) return fail(SPARCML_EINVAL, "stream %d: inputs must be sparse", r);
        if (s.qbits != *qbits) return fail(SPARCML_EINVAL, "stream %d: all streams must share qbits", r);
        if (s.qbits && !valid_bits(s.qbits)) return fail(SPARCML_EINVAL, "stream %d: qbits must be 0, 2, 4 or 8", r);
        if (s.nnz > N) return fail(SPARCML_EINVAL, "stream %d: nnz > N", r);
        if (s.qbits && !s.qscale) return fail(SPARCML_EINVAL, "stream %d: qscale is NULL", r);
        if (s.nnz) {
            if (!s.idx) return fail(SPARCML_EINVAL, "stream %d: idx is NULL", r);
            if (s.qbits ? !s.qval : !s.val) return fail(SPARCML_EINVAL, "stream %d: values are NULL", r);
        }
        *max_nnz = std::max(*max_nnz, s.nnz);
        *sum_nnz += s.nnz;
    }
    return SPARCML_OK;
}

bool valid_bucket(uint64_t b) { return b >= 4 && b <= 8192 && (b & (b - 1)) == 0; }

// Shared argument checks of the QSGD entry points.
int quant_validate(int P, const sparcml_stream* in, int bits, uint8_t* const* out_q, float* out_scale,
                   std::vector<const float*>* vals, std::vector<uint64_t>* n, uint64_t* max_n)
{
    if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
    if (!valid_bits((uint32_t)bits)) return fail(SPARCML_EINVAL, "bits must be 2, 4 or 8");
    if (!in || !out_q || !out_scale) return fail(SPARCML_EINVAL, "NULL argument");
    vals->assign(P, nullptr);
    n->assign(P, 0);
    *max_n = 0;
    for (int r = 0; r < P; ++r) {
        if (in[r].qbits) return fail(SPARCML_EINVAL, "stream %d: input must hold fp32 values", r);
        // the random draw of element j comes from counter word j >> 2 (32 bits)
        if (in[r].nnz > (1ull << 34))
            return fail(SPARCML_EINVAL, "stream %d: more than 2^34 entries (the Philox counter word is 32 bits)", r);
        if (in[r].nnz && (!in[r].val || !out_q[r])) return fail(SPARCML_EINVAL, "stream %d: NULL pointer", r);
        (*vals)[r] = in[r].val;
        (*n)[r] = in[r].nnz;
        *max_n = std::max(*max_n, (*n)[r]);
    }
    return SPARCML_OK;
}

// Ranks of the power-of-two tree that the kernels reduce.  For P not a
// power of two (App. A), with P2 the largest power of two below P, rank P2+i
// is summed into rank i first (i < P - P2), then recursive doubling runs
// over the P2 participants.  That is the tree over 2*P2 ranks in which
// participant i sits at 2i and its partner P2+i at 2i+1 (empty for i >=
// P - P2): level 1 is the step in front, the levels above it recursive
// doubling.
int tree_ranks(int P)
{
    if (is_pow2(P)) return P;
    int P2 = 1;
    while (2 * P2 <= P) P2 *= 2;
    return 2 * P2;
}

// Workspace of a reduce of P streams over N indices, enough for fp32 values
// and for QSGD codes alike.
size_t reduce_ws_any(int P, uint64_t N, uint64_t max_nnz, double delta)
{
    ReducePlan p0, pq;
    reduce_plan(tree_ranks(P), N, max_nnz, (uint64_t)P * max_nnz, delta, 0, &p0);
    reduce_plan(tree_ranks(P), N, max_nnz, (uint64_t)P * max_nnz, delta, 4, &pq);
    return std::max(reduce_workspace(p0), reduce_workspace(pq));
}

uint64_t threshold(uint64_t N, double delta)
{
    const double t = floor(delta * (double)N);
    return t >= 18446744073709551615.0 ? UINT64_MAX : (uint64_t)t;
}

// The reduction of the index range [lo, hi) of N (the whole vector: [0, N)):
// every stream's indices lie in the range; a dense result holds hi - lo
// values (index lo + i at i), a sparse one absolute indices.  result ==
// NULL: the root header is read back into *out; otherwise it is written to
// result (device) and the call does not wait.
// ------------------------------------------------------------------------
// Scratch memory of sparcml_sparse_reduce_async_noalloc (for callers that
// cannot allocate): a file-scope device array, which every GPU the library
// runs on holds until the process ends.  In host code `scratch` names a
// host-side stand-in, not device memory: host code only ever uses the
// per-device address hipGetSymbolAddress returns for it.
static __device__ __align__(256) uint8_t scratch[SPARCML_NOALLOC_SCRATCH_BYTES];

constexpr int kScratchDevs = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevs];  // device address of `scratch`, per device

// Address of the current device's `scratch`, looked up on the first call on
// that device (with it current) and kept.
int scratch_on_current_device(void** ptr)
{
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev < 0 || dev >= kScratchDevs)
        return fail(SPARCML_EINVAL, "device %d: the scratch table covers devices 0..%d", dev, kScratchDevs - 1);
    std::lock_guard<std::mutex> g(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!p) return fail(SPARCML_EHIP, "hipGetSymbolAddress(scratch) returned NULL");
        g_scratch_ptr[dev] = p;
    }
    *ptr = g_scratch_ptr[dev];
    return SPARCML_OK;
}

// use_scratch: the workspace is the current device's `scratch` (ws and
// ws_bytes are ignored); a call that needs more is rejected.
int reduce_impl(int P, const sparcml_stream* streams, uint64_t N, uint64_t lo, uint64_t hi, double delta,
                sparcml_stream* out, uint64_t* node_nnz, uint8_t* node_dense, void* ws, size_t ws_bytes,
                void* stream, sparcml_result* result = nullptr, bool use_scratch = false)
{
    try {
        uint32_t qbits;
        uint64_t max_nnz, sum_nnz;
        int rc = reduce_validate(P, streams, N, delta, &qbits, &max_nnz, &sum_nnz);
        if (rc) return rc;
        const uint64_t R = hi - lo;  // range size
        if (max_nnz > R) return fail(SPARCML_EINVAL, "a stream has more entries than the range has indices");
        if (!out || !out->val) return fail(SPARCML_EINVAL, "out / out->val is NULL");
        if (out->qbits) return fail(SPARCML_EINVAL, "out->qbits must be 0");
        const uint64_t thr = threshold(R, delta);
        const hipStream_t s = (hipStream_t)stream;
        hipError_t e;

        ReduceResult* dres = reinterpret_cast<ReduceResult*>(result);
        if (P == 1) {
            const sparcml_stream& a = streams[0];
            if (a.nnz > thr) {
                e = densify_run(a.idx, a.val, a.qval, a.qscale, qbits, a.nnz, R, 0, out->val, s, lo);
                if (e == hipSuccess && dres) e = set_result_run(dres, R, 1, s);
                if (e != hipSuccess) return hip_fail(e, "densify");
                if (!dres) {
                    out->nnz = R;
                    out->is_dense = 1;
                }
                return SPARCML_OK;
            }
            if (a.nnz && !out->idx) return fail(SPARCML_EINVAL, "out->idx is NULL");
            if (out->nnz < a.nnz) return fail(SPARCML_ECAPACITY, "out capacity %llu < %llu",
                                              (unsigned long long)out->nnz, (unsigned long long)a.nnz);
            if (a.nnz) {
                e = hipMemcpyAsync(out->idx, a.idx, a.nnz * sizeof(uint32_t), hipMemcpyDeviceToDevice, s);
                if (e == hipSuccess)
                    e = qbits ? dequant_run(a.qval, a.qscale, qbits, a.nnz, out->val, s)
                              : hipMemcpyAsync(out->val, a.val, a.nnz * sizeof(float),
                                               hipMemcpyDeviceToDevice, s);
                if (e != hipSuccess) return hip_fail(e, "copy");
            }
            if (dres) {
                if ((e = set_result_run(dres, a.nnz, 0, s)) != hipSuccess) return hip_fail(e, "result");
            } else {
                out->nnz = a.nnz;
                out->is_dense = 0;
            }
            return SPARCML_OK;
        }

        const uint64_t cap = std::min(thr, sum_nnz);
        if (cap && !out->idx) return fail(SPARCML_EINVAL, "out->idx is NULL");
        if (out->nnz < cap)
            return fail(SPARCML_ECAPACITY, "out capacity %llu < min(thr, sum nnz) = %llu",
                        (unsigned long long)out->nnz, (unsigned long long)cap);
        const int PT = tree_ranks(P);
        ReducePlan plan;
        reduce_plan(PT, R, max_nnz, sum_nnz, delta, (int)qbits, &plan, lo);
        const size_t need = reduce_workspace(plan);
        if (use_scratch) {
            if (need > (size_t)SPARCML_NOALLOC_SCRATCH_BYTES)
                return fail(SPARCML_EWORKSPACE,
                            "this reduce needs %zu bytes of scratch; the allocation-free entry point holds %zu",
                            need, (size_t)SPARCML_NOALLOC_SCRATCH_BYTES);
            rc = scratch_on_current_device(&ws);
            if (rc) return rc;
            ws_bytes = SPARCML_NOALLOC_SCRATCH_BYTES;
        }
        if (!ws || ws_bytes < need) return fail(SPARCML_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);

        // tree slot of every rank; empty slots keep a readable scale pointer
        // (a fixed array: the reduce path makes no host allocation)
        StreamDesc tab[256];
        for (int r = 0; r < PT; ++r) tab[r] = StreamDesc{nullptr, nullptr, nullptr, streams[0].qscale, 0, 0};
        const int P2 = PT == P ? P : PT / 2;
        for (int r = 0; r < P; ++r) {
            const int slot = PT == P ? r : (r < P2 ? 2 * r : 2 * (r - P2) + 1);
            tab[slot] = StreamDesc{streams[r].idx, streams[r].val, streams[r].qval, streams[r].qscale,
                                   streams[r].nnz, 0};
        }
        const uint32_t nfold = PT == P ? (uint32_t)(P / 2) : (uint32_t)(P - P2);
        ReduceResult res{};
        e = reduce_run(plan, tab, out->idx, out->val, node_nnz, node_dense, ws, s, &res, nfold, dres, out->nnz);
        if (e != hipSuccess) return hip_fail(e, "sparse_reduce");
        if (!dres && (res.pad & 2u))
            return fail(SPARCML_EUNSORTED, "sparse_reduce: streams that do not ascend were met; "
                                           "the outputs are incomplete");
        if (!dres && res.pad)
            return fail(SPARCML_EHIP, "sparse_reduce: a segment of the merge path gave up waiting for its "
                                      "predecessors' sizes; the outputs are incomplete");
        if (!dres) {
            out->nnz = res.nnz;
            out->is_dense = res.dense;
        }
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

}  // namespace

extern "C" {

const char* sparcml_strerror(int status)
{
    switch (status) {
    case SPARCML_OK: return "success";
    case SPARCML_EINVAL: return "invalid argument";
    case SPARCML_ECAPACITY: return "output capacity too small";
    case SPARCML_EWORKSPACE: return "workspace missing or too small";
    case SPARCML_EUNSORTED: return "stream indices not strictly ascending or out of range";
    case SPARCML_EHIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

const char* sparcml_last_error(void) { return g_last_error; }

int sparcml_timing_enable(int on) { return timer_enable(on); }

int sparcml_timing_read(int group, float* ms)
{
    const int rc = timer_read(group, ms);
    if (rc == -1) return fail(SPARCML_EINVAL, "no timing record for group %d", group);
    if (rc != 0) return fail(SPARCML_EHIP, "event query failed");
    return SPARCML_OK;
}

int sparcml_workspace_size(int op, int P, uint64_t N, uint64_t max_nnz, double delta, size_t* bytes)
{
    if (!bytes) return fail(SPARCML_EINVAL, "bytes is NULL");
    switch (op) {
    case SPARCML_OP_TOPK:
        if (P < 1 || P > 65535 || !valid_n(N) || max_nnz > N) return fail(SPARCML_EINVAL, "bad top-k sizes");
        *bytes = max_nnz ? topk_workspace(P, N, max_nnz) : 0;
        return SPARCML_OK;
    case SPARCML_OP_QUANTIZE:
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        *bytes = quant_workspace(P, max_nnz);
        return SPARCML_OK;
    case SPARCML_OP_QUANTIZE_BUCKETED:
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        *bytes = quant_buckets_workspace(P);
        return SPARCML_OK;
    case SPARCML_OP_CONCAT:
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        *bytes = concat_workspace(P);
        return SPARCML_OK;
    case SPARCML_OP_REDUCE: {
        if (P < 1 || P > 256 || !valid_n(N) || !(delta > 0.0) || max_nnz > N)
            return fail(SPARCML_EINVAL, "bad reduce sizes");
        // the call's sum of nnz is at most P * max_nnz, which never needs a
        // smaller workspace than the call itself; the plan of fp32 values and
        // that of QSGD codes may differ (kernel occupancy), so the larger
        *bytes = P == 1 ? 0 : reduce_ws_any(P, N, max_nnz, delta);
        return SPARCML_OK;
    }
    case SPARCML_OP_DENSIFY:
        *bytes = 0;
        return SPARCML_OK;
    case SPARCML_OP_VALIDATE:
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        *bytes = validate_workspace(P);
        return SPARCML_OK;
    default: return fail(SPARCML_EINVAL, "unknown op %d", op);
    }
}

int sparcml_topk_sparsify(int P, const float* x, uint64_t N, uint64_t k, uint32_t* out_idx,
                          float* out_val, float* residual, void* ws, size_t ws_bytes, void* stream)
{
    try {
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
        if (k > N) return fail(SPARCML_EINVAL, "k > N");
        if (!x) return fail(SPARCML_EINVAL, "x is NULL");
        if (k && (!out_idx || !out_val)) return fail(SPARCML_EINVAL, "outputs are NULL");
        const size_t need = k ? topk_workspace(P, N, k) : 0;
        if (need && (!ws || ws_bytes < need))
            return fail(SPARCML_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
        hipError_t e = topk_run(P, x, N, k, out_idx, out_val, residual, ws, (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "topk");
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

int sparcml_topk_bucketed(int P, const float* grad, float* eps, uint64_t N, float alpha, uint64_t bucket,
                          uint64_t kb, uint32_t* out_idx, float* out_val, void* stream)
{
    try {
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
        if (bucket < 64 || bucket > 4096 || (bucket & (bucket - 1)))
            return fail(SPARCML_EINVAL, "bucket must be a power of two in [64, 4096]");
        if (kb < 1 || kb > 64) return fail(SPARCML_EINVAL, "kb must be in [1, 64]");
        if (!eps || !out_idx || !out_val) return fail(SPARCML_EINVAL, "NULL argument");
        if (isnan(alpha) || isinf(alpha)) return fail(SPARCML_EINVAL, "alpha must be finite");
        hipError_t e = topk_buckets_run(P, grad, eps, N, alpha, (uint32_t)bucket, (uint32_t)kb, out_idx,
                                        out_val, (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "topk_bucketed");
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

uint64_t sparcml_topk_bucketed_count(uint64_t N, uint64_t bucket, uint64_t kb)
{
    if (!valid_n(N) || bucket == 0 || kb == 0) return 0;
    return topk_buckets_count(N, bucket, kb);
}

int sparcml_quantize(int P, const sparcml_stream* in, int bits, uint64_t seed, uint8_t* const* out_q,
                     float* out_scale, float* const* out_deq, void* ws, size_t ws_bytes, void* stream)
{
    try {
        std::vector<const float*> vals;
        std::vector<uint64_t> n;
        uint64_t max_n = 0;
        int rc = quant_validate(P, in, bits, out_q, out_scale, &vals, &n, &max_n);
        if (rc) return rc;
        const size_t need = quant_workspace(P, max_n);
        if (!ws || ws_bytes < need) return fail(SPARCML_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
        hipError_t e = quant_run(P, vals.data(), n.data(), bits, seed, out_q, out_scale, out_deq, ws,
                                 (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "quantize");
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

int sparcml_quantize_bucketed(int P, const sparcml_stream* in, int bits, uint64_t bucket, uint64_t seed,
                              uint8_t* const* out_q, float* out_scale, float* const* out_deq, void* ws,
                              size_t ws_bytes, void* stream)
{
    try {
        std::vector<const float*> vals;
        std::vector<uint64_t> n;
        uint64_t max_n = 0;
        int rc = quant_validate(P, in, bits, out_q, out_scale, &vals, &n, &max_n);
        if (rc) return rc;
        if (!valid_bucket(bucket)) return fail(SPARCML_EINVAL, "bucket must be a power of two in [4, 8192]");
        const size_t need = quant_buckets_workspace(P);
        if (!ws || ws_bytes < need) return fail(SPARCML_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
        hipError_t e = quant_buckets_run(P, vals.data(), n.data(), bits, (uint32_t)bucket, seed, out_q,
                                         out_scale, out_deq, ws, (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "quantize_bucketed");
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

int sparcml_sparse_reduce(int P, const sparcml_stream* streams, uint64_t N, double delta,
                          sparcml_stream* out, uint64_t* node_nnz, uint8_t* node_dense, void* ws,
                          size_t ws_bytes, void* stream)
{
    return reduce_impl(P, streams, N, 0, N, delta, out, node_nnz, node_dense, ws, ws_bytes, stream);
}

int sparcml_sparse_reduce_range(int P, const sparcml_stream* streams, uint64_t N, uint64_t lo,
                                uint64_t hi, double delta, sparcml_stream* out, uint64_t* node_nnz,
                                uint8_t* node_dense, void* ws, size_t ws_bytes, void* stream)
{
    if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
    if (!(lo < hi && hi <= N)) return fail(SPARCML_EINVAL, "need 0 <= lo < hi <= N");
    return reduce_impl(P, streams, N, lo, hi, delta, out, node_nnz, node_dense, ws, ws_bytes, stream);
}

int sparcml_concat(int P, const sparcml_stream* parts, const uint64_t* bounds, uint64_t N, double delta,
                   uint64_t bucket, sparcml_stream* out, void* ws, size_t ws_bytes, void* stream)
{
    try {
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
        if (!(delta > 0.0) || isnan(delta)) return fail(SPARCML_EINVAL, "delta must be > 0");
        if (!parts || !bounds || !out) return fail(SPARCML_EINVAL, "NULL argument");
        if (bounds[0] != 0 || bounds[P] != N) return fail(SPARCML_EINVAL, "bounds must run from 0 to N");
        if (bucket && !valid_bucket(bucket)) return fail(SPARCML_EINVAL, "bucket must be 0 or a power of two in [4, 8192]");
        const uint32_t qbits = parts[0].qbits;
        std::vector<ConcatPart> cp(P);
        uint64_t total = 0;
        bool any_dense = false;
        for (int p = 0; p < P; ++p) {
            const sparcml_stream& a = parts[p];
            if (bounds[p + 1] < bounds[p]) return fail(SPARCML_EINVAL, "bounds must not decrease (part %d)", p);
            const uint64_t len = bounds[p + 1] - bounds[p];
            if (a.qbits != qbits) return fail(SPARCML_EINVAL, "part %d: all parts must share qbits", p);
            if (qbits && !valid_bits(qbits)) return fail(SPARCML_EINVAL, "part %d: qbits must be 0, 2, 4 or 8", p);
            if (a.is_dense ? a.nnz != len : a.nnz > len)
                return fail(SPARCML_EINVAL, "part %d: %s", p, a.is_dense ? "a dense part holds its range's values"
                                                                          : "more entries than its range has indices");
            if (a.nnz) {
                if (!a.is_dense && !a.idx) return fail(SPARCML_EINVAL, "part %d: idx is NULL", p);
                if (qbits ? (!a.qval || !a.qscale) : !a.val) return fail(SPARCML_EINVAL, "part %d: values are NULL", p);
            }
            cp[p] = ConcatPart{a.idx, a.val, a.qval, a.qscale, a.nnz, bounds[p], len, a.is_dense ? 1 : 0};
            any_dense = any_dense || a.is_dense;
            total += a.nnz;
        }
        const bool dense = any_dense || total > threshold(N, delta);
        if (!out->val) return fail(SPARCML_EINVAL, "out->val is NULL");
        if (out->qbits) return fail(SPARCML_EINVAL, "out->qbits must be 0");
        if (!dense) {
            if (total && !out->idx) return fail(SPARCML_EINVAL, "out->idx is NULL");
            if (out->nnz < total)
                return fail(SPARCML_ECAPACITY, "out capacity %llu < %llu entries", (unsigned long long)out->nnz,
                            (unsigned long long)total);
        }
        const size_t need = concat_workspace(P);
        if (!ws || ws_bytes < need) return fail(SPARCML_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
        hipError_t e = concat_run(P, cp.data(), qbits, bucket, dense ? 1 : 0, out->idx, out->val, ws,
                                  (hipStream_t)stream);
        if (e != hipSuccess) return hip_fail(e, "concat");
        out->nnz = dense ? N : total;
        out->is_dense = dense ? 1 : 0;
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

int sparcml_sparse_reduce_async(int P, const sparcml_stream* streams, uint64_t N, uint64_t lo, uint64_t hi,
                                double delta, const sparcml_stream* out, uint64_t* node_nnz,
                                uint8_t* node_dense, sparcml_result* result, void* ws, size_t ws_bytes,
                                void* stream)
{
    if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
    if (!(lo < hi && hi <= N)) return fail(SPARCML_EINVAL, "need 0 <= lo < hi <= N");
    if (!result) return fail(SPARCML_EINVAL, "result is NULL");
    if (!out) return fail(SPARCML_EINVAL, "out is NULL");
    sparcml_stream o = *out;  // capacity and pointers only; never written
    return reduce_impl(P, streams, N, lo, hi, delta, &o, node_nnz, node_dense, ws, ws_bytes, stream, result);
}

int sparcml_sparse_reduce_async_noalloc(int P, const sparcml_stream* streams, uint64_t N, uint64_t lo,
                                        uint64_t hi, double delta, const sparcml_stream* out,
                                        uint64_t* node_nnz, uint8_t* node_dense, sparcml_result* result,
                                        void* stream)
{
    if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
    if (!(lo < hi && hi <= N)) return fail(SPARCML_EINVAL, "need 0 <= lo < hi <= N");
    if (!result) return fail(SPARCML_EINVAL, "result is NULL");
    if (!out) return fail(SPARCML_EINVAL, "out is NULL");
    sparcml_stream o = *out;  // capacity and pointers only; never written
    return reduce_impl(P, streams, N, lo, hi, delta, &o, node_nnz, node_dense, nullptr, 0, stream, result,
                       /*use_scratch=*/true);
}

int sparcml_validate_streams(int P, const sparcml_stream* streams, uint64_t lo, uint64_t hi, void* ws,
                             size_t ws_bytes, void* stream)
{
    try {
        if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
        if (!streams) return fail(SPARCML_EINVAL, "streams is NULL");
        if (!(lo < hi && hi <= (1ull << 32))) return fail(SPARCML_EINVAL, "need lo < hi <= 2^32");
        std::vector<const uint32_t*> idx(P);
        std::vector<uint64_t> nnz(P);
        for (int r = 0; r < P; ++r) {
            if (streams[r].is_dense) return fail(SPARCML_EINVAL, "stream %d: a dense stream has no indices", r);
            if (streams[r].nnz && !streams[r].idx) return fail(SPARCML_EINVAL, "stream %d: idx is NULL", r);
            if (streams[r].nnz >= (1ull << 32)) return fail(SPARCML_EINVAL, "stream %d: nnz >= 2^32", r);
            idx[r] = streams[r].idx;
            nnz[r] = streams[r].nnz;
        }
        const size_t need = validate_workspace(P);
        if (!ws || ws_bytes < need) return fail(SPARCML_EWORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
        int bad_stream = -1;
        uint64_t bad_pos = 0;
        hipError_t e = validate_run(P, idx.data(), nnz.data(), lo, hi, ws, (hipStream_t)stream, &bad_stream, &bad_pos);
        if (e != hipSuccess) return hip_fail(e, "validate");
        if (bad_stream >= 0)
            return fail(SPARCML_EUNSORTED,
                        "stream %d, position %llu: index not strictly above its predecessor or outside [%llu, %llu)",
                        bad_stream, (unsigned long long)bad_pos, (unsigned long long)lo, (unsigned long long)hi);
        return SPARCML_OK;
    } catch (const std::exception& ex) {
        return fail(SPARCML_EHIP, "host exception: %s", ex.what());
    }
}

int sparcml_split_bounds(int P, uint64_t N, uint64_t* bounds)
{
    if (P < 1 || P > 65535) return fail(SPARCML_EINVAL, "P must be in [1, 65535]");
    if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
    if (!bounds) return fail(SPARCML_EINVAL, "bounds is NULL");
    const uint64_t each = N / (uint64_t)P;  // App. A: floor(N/P) per node, the rest to the last
    for (int s = 0; s < P; ++s) bounds[s] = (uint64_t)s * each;
    bounds[P] = N;
    return SPARCML_OK;
}

int sparcml_densify(const sparcml_stream* in, uint64_t N, float* dense, void* stream)
{
    if (!in || !dense) return fail(SPARCML_EINVAL, "NULL argument");
    if (!valid_n(N)) return fail(SPARCML_EINVAL, "N must be in [1, 2^32)");
    if (in->qbits && !valid_bits(in->qbits)) return fail(SPARCML_EINVAL, "qbits must be 0, 2, 4 or 8");
    if (in->qbits && !in->qscale) return fail(SPARCML_EINVAL, "qscale is NULL");
    const bool has_vals = in->qbits ? in->qval != nullptr : in->val != nullptr;
    if (in->is_dense) {
        if (!has_vals) return fail(SPARCML_EINVAL, "values are NULL");
    } else {
        if (in->nnz > N) return fail(SPARCML_EINVAL, "nnz > N");
        if (in->nnz && (!in->idx || !has_vals)) return fail(SPARCML_EINVAL, "NULL stream arrays");
    }
    hipError_t e = densify_run(in->idx, in->val, in->qval, in->qscale, in->qbits, in->nnz, N,
                               in->is_dense ? 1 : 0, dense, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "densify");
    return SPARCML_OK;
}

}  // extern "C"
