// Small-data reduction in one launch (§5.3.1: for small messages recursive
// doubling is the latency-optimal schedule; §5.1 "Efficient Summation").
//
// When the P' tree slots hold at most thr entries together, no tree node can
// switch to dense (a sparse node's size is at most the sum of its leaves'
// sizes), so the whole reduction is a tree of sorted-list merges.  When the
// entries also fit in one workgroup's LDS, that workgroup runs the tree
// itself, literally in recursive-doubling order:
//
//  * the slot streams are loaded side by side into LDS (QSGD codes
//    dequantized on the way in), slot s at run start S[s];
//  * level t merges, for every node g at once, its two children -- the runs
//    at S[g * 2^t] and S[g * 2^t + 2^(t-1)] -- into the node's run at
//    S[g * 2^t]: an index present in both children gets left + right;
//  * the merge is cut into units of kMV merged positions (merge path: the
//    split of a unit's first position between the two children is found by
//    binary search); a unit's outputs stay in registers until every unit has
//    read its inputs, so the level is merged in place;
//  * per-unit output counts, scanned across the workgroup, give the output
//    positions; per-node counts are the nodes' union sizes (what the switch
//    rule reports per node).
//
// The root run is then copied out.  One launch, no counters to clear, no
// second pass; the slot table travels in the kernel arguments.
//
// A level costs about 4.5 us of dependent LDS round trips and barriers even
// when it holds few entries, while the tile pipeline costs about 23-30 us of
// launches for any small input (measured on MI355X, P = 4..32, 256..16384
// entries).  So this path is taken where it is the faster one: at most 8
// slots (three levels), with at most 16384 / 8192 / 1024 entries for one,
// two, three levels.
#include "internal.h"
#include "qsgd_device.h"

namespace sparcml {
namespace {

constexpr int kMNT = 1024;          // threads
constexpr uint32_t kMCap = 16384;   // entries held in LDS (idx + value: 128 KB)
constexpr int kMV = 9;              // merged positions per unit (odd: adjacent units fall in different LDS banks)
constexpr int kMUPT = 2;            // units per thread (kMCap / kMV units, one more per node at most)
constexpr int kMKL = kMCap / kMNT;  // entries loaded per thread
constexpr int kMKB = 8;             // of which loaded at once
constexpr uint32_t kMSlots = 8;     // slots (the kernel-argument table)
static_assert(kMCap / kMV + 1 + kMSlots / 2 <= (uint32_t)kMNT * kMUPT, "too few units for the nodes of a level");

struct MTable {
    StreamDesc d[kMSlots];
};

struct MArgs {
    uint32_t PT, L, qbits, nfold;
    uint32_t* out_idx;
    float* out_val;
    uint64_t* node_nnz;
    uint8_t* node_dense;
    ReduceResult* hdr;
    ReduceResult* result;
};

// Exclusive scan of v over the workgroup; *total = the sum over all threads.
__device__ __forceinline__ uint32_t wg_excl_scan(uint32_t v, uint32_t* s_w, uint32_t* total)
{
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    const uint32_t incl = wave_scan(v);
    __syncthreads();  // s_w free from any earlier use
    if (lane == 63u) s_w[wv] = incl;
    __syncthreads();
    uint32_t before = 0, t = 0;
#pragma unroll
    for (uint32_t w = 0; w < (uint32_t)kMNT / 64u; ++w) {
        const uint32_t x = s_w[w];
        before += w < wv ? x : 0u;
        t += x;
    }
    *total = t;
    return incl - v + before;
}

// Largest i in [0, n) with a[i] <= x (a ascending, a[0] <= x, n <= 2^LOG
// + 1): LOG + 1 fixed steps without branches, so that a thread's
// independent searches overlap.
template <int LOG>
__device__ __forceinline__ uint32_t last_at_most(const uint32_t* a, uint32_t n, uint32_t x)
{
    uint32_t pos = 0;
#pragma unroll
    for (int k = LOG; k >= 0; --k) {
        const uint32_t c = pos + (1u << k);
        pos = c < n && a[c < n ? c : 0u] <= x ? c : pos;
    }
    return pos;
}

// Past every index: indices lie below 2^32 - 1 (N < 2^32, and a range ends
// at or below N).
constexpr uint32_t kNone = 0xFFFFFFFFu;

template <bool QUANT>
__global__ void __launch_bounds__(kMNT) k_merge_small(MTable kt, MArgs a)
{
    __shared__ uint32_t s_idx[kMCap];
    __shared__ float s_val[kMCap];
    __shared__ uint32_t s_start[kMSlots + 1];  // run start of each slot; s_start[PT] = all entries
    __shared__ uint32_t s_len[kMSlots];    // current run length, kept at the node's first slot
    __shared__ uint32_t s_ub[kMSlots / 2 + 1];  // first unit of each node of a level; s_ub[nodes] = units
    __shared__ uint32_t s_nb[kMSlots / 2];  // scan value at each node's first unit
    __shared__ uint32_t s_lc[kMSlots / 2];  // outputs of each node of the level (its union size)
    __shared__ uint32_t s_cnt[kMSlots - 1];  // union size of every node, level order
    __shared__ const uint32_t* s_pi[kMSlots];
    __shared__ const void* s_pv[kMSlots];  // values, or QSGD codes
    __shared__ float s_unit[QUANT ? kMSlots : 1];
    __shared__ uint32_t s_w[kMNT / 64];
    const uint32_t tid = threadIdx.x, PT = a.PT;

    // the slot table and each slot's run start
    uint32_t n = 0;
    if (tid < PT) {
        const StreamDesc d = kt.d[tid];
        n = (uint32_t)d.nnz;
        s_pi[tid] = d.idx;
        s_pv[tid] = QUANT ? static_cast<const void*>(d.qval) : static_cast<const void*>(d.val);
        if (QUANT) s_unit[tid] = n ? level_unit(*d.qscale, a.qbits) : 0.0f;
        s_len[tid] = n;
    }
    uint32_t total;
    const uint32_t st = wg_excl_scan(n, s_w, &total);
    if (tid <= PT) s_start[tid] = st;  // tid == PT: the total
    __syncthreads();

    // load: entry e of the concatenation is entry e - S[s] of slot s; in
    // batches of kMKB entries per thread whose loads are all issued before
    // any is stored
    const uint32_t wfirst = (uint32_t)__builtin_amdgcn_readfirstlane((int)(tid & ~63u));  // the wave's lane 0
    for (int b = 0; b < kMKL; b += kMKB) {
        if (wfirst + (uint32_t)b * kMNT >= total) break;  // the wave has no entry left
        uint32_t slot[kMKB], pos[kMKB];
#pragma unroll
        for (int k = 0; k < kMKB; ++k) {
            const uint32_t e = tid + (uint32_t)(b + k) * kMNT;
            slot[k] = e < total ? last_at_most<3>(s_start, PT, e) : 0u;
            pos[k] = e - s_start[slot[k]];
        }
        uint32_t gi[kMKB];
        float gv[kMKB];
#pragma unroll
        for (int k = 0; k < kMKB; ++k) {
            const uint32_t e = tid + (uint32_t)(b + k) * kMNT;
            if (e < total) {
                const uint32_t s = slot[k];
                gi[k] = s_pi[s][pos[k]];
                if (QUANT) {
                    const uint32_t code = load_code(static_cast<const uint8_t*>(s_pv[s]), pos[k], a.qbits);
                    gv[k] = dequant(code, a.qbits, s_unit[s]);
                } else {
                    gv[k] = static_cast<const float*>(s_pv[s])[pos[k]];
                }
            }
        }
#pragma unroll
        for (int k = 0; k < kMKB; ++k) {
            const uint32_t e = tid + (uint32_t)(b + k) * kMNT;
            if (e < total) {
                s_idx[e] = gi[k];
                s_val[e] = gv[k];
            }
        }
    }
    __syncthreads();

    // the tree, level by level
    uint32_t node_base = 0;  // level-order number of the level's first node
    for (uint32_t t = 1; t <= a.L; ++t) {
        const uint32_t nodes = PT >> t, half = 1u << (t - 1u);
        uint32_t units = 0;
        if (tid < nodes) {
            const uint32_t f = tid << t;
            units = (s_len[f] + s_len[f + half] + (uint32_t)kMV - 1u) / (uint32_t)kMV;
            s_lc[tid] = 0u;
        }
        uint32_t U;
        const uint32_t ub = wg_excl_scan(units, s_w, &U);
        if (tid <= nodes) s_ub[tid] = ub;
        __syncthreads();

        // merge this thread's units into registers, their dependent LDS
        // reads interleaved; unit q * kMNT + tid, so that the lanes of a
        // wave work on adjacent units, kMV (odd) entries apart: no LDS bank
        // conflicts
        uint32_t key[kMUPT][kMV];
        float val[kMUPT][kMV];
        uint32_t valid[kMUPT], cnt[kMUPT], node[kMUPT], sa[kMUPT];
        uint32_t rem[kMUPT], ia[kMUPT], jb[kMUPT], na[kMUPT], nb[kMUPT], sb[kMUPT], d0[kMUPT], lo[kMUPT],
            hi[kMUPT];
        bool wq[kMUPT];  // the wave has a unit q (uniform): the others skip its work
#pragma unroll
        for (int q = 0; q < kMUPT; ++q) {
            const uint32_t u = (uint32_t)q * kMNT + tid;
            wq[q] = (uint32_t)q * kMNT + wfirst < U;
            valid[q] = cnt[q] = node[q] = sa[q] = 0u;
            rem[q] = na[q] = nb[q] = sb[q] = d0[q] = lo[q] = hi[q] = ia[q] = jb[q] = 0u;
            if (wq[q] && u < U) {
                const uint32_t g = last_at_most<2>(s_ub, nodes, u);  // node of the unit (units > 0)
                const uint32_t f = g << t;
                node[q] = g;
                sa[q] = s_start[f];
                na[q] = s_len[f];
                sb[q] = s_start[f + half];
                nb[q] = s_len[f + half];
                d0[q] = (u - s_ub[g]) * (uint32_t)kMV;
                rem[q] = min((uint32_t)kMV, na[q] + nb[q] - d0[q]);
                lo[q] = d0[q] > nb[q] ? d0[q] - nb[q] : 0u;
                hi[q] = min(d0[q], na[q]);
            }
        }
        // merge path: ia entries of the left child and d0 - ia of the right
        // one come before position d0 (left first on equal keys): the
        // largest c in [lo, hi] whose left entry c - 1 is at most the right
        // entry d0 - c, found in fixed steps
#pragma unroll
        for (int q = 0; q < kMUPT; ++q) ia[q] = lo[q];
        const int top = 31 - __clz(total | 1u);  // hi - lo <= total < 2^(top + 1)
        for (int k = top; k >= 0; --k) {
#pragma unroll
            for (int q = 0; q < kMUPT; ++q) {
                if (!wq[q]) continue;
                const uint32_t c = ia[q] + (1u << k);
                const bool in = c <= hi[q];
                const uint32_t x = s_idx[in ? sa[q] + c - 1u : 0u], y = s_idx[in ? sb[q] + d0[q] - c : 0u];
                ia[q] = in && x <= y ? c : ia[q];
            }
        }
        uint32_t ka[kMUPT], kb[kMUPT];
        float va[kMUPT], vb[kMUPT];
        bool skip[kMUPT];
#pragma unroll
        for (int q = 0; q < kMUPT; ++q) {
            ka[q] = kb[q] = kNone;
            va[q] = vb[q] = 0.0f;
            skip[q] = false;
            if (!wq[q]) continue;
            jb[q] = d0[q] - ia[q];
            const bool ina = ia[q] < na[q], inb = jb[q] < nb[q];
            ka[q] = ina ? s_idx[sa[q] + ia[q]] : kNone;
            va[q] = ina ? s_val[sa[q] + ia[q]] : 0.0f;
            kb[q] = inb ? s_idx[sb[q] + jb[q]] : kNone;
            vb[q] = inb ? s_val[sb[q] + jb[q]] : 0.0f;
            // a right entry equal to the left entry before the split was
            // summed by the unit that took that left entry
            skip[q] = inb && ia[q] > 0u && rem[q] && s_idx[sa[q] + ia[q] - 1u] == kb[q];
        }
        // one merged position per step, without branches: take the left
        // head (summed with an equal right head), or the right head, or skip
        // the right twin of a pair summed one step before; then reload the
        // side that moved
#pragma unroll
        for (int s = 0; s < kMV; ++s) {
#pragma unroll
            for (int q = 0; q < kMUPT; ++q) {
                key[q][s] = 0u;
                val[q][s] = 0.0f;
                if (!wq[q]) continue;
                const bool act = (uint32_t)s < rem[q];
                const bool tA = act && !skip[q] && ka[q] <= kb[q];
                const bool tB = act && !tA;
                const bool pair = tA && ka[q] == kb[q];
                const bool emit = act && !skip[q];
                key[q][s] = tA ? ka[q] : kb[q];
                val[q][s] = pair ? va[q] + vb[q] : (tA ? va[q] : vb[q]);  // left + right
                valid[q] |= emit ? 1u << s : 0u;
                cnt[q] += emit ? 1u : 0u;
                skip[q] = act ? pair : skip[q];
                ia[q] += tA ? 1u : 0u;
                jb[q] += tB ? 1u : 0u;
                const bool in = tA ? ia[q] < na[q] : jb[q] < nb[q];
                const uint32_t at = in ? (tA ? sa[q] + ia[q] : sb[q] + jb[q]) : 0u;
                const uint32_t nk = in ? s_idx[at] : kNone;
                const float nv = in ? s_val[at] : 0.0f;
                ka[q] = tA ? nk : ka[q];
                va[q] = tA ? nv : va[q];
                kb[q] = tB ? nk : kb[q];
                vb[q] = tB ? nv : vb[q];
            }
        }

        // output positions: units in order (all q = 0 units, then q = 1, ...),
        // by a scan per q, relative to the node's first unit
        uint32_t xq[kMUPT], base = 0;
#pragma unroll
        for (int q = 0; q < kMUPT; ++q) {
            uint32_t tot;
            xq[q] = base + wg_excl_scan(cnt[q], s_w, &tot);  // past the first: every read of the level done
            base += tot;
        }
#pragma unroll
        for (int q = 0; q < kMUPT; ++q) {
            const uint32_t u = (uint32_t)q * kMNT + tid;
            if (u < U) {
                if (u == s_ub[node[q]]) s_nb[node[q]] = xq[q];
                if (cnt[q]) atomicAdd(&s_lc[node[q]], cnt[q]);
            }
        }
        __syncthreads();
#pragma unroll
        for (int q = 0; q < kMUPT; ++q) {
            if (!valid[q]) continue;
            uint32_t p = sa[q] + xq[q] - s_nb[node[q]];  // the node's run starts at its left child's
#pragma unroll
            for (int s = 0; s < kMV; ++s) {
                if (valid[q] & (1u << s)) {
                    s_idx[p] = key[q][s];
                    s_val[p] = val[q][s];
                    ++p;
                }
            }
        }
        __syncthreads();
        if (tid < nodes) {
            s_len[tid << t] = s_lc[tid];
            s_cnt[node_base + tid] = s_lc[tid];
        }
        node_base += nodes;
        __syncthreads();
    }

    // the root run, the per-node sizes (all sparse) and the result header
    const uint32_t root = s_len[0];
    for (uint32_t e = tid; e < root; e += kMNT) {
        a.out_idx[e] = s_idx[e];
        a.out_val[e] = s_val[e];
    }
    if (tid + 1u < PT && (tid >= PT / 2u || tid < a.nfold)) {
        const uint32_t o = tid < PT / 2u ? tid : tid - PT / 2u + a.nfold;
        if (a.node_nnz) a.node_nnz[o] = s_cnt[tid];
        if (a.node_dense) a.node_dense[o] = 0u;
    }
    if (tid == 0) {
        const ReduceResult r{root, 0u, 0u};
        *a.hdr = r;
        if (a.result) *a.result = r;
    }
}

}  // namespace

bool merge_small_fits(uint32_t PT, uint64_t sum_nnz, uint64_t thr)
{
    if (PT < 2 || PT > kMSlots || sum_nnz > thr) return false;  // every node sparse
    const uint64_t most = PT == 2 ? kMCap : (PT == 4 ? 8192u : 1024u);
    return sum_nnz <= most;
}

hipError_t merge_small_run(uint32_t PT, uint32_t L, uint32_t qbits, uint32_t nfold, const StreamDesc* host_tab,
                           uint32_t* out_idx, float* out_val, uint64_t* node_nnz, uint8_t* node_dense,
                           ReduceResult* hdr, ReduceResult* result, hipStream_t s)
{
    if (PT > kMSlots) return hipErrorInvalidValue;
    MTable kt{};
    MArgs a{};
    a.PT = PT;
    a.L = L;
    a.qbits = qbits;
    a.nfold = nfold;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.node_nnz = node_nnz;
    a.node_dense = node_dense;
    a.hdr = hdr;
    a.result = result;
    for (uint32_t r = 0; r < PT; ++r) kt.d[r] = host_tab[r];
    timer_begin(kTReduceMerge, s);
    if (qbits) hipLaunchKernelGGL(k_merge_small<true>, dim3(1), dim3(kMNT), 0, s, kt, a);
    else hipLaunchKernelGGL(k_merge_small<false>, dim3(1), dim3(kMNT), 0, s, kt, a);
    timer_end(kTReduceMerge, s);
    return hipGetLastError();
}

}  // namespace sparcml
