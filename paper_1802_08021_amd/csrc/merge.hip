// Sparse reduce as a tree of sorted-list merges, for inputs whose tree nodes
// all stay sparse (§5.1 "Efficient Summation"; §5.3.1 recursive doubling).
//
// When the P' tree slots hold at most thr entries together, no node can
// switch to dense (a sparse node's size is at most the sum of its leaves'
// sizes), and the reduction is the paper's merge tree itself.  A workgroup
// runs it for the entries of an index range, literally in recursive-doubling
// order:
//
//  * the slot streams' entries in the range are loaded side by side into LDS
//    (QSGD codes dequantized on the way in), slot s at run start S[s];
//  * level t merges, for every node g at once, its two children (the slots'
//    runs at level 1, else the runs of level t-1's nodes 2g and 2g+1) into
//    the node's run: an index present in both children gets left + right;
//  * the merge is cut into units of MV merged positions (merge path: the
//    split of a unit's first position between the two children is found by
//    binary search); a unit's outputs stay in registers until every unit has
//    read its inputs, so the level is merged in place;
//  * per-unit output counts, scanned across the workgroup, give the output
//    positions: a level's node runs lie one after another in node order;
//    per-node counts are the nodes' union sizes (what the switch rule
//    reports per node).
//
// Ranges of few entries (at most kSortPer a thread) take the same tree in
// one pass instead (sort_merge): every entry's place in the root's order
// from binary searches, then the sums of each index in the tree's order.
//
// Two kernels use it.  k_merge_small: one workgroup takes the whole range
// (one launch, the slot table in the kernel arguments).  A level costs about
// 4.5 us of dependent LDS round trips and barriers even when it holds few
// entries, while the tile pipeline costs about 23-30 us of launches for any
// small input (measured on MI355X, P = 4..32, 256..16384 entries), so it is
// taken for at most 8 slots with at most 16384 / 8192 / 1024 entries for
// one, two, three levels.  k_merge_seg: the range is cut into segments of
// equal width (about kSegEntries expected entries each, at least kSegMin
// segments), one small workgroup per segment (several per CU), all at
// once; a segment's output offset comes
// from a decoupled look-back over the segments' union sizes (a workgroup
// waits only on segments whose ticket is lower than its own, which have
// started and publish their sizes before they wait on anyone), and the last
// workgroup to finish reports the node sizes.  A segment with more entries
// than the LDS holds is merged piece by piece (its index range halved until
// each piece fits), once to count and once more to write.
#include "internal.h"
#include "qsgd_device.h"

#include <algorithm>

namespace sparcml {
namespace {

constexpr uint32_t kMSlots = 64;     // slots the LDS tables hold
constexpr uint32_t kSmallSlots = 8;  // slots of the one-workgroup path (its argument table)
constexpr uint32_t kMaxLevels = 6;   // levels of a kMSlots-slot tree

// Threads, LDS entries, units per thread and merged positions per unit
// (odd: the units of adjacent lanes start in different LDS banks) of a
// merge workgroup.  A thread's units merge side by side, so their dependent
// reads overlap: short units shorten a level when few threads have work.
template <int NT_, uint32_t CAP_, int UPT_, int MV_>
struct MCfg {
    static constexpr int NT = NT_;
    static constexpr uint32_t CAP = CAP_;
    static constexpr int UPT = UPT_;
    static constexpr int MV = MV_;
    static constexpr int KL = (int)(CAP / NT);  // entries loaded per thread
    static constexpr int KB = KL < 8 ? KL : 8;  // of which loaded at once
    static_assert(CAP / MV + 1 + kMSlots / 2 <= (uint32_t)NT * UPT, "too few units for the nodes of a level");
    static_assert(MV % 2 == 1 && MV <= 32, "odd unit, one mask bit per position");
};
using SmallCfg = MCfg<1024, 16384, 2, 9>;  // the whole input in one workgroup (128 KB of entries)
// one segment per workgroup (32 KB), several workgroups per CU: units of 9
// positions, or of 3 for segments whose units fit one a thread
using SegCfg = MCfg<512, 4096, 1, 9>;
using SegShortCfg = MCfg<512, 4096, 3, 3>;

template <class C>
struct MLds {
    uint32_t idx[C::CAP];
    float val[C::CAP];
    uint32_t start[kMSlots + 1];   // run start of each slot; start[PT] = all entries
    uint32_t len[kMSlots];         // run length of each slot
    uint32_t rs[2][kMSlots / 2];   // run start of each node of a level, by level parity
    uint32_t lc[2][kMSlots / 2];   // run length of each node of a level (its union size), by level parity
    uint32_t cnt[kMSlots - 1];     // union size of every node, level order
    const uint32_t* pi[kMSlots];   // slot index streams
    const void* pv[kMSlots];       // slot values, or QSGD codes
    uint32_t first[kMSlots];       // stream position of the slot's first entry in the range
    float unit[kMSlots];           // QSGD level unit of the slot
    uint8_t rk[C::CAP];            // one-pass order: the slot of each entry
    uint32_t lmax;                 // one-pass order: the longest slot run
    uint32_t ecnt[(kMaxLevels + 1) * kMSlots];  // one-pass order: entries by level span and slot
    uint32_t w[C::NT / 64];
    uint2 w2[C::NT / 64];
};

// Past every index: indices lie below 2^32 - 1 (N < 2^32, and a range ends
// at or below N).
constexpr uint32_t kNone = 0xFFFFFFFFu;

// Stream pointers kept in LDS are generic; read through them as global
// memory, so that the reads are not FLAT accesses (which also count against
// the LDS wait counter).
typedef const uint32_t __attribute__((address_space(1)))* g_u32p;
typedef const float __attribute__((address_space(1)))* g_f32p;
typedef const uint8_t __attribute__((address_space(1)))* g_u8p;
__device__ __forceinline__ g_u32p as_global(const uint32_t* p) { return (g_u32p)p; }
__device__ __forceinline__ g_f32p as_global(const float* p) { return (g_f32p)p; }
__device__ __forceinline__ g_u8p as_global(const uint8_t* p) { return (g_u8p)p; }

// Exclusive scan of v over the workgroup; *total = the sum over all threads.
// FREE: the caller knows s_w free (a barrier since its last reads).
template <int NT, bool FREE = false>
__device__ __forceinline__ uint32_t wg_excl_scan(uint32_t v, uint32_t* s_w, uint32_t* total)
{
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    const uint32_t incl = wave_scan(v);
    if (!FREE) __syncthreads();  // s_w free from any earlier use
    if (lane == 63u) s_w[wv] = incl;
    __syncthreads();
    uint32_t before = 0, t = 0;
#pragma unroll
    for (uint32_t w = 0; w < (uint32_t)NT / 64u; ++w) {
        const uint32_t x = s_w[w];
        before += w < wv ? x : 0u;
        t += x;
    }
    *total = t;
    return incl - v + before;
}

// Exclusive scans of a and b over the workgroup (the barriers of one);
// *ta, *tb = the sums over all threads.
template <int NT, bool FREE = false>
__device__ __forceinline__ uint2 wg_excl_scan2(uint32_t a, uint32_t b, uint2* s_w, uint32_t* ta, uint32_t* tb)
{
    const uint32_t lane = threadIdx.x & 63u, wv = threadIdx.x >> 6;
    const uint32_t ia = wave_scan(a), ib = wave_scan(b);
    if (!FREE) __syncthreads();  // s_w free from any earlier use
    if (lane == 63u) s_w[wv] = make_uint2(ia, ib);
    __syncthreads();
    uint32_t ba = 0, bb = 0, xa = 0, xb = 0;
#pragma unroll
    for (uint32_t w = 0; w < (uint32_t)NT / 64u; ++w) {
        const uint2 x = s_w[w];
        ba += w < wv ? x.x : 0u;
        bb += w < wv ? x.y : 0u;
        xa += x.x;
        xb += x.y;
    }
    *ta = xa;
    *tb = xb;
    return make_uint2(ia - a + ba, ib - b + bb);
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

// Run starts from this thread's slot size n (threads >= PT pass 0); returns
// the number of entries.
template <class C>
__device__ __forceinline__ uint32_t slot_starts(MLds<C>& m, uint32_t PT, uint32_t n)
{
    uint32_t total;
    const uint32_t st = wg_excl_scan<C::NT>(n, m.w, &total);
    if (threadIdx.x <= PT) m.start[threadIdx.x] = st;  // thread PT: the total
    if (threadIdx.x < PT) m.len[threadIdx.x] = n;
    __syncthreads();
    return total;
}

// Entry e of the concatenation is entry e - S[s] of slot s, at stream
// position first[s] + e - S[s]; in batches of KB entries per thread whose
// loads are all issued before any is stored.
template <class C, bool QUANT>
__device__ __forceinline__ void load_runs(MLds<C>& m, uint32_t PT, uint32_t total, uint32_t qbits)
{
    const uint32_t tid = threadIdx.x;
    const uint32_t wfirst = (uint32_t)__builtin_amdgcn_readfirstlane((int)(tid & ~63u));  // the wave's lane 0
    for (int b = 0; b < C::KL; b += C::KB) {
        if (wfirst + (uint32_t)b * C::NT >= total) break;  // the wave has no entry left
        uint32_t slot[C::KB], pos[C::KB];
#pragma unroll
        for (int k = 0; k < C::KB; ++k) {
            const uint32_t e = tid + (uint32_t)(b + k) * C::NT;
            slot[k] = e < total ? last_at_most<6>(m.start, PT, e) : 0u;
            pos[k] = m.first[slot[k]] + e - m.start[slot[k]];
        }
        uint32_t gi[C::KB];
        float gv[C::KB];
#pragma unroll
        for (int k = 0; k < C::KB; ++k) {
            const uint32_t e = tid + (uint32_t)(b + k) * C::NT;
            if (e < total) {
                const uint32_t s = slot[k];
                gi[k] = as_global(m.pi[s])[pos[k]];
                if (QUANT) {
                    const uint32_t code = load_code(as_global(static_cast<const uint8_t*>(m.pv[s])), pos[k], qbits);
                    gv[k] = dequant(code, qbits, m.unit[s]);
                } else {
                    gv[k] = as_global(static_cast<const float*>(m.pv[s]))[pos[k]];
                }
            }
        }
#pragma unroll
        for (int k = 0; k < C::KB; ++k) {
            const uint32_t e = tid + (uint32_t)(b + k) * C::NT;
            if (e < total) {
                m.idx[e] = gi[k];
                m.val[e] = gv[k];
            }
        }
    }
    __syncthreads();
}

// The tree over the loaded runs, level by level; returns the root's length
// (its run starts at 0) and leaves every node's union size in m.cnt.  A
// level's node runs are written one after another, in node order, at their
// scan positions; a level has two barriers: the scan's, past which every
// read of the level is done, and the last, past which its runs are written.
template <class C>
__device__ __forceinline__ uint32_t merge_levels(MLds<C>& m, uint32_t PT, uint32_t L)
{
    constexpr int NT = C::NT, UPT = C::UPT, MV = C::MV;
    const uint32_t tid = threadIdx.x, lane = tid & 63u;
    const uint32_t wfirst = (uint32_t)__builtin_amdgcn_readfirstlane((int)(tid & ~63u));
    if (L == 0u) return m.len[0];
    // the children of level t's nodes: the slots' runs at level 1, else the
    // runs of level t - 1's nodes
    auto cstart = [&](uint32_t t, uint32_t c) -> uint32_t { return t == 1u ? m.start[c] : m.rs[(t - 1u) & 1u][c]; };
    auto clen = [&](uint32_t t, uint32_t c) -> uint32_t { return t == 1u ? m.len[c] : m.lc[(t - 1u) & 1u][c]; };
    // level 1's node counters (ordered before its atomics by its scan)
    if (tid < kMSlots / 2u) m.lc[1][tid] = 0u;
    uint32_t node_base = 0;  // level-order number of the level's first node
    for (uint32_t t = 1; t <= L; ++t) {
        const uint32_t nodes = PT >> t;
        uint32_t* const lc = m.lc[t & 1u];
        // Every wave: the units of the level's nodes (lane g: node g's, for
        // its children's entries), their first units by a wave scan, and all.
        uint32_t ug = 0;
        if (lane < nodes) ug = (clen(t, 2u * lane) + clen(t, 2u * lane + 1u) + (uint32_t)MV - 1u) / (uint32_t)MV;
        const uint32_t ui = wave_scan(ug), ub_l = ui - ug;  // lane g: node g's first unit
        const uint32_t U = (uint32_t)__builtin_amdgcn_readlane((int)ui, (int)(nodes - 1u));
        // the previous level's node sizes, final past its last barrier
        if (t > 1u && tid < 2u * nodes) m.cnt[node_base - 2u * nodes + tid] = clen(t, tid);
        // node of each unit q * NT + tid: the nodes whose first unit is at or
        // below it, less one (gq), and that node's first unit (fq).  Outside
        // any branch on the unit: a readlane takes the lane's register whether
        // or not the lane is active, and a value used only in a branch may be
        // computed there, for the active lanes alone.
        uint32_t gq[UPT], fq[UPT];
#pragma unroll
        for (int q = 0; q < UPT; ++q) gq[q] = fq[q] = 0u;
        if (wfirst < U) {  // (uniform)
            for (uint32_t i = 1; i < nodes; ++i) {
                const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)ub_l, (int)i);
#pragma unroll
                for (int q = 0; q < UPT; ++q) {
                    const uint32_t u = (uint32_t)q * NT + tid;
                    gq[q] += b <= u ? 1u : 0u;
                    fq[q] = b <= u ? b : fq[q];
                }
            }
        }

        // merge this thread's units into registers, their dependent LDS
        // reads interleaved; unit q * NT + tid, so that while units are few
        // each lane of a wave takes one
        uint32_t key[UPT][MV];
        float val[UPT][MV];
        uint32_t valid[UPT], cnt[UPT], node[UPT], sa[UPT];
        bool first[UPT];  // the unit is its node's first
        uint32_t rem[UPT], ia[UPT], jb[UPT], na[UPT], nb[UPT], sb[UPT], d0[UPT], lo[UPT], hi[UPT];
        bool wq[UPT];  // the wave has a unit q (uniform): the others skip its work
#pragma unroll
        for (int q = 0; q < UPT; ++q) {
            const uint32_t u = (uint32_t)q * NT + tid;
            wq[q] = (uint32_t)q * NT + wfirst < U;
            valid[q] = cnt[q] = node[q] = sa[q] = 0u;
            first[q] = false;
            rem[q] = na[q] = nb[q] = sb[q] = d0[q] = lo[q] = hi[q] = ia[q] = jb[q] = 0u;
            if (wq[q] && u < U) {
                const uint32_t g = gq[q], fu = fq[q];
                node[q] = g;
                first[q] = u == fu;
                sa[q] = cstart(t, 2u * g);
                na[q] = clen(t, 2u * g);
                sb[q] = cstart(t, 2u * g + 1u);
                nb[q] = clen(t, 2u * g + 1u);
                d0[q] = (u - fu) * (uint32_t)MV;
                rem[q] = min((uint32_t)MV, na[q] + nb[q] - d0[q]);
                lo[q] = d0[q] > nb[q] ? d0[q] - nb[q] : 0u;
                hi[q] = min(d0[q], na[q]);
            }
        }
        // merge path: ia entries of the left child and d0 - ia of the right
        // one come before position d0 (left first on equal keys): the
        // largest c in [lo, hi] whose left entry c - 1 is at most the right
        // entry d0 - c, found in fixed steps
        uint32_t span = 0;  // the widest search range of this thread's units
#pragma unroll
        for (int q = 0; q < UPT; ++q) {
            ia[q] = lo[q];
            span = max(span, hi[q] - lo[q]);
        }
        // (two bits a step: the predicate is monotone in c, so of the three
        // candidates ia + b, ia + 2b, ia + 3b the ones that hold are a prefix
        // and their count is the step's pair of bits; the six reads of a step
        // do not wait on one another)
        const int top = 31 - __clz(span | 1u);  // span < 2^(top + 1)
        auto holds = [&](int q, uint32_t c) -> uint32_t {
            const bool in = c <= hi[q];
            const uint32_t x = m.idx[in ? sa[q] + c - 1u : 0u], y = m.idx[in ? sb[q] + d0[q] - c : 0u];
            return in && x <= y ? 1u : 0u;
        };
        int k = top;
        for (; k >= 1; k -= 2) {
#pragma unroll
            for (int q = 0; q < UPT; ++q) {
                if (!wq[q]) continue;
                const uint32_t b = 1u << (k - 1);
                const uint32_t n = holds(q, ia[q] + b) + holds(q, ia[q] + 2u * b) + holds(q, ia[q] + 3u * b);
                ia[q] += n * b;
            }
        }
        if (k == 0) {
#pragma unroll
            for (int q = 0; q < UPT; ++q)
                if (wq[q]) ia[q] += holds(q, ia[q] + 1u);
        }
        // the heads of both children (ka, kb) and the entries after them
        // (ka1, kb1; kNone past the end)
        uint32_t ka[UPT], kb[UPT], ka1[UPT], kb1[UPT];
        float va[UPT], vb[UPT], va1[UPT], vb1[UPT];
        bool skip[UPT];
        auto entry = [&](uint32_t base, uint32_t i, uint32_t n, uint32_t& k, float& v) {
            const bool in = i < n;
            k = in ? m.idx[base + i] : kNone;
            v = in ? m.val[base + i] : 0.0f;
        };
#pragma unroll
        for (int q = 0; q < UPT; ++q) {
            ka[q] = kb[q] = ka1[q] = kb1[q] = kNone;
            va[q] = vb[q] = va1[q] = vb1[q] = 0.0f;
            skip[q] = false;
            if (!wq[q]) continue;
            jb[q] = d0[q] - ia[q];
            entry(sa[q], ia[q], na[q], ka[q], va[q]);
            entry(sb[q], jb[q], nb[q], kb[q], vb[q]);
            entry(sa[q], ia[q] + 1u, na[q], ka1[q], va1[q]);
            entry(sb[q], jb[q] + 1u, nb[q], kb1[q], vb1[q]);
            // a right entry equal to the left entry before the split was
            // summed by the unit that took that left entry
            skip[q] = jb[q] < nb[q] && ia[q] > 0u && rem[q] && m.idx[sa[q] + ia[q] - 1u] == kb[q];
        }
        // one merged position per step, without branches: take the left
        // head (summed with an equal right head), or the right head, or skip
        // the right twin of a pair summed one step before.  The side that
        // moved takes its next entry, read one step ahead; then the entries
        // after both heads are read for the next step, so that no step waits
        // on a read of its own.
#pragma unroll
        for (int s = 0; s < MV; ++s) {
#pragma unroll
            for (int q = 0; q < UPT; ++q) {
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
                ka[q] = tA ? ka1[q] : ka[q];
                va[q] = tA ? va1[q] : va[q];
                kb[q] = tB ? kb1[q] : kb[q];
                vb[q] = tB ? vb1[q] : vb[q];
                if (s + 1 < MV) {
                    entry(sa[q], ia[q] + 1u, na[q], ka1[q], va1[q]);
                    entry(sb[q], jb[q] + 1u, nb[q], kb1[q], vb1[q]);
                }
            }
        }

        // output positions: units in order (all q = 0 units, then q = 1, ...),
        // relative to the node's first unit: one scan of the unit counts
        // packed two to a word, 16 bits each (a level's count of every q is
        // at most NT * MV < 2^16), past whose first barrier every read of the
        // level is done
        static_assert(NT * MV < 65536 && UPT <= 4, "packed unit counts");
        uint32_t xq[UPT];
        {
            uint32_t p0 = 0, p1 = 0;
#pragma unroll
            for (int q = 0; q < UPT; ++q) {
                if (q < 2) p0 |= cnt[q] << (16 * q);
                else p1 |= cnt[q] << (16 * (q - 2));
            }
            // (the scan words are free: every read of them was before the
            // previous level's last barrier, or before the caller's)
            uint32_t t0 = 0, t1 = 0;
            uint2 e;
            if (UPT > 2) {
                e = wg_excl_scan2<NT, true>(p0, p1, m.w2, &t0, &t1);
            } else {
                e.x = wg_excl_scan<NT, true>(p0, m.w, &t0);
                e.y = 0u;
            }
            uint32_t base = 0;
#pragma unroll
            for (int q = 0; q < UPT; ++q) {
                const uint32_t ew = q < 2 ? e.x : e.y, tw = q < 2 ? t0 : t1, sh = 16u * (q & 1);
                xq[q] = base + ((ew >> sh) & 0xFFFFu);
                base += (tw >> sh) & 0xFFFFu;
            }
        }
        // node runs start where their first unit's outputs do; node sizes
        // add up; the next level's counters (the previous level's sizes,
        // read by now) are cleared
#pragma unroll
        for (int q = 0; q < UPT; ++q) {
            if ((uint32_t)q * NT + tid < U) {
                if (first[q]) m.rs[t & 1u][node[q]] = xq[q];
                if (cnt[q]) atomicAdd(&lc[node[q]], cnt[q]);
            }
        }
        if (t < L && tid < (nodes >> 1)) m.lc[(t + 1u) & 1u][tid] = 0u;
#pragma unroll
        for (int q = 0; q < UPT; ++q) {
            if (!valid[q]) continue;
            uint32_t p = xq[q];
#pragma unroll
            for (int s = 0; s < MV; ++s) {
                if (valid[q] & (1u << s)) {
                    m.idx[p] = key[q][s];
                    m.val[p] = val[q][s];
                    ++p;
                }
            }
        }
        node_base += nodes;
        __syncthreads();
    }
    // the root (its run starts at 0)
    const uint32_t root = m.lc[L & 1u][0];
    if (tid == 0) m.cnt[node_base - 1u] = root;
    __syncthreads();  // m.cnt whole
    return root;
}

// The same tree in one pass, for ranges of few entries (at most kSortPer
// a thread).  The root's entries come in the order of (index, slot), and
// the node sums at an index follow the tree over the slots present there:
//
//  * an entry's place in that order is its position in its own run plus,
//    for every other slot, the entries of that slot's run that precede it
//    (indices below its own, and equal ones of lower slots): fixed-step
//    binary searches, eight slots side by side, and G lanes per entry
//    (each taking every G-th slot; G up to 8 while entries are few, and at
//    most PT / 8 so that a lane keeps eight slots);
//  * the entries move to their places, with their slots, so an index's
//    entries are consecutive and in slot order;
//  * two neighbouring slots r' < r there first share a node at level h + 1,
//    h the highest bit in which they differ (the separator).  The sum is
//    taken with a stack: before a value is pushed, the pending sums whose
//    separator lies below its own are folded (left + right), which adds
//    exactly the pairs of children that both hold a value, in the tree's
//    order;
//  * an entry opens a group of its index at levels 1..h below the node it
//    shares with its predecessor (the next lower slot present), at every
//    level if it has none; counts of those spans per slot, summed over a
//    node's slots (one wave per level), give every node's union size.
// Returns the root's length (its run at 0) and leaves the node sizes in
// m.cnt, as merge_levels does.
constexpr uint32_t kSortPer = 2;

template <class C>
__device__ __forceinline__ bool sort_fits(uint32_t total)
{
    return total <= kSortPer * (uint32_t)C::NT;
}

template <class C, bool QUANT>
__device__ __forceinline__ uint32_t sort_merge(MLds<C>& m, uint32_t PT, uint32_t L, uint32_t total, uint32_t qbits)
{
    constexpr int NT = C::NT, KR = (int)kSortPer;
    static_assert(3u * kSortPer * (uint32_t)NT <= C::CAP, "a search reads below 3 kSortPer NT");
    const uint32_t tid = threadIdx.x, lane = tid & 63u, wv = tid >> 6;
    const uint32_t wfirst = (uint32_t)__builtin_amdgcn_readfirstlane((int)(tid & ~63u));
    for (uint32_t i = tid; i < (kMaxLevels + 1u) * kMSlots; i += NT) m.ecnt[i] = 0u;
    if (wv == 0u) {  // the longest run (PT <= 64: one wave)
        uint32_t n = lane < PT ? m.len[lane] : 0u;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) n = max(n, (uint32_t)__shfl_xor((int)n, o));
        if (lane == 0u) m.lmax = n;
    }

    // entries tid + k NT in the slots' layout: index, value and slot to LDS
    {
        uint32_t sl[KR], pos[KR], xi[KR];
        float xv[KR];
#pragma unroll
        for (int k = 0; k < KR; ++k) {
            const uint32_t e = tid + (uint32_t)k * NT;
            sl[k] = pos[k] = xi[k] = 0u;
            xv[k] = 0.0f;
            if (e < total) {
                const uint32_t s = last_at_most<6>(m.start, PT, e);
                sl[k] = s;
                pos[k] = m.first[s] + e - m.start[s];
            }
        }
#pragma unroll
        for (int k = 0; k < KR; ++k) {
            if (tid + (uint32_t)k * NT < total) {
                const uint32_t s = sl[k];
                xi[k] = as_global(m.pi[s])[pos[k]];
                if (QUANT) {
                    const uint32_t code = load_code(as_global(static_cast<const uint8_t*>(m.pv[s])), pos[k], qbits);
                    xv[k] = dequant(code, qbits, m.unit[s]);
                } else {
                    xv[k] = as_global(static_cast<const float*>(m.pv[s]))[pos[k]];
                }
            }
        }
#pragma unroll
        for (int k = 0; k < KR; ++k) {
            const uint32_t e = tid + (uint32_t)k * NT;
            if (e < total) {
                m.idx[e] = xi[k];
                m.val[e] = xv[k];
                m.rk[e] = (uint8_t)sl[k];
            }
        }
    }
    __syncthreads();

    // places: item it = tid + k NT searches for entry it / G in the slots
    // it % G, it % G + G, ...; the G lanes' counts are added across lanes.
    // A count is bounded by its run's length, so a place is below total
    // whatever the indices.
    uint32_t lg = 0;  // log2 G (uniform): while items fit the threads and a lane keeps eight slots
    while (lg < 3u && (total << (lg + 1u)) <= (uint32_t)NT && (8u << (lg + 1u)) <= PT) ++lg;
    const uint32_t G = 1u << lg;
    const int steps = 32 - __clz((int)__builtin_amdgcn_readfirstlane((int)m.lmax));
    uint32_t at[KR], ex[KR], es[KR];
    float ev[KR];
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        at[k] = ex[k] = es[k] = 0u;
        ev[k] = 0.0f;
        if (wfirst + (uint32_t)k * NT >= (total << lg)) continue;  // no item in the wave (uniform)
        const uint32_t it = tid + (uint32_t)k * NT, e = it >> lg, h = it & (G - 1u);
        const bool in = e < total;
        const uint32_t ec = in ? e : 0u;
        const uint32_t x = m.idx[ec], s = m.rk[ec] & (kMSlots - 1u);
        ex[k] = x;
        es[k] = s;
        ev[k] = m.val[ec];
        uint32_t cnt = in && h == 0u ? ec - m.start[s] : 0u;  // own position, by the first lane
        for (uint32_t b0 = 0; b0 < PT; b0 += 8u << lg) {
            uint32_t c[8], st1[8], n[8], xt[8];
#pragma unroll
            for (uint32_t j = 0; j < 8u; ++j) {
                const uint32_t s2 = b0 + h + (j << lg), s2c = min(s2, kMSlots - 1u);
                const uint32_t len = m.len[s2c];
                st1[j] = s2 < PT ? m.start[s2c] - 1u : 0u;
                n[j] = in && s2 < PT && s2 != s ? len : 0u;
                xt[j] = s2 < s ? x + 1u : x;  // lower slots: equal indices precede too
                c[j] = 0u;
            }
            for (int t = steps - 1; t >= 0; --t) {
#pragma unroll
                for (uint32_t j = 0; j < 8u; ++j) {
                    // (read whether or not cc lies in the run: start + cc - 1
                    // < total + 2 lmax, inside the array.  The test is bitwise:
                    // a short-circuit one would be compiled into a branch
                    // around the read, with a wait of its own)
                    const uint32_t cc = c[j] + (1u << t);
                    const uint32_t y = m.idx[st1[j] + cc];
                    const uint32_t take = (uint32_t)(y < xt[j]) & (uint32_t)(cc <= n[j]);
                    c[j] = take ? cc : c[j];
                }
            }
#pragma unroll
            for (uint32_t j = 0; j < 8u; ++j) cnt += c[j];
        }
        for (uint32_t o = 1; o < G; o <<= 1) cnt += (uint32_t)__shfl_xor((int)cnt, (int)o);
        at[k] = in && h == 0u ? cnt : kNone;
    }
    __syncthreads();  // every search read done
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        if (at[k] != kNone && wfirst + (uint32_t)k * NT < (total << lg)) {
            m.idx[at[k]] = ex[k];
            m.val[at[k]] = ev[k];
            m.rk[at[k]] = (uint8_t)es[k];
        }
    }
    __syncthreads();

    // ordered positions tid KR + k: group spans, and the sum of each index
    // whose first entry is here (the stack in place over the index's values)
    uint32_t ox[KR], heads = 0, nh = 0;
    float ov[KR];
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        const uint32_t p = tid * (uint32_t)KR + (uint32_t)k;
        ox[k] = 0u;
        ov[k] = 0.0f;
        if (p >= total) continue;
        const uint32_t xp = m.idx[p], r = m.rk[p] & (kMSlots - 1u);
        const bool head = p == 0u || m.idx[p - 1u] != xp;
        uint32_t span = L;
        if (!head) {
            const uint32_t d = r ^ m.rk[p - 1u];
            span = d ? min(31u - (uint32_t)__clz((int)d), L) : 0u;
        }
        if (span) atomicAdd(&m.ecnt[span * kMSlots + r], 1u);
        if (!head) continue;
        uint32_t i = p + 1u;
        if (i < total && m.idx[i] == xp) {
            // stack: values at p .. p + sp - 1, pending separators as bits
            // (strictly falling from the bottom: the lowest is the top)
            uint32_t sp = 1u, pend = 0u, prev = r;
            auto fold = [&]() {
                m.val[p + sp - 2u] = m.val[p + sp - 2u] + m.val[p + sp - 1u];
                --sp;
                pend &= pend - 1u;
            };
            do {
                const uint32_t ri = m.rk[i];
                const float vi = m.val[i];
                const uint32_t d = ri ^ prev;
                const uint32_t h = d ? 31u - (uint32_t)__clz((int)d) : 0u;
                while (pend && (uint32_t)__builtin_ctz(pend) < h) fold();
                pend |= 1u << h;
                m.val[p + sp] = vi;  // (p + sp <= i: read already)
                ++sp;
                prev = ri;
                ++i;
            } while (i < total && m.idx[i] == xp);
            while (pend) fold();
        }
        ox[k] = xp;
        ov[k] = m.val[p];
        heads |= 1u << k;
        ++nh;
    }
    uint32_t R;
    uint32_t o = wg_excl_scan<NT>(nh, m.w, &R);  // its first barrier: every read above done
#pragma unroll
    for (int k = 0; k < KR; ++k) {
        if (heads & (1u << k)) {
            m.idx[o] = ox[k];
            m.val[o] = ov[k];
            ++o;
        }
    }
    // node sizes, level order: wave l - 1 takes level l (below the root),
    // lane r slot r's spans that reach level l, summed over the node's 2^l
    // slots across lanes; the root holds every index once
    if (wv + 1u < L) {  // (uniform)
        const uint32_t l = wv + 1u;
        uint32_t c = 0;
        if (lane < PT) {
#pragma unroll
            for (uint32_t j = 1; j <= kMaxLevels; ++j) c += j >= l && j <= L ? m.ecnt[j * kMSlots + lane] : 0u;
        }
        for (uint32_t d = 1; d < (1u << l); d <<= 1) c += (uint32_t)__shfl_xor((int)c, (int)d);
        if (lane < PT && (lane & ((1u << l) - 1u)) == 0u) m.cnt[PT - (PT >> (l - 1u)) + (lane >> l)] = c;
    }
    if (tid == 0u) m.cnt[PT - 2u] = R;
    __syncthreads();
    return R;
}

// Node t of the P'-slot tree (level order) goes to position o of node_nnz /
// node_dense: the first nfold level-1 nodes, then every higher node.
__device__ __forceinline__ bool report_slot(uint32_t t, uint32_t PT, uint32_t nfold, uint32_t* o)
{
    if (t + 1u >= PT || (t < PT / 2u && t >= nfold)) return false;
    *o = t < PT / 2u ? t : t - PT / 2u + nfold;
    return true;
}

// ------------------------------------------------------------------------
// One workgroup, the whole range.

struct MTable {
    StreamDesc d[kSmallSlots];
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

template <bool QUANT>
__global__ void __launch_bounds__(SmallCfg::NT) k_merge_small(MTable kt, MArgs a)
{
    using C = SmallCfg;
    __shared__ MLds<C> m;
    const uint32_t tid = threadIdx.x, PT = a.PT;
    uint32_t n = 0;
    if (tid < PT) {
        const StreamDesc d = kt.d[tid];
        n = (uint32_t)d.nnz;
        m.pi[tid] = d.idx;
        m.pv[tid] = QUANT ? static_cast<const void*>(d.qval) : static_cast<const void*>(d.val);
        m.first[tid] = 0u;
        if (QUANT) m.unit[tid] = n ? level_unit(*d.qscale, a.qbits) : 0.0f;
    }
    const uint32_t total = slot_starts(m, PT, n);
    uint32_t root;
    if (sort_fits<C>(total)) {
        root = sort_merge<C, QUANT>(m, PT, a.L, total, a.qbits);
    } else {
        load_runs<C, QUANT>(m, PT, total, a.qbits);
        root = merge_levels(m, PT, a.L);
    }
    for (uint32_t e = tid; e < root; e += C::NT) {
        a.out_idx[e] = m.idx[e];
        a.out_val[e] = m.val[e];
    }
    uint32_t o;
    if (report_slot(tid, PT, a.nfold, &o)) {
        if (a.node_nnz) a.node_nnz[o] = m.cnt[tid];
        if (a.node_dense) a.node_dense[o] = 0u;
    }
    if (tid == 0) {
        const ReduceResult r{root, 0u, 0u};
        *a.hdr = r;
        if (a.result) *a.result = r;
    }
}

// ------------------------------------------------------------------------
// One workgroup per segment.

struct SArgs {
    const StreamDesc* tab;
    const uint32_t* off;  // [PT][nseg + 1] stream position of each segment's first entry
    SegState st;
    uint32_t PT, L, qbits, nfold, nseg;
    uint64_t lo, segw, N;  // range [lo, lo + N); segment s: [lo + s segw, lo + min((s + 1) segw, N))
    uint32_t* out_idx;
    float* out_val;
    uint64_t* node_nnz;
    uint8_t* node_dense;
    ReduceResult* hdr;
    ReduceResult* result;
};

// look-back words: status (1 the segment's own size, 2 the sum through it)
// in the top two bits, the size or sum below
constexpr unsigned long long kAgg = 1ull << 62, kIncl = 2ull << 62, kValMask = (1ull << 62) - 1ull;
constexpr uint32_t kSpinLimit = 1u << 24;  // polls of one predecessor before the look-back gives up

// First position in [a, b) of a sorted stream whose index is at least x.
__device__ __forceinline__ uint32_t first_at_least(const uint32_t* idx, uint32_t a, uint32_t b, uint64_t x)
{
    while (a < b) {
        const uint32_t mid = a + ((b - a) >> 1);
        if ((uint64_t)as_global(idx)[mid] < x) a = mid + 1u;
        else b = mid;
    }
    return a;
}

// The pieces of a segment that does not fit, in index order: its range
// halved until each piece does (one index holds at most PT entries).
// write = false: count (the pieces' node sizes added to s_acc); true: write
// the pieces' roots from `at` on.  Returns the entries of the roots.  Whole
// workgroup; slot r's entries in the segment are at stream positions [ra, rb).
template <bool QUANT, class C>
__device__ __forceinline__ unsigned long long seg_pieces(MLds<C>& m, const SArgs& a, bool write,
                                                         unsigned long long at, uint32_t ra, uint32_t rb,
                                                         uint64_t c0, uint64_t c1, uint32_t* s_acc,
                                                         uint64_t* s_lo, uint64_t* s_hi, uint32_t* s_depth,
                                                         uint32_t* s_fits)
{
    const uint32_t tid = threadIdx.x, PT = a.PT;
    unsigned long long done = 0;
    if (tid == 0) {
        *s_depth = 1u;
        s_lo[0] = c0;
        s_hi[0] = c1;
    }
    __syncthreads();
    while (*s_depth) {
        const uint32_t depth = *s_depth;
        const uint64_t x0 = s_lo[depth - 1u], x1 = s_hi[depth - 1u];
        uint32_t n = 0;
        if (tid < PT) {
            const uint32_t p0 = first_at_least(m.pi[tid], ra, rb, x0);
            const uint32_t p1 = first_at_least(m.pi[tid], p0, rb, x1);
            m.first[tid] = p0;
            n = p1 - p0;
        }
        const uint32_t pt = slot_starts(m, PT, n);  // its barriers follow every read of the stack top
        if (tid == 0) {
            // a single index holds at most PT entries of valid streams; more
            // (unsorted input) is reported and the index skipped
            *s_fits = pt <= C::CAP ? 1u : (x1 - x0 <= 1u ? 2u : 0u);
            if (*s_fits == 2u) atomicOr(a.st.err, 2u);
            if (*s_fits) {
                *s_depth = depth - 1u;
            } else {  // halves, the lower one on top
                const uint64_t mid = x0 + (x1 - x0) / 2u;
                s_lo[depth - 1u] = mid;
                s_lo[depth] = x0;
                s_hi[depth] = mid;
                *s_depth = depth + 1u;
            }
        }
        __syncthreads();
        if (*s_fits != 1u) continue;
        load_runs<C, QUANT>(m, PT, pt, a.qbits);
        const uint32_t root = merge_levels(m, PT, a.L);
        if (write) {
            for (uint32_t e = tid; e < root; e += C::NT) {
                a.out_idx[at + done + e] = m.idx[e];
                a.out_val[at + done + e] = m.val[e];
            }
        } else if (tid + 1u < PT) {
            s_acc[tid] += m.cnt[tid];
        }
        done += root;
        __syncthreads();
    }
    return done;
}

template <bool QUANT, class C>
__global__ void __launch_bounds__(C::NT) k_merge_seg(SArgs a)
{
    __shared__ MLds<C> m;
    __shared__ uint32_t s_seg, s_last, s_ok;
    __shared__ unsigned long long s_excl;
    __shared__ uint32_t s_acc[kMSlots - 1];  // node sizes of the segment
    __shared__ uint64_t s_lo[40], s_hi[40];  // pieces still to do (a stack)
    __shared__ uint32_t s_depth, s_fits;
    const uint32_t tid = threadIdx.x, PT = a.PT;
    // the slot's descriptor (and level unit) are read while the ticket is
    // taken
    StreamDesc d{};
    float unit = 0.0f;
    if (tid < PT) {
        d = a.tab[tid];
        if (QUANT && d.nnz) unit = level_unit(*d.qscale, a.qbits);
    }
    if (tid == 0) s_seg = atomicAdd(a.st.ticket, 1u);
    __syncthreads();
    const uint32_t s = s_seg, stride = a.nseg + 1u;
    uint32_t ra = 0, rb = 0;  // this slot's entries in the segment: stream positions [ra, rb)
    if (tid < PT) {
        // (offsets clamped to the stream: one that does not ascend leaves
        // some unwritten)
        const uint32_t nz = (uint32_t)d.nnz;
        ra = min(a.off[tid * stride + s], nz);
        rb = min(a.off[tid * stride + s + 1u], nz);
        if (rb < ra) {  // only for streams that do not ascend: reported, the slot skipped
            atomicOr(a.st.err, 2u);
            rb = ra;
        }
        m.pi[tid] = d.idx;
        m.pv[tid] = QUANT ? static_cast<const void*>(d.qval) : static_cast<const void*>(d.val);
        m.first[tid] = ra;
        if (QUANT) m.unit[tid] = unit;
    }
    if (tid < kMSlots - 1u) s_acc[tid] = 0u;
    const uint32_t total = slot_starts(m, PT, rb - ra);
    const uint64_t c0 = a.lo + (uint64_t)s * a.segw, c1 = a.lo + min((uint64_t)(s + 1u) * a.segw, a.N);

    // this segment's union size (and node sizes)
    unsigned long long R;
    const bool big = total > C::CAP;  // uniform
    if (!big && sort_fits<C>(total)) {
        R = sort_merge<C, QUANT>(m, PT, a.L, total, a.qbits);
        if (tid + 1u < PT) s_acc[tid] = m.cnt[tid];
    } else if (!big) {
        load_runs<C, QUANT>(m, PT, total, a.qbits);
        R = merge_levels(m, PT, a.L);
        if (tid + 1u < PT) s_acc[tid] = m.cnt[tid];
    } else {
        R = seg_pieces<QUANT, C>(m, a, false, 0ull, ra, rb, c0, c1, s_acc, s_lo, s_hi, &s_depth, &s_fits);
    }
    __syncthreads();

    // its output offset: decoupled look-back over the lower segments, by the
    // first wave, 64 predecessors at a time (lane l reads segment j0 - 1 - l;
    // those below segment 0 read as a finished sum of 0): the sizes up to the
    // nearest finished sum are added once every one of them is there
    if (tid < 64u) {
        unsigned long long* f = a.st.flags;
        const uint32_t lane = tid;
        if (lane == 0)
            __hip_atomic_store(&f[s], (s ? kAgg : kIncl) | R, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        unsigned long long excl = 0;
        uint32_t ok = 1u, spins = 0;
        int j0 = (int)s;
        while (j0 > 0) {
            const int j = j0 - 1 - (int)lane;
            const unsigned long long v =
                j >= 0 ? __hip_atomic_load(&f[j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : kIncl;
            const uint64_t fin = __ballot((v >> 62) == 2ull), miss = __ballot((v >> 62) == 0ull);
            const uint32_t upto = fin ? (uint32_t)__builtin_ctzll(fin) : 64u;  // nearest finished sum
            const uint64_t need = upto >= 63u ? ~0ull : (2ull << upto) - 1ull;
            if (miss & need) {  // a size still missing: wait and read again
                if (++spins > kSpinLimit) {
                    ok = 0u;
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
                continue;
            }
            unsigned long long part = lane <= upto ? (v & kValMask) : 0ull;
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o);
            excl += part;
            if (upto < 64u) break;
            j0 -= 64;
        }
        if (lane == 0) {
            if (ok) {
                if (s) __hip_atomic_store(&f[s], kIncl | (excl + R), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            } else {
                atomicOr(a.st.err, 1u);  // bit 0: a look-back gave up
            }
            s_excl = excl;
            s_ok = ok;
        }
    }
    __syncthreads();
    if (s_ok) {
        if (!big) {
            for (uint32_t e = tid; e < (uint32_t)R; e += C::NT) {
                a.out_idx[s_excl + e] = m.idx[e];
                a.out_val[s_excl + e] = m.val[e];
            }
        } else {
            seg_pieces<QUANT, C>(m, a, true, s_excl, ra, rb, c0, c1, s_acc, s_lo, s_hi, &s_depth, &s_fits);
        }
    }

    // node sizes; the last workgroup to finish reports them and the root.
    // The first wave adds the segment's node sizes (device atomics) and
    // waits until they are acknowledged before counting itself done, so the
    // workgroup that counts last finds every size added.  (No release
    // fence: on this chip that writes back the whole L2, and hundreds of
    // them stall the look-back of the other segments.)
    if (tid < 64u) {
        if (tid + 1u < PT && s_acc[tid]) atomicAdd(&a.st.node_cnt[tid], s_acc[tid]);
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        if (tid == 0) {
            const uint32_t prev = atomicAdd(a.st.done, 1u);
            s_last = prev + 1u == a.nseg ? 1u : 0u;
        }
    }
    __syncthreads();
    if (!s_last) return;
    uint32_t o;
    if (report_slot(tid, PT, a.nfold, &o)) {
        const uint32_t c = __hip_atomic_load(&a.st.node_cnt[tid], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (a.node_nnz) a.node_nnz[o] = c;
        if (a.node_dense) a.node_dense[o] = 0u;
    }
    if (tid == 0) {
        const uint32_t root = __hip_atomic_load(&a.st.node_cnt[PT - 2u], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const uint32_t err = __hip_atomic_load(a.st.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        const ReduceResult r{root, 0u, err};
        *a.hdr = r;
        if (a.result) *a.result = r;
    }
}

}  // namespace

bool merge_small_fits(uint32_t PT, uint64_t sum_nnz, uint64_t thr)
{
    if (PT < 2 || PT > kSmallSlots || sum_nnz > thr) return false;  // every node sparse
    const uint64_t most = PT == 2 ? SmallCfg::CAP : (PT == 4 ? 8192u : 1024u);
    return sum_nnz <= most;
}

hipError_t merge_small_run(uint32_t PT, uint32_t L, uint32_t qbits, uint32_t nfold, const StreamDesc* host_tab,
                           uint32_t* out_idx, float* out_val, uint64_t* node_nnz, uint8_t* node_dense,
                           ReduceResult* hdr, ReduceResult* result, hipStream_t s)
{
    if (PT > kSmallSlots) return hipErrorInvalidValue;
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
    if (qbits) hipLaunchKernelGGL(k_merge_small<true>, dim3(1), dim3(SmallCfg::NT), 0, s, kt, a);
    else hipLaunchKernelGGL(k_merge_small<false>, dim3(1), dim3(SmallCfg::NT), 0, s, kt, a);
    timer_end(kTReduceMerge, s);
    return hipGetLastError();
}

bool merge_seg_fits(uint32_t PT, uint64_t sum_nnz, uint64_t thr)
{
    return PT >= 2 && PT <= kMSlots && sum_nnz <= thr && sum_nnz <= kSegMaxEntries;
}

void merge_seg_shape(uint64_t R, uint64_t sum_nnz, uint32_t* nseg, uint64_t* segw)
{
    // about kSegEntries expected entries a segment, but at least kSegMin
    // segments: a smaller segment loads sooner and its merge-path searches
    // are shorter, and the chip holds far more workgroups than that
    uint64_t n = std::max<uint64_t>((sum_nnz + kSegEntries - 1) / kSegEntries, kSegMin);
    n = std::max<uint64_t>(1, std::min<uint64_t>(std::min<uint64_t>(n, kSegMax), R));
    const uint64_t w = (R + n - 1) / n;
    *segw = w;
    *nseg = (uint32_t)((R + w - 1) / w);
}

bool merge_seg_short(uint64_t sum_nnz, uint32_t nseg)
{
    // the units of a segment (its expected entries over 3) fit one a thread
    return nseg && (sum_nnz + nseg - 1) / nseg <= 3u * (uint64_t)SegShortCfg::NT;
}

hipError_t merge_seg_run(uint32_t PT, uint32_t L, uint32_t qbits, uint32_t nfold, const StreamDesc* dev_tab,
                         const uint32_t* off, const SegState& st, uint32_t nseg, uint64_t lo, uint64_t segw,
                         uint64_t N, uint32_t* out_idx, float* out_val, uint64_t* node_nnz, uint8_t* node_dense,
                         ReduceResult* hdr, ReduceResult* result, bool short_units, hipStream_t s)
{
    if (PT > kMSlots || nseg == 0 || nseg > kSegMax) return hipErrorInvalidValue;
    SArgs a{};
    a.tab = dev_tab;
    a.off = off;
    a.st = st;
    a.PT = PT;
    a.L = L;
    a.qbits = qbits;
    a.nfold = nfold;
    a.nseg = nseg;
    a.lo = lo;
    a.segw = segw;
    a.N = N;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.node_nnz = node_nnz;
    a.node_dense = node_dense;
    a.hdr = hdr;
    a.result = result;
    timer_begin(kTReduceMerge, s);
    if (short_units) {
        if (qbits) hipLaunchKernelGGL((k_merge_seg<true, SegShortCfg>), dim3(nseg), dim3(SegShortCfg::NT), 0, s, a);
        else hipLaunchKernelGGL((k_merge_seg<false, SegShortCfg>), dim3(nseg), dim3(SegShortCfg::NT), 0, s, a);
    } else {
        if (qbits) hipLaunchKernelGGL((k_merge_seg<true, SegCfg>), dim3(nseg), dim3(SegCfg::NT), 0, s, a);
        else hipLaunchKernelGGL((k_merge_seg<false, SegCfg>), dim3(nseg), dim3(SegCfg::NT), 0, s, a);
    }
    timer_end(kTReduceMerge, s);
    return hipGetLastError();
}

}  // namespace sparcml
