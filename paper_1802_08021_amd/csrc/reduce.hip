// Sparse allreduce of P sparse streams on one gfx950 GPU: the local
// reduction work of SparCML's recursive-doubling sparse allreduce (§5.3.1,
// Fig. 2) with the sparse->dense switch of §5.1.
//
// Design (why it differs from a level-by-level merge): every rank's stream
// lives in HBM, so instead of materialising the P-1 intermediate streams of
// the tree (which moves log2(P) times the data), the coordinate space is cut
// into tiles of T indices and each tile evaluates the whole tree at once:
//
//  * a rank bitmask per coordinate (LDS) records which ranks hold it; the
//    popcount prefix of the mask places each rank's value in rank order;
//  * a per-coordinate walk over the present ranks sums the values with the
//    exact association of the tree: two ranks first meet at the level given
//    by the highest differing bit of their numbers, so a stack keyed by that
//    level reproduces ((r0+r1)+(r2+r3))... for any subset of ranks;
//  * the exact union size of every tree node -- what the switch rule needs --
//    is counted on the side: the entry of rank r whose predecessor (next
//    lower present rank) differs from r first at bit h opens a new group at
//    levels 1..h (all levels if it has no predecessor);
//  * a dense node's value at an index equals the tree sum (+0.0 where no rank
//    contributes), so a dense root is written tile by tile, once.
//
// Passes: partition (per-chunk stream offsets) -> tile pass (COUNT, or DENSE
// when the root is likely dense) -> slow pass for tiles that overflow the
// fast path's LDS budget -> decide (switch rule over the node counts) ->
// [scan of per-tile union sizes -> SPARSE_WRITE tile and slow passes].
#include "internal.h"
#include "qsgd_device.h"

#include <algorithm>

namespace sparcml {
namespace {

enum Mode { kCount = 0, kDense = 1, kSparseWrite = 2 };

// Pointers that live in memory (descriptor tables, LDS) are generic unless
// marked: generic (FLAT) loads also count against the LDS wait counter and
// would serialize the LDS work behind every HBM access.
typedef const uint32_t __attribute__((address_space(1))) g_u32;
typedef const uint8_t __attribute__((address_space(1))) g_u8;
typedef const float __attribute__((address_space(1))) g_f32;
constexpr uint32_t kCap = 4096;  // entries per tile on the fast path
constexpr uint32_t kWin = 64;    // entries read per rank per tile (one wave)
constexpr int kSlowNT = 256;
constexpr int kSlowTS = 1024;    // coordinates per slow-path sub-tile

// MW = 32-bit rank-mask words per coordinate = ceil(P / 32).  Every fast
// tile kernel has 256 threads; TMAX coordinates of masks take 16 KB of LDS;
// CAP entries per tile fit the fast path.  Ranks are read in pairs: one
// 64-lane load covers a 32-entry window of two ranks.
template <int MW>
struct Shape {
    static constexpr int NT = 256, NW = 4;
    static constexpr int TMAX = 4096 / MW;
    static constexpr int LMAX = MW == 1 ? 5 : (MW == 2 ? 6 : (MW == 4 ? 7 : 8));
    static constexpr int PMAX = 32 * MW;
    static constexpr int CAP = 2048;
    static constexpr int SLOTS = PMAX / 2 / NW;  // rank pairs per wave
};
constexpr uint32_t kHalf = 32;  // window per rank per tile

struct Args {
    const StreamDesc* tab;
    const uint32_t* off;       // [P][nchunks+1] first entry of each chunk
    uint32_t* tile_cnt;        // [ntiles] union size of the root per tile
    const uint32_t* tile_off;  // [ntiles] exclusive scan of tile_cnt
    uint32_t* slow_list;       // [ntiles]
    uint32_t* slow_count;      // [1]
    uint32_t* node_cnt;        // [P-1] union size per tree node
    uint32_t* out_idx;
    float* out_val;
    uint32_t P, L, N, T, ntiles, nchunks, tpc, qbits;
};

__device__ __forceinline__ uint32_t lower_bound(const uint32_t* a, uint32_t lo, uint32_t hi,
                                                uint64_t x)
{
    while (lo < hi) {
        const uint32_t mid = lo + ((hi - lo) >> 1);
        if ((uint64_t)a[mid] < x) lo = mid + 1;
        else hi = mid;
    }
    return lo;
}

// The MW rank-mask words of index j (vector LDS access where possible).
template <int MW>
__device__ __forceinline__ void load_mask(const uint32_t* m, uint32_t j, uint32_t (&w)[MW])
{
    if constexpr (MW == 1) {
        w[0] = m[j];
    } else if constexpr (MW == 2) {
        const uint2 v = reinterpret_cast<const uint2*>(m)[j];
        w[0] = v.x;
        w[1] = v.y;
    } else {
#pragma unroll
        for (int k = 0; k < MW / 4; ++k) {
            const uint4 v = reinterpret_cast<const uint4*>(m)[j * (MW / 4) + k];
            w[4 * k] = v.x;
            w[4 * k + 1] = v.y;
            w[4 * k + 2] = v.z;
            w[4 * k + 3] = v.w;
        }
    }
}

template <int MW>
__device__ __forceinline__ void clear_mask(uint32_t* m, uint32_t j)
{
    if constexpr (MW == 1) {
        m[j] = 0u;
    } else if constexpr (MW == 2) {
        reinterpret_cast<uint2*>(m)[j] = make_uint2(0u, 0u);
    } else {
#pragma unroll
        for (int k = 0; k < MW / 4; ++k) reinterpret_cast<uint4*>(m)[j * (MW / 4) + k] = make_uint4(0u, 0u, 0u, 0u);
    }
}

// Level t (1-based) and group g of internal node `node` in level order.
__device__ __forceinline__ void node_coords(uint32_t node, uint32_t P, uint32_t* t, uint32_t* g)
{
    uint32_t lvl = 1, base = 0;
    while (node >= base + (P >> lvl)) {
        base += P >> lvl;
        ++lvl;
    }
    *t = lvl;
    *g = node - base;
}

// Turn per-rank counts into node union sizes and add them to the global
// counters.  E[r][d], d < L: entries of rank r whose predecessor (next lower
// rank present at the same index) first differs from r at bit d -- such an
// entry opens a new group at levels 1..d; E[r][L]: all entries of rank r,
// of which those without predecessor open new groups at every level.
// Node (t, g) counts the entries of its ranks that open a group at level t.
template <int NT>
__device__ void flush_counts(uint32_t* E, const Args& a)
{
    const uint32_t P = a.P, L = a.L, W = L + 1;
    for (uint32_t r = threadIdx.x; r < P; r += NT) {
        uint32_t acc = E[r * W + L];
        for (uint32_t d = 0; d < L; ++d) acc -= E[r * W + d];
        E[r * W + L] = acc;
        for (int d = (int)L - 1; d >= 1; --d) {
            acc += E[r * W + d];
            E[r * W + d] = acc;
        }
    }
    __syncthreads();
    for (uint32_t node = threadIdx.x; node + 1 < P; node += NT) {
        uint32_t t, g;
        node_coords(node, P, &t, &g);
        uint32_t sum = 0;
        for (uint32_t r = g << t; r < ((g + 1) << t); ++r) sum += E[r * W + t];
        if (sum) atomicAdd(&a.node_cnt[node], sum);
    }
}

// ------------------------------------------------------------------------
// Fast tile pass.  One workgroup walks a chunk of consecutive tiles of T
// indices.  Per tile:
//   A  each wave reads a 32-entry window of two ranks per 64-lane load and
//      counts, by ballot, how many fall in the tile;
//   B  the entries are compacted into LDS (rank-major) and their rank bits
//      set in the per-index masks;
//   2  per index: ranks present (popcount), exclusive scan -> where each
//      index's values start, in rank order;
//   3  per entry: value placed at its index's start plus the number of lower
//      ranks present; entries with a predecessor counted by split level;
//   4  per thread: a flat walk over its indices' values, summing each index
//      with the tree's association, then one write of the tile.
// Tiles where a rank fills its window or with more than CAP entries go to
// the slow pass.
template <int MW, int MODE, bool QUANT>
__global__ void __launch_bounds__(256) k_tiles(Args a)
{
    using S = Shape<MW>;
    constexpr int NT = S::NT, NW = S::NW, TMAX = S::TMAX, LMAX = S::LMAX, PMAX = S::PMAX;
    constexpr int CAP = S::CAP, SLOTS = S::SLOTS, CPTMAX = TMAX / NT;
    __shared__ uint4 s_mask4[TMAX * MW / 4];
    __shared__ uint32_t s_ent[2 * CAP];  // [0,CAP): index<<8 | rank; [CAP,2CAP): value bits
    __shared__ float s_vals[MODE == kCount ? 1 : CAP];
    __shared__ uint16_t s_bin[MODE == kCount ? 1 : TMAX];
    __shared__ uint32_t s_E[MODE == kSparseWrite ? 1 : PMAX * (LMAX + 1)];
    __shared__ uint32_t s_cur[PMAX], s_end[PMAX], s_cnt[PMAX], s_last[PMAX];
    __shared__ g_u32* s_ip[PMAX];
    __shared__ g_u32* s_vp[PMAX];  // fp32 bits, or packed codes (byte-addressed)
    __shared__ float s_unit[QUANT ? PMAX : 1];
    __shared__ uint32_t s_wsum[CPTMAX * NW];
    __shared__ uint32_t s_slow;
    uint32_t* s_mask = reinterpret_cast<uint32_t*>(s_mask4);
    uint32_t* s_entv = s_ent + CAP;
    float* s_out = reinterpret_cast<float*>(s_ent);  // phase 4 only (T <= 2*CAP)

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t half = (uint32_t)lane >> 5, sl = (uint32_t)lane & 31u;
    const uint32_t P = a.P, L = a.L, T = a.T, CPT = T / NT, W = L + 1;
    const uint32_t chunk = blockIdx.x, stride = a.nchunks + 1;
    const uint32_t t0 = chunk * a.tpc, t1 = min(t0 + a.tpc, a.ntiles);
    const uint32_t RPL = P > 64 ? P / 64 : 1;  // ranks per lane in the rank scan

    for (uint32_t r = tid; r < P; r += NT) {
        const StreamDesc* d = &a.tab[r];
        s_cur[r] = a.off[r * stride + chunk];
        s_end[r] = a.off[r * stride + chunk + 1];
        // empty streams read (and discard) a word of the descriptor table
        const bool empty = d->nnz == 0;
        s_last[r] = empty ? 0u : (uint32_t)(d->nnz - 1);
        const void* ip = empty ? static_cast<const void*>(a.tab) : static_cast<const void*>(d->idx);
        const void* vp = empty ? static_cast<const void*>(a.tab)
                               : (QUANT ? static_cast<const void*>(d->qval) : static_cast<const void*>(d->val));
        s_ip[r] = (g_u32*)ip;
        s_vp[r] = (g_u32*)vp;
        if (QUANT) s_unit[r] = level_unit(*d->qscale, a.qbits);
    }
    if (MODE != kSparseWrite)
        for (uint32_t i = tid; i < P * W; i += NT) s_E[i] = 0;
    for (uint32_t i = tid; i < TMAX * MW / 4; i += NT) s_mask4[i] = make_uint4(0u, 0u, 0u, 0u);

    for (uint32_t tile = t0; tile < t1; ++tile) {
        const uint32_t tlo = tile * T;
        const uint32_t thi = (uint32_t)min((uint64_t)tlo + T, (uint64_t)a.N);
        __syncthreads();
        if (tid == 0) s_slow = 0;

        // A: windows of two ranks per load.  Straight-line code: every load
        // is issued before any is used (ranks past P read rank P-1 and are
        // masked out afterwards).
        uint32_t xs[SLOTS], vs[SLOTS], okbits = 0;
#pragma unroll
        for (int q = 0; q < SLOTS; ++q) {
            const uint32_t r = 2 * (uint32_t)(wv * SLOTS + q) + half;
            const uint32_t rr = min(r, P - 1);
            const uint32_t i = s_cur[rr] + sl;
            const uint32_t ic = min(i, s_last[rr]);
            xs[q] = s_ip[rr][ic];
            if (QUANT) {
                const uint32_t plog = a.qbits == 8u ? 0u : (a.qbits == 4u ? 1u : 2u);
                const uint32_t byte = ((g_u8*)s_vp[rr])[ic >> plog];
                vs[q] = (byte >> ((ic & ((1u << plog) - 1u)) * a.qbits)) & ((1u << a.qbits) - 1u);
            } else {
                vs[q] = s_vp[rr][ic];
            }
            okbits |= (uint32_t)(r < P && i < s_end[rr]) << q;
        }
        uint32_t inbits = 0;
#pragma unroll
        for (int q = 0; q < SLOTS; ++q) {
            const bool in = ((okbits >> q) & 1u) && xs[q] >= tlo && xs[q] < thi;
            inbits |= (uint32_t)in << q;
            const uint64_t bal = __ballot(in);
            const uint32_t c = (uint32_t)__popc((uint32_t)(bal >> (32 * half)));
            if (sl == 0) {
                s_cnt[2 * (uint32_t)(wv * SLOTS + q) + half] = c;
                if (c == kHalf) s_slow = 1u;
            }
        }
        __syncthreads();

        // Every wave scans the per-rank counts itself (RPL ranks per lane).
        uint32_t lsum = 0;
        for (uint32_t k = 0; k < RPL; ++k) {
            const uint32_t r = (uint32_t)lane * RPL + k;
            lsum += r < P ? s_cnt[r] : 0u;
        }
        uint32_t lincl = lsum;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = __shfl_up(lincl, o);
            if (lane >= o) lincl += y;
        }
        const uint32_t total = __shfl(lincl, 63);
        const uint32_t lexcl = lincl - lsum;

        if (s_slow || total > (uint32_t)CAP) {
            // Defer the tile and move every cursor past it (a rank may hold
            // more than one window's worth of entries here).
            for (int k = 0; k < 2 * SLOTS; ++k) {
                const uint32_t r = (uint32_t)(wv * 2 * SLOTS + k);
                if (r >= P) break;
                uint32_t n = s_cnt[r];
                if (n == kHalf) {
                    g_u32* idx = s_ip[r];
                    const uint32_t base = s_cur[r], end = s_end[r];
                    for (;;) {
                        const uint32_t i = base + n + lane;
                        const bool in = i < end && idx[i] < thi;
                        const uint32_t c = (uint32_t)__popcll(__ballot(in));
                        n += c;
                        if (c < 64) break;
                    }
                }
                if (lane == 0) s_cur[r] += n;
            }
            if (tid == 0) {
                const uint32_t k = atomicAdd(a.slow_count, 1u);
                a.slow_list[k] = tile;
            }
            continue;
        }

        // B: compact the entries (rank-major) and set the rank bits.
#pragma unroll
        for (int q = 0; q < SLOTS; ++q) {
            const uint32_t u = (uint32_t)(wv * SLOTS + q);
            if (2 * u < P) {
                const uint32_t r = 2 * u + half;
                const uint32_t lr = r / RPL;
                uint32_t base = __shfl(lexcl, (int)lr);
                for (uint32_t k = lr * RPL; k < r; ++k) base += s_cnt[k];
                if ((inbits >> q) & 1u) {
                    const uint32_t j = xs[q] - tlo;
                    s_ent[base + sl] = (j << 8) | r;
                    s_entv[base + sl] = vs[q];
                    atomicOr(&s_mask[j * MW + (r >> 5)], 1u << (r & 31u));
                }
            }
        }
        if (MODE != kSparseWrite)
            for (uint32_t r = tid; r < P; r += NT) s_E[r * W + L] += s_cnt[r];
        for (uint32_t r = tid; r < P; r += NT) s_cur[r] += s_cnt[r];
        __syncthreads();

        // 2: ranks per index.  Thread t owns indices q*NT + t (q < CPT), so
        // per-lane LDS accesses are consecutive (no bank conflicts) and the
        // dense write coalesces.  Exclusive scan over indices in order: one
        // wave scan per round q, the wave totals of all rounds exchanged
        // through LDS at once; packed (entries low 16 bits, non-empty high).
        uint32_t pk[CPTMAX], ex[CPTMAX];
#pragma unroll
        for (int q = 0; q < CPTMAX; ++q) {
            pk[q] = 0;
            ex[q] = 0;
            if ((uint32_t)q < CPT) {
                uint32_t w[MW];
                load_mask<MW>(s_mask, (uint32_t)q * NT + tid, w);
                uint32_t m = 0;
#pragma unroll
                for (int k = 0; k < MW; ++k) m += __popc(w[k]);
                pk[q] = m | ((m != 0u) << 16);
                uint32_t incl = pk[q];
#pragma unroll
                for (int o = 1; o < 64; o <<= 1) {
                    const uint32_t y = __shfl_up(incl, o);
                    if (lane >= o) incl += y;
                }
                ex[q] = incl - pk[q];
                if (lane == 63) s_wsum[q * NW + wv] = incl;
            }
        }
        __syncthreads();
        uint32_t run = 0;
#pragma unroll
        for (int q = 0; q < CPTMAX; ++q) {
            if ((uint32_t)q < CPT) {
                uint32_t before = 0, rtot = 0;
#pragma unroll
                for (int w = 0; w < NW; ++w) {
                    const uint32_t v = s_wsum[q * NW + w];
                    if (w < wv) before += v;
                    rtot += v;
                }
                ex[q] += run + before;
                run += rtot;
                if (MODE != kCount) s_bin[(uint32_t)q * NT + tid] = (uint16_t)(ex[q] & 0xFFFFu);
            }
        }
        if (MODE != kSparseWrite && tid == 0) a.tile_cnt[tile] = run >> 16;
        __syncthreads();

        // 3: per entry -- rank-ordered placement and split-level counts.
        for (uint32_t e = tid; e < total; e += NT) {
            const uint32_t ent = s_ent[e];
            const uint32_t r = ent & 0xFFu, j = ent >> 8;
            uint32_t w[MW];
            load_mask<MW>(s_mask, j, w);
            const uint32_t rw = r >> 5, lowbits = (1u << (r & 31u)) - 1u;
            if (MODE != kCount) {
                uint32_t below = 0;
#pragma unroll
                for (int k = 0; k < MW; ++k)
                    below += (uint32_t)k < rw ? __popc(w[k])
                                              : ((uint32_t)k == rw ? __popc(w[k] & lowbits) : 0u);
                const uint32_t vb = s_entv[e];
                const float v = QUANT ? dequant(vb, a.qbits, s_unit[r]) : __uint_as_float(vb);
                s_vals[s_bin[j] + below] = v;
            }
            if (MODE != kSparseWrite) {
                int prev = -1;
#pragma unroll
                for (int k = MW - 1; k >= 0; --k) {
                    const uint32_t cand = (uint32_t)k < rw ? w[k]
                                                           : ((uint32_t)k == rw ? (w[k] & lowbits) : 0u);
                    if (prev < 0 && cand) prev = k * 32 + 31 - (int)__clz(cand);
                }
                if (prev >= 0) atomicAdd(&s_E[r * W + (31u - (uint32_t)__clz(r ^ (uint32_t)prev))], 1u);
            }
        }
        __syncthreads();
        if (MODE == kCount) {
            for (uint32_t q = 0; q < CPT; ++q) clear_mask<MW>(s_mask, q * NT + tid);
            continue;
        }

        // 4: flat walk over this thread's entries, index by index (q order),
        // summing each index's values with the tree's association.
        uint32_t nent = 0;
#pragma unroll
        for (int q = 0; q < CPTMAX; ++q) nent += pk[q] & 0xFFFFu;
        if (MODE == kDense)
            for (uint32_t q = 0; q < CPT; ++q) s_out[q * NT + tid] = 0.0f;
        uint32_t q = 0, bits[MW];
        load_mask<MW>(s_mask, tid, bits);
        uint32_t pos = s_bin[tid];
        float slot[LMAX];
#pragma unroll
        for (int l = 0; l < LMAX; ++l) slot[l] = 0.0f;
        float cur = 0.0f;
        uint32_t pend = 0;
        int last = -1;
        for (uint32_t it = 0; it < nent; ++it) {
            for (;;) {  // next index with ranks left (nent guarantees one)
                uint32_t any = 0;
#pragma unroll
                for (int k = 0; k < MW; ++k) any |= bits[k];
                if (any) break;
                ++q;
                load_mask<MW>(s_mask, q * NT + tid, bits);
                pos = s_bin[q * NT + tid];
            }
            int r = -1;
#pragma unroll
            for (int k = 0; k < MW; ++k) {
                if (r < 0 && bits[k]) {
                    r = k * 32 + (__ffs(bits[k]) - 1);
                    bits[k] &= bits[k] - 1u;
                }
            }
            const float v = s_vals[pos++];
            if (last >= 0) {
                const int sep = 31 - (int)__clz((uint32_t)(r ^ last));
#pragma unroll
                for (int l = 0; l < LMAX; ++l)
                    if (l < sep && ((pend >> l) & 1u)) cur = slot[l] + cur;
                pend = (pend & ~((1u << sep) - 1u)) | (1u << sep);
#pragma unroll
                for (int l = 0; l < LMAX; ++l)
                    if (l == sep) slot[l] = cur;
            }
            cur = v;
            last = r;
            uint32_t left = 0;
#pragma unroll
            for (int k = 0; k < MW; ++k) left |= bits[k];
            if (!left) {  // index q*NT + tid complete
#pragma unroll
                for (int l = 0; l < LMAX; ++l)
                    if ((pend >> l) & 1u) cur = slot[l] + cur;
                const uint32_t j = q * NT + tid;
                if (MODE == kDense) {
                    s_out[j] = cur + 0.0f;
                } else {
                    uint32_t nz = 0;
#pragma unroll
                    for (int qq = 0; qq < CPTMAX; ++qq)
                        if ((uint32_t)qq == q) nz = ex[qq] >> 16;
                    const uint32_t o = a.tile_off[tile] + nz;
                    a.out_idx[o] = tlo + j;
                    a.out_val[o] = cur;
                }
                pend = 0;
                last = -1;
            }
        }
        for (uint32_t k = 0; k < CPT; ++k) clear_mask<MW>(s_mask, k * NT + tid);
        if (MODE == kDense) {
            for (uint32_t k = 0; k < CPT; ++k) {
                const uint32_t j = k * NT + tid;
                if ((uint64_t)tlo + j < thi) a.out_val[(uint64_t)tlo + j] = s_out[j];
            }
        }
    }
    __syncthreads();
    if (MODE != kSparseWrite) flush_counts<NT>(s_E, a);
}

// ------------------------------------------------------------------------
// Slow pass: one workgroup per deferred tile, any number of entries.  Ranks
// are taken in order; each coordinate keeps the tree-sum stack in LDS
// (current value, last rank, pending-level bits, one slot per level).
template <int MW, int MODE, bool QUANT>
__global__ void __launch_bounds__(kSlowNT) k_slow(Args a)
{
    constexpr int NT = kSlowNT, TS = kSlowTS, LMAX = Shape<MW>::LMAX, PMAX = 32 * MW;
    __shared__ float s_slot[LMAX][TS];
    __shared__ float s_curv[TS];
    __shared__ int16_t s_last[TS];
    __shared__ uint16_t s_pend[TS];
    __shared__ uint32_t s_E[PMAX * (LMAX + 1)];
    __shared__ uint32_t s_lo[PMAX], s_hi[PMAX];
    __shared__ float s_unit[QUANT ? PMAX : 1];
    __shared__ uint32_t s_wsum[NT / 64];

    const uint32_t nslow = *a.slow_count;
    if (blockIdx.x >= nslow) return;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const uint32_t P = a.P, L = a.L;
    for (uint32_t r = tid; r < P; r += NT)
        if (QUANT) s_unit[r] = level_unit(*a.tab[r].qscale, a.qbits);
    for (uint32_t i = tid; i < P * (L + 1); i += NT) s_E[i] = 0;

    for (uint32_t k = blockIdx.x; k < nslow; k += gridDim.x) {
        const uint32_t tile = a.slow_list[k];
        const uint32_t tlo = tile * a.T;
        const uint32_t thi = (uint32_t)min((uint64_t)tlo + a.T, (uint64_t)a.N);
        __syncthreads();
        for (uint32_t r = tid; r < P; r += NT)
            s_lo[r] = lower_bound(a.tab[r].idx, 0u, (uint32_t)a.tab[r].nnz, tlo);
        uint32_t tile_nz = 0;
        for (uint64_t sub = tlo; sub < thi; sub += TS) {
            const uint32_t sub_hi = (uint32_t)min(sub + TS, (uint64_t)thi);
            const uint32_t width = sub_hi - (uint32_t)sub;
            __syncthreads();
            for (uint32_t j = tid; j < TS; j += NT) {
                s_last[j] = -1;
                s_pend[j] = 0;
            }
            for (uint32_t r = tid; r < P; r += NT)
                s_hi[r] = lower_bound(a.tab[r].idx, s_lo[r], (uint32_t)a.tab[r].nnz, sub_hi);
            __syncthreads();
            for (uint32_t r = 0; r < P; ++r) {
                const uint32_t lo = s_lo[r], hi = s_hi[r];
                if (lo == hi) continue;
                const StreamDesc* d = &a.tab[r];
                g_u32* gidx = (g_u32*)d->idx;
                g_f32* gval = (g_f32*)d->val;
                g_u8* gq = (g_u8*)d->qval;
                for (uint32_t i = lo + tid; i < hi; i += NT) {
                    const uint32_t j = gidx[i] - (uint32_t)sub;
                    if (j >= width) continue;
                    float v;
                    if (QUANT) {
                        const uint32_t plog = a.qbits == 8u ? 0u : (a.qbits == 4u ? 1u : 2u);
                        const uint32_t byte = gq[i >> plog];
                        const uint32_t code = (byte >> ((i & ((1u << plog) - 1u)) * a.qbits)) & ((1u << a.qbits) - 1u);
                        v = dequant(code, a.qbits, s_unit[r]);
                    } else {
                        v = gval[i];
                    }
                    const int last = s_last[j];
                    if (last >= 0) {
                        const uint32_t sep = 31u - (uint32_t)__clz(r ^ (uint32_t)last);
                        float cur = s_curv[j];
                        uint32_t pend = s_pend[j];
#pragma unroll
                        for (int l = 0; l < LMAX; ++l)
                            if ((uint32_t)l < sep && ((pend >> l) & 1u)) cur = s_slot[l][j] + cur;
                        pend = (pend & ~((1u << sep) - 1u)) | (1u << sep);
                        s_slot[sep][j] = cur;
                        s_pend[j] = (uint16_t)pend;
                        if (MODE != kSparseWrite) atomicAdd(&s_E[r * (L + 1) + sep], 1u);
                    }
                    s_curv[j] = v;
                    s_last[j] = (int16_t)r;
                }
                if (MODE != kSparseWrite && tid == 0) s_E[r * (L + 1) + L] += hi - lo;
                __syncthreads();
            }
            __syncthreads();
            for (uint32_t r = tid; r < P; r += NT) s_lo[r] = s_hi[r];

            // Finalize 4 consecutive coordinates per thread.
            float vals[4];
            uint32_t nzbits = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t j = tid * 4 + q;
                vals[q] = 0.0f;
                if (j < width && s_last[j] >= 0) {
                    float cur = s_curv[j];
                    const uint32_t pend = s_pend[j];
#pragma unroll
                    for (int l = 0; l < LMAX; ++l)
                        if ((pend >> l) & 1u) cur = s_slot[l][j] + cur;
                    vals[q] = cur;
                    nzbits |= 1u << q;
                }
            }
            const uint32_t c = (uint32_t)__popc(nzbits);
            uint32_t incl = c;
#pragma unroll
            for (int o = 1; o < 64; o <<= 1) {
                const uint32_t y = __shfl_up(incl, o);
                if (lane >= o) incl += y;
            }
            if (lane == 63) s_wsum[wv] = incl;
            __syncthreads();
            uint32_t excl = incl - c, total = 0;
            for (int w = 0; w < NT / 64; ++w) {
                const uint32_t v = s_wsum[w];
                if (w < wv) excl += v;
                total += v;
            }
            if (MODE == kDense) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const uint32_t j = tid * 4 + q;
                    if (j < width) a.out_val[sub + j] = ((nzbits >> q) & 1u) ? vals[q] + 0.0f : 0.0f;
                }
            } else if (MODE == kSparseWrite) {
                uint32_t o = a.tile_off[tile] + tile_nz + excl;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if ((nzbits >> q) & 1u) {
                        a.out_idx[o] = (uint32_t)sub + tid * 4 + q;
                        a.out_val[o] = vals[q];
                        ++o;
                    }
                }
            }
            tile_nz += total;
        }
        if (MODE != kSparseWrite && tid == 0) a.tile_cnt[tile] = tile_nz;
    }
    __syncthreads();
    if (MODE != kSparseWrite) flush_counts<NT>(s_E, a);
}

// ------------------------------------------------------------------------
// Per-chunk start offsets of every stream (binary search) and zeroing of the
// counters the passes accumulate into.
__global__ void k_partition(const StreamDesc* tab, uint32_t* off, uint32_t P, uint32_t nchunks,
                            uint64_t chunk_coords, uint64_t N, uint32_t* zero, uint32_t nzero)
{
    const uint32_t gid = blockIdx.x * blockDim.x + threadIdx.x;
    if (gid < nzero) zero[gid] = 0u;
    const uint32_t stride = nchunks + 1;
    if (gid >= P * stride) return;
    const uint32_t r = gid / stride, c = gid % stride;
    const uint32_t nnz = (uint32_t)tab[r].nnz;
    uint32_t res = nnz;
    if (c < nchunks) res = lower_bound(tab[r].idx, 0u, nnz, min((uint64_t)c * chunk_coords, N));
    off[gid] = res;
}

// Switch rule over the tree (§5.1): node dense iff a child is dense or the
// children's nnz sum exceeds thr; a sparse node's nnz is its union size.
__global__ void k_decide(const StreamDesc* tab, const uint32_t* node_cnt, uint32_t P, uint64_t N,
                         uint64_t thr, uint64_t* node_nnz, uint8_t* node_dense, ReduceResult* hdr)
{
    __shared__ uint64_t s_n[256];
    __shared__ uint8_t s_d[256];
    if (threadIdx.x != 0) return;
    for (uint32_t r = 0; r < P; ++r) {
        s_n[r] = tab[r].nnz;
        s_d[r] = 0;
    }
    uint32_t width = P, node = 0;
    while (width > 1) {
        for (uint32_t g = 0; g < width / 2; ++g) {
            const bool dense = s_d[2 * g] || s_d[2 * g + 1] || (s_n[2 * g] + s_n[2 * g + 1] > thr);
            const uint64_t nnz = dense ? N : (uint64_t)node_cnt[node];
            if (node_nnz) node_nnz[node] = nnz;
            if (node_dense) node_dense[node] = dense ? 1 : 0;
            s_n[g] = nnz;
            s_d[g] = dense ? 1 : 0;
            ++node;
        }
        width /= 2;
    }
    hdr->nnz = s_n[0];
    hdr->dense = s_d[0];
    hdr->pad = 0;
}

// Exclusive scan of the per-tile root union sizes (one workgroup); also
// clears the deferred-tile counter for the write pass.
__global__ void __launch_bounds__(1024) k_scan_tiles(const uint32_t* cnt, uint32_t* off, uint32_t n,
                                                     uint32_t* slow_count)
{
    __shared__ uint32_t s_wsum[16];
    const uint32_t tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    const uint32_t per = (n + 1023) / 1024;
    const uint32_t lo = min(tid * per, n), hi = min(lo + per, n);
    uint32_t acc = 0;
    for (uint32_t i = lo; i < hi; ++i) acc += cnt[i];
    uint32_t incl = acc;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o);
        if (lane >= (uint32_t)o) incl += y;
    }
    if (lane == 63) s_wsum[wv] = incl;
    __syncthreads();
    uint32_t run = incl - acc;
    for (uint32_t w = 0; w < wv; ++w) run += s_wsum[w];
    for (uint32_t i = lo; i < hi; ++i) {
        off[i] = run;
        run += cnt[i];
    }
    if (tid == 0) *slow_count = 0u;
}

template <int MW, int MODE>
hipError_t launch_tiles_q(const Args& a, bool quant, hipStream_t s)
{
    const dim3 grid(a.nchunks), block(256);
    const int slot = MODE == kSparseWrite ? kTReduceWrite : kTReducePass;
    timer_begin(slot, s);
    if (quant) hipLaunchKernelGGL((k_tiles<MW, MODE, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_tiles<MW, MODE, false>), grid, block, 0, s, a);
    timer_end(slot, s);
    const uint32_t sg = std::min<uint32_t>(a.ntiles, 256u);
    if (MODE != kSparseWrite) timer_begin(kTReduceSlow, s);
    if (quant) hipLaunchKernelGGL((k_slow<MW, MODE, true>), dim3(sg), dim3(kSlowNT), 0, s, a);
    else hipLaunchKernelGGL((k_slow<MW, MODE, false>), dim3(sg), dim3(kSlowNT), 0, s, a);
    if (MODE != kSparseWrite) timer_end(kTReduceSlow, s);
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_pass(const Args& a, uint32_t MW, bool quant, hipStream_t s)
{
    switch (MW) {
    case 1: return launch_tiles_q<1, MODE>(a, quant, s);
    case 2: return launch_tiles_q<2, MODE>(a, quant, s);
    case 4: return launch_tiles_q<4, MODE>(a, quant, s);
    default: return launch_tiles_q<8, MODE>(a, quant, s);
    }
}

struct Layout {
    StreamDesc* tab;
    uint32_t *off, *zero, *node_cnt, *slow_count, *tile_cnt, *tile_off, *slow_list;
    ReduceResult* hdr;
    size_t bytes;
};

Layout layout(const ReducePlan& p, void* ws)
{
    Carve c(ws);
    Layout l;
    l.tab = c.take<StreamDesc>(p.P);
    l.off = c.take<uint32_t>((size_t)p.P * (p.nchunks + 1));
    l.zero = c.take<uint32_t>((size_t)p.P + 1);
    l.node_cnt = l.zero;
    l.slow_count = l.zero ? l.zero + p.P : nullptr;
    l.tile_cnt = c.take<uint32_t>(p.ntiles);
    l.tile_off = c.take<uint32_t>(p.ntiles);
    l.slow_list = c.take<uint32_t>(p.ntiles);
    l.hdr = c.take<ReduceResult>(1);
    l.bytes = align_up(c.used, 256);
    return l;
}

}  // namespace

int reduce_plan(int P, uint64_t N, uint64_t max_nnz, uint64_t sum_nnz, double delta, int qbits,
                ReducePlan* plan)
{
    ReducePlan p{};
    p.P = (uint32_t)P;
    p.L = 0;
    while ((1u << p.L) < p.P) ++p.L;
    p.MW = p.P <= 32 ? 1u : p.P / 32u;
    const uint64_t NT = 256, TMAX = 4096 / p.MW, CAP = 2048;
    // Tile size: the largest power of two (256 .. TMAX) for which a tile
    // holds on average at most 70% of CAP entries and a rank at most half of
    // its 32-entry window, so that the slow pass stays rare.
    uint64_t T = NT;
    const double want_total = sum_nnz ? 0.7 * (double)CAP * (double)N / (double)sum_nnz : 1e30;
    const double want_rank = max_nnz ? 16.0 * (double)N / (double)max_nnz : 1e30;
    while (T * 2 <= TMAX && (double)(T * 2) <= want_total && (double)(T * 2) <= want_rank) T *= 2;
    uint64_t Np2 = NT;
    while (Np2 < N) Np2 *= 2;
    if (T > Np2) T = Np2;
    p.T = (uint32_t)T;
    p.N = N;
    p.ntiles = (uint32_t)((N + T - 1) / T);
    uint32_t nch = std::min<uint32_t>(p.ntiles, 768u);
    p.tiles_per_chunk = (p.ntiles + nch - 1) / nch;
    p.nchunks = (p.ntiles + p.tiles_per_chunk - 1) / p.tiles_per_chunk;
    const double t = std::floor(delta * (double)N);
    p.thr = t >= 18446744073709551615.0 ? UINT64_MAX : (uint64_t)t;
    p.sum_nnz = sum_nnz;
    p.qbits = (uint32_t)qbits;
    p.speculate_dense = sum_nnz > p.thr ? 1 : 0;
    *plan = p;
    return 0;
}

size_t reduce_workspace(const ReducePlan& p) { return layout(p, nullptr).bytes; }

hipError_t reduce_run(const ReducePlan& p, const StreamDesc* host_tab, uint32_t* out_idx,
                      float* out_val, uint64_t* node_nnz, uint8_t* node_dense, void* ws,
                      hipStream_t s, ReduceResult* res)
{
    const Layout l = layout(p, ws);
    hipError_t e = upload(l.tab, host_tab, sizeof(StreamDesc) * p.P, s);
    if (e != hipSuccess) return e;

    const uint32_t nthreads = std::max<uint32_t>(p.P * (p.nchunks + 1), p.P + 1);
    hipLaunchKernelGGL(k_partition, dim3((nthreads + 255) / 256), dim3(256), 0, s, l.tab, l.off,
                       p.P, p.nchunks, (uint64_t)p.tiles_per_chunk * p.T, p.N, l.zero, p.P + 1);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    Args a{};
    a.tab = l.tab;
    a.off = l.off;
    a.tile_cnt = l.tile_cnt;
    a.tile_off = l.tile_off;
    a.slow_list = l.slow_list;
    a.slow_count = l.slow_count;
    a.node_cnt = l.node_cnt;
    a.out_idx = out_idx;
    a.out_val = out_val;
    a.P = p.P;
    a.L = p.L;
    a.N = (uint32_t)p.N;
    a.T = p.T;
    a.ntiles = p.ntiles;
    a.nchunks = p.nchunks;
    a.tpc = p.tiles_per_chunk;
    a.qbits = p.qbits;
    const bool quant = p.qbits != 0;

    e = p.speculate_dense ? launch_pass<kDense>(a, p.MW, quant, s)
                          : launch_pass<kCount>(a, p.MW, quant, s);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_decide, dim3(1), dim3(64), 0, s, l.tab, l.node_cnt, p.P, p.N, p.thr,
                       node_nnz, node_dense, l.hdr);
    if ((e = hipGetLastError()) != hipSuccess) return e;

    if (p.speculate_dense) {
        if ((e = hipMemcpyAsync(res, l.hdr, sizeof(ReduceResult), hipMemcpyDeviceToHost, s)) !=
            hipSuccess)
            return e;
        if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
        if (res->dense) return hipSuccess;
    }
    // Sparse root: positions from the per-tile union sizes, then write.
    hipLaunchKernelGGL(k_scan_tiles, dim3(1), dim3(1024), 0, s, l.tile_cnt, l.tile_off, p.ntiles,
                       l.slow_count);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if ((e = launch_pass<kSparseWrite>(a, p.MW, quant, s)) != hipSuccess) return e;
    if ((e = hipMemcpyAsync(res, l.hdr, sizeof(ReduceResult), hipMemcpyDeviceToHost, s)) !=
        hipSuccess)
        return e;
    return hipStreamSynchronize(s);
}

}  // namespace sparcml
