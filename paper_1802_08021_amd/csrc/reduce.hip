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
#include <cmath>

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
    static constexpr int TMAX = MW <= 2 ? 2048 : 4096 / MW;
    static constexpr int LMAX = MW == 1 ? 5 : (MW == 2 ? 6 : (MW == 4 ? 7 : 8));
    static constexpr int PMAX = 32 * MW;
    static constexpr int SLOTS = PMAX / 2 / NW;  // rank pairs per wave
    // per tile: values past the second of an index, and rank-ordered values
    // of indices with five or more ranks
    static constexpr uint32_t OVCAP = TMAX / 2, BINCAP = TMAX / 2;
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
//   1  insertion -- each wave holds a 32-entry window of two ranks per 64-lane
//      register (prefetched during the previous tile); every entry inside
//      the tile sets its rank bit in the index's mask and takes an arrival
//      number; the first two values of an index go to a pair slot, later
//      ones to an overflow chain.  All atomics of all windows are issued
//      before any result is used (lanes outside the tile hit per-lane dummy
//      words), so their latencies overlap;
//   2  per index (thread t owns indices q*NT + t): with at most two ranks the
//      sum needs no ordering (v0 + v1 is commutative) and is written here;
//   3  three or four ranks: values sorted by rank in registers and summed
//      with the tree's association, which for a sorted run of ranks is
//      decided by the separators (highest differing bit of neighbours): the
//      largest separator is the top split;
//   4  five or more ranks: values placed in rank order (popcount of the lower
//      rank bits) and summed by a stack keyed by separator level.
// Union sizes of the tree nodes are counted on the side: an entry whose
// predecessor (next lower rank present at the index) first differs from it
// at bit h opens a group at levels 1..h; one without predecessor opens a
// group at every level.  Tiles whose overflow values or rank-ordered values
// would not fit go to the slow pass.
template <int MW, int MODE, bool QUANT>
__global__ void __launch_bounds__(256) k_tiles(Args a)
{
    using S = Shape<MW>;
    constexpr int NT = S::NT, NW = S::NW, TMAX = S::TMAX, LMAX = S::LMAX, PMAX = S::PMAX;
    constexpr int SLOTS = S::SLOTS, CPTMAX = TMAX / NT;
    constexpr uint32_t OVCAP = S::OVCAP, BINCAP = S::BINCAP;
    constexpr uint32_t kNone = 0xFFFFu;
    __shared__ uint4 s_mask4[(TMAX + 64) * MW / 4];  // + one dummy index per lane
    __shared__ uint32_t s_cnt[TMAX + 64];  // arrivals (low 16 bits); sparse position (high)
    __shared__ float2 s_pv[TMAX];          // first two values
    __shared__ uint32_t s_pr[TMAX];        // their ranks: r0 | r1 << 8
    __shared__ uint32_t s_head[TMAX];      // overflow chain head
    __shared__ uint2 s_ov[OVCAP];          // {value bits, rank | next << 16}
    __shared__ float s_bins[MODE == kCount ? 1 : BINCAP];
    __shared__ uint32_t s_list[TMAX];      // [0, nA): 3-4 ranks; from the top: 5+ ranks
    __shared__ uint32_t s_E[MODE == kSparseWrite ? 1 : PMAX * (LMAX + 1)];
    __shared__ uint32_t s_rcnt[PMAX];
    __shared__ uint32_t s_cur[PMAX], s_end[PMAX], s_last[PMAX];
    __shared__ g_u32* s_ip[PMAX];
    __shared__ g_u32* s_vp[PMAX];
    __shared__ float s_unit[QUANT ? PMAX : 1];
    __shared__ uint32_t s_wsum[CPTMAX * NW];
    __shared__ uint32_t s_ovn, s_bsum, s_nA, s_nB, s_binn;
    uint32_t* s_mask = reinterpret_cast<uint32_t*>(s_mask4);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t half = (uint32_t)lane >> 5, sl = (uint32_t)lane & 31u;
    const uint32_t P = a.P, L = a.L, T = a.T, CPT = T / NT, W = L + 1;
    const uint32_t chunk = blockIdx.x, stride = a.nchunks + 1;
    const uint32_t t0 = chunk * a.tpc, t1 = min(t0 + a.tpc, a.ntiles);
    const uint32_t plog = a.qbits == 8u ? 0u : (a.qbits == 4u ? 1u : 2u);
    const uint32_t cmask = QUANT ? (1u << a.qbits) - 1u : 0u;
    const uint64_t ltmask = (1ull << lane) - 1ull;

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
    __syncthreads();

    // Window of rank r (this lane's half) starting at stream position `pos`;
    // positions at or past `end` read as index 0xFFFFFFFF (in no tile).
    auto load_window = [&](uint32_t r, uint32_t pos, uint32_t end, uint32_t& x, uint32_t& v) {
        const uint32_t i = pos + sl;
        const uint32_t ic = min(i, s_last[r]);
        const uint32_t xi = s_ip[r][ic];
        if (QUANT) {
            const uint32_t byte = ((g_u8*)s_vp[r])[ic >> plog];
            v = (byte >> ((ic & ((1u << plog) - 1u)) * a.qbits)) & cmask;
        } else {
            v = s_vp[r][ic];
        }
        x = i < end ? xi : 0xFFFFFFFFu;
    };
    auto value_of = [&](uint32_t vbits, uint32_t r) -> float {
        return QUANT ? dequant(vbits, a.qbits, s_unit[r]) : __uint_as_float(vbits);
    };

    uint32_t xs[SLOTS], vs[SLOTS];
#pragma unroll
    for (int q = 0; q < SLOTS; ++q) {
        const uint32_t r = 2 * (uint32_t)(wv * SLOTS + q) + half;
        const uint32_t rr = min(r, P - 1);
        load_window(rr, s_cur[rr], r < P ? s_end[rr] : 0u, xs[q], vs[q]);
    }

    for (uint32_t tile = t0; tile < t1; ++tile) {
        const uint32_t tlo = tile * T;
        const uint32_t thi = (uint32_t)min((uint64_t)tlo + T, (uint64_t)a.N);

        // Reset this thread's indices and the tile counters once every reader
        // of the previous tile is done.
        __syncthreads();
        for (uint32_t k = 0; k < CPT; ++k) {
            const uint32_t j = k * NT + tid;
            clear_mask<MW>(s_mask, j);
            s_cnt[j] = 0u;
            s_pr[j] = 0u;
            s_head[j] = kNone;
        }
        if (tid == 0) {
            s_ovn = 0;
            s_bsum = 0;
            s_nA = 0;
            s_nB = 0;
            s_binn = 0;
        }
        __syncthreads();

        // 1: insertion.  Sweep A issues every atomic; sweep B stores values.
        uint32_t arr[SLOTS], inb = 0;
#pragma unroll
        for (int q = 0; q < SLOTS; ++q) {
            const uint32_t u = (uint32_t)(wv * SLOTS + q);
            const uint32_t r = 2 * u + half;
            const bool in = 2 * u < P && xs[q] >= tlo && xs[q] < thi;
            const uint32_t j = in ? xs[q] - tlo : (uint32_t)TMAX + (uint32_t)lane;
            atomicOr(&s_mask[j * MW + (r >> 5)], 1u << (r & 31u));
            arr[q] = atomicAdd(&s_cnt[j], 1u);
            inb |= (uint32_t)in << q;
        }
        auto store_value = [&](uint32_t j, uint32_t r, uint32_t k, float v) {
            if (k < 2u) {
                if (k == 0u) s_pv[j].x = v;
                else s_pv[j].y = v;
                atomicOr(&s_pr[j], r << (8u * k));
            } else {
                const uint32_t o = atomicAdd(&s_ovn, 1u);
                if (o < OVCAP) {
                    const uint32_t prev = atomicExch(&s_head[j], o);
                    s_ov[o] = make_uint2(__float_as_uint(v), r | (prev << 16));
                }
            }
        };
#pragma unroll
        for (int q = 0; q < SLOTS; ++q) {
            if ((inb >> q) & 1u) {
                const uint32_t r = 2 * (uint32_t)(wv * SLOTS + q) + half;
                store_value(xs[q] - tlo, r, arr[q], value_of(vs[q], r));
            }
        }
        // Counts, the rare continuation of a window that was entirely inside
        // the tile, and the prefetch of the next tile's windows.
#pragma unroll
        for (int q = 0; q < SLOTS; ++q) {
            const uint32_t u = (uint32_t)(wv * SLOTS + q);
            if (2 * u < P) {
                const uint32_t r = 2 * u + half;
                const uint64_t bal = __ballot((inb >> q) & 1u);
                uint32_t n = (uint32_t)__popc((uint32_t)(bal >> (32 * half)));
                const uint32_t end = s_end[r];
                uint32_t pos = s_cur[r];
                bool more = n == kHalf;
                while (__ballot(more)) {
                    uint32_t x = 0xFFFFFFFFu, v = 0u;
                    if (more) load_window(r, pos + n, end, x, v);
                    const bool in = more && x >= tlo && x < thi;
                    if (in) {
                        const uint32_t j = x - tlo;
                        atomicOr(&s_mask[j * MW + (r >> 5)], 1u << (r & 31u));
                        const uint32_t k = atomicAdd(&s_cnt[j], 1u);
                        store_value(j, r, k, value_of(v, r));
                    }
                    const uint64_t b2 = __ballot(in);
                    const uint32_t c = (uint32_t)__popc((uint32_t)(b2 >> (32 * half)));
                    n += c;
                    more = more && c == kHalf;
                }
                pos += n;
                if (sl == 0) {
                    s_cur[r] = pos;
                    s_rcnt[r] = n;
                }
                load_window(r, pos, end, xs[q], vs[q]);
            }
        }
        __syncthreads();
        if (s_ovn > OVCAP) {
            if (tid == 0) {
                const uint32_t k = atomicAdd(a.slow_count, 1u);
                a.slow_list[k] = tile;
            }
            continue;
        }

        // 2a: ranks per index; non-empty indices counted in index order; the
        // 5+ rank indices' value count checked against the bin capacity.
        uint32_t ms[CPTMAX], nzb[CPTMAX];
#pragma unroll
        for (int q = 0; q < CPTMAX; ++q) {
            ms[q] = 0;
            nzb[q] = 0;
            if ((uint32_t)q < CPT) {
                ms[q] = s_cnt[(uint32_t)q * NT + tid] & 0xFFFFu;
                const uint64_t b = __ballot(ms[q] != 0u);
                nzb[q] = (uint32_t)__popcll(b & ltmask);
                if (lane == 0) s_wsum[q * NW + wv] = (uint32_t)__popcll(b);
                if (ms[q] >= 5u) atomicAdd(&s_bsum, ms[q]);
            }
        }
        __syncthreads();
        if (s_bsum > BINCAP) {
            if (tid == 0) {
                const uint32_t k = atomicAdd(a.slow_count, 1u);
                a.slow_list[k] = tile;
            }
            continue;
        }
        if (MODE != kSparseWrite)
            for (uint32_t r = tid; r < P; r += NT) s_E[r * W + L] += s_rcnt[r];
        uint32_t run = 0;
#pragma unroll
        for (int q = 0; q < CPTMAX; ++q) {
            if ((uint32_t)q < CPT) {
                uint32_t before = 0, rtot = 0;
#pragma unroll
                for (int w = 0; w < NW; ++w) {
                    const uint32_t c = s_wsum[q * NW + w];
                    if (w < wv) before += c;
                    rtot += c;
                }
                nzb[q] += run + before;
                run += rtot;
            }
        }
        if (MODE != kSparseWrite && tid == 0) a.tile_cnt[tile] = run;

        // 2b: at most two ranks: finish here; more: to the lists.
        const uint32_t toff = MODE == kSparseWrite ? a.tile_off[tile] : 0u;
#pragma unroll
        for (int q = 0; q < CPTMAX; ++q) {
            if ((uint32_t)q < CPT) {
                const uint32_t j = (uint32_t)q * NT + tid;
                const uint32_t m = ms[q];
                if (m == 2u && MODE != kSparseWrite) {
                    const uint32_t pr = s_pr[j];
                    const uint32_t r0 = pr & 0xFFu, r1 = (pr >> 8) & 0xFFu;
                    atomicAdd(&s_E[max(r0, r1) * W + (31u - (uint32_t)__clz(r0 ^ r1))], 1u);
                }
                if (MODE != kCount) {
                    float sum = 0.0f;
                    if (m != 0u && m <= 2u) {
                        const float2 pv = s_pv[j];
                        sum = m == 1u ? pv.x : pv.x + pv.y;
                    }
                    if (MODE == kDense) {
                        if (m <= 2u && (uint64_t)tlo + j < thi) a.out_val[(uint64_t)tlo + j] = m ? sum + 0.0f : 0.0f;
                    } else if (m != 0u && m <= 2u) {
                        a.out_idx[toff + nzb[q]] = tlo + j;
                        a.out_val[toff + nzb[q]] = sum;
                    }
                }
                const bool la = m == 3u || m == 4u, lb = m >= 5u;
                const uint64_t ba = __ballot(la), bb = __ballot(lb);
                uint32_t pa = 0, pb = 0;
                if (lane == 0) {
                    if (ba) pa = atomicAdd(&s_nA, (uint32_t)__popcll(ba));
                    if (bb) pb = atomicAdd(&s_nB, (uint32_t)__popcll(bb));
                }
                pa = __shfl(pa, 0) + (uint32_t)__popcll(ba & ltmask);
                pb = __shfl(pb, 0) + (uint32_t)__popcll(bb & ltmask);
                const uint32_t item = j | (nzb[q] << 16);
                if (la) s_list[pa] = item;
                if (lb) s_list[(uint32_t)TMAX - 1u - pb] = item;
            }
        }
        __syncthreads();
        const uint32_t nA = s_nA, nB = s_nB;

        // 3: three or four ranks, in registers.
        for (uint32_t wi = tid; wi < nA; wi += NT) {
            const uint32_t item = s_list[wi];
            const uint32_t j = item & 0xFFFFu;
            const uint32_t m = s_cnt[j] & 0xFFFFu;
            const uint32_t pr = s_pr[j];
            uint32_t rk[4];
            float vv[4];
            rk[0] = pr & 0xFFu;
            rk[1] = (pr >> 8) & 0xFFu;
            if (MODE != kCount) {
                const float2 pv = s_pv[j];
                vv[0] = pv.x;
                vv[1] = pv.y;
            } else {
                vv[0] = vv[1] = 0.0f;
            }
            const uint2 o2 = s_ov[s_head[j]];
            rk[2] = o2.y & 0xFFFFu;
            vv[2] = __uint_as_float(o2.x);
            rk[3] = 0x100u;  // sentinel above every rank
            vv[3] = 0.0f;
            if (m == 4u) {
                const uint2 o3 = s_ov[o2.y >> 16];
                rk[3] = o3.y & 0xFFFFu;
                vv[3] = __uint_as_float(o3.x);
            }
            auto cswap = [&](int x, int y) {
                const bool s = rk[x] > rk[y];
                const uint32_t tr = rk[x];
                const float tv = vv[x];
                rk[x] = s ? rk[y] : rk[x];
                rk[y] = s ? tr : rk[y];
                vv[x] = s ? vv[y] : vv[x];
                vv[y] = s ? tv : vv[y];
            };
            cswap(0, 1);
            cswap(2, 3);
            cswap(0, 2);
            cswap(1, 3);
            cswap(1, 2);
            const uint32_t c1 = 31u - (uint32_t)__clz(rk[0] ^ rk[1]);
            const uint32_t c2 = 31u - (uint32_t)__clz(rk[1] ^ rk[2]);
            if (MODE != kSparseWrite) {
                atomicAdd(&s_E[rk[1] * W + c1], 1u);
                atomicAdd(&s_E[rk[2] * W + c2], 1u);
            }
            uint32_t c3 = 0;
            if (m == 4u) {
                c3 = 31u - (uint32_t)__clz(rk[2] ^ rk[3]);
                if (MODE != kSparseWrite) atomicAdd(&s_E[rk[3] * W + c3], 1u);
            }
            if (MODE != kCount) {
                float sum;
                const float t012 = c1 < c2 ? (vv[0] + vv[1]) + vv[2] : vv[0] + (vv[1] + vv[2]);
                if (m == 3u) {
                    sum = t012;
                } else if (c2 > c1 && c2 > c3) {
                    sum = (vv[0] + vv[1]) + (vv[2] + vv[3]);
                } else if (c1 > c3) {
                    sum = vv[0] + (c2 < c3 ? (vv[1] + vv[2]) + vv[3] : vv[1] + (vv[2] + vv[3]));
                } else {
                    sum = t012 + vv[3];
                }
                if (MODE == kDense) {
                    a.out_val[(uint64_t)tlo + j] = sum + 0.0f;
                } else {
                    a.out_idx[toff + (item >> 16)] = tlo + j;
                    a.out_val[toff + (item >> 16)] = sum;
                }
            }
        }

        // 4: five or more ranks: rank-ordered values, stack walk.
        for (uint32_t wi = tid; wi < nB; wi += NT) {
            const uint32_t item = s_list[(uint32_t)TMAX - 1u - wi];
            const uint32_t j = item & 0xFFFFu;
            const uint32_t m = s_cnt[j] & 0xFFFFu;
            uint32_t w[MW];
            load_mask<MW>(s_mask, j, w);
            uint32_t start = 0;
            if (MODE != kCount) {
                start = atomicAdd(&s_binn, m);
                auto place = [&](uint32_t r, float v) {
                    const uint32_t rw = r >> 5, low = (1u << (r & 31u)) - 1u;
                    uint32_t below = 0;
#pragma unroll
                    for (int k = 0; k < MW; ++k)
                        below += (uint32_t)k < rw ? __popc(w[k]) : ((uint32_t)k == rw ? __popc(w[k] & low) : 0u);
                    s_bins[start + below] = v;
                };
                const float2 pv = s_pv[j];
                const uint32_t pr = s_pr[j];
                place(pr & 0xFFu, pv.x);
                place((pr >> 8) & 0xFFu, pv.y);
                for (uint32_t o = s_head[j]; o != kNone;) {
                    const uint2 it = s_ov[o];
                    place(it.y & 0xFFFFu, __uint_as_float(it.x));
                    o = it.y >> 16;
                }
            }
            float slot[LMAX];
#pragma unroll
            for (int l = 0; l < LMAX; ++l) slot[l] = 0.0f;
            float cur = 0.0f;
            uint32_t pend = 0, pos = start;
            int last = -1;
#pragma unroll
            for (int k = 0; k < MW; ++k) {
                uint32_t bits = w[k];
                while (bits) {
                    const int r = k * 32 + (__ffs(bits) - 1);
                    bits &= bits - 1u;
                    if (last >= 0) {
                        const int sep = 31 - (int)__clz((uint32_t)(r ^ last));
                        if (MODE != kSparseWrite) atomicAdd(&s_E[(uint32_t)r * W + (uint32_t)sep], 1u);
                        if (MODE != kCount) {
#pragma unroll
                            for (int l = 0; l < LMAX; ++l)
                                if (l < sep && ((pend >> l) & 1u)) cur = slot[l] + cur;
                            pend = (pend & ~((1u << sep) - 1u)) | (1u << sep);
#pragma unroll
                            for (int l = 0; l < LMAX; ++l)
                                if (l == sep) slot[l] = cur;
                        }
                    }
                    if (MODE != kCount) cur = s_bins[pos++];
                    last = r;
                }
            }
            if (MODE != kCount) {
#pragma unroll
                for (int l = 0; l < LMAX; ++l)
                    if ((pend >> l) & 1u) cur = slot[l] + cur;
                if (MODE == kDense) {
                    a.out_val[(uint64_t)tlo + j] = cur + 0.0f;
                } else {
                    a.out_idx[toff + (item >> 16)] = tlo + j;
                    a.out_val[toff + (item >> 16)] = cur;
                }
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
    const uint64_t NT = 256;
    const uint64_t TMAX = p.MW <= 2 ? 2048 : 4096 / p.MW;
    // Tile size: the largest power of two (256 .. TMAX) for which, with the
    // entries spread uniformly, a rank fills at most half of its 32-entry
    // window and the expected overflow values, worklist indices and
    // rank-ordered values stay under half of their per-tile capacity
    // (Poisson model of the ranks present per index, mean lambda).
    const double lam = (double)sum_nnz / (double)N;
    const double e = std::exp(-lam);
    const double p4 = 1.0 - e * (1.0 + lam + lam * lam / 2 + lam * lam * lam / 6);  // P(m >= 5)
    const double ovf = std::max(0.0, lam - 2.0 + 2.0 * e + lam * e);              // E[(m-2)+]
    const double bins = std::max(0.0, lam - e * lam * (1.0 + lam + lam * lam / 2 + lam * lam * lam / 6));  // E[m; m >= 5]
    // capacities are TMAX/2 values each; aim for a quarter of TMAX in expectation
    const double want_rank = max_nnz ? 16.0 * (double)N / (double)max_nnz : 1e30;
    const double want_ov = ovf > 0 ? 0.25 * (double)TMAX / ovf : 1e30;
    const double want_bins = bins > 0 ? 0.25 * (double)TMAX / bins : 1e30;
    (void)p4;
    const double want = std::min(want_rank, std::min(want_ov, want_bins));
    uint64_t T = NT;
    while (T * 2 <= TMAX && (double)(T * 2) <= want) T *= 2;
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
