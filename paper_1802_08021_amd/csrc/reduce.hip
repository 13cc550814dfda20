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
constexpr uint32_t kCap = 4096;  // entries per tile on the fast path
constexpr uint32_t kWin = 64;    // entries read per rank per tile (one wave)
constexpr int kSlowNT = 256;
constexpr int kSlowTS = 1024;    // coordinates per slow-path sub-tile

template <int MW>
struct Shape;  // MW = 32-bit mask words per coordinate = ceil(P / 32)
template <>
struct Shape<1> { static constexpr int NT = 256, TMAX = 4096, LMAX = 5; };
template <>
struct Shape<2> { static constexpr int NT = 256, TMAX = 4096, LMAX = 6; };
template <>
struct Shape<4> { static constexpr int NT = 256, TMAX = 2048, LMAX = 7; };
template <>
struct Shape<8> { static constexpr int NT = 512, TMAX = 1024, LMAX = 8; };

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

// Turn per-(rank, depth) counts into node union sizes and add them to the
// global counters.  E[r][d] = entries of rank r that open new groups at
// levels 1..d; node (t,g) counts the entries of its ranks with depth >= t.
template <int NT>
__device__ void flush_counts(uint32_t* E, const Args& a)
{
    const uint32_t P = a.P, L = a.L, W = L + 1;
    for (uint32_t r = threadIdx.x; r < P; r += NT) {
        uint32_t acc = 0;
        for (int d = (int)L; d >= 1; --d) {
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
// Fast tile pass.  One workgroup walks a chunk of consecutive tiles; wave w
// owns ranks [w*RPW, (w+1)*RPW) and reads a 64-entry window of each per
// tile.  Tiles where a rank has >= 64 entries or the tile has > kCap entries
// are deferred to the slow pass.
template <int MW, int MODE, bool QUANT>
__global__ void __launch_bounds__(Shape<MW>::NT) k_tiles(Args a)
{
    constexpr int NT = Shape<MW>::NT, NW = NT / 64, TMAX = Shape<MW>::TMAX;
    constexpr int LMAX = Shape<MW>::LMAX, PMAX = 32 * MW, RPW = PMAX / NW;
    __shared__ uint32_t s_mask[TMAX * MW];
    __shared__ float s_vals[MODE == kCount ? 1 : kCap];
    __shared__ uint16_t s_bin[MODE == kCount ? 1 : TMAX];
    __shared__ uint32_t s_E[MODE == kSparseWrite ? 1 : PMAX * (LMAX + 1)];
    __shared__ uint32_t s_cur[PMAX], s_end[PMAX], s_cnt[PMAX];
    __shared__ float s_unit[QUANT ? PMAX : 1];
    __shared__ uint32_t s_wsum[NW];
    __shared__ uint32_t s_total, s_slow;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t P = a.P, L = a.L, T = a.T, CPT = T / NT;
    const uint32_t chunk = blockIdx.x, stride = a.nchunks + 1;
    const uint32_t t0 = chunk * a.tpc, t1 = min(t0 + a.tpc, a.ntiles);

    for (uint32_t r = tid; r < P; r += NT) {
        s_cur[r] = a.off[r * stride + chunk];
        s_end[r] = a.off[r * stride + chunk + 1];
        if (QUANT)
            s_unit[r] = level_unit(*a.tab[r].qscale, a.qbits);
    }
    if (MODE != kSparseWrite)
        for (uint32_t i = tid; i < P * (L + 1); i += NT) s_E[i] = 0;

    for (uint32_t tile = t0; tile < t1; ++tile) {
        const uint32_t tlo = tile * T;
        const uint32_t thi = (uint32_t)min((uint64_t)tlo + T, (uint64_t)a.N);
        __syncthreads();
        for (uint32_t i = tid; i < T * MW / 4; i += NT)
            reinterpret_cast<uint4*>(s_mask)[i] = make_uint4(0u, 0u, 0u, 0u);
        if (tid == 0) {
            s_total = 0;
            s_slow = 0;
        }
        __syncthreads();

        // Phase 1: windows, rank bits, per-rank counts.
        uint32_t xs[RPW], vs[RPW], inmask = 0;
#pragma unroll
        for (int s = 0; s < RPW; ++s) {
            const uint32_t r = wv * RPW + s;
            xs[s] = 0xFFFFFFFFu;
            vs[s] = 0u;
            if (r < P) {
                const uint32_t i = s_cur[r] + lane;
                if (i < s_end[r]) {
                    const StreamDesc* d = &a.tab[r];
                    xs[s] = d->idx[i];
                    vs[s] = QUANT ? load_code(d->qval, i, a.qbits) : __float_as_uint(d->val[i]);
                }
            }
        }
#pragma unroll
        for (int s = 0; s < RPW; ++s) {
            const uint32_t r = wv * RPW + s;
            if (r < P) {
                const bool in = xs[s] >= tlo && xs[s] < thi;
                const uint64_t bal = __ballot(in);
                if (in) {
                    atomicOr(&s_mask[(xs[s] - tlo) * MW + (r >> 5)], 1u << (r & 31u));
                    inmask |= 1u << s;
                }
                if (lane == 0) {
                    const uint32_t c = (uint32_t)__popcll(bal);
                    s_cnt[r] = c;
                    atomicAdd(&s_total, c);
                    if (c == kWin) s_slow = 1u;
                }
            }
        }
        __syncthreads();

        if (s_slow || s_total > kCap) {
            // Defer the tile; move every cursor past it (a rank may hold more
            // than one window's worth of entries here).
            for (int s = 0; s < RPW; ++s) {
                const uint32_t r = wv * RPW + s;
                if (r >= P) break;
                uint32_t n = s_cnt[r];
                if (n == kWin) {
                    const uint32_t* idx = a.tab[r].idx;
                    const uint32_t base = s_cur[r], end = s_end[r];
                    for (;;) {
                        const uint32_t i = base + n + lane;
                        const bool in = i < end && idx[i] < thi;
                        const uint32_t c = (uint32_t)__popcll(__ballot(in));
                        n += c;
                        if (c < kWin) break;
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
        for (uint32_t r = tid; r < P; r += NT) s_cur[r] += s_cnt[r];

        // Phase 2: per-coordinate rank counts; exclusive scan packs
        // (entries below 16 bits, non-empty coordinates above).
        const uint32_t j0 = tid * CPT;
        uint32_t acc = 0;
        for (uint32_t q = 0; q < CPT; ++q) {
            uint32_t m = 0;
#pragma unroll
            for (int w = 0; w < MW; ++w) m += __popc(s_mask[(j0 + q) * MW + w]);
            acc += m | ((m != 0u) << 16);
        }
        uint32_t incl = acc;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const uint32_t y = __shfl_up(incl, o);
            if (lane >= o) incl += y;
        }
        if (lane == 63) s_wsum[wv] = incl;
        __syncthreads();
        uint32_t excl = incl - acc, total = 0;
#pragma unroll
        for (int w = 0; w < NW; ++w) {
            const uint32_t v = s_wsum[w];
            if (w < wv) excl += v;
            total += v;
        }
        if (MODE != kSparseWrite && tid == 0) a.tile_cnt[tile] = total >> 16;
        if (MODE != kCount) {
            uint32_t run = excl;
            for (uint32_t q = 0; q < CPT; ++q) {
                uint32_t m = 0;
#pragma unroll
                for (int w = 0; w < MW; ++w) m += __popc(s_mask[(j0 + q) * MW + w]);
                s_bin[j0 + q] = (uint16_t)(run & 0xFFFFu);
                run += m | ((m != 0u) << 16);
            }
        }
        __syncthreads();

        // Phase 3: place values in rank order; count node memberships.
#pragma unroll
        for (int s = 0; s < RPW; ++s) {
            const uint32_t r = wv * RPW + s;
            if (r < P && ((inmask >> s) & 1u)) {
                const uint32_t j = xs[s] - tlo;
                uint32_t w[MW];
#pragma unroll
                for (int k = 0; k < MW; ++k) w[k] = s_mask[j * MW + k];
                const uint32_t rw = r >> 5, lowbits = (1u << (r & 31u)) - 1u;
                if (MODE != kCount) {
                    uint32_t below = 0;
#pragma unroll
                    for (int k = 0; k < MW; ++k)
                        below += (uint32_t)k < rw ? __popc(w[k])
                                                  : ((uint32_t)k == rw ? __popc(w[k] & lowbits) : 0u);
                    const float v = QUANT ? dequant(vs[s], a.qbits, s_unit[r]) : __uint_as_float(vs[s]);
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
                    const uint32_t depth = prev < 0 ? L : (31u - (uint32_t)__clz(r ^ (uint32_t)prev));
                    if (depth) atomicAdd(&s_E[r * (L + 1) + depth], 1u);
                }
            }
        }
        if (MODE == kCount) continue;
        __syncthreads();

        // Phase 4: tree sum per coordinate, write the tile once.
        uint32_t run = excl;
        for (uint32_t q = 0; q < CPT; ++q) {
            const uint32_t j = j0 + q;
            uint32_t w[MW], m = 0;
#pragma unroll
            for (int k = 0; k < MW; ++k) {
                w[k] = s_mask[j * MW + k];
                m += __popc(w[k]);
            }
            float sum = 0.0f;
            if (m) {
                uint32_t pos = run & 0xFFFFu, pend = 0;
                float slot[LMAX];
#pragma unroll
                for (int l = 0; l < LMAX; ++l) slot[l] = 0.0f;
                float cur = 0.0f;
                int last = -1;
#pragma unroll
                for (int k = 0; k < MW; ++k) {
                    uint32_t bits = w[k];
                    while (bits) {
                        const int r = k * 32 + (__ffs(bits) - 1);
                        bits &= bits - 1u;
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
                    }
                }
#pragma unroll
                for (int l = 0; l < LMAX; ++l)
                    if ((pend >> l) & 1u) cur = slot[l] + cur;
                sum = cur;
            }
            if (MODE == kDense) {
                if ((uint64_t)tlo + j < thi) a.out_val[(uint64_t)tlo + j] = m ? sum + 0.0f : 0.0f;
            } else if (m) {
                const uint32_t o = a.tile_off[tile] + (run >> 16);
                a.out_idx[o] = tlo + j;
                a.out_val[o] = sum;
            }
            run += m | ((m != 0u) << 16);
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
                for (uint32_t i = lo + tid; i < hi; i += NT) {
                    const uint32_t j = d->idx[i] - (uint32_t)sub;
                    if (j >= width) continue;
                    const float v = QUANT ? dequant(load_code(d->qval, i, a.qbits), a.qbits, s_unit[r])
                                          : d->val[i];
                    const int last = s_last[j];
                    uint32_t depth;
                    if (last < 0) {
                        depth = L;
                    } else {
                        const uint32_t sep = 31u - (uint32_t)__clz(r ^ (uint32_t)last);
                        float cur = s_curv[j];
                        uint32_t pend = s_pend[j];
#pragma unroll
                        for (int l = 0; l < LMAX; ++l)
                            if ((uint32_t)l < sep && ((pend >> l) & 1u)) cur = s_slot[l][j] + cur;
                        pend = (pend & ~((1u << sep) - 1u)) | (1u << sep);
                        s_slot[sep][j] = cur;
                        s_pend[j] = (uint16_t)pend;
                        depth = sep;
                    }
                    s_curv[j] = v;
                    s_last[j] = (int16_t)r;
                    if (MODE != kSparseWrite && depth) atomicAdd(&s_E[r * (L + 1) + depth], 1u);
                }
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
    const dim3 grid(a.nchunks), block(Shape<MW>::NT);
    if (quant) hipLaunchKernelGGL((k_tiles<MW, MODE, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_tiles<MW, MODE, false>), grid, block, 0, s, a);
    const uint32_t sg = std::min<uint32_t>(a.ntiles, 256u);
    if (quant) hipLaunchKernelGGL((k_slow<MW, MODE, true>), dim3(sg), dim3(kSlowNT), 0, s, a);
    else hipLaunchKernelGGL((k_slow<MW, MODE, false>), dim3(sg), dim3(kSlowNT), 0, s, a);
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
    const uint32_t NT = p.MW == 8 ? 512u : 256u;
    const uint32_t TMAX = p.MW == 1 ? 4096u : (p.MW == 2 ? 4096u : (p.MW == 4 ? 2048u : 1024u));
    // Aim for about 32 entries per rank per tile (half a window) so that a
    // rank rarely fills its 64-entry window.
    uint64_t T = TMAX;
    if (max_nnz > 0) {
        const uint64_t want = (32u * N) / max_nnz;
        uint64_t t = NT;
        while (t * 2 <= want && t * 2 <= TMAX) t *= 2;
        T = t;
    }
    uint64_t Np2 = NT;
    while (Np2 < N) Np2 *= 2;
    if (T > Np2) T = Np2;
    p.T = (uint32_t)T;
    p.N = N;
    p.ntiles = (uint32_t)((N + T - 1) / T);
    uint32_t nch = std::min<uint32_t>(p.ntiles, 512u);
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
