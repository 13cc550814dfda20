// Sparse allreduce of P sparse streams on one gfx950 GPU: the local
// reduction work of SparCML's recursive-doubling sparse allreduce (§5.3.1,
// Fig. 2) with the sparse->dense switch of §5.1.
//
// Design (why it differs from a level-by-level merge): every rank's stream
// lives in HBM, so instead of materialising the P-1 intermediate streams of
// the tree (which moves log2(P) times the data), the coordinate space is cut
// into tiles of T indices and each tile evaluates the whole tree at once:
//
//  * every entry of the tile takes an arrival number at its coordinate (an
//    LDS atomic on a word that also sums the arrived ranks); the first
//    arrival leaves its value there;
//  * the later arrivals are summed with the exact association of the tree:
//    two ranks first meet at the level given by the highest differing bit of
//    their numbers (their separator), and the root of any subset of ranks
//    splits at the largest separator between rank-order neighbours -- so two
//    ranks need one addition, three or four a closed form of the separators,
//    five a sorting network, and more a walk that reduces the tree level by
//    level across the lanes of a row;
//  * the exact union size of every tree node -- what the switch rule needs --
//    is counted on the side: the entry of rank r whose predecessor (next
//    lower present rank) differs from r first at bit h opens a new group at
//    levels 1..h (all levels if it has no predecessor);
//  * a dense node's value at an index equals the tree sum (+0.0 where no rank
//    contributes), so a dense root is written tile by tile, once.
//
// Passes: partition (per-chunk stream offsets) -> tile pass (COUNT, or DENSE
// when the root is likely dense) -> slow pass for tiles that overflow the
// fast path's LDS budget -> decide (switch rule over the node counts) and,
// in the same launch, the scan of per-tile union sizes -> [SPARSE_WRITE tile
// and slow passes].
#include "internal.h"

#include <atomic>
#include "qsgd_device.h"

#include <algorithm>
#include <cmath>
#include <cstddef>
#include <cstring>

namespace sparcml {
namespace {

enum Mode { kCount = 0, kDense = 1, kSparseWrite = 2 };

// Pointers that live in memory are generic unless marked: generic (FLAT)
// loads also count against the LDS wait counter and would serialize LDS
// work behind every HBM access.  The descriptor table is read through the
// constant address space so that its uniform loads become scalar loads.
typedef const uint32_t __attribute__((address_space(1))) g_u32;
typedef const uint8_t __attribute__((address_space(1))) g_u8;
typedef const float __attribute__((address_space(1))) g_f32;
typedef const StreamDesc __attribute__((address_space(4)))* c_desc;

constexpr int kSlowNT = 256;
constexpr int kSlowTS = 1024;  // coordinates per slow-path sub-tile

// Tree levels for up to 32*MW ranks (slow pass).
template <int MW>
struct SlowShape {
    static constexpr int PMAX = 32 * MW;
    static constexpr int LMAX = MW == 1 ? 5 : (MW == 2 ? 6 : (MW == 4 ? 7 : 8));
};

// Fast tile pass for up to PMAX ranks.  A wave owns SLMAX ranks ("slots");
// per tile it reads a 64-entry window of each slot's stream (one entry per
// lane) and compacts the entries inside the tile into its own region of at
// most ECAP entries.  TMAX coordinates per tile; CAP staged entries (those
// of indices held by three or more ranks).  Above 32 ranks a 1024-thread
// workgroup holds about 147 KB of LDS, so one runs per CU (four waves per
// SIMD); up to 32 ranks 512 threads and half the tile.
template <int PMAX>
struct Fast {
    static constexpr int NT = PMAX <= 32 ? 512 : 1024;
    static constexpr int WPE = 4;                   // waves per SIMD (LDS and registers)
    static constexpr int NW = NT / 64;
    static constexpr int SLMAX = PMAX / NW < 1 ? 1 : PMAX / NW;
    static constexpr int TMAX = PMAX <= 32 ? 2048 : 4096;
    static constexpr int CPT = TMAX / NT;           // coordinates per thread (4)
    static constexpr uint32_t CAP = TMAX * 3 / 4;   // staged later arrivals
    static constexpr uint32_t CWC = 128;            // indices with three or more ranks per wave
    static constexpr uint32_t CCAP = NW * CWC;
    static constexpr uint32_t ECAP = PMAX >= 256 ? 384 : 448;  // compacted entries per wave
    static constexpr int LMAX = PMAX <= 16 ? 4 : (PMAX <= 32 ? 5 : (PMAX <= 64 ? 6 : (PMAX <= 128 ? 7 : 8)));
};
constexpr uint32_t kWin = 64;  // window entries per rank per tile

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
    uint32_t out_vec;          // out_val is 16-byte aligned
    uint32_t lo;               // first index of the range [lo, lo + N); dense output is relative
    const ReduceResult* skip;  // sparse-output passes: return at once if skip->dense (NULL: never)
    uint32_t out_cap;          // entries out_idx holds: the sparse-output passes write no further
    uint32_t* err_hdr;         // error bits of the root header (bit 1: a result past out_cap) ...
    uint32_t* err_res;         // ... and of the caller's device header (NULL: none)
};

// One entry of a sparse root at position o.  Positions come from per-tile
// union sizes that the count pass and this pass take alike, so for streams
// that ascend o < root nnz <= out_cap; streams that do not can make them
// disagree, and such entries are dropped and reported (bit 1 of the header)
// instead of written past the caller's buffer.
__device__ __forceinline__ void put_sparse(const Args& a, uint32_t o, uint32_t index, float v)
{
    if (o < a.out_cap) {
        a.out_idx[o] = index;
        a.out_val[o] = v;
    } else {
        atomicOr(a.err_hdr, 2u);
        if (a.err_res) atomicOr(a.err_res, 2u);
    }
}

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

// Turn per-rank counts into node union sizes and add them to the global
// counters.  E[r][d], d < L: entries of rank r whose predecessor (next lower
// rank present at the same index) first differs from r at bit d -- such an
// entry opens a new group at levels 1..d; E[r][L]: all entries of rank r,
// of which those without predecessor open new groups at every level.
// Node (t, g) counts the entries of its ranks that open a group at level t.
template <int NT, int RS>
__device__ void flush_counts(uint32_t* E, const Args& a)
{
    const uint32_t P = a.P, L = a.L, W = L + 1;
    // E[r][d] lives at d * RS + r (rank-contiguous rows) or r * W + d.
    auto at = [&](uint32_t r, uint32_t d) -> uint32_t { return RS ? d * RS + r : r * W + d; };
    for (uint32_t r = threadIdx.x; r < P; r += NT) {
        uint32_t acc = E[at(r, L)];
        for (uint32_t d = 0; d < L; ++d) acc -= E[at(r, d)];
        E[at(r, L)] = acc;
        for (int d = (int)L - 1; d >= 1; --d) {
            acc += E[at(r, (uint32_t)d)];
            E[at(r, (uint32_t)d)] = acc;
        }
    }
    __syncthreads();
    for (uint32_t node = threadIdx.x; node + 1 < P; node += NT) {
        uint32_t t, g;
        node_coords(node, P, &t, &g);
        uint32_t sum = 0;
        for (uint32_t r = g << t; r < ((g + 1) << t); ++r) sum += E[at(r, t)];
        if (sum) atomicAdd(&a.node_cnt[node], sum);
    }
}

// Masks of the active lanes where a == b, a < b (unsigned): one compare each.
__device__ __forceinline__ uint64_t lanes_eq(uint32_t a, uint32_t b)
{
    return __builtin_amdgcn_uicmp(a, b, 32);  // ICMP_EQ
}
__device__ __forceinline__ uint64_t lanes_lt(uint32_t a, uint32_t b)
{
    return __builtin_amdgcn_uicmp(a, b, 36);  // ICMP_ULT
}

// base + the number of lanes below this one set in m.
__device__ __forceinline__ uint32_t below_count(uint64_t m, uint32_t base)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, base));
}

// A tree node: the sum of its two children when both hold a value, else the
// one that does (px, py: whether x, y hold one).
__device__ __forceinline__ float tree_join(float x, uint32_t px, float y, uint32_t py)
{
    return px && py ? x + y : (px ? x : y);
}

// One level of a tree over the lanes of rows of 16: lane i (a multiple of
// 2H) joins lane i + H (DPP row_shl:H).  All lanes must be active.
template <int H>
__device__ __forceinline__ void tree_level(float& v, uint32_t& pr, uint32_t lane)
{
    const float ov = __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x100 + H, 0xF, 0xF, true));
    const uint32_t op = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)pr, 0x100 + H, 0xF, 0xF, true);
    const bool at = (lane & (2u * H - 1u)) == 0u;
    v = at ? tree_join(v, pr, ov, op) : v;
    pr = at ? (pr | op) : pr;
}

// Tree sums of three and four values in rank order, given the separator
// levels between neighbours (distinct within the run): the root splits at the
// largest separator.
__device__ __forceinline__ float tree3(float a, float b, float c, uint32_t x, uint32_t y)
{
    return x < y ? (a + b) + c : a + (b + c);
}
__device__ __forceinline__ float tree4(float a, float b, float c, float d, uint32_t x, uint32_t y, uint32_t z)
{
    if (y > x && y > z) return (a + b) + (c + d);
    return x > z ? a + tree3(b, c, d, y, z) : tree3(a, b, c, x, y) + d;
}

// Level at which ranks a != b first meet: their highest differing bit
// (the | 1 keeps equal ranks, which valid streams never produce, in range).
__device__ __forceinline__ uint32_t sep_level(uint32_t a, uint32_t b)
{
    return 31u - (uint32_t)__clz((a ^ b) | 1u);
}

// ------------------------------------------------------------------------
// Fast tile pass.  One workgroup walks a chunk of consecutive tiles of T
// coordinates; per tile:
//   P1  every window entry inside the tile takes an arrival number at its
//       coordinate (LDS atomic); the first arrival leaves its rank and
//       value there.  A window that lies entirely inside the tile is
//       continued (rare) into the side buffer.  The next tile's windows are
//       then requested, so their loads overlap the rest of this tile.
//   scan  per coordinate: m ranks; coordinates with m >= 3 get a staging
//       range and a list slot (m = 3..4 and m >= 5 apart); non-empty ones
//       their output position (sparse output).
//   P2  m = 1: done (the first value stands); m = 2: the second arrival adds
//       its value to the first -- a single addition is the same in either
//       order -- and counts its pair for the node sizes; m >= 3: the entry
//       is staged at its coordinate's range.
//   walk  m = 3..4: ranks sorted in registers, sum with the association the
//       separators dictate; m >= 5: staged entries put in rank order, then a
//       stack keyed by separator level adds them in tree order.
//   store (dense result) the tile leaves LDS in 16-byte stores.
// Union sizes of the tree nodes are counted on the side (flush_counts).
// Tiles whose staged entries, side entries or total entries exceed the LDS
// budget are deferred to the slow pass.
template <int PMAX, int MODE, bool QUANT>
__global__ void __launch_bounds__(Fast<PMAX>::NT, Fast<PMAX>::WPE) k_tiles(Args a)
{
    using F = Fast<PMAX>;
    constexpr int NT = F::NT, NW = F::NW, SLMAX = F::SLMAX, TMAX = F::TMAX, CPT = F::CPT;
    constexpr uint32_t CAP = F::CAP, ECAP = F::ECAP, ERGN = ECAP + 64, CWC = F::CWC, CCAP = F::CCAP;
    constexpr int LMAX = F::LMAX;
    constexpr bool VALS = MODE != kCount, CNTS = MODE != kSparseWrite;
    constexpr uint32_t EW = PMAX * (LMAX + 1);  // node-count words; 64 dummies follow
    constexpr int PW = (PMAX + 31) / 32;        // rank-mask words
    constexpr uint32_t RROWS = PMAX >= 256 ? 2u : 4u;  // indices per wave in the row walk
    constexpr uint32_t RK = PMAX / 16;                  // ranks per lane in the row walk
    if (MODE == kSparseWrite && a.skip && a.skip->dense) return;  // the root is dense: nothing to write
    static_assert(NW * RROWS * (PMAX + PW) <= 2 * NW * (int)ERGN, "walk buffers alias the entry regions");

    // Per index: arrivals | (sum of the arrived ranks) << 16 -- the second
    // arrival reads the first one's rank there -- then m | aux << 9 with aux
    // the staging start of an index with three or more ranks (sparse output:
    // the output position of every non-empty index, the staging start apart);
    // the first arrival's value (dense: then the result).
    __shared__ __align__(16) uint32_t s_cnt[TMAX + 64];  // 64 dummies for idle lanes
    __shared__ __align__(16) float s_out[VALS ? TMAX + 64 : 4];  // first value; dense: the sum
    __shared__ uint16_t s_start[MODE == kSparseWrite ? TMAX : 1];  // staging start (sparse output)
    // Per wave: the tile's entries {j | rank << 12 | code position << 20, raw
    // value word}, then its later arrivals {j | rank << 12 | arrival number
    // << 20, value}.  The walk of indices with more than eight ranks reuses
    // the space.
    __shared__ __align__(16) uint2 s_ent[NW * ERGN];
    __shared__ float s_sv[VALS ? CAP + 8 : 1];             // later values by index, arrival order
    __shared__ uint8_t s_sr[CAP + 8];                      // and their ranks
    __shared__ uint16_t s_cands[NW * (CWC + 64)];          // per wave: indices with three or more ranks
    __shared__ uint32_t s_lista[CCAP];                     // 3-4 ranks: j | start << 12
    __shared__ uint32_t s_listb[CCAP];                     // 6+ ranks from the bottom, 5 from the top
    __shared__ uint32_t s_E[CNTS ? EW + 64 : 1];
    // Per wave and slot: {stream position, entries in this tile, chunk end,
    // last readable entry}, {index base, value base}, {level unit}.  Slot s
    // of wave w is rank s*NW + w (waves interleave, so small P still spreads
    // over all waves); ranks past P have an empty window over a readable
    // dummy address.  A wave reads its slots at fixed offsets.
    __shared__ uint4 s_slot[NW * SLMAX * 3];
    __shared__ uint32_t s_wtot[NW];
    // tile counters: staged values | list A << 16 | list B << 32 | five-rank
    // list << 48 (each below 2^16), non-empty indices, overflow flag
    __shared__ uint64_t s_alloc;
    __shared__ uint32_t s_ne, s_flag;
    // per wave and row of the row walk: values by rank, ranks present
    float* const s_wv = reinterpret_cast<float*>(s_ent);
    uint32_t* const s_wp = reinterpret_cast<uint32_t*>(s_ent) + NW * RROWS * PMAX;

    const uint32_t tid = threadIdx.x, lane = tid & 63u;
    const uint32_t wv = __builtin_amdgcn_readfirstlane(tid >> 6);
    const uint32_t P = a.P, L = a.L, T = a.T;
    const uint32_t chunk = blockIdx.x, stride = a.nchunks + 1;
    const uint32_t t0 = chunk * a.tpc, t1 = min(t0 + a.tpc, a.ntiles);
    const uint32_t qbits = a.qbits, qlog = qbits == 8u ? 3u : (qbits == 4u ? 2u : 1u);
    const uint32_t plog = qbits == 8u ? 0u : (qbits == 4u ? 1u : 2u);
    const uint32_t EB = wv * ERGN;  // this wave's entry region

    // Loop-invariant values (LDS addresses of a thread's coordinates) would
    // be hoisted out of the tile loop and held in registers or spilled; an
    // opaque copy of the thread number keeps them next to their use.
    auto opaque_v = [](uint32_t v) -> uint32_t {
        asm volatile("" : "+v"(v));
        return v;
    };
    uint4* const sw = s_slot + 3u * SLMAX * wv;  // this wave's slots
    // entries of rank r in the current tile
    auto rank_count = [&](uint32_t r) -> uint32_t { return s_slot[3u * ((r % NW) * SLMAX + r / NW)].y; };
    auto reset_counters = [&]() {
        s_alloc = 0u;
        s_ne = s_flag = 0u;
    };

    for (uint32_t r = tid; r < (uint32_t)PMAX; r += NT) {
        uint2 pn = make_uint2(0u, 0u), el = make_uint2(0u, 0u);  // {position, count}, {end, last}
        uint64_t ib = reinterpret_cast<uint64_t>(a.tab), vb = ib;  // readable dummy
        float unit = 0.0f;
        if (r < P) {
            const StreamDesc& d = a.tab[r];
            pn.x = a.off[r * stride + chunk];
            el.x = a.off[r * stride + chunk + 1];
            if (d.nnz) {
                el.y = (uint32_t)(d.nnz - 1u);
                ib = reinterpret_cast<uint64_t>(d.idx);
                vb = reinterpret_cast<uint64_t>(QUANT ? static_cast<const void*>(d.qval)
                                                      : static_cast<const void*>(d.val));
            }
            if (QUANT && VALS) unit = level_unit(*d.qscale, qbits);
        }
        uint4* const sl = s_slot + 3u * ((r % NW) * SLMAX + r / NW);
        sl[0] = make_uint4(pn.x, pn.y, el.x, el.y);
        sl[1] = make_uint4((uint32_t)ib, (uint32_t)(ib >> 32), (uint32_t)vb, (uint32_t)(vb >> 32));
        sl[2] = make_uint4(__float_as_uint(unit), 0u, 0u, 0u);
    }
    for (uint32_t i = tid; i < TMAX + 64; i += NT) {
        s_cnt[i] = 0u;
        if (VALS) s_out[i] = 0.0f;
    }
    if (CNTS)
        for (uint32_t i = tid; i < EW + 64; i += NT) s_E[i] = 0u;
    if (tid == 0) reset_counters();
    __syncthreads();

    // Window of a stream at position pos: raw index and raw value word (fp32
    // bits, or the byte holding the entry's code).  Positions past the
    // stream's end read its last entry (they lie past the chunk end too).
    auto load_win_at = [&](const uint4& b, uint32_t last, uint32_t pos, uint32_t& x, uint32_t& v) {
        const uint32_t i = min(pos + lane, last);
        const uint64_t ib = ((uint64_t)b.y << 32) | b.x;
        x = *reinterpret_cast<g_u32*>(ib + 4ull * i);
        v = 0u;
        if (VALS) {
            const uint64_t vb = ((uint64_t)b.w << 32) | b.z;
            if (QUANT) v = *reinterpret_cast<g_u8*>(vb + (i >> plog));
            else v = *reinterpret_cast<g_u32*>(vb + 4ull * i);
        }
    };
    // Value bits of a window entry at stream position pos + lane: the fp32
    // word, or the entry's code (its bits of the byte) dequantized.
    // (+-level * unit, level 0 giving +0: the sign bit set on a nonzero
    // level negates the product.)
    const uint32_t hbit = 1u << (qbits - 1u);
    auto decode = [&](uint32_t v, uint32_t pos, float unit) -> uint32_t {
        if (!QUANT) return v;
        const uint32_t code = __builtin_amdgcn_ubfe(v, ((lane + pos) << qlog) & 7u, qbits);
        const uint32_t lev = code & (hbit - 1u);
        const float mag = __fmul_rn((float)lev, unit);
        const float val = code > hbit ? -mag : mag;
        return lev ? __float_as_uint(val) : 0u;
    };
    // Append a window to this wave's entry region as {j | rank << 12, value
    // bits}: the in-tile entries of a window are a prefix of it (streams are
    // ascending), so lane i goes to position base + i; the lanes past the
    // prefix write slack that the next window or the region's 64 spare
    // entries take.  Nothing is written once the region is full.
    auto append = [&](uint32_t base, uint32_t jr, uint32_t v) {
        if (base <= ECAP) s_ent[EB + base + lane] = make_uint2(jr, v);
    };

    // xr, vr: raw window words of every slot (in flight during a tile).
    uint32_t xr[SLMAX], vr[SLMAX];
#pragma unroll
    for (int s = 0; s < SLMAX; ++s) load_win_at(sw[3 * s + 1], sw[3 * s].w, sw[3 * s].x, xr[s], vr[s]);

    for (uint32_t tile = t0; tile < t1; ++tile) {
        const uint32_t trel = tile * T, tlo = a.lo + trel;  // tile start, in the range and absolute
        const uint32_t TT = (uint32_t)min((uint64_t)T, (uint64_t)a.N - trel);  // tile width
        const uint32_t toff = MODE == kSparseWrite ? a.tile_off[tile] : 0u;

        // P1w: the in-tile entries of every window, compacted into this
        // wave's region (no other wave touches it, so no barrier follows).
        // A window entirely inside the tile is continued at once; then the
        // slot's next window is requested, so that its load overlaps the
        // rest of this tile.
        uint32_t nent = 0u;
        // This tile's windows were requested a whole tile ago: wait for all of
        // them here, once (vmcnt(0)), so that no later use waits behind the
        // next tile's requests issued below.
        __builtin_amdgcn_s_waitcnt(0x0F70);
        constexpr int G1 = SLMAX < 4 ? SLMAX : 4;
#pragma unroll
        for (int g0 = 0; g0 < SLMAX; g0 += G1) {
            uint4 st[G1], bs[G1];
            float un[G1];
#pragma unroll
            for (int q = 0; q < G1; ++q) {
                st[q] = sw[3 * (g0 + q)];
                bs[q] = sw[3 * (g0 + q) + 1];
                un[q] = QUANT && VALS ? __uint_as_float(sw[3 * (g0 + q) + 2].x) : 0.0f;
            }
#pragma unroll
            for (int q = 0; q < G1; ++q) {
                const int s = g0 + q;
                // (j | rank << 12) of an in-tile entry x is x plus this
                const uint32_t jr0 = (((uint32_t)s * NW + wv) << 12) - tlo;
                uint32_t pos = st[q].x;
                const uint32_t end = st[q].z, last = st[q].w;
                uint32_t n = (uint32_t)__popcll(lanes_lt(xr[s] - tlo, TT) & lanes_lt(lane, end - pos));
                append(nent, xr[s] + jr0, VALS ? decode(vr[s], pos, un[q]) : 0u);
                nent += n;
                pos += n;
                uint32_t cnt = n;
                if (n == kWin) {  // rare: continue the window
                    do {
                        uint32_t x2, v2;
                        load_win_at(bs[q], last, pos, x2, v2);
                        n = (uint32_t)__popcll(lanes_lt(x2 - tlo, TT) & lanes_lt(lane, end - pos));
                        append(nent, x2 + jr0, VALS ? decode(v2, pos, un[q]) : 0u);
                        nent += n;
                        pos += n;
                        cnt += n;
                    } while (n == kWin);
                }
                // every lane stores the same {position, count}
                *reinterpret_cast<uint2*>(&sw[3 * s]) = make_uint2(pos, cnt);
                load_win_at(bs[q], last, pos, xr[s], vr[s]);
            }
        }
        if (nent > ECAP && lane == 0u) s_flag = 1u;
        const uint32_t ne_w = min(nent, ECAP);
        // P1e: arrival numbers of this wave's entries, two per lane and step
        // so that their LDS round trips overlap (idle lanes count at dummy
        // words).  The first arrival leaves its value at the index; the later
        // ones are compacted to the front of the wave's region (never past
        // what the wave has read) with their arrival number -- the second
        // with the first one's rank instead, and a flag -- and the third
        // lists its index as one with three or more ranks.  The next step's
        // entries, which this step never overwrites, are read ahead.
        // (Lanes read entries other lanes of the wave wrote: the fence orders
        // them for the compiler.)
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        const uint32_t CB = wv * (CWC + 64u);  // this wave's candidate region
        uint32_t nlat = 0u, ncw = 0u, nfirst = 0u;
        uint2 nx0 = s_ent[EB + lane], nx1 = s_ent[EB + 64u + lane];
        for (uint32_t b = 0; b < ne_w; b += 128u) {
            const uint2 en0 = nx0, en1 = nx1;
            const bool ok0 = b + lane < ne_w, ok1 = b + 64u + lane < ne_w;
            const uint32_t j0 = en0.x & 0xFFFu, j1 = en1.x & 0xFFFu;
            const uint32_t w0 = atomicAdd(&s_cnt[ok0 ? j0 : TMAX + lane], 1u + ((en0.x >> 12) << 16));
            const uint32_t w1 = atomicAdd(&s_cnt[ok1 ? j1 : TMAX + lane], 1u + ((en1.x >> 12) << 16));
            const uint32_t k0 = w0 & 0xFFFFu, k1 = w1 & 0xFFFFu;
            nx0 = s_ent[EB + min(b + 128u + lane, ECAP - 1u)];
            nx1 = s_ent[EB + min(b + 192u + lane, ECAP - 1u)];
            const bool f0 = ok0 && k0 == 0u, f1 = ok1 && k1 == 0u;
            const bool l0 = ok0 && k0 != 0u, l1 = ok1 && k1 != 0u;
            const bool c0 = ok0 && k0 == 2u, c1 = ok1 && k1 == 2u;
            // Writes are unconditional: a lane with nothing to write aims at
            // a dummy word (past the tile, the region's slack, the list's end).
            const uint32_t fj0 = f0 ? j0 : TMAX + lane, fj1 = f1 ? j1 : TMAX + lane;
            if (VALS) s_out[fj0] = MODE == kDense ? __uint_as_float(en0.y) + 0.0f : __uint_as_float(en0.y);
            if (VALS) s_out[fj1] = MODE == kDense ? __uint_as_float(en1.y) + 0.0f : __uint_as_float(en1.y);
            // lane masks from single comparisons, combined on the scalar unit
            const uint64_t OK0 = lanes_lt(b + lane, ne_w), OK1 = lanes_lt(b + 64u + lane, ne_w);
            const uint64_t Z0 = lanes_eq(k0, 0u), Z1 = lanes_eq(k1, 0u);
            const uint64_t L0 = OK0 & ~Z0, L1 = OK1 & ~Z1;
            const uint64_t C0 = OK0 & lanes_eq(k0, 2u), C1 = OK1 & lanes_eq(k1, 2u);
            if (CNTS) nfirst += (uint32_t)__popcll(OK0 & Z0) + (uint32_t)__popcll(OK1 & Z1);
            const uint32_t p0 = below_count(L0, nlat);
            nlat += (uint32_t)__popcll(L0);
            const uint32_t p1 = below_count(L1, nlat);
            nlat += (uint32_t)__popcll(L1);
            const uint32_t q0 = below_count(C0, ncw);
            ncw += (uint32_t)__popcll(C0);
            const uint32_t q1 = below_count(C1, ncw);
            ncw += (uint32_t)__popcll(C1);
            // {j | rank << 12 | (k, or for k = 1 the first rank | 1 << 8) << 20, value}
            const uint32_t t0 = k0 == 1u ? (w0 >> 16) | 0x100u : k0, t1 = k1 == 1u ? (w1 >> 16) | 0x100u : k1;
            s_ent[EB + (l0 ? p0 : ECAP + lane)] = make_uint2(en0.x | t0 << 20, en0.y);
            s_ent[EB + (l1 ? p1 : ECAP + lane)] = make_uint2(en1.x | t1 << 20, en1.y);
            s_cands[CB + (c0 && q0 < CWC ? q0 : CWC + lane)] = (uint16_t)j0;
            s_cands[CB + (c1 && q1 < CWC ? q1 : CWC + lane)] = (uint16_t)j1;
        }
        if (lane == 0u) {
            if (CNTS && nfirst) atomicAdd(&s_ne, nfirst);
            if (ncw > CWC) s_flag = 1u;
        }
        __syncthreads();

        const bool over = s_flag != 0u;
        if (!over) {
            if (MODE == kSparseWrite) {
                // output position (index order) of every non-empty index; a
                // single value is written out here
                const uint32_t jb = opaque_v(tid) * CPT;
                uint32_t mc[CPT];
#pragma unroll
                for (int c = 0; c < CPT; c += 4) {
                    const uint4 q = *reinterpret_cast<const uint4*>(&s_cnt[jb + c]);
                    mc[c] = q.x;
                    mc[c + 1] = q.y;
                    mc[c + 2] = q.z;
                    mc[c + 3] = q.w;
                }
                uint32_t ne = 0u;
#pragma unroll
                for (int c = 0; c < CPT; ++c) ne += mc[c] != 0u ? 1u : 0u;
                const uint32_t incl = wave_scan(ne);
                if (lane == 63u) s_wtot[wv] = incl;
                __syncthreads();
                const uint32_t wt = lane < (uint32_t)NW ? s_wtot[lane] : 0u;
                const uint32_t xs = wave_scan(wt);
                uint32_t nrun = incl - ne + (uint32_t)__builtin_amdgcn_readlane((int)(xs - wt), (int)wv);
#pragma unroll
                for (int c = 0; c < CPT; ++c) {
                    const uint32_t m = mc[c] & 0xFFFFu, j = jb + (uint32_t)c;
                    if (m == 1u) {
                        put_sparse(a, toff + nrun, tlo + j, s_out[j]);
                    } else if (m != 0u) {
                        s_cnt[j] = m | nrun << 9;
                    }
                    nrun += m != 0u ? 1u : 0u;
                }
                __syncthreads();
            }
            // Candidates of this wave, one per lane: the staging range of the
            // later arrivals and the walk list by rank count.
            for (uint32_t b = 0; b < ncw; b += 64u) {
                const uint32_t i = b + lane;
                const bool act = i < ncw;
                const uint32_t j = act ? (uint32_t)s_cands[CB + i] : 0u;
                const uint32_t m = act ? s_cnt[j] & 0x1FFu : 0u;
                const uint32_t ext = m;  // all m values, the first staged by the second arrival
                const uint32_t incl = wave_scan(ext);
                const bool ca = act && m <= 4u, cb = act && m > 5u, c5 = act && m == 5u;
                const uint64_t ACT = lanes_lt(i, ncw);
                const uint64_t BA = ACT & lanes_lt(m, 5u), BB = ACT & ~lanes_lt(m, 6u), B5 = ACT & lanes_eq(m, 5u);
                // one reservation for the staging range and the three lists
                const uint64_t want = (uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)incl, 63) |
                                      (uint64_t)__popcll(BA) << 16 | (uint64_t)__popcll(BB) << 32 |
                                      (uint64_t)__popcll(B5) << 48;
                uint64_t got = 0u;
                if (lane == 0u) got = atomicAdd(&s_alloc, want);
                const uint32_t glo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)got);
                const uint32_t ghi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(got >> 32));
                const uint32_t start = (glo & 0xFFFFu) + incl - ext;
                const uint32_t pa = below_count(BA, glo >> 16);
                const uint32_t pb = below_count(BB, ghi & 0xFFFFu);
                const uint32_t p5 = below_count(B5, ghi >> 16);
                if (act && start + ext <= CAP) {
                    if (MODE == kSparseWrite) s_start[j] = (uint16_t)start;
                    else s_cnt[j] = m | start << 9;
                    const uint32_t item = j | start << 12;
                    if (ca) s_lista[pa] = item;
                    if (cb) s_listb[pb] = item;
                    if (c5) s_listb[CCAP - 1u - p5] = item;
                }
            }
        }
        __syncthreads();
        const uint64_t al = s_alloc;
        const bool defer = over || (uint32_t)(al & 0xFFFFu) > CAP;
        const uint32_t NE = s_ne, NA = (uint32_t)(al >> 16) & 0xFFFFu;
        const uint32_t NB = (uint32_t)(al >> 32) & 0xFFFFu, N5 = (uint32_t)(al >> 48);

        if (!defer) {
            if (CNTS && tid == 0) a.tile_cnt[tile] = NE;
            // P2, per later arrival of this wave: an index with two ranks is
            // finished here -- a single addition is the same in either order --
            // and counts its pair for the node sizes; otherwise the value is
            // staged at its index's range in arrival order, the second arrival
            // staging the first one's value and rank as well.
            // Two entries per lane and step; every read of a step comes before
            // its writes (no two entries of a step finish the same pair).
            auto place = [&](uint2 en, uint32_t sc, uint32_t st, float first) {
                const uint32_t jj = en.x & 0xFFFu, r = (en.x >> 12) & 0xFFu, t = en.x >> 20;
                const bool second = t >= 0x100u;
                const uint32_t r0 = t & 0xFFu;  // the first rank (second arrival)
                if ((sc & 0x1FFu) == 2u) {
                    if (CNTS) atomicAdd(&s_E[sep_level(r0, r) * PMAX + max(r0, r)], 1u);
                    if (VALS) {
                        const float sum = first + __uint_as_float(en.y);
                        if (MODE == kDense) {
                            s_out[jj] = sum;
                        } else {
                            put_sparse(a, toff + (sc >> 9), tlo + jj, sum);
                        }
                    }
                } else {
                    const uint32_t at = st + (second ? 1u : t);
                    s_sr[at] = (uint8_t)r;
                    if (VALS) s_sv[at] = __uint_as_float(en.y);
                    if (second) {
                        s_sr[st] = (uint8_t)r0;
                        if (VALS) s_sv[st] = first;
                    }
                }
            };
            for (uint32_t i = lane; i < nlat; i += 128u) {
                const bool two = i + 64u < nlat;
                const uint2 e0 = s_ent[EB + i];
                const uint2 e1 = s_ent[EB + (two ? i + 64u : i)];
                const uint32_t ja = e0.x & 0xFFFu, jb = e1.x & 0xFFFu;
                const uint32_t sa = s_cnt[ja], sb = s_cnt[jb];
                const uint32_t ta = MODE == kSparseWrite ? (uint32_t)s_start[ja] : sa >> 9;
                const uint32_t tb = MODE == kSparseWrite ? (uint32_t)s_start[jb] : sb >> 9;
                const float oa = VALS ? s_out[ja] : 0.0f, ob = VALS ? s_out[jb] : 0.0f;
                place(e0, sa, ta, oa);
                if (two) place(e1, sb, tb, ob);
            }
            __syncthreads();
            if (tid == 0) reset_counters();  // every thread has read them

            auto emit = [&](uint32_t jj, float sum) {
                if (MODE == kDense) {
                    s_out[jj] = sum + 0.0f;
                } else {
                    put_sparse(a, toff + (s_cnt[jj] >> 9), tlo + jj, sum);
                }
            };
            auto cswap_rv = [](uint32_t* rk, float* vv, int x, int y) {
                const bool sw = rk[x] > rk[y];
                const uint32_t tr = rk[x];
                const float tv = vv[x];
                rk[x] = sw ? rk[y] : rk[x];
                rk[y] = sw ? tr : rk[y];
                vv[x] = sw ? vv[y] : vv[x];
                vv[y] = sw ? tv : vv[y];
            };
            // Waves 4q + s run on SIMD s (round-robin placement).  The walk of
            // three or four ranks fills the waves of SIMDs 0-2 from the first.
            // The row walk takes the waves of SIMD 3 first when its rows fit
            // there (those the walk above leaves free), else waves from the
            // other end (those of SIMDs 0-2 from the last, then SIMD 3's), so
            // that the two spread over the four SIMDs.
            constexpr uint32_t G3 = (NW / 4) * 3;
            static_assert(NW % 4 == 0, "four SIMDs");
            const uint32_t wslot = (wv & 3u) != 3u ? (wv >> 2) * 3u + (wv & 3u) : G3 + (wv >> 2);
            // Walk: indices with three or four ranks -- sorted by a network,
            // summed with the association their separators dictate.
            for (uint32_t i = wslot * 64u + lane; i < NA; i += NT) {
                const uint32_t item = s_lista[i];
                const uint32_t jj = item & 0xFFFu, st0 = item >> 12;
                const uint32_t mm = s_cnt[jj] & 0x1FFu;
                uint32_t rk[4];
                float vv[4];
                rk[0] = s_sr[st0];
                rk[1] = s_sr[st0 + 1];
                rk[2] = s_sr[st0 + 2];
                rk[3] = mm == 4u ? (uint32_t)s_sr[st0 + 3] : 0x100u;  // above every rank
                if (VALS) {
                    vv[0] = s_sv[st0];
                    vv[1] = s_sv[st0 + 1];
                    vv[2] = s_sv[st0 + 2];
                    vv[3] = mm == 4u ? s_sv[st0 + 3] : 0.0f;
                } else {
                    vv[0] = vv[1] = vv[2] = vv[3] = 0.0f;
                }
                cswap_rv(rk, vv, 0, 1);
                cswap_rv(rk, vv, 2, 3);
                cswap_rv(rk, vv, 0, 2);
                cswap_rv(rk, vv, 1, 3);
                cswap_rv(rk, vv, 1, 2);
                const uint32_t c1 = sep_level(rk[0], rk[1]), c2 = sep_level(rk[1], rk[2]);
                const uint32_t c3 = mm == 4u ? sep_level(rk[2], rk[3]) : 0u;
                if (CNTS) {
                    atomicAdd(&s_E[c1 * PMAX + rk[1]], 1u);
                    atomicAdd(&s_E[c2 * PMAX + rk[2]], 1u);
                    atomicAdd(&s_E[mm == 4u ? c3 * PMAX + rk[3] : EW + lane], 1u);
                }
                if (VALS) emit(jj, mm == 3u ? tree3(vv[0], vv[1], vv[2], c1, c2)
                                            : tree4(vv[0], vv[1], vv[2], vv[3], c1, c2, c3));
            }
            // Walk: indices with five ranks, one per thread (from the top
            // thread down, so that they share few waves with the above): a
            // sorting network, then the root splits at the largest separator
            // into parts of at most four, summed by the forms above.
            for (uint32_t i = NT - 1u - tid; i < N5; i += NT) {
                const uint32_t item = s_listb[CCAP - 1u - i];
                const uint32_t jj = item & 0xFFFu, st0 = item >> 12;
                uint32_t rk[5];
                float vv[5];
#pragma unroll
                for (int e = 0; e < 5; ++e) {
                    rk[e] = s_sr[st0 + e];
                    vv[e] = VALS ? s_sv[st0 + e] : 0.0f;
                }
                cswap_rv(rk, vv, 0, 3); cswap_rv(rk, vv, 1, 4); cswap_rv(rk, vv, 0, 2);
                cswap_rv(rk, vv, 1, 3); cswap_rv(rk, vv, 0, 1); cswap_rv(rk, vv, 2, 4);
                cswap_rv(rk, vv, 1, 2); cswap_rv(rk, vv, 3, 4); cswap_rv(rk, vv, 2, 3);
                const uint32_t c1 = sep_level(rk[0], rk[1]), c2 = sep_level(rk[1], rk[2]);
                const uint32_t c3 = sep_level(rk[2], rk[3]), c4 = sep_level(rk[3], rk[4]);
                if (CNTS) {
                    atomicAdd(&s_E[c1 * PMAX + rk[1]], 1u);
                    atomicAdd(&s_E[c2 * PMAX + rk[2]], 1u);
                    atomicAdd(&s_E[c3 * PMAX + rk[3]], 1u);
                    atomicAdd(&s_E[c4 * PMAX + rk[4]], 1u);
                }
                if (VALS) {
                    const float t012 = tree3(vv[0], vv[1], vv[2], c1, c2);
                    const float t234 = tree3(vv[2], vv[3], vv[4], c3, c4);
                    const float t0123 = tree4(vv[0], vv[1], vv[2], vv[3], c1, c2, c3);
                    const float t1234 = tree4(vv[1], vv[2], vv[3], vv[4], c2, c3, c4);
                    const uint32_t top = max(max(c1, c2), max(c3, c4));
                    float sum;
                    if (c1 == top) sum = vv[0] + t1234;
                    else if (c2 == top) sum = (vv[0] + vv[1]) + t234;
                    else if (c3 == top) sum = t012 + (vv[3] + vv[4]);
                    else sum = t0123 + vv[4];
                    emit(jj, sum);
                }
            }
            // Walk: indices with six or more ranks, one per row of 16 lanes
            // (ROWS per wave and pass).  Lane l of a row holds ranks l*K ..
            // l*K+K-1 of its index: the values are scattered by rank to the
            // row's region and the tree is evaluated level by level, within
            // the lane and then across the row (DPP) -- a node is the sum of its
            // two children when both hold a value, else the one that does: the
            // recursive doubling of the ranks present.  A present rank's
            // predecessor (for the node sizes) is the previous present one in
            // its lane, else the highest present one in the row's lower lanes.
            {
                const uint32_t row = min(lane >> 4, RROWS - 1u), l16 = lane & 15u;
                float* const rval = s_wv + (wv * RROWS + row) * PMAX;
                uint32_t* const rpre = s_wp + (wv * RROWS + row) * PW;
                const uint32_t base = l16 * RK;
                const bool few = NB <= (uint32_t)(NW / 4) * RROWS;
                // (at 64 ranks, where many rows are common -- about 36 a tile
                // at c4 -- they go round robin over SIMDs 2, 1, 0, 3, each
                // from its last wave down, SIMD 3's last wave walking the
                // five-rank list: 0.279 -> 0.275 ms at c4; the wider kernels
                // keep the order their register allocation was measured with,
                // the round robin costing c5 0.3%)
                const uint32_t rq_many =
                    PMAX != 64 ? (wslot < G3 ? G3 - 1u - wslot : wslot)
                               : ((wv & 3u) == 3u ? ((wv >> 2) == 3u ? 3u : 2u - (wv >> 2)) : 3u - (wv >> 2)) * 4u +
                                     ((wv & 3u) == 3u ? 3u : 2u - (wv & 3u));
                const uint32_t rq = few ? (wslot >= G3 ? wslot - G3 : (uint32_t)NW / 4u + G3 - 1u - wslot) : rq_many;
                for (uint32_t b0 = rq * RROWS; b0 < NB; b0 += RROWS * NW) {
                    const uint32_t i = b0 + row;
                    const bool act = (lane >> 4) < RROWS && i < NB;
                    const uint32_t item = act ? s_listb[i] : 0u;
                    const uint32_t jj = item & 0xFFFu, st0 = item >> 12;
                    const uint32_t mm = act ? s_cnt[jj] & 0x1FFu : 0u;
                    if ((lane >> 4) < RROWS && l16 < (uint32_t)PW) rpre[l16] = 0u;
                    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                    for (uint32_t e = l16; e < mm; e += 16u) {
                        const uint32_t r = s_sr[st0 + e];
                        if (VALS) rval[r] = s_sv[st0 + e];
                        atomicOr(&rpre[r >> 5], 1u << (r & 31u));
                    }
                    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                    const uint32_t bits = act ? (rpre[base >> 5] >> (base & 31u)) & (RK == 32 ? ~0u : (1u << RK) - 1u) : 0u;
                    if (CNTS) {
                        // (rank + 1) of the highest present rank in lower lanes of the row
                        uint32_t top = bits ? base + 32u - (uint32_t)__clz(bits) : 0u;
                        top = max(top, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)top, 0x111, 0xF, 0xF, true));
                        top = max(top, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)top, 0x112, 0xF, 0xF, true));
                        top = max(top, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)top, 0x114, 0xF, 0xF, true));
                        top = max(top, (uint32_t)__builtin_amdgcn_update_dpp(0, (int)top, 0x118, 0xF, 0xF, true));
                        uint32_t prev = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)top, 0x111, 0xF, 0xF, true);
#pragma unroll
                        for (uint32_t q = 0; q < RK; ++q) {
                            const bool pres = (bits >> q) & 1u;
                            const uint32_t r = base + q;
                            atomicAdd(&s_E[pres && prev ? sep_level(prev - 1u, r) * PMAX + r : EW + lane], 1u);
                            prev = pres ? r + 1u : prev;
                        }
                    }
                    if (VALS) {
                        float lv[RK];
                        bool lp[RK];
#pragma unroll
                        for (uint32_t q = 0; q < RK; ++q) {
                            lp[q] = (bits >> q) & 1u;
                            lv[q] = lp[q] ? rval[base + q] : 0.0f;
                        }
#pragma unroll
                        for (uint32_t h = 1; h < RK; h <<= 1) {
#pragma unroll
                            for (uint32_t q = 0; q < RK; q += 2 * h) {
                                lv[q] = tree_join(lv[q], lp[q], lv[q + h], lp[q + h]);
                                lp[q] = lp[q] || lp[q + h];
                            }
                        }
                        float v = lv[0];
                        uint32_t pr = lp[0] ? 1u : 0u;
                        tree_level<1>(v, pr, lane);
                        tree_level<2>(v, pr, lane);
                        tree_level<4>(v, pr, lane);
                        tree_level<8>(v, pr, lane);
                        if (act && l16 == 0u) emit(jj, v);
                    }
                    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
                }
            }
            __syncthreads();

            // Store the dense tile; clear the tile state.
            for (uint32_t c = opaque_v(tid) * 4u; c < T; c += NT * 4u) {
                if (MODE == kDense) {
                    const float4 v = *reinterpret_cast<const float4*>(&s_out[c]);
                    *reinterpret_cast<float4*>(&s_out[c]) = make_float4(0.f, 0.f, 0.f, 0.f);
                    const uint64_t g = (uint64_t)trel + c;
                    if (a.out_vec && c + 4u <= TT) {
                        store_nt(a.out_val + g, v);
                    } else {
                        if (c < TT) a.out_val[g] = v.x;
                        if (c + 1u < TT) a.out_val[g + 1] = v.y;
                        if (c + 2u < TT) a.out_val[g + 2] = v.z;
                        if (c + 3u < TT) a.out_val[g + 3] = v.w;
                    }
                }
                *reinterpret_cast<uint4*>(&s_cnt[c]) = make_uint4(0u, 0u, 0u, 0u);
            }
        } else {
            __syncthreads();  // every thread has read the counters
            // the slow pass counts this tile's entries of every rank
            if (CNTS)
                for (uint32_t r = tid; r < P; r += NT) s_E[L * PMAX + r] -= rank_count(r);
            if (tid == 0) {
                reset_counters();
                const uint32_t k = atomicAdd(a.slow_count, 1u);
                a.slow_list[k] = tile;
            }
            for (uint32_t c = opaque_v(tid) * 4u; c < T; c += NT * 4u) {
                *reinterpret_cast<uint4*>(&s_cnt[c]) = make_uint4(0u, 0u, 0u, 0u);
                if (VALS) *reinterpret_cast<float4*>(&s_out[c]) = make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
        __syncthreads();
    }
    __syncthreads();
    if (CNTS) {
        // all entries of the chunk's streams (less those of deferred tiles,
        // subtracted above)
        for (uint32_t r = tid; r < P; r += NT)
            s_E[L * PMAX + r] += a.off[r * stride + chunk + 1] - a.off[r * stride + chunk];
        __syncthreads();
        flush_counts<NT, PMAX>(s_E, a);
    }
}

// ------------------------------------------------------------------------
// Slow pass: one workgroup per deferred tile, any number of entries.  Ranks
// are taken in order; each coordinate keeps the tree-sum stack in LDS
// (current value, last rank, pending-level bits, one slot per level).
template <int MW, int MODE, bool QUANT>
__global__ void __launch_bounds__(kSlowNT) k_slow(Args a)
{
    constexpr int NT = kSlowNT, TS = kSlowTS, LMAX = SlowShape<MW>::LMAX, PMAX = 32 * MW;
    if (MODE == kSparseWrite && a.skip && a.skip->dense) return;  // the root is dense: nothing to write
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
        const uint32_t tlo = a.lo + tile * a.T;
        const uint32_t thi = (uint32_t)min((uint64_t)tlo + a.T, (uint64_t)a.lo + a.N);
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
                    if (j < width) a.out_val[sub - a.lo + j] = ((nzbits >> q) & 1u) ? vals[q] + 0.0f : 0.0f;
                }
            } else if (MODE == kSparseWrite) {
                uint32_t o = a.tile_off[tile] + tile_nz + excl;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if ((nzbits >> q) & 1u) {
                        put_sparse(a, o, (uint32_t)sub + tid * 4 + q, vals[q]);
                        ++o;
                    }
                }
            }
            tile_nz += total;
        }
        if (MODE != kSparseWrite && tid == 0) a.tile_cnt[tile] = tile_nz;
    }
    __syncthreads();
    if (MODE != kSparseWrite) flush_counts<NT, 0>(s_E, a);
}

// ------------------------------------------------------------------------
// Stream r's descriptor from the launch's arguments (fmt != kDescNone).
static_assert(sizeof(StreamDesc) == 48 && offsetof(StreamDesc, idx) == 0 && offsetof(StreamDesc, val) == 8 &&
                  offsetof(StreamDesc, qval) == 16 && offsetof(StreamDesc, qscale) == 24 &&
                  offsetof(StreamDesc, nnz) == 32,
              "descriptor words");
__device__ __forceinline__ StreamDesc arg_desc(const DescArgs& tb, uint32_t r)
{
    auto word2 = [&](uint32_t i) -> uint64_t { return (uint64_t)tb.words[i] | (uint64_t)tb.words[i + 1] << 32; };
    StreamDesc d{};
    if (tb.fmt == kDescFull) {
        const uint32_t b = r * (uint32_t)(sizeof(StreamDesc) / 4);
        d.idx = reinterpret_cast<const uint32_t*>(word2(b));
        d.val = reinterpret_cast<const float*>(word2(b + 2u));
        d.qval = reinterpret_cast<const uint8_t*>(word2(b + 4u));
        d.qscale = reinterpret_cast<const float*>(word2(b + 6u));
        d.nnz = word2(b + 8u);
    } else {
        const uint32_t b = r * 5u;
        d.idx = reinterpret_cast<const uint32_t*>(word2(b));
        if (tb.fmt == kDescCodes) {
            d.qval = reinterpret_cast<const uint8_t*>(word2(b + 2u));
            d.qscale = tb.scale0 + r;
        } else {
            d.val = reinterpret_cast<const float*>(word2(b + 2u));
        }
        d.nnz = tb.words[b + 4u];
    }
    return d;
}

// Per-chunk start offsets of every stream and zeroing of the counters the
// passes accumulate into; workgroup r takes stream r.  A sample of the
// stream (every stride-th index, at most kPartSamples, read at once) narrows
// each chunk start's search to one stride of positions, so a search waits on
// about half the dependent loads of a binary search over the whole stream.
// When the descriptors travel in the arguments this launch also stores them
// to `tab` for the later passes, and reads its own from the arguments.
constexpr uint32_t kPartSamples = 1024;
__global__ void __launch_bounds__(256) k_partition(StreamDesc* tab, DescArgs tb, uint32_t* off, uint32_t nchunks,
                                                   uint64_t chunk_coords, uint64_t lo, uint64_t N, uint32_t* zero,
                                                   uint32_t nzero)
{
    __shared__ uint32_t s_smp[kPartSamples];
    const uint32_t r = blockIdx.x, tid = threadIdx.x;
    if (r == 0)
        for (uint32_t i = tid; i < nzero; i += blockDim.x) zero[i] = 0u;
    const uint32_t* idx;
    uint32_t nnz;
    if (tb.fmt != kDescNone) {
        const StreamDesc d = arg_desc(tb, r);
        if (tid == 0) tab[r] = d;
        idx = d.idx;
        nnz = (uint32_t)d.nnz;
    } else {
        idx = tab[r].idx;
        nnz = (uint32_t)tab[r].nnz;
    }
    // samples j < ns: the index at position j * stride
    const uint32_t stride = nnz > kPartSamples ? (uint32_t)(((uint64_t)nnz + kPartSamples - 1u) / kPartSamples) : 1u;
    const uint32_t ns = (uint32_t)(((uint64_t)nnz + stride - 1u) / stride);
    for (uint32_t j = tid; j < ns; j += blockDim.x) s_smp[j] = idx[(uint64_t)j * stride];
    __syncthreads();
    uint32_t* const o = off + (uint64_t)r * (nchunks + 1u);
    for (uint32_t c = tid; c <= nchunks; c += blockDim.x) {
        uint32_t res = nnz;
        if (c < nchunks) {
            const uint64_t x = lo + min((uint64_t)c * chunk_coords, N);
            // js samples lie below x: the first position at or past x is
            // above sample js - 1's and at most sample js's
            uint32_t a = 0u, b = ns;
            while (a < b) {
                const uint32_t m = a + ((b - a) >> 1);
                if ((uint64_t)s_smp[m] < x) a = m + 1u;
                else b = m;
            }
            const uint32_t pa = a ? (a - 1u) * stride + 1u : 0u;
            const uint32_t pb = (uint32_t)min((uint64_t)a * stride, (uint64_t)nnz);
            res = lower_bound(idx, min(pa, pb), pb, x);
        }
        o[c] = res;
    }
}

// Per-segment start offsets of every stream by one pass over its entries,
// for the merge path (whose inputs are few: a pass reads less than the
// searches wait for), and zeroing of that path's counters; the descriptor
// table as in k_partition.  Segment s of the range starts at index
// lo + s segw; for an ascending stream, off[s] = the first position whose
// index is at least that start, so entry e is the offset of every segment
// s with k(idx[e - 1]) <= s < k(idx[e]), where k(x) counts the segment
// starts (of the first nseg) at or below x (k = 0 before the first entry,
// nseg + 1 past the last).  Grid: x over positions 0..nnz of a stream,
// y over streams.  A stream that does not ascend leaves some offsets
// unwritten: the merge path clamps every offset to its stream.
__global__ void k_partition_pass(StreamDesc* tab, DescArgs tb, uint32_t* off, uint32_t nseg, uint64_t segw,
                                 uint64_t lo, uint32_t* zero, uint32_t nzero)
{
    const uint32_t r = blockIdx.y, e = blockIdx.x * blockDim.x + threadIdx.x;
    if (r == 0) {
        if (e < nzero) zero[e] = 0u;
        if (tb.fmt != kDescNone && e < gridDim.y) tab[e] = arg_desc(tb, e);
    }
    const uint32_t* idx;
    uint32_t nnz;
    if (tb.fmt != kDescNone) {
        const StreamDesc d = arg_desc(tb, r);
        idx = d.idx;
        nnz = (uint32_t)d.nnz;
    } else {
        idx = tab[r].idx;
        nnz = (uint32_t)tab[r].nnz;
    }
    if (e > nnz) return;
    auto k = [&](uint32_t x) -> uint32_t {
        if ((uint64_t)x < lo) return 0u;
        const uint64_t d = (uint64_t)x - lo;  // < 2^32
        const uint64_t q = segw - 1ull >= 0xFFFFFFFFull ? 0ull : (uint64_t)((uint32_t)d / (uint32_t)segw);
        return (uint32_t)min(q + 1ull, (uint64_t)nseg);
    };
    const uint32_t ka = e == 0u ? 0u : k(idx[e - 1u]);
    const uint32_t kb = e == nnz ? nseg + 1u : k(idx[e]);
    uint32_t* o = off + (size_t)r * (nseg + 1u);
    for (uint32_t s = ka; s < kb; ++s) o[s] = e;
}

// Switch rule over the tree (§5.1): node dense iff a child is dense or the
// children's nnz sum exceeds thr; a sparse node's nnz is its union size.
// Nodes are reported in level order; only the first nfold nodes of level
// 1 are reported (all of them for a power-of-two rank count: nfold = P/2),
// the higher levels follow them.
// Exclusive scan of the per-tile root union sizes by one 1024-thread
// workgroup; also clears the deferred-tile counter for the write pass.
__device__ void scan_tiles(const uint32_t* cnt, uint32_t* off, uint32_t n, uint32_t* slow_count)
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

// The switch rule over the node sizes (threads 0-255), then, unless the root
// is dense, the exclusive scan of the per-tile root union sizes that gives
// the sparse write pass its output offsets (all 1024 threads; it also clears
// the deferred-tile counter for that pass).  One workgroup.
__global__ void __launch_bounds__(1024) k_decide_scan(const StreamDesc* tab, const uint32_t* node_cnt, uint32_t P,
                                                      uint64_t N, uint64_t thr, uint64_t* node_nnz,
                                                      uint8_t* node_dense, ReduceResult* hdr, uint32_t nfold,
                                                      ReduceResult* result, const uint32_t* cnt, uint32_t* off,
                                                      uint32_t n, uint32_t* slow_count)
{
    // Stream sizes and node union sizes are read by all threads at once, the
    // rule is applied level by level in LDS, and all threads store.
    __shared__ uint64_t s_n[256];    // per group of the current level
    __shared__ uint8_t s_d[256];
    __shared__ uint32_t s_c[256];    // union sizes, level order
    __shared__ uint64_t s_nn[256];   // decided node sizes
    __shared__ uint8_t s_nd[256];
    const uint32_t t = threadIdx.x;
    if (t < P) {
        s_n[t] = tab[t].nnz;
        s_d[t] = 0;
    }
    if (t + 1 < P) s_c[t] = node_cnt[t];
    __syncthreads();
    // level by level (children of group g at 2g, 2g+1), one thread per node
    uint32_t node = 0;
    for (uint32_t width = P; width > 1; width /= 2) {
        const uint32_t g = t;
        bool dense = false;
        uint64_t nnz = 0;
        if (g < width / 2) {
            dense = s_d[2 * g] || s_d[2 * g + 1] || (s_n[2 * g] + s_n[2 * g + 1] > thr);
            nnz = dense ? N : (uint64_t)s_c[node + g];
            s_nn[node + g] = nnz;
            s_nd[node + g] = dense ? 1 : 0;
        }
        __syncthreads();
        if (g < width / 2) {
            s_n[g] = nnz;
            s_d[g] = dense ? 1 : 0;
        }
        __syncthreads();
        node += width / 2;
    }
    if (t == 0) {
        hdr->nnz = s_n[0];
        hdr->dense = s_d[0];
        hdr->pad = 0;
        if (result) *result = ReduceResult{s_n[0], s_d[0], 0u};
    }
    __syncthreads();
    if (t + 1 < P && (t >= P / 2 || t < nfold)) {
        const uint32_t o = t < P / 2 ? t : t - P / 2 + nfold;
        if (node_nnz) node_nnz[o] = s_nn[t];
        if (node_dense) node_dense[o] = s_nd[t];
    }
    if (s_d[0]) return;  // the root is dense: no sparse output (whole workgroup)
    scan_tiles(cnt, off, n, slow_count);
}

__global__ void k_set_result(ReduceResult* r, uint64_t nnz, uint32_t dense)
{
    if (threadIdx.x == 0) *r = ReduceResult{nnz, dense, 0u};
}

template <int PMAX, int MODE>
hipError_t launch_tiles_q(const Args& a, bool quant, hipStream_t s)
{
    constexpr int SMW = PMAX <= 32 ? 1 : PMAX / 32;
    const dim3 grid(a.nchunks), block(Fast<PMAX>::NT);
    const int slot = MODE == kSparseWrite ? kTReduceWrite : kTReducePass;
    timer_begin(slot, s);
    if (quant) hipLaunchKernelGGL((k_tiles<PMAX, MODE, true>), grid, block, 0, s, a);
    else hipLaunchKernelGGL((k_tiles<PMAX, MODE, false>), grid, block, 0, s, a);
    timer_end(slot, s);
    const uint32_t sg = std::min<uint32_t>(a.ntiles, 256u);
    if (MODE != kSparseWrite) timer_begin(kTReduceSlow, s);
    if (quant) hipLaunchKernelGGL((k_slow<SMW, MODE, true>), dim3(sg), dim3(kSlowNT), 0, s, a);
    else hipLaunchKernelGGL((k_slow<SMW, MODE, false>), dim3(sg), dim3(kSlowNT), 0, s, a);
    if (MODE != kSparseWrite) timer_end(kTReduceSlow, s);
    return hipGetLastError();
}

// Workgroups of the tile pass that the current device holds at once (the
// fewest over the three modes), 0 if it cannot be queried.
template <int PMAX, bool QUANT>
int tiles_occupancy()
{
    constexpr int NT = Fast<PMAX>::NT;
    int best = 1 << 30, n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_tiles<PMAX, kCount, QUANT>, NT, 0) != hipSuccess)
        return 0;
    best = std::min(best, n);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_tiles<PMAX, kDense, QUANT>, NT, 0) != hipSuccess)
        return 0;
    best = std::min(best, n);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, k_tiles<PMAX, kSparseWrite, QUANT>, NT, 0) != hipSuccess)
        return 0;
    return std::min(best, n);
}

// Chunks of the tile pass: as many as workgroups fit on the device at once,
// so that the grid runs as a single wave of equal chunks.  Without a device
// (size queries on a host with no GPU) a fixed 512.
uint32_t resident_chunks(uint32_t pk, bool quant)
{
    // per device, rank class and value kind; 0 = not queried yet (a race
    // between threads only computes the same value twice)
    constexpr int kCacheDevs = 64;
    static std::atomic<uint32_t> cache[kCacheDevs][5][2];
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) {
        (void)hipGetLastError();
        return 512u;
    }
    const int cls = pk == 16 ? 0 : (pk == 32 ? 1 : (pk == 64 ? 2 : (pk == 128 ? 3 : 4)));
    std::atomic<uint32_t>* slot = dev >= 0 && dev < kCacheDevs ? &cache[dev][cls][quant ? 1 : 0] : nullptr;
    if (slot) {
        const uint32_t v = slot->load(std::memory_order_relaxed);
        if (v) return v;
    }
    int occ = 0;
    switch (pk) {
    case 16: occ = quant ? tiles_occupancy<16, true>() : tiles_occupancy<16, false>(); break;
    case 32: occ = quant ? tiles_occupancy<32, true>() : tiles_occupancy<32, false>(); break;
    case 64: occ = quant ? tiles_occupancy<64, true>() : tiles_occupancy<64, false>(); break;
    case 128: occ = quant ? tiles_occupancy<128, true>() : tiles_occupancy<128, false>(); break;
    default: occ = quant ? tiles_occupancy<256, true>() : tiles_occupancy<256, false>(); break;
    }
    if (occ <= 0) {
        (void)hipGetLastError();
        occ = 1;
    }
    const uint32_t n = (uint32_t)occ * (uint32_t)cus;
    if (slot) slot->store(n, std::memory_order_relaxed);
    return n;
}

template <int MODE>
hipError_t launch_pass(const Args& a, uint32_t pk, bool quant, hipStream_t s)
{
    switch (pk) {
    case 16: return launch_tiles_q<16, MODE>(a, quant, s);
    case 32: return launch_tiles_q<32, MODE>(a, quant, s);
    case 64: return launch_tiles_q<64, MODE>(a, quant, s);
    case 128: return launch_tiles_q<128, MODE>(a, quant, s);
    default: return launch_tiles_q<256, MODE>(a, quant, s);
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
    // stream offsets at the tile pass's chunks, or at the merge path's
    // segments; counters zeroed by the partition launch (either path's)
    l.off = c.take<uint32_t>((size_t)p.P * (std::max<uint32_t>(p.nchunks, kSegMax) + 1));
    l.zero = c.take<uint32_t>(std::max<size_t>((size_t)p.P + 1, kSegStateWords + 2 * (size_t)kSegMax));
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
                ReducePlan* plan, uint64_t lo)
{
    ReducePlan p{};
    p.lo = lo;
    p.P = (uint32_t)P;
    p.L = 0;
    while ((1u << p.L) < p.P) ++p.L;
    p.PK = p.P <= 16 ? 16u : (p.P <= 32 ? 32u : (p.P <= 64 ? 64u : (p.P <= 128 ? 128u : 256u)));
    // Tile size: fixed per rank class (the LDS layout of the tile pass).
    const uint64_t T = p.PK <= 32 ? 2048 : 4096;
    p.T = (uint32_t)T;
    p.N = N;
    p.ntiles = (uint32_t)((N + T - 1) / T);
    uint32_t nch = std::min<uint32_t>(p.ntiles, resident_chunks(p.PK, qbits != 0));
    p.tiles_per_chunk = (p.ntiles + nch - 1) / nch;
    p.nchunks = (p.ntiles + p.tiles_per_chunk - 1) / p.tiles_per_chunk;
    const double t = std::floor(delta * (double)N);
    p.thr = t >= 18446744073709551615.0 ? UINT64_MAX : (uint64_t)t;
    p.sum_nnz = sum_nnz;
    p.max_nnz = max_nnz;
    p.qbits = (uint32_t)qbits;
    p.speculate_dense = sum_nnz > p.thr ? 1 : 0;
    p.small = merge_small_fits(p.P, sum_nnz, p.thr) ? 1 : 0;
    p.seg = !p.small && merge_seg_fits(p.P, sum_nnz, p.thr) ? 1 : 0;
    p.nseg = 0;
    p.segw = 0;
    if (p.seg) merge_seg_shape(N, sum_nnz, &p.nseg, &p.segw);
    *plan = p;
    return 0;
}

size_t reduce_workspace(const ReducePlan& p) { return layout(p, nullptr).bytes; }

hipError_t set_result_run(ReduceResult* r, uint64_t nnz, uint32_t dense, hipStream_t s)
{
    hipLaunchKernelGGL(k_set_result, dim3(1), dim3(64), 0, s, r, nnz, dense);
    return hipGetLastError();
}

hipError_t reduce_run(const ReducePlan& p, const StreamDesc* host_tab, uint32_t* out_idx,
                      float* out_val, uint64_t* node_nnz, uint8_t* node_dense, void* ws,
                      hipStream_t s, ReduceResult* res, uint32_t nfold, ReduceResult* dev_result,
                      uint64_t out_cap)
{
    const Layout l = layout(p, ws);
    hipError_t e;
    if (p.small) {
        // few slots, every node sparse, few entries: one workgroup, one launch
        e = merge_small_run(p.P, p.L, p.qbits, nfold, host_tab, out_idx, out_val, node_nnz, node_dense, l.hdr,
                            dev_result, s);
        if (e != hipSuccess || dev_result) return e;
        if ((e = hipMemcpyAsync(res, l.hdr, sizeof(ReduceResult), hipMemcpyDeviceToHost, s)) != hipSuccess)
            return e;
        return hipStreamSynchronize(s);
    }
    // the descriptor table: in the partition launch's arguments when it fits
    // there (whole, or 5 words a stream when every stream's level unit
    // follows the previous one's), else uploaded first
    const size_t tab_bytes = sizeof(StreamDesc) * p.P;
    DescArgs tb;
    tb.nwords = 0;
    tb.fmt = kDescNone;
    tb.scale0 = nullptr;
    bool scales_follow = true;
    for (uint32_t r = 1; r < p.P && scales_follow; ++r) scales_follow = host_tab[r].qscale == host_tab[0].qscale + r;
    if (tab_bytes <= sizeof(tb.words)) {
        tb.fmt = kDescFull;
        tb.nwords = (uint32_t)(tab_bytes / 4);
        memcpy(tb.words, host_tab, tab_bytes);
    } else if (5u * p.P <= (uint32_t)kBlobWords && (!p.qbits || scales_follow)) {
        tb.fmt = p.qbits ? kDescCodes : kDescValues;
        tb.nwords = 5u * p.P;
        tb.scale0 = host_tab[0].qscale;
        for (uint32_t r = 0; r < p.P; ++r) {
            const uint64_t a = reinterpret_cast<uint64_t>(host_tab[r].idx);
            const uint64_t b = reinterpret_cast<uint64_t>(p.qbits ? static_cast<const void*>(host_tab[r].qval)
                                                                  : static_cast<const void*>(host_tab[r].val));
            uint32_t* w = tb.words + 5u * r;
            w[0] = (uint32_t)a;
            w[1] = (uint32_t)(a >> 32);
            w[2] = (uint32_t)b;
            w[3] = (uint32_t)(b >> 32);
            w[4] = (uint32_t)host_tab[r].nnz;
        }
    } else if ((e = upload(l.tab, host_tab, tab_bytes, s)) != hipSuccess) {
        return e;
    }
    // offsets of every stream at the tile pass's chunks (searches) or the
    // merge path's segments (one pass over the entries), and that path's
    // counters cleared
    if (p.seg) {
        const uint32_t nzero = kSegStateWords + 2u * p.nseg;
        const uint64_t nthreads = std::max<uint64_t>(p.max_nnz + 1u, std::max<uint32_t>(nzero, p.P));
        hipLaunchKernelGGL(k_partition_pass, dim3((uint32_t)((nthreads + 255) / 256), p.P), dim3(256), 0, s, l.tab,
                           tb, l.off, p.nseg, p.segw, p.lo, l.zero, nzero);
    } else {
        const uint32_t nzero = p.P + 1u;
        hipLaunchKernelGGL(k_partition, dim3(p.P), dim3(256), 0, s, l.tab, tb, l.off, p.nchunks,
                           (uint64_t)p.tiles_per_chunk * p.T, p.lo, p.N, l.zero, nzero);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;

    if (p.seg) {
        // every node sparse: the merge tree, one workgroup per segment
        SegState st;
        st.node_cnt = l.zero;
        st.ticket = l.zero + 64;
        st.done = l.zero + 65;
        st.err = l.zero + 66;
        st.flags = reinterpret_cast<unsigned long long*>(l.zero + kSegStateWords);
        e = merge_seg_run(p.P, p.L, p.qbits, nfold, l.tab, l.off, st, p.nseg, p.lo, p.segw, p.N, out_idx,
                          out_val, node_nnz, node_dense, l.hdr, dev_result, merge_seg_short(p.sum_nnz, p.nseg), s);
        if (e != hipSuccess || dev_result) return e;
        if ((e = hipMemcpyAsync(res, l.hdr, sizeof(ReduceResult), hipMemcpyDeviceToHost, s)) != hipSuccess)
            return e;
        return hipStreamSynchronize(s);  // res->pad nonzero: a look-back gave up (the caller reports it)
    }

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
    a.lo = (uint32_t)p.lo;
    a.T = p.T;
    a.ntiles = p.ntiles;
    a.nchunks = p.nchunks;
    a.tpc = p.tiles_per_chunk;
    a.qbits = p.qbits;
    a.out_vec = (reinterpret_cast<uintptr_t>(out_val) & 15u) == 0 ? 1u : 0u;
    a.out_cap = (uint32_t)std::min<uint64_t>(out_cap, 0xFFFFFFFFull);
    a.err_hdr = &l.hdr->pad;
    a.err_res = dev_result ? &dev_result->pad : nullptr;
    const bool quant = p.qbits != 0;

    e = p.speculate_dense ? launch_pass<kDense>(a, p.PK, quant, s)
                          : launch_pass<kCount>(a, p.PK, quant, s);
    if (e != hipSuccess) return e;
    // the switch rule, then (sparse root) the output offsets of the write pass
    hipLaunchKernelGGL(k_decide_scan, dim3(1), dim3(1024), 0, s, l.tab, l.node_cnt, p.P, p.N, p.thr,
                       node_nnz, node_dense, l.hdr, nfold, dev_result, l.tile_cnt, l.tile_off, p.ntiles,
                       l.slow_count);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    // the sparse-output passes return at once on the device when the root is
    // dense (the offsets are then not computed)
    a.skip = l.hdr;

    if (dev_result) return launch_pass<kSparseWrite>(a, p.PK, quant, s);  // no host round trip
    if (p.speculate_dense) {
        if ((e = hipMemcpyAsync(res, l.hdr, sizeof(ReduceResult), hipMemcpyDeviceToHost, s)) !=
            hipSuccess)
            return e;
        if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
        if (res->dense) return hipSuccess;
    }
    // Sparse root: write at the offsets from the per-tile union sizes.
    if ((e = launch_pass<kSparseWrite>(a, p.PK, quant, s)) != hipSuccess) return e;
    if ((e = hipMemcpyAsync(res, l.hdr, sizeof(ReduceResult), hipMemcpyDeviceToHost, s)) !=
        hipSuccess)
        return e;
    return hipStreamSynchronize(s);
}

}  // namespace sparcml
