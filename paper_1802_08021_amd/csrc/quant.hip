// QSGD stochastic quantization on gfx950 (§2.2 "Quantization", §6): one
// bucket per stream or buckets of B consecutive entries, scale = the
// bucket's L2 norm, s = 2^(bits-1)-1 levels plus a sign bit, unbiased
// stochastic rounding driven by Philox4x32-10.
//
// The norm is a fixed adjacent-pair tree in fp64 (zero-padded to a power of
// two), so it is reproducible bit for bit: 64 consecutive squares are summed
// by a lane butterfly, 32 such groups by a second butterfly, waves and
// blocks in tree order, and block partials by further aligned trees.
#include "internal.h"

#include <algorithm>

namespace sparcml {
namespace {

constexpr uint32_t kSeg = 8192;  // elements per first-level partial (256 threads)

struct QDesc {
    const float* val;
    uint8_t* q;
    float* deq;
    uint64_t n;
};

// Stream r's descriptor: from the launch's arguments (ARGS: six words a
// stream, val, q and n; no dequantized copy), else from the uploaded table.
// (A template parameter: chosen at run time, the two sources were merged by
// the compiler into one generic pointer and a vector load per workgroup;
// each instantiation now reads its own source with scalar loads.)
template <bool ARGS>
__device__ __forceinline__ QDesc qdesc(const QDesc* tab, const Blob& tb, uint32_t r)
{
    if (!ARGS) return tab[r];
    const uint32_t* w = tb.words + 6u * r;
    QDesc d;
    d.val = reinterpret_cast<const float*>((uint64_t)w[0] | (uint64_t)w[1] << 32);
    d.q = reinterpret_cast<uint8_t*>((uint64_t)w[2] | (uint64_t)w[3] << 32);
    d.deq = nullptr;
    d.n = (uint64_t)w[4] | (uint64_t)w[5] << 32;
    return d;
}

__device__ __forceinline__ double butterfly_sum(double v, int width)
{
    for (int o = 1; o < width; o <<= 1) v = v + __shfl_xor(v, o);
    return v;
}

// partial[r][b] = tree sum of v^2 over elements [b*kSeg, (b+1)*kSeg) of
// stream r (zeros past the end); with one block a stream (scale non-null)
// that is the norm^2, and scale[r] = its square root.  A wave covers 2048
// consecutive elements in eight steps of 256: each lane squares four
// consecutive elements and adds them pairwise, a lane butterfly joins the 64
// lanes' subtrees, and the eight step sums are joined pairwise at the end --
// the same adjacent-pair tree, with the eight independent butterflies in
// flight together.
// Tree sum of v^2 over the 2048 elements [base, base + 2048) (zeros past
// n) by one wave, in eight steps of 256: each lane squares four consecutive
// elements and adds them pairwise, a lane butterfly joins the 64 lanes'
// subtrees, and the eight step sums are joined pairwise at the end -- the
// adjacent-pair tree, with the eight independent butterflies in flight
// together.  STREAM: nontemporal loads (values not read again soon).
template <bool STREAM>
__device__ __forceinline__ double wave_sumsq(const float* v, uint64_t n, uint64_t base, int lane)
{
    const bool vec = (reinterpret_cast<uintptr_t>(v) & 15u) == 0;
    double part[8];
#pragma unroll
    for (int it = 0; it < 8; ++it) {
        const uint64_t e = base + (uint64_t)it * 256 + (uint64_t)lane * 4;
        float4 x;
        if (vec && e + 4 <= n) {
            x = STREAM ? load_nt(v + e) : *reinterpret_cast<const float4*>(v + e);
        } else {
            x.x = e < n ? v[e] : 0.0f;
            x.y = e + 1 < n ? v[e + 1] : 0.0f;
            x.z = e + 2 < n ? v[e + 2] : 0.0f;
            x.w = e + 3 < n ? v[e + 3] : 0.0f;
        }
        const double sq = ((double)x.x * (double)x.x + (double)x.y * (double)x.y) +
                          ((double)x.z * (double)x.z + (double)x.w * (double)x.w);
        part[it] = butterfly_sum(sq, 64);
    }
    return ((part[0] + part[1]) + (part[2] + part[3])) + ((part[4] + part[5]) + (part[6] + part[7]));
}

// partial[r][b] = tree sum of v^2 over elements [b*kSeg, (b+1)*kSeg) of
// stream r (zeros past the end), a wave per 2048 elements and the four
// wave sums pairwise; with one block a stream (scale non-null) that is the
// norm^2, and scale[r] = its square root.
template <bool ARGS>
__global__ void __launch_bounds__(256) k_sumsq_partial(const QDesc* tab, Blob tb, double* partial, uint32_t Q,
                                                       float* scale)
{
    __shared__ double s_w[4];
    const uint32_t r = blockIdx.y, b = blockIdx.x;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const QDesc d = qdesc<ARGS>(tab, tb, r);
    const double w = wave_sumsq<true>(d.val, d.n, (uint64_t)b * kSeg + (uint64_t)wv * 2048, lane);
    if (lane == 0) s_w[wv] = w;
    __syncthreads();
    if (threadIdx.x == 0) {
        const double t = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
        partial[(uint64_t)r * Q + b] = t;
        if (scale) scale[r] = (float)sqrt(t);
    }
}

// out[r][b] = tree sum of in[r][b*1024 .. b*1024+1024) (zeros past count);
// at the last level (scale non-null, one block a stream) also scale[r] =
// the square root of the norm^2.
__global__ void __launch_bounds__(1024) k_sum_f64(const double* in, uint32_t count, double* out,
                                                  uint32_t out_count, float* scale)
{
    __shared__ double s_w[16];
    const uint32_t r = blockIdx.y, b = blockIdx.x;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const uint32_t e = b * 1024 + threadIdx.x;
    const double x = e < count ? in[(uint64_t)r * count + e] : 0.0;
    const double w = butterfly_sum(x, 64);
    if (lane == 0) s_w[wv] = w;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t[16];
        for (int i = 0; i < 16; ++i) t[i] = s_w[i];
        for (int width = 16; width > 1; width >>= 1)
            for (int i = 0; i < width / 2; ++i) t[i] = t[2 * i] + t[2 * i + 1];
        out[(uint64_t)r * out_count + b] = t[0];
        if (scale) scale[r] = (float)sqrt(t[0]);
    }
}

// Philox4x32-10 (Salmon et al., SC'11): ten rounds of two 32x32->64
// multiplies with the high halves mixed into the other words and the key,
// the key advanced by the Weyl constants between rounds.
__device__ __forceinline__ uint4 philox(uint4 c, uint32_t k0, uint32_t k1)
{
#pragma unroll
    for (int i = 0; i < 10; ++i) {
        if (i) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        // full 64-bit products: one v_mad_u64_u32 each instead of a low and
        // a high multiply
        const uint64_t p0 = (uint64_t)0xD2511F53u * c.x, p1 = (uint64_t)0xCD9E8D57u * c.z;
        const uint32_t lo0 = (uint32_t)p0, hi0 = (uint32_t)(p0 >> 32);
        const uint32_t lo1 = (uint32_t)p1, hi1 = (uint32_t)(p1 >> 32);
        c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
    }
    return c;
}

// Elements e0 .. e0 + 32/BITS - 1 of stream r quantized into one 32-bit
// word of codes (4 elements per Philox block), the dequantized values
// stored too when the stream asks for them.
template <int BITS>
__device__ __forceinline__ void quant_word(const QDesc& d, uint32_t r, uint64_t e0, float scale, uint32_t k0,
                                           uint32_t k1)
{
    constexpr int EPT = 32 / BITS;
    constexpr uint32_t S = (1u << (BITS - 1)) - 1u;
    const float inv = scale > 0.0f ? __fdiv_rn((float)S, scale) : 0.0f;
    const float unit = __fdiv_rn(scale, (float)S);
    float x[EPT];
    const bool full = e0 + EPT <= d.n;
    if (full && ((reinterpret_cast<uintptr_t>(d.val + e0) & 15u) == 0)) {
#pragma unroll
        for (int i = 0; i < EPT; i += 4) {
            const float4 t = *reinterpret_cast<const float4*>(d.val + e0 + i);
            x[i] = t.x;
            x[i + 1] = t.y;
            x[i + 2] = t.z;
            x[i + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i) x[i] = e0 + i < d.n ? d.val[e0 + i] : 0.0f;
    }
    uint32_t word = 0;
#pragma unroll
    for (int g = 0; g < EPT; g += 4) {
        const uint64_t blk = (e0 + g) >> 2;
        const uint4 w4 = philox(make_uint4((uint32_t)blk, r, 0u, 0u), k0, k1);
        const uint32_t wr[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ii = g + i;
            uint32_t l = 0;
            if (scale > 0.0f) {
                const float a = __fmul_rn(fabsf(x[ii]), inv);
                l = (uint32_t)a;
                const float f = __fsub_rn(a, (float)l);
                const float u = (float)(wr[i] >> 8) * 0x1p-24f;
                l += u < f ? 1u : 0u;
                l = l > S ? S : l;
            }
            const uint32_t sign = (x[ii] < 0.0f && l > 0u) ? 1u : 0u;
            const uint32_t code = (sign << (BITS - 1)) | l;
            word |= code << (ii * BITS);
            if (d.deq && e0 + ii < d.n) {
                const float mag = __fmul_rn((float)l, unit);
                d.deq[e0 + ii] = l == 0u ? 0.0f : (sign ? -mag : mag);
            }
        }
    }
    const uint64_t byte0 = e0 * BITS / 8;
    const uint64_t nbytes = (d.n * BITS + 7) / 8;
    if (byte0 + 4 <= nbytes && ((reinterpret_cast<uintptr_t>(d.q + byte0) & 3u) == 0)) {
        *reinterpret_cast<uint32_t*>(d.q + byte0) = word;
    } else {
        for (int i = 0; i < 4; ++i)
            if (byte0 + i < nbytes) d.q[byte0 + i] = (uint8_t)(word >> (8 * i));
    }
}

// Each thread quantizes 32/bits consecutive elements into one word.
template <int BITS, bool ARGS>
__global__ void __launch_bounds__(256) k_quantize(const QDesc* tab, Blob tb, const float* scales, uint32_t k0,
                                                  uint32_t k1)
{
    constexpr int EPT = 32 / BITS;
    const uint32_t r = blockIdx.y;
    const QDesc d = qdesc<ARGS>(tab, tb, r);
    const uint64_t e0 = ((uint64_t)blockIdx.x * 256 + threadIdx.x) * EPT;
    if (e0 >= d.n) return;
    quant_word<BITS>(d, r, e0, scales[r], k0, k1);
}

// Streams of at most kSmallQ elements: one 1024-thread workgroup a stream
// takes both passes, one launch instead of three.  Waves 4b..4b+3 sum block
// b's squares as k_sumsq_partial does, the four block partials are joined
// pairwise (the tree k_sum_f64 forms over them: the partials of blocks past
// the stream are +0.0, and adding +0.0 is exact), then the workgroup codes
// the stream as k_quantize does (its values read again, now from the cache).
constexpr uint64_t kSmallQ = 4 * kSeg;

template <int BITS, bool ARGS>
__global__ void __launch_bounds__(1024) k_quant_small(const QDesc* tab, Blob tb, float* scales, uint32_t k0,
                                                      uint32_t k1)
{
    constexpr int EPT = 32 / BITS;
    __shared__ double s_w[16];
    __shared__ float s_scale;
    const uint32_t r = blockIdx.x;
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const QDesc d = qdesc<ARGS>(tab, tb, r);
    const double w = wave_sumsq<false>(d.val, d.n, (uint64_t)(wv >> 2) * kSeg + (uint64_t)(wv & 3) * 2048, lane);
    if (lane == 0) s_w[wv] = w;
    __syncthreads();
    if (threadIdx.x == 0) {
        double p[4];
#pragma unroll
        for (int b = 0; b < 4; ++b) p[b] = (s_w[4 * b] + s_w[4 * b + 1]) + (s_w[4 * b + 2] + s_w[4 * b + 3]);
        const float sc = (float)sqrt((p[0] + p[1]) + (p[2] + p[3]));
        scales[r] = sc;
        s_scale = sc;
    }
    __syncthreads();
    const float scale = s_scale;
    for (uint64_t e0 = (uint64_t)threadIdx.x * EPT; e0 < d.n; e0 += 1024u * EPT)
        quant_word<BITS>(d, r, e0, scale, k0, k1);
}

// Bucketed QSGD in one pass: a bucket of B (a power of two, 4..8192)
// consecutive entries is held in the registers of G = B / EPT consecutive
// threads, EPT = max(4, B / 256) consecutive entries each.  Its norm is the
// adjacent-pair tree in fp64: each thread's EPT squares, then a lane
// butterfly over min(G, 64) lanes, then (G > 64) the waves' sums pairwise.
// The codes are drawn as in the per-stream scheme (Philox word j&3 of
// counter (j>>2, r, 0, 0) for element j of stream r) and written once.
struct QBDesc {
    const float* val;
    uint8_t* q;
    float* deq;
    uint64_t n;
    uint64_t soff;  // index of the stream's first scale
};

template <int BITS, int EPT>
__global__ void __launch_bounds__(256) k_quantize_buckets(const QBDesc* tab, float* scales, uint32_t B,
                                                          uint32_t k0, uint32_t k1)
{
    constexpr uint32_t S = (1u << (BITS - 1)) - 1u;
    __shared__ double s_w[4];
    const uint32_t r = blockIdx.y;
    const QBDesc d = tab[r];
    const uint64_t blk0 = (uint64_t)blockIdx.x * 256 * EPT;
    if (blk0 >= d.n) return;  // uniform over the block
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const uint32_t G = B / EPT;  // threads per bucket (1..256)
    const uint64_t e0 = blk0 + (uint64_t)threadIdx.x * EPT;

    float x[EPT];
    const bool full = e0 + EPT <= d.n;
    if (full && ((reinterpret_cast<uintptr_t>(d.val + e0) & 15u) == 0)) {
#pragma unroll
        for (int i = 0; i < EPT; i += 4) {
            const float4 t = *reinterpret_cast<const float4*>(d.val + e0 + i);
            x[i] = t.x;
            x[i + 1] = t.y;
            x[i + 2] = t.z;
            x[i + 3] = t.w;
        }
    } else {
#pragma unroll
        for (int i = 0; i < EPT; ++i) x[i] = e0 + i < d.n ? d.val[e0 + i] : 0.0f;
    }
    double t[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) t[i] = (double)x[i] * (double)x[i];
#pragma unroll
    for (int w = EPT; w > 1; w >>= 1)
#pragma unroll
        for (int i = 0; i < w / 2; ++i) t[i] = t[2 * i] + t[2 * i + 1];
    double sum = t[0];
    const int width = G < 64u ? (int)G : 64;
    for (int o = 1; o < width; o <<= 1) sum = sum + __shfl_xor(sum, o);
    if (G > 64u) {  // (uniform) a bucket spans two or four waves
        if (lane == 0) s_w[wv] = sum;
        __syncthreads();
        if (G == 128u) sum = (wv < 2) ? s_w[0] + s_w[1] : s_w[2] + s_w[3];
        else sum = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
    }
    const float scale = (float)sqrt(sum);
    if (e0 % B == 0 && e0 < d.n) scales[d.soff + e0 / B] = scale;

    const float inv = scale > 0.0f ? __fdiv_rn((float)S, scale) : 0.0f;
    const float unit = __fdiv_rn(scale, (float)S);
    constexpr int NW = (EPT * BITS + 31) / 32;  // code words of this thread
    uint32_t word[NW];
#pragma unroll
    for (int w = 0; w < NW; ++w) word[w] = 0u;
#pragma unroll
    for (int g = 0; g < EPT; g += 4) {
        const uint4 w4 = philox(make_uint4((uint32_t)((e0 + g) >> 2), r, 0u, 0u), k0, k1);
        const uint32_t wr[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int ii = g + i;
            uint32_t l = 0;
            if (scale > 0.0f) {
                const float a = __fmul_rn(fabsf(x[ii]), inv);
                l = (uint32_t)a;
                const float f = __fsub_rn(a, (float)l);
                const float u = (float)(wr[i] >> 8) * 0x1p-24f;
                l += u < f ? 1u : 0u;
                l = l > S ? S : l;
            }
            const uint32_t sign = (x[ii] < 0.0f && l > 0u) ? 1u : 0u;
            const uint32_t code = (sign << (BITS - 1)) | l;
            word[(ii * BITS) / 32] |= code << ((ii * BITS) % 32);
            if (d.deq && e0 + ii < d.n) {
                const float mag = __fmul_rn((float)l, unit);
                d.deq[e0 + ii] = l == 0u ? 0.0f : (sign ? -mag : mag);
            }
        }
    }
    // EPT * BITS / 8 bytes of codes at byte e0 * BITS / 8
    constexpr int NB = EPT * BITS / 8;
    const uint64_t byte0 = e0 * BITS / 8;
    const uint64_t nbytes = (d.n * BITS + 7) / 8;
    uint8_t* q = d.q + byte0;
    if (NB >= 4 && byte0 + NB <= nbytes && ((reinterpret_cast<uintptr_t>(q) & 3u) == 0)) {
#pragma unroll
        for (int w = 0; w < NW; ++w) reinterpret_cast<uint32_t*>(q)[w] = word[w];
    } else if (NB == 2 && byte0 + 2 <= nbytes && ((reinterpret_cast<uintptr_t>(q) & 1u) == 0)) {
        *reinterpret_cast<uint16_t*>(q) = (uint16_t)word[0];
    } else {
#pragma unroll
        for (int i = 0; i < NB; ++i)
            if (byte0 + i < nbytes) q[i] = (uint8_t)(word[i / 4] >> (8 * (i % 4)));
    }
}

struct QLayout {
    QDesc* tab;
    double* part[4];
    uint32_t count[4];
    int levels;
    double* norm2;
    size_t bytes;
};

QLayout qlayout(int P, uint64_t max_n, void* ws)
{
    Carve c(ws);
    QLayout l{};
    l.tab = c.take<QDesc>(P);
    uint64_t cnt = std::max<uint64_t>(1, (max_n + kSeg - 1) / kSeg);
    l.levels = 0;
    l.count[0] = (uint32_t)cnt;
    l.part[0] = c.take<double>((size_t)P * cnt);
    while (cnt > 1) {
        cnt = (cnt + 1023) / 1024;
        ++l.levels;
        l.count[l.levels] = (uint32_t)cnt;
        l.part[l.levels] = c.take<double>((size_t)P * cnt);
    }
    l.norm2 = l.part[l.levels];
    l.bytes = align_up(c.used, 256);
    return l;
}

template <int BITS>
void launch_buckets(dim3 grid, int ept, hipStream_t s, const QBDesc* tab, float* scales, uint32_t B,
                    uint32_t k0, uint32_t k1)
{
    switch (ept) {
    case 4: hipLaunchKernelGGL((k_quantize_buckets<BITS, 4>), grid, dim3(256), 0, s, tab, scales, B, k0, k1); break;
    case 8: hipLaunchKernelGGL((k_quantize_buckets<BITS, 8>), grid, dim3(256), 0, s, tab, scales, B, k0, k1); break;
    case 16: hipLaunchKernelGGL((k_quantize_buckets<BITS, 16>), grid, dim3(256), 0, s, tab, scales, B, k0, k1); break;
    default: hipLaunchKernelGGL((k_quantize_buckets<BITS, 32>), grid, dim3(256), 0, s, tab, scales, B, k0, k1); break;
    }
}

}  // namespace

size_t quant_workspace(int P, uint64_t max_n) { return qlayout(P, max_n, nullptr).bytes; }

size_t quant_buckets_workspace(int P) { return align_up(sizeof(QBDesc) * (size_t)P, 256); }

hipError_t quant_buckets_run(int P, const float* const* vals, const uint64_t* n, int bits,
                             uint32_t bucket, uint64_t seed, uint8_t* const* out_q, float* out_scale,
                             float* const* out_deq, void* ws, hipStream_t s)
{
    uint64_t max_n = 0, soff = 0;
    QBDesc* host = new QBDesc[P];
    for (int r = 0; r < P; ++r) {
        host[r] = QBDesc{vals[r], out_q[r], out_deq ? out_deq[r] : nullptr, n[r], soff};
        soff += (n[r] + bucket - 1) / bucket;
        max_n = std::max(max_n, n[r]);
    }
    QBDesc* tab = static_cast<QBDesc*>(ws);
    hipError_t e = upload(tab, host, sizeof(QBDesc) * P, s);
    delete[] host;
    if (e != hipSuccess || max_n == 0) return e;
    const int ept = bucket <= 1024u ? 4 : (int)(bucket / 256u);
    const uint64_t per_block = 256ull * ept;
    const dim3 grid((uint32_t)((max_n + per_block - 1) / per_block), P);
    const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
    timer_begin(kTQuantCodes, s);
    if (bits == 2) launch_buckets<2>(grid, ept, s, tab, out_scale, bucket, k0, k1);
    else if (bits == 4) launch_buckets<4>(grid, ept, s, tab, out_scale, bucket, k0, k1);
    else launch_buckets<8>(grid, ept, s, tab, out_scale, bucket, k0, k1);
    timer_end(kTQuantCodes, s);
    return hipGetLastError();
}

hipError_t quant_run(int P, const float* const* vals, const uint64_t* n, int bits, uint64_t seed,
                     uint8_t* const* out_q, float* out_scale, float* const* out_deq, void* ws,
                     hipStream_t s)
{
    uint64_t max_n = 0;
    for (int r = 0; r < P; ++r) max_n = std::max(max_n, n[r]);
    const QLayout l = qlayout(P, max_n, ws);
    // the descriptor table: in both launches' arguments when it fits there
    // (no dequantized copies), else uploaded first
    Blob tb;
    tb.nwords = 0;
    hipError_t e = hipSuccess;
    if (!out_deq && 6u * (uint32_t)P <= (uint32_t)kBlobWords) {
        tb.nwords = 6u * (uint32_t)P;
        for (int r = 0; r < P; ++r) {
            const uint64_t a = reinterpret_cast<uint64_t>(vals[r]), b = reinterpret_cast<uint64_t>(out_q[r]);
            uint32_t* w = tb.words + 6 * r;
            w[0] = (uint32_t)a;
            w[1] = (uint32_t)(a >> 32);
            w[2] = (uint32_t)b;
            w[3] = (uint32_t)(b >> 32);
            w[4] = (uint32_t)n[r];
            w[5] = (uint32_t)(n[r] >> 32);
        }
    } else {
        QDesc* host = new QDesc[P];
        for (int r = 0; r < P; ++r)
            host[r] = QDesc{vals[r], out_q[r], out_deq ? out_deq[r] : nullptr, n[r]};
        e = upload(l.tab, host, sizeof(QDesc) * P, s);
        delete[] host;
        if (e != hipSuccess) return e;
    }

    const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
    if (max_n > 0 && max_n <= kSmallQ) {  // short streams: norm and codes in one launch
        timer_begin(kTQuantCodes, s);
        const dim3 g((uint32_t)P), blk(1024);
        if (tb.nwords) {
            if (bits == 2) hipLaunchKernelGGL((k_quant_small<2, true>), g, blk, 0, s, l.tab, tb, out_scale, k0, k1);
            else if (bits == 4) hipLaunchKernelGGL((k_quant_small<4, true>), g, blk, 0, s, l.tab, tb, out_scale, k0, k1);
            else hipLaunchKernelGGL((k_quant_small<8, true>), g, blk, 0, s, l.tab, tb, out_scale, k0, k1);
        } else {
            if (bits == 2) hipLaunchKernelGGL((k_quant_small<2, false>), g, blk, 0, s, l.tab, tb, out_scale, k0, k1);
            else if (bits == 4) hipLaunchKernelGGL((k_quant_small<4, false>), g, blk, 0, s, l.tab, tb, out_scale, k0, k1);
            else hipLaunchKernelGGL((k_quant_small<8, false>), g, blk, 0, s, l.tab, tb, out_scale, k0, k1);
        }
        timer_end(kTQuantCodes, s);
        return hipGetLastError();
    }
    // norms; the launch that finishes a stream's norm also writes its scale
    timer_begin(kTQuantNorm, s);
    float* const scale0 = l.levels == 0 ? out_scale : nullptr;
    if (tb.nwords)
        hipLaunchKernelGGL(k_sumsq_partial<true>, dim3(l.count[0], P), dim3(256), 0, s, l.tab, tb, l.part[0],
                           l.count[0], scale0);
    else
        hipLaunchKernelGGL(k_sumsq_partial<false>, dim3(l.count[0], P), dim3(256), 0, s, l.tab, tb, l.part[0],
                           l.count[0], scale0);
    timer_end(kTQuantNorm, s);
    for (int lv = 1; lv <= l.levels; ++lv)
        hipLaunchKernelGGL(k_sum_f64, dim3(l.count[lv], P), dim3(1024), 0, s, l.part[lv - 1],
                           l.count[lv - 1], l.part[lv], l.count[lv], lv == l.levels ? out_scale : nullptr);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (max_n == 0) return hipSuccess;
    const uint64_t per_block = 256ull * (32 / bits);
    const dim3 grid((uint32_t)((max_n + per_block - 1) / per_block), P);
    timer_begin(kTQuantCodes, s);
    if (tb.nwords) {
        if (bits == 2) hipLaunchKernelGGL((k_quantize<2, true>), grid, dim3(256), 0, s, l.tab, tb, out_scale, k0, k1);
        else if (bits == 4) hipLaunchKernelGGL((k_quantize<4, true>), grid, dim3(256), 0, s, l.tab, tb, out_scale, k0, k1);
        else hipLaunchKernelGGL((k_quantize<8, true>), grid, dim3(256), 0, s, l.tab, tb, out_scale, k0, k1);
    } else {
        if (bits == 2) hipLaunchKernelGGL((k_quantize<2, false>), grid, dim3(256), 0, s, l.tab, tb, out_scale, k0, k1);
        else if (bits == 4) hipLaunchKernelGGL((k_quantize<4, false>), grid, dim3(256), 0, s, l.tab, tb, out_scale, k0, k1);
        else hipLaunchKernelGGL((k_quantize<8, false>), grid, dim3(256), 0, s, l.tab, tb, out_scale, k0, k1);
    }
    timer_end(kTQuantCodes, s);
    return hipGetLastError();
}

}  // namespace sparcml
