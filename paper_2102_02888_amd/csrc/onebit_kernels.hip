// gfx950 kernels of the 1-bit Adam hot path (arXiv 2102.02888).
//
// Every kernel streams over the flat parameter buffer and, except for the
// chunk owners' decode-and-average (bound by vector ALU issue), is bound by
// HBM bandwidth; no MFMA (nothing here is a dense contraction).  Work is cut
// into tiles of up to 1024 elements that never cross a segment; one
// wavefront (64 lanes) owns one tile, each lane holding 4 sub-blocks x float4
// = 16 elements (in the packed worker pass two waves share a tile, 2
// sub-blocks each), so every global load/store is a 128-bit access and a
// wave moves 1 KiB per instruction.  A sub-block of 256 elements spans four 16-lane DPP rows, and
// each row's 64 elements form one LSB-first uint64 sign word (bit b of word w
// of the tile <=> element 64w+b), assembled with a row-wide OR of the lanes'
// 4-bit nibbles.
//
// Arithmetic contract (shared with the layout/format description in
// onebit.h): fp32 values, one rounding per operation (built with
// -ffp-contract=off), correctly rounded sqrt and division, fp64 reductions
// rounded once to fp32.  Reductions over a segment are deterministic:
// per-tile partial sums (a fixed lane reduction order) are written to a
// workspace and summed in a fixed order by a finalize kernel; no atomics.
#include "onebit_internal.h"
#include <algorithm>
#include <mutex>

namespace onebit {
namespace {

// Four consecutive floats.  The native vector type lets the non-temporal
// builtins take it; every stream here is touched once per launch, so loads
// and stores are non-temporal (they do not displace other data in the caches
// on the way to HBM).
typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
typedef uint32_t v2u32 __attribute__((ext_vector_type(2)));

// Full tiles move through raw buffer instructions: the base sits in scalar
// registers and each lane adds a 32-bit byte offset, and the cache policy is
// an operand.  Loads are non-temporal (nt); stores are non-temporal at device
// scope (nt and sc1), which drains the streams of written state to HBM faster
// than nt alone.  The resource covers 2 GiB from the base, far more than a
// tile; its fourth word is the gfx9-family buffer format word.
constexpr int kStreamLoad = 2;        // nt
constexpr int kStreamStore = 2 | 16;  // nt, sc1

// Resource for a wave-uniform base p (a tile's start in some row: every
// caller's p is the same in all lanes).  p is read from the first active lane,
// so the base stays in scalar registers even where the compiler holds it in
// vector registers, with no per-access loop over distinct lane values.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t stream_rsrc(const void *p)
{
    const uint64_t a = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0,
                                             0x7FFFFFFF, 0x00020000);
}

// Loads elements li..li+3 of p; FULL means the whole tile is in range (a
// wave-uniform fact), otherwise lanes past len read zeros.
template <bool FULL>
__device__ __forceinline__ v4f ld4(const float *__restrict__ p, int li, int len)
{
    if (FULL)
        return __builtin_bit_cast(
            v4f, __builtin_amdgcn_raw_buffer_load_b128(stream_rsrc(p), li * 4, 0, kStreamLoad));
    if (li + 4 <= len) return __builtin_nontemporal_load((const v4f *)(p + li));
    v4f r = {0.f, 0.f, 0.f, 0.f};
    if (li < len) r.x = p[li];
    if (li + 1 < len) r.y = p[li + 1];
    if (li + 2 < len) r.z = p[li + 2];
    return r;
}

// Stores elements li..li+3 of p.  Full tiles store non-temporally; partial
// tiles store plainly (lanes past len store nothing), because their waves
// may still load after storing.
template <bool FULL>
__device__ __forceinline__ void st4(float *__restrict__ p, int li, int len, v4f v)
{
    if (FULL) {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, v), stream_rsrc(p),
                                               li * 4, 0, kStreamStore);
        return;
    }
    if (li + 4 <= len) {
        *(v4f *)(p + li) = v;
        return;
    }
    if (li < len) p[li] = v.x;
    if (li + 1 < len) p[li + 1] = v.y;
    if (li + 2 < len) p[li + 2] = v.z;
}

// Gradient element types.  16-bit gradients are widened to fp32 exactly
// (bf16 by a 16-bit shift, fp16 by the hardware conversion), so the method's
// arithmetic is the same as for fp32 gradients of those values.
struct GradF32 {
    using T = float;
};
struct GradBF16 {
    using T = uint16_t;
};
struct GradF16 {
    using T = _Float16;
};

__device__ __forceinline__ float widen(uint16_t a) { return __uint_as_float((uint32_t)a << 16); }
__device__ __forceinline__ float widen(_Float16 a) { return (float)a; }

typedef uint16_t v4u16 __attribute__((ext_vector_type(4)));
typedef _Float16 v4f16 __attribute__((ext_vector_type(4)));

// Gradient elements li..li+3 as fp32 (zeros past len when !FULL).
template <bool FULL, class G>
__device__ __forceinline__ v4f ldg4(const typename G::T *__restrict__ p, int li, int len)
{
    if constexpr (sizeof(typename G::T) == 4) {
        return ld4<FULL>((const float *)p, li, len);
    } else {
        v4f r = {0.f, 0.f, 0.f, 0.f};
        if (FULL || li + 4 <= len) {
            const v2u32 w =
                FULL ? __builtin_amdgcn_raw_buffer_load_b64(stream_rsrc(p), li * 2, 0, kStreamLoad)
                     : __builtin_nontemporal_load((const v2u32 *)(p + li));
            if constexpr (__is_same(typename G::T, uint16_t)) {
                const v4u16 h = __builtin_bit_cast(v4u16, w);
#pragma unroll
                for (int c = 0; c < 4; ++c) r[c] = widen((uint16_t)h[c]);
            } else {
                const v4f16 h = __builtin_bit_cast(v4f16, w);
#pragma unroll
                for (int c = 0; c < 4; ++c) r[c] = widen((_Float16)h[c]);
            }
            return r;
        }
        if (li < len) r.x = widen(p[li]);
        if (li + 1 < len) r.y = widen(p[li + 1]);
        if (li + 2 < len) r.z = widen(p[li + 2]);
        return r;
    }
}

// OR of a 32-bit value over the 16 lanes of each DPP row (every lane of the
// row receives the result).  xor-1 and xor-2 quad permutes OR each quad; the
// row rotations by 4 and by 8 then OR the four quads, whichever way the
// rotation turns.
__device__ __forceinline__ uint32_t row_or16(uint32_t v)
{
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);   // quad_perm 1,0,3,2
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);   // quad_perm 2,3,0,1
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x124, 0xF, 0xF, false);  // row_ror 4
    v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x128, 0xF, 0xF, false);  // row_ror 8
    return v;
}

// Sign word of 64 consecutive elements held by one 16-lane row, 4 per lane:
// lane L of the row contributes its 4 sign bits (nib, element 4L+c at bit c)
// at bit positions 4L..4L+3.  Every lane of the row receives the word.
__device__ __forceinline__ uint64_t row_sign_word(uint32_t nib, int lane)
{
    const int r = lane & 15;
    const uint32_t lo = r < 8 ? nib << (4 * r) : 0u;
    const uint32_t hi = r >= 8 ? nib << (4 * (r - 8)) : 0u;
    return ((uint64_t)row_or16(hi) << 32) | (uint64_t)row_or16(lo);
}

// DPP move of an fp64 value (both 32-bit halves); lanes the pattern does not
// reach get 0.0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double dpp_f64(double v)
{
    const int lo = __builtin_amdgcn_update_dpp(0, __double2loint(v), CTRL, ROW_MASK, 0xF, false);
    const int hi = __builtin_amdgcn_update_dpp(0, __double2hiint(v), CTRL, ROW_MASK, 0xF, false);
    return __hiloint2double(hi, lo);
}

// Deterministic wave-wide fp64 sums (every lane gets the same value).
// wave_sum: xor butterfly through lane shuffles (cross-lane traffic goes
// through the LDS crossbar, off the vector ALU).
__device__ __forceinline__ double wave_sum(double a)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) a += __shfl_xor(a, off, kWave);
    return a;
}

// wave_sum_dpp: a fixed tree of DPP row shifts and row broadcasts read from
// lane 63; fewer instructions, but six dependent vector steps.  The worker
// pass (short waves, bound by memory latency) measured ~0.6% slower with it,
// the ALU-bound chunk-owner pass faster.
__device__ __forceinline__ double wave_sum_dpp(double a)
{
    a += dpp_f64<0x111, 0xF>(a);  // row_shr 1
    a += dpp_f64<0x112, 0xF>(a);  // row_shr 2
    a += dpp_f64<0x114, 0xF>(a);  // row_shr 4
    a += dpp_f64<0x118, 0xF>(a);  // row_shr 8
    a += dpp_f64<0x142, 0xA>(a);  // row_bcast 15
    a += dpp_f64<0x143, 0xC>(a);  // row_bcast 31
    const int lo = __builtin_amdgcn_readlane(__double2loint(a), kWave - 1);
    const int hi = __builtin_amdgcn_readlane(__double2hiint(a), kWave - 1);
    return __hiloint2double(hi, lo);
}

// This block's logical number in a grid launched by xcd_grid (one contiguous
// eighth of the logical blocks per XCD).
__device__ __forceinline__ int64_t xcd_block() { return xcd_block_of(blockIdx.x, gridDim.x); }

// This wave's number within its workgroup, as a wave-uniform (scalar) value,
// so that tile indices, tile descriptors and the addresses derived from them
// stay in scalar registers.  The chunk owners' kernels use it; the streaming
// kernels keep the plain form, since with the scalar one the compiler spills
// their scalar registers (their buffer bases are made uniform by stream_rsrc).
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// Error from the compensated form: z - C[z] given z and its segment scale s.
__device__ __forceinline__ float error_of(float z, float s) { return z >= 0.f ? z - s : z + s; }

// ---------------------------------------------------------------------------
// Warm-up Adam (eq. (alg:v)) on the average of n_grads gradient rows.
//
// The row-summing kernels (this one and the 32-bit comparison step) give the
// 16 waves of a workgroup 16 consecutive tiles and read each gradient row
// together, with a workgroup barrier after every row: each row is then
// streamed in 64 KB runs rather than in 16 independent 4 KB pieces.  Waves
// without a tile keep the pace.  Every wave of a workgroup runs the same row
// loop, so every wave reaches every barrier.
// ---------------------------------------------------------------------------
// One gradient row of the tile as fp32 (zeros past the tile when !FULL).
template <bool FULL, class G>
__device__ __forceinline__ void load_grad_row(v4f (&gv)[kSubBlocks],
                                              const typename G::T *__restrict__ row, int lane,
                                              int len)
{
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) gv[b] = ldg4<FULL, G>(row, b * (kWave * 4) + 4 * lane, len);
}

// sum += one loaded gradient row (fp64, rows added in row order)
__device__ __forceinline__ void add_grad_row(double (&sum)[kSubBlocks][4],
                                             const v4f (&gv)[kSubBlocks])
{
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[b][c] += (double)gv[b][c];
}

// sum = the n gradient rows of the tile, added in row order, with a
// workgroup barrier after every row; every wave runs the same number of
// barriers (active: the wave has a tile).  Issuing row i+1's loads before
// adding row i measured the same (8.79 against 8.74 ms on the BERT-Large
// shape, same buffers), and without the barriers the pass is 6% slower.
template <bool FULL, class G>
__device__ __forceinline__ void warmup_rows_walk(double (&sum)[kSubBlocks][4], const Tile &tile,
                                                 int lane, bool active,
                                                 const typename G::T *__restrict__ g,
                                                 int64_t g_ld, int n)
{
    for (int i = 0; i < n; ++i) {
        if (active) {
            v4f gv[kSubBlocks];
            load_grad_row<FULL, G>(gv, g + tile.start + (int64_t)i * g_ld, lane, tile.len);
            add_grad_row(sum, gv);
        }
        __builtin_amdgcn_s_barrier();  // the workgroup reads each row together
    }
}

// Adam on the averaged gradient sum / n; loads of x, m, v precede the stores.
template <bool FULL>
__device__ __forceinline__ void warmup_update(const double (&sum)[kSubBlocks][4], int64_t base,
                                              int len, int lane, float *__restrict__ x,
                                              float *__restrict__ m, float *__restrict__ v,
                                              double dn, float lr, float beta1, float omb1,
                                              float beta2, float omb2, float eps, int use_bc,
                                              float bc1, float bc2)
{
    v4f xv[kSubBlocks], mv[kSubBlocks], vv[kSubBlocks];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        xv[b] = ld4<FULL>(x + base, li, len);
        mv[b] = ld4<FULL>(m + base, li, len);
        vv[b] = ld4<FULL>(v + base, li, len);
    }
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float gbar = (float)(sum[b][c] / dn);
            float mn = beta1 * mv[b][c];
            mn = mn + omb1 * gbar;
            const float gsq = gbar * gbar;
            float vn = beta2 * vv[b][c];
            vn = vn + omb2 * gsq;
            float mh = mn, vh = vn;
            if (use_bc) {
                mh = mn / bc1;
                vh = vn / bc2;
            }
            const float denom = __builtin_sqrtf(vh) + eps;
            const float ratio = mh / denom;
            const float step = lr * ratio;
            xv[b][c] = xv[b][c] - step;
            mv[b][c] = mn;
            vv[b][c] = vn;
        }
        st4<FULL>(x + base, li, len, xv[b]);
        st4<FULL>(m + base, li, len, mv[b]);
        st4<FULL>(v + base, li, len, vv[b]);
    }
}

// ---------------------------------------------------------------------------
// Adam step whose gradient is a decoded message (g = bit ? scale : -scale);
// the "Adam(1-bit Naive)" comparison variant of Section 7.2 updates m and v
// from the compressed gradient this way.  Loads first, then stores.
// ---------------------------------------------------------------------------
template <bool FULL, int SB>
__device__ __forceinline__ void adam_message_tile(const Tile &tile, int lane, int sb0,
                                                  const uint64_t *__restrict__ bits, float s,
                                                  float *__restrict__ x, float *__restrict__ m,
                                                  float *__restrict__ v, float lr, float beta1,
                                                  float omb1, float beta2, float omb2,
                                                  float eps, int use_bc, float bc1, float bc2)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    uint64_t word[SB];
    v4f xv[SB], mv[SB], vv[SB];
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int sb = sb0 + b;
        const int li = sb * (kWave * 4) + 4 * lane;
        word[b] = (FULL || li < len) ? bits[(base >> 6) + 4 * sb + (lane >> 4)] : 0ull;
        xv[b] = ld4<FULL>(x + base, li, len);
        mv[b] = ld4<FULL>(m + base, li, len);
        vv[b] = ld4<FULL>(v + base, li, len);
    }
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int li = (sb0 + b) * (kWave * 4) + 4 * lane;
        const uint32_t nib = (uint32_t)(word[b] >> (4 * (lane & 15))) & 0xFu;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float gbar = ((nib >> c) & 1u) ? s : -s;
            float mn = beta1 * mv[b][c];
            mn = mn + omb1 * gbar;
            const float gsq = gbar * gbar;
            float vn = beta2 * vv[b][c];
            vn = vn + omb2 * gsq;
            float mh = mn, vh = vn;
            if (use_bc) {
                mh = mn / bc1;
                vh = vn / bc2;
            }
            const float denom = __builtin_sqrtf(vh) + eps;
            const float ratio = mh / denom;
            const float step = lr * ratio;
            xv[b][c] = xv[b][c] - step;
            mv[b][c] = mn;
            vv[b][c] = vn;
        }
        st4<FULL>(x + base, li, len, xv[b]);
        st4<FULL>(m + base, li, len, mv[b]);
        st4<FULL>(v + base, li, len, vv[b]);
    }
}

// One 256-element sub-block per wave, four waves per tile, as in the update
// (fewer bytes in flight per wave).
constexpr int kAdamMessageSubBlocks = 1;
constexpr int kAdamMessageWavesPerTile = kSubBlocks / kAdamMessageSubBlocks;

__global__ __launch_bounds__(kBlock) void k_adam_message(
    const Tile *__restrict__ tiles, int64_t num_tiles, const uint64_t *__restrict__ bits,
    const float *__restrict__ scales, float *__restrict__ x, float *__restrict__ m,
    float *__restrict__ v, float lr, float beta1, float omb1, float beta2, float omb2, float eps,
    int use_bc, float bc1, float bc2)
{
    constexpr int SB = kAdamMessageSubBlocks;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t w = xcd_block() * kWavesPerBlock + (threadIdx.x >> 6);
    const int64_t t = w / kAdamMessageWavesPerTile;
    const int sb0 = (int)(w % kAdamMessageWavesPerTile) * SB;
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const float s = scales[tile.seg];
    if (tile.len == kTileElems)
        adam_message_tile<true, SB>(tile, lane, sb0, bits, s, x, m, v, lr, beta1, omb1, beta2,
                                    omb2, eps, use_bc, bc1, bc2);
    else
        adam_message_tile<false, SB>(tile, lane, sb0, bits, s, x, m, v, lr, beta1, omb1, beta2,
                                     omb2, eps, use_bc, bc1, bc2);
}

// ---------------------------------------------------------------------------
// "1-bit Adam (32-bits)" comparison variant (Section 7.2): the compression
// stage with the identity compressor -- variance frozen, momenta averaged
// uncompressed.  m_i = beta1 m + (1-beta1) g_i per worker, m = mean_i m_i
// (fp64 sum in worker order, one rounding), x -= lr m / sqrt(v + eps).
// ---------------------------------------------------------------------------
template <bool FULL>
__device__ __forceinline__ void uncompressed_load(int64_t base, int len, int lane,
                                                  const float *__restrict__ x,
                                                  const float *__restrict__ m,
                                                  const float *__restrict__ v, float beta1,
                                                  v4f (&bm)[kSubBlocks], v4f (&xv)[kSubBlocks],
                                                  v4f (&vv)[kSubBlocks])
{
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        bm[b] = beta1 * ld4<FULL>(m + base, li, len);
        xv[b] = ld4<FULL>(x + base, li, len);
        vv[b] = ld4<FULL>(v + base, li, len);
    }
}

// sum += worker i's momentum beta1 m + (1 - beta1) g_i (fp32, then fp64 sum)
template <bool FULL, class G>
__device__ __forceinline__ void add_momentum_row(double (&sum)[kSubBlocks][4],
                                                 const v4f (&bm)[kSubBlocks],
                                                 const typename G::T *__restrict__ row, int lane,
                                                 int len, float omb1)
{
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const v4f gv = ldg4<FULL, G>(row, b * (kWave * 4) + 4 * lane, len);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            float mi = omb1 * gv[c];
            mi = bm[b][c] + mi;
            sum[b][c] += (double)mi;
        }
    }
}

template <bool FULL>
__device__ __forceinline__ void uncompressed_store(const double (&sum)[kSubBlocks][4], int64_t base,
                                                   int len, int lane, v4f (&xv)[kSubBlocks],
                                                   const v4f (&vv)[kSubBlocks],
                                                   float *__restrict__ x, float *__restrict__ m,
                                                   double dn, float lr, float eps)
{
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        v4f mv;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float mbar = (float)(sum[b][c] / dn);
            const float denom = __builtin_sqrtf(vv[b][c] + eps);
            const float ratio = mbar / denom;
            const float step = lr * ratio;
            xv[b][c] = xv[b][c] - step;
            mv[c] = mbar;
        }
        st4<FULL>(x + base, li, len, xv[b]);
        st4<FULL>(m + base, li, len, mv);
    }
}

template <class G>
__global__ __launch_bounds__(kRowBlock) void k_uncompressed(
    const Tile *__restrict__ tiles, int64_t num_tiles, float *__restrict__ x,
    float *__restrict__ m, const float *__restrict__ v, const typename G::T *__restrict__ g,
    int64_t g_ld, int n, float lr, float beta1, float omb1, float eps)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = xcd_block() * kRowWaves + (threadIdx.x >> 6);
    const bool active = t < num_tiles;
    Tile tile{0, 0, 0};
    if (active) tile = tiles[t];
    const bool full = tile.len == kTileElems;
    v4f bm[kSubBlocks], xv[kSubBlocks], vv[kSubBlocks];
    if (full)
        uncompressed_load<true>(tile.start, tile.len, lane, x, m, v, beta1, bm, xv, vv);
    else
        uncompressed_load<false>(tile.start, tile.len, lane, x, m, v, beta1, bm, xv, vv);
    double sum[kSubBlocks][4];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[b][c] = 0.0;
    for (int i = 0; i < n; ++i) {
        const typename G::T *row = g + (int64_t)i * g_ld + tile.start;
        if (full)
            add_momentum_row<true, G>(sum, bm, row, lane, tile.len, omb1);
        else if (active)
            add_momentum_row<false, G>(sum, bm, row, lane, tile.len, omb1);
        __builtin_amdgcn_s_barrier();  // the workgroup reads each row together
    }
    if (!active) return;
    const double dn = (double)n;
    if (full)
        uncompressed_store<true>(sum, tile.start, tile.len, lane, xv, vv, x, m, dn, lr, eps);
    else
        uncompressed_store<false>(sum, tile.start, tile.len, lane, xv, vv, x, m, dn, lr, eps);
}

template <class G>
__global__ __launch_bounds__(kRowBlock) void k_warmup(
    const Tile *__restrict__ tiles, int64_t num_tiles, float *__restrict__ x,
    float *__restrict__ m, float *__restrict__ v, const typename G::T *__restrict__ g, int64_t g_ld,
    int n_grads, float lr, float beta1, float omb1, float beta2, float omb2, float eps,
    int use_bc, float bc1, float bc2)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = xcd_block() * kRowWaves + (threadIdx.x >> 6);
    const bool active = t < num_tiles;
    Tile tile{0, 0, 0};
    if (active) tile = tiles[t];
    const bool full = tile.len == kTileElems;
    double sum[kSubBlocks][4];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[b][c] = 0.0;
    if (full)
        warmup_rows_walk<true, G>(sum, tile, lane, true, g, g_ld, n_grads);
    else
        warmup_rows_walk<false, G>(sum, tile, lane, active, g, g_ld, n_grads);
    if (!active) return;
    const double dn = (double)n_grads;
    if (full)
        warmup_update<true>(sum, tile.start, tile.len, lane, x, m, v, dn, lr, beta1, omb1,
                            beta2, omb2, eps, use_bc, bc1, bc2);
    else
        warmup_update<false>(sum, tile.start, tile.len, lane, x, m, v, dn, lr, beta1, omb1,
                             beta2, omb2, eps, use_bc, bc1, bc2);
}

// ---------------------------------------------------------------------------
// Worker pass: for each local worker i, z_i = (beta1 m + (1-beta1) g_i) + delta_i,
// sign words of z_i, per-tile partial sum of z_i^2, and z_i written back as the
// new compensated error state.
//
// Packed momentum (every step after the first): a two-wave workgroup handles
// one tile for a group of consecutive workers (one worker in practice), wave h
// holding sub-blocks 2h and 2h+1, and the items run group-major, split into
// one contiguous eighth per XCD: the waves in flight on an XCD work on the
// same few worker rows, so each XCD streams through 2 x group rows of
// (g, error state) at a time instead of all 2n.  Half a tile per wave keeps
// fewer bytes in flight per wave at a higher occupancy (80 instead of ~120
// VGPRs), which the mix of two read streams and one written stream favours.
// The momentum of a tile is re-derived by every worker, 1/8 byte per element
// per worker from a sign array small enough to stay in the last-level cache.
// An fp32 momentum (the first compression step) is read once per tile for all
// local workers instead, by k_worker_rows.
// ---------------------------------------------------------------------------
// Sub-blocks per wave of the packed worker pass, and its waves per tile.
constexpr int kWorkerSubBlocks = 2;
static_assert(kSubBlocks / kWorkerSubBlocks == kWorkerWavesPerBlock,
              "the packed worker pass gives each wave of a workgroup part of one tile");

// The shared momentum m_{t-1} of sub-blocks sb0 .. sb0+SB-1 of the tile times
// beta1.  PACKED: m_{t-1} is the previous step's gathered server message,
// decoded from its sign words and segment scale (+-scale, exactly the fp32
// value the update would have stored), so no fp32 momentum buffer is read.
template <bool FULL, bool PACKED, int SB>
__device__ __forceinline__ void beta1_momentum(v4f (&bm)[SB], const Tile &tile, int lane, int sb0,
                                               const float *__restrict__ m,
                                               const uint64_t *__restrict__ m_bits,
                                               const float *__restrict__ m_scales, float beta1)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    if (PACKED) {
        const float s = m_scales[tile.seg];
#pragma unroll
        for (int b = 0; b < SB; ++b) {
            const int sb = sb0 + b;
            const int li = sb * (kWave * 4) + 4 * lane;
            const uint64_t word =
                (FULL || li < len) ? m_bits[(base >> 6) + 4 * sb + (lane >> 4)] : 0ull;
            const uint32_t nib = (uint32_t)(word >> (4 * (lane & 15))) & 0xFu;
#pragma unroll
            for (int c = 0; c < 4; ++c) bm[b][c] = beta1 * (((nib >> c) & 1u) ? s : -s);
        }
    } else {
#pragma unroll
        for (int b = 0; b < SB; ++b)
            bm[b] = beta1 * ld4<FULL>(m + base, (sb0 + b) * (kWave * 4) + 4 * lane, len);
    }
}

// Worker i's row over sub-blocks sb0 .. sb0+SB-1 of the tile: z_i from the
// momentum term bm = beta1 m, the gradient row and the previous compensated
// value; its sign words, sum of squares and new compensated value.  Split into
// the loads of the row and the arithmetic and stores, so that a caller can
// issue the next row's loads before this row's stores.
template <bool FULL, class G, int SB>
__device__ __forceinline__ void worker_row_load(const Tile &tile, int lane, int sb0, int i,
                                                const typename G::T *__restrict__ g, int64_t g_ld,
                                                const float *__restrict__ err, int64_t err_ld,
                                                const float *__restrict__ scales,
                                                int64_t scales_ld, v4f (&gv)[SB], v4f (&cv)[SB],
                                                float &sp)
{
    const int len = tile.len;
    sp = scales[(int64_t)i * scales_ld + tile.seg];
    const typename G::T *gi = g + (int64_t)i * g_ld + tile.start;
    const float *ei = err + (int64_t)i * err_ld + tile.start;
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int li = (sb0 + b) * (kWave * 4) + 4 * lane;
        gv[b] = ldg4<FULL, G>(gi, li, len);
        cv[b] = ld4<FULL>(ei, li, len);
    }
}

// Returns this wave's sum of z_i^2 over its sub-blocks (lanes summed in a
// fixed order); the caller writes the tile's partial sum.  Each sub-block is
// stored as soon as it is computed: computing every sub-block first keeps
// more values live, and at the worker pass's 80 VGPRs the compiler then
// issues a 16-bit-gradient row's loads one after another (measured 5.7%
// slower for bf16 gradients, no faster for fp32).
template <bool FULL, int SB>
__device__ __forceinline__ double worker_row_store(const Tile &tile, int lane, int sb0,
                                                   const v4f (&bm)[SB], int i, const v4f (&gv)[SB],
                                                   const v4f (&cv)[SB], float sp,
                                                   float *__restrict__ err, int64_t err_ld,
                                                   uint64_t *__restrict__ bits, int64_t bits_ld,
                                                   float omb1)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    const int nwords = (len + 63) >> 6;
    float *ei = err + (int64_t)i * err_ld + base;
    uint64_t *bi = bits + (int64_t)i * bits_ld + (base >> 6);
    double acc = 0.0;
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int li = (sb0 + b) * (kWave * 4) + 4 * lane;
        v4f zv;
        uint32_t nib = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float d = error_of(cv[b][c], sp);
            float mi = omb1 * gv[b][c];
            mi = bm[b][c] + mi;
            const float z = mi + d;
            zv[c] = z;
            const bool valid = FULL || li + c < len;
            const double zd = valid ? (double)z : 0.0;
            acc += zd * zd;
            nib |= (valid && z >= 0.f) ? (1u << c) : 0u;
        }
        st4<FULL>(ei, li, len, zv);
        const uint64_t word = row_sign_word(nib, lane);
        const int w = 4 * (sb0 + b) + (lane >> 4);
        if ((lane & 15) == 0 && (FULL || w < nwords)) bi[w] = word;
    }
    return wave_sum(acc);
}

// The tile for workers [i0, i1), this wave's sub-blocks of the momentum term
// loaded or decoded once.  The waves' sums of each row meet in red (two slots,
// alternating by row: a wave can be at most one row ahead of the other, so
// the slot it writes is never the one still being read) and wave 0 adds them
// in wave order.  Every wave of the workgroup runs the same rows, so every
// wave reaches every barrier.
template <bool FULL, bool PACKED, class G>
__device__ __forceinline__ void worker_tile(
    double (&red)[2][kWorkerWavesPerBlock], int &slot, const Tile &tile, int64_t t, int lane,
    int wv, int64_t num_tiles, const float *__restrict__ m, const uint64_t *__restrict__ m_bits,
    const float *__restrict__ m_scales, const typename G::T *__restrict__ g, int64_t g_ld,
    float *__restrict__ err, int64_t err_ld, const float *__restrict__ scales, int64_t scales_ld,
    uint64_t *__restrict__ bits, int64_t bits_ld, double *__restrict__ partial, int i0, int i1,
    float beta1, float omb1)
{
    constexpr int SB = kWorkerSubBlocks;
    const int sb0 = wv * SB;
    v4f bm[SB];
    beta1_momentum<FULL, PACKED, SB>(bm, tile, lane, sb0, m, m_bits, m_scales, beta1);
    for (int i = i0; i < i1; ++i) {
        v4f gv[SB], cv[SB];
        float sp;
        worker_row_load<FULL, G, SB>(tile, lane, sb0, i, g, g_ld, err, err_ld, scales, scales_ld,
                                     gv, cv, sp);
        const double acc = worker_row_store<FULL, SB>(tile, lane, sb0, bm, i, gv, cv, sp, err,
                                                      err_ld, bits, bits_ld, omb1);
        if (lane == 0) red[slot][wv] = acc;
        __syncthreads();
        if (wv == 0 && lane == 0) {
            double sum = red[slot][0];
#pragma unroll
            for (int k = 1; k < kWorkerWavesPerBlock; ++k) sum += red[slot][k];
            partial[(int64_t)i * num_tiles + t] = sum;
        }
        slot ^= 1;
    }
}

// Waves per SIMD of the worker pass.  With fp32 gradients the kernel's
// register count sits at the six-wave limit (80 VGPRs; without the hint the
// compiler settles on 85 and five waves).  A 16-bit gradient row needs half
// the registers for its loads, and seven waves (72 VGPRs, no spills) ran the
// bf16 and fp16 passes 0.5-0.8% faster than six on the BERT shapes and 2.2%
// on the 5,000-tensor stress workload; eight spill.
template <class G>
constexpr int kWorkerWavesPerSimd = sizeof(typename G::T) == 2 ? 7 : 6;

template <bool PACKED, class G>
__global__ __launch_bounds__(kWorkerBlock) __attribute__((amdgpu_waves_per_eu(kWorkerWavesPerSimd<G>))) void k_worker_pass(
    const Tile *__restrict__ tiles, int64_t num_tiles, const float *__restrict__ m,
    const uint64_t *__restrict__ m_bits, const float *__restrict__ m_scales,
    const typename G::T *__restrict__ g, int64_t g_ld, float *__restrict__ err, int64_t err_ld,
    const float *__restrict__ scales, int64_t scales_ld, uint64_t *__restrict__ bits,
    int64_t bits_ld, double *__restrict__ partial, int n_local, int group, int64_t num_items,
    float beta1, float omb1)
{
    __shared__ double red[2][kWorkerWavesPerBlock];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    int slot = 0;
    // each XCD walks one contiguous eighth of the items, one item per workgroup
    const ItemWalk walk = xcd_item_walk(blockIdx.x, gridDim.x, num_items);
    for (int64_t item = walk.first; item < walk.end; item += walk.stride) {
        const int64_t grp = item / num_tiles;
        const int64_t t = item - grp * num_tiles;
        const int i0 = (int)grp * group;
        const int i1 = min(n_local, i0 + group);
        const Tile tile = tiles[t];
        if (tile.len == kTileElems)
            worker_tile<true, PACKED, G>(red, slot, tile, t, lane, wv, num_tiles, m, m_bits,
                                         m_scales, g, g_ld, err, err_ld, scales, scales_ld, bits,
                                         bits_ld, partial, i0, i1, beta1, omb1);
        else
            worker_tile<false, PACKED, G>(red, slot, tile, t, lane, wv, num_tiles, m, m_bits,
                                          m_scales, g, g_ld, err, err_ld, scales, scales_ld, bits,
                                          bits_ld, partial, i0, i1, beta1, omb1);
    }
}

// ---------------------------------------------------------------------------
// The worker pass with an fp32 momentum (the first compression step): m is
// read once per tile for all local workers, and the 16 waves of a workgroup
// walk the worker rows together (one barrier per row), as in the warm-up.
// The rows are double-buffered: row i+1's loads (gradient, error state and
// scale) are issued before row i's arithmetic and stores, so each wave keeps
// two rows of loads in flight and never waits on a load issued right after
// its own stores (measured 23.75 against 23.86 ms for one row at a time, and
// 24.76 ms without the barriers, on the BERT-Large shape, same buffers).
// As in the packed pass, two waves share each tile, half a tile each (8 tiles
// per workgroup); the pair's sums of squares of row i meet in red[i & 1] at
// the barrier after row i, and the pair's first wave adds them in wave order
// and writes the partial sum.  A wave writes red[i & 1] again only after the
// next barrier, by which time the read of row i is done.
// ---------------------------------------------------------------------------
template <bool FULL, class G, int SB>
__device__ __forceinline__ void worker_rows_walk(
    double (&red)[2][kRowWaves], const Tile &tile, int64_t t, int lane, int wv, int64_t num_tiles,
    bool active, const v4f (&bm)[SB], const typename G::T *__restrict__ g, int64_t g_ld,
    float *__restrict__ err, int64_t err_ld, const float *__restrict__ scales, int64_t scales_ld,
    uint64_t *__restrict__ bits, int64_t bits_ld, double *__restrict__ partial, int n_local,
    float omb1)
{
    constexpr int W = kSubBlocks / SB;
    const int sb0 = (wv % W) * SB;
    v4f ga[SB], ca[SB], gb[SB], cb[SB];
    float sa = 0.f, sb = 0.f;
#define ROW_LOAD(i, gv, cv, sp) \
    worker_row_load<FULL, G, SB>(tile, lane, sb0, i, g, g_ld, err, err_ld, scales, scales_ld, gv, cv, sp)
#define ROW_STORE(i, gv, cv, sp)                                                                   \
    do {                                                                                           \
        const double acc = worker_row_store<FULL, SB>(tile, lane, sb0, bm, i, gv, cv, sp, err,     \
                                                      err_ld, bits, bits_ld, omb1);                \
        if (W == 1) {                                                                              \
            if (lane == 0) partial[(int64_t)(i) * num_tiles + t] = acc;                            \
        } else if (lane == 0) {                                                                    \
            red[(i) & 1][wv] = acc;                                                                \
        }                                                                                          \
    } while (0)
#define ROW_SUM(i)                                                                                 \
    do {                                                                                           \
        if (W > 1 && active && wv % W == 0 && lane == 0) {                                         \
            double s_ = red[(i) & 1][wv];                                                          \
            for (int k_ = 1; k_ < W; ++k_) s_ += red[(i) & 1][wv + k_];                            \
            partial[(int64_t)(i) * num_tiles + t] = s_;                                            \
        }                                                                                          \
    } while (0)
    if (active) ROW_LOAD(0, ga, ca, sa);
    int i = 0;
    for (; i + 2 < n_local; i += 2) {
        if (active) ROW_LOAD(i + 1, gb, cb, sb);
        if (active) ROW_STORE(i, ga, ca, sa);
        __builtin_amdgcn_s_barrier();
        ROW_SUM(i);
        if (active) ROW_LOAD(i + 2, ga, ca, sa);
        if (active) ROW_STORE(i + 1, gb, cb, sb);
        __builtin_amdgcn_s_barrier();
        ROW_SUM(i + 1);
    }
    if (i + 1 < n_local) {
        if (active) ROW_LOAD(i + 1, gb, cb, sb);
        if (active) ROW_STORE(i, ga, ca, sa);
        __builtin_amdgcn_s_barrier();
        ROW_SUM(i);
        if (active) ROW_STORE(i + 1, gb, cb, sb);
        __builtin_amdgcn_s_barrier();
        ROW_SUM(i + 1);
    } else {
        if (active) ROW_STORE(i, ga, ca, sa);
        __builtin_amdgcn_s_barrier();
        ROW_SUM(i);
    }
#undef ROW_LOAD
#undef ROW_STORE
#undef ROW_SUM
}

template <class G>
__global__ __launch_bounds__(kRowBlock) void k_worker_rows(
    const Tile *__restrict__ tiles, int64_t num_tiles, const float *__restrict__ m,
    const typename G::T *__restrict__ g, int64_t g_ld, float *__restrict__ err, int64_t err_ld,
    const float *__restrict__ scales, int64_t scales_ld, uint64_t *__restrict__ bits,
    int64_t bits_ld, double *__restrict__ partial, int n_local, float beta1, float omb1,
    int64_t tile_base)
{
    constexpr int SB = kWorkerSubBlocks;
    constexpr int W = kSubBlocks / SB;
    static_assert(W * kWorkerRowTiles == kRowWaves, "two waves per tile");
    __shared__ double red[2][kRowWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int64_t t = tile_base + xcd_block() * kWorkerRowTiles + wv / W;
    const bool active = t < num_tiles;
    Tile tile{0, 0, 0};
    if (active) tile = tiles[t];
    const bool full = tile.len == kTileElems;
    v4f bm[SB];
    if (full) {
        beta1_momentum<true, false, SB>(bm, tile, lane, (wv % W) * SB, m, nullptr, nullptr, beta1);
        worker_rows_walk<true, G, SB>(red, tile, t, lane, wv, num_tiles, true, bm, g, g_ld, err,
                                      err_ld, scales, scales_ld, bits, bits_ld, partial, n_local, omb1);
    } else {
        beta1_momentum<false, false, SB>(bm, tile, lane, (wv % W) * SB, m, nullptr, nullptr, beta1);
        worker_rows_walk<false, G, SB>(red, tile, t, lane, wv, num_tiles, active, bm, g, g_ld, err,
                                       err_ld, scales, scales_ld, bits, bits_ld, partial, n_local,
                                       omb1);
    }
}

// ---------------------------------------------------------------------------
// Scale finalize: scale = fp32(sqrt(sum over the segment's tiles / len)),
// summed in a fixed order (so results do not depend on scheduling); empty
// segments get 0.  THREADS lanes cooperate on one (row, segment) pair: a
// wave when segments have few tiles, a whole block when they have many.
// ---------------------------------------------------------------------------
template <int THREADS>
__device__ __forceinline__ float finalize_one(const double *__restrict__ part, int64_t tb,
                                              int64_t te, int64_t len, double *red)
{
    const int tid = threadIdx.x % THREADS;
    double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
    int64_t t = tb + tid;
    for (; t + 3 * THREADS < te; t += 4 * THREADS) {
        s0 += part[t];
        s1 += part[t + THREADS];
        s2 += part[t + 2 * THREADS];
        s3 += part[t + 3 * THREADS];
    }
    for (; t < te; t += THREADS) s0 += part[t];
    double s = wave_sum((s0 + s1) + (s2 + s3));
    if (THREADS > kWave) {
        const int wv = tid / kWave;
        if ((tid & (kWave - 1)) == 0) red[wv] = s;
        __syncthreads();
        s = red[0];
        for (int w = 1; w < THREADS / kWave; ++w) s += red[w];
    }
    return len > 0 ? (float)__builtin_sqrt(s / (double)len) : 0.0f;
}

// Pair p -> (row i, segment q).  Worker form: all S segments of each row.
// Server form: segments k*n + j for j in [jb, je) and every tensor k.
template <int THREADS>
__global__ __launch_bounds__(kBlock) void k_finalize(
    DeviceTables tb, int64_t num_pairs, int64_t num_segments, int server_form, int n, int jb,
    int je, const double *__restrict__ partial, int64_t part_ld, float *__restrict__ scales,
    int64_t scales_ld)
{
    __shared__ double red[kBlock / kWave];
    // THREADS lanes per pair; the grid may be smaller than the pair count, so
    // each group of lanes strides over pairs (uniform per block or per wave)
    const int64_t stride = (int64_t)gridDim.x * (kBlock / THREADS);
    for (int64_t p = (int64_t)blockIdx.x * (kBlock / THREADS) + threadIdx.x / THREADS;
         p < num_pairs; p += stride) {
        int64_t i, q;
        if (server_form) {
            const int cnt = je - jb;
            i = 0;
            q = (p / cnt) * n + jb + (p % cnt);
        } else {
            i = p / num_segments;
            q = p % num_segments;
        }
        const float s = finalize_one<THREADS>(partial + i * part_ld, tb.seg_tile_begin[q],
                                              tb.seg_tile_end[q], tb.seg_len[q], red);
        if (threadIdx.x % THREADS == 0) scales[i * scales_ld + q] = s;
        if (THREADS > kWave) __syncthreads();  // red is reused by the next pair
    }
}

// ---------------------------------------------------------------------------
// Server pass over the tiles of the owned chunks: decode and average the n
// incoming messages, add the server error, write the sign words and the new
// compensated server state, and the tile's sum of squares.
//
// Each wave owns its own LDS region, so it synchronises only with itself (no
// workgroup barrier); a tile's error-state loads are issued first so that
// they overlap the sign-word traffic.  Incoming sign words are
// staged in LDS 32 worker rows at a time (coalesced 128-byte row reads),
// transposed so that the words of consecutive workers for one 32-element
// half-word are adjacent.  For the table lookups each group of 8 workers is
// then regrouped in place, four 8x8 bit transposes per (half-word, group):
// afterwards each LDS byte holds the 8 workers' bits of one element, the
// element's table index.
//
// The average is an fp64 sum of +-scale over the workers in worker order.
// When every partial sum of the segment's scales is exactly representable in
// fp64 (the scales' exponents span at most 29 - ceil(log2 n) binades; true
// for any realistic message set) the sum is exact, so it may be formed in any
// grouping: then each group of 8 workers is one lookup in a 256-entry table
// of its signed scale sums, indexed by the 8 workers' bits of the element.
// The 256-entry tables are sums of two 16-entry tables, each built from 4
// scales; they depend on the segment's scales only.  Otherwise every worker
// is added one by one.  Both give the oracle's sum.
// ---------------------------------------------------------------------------
// Wave-wide max of an int through DPP: shifts within each 16-lane row, then
// row broadcasts carry the row maxima up to lane 63, which every lane reads.
__device__ __forceinline__ int wave_max(int v)
{
    constexpr int lo = INT32_MIN;
    v = max(v, __builtin_amdgcn_update_dpp(lo, v, 0x111, 0xF, 0xF, false));  // row_shr 1
    v = max(v, __builtin_amdgcn_update_dpp(lo, v, 0x112, 0xF, 0xF, false));  // row_shr 2
    v = max(v, __builtin_amdgcn_update_dpp(lo, v, 0x114, 0xF, 0xF, false));  // row_shr 4
    v = max(v, __builtin_amdgcn_update_dpp(lo, v, 0x118, 0xF, 0xF, false));  // row_shr 8
    v = max(v, __builtin_amdgcn_update_dpp(lo, v, 0x142, 0xA, 0xF, false));  // row_bcast 15
    v = max(v, __builtin_amdgcn_update_dpp(lo, v, 0x143, 0xC, 0xF, false));  // row_bcast 31
    return __builtin_amdgcn_readlane(v, kWave - 1);
}

__device__ __forceinline__ int wave_min(int v) { return -wave_max(-v); }

__device__ __forceinline__ void wave_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// One sub-block (256 elements) of the server pass's last part: average, add
// the server error, store the new compensated error state and the sign words;
// returns this wave's fp64 sum of squares of the sub-block (every lane gets
// it).  sum[c] and cv[c] are the lane's elements b*256 + 4*lane + c.
template <bool FULL, bool POW2>
__device__ __forceinline__ double server_epilogue_sub(const double (&sum)[4], v4f cv,
                                                      float sprev, int n, int lane,
                                                      const Tile &tile, int b,
                                                      float *__restrict__ serr,
                                                      uint64_t *__restrict__ sbits)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    const int nwords = (len + 63) >> 6;
    const double dn = (double)n;
    const double inv_n = 1.0 / dn;
    const int li = b * (kWave * 4) + 4 * lane;
    double acc = 0.0;
    v4f zv;
    uint32_t nib = 0;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        // avg = sum / n rounded to fp32 (for a power-of-two n, sum * (1/n) is
        // the same exact scaling), then the compensated value and its square
        const float avg = (float)(POW2 ? sum[c] * inv_n : sum[c] / dn);
        const float z = avg + error_of(cv[c], sprev);
        zv[c] = z;
        const bool valid = FULL || li + c < len;
        const double zd = valid ? (double)z : 0.0;
        // zd * zd is exact in fp64 (a 24-bit significand squared), so the
        // fused form rounds exactly as the separate multiply and add would
        acc = __builtin_fma(zd, zd, acc);
        nib |= (valid && z >= 0.f) ? (1u << c) : 0u;
    }
    st4<FULL>(serr + base, li, len, zv);
    const uint64_t word = row_sign_word(nib, lane);
    const int w = 4 * b + (lane >> 4);
    if ((lane & 15) == 0 && (FULL || w < nwords)) sbits[(base >> 6) + w] = word;
    return acc;
}

// LDS row stride (in 32-bit words) of the sign staging: a multiple of 4 keeps
// 128-bit accesses aligned, and 40 puts the 64 words a wave reads at once in
// the accumulation on 64 different banks.
constexpr int kBitsStride = kServerRowBatch + 8;

// One wave's LDS working set for a batch of up to kServerRowBatch incoming
// rows of one tile: the sign words, transposed ([half-word h][row r]), the
// rows' scales, and the lookup tables built from them (the 256-entry tables
// of two groups of 8 rows at a time).
struct ServerBatchLds {
    uint32_t bits[2 * kTileWords][kBitsStride];
    double lut4[kServerRowBatch / 4][16];
    double lut8[2][256];
    float scale[kServerRowBatch];
};

// One wave's LDS working set in the one-wave-per-tile pass (n <= 8 G8 <=
// kServerRowBatch): the 256-entry tables of all G8 groups of 8 rows, held at
// once, are built from the 16-entry tables before the tile's words are staged
// (so those share the staging area).  G8 follows n, so that smaller n leave
// room for more workgroups per CU.
template <int G8>
struct ServerTileLds {
    union {
        uint32_t bits[2 * kTileWords][kBitsStride];
        double lut4[kServerRowBatch / 4][16];
    };
    double lut8[G8][256];
    float scale[kServerRowBatch];
};

// 8x8 bit transposes of the four byte columns of 8 words: bit j of byte b of
// a[k] moves to bit k of byte b of a[j] (three rounds of block swaps: 4x4,
// 2x2, 1x1 bits, each on all four bytes at once).
__device__ __forceinline__ void transpose_bits8x8(uint32_t (&a)[8])
{
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const uint32_t t = ((a[k] >> 4) ^ a[k + 4]) & 0x0F0F0F0Fu;
        a[k] ^= t << 4;
        a[k + 4] ^= t;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int k = (i & 1) + 4 * (i >> 1);  // 0, 1, 4, 5
        const uint32_t t = ((a[k] >> 2) ^ a[k + 2]) & 0x33333333u;
        a[k] ^= t << 2;
        a[k + 2] ^= t;
    }
#pragma unroll
    for (int k = 0; k < 8; k += 2) {
        const uint32_t t = ((a[k] >> 1) ^ a[k + 1]) & 0x55555555u;
        a[k] ^= t << 1;
        a[k + 1] ^= t;
    }
}

// The incoming sign words and scales of one tile as the chunk owner reads
// them: row i's word for tile word wi is at words[i * bits_ld + wi], its
// scale at scales[i * scales_ld].
struct ServerRows {
    const uint64_t *words;   // the tile's first word in row 0
    int64_t bits_ld;
    const float *scales;     // the segment's scale in row 0
    int64_t scales_ld;
    int nwords;              // words of the tile
    bool full;               // a full tile
};

// Loads the words of rows [r0, r0 + rows) of the tile (rows <=
// kServerRowBatch): lane L takes word wi = L % 16 of rows r0 + L/16 + 4k.
__device__ __forceinline__ void server_load_words(const ServerRows &in, int r0, int rows,
                                                  int lane, uint64_t (&stg)[kServerRowBatch / 4])
{
    const int wi = lane & (kTileWords - 1);
    const uint64_t *p = in.words + (int64_t)(r0 + (lane >> 4)) * in.bits_ld + wi;
    const int64_t step = 4 * in.bits_ld;
    if (in.full && rows == kServerRowBatch) {  // wave-uniform: every load in range
#pragma unroll
        for (int k = 0; k < kServerRowBatch / 4; ++k) stg[k] = __builtin_nontemporal_load(p + k * step);
    } else {
#pragma unroll
        for (int k = 0; k < kServerRowBatch / 4; ++k) {
            const int r = (lane >> 4) + 4 * k;
            stg[k] = (r < rows && wi < in.nwords) ? __builtin_nontemporal_load(p + k * step) : 0ull;
        }
    }
}

// The words of rows [r0, r0 + rows) and the scale of row r0 + lane.
__device__ __forceinline__ void server_load_batch(const ServerRows &in, int r0, int rows,
                                                  int lane, uint64_t (&stg)[kServerRowBatch / 4],
                                                  float &scl)
{
    server_load_words(in, r0, rows, lane, stg);
    scl = lane < rows ? in.scales[(int64_t)(r0 + lane) * in.scales_ld] : 0.f;
}

// Writes loaded words into the wave's staging area (rows past the batch's
// last row, up to the next multiple of 8, get zero words).
template <class Lds>
__device__ __forceinline__ void server_stage_words(Lds &L, const ServerRows &in, int rows,
                                                   int lane,
                                                   const uint64_t (&stg)[kServerRowBatch / 4])
{
    const int wi = lane & (kTileWords - 1);
    const int rows8 = (rows + 7) & ~7;
    if (in.full && rows == kServerRowBatch) {  // wave-uniform
#pragma unroll
        for (int k = 0; k < kServerRowBatch / 4; ++k) {
            const int r = (lane >> 4) + 4 * k;
            L.bits[2 * wi][r] = (uint32_t)stg[k];
            L.bits[2 * wi + 1][r] = (uint32_t)(stg[k] >> 32);
        }
    } else {
#pragma unroll
        for (int k = 0; k < kServerRowBatch / 4; ++k) {
            const int r = (lane >> 4) + 4 * k;
            if (r < rows8 && wi < in.nwords) {
                L.bits[2 * wi][r] = (uint32_t)stg[k];
                L.bits[2 * wi + 1][r] = (uint32_t)(stg[k] >> 32);
            }
        }
    }
}

// Stages a loaded batch: its words, and the scale of row `lane`.
template <class Lds>
__device__ __forceinline__ void server_stage_batch(Lds &L, const ServerRows &in,
                                                   int rows, int lane,
                                                   const uint64_t (&stg)[kServerRowBatch / 4],
                                                   float scl)
{
    server_stage_words(L, in, rows, lane, stg);
    if (lane < rows) L.scale[lane] = scl;
}

// The 16-entry tables of 4 rows, two per group of 8 (rows past the last row
// add 0): lut4[q][idx] is the sum over k < 4 of +-scale[4q + k], + where bit
// k of idx is set.
template <class Lds>
__device__ __forceinline__ void server_build_lut4(Lds &L, int rows, int lane)
{
    const int groups8 = (rows + 7) >> 3;
    for (int e = lane; e < 32 * groups8; e += kWave) {
        const int q = e >> 4, idx = e & 15;
        double v = 0.0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int r = 4 * q + k;
            if (r < rows) {
                const double sc = (double)L.scale[r];
                v += ((idx >> k) & 1) ? sc : -sc;
            }
        }
        L.lut4[q][idx] = v;
    }
}

// Regroups each staged (half-word, group of 8 rows) block in place by four
// 8x8 bit transposes, after which byte e>>3 of word r8 + (e&7) of the block is
// element e's table index (the 8 rows' bits of e).
template <class Lds>
__device__ __forceinline__ void server_regroup_bits(Lds &L, int rows, int lane)
{
    const int groups8 = (rows + 7) >> 3;
#pragma unroll 1
    for (int k = 0; k < (2 * kTileWords) * (kServerRowBatch / 8) / kWave; ++k) {
        const int blk = lane + kWave * k;
        const int hwb = blk & (2 * kTileWords - 1), gb = blk / (2 * kTileWords);
        if (gb < groups8) {
            uint32_t *p = &L.bits[hwb][8 * gb];
            const uint4 u0 = *(const uint4 *)p;
            const uint4 u1 = *(const uint4 *)(p + 4);
            uint32_t a[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
            transpose_bits8x8(a);
            *(uint4 *)p = make_uint4(a[0], a[1], a[2], a[3]);
            *(uint4 *)(p + 4) = make_uint4(a[4], a[5], a[6], a[7]);
        }
    }
}

// sum += the group of 8 rows starting at row r8, one lookup per element in
// its 256-entry table lut (regrouped words).  Two sub-blocks at a time: their
// 8 table indices first, then the 8 lookups, then the adds, so that the LDS
// round trips overlap.
template <class Lds>
__device__ __forceinline__ void server_lookup_group(double (&sum)[kSubBlocks][4], const Lds &L,
                                                    int r8, const double *lut, int lane)
{
    const int half = (lane >> 3) & 1;
#pragma unroll
    for (int bh = 0; bh < kSubBlocks; bh += 2) {
        uint32_t idx[2][4];
#pragma unroll
        for (int bb = 0; bb < 2; ++bb) {
            const int hw = 2 * (4 * (bh + bb) + (lane >> 4)) + half;
            // the lane's elements e = 4 (lane & 7) + c of the half-word:
            // byte e >> 3 of word e & 7 holds the 8 rows' bits of e
            const uint8_t *blk = (const uint8_t *)&L.bits[hw][r8];
            const int o = 16 * (lane & 1) + ((lane & 7) >> 1);
#pragma unroll
            for (int c = 0; c < 4; ++c) idx[bb][c] = blk[o + 4 * c];
        }
        double val[2][4];
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
            for (int c = 0; c < 4; ++c) val[bb][c] = lut[idx[bb][c]];
#pragma unroll
        for (int bb = 0; bb < 2; ++bb)
#pragma unroll
            for (int c = 0; c < 4; ++c) sum[bh + bb][c] += val[bb][c];
    }
}

// sum += the staged batch's decoded messages, grouped: each group of 8 rows is
// one lookup in a 256-entry table of its signed scale sums (exact, so any
// grouping gives the worker-order sum).  The 16-entry tables of 4 rows are
// built first, then the staged words are regrouped; the 256-entry tables are
// built two groups at a time.
__device__ __forceinline__ void server_batch_grouped(double (&sum)[kSubBlocks][4],
                                                     ServerBatchLds &L, int rows, int lane)
{
    const int groups8 = (rows + 7) >> 3;
    server_build_lut4(L, rows, lane);
    server_regroup_bits(L, rows, lane);
    wave_sync();
    for (int g0 = 0; 8 * g0 < rows; g0 += 2) {
        const int gcnt = min(2, groups8 - g0);
#pragma unroll
        for (int k = 0; k < 512 / kWave; ++k) {
            const int e = lane + kWave * k;
            const int g = e >> 8, idx = e & 255;  // g = k / 4: uniform
            if (g < gcnt) {
                const int q = 2 * (g0 + g);
                L.lut8[g][idx] = L.lut4[q][idx & 15] + L.lut4[q + 1][idx >> 4];
            }
        }
        wave_sync();
        for (int g = 0; g < gcnt; ++g) server_lookup_group(sum, L, 8 * (g0 + g), L.lut8[g], lane);
        wave_sync();
    }
}

// sum += the staged batch's decoded messages one worker at a time, in row
// order (the path for scale sets whose partial sums may round).
template <class Lds>
__device__ __forceinline__ void server_batch_one_by_one(double (&sum)[kSubBlocks][4],
                                                        const Lds &L, int rows, int lane)
{
    const int half = (lane >> 3) & 1;
    const int shift = 4 * (lane & 7);
    for (int r = 0; r < rows; ++r) {
        const double sp = (double)L.scale[r];
        const double sn = -sp;
#pragma unroll
        for (int b = 0; b < kSubBlocks; ++b) {
            const uint32_t nib = (L.bits[2 * (4 * b + (lane >> 4)) + half][r] >> shift) & 0xFu;
#pragma unroll
            for (int c = 0; c < 4; ++c) sum[b][c] += ((nib >> c) & 1u) ? sp : sn;
        }
    }
}

// Whether the segment's incoming scales allow the grouped sum: every partial
// sum of +-scales is exact in fp64 when the nonzero scales' exponents span at
// most grouping_limit = 29 - ceil(log2 n) binades (and none is Inf or NaN).
// `first` holds the scale of row `lane` when n <= kServerRowBatch (already
// loaded); otherwise all n scales are read.  Every lane gets the answer.
__device__ __forceinline__ bool server_grouped(const ServerRows &in, int n, int grouping_limit,
                                               int lane, float first)
{
    int emax = 0, emin = 1 << 20;
    auto widen = [&](float sc) {
        const uint32_t u = __float_as_uint(sc) & 0x7FFFFFFFu;
        if (u == 0) return;
        const int e = max((int)(u >> 23), 1);
        emax = max(emax, e);
        emin = min(emin, e);
    };
    if (n <= kServerRowBatch)
        widen(first);
    else
        for (int r = lane; r < n; r += kWave) widen(in.scales[(int64_t)r * in.scales_ld]);
    emax = wave_max(emax);
    emin = wave_min(emin);
    return emax < 255 && (emax == 0 || emax - emin <= grouping_limit);
}

// The last part of a tile for every sub-block: average, add the server error,
// store the new compensated error state and the sign words; returns the
// wave's fp64 sum of squares of the tile (every lane gets it).  FULL and POW2
// are wave-uniform, so each wave runs one variant.
__device__ __forceinline__ double server_epilogue(const double (&sum)[kSubBlocks][4],
                                                  const v4f (&cv)[kSubBlocks], float sprev, int n,
                                                  int lane, const Tile &tile, bool full,
                                                  float *__restrict__ serr,
                                                  uint64_t *__restrict__ sbits)
{
    const bool pow2 = (n & (n - 1)) == 0;
    double acc = 0.0;
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        if (full && pow2)
            acc += server_epilogue_sub<true, true>(sum[b], cv[b], sprev, n, lane, tile, b, serr, sbits);
        else if (full)
            acc += server_epilogue_sub<true, false>(sum[b], cv[b], sprev, n, lane, tile, b, serr, sbits);
        else if (pow2)
            acc += server_epilogue_sub<false, true>(sum[b], cv[b], sprev, n, lane, tile, b, serr, sbits);
        else
            acc += server_epilogue_sub<false, false>(sum[b], cv[b], sprev, n, lane, tile, b, serr, sbits);
    }
    return wave_sum_dpp(acc);
}

// ---------------------------------------------------------------------------
// Tables of the owned segments, built once per call when the caller's
// workspace holds them: for owned segment u (segment q = k*n + j of chunk j
// in [cb, cb + nown), u = k*nown + j - cb) flags[u] says whether the grouped
// sum applies, and if so tables[(u*groups8 + g)*256 + idx] is the signed sum
// of the scales of rows 8g .. 8g+7 (+ where bit k of idx is set; rows past n
// add nothing).  One workgroup per (owned segment, group); each decides on
// the segment's flag by itself, and group 0's writes it.  Every entry is an
// exact fp64 sum when the flag is set, so it equals the in-kernel tables'.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_server_tables(
    int n, int cb, int nown, int grouping_limit, const float *__restrict__ wscales,
    int64_t scales_ld, int64_t scales_seg_base, double *__restrict__ tables,
    int32_t *__restrict__ flags)
{
    const int groups8 = (n + 7) >> 3;
    const int64_t u = blockIdx.x / groups8;
    const int g = blockIdx.x - u * groups8;
    const int64_t q = (u / nown) * n + cb + (u % nown);
    const float *sc = wscales + (q - scales_seg_base);
    const int lane = threadIdx.x & (kWave - 1);
    const ServerRows in{nullptr, 0, sc, scales_ld, 0, false};
    // every wave reads the n scales and reaches the same decision
    const float first = (n <= kServerRowBatch && lane < n) ? sc[(int64_t)lane * scales_ld] : 0.f;
    const bool ok = server_grouped(in, n, grouping_limit, lane, first);
    if (g == 0 && threadIdx.x == 0) flags[u] = ok ? 1 : 0;
    if (!ok) return;
    static_assert(kBlock == 256, "one table entry per thread");
    const int idx = threadIdx.x;
    double v = 0.0;
    for (int k = 0; k < 8 && 8 * g + k < n; ++k) {
        const double s = (double)sc[(int64_t)(8 * g + k) * scales_ld];
        v += ((idx >> k) & 1) ? s : -s;
    }
    tables[((u * groups8) + g) * 256 + idx] = v;
}

// Where a call's owned-segment tables and flags are, for the passes that copy
// them (passed by value as a kernel argument).
struct ServerTables {
    const double *tables;
    const int32_t *flags;
    int cb;    // first owned chunk
    int nown;  // owned chunks
};

// Copies the 256-entry tables of groups [g0, g0 + gcnt) of owned segment u
// into lut (gcnt 2 KB tables) with direct global-to-LDS loads, 1 KB per
// instruction: lane L's 16 bytes land at byte 16 L of each kilobyte.  The
// caller waits for them (vmcnt) before reading lut.
__device__ __forceinline__ void server_fetch_tables(double *lut, const ServerTables &st,
                                                    int64_t u, int groups8, int g0, int gcnt,
                                                    int lane)
{
    const char *src = (const char *)(st.tables + (u * groups8 + g0) * 256) + 16 * lane;
    for (int k = 0; k < 2 * gcnt; ++k)
        __builtin_amdgcn_global_load_lds((const void *)(src + 1024 * k),
                                         (__attribute__((address_space(3))) void *)((char *)lut +
                                                                                    1024 * k),
                                         16, 0, 0);
}

// Owned segment index of segment q.
__device__ __forceinline__ int64_t owned_segment(int64_t q, int n, const ServerTables &st)
{
    const int64_t k = q / n;
    return k * st.nown + (q - k * n) - st.cb;
}

// Waits for every vector memory operation of the wave, the direct-to-LDS
// table loads included (the compiler does not track those): s_waitcnt with
// vmcnt 0 (bits 3:0 and 15:14) and the expcnt (6:4) and lgkmcnt (11:8) fields
// at their maxima, which wait for nothing.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// ---------------------------------------------------------------------------
// Chunk owners' pass for n <= kServerRowBatch, one wave per tile, building
// the tables itself.  The tile's error-state and sign-word loads are issued
// first; the wave then reads the segment's scales, decides between the
// grouped and the one-by-one sum, and builds the 256-entry tables of every
// group of 8 workers (the 16-entry tables first, in the staging area, before
// the words are staged).  The words are then staged and regrouped, every
// group is looked up, and the tile is finished.  Each wave owns its LDS area,
// so it synchronises only with itself.
// ---------------------------------------------------------------------------
// With one group of 8 workers (n <= 8) the tables leave LDS for five
// workgroups per CU; asking for five waves per SIMD keeps the registers
// there too (95 instead of 126 VGPRs, no spills): 0.90 -> 0.86 ms on the
// stress workload.  Larger G8 is limited by its LDS.
template <int G8>  // groups of 8 workers the LDS tables hold: n <= 8 G8
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(G8 == 1 ? 5 : 1))) void k_server_pass(
    const Tile *__restrict__ tiles, const int32_t *__restrict__ chunk_tiles, int64_t tile_begin,
    int64_t tile_count, int n,
    int grouping_limit, const uint64_t *__restrict__ wbits, int64_t bits_ld,
    int64_t bits_word_base, const float *__restrict__ wscales, int64_t scales_ld,
    int64_t scales_seg_base, float *__restrict__ serr, const float *__restrict__ sscales,
    uint64_t *__restrict__ sbits, double *__restrict__ partial)
{
    __shared__ __align__(16) ServerTileLds<G8> s_lds[kWavesPerBlock];
    const int lane = threadIdx.x & (kWave - 1);
    // wave-uniform: the tile and its fields live in scalar registers
    const int wv = wave_id();
    const int64_t rel = xcd_block() * kWavesPerBlock + wv;
    if (rel >= tile_count) return;
    ServerTileLds<G8> &L = s_lds[wv];
    const int groups8 = (n + 7) >> 3;
    const int64_t t = chunk_tiles[tile_begin + rel];
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const ServerRows in{wbits + ((base >> 6) - bits_word_base), bits_ld,
                        wscales + ((int64_t)tile.seg - scales_seg_base), scales_ld,
                        (len + 63) >> 6, len == kTileElems};
    const float sprev = sscales[tile.seg];
    v4f cv[kSubBlocks];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        cv[b] = in.full ? ld4<true>(serr + base, li, len) : ld4<false>(serr + base, li, len);
    }
    uint64_t stg[kServerRowBatch / 4];
    server_load_words(in, 0, n, lane, stg);
    const float scl = lane < n ? in.scales[(int64_t)lane * in.scales_ld] : 0.f;
    const bool grouped = server_grouped(in, n, grouping_limit, lane, scl);
    if (lane < n) L.scale[lane] = scl;
    if (grouped) {
        wave_sync();
        server_build_lut4(L, n, lane);
        wave_sync();
#pragma unroll
        for (int k = 0; k < G8 * 256 / kWave; ++k) {
            const int e = lane + kWave * k;
            const int g = e >> 8, idx = e & 255;  // g = k / 4: uniform
            if (g < groups8)
                L.lut8[g][idx] = L.lut4[2 * g][idx & 15] + L.lut4[2 * g + 1][idx >> 4];
        }
        wave_sync();  // lut4 shares the staging area
    }
    server_stage_words(L, in, n, lane, stg);
    wave_sync();
    double sum[kSubBlocks][4];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[b][c] = 0.0;
    if (grouped) {
        server_regroup_bits(L, n, lane);
        wave_sync();
        for (int g = 0; g < groups8; ++g) server_lookup_group(sum, L, 8 * g, L.lut8[g], lane);
    } else {
        server_batch_one_by_one(sum, L, n, lane);
    }
    const double acc = server_epilogue(sum, cv, sprev, n, lane, tile, in.full, serr, sbits);
    if (lane == 0) partial[t] = acc;
}

// ---------------------------------------------------------------------------
// Chunk owners' pass for n <= kServerRowBatch with the tables in the
// workspace: each workgroup takes up to kWavesPerBlock consecutive tiles of
// one segment (entry b of `blocks`, one tile per wave) and shares one copy of
// the segment's tables, wave g copying group g's.  The tile loads are issued
// first; after one workgroup barrier (tables and staged words in place) each
// wave regroups its own words, looks every group up and finishes its tile.
// One shared table set instead of one per wave leaves room in LDS for five
// workgroups per CU.
// ---------------------------------------------------------------------------
struct ServerSharedLds {
    uint32_t bits[kWavesPerBlock][2 * kTileWords][kBitsStride];
    double lut8[kServerRowBatch / 8][256];
    float scale[kServerRowBatch];
};

// One wave's part of it, in the form the staging and summing helpers take.
struct ServerWaveLds {
    uint32_t (&bits)[2 * kTileWords][kBitsStride];
    float (&scale)[kServerRowBatch];
};

// Five waves per SIMD (90 instead of 122 VGPRs, no spills; the 28.8 KB of
// LDS per workgroup allows five per CU): 0.71 -> 0.69 ms on the BERT-Large
// shape, 0.21 -> 0.19 ms on BERT-Base.
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(5))) void k_server_shared(
    const Tile *__restrict__ tiles, const int32_t *__restrict__ chunk_tiles,
    const int32_t *__restrict__ blocks, int64_t num_blocks, int n,
    const uint64_t *__restrict__ wbits, int64_t bits_ld, int64_t bits_word_base,
    const float *__restrict__ wscales, int64_t scales_ld, int64_t scales_seg_base,
    float *__restrict__ serr, const float *__restrict__ sscales, uint64_t *__restrict__ sbits,
    double *__restrict__ partial, ServerTables st)
{
    __shared__ __align__(16) ServerSharedLds S;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = wave_id();
    const int64_t b = xcd_block();
    if (b >= num_blocks) return;  // the whole workgroup
    const int32_t entry = blocks[b];
    const int64_t first = server_block_first(entry);
    const bool has = wv < server_block_tiles(entry);
    const int groups8 = (n + 7) >> 3;
    // every tile of the workgroup is in this segment
    const int seg = tiles[chunk_tiles[first]].seg;
    const int64_t u = owned_segment(seg, n, st);
    const bool grouped = st.flags[u] != 0;
    const int64_t t = chunk_tiles[first + (has ? wv : 0)];
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const ServerRows in{wbits + ((base >> 6) - bits_word_base), bits_ld,
                        wscales + ((int64_t)seg - scales_seg_base), scales_ld,
                        (len + 63) >> 6, len == kTileElems};
    const float sprev = sscales[seg];
    v4f cv[kSubBlocks];
    uint64_t stg[kServerRowBatch / 4];
    if (has) {
#pragma unroll
        for (int k = 0; k < kSubBlocks; ++k) {
            const int li = k * (kWave * 4) + 4 * lane;
            cv[k] = in.full ? ld4<true>(serr + base, li, len) : ld4<false>(serr + base, li, len);
        }
        server_load_words(in, 0, n, lane, stg);
    }
    if (grouped) {
        if (wv < groups8) server_fetch_tables(&S.lut8[wv][0], st, u, groups8, wv, 1, lane);
    } else if (wv == 0 && lane < n) {
        S.scale[lane] = in.scales[(int64_t)lane * in.scales_ld];
    }
    ServerWaveLds L{S.bits[wv], S.scale};
    if (has) server_stage_words(L, in, n, lane, stg);
    wait_vmem();
    __syncthreads();
    if (!has) return;
    double sum[kSubBlocks][4];
#pragma unroll
    for (int k = 0; k < kSubBlocks; ++k)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[k][c] = 0.0;
    if (grouped) {
        server_regroup_bits(L, n, lane);
        wave_sync();
        for (int g = 0; g < groups8; ++g) server_lookup_group(sum, L, 8 * g, S.lut8[g], lane);
    } else {
        server_batch_one_by_one(sum, L, n, lane);
    }
    const double acc = server_epilogue(sum, cv, sprev, n, lane, tile, in.full, serr, sbits);
    if (lane == 0) partial[t] = acc;
}

// ---------------------------------------------------------------------------
// Chunk owners' pass for many workers (n > kServerRowBatch) with the tables in
// the workspace: one workgroup per tile, wave w owning sub-block w of it (256
// elements: words 4w .. 4w+3).  The waves walk the incoming rows together in
// batches of kServerRowBatch: each loads and stages its own sub-block's words
// of the batch (4 words of each of 32 rows), the four share the batch's
// tables (wave g copies group g's), and the next batch's words and tables are
// on their way while a batch is looked up (two table buffers, one workgroup
// barrier per batch).  No partial sums are exchanged: each wave finishes its
// own sub-block, and the tile's sum of squares adds the four waves' in a
// fixed order.
// ---------------------------------------------------------------------------
struct ServerSubLds {
    uint32_t bits[kSubBlocks][2 * kTileWords / kSubBlocks][kBitsStride];  // each wave's 8 half-words
    double lut8[2][kServerRowBatch / 8][256];  // batch b's tables in lut8[b & 1]
    float scale[2][kServerRowBatch];           // batch b's scales (one-by-one sum)
    double red[kSubBlocks];
};

// Loads the words of sub-block w of rows [r0, r0 + rows) of the tile (rows <=
// kServerRowBatch): lane L takes word 4w + L % 4 of rows r0 + L/4 and
// r0 + L/4 + 16 (zero past the batch's rows and the tile's words).
__device__ __forceinline__ void server_load_sub_words(const ServerRows &in, int w, int r0,
                                                      int rows, int lane, uint64_t (&stg)[2])
{
    const int wi = 4 * w + (lane & 3);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int r = (lane >> 2) + 16 * k;
        stg[k] = (r < rows && wi < in.nwords)
                     ? __builtin_nontemporal_load(in.words + (int64_t)(r0 + r) * in.bits_ld + wi)
                     : 0ull;
    }
}

// Writes them into the wave's staging area ([local half-word][row]; the
// rows past the batch's last row, up to the next multiple of 8, get zero
// words).
__device__ __forceinline__ void server_stage_sub_words(uint32_t (&bits)[2 * kTileWords /
                                                                          kSubBlocks][kBitsStride],
                                                       int rows, int lane,
                                                       const uint64_t (&stg)[2])
{
    const int j = lane & 3;
    const int rows8 = (rows + 7) & ~7;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int r = (lane >> 2) + 16 * k;
        if (r < rows8) {
            bits[2 * j][r] = (uint32_t)stg[k];
            bits[2 * j + 1][r] = (uint32_t)(stg[k] >> 32);
        }
    }
}

__global__ __launch_bounds__(kSubBlocks * kWave) void k_server_subblocks(
    const Tile *__restrict__ tiles, const int32_t *__restrict__ chunk_tiles, int64_t tile_begin,
    int64_t tile_count, int n, const uint64_t *__restrict__ wbits, int64_t bits_ld,
    int64_t bits_word_base, const float *__restrict__ wscales, int64_t scales_ld,
    int64_t scales_seg_base, float *__restrict__ serr, const float *__restrict__ sscales,
    uint64_t *__restrict__ sbits, double *__restrict__ partial, ServerTables st)
{
    __shared__ __align__(16) ServerSubLds S;
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = wave_id();
    const int64_t rel = xcd_block();
    if (rel >= tile_count) return;  // the whole workgroup
    const int64_t t = chunk_tiles[tile_begin + rel];
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const ServerRows in{wbits + ((base >> 6) - bits_word_base), bits_ld,
                        wscales + ((int64_t)tile.seg - scales_seg_base), scales_ld,
                        (len + 63) >> 6, len == kTileElems};
    const int groups8 = (n + 7) >> 3;
    const int64_t u = owned_segment(tile.seg, n, st);
    const bool grouped = st.flags[u] != 0;
    const float sprev = sscales[tile.seg];
    const int li = wv * (kWave * 4) + 4 * lane;  // this wave's sub-block
    const v4f cv = in.full ? ld4<true>(serr + base, li, len) : ld4<false>(serr + base, li, len);
    uint64_t stg[2];
    const int rows0 = min(kServerRowBatch, n);
    server_load_sub_words(in, wv, 0, rows0, lane, stg);
    if (grouped && wv < ((rows0 + 7) >> 3))
        server_fetch_tables(&S.lut8[0][wv][0], st, u, groups8, wv, 1, lane);
    auto &bits = S.bits[wv];
    const int hw = lane >> 3;  // the lane's half-word of the sub-block
    const int o = 16 * (lane & 1) + ((lane & 7) >> 1);
    double sum[4] = {0.0, 0.0, 0.0, 0.0};
    for (int r0 = 0; r0 < n; r0 += kServerRowBatch) {  // workgroup-uniform
        const int cur = (r0 / kServerRowBatch) & 1;
        const int rows = min(kServerRowBatch, n - r0);
        const int g8 = (rows + 7) >> 3;
        if (!grouped && wv == 0 && lane < rows)
            S.scale[cur][lane] = in.scales[(int64_t)(r0 + lane) * in.scales_ld];
        server_stage_sub_words(bits, rows, lane, stg);
        wait_vmem();
        // this batch's tables, scales and words are in place, and every wave
        // is done with the previous batch (whose buffers come next)
        __syncthreads();
        const int r1 = r0 + kServerRowBatch;
        if (r1 < n) {
            const int rows1 = min(kServerRowBatch, n - r1);
            if (grouped && wv < ((rows1 + 7) >> 3))
                server_fetch_tables(&S.lut8[cur ^ 1][wv][0], st, u, groups8, (r1 >> 3) + wv, 1,
                                    lane);
            server_load_sub_words(in, wv, r1, rows1, lane, stg);
        }
        if (grouped) {
            // regroup the sub-block's (half-word, group of 8 rows) blocks
            if (lane < 8 * g8) {
                uint32_t *p = &bits[lane & 7][8 * (lane >> 3)];
                const uint4 u0 = *(const uint4 *)p;
                const uint4 u1 = *(const uint4 *)(p + 4);
                uint32_t a[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
                transpose_bits8x8(a);
                *(uint4 *)p = make_uint4(a[0], a[1], a[2], a[3]);
                *(uint4 *)(p + 4) = make_uint4(a[4], a[5], a[6], a[7]);
            }
            wave_sync();
            for (int g = 0; g < g8; ++g) {
                const uint8_t *blk = (const uint8_t *)&bits[hw][8 * g];
                uint32_t idx[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) idx[c] = blk[o + 4 * c];
                double val[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) val[c] = S.lut8[cur][g][idx[c]];
#pragma unroll
                for (int c = 0; c < 4; ++c) sum[c] += val[c];
            }
        } else {
            const int shift = 4 * (lane & 7);
            for (int r = 0; r < rows; ++r) {
                const double sp = (double)S.scale[cur][r];
                const uint32_t nib = (bits[hw][r] >> shift) & 0xFu;
#pragma unroll
                for (int c = 0; c < 4; ++c) sum[c] += ((nib >> c) & 1u) ? sp : -sp;
            }
        }
        wave_sync();  // before this wave's staging area takes the next batch
    }
    const bool pow2 = (n & (n - 1)) == 0;
    double acc;
    if (in.full && pow2)
        acc = server_epilogue_sub<true, true>(sum, cv, sprev, n, lane, tile, wv, serr, sbits);
    else if (in.full)
        acc = server_epilogue_sub<true, false>(sum, cv, sprev, n, lane, tile, wv, serr, sbits);
    else if (pow2)
        acc = server_epilogue_sub<false, true>(sum, cv, sprev, n, lane, tile, wv, serr, sbits);
    else
        acc = server_epilogue_sub<false, false>(sum, cv, sprev, n, lane, tile, wv, serr, sbits);
    acc = wave_sum_dpp(acc);
    if (lane == 0) S.red[wv] = acc;
    __syncthreads();
    if (threadIdx.x == 0) partial[t] = (S.red[0] + S.red[1]) + (S.red[2] + S.red[3]);
}

// ---------------------------------------------------------------------------
// Chunk owners' pass for many workers (n > kServerRowBatch): the
// kSplitWaves waves of a workgroup share one tile.  When the grouped sum
// applies, wave w takes row batches w, w + kSplitWaves, ...; the waves' exact
// partial sums are then added through LDS (exact, so in any order), and wave
// w finishes sub-block w of the tile.  Otherwise wave 0 adds every row one by
// one in worker order and hands the other waves their sub-blocks.  Every wave
// reads the n scales and builds each batch's tables itself (the pass with the
// tables in the workspace is k_server_subblocks).
// ---------------------------------------------------------------------------
constexpr int kSplitWaves = kSubBlocks;

__global__ __launch_bounds__(kSplitWaves * kWave) void k_server_split(
    const Tile *__restrict__ tiles, const int32_t *__restrict__ chunk_tiles, int64_t tile_begin,
    int64_t tile_count, int n, int grouping_limit, const uint64_t *__restrict__ wbits,
    int64_t bits_ld, int64_t bits_word_base, const float *__restrict__ wscales,
    int64_t scales_ld, int64_t scales_seg_base, float *__restrict__ serr,
    const float *__restrict__ sscales, uint64_t *__restrict__ sbits, double *__restrict__ partial)
{
    // the staging areas while rows are summed, then the exchange of partial
    // sums: xch[sub-block][source wave][element of the sub-block]
    union SplitLds {
        ServerBatchLds batch[kSplitWaves];
        double xch[kSubBlocks][kSplitWaves][kWave * 4];
    };
    __shared__ __align__(16) SplitLds s_lds;
    __shared__ double s_red[kSplitWaves];
    const int lane = threadIdx.x & (kWave - 1);
    const int wv = wave_id();
    const int64_t rel = xcd_block();
    if (rel >= tile_count) return;  // the whole workgroup
    const int64_t t = chunk_tiles[tile_begin + rel];
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const ServerRows in{wbits + ((base >> 6) - bits_word_base), bits_ld,
                        wscales + ((int64_t)tile.seg - scales_seg_base), scales_ld,
                        (len + 63) >> 6, len == kTileElems};
    ServerBatchLds &L = s_lds.batch[wv];

    const float sprev = sscales[tile.seg];
    const int li = wv * (kWave * 4) + 4 * lane;  // this wave's sub-block
    const v4f cv = in.full ? ld4<true>(serr + base, li, len) : ld4<false>(serr + base, li, len);
    uint64_t stg[kServerRowBatch / 4];
    float scl = 0.f;
    const int rfirst = kServerRowBatch * wv;  // may be past n when n <= 96: no rows then
    server_load_batch(in, rfirst, max(0, min(kServerRowBatch, n - rfirst)), lane, stg, scl);
    // every wave reads all n scales and reaches the same decision
    const bool grouped = server_grouped(in, n, grouping_limit, lane, 0.f);
    double sum[kSubBlocks][4];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[b][c] = 0.0;
    if (grouped) {
        constexpr int kStep = kServerRowBatch * kSplitWaves;
        for (int r0 = rfirst; r0 < n; r0 += kStep) {
            const int rows = min(kServerRowBatch, n - r0);
            server_stage_batch(L, in, rows, lane, stg, scl);
            // the next batch's words travel while this one is summed
            if (r0 + kStep < n)
                server_load_batch(in, r0 + kStep, min(kServerRowBatch, n - r0 - kStep), lane, stg,
                                  scl);
            wave_sync();
            server_batch_grouped(sum, L, rows, lane);
            wave_sync();
        }
    } else if (wv == 0) {
        for (int r0 = 0; r0 < n; r0 += kServerRowBatch) {
            const int rows = min(kServerRowBatch, n - r0);
            if (r0 > 0) server_load_batch(in, r0, rows, lane, stg, scl);
            server_stage_batch(L, in, rows, lane, stg, scl);
            wave_sync();
            server_batch_one_by_one(sum, L, rows, lane);
            wave_sync();
        }
    }
    __syncthreads();  // every wave is done with its staging area
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        if (b == wv) continue;
        double2 *dst = (double2 *)&s_lds.xch[b][wv][4 * lane];
        dst[0] = make_double2(sum[b][0], sum[b][1]);
        dst[1] = make_double2(sum[b][2], sum[b][3]);
    }
    __syncthreads();
    double s4[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) s4[c] = sum[wv][c];
#pragma unroll
    for (int w = 0; w < kSplitWaves; ++w) {
        if (w == wv) continue;
        const double2 *src = (const double2 *)&s_lds.xch[wv][w][4 * lane];
        const double2 a = src[0], b = src[1];
        s4[0] += a.x;
        s4[1] += a.y;
        s4[2] += b.x;
        s4[3] += b.y;
    }
    const bool pow2 = (n & (n - 1)) == 0;
    double acc;
    if (in.full && pow2)
        acc = server_epilogue_sub<true, true>(s4, cv, sprev, n, lane, tile, wv, serr, sbits);
    else if (in.full)
        acc = server_epilogue_sub<true, false>(s4, cv, sprev, n, lane, tile, wv, serr, sbits);
    else if (pow2)
        acc = server_epilogue_sub<false, true>(s4, cv, sprev, n, lane, tile, wv, serr, sbits);
    else
        acc = server_epilogue_sub<false, false>(s4, cv, sprev, n, lane, tile, wv, serr, sbits);
    acc = wave_sum_dpp(acc);
    if (lane == 0) s_red[wv] = acc;
    __syncthreads();
    if (threadIdx.x == 0) partial[t] = (s_red[0] + s_red[1]) + (s_red[2] + s_red[3]);
}


// ---------------------------------------------------------------------------
// Decompress + preconditioned update: x -= lr * (+-scale) / sqrt(v + eps).
// ---------------------------------------------------------------------------
// Every load of a wave's part of the tile is issued before its first store.
// Kernels here keep that order wherever a wave would otherwise re-read data
// after storing: on
// this hardware a variant that interleaved the sign-word loads with the
// stores returned wrong words for about 1% of the elements of a 334M-element
// launch (exact on small grids), and the loads-first form is exact.
// Sub-blocks sb0 .. sb0+SB-1 of the tile.
template <bool FULL, int SB>
__device__ __forceinline__ void update_tile(const Tile &tile, int lane, int sb0,
                                            const uint64_t *__restrict__ sbits, float s,
                                            float *__restrict__ x, float *__restrict__ m_out,
                                            const float *__restrict__ v, float lr, float eps)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    uint64_t word[SB];
    v4f xv[SB], vv[SB];
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int sb = sb0 + b;
        const int li = sb * (kWave * 4) + 4 * lane;
        const bool in = FULL || li < len;
        word[b] = in ? sbits[(base >> 6) + 4 * sb + (lane >> 4)] : 0ull;
        xv[b] = ld4<FULL>(x + base, li, len);
        vv[b] = ld4<FULL>(v + base, li, len);
    }
#pragma unroll
    for (int b = 0; b < SB; ++b) {
        const int li = (sb0 + b) * (kWave * 4) + 4 * lane;
        const uint32_t nib = (uint32_t)(word[b] >> (4 * (lane & 15))) & 0xFu;
        v4f mv;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float mbar = ((nib >> c) & 1u) ? s : -s;
            const float denom = __builtin_sqrtf(vv[b][c] + eps);
            const float ratio = mbar / denom;
            const float step = lr * ratio;
            xv[b][c] = xv[b][c] - step;
            mv[c] = mbar;
        }
        st4<FULL>(x + base, li, len, xv[b]);
        if (m_out) st4<FULL>(m_out + base, li, len, mv);
    }
}

// One 256-element sub-block per wave, four waves per tile: each wave keeps
// 2 KB of loads in flight instead of 8 KB (a whole tile), which the mix of
// two read streams and one written stream favours: 0.667 -> 0.619 ms on the
// BERT-Large shape, 1.112 -> 1.033 ms on the 5,000-tensor stress workload
// (half a tile per wave: 0.640 and 1.070 ms), in one A/B process each.
constexpr int kUpdateSubBlocks = 1;
constexpr int kUpdateWavesPerTile = kSubBlocks / kUpdateSubBlocks;

__global__ __launch_bounds__(kBlock) void k_update(
    const Tile *__restrict__ tiles, int64_t num_tiles, const uint64_t *__restrict__ sbits,
    const float *__restrict__ sscales, float *__restrict__ x, float *__restrict__ m_out,
    const float *__restrict__ v, float lr, float eps)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t w = xcd_block() * kWavesPerBlock + (threadIdx.x >> 6);
    const int64_t t = w / kUpdateWavesPerTile;
    const int sb0 = (int)(w % kUpdateWavesPerTile) * kUpdateSubBlocks;
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const float s = sscales[tile.seg];
    if (tile.len == kTileElems)
        update_tile<true, kUpdateSubBlocks>(tile, lane, sb0, sbits, s, x, m_out, v, lr, eps);
    else
        update_tile<false, kUpdateSubBlocks>(tile, lane, sb0, sbits, s, x, m_out, v, lr, eps);
}

// ---------------------------------------------------------------------------
// Explicit error from the compensated form.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_materialize(
    const Tile *__restrict__ tiles, int64_t num_tiles, int rows, const float *err,
    int64_t err_ld, const float *__restrict__ scales, int64_t scales_ld, float *out,
    int64_t out_ld)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = xcd_block() * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    for (int r = 0; r < rows; ++r) {
        const float s = scales[(int64_t)r * scales_ld + tile.seg];
#pragma unroll
        for (int b = 0; b < kSubBlocks; ++b) {
            const int li = b * (kWave * 4) + 4 * lane;
            if (li >= len) break;
            v4f zv = ld4<false>(err + (int64_t)r * err_ld + base, li, len);
#pragma unroll
            for (int c = 0; c < 4; ++c) zv[c] = error_of(zv[c], s);
            st4<false>(out + (int64_t)r * out_ld + base, li, len, zv);
        }
    }
}

// ---------------------------------------------------------------------------
// Decoded message: out = +-scale of each element's segment.
// ---------------------------------------------------------------------------
template <bool FULL>
__device__ __forceinline__ void decode_tile(const Tile &tile, int lane,
                                            const uint64_t *__restrict__ bits, float s,
                                            float *__restrict__ out)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    uint64_t word[kSubBlocks];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        word[b] = (FULL || li < len) ? bits[(base >> 6) + 4 * b + (lane >> 4)] : 0ull;
    }
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        const uint32_t nib = (uint32_t)(word[b] >> (4 * (lane & 15))) & 0xFu;
        v4f v;
#pragma unroll
        for (int c = 0; c < 4; ++c) v[c] = ((nib >> c) & 1u) ? s : -s;
        st4<FULL>(out + base, li, len, v);
    }
}

__global__ __launch_bounds__(kBlock) void k_decode(const Tile *__restrict__ tiles,
                                                   int64_t num_tiles,
                                                   const uint64_t *__restrict__ bits,
                                                   const float *__restrict__ scales,
                                                   float *__restrict__ out)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = xcd_block() * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const float s = scales[tile.seg];
    if (tile.len == kTileElems) decode_tile<true>(tile, lane, bits, s, out);
    else decode_tile<false>(tile, lane, bits, s, out);
}

// ---------------------------------------------------------------------------
// l1 norm of a buffer over the real elements (the variance-stability
// indicator of Section 7.1): per-tile fp64 partial sums of |v| (fixed lane
// order), then one workgroup sums the partials in a fixed order.
// ---------------------------------------------------------------------------
template <bool FULL>
__device__ __forceinline__ double l1_tile(const Tile &tile, int lane, const float *__restrict__ v)
{
    const int len = tile.len;
    const int64_t base = tile.start;
    v4f vv[kSubBlocks];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) vv[b] = ld4<FULL>(v + base, b * (kWave * 4) + 4 * lane, len);
    double acc = 0.0;
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc += (double)__builtin_fabsf(vv[b][c]);
    return acc;
}

__global__ __launch_bounds__(kBlock) void k_l1_partial(const Tile *__restrict__ tiles,
                                                       int64_t num_tiles,
                                                       const float *__restrict__ v,
                                                       double *__restrict__ partial)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = xcd_block() * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    double acc = tile.len == kTileElems ? l1_tile<true>(tile, lane, v) : l1_tile<false>(tile, lane, v);
    acc = wave_sum(acc);
    if (lane == 0) partial[t] = acc;
}

__global__ __launch_bounds__(kBlock) void k_l1_final(const double *__restrict__ partial,
                                                     int64_t num_tiles, double *__restrict__ out)
{
    __shared__ double red[kWavesPerBlock];
    double s = 0.0;
    for (int64_t t = threadIdx.x; t < num_tiles; t += kBlock) s += partial[t];
    s = wave_sum(s);
    if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) out[0] = ((red[0] + red[1]) + red[2]) + red[3];
}

// Workgroups (of kWavesPerBlock waves) for one wave per item.
inline int64_t blocks_for(int64_t waves) { return xcd_grid(waves, kWavesPerBlock); }

}  // namespace

template <class G>
static hipError_t launch_warmup_t(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                                  float *v, const void *g, int64_t g_ld, int n_grads, float lr,
                                  float beta1, float beta2, float eps, int use_bc, float bc1,
                                  float bc2, hipStream_t s)
{
    const float omb1 = 1.0f - beta1, omb2 = 1.0f - beta2;
    hipLaunchKernelGGL(k_warmup<G>, dim3((unsigned)xcd_grid(num_tiles, kRowWaves)), dim3(kRowBlock), 0, s,
                       tb.tiles,
                       num_tiles, x, m, v, (const typename G::T *)g, g_ld, n_grads, lr, beta1,
                       omb1, beta2, omb2, eps, use_bc, bc1, bc2);
    return hipGetLastError();
}

hipError_t launch_warmup(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                         float *v, const void *g, int grad_dtype, int64_t g_ld, int n_grads,
                         float lr, float beta1, float beta2, float eps, int use_bc, float bc1,
                         float bc2, hipStream_t s)
{
    switch (grad_dtype) {
    case kGradBF16:
        return launch_warmup_t<GradBF16>(tb, num_tiles, x, m, v, g, g_ld, n_grads, lr, beta1,
                                         beta2, eps, use_bc, bc1, bc2, s);
    case kGradF16:
        return launch_warmup_t<GradF16>(tb, num_tiles, x, m, v, g, g_ld, n_grads, lr, beta1,
                                        beta2, eps, use_bc, bc1, bc2, s);
    default:
        return launch_warmup_t<GradF32>(tb, num_tiles, x, m, v, g, g_ld, n_grads, lr, beta1,
                                        beta2, eps, use_bc, bc1, bc2, s);
    }
}

template <bool PACKED, class G>
static void launch_worker_t(const DeviceTables &tb, int64_t num_tiles, const float *m,
                            const uint64_t *m_bits, const float *m_scales, const void *g,
                            int64_t g_ld, float *err, int64_t err_ld, const float *scales,
                            int64_t scales_ld, uint64_t *bits, int64_t bits_ld, double *partial,
                            int n_local, int group, float beta1, hipStream_t s)
{
    const float omb1 = 1.0f - beta1;
    if constexpr (PACKED) {
        const int64_t groups = (n_local + group - 1) / group;
        const int64_t items = groups * num_tiles;
        const int64_t blocks = worker_grid(items, kMaxWorkerGridBlocks);
        hipLaunchKernelGGL((k_worker_pass<PACKED, G>), dim3((unsigned)blocks), dim3(kWorkerBlock),
                           0, s, tb.tiles, num_tiles, m, m_bits, m_scales,
                           (const typename G::T *)g, g_ld, err, err_ld, scales, scales_ld, bits,
                           bits_ld, partial, n_local, group, items, beta1, omb1);
    } else {
        (void)m_bits;
        (void)m_scales;
        (void)group;
        // every launch but the last covers exactly kMaxLaunchTiles tiles (its
        // grid has no spare workgroups), and the last one's spare waves see
        // t >= num_tiles
        static_assert(kMaxLaunchTiles % (kWorkerRowTiles * kXcds) == 0, "whole grids");
        for (int64_t base = 0; base < num_tiles; base += kMaxLaunchTiles) {
            const int64_t count = launch_piece(num_tiles, base);
            hipLaunchKernelGGL(k_worker_rows<G>, dim3((unsigned)xcd_grid(count, kWorkerRowTiles)),
                               dim3(kRowBlock), 0, s, tb.tiles, num_tiles, m,
                               (const typename G::T *)g, g_ld, err, err_ld, scales, scales_ld,
                               bits, bits_ld, partial, n_local, beta1, omb1, base);
        }
    }
}

template <class G>
static void launch_worker_g(const DeviceTables &tb, int64_t num_tiles, const float *m,
                            const uint64_t *m_bits, const float *m_scales, const void *g,
                            int64_t g_ld, float *err, int64_t err_ld, const float *scales,
                            int64_t scales_ld, uint64_t *bits, int64_t bits_ld, double *partial,
                            int n_local, int group, float beta1, hipStream_t s)
{
    if (m)
        launch_worker_t<false, G>(tb, num_tiles, m, m_bits, m_scales, g, g_ld, err, err_ld,
                                  scales, scales_ld, bits, bits_ld, partial, n_local, group,
                                  beta1, s);
    else
        launch_worker_t<true, G>(tb, num_tiles, m, m_bits, m_scales, g, g_ld, err, err_ld,
                                 scales, scales_ld, bits, bits_ld, partial, n_local, group,
                                 beta1, s);
}

hipError_t launch_worker_pass(const DeviceTables &tb, int64_t num_tiles, const float *m,
                              const uint64_t *m_bits, const float *m_scales, const void *g,
                              int grad_dtype, int64_t g_ld, float *err, int64_t err_ld,
                              const float *scales, int64_t scales_ld, uint64_t *bits,
                              int64_t bits_ld, double *partial, int n_local, int group,
                              float beta1, hipStream_t s)
{
    if (group < 1 || group > n_local) group = n_local;
    switch (grad_dtype) {
    case kGradBF16:
        launch_worker_g<GradBF16>(tb, num_tiles, m, m_bits, m_scales, g, g_ld, err, err_ld,
                                  scales, scales_ld, bits, bits_ld, partial, n_local, group,
                                  beta1, s);
        break;
    case kGradF16:
        launch_worker_g<GradF16>(tb, num_tiles, m, m_bits, m_scales, g, g_ld, err, err_ld,
                                 scales, scales_ld, bits, bits_ld, partial, n_local, group,
                                 beta1, s);
        break;
    default:
        launch_worker_g<GradF32>(tb, num_tiles, m, m_bits, m_scales, g, g_ld, err, err_ld,
                                 scales, scales_ld, bits, bits_ld, partial, n_local, group,
                                 beta1, s);
    }
    return hipGetLastError();
}

hipError_t launch_adam_message(const DeviceTables &tb, int64_t num_tiles, const uint64_t *bits,
                               const float *scales, float *x, float *m, float *v, float lr,
                               float beta1, float beta2, float eps, int use_bc, float bc1,
                               float bc2, hipStream_t s)
{
    const float omb1 = 1.0f - beta1, omb2 = 1.0f - beta2;
    hipLaunchKernelGGL(k_adam_message, dim3((unsigned)blocks_for(num_tiles * kAdamMessageWavesPerTile)),
                       dim3(kBlock), 0, s,
                       tb.tiles, num_tiles, bits, scales, x, m, v, lr, beta1, omb1, beta2, omb2,
                       eps, use_bc, bc1, bc2);
    return hipGetLastError();
}

template <class G>
static void launch_uncompressed_t(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                                  const float *v, const void *g, int64_t g_ld, int n, float lr,
                                  float beta1, float eps, hipStream_t s)
{
    const float omb1 = 1.0f - beta1;
    hipLaunchKernelGGL(k_uncompressed<G>, dim3((unsigned)xcd_grid(num_tiles, kRowWaves)),
                       dim3(kRowBlock), 0, s,
                       tb.tiles, num_tiles, x, m, v, (const typename G::T *)g, g_ld, n, lr, beta1,
                       omb1, eps);
}

hipError_t launch_uncompressed(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                               const float *v, const void *g, int grad_dtype, int64_t g_ld,
                               int n, float lr, float beta1, float eps, hipStream_t s)
{
    switch (grad_dtype) {
    case kGradBF16:
        launch_uncompressed_t<GradBF16>(tb, num_tiles, x, m, v, g, g_ld, n, lr, beta1, eps, s);
        break;
    case kGradF16:
        launch_uncompressed_t<GradF16>(tb, num_tiles, x, m, v, g, g_ld, n, lr, beta1, eps, s);
        break;
    default:
        launch_uncompressed_t<GradF32>(tb, num_tiles, x, m, v, g, g_ld, n, lr, beta1, eps, s);
    }
    return hipGetLastError();
}

hipError_t launch_l1_norm(const DeviceTables &tb, int64_t num_tiles, const float *v,
                          double *partial, double *out, hipStream_t s)
{
    if (num_tiles > 0)
        hipLaunchKernelGGL(k_l1_partial, dim3((unsigned)blocks_for(num_tiles)), dim3(kBlock), 0, s,
                           tb.tiles, num_tiles, v, partial);
    hipLaunchKernelGGL(k_l1_final, dim3(1), dim3(kBlock), 0, s, partial, num_tiles, out);
    return hipGetLastError();
}

hipError_t launch_decode(const DeviceTables &tb, int64_t num_tiles, const uint64_t *bits,
                         const float *scales, float *out, hipStream_t s)
{
    hipLaunchKernelGGL(k_decode, dim3((unsigned)blocks_for(num_tiles)), dim3(kBlock), 0, s, tb.tiles,
                       num_tiles, bits, scales, out);
    return hipGetLastError();
}

hipError_t launch_finalize(const DeviceTables &tb, int64_t max_seg_tiles, int64_t num_pairs,
                           int64_t num_segments, int server_form, int n, int jb, int je,
                           const double *partial, int64_t part_ld, float *scales,
                           int64_t scales_ld, hipStream_t s)
{
    if (num_pairs <= 0) return hipSuccess;
    if (max_seg_tiles > 4 * kWave) {
        hipLaunchKernelGGL(k_finalize<kBlock>, dim3((unsigned)std::min(num_pairs, kMaxGridBlocks)),
                           dim3(kBlock), 0, s, tb,
                           num_pairs, num_segments, server_form, n, jb, je, partial, part_ld,
                           scales, scales_ld);
    } else {
        hipLaunchKernelGGL(k_finalize<kWave>,
                           dim3((unsigned)std::min(blocks_for(num_pairs), kMaxGridBlocks)),
                           dim3(kBlock), 0, s,
                           tb, num_pairs, num_segments, server_form, n, jb, je, partial, part_ld,
                           scales, scales_ld);
    }
    return hipGetLastError();
}

size_t server_table_bytes(int n, int64_t segments)
{
    return (size_t)segments * (size_t)((n + 7) / 8) * 256 * sizeof(double);
}

hipError_t launch_server_pass(const DeviceTables &tb, int64_t tile_begin, int64_t tile_count,
                              int n, const uint64_t *wbits, int64_t bits_ld,
                              int64_t bits_word_base, const float *wscales, int64_t scales_ld,
                              int64_t scales_seg_base, float *serr, float *sscales,
                              uint64_t *sbits, double *partial, int num_tensors, int cb,
                              int nown, double *tables, int32_t *flags,
                              const int32_t *server_blocks, int64_t num_blocks, hipStream_t s)
{
    int log2n = 0;
    while ((1 << log2n) < n) ++log2n;
    const int grouping_limit = 29 - log2n;
    const ServerTables st{tables, flags, cb, nown};
    const bool use_tables = tables != nullptr;
    if (use_tables)
        hipLaunchKernelGGL(k_server_tables,
                           dim3((unsigned)((int64_t)num_tensors * nown * ((n + 7) / 8))),
                           dim3(kBlock), 0, s, n, cb, nown, grouping_limit, wscales, scales_ld,
                           scales_seg_base, tables, flags);
    // more than one batch of rows: the waves of a workgroup share each tile
    // (one workgroup per tile, launched kMaxLaunchTiles tiles at a time)
    if (n > kServerRowBatch) {
        for (int64_t off = 0; off < tile_count; off += kMaxLaunchTiles) {
            const int64_t count = launch_piece(tile_count, off);
            const dim3 grid((unsigned)xcd_grid(count, 1));
            if (use_tables)
                hipLaunchKernelGGL(k_server_subblocks, grid, dim3(kSubBlocks * kWave), 0, s,
                                   tb.tiles, tb.chunk_tiles, tile_begin + off, count, n, wbits,
                                   bits_ld, bits_word_base, wscales, scales_ld, scales_seg_base,
                                   serr, sscales, sbits, partial, st);
            else
                hipLaunchKernelGGL(k_server_split, grid, dim3(kSplitWaves * kWave), 0, s,
                                   tb.tiles, tb.chunk_tiles, tile_begin + off, count, n,
                                   grouping_limit, wbits, bits_ld, bits_word_base, wscales,
                                   scales_ld, scales_seg_base, serr, sscales, sbits, partial);
        }
    } else if (use_tables) {
        // a workgroup per entry of the block list (up to one per tile)
        for (int64_t off = 0; off < num_blocks; off += kMaxLaunchTiles) {
            const int64_t count = launch_piece(num_blocks, off);
            hipLaunchKernelGGL(k_server_shared, dim3((unsigned)xcd_grid(count, 1)), dim3(kBlock),
                               0, s, tb.tiles, tb.chunk_tiles, server_blocks + off, count, n,
                               wbits, bits_ld, bits_word_base, wscales, scales_ld,
                               scales_seg_base, serr, sscales, sbits, partial, st);
        }
    } else {
        // tables for as many groups of 8 as n needs: more workgroups per CU
        // for small n
        const dim3 grid((unsigned)blocks_for(tile_count)), block(kBlock);
        if (n <= 8)
            hipLaunchKernelGGL(k_server_pass<1>, grid, block, 0, s, tb.tiles, tb.chunk_tiles,
                               tile_begin, tile_count, n, grouping_limit, wbits, bits_ld,
                               bits_word_base, wscales, scales_ld, scales_seg_base, serr, sscales,
                               sbits, partial);
        else if (n <= 16)
            hipLaunchKernelGGL(k_server_pass<2>, grid, block, 0, s, tb.tiles, tb.chunk_tiles,
                               tile_begin, tile_count, n, grouping_limit, wbits, bits_ld,
                               bits_word_base, wscales, scales_ld, scales_seg_base, serr, sscales,
                               sbits, partial);
        else
            hipLaunchKernelGGL(k_server_pass<4>, grid, block, 0, s, tb.tiles, tb.chunk_tiles,
                               tile_begin, tile_count, n, grouping_limit, wbits, bits_ld,
                               bits_word_base, wscales, scales_ld, scales_seg_base, serr, sscales,
                               sbits, partial);
    }
    return hipGetLastError();
}

hipError_t launch_update(const DeviceTables &tb, int64_t num_tiles, const uint64_t *sbits,
                         const float *sscales, float *x, float *m_out, const float *v,
                         float lr, float eps, hipStream_t s)
{
    hipLaunchKernelGGL(k_update, dim3((unsigned)blocks_for(num_tiles * kUpdateWavesPerTile)),
                       dim3(kBlock), 0, s, tb.tiles,
                       num_tiles, sbits, sscales, x, m_out, v, lr, eps);
    return hipGetLastError();
}

hipError_t launch_materialize(const DeviceTables &tb, int64_t num_tiles, int rows,
                              const float *err, int64_t err_ld, const float *scales,
                              int64_t scales_ld, float *out, int64_t out_ld, hipStream_t s)
{
    hipLaunchKernelGGL(k_materialize, dim3((unsigned)blocks_for(num_tiles)), dim3(kBlock), 0, s,
                       tb.tiles, num_tiles, rows, err, err_ld, scales, scales_ld, out, out_ld);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Scratch memory of the entry point that allocates nothing: the per-tile
// fp64 partial sums that the caller's workspace holds otherwise.  Host code
// never uses the array's name as an address (on the host it is only a
// handle for the symbol lookup); it uses the per-device address that
// hipGetSymbolAddress returns.
// ---------------------------------------------------------------------------
static __device__ __align__(256) double scratch[kScratchBytes / sizeof(double)];

namespace {
std::once_flag g_scratch_once[kMaxScratchDevices];
void *g_scratch_ptr[kMaxScratchDevices];
hipError_t g_scratch_err[kMaxScratchDevices];
}  // namespace

hipError_t scratch_address(int device, void **ptr)
{
    *ptr = nullptr;
    if (device < 0 || device >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::call_once(g_scratch_once[device], [device] {
        int prev = -1;
        hipError_t e = hipGetDevice(&prev);
        if (e == hipSuccess && prev != device) e = hipSetDevice(device);
        void *p = nullptr;
        if (e == hipSuccess) e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (prev >= 0 && prev != device) {
            const hipError_t r = hipSetDevice(prev);
            if (e == hipSuccess) e = r;
        }
        g_scratch_err[device] = e;
        g_scratch_ptr[device] = e == hipSuccess ? p : nullptr;
    });
    *ptr = g_scratch_ptr[device];
    return g_scratch_err[device];
}

}  // namespace onebit
