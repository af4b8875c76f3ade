// gfx950 kernels of the 1-bit Adam hot path (arXiv 2102.02888).
//
// Every kernel is a bandwidth-bound stream over the flat parameter buffer; no
// MFMA (nothing here is a dense contraction).  Work is cut into tiles of up
// to 1024 elements that never cross a segment; one wavefront (64 lanes) owns
// one tile, each lane holding 4 sub-blocks x float4 = 16 elements, so every
// global load/store is a 128-bit access and a wave moves 1 KiB per
// instruction.  A sub-block of 256 elements spans four 16-lane DPP rows, and
// each row's 64 elements form one LSB-first uint64 sign word (bit b of word w
// of the tile <=> element 64w+b), assembled with a row-wide OR of the lanes'
// 4-bit nibbles.
//
// Arithmetic contract (shared with the layout/format description in
// onebit.h): fp32 values, one rounding per operation (built with
// -ffp-contract=off), correctly rounded sqrt and division, fp64 reductions
// rounded once to fp32.  Reductions over a segment are deterministic:
// per-tile partial sums (fixed lane order, xor butterfly) are written to a
// workspace and summed in a fixed order by a finalize kernel; no atomics.
#include "onebit_internal.h"

namespace onebit {
namespace {

__device__ __forceinline__ float4 load4(const float *__restrict__ p, int li, int len)
{
    if (li + 4 <= len) return *reinterpret_cast<const float4 *>(p + li);
    float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
    if (li < len) r.x = p[li];
    if (li + 1 < len) r.y = p[li + 1];
    if (li + 2 < len) r.z = p[li + 2];
    return r;
}

__device__ __forceinline__ void store4(float *__restrict__ p, int li, int len, float4 v)
{
    if (li + 4 <= len) {
        *reinterpret_cast<float4 *>(p + li) = v;
        return;
    }
    if (li < len) p[li] = v.x;
    if (li + 1 < len) p[li + 1] = v.y;
    if (li + 2 < len) p[li + 2] = v.z;
}

__device__ __forceinline__ float comp(const float4 &v, int c)
{
    return c == 0 ? v.x : c == 1 ? v.y : c == 2 ? v.z : v.w;
}

__device__ __forceinline__ void set_comp(float4 &v, int c, float a)
{
    if (c == 0) v.x = a;
    else if (c == 1) v.y = a;
    else if (c == 2) v.z = a;
    else v.w = a;
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

// Deterministic wave-wide fp64 sum (every lane gets the same value).
__device__ __forceinline__ double wave_sum(double a)
{
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) a += __shfl_xor(a, off, kWave);
    return a;
}

// Error from the compensated form: z - C[z] given z and its segment scale s.
__device__ __forceinline__ float error_of(float z, float s) { return z >= 0.f ? z - s : z + s; }

// ---------------------------------------------------------------------------
// Warm-up Adam (eq. (alg:v)) on the average of n_grads gradient rows.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_warmup(
    const Tile *__restrict__ tiles, int64_t num_tiles, float *__restrict__ x,
    float *__restrict__ m, float *__restrict__ v, const float *__restrict__ g, int64_t g_ld,
    int n_grads, float lr, float beta1, float omb1, float beta2, float omb2, float eps,
    int use_bc, float bc1, float bc2)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const double inv_n_div = (double)n_grads;
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        if (li >= len) break;
        double sum[4] = {0.0, 0.0, 0.0, 0.0};
        for (int i = 0; i < n_grads; ++i) {
            const float4 gv = load4(g + (int64_t)i * g_ld + base, li, len);
#pragma unroll
            for (int c = 0; c < 4; ++c) sum[c] += (double)comp(gv, c);
        }
        float4 xv = load4(x + base, li, len);
        float4 mv = load4(m + base, li, len);
        float4 vv = load4(v + base, li, len);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float gbar = (float)(sum[c] / inv_n_div);
            float mn = beta1 * comp(mv, c);
            mn = mn + omb1 * gbar;
            const float gsq = gbar * gbar;
            float vn = beta2 * comp(vv, c);
            vn = vn + omb2 * gsq;
            float mh = mn, vh = vn;
            if (use_bc) {
                mh = mn / bc1;
                vh = vn / bc2;
            }
            const float denom = __builtin_sqrtf(vh) + eps;
            const float ratio = mh / denom;
            const float step = lr * ratio;
            set_comp(xv, c, comp(xv, c) - step);
            set_comp(mv, c, mn);
            set_comp(vv, c, vn);
        }
        store4(x + base, li, len, xv);
        store4(m + base, li, len, mv);
        store4(v + base, li, len, vv);
    }
}

// ---------------------------------------------------------------------------
// Worker pass: for each local worker i, z_i = (beta1 m + (1-beta1) g_i) + delta_i,
// sign words of z_i, per-tile partial sum of z_i^2, and z_i written back as the
// new compensated error state.  m is read once per tile for all workers.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_worker_pass(
    const Tile *__restrict__ tiles, int64_t num_tiles, const float *__restrict__ m,
    const float *__restrict__ g, int64_t g_ld, float *__restrict__ err, int64_t err_ld,
    const float *__restrict__ scales, int64_t scales_ld, uint64_t *__restrict__ bits,
    int64_t bits_ld, double *__restrict__ partial, int n_local, float beta1, float omb1)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const int nwords = (len + 63) >> 6;

    float bm[kSubBlocks][4];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const float4 mv = load4(m + base, b * (kWave * 4) + 4 * lane, len);
#pragma unroll
        for (int c = 0; c < 4; ++c) bm[b][c] = beta1 * comp(mv, c);
    }

    for (int i = 0; i < n_local; ++i) {
        const float sp = scales[(int64_t)i * scales_ld + tile.seg];
        const float *gi = g + (int64_t)i * g_ld + base;
        float *ei = err + (int64_t)i * err_ld + base;
        uint64_t *bi = bits + (int64_t)i * bits_ld + (base >> 6);
        double acc = 0.0;
#pragma unroll
        for (int b = 0; b < kSubBlocks; ++b) {
            const int li = b * (kWave * 4) + 4 * lane;
            const float4 gv = load4(gi, li, len);
            const float4 cv = load4(ei, li, len);
            float4 zv;
            uint32_t nib = 0;
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const float d = error_of(comp(cv, c), sp);
                float mi = omb1 * comp(gv, c);
                mi = bm[b][c] + mi;
                const float z = mi + d;
                set_comp(zv, c, z);
                const bool valid = li + c < len;
                const double zd = valid ? (double)z : 0.0;
                acc += zd * zd;
                nib |= (valid && z >= 0.f) ? (1u << c) : 0u;
            }
            store4(ei, li, len, zv);
            const uint64_t word = row_sign_word(nib, lane);
            const int w = 4 * b + (lane >> 4);
            if ((lane & 15) == 0 && w < nwords) bi[w] = word;
        }
        acc = wave_sum(acc);
        if (lane == 0) partial[(int64_t)i * num_tiles + t] = acc;
    }
}

// ---------------------------------------------------------------------------
// Scale finalize: scale = fp32(sqrt(sum over the segment's tiles / len)),
// summed by one wave in a fixed order; empty segments get 0.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float finalize_one(const double *__restrict__ part, int64_t tb,
                                              int64_t te, int64_t len, int lane)
{
    double s = 0.0;
    for (int64_t t = tb + lane; t < te; t += kWave) s += part[t];
    s = wave_sum(s);
    return len > 0 ? (float)__builtin_sqrt(s / (double)len) : 0.0f;
}

__global__ __launch_bounds__(kBlock) void k_worker_finalize(
    DeviceTables tb, int64_t num_segments, int rows, const double *__restrict__ partial,
    int64_t part_ld, float *__restrict__ scales, int64_t scales_ld)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t p = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (p >= (int64_t)rows * num_segments) return;
    const int64_t i = p / num_segments, q = p % num_segments;
    const float s = finalize_one(partial + i * part_ld, tb.seg_tile_begin[q],
                                 tb.seg_tile_end[q], tb.seg_len[q], lane);
    if (lane == 0) scales[i * scales_ld + q] = s;
}

__global__ __launch_bounds__(kBlock) void k_server_finalize(
    DeviceTables tb, int K, int n, int jb, int je, const double *__restrict__ partial,
    float *__restrict__ sscales)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t p = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    const int cnt = je - jb;
    if (p >= (int64_t)K * cnt) return;
    const int64_t q = (p / cnt) * n + jb + (p % cnt);
    const float s = finalize_one(partial, tb.seg_tile_begin[q], tb.seg_tile_end[q],
                                 tb.seg_len[q], lane);
    if (lane == 0) sscales[q] = s;
}

// ---------------------------------------------------------------------------
// Server pass over the tiles of the owned chunks: decode and average the n
// incoming messages (fp64, worker order), add the server error, write the
// sign words and the new compensated server state, and the tile's sum of
// squares.  Incoming sign words are staged in LDS 32 worker rows at a time
// with coalesced 128-byte row reads; each lane then reads the one word that
// covers its 4 elements of a sub-block (a broadcast read, no bank conflict).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_server_pass(
    const Tile *__restrict__ tiles, int64_t tile_begin, int64_t tile_count, int n,
    const uint64_t *__restrict__ wbits, int64_t bits_ld, int64_t bits_word_base,
    const float *__restrict__ wscales, int64_t scales_ld, int64_t scales_seg_base,
    float *__restrict__ serr, const float *__restrict__ sscales,
    uint64_t *__restrict__ sbits, double *__restrict__ partial)
{
    __shared__ uint64_t s_bits[kWavesPerBlock][kServerRowBatch][kTileWords];
    __shared__ float s_scale[kWavesPerBlock][kServerRowBatch];

    const int lane = threadIdx.x & (kWave - 1);
    const int wv = threadIdx.x >> 6;
    const int64_t rel = (int64_t)blockIdx.x * kWavesPerBlock + wv;
    const bool active = rel < tile_count;  // no early exit: the block syncs below
    const int64_t t = tile_begin + (active ? rel : 0);
    const Tile tile = tiles[t];
    const int len = active ? tile.len : 0;
    const int64_t base = tile.start;
    const int nwords = (len + 63) >> 6;
    const int64_t w0 = (base >> 6) - bits_word_base;
    const int64_t sq = (int64_t)tile.seg - scales_seg_base;

    double sum[kSubBlocks][4];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b)
#pragma unroll
        for (int c = 0; c < 4; ++c) sum[b][c] = 0.0;

    for (int r0 = 0; r0 < n; r0 += kServerRowBatch) {
        const int rows = min(kServerRowBatch, n - r0);
        {
            const int wi = lane & (kTileWords - 1);
#pragma unroll
            for (int k = 0; k < kServerRowBatch / 4; ++k) {
                const int r = (lane >> 4) + 4 * k;
                if (r < rows && wi < nwords)
                    s_bits[wv][r][wi] = wbits[(int64_t)(r0 + r) * bits_ld + w0 + wi];
            }
            if (lane < rows && active)
                s_scale[wv][lane] = wscales[(int64_t)(r0 + lane) * scales_ld + sq];
        }
        __syncthreads();
        if (active) {
            for (int r = 0; r < rows; ++r) {
                const double sp = (double)s_scale[wv][r];
                const double sn = -sp;
#pragma unroll
                for (int b = 0; b < kSubBlocks; ++b) {
                    const uint64_t word = s_bits[wv][r][4 * b + (lane >> 4)];
                    const uint32_t nib = (uint32_t)(word >> (4 * (lane & 15))) & 0xFu;
#pragma unroll
                    for (int c = 0; c < 4; ++c) sum[b][c] += ((nib >> c) & 1u) ? sp : sn;
                }
            }
        }
        __syncthreads();
    }
    if (!active) return;

    const float sprev = sscales[tile.seg];
    const double dn = (double)n;
    double acc = 0.0;
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        const float4 cv = load4(serr + base, li, len);
        float4 zv;
        uint32_t nib = 0;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float avg = (float)(sum[b][c] / dn);
            const float z = avg + error_of(comp(cv, c), sprev);
            set_comp(zv, c, z);
            const bool valid = li + c < len;
            const double zd = valid ? (double)z : 0.0;
            acc += zd * zd;
            nib |= (valid && z >= 0.f) ? (1u << c) : 0u;
        }
        store4(serr + base, li, len, zv);
        const uint64_t word = row_sign_word(nib, lane);
        const int w = 4 * b + (lane >> 4);
        if ((lane & 15) == 0 && w < nwords) sbits[(base >> 6) + w] = word;
    }
    acc = wave_sum(acc);
    if (lane == 0) partial[t] = acc;
}

// ---------------------------------------------------------------------------
// Decompress + preconditioned update: x -= lr * (+-scale) / sqrt(v + eps).
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kBlock) void k_update(
    const Tile *__restrict__ tiles, int64_t num_tiles, const uint64_t *__restrict__ sbits,
    const float *__restrict__ sscales, float *__restrict__ x, float *__restrict__ m_out,
    const float *__restrict__ v, float lr, float eps)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
    if (t >= num_tiles) return;
    const Tile tile = tiles[t];
    const int len = tile.len;
    const int64_t base = tile.start;
    const float s = sscales[tile.seg];
#pragma unroll
    for (int b = 0; b < kSubBlocks; ++b) {
        const int li = b * (kWave * 4) + 4 * lane;
        if (li >= len) break;
        const uint64_t word = sbits[(base >> 6) + 4 * b + (lane >> 4)];
        const uint32_t nib = (uint32_t)(word >> (4 * (lane & 15))) & 0xFu;
        float4 xv = load4(x + base, li, len);
        const float4 vv = load4(v + base, li, len);
        float4 mv;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float mbar = ((nib >> c) & 1u) ? s : -s;
            const float denom = __builtin_sqrtf(comp(vv, c) + eps);
            const float ratio = mbar / denom;
            const float step = lr * ratio;
            set_comp(xv, c, comp(xv, c) - step);
            set_comp(mv, c, mbar);
        }
        store4(x + base, li, len, xv);
        if (m_out) store4(m_out + base, li, len, mv);
    }
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
    const int64_t t = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
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
            float4 zv = load4(err + (int64_t)r * err_ld + base, li, len);
#pragma unroll
            for (int c = 0; c < 4; ++c) set_comp(zv, c, error_of(comp(zv, c), s));
            store4(out + (int64_t)r * out_ld + base, li, len, zv);
        }
    }
}

inline unsigned blocks_for(int64_t waves)
{
    return (unsigned)((waves + kWavesPerBlock - 1) / kWavesPerBlock);
}

}  // namespace

hipError_t launch_warmup(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                         float *v, const float *g, int64_t g_ld, int n_grads, float lr,
                         float beta1, float beta2, float eps, int use_bc, float bc1,
                         float bc2, hipStream_t s)
{
    const float omb1 = 1.0f - beta1, omb2 = 1.0f - beta2;
    hipLaunchKernelGGL(k_warmup, dim3(blocks_for(num_tiles)), dim3(kBlock), 0, s, tb.tiles,
                       num_tiles, x, m, v, g, g_ld, n_grads, lr, beta1, omb1, beta2, omb2,
                       eps, use_bc, bc1, bc2);
    return hipGetLastError();
}

hipError_t launch_worker_pass(const DeviceTables &tb, int64_t num_tiles, const float *m,
                              const float *g, int64_t g_ld, float *err, int64_t err_ld,
                              const float *scales, int64_t scales_ld, uint64_t *bits,
                              int64_t bits_ld, double *partial, int n_local, float beta1,
                              hipStream_t s)
{
    const float omb1 = 1.0f - beta1;
    hipLaunchKernelGGL(k_worker_pass, dim3(blocks_for(num_tiles)), dim3(kBlock), 0, s,
                       tb.tiles, num_tiles, m, g, g_ld, err, err_ld, scales, scales_ld, bits,
                       bits_ld, partial, n_local, beta1, omb1);
    return hipGetLastError();
}

hipError_t launch_worker_finalize(const DeviceTables &tb, int64_t num_segments, int rows,
                                  const double *partial, int64_t part_ld, float *scales,
                                  int64_t scales_ld, hipStream_t s)
{
    hipLaunchKernelGGL(k_worker_finalize, dim3(blocks_for((int64_t)rows * num_segments)),
                       dim3(kBlock), 0, s, tb, num_segments, rows, partial, part_ld, scales,
                       scales_ld);
    return hipGetLastError();
}

hipError_t launch_server_pass(const DeviceTables &tb, int64_t tile_begin, int64_t tile_count,
                              int n, const uint64_t *wbits, int64_t bits_ld,
                              int64_t bits_word_base, const float *wscales, int64_t scales_ld,
                              int64_t scales_seg_base, float *serr, float *sscales,
                              uint64_t *sbits, double *partial, hipStream_t s)
{
    hipLaunchKernelGGL(k_server_pass, dim3(blocks_for(tile_count)), dim3(kBlock), 0, s,
                       tb.tiles, tile_begin, tile_count, n, wbits, bits_ld, bits_word_base,
                       wscales, scales_ld, scales_seg_base, serr, sscales, sbits, partial);
    return hipGetLastError();
}

hipError_t launch_server_finalize(const DeviceTables &tb, int K, int n, int jb, int je,
                                  const double *partial, float *sscales, hipStream_t s)
{
    hipLaunchKernelGGL(k_server_finalize, dim3(blocks_for((int64_t)K * (je - jb))),
                       dim3(kBlock), 0, s, tb, K, n, jb, je, partial, sscales);
    return hipGetLastError();
}

hipError_t launch_update(const DeviceTables &tb, int64_t num_tiles, const uint64_t *sbits,
                         const float *sscales, float *x, float *m_out, const float *v,
                         float lr, float eps, hipStream_t s)
{
    hipLaunchKernelGGL(k_update, dim3(blocks_for(num_tiles)), dim3(kBlock), 0, s, tb.tiles,
                       num_tiles, sbits, sscales, x, m_out, v, lr, eps);
    return hipGetLastError();
}

hipError_t launch_materialize(const DeviceTables &tb, int64_t num_tiles, int rows,
                              const float *err, int64_t err_ld, const float *scales,
                              int64_t scales_ld, float *out, int64_t out_ld, hipStream_t s)
{
    hipLaunchKernelGGL(k_materialize, dim3(blocks_for(num_tiles)), dim3(kBlock), 0, s,
                       tb.tiles, num_tiles, rows, err, err_ld, scales, scales_ld, out, out_ld);
    return hipGetLastError();
}

}  // namespace onebit
