// HBM streaming ceilings for the access mixes of the library's passes.
//
// A small library of its own (libhbmprobe.so, not part of libonebit.so) that
// times plain streaming kernels with the same load and store forms as the
// passes (128-bit buffer loads and stores, non-temporal; workgroups
// renumbered so that each XCD takes one contiguous eighth of the grid) on
// caller-allocated device buffers: the median of 7 timed launches after one
// untimed one.  The mixes:
//
//   read     one stream read (the flat read rate of the memory system);
//   copy     one stream read, another written;
//   mix      two streams read, the second rewritten in place: b = a + b, the
//            mix of the worker pass (gradient and error state read, error
//            state rewritten) and of the update and the chunk owners' pass;
//   rowsum   R rows of D floats summed per 1024-element tile in row order in
//            fp64 and written once in fp32: the warm-up's read pattern (one
//            tile per wave, W-wave workgroups, a barrier after every B rows).
//
// For read, copy and mix, K is the number of 1 KB pieces of each stream one
// wave keeps in flight, and lds the bytes of (unused) LDS each workgroup
// allocates, which caps the workgroups per CU and so the bytes in flight per
// SIMD.  k_read stores to its sink only for one impossible-looking sum (it
// keeps the loads live); the caller passes a sink of at least 4 bytes anyway.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <vector>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kXcds = 8;
constexpr int kStreamLoad = 2;        // nt
constexpr int kStreamStore = 2 | 16;  // nt, sc1
constexpr int kPieceFloats = 256;     // 1 KB: 64 lanes x 16 B

// Buffer resource over p with the maximum range; the base goes through
// readfirstlane so that the compiler knows it is wave-uniform.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t stream_rsrc(const void *p)
{
    const uint64_t a = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0,
                                             0x7FFFFFFF, 0x00020000);
}

__device__ __forceinline__ v4f load16(__amdgpu_buffer_rsrc_t r, int byte_off)
{
    return __builtin_bit_cast(v4f, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0,
                                                                         kStreamLoad));
}

__device__ __forceinline__ void store16(__amdgpu_buffer_rsrc_t r, int byte_off, v4f v)
{
    __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, v), r, byte_off, 0,
                                           kStreamStore);
}

// The chip hands workgroups to its XCDs round-robin; with a grid that is a
// multiple of 8 this renumbering gives XCD x the x-th contiguous eighth.
__device__ __forceinline__ int64_t xcd_block()
{
    const int64_t b = blockIdx.x, per = gridDim.x / kXcds;
    return (b % kXcds) * per + b / kXcds;
}

constexpr int kStreamWaves = 4;  // waves per workgroup of the stream kernels

// Wave w streams pieces [w K, w K + K); pieces is a multiple of K.
template <int K>
__global__ __launch_bounds__(kStreamWaves * kWave) void k_read(const float *__restrict__ a,
                                                               int64_t pieces,
                                                               float *__restrict__ sink)
{
    extern __shared__ float occupancy_cap[];
    (void)occupancy_cap;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t p0 = (xcd_block() * kStreamWaves + (threadIdx.x >> 6)) * K;
    if (p0 >= pieces) return;
    const __amdgpu_buffer_rsrc_t r = stream_rsrc(a + p0 * kPieceFloats);
    v4f acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < K; ++k) acc += load16(r, (k * kWave + lane) * 16);
    if (acc.x == 1234.5f && acc.y == -1.0f) sink[0] = acc.z;
}

template <int K>
__global__ __launch_bounds__(kStreamWaves * kWave) void k_copy(const float *__restrict__ a,
                                                               float *__restrict__ b,
                                                               int64_t pieces)
{
    extern __shared__ float occupancy_cap[];
    (void)occupancy_cap;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t p0 = (xcd_block() * kStreamWaves + (threadIdx.x >> 6)) * K;
    if (p0 >= pieces) return;
    const __amdgpu_buffer_rsrc_t ra = stream_rsrc(a + p0 * kPieceFloats);
    const __amdgpu_buffer_rsrc_t rb = stream_rsrc(b + p0 * kPieceFloats);
    v4f x[K];
#pragma unroll
    for (int k = 0; k < K; ++k) x[k] = load16(ra, (k * kWave + lane) * 16);
#pragma unroll
    for (int k = 0; k < K; ++k) store16(rb, (k * kWave + lane) * 16, x[k]);
}

template <int K>
__global__ __launch_bounds__(kStreamWaves * kWave) void k_mix(const float *__restrict__ a,
                                                              float *__restrict__ b,
                                                              int64_t pieces)
{
    extern __shared__ float occupancy_cap[];
    (void)occupancy_cap;
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t p0 = (xcd_block() * kStreamWaves + (threadIdx.x >> 6)) * K;
    if (p0 >= pieces) return;
    const __amdgpu_buffer_rsrc_t ra = stream_rsrc(a + p0 * kPieceFloats);
    const __amdgpu_buffer_rsrc_t rb = stream_rsrc(b + p0 * kPieceFloats);
    v4f x[K], y[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
        x[k] = load16(ra, (k * kWave + lane) * 16);
        y[k] = load16(rb, (k * kWave + lane) * 16);
    }
#pragma unroll
    for (int k = 0; k < K; ++k) store16(rb, (k * kWave + lane) * 16, x[k] + y[k]);
}

constexpr int kTile = 1024;

// One 1024-element tile per wave, W waves per workgroup walking the R rows
// together: B rows loaded, then added in row order, then a barrier.  Waves
// past the last tile load nothing but still reach every barrier.  R is a
// multiple of B; D a multiple of 1024.
template <int W, int B>
__global__ __launch_bounds__(W * kWave) void k_rowsum(const float *__restrict__ g, int64_t D,
                                                      int R, int64_t tiles,
                                                      float *__restrict__ out)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int64_t t = xcd_block() * W + (threadIdx.x >> 6);
    const bool active = t < tiles;
    const int64_t base = active ? t * kTile : 0;
    double s[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) s[k] = 0.0;
    for (int r = 0; r < R; r += B) {
        if (active) {
            v4f v[B][4];
#pragma unroll
            for (int q = 0; q < B; ++q) {
                const __amdgpu_buffer_rsrc_t rr = stream_rsrc(g + (int64_t)(r + q) * D + base);
#pragma unroll
                for (int c = 0; c < 4; ++c) v[q][c] = load16(rr, (c * kWave + lane) * 16);
            }
#pragma unroll
            for (int q = 0; q < B; ++q)
#pragma unroll
                for (int c = 0; c < 4; ++c)
#pragma unroll
                    for (int e = 0; e < 4; ++e) s[4 * c + e] += (double)v[q][c][e];
        }
        __builtin_amdgcn_s_barrier();
    }
    if (!active) return;
    const __amdgpu_buffer_rsrc_t ro = stream_rsrc(out + base);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        const v4f o = {(float)s[4 * c], (float)s[4 * c + 1], (float)s[4 * c + 2],
                       (float)s[4 * c + 3]};
        store16(ro, (c * kWave + lane) * 16, o);
    }
}

int64_t grid_for(int64_t waves, int waves_per_block)
{
    const int64_t blocks = (waves + waves_per_block - 1) / waves_per_block;
    return (blocks + kXcds - 1) / kXcds * kXcds;
}

// Median of 7 timed launches (after one untimed) on stream s, in *ms.
template <class F>
hipError_t median_ms(F launch, hipStream_t s, float *ms)
{
    hipEvent_t e0 = nullptr, e1 = nullptr;
    hipError_t err = hipEventCreate(&e0);
    if (err == hipSuccess) err = hipEventCreate(&e1);
    std::vector<float> ts;
    if (err == hipSuccess) {
        launch();
        err = hipGetLastError();
    }
    if (err == hipSuccess) err = hipStreamSynchronize(s);
    for (int r = 0; r < 7 && err == hipSuccess; ++r) {
        err = hipEventRecord(e0, s);
        if (err == hipSuccess) {
            launch();
            err = hipGetLastError();
        }
        if (err == hipSuccess) err = hipEventRecord(e1, s);
        if (err == hipSuccess) err = hipEventSynchronize(e1);
        float t = 0.f;
        if (err == hipSuccess) err = hipEventElapsedTime(&t, e0, e1);
        ts.push_back(t);
    }
    if (e0) (void)hipEventDestroy(e0);
    if (e1) (void)hipEventDestroy(e1);
    if (err != hipSuccess) return err;
    std::sort(ts.begin(), ts.end());
    *ms = ts[ts.size() / 2];
    return hipSuccess;
}

template <int K>
hipError_t stream_case(int kind, const float *a, float *b, float *sink, int64_t pieces, int lds,
                       hipStream_t s, float *ms)
{
    const dim3 grid((unsigned)grid_for(pieces / K, kStreamWaves)), block(kStreamWaves * kWave);
    switch (kind) {
    case 0:
        return median_ms([&] { hipLaunchKernelGGL(k_read<K>, grid, block, lds, s, a, pieces,
                                                  sink); }, s, ms);
    case 1:
        return median_ms([&] { hipLaunchKernelGGL(k_copy<K>, grid, block, lds, s, a, b,
                                                  pieces); }, s, ms);
    default:
        return median_ms([&] { hipLaunchKernelGGL(k_mix<K>, grid, block, lds, s, a, b,
                                                  pieces); }, s, ms);
    }
}

}  // namespace

extern "C" {

// One streaming case over device buffers a and b of `floats` floats each
// (a multiple of 1024; a is only read, b is written by copy and mix) and a
// 4-byte sink, on stream s.  kind: 0 read a, 1 copy a to b, 2 mix b = a + b.
// k: 1 KB pieces per stream per wave, 1, 2 or 4.  lds: bytes of LDS per
// 4-wave workgroup, 0 to 65536.  Writes the median time in ms to *ms.
// Returns 0, -1 for an invalid argument, or the HIP error code.
int hbm_probe_stream(int kind, int k, int lds, const float *a, float *b, float *sink,
                     int64_t floats, hipStream_t s, float *ms)
{
    if (kind < 0 || kind > 2 || !a || !sink || !ms || (kind > 0 && !b) || floats <= 0 ||
        floats % 1024 || lds < 0 || lds > 65536)
        return -1;
    const int64_t pieces = floats / kPieceFloats;
    if (grid_for(pieces, kStreamWaves) > 0x7FFFFFF0) return -1;  // k = 1's grid
    hipError_t e;
    switch (k) {
    case 1: e = stream_case<1>(kind, a, b, sink, pieces, lds, s, ms); break;
    case 2: e = stream_case<2>(kind, a, b, sink, pieces, lds, s, ms); break;
    case 4: e = stream_case<4>(kind, a, b, sink, pieces, lds, s, ms); break;
    default: return -1;
    }
    return (int)e;
}

// The warm-up's read pattern: R rows of D floats at g (row r at g + r D; D a
// multiple of 1024) summed per 1024-element tile in row order in fp64 and
// written once to out (D floats), one tile per wave, w waves per workgroup
// (4, 8 or 16) and a barrier after every b rows (1 or 2; R a multiple of
// b), on stream s.  Writes the median time in ms to *ms.  Returns 0, -1 for
// an invalid argument, or the HIP error code.
int hbm_probe_rowsum(int w, int b, const float *g, int64_t D, int R, float *out, hipStream_t s,
                     float *ms)
{
    const bool shape = (w == 16 && (b == 1 || b == 2)) || ((w == 8 || w == 4) && b == 1);
    if (!shape || !g || !out || !ms || D <= 0 || D % kTile || R <= 0 || R % b) return -1;
    const int64_t tiles = D / kTile;
    if (grid_for(tiles, w) > 0x7FFFFFF0) return -1;
#define ROWSUM(W, B)                                                                           \
    median_ms([&] { hipLaunchKernelGGL((k_rowsum<W, B>), dim3((unsigned)grid_for(tiles, W)),     \
                                       dim3(W * kWave), 0, s, g, D, R, tiles, out); }, s, ms)
    hipError_t e;
    if (w == 16 && b == 1) e = ROWSUM(16, 1);
    else if (w == 16 && b == 2) e = ROWSUM(16, 2);
    else if (w == 8 && b == 1) e = ROWSUM(8, 1);
    else if (w == 4 && b == 1) e = ROWSUM(4, 1);
    else return -1;
#undef ROWSUM
    return (int)e;
}

}  // extern "C"
