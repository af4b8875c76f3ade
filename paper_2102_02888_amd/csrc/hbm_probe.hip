// HBM streaming ceilings for the access mixes of the library's passes.
//
// A standalone program (not part of libonebit.so) that times plain streaming
// kernels with the same load and store forms as the passes (128-bit buffer
// loads and stores, non-temporal; workgroups renumbered so that each XCD takes
// one contiguous eighth of the grid) and prints one line per case: the median
// of 7 timed launches and the bytes moved per second.  The mixes:
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
// SIMD.  Every buffer is zero-filled, so the sums are 0 and the sink store in
// k_read never happens (it keeps the loads live).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

namespace {

typedef float v4f __attribute__((ext_vector_type(4)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;
constexpr int kXcds = 8;
constexpr int kStreamLoad = 2;        // nt
constexpr int kStreamStore = 2 | 16;  // nt, sc1
constexpr int kPieceFloats = 256;     // 1 KB: 64 lanes x 16 B
constexpr double kPeakGBs = 8000.0;

#define CHECK(x)                                                                          \
    do {                                                                                  \
        hipError_t e_ = (x);                                                              \
        if (e_ != hipSuccess) {                                                           \
            fprintf(stderr, "hbm_probe: %s: %s\n", #x, hipGetErrorString(e_));            \
            exit(1);                                                                      \
        }                                                                                 \
    } while (0)

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

template <class F>
float median_ms(F launch)
{
    hipEvent_t e0, e1;
    CHECK(hipEventCreate(&e0));
    CHECK(hipEventCreate(&e1));
    launch();
    CHECK(hipGetLastError());
    CHECK(hipDeviceSynchronize());
    std::vector<float> ts;
    for (int r = 0; r < 7; ++r) {
        CHECK(hipEventRecord(e0, 0));
        launch();
        CHECK(hipEventRecord(e1, 0));
        CHECK(hipEventSynchronize(e1));
        float ms = 0.f;
        CHECK(hipEventElapsedTime(&ms, e0, e1));
        ts.push_back(ms);
    }
    CHECK(hipEventDestroy(e0));
    CHECK(hipEventDestroy(e1));
    std::sort(ts.begin(), ts.end());
    return ts[ts.size() / 2];
}

void report(const char *name, int K, int lds, int waves_per_cu, double bytes, float ms)
{
    const double gbs = bytes / ms / 1e6;
    printf("%-4s K=%d lds=%5d (<= %2d waves/CU, <= %2d KB/SIMD of loads in flight)  %8.3f ms  "
           "%6.0f GB/s  %.3f\n",
           name, K, lds, waves_per_cu, waves_per_cu / 4 * K * (name[0] == 'm' ? 2 : 1), ms, gbs,
           gbs / kPeakGBs);
    fflush(stdout);
}

// Upper bound on the waves per CU of a 4-wave workgroup that allocates lds
// bytes of LDS: the 160 KB of LDS per CU and 8 waves per SIMD (32 per CU).
int stream_waves_per_cu(int lds)
{
    const int by_lds = lds > 0 ? (160 * 1024) / lds : 8;
    return std::min(8, by_lds) * kStreamWaves;
}

template <int K>
void stream_cases(float *a, float *b, float *sink, int64_t floats, int lds)
{
    const int64_t pieces = floats / kPieceFloats;  // a multiple of every K used
    const int64_t grid = grid_for(pieces / K, kStreamWaves);
    const dim3 block(kStreamWaves * kWave);
    const double stream = (double)floats * 4;
    const int wpc = stream_waves_per_cu(lds);
    report("read", K, lds, wpc, stream,
           median_ms([&] { hipLaunchKernelGGL(k_read<K>, dim3(grid), block, lds, 0, a, pieces,
                                              sink); }));
    report("copy", K, lds, wpc, 2 * stream,
           median_ms([&] { hipLaunchKernelGGL(k_copy<K>, dim3(grid), block, lds, 0, a, b,
                                              pieces); }));
    report("mix", K, lds, wpc, 3 * stream,
           median_ms([&] { hipLaunchKernelGGL(k_mix<K>, dim3(grid), block, lds, 0, a, b,
                                              pieces); }));
}

template <int W, int B>
void rowsum_case(const float *g, int64_t D, int R, float *out)
{
    const int64_t tiles = D / kTile;
    const int64_t grid = grid_for(tiles, W);
    const double bytes = (double)R * D * 4 + (double)D * 4;
    const float ms = median_ms([&] {
        hipLaunchKernelGGL((k_rowsum<W, B>), dim3(grid), dim3(W * kWave), 0, 0, g, D, R, tiles,
                           out);
    });
    printf("rowsum R=%d W=%2d B=%d  %8.3f ms  %6.0f GB/s  %.3f\n", R, W, B, ms,
           bytes / ms / 1e6, bytes / ms / 1e6 / kPeakGBs);
    fflush(stdout);
}

}  // namespace

int main()
{
    hipDeviceProp_t prop;
    CHECK(hipGetDeviceProperties(&prop, 0));
    printf("device %s (%s), %d CUs\n", prop.name, prop.gcnArchName, prop.multiProcessorCount);

    // Streams of 4 GiB each: far beyond the 256 MB last-level cache.
    const int64_t floats = (int64_t)1 << 30;
    float *a = nullptr, *b = nullptr, *sink = nullptr;
    CHECK(hipMalloc(&a, floats * 4));
    CHECK(hipMalloc(&b, floats * 4));
    CHECK(hipMalloc(&sink, 4));
    CHECK(hipMemset(a, 0, floats * 4));
    CHECK(hipMemset(b, 0, floats * 4));
    printf("read / copy / mix over %lld MiB streams\n", (long long)(floats * 4 >> 20));
    fflush(stdout);
    for (int lds : {0, 40960, 65536}) {
        stream_cases<1>(a, b, sink, floats, lds);
        stream_cases<2>(a, b, sink, floats, lds);
        stream_cases<4>(a, b, sink, floats, lds);
    }
    CHECK(hipFree(a));
    CHECK(hipFree(b));
    CHECK(hipFree(sink));

    // The warm-up's pattern on the BERT-Large shape: 32 rows of 334,088,192 floats.
    const int R = 32;
    const int64_t D = 334088192;  // 326,258 tiles of 1024
    float *g = nullptr, *out = nullptr;
    CHECK(hipMalloc(&g, (size_t)R * D * 4));
    CHECK(hipMalloc(&out, (size_t)D * 4));
    CHECK(hipMemset(g, 0, (size_t)R * D * 4));
    CHECK(hipMemset(out, 0, (size_t)D * 4));
    printf("rowsum over %d rows of %lld floats (%.1f GB read)\n", R, (long long)D,
           (double)R * D * 4 / 1e9);
    fflush(stdout);
    rowsum_case<16, 1>(g, D, R, out);
    rowsum_case<16, 2>(g, D, R, out);
    rowsum_case<8, 1>(g, D, R, out);
    rowsum_case<4, 1>(g, D, R, out);
    {
        // the same bytes read flat
        const int64_t fl = (int64_t)R * D, pieces = fl / kPieceFloats;
        const float ms = median_ms([&] {
            hipLaunchKernelGGL(k_read<4>, dim3(grid_for(pieces / 4, kStreamWaves)),
                               dim3(kStreamWaves * kWave), 0, 0, g, pieces, out);
        });
        printf("flat read of the %d rows  %8.3f ms  %6.0f GB/s  %.3f\n", R, ms,
               (double)fl * 4 / ms / 1e6, (double)fl * 4 / ms / 1e6 / kPeakGBs);
    }
    CHECK(hipFree(g));
    CHECK(hipFree(out));
    printf("done\n");
    return 0;
}
