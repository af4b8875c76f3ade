// Internal interface between the C-ABI layer and the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "onebit_grid.h"

namespace onebit {

// A unit of work: up to kTileElems consecutive elements of one segment,
// starting on a 64-element (one sign word) boundary.  One wavefront owns one
// tile (one tile of one worker row, in the packed worker pass); the launch
// shapes are in onebit_grid.h.
struct Tile {
    int64_t start;  // first flat element (multiple of 64)
    int32_t len;    // elements in the tile, 1..kTileElems
    int32_t seg;    // segment q = k*n + j
};

constexpr int kSubBlocks = 4;                       // float4 loads per lane per array
constexpr int kTileElems = kWave * 4 * kSubBlocks;  // 1024 elements = 16 sign words
constexpr int kTileWords = kTileElems / 64;
constexpr int kServerRowBatch = 32;                 // worker rows staged in LDS at a time

// Device-side layout tables owned by a plan.
struct DeviceTables {
    const Tile *tiles;             // [T], in address (segment) order
    const int32_t *chunk_tiles;    // [T], tile ids in chunk-major order
    const int64_t *seg_tile_begin; // [S]
    const int64_t *seg_tile_end;   // [S]
    const int64_t *seg_len;        // [S]
    const int32_t *server_blocks;  // chunk owners' shared-table workgroups, chunk-major
                                   // (entries of onebit_grid.h's server_block_entry)
};

// Gradient element types (the values of the ONEBIT_GRAD_* constants).
constexpr int kGradF32 = 0;
constexpr int kGradBF16 = 1;
constexpr int kGradF16 = 2;

hipError_t launch_warmup(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                         float *v, const void *g, int grad_dtype, int64_t g_ld, int n_grads,
                         float lr, float beta1, float beta2, float eps, int use_bc, float bc1,
                         float bc2, hipStream_t s);

// m != NULL: fp32 momentum; m == NULL: momentum decoded from (m_bits, m_scales).
// group: workers handled by one workgroup per tile (1..n_local); the grid
// runs over groups first, then tiles.
hipError_t launch_worker_pass(const DeviceTables &tb, int64_t num_tiles, const float *m,
                              const uint64_t *m_bits, const float *m_scales, const void *g,
                              int grad_dtype, int64_t g_ld, float *err, int64_t err_ld,
                              const float *scales, int64_t scales_ld, uint64_t *bits,
                              int64_t bits_ld, double *partial, int n_local, int group,
                              float beta1, hipStream_t s);

hipError_t launch_adam_message(const DeviceTables &tb, int64_t num_tiles, const uint64_t *bits,
                               const float *scales, float *x, float *m, float *v, float lr,
                               float beta1, float beta2, float eps, int use_bc, float bc1,
                               float bc2, hipStream_t s);

hipError_t launch_uncompressed(const DeviceTables &tb, int64_t num_tiles, float *x, float *m,
                               const float *v, const void *g, int grad_dtype, int64_t g_ld,
                               int n, float lr, float beta1, float eps, hipStream_t s);

// out[0] = sum of |v| over the real elements (fp64, fixed order); partial: [T].
hipError_t launch_l1_norm(const DeviceTables &tb, int64_t num_tiles, const float *v,
                          double *partial, double *out, hipStream_t s);

hipError_t launch_decode(const DeviceTables &tb, int64_t num_tiles, const uint64_t *bits,
                         const float *scales, float *out, hipStream_t s);

// Segment scales from per-tile partial sums.  Worker form (server_form = 0):
// num_pairs = rows * num_segments, scale[i*scales_ld + q] from
// partial[i*part_ld + tiles of q].  Server form: num_pairs = K * (je - jb),
// segments k*n + j for j in [jb, je), one row.  max_seg_tiles picks a wave
// or a block per pair.
hipError_t launch_finalize(const DeviceTables &tb, int64_t max_seg_tiles, int64_t num_pairs,
                           int64_t num_segments, int server_form, int n, int jb, int je,
                           const double *partial, int64_t part_ld, float *scales,
                           int64_t scales_ld, hipStream_t s);

// Bytes of the chunk owners' lookup tables for `segments` owned segments.
size_t server_table_bytes(int n, int64_t segments);

// The chunk owners' pass over tiles [tile_begin, tile_begin + tile_count) of
// the chunk-major tile list, for chunks [cb, cb + nown) of num_tensors
// tensors.  tables != NULL (at least server_table_bytes(n, num_tensors *
// nown) bytes, 256-byte aligned) and flags (num_tensors * nown int32): the
// owned segments' tables are built there first and copied by the pass, which
// for n <= 32 runs the num_blocks shared-table workgroups of server_blocks
// (the call's range of DeviceTables::server_blocks); tables == NULL: the
// pass builds them per tile.
hipError_t launch_server_pass(const DeviceTables &tb, int64_t tile_begin, int64_t tile_count,
                              int n, const uint64_t *wbits, int64_t bits_ld,
                              int64_t bits_word_base, const float *wscales, int64_t scales_ld,
                              int64_t scales_seg_base, float *serr, float *sscales,
                              uint64_t *sbits, double *partial, int num_tensors, int cb,
                              int nown, double *tables, int32_t *flags,
                              const int32_t *server_blocks, int64_t num_blocks, hipStream_t s);

hipError_t launch_update(const DeviceTables &tb, int64_t num_tiles, const uint64_t *sbits,
                         const float *sscales, float *x, float *m_out, const float *v,
                         float lr, float eps, hipStream_t s);

// The library's own scratch memory, for callers that cannot allocate: a
// static device array of kScratchBytes on every device the library runs on,
// held until the process ends.  scratch_address() returns its device address
// on `device` (looked up once per device, with that device made current for
// the lookup and restored afterwards), or an error for a device index at or
// above kMaxScratchDevices or a failed lookup.  Every call on one device
// shares the array.
constexpr size_t kScratchBytes = (size_t)96 << 20;
constexpr int kMaxScratchDevices = 64;
hipError_t scratch_address(int device, void **ptr);

hipError_t launch_materialize(const DeviceTables &tb, int64_t num_tiles, int rows,
                              const float *err, int64_t err_ld, const float *scales,
                              int64_t scales_ld, float *out, int64_t out_ld, hipStream_t s);

}  // namespace onebit
