// C ABI of the 1-bit Adam hot path: plans (layout and tile tables), argument
// validation, and stream-ordered kernel launches.  See include/onebit.h for
// the contract of every entry point.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <memory>
#include <new>
#include <vector>

#include "../../include/onebit.h"
#include "onebit_internal.h"

static_assert(onebit::kScratchBytes == ONEBIT_NOALLOC_SCRATCH_BYTES,
              "the scratch array and the header's limit must agree");

using onebit::DeviceTables;
using onebit::kTileElems;
using onebit::Tile;

struct onebit_plan_s {
    int device = 0;
    int32_t K = 0, n = 0;
    int64_t d = 0, D = 0, W = 0, S = 0, T = 0;
    int64_t max_seg_tiles = 0;                          // most tiles in one segment
    std::vector<int64_t> tensor_off, chunk_len, seg_begin, seg_end;
    std::vector<int64_t> seg_tile_begin, seg_tile_end;  // [S]
    std::vector<int64_t> chunk_tile_begin;              // [n+1], into chunk_tiles
    std::vector<int64_t> chunk_word_lo, chunk_word_hi;  // [n], words touched by chunk j
    std::vector<int64_t> chunk_block_begin;  // [n+1], into the shared-table workgroups
    void *dev_mem = nullptr;                            // one allocation for all tables
    DeviceTables tb{};
    size_t table_bytes = 0;  // chunk owners' lookup tables in the workspace (0: none)
    int32_t server_tables = ONEBIT_SERVER_TABLES_AUTO;  // onebit_plan_set_server_tables
    size_t workspace_bytes = 0;
};

namespace {

thread_local char g_last_error[512] = "";

int fail(int status, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return status;
}

int hip_fail(hipError_t e, const char *where)
{
    return fail(ONEBIT_EHIP, "%s: %s", where, hipGetErrorString(e));
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

size_t round_up(size_t a, size_t m) { return (a + m - 1) / m * m; }

// Workspace: per-tile fp64 partial sums, n rows for the workers then one row
// for the chunk owners; then, when the plan keeps them, the chunk owners'
// lookup tables of every segment and one flag per segment.
size_t worker_partial_offset(const onebit_plan_s *) { return 0; }
size_t server_partial_offset(const onebit_plan_s *p)
{
    return round_up((size_t)p->n * (size_t)p->T * sizeof(double), 256);
}
size_t server_table_offset(const onebit_plan_s *p)
{
    return server_partial_offset(p) + round_up((size_t)p->T * sizeof(double) + 1, 256);
}
size_t server_flag_offset(const onebit_plan_s *p)
{
    return server_table_offset(p) + p->table_bytes;
}

// The tables of a plan's segments are kept in the workspace (built once per
// chunk owners' call instead of once per tile) when all of them fit in this
// many bytes: 256 KB for a BERT-Large-sized buffer with n = 32, 16 MB for
// one tensor with n = 256.
constexpr size_t kServerTableBudget = (size_t)32 << 20;
// ... and a call uses them when its segments average at least this many tiles
// and its tiles times its groups of 8 workers (the table builds it saves) reach
// kServerTableMinWork: below that the table kernel's own launch costs more
// (1-3 us on calls of 1,024 to 16,384 tiles with n = 4 to 32).
constexpr int64_t kServerTableMinTiles = 4;
constexpr int64_t kServerTableMinWork = 32768;

int check_plan(const onebit_plan_s *p)
{
    if (!p) return fail(ONEBIT_EINVAL, "plan is NULL");
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev != p->device)
        return fail(ONEBIT_EINVAL, "plan was created on device %d, current device is %d",
                    p->device, dev);
    return ONEBIT_OK;
}

// Element buffers ([D] floats, rows of D, [W] words, rows of W): NULL is
// accepted only for a plan with no elements (D = 0, nothing is touched).
int check_f32(const onebit_plan_s *p, const void *ptr, const char *name)
{
    if (!ptr) return p->D == 0 ? ONEBIT_OK : fail(ONEBIT_EINVAL, "%s is NULL", name);
    if (!aligned(ptr, 16)) return fail(ONEBIT_EALIGN, "%s is not 16-byte aligned", name);
    return ONEBIT_OK;
}

int check_u64(const onebit_plan_s *p, const void *ptr, const char *name)
{
    if (!ptr) return p->D == 0 ? ONEBIT_OK : fail(ONEBIT_EINVAL, "%s is NULL", name);
    if (!aligned(ptr, 8)) return fail(ONEBIT_EALIGN, "%s is not 8-byte aligned", name);
    return ONEBIT_OK;
}

int check_grads(const onebit_plan_s *p, const void *g, int32_t dtype)
{
    if (dtype != ONEBIT_GRAD_F32 && dtype != ONEBIT_GRAD_BF16 && dtype != ONEBIT_GRAD_F16)
        return fail(ONEBIT_EINVAL, "grad_dtype %d is not one of ONEBIT_GRAD_*", dtype);
    if (!g) return p->D == 0 ? ONEBIT_OK : fail(ONEBIT_EINVAL, "grads is NULL");
    const size_t need = dtype == ONEBIT_GRAD_F32 ? 16 : 8;
    if (!aligned(g, need)) return fail(ONEBIT_EALIGN, "grads is not %zu-byte aligned", need);
    return ONEBIT_OK;
}

int check_ld(int64_t ld, int64_t need, bool mult4, const char *name)
{
    if (ld < need) return fail(ONEBIT_EINVAL, "%s = %lld is below %lld", name, (long long)ld,
                               (long long)need);
    if (mult4 && need > 0 && ld % 4 != 0) return fail(ONEBIT_EALIGN, "%s = %lld is not a multiple of 4",
                                          name, (long long)ld);
    return ONEBIT_OK;
}

#define TRY(expr)                         \
    do {                                  \
        int _st = (expr);                 \
        if (_st != ONEBIT_OK) return _st; \
    } while (0)

#define TRY_HIP(expr, where)                       \
    do {                                           \
        hipError_t _e = (expr);                    \
        if (_e != hipSuccess) return hip_fail(_e, where); \
    } while (0)

int64_t chunk_len(int64_t d, int32_t n)
{
    if (d <= 0) return 0;
    const int64_t per = (d + (int64_t)n * 64 - 1) / ((int64_t)n * 64);
    return per * 64;
}

// Builds the layout and tile tables of a plan (arguments already checked).
// Host allocations may throw std::bad_alloc; the caller turns that into
// ONEBIT_ENOMEM.
int plan_create_impl(const int64_t *tensor_numel, int32_t num_tensors, int32_t n_workers,
                     onebit_plan *out)
{
    std::unique_ptr<onebit_plan_s> owner(new onebit_plan_s);
    onebit_plan_s *p = owner.get();
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    const int32_t K = num_tensors, n = n_workers;
    p->K = K;
    p->n = n;
    p->S = (int64_t)K * n;
    p->tensor_off.resize(K);
    p->chunk_len.resize(K);
    p->seg_begin.resize(p->S);
    p->seg_end.resize(p->S);
    int64_t off = 0, d = 0;
    for (int32_t k = 0; k < K; ++k) {
        const int64_t dk = tensor_numel[k];
        const int64_t c = chunk_len(dk, n);
        p->tensor_off[k] = off;
        p->chunk_len[k] = c;
        for (int32_t j = 0; j < n; ++j) {
            const int64_t b = std::min<int64_t>((int64_t)j * c, dk);
            const int64_t en = std::min<int64_t>((int64_t)(j + 1) * c, dk);
            p->seg_begin[(int64_t)k * n + j] = off + b;
            p->seg_end[(int64_t)k * n + j] = off + en;
        }
        off += (dk + 63) / 64 * 64;
        d += dk;
        if (off >= ((int64_t)1 << 40))
            return fail(ONEBIT_EINVAL, "padded length exceeds 2^40 elements");
    }
    p->d = d;
    p->D = off;
    p->W = off / 64;

    // Tiles are cut at multiples of kTileElems of the flat index (a segment
    // that starts or ends between two such points gets a short tile there),
    // so that every full tile's sign words are 128-byte aligned.
    auto tiles_of = [](int64_t b, int64_t e) -> int64_t {
        if (e <= b) return 0;
        return (e - 1) / kTileElems - b / kTileElems + 1;
    };
    // Below 2^25 tiles every launch stays below 2^32 work-items (the grid
    // header's launch shapes and pieces).
    int64_t tile_count = 0;
    for (int64_t q = 0; q < p->S; ++q) tile_count += tiles_of(p->seg_begin[q], p->seg_end[q]);
    if (tile_count >= ((int64_t)1 << 25))
        return fail(ONEBIT_EINVAL, "%lld tiles: plans are limited to 2^25 tiles of %d elements",
                    (long long)tile_count, kTileElems);

    // Tiles in address order (segment by segment), so that passes over all
    // of d stream through memory; the tiles of chunk owner j are listed
    // separately, chunk-major, as one contiguous range of chunk_tiles.
    std::vector<Tile> tiles;
    tiles.reserve(tile_count);
    p->seg_tile_begin.assign(p->S, 0);
    p->seg_tile_end.assign(p->S, 0);
    p->chunk_tile_begin.assign(n + 1, 0);
    p->chunk_word_lo.assign(n, INT64_MAX);
    p->chunk_word_hi.assign(n, -1);
    std::vector<int64_t> seg_len(p->S);
    for (int64_t q = 0; q < p->S; ++q) {
        const int64_t b = p->seg_begin[q], en = p->seg_end[q];
        seg_len[q] = en - b;
        p->seg_tile_begin[q] = (int64_t)tiles.size();
        for (int64_t s = b; s < en;) {
            const int64_t next = std::min<int64_t>(en, (s / kTileElems + 1) * kTileElems);
            Tile t;
            t.start = s;
            t.len = (int32_t)(next - s);
            t.seg = (int32_t)q;
            tiles.push_back(t);
            s = next;
        }
        p->seg_tile_end[q] = (int64_t)tiles.size();
        p->max_seg_tiles = std::max(p->max_seg_tiles, p->seg_tile_end[q] - p->seg_tile_begin[q]);
    }
    std::vector<int32_t> chunk_tiles;
    chunk_tiles.reserve(tiles.size());
    // the chunk owners' shared-table workgroups: up to kWavesPerBlock
    // consecutive tiles of one segment each, in the same chunk-major order
    std::vector<int32_t> server_blocks;
    p->chunk_block_begin.assign(n + 1, 0);
    for (int32_t j = 0; j < n; ++j) {
        p->chunk_tile_begin[j] = (int64_t)chunk_tiles.size();
        p->chunk_block_begin[j] = (int64_t)server_blocks.size();
        for (int32_t k = 0; k < K; ++k) {
            const int64_t q = (int64_t)k * n + j;
            const int64_t pos = (int64_t)chunk_tiles.size();
            const int64_t cnt = p->seg_tile_end[q] - p->seg_tile_begin[q];
            for (int64_t i = 0; i < onebit::server_blocks_of(cnt); ++i)
                server_blocks.push_back(onebit::server_block_entry(pos, cnt, i));
            for (int64_t t = p->seg_tile_begin[q]; t < p->seg_tile_end[q]; ++t)
                chunk_tiles.push_back((int32_t)t);
            const int64_t b = p->seg_begin[q], en = p->seg_end[q];
            if (en > b) {
                p->chunk_word_lo[j] = std::min(p->chunk_word_lo[j], b / 64);
                p->chunk_word_hi[j] = std::max(p->chunk_word_hi[j], (en - 1) / 64);
            }
        }
    }
    p->chunk_tile_begin[n] = (int64_t)chunk_tiles.size();
    p->chunk_block_begin[n] = (int64_t)server_blocks.size();
    p->T = (int64_t)tiles.size();

    const size_t tiles_bytes = round_up(tiles.size() * sizeof(Tile) + 1, 256);
    const size_t order_bytes = round_up(chunk_tiles.size() * sizeof(int32_t) + 1, 256);
    const size_t seg_bytes = round_up((size_t)p->S * sizeof(int64_t), 256);
    const size_t block_bytes = round_up(server_blocks.size() * sizeof(int32_t) + 1, 256);
    const size_t seg0 = tiles_bytes + order_bytes;
    const size_t blocks0 = seg0 + 3 * seg_bytes;
    const size_t total = blocks0 + block_bytes;
    std::vector<char> host(total, 0);
    if (!tiles.empty()) {
        std::memcpy(host.data(), tiles.data(), tiles.size() * sizeof(Tile));
        std::memcpy(host.data() + tiles_bytes, chunk_tiles.data(),
                    chunk_tiles.size() * sizeof(int32_t));
        std::memcpy(host.data() + blocks0, server_blocks.data(),
                    server_blocks.size() * sizeof(int32_t));
    }
    std::memcpy(host.data() + seg0, p->seg_tile_begin.data(), p->S * sizeof(int64_t));
    std::memcpy(host.data() + seg0 + seg_bytes, p->seg_tile_end.data(), p->S * sizeof(int64_t));
    std::memcpy(host.data() + seg0 + 2 * seg_bytes, seg_len.data(), p->S * sizeof(int64_t));
    // Every host allocation is done; from here on nothing throws.
    e = hipMalloc(&p->dev_mem, total);
    if (e != hipSuccess)
        return fail(ONEBIT_ENOMEM, "hipMalloc of %zu bytes of plan tables: %s", total,
                    hipGetErrorString(e));
    e = hipMemcpy(p->dev_mem, host.data(), total, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipFree(p->dev_mem);
        return hip_fail(e, "hipMemcpy of plan tables");
    }
    char *base = (char *)p->dev_mem;
    Tile *d_tiles = (Tile *)base;
    int32_t *d_order = (int32_t *)(base + tiles_bytes);
    int64_t *d_stb = (int64_t *)(base + seg0);
    int64_t *d_ste = (int64_t *)(base + seg0 + seg_bytes);
    int64_t *d_sl = (int64_t *)(base + seg0 + 2 * seg_bytes);
    p->tb.tiles = d_tiles;
    p->tb.chunk_tiles = d_order;
    p->tb.seg_tile_begin = d_stb;
    p->tb.seg_tile_end = d_ste;
    p->tb.seg_len = d_sl;
    p->tb.server_blocks = (const int32_t *)(base + blocks0);
    const size_t seg_tables = onebit::server_table_bytes(p->n, 1);
    p->table_bytes = (size_t)p->S <= kServerTableBudget / seg_tables
                         ? onebit::server_table_bytes(p->n, p->S)
                         : 0;
    p->workspace_bytes = server_flag_offset(p) +
                         (p->table_bytes ? round_up((size_t)p->S * sizeof(int32_t), 256) : 0);
    *out = owner.release();
    return ONEBIT_OK;
}

// The three calls of a compression step, each split into its argument
// checks and its launches, so that the fused step checks everything before
// its first launch.
int check_worker(const onebit_plan_s *p, const float *m, const uint64_t *m_bits,
                 const float *m_scales, const void *grads, int32_t grad_dtype, int64_t grad_ld,
                 int32_t n_local, const float *worker_err, int64_t err_ld,
                 const uint64_t *worker_bits, int64_t bits_ld, const float *worker_scales,
                 int64_t scales_ld, const void *workspace)
{
    if (m) {
        TRY(check_f32(p, m, "m"));
    } else {
        TRY(check_u64(p, m_bits, "m_bits (m is NULL)"));
        if (!m_scales) return fail(ONEBIT_EINVAL, "m_scales is NULL (m is NULL)");
        if (!aligned(m_scales, 4)) return fail(ONEBIT_EALIGN, "m_scales misaligned");
    }
    TRY(check_grads(p, grads, grad_dtype));
    TRY(check_f32(p, worker_err, "worker_err"));
    TRY(check_u64(p, worker_bits, "worker_bits"));
    if (!worker_scales) return fail(ONEBIT_EINVAL, "worker_scales is NULL");
    if (!aligned(worker_scales, 4)) return fail(ONEBIT_EALIGN, "worker_scales misaligned");
    if (!workspace) return fail(ONEBIT_EINVAL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(ONEBIT_EALIGN, "workspace is not 256-byte aligned");
    if (n_local < 1 || n_local > p->n)
        return fail(ONEBIT_EINVAL, "n_local = %d outside [1, %d]", n_local, p->n);
    TRY(check_ld(grad_ld, p->D, n_local > 1, "grad_ld"));
    TRY(check_ld(err_ld, p->D, n_local > 1, "err_ld"));
    TRY(check_ld(bits_ld, p->W, false, "bits_ld"));
    TRY(check_ld(scales_ld, p->S, false, "scales_ld"));
    return ONEBIT_OK;
}

int run_worker(const onebit_plan_s *p, const float *m, const uint64_t *m_bits,
               const float *m_scales, const void *grads, int32_t grad_dtype, int64_t grad_ld,
               int32_t n_local, float *worker_err, int64_t err_ld, uint64_t *worker_bits,
               int64_t bits_ld, float *worker_scales, int64_t scales_ld, float beta1,
               void *workspace, hipStream_t s)
{
    double *part = (double *)((char *)workspace + worker_partial_offset(p));
    // Packed momentum costs 1/8 byte per element to re-derive, so each
    // workgroup takes one (worker, tile) item and all workgroups in flight
    // stream the same two rows (gradient and error state of one worker); an
    // fp32 momentum is read once per tile for all local workers instead.
    const int group = m ? n_local : 1;
    if (p->T > 0)
        TRY_HIP(onebit::launch_worker_pass(p->tb, p->T, m, m_bits, m_scales, grads, grad_dtype,
                                           grad_ld, worker_err, err_ld, worker_scales, scales_ld,
                                           worker_bits, bits_ld, part, n_local, group, beta1, s),
                "worker kernel launch");
    TRY_HIP(onebit::launch_finalize(p->tb, p->max_seg_tiles, (int64_t)n_local * p->S, p->S, 0,
                                    p->n, 0, 0, part, p->T, worker_scales, scales_ld, s),
            "worker scale kernel launch");
    return ONEBIT_OK;
}

int check_server(const onebit_plan_s *p, int32_t server_begin, int32_t server_end,
                 const uint64_t *worker_bits, int64_t bits_ld, int64_t bits_word_base,
                 const float *worker_scales, int64_t scales_ld, int64_t scales_seg_base,
                 const float *server_err, const uint64_t *server_bits,
                 const float *server_scales, const void *workspace)
{
    TRY(check_u64(p, worker_bits, "worker_bits"));
    if (!worker_scales) return fail(ONEBIT_EINVAL, "worker_scales is NULL");
    if (!aligned(worker_scales, 4)) return fail(ONEBIT_EALIGN, "worker_scales misaligned");
    TRY(check_f32(p, server_err, "server_err"));
    TRY(check_u64(p, server_bits, "server_bits"));
    if (!server_scales) return fail(ONEBIT_EINVAL, "server_scales is NULL");
    if (!aligned(server_scales, 4)) return fail(ONEBIT_EALIGN, "server_scales misaligned");
    if (!workspace) return fail(ONEBIT_EINVAL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(ONEBIT_EALIGN, "workspace is not 256-byte aligned");
    if (server_begin < 0 || server_end > p->n || server_begin >= server_end)
        return fail(ONEBIT_EINVAL, "chunk range [%d, %d) is empty or outside [0, %d)",
                    server_begin, server_end, p->n);
    // Incoming words and scales must cover every owned segment.
    int64_t wlo = INT64_MAX, whi = -1;
    for (int32_t j = server_begin; j < server_end; ++j) {
        if (p->chunk_word_hi[j] < 0) continue;
        wlo = std::min(wlo, p->chunk_word_lo[j]);
        whi = std::max(whi, p->chunk_word_hi[j]);
    }
    if (whi >= 0) {
        if (bits_word_base < 0 || bits_word_base > wlo)
            return fail(ONEBIT_EINVAL, "bits_word_base %lld is not in [0, %lld]",
                        (long long)bits_word_base, (long long)wlo);
        TRY(check_ld(bits_ld, whi + 1 - bits_word_base, false, "bits_ld"));
    }
    const int64_t qlo = server_begin, qhi = (int64_t)(p->K - 1) * p->n + (server_end - 1);
    if (scales_seg_base < 0 || scales_seg_base > qlo)
        return fail(ONEBIT_EINVAL, "scales_seg_base %lld is not in [0, %lld]",
                    (long long)scales_seg_base, (long long)qlo);
    TRY(check_ld(scales_ld, qhi + 1 - scales_seg_base, false, "scales_ld"));
    return ONEBIT_OK;
}

int run_server(const onebit_plan_s *p, int32_t server_begin, int32_t server_end,
               const uint64_t *worker_bits, int64_t bits_ld, int64_t bits_word_base,
               const float *worker_scales, int64_t scales_ld, int64_t scales_seg_base,
               float *server_err, uint64_t *server_bits, float *server_scales, void *workspace,
               hipStream_t s)
{
    const int64_t tb = p->chunk_tile_begin[server_begin];
    const int64_t tc = p->chunk_tile_begin[server_end] - tb;
    double *part = (double *)((char *)workspace + server_partial_offset(p));
    const int nown = server_end - server_begin;
    const int64_t owned = (int64_t)p->K * nown;
    const bool worth = tc >= kServerTableMinTiles * owned &&
                       tc * ((p->n + 7) / 8) >= kServerTableMinWork;
    const bool use_tables = p->table_bytes > 0 &&
                            (p->server_tables == ONEBIT_SERVER_TABLES_ON ||
                             (p->server_tables == ONEBIT_SERVER_TABLES_AUTO && worth));
    double *tables = use_tables ? (double *)((char *)workspace + server_table_offset(p)) : nullptr;
    int32_t *flags = use_tables ? (int32_t *)((char *)workspace + server_flag_offset(p)) : nullptr;
    const int64_t bb = p->chunk_block_begin[server_begin];
    const int64_t nb = p->chunk_block_begin[server_end] - bb;
    if (tc > 0)
        TRY_HIP(onebit::launch_server_pass(p->tb, tb, tc, p->n, worker_bits, bits_ld,
                                           bits_word_base, worker_scales, scales_ld,
                                           scales_seg_base, server_err, server_scales,
                                           server_bits, part, p->K, server_begin, nown, tables,
                                           flags, p->tb.server_blocks + bb, nb, s),
                "server kernel launch");
    TRY_HIP(onebit::launch_finalize(p->tb, p->max_seg_tiles,
                                    (int64_t)p->K * (server_end - server_begin), p->S, 1, p->n,
                                    server_begin, server_end, part, p->T, server_scales, 0, s),
            "server scale kernel launch");
    return ONEBIT_OK;
}

int check_update(const onebit_plan_s *p, const uint64_t *server_bits,
                 const float *server_scales, const float *x, const float *m_out,
                 const float *v_frozen)
{
    TRY(check_u64(p, server_bits, "server_bits"));
    if (!server_scales) return fail(ONEBIT_EINVAL, "server_scales is NULL");
    if (!aligned(server_scales, 4)) return fail(ONEBIT_EALIGN, "server_scales misaligned");
    TRY(check_f32(p, x, "x"));
    if (m_out) TRY(check_f32(p, m_out, "m_out"));
    TRY(check_f32(p, v_frozen, "v_frozen"));
    return ONEBIT_OK;
}

int run_update(const onebit_plan_s *p, const uint64_t *server_bits, const float *server_scales,
               float *x, float *m_out, const float *v_frozen, float lr, float eps, hipStream_t s)
{
    if (p->T == 0) return ONEBIT_OK;
    TRY_HIP(onebit::launch_update(p->tb, p->T, server_bits, server_scales, x, m_out, v_frozen,
                                  lr, eps, s),
            "update kernel launch");
    return ONEBIT_OK;
}

int record(void *const *events, int k, hipStream_t s)
{
    if (events && events[k])
        TRY_HIP(hipEventRecord((hipEvent_t)events[k], s), "hipEventRecord");
    return ONEBIT_OK;
}

// The fused step: all n workers (rows of W words and S scales), all n chunk
// owners reading those rows in place, the update writing m when m is given.
int step_impl(onebit_plan_s *p, float *x, float *m, const float *v_frozen, const void *grads,
              int32_t grad_dtype, int64_t grad_ld, float *worker_err, int64_t err_ld,
              float *server_err, uint64_t *worker_bits, float *worker_scales,
              uint64_t *server_bits, float *server_scales, float lr, float beta1, float eps,
              void *workspace, void *const *events, hipStream_t s)
{
    TRY(check_plan(p));
    // Every argument is checked before the first launch, so an error writes nothing.
    TRY(check_worker(p, m, server_bits, server_scales, grads, grad_dtype, grad_ld, p->n,
                     worker_err, err_ld, worker_bits, p->W, worker_scales, p->S, workspace));
    TRY(check_server(p, 0, p->n, worker_bits, p->W, 0, worker_scales, p->S, 0, server_err,
                     server_bits, server_scales, workspace));
    TRY(check_update(p, server_bits, server_scales, x, m, v_frozen));
    TRY(record(events, 0, s));
    TRY(run_worker(p, m, server_bits, server_scales, grads, grad_dtype, grad_ld, p->n,
                   worker_err, err_ld, worker_bits, p->W, worker_scales, p->S, beta1, workspace,
                   s));
    TRY(record(events, 1, s));
    TRY(run_server(p, 0, p->n, worker_bits, p->W, 0, worker_scales, p->S, 0, server_err,
                   server_bits, server_scales, workspace, s));
    TRY(record(events, 2, s));
    TRY(run_update(p, server_bits, server_scales, x, m, v_frozen, lr, eps, s));
    return record(events, 3, s);
}

}  // namespace

extern "C" {

const char *onebit_status_str(int32_t status)
{
    switch (status) {
    case ONEBIT_OK: return "ONEBIT_OK";
    case ONEBIT_EINVAL: return "ONEBIT_EINVAL";
    case ONEBIT_EALIGN: return "ONEBIT_EALIGN";
    case ONEBIT_EHIP: return "ONEBIT_EHIP";
    case ONEBIT_ENOMEM: return "ONEBIT_ENOMEM";
    default: return "ONEBIT_UNKNOWN";
    }
}

const char *onebit_last_error(void) { return g_last_error; }

int onebit_plan_create(const int64_t *tensor_numel, int32_t num_tensors, int32_t n_workers,
                       onebit_plan *out)
{
    if (!out) return fail(ONEBIT_EINVAL, "out is NULL");
    *out = nullptr;
    if (!tensor_numel) return fail(ONEBIT_EINVAL, "tensor_numel is NULL");
    if (num_tensors < 1) return fail(ONEBIT_EINVAL, "num_tensors < 1");
    if (n_workers < 1) return fail(ONEBIT_EINVAL, "n_workers < 1");
    for (int32_t k = 0; k < num_tensors; ++k) {
        if (tensor_numel[k] < 0) return fail(ONEBIT_EINVAL, "tensor_numel[%d] < 0", k);
        // bounds the layout arithmetic (the padded total is limited to 2^40 below)
        if (tensor_numel[k] > ((int64_t)1 << 40))
            return fail(ONEBIT_EINVAL, "tensor_numel[%d] exceeds 2^40", k);
    }
    if ((int64_t)num_tensors * n_workers > INT32_MAX)
        return fail(ONEBIT_EINVAL, "num_tensors * n_workers = %lld segments exceeds 2^31 - 1",
                    (long long)num_tensors * n_workers);
    try {
        return plan_create_impl(tensor_numel, num_tensors, n_workers, out);
    } catch (const std::bad_alloc &) {
        return fail(ONEBIT_ENOMEM, "host allocation failed");
    }
}

int onebit_plan_destroy(onebit_plan p)
{
    if (!p) return fail(ONEBIT_EINVAL, "plan is NULL");
    int prev = -1;
    (void)hipGetDevice(&prev);
    if (prev != p->device) (void)hipSetDevice(p->device);
    hipError_t e = hipFree(p->dev_mem);
    if (prev >= 0 && prev != p->device) (void)hipSetDevice(prev);
    delete p;
    if (e != hipSuccess) return hip_fail(e, "hipFree of plan tables");
    return ONEBIT_OK;
}

int onebit_plan_get_info(onebit_plan p, onebit_plan_sizes *info)
{
    if (!p) return fail(ONEBIT_EINVAL, "plan is NULL");
    if (!info) return fail(ONEBIT_EINVAL, "info is NULL");
    info->d = p->d;
    info->padded_len = p->D;
    info->words = p->W;
    info->num_tensors = p->K;
    info->num_segments = p->S;
    info->num_tiles = p->T;
    info->n_workers = p->n;
    info->tile_elems = kTileElems;
    info->workspace_bytes = p->workspace_bytes;
    return ONEBIT_OK;
}

int onebit_plan_get_layout(onebit_plan p, int64_t *tensor_offset, int64_t *seg_begin,
                           int64_t *seg_end)
{
    if (!p) return fail(ONEBIT_EINVAL, "plan is NULL");
    if (tensor_offset) std::memcpy(tensor_offset, p->tensor_off.data(), p->K * sizeof(int64_t));
    if (seg_begin) std::memcpy(seg_begin, p->seg_begin.data(), p->S * sizeof(int64_t));
    if (seg_end) std::memcpy(seg_end, p->seg_end.data(), p->S * sizeof(int64_t));
    return ONEBIT_OK;
}

int onebit_plan_set_server_tables(onebit_plan p, int32_t mode)
{
    if (!p) return fail(ONEBIT_EINVAL, "plan is NULL");
    if (mode != ONEBIT_SERVER_TABLES_OFF && mode != ONEBIT_SERVER_TABLES_AUTO &&
        mode != ONEBIT_SERVER_TABLES_ON)
        return fail(ONEBIT_EINVAL, "server table mode %d is not 0, 1 or 2", mode);
    p->server_tables = mode;
    return ONEBIT_OK;
}

int onebit_plan_info(onebit_plan p, int64_t *padded_len, int64_t *words, int64_t *num_segments,
                     int64_t *chunk_len, size_t *workspace_bytes)
{
    if (!p) return fail(ONEBIT_EINVAL, "plan is NULL");
    if (padded_len) *padded_len = p->D;
    if (words) *words = p->W;
    if (num_segments) *num_segments = p->S;
    if (chunk_len) std::memcpy(chunk_len, p->chunk_len.data(), p->K * sizeof(int64_t));
    if (workspace_bytes) *workspace_bytes = p->workspace_bytes;
    return ONEBIT_OK;
}

int onebit_warmup_adam_step(onebit_plan p, float *x, float *m, float *v, const void *grads,
                            int32_t grad_dtype, int64_t grad_ld, int32_t n_grads, float lr,
                            float beta1,
                            float beta2, float eps, int32_t bias_correction, int64_t step,
                            onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_f32(p, x, "x"));
    TRY(check_f32(p, m, "m"));
    TRY(check_f32(p, v, "v"));
    TRY(check_grads(p, grads, grad_dtype));
    if (n_grads < 1) return fail(ONEBIT_EINVAL, "n_grads < 1");
    if (step < 1) return fail(ONEBIT_EINVAL, "step < 1 (steps are 1-based)");
    TRY(check_ld(grad_ld, p->D, n_grads > 1, "grad_ld"));
    if (p->T == 0) return ONEBIT_OK;
    float bc1 = 1.0f, bc2 = 1.0f;
    if (bias_correction) {
        bc1 = (float)(1.0 - std::pow((double)beta1, (double)step));
        bc2 = (float)(1.0 - std::pow((double)beta2, (double)step));
    }
    TRY_HIP(onebit::launch_warmup(p->tb, p->T, x, m, v, grads, grad_dtype, grad_ld, n_grads, lr,
                                  beta1,
                                  beta2, eps, bias_correction ? 1 : 0, bc1, bc2,
                                  (hipStream_t)stream),
            "warm-up kernel launch");
    return ONEBIT_OK;
}

int onebit_worker_compress(onebit_plan p, const float *m, const uint64_t *m_bits,
                           const float *m_scales, const void *grads, int32_t grad_dtype,
                           int64_t grad_ld, int32_t n_local, float *worker_err, int64_t err_ld,
                           uint64_t *worker_bits, int64_t bits_ld, float *worker_scales,
                           int64_t scales_ld, float beta1, void *workspace,
                           onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_worker(p, m, m_bits, m_scales, grads, grad_dtype, grad_ld, n_local, worker_err,
                     err_ld, worker_bits, bits_ld, worker_scales, scales_ld, workspace));
    return run_worker(p, m, m_bits, m_scales, grads, grad_dtype, grad_ld, n_local, worker_err,
                      err_ld, worker_bits, bits_ld, worker_scales, scales_ld, beta1, workspace,
                      (hipStream_t)stream);
}

int onebit_server_reduce_compress(onebit_plan p, int32_t server_begin, int32_t server_end,
                                  const uint64_t *worker_bits, int64_t bits_ld,
                                  int64_t bits_word_base, const float *worker_scales,
                                  int64_t scales_ld, int64_t scales_seg_base, float *server_err,
                                  uint64_t *server_bits, float *server_scales, void *workspace,
                                  onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_server(p, server_begin, server_end, worker_bits, bits_ld, bits_word_base,
                     worker_scales, scales_ld, scales_seg_base, server_err, server_bits,
                     server_scales, workspace));
    return run_server(p, server_begin, server_end, worker_bits, bits_ld, bits_word_base,
                      worker_scales, scales_ld, scales_seg_base, server_err, server_bits,
                      server_scales, workspace, (hipStream_t)stream);
}

int onebit_decompress_update(onebit_plan p, const uint64_t *server_bits,
                             const float *server_scales, float *x, float *m_out,
                             const float *v_frozen, float lr, float eps, onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_update(p, server_bits, server_scales, x, m_out, v_frozen));
    return run_update(p, server_bits, server_scales, x, m_out, v_frozen, lr, eps,
                      (hipStream_t)stream);
}

int onebit_step(onebit_plan p, float *x, float *m, const float *v_frozen, const void *grads,
                int32_t grad_dtype, int64_t grad_ld, float *worker_err, int64_t err_ld, float *server_err,
                uint64_t *worker_bits, float *worker_scales, uint64_t *server_bits,
                float *server_scales, float lr, float beta1, float eps, void *workspace,
                onebit_stream stream)
{
    return step_impl(p, x, m, v_frozen, grads, grad_dtype, grad_ld, worker_err, err_ld,
                     server_err, worker_bits, worker_scales, server_bits, server_scales, lr,
                     beta1, eps, workspace, nullptr, (hipStream_t)stream);
}

int onebit_step_noalloc(onebit_plan p, float *x, float *m, const float *v_frozen,
                        const void *grads, int32_t grad_dtype, int64_t grad_ld,
                        float *worker_err, int64_t err_ld, float *server_err,
                        uint64_t *worker_bits, float *worker_scales, uint64_t *server_bits,
                        float *server_scales, float lr, float beta1, float eps,
                        onebit_stream stream)
{
    TRY(check_plan(p));
    if (p->workspace_bytes > onebit::kScratchBytes)
        return fail(ONEBIT_EINVAL,
                    "the plan needs %zu bytes of workspace; onebit_step_noalloc's scratch holds "
                    "%zu (use onebit_step with a caller workspace)",
                    p->workspace_bytes, onebit::kScratchBytes);
    void *scratch = nullptr;
    TRY_HIP(onebit::scratch_address(p->device, &scratch), "scratch symbol lookup");
    return step_impl(p, x, m, v_frozen, grads, grad_dtype, grad_ld, worker_err, err_ld,
                     server_err, worker_bits, worker_scales, server_bits, server_scales, lr,
                     beta1, eps, scratch, nullptr, (hipStream_t)stream);
}

int onebit_step_events(onebit_plan p, float *x, float *m, const float *v_frozen,
                       const void *grads, int32_t grad_dtype, int64_t grad_ld, float *worker_err,
                       int64_t err_ld, float *server_err, uint64_t *worker_bits,
                       float *worker_scales, uint64_t *server_bits, float *server_scales,
                       float lr, float beta1, float eps, void *workspace, void *const *events,
                       onebit_stream stream)
{
    if (!events) return fail(ONEBIT_EINVAL, "events is NULL");
    return step_impl(p, x, m, v_frozen, grads, grad_dtype, grad_ld, worker_err, err_ld,
                     server_err, worker_bits, worker_scales, server_bits, server_scales, lr,
                     beta1, eps, workspace, events, (hipStream_t)stream);
}

int onebit_adam_message_step(onebit_plan p, float *x, float *m, float *v, const uint64_t *bits,
                             const float *scales, float lr, float beta1, float beta2, float eps,
                             int32_t bias_correction, int64_t step, onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_f32(p, x, "x"));
    TRY(check_f32(p, m, "m"));
    TRY(check_f32(p, v, "v"));
    TRY(check_u64(p, bits, "bits"));
    if (!scales) return fail(ONEBIT_EINVAL, "scales is NULL");
    if (!aligned(scales, 4)) return fail(ONEBIT_EALIGN, "scales misaligned");
    if (step < 1) return fail(ONEBIT_EINVAL, "step < 1 (steps are 1-based)");
    if (p->T == 0) return ONEBIT_OK;
    float bc1 = 1.0f, bc2 = 1.0f;
    if (bias_correction) {
        bc1 = (float)(1.0 - std::pow((double)beta1, (double)step));
        bc2 = (float)(1.0 - std::pow((double)beta2, (double)step));
    }
    TRY_HIP(onebit::launch_adam_message(p->tb, p->T, bits, scales, x, m, v, lr, beta1, beta2, eps,
                                        bias_correction ? 1 : 0, bc1, bc2, (hipStream_t)stream),
            "message Adam kernel launch");
    return ONEBIT_OK;
}

int onebit_uncompressed_step(onebit_plan p, float *x, float *m, const float *v_frozen,
                             const void *grads, int32_t grad_dtype, int64_t grad_ld,
                             int32_t n_grads, float lr, float beta1, float eps,
                             onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_f32(p, x, "x"));
    TRY(check_f32(p, m, "m"));
    TRY(check_f32(p, v_frozen, "v_frozen"));
    TRY(check_grads(p, grads, grad_dtype));
    if (n_grads < 1) return fail(ONEBIT_EINVAL, "n_grads < 1");
    TRY(check_ld(grad_ld, p->D, n_grads > 1, "grad_ld"));
    if (p->T == 0) return ONEBIT_OK;
    TRY_HIP(onebit::launch_uncompressed(p->tb, p->T, x, m, v_frozen, grads, grad_dtype, grad_ld,
                                        n_grads, lr, beta1, eps, (hipStream_t)stream),
            "uncompressed step kernel launch");
    return ONEBIT_OK;
}

int onebit_l1_norm(onebit_plan p, const float *v, void *workspace, double *out,
                   onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_f32(p, v, "v"));
    if (!workspace) return fail(ONEBIT_EINVAL, "workspace is NULL");
    if (!aligned(workspace, 256)) return fail(ONEBIT_EALIGN, "workspace is not 256-byte aligned");
    if (!out) return fail(ONEBIT_EINVAL, "out is NULL");
    if (!aligned(out, 8)) return fail(ONEBIT_EALIGN, "out is not 8-byte aligned");
    double *part = (double *)((char *)workspace + server_partial_offset(p));
    TRY_HIP(onebit::launch_l1_norm(p->tb, p->T, v, part, out, (hipStream_t)stream),
            "l1 norm kernel launch");
    return ONEBIT_OK;
}

int onebit_decode(onebit_plan p, const uint64_t *bits, const float *scales, float *out,
                  onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_u64(p, bits, "bits"));
    if (!scales) return fail(ONEBIT_EINVAL, "scales is NULL");
    if (!aligned(scales, 4)) return fail(ONEBIT_EALIGN, "scales misaligned");
    TRY(check_f32(p, out, "out"));
    if (p->T == 0) return ONEBIT_OK;
    TRY_HIP(onebit::launch_decode(p->tb, p->T, bits, scales, out, (hipStream_t)stream),
            "decode kernel launch");
    return ONEBIT_OK;
}

int onebit_error_materialize(onebit_plan p, const float *err_state, int64_t err_ld,
                             const float *scales, int64_t scales_ld, int32_t rows,
                             float *delta_out, int64_t out_ld, onebit_stream stream)
{
    TRY(check_plan(p));
    TRY(check_f32(p, err_state, "err_state"));
    TRY(check_f32(p, delta_out, "delta_out"));
    if (!scales) return fail(ONEBIT_EINVAL, "scales is NULL");
    if (!aligned(scales, 4)) return fail(ONEBIT_EALIGN, "scales misaligned");
    if (rows < 1) return fail(ONEBIT_EINVAL, "rows < 1");
    TRY(check_ld(err_ld, p->D, rows > 1, "err_ld"));
    TRY(check_ld(out_ld, p->D, rows > 1, "out_ld"));
    TRY(check_ld(scales_ld, rows > 1 ? p->S : 0, false, "scales_ld"));
    if (delta_out == err_state && out_ld != err_ld)
        return fail(ONEBIT_EINVAL, "in-place materialize needs out_ld == err_ld");
    if (p->T == 0) return ONEBIT_OK;
    TRY_HIP(onebit::launch_materialize(p->tb, p->T, rows, err_state, err_ld, scales, scales_ld,
                                       delta_out, out_ld, (hipStream_t)stream),
            "materialize kernel launch");
    return ONEBIT_OK;
}

}  // extern "C"
