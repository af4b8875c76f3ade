// Enumerates launches of the tile kernels on the host, with the same grid
// functions the kernels and their launchers use, and checks that every tile
// (one wave per tile) or worker item (XCD-contiguous walk, possibly strided)
// is taken by exactly one wave.  Exit status 0 when every case passes.
#include "onebit_grid.h"

#include <cstdio>
#include <vector>

using namespace onebit;

static int failures = 0;
static long cases = 0;

static void fail(const char *what, long long a, long long b)
{
    if (failures < 20) std::printf("FAIL %s (%lld, %lld)\n", what, a, b);
    ++failures;
}

// waves_per_block tiles per block (one wave per tile, or one pair of waves),
// logical block order.
static void check_tiles(int64_t tiles, int waves_per_block)
{
    ++cases;
    const int64_t grid = xcd_grid(tiles, waves_per_block);
    if (grid % kXcds) fail("tile grid not a multiple of the XCD count", tiles, grid);
    if (grid * waves_per_block < tiles) fail("tile grid too small", tiles, grid);
    std::vector<unsigned char> seen((size_t)tiles, 0);
    std::vector<unsigned char> lseen((size_t)grid, 0);
    for (int64_t b = 0; b < grid; ++b) {
        const int64_t lb = xcd_block_of(b, grid);
        if (lb < 0 || lb >= grid) { fail("logical block out of range", b, grid); continue; }
        if (lseen[(size_t)lb]++) fail("logical block taken twice", lb, grid);
        for (int w = 0; w < waves_per_block; ++w) {
            const int64_t t = lb * waves_per_block + w;
            if (t < tiles && seen[(size_t)t]++) fail("tile taken twice", t, tiles);
        }
    }
    for (int64_t t = 0; t < tiles; ++t)
        if (!seen[(size_t)t]) fail("tile not taken", t, tiles);
}

// The chunk owners' shared-table workgroups of a list of segments with the
// given tile counts, laid out one after another from list position base:
// every tile is taken once, by a workgroup of that segment, as wave
// (position - first).
static void check_server_blocks(const std::vector<int64_t> &counts, int64_t base = 0)
{
    ++cases;
    int64_t total = 0;
    for (int64_t c : counts) total += c;
    std::vector<int> owner((size_t)total, -1);
    std::vector<int> seen((size_t)total, 0);
    int64_t pos = 0;
    for (size_t q = 0; q < counts.size(); ++q) {
        for (int64_t t = pos; t < pos + counts[q]; ++t) owner[(size_t)t] = (int)q;
        pos += counts[q];
    }
    pos = 0;
    for (size_t q = 0; q < counts.size(); ++q) {
        const int64_t nb = server_blocks_of(counts[q]);
        for (int64_t i = 0; i < nb; ++i) {
            const int32_t e = server_block_entry(base + pos, counts[q], i);
            const int64_t first = server_block_first(e) - base;
            const int tiles = server_block_tiles(e);
            if (tiles < 1 || tiles > kWavesPerBlock) fail("workgroup tile count", tiles, (long long)q);
            for (int w = 0; w < tiles; ++w) {
                const int64_t t = first + w;
                if (t < 0 || t >= total) { fail("workgroup tile out of range", t, total); break; }
                if (owner[(size_t)t] != (int)q) fail("workgroup crosses a segment", t, (long long)q);
                ++seen[(size_t)t];
            }
        }
        pos += counts[q];
    }
    for (int64_t t = 0; t < total; ++t)
        if (seen[(size_t)t] != 1) { fail("tile taken other than once", t, seen[(size_t)t]); break; }
}

// The worker pass: items walked per XCD, one workgroup per item, with a grid
// capped at max_blocks.
static void check_worker(int64_t items, int64_t max_blocks)
{
    ++cases;
    const int64_t grid = worker_grid(items, max_blocks);
    if (grid % kXcds) fail("worker grid not a multiple of the XCD count", items, grid);
    if (grid > max_blocks + kXcds - 1) fail("worker grid above its cap", items, grid);
    std::vector<unsigned char> seen((size_t)items, 0);
    for (int64_t b = 0; b < grid; ++b) {
        const ItemWalk walk = xcd_item_walk(b, grid, items);
        if (walk.stride <= 0) { fail("non-positive stride", items, grid); return; }
        for (int64_t i = walk.first; i < walk.end; i += walk.stride) {
            if (i < 0 || i >= items) { fail("item out of range", i, items); break; }
            if (seen[(size_t)i]++) fail("item taken twice", i, items);
        }
    }
    for (int64_t i = 0; i < items; ++i)
        if (!seen[(size_t)i]) { fail("item not taken", i, items); break; }
}

// The first compression step's launches: pieces of at most kMaxLaunchTiles
// tiles, kWorkerRowTiles tiles per 16-wave workgroup, two waves per tile
// (wave w of logical block lb takes half w % 2 of tile base + lb * 8 + w / 2,
// active below the plan's tile count).  Every half tile is taken once and no
// launch reaches 2^32 work-items.  enumerate = false checks the launch sizes
// only (for counts too large to enumerate here).
static void check_row_pieces(int64_t tiles, bool enumerate)
{
    ++cases;
    std::vector<unsigned char> seen(enumerate ? (size_t)tiles * 2 : 0, 0);
    int64_t covered = 0;
    for (int64_t base = 0; base < tiles; base += kMaxLaunchTiles) {
        const int64_t count = launch_piece(tiles, base);
        if (count <= 0 || count > kMaxLaunchTiles) { fail("bad piece", base, count); return; }
        const int64_t grid = xcd_grid(count, kWorkerRowTiles);
        if (grid * kRowBlock >= ((int64_t)1 << 32)) fail("row launch of 2^32 work-items", tiles, grid);
        if (base + count < tiles && grid * kWorkerRowTiles != count)
            fail("spare workgroups in a piece before the last", tiles, base);
        covered += count;
        if (!enumerate) continue;
        for (int64_t b = 0; b < grid; ++b) {
            const int64_t lb = xcd_block_of(b, grid);
            for (int w = 0; w < kRowWaves; ++w) {
                const int64_t t = base + lb * kWorkerRowTiles + w / 2;
                if (t >= tiles) continue;
                if (seen[(size_t)(2 * t + w % 2)]++) fail("half tile taken twice", t, tiles);
            }
        }
    }
    if (covered != tiles) fail("pieces do not cover the tiles", covered, tiles);
    for (size_t i = 0; i < seen.size(); ++i)
        if (!seen[i]) { fail("half tile not taken", (long long)i / 2, tiles); break; }
}

// The chunk owners' launches with one 256-thread workgroup per tile (or per
// entry of the shared-table block list): pieces below 2^32 work-items that
// cover the range.
static void check_server_pieces(int64_t count_total)
{
    ++cases;
    int64_t covered = 0;
    for (int64_t off = 0; off < count_total; off += kMaxLaunchTiles) {
        const int64_t count = launch_piece(count_total, off);
        const int64_t grid = xcd_grid(count, 1);
        if (grid * 256 >= ((int64_t)1 << 32)) fail("server launch of 2^32 work-items", count_total, grid);
        covered += count;
    }
    if (covered != count_total) fail("server pieces do not cover the range", covered, count_total);
}

int main()
{
    for (int64_t t : {1LL, 7LL, 8LL, 63LL, 64LL, 65LL, 326288LL, (1LL << 22) - 1, 1LL << 22,
                      (1LL << 22) + 1, 3 * (1LL << 22) + 5})
        check_row_pieces(t, true);
    for (int64_t t : {(1LL << 25) - 1, (1LL << 25) - 64, (1LL << 24) + 3})
        check_row_pieces(t, false);
    for (int64_t t : {1LL, 1275LL, 326288LL, (1LL << 22) + 1, (1LL << 24) - 1, (1LL << 25) - 1})
        check_server_pieces(t);
    // tiles per block: the streaming kernels (kWavesPerBlock), the row-summing
    // ones (kRowWaves) and the first compression step (kWorkerRowTiles, two
    // waves per tile)
    for (int wpb : {kWavesPerBlock, kRowWaves, kWorkerRowTiles}) {
        for (int64_t t = 1; t <= 600; ++t) check_tiles(t, wpb);
        // BERT-Large (326,288 tiles) and the stress workload's tile counts
        for (int64_t t : {326288LL, 542089LL, 106344LL, 1275LL}) check_tiles(t, wpb);
    }

    // segments of 0..40 tiles, BERT-Large's 32 segments of about 10,200 tiles
    // and entries near the 2^25-tile limit
    {
        std::vector<int64_t> counts;
        for (int64_t c = 0; c <= 40; ++c) counts.push_back(c);
        check_server_blocks(counts);
        check_server_blocks(std::vector<int64_t>(32, 10196));
        check_server_blocks({9, 5, 1, 2}, (1LL << 25) - 17);
    }

    for (int64_t items = 1; items <= 700; ++items)
        for (int64_t cap : {1LL, 3LL, 8LL, 9LL, 24LL, 64LL, (long long)kMaxWorkerGridBlocks})
            check_worker(items, cap);
    // BERT-Large, n = 32: one item per wave under the real cap, and strided
    // walks under smaller caps (including the former 2^22-block cap)
    const int64_t bert = 32LL * 326288;
    for (int64_t cap : {(long long)kMaxWorkerGridBlocks, (long long)kMaxGridBlocks, 1000003LL, 4096LL})
        check_worker(bert, cap);
    // item counts whose eighths are ragged
    for (int64_t items : {8LL * 1000 + 7, 8LL * 1000 + 1, 123457LL})
        for (int64_t cap : {5LL, 40LL, 1000LL})
            check_worker(items, cap);

    if (failures) {
        std::printf("grid_check: %d failure(s) in %ld cases\n", failures, cases);
        return 1;
    }
    std::printf("grid_check: ok (%ld cases)\n", cases);
    return 0;
}
