// Launch shapes of the tile kernels and the order in which their waves take
// work.  Integer arithmetic only, with no HIP dependency, so that a host
// program can enumerate a whole launch and check that every tile or item is
// taken by exactly one wave.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define ONEBIT_HD __host__ __device__
#else
#define ONEBIT_HD
#endif

namespace onebit {

constexpr int kWave = 64;
constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;
// The packed worker pass runs one tile per two-wave workgroup, half a tile
// per wave.
constexpr int kWorkerWavesPerBlock = 2;
constexpr int kWorkerBlock = kWave * kWorkerWavesPerBlock;

// The kernels that sum the n gradient rows of each tile (warm-up, the 32-bit
// comparison step) run 16-wave workgroups over 16 consecutive tiles.
constexpr int kRowWaves = 16;
constexpr int kRowBlock = kWave * kRowWaves;
// The first compression step's row walk gives two waves to each tile (half a
// tile each), so its 16-wave workgroups cover 8 tiles.
constexpr int kWorkerRowTiles = kRowWaves / kWorkerWavesPerBlock;

// Workgroups are dispatched to the chip's 8 XCDs round-robin (block b runs on
// XCD (b + c) % 8 for a fixed c), and each XCD has its own L2.  Grids are
// launched as multiples of 8 blocks and renumbered so that each XCD takes one
// contiguous eighth of the work: every XCD then streams its own address range
// instead of all eight interleaving pieces of the same streams.
constexpr int kXcds = 8;

// Plans keep the tile count below 2^25, so a grid of one wave per tile stays
// far below the 2^32 work-item limit.  Kernels over larger pair counts cap
// their grid at kMaxGridBlocks and stride.  The worker grid (128-thread
// blocks) may reach 2^24 blocks, 2^31 work-items, so that a BERT-Large-sized
// pass (n = 32) runs one item per workgroup.  Kernels that give more than 64
// threads to a tile (the first compression step: 128; the chunk owners'
// per-tile workgroups: up to 256) are launched over at most kMaxLaunchTiles
// tiles (or table-sharing workgroups) at a time, at most 2^30 work-items per
// launch.
constexpr int64_t kMaxGridBlocks = (int64_t)1 << 22;
constexpr int64_t kMaxWorkerGridBlocks = (int64_t)1 << 24;
constexpr int64_t kMaxLaunchTiles = (int64_t)1 << 22;

// Tiles (or workgroups) of the launch that starts at base, of total.
ONEBIT_HD inline int64_t launch_piece(int64_t total, int64_t base)
{
    return total - base < kMaxLaunchTiles ? total - base : kMaxLaunchTiles;
}

// Blocks for one wave per item at waves_per_block waves per block, rounded up
// to a multiple of kXcds (0 for no items).
ONEBIT_HD inline int64_t xcd_grid(int64_t waves, int waves_per_block)
{
    const int64_t blocks = (waves + waves_per_block - 1) / waves_per_block;
    return (blocks + kXcds - 1) / kXcds * kXcds;
}

// Logical block of physical block b in a grid of `grid` blocks (a multiple of
// kXcds): the blocks of XCD x are logical blocks [x, x + 1) * grid / kXcds.
ONEBIT_HD inline int64_t xcd_block_of(int64_t b, int64_t grid)
{
    return (b % kXcds) * (grid / kXcds) + b / kXcds;
}

// Chunk owners' workgroups that share one segment's lookup tables: each takes
// up to kWavesPerBlock consecutive tiles of one segment in the chunk-major
// tile list, one per wave.  A segment whose tiles sit at list positions
// [pos, pos + count) gets server_blocks_of(count) workgroups; entry i is
// server_block_entry(pos, count, i), from which the kernel reads the first
// position and the number of tiles.  Positions stay below 2^25 (the plans'
// tile limit), so an entry fits an int32.
ONEBIT_HD inline int64_t server_blocks_of(int64_t count)
{
    return (count + kWavesPerBlock - 1) / kWavesPerBlock;
}

ONEBIT_HD inline int32_t server_block_entry(int64_t pos, int64_t count, int64_t i)
{
    const int64_t first = pos + i * kWavesPerBlock;
    const int64_t left = pos + count - first;
    return (int32_t)(first * 8 + (left < kWavesPerBlock ? left : kWavesPerBlock));
}

ONEBIT_HD inline int64_t server_block_first(int32_t entry) { return entry >> 3; }
ONEBIT_HD inline int server_block_tiles(int32_t entry) { return entry & 7; }

// Worker pass: items [0, num_items) are cut into kXcds contiguous ranges and
// XCD x walks range x with its grid / kXcds blocks; a grid smaller than the
// item count strides within the range.  Physical block b (all its waves
// together) takes items first, first + stride, ... below end.
struct ItemWalk {
    int64_t first;
    int64_t end;
    int64_t stride;
};

ONEBIT_HD inline ItemWalk xcd_item_walk(int64_t b, int64_t grid, int64_t num_items)
{
    const int64_t per_xcd = (num_items + kXcds - 1) / kXcds;
    const int64_t begin = (b % kXcds) * per_xcd;
    ItemWalk r;
    r.first = begin + b / kXcds;
    r.end = begin + per_xcd < num_items ? begin + per_xcd : num_items;
    r.stride = grid / kXcds;
    return r;
}

// Worker grid: one workgroup per item, at most max_blocks blocks, rounded up
// to a multiple of kXcds.
ONEBIT_HD inline int64_t worker_grid(int64_t items, int64_t max_blocks)
{
    int64_t blocks = items;
    if (blocks > max_blocks) blocks = max_blocks;
    return (blocks + kXcds - 1) / kXcds * kXcds;
}

}  // namespace onebit
