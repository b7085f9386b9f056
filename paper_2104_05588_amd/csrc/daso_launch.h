// Internal interface between the C-ABI entry points (daso_api.hip) and the
// kernels (daso_kernels.hip).  Not part of the public ABI.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

#include "daso.h"

namespace daso {

// Work decomposition.  A launch covers up to kLaunchBuckets buckets.  Tiles lie
// on one grid counted from element 0 (see tiles_of); each bucket [start, end)
// takes the grid tiles it overlaps, the first and last clipped to the bucket.
// One 256-thread workgroup processes one tile, each
// thread one batch of vectors whose loads are all issued before any store.  The
// batch, and so the tile, depends on the kernel instance: two vectors per thread
// (2048-element tiles) when a vector's inputs take at most 48 registers, one
// (1024-element tiles) otherwise.  tile_elems() tells the host which.
//
// Tuning parameters (compile-time; the defaults are the measured best on MI355X).
#ifndef DASO_BATCH
#define DASO_BATCH 2
#endif
#ifndef DASO_NT_PARAMS
#define DASO_NT_PARAMS 1
#endif
constexpr int kBlock = 256;
constexpr int kVec = 4;
constexpr int kBatch = DASO_BATCH;               // most vectors per thread and tile
constexpr bool kNtParams = DASO_NT_PARAMS != 0;  // non-temporal access to params/momentum
constexpr int kGenericIters = 2;                 // vectors per thread for runtime stream counts
constexpr int kLaunchBuckets = 64;
// Tile order across the 8 XCDs: workgroups go to the XCDs in turn, and a
// launch runs faster when each XCD takes runs of consecutive tiles.
//  - Fused step from 9 streams: runs of ntiles / 512 tiles rounded down to a
//    power of two (about 64 blocks of 8 runs per launch): 16 tiles of 2048
//    elements for the resnet50-shaped step, 128 of 1024 for the
//    segmentation-shaped one, 512 of 1024 for the GPT-shaped one.  Measured on
//    MI355X against the runs that were best for a fixed stream count: the
//    GPT-shaped step 2 to 3% faster with 256 to 512 tiles than with 32 (two
//    boxes), the same 45 streams over the 25.6M-parameter set best at 16 to 32,
//    the resnet50-shaped step best at 32K elements, the segmentation-shaped one
//    at 128K to 512K or plain order under the occupancy cap below.
//  - Other launches: runs of 32 tiles from 32 streams, 16 from 20 (+4 to 5%
//    with 45 streams, -2.3 to +5.5% with 25), plain order below (the separate
//    entry points move by about 1% either way).
constexpr int kXcdRunFusedStreams = 9;         // fused step: runs scaled to the launch from here
constexpr int64_t kXcdRunBlocksPerLaunch = 64;  // fused step: about this many blocks of 8 runs
constexpr int kXcdRunMidStreams = 20;   // other launches: runs of kXcdRunMid tiles from here
constexpr int kXcdRunMid = 16;
constexpr int kXcdRunManyStreams = 32;  // other launches: runs of kXcdRunMany tiles from here
constexpr int kXcdRunMany = 32;

// Occupancy of the fused step.  Loads of a workgroup's whole tile are in flight
// at once, and the step runs faster with fewer of them: a fused launch of at
// least kCapStreams streams holds enough LDS per workgroup (the kernel uses none
// of it) that at most kCapWorkgroupsPerCU share a CU, i.e. 2 waves per SIMD.
// Measured on four MI355X boxes: the resnet50-shaped step 2.5 to 5% faster
// (212.9 against 223.6 us cold on one), the segmentation-shaped one 2.6 to 4%,
// the node shapes from g = 4, P = 2 up 1 to 5%; 3 per CU gains at most 1%, 1
// per CU loses 10%.  Launches of fewer streams keep their occupancy (the local
// step g = 4, P = 0 with 9 streams is 1% slower capped; the pack with 2 is 40%
// slower), as do the separate entry points.
constexpr int kCapStreams = 10;
constexpr int kCapWorkgroupsPerCU = 2;
constexpr int32_t kCuLdsBytes = 160 * 1024;  // LDS per CU on gfx950

// LDS per workgroup that lets at most k workgroups share a CU: a 1 KB margin
// covers the kernel's own few bytes of LDS and the allocation granule.
inline int32_t lds_for_workgroups_per_cu(int32_t k) { return k >= 1 ? kCuLdsBytes / k - 1024 : 0; }

// An eager fused launch with statistics of at most this many tiles has its
// last workgroup sum the statistics (StepArgs::done) instead of a second
// launch: each of its workgroups pays an agent-scope fence (about 0.1 us of GPU
// time each), which is cheaper than a launch's host cost for a few dozen
// workgroups and far dearer for thousands.  Captured calls keep the second
// launch, whose host cost a graph replay does not pay.
constexpr int64_t kFinishStatsMaxTiles = 64;

// Bytes at the start of a statistics scratch buffer that hold the counter of
// StepArgs::done (zero whenever no launch is running); the tile partials and
// the bucket table follow.
constexpr size_t kStatsCounterBytes = 256;

enum Mode : int { kModeAvg = 0, kModePack = 1, kModeMerge = 2, kModeFused = 3 };

struct TileBucket {
  int64_t start;       // first element of the bucket
  int64_t end;         // one past its last element
  int32_t first_tile;  // index of its first tile within the launch
  int32_t S;           // staleness of Eq. (1)
};

// Per-tile side-output partial, reduced per bucket by stats_kernel.
struct TilePartial {
  double grad_sq;
  double delta_sq;
  uint64_t nonfinite;
};

// Kernel arguments, passed by value (about 2.7 KB).
struct StepArgs {
  const float* grads[DASO_MAX_G];
  const void* stale[DASO_MAX_P];  // bf16 patterns, or fp32 when xf32
  const float* src;      // pack: source fp32
  float* x;              // params (merge/fused, in place)
  float* m;              // momentum (fused, in place)
  void* wire;            // packed output (bf16, or fp32 when xf32) or nullptr
  float* gavg;           // local average output or nullptr
  TilePartial* partials; // per-tile partials (stats only)
  int32_t* tile_table;   // (stats only) nb + 1 entries written by workgroup 0 for stats_kernel:
                         // the first tile of each bucket, then ntiles
  daso_bucket_stats* stats;  // per-bucket outputs (stats only), already offset to this launch
  uint32_t* done;        // (stats only) nonnull: no stats_kernel; the workgroup that finishes last
                         // sums the statistics.  A counter that is zero before the launch and
                         // that the launch leaves at zero.
  int32_t g;
  int32_t P;
  float lr;
  float mu;
  float wd;
  uint32_t flags;
  int32_t nb;            // buckets in this launch
  int32_t ntiles;        // tiles in this launch
  int32_t xcd_run;       // > 1: each XCD takes runs of this many consecutive tiles
  int32_t xf32;          // nonzero: fp32 exchange (stale copies and wire are fp32)
  TileBucket b[kLaunchBuckets];
};

// Arguments of stats_kernel, kept to a few pointers: the host cost of a launch
// grows with the size of its arguments (about 2.7 us with 16 bytes, 4 us with
// 2.7 KB on MI355X), and the bucket ranges it needs are in tile_table.
struct StatsArgs {
  const TilePartial* partials;
  const int32_t* tile_table;
  daso_bucket_stats* stats;
  int32_t nb;
};

// Workgroups are dispatched to the 8 XCDs of the chip in turn (workgroup w to
// XCD w % 8).  xcd_runs renumbers workgroup w so that each XCD takes runs of
// `run` consecutive tiles: the k-th workgroup of XCD x in block b (of 8 * run
// tiles) gets tile b * 8 * run + x * run + k.  Workgroups past the last whole
// block keep their number.  A bijection of [0, grid); run = 1 is the identity.
__device__ __forceinline__ int xcd_runs(int w, int grid, int run) {
  const int block = 8 * run;
  if (w >= (grid / block) * block) return w;
  const int j = w >> 3, x = w & 7;
  return (j / run) * block + x * run + (j % run);
}

// Tiles lie on one grid of `tile` elements counted from element 0, so that a
// wavefront's accesses start on whole cache lines wherever a bucket begins; a
// bucket [start, end) takes the grid tiles it overlaps, clipped to its range.
inline int64_t tiles_of(int64_t start, int64_t end, int64_t tile) {
  if (end <= start) return 0;
  return (end - 1) / tile - start / tile + 1;
}

// Elements per tile of the kernel instance that launch_step picks for these
// arguments (mode, stream counts, exchange type).
int64_t tile_elems(Mode mode, bool with_stats, const StepArgs& args);

// Enqueue one launch of `mode` over the buckets in `args` (args.ntiles tiles,
// counted with tile_elems()) on `grid` workgroups (one per tile, or fewer, each
// then looping over tiles grid apart), each holding `lds` bytes of LDS.
hipError_t launch_step(Mode mode, bool with_stats, const StepArgs& args, uint32_t grid, uint32_t lds,
                       hipStream_t stream);

// Enqueue the zeroing of the counter at the start of a new statistics buffer.
hipError_t clear_stats_counter(void* buffer, hipStream_t stream);

}  // namespace daso
