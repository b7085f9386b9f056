// Internal interface between the C-ABI entry points (daso_api.hip) and the
// kernels (daso_kernels.hip).  Not part of the public ABI.
#pragma once

#include <stdint.h>
#include <hip/hip_runtime.h>

#include "daso.h"

namespace daso {

// Work decomposition.  A launch covers up to kLaunchBuckets buckets.  Each bucket
// [start, end) is cut into tiles of kTile elements aligned to kVec-element
// vectors (the first tile of a bucket starts at the bucket start rounded down to
// a vector boundary and is clipped to the bucket); a 256-thread workgroup
// processes a tile as kIters vectors of kVec elements per thread.
// Tuning parameters (compile-time; the defaults are the measured best on MI355X).
#ifndef DASO_TILE_ITERS
#define DASO_TILE_ITERS 2
#endif
#ifndef DASO_BATCH
#define DASO_BATCH 2
#endif
#ifndef DASO_BLOCKS_PER_CU
#define DASO_BLOCKS_PER_CU 0
#endif
#ifndef DASO_NT_PARAMS
#define DASO_NT_PARAMS 1
#endif
#ifndef DASO_BLOCK
#define DASO_BLOCK 256
#endif
constexpr int kBlock = DASO_BLOCK;
constexpr int kVec = 4;
constexpr int kIters = DASO_TILE_ITERS;
constexpr int kBatch = DASO_BATCH;           // vectors whose loads are issued together
constexpr int kBlocksPerCU = DASO_BLOCKS_PER_CU;  // 0: one workgroup per tile
constexpr bool kNtParams = DASO_NT_PARAMS != 0;   // non-temporal access to params/momentum
// Streams (inputs + outputs) from which each XCD is given a contiguous run of
// tiles; measured: a gain with 42 streams, a loss with 17 and 25.
constexpr int kXcdOrderMinStreams = 32;
constexpr int64_t kTile = int64_t(kBlock) * kVec * kIters;
constexpr int kLaunchBuckets = 64;

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
  daso_bucket_stats* stats;  // per-bucket outputs (stats only), already offset to this launch
  int32_t g;
  int32_t P;
  float lr;
  float mu;
  float wd;
  uint32_t flags;
  int32_t nb;            // buckets in this launch
  int32_t ntiles;        // tiles in this launch
  int32_t xcd_order;     // nonzero: renumber workgroups XCD-contiguously
  int32_t xf32;          // nonzero: fp32 exchange (stale copies and wire are fp32)
  TileBucket b[kLaunchBuckets];
};

// Number of tiles bucket [start, end) is cut into.
inline int64_t tiles_of(int64_t start, int64_t end) {
  if (end <= start) return 0;
  const int64_t a = start & ~int64_t(kVec - 1);
  return (end - a + kTile - 1) / kTile;
}

// Enqueue one launch of `mode` over the buckets in `args` with `grid`
// workgroups (1 <= grid <= args.ntiles), which take the tiles in turn.
hipError_t launch_step(Mode mode, bool with_stats, const StepArgs& args, int grid, hipStream_t stream);

}  // namespace daso
