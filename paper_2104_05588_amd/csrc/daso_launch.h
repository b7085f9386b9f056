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
// a vector boundary and is clipped to the bucket); one 256-thread workgroup
// processes one tile, kIters vectors of kVec elements per thread.
constexpr int kBlock = 256;
constexpr int kVec = 4;
constexpr int kIters = 8;
constexpr int64_t kTile = int64_t(kBlock) * kVec * kIters;  // 8192 elements
constexpr int kLaunchBuckets = 64;

enum Mode : int { kModeAvg = 0, kModePack = 1, kModeMerge = 2, kModeFused = 3 };

struct TileBucket {
  int64_t start;       // first element of the bucket
  int64_t end;         // one past its last element
  int32_t first_tile;  // index of its first tile within the launch
  int32_t S;           // staleness of Eq. (1)
};

// Per-tile side-output partial, reduced per bucket by the last workgroup.
struct TilePartial {
  double grad_sq;
  double delta_sq;
  uint64_t nonfinite;
};

// Kernel arguments, passed by value (about 2.7 KB).
struct StepArgs {
  const float* grads[DASO_MAX_G];
  const uint16_t* stale[DASO_MAX_P];
  const float* src;      // pack: source fp32
  float* x;              // params (merge/fused, in place)
  float* m;              // momentum (fused, in place)
  uint16_t* wire;        // packed output or nullptr
  float* gavg;           // local average output or nullptr
  TilePartial* partials; // per-tile partials (stats only)
  daso_bucket_stats* stats;  // per-bucket outputs (stats only), already offset to this launch
  unsigned int* counter; // finished-workgroup counter (stats only), zero between launches
  int32_t g;
  int32_t P;
  float lr;
  float mu;
  float wd;
  uint32_t flags;
  int32_t nb;            // buckets in this launch
  int32_t ntiles;        // tiles in this launch
  TileBucket b[kLaunchBuckets];
};

// Number of tiles bucket [start, end) is cut into.
inline int64_t tiles_of(int64_t start, int64_t end) {
  if (end <= start) return 0;
  const int64_t a = start & ~int64_t(kVec - 1);
  return (end - a + kTile - 1) / kTile;
}

// Enqueue one launch of `mode` over the buckets in `args` (grid = args.ntiles).
hipError_t launch_step(Mode mode, bool with_stats, const StepArgs& args, hipStream_t stream);

}  // namespace daso
