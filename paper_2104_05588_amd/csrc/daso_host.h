// Host-only argument checking of the C ABI (no HIP calls).  Compiled into the
// library and, for the sanitizer tests, on its own with the host compiler.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "daso.h"

namespace daso {
namespace host {

constexpr int32_t kMaxS = DASO_MAX_S;  // 2S and 2S + P stay exact in binary32

// Buckets must tile [0, n): sorted by start they lie back to back; S in [0, kMaxS].
int check_buckets(const daso_bucket* b, int32_t nb, int64_t n);

// A checked fused step: the exchanged copies and the wire resolved to the
// exchange type (esz = 2 for bf16, 4 for fp32).
struct FusedView {
  const void* const* stale;
  void* wire;
  size_t esz;
  bool xf32;
};

// Workgroups of a launch over `ntiles` tiles (one 256-thread workgroup per
// tile) whose XCD runs are `run` tiles long: one per tile up to kMaxGrid, the
// largest multiple of the run block (8 * run) within kMaxGrid beyond that, the
// kernel looping over the remaining tiles.  The dispatch packet counts the grid
// in work-items in 32 bits, so a grid of 256-thread workgroups must stay below
// 2^24; kMaxGrid (4096 workgroups per CU) is far above what fills the chip.
constexpr int64_t kMaxGrid = int64_t(1) << 20;
int64_t launch_grid(int64_t ntiles, int32_t run);

// Each returns DASO_OK or the status the entry point must return; n == 0 is
// DASO_OK once the counts are valid (the caller then launches nothing).
int check_local_avg(const float* const* grads, int32_t g, const float* out, int64_t n);
int check_pack(const float* src, const uint16_t* wire, int64_t n);
int check_merge(const float* params, const void* const* stale, int32_t P, const daso_bucket* buckets,
                int32_t nbuckets, const void* wire, int64_t n, size_t esz);
int check_fused(const daso_sync_args& s, FusedView* view);

}  // namespace host
}  // namespace daso
