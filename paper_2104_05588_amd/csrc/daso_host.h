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

// Each returns DASO_OK or the status the entry point must return; n == 0 is
// DASO_OK once the counts are valid (the caller then launches nothing).
int check_local_avg(const float* const* grads, int32_t g, const float* out, int64_t n);
int check_pack(const float* src, const uint16_t* wire, int64_t n);
int check_merge(const float* params, const void* const* stale, int32_t P, const daso_bucket* buckets,
                int32_t nbuckets, const void* wire, int64_t n, size_t esz);
int check_fused(const daso_sync_args& s, FusedView* view);

}  // namespace host
}  // namespace daso
