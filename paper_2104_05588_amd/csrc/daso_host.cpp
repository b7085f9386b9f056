// Host-only parts of the C ABI: argument checks, the bucket planner, status
// strings.  No HIP calls.
#include "daso_host.h"

#include <algorithm>
#include <utility>
#include <vector>

namespace daso {
namespace host {
namespace {

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Span {
  uintptr_t lo, hi;  // [lo, hi) in bytes
};

Span span_of(const void* p, int64_t n, size_t esz) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return {lo, lo + static_cast<uintptr_t>(n) * esz};
}

bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

int check_ptr_table(const void* const* p, int32_t count) {
  if (count > 0 && p == nullptr) return DASO_EINVAL;
  for (int32_t i = 0; i < count; ++i) {
    if (p[i] == nullptr) return DASO_EINVAL;
    if (!aligned16(p[i])) return DASO_EALIGN;
  }
  return DASO_OK;
}

int check_out(const void* p) {
  if (p == nullptr) return DASO_EINVAL;
  return aligned16(p) ? DASO_OK : DASO_EALIGN;
}

}  // namespace

int check_buckets(const daso_bucket* b, int32_t nb, int64_t n) {
  if (nb < 1 || b == nullptr) return DASO_EINVAL;
  std::vector<std::pair<int64_t, int64_t>> s;
  s.reserve(static_cast<size_t>(nb));
  for (int32_t i = 0; i < nb; ++i) {
    if (b[i].numel < 0 || b[i].start < 0 || b[i].S < 0 || b[i].S > kMaxS || b[i].reserved != 0)
      return DASO_EINVAL;
    s.emplace_back(b[i].start, b[i].numel);
  }
  std::sort(s.begin(), s.end());
  int64_t pos = 0;
  for (const auto& e : s) {
    if (e.first != pos || e.second > INT64_MAX - pos) return DASO_EINVAL;
    pos += e.second;
  }
  return pos == n ? DASO_OK : DASO_EINVAL;
}

int check_local_avg(const float* const* grads, int32_t g, const float* out, int64_t n) {
  if (n < 0 || n > DASO_MAX_N || g < 1 || g > DASO_MAX_G) return DASO_EINVAL;
  if (n == 0) return DASO_OK;
  int rc = check_ptr_table(reinterpret_cast<const void* const*>(grads), g);
  if (rc != DASO_OK) return rc;
  if ((rc = check_out(out)) != DASO_OK) return rc;
  const Span so = span_of(out, n, 4);
  for (int32_t r = 0; r < g; ++r)
    if (grads[r] != out && overlaps(so, span_of(grads[r], n, 4))) return DASO_EALIAS;
  return DASO_OK;
}

int check_pack(const float* src, const uint16_t* wire, int64_t n) {
  if (n < 0 || n > DASO_MAX_N) return DASO_EINVAL;
  if (n == 0) return DASO_OK;
  int rc = check_out(src);
  if (rc != DASO_OK) return rc;
  if ((rc = check_out(wire)) != DASO_OK) return rc;
  return overlaps(span_of(src, n, 4), span_of(wire, n, 2)) ? DASO_EALIAS : DASO_OK;
}

int check_merge(const float* params, const void* const* stale, int32_t P, const daso_bucket* buckets,
                int32_t nbuckets, const void* wire, int64_t n, size_t esz) {
  if (n < 0 || n > DASO_MAX_N || P < 0 || P > DASO_MAX_P) return DASO_EINVAL;
  if (n == 0) return DASO_OK;
  int rc = check_out(params);
  if (rc != DASO_OK) return rc;
  if ((rc = check_ptr_table(stale, P)) != DASO_OK) return rc;
  if (wire && !aligned16(wire)) return DASO_EALIGN;
  if ((rc = check_buckets(buckets, nbuckets, n)) != DASO_OK) return rc;
  const Span sx = span_of(params, n, 4);
  for (int32_t i = 0; i < P; ++i)
    if (overlaps(sx, span_of(stale[i], n, esz))) return DASO_EALIAS;
  if (wire) {
    const Span sw = span_of(wire, n, esz);
    if (overlaps(sw, sx)) return DASO_EALIAS;
    for (int32_t i = 0; i < P; ++i)
      if (overlaps(sw, span_of(stale[i], n, esz))) return DASO_EALIAS;
  }
  return DASO_OK;
}

int check_fused(const daso_sync_args& s, FusedView* view) {
  if (s.n < 0 || s.n > DASO_MAX_N || s.g < 1 || s.g > DASO_MAX_G || s.P < 0 || s.P > DASO_MAX_P) return DASO_EINVAL;
  if ((s.flags & ~(DASO_PACK_PRE_MERGE | DASO_EXCHANGE_F32)) != 0) return DASO_EINVAL;
  const bool xf32 = (s.flags & DASO_EXCHANGE_F32) != 0;
  // the exchanged copies and the wire, in the exchange type
  FusedView v;
  v.xf32 = xf32;
  v.stale = xf32 ? reinterpret_cast<const void* const*>(s.stale_f32) : reinterpret_cast<const void* const*>(s.stale);
  v.wire = xf32 ? static_cast<void*>(s.wire_f32) : static_cast<void*>(s.wire);
  v.esz = xf32 ? 4 : 2;
  if (xf32 ? (s.stale != nullptr || s.wire != nullptr) : (s.stale_f32 != nullptr || s.wire_f32 != nullptr))
    return DASO_EINVAL;
  *view = v;
  if (s.n == 0) return DASO_OK;
  int rc = check_ptr_table(reinterpret_cast<const void* const*>(s.grads), s.g);
  if (rc != DASO_OK) return rc;
  if ((rc = check_ptr_table(v.stale, s.P)) != DASO_OK) return rc;
  if ((rc = check_out(s.params)) != DASO_OK) return rc;
  if ((rc = check_out(s.momentum)) != DASO_OK) return rc;
  if (v.wire && !aligned16(v.wire)) return DASO_EALIGN;
  if (s.grad_avg && !aligned16(s.grad_avg)) return DASO_EALIGN;
  if (s.stats && (reinterpret_cast<uintptr_t>(s.stats) & 7u) != 0) return DASO_EALIGN;
  if ((rc = check_buckets(s.buckets, s.nbuckets, s.n)) != DASO_OK) return rc;

  // outputs: params and momentum (in place), wire, stats, grad_avg
  std::vector<Span> inputs;
  for (int32_t r = 0; r < s.g; ++r) inputs.push_back(span_of(s.grads[r], s.n, 4));
  for (int32_t i = 0; i < s.P; ++i) inputs.push_back(span_of(v.stale[i], s.n, v.esz));
  std::vector<Span> outs = {span_of(s.params, s.n, 4), span_of(s.momentum, s.n, 4)};
  if (v.wire) outs.push_back(span_of(v.wire, s.n, v.esz));
  if (s.stats) outs.push_back(span_of(s.stats, s.nbuckets, sizeof(daso_bucket_stats)));
  for (size_t i = 0; i < outs.size(); ++i) {
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (overlaps(outs[i], outs[j])) return DASO_EALIAS;
    for (const Span& in : inputs)
      if (overlaps(outs[i], in)) return DASO_EALIAS;
  }
  if (s.grad_avg) {
    // may be exactly one of the gradient buffers, and nothing else
    const Span sg = span_of(s.grad_avg, s.n, 4);
    for (const Span& o : outs)
      if (overlaps(sg, o)) return DASO_EALIAS;
    for (int32_t i = 0; i < s.P; ++i)
      if (overlaps(sg, inputs[static_cast<size_t>(s.g + i)])) return DASO_EALIAS;
    for (int32_t r = 0; r < s.g; ++r)
      if (s.grads[r] != s.grad_avg && overlaps(sg, inputs[static_cast<size_t>(r)])) return DASO_EALIAS;
  }
  return DASO_OK;
}

int64_t launch_grid(int64_t ntiles, int32_t run) {
  if (ntiles < 1) return 1;
  if (ntiles <= kMaxGrid) return ntiles;
  const int64_t block = 8 * static_cast<int64_t>(run < 1 ? 1 : run);
  const int64_t whole = (kMaxGrid / block) * block;
  return whole > 0 ? whole : kMaxGrid;
}

}  // namespace host
}  // namespace daso

extern "C" {

int daso_abi_version(void) { return 102; }

int32_t daso_plan_buckets(const int64_t* numels, int32_t ntensors, int64_t cap_elems, const int32_t* S_cycle,
                          int32_t n_cycle, daso_bucket* out, int32_t out_cap) {
  using daso::host::kMaxS;
  if (ntensors < 0 || cap_elems < 1 || n_cycle < 1 || S_cycle == nullptr || out_cap < 0) return DASO_EINVAL;
  if (ntensors > 0 && numels == nullptr) return DASO_EINVAL;
  if (out_cap > 0 && out == nullptr) return DASO_EINVAL;
  for (int32_t c = 0; c < n_cycle; ++c)
    if (S_cycle[c] < 0 || S_cycle[c] > kMaxS) return DASO_EINVAL;
  int64_t end = 0;
  for (int32_t i = 0; i < ntensors; ++i) {
    if (numels[i] < 0 || numels[i] > INT64_MAX - end) return DASO_EINVAL;
    end += numels[i];
  }
  int32_t count = 0;
  auto emit = [&](int64_t start, int64_t numel) {
    if (count < out_cap) out[count] = daso_bucket{start, numel, S_cycle[count % n_cycle], 0};
    ++count;
  };
  int64_t size = 0;
  for (int32_t i = ntensors - 1; i >= 0; --i) {
    size += numels[i];
    if (size >= cap_elems) {
      emit(end - size, size);
      end -= size;
      size = 0;
    }
  }
  if (size > 0) emit(0, size);
  return count;
}

const char* daso_status_string(int status) {
  switch (status) {
    case DASO_OK: return "DASO_OK: success";
    case DASO_EINVAL:
      return "DASO_EINVAL: invalid argument (null pointer, count out of range, S outside [0, DASO_MAX_S], buckets not tiling [0, n), or a stream of another device)";
    case DASO_EALIGN: return "DASO_EALIGN: a device buffer is not 16-byte aligned";
    case DASO_EALIAS: return "DASO_EALIAS: an output buffer overlaps another buffer";
    case DASO_EHIP: return "DASO_EHIP: a HIP call failed";
    case DASO_ENOSPACE:
      return "DASO_ENOSPACE: the statistics need more scratch than the fixed array of "
             "daso_fused_sync_step_noalloc holds (DASO_NOALLOC_SCRATCH_BYTES: 24 bytes per tile plus 260)";
    default: return "unknown DASO status";
  }
}

}  // extern "C"
