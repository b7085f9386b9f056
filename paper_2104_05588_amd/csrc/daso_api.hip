// C-ABI entry points of the DASO synchronisation library: argument checks,
// bucket tables, the per-stream statistics workspace, and launches.
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <utility>
#include <vector>

#include "daso_launch.h"

namespace {

using daso::StepArgs;
using daso::TileBucket;
using daso::TilePartial;

constexpr int32_t kMaxS = 1 << 20;  // 2S and 2S + P stay exact in binary32

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Span {
  uintptr_t lo, hi;  // [lo, hi) in bytes
};

Span span_of(const void* p, int64_t n, size_t esz) {
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p);
  return {lo, lo + static_cast<uintptr_t>(n) * esz};
}

bool overlaps(Span a, Span b) { return a.lo < b.hi && b.lo < a.hi; }

// Buckets must tile [0, n): sorted by start they are back to back.
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
    if (e.first != pos) return DASO_EINVAL;
    pos += e.second;
  }
  return pos == n ? DASO_OK : DASO_EINVAL;
}

// ---------------------------------------------------------------- workspace
// Per (device, stream): the per-tile statistics partials of a fused launch.
// Allocated on first use and replaced by one at least twice as large when a
// larger launch needs it.  A replaced buffer is never freed: launches already
// queued, and graphs captured earlier, may still use it; the doubling keeps the
// total within twice the largest buffer.  Every launch writes each partial it
// later reads, so the contents never need clearing.
struct Workspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};

std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;

int workspace_for(hipStream_t stream, size_t need, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return DASO_EHIP;
  std::lock_guard<std::mutex> lock(g_ws_mu);
  Workspace& w = g_ws[{dev, stream}];
  if (w.bytes < need) {
    const size_t bytes = std::max<size_t>({need, 2 * w.bytes, size_t(1) << 20});
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return DASO_EHIP;
    w.ptr = p;  // the previous buffer, if any, stays allocated (see above)
    w.bytes = bytes;
  }
  *out = w.ptr;
  return DASO_OK;
}

// -------------------------------------------------------------- launching
struct Group {
  int32_t first;  // index of its first bucket in the caller's table
  int32_t count;
  int64_t ntiles;
};

// Cut the caller's bucket table into launches of at most kLaunchBuckets buckets.
std::vector<Group> group_buckets(const daso_bucket* b, int32_t nb) {
  std::vector<Group> out;
  for (int32_t i = 0; i < nb; i += daso::kLaunchBuckets) {
    Group gr{i, std::min<int32_t>(daso::kLaunchBuckets, nb - i), 0};
    for (int32_t k = 0; k < gr.count; ++k)
      gr.ntiles += daso::tiles_of(b[i + k].start, b[i + k].start + b[i + k].numel);
    out.push_back(gr);
  }
  return out;
}

void fill_group(StepArgs& a, const daso_bucket* b, const Group& gr) {
  int64_t t = 0;
  for (int32_t k = 0; k < gr.count; ++k) {
    const daso_bucket& s = b[gr.first + k];
    a.b[k].start = s.start;
    a.b[k].end = s.start + s.numel;
    a.b[k].first_tile = static_cast<int32_t>(t);
    a.b[k].S = s.S;
    t += daso::tiles_of(s.start, s.start + s.numel);
  }
  a.nb = gr.count;
  // A launch needs at least one workgroup, even over empty buckets, so that
  // their statistics are still written (as zeros).
  a.ntiles = static_cast<int32_t>(std::max<int64_t>(t, 1));
}

// Compute units of the current device (cached per device).
int compute_units() {
  static std::mutex mu;
  static std::map<int, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) n = 0;
  cache[dev] = n;
  return n;
}

// Workgroups for a launch of `ntiles` tiles: one per tile, or a fixed number
// per compute unit that take the tiles in turn.
int grid_for(int32_t ntiles) {
  if (daso::kBlocksPerCU <= 0) return ntiles;
  const int cus = compute_units();
  if (cus <= 0) return ntiles;
  return static_cast<int>(std::min<int64_t>(ntiles, int64_t(cus) * daso::kBlocksPerCU));
}

int run_groups(daso::Mode mode, StepArgs& a, const daso_bucket* b, int32_t nb,
               daso_bucket_stats* stats, hipStream_t stream) {
  const std::vector<Group> groups = group_buckets(b, nb);
  int64_t max_tiles = 1;
  for (const auto& gr : groups) {
    if (gr.ntiles > INT32_MAX) return DASO_EINVAL;
    max_tiles = std::max(max_tiles, gr.ntiles);
  }
  const bool with_stats = (mode == daso::kModeFused) && stats != nullptr;
  int streams = 2;
  if (mode == daso::kModeAvg) streams = a.g + 1;
  if (mode == daso::kModeMerge) streams = a.P + 2 + (a.wire ? 1 : 0);
  if (mode == daso::kModeFused) streams = a.g + a.P + 4 + (a.wire ? 1 : 0) + (a.gavg ? 1 : 0);
  a.xcd_order = streams >= daso::kXcdOrderMinStreams ? 1 : 0;
  if (with_stats) {
    void* ws = nullptr;
    const int rc = workspace_for(stream, static_cast<size_t>(max_tiles) * sizeof(TilePartial), &ws);
    if (rc != DASO_OK) return rc;
    a.partials = static_cast<TilePartial*>(ws);
  }
  for (const auto& gr : groups) {
    fill_group(a, b, gr);
    a.stats = with_stats ? stats + gr.first : nullptr;
    if (daso::launch_step(mode, with_stats, a, grid_for(a.ntiles), stream) != hipSuccess) return DASO_EHIP;
  }
  return DASO_OK;
}

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

extern "C" {

int daso_abi_version(void) { return 100; }

int32_t daso_plan_buckets(const int64_t* numels, int32_t ntensors, int64_t cap_elems, const int32_t* S_cycle,
                          int32_t n_cycle, daso_bucket* out, int32_t out_cap) {
  if (ntensors < 0 || cap_elems < 1 || n_cycle < 1 || S_cycle == nullptr || out_cap < 0) return DASO_EINVAL;
  if (ntensors > 0 && numels == nullptr) return DASO_EINVAL;
  if (out_cap > 0 && out == nullptr) return DASO_EINVAL;
  for (int32_t c = 0; c < n_cycle; ++c)
    if (S_cycle[c] < 0 || S_cycle[c] > kMaxS) return DASO_EINVAL;
  int64_t end = 0;
  for (int32_t i = 0; i < ntensors; ++i) {
    if (numels[i] < 0) return DASO_EINVAL;
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
    case DASO_EINVAL: return "DASO_EINVAL: invalid argument (null pointer, count out of range, S < 0, or buckets not tiling [0, n))";
    case DASO_EALIGN: return "DASO_EALIGN: a device buffer is not 16-byte aligned";
    case DASO_EALIAS: return "DASO_EALIAS: an output buffer overlaps another buffer";
    case DASO_EHIP: return "DASO_EHIP: a HIP call failed";
    default: return "unknown DASO status";
  }
}

int daso_local_avg(const float* const* grads, int32_t g, float* out, int64_t n, hipStream_t stream) {
  if (n < 0 || g < 1 || g > DASO_MAX_G) return DASO_EINVAL;
  if (n == 0) return DASO_OK;
  int rc = check_ptr_table(reinterpret_cast<const void* const*>(grads), g);
  if (rc != DASO_OK) return rc;
  if ((rc = check_out(out)) != DASO_OK) return rc;
  const Span so = span_of(out, n, 4);
  for (int32_t r = 0; r < g; ++r)
    if (grads[r] != out && overlaps(so, span_of(grads[r], n, 4))) return DASO_EALIAS;

  StepArgs a;
  memset(&a, 0, sizeof(a));
  for (int32_t r = 0; r < g; ++r) a.grads[r] = grads[r];
  a.g = g;
  a.gavg = out;
  const daso_bucket whole = {0, n, 0, 0};
  return run_groups(daso::kModeAvg, a, &whole, 1, nullptr, stream);
}

int daso_pack_bf16(const float* src, uint16_t* wire, int64_t n, hipStream_t stream) {
  if (n < 0) return DASO_EINVAL;
  if (n == 0) return DASO_OK;
  int rc = check_out(src);
  if (rc != DASO_OK) return rc;
  if ((rc = check_out(wire)) != DASO_OK) return rc;
  if (overlaps(span_of(src, n, 4), span_of(wire, n, 2))) return DASO_EALIAS;

  StepArgs a;
  memset(&a, 0, sizeof(a));
  a.src = src;
  a.wire = wire;
  const daso_bucket whole = {0, n, 0, 0};
  return run_groups(daso::kModePack, a, &whole, 1, nullptr, stream);
}

}  // extern "C"

namespace {

// Eq. (1) merge with copies and wire of `esz` bytes per element (2: bf16, 4: fp32).
int merge_impl(float* params, const void* const* stale, int32_t P, const daso_bucket* buckets, int32_t nbuckets,
               void* wire, int64_t n, size_t esz, hipStream_t stream) {
  if (n < 0 || P < 0 || P > DASO_MAX_P) return DASO_EINVAL;
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

  StepArgs a;
  memset(&a, 0, sizeof(a));
  for (int32_t i = 0; i < P; ++i) a.stale[i] = stale[i];
  a.P = P;
  a.x = params;
  a.wire = wire;
  a.xf32 = esz == 4 ? 1 : 0;
  return run_groups(daso::kModeMerge, a, buckets, nbuckets, nullptr, stream);
}

}  // namespace

extern "C" {

int daso_global_merge(float* params, const uint16_t* const* stale, int32_t P, const daso_bucket* buckets,
                      int32_t nbuckets, uint16_t* wire, int64_t n, hipStream_t stream) {
  return merge_impl(params, reinterpret_cast<const void* const*>(stale), P, buckets, nbuckets, wire, n, 2, stream);
}

int daso_global_merge_f32(float* params, const float* const* stale, int32_t P, const daso_bucket* buckets,
                          int32_t nbuckets, float* wire, int64_t n, hipStream_t stream) {
  return merge_impl(params, reinterpret_cast<const void* const*>(stale), P, buckets, nbuckets, wire, n, 4, stream);
}

int daso_fused_sync_step(const daso_sync_args* args, hipStream_t stream) {
  if (args == nullptr) return DASO_EINVAL;
  const daso_sync_args& s = *args;
  if (s.n < 0 || s.g < 1 || s.g > DASO_MAX_G || s.P < 0 || s.P > DASO_MAX_P) return DASO_EINVAL;
  if ((s.flags & ~(DASO_PACK_PRE_MERGE | DASO_EXCHANGE_F32)) != 0) return DASO_EINVAL;
  const bool xf32 = (s.flags & DASO_EXCHANGE_F32) != 0;
  // the exchanged copies and the wire, in the exchange type
  const void* const* stale = xf32 ? reinterpret_cast<const void* const*>(s.stale_f32)
                                  : reinterpret_cast<const void* const*>(s.stale);
  void* wire = xf32 ? static_cast<void*>(s.wire_f32) : static_cast<void*>(s.wire);
  const size_t esz = xf32 ? 4 : 2;
  if (xf32 ? (s.stale != nullptr || s.wire != nullptr) : (s.stale_f32 != nullptr || s.wire_f32 != nullptr))
    return DASO_EINVAL;
  if (s.n == 0) return DASO_OK;
  int rc = check_ptr_table(reinterpret_cast<const void* const*>(s.grads), s.g);
  if (rc != DASO_OK) return rc;
  if ((rc = check_ptr_table(stale, s.P)) != DASO_OK) return rc;
  if ((rc = check_out(s.params)) != DASO_OK) return rc;
  if ((rc = check_out(s.momentum)) != DASO_OK) return rc;
  if (wire && !aligned16(wire)) return DASO_EALIGN;
  if (s.grad_avg && !aligned16(s.grad_avg)) return DASO_EALIGN;
  if (s.stats && (reinterpret_cast<uintptr_t>(s.stats) & 7u) != 0) return DASO_EALIGN;
  if ((rc = check_buckets(s.buckets, s.nbuckets, s.n)) != DASO_OK) return rc;

  // outputs: params and momentum (in place), wire, grad_avg, stats
  const Span sx = span_of(s.params, s.n, 4);
  const Span sm = span_of(s.momentum, s.n, 4);
  std::vector<Span> inputs;
  for (int32_t r = 0; r < s.g; ++r) inputs.push_back(span_of(s.grads[r], s.n, 4));
  for (int32_t i = 0; i < s.P; ++i) inputs.push_back(span_of(stale[i], s.n, esz));
  std::vector<Span> outs = {sx, sm};
  if (wire) outs.push_back(span_of(wire, s.n, esz));
  if (s.stats) outs.push_back(span_of(s.stats, s.nbuckets, sizeof(daso_bucket_stats)));
  for (size_t i = 0; i < outs.size(); ++i) {
    for (size_t j = i + 1; j < outs.size(); ++j)
      if (overlaps(outs[i], outs[j])) return DASO_EALIAS;
    for (const Span& in : inputs)
      if (overlaps(outs[i], in)) return DASO_EALIAS;
  }
  if (s.grad_avg) {
    const Span sg = span_of(s.grad_avg, s.n, 4);
    for (const Span& o : outs)
      if (overlaps(sg, o)) return DASO_EALIAS;
    for (int32_t i = 0; i < s.P; ++i)
      if (overlaps(sg, inputs[static_cast<size_t>(s.g + i)])) return DASO_EALIAS;
    for (int32_t r = 0; r < s.g; ++r)
      if (s.grads[r] != s.grad_avg && overlaps(sg, inputs[static_cast<size_t>(r)])) return DASO_EALIAS;
  }

  StepArgs a;
  memset(&a, 0, sizeof(a));
  for (int32_t r = 0; r < s.g; ++r) a.grads[r] = s.grads[r];
  for (int32_t i = 0; i < s.P; ++i) a.stale[i] = stale[i];
  a.g = s.g;
  a.P = s.P;
  a.x = s.params;
  a.m = s.momentum;
  a.wire = wire;
  a.xf32 = xf32 ? 1 : 0;
  a.gavg = s.grad_avg;
  a.lr = s.lr;
  a.mu = s.mu;
  a.wd = s.weight_decay;
  a.flags = s.flags;
  return run_groups(daso::kModeFused, a, s.buckets, s.nbuckets, s.stats, stream);
}

}  // extern "C"
