// C-ABI entry points of the DASO synchronisation library that touch the GPU:
// the per-stream statistics workspace, bucket grouping and launches.  Argument
// checking is in daso_host.cpp.
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <map>
#include <mutex>
#include <utility>

#include "daso_host.h"
#include "daso_launch.h"

namespace {

// Kernel arguments are passed by value and limited to 4 KB.
static_assert(sizeof(daso::StepArgs) <= 4096, "StepArgs must fit the 4 KB kernel-argument limit");

using daso::StepArgs;
using daso::TileBucket;
using daso::TilePartial;

// ---------------------------------------------------------------- workspace
// Per (device, stream): the counter of launches that sum their own statistics
// (kStatsCounterBytes), the per-tile statistics partials of a fused launch and
// the launch's table of bucket tile ranges.  Allocated on first use and
// replaced by one at least twice as large when a larger launch needs it.  A
// replaced buffer is never freed: launches already queued, and graphs captured
// earlier, may still use it; the doubling keeps the total within twice the
// largest buffer.  The counter is zeroed once, by a kernel that the first
// eager (not captured) call needing it queues on the stream, and every launch
// that uses it leaves it at zero; every launch writes each partial and table
// entry it later reads, so the rest never needs clearing.  A call holds the
// entry's lock
// from choosing the buffer until its last launch is queued, so that two host
// threads sharing a stream cannot queue one call's step between the other
// call's step and its statistics pass.
struct Workspace {
  std::mutex mu;
  void* ptr = nullptr;
  size_t bytes = 0;
  bool counter_zeroed = false;  // the zeroing of ptr's counter is queued on the stream
};

std::mutex g_ws_mu;  // guards the map itself; nodes never move or go away
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;

Workspace& workspace_entry(int dev, hipStream_t stream) {
  std::lock_guard<std::mutex> lock(g_ws_mu);
  return g_ws[{dev, stream}];
}

// With w.mu held: make w hold at least `need` bytes.
int reserve(Workspace& w, size_t need) {
  if (w.bytes < need) {
    const size_t bytes = std::max<size_t>({need, 2 * w.bytes, size_t(1) << 20});
    void* p = nullptr;
    if (hipMalloc(&p, bytes) != hipSuccess) return DASO_EHIP;
    w.ptr = p;  // the previous buffer, if any, stays allocated (see above)
    w.bytes = bytes;
    w.counter_zeroed = false;
  }
  return DASO_OK;
}

// With w.mu held, from an eager call: queue the zeroing of w's counter on
// `stream` once per buffer, before any launch that uses it.
int zero_counter_once(Workspace& w, hipStream_t stream) {
  if (w.counter_zeroed) return DASO_OK;
  if (daso::clear_stats_counter(w.ptr, stream) != hipSuccess) return DASO_EHIP;
  w.counter_zeroed = true;
  return DASO_OK;
}

// ---------------------------------------------------------- fixed scratch
// The statistics scratch of daso_fused_sync_step_noalloc: one array of fixed
// size in device memory, of which every GPU the library runs on holds its own
// copy until the process ends.  In host code `scratch` names a host-side stand-in,
// not device memory: the device address is looked up once per device with
// hipGetSymbolAddress (with that device current) and only that address is
// handed to kernels.  It has the workspace's layout, but its first
// kStatsCounterBytes are never used: calls through it keep the statistics
// kernel (see run_groups).  The kernels write every partial and table entry
// they read later, so the array never needs clearing.
constexpr size_t kScratchBytes = DASO_NOALLOC_SCRATCH_BYTES;
static_assert(kScratchBytes % 256 == 0, "the scratch size is a whole number of 256-byte blocks");
static_assert(daso::kStatsCounterBytes % 256 == 0, "the partials start on a 256-byte boundary");
static __device__ __align__(256) uint64_t scratch[kScratchBytes / sizeof(uint64_t)];

constexpr int kMaxDevices = 64;

struct ScratchSlot {
  std::once_flag once;
  hipError_t err = hipSuccess;
  void* ptr = nullptr;
  std::mutex mu;  // held by a call from choosing the buffer until its last launch is queued
};
ScratchSlot g_scratch[kMaxDevices];

// The device address of `scratch` on device `dev`, which must be current.
int scratch_slot(int dev, ScratchSlot** out) {
  if (dev < 0 || dev >= kMaxDevices) return DASO_EHIP;
  ScratchSlot& s = g_scratch[dev];
  std::call_once(s.once, [&s] { s.err = hipGetSymbolAddress(&s.ptr, HIP_SYMBOL(scratch)); });
  if (s.err != hipSuccess || s.ptr == nullptr) return DASO_EHIP;
  *out = &s;
  return DASO_OK;
}

// -------------------------------------------------------------- launching
struct Group {
  int32_t first;  // index of its first bucket in the caller's table
  int32_t count;
  int64_t ntiles;
};

// The caller's bucket table is cut into launches of at most kLaunchBuckets
// buckets; group(i) is the launch starting at bucket i (no allocation).
Group group_at(const daso_bucket* b, int32_t nb, int32_t i, int64_t tile) {
  Group gr{i, std::min<int32_t>(daso::kLaunchBuckets, nb - i), 0};
  for (int32_t k = 0; k < gr.count; ++k)
    gr.ntiles += daso::tiles_of(b[i + k].start, b[i + k].start + b[i + k].numel, tile);
  return gr;
}

void fill_group(StepArgs& a, const daso_bucket* b, const Group& gr, int64_t tile) {
  int64_t t = 0;
  for (int32_t k = 0; k < gr.count; ++k) {
    const daso_bucket& s = b[gr.first + k];
    a.b[k].start = s.start;
    a.b[k].end = s.start + s.numel;
    a.b[k].first_tile = static_cast<int32_t>(t);
    a.b[k].S = s.S;
    t += daso::tiles_of(s.start, s.start + s.numel, tile);
  }
  a.nb = gr.count;
  // A launch needs at least one workgroup, even over empty buckets, so that
  // their statistics are still written (as zeros).
  a.ntiles = static_cast<int32_t>(std::max<int64_t>(t, 1));
}

// A non-negative integer from the environment, read once per variable by the
// caller's static; `fallback` when unset, malformed or above `max`.
int64_t env_count(const char* name, int64_t fallback, int64_t max) {
  const char* e = getenv(name);
  if (e == nullptr || *e == '\0') return fallback;
  char* end = nullptr;
  const long long x = strtoll(e, &end, 10);
  return (end != e && *end == '\0' && x >= 0 && x <= max) ? static_cast<int64_t>(x) : fallback;
}

// DASO_FUSED_RUN_ELEMS, when set to a number of elements, replaces the run
// length of fused launches of kXcdRunFusedStreams streams or more (0: plain
// order); DASO_FUSED_WG_PER_CU, when set, replaces the workgroups-per-CU cap of
// fused launches of kCapStreams streams or more (0: no cap).  Neither ever
// changes a result; they exist to reproduce the measurements behind the
// defaults.  Each is read once per process.
int64_t fused_run_elems_override() {
  static const int64_t v = env_count("DASO_FUSED_RUN_ELEMS", -1, int64_t(1) << 30);
  return v;
}
int64_t fused_cap_override() {
  static const int64_t v = env_count("DASO_FUSED_WG_PER_CU", -1, 64);
  return v;
}

// Streams a launch touches (the tile-order and occupancy rules go by it).
int launch_streams(daso::Mode mode, const StepArgs& a) {
  if (mode == daso::kModeAvg) return a.g + 1;
  if (mode == daso::kModeMerge) return a.P + 2 + (a.wire ? 1 : 0);
  if (mode == daso::kModeFused) return a.g + a.P + 4 + (a.wire ? 1 : 0) + (a.gavg ? 1 : 0);
  return 2;
}

// Tiles per XCD run of one launch of `ntiles` tiles of `tile` elements (the
// rule and its measurements are stated with the constants in daso_launch.h).
int32_t xcd_run_of(daso::Mode mode, int streams, int64_t ntiles, int64_t tile) {
  if (mode == daso::kModeFused && streams >= daso::kXcdRunFusedStreams) {
    const int64_t over = fused_run_elems_override();
    if (over >= 0) return static_cast<int32_t>(std::max<int64_t>(1, over / tile));
    int64_t run = 1;
    while (run * 2 <= ntiles / (8 * daso::kXcdRunBlocksPerLaunch) && run < (int64_t(1) << 20)) run *= 2;
    return static_cast<int32_t>(run);
  }
  if (streams >= daso::kXcdRunManyStreams) return daso::kXcdRunMany;
  if (streams >= daso::kXcdRunMidStreams) return daso::kXcdRunMid;
  return 1;
}

// LDS per workgroup of a launch: the occupancy cap of the fused step.
int32_t lds_of(daso::Mode mode, int streams) {
  if (mode != daso::kModeFused) return 0;
  const int64_t over = fused_cap_override();
  if (over >= 0) return daso::lds_for_workgroups_per_cu(static_cast<int32_t>(over));
  return streams >= daso::kCapStreams ? daso::lds_for_workgroups_per_cu(daso::kCapWorkgroupsPerCU) : 0;
}

// The current device, which must also be the device of `stream` (kernels run
// on the stream's device and the buffers and workspace live on the current one).
int current_device(hipStream_t stream, int* dev) {
  if (hipGetDevice(dev) != hipSuccess) return DASO_EHIP;
  if (stream == nullptr) return DASO_OK;
  hipDevice_t sdev = 0;
  if (hipStreamGetDevice(stream, &sdev) != hipSuccess) return DASO_EHIP;
  return sdev == *dev ? DASO_OK : DASO_EINVAL;
}

// ----------------------------------------------------------- tile-order choice
// The rule's run length is the best measured for most fused shapes, but some
// (the segmentation-shaped step) run 2 to 5% faster in plain order.  For each
// fused launch shape of a single launch, the first call is left out (it can
// carry one-off costs: the first launch of a kernel in a process takes
// milliseconds), then kTuneSamples calls alternate between the rule's run
// length and plain order, each bracketed by two events on the call's stream.
// Once all of them have completed, which later calls poll with hipEventQuery
// (never waiting), plain order is kept for the shape if its fastest sample beat
// the rule's by at least 1%, the rule's runs otherwise; until then calls take
// the rule's run length.
// The order never changes a result.  No sample is taken by a captured call, by
// daso_fused_sync_step_noalloc (it only reads a choice already made), or when
// DASO_FUSED_RUN_ELEMS or DASO_FUSED_TUNE=0 is set.
constexpr int kTuneSkip = 1;                // calls of a shape before sampling starts
constexpr int kTuneSamples = 6;             // rule, plain, rule, plain, rule, plain
constexpr float kTunePlainMargin = 0.99f;   // plain order must be at least 1% faster

bool tuning_enabled() {
  static const bool v = env_count("DASO_FUSED_TUNE", 1, 1) != 0 && fused_run_elems_override() < 0;
  return v;
}

struct TuneKey {
  int dev;
  int32_t g, P, xf32, stats, outputs;
  int64_t n;
  uint64_t layout;  // hash of the bucket table
  bool operator<(const TuneKey& o) const {
    if (dev != o.dev) return dev < o.dev;
    if (g != o.g) return g < o.g;
    if (P != o.P) return P < o.P;
    if (xf32 != o.xf32) return xf32 < o.xf32;
    if (stats != o.stats) return stats < o.stats;
    if (outputs != o.outputs) return outputs < o.outputs;
    if (n != o.n) return n < o.n;
    return layout < o.layout;
  }
};

struct Tune {
  std::mutex mu;
  hipEvent_t ev[kTuneSamples][2] = {};
  int skipped = 0;     // calls left out before the first sample
  int taken = 0;       // samples whose launches are queued
  int32_t chosen = 0;  // tiles per run once decided, 0 before
  bool off = false;    // an event call failed: keep the rule for this shape
};

std::mutex g_tune_mu;  // guards the map itself; nodes never move or go away
std::map<TuneKey, Tune> g_tune;

uint64_t layout_hash(const daso_bucket* b, int32_t nb) {
  uint64_t h = 1469598103934665603ull;  // FNV-1a over the bucket ranges
  auto mix = [&h](uint64_t v) {
    for (int k = 0; k < 8; ++k) {
      h ^= (v >> (8 * k)) & 0xFFu;
      h *= 1099511628211ull;
    }
  };
  for (int32_t i = 0; i < nb; ++i) {
    mix(static_cast<uint64_t>(b[i].start));
    mix(static_cast<uint64_t>(b[i].numel));
  }
  return h;
}

TuneKey tune_key(int dev, const StepArgs& a, bool with_stats, const daso_bucket* b, int32_t nb) {
  int64_t n = 0;  // the buckets tile [0, n)
  for (int32_t i = 0; i < nb; ++i) n += b[i].numel;
  return TuneKey{dev, a.g, a.P, a.xf32, with_stats ? 1 : 0, (a.wire ? 1 : 0) | (a.gavg ? 2 : 0), n,
                 layout_hash(b, nb)};
}

// The decided run length of a shape, or 0.  Never inserts.
int32_t tuned_run(const TuneKey& k) {
  std::lock_guard<std::mutex> lock(g_tune_mu);
  const auto it = g_tune.find(k);
  if (it == g_tune.end()) return 0;
  std::lock_guard<std::mutex> tl(it->second.mu);
  return it->second.chosen;
}

Tune& tune_entry(const TuneKey& k) {
  std::lock_guard<std::mutex> lock(g_tune_mu);
  return g_tune[k];
}

// With t.mu held, after all samples were queued: decide once every sample has
// completed (calls of one shape may sample on different streams, so the last
// queued need not be the last to finish).  The queries run only when no error
// is pending on this thread, and any status they leave is cleared, so a
// caller's error is neither consumed nor masked and none is left behind.
void try_decide(Tune& t, int32_t rule) {
  if (hipPeekAtLastError() != hipSuccess) return;
  for (int k = 0; k < kTuneSamples; ++k) {
    const hipError_t q = hipEventQuery(t.ev[k][1]);
    if (q == hipSuccess) continue;
    if (hipPeekAtLastError() != hipSuccess) (void)hipGetLastError();
    if (q != hipErrorNotReady) t.off = true;
    return;
  }
  float best[2] = {1e30f, 1e30f};
  for (int k = 0; k < kTuneSamples; ++k) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, t.ev[k][0], t.ev[k][1]) != hipSuccess) {
      if (hipPeekAtLastError() != hipSuccess) (void)hipGetLastError();
      t.off = true;
      return;
    }
    best[k % 2] = std::min(best[k % 2], ms);
  }
  // plain order only when it measured clearly faster: the rule's runs are the
  // measured default, and two samples each cannot separate closer orders
  t.chosen = best[1] < kTunePlainMargin * best[0] ? 1 : rule;
  for (auto& e : t.ev) {
    for (hipEvent_t& x : e) {
      if (x) (void)hipEventDestroy(x);
      x = nullptr;
    }
  }
}

// A failed HIP call made only for the sampling gives up sampling for the
// shape; the error it left is dropped when no error was pending before it, so
// that the library never leaves an error of its own behind.
void give_up(Tune& t, bool was_clean) {
  t.off = true;
  if (was_clean && hipPeekAtLastError() != hipSuccess) (void)hipGetLastError();
}

// Where a fused launch with statistics keeps its tile partials and table.
enum class Space {
  kAllocated,  // the per-(device, stream) workspace, allocated on first use
  kFixed,      // the fixed `scratch` array; calls needing more fail with DASO_ENOSPACE
};

int run_groups(daso::Mode mode, StepArgs& a, const daso_bucket* b, int32_t nb,
               daso_bucket_stats* stats, hipStream_t stream, Space space = Space::kAllocated) {
  const bool with_stats = (mode == daso::kModeFused) && stats != nullptr;
  const int64_t tile = daso::tile_elems(mode, with_stats, a);
  int64_t max_tiles = 1;
  for (int32_t i = 0; i < nb; i += daso::kLaunchBuckets) {
    const Group gr = group_at(b, nb, i, tile);
    if (gr.ntiles > INT32_MAX) return DASO_EINVAL;
    max_tiles = std::max(max_tiles, gr.ntiles);
  }
  // statistics scratch: the counter, the tile partials, then the table of bucket tile ranges
  const size_t partials_at = daso::kStatsCounterBytes;
  const size_t table_at = partials_at + static_cast<size_t>(max_tiles) * sizeof(TilePartial);
  const size_t need = table_at + (daso::kLaunchBuckets + 1) * sizeof(int32_t);
  if (with_stats && space == Space::kFixed && need > kScratchBytes) return DASO_ENOSPACE;
  int dev = 0;
  const int drc = current_device(stream, &dev);
  if (drc != DASO_OK) return drc;
  const int streams = launch_streams(mode, a);
  const int32_t lds = lds_of(mode, streams);
  std::unique_lock<std::mutex> hold;
  uint32_t* counter = nullptr;
  bool capturing = true;  // unless the stream is known not to be capturing
  if (with_stats) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusActive;
    capturing = hipStreamIsCapturing(stream, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
    void* base = nullptr;
    if (space == Space::kFixed) {
      ScratchSlot* slot = nullptr;
      const int rc = scratch_slot(dev, &slot);
      if (rc != DASO_OK) return rc;
      hold = std::unique_lock<std::mutex>(slot->mu);
      base = slot->ptr;
    } else {
      Workspace& w = workspace_entry(dev, stream);
      hold = std::unique_lock<std::mutex>(w.mu);
      const int rc = reserve(w, need);
      if (rc != DASO_OK) return rc;
      base = w.ptr;
      // the last-workgroup statistics of small eager launches count in w's counter
      if (!capturing) {
        const int zc = zero_counter_once(w, stream);
        if (zc != DASO_OK) return zc;
        counter = static_cast<uint32_t*>(base);
      }
    }
    a.partials = reinterpret_cast<TilePartial*>(static_cast<char*>(base) + partials_at);
    a.tile_table = reinterpret_cast<int32_t*>(static_cast<char*>(base) + table_at);
  }
  // the tile order of a single fused launch may be chosen per shape (above)
  const bool choosable = mode == daso::kModeFused && streams >= daso::kXcdRunFusedStreams &&
                         nb <= daso::kLaunchBuckets && tuning_enabled();
  for (int32_t i = 0; i < nb; i += daso::kLaunchBuckets) {
    const Group gr = group_at(b, nb, i, tile);
    fill_group(a, b, gr, tile);
    a.stats = with_stats ? stats + gr.first : nullptr;
    // an eager launch of few tiles sums its own statistics in its last
    // workgroup: that saves a launch's host cost (about 2.6 us) for fences that
    // cost the GPU about 0.1 us per workgroup; a graph replays launches without
    // that host cost, so a captured call keeps the statistics kernel (counter
    // stays null), and so does the no-alloc entry point, whose scratch every
    // call on the GPU shares: two of its calls racing on another stream could
    // leave a counter wrong for later calls, not only their own statistics
    a.done = (counter != nullptr && a.ntiles <= daso::kFinishStatsMaxTiles) ? counter : nullptr;
    const int32_t rule = xcd_run_of(mode, streams, a.ntiles, tile);
    a.xcd_run = rule;
    Tune* t = nullptr;
    std::unique_lock<std::mutex> tl;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    bool clean = true;  // no HIP error was pending when sampling started
    if (choosable) {
      const TuneKey key = tune_key(dev, a, with_stats, b, nb);
      if (space == Space::kFixed) {
        const int32_t c = tuned_run(key);
        if (c > 0) a.xcd_run = c;
      } else {
        t = &tune_entry(key);
        tl = std::unique_lock<std::mutex>(t->mu);
        if (t->chosen > 0) {
          a.xcd_run = t->chosen;
        } else if (!t->off && t->skipped < kTuneSkip) {
          ++t->skipped;
        } else if (!t->off && t->taken < kTuneSamples) {
          clean = hipPeekAtLastError() == hipSuccess;
          hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
          if (hipStreamIsCapturing(stream, &cs) != hipSuccess) {
            give_up(*t, clean);
          } else if (cs == hipStreamCaptureStatusNone) {
            hipEvent_t(&ev)[2] = t->ev[t->taken];
            if ((ev[0] || hipEventCreate(&ev[0]) == hipSuccess) && (ev[1] || hipEventCreate(&ev[1]) == hipSuccess)) {
              e0 = ev[0];
              e1 = ev[1];
              a.xcd_run = (t->taken % 2 == 0) ? rule : 1;
            } else {
              give_up(*t, clean);
            }
          }
        } else if (!t->off && t->taken == kTuneSamples) {
          try_decide(*t, rule);
          if (t->chosen > 0) a.xcd_run = t->chosen;
        }
      }
    }
    const int64_t grid = daso::host::launch_grid(a.ntiles, a.xcd_run);
    if (e0 && hipEventRecord(e0, stream) != hipSuccess) {
      give_up(*t, clean);
      e1 = nullptr;
    }
    if (daso::launch_step(mode, with_stats, a, static_cast<uint32_t>(grid), static_cast<uint32_t>(lds), stream) !=
        hipSuccess)
      return DASO_EHIP;
    if (e1) {
      if (hipEventRecord(e1, stream) == hipSuccess) {
        ++t->taken;
      } else {
        give_up(*t, clean);
      }
    }
  }
  return DASO_OK;
}

}  // namespace

extern "C" {

int daso_local_avg(const float* const* grads, int32_t g, float* out, int64_t n, hipStream_t stream) {
  const int rc = daso::host::check_local_avg(grads, g, out, n);
  if (rc != DASO_OK || n == 0) return rc;
  StepArgs a;
  memset(&a, 0, sizeof(a));
  for (int32_t r = 0; r < g; ++r) a.grads[r] = grads[r];
  a.g = g;
  a.gavg = out;
  const daso_bucket whole = {0, n, 0, 0};
  return run_groups(daso::kModeAvg, a, &whole, 1, nullptr, stream);
}

int daso_pack_bf16(const float* src, uint16_t* wire, int64_t n, hipStream_t stream) {
  const int rc = daso::host::check_pack(src, wire, n);
  if (rc != DASO_OK || n == 0) return rc;
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
  const int rc = daso::host::check_merge(params, stale, P, buckets, nbuckets, wire, n, esz);
  if (rc != DASO_OK || n == 0) return rc;
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

}  // extern "C"

namespace {

// Checks a fused call and fills the kernel arguments that do not depend on the
// launch (streams, counts, constants).  With n == 0 only the counts and the
// exchange type are filled: no pointer is looked at.
int fused_args(const daso_sync_args* args, StepArgs& a) {
  if (args == nullptr) return DASO_EINVAL;
  const daso_sync_args& s = *args;
  daso::host::FusedView v;
  const int rc = daso::host::check_fused(s, &v);
  if (rc != DASO_OK) return rc;
  memset(&a, 0, sizeof(a));
  a.g = s.g;
  a.P = s.P;
  a.xf32 = (s.flags & DASO_EXCHANGE_F32) ? 1 : 0;
  if (s.n == 0) return DASO_OK;
  for (int32_t r = 0; r < s.g; ++r) a.grads[r] = s.grads[r];
  for (int32_t i = 0; i < s.P; ++i) a.stale[i] = v.stale[i];
  a.g = s.g;
  a.P = s.P;
  a.x = s.params;
  a.m = s.momentum;
  a.wire = v.wire;
  a.gavg = s.grad_avg;
  a.lr = s.lr;
  a.mu = s.mu;
  a.wd = s.weight_decay;
  a.flags = s.flags;
  return DASO_OK;
}

int fused_impl(const daso_sync_args* args, hipStream_t stream, Space space) {
  StepArgs a;
  const int rc = fused_args(args, a);
  if (rc != DASO_OK || args->n == 0) return rc;
  return run_groups(daso::kModeFused, a, args->buckets, args->nbuckets, args->stats, stream, space);
}

}  // namespace

extern "C" {

int daso_fused_sync_step(const daso_sync_args* args, hipStream_t stream) {
  return fused_impl(args, stream, Space::kAllocated);
}

int daso_fused_sync_step_noalloc(const daso_sync_args* args, hipStream_t stream) {
  return fused_impl(args, stream, Space::kFixed);
}

int daso_fused_launch_config(const daso_sync_args* args, daso_launch_config* out) {
  if (out == nullptr) return DASO_EINVAL;
  StepArgs a;
  const int rc = fused_args(args, a);
  if (rc != DASO_OK) return rc;
  const bool with_stats = args->stats != nullptr;
  const int64_t tile = daso::tile_elems(daso::kModeFused, with_stats, a);
  const int streams = launch_streams(daso::kModeFused, a);
  int64_t ntiles = 0;
  if (args->n > 0)
    for (int32_t k = 0; k < std::min<int32_t>(args->nbuckets, daso::kLaunchBuckets); ++k)
      ntiles += daso::tiles_of(args->buckets[k].start, args->buckets[k].start + args->buckets[k].numel, tile);
  out->tile_elems = tile;
  out->ntiles = ntiles;
  out->xcd_run_tiles = xcd_run_of(daso::kModeFused, streams, std::max<int64_t>(ntiles, 1), tile);
  out->lds_bytes = lds_of(daso::kModeFused, streams);
  // a tile order already chosen for this shape on the current device replaces the rule's
  int dev = 0;
  if (args->n > 0 && streams >= daso::kXcdRunFusedStreams && args->nbuckets <= daso::kLaunchBuckets &&
      tuning_enabled() && hipGetDevice(&dev) == hipSuccess) {
    const int32_t c = tuned_run(tune_key(dev, a, with_stats, args->buckets, args->nbuckets));
    if (c > 0) out->xcd_run_tiles = c;
  }
  return DASO_OK;
}

}  // extern "C"
