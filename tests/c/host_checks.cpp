// Exercises the library's host-only code (argument checks, bucket planner,
// schedule controller) under AddressSanitizer and UndefinedBehaviorSanitizer.
// Built with the host compiler alone; fake device addresses are never
// dereferenced.  Exit status 0 when every expectation holds.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <random>
#include <vector>

#include "daso.h"
#include "daso_host.h"

static int failures = 0;
#define EXPECT(cond)                                                     \
  do {                                                                   \
    if (!(cond)) {                                                       \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__,  \
                   __LINE__, #cond);                                     \
      ++failures;                                                        \
    }                                                                    \
  } while (0)

// Reference for a bucket table tiling [0, n) (small n): every element covered
// exactly once, and an empty bucket only where a bucket starts or ends (0, n,
// or a boundary of a non-empty bucket), never strictly inside one.
static bool tiles(const std::vector<daso_bucket>& b, int64_t n) {
  std::vector<int> cover(static_cast<size_t>(n), 0);
  std::vector<bool> edge(static_cast<size_t>(n) + 1, false);
  edge[0] = edge[static_cast<size_t>(n)] = true;
  for (const auto& k : b) {
    if (k.start < 0 || k.numel < 0 || k.S < 0 || k.S > daso::host::kMaxS || k.reserved != 0) return false;
    if (k.start + k.numel > n) return false;
    for (int64_t j = k.start; j < k.start + k.numel; ++j) ++cover[static_cast<size_t>(j)];
    if (k.numel > 0) edge[static_cast<size_t>(k.start)] = edge[static_cast<size_t>(k.start + k.numel)] = true;
  }
  for (int c : cover)
    if (c != 1) return false;
  for (const auto& k : b)
    if (k.numel == 0 && !edge[static_cast<size_t>(k.start)]) return false;
  return !b.empty();
}

static void bucket_checks(std::mt19937_64& rng) {
  for (int trial = 0; trial < 20000; ++trial) {
    const int64_t n = static_cast<int64_t>(rng() % 60);
    std::vector<daso_bucket> b;
    int64_t pos = 0;
    while (pos < n) {
      const int64_t k = 1 + static_cast<int64_t>(rng() % 9);
      b.push_back({pos, std::min(k, n - pos), static_cast<int32_t>(rng() % 5), 0});
      pos += b.back().numel;
    }
    if (b.empty()) b.push_back({0, 0, 1, 0});
    switch (rng() % 6) {  // perturb some tables
      case 0: b[rng() % b.size()].numel += 1; break;
      case 1: b[rng() % b.size()].start -= 1; break;
      case 2: b[rng() % b.size()].S = -1; break;
      case 3: b.push_back({static_cast<int64_t>(rng() % (n + 1)), 0, 2, 0}); break;
      case 4: std::swap(b.front(), b.back()); break;
      default: break;
    }
    const int rc = daso::host::check_buckets(b.data(), static_cast<int32_t>(b.size()), n);
    EXPECT((rc == DASO_OK) == tiles(b, n));
  }
  EXPECT(daso::host::check_buckets(nullptr, 1, 0) == DASO_EINVAL);
  daso_bucket huge[2] = {{0, INT64_MAX, 1, 0}, {INT64_MAX, 5, 1, 0}};
  EXPECT(daso::host::check_buckets(huge, 2, 4) == DASO_EINVAL);  // no overflow on the running sum
}

static void planner_checks(std::mt19937_64& rng) {
  for (int trial = 0; trial < 5000; ++trial) {
    const int nt = static_cast<int>(rng() % 30);
    std::vector<int64_t> numels(static_cast<size_t>(nt));
    int64_t total = 0;
    for (auto& k : numels) total += (k = static_cast<int64_t>(rng() % 500));
    const int64_t cap = 1 + static_cast<int64_t>(rng() % 2000);
    const int32_t cyc[3] = {1, 2, 4};
    const int32_t count = daso_plan_buckets(numels.data(), nt, cap, cyc, 3, nullptr, 0);
    EXPECT(count >= 0);
    std::vector<daso_bucket> out(static_cast<size_t>(count > 0 ? count : 1));
    EXPECT(daso_plan_buckets(numels.data(), nt, cap, cyc, 3, out.data(), count) == count);
    out.resize(static_cast<size_t>(count));
    if (total > 0 && total < 60 * 1000) {
      EXPECT(daso::host::check_buckets(out.data(), count, total) == DASO_OK);
    }
    for (int32_t b = 0; b + 1 < count; ++b) EXPECT(out[static_cast<size_t>(b)].numel >= cap);
    // a short output array gets the first buckets only
    if (count > 1) {
      std::vector<daso_bucket> two(1);
      EXPECT(daso_plan_buckets(numels.data(), nt, cap, cyc, 3, two.data(), 1) == count);
      EXPECT(two[0].start == out[0].start && two[0].numel == out[0].numel);
    }
  }
  const int64_t bad[2] = {3, -1};
  const int32_t one = 1;
  EXPECT(daso_plan_buckets(bad, 2, 10, &one, 1, nullptr, 0) == DASO_EINVAL);
  const int64_t big[2] = {INT64_MAX, 5};
  EXPECT(daso_plan_buckets(big, 2, 10, &one, 1, nullptr, 0) == DASO_EINVAL);
}

static void argument_checks() {
  const uintptr_t A = 0x10000000, MB = 1 << 20;
  auto P = [](uintptr_t v) { return reinterpret_cast<void*>(v); };
  const float* g4[4] = {(const float*)P(A), (const float*)P(A + MB), (const float*)P(A + 2 * MB),
                        (const float*)P(A + 3 * MB)};
  EXPECT(daso::host::check_local_avg(g4, 4, (const float*)P(A + 8 * MB), 1000) == DASO_OK);
  EXPECT(daso::host::check_local_avg(g4, 4, g4[2], 1000) == DASO_OK);                  // in place
  EXPECT(daso::host::check_local_avg(g4, 4, (const float*)P(A + MB + 64), 1000) == DASO_EALIAS);
  EXPECT(daso::host::check_local_avg(g4, 0, (const float*)P(A + 8 * MB), 1000) == DASO_EINVAL);
  EXPECT(daso::host::check_local_avg(nullptr, 4, nullptr, 0) == DASO_OK);                // n == 0: no pointer needed
  EXPECT(daso::host::check_pack((const float*)P(A), (const uint16_t*)P(A + 1008), 1000) == DASO_EALIAS);
  EXPECT(daso::host::check_pack(nullptr, nullptr, 0) == DASO_OK);

  const void* st[2] = {P(A + MB), P(A + 2 * MB)};
  const daso_bucket bk[2] = {{0, 600, 1, 0}, {600, 400, 2, 0}};
  EXPECT(daso::host::check_merge((const float*)P(A), st, 2, bk, 2, nullptr, 1000, 2) == DASO_OK);
  EXPECT(daso::host::check_merge((const float*)P(A), st, 2, bk, 2, P(A + 2 * MB + 512), 1000, 2) == DASO_EALIAS);
  EXPECT(daso::host::check_merge((const float*)P(A), st, 2, bk, 2, P(A + MB + 1008), 1000, 4) == DASO_EALIAS);

  const float* g2[2] = {(const float*)P(A), (const float*)P(A + MB)};
  const uint16_t* s2[2] = {(const uint16_t*)P(A + 10 * MB), (const uint16_t*)P(A + 11 * MB)};
  const daso_bucket one[1] = {{0, 1000, 2, 0}};
  daso_sync_args s{};
  s.n = 1000;
  s.g = 2;
  s.P = 2;
  s.grads = g2;
  s.stale = s2;
  s.params = (float*)P(A + 20 * MB);
  s.momentum = (float*)P(A + 21 * MB);
  s.wire = (uint16_t*)P(A + 22 * MB);
  s.buckets = one;
  s.nbuckets = 1;
  daso::host::FusedView v{};
  EXPECT(daso::host::check_fused(s, &v) == DASO_OK && !v.xf32 && v.esz == 2);
  s.grad_avg = const_cast<float*>(g2[1]);
  EXPECT(daso::host::check_fused(s, &v) == DASO_OK);                                     // allowed alias
  s.grad_avg = (float*)P(A + MB + 16);
  EXPECT(daso::host::check_fused(s, &v) == DASO_EALIAS);
  s.grad_avg = nullptr;
  s.flags = DASO_EXCHANGE_F32;
  EXPECT(daso::host::check_fused(s, &v) == DASO_EINVAL);                                 // stale still set
  const float* f2[2] = {(const float*)P(A + 10 * MB), (const float*)P(A + 11 * MB)};
  s.stale = nullptr;
  s.wire = nullptr;
  s.stale_f32 = f2;
  s.wire_f32 = (float*)P(A + 22 * MB);
  EXPECT(daso::host::check_fused(s, &v) == DASO_OK && v.xf32 && v.esz == 4);
  s.wire_f32 = (float*)P(A + 10 * MB + 2000);
  EXPECT(daso::host::check_fused(s, &v) == DASO_EALIAS);
}

static void schedule_checks(std::mt19937_64& rng) {
  for (int trial = 0; trial < 3000; ++trial) {
    daso_schedule_config c{};
    c.total_epochs = 1 + static_cast<int32_t>(rng() % 10);
    c.warmup_epochs = static_cast<int32_t>(rng() % (c.total_epochs + 1));
    c.cooldown_epochs = static_cast<int32_t>(rng() % (c.total_epochs - c.warmup_epochs + 1));
    c.batches_per_epoch = 1 + static_cast<int32_t>(rng() % 30);
    c.B_init = 1 + static_cast<int32_t>(rng() % 12);
    c.W_init = static_cast<int32_t>(rng() % (c.B_init + 1));
    c.group_count = 1 + static_cast<int32_t>(rng() % 8);
    c.local_rank = static_cast<int32_t>(rng() % c.group_count);
    c.patience = 1 + static_cast<int32_t>(rng() % 3);
    c.plateau_rel_tol = (rng() % 3) * 0.01;
    daso_schedule* s = nullptr;
    EXPECT(daso_schedule_create(&c, &s) == DASO_OK);
    daso_batch_plan p{};
    int64_t steps = 0, sends = 0, merges = 0;
    double loss = 1.0;
    while (true) {
      const int rc = daso_schedule_next(s, &p);
      if (rc == 0) break;
      EXPECT(rc == 1);
      EXPECT(p.step == steps);
      ++steps;
      const bool blocking = p.phase != DASO_PHASE_CYCLING;
      EXPECT(p.B >= 1 && p.W >= 1 && p.W <= c.B_init);
      if (blocking) EXPECT((p.actions & (DASO_ACT_BLOCKING | DASO_ACT_RECV_BCAST)) && p.S == 0);
      if (p.actions & DASO_ACT_MERGE) {
        EXPECT(!blocking && p.S >= 1 && p.merge_group == c.local_rank);
        ++merges;
      }
      if (p.actions & DASO_ACT_SEND) {
        EXPECT(!blocking && p.sync_group == c.local_rank);
        ++sends;
      }
      if (p.batch == c.batches_per_epoch - 1) {
        EXPECT(daso_schedule_next(s, &p) == DASO_EINVAL);  // the loss must come first
        loss *= (rng() % 2) ? 0.999 : 0.5;
        EXPECT(daso_schedule_end_epoch(s, loss) == DASO_OK);
      }
    }
    EXPECT(steps == int64_t(c.total_epochs) * c.batches_per_epoch);
    EXPECT(sends == merges);  // every exchange this GPU starts lands in time
    EXPECT(daso_schedule_end_epoch(s, 1.0) == DASO_EINVAL);
    daso_schedule_destroy(s);
  }
  daso_schedule_config bad{};
  daso_schedule* s = nullptr;
  EXPECT(daso_schedule_create(&bad, &s) == DASO_EINVAL);
  daso_schedule_destroy(nullptr);
}

// The launch grid: one workgroup per tile up to the cap, a whole number of
// XCD-run blocks beyond it, and always within the 32-bit work-item count of a
// dispatch of 256-thread workgroups.
static void grid_checks() {
  const int64_t cap = daso::host::kMaxGrid;
  EXPECT(cap * 256 < (int64_t(1) << 32));
  const int32_t runs[] = {1, 2, 3, 16, 32, 40, 1 << 20};
  const int64_t counts[] = {1, 2, 255, 256, 4097, cap - 1, cap, cap + 1, 3 * cap + 7,
                            int64_t(1) << 24, (int64_t(1) << 31) - 1};
  for (int32_t run : runs) {
    for (int64_t nt : counts) {
      const int64_t g = daso::host::launch_grid(nt, run);
      EXPECT(g >= 1 && g <= cap && g <= nt);
      if (nt <= cap) EXPECT(g == nt);
      if (nt > cap && 8 * int64_t(run) <= cap) EXPECT(g % (8 * int64_t(run)) == 0 && g > cap - 8 * int64_t(run));
    }
  }
  EXPECT(daso::host::launch_grid(0, 1) == 1);
}

int main() {
  std::mt19937_64 rng(2104);
  bucket_checks(rng);
  planner_checks(rng);
  argument_checks();
  schedule_checks(rng);
  grid_checks();
  if (failures) std::fprintf(stderr, "%d expectation(s) failed\n", failures);
  else std::printf("host checks ok\n");
  return failures ? 1 : 0;
}
