// Bandwidth ceilings of the fused step's memory access pattern, for the bench
// only (a library of its own, outside the C ABI of include/daso.h).
//
// Each probe kernel makes exactly the loads and stores of a fused step, on the
// same tile grid, tile size and tile order, with the same access widths (16
// bytes per lane for fp32 streams, 8 for bf16) and non-temporal hints, and none
// of its arithmetic: R32 fp32 and R16 bf16 streams read, W32 fp32 and W16 bf16
// streams written.  Taking the reads alone, the writes alone and both mixed,
// they measure what the step's access mix can reach on a given part; a one-
// stream copy gives the plain copy rate.  Two more mixed probes take bf16 at 16
// bytes per lane, to price the wider bf16 access, and a phased probe separates
// reads from writes across the whole chip, as the separated bound assumes.
//
// Safety: every stream holds at least n elements and n is a multiple of 4, of 8
// for the 16-byte bf16 probes (checked by daso_probe_run before any launch), so a
// thread touches the vector at element e0 only when e0 < n, which keeps the
// whole vector inside every buffer.  The grid is at most the tile count of the
// probe's own tile size, each workgroup looping over tiles grid apart, so every
// tile is visited once.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "daso_launch.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kProbeBlock = 256;
constexpr int kMaxRead = 48;
constexpr int kMaxWrite = 4;

struct ProbeArgs {
  const void* rd32[kMaxRead];  // fp32 streams read
  const void* rd16[kMaxRead];  // bf16 streams read
  void* wr32[kMaxWrite];       // fp32 streams written
  void* wr16[kMaxWrite];       // bf16 streams written
  uint32_t* sink;              // one word: a read-only probe stores its fold here when sink_flag != 0
  int64_t n;                   // elements per stream, a multiple of 4 (of 8 for the 16-byte bf16 probes)
  int32_t ntiles;
  int32_t xcd_run;
  int32_t sink_flag;           // 0 in every run; keeps the loads of a read-only probe alive
};

template <int R32, int R16, int W32, int W16, int ITERS>
__global__ __launch_bounds__(kProbeBlock) void probe_kernel(const ProbeArgs a) {
  constexpr int64_t kTile = int64_t(kProbeBlock) * 4 * ITERS;
  const int w0 = a.xcd_run > 1 ? daso::xcd_runs(static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), a.xcd_run)
                               : static_cast<int>(blockIdx.x);
  for (int64_t t = w0; t < a.ntiles; t += gridDim.x) {
    const int64_t base = t * kTile + int64_t(threadIdx.x) * 4;
    u32x4 r32[ITERS][R32 > 0 ? R32 : 1];
    u32x2 r16[ITERS][R16 > 0 ? R16 : 1];
    // every load of the thread's vectors first, as the step issues them
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int64_t e0 = base + int64_t(it) * kProbeBlock * 4;
      if (e0 < a.n) {
#pragma unroll
        for (int s = 0; s < R32; ++s)
          r32[it][s] = __builtin_nontemporal_load(static_cast<const u32x4*>(a.rd32[s]) + e0 / 4);
#pragma unroll
        for (int s = 0; s < R16; ++s)
          r16[it][s] = __builtin_nontemporal_load(static_cast<const u32x2*>(a.rd16[s]) + e0 / 4);
      }
    }
#pragma unroll
    for (int it = 0; it < ITERS; ++it) {
      const int64_t e0 = base + int64_t(it) * kProbeBlock * 4;
      if (e0 >= a.n) continue;
      u32x4 v = {static_cast<uint32_t>(e0), 1u, 2u, 3u};
#pragma unroll
      for (int s = 0; s < R32; ++s) v ^= r32[it][s];
#pragma unroll
      for (int s = 0; s < R16; ++s) {
        v.x ^= r16[it][s].x;
        v.y ^= r16[it][s].y;
      }
#pragma unroll
      for (int w = 0; w < W32; ++w) __builtin_nontemporal_store(v, static_cast<u32x4*>(a.wr32[w]) + e0 / 4);
#pragma unroll
      for (int w = 0; w < W16; ++w) {
        const u32x2 h = {v.x, v.y};
        __builtin_nontemporal_store(h, static_cast<u32x2*>(a.wr16[w]) + e0 / 4);
      }
      if constexpr (W32 + W16 == 0) {
        if (a.sink_flag) a.sink[0] = v.x ^ v.y ^ v.z ^ v.w;
      }
    }
  }
}

// The same mix on 2048-element tiles with bf16 accessed at 16 bytes per lane,
// in two forms.  SAME: each lane takes its own 8 consecutive elements, fp32 as
// two adjacent 16-byte accesses (a 32-byte stride between lanes), bf16 as one
// 16-byte access: the layout a step would need to keep a lane's elements
// together.  !SAME: fp32 as the step takes it (lane i at elements 4i and
// 1024 + 4i of the tile, every access contiguous across the wavefront), bf16 at
// elements 8i to 8i + 7: a lane then holds different elements of the two types,
// which a step would have to exchange between lanes; this bounds what the wider
// bf16 access alone could give.  Every stream holds at least n elements and n
// is a multiple of 8, so each guarded vector lies inside its buffer.
template <int R32, int R16, int W32, int W16, bool SAME>
__global__ __launch_bounds__(kProbeBlock) void probe_wide_kernel(const ProbeArgs a) {
  constexpr int64_t kTile = int64_t(kProbeBlock) * 8;
  const int w0 = a.xcd_run > 1 ? daso::xcd_runs(static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), a.xcd_run)
                               : static_cast<int>(blockIdx.x);
  for (int64_t t = w0; t < a.ntiles; t += gridDim.x) {
    const int64_t e16 = t * kTile + int64_t(threadIdx.x) * 8;  // the lane's bf16 vector
    int64_t e32[2];                                             // the lane's fp32 vectors
    e32[0] = SAME ? e16 : t * kTile + int64_t(threadIdx.x) * 4;
    e32[1] = SAME ? e16 + 4 : e32[0] + int64_t(kProbeBlock) * 4;
    const bool in16 = e16 < a.n, in32[2] = {e32[0] < a.n, e32[1] < a.n};
    u32x4 r32[R32 > 0 ? R32 : 1][2];
    u32x4 r16[R16 > 0 ? R16 : 1];
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (in32[h]) {
#pragma unroll
        for (int s = 0; s < R32; ++s)
          r32[s][h] = __builtin_nontemporal_load(static_cast<const u32x4*>(a.rd32[s]) + e32[h] / 4);
      }
    if (in16) {
#pragma unroll
      for (int s = 0; s < R16; ++s) r16[s] = __builtin_nontemporal_load(static_cast<const u32x4*>(a.rd16[s]) + e16 / 8);
    }
    u32x4 v[2] = {{static_cast<uint32_t>(e16), 1u, 2u, 3u}, {static_cast<uint32_t>(e16), 5u, 6u, 7u}};
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (in32[h]) {
#pragma unroll
        for (int s = 0; s < R32; ++s) v[h] ^= r32[s][h];
      }
    u32x4 v16 = v[0] ^ v[1];
    if (in16) {
#pragma unroll
      for (int s = 0; s < R16; ++s) v16 ^= r16[s];
    }
#pragma unroll
    for (int h = 0; h < 2; ++h)
      if (in32[h]) {
#pragma unroll
        for (int w = 0; w < W32; ++w) __builtin_nontemporal_store(v[h] ^ v16, static_cast<u32x4*>(a.wr32[w]) + e32[h] / 4);
      }
    if (in16) {
#pragma unroll
      for (int w = 0; w < W16; ++w) __builtin_nontemporal_store(v16, static_cast<u32x4*>(a.wr16[w]) + e16 / 8);
    }
  }
}

// Reads and writes separated across the whole chip: every workgroup reads K
// tiles of the step's mix (the values of probe_kernel<R32, R16, 2, 1, ITERS>)
// into LDS, all workgroups meet, every workgroup writes its K tiles' outputs,
// all meet again, and so on.  This is the schedule the separated bound assumes,
// made real.  The meeting is a counter in device memory that every workgroup
// raises once per meeting (an agent-scope atomic add) and then polls; a wait
// longer than spin_limit polls gives up, counts itself in *late and goes on, so
// every wait ends even if some workgroup were never to arrive.  The launch is
// cooperative, so all workgroups are resident at once.  Every workgroup runs
// the same number of rounds and meetings; tile t of round r is r * gridDim.x * K
// + blockIdx.x * K + k, each guarded by the tile count and the element count.
struct PhasedArgs {
  ProbeArgs p;
  uint32_t* ctr;   // meeting counter, zeroed before the launch
  uint32_t* late;  // waits that gave up
  int32_t spin_limit;
};

__device__ __forceinline__ void meet(const PhasedArgs& a, uint32_t target) {
  __syncthreads();
  if (threadIdx.x == 0) {
    __hip_atomic_fetch_add(a.ctr, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int32_t polls = 0;
    while (__hip_atomic_load(a.ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      if (++polls > a.spin_limit) {
        __hip_atomic_fetch_add(a.late, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  __syncthreads();
}

template <int R32, int R16, int ITERS, int K>
__global__ __launch_bounds__(kProbeBlock) void phased_kernel(const PhasedArgs a) {
  extern __shared__ u32x4 staged[];  // [K][ITERS][kProbeBlock]
  constexpr int64_t kTile = int64_t(kProbeBlock) * 4 * ITERS;
  const ProbeArgs& q = a.p;
  uint32_t met = 0;
  for (int64_t base = 0; base < q.ntiles; base += int64_t(gridDim.x) * K) {
#pragma unroll 1
    for (int k = 0; k < K; ++k) {
      const int64_t t = base + int64_t(blockIdx.x) * K + k;
      if (t >= q.ntiles) break;
      u32x4 r32[ITERS][R32];
      u32x2 r16[ITERS][R16];
#pragma unroll
      for (int it = 0; it < ITERS; ++it) {
        const int64_t e0 = t * kTile + int64_t(threadIdx.x) * 4 + int64_t(it) * kProbeBlock * 4;
        if (e0 < q.n) {
#pragma unroll
          for (int s = 0; s < R32; ++s)
            r32[it][s] = __builtin_nontemporal_load(static_cast<const u32x4*>(q.rd32[s]) + e0 / 4);
#pragma unroll
          for (int s = 0; s < R16; ++s)
            r16[it][s] = __builtin_nontemporal_load(static_cast<const u32x2*>(q.rd16[s]) + e0 / 4);
        }
      }
#pragma unroll
      for (int it = 0; it < ITERS; ++it) {
        const int64_t e0 = t * kTile + int64_t(threadIdx.x) * 4 + int64_t(it) * kProbeBlock * 4;
        if (e0 >= q.n) continue;
        u32x4 v = {static_cast<uint32_t>(e0), 1u, 2u, 3u};
#pragma unroll
        for (int s = 0; s < R32; ++s) v ^= r32[it][s];
#pragma unroll
        for (int s = 0; s < R16; ++s) {
          v.x ^= r16[it][s].x;
          v.y ^= r16[it][s].y;
        }
        staged[(k * ITERS + it) * kProbeBlock + threadIdx.x] = v;
      }
    }
    met += gridDim.x;
    meet(a, met);
#pragma unroll 1
    for (int k = 0; k < K; ++k) {
      const int64_t t = base + int64_t(blockIdx.x) * K + k;
      if (t >= q.ntiles) break;
#pragma unroll
      for (int it = 0; it < ITERS; ++it) {
        const int64_t e0 = t * kTile + int64_t(threadIdx.x) * 4 + int64_t(it) * kProbeBlock * 4;
        if (e0 >= q.n) continue;
        const u32x4 v = staged[(k * ITERS + it) * kProbeBlock + threadIdx.x];
        __builtin_nontemporal_store(v, static_cast<u32x4*>(q.wr32[0]) + e0 / 4);
        __builtin_nontemporal_store(v, static_cast<u32x4*>(q.wr32[1]) + e0 / 4);
        const u32x2 h = {v.x, v.y};
        __builtin_nontemporal_store(h, static_cast<u32x2*>(q.wr16[0]) + e0 / 4);
      }
    }
    met += gridDim.x;
    meet(a, met);
  }
}

// Tiles staged per workgroup and round: as many as fit 72 KB of LDS, so that
// two workgroups share a CU as in the step's launches.
template <int ITERS>
constexpr int phased_tiles() {
  return (72 * 1024) / (ITERS * kProbeBlock * 16);
}

template <int R32, int R16, int W32, int W16, int ITERS>
hipError_t launch(const ProbeArgs& a, uint32_t grid, uint32_t lds, hipStream_t stream) {
  void* args[] = {const_cast<ProbeArgs*>(&a)};
  const void* k;
  if constexpr (ITERS == 0)
    k = reinterpret_cast<const void*>(&probe_wide_kernel<R32, R16, W32, W16, true>);
  else if constexpr (ITERS == -1)
    k = reinterpret_cast<const void*>(&probe_wide_kernel<R32, R16, W32, W16, false>);
  else
    k = reinterpret_cast<const void*>(&probe_kernel<R32, R16, W32, W16, ITERS>);
  return hipLaunchKernel(k, dim3(grid), dim3(kProbeBlock), args, lds, stream);
}

// The access shapes of the fused step on the five workloads (g + 2 fp32 reads,
// P bf16 reads; params and momentum written in fp32, the wire in bf16; 2048-
// element tiles up to 8 copies, 1024 beyond), their reads alone and writes
// alone, and a plain copy.
#define DASO_PROBE_SHAPES(X)                                                   \
  X(6, 2, 2, 1, 2) X(6, 2, 0, 0, 2) X(0, 0, 2, 1, 2)   /* g=4, P=2  */        \
  X(6, 4, 2, 1, 2) X(6, 4, 0, 0, 2)                    /* g=4, P=4  */        \
  X(6, 8, 2, 1, 2) X(6, 8, 0, 0, 2)                    /* g=4, P=8  */        \
  X(6, 16, 2, 1, 1) X(6, 16, 0, 0, 1) X(0, 0, 2, 1, 1) /* g=4, P=16 */        \
  X(10, 32, 2, 1, 1) X(10, 32, 0, 0, 1)                /* g=8, P=32 */        \
  X(1, 0, 1, 0, 2)                                     /* copy      */        \
  X(6, 8, 2, 1, 0) X(6, 8, 2, 1, -1)                   /* g=4, P=8, bf16 16 B */

}  // namespace

extern "C" {

// Runs one probe: r32/r16 read streams and w32/w16 written streams (host arrays
// of device pointers, each stream at least n elements of 4 or 2 bytes), tiles of
// 1024 * iters elements (iters 1 or 2, 4-element vectors; iters 0 and -1: the
// two 16-byte bf16 forms of probe_wide_kernel, SAME and not, on 2048-element
// tiles, n a multiple of 8) in runs of xcd_run tiles per XCD, each workgroup holding
// lds_bytes of (unused) LDS, which caps how many share a CU, as the step's
// launches do.  Returns 0, -1 for a shape without an instance or invalid
// sizes/pointers, -4 when the launch fails.  Nothing is launched on -1.
int daso_probe_run(const void* const* rd32, int32_t r32, const void* const* rd16, int32_t r16, void* const* wr32,
                   int32_t w32, void* const* wr16, int32_t w16, uint32_t* sink, int64_t n, int32_t iters,
                   int32_t xcd_run, int32_t lds_bytes, hipStream_t stream) {
  if (n <= 0 || n % 4 != 0 || iters < -1 || iters > 2 || xcd_run < 1 || sink == nullptr) return -1;
  if (iters <= 0 && n % 8 != 0) return -1;
  if (lds_bytes < 0 || lds_bytes > 160 * 1024) return -1;
  if (r32 < 0 || r32 > kMaxRead || r16 < 0 || r16 > kMaxRead || w32 < 0 || w32 > kMaxWrite || w16 < 0 ||
      w16 > kMaxWrite)
    return -1;
  ProbeArgs a = {};
  for (int i = 0; i < r32; ++i) {
    if (rd32 == nullptr || rd32[i] == nullptr || (reinterpret_cast<uintptr_t>(rd32[i]) & 15u)) return -1;
    a.rd32[i] = rd32[i];
  }
  for (int i = 0; i < r16; ++i) {
    if (rd16 == nullptr || rd16[i] == nullptr || (reinterpret_cast<uintptr_t>(rd16[i]) & 15u)) return -1;
    a.rd16[i] = rd16[i];
  }
  for (int i = 0; i < w32; ++i) {
    if (wr32 == nullptr || wr32[i] == nullptr || (reinterpret_cast<uintptr_t>(wr32[i]) & 15u)) return -1;
    a.wr32[i] = wr32[i];
  }
  for (int i = 0; i < w16; ++i) {
    if (wr16 == nullptr || wr16[i] == nullptr || (reinterpret_cast<uintptr_t>(wr16[i]) & 15u)) return -1;
    a.wr16[i] = wr16[i];
  }
  const int64_t tile = int64_t(kProbeBlock) * (iters <= 0 ? 8 : 4 * iters);
  const int64_t ntiles = (n + tile - 1) / tile;
  if (ntiles > INT32_MAX) return -1;
  a.sink = sink;
  a.n = n;
  a.ntiles = static_cast<int32_t>(ntiles);
  a.xcd_run = xcd_run;
  a.sink_flag = 0;
  const int64_t block = 8 * int64_t(xcd_run);
  const int64_t cap = int64_t(1) << 20;
  const int64_t grid = ntiles <= cap ? ntiles : (block <= cap ? (cap / block) * block : cap);
  const uint32_t g32 = static_cast<uint32_t>(grid), lds = static_cast<uint32_t>(lds_bytes);
#define DASO_PROBE_CASE(A, B, C, D, E)                                      \
  if (r32 == (A) && r16 == (B) && w32 == (C) && w16 == (D) && iters == (E)) \
    return launch<A, B, C, D, E>(a, g32, lds, stream) == hipSuccess ? 0 : -4;
  DASO_PROBE_SHAPES(DASO_PROBE_CASE)
#undef DASO_PROBE_CASE
  return -1;
}

// Runs phased_kernel over r32 fp32 and r16 bf16 read streams and the step's
// three written streams (wr32[0..1] fp32, wr16[0] bf16), each at least n
// elements (n a multiple of 4), on nwg workgroups (a cooperative launch: all of
// them resident at once, else the launch fails).  iters as in daso_probe_run
// (1 or 2 four-element vectors per thread); shapes: g = 4, P = 8 (6, 8, iters
// 2) and g = 8, P = 32 (10, 32, iters 1).  ctr is one device word that the
// call zeroes on `stream` before the launch; late (one device word, not
// cleared) gains one for every wait that gave up after spin_limit polls.
// Returns 0, -1 for invalid arguments or a shape without an instance (nothing
// launched), -4 when a HIP call fails.
int daso_probe_phased(const void* const* rd32, int32_t r32, const void* const* rd16, int32_t r16, void* const* wr32,
                      void* const* wr16, uint32_t* ctr, uint32_t* late, int64_t n, int32_t iters, int32_t nwg,
                      int32_t spin_limit, hipStream_t stream) {
  if (n <= 0 || n % 4 != 0 || nwg < 1 || nwg > 4096 || spin_limit < 1 || ctr == nullptr || late == nullptr) return -1;
  if (r32 < 0 || r32 > kMaxRead || r16 < 0 || r16 > kMaxRead || wr32 == nullptr || wr16 == nullptr) return -1;
  PhasedArgs a = {};
  for (int i = 0; i < r32; ++i) {
    if (rd32 == nullptr || rd32[i] == nullptr || (reinterpret_cast<uintptr_t>(rd32[i]) & 15u)) return -1;
    a.p.rd32[i] = rd32[i];
  }
  for (int i = 0; i < r16; ++i) {
    if (rd16 == nullptr || rd16[i] == nullptr || (reinterpret_cast<uintptr_t>(rd16[i]) & 15u)) return -1;
    a.p.rd16[i] = rd16[i];
  }
  for (int i = 0; i < 2; ++i) {
    if (wr32[i] == nullptr || (reinterpret_cast<uintptr_t>(wr32[i]) & 15u)) return -1;
    a.p.wr32[i] = wr32[i];
  }
  if (wr16[0] == nullptr || (reinterpret_cast<uintptr_t>(wr16[0]) & 15u)) return -1;
  a.p.wr16[0] = wr16[0];
  const void* k = nullptr;
  int tiles = 0;
  if (r32 == 6 && r16 == 8 && iters == 2) {
    k = reinterpret_cast<const void*>(&phased_kernel<6, 8, 2, phased_tiles<2>()>);
    tiles = phased_tiles<2>();
  } else if (r32 == 10 && r16 == 32 && iters == 1) {
    k = reinterpret_cast<const void*>(&phased_kernel<10, 32, 1, phased_tiles<1>()>);
    tiles = phased_tiles<1>();
  } else {
    return -1;
  }
  const int64_t tile = int64_t(kProbeBlock) * 4 * iters;
  const int64_t ntiles = (n + tile - 1) / tile;
  const int64_t rounds = (ntiles + int64_t(nwg) * tiles - 1) / (int64_t(nwg) * tiles);
  if (ntiles > INT32_MAX || rounds * 2 * nwg > int64_t(UINT32_MAX)) return -1;
  a.p.n = n;
  a.p.ntiles = static_cast<int32_t>(ntiles);
  a.p.xcd_run = 1;
  a.ctr = ctr;
  a.late = late;
  a.spin_limit = spin_limit;
  const uint32_t lds = static_cast<uint32_t>(tiles) * iters * kProbeBlock * 16;
  if (hipMemsetAsync(ctr, 0, sizeof(uint32_t), stream) != hipSuccess) return -4;
  void* args[] = {&a};
  return hipLaunchCooperativeKernel(k, dim3(static_cast<uint32_t>(nwg)), dim3(kProbeBlock), args, lds, stream) ==
                 hipSuccess
             ? 0
             : -4;
}

}  // extern "C"
