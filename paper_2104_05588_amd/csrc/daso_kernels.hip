// HIP kernels of the DASO synchronisation step for CDNA4 (gfx950).
//
// The step is a pure streaming computation: every output element depends only
// on the same element of each input stream, so the kernels read each stream
// once with 16-byte (fp32) or 8-byte (bf16) coalesced loads, keep everything
// in registers, and write each output once.  It is bound by HBM bandwidth, not
// arithmetic; there is no contraction, so no MFMA.
//
// Arithmetic follows the binary32 operation order stated in daso.h exactly
// (local average: Section 3, Figure 2; optimizer step: Sections 3.1 and 4;
// merge: Eq. (1); bf16 packing: Sections 3 and 4).  Floating-point contraction
// is off for this file and division is the correctly rounded one, so the
// results match a plain IEEE binary32 evaluation bit for bit.
#include "daso_launch.h"

#pragma clang fp contract(off)

namespace daso {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------ memory helpers
// FULL: the 4-element vector lies inside the tile; otherwise `mask` selects
// the elements to touch (bit k = element e0 + k) and the rest read as 0.
template <bool FULL, bool STREAM>
__device__ __forceinline__ f32x4 load_f32(const float* __restrict__ p, int64_t e0, unsigned mask) {
  if constexpr (FULL) {
    const f32x4* v = reinterpret_cast<const f32x4*>(p + e0);
    if constexpr (STREAM) return __builtin_nontemporal_load(v);
    else return *v;
  } else {
    f32x4 r = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (mask & (1u << k)) r[k] = p[e0 + k];
    return r;
  }
}

template <bool FULL>
__device__ __forceinline__ u32x2 load_bf16(const uint16_t* __restrict__ p, int64_t e0, unsigned mask) {
  if constexpr (FULL) {
    return __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p + e0));
  } else {
    uint32_t h[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (mask & (1u << k)) h[k] = p[e0 + k];
    u32x2 r;
    r.x = h[0] | (h[1] << 16);
    r.y = h[2] | (h[3] << 16);
    return r;
  }
}

template <bool FULL, bool STREAM>
__device__ __forceinline__ void store_f32(float* __restrict__ p, int64_t e0, unsigned mask, f32x4 v) {
  if constexpr (FULL) {
    f32x4* d = reinterpret_cast<f32x4*>(p + e0);
    if constexpr (STREAM) __builtin_nontemporal_store(v, d);
    else *d = v;
  } else {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (mask & (1u << k)) p[e0 + k] = v[k];
  }
}

template <bool FULL>
__device__ __forceinline__ void store_bf16(uint16_t* __restrict__ p, int64_t e0, unsigned mask, u32x2 w) {
  if constexpr (FULL) {
    __builtin_nontemporal_store(w, reinterpret_cast<u32x2*>(p + e0));
  } else {
    const uint32_t h[4] = {w.x & 0xFFFFu, w.x >> 16, w.y & 0xFFFFu, w.y >> 16};
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if (mask & (1u << k)) p[e0 + k] = static_cast<uint16_t>(h[k]);
  }
}

// ------------------------------------------------------------ bf16 helpers
// binary32 -> bfloat16, round to nearest even: add 0x7FFF plus the lowest kept
// bit and drop the low half; a mantissa carry moves to the next binade or to
// infinity.  NaN becomes the quiet NaN 0x7FC0.
__device__ __forceinline__ uint32_t bf16_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t r = (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
  return ((u & 0x7FFFFFFFu) > 0x7F800000u) ? 0x7FC0u : r;
}

__device__ __forceinline__ u32x2 pack4(f32x4 v) {
  u32x2 w;
  w.x = bf16_rne(v.x) | (bf16_rne(v.y) << 16);
  w.y = bf16_rne(v.z) | (bf16_rne(v.w) << 16);
  return w;
}

// Exact bfloat16 -> binary32: the pattern becomes the top half.
__device__ __forceinline__ f32x4 widen4(u32x2 h) {
  f32x4 r;
  r.x = __uint_as_float(h.x << 16);
  r.y = __uint_as_float(h.x & 0xFFFF0000u);
  r.z = __uint_as_float(h.y << 16);
  r.w = __uint_as_float(h.y & 0xFFFF0000u);
  return r;
}

// The exchanged copies and the wire are bf16 (XF = false) or fp32 (XF = true,
// the non-blocking exchange of Section 3, which is not cast).
template <bool XF>
struct XType {
  using T = u32x2;
};
template <>
struct XType<true> {
  using T = f32x4;
};

template <bool XF, bool FULL>
__device__ __forceinline__ typename XType<XF>::T load_x(const void* p, int64_t e0, unsigned mask) {
  if constexpr (XF) return load_f32<FULL, true>(static_cast<const float*>(p), e0, mask);
  else return load_bf16<FULL>(static_cast<const uint16_t*>(p), e0, mask);
}

template <bool XF>
__device__ __forceinline__ f32x4 received(typename XType<XF>::T v) {
  if constexpr (XF) return v;
  else return widen4(v);
}

template <bool XF, bool FULL>
__device__ __forceinline__ void store_wire(void* p, int64_t e0, unsigned mask, f32x4 v) {
  if constexpr (XF) store_f32<FULL, true>(static_cast<float*>(p), e0, mask, v);
  else store_bf16<FULL>(static_cast<uint16_t*>(p), e0, mask, pack4(v));
}

// Division by a per-bucket or per-call constant.  For a power of two the
// product with its (exact) reciprocal equals the correctly rounded quotient.
struct Divisor {
  float d;
  float inv;
  bool pow2;
};

__device__ __forceinline__ Divisor make_divisor(int k) {
  Divisor v;
  v.d = static_cast<float>(k);
  v.pow2 = k > 0 && (k & (k - 1)) == 0;
  v.inv = v.pow2 ? 1.0f / v.d : 0.0f;
  return v;
}

__device__ __forceinline__ f32x4 divide(f32x4 a, const Divisor& q) {
  if (q.pow2) return a * q.inv;
  f32x4 r;
  r.x = a.x / q.d;
  r.y = a.y / q.d;
  r.z = a.z / q.d;
  r.w = a.w / q.d;
  return r;
}

// --------------------------------------------------------------- statistics
// Per-thread sums over a tile (the count fits 32 bits: at most 32 elements per
// thread); the cross-tile reduction uses a 64-bit count.
template <typename CountT>
struct AccT {
  double gsq;
  double dsq;
  CountT nf;
};
using Acc = AccT<uint32_t>;
using Acc64 = AccT<uint64_t>;

__device__ __forceinline__ void accumulate(Acc& acc, f32x4 gbar, f32x4 xl, f32x4 xn, unsigned mask) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    if (mask & (1u << k)) {
      const double gv = static_cast<double>(gbar[k]);
      const double dv = static_cast<double>(xn[k]) - static_cast<double>(xl[k]);
      acc.gsq += gv * gv;
      acc.dsq += dv * dv;
      acc.nf += ((__float_as_uint(xn[k]) & 0x7F800000u) == 0x7F800000u) ? 1u : 0u;
    }
  }
}

// Deterministic block sum: a fixed xor-butterfly inside each wavefront, then the
// wavefront sums in index order.  Result valid in thread 0.
template <typename CountT>
__device__ __forceinline__ AccT<CountT> block_sum(AccT<CountT> v) {
  __shared__ double s_g[kBlock / 64];
  __shared__ double s_d[kBlock / 64];
  __shared__ CountT s_n[kBlock / 64];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    v.gsq += __shfl_xor(v.gsq, off, 64);
    v.dsq += __shfl_xor(v.dsq, off, 64);
    v.nf += __shfl_xor(v.nf, off, 64);
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    s_g[wave] = v.gsq;
    s_d[wave] = v.dsq;
    s_n[wave] = v.nf;
  }
  __syncthreads();
  AccT<CountT> r = {0.0, 0.0, 0};
  if (threadIdx.x == 0) {
    for (int w = 0; w < kBlock / 64; ++w) {
      r.gsq += s_g[w];
      r.dsq += s_d[w];
      r.nf += s_n[w];
    }
  }
  __syncthreads();
  return r;
}

// ------------------------------------------- arithmetic shared by both paths
// The local average's output: the local-average entry point stores it
// (streaming); the fused step stores it only when asked for.
template <int MODE, bool FULL>
__device__ __forceinline__ void store_avg(const StepArgs& a, int64_t e0, unsigned mask, f32x4 gbar) {
  if constexpr (MODE == kModeAvg) store_f32<FULL, true>(a.gavg, e0, mask, gbar);
  else if (a.gavg) store_f32<FULL, false>(a.gavg, e0, mask, gbar);
}

// The start of Eq. (1)'s sum: the local term 2S * xl.  S = 0 is the blocking
// synchronisation of Section 3, the plain average of the exchanged copies, so
// the local state is left out: the sum starts from -0, the identity of IEEE
// addition (-0 + c == c for every c), and a non-finite xl cannot reach it.
__device__ __forceinline__ f32x4 merge_start(float two_s, f32x4 xl) {
  if (two_s != 0.0f) return two_s * xl;
  return f32x4{-0.0f, -0.0f, -0.0f, -0.0f};
}

// The optimizer step (Section 3.1; PyTorch SGD with momentum, coupled weight
// decay that is skipped when zero): the local state xl; m becomes the new
// momentum.
__device__ __forceinline__ f32x4 sgd_momentum4(const StepArgs& a, f32x4 x, f32x4& m, f32x4 gbar) {
  f32x4 d = gbar;
  if (a.wd != 0.0f) d = gbar + (a.wd * x);
  m = (a.mu * m) + d;
  return x - (a.lr * m);
}

// The outputs after the merge: params, the wire (of x' or, with
// DASO_PACK_PRE_MERGE, of xl) and the statistics.
template <int MODE, bool FULL, bool STATS, bool XF>
__device__ __forceinline__ void store_results(const StepArgs& a, int64_t e0, unsigned mask, f32x4 gbar, f32x4 xl,
                                              f32x4 xn, Acc& acc) {
  store_f32<FULL, kNtParams>(a.x, e0, mask, xn);
  if (a.wire) {
    const bool pre = (MODE == kModeFused) && (a.flags & DASO_PACK_PRE_MERGE);
    store_wire<XF, FULL>(a.wire, e0, mask, pre ? xl : xn);
  }
  if constexpr (STATS && MODE == kModeFused) accumulate(acc, gbar, xl, xn, mask);
}

// ----------------------------------------------------------- one 4-vector
// Stream counts known only at run time: each input is folded in as it loads.
template <int MODE, int G, int PP, bool FULL, bool STATS, bool XF>
__device__ __forceinline__ void step_vec(const StepArgs& a, int64_t e0, unsigned mask, float two_s,
                                         const Divisor& qg, const Divisor& qm, Acc& acc) {
  if constexpr (MODE == kModePack) {
    const f32x4 v = load_f32<FULL, true>(a.src, e0, mask);
    store_wire<false, FULL>(a.wire, e0, mask, v);
    return;
  }
  const int g = (G > 0) ? G : a.g;
  const int P = (PP >= 0) ? PP : a.P;

  f32x4 gbar = {0.f, 0.f, 0.f, 0.f};
  if constexpr (MODE == kModeAvg || MODE == kModeFused) {
    f32x4 s = load_f32<FULL, true>(a.grads[0], e0, mask);
#pragma unroll
    for (int r = 1; r < g; ++r) s = s + load_f32<FULL, true>(a.grads[r], e0, mask);
    gbar = divide(s, qg);
    store_avg<MODE, FULL>(a, e0, mask, gbar);
    if constexpr (MODE == kModeAvg) return;
  }

  const f32x4 x = load_f32<FULL, kNtParams>(a.x, e0, mask);
  f32x4 xl = x;
  if constexpr (MODE == kModeFused) {
    f32x4 m = load_f32<FULL, kNtParams>(a.m, e0, mask);
    xl = sgd_momentum4(a, x, m, gbar);
    store_f32<FULL, kNtParams>(a.m, e0, mask, m);
  }

  f32x4 xn = xl;
  if (P > 0) {
    f32x4 acc4 = merge_start(two_s, xl);
#pragma unroll
    for (int i = 0; i < P; ++i) acc4 = acc4 + received<XF>(load_x<XF, FULL>(a.stale[i], e0, mask));
    xn = divide(acc4, qm);
  }
  store_results<MODE, FULL, STATS, XF>(a, e0, mask, gbar, xl, xn, acc);
}

// ------------------------------------- batched vectors (stream counts known)
// All loads of a batch of vectors are issued before the first store, so that a
// wavefront keeps every stream of several vectors in flight at once (the
// compiler cannot move later loads above earlier stores by itself: it cannot
// prove that the streams do not overlap).
// Stream counts: G > 0 and PP >= 0 are exact; G < 0 and PP <= -2 are run-time
// counts bounded by -G and -PP, whose missing streams are skipped (predicated);
// G == 0 and PP == -1 are unbounded run-time counts (the step_vec path).
template <int G>
constexpr int g_slots() { return G > 0 ? G : (G < 0 ? -G : 0); }
template <int PP>
constexpr int p_slots() { return PP >= 0 ? PP : (PP <= -2 ? -PP : 0); }

template <int MODE, int G, int PP, bool XF>
struct VecIn {
  static constexpr int kG = (MODE == kModeAvg || MODE == kModeFused) ? g_slots<G>() : 0;
  static constexpr int kP = (MODE == kModeMerge || MODE == kModeFused) ? p_slots<PP>() : 0;
  f32x4 g[kG > 0 ? kG : 1];
  f32x4 x;  // params (merge, fused) or the source (pack)
  f32x4 m;  // momentum (fused)
  typename XType<XF>::T s[kP > 0 ? kP : 1];
};

template <int MODE, int G, int PP, bool XF, bool FULL>
__device__ __forceinline__ void load_in(const StepArgs& a, int64_t e0, unsigned mask, VecIn<MODE, G, PP, XF>& v) {
  using V = VecIn<MODE, G, PP, XF>;
#pragma unroll
  for (int r = 0; r < V::kG; ++r)
    if (G > 0 || r < a.g) v.g[r] = load_f32<FULL, true>(a.grads[r], e0, mask);
  if constexpr (MODE == kModePack) v.x = load_f32<FULL, true>(a.src, e0, mask);
  if constexpr (MODE == kModeMerge || MODE == kModeFused) v.x = load_f32<FULL, kNtParams>(a.x, e0, mask);
  if constexpr (MODE == kModeFused) v.m = load_f32<FULL, kNtParams>(a.m, e0, mask);
#pragma unroll
  for (int i = 0; i < V::kP; ++i)
    if (PP >= 0 || i < a.P) v.s[i] = load_x<XF, FULL>(a.stale[i], e0, mask);
}

template <int MODE, int G, int PP, bool XF, bool FULL, bool STATS>
__device__ __forceinline__ void finish(const StepArgs& a, int64_t e0, unsigned mask,
                                       const VecIn<MODE, G, PP, XF>& v, float two_s, const Divisor& qg,
                                       const Divisor& qm, Acc& acc) {
  using V = VecIn<MODE, G, PP, XF>;
  if constexpr (MODE == kModePack) {
    store_wire<false, FULL>(a.wire, e0, mask, v.x);
    return;
  }
  f32x4 gbar = {0.f, 0.f, 0.f, 0.f};
  if constexpr (V::kG > 0) {
    f32x4 s = v.g[0];
#pragma unroll
    for (int r = 1; r < V::kG; ++r)
      if (G > 0 || r < a.g) s = s + v.g[r];
    gbar = divide(s, qg);
    store_avg<MODE, FULL>(a, e0, mask, gbar);
    if constexpr (MODE == kModeAvg) return;
  }
  f32x4 xl = v.x;
  if constexpr (MODE == kModeFused) {
    f32x4 m = v.m;
    xl = sgd_momentum4(a, v.x, m, gbar);
    store_f32<FULL, kNtParams>(a.m, e0, mask, m);
  }
  f32x4 xn = xl;
  if constexpr (V::kP > 0) {
    if (PP >= 0 || a.P > 0) {
      f32x4 acc4 = merge_start(two_s, xl);
#pragma unroll
      for (int i = 0; i < V::kP; ++i)
        if (PP >= 0 || i < a.P) acc4 = acc4 + received<XF>(v.s[i]);
      xn = divide(acc4, qm);
    }
  }
  store_results<MODE, FULL, STATS, XF>(a, e0, mask, gbar, xl, xn, acc);
}

// Whether an instance has compile-time stream counts or bounds (and so the
// batched path).
template <int MODE, int G, int PP>
constexpr bool batched() {
  if constexpr (MODE == kModePack) return true;
  if constexpr (MODE == kModeAvg) return G != 0;
  if constexpr (MODE == kModeMerge) return PP != -1;
  return G != 0 && PP != -1;
}

// Vectors per thread and tile: a batch of kBatch when a vector's inputs fit in
// 48 VGPRs, else one (measured: 2048-element tiles are best for the 40-register
// resnet50 step, 1024-element tiles for the 56- and 104-register ones); the
// runtime-count instances take kGenericIters vectors one after the other.
template <int MODE, int G, int PP, bool XF>
constexpr int iters_of() {
  if constexpr (!batched<MODE, G, PP>()) {
    return kGenericIters;
  } else {
    using V = VecIn<MODE, G, PP, XF>;
    constexpr int regs = 4 * V::kG + (XF ? 4 : 2) * V::kP + ((MODE == kModeFused) ? 8 : 4);
    return regs <= 48 ? kBatch : 1;
  }
}

template <int MODE, int G, int PP, bool XF>
constexpr int64_t tile_of() {
  return int64_t(kBlock) * kVec * iters_of<MODE, G, PP, XF>();
}

// ------------------------------------------------------------------- tiles
template <int MODE, int G, int PP, bool STATS, bool XF>
__device__ __forceinline__ void run_tile(const StepArgs& a, int64_t abase, int64_t tlo, int64_t thi, float two_s,
                                         const Divisor& qg, const Divisor& qm, Acc& acc) {
  constexpr bool kBatched = batched<MODE, G, PP>();
  constexpr int kIters = iters_of<MODE, G, PP, XF>();
  const int64_t t0 = abase + int64_t(threadIdx.x) * kVec;
  if constexpr (kBatched) {
    if (tlo == abase && thi == abase + tile_of<MODE, G, PP, XF>()) {
      // a whole tile: all loads of the thread's kIters vectors, then the stores
      VecIn<MODE, G, PP, XF> v[kIters];
#pragma unroll
      for (int b = 0; b < kIters; ++b) load_in<MODE, G, PP, XF, true>(a, t0 + int64_t(b) * kBlock * kVec, 0xFu, v[b]);
#pragma unroll
      for (int b = 0; b < kIters; ++b)
        finish<MODE, G, PP, XF, true, STATS>(a, t0 + int64_t(b) * kBlock * kVec, 0xFu, v[b], two_s, qg, qm, acc);
      return;
    }
  }
  for (int it = 0; it < kIters; ++it) {
    const int64_t e0 = t0 + int64_t(it) * kBlock * kVec;
    const bool full = e0 >= tlo && e0 + kVec <= thi;
    unsigned mask = 0xFu;
    if (!full) {
      if (e0 + kVec <= tlo || e0 >= thi) continue;
      mask = 0;
#pragma unroll
      for (int k = 0; k < kVec; ++k)
        if (e0 + k >= tlo && e0 + k < thi) mask |= 1u << k;
    }
    if constexpr (kBatched) {
      if (full) {
        VecIn<MODE, G, PP, XF> v;
        load_in<MODE, G, PP, XF, true>(a, e0, mask, v);
        finish<MODE, G, PP, XF, true, STATS>(a, e0, mask, v, two_s, qg, qm, acc);
      } else {
        // A vector cut by the bucket edge takes its elements one by one; folding
        // each stream in as it loads keeps this rarely run path from holding
        // every stream's addresses and values at once, which would otherwise set
        // the register count, and so the occupancy, of the whole kernel.
        step_vec<MODE, G, PP, false, STATS, XF>(a, e0, mask, two_s, qg, qm, acc);
      }
    } else {
      if (full) step_vec<MODE, G, PP, true, STATS, XF>(a, e0, mask, two_s, qg, qm, acc);
      else step_vec<MODE, G, PP, false, STATS, XF>(a, e0, mask, two_s, qg, qm, acc);
    }
  }
}

// The statistics of one bucket: the whole workgroup sums the tile partials
// [t0, t1) in a fixed assignment and reduction tree (thread k adds partials
// t0 + k, t0 + k + kBlock, ... in that order), so the result does not depend on
// timing, on which kernel runs it or on kLoads.  Valid in thread 0.
// The sum is latency-bound: each thread issues the loads of up to kLoads
// partials before it adds them in tile order.  Missing ones count as zeros,
// which leaves every sum unchanged (sums of squares are never -0).
template <int kLoads>
__device__ __forceinline__ Acc64 bucket_stats(const TilePartial* partials, int t0, int t1) {
  Acc64 v = {0.0, 0.0, 0};
  for (int base = t0 + static_cast<int>(threadIdx.x); base < t1; base += kBlock * kLoads) {
    TilePartial p[kLoads];
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      const int j = base + u * kBlock;
      p[u] = j < t1 ? partials[j] : TilePartial{0.0, 0.0, 0};
    }
#pragma unroll
    for (int u = 0; u < kLoads; ++u) {
      v.gsq += p[u].grad_sq;
      v.dsq += p[u].delta_sq;
      v.nf += p[u].nonfinite;
    }
  }
  return block_sum(v);
}

__device__ __forceinline__ void put_stats(daso_bucket_stats* out, const Acc64& r) {
  out->grad_sq = r.gsq;
  out->delta_sq = r.dsq;
  out->nonfinite = r.nf;
}

// A launch of few tiles sums its statistics in its own last workgroup instead
// of a second launch.  Each workgroup makes its partials visible to the whole
// chip (an agent-scope release fence: the XCD's L2 writes them back) and then
// counts itself done; the one that counts last takes an acquire fence and sums
// every bucket with the same code and order as stats_kernel, so the results
// are the same bits, and sets the counter back to zero for the next launch.
// The fences cost about 0.1 us per workgroup, which is why only small launches
// (at most kFinishStatsMaxTiles tiles, one workgroup each) take this path.
__device__ __forceinline__ void finish_stats_if_last(const StepArgs& a) {
  __shared__ bool last;
  __syncthreads();  // thread 0 has written this workgroup's partials
  if (threadIdx.x == 0) {
    __threadfence();
    last = atomicAdd(a.done, 1u) == gridDim.x - 1;
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  for (int i = 0; i < a.nb; ++i) {
    const int t1 = i + 1 < a.nb ? a.b[i + 1].first_tile : a.ntiles;
    const Acc64 r = bucket_stats<1>(a.partials, a.b[i].first_tile, t1);  // at most one partial per thread
    if (threadIdx.x == 0) put_stats(a.stats + i, r);
  }
  if (threadIdx.x == 0) atomicExch(a.done, 0u);
}

// ------------------------------------------------------------------- kernel
// One workgroup per tile; the loop serves a grid smaller than the tiles (the
// host caps the grid for launches of more than 2^20 tiles).
template <int MODE, int G, int PP, bool STATS, bool XF>
__global__ __launch_bounds__(kBlock) void step_kernel(const StepArgs a) {
  constexpr int64_t kTile = tile_of<MODE, G, PP, XF>();
  const int P = (PP >= 0) ? PP : a.P;
  const Divisor qg = make_divisor((G > 0) ? G : a.g);
  const int w0 = a.xcd_run > 1 ? xcd_runs(static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), a.xcd_run)
                               : static_cast<int>(blockIdx.x);
  if constexpr (STATS && MODE == kModeFused) {
    // the bucket ranges for stats_kernel (the grid has at least one workgroup)
    const int k = static_cast<int>(threadIdx.x);
    if (blockIdx.x == 0 && k <= a.nb) a.tile_table[k] = k < a.nb ? a.b[k].first_tile : a.ntiles;
  }
  for (int64_t t = w0; t < a.ntiles; t += gridDim.x) {
    const int tile = static_cast<int>(t);
    // bucket owning this tile: the last one whose first tile is <= tile
    int lo = 0, hi = a.nb - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.b[mid].first_tile <= tile) lo = mid;
      else hi = mid - 1;
    }
    const TileBucket bk = a.b[lo];
    const int64_t abase = (bk.start / kTile + int64_t(tile - bk.first_tile)) * kTile;  // on the tile grid
    const int64_t tlo = bk.start > abase ? bk.start : abase;
    const int64_t thi = bk.end < abase + kTile ? bk.end : abase + kTile;
    const float two_s = static_cast<float>(2 * bk.S);
    const Divisor qm = make_divisor(2 * bk.S + P);

    Acc acc = {0.0, 0.0, 0u};
    run_tile<MODE, G, PP, STATS, XF>(a, abase, tlo, thi, two_s, qg, qm, acc);
    if constexpr (STATS && MODE == kModeFused) {
      const Acc t = block_sum(acc);
      if (threadIdx.x == 0) {
        TilePartial* pt = a.partials + tile;
        pt->grad_sq = t.gsq;
        pt->delta_sq = t.dsq;
        pt->nonfinite = static_cast<uint64_t>(t.nf);
      }
    }
  }
  if constexpr (STATS && MODE == kModeFused) {
    if (a.done != nullptr) finish_stats_if_last(a);
  }
}

// Sets the counter of StepArgs::done at the start of a new statistics buffer
// to zero (a kernel rather than a memset, so that it may also sit in a graph).
__global__ void clear_counter_kernel(uint32_t* counter) {
  if (threadIdx.x == 0) *counter = 0u;
}

// Statistics of one launch: workgroup i sums the tile partials of bucket i.
// Runs after step_kernel on the same stream, which makes every partial, and the
// tile table, visible without any fence inside step_kernel.
__global__ __launch_bounds__(kBlock) void stats_kernel(const StatsArgs a) {
  const int i = static_cast<int>(blockIdx.x);
  // 16 loads per thread in flight: about 12 partials each for a 25 MiB bucket of 2048-element tiles
  const Acc64 r = bucket_stats<16>(a.partials, a.tile_table[i], a.tile_table[i + 1]);
  if (threadIdx.x == 0) put_stats(a.stats + i, r);
}

// Fused instances with compile-time stream counts for the node shapes: g = 4
// or 8 replicas (the GPUs of a node) with P in {2, 4, 8, 16, 32} exchanged
// copies (the nodes of a group), bf16 or fp32, and the local step (P = 0).
// Other pairs run an instance with bounded counts (below) or the run-time-count
// instance, which measured 3 to 7% slower than exact ones on the node shapes.
template <bool STATS, typename F>
auto dispatch_fused(const StepArgs& a, const F& f) {
  if (a.xf32) {
    if (a.g == 4 || a.g == 8) {
      const bool g8 = a.g == 8;
      switch (a.P) {
        case 2: return g8 ? f.template run<kModeFused, 8, 2, STATS, true>() : f.template run<kModeFused, 4, 2, STATS, true>();
        case 4: return g8 ? f.template run<kModeFused, 8, 4, STATS, true>() : f.template run<kModeFused, 4, 4, STATS, true>();
        case 8: return g8 ? f.template run<kModeFused, 8, 8, STATS, true>() : f.template run<kModeFused, 4, 8, STATS, true>();
        case 16: return g8 ? f.template run<kModeFused, 8, 16, STATS, true>() : f.template run<kModeFused, 4, 16, STATS, true>();
        case 32: return g8 ? f.template run<kModeFused, 8, 32, STATS, true>() : f.template run<kModeFused, 4, 32, STATS, true>();
        default: break;
      }
    }
    return f.template run<kModeFused, 0, -1, STATS, true>();
  }
  if (a.P == 0) {  // the local step of most cycling batches (no copies arrive)
    switch (a.g) {
      case 1: return f.template run<kModeFused, 1, 0, STATS, false>();
      case 2: return f.template run<kModeFused, 2, 0, STATS, false>();
      case 4: return f.template run<kModeFused, 4, 0, STATS, false>();
      case 8: return f.template run<kModeFused, 8, 0, STATS, false>();
      default: break;
    }
  }
  if (a.g == 4) {
    switch (a.P) {
      case 2: return f.template run<kModeFused, 4, 2, STATS, false>();
      case 4: return f.template run<kModeFused, 4, 4, STATS, false>();
      case 8: return f.template run<kModeFused, 4, 8, STATS, false>();
      case 16: return f.template run<kModeFused, 4, 16, STATS, false>();
      case 32: return f.template run<kModeFused, 4, 32, STATS, false>();
      default: break;
    }
  }
  if (a.g == 8) {
    switch (a.P) {
      case 2: return f.template run<kModeFused, 8, 2, STATS, false>();
      case 4: return f.template run<kModeFused, 8, 4, STATS, false>();
      case 8: return f.template run<kModeFused, 8, 8, STATS, false>();
      case 16: return f.template run<kModeFused, 8, 16, STATS, false>();
      case 32: return f.template run<kModeFused, 8, 32, STATS, false>();
      default: break;
    }
  }
  // other counts up to 8 replicas and 16 copies: instances bounded by 4 or 8
  // and 8 or 16 streams, the missing ones skipped (measured 4 to 7% faster than
  // the run-time-count instance there; slower beyond 16 copies, and no faster
  // for g = 8 with fewer than 8 copies)
  if (a.g <= 4 && a.P <= 16) {
    if (a.P <= 8) return f.template run<kModeFused, -4, -8, STATS, false>();
    return f.template run<kModeFused, -4, -16, STATS, false>();
  }
  if (a.g <= 8 && a.P <= 16 && (a.g < 8 || a.P > 8)) {
    if (a.P <= 8) return f.template run<kModeFused, -8, -8, STATS, false>();
    return f.template run<kModeFused, -8, -16, STATS, false>();
  }
  return f.template run<kModeFused, 0, -1, STATS, false>();
}

// The instance for a call, chosen in one place: `f.template run<MODE, G, PP,
// STATS, XF>()` is called for it, both to launch and to size the tiles, so the
// two always agree.  Fully unrolled instances exist for common stream counts;
// any other count takes the runtime-count instance, which computes the same bits.
template <typename F>
auto dispatch(Mode mode, bool with_stats, const StepArgs& a, const F& f) {
  switch (mode) {
    case kModeAvg:
      switch (a.g) {
        case 1: return f.template run<kModeAvg, 1, -1, false, false>();
        case 2: return f.template run<kModeAvg, 2, -1, false, false>();
        case 4: return f.template run<kModeAvg, 4, -1, false, false>();
        case 8: return f.template run<kModeAvg, 8, -1, false, false>();
        default:
          if (a.g <= 8) return f.template run<kModeAvg, -8, -1, false, false>();
          return f.template run<kModeAvg, 0, -1, false, false>();
      }
    case kModePack:
      return f.template run<kModePack, 0, -1, false, false>();
    case kModeMerge:
      if (a.xf32) {
        if (a.P == 8) return f.template run<kModeMerge, 0, 8, false, true>();
        return f.template run<kModeMerge, 0, -1, false, true>();
      }
      switch (a.P) {
        case 0: return f.template run<kModeMerge, 0, 0, false, false>();
        case 2: return f.template run<kModeMerge, 0, 2, false, false>();
        case 4: return f.template run<kModeMerge, 0, 4, false, false>();
        case 8: return f.template run<kModeMerge, 0, 8, false, false>();
        case 16: return f.template run<kModeMerge, 0, 16, false, false>();
        case 32: return f.template run<kModeMerge, 0, 32, false, false>();
        default:
          if (a.P <= 8) return f.template run<kModeMerge, 0, -8, false, false>();
          if (a.P <= 16) return f.template run<kModeMerge, 0, -16, false, false>();
          return f.template run<kModeMerge, 0, -1, false, false>();
      }
    case kModeFused:
    default:
      if (with_stats) return dispatch_fused<true>(a, f);
      return dispatch_fused<false>(a, f);
  }
}

// Launches report their own status (hipLaunchKernel's return value), so an
// error left behind by an earlier, unrelated HIP call is neither blamed on
// this call nor consumed by it.
struct Launcher {
  const StepArgs& a;
  uint32_t grid;
  uint32_t lds;  // LDS held per workgroup (unused by the kernel; caps workgroups per CU)
  hipStream_t stream;
  template <int MODE, int G, int PP, bool STATS, bool XF>
  hipError_t run() const {
    void* args[] = {const_cast<StepArgs*>(&a)};
    const hipError_t e = hipLaunchKernel(reinterpret_cast<const void*>(&step_kernel<MODE, G, PP, STATS, XF>),
                                         dim3(grid), dim3(kBlock), args, lds, stream);
    if (e != hipSuccess || !STATS || a.done != nullptr) return e;
    StatsArgs sa = {a.partials, a.tile_table, a.stats, a.nb};
    void* sargs[] = {&sa};
    return hipLaunchKernel(reinterpret_cast<const void*>(&stats_kernel), dim3(a.nb), dim3(kBlock), sargs, 0, stream);
  }
};

struct TileSize {
  template <int MODE, int G, int PP, bool STATS, bool XF>
  int64_t run() const {
    return tile_of<MODE, G, PP, XF>();
  }
};

}  // namespace

int64_t tile_elems(Mode mode, bool with_stats, const StepArgs& a) {
  return dispatch(mode, with_stats, a, TileSize{});
}

hipError_t launch_step(Mode mode, bool with_stats, const StepArgs& a, uint32_t grid, uint32_t lds,
                       hipStream_t stream) {
  return dispatch(mode, with_stats, a, Launcher{a, grid, lds, stream});
}

hipError_t clear_stats_counter(void* buffer, hipStream_t stream) {
  void* args[] = {&buffer};
  return hipLaunchKernel(reinterpret_cast<const void*>(&clear_counter_kernel), dim3(1), dim3(64), args, 0, stream);
}

}  // namespace daso
