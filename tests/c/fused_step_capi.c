/* A plain C client of the DASO library: reads one fused-step problem from a
 * file, runs daso_fused_sync_step on device buffers from hipMalloc, and writes
 * the results.  Used by the GPU tests to show the C ABI works without Python.
 *
 * usage: fused_step_capi <input> <output>
 * input:  int64 n; int32 g, P, nbuckets; float lr, mu, wd; uint32 flags;
 *         nbuckets x {int64 start, int64 numel, int32 S, int32 0};
 *         g x n float grads; n float params; n float momentum; P x n uint16 stale
 * output: n float params; n float momentum; n uint16 wire; nbuckets x daso_bucket_stats
 */
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "daso.h"

#define HIP_OK(call)                                                        \
  do {                                                                      \
    hipError_t e_ = (call);                                                 \
    if (e_ != hipSuccess) {                                                 \
      fprintf(stderr, "%s failed: %s\n", #call, hipGetErrorString(e_));     \
      exit(3);                                                              \
    }                                                                       \
  } while (0)

static void read_all(FILE* f, void* p, size_t bytes) {
  if (bytes && fread(p, 1, bytes, f) != bytes) {
    fprintf(stderr, "short input\n");
    exit(2);
  }
}

static void* device_alloc(size_t bytes) {
  void* d = NULL;
  HIP_OK(hipMalloc(&d, bytes ? bytes : 16));
  return d;
}

static void* upload(const void* host, size_t bytes) {
  void* d = device_alloc(bytes);
  if (bytes) HIP_OK(hipMemcpy(d, host, bytes, hipMemcpyHostToDevice));
  return d;
}

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s <input> <output>\n", argv[0]);
    return 2;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  int64_t n;
  int32_t g, P, nb;
  float lr, mu, wd;
  uint32_t flags;
  read_all(in, &n, 8);
  read_all(in, &g, 4);
  read_all(in, &P, 4);
  read_all(in, &nb, 4);
  read_all(in, &lr, 4);
  read_all(in, &mu, 4);
  read_all(in, &wd, 4);
  read_all(in, &flags, 4);
  if (n < 0 || g < 1 || g > DASO_MAX_G || P < 0 || P > DASO_MAX_P || nb < 1) return 2;
  daso_bucket* buckets = (daso_bucket*)calloc((size_t)nb, sizeof(daso_bucket));
  read_all(in, buckets, (size_t)nb * sizeof(daso_bucket));

  const size_t f32 = (size_t)n * 4, b16 = (size_t)n * 2;
  /* pinned staging buffer: transfers go through memory allocated as pinned */
  void* host = NULL;
  HIP_OK(hipHostMalloc(&host, f32 > 0 ? f32 : 16, hipHostMallocDefault));
  const float* grads[DASO_MAX_G];
  const uint16_t* stale[DASO_MAX_P];
  for (int r = 0; r < g; ++r) {
    read_all(in, host, f32);
    grads[r] = (const float*)upload(host, f32);
  }
  read_all(in, host, f32);
  float* params = (float*)upload(host, f32);
  read_all(in, host, f32);
  float* momentum = (float*)upload(host, f32);
  for (int i = 0; i < P; ++i) {
    read_all(in, host, b16);
    stale[i] = (const uint16_t*)upload(host, b16);
  }
  fclose(in);
  uint16_t* wire = (uint16_t*)device_alloc(b16);
  daso_bucket_stats* stats = (daso_bucket_stats*)device_alloc((size_t)nb * sizeof(daso_bucket_stats));

  hipStream_t stream;
  HIP_OK(hipStreamCreate(&stream));
  daso_sync_args a;
  memset(&a, 0, sizeof(a));
  a.n = n;
  a.g = g;
  a.P = P;
  a.grads = grads;
  a.stale = stale;
  a.params = params;
  a.momentum = momentum;
  a.wire = wire;
  a.buckets = buckets;
  a.nbuckets = nb;
  a.lr = lr;
  a.mu = mu;
  a.weight_decay = wd;
  a.flags = flags;
  a.stats = stats;
  const int rc = daso_fused_sync_step(&a, stream);
  if (rc != DASO_OK) {
    fprintf(stderr, "daso_fused_sync_step: %s\n", daso_status_string(rc));
    return 4;
  }
  HIP_OK(hipStreamSynchronize(stream));

  FILE* out = fopen(argv[2], "wb");
  if (!out) return 2;
  HIP_OK(hipMemcpy(host, params, f32, hipMemcpyDeviceToHost));
  fwrite(host, 1, f32, out);
  HIP_OK(hipMemcpy(host, momentum, f32, hipMemcpyDeviceToHost));
  fwrite(host, 1, f32, out);
  HIP_OK(hipMemcpy(host, wire, b16, hipMemcpyDeviceToHost));
  fwrite(host, 1, b16, out);
  const size_t sbytes = (size_t)nb * sizeof(daso_bucket_stats);
  void* hs = NULL;
  HIP_OK(hipHostMalloc(&hs, sbytes, hipHostMallocDefault));
  HIP_OK(hipMemcpy(hs, stats, sbytes, hipMemcpyDeviceToHost));
  fwrite(hs, 1, sbytes, out);
  fclose(out);
  printf("ok n=%lld g=%d P=%d buckets=%d abi=%d\n", (long long)n, g, P, nb, daso_abi_version());
  return 0;
}
