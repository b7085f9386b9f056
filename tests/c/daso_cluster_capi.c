/* A plain C program that runs DASO end to end through the C ABI alone: one
 * native schedule controller per simulated node decides every batch (phase,
 * exchange, merge), daso_fused_sync_step does each node's step, and the
 * exchanges between the nodes are simulated as device-to-device copies of their
 * bf16 wires that are handed over S batches later (blocking ones at once, then
 * averaged with daso_global_merge and S = 0).  Every node takes the role of
 * its group's member (group_count = 1), as in a cluster with one GPU per node.
 * Used by the GPU tests to show the native controller and kernels work without
 * Python; the results are compared with an oracle simulation.
 *
 * usage: daso_cluster_capi <input> <output>
 * input:  int32 nodes, g, n, nspans, epochs, warmup, cooldown, batches, B, W, patience;
 *         double plateau_rel_tol; float lr, mu;
 *         nspans x {int64 start, int64 numel}; epochs x double loss;
 *         nodes x n float initial params;
 *         then, batch by batch and node by node, g x n float gradients
 * output: nodes x n float params, nodes x n float momentum,
 *         epochs x batches x int32 actions (as planned for node 0)
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

#define DASO_OK_OR_DIE(call)                                                \
  do {                                                                      \
    int s_ = (call);                                                        \
    if (s_ != DASO_OK) {                                                    \
      fprintf(stderr, "%s failed: %s\n", #call, daso_status_string(s_));    \
      exit(4);                                                              \
    }                                                                       \
  } while (0)

enum { kMaxNodes = 16, kMaxSpans = 64 };

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

int main(int argc, char** argv) {
  if (argc != 3) {
    fprintf(stderr, "usage: %s <input> <output>\n", argv[0]);
    return 2;
  }
  FILE* in = fopen(argv[1], "rb");
  if (!in) return 2;
  int32_t hdr[11];
  double tol;
  float lr, mu;
  read_all(in, hdr, sizeof hdr);
  read_all(in, &tol, 8);
  read_all(in, &lr, 4);
  read_all(in, &mu, 4);
  const int nodes = hdr[0], g = hdr[1], n = hdr[2], nspans = hdr[3];
  const int epochs = hdr[4], batches = hdr[7];
  if (nodes < 1 || nodes > kMaxNodes || g < 1 || g > DASO_MAX_G || n < 1 || nspans < 1 || nspans > kMaxSpans ||
      epochs < 1 || batches < 1)
    return 2;

  int64_t spans[kMaxSpans][2];
  read_all(in, spans, (size_t)nspans * 16);
  double* losses = (double*)malloc((size_t)epochs * sizeof(double));
  read_all(in, losses, (size_t)epochs * sizeof(double));

  const size_t f32 = (size_t)n * 4, b16 = (size_t)n * 2;
  float* host = NULL;
  HIP_OK(hipHostMalloc((void**)&host, f32, hipHostMallocDefault));

  /* one controller and one set of buffers per simulated node */
  daso_schedule* sched[kMaxNodes];
  float* params[kMaxNodes];
  float* momentum[kMaxNodes];
  uint16_t* wire[kMaxNodes];
  float* grads[kMaxNodes][DASO_MAX_G];
  daso_schedule_config cfg;
  cfg.total_epochs = epochs;
  cfg.warmup_epochs = hdr[5];
  cfg.cooldown_epochs = hdr[6];
  cfg.batches_per_epoch = batches;
  cfg.B_init = hdr[8];
  cfg.W_init = hdr[9];
  cfg.group_count = 1;
  cfg.local_rank = 0;
  cfg.patience = hdr[10];
  cfg.plateau_rel_tol = tol;
  for (int k = 0; k < nodes; ++k) {
    DASO_OK_OR_DIE(daso_schedule_create(&cfg, &sched[k]));
    read_all(in, host, f32);
    params[k] = (float*)device_alloc(f32);
    HIP_OK(hipMemcpy(params[k], host, f32, hipMemcpyHostToDevice));
    momentum[k] = (float*)device_alloc(f32);
    HIP_OK(hipMemset(momentum[k], 0, f32));
    wire[k] = (uint16_t*)device_alloc(b16);
    for (int r = 0; r < g; ++r) grads[k][r] = (float*)device_alloc(f32);
  }

  /* copies sent after batch t, handed over S batches later */
  const int steps = epochs * batches;
  uint16_t** sent = (uint16_t**)calloc((size_t)steps * (size_t)nodes, sizeof(uint16_t*));
  int32_t* actions = (int32_t*)calloc((size_t)steps, sizeof(int32_t));
  daso_bucket buckets[kMaxSpans];

  for (int t = 0; t < steps; ++t) {
    daso_batch_plan plan[kMaxNodes];
    for (int k = 0; k < nodes; ++k) {
      if (daso_schedule_next(sched[k], &plan[k]) != 1) {
        fprintf(stderr, "schedule ended early at batch %d\n", t);
        return 5;
      }
      if (plan[k].actions != plan[0].actions || plan[k].S != plan[0].S) {
        fprintf(stderr, "nodes disagree at batch %d\n", t);
        return 5;
      }
    }
    const uint32_t acts = plan[0].actions;
    actions[t] = (int32_t)acts;
    const int merge = (acts & DASO_ACT_MERGE) != 0;
    const int S = merge ? plan[0].S : 0;
    if (merge) {
      if (S < 1 || S > t) {
        fprintf(stderr, "bad staleness %d at batch %d\n", S, t);
        return 5;
      }
      for (int k = 0; k < nodes; ++k)
        if (sent[(size_t)(t - S) * (size_t)nodes + (size_t)k] == NULL) {
          fprintf(stderr, "nothing was sent at batch %d for the merge at batch %d\n", t - S, t);
          return 5;
        }
    }
    for (int b = 0; b < nspans; ++b) {
      buckets[b].start = spans[b][0];
      buckets[b].numel = spans[b][1];
      buckets[b].S = S;
      buckets[b].reserved = 0;
    }
    for (int k = 0; k < nodes; ++k) {
      for (int r = 0; r < g; ++r) {
        read_all(in, host, f32);
        HIP_OK(hipMemcpy(grads[k][r], host, f32, hipMemcpyHostToDevice));
      }
      daso_sync_args a;
      memset(&a, 0, sizeof a);
      a.n = n;
      a.g = g;
      a.P = merge ? nodes : 0;
      a.grads = (const float* const*)grads[k];
      a.stale = merge ? (const uint16_t* const*)&sent[(size_t)(t - S) * (size_t)nodes] : NULL;
      a.params = params[k];
      a.momentum = momentum[k];
      a.wire = (acts & (DASO_ACT_SEND | DASO_ACT_BLOCKING)) ? wire[k] : NULL;
      a.buckets = buckets;
      a.nbuckets = nspans;
      a.lr = lr;
      a.mu = mu;
      DASO_OK_OR_DIE(daso_fused_sync_step(&a, 0));
    }
    if (acts & DASO_ACT_BLOCKING) {
      /* blocking exchange: every node averages all the wires at once (S = 0) */
      for (int b = 0; b < nspans; ++b) buckets[b].S = 0;
      for (int k = 0; k < nodes; ++k)
        DASO_OK_OR_DIE(daso_global_merge(params[k], (const uint16_t* const*)wire, nodes, buckets, nspans, NULL,
                                         n, 0));
    }
    if (acts & DASO_ACT_SEND) {
      for (int k = 0; k < nodes; ++k) {
        uint16_t* copy = (uint16_t*)device_alloc(b16);
        HIP_OK(hipMemcpy(copy, wire[k], b16, hipMemcpyDeviceToDevice));
        sent[(size_t)t * (size_t)nodes + (size_t)k] = copy;
      }
    }
    if (plan[0].batch == batches - 1)
      for (int k = 0; k < nodes; ++k) DASO_OK_OR_DIE(daso_schedule_end_epoch(sched[k], losses[plan[0].epoch]));
  }
  HIP_OK(hipDeviceSynchronize());

  FILE* out = fopen(argv[2], "wb");
  if (!out) return 2;
  for (int k = 0; k < nodes; ++k) {
    HIP_OK(hipMemcpy(host, params[k], f32, hipMemcpyDeviceToHost));
    fwrite(host, 1, f32, out);
  }
  for (int k = 0; k < nodes; ++k) {
    HIP_OK(hipMemcpy(host, momentum[k], f32, hipMemcpyDeviceToHost));
    fwrite(host, 1, f32, out);
  }
  fwrite(actions, sizeof(int32_t), (size_t)steps, out);
  fclose(out);
  for (int k = 0; k < nodes; ++k) daso_schedule_destroy(sched[k]);
  return 0;
}
