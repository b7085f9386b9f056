// Phase and exchange-schedule controller of DASO (host only), declared in daso.h.
#include <cmath>
#include <map>
#include <new>

#include "daso.h"

namespace {

struct Pending {
  int32_t group;  // group whose member merges the copies
  int32_t S;      // batches the copies are late
};

}  // namespace

struct daso_schedule {
  daso_schedule_config cfg;
  int32_t W0 = 1;           // initial W after defaulting
  int32_t B = 1, W = 1;     // values in force
  int32_t nextB = 1, nextW = 1;  // values for the next epoch
  int64_t step = 0;         // next step to plan
  int32_t since_sync = 0;   // cycling batches since the last exchange started (or cycling began)
  int64_t exchanges = 0;    // exchanges started so far (blocking and non-blocking): rotation counter
  bool awaiting_loss = false;
  bool have_best = false;
  double best = 0.0;
  int32_t bad_epochs = 0;
  std::map<int64_t, Pending> pending;  // by the step after which the copies arrive

  int32_t phase_of(int32_t epoch) const {
    if (epoch < cfg.warmup_epochs) return DASO_PHASE_WARMUP;
    if (epoch >= cfg.total_epochs - cfg.cooldown_epochs) return DASO_PHASE_COOLDOWN;
    return DASO_PHASE_CYCLING;
  }

  // last step of the cycling phase (-1 when there is none)
  int64_t last_cycling_step() const {
    const int32_t first_cool = cfg.total_epochs - cfg.cooldown_epochs;
    if (first_cool <= cfg.warmup_epochs) return -1;
    return int64_t(first_cool) * cfg.batches_per_epoch - 1;
  }
};

extern "C" {

int daso_schedule_create(const daso_schedule_config* c, daso_schedule** out) {
  if (c == nullptr || out == nullptr) return DASO_EINVAL;
  if (c->total_epochs < 1 || c->warmup_epochs < 0 || c->cooldown_epochs < 0 ||
      int64_t(c->warmup_epochs) + c->cooldown_epochs > c->total_epochs || c->batches_per_epoch < 1 ||
      c->B_init < 1 || c->W_init < 0 || c->W_init > c->B_init || c->group_count < 1 || c->local_rank < 0 ||
      c->local_rank >= c->group_count || c->patience < 1 || !(c->plateau_rel_tol >= 0.0) ||
      !std::isfinite(c->plateau_rel_tol))
    return DASO_EINVAL;
  daso_schedule* s = new (std::nothrow) daso_schedule();
  if (s == nullptr) return DASO_EINVAL;
  s->cfg = *c;
  s->W0 = c->W_init > 0 ? c->W_init : (c->B_init / 4 > 1 ? c->B_init / 4 : 1);
  s->B = s->nextB = c->B_init;
  s->W = s->nextW = s->W0;
  *out = s;
  return DASO_OK;
}

void daso_schedule_destroy(daso_schedule* s) { delete s; }

int daso_schedule_next(daso_schedule* s, daso_batch_plan* plan) {
  if (s == nullptr || plan == nullptr) return DASO_EINVAL;
  if (s->awaiting_loss) return DASO_EINVAL;
  const daso_schedule_config& c = s->cfg;
  const int64_t total = int64_t(c.total_epochs) * c.batches_per_epoch;
  if (s->step >= total) return 0;

  const int32_t epoch = static_cast<int32_t>(s->step / c.batches_per_epoch);
  const int32_t batch = static_cast<int32_t>(s->step % c.batches_per_epoch);
  if (batch == 0) {  // values decided at the end of the previous epoch take effect
    if (s->nextB != s->B || s->nextW != s->W) s->since_sync = 0;
    s->B = s->nextB;
    s->W = s->nextW;
  }
  const int32_t phase = s->phase_of(epoch);

  daso_batch_plan p;
  p.step = s->step;
  p.epoch = epoch;
  p.batch = batch;
  p.phase = phase;
  p.B = s->B;
  p.W = s->W;
  p.actions = 0;
  p.S = -1;
  p.sync_group = -1;
  p.merge_group = -1;

  // copies that arrive after this batch
  const auto arrived = s->pending.find(s->step);
  if (arrived != s->pending.end()) {
    const Pending q = arrived->second;
    s->pending.erase(arrived);
    p.merge_group = q.group;
    p.S = q.S;
    p.actions |= (q.group == c.local_rank) ? DASO_ACT_MERGE : DASO_ACT_RECV_BCAST;
  }

  if (phase == DASO_PHASE_CYCLING) {
    ++s->since_sync;
    if (s->since_sync >= s->B) {
      s->since_sync = 0;
      // an exchange starts unless its copies would land after the cycling
      // phase or in a batch where another exchange's copies land
      const int64_t due = s->step + s->W;
      if (due <= s->last_cycling_step() && s->pending.count(due) == 0) {
        const int32_t grp = static_cast<int32_t>(s->exchanges % c.group_count);
        ++s->exchanges;
        s->pending.emplace(due, Pending{grp, s->W});
        p.sync_group = grp;
        if (grp == c.local_rank) p.actions |= DASO_ACT_SEND;
      }
    }
  } else {
    const int32_t grp = static_cast<int32_t>(s->exchanges % c.group_count);
    ++s->exchanges;
    p.sync_group = grp;
    p.merge_group = grp;
    p.S = 0;
    p.actions |= (grp == c.local_rank) ? DASO_ACT_BLOCKING : DASO_ACT_RECV_BCAST;
  }

  if (batch == c.batches_per_epoch - 1) s->awaiting_loss = true;
  ++s->step;
  *plan = p;
  return 1;
}

int daso_schedule_end_epoch(daso_schedule* s, double loss) {
  if (s == nullptr || !s->awaiting_loss || std::isnan(loss)) return DASO_EINVAL;
  s->awaiting_loss = false;
  const daso_schedule_config& c = s->cfg;
  const int32_t epoch = static_cast<int32_t>((s->step - 1) / c.batches_per_epoch);
  if (s->phase_of(epoch) != DASO_PHASE_CYCLING) return DASO_OK;
  if (!s->have_best || loss < s->best - c.plateau_rel_tol * std::fabs(s->best)) {
    s->have_best = true;
    s->best = loss;
    s->bad_epochs = 0;
    return DASO_OK;
  }
  if (++s->bad_epochs < c.patience) return DASO_OK;
  s->bad_epochs = 0;
  if (s->B == 1 && s->W == 1) {
    s->nextB = c.B_init;
    s->nextW = s->W0;
  } else {
    s->nextB = s->B / 2 > 1 ? s->B / 2 : 1;
    s->nextW = s->W / 2 > 1 ? s->W / 2 : 1;
  }
  return DASO_OK;
}

}  // extern "C"
