// Step-tag tracker: when may the controller stop the normal ranks, and from
// which step's state does recovery resume (Section III-E: its parts on the
// step to resume from and on when to stop the normal processes).
//
// Every training process sets its tag to i when forward of step i starts,
// to -1 when its optimizer step starts, and to i+1 when the optimizer step
// ends; monitors report the tag with each heartbeat (Section III-C).  A
// barrier merged into the gradient all-reduce keeps all ranks in one phase:
// after a failure in forward/backward every normal rank stays at i, after a
// failure in the optimizer step every normal rank ends at i+1.  So once every
// normal rank reports the same tag T >= 0, stopping is safe and the replicas
// hold the state at the start of step T.
//
// Readings (the paper is silent on them):
//  * a tag describes the rank only as of its heartbeat, so the decision uses
//    a normal rank's tag only if it was reported after the last failure was
//    detected; an older report may show i from a rank that has since entered
//    its optimizer step, which would restore the wrong step;
//  * a failure is detected when a monitor or device plugin reports it, or
//    when the rank has been silent for longer than the timeout (detection
//    time = last heartbeat + timeout: the rank would have reported within one
//    heartbeat period, shorter than the timeout, had it been alive);
//  * under the barrier, fresh tags of normal ranks are either all i or a mix
//    of -1 and i+1; any other mix is inconsistent;
//  * if every rank of some data-parallel group has failed, no replica exists
//    and the fallback is a checkpoint (Section III-G).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <limits>
#include <new>
#include <vector>

#include "flashrestore.h"

struct fr_tracker {
  uint32_t n_ranks = 0;
  double timeout_s = 0;
  double created_s = 0;
  std::vector<uint32_t> group;     // data-parallel group of each rank
  std::vector<int64_t> tag;        // last reported tag
  std::vector<uint8_t> reported;   // any heartbeat yet
  std::vector<double> last_seen;   // time of the last heartbeat
  std::vector<uint8_t> failed;     // failure reported by a monitor or device plugin
  std::vector<double> failed_at;   // time of that report
};

namespace {

bool is_failed(const fr_tracker* t, uint32_t r, double now) {
  if (t->failed[r]) return true;
  const double seen = t->reported[r] ? t->last_seen[r] : t->created_s;
  return now - seen > t->timeout_s;
}

// When the failure of a failed rank was detected.
double detected_at(const fr_tracker* t, uint32_t r) {
  const double seen = t->reported[r] ? t->last_seen[r] : t->created_s;
  const double by_timeout = seen + t->timeout_s;
  return t->failed[r] ? std::min(t->failed_at[r], by_timeout) : by_timeout;
}

}  // namespace

extern "C" int fr_tracker_create(uint32_t n_ranks, const uint32_t* dp_group, double timeout_s,
                                 double now_s, fr_tracker** out) {
  if (!out || n_ranks == 0 || !(timeout_s > 0) || !std::isfinite(timeout_s) || !std::isfinite(now_s))
    return FR_E_INVAL;
  if (dp_group)
    for (uint32_t r = 0; r < n_ranks; r++)
      if (dp_group[r] >= n_ranks) return FR_E_INVAL;  // group ids are 0 .. n_ranks - 1
  fr_tracker* t = new (std::nothrow) fr_tracker();
  if (!t) return FR_E_NOMEM;
  try {
    t->n_ranks = n_ranks;
    t->timeout_s = timeout_s;
    t->created_s = now_s;
    t->group.assign(n_ranks, 0);
    if (dp_group) t->group.assign(dp_group, dp_group + n_ranks);
    t->tag.assign(n_ranks, 0);
    t->reported.assign(n_ranks, 0);
    t->last_seen.assign(n_ranks, now_s);
    t->failed.assign(n_ranks, 0);
    t->failed_at.assign(n_ranks, 0.0);
  } catch (const std::bad_alloc&) {
    delete t;
    return FR_E_NOMEM;
  }
  *out = t;
  return FR_OK;
}

extern "C" int fr_tracker_destroy(fr_tracker* t) {
  delete t;
  return FR_OK;
}

extern "C" int fr_tracker_heartbeat(fr_tracker* t, uint32_t rank, int64_t step_tag, double now_s) {
  if (!t || rank >= t->n_ranks || step_tag < -1 || !std::isfinite(now_s)) return FR_E_INVAL;
  t->tag[rank] = step_tag;
  t->reported[rank] = 1;
  t->last_seen[rank] = now_s;
  return FR_OK;
}

extern "C" int fr_tracker_report_failure(fr_tracker* t, uint32_t rank, double now_s) {
  if (!t || rank >= t->n_ranks || !std::isfinite(now_s)) return FR_E_INVAL;
  if (!t->failed[rank]) {
    t->failed[rank] = 1;
    t->failed_at[rank] = now_s;
  }
  return FR_OK;
}

extern "C" int fr_tracker_decide(const fr_tracker* t, double now_s, fr_decision* out) {
  if (!t || !out || !std::isfinite(now_s)) return FR_E_INVAL;
  fr_decision d{};
  d.resume_step = -1;
  d.action = FR_ACT_CONTINUE;
  // failed ranks and groups left without a live replica
  std::vector<uint32_t> live_in_group;
  try {
    uint32_t max_group = 0;
    for (uint32_t r = 0; r < t->n_ranks; r++) max_group = std::max(max_group, t->group[r]);
    live_in_group.assign(size_t(max_group) + 1, 0);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  for (uint32_t r = 0; r < t->n_ranks; r++) {
    if (is_failed(t, r, now_s)) d.n_failed++;
    else live_in_group[t->group[r]]++;
  }
  if (d.n_failed == 0) {
    d.action = FR_ACT_CONTINUE;
    *out = d;
    return FR_OK;
  }
  for (uint32_t r = 0; r < t->n_ranks; r++) {
    if (live_in_group[t->group[r]] == 0) {
      d.action = FR_ACT_CHECKPOINT_FALLBACK;
      *out = d;
      return FR_OK;
    }
  }
  // fresh tags of the normal ranks: reported after the last detection
  double fresh_after = -std::numeric_limits<double>::infinity();
  for (uint32_t r = 0; r < t->n_ranks; r++)
    if (is_failed(t, r, now_s)) fresh_after = std::max(fresh_after, detected_at(t, r));
  int64_t lo = std::numeric_limits<int64_t>::max(), hi = std::numeric_limits<int64_t>::min();
  for (uint32_t r = 0; r < t->n_ranks; r++) {
    if (is_failed(t, r, now_s)) continue;
    // silent since the failure, or inside an optimizer step
    if (!t->reported[r] || t->last_seen[r] < fresh_after || t->tag[r] < 0) {
      d.n_waiting++;
      continue;
    }
    lo = std::min(lo, t->tag[r]);
    hi = std::max(hi, t->tag[r]);
  }
  if (d.n_waiting > 0) {
    d.action = FR_ACT_WAIT;
  } else if (lo == hi) {
    d.action = FR_ACT_STOP_AND_RESTORE;
    d.resume_step = lo;
  } else {
    d.action = FR_ACT_INCONSISTENT;
  }
  *out = d;
  return FR_OK;
}

extern "C" int fr_tracker_failed_ranks(const fr_tracker* t, double now_s, uint32_t* ranks,
                                       uint32_t cap, uint32_t* n_failed) {
  if (!t || !n_failed || (cap && !ranks)) return FR_E_INVAL;
  uint32_t n = 0;
  for (uint32_t r = 0; r < t->n_ranks; r++) {
    if (!is_failed(t, r, now_s)) continue;
    if (n < cap) ranks[n] = r;
    n++;
  }
  *n_failed = n;
  return n > cap ? FR_E_RANGE : FR_OK;
}

// Donor choice (Section III-D stage 3: the controller determines the normal
// device whose state restores each new one): for every failed rank, a live
// rank of its data-parallel group; the failed ranks of a group are spread
// over its live ranks in rank order so that no donor serves two while another
// serves none.
extern "C" int fr_tracker_donors(const fr_tracker* t, double now_s, int32_t* donor) {
  if (!t || !donor) return FR_E_INVAL;
  std::vector<std::vector<uint32_t>> live;
  std::vector<uint32_t> next;
  try {
    uint32_t max_group = 0;
    for (uint32_t r = 0; r < t->n_ranks; r++) max_group = std::max(max_group, t->group[r]);
    live.resize(size_t(max_group) + 1);
    next.assign(size_t(max_group) + 1, 0);
    for (uint32_t r = 0; r < t->n_ranks; r++)
      if (!is_failed(t, r, now_s)) live[t->group[r]].push_back(r);
  } catch (const std::bad_alloc&) {
    return FR_E_NOMEM;
  }
  for (uint32_t r = 0; r < t->n_ranks; r++) {
    donor[r] = -1;
    if (!is_failed(t, r, now_s)) continue;
    const std::vector<uint32_t>& g = live[t->group[r]];
    if (g.empty()) continue;
    donor[r] = int32_t(g[next[t->group[r]]++ % g.size()]);
  }
  return FR_OK;
}
