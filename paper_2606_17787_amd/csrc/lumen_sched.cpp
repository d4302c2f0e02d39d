// Checkpoint placement and recovery scheduling; specified in
// include/lumen_sched.h.

#include <stdint.h>

#include <algorithm>
#include <map>
#include <new>
#include <utility>
#include <vector>

#include "lumen_kv_ckpt.h"
#include "lumen_sched.h"

namespace {

struct WorkerState {
  int64_t budget = 0;
  double q = 0.0;
  int64_t queued = 0, running = 0;
  bool alive = true;
  int64_t used = 0;      // reserved bytes
  int64_t held_sum = 0;  // sum of the reserved bytes of held checkpoints
  std::map<int64_t, int64_t> held;  // request -> reserved bytes
};

struct RequestState {
  int32_t serving = -1;
  int64_t reserved = 0;
  int32_t holder = -1;
  int64_t persisted = 0;
};

}  // namespace

struct lumen_sched {
  std::vector<WorkerState> w;
  double bw = 1.0, lambda = 1.0;
  std::map<int64_t, RequestState> req;  // ordered: dispatch by request id
};

namespace {

void drop_checkpoint(lumen_sched *s, int64_t id, RequestState &r) {
  if (r.holder < 0) return;
  WorkerState &h = s->w[r.holder];
  auto it = h.held.find(id);
  if (it != h.held.end()) {
    h.used -= it->second;
    h.held_sum -= it->second;
    h.held.erase(it);
  }
  r.holder = -1;
}

}  // namespace

extern "C" {

lumen_sched *lumen_sched_create(int32_t num_workers,
                                const int64_t *budget_bytes,
                                double h2d_bytes_per_s, double lambda) {
  if (num_workers < 1 || !budget_bytes || !(h2d_bytes_per_s > 0) ||
      !(lambda >= 0))
    return nullptr;
  lumen_sched *s = new (std::nothrow) lumen_sched;
  if (!s) return nullptr;
  try {
    s->w.resize(size_t(num_workers));
  } catch (const std::bad_alloc &) {
    delete s;
    return nullptr;
  }
  for (int32_t i = 0; i < num_workers; ++i) s->w[i].budget = budget_bytes[i];
  s->bw = h2d_bytes_per_s;
  s->lambda = lambda;
  return s;
}

void lumen_sched_destroy(lumen_sched *s) { delete s; }

int lumen_sched_set_worker(lumen_sched *s, int32_t worker,
                           double queueing_delay, int64_t queued,
                           int64_t running) {
  if (!s || worker < 0 || size_t(worker) >= s->w.size() || queued < 0 ||
      running < 0)
    return LUMEN_ERR_INVALID_ARG;
  WorkerState &w = s->w[worker];
  w.q = queueing_delay;
  w.queued = queued;
  w.running = running;
  return LUMEN_OK;
}

int lumen_sched_place(lumen_sched *s, int64_t request, int32_t serving,
                      int64_t reserved_bytes, int32_t *holder) {
  if (!s || !holder || serving < 0 || size_t(serving) >= s->w.size() ||
      reserved_bytes < 0 || s->req.count(request))
    return LUMEN_ERR_INVALID_ARG;
  int32_t best = -1;
  double best_score = 0.0;
  for (size_t i = 0; i < s->w.size(); ++i) {
    const WorkerState &w = s->w[i];
    if (int32_t(i) == serving || !w.alive) continue;
    if (w.budget - w.used < reserved_bytes) continue;  // not in F(r)
    // p_w(r): mean reserved footprint after adding r, over the bandwidth
    const double mean = double(w.held_sum + reserved_bytes) /
                        double(int64_t(w.held.size()) + 1);
    const double score = w.q + s->lambda * (mean / s->bw);
    if (best < 0 || score < best_score) {
      best = int32_t(i);
      best_score = score;
    }
  }
  RequestState r;
  r.serving = serving;
  r.reserved = reserved_bytes;
  r.holder = best;
  // Both insertions allocate; the second one failing undoes the first, so
  // a failed placement changes nothing.
  try {
    auto ins = s->req.emplace(request, r).first;
    if (best >= 0) {
      try {
        s->w[best].held.emplace(request, reserved_bytes);
      } catch (const std::bad_alloc &) {
        s->req.erase(ins);
        throw;
      }
    }
  } catch (const std::bad_alloc &) {
    return LUMEN_ERR_CAPACITY;
  }
  if (best >= 0) {
    WorkerState &h = s->w[best];
    h.used += reserved_bytes;
    h.held_sum += reserved_bytes;
  }
  *holder = best;
  return LUMEN_OK;
}

int lumen_sched_set_persisted(lumen_sched *s, int64_t request,
                              int64_t bytes) {
  if (!s || bytes < 0) return LUMEN_ERR_INVALID_ARG;
  auto it = s->req.find(request);
  if (it == s->req.end()) return LUMEN_ERR_INVALID_ARG;
  it->second.persisted = bytes;
  return LUMEN_OK;
}

int lumen_sched_release(lumen_sched *s, int64_t request) {
  if (!s) return LUMEN_ERR_INVALID_ARG;
  auto it = s->req.find(request);
  if (it == s->req.end()) return LUMEN_ERR_INVALID_ARG;
  drop_checkpoint(s, request, it->second);
  s->req.erase(it);
  return LUMEN_OK;
}

int lumen_sched_holder(lumen_sched *s, int64_t request, int32_t *holder) {
  if (!s || !holder) return LUMEN_ERR_INVALID_ARG;
  auto it = s->req.find(request);
  if (it == s->req.end()) return LUMEN_ERR_INVALID_ARG;
  *holder = it->second.holder;
  return LUMEN_OK;
}

int64_t lumen_sched_reserved(lumen_sched *s, int32_t worker) {
  if (!s || worker < 0 || size_t(worker) >= s->w.size())
    return LUMEN_ERR_INVALID_ARG;
  return s->w[worker].used;
}

int lumen_sched_recover(lumen_sched *s, const int32_t *failed,
                        int32_t num_failed, int64_t *out_request,
                        int32_t *out_worker, int8_t *out_reuse,
                        int64_t max_out, int64_t *num_out) {
  if (!s || num_failed < 0 || (num_failed > 0 && !failed) || !num_out)
    return LUMEN_ERR_INVALID_ARG;
  const size_t nw = s->w.size();
  for (int32_t k = 0; k < num_failed; ++k)
    if (failed[k] < 0 || size_t(failed[k]) >= nw) return LUMEN_ERR_INVALID_ARG;
  int64_t count = 0;
  try {
    // Decide everything first, on local copies: nothing in the scheduler
    // changes until every allocation has succeeded.
    std::vector<char> dead(nw, 0);
    for (int32_t k = 0; k < num_failed; ++k) dead[failed[k]] = 1;
    for (size_t i = 0; i < nw; ++i)
      if (!s->w[i].alive) dead[i] = 1;
    for (auto &kv : s->req)
      if (dead[kv.second.serving]) ++count;
    if (count > max_out || (count > 0 && (!out_request || !out_worker ||
                                          !out_reuse)))
      return LUMEN_ERR_INVALID_ARG;
    // Survivors, and the interrupted requests in increasing id.  A
    // checkpoint is usable only if its holder survives: the failed
    // workers' checkpoints are lost with them.
    std::vector<int32_t> alive;
    for (size_t i = 0; i < nw; ++i)
      if (!dead[i]) alive.push_back(int32_t(i));
    std::vector<int64_t> ids;
    std::vector<const RequestState *> rs;
    for (auto &kv : s->req)
      if (dead[kv.second.serving]) {
        ids.push_back(kv.first);
        rs.push_back(&kv.second);
      }
    std::vector<int64_t> extra(nw, 0);  // newly assigned interrupted requests
    std::vector<int32_t> where(ids.size(), -1);
    std::vector<char> reuse(ids.size(), 0);
    auto load = [&](int32_t i) {
      return s->w[i].queued + s->w[i].running + extra[i];
    };
    auto least_loaded = [&]() {
      int32_t best = -1;
      for (int32_t i : alive)
        if (best < 0 || load(i) < load(best)) best = i;
      return best;
    };
    // Initial dispatch: to the surviving holder, else the least loaded.
    for (size_t k = 0; k < ids.size(); ++k) {
      const RequestState &r = *rs[k];
      if (r.holder >= 0 && !dead[r.holder]) {
        where[k] = r.holder;
        reuse[k] = 1;
      } else {
        where[k] = least_loaded();
        reuse[k] = 0;
      }
      if (where[k] >= 0) ++extra[where[k]];
    }

    // Average-based request-count rebalancing.  Each worker keeps its
    // assigned interrupted requests ordered by (usable checkpoint size,
    // request id), recomputed ones counting size 0, so the next one to
    // shed is always its first.
    if (!alive.empty() && !ids.empty()) {
      int64_t total = 0;
      for (int32_t i : alive) total += load(i);
      const double avg = double(total) / double(alive.size());
      std::vector<std::vector<std::pair<int64_t, size_t>>> cand(nw);
      for (size_t k = 0; k < ids.size(); ++k)
        if (where[k] >= 0)
          cand[where[k]].push_back({reuse[k] ? rs[k]->persisted : 0, k});
      for (auto &c : cand) std::sort(c.rbegin(), c.rend());  // smallest last
      std::vector<int32_t> order(alive);
      while (true) {
        const int32_t dst = least_loaded();
        std::stable_sort(order.begin(), order.end(),
                         [&](int32_t a, int32_t b) {
                           return load(a) > load(b);
                         });
        bool moved = false;
        for (int32_t src : order) {
          if (!(double(load(src)) > avg)) break;
          if (load(dst) + 1 >= load(src) || cand[src].empty()) continue;
          const size_t pick = cand[src].back().second;
          cand[src].pop_back();
          --extra[src];
          ++extra[dst];
          where[pick] = dst;
          reuse[pick] = 0;
          // a moved request is recomputed: size 0, ahead of dst's others
          auto &d = cand[dst];
          d.insert(std::upper_bound(d.begin(), d.end(),
                                    std::make_pair(int64_t(0), pick),
                                    [](const std::pair<int64_t, size_t> &a,
                                       const std::pair<int64_t, size_t> &b) {
                                      return a > b;
                                    }),
                   {int64_t(0), pick});
          moved = true;
          break;
        }
        if (!moved) break;
      }
    }

    // Commit (allocates nothing).  The failed workers and their
    // checkpoints go; recovered requests run where dispatched and their old
    // checkpoints go too.  With no survivor at all a request stays on its
    // failed worker and is reported again (worker -1) by the next recovery
    // event.
    for (size_t i = 0; i < nw; ++i) {
      if (!dead[i]) continue;
      WorkerState &w = s->w[i];
      w.alive = false;
      for (auto &h : w.held) {
        auto it = s->req.find(h.first);
        if (it != s->req.end()) it->second.holder = -1;
      }
      w.held.clear();
      w.used = 0;
      w.held_sum = 0;
    }
    for (size_t k = 0; k < ids.size(); ++k) {
      RequestState &r = s->req.find(ids[k])->second;
      drop_checkpoint(s, ids[k], r);
      if (where[k] >= 0) r.serving = where[k];
      r.persisted = 0;
      out_request[k] = ids[k];
      out_worker[k] = where[k];
      out_reuse[k] = reuse[k];
    }
    *num_out = int64_t(ids.size());
  } catch (const std::bad_alloc &) {
    return LUMEN_ERR_CAPACITY;
  }
  return LUMEN_OK;
}

}  // extern "C"
