// Schedule-side pieces of ReCycle on the host: Failure Normalization
// (section 4.2.1, Algorithm 1) and a unit-slot schedule simulator of DP x PP
// workers running 1F1B with re-routed micro-batches (section 3.1), Decoupled
// BackProp (section 3.2) and the Staggered Optimizer (section 3.3).  The
// simulator's per-worker op lists are the Planner-style op lists a stage
// handle executes.
#include <algorithm>
#include <climits>
#include <cstring>
#include <map>
#include <set>
#include <string>
#include <vector>

#include "recycle_stage.h"

rc_status rc_set_error(rc_status s, const std::string& msg);  // defined in stage.cpp

namespace {

// Extra slots for f failures on one stage: re-routed work (3 slots per
// micro-batch: F, B_input, B_weight) minus the bubbles of the DP - f
// surviving peers (3 (PP - 1) each); never negative.
long long norm_cost(int dp, int pp, int mb, int f) {
  if (f <= 0) return 0;
  const long long c = 3LL * mb * f - 3LL * (dp - f) * (pp - 1);
  return c > 0 ? c : 0;
}

struct Key {  // one micro-batch at one stage in one iteration
  int it, i, j, k;
  bool operator<(const Key& o) const {
    if (it != o.it) return it < o.it;
    if (i != o.i) return i < o.i;
    if (k != o.k) return k < o.k;
    return j < o.j;
  }
};

}  // namespace

extern "C" {

rc_status rc_failure_normalization(int32_t dp, int32_t pp, int32_t mb, int32_t failures,
                                   int32_t* per_stage, int64_t* overhead) {
  if (dp < 2 || pp < 1 || mb < 1 || failures < 0 || !per_stage || !overhead)
    return rc_set_error(RC_ERR_INVALID_ARG, "need dp >= 2, pp >= 1, mb >= 1, failures >= 0 and outputs");
  if ((long long)failures > (long long)pp * (dp - 1))
    return rc_set_error(RC_ERR_INVALID_ARG, "more failures than the pipeline can survive");
  const long long INF = LLONG_MAX / 4;
  const int F = failures;
  // best[f] over stages 0..i, and the choice x of stage i for back-tracking
  std::vector<long long> prev(F + 1, INF), cur(F + 1, INF);
  std::vector<std::vector<int>> choice(pp, std::vector<int>(F + 1, -1));
  for (int f = 0; f <= F && f <= dp - 1; ++f) {
    prev[f] = norm_cost(dp, pp, mb, f);
    choice[0][f] = f;
  }
  for (int i = 1; i < pp; ++i) {
    for (int f = 0; f <= F; ++f) {
      long long best = INF;
      int bx = -1;
      for (int x = 0; x <= f && x <= dp - 1; ++x) {
        if (prev[f - x] >= INF) continue;
        const long long c = prev[f - x] + norm_cost(dp, pp, mb, x);
        if (c <= best) {  // ties: the larger x, i.e. the later stage
          best = c;
          bx = x;
        }
      }
      cur[f] = best;
      choice[i][f] = bx;
    }
    std::swap(prev, cur);
  }
  if (prev[F] >= INF) return rc_set_error(RC_ERR_INVALID_ARG, "no feasible assignment");
  int f = F;
  for (int i = pp - 1; i >= 0; --i) {
    per_stage[i] = choice[i][f];
    f -= choice[i][f];
  }
  *overhead = prev[F];
  return RC_OK;
}

rc_status rc_schedule_simulate(const rc_sim_config* c, rc_sim_result* res, rc_sim_op* ops, int32_t cap,
                               int32_t* n_ops) {
  if (!c || !res || !n_ops || cap < 0 || (cap > 0 && !ops))
    return rc_set_error(RC_ERR_INVALID_ARG, "bad simulate arguments");
  const int dp = c->dp, pp = c->pp, mb = c->mb;
  if (dp < 1 || pp < 1 || mb < 1 || c->iterations < 1 || c->iterations > RC_SIM_MAX_ITER ||
      c->n_failed < 0 || (c->n_failed > 0 && !c->failed))
    return rc_set_error(RC_ERR_INVALID_ARG, "bad simulate configuration");
  // alive workers and round-robin re-routing of a failed worker's micro-batches
  std::vector<char> dead(dp * pp, 0);
  for (int q = 0; q < c->n_failed; ++q) {
    const int k = c->failed[2 * q], i = c->failed[2 * q + 1];
    if (k < 0 || k >= dp || i < 0 || i >= pp) return rc_set_error(RC_ERR_INVALID_ARG, "failed worker out of range");
    dead[k * pp + i] = 1;
  }
  std::vector<int> runner(pp * dp * mb);  // (i, k, j) -> executing pipeline
  for (int i = 0; i < pp; ++i) {
    std::vector<int> alive;
    for (int k = 0; k < dp; ++k)
      if (!dead[k * pp + i]) alive.push_back(k);
    if (alive.empty()) return rc_set_error(RC_ERR_INVALID_ARG, "a stage lost all its workers");
    for (int k = 0; k < dp; ++k)
      for (int j = 0; j < mb; ++j)
        runner[(i * dp + k) * mb + j] = dead[k * pp + i] ? alive[j % alive.size()] : k;
  }
  struct Worker {
    int k, i;
    long long free_at = 0, start = 0, busy = 0;
    std::set<std::pair<int, int>> pending, inflight;  // (k, j) ordered by origin then index
    std::vector<std::pair<int, int>> deferred;
  };
  std::vector<Worker> ws;
  for (int k = 0; k < dp; ++k)
    for (int i = 0; i < pp; ++i)
      if (!dead[k * pp + i]) {
        Worker w;
        w.k = k;
        w.i = i;
        ws.push_back(w);
      }
  const int bdur = c->decoupled ? 1 : 2;
  std::map<Key, long long> done_f, done_b;
  int nrec = 0;
  long long t0 = 0;
  std::memset(res, 0, sizeof(*res));
  for (int it = 0; it < c->iterations; ++it) {
    long long remaining = 0;
    for (auto& w : ws) {
      w.pending.clear();
      w.inflight.clear();
      w.deferred.clear();
      for (int k = 0; k < dp; ++k)
        for (int j = 0; j < mb; ++j)
          if (runner[(w.i * dp + k) * mb + j] == w.k) w.pending.insert({k, j});
      remaining += (long long)w.pending.size() * (c->decoupled ? 3 : 2);
      w.free_at = std::max(t0, w.start);
    }
    // event-driven: advance to the next time at which a worker frees or an op
    // completes; at each such time every free worker (in (k, i) order) picks
    // with the state completed by then.
    std::set<long long> times;
    for (auto& w : ws) times.insert(w.free_at);
    while (remaining > 0) {
      if (times.empty()) return rc_set_error(RC_ERR_INVALID_ARG, "schedule cannot make progress");
      const long long now = *times.begin();
      times.erase(times.begin());
      bool any = false;
      for (auto& w : ws) {
        if (w.free_at > now) continue;
        const int i = w.i;
        int kind = -1;
        std::pair<int, int> sel;
        for (auto& q : w.inflight) {  // ready backward first
          const Key key{it, i, q.second, q.first};
          auto f = done_f.find(key);
          bool ready = f != done_f.end() && f->second <= now;
          if (ready && i < pp - 1) {
            auto b = done_b.find(Key{it, i + 1, q.second, q.first});
            ready = b != done_b.end() && b->second <= now;
          }
          if (ready) {
            kind = RC_OP_B;
            sel = q;
            break;
          }
        }
        const bool room = c->inflight_cap == 0 || (int)w.inflight.size() < pp - i;
        if (kind < 0 && room) {
          for (auto& q : w.pending) {
            bool ready = i == 0;
            if (!ready) {
              auto f = done_f.find(Key{it, i - 1, q.second, q.first});
              ready = f != done_f.end() && f->second <= now;
            }
            if (ready) {
              kind = RC_OP_F;
              sel = q;
              break;
            }
          }
        }
        if (kind < 0 && !w.deferred.empty()) {
          kind = RC_OP_W;
          sel = w.deferred.front();
        }
        if (kind < 0) continue;
        const Key key{it, i, sel.second, sel.first};
        long long dur = 1;
        if (kind == RC_OP_F) {
          w.pending.erase(sel);
          w.inflight.insert(sel);
          done_f[key] = now + 1;
        } else if (kind == RC_OP_B) {
          w.inflight.erase(sel);
          dur = bdur;
          done_b[key] = now + dur;
          if (c->decoupled) w.deferred.push_back(sel);
        } else {
          w.deferred.erase(w.deferred.begin());
        }
        w.free_at = now + dur;
        w.busy += dur;
        times.insert(now + dur);
        --remaining;
        any = true;
        if (nrec < cap) {
          rc_sim_op& o = ops[nrec];
          o.slot = (int32_t)now;
          o.op = kind;
          o.iter = it;
          o.stage = i;
          o.j = sel.second;
          o.k = sel.first;
          o.k_s = w.k;
          o.dur = (int32_t)dur;
        }
        ++nrec;
      }
      if (!any && times.empty()) return rc_set_error(RC_ERR_INVALID_ARG, "schedule cannot make progress");
    }
    long long end = 0;
    for (auto& w : ws) end = std::max(end, w.free_at);
    res->iter_end[it] = (int32_t)end;
    if (c->staggered) {
      // stage i starts the next iteration once all of its workers are done
      for (int i = 0; i < pp; ++i) {
        long long se = 0;
        for (auto& w : ws)
          if (w.i == i) se = std::max(se, w.free_at);
        for (auto& w : ws)
          if (w.i == i) w.start = se;
      }
      t0 = LLONG_MAX;
      for (auto& w : ws) t0 = std::min(t0, w.start);
    } else {
      t0 = end;
      for (auto& w : ws) w.start = end;
    }
    res->makespan = std::max(res->makespan, (int32_t)end);
  }
  res->workers = (int32_t)ws.size();
  long long busy_max = 0;
  for (auto& w : ws) busy_max = std::max(busy_max, w.busy);
  res->busy_max = (int32_t)busy_max;
  *n_ops = nrec;
  return RC_OK;
}

}  // extern "C"
