// Round-based step scheduler of TetriServe (section 4.2): deadline-aware GPU
// allocation of one request and the per-round packing of requests onto GPUs.
// Host code only; the C ABI is declared in include/tetri_sched.h.
#include "../../../include/tetri_sched.h"

#include <algorithm>
#include <array>
#include <cstdint>
#include <vector>

namespace {

constexpr int32_t kNone = -1;

// degrees usable on max_gpus GPUs: indices j with 2^j <= max_gpus and a profiled time
std::vector<int> usable_degrees(const int64_t* step_us, int32_t n_degrees, int32_t max_gpus) {
  std::vector<int> js;
  for (int j = 0; j < n_degrees; ++j)
    if ((int64_t(1) << j) <= max_gpus && step_us[j] > 0) js.push_back(j);
  return js;
}

// A partial or complete split of steps over the usable degrees.
struct Split {
  int64_t time = 0;  // sum n_j T(2^j)
  int64_t cost = 0;  // sum n_j 2^j T(2^j)
  std::array<int32_t, TS_MAX_DEGREES> n{};  // steps per usable degree, in increasing degree order
};

// composition preference: more steps on smaller degrees (lexicographic from the first degree)
bool prefer(const Split& a, const Split& b) {
  for (int d = 0; d < TS_MAX_DEGREES; ++d)
    if (a.n[d] != b.n[d]) return a.n[d] > b.n[d];
  return false;
}

// non-dominated splits in (time, cost); among equal pairs the preferred composition
void prune(std::vector<Split>& v) {
  std::sort(v.begin(), v.end(), [](const Split& a, const Split& b) {
    if (a.time != b.time) return a.time < b.time;
    if (a.cost != b.cost) return a.cost < b.cost;
    return prefer(a, b);
  });
  std::vector<Split> keep;
  for (const Split& s : v)
    if (keep.empty() || s.cost < keep.back().cost) keep.push_back(s);
  v.swap(keep);
}

int64_t step_time_of(const int64_t* step_us, int32_t gpus) {
  if (gpus <= 0 || (gpus & (gpus - 1)) != 0) return 0;
  int j = 0;
  while ((1 << j) < gpus) ++j;
  return j < TS_MAX_DEGREES ? step_us[j] : 0;
}

// One thing a request can do in the coming round (section 4.2.2): stay idle
// (alloc = kNone, no GPUs), or run one of its planned allocations for as many
// of that allocation's steps as fit in the round.  `alive`: whether it can
// still meet its deadline afterwards, if every step it has left then ran at
// its fastest degree.
struct Choice {
  int32_t alloc;
  int32_t gpus;
  int32_t steps;
  int32_t alive;
};

// What a packing achieves: requests kept alive first, then fewer GPUs (GPUs
// left over go to late requests and to scale-up).
struct Value {
  int32_t alive = 0;
  int32_t gpus = 0;
};
bool better(const Value& a, const Value& b) { return a.alive != b.alive ? a.alive > b.alive : a.gpus < b.gpus; }
bool same(const Value& a, const Value& b) { return a.alive == b.alive && a.gpus == b.gpus; }

std::vector<Choice> round_choices(const ts_request& r, int32_t n_gpus, int64_t round_us, int64_t round_end_us) {
  int64_t fastest = 0;
  for (int j : usable_degrees(r.step_us, TS_MAX_DEGREES, n_gpus))
    if (fastest == 0 || r.step_us[j] < fastest) fastest = r.step_us[j];
  // steps of each allocation that fit in one round
  std::vector<int32_t> fit(r.n_allocs, 0);
  for (int m = 0; m < r.n_allocs; ++m) {
    const int64_t t = step_time_of(r.step_us, r.allocs[m].gpus);
    if (t > 0) fit[m] = int32_t(std::min<int64_t>(r.allocs[m].steps, round_us / t));
  }
  // alive after running `ran` steps of allocation `m` (none for kNone)
  auto alive_after = [&](int32_t m) {
    int64_t left = 0;
    for (int a = 0; a < r.n_allocs; ++a) left += r.allocs[a].steps - (a == m ? fit[a] : 0);
    return int32_t(round_end_us + left * fastest <= r.deadline_us);
  };
  std::vector<Choice> out{Choice{kNone, 0, 0, alive_after(kNone)}};
  for (int m = 0; m < r.n_allocs; ++m)
    if (fit[m] > 0 && r.allocs[m].gpus <= n_gpus) out.push_back(Choice{m, r.allocs[m].gpus, fit[m], alive_after(m)});
  return out;
}

}  // namespace

extern "C" ts_status ts_allocate(const int64_t* step_us, int32_t n_degrees, int32_t max_gpus, int32_t steps,
                                 int64_t budget_us, ts_alloc* out, int32_t* n_out, int64_t* gpu_time_us,
                                 int64_t* time_us) {
  if (!step_us || !out || !n_out || !gpu_time_us || !time_us) return TS_ERR_INVALID_ARG;
  if (n_degrees < 1 || n_degrees > TS_MAX_DEGREES || max_gpus < 1 || max_gpus > TS_MAX_GPUS || steps < 0 ||
      steps > TS_MAX_STEPS)
    return TS_ERR_INVALID_ARG;
  for (int j = 0; j < n_degrees; ++j)
    if (step_us[j] < 0) return TS_ERR_INVALID_ARG;
  const std::vector<int> js = usable_degrees(step_us, n_degrees, max_gpus);
  if (js.empty()) return TS_ERR_INVALID_ARG;
  if (steps == 0) {
    *n_out = 0;
    *gpu_time_us = 0;
    *time_us = 0;
    return TS_OK;
  }
  // front[s]: non-dominated splits of s steps over the degrees seen so far,
  // none of them over budget (times only grow as degrees are added)
  std::vector<std::vector<Split>> front(steps + 1);
  front[0].push_back(Split{});
  for (size_t d = 0; d < js.size(); ++d) {
    const int64_t t = step_us[js[d]], c = t << js[d];
    std::vector<std::vector<Split>> next(steps + 1);
    for (int s0 = 0; s0 <= steps; ++s0)
      for (const Split& p : front[s0])
        for (int add = 0; s0 + add <= steps; ++add) {
          Split q = p;
          q.time += add * t;
          q.cost += add * c;
          if (q.time > budget_us) break;
          q.n[d] = add;
          next[s0 + add].push_back(q);
        }
    for (auto& v : next) prune(v);
    front.swap(next);
  }
  ts_status st = TS_OK;
  Split best;
  bool found = false;
  for (const Split& p : front[steps]) {
    const bool better = !found || p.cost < best.cost || (p.cost == best.cost && p.time < best.time) ||
                        (p.cost == best.cost && p.time == best.time && prefer(p, best));
    if (better) {
      best = p;
      found = true;
    }
  }
  if (!found) {
    // no split meets the budget: all steps on the fastest degree (ties: the smaller k)
    size_t f = 0;
    for (size_t d = 1; d < js.size(); ++d)
      if (step_us[js[d]] < step_us[js[f]]) f = d;
    best = Split{};
    best.n[f] = steps;
    best.time = steps * step_us[js[f]];
    best.cost = best.time << js[f];
    st = TS_INFEASIBLE;
  }
  int32_t k = 0;
  for (size_t d = 0; d < js.size(); ++d)
    if (best.n[d] > 0) out[k++] = ts_alloc{best.n[d], int32_t(1) << js[d]};
  *n_out = k;
  *gpu_time_us = best.cost;
  *time_us = best.time;
  return st;
}

extern "C" ts_status ts_round_schedule(const ts_request* reqs, int32_t n_req, int32_t n_gpus, int64_t round_us,
                                       int64_t now_us, ts_decision* out, int32_t* survivors, int32_t* gpus_used) {
  if (n_req < 0 || (n_req > 0 && (!reqs || !out)) || !survivors || !gpus_used) return TS_ERR_INVALID_ARG;
  if (n_gpus < 1 || n_gpus > TS_MAX_GPUS || round_us <= 0) return TS_ERR_INVALID_ARG;
  for (int i = 0; i < n_req; ++i) {
    const ts_request& r = reqs[i];
    if (r.n_allocs < 0 || r.n_allocs > TS_MAX_ALLOCS) return TS_ERR_INVALID_ARG;
    for (int j = 0; j < TS_MAX_DEGREES; ++j)
      if (r.step_us[j] < 0) return TS_ERR_INVALID_ARG;
    for (int m = 0; m < r.n_allocs; ++m)
      if (r.allocs[m].steps < 0 || r.allocs[m].gpus < 1) return TS_ERR_INVALID_ARG;
    if (usable_degrees(r.step_us, TS_MAX_DEGREES, n_gpus).empty()) return TS_ERR_INVALID_ARG;
  }
  const int64_t round_end = now_us + round_us;
  std::vector<std::vector<Choice>> choices(n_req);
  std::vector<int64_t> steps_left(n_req, 0);
  for (int i = 0; i < n_req; ++i) {
    choices[i] = round_choices(reqs[i], n_gpus, round_us, round_end);
    for (int m = 0; m < reqs[i].n_allocs; ++m) steps_left[i] += reqs[i].allocs[m].steps;
  }

  // Pack one choice per request into the N GPUs, maximising the requests kept
  // alive (a knapsack with one group of choices per request).  best[i][g] is
  // the best Value of requests i.. on at most g GPUs, filled from the last
  // request backwards.
  const int N = n_gpus;
  std::vector<std::vector<Value>> best(n_req + 1, std::vector<Value>(N + 1));
  for (int i = n_req - 1; i >= 0; --i)
    for (int g = 0; g <= N; ++g) {
      bool set = false;
      for (const Choice& ch : choices[i]) {
        if (ch.gpus > g) continue;
        const Value& rest = best[i + 1][g - ch.gpus];
        const Value v{ch.alive + rest.alive, ch.gpus + rest.gpus};
        if (!set || better(v, best[i][g])) best[i][g] = v;
        set = true;
      }
    }
  // Read the plan forwards: each request takes its first choice (idle, then
  // allocations in order) that still reaches the best value.
  int32_t used = 0;
  for (int i = 0, g = N; i < n_req; ++i) {
    for (const Choice& ch : choices[i]) {
      if (ch.gpus > g) continue;
      const Value& rest = best[i + 1][g - ch.gpus];
      if (same(Value{ch.alive + rest.alive, ch.gpus + rest.gpus}, best[i][g])) {
        out[i] = ts_decision{ch.alloc, ch.gpus, ch.steps, ch.alive, 0};
        g -= ch.gpus;
        used += ch.gpus;
        break;
      }
    }
  }

  // Requests that cannot stay alive whatever they run get one leftover GPU
  // each, earliest deadline first, for the steps that fit in the round.
  std::vector<int> late;
  for (int i = 0; i < n_req; ++i)
    if (std::none_of(choices[i].begin(), choices[i].end(), [](const Choice& ch) { return ch.alive != 0; }))
      late.push_back(i);
  std::stable_sort(late.begin(), late.end(),
                   [&](int a, int b) { return reqs[a].deadline_us < reqs[b].deadline_us; });
  for (int i : late) {
    if (used >= N) break;
    const int64_t t1 = reqs[i].step_us[0];
    const int64_t q1 = t1 > 0 ? std::min<int64_t>(steps_left[i], round_us / t1) : 0;
    if (q1 <= 0 || out[i].gpus != 0) continue;
    out[i] = ts_decision{kNone, 1, int32_t(q1), 0, 1};
    used += 1;
  }
  *survivors = n_req > 0 ? best[0][N].alive : 0;
  *gpus_used = used;
  return TS_OK;
}

extern "C" ts_status ts_select_batch(const ts_request* reqs, int32_t n_req, const int64_t* batch_us, int32_t max_b,
                                     int64_t round_us, int64_t now_us, int32_t* members, int32_t* b) {
  if (n_req < 0 || (n_req > 0 && (!reqs || !members)) || !batch_us || !b || max_b < 1 || round_us <= 0)
    return TS_ERR_INVALID_ARG;
  if (batch_us[1] <= 0) return TS_ERR_INVALID_ARG;
  for (int32_t x = 1; x <= max_b; ++x)
    if (batch_us[x] < 0) return TS_ERR_INVALID_ARG;
  for (int i = 0; i < n_req; ++i) {
    const ts_request& r = reqs[i];
    if (r.n_allocs < 0 || r.n_allocs > TS_MAX_ALLOCS) return TS_ERR_INVALID_ARG;
    for (int m = 0; m < r.n_allocs; ++m)
      if (r.allocs[m].steps < 0) return TS_ERR_INVALID_ARG;
    if (usable_degrees(r.step_us, TS_MAX_DEGREES, TS_MAX_GPUS).empty()) return TS_ERR_INVALID_ARG;
  }
  std::vector<int32_t> order(n_req);
  for (int i = 0; i < n_req; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t x, int32_t y) { return reqs[x].deadline_us < reqs[y].deadline_us; });
  const int64_t t_next = now_us + round_us;
  auto survives = [&](int32_t i, int64_t q) {
    const ts_request& r = reqs[i];
    int64_t left = 0, t_min = 0;
    for (int m = 0; m < r.n_allocs; ++m) left += r.allocs[m].steps;
    for (int j : usable_degrees(r.step_us, TS_MAX_DEGREES, TS_MAX_GPUS))
      if (t_min == 0 || r.step_us[j] < t_min) t_min = r.step_us[j];
    return t_next + (left - std::min(left, q)) * t_min <= r.deadline_us;
  };
  const int64_t q1 = round_us / batch_us[1];
  int32_t best = n_req > 0 ? 1 : 0;
  for (int32_t x = 2; x <= std::min(max_b, n_req); ++x) {
    if (batch_us[x] <= 0) continue;
    const int64_t qb = round_us / batch_us[x];
    if (qb <= 0) continue;
    bool ok = true;
    for (int32_t p = 0; p < x && ok; ++p) ok = !survives(order[p], q1) || survives(order[p], qb);
    if (ok) best = x;
  }
  for (int i = 0; i < n_req; ++i) members[i] = order[i];
  *b = best;
  return TS_OK;
}
