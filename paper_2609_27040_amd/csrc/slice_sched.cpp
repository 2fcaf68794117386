// Slice scheduling across GPUs (Greedy-Least-Loaded) and bursty preemption
// control: host policy behind the ema_sched_* entry points.
#include <algorithm>
#include <cstdint>
#include <map>
#include <string>
#include <utility>
#include <vector>

#include "ema_slice.h"

namespace ema {
int set_error(int code, const std::string& msg);   // ema_slice.cpp
int internal_error();                              // ema_slice.cpp, from a catch handler
}

struct ema_sched {
  int32_t m = 0;
  int32_t units = 0;
  int64_t window = 0;
  std::vector<int32_t> use;         // [m][m]: units GPU i holds on slice {i, j}
  std::vector<int32_t> cap;         // [m][m]: cap of GPU i on slice {i, j}, -1 none
  std::vector<int64_t> cap_until;   // [m][m]: tick the cap lifts
  std::map<std::pair<int32_t, int32_t>, std::vector<int32_t>> placed;   // (gpu, req) -> peers

  int32_t total(int32_t i, int32_t j) const { return use[i * m + j] + use[j * m + i]; }
  bool capped(int32_t i, int32_t j, int64_t t) const {
    return cap[i * m + j] >= 0 && t < cap_until[i * m + j];
  }
};

using ema::set_error;

extern "C" {

int ema_sched_create(int32_t n_gpus, int32_t slice_units, int64_t cap_window, ema_sched_t* out) try {
  if (!out) return set_error(EMA_ERR_INVAL, "sched_create: NULL out");
  *out = nullptr;
  if (n_gpus < 2 || n_gpus > 4096 || slice_units < 1 || cap_window < 0)
    return set_error(EMA_ERR_INVAL, "sched_create: bad n_gpus, slice_units or cap_window");
  ema_sched* s = new ema_sched;
  s->m = n_gpus;
  s->units = slice_units;
  s->window = cap_window;
  s->use.assign(size_t(n_gpus) * n_gpus, 0);
  s->cap.assign(size_t(n_gpus) * n_gpus, -1);
  s->cap_until.assign(size_t(n_gpus) * n_gpus, 0);
  *out = s;
  return EMA_OK;
} catch (...) {
  return ema::internal_error();
}

int ema_sched_destroy(ema_sched_t s) try {
  if (!s) return set_error(EMA_ERR_INVAL, "sched_destroy: NULL handle");
  delete s;
  return EMA_OK;
} catch (...) {
  return ema::internal_error();
}

int ema_sched_place(ema_sched_t s, int32_t gpu, int32_t req, int32_t n, int64_t t,
                    int32_t* out_peer, int32_t* placed) try {
  if (!s || gpu < 0 || gpu >= s->m || req < 0 || n < 0 || (n > 0 && !out_peer))
    return set_error(EMA_ERR_INVAL, "sched_place: bad arguments");
  // allocate first: a failed host allocation changes nothing
  auto slot = s->placed.try_emplace({gpu, req}).first;
  auto& mine = slot->second;
  try {
    mine.reserve(mine.size() + size_t(n));
  } catch (...) {
    if (mine.empty()) s->placed.erase(slot);
    throw;
  }
  int32_t done = 0;
  for (int32_t k = 0; k < n; ++k) {
    int32_t best = -1;
    for (int32_t j = 0; j < s->m; ++j) {
      if (j == gpu || s->total(gpu, j) >= s->units) continue;
      if (s->capped(gpu, j, t) && s->use[gpu * s->m + j] >= s->cap[gpu * s->m + j]) continue;
      if (best < 0 || s->total(gpu, j) < s->total(gpu, best)) best = j;
    }
    out_peer[k] = best;
    if (best >= 0) {
      ++s->use[gpu * s->m + best];
      mine.push_back(best);
      ++done;
    }
  }
  if (placed) *placed = done;
  return EMA_OK;
} catch (...) {
  return ema::internal_error();
}

int ema_sched_release(ema_sched_t s, int32_t gpu, int32_t req, int32_t n) try {
  if (!s || gpu < 0 || gpu >= s->m || n < 0)
    return set_error(EMA_ERR_INVAL, "sched_release: bad arguments");
  auto it = s->placed.find({gpu, req});
  const int32_t held = it == s->placed.end() ? 0 : int32_t(it->second.size());
  if (n > held) return set_error(EMA_ERR_INVAL, "sched_release: more units than the request holds");
  for (int32_t k = 0; k < n; ++k) {
    --s->use[gpu * s->m + it->second.back()];
    it->second.pop_back();
  }
  if (it != s->placed.end() && it->second.empty()) s->placed.erase(it);
  return EMA_OK;
} catch (...) {
  return ema::internal_error();
}

int ema_sched_preempted(ema_sched_t s, int32_t gpu, int32_t peer, int64_t t) try {
  if (!s || gpu < 0 || gpu >= s->m || peer < 0 || peer >= s->m || peer == gpu)
    return set_error(EMA_ERR_INVAL, "sched_preempted: bad arguments");
  if (s->window == 0) return EMA_OK;
  const size_t e = size_t(gpu) * s->m + peer;
  const int32_t level = s->use[e];
  if (2 * int64_t(level) <= s->units) return EMA_OK;   // within its half: no cap
  // a new cap, or a lower one; any such preemption restarts the window
  if (!s->capped(gpu, peer, t) || level < s->cap[e]) s->cap[e] = level;
  s->cap_until[e] = t + s->window;
  return EMA_OK;
} catch (...) {
  return ema::internal_error();
}

int ema_sched_usage(ema_sched_t s, int64_t t, int32_t* use, int32_t* cap) try {
  if (!s || !use) return set_error(EMA_ERR_INVAL, "sched_usage: NULL argument");
  for (size_t e = 0; e < s->use.size(); ++e) {
    use[e] = s->use[e];
    if (cap) cap[e] = s->capped(int32_t(e / s->m), int32_t(e % s->m), t) ? s->cap[e] : -1;
  }
  return EMA_OK;
} catch (...) {
  return ema::internal_error();
}

}  // extern "C"
