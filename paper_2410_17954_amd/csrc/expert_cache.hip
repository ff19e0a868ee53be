// Expert cache engine (Sec. 3.4): the cross-layer slot plan built from the
// predicted demand (PLEC, Sec. 3.4.1), its run with real-time correction of
// mispredictions, the per-layer LRU cache it is compared with, and the
// loading of whole experts from host memory into device cache slots.
//
// Planning and simulation are host code over small integer tables; the loads
// are asynchronous copies on the caller's stream, so they overlap kernels
// running on other streams (the correction loads experts while resident ones
// compute).
#include "common.h"

#include <algorithm>
#include <vector>

namespace moe {
namespace {

struct Item {
  int32_t l, e;
};

// Load order: every (layer, expert) with demand > 0; layers in execution
// order, larger demand first, equal demand lower expert id first.
std::vector<Item> load_order(const int32_t* demand, int L, int E) {
  std::vector<Item> v;
  for (int l = 0; l < L; ++l)
    for (int e = 0; e < E; ++e)
      if (demand[(int64_t)l * E + e] > 0) v.push_back(Item{l, e});
  std::stable_sort(v.begin(), v.end(), [&](const Item& a, const Item& b) {
    if (a.l != b.l) return a.l < b.l;
    const int32_t da = demand[(int64_t)a.l * E + a.e], db = demand[(int64_t)b.l * E + b.e];
    if (da != db) return da > db;
    return a.e < b.e;
  });
  return v;
}

}  // namespace
}  // namespace moe

extern "C" int moe_plan_slots(const int32_t* demand, int32_t E, int32_t S,
                              int32_t* slot_of_expert) {
  MOE_CHECK_ARG(demand && slot_of_expert && E >= 1);
  std::vector<int32_t> ids(E);
  for (int32_t e = 0; e < E; ++e) ids[e] = e;
  // larger demand first; equal demand, lower id first
  std::stable_sort(ids.begin(), ids.end(),
                   [&](int32_t a, int32_t b) { return demand[a] > demand[b]; });
  const int32_t n = S < 0 ? 0 : (S > E ? E : S);
  std::vector<char> chosen(E, 0);
  for (int32_t i = 0; i < n; ++i) chosen[ids[i]] = 1;
  int32_t next = 0;
  for (int32_t e = 0; e < E; ++e) slot_of_expert[e] = chosen[e] ? next++ : -1;
  return MOE_OK;
}

extern "C" int moe_plec_order(const int32_t* demand, int32_t L, int32_t E, int32_t* items,
                              int32_t* n_items) {
  using namespace moe;
  MOE_CHECK_ARG(demand && items && n_items && L >= 1 && E >= 1);
  const std::vector<Item> v = load_order(demand, L, E);
  for (size_t i = 0; i < v.size(); ++i) {
    items[2 * i] = v[i].l;
    items[2 * i + 1] = v[i].e;
  }
  *n_items = (int32_t)v.size();
  return MOE_OK;
}

extern "C" int moe_plec_run(const int32_t* pred_demand, const int32_t* actual_demand, int32_t L,
                            int32_t E, int32_t budget, int32_t* prefetch, int32_t* n_prefetch,
                            int64_t* hits, int64_t* needed, int64_t* loads) {
  using namespace moe;
  MOE_CHECK_ARG(pred_demand && actual_demand && hits && needed && loads && L >= 1 && E >= 1 &&
                budget >= 0);
  const std::vector<Item> order = load_order(pred_demand, L, E);
  // Residency table: rank[l * E + e] = position in the load order (or a
  // position past it for correction loads), res[...] = resident.
  const int64_t LE = (int64_t)L * E;
  std::vector<int64_t> rank(LE, -1);
  for (size_t i = 0; i < order.size(); ++i) rank[(int64_t)order[i].l * E + order[i].e] = (int64_t)i;
  std::vector<char> res(LE, 0), queued(LE, 0);
  for (const Item& it : order) queued[(int64_t)it.l * E + it.e] = 1;
  int64_t n_res = 0, n_loads = 0;
  auto fill = [&](int current) {
    // walk the order from the front; items of layers that have run are dropped
    for (size_t i = 0; i < order.size() && n_res < budget; ++i) {
      const int64_t c = (int64_t)order[i].l * E + order[i].e;
      if (!queued[c]) continue;
      if (order[i].l < current) {
        queued[c] = 0;
        continue;
      }
      queued[c] = 0;
      res[c] = 1;
      ++n_res;
      ++n_loads;
    }
  };
  fill(0);
  if (prefetch && n_prefetch) {
    int32_t n = 0;
    for (const Item& it : order)
      if (res[(int64_t)it.l * E + it.e]) {
        prefetch[2 * n] = it.l;
        prefetch[2 * n + 1] = it.e;
        ++n;
      }
    *n_prefetch = n;
  }
  for (int l = 0; l < L; ++l) {
    const int32_t* act = actual_demand + (int64_t)l * E;
    int64_t h = 0, nd = 0;
    for (int e = 0; e < E; ++e) {
      if (act[e] <= 0) continue;
      ++nd;
      const int64_t c = (int64_t)l * E + e;
      if (res[c]) {
        ++h;
        continue;
      }
      ++n_loads;                                     // the correction load
      if (n_res < budget) {
        res[c] = 1;
        ++n_res;
        continue;
      }
      // victim: an unused expert of this layer latest in load order, else the
      // item of a later layer latest in load order (queued again)
      int64_t victim = -1, vrank = -2;
      for (int f = 0; f < E; ++f) {
        const int64_t cf = (int64_t)l * E + f;
        if (res[cf] && act[f] <= 0 && rank[cf] > vrank) {
          victim = cf;
          vrank = rank[cf];
        }
      }
      if (victim < 0) {
        for (int64_t cf = (int64_t)(l + 1) * E; cf < LE; ++cf)
          if (res[cf] && rank[cf] > vrank) {
            victim = cf;
            vrank = rank[cf];
          }
        if (victim >= 0) queued[victim] = 1;
      }
      if (victim < 0) continue;                      // served without caching
      res[victim] = 0;
      res[c] = 1;
    }
    hits[l] = h;
    needed[l] = nd;
    for (int e = 0; e < E; ++e) {
      const int64_t c = (int64_t)l * E + e;
      if (res[c]) {
        res[c] = 0;
        --n_res;
      }
    }
    fill(l + 1);
  }
  *loads = n_loads;
  return MOE_OK;
}

extern "C" int moe_lru_run(const int32_t* actual_demand, int32_t B, int32_t L, int32_t E,
                           int32_t capacity, int64_t* hits, int64_t* needed) {
  using namespace moe;
  MOE_CHECK_ARG(actual_demand && hits && needed && B >= 0 && L >= 1 && E >= 1 && capacity >= 0);
  // last-use stamps per (layer, expert); a layer's cache is its resident set
  std::vector<int64_t> stamp((int64_t)L * E, -1);
  std::vector<char> res((int64_t)L * E, 0);
  std::vector<int32_t> count(L, 0);
  int64_t h = 0, nd = 0, clock = 0;
  for (int b = 0; b < B; ++b)
    for (int l = 0; l < L; ++l) {
      const int32_t* act = actual_demand + ((int64_t)b * L + l) * E;
      for (int e = 0; e < E; ++e) {
        if (act[e] <= 0) continue;
        ++nd;
        const int64_t c = (int64_t)l * E + e;
        if (res[c]) {
          ++h;
          stamp[c] = clock++;
          continue;
        }
        if (capacity == 0) continue;
        res[c] = 1;
        stamp[c] = clock++;
        if (++count[l] > capacity) {                 // evict the least recent
          int64_t victim = -1;
          for (int f = 0; f < E; ++f) {
            const int64_t cf = (int64_t)l * E + f;
            if (res[cf] && (victim < 0 || stamp[cf] < stamp[victim])) victim = cf;
          }
          res[victim] = 0;
          --count[l];
        }
      }
    }
  *hits = h;
  *needed = nd;
  return MOE_OK;
}

extern "C" int moe_load_experts(const void* w_gate_src, const void* w_up_src,
                                const void* w_down_src, int32_t E_store, void* w_gate,
                                void* w_up, void* w_down, int32_t S, int64_t H, int64_t F,
                                int32_t dtype, const int32_t* expert_ids,
                                const int32_t* slot_ids, int32_t n, void* stream) {
  using namespace moe;
  MOE_CHECK_ARG(n >= 0 && E_store >= 1 && S >= 1 && H >= 1 && F >= 1 && valid_dtype(dtype));
  if (n == 0) return MOE_OK;
  MOE_CHECK_ARG(w_gate_src && w_up_src && w_down_src && w_gate && w_up && w_down && expert_ids &&
                slot_ids);
  for (int32_t i = 0; i < n; ++i) {
    MOE_CHECK_ARG(expert_ids[i] >= 0 && expert_ids[i] < E_store);
    MOE_CHECK_ARG(slot_ids[i] >= 0 && slot_ids[i] < S);
    for (int32_t j = 0; j < i; ++j) MOE_CHECK_ARG(slot_ids[j] != slot_ids[i]);
  }
  const size_t esz = dtype == MOE_BF16 ? 2 : 4;
  const size_t block = (size_t)H * (size_t)F * esz;  // one expert's matrix
  hipStream_t st = as_stream(stream);
  for (int32_t i = 0; i < n; ++i) {
    const size_t src = (size_t)expert_ids[i] * block, dst = (size_t)slot_ids[i] * block;
    const void* srcs[3] = {w_gate_src, w_up_src, w_down_src};
    void* dsts[3] = {w_gate, w_up, w_down};
    for (int m = 0; m < 3; ++m)
      if (hipMemcpyAsync(static_cast<char*>(dsts[m]) + dst,
                         static_cast<const char*>(srcs[m]) + src, block, hipMemcpyDefault,
                         st) != hipSuccess)
        return MOE_ERR_HIP;
  }
  return MOE_OK;
}
