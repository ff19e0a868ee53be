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

// ---------------------------------------------------------------- planner
// The PLEC policy as a state machine over (layer, expert) cells that also
// assigns cache slots, so that a run can execute its loads: begin (the
// prefetch before the first layer), then per layer `layer` (the layer's
// actual demand is known: hits, and correction loads for the misses) and
// `advance` (the layer has run: its slots are freed and refilled with later
// layers' items in load order). Free slots are taken lowest index first.
// The state lives in caller-provided host memory (moe_plec_state_bytes).
namespace moe {
namespace {

struct PlecHead {
  int32_t L, E, budget, n_order, n_res, next_layer;
  int64_t n_loads;
};

struct PlecView {
  PlecHead* h;
  int32_t* order_l;     // [LE] load order (n_order items)
  int32_t* order_e;
  int64_t* rank;        // [LE] position in the load order, -1 if absent
  int32_t* slot_of;     // [LE] slot holding the cell, -1 if not resident
  int32_t* owner;       // [budget] cell held by the slot, -1 if free
  uint8_t* queued;      // [LE] waiting in the load order
};

size_t plec_bytes(int64_t L, int64_t E, int64_t budget) {
  const int64_t LE = L * E;
  return align_up(sizeof(PlecHead), 8) + align_up((size_t)LE * 8, 8) + (size_t)LE * 8 +
         (size_t)LE * 4 + align_up((size_t)budget * 4, 8) + (size_t)LE;
}

PlecView plec_view(void* state) {
  PlecView v;
  char* p = static_cast<char*>(state);
  v.h = reinterpret_cast<PlecHead*>(p);
  const int64_t LE = (int64_t)v.h->L * v.h->E;
  p += align_up(sizeof(PlecHead), 8);
  v.order_l = reinterpret_cast<int32_t*>(p);
  v.order_e = v.order_l + LE;
  p += align_up((size_t)LE * 8, 8);
  v.rank = reinterpret_cast<int64_t*>(p);
  p += (size_t)LE * 8;
  v.slot_of = reinterpret_cast<int32_t*>(p);
  p += (size_t)LE * 4;
  v.owner = reinterpret_cast<int32_t*>(p);
  p += align_up((size_t)v.h->budget * 4, 8);
  v.queued = reinterpret_cast<uint8_t*>(p);
  return v;
}

int32_t free_slot(const PlecView& v) {
  for (int32_t q = 0; q < v.h->budget; ++q)
    if (v.owner[q] < 0) return q;
  return -1;
}

void emit(int32_t* loads, int32_t* n, int64_t cell, int32_t E, int32_t slot) {
  if (loads) {
    loads[3 * *n] = (int32_t)(cell / E);
    loads[3 * *n + 1] = (int32_t)(cell % E);
    loads[3 * *n + 2] = slot;
  }
  ++*n;
}

// Walk the load order from the front: items of layers before `current` are
// dropped, the others are loaded into free slots while there are any.
void plec_fill(const PlecView& v, int current, int32_t* loads, int32_t* n) {
  const int32_t E = v.h->E;
  for (int32_t i = 0; i < v.h->n_order && v.h->n_res < v.h->budget; ++i) {
    const int64_t c = (int64_t)v.order_l[i] * E + v.order_e[i];
    if (!v.queued[c]) continue;
    v.queued[c] = 0;
    if (v.order_l[i] < current) continue;
    const int32_t q = free_slot(v);
    v.owner[q] = (int32_t)c;
    v.slot_of[c] = q;
    ++v.h->n_res;
    ++v.h->n_loads;
    emit(loads, n, c, E, q);
  }
}

}  // namespace
}  // namespace moe

extern "C" size_t moe_plec_state_bytes(int32_t L, int32_t E, int32_t budget) {
  if (L < 1 || E < 1 || budget < 0) return 0;
  return moe::plec_bytes(L, E, budget);
}

extern "C" int moe_plec_begin(const int32_t* pred_demand, int32_t L, int32_t E, int32_t budget,
                              void* state, size_t state_bytes, int32_t* loads,
                              int32_t* n_loads) {
  using namespace moe;
  MOE_CHECK_ARG(pred_demand && state && n_loads && L >= 1 && E >= 1 && budget >= 0);
  MOE_CHECK_ARG((int64_t)L * E < ((int64_t)1 << 30));
  MOE_CHECK_ARG(state_bytes >= plec_bytes(L, E, budget));
  PlecHead* h = static_cast<PlecHead*>(state);
  *h = PlecHead{L, E, budget, 0, 0, 0, 0};
  const PlecView v = plec_view(state);
  const int64_t LE = (int64_t)L * E;
  const std::vector<Item> order = load_order(pred_demand, L, E);
  h->n_order = (int32_t)order.size();
  for (int64_t c = 0; c < LE; ++c) {
    v.rank[c] = -1;
    v.slot_of[c] = -1;
    v.queued[c] = 0;
  }
  for (int32_t q = 0; q < budget; ++q) v.owner[q] = -1;
  for (size_t i = 0; i < order.size(); ++i) {
    v.order_l[i] = order[i].l;
    v.order_e[i] = order[i].e;
    const int64_t c = (int64_t)order[i].l * E + order[i].e;
    v.rank[c] = (int64_t)i;
    v.queued[c] = 1;
  }
  *n_loads = 0;
  plec_fill(v, 0, loads, n_loads);
  return MOE_OK;
}

extern "C" int moe_plec_layer(void* state, int32_t l, const int32_t* actual_demand,
                              int32_t* slot_of_expert, int32_t* loads, int32_t* n_loads,
                              int64_t* hits, int64_t* needed) {
  using namespace moe;
  MOE_CHECK_ARG(state && actual_demand && n_loads && hits && needed);
  const PlecView v = plec_view(state);
  const int32_t L = v.h->L, E = v.h->E;
  MOE_CHECK_ARG(l == v.h->next_layer && l >= 0 && l < L);
  const int32_t* act = actual_demand;
  int64_t h = 0, nd = 0;
  *n_loads = 0;
  for (int e = 0; e < E; ++e) {
    if (act[e] <= 0) continue;
    ++nd;
    const int64_t c = (int64_t)l * E + e;
    if (v.slot_of[c] >= 0) {
      ++h;
      continue;
    }
    ++v.h->n_loads;                                  // the correction load
    if (v.h->n_res < v.h->budget) {
      const int32_t q = free_slot(v);
      v.owner[q] = (int32_t)c;
      v.slot_of[c] = q;
      ++v.h->n_res;
      emit(loads, n_loads, c, E, q);
      continue;
    }
    // victim: an unused expert of this layer latest in load order, else the
    // item of a later layer latest in load order (queued again)
    int64_t victim = -1, vrank = -2;
    for (int f = 0; f < E; ++f) {
      const int64_t cf = (int64_t)l * E + f;
      if (v.slot_of[cf] >= 0 && act[f] <= 0 && v.rank[cf] > vrank) {
        victim = cf;
        vrank = v.rank[cf];
      }
    }
    if (victim < 0) {
      for (int64_t cf = (int64_t)(l + 1) * E; cf < (int64_t)L * E; ++cf)
        if (v.slot_of[cf] >= 0 && v.rank[cf] > vrank) {
          victim = cf;
          vrank = v.rank[cf];
        }
      if (victim >= 0) v.queued[victim] = 1;
    }
    if (victim < 0) {                                // served without caching
      emit(loads, n_loads, c, E, -1);
      continue;
    }
    const int32_t q = v.slot_of[victim];
    v.slot_of[victim] = -1;
    v.owner[q] = (int32_t)c;
    v.slot_of[c] = q;
    emit(loads, n_loads, c, E, q);
  }
  if (slot_of_expert)
    for (int e = 0; e < E; ++e) slot_of_expert[e] = v.slot_of[(int64_t)l * E + e];
  *hits = h;
  *needed = nd;
  return MOE_OK;
}

extern "C" int moe_plec_advance(void* state, int32_t l, int32_t* loads, int32_t* n_loads) {
  using namespace moe;
  MOE_CHECK_ARG(state && n_loads);
  const PlecView v = plec_view(state);
  const int32_t L = v.h->L, E = v.h->E;
  MOE_CHECK_ARG(l == v.h->next_layer && l >= 0 && l < L);
  for (int e = 0; e < E; ++e) {
    const int64_t c = (int64_t)l * E + e;
    if (v.slot_of[c] >= 0) {
      v.owner[v.slot_of[c]] = -1;
      v.slot_of[c] = -1;
      --v.h->n_res;
    }
  }
  v.h->next_layer = l + 1;
  *n_loads = 0;
  if (l + 1 < L) plec_fill(v, l + 1, loads, n_loads);
  return MOE_OK;
}

extern "C" int moe_plec_run(const int32_t* pred_demand, const int32_t* actual_demand, int32_t L,
                            int32_t E, int32_t budget, int32_t* prefetch, int32_t* n_prefetch,
                            int64_t* hits, int64_t* needed, int64_t* loads) {
  using namespace moe;
  MOE_CHECK_ARG(pred_demand && actual_demand && hits && needed && loads && L >= 1 && E >= 1 &&
                budget >= 0);
  MOE_CHECK_ARG((int64_t)L * E < ((int64_t)1 << 30));
  std::vector<char> state(plec_bytes(L, E, budget));
  std::vector<int32_t> batch(3 * (size_t)std::max<int64_t>((int64_t)budget, E));
  int32_t n = 0;
  int rc = moe_plec_begin(pred_demand, L, E, budget, state.data(), state.size(), batch.data(), &n);
  if (rc != MOE_OK) return rc;
  if (prefetch && n_prefetch) {
    // the prefetched items in load order
    const PlecView v = plec_view(state.data());
    int32_t m = 0;
    for (int32_t i = 0; i < v.h->n_order; ++i) {
      const int64_t c = (int64_t)v.order_l[i] * E + v.order_e[i];
      if (v.slot_of[c] >= 0) {
        prefetch[2 * m] = v.order_l[i];
        prefetch[2 * m + 1] = v.order_e[i];
        ++m;
      }
    }
    *n_prefetch = m;
  }
  for (int32_t l = 0; l < L; ++l) {
    rc = moe_plec_layer(state.data(), l, actual_demand + (int64_t)l * E, nullptr, nullptr, &n,
                        &hits[l], &needed[l]);
    if (rc != MOE_OK) return rc;
    rc = moe_plec_advance(state.data(), l, nullptr, &n);
    if (rc != MOE_OK) return rc;
  }
  *loads = plec_view(state.data()).h->n_loads;
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
