// Per-layer HBM expert cache of a mixture-of-experts decoder: which expert
// sits in which slot, least-recently-used replacement, and the ahead-of-time
// insertion of experts predicted by the fast residual stream (Sec. 2.3.3:
// the least recently used experts are replaced by the speculated ones; the
// experts of layers 2i+2 and 2i+3 are predicted while layer i runs, and the
// experts still missing when a layer's MLP starts are loaded on demand).
//
// The paper leaves the bookkeeping open; the rules implemented here:
//  - each layer has its own C slots; the cache starts warm with experts
//    0..C-1 in slots 0..C-1, expert 0 the least recently used;
//  - one clock for all layers stamps every use and every insertion;
//  - use(layer, S): the needed experts S (router order) that are resident are
//    refreshed first, in S order; each missing one is then placed, in S order,
//    into the slot with the oldest stamp among the experts that are neither
//    needed now nor predicted for this layer in the current token (if all are,
//    the oldest among those not needed now);
//  - predict(layer, P): for each predicted expert in order, a resident one is
//    refreshed; a missing one replaces the oldest expert not in P and is
//    marked as prefetched until it is used or evicted;
//  - a hit is logical: the expert is resident or its copy is in flight.
//
// Pure host code: the GPU runtime turns the slot placements into copies, and
// a replay entry point runs it on a recorded trace without any device.
#pragma once
#include <stdint.h>

#include <algorithm>
#include <vector>

namespace m2r2 {

struct CacheCounters {
  int64_t hits = 0, misses = 0, prefetch_issued = 0, prefetch_used = 0, prefetch_wasted = 0, loads = 0;
  int64_t pred_correct = 0, pred_total = 0;
  int64_t copies_failed = 0;   // copies that could not start or completed with an error (slot invalidated)
  std::vector<int64_t> layer_misses;
};

class ExpertCachePolicy {
 public:
  struct Layer {
    std::vector<int> expert_in;     // [C] expert held by the slot (-1: empty)
    std::vector<int64_t> stamp;     // [C]
    std::vector<char> prefetched;   // [C]
    std::vector<int> slot_of;       // [E] slot of the expert (-1: not resident)
    std::vector<int> predicted;     // experts predicted for this layer in the current token
    bool has_pred = false;
  };

  void init(int n_layers, int n_experts, int slots) {
    E_ = n_experts;
    C_ = slots;
    layers_.assign(n_layers, Layer{});
    warm();
  }

  // Warm start and zero counters.
  void warm() {
    clock_ = 0;
    for (Layer& L : layers_) {
      L.expert_in.assign(C_, -1);
      L.stamp.assign(C_, 0);
      L.prefetched.assign(C_, 0);
      L.slot_of.assign(E_, -1);
      for (int e = 0; e < C_; ++e) {
        L.expert_in[e] = e;
        L.stamp[e] = e - C_;
        L.slot_of[e] = e;
      }
      L.predicted.clear();
      L.has_pred = false;
    }
    cnt_ = CacheCounters{};
    cnt_.layer_misses.assign(layers_.size(), 0);
  }

  // Predictions belong to one token: forget them once its step is done.
  void end_token() {
    for (Layer& L : layers_) {
      L.predicted.clear();
      L.has_pred = false;
    }
  }

  // Layer `l` runs with the needed experts need[0..k).  slot_out[j] receives
  // the slot of need[j]; load_out[j] is set when that expert must be copied
  // into the slot (a miss).
  void use(int l, const int* need, int k, int* slot_out, bool* load_out) {
    Layer& L = layers_[l];
    if (L.has_pred) {
      cnt_.pred_total += (int64_t)L.predicted.size();
      for (int e : L.predicted)
        if (std::find(need, need + k, e) != need + k) ++cnt_.pred_correct;
    }
    for (int j = 0; j < k; ++j) {
      load_out[j] = false;
      const int s = L.slot_of[need[j]];
      slot_out[j] = s;
      if (s < 0) continue;
      ++cnt_.hits;
      if (L.prefetched[s]) {
        L.prefetched[s] = 0;
        ++cnt_.prefetch_used;
      }
      L.stamp[s] = ++clock_;
    }
    for (int j = 0; j < k; ++j) {
      if (slot_out[j] >= 0) continue;
      ++cnt_.misses;
      ++cnt_.layer_misses[l];
      const int e = need[j];
      auto excluded = [&](int x) {
        return std::find(need, need + k, x) != need + k ||
               std::find(L.predicted.begin(), L.predicted.end(), x) != L.predicted.end();
      };
      auto needed = [&](int x) { return std::find(need, need + k, x) != need + k; };
      int s = victim(L, excluded);
      if (s < 0) s = victim(L, needed);
      slot_out[j] = place(L, s, e);
      load_out[j] = true;
    }
  }

  // Experts fixed in HBM without replacement (the first strategy the paper
  // compares with, Sec. 3.3): experts 0..C-k-1 stay in slots 0..C-k-1 (where
  // the warm start put them); every other needed expert is a miss and goes,
  // at every use, into staging slot C-k+j, j its rank among the layer's
  // misses.  No stamps move.
  void use_fixed(int l, const int* need, int k, int* slot_out, bool* load_out) {
    const int fixed = C_ - k;
    int j = 0;
    for (int i = 0; i < k; ++i) {
      if (need[i] < fixed) {
        ++cnt_.hits;
        slot_out[i] = need[i];
        load_out[i] = false;
      } else {
        ++cnt_.misses;
        ++cnt_.layer_misses[l];
        ++cnt_.loads;
        slot_out[i] = fixed + j++;
        load_out[i] = true;
      }
    }
  }

  // Experts pred[0..n) (entries < 0 ignored) are predicted for layer l.
  // For each expert that must be copied, its slot is appended to slots_out
  // and the expert to experts_out.
  void predict(int l, const int* pred, int n, std::vector<int>* slots_out, std::vector<int>* experts_out) {
    Layer& L = layers_[l];
    L.predicted.clear();
    for (int j = 0; j < n; ++j)
      if (pred[j] >= 0) L.predicted.push_back(pred[j]);
    L.has_pred = true;
    for (int e : L.predicted) {
      const int s0 = L.slot_of[e];
      if (s0 >= 0) {
        L.stamp[s0] = ++clock_;
        continue;
      }
      auto excluded = [&](int x) { return std::find(L.predicted.begin(), L.predicted.end(), x) != L.predicted.end(); };
      int s = victim(L, excluded);
      if (s < 0) s = victim(L, [](int) { return false; });
      s = place(L, s, e);
      L.prefetched[s] = 1;
      ++cnt_.prefetch_issued;
      slots_out->push_back(s);
      experts_out->push_back(e);
    }
  }

  // The copy into slot s of layer l failed (it could not start, or completed
  // with an error): the slot holds no expert any more and is the first taken
  // by the next placement; a later use of the expert it was to hold is a
  // miss, loaded on demand.
  void invalidate(int l, int s) {
    Layer& L = layers_[l];
    const int e = L.expert_in[s];
    if (e >= 0) L.slot_of[e] = -1;
    L.expert_in[s] = -1;
    L.prefetched[s] = 0;
    ++cnt_.copies_failed;
  }

  // Place needed expert need[j] of layer l, which is not resident (its
  // earlier copy failed after the hit was counted), as a load: the victim
  // rules of use(); returns the slot.
  int place_needed(int l, const int* need, int k, int j) {
    Layer& L = layers_[l];
    auto excluded = [&](int x) {
      return std::find(need, need + k, x) != need + k ||
             std::find(L.predicted.begin(), L.predicted.end(), x) != L.predicted.end();
    };
    auto needed = [&](int x) { return std::find(need, need + k, x) != need + k; };
    int s = victim(L, excluded);
    if (s < 0) s = victim(L, needed);
    return place(L, s, need[j]);
  }

  const CacheCounters& counters() const { return cnt_; }
  const Layer& layer(int l) const { return layers_[l]; }
  int slots() const { return C_; }

 private:
  // Empty slot, else the occupied slot with the oldest stamp whose expert is
  // not excluded; -1 if every occupant is excluded.
  template <class Excl>
  int victim(const Layer& L, Excl excluded) const {
    for (int s = 0; s < C_; ++s)
      if (L.expert_in[s] < 0) return s;
    int best = -1;
    for (int s = 0; s < C_; ++s) {
      if (excluded(L.expert_in[s])) continue;
      if (best < 0 || L.stamp[s] < L.stamp[best]) best = s;
    }
    return best;
  }

  int place(Layer& L, int s, int e) {
    const int old = L.expert_in[s];
    if (old >= 0) {
      if (L.prefetched[s]) ++cnt_.prefetch_wasted;
      L.slot_of[old] = -1;
    }
    L.prefetched[s] = 0;
    L.expert_in[s] = e;
    L.slot_of[e] = s;
    L.stamp[s] = ++clock_;
    ++cnt_.loads;
    return s;
  }

  int E_ = 0, C_ = 0;
  int64_t clock_ = 0;
  std::vector<Layer> layers_;
  CacheCounters cnt_;
};

}  // namespace m2r2
