// Host scheduler of expert copies (Sec. 2.3.3, App. B): the placements of
// ExpertCachePolicy turned into copies through a copy engine, with the
// handling of copies that fail.  The GPU runtime's engine copies from the
// pinned host store on side streams and tracks each slot's last copy with an
// event; the host tests drive the same scheduler with a fake engine that
// delays copies, refuses them, or completes them with an error.
//
// Rules:
//  - prefetch(l, P): the policy's predictions for layer l become copies; a
//    copy that cannot start is dropped and its slot invalidated (the expert
//    is then not resident, and its use becomes an on-demand load);
//  - acquire(l, S): the needed experts' slots; the misses are loaded on
//    demand.  A needed expert whose copy (a prefetch, or an earlier load)
//    completed with an error is invalidated and loaded again on demand;
//  - a demand copy that cannot start is an error (there is no other copy to
//    fall back to): acquire returns false, and the slots of that copy and of
//    the layer's demand copies not started after it are invalidated;
//  - a copy still in flight when acquire runs is waited for by the layer's
//    compute; its failure is an error of the step (on the GPU, the device's
//    error state, reported by the next call).
#pragma once
#include "expert_cache.h"

namespace m2r2 {

class ExpertCopyEngine {
 public:
  enum State { kDone = 0, kPending = 1, kFailed = -1 };
  virtual ~ExpertCopyEngine() = default;
  // Start copying expert e of layer l into slot s (demand: a miss of the
  // layer about to run; else a prefetch).  False: nothing was enqueued.
  virtual bool start(int l, int s, int e, bool demand) = 0;
  // State of the last copy started into slot s of layer l (kDone if none).
  virtual State state(int l, int s) = 0;
};

class ExpertScheduler {
 public:
  ExpertScheduler(ExpertCachePolicy& pol, ExpertCopyEngine& eng) : pol_(pol), eng_(eng) {}

  void prefetch(int l, const int* pred, int n) {
    slots_.clear();
    experts_.clear();
    pol_.predict(l, pred, n, &slots_, &experts_);
    for (size_t q = 0; q < slots_.size(); ++q)
      if (!eng_.start(l, slots_[q], experts_[q], false)) pol_.invalidate(l, slots_[q]);
  }

  // slot_out[j]: the slot of need[j]; load_out[j]: a demand copy was started
  // for it.  Needed slots may still have copies in flight (kPending): the
  // caller orders the layer's compute after them.
  bool acquire(int l, const int* need, int k, int* slot_out, bool* load_out) {
    pol_.use(l, need, k, slot_out, load_out);
    for (int j = 0; j < k; ++j) {
      if (load_out[j] || eng_.state(l, slot_out[j]) != ExpertCopyEngine::kFailed) continue;
      pol_.invalidate(l, slot_out[j]);
      slot_out[j] = pol_.place_needed(l, need, k, j);
      load_out[j] = true;
    }
    for (int j = 0; j < k; ++j) {
      if (load_out[j] && !eng_.start(l, slot_out[j], need[j], true)) {
        // this copy and the later ones, which are then not started, leave
        // their slots empty
        for (int i = j; i < k; ++i)
          if (load_out[i]) pol_.invalidate(l, slot_out[i]);
        return false;
      }
    }
    return true;
  }

 private:
  ExpertCachePolicy& pol_;
  ExpertCopyEngine& eng_;
  std::vector<int> slots_, experts_;
};

}  // namespace m2r2
