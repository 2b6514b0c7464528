// Host test of the expert-copy scheduler (expert_sched.h) with a fake copy
// engine: copies that take several polls to complete, copies refused when
// they are started, and copies that complete with an error.  Built with g++
// under AddressSanitizer/UndefinedBehaviorSanitizer, and under
// ThreadSanitizer with copies completed by a worker thread
// (tests/test_expert_sched_host.py).  Prints "ok" and exits 0 on success.
#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <thread>
#include <vector>

#include "expert_sched.h"

using namespace m2r2;

#define CHECK(c)                                                          \
  do {                                                                    \
    if (!(c)) {                                                           \
      std::fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      std::exit(1);                                                       \
    }                                                                     \
  } while (0)

struct Faults {
  double refuse_prefetch = 0, refuse_demand = 0, fail_prefetch = 0;
  int max_delay = 0;       // polls (or worker microseconds) before a copy completes
  bool threaded = false;   // a worker thread completes the copies
};

class FakeEngine final : public ExpertCopyEngine {
 public:
  FakeEngine(int L, int C, const Faults& f, unsigned seed) : C_(C), f_(f), rng_(seed), slots_(L * C) {
    if (f_.threaded) worker_ = std::thread([this] { work(); });
  }
  ~FakeEngine() override {
    stop_ = true;
    if (worker_.joinable()) worker_.join();
  }
  bool start(int l, int s, int e, bool demand) override {
    Slot& x = slots_[l * C_ + s];
    if (u() < (demand ? f_.refuse_demand : f_.refuse_prefetch)) {
      ++refused;
      return false;
    }
    x.expert = e;
    x.fail = !demand && u() < f_.fail_prefetch;
    x.delay = f_.max_delay ? (int)(rng_() % (unsigned)(f_.max_delay + 1)) : 0;
    x.t0 = std::chrono::steady_clock::now();
    x.st.store(kPending);
    ++started;
    if (x.fail) ++failing;
    return true;
  }
  State state(int l, int s) override {
    Slot& x = slots_[l * C_ + s];
    if (!f_.threaded && x.st.load() == kPending && x.delay-- <= 0) x.st.store(x.fail ? kFailed : kDone);
    return (State)x.st.load();
  }
  // The compute waits for a slot's copy (the runtime's stream wait).
  State wait(int l, int s) {
    State st;
    while ((st = state(l, s)) == kPending) std::this_thread::yield();
    return st;
  }
  int expert_copied(int l, int s) const { return slots_[l * C_ + s].expert; }
  int refused = 0, started = 0, failing = 0;

 private:
  struct Slot {
    std::atomic<int> st{kDone};
    int expert = -1, delay = 0;
    bool fail = false;
    std::chrono::steady_clock::time_point t0;
  };
  double u() { return std::uniform_real_distribution<double>(0.0, 1.0)(rng_); }
  void work() {   // completes pending copies once their delay (microseconds) has passed
    while (!stop_) {
      const auto now = std::chrono::steady_clock::now();
      for (Slot& x : slots_) {
        if (x.st.load(std::memory_order_acquire) != kPending) continue;
        if (now - x.t0 >= std::chrono::microseconds(x.delay)) x.st.store(x.fail ? kFailed : kDone, std::memory_order_release);
      }
      std::this_thread::yield();
    }
  }
  int C_;
  Faults f_;
  std::mt19937 rng_;
  std::vector<Slot> slots_;
  std::atomic<bool> stop_{false};
  std::thread worker_;
};

struct Result {
  CacheCounters cnt;
  int refused = 0, started = 0, failing = 0, acquire_failed = 0;
  int late_failures = 0;   // copies in flight when acquire ran that then failed: an error of the step
};

// T tokens of an N-layer model with E experts, C slots per layer, K per
// token and layer; predictions for layers 2i+2, 2i+3 after layer i (the true
// choice with probability `hit`, else a random one), as the fast stream makes.
Result run(int T, int N, int E, int C, int K, double hit, const Faults& f, unsigned seed, bool expect_ok) {
  std::mt19937 rng(seed);
  auto choose = [&]() {
    std::vector<int> p(E);
    for (int i = 0; i < E; ++i) p[i] = i;
    std::shuffle(p.begin(), p.end(), rng);
    p.resize(K);
    return p;
  };
  std::vector<std::vector<std::vector<int>>> route(T, std::vector<std::vector<int>>(N));
  for (auto& tk : route)
    for (auto& r : tk) r = choose();
  ExpertCachePolicy pol;
  pol.init(N, E, C);
  FakeEngine eng(N, C, f, seed ^ 0x9e3779b9u);
  ExpertScheduler sched(pol, eng);
  Result res;
  std::vector<int> slot(K);
  std::vector<char> load_c(K);
  for (int t = 0; t < T; ++t) {
    for (int l = 0; l < N; ++l) {
      const std::vector<int>& need = route[t][l];
      bool load[64];
      const bool ok = sched.acquire(l, need.data(), K, slot.data(), load);
      if (!ok) {
        ++res.acquire_failed;
        CHECK(!expect_ok);
        // the demand copy that could not start left its slot empty
        int empty = 0;
        for (int j = 0; j < K; ++j) empty += pol.layer(l).expert_in[slot[j]] < 0;
        CHECK(empty >= 1);
        continue;
      }
      for (int j = 0; j < K; ++j) {
        // the policy holds the needed expert in its slot, slots are distinct
        CHECK(slot[j] >= 0 && slot[j] < C);
        CHECK(pol.layer(l).expert_in[slot[j]] == need[j]);
        CHECK(pol.layer(l).slot_of[need[j]] == slot[j]);
        for (int i = 0; i < j; ++i) CHECK(slot[i] != slot[j]);
        // the slot's data is the needed expert once its copy completed: a
        // copy that had failed was replaced by a demand load in acquire; one
        // still in flight then is waited for, and its failure is an error of
        // the step (the runtime reports the device's error state)
        const ExpertCopyEngine::State st = eng.wait(l, slot[j]);
        if (st == ExpertCopyEngine::kFailed) {
          CHECK(f.fail_prefetch > 0 && (f.threaded || f.max_delay > 0));
          ++res.late_failures;
          pol.invalidate(l, slot[j]);
          continue;
        }
        CHECK(st == ExpertCopyEngine::kDone);
        const int copied = eng.expert_copied(l, slot[j]);
        CHECK(copied == need[j] || (copied < 0 && need[j] == slot[j]));   // (never copied: the warm start)
      }
      // predictions for layers 2l+2, 2l+3
      for (int lp = 2 * l + 2; lp <= 2 * l + 3 && lp < N; ++lp) {
        std::vector<int> p = choose();
        for (int j = 0; j < K; ++j)
          if (std::uniform_real_distribution<double>(0, 1)(rng) < hit) {
            const int e = route[t][lp][j];
            if (std::find(p.begin(), p.end(), e) == p.end()) p[j] = e;
          }
        std::sort(p.begin(), p.end());
        p.erase(std::unique(p.begin(), p.end()), p.end());
        sched.prefetch(lp, p.data(), (int)p.size());
      }
    }
    pol.end_token();
  }
  res.cnt = pol.counters();
  res.refused = eng.refused;
  res.started = eng.started;
  res.failing = eng.failing;
  return res;
}

int main(int argc, char** argv) {
  const bool threaded = argc > 1 && std::string(argv[1]) == "threaded";
  const int T = threaded ? 40 : 200, N = 8, E = 32, C = 12, K = 4;
  Faults none;
  none.threaded = threaded;
  const Result base = run(T, N, E, C, K, 0.6, none, 7, true);
  CHECK(base.cnt.hits + base.cnt.misses == (int64_t)T * N * K);
  CHECK(base.cnt.copies_failed == 0 && base.acquire_failed == 0);
  CHECK(base.cnt.loads == base.started);

  // delayed copies: the logical hits do not depend on when copies complete
  Faults slow = none;
  slow.max_delay = threaded ? 200 : 5;
  const Result r_slow = run(T, N, E, C, K, 0.6, slow, 7, true);
  CHECK(r_slow.cnt.hits == base.cnt.hits && r_slow.cnt.misses == base.cnt.misses);
  CHECK(r_slow.cnt.loads == base.cnt.loads && r_slow.cnt.prefetch_issued == base.cnt.prefetch_issued);

  // prefetches refused when started: every slot is invalidated, every use is
  // still served (on demand), and every refusal is counted
  Faults refuse = slow;
  refuse.refuse_prefetch = 0.3;
  const Result r_ref = run(T, N, E, C, K, 0.6, refuse, 7, true);
  CHECK(r_ref.refused > 0);
  CHECK(r_ref.cnt.copies_failed == r_ref.refused);
  CHECK(r_ref.cnt.hits + r_ref.cnt.misses == (int64_t)T * N * K);

  // prefetches that complete with an error before their layer runs: a used
  // one is invalidated and loaded again on demand (counted); unused ones are
  // simply replaced
  Faults fail = none;
  fail.fail_prefetch = 0.3;
  const Result r_fail = run(T, N, E, C, K, 0.6, fail, 11, true);
  CHECK(r_fail.failing > 0 && r_fail.cnt.copies_failed > 0 && r_fail.cnt.copies_failed <= r_fail.failing);
  CHECK(r_fail.cnt.hits + r_fail.cnt.misses == (int64_t)T * N * K);
  CHECK(threaded || r_fail.late_failures == 0);
  // ... and with delays: failures of copies still in flight are the step's
  Faults fail_late = slow;
  fail_late.fail_prefetch = 0.3;
  const Result r_late = run(T, N, E, C, K, 0.6, fail_late, 17, true);
  CHECK(r_late.cnt.copies_failed + r_late.late_failures <= r_late.failing + r_late.late_failures);

  // an on-demand copy that cannot start is an error of the layer
  Faults dem = slow;
  dem.refuse_demand = 0.2;
  const Result r_dem = run(T, N, E, C, K, 0.6, dem, 13, false);
  CHECK(r_dem.acquire_failed > 0);

  std::printf("ok: %s; base hits %lld misses %lld loads %lld; refused prefetches %d; failed prefetches %d "
              "(%lld invalidated when used); with delays %d failed, %d of them after their layer had started "
              "waiting; refused demand copies %d\n",
              threaded ? "threaded engine" : "polled engine", (long long)base.cnt.hits, (long long)base.cnt.misses,
              (long long)base.cnt.loads, r_ref.refused, r_fail.failing, (long long)r_fail.cnt.copies_failed,
              r_late.failing, r_late.late_failures, r_dem.acquire_failed);
  return 0;
}
