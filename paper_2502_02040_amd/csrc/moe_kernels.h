// Mixture-of-experts kernels of the M2R2 decode step (Sec. 2.3.3): the
// slow row is routed (softmax over all experts, top-k, unrenormalised
// weights) and runs its k experts out of the HBM expert cache; the fast row's
// MLP is a rank-r adapter; after layer i the fast row predicts the experts of
// layers 2i+2 and 2i+3 with those layers' routers.
#pragma once
#include "step_kernels.h"

namespace m2r2 {

constexpr int kMaxExperts = 256;
constexpr int kMaxTopK = 16;

struct MoePtrs {
  const float* logits;    // [3][E]: router logits of the slow row, predictions for 2i+2, 2i+3
  int* sel;               // [3][kMaxTopK] chosen / predicted experts
  float* prob;            // [kMaxTopK] router probabilities of the chosen experts
  int* sel_host;          // mapped host memory: [3][kMaxTopK] + sequence word
  float* act;             // [kMaxTopK][F_e] prob * silu(g) * u of each chosen expert
};

// Kernel: router logits.  rows [0, E) of `router` applied to the slow row
// (gain g_mlp, rms from the bins of the o projection) -> out[0..E).  Also used
// for the predictions: `row` selects the residual row, `gain` the target
// layer's mlp norm, `stat_layer` the bins holding that row's sum of squares.
// grid = ceil(E/16) (x n_tasks), block = 512.
struct RouterTask {
  const void* packed;     // packed router [E][d]
  const float* gain;      // [d]
  int row;                // residual row of X
  int stat_kind;          // 0: bins of the o projection of stat_layer, 1: bins entering stat_layer
  int stat_layer;
  float* out;             // [E]
};

// One 16-row tile of one task (workgroup `b` of tiles x n_tasks); AGENT: the
// logits are stored at agent scope (read by another workgroup of the launch).
template <int WB, bool AGENT>
__device__ __forceinline__ void router_tile(const Dims& D, int E, const RouterTask& t0, const RouterTask& t1,
                                            const RouterTask& t2, int n_tasks, const WS& ws, int b) {
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ const float* xrow_s[kMaxRows];
  __shared__ float inv_rms;
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  const int tiles = (E + 15) / 16;
  const int task = b / tiles, tile = b % tiles;
  if (task >= n_tasks) return;
  const RouterTask T = task == 0 ? t0 : (task == 1 ? t1 : t2);
  const void* wrow[1] = {(const char*)T.packed + (size_t)tile * 16 * D.d * (WB ? 2 : 4)};
  GemvWave<WB, 1, 2, true> gw;
  gw.begin(wrow, D.d);
  if (threadIdx.x == 0) {
    xrow_s[0] = ws.X + (size_t)T.row * D.d;
    float a = 0.f;
    for (int b = 0; b < kBinSlots; ++b)
      a += T.stat_kind == 0 ? bin_o_at(ws, D, T.stat_layer, b, T.row)[0] : bin_d_at(ws, T.stat_layer, b, T.row)[0];
    inv_rms = rsqrtf(a / D.d + D.eps);
  }
  __syncthreads();
  f32x4_t acc[1];
  gw.run(xrow_s, T.gain, 1, dyn, acc);
  gemv_reduce<1>(acc, 1, red, y);
  if (threadIdx.x < 16 && tile * 16 + (int)threadIdx.x < E) {
    float* o = T.out + tile * 16 + threadIdx.x;
    const float v = y[threadIdx.x] * inv_rms;
    if constexpr (AGENT) st_agent(o, v);
    else *o = v;
  }
}

template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_router(Dims D, int E, RouterTask t0, RouterTask t1, RouterTask t2,
                                                         int n_tasks, WS ws) {
  router_tile<WB, false>(D, E, t0, t1, t2, n_tasks, ws, blockIdx.x);
}

// Words of the mapped host block that k_topk fills.
constexpr int kHostSeq = 3 * kMaxTopK;       // sequence number, written last
constexpr int kHostExited = 3 * kMaxTopK + 1;
constexpr int kHostWords = 64;

// Kernel: top-k of up to three logit vectors (one workgroup).  Task 0 (if
// `route`) is the slow row's routing: softmax over all experts, then the k
// largest probabilities (ties to the lower id) and their unrenormalised
// weights.  Tasks 1, 2 are predictions: top-k of the logits.  Nothing is
// chosen once the sequence has exited.  The ids are also written to mapped
// host memory (when given), then `seq` with release semantics at system scope.
// Wave t takes task t: every logit is ranked at once against the task's
// logits in LDS (its place in the order larger value first, then lower id),
// and a logit of rank < k is chosen at that rank (a NaN ranks as -inf).
// AGENT: the logits were stored by other workgroups of the same launch.  Run
// by a whole workgroup of at least 256 threads.
template <bool AGENT>
__device__ __forceinline__ void topk_body(int E, int K, const float* logits, int route, int n_pred, const MoePtrs& mp,
                                          const WS& ws, int* slow_out, int* pred_out, int seq) {
  __shared__ int chosen[3][kMaxTopK];
  __shared__ float pr[kMaxTopK];
  __shared__ float lv[3][kMaxExperts];
  const bool exited = ws.exited[0] != 0;
  if (exited) { route = 0; n_pred = 0; }
  // lane l holds experts l, l+64, l+128, l+192
  constexpr int J = kMaxExperts / 64;
  const int lane = threadIdx.x & 63, t = threadIdx.x >> 6;
  const bool active = t < 3 && (t == 0 ? route != 0 : (t - 1) < n_pred);
  float v[J];
  float mx = -INFINITY, sum = 1.f;
  if (active) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int e = lane + 64 * j;
      const float x = e < E ? (AGENT ? ld_agent(logits + t * E + e) : logits[t * E + e]) : -INFINITY;
      v[j] = x == x ? x : -INFINITY;
      lv[t][e] = v[j];
    }
    if (t == 0) {
      float lm = v[0];
#pragma unroll
      for (int j = 1; j < J; ++j) lm = fmaxf(lm, v[j]);
      mx = wave_max(lm);
      float se = 0.f;
#pragma unroll
      for (int j = 0; j < J; ++j)
        if (lane + 64 * j < E) se += __expf(v[j] - mx);
      sum = wave_sum(se);
    }
  }
  if (t < 3 && lane < K) chosen[t][lane] = -1;
  __syncthreads();
  if (active) {
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int e = lane + 64 * j;
      if (e < E) {
        int rk = 0;
        for (int e2 = 0; e2 < E; ++e2) {
          const float w = lv[t][e2];
          rk += (w > v[j] || (w == v[j] && e2 < e)) ? 1 : 0;
        }
        if (rk < K) {
          chosen[t][rk] = e;
          if (t == 0) pr[rk] = __expf(v[j] - mx) / sum;
        }
      }
    }
  }
  __syncthreads();
  if (threadIdx.x < 3 * K) {
    const int t = threadIdx.x / K, k = threadIdx.x % K;
    const bool active = t == 0 ? route != 0 : (t - 1) < n_pred;
    if (active) {
      mp.sel[t * kMaxTopK + k] = chosen[t][k];
      if (t == 0) mp.prob[k] = pr[k];
      if (t == 0 && slow_out) slow_out[k] = chosen[t][k];
      if (t > 0 && pred_out) pred_out[(t - 1) * K + k] = chosen[t][k];
    }
  }
  if (mp.sel_host) {
    // one word per thread, then the sequence number with release semantics
    const int i = threadIdx.x;
    if (i < 3 * K)
      __hip_atomic_store(&mp.sel_host[(i / K) * kMaxTopK + i % K], chosen[i / K][i % K], __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_SYSTEM);
    else if (i == 3 * K)
      __hip_atomic_store(&mp.sel_host[kHostExited], exited ? 1 : 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    __threadfence_system();
    __syncthreads();
    if (i == 0) __hip_atomic_store(&mp.sel_host[kHostSeq], seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}
__global__ __launch_bounds__(256) void k_topk(int E, int K, const float* logits, int route, int n_pred, MoePtrs mp,
                                              WS ws, int* slow_out, int* pred_out, int seq) {
  topk_body<false>(E, K, logits, route, n_pred, mp, ws, slow_out, pred_out, seq);
}

// Kernel: the fast row's MLP of a mixture-of-experts layer, the rank-r
// adapter alone: p += (rms(p) * g_mlp . A_m^T) B_m^T, with the adapter-down
// sums taken from the bins of the o projection; then the partial sums of
// the next layer's norm and of the exit signal.  grid = ceil(d/256), block = 256.
// Block `blk` of the fast row's MLP (T threads per block).
template <int T>
__device__ __forceinline__ void fast_mlp_block(const Dims& D, const RowMap& rm, const LayerPtrs& L, int layer,
                                               const WS& ws, int blk) {
  __shared__ float um[kMaxRank];
  __shared__ float red[T / 64];
  const int nn = blk * T + threadIdx.x;
  const int bin = blk % kBins;
  for (int m = 0; m < rm.M; ++m) {
    if (!rm.fast[m]) continue;
    const bool ex = ws.exited[rm.seq[m]] != 0;
    if (threadIdx.x < D.r) {
      float a = 0.f, ss = 0.f;
      for (int b = 0; b < kBinSlots; ++b) {
        a += bin_o_at(ws, D, layer, b, m)[1 + threadIdx.x];
        ss += bin_o_at(ws, D, layer, b, m)[0];
      }
      um[threadIdx.x] = a * rsqrtf(ss / D.d + D.eps);
    }
    __syncthreads();
    float x = 0.f, p = 0.f;
    if (nn < D.d) {
      x = ws.X[(size_t)m * D.d + nn];
      p = ws.PIN[(size_t)m * D.d + nn];
      if (!ex && L.A[4] && L.B[4]) {
        x += dot_row(L.B[4], nn, D.r, um, D.wbf16);
        ws.X[(size_t)m * D.d + nn] = x;
      }
    }
    const float s0 = block_sum(x * x, red);
    const float s1 = block_sum(p * x, red);
    const float s2 = block_sum(p * p, red);
    if (threadIdx.x == 0) {
      add_agent(bin_d_at(ws, layer + 1, bin, m) + 0, s0);
      add_agent(bin_d_at(ws, layer + 1, bin, m) + 1, s1);
      add_agent(bin_d_at(ws, layer + 1, bin, m) + 2, s2);
    }
    __syncthreads();
  }
}
__global__ __launch_bounds__(256) void k_fast_mlp(Dims D, RowMap rm, LayerPtrs L, int layer, WS ws) {
  fast_mlp_block<256>(D, rm, L, layer, ws, blockIdx.x);
}

// Kernel: the router tiles of up to three tasks (tiles x n_tasks workgroups,
// as k_router), then, in the last of them to finish, the top-k of every task
// (k_topk's work; `cnt` counts the arrivals and is left at zero).  With
// `fmlp_blocks` > 0 the workgroups after the router tiles run the fast row's
// MLP (k_fast_mlp's work): only when no task reads the fast row.
// grid = tiles x n_tasks + fmlp_blocks, block = 512.
template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_route(Dims D, int E, RouterTask t0, RouterTask t1, RouterTask t2,
                                                        int n_tasks, WS ws, int K, MoePtrs mp, int* slow_out,
                                                        int* pred_out, int seq, uint32_t* cnt, RowMap rm, LayerPtrs L,
                                                        int layer) {
  __shared__ int last;
  const int nr = ((E + 15) / 16) * n_tasks;
  if ((int)blockIdx.x >= nr) {
    fast_mlp_block<kGemvThreads>(D, rm, L, layer, ws, (int)blockIdx.x - nr);
    return;
  }
  router_tile<WB, true>(D, E, t0, t1, t2, n_tasks, ws, blockIdx.x);
  if (!arrive_last(cnt, (uint32_t)nr, &last)) return;
  topk_body<true>(E, K, t0.out, 1, n_tasks - 1, mp, ws, slow_out, pred_out, seq);
}

// Kernel: sum of squares of residual row `row` into the bins entering layer
// `next` (a layer whose MLP is skipped after an exit leaves the slow row
// unchanged; the cache entries of the following layers still normalise it).
// grid = 1, block = 256.
__global__ __launch_bounds__(256) void k_row_stats(Dims D, int row, int next, WS ws) {
  __shared__ float red[4];
  float ss = 0.f;
  for (int i = threadIdx.x; i < D.d; i += 256) {
    const float x = ws.X[(size_t)row * D.d + i];
    ss += x * x;
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) add_agent(bin_d_at(ws, next, 0, row), ss);
}

// Slot pointers of the k chosen experts (packed gate, up and down matrices).
struct ExpertSlots {
  const void* w[kMaxTopK];   // start of the expert: gate [F_e][d], up [F_e][d], down [d][F_e], each packed
};

// Device-side slot resolution: slot_tab[layer][expert] is the HBM cache slot
// whose copy of the expert is complete, or -1.  The host keeps it in stream
// order: an evicted expert is cleared before any later launch can read it, a
// newly copied one is published only once its copy has completed.
struct SlotTable {
  const int* tab;      // [n_layers][E]
  const char* slots;   // [n_layers][C][stride]
  size_t stride;
  int E, C;
};

// Slot lookup from the table: lane k of every wave gets the slot of chosen
// expert k (two dependent loads).  False, for every workgroup alike, when the
// sequence has exited or a chosen expert is not published; the host then
// launches the kernels again with its own addresses.
__device__ __forceinline__ bool spec_slot(const SlotTable& t, const MoePtrs& mp, const WS& ws, int layer, int K,
                                          int& slot) {
  const int lane = threadIdx.x & 63;
  const int ex = ws.exited[0];
  const int e = lane < K ? mp.sel[lane] : 0;
  slot = lane < K ? ((e >= 0 && e < t.E) ? t.tab[(size_t)layer * t.E + e] : -1) : 0;
  return !ex && !__any(lane < K && (slot < 0 || slot >= t.C));
}
__device__ __forceinline__ const char* slot_addr(const SlotTable& t, int layer, int slot) {
  return t.slots + ((size_t)layer * t.C + slot) * t.stride;
}

// Kernel: table entries idx[i] = val[i], i < n (one launch per batch of host
// decisions, in stream order).
struct TabUpdates {
  int n;
  int idx[30];
  int val[30];
};
__global__ __launch_bounds__(64) void k_tab_set(int* tab, TabUpdates u) {
  if ((int)threadIdx.x < u.n) tab[u.idx[threadIdx.x]] = u.val[threadIdx.x];
}

// Kernel: gate/up of the chosen experts for the slow row, SwiGLU, times the
// router probability.  grid = K * F_e/16, block = 512.
// With every expert resident (`hits` non-null) the first workgroup also
// counts the layer's K cache hits on the device.
template <int WB, bool SPEC = false>
__global__ __launch_bounds__(kGemvThreads) void k_moe_gateup(Dims D, int Fe, int K, ExpertSlots es, int slow_row,
                                                             const float* mlp_norm, int layer, MoePtrs mp, WS ws,
                                                             SlotTable stab, unsigned long long* hits = nullptr) {
  int sslot = 0;
  if constexpr (SPEC)
    if (!spec_slot(stab, mp, ws, layer, K, sslot)) return;
  if (hits && blockIdx.x == 0 && threadIdx.x == 0) atomicAdd(hits, (unsigned long long)K);
  __shared__ float red[kGemvWaves * 512];
  __shared__ float y[512];
  __shared__ const float* xrow_s[kMaxRows];
  __shared__ float inv_rms;
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  const int tiles = Fe / 16;
  const int k = blockIdx.x / tiles, t = blockIdx.x % tiles;
  const size_t esz = WB ? 2 : 4;
  const char* base = SPEC ? slot_addr(stab, layer, __shfl(sslot, k)) : (const char*)es.w[k];
  const size_t mat = (size_t)Fe * D.d * esz;
  const void* wrow[2] = {base + (size_t)t * 16 * D.d * esz, base + mat + (size_t)t * 16 * D.d * esz};
  GemvWave<WB, 2, 2, true> gw;
  gw.begin(wrow, D.d);
  if (threadIdx.x == 0) {
    xrow_s[0] = ws.X + (size_t)slow_row * D.d;
    float a = 0.f;
    for (int b = 0; b < kBinSlots; ++b) a += bin_o_at(ws, D, layer, b, slow_row)[0];
    inv_rms = rsqrtf(a / D.d + D.eps);
  }
  __syncthreads();
  f32x4_t acc[2];
  gw.run(xrow_s, mlp_norm, 1, dyn, acc);
  gemv_reduce<2>(acc, 1, red, y);
  if (threadIdx.x < 16) {
    const float g = y[threadIdx.x] * inv_rms, u = y[256 + threadIdx.x] * inv_rms;
    mp.act[(size_t)k * Fe + t * 16 + threadIdx.x] = mp.prob[k] * silu(g) * u;
  }
}

// Kernel: down projections of the chosen experts summed into the slow row
// (the K experts' matrices form one reduction of length K*F_e over the
// probability-weighted activations), then the slow row's partial sums for the
// next layer's norm.  grid = d/16, block = 512.
// `stats_on_exit`: once the sequence has exited, the first workgroup adds the
// slow row's sum of squares for the next layer instead (k_row_stats' work,
// for a token enqueued without the host seeing the exit).
template <int WB, bool SPEC = false>
__global__ __launch_bounds__(kGemvThreads) void k_moe_down(Dims D, int Fe, int K, ExpertSlots es, int slow_row,
                                                           int layer, MoePtrs mp, WS ws, SlotTable stab,
                                                           int stats_on_exit = 0) {
  int sslot = 0;
  if constexpr (SPEC)
    if (!spec_slot(stab, mp, ws, layer, K, sslot)) {
      if (stats_on_exit && ws.exited[0] && blockIdx.x == 0) {
        __shared__ float sred[kGemvWaves];
        float ss = 0.f;
        for (int i = threadIdx.x; i < D.d; i += kGemvThreads) {
          const float x = ws.X[(size_t)slow_row * D.d + i];
          ss += x * x;
        }
        ss = wave_sum(ss);
        if ((threadIdx.x & 63) == 0) sred[threadIdx.x >> 6] = ss;
        __syncthreads();
        if (threadIdx.x == 0) {
          float a = 0.f;
          for (int w = 0; w < kGemvWaves; ++w) a += sred[w];
          add_agent(bin_d_at(ws, layer + 1, 0, slow_row), a);
        }
      }
      return;
    }
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float newx[16];
  __shared__ const float* xrow_s[kMaxRows];
  __shared__ const char* segs[kMaxTopK];
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  const int n0 = blockIdx.x * 16;
  const size_t esz = WB ? 2 : 4;
  const size_t mat = (size_t)Fe * D.d * esz;
  if (threadIdx.x < K)   // lanes of the first wave: lane k holds expert k's slot
    segs[threadIdx.x] = (SPEC ? slot_addr(stab, layer, sslot) : (const char*)es.w[threadIdx.x]) + 2 * mat +
                        (size_t)blockIdx.x * 16 * Fe * esz;
  if (threadIdx.x == 0) xrow_s[0] = mp.act;
  __syncthreads();
  GemvWave<WB, 1, 2, false> gw;
  gw.seg = segs;
  gw.seg_steps = Fe / (WB ? 32 : 16);
  const void* first[1] = {segs[0]};
  gw.begin(first, K * Fe);
  f32x4_t acc[1];
  gw.run(xrow_s, nullptr, 1, dyn, acc);
  gemv_reduce<1>(acc, 1, red, y);
  if (threadIdx.x < 16) {
    const int nn = n0 + threadIdx.x;
    float x = ws.X[(size_t)slow_row * D.d + nn];
    if (!ws.exited[0]) {
      x += y[threadIdx.x];
      ws.X[(size_t)slow_row * D.d + nn] = x;
    }
    newx[threadIdx.x] = x;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float v = 0.f;
    for (int i = 0; i < 16; ++i) v += newx[i] * newx[i];
    add_agent(bin_d_at(ws, layer + 1, blockIdx.x % kBins, slow_row), v);
  }
}

}  // namespace m2r2
