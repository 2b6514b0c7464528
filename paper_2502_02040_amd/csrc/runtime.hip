// Host runtime and C ABI of the M2R2 decode path (see include/m2r2.h).
#include <hip/hip_runtime.h>

#include <immintrin.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "expert_cache.h"
#include "expert_sched.h"
#include "m2r2.h"
#include "m2r2_measure.h"
#include "moe_kernels.h"
#include "step_kernels.h"
#include "sk_kernels.h"
#include "sk_attn.h"
#include "rw_kernels.h"
#include "arla.h"
#include "persist.h"
#include "flops.h"

using namespace m2r2;

// Scratch of m2r2_decode_step_noalloc: the per-call scratch block of a
// context (residual rows, row statistics, attention partials, arg-max
// partials, arrival counters) placed in this file-scope device array instead
// of the context's workspace.  Every GPU the library runs on holds its own
// copy until the process ends; all such calls on one GPU share it.  Host code
// never passes the array's name to a kernel (on the host it is only a
// stand-in symbol): its device address is looked up once per device with
// hipGetSymbolAddress and used instead.
constexpr size_t kNoAllocScratchBytes = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};   // device address of `scratch` on each device, once looked up

// Look up the device address of `scratch` on device `dev` (current) once.
hipError_t scratch_setup(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev]) return hipSuccess;
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e == hipSuccess) g_scratch_ptr[dev] = p;
  return e;
}

void* scratch_ptr(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  return g_scratch_ptr[dev];
}

__global__ void k_fill_u32(uint32_t* p, int n, uint32_t v) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = v;
}

thread_local std::string g_err;

m2r2_status fail(m2r2_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                                   \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) return fail(M2R2_E_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

constexpr int kPerMaxBase = kScoreCap;

int per_max(int rows) { return (kPerMaxBase / std::max(rows, 1)) & ~15; }

// Context splits of the attention for `nseq` sequences of `rows` rows each:
// at least about 256 workgroups in total, at most 128 tokens per split (the
// attention kernel puts 128 tokens of keys and values in flight before it
// forms q), at least as many as the LDS score buffer requires, at most 63
// (the merge holds 64 partials).
int choose_splits(int nseq, int rows, int H, int max_ctx) {
  const int target = std::max(1, (256 + nseq * H - 1) / (nseq * H));
  const int prefetched = std::max(1, (max_ctx + 127) / 128);
  const int need = std::max(1, (max_ctx + per_max(rows) - 1) / per_max(rows));
  return std::min(63, std::max(need, std::max(target, prefetched)));
}

struct Layout {
  size_t packed;                         // start of the packed projection matrices
  std::vector<size_t> lay_off;           // per layer: pq pk pv pa po pg pu pd (8 offsets)
  size_t lm;                             // packed LM head
  size_t X, PIN, QKV, O, ACT, bin_d, bin_o, bin_gu, uo, att, att_cnt, lm_val, lm_idx, lm_cnt, exited, exitb,
      reinit, err, sig, arla_kv, arla_q, arla_sig, arla_cnt, rope, sk_part, sk_cnt, total;
  size_t fsc, fqkv, lrz;                 // FLOPs-optimised fast stream: slow scores, fast q/k/v, low-rank head
  size_t scratch_begin, counters_begin, scratch_end;   // per-call scratch [begin, end), counters [counters_begin, end)
  size_t pk_sd, pk_so, pk_sgu, pk_bar, pk_rel, layers_d;   // one-launch step: statistics slots, barrier, layer table
  int pk_so_w, pk_sgu_w;
  // mixture of experts: router logits, choices, probabilities, activations,
  // and the expert cache ([n_layers][slots] slots of expert_stride bytes)
  size_t moe_logits, moe_sel, moe_prob, moe_act, moe_slots, moe_tab, moe_hits;
  size_t expert_bytes, expert_stride;
  int TD, TF, TV, S_max;
  size_t sk_slots;                       // partial-sum slots of the stream-K GEMVs
  int lm_slots;                          // arg-max partial slots (per LM-head tile or workgroup)
};

bool is_moe(const m2r2_config& c) { return c.n_experts > 0; }
bool is_flops(const m2r2_config& c) {
  return c.fast_heads > 0 || c.fast_topk > 0 || c.fast_mlp_adapter != 0 || c.head_rank > 0;
}

// Packed gate + up ([F_e][d] each) + down ([d][F_e]).
size_t expert_bytes_of(const m2r2_config& c) {
  const int wb = c.wdtype == M2R2_BF16;
  return 2 * packed_bytes(c.expert_ffn, c.d_model, wb) + packed_bytes(c.d_model, c.expert_ffn, wb);
}

// Workgroups the GPU holds at once for each tile GEMV kernel (filled at
// context creation from the occupancy of the kernel with its LDS):
// index [wb][row class 0: 2 rows, 1: 16 rows][kernel 0 qkv, 1 o, 2 gate/up,
// 3 down, 4 head].
struct Resident {
  int n[2][3][5];
};

// Row classes of the tile GEMVs: up to 2, 8 or 16 activation rows staged.
constexpr int row_class(int mt) { return mt <= 2 ? 0 : (mt <= 8 ? 2 : 1); }

// ---- stream-K GEMV plans ----------------------------------------------------
constexpr int kSkMaxWaves = 8 * 320;   // partial slots are sized for up to 320 compute units
constexpr int kSkMinLds = 82 * 1024;   // dynamic LDS of every stream-K launch: one workgroup per compute unit
constexpr int kLmMinSlots = 1024;      // arg-max slots: at least one per workgroup of a one-per-compute-unit launch

SkPlan sk_plan(int ntiles, int nblk, int W, bool pair) {
  SkPlan p{};
  p.ntiles = ntiles;
  p.nblk = nblk;
  p.W = W;
  const long long T = (long long)ntiles * nblk;
  // equal ranges over all waves, but long enough that a tile has at most
  // kSkMaxSeg segments (small matrices leave waves idle)
  long long L = std::max({1LL, (T + W - 1) / W, (long long)(nblk + kSkMaxSeg - 2) / (kSkMaxSeg - 1)});
  if (pair && (L & 1)) ++L;
  p.L = (int)L;
  int smax = 1;
  for (int t = 0; t < ntiles; ++t)
    smax = std::max(smax, std::min(sk_last_wave(p, t), W - 1) - sk_first_wave(p, t) + 1);
  p.smax = smax;
  return p;
}

// Plans of the five matrix kinds: 0 qkv (+ adapter-down rows), 1 o, 2 gate/up pairs, 3 down, 4 LM head.
void sk_plans(const m2r2_config& c, int W, SkPlan (&out)[5]) {
  const int kstep = c.wdtype == M2R2_BF16 ? 32 : 16;
  const int d = c.d_model, q = c.n_heads * c.head_dim, r = c.rank, F = std::max(c.ffn, kstep);
  out[0] = sk_plan(3 * ((q + 15) / 16) + (3 * r + 15) / 16, d / kstep, W, false);
  out[1] = sk_plan((d + 15) / 16, q / kstep, W, false);
  out[2] = sk_plan((F + 15) / 16, 2 * (d / kstep), W, true);
  out[3] = sk_plan((d + 15) / 16, F / kstep, W, false);
  out[4] = sk_plan((c.vocab + 15) / 16, d / kstep, W, false);
}

size_t sk_slot_bound(const m2r2_config& c) {
  if (c.n_experts > 0) return 0;
  size_t n = 0;
  for (int W : {kSkMaxWaves, 8 * 256, 8 * 128, 8 * 64}) {
    SkPlan p[5];
    sk_plans(c, W, p);
    for (const SkPlan& x : p) n = std::max(n, (size_t)x.ntiles * x.smax);
  }
  return n;
}

Layout make_layout(const m2r2_config& c, int max_batch, int max_chunk, int max_ctx) {
  Layout L{};
  const int d = c.d_model, qdim = c.n_heads * c.head_dim, r = c.rank;
  const int nqkv = 3 * qdim + 3 * r;
  L.TD = (d + 15) / 16;
  L.TF = (c.ffn + 15) / 16;
  L.TV = (c.vocab + 15) / 16;
  int smax = 1;
  for (int nseq = 1; nseq <= max_batch; ++nseq) {
    smax = std::max(smax, choose_splits(nseq, 2, c.n_heads, max_ctx));
    smax = std::max(smax, choose_splits(nseq, 1, c.n_heads, max_ctx));
  }
  smax = std::max(smax, choose_splits(1, max_chunk, c.n_heads, max_ctx));
  L.S_max = smax;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) & ~(size_t)255;
    return o;
  };
  const int wb = c.wdtype == M2R2_BF16;
  L.packed = 0;
  const bool moe = is_moe(c);
  for (int l = 0; l < c.n_layers; ++l) {
    L.lay_off.push_back(take(packed_bytes(qdim, d, wb)));
    L.lay_off.push_back(take(packed_bytes(qdim, d, wb)));
    L.lay_off.push_back(take(packed_bytes(qdim, d, wb)));
    L.lay_off.push_back(take(packed_bytes(3 * r, d, wb)));
    L.lay_off.push_back(take(packed_bytes(d, qdim, wb)));
    if (moe) {   // slot 5: the router; 6, 7 unused
      L.lay_off.push_back(take(packed_bytes(c.n_experts, d, wb)));
      L.lay_off.push_back(0);
      L.lay_off.push_back(0);
    } else {
      L.lay_off.push_back(take(2 * packed_bytes(c.ffn, d, wb)));   // gate and up, interleaved tile pairs
      L.lay_off.push_back(0);
      L.lay_off.push_back(take(packed_bytes(d, c.ffn, wb)));
    }
  }
  L.lm = take(packed_bytes(c.vocab, d, wb));
  // ---- per-call scratch: one contiguous block (the no-allocation decode
  // step rebases exactly this block onto its static device array)
  L.scratch_begin = off;
  L.X = take(sizeof(float) * kMaxRows * d);
  L.PIN = take(sizeof(float) * kMaxRows * d);
  L.QKV = take(sizeof(float) * kMaxRows * nqkv);
  L.O = take(sizeof(float) * kMaxRows * qdim);
  L.ACT = take(sizeof(float) * kMaxRows * std::max(c.ffn, 1));
  L.bin_d = take(sizeof(float) * (c.n_layers + 1) * kBinSlots * kMaxRows * 4);
  L.bin_o = take(sizeof(float) * c.n_layers * kBinSlots * kMaxRows * (1 + 2 * r));
  L.bin_gu = take(sizeof(float) * c.n_layers * kBinSlots * kMaxRows * std::max(r, 1));
  L.uo = take(sizeof(float) * kMaxRows * c.n_heads * std::max(r, 1));
  L.att = take(sizeof(float) * (size_t)std::max(max_batch, 1) * c.n_heads * (smax + 1) * kMaxRows *
               (c.head_dim + 2 + r));
  // per-tile (or, for the row-per-wave head, per-workgroup) arg-max partials
  L.lm_slots = std::max(L.TV, kLmMinSlots);
  L.lm_val = take(sizeof(float) * L.lm_slots * kMaxRows);
  L.lm_idx = take(sizeof(int) * L.lm_slots * kMaxRows);
  L.exited = take(sizeof(int) * kMaxSeq);
  L.exitb = take(sizeof(int) * kMaxSeq);
  L.reinit = take(sizeof(int) * c.n_layers * kMaxSeq);
  L.sig = take(sizeof(float) * kMaxSeq * c.n_layers);
  L.arla_kv = take(sizeof(float) * 2 * c.n_layers * 2 * kArlaDim);   // after each layer, then at each gate
  L.arla_q = take(sizeof(float) * kArlaDim);
  L.arla_sig = take(sizeof(float) * kMaxSeq);
  L.sk_slots = sk_slot_bound(c);
  L.sk_part = take(sizeof(float) * 64 * std::max<size_t>(L.sk_slots, 1));
  // the one-launch step's per-workgroup statistics slots
  L.pk_so_w = (2 + 2 * r + 3) & ~3;
  L.pk_sgu_w = (r + 3) & ~3;
  L.pk_sd = take(sizeof(float) * kPkMaxWG * kPkSdW);
  L.pk_so = take(sizeof(float) * kPkMaxWG * L.pk_so_w);
  L.pk_sgu = take(sizeof(float) * kPkMaxWG * L.pk_sgu_w);
  // FLOPs-optimised fast stream (one sequence)
  const int fh = c.fast_heads > 0 ? c.fast_heads : c.n_heads;
  const bool flops = c.fast_heads > 0 || c.fast_topk > 0 || c.fast_mlp_adapter || c.head_rank > 0;
  L.fsc = take(flops ? sizeof(float) * (size_t)fh * max_ctx : 0);
  L.fqkv = take(flops ? sizeof(float) * (size_t)fh * 3 * c.head_dim : 0);
  L.lrz = take(sizeof(float) * std::max(c.head_rank, 1));
  // arrival counters (zero between passes: the last arriver resets them)
  L.counters_begin = off;
  L.att_cnt = take(sizeof(uint32_t) * kMaxSeq * c.n_heads);
  L.lm_cnt = take(sizeof(uint32_t));
  L.arla_cnt = take(sizeof(uint32_t));
  L.sk_cnt = take(sizeof(uint32_t) * (65 + std::max({L.TD, L.TF, L.TV, 3 * ((qdim + 15) / 16) + (3 * r + 15) / 16})));
  L.pk_bar = take(sizeof(uint32_t) * kPkRelStride * kPkGroups);
  L.pk_rel = take(sizeof(uint32_t) * kPkRelStride * kPkGroups);
  L.scratch_end = off;
  // ---- context state: sticky error bits, RoPE table, expert cache
  L.err = take(sizeof(int));
  L.layers_d = take(sizeof(LayerPtrs) * c.n_layers);
  L.rope = take(sizeof(float) * 2 * (size_t)max_ctx * (c.head_dim / 2));
  if (moe) {
    L.moe_logits = take(sizeof(float) * 3 * c.n_experts);
    L.moe_sel = take(sizeof(int) * 3 * kMaxTopK);
    L.moe_prob = take(sizeof(float) * kMaxTopK);
    L.moe_act = take(sizeof(float) * (size_t)c.top_k * c.expert_ffn);
    L.expert_bytes = expert_bytes_of(c);
    L.expert_stride = (L.expert_bytes + 255) & ~(size_t)255;
    L.moe_slots = take(L.expert_stride * c.n_layers * c.expert_slots);
    L.moe_tab = take(sizeof(int) * c.n_layers * c.n_experts);
    L.moe_hits = take(256);   // device hit counter (offset 0), arrival counter of k_route (offset 128)
  }
  L.total = off;
  return L;
}

m2r2_status check_config(const m2r2_config* c, int max_batch, int max_chunk, int max_ctx) {
  if (!c) return fail(M2R2_E_INVALID, "config is NULL");
  if (c->wdtype != M2R2_F32 && c->wdtype != M2R2_BF16) return fail(M2R2_E_DTYPE, "wdtype %d", c->wdtype);
  if (c->kvdtype != M2R2_F32 && c->kvdtype != M2R2_BF16) return fail(M2R2_E_DTYPE, "kvdtype %d", c->kvdtype);
  const int kstep = c->wdtype == M2R2_BF16 ? 32 : 16;
  if (c->n_layers < 1 || c->n_layers > 127) return fail(M2R2_E_SHAPE, "n_layers %d not in [1,127]", c->n_layers);
  if (c->d_model <= 0 || c->d_model % kstep) return fail(M2R2_E_SHAPE, "d_model %d not a multiple of %d", c->d_model, kstep);
  if (c->n_experts < 0) return fail(M2R2_E_SHAPE, "n_experts %d", c->n_experts);
  if (!is_moe(*c) && (c->ffn <= 0 || c->ffn % kstep))
    return fail(M2R2_E_SHAPE, "ffn %d not a multiple of %d", c->ffn, kstep);
  if (is_moe(*c)) {
    if (c->n_experts > kMaxExperts) return fail(M2R2_E_SHAPE, "n_experts %d > %d", c->n_experts, kMaxExperts);
    if (c->top_k < 1 || c->top_k > kMaxTopK || c->top_k > c->n_experts)
      return fail(M2R2_E_SHAPE, "top_k %d not in [1, min(%d, n_experts)]", c->top_k, kMaxTopK);
    if (c->expert_ffn <= 0 || c->expert_ffn % kstep)
      return fail(M2R2_E_SHAPE, "expert_ffn %d not a multiple of %d", c->expert_ffn, kstep);
    if (c->expert_slots < c->top_k || c->expert_slots > c->n_experts)
      return fail(M2R2_E_SHAPE, "expert_slots %d not in [top_k, n_experts]", c->expert_slots);
    if (max_batch != 1) return fail(M2R2_E_UNSUPPORTED, "mixture-of-experts decoding takes max_batch 1");
  }
  if (c->head_dim != 64 && c->head_dim != 96 && c->head_dim != 128)
    return fail(M2R2_E_UNSUPPORTED, "head_dim %d (supported: 64, 96, 128)", c->head_dim);
  if (c->n_heads < 1 || (c->n_heads * c->head_dim) % kstep)
    return fail(M2R2_E_SHAPE, "n_heads*head_dim %d not a multiple of %d", c->n_heads * c->head_dim, kstep);
  if (c->rank < 1 || c->rank > kMaxRank) return fail(M2R2_E_SHAPE, "rank %d not in [1,%d]", c->rank, kMaxRank);
  if (std::max({c->d_model, c->n_heads * c->head_dim, c->ffn}) > 16384)
    return fail(M2R2_E_UNSUPPORTED, "reduction length above 16384 (activation rows are held in LDS)");
  if (c->vocab < 1) return fail(M2R2_E_SHAPE, "vocab %d", c->vocab);
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail(M2R2_E_INVALID, "rms_eps/rope_theta");
  if (max_batch < 1 || max_batch > 8) return fail(M2R2_E_SHAPE, "max_batch %d not in [1,8]", max_batch);
  if (max_chunk < 1 || max_chunk > kMaxRows) return fail(M2R2_E_SHAPE, "max_chunk %d not in [1,16]", max_chunk);
  if (max_ctx < 1) return fail(M2R2_E_SHAPE, "max_ctx %d", max_ctx);
  if (c->fast_heads < 0 || c->fast_heads > c->n_heads)
    return fail(M2R2_E_SHAPE, "fast_heads %d not in [0, n_heads]", c->fast_heads);
  if (c->fast_topk < 0) return fail(M2R2_E_SHAPE, "fast_topk %d", c->fast_topk);
  if (c->fast_mlp_adapter != 0 && c->fast_mlp_adapter != 1)
    return fail(M2R2_E_INVALID, "fast_mlp_adapter %d not 0 or 1", c->fast_mlp_adapter);
  if (c->head_rank < 0 || c->head_rank > 256) return fail(M2R2_E_SHAPE, "head_rank %d not in [0,256]", c->head_rank);
  if (is_flops(*c)) {
    if (is_moe(*c)) return fail(M2R2_E_UNSUPPORTED, "the FLOPs-optimised fast stream is for dense models");
    if (max_ctx > kFaMaxCtx)
      return fail(M2R2_E_UNSUPPORTED, "FLOPs-optimised fast stream: max_ctx %d above %d", max_ctx, kFaMaxCtx);
  }
  return M2R2_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

// Host side of the expert cache of a mixture-of-experts context.
struct MoeState {
  bool on = false;
  int E = 0, K = 0, Fe = 0, C = 0;
  size_t ebytes = 0, stride = 0;
  const char* store_h = nullptr;   // pinned host store [n_layers][E][ebytes]
  char* slots_d = nullptr;         // [n_layers][C][stride]
  std::vector<const void*> router; // packed router per layer
  MoePtrs mp{};
  int* host_words = nullptr;       // mapped host block written by k_topk
  int seq = 0;
  int policy = M2R2_MOE_AHEAD_OF_TIME;
  std::vector<int> preload;        // [preload_tokens][n_layers][K] random-preload draws
  int preload_tokens = 0;
  int64_t token = 0;               // decode steps since the last warm start
  ExpertCachePolicy pol;
  std::vector<hipEvent_t> slot_ev;   // [n_layers*C] last copy into the slot
  std::vector<char> slot_pending;    // a copy was recorded and not yet seen complete
  std::vector<hipEvent_t> layer_done;  // [n_layers] the layer's expert kernels, recorded on the compute stream
  std::vector<char> layer_done_rec;
  hipStream_t copy_demand = nullptr, copy_ahead = nullptr;
  int64_t h2d_bytes = 0, copy_waits = 0, host_wait_ns = 0;
  // device-side slot resolution: the expert kernels are launched right after
  // the routing kernels and read the slots from tab_d; the host launches them
  // again with its own slots only when a chosen expert is not published there
  bool spec = true;
  int* tab_d = nullptr;             // [n_layers][E] slot of a completed copy, or -1
  std::vector<int> tab;             // tab_d once every enqueued update has run
  std::vector<int> tab_idx, tab_val;   // updates still to enqueue
  struct Pending { int l, slot, e; };
  std::vector<Pending> pend;        // copies published once they are complete
  // a cache of E slots under the LRU policy holds every expert: tokens are
  // enqueued whole, without waiting for any routing, and the expert kernel
  // counts the hits on the device
  unsigned long long* hits_d = nullptr;
  bool hits_dev_used = false;       // hits_d may be non-zero
  uint32_t* route_cnt_d = nullptr;  // arrivals of the router workgroups (k_route), zero between launches
};

struct m2r2_ctx {
  m2r2_config cfg;
  int device = 0;   // the device the context was created on
  char* ws_base = nullptr;   // the workspace
  Dims D;
  Layout lay;
  std::vector<LayerPtrs> layers;
  const void* embed;
  const float* final_norm;
  const void* lm_head;   // packed
  const void* lm_head_rm;   // the caller's row-major LM head
  const void* head_a = nullptr;   // low-rank head of the FLOPs-optimised fast stream (or NULL)
  const void* head_b = nullptr;
  std::vector<const void*> fmlp_a, fmlp_b;   // its adapter-only fast MLP: A_m, B_m per layer
  int max_batch, max_chunk, max_ctx;
  WS ws;
  // kernel timing (measurement only)
  Resident resident;
  // stream-K GEMVs of the one- and two-row class
  bool sk_on = false;
  int sk_grid = 0;
  int sk_attn_S = 0;   // splits of the stream-K path's attention (0: the general attention kernel)
  bool rw_on = false;  // row-per-wave GEMVs for the one- and two-row class
  int rw_nch[3] = {0, 0, 0};   // 1 KB pieces per row for reductions over d, qdim, ffn
  int rw_nw[2] = {8, 8};       // waves per workgroup of the o and down projections
  int attn_chunks = 0;         // batched short-chain attention: 128-token chunks per split (0: by size)
  // one-launch decode step (one sequence, one or two rows): instantiation,
  // grid (one workgroup per compute unit), attention splits per head, LDS
  struct {
    int kind = -1;   // index into M2R2_PK_SHAPES, -1: not available
    int grid = 0, S = 0;
    size_t lds = 0;
    float *sd = nullptr, *so = nullptr, *sgu = nullptr;
    uint32_t *bar = nullptr, *rel = nullptr;
    const LayerPtrs* layers_d = nullptr;
  } pk;
  SkPlan sk[5];
  SkWS skws{};
  int timed_class = -1;
  std::vector<hipEvent_t> ev;   // pairs
  int ev_used = 0;
  MoeState moe;
  // latent-attention exit router weights (borrowed device pointers; on = set)
  struct {
    bool on = false;
    const char* wq = nullptr;
    const char* wk = nullptr;
    const char* wv = nullptr;
    const float* w_out = nullptr;
    const float* b_out = nullptr;
  } arla;
};

namespace {

m2r2_status check_kv(const m2r2_ctx* c, const m2r2_kv* kv) {
  if (!kv || !kv->k_pages || !kv->v_pages || !kv->block_table_d || !kv->seq_lens_d)
    return fail(M2R2_E_INVALID, "kv descriptor or one of its pointers is NULL");
  if (kv->num_blocks < 1 || kv->block_size < 1 || kv->max_blocks_per_seq < 1)
    return fail(M2R2_E_SHAPE, "kv sizes");
  if (!aligned16(kv->k_pages) || !aligned16(kv->v_pages)) return fail(M2R2_E_INVALID, "kv pages not 16-byte aligned");
  (void)c;
  return M2R2_OK;
}

KVPtrs kv_ptrs(const m2r2_kv* kv) {
  return KVPtrs{kv->k_pages, kv->v_pages, kv->block_table_d, kv->seq_lens_d, kv->num_blocks, kv->block_size,
                kv->max_blocks_per_seq};
}

constexpr int kMaxTimed = 1024;

// Launch `fn` bracketed by timing events when its class is being timed.
template <class F>
m2r2_status timed(m2r2_ctx* c, int cls, hipStream_t st, F&& fn) {
  const bool on = c->timed_class == cls && c->ev_used < kMaxTimed;
  if (on) {
    if ((int)c->ev.size() < 2 * (c->ev_used + 1)) {
      hipEvent_t a, b;
      HIP_TRY(hipEventCreate(&a));
      HIP_TRY(hipEventCreate(&b));
      c->ev.push_back(a);
      c->ev.push_back(b);
    }
    HIP_TRY(hipEventRecord(c->ev[2 * c->ev_used], st));
  }
  fn();
  if (on) {
    HIP_TRY(hipEventRecord(c->ev[2 * c->ev_used + 1], st));
    ++c->ev_used;
  }
  return M2R2_OK;
}

#define TIMED(cls, launch)                                                   \
  do {                                                                       \
    if (m2r2_status s_ = timed(c, cls, st, [&]() { launch; })) return s_;   \
  } while (0)

// Grid sizes and dynamic LDS of the tile GEMV launches of one pass.
struct Grids {
  int qkv, o, gu, head;
  size_t l_d, l_q, l_f;   // LDS for reduction lengths d, H*hd, ffn
};

template <int WB, int MT>
Grids grids(const m2r2_ctx* c) {
  const Dims& D = c->D;
  const int* cap = c->resident.n[WB][row_class(MT)];
  Grids g;
  g.qkv = std::min(3 * (D.qdim / 16) + (3 * D.r + 15) / 16, cap[0]);
  g.o = std::min(D.d / 16, std::min(cap[1], cap[3]));
  g.gu = std::min(std::max(D.F / 16, 1), cap[2]);
  g.head = std::min(c->lay.TV, cap[4]);
  g.l_d = tile_lds_bytes(WB, MT, D.d);
  g.l_q = tile_lds_bytes(WB, MT, D.qdim);
  g.l_f = tile_lds_bytes(WB, MT, std::max(D.F, 1));
  return g;
}

size_t sk_lds(int K) { return (size_t)std::max(sk_act_bytes(K), kSkMinLds); }

// ---- row-per-wave GEMVs: kernels instantiated for these piece counts per row
#define M2R2_RW_NCH(X) X(1) X(2) X(4) X(6) X(8) X(16)
bool rw_nch_ok(int n) {
#define M2R2_RW_CASE(N) if (n == N) return true;
  M2R2_RW_NCH(M2R2_RW_CASE)
#undef M2R2_RW_CASE
  return false;
}
#define M2R2_RW_LAUNCHER(NAME, ...)                                                                     \
  template <int WB, class... A>                                                                       \
  void NAME##_launch(int nch, int grid, size_t lds, hipStream_t st, A... args) {                      \
    switch (nch) {                                                                                    \
      case 1: NAME<WB, 1, 1><<<grid, kRwThreads, lds, st>>>(args...); break;                          \
      case 2: NAME<WB, 2, 1><<<grid, kRwThreads, lds, st>>>(args...); break;                          \
      case 4: NAME<WB, 4, 1><<<grid, kRwThreads, lds, st>>>(args...); break;                          \
      case 6: NAME<WB, 6, 1><<<grid, kRwThreads, lds, st>>>(args...); break;                          \
      case 8: NAME<WB, 8, 1><<<grid, kRwThreads, lds, st>>>(args...); break;                          \
      case 16: NAME<WB, 8, 2><<<grid, kRwThreads, lds, st>>>(args...); break;                         \
    }                                                                                                 \
  }
M2R2_RW_LAUNCHER(kr_qkv)
M2R2_RW_LAUNCHER(kr_gateup)
M2R2_RW_LAUNCHER(kr_head)
// o projection and down projection: 8 or 12 waves per workgroup (12 when the
// rows then split evenly over the waves, as d = 3072 over 256 x 12 does)
#define M2R2_RW_LAUNCHER_NW(NAME)                                                                      \
  template <int WB, int NW, class... A>                                                               \
  void NAME##_launch_w(int nch, int grid, size_t lds, hipStream_t st, A... args) {                    \
    switch (nch) {                                                                                    \
      case 1: NAME<WB, 1, 1, NW><<<grid, 64 * NW, lds, st>>>(args...); break;                         \
      case 2: NAME<WB, 2, 1, NW><<<grid, 64 * NW, lds, st>>>(args...); break;                         \
      case 4: NAME<WB, 4, 1, NW><<<grid, 64 * NW, lds, st>>>(args...); break;                         \
      case 6: NAME<WB, 6, 1, NW><<<grid, 64 * NW, lds, st>>>(args...); break;                         \
      case 8: NAME<WB, 8, 1, NW><<<grid, 64 * NW, lds, st>>>(args...); break;                         \
      case 16: NAME<WB, 8, 2, NW><<<grid, 64 * NW, lds, st>>>(args...); break;                        \
    }                                                                                                 \
  }                                                                                                   \
  template <int WB, class... A>                                                                       \
  void NAME##_launch(int nch, int nw, int grid, size_t lds, hipStream_t st, A... args) {              \
    if (nw == 12) NAME##_launch_w<WB, 12>(nch, grid, lds, st, args...);                               \
    else NAME##_launch_w<WB, 8>(nch, grid, lds, st, args...);                                         \
  }
M2R2_RW_LAUNCHER_NW(kr_oproj)
M2R2_RW_LAUNCHER_NW(kr_down)

// Exit router after layer l (l = -1: before layer 0) of a one-sequence dual
// step with the router on.  Row 0 is the slow row, row 1 the fast one.  The
// launch projects the fast state after l into the slots of the next gate b;
// at the layer before b also the query, and, while the slow row still holds
// the state the fast row restarts from at b, that state for the gate after
// b; before layer 0 the embedding for the first gate.  At b it scores.
bool host_is_gate(const StepIO& io, int b) {
  if (b <= 0 || b >= 128) return false;
  return b < 64 ? ((io.gate_mask_lo >> b) & 1ull) : ((io.gate_mask_hi >> (b - 64)) & 1ull);
}

template <int WB>
hipError_t arla_after(m2r2_ctx* c, const StepIO& io, int l, hipStream_t st) {
  if (!io.arla_sig) return hipSuccess;
  const int N = c->D.n_layers;
  auto next_gate = [&](int from) {
    while (from < N && !host_is_gate(io, from)) ++from;
    return from;
  };
  const int b = next_gate(l + 1);
  if (b >= N) return hipSuccess;   // no gate after this layer
  int first = l < 0 ? 0 : l;
  while (first > 0 && !host_is_gate(io, first)) --first;
  const size_t blk = (size_t)kArlaDim * c->D.d * (WB ? 2 : 4);
  const int slot = 2 * kArlaDim;
  ArlaArgs a{};
  a.w_out = c->arla.w_out + (size_t)b * kArlaDim;
  a.b_out = c->arla.b_out + b;
  a.layer = l;
  a.first = first;
  a.gate_now = l >= 0 && b == l + 1;
  auto job = [&](const char* w, int bnd, int row, int dst) { a.job[a.njobs++] = ArlaJob{w + bnd * blk, row, dst}; };
  if (l < 0) {
    job(c->arla.wk, b, 0, N * slot);
    job(c->arla.wv, b, 0, N * slot + kArlaDim);
  } else {
    job(c->arla.wk, b, 1, l * slot);
    job(c->arla.wv, b, 1, l * slot + kArlaDim);
  }
  if (a.gate_now) {
    job(c->arla.wq, b, 1, -1);
    const int b2 = next_gate(b + 1);
    if (b2 < N) {
      job(c->arla.wk, b2, 0, (N + b) * slot);
      job(c->arla.wv, b2, 0, (N + b) * slot + kArlaDim);
    }
  }
  k_arla<WB><<<a.njobs * (kArlaDim / kArlaWaves), kArlaThreads, 0, st>>>(c->D, c->ws, a);
  return hipGetLastError();
}

// The dual-stream step of one sequence in the FLOPs-optimised form (Sec. 2.5):
// the split attention leaves the fast row to k_fattn (kept heads, selected
// positions); with the adapter-only fast MLP, k_fast_mlp applies it and the
// gate/up and down kernels see the slow row alone; an exited fast row's
// token comes from the low-rank head.
template <int WB, int KB, int HD>
m2r2_status run_layers_flops(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int n_layers_run,
                             hipStream_t st) {
  const Dims& D = c->D;
  const int G = c->sk_grid;
  const size_t lds = (size_t)kSkMinLds;
  const int nd = c->rw_nch[0], nq = c->rw_nch[1], nf = c->rw_nch[2];
  const bool fattn = D.fh > 0 || D.ftk > 0;
  const int fh = D.fh > 0 ? D.fh : D.H;
  RowMap rs = rm;   // the slow row alone (row 0)
  rs.M = 1;
  rs.cnt[0] = 1;
  const RowMap& rmlp = D.fmlp ? rs : rm;
  for (int l = 0; l < n_layers_run; ++l) {
    const LayerPtrs& L = c->layers[l];
    // the o projection sums the MLP adapter's down-projection, k_fast_mlp
    // applies its up factor: both take it in the gate slot ([rank][d], [d][rank])
    LayerPtrs Lo = L;
    if (D.fmlp) {
      Lo.A[4] = c->fmlp_a[l];
      Lo.B[4] = c->fmlp_b[l];
    }
    TIMED(0, (kr_qkv_launch<WB>(nd, G, lds, st, D, L, rm, c->ws, io, l)));
    TIMED(1, (ks_attn<WB, KB, HD><<<dim3(c->sk_attn_S, D.H, rm.nseq), kSkAttnThreads,
                                     sk_attn_lds_bytes(HD, D.r, WB), st>>>(D, L, rm, c->ws, io, kv, l, c->sk_attn_S)));
    if (fattn)
      TIMED(1, (k_fattn<KB, HD><<<fh, kFaThreads, fattn_lds_bytes(c->max_ctx), st>>>(D, L, rm, c->ws, io, kv, l)));
    TIMED(2, (kr_oproj_launch<WB>(nq, c->rw_nw[0], G, lds, st, D, Lo, rm, c->ws, io, l)));
    if (D.fmlp) TIMED(10, (k_fast_mlp<<<(D.d + 255) / 256, 256, 0, st>>>(D, rm, Lo, l, c->ws)));
    TIMED(3, (kr_gateup_launch<WB>(nd, G, lds, st, D, L, rmlp, c->ws, io, l)));
    TIMED(4, (kr_down_launch<WB>(nf, c->rw_nw[1], G, lds, st, D, L, rmlp, c->ws, io, l)));
  }
  if (D.hr > 0)
    TIMED(5, (k_lr_z<WB><<<(D.hr + 7) / 8, 512, sizeof(float) * D.d, st>>>(D, c->final_norm, c->head_a, rm, c->ws)));
  TIMED(5, (kr_head_launch<WB>(nd, G, lds, st, D, c->lm_head_rm, c->final_norm, rm, c->ws, io, kv, c->skws,
                                n_layers_run, c->head_b)));
  HIP_TRY(hipGetLastError());
  return M2R2_OK;
}

bool has_fast_row(const RowMap& rm) {
  for (int m = 0; m < rm.M; ++m)
    if (rm.fast[m]) return true;
  return false;
}

// One or two rows: row-per-wave GEMVs and the short-chain attention.
template <int WB, int KB, int HD>
m2r2_status run_layers_rw(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int n_layers_run,
                          hipStream_t st) {
  const Dims& D = c->D;
  if (is_flops(c->cfg) && has_fast_row(rm)) return run_layers_flops<WB, KB, HD>(c, rm, io, kv, n_layers_run, st);
  const int G = c->sk_grid;
  const size_t lds = (size_t)kSkMinLds;
  const int nd = c->rw_nch[0], nq = c->rw_nch[1], nf = c->rw_nch[2];
  // attention: one 128-token chunk per split (two only when M2R2_ATTN_CHUNKS
  // asks for it: measured no faster at one sequence)
  const int S2 = c->attn_chunks == 2 ? (c->max_ctx + 2 * kSkAttnP - 1) / (2 * kSkAttnP) : 0;
  HIP_TRY(arla_after<WB>(c, io, -1, st));   // the first interval's restart state
  for (int l = 0; l < n_layers_run; ++l) {
    const LayerPtrs& L = c->layers[l];
    TIMED(0, (kr_qkv_launch<WB>(nd, G, lds, st, D, L, rm, c->ws, io, l)));
    if (S2 > 0)
      TIMED(1, (ks_attn<WB, KB, HD, 2><<<dim3(S2, D.H, rm.nseq), kSkAttnThreads, sk_attn_lds_bytes(HD, D.r, WB),
                                          st>>>(D, L, rm, c->ws, io, kv, l, S2)));
    else
      TIMED(1, (ks_attn<WB, KB, HD><<<dim3(c->sk_attn_S, D.H, rm.nseq), kSkAttnThreads,
                                       sk_attn_lds_bytes(HD, D.r, WB), st>>>(D, L, rm, c->ws, io, kv, l, c->sk_attn_S)));
    TIMED(2, (kr_oproj_launch<WB>(nq, c->rw_nw[0], G, lds, st, D, L, rm, c->ws, io, l)));
    TIMED(3, (kr_gateup_launch<WB>(nd, G, lds, st, D, L, rm, c->ws, io, l)));
    TIMED(4, (kr_down_launch<WB>(nf, c->rw_nw[1], G, lds, st, D, L, rm, c->ws, io, l)));
    HIP_TRY(arla_after<WB>(c, io, l, st));
  }
  TIMED(5, (kr_head_launch<WB>(nd, G, lds, st, D, c->lm_head_rm, c->final_norm, rm, c->ws, io, kv, c->skws,
                                n_layers_run, c->head_b)));
  HIP_TRY(hipGetLastError());
  return M2R2_OK;
}

// One or two rows: stream-K GEMVs, one workgroup per compute unit.
template <int WB, int KB, int HD>
m2r2_status run_layers_sk(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int n_layers_run,
                          hipStream_t st) {
  const Dims& D = c->D;
  int rows_per_seq = 1;
  for (int s = 0; s < rm.nseq; ++s) rows_per_seq = std::max(rows_per_seq, (int)rm.cnt[s]);
  const int S = choose_splits(rm.nseq, rows_per_seq, D.H, c->max_ctx);
  if (S > c->lay.S_max) return fail(M2R2_E_SHAPE, "attention splits exceed the workspace");
  if (S + 1 > 64) return fail(M2R2_E_SHAPE, "context too long for the attention merge (max_ctx %d)", c->max_ctx);
  const size_t smem = attn_smem_bytes();
  const int G = c->sk_grid;
  const size_t ld = sk_lds(D.d), lq = sk_lds(D.qdim), lf = sk_lds(D.F);
  const SkWS& sk = c->skws;
  HIP_TRY(arla_after<WB>(c, io, -1, st));   // the first interval's restart state
  for (int l = 0; l < n_layers_run; ++l) {
    const LayerPtrs& L = c->layers[l];
    TIMED(0, (ks_qkv<WB><<<G, kSkThreads, ld, st>>>(D, L, rm, c->ws, io, c->sk[0], sk, l)));
    if (c->sk_attn_S)
      TIMED(1, (ks_attn<WB, KB, HD><<<dim3(c->sk_attn_S, D.H, rm.nseq), kSkAttnThreads,
                                       sk_attn_lds_bytes(HD, D.r, WB), st>>>(D, L, rm, c->ws, io, kv, l, c->sk_attn_S)));
    else
      TIMED(1, (k_attn<KB, HD><<<dim3(S + 1, D.H, rm.nseq), kAttnThreads, smem, st>>>(D, L, rm, c->ws, io, kv, l, S)));
    TIMED(2, (ks_oproj<WB><<<G, kSkThreads, lq, st>>>(D, L, rm, c->ws, io, c->sk[1], sk, l)));
    TIMED(3, (ks_gateup<WB><<<G, kSkThreads, ld, st>>>(D, L, rm, c->ws, io, c->sk[2], sk, l)));
    TIMED(4, (ks_down<WB><<<G, kSkThreads, lf, st>>>(D, L, rm, c->ws, io, c->sk[3], sk, l)));
    HIP_TRY(arla_after<WB>(c, io, l, st));
  }
  TIMED(5, (ks_head<WB><<<G, kSkThreads, ld, st>>>(D, c->lm_head, c->final_norm, rm, c->ws, io, kv, c->sk[4], sk,
                                                   n_layers_run)));
  HIP_TRY(hipGetLastError());
  return M2R2_OK;
}

template <int WB, int KB, int HD, int MT>
m2r2_status run_layers_t(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int n_layers_run,
                         hipStream_t st) {
  if (is_flops(c->cfg) && has_fast_row(rm) && (rm.nseq != 1 || rm.M != 2 || !c->rw_on || !c->sk_attn_S))
    return fail(M2R2_E_UNSUPPORTED, "the FLOPs-optimised fast stream runs one sequence's dual-stream step on shapes "
                                    "whose rows are whole multiples of 1 KB");
  if constexpr (MT == 2) {
    if (c->rw_on) return run_layers_rw<WB, KB, HD>(c, rm, io, kv, n_layers_run, st);
    if (c->sk_on) return run_layers_sk<WB, KB, HD>(c, rm, io, kv, n_layers_run, st);
  }
  const Dims& D = c->D;
  const int nqkv = 3 * D.qdim + 3 * D.r;
  int rows_per_seq = 1;
  for (int s = 0; s < rm.nseq; ++s) rows_per_seq = std::max(rows_per_seq, (int)rm.cnt[s]);
  // one or two rows per sequence (batched decoding): the short-chain
  // attention with fixed splits; longer chunks: the general kernel
  const bool short_attn = c->sk_attn_S > 0 && rows_per_seq <= 2;
  // many splits in flight (batched long contexts): two 128-token chunks per
  // split, the second chunk's loads overlapping the first chunk's work
  const int NCA = c->attn_chunks != 0 ? c->attn_chunks
                  : ((long long)rm.nseq * D.H * c->sk_attn_S >= 8LL * c->sk_grid ? 2 : 1);
  const int S2 = short_attn && NCA > 1 ? (c->max_ctx + NCA * kSkAttnP - 1) / (NCA * kSkAttnP) : 0;
  const int S = choose_splits(rm.nseq, rows_per_seq, D.H, c->max_ctx);
  if (!short_attn && S > c->lay.S_max) return fail(M2R2_E_SHAPE, "attention splits exceed the workspace");
  if (!short_attn && S + 1 > 64)
    return fail(M2R2_E_SHAPE, "context too long for the attention merge (max_ctx %d)", c->max_ctx);
  const size_t smem = attn_smem_bytes();
  const Grids G = grids<WB, MT>(c);
  HIP_TRY(arla_after<WB>(c, io, -1, st));   // the first interval's restart state
  for (int l = 0; l < n_layers_run; ++l) {
    const LayerPtrs& L = c->layers[l];
    TIMED(0, (k_qkv<WB, MT><<<G.qkv, kGemvThreads, G.l_d, st>>>(D, L, rm, c->ws, io, l)));
    if (short_attn && S2 > 0 && NCA == 4)
      TIMED(1, (ks_attn<WB, KB, HD, 4><<<dim3(S2, D.H, rm.nseq), kSkAttnThreads, sk_attn_lds_bytes(HD, D.r, WB),
                                          st>>>(D, L, rm, c->ws, io, kv, l, S2)));
    else if (short_attn && S2 > 0)
      TIMED(1, (ks_attn<WB, KB, HD, 2><<<dim3(S2, D.H, rm.nseq), kSkAttnThreads, sk_attn_lds_bytes(HD, D.r, WB),
                                          st>>>(D, L, rm, c->ws, io, kv, l, S2)));
    else if (short_attn)
      TIMED(1, (ks_attn<WB, KB, HD><<<dim3(c->sk_attn_S, D.H, rm.nseq), kSkAttnThreads,
                                       sk_attn_lds_bytes(HD, D.r, WB), st>>>(D, L, rm, c->ws, io, kv, l, c->sk_attn_S)));
    else
      TIMED(1, (k_attn<KB, HD><<<dim3(S + 1, D.H, rm.nseq), kAttnThreads, smem, st>>>(D, L, rm, c->ws, io, kv, l, S)));
    TIMED(2, (k_oproj<WB, MT><<<G.o, kGemvThreads, G.l_q, st>>>(D, L, rm, c->ws, io, l)));
    TIMED(3, (k_gateup<WB, MT><<<G.gu, kGemvThreads, G.l_d, st>>>(D, L, rm, c->ws, io, l)));
    TIMED(4, (k_down<WB, MT><<<G.o, kGemvThreads, G.l_f, st>>>(D, L, rm, c->ws, io, l)));
    HIP_TRY(arla_after<WB>(c, io, l, st));
  }
  TIMED(5, (k_head<WB, MT><<<G.head, kGemvThreads, G.l_d, st>>>(D, c->lm_head, c->final_norm, rm, c->ws, io, kv,
                                                              c->lay.TV, n_layers_run)));
  HIP_TRY(hipGetLastError());
  return M2R2_OK;
}

template <int WB, int KB, int HD>
m2r2_status run_mt(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int nl, hipStream_t st) {
  if (rm.M <= 2) return run_layers_t<WB, KB, HD, 2>(c, rm, io, kv, nl, st);
  // up to 8 rows (a verification chunk of up to 7 drafts, a prefill tail):
  // half the activation rows to stage per tile
  if (rm.M <= 8) return run_layers_t<WB, KB, HD, 8>(c, rm, io, kv, nl, st);
  return run_layers_t<WB, KB, HD, 16>(c, rm, io, kv, nl, st);
}

template <int WB, int KB>
m2r2_status run_hd(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int nl, hipStream_t st) {
  switch (c->D.hd) {
    case 64: return run_mt<WB, KB, 64>(c, rm, io, kv, nl, st);
    case 96: return run_mt<WB, KB, 96>(c, rm, io, kv, nl, st);
    case 128: return run_mt<WB, KB, 128>(c, rm, io, kv, nl, st);
  }
  return fail(M2R2_E_UNSUPPORTED, "head_dim");
}

// Pack the projection matrices of every layer and the LM head into the
// workspace (null stream).
hipError_t pack_one(int wb, PackSrc src, int rows, int K, void* dst) {
  const size_t chunks = (size_t)((rows + 15) / 16) * (K / (wb ? 32 : 16)) * 64;
  const int grid = (int)std::min<size_t>(8192, (chunks + 255) / 256);
  if (wb) k_pack<1><<<grid, 256>>>(src, rows, K, dst);
  else k_pack<0><<<grid, 256>>>(src, rows, K, dst);
  return hipGetLastError();
}

hipError_t pack_all(m2r2_ctx* c, const m2r2_weights* w, void* workspace) {
  const m2r2_config& cf = c->cfg;
  const int wb = cf.wdtype == M2R2_BF16, d = cf.d_model, q = cf.n_heads * cf.head_dim, r = cf.rank, F = cf.ffn;
  char* b = (char*)workspace;
  auto one = [](const void* p, int rows) { return PackSrc{{p, nullptr, nullptr}, {rows, 0, 0}}; };
  hipError_t e = hipSuccess;
  for (int l = 0; l < cf.n_layers && e == hipSuccess; ++l) {
    const m2r2_layer_weights& L = w->layers[l];
    const size_t* o = &c->lay.lay_off[8 * l];
    e = pack_one(wb, one(L.wq, q), q, d, b + o[0]);
    if (e == hipSuccess) e = pack_one(wb, one(L.wk, q), q, d, b + o[1]);
    if (e == hipSuccess) e = pack_one(wb, one(L.wv, q), q, d, b + o[2]);
    if (e == hipSuccess) e = pack_one(wb, PackSrc{{L.A[0], L.A[1], L.A[2]}, {r, r, r}}, 3 * r, d, b + o[3]);
    if (e == hipSuccess) e = pack_one(wb, one(L.wo, d), d, q, b + o[4]);
    if (is_moe(cf)) {
      if (e == hipSuccess) e = pack_one(wb, one(L.router, cf.n_experts), cf.n_experts, d, b + o[5]);
      continue;
    }
    if (e == hipSuccess) {
      const size_t chunks = (size_t)((F + 15) / 16) * 2 * (d / (wb ? 32 : 16)) * 64;
      const int grid = (int)std::min<size_t>(8192, (chunks + 255) / 256);
      if (wb) k_pack_pair<1><<<grid, 256>>>(L.wg, L.wu, F, d, b + o[5]);
      else k_pack_pair<0><<<grid, 256>>>(L.wg, L.wu, F, d, b + o[5]);
      e = hipGetLastError();
    }
    if (e == hipSuccess) e = pack_one(wb, one(L.wd, d), d, F, b + o[7]);
  }
  if (e == hipSuccess) e = pack_one(wb, one(w->lm_head, cf.vocab), cf.vocab, d, b + c->lay.lm);
  return e;
}

// Allow the tile GEMV kernels the dynamic LDS they take (> 64 KB: resident
// rows of long reductions, 16-row chunk staging).
// and record how many workgroups of each the GPU holds at once.
template <int WB, int MT>
hipError_t set_lds_limits(const m2r2_config& c, Resident& res) {
  const int q = c.n_heads * c.head_dim;
  const int K = std::max({c.d_model, q, c.ffn});
  const int bytes = tile_lds_bytes(WB, MT, K);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const void* fns[] = {(const void*)k_qkv<WB, MT>, (const void*)k_oproj<WB, MT>, (const void*)k_gateup<WB, MT>,
                       (const void*)k_down<WB, MT>, (const void*)k_head<WB, MT>};
  const int kk[] = {c.d_model, q, c.d_model, std::max(c.ffn, 1), c.d_model};
  for (int i = 0; i < 5 && e == hipSuccess; ++i) {
    e = hipFuncSetAttribute(fns[i], hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    int per_cu = 0;
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fns[i], kGemvThreads, tile_lds_bytes(WB, MT, kk[i]));
    res.n[WB][row_class(MT)][i] = std::max(1, per_cu) * std::max(1, cus);
  }
  return e;
}

template <int WB>
hipError_t sk_set_lds(int bytes) {
  const void* fns[] = {(const void*)ks_qkv<WB>, (const void*)ks_oproj<WB>, (const void*)ks_gateup<WB>,
                       (const void*)ks_down<WB>, (const void*)ks_head<WB>};
  hipError_t e = hipSuccess;
  for (const void* f : fns)
    if (e == hipSuccess) e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  return e;
}

// k_fattn holds the scores and positions of the whole cache in LDS
hipError_t fattn_set_lds(int bytes) {
  const void* fns[] = {(const void*)k_fattn<0, 64>, (const void*)k_fattn<0, 96>, (const void*)k_fattn<0, 128>,
                       (const void*)k_fattn<1, 64>, (const void*)k_fattn<1, 96>, (const void*)k_fattn<1, 128>};
  hipError_t e = hipSuccess;
  for (const void* f : fns)
    if (e == hipSuccess) e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  return e;
}

bool getenv_zero(const char* name) {
  const char* v = getenv(name);
  return v && v[0] == '0';
}

template <int WB>
hipError_t rw_set_lds(int bytes) {
  hipError_t e = hipSuccess;
#define M2R2_RW_ATTR(N, S)                                                                                    \
  for (const void* f : {(const void*)kr_qkv<WB, N, S>, (const void*)kr_oproj<WB, N, S>,                        \
                        (const void*)kr_gateup<WB, N, S>, (const void*)kr_down<WB, N, S>,                       \
                        (const void*)kr_head<WB, N, S>})                                                      \
    if (e == hipSuccess) e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  M2R2_RW_ATTR(1, 1) M2R2_RW_ATTR(2, 1) M2R2_RW_ATTR(4, 1) M2R2_RW_ATTR(6, 1) M2R2_RW_ATTR(8, 1) M2R2_RW_ATTR(8, 2)
#undef M2R2_RW_ATTR
#define M2R2_RW_ATTR12(N, S)                                                                                  \
  for (const void* f : {(const void*)kr_oproj<WB, N, S, 12>, (const void*)kr_down<WB, N, S, 12>})              \
    if (e == hipSuccess) e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
  M2R2_RW_ATTR12(1, 1) M2R2_RW_ATTR12(2, 1) M2R2_RW_ATTR12(4, 1) M2R2_RW_ATTR12(6, 1) M2R2_RW_ATTR12(8, 1)
  M2R2_RW_ATTR12(8, 2)
#undef M2R2_RW_ATTR12
  return e;
}

// Decide whether the one- and two-row class runs the stream-K GEMVs: dense
// models whose every matrix has at least 8 blocks per tile, whose projection
// matrices q|k|v|adapter-down are consecutive, and whose partial slots fit.
// M2R2_STREAMK=0 in the environment selects the per-tile GEMVs instead.
hipError_t sk_setup(m2r2_ctx* c) {
  c->sk_on = false;
  const m2r2_config& cf = c->cfg;
  // a mixture-of-experts model uses the row-per-wave q/k/v and o projections,
  // the short-chain attention and the row-per-wave head (its MLP has kernels
  // of its own); the stream-K GEMVs, whose partial slots its layout does not
  // hold, stay off
  const bool moe = is_moe(cf);
  const char* env = getenv("M2R2_STREAMK");
  if (env && env[0] == '0') return hipSuccess;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess || cus < 1) return e;
  const int W = kSkWaves * cus;
  sk_plans(cf, W, c->sk);
  bool ok = true;
  if (!moe)
    for (const SkPlan& p : c->sk)
      ok = ok && p.nblk >= 8 && p.smax <= kSkMaxSeg && (p.L + p.nblk - 1) / p.nblk + 1 <= 64 &&
           (size_t)p.ntiles * p.smax <= c->lay.sk_slots;
  const Dims& D = c->D;
  const int K = moe ? std::max(D.d, D.qdim) : std::max({D.d, D.qdim, D.F});
  ok = ok && K <= kSkMaxK && sk_lds(K) <= 160 * 1024;
  const size_t tb = (size_t)16 * D.d * (D.wbf16 ? 2 : 4), tq = (size_t)(D.qdim / 16) * tb;
  for (const LayerPtrs& L : c->layers)
    ok = ok && (const char*)L.pk == (const char*)L.pq + tq && (const char*)L.pv == (const char*)L.pk + tq &&
         (const char*)L.pa == (const char*)L.pv + tq;
  ok = ok && cus <= c->lay.lm_slots;   // one arg-max slot per workgroup of the row-per-wave head
  if (!ok) return hipSuccess;
  e = D.wbf16 ? sk_set_lds<1>((int)sk_lds(K)) : sk_set_lds<0>((int)sk_lds(K));
  if (e == hipSuccess) {
    c->sk_on = !moe;
    c->sk_grid = cus;
    // attention of the stream-K path: fixed 128-token splits over the cache
    // capacity (at most 64, within the workspace's partial slots), the head's
    // B rows in at most three 16-byte pieces per thread, A_o in two
    const int S = (c->max_ctx + kSkAttnP - 1) / kSkAttnP;
    const int wsz = D.wbf16 ? 2 : 4;
    const bool ok_a = S <= 64 && S <= c->lay.S_max && D.hd * D.r * wsz <= 2 * kSkAttnThreads * 16 &&
                      (D.hd * D.r * wsz) % 16 == 0 && D.r * D.hd / 8 <= 2 * kSkAttnThreads;
    c->sk_attn_S = ok_a ? S : 0;
    // M2R2_ATTN_CHUNKS=1, 2 or 4 fixes the chunks per split of the batched
    // attention (tests exercise both forms at small sizes)
    if (const char* ac = getenv("M2R2_ATTN_CHUNKS"))
      c->attn_chunks = (ac[0] == '1' || ac[0] == '2' || ac[0] == '4') ? ac[0] - '0' : 0;
    // row-per-wave GEMVs: rows of whole 1 KB pieces, a piece count with a
    // kernel, adapter up-factor rows of whole 16-byte pieces, and the
    // short-chain attention
    const int epp = 64 * (D.wbf16 ? 8 : 4);   // elements per 1 KB piece
    const int Ks[3] = {D.d, D.qdim, D.F};
    bool ok_r = c->sk_attn_S > 0 && (D.r * wsz) % 16 == 0 && D.r * wsz <= kRwMaxBRowBytes &&
                !getenv_zero("M2R2_ROWWAVE");
    for (int i = 0; i < (moe ? 2 : 3); ++i) {
      c->rw_nch[i] = Ks[i] / epp;
      ok_r = ok_r && Ks[i] % epp == 0 && rw_nch_ok(c->rw_nch[i]) && Ks[i] <= kSkMaxK;
    }
    // the waves split their units with 32-bit products unit * wave count
    const long long nmax = std::max<long long>({3LL * D.qdim + 3LL * D.r, D.d, D.F, D.V});
    ok_r = ok_r && nmax * cus * 12 < (1LL << 32);
    // o and down projections (D.d output rows each): 12 waves per workgroup
    // when that puts the same number of rows on every wave and the rows are
    // long (at least 8 KB; for short rows the extra waves' staging costs
    // more than the uneven split: measured)
    auto eff = [&](int nw) {
      const double avg = (double)D.d / ((double)cus * nw);
      return avg / std::ceil(avg);
    };
    const bool even12 = eff(12) > eff(8) + 1e-9;
    c->rw_nw[0] = even12 && (size_t)D.qdim * wsz >= 8192 ? 12 : 8;
    c->rw_nw[1] = even12 && (size_t)D.F * wsz >= 8192 ? 12 : 8;
    if (ok_r) e = D.wbf16 ? rw_set_lds<1>(kSkMinLds) : rw_set_lds<0>(kSkMinLds);
    c->rw_on = ok_r && e == hipSuccess;
  }
  return e;
}

// ---- the one-launch decode step (persist.h) -----------------------------------
// Instantiations: (index, weight bf16, cache bf16, head_dim, 1 KB pieces per
// row of length d, H*hd, ffn).  Phi-3-mini shape; the tiny float32 and the
// small bfloat16 test decoders.
#define M2R2_PK_SHAPES(X) X(0, 1, 1, 96, 6, 6, 16) X(1, 0, 0, 64, 1, 1, 4) X(2, 1, 1, 128, 1, 1, 2)

template <int WB, int KB, int HD, int ND, int NQ, int NF>
hipError_t pk_attr(size_t lds, int* per_cu) {
  const void* f = (const void*)kp_step<WB, KB, HD, ND, NQ, NF>;
  hipError_t e = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(per_cu, f, kPkThreads, lds);
  return e;
}

// Use the one-launch step for this context when its shape has an
// instantiation: dense, rows of whole 1 KB pieces (the row-per-wave
// streams), rank a multiple of 4 with the o-projection slot (2 + 2r floats)
// within 64, every head at least one attention split, one workgroup per
// compute unit resident.
hipError_t pk_setup(m2r2_ctx* c) {
  c->pk.kind = -1;
  const Dims& D = c->D;
  // M2R2_ONE_LAUNCH=0 keeps one sequence on the multi-kernel path
  if (is_moe(c->cfg) || !c->rw_on || getenv_zero("M2R2_ONE_LAUNCH")) return hipSuccess;
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (D.r % 4 || 2 + 2 * D.r > 64 || cus < 1 || cus > kPkMaxWG || D.H > cus) return hipSuccess;
  const int S = std::min(kPkMaxSplits, std::max(1, cus / D.H));
  if (S > c->lay.S_max) return hipSuccess;
  const int nd = c->rw_nch[0], nq = c->rw_nch[1], nf = c->rw_nch[2];
  const size_t lds = pk_lds_bytes(D.hd, D.wbf16, std::max({D.d, D.qdim, D.F}));
  if (lds > 150 * 1024) return hipSuccess;
  int kind = -1, per_cu = 0;
#define M2R2_PK_MATCH(K, WB, KB, HD, ND, NQ, NF)                                                       \
  if (kind < 0 && D.wbf16 == WB && D.kvbf16 == KB && D.hd == HD && nd == ND && nq == NQ && nf == NF) { \
    kind = K;                                                                                         \
    e = pk_attr<WB, KB, HD, ND, NQ, NF>(lds, &per_cu);                                                \
  }
  M2R2_PK_SHAPES(M2R2_PK_MATCH)
#undef M2R2_PK_MATCH
  if (e != hipSuccess || kind < 0 || per_cu < 1) return e;
  char* b = c->ws_base;
  e = hipMemcpy(b + c->lay.layers_d, c->layers.data(), sizeof(LayerPtrs) * D.n_layers, hipMemcpyHostToDevice);
  if (e != hipSuccess) return e;
  c->pk.kind = kind;
  c->pk.grid = cus;
  c->pk.S = S;
  c->pk.lds = lds;
  c->pk.layers_d = (const LayerPtrs*)(b + c->lay.layers_d);
  c->pk.sd = (float*)(b + c->lay.pk_sd);
  c->pk.so = (float*)(b + c->lay.pk_so);
  c->pk.sgu = (float*)(b + c->lay.pk_sgu);
  c->pk.bar = (uint32_t*)(b + c->lay.pk_bar);
  c->pk.rel = (uint32_t*)(b + c->lay.pk_rel);
  return hipSuccess;
}

bool pk_eligible(const m2r2_ctx* c, const RowMap& rm, const StepIO& io) {
  return c->pk.kind >= 0 && !is_flops(c->cfg) && rm.nseq == 1 && rm.M >= 1 && rm.M <= 2 && !rm.head_all && !io.arla_sig &&
         rm.first[0] == 0 && rm.cnt[0] == rm.M;
}

m2r2_status run_pk(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int nl, hipStream_t st) {
  PkArgs a;
  a.D = c->D;
  a.layers = c->pk.layers_d;
  a.embed = c->embed;
  a.lm_head = c->lm_head_rm;
  a.final_norm = c->final_norm;
  a.rm = rm;
  a.ws = c->ws;
  a.io = io;
  a.kv = kv;
  a.sd = c->pk.sd;
  a.so = c->pk.so;
  a.sgu = c->pk.sgu;
  a.bar = PkBar{c->pk.bar, c->pk.rel};
  a.n_layers_run = nl;
  a.S = c->pk.S;
  a.so_w = c->lay.pk_so_w;
  a.sgu_w = c->lay.pk_sgu_w;
  const int grid = c->pk.grid;
  const size_t lds = c->pk.lds;
#define M2R2_PK_LAUNCH(K, WB, KB, HD, ND, NQ, NF) \
  case K: TIMED(11, (kp_step<WB, KB, HD, ND, NQ, NF><<<grid, kPkThreads, lds, st>>>(a))); break;
  switch (c->pk.kind) {
    M2R2_PK_SHAPES(M2R2_PK_LAUNCH)
    default: return fail(M2R2_E_STATE, "no one-launch step for this context");
  }
#undef M2R2_PK_LAUNCH
  HIP_TRY(hipGetLastError());
  return M2R2_OK;
}

// Embedding, n_layers_run layers, head (one launch where the shape allows).
m2r2_status run_pass(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int nl, hipStream_t st) {
  if (pk_eligible(c, rm, io)) return run_pk(c, rm, io, kv, nl, st);
  TIMED(6, (k_embed<<<rm.M + kEmbedZeroBlocks, 256, 0, st>>>(c->D, c->embed, rm, c->ws, io, 1)));
  HIP_TRY(hipGetLastError());
  const int wb = c->D.wbf16, kb = c->D.kvbf16;
  if (wb && kb) return run_hd<1, 1>(c, rm, io, kv, nl, st);
  if (wb && !kb) return run_hd<1, 0>(c, rm, io, kv, nl, st);
  if (!wb && kb) return run_hd<0, 1>(c, rm, io, kv, nl, st);
  return run_hd<0, 0>(c, rm, io, kv, nl, st);
}

// ---- mixture of experts --------------------------------------------------------

// Copy expert e of layer l from the host store into slot `slot` on copy
// stream cs, after the layer's last expert kernels (the slot's previous
// occupant may still be read) and after any earlier copy into the slot.
hipError_t moe_copy(m2r2_ctx* c, int l, int slot, int e, hipStream_t cs) {
  MoeState& M = c->moe;
  const int i = l * M.C + slot;
  hipError_t r = hipSuccess;
  if (M.layer_done_rec[l]) r = hipStreamWaitEvent(cs, M.layer_done[l], 0);
  if (r == hipSuccess && M.slot_pending[i]) r = hipStreamWaitEvent(cs, M.slot_ev[i], 0);
  if (r == hipSuccess)
    r = hipMemcpyAsync(M.slots_d + (size_t)i * M.stride, M.store_h + ((size_t)l * M.E + e) * M.ebytes, M.ebytes,
                       hipMemcpyHostToDevice, cs);
  if (r == hipSuccess) r = hipEventRecord(M.slot_ev[i], cs);
  if (r == hipSuccess) {
    M.slot_pending[i] = 1;
    M.h2d_bytes += (int64_t)M.ebytes;
  }
  return r;
}

// Wait until k_topk has published sequence number `seq` in the mapped block.
m2r2_status wait_routing(m2r2_ctx* c, int seq, hipStream_t st) {
  using clk = std::chrono::steady_clock;
  const auto t0 = clk::now();
  int* w = &c->moe.host_words[kHostSeq];
  uint64_t spins = 0;
  while (__atomic_load_n(w, __ATOMIC_ACQUIRE) != seq) {
    if ((++spins & 0xfff) == 0) {
      const hipError_t q = hipStreamQuery(st);
      if (q != hipSuccess && q != hipErrorNotReady) return fail(M2R2_E_HIP, "routing: %s", hipGetErrorString(q));
      if (q == hipSuccess && __atomic_load_n(w, __ATOMIC_ACQUIRE) != seq)
        return fail(M2R2_E_HIP, "routing result missing after the stream drained");
      if (clk::now() - t0 > std::chrono::seconds(60)) return fail(M2R2_E_HIP, "timed out waiting for routing");
    }
    _mm_pause();
  }
  c->moe.host_wait_ns += std::chrono::duration_cast<std::chrono::nanoseconds>(clk::now() - t0).count();
  return M2R2_OK;
}

// ---- the device slot table ----
void tab_put(MoeState& M, int l, int e, int slot) {
  if (!M.spec) return;
  const int i = l * M.E + e;
  if (M.tab[i] == slot) return;
  M.tab[i] = slot;
  M.tab_idx.push_back(i);
  M.tab_val.push_back(slot);
}

// The expert held in `slot` of layer l (if published) is about to be replaced.
void tab_evict_slot(MoeState& M, int l, int slot) {
  for (int e = 0; e < M.E; ++e)
    if (M.tab[l * M.E + e] == slot) tab_put(M, l, e, -1);
}

// Publish the copies that have completed (and still hold their expert).
void tab_publish_done(MoeState& M) {
  size_t keep = 0;
  for (size_t j = 0; j < M.pend.size(); ++j) {
    const MoeState::Pending p = M.pend[j];
    const int i = p.l * M.C + p.slot;
    if (M.pol.layer(p.l).expert_in[p.slot] != p.e) continue;   // replaced since: drop
    if (M.slot_pending[i]) {
      if (hipEventQuery(M.slot_ev[i]) != hipSuccess) {
        M.pend[keep++] = p;
        continue;
      }
      M.slot_pending[i] = 0;
    }
    tab_put(M, p.l, p.e, p.slot);
  }
  M.pend.resize(keep);
}

hipError_t tab_flush(m2r2_ctx* c, hipStream_t st) {
  MoeState& M = c->moe;
  for (size_t j0 = 0; j0 < M.tab_idx.size(); j0 += 30) {
    TabUpdates u{};
    u.n = (int)std::min<size_t>(30, M.tab_idx.size() - j0);
    for (int j = 0; j < u.n; ++j) {
      u.idx[j] = M.tab_idx[j0 + j];
      u.val[j] = M.tab_val[j0 + j];
    }
    k_tab_set<<<1, 64, 0, st>>>(M.tab_d, u);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  M.tab_idx.clear();
  M.tab_val.clear();
  return hipSuccess;
}

// Dual-stream (or slow-only) pass of a mixture-of-experts model, batch 1:
// rows 0 (slow) and 1 (fast).
// The expert copies of the scheduler: from the pinned host store on the
// demand or the ahead-of-time stream, one event per slot.  A copy that cannot
// be enqueued leaves nothing behind (the error is cleared); a slot whose
// event reports an error holds no valid expert.
class HipExpertEngine final : public ExpertCopyEngine {
 public:
  explicit HipExpertEngine(m2r2_ctx* c) : c_(c) {}
  bool start(int l, int s, int e, bool demand) override {
    MoeState& M = c_->moe;
    tab_evict_slot(M, l, s);
    if (moe_copy(c_, l, s, e, demand ? M.copy_demand : M.copy_ahead) != hipSuccess) {
      (void)hipGetLastError();
      return false;
    }
    if (!demand && M.spec) M.pend.push_back({l, s, e});
    return true;
  }
  State state(int l, int s) override {
    MoeState& M = c_->moe;
    const int i = l * M.C + s;
    if (!M.slot_pending[i]) return kDone;
    const hipError_t q = hipEventQuery(M.slot_ev[i]);
    if (q == hipSuccess) {
      M.slot_pending[i] = 0;
      return kDone;
    }
    if (q == hipErrorNotReady) return kPending;
    (void)hipGetLastError();
    return kFailed;   // (stays failed until a new copy into the slot is started)
  }

 private:
  m2r2_ctx* c_;
};

template <int WB, int KB, int HD>
m2r2_status run_moe_t(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, const m2r2_step_out* out,
                      bool dual, hipStream_t st) {
  constexpr int MT = 2;
  const Dims& D = c->D;
  MoeState& M = c->moe;
  const int S = choose_splits(1, rm.M, D.H, c->max_ctx);
  if (S > c->lay.S_max || S + 1 > 64) return fail(M2R2_E_SHAPE, "attention splits exceed the workspace");
  const size_t smem = attn_smem_bytes();
  const size_t gl = gemv_lds_bytes(WB, MT);
  const bool ahead = dual && M.policy == M2R2_MOE_AHEAD_OF_TIME;
  const bool prev = M.policy == M2R2_MOE_PREVIOUS_LAYER;
  const bool fixed = M.policy == M2R2_MOE_FIXED;
  const int* random_row = nullptr;   // this token's random-preload draws
  if (M.policy == M2R2_MOE_RANDOM_PRELOAD) {
    if (M.preload_tokens < 1) return fail(M2R2_E_STATE, "random preload without a table");
    random_row = M.preload.data() + (size_t)(M.token % M.preload_tokens) * D.n_layers * M.K;
  }
  // fast-row predictions: for the ahead-of-time copies, or reported on request
  const bool want_pred = dual && !prev && (ahead || (out && out->pred_experts_d));
  const Grids G = grids<WB, MT>(c);
  const int tiles = (M.E + 15) / 16;
  float* logits = (float*)M.mp.logits;
  // every expert of every layer resident and published: nothing the host
  // would decide depends on the routing (the LRU policy only counts hits)
  tab_publish_done(M);
  const bool resident = M.spec && M.C == M.E && M.policy == M2R2_MOE_ON_DEMAND && M.pend.empty() &&
                        std::all_of(M.tab.begin(), M.tab.end(), [](int v) { return v >= 0; });
  if (resident) {
    HIP_TRY(tab_flush(c, st));
    M.hits_dev_used = true;
  }
  for (int l = 0; l < D.n_layers; ++l) {
    const LayerPtrs& L = c->layers[l];
    if (c->rw_on) {
      TIMED(0, (kr_qkv_launch<WB>(c->rw_nch[0], c->sk_grid, (size_t)kSkMinLds, st, D, L, rm, c->ws, io, l)));
      TIMED(1, (ks_attn<WB, KB, HD><<<dim3(c->sk_attn_S, D.H, rm.nseq), kSkAttnThreads,
                                       sk_attn_lds_bytes(HD, D.r, WB), st>>>(D, L, rm, c->ws, io, kv, l, c->sk_attn_S)));
      TIMED(2, (kr_oproj_launch<WB>(c->rw_nch[1], c->rw_nw[0], c->sk_grid, (size_t)kSkMinLds, st, D, L, rm, c->ws,
                                    io, l)));
    } else {
      TIMED(0, (k_qkv<WB, MT><<<G.qkv, kGemvThreads, G.l_d, st>>>(D, L, rm, c->ws, io, l)));
      TIMED(1, (k_attn<KB, HD><<<dim3(S + 1, D.H, 1), kAttnThreads, smem, st>>>(D, L, rm, c->ws, io, kv, l, S)));
      TIMED(2, (k_oproj<WB, MT><<<G.o, kGemvThreads, G.l_q, st>>>(D, L, rm, c->ws, io, l)));
    }
    // routing of the slow row, predictions for layers 2l+2 and 2l+3 from the fast row
    RouterTask t[3] = {};
    t[0] = RouterTask{M.router[l], L.mlp_norm, 0, 0, l, logits};
    int n_pred = 0;
    if (want_pred)
      for (int lp = 2 * l + 2; lp <= 2 * l + 3 && lp < D.n_layers; ++lp, ++n_pred)
        t[1 + n_pred] = RouterTask{M.router[lp], c->layers[lp].mlp_norm, 1, 1, l + 1, logits + (1 + n_pred) * M.E};
    // previous-layer speculation (Sec. 3.3): layer l+1's router on the same
    // slow-row vector that layer l routes
    if (prev && l + 1 < D.n_layers)
      t[1 + n_pred++] = RouterTask{M.router[l + 1], c->layers[l + 1].mlp_norm, 0, 0, l, logits + M.E};
    // the fast row's MLP runs inside the routing launch unless a prediction
    // task reads the fast row it produces
    const int fmlp_blocks = dual && n_pred == 0 ? (D.d + kGemvThreads - 1) / kGemvThreads : 0;
    if (dual && !fmlp_blocks) TIMED(10, (k_fast_mlp<<<(D.d + 255) / 256, 256, 0, st>>>(D, rm, L, l, c->ws)));
    int* slow_out = out->slow_experts_d ? out->slow_experts_d + l * M.K : nullptr;
    int* pred_out = (out->pred_experts_d && n_pred) ? out->pred_experts_d + (prev ? l + 1 : 2 * l + 2) * M.K
                                                    : nullptr;
    const int seq = resident ? 0 : ++M.seq;
    MoePtrs mpk = M.mp;
    if (resident) mpk.sel_host = nullptr;   // no host reads this layer's routing
    // router tiles, then the top-k in the last of them to finish
    TIMED(10, (k_route<WB><<<tiles * (1 + n_pred) + fmlp_blocks, kGemvThreads, gl, st>>>(
                  D, M.E, t[0], t[1], t[2], 1 + n_pred, c->ws, M.K, mpk, slow_out, pred_out, seq, M.route_cnt_d, rm, L,
                  l)));
    HIP_TRY(hipGetLastError());
    const SlotTable stab{M.tab_d, M.slots_d, M.stride, M.E, M.C};
    if (resident) {
      // the experts from the table; an exited row's statistics from the down kernel
      TIMED(8, (k_moe_gateup<WB, true><<<M.K * (M.Fe / 16), kGemvThreads, gl, st>>>(D, M.Fe, M.K, ExpertSlots{}, 0,
                                                                                   L.mlp_norm, l, M.mp, c->ws, stab,
                                                                                   M.hits_d)));
      TIMED(9, (k_moe_down<WB, true><<<c->lay.TD, kGemvThreads, gl, st>>>(D, M.Fe, M.K, ExpertSlots{}, 0, l, M.mp,
                                                                         c->ws, stab, 1)));
      HIP_TRY(hipGetLastError());
      HIP_TRY(hipEventRecord(M.layer_done[l], st));
      M.layer_done_rec[l] = 1;
      continue;
    }
    if (M.spec) {
      // the experts from the slots the table publishes, without waiting for
      // the host (they return at once if a chosen expert is not published)
      tab_publish_done(M);
      HIP_TRY(tab_flush(c, st));
      TIMED(8, (k_moe_gateup<WB, true><<<M.K * (M.Fe / 16), kGemvThreads, gl, st>>>(D, M.Fe, M.K, ExpertSlots{}, 0,
                                                                                   L.mlp_norm, l, M.mp, c->ws, stab)));
      TIMED(9, (k_moe_down<WB, true><<<c->lay.TD, kGemvThreads, gl, st>>>(D, M.Fe, M.K, ExpertSlots{}, 0, l, M.mp,
                                                                         c->ws, stab)));
      HIP_TRY(hipGetLastError());
      HIP_TRY(hipEventRecord(M.layer_done[l], st));
      M.layer_done_rec[l] = 1;
    }
    if (m2r2_status s = wait_routing(c, seq, st)) return s;
    if (M.host_words[kHostExited]) {   // exited: no MLP for the remaining layers
      TIMED(10, (k_row_stats<<<1, 256, 0, st>>>(D, 0, l + 1, c->ws)));
      HIP_TRY(hipGetLastError());
      continue;
    }
    int need[kMaxTopK], slot[kMaxTopK];
    bool load[kMaxTopK];
    for (int k = 0; k < M.K; ++k) {
      need[k] = M.host_words[k];
      if (need[k] < 0 || need[k] >= M.E) return fail(M2R2_E_HIP, "layer %d: router returned expert %d", l, need[k]);
    }
    HipExpertEngine eng(c);
    ExpertScheduler sched(M.pol, eng);
    if (fixed)
      M.pol.use_fixed(l, need, M.K, slot, load);
    else if (!sched.acquire(l, need, M.K, slot, load))
      return fail(M2R2_E_HIP, "layer %d: an on-demand expert copy could not be enqueued", l);
    // did the launches above find every chosen expert in its slot?
    bool done = M.spec;
    for (int k = 0; k < M.K && done; ++k) done = M.tab[l * M.E + need[k]] == slot[k];
    if (!done) {
    if (fixed)   // (the scheduler started the other policies' on-demand copies)
      for (int k = 0; k < M.K; ++k)
        if (load[k]) {
          tab_evict_slot(M, l, slot[k]);
          HIP_TRY(moe_copy(c, l, slot[k], need[k], M.copy_demand));
        }
    ExpertSlots es{};
    for (int k = 0; k < M.K; ++k) {
      const int i = l * M.C + slot[k];
      if (M.slot_pending[i]) {
        const hipError_t q = hipEventQuery(M.slot_ev[i]);
        if (q == hipSuccess) {
          M.slot_pending[i] = 0;
        } else if (q == hipErrorNotReady) {
          HIP_TRY(hipStreamWaitEvent(st, M.slot_ev[i], 0));
          ++M.copy_waits;
        } else {
          return fail(M2R2_E_HIP, "expert copy: %s", hipGetErrorString(q));
        }
      }
      es.w[k] = M.slots_d + (size_t)i * M.stride;
    }
    TIMED(8, (k_moe_gateup<WB><<<M.K * (M.Fe / 16), kGemvThreads, gl, st>>>(D, M.Fe, M.K, es, 0, L.mlp_norm, l, M.mp,
                                                                           c->ws, stab)));
    TIMED(9, (k_moe_down<WB><<<c->lay.TD, kGemvThreads, gl, st>>>(D, M.Fe, M.K, es, 0, l, M.mp, c->ws, stab)));
    HIP_TRY(hipGetLastError());
    HIP_TRY(hipEventRecord(M.layer_done[l], st));
    M.layer_done_rec[l] = 1;
    // the copies above are complete for every later launch on `st`
    if (!fixed)
      for (int k = 0; k < M.K; ++k)
        if (load[k]) tab_put(M, l, need[k], slot[k]);
    }
    // prefetches: a copy that cannot be enqueued invalidates its slot (the
    // expert is then loaded on demand when it is used)
    auto preload = [&](int lp, const int* ids) -> hipError_t {
      sched.prefetch(lp, ids, M.K);
      return hipSuccess;
    };
    if (ahead)
      for (int j = 0; j < n_pred; ++j) HIP_TRY(preload(2 * l + 2 + j, M.host_words + (1 + j) * kMaxTopK));
    if (prev && n_pred) HIP_TRY(preload(l + 1, M.host_words + kMaxTopK));
    if (random_row && l + 1 < D.n_layers) HIP_TRY(preload(l + 1, random_row + (l + 1) * M.K));
  }
  if (c->rw_on)
    TIMED(5, (kr_head_launch<WB>(c->rw_nch[0], c->sk_grid, (size_t)kSkMinLds, st, D, c->lm_head_rm, c->final_norm, rm,
                                  c->ws, io, kv, c->skws, D.n_layers, (const void*)nullptr)));
  else
    TIMED(5, (k_head<WB, MT><<<G.head, kGemvThreads, G.l_d, st>>>(D, c->lm_head, c->final_norm, rm, c->ws, io, kv,
                                                                c->lay.TV, D.n_layers)));
  HIP_TRY(hipGetLastError());
  M.pol.end_token();
  ++M.token;
  return M2R2_OK;
}

template <int WB, int KB>
m2r2_status run_moe_hd(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, const m2r2_step_out* out,
                       bool dual, hipStream_t st) {
  switch (c->D.hd) {
    case 64: return run_moe_t<WB, KB, 64>(c, rm, io, kv, out, dual, st);
    case 96: return run_moe_t<WB, KB, 96>(c, rm, io, kv, out, dual, st);
    case 128: return run_moe_t<WB, KB, 128>(c, rm, io, kv, out, dual, st);
  }
  return fail(M2R2_E_UNSUPPORTED, "head_dim");
}

m2r2_status run_moe_pass(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, const m2r2_step_out* out,
                         bool dual, hipStream_t st) {
  const int N = c->D.n_layers, K = c->moe.K;
  if (out->slow_experts_d) HIP_TRY(hipMemsetAsync(out->slow_experts_d, 0xff, sizeof(int32_t) * N * K, st));
  if (out->pred_experts_d) HIP_TRY(hipMemsetAsync(out->pred_experts_d, 0xff, sizeof(int32_t) * N * K, st));
  TIMED(6, (k_embed<<<rm.M + kEmbedZeroBlocks, 256, 0, st>>>(c->D, c->embed, rm, c->ws, io, 1)));
  HIP_TRY(hipGetLastError());
  const int wb = c->D.wbf16, kb = c->D.kvbf16;
  if (wb && kb) return run_moe_hd<1, 1>(c, rm, io, kv, out, dual, st);
  if (wb && !kb) return run_moe_hd<1, 0>(c, rm, io, kv, out, dual, st);
  if (!wb && kb) return run_moe_hd<0, 1>(c, rm, io, kv, out, dual, st);
  return run_moe_hd<0, 0>(c, rm, io, kv, out, dual, st);
}

template <int WB>
hipError_t set_moe_lds_limits() {
  const int bytes = gemv_lds_bytes(WB, 2);
  hipError_t e = hipSuccess;
  const void* fns[] = {(const void*)k_router<WB>, (const void*)k_route<WB>, (const void*)k_moe_gateup<WB>,
                       (const void*)k_moe_down<WB>,
                       (const void*)k_moe_gateup<WB, true>, (const void*)k_moe_down<WB, true>};
  for (const void* f : fns) {
    hipError_t r = hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
    if (r != hipSuccess) e = r;
  }
  return e;
}

// Warm start of the expert cache: experts 0..C-1 in slots 0..C-1 of every
// layer (synchronous).
hipError_t moe_warm(m2r2_ctx* c) {
  MoeState& M = c->moe;
  hipError_t e = hipDeviceSynchronize();
  M.pol.warm();
  for (int l = 0; l < c->D.n_layers && e == hipSuccess; ++l)
    for (int s = 0; s < M.C && e == hipSuccess; ++s)
      e = hipMemcpyAsync(M.slots_d + ((size_t)l * M.C + s) * M.stride, M.store_h + ((size_t)l * M.E + s) * M.ebytes,
                         M.ebytes, hipMemcpyHostToDevice, M.copy_demand);
  if (e == hipSuccess) e = hipStreamSynchronize(M.copy_demand);
  std::fill(M.slot_pending.begin(), M.slot_pending.end(), 0);
  std::fill(M.layer_done_rec.begin(), M.layer_done_rec.end(), 0);
  M.h2d_bytes = M.copy_waits = M.host_wait_ns = 0;
  M.token = 0;
  // the slot table: the warm experts, except that the fixed-experts policy
  // publishes only the ones it keeps (the last top_k slots are its staging)
  const int n_pub = M.policy == M2R2_MOE_FIXED ? M.C - M.K : M.C;
  M.tab.assign((size_t)c->D.n_layers * M.E, -1);
  for (int l = 0; l < c->D.n_layers; ++l)
    for (int s = 0; s < n_pub; ++s) M.tab[(size_t)l * M.E + s] = s;
  M.tab_idx.clear();
  M.tab_val.clear();
  M.pend.clear();
  if (e == hipSuccess) e = hipMemcpy(M.tab_d, M.tab.data(), sizeof(int) * M.tab.size(), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = hipMemset(M.hits_d, 0, 256);   // (and the router arrival counter)
  if (e == hipSuccess) e = hipDeviceSynchronize();
  M.hits_dev_used = false;
  return e;
}

void fill_stats(const CacheCounters& k, m2r2_moe_counters* o) {
  memset(o, 0, sizeof *o);
  o->hits = k.hits; o->misses = k.misses; o->prefetch_issued = k.prefetch_issued; o->prefetch_used = k.prefetch_used;
  o->prefetch_wasted = k.prefetch_wasted; o->loads = k.loads; o->pred_correct = k.pred_correct;
  o->pred_total = k.pred_total; o->copies_failed = k.copies_failed;
  for (size_t l = 0; l < k.layer_misses.size() && l < 128; ++l) o->layer_misses[l] = k.layer_misses[l];
}

void moe_release(MoeState& M) {
  if (M.copy_demand) (void)hipStreamSynchronize(M.copy_demand);
  if (M.copy_ahead) (void)hipStreamSynchronize(M.copy_ahead);
  for (hipEvent_t e : M.slot_ev) (void)hipEventDestroy(e);
  for (hipEvent_t e : M.layer_done) (void)hipEventDestroy(e);
  M.slot_ev.clear();
  M.layer_done.clear();
  if (M.copy_demand) (void)hipStreamDestroy(M.copy_demand);
  if (M.copy_ahead) (void)hipStreamDestroy(M.copy_ahead);
  if (M.host_words) (void)hipHostFree(M.host_words);
  M.copy_demand = M.copy_ahead = nullptr;
  M.host_words = nullptr;
}

RowMap empty_rowmap() {
  RowMap rm;
  memset(&rm, 0, sizeof rm);
  for (int i = 0; i < kMaxRows; ++i) rm.slow_of[i] = -1;
  return rm;
}

StepIO empty_io() {
  StepIO io;
  memset(&io, 0, sizeof io);
  return io;
}

}  // namespace

extern "C" {

M2R2_API const char* m2r2_last_error(void) { return g_err.c_str(); }

M2R2_API m2r2_status m2r2_workspace_size(const m2r2_config* cfg, int32_t max_batch, int32_t max_chunk,
                                         int32_t max_ctx, size_t* bytes_out) {
  m2r2_status st = check_config(cfg, max_batch, max_chunk, max_ctx);
  if (st) return st;
  if (!bytes_out) return fail(M2R2_E_INVALID, "bytes_out is NULL");
  *bytes_out = make_layout(*cfg, max_batch, max_chunk, max_ctx).total;
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_create(const m2r2_config* cfg, const m2r2_weights* w, int32_t max_batch,
                                 int32_t max_chunk, int32_t max_ctx, void* workspace, size_t ws_bytes,
                                 m2r2_ctx** out) {
  m2r2_status st = check_config(cfg, max_batch, max_chunk, max_ctx);
  if (st) return st;
  if (!w || !w->embed || !w->final_norm || !w->lm_head || !w->layers || !out)
    return fail(M2R2_E_INVALID, "weights (embed, final_norm, lm_head, layers) or out is NULL");
  if (!workspace || ((uintptr_t)workspace & 255)) return fail(M2R2_E_INVALID, "workspace NULL or not 256-byte aligned");
  const Layout lay = make_layout(*cfg, max_batch, max_chunk, max_ctx);
  if (ws_bytes < lay.total) return fail(M2R2_E_NOMEM, "workspace %zu bytes < %zu needed", ws_bytes, lay.total);
  const bool moe = is_moe(*cfg);
  if (moe && !w->experts_h) return fail(M2R2_E_INVALID, "mixture of experts: experts_h is NULL");
  if (cfg->head_rank > 0 && (!w->head_a || !w->head_b))
    return fail(M2R2_E_INVALID, "head_rank %d: head_a/head_b is NULL", cfg->head_rank);
  for (int l = 0; l < cfg->n_layers; ++l) {
    const m2r2_layer_weights& L = w->layers[l];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.mlp_norm)
      return fail(M2R2_E_INVALID, "layer %d: a base weight pointer is NULL", l);
    if (!moe && (!L.wg || !L.wu || !L.wd)) return fail(M2R2_E_INVALID, "layer %d: an MLP weight pointer is NULL", l);
    if (moe && !L.router) return fail(M2R2_E_INVALID, "layer %d: router is NULL", l);
    const void* ps[] = {L.wq, L.wk, L.wv, L.wo, L.wg, L.wu, L.wd, L.router, w->embed, w->lm_head};
    for (const void* p : ps)
      if (!aligned16(p)) return fail(M2R2_E_INVALID, "layer %d: weight not 16-byte aligned", l);
    for (int a = 0; a < 7; ++a) {
      if ((L.A[a] == nullptr) != (L.B[a] == nullptr))
        return fail(M2R2_E_INVALID, "layer %d adapter %d: A and B must be both set or both NULL", l, a);
      if (!aligned16(L.A[a])) return fail(M2R2_E_INVALID, "layer %d adapter %d: A not 16-byte aligned", l, a);
      if (moe && a >= 4 && L.A[a])
        return fail(M2R2_E_INVALID, "layer %d: a mixture-of-experts layer takes A_m/B_m, not adapter %d", l, a);
    }
    if ((L.A_m == nullptr) != (L.B_m == nullptr))
      return fail(M2R2_E_INVALID, "layer %d: A_m and B_m must be both set or both NULL", l);
  }
  m2r2_ctx* c = new (std::nothrow) m2r2_ctx();
  if (!c) return fail(M2R2_E_NOMEM, "host allocation");
  c->cfg = *cfg;
  c->lay = lay;
  c->max_batch = max_batch;
  c->max_chunk = max_chunk;
  c->max_ctx = max_ctx;
  c->embed = w->embed;
  c->final_norm = w->final_norm;
  c->lm_head = (char*)workspace + lay.lm;
  c->lm_head_rm = w->lm_head;
  Dims& D = c->D;
  D.n_layers = cfg->n_layers; D.d = cfg->d_model; D.H = cfg->n_heads; D.hd = cfg->head_dim;
  D.qdim = cfg->n_heads * cfg->head_dim; D.F = cfg->ffn; D.V = cfg->vocab; D.r = cfg->rank;
  D.eps = cfg->rms_eps; D.theta = cfg->rope_theta; D.wbf16 = cfg->wdtype == M2R2_BF16; D.kvbf16 = cfg->kvdtype == M2R2_BF16;
  D.fh = cfg->fast_heads; D.ftk = cfg->fast_topk; D.fmlp = cfg->fast_mlp_adapter; D.hr = cfg->head_rank;
  if (cfg->head_rank > 0) {
    c->head_a = w->head_a;
    c->head_b = w->head_b;
  }
  c->layers.resize(cfg->n_layers);
  for (int l = 0; l < cfg->n_layers; ++l) {
    const m2r2_layer_weights& s = w->layers[l];
    LayerPtrs& L = c->layers[l];
    L.attn_norm = s.attn_norm;
    L.mlp_norm = s.mlp_norm;
    char* wsb = (char*)workspace;
    const size_t* o = &lay.lay_off[8 * l];
    L.pq = wsb + o[0]; L.pk = wsb + o[1]; L.pv = wsb + o[2]; L.pa = wsb + o[3];
    L.po = wsb + o[4];
    L.wq = s.wq; L.wk = s.wk; L.wv = s.wv; L.wo = s.wo; L.wg = s.wg; L.wu = s.wu; L.wd = s.wd;
    for (int a = 0; a < 7; ++a) { L.A[a] = s.A[a]; L.B[a] = s.B[a]; }
    if (moe) {
      // the fast MLP adapter rides in the gate slot: the o projection sums its
      // adapter-down partials, the fast MLP kernel applies its up factor
      L.pg = L.pu = L.pd = nullptr;
      L.A[4] = s.A_m; L.B[4] = s.B_m;
      c->moe.router.push_back(wsb + o[5]);
    } else {
      L.pg = wsb + o[5]; L.pu = nullptr; L.pd = wsb + o[7];
      if (cfg->fast_mlp_adapter) {
        // FLOPs-optimised form: the fast MLP is the adapter alone; the gate,
        // up and down slots stay empty (the gate/up kernels read a gate
        // adapter's up factor as [ffn][rank]); the o projection and the fast
        // MLP kernel get a copy of the layer with A_m/B_m in the gate slot
        L.A[4] = L.B[4] = L.A[5] = L.B[5] = L.A[6] = L.B[6] = nullptr;
        c->fmlp_a.push_back(s.A_m);
        c->fmlp_b.push_back(s.B_m);
      }
    }
  }
  char* b = (char*)workspace;
  c->ws_base = b;
  WS& ws = c->ws;
  ws.X = (float*)(b + lay.X); ws.PIN = (float*)(b + lay.PIN); ws.QKV = (float*)(b + lay.QKV);
  ws.O = (float*)(b + lay.O); ws.ACT = (float*)(b + lay.ACT); ws.bin_d = (float*)(b + lay.bin_d);
  ws.bin_o = (float*)(b + lay.bin_o); ws.bin_gu = (float*)(b + lay.bin_gu); ws.uo = (float*)(b + lay.uo);
  ws.att = (float*)(b + lay.att); ws.att_cnt = (uint32_t*)(b + lay.att_cnt); ws.lm_val = (float*)(b + lay.lm_val);
  ws.lm_idx = (int*)(b + lay.lm_idx); ws.lm_cnt = (uint32_t*)(b + lay.lm_cnt); ws.exited = (int*)(b + lay.exited);
  ws.exitb = (int*)(b + lay.exitb); ws.reinit = (int*)(b + lay.reinit); ws.err = (int*)(b + lay.err);
  ws.sig = (float*)(b + lay.sig);
  ws.arla_kv = (float*)(b + lay.arla_kv); ws.arla_q = (float*)(b + lay.arla_q);
  ws.arla_sig = (float*)(b + lay.arla_sig); ws.arla_cnt = (uint32_t*)(b + lay.arla_cnt);
  ws.rope = (const float2*)(b + lay.rope);
  ws.rope_len = max_ctx;
  ws.fsc = (float*)(b + lay.fsc); ws.fqkv = (float*)(b + lay.fqkv); ws.lrz = (float*)(b + lay.lrz);
  c->skws.part = (float*)(b + lay.sk_part);
  c->skws.hier = (uint32_t*)(b + lay.sk_cnt);
  c->skws.cnt = c->skws.hier + 65;

  hipError_t e = hipGetDevice(&c->device);
  // the no-allocation decode step's scratch: its address on this device
  if (e == hipSuccess) e = scratch_setup(c->device);
  if (e == hipSuccess) e = hipMemset(workspace, 0, lay.total);
  if (e == hipSuccess) {
    // RoPE table: angle pos * theta^(-2j/hd) evaluated in double precision
    const int half = cfg->head_dim / 2;
    std::vector<float> t((size_t)max_ctx * half * 2);
    for (int pos = 0; pos < max_ctx; ++pos)
      for (int j = 0; j < half; ++j) {
        const double ang = (double)pos * std::pow((double)cfg->rope_theta, -2.0 * j / cfg->head_dim);
        t[((size_t)pos * half + j) * 2] = (float)std::cos(ang);
        t[((size_t)pos * half + j) * 2 + 1] = (float)std::sin(ang);
      }
    e = hipMemcpy(b + lay.rope, t.data(), t.size() * sizeof(float), hipMemcpyHostToDevice);
  }
  if (e == hipSuccess) e = pack_all(c, w, workspace);
  if (e == hipSuccess) e = set_lds_limits<0, 2>(*cfg, c->resident);
  if (e == hipSuccess) e = set_lds_limits<1, 2>(*cfg, c->resident);
  if (e == hipSuccess) e = set_lds_limits<0, 8>(*cfg, c->resident);
  if (e == hipSuccess) e = set_lds_limits<1, 8>(*cfg, c->resident);
  if (e == hipSuccess) e = set_lds_limits<0, 16>(*cfg, c->resident);
  if (e == hipSuccess) e = set_lds_limits<1, 16>(*cfg, c->resident);
  if (e == hipSuccess) e = sk_setup(c);
  if (e == hipSuccess) e = pk_setup(c);
  if (e == hipSuccess && is_flops(*cfg)) e = fattn_set_lds((int)fattn_lds_bytes(max_ctx));
  if (e == hipSuccess && moe) {
    MoeState& M = c->moe;
    M.on = true;
    M.E = cfg->n_experts; M.K = cfg->top_k; M.Fe = cfg->expert_ffn; M.C = cfg->expert_slots;
    M.ebytes = lay.expert_bytes;
    M.stride = lay.expert_stride;
    M.store_h = (const char*)w->experts_h;
    M.slots_d = b + lay.moe_slots;
    M.tab_d = (int*)(b + lay.moe_tab);
    M.hits_d = (unsigned long long*)(b + lay.moe_hits);
    M.route_cnt_d = (uint32_t*)(b + lay.moe_hits + 128);
    M.mp.logits = (const float*)(b + lay.moe_logits);
    M.mp.sel = (int*)(b + lay.moe_sel);
    M.mp.prob = (float*)(b + lay.moe_prob);
    M.mp.act = (float*)(b + lay.moe_act);
    e = hipHostMalloc((void**)&M.host_words, sizeof(int) * kHostWords, hipHostMallocMapped | hipHostMallocCoherent);
    if (e == hipSuccess) {
      memset(M.host_words, 0, sizeof(int) * kHostWords);
      e = hipHostGetDevicePointer((void**)&M.mp.sel_host, M.host_words, 0);
    }
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&M.copy_demand, hipStreamNonBlocking);
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&M.copy_ahead, hipStreamNonBlocking);
    const int n_ev = cfg->n_layers * M.C;
    for (int i = 0; i < n_ev && e == hipSuccess; ++i) {
      hipEvent_t ev;
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e == hipSuccess) M.slot_ev.push_back(ev);
    }
    for (int l = 0; l < cfg->n_layers && e == hipSuccess; ++l) {
      hipEvent_t ev;
      e = hipEventCreateWithFlags(&ev, hipEventDisableTiming);
      if (e == hipSuccess) M.layer_done.push_back(ev);
    }
    M.slot_pending.assign(n_ev, 0);
    M.layer_done_rec.assign(cfg->n_layers, 0);
    M.pol.init(cfg->n_layers, M.E, M.C);
    M.spec = !getenv_zero("M2R2_MOE_DEVICE_SLOTS");
    if (e == hipSuccess) e = set_moe_lds_limits<0>();
    if (e == hipSuccess) e = set_moe_lds_limits<1>();
    if (e == hipSuccess) e = moe_warm(c);
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    moe_release(c->moe);
    delete c;
    return fail(M2R2_E_HIP, "workspace init: %s", hipGetErrorString(e));
  }
  *out = c;
  return M2R2_OK;
}

M2R2_API void m2r2_destroy(m2r2_ctx* ctx) {
  if (!ctx) return;
  for (hipEvent_t e : ctx->ev) (void)hipEventDestroy(e);
  moe_release(ctx->moe);
  delete ctx;
}

M2R2_API m2r2_status m2r2_timing_enable(m2r2_ctx* c, int32_t kernel_class) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (kernel_class < -1 || kernel_class > 11) return fail(M2R2_E_INVALID, "kernel class %d", kernel_class);
  c->timed_class = kernel_class;
  c->ev_used = 0;   // a new record
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_timing_read(m2r2_ctx* c, double* ms_sum, int32_t* launches) {
  if (!c || !ms_sum || !launches) return fail(M2R2_E_INVALID, "NULL argument");
  double sum = 0.0;
  for (int i = 0; i < c->ev_used; ++i) {
    HIP_TRY(hipEventSynchronize(c->ev[2 * i + 1]));
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, c->ev[2 * i], c->ev[2 * i + 1]));
    sum += ms;
  }
  *ms_sum = sum;
  *launches = c->ev_used;
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_time_gateup_layers(m2r2_ctx* c, int32_t dual, hipStream_t st, double* avg_ms) {
  if (!c || !avg_ms) return fail(M2R2_E_INVALID, "NULL argument");
  if (!c->rw_on || c->moe.on) return fail(M2R2_E_UNSUPPORTED, "the decode class does not use the row-per-wave kernels");
  const Dims& D = c->D;
  RowMap rm = empty_rowmap();
  rm.nseq = 1;
  rm.M = dual ? 2 : 1;
  rm.first[0] = 0;
  rm.cnt[0] = rm.M;
  rm.seq[0] = 0; rm.fast[0] = 0; rm.wr[0] = 1;
  if (dual) { rm.seq[1] = 0; rm.fast[1] = 1; rm.wr[1] = 0; rm.slow_of[1] = 0; }
  const StepIO io = empty_io();
  hipEvent_t a, b;
  HIP_TRY(hipEventCreate(&a));
  HIP_TRY(hipEventCreate(&b));
  hipError_t e = hipEventRecord(a, st);
  for (int l = 0; l < D.n_layers && e == hipSuccess; ++l) {
    if (D.wbf16) kr_gateup_launch<1>(c->rw_nch[0], c->sk_grid, (size_t)kSkMinLds, st, D, c->layers[l], rm, c->ws, io, l);
    else kr_gateup_launch<0>(c->rw_nch[0], c->sk_grid, (size_t)kSkMinLds, st, D, c->layers[l], rm, c->ws, io, l);
    e = hipGetLastError();
  }
  if (e == hipSuccess) e = hipEventRecord(b, st);
  if (e == hipSuccess) e = hipEventSynchronize(b);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, a, b);
  (void)hipEventDestroy(a);
  (void)hipEventDestroy(b);
  HIP_TRY(e);
  *avg_ms = (double)ms / D.n_layers;
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_device_errors(m2r2_ctx* c, hipStream_t stream, int32_t* bits) {
  if (!c || !bits) return fail(M2R2_E_INVALID, "NULL argument");
  HIP_TRY(hipMemcpyAsync(bits, c->ws.err, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_sync_check(m2r2_ctx* c, hipStream_t stream) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  hipError_t e = hipStreamSynchronize(stream);
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) return fail(M2R2_E_HIP, "asynchronous error: %s", hipGetErrorString(e));
  int32_t bits = 0;
  HIP_TRY(hipMemcpyAsync(&bits, c->ws.err, sizeof(int32_t), hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  if (bits) return fail(M2R2_E_STATE, "device error bits %#x", (unsigned)bits);
  return M2R2_OK;
}

}  // extern "C"

namespace {

// A decode step's arguments, checked and turned into the row map and the
// kernels' I/O block before anything is enqueued.
struct StepCall {
  RowMap rm;
  StepIO io;
  bool arla = false;   // the exit router decides the gates
};

m2r2_status decode_prepare(m2r2_ctx* c, int32_t batch, int32_t dual, const int32_t* tokens_d, int32_t* positions_d,
                           const m2r2_kv* kv, const m2r2_exit* ex, const m2r2_step_out* out, StepCall* sc) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (batch < 1 || batch > c->max_batch) return fail(M2R2_E_SHAPE, "batch %d not in [1,%d]", batch, c->max_batch);
  if (!tokens_d || !positions_d || !out || !out->next_token_d) return fail(M2R2_E_INVALID, "NULL tokens/positions/out");
  if (m2r2_status s = check_kv(c, kv)) return s;
  StepIO& io = sc->io;
  io = empty_io();
  io.tokens = tokens_d;
  io.positions = positions_d;
  io.next_token = out->next_token_d;
  io.exit_b_out = out->exit_boundary_d;
  io.signal_out = out->signal_d;
  io.logits_out = out->logits_d;
  io.h_out = out->h_out_d;
  io.p_out = out->p_out_d;
  io.advance = out->advance;
  io.mode = EX_OFF;
  if (dual && ex) {
    if (ex->mode < M2R2_EXIT_OFF || ex->mode > M2R2_EXIT_EXIT) return fail(M2R2_E_INVALID, "exit mode %d", ex->mode);
    if (ex->n_gates < 0 || (ex->n_gates > 0 && !ex->gates_h)) return fail(M2R2_E_INVALID, "gates");
    io.mode = ex->mode;
    io.tau = ex->tau;
    for (int i = 0; i < ex->n_gates; ++i) {
      const int g = ex->gates_h[i];
      if (g < 1 || g >= c->D.n_layers) return fail(M2R2_E_SHAPE, "gate %d not in [1,%d]", g, c->D.n_layers - 1);
      if (g < 64) io.gate_mask_lo |= 1ull << g;
      else io.gate_mask_hi |= 1ull << (g - 64);
    }
  }
  RowMap& rm = sc->rm;
  rm = empty_rowmap();
  rm.nseq = batch;
  const int per = dual ? 2 : 1;
  rm.M = batch * per;
  for (int s = 0; s < batch; ++s) {
    const int m = s * per;
    rm.first[s] = m;
    rm.cnt[s] = per;
    rm.seq[m] = s; rm.fast[m] = 0; rm.idx[m] = 0; rm.wr[m] = 1; rm.tok[m] = s;
    if (dual) {
      rm.seq[m + 1] = s; rm.fast[m + 1] = 1; rm.idx[m + 1] = 0; rm.wr[m + 1] = 0; rm.tok[m + 1] = s;
      rm.slow_of[m + 1] = m;
    }
  }
  if (c->moe.on && batch != 1) return fail(M2R2_E_UNSUPPORTED, "mixture-of-experts decoding takes batch 1");
  sc->arla = !c->moe.on && c->arla.on && io.mode != EX_OFF && (io.gate_mask_lo | io.gate_mask_hi);
  if (sc->arla && batch != 1) return fail(M2R2_E_UNSUPPORTED, "the latent-attention exit router takes batch 1");
  return M2R2_OK;
}

m2r2_status decode_launch(m2r2_ctx* c, StepCall& sc, const m2r2_kv* kv, const m2r2_step_out* out, int32_t dual,
                          hipStream_t stream) {
  if (c->moe.on) return run_moe_pass(c, sc.rm, sc.io, kv_ptrs(kv), out, dual != 0, stream);
  if (sc.arla) sc.io.arla_sig = c->ws.arla_sig;
  return run_pass(c, sc.rm, sc.io, kv_ptrs(kv), c->D.n_layers, stream);
}

// For the duration of one call, the context's per-call scratch pointers
// point into `dst` (the same offsets within the scratch block) instead of
// the workspace; restored on destruction.
struct ScratchRebase {
  m2r2_ctx* c;
  WS ws;
  SkWS sk;
  decltype(m2r2_ctx::pk) pk;
  ScratchRebase(m2r2_ctx* ctx, char* dst) : c(ctx), ws(ctx->ws), sk(ctx->skws), pk(ctx->pk) {
    const char* lo = c->ws_base + c->lay.scratch_begin;
    const char* hi = c->ws_base + c->lay.scratch_end;
    auto rb = [&](auto* p) {
      const char* q = (const char*)p;
      return (q >= lo && q < hi) ? (decltype(p))(dst + (q - lo)) : p;
    };
    WS& w = c->ws;
    w.X = rb(w.X); w.PIN = rb(w.PIN); w.QKV = rb(w.QKV); w.O = rb(w.O); w.ACT = rb(w.ACT);
    w.bin_d = rb(w.bin_d); w.bin_o = rb(w.bin_o); w.bin_gu = rb(w.bin_gu); w.uo = rb(w.uo); w.att = rb(w.att);
    w.att_cnt = rb(w.att_cnt); w.lm_val = rb(w.lm_val); w.lm_idx = rb(w.lm_idx); w.lm_cnt = rb(w.lm_cnt);
    w.exited = rb(w.exited); w.exitb = rb(w.exitb); w.reinit = rb(w.reinit); w.sig = rb(w.sig);
    w.arla_kv = rb(w.arla_kv); w.arla_q = rb(w.arla_q); w.arla_sig = rb(w.arla_sig); w.arla_cnt = rb(w.arla_cnt);
    w.fsc = rb(w.fsc); w.fqkv = rb(w.fqkv); w.lrz = rb(w.lrz);
    c->skws.part = rb(c->skws.part); c->skws.hier = rb(c->skws.hier); c->skws.cnt = rb(c->skws.cnt);
    c->pk.sd = rb(c->pk.sd); c->pk.so = rb(c->pk.so); c->pk.sgu = rb(c->pk.sgu); c->pk.bar = rb(c->pk.bar); c->pk.rel = rb(c->pk.rel);
  }
  ~ScratchRebase() {
    c->ws = ws;
    c->skws = sk;
    c->pk = pk;
  }
};

}  // namespace

extern "C" {

M2R2_API m2r2_status m2r2_decode_step(m2r2_ctx* c, int32_t batch, int32_t dual, const int32_t* tokens_d,
                                      int32_t* positions_d, const m2r2_kv* kv, const m2r2_exit* ex,
                                      const m2r2_step_out* out, hipStream_t stream) {
  StepCall sc;
  if (m2r2_status s = decode_prepare(c, batch, dual, tokens_d, positions_d, kv, ex, out, &sc)) return s;
  return decode_launch(c, sc, kv, out, dual, stream);
}

M2R2_API m2r2_status m2r2_decode_step_noalloc(m2r2_ctx* c, int32_t batch, int32_t dual, const int32_t* tokens_d,
                                              int32_t* positions_d, const m2r2_kv* kv, const m2r2_exit* ex,
                                              const m2r2_step_out* out, hipStream_t stream) {
  StepCall sc;
  if (m2r2_status s = decode_prepare(c, batch, dual, tokens_d, positions_d, kv, ex, out, &sc)) return s;
  if (c->moe.on)
    return fail(M2R2_E_UNSUPPORTED, "the no-allocation decode step is for dense models (an expert cache is "
                                    "context state in the workspace)");
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev != c->device)
    return fail(M2R2_E_STATE, "context created on device %d, but device %d is current", c->device, dev);
  const size_t need = c->lay.scratch_end - c->lay.scratch_begin;
  if (need > kNoAllocScratchBytes)
    return fail(M2R2_E_SHAPE, "the context's per-call scratch needs %zu bytes, above the static maximum of %zu "
                              "(create the context with a smaller max_batch or max_ctx)", need, kNoAllocScratchBytes);
  char* sp = (char*)scratch_ptr(dev);
  if (!sp) return fail(M2R2_E_STATE, "no scratch address on device %d", dev);
  // the arrival counters must start at zero (a fill kernel, not a memset:
  // the call may be captured into a graph)
  const size_t cnt_off = c->lay.counters_begin - c->lay.scratch_begin;
  const int n_cnt = (int)((c->lay.scratch_end - c->lay.counters_begin) / sizeof(uint32_t));
  k_fill_u32<<<std::max(1, std::min(64, (n_cnt + 255) / 256)), 256, 0, stream>>>((uint32_t*)(sp + cnt_off), n_cnt, 0u);
  HIP_TRY(hipGetLastError());
  ScratchRebase swap(c, sp);
  return decode_launch(c, sc, kv, out, dual, stream);
}

M2R2_API m2r2_status m2r2_set_arla(m2r2_ctx* c, const m2r2_arla* w) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (c->moe.on) return fail(M2R2_E_UNSUPPORTED, "the latent-attention exit router is for dense models");
  if (is_flops(c->cfg)) return fail(M2R2_E_UNSUPPORTED, "the exit router with the FLOPs-optimised fast stream");
  if (!w) {
    c->arla.on = false;
    return M2R2_OK;
  }
  if (!w->wq || !w->wk || !w->wv || !w->w_out || !w->b_out) return fail(M2R2_E_INVALID, "NULL router weight");
  c->arla.wq = (const char*)w->wq;
  c->arla.wk = (const char*)w->wk;
  c->arla.wv = (const char*)w->wv;
  c->arla.w_out = w->w_out;
  c->arla.b_out = w->b_out;
  c->arla.on = true;
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_draft(m2r2_ctx* c, const int32_t* last_token_d, const int32_t* positions_d,
                                int32_t exit_layer, int32_t gamma, const m2r2_kv* kv, int32_t* drafts_d,
                                hipStream_t stream) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (!last_token_d || !positions_d || !drafts_d) return fail(M2R2_E_INVALID, "NULL token/position/drafts");
  if (c->moe.on) return fail(M2R2_E_UNSUPPORTED, "drafting is implemented for dense models");
  if (is_flops(c->cfg))
    return fail(M2R2_E_UNSUPPORTED, "a fast-only draft has no slow-row scores: the FLOPs-optimised fast stream "
                                    "is the dual-stream step's");
  if (exit_layer < 1 || exit_layer > c->D.n_layers) return fail(M2R2_E_SHAPE, "exit_layer %d", exit_layer);
  if (gamma < 1 || gamma > 64) return fail(M2R2_E_SHAPE, "gamma %d not in [1,64]", gamma);
  if (m2r2_status s = check_kv(c, kv)) return s;
  RowMap rm = empty_rowmap();
  rm.M = 1; rm.nseq = 1; rm.first[0] = 0; rm.cnt[0] = 1;
  rm.seq[0] = 0; rm.fast[0] = 1; rm.idx[0] = 0; rm.wr[0] = 1; rm.tok[0] = 0; rm.slow_of[0] = -1;
  for (int j = 0; j < gamma; ++j) {
    StepIO io = empty_io();
    io.tokens = j == 0 ? last_token_d : drafts_d + (j - 1);
    io.positions = const_cast<int32_t*>(positions_d);
    io.next_token = drafts_d;
    io.draft_slot = j;
    io.mode = EX_OFF;
    rm.pos_offset = j;
    if (m2r2_status s = run_pass(c, rm, io, kv_ptrs(kv), exit_layer, stream)) return s;
  }
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_verify(m2r2_ctx* c, const int32_t* chunk_d, int32_t n, int32_t* positions_d,
                                 const m2r2_kv* kv, int32_t* targets_d, int32_t* n_accepted_d,
                                 int32_t* bonus_token_d, hipStream_t stream) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (!chunk_d || !positions_d || !targets_d) return fail(M2R2_E_INVALID, "NULL chunk/positions/targets");
  if (c->moe.on) return fail(M2R2_E_UNSUPPORTED, "chunk verification is implemented for dense models");
  if (n < 1 || n > c->max_chunk) return fail(M2R2_E_SHAPE, "chunk %d not in [1,%d]", n, c->max_chunk);
  if (m2r2_status s = check_kv(c, kv)) return s;
  RowMap rm = empty_rowmap();
  rm.M = n; rm.nseq = 1; rm.first[0] = 0; rm.cnt[0] = n; rm.head_all = 1;
  for (int i = 0; i < n; ++i) {
    rm.seq[i] = 0; rm.fast[i] = 0; rm.idx[i] = i; rm.wr[i] = 1; rm.tok[i] = i;
  }
  StepIO io = empty_io();
  io.tokens = chunk_d;
  io.positions = positions_d;
  io.targets = targets_d;
  io.n_acc = n_accepted_d;
  io.bonus = bonus_token_d;
  io.n_chunk = n;
  io.mode = EX_OFF;
  return run_pass(c, rm, io, kv_ptrs(kv), c->D.n_layers, stream);
}

M2R2_API m2r2_status m2r2_expert_bytes(const m2r2_config* cfg, size_t* bytes_out) {
  if (!cfg || !bytes_out) return fail(M2R2_E_INVALID, "NULL argument");
  if (cfg->wdtype != M2R2_F32 && cfg->wdtype != M2R2_BF16) return fail(M2R2_E_DTYPE, "wdtype %d", cfg->wdtype);
  const int kstep = cfg->wdtype == M2R2_BF16 ? 32 : 16;
  if (!is_moe(*cfg)) return fail(M2R2_E_SHAPE, "not a mixture-of-experts config");
  if (cfg->d_model <= 0 || cfg->d_model % kstep || cfg->expert_ffn <= 0 || cfg->expert_ffn % kstep)
    return fail(M2R2_E_SHAPE, "d_model and expert_ffn must be positive multiples of %d", kstep);
  *bytes_out = expert_bytes_of(*cfg);
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_pack_expert(const m2r2_config* cfg, const void* wg_h, const void* wu_h, const void* wd_h,
                                      void* dst_h) {
  size_t total = 0;
  if (m2r2_status st = m2r2_expert_bytes(cfg, &total)) return st;
  if (!wg_h || !wu_h || !wd_h || !dst_h) return fail(M2R2_E_INVALID, "NULL matrix or destination");
  const int wb = cfg->wdtype == M2R2_BF16, esz = wb ? 2 : 4, kstep = wb ? 32 : 16, epl = kstep / 4;
  const int d = cfg->d_model, Fe = cfg->expert_ffn;
  char* dst = (char*)dst_h;
  // same tile-packed layout as the device packing kernel
  auto pack = [&](const char* src, int rows, int K, char* out) {
    const int S = K / kstep;
    const int tiles = (rows + 15) / 16;
    for (int t = 0; t < tiles; ++t)
      for (int st = 0; st < S; ++st)
        for (int l = 0; l < 64; ++l) {
          const int r = t * 16 + (l & 15), col = st * kstep + epl * (l >> 4);
          char* o = out + (((size_t)t * S + st) * 64 + l) * 16;
          if (r < rows) memcpy(o, src + ((size_t)r * K + col) * esz, 16);
          else memset(o, 0, 16);
        }
  };
  const size_t mat = packed_bytes(Fe, d, wb);
  pack((const char*)wg_h, Fe, d, dst);
  pack((const char*)wu_h, Fe, d, dst + mat);
  pack((const char*)wd_h, d, Fe, dst + 2 * mat);
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_moe_set_policy(m2r2_ctx* c, int32_t policy) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (!c->moe.on) return fail(M2R2_E_STATE, "not a mixture-of-experts context");
  if (policy < M2R2_MOE_ON_DEMAND || policy > M2R2_MOE_PREVIOUS_LAYER) return fail(M2R2_E_INVALID, "policy %d", policy);
  c->moe.policy = policy;
  HIP_TRY(moe_warm(c));
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_moe_set_preload_table(m2r2_ctx* c, const int32_t* ids_h, int32_t n_tokens) {
  if (!c || !ids_h) return fail(M2R2_E_INVALID, "NULL argument");
  MoeState& M = c->moe;
  if (!M.on) return fail(M2R2_E_STATE, "not a mixture-of-experts context");
  if (n_tokens < 1) return fail(M2R2_E_SHAPE, "n_tokens %d", n_tokens);
  const size_t n = (size_t)n_tokens * c->D.n_layers * M.K;
  for (size_t i = 0; i < n; ++i)
    if (ids_h[i] < -1 || ids_h[i] >= M.E) return fail(M2R2_E_SHAPE, "preload expert id %d", ids_h[i]);
  M.preload.assign(ids_h, ids_h + n);
  M.preload_tokens = n_tokens;
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_prefetch_experts(m2r2_ctx* c, int32_t layer, const int32_t* ids_h, int32_t n,
                                           int32_t priority, hipStream_t copy_stream) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  MoeState& M = c->moe;
  if (!M.on) return fail(M2R2_E_STATE, "not a mixture-of-experts context");
  if (M.policy == M2R2_MOE_FIXED) return fail(M2R2_E_STATE, "the fixed-experts policy takes no prefetches");
  if (layer < 0 || layer >= c->D.n_layers) return fail(M2R2_E_SHAPE, "layer %d", layer);
  if (n < 0 || n > M.C || (n > 0 && !ids_h)) return fail(M2R2_E_SHAPE, "n %d not in [0, slots]", n);
  for (int i = 0; i < n; ++i) {
    if (ids_h[i] >= M.E) return fail(M2R2_E_SHAPE, "expert id %d >= n_experts", ids_h[i]);
    for (int j = 0; j < i; ++j)
      if (ids_h[i] >= 0 && ids_h[i] == ids_h[j]) return fail(M2R2_E_INVALID, "expert %d listed twice", ids_h[i]);
  }
  hipStream_t cs = copy_stream ? copy_stream : (priority ? M.copy_demand : M.copy_ahead);
  std::vector<int> slots, experts;
  M.pol.predict(layer, ids_h, n, &slots, &experts);
  for (size_t q = 0; q < slots.size(); ++q) {
    tab_evict_slot(M, layer, slots[q]);
    if (moe_copy(c, layer, slots[q], experts[q], cs) != hipSuccess) {
      (void)hipGetLastError();
      M.pol.invalidate(layer, slots[q]);   // not resident: a later use loads it on demand
      continue;
    }
    if (M.spec) M.pend.push_back({layer, slots[q], experts[q]});
  }
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_moe_reset(m2r2_ctx* c) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (!c->moe.on) return fail(M2R2_E_STATE, "not a mixture-of-experts context");
  HIP_TRY(moe_warm(c));
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_moe_stats(m2r2_ctx* c, m2r2_moe_counters* out) {
  if (!c || !out) return fail(M2R2_E_INVALID, "NULL argument");
  if (!c->moe.on) return fail(M2R2_E_STATE, "not a mixture-of-experts context");
  fill_stats(c->moe.pol.counters(), out);
  if (c->moe.hits_dev_used) {   // hits counted by the expert kernels of resident tokens
    unsigned long long h = 0;
    HIP_TRY(hipDeviceSynchronize());
    HIP_TRY(hipMemcpy(&h, c->moe.hits_d, sizeof h, hipMemcpyDeviceToHost));
    out->hits += (int64_t)h;
  }
  out->h2d_bytes = c->moe.h2d_bytes;
  out->copy_waits = c->moe.copy_waits;
  out->host_wait_ns = c->moe.host_wait_ns;
  return M2R2_OK;
}

M2R2_API m2r2_status m2r2_expert_cache_replay(int32_t n_layers, int32_t n_experts, int32_t top_k, int32_t slots,
                                              int32_t n_tokens, const int32_t* slow_h, const int32_t* pred_h,
                                              int32_t policy, m2r2_moe_counters* out) {
  if (!slow_h || !out) return fail(M2R2_E_INVALID, "NULL argument");
  if (policy < M2R2_MOE_ON_DEMAND || policy > M2R2_MOE_PREVIOUS_LAYER) return fail(M2R2_E_INVALID, "policy %d", policy);
  if (n_layers < 1 || n_layers > 127 || n_experts < 1 || top_k < 1 || top_k > kMaxTopK || n_tokens < 0)
    return fail(M2R2_E_SHAPE, "sizes");
  if (slots < top_k || slots > n_experts) return fail(M2R2_E_SHAPE, "need top_k <= slots <= n_experts");
  const size_t per_tok = (size_t)n_layers * top_k;
  for (size_t i = 0; i < per_tok * n_tokens; ++i) {
    if (slow_h[i] < 0 || slow_h[i] >= n_experts) return fail(M2R2_E_SHAPE, "slow expert id %d", slow_h[i]);
    if (pred_h && pred_h[i] >= n_experts) return fail(M2R2_E_SHAPE, "predicted expert id %d", pred_h[i]);
  }
  ExpertCachePolicy pol;
  pol.init(n_layers, n_experts, slots);
  int slot[kMaxTopK];
  bool load[kMaxTopK];
  std::vector<int> s1, e1;
  for (int t = 0; t < n_tokens; ++t) {
    for (int l = 0; l < n_layers; ++l) {
      const int32_t* need = slow_h + t * per_tok + l * top_k;
      if (policy == M2R2_MOE_FIXED) {
        pol.use_fixed(l, need, top_k, slot, load);
        continue;
      }
      pol.use(l, need, top_k, slot, load);
      if (!pred_h || policy == M2R2_MOE_ON_DEMAND) continue;
      const int lp0 = policy == M2R2_MOE_AHEAD_OF_TIME ? 2 * l + 2 : l + 1;
      const int lp1 = policy == M2R2_MOE_AHEAD_OF_TIME ? 2 * l + 3 : l + 1;
      for (int lp = lp0; lp <= lp1 && lp < n_layers; ++lp)
        pol.predict(lp, pred_h + t * per_tok + lp * top_k, top_k, &s1, &e1);
    }
    pol.end_token();
  }
  fill_stats(pol.counters(), out);
  return M2R2_OK;
}

}  // extern "C"
