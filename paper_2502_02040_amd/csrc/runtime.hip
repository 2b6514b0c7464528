// Host runtime and C ABI of the M2R2 decode path (see include/m2r2.h).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "m2r2.h"
#include "step_kernels.h"

using namespace m2r2;

namespace {

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

// Context splits of the attention for `nseq` sequences of `rows` rows each.
int choose_splits(int nseq, int rows, int H, int max_ctx) {
  const int target = std::max(1, (1024 + nseq * H - 1) / (nseq * H));
  const int useful = std::max(1, (max_ctx + 63) / 64);
  const int need = std::max(1, (max_ctx + per_max(rows) - 1) / per_max(rows));
  return std::max(need, std::min(target, useful));
}

struct Layout {
  size_t X, PIN, QKV, O, ACT, part_d, part_o, part_gu, uo, att, att_cnt, lm_val, lm_idx, lm_cnt, exited, exitb,
      reinit, err, sig, total;
  int TD, TF, TV, S_max;
};

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
  L.X = take(sizeof(float) * kMaxRows * d);
  L.PIN = take(sizeof(float) * kMaxRows * d);
  L.QKV = take(sizeof(float) * kMaxRows * nqkv);
  L.O = take(sizeof(float) * kMaxRows * qdim);
  L.ACT = take(sizeof(float) * kMaxRows * std::max(c.ffn, 1));
  L.part_d = take(sizeof(float) * L.TD * kMaxRows * 4);
  L.part_o = take(sizeof(float) * L.TD * kMaxRows * (1 + 2 * r));
  L.part_gu = take(sizeof(float) * L.TF * kMaxRows * std::max(r, 1));
  L.uo = take(sizeof(float) * kMaxRows * c.n_heads * std::max(r, 1));
  L.att = take(sizeof(float) * (size_t)std::max(max_batch, 1) * c.n_heads * smax * kMaxRows * (c.head_dim + 2));
  L.att_cnt = take(sizeof(uint32_t) * kMaxSeq * c.n_heads);
  L.lm_val = take(sizeof(float) * L.TV * kMaxRows);
  L.lm_idx = take(sizeof(int) * L.TV * kMaxRows);
  L.lm_cnt = take(sizeof(uint32_t));
  L.exited = take(sizeof(int) * kMaxSeq);
  L.exitb = take(sizeof(int) * kMaxSeq);
  L.reinit = take(sizeof(int) * c.n_layers * kMaxSeq);
  L.err = take(sizeof(int));
  L.sig = take(sizeof(float) * kMaxSeq * c.n_layers);
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
  if (c->ffn <= 0 || c->ffn % kstep) return fail(M2R2_E_SHAPE, "ffn %d not a multiple of %d", c->ffn, kstep);
  if (c->head_dim != 64 && c->head_dim != 96 && c->head_dim != 128)
    return fail(M2R2_E_UNSUPPORTED, "head_dim %d (supported: 64, 96, 128)", c->head_dim);
  if (c->n_heads < 1 || (c->n_heads * c->head_dim) % kstep)
    return fail(M2R2_E_SHAPE, "n_heads*head_dim %d not a multiple of %d", c->n_heads * c->head_dim, kstep);
  if (c->rank < 1 || c->rank > kMaxRank) return fail(M2R2_E_SHAPE, "rank %d not in [1,%d]", c->rank, kMaxRank);
  if (c->vocab < 1) return fail(M2R2_E_SHAPE, "vocab %d", c->vocab);
  if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f)) return fail(M2R2_E_INVALID, "rms_eps/rope_theta");
  if (max_batch < 1 || max_batch > 8) return fail(M2R2_E_SHAPE, "max_batch %d not in [1,8]", max_batch);
  if (max_chunk < 1 || max_chunk > kMaxRows) return fail(M2R2_E_SHAPE, "max_chunk %d not in [1,16]", max_chunk);
  if (max_ctx < 1) return fail(M2R2_E_SHAPE, "max_ctx %d", max_ctx);
  return M2R2_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

struct m2r2_ctx {
  m2r2_config cfg;
  Dims D;
  Layout lay;
  std::vector<LayerPtrs> layers;
  const void* embed;
  const float* final_norm;
  const void* lm_head;
  int max_batch, max_chunk, max_ctx;
  WS ws;
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

template <int WB, int KB, int HD>
m2r2_status run_layers_t(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int n_layers_run,
                         hipStream_t st) {
  const Dims& D = c->D;
  const int nqkv = 3 * D.qdim + 3 * D.r;
  int rows_per_seq = 1;
  for (int s = 0; s < rm.nseq; ++s) rows_per_seq = std::max(rows_per_seq, (int)rm.cnt[s]);
  const int S = choose_splits(rm.nseq, rows_per_seq, D.H, c->max_ctx);
  if (S > c->lay.S_max) return fail(M2R2_E_SHAPE, "attention splits exceed the workspace");
  const size_t smem = attn_smem_bytes();
  for (int l = 0; l < n_layers_run; ++l) {
    const LayerPtrs& L = c->layers[l];
    k_qkv<WB><<<(nqkv + 15) / 16, kGemvThreads, 0, st>>>(D, L, rm, c->ws, io, l, l == 0 ? 1 : c->lay.TD);
    k_attn<KB, HD><<<dim3(S, D.H, rm.nseq), kAttnThreads, smem, st>>>(D, L, rm, c->ws, io, kv, l, S);
    k_oproj<WB><<<c->lay.TD, kGemvThreads, 0, st>>>(D, L, rm, c->ws, io, l);
    k_gateup<WB><<<c->lay.TF, kGemvThreads, 0, st>>>(D, L, rm, c->ws, io, c->lay.TD);
    k_down<WB><<<c->lay.TD, kGemvThreads, 0, st>>>(D, L, rm, c->ws, io, c->lay.TF);
  }
  k_head<WB><<<c->lay.TV, kGemvThreads, 0, st>>>(D, c->lm_head, c->final_norm, rm, c->ws, io, kv,
                                                 n_layers_run == 0 ? 1 : c->lay.TD, c->lay.TV);
  HIP_TRY(hipGetLastError());
  return M2R2_OK;
}

template <int WB, int KB>
m2r2_status run_hd(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int nl, hipStream_t st) {
  switch (c->D.hd) {
    case 64: return run_layers_t<WB, KB, 64>(c, rm, io, kv, nl, st);
    case 96: return run_layers_t<WB, KB, 96>(c, rm, io, kv, nl, st);
    case 128: return run_layers_t<WB, KB, 128>(c, rm, io, kv, nl, st);
  }
  return fail(M2R2_E_UNSUPPORTED, "head_dim");
}

// Embedding, n_layers_run layers, head.
m2r2_status run_pass(m2r2_ctx* c, const RowMap& rm, const StepIO& io, const KVPtrs& kv, int nl, hipStream_t st) {
  k_embed<<<rm.M, 256, 0, st>>>(c->D, c->embed, rm, c->ws, io, 1);
  HIP_TRY(hipGetLastError());
  const int wb = c->D.wbf16, kb = c->D.kvbf16;
  if (wb && kb) return run_hd<1, 1>(c, rm, io, kv, nl, st);
  if (wb && !kb) return run_hd<1, 0>(c, rm, io, kv, nl, st);
  if (!wb && kb) return run_hd<0, 1>(c, rm, io, kv, nl, st);
  return run_hd<0, 0>(c, rm, io, kv, nl, st);
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
  for (int l = 0; l < cfg->n_layers; ++l) {
    const m2r2_layer_weights& L = w->layers[l];
    if (!L.attn_norm || !L.wq || !L.wk || !L.wv || !L.wo || !L.mlp_norm || !L.wg || !L.wu || !L.wd)
      return fail(M2R2_E_INVALID, "layer %d: a base weight pointer is NULL", l);
    const void* ps[] = {L.wq, L.wk, L.wv, L.wo, L.wg, L.wu, L.wd, w->embed, w->lm_head};
    for (const void* p : ps)
      if (!aligned16(p)) return fail(M2R2_E_INVALID, "layer %d: weight not 16-byte aligned", l);
    for (int a = 0; a < 7; ++a)
      if ((L.A[a] == nullptr) != (L.B[a] == nullptr))
        return fail(M2R2_E_INVALID, "layer %d adapter %d: A and B must be both set or both NULL", l, a);
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
  c->lm_head = w->lm_head;
  Dims& D = c->D;
  D.n_layers = cfg->n_layers; D.d = cfg->d_model; D.H = cfg->n_heads; D.hd = cfg->head_dim;
  D.qdim = cfg->n_heads * cfg->head_dim; D.F = cfg->ffn; D.V = cfg->vocab; D.r = cfg->rank;
  D.eps = cfg->rms_eps; D.theta = cfg->rope_theta; D.wbf16 = cfg->wdtype == M2R2_BF16; D.kvbf16 = cfg->kvdtype == M2R2_BF16;
  c->layers.resize(cfg->n_layers);
  for (int l = 0; l < cfg->n_layers; ++l) {
    const m2r2_layer_weights& s = w->layers[l];
    LayerPtrs& L = c->layers[l];
    L.attn_norm = s.attn_norm; L.wq = s.wq; L.wk = s.wk; L.wv = s.wv; L.wo = s.wo;
    L.mlp_norm = s.mlp_norm; L.wg = s.wg; L.wu = s.wu; L.wd = s.wd;
    for (int a = 0; a < 7; ++a) { L.A[a] = s.A[a]; L.B[a] = s.B[a]; }
  }
  char* b = (char*)workspace;
  WS& ws = c->ws;
  ws.X = (float*)(b + lay.X); ws.PIN = (float*)(b + lay.PIN); ws.QKV = (float*)(b + lay.QKV);
  ws.O = (float*)(b + lay.O); ws.ACT = (float*)(b + lay.ACT); ws.part_d = (float*)(b + lay.part_d);
  ws.part_o = (float*)(b + lay.part_o); ws.part_gu = (float*)(b + lay.part_gu); ws.uo = (float*)(b + lay.uo);
  ws.att = (float*)(b + lay.att); ws.att_cnt = (uint32_t*)(b + lay.att_cnt); ws.lm_val = (float*)(b + lay.lm_val);
  ws.lm_idx = (int*)(b + lay.lm_idx); ws.lm_cnt = (uint32_t*)(b + lay.lm_cnt); ws.exited = (int*)(b + lay.exited);
  ws.exitb = (int*)(b + lay.exitb); ws.reinit = (int*)(b + lay.reinit); ws.err = (int*)(b + lay.err);
  ws.sig = (float*)(b + lay.sig);
  hipError_t e = hipMemset(workspace, 0, lay.total);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    delete c;
    return fail(M2R2_E_HIP, "workspace init: %s", hipGetErrorString(e));
  }
  *out = c;
  return M2R2_OK;
}

M2R2_API void m2r2_destroy(m2r2_ctx* ctx) { delete ctx; }

M2R2_API m2r2_status m2r2_decode_step(m2r2_ctx* c, int32_t batch, int32_t dual, const int32_t* tokens_d,
                                      int32_t* positions_d, const m2r2_kv* kv, const m2r2_exit* ex,
                                      const m2r2_step_out* out, hipStream_t stream) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (batch < 1 || batch > c->max_batch) return fail(M2R2_E_SHAPE, "batch %d not in [1,%d]", batch, c->max_batch);
  if (!tokens_d || !positions_d || !out || !out->next_token_d) return fail(M2R2_E_INVALID, "NULL tokens/positions/out");
  if (m2r2_status s = check_kv(c, kv)) return s;
  StepIO io = empty_io();
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
  RowMap rm = empty_rowmap();
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
  return run_pass(c, rm, io, kv_ptrs(kv), c->D.n_layers, stream);
}

M2R2_API m2r2_status m2r2_draft(m2r2_ctx* c, const int32_t* last_token_d, const int32_t* positions_d,
                                int32_t exit_layer, int32_t gamma, const m2r2_kv* kv, int32_t* drafts_d,
                                hipStream_t stream) {
  if (!c) return fail(M2R2_E_INVALID, "ctx is NULL");
  if (!last_token_d || !positions_d || !drafts_d) return fail(M2R2_E_INVALID, "NULL token/position/drafts");
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

}  // extern "C"
