// Decode-path kernels for gfx950: the dual-stream layer step of M2R2
// (slow residual h, Eq. 1; accelerated residual p, Eq. 2), its chunked slow
// forward (verification / prefill) and its fast-only draft.
//
// A "row" is one residual vector of one sequence: the slow row, the fast
// row, or one token of a slow chunk.  Up to 16 rows are processed by every
// kernel; each weight element is read from HBM once and applied to all rows
// (an MFMA tile is 16 rows high, so the rows ride in the MFMA's M dimension).
//
// Per layer the step launches five kernels:
//   qkv    : gate logic for the boundary before the layer, then
//            [Wq;Wk;Wv;Aq;Ak;Av] x rms(x)*g_att          (adapter-down rows appended)
//   attn   : per (sequence, head, context split): q/k/v with adapter-up and
//            RoPE, slow k/v written to the paged cache, split attention over
//            the shared cache; the last split merges and adds each row's own
//            keys (fast row: its own exact k/v; slow rows: the chunk so far)
//   o      : Wo, residual add, adapter; partial sums for the next norm and
//            for the gate/up adapter-down projection
//   gateup : [Wg;Wu] paired tiles, adapter-up, SiLU(g)*u; partials of the
//            down adapter-down projection
//   down   : Wd, residual add, adapter; partial sums for the next layer's
//            norm and for the exit signal cos(p_in, p_out)
// and the head kernel runs the final norm, the LM head and a two-level argmax.
#pragma once
#include "device_common.h"

namespace m2r2 {

enum { EX_OFF = 0, EX_OBSERVE = 1, EX_EXIT = 2 };

struct Dims {
  int n_layers, d, H, hd, qdim, F, V, r;
  float eps, theta;
  int wbf16, kvbf16;
};

struct LayerPtrs {
  const float* attn_norm;
  const void *wq, *wk, *wv, *wo;
  const float* mlp_norm;
  const void *wg, *wu, *wd;
  const void* A[7];
  const void* B[7];
};

// Row bookkeeping, passed by value.  Rows of one sequence are contiguous.
struct RowMap {
  int M, nseq;
  int head_all;          // every row feeds the LM head (chunk verification)
  int pos_offset;        // added to positions_d[s] (draft step j uses t + j)
  int8_t seq[kMaxRows];  // sequence of the row
  int8_t fast[kMaxRows]; // accelerated row
  int8_t idx[kMaxRows];  // position offset of the row within its sequence
  int8_t wr[kMaxRows];   // row writes its key/value to the cache
  int8_t slow_of[kMaxRows];  // fast row: slow row of the same sequence (-1: none)
  int8_t tok[kMaxRows];  // index into the token array
  int8_t first[kMaxSeq], cnt[kMaxSeq];
};

struct KVPtrs {
  void* k;
  void* v;
  const int* bt;     // [nseq][mbps]
  int* seq_lens;
  int num_blocks, bs, mbps;
};

// Workspace views (all device pointers).
struct WS {
  float* X;        // [16][d]       residual rows
  float* PIN;      // [16][d]       fast rows at layer entry
  float* QKV;      // [16][nqkv]    q|k|v|u_q|u_k|u_v (already divided by rms)
  float* O;        // [16][qdim]    attention output
  float* ACT;      // [16][F]       SwiGLU activation
  float* part_d;   // [TD][16][4]   per 16-row tile of d: sum x^2, sum pin*x, sum pin^2
  float* part_o;   // [TD][16][1+2r] sum x^2, adapter-down partials of gate and up
  float* part_gu;  // [TF][16][r]   adapter-down partials of down
  float* uo;       // [16][H][r]    adapter-down of o, per head
  float* att;      // [nseq][H][S][rows][hd+2] split partials
  uint32_t* att_cnt;  // [16][H] arrival counters
  float* lm_val;   // [TV][16]
  int* lm_idx;     // [TV][16]
  uint32_t* lm_cnt;
  int* exited;     // [16]
  int* exitb;      // [16]
  int* reinit;     // [n_layers][16]
  int* err;        // sticky device error bits
  float* sig;      // [16][n_layers] scratch signal (copied to the caller's buffer if any)
};

struct StepIO {
  const int* tokens;     // token array indexed by RowMap::tok
  int* positions;        // [nseq]
  int* next_token;       // decode/draft: [nseq] (draft: drafts array, written at draft_slot)
  int draft_slot;
  int* exit_b_out;
  float* signal_out;     // [nseq][n_layers]
  float* logits_out;     // [rows fed to the head][V]
  float* h_out;
  float* p_out;
  int advance;
  // verification
  int* targets;
  int* n_acc;
  int* bonus;
  int n_chunk;
  // exit settings
  int mode;
  float tau;
  unsigned long long gate_mask_lo, gate_mask_hi;   // bit b: boundary b is a gate (b < 128)
};

__device__ __forceinline__ bool is_gate(const StepIO& io, int b) {
  if (b <= 0) return false;
  if (b < 64) return (io.gate_mask_lo >> b) & 1ull;
  if (b < 128) return (io.gate_mask_hi >> (b - 64)) & 1ull;
  return false;
}

__device__ __forceinline__ int row_pos(const RowMap& rm, const StepIO& io, int m) {
  return io.positions[rm.seq[m]] + rm.pos_offset + rm.idx[m];
}

// ============================================================================
// Small-M GEMV core on MFMA.
//
// One workgroup of 8 waves owns a tile of 16 consecutive weight rows (two
// tiles for the paired gate/up projection).  The waves split the reduction
// dimension; each lane streams 16-byte pieces of one weight row with
// non-temporal loads and the matching 8 (bf16) or 4 (f32) activations of up
// to 16 rows.  bf16 weights: v_mfma_f32_16x16x32_bf16 with the fp32
// activations split into bf16 hi + lo parts (two MFMAs, ~16 significant bits
// of the activation).  f32 weights: four v_mfma_f32_16x16x4_f32 per 16-byte
// piece (exact fp32 products).  Accumulation is fp32.  The 8 partial results
// are summed through LDS.
// ============================================================================
constexpr int kGemvWaves = 8;
constexpr int kGemvThreads = kGemvWaves * 64;
constexpr int kBatch = 8;   // K-steps whose weight loads are in flight per wave

struct XSrc {
  const float* row;   // activation row of this lane's m (nullptr: zero)
  const float* gain;  // per-k gain or nullptr
};

template <int WB>
__device__ __forceinline__ void mfma_step(const u32x4_t w, const float* xr, const float* g, int k, int grp,
                                          f32x4_t& acc) {
  if constexpr (WB) {
    float xv[8];
    if (xr) {
      float4 a = ld4(xr + k + 8 * grp), b = ld4(xr + k + 8 * grp + 4);
      xv[0] = a.x; xv[1] = a.y; xv[2] = a.z; xv[3] = a.w; xv[4] = b.x; xv[5] = b.y; xv[6] = b.z; xv[7] = b.w;
      if (g) {
        float4 ga = ld4(g + k + 8 * grp), gb = ld4(g + k + 8 * grp + 4);
        xv[0] *= ga.x; xv[1] *= ga.y; xv[2] *= ga.z; xv[3] *= ga.w;
        xv[4] *= gb.x; xv[5] *= gb.y; xv[6] *= gb.z; xv[7] *= gb.w;
      }
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) xv[i] = 0.f;
    }
    bf16x8_t hi, lo;
    split_hi_lo(xv, hi, lo);
    const bf16x8_t wb = __builtin_bit_cast(bf16x8_t, w);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(hi, wb, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(lo, wb, acc, 0, 0, 0);
  } else {
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
    if (xr) {
      a = ld4(xr + k + 4 * grp);
      if (g) {
        float4 ga = ld4(g + k + 4 * grp);
        a.x *= ga.x; a.y *= ga.y; a.z *= ga.z; a.w *= ga.w;
      }
    }
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, __uint_as_float(w[0]), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, __uint_as_float(w[1]), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, __uint_as_float(w[2]), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, __uint_as_float(w[3]), acc, 0, 0, 0);
  }
}

// Accumulate NT tiles over this wave's K range.  wrow[t]: this lane's weight
// row of tile t (nullptr: row absent -> contributes 0).
template <int WB, int NT>
__device__ __forceinline__ void gemv_wave(const void* const (&wrow)[NT], XSrc xs, int K, f32x4_t (&acc)[NT]) {
  constexpr int KSTEP = WB ? 32 : 16;
  constexpr int EPL = WB ? 8 : 4;          // elements per lane per step
  constexpr int ESZ = WB ? 2 : 4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int grp = lane >> 4;
  const int nsteps = K / KSTEP;
  const int per = (nsteps + kGemvWaves - 1) / kGemvWaves;
  const int s0 = wave * per;
  const int s1 = min(nsteps, s0 + per);
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  for (int sb = s0; sb < s1; sb += kBatch) {
    u32x4_t w[NT][kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (sb + j < s1) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          if (wrow[t])
            w[t][j] = ld_stream((const char*)wrow[t] + ((size_t)(sb + j) * KSTEP + EPL * grp) * ESZ);
          else
            w[t][j] = u32x4_t{0u, 0u, 0u, 0u};
        }
      }
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (sb + j < s1) {
        const int k = (sb + j) * KSTEP;
#pragma unroll
        for (int t = 0; t < NT; ++t) mfma_step<WB>(w[t][j], xs.row, xs.gain, k, grp, acc[t]);
      }
    }
  }
}

// Sum the per-wave accumulators into y[t][m][n] (LDS, NT x 16 x 16 floats).
// red: LDS scratch of kGemvWaves * NT * 256 floats.
template <int NT>
__device__ __forceinline__ void gemv_reduce(const f32x4_t (&acc)[NT], int M, float* red, float* y) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, mb = (lane >> 4) * 4;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (mb + i < M) red[((wave * NT + t) * 16 + mb + i) * 16 + n] = acc[t][i];
  __syncthreads();
  for (int e = threadIdx.x; e < NT * 256; e += kGemvThreads) {
    const int t = e >> 8, m = (e >> 4) & 15;
    if (m < M) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < kGemvWaves; ++w) s += red[((w * NT + t) * 16 + m) * 16 + (e & 15)];
      y[e] = s;
    }
  }
  __syncthreads();
}

__device__ __forceinline__ float ld_w(const void* p, size_t i, int wb) {
  return wb ? bf16_to_f32(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}

// ============================================================================
// Kernel: embedding gather + per-step control initialisation.
// grid = M rows, block = 256.
// ============================================================================
__global__ __launch_bounds__(256) void k_embed(Dims D, const void* embed, RowMap rm, WS ws, StepIO io, int init_ctl) {
  __shared__ float red[4];
  const int m = blockIdx.x;
  const int tok = io.tokens[rm.tok[m]];
  const bool ok = tok >= 0 && tok < D.V;
  if (!ok && threadIdx.x == 0) atomicOr(ws.err, 1);
  float ss = 0.f;
  for (int i = threadIdx.x; i < D.d; i += 256) {
    const float v = ok ? ld_w(embed, (size_t)tok * D.d + i, D.wbf16) : 0.f;
    ws.X[m * D.d + i] = v;
    ws.PIN[m * D.d + i] = v;
    ss += v * v;
  }
  ss = block_sum(ss, red);
  if (threadIdx.x == 0) {
    float* pd = ws.part_d + m * 4;
    pd[0] = ss; pd[1] = ss; pd[2] = ss; pd[3] = 0.f;
  }
  if (init_ctl && m == 0) {
    for (int s = threadIdx.x; s < kMaxSeq; s += 256) {
      ws.exited[s] = 0;
      ws.exitb[s] = D.n_layers;
    }
  }
}

// Gate decision for the boundary before `layer`, identical in every
// workgroup (same inputs, same summation order).  Fills, per sequence,
// reinit (p <- h for this layer) and the updated exited flag / boundary;
// sig[s] receives the signal of layer-1.
__device__ void gate_logic(const Dims& D, const RowMap& rm, const WS& ws, const StepIO& io, int layer,
                           const float* ssum /* [16][4] */, int* reinit_s, int* exited_s, int* exitb_s, float* sig_s) {
  for (int s = 0; s < rm.nseq; ++s) {
    int ex = ws.exited[s], eb = ws.exitb[s], ri = 0;
    float sg = 0.f;
    const int f = rm.first[s] + rm.cnt[s] - 1;
    if (layer > 0 && rm.fast[f]) {
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      sg = dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
      if (!ex && io.mode != EX_OFF && is_gate(io, layer) && rm.slow_of[f] >= 0) {
        const bool fired = sg >= io.tau;
        if (fired && eb == D.n_layers) eb = layer;
        if (io.mode == EX_EXIT && fired) ex = 1;
        else ri = 1;
      }
    }
    reinit_s[s] = ri; exited_s[s] = ex; exitb_s[s] = eb; sig_s[s] = sg;
  }
}

// ============================================================================
// Kernel: QKV projection of every row (+ adapter-down rows), with the gate
// decision of the preceding boundary.  grid = tiles of 16 rows over
// [Wq; Wk; Wv; Aq; Ak; Av], block = 512.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_qkv(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer,
                                                      int n_part) {
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int reinit_s[kMaxSeq], exited_s[kMaxSeq], exitb_s[kMaxSeq];
  __shared__ float sig_s[kMaxSeq];
  __shared__ float inv_rms[kMaxRows];
  __shared__ int src_s[kMaxRows];
  const int nq = D.qdim;
  const int nqkv = 3 * nq + 3 * D.r;
  const int n0 = blockIdx.x * 16;
  // this lane's weight row
  const int lane = threadIdx.x & 63;
  const int n = n0 + (lane & 15);
  const void* wrow[1] = {nullptr};
  {
    const size_t esz = WB ? 2 : 4;
    if (n < 3 * nq) {
      const void* base = n < nq ? L.wq : (n < 2 * nq ? L.wk : L.wv);
      wrow[0] = (const char*)base + (size_t)(n % nq) * D.d * esz;
    } else if (n < nqkv) {
      const int a = (n - 3 * nq) / D.r, j = (n - 3 * nq) % D.r;
      if (L.A[a]) wrow[0] = (const char*)L.A[a] + (size_t)j * D.d * esz;
    }
  }
  // partial sums of the previous kernel -> per-row statistics
  for (int e = threadIdx.x; e < rm.M * 4; e += kGemvThreads) {
    float s = 0.f;
    for (int t = 0; t < n_part; ++t) s += ws.part_d[(t * kMaxRows) * 4 + e];
    ssum[e] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    gate_logic(D, rm, ws, io, layer, ssum, reinit_s, exited_s, exitb_s, sig_s);
    for (int m = 0; m < rm.M; ++m) {
      const int s = rm.seq[m];
      int src = m;
      if (rm.fast[m] && reinit_s[s]) src = rm.slow_of[m];
      src_s[m] = src;
      inv_rms[m] = rsqrtf(ssum[src * 4] / D.d + D.eps);
    }
  }
  __syncthreads();
  if (blockIdx.x == 0 && threadIdx.x < rm.nseq) {
    const int s = threadIdx.x;
    ws.reinit[layer * kMaxSeq + s] = reinit_s[s];
    ws.exited[s] = exited_s[s];
    ws.exitb[s] = exitb_s[s];
    if (layer > 0) ws.sig[s * D.n_layers + layer - 1] = sig_s[s];
  }
  // every sequence stopped: only the K and V rows are still needed
  bool all_exited = true;
  for (int s = 0; s < rm.nseq; ++s) all_exited &= exited_s[s] != 0;
  if (all_exited && (n0 < nq || n0 >= 3 * nq)) return;

  XSrc xs{nullptr, L.attn_norm};
  const int mrow = lane & 15;
  if (mrow < rm.M) xs.row = ws.X + (size_t)src_s[mrow] * D.d;
  f32x4_t acc[1];
  gemv_wave<WB, 1>(wrow, xs, D.d, acc);
  gemv_reduce<1>(acc, rm.M, red, y);
  for (int e = threadIdx.x; e < rm.M * 16; e += kGemvThreads) {
    const int m = e >> 4, nn = n0 + (e & 15);
    if (nn < nqkv) ws.QKV[(size_t)m * nqkv + nn] = y[e] * inv_rms[m];
  }
}

// ============================================================================
// Kernel: attention with the shared KV cache.
// grid = (splits, H, nseq), block = 256.
// ============================================================================
constexpr int kAttnThreads = 256;
constexpr int kScoreCap = 4096;   // scores held in LDS per workgroup (rows x tokens)

// q, k or v (which = 0, 1, 2) of row m, head h, before RoPE: base projection
// plus, for fast rows, the adapter-up term.
__device__ __forceinline__ float proj_elem(const Dims& D, const LayerPtrs& L, const RowMap& rm, const WS& ws, int m,
                                           int which, int h, int d) {
  const int nqkv = 3 * D.qdim + 3 * D.r;
  const float* row = ws.QKV + (size_t)m * nqkv;
  const int c = h * D.hd + d;
  float v = row[which * D.qdim + c];
  if (rm.fast[m] && L.B[which] && L.A[which]) {
    const float* u = row + 3 * D.qdim + which * D.r;
    for (int j = 0; j < D.r; ++j) v += ld_w(L.B[which], (size_t)c * D.r + j, D.wbf16) * u[j];
  }
  return v;
}

// Fill out[R][hd] with q (which=0) or k (which=1) after RoPE, or v (which=2).
__device__ void head_vectors(const Dims& D, const LayerPtrs& L, const RowMap& rm, const WS& ws, const StepIO& io,
                             int first, int R, int which, int h, float* out) {
  const int hd = D.hd, half = hd / 2;
  for (int e = threadIdx.x; e < R * hd; e += kAttnThreads) {
    const int i = e / hd, d = e % hd;
    out[e] = proj_elem(D, L, rm, ws, first + i, which, h, d);
  }
  __syncthreads();
  if (which < 2) {
    for (int e = threadIdx.x; e < R * half; e += kAttnThreads) {
      const int i = e / half, j = e % half;
      const double pos = (double)row_pos(rm, io, first + i);
      const double ang = pos * pow((double)D.theta, -2.0 * j / hd);
      const float c = (float)cos(ang), s = (float)sin(ang);
      const float a = out[i * hd + j], b = out[i * hd + j + half];
      out[i * hd + j] = a * c - b * s;
      out[i * hd + j + half] = b * c + a * s;
    }
    __syncthreads();
  }
}

// Element index of (layer, sequence s, position pos, head h, dim d) in the
// pages [n_layers][num_blocks][H][bs][hd]; ok = false when the position is
// outside the sequence's block table or the block id is out of range.
__device__ __forceinline__ size_t kv_index(const KVPtrs& kv, const Dims& D, int layer, int s, int pos, int h, int d,
                                           bool& ok) {
  const int lb = pos / kv.bs;
  ok = pos >= 0 && lb < kv.mbps;
  const int blk = ok ? kv.bt[s * kv.mbps + lb] : 0;
  ok = ok && blk >= 0 && blk < kv.num_blocks;
  return ((((size_t)layer * kv.num_blocks + (ok ? blk : 0)) * D.H + h) * kv.bs + pos % kv.bs) * D.hd + d;
}

__device__ __forceinline__ float kv_load(const void* base, size_t i, int bf) {
  return bf ? bf16_to_f32(((const uint16_t*)base)[i]) : ((const float*)base)[i];
}
__device__ __forceinline__ float kv_round(float x, int bf) { return bf ? round_bf16(x) : x; }

template <int KB, int HD>
__device__ __forceinline__ void kv_row_load(const void* base, size_t ix, bool ok, float (&out)[HD / 4]) {
  constexpr int DPL = HD / 4;
  if constexpr (KB) {
#pragma unroll
    for (int c = 0; c < DPL; c += 8) {
      u32x4_t w = ok ? *(const u32x4_t*)((const uint16_t*)base + ix + c) : u32x4_t{0u, 0u, 0u, 0u};
#pragma unroll
      for (int i = 0; i < 4; ++i) { out[c + 2 * i] = bf16lo(w[i]); out[c + 2 * i + 1] = bf16hi(w[i]); }
    }
  } else {
#pragma unroll
    for (int c = 0; c < DPL; c += 4) {
      float4 w = ok ? *(const float4*)((const float*)base + ix + c) : make_float4(0.f, 0.f, 0.f, 0.f);
      out[c] = w.x; out[c + 1] = w.y; out[c + 2] = w.z; out[c + 3] = w.w;
    }
  }
}

constexpr size_t attn_smem_bytes() {
  return (size_t)(3 * kMaxRows * kMaxHeadDim + kScoreCap + 8 * kMaxHeadDim) * sizeof(float);
}

template <int KB, int HD>
__global__ __launch_bounds__(kAttnThreads) void k_attn(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, KVPtrs kv,
                                                       int layer, int n_split) {
  extern __shared__ float sm[];
  constexpr int DPL = HD / 4;             // dims per lane (4 lanes per token)
  const int split = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int hd = HD, R = rm.cnt[s], first = rm.first[s];
  const float scale = rsqrtf((float)hd);
  float* q = sm;                           // [R][hd]
  float* kx = q + kMaxRows * kMaxHeadDim;  // [R][hd]
  float* vx = kx + kMaxRows * kMaxHeadDim; // [R][hd]
  float* sc = vx + kMaxRows * kMaxHeadDim; // [R][per] scores, then probabilities
  float* redp = sc + kScoreCap;            // [4 waves][2 rows][hd]
  __shared__ float rowm[kMaxRows], rowl[kMaxRows];
  __shared__ int last_flag;

  const int ctx = io.positions[s] + rm.pos_offset;
  const bool frozen = ws.exited[s] != 0;

  // cache writes of this layer: rows flagged `wr` (slow rows; the fast row when drafting)
  if (split == 0) {
    bool any = false;
    for (int i = 0; i < R; ++i) any |= rm.wr[first + i] != 0;
    if (any) {
      head_vectors(D, L, rm, ws, io, first, R, 1, h, kx);
      head_vectors(D, L, rm, ws, io, first, R, 2, h, vx);
      for (int e = threadIdx.x; e < R * hd; e += kAttnThreads) {
        const int i = e / hd, d = e % hd;
        if (!rm.wr[first + i]) continue;
        bool ok;
        const size_t ix = kv_index(kv, D, layer, s, ctx + rm.idx[first + i], h, d, ok);
        if (!ok) { atomicOr(ws.err, 2); continue; }
        if (KB) {
          ((uint16_t*)kv.k)[ix] = (uint16_t)f32_to_bf16_bits(kx[e]);
          ((uint16_t*)kv.v)[ix] = (uint16_t)f32_to_bf16_bits(vx[e]);
        } else {
          ((float*)kv.k)[ix] = kx[e];
          ((float*)kv.v)[ix] = vx[e];
        }
      }
      __syncthreads();
    }
  }
  if (frozen) return;   // exited sequence: only its cache entries are produced

  head_vectors(D, L, rm, ws, io, first, R, 0, h, q);

  // ---- this split's share of the cached context [0, ctx) -------------------
  const int per = ((ctx + n_split - 1) / n_split + 15) & ~15;
  if (per * R > kScoreCap) {             // the host sizes splits so that this cannot happen
    if (threadIdx.x == 0) atomicOr(ws.err, 4);
    return;
  }
  const int t0 = min(ctx, split * per), t1 = min(ctx, t0 + per);
  const int nt = t1 - t0;
  const int sub = threadIdx.x & 3, slot = threadIdx.x >> 2;
  const int d0 = sub * DPL;
  for (int j = slot; j < nt; j += kAttnThreads / 4) {
    bool ok;
    const size_t base = kv_index(kv, D, layer, s, t0 + j, h, d0, ok);
    float kk[DPL];
    kv_row_load<KB, HD>(kv.k, base, ok, kk);
    for (int i = 0; i < R; ++i) {
      float p = 0.f;
#pragma unroll
      for (int c = 0; c < DPL; ++c) p += q[i * hd + d0 + c] * kk[c];
      p += __shfl_xor(p, 1);
      p += __shfl_xor(p, 2);
      if (sub == 0) sc[i * per + j] = p * scale;
    }
  }
  __syncthreads();
  {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int i = w; i < R; i += 4) {
      float mx = -INFINITY;
      for (int j = lane; j < nt; j += 64) mx = fmaxf(mx, sc[i * per + j]);
      mx = wave_max(mx);
      float l = 0.f;
      for (int j = lane; j < nt; j += 64) {
        const float e = __expf(sc[i * per + j] - mx);
        sc[i * per + j] = e;
        l += e;
      }
      l = wave_sum(l);
      if (lane == 0) { rowm[i] = mx; rowl[i] = l; }
    }
  }
  __syncthreads();
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  float* attp = ws.att + ((((size_t)s * D.H + h) * n_split + split) * kMaxRows) * (hd + 2);
  for (int i0 = 0; i0 < R; i0 += 2) {
    const bool two = i0 + 1 < R;
    float acc0[DPL], acc1[DPL];
#pragma unroll
    for (int c = 0; c < DPL; ++c) { acc0[c] = 0.f; acc1[c] = 0.f; }
    for (int j = slot; j < nt; j += kAttnThreads / 4) {
      bool ok;
      const size_t base = kv_index(kv, D, layer, s, t0 + j, h, d0, ok);
      float vv[DPL];
      kv_row_load<KB, HD>(kv.v, base, ok, vv);
      const float p0 = sc[i0 * per + j];
      const float p1 = two ? sc[(i0 + 1) * per + j] : 0.f;
#pragma unroll
      for (int c = 0; c < DPL; ++c) { acc0[c] += p0 * vv[c]; acc1[c] += p1 * vv[c]; }
    }
#pragma unroll
    for (int c = 0; c < DPL; ++c) {
      float a = acc0[c], b = acc1[c];
      a += __shfl_xor(a, 4); b += __shfl_xor(b, 4);
      a += __shfl_xor(a, 8); b += __shfl_xor(b, 8);
      a += __shfl_xor(a, 16); b += __shfl_xor(b, 16);
      a += __shfl_xor(a, 32); b += __shfl_xor(b, 32);
      acc0[c] = a; acc1[c] = b;
    }
    if (lane < 4) {
#pragma unroll
      for (int c = 0; c < DPL; ++c) {
        redp[(wv * 2 + 0) * hd + d0 + c] = acc0[c];
        redp[(wv * 2 + 1) * hd + d0 + c] = acc1[c];
      }
    }
    __syncthreads();
    for (int e = threadIdx.x; e < 2 * hd; e += kAttnThreads) {
      const int a = e / hd, d = e % hd;
      if (i0 + a < R) {
        float v = 0.f;
        for (int w = 0; w < 4; ++w) v += redp[(w * 2 + a) * hd + d];
        attp[(size_t)(i0 + a) * (hd + 2) + 2 + d] = v;
      }
    }
    __syncthreads();
  }
  for (int i = threadIdx.x; i < R; i += kAttnThreads) {
    attp[(size_t)i * (hd + 2)] = nt > 0 ? rowm[i] : -INFINITY;
    attp[(size_t)i * (hd + 2) + 1] = nt > 0 ? rowl[i] : 0.f;
  }

  // ---- the last split of this (sequence, head) merges ------------------------
  if (!arrive_last(ws.att_cnt + s * D.H + h, n_split, &last_flag)) return;

  head_vectors(D, L, rm, ws, io, first, R, 1, h, kx);
  head_vectors(D, L, rm, ws, io, first, R, 2, h, vx);
  // the rows' own keys: a slow row sees the chunk's slow rows up to itself (as
  // stored in the cache); a fast row sees only its own exact key/value.
  float* ownsc = sc;   // [R][R]
  for (int e = threadIdx.x; e < R * R; e += kAttnThreads) {
    const int i = e / R, jj = e % R;
    const int mi = first + i, mj = first + jj;
    bool vis;
    if (rm.fast[mi]) vis = (jj == i);
    else vis = !rm.fast[mj] && rm.idx[mj] <= rm.idx[mi];
    float p = -INFINITY;
    if (vis) {
      p = 0.f;
      const bool rnd = !rm.fast[mi];
      for (int d = 0; d < hd; ++d) {
        const float kk = rnd ? kv_round(kx[jj * hd + d], KB) : kx[jj * hd + d];
        p += q[i * hd + d] * kk;
      }
      p *= scale;
    }
    ownsc[e] = p;
  }
  __syncthreads();
  const float* att0 = ws.att + (((size_t)s * D.H + h) * n_split) * kMaxRows * (hd + 2);
  for (int e = threadIdx.x; e < R * hd; e += kAttnThreads) {
    const int i = e / hd, d = e % hd;
    const int mi = first + i;
    float M = -INFINITY;
    for (int sp = 0; sp < n_split; ++sp) {
      const float* pp = att0 + ((size_t)sp * kMaxRows + i) * (hd + 2);
      if (pp[1] > 0.f) M = fmaxf(M, pp[0]);
    }
    for (int jj = 0; jj < R; ++jj) M = fmaxf(M, ownsc[i * R + jj]);
    float Lsum = 0.f, o = 0.f;
    for (int sp = 0; sp < n_split; ++sp) {
      const float* pp = att0 + ((size_t)sp * kMaxRows + i) * (hd + 2);
      if (pp[1] > 0.f) {
        const float w = __expf(pp[0] - M);
        Lsum += w * pp[1];
        o += w * pp[2 + d];
      }
    }
    const bool rnd = !rm.fast[mi];
    for (int jj = 0; jj < R; ++jj) {
      const float sj = ownsc[i * R + jj];
      if (sj == -INFINITY) continue;
      const float w = __expf(sj - M);
      Lsum += w;
      o += w * (rnd ? kv_round(vx[jj * hd + d], KB) : vx[jj * hd + d]);
    }
    o /= Lsum;
    ws.O[(size_t)mi * D.qdim + h * hd + d] = o;
    q[e] = o;   // keep for the o adapter-down
  }
  __syncthreads();
  // adapter-down of the o projection for fast rows: u_o[h] = A_o[:, head cols] . o_h
  for (int e = threadIdx.x; e < R * D.r; e += kAttnThreads) {
    const int i = e / D.r, j = e % D.r;
    const int mi = first + i;
    float u = 0.f;
    if (rm.fast[mi] && L.A[3])
      for (int d = 0; d < hd; ++d) u += ld_w(L.A[3], (size_t)j * D.qdim + h * hd + d, D.wbf16) * q[i * hd + d];
    ws.uo[((size_t)mi * D.H + h) * D.r + j] = u;
  }
}

// ============================================================================
// Kernel: output projection + residual add (+ adapter on the fast row).
// grid = d/16 tiles, block = 512.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_oproj(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float uo_s[kMaxRows * kMaxRank];
  __shared__ float newx[256];
  const int n0 = blockIdx.x * 16;
  const int lane = threadIdx.x & 63;
  const size_t esz = WB ? 2 : 4;
  bool all_exited = true;
  for (int s = 0; s < rm.nseq; ++s) all_exited &= ws.exited[s] != 0;
  if (all_exited) return;
  const void* wrow[1] = {(const char*)L.wo + (size_t)(n0 + (lane & 15)) * D.qdim * esz};
  XSrc xs{nullptr, nullptr};
  if ((lane & 15) < rm.M) xs.row = ws.O + (size_t)(lane & 15) * D.qdim;
  f32x4_t acc[1];
  gemv_wave<WB, 1>(wrow, xs, D.qdim, acc);
  // adapter-down of o, summed over heads
  for (int e = threadIdx.x; e < rm.M * D.r; e += kGemvThreads) {
    const int m = e / D.r, j = e % D.r;
    float u = 0.f;
    if (rm.fast[m] && L.A[3])
      for (int hh = 0; hh < D.H; ++hh) u += ws.uo[((size_t)m * D.H + hh) * D.r + j];
    uo_s[e] = u;
  }
  gemv_reduce<1>(acc, rm.M, red, y);
  // epilogue: thread e -> (m, n) ; read everything first, write after a barrier
  const int e = threadIdx.x;
  const int m = e >> 4, nn = n0 + (e & 15);
  float xnew = 0.f, pin = 0.f;
  bool upd = false;
  if (e < rm.M * 16) {
    const int s = rm.seq[m];
    const bool ex = ws.exited[s] != 0;
    const float xo = ws.X[(size_t)m * D.d + nn];
    xnew = xo;
    if (!ex) {
      upd = true;
      if (rm.fast[m]) {
        const bool ri = ws.reinit[layer * kMaxSeq + s] != 0;
        pin = ri ? ws.X[(size_t)rm.slow_of[m] * D.d + nn] : xo;
        float ad = 0.f;
        if (L.B[3] && L.A[3])
          for (int j = 0; j < D.r; ++j) ad += ld_w(L.B[3], (size_t)nn * D.r + j, D.wbf16) * uo_s[m * D.r + j];
        xnew = pin + y[e] + ad;
      } else {
        xnew = xo + y[e];
      }
    }
    newx[e] = xnew;
  }
  __syncthreads();
  if (e < rm.M * 16) {
    if (upd) {
      ws.X[(size_t)m * D.d + nn] = xnew;
      if (rm.fast[m]) ws.PIN[(size_t)m * D.d + nn] = pin;
    }
  }
  // partial sums for the gate/up prologue: sum x^2 and the adapter-down of
  // gate and up (fast rows): sum_n A[j][n] g_mlp[n] x[n]
  const int PO = 1 + 2 * D.r;
  float* po = ws.part_o + ((size_t)blockIdx.x * kMaxRows) * PO;
  for (int q = threadIdx.x; q < rm.M * PO; q += kGemvThreads) {
    const int mm = q / PO, c = q % PO;
    float v = 0.f;
    if (c == 0) {
      for (int i = 0; i < 16; ++i) v += newx[mm * 16 + i] * newx[mm * 16 + i];
    } else if (rm.fast[mm]) {
      const int which = (c - 1) / D.r, j = (c - 1) % D.r;   // 0: gate (A[4]), 1: up (A[5])
      const void* A = L.A[4 + which];
      if (A)
        for (int i = 0; i < 16; ++i)
          v += ld_w(A, (size_t)j * D.d + n0 + i, D.wbf16) * L.mlp_norm[n0 + i] * newx[mm * 16 + i];
    }
    po[(size_t)mm * PO + c] = v;
  }
}

// ============================================================================
// Kernel: gate/up projections (paired tiles), adapter-up, SwiGLU.
// grid = F/16 tiles, block = 512.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_gateup(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io,
                                                         int n_part) {
  __shared__ float red[kGemvWaves * 512];
  __shared__ float y[512];
  __shared__ float stat[kMaxRows * (1 + 2 * kMaxRank)];
  __shared__ float inv_rms[kMaxRows];
  __shared__ float act[256];
  const int n0 = blockIdx.x * 16;
  const int lane = threadIdx.x & 63;
  const size_t esz = WB ? 2 : 4;
  bool all_exited = true;
  for (int s = 0; s < rm.nseq; ++s) all_exited &= ws.exited[s] != 0;
  if (all_exited) return;
  const int n = n0 + (lane & 15);
  const void* wrow[2] = {(const char*)L.wg + (size_t)n * D.d * esz, (const char*)L.wu + (size_t)n * D.d * esz};
  XSrc xs{nullptr, L.mlp_norm};
  if ((lane & 15) < rm.M) xs.row = ws.X + (size_t)(lane & 15) * D.d;
  f32x4_t acc[2];
  gemv_wave<WB, 2>(wrow, xs, D.d, acc);
  const int PO = 1 + 2 * D.r;
  for (int q = threadIdx.x; q < rm.M * PO; q += kGemvThreads) {
    const int mm = q / PO, c = q % PO;
    float v = 0.f;
    for (int t = 0; t < n_part; ++t) v += ws.part_o[((size_t)t * kMaxRows + mm) * PO + c];
    stat[q] = v;
  }
  __syncthreads();
  if (threadIdx.x < rm.M) inv_rms[threadIdx.x] = rsqrtf(stat[threadIdx.x * PO] / D.d + D.eps);
  gemv_reduce<2>(acc, rm.M, red, y);
  const int e = threadIdx.x;
  if (e < rm.M * 16) {
    const int m = e >> 4, nn = n0 + (e & 15);
    const float ir = inv_rms[m];
    float g = y[e] * ir, u = y[256 + e] * ir;
    if (rm.fast[m]) {
      if (L.B[4] && L.A[4])
        for (int j = 0; j < D.r; ++j) g += ld_w(L.B[4], (size_t)nn * D.r + j, D.wbf16) * stat[m * PO + 1 + j] * ir;
      if (L.B[5] && L.A[5])
        for (int j = 0; j < D.r; ++j)
          u += ld_w(L.B[5], (size_t)nn * D.r + j, D.wbf16) * stat[m * PO + 1 + D.r + j] * ir;
    }
    const float a = silu(g) * u;
    ws.ACT[(size_t)m * D.F + nn] = a;
    act[e] = a;
  }
  __syncthreads();
  // partials of the down adapter-down: sum_n A_d[j][n] a[n]
  float* pg = ws.part_gu + ((size_t)blockIdx.x * kMaxRows) * D.r;
  for (int q = threadIdx.x; q < rm.M * D.r; q += kGemvThreads) {
    const int mm = q / D.r, j = q % D.r;
    float v = 0.f;
    if (rm.fast[mm] && L.A[6])
      for (int i = 0; i < 16; ++i) v += ld_w(L.A[6], (size_t)j * D.F + n0 + i, D.wbf16) * act[mm * 16 + i];
    pg[(size_t)mm * D.r + j] = v;
  }
}

// ============================================================================
// Kernel: down projection + residual add (+ adapter), partial sums for the
// next layer's norm and the exit signal.  grid = d/16 tiles, block = 512.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_down(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int n_part) {
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float ud[kMaxRows * kMaxRank];
  __shared__ float newx[256], pin_s[256];
  const int n0 = blockIdx.x * 16;
  const int lane = threadIdx.x & 63;
  const size_t esz = WB ? 2 : 4;
  bool all_exited = true;
  for (int s = 0; s < rm.nseq; ++s) all_exited &= ws.exited[s] != 0;
  const int e = threadIdx.x;
  if (!all_exited) {
    const void* wrow[1] = {(const char*)L.wd + (size_t)(n0 + (lane & 15)) * D.F * esz};
    XSrc xs{nullptr, nullptr};
    if ((lane & 15) < rm.M) xs.row = ws.ACT + (size_t)(lane & 15) * D.F;
    f32x4_t acc[1];
    gemv_wave<WB, 1>(wrow, xs, D.F, acc);
    for (int q = threadIdx.x; q < rm.M * D.r; q += kGemvThreads) {
      const int m = q / D.r, j = q % D.r;
      float u = 0.f;
      if (rm.fast[m] && L.A[6])
        for (int t = 0; t < n_part; ++t) u += ws.part_gu[((size_t)t * kMaxRows + m) * D.r + j];
      ud[q] = u;
    }
    gemv_reduce<1>(acc, rm.M, red, y);
  }
  if (e < rm.M * 16) {
    const int m = e >> 4, nn = n0 + (e & 15);
    const int s = rm.seq[m];
    const bool ex = ws.exited[s] != 0;
    float x = ws.X[(size_t)m * D.d + nn];
    if (!ex) {
      x += y[e];
      if (rm.fast[m] && L.B[6] && L.A[6])
        for (int j = 0; j < D.r; ++j) x += ld_w(L.B[6], (size_t)nn * D.r + j, D.wbf16) * ud[m * D.r + j];
      ws.X[(size_t)m * D.d + nn] = x;
    }
    newx[e] = x;
    pin_s[e] = rm.fast[m] ? ws.PIN[(size_t)m * D.d + nn] : 0.f;
  }
  __syncthreads();
  float* pd = ws.part_d + ((size_t)blockIdx.x * kMaxRows) * 4;
  for (int q = threadIdx.x; q < rm.M * 4; q += kGemvThreads) {
    const int mm = q >> 2, c = q & 3;
    float v = 0.f;
    for (int i = 0; i < 16; ++i) {
      const float x = newx[mm * 16 + i], p = pin_s[mm * 16 + i];
      v += c == 0 ? x * x : (c == 1 ? p * x : (c == 2 ? p * p : 0.f));
    }
    pd[q] = v;
  }
}

// ============================================================================
// Kernel: final norm + LM head + argmax; the last workgroup finishes the step
// (tokens, exit bookkeeping, acceptance of a verified chunk).
// grid = V/16 tiles, block = 512.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kGemvThreads) void k_head(Dims D, const void* lm_head, const float* final_norm, RowMap rm,
                                                       WS ws, StepIO io, KVPtrs kv, int n_part, int n_tiles) {
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int hrow[kMaxRows];
  __shared__ int nh_s;
  __shared__ float inv_rms[kMaxRows];
  __shared__ int last_flag;
  const int n0 = blockIdx.x * 16;
  const int lane = threadIdx.x & 63;
  const size_t esz = WB ? 2 : 4;
  const int nrow = min(n0 + (lane & 15), D.V - 1);
  const void* wrow[1] = {(const char*)lm_head + (size_t)nrow * D.d * esz};
  for (int q = threadIdx.x; q < rm.M * 4; q += kGemvThreads) {
    float v = 0.f;
    for (int t = 0; t < n_part; ++t) v += ws.part_d[((size_t)t * kMaxRows) * 4 + q];
    ssum[q] = v;
  }
  if (threadIdx.x == 0) {
    // rows fed to the head
    int nh = 0;
    if (rm.head_all) {
      for (int m = 0; m < rm.M; ++m) hrow[nh++] = m;
    } else {
      for (int s = 0; s < rm.nseq; ++s) {
        const int f = rm.first[s], c = rm.cnt[s];
        int pick = f;                       // slow row
        if (rm.fast[f + c - 1] && (ws.exited[s] || rm.slow_of[f + c - 1] < 0)) pick = f + c - 1;
        hrow[nh++] = pick;
      }
    }
    nh_s = nh;
  }
  __syncthreads();
  if (threadIdx.x < nh_s) inv_rms[threadIdx.x] = rsqrtf(ssum[hrow[threadIdx.x] * 4] / D.d + D.eps);
  const int nh = nh_s;
  XSrc xs{nullptr, final_norm};
  if ((lane & 15) < nh) xs.row = ws.X + (size_t)hrow[lane & 15] * D.d;
  f32x4_t acc[1];
  gemv_wave<WB, 1>(wrow, xs, D.d, acc);
  gemv_reduce<1>(acc, nh, red, y);
  // logits and per-tile argmax (lowest index on ties)
  const int e = threadIdx.x;
  if (e < nh * 16) {
    const int k = e >> 4, nn = n0 + (e & 15);
    float z = y[e] * inv_rms[k];
    if (nn >= D.V) z = -INFINITY;
    else if (io.logits_out) io.logits_out[(size_t)k * D.V + nn] = z;
    int idx = nn;
    // reduce over the 16 consecutive lanes holding this row's tile
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      const float z2 = __shfl_xor(z, o);
      const int i2 = __shfl_xor(idx, o);
      if (z2 > z || (z2 == z && i2 < idx)) { z = z2; idx = i2; }
    }
    if ((e & 15) == 0) {
      ws.lm_val[(size_t)blockIdx.x * kMaxRows + k] = z;
      ws.lm_idx[(size_t)blockIdx.x * kMaxRows + k] = idx;
    }
  }
  if (!arrive_last(ws.lm_cnt, n_tiles, &last_flag)) return;

  // ---- last workgroup: global argmax per head row, then bookkeeping ----------
  __shared__ int best_s[kMaxRows];
  const int wave = threadIdx.x >> 6;
  for (int k = wave; k < nh; k += kGemvWaves) {
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int t = lane; t < n_tiles; t += 64) {
      const float z = ws.lm_val[(size_t)t * kMaxRows + k];
      const int i = ws.lm_idx[(size_t)t * kMaxRows + k];
      if (z > bz || (z == bz && i < bi)) { bz = z; bi = i; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float z2 = __shfl_xor(bz, o);
      const int i2 = __shfl_xor(bi, o);
      if (z2 > bz || (z2 == bz && i2 < bi)) { bz = z2; bi = i2; }
    }
    if (lane == 0) best_s[k] = bi;
  }
  __syncthreads();
  if (rm.head_all) {
    // chunk verification / prefill (one sequence)
    if (threadIdx.x == 0) {
      const int t = io.positions[0];
      for (int k = 0; k < nh; ++k) io.targets[k] = best_s[k];
      int keep = nh;
      if (io.n_acc) {
        int j = 0;
        while (j < nh - 1 && io.tokens[j + 1] == best_s[j]) ++j;
        io.n_acc[0] = j;
        if (io.bonus) io.bonus[0] = best_s[j];
        keep = j + 1;
      }
      kv.seq_lens[0] = t + keep;
      io.positions[0] = t + keep;
    }
    return;
  }
  // decode step / draft step
  for (int s = threadIdx.x; s < rm.nseq; s += kGemvThreads) {
    const int f = rm.first[s] + rm.cnt[s] - 1;
    io.next_token[s + io.draft_slot] = best_s[s];
    const int t = io.positions[s] + rm.pos_offset;
    if (rm.slow_of[f] >= 0 || !rm.fast[f]) kv.seq_lens[s] = t + 1;
    if (rm.fast[f] && rm.slow_of[f] >= 0) {
      // signal of the last layer
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      ws.sig[s * D.n_layers + D.n_layers - 1] = ws.exited[s] ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
    }
    if (io.exit_b_out) io.exit_b_out[s] = ws.exitb[s];
    if (io.advance) io.positions[s] = io.positions[s] + 1;
  }
  __syncthreads();
  if (io.signal_out) {
    for (int q = threadIdx.x; q < rm.nseq * D.n_layers; q += kGemvThreads) {
      const int s = q / D.n_layers, l = q % D.n_layers;
      const int f = rm.first[s] + rm.cnt[s] - 1;
      float v = ws.sig[q];
      // layers after an exit were not run
      if (!rm.fast[f] || rm.slow_of[f] < 0 || (ws.exited[s] && l >= ws.exitb[s])) v = 0.f;
      io.signal_out[q] = v;
    }
  }
  if (io.h_out || io.p_out) {
    for (int q = threadIdx.x; q < rm.nseq * D.d; q += kGemvThreads) {
      const int s = q / D.d, i = q % D.d;
      const int f = rm.first[s], c = rm.cnt[s];
      if (io.h_out) io.h_out[q] = ws.X[(size_t)f * D.d + i];
      if (io.p_out) io.p_out[q] = ws.X[(size_t)(f + c - 1) * D.d + i];
    }
  }
}

}  // namespace m2r2
