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
  // FLOPs-optimised fast stream (Sec. 2.5; all zero: the memory-bound form):
  // fast heads kept, positions each attends to, adapter-only fast MLP, rank
  // of the fast row's head
  int fh, ftk, fmlp, hr;
};

// Projection matrices are read from a tile-packed copy (pack_index below):
// pq/pk/pv/pa (q, k, v and the stacked adapter-down rows [A_q; A_k; A_v],
// consecutive in memory), po, pg (gate and up as interleaved tile pairs; pu
// is unused), pd.  Adapter factors and norms stay row-major.
struct LayerPtrs {
  const float* attn_norm;
  const float* mlp_norm;
  const void *pq, *pk, *pv, *pa, *po, *pg, *pu, *pd;
  const void *wq, *wk, *wv, *wo, *wg, *wu, *wd;   // the caller's row-major matrices
  const void* A[7];
  const void* B[7];
};

// Tile-packed weight layout.  A [rows][K] matrix is stored as 16-row tiles;
// within a tile, K is cut into MFMA steps (32 bf16 or 16 f32 elements) and
// each step is one 1 KB block holding, for lane l of a wave, the 16 bytes
// row (l % 16), elements [step*KSTEP + EPL*(l/16), +EPL) -- exactly the B
// operand of one MFMA, so each wave load is 1 KB contiguous.  Rows past the
// end of the matrix are zero.
__host__ __device__ constexpr size_t packed_bytes(int rows, int K, int wb) {
  return (size_t)((rows + 15) / 16) * 16 * K * (wb ? 2 : 4);
}

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
  // Row statistics and adapter-down projections are sums over a whole row,
  // which the producing kernel holds in 16-row tiles.  Each workgroup adds its
  // tile's share with float atomics into one of kBins bins of the layer; the
  // consumer (the next kernel) sums the kBins bins.  Bins are zeroed by the
  // embedding kernel at the start of every pass.
  float* bin_d;    // [n_layers+1][kBins][16][4]   sum x^2, sum pin*x, sum pin^2 (entering layer l)
  float* bin_o;    // [n_layers][kBins][16][1+2r]  sum x^2, adapter-down of gate and up
  float* bin_gu;   // [n_layers][kBins][16][r]     adapter-down of down
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
  float* arla_kv;  // [n_layers][2][64] latent keys and values of the fast states (exit router)
  float* arla_q;   // [64] latent query at a gate
  float* arla_sig; // [16] router score of the last gate
  uint32_t* arla_cnt;   // arrival counter of the router kernel
  const float2* rope;  // [rope_len][hd/2] (cos, sin), built in double precision on the host
  int rope_len;
  // FLOPs-optimised fast stream (one sequence)
  float* fsc;      // [fast heads][rope_len] scaled slow-row scores of the cached positions
  float* fqkv;     // [fast heads][3][hd] the fast row's q, k (after RoPE) and v
  float* lrz;      // [head_rank] low-rank head: the emitted row times head_a
};

// Bins per layer and row: kBinSlots are stored (and zeroed every pass); the
// per-tile kernels use the first kBins, the stream-K and row-per-wave kernels
// spread their atomics over all kBinSlots (a workgroup adds into slot
// blockIdx % kBinSlots).  Every consumer workgroup reads all slots, so the
// count trades atomic contention against the bytes each consumer stages:
// 16 (64 made the gate/up staging 1.2 us longer, 8 was no faster).
constexpr int kBins = 8;
constexpr int kBinSlots = 16;

__device__ __forceinline__ float* bin_d_at(const WS& ws, int l, int b, int m) { return ws.bin_d + (((size_t)l * kBinSlots + b) * kMaxRows + m) * 4; }
__device__ __forceinline__ float* bin_o_at(const WS& ws, const Dims& D, int l, int b, int m) {
  return ws.bin_o + (((size_t)l * kBinSlots + b) * kMaxRows + m) * (1 + 2 * D.r);
}
__device__ __forceinline__ float* bin_gu_at(const WS& ws, const Dims& D, int l, int b, int m) {
  return ws.bin_gu + (((size_t)l * kBinSlots + b) * kMaxRows + m) * D.r;
}
__device__ __forceinline__ void add_agent(float* p, float v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

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
  // latent-attention exit router: score of the gate just passed, written by
  // the router kernel after the layer before the gate (null: cosine signal)
  const float* arla_sig;
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
// dimension into contiguous ranges.  A wave walks its range in chunks of 8
// K-steps: the weight pieces of the next chunk are already in flight (16-byte
// non-temporal loads, one weight row per lane group) while the activations of
// the current chunk (up to 16 rows, times the norm gain when there is one) are
// copied from global memory into the wave's own LDS region in MFMA fragment
// order.  bf16 weights: v_mfma_f32_16x16x32_bf16 with each fp32 activation
// split into bf16 hi + lo parts (two MFMAs, 16 significant bits of the
// activation).  f32 weights: four v_mfma_f32_16x16x4_f32 per 16-byte piece
// (exact fp32 products).  Accumulation is fp32; the 8 per-wave results are
// summed through LDS (gemv_reduce).
// ============================================================================
constexpr int kGemvWaves = 8;
constexpr int kGemvThreads = kGemvWaves * 64;
constexpr int kChunk = 8;   // K-steps per chunk

// Dynamic LDS bytes of the activation staging for the row class MT.
__host__ __device__ constexpr int gemv_lds_bytes(int wb, int MT) {
  return kGemvWaves * MT * kChunk * (wb ? 32 * 4 : 16 * 4);
}

// 16-byte load through a global-address-space pointer (no flat access).
typedef float f32x4v_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float4 ldg4(const float* p) {
  const f32x4v_t v = *(const __attribute__((address_space(1))) f32x4v_t*)(p);
  return make_float4(v.x, v.y, v.z, v.w);
}

// MT: row-count class (2 or 16) the code is unrolled for; M <= MT rows are live.
// GAIN: activations are multiplied by a per-k gain while staged.
template <int WB, int NT, int MT, bool GAIN>
struct GemvWave {
  static constexpr int KSTEP = WB ? 32 : 16;   // K per MFMA step
  static constexpr int P = KSTEP / 4;          // float4 pieces per step and row
  u32x4_t w[NT][kChunk];
  const char* base[NT];   // this lane's 16 bytes of step 0 of each tile
  int s0, s1;
  // segmented reduction (NT == 1): steps [k*seg_steps, (k+1)*seg_steps) come
  // from the tile at seg[k] (the K experts of a mixture-of-experts layer)
  const char* const* seg = nullptr;
  int seg_steps = 0;

  __device__ __forceinline__ const char* step_ptr(int t, int sj) const {
    if (seg_steps) return seg[sj / seg_steps] + (size_t)(sj % seg_steps) * 1024 + (threadIdx.x & 63) * 16;
    return base[t] + (size_t)sj * 1024;
  }
  __device__ __forceinline__ u32x4_t ld_step(int t, int sj) const {
    // global-address-space load (the segment pointers come from LDS)
    return __builtin_nontemporal_load((const __attribute__((address_space(1))) u32x4_t*)step_ptr(t, sj));
  }

  __device__ __forceinline__ void load(int sb, u32x4_t (&dst)[NT][kChunk]) const {
#pragma unroll
    for (int j = 0; j < kChunk; ++j) {
      const int sj = min(sb + j, s1 - 1);   // steps past the range repeat a valid address; never used
#pragma unroll
      for (int t = 0; t < NT; ++t) dst[t][j] = ld_step(t, sj);
    }
  }

  // tile[t]: packed tile of NT.  Split the K steps over the waves and put the
  // first chunk's loads in flight.
  __device__ __forceinline__ void begin(const void* const (&tile)[NT], int K) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int nsteps = K / KSTEP;
    const int per = (nsteps + kGemvWaves - 1) / kGemvWaves;
    s0 = min(nsteps, wave * per);
    s1 = min(nsteps, s0 + per);
#pragma unroll
    for (int t = 0; t < NT; ++t) base[t] = (const char*)tile[t] + lane * 16;
    load(s0, w);   // unconditional: clamped addresses are valid even for an empty range
  }

  // One chunk: activations of steps [sb, sb+kChunk) are loaded, then the
  // weights of the following chunk are put in flight (into wnext), then the
  // activations are staged in MFMA fragment order and the MFMAs consume wcur.
  // Scheduling barriers keep that order so that waiting for the activations
  // never waits for the prefetched weights.  All MT row slots are staged (rows
  // >= M repeat row 0 and only feed output rows that are discarded); steps
  // past the range are staged as zeros (they add 0 x repeated weights).
  __device__ __forceinline__ void chunk(int sb, const float* const (&xr)[MT], const float* gain, char* my,
                                        const u32x4_t (&wcur)[NT][kChunk], u32x4_t (&wnext)[NT][kChunk],
                                        f32x4_t (&acc)[NT]) const {
    const int lane = threadIdx.x & 63;
    const int mr = lane & 15, grp = lane >> 4;
    const int q = WB ? lane : (lane & 31);       // float4 piece of the chunk this lane stages
    const int mread = mr < MT ? mr : MT - 1;
    const int nst = min(kChunk, s1 - sb);
    const bool live = q < nst * P;
    const int kq = sb * KSTEP + 4 * (live ? q : 0);
    float4 xv[MT];
    float4 gv = make_float4(1.f, 1.f, 1.f, 1.f);
    if constexpr (GAIN) gv = ldg4(gain + kq);
#pragma unroll
    for (int m = 0; m < MT; ++m) xv[m] = ldg4(xr[m] + kq);
    __builtin_amdgcn_sched_barrier(0);
    load(sb + kChunk, wnext);
    __builtin_amdgcn_sched_barrier(0);
    const int j = q / P, e = (q % P) * 4;
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      float4 v = xv[m];
      v.x = live ? v.x * gv.x : 0.f;
      v.y = live ? v.y * gv.y : 0.f;
      v.z = live ? v.z * gv.z : 0.f;
      v.w = live ? v.w * gv.w : 0.f;
      if constexpr (WB) {
        uint16_t* hi = (uint16_t*)my;
        uint16_t* lo = hi + kChunk * MT * 32;
        const float xs[4] = {v.x, v.y, v.z, v.w};
        uint32_t h[4], l[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          h[i] = f32_to_bf16_bits(xs[i]);
          l[i] = f32_to_bf16_bits(xs[i] - __uint_as_float(h[i] << 16));
        }
        const int o = (j * MT + m) * 32 + e;
        *(uint2*)(hi + o) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
        *(uint2*)(lo + o) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
      } else {
        *(float4*)((float*)my + (j * MT + m) * 16 + e) = v;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int jj = 0; jj < kChunk; ++jj) {
      if constexpr (WB) {
        const uint16_t* hi = (const uint16_t*)my;
        const uint16_t* lo = hi + kChunk * MT * 32;
        const int o = (jj * MT + mread) * 32 + 8 * grp;
        const bf16x8_t a_hi = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(hi + o));
        const bf16x8_t a_lo = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(lo + o));
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          const bf16x8_t bw = __builtin_bit_cast(bf16x8_t, wcur[t][jj]);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_hi, bw, acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_lo, bw, acc[t], 0, 0, 0);
        }
      } else {
        const float4 a = *(const float4*)((const float*)my + (jj * MT + mread) * 16 + 4 * grp);
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, __uint_as_float(wcur[t][jj][0]), acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, __uint_as_float(wcur[t][jj][1]), acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, __uint_as_float(wcur[t][jj][2]), acc[t], 0, 0, 0);
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, __uint_as_float(wcur[t][jj][3]), acc[t], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_wave_barrier();
  }

  // Run the wave's K range.  xrow: M activation row pointers (LDS array);
  // lds: the workgroup's dynamic staging area (gemv_lds_bytes(WB, MT)).
  __device__ __forceinline__ void run(const float* const* xrow, const float* gain, int M, char* lds,
                                      f32x4_t (&acc)[NT]) {
    const int wave = threadIdx.x >> 6;
    char* my = lds + wave * (MT * kChunk * KSTEP * 4);
    const float* xr[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) xr[m] = xrow[m < M ? m : 0];
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    u32x4_t w2[NT][kChunk];
    for (int sb = s0; sb < s1; sb += 2 * kChunk) {
      chunk(sb, xr, gain, my, w, w2, acc);
      if (sb + kChunk >= s1) break;
      chunk(sb + kChunk, xr, gain, my, w2, w, acc);
    }
  }
};

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


// ============================================================================
// Persistent tile GEMV.
//
// A launch has at most as many workgroups as the GPU holds at once; each
// workgroup walks the tiles blockIdx.x, blockIdx.x + gridDim.x, ... (a tile is
// 16 weight rows).  Its 8 waves split every tile's K-steps into the same
// contiguous ranges and stream them in chunks of 8 one-kilobyte blocks, one
// continuous sequence over all of the workgroup's tiles: the next chunk --
// possibly the first of the next tile -- is in flight while the current one
// is multiplied, so the LDS reduction and epilogue of one tile overlap the
// next tile's loads.  Per-wave partial sums are added through LDS (gemv_reduce) in
// a fixed order and the epilogue runs workgroup-wide.
//
// Activations: for the 2-row class the input rows (times the norm gain) are
// staged once in LDS in MFMA fragment order, each wave its own K range -- bf16 weights:
// hi and lo bf16 planes [step][row][32] (two MFMAs, 16 significant bits of the
// activation); f32 weights: [step][row][16] -- so the stream loop only loads
// weights and reads fragments from LDS.  The 16-row class stages each chunk's
// activations in the wave's own LDS region as it goes.
// ============================================================================
__device__ __forceinline__ u32x4_t ld_glob(const char* p) {
  return __builtin_nontemporal_load((const __attribute__((address_space(1))) u32x4_t*)p);
}

// Dynamic LDS of a tile GEMV launch with reduction length K.
__host__ __device__ constexpr int tile_lds_bytes(int wb, int MT, int K) {
  return MT <= 2 ? MT * K * 4 : kGemvWaves * MT * (MT <= 8 ? kChunk : kChunk / 2) * (wb ? 32 : 16) * 4;
}

template <int WB, int MT, int BS = 1024>
struct TileGemv {
  static constexpr int KSTEP = WB ? 32 : 16;
  static constexpr int P = KSTEP / 4;
  static constexpr bool XRES = MT <= 2;
  // the next chunk's activations are requested one chunk ahead; 16 rows take
  // chunks of half as many K-steps so that they fit the registers
  static constexpr bool XPIPE = !XRES;
  static constexpr int KC = MT <= 8 ? kChunk : kChunk / 2;   // K-steps per chunk
  static constexpr int PPR = KC * P;                          // float4 pieces of one row in a chunk
  static constexpr int RP = 64 / PPR;                         // rows one pass of the lanes covers
  static constexpr int NX = (MT + RP - 1) / RP;               // activation pieces per lane
  static_assert(64 % PPR == 0 && MT % RP == 0, "chunk pieces tile the wave");
  u32x4_t w[KC], w2[KC];
  int nsteps, s0, s1, nchunks;
  char* xl;                   // LDS: resident rows (XRES) or per-wave chunk staging
  const float* xr[MT];        // activation rows (16-row class)
  const float* gain;
  float4 xa[NX];              // activations of the chunk to stage next (not resident)
  float4 ga;                  // and its gain (row 0 again without a gain: never used)
  bool xfetched = false;      // the first chunk's activations were requested before the prime

  __device__ __forceinline__ void init(int K, char* lds) {
    const int wave = threadIdx.x >> 6;
    nsteps = K / KSTEP;
    const int per = (nsteps + kGemvWaves - 1) / kGemvWaves;
    s0 = min(nsteps, wave * per);
    s1 = min(nsteps, s0 + per);
    nchunks = (s1 - s0 + KC - 1) / KC;
    xl = XRES ? lds : lds + wave * (MT * KC * KSTEP * 4);
  }

  // blocks sb.. of the tile at `base` (this lane's 16 bytes); blocks past the
  // wave's range repeat its last block (a cache hit, never used)
  __device__ __forceinline__ void load(const char* base, int sb, u32x4_t (&dst)[KC]) const {
#pragma unroll
    for (int j = 0; j < KC; ++j) dst[j] = ld_glob(base + (size_t)max(min(sb + j, s1 - 1), 0) * BS);
  }

  // The first two chunks of the workgroup's chunk sequence (tile i starts at
  // ptr(i)), put in flight before the kernel's prologue.
  template <class Ptr>
  // Unconditional (a wave without steps loads the tile's last block, never
  // used): the loads issued before it are then waited for by count, never
  // behind these.  The launching kernels guarantee n_local >= 1.
  __device__ __forceinline__ void prime(int n_local, const Ptr& ptr) {
    const int lo16 = (threadIdx.x & 63) * 16;
    // second chunk: in the first tile, else the next tile, else repeats of the last block
    const bool next_tile = nchunks == 1 && n_local > 1;
    const char* b2 = next_tile ? ptr(1) : ptr(0);
    const int sb2 = nchunks > 1 ? s0 + KC : (next_tile ? s0 : s1);
    load(ptr(0) + lo16, s0, w);
    load(b2 + lo16, sb2, w2);
  }

  // Activation rows (rows >= M repeat row 0), multiplied by `gn` when given.
  // Resident class: every wave stages the steps of its own K range now (the
  // LDS layout is indexed by step, the ranges are disjoint, and a wave reads
  // only its own steps, so no workgroup barrier is needed).
  __device__ __forceinline__ void set_rows(const float* const* xrow, const float* gn, int M, int K) {
#pragma unroll
    for (int m = 0; m < MT; ++m) xr[m] = xrow[m < M ? m : 0];
    gain = gn;
    if constexpr (XRES) {
      const int lane = threadIdx.x & 63;
      const int per_step = MT * P;   // float4 pieces of one step (all rows)
      for (int i = lane; i < (s1 - s0) * per_step; i += 64) {
        const int st = s0 + i / per_step, rem = i % per_step;
        const int m = rem / P, e = (rem % P) * 4;
        const int k = st * KSTEP + e;
        float4 v = ldg4(xrow[m < M ? m : 0] + k);   // (a runtime index into xr[] would put this object in scratch)
        if (gn) {
          const float4 g = ldg4(gn + k);
          v.x *= g.x; v.y *= g.y; v.z *= g.z; v.w *= g.w;
        }
        if constexpr (WB) {
          uint16_t* hi = (uint16_t*)xl;
          uint16_t* lo = hi + nsteps * MT * 32;
          const float xs[4] = {v.x, v.y, v.z, v.w};
          uint32_t h[4], l[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            h[q] = f32_to_bf16_bits(xs[q]);
            l[q] = f32_to_bf16_bits(xs[q] - __uint_as_float(h[q] << 16));
          }
          const int o = (st * MT + m) * 32 + e;
          *(uint2*)(hi + o) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
          *(uint2*)(lo + o) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
        } else {
          *(float4*)((float*)xl + (st * MT + m) * 16 + e) = v;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
  }

  // ---- resident rows in two halves (2-row class) ---------------------------
  // Loads are waited for in issue order, so anything a kernel needs before
  // its weights arrive must be issued before prime().  load_pieces issues this
  // wave's activation pieces of the candidate rows (and the gain) into
  // registers; store_pieces stages them into LDS after prime(), row m taken
  // from candidate sel[m].  Pieces past PM per lane (very long reductions) are
  // loaded and staged by store_pieces itself.
  template <int PM>
  struct Pieces {
    float4 v[PM][MT];
    float4 g[PM];
  };

  template <int PM>
  __device__ __forceinline__ void load_pieces(const float* const (&rows)[MT], const float* gn, Pieces<PM>& xp) const {
    const int lane = threadIdx.x & 63;
    const int npc = (s1 - s0) * P;
#pragma unroll
    for (int p = 0; p < PM; ++p) {
      const int q = lane + 64 * p;
      const int k = (s0 < s1 ? s0 * KSTEP : 0) + 4 * (q < npc ? q : 0);
#pragma unroll
      for (int m = 0; m < MT; ++m) xp.v[p][m] = ldg4(rows[m] + k);
      xp.g[p] = ldg4((gn ? gn : rows[0]) + k);   // unconditional (ignored without a gain)
    }
  }

  __device__ __forceinline__ void put_piece(int k, int m, float4 v) const {
    const int st = k / KSTEP, e = k - st * KSTEP;
    if constexpr (WB) {
      uint16_t* hi = (uint16_t*)xl;
      uint16_t* lo = hi + nsteps * MT * 32;
      const float xs[4] = {v.x, v.y, v.z, v.w};
      uint32_t h[4], l[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        h[q] = f32_to_bf16_bits(xs[q]);
        l[q] = f32_to_bf16_bits(xs[q] - __uint_as_float(h[q] << 16));
      }
      const int o = (st * MT + m) * 32 + e;
      *(uint2*)(hi + o) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
      *(uint2*)(lo + o) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
    } else {
      *(float4*)((float*)xl + (st * MT + m) * 16 + e) = v;
    }
  }

  template <int PM>
  __device__ __forceinline__ void store_pieces(const Pieces<PM>& xp, const float* const (&rows)[MT], const float* gn,
                                               const int (&sel)[MT]) {
    const int lane = threadIdx.x & 63;
    const int npc = (s1 - s0) * P;
#pragma unroll
    for (int p = 0; p < PM; ++p) {
      const int q = lane + 64 * p;
      if (q < npc) {
        const int k = s0 * KSTEP + 4 * q;
#pragma unroll
        for (int m = 0; m < MT; ++m) {
          float4 v = xp.v[p][0];
#pragma unroll
          for (int c = 1; c < MT; ++c)
            if (sel[m] == c) v = xp.v[p][c];
          if (gn) {
            const float4 g = xp.g[p];
            v.x *= g.x; v.y *= g.y; v.z *= g.z; v.w *= g.w;
          }
          put_piece(k, m, v);
        }
      }
    }
    for (int q = lane + 64 * PM; q < npc; q += 64) {
      const int k = s0 * KSTEP + 4 * q;
      const float4 g = gn ? ldg4(gn + k) : make_float4(1.f, 1.f, 1.f, 1.f);
#pragma unroll
      for (int m = 0; m < MT; ++m) {
        float4 v = ldg4(rows[0] + k);
#pragma unroll
        for (int c = 1; c < MT; ++c)
          if (sel[m] == c) v = ldg4(rows[c] + k);
        v.x *= g.x; v.y *= g.y; v.z *= g.z; v.w *= g.w;
        put_piece(k, m, v);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // Not resident, rows known at kernel start: the rows (rows >= M repeat a
  // live row) and the first chunk's activations, requested before the
  // weights are primed so that waiting for them never waits for the weights.
  __device__ __forceinline__ void early_rows(const float* const (&rows)[MT], const float* gn) {
#pragma unroll
    for (int m = 0; m < MT; ++m) xr[m] = rows[m];
    gain = gn;
    fetch_x(s0);
    xfetched = true;
  }

  // 16-row class: request the activations (and gains) of the chunk at steps
  // sb.. into xa / ga.  Unconditional loads at clamped addresses.
  __device__ __forceinline__ void fetch_x(int sb) {
    const int lane = threadIdx.x & 63;
    const int q = lane % PPR, r0 = lane / PPR;   // piece q of rows r0, r0 + RP, ...
    const bool live = q < min(KC, s1 - sb) * P;
    const int kq = sb * KSTEP + 4 * (live ? q : 0);
    ga = ldg4((gain ? gain : xr[0]) + kq);
#pragma unroll
    for (int j = 0; j < NX; ++j) {
      // a select over opaque values (a select over the array's elements would
      // become a runtime index into xr[], i.e. scratch memory)
      const float* rp = xr[j * RP];
      asm volatile("" : "+v"(rp));
#pragma unroll
      for (int c = 1; c < RP; ++c) {
        const float* pc = xr[j * RP + c];
        asm volatile("" : "+v"(pc));
        if (r0 == c) rp = pc;
      }
      xa[j] = ldg4(rp + kq);
    }
  }

  // One chunk of steps [sb, sb+8) ∩ [.., s1): the MFMAs consume buf, then buf
  // is refilled with the chunk two ahead (nbase, nsb), so two chunks are in
  // flight while the wave multiplies.  16-row class: the chunk's activations
  // were requested one chunk earlier (xa); once they are staged, those of the
  // next chunk (steps xsb..) are requested before the weights two ahead, so
  // that waiting for them never waits for weights that are not yet needed.
  __device__ __forceinline__ void chunk(int sb, const char* nbase, int nsb, u32x4_t (&buf)[KC], f32x4_t& acc,
                                        int xsb) {
    const int lane = threadIdx.x & 63;
    const int mr = lane & 15, grp = lane >> 4;
    const int mread = mr < MT ? mr : MT - 1;
    const int nst = min(KC, s1 - sb);
    if constexpr (XRES) {
#pragma unroll
      for (int jj = 0; jj < KC; ++jj) {
        const int st = min(sb + jj, nsteps - 1);
        const bool on = jj < nst;
        if constexpr (WB) {
          const uint16_t* hi = (const uint16_t*)xl;
          const uint16_t* lo = hi + nsteps * MT * 32;
          const int o = (st * MT + mread) * 32 + 8 * grp;
          u32x4_t h = *(const u32x4_t*)(hi + o), l = *(const u32x4_t*)(lo + o);
          if (!on) { h = u32x4_t{0u, 0u, 0u, 0u}; l = h; }
          const bf16x8_t bw = __builtin_bit_cast(bf16x8_t, buf[jj]);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, h), bw, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, l), bw, acc, 0, 0, 0);
        } else {
          float4 a = *(const float4*)((const float*)xl + (st * MT + mread) * 16 + 4 * grp);
          if (!on) a = make_float4(0.f, 0.f, 0.f, 0.f);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, __uint_as_float(buf[jj][0]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, __uint_as_float(buf[jj][1]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, __uint_as_float(buf[jj][2]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, __uint_as_float(buf[jj][3]), acc, 0, 0, 0);
        }
      }
    } else {
      // stage this chunk's activations (requested one chunk earlier)
      const int q = lane % PPR, r0 = lane / PPR;
      const bool live = q < nst * P;
      const float4 gv = gain ? ga : make_float4(1.f, 1.f, 1.f, 1.f);
      char* my = xl;
      const int j = q / P, e = (q % P) * 4;
#pragma unroll
      for (int jx = 0; jx < NX; ++jx) {
        const int m = r0 + RP * jx;
        float4 v = xa[jx];
        v.x = live ? v.x * gv.x : 0.f;
        v.y = live ? v.y * gv.y : 0.f;
        v.z = live ? v.z * gv.z : 0.f;
        v.w = live ? v.w * gv.w : 0.f;
        if constexpr (WB) {
          uint16_t* hi = (uint16_t*)my;
          uint16_t* lo = hi + KC * MT * 32;
          const float xs[4] = {v.x, v.y, v.z, v.w};
          uint32_t h[4], l[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            h[i] = f32_to_bf16_bits(xs[i]);
            l[i] = f32_to_bf16_bits(xs[i] - __uint_as_float(h[i] << 16));
          }
          const int o = (j * MT + m) * 32 + e;
          *(uint2*)(hi + o) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
          *(uint2*)(lo + o) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
        } else {
          *(float4*)((float*)my + (j * MT + m) * 16 + e) = v;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      __builtin_amdgcn_sched_barrier(0);
      fetch_x(xsb);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int jj = 0; jj < KC; ++jj) {
        if constexpr (WB) {
          const uint16_t* hi = (const uint16_t*)my;
          const uint16_t* lo = hi + KC * MT * 32;
          const int o = (jj * MT + mread) * 32 + 8 * grp;
          const bf16x8_t a_hi = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(hi + o));
          const bf16x8_t a_lo = __builtin_bit_cast(bf16x8_t, *(const u32x4_t*)(lo + o));
          const bf16x8_t bw = __builtin_bit_cast(bf16x8_t, buf[jj]);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_hi, bw, acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a_lo, bw, acc, 0, 0, 0);
        } else {
          const float4 a = *(const float4*)((const float*)my + (jj * MT + mread) * 16 + 4 * grp);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, __uint_as_float(buf[jj][0]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, __uint_as_float(buf[jj][1]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, __uint_as_float(buf[jj][2]), acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, __uint_as_float(buf[jj][3]), acc, 0, 0, 0);
        }
      }
      __builtin_amdgcn_wave_barrier();
    }
    load(nbase, nsb, buf);
  }

  // Stream the workgroup's tiles: local tile i (i < n_local) starts at
  // ptr(i).  When every wave has finished tile i, epi(i, acc) runs
  // workgroup-wide (it reduces the per-wave accumulators); later chunks are
  // in flight by then.  Chunk c of the sequence is in w (c even) or w2 (c odd).
  template <class Ptr, class Epi>
  __device__ __forceinline__ void run(int n_local, const Ptr& ptr, Epi& epi) {
    f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
    if (s0 >= s1) {   // a wave without steps still takes part in every epilogue
      for (int i = 0; i < n_local; ++i) epi(i, acc);
      return;
    }
    const int lo16 = (threadIdx.x & 63) * 16;
    int i = 0, k = 0;     // current chunk
    int i2 = 0, k2 = 0;   // the chunk two ahead
    for (int a = 0; a < 2; ++a)
      if (++k2 == nchunks) { k2 = 0; ++i2; }
    const char* cur_tile = ptr(0);
    if constexpr (XPIPE)
      if (!xfetched) fetch_x(s0);
    // steps of the chunk after chunk k (activations repeat from tile to tile)
    auto xnext = [&](int kk) { return s0 + (kk + 1 == nchunks ? 0 : kk + 1) * KC; };
    auto step = [&](u32x4_t (&buf)[KC]) -> bool {
      const bool more2 = i2 < n_local;
      const char* nb = more2 ? ptr(i2) + lo16 : cur_tile + lo16;
      chunk(s0 + k * KC, nb, more2 ? s0 + k2 * KC : s1, buf, acc, xnext(k));
      if (k == nchunks - 1) {
        epi(i, acc);
        acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
      if (++k == nchunks) { k = 0; ++i; }
      if (++k2 == nchunks) { k2 = 0; ++i2; }
      if (i >= n_local) return true;
      if (k == 0) cur_tile = ptr(i);
      return false;
    };
    // The first chunk runs before the loop: every path into the loop then
    // issues its loads in the same order (next chunk's activations, then the
    // weights two ahead), so the compiler's waits for the activations never
    // wait for weights that are not yet needed.
    if (step(w)) return;
    for (;;) {
      if (step(w2)) return;
      if (step(w)) return;
    }
  }
};

__device__ __forceinline__ float ld_w(const void* p, size_t i, int wb) {
  return wb ? bf16_to_f32(((const uint16_t*)p)[i]) : ((const float*)p)[i];
}

// sum_{j<r} W[row][j] * u[j] for a [rows][r] matrix (adapter B factors);
// 16-byte loads when the row is 16-byte aligned.
__device__ __forceinline__ float dot_row(const void* W, size_t row, int r, const float* u, int wb) {
  float v = 0.f;
  const size_t b = row * r;
  if (wb && (r & 7) == 0) {
    const u32x4_t* p = (const u32x4_t*)((const uint16_t*)W + b);
    for (int j = 0; j < r; j += 8) {
      const u32x4_t w = p[j / 8];
#pragma unroll
      for (int i = 0; i < 4; ++i) v += bf16lo(w[i]) * u[j + 2 * i] + bf16hi(w[i]) * u[j + 2 * i + 1];
    }
    return v;
  }
  if (!wb && (r & 3) == 0) {
    const float4* p = (const float4*)((const float*)W + b);
    for (int j = 0; j < r; j += 4) {
      const float4 w = p[j / 4];
      v += w.x * u[j] + w.y * u[j + 1] + w.z * u[j + 2] + w.w * u[j + 3];
    }
    return v;
  }
#pragma unroll 8
  for (int j = 0; j < r; ++j) v += ld_w(W, b + j, wb) * u[j];
  return v;
}

// The same with the weight dtype fixed at compile time (no branch between
// two loads, which would make the wave wait for every load in flight).
template <int WB>
__device__ __forceinline__ float ld_wt(const void* p, size_t i) {
  if constexpr (WB) return bf16_to_f32(((const uint16_t*)p)[i]);
  else return ((const float*)p)[i];
}
template <int WB>
__device__ __forceinline__ float dot_row_t(const void* W, size_t row, int r, const float* u) {
  float v = 0.f;
  const size_t b = row * r;
  if constexpr (WB) {
    if ((r & 7) == 0) {
      const u32x4_t* p = (const u32x4_t*)((const uint16_t*)W + b);
      for (int j = 0; j < r; j += 8) {
        const u32x4_t w = p[j / 8];
#pragma unroll
        for (int i = 0; i < 4; ++i) v += bf16lo(w[i]) * u[j + 2 * i] + bf16hi(w[i]) * u[j + 2 * i + 1];
      }
      return v;
    }
  } else {
    if ((r & 3) == 0) {
      const float4* p = (const float4*)((const float*)W + b);
      for (int j = 0; j < r; j += 4) {
        const float4 w = p[j / 4];
        v += w.x * u[j] + w.y * u[j + 1] + w.z * u[j + 2] + w.w * u[j + 3];
      }
      return v;
    }
  }
  for (int j = 0; j < r; ++j) v += ld_wt<WB>(W, b + j) * u[j];
  return v;
}

// Raw bits of a weight element (bf16 zero-extended or f32), to be turned
// into a float later (raw_f): loads issued before the weights are primed
// must not be consumed before the prime.
template <int WB>
__device__ __forceinline__ uint32_t ld_raw(const void* p, size_t i) {
  if constexpr (WB) return ((const uint16_t*)p)[i];
  else return ((const uint32_t*)p)[i];
}
template <int WB>
__device__ __forceinline__ float raw_f(uint32_t r) {
  return WB ? __uint_as_float(r << 16) : __uint_as_float(r);
}

// The row map is a kernel argument; indexing it at a runtime index is a
// vector load from the argument segment, and waiting for one after the weight
// loads are in flight waits for all of them.  Prologues therefore read the
// argument words into registers before the weights are primed and keep a
// copy in LDS.
static_assert(sizeof(RowMap) % 4 == 0, "row map copied as words");
constexpr int kRmWords = (int)(sizeof(RowMap) / 4);
union SkRmLds {
  RowMap rm;
  int w[kRmWords];
};
// Copy of the map into LDS by the first wave (readable after the next
// workgroup barrier).  The words are read with constant indices, i.e. scalar
// loads through the constant cache (a lane-indexed read of a kernel argument
// would be a vector load from the argument segment, which misses every cache
// at kernel start); lane i stores word i.
__device__ __forceinline__ void sk_rm_copy(SkRmLds& dst, const RowMap& rm) {
  static_assert(kRmWords <= 64, "one word per lane of the first wave");
  if (threadIdx.x >= 64) return;
  const int* w = (const int*)&rm;
  const int t = (int)threadIdx.x;
  int wv[kRmWords];
#pragma unroll
  for (int i = 0; i < kRmWords; ++i) {
    wv[i] = w[i];
    asm volatile("" : "+s"(wv[i]));   // opaque: the select below stays a select of values
  }
  int v = wv[kRmWords - 1];
#pragma unroll
  for (int i = 0; i < kRmWords - 1; ++i) v = t == i ? wv[i] : v;
  if (t < kRmWords) dst.w[t] = v;
}

// Element m of a per-row field of the row map, for a per-thread m: built
// from selects over constant indices (the row map is a kernel argument, so
// these are scalar loads; a runtime index would become a vector load and a
// wait for every load in flight).
__device__ __forceinline__ int rsel(const int8_t (&a)[kMaxRows], int m) {
  int v = a[0];
#pragma unroll
  for (int c = 1; c < kMaxRows; ++c) v = (m == c) ? (int)a[c] : v;
  return v;
}

// out[o] = sum_{t<n} src[t*stride + o] for o < n_out with every thread of the
// block; the summation order depends only on (n, n_out, blockDim).  src is
// read with device-coherent loads (it was written by other workgroups of the
// same kernel).  `scratch` holds blockDim.x floats.  Ends with a barrier.
__device__ void column_sums(const float* src, int n, int stride, int n_out, float* out, float* scratch) {
  const int T = blockDim.x;
  if (n_out >= T / 2) {
    for (int o = threadIdx.x; o < n_out; o += T) {
      float a = 0.f;
#pragma unroll 8
      for (int t = 0; t < n; ++t) a += ld_agent(src + (size_t)t * stride + o);
      out[o] = a;
    }
    __syncthreads();
    return;
  }
  const int G = T / n_out;
  const int o = threadIdx.x % n_out, g = threadIdx.x / n_out;
  float a = 0.f;
  if (g < G) {
#pragma unroll 8
    for (int t = g; t < n; t += G) a += ld_agent(src + (size_t)t * stride + o);
  }
  scratch[threadIdx.x] = a;
  __syncthreads();
  if (threadIdx.x < n_out) {
    float b = 0.f;
    for (int gg = 0; gg < G; ++gg) b += scratch[gg * n_out + threadIdx.x];
    out[threadIdx.x] = b;
  }
  __syncthreads();
}

// ============================================================================
// Kernel: pack up to three stacked row-major matrices [rows_g][K] into the
// tile-packed layout (one-time, at context creation).
// ============================================================================
struct PackSrc {
  const void* p[3];
  int rows[3];
};

template <int WB>
__global__ __launch_bounds__(256) void k_pack(PackSrc src, int total_rows, int K, void* dst) {
  constexpr int KSTEP = WB ? 32 : 16, EPL = WB ? 8 : 4, ESZ = WB ? 2 : 4;
  const int S = K / KSTEP;
  const size_t n = (size_t)((total_rows + 15) / 16) * S * 64;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    const size_t ts = i >> 6;
    const int s = (int)(ts % S);
    const size_t t = ts / S;
    int r = (int)(t * 16) + (l & 15);
    const int col = s * KSTEP + EPL * (l >> 4);
    u32x4_t v = {0u, 0u, 0u, 0u};
    for (int g = 0; g < 3; ++g) {
      if (r < src.rows[g]) {
        if (src.p[g]) v = *(const u32x4_t*)((const char*)src.p[g] + ((size_t)r * K + col) * ESZ);
        break;
      }
      r -= src.rows[g];
    }
    *(u32x4_t*)((char*)dst + i * 16) = v;
  }
}

// Pack the gate and up matrices ([rows][K] each) as interleaved tile pairs:
// pair t holds gate rows 16t.. and up rows 16t..; K-step s of the gate is
// block 2s of the pair, of the up projection block 2s+1.
template <int WB>
__global__ __launch_bounds__(256) void k_pack_pair(const void* wg, const void* wu, int rows, int K, void* dst) {
  constexpr int KSTEP = WB ? 32 : 16, EPL = WB ? 8 : 4, ESZ = WB ? 2 : 4;
  const int S = K / KSTEP;
  const size_t n = (size_t)((rows + 15) / 16) * 2 * S * 64;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    const size_t ts = i >> 6;
    const int j = (int)(ts % (2 * S));
    const size_t t = ts / (2 * S);
    const int r = (int)(t * 16) + (l & 15);
    const int col = (j >> 1) * KSTEP + EPL * (l >> 4);
    const void* src = (j & 1) ? wu : wg;
    u32x4_t v = {0u, 0u, 0u, 0u};
    if (r < rows) v = *(const u32x4_t*)((const char*)src + ((size_t)r * K + col) * ESZ);
    *(u32x4_t*)((char*)dst + i * 16) = v;
  }
}

// ============================================================================
// Kernel: embedding gather + per-step control initialisation + zeroed bins.
// grid = M rows + kEmbedZeroBlocks, block = 256.  Block m < M gathers row m
// and writes its layer-0 bins (every slot); the other blocks zero the bins
// of every later layer (all slots, the M rows in use).
// ============================================================================
constexpr int kEmbedZeroBlocks = 64;

__global__ __launch_bounds__(256) void k_embed(Dims D, const void* embed, RowMap rm, WS ws, StepIO io, int init_ctl) {
  __shared__ float red[4];
  if ((int)blockIdx.x >= rm.M) {
    // zero bin_d of layers 1..n_layers, bin_o and bin_gu: every (layer, slot)
    // block holds kMaxRows rows of nv values, of which rows < M are used
    const int nvs[3] = {4, 1 + 2 * D.r, D.r};
    float* bases[3] = {ws.bin_d + (size_t)kBinSlots * kMaxRows * 4, ws.bin_o, ws.bin_gu};
    const int nblk = D.n_layers * kBinSlots;
    const int stride = (gridDim.x - rm.M) * 256;
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      const int used = rm.M * nvs[a], n = nblk * used;
      for (int i = (blockIdx.x - rm.M) * 256 + threadIdx.x; i < n; i += stride) {
        const int blk = i / used;
        bases[a][(size_t)blk * kMaxRows * nvs[a] + (i - blk * used)] = 0.f;
      }
    }
    return;
  }
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
  // layer-0 bins of this row: slot 0 holds the sums, the other slots zero
  for (int i = threadIdx.x; i < kBinSlots * 4; i += 256) {
    const int b = i / 4, c = i % 4;
    bin_d_at(ws, 0, b, m)[c] = (b == 0 && c < 3) ? ss : 0.f;
  }
  if (init_ctl && m == 0) {
    for (int s = threadIdx.x; s < kMaxSeq; s += 256) {
      ws.exited[s] = 0;
      ws.exitb[s] = D.n_layers;
    }
  }
}

// Gate decision of sequence s for the boundary before `layer`, identical in
// every workgroup (same inputs, same summation order): reinit (p <- h for
// this layer) and the updated exited flag / boundary; sig[s] receives the
// signal of layer-1.
__device__ void gate_logic(const Dims& D, const RowMap& rm, const int* ex_in, const int* eb_in, const StepIO& io,
                           int layer, const float* ssum /* [16][4] */, const float* asig, int* reinit_s, int* exited_s,
                           int* exitb_s, float* sig_s, int s) {
  {
    int ex = ex_in[s], eb = eb_in[s], ri = 0;
    float sg = 0.f;
    const int f = rm.first[s] + rm.cnt[s] - 1;
    if (layer > 0 && rm.fast[f]) {
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      sg = dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
      if (io.arla_sig && is_gate(io, layer)) sg = asig[s];   // the router scores, read before the weights
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

// uo_s[m][j] = sum over heads h (in order) of uo[m][h][j] for every fast row
// m: the o-adapter's down-projection, summed over the heads, all rows at
// once (every thread one (row, j) pair, its loads independent).  Read after
// the caller's next barrier.
__device__ __forceinline__ void fast_uo_sums(const Dims& D, const RowMap& rml, int M, const float* uo, float* uo_s) {
  for (int e = threadIdx.x; e < M * D.r; e += blockDim.x) {
    const int m = e / D.r, o = e - m * D.r;
    if (!rml.fast[m]) continue;
    const float* src = uo + (size_t)m * D.H * D.r + o;
    float a = 0.f;
#pragma unroll 8
    for (int h = 0; h < D.H; ++h) a += ld_agent(src + (size_t)h * D.r);
    uo_s[e] = a;
  }
}

// ============================================================================
// Kernel: QKV projection of every row (+ adapter-down rows), with the gate
// decision of the preceding boundary.  grid = tiles of 16 rows over
// [Wq; Wk; Wv; Aq; Ak; Av], block = 512.
// ============================================================================
template <int WB, int MT>
__global__ __launch_bounds__(kGemvThreads) void k_qkv(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  using TG = TileGemv<WB, MT>;
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int ex_in[kMaxSeq], eb_in[kMaxSeq];
  __shared__ int reinit_s[kMaxSeq], exited_s[kMaxSeq], exitb_s[kMaxSeq];
  __shared__ float sig_s[kMaxSeq], asig_s[kMaxSeq];
  __shared__ float inv_rms[kMaxRows];
  __shared__ int src_s[kMaxRows];
  __shared__ const float* xrow_s[kMaxRows];
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  __shared__ SkRmLds rmu;   // the row map, for per-thread indices (read after the first barrier)
  const RowMap& rml = rmu.rm;
  const int nq = D.qdim, tq = nq / 16;
  const int nqkv = 3 * nq + 3 * D.r;
  const int ntiles = 3 * tq + (3 * D.r + 15) / 16;
  const size_t tb = (size_t)16 * D.d * (WB ? 2 : 4);   // bytes of one packed tile
  // tile t: Wq, Wk, Wv, then the stacked adapter-down rows [A_q; A_k; A_v]
  // the four base pointers as values (a select over the kernel-argument
  // fields would become a vector load from the argument segment)
  const char* bq = (const char*)L.pq;
  const char* bk = (const char*)L.pk;
  const char* bv_ = (const char*)L.pv;
  const char* ba = (const char*)L.pa;
  asm volatile("" : "+s"(bq), "+s"(bk), "+s"(bv_), "+s"(ba));
  auto tile_ptr = [bq, bk, bv_, ba, tq, tb](int t) -> const char* {
    if (t < 3 * tq) {
      const int which = t / tq;
      return (which == 0 ? bq : (which == 1 ? bk : bv_)) + (size_t)(t - which * tq) * tb;
    }
    return ba + (size_t)(t - 3 * tq) * tb;
  };
  if ((int)blockIdx.x >= ntiles) return;
  auto ptr = [&](int i) { return tile_ptr(blockIdx.x + i * gridDim.x); };
  const int n_local = (ntiles - blockIdx.x + gridDim.x - 1) / gridDim.x;
  TG tg;
  tg.init(D.d, dyn);
  // ---- everything needed before the weights: issued first ----
  // (unconditional loads at clamped indices; consumed after the prime)
  float bv[kBins];
  {
    const int q = min((int)threadIdx.x, rm.M * 4 - 1);
#pragma unroll
    for (int b = 0; b < kBins; ++b) bv[b] = bin_d_at(ws, layer, b, q >> 2)[q & 3];
  }
  const int sq0 = min((int)threadIdx.x, rm.nseq - 1);
  const int exv = ws.exited[sq0], ebv = ws.exitb[sq0];
  const float asv = (io.arla_sig ? io.arla_sig : ws.arla_sig)[sq0];   // unconditional: used only with the router
  const float* rows[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) rows[m] = ws.X + (size_t)min(m, rm.M - 1) * D.d;
  typename TG::template Pieces<2> xp;
  if constexpr (TG::XRES) tg.load_pieces(rows, L.attn_norm, xp);
  __builtin_amdgcn_sched_barrier(0);
  tg.prime(n_local, ptr);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  if (threadIdx.x < rm.M * 4) {
    float a = 0.f;
#pragma unroll
    for (int b = 0; b < kBins; ++b) a += bv[b];
    ssum[threadIdx.x] = a;
  }
  if (threadIdx.x < rm.nseq) {
    ex_in[threadIdx.x] = exv;
    eb_in[threadIdx.x] = ebv;
    asig_s[threadIdx.x] = asv;
  }
  __syncthreads();
  // one thread per sequence, then one per row (serial loops of dependent LDS
  // reads on one thread took microseconds)
  if (threadIdx.x < rm.nseq)
    gate_logic(D, rml, ex_in, eb_in, io, layer, ssum, asig_s, reinit_s, exited_s, exitb_s, sig_s, threadIdx.x);
  __syncthreads();
  if (threadIdx.x < rm.M) {
    const int m = threadIdx.x;
    const int sq = rml.seq[m];
    int src = m;
    if (rml.fast[m] && reinit_s[sq]) src = rml.slow_of[m];
    src_s[m] = src;
    xrow_s[m] = ws.X + (size_t)src * D.d;
    inv_rms[m] = rsqrtf(ssum[src * 4] / D.d + D.eps);
  }
  __syncthreads();
  if (blockIdx.x == 0 && threadIdx.x < rm.nseq) {
    const int sq = threadIdx.x;
    ws.reinit[layer * kMaxSeq + sq] = reinit_s[sq];
    ws.exited[sq] = exited_s[sq];
    ws.exitb[sq] = exitb_s[sq];
    if (layer > 0) ws.sig[sq * D.n_layers + layer - 1] = sig_s[sq];
  }
  if constexpr (TG::XRES) {
    int sel[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) sel[m] = m < rm.M ? src_s[m] : 0;
    tg.store_pieces(xp, rows, L.attn_norm, sel);
  } else {
    tg.set_rows(xrow_s, L.attn_norm, rm.M, D.d);
  }
  auto epi = [&](int i, const f32x4_t& a) {
    const int t = blockIdx.x + i * gridDim.x;
    f32x4_t acc[1] = {a};
    gemv_reduce<1>(acc, rm.M, red, y);
    for (int e = threadIdx.x; e < rm.M * 16; e += kGemvThreads) {
      const int m = e >> 4, nn = t * 16 + (e & 15);
      if (nn < nqkv) ws.QKV[(size_t)m * nqkv + nn] = y[e] * inv_rms[m];
    }
  };
  tg.run(n_local, ptr, epi);
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
  if (rm.fast[m] && L.B[which] && L.A[which]) v += dot_row(L.B[which], c, D.r, row + 3 * D.qdim + which * D.r, D.wbf16);
  return v;
}

// Fill out[R][hd] with q (which=0) or k (which=1) after RoPE, or v (which=2).
__device__ __forceinline__ void head_vectors(const Dims& D, const LayerPtrs& L, const RowMap& rm, const WS& ws,
                                             const StepIO& io,
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
      int pos = row_pos(rm, io, first + i);
      if (pos < 0 || pos >= ws.rope_len) {
        atomicOr(ws.err, 8);
        pos = 0;
      }
      const float2 cs = ws.rope[(size_t)pos * half + j];   // cos, sin of pos * theta^(-2j/hd)
      const float c = cs.x, s = cs.y;
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

// Attention partial of one (sequence, head, split) and row: running max m,
// sum of exponentials l, unnormalised accumulator acc[hd] and the o-adapter
// down-projection of acc (fast rows), r floats.  Layout of ws.att:
// [seq][H][splits+1][16 rows][2 + hd + r]; split index `splits` holds the
// rows' own keys.
__device__ __forceinline__ float* att_part(const WS& ws, const Dims& D, int s, int h, int sp, int n_split, int i) {
  const int stride = 2 + D.hd + D.r;
  return ws.att + ((((size_t)s * D.H + h) * (n_split + 1) + sp) * kMaxRows + i) * stride;
}

// Merge the partials of one (sequence, head): the output o of every row and,
// for fast rows, the o-adapter down-projection of that head.  The partials
// were written by other workgroups: device-coherent loads.
__device__ __forceinline__ void attn_merge(const Dims& D, const RowMap& rm, const WS& ws, int s, int h, int n_split) {
  __shared__ float stat[kMaxRows * 64 * 2];   // m, l of every split (n_split + 1 <= 64)
  __shared__ float wgt[kMaxRows * 64];
  __shared__ float linv[kMaxRows];
  const int R = rm.cnt[s], first = rm.first[s];
  const int S1 = n_split + 1;
  for (int e = threadIdx.x; e < R * S1; e += blockDim.x) {
    const int i = e / S1, sp = e % S1;
    const float* pp = att_part(ws, D, s, h, sp, n_split, i);
    stat[(i * 64 + sp) * 2] = ld_agent(pp);
    stat[(i * 64 + sp) * 2 + 1] = ld_agent(pp + 1);
  }
  __syncthreads();
  if (threadIdx.x < R) {
    const int i = threadIdx.x;
    float M = -INFINITY;
    for (int sp = 0; sp < S1; ++sp)
      if (stat[(i * 64 + sp) * 2 + 1] > 0.f) M = fmaxf(M, stat[(i * 64 + sp) * 2]);
    float Lsum = 0.f;
    for (int sp = 0; sp < S1; ++sp) {
      const float l = stat[(i * 64 + sp) * 2 + 1];
      const float w = l > 0.f ? __expf(stat[(i * 64 + sp) * 2] - M) : 0.f;
      wgt[i * 64 + sp] = w;
      Lsum += w * l;
    }
    linv[i] = 1.f / Lsum;
  }
  __syncthreads();
  const int W = D.hd + D.r;
  for (int e = threadIdx.x; e < R * W; e += blockDim.x) {
    const int i = e / W, c = e % W;
    float v = 0.f;
    for (int sp0 = 0; sp0 < S1; sp0 += 8) {
      float part[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) part[u] = ld_agent(att_part(ws, D, s, h, min(sp0 + u, S1 - 1), n_split, i) + 2 + c);
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (sp0 + u < S1) v += wgt[i * 64 + sp0 + u] * part[u];
    }
    v *= linv[i];
    const int mi = first + i;
    if (c < D.hd) ws.O[(size_t)mi * D.qdim + h * D.hd + c] = v;
    else ws.uo[((size_t)mi * D.H + h) * D.r + (c - D.hd)] = rm.fast[mi] ? v : 0.f;
  }
}

// Kernel: attention over the shared cache, one context split per workgroup,
// plus one workgroup per (sequence, head) for the rows' own keys and the cache
// writes; the last workgroup of a (sequence, head) to finish merges the
// partials.  A split's first 128 cached keys and values (usually all of them)
// are put in flight before q is formed.  grid = (splits + 1, H, nseq),
// block = 256.
constexpr int kAttnPrefetch = 2;   // tokens per thread loaded ahead (x 64 slots = 128 tokens)

template <int KB, int HD>
__global__ __launch_bounds__(kAttnThreads) void k_attn(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, KVPtrs kv,
                                                       int layer, int n_split) {
  extern __shared__ float sm[];
  __shared__ SkRmLds rmu;   // the row map in LDS: the helpers index it per thread
  const RowMap& rml = rmu.rm;
  sk_rm_copy(rmu, rm);
  __syncthreads();
  constexpr int DPL = HD / 4;             // dims per lane (4 lanes per token)
  const int split = blockIdx.x, h = blockIdx.y, s = blockIdx.z;
  const int hd = HD, R = rml.cnt[s], first = rml.first[s];
  const float scale = rsqrtf((float)hd);
  float* q = sm;                           // [R][hd]
  float* kx = q + kMaxRows * kMaxHeadDim;  // [R][hd]
  float* vx = kx + kMaxRows * kMaxHeadDim; // [R][hd]
  float* sc = vx + kMaxRows * kMaxHeadDim; // [R][per] scores, then probabilities
  float* redp = sc + kScoreCap;            // [4 waves][2 rows][hd]
  __shared__ float rowm[kMaxRows], rowl[kMaxRows];
  __shared__ float uacc_s[kMaxRows * kMaxRank];
  __shared__ int last_flag;

  const int ctx = io.positions[s] + rm.pos_offset;
  const bool frozen = ws.exited[s] != 0;
  const bool own = split == n_split;
  bool store = !frozen;   // this workgroup produces a partial

  if (own) {
    // ---- the rows' own keys and the cache writes -------------------------------
    head_vectors(D, L, rml, ws, io, first, R, 1, h, kx);
    head_vectors(D, L, rml, ws, io, first, R, 2, h, vx);
    for (int e = threadIdx.x; e < R * hd; e += kAttnThreads) {
      const int i = e / hd, d = e % hd;
      if (!rml.wr[first + i]) continue;
      bool ok;
      const size_t ix = kv_index(kv, D, layer, s, ctx + rml.idx[first + i], h, d, ok);
      if (!ok) { atomicOr(ws.err, 2); continue; }
      if (KB) {
        ((uint16_t*)kv.k)[ix] = (uint16_t)f32_to_bf16_bits(kx[e]);
        ((uint16_t*)kv.v)[ix] = (uint16_t)f32_to_bf16_bits(vx[e]);
      } else {
        ((float*)kv.k)[ix] = kx[e];
        ((float*)kv.v)[ix] = vx[e];
      }
    }
    if (!frozen) {
      head_vectors(D, L, rml, ws, io, first, R, 0, h, q);
      // a slow row sees the chunk's slow rows up to itself (as stored in the
      // cache); a fast row sees only its own exact key/value
      float* ownsc = sc;   // [R][R]
      for (int e = threadIdx.x; e < R * R; e += kAttnThreads) {
        const int i = e / R, jj = e % R;
        const int mi = first + i, mj = first + jj;
        bool vis;
        if (rml.fast[mi]) vis = (jj == i);
        else vis = !rml.fast[mj] && rml.idx[mj] <= rml.idx[mi];
        float p = -INFINITY;
        if (vis) {
          p = 0.f;
          const bool rnd = !rml.fast[mi];
          for (int d = 0; d < hd; ++d) {
            const float kk = rnd ? kv_round(kx[jj * hd + d], KB) : kx[jj * hd + d];
            p += q[i * hd + d] * kk;
          }
          p *= scale;
        }
        ownsc[e] = p;
      }
      __syncthreads();
      if (threadIdx.x < R) {
        const int i = threadIdx.x;
        float mx = -INFINITY;
        for (int jj = 0; jj < R; ++jj) mx = fmaxf(mx, ownsc[i * R + jj]);
        float l = 0.f;
        for (int jj = 0; jj < R; ++jj) {
          const float v = ownsc[i * R + jj] == -INFINITY ? 0.f : __expf(ownsc[i * R + jj] - mx);
          ownsc[i * R + jj] = v;
          l += v;
        }
        rowm[i] = mx;
        rowl[i] = l;
      }
      __syncthreads();
      for (int e = threadIdx.x; e < R * hd; e += kAttnThreads) {
        const int i = e / hd, d = e % hd;
        const bool rnd = !rml.fast[first + i];
        float a = 0.f;
        for (int jj = 0; jj < R; ++jj) {
          const float w = ownsc[i * R + jj];
          if (w != 0.f) a += w * (rnd ? kv_round(vx[jj * hd + d], KB) : vx[jj * hd + d]);
        }
        q[e] = a;   // acc of the own-key partial
      }
      __syncthreads();
    }
  } else if (!frozen) {
    // ---- this split's share of the cached context [0, ctx) -------------------
    const int per = ((ctx + n_split - 1) / n_split + 15) & ~15;
    const int t0 = min(ctx, split * per), t1 = min(ctx, t0 + per);
    const int nt = t1 - t0;
    const int sub = threadIdx.x & 3, slot = threadIdx.x >> 2;
    const int d0 = sub * DPL;
    // keys and values of the first tokens, in flight while q is formed
    float kpf[kAttnPrefetch][DPL], vpf[kAttnPrefetch][DPL];
#pragma unroll
    for (int it = 0; it < kAttnPrefetch; ++it) {
      const int j = slot + it * (kAttnThreads / 4);
      bool ok;
      const size_t base = kv_index(kv, D, layer, s, t0 + min(j, max(nt - 1, 0)), h, d0, ok);
      kv_row_load<KB, HD>(kv.k, base, ok && j < nt, kpf[it]);
      kv_row_load<KB, HD>(kv.v, base, ok && j < nt, vpf[it]);
    }
    head_vectors(D, L, rml, ws, io, first, R, 0, h, q);
    if (per * R > kScoreCap) {             // the host sizes splits so that this cannot happen
      if (threadIdx.x == 0) atomicOr(ws.err, 4);
      store = false;
    } else {
      {
        int it = 0;
        for (int j = slot; j < nt; j += kAttnThreads / 4, ++it) {
          float kk[DPL];
          if (it < kAttnPrefetch) {
#pragma unroll
            for (int c = 0; c < DPL; ++c) kk[c] = it == 0 ? kpf[0][c] : kpf[kAttnPrefetch - 1][c];
          } else {
            bool ok;
            const size_t base = kv_index(kv, D, layer, s, t0 + j, h, d0, ok);
            kv_row_load<KB, HD>(kv.k, base, ok, kk);
          }
          for (int i = 0; i < R; ++i) {
            float p = 0.f;
#pragma unroll
            for (int c = 0; c < DPL; ++c) p += q[i * hd + d0 + c] * kk[c];
            p += __shfl_xor(p, 1);
            p += __shfl_xor(p, 2);
            if (sub == 0) sc[i * per + j] = p * scale;
          }
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
          if (lane == 0) { rowm[i] = nt > 0 ? mx : -INFINITY; rowl[i] = nt > 0 ? l : 0.f; }
        }
      }
      __syncthreads();
      const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
      for (int i0 = 0; i0 < R; i0 += 2) {
        const bool two = i0 + 1 < R;
        float acc0[DPL], acc1[DPL];
#pragma unroll
        for (int c = 0; c < DPL; ++c) { acc0[c] = 0.f; acc1[c] = 0.f; }
        int it = 0;
        for (int j = slot; j < nt; j += kAttnThreads / 4, ++it) {
          float vv[DPL];
          if (it < kAttnPrefetch) {
#pragma unroll
            for (int c = 0; c < DPL; ++c) vv[c] = it == 0 ? vpf[0][c] : vpf[kAttnPrefetch - 1][c];
          } else {
            bool ok;
            const size_t base = kv_index(kv, D, layer, s, t0 + j, h, d0, ok);
            kv_row_load<KB, HD>(kv.v, base, ok, vv);
          }
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
            q[(i0 + a) * hd + d] = v;   // q is no longer needed: reuse it for acc
          }
        }
        __syncthreads();
      }
    }
  }
  if (store) {
    // ---- store the partial: m, l, acc, and A_o[:, head cols] . acc (fast rows) ----
    // A_o[j][h*hd + d] . acc_i[d]: 8 dims per thread, then a sum over hd/8 threads
    constexpr int PCS = HD / 8;
    float* up = redp;
    for (int i0 = 0; i0 < R; ++i0) {
      if (!rml.fast[first + i0] || !L.A[3]) {
        for (int j = threadIdx.x; j < D.r; j += kAttnThreads) uacc_s[i0 * D.r + j] = 0.f;
        continue;
      }
      for (int e = threadIdx.x; e < D.r * PCS; e += kAttnThreads) {
        const int j = e / PCS, pc = e % PCS;
        const size_t base = (size_t)j * D.qdim + h * hd + pc * 8;
        float u = 0.f;
#pragma unroll
        for (int t = 0; t < 8; ++t) u += ld_w(L.A[3], base + t, D.wbf16) * q[i0 * hd + pc * 8 + t];
        up[e] = u;
      }
      __syncthreads();
      for (int j = threadIdx.x; j < D.r; j += kAttnThreads) {
        float u = 0.f;
        for (int pc = 0; pc < PCS; ++pc) u += up[j * PCS + pc];
        uacc_s[i0 * D.r + j] = u;
      }
      __syncthreads();
    }
    __syncthreads();
    for (int i = 0; i < R; ++i) {
      float* pp = att_part(ws, D, s, h, split, n_split, i);
      for (int e = threadIdx.x; e < 2 + hd + D.r; e += kAttnThreads) {
        float v;
        if (e == 0) v = rowm[i];
        else if (e == 1) v = rowl[i];
        else if (e < 2 + hd) v = q[i * hd + e - 2];
        else v = uacc_s[i * D.r + e - 2 - hd];
        st_agent(pp + e, v);
      }
    }
  }
  // every workgroup of the (sequence, head) counts in; the last one merges
  if (!arrive_last(&ws.att_cnt[s * D.H + h], n_split + 1, &last_flag)) return;
  if (frozen) return;
  attn_merge(D, rml, ws, s, h, n_split);
}

// ============================================================================
// Kernel: output projection + residual add (+ adapter on the fast row);
// partial sums for the gate/up prologue.  Persistent tile GEMV, grid <= d/16.
// The epilogue operands of the workgroup's first tile (old residual values,
// the B_o rows, the A_g/A_u columns and gains, the exit flags) are issued
// before the weights, so that epilogue waits for nothing but the reduction.
// ============================================================================
template <int WB, int MT>
__global__ __launch_bounds__(kGemvThreads) void k_oproj(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  using TG = TileGemv<WB, MT>;
  constexpr bool PRE = TG::XRES;
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float uo_s[kMaxRows * kMaxRank];
  __shared__ float newx[256];
  __shared__ float xo_s[kMaxRows * 16];      // first tile: X of every row
  __shared__ float bo_s[16 * kMaxRank];      // first tile: B_o rows
  __shared__ float agu_s[2 * kMaxRank * 16]; // first tile: A_g, A_u columns times g_mlp
  __shared__ float ud_s[2 * kGemvThreads];   // per-head o-adapter values of the fast row (PRE)
  __shared__ int flag_s[2 * kMaxSeq];        // exited, reinit
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  __shared__ SkRmLds rmu;   // the row map, for per-thread indices (read after the first barrier)
  const RowMap& rml = rmu.rm;
  const int ntiles = D.d / 16;
  if ((int)blockIdx.x >= ntiles) return;
  if (io.mode == EX_EXIT) {
    bool all_exited = true;
    for (int sq = 0; sq < rm.nseq; ++sq) all_exited &= ws.exited[sq] != 0;
    if (all_exited) return;
  }
  const size_t tb = (size_t)16 * D.qdim * (WB ? 2 : 4);
  auto tile_ptr = [&](int t) -> const char* { return (const char*)L.po + (size_t)t * tb; };
  auto ptr = [&](int i) { return tile_ptr(blockIdx.x + i * gridDim.x); };
  const int n_local = (ntiles - blockIdx.x + gridDim.x - 1) / gridDim.x;
  const int PO = 1 + 2 * D.r;
  const int n00 = blockIdx.x * 16;
  int fast_m = -1;   // the fast row (2-row class: at most one); constant indices keep rm in scalar registers
#pragma unroll
  for (int m = 0; m < kMaxRows; ++m)
    if (m < rm.M && rm.fast[m]) fast_m = m;
  TG tg;
  tg.init(D.qdim, dyn);
  const float* rows[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) rows[m] = ws.O + (size_t)min(m, rm.M - 1) * D.qdim;
  typename TG::template Pieces<2> xp;
  float pre[3] = {0.f, 0.f, 0.f};
  uint32_t praw = 0, araw = 0;
  float gmlp = 0.f;
  int fl = 0;
  const int tid = threadIdx.x;
  const int HR = D.H * D.r;
  const bool pre_uo = PRE && HR <= 2 * kGemvThreads;     // per-head values fit two per thread
  const bool pre_agu = 2 * D.r * 16 <= kGemvThreads;
  // ---- everything needed before the weights: issued first, unconditional
  // loads at clamped indices (a load under a branch, or a value consumed
  // right away, would make the wave wait before the prime); the first
  // tile's epilogue operands in every class ----
  if constexpr (!PRE) tg.early_rows(rows, nullptr);
  if constexpr (PRE) {
    tg.load_pieces(rows, nullptr, xp);
    const int fm = fast_m >= 0 ? fast_m : 0;
    pre[0] = ws.uo[(size_t)fm * HR + min(tid, HR - 1)];
    pre[1] = ws.uo[(size_t)fm * HR + min(tid + kGemvThreads, HR - 1)];
  }
  {
    const int mx = min(tid >> 4, rm.M - 1);
    pre[2] = ws.X[(size_t)mx * D.d + n00 + (tid & 15)];
    const int bq = min(tid, 16 * D.r - 1);
    praw = ld_raw<WB>(L.B[3] ? L.B[3] : L.po, (size_t)(n00 + bq / D.r) * D.r + bq % D.r);
    const int aq = min(tid, 2 * D.r * 16 - 1);
    const int which = aq / (D.r * 16), j = (aq / 16) % D.r, i = aq % 16;
    const void* A = which ? L.A[5] : L.A[4];
    araw = ld_raw<WB>(A ? A : L.po, (size_t)j * D.d + n00 + i);
    gmlp = L.mlp_norm[n00 + i];
    const int fq = min(tid, 2 * rm.nseq - 1);
    fl = fq < rm.nseq ? ws.exited[fq] : ws.reinit[layer * kMaxSeq + fq - rm.nseq];
  }
  __builtin_amdgcn_sched_barrier(0);
  tg.prime(n_local, ptr);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  for (int e = threadIdx.x; e < rm.M * D.r; e += kGemvThreads) uo_s[e] = 0.f;
  if constexpr (PRE) {
    ud_s[tid] = pre[0];
    ud_s[tid + kGemvThreads] = pre[1];
  }
  {
    if (tid < rm.M * 16) xo_s[tid] = pre[2];
    if (tid < 16 * D.r) bo_s[tid] = L.B[3] ? raw_f<WB>(praw) : 0.f;
    if (pre_agu && tid < 2 * D.r * 16) {
      const void* A = (tid / (D.r * 16)) ? L.A[5] : L.A[4];
      agu_s[tid] = A ? raw_f<WB>(araw) * gmlp : 0.f;
    }
    if (tid < 2 * rm.nseq) flag_s[tid] = fl;
  }
  __syncthreads();
  if constexpr (PRE) {
    // adapter-down of o summed over heads: uo is [H][r] per row
    if (pre_uo) {
      if (fast_m >= 0 && L.A[3] && tid < D.r) {
        float a = 0.f;
        for (int h = 0; h < D.H; ++h) a += ud_s[h * D.r + tid];
        uo_s[fast_m * D.r + tid] = a;
      }
    } else if (L.A[3]) {
      fast_uo_sums(D, rml, rm.M, ws.uo, uo_s);
    }
    int sel[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) sel[m] = m < rm.M ? m : 0;
    tg.store_pieces(xp, rows, nullptr, sel);
  } else {
    if (L.A[3]) fast_uo_sums(D, rml, rm.M, ws.uo, uo_s);
  }
  __syncthreads();
  auto epi = [&](int i, const f32x4_t& a) {
    const int t = blockIdx.x + i * gridDim.x;
    const bool first = i == 0;   // operands already in LDS
    f32x4_t acc[1] = {a};
    gemv_reduce<1>(acc, rm.M, red, y);
    const int n0 = t * 16;
    // epilogue: read everything first (a fast row restarting at a gate reads
    // its slow row's old value), write after a barrier
    const int e = threadIdx.x;
    const int m = e >> 4, nn = n0 + (e & 15);
    float xnew = 0.f, pin = 0.f;
    bool upd = false;
    if (e < rm.M * 16) {
      const int sq = rml.seq[m];
      const float xo = first ? xo_s[e] : ws.X[(size_t)m * D.d + nn];
      xnew = xo;
      const bool ex = first ? flag_s[sq] != 0 : ws.exited[sq] != 0;
      if (!ex) {
        upd = true;
        if (rml.fast[m]) {
          const bool ri = first ? flag_s[rm.nseq + sq] != 0 : ws.reinit[layer * kMaxSeq + sq] != 0;
          const int so = rml.slow_of[m];
          pin = ri ? (first ? xo_s[so * 16 + (e & 15)] : ws.X[(size_t)so * D.d + nn]) : xo;
          float ad = 0.f;
          if (L.B[3] && L.A[3]) {
            if (first) {
              for (int j = 0; j < D.r; ++j) ad += bo_s[(e & 15) * D.r + j] * uo_s[m * D.r + j];
            } else {
              ad = dot_row_t<WB>(L.B[3], nn, D.r, uo_s + m * D.r);
            }
          }
          xnew = pin + y[e] + ad;
        } else {
          xnew = xo + y[e];
        }
      }
      newx[e] = xnew;
    }
    __syncthreads();
    if (upd) {
      ws.X[(size_t)m * D.d + nn] = xnew;
      if (rml.fast[m]) ws.PIN[(size_t)m * D.d + nn] = pin;
    }
    // partial sums for the gate/up prologue: sum x^2 and the adapter-down of
    // gate and up (fast rows): sum_n A[j][n] g_mlp[n] x[n]
    const int bin = t % kBins;
    for (int q = threadIdx.x; q < rm.M * PO; q += kGemvThreads) {
      const int mm = q / PO, c = q % PO;
      float v = 0.f;
      if (c == 0) {
        for (int ii = 0; ii < 16; ++ii) v += newx[mm * 16 + ii] * newx[mm * 16 + ii];
      } else if (rml.fast[mm]) {
        const int which = (c - 1) / D.r, j = (c - 1) % D.r;   // 0: gate (A[4]), 1: up (A[5])
        const void* A = which ? L.A[5] : L.A[4];
        if (A) {
          if (first && pre_agu) {
            for (int ii = 0; ii < 16; ++ii) v += agu_s[(which * D.r + j) * 16 + ii] * newx[mm * 16 + ii];
          } else {
            for (int ii = 0; ii < 16; ++ii)
              v += ld_wt<WB>(A, (size_t)j * D.d + n0 + ii) * L.mlp_norm[n0 + ii] * newx[mm * 16 + ii];
          }
        }
      }
      if (c == 0 || rml.fast[mm]) add_agent(bin_o_at(ws, D, layer, bin, mm) + c, v);
    }
    __syncthreads();
  };
  tg.run(n_local, ptr, epi);
}

// ============================================================================
// Kernel: gate/up projections (the gate and up tiles of the same 16 rows, one
// after the other), adapter-up, SwiGLU; partial sums of the down adapter's
// down-projection.  Persistent tile GEMV, grid <= ffn/16.  The row
// statistics and the first pair's B_g, B_u rows and A_d columns are issued
// before the weights (the 2-row class also its activation pieces).
// ============================================================================
template <int WB, int MT>
__global__ __launch_bounds__(kGemvThreads) void k_gateup(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  using TG = TileGemv<WB, MT, 2048>;   // gate and up blocks alternate in the pair layout
  constexpr bool PRE = TG::XRES;
  __shared__ float red[kGemvWaves * 512];
  __shared__ float y[512];
  __shared__ float stat[kMaxRows * (1 + 2 * kMaxRank)];
  __shared__ float inv_rms[kMaxRows];
  __shared__ float act[256];
  __shared__ float bgu_s[2 * 16 * kMaxRank];   // first pair: B_g, B_u rows
  __shared__ float ad_s[kMaxRank * 16];        // first pair: A_d columns
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  __shared__ SkRmLds rmu;   // the row map, for per-thread indices (read after the first barrier)
  const RowMap& rml = rmu.rm;
  const int ntiles = D.F / 16;
  if ((int)blockIdx.x >= ntiles) return;
  if (io.mode == EX_EXIT) {
    bool all_exited = true;
    for (int sq = 0; sq < rm.nseq; ++sq) all_exited &= ws.exited[sq] != 0;
    if (all_exited) return;
  }
  const size_t tb = (size_t)16 * D.d * (WB ? 2 : 4);
  // local tiles 2i and 2i+1: the gate and up tiles of rows 16*t, t = blockIdx.x + i*gridDim.x, in the
  // interleaved pair layout (pair t at 2*t*tb; gate step s at block 2s, up step s at block 2s+1)
  auto ptr = [&](int i) {
    return (const char*)L.pg + (size_t)(blockIdx.x + (i >> 1) * gridDim.x) * 2 * tb + (i & 1) * 1024;
  };
  const int n_local = 2 * ((ntiles - blockIdx.x + gridDim.x - 1) / gridDim.x);
  const int PO = 1 + 2 * D.r;
  const int n00 = blockIdx.x * 16;
  const int tid = threadIdx.x;
  const bool pre_b = 2 * 16 * D.r <= kGemvThreads;
  TG tg;
  tg.init(D.d, dyn);
  // ---- everything needed before the weights: issued first ----
  // (unconditional loads at clamped indices; consumed after the prime)
  float sv[kBins];
  {
    const int q = min(tid, rm.M * PO - 1);
#pragma unroll
    for (int b = 0; b < kBins; ++b) sv[b] = bin_o_at(ws, D, layer, b, q / PO)[q % PO];
  }
  const float* rows[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) rows[m] = ws.X + (size_t)min(m, rm.M - 1) * D.d;
  typename TG::template Pieces<2> xp;
  uint32_t pb = 0, pa = 0;
  if constexpr (PRE) tg.load_pieces(rows, L.mlp_norm, xp);
  else tg.early_rows(rows, L.mlp_norm);
  {   // the first pair's epilogue operands (every class)
    const int bq = min(tid, 2 * 16 * D.r - 1);
    const int which = bq / (16 * D.r), rr = (bq / D.r) % 16, j = bq % D.r;
    const void* B = which ? L.B[5] : L.B[4];
    pb = ld_raw<WB>(B ? B : L.pg, (size_t)(n00 + rr) * D.r + j);
    const int aq = min(tid, D.r * 16 - 1);
    pa = ld_raw<WB>(L.A[6] ? L.A[6] : L.pg, (size_t)(aq / 16) * D.F + n00 + (aq % 16));
  }
  __builtin_amdgcn_sched_barrier(0);
  tg.prime(n_local, ptr);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  if (tid < rm.M * PO) {
    float a = 0.f;
#pragma unroll
    for (int b = 0; b < kBins; ++b) a += sv[b];
    stat[tid] = a;
  }
  if (pre_b && tid < 2 * 16 * D.r) {
    const int which = tid / (16 * D.r);
    const bool has = which ? (L.B[5] && L.A[5]) : (L.B[4] && L.A[4]);
    bgu_s[tid] = has ? raw_f<WB>(pb) : 0.f;
  }
  if (tid < D.r * 16) ad_s[tid] = L.A[6] ? raw_f<WB>(pa) : 0.f;
  __syncthreads();
  if (tid < rm.M) inv_rms[tid] = rsqrtf(stat[tid * PO] / D.d + D.eps);
  if constexpr (PRE) {
    int sel[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) sel[m] = m < rm.M ? m : 0;
    tg.store_pieces(xp, rows, L.mlp_norm, sel);
  }
  __syncthreads();
  f32x4_t acc_g = {0.f, 0.f, 0.f, 0.f};
  auto epi = [&](int i, const f32x4_t& a) {
    if (!(i & 1)) {
      acc_g = a;
      return;
    }
    const int t = blockIdx.x + (i >> 1) * gridDim.x;
    const bool first = i == 1;
    f32x4_t acc[2] = {acc_g, a};
    gemv_reduce<2>(acc, rm.M, red, y);
    const int n0 = t * 16;
    const int e = threadIdx.x;
    if (e < rm.M * 16) {
      const int m = e >> 4, nn = n0 + (e & 15);
      const float ir = inv_rms[m];
      float g = y[e] * ir, u = y[256 + e] * ir;
      if (rml.fast[m]) {
        if (first && pre_b) {
          float dg = 0.f, du = 0.f;
          for (int j = 0; j < D.r; ++j) {
            dg += bgu_s[(e & 15) * D.r + j] * stat[m * PO + 1 + j];
            du += bgu_s[(16 + (e & 15)) * D.r + j] * stat[m * PO + 1 + D.r + j];
          }
          g += dg * ir;
          u += du * ir;
        } else {
          if (L.B[4] && L.A[4]) g += dot_row_t<WB>(L.B[4], nn, D.r, stat + m * PO + 1) * ir;
          if (L.B[5] && L.A[5]) u += dot_row_t<WB>(L.B[5], nn, D.r, stat + m * PO + 1 + D.r) * ir;
        }
      }
      const float av = silu(g) * u;
      ws.ACT[(size_t)m * D.F + nn] = av;
      act[e] = av;
    }
    __syncthreads();
    // partials of the down adapter-down: sum_n A_d[j][n] a[n]
    const int bin = t % kBins;
    for (int q = threadIdx.x; q < rm.M * D.r; q += kGemvThreads) {
      const int mm = q / D.r, j = q % D.r;
      if (!rml.fast[mm] || !L.A[6]) continue;
      float v = 0.f;
      if (first) {
        for (int ii = 0; ii < 16; ++ii) v += ad_s[j * 16 + ii] * act[mm * 16 + ii];
      } else {
        for (int ii = 0; ii < 16; ++ii) v += ld_wt<WB>(L.A[6], (size_t)j * D.F + n0 + ii) * act[mm * 16 + ii];
      }
      add_agent(bin_gu_at(ws, D, layer, bin, mm) + j, v);
    }
    __syncthreads();
  };
  tg.run(n_local, ptr, epi);
}

// Partial sums entering layer `next` (sum x^2, sum pin*x, sum pin^2 of every
// row) when no kernel updates the rows: every sequence has exited.  One
// workgroup.
__device__ void rows_unchanged_stats(const Dims& D, const RowMap& rm, const WS& ws, int next) {
  __shared__ float red[kGemvWaves];
  for (int m = 0; m < rm.M; ++m) {
    float a = 0.f, b = 0.f, c = 0.f;
    for (int i = threadIdx.x; i < D.d; i += blockDim.x) {
      const float x = ws.X[(size_t)m * D.d + i];
      const float p = rsel(rm.fast, m) ? ws.PIN[(size_t)m * D.d + i] : 0.f;
      a += x * x; b += p * x; c += p * p;
    }
    a = block_sum(a, red);
    b = block_sum(b, red);
    c = block_sum(c, red);
    if (threadIdx.x == 0) {
      add_agent(bin_d_at(ws, next, 0, m) + 0, a);
      add_agent(bin_d_at(ws, next, 0, m) + 1, b);
      add_agent(bin_d_at(ws, next, 0, m) + 2, c);
    }
    __syncthreads();
  }
}

// ============================================================================
// Kernel: down projection + residual add (+ adapter); partial sums for the
// next layer's norm and the exit signal.  Persistent tile GEMV, grid <= d/16.
// The adapter sums and the first tile's residual values, fast-row inputs and
// B_d rows are issued before the weights (the 2-row class also its
// activation pieces).
// ============================================================================
template <int WB, int MT>
__global__ __launch_bounds__(kGemvThreads) void k_down(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  using TG = TileGemv<WB, MT>;
  constexpr bool PRE = TG::XRES;
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float ud[kMaxRows * kMaxRank];
  __shared__ float newx[256], pin_s[256];
  __shared__ float xo_s[kMaxRows * 16], pino_s[kMaxRows * 16];   // first tile
  __shared__ float bd_s[16 * kMaxRank];                          // first tile: B_d rows
  __shared__ int ex_s[kMaxSeq];                                  // exited
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  __shared__ SkRmLds rmu;   // the row map, for per-thread indices (read after the first barrier)
  const RowMap& rml = rmu.rm;
  const int ntiles = D.d / 16;
  if ((int)blockIdx.x >= ntiles) return;
  if (io.mode == EX_EXIT) {
    bool all_exited = true;
    for (int sq = 0; sq < rm.nseq; ++sq) all_exited &= ws.exited[sq] != 0;
    if (all_exited) {
      if (blockIdx.x == 0) rows_unchanged_stats(D, rm, ws, layer + 1);
      return;
    }
  }
  const size_t tb = (size_t)16 * D.F * (WB ? 2 : 4);
  auto tile_ptr = [&](int t) -> const char* { return (const char*)L.pd + (size_t)t * tb; };
  auto ptr = [&](int i) { return tile_ptr(blockIdx.x + i * gridDim.x); };
  const int n_local = (ntiles - blockIdx.x + gridDim.x - 1) / gridDim.x;
  const int n00 = blockIdx.x * 16;
  const int tid = threadIdx.x;
  TG tg;
  tg.init(D.F, dyn);
  // ---- everything needed before the weights: issued first ----
  // (unconditional loads at clamped indices; consumed after the prime)
  float uv[kBins];
  {
    const int q = min(tid, rm.M * D.r - 1);
#pragma unroll
    for (int b = 0; b < kBins; ++b) uv[b] = bin_gu_at(ws, D, layer, b, q / D.r)[q % D.r];
  }
  const float* rows[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) rows[m] = ws.ACT + (size_t)min(m, rm.M - 1) * D.F;
  typename TG::template Pieces<4> xp;
  float px = 0.f, pp = 0.f;
  uint32_t pb = 0;
  int pe = 0;
  if constexpr (PRE) tg.load_pieces(rows, nullptr, xp);
  else tg.early_rows(rows, nullptr);
  {   // the first tile's epilogue operands (every class)
    const int m = min(tid >> 4, rm.M - 1);
    px = ws.X[(size_t)m * D.d + n00 + (tid & 15)];
    pp = ws.PIN[(size_t)m * D.d + n00 + (tid & 15)];
    const int bq = min(tid, 16 * D.r - 1);
    pb = ld_raw<WB>(L.B[6] ? L.B[6] : L.pd, (size_t)(n00 + bq / D.r) * D.r + bq % D.r);
    pe = ws.exited[min(tid, rm.nseq - 1)];
  }
  __builtin_amdgcn_sched_barrier(0);
  tg.prime(n_local, ptr);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  if (tid < rm.M * D.r) {
    float a = 0.f;
#pragma unroll
    for (int b = 0; b < kBins; ++b) a += uv[b];
    ud[tid] = a;
  }
  {
    if (tid < rm.M * 16) {
      xo_s[tid] = px;
      pino_s[tid] = pp;   // used for fast rows only
    }
    if (tid < 16 * D.r) bd_s[tid] = (L.B[6] && L.A[6]) ? raw_f<WB>(pb) : 0.f;
    if (tid < rm.nseq) ex_s[tid] = pe;
  }
  __syncthreads();
  if constexpr (PRE) {
    int sel[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) sel[m] = m < rm.M ? m : 0;
    tg.store_pieces(xp, rows, nullptr, sel);
  }
  auto epi = [&](int i, const f32x4_t& a) {
    const int t = blockIdx.x + i * gridDim.x;
    const bool first = i == 0;
    f32x4_t acc[1] = {a};
    gemv_reduce<1>(acc, rm.M, red, y);
    const int n0 = t * 16;
    const int e = threadIdx.x;
    if (e < rm.M * 16) {
      const int m = e >> 4, nn = n0 + (e & 15);
      float x = first ? xo_s[e] : ws.X[(size_t)m * D.d + nn];
      const bool ex = first ? ex_s[rml.seq[m]] != 0 : ws.exited[rml.seq[m]] != 0;
      if (!ex) {
        x += y[e];
        if (rml.fast[m] && L.B[6] && L.A[6]) {
          if (first) {
            float ad = 0.f;
            for (int j = 0; j < D.r; ++j) ad += bd_s[(e & 15) * D.r + j] * ud[m * D.r + j];
            x += ad;
          } else {
            x += dot_row_t<WB>(L.B[6], nn, D.r, ud + m * D.r);
          }
        }
        ws.X[(size_t)m * D.d + nn] = x;
      }
      newx[e] = x;
      pin_s[e] = rml.fast[m] ? (first ? pino_s[e] : ws.PIN[(size_t)m * D.d + nn]) : 0.f;
    }
    __syncthreads();
    const int bin = t % kBins;
    for (int q = threadIdx.x; q < rm.M * 3; q += kGemvThreads) {
      const int mm = q / 3, c = q % 3;
      float v = 0.f;
      for (int ii = 0; ii < 16; ++ii) {
        const float x = newx[mm * 16 + ii], p = pin_s[mm * 16 + ii];
        v += c == 0 ? x * x : (c == 1 ? p * x : p * p);
      }
      add_agent(bin_d_at(ws, layer + 1, bin, mm) + c, v);
    }
    __syncthreads();
  };
  tg.run(n_local, ptr, epi);
}

// ============================================================================
// Kernel: final norm + LM head + argmax; the last workgroup to finish takes
// the global arg-max and finishes the step (tokens, exit bookkeeping,
// acceptance of a verified chunk).  Persistent tile GEMV, grid <= V/16.
// ============================================================================
template <int WB, int MT>
__global__ __launch_bounds__(kGemvThreads) void k_head(Dims D, const void* lm_head, const float* final_norm, RowMap rm,
                                                       WS ws, StepIO io, KVPtrs kv, int n_tiles, int n_layers_run) {
  __shared__ float red[kGemvWaves * 256];
  __shared__ float y[256];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int hrow[kMaxRows];
  __shared__ int nh_s;
  __shared__ float inv_rms[kMaxRows];
  __shared__ int last_flag;
  __shared__ const float* xrow_s[kMaxRows];
  extern __shared__ __attribute__((aligned(16))) char dyn[];
  __shared__ SkRmLds rmu;   // the row map, for per-thread indices (read after the first barrier)
  const RowMap& rml = rmu.rm;
  if ((int)blockIdx.x >= n_tiles) return;
  using TG = TileGemv<WB, MT>;
  const int lane = threadIdx.x & 63;
  const size_t tb = (size_t)16 * D.d * (WB ? 2 : 4);
  auto tile_ptr = [&](int t) -> const char* { return (const char*)lm_head + (size_t)t * tb; };
  auto ptr = [&](int i) { return tile_ptr(blockIdx.x + i * gridDim.x); };
  const int n_local = (n_tiles - blockIdx.x + gridDim.x - 1) / gridDim.x;
  __shared__ int ex_in[kMaxSeq];
  TG tg;
  tg.init(D.d, dyn);
  // ---- everything needed before the weights: issued first ----
  // (unconditional loads at clamped indices; consumed after the prime)
  float bv[kBins];
  {
    const int q = min((int)threadIdx.x, rm.M * 4 - 1);
#pragma unroll
    for (int b = 0; b < kBins; ++b) bv[b] = bin_d_at(ws, n_layers_run, b, q >> 2)[q & 3];
  }
  const int exv = ws.exited[min((int)threadIdx.x, rm.nseq - 1)];
  const float* rows[MT];
#pragma unroll
  for (int m = 0; m < MT; ++m) rows[m] = ws.X + (size_t)min(m, rm.M - 1) * D.d;
  typename TG::template Pieces<2> xp;
  if constexpr (TG::XRES) tg.load_pieces(rows, final_norm, xp);
  __builtin_amdgcn_sched_barrier(0);
  tg.prime(n_local, ptr);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  if (threadIdx.x < rm.M * 4) {
    float a = 0.f;
#pragma unroll
    for (int b = 0; b < kBins; ++b) a += bv[b];
    ssum[threadIdx.x] = a;
  }
  if (threadIdx.x < rm.nseq) ex_in[threadIdx.x] = exv;
  __syncthreads();
  // rows fed to the head: every row of a chunk, else one per sequence (one
  // thread each: a serial loop of dependent LDS reads took microseconds)
  if (rm.head_all) {
    if (threadIdx.x < rm.M) hrow[threadIdx.x] = threadIdx.x;
    if (threadIdx.x == 0) nh_s = rm.M;
  } else {
    const int sq = threadIdx.x;
    if (sq < rm.nseq) {
      const int f = rml.first[sq], c = rml.cnt[sq];
      int pick = f;                       // slow row
      if (rml.fast[f + c - 1] && (ex_in[sq] || rml.slow_of[f + c - 1] < 0)) pick = f + c - 1;
      hrow[sq] = pick;
    }
    if (threadIdx.x == 0) nh_s = rm.nseq;
  }
  __syncthreads();
  if (threadIdx.x < nh_s) {
    inv_rms[threadIdx.x] = rsqrtf(ssum[hrow[threadIdx.x] * 4] / D.d + D.eps);
    xrow_s[threadIdx.x] = ws.X + (size_t)hrow[threadIdx.x] * D.d;
  }
  __syncthreads();
  const int nh = nh_s;
  if constexpr (TG::XRES) {
    int sel[MT];
#pragma unroll
    for (int m = 0; m < MT; ++m) sel[m] = m < nh ? hrow[m] : 0;
    tg.store_pieces(xp, rows, final_norm, sel);
  } else {
    tg.set_rows(xrow_s, final_norm, nh, D.d);
  }
  auto epi = [&](int i, const f32x4_t& a) {
    const int t = blockIdx.x + i * gridDim.x;
    f32x4_t acc[1] = {a};
    gemv_reduce<1>(acc, nh, red, y);
    // logits and the tile's arg-max per head row (lowest index on ties)
    const int e = threadIdx.x;
    if (e < nh * 16) {
      const int k = e >> 4, nn = t * 16 + (e & 15);
      float z = y[e] * inv_rms[k];
      if (nn >= D.V) z = -INFINITY;
      else if (io.logits_out) io.logits_out[(size_t)k * D.V + nn] = z;
      int idx = nn;
#pragma unroll
      for (int o = 8; o > 0; o >>= 1) {
        const float z2 = __shfl_xor(z, o);
        const int i2 = __shfl_xor(idx, o);
        if (z2 > z || (z2 == z && i2 < idx)) { z = z2; idx = i2; }
      }
      if ((e & 15) == 0) {
        st_agent(&ws.lm_val[(size_t)t * kMaxRows + k], z);
        st_agent(&ws.lm_idx[(size_t)t * kMaxRows + k], idx);
      }
    }
  };
  tg.run(n_local, ptr, epi);
  if (!arrive_last(ws.lm_cnt, gridDim.x, &last_flag)) return;

  // ---- last workgroup: global argmax per head row, then bookkeeping ----------
  __shared__ int best_s[kMaxRows];
  const int wave = threadIdx.x >> 6;
  for (int k = wave; k < nh; k += kGemvWaves) {
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int t = lane; t < n_tiles; t += 64) {
      const float z = ld_agent(&ws.lm_val[(size_t)t * kMaxRows + k]);
      const int i = ld_agent(&ws.lm_idx[(size_t)t * kMaxRows + k]);
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
  for (int sq = threadIdx.x; sq < rm.nseq; sq += kGemvThreads) {
    const int f = rml.first[sq] + rml.cnt[sq] - 1;
    io.next_token[sq + io.draft_slot] = best_s[sq];
    const int t = io.positions[sq] + rm.pos_offset;
    if (rml.slow_of[f] >= 0 || !rml.fast[f]) kv.seq_lens[sq] = t + 1;
    if (rml.fast[f] && rml.slow_of[f] >= 0) {
      // signal of the last layer
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      ws.sig[sq * D.n_layers + D.n_layers - 1] = ws.exited[sq] ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
    }
    if (io.exit_b_out) io.exit_b_out[sq] = ws.exitb[sq];
    if (io.advance) io.positions[sq] = io.positions[sq] + 1;
  }
  __syncthreads();
  if (io.signal_out) {
    for (int q = threadIdx.x; q < rm.nseq * D.n_layers; q += kGemvThreads) {
      const int sq = q / D.n_layers, l = q % D.n_layers;
      const int f = rml.first[sq] + rml.cnt[sq] - 1;
      float v = ws.sig[q];
      // layers after an exit were not run
      if (!rml.fast[f] || rml.slow_of[f] < 0 || (ws.exited[sq] && l >= ws.exitb[sq])) v = 0.f;
      io.signal_out[q] = v;
    }
  }
  if (io.h_out || io.p_out) {
    for (int q = threadIdx.x; q < rm.nseq * D.d; q += kGemvThreads) {
      const int sq = q / D.d, i = q % D.d;
      const int f = rml.first[sq], c = rml.cnt[sq];
      if (io.h_out) io.h_out[q] = ws.X[(size_t)f * D.d + i];
      if (io.p_out) io.p_out[q] = ws.X[(size_t)(f + c - 1) * D.d + i];
    }
  }
}

}  // namespace m2r2
