// Stream-K decode GEMVs for one or two rows: the dual-stream decode step
// (slow row h of Eq. 1 and fast row p of Eq. 2 of one sequence), plain
// single-stream decoding, drafting, and short verification chunks.
//
// A packed projection matrix is a contiguous sequence of 1 KB blocks (tile t,
// K-step s at block t*nblk + s; see the tile-packed layout in
// step_kernels.h).  The launch has one workgroup of 8 waves per compute unit
// and every wave streams one contiguous, equally long range of blocks, so all
// waves move the same number of bytes whatever the matrix shape.  A range may
// start or end inside a tile: each wave keeps one MFMA accumulator per tile
// it touches and stores it as a partial sum (segment) of that tile.  When a
// wave has finished its range it counts its segments in; the wave completing
// a tile sums the tile's segments in segment order (results do not depend on
// timing) and runs the tile's epilogue: residual update, adapters, SwiGLU,
// row statistics for the next kernel, logits and arg-max.
//
// The activation rows (times the norm gain) are staged once per workgroup in
// LDS as bf16 hi + lo planes in MFMA fragment order (bf16 weights: two
// v_mfma_f32_16x16x32_bf16 per block, 16 significant bits of the fp32
// activation) or as fp32 (four v_mfma_f32_16x16x4_f32 per block).  The 1/rms
// factor of the pre-norm is applied in the epilogue.
//
// The gate and up matrices are packed as interleaved pairs: tile t of the
// pair holds gate rows 16t..16t+15 and up rows 16t..16t+15, K-step s of the
// gate at block 2s and of the up projection at block 2s+1.  Wave ranges have
// an even length, so block parity tells gate from up at compile time.
#pragma once
#include "step_kernels.h"

namespace m2r2 {

constexpr int kSkWaves = 8;
constexpr int kSkThreads = 64 * kSkWaves;
constexpr int kSkPM = 4;   // activation pieces per thread held in registers
constexpr int kSkMaxK = 4 * kSkThreads * kSkPM;   // longest reduction (8192): the rows fit the pieces

// Work split of one matrix kind (host-computed; identical for every layer).
struct SkPlan {
  int ntiles;   // tiles (tile pairs for gate/up)
  int nblk;     // 1 KB blocks per tile
  int L;        // blocks per wave (even for gate/up)
  int smax;     // partial slots per tile (most waves touching one tile)
  int W;        // waves in the launch
};

__host__ __device__ inline int sk_first_wave(const SkPlan& p, int t) {
  return (int)(((long long)t * p.nblk) / p.L);
}
__host__ __device__ inline int sk_last_wave(const SkPlan& p, int t) {
  return (int)((((long long)t + 1) * p.nblk - 1) / p.L);
}

// LDS bytes of the staged activation rows for reduction length K.
__host__ __device__ constexpr int sk_act_bytes(int K) { return 8 * K; }

// Partial-sum slots and tile counters of the stream-K GEMVs.
struct SkWS {
  float* part;      // [tiles * smax][64]
  uint32_t* cnt;    // [tiles] arrival counters (zero between launches)
  uint32_t* hier;   // [64 + 1] two-level arrival counters of whole waves (zero between launches)
};

// Every wave with work counts in once (64 groups, then one counter for the
// groups); returns true in the wave that arrives last, which may then read
// what every other wave stored (agent scope) before it arrived.
__device__ __forceinline__ bool sk_arrive_all(const SkWS& sk, int gw, int n_active) {
  const int lane = threadIdx.x & 63;
  __builtin_amdgcn_s_waitcnt(0);
  uint32_t last = 0;
  if (lane == 0) {
    const int g = gw & 63;
    const uint32_t ng = (uint32_t)((n_active - g + 63) / 64);
    const uint32_t o1 = __hip_atomic_fetch_add(&sk.hier[g], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (o1 == ng - 1) {
      __hip_atomic_store(&sk.hier[g], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const uint32_t ngroups = (uint32_t)min(n_active, 64);
      const uint32_t o2 = __hip_atomic_fetch_add(&sk.hier[64], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (o2 == ngroups - 1) {
        __hip_atomic_store(&sk.hier[64], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        last = 1;
      }
    }
  }
  return __shfl(last, 0) != 0;
}

// ---------------------------------------------------------------------------
// Activation staging: each thread loads, for kSkPM groups of 4 consecutive k,
// both candidate rows and the gain into registers (issued before the weights
// are primed), and stores the selected rows into LDS afterwards.
// ---------------------------------------------------------------------------
template <int PM = kSkPM>
struct SkPiecesT {
  static constexpr int N = PM;
  float4 v[PM][2];
  float4 g[PM];
};
using SkPieces = SkPiecesT<kSkPM>;

template <int PM>
__device__ __forceinline__ void sk_load_pieces(const float* r0, const float* r1, const float* gain, int K,
                                               SkPiecesT<PM>& xp) {
  const int nq = K / 4;
#pragma unroll
  for (int p = 0; p < PM; ++p) {
    const int q = min((int)threadIdx.x + kSkThreads * p, nq - 1);
    xp.v[p][0] = ldg4(r0 + 4 * q);
    xp.v[p][1] = ldg4(r1 + 4 * q);
    xp.g[p] = ldg4((gain ? gain : r0) + 4 * q);
  }
}

template <int WB>
__device__ __forceinline__ void sk_put(char* lds, int nsteps, int k, int m, float4 v) {
  if constexpr (WB) {
    const int st = k >> 5, e = k & 31;
    uint16_t* hi = (uint16_t*)lds;
    uint16_t* lo = hi + nsteps * 64;
    const float xs[4] = {v.x, v.y, v.z, v.w};
    uint32_t h[4], l[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      h[i] = f32_to_bf16_bits(xs[i]);
      l[i] = f32_to_bf16_bits(xs[i] - __uint_as_float(h[i] << 16));
    }
    const int o = (st * 2 + m) * 32 + e;
    *(uint2*)(hi + o) = make_uint2(h[0] | (h[1] << 16), h[2] | (h[3] << 16));
    *(uint2*)(lo + o) = make_uint2(l[0] | (l[1] << 16), l[2] | (l[3] << 16));
  } else {
    const int st = k >> 4, e = k & 15;
    *(float4*)((float*)lds + (st * 2 + m) * 16 + e) = v;
  }
}

// Store row m (m = 0, 1) = candidate sel[m] times the gain (K <= kSkMaxK).
// Ends with a workgroup barrier.
template <int WB>
__device__ __forceinline__ void sk_store_pieces(const SkPieces& xp, const float* r0, const float* r1,
                                                const float* gain, int K, int sel0, int sel1, char* lds) {
  const int nq = K / 4, nsteps = K / (WB ? 32 : 16);
#pragma unroll
  for (int p = 0; p < kSkPM; ++p) {
    const int q = (int)threadIdx.x + kSkThreads * p;
    if (q < nq) {
      const float4 g = gain ? xp.g[p] : make_float4(1.f, 1.f, 1.f, 1.f);
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        const int sm = m ? sel1 : sel0;
        float4 v = sm ? xp.v[p][1] : xp.v[p][0];
        v.x *= g.x; v.y *= g.y; v.z *= g.z; v.w *= g.w;
        sk_put<WB>(lds, nsteps, 4 * q, m, v);
      }
    }
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// Row statistics: sums over the kBinSlots bins of nv values (value q of bin b
// at base[b * stride + q]).  Every thread loads NPT bin entries before the
// weights are primed, consecutive threads reading consecutive values of one
// bin; sk_bins_sum adds them in bin order (results do not depend on timing)
// through the LDS scratch (nv * kBinSlots floats) into out[nv].
// ---------------------------------------------------------------------------
template <int T = kSkThreads, int NPT>
__device__ __forceinline__ void sk_bins_load(int nv, const float* base, int stride, float (&v)[NPT]) {
  // element i = threadIdx.x + T * k (T threads) as (bin b, value q), stepped
  // without a division per element
  int b = (int)threadIdx.x / nv, q = (int)threadIdx.x - b * nv;
  const int db = T / nv, dq = T - db * nv;
#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const bool in = b < kBinSlots;   // past the end: read the last entry
    v[k] = base[(size_t)(in ? b : kBinSlots - 1) * stride + (in ? q : nv - 1)];
    b += db;
    q += dq;
    if (q >= nv) { q -= nv; ++b; }
  }
}
template <int T = kSkThreads, int NPT>
__device__ __forceinline__ void sk_bins_sum(int nv, const float (&v)[NPT], float* scratch, float* out) {
  const int n = nv * kBinSlots;
#pragma unroll
  for (int k = 0; k < NPT; ++k) {
    const int i = (int)threadIdx.x + T * k;
    if (i < n) scratch[i] = v[k];
  }
  __syncthreads();
  if ((int)threadIdx.x < nv) {
    float a = 0.f;
#pragma unroll
    for (int b = 0; b < kBinSlots; ++b) a += scratch[b * nv + threadIdx.x];
    out[threadIdx.x] = a;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// The streaming wave.
// ---------------------------------------------------------------------------
template <int WB, bool PAIR>
struct SkStream {
  static constexpr int NA = PAIR ? 2 : 1;
  u32x4_t wA[8], wB[8];
  const char* lb;   // this lane's 16 bytes of block 0
  int b0, b1, nsteps;

  __device__ __forceinline__ void init(const SkPlan& p, const void* base, int gw, int K) {
    const long long T = (long long)p.ntiles * p.nblk;
    b0 = (int)min((long long)gw * p.L, T);
    b1 = (int)min((long long)b0 + p.L, T);
    lb = (const char*)base + (threadIdx.x & 63) * 16;
    nsteps = K / (WB ? 32 : 16);
  }
  // blocks cb..cb+7; blocks past the range repeat its last block (block 0
  // for an empty range; never used).  Loads are never conditional: the
  // compiler's wait counts stay exact only when every path issues the same
  // loads.
  __device__ __forceinline__ void load(int cb, u32x4_t (&dst)[8]) const {
#pragma unroll
    for (int j = 0; j < 8; ++j) dst[j] = ld_glob(lb + (size_t)max(min(cb + j, b1 - 1), 0) * 1024);
  }
  // The first chunk only: a compute unit keeps about 64 KB of loads in
  // flight, and a wave issuing more waits at the issue, before the
  // prologue's own work.
  __device__ __forceinline__ void prime() { load(b0, wA); }

  // One chunk: blocks cb..cb+7 of the range in buf.  Blocks of tile t go to
  // aA, blocks of tile t+1 (at most one boundary per chunk: nblk >= 8) to aB.
  template <class Flush>
  __device__ __forceinline__ void chunk(const SkPlan& p, const char* act, int cb, u32x4_t (&buf)[8], int& t, int& s,
                                        f32x4_t (&aA)[NA], f32x4_t (&aB)[NA], Flush& flush) {
    const int lane = threadIdx.x & 63;
    const int mread = min(lane & 15, 1), grp = lane >> 4;
    const int nv = min(8, b1 - cb);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      int sj = s + j;
      const bool nx = sj >= p.nblk;
      sj = nx ? sj - p.nblk : sj;
      const int kst = PAIR ? (sj >> 1) : sj;
      const bool on = j < nv;
      const int which = PAIR ? (j & 1) : 0;   // a constant after unrolling
      f32x4_t src = nx ? aB[which] : aA[which];
      if constexpr (WB) {
        const uint16_t* hi = (const uint16_t*)act;
        const uint16_t* lo = hi + nsteps * 64;
        const int o = (kst * 2 + mread) * 32 + 8 * grp;
        u32x4_t h = *(const u32x4_t*)(hi + o), l = *(const u32x4_t*)(lo + o);
        if (!on) { h = u32x4_t{0u, 0u, 0u, 0u}; l = h; }
        const bf16x8_t bw = __builtin_bit_cast(bf16x8_t, buf[j]);
        src = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, h), bw, src, 0, 0, 0);
        src = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, l), bw, src, 0, 0, 0);
      } else {
        float4 a = *(const float4*)((const float*)act + (kst * 2 + mread) * 16 + 4 * grp);
        if (!on) a = make_float4(0.f, 0.f, 0.f, 0.f);
        src = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, __uint_as_float(buf[j][0]), src, 0, 0, 0);
        src = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, __uint_as_float(buf[j][1]), src, 0, 0, 0);
        src = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, __uint_as_float(buf[j][2]), src, 0, 0, 0);
        src = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, __uint_as_float(buf[j][3]), src, 0, 0, 0);
      }
      aA[which] = nx ? aA[which] : src;
      aB[which] = nx ? src : aB[which];
    }
    s += nv;
    if (s >= p.nblk) {   // tile t is complete in this range
      flush(t, aA);
#pragma unroll
      for (int i = 0; i < NA; ++i) {
        aA[i] = aB[i];
        aB[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
      ++t;
      s -= p.nblk;
    }
    if (cb + 8 >= b1 && s > 0) flush(t, aA);   // the range ends inside tile t
    load(cb + 16, buf);
  }

  // Stream the range; flush(t, acc) is called once per tile segment, in order.
  template <class Flush>
  __device__ __forceinline__ void run(const SkPlan& p, const char* act, Flush& flush) {
    if (b0 >= b1) return;
    int t = b0 / p.nblk, s = b0 - t * p.nblk;
    f32x4_t aA[NA], aB[NA];
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      aA[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      aB[i] = aA[i];
    }
    load(b0 + 8, wB);
    for (int cb = b0;;) {
      chunk(p, act, cb, wA, t, s, aA, aB, flush);
      cb += 8;
      if (cb >= b1) break;
      chunk(p, act, cb, wB, t, s, aA, aB, flush);
      cb += 8;
      if (cb >= b1) break;
    }
  }
};

// Store a tile segment (rows 0..1 of the 16x16 accumulator; PAIR: gate then
// up) into its partial slot.  Lanes 0..15 hold rows 0..3 of column lane.
template <bool PAIR>
__device__ __forceinline__ void sk_store_part(const SkPlan& p, const SkWS& sk, int gw, int t,
                                              const f32x4_t (&a)[PAIR ? 2 : 1]) {
  const int lane = threadIdx.x & 63;
  const int slot = t * p.smax + (gw - sk_first_wave(p, t));
  float* dst = sk.part + (size_t)slot * 64;
  if (lane < 16) {
#pragma unroll
    for (int i = 0; i < (PAIR ? 2 : 1); ++i) {
      st_agent(dst + 32 * i + lane, a[i][0]);
      st_agent(dst + 32 * i + 16 + lane, a[i][1]);
    }
  }
}

// After the wave's range: count its segments in (one atomic per tile, all
// tiles at once); for every tile this wave completes, sum the tile's
// segments in segment order and call epi(t, y, yu) with y = the sum for lane
// l < 32 (row l >> 4, column l & 15; PAIR: yu = the up projection's).
// Wave-level.
constexpr int kSkMaxSeg = 16;   // segments per tile (the host keeps smax <= 16)

template <bool PAIR, class Epi>
__device__ __forceinline__ void sk_finish(const SkPlan& p, const SkWS& sk, int gw, int b0, int b1, Epi& epi) {
  if (b0 >= b1) return;
  const int lane = threadIdx.x & 63;
  __builtin_amdgcn_s_waitcnt(0);   // the partial stores are complete
  const int t0 = b0 / p.nblk, nt = (b1 - 1) / p.nblk - t0 + 1;   // tiles touched (<= 64)
  bool last = false;
  if (lane < nt) {
    const int t = t0 + lane;
    const int wf = sk_first_wave(p, t), wl = min(sk_last_wave(p, t), p.W - 1);
    const uint32_t nseg = (uint32_t)(wl - wf + 1);
    const uint32_t old = __hip_atomic_fetch_add(&sk.cnt[t], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last = old == nseg - 1;
    if (last) __hip_atomic_store(&sk.cnt[t], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  uint64_t mask = __ballot(last);
  while (mask) {
    const int i = __builtin_ctzll(mask);
    mask &= mask - 1;
    const int t = t0 + i;
    const int wf = sk_first_wave(p, t), wl = min(sk_last_wave(p, t), p.W - 1);
    const int nseg = wl - wf + 1;
    const float* src = sk.part + (size_t)t * p.smax * 64 + (lane & 31);
    float v[kSkMaxSeg], vu[kSkMaxSeg];
#pragma unroll
    for (int k = 0; k < kSkMaxSeg; ++k) {
      v[k] = ld_agent(src + (size_t)min(k, nseg - 1) * 64);
      if (PAIR) vu[k] = ld_agent(src + (size_t)min(k, nseg - 1) * 64 + 32);
    }
    float y = 0.f, yu = 0.f;
#pragma unroll
    for (int k = 0; k < kSkMaxSeg; ++k) {
      if (k < nseg) {
        y += v[k];
        if (PAIR) yu += vu[k];
      }
    }
    epi(t, y, yu);
  }
}

// sum_{j<r} B[row][j] u[j] for an adapter up-factor B [rows][r] (r <= 32,
// r a multiple of 8 (bf16) or 4 (f32)): every load issued before use.
template <int WB>
__device__ __forceinline__ float sk_dot_b(const void* B, int row, int r, const float* u) {
  constexpr int EPC = WB ? 8 : 4;                 // elements per 16-byte chunk
  constexpr int NC = kMaxRank / EPC;
  const int nc = r / EPC;
  const u32x4_t* p = (const u32x4_t*)((const char*)B + (size_t)row * r * (WB ? 2 : 4));
  u32x4_t c[NC];
#pragma unroll
  for (int i = 0; i < NC; ++i) c[i] = p[min(i, nc - 1)];
  float v = 0.f;
#pragma unroll
  for (int i = 0; i < NC; ++i) {
    if (i >= nc) break;
    if constexpr (WB) {
#pragma unroll
      for (int k = 0; k < 4; ++k) v += bf16lo(c[i][k]) * u[8 * i + 2 * k] + bf16hi(c[i][k]) * u[8 * i + 2 * k + 1];
    } else {
#pragma unroll
      for (int k = 0; k < 4; ++k) v += __uint_as_float(c[i][k]) * u[4 * i + k];
    }
  }
  return v;
}

// sum_{i<16} A[j][n0 + i] x[i] for one row j of an adapter down-factor A
// [r][n] (16 consecutive elements: two 16-byte loads for bf16, four for f32).
template <int WB>
__device__ __forceinline__ void sk_load_a16(const void* A, size_t off, u32x4_t (&c)[WB ? 2 : 4]) {
  const u32x4_t* p = (const u32x4_t*)((const char*)A + off * (WB ? 2 : 4));
#pragma unroll
  for (int i = 0; i < (WB ? 2 : 4); ++i) c[i] = p[i];
}
template <int WB>
__device__ __forceinline__ float sk_dot_a16(const u32x4_t (&c)[WB ? 2 : 4], const float* x) {
  float v = 0.f;
#pragma unroll
  for (int i = 0; i < (WB ? 2 : 4); ++i) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if constexpr (WB) v += bf16lo(c[i][k]) * x[8 * i + 2 * k] + bf16hi(c[i][k]) * x[8 * i + 2 * k + 1];
      else v += __uint_as_float(c[i][k]) * x[4 * i + k];
    }
  }
  return v;
}

__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0): this wave's LDS writes are done
  __builtin_amdgcn_wave_barrier();
}

// Sum over the 16 lanes of a row group (lanes 16m .. 16m+15).
__device__ __forceinline__ float sum16(float v) { return row_sum16(v); }

// The gate decision of gate_logic for at most two sequences.
__device__ __forceinline__ void sk_gate_logic(const Dims& D, const RowMap& rm, const int* ex_in, const int* eb_in,
                                              const StepIO& io, int layer, const float* ssum, int* reinit_s,
                                              int* exited_s, int* exitb_s, float* sig_s) {
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    if (s >= rm.nseq) break;
    int ex = ex_in[s], eb = eb_in[s], ri = 0;
    float sg = 0.f;
    const int f = rm.first[s] + rm.cnt[s] - 1;
    if (layer > 0 && rm.fast[f]) {
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      sg = dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
      if (io.arla_sig && is_gate(io, layer)) sg = io.arla_sig[s];
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

__device__ __forceinline__ bool sk_all_exited(const RowMap& rm, const WS& ws) {
  bool all = true;
  for (int sq = 0; sq < rm.nseq; ++sq) all &= ws.exited[sq] != 0;
  return all;
}

// ============================================================================
// QKV: [Wq; Wk; Wv; A_q; A_k; A_v] x rms(x) g_att, with the gate decision of
// the boundary before the layer.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kSkThreads) void ks_qkv(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, SkPlan P,
                                                     SkWS sk, int layer) {
  extern __shared__ __attribute__((aligned(16))) char act[];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int ex_in[kMaxSeq], eb_in[kMaxSeq];
  __shared__ int reinit_s[kMaxSeq], exited_s[kMaxSeq], exitb_s[kMaxSeq];
  __shared__ float sig_s[kMaxSeq];
  __shared__ float inv_rms[2];
  __shared__ int src_s[2];
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, gw = blockIdx.x * kSkWaves + (tid >> 6);
  SkStream<WB, false> st;
  st.init(P, L.pq, gw, D.d);
  // loads needed before the weights: issued first
  float bv[1];
  sk_bins_load(rm.M * 4, bin_d_at(ws, layer, 0, 0), kMaxRows * 4, bv);
  const int sq0 = min(tid, rm.nseq - 1);
  const int exv = ws.exited[sq0], ebv = ws.exitb[sq0];
  const float* r0 = ws.X;
  const float* r1 = ws.X + (size_t)(rm.M > 1 ? 1 : 0) * D.d;
  SkPieces xp;
  sk_load_pieces(r0, r1, L.attn_norm, D.d, xp);
  __builtin_amdgcn_sched_barrier(0);
  st.prime();
  __builtin_amdgcn_sched_barrier(0);
  if (tid < rm.nseq) { ex_in[tid] = exv; eb_in[tid] = ebv; }
  sk_rm_copy(rmu, rm);
  sk_bins_sum(rm.M * 4, bv, (float*)act, ssum);
  if (tid == 0) {
    sk_gate_logic(D, rml, ex_in, eb_in, io, layer, ssum, reinit_s, exited_s, exitb_s, sig_s);
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      const int mm = min(m, rm.M - 1);
      int src = mm;
      if (rml.fast[mm] && reinit_s[rml.seq[mm]]) src = rml.slow_of[mm];
      src_s[m] = src;
      inv_rms[m] = rsqrtf(ssum[src * 4] / D.d + D.eps);
    }
  }
  __syncthreads();
  if (blockIdx.x == 0 && tid < rm.nseq) {
    ws.reinit[layer * kMaxSeq + tid] = reinit_s[tid];
    ws.exited[tid] = exited_s[tid];
    ws.exitb[tid] = exitb_s[tid];
    if (layer > 0) ws.sig[tid * D.n_layers + layer - 1] = sig_s[tid];
  }
  sk_store_pieces<WB>(xp, r0, r1, L.attn_norm, D.d, src_s[0], src_s[1], act);
  auto flush = [&](int t, const f32x4_t (&a)[1]) { sk_store_part<false>(P, sk, gw, t, a); };
  st.run(P, act, flush);
  const int nqkv = 3 * D.qdim + 3 * D.r;
  auto epi = [&](int t, float y, float) {
    const int lane = tid & 63, m = lane >> 4, nn = t * 16 + (lane & 15);
    if (lane < 32 && m < rm.M && nn < nqkv) ws.QKV[(size_t)m * nqkv + nn] = y * inv_rms[m];
  };
  sk_finish<false>(P, sk, gw, st.b0, st.b1, epi);
}

// ============================================================================
// Output projection + residual (+ adapter on fast rows); partial sums for the
// gate/up prologue (sum x^2, adapter-down of gate and up).
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kSkThreads) void ks_oproj(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, SkPlan P,
                                                       SkWS sk, int layer) {
  extern __shared__ __attribute__((aligned(16))) char act[];
  __shared__ float ud_s[2 * kSkThreads];
  __shared__ float uo_s[2 * kMaxRank];
  __shared__ float esc_s[kSkWaves][64];   // per-wave epilogue scratch
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, gw = blockIdx.x * kSkWaves + (tid >> 6);
  if (io.mode == EX_EXIT && sk_all_exited(rm, ws)) return;
  SkStream<WB, false> st;
  st.init(P, L.po, gw, D.qdim);
  const int HR = D.H * D.r;
  const float* r0 = ws.O;
  const float* r1 = ws.O + (size_t)(rm.M > 1 ? 1 : 0) * D.qdim;
  SkPieces xp;
  sk_load_pieces(r0, r1, nullptr, D.qdim, xp);
  // per-head adapter-down of o of both rows: element q of [2][H][r]
  float u0 = ws.uo[min(tid, 2 * HR - 1)];
  float u1 = ws.uo[min(tid + kSkThreads, 2 * HR - 1)];
  __builtin_amdgcn_sched_barrier(0);
  st.prime();
  __builtin_amdgcn_sched_barrier(0);
  const bool has_o = L.A[3] && L.B[3];
  sk_rm_copy(rmu, rm);
  __syncthreads();
  if (2 * HR <= 2 * kSkThreads) {
    ud_s[tid] = u0;
    ud_s[tid + kSkThreads] = u1;
    __syncthreads();
    if (tid < 2 * D.r) {
      const int m = tid / D.r, j = tid % D.r;
      float a = 0.f;
      if (has_o && m < rm.M && rml.fast[m]) {
#pragma unroll 8
        for (int h = 0; h < D.H; ++h) a += ud_s[(m * D.H + h) * D.r + j];
      }
      uo_s[tid] = a;
    }
  } else {
    if (tid < 2 * D.r) {
      const int m = tid / D.r, j = tid % D.r;
      float a = 0.f;
      if (has_o && m < rm.M && rml.fast[m])
        for (int h = 0; h < D.H; ++h) a += ws.uo[(m * D.H + h) * D.r + j];
      uo_s[tid] = a;
    }
  }
  sk_store_pieces<WB>(xp, r0, r1, nullptr, D.qdim, 0, 1, act);
  auto flush = [&](int t, const f32x4_t (&a)[1]) { sk_store_part<false>(P, sk, gw, t, a); };
  st.run(P, act, flush);
  float* esc = esc_s[tid >> 6];
  auto epi = [&](int t, float y, float) {
    const int lane = tid & 63, m = lane >> 4, n = lane & 15;
    const int n0 = t * 16, nn = n0 + n;
    const bool live = lane < 32 && m < rm.M;
    const int mm = live ? m : 0;
    const int sq = rsel(rm.seq, mm);
    const bool fast = rsel(rm.fast, mm) != 0;
    const int so = max(rsel(rm.slow_of, mm), 0);
    // adapter-down rows of gate and up for the gate/up prologue: lane c < 2r
    // takes row c % r of A_g (c < r) or A_u, 16 consecutive elements
    const int c = min(lane, 2 * D.r - 1);
    const void* Ac = c < D.r ? L.A[4] : L.A[5];
    u32x4_t ac[WB ? 2 : 4];
    sk_load_a16<WB>(Ac ? Ac : L.po, Ac ? (size_t)(c % D.r) * D.d + n0 : 0, ac);
    const float g16 = L.mlp_norm[n0 + (lane & 15)];
    // read everything before any write: a fast row restarting at a gate
    // reads its slow row's old value
    const float xo = ws.X[(size_t)mm * D.d + nn];
    const float xs = ws.X[(size_t)so * D.d + nn];
    const bool ex = ws.exited[sq] != 0;
    const bool ri = ws.reinit[layer * kMaxSeq + sq] != 0;
    const float ad = (fast && has_o) ? sk_dot_b<WB>(L.B[3], nn, D.r, uo_s + mm * D.r) : 0.f;
    float xnew = xo, pin = 0.f;
    if (live && !ex) {
      if (fast) {
        pin = ri ? xs : xo;
        xnew = pin + y + ad;
      } else {
        xnew = xo + y;
      }
    }
    if (live && !ex) {
      ws.X[(size_t)mm * D.d + nn] = xnew;
      if (fast) ws.PIN[(size_t)mm * D.d + nn] = pin;
    }
    // partial sums for the gate/up prologue: sum x^2 per row, and for fast
    // rows sum_n A[j][n] g_mlp[n] x[n] (lane c of the wave)
    const int bin = t % kBinSlots;
    const float xv = live ? xnew : 0.f;
    const float s2 = sum16(xv * xv);
    if (live && n == 0) add_agent(bin_o_at(ws, D, layer, bin, mm), s2);
    if (lane < 32) esc[lane] = xv * g16;
    wave_lds_sync();
    if (lane < 2 * D.r && (L.A[4] || L.A[5]) && Ac) {
      for (int r = 0; r < rm.M; ++r) {
        if (!rsel(rm.fast, r)) continue;
        const float v = sk_dot_a16<WB>(ac, esc + 16 * r);
        add_agent(bin_o_at(ws, D, layer, bin, r) + 1 + c, v);
      }
    }
    wave_lds_sync();
  };
  sk_finish<false>(P, sk, gw, st.b0, st.b1, epi);
}

// ============================================================================
// Gate/up (interleaved pairs) + adapter-up + SwiGLU; partial sums of the down
// adapter's down-projection.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kSkThreads) void ks_gateup(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, SkPlan P,
                                                        SkWS sk, int layer) {
  extern __shared__ __attribute__((aligned(16))) char act[];
  __shared__ float stat[2 * (1 + 2 * kMaxRank)];
  __shared__ float inv_rms[2];
  __shared__ float esc_s[kSkWaves][64];   // per-wave epilogue scratch
  const int tid = threadIdx.x, gw = blockIdx.x * kSkWaves + (tid >> 6);
  if (io.mode == EX_EXIT && sk_all_exited(rm, ws)) return;
  SkStream<WB, true> st;
  st.init(P, L.pg, gw, D.d);
  const int PO = 1 + 2 * D.r;
  float sv[(2 * (1 + 2 * kMaxRank) * kBinSlots + kSkThreads - 1) / kSkThreads];
  sk_bins_load(rm.M * PO, bin_o_at(ws, D, layer, 0, 0), kMaxRows * PO, sv);
  const float* r0 = ws.X;
  const float* r1 = ws.X + (size_t)(rm.M > 1 ? 1 : 0) * D.d;
  SkPieces xp;
  sk_load_pieces(r0, r1, L.mlp_norm, D.d, xp);
  __builtin_amdgcn_sched_barrier(0);
  st.prime();
  __builtin_amdgcn_sched_barrier(0);
  sk_bins_sum(rm.M * PO, sv, (float*)act, stat);
  if (tid < 2) inv_rms[tid] = rsqrtf(stat[min(tid, rm.M - 1) * PO] / D.d + D.eps);
  sk_store_pieces<WB>(xp, r0, r1, L.mlp_norm, D.d, 0, 1, act);
  auto flush = [&](int t, const f32x4_t (&a)[2]) { sk_store_part<true>(P, sk, gw, t, a); };
  st.run(P, act, flush);
  float* esc = esc_s[tid >> 6];
  auto epi = [&](int t, float yg, float yu) {
    const int lane = tid & 63, m = lane >> 4, n = lane & 15;
    const int n0 = t * 16, nn = n0 + n;
    const bool live = lane < 32 && m < rm.M;
    const int mm = live ? m : 0;
    const bool fast = rsel(rm.fast, mm) != 0;
    // the down adapter's A_d row j = lane (j < r), 16 consecutive elements
    const int j = min(lane, D.r - 1);
    u32x4_t ac[WB ? 2 : 4];
    sk_load_a16<WB>(L.A[6] ? L.A[6] : L.pg, L.A[6] ? (size_t)j * D.F + n0 : 0, ac);
    const float ir = inv_rms[mm];
    float g = yg * ir, u = yu * ir;
    const float dg = (fast && L.B[4] && L.A[4]) ? sk_dot_b<WB>(L.B[4], nn, D.r, stat + mm * PO + 1) : 0.f;
    const float du = (fast && L.B[5] && L.A[5]) ? sk_dot_b<WB>(L.B[5], nn, D.r, stat + mm * PO + 1 + D.r) : 0.f;
    g += dg * ir;
    u += du * ir;
    const float av = live ? silu(g) * u : 0.f;
    if (live) ws.ACT[(size_t)mm * D.F + nn] = av;
    if (L.A[6]) {
      const int bin = t % kBinSlots;
      if (lane < 32) esc[lane] = av;
      wave_lds_sync();
      if (lane < D.r) {
        for (int r = 0; r < rm.M; ++r) {
          if (!rsel(rm.fast, r)) continue;
          add_agent(bin_gu_at(ws, D, layer, bin, r) + j, sk_dot_a16<WB>(ac, esc + 16 * r));
        }
      }
      wave_lds_sync();
    }
  };
  sk_finish<true>(P, sk, gw, st.b0, st.b1, epi);
}

// ============================================================================
// Down projection + residual (+ adapter); partial sums for the next layer's
// norm and the exit signal.
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kSkThreads) void ks_down(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, SkPlan P,
                                                      SkWS sk, int layer) {
  extern __shared__ __attribute__((aligned(16))) char act[];
  __shared__ float ud[2 * kMaxRank];
  const int tid = threadIdx.x, gw = blockIdx.x * kSkWaves + (tid >> 6);
  if (io.mode == EX_EXIT && sk_all_exited(rm, ws)) {
    if (blockIdx.x == 0) rows_unchanged_stats(D, rm, ws, layer + 1);
    return;
  }
  SkStream<WB, false> st;
  st.init(P, L.pd, gw, D.F);
  float uv[(2 * kMaxRank * kBinSlots + kSkThreads - 1) / kSkThreads];
  sk_bins_load(rm.M * D.r, bin_gu_at(ws, D, layer, 0, 0), kMaxRows * D.r, uv);
  const float* r0 = ws.ACT;
  const float* r1 = ws.ACT + (size_t)(rm.M > 1 ? 1 : 0) * D.F;
  SkPieces xp;
  sk_load_pieces(r0, r1, nullptr, D.F, xp);
  __builtin_amdgcn_sched_barrier(0);
  st.prime();
  __builtin_amdgcn_sched_barrier(0);
  sk_bins_sum(rm.M * D.r, uv, (float*)act, ud);
  sk_store_pieces<WB>(xp, r0, r1, nullptr, D.F, 0, 1, act);
  auto flush = [&](int t, const f32x4_t (&a)[1]) { sk_store_part<false>(P, sk, gw, t, a); };
  st.run(P, act, flush);
  const bool has_d = L.A[6] && L.B[6];
  auto epi = [&](int t, float y, float) {
    const int lane = tid & 63, m = lane >> 4, n = lane & 15;
    const int nn = t * 16 + n;
    const bool live = lane < 32 && m < rm.M;
    const int mm = live ? m : 0;
    const bool fast = rsel(rm.fast, mm) != 0;
    float x = ws.X[(size_t)mm * D.d + nn];
    const float pin = fast ? ws.PIN[(size_t)mm * D.d + nn] : 0.f;
    const float bd = (fast && has_d) ? sk_dot_b<WB>(L.B[6], nn, D.r, ud + mm * D.r) : 0.f;
    const bool ex = ws.exited[rsel(rm.seq, mm)] != 0;
    if (live && !ex) {
      x += y;
      if (fast && has_d) x += bd;
      ws.X[(size_t)mm * D.d + nn] = x;
    }
    const float xv = live ? x : 0.f, pv = live ? pin : 0.f;
    const float a = sum16(xv * xv), b = sum16(pv * xv), c = sum16(pv * pv);
    if (live && n == 0) {
      float* bd = bin_d_at(ws, layer + 1, t % kBinSlots, mm);
      add_agent(bd + 0, a);
      add_agent(bd + 1, b);
      add_agent(bd + 2, c);
    }
  };
  sk_finish<false>(P, sk, gw, st.b0, st.b1, epi);
}

// ============================================================================
// Final norm + LM head + arg-max; the wave completing the last tile finishes
// the step (tokens, exit bookkeeping, acceptance of a verified chunk).
// ============================================================================
template <int WB>
__global__ __launch_bounds__(kSkThreads) void ks_head(Dims D, const void* lm_head, const float* final_norm, RowMap rm,
                                                      WS ws, StepIO io, KVPtrs kv, SkPlan P, SkWS sk,
                                                      int n_layers_run) {
  extern __shared__ __attribute__((aligned(16))) char act[];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int hrow[2];
  __shared__ int nh_s;
  __shared__ float inv_rms[2];
  __shared__ int ex_in[kMaxSeq];
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, gw = blockIdx.x * kSkWaves + (tid >> 6);
  SkStream<WB, false> st;
  st.init(P, lm_head, gw, D.d);
  float bv[1];
  sk_bins_load(rm.M * 4, bin_d_at(ws, n_layers_run, 0, 0), kMaxRows * 4, bv);
  const int exv = ws.exited[min(tid, rm.nseq - 1)];
  const float* r0 = ws.X;
  const float* r1 = ws.X + (size_t)(rm.M > 1 ? 1 : 0) * D.d;
  SkPieces xp;
  sk_load_pieces(r0, r1, final_norm, D.d, xp);
  __builtin_amdgcn_sched_barrier(0);
  st.prime();
  __builtin_amdgcn_sched_barrier(0);
  if (tid < rm.nseq) ex_in[tid] = exv;
  sk_rm_copy(rmu, rm);
  sk_bins_sum(rm.M * 4, bv, (float*)act, ssum);
  if (tid == 0) {
    // rows fed to the head
    int nh = 0;
    if (rm.head_all) {
      for (int m = 0; m < rm.M; ++m) hrow[nh++] = m;
    } else {
#pragma unroll
      for (int sq = 0; sq < 2; ++sq) {
        if (sq >= rm.nseq) break;
        const int f = rml.first[sq], l = f + rml.cnt[sq] - 1;
        int pick = f;   // slow row
        if (rml.fast[l] && (ex_in[sq] || rml.slow_of[l] < 0)) pick = l;
        hrow[sq] = pick;
        ++nh;
      }
    }
    nh_s = nh;
    for (int k = 0; k < 2; ++k) {
      const int hr = hrow[min(k, nh - 1)];
      inv_rms[k] = rsqrtf(ssum[hr * 4] / D.d + D.eps);
    }
  }
  __syncthreads();
  const int nh = nh_s;
  sk_store_pieces<WB>(xp, r0, r1, final_norm, D.d, hrow[0], hrow[min(1, nh - 1)], act);
  auto flush = [&](int t, const f32x4_t (&a)[1]) { sk_store_part<false>(P, sk, gw, t, a); };
  st.run(P, act, flush);
  const int lane = tid & 63;
  auto epi = [&](int t, float y, float) {
    const int k = lane >> 4, n = lane & 15, nn = t * 16 + n;
    const bool live = lane < 32 && k < nh;
    float z = y * inv_rms[min(k, 1)];
    if (nn >= D.V || !live) z = -INFINITY;
    else if (io.logits_out) io.logits_out[(size_t)k * D.V + nn] = z;
    int idx = nn;
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) {
      const float z2 = __shfl_xor(z, o);
      const int i2 = __shfl_xor(idx, o);
      if (z2 > z || (z2 == z && i2 < idx)) { z = z2; idx = i2; }
    }
    if (live && n == 0) {
      st_agent(&ws.lm_val[(size_t)t * kMaxRows + k], z);
      st_agent(&ws.lm_idx[(size_t)t * kMaxRows + k], idx);
    }
  };
  sk_finish<false>(P, sk, gw, st.b0, st.b1, epi);
  if (st.b0 >= st.b1) return;
  const int n_active = (int)(((long long)P.ntiles * P.nblk + P.L - 1) / P.L);
  if (!sk_arrive_all(sk, gw, n_active)) return;

  // ---- the last tile: global arg-max per head row, then bookkeeping ---------
  int best[2] = {0, 0};
  for (int k = 0; k < nh; ++k) {
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int t0 = 0; t0 < P.ntiles; t0 += 64 * 16) {   // 16 loads per lane in flight at a time
      float zv[16];
      int iv[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int t = min(t0 + lane + 64 * u, P.ntiles - 1);
        zv[u] = ld_agent(&ws.lm_val[(size_t)t * kMaxRows + k]);
        iv[u] = ld_agent(&ws.lm_idx[(size_t)t * kMaxRows + k]);
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (zv[u] > bz || (zv[u] == bz && iv[u] < bi)) { bz = zv[u]; bi = iv[u]; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float z2 = __shfl_xor(bz, o);
      const int i2 = __shfl_xor(bi, o);
      if (z2 > bz || (z2 == bz && i2 < bi)) { bz = z2; bi = i2; }
    }
    best[k] = bi;
  }
  if (rm.head_all) {
    // chunk verification / prefill (one sequence, at most two rows)
    if (lane == 0) {
      const int t = io.positions[0];
      for (int k = 0; k < nh; ++k) io.targets[k] = best[k];
      int keep = nh;
      if (io.n_acc) {
        int j = 0;
        while (j < nh - 1 && io.tokens[j + 1] == best[j]) ++j;
        io.n_acc[0] = j;
        if (io.bonus) io.bonus[0] = best[j];
        keep = j + 1;
      }
      kv.seq_lens[0] = t + keep;
      io.positions[0] = t + keep;
    }
    return;
  }
  // decode step / draft step (one head row per sequence)
  if (lane < rm.nseq) {
    const int sq = lane;
    const int f = rm.first[sq] + rm.cnt[sq] - 1;
    io.next_token[sq + io.draft_slot] = best[sq];
    const int t = io.positions[sq] + rm.pos_offset;
    if (rsel(rm.slow_of, f) >= 0 || !rsel(rm.fast, f)) kv.seq_lens[sq] = t + 1;
    if (rsel(rm.fast, f) && rsel(rm.slow_of, f) >= 0) {
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      ws.sig[sq * D.n_layers + D.n_layers - 1] = ws.exited[sq] ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
    }
    if (io.exit_b_out) io.exit_b_out[sq] = ws.exitb[sq];
    if (io.advance) io.positions[sq] = io.positions[sq] + 1;
  }
  if (io.signal_out) {
    for (int q = lane; q < rm.nseq * D.n_layers; q += 64) {
      const int sq = q / D.n_layers, l = q % D.n_layers;
      const int f = rm.first[sq] + rm.cnt[sq] - 1;
      float v = ws.sig[q];
      if (l == D.n_layers - 1) {   // written above by another lane: recomputed here
        const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
        v = ws.exited[sq] ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
      }
      if (!rsel(rm.fast, f) || rsel(rm.slow_of, f) < 0 || (ws.exited[sq] && l >= ws.exitb[sq])) v = 0.f;
      io.signal_out[q] = v;
    }
  }
  if (io.h_out || io.p_out) {
    for (int q = lane; q < rm.nseq * D.d; q += 64) {
      const int sq = q / D.d, i = q % D.d;
      const int f = rm.first[sq], c = rm.cnt[sq];
      if (io.h_out) io.h_out[q] = ws.X[(size_t)f * D.d + i];
      if (io.p_out) io.p_out[q] = ws.X[(size_t)(f + c - 1) * D.d + i];
    }
  }
}

}  // namespace m2r2
