// One-launch decode step for one sequence (one or two rows: the slow row h
// of Eq. 1 and the fast row p of Eq. 2, plain decoding, or a draft pass of
// the fast row alone): every layer's phases -- q/k/v projections, shared-KV
// attention (Sec. 2.2), output projection, gate/up and down projections --
// and the final norm, LM head and arg-max run in one persistent launch of
// one 8-wave workgroup per compute unit.
//
// Why: a decode step at batch 1 streams every weight once and does about two
// flops per byte, so the HBM stream is the roofline.  Run as one kernel per
// phase, every phase pays a start (launch, prologue, the first activation
// bytes arriving several microseconds after the first weight request) and a
// tail (waves finishing at different times) during which the HBM pipe is
// partly idle.  Here the phases are separated by a split grid barrier
// instead: a workgroup that has finished a phase counts itself in (arrive),
// then requests the first weight units of the next phase into registers
// (they do not depend on the phase still running elsewhere), and only then
// waits for the others.  The weights are in flight across the barrier.
//
// Data that one phase hands to the next (residual rows, q/k/v, attention
// output, SwiGLU activations) is written with agent-scope stores and read
// with agent-scope loads (sc1: coherent across the XCDs' L2 caches).  Row
// statistics that a phase needs over a whole row (sum of squares for the
// RMSNorm, the exit signal's dot products, the adapters' down-projections)
// are written by every workgroup into its own slot and summed by each
// consumer in one fixed order: the step is deterministic, run to run.
//
// The grid barrier polls its group flags with a time limit: if
// the workgroups were not all resident (they are, one per compute unit, when
// nothing else runs), every wave gives up after the limit, sets device error
// bit 16 and runs to the end, so the launch always drains.
#pragma once
#include "rw_kernels.h"

namespace m2r2 {

constexpr int kPkWaves = 8;
constexpr int kPkThreads = 64 * kPkWaves;
constexpr int kPkMaxWG = 320;            // statistics slots are sized for up to 320 workgroups
constexpr int kPkSdW = 8;                // slot floats of the layer-input statistics: rows 0, 1 x (x^2, pin.x, pin^2, 0)
constexpr int kPkChunk = 128;            // attention tokens per chunk (4 lanes per token)
constexpr int kPkMaxSplits = 32;         // attention splits per head
constexpr uint64_t kPkSpinTicks = 200000000ull;   // grid-barrier time limit: 2 s of the 100 MHz clock

// 1 KB pieces per row -> (pieces per sub-unit, sub-units per row)
template <int N>
struct PkPc {
  static constexpr int NCH = N > 8 ? 8 : N;
  static constexpr int NS = N > 8 ? N / 8 : 1;
};

constexpr int kPkRelStride = 32;   // uint32 words between barrier words (128 bytes)

constexpr int kPkGroups = 8;       // arrival groups of the grid barrier

struct PkBar {
  uint32_t* ctr;    // [kPkGroups][kPkRelStride] arrivals of each group in this launch
  uint32_t* flag;   // [kPkGroups][kPkRelStride] epoch of each group's last completed count
};

struct PkArgs {
  Dims D;
  const LayerPtrs* layers;   // device array [n_layers]
  const void* embed;
  const void* lm_head;       // row-major [V][d]
  const float* final_norm;
  RowMap rm;
  WS ws;
  StepIO io;
  KVPtrs kv;
  float* sd;                 // [kPkSdW/4][G][4] rows' x^2, pin.x, pin^2 leaving the down projection
  float* so;                 // [so_w/4][G][4] x^2 of rows 0, 1 after the o projection; gate, up adapter-down (fast row)
  float* sgu;                // [sgu_w/4][G][4] down adapter-down of the fast row
  PkBar bar;                 // grid barrier: group counters and flags, zero at launch, reset by the last workgroup
  int n_layers_run;
  int S;                     // attention splits per head
  int so_w, sgu_w;
};

// ---------------------------------------------------------------------------
// Coherent (agent-scope) 16-byte loads through a buffer resource: the base is
// uniform, the byte offset per lane.
// ---------------------------------------------------------------------------
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pk_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}
__device__ __forceinline__ float4 pk_ld4(__amdgpu_buffer_rsrc_t rs, int byte_off) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(rs, byte_off, 0, 16 /* sc1 */);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]), __uint_as_float(v[3]));
}

// ---------------------------------------------------------------------------
// Split grid barrier over arrival groups.  Workgroup b belongs to group
// b % kPkGroups (under the default dispatch, one group per XCD).  Arrival:
// one agent-scope atomic add on the group's counter; the workgroup whose add
// completes its group's count for this epoch stores the epoch into the
// group's flag.  Waiting: one wave polls the kPkGroups flags (one 128-byte
// line each) until all have reached the epoch.  Measured on this chip with
// no work between barriers: 2.0 us per barrier, against 4.2 us for one
// counter over all workgroups whose last arriver releases every workgroup
// (same-address atomics serialise at the memory side, and the release is a
// second round trip).
// ---------------------------------------------------------------------------
// Count this workgroup in once every wave's stores are complete; `epoch` is
// the barrier's number in the launch (1, 2, ...), so a group's count
// completes at epoch * (its size) arrivals.
__device__ __forceinline__ void pk_arrive(const PkBar& b, uint32_t epoch) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const int g = blockIdx.x % kPkGroups;
    const uint32_t per = (gridDim.x - g + kPkGroups - 1) / kPkGroups;
    const uint32_t old = __hip_atomic_fetch_add(&b.ctr[g * kPkRelStride], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (old == epoch * per - 1)
      __hip_atomic_store(&b.flag[g * kPkRelStride], epoch, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}
// Wait until every group's flag has reached `epoch` (or the time limit).
__device__ __forceinline__ void pk_wait(const PkBar& b, uint32_t epoch, int* err, int* broken) {
  if (threadIdx.x < 64 && !*broken) {
    const int ng = min(kPkGroups, (int)gridDim.x);
    const uint64_t t0 = wall_clock64();
    while (true) {
      const bool ok = (int)threadIdx.x >= ng ||
                      __hip_atomic_load(&b.flag[threadIdx.x * kPkRelStride], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= epoch;
      if (__all(ok)) break;
      if (wall_clock64() - t0 > kPkSpinTicks) {   // uniform: the clock is a scalar read
        if (threadIdx.x == 0) {
          atomicOr(err, 16);
          *broken = 1;
        }
        break;
      }
    }
  }
  __syncthreads();
}

// out[0..C) = sum over the G workgroup slots of column c, in one fixed order
// (the same in every workgroup and every run).  C is a multiple of 4, at most
// 64.  Layout: with T (the workgroup slots) column c of slot s at
// ((c / 4) G + s) 4 + c % 4, so that the lanes of a wave read consecutive
// slots' float4 from one contiguous run (a slot per 16 bytes, not one cache
// line per lane); without T at s C + c.  red holds kPkWaves float4.  Ends
// with a workgroup barrier.
template <bool T>
__device__ __forceinline__ void pk_slot_sum(const float* slots, int G, int C, float* red, float* out) {
  const int C4 = C / 4;
  int tpc = 1;   // threads per float4 column: a power of two, 32 or 64 for C <= 64 (no cross-wave step)
  while (tpc < 64 && 2 * tpc * C4 <= kPkThreads) tpc *= 2;
  const int t = threadIdx.x, c = t / tpc, j = t % tpc;
  const __amdgpu_buffer_rsrc_t rs = pk_rsrc(slots);
  constexpr int NL = kPkMaxWG / 32;
  float4 v[NL];
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int s = j + i * tpc;
    v[i] = (c < C4 && s < G) ? pk_ld4(rs, (T ? (c * G + s) * 4 : s * C + 4 * c) * 4) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  float4 a = v[0];
#pragma unroll
  for (int i = 1; i < NL; ++i) {
    a.x += v[i].x; a.y += v[i].y; a.z += v[i].z; a.w += v[i].w;
  }
  // within a row of 16 lanes by DPP, across rows by lane exchanges
  a.x = row_sum16(a.x); a.y = row_sum16(a.y); a.z = row_sum16(a.z); a.w = row_sum16(a.w);
  const int tl = tpc < 64 ? tpc : 64;
  for (int o = 16; o < tl; o <<= 1) {
    a.x += __shfl_xor(a.x, o);
    a.y += __shfl_xor(a.y, o);
    a.z += __shfl_xor(a.z, o);
    a.w += __shfl_xor(a.w, o);
  }
  if (tpc > 64) {
    const int wpc = tpc / 64;   // waves per column
    if ((t & 63) == 0) ((float4*)red)[t >> 6] = a;
    __syncthreads();
    if (t < C4) {
      float4 s = ((float4*)red)[t * wpc];
      for (int w = 1; w < wpc; ++w) {
        const float4 b = ((float4*)red)[t * wpc + w];
        s.x += b.x; s.y += b.y; s.z += b.z; s.w += b.w;
      }
      ((float4*)out)[t] = s;
    }
  } else if (j == 0 && c < C4) {
    ((float4*)out)[c] = a;
  }
  __syncthreads();
}

// Activation rows at float offsets off0, off1 of `base` (coherent loads) and
// the gain (plain loads) into registers; rw_store_pieces puts them in LDS.
template <int PM>
__device__ __forceinline__ void pk_load_rows(const float* base, int off0, int off1, const float* gain, int K,
                                             RwPieces<PM>& xp) {
  const __amdgpu_buffer_rsrc_t rs = pk_rsrc(base);
  const int nq = K / 4;
#pragma unroll
  for (int p = 0; p < PM; ++p) {
    const int q = rw_piece_q<kPkThreads>(p, nq);
    xp.v[p][0] = pk_ld4(rs, (off0 + 4 * q) * 4);
    xp.v[p][1] = pk_ld4(rs, (off1 + 4 * q) * 4);
    if (gain) xp.g[p] = ldg4(gain + 4 * q);
  }
}

// Sum over the workgroup of one value per wave lane (lane i of every wave
// holds value i, i < n) into the G-slot array `slot` at [blockIdx][o + i],
// with agent-scope stores.
// Column k of this workgroup's slot in a [C/4][G][4] slot array.
__device__ __forceinline__ float* pk_slot_at(float* slots, int k) {
  return slots + (((size_t)(k >> 2) * gridDim.x + blockIdx.x) << 2) + (k & 3);
}
template <int NW>
__device__ __forceinline__ void pk_wg_store(float v, int n, float* scratch, float* tot, float* slots, int k0) {
  rw_wg_sum<NW>(v, n, scratch, tot);
  if ((int)threadIdx.x < n) st_agent(pk_slot_at(slots, k0 + (int)threadIdx.x), tot[threadIdx.x]);
}

// ---------------------------------------------------------------------------
// Epilogues (one output unit of a wave; y[0][m] = dot product with staged row m)
// ---------------------------------------------------------------------------
struct PkQkvEpi {
  struct Ops {};
  int M;
  const int* src;
  const float* ir;
  float* QKV;
  int nqkv, qd, r;
  int has;   // bit w: adapter w (q, k, v) present
  __device__ void fetch(int, Ops&) const {}
  __device__ void run(int u, const float (&y)[1][2], const Ops&) const {
    const int lane = threadIdx.x & 63;
    if (lane < M) {
      float v = y[0][src[lane]] * ir[lane];
      if (u >= 3 * qd) {
        const int w = (u - 3 * qd) / r;
        if (!((has >> w) & 1)) v = 0.f;
      }
      st_agent(&QKV[(size_t)lane * nqkv + u], v);
    }
  }
};

template <int WB>
struct PkOEpi {
  struct Ops {
    float x0, x1, g;
    typename RwRaw<WB>::type a;   // A_g[c][n] (c < r) or A_u[c - r][n] of this lane's c
    RwBRow<WB> b;
  };
  int d, r;
  const float* mlp_norm;
  const void* Ag;    // gate adapter down-factor (may be null)
  const void* Au;    // up adapter down-factor (may be null)
  const void* Bo;    // o adapter up-factor (used when has_o)
  const RowMap* rm;
  const float* uo;   // [r] o-adapter down-projection of the fast row
  WS ws;
  int fm, ri;        // fast row (-1: none); p restarts from h at this layer
  bool has_o;
  float accx, accf;
  __device__ void fetch(int n, Ops& o) const {
    const int lane = threadIdx.x & 63;
    o.x0 = ld_agent(&ws.X[n]);
    o.x1 = ld_agent(&ws.X[(size_t)d + n]);
    o.g = mlp_norm[n];
    const int c = lane % (2 * r);
    const void* A = c < r ? Ag : Au;
    o.a = rw_wt_raw<WB>(A ? A : (const void*)mlp_norm, A ? (size_t)(c % r) * d + n : 0);
    o.b.load(has_o ? Bo : (const void*)mlp_norm, has_o ? n : 0, r);
  }
  __device__ void run(int n, const float (&y)[1][2], const Ops& o) {
    const int lane = threadIdx.x & 63;
    float xnew[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      xnew[m] = 0.f;
      if (m >= rm->M) continue;
      const bool fast = rm->fast[m] != 0;
      const float xo = m ? o.x1 : o.x0;
      const float xs = rm->slow_of[m] == 1 ? o.x1 : o.x0;
      float xn, pin = 0.f;
      if (fast) {
        pin = ri ? xs : xo;
        xn = pin + y[0][m] + (has_o ? o.b.dot(uo, r) : 0.f);
      } else {
        xn = xo + y[0][m];
      }
      if (lane == m) {
        st_agent(&ws.X[(size_t)m * d + n], xn);
        if (fast) st_agent(&ws.PIN[(size_t)m * d + n], pin);
      }
      xnew[m] = xn;
    }
    accx += lane == 0 ? xnew[0] * xnew[0] : (lane == 1 ? xnew[1] * xnew[1] : 0.f);
    if (fm >= 0) accf += rw_wt<WB>(o.a) * o.g * xnew[fm];
  }
};

template <int WB>
struct PkGuEpi {
  struct Ops {
    typename RwRaw<WB>::type a;   // A_d[lane % r][j]
    RwBRow<WB> bg, bu;
  };
  int F, r;
  const float* fb;   // a valid stand-in address for absent factors
  const void* Ad;    // down adapter down-factor (may be null)
  const void* Bg;    // gate adapter up-factor (used when hg)
  const void* Bu;    // up adapter up-factor (used when hu)
  const RowMap* rm;
  const float* stat;   // [2 + 2r]: x^2 of rows 0, 1; gate and up adapter-down of the fast row
  const float* ir;
  WS ws;
  int fm;
  bool hg, hu;
  float yg0, yg1;
  float accf;
  __device__ void fetch(int h, Ops& o) const {
    const int lane = threadIdx.x & 63, j = h >> 1;
    o.a = rw_wt_raw<WB>(Ad ? Ad : (const void*)fb, Ad ? (size_t)(lane % r) * F + j : 0);
    o.bg.load(hg ? Bg : (const void*)fb, hg ? j : 0, r);
    o.bu.load(hu ? Bu : (const void*)fb, hu ? j : 0, r);
  }
  __device__ void run(int h, const float (&y)[1][2], const Ops& o) {
    if (!(h & 1)) {
      yg0 = y[0][0];
      yg1 = y[0][1];
      return;
    }
    const int lane = threadIdx.x & 63, j = h >> 1;
    float av[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      av[m] = 0.f;
      if (m >= rm->M) continue;
      float g = (m ? yg1 : yg0) * ir[m], u = y[0][m] * ir[m];
      if (m == fm) {
        if (hg) g += o.bg.dot(stat + 2, r) * ir[m];
        if (hu) u += o.bu.dot(stat + 2 + r, r) * ir[m];
      }
      av[m] = silu(g) * u;
      if (lane == m) st_agent(&ws.ACT[(size_t)m * F + j], av[m]);
    }
    if (fm >= 0) accf += rw_wt<WB>(o.a) * av[fm];
  }
};

template <int WB>
struct PkDnEpi {
  struct Ops {
    float x0, x1, p0, p1;
    RwBRow<WB> b;
  };
  int d, r;
  const float* fb;   // a valid stand-in address
  const void* Bd;    // down adapter up-factor (used when hd)
  const RowMap* rm;
  const float* ud;   // [r] down adapter-down of the fast row
  WS ws;
  int fm;
  bool hd;
  float acc;
  __device__ void fetch(int n, Ops& o) const {
    o.x0 = ld_agent(&ws.X[n]);
    o.x1 = ld_agent(&ws.X[(size_t)d + n]);
    o.p0 = ld_agent(&ws.PIN[n]);
    o.p1 = ld_agent(&ws.PIN[(size_t)d + n]);
    o.b.load(hd ? Bd : (const void*)fb, hd ? n : 0, r);
  }
  __device__ void run(int n, const float (&y)[1][2], const Ops& o) {
    const int lane = threadIdx.x & 63;
    float xv[2], pv[2];
#pragma unroll
    for (int m = 0; m < 2; ++m) {
      xv[m] = 0.f;
      pv[m] = 0.f;
      if (m >= rm->M) continue;
      float x = (m ? o.x1 : o.x0) + y[0][m];
      if (m == fm && hd) x += o.b.dot(ud, r);
      if (lane == m) st_agent(&ws.X[(size_t)m * d + n], x);
      xv[m] = x;
      pv[m] = m == fm ? (m ? o.p1 : o.p0) : 0.f;
    }
    if (lane < 8) {   // slot layout [m * 4 + c]: x^2, pin.x, pin^2, 0
      const int m = lane >> 2, c = lane & 3;
      acc += c == 0 ? xv[m] * xv[m] : (c == 1 ? pv[m] * xv[m] : (c == 2 ? pv[m] * pv[m] : 0.f));
    }
  }
};

struct PkHeadEpi {
  struct Ops {};
  int hrow;
  float ir;
  float* logits;
  float bz;
  int bi;
  __device__ void fetch(int, Ops&) const {}
  __device__ void run(int v, const float (&y)[1][2], const Ops&) {
    const float z = y[0][hrow] * ir;
    if (logits && (threadIdx.x & 63) == 0) logits[v] = z;
    if (z > bz) { bz = z; bi = v; }   // units in increasing order: the lowest index wins ties
  }
};

// Small per-workgroup state in LDS.
struct PkShared {
  SkRmLds rmu;
  const char* base[6];   // row bases of the current phase's matrices (q, k, v, A_q, A_k, A_v; gate, up)
  float ssum[kMaxRows * 4];
  float stat[2 * kMaxRank + 8];
  float red[kPkWaves * 4];
  float wsum[kPkWaves * 64];
  float tot[64];
  float inv_rms[2];
  int src[2];
  int ex, eb, ri, broken, last_flag;
  float bz[kPkWaves];
  int bi[kPkWaves];
};

// Attention-phase arrays, carved from the dynamic LDS (the activation rows
// of the projection phases are not live during attention).
template <int HD, int WB>
struct PkAttLds {
  float q[2][HD], k[2][HD], v[2][HD];
  float u[2][3][kMaxRank];
  float sc[2][2 * kPkChunk + 2];   // a pair of chunks, then the own keys
  float pvred[32][2][HD];
  float mw[2][kPkMaxSplits], ml[2][kPkMaxSplits];
  float rowm[2], rowl[2], lastw[2], fin_m[2], fin_l[2], linv[2];
  float uop[kMaxRank * (HD / 8)];
  __attribute__((aligned(16))) char bsl[3 * HD * kMaxRank * (WB ? 2 : 4)];
};

// Dynamic LDS bytes of the step: the larger of the activation rows (two rows
// of the longest reduction) and the attention arrays.
__host__ __device__ constexpr size_t pk_lds_bytes(int hd, int wb, int kmax) {
  const size_t act = (size_t)2 * kmax * 4;
  // (the f32 layout of the attention arrays bounds the bf16 one)
  const size_t att = hd == 64 ? sizeof(PkAttLds<64, 0>) : hd == 96 ? sizeof(PkAttLds<96, 0>) : sizeof(PkAttLds<128, 0>);
  (void)wb;
  return ((act > att ? act : att) + 255) & ~(size_t)255;
}

// The step's arguments, read through an opaque pointer to the kernel-argument
// segment at the start of every phase: the compiler then cannot hoist a
// phase's argument loads and index arithmetic out of the layer loop and keep
// them live across the other phases (which made the whole step spill).
__device__ __forceinline__ const PkArgs& pk_args() {
  auto p = (const __attribute__((address_space(4))) PkArgs*)__builtin_amdgcn_kernarg_segment_ptr();
  asm volatile("" : "+s"(p));
  return *(const PkArgs*)p;
}
__device__ __forceinline__ int pk_opaque_tid() {
  int t = (int)threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// Names every phase uses.
#define PK_PROLOGUE                                                                               \
  extern __shared__ __attribute__((aligned(16))) float pk_dyn[];                                  \
  const PkArgs& P = pk_args();                                                                         \
  const Dims D = P.D;                                                                             \
  const int tid = pk_opaque_tid(), lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6); \
  const int G = gridDim.x, W = G * kPkWaves, gw = blockIdx.x * kPkWaves + wv;                    \
  const int qd = D.qdim, r = D.r, nqkv = 3 * qd + 3 * r, esz = WB ? 2 : 4, d = D.d;              \
  const int M = P.rm.M;                                                                           \
  const int fm = M > 1 ? 1 : (P.rm.fast[0] ? 0 : -1);                                            \
  const int posv = P.io.positions[0];                                                             \
  const int ctx = posv + P.rm.pos_offset;                                                         \
  const RowMap& rml = sh.rmu.rm;                                                                  \
  (void)lane; (void)W; (void)gw; (void)nqkv; (void)esz; (void)fm; (void)ctx; (void)qd; (void)r;   \
  (void)M; (void)d; (void)posv; (void)rml;

// q, k, v projections of layer l (the first waits for no one).
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__device__ __forceinline__ void pk_phase_qkv(int l, uint32_t& target, PkShared& sh) {
  PK_PROLOGUE
  using CD = PkPc<ND>;
  using CQ = PkPc<NQ>;
  using CF = PkPc<NF>;
  (void)sizeof(CD); (void)sizeof(CQ); (void)sizeof(CF);
  const LayerPtrs* Lp = P.layers + l;   // uniform: scalar loads
  (void)Lp;
    // ======================= q, k, v (+ adapter-down rows) ===================
    {
      const int nu = 3 * qd + 3 * r;
      const float* attn_norm = Lp->attn_norm;
      const bool hasA[3] = {Lp->A[0] != nullptr, Lp->A[1] != nullptr, Lp->A[2] != nullptr};
      if (tid == 0) {
        sh.base[0] = (const char*)Lp->wq;
        sh.base[1] = (const char*)Lp->wk;
        sh.base[2] = (const char*)Lp->wv;
        for (int a = 0; a < 3; ++a) sh.base[3 + a] = hasA[a] ? (const char*)Lp->A[a] : (const char*)Lp->wq;
      }
      __syncthreads();
      // unit u: row u of [Wq; Wk; Wv; A_q; A_k; A_v] (a missing adapter reads
      // any row: its result is zeroed); the bases come from LDS, whose reads
      // do not wait for the weight loads in flight
      auto row_ptr = [=, &sh](int u, int) -> const void* {
        const size_t rb = (size_t)d * esz;
        const int seg = u < 3 * qd ? u / qd : 3 + (u - 3 * qd) / r;
        const int row = u < 3 * qd ? u - seg * qd : (u - 3 * qd) % r;
        return sh.base[seg] + row * rb;
      };
      auto range = [&](bool kv_only, int& u0, int& u1) {
        if (kv_only) {
          rw_range(2 * qd, W, gw, u0, u1);
          u0 += qd;
          u1 += qd;
        } else {
          rw_range(nu, W, gw, u0, u1);
        }
      };
      const bool ex_before = sh.ex != 0 && P.io.mode == EX_EXIT;
      int u0, u1;
      range(ex_before, u0, u1);
      RwStream<WB, CD::NCH, 1, CD::NS> st;
      PkQkvEpi epi{M, sh.src, sh.inv_rms, P.ws.QKV, nqkv, qd, r, (int)hasA[0] | ((int)hasA[1] << 1) | ((int)hasA[2] << 2)};
      PkQkvEpi::Ops ops[decltype(st)::P];
      st.begin_all(row_ptr, u0, u1, epi, ops);
      // gate inputs that do not depend on the layer's statistics, read while
      // the barrier is pending (one sequence: its last row is the fast row)
      int g_f = 0, g_fast = 0, g_slow = -1, g_r0 = 0, g_r1 = 0;
      if (tid == 0) {
        g_f = rml.first[0] + rml.cnt[0] - 1;
        g_fast = rml.fast[g_f];
        g_slow = rml.slow_of[g_f];
        g_r0 = rml.fast[0] ? rml.slow_of[0] : 0;
        g_r1 = rml.fast[M - 1] ? rml.slow_of[M - 1] : M - 1;
      }
      const bool g_gate = is_gate(P.io, l);
      const int g_mode = P.io.mode;
      const float g_tau = P.io.tau;
      const float* g_asig = P.io.arla_sig;
      if (l > 0) {
        target += 1;
        pk_wait(P.bar, target, P.ws.err, &sh.broken);
      }
      constexpr int PM = RwPM<WB, CD::NCH, CD::NS, kPkThreads>::value;
      RwPieces<PM> xp;
      if (l == 0) {
        // the embedding of the step's token: both rows start from it (p <- h)
        const int tok = P.io.tokens[P.rm.tok[0]];
        const bool ok = tok >= 0 && tok < D.V;
        if (!ok && tid == 0 && blockIdx.x == 0) atomicOr(P.ws.err, 1);
        const int nq = d / 4;
        float ss = 0.f;
#pragma unroll
        for (int p = 0; p < PM; ++p) {
          const int q = rw_piece_q<kPkThreads>(p, nq);
          float4 e = make_float4(0.f, 0.f, 0.f, 0.f);
          if (ok) {
            const size_t i0 = (size_t)tok * d + 4 * q;
            if constexpr (WB) {
              const uint2 b = *(const uint2*)((const uint16_t*)P.embed + i0);
              e = make_float4(bf16lo(b.x), bf16hi(b.x), bf16lo(b.y), bf16hi(b.y));
            } else {
              e = *(const float4*)((const float*)P.embed + i0);
            }
          }
          xp.v[p][0] = e;
          xp.v[p][1] = e;
          xp.g[p] = ldg4(attn_norm + 4 * q);
          if ((int)tid + kPkThreads * p < nq) ss += e.x * e.x + e.y * e.y + e.z * e.z + e.w * e.w;
        }
        // X and PIN of every row start at the embedding (read by later phases)
        for (int q = blockIdx.x * kPkThreads + tid; q < nq; q += G * kPkThreads) {
          float4 e = make_float4(0.f, 0.f, 0.f, 0.f);
          if (ok) {
            const size_t i0 = (size_t)tok * d + 4 * q;
            if constexpr (WB) {
              const uint2 b = *(const uint2*)((const uint16_t*)P.embed + i0);
              e = make_float4(bf16lo(b.x), bf16hi(b.x), bf16lo(b.y), bf16hi(b.y));
            } else {
              e = *(const float4*)((const float*)P.embed + i0);
            }
          }
          const float ev[4] = {e.x, e.y, e.z, e.w};
          for (int m = 0; m < M; ++m)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              st_agent(&P.ws.X[(size_t)m * d + 4 * q + k], ev[k]);
              st_agent(&P.ws.PIN[(size_t)m * d + 4 * q + k], ev[k]);
            }
        }
        ss = block_sum(ss, sh.red);
        if (tid < 2 * 4) sh.ssum[tid] = (tid & 3) < 3 ? ss : 0.f;
        __syncthreads();
      } else {
        pk_load_rows<PM>(P.ws.X, 0, (M > 1 ? 1 : 0) * d, attn_norm, d, xp);
        pk_slot_sum<true>(P.sd, G, kPkSdW, sh.red, sh.ssum);
      }
      int newly = 0;
      if (tid == 0) {
        // the gate rule of sk_gate_logic for the one sequence: the exit signal
        // (cosine of the fast row's update, or the router score) decides at a
        // gate; a gate that does not exit re-initialises the fast row
        int ex = sh.ex, eb = sh.eb, ri = 0;
        float sg = 0.f;
        if (l > 0 && g_fast) {
          const float dot = sh.ssum[g_f * 4 + 1], pin2 = sh.ssum[g_f * 4 + 2], pp = sh.ssum[g_f * 4 + 0];
          sg = dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
          if (g_asig && g_gate) sg = g_asig[0];
          if (!ex && g_mode != EX_OFF && g_gate && g_slow >= 0) {
            const bool fired = sg >= g_tau;
            if (fired && eb == D.n_layers) eb = l;
            if (g_mode == EX_EXIT && fired) ex = 1;
            else ri = 1;
          }
        }
        newly = ex && !sh.ex;
        sh.ri = ri;
        sh.ex = ex;
        sh.eb = eb;
        if (blockIdx.x == 0 && l > 0) st_agent(&P.ws.sig[l - 1], sg);
        // the rows' norm sources: a re-initialised fast row takes its slow row's
        const int s0 = ri ? g_r0 : 0, s1 = ri ? g_r1 : M - 1;
        sh.src[0] = s0;
        sh.src[1] = s1;
        sh.inv_rms[0] = rsqrtf(sh.ssum[s0 * 4] / d + D.eps);
        sh.inv_rms[1] = rsqrtf(sh.ssum[s1 * 4] / d + D.eps);
        sh.last_flag = newly;
      }
      __syncthreads();
      if (sh.last_flag && P.io.mode == EX_EXIT) {
        // the sequence exits at this boundary: the layer only fills its
        // cache entries from the slow row (the units primed above are dropped)
        range(true, u0, u1);
        st.begin_all(row_ptr, u0, u1, epi, ops);
      }
      rw_store_pieces<true, PM, kPkThreads>(xp, d, pk_dyn);
      st.template run<true>(row_ptr, u0, u1, pk_dyn, d, epi, ops);
      pk_arrive(P.bar, target + 1);
    }

}

// Shared-KV attention of layer l.
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__device__ __forceinline__ void pk_phase_att(int l, uint32_t& target, PkShared& sh) {
  PK_PROLOGUE
  using CD = PkPc<ND>;
  using CQ = PkPc<NQ>;
  using CF = PkPc<NF>;
  (void)sizeof(CD); (void)sizeof(CQ); (void)sizeof(CF);
  const LayerPtrs* Lp = P.layers + l;   // uniform: scalar loads
  (void)Lp;
    // ======================= shared-KV attention =============================
    {
      constexpr int DPL = HD / 4;                  // dims per lane, 4 lanes per token
      constexpr int KESZ = KB ? 2 : 4;
      constexpr int NCH = DPL * KESZ / 16;         // 16-byte pieces per lane and token
      constexpr int WESZ = WB ? 2 : 4;
      PkAttLds<HD, WB>& A = *(PkAttLds<HD, WB>*)pk_dyn;
      const int S = P.S, H = D.H;
      const int task = blockIdx.x;
      const bool has = task < H * S;
      const int h = has ? task / S : 0, sp = has ? task % S : 0;
      const int slot = tid >> 2, sub = tid & 3, d0 = sub * DPL;
      const float scale = rsqrtf((float)HD);
      const int Tn = (ctx + S - 1) / S;
      const int t0 = min(ctx, sp * Tn), t1 = min(ctx, t0 + Tn);
      const int nch = max(1, (t1 - t0 + kPkChunk - 1) / kPkChunk);
      const bool own = sp == S - 1;
      const int R = M;
      const bool frozen = sh.ex != 0;
      const KVPtrs& kv = P.kv;
      const void* LB[3] = {Lp->B[0], Lp->B[1], Lp->B[2]};
      const bool LA[3] = {Lp->A[0] != nullptr, Lp->A[1] != nullptr, Lp->A[2] != nullptr};
      const void* Ao = Lp->A[3];
      // ---- primed before the barrier: keys/values of the first two chunks,
      // the head's adapter up-factor rows, A_o columns, the RoPE entries
      auto blk_of = [&](int tp) {
        int b = kv.bt[min(max(tp, 0) / kv.bs, kv.mbps - 1)];
        return (b >= 0 && b < kv.num_blocks) ? b : 0;
      };
      auto load_chunk = [&](const void* base, int ch, u32x4_t (&dst)[NCH]) {
        const int tp = t0 + ch * kPkChunk + slot;
        const int b = blk_of(tp);
        const size_t ix = ((((size_t)l * kv.num_blocks + b) * H + h) * kv.bs + max(tp, 0) % kv.bs) * HD + d0;
#pragma unroll
        for (int c = 0; c < NCH; ++c) dst[c] = *(const u32x4_t*)((const char*)base + ix * KESZ + 16 * c);
      };
      u32x4_t kr[2][NCH], vr[2][NCH];
      const bool work = has && !frozen;
      if (work) {
        load_chunk(kv.k, 0, kr[0]);
        load_chunk(kv.v, 0, vr[0]);
        load_chunk(kv.k, min(1, nch - 1), kr[1]);
        load_chunk(kv.v, min(1, nch - 1), vr[1]);
      }
      const int ppieces = HD * r * WESZ / 16;   // 16-byte pieces per projection (<= 2 per thread)
      u32x4_t bp[3][2];
#pragma unroll
      for (int w = 0; w < 3; ++w) {
        const u32x4_t* B = (const u32x4_t*)((const char*)(LB[w] ? LB[w] : (const void*)P.ws.QKV) +
                                            (size_t)h * HD * r * WESZ);
#pragma unroll
        for (int k = 0; k < 2; ++k) {
          const int o = min(tid + kPkThreads * k, ppieces - 1);
          bp[w][k] = (LB[w] && has) ? B[o] : u32x4_t{0u, 0u, 0u, 0u};
        }
      }
      const int apieces = r * HD / 8;
      u32x4_t ap = u32x4_t{0u, 0u, 0u, 0u};
      {
        const int i = min(tid, apieces - 1);
        const int j = i / (HD / 8), c = i % (HD / 8);
        if (WB && Ao && has) ap = *(const u32x4_t*)((const uint16_t*)Ao + (size_t)j * qd + h * HD + 8 * c);
      }
      const int e_m = min(tid / HD, 1), e_d = tid % HD;
      float2 cs;
      {
        int pos = ctx + rml.idx[min(e_m, M - 1)];
        if (pos < 0 || pos >= P.ws.rope_len) {
          if (tid == 0 && has) atomicOr(P.ws.err, 8);
          pos = 0;
        }
        cs = P.ws.rope[(size_t)pos * (HD / 2) + (e_d % (HD / 2))];
      }
      target += 1;
      pk_wait(P.bar, target, P.ws.err, &sh.broken);
      if (has) {
        // ---- projections of this head (coherent loads)
        float pv[3];
        {
          const int row = min(e_m, M - 1);
#pragma unroll
          for (int w = 0; w < 3; ++w) pv[w] = ld_agent(&P.ws.QKV[(size_t)row * nqkv + w * qd + h * HD + e_d]);
        }
        float uv;
        {
          const int q = min(tid, 2 * 3 * r - 1);
          const int row = min(q / (3 * r), M - 1);
          uv = ld_agent(&P.ws.QKV[(size_t)row * nqkv + 3 * qd + q % (3 * r)]);
        }
#pragma unroll
        for (int w = 0; w < 3; ++w)
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            const int o = tid + kPkThreads * k;
            if (o < ppieces) ((u32x4_t*)A.bsl)[w * ppieces + o] = bp[w][k];
          }
        if (tid < 2 * 3 * r) A.u[tid / (3 * r)][(tid % (3 * r)) / r][tid % r] = uv;
        __syncthreads();
        // q, k, v: base projection plus the adapter up-projection on the fast row
        const bool erow = tid < R * HD;
        const bool efast = erow && rml.fast[e_m];
        float pre[3];
#pragma unroll
        for (int w = 0; w < 3; ++w) {
          float a = pv[w];
          if (efast && LA[w] && LB[w]) {
            const char* br = A.bsl + ((size_t)w * HD + e_d) * r * WESZ;
            for (int j = 0; j < r; ++j) {
              const float b = WB ? bf16_to_f32(((const uint16_t*)br)[j]) : ((const float*)br)[j];
              a += b * A.u[e_m][w][j];
            }
          }
          pre[w] = a;
        }
        if (erow) {
          A.q[e_m][e_d] = pre[0];
          A.k[e_m][e_d] = pre[1];
          A.v[e_m][e_d] = pre[2];
        }
        __syncthreads();
        float qr = 0.f, krr = 0.f;
        if (erow) {
          const int half = HD / 2, j = e_d % half;
          const float c = cs.x, sn = cs.y;
          const float qa = A.q[e_m][j], qb = A.q[e_m][j + half];
          const float ka = A.k[e_m][j], kb = A.k[e_m][j + half];
          qr = e_d < half ? qa * c - qb * sn : qb * c + qa * sn;
          krr = e_d < half ? ka * c - kb * sn : kb * c + ka * sn;
        }
        __syncthreads();
        if (erow) {
          A.q[e_m][e_d] = qr;
          A.k[e_m][e_d] = krr;
        }
        __syncthreads();
        // ---- the own split writes the slow rows' key/value to the cache
        if (own && erow && rml.wr[e_m]) {
          const int pos = ctx + rml.idx[e_m];
          const int lb = pos / kv.bs;
          const bool okb = pos >= 0 && lb < kv.mbps;
          const int b = okb ? kv.bt[lb] : -1;
          if (!okb || b < 0 || b >= kv.num_blocks) {
            atomicOr(P.ws.err, 2);
          } else {
            const size_t ix = ((((size_t)l * kv.num_blocks + b) * H + h) * kv.bs + pos % kv.bs) * HD + e_d;
            if (KB) {
              ((uint16_t*)kv.k)[ix] = (uint16_t)f32_to_bf16_bits(A.k[e_m][e_d]);
              ((uint16_t*)kv.v)[ix] = (uint16_t)f32_to_bf16_bits(A.v[e_m][e_d]);
            } else {
              ((float*)kv.k)[ix] = A.k[e_m][e_d];
              ((float*)kv.v)[ix] = A.v[e_m][e_d];
            }
          }
        }
      }
      if (work) {
        float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
        float acc0[DPL], acc1[DPL];
#pragma unroll
        for (int c = 0; c < DPL; ++c) { acc0[c] = 0.f; acc1[c] = 0.f; }
        // Chunks are taken in pairs (ch, ch + 1): every thread slot scores one
        // token of each, one softmax covers both and their P V is summed in
        // one pass (a split of 129..256 positions costs one pass, not two).
        // Pairs combine online (running max, sum and accumulator per row).
        auto scores = [&](int ch, u32x4_t (&kb)[NCH], int off) {
          const int c0 = t0 + ch * kPkChunk;
          const int nt = max(0, min(t1, c0 + kPkChunk) - c0);
          float kk[DPL];
#pragma unroll
          for (int c = 0; c < NCH; ++c) {
            if constexpr (KB) {
#pragma unroll
              for (int i = 0; i < 4; ++i) { kk[8 * c + 2 * i] = bf16lo(kb[c][i]); kk[8 * c + 2 * i + 1] = bf16hi(kb[c][i]); }
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) kk[4 * c + i] = __uint_as_float(kb[c][i]);
            }
          }
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            float p = 0.f;
#pragma unroll
            for (int c = 0; c < DPL; ++c) p += A.q[i][d0 + c] * kk[c];
            p = quad_sum(p);
            if (sub == 0 && i < R) A.sc[i][off + slot] = slot < nt ? p * scale : -INFINITY;
          }
        };
        auto pv = [&](u32x4_t (&vb)[NCH], float p0, float p1) {
#pragma unroll
          for (int c = 0; c < NCH; ++c) {
            if constexpr (KB) {
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const float a = bf16lo(vb[c][i]), b = bf16hi(vb[c][i]);
                acc0[8 * c + 2 * i] += p0 * a; acc0[8 * c + 2 * i + 1] += p0 * b;
                acc1[8 * c + 2 * i] += p1 * a; acc1[8 * c + 2 * i + 1] += p1 * b;
              }
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const float a = __uint_as_float(vb[c][i]);
                acc0[4 * c + i] += p0 * a;
                acc1[4 * c + i] += p1 * a;
              }
            }
          }
        };
        constexpr int kOwn = 2 * kPkChunk;   // sc index of the own keys
        for (int ch = 0; ch < nch; ch += 2) {
          const bool two = ch + 1 < nch;
          const bool last = ch + 2 >= nch;
          scores(ch, kr[0], 0);
          if (two) {
            scores(ch + 1, kr[1], kPkChunk);
          } else if (sub == 0) {
            A.sc[0][kPkChunk + slot] = -INFINITY;
            A.sc[1][kPkChunk + slot] = -INFINITY;
          }
          // the next pair's keys are in flight during this pair's softmax and P V
          if (ch + 2 < nch) load_chunk(kv.k, ch + 2, kr[0]);
          if (ch + 3 < nch) load_chunk(kv.k, ch + 3, kr[1]);
          // own keys (own split, last pair): a slow row sees the slow row (its
          // own key, rounded as cached); a fast row only its own exact key
          if (own && last && wv < 4) {
            const int i = wv >> 1, jj = wv & 1;
            if (i < R) {
              const bool vis = jj < R && (rml.fast[i] ? (jj == i) : (!rml.fast[min(jj, R - 1)] &&
                                                                     rml.idx[min(jj, R - 1)] <= rml.idx[i]));
              const bool rnd = !rml.fast[i];
              float p = 0.f;
              for (int dd = lane; dd < HD; dd += 64) {
                const float kk = A.k[min(jj, R - 1)][dd];
                p += A.q[i][dd] * (rnd && KB ? round_bf16(kk) : kk);
              }
              p = wave_sum(p);
              if (lane == 0) A.sc[i][kOwn + jj] = vis ? p * scale : -INFINITY;
            }
          } else if (tid < 4) {
            A.sc[tid >> 1][kOwn + (tid & 1)] = -INFINITY;
          }
          __syncthreads();
          if (wv < R) {
            const int i = wv;
            float mx = -INFINITY;
            for (int j = lane; j < kOwn + 2; j += 64) mx = fmaxf(mx, A.sc[i][j]);
            mx = wave_max(mx);
            float ls = 0.f;
            for (int j = lane; j < kOwn + 2; j += 64) {
              const float z = A.sc[i][j];
              const float ev = z == -INFINITY ? 0.f : __expf(z - mx);
              A.sc[i][j] = ev;
              ls += ev;
            }
            ls = wave_sum(ls);
            if (lane == 0) { A.rowm[i] = ls > 0.f ? mx : -INFINITY; A.rowl[i] = ls; }
          }
          __syncthreads();
          float wc[2];
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            const float mc = A.rowm[min(i, R - 1)], lc = A.rowl[min(i, R - 1)];
            const float mn = fmaxf(m_run[i], mc);
            const float wr = m_run[i] == -INFINITY ? 0.f : __expf(m_run[i] - mn);
            wc[i] = mc == -INFINITY ? 0.f : __expf(mc - mn);
            l_run[i] = l_run[i] * wr + lc * wc[i];
            m_run[i] = mn;
#pragma unroll
            for (int c = 0; c < DPL; ++c) {
              if (i == 0) acc0[c] *= wr;
              else acc1[c] *= wr;
            }
          }
          pv(vr[0], A.sc[0][slot] * wc[0], R > 1 ? A.sc[1][slot] * wc[1] : 0.f);
          if (two) pv(vr[1], A.sc[0][kPkChunk + slot] * wc[0], R > 1 ? A.sc[1][kPkChunk + slot] * wc[1] : 0.f);
          if (ch + 2 < nch) load_chunk(kv.v, ch + 2, vr[0]);
          if (ch + 3 < nch) load_chunk(kv.v, ch + 3, vr[1]);
          if (!last) {
            __syncthreads();   // the next pair's scores overwrite sc
          } else if (tid < 2) {
            A.lastw[tid] = wc[tid];
          }
        }
        if (tid < 2) { A.fin_m[tid] = m_run[tid]; A.fin_l[tid] = l_run[tid]; }
        // sum over the 4 token slots of a 16-lane row (DPP), then the 32 row
        // partials (4 rows x 8 waves) through LDS
#pragma unroll
        for (int c = 0; c < DPL; ++c) {
          acc0[c] = row_sum_stride4(acc0[c]);
          acc1[c] = row_sum_stride4(acc1[c]);
        }
        if ((lane & 15) < 4) {
          const int g = wv * 4 + (lane >> 4);
#pragma unroll
          for (int c = 0; c < DPL; ++c) {
            A.pvred[g][0][d0 + c] = acc0[c];
            A.pvred[g][1][d0 + c] = acc1[c];
          }
        }
        __syncthreads();
        for (int e = tid; e < R * HD; e += kPkThreads) {
          const int i = e / HD, dd = e % HD;
          float a = 0.f;
#pragma unroll 8
          for (int g = 0; g < 32; ++g) a += A.pvred[g][i][dd];
          if (own) {
            const bool rnd = !rml.fast[i];
            for (int jj = 0; jj < R; ++jj) {
              const float w = A.sc[i][2 * kPkChunk + jj] * A.lastw[i];
              if (w != 0.f) a += w * (rnd && KB ? round_bf16(A.v[jj][dd]) : A.v[jj][dd]);
            }
          }
          float* pp = P.ws.att + (((size_t)h * (S + 1) + sp) * kMaxRows + i) * (2 + HD + r);
          st_agent(pp + 2 + dd, a);
          if (dd == 0) {
            st_agent(pp, A.fin_m[i]);
            st_agent(pp + 1, A.fin_l[i]);
          }
        }
        // ---- every split counts in; the last of the head merges them
        if (arrive_last(&P.ws.att_cnt[h], S, &sh.last_flag)) {
          const size_t pbase = ((size_t)h * (S + 1)) * kMaxRows;
          const int me = min(tid, R * S - 1), mi_ = me / S, ms_ = me % S;
          const float* mp = P.ws.att + (pbase + (size_t)ms_ * kMaxRows + mi_) * (2 + HD + r);
          const float pm = ld_agent(mp), pl = ld_agent(mp + 1);
          const int ei = min(tid, R * HD - 1) / HD, ed = min(tid, R * HD - 1) % HD;
          float part[8];
#pragma unroll
          for (int u = 0; u < 8; ++u)
            part[u] = ld_agent(P.ws.att + (pbase + (size_t)min(u, S - 1) * kMaxRows + ei) * (2 + HD + r) + 2 + ed);
          if (tid < R * S) {
            A.mw[mi_][ms_] = pm;
            A.ml[mi_][ms_] = pl;
          }
          __syncthreads();
          if (tid < R) {
            const int i = tid;
            float Mx = -INFINITY;
            for (int s2 = 0; s2 < S; ++s2)
              if (A.ml[i][s2] > 0.f) Mx = fmaxf(Mx, A.mw[i][s2]);
            float Ls = 0.f;
            for (int s2 = 0; s2 < S; ++s2) {
              const float lv = A.ml[i][s2];
              const float w = lv > 0.f ? __expf(A.mw[i][s2] - Mx) : 0.f;
              A.mw[i][s2] = w;
              Ls += w * lv;
            }
            A.linv[i] = Ls > 0.f ? 1.f / Ls : 0.f;
          }
          __syncthreads();
          if (tid < R * HD) {
            float v = 0.f;
#pragma unroll
            for (int u = 0; u < 8; ++u)
              if (u < S) v += A.mw[ei][u] * part[u];
            for (int u = 8; u < S; ++u)
              v += A.mw[ei][u] * ld_agent(P.ws.att + (pbase + (size_t)u * kMaxRows + ei) * (2 + HD + r) + 2 + ed);
            v *= A.linv[ei];
            A.q[ei][ed] = v;   // o of row ei (q is no longer needed)
            st_agent(&P.ws.O[(size_t)ei * qd + h * HD + ed], v);
          }
          __syncthreads();
          // o-adapter down-projection share of this head (fast row):
          // uo[row][h][j] = sum_d A_o[j][h*HD + d] o[d]
          for (int i = 0; i < R; ++i) {
            const bool fast = rml.fast[i] && Ao;
            if constexpr (WB) {
              if (tid < apieces) {
                const int c = tid % (HD / 8);
                float a = 0.f;
#pragma unroll
                for (int w = 0; w < 4; ++w)
                  a += bf16lo(ap[w]) * A.q[i][8 * c + 2 * w] + bf16hi(ap[w]) * A.q[i][8 * c + 2 * w + 1];
                A.uop[tid] = a;
              }
              __syncthreads();
              if (tid < r) {
                float a = 0.f;
                for (int c = 0; c < HD / 8; ++c) a += A.uop[tid * (HD / 8) + c];
                st_agent(&P.ws.uo[((size_t)i * H + h) * r + tid], fast ? a : 0.f);
              }
              __syncthreads();
            } else {
              if (tid < r) {
                float a = 0.f;
                if (fast) {
                  const float* arow = (const float*)Ao + (size_t)tid * qd + h * HD;
                  for (int dd = 0; dd < HD; ++dd) a += arow[dd] * A.q[i][dd];
                }
                st_agent(&P.ws.uo[((size_t)i * H + h) * r + tid], a);
              }
            }
          }
        }
      }
      pk_arrive(P.bar, target + 1);
    }

}

// Output projection + residual of layer l.
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__device__ __forceinline__ void pk_phase_o(int l, uint32_t& target, PkShared& sh) {
  PK_PROLOGUE
  using CD = PkPc<ND>;
  using CQ = PkPc<NQ>;
  using CF = PkPc<NF>;
  (void)sizeof(CD); (void)sizeof(CQ); (void)sizeof(CF);
  const LayerPtrs* Lp = P.layers + l;   // uniform: scalar loads
  (void)Lp;
    // ======================= output projection + residual ====================
    {
      const char* wo = (const char*)Lp->wo;
      auto row_ptr = [=](int u, int) -> const void* { return wo + (size_t)u * qd * esz; };
      int u0, u1;
      rw_range(d, W, gw, u0, u1);
      RwStream<WB, CQ::NCH, 1, CQ::NS> st;
      const bool has_o = Lp->A[3] && Lp->B[3];
      PkOEpi<WB> epi{d, r, Lp->mlp_norm, Lp->A[4], Lp->A[5], Lp->B[3], &rml, sh.stat, P.ws, fm, 0, has_o, 0.f, 0.f};
      typename PkOEpi<WB>::Ops ops[decltype(st)::P];
      st.begin_all(row_ptr, u0, u1, epi, ops);
      target += 1;
      pk_wait(P.bar, target, P.ws.err, &sh.broken);
      epi.ri = sh.ri;
      constexpr int PM = RwPM<WB, CQ::NCH, CQ::NS, kPkThreads>::value;
      RwPieces<PM> xp;
      pk_load_rows<PM>(P.ws.O, 0, (M > 1 ? 1 : 0) * qd, nullptr, qd, xp);
      if (fm >= 0 && has_o) {
        pk_slot_sum<false>(P.ws.uo + (size_t)fm * D.H * r, D.H, r, sh.red, sh.stat);
      }
      rw_store_pieces<false, PM, kPkThreads>(xp, qd, pk_dyn);
      st.template run<true>(row_ptr, u0, u1, pk_dyn, qd, epi, ops);
      pk_wg_store<kPkWaves>(epi.accx, 2, sh.wsum, sh.tot, P.so, 0);
      pk_wg_store<kPkWaves>(fm >= 0 ? epi.accf : 0.f, 2 * r, sh.wsum, sh.tot, P.so, 2);
      if (tid >= 2 + 2 * r && tid < P.so_w) st_agent(pk_slot_at(P.so, tid), 0.f);   // the slot's padding
      pk_arrive(P.bar, target + 1);
    }

}

// Gate/up projections + SwiGLU of layer l.
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__device__ __forceinline__ void pk_phase_gu(int l, uint32_t& target, PkShared& sh) {
  PK_PROLOGUE
  using CD = PkPc<ND>;
  using CQ = PkPc<NQ>;
  using CF = PkPc<NF>;
  (void)sizeof(CD); (void)sizeof(CQ); (void)sizeof(CF);
  const LayerPtrs* Lp = P.layers + l;   // uniform: scalar loads
  (void)Lp;
    // ======================= gate/up + SwiGLU ================================
    {
      const float* mlp_norm = Lp->mlp_norm;
      if (tid == 0) {
        sh.base[0] = (const char*)Lp->wg;
        sh.base[1] = (const char*)Lp->wu;
      }
      __syncthreads();
      auto row_ptr = [=, &sh](int hu, int) -> const void* { return sh.base[hu & 1] + (size_t)(hu >> 1) * d * esz; };
      int j0, j1;
      rw_range(D.F, W, gw, j0, j1);
      const int u0 = 2 * j0, u1 = 2 * j1;
      RwStream<WB, CD::NCH, 1, CD::NS> st;
      PkGuEpi<WB> epi{D.F, r, mlp_norm, Lp->A[6], Lp->B[4], Lp->B[5], &rml, sh.stat, sh.inv_rms, P.ws, fm, Lp->A[4] && Lp->B[4], Lp->A[5] && Lp->B[5],
                      0.f, 0.f, 0.f};
      typename PkGuEpi<WB>::Ops ops[decltype(st)::P];
      st.begin_all(row_ptr, u0, u1, epi, ops);
      target += 1;
      pk_wait(P.bar, target, P.ws.err, &sh.broken);
      constexpr int PM = RwPM<WB, CD::NCH, CD::NS, kPkThreads>::value;
      RwPieces<PM> xp;
      pk_load_rows<PM>(P.ws.X, 0, (M > 1 ? 1 : 0) * d, mlp_norm, d, xp);
      pk_slot_sum<true>(P.so, G, P.so_w, sh.red, sh.stat);
      if (tid < 2) sh.inv_rms[tid] = rsqrtf(sh.stat[min(tid, M - 1)] / d + D.eps);
      rw_store_pieces<true, PM, kPkThreads>(xp, d, pk_dyn);
      st.template run<true>(row_ptr, u0, u1, pk_dyn, d, epi, ops);
      pk_wg_store<kPkWaves>(fm >= 0 ? epi.accf : 0.f, r, sh.wsum, sh.tot, P.sgu, 0);
      pk_arrive(P.bar, target + 1);
    }

}

// Down projection + residual of layer l.
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__device__ __forceinline__ void pk_phase_dn(int l, uint32_t& target, PkShared& sh) {
  PK_PROLOGUE
  using CD = PkPc<ND>;
  using CQ = PkPc<NQ>;
  using CF = PkPc<NF>;
  (void)sizeof(CD); (void)sizeof(CQ); (void)sizeof(CF);
  const LayerPtrs* Lp = P.layers + l;   // uniform: scalar loads
  (void)Lp;
    // ======================= down projection + residual ======================
    {
      const char* wd = (const char*)Lp->wd;
      auto row_ptr = [=](int u, int) -> const void* { return wd + (size_t)u * D.F * esz; };
      int u0, u1;
      rw_range(d, W, gw, u0, u1);
      RwStream<WB, CF::NCH, 1, CF::NS> st;
      const bool hd_ad = Lp->A[6] && Lp->B[6];
      PkDnEpi<WB> epi{d, r, Lp->mlp_norm, Lp->B[6], &rml, sh.stat, P.ws, fm, hd_ad, 0.f};
      typename PkDnEpi<WB>::Ops ops[decltype(st)::P];
      st.begin_all(row_ptr, u0, u1, epi, ops);
      target += 1;
      pk_wait(P.bar, target, P.ws.err, &sh.broken);
      constexpr int PM = RwPM<WB, CF::NCH, CF::NS, kPkThreads>::value;
      RwPieces<PM> xp;
      pk_load_rows<PM>(P.ws.ACT, 0, (M > 1 ? 1 : 0) * D.F, nullptr, D.F, xp);
      if (fm >= 0 && hd_ad) pk_slot_sum<true>(P.sgu, G, P.sgu_w, sh.red, sh.stat);
      rw_store_pieces<false, PM, kPkThreads>(xp, D.F, pk_dyn);
      st.template run<true>(row_ptr, u0, u1, pk_dyn, D.F, epi, ops);
      pk_wg_store<kPkWaves>(epi.acc, kPkSdW, sh.wsum, sh.tot, P.sd, 0);
      pk_arrive(P.bar, target + 1);
    }
}

// Final norm + LM head + arg-max; the last workgroup finishes the step.
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__device__ __forceinline__ void pk_phase_head(int l, uint32_t& target, PkShared& sh) {
  PK_PROLOGUE
  const int nl = l;   // layers run
  using CD = PkPc<ND>;
  using CQ = PkPc<NQ>;
  using CF = PkPc<NF>;
  (void)sizeof(CD); (void)sizeof(CQ); (void)sizeof(CF);
  const LayerPtrs* Lp = P.layers + l;   // uniform: scalar loads
  (void)Lp;
  {
    auto row_ptr = [=](int u, int) -> const void* { return (const char*)P.lm_head + (size_t)u * d * esz; };
    int u0, u1;
    rw_range(D.V, W, gw, u0, u1);
    RwStream<WB, CD::NCH, 1, CD::NS> st;
    PkHeadEpi epi{0, 0.f, P.io.logits_out, -INFINITY, 0x7fffffff};
    PkHeadEpi::Ops ops[decltype(st)::P];
    st.begin_all(row_ptr, u0, u1, epi, ops);
    target += 1;
    pk_wait(P.bar, target, P.ws.err, &sh.broken);
    constexpr int PM = RwPM<WB, CD::NCH, CD::NS, kPkThreads>::value;
    RwPieces<PM> xp;
    pk_load_rows<PM>(P.ws.X, 0, (M > 1 ? 1 : 0) * d, P.final_norm, d, xp);
    pk_slot_sum<true>(P.sd, G, kPkSdW, sh.red, sh.ssum);
    if (tid == 0) {
      // the row fed to the head: the slow row, or the fast row when it exited
      // at a gate or runs alone (a draft)
      const int f = M - 1;
      int pick = 0;
      if (rml.fast[f] && (sh.ex || rml.slow_of[f] < 0)) pick = f;
      sh.src[0] = pick;
      sh.inv_rms[0] = rsqrtf(sh.ssum[pick * 4] / d + D.eps);
    }
    __syncthreads();
    epi.hrow = sh.src[0];
    epi.ir = sh.inv_rms[0];
    rw_store_pieces<true, PM, kPkThreads>(xp, d, pk_dyn);
    st.template run<true>(row_ptr, u0, u1, pk_dyn, d, epi, ops);
    if (lane == 0) {
      sh.bz[wv] = epi.bz;
      sh.bi[wv] = epi.bi;
    }
    __syncthreads();
    if (tid == 0) {
      float bz = -INFINITY;
      int bi = 0x7fffffff;
      for (int w = 0; w < kPkWaves; ++w)
        if (sh.bz[w] > bz || (sh.bz[w] == bz && sh.bi[w] < bi)) { bz = sh.bz[w]; bi = sh.bi[w]; }
      st_agent(&P.ws.lm_val[(size_t)blockIdx.x * kMaxRows], bz);
      st_agent(&P.ws.lm_idx[(size_t)blockIdx.x * kMaxRows], bi);
    }
    if (!arrive_last(P.ws.lm_cnt, G, &sh.last_flag)) return;
    // ---- the last workgroup: global arg-max and the step's bookkeeping
    // reset the barrier for the next launch (every workgroup has passed its last wait)
    if (tid < kPkGroups) {
      __hip_atomic_store(&P.bar.ctr[tid * kPkRelStride], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&P.bar.flag[tid * kPkRelStride], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    if (wv != 0) return;
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int t0 = 0; t0 < G; t0 += 64 * 8) {
      float zv[8];
      int iv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = min(t0 + lane + 64 * u, G - 1);
        zv[u] = ld_agent(&P.ws.lm_val[(size_t)t * kMaxRows]);
        iv[u] = ld_agent(&P.ws.lm_idx[(size_t)t * kMaxRows]);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (zv[u] > bz || (zv[u] == bz && iv[u] < bi)) { bz = zv[u]; bi = iv[u]; }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float z2 = __shfl_xor(bz, o);
      const int i2 = __shfl_xor(bi, o);
      if (z2 > bz || (z2 == bz && i2 < bi)) { bz = z2; bi = i2; }
    }
    const int f = M - 1;
    const bool sig_on = rml.fast[f] && rml.slow_of[f] >= 0;
    const float dot = sh.ssum[f * 4 + 1], pin2 = sh.ssum[f * 4 + 2], pp = sh.ssum[f * 4 + 0];
    const float last_sig = sh.ex ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
    if (lane == 0) {
      P.io.next_token[P.io.draft_slot] = bi;
      const int t = posv + P.rm.pos_offset;
      if (rml.slow_of[f] >= 0 || !rml.fast[f]) P.kv.seq_lens[0] = t + 1;
      if (sig_on && nl == D.n_layers) st_agent(&P.ws.sig[D.n_layers - 1], last_sig);
      if (P.io.exit_b_out) P.io.exit_b_out[0] = sh.eb;
      if (P.io.advance) P.io.positions[0] = posv + 1;
    }
    if (P.io.signal_out) {
      for (int q = lane; q < D.n_layers; q += 64) {
        float v = q < nl - 1 ? ld_agent(&P.ws.sig[q]) : 0.f;
        if (q == D.n_layers - 1 && nl == D.n_layers) v = last_sig;
        if (!sig_on || (sh.ex && q >= sh.eb)) v = 0.f;
        P.io.signal_out[q] = v;
      }
    }
    if (P.io.h_out || P.io.p_out) {
      for (int i = lane; i < d; i += 64) {
        if (P.io.h_out) P.io.h_out[i] = ld_agent(&P.ws.X[i]);
        if (P.io.p_out) P.io.p_out[i] = ld_agent(&P.ws.X[(size_t)f * d + i]);
      }
    }
  }
}

// ============================================================================
// The step.  ND, NQ, NF: 1 KB pieces per row of reduction length d, H*hd, F.
// ============================================================================
template <int WB, int KB, int HD, int ND, int NQ, int NF>
__global__ __launch_bounds__(kPkThreads) void kp_step(PkArgs args) {
  __shared__ PkShared sh;
  (void)args;   // read through pk_args()
  {
    const PkArgs& P = pk_args();
    sk_rm_copy(sh.rmu, P.rm);
    if (threadIdx.x == 0) {
      sh.ex = 0;
      sh.eb = P.D.n_layers;
      sh.ri = 0;
      sh.broken = 0;
    }
  }
  __syncthreads();
  uint32_t target = 0;
  const int nl = pk_args().n_layers_run;
  for (int l = 0; l < nl; ++l) {
    pk_phase_qkv<WB, KB, HD, ND, NQ, NF>(l, target, sh);
    pk_phase_att<WB, KB, HD, ND, NQ, NF>(l, target, sh);
    if (sh.ex) continue;   // exited (EXIT mode): the rest of the layer is skipped, by every workgroup alike
    pk_phase_o<WB, KB, HD, ND, NQ, NF>(l, target, sh);
    pk_phase_gu<WB, KB, HD, ND, NQ, NF>(l, target, sh);
    pk_phase_dn<WB, KB, HD, ND, NQ, NF>(l, target, sh);
  }
  pk_phase_head<WB, KB, HD, ND, NQ, NF>(nl, target, sh);
}

}  // namespace m2r2
