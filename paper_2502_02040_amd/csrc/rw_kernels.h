// Row-per-wave decode GEMVs for one or two activation rows: the dual-stream
// decode step (slow row h of Eq. 1 and fast row p of Eq. 2 of one sequence),
// plain decoding, drafting and two-row verification chunks.
//
// Every wave owns a contiguous range of output units (one weight row, or a
// gate row and the up row of the same index) and computes each unit's full
// dot products itself: the lanes read one row as 1 KB pieces of 16 bytes per
// lane straight from the row-major weights, multiply them with the
// activation rows held in LDS (fp32, times the norm gain) in fp32, and sum
// across the wave.  No partial sums leave the wave, so the unit's epilogue
// (residual update, adapters, SwiGLU, logits) runs right away while the next
// unit's weights and epilogue operands are already in flight.  Units are
// split evenly over one workgroup of 8 waves per compute unit, so every
// compute unit streams the same number of bytes whatever the matrix shape.
// The row statistics the next kernel needs (sum of squares, adapter
// down-projections, exit-signal dot products) are summed per workgroup and
// added into one of kBinSlots bins with device-scope atomics.
#pragma once
#include "sk_kernels.h"

namespace m2r2 {

constexpr int kRwWaves = 8;
constexpr int kRwThreads = 64 * kRwWaves;

// Activation pieces (4 floats) per thread for a reduction of NS * NCH pieces
// of 1 KB per row.
template <int WB, int NCH, int NS, int T = kRwThreads>
struct RwPM {
  static constexpr int K = NS * NCH * 64 * (WB ? 8 : 4);
  static constexpr int value = (K / 4 + T - 1) / T;
};

// Units [u0, u1) of wave gw of W for n units (n * W < 2^32, checked by the
// host; gw is wave-uniform, so this is scalar arithmetic).
__device__ __forceinline__ void rw_range(int n, int W, int gw, int& u0, int& u1) {
  u0 = (int)((unsigned)gw * (unsigned)n / (unsigned)W);
  u1 = (int)((unsigned)(gw + 1) * (unsigned)n / (unsigned)W);
}

// Activation rows (and the norm gain when G) read into registers before the
// weights are primed, then stored into LDS as fp32 [2][K]: row m = candidate
// m times the gain.
template <int PM>
struct RwPieces {
  float4 v[PM][2];
  float4 g[PM];
};
// float4 index of piece p of this thread (pieces past the row repeat the last)
template <int T>
__device__ __forceinline__ int rw_piece_q(int p, int nq) { return min((int)threadIdx.x + T * p, nq - 1); }
template <bool G, int PM, int T = kRwThreads>
__device__ __forceinline__ void rw_load_pieces(const float* r0, const float* r1, const float* gain, int K,
                                               RwPieces<PM>& xp) {
  const int nq = K / 4;
#pragma unroll
  for (int p = 0; p < PM; ++p) {
    const int q = rw_piece_q<T>(p, nq);
    xp.v[p][0] = ldg4(r0 + 4 * q);
    xp.v[p][1] = ldg4(r1 + 4 * q);
    if constexpr (G) xp.g[p] = ldg4(gain + 4 * q);
  }
}
// Ends with a workgroup barrier.
template <bool G, int PM, int T = kRwThreads>
__device__ __forceinline__ void rw_store_pieces(const RwPieces<PM>& xp, int K, float* act) {
  const int nq = K / 4;
#pragma unroll
  for (int p = 0; p < PM; ++p) {
    if ((int)threadIdx.x + T * p < nq) {
      const int q = rw_piece_q<T>(p, nq);
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        float4 v = xp.v[p][m];
        if constexpr (G) {
          const float4 g = xp.g[p];
          v.x *= g.x; v.y *= g.y; v.z *= g.z; v.w *= g.w;
        }
        *(float4*)(act + (size_t)m * K + 4 * q) = v;
      }
    }
  }
  __syncthreads();
}

// One weight element as raw bits (bf16 in the low half, or fp32), loaded
// without converting: the epilogue operand groups must not wait for their
// loads; the epilogue converts with rw_wt().
template <int WB>
struct RwRaw {
  using type = uint16_t;
};
template <>
struct RwRaw<0> {
  using type = uint32_t;
};
template <int WB>
__device__ __forceinline__ typename RwRaw<WB>::type rw_wt_raw(const void* p, size_t i) {
  return ((const typename RwRaw<WB>::type*)p)[i];
}
template <int WB>
__device__ __forceinline__ float rw_wt(typename RwRaw<WB>::type bits) {
  if constexpr (WB) return __uint_as_float((uint32_t)bits << 16);
  else return __uint_as_float(bits);
}

// Sum over the 64 lanes of a wave (every lane gets it).
__device__ __forceinline__ float wave_allsum(float v) {
  v = row_sum16(v);
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}

// The weight stream of one wave: U rows per unit, each row NS * NCH pieces of
// 1 KB, read NCH pieces (a sub-unit) at a time.  Rows of one sub-unit keep P
// units in flight (a ring of P register buffers); rows of two sub-units keep
// both halves of one unit and the next unit's first half in flight.
template <int WB, int NCH, int U, int NS, int PD = 2>
struct RwStream {
  static constexpr int EPL = WB ? 8 : 4;   // weight elements per lane and piece
  static constexpr int P = PD;             // register buffers (operand sets)
  static_assert(NS == 1 || P == 2, "rows of two sub-units use two buffers");
  u32x4_t bb[P][U][NCH];

  // The loads of one sub-unit are issued as a group (nothing is scheduled
  // into or across it): the compiler's in-order wait counts then agree
  // between the loop entry and its back edge, so a wait for one piece never
  // waits for the loads issued after it.
  template <class PF>
  __device__ __forceinline__ void load(const PF& row_ptr, int unit, int sub, u32x4_t (&dst)[U][NCH]) const {
    const int lane = threadIdx.x & 63;
    const char* p[U];
#pragma unroll
    for (int u = 0; u < U; ++u) p[u] = (const char*)row_ptr(unit, u) + (size_t)sub * NCH * 1024 + lane * 16;
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int c = 0; c < NCH; ++c) dst[u][c] = ld_glob(p[u] + (size_t)c * 1024);
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  // A unit's epilogue operand loads, issued as a group after the weights
  // before it (compiler memory barriers keep the optimizer from hoisting
  // them, whose addresses are known early, above the weight loads).
  template <class Epi, class F>
  __device__ __forceinline__ static void fetch_grouped(const Epi&, const F& f) {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    f();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
  }

  // a[u][m] += lane partial dot products of sub-unit `sub` with activation rows m.
  __device__ __forceinline__ void dot(const u32x4_t (&w)[U][NCH], const float* act, int K, int sub,
                                      float (&a)[U][2]) const {
    const int lane = threadIdx.x & 63;
    if constexpr (NS > 1) {
      // A row of several sub-units: re-read the activations from LDS for
      // every sub-unit.  (The optimizer would otherwise keep the values read
      // for one unit live for the next, which needs more registers than a
      // wave has.)  The opaque zero offset keeps the reads distinct.
      int zoff = 0;
      asm volatile("" : "+s"(zoff));
      act += zoff;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float a0 = a[u][0], a1 = a[u][1];
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const int k = (sub * NCH + c) * 64 * EPL + lane * EPL;
        if constexpr (WB) {
          const float4 x0a = *(const float4*)(act + k), x0b = *(const float4*)(act + k + 4);
          const float4 x1a = *(const float4*)(act + K + k), x1b = *(const float4*)(act + K + k + 4);
          const float w0 = bf16lo(w[u][c][0]), w1 = bf16hi(w[u][c][0]), w2 = bf16lo(w[u][c][1]), w3 = bf16hi(w[u][c][1]);
          const float w4 = bf16lo(w[u][c][2]), w5 = bf16hi(w[u][c][2]), w6 = bf16lo(w[u][c][3]), w7 = bf16hi(w[u][c][3]);
          a0 += w0 * x0a.x + w1 * x0a.y + w2 * x0a.z + w3 * x0a.w + w4 * x0b.x + w5 * x0b.y + w6 * x0b.z + w7 * x0b.w;
          a1 += w0 * x1a.x + w1 * x1a.y + w2 * x1a.z + w3 * x1a.w + w4 * x1b.x + w5 * x1b.y + w6 * x1b.z + w7 * x1b.w;
          // finish every two pieces in place: the sums are pinned by an
          // empty asm (the optimizer would otherwise sink the arithmetic to
          // the end and read every piece's activations first) and the
          // activation reads of later pieces are not hoisted above it
          if (c % 2 == 1) {
            asm volatile("" : "+v"(a0), "+v"(a1));
            __builtin_amdgcn_sched_barrier(0);
          }
        } else {
          const float4 x0 = *(const float4*)(act + k), x1 = *(const float4*)(act + K + k);
          const float w0 = __uint_as_float(w[u][c][0]), w1 = __uint_as_float(w[u][c][1]);
          const float w2 = __uint_as_float(w[u][c][2]), w3 = __uint_as_float(w[u][c][3]);
          a0 += w0 * x0.x + w1 * x0.y + w2 * x0.z + w3 * x0.w;
          a1 += w0 * x1.x + w1 * x1.y + w2 * x1.z + w3 * x1.w;
          if (c % 4 == 3) {   // as above, every four (smaller) pieces
            asm volatile("" : "+v"(a0), "+v"(a1));
            __builtin_amdgcn_sched_barrier(0);
          }
        }
      }
      a[u][0] = a0;
      a[u][1] = a1;
    }
  }

  __device__ __forceinline__ static void zero(float (&a)[U][2]) {
#pragma unroll
    for (int u = 0; u < U; ++u) a[u][0] = a[u][1] = 0.f;
  }
  __device__ __forceinline__ static void finish(float (&a)[U][2]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      a[u][0] = wave_allsum(a[u][0]);
      a[u][1] = wave_allsum(a[u][1]);
    }
  }

  // Issue the first weights of the range [u0, u1) and their epilogue
  // operands, ahead of the activation staging: sub-unit 0 of unit u0 (the
  // other buffers are filled when the stream starts: more loads before the
  // staging delay the staging's own, and its barriers wait for every wave).  Every load is unconditional (the
  // compiler's wait counts stay exact): units past the range read the
  // range's last unit again, an empty range (u0 < n always) reads unit u0.
  static constexpr int kBegin = 1;
  template <class PF, class Epi>
  __device__ __forceinline__ void begin(const PF& row_ptr, int u0, int u1, const Epi& epi,
                                        typename Epi::Ops (&ops)[P]) {
    const int last = max(u1 - 1, u0);
    if constexpr (NS == 1) {
#pragma unroll
      for (int i = 0; i < kBegin; ++i) {
        load(row_ptr, min(u0 + i, last), 0, bb[i]);
        fetch_grouped(epi, [&] { epi.fetch(min(u0 + i, last), ops[i]); });
      }
    } else {
      static_assert(NS == 2, "one or two sub-units per unit");
      load(row_ptr, u0, 0, bb[0]);
      fetch_grouped(epi, [&] { epi.fetch(u0, ops[0]); });
    }
  }

  // Issue every register buffer's first weights (and their epilogue
  // operands) for the range [u0, u1): for a phase whose activations are not
  // there yet, so that all of them are in flight while it waits; run<true>()
  // then streams on without issuing them again.  Loads stay unconditional
  // and in range as in begin().
  template <class PF, class Epi>
  __device__ __forceinline__ void begin_all(const PF& row_ptr, int u0, int u1, const Epi& epi,
                                            typename Epi::Ops (&ops)[P]) {
    const int last = max(u1 - 1, u0);
    if constexpr (NS == 1) {
#pragma unroll
      for (int i = 0; i < P; ++i) {
        load(row_ptr, min(u0 + i, last), 0, bb[i]);
        fetch_grouped(epi, [&] { epi.fetch(min(u0 + i, last), ops[i]); });
      }
    } else {
      load(row_ptr, u0, 0, bb[0]);
      fetch_grouped(epi, [&] { epi.fetch(u0, ops[0]); });
      load(row_ptr, u0, 1, bb[1]);
    }
  }

  // Stream units [u0, u1) after begin(): epi.fetch(unit, ops) issues a unit's
  // epilogue operands (in flight with its weights), epi.run(unit, y, ops)
  // runs the epilogue.  Inside the loops every iteration issues the same
  // loads; the last units are finished after the loop, so nothing past the
  // range is read.
  template <bool PRIMED = false, class PF, class Epi>
  __device__ __forceinline__ void run(const PF& row_ptr, int u0, int u1, const float* act, int K, Epi& epi,
                                      typename Epi::Ops (&ops)[P]) {
    if (u0 >= u1) return;
    float y[U][2];
    int u = u0;
    if constexpr (NS == 1) {
      if constexpr (!PRIMED) {
        const int last = u1 - 1;
#pragma unroll
        for (int i = kBegin; i < P; ++i) {
          load(row_ptr, min(u0 + i, last), 0, bb[i]);
          fetch_grouped(epi, [&] { epi.fetch(min(u0 + i, last), ops[i]); });
        }
      }
      // buffer i holds unit u + i; a unit's buffer is refilled with the unit
      // P further on as soon as its dot products are done
      for (; u + 2 * P - 1 < u1; u += P) {
#pragma unroll
        for (int i = 0; i < P; ++i) {
          zero(y);
          dot(bb[i], act, K, 0, y);
          load(row_ptr, u + i + P, 0, bb[i]);
          finish(y);
          epi.run(u + i, y, ops[i]);
          fetch_grouped(epi, [&] { epi.fetch(u + i + P, ops[i]); });
        }
      }
      // the last 1 .. 2P-1 units: refills are conditional here (what they
      // bring is needed next anyway); the blocks have no else branches (the
      // compiler would hoist a common prefix of two branches above them,
      // converting every weight of the unit at once)
      const int left = u1 - u;
#pragma unroll
      for (int i = 0; i < 2 * P - 1; ++i) {
        if (i < left) {
          zero(y);
          dot(bb[i % P], act, K, 0, y);
          if (i + P < left) load(row_ptr, u + i + P, 0, bb[i % P]);
          finish(y);
          epi.run(u + i, y, ops[i % P]);
          if (i + P < left) epi.fetch(u + i + P, ops[i % P]);
        }
      }
    } else {
      if constexpr (!PRIMED) load(row_ptr, u0, 1, bb[1]);   // the second half of the first unit
      // unit u in bb[0] (sub-unit 0) and bb[1] (sub-unit 1), its operands in ops[0];
      // two units per iteration so the operand buffers alternate in place
      for (; u + 2 < u1; u += 2) {
        zero(y);
        dot(bb[0], act, K, 0, y);
        load(row_ptr, u + 1, 0, bb[0]);
        fetch_grouped(epi, [&] { epi.fetch(u + 1, ops[1]); });
        dot(bb[1], act, K, 1, y);
        load(row_ptr, u + 1, 1, bb[1]);
        finish(y);
        epi.run(u, y, ops[0]);
        zero(y);
        dot(bb[0], act, K, 0, y);
        load(row_ptr, u + 2, 0, bb[0]);
        fetch_grouped(epi, [&] { epi.fetch(u + 2, ops[0]); });
        dot(bb[1], act, K, 1, y);
        load(row_ptr, u + 2, 1, bb[1]);
        finish(y);
        epi.run(u + 1, y, ops[1]);
      }
      // the last one or two units (conditional loads, no common branch prefix)
      const bool two = u + 1 < u1;
      zero(y);
      dot(bb[0], act, K, 0, y);
      if (two) {
        load(row_ptr, u + 1, 0, bb[0]);
        fetch_grouped(epi, [&] { epi.fetch(u + 1, ops[1]); });
      }
      dot(bb[1], act, K, 1, y);
      if (two) load(row_ptr, u + 1, 1, bb[1]);
      finish(y);
      epi.run(u, y, ops[0]);
      if (two) {
        zero(y);
        dot(bb[0], act, K, 0, y);
        dot(bb[1], act, K, 1, y);
        finish(y);
        epi.run(u + 1, y, ops[1]);
      }
    }
  }
};

// Workgroup sum of per-wave values v[0..n) (n <= 64, lane i of each of the
// NW waves holds value i) into out[0..n) (LDS); scratch holds NW * 64 floats.
template <int NW = kRwWaves>
__device__ __forceinline__ void rw_wg_sum(float v, int n, float* scratch, float* out) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  scratch[wv * 64 + lane] = v;
  __syncthreads();
  if ((int)threadIdx.x < n) {
    float a = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) a += scratch[w * 64 + threadIdx.x];
    out[threadIdx.x] = a;
  }
  __syncthreads();
}

// Adapter up-factor row (at most 32 bytes: r <= 16 bf16 / 8 f32 values) as
// 16-byte pieces held by every lane, and its dot with u (LDS).
constexpr int kRwMaxBRowBytes = 32;
template <int WB>
struct RwBRow {
  static constexpr int NP = kRwMaxBRowBytes / 16;
  u32x4_t p[NP];
  __device__ __forceinline__ void load(const void* B, int row, int r) {
    const int np = r * (WB ? 2 : 4) / 16;
    const u32x4_t* s = (const u32x4_t*)((const char*)B + (size_t)row * r * (WB ? 2 : 4));
#pragma unroll
    for (int i = 0; i < NP; ++i) p[i] = s[min(i, np - 1)];
  }
  __device__ __forceinline__ float dot(const float* u, int r) const {
    const int np = r * (WB ? 2 : 4) / 16;
    float v = 0.f;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      if (i >= np) break;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if constexpr (WB) v += bf16lo(p[i][k]) * u[8 * i + 2 * k] + bf16hi(p[i][k]) * u[8 * i + 2 * k + 1];
        else v += __uint_as_float(p[i][k]) * u[4 * i + k];
      }
    }
    return v;
  }
};

// ============================================================================
// QKV: rows of [Wq; Wk; Wv; A_q; A_k; A_v] times rms(x) g_att, with the gate
// decision of the boundary before the layer.  A fast row restarting at a
// gate (p <- h) takes its slow row's results: both rows are projected.
// ============================================================================
template <int WB, int NCH, int NS>
__global__ __launch_bounds__(kRwThreads) void kr_qkv(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  extern __shared__ __attribute__((aligned(16))) float actf[];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int ex_in[kMaxSeq], eb_in[kMaxSeq];
  __shared__ int reinit_s[kMaxSeq], exited_s[kMaxSeq], exitb_s[kMaxSeq];
  __shared__ float sig_s[kMaxSeq];
  __shared__ float inv_rms[2];
  __shared__ int src_s[2];
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, gw = blockIdx.x * kRwWaves + __builtin_amdgcn_readfirstlane(tid >> 6);
  const int esz = WB ? 2 : 4, qd = D.qdim, r = D.r;
  const int nu = 3 * qd + 3 * r;
  const void* Ap[3] = {L.A[0], L.A[1], L.A[2]};
  auto row_ptr = [&](int u, int) -> const void* {
    const size_t rb = (size_t)D.d * esz;
    if (u < qd) return (const char*)L.wq + u * rb;
    if (u < 2 * qd) return (const char*)L.wk + (u - qd) * rb;
    if (u < 3 * qd) return (const char*)L.wv + (u - 2 * qd) * rb;
    const int a = u - 3 * qd, w = a / r;
    const void* A = w == 0 ? Ap[0] : (w == 1 ? Ap[1] : Ap[2]);
    return A ? (const char*)A + (a % r) * rb : L.wq;   // missing adapter: any row (result zeroed)
  };
  int u0, u1;
  rw_range(nu, gridDim.x * kRwWaves, gw, u0, u1);
  RwStream<WB, NCH, 1, NS> st;
  float bv[1];
  sk_bins_load(rm.M * 4, bin_d_at(ws, layer, 0, 0), kMaxRows * 4, bv);
  const int sq0 = min(tid, rm.nseq - 1);
  const int exv = ws.exited[sq0], ebv = ws.exitb[sq0];
  RwPieces<RwPM<WB, NCH, NS>::value> xp;
  rw_load_pieces<true>(ws.X, ws.X + (size_t)(rm.M > 1 ? 1 : 0) * D.d, L.attn_norm, D.d, xp);
  const int nqkv = nu;
  struct Epi {
    struct Ops {};
    const RowMap* rm;
    const int* src;
    const float* ir;
    float* QKV;
    int nqkv, qd, r;
    const void* const* Ap;
    __device__ void fetch(int, Ops&) const {}
    __device__ void run(int u, const float (&y)[1][2], const Ops&) const {
      const int lane = threadIdx.x & 63;
      if (lane < rm->M) {
        const int s = src[lane];
        float v = y[0][s] * ir[lane];
        if (u >= 3 * qd) {
          const int w = (u - 3 * qd) / r;
          if (!(w == 0 ? Ap[0] : (w == 1 ? Ap[1] : Ap[2]))) v = 0.f;
        }
        QKV[(size_t)lane * nqkv + u] = v;
      }
    }
  } epi{&rml, src_s, inv_rms, ws.QKV, nqkv, qd, r, Ap};
  typename Epi::Ops ops[decltype(st)::P];
  __builtin_amdgcn_sched_barrier(0);
  st.begin(row_ptr, u0, u1, epi, ops);
  __builtin_amdgcn_sched_barrier(0);
  if (tid < rm.nseq) { ex_in[tid] = exv; eb_in[tid] = ebv; }
  sk_rm_copy(rmu, rm);
  sk_bins_sum(rm.M * 4, bv, actf, ssum);
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
  rw_store_pieces<true>(xp, D.d, actf);
  // EXIT mode, every sequence exited (at this boundary or before): the layer
  // only fills its cache entries from the slow rows, so only the k and v rows
  // are needed; they are spread over all waves (the units primed above are
  // dropped)
  bool all_ex = io.mode == EX_EXIT;
  for (int sq = 0; sq < rm.nseq; ++sq) all_ex = all_ex && exited_s[sq] != 0;
  if (all_ex) {
    int v0, v1;
    rw_range(2 * qd, gridDim.x * kRwWaves, gw, v0, v1);
    v0 += qd;
    v1 += qd;
    st.begin(row_ptr, v0, v1, epi, ops);
    st.run(row_ptr, v0, v1, actf, D.d, epi, ops);
  } else {
    st.run(row_ptr, u0, u1, actf, D.d, epi, ops);
  }
}

// ============================================================================
// Output projection + residual (+ adapter on fast rows); partial sums for the
// gate/up prologue (sum x^2, adapter-down of gate and up).
// ============================================================================
template <int WB, int NCH, int NS, int NW = kRwWaves>
__global__ __launch_bounds__(64 * NW) void kr_oproj(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  extern __shared__ __attribute__((aligned(16))) float actf[];
  __shared__ float ud_s[2 * (64 * NW)];
  __shared__ float uo_s[2 * kMaxRank];
  __shared__ float wsum[NW * 64];
  __shared__ float tot[64];
  __shared__ int flag_s[2 * kMaxSeq];   // exited, reinit per sequence
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, lane = tid & 63, gw = blockIdx.x * NW + __builtin_amdgcn_readfirstlane(tid >> 6);
  if (io.mode == EX_EXIT && sk_all_exited(rm, ws)) return;
  const int esz = WB ? 2 : 4, r = D.r, HR = D.H * D.r;
  auto row_ptr = [&](int u, int) -> const void* { return (const char*)L.wo + (size_t)u * D.qdim * esz; };
  int u0, u1;
  rw_range(D.d, gridDim.x * NW, gw, u0, u1);
  RwStream<WB, NCH, 1, NS> st;
  RwPieces<RwPM<WB, NCH, NS, 64 * NW>::value> xp;
  rw_load_pieces<false, RwPM<WB, NCH, NS, 64 * NW>::value, 64 * NW>(ws.O, ws.O + (size_t)(rm.M > 1 ? 1 : 0) * D.qdim, nullptr, D.qdim, xp);
  const float uv0 = ws.uo[min(tid, 2 * HR - 1)];
  const float uv1 = ws.uo[min(tid + (64 * NW), 2 * HR - 1)];
  const int fe = ws.exited[min(tid, kMaxSeq - 1)];
  const int fr = ws.reinit[layer * kMaxSeq + min(tid, kMaxSeq - 1)];
  const bool has_o = L.A[3] && L.B[3];
  // per-wave sums: lane m (< 2): sum x^2 of row m; lane c (< 2r): the
  // adapter-down partial c of row 0 (acc0) and row 1 (acc1) when fast
  struct Epi {
    struct Ops {
      float x0, x1, g;
      typename RwRaw<WB>::type a;   // A_g[c][n] (c < r) or A_u[c - r][n] of this lane's c (raw bits)
      RwBRow<WB> b;
    };
    const Dims* D;
    const LayerPtrs* L;
    const RowMap* rm;
    const int* flag;
    const float* uo;
    WS ws;
    int layer;
    bool has_o;
    float accx, acc0, acc1;
    __device__ void fetch(int n, Ops& o) const {
      // every load unconditional (missing factors read a valid stand-in)
      const int lane = threadIdx.x & 63, r = D->r;
      o.x0 = ws.X[n];
      o.x1 = ws.X[(size_t)D->d + n];
      o.g = L->mlp_norm[n];
      const int c = lane % (2 * r);
      const void* A = c < r ? L->A[4] : L->A[5];
      o.a = rw_wt_raw<WB>(A ? A : (const void*)L->mlp_norm, A ? (size_t)(c % r) * D->d + n : 0);
      o.b.load(has_o ? L->B[3] : (const void*)L->mlp_norm, has_o ? n : 0, r);
    }
    __device__ void run(int n, const float (&y)[1][2], const Ops& o) {
      const int lane = threadIdx.x & 63, r = D->r;
      float xnew[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        xnew[m] = 0.f;
        if (m >= rm->M) continue;
        const int sq = rm->seq[m];
        const bool ex = flag[sq] != 0, ri = flag[kMaxSeq + sq] != 0, fast = rm->fast[m] != 0;
        const float xo = m ? o.x1 : o.x0;
        const float xs = rm->slow_of[m] == 1 ? o.x1 : o.x0;
        float xn = xo, pin = 0.f;
        if (!ex) {
          if (fast) {
            pin = ri ? xs : xo;
            xn = pin + y[0][m] + (has_o ? o.b.dot(uo + m * r, r) : 0.f);
          } else {
            xn = xo + y[0][m];
          }
          if (lane == m) {
            ws.X[(size_t)m * D->d + n] = xn;
            if (fast) ws.PIN[(size_t)m * D->d + n] = pin;
          }
        }
        xnew[m] = xn;
      }
      accx += lane == 0 ? xnew[0] * xnew[0] : (lane == 1 ? xnew[1] * xnew[1] : 0.f);
      const float ga = rw_wt<WB>(o.a) * o.g;
      if (rm->fast[0]) acc0 += ga * xnew[0];
      if (rm->M > 1 && rm->fast[1]) acc1 += ga * xnew[1];
    }
  } epi{&D, &L, &rml, flag_s, uo_s, ws, layer, has_o, 0.f, 0.f, 0.f};
  typename Epi::Ops ops[decltype(st)::P];
  __builtin_amdgcn_sched_barrier(0);
  st.begin(row_ptr, u0, u1, epi, ops);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  if (tid < kMaxSeq) { flag_s[tid] = fe; flag_s[kMaxSeq + tid] = fr; }
  ud_s[tid] = uv0;
  ud_s[tid + (64 * NW)] = uv1;
  __syncthreads();
  if (tid < 2 * r) {
    const int m = tid / r, j = tid % r;
    float a = 0.f;
    if (has_o && m < rm.M && rml.fast[m] && 2 * HR <= 2 * (64 * NW)) {
#pragma unroll 8
      for (int h = 0; h < D.H; ++h) a += ud_s[(m * D.H + h) * r + j];
    } else if (has_o && m < rm.M && rml.fast[m]) {
      for (int h = 0; h < D.H; ++h) a += ws.uo[(m * D.H + h) * r + j];
    }
    uo_s[tid] = a;
  }
  rw_store_pieces<false, RwPM<WB, NCH, NS, 64 * NW>::value, 64 * NW>(xp, D.qdim, actf);
  st.run(row_ptr, u0, u1, actf, D.qdim, epi, ops);
  const int bin = blockIdx.x % kBinSlots;
  rw_wg_sum<NW>(epi.accx, 2, wsum, tot);
  if (tid < rm.M) add_agent(bin_o_at(ws, D, layer, bin, tid), tot[tid]);
  for (int m = 0; m < 2; ++m) {
    rw_wg_sum<NW>(m ? epi.acc1 : epi.acc0, 2 * r, wsum, tot);
    if (tid < 2 * r && m < rm.M && rml.fast[m] && (tid < r ? L.A[4] : L.A[5]))
      add_agent(bin_o_at(ws, D, layer, bin, m) + 1 + tid, tot[tid]);
  }
}

// ============================================================================
// Gate/up + adapter-up + SwiGLU; partial sums of the down adapter's
// down-projection.  The stream runs over half-units: gate row j (2j), then
// up row j (2j + 1); the epilogue of pair j runs after its up row.
// ============================================================================
template <int WB, int NCH, int NS>
__global__ __launch_bounds__(kRwThreads) void kr_gateup(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  extern __shared__ __attribute__((aligned(16))) float actf[];
  __shared__ float stat[2 * (1 + 2 * kMaxRank)];
  __shared__ float inv_rms[2];
  __shared__ float wsum[kRwWaves * 64];
  __shared__ float tot[64];
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, gw = blockIdx.x * kRwWaves + __builtin_amdgcn_readfirstlane(tid >> 6);
  if (io.mode == EX_EXIT && sk_all_exited(rm, ws)) return;
  const int esz = WB ? 2 : 4, r = D.r, PO = 1 + 2 * r;
  auto row_ptr = [&](int hu, int) -> const void* {
    return (const char*)((hu & 1) ? L.wu : L.wg) + (size_t)(hu >> 1) * D.d * esz;
  };
  int j0, j1;
  rw_range(D.F, gridDim.x * kRwWaves, gw, j0, j1);
  const int u0 = 2 * j0, u1 = 2 * j1;
  RwStream<WB, NCH, 1, NS> st;
  float sv[(2 * (1 + 2 * kMaxRank) * kBinSlots + kSkThreads - 1) / kSkThreads];
  sk_bins_load(rm.M * PO, bin_o_at(ws, D, layer, 0, 0), kMaxRows * PO, sv);
  RwPieces<RwPM<WB, NCH, NS>::value> xp;
  rw_load_pieces<true>(ws.X, ws.X + (size_t)(rm.M > 1 ? 1 : 0) * D.d, L.mlp_norm, D.d, xp);
  struct Epi {
    struct Ops {
      typename RwRaw<WB>::type a;   // A_d[lane % r][j] (raw bits)
      RwBRow<WB> bg, bu;
    };
    const Dims* D;
    const LayerPtrs* L;
    const RowMap* rm;
    const float* stat;
    const float* ir;
    WS ws;
    bool hg, hu;
    float yg0, yg1;   // the gate results of the current pair
    float acc0, acc1;
    __device__ void fetch(int h, Ops& o) const {
      const int lane = threadIdx.x & 63, r = D->r, j = h >> 1;
      const void* fb = (const void*)L->mlp_norm;   // stand-in for missing factors (loads stay unconditional)
      o.a = rw_wt_raw<WB>(L->A[6] ? L->A[6] : fb, L->A[6] ? (size_t)(lane % r) * D->F + j : 0);
      o.bg.load(hg ? L->B[4] : fb, hg ? j : 0, r);
      o.bu.load(hu ? L->B[5] : fb, hu ? j : 0, r);
    }
    __device__ void run(int h, const float (&y)[1][2], const Ops& o) {
      if (!(h & 1)) {
        yg0 = y[0][0];
        yg1 = y[0][1];
        return;
      }
      const int lane = threadIdx.x & 63, r = D->r, PO = 1 + 2 * r, j = h >> 1;
      float av[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        av[m] = 0.f;
        if (m >= rm->M) continue;
        float g = (m ? yg1 : yg0) * ir[m], u = y[0][m] * ir[m];
        if (rm->fast[m]) {
          if (hg) g += o.bg.dot(stat + m * PO + 1, r) * ir[m];
          if (hu) u += o.bu.dot(stat + m * PO + 1 + r, r) * ir[m];
        }
        av[m] = silu(g) * u;
        if (lane == m) ws.ACT[(size_t)m * D->F + j] = av[m];
      }
      const float aw = rw_wt<WB>(o.a);
      if (rm->fast[0]) acc0 += aw * av[0];
      if (rm->M > 1 && rm->fast[1]) acc1 += aw * av[1];
    }
  } epi{&D, &L, &rml, stat, inv_rms, ws, L.A[4] && L.B[4], L.A[5] && L.B[5], 0.f, 0.f, 0.f, 0.f};
  typename Epi::Ops ops[decltype(st)::P];
  __builtin_amdgcn_sched_barrier(0);
  st.begin(row_ptr, u0, u1, epi, ops);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  sk_bins_sum(rm.M * PO, sv, actf, stat);
  if (tid < 2) inv_rms[tid] = rsqrtf(stat[min(tid, rm.M - 1) * PO] / D.d + D.eps);
  rw_store_pieces<true>(xp, D.d, actf);
  st.run(row_ptr, u0, u1, actf, D.d, epi, ops);
  for (int m = 0; m < 2; ++m) {
    rw_wg_sum(m ? epi.acc1 : epi.acc0, r, wsum, tot);
    if (tid < r && L.A[6] && m < rm.M && rml.fast[m])
      add_agent(bin_gu_at(ws, D, layer, blockIdx.x % kBinSlots, m) + tid, tot[tid]);
  }
}

// ============================================================================
// Down projection + residual (+ adapter); partial sums for the next layer's
// norm and the exit signal.
// ============================================================================
template <int WB, int NCH, int NS, int NW = kRwWaves>
__global__ __launch_bounds__(64 * NW) void kr_down(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, int layer) {
  extern __shared__ __attribute__((aligned(16))) float actf[];
  __shared__ float ud[2 * kMaxRank];
  __shared__ float wsum[NW * 64];
  __shared__ float tot[64];
  __shared__ int ex_s[kMaxSeq];
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, gw = blockIdx.x * NW + __builtin_amdgcn_readfirstlane(tid >> 6);
  if (io.mode == EX_EXIT && sk_all_exited(rm, ws)) {
    if (blockIdx.x == 0) rows_unchanged_stats(D, rm, ws, layer + 1);
    return;
  }
  const int esz = WB ? 2 : 4, r = D.r;
  auto row_ptr = [&](int u, int) -> const void* { return (const char*)L.wd + (size_t)u * D.F * esz; };
  int u0, u1;
  rw_range(D.d, gridDim.x * NW, gw, u0, u1);
  RwStream<WB, NCH, 1, NS> st;
  float uv[(2 * kMaxRank * kBinSlots + 64 * NW - 1) / (64 * NW)];
  sk_bins_load<64 * NW>(rm.M * r, bin_gu_at(ws, D, layer, 0, 0), kMaxRows * r, uv);
  RwPieces<RwPM<WB, NCH, NS, 64 * NW>::value> xp;
  rw_load_pieces<false, RwPM<WB, NCH, NS, 64 * NW>::value, 64 * NW>(ws.ACT, ws.ACT + (size_t)(rm.M > 1 ? 1 : 0) * D.F, nullptr, D.F, xp);
  const int exv = ws.exited[min(tid, kMaxSeq - 1)];
  struct Epi {
    struct Ops {
      float x0, x1, p0, p1;
      RwBRow<WB> b;
    };
    const Dims* D;
    const LayerPtrs* L;
    const RowMap* rm;
    const float* ud;
    const int* ex;
    WS ws;
    bool hd;
    float acc;
    __device__ void fetch(int n, Ops& o) const {
      o.x0 = ws.X[n];
      o.x1 = ws.X[(size_t)D->d + n];
      o.p0 = ws.PIN[n];
      o.p1 = ws.PIN[(size_t)D->d + n];
      o.b.load(hd ? L->B[6] : (const void*)ws.X, hd ? n : 0, D->r);
    }
    __device__ void run(int n, const float (&y)[1][2], const Ops& o) {
      const int lane = threadIdx.x & 63;
      float xv[2], pv[2];
#pragma unroll
      for (int m = 0; m < 2; ++m) {
        xv[m] = 0.f;
        pv[m] = 0.f;
        if (m >= rm->M) continue;
        const bool fast = rm->fast[m] != 0;
        float x = m ? o.x1 : o.x0;
        if (!ex[rm->seq[m]]) {
          x += y[0][m];
          if (fast && hd) x += o.b.dot(ud + m * D->r, D->r);
          if (lane == m) ws.X[(size_t)m * D->d + n] = x;
        }
        xv[m] = x;
        pv[m] = fast ? (m ? o.p1 : o.p0) : 0.f;
      }
      if (lane < 6) {
        const int m = lane / 3, c = lane % 3;
        acc += c == 0 ? xv[m] * xv[m] : (c == 1 ? pv[m] * xv[m] : pv[m] * pv[m]);
      }
    }
  } epi{&D, &L, &rml, ud, ex_s, ws, L.A[6] && L.B[6], 0.f};
  typename Epi::Ops ops[decltype(st)::P];
  __builtin_amdgcn_sched_barrier(0);
  st.begin(row_ptr, u0, u1, epi, ops);
  __builtin_amdgcn_sched_barrier(0);
  sk_rm_copy(rmu, rm);
  if (tid < kMaxSeq) ex_s[tid] = exv;
  sk_bins_sum<64 * NW>(rm.M * r, uv, actf, ud);
  rw_store_pieces<false, RwPM<WB, NCH, NS, 64 * NW>::value, 64 * NW>(xp, D.F, actf);
  st.run(row_ptr, u0, u1, actf, D.F, epi, ops);
  rw_wg_sum<NW>(epi.acc, 6, wsum, tot);
  if (tid < 2 * 3 && tid / 3 < rm.M) add_agent(bin_d_at(ws, layer + 1, blockIdx.x % kBinSlots, tid / 3) + tid % 3, tot[tid]);
}

// ============================================================================
// Final norm + LM head + arg-max; the last workgroup to finish finishes the
// step (tokens, exit bookkeeping, acceptance of a verified chunk).
// ============================================================================
template <int WB, int NCH, int NS>
__global__ __launch_bounds__(kRwThreads) void kr_head(Dims D, const void* lm_head, const float* final_norm, RowMap rm,
                                                      WS ws, StepIO io, KVPtrs kv, SkWS sk, int n_layers_run,
                                                      const void* head_b) {
  extern __shared__ __attribute__((aligned(16))) float actf[];
  __shared__ float ssum[kMaxRows * 4];
  __shared__ int hrow[2];
  __shared__ int nh_s;
  __shared__ float inv_rms[2];
  __shared__ int ex_in[kMaxSeq];
  __shared__ float bz_s[kRwWaves][2];
  __shared__ int bi_s[kRwWaves][2];
  __shared__ SkRmLds rmu;
  const RowMap& rml = rmu.rm;
  const int tid = threadIdx.x, lane = tid & 63, wv = __builtin_amdgcn_readfirstlane(tid >> 6), gw = blockIdx.x * kRwWaves + wv;
  const int esz = WB ? 2 : 4;
  auto row_ptr = [&](int u, int) -> const void* { return (const char*)lm_head + (size_t)u * D.d * esz; };
  int u0, u1;
  rw_range(D.V, gridDim.x * kRwWaves, gw, u0, u1);
  RwStream<WB, NCH, 1, NS> st;
  float bv[1];
  sk_bins_load(rm.M * 4, bin_d_at(ws, n_layers_run, 0, 0), kMaxRows * 4, bv);
  const int exv = ws.exited[min(tid, rm.nseq - 1)];
  // FLOPs-optimised form (Sec. 2.5): the fast row that exited emits its token
  // from the low-rank head, whose first factor k_lr_z has applied (lrz); the
  // LM head is then not streamed (one sequence: the flag is uniform)
  const bool lowrank = D.hr > 0 && head_b && rm.nseq == 1 && !rm.head_all && rm.M == 2 && rm.fast[1] &&
                       rm.slow_of[1] >= 0 && ws.exited[0] != 0;
  const int lv0 = u0, lv1 = u1;
  if (lowrank) u1 = u0;
  const float* X1 = ws.X + (size_t)(rm.M > 1 ? 1 : 0) * D.d;
  RwPieces<RwPM<WB, NCH, NS>::value> xp;
  rw_load_pieces<true>(ws.X, X1, final_norm, D.d, xp);
  struct Epi {
    struct Ops {};
    const Dims* D;
    const int* hrow;
    const float* ir;
    float* logits;
    int nh;
    float bz[2];
    int bi[2];
    __device__ void fetch(int, Ops&) const {}
    __device__ void run(int v, const float (&y)[1][2], const Ops&) {
      const int lane = threadIdx.x & 63;
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        if (k >= nh) continue;
        const float z = y[0][hrow[k]] * ir[k];
        if (logits && lane == k) logits[(size_t)k * D->V + v] = z;
        if (z > bz[k]) { bz[k] = z; bi[k] = v; }   // rows in increasing order: the lowest index wins ties
      }
    }
  } epi{&D, hrow, inv_rms, io.logits_out, 0, {-INFINITY, -INFINITY}, {0x7fffffff, 0x7fffffff}};
  typename Epi::Ops ops[decltype(st)::P];
  __builtin_amdgcn_sched_barrier(0);
  st.begin(row_ptr, u0, u1, epi, ops);
  __builtin_amdgcn_sched_barrier(0);
  if (tid < rm.nseq) ex_in[tid] = exv;
  sk_rm_copy(rmu, rm);
  sk_bins_sum(rm.M * 4, bv, actf, ssum);
  if (tid == 0) {
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
    for (int k = 0; k < 2; ++k) inv_rms[k] = rsqrtf(ssum[hrow[min(k, nh - 1)] * 4] / D.d + D.eps);
  }
  __syncthreads();
  const int nh = nh_s;
  // head row k reads activation row hrow[k] (the staged rows are X[0] and X[1])
  rw_store_pieces<true>(xp, D.d, actf);
  epi.nh = nh;
  st.run(row_ptr, u0, u1, actf, D.d, epi, ops);
  if (lowrank) {
    // logits z_v = head_b[v] . lrz for this wave's rows, one row per lane
    const int hr = D.hr;
    for (int j = tid; j < hr; j += kRwThreads) actf[j] = ws.lrz[j];
    __syncthreads();
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int v0 = lv0; v0 < lv1; v0 += 64) {
      const int v = v0 + lane;
      if (v < lv1) {
        float z = 0.f;
        for (int j = 0; j < hr; ++j) z += rw_wt<WB>(rw_wt_raw<WB>(head_b, (size_t)v * hr + j)) * actf[j];
        if (io.logits_out) io.logits_out[v] = z;
        if (z > bz) { bz = z; bi = v; }   // each lane's rows rise: the lowest index wins its ties
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float z2 = __shfl_xor(bz, o);
      const int i2 = __shfl_xor(bi, o);
      if (z2 > bz || (z2 == bz && i2 < bi)) { bz = z2; bi = i2; }
    }
    epi.bz[0] = bz;
    epi.bi[0] = bi;
  }
  if (lane == 0) {
    bz_s[wv][0] = epi.bz[0]; bz_s[wv][1] = epi.bz[1];
    bi_s[wv][0] = epi.bi[0]; bi_s[wv][1] = epi.bi[1];
  }
  __syncthreads();
  if (tid < 2) {
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int w = 0; w < kRwWaves; ++w) {
      const float z = bz_s[w][tid];
      const int i = bi_s[w][tid];
      if (z > bz || (z == bz && i < bi)) { bz = z; bi = i; }
    }
    st_agent(&ws.lm_val[(size_t)blockIdx.x * kMaxRows + tid], bz);
    st_agent(&ws.lm_idx[(size_t)blockIdx.x * kMaxRows + tid], bi);
  }
  if (wv != 0) return;
  if (!sk_arrive_all(sk, blockIdx.x, gridDim.x)) return;

  // ---- the last workgroup (wave 0): global arg-max per head row, then bookkeeping
  const int G = gridDim.x;
  int best[2] = {0, 0};
  for (int k = 0; k < nh; ++k) {
    float bz = -INFINITY;
    int bi = 0x7fffffff;
    for (int t0 = 0; t0 < G; t0 += 64 * 8) {
      float zv[8];
      int iv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int t = min(t0 + lane + 64 * u, G - 1);
        zv[u] = ld_agent(&ws.lm_val[(size_t)t * kMaxRows + k]);
        iv[u] = ld_agent(&ws.lm_idx[(size_t)t * kMaxRows + k]);
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
    best[k] = bi;
  }
  if (rm.head_all) {
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
  if (lane < rm.nseq) {
    const int sq = lane;
    const int f = rml.first[sq] + rml.cnt[sq] - 1;
    io.next_token[sq + io.draft_slot] = best[sq];
    const int t = io.positions[sq] + rm.pos_offset;
    if (rml.slow_of[f] >= 0 || !rml.fast[f]) kv.seq_lens[sq] = t + 1;
    if (rml.fast[f] && rml.slow_of[f] >= 0) {
      const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
      ws.sig[sq * D.n_layers + D.n_layers - 1] = ws.exited[sq] ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
    }
    if (io.exit_b_out) io.exit_b_out[sq] = ws.exitb[sq];
    if (io.advance) io.positions[sq] = io.positions[sq] + 1;
  }
  if (io.signal_out) {
    for (int q = lane; q < rm.nseq * D.n_layers; q += 64) {
      const int sq = q / D.n_layers, l = q % D.n_layers;
      const int f = rml.first[sq] + rml.cnt[sq] - 1;
      float v = ws.sig[q];
      if (l == D.n_layers - 1) {   // written above by another lane: recomputed here
        const float dot = ssum[f * 4 + 1], pin2 = ssum[f * 4 + 2], pp = ssum[f * 4 + 0];
        v = ws.exited[sq] ? 0.f : dot * rsqrtf(fmaxf(pin2 * pp, 1e-30f));
      }
      if (!rml.fast[f] || rml.slow_of[f] < 0 || (ws.exited[sq] && l >= ws.exitb[sq])) v = 0.f;
      io.signal_out[q] = v;
    }
  }
  if (io.h_out || io.p_out) {
    for (int q = lane; q < rm.nseq * D.d; q += 64) {
      const int sq = q / D.d, i = q % D.d;
      const int f = rml.first[sq], c = rml.cnt[sq];
      if (io.h_out) io.h_out[q] = ws.X[(size_t)f * D.d + i];
      if (io.p_out) io.p_out[q] = ws.X[(size_t)(f + c - 1) * D.d + i];
    }
  }
}

}  // namespace m2r2
