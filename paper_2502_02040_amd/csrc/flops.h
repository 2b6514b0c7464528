// FLOPs-optimised accelerated stream (Sec. 2.5), one sequence: the fast row
// keeps its first fast_heads heads; fast head j attends to the fast_topk
// cached positions that the slow row's head j scores highest at the same
// layer (ties to the lower position), plus its own key and value; its MLP is
// the rank-r adapter alone; a token it emits comes from a low-rank head.
//
// Kernels (launched by the multi-kernel one- and two-row pass):
//  * ks_attn, in this form, leaves the fast row out of the split attention
//    (its partials carry no weight, so the merge writes a zero attention
//    output and o-adapter share for it), stores the slow row's scaled scores
//    of the cached positions of heads < fast_heads (ws.fsc) and the fast
//    row's q, k (after RoPE) and v of those heads (ws.fqkv).
//  * k_fattn, one workgroup per kept head, after ks_attn: selects the
//    positions (radix select over order-preserving keys of the scores, then
//    the lowest positions among the keys equal to the threshold), attends
//    over them and the own key/value, and overwrites the fast row's attention
//    output and o-adapter share of the head.
//  * k_fast_mlp (the mixture-of-experts fast MLP kernel) applies the MLP
//    adapter; the gate/up and down kernels then run on the slow row alone.
//  * k_lr_z: when the fast row exited at a gate (EXIT mode), its first
//    low-rank factor: lrz = head_a (rms(p) * final_norm); kr_head then takes
//    the logits head_b lrz instead of streaming the LM head.
#pragma once
#include "sk_attn.h"

namespace m2r2 {

constexpr int kFaThreads = 256;     // 64 token slots x 4 lanes, as in the split attention
constexpr int kFaMaxCtx = 16384;    // cached positions a kept head selects from (LDS: 8 bytes each)

__host__ __device__ constexpr size_t fattn_lds_bytes(int cap) { return (size_t)cap * 8; }

// Order-preserving key of a score: a larger score has a larger key.
__device__ __forceinline__ uint32_t fa_key(float s) {
  const uint32_t b = __float_as_uint(s);
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}

// Exclusive prefix sum over the block (kFaThreads threads, one value each);
// *total receives the sum.  tmp holds 4 ints.  Contains workgroup barriers.
__device__ __forceinline__ int fa_scan(int v, int* tmp, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(inc, o);
    if (lane >= o) inc += t;
  }
  __syncthreads();   // tmp may still be read by the previous scan
  if (lane == 63) tmp[w] = inc;
  __syncthreads();
  int base = 0;
  for (int i = 0; i < w; ++i) base += tmp[i];
  *total = tmp[0] + tmp[1] + tmp[2] + tmp[3];
  return base + inc - v;
}

// grid = fast heads, block = kFaThreads, dynamic LDS = fattn_lds_bytes(rope_len).
template <int KB, int HD>
__global__ __launch_bounds__(kFaThreads) void k_fattn(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, KVPtrs kv,
                                                     int layer) {
  extern __shared__ __attribute__((aligned(16))) uint32_t fa_dyn[];
  constexpr int DPL = HD / 4;                  // dims per lane, 4 lanes per token
  constexpr int KESZ = KB ? 2 : 4;
  constexpr int NCH = DPL * KESZ / 16;         // 16-byte pieces per lane and token
  __shared__ float q_s[HD], k_s[HD], v_s[HD], o_s[HD];
  __shared__ float pvred[16][HD];
  __shared__ int hist[256];
  __shared__ int tmp[4];
  __shared__ int dig_s, gt_s;
  __shared__ float red[4];
  __shared__ float own_s;
  const int h = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (ws.exited[0]) return;   // exited at a gate (EXIT mode): the fast row is done
  const int fr = rm.M - 1;    // the fast row (rows: slow, fast)
  const int cap = ws.rope_len;
  const int n = min(max(io.positions[0] + rm.pos_offset, 0), cap);   // cached positions [0, n)
  uint32_t* key = fa_dyn;                  // [cap] keys, later the selected positions' weights
  int* sel = (int*)(fa_dyn + cap);         // [cap] selected positions, increasing
  const float* scg = ws.fsc + (size_t)h * cap;
  if (tid < HD) {
    const float* f = ws.fqkv + (size_t)h * 3 * HD;
    q_s[tid] = f[tid];
    k_s[tid] = f[HD + tid];
    v_s[tid] = f[2 * HD + tid];
  }
  // ---- the positions this head attends to -----------------------------------
  const int k = D.ftk;
  int nsel = n;
  if (k <= 0 || n <= k) {
    for (int t = tid; t < n; t += kFaThreads) sel[t] = t;
  } else {
    for (int t = tid; t < n; t += kFaThreads) key[t] = fa_key(scg[t]);
    // the k-th largest key, 8 bits at a time from the top
    uint32_t prefix = 0, mask = 0;
    int need = k;   // elements still to take at or below the prefix
    for (int shift = 24; shift >= 0; shift -= 8) {
      hist[tid] = 0;
      __syncthreads();
      for (int t = tid; t < n; t += kFaThreads) {
        const uint32_t u = key[t];
        if ((u & mask) == prefix) atomicAdd(&hist[(u >> shift) & 255], 1);
      }
      __syncthreads();
      if (wv == 0) {
        int c[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) c[i] = hist[4 * lane + i];
        const int s4 = c[0] + c[1] + c[2] + c[3];
        int incl = s4;   // sum over this lane and the lanes above it (higher digits)
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
          const int t = __shfl_down(incl, o);
          if (lane + o < 64) incl += t;
        }
        int acc = incl - s4;   // count in digits above this lane's four
#pragma unroll
        for (int i = 3; i >= 0; --i) {
          if (acc < need && acc + c[i] >= need) {   // exactly one digit of the block satisfies this
            dig_s = 4 * lane + i;
            gt_s = acc;
          }
          acc += c[i];
        }
      }
      __syncthreads();
      prefix |= (uint32_t)dig_s << shift;
      mask |= 255u << shift;
      need -= gt_s;
    }
    // keys above the threshold, then the `need` lowest positions equal to it
    const int per = (n + kFaThreads - 1) / kFaThreads;
    const int a = min(n, tid * per), b = min(n, a + per);
    int eq = 0;
    for (int t = a; t < b; ++t) eq += key[t] == prefix;
    int tot = 0;
    const int eq0 = fa_scan(eq, tmp, &tot);
    int cnt = 0;
    for (int t = a, e = eq0; t < b; ++t) {
      const uint32_t u = key[t];
      cnt += u > prefix || (u == prefix && e < need);
      e += u == prefix;
    }
    const int o0 = fa_scan(cnt, tmp, &tot);
    for (int t = a, e = eq0, o = o0; t < b; ++t) {
      const uint32_t u = key[t];
      if (u > prefix || (u == prefix && e < need)) sel[o++] = t;
      e += u == prefix;
    }
    nsel = tot;
  }
  __syncthreads();
  // ---- scores of the selected positions with the fast query -----------------
  float* wsel = (float*)key;   // [nsel] scores, then softmax weights
  const float scale = rsqrtf((float)HD);
  const int slot = tid >> 2, sub = tid & 3, d0 = sub * DPL;
  auto row_ix = [&](int t) {
    int b = kv.bt[min(t / kv.bs, kv.mbps - 1)];
    b = (b >= 0 && b < kv.num_blocks) ? b : 0;
    return ((((size_t)layer * kv.num_blocks + b) * D.H + h) * kv.bs + t % kv.bs) * HD + d0;
  };
  for (int i0 = 0; i0 < nsel; i0 += 64) {
    const int i = i0 + slot;
    float p = 0.f;
    if (i < nsel) {
      const size_t ix = row_ix(sel[i]);
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const u32x4_t kk = *(const u32x4_t*)((const char*)kv.k + ix * KESZ + 16 * c);
        if constexpr (KB) {
#pragma unroll
          for (int w = 0; w < 4; ++w)
            p += q_s[d0 + 8 * c + 2 * w] * bf16lo(kk[w]) + q_s[d0 + 8 * c + 2 * w + 1] * bf16hi(kk[w]);
        } else {
#pragma unroll
          for (int w = 0; w < 4; ++w) p += q_s[d0 + 4 * c + w] * __uint_as_float(kk[w]);
        }
      }
    }
    p = quad_sum(p);
    if (sub == 0 && i < nsel) wsel[i] = p * scale;
  }
  if (wv == 0) {   // the own key: exact (the fast row's key/value are never cached)
    float p = 0.f;
    for (int dd = lane; dd < HD; dd += 64) p += q_s[dd] * k_s[dd];
    p = wave_sum(p);
    if (lane == 0) own_s = p * scale;
  }
  __syncthreads();
  const float own = own_s;
  float mx = own;
  for (int i = tid; i < nsel; i += kFaThreads) mx = fmaxf(mx, wsel[i]);
  mx = block_max(mx, red);
  float ls = 0.f;
  for (int i = tid; i < nsel; i += kFaThreads) {
    const float e = __expf(wsel[i] - mx);
    wsel[i] = e;
    ls += e;
  }
  const float eo = __expf(own - mx);
  ls = block_sum(ls, red) + eo;   // (block_sum ends with the weights visible to every thread)
  // ---- weighted values ----------------------------------------------------------
  float acc[DPL];
#pragma unroll
  for (int c = 0; c < DPL; ++c) acc[c] = 0.f;
  for (int i0 = 0; i0 < nsel; i0 += 64) {
    const int i = i0 + slot;
    if (i < nsel) {
      const float pw = wsel[i];
      const size_t ix = row_ix(sel[i]);
#pragma unroll
      for (int c = 0; c < NCH; ++c) {
        const u32x4_t vv = *(const u32x4_t*)((const char*)kv.v + ix * KESZ + 16 * c);
        if constexpr (KB) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            acc[8 * c + 2 * w] += pw * bf16lo(vv[w]);
            acc[8 * c + 2 * w + 1] += pw * bf16hi(vv[w]);
          }
        } else {
#pragma unroll
          for (int w = 0; w < 4; ++w) acc[4 * c + w] += pw * __uint_as_float(vv[w]);
        }
      }
    }
  }
  // sum over the 4 token slots of a 16-lane row (DPP), then the 16 row partials
#pragma unroll
  for (int c = 0; c < DPL; ++c) acc[c] = row_sum_stride4(acc[c]);
  if ((lane & 15) < 4) {
    const int g = wv * 4 + (lane >> 4);
#pragma unroll
    for (int c = 0; c < DPL; ++c) pvred[g][d0 + c] = acc[c];
  }
  __syncthreads();
  if (tid < HD) {
    float o = eo * v_s[tid];
#pragma unroll
    for (int g = 0; g < 16; ++g) o += pvred[g][tid];
    o /= ls;
    o_s[tid] = o;
    ws.O[(size_t)fr * D.qdim + h * HD + tid] = o;
  }
  __syncthreads();
  // the head's share of the o-adapter down-projection of the fast row:
  // uo[fr][h][j] = sum_d A_o[j][h*HD + d] o[d]
  if (L.A[3]) {
    for (int j = wv; j < D.r; j += kFaThreads / 64) {
      float a = 0.f;
      for (int dd = lane; dd < HD; dd += 64) {
        const size_t e = (size_t)j * D.qdim + h * HD + dd;
        a += (D.wbf16 ? bf16_to_f32(((const uint16_t*)L.A[3])[e]) : ((const float*)L.A[3])[e]) * o_s[dd];
      }
      a = wave_sum(a);
      if (lane == 0) ws.uo[((size_t)fr * D.H + h) * D.r + j] = a;
    }
  }
}

// First factor of the low-rank head for a fast row that exited: lrz[j] =
// head_a[j] . (p * final_norm) / rms(p).  grid = ceil(head_rank / 8),
// block = 512 (a wave per row), dynamic LDS = d floats.
template <int WB>
__global__ __launch_bounds__(512) void k_lr_z(Dims D, const float* final_norm, const void* head_a, RowMap rm, WS ws) {
  extern __shared__ __attribute__((aligned(16))) float lz_x[];
  __shared__ float red[8];
  if (!ws.exited[0]) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const float* p = ws.X + (size_t)(rm.M - 1) * D.d;
  float ss = 0.f;
  for (int i = tid; i < D.d; i += 512) {
    const float x = p[i];
    ss += x * x;
    lz_x[i] = x * final_norm[i];
  }
  ss = block_sum(ss, red);
  const float inv = rsqrtf(ss / D.d + D.eps);
  const int j = blockIdx.x * 8 + wv;
  if (j >= D.hr) return;
  float a = 0.f;
  for (int i = lane; i < D.d; i += 64) {
    const size_t e = (size_t)j * D.d + i;
    a += (WB ? bf16_to_f32(((const uint16_t*)head_a)[e]) : ((const float*)head_a)[e]) * lz_x[i];
  }
  a = wave_sum(a);
  if (lane == 0) ws.lrz[j] = a * inv;
}

}  // namespace m2r2
