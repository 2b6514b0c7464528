// Latent-attention exit router (Sec. 2.3.1, "Accelerated Residual Latent
// Attention"; Fig. 4a) on the fast row of a one-sequence decode step.
//
// After every layer l whose next gate b exists, the fast state p (X row of
// the fast row, after the layer, before the gate restarts it) is normalised
// to unit RMS (no gain) and projected into a 64-wide latent key and value
// with boundary b's matrices; they are kept per layer.  After layer b-1 the
// kernel also projects the latent query; the last workgroup to arrive then
// attends from that query over the keys and values of layers
// [previous gate (or 0), b-1] (softmax, scale 1/8) and reads the pooled value
// out through a linear map and a sigmoid.  The next layer's gate logic takes
// that probability in place of the cosine signal.  The paper leaves the
// query, the normalisation and the readout open; the choices here are the
// ones the oracle states.
//
// Bytes per launch: 128 (192 at a gate) latent rows of d weights, plus the
// fast row; a few hundred KB against the layer's hundreds of MB, so the
// kernel is bound by its launch and the one reduction per workgroup.
#pragma once
#include "device_common.h"
#include "step_kernels.h"

namespace m2r2 {

constexpr int kArlaDim = 64;
constexpr int kArlaThreads = 256;
constexpr int kArlaWaves = kArlaThreads / 64;

struct ArlaArgs {
  const void* wq;      // [64][d] of the boundary, weight dtype, row-major
  const void* wk;
  const void* wv;
  const float* w_out;  // [64] readout of the boundary
  const float* b_out;  // the boundary's bias
  int row;             // X row of the fast state
  int layer;           // the layer just finished
  int first;           // first layer of the gate's interval
  int gate_now;        // layer + 1 is the gate: project the query and score
};

// grid = ceil((gate_now ? 192 : 128) / 4) workgroups, one wave per latent row.
template <int WB>
__global__ __launch_bounds__(kArlaThreads) void k_arla(Dims D, WS ws, ArlaArgs a) {
  __shared__ float red[kArlaWaves];
  __shared__ int last_flag;
  if (ws.exited[0]) return;   // EXIT mode after the exit: nothing reads the router any more
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const float* x = ws.X + (size_t)a.row * D.d;
  // groups of 8 elements (16 B of bf16 weights, 32 B of fp32 ones), four
  // groups per lane in flight at a time, when every row starts 16-byte
  // aligned (d a multiple of 8); otherwise element by element
  const int ng = D.d % 8 == 0 ? D.d / 8 : 0;
  float ss = 0.f;
  for (int g = tid; g < ng; g += kArlaThreads) {
    const float4 u = ld4(x + 8 * g), v = ld4(x + 8 * g + 4);
    ss += u.x * u.x + u.y * u.y + u.z * u.z + u.w * u.w + v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  for (int i = 8 * ng + tid; i < D.d; i += kArlaThreads) ss += x[i] * x[i];
  const float inv = rsqrtf(block_sum(ss, red) / D.d + D.eps);
  const int n_out = (a.gate_now ? 3 : 2) * kArlaDim;
  const int o = blockIdx.x * kArlaWaves + wave;
  if (o < n_out) {
    const int mat = o / kArlaDim, j = o % kArlaDim;
    const void* W = mat == 0 ? a.wk : (mat == 1 ? a.wv : a.wq);
    const char* wr = (const char*)W + (size_t)j * D.d * (WB ? 2 : 4);
    float acc = 0.f;
    for (int g0 = 0; g0 < ng; g0 += 4 * 64) {
      float w[4][8];
      float4 xa[4], xb[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int g = min(g0 + u * 64 + lane, ng - 1);   // clamped: valid address, product dropped below
        xa[u] = ld4(x + 8 * g);
        xb[u] = ld4(x + 8 * g + 4);
        if constexpr (WB) {
          const u32x4_t r = *(const u32x4_t*)(wr + (size_t)g * 16);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            w[u][2 * e] = bf16lo(r[e]);
            w[u][2 * e + 1] = bf16hi(r[e]);
          }
        } else {
          const float4 p = ld4((const float*)wr + 8 * g), q = ld4((const float*)wr + 8 * g + 4);
          w[u][0] = p.x; w[u][1] = p.y; w[u][2] = p.z; w[u][3] = p.w;
          w[u][4] = q.x; w[u][5] = q.y; w[u][6] = q.z; w[u][7] = q.w;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float4 p = xa[u], q = xb[u];
        const float d8 = w[u][0] * p.x + w[u][1] * p.y + w[u][2] * p.z + w[u][3] * p.w + w[u][4] * q.x +
                         w[u][5] * q.y + w[u][6] * q.z + w[u][7] * q.w;
        acc += g0 + u * 64 + lane < ng ? d8 : 0.f;
      }
    }
    for (int i = 8 * ng + lane; i < D.d; i += 64) {
      const float w = WB ? bf16_to_f32(((const uint16_t*)wr)[i]) : ((const float*)wr)[i];
      acc += w * x[i];
    }
    acc = wave_sum(acc) * inv;
    if (lane == 0) {
      if (mat < 2) st_agent(&ws.arla_kv[(size_t)a.layer * 2 * kArlaDim + o], acc);
      else st_agent(&ws.arla_q[j], acc);
    }
  }
  if (!a.gate_now) return;
  if (!arrive_last(ws.arla_cnt, gridDim.x, &last_flag)) return;
  if (wave != 0) return;
  // lane j holds latent component j: scores by wave reductions, the softmax
  // in two passes (maximum, then the weighted sum)
  const float q = ld_agent(&ws.arla_q[lane]);
  float m = -INFINITY;
  for (int l = a.first; l <= a.layer; ++l)
    m = fmaxf(m, wave_sum(q * ld_agent(&ws.arla_kv[(size_t)l * 2 * kArlaDim + lane])) * 0.125f);
  float den = 0.f, ov = 0.f;
  for (int l = a.first; l <= a.layer; ++l) {
    const float* kv = ws.arla_kv + (size_t)l * 2 * kArlaDim;
    const float e = __expf(wave_sum(q * ld_agent(kv + lane)) * 0.125f - m);
    den += e;
    ov += e * ld_agent(kv + kArlaDim + lane);
  }
  const float logit = wave_sum(a.w_out[lane] * (ov / den)) + a.b_out[0];
  if (lane == 0) ws.arla_sig[0] = 1.f / (1.f + __expf(-logit));
}

}  // namespace m2r2
