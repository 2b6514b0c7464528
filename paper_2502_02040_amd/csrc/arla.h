// Latent-attention exit router (Sec. 2.3.1, "Accelerated Residual Latent
// Attention"; Fig. 4a) on the fast row of a one-sequence decode step.
//
// The interval of a gate b that follows gate g (or the start of the step,
// g = 0) holds the state the fast row restarts from at g (the slow state
// there; the token embedding for g = 0) and the fast state after each of the
// layers g .. b-1.  Every state is normalised to unit RMS (no gain) and
// projected into a 64-wide latent key and value with boundary b's matrices:
// the restart state by the launch that precedes layer g (the one before
// layer 0, or the one after layer g-1, while the slow row still holds it),
// the fast states by the launch after their layer.  The launch after layer
// b-1 also projects the latent query of the newest state; its last
// workgroup then attends from that query over the interval's keys and
// values (softmax, scale 1/8) and reads the pooled value out through a
// linear map and a sigmoid.  The next layer's gate logic takes that
// probability in place of the cosine signal.  The paper leaves the query,
// the normalisation and the readout open; the choices here are the ones the
// oracle states.
//
// Bytes per launch: 128 to 320 latent rows of d weights, plus one or two
// residual rows; a few hundred KB against the layer's hundreds of MB, so the
// kernel is bound by its launch and the one reduction per workgroup.
#pragma once
#include "device_common.h"
#include "step_kernels.h"

namespace m2r2 {

constexpr int kArlaDim = 64;
constexpr int kArlaThreads = 256;
constexpr int kArlaWaves = kArlaThreads / 64;

constexpr int kArlaMaxJobs = 5;

// 64 latent rows: W [64][d] (weight dtype, row-major) applied to the
// RMS-normalised residual row X[row]; the results go to ws.arla_kv + dst, or
// to the query ws.arla_q when dst < 0.
struct ArlaJob {
  const void* w;
  int row;
  int dst;
};

// Latent slots in ws.arla_kv, 2 x 64 floats each (key, then value): slot l
// (l < n_layers) holds the fast state after layer l, slot n_layers + g the
// state the fast row restarts from at gate g (g = 0: the embedding).
struct ArlaArgs {
  ArlaJob job[kArlaMaxJobs];
  int njobs;
  const float* w_out;  // [64] readout of the gate's boundary
  const float* b_out;  // the boundary's bias
  int layer;           // the layer just finished (-1: before layer 0)
  int first;           // the gate that opens the interval (0: the step's start)
  int gate_now;        // layer + 1 is a gate: score it after the projections
};

// grid = njobs * 16 workgroups of four waves, one wave per latent row; the
// 16 workgroups of a job share its residual row.
template <int WB>
__global__ __launch_bounds__(kArlaThreads) void k_arla(Dims D, WS ws, ArlaArgs a) {
  __shared__ float red[kArlaWaves];
  __shared__ int last_flag;
  if (ws.exited[0]) return;   // EXIT mode after the exit: nothing reads the router any more
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  constexpr int kBlocksPerJob = kArlaDim / kArlaWaves;
  const ArlaJob& jb = a.job[blockIdx.x / kBlocksPerJob];
  const float* x = ws.X + (size_t)jb.row * D.d;
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
  const int j = (blockIdx.x % kBlocksPerJob) * kArlaWaves + wave;   // latent row of the job
  {
    const char* wr = (const char*)jb.w + (size_t)j * D.d * (WB ? 2 : 4);
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
    if (lane == 0) st_agent(jb.dst >= 0 ? &ws.arla_kv[(size_t)jb.dst + j] : &ws.arla_q[j], acc);
  }
  if (!a.gate_now) return;
  if (!arrive_last(ws.arla_cnt, gridDim.x, &last_flag)) return;
  if (wave != 0) return;
  // lane j holds latent component j: scores by wave reductions, the softmax
  // in two passes (maximum, then the weighted sum); the interval is the
  // restart slot of gate `first`, then the slots of layers first .. layer
  const float q = ld_agent(&ws.arla_q[lane]);
  auto slot = [&](int s) {
    return ws.arla_kv + (size_t)(s < a.first ? D.n_layers + a.first : s) * 2 * kArlaDim;
  };
  float m = -INFINITY;
  for (int s = a.first - 1; s <= a.layer; ++s) m = fmaxf(m, wave_sum(q * ld_agent(slot(s) + lane)) * 0.125f);
  float den = 0.f, ov = 0.f;
  for (int s = a.first - 1; s <= a.layer; ++s) {
    const float* kv = slot(s);
    const float e = __expf(wave_sum(q * ld_agent(kv + lane)) * 0.125f - m);
    den += e;
    ov += e * ld_agent(kv + kArlaDim + lane);
  }
  const float logit = wave_sum(a.w_out[lane] * (ov / den)) + a.b_out[0];
  if (lane == 0) ws.arla_sig[0] = 1.f / (1.f + __expf(-logit));
}

}  // namespace m2r2
