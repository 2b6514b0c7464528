// Shared-KV decode attention for one or two rows per sequence (the slow and
// fast row of the dual-stream step, one row of plain decoding or drafting,
// or two rows of a short verification chunk), written to keep the chain of
// dependent memory round trips short.
//
// The cached context [0, ctx) of a sequence is cut into fixed splits of
// kSkAttnP tokens over the whole cache capacity, so a split's block-table
// entries are loaded together with the position, the projection outputs, the
// adapter factors and the A_o rows (round one); its keys, values and the
// RoPE table entries follow in round two.  The split holding position ctx
// also forms the rows' own keys and values (adapter-up and RoPE), writes the
// slow rows' key/value to the paged cache and adds the own-key terms: a slow
// row sees the chunk's slow rows up to itself (their cached, rounded values),
// a fast row only its own exact key/value (shared-KV attention of the fast
// stream).  Each split stores its softmax partial (max, sum, unnormalised
// accumulator); the last split of a (sequence, head) to arrive merges them
// (online-softmax combine), writes the attention output and, for fast rows,
// the head's share of the o-adapter down-projection A_o[:, head] o.
#pragma once
#include "sk_kernels.h"

namespace m2r2 {

constexpr int kSkAttnP = 128;        // tokens per split
constexpr int kSkAttnThreads = 256;  // 64 token slots x 4 lanes

// Dynamic LDS: the head's rows of B_q, B_k, B_v (raw weights).
__host__ __device__ constexpr int sk_attn_lds_bytes(int hd, int r, int wb) { return 3 * hd * r * (wb ? 2 : 4); }

template <int WB, int KB, int HD, int NC = 1>
__global__ __launch_bounds__(kSkAttnThreads) void ks_attn(Dims D, LayerPtrs L, RowMap rm, WS ws, StepIO io, KVPtrs kv,
                                                          int layer, int S) {
  // NC chunks of kSkAttnP tokens per split: the next chunk's keys (values)
  // are loaded while the current chunk's softmax (next scores) runs, and the
  // chunks are combined online (running max, sum and accumulator per row)
  extern __shared__ __attribute__((aligned(16))) char bsl[];   // [3][HD][r] raw B rows of q, k, v
  constexpr int DPL = HD / 4;                                  // dims per lane, 4 lanes per token
  constexpr int KESZ = KB ? 2 : 4;
  constexpr int NCH = DPL * KESZ / 16;                         // 16-byte pieces per lane and token
  constexpr int TPT = kSkAttnP / 64;                           // tokens per thread and chunk
  constexpr int SPL = NC * kSkAttnP;                           // tokens per split
  constexpr int WESZ = WB ? 2 : 4;
  __shared__ float q_s[2][HD], k_s[2][HD], v_s[2][HD];
  __shared__ float u_s[2][3][kMaxRank];
  __shared__ float sc[2][kSkAttnP + 2];
  __shared__ float lastw[2];   // weight of the last chunk's terms in the combined partial
  __shared__ float fin_m[2], fin_l[2];   // the combined partial's max and sum per row
  __shared__ float red[4][2][HD];
  __shared__ float pvred[16][2][HD];
  __shared__ float rowm[2], rowl[2];
  __shared__ float mw[2][64];
  __shared__ float linv[2];
  __shared__ float uop[kMaxRank * (HD / 8)];
  __shared__ SkRmLds rmu;
  __shared__ int last_flag;
  const RowMap& rml = rmu.rm;
  const int sp = blockIdx.x, h = blockIdx.y, sq = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int slot = tid >> 2, sub = tid & 3, d0 = sub * DPL;
  const int r = D.r, qd = D.qdim, nqkv = 3 * qd + 3 * r;
  const float scale = rsqrtf((float)HD);

  // ---- round one: everything that does not depend on the position ----------
  const int posv = io.positions[sq];
  const int exv = ws.exited[sq];
  int blk[NC][TPT];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int it = 0; it < TPT; ++it) {
      const int tp = sp * SPL + c * kSkAttnP + slot + 64 * it;
      blk[c][it] = kv.bt[sq * kv.mbps + min(tp / kv.bs, kv.mbps - 1)];
    }
  // projection outputs of row m = e / HD, dim d = e % HD (rows of this
  // sequence: the map is read below; row indices are clamped to the batch)
  const int e_m = min(tid / HD, 1), e_d = tid % HD;
  // first row of sequence sq (scalar: constant-index reads of the map, a
  // uniform select; the sequence's rows are [first, first + cnt))
  int prow0 = rm.first[0];
#pragma unroll
  for (int i = 1; i < kMaxSeq; ++i) prow0 = sq == i ? (int)rm.first[i] : prow0;
  float pv[3];
  {
    const int row = min(prow0 + e_m, rm.M - 1);
#pragma unroll
    for (int w = 0; w < 3; ++w) pv[w] = ws.QKV[(size_t)row * nqkv + w * qd + h * HD + e_d];
  }
  float uv = 0.f;
  {
    const int q = min(tid, 2 * 3 * r - 1);
    const int row = min(prow0 + q / (3 * r), rm.M - 1);
    uv = ws.QKV[(size_t)row * nqkv + 3 * qd + q % (3 * r)];
  }
  // B rows of q, k, v for this head: 16-byte pieces (projection w at constant
  // indices: a runtime index into the pointer array is a dependent load)
  const int ppieces = HD * r * WESZ / 16;   // pieces per projection (<= 2 * kSkAttnThreads)
  u32x4_t bp[3][2];
#pragma unroll
  for (int w = 0; w < 3; ++w) {
    const u32x4_t* B = (const u32x4_t*)((const char*)(L.B[w] ? L.B[w] : (const void*)ws.QKV) + (size_t)h * HD * r * WESZ);
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int o = min(tid + kSkAttnThreads * k, ppieces - 1);
      bp[w][k] = L.B[w] ? B[o] : u32x4_t{0u, 0u, 0u, 0u};
    }
  }
  // A_o[j][h*HD + 8c .. +8) (bf16), for the o-adapter share of the merge
  const int apieces = r * HD / 8;
  u32x4_t ap[2];
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int i = min(tid + kSkAttnThreads * k, apieces - 1);
    const int j = i / (HD / 8), c = i % (HD / 8);
    ap[k] = (WB && L.A[3]) ? *(const u32x4_t*)((const uint16_t*)L.A[3] + (size_t)j * qd + h * HD + 8 * c)
                           : u32x4_t{0u, 0u, 0u, 0u};
  }

  // ---- round-one values into LDS (the wait for them drains nothing else) ------
  sk_rm_copy(rmu, rm);
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const int o = tid + kSkAttnThreads * k;
      if (o < ppieces) ((u32x4_t*)bsl)[w * ppieces + o] = bp[w][k];
    }
  if (tid < 2 * 3 * r) u_s[tid / (3 * r)][(tid % (3 * r)) / r][tid % r] = uv;
  __syncthreads();
  const int first = rml.first[sq], R = rml.cnt[sq];
  const int ctx = posv + rm.pos_offset;
  // FLOPs-optimised form (Sec. 2.5, one sequence): the fast row attends in
  // k_fattn; here its partials carry no weight, the slow row's scores of the
  // kept heads and the fast row's q, k, v of those heads are stored for it
  const bool flops = (D.fh > 0 || D.ftk > 0) && R == 2 && rml.fast[first + 1];
  const bool fkeep = flops && h < (D.fh > 0 ? D.fh : D.H);
  const bool frozen = exv != 0;
  const int t0 = sp * SPL;
  const int own_sp = min(ctx / SPL, S - 1);
  const bool own = sp == own_sp;
  // an exited sequence (EXIT mode): only the own split has work (the cache
  // entries of the slow rows); no split stores a partial or counts in
  if (frozen && !own) return;

  // ---- round two: the RoPE entry of this thread's row, then keys and values ---
  float2 cs;
  {
    int pos = ctx + rml.idx[min(first + e_m, rm.M - 1)];
    if (pos < 0 || pos >= ws.rope_len) {
      if (tid == 0) atomicOr(ws.err, 8);
      pos = 0;
    }
    cs = ws.rope[(size_t)pos * (HD / 2) + (e_d % (HD / 2))];
  }
  u32x4_t kr[TPT][NCH], vr[TPT][NCH];
  // keys (or values) of chunk ch into dst
  auto load_chunk = [&](const void* base, int ch, u32x4_t (&dst)[TPT][NCH]) {
#pragma unroll
    for (int it = 0; it < TPT; ++it) {
      const int tp = t0 + ch * kSkAttnP + slot + 64 * it;
      int b = blk[ch][it];
      b = (b >= 0 && b < kv.num_blocks) ? b : 0;
      const size_t ix = ((((size_t)layer * kv.num_blocks + b) * D.H + h) * kv.bs + tp % kv.bs) * HD + d0;
#pragma unroll
      for (int c = 0; c < NCH; ++c) dst[it][c] = *(const u32x4_t*)((const char*)base + ix * KESZ + 16 * c);
    }
  };
  load_chunk(kv.k, 0, kr);
  load_chunk(kv.v, 0, vr);

  // q (and k, v) before RoPE: base projection + adapter-up on fast rows
  const bool erow = tid < R * HD;
  const bool efast = erow && rml.fast[first + e_m];
  float pre[3];
#pragma unroll
  for (int w = 0; w < 3; ++w) {
    float a = pv[w];
    if (efast && L.A[w] && L.B[w]) {
      const char* br = bsl + ((size_t)w * HD + e_d) * r * WESZ;
#pragma unroll
      for (int j = 0; j < kMaxRank; ++j) {
        if (j >= r) break;
        const float b = WB ? bf16_to_f32(((const uint16_t*)br)[j]) : ((const float*)br)[j];
        a += b * u_s[e_m][w][j];
      }
    }
    pre[w] = a;
  }
  if (erow) {
    q_s[e_m][e_d] = pre[0];
    k_s[e_m][e_d] = pre[1];
    v_s[e_m][e_d] = pre[2];
  }
  __syncthreads();
  // RoPE on q and k (rotate-half pairs d, d + HD/2)
  float qr = 0.f, kr1 = 0.f;
  if (erow) {
    const int half = HD / 2, j = e_d % half;
    const float c = cs.x, sn = cs.y;
    const float qa = q_s[e_m][j], qb = q_s[e_m][j + half];
    const float ka = k_s[e_m][j], kb = k_s[e_m][j + half];
    qr = e_d < half ? qa * c - qb * sn : qb * c + qa * sn;
    kr1 = e_d < half ? ka * c - kb * sn : kb * c + ka * sn;
  }
  __syncthreads();
  if (erow) {
    q_s[e_m][e_d] = qr;
    k_s[e_m][e_d] = kr1;
  }
  __syncthreads();
  if (fkeep && own && erow && rml.fast[first + e_m]) {
    float* f = ws.fqkv + (size_t)h * 3 * HD;
    f[e_d] = q_s[e_m][e_d];
    f[HD + e_d] = k_s[e_m][e_d];
    f[2 * HD + e_d] = v_s[e_m][e_d];
  }

  // ---- own split: cache writes of the slow rows -----------------------------
  if (own && erow && rml.wr[first + e_m]) {
    const int pos = ctx + rml.idx[first + e_m];
    const int lb = pos / kv.bs;
    const bool okb = pos >= 0 && lb < kv.mbps;
    const int b = okb ? kv.bt[sq * kv.mbps + lb] : -1;
    if (!okb || b < 0 || b >= kv.num_blocks) {
      atomicOr(ws.err, 2);
    } else {
      const size_t ix = ((((size_t)layer * kv.num_blocks + b) * D.H + h) * kv.bs + pos % kv.bs) * HD + e_d;
      if (KB) {
        ((uint16_t*)kv.k)[ix] = (uint16_t)f32_to_bf16_bits(k_s[e_m][e_d]);
        ((uint16_t*)kv.v)[ix] = (uint16_t)f32_to_bf16_bits(v_s[e_m][e_d]);
      } else {
        ((float*)kv.k)[ix] = k_s[e_m][e_d];
        ((float*)kv.v)[ix] = v_s[e_m][e_d];
      }
    }
  }

  if (!frozen) {
    float m_run[2] = {-INFINITY, -INFINITY}, l_run[2] = {0.f, 0.f};
    float acc0[DPL], acc1[DPL];
#pragma unroll
    for (int c = 0; c < DPL; ++c) { acc0[c] = 0.f; acc1[c] = 0.f; }
#pragma unroll
    for (int ch = 0; ch < NC; ++ch) {
      const bool last = ch == NC - 1;
      const int nt = max(0, min(ctx, t0 + (ch + 1) * kSkAttnP) - (t0 + ch * kSkAttnP));   // cached tokens of the chunk
      // ---- scores of the chunk's cached tokens ------------------------------
#pragma unroll
      for (int it = 0; it < TPT; ++it) {
        const int j = slot + 64 * it;
        float kk[DPL];
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          if constexpr (KB) {
#pragma unroll
            for (int i = 0; i < 4; ++i) { kk[8 * c + 2 * i] = bf16lo(kr[it][c][i]); kk[8 * c + 2 * i + 1] = bf16hi(kr[it][c][i]); }
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) kk[4 * c + i] = __uint_as_float(kr[it][c][i]);
          }
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          float p = 0.f;
#pragma unroll
          for (int c = 0; c < DPL; ++c) p += q_s[i][d0 + c] * kk[c];
          p = quad_sum(p);
          if (sub == 0 && i < R) {
            const bool f = flops && rml.fast[first + i];
            sc[i][j] = (j < nt && !f) ? p * scale : -INFINITY;
            if (fkeep && !rml.fast[first + i] && j < nt)
              ws.fsc[(size_t)h * ws.rope_len + t0 + ch * kSkAttnP + j] = p * scale;
          }
        }
      }
      if (ch + 1 < NC) load_chunk(kv.k, ch + 1, kr);   // in flight during this chunk's softmax and P V
      // ---- own keys (own split, with the last chunk): slow rows see the
      // chunk's slow rows up to themselves (rounded as cached), a fast row
      // only its own exact key ------------------------------------------------
      if (own && last) {   // wave wv: row i = wv >> 1, own key jj = wv & 1
        const int i = wv >> 1, jj = wv & 1;
        if (i < R) {
          const int mi = first + i, mj = first + min(jj, R - 1);
          const bool vis = jj < R && !(flops && rml.fast[mi]) &&
                           (rml.fast[mi] ? (jj == i) : (!rml.fast[mj] && rml.idx[mj] <= rml.idx[mi]));
          const bool rnd = !rml.fast[mi];
          float p = 0.f;
          for (int d = lane; d < HD; d += 64) {
            const float kk = k_s[min(jj, R - 1)][d];
            p += q_s[i][d] * (rnd && KB ? round_bf16(kk) : kk);
          }
          p = wave_sum(p);
          if (lane == 0) sc[i][kSkAttnP + jj] = vis ? p * scale : -INFINITY;
        }
      }
      __syncthreads();
      // ---- softmax of the chunk per row (wave i handles row i) ---------------
      const int ntot = kSkAttnP + (own && last ? 2 : 0);
      if (wv < R) {
        const int i = wv;
        float mx = -INFINITY;
        for (int j = lane; j < ntot; j += 64) mx = fmaxf(mx, sc[i][j]);
        mx = wave_max(mx);
        float l = 0.f;
        for (int j = lane; j < ntot; j += 64) {
          const float z = sc[i][j];
          const float ev = z == -INFINITY ? 0.f : __expf(z - mx);
          sc[i][j] = ev;
          l += ev;
        }
        l = wave_sum(l);
        if (lane == 0) { rowm[i] = l > 0.f ? mx : -INFINITY; rowl[i] = l; }
      }
      __syncthreads();
      // ---- P V of the chunk, combined with the chunks before ------------------
      float wc[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const float mc = rowm[min(i, R - 1)], lc = rowl[min(i, R - 1)];
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
#pragma unroll
      for (int it = 0; it < TPT; ++it) {
        const int j = slot + 64 * it;
        const float p0 = sc[0][j] * wc[0], p1 = R > 1 ? sc[1][j] * wc[1] : 0.f;
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
          if constexpr (KB) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float a = bf16lo(vr[it][c][i]), b = bf16hi(vr[it][c][i]);
              acc0[8 * c + 2 * i] += p0 * a; acc0[8 * c + 2 * i + 1] += p0 * b;
              acc1[8 * c + 2 * i] += p1 * a; acc1[8 * c + 2 * i + 1] += p1 * b;
            }
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const float a = __uint_as_float(vr[it][c][i]);
              acc0[4 * c + i] += p0 * a;
              acc1[4 * c + i] += p1 * a;
            }
          }
        }
      }
      if (ch + 1 < NC) {
        load_chunk(kv.v, ch + 1, vr);   // in flight during the next chunk's scores
        __syncthreads();                 // the next chunk's scores overwrite sc
      } else if (tid < 2) {
        lastw[tid] = wc[tid];
      }
    }
    if (tid < 2) { fin_m[tid] = m_run[tid]; fin_l[tid] = l_run[tid]; }
    // sum over the 4 token slots of a row (DPP), then the 16 row partials
    // (4 rows of 16 lanes x 4 waves) through LDS
#pragma unroll
    for (int c = 0; c < DPL; ++c) {
      acc0[c] = row_sum_stride4(acc0[c]);
      acc1[c] = row_sum_stride4(acc1[c]);
    }
    if ((lane & 15) < 4) {
      const int g = wv * 4 + (lane >> 4);
#pragma unroll
      for (int c = 0; c < DPL; ++c) {
        pvred[g][0][d0 + c] = acc0[c];
        pvred[g][1][d0 + c] = acc1[c];
      }
    }
    __syncthreads();
    // own keys' values: slow rows their rounded cached values, fast rows exact
    for (int e = tid; e < R * HD; e += kSkAttnThreads) {
      const int i = e / HD, d = e % HD;
      float a = 0.f;
#pragma unroll
      for (int g = 0; g < 16; ++g) a += pvred[g][i][d];
      if (own) {
        const bool rnd = !rml.fast[first + i];
        for (int jj = 0; jj < R; ++jj) {
          const float w = sc[i][kSkAttnP + jj] * lastw[i];
          if (w != 0.f) a += w * (rnd && KB ? round_bf16(v_s[jj][d]) : v_s[jj][d]);
        }
      }
      // partial: [m, l, acc[HD]] per row
      float* pp = ws.att + ((((size_t)sq * D.H + h) * (S + 1) + sp) * kMaxRows + i) * (2 + HD + r);
      st_agent(pp + 2 + d, a);
      if (d == 0) {
        st_agent(pp, fin_m[i]);
        st_agent(pp + 1, fin_l[i]);
      }
    }
  }
  // ---- every split counts in; the last merges --------------------------------
  if (frozen) return;
  if (!arrive_last(&ws.att_cnt[sq * D.H + h], S, &last_flag)) return;
  // every partial's max, sum and this thread's accumulator element, loaded together
  const size_t pbase = (((size_t)sq * D.H + h) * (S + 1)) * kMaxRows;
  const int me = min(tid, R * S - 1), mi_ = me / S, ms_ = me % S;
  const float* mp = ws.att + (pbase + (size_t)ms_ * kMaxRows + mi_) * (2 + HD + r);
  const float pm = ld_agent(mp), pl = ld_agent(mp + 1);
  const int ei = min(tid, R * HD - 1) / HD, ed = min(tid, R * HD - 1) % HD;
  float part[16];   // the first 16 partials (more are read in the combine loop)
#pragma unroll
  for (int u = 0; u < 16; ++u)
    part[u] = ld_agent(ws.att + (pbase + (size_t)min(u, S - 1) * kMaxRows + ei) * (2 + HD + r) + 2 + ed);
  if (tid < R * S) {
    mw[mi_][ms_] = pm;
    red[0][mi_][ms_] = pl;   // (red is free here; S <= 64 <= HD)
  }
  __syncthreads();
  if (tid < R) {
    const int i = tid;
    float M = -INFINITY;
    for (int s2 = 0; s2 < S; ++s2)
      if (red[0][i][s2] > 0.f) M = fmaxf(M, mw[i][s2]);
    float Ls = 0.f;
    for (int s2 = 0; s2 < S; ++s2) {
      const float l = red[0][i][s2];
      const float w = l > 0.f ? __expf(mw[i][s2] - M) : 0.f;
      mw[i][s2] = w;
      Ls += w * l;
    }
    linv[i] = Ls > 0.f ? 1.f / Ls : 0.f;
  }
  __syncthreads();
  if (tid < R * HD) {
    float v = 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (u < S) v += mw[ei][u] * part[u];
    for (int u = 16; u < S; ++u)
      v += mw[ei][u] * ld_agent(ws.att + (pbase + (size_t)u * kMaxRows + ei) * (2 + HD + r) + 2 + ed);
    v *= linv[ei];
    q_s[ei][ed] = v;   // o of row ei (q is no longer needed)
    ws.O[(size_t)(first + ei) * qd + h * HD + ed] = v;
  }
  __syncthreads();
  // o-adapter down-projection share of this head: uo[row][h][j] = sum_d A_o[j][h*HD + d] o[d]
  for (int i = 0; i < R; ++i) {
    const bool fast = rml.fast[first + i] && L.A[3];
    if constexpr (WB) {
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int pi = tid + kSkAttnThreads * k;
        if (pi < apieces) {
          const int c = pi % (HD / 8);
          float a = 0.f;
#pragma unroll
          for (int w = 0; w < 4; ++w)
            a += bf16lo(ap[k][w]) * q_s[i][8 * c + 2 * w] + bf16hi(ap[k][w]) * q_s[i][8 * c + 2 * w + 1];
          uop[pi] = a;
        }
      }
      __syncthreads();
      if (tid < r) {
        float a = 0.f;
        for (int c = 0; c < HD / 8; ++c) a += uop[tid * (HD / 8) + c];
        ws.uo[((size_t)(first + i) * D.H + h) * r + tid] = fast ? a : 0.f;
      }
      __syncthreads();
    } else {
      // f32 adapters (small configurations): one row of A_o per thread
      if (tid < r) {
        float a = 0.f;
        if (fast) {
          const float* arow = (const float*)L.A[3] + (size_t)tid * qd + h * HD;
          for (int d = 0; d < HD; ++d) a += arow[d] * q_s[i][d];
        }
        ws.uo[((size_t)(first + i) * D.H + h) * r + tid] = a;
      }
    }
  }
}

}  // namespace m2r2
