// Device-side building blocks shared by the decode kernels (gfx950).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

namespace m2r2 {

constexpr int kMaxRows = 16;     // rows of one GEMV (an MFMA tile is 16 rows high)
constexpr int kMaxSeq = 16;
constexpr int kMaxRank = 32;
constexpr int kMaxHeadDim = 128;

// ----------------------------------------------------------------------------
// bfloat16 <-> float32
// ----------------------------------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round to nearest even (inputs are finite).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return u >> 16;
}
__device__ __forceinline__ float round_bf16(float f) { return __uint_as_float(f32_to_bf16_bits(f) << 16); }

// Split 8 floats into bf16 hi + lo parts (x ~= hi + lo with 16 significant bits).
__device__ __forceinline__ void split_hi_lo(const float (&x)[8], bf16x8_t& hi, bf16x8_t& lo) {
  u32x4_t h, l;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t a = f32_to_bf16_bits(x[2 * i]), b = f32_to_bf16_bits(x[2 * i + 1]);
    float ra = x[2 * i] - __uint_as_float(a << 16), rb = x[2 * i + 1] - __uint_as_float(b << 16);
    h[i] = a | (b << 16);
    l[i] = f32_to_bf16_bits(ra) | (f32_to_bf16_bits(rb) << 16);
  }
  hi = __builtin_bit_cast(bf16x8_t, h);
  lo = __builtin_bit_cast(bf16x8_t, l);
}

// ----------------------------------------------------------------------------
// Loads
// ----------------------------------------------------------------------------
__device__ __forceinline__ u32x4_t ld_stream(const void* p) {
  // weights are read exactly once per step: non-temporal hint
  return __builtin_nontemporal_load((const u32x4_t*)p);
}
__device__ __forceinline__ float4 ld4(const float* p) { return *(const float4*)p; }

// ----------------------------------------------------------------------------
// Wave reductions (64 lanes)
// ----------------------------------------------------------------------------
// Lane exchanges inside a row of 16 lanes through DPP (a VALU operand
// modifier; __shfl_xor compiles to ds_bpermute, an LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E, kDppRowHalfMirror = 0x141, kDppRowMirror = 0x140,
              kDppRowRor4 = 0x124, kDppRowRor8 = 0x128;
// sum over the 4 lanes of a quad (every lane of the quad gets it)
__device__ __forceinline__ float quad_sum(float v) {
  v += dpp_f<kDppQuadXor1>(v);
  return v + dpp_f<kDppQuadXor2>(v);
}
// sum over the 16 lanes of a row (every lane of the row gets it)
__device__ __forceinline__ float row_sum16(float v) {
  v = quad_sum(v);
  v += dpp_f<kDppRowHalfMirror>(v);
  return v + dpp_f<kDppRowMirror>(v);
}
// sum over the lanes l, l+4, l+8, l+12 of a row
__device__ __forceinline__ float row_sum_stride4(float v) {
  v += dpp_f<kDppRowRor8>(v);
  return v + dpp_f<kDppRowRor4>(v);
}
// maximum over the 16 lanes of a row (a lane whose source is disabled keeps
// its own value)
template <int CTRL>
__device__ __forceinline__ float dpp_keep(float v) {
  const int b = __builtin_bit_cast(int, v);
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(b, b, CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row_max16(float v) {
  v = fmaxf(v, dpp_keep<kDppQuadXor1>(v));
  v = fmaxf(v, dpp_keep<kDppQuadXor2>(v));
  v = fmaxf(v, dpp_keep<kDppRowHalfMirror>(v));
  return fmaxf(v, dpp_keep<kDppRowMirror>(v));
}
// Sum and maximum over the 64 lanes (every lane gets it): the rows of 16 by
// DPP, then two lane exchanges across rows.
__device__ __forceinline__ float wave_sum(float v) {
  v = row_sum16(v);
  v += __shfl_xor(v, 16);
  return v + __shfl_xor(v, 32);
}
__device__ __forceinline__ float wave_max(float v) {
  v = row_max16(v);
  v = fmaxf(v, __shfl_xor(v, 16));
  return fmaxf(v, __shfl_xor(v, 32));
}

// Block-wide sum of one value per thread; `red` holds blockDim/64 floats.
__device__ __forceinline__ float block_sum(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_sum(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
  for (int i = 0; i < nw; ++i) s += red[i];
  return s;
}
__device__ __forceinline__ float block_max(float v, float* red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  v = wave_max(v);
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = -INFINITY;
  for (int i = 0; i < nw; ++i) s = fmaxf(s, red[i]);
  return s;
}

// Device-coherent (agent scope) stores and loads.  Data that one workgroup
// hands to another workgroup of the same kernel goes through these: they are
// performed at the device coherence point (sc1), so no L2 write-back or
// invalidate is needed; a release/acquire fence at agent scope per workgroup
// would flush the L2 and costs an order of magnitude more than the kernel.
__device__ __forceinline__ void st_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(int* p, int v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int ld_agent(const int* p) {
  return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Arrival counter for "the last workgroup finishes the job": every thread
// waits until its st_agent stores are complete, then one thread counts the
// workgroup in.  The workgroup that observes `total-1` resets the counter (for
// the next launch) and may read the others' st_agent data with ld_agent.
__device__ __forceinline__ bool arrive_last(uint32_t* counter, uint32_t total, int* flag_lds) {
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t old = __hip_atomic_fetch_add(counter, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = (old == total - 1);
    if (last) __hip_atomic_store(counter, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *flag_lds = last;
  }
  __syncthreads();
  return *flag_lds != 0;
}

__device__ __forceinline__ float silu(float x) { return x / (1.f + __expf(-x)); }

}  // namespace m2r2
