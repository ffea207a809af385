// Shared device/host helpers of libwd (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wd {

// ---- bf16 storage -----------------------------------------------------------
// bf16 values are stored as raw uint16 bit patterns (the upper half of fp32).

__device__ __forceinline__ float bf2f(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// fp32 -> bf16, round to nearest even; NaN stays NaN.
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Activation element types: fp32 models keep float, bf16 models store uint16.
template <typename T> struct Elem;
template <> struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
  __device__ __forceinline__ static float to_f(float v) { return v; }
  __device__ __forceinline__ static float from_f(float v) { return v; }
};
template <> struct Elem<uint16_t> {
  __device__ __forceinline__ static float load(const uint16_t* p) { return bf2f(*p); }
  __device__ __forceinline__ static float to_f(uint16_t v) { return bf2f(v); }
  __device__ __forceinline__ static uint16_t from_f(float v) { return f2bf(v); }
};

// ---- MFMA -----------------------------------------------------------------------
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// D[16x16] += A[16x32] * B[32x16] (bf16 in, fp32 accumulate).
// Lane l holds A[l%16][(l/16)*8 + i] and B[(l/16)*8 + i][l%16], i = 0..7;
// D: lane l holds D[(l/16)*4 + j][l%16], j = 0..3.
__device__ __forceinline__ f32x4 mfma16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// ---- wave / block reductions (wave64) ---------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// Sum of p[s * stride] for s = 0..S-1, added in order of s.  Loads go out
// in batches from clamped addresses, so a wave waits for one round trip per
// batch rather than one per partial; the out-of-range lanes of the last batch
// add zero.  Batches of 4 when S <= 4 (the few-row split-K products), else 8:
// no load is issued for a partial that does not exist up to 4.
template <int NB, typename V>
__device__ __forceinline__ V split_sum_nb(const V* __restrict__ p, long stride, int S) {
  V acc{};
  for (int s0 = 0; s0 < S; s0 += NB) {
    V t[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) t[j] = p[(long)min(s0 + j, S - 1) * stride];
#pragma unroll
    for (int j = 0; j < NB; ++j) acc += s0 + j < S ? t[j] : V{};
  }
  return acc;
}
template <typename V>
__device__ __forceinline__ V split_sum(const V* __restrict__ p, long stride, int S) {
  return S <= 4 ? split_sum_nb<4>(p, stride, S) : split_sum_nb<8>(p, stride, S);
}

// Two such sums over the same split index with their loads interleaved.
template <int NB, typename V>
__device__ __forceinline__ void split_sum2_nb(const V* __restrict__ p, const V* __restrict__ q,
                                              long stride, int S, V& a, V& b) {
  a = V{};
  b = V{};
  for (int s0 = 0; s0 < S; s0 += NB) {
    V t[NB], u[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const long o = (long)min(s0 + j, S - 1) * stride;
      t[j] = p[o];
      u[j] = q[o];
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      a += s0 + j < S ? t[j] : V{};
      b += s0 + j < S ? u[j] : V{};
    }
  }
}
template <typename V>
__device__ __forceinline__ void split_sum2(const V* __restrict__ p, const V* __restrict__ q,
                                           long stride, int S, V& a, V& b) {
  if (S <= 4)
    split_sum2_nb<4>(p, q, stride, S, a, b);
  else
    split_sum2_nb<8>(p, q, stride, S, a, b);
}

// Sum over the block (blockDim.x a multiple of 64, <= 1024); every thread gets
// the total.  The summation order is fixed, so results are reproducible.
__device__ __forceinline__ float block_sum(float v, float* red /* >= 16 floats of LDS */) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float t = 0.f;
  for (int i = 0; i < nw; ++i) t += red[i];
  return t;
}

}  // namespace wd

// Geometry of one step, passed to kernels by value (no device copy needed).
#define WD_MAX_BATCH 64
struct WdStepGeom {
  int32_t batch;
  int32_t ctx[WD_MAX_BATCH];    // attended prefix length of each sequence this step
  int32_t row0[WD_MAX_BATCH];   // first row of each sequence in this step's row set
  int32_t nrows[WD_MAX_BATCH];  // rows of each sequence in this step's row set
  int32_t off[WD_MAX_BATCH];    // first token of each sequence in the token / K/V arrays
  int32_t mode[WD_MAX_BATCH];   // rows of the sequence: 0 refresh, 1 normal, 2 full, -1 none
  int32_t nact[WD_MAX_BATCH];   // active positions of the sequence this step
  int32_t end[WD_MAX_BATCH];    // live end: S, or one past the first decoded <eos>
};
