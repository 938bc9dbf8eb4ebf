// Device-side helpers shared by the Whisper-Flash kernels (gfx950, wave64).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace wf {

constexpr int kRows = 9;          // rows per slot in a verify / draft pass (anchor + 8)
constexpr int kHeadDim = 64;
constexpr int kPage = 16;         // tokens per self-attention KV page
constexpr int kStateInts = 16;    // per-slot state words
constexpr int kMaxFrames = 2048;  // largest supported number of acoustic frames
constexpr int kMaxCtx = 448;      // largest supported text context

// per-slot state word indices
enum {
  ST_L = 0,        // target cache length == anchor position
  ST_ANCHOR = 1,   // latest emitted token, not yet processed by the target
  ST_EMITTED = 2,  // tokens emitted so far (including the prefill's first token)
  ST_MAX_NEW = 3,  // output budget
  ST_DONE = 4,
  ST_STEP = 5,     // verify calls since prefill
  ST_POS0 = 6,     // first position of the rows of the current pass
  ST_NV = 7,       // valid rows of the current pass (0..9)
  ST_HPOS = 8,     // first position of rows whose drafter history is pending
  ST_HN = 9,       // number of pending history rows
  ST_K = 10,       // candidates verified in the last verify
  ST_A = 11,       // candidates accepted in the last verify
  ST_LEN = 12,     // prompt length
  ST_LIVE = 13,    // slot has been prefilled
};

// Matrix-core fragment orders.  v_mfma_f32_16x16x32_bf16 reads, per lane l, 8
// consecutive k of row (or column) l % 16 starting at k = 8 * (l / 16);
// v_mfma_f32_32x32x16_bf16 reads 8 consecutive k of row l % 32 starting at
// k = 8 * (l / 32).  Weights are stored tile by tile ([tile][k-step][lane][8]) and
// activation operands k-step by k-step ([k-step][tile][lane][8]), so that one
// wave's fragment load is 1 KB of contiguous memory.
__host__ __device__ __forceinline__ size_t wfrag16_index(int n, int k, int ksteps) {
  return ((size_t)((n >> 4) * ksteps + (k >> 5)) * 64 + (n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7);
}
__host__ __device__ __forceinline__ size_t wfrag32_index(int n, int k, int ksteps) {
  return ((size_t)((n >> 5) * ksteps + (k >> 4)) * 64 + (n & 31) + 32 * ((k & 15) >> 3)) * 8 + (k & 7);
}
__host__ __device__ __forceinline__ size_t afrag16_index(int m, int k, int mtiles) {
  return ((size_t)((k >> 5) * mtiles + (m >> 4)) * 64 + (m & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7);
}
__host__ __device__ __forceinline__ size_t afrag32_index(int m, int k, int mtiles) {
  return ((size_t)((k >> 4) * mtiles + (m >> 5)) * 64 + (m & 31) + 32 * ((k & 15) >> 3)) * 8 + (k & 7);
}

// bf16 storage element: the upper 16 bits of an fp32 value.
struct bf16 {
  uint16_t u;
};

__device__ __forceinline__ float to_f(float v) { return v; }
__device__ __forceinline__ float to_f(bf16 v) { return __uint_as_float(((uint32_t)v.u) << 16); }

template <typename S>
__device__ __forceinline__ S from_f(float f);
template <>
__device__ __forceinline__ float from_f<float>(float f) { return f; }
// round to nearest even; NaN stays NaN
template <>
__device__ __forceinline__ bf16 from_f<bf16>(float f) {
  uint32_t u = __float_as_uint(f);
  bf16 r;
  if ((u & 0x7fffffffu) > 0x7f800000u) {
    r.u = (uint16_t)((u >> 16) | 0x40u);
  } else {
    u += 0x7fffu + ((u >> 16) & 1u);
    r.u = (uint16_t)(u >> 16);
  }
  return r;
}

// Load 8 consecutive storage elements as fp32 (p must be 16-byte aligned for bf16,
// 32-byte aligned for fp32).
__device__ __forceinline__ void ld8(const float* p, float* o) {
  float4 a = *reinterpret_cast<const float4*>(p);
  float4 b = *reinterpret_cast<const float4*>(p + 4);
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
  o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
__device__ __forceinline__ void ld8(const bf16* p, float* o) {
  uint4 v = *reinterpret_cast<const uint4*>(p);
  o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
  o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
  o[4] = __uint_as_float(v.z << 16); o[5] = __uint_as_float(v.z & 0xffff0000u);
  o[6] = __uint_as_float(v.w << 16); o[7] = __uint_as_float(v.w & 0xffff0000u);
}

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

// (value, index) maximum with ties to the lowest index; NaN compares as larger
// than everything so a non-finite row is visible to the status check.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  bool vn = v != v, bn = bv != bv;
  if (vn != bn) return vn;
  if (v != bv) return v > bv;
  return i < bi;
}

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752440f)); }

}  // namespace wf
