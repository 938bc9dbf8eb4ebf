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
  ST_PG0 = 14,     // cache page of position ST_POS0
  ST_PG1 = 15,     // the page after it (rows of the pass that cross a page boundary)
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
// round to nearest even; NaN stays NaN (branch-free)
__device__ __forceinline__ uint32_t bf16_bits_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  const uint32_t rne = (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
  return (u & 0x7fffffffu) > 0x7f800000u ? ((u >> 16) | 0x40u) : rne;
}
template <>
__device__ __forceinline__ bf16 from_f<bf16>(float f) {
  bf16 r;
  r.u = (uint16_t)bf16_bits_rne(f);
  return r;
}

// Exact three-term bf16 split of an fp32 value: hi keeps the top 8 significand
// bits (truncated), mid the next 8 bits of the exact remainder, lo the rest (at
// most 8 bits, so exact in bf16); hi + mid + lo == f for finite f away from the
// denormal range.  Returned as bf16 bit patterns.
__device__ __forceinline__ void split3_bits(float f, uint32_t& hi, uint32_t& mid, uint32_t& lo) {
  const uint32_t u = __float_as_uint(f);
  const float r1 = f - __uint_as_float(u & 0xffff0000u);
  const uint32_t v = __float_as_uint(r1);
  const float r2 = r1 - __uint_as_float(v & 0xffff0000u);
  hi = u >> 16;
  mid = v >> 16;
  lo = __float_as_uint(r2) >> 16;
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

// Cross-lane moves through the DPP modifier (no LDS round trip).
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xf, 0xf, false));
}
constexpr int kDppXor1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;  // lane i <-> 7 - i within 8 lanes
constexpr int kDppMirror = 0x140;      // lane i <-> 15 - i within 16 lanes
constexpr int kDppRor8 = 0x128;        // lane i <- lane (i + 8) mod 16 within 16 lanes

__device__ __forceinline__ float lane_f(float v, int l) { return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l)); }

// sum / max over the 8 lanes of an aligned group (result in every lane of the group)
__device__ __forceinline__ float sum8(float v) {
  v += dpp<kDppXor1>(v);
  v += dpp<kDppXor2>(v);
  return v + dpp<kDppHalfMirror>(v);
}
// sum / max over the 16 lanes of a row (result in every lane of the row)
__device__ __forceinline__ float sum16(float v) {
  v = sum8(v);
  return v + dpp<kDppMirror>(v);
}
__device__ __forceinline__ float max16(float v) {
  v = fmaxf(v, dpp<kDppXor1>(v));
  v = fmaxf(v, dpp<kDppXor2>(v));
  v = fmaxf(v, dpp<kDppHalfMirror>(v));
  return fmaxf(v, dpp<kDppMirror>(v));
}
// whole-wave sum / max, uniform result (fixed order: rows 0..3)
__device__ __forceinline__ float wave_sum(float v) {
  v = sum16(v);
  return (lane_f(v, 15) + lane_f(v, 31)) + (lane_f(v, 47) + lane_f(v, 63));
}
__device__ __forceinline__ float wave_max(float v) {
  v = max16(v);
  return fmaxf(fmaxf(lane_f(v, 15), lane_f(v, 31)), fmaxf(lane_f(v, 47), lane_f(v, 63)));
}

// (value, index) maximum with ties to the lowest index; NaN compares as larger
// than everything so a non-finite row is visible to the status check.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  bool vn = v != v, bn = bv != bv;
  if (vn != bn) return vn;
  if (v != bv) return v > bv;
  return i < bi;
}

// A stored parameter element as raw bits, converted only where it is used (so no
// instruction right after the load waits for it).
template <typename S>
__device__ __forceinline__ uint32_t ld_bits(const void* p, int i) {
  if constexpr (sizeof(S) == 2) return reinterpret_cast<const uint16_t*>(p)[i];
  else return reinterpret_cast<const uint32_t*>(p)[i];
}
template <typename S>
__device__ __forceinline__ float from_bits(uint32_t b) {
  if constexpr (sizeof(S) == 2) return __uint_as_float(b << 16);
  else return __uint_as_float(b);
}

// Launch timing for profiled calls.  A timing slot holds, per XCD (the chip's
// eight dies) and per block-number residue mod 8, the earliest block start and
// the latest block end (the block's last wave to leave, found with an LDS
// count), read from the chip's constant-rate wall clock.  The launch lasts the
// longest per-XCD span.  Spreading the global atomics over 64 words keeps them
// from queueing on one address (which slowed large launches measurably).  A
// null slot (the normal case) costs one uniform branch.
constexpr int kStampXcds = 8, kStampSub = 8;
constexpr int kStampWords = 2 * kStampXcds * kStampSub;  // per launch: (start, end) pairs
__device__ __forceinline__ int xcc_id() {
  return (int)__builtin_amdgcn_s_getreg((20) | (0 << 6) | (3 << 11)) & (kStampXcds - 1);  // HW_REG_XCC_ID[3:0]
}
__device__ __forceinline__ unsigned long long* stamp_pair(unsigned long long* s) {
  const unsigned blk = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  return s + 2 * (xcc_id() * kStampSub + (int)(blk & (kStampSub - 1)));
}
struct StampScope {
  unsigned long long* s;
  unsigned* left;
  // Must be the kernel's first statement: every thread of the block runs it.
  // nthreads is the block size every launch of the kernel uses (a compile-time
  // constant, so no load of the launch's dimensions delays the start).
  __device__ __forceinline__ StampScope(unsigned long long* p, int nthreads) : s(p) {
    __shared__ unsigned waves_left;
    left = &waves_left;
    if (s) {
      if (threadIdx.x == 0) {
        waves_left = (unsigned)(nthreads + 63) / 64;
        atomicMin(stamp_pair(s), (unsigned long long)wall_clock64());
      }
      __syncthreads();
    }
  }
  __device__ __forceinline__ ~StampScope() {
    if (s && (threadIdx.x & 63) == 0 && atomicSub(left, 1u) == 1u)
      atomicMax(stamp_pair(s) + 1, (unsigned long long)wall_clock64());
  }
};
constexpr int kStampSlots = 4096;  // instrumented launches per profiled call (kStampWords each)

// ---------------------------------------------------------------- counter-based randomness
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds mapping a 256-bit
// counter and a 128-bit key to 256 bits.  A round multiplies words 0 and 2 by two
// fixed 64-bit constants, swaps the halves of the 128-bit products into the
// other words and mixes in the key; the key advances by two Weyl increments
// between rounds.
constexpr uint64_t kPhiloxM0 = 0xD2E7470EE14C6C93ull;
constexpr uint64_t kPhiloxM1 = 0xCA5A826395121157ull;
constexpr uint64_t kPhiloxW0 = 0x9E3779B97F4A7C15ull;
constexpr uint64_t kPhiloxW1 = 0xBB67AE8584CAA73Bull;

struct Philox4 {
  uint64_t w[4];
};

__host__ __device__ __forceinline__ uint64_t mul_hi64(uint64_t a, uint64_t b) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __umul64hi(a, b);
#else
  return (uint64_t)(((unsigned __int128)a * b) >> 64);
#endif
}

__host__ __device__ __forceinline__ Philox4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3,
                                                         uint64_t k0, uint64_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += kPhiloxW0;
      k1 += kPhiloxW1;
    }
    const uint64_t lo0 = kPhiloxM0 * c0, hi0 = mul_hi64(kPhiloxM0, c0);
    const uint64_t lo1 = kPhiloxM1 * c2, hi1 = mul_hi64(kPhiloxM1, c2);
    const uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
  }
  return Philox4{{c0, c1, c2, c3}};
}

// Decoding randomness: key (seed, 0), counter (purpose << 32 | slot, step, pos, v >> 2),
// word v & 3.  purpose: 1 prefill, 2 plain, 3 draft, 4 acceptance, 5 residual, 6 bonus.
enum { RNG_PREFILL = 1, RNG_PLAIN = 2, RNG_DRAFT = 3, RNG_ACC = 4, RNG_RES = 5, RNG_BON = 6 };
__host__ __device__ __forceinline__ uint64_t rng_word(uint64_t seed, int purpose, int slot, int step, int pos, int v) {
  const Philox4 r = philox4x64_10(((uint64_t)purpose << 32) | (uint32_t)slot, (uint64_t)(uint32_t)step,
                                  (uint64_t)(uint32_t)pos, (uint64_t)((uint32_t)v >> 2), seed, 0);
  const int j = v & 3;  // select without indexing, so the words stay in registers
  return j == 0 ? r.w[0] : j == 1 ? r.w[1] : j == 2 ? r.w[2] : r.w[3];
}
// fp32 uniform in (0, 1): the top 23 bits plus one half, scaled by 2^-23
__device__ __forceinline__ float rng_uniform(uint64_t x) { return ((float)(x >> 41) + 0.5f) * 0x1p-23f; }
// Gumbel noise -log(-log(u)) in fp32
__device__ __forceinline__ float rng_gumbel(uint64_t x) { return -logf(-logf(rng_uniform(x))); }

__device__ __forceinline__ float gelu_erf(float x) { return 0.5f * x * (1.0f + erff(x * 0.70710678118654752440f)); }

}  // namespace wf
