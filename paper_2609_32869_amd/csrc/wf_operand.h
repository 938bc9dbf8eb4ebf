// Writing activation values into matrix operands (internal).
#pragma once
#include "wf_kernels.h"

namespace wf {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

__device__ __forceinline__ size_t op_index(const Operand& o, int m, int k) {
  if (o.kind == OP_F16) return afrag16_index(m, k, o.mt);
  if (o.kind == OP_F32) return afrag32_index(m, k, o.mt);
  return (size_t)m * o.ld + k;
}

// Write value v of activation row `row` (= slot * 9 + i), column `col`.  bf16
// with nsplit = 3 (batch 1): the exact three-term split hi + mid + lo == v at rows
// row, R9 + row, 2 R9 + row.  nsplit = 2 (several slots, 16-row fragment order):
// hi (v truncated to bf16) in the operand and lo = RNE(v - hi) at the same place
// of a second plane right after it (mt * 16 * ld elements on), so hi + lo
// equals v to 2^-17 relative and the two products share one accumulator.
// Otherwise the value rounded to the storage type.
__device__ __forceinline__ void put_operand(const Operand& o, int, int, int row, int col, float v, float) {
  reinterpret_cast<float*>(o.p)[op_index(o, row, col)] = v;
}
__device__ __forceinline__ void put_operand(const Operand& o, int nsplit, int R9, int row, int col, float v, bf16) {
  uint16_t* A = reinterpret_cast<uint16_t*>(o.p);
  if (nsplit == 3) {
    uint32_t hi, mid, lo;
    split3_bits(v, hi, mid, lo);
    A[op_index(o, row, col)] = (uint16_t)hi;
    A[op_index(o, R9 + row, col)] = (uint16_t)mid;
    A[op_index(o, 2 * R9 + row, col)] = (uint16_t)lo;
  } else if (nsplit == 2) {
    const uint32_t hb = __float_as_uint(v) & 0xffff0000u;
    const size_t i = op_index(o, row, col);
    A[i] = (uint16_t)(hb >> 16);
    A[i + (size_t)o.mt * 16 * o.ld] = (uint16_t)bf16_bits_rne(v - __uint_as_float(hb));
  } else {
    A[op_index(o, row, col)] = (uint16_t)bf16_bits_rne(v);
  }
}
template <typename S>
__device__ __forceinline__ void put_op(const Operand& o, int nsplit, int R9, int row, int col, float v) {
  put_operand(o, nsplit, R9, row, col, v, S{});
}

// The same for the 8 values of row `row`, columns col .. col + 7 (col a multiple of
// 8): they are contiguous in every operand order, so each term is one 16-byte store.
__device__ __forceinline__ uint4 pack8_bits(const uint32_t* h) {
  return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
}
__device__ __forceinline__ void put_operand8(const Operand& o, int, int, int row, int col, const float* v, float) {
  float* p = reinterpret_cast<float*>(o.p) + op_index(o, row, col);
  *reinterpret_cast<float4*>(p) = make_float4(v[0], v[1], v[2], v[3]);
  *reinterpret_cast<float4*>(p + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
__device__ __forceinline__ void put_operand8(const Operand& o, int nsplit, int R9, int row, int col, const float* v, bf16) {
  uint4* A = reinterpret_cast<uint4*>(o.p);
  uint32_t h[8], m[8], l[8];
  if (nsplit == 3) {
#pragma unroll
    for (int e = 0; e < 8; ++e) split3_bits(v[e], h[e], m[e], l[e]);
    A[op_index(o, row, col) / 8] = pack8_bits(h);
    A[op_index(o, R9 + row, col) / 8] = pack8_bits(m);
    A[op_index(o, 2 * R9 + row, col) / 8] = pack8_bits(l);
  } else if (nsplit == 2) {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t hb = __float_as_uint(v[e]) & 0xffff0000u;
      h[e] = hb >> 16;
      l[e] = bf16_bits_rne(v[e] - __uint_as_float(hb));
    }
    const size_t i = op_index(o, row, col);
    A[i / 8] = pack8_bits(h);
    A[(i + (size_t)o.mt * 16 * o.ld) / 8] = pack8_bits(l);
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) h[e] = bf16_bits_rne(v[e]);
    A[op_index(o, row, col) / 8] = pack8_bits(h);
  }
}
template <typename S>
__device__ __forceinline__ void put_op8(const Operand& o, int nsplit, int R9, int row, int col, const float* v) {
  put_operand8(o, nsplit, R9, row, col, v, S{});
}

}  // namespace wf
