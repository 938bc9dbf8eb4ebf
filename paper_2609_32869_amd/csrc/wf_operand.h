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

// Write value v of activation row `row` (= slot * 9 + i), column `col`.  bf16 with
// nsplit = 3: three bf16 terms hi + mid + lo, at rows row, R9 + row, 2 R9 + row,
// whose sum is v to fp32 precision; otherwise the value in the storage type.
__device__ __forceinline__ void put_operand(const Operand& o, int, int, int row, int col, float v, float) {
  reinterpret_cast<float*>(o.p)[op_index(o, row, col)] = v;
}
__device__ __forceinline__ void put_operand(const Operand& o, int nsplit, int R9, int row, int col, float v, bf16) {
  bf16* A = reinterpret_cast<bf16*>(o.p);
  const bf16 hi = from_f<bf16>(v);
  A[op_index(o, row, col)] = hi;
  if (nsplit == 3) {
    const float r1 = v - to_f(hi);
    const bf16 mid = from_f<bf16>(r1);
    const bf16 lo = from_f<bf16>(r1 - to_f(mid));
    A[op_index(o, R9 + row, col)] = mid;
    A[op_index(o, 2 * R9 + row, col)] = lo;
  }
}
template <typename S>
__device__ __forceinline__ void put_op(const Operand& o, int nsplit, int R9, int row, int col, float v) {
  put_operand(o, nsplit, R9, row, col, v, S{});
}

}  // namespace wf
