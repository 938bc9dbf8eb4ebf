// Matrix-core GEMM for the request-time products (bf16 operands, fp32
// accumulation): C[m, n] = sum_k A[m, k] B[n, k] (+ bias[n]), A [M, K] and
// B [N, K] row-major bf16 (a weight matrix [out, in] is B as stored), with one
// of several epilogues.  It computes the acoustic keys and values of every
// decoder block for a new request (Appendix A.5) and the products of the
// audio encoder.
//
// Tiling: BMT x 128 output tiles (BMT = 128, or 64 when 128-row tiles would
// leave CUs idle), k in steps of 64, 256 threads = 2 x 2 waves of BMT/2 x 64
// (BMT/64 x 2 tiles of v_mfma_f32_32x32x16_bf16).  A and B tiles are copied
// straight from memory into LDS stages (global_load_lds_dwordx4): two stages one
// k-step ahead for 128-row tiles (two blocks share a CU), four stages three
// k-steps ahead for 64-row tiles (16-byte chunks, chunk q of row r stored at
// q ^ (r & 7) so that the eight rows a wave's lane group reads fall in different
// banks).
// The finished tile goes through LDS again so that every epilogue writes 16-byte
// runs of consecutive elements.
#include <algorithm>

#include "wf_common.h"
#include "wf_kernels.h"
#include "wf_operand.h"

namespace wf {

namespace {

typedef __attribute__((address_space(3))) void lds_void;
constexpr int BN = kMmTile, BK = kMmK, NT = 256;
constexpr int kChunksB = BN * BK / 8;  // 16-byte chunks of a B tile (1024)
constexpr int kCt = BN + 1;            // row stride of the staged output tile (floats)


__device__ __forceinline__ uint4 pack8(const float* v) {
  uint4 r;
  r.x = bf16_bits_rne(v[0]) | (bf16_bits_rne(v[1]) << 16);
  r.y = bf16_bits_rne(v[2]) | (bf16_bits_rne(v[3]) << 16);
  r.z = bf16_bits_rne(v[4]) | (bf16_bits_rne(v[5]) << 16);
  r.w = bf16_bits_rne(v[6]) | (bf16_bits_rne(v[7]) << 16);
  return r;
}

}  // namespace

// Four LDS stages, separate objects so that the compiler sees a copy into one
// stage cannot alias reads of another; each holds one k-step's A and B tiles
// (16-byte chunks, chunk c of row r at r * 8 + (c ^ (r & 7))), and after the loop
// two of them hold the output tile's two 64-row halves ([64][kCt] fp32).
constexpr int kStageU4 = (64 * kCt * 4 + 15) / 16;  // >= 2048 chunks of a 128-row A + B stage
static_assert(kStageU4 >= 2 * kChunksB, "stage holds a 128-row k-step");
__shared__ uint4 g_mm0[kStageU4], g_mm1[kStageU4], g_mm2[kStageU4], g_mm3[kStageU4];

template <int EP, int BM, int NS>
__global__ void __launch_bounds__(NT) k_mm(MmArgs a) {
  static_assert(NS == 2 || NS == 4, "two or four stages");
  constexpr int kChunksA = BM * BK / 8, JA = kChunksA / NT, MI = BM / 64;
  // copies per wave and k-step: JA of A, 4 of B; a step waits until at most the
  // NS - 2 later k-steps' copies are outstanding (and its earlier LDS reads are done)
  constexpr int kCopies = JA + 4, kVm = (NS - 2) * kCopies;
  constexpr int kWait = (kVm & 15) | ((kVm >> 4) << 14) | (7 << 4) | (0 << 8);
  const int z = blockIdx.z;
  const bf16* A = a.A + (size_t)z * a.sA;
  const bf16* B = a.B + (size_t)z * a.sB;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int nk = a.K / BK, nbB = a.nb > 0 ? a.nb : a.N;

  // this lane's copy sources: LDS chunk slot s = (w * J + j) * 64 + lane holds row
  // s / 8, chunk (s % 8) ^ (row & 7) of the tile (rows past the matrix re-read its
  // last row; their results are not written)
  const bf16* srcA[JA];
  const bf16* srcB[4];
#pragma unroll
  for (int j = 0; j < JA; ++j) {
    const int slot = (w * JA + j) * 64 + lane, row = slot >> 3, ch = (slot & 7) ^ (row & 7);
    srcA[j] = A + (size_t)min(m0 + row, a.M - 1) * a.lda + 8 * ch;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int slot = (w * 4 + j) * 64 + lane, row = slot >> 3, ch = (slot & 7) ^ (row & 7);
    srcB[j] = B + (size_t)min(n0 + row, nbB - 1) * a.ldb + 8 * ch;
  }
  auto copy = [&](int kt, uint4* stage) {  // k-step kt (past the last: the last one)
    const int k0 = min(kt, nk - 1) * BK;
#pragma unroll
    for (int j = 0; j < JA; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(srcA[j] + k0), (lds_void*)&stage[(w * JA + j) * 64], 16, 0, 0);
#pragma unroll
    for (int j = 0; j < 4; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(srcB[j] + k0), (lds_void*)&stage[kChunksA + (w * 4 + j) * 64],
                                       16, 0, 0);
  };

  floatx16 acc[MI][2];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][jj][v] = 0.f;

  // fragment rows of this lane: row (lane % 32) of each 32-row tile, k chunk
  // 2 s + lane / 32 of k-substep s
  const int lr = lane & 31, lk = lane >> 5;
  auto step = [&](int kt, const uint4* la, uint4* nxt) {
    __builtin_amdgcn_s_waitcnt(kWait);
    __builtin_amdgcn_s_barrier();
    copy(kt + NS - 1, nxt);  // every step issues its copies, so the wait count stays exact
    if (kt < nk) {
      const uint4* lb = la + kChunksA;
#pragma unroll
      for (int s = 0; s < BK / 16; ++s) {
        const int q = 2 * s + lk;
        bf16x8 af[MI], bf[2];
#pragma unroll
        for (int i = 0; i < MI; ++i) {
          const int row = wm * (BM / 2) + i * 32 + lr;
          af[i] = __builtin_bit_cast(bf16x8, la[row * 8 + (q ^ (row & 7))]);
        }
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          const int row = wn * 64 + jj * 32 + lr;
          bf[jj] = __builtin_bit_cast(bf16x8, lb[row * 8 + (q ^ (row & 7))]);
        }
#pragma unroll
        for (int i = 0; i < MI; ++i)
#pragma unroll
          for (int jj = 0; jj < 2; ++jj)
            acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bf[jj], acc[i][jj], 0, 0, 0);
      }
    }
  };
  if constexpr (NS == 4) {
    copy(0, g_mm0);
    copy(1, g_mm1);
    copy(2, g_mm2);
    for (int kt = 0; kt < nk; kt += 4) {
      step(kt, g_mm0, g_mm3);
      step(kt + 1, g_mm1, g_mm0);
      step(kt + 2, g_mm2, g_mm1);
      step(kt + 3, g_mm3, g_mm2);
    }
  } else {  // two stages (66 KB of LDS: two blocks per CU), one k-step ahead
    copy(0, g_mm0);
    for (int kt = 0; kt < nk; kt += 2) {
      step(kt, g_mm0, g_mm1);
      step(kt + 1, g_mm1, g_mm0);
    }
  }
  __builtin_amdgcn_s_waitcnt((0 & 15) | (7 << 4) | (15 << 8));  // every copy has landed
  __syncthreads();

  // stage the tile (+ bias, activation) in LDS: acc element v of a 32 x 32 tile is
  // row 8 (v / 4) + 4 (lane / 32) + v % 4, column lane % 32; rows 0..63 in one
  // stage object, 64..127 in another
  float* ct0 = reinterpret_cast<float*>(g_mm0);
  float* ct1 = reinterpret_cast<float*>(g_mm1);
  auto ct = [&](int r) -> float* { return (r < 64 ? ct0 : ct1) + (r & 63) * kCt; };
  const bf16* bias = a.bias ? a.bias + (size_t)z * a.sBias : nullptr;
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) {
    const int cl = wn * 64 + jj * 32 + lr;
    const float bv = bias ? to_f(bias[min(n0 + cl, a.N - 1)]) : 0.f;
#pragma unroll
    for (int i = 0; i < MI; ++i)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int rl = wm * (BM / 2) + i * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
        float x = acc[i][jj][v] * a.scale + bv;
        if (EP == MM_BF16_GELU) x = gelu_erf(x);
        ct(rl)[cl] = x;
      }
  }
  __syncthreads();

  if (EP == MM_XKV || EP == MM_QKV_ENC) {
    // columns [0, nrow) row-major bf16 (keys, or queries | keys), columns
    // [nrow, N) values transposed per head: MM_XKV in 256-frame pieces
    // [head][frame / 256][dim][256] after the keys [head][frame][64]; MM_QKV_ENC as
    // [head][dim][ldv] in out2.  Frames from M to the padded count are zeros.
    const int nrow = EP == MM_XKV ? a.d : 2 * a.d;
    bf16* out = reinterpret_cast<bf16*>(a.out) + (size_t)z * a.sO;
    // row-major part: items (row, 8 columns)
    for (int it = t; it < BM * (BN / 8); it += NT) {
      const int rl = it / (BN / 8), c8 = (it % (BN / 8)) * 8, f = m0 + rl, n = n0 + c8;
      if (f >= a.M || n >= nrow) continue;
      const uint4 pk = pack8(ct(rl) + c8);
      if (EP == MM_XKV) {
        const int head = n >> 6, dim = n & 63;
        *reinterpret_cast<uint4*>(out + ((size_t)head * a.M + f) * kHeadDim + dim) = pk;
      } else {
        *reinterpret_cast<uint4*>(out + (size_t)f * a.ldo + n) = pk;
      }
    }
    // transposed part: items (column, 8 frames)
    for (int it = t; it < BN * (BM / 8); it += NT) {
      const int cl = it / (BM / 8), r8 = (it % (BM / 8)) * 8, n = n0 + cl, f = m0 + r8;
      if (n < nrow || n >= a.N || f >= a.vt_frames) continue;
      const int col = n - nrow, head = col >> 6, dim = col & 63;
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = f + e < a.M ? ct(r8 + e)[cl] : 0.f;
      const uint4 pk = pack8(v);
      if (EP == MM_XKV) {
        bf16* vt = out + (size_t)a.n_head * a.M * kHeadDim + (size_t)head * kHeadDim * a.vt_frames;
        *reinterpret_cast<uint4*>(vt + vt_index(dim, f)) = pk;
      } else {
        bf16* vt = reinterpret_cast<bf16*>(a.out2) + (size_t)z * a.sO2;
        *reinterpret_cast<uint4*>(vt + ((size_t)head * kHeadDim + dim) * a.vt_frames + f) = pk;
      }
    }
    return;
  }
  // row-major outputs: items (row, 8 columns)
  for (int it = t; it < BM * (BN / 8); it += NT) {
    const int rl = it / (BN / 8), c8 = (it % (BN / 8)) * 8, f = m0 + rl, n = n0 + c8;
    if (f >= a.M || n >= a.N) continue;
    const float* src = ct(rl) + c8;
    if (EP == MM_BF16 || EP == MM_BF16_GELU) {
      bf16* out = reinterpret_cast<bf16*>(a.out) + (size_t)z * a.sO;
      *reinterpret_cast<uint4*>(out + (size_t)f * a.ldo + n) = pack8(src);
    } else {
      float* out = reinterpret_cast<float*>(a.out) + (size_t)z * a.sO + (size_t)f * a.ldo + n;
      float4 lo = make_float4(src[0], src[1], src[2], src[3]), hi = make_float4(src[4], src[5], src[6], src[7]);
      if (EP == MM_GELU_ADD_F32) {
        const float* ad = a.add + (size_t)f * a.ldadd + n;
        lo.x = gelu_erf(lo.x) + ad[0]; lo.y = gelu_erf(lo.y) + ad[1];
        lo.z = gelu_erf(lo.z) + ad[2]; lo.w = gelu_erf(lo.w) + ad[3];
        hi.x = gelu_erf(hi.x) + ad[4]; hi.y = gelu_erf(hi.y) + ad[5];
        hi.z = gelu_erf(hi.z) + ad[6]; hi.w = gelu_erf(hi.w) + ad[7];
      }
      if (EP == MM_RESID) {  // residual rows: each element has exactly one writer
        const float4 o0 = *reinterpret_cast<const float4*>(out), o1 = *reinterpret_cast<const float4*>(out + 4);
        lo.x += o0.x; lo.y += o0.y; lo.z += o0.z; lo.w += o0.w;
        hi.x += o1.x; hi.y += o1.y; hi.z += o1.z; hi.w += o1.w;
      }
      *reinterpret_cast<float4*>(out) = lo;
      *reinterpret_cast<float4*>(out + 4) = hi;
    }
  }
}

// Shapes the kernel assumes: K a multiple of 64, N a multiple of 8, 16-byte
// aligned rows (lda, ldb, ldo multiples of 8), and for the transposed epilogues
// head width 64 with the value columns after the row-major ones.
int mm_check(const MmArgs& a, int ep) {
  if (a.M < 1 || a.N < 1 || a.K < kMmK || a.K % kMmK) return -1;
  if (a.N % 8 || a.lda % 8 || a.ldb % 8 || a.lda < a.K || a.ldb < a.K) return -1;
  if ((ep == MM_BF16 || ep == MM_BF16_GELU || ep == MM_F32 || ep == MM_RESID || ep == MM_GELU_ADD_F32) &&
      (a.ldo % 8 || a.ldo < a.N))
    return -1;
  if (ep == MM_GELU_ADD_F32 && (!a.add || a.ldadd < a.N)) return -1;
  if (ep == MM_XKV && (a.N != 2 * a.d || a.d % kHeadDim || a.vt_frames < a.M || a.vt_frames % kVtPiece)) return -1;
  if (ep == MM_QKV_ENC && (a.N != 3 * a.d || a.d % kHeadDim || a.vt_frames < a.M || a.vt_frames % 8 || a.ldo % 8 ||
                           a.ldo < 2 * a.d))
    return -1;
  return 0;
}

template <int BM, int NS>
static void mm_launch(const MmArgs& a, int ep, int batch, hipStream_t st) {
  const dim3 grid((std::max(a.M, (ep == MM_XKV || ep == MM_QKV_ENC) ? a.vt_frames : a.M) + BM - 1) / BM,
                  (a.N + BN - 1) / BN, batch);
  switch (ep) {
    case MM_F32: k_mm<MM_F32, BM, NS><<<grid, NT, 0, st>>>(a); break;
    case MM_BF16: k_mm<MM_BF16, BM, NS><<<grid, NT, 0, st>>>(a); break;
    case MM_BF16_GELU: k_mm<MM_BF16_GELU, BM, NS><<<grid, NT, 0, st>>>(a); break;
    case MM_RESID: k_mm<MM_RESID, BM, NS><<<grid, NT, 0, st>>>(a); break;
    case MM_XKV: k_mm<MM_XKV, BM, NS><<<grid, NT, 0, st>>>(a); break;
    case MM_QKV_ENC: k_mm<MM_QKV_ENC, BM, NS><<<grid, NT, 0, st>>>(a); break;
    case MM_GELU_ADD_F32: k_mm<MM_GELU_ADD_F32, BM, NS><<<grid, NT, 0, st>>>(a); break;
  }
}

// 128-row tiles in two stages (two blocks fit on a CU), or, when the 128-row grid
// would cover fewer blocks than the chip has CUs (256), 64-row tiles in four
// stages (one block per CU, three k-steps of copies in flight)
void mm(const MmArgs& a, int ep, int batch, hipStream_t st) {
  const int rows = std::max(a.M, (ep == MM_XKV || ep == MM_QKV_ENC) ? a.vt_frames : a.M);
  const long long blocks128 = (long long)((rows + 127) / 128) * ((a.N + BN - 1) / BN) * batch;
  if (blocks128 < 256) mm_launch<64, 4>(a, ep, batch, st);
  else mm_launch<128, 2>(a, ep, batch, st);
}

}  // namespace wf
