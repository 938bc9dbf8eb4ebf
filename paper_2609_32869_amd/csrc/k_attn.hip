// Attention kernels (gfx950): one block per (head, query row).
//
// A block owns one query row of one head and all of that row's keys, so no
// partial results are merged across blocks.  Keys and values are read eight rows
// at a time: lane l takes dims 8*(l%8)..+7 of key l/8, so one wave load is eight
// consecutive 64-wide rows (1 KB of bf16).  Scores of all keys stay in LDS; the
// softmax is exact (max, then sum) in fp32.  The nine row-blocks of a head are
// numbered so they share blockIdx % 8 and therefore one XCD and its L2, which
// serves the key/value rows to the other eight after the first reads them.
#include "../../include/wf.h"
#include "wf_operand.h"

namespace wf {

__device__ __forceinline__ bool head_row(int b, int H, int& head, int& row) {
  const int x = b & 7, i = b >> 3;
  head = x + 8 * (i / kRows);
  row = i % kRows;
  return head < H;
}

template <int NT>
__device__ __forceinline__ float block_max(float v, float* red) {
  v = wave_max(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) m = fmaxf(m, red[i]);
  return m;
}
template <int NT>
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) s += red[i];
  return s;
}

// sum over the 8 lanes of one key (lane bits 0..2)
__device__ __forceinline__ float key_sum(float s) { return sum8(s); }

// Eight consecutive storage elements of a key/value row, kept packed until used.
template <typename S>
struct Raw8;
template <>
struct Raw8<bf16> {
  uint4 v;
  __device__ __forceinline__ void load(const bf16* p) { v = *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ void zero() { v = make_uint4(0u, 0u, 0u, 0u); }
  __device__ __forceinline__ void unpack(float* o) const {
    o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
    o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
    o[4] = __uint_as_float(v.z << 16); o[5] = __uint_as_float(v.z & 0xffff0000u);
    o[6] = __uint_as_float(v.w << 16); o[7] = __uint_as_float(v.w & 0xffff0000u);
  }
};
template <>
struct Raw8<float> {
  float4 a, b;
  __device__ __forceinline__ void load(const float* p) {
    a = *reinterpret_cast<const float4*>(p);
    b = *reinterpret_cast<const float4*>(p + 4);
  }
  __device__ __forceinline__ void zero() { a = b = make_float4(0.f, 0.f, 0.f, 0.f); }
  __device__ __forceinline__ void unpack(float* o) const {
    o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w;
    o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
  }
};

// Scores of keys [0, nk) whose rows are at rowptr(j) (64 storage elements each,
// eight consecutive keys contiguous) into sc[]; q8 = this lane's 8 query dims.
// A wave issues the loads of B key octets before the first use.
template <typename S, int NT, int B, typename RowPtr>
__device__ __forceinline__ void score_pass(const float* q8, int nk, RowPtr rowptr, float* sc) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane & 7, kl = lane >> 3;
  constexpr int NW = NT / 64;
  const int noct = (nk + 7) >> 3;
  for (int o0 = w; o0 < noct; o0 += NW * B) {
    Raw8<S> kv[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int key = (o0 + NW * b) * 8 + kl;
      if (key < nk) kv[b].load(rowptr(key) + 8 * g);
      else kv[b].zero();
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float k8[8];
      kv[b].unpack(k8);
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) s = fmaf(q8[e], k8[e], s);
      s = key_sum(s);
      const int key = (o0 + NW * b) * 8 + kl;
      if (g == 0 && key < nk) sc[key] = s;
    }
  }
}

// acc[8] += p[key] * V[key][8g..8g+7] over keys [0, nk) (per-lane partials)
template <typename S, int NT, int B, typename RowPtr>
__device__ __forceinline__ void value_pass(float* acc, int nk, RowPtr rowptr, const float* p) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane & 7, kl = lane >> 3;
  constexpr int NW = NT / 64;
  const int noct = (nk + 7) >> 3;
  for (int o0 = w; o0 < noct; o0 += NW * B) {
    Raw8<S> vv[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int key = (o0 + NW * b) * 8 + kl;
      if (key < nk) vv[b].load(rowptr(key) + 8 * g);
      else vv[b].zero();
    }
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int key = (o0 + NW * b) * 8 + kl;
      const float pk = key < nk ? p[key] : 0.f;
      float v8[8];
      vv[b].unpack(v8);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(pk, v8[e], acc[e]);
    }
  }
}

// reduce acc over the 8 key lanes (bits 3..5) and the waves; returns the 64-wide
// unnormalised output in part[0][*]
template <int NT>
__device__ __forceinline__ void reduce_out(float* acc, float (*part)[64]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane & 7;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    acc[e] += __shfl_xor(acc[e], 8, 64);
    acc[e] += __shfl_xor(acc[e], 16, 64);
    acc[e] += __shfl_xor(acc[e], 32, 64);
  }
  if (lane < 8) {
#pragma unroll
    for (int e = 0; e < 8; ++e) part[w][8 * g + e] = acc[e];
  }
  __syncthreads();
}

// softmax in place over sc[0, nk): exp(s - max); returns the sum
template <int NT>
__device__ __forceinline__ float softmax_pass(float* sc, int nk, float* red) {
  float m = -INFINITY;
  for (int j = threadIdx.x; j < nk; j += NT) m = fmaxf(m, sc[j]);
  m = block_max<NT>(m, red);
  float l = 0.f;
  for (int j = threadIdx.x; j < nk; j += NT) {
    const float e = __expf(sc[j] - m);
    sc[j] = e;
    l += e;
  }
  return block_sum<NT>(l, red);
}

// ---------------------------------------------------------------- one query row, all keys
// Attention of one query row over keys [0, nk) whose rows start roff(j) elements
// into Kb and Vb (eight consecutive keys contiguous).  Wave w takes key octets w, w + NW, ... in
// batches of B, with the key and value loads of a batch issued together.  The
// wave keeps a running maximum m, a running sum l of exp(s - m) and the weighted
// value sums acc (lane dims 8g..8g+7, partial over the lane's keys); the waves'
// states are merged once at the end (softmax is exact: every key is seen).
template <typename S, int NW, int B, typename RowOff>
__device__ __forceinline__ void attend_wave(const float* q8, int nk, const S* __restrict__ Kb, const S* __restrict__ Vb,
                                            RowOff roff, float& m, float& l, float* acc) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane & 7, kl = lane >> 3;
  const int noct = (nk + 7) >> 3;
  m = -INFINITY;
  l = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int o0 = w; o0 < noct; o0 += NW * B) {
    Raw8<S> kr[B], vr[B];
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const int key = (o0 + NW * b) * 8 + kl;
      if (key < nk) {
        const uint32_t o = roff(key) + 8 * g;
        kr[b].load(Kb + o);
        vr[b].load(Vb + o);
      } else {
        kr[b].zero();
        vr[b].zero();
      }
    }
    float sc[B];
    float bm = -INFINITY;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      float k8[8];
      kr[b].unpack(k8);
      float t = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) t = fmaf(q8[e], k8[e], t);
      t = key_sum(t);
      sc[b] = (o0 + NW * b) * 8 + kl < nk ? t : -INFINITY;
      bm = fmaxf(bm, sc[b]);
    }
    // key o0 * 8 < nk is in this batch, so mn is finite
    const float mn = fmaxf(m, wave_max(bm));
    const float f = __expf(m - mn);
    l *= f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= f;
#pragma unroll
    for (int b = 0; b < B; ++b) {
      const float p = __expf(sc[b] - mn);  // 0 for keys past nk
      l += g == 0 ? p : 0.f;
      float v8[8];
      vr[b].unpack(v8);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(p, v8[e], acc[e]);
    }
    m = mn;
  }
}

// Merge the NW wave states; threads 0..63 return output dim threadIdx.x.
// part holds, per wave and 16-lane row, the row's value sums (after folding key
// lanes 8..15 of the row onto 0..7).
template <int NW>
__device__ __forceinline__ float merge_waves(float m, float l, float* acc, float (*part)[4][64], float* pm, float* pl) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane & 7;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] += dpp<kDppRor8>(acc[e]);
  l = wave_sum(l);
  if ((lane & 8) == 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) part[w][lane >> 4][8 * g + e] = acc[e];
  }
  if (lane == 0) {
    pm[w] = m;
    pl[w] = l;
  }
  __syncthreads();
  float o = 0.f;
  if (threadIdx.x < kHeadDim) {
    float M = pm[0];
#pragma unroll
    for (int i = 1; i < NW; ++i) M = fmaxf(M, pm[i]);
    float L = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const float f = __expf(pm[i] - M);  // 0 for a wave without keys
      L += pl[i] * f;
      o += ((part[i][0][threadIdx.x] + part[i][1][threadIdx.x]) + (part[i][2][threadIdx.x] + part[i][3][threadIdx.x])) * f;
    }
    o /= L;
  }
  return o;
}

// ---------------------------------------------------------------- cross-attention
// Query row i of slot s against all acoustic frames of one head (no mask).
constexpr int kCrossThreads = 512;
template <typename S>
constexpr int kCrossB = sizeof(S) == 2 ? 24 : 12;  // key octets in flight per wave
template <typename S>
__global__ void __launch_bounds__(kCrossThreads) k_attn_cross(CrossArgs a) {
  StampScope stamp_scope(a.stamp, kCrossThreads);
  constexpr int NW = kCrossThreads / 64;
  __shared__ float part[NW][4][64];
  __shared__ float pm[NW], pl[NW];
  int head, row;
  if (!head_row(blockIdx.x, a.n_head, head, row)) return;
  const int slot = a.slot0 + blockIdx.y;
  const int lane = threadIdx.x & 63, g = lane & 7;
  const float* qr = a.q + (size_t)(slot * kRows + row) * a.ldq + head * kHeadDim + 8 * g;
  float q8[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) q8[e] = qr[e] * 0.125f;
  const S* Kx = reinterpret_cast<const S*>(a.kv) + ((size_t)slot * 2 * a.n_head + head) * a.n_frames * kHeadDim;
  const S* Vx = Kx + (size_t)a.n_head * a.n_frames * kHeadDim;
  float m, l, acc[8];
  attend_wave<S, NW, kCrossB<S>>(q8, a.n_frames, Kx, Vx, [](int j) { return (uint32_t)j * kHeadDim; }, m, l, acc);
  const float o = merge_waves<NW>(m, l, acc, part, pm, pl);
  if (threadIdx.x < kHeadDim)
    put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + row, head * kHeadDim + threadIdx.x, o);
}

// ---------------------------------------------------------------- cross-attention, all rows per block
// Block (head, slot, chunk) computes all nine query rows of one slot over one
// chunk of the frames, so each key / value byte is read once.  The chunk's scores
// live in LDS ([frame][12] fp32):
//   pass 1  scores (bf16 keys: matrix-core tiles of 16 frames against the query
//           rows as hi + lo bf16 planes; fp32 keys: a key's 64-dim product
//           summed over its 8 lanes);
//   sweeps  one thread per (frame, row): the row maxima m, then p = exp(s - m)
//           in place and the row sums l, each reduced in a fixed order (one wave
//           per row);
//   pass 2  acc += p * v over the values (no rescaling; the first value loads
//           are issued before the sweeps), then the 8 key lanes and the waves
//           merge.
// With one chunk the block divides by l and stores.  With several, each block
// stores (max, l, acc) and a second kernel merges the chunks in chunk order:
// out = sum_c e^(m_c - m) acc_c / sum_c e^(m_c - m) l_c.
// The per-wave sums reuse the score buffer once every wave is done with it.
constexpr int kXrThreads = 512;
constexpr int kXrWaves = kXrThreads / 64;
constexpr int kXrStride = 12;                     // floats per frame in the score buffer (9 rows, padded)
constexpr int kXrSweepKeys = kXrThreads / kRows;  // frames per sweep step (56)
inline size_t xr_lds_bytes(int chunk) {
  const size_t sc = (size_t)chunk * kXrStride, wacc = (size_t)kXrWaves * kRows * 64;
  return 4 * (sc > wacc ? sc : wacc);
}
// Sum of acc[r][e] over the eight key lanes of each dim group (lane bits 3..5),
// scattered so that lane l ends with out[r] = the sums of dim 8 (l % 8) + l / 8
// for the nine rows.  Each level halves the values a lane holds: the half-wave
// swap pairs dims e and e + 4 (lanes < 32 keep e), the row-pair swap pairs e and
// e + 2 (even 16-lane rows keep e), a DPP rotation by 8 within 16 lanes pairs e and
// e + 1 (lanes with bit 3 clear keep e).  63 exchanges instead of 72 full folds.
__device__ __forceinline__ void scatter_key_lanes(float (*acc)[8], float* out) {
  const bool hi8 = (threadIdx.x & 8) != 0;
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    float u[4], v[2];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[r][e]), __float_as_uint(acc[r][e + 4]), false, false);
      u[e] = __uint_as_float(x[0]) + __uint_as_float(x[1]);
    }
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const auto x = __builtin_amdgcn_permlane16_swap(__float_as_uint(u[e]), __float_as_uint(u[e + 2]), false, false);
      v[e] = __uint_as_float(x[0]) + __uint_as_float(x[1]);
    }
    out[r] = (hi8 ? v[1] : v[0]) + dpp<kDppRor8>(hi8 ? v[0] : v[1]);
  }
}

// Pass 1 on the matrix cores (bf16 keys): S^T[frame][row] = K[frame] . q[row] over
// 16-frame tiles with v_mfma_f32_16x16x32_bf16.  The key tile is the A operand read
// straight from the row-major key rows (lane l: frame l % 16, dims 8 (l / 16)..+7
// and the same 32 further on); the scaled query rows are the B operand as two bf16
// planes, hi (truncated) and lo = RNE(q - hi), both multiplied into the same
// accumulator so the scores keep fp32 accuracy.  Lane l receives rows l % 16
// (>= 9: zero padding, not stored) of frames 4 (l / 16)..+3 of the tile.  Each
// wave keeps the next stage of kXrTiles tiles (8 KB) in flight while it multiplies.
constexpr int kXrTiles = 4;
__device__ __forceinline__ void xr_scores_mfma(const CrossArgs& a, int slot, int head, const bf16* Kx, int nk,
                                               float* sc) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, n = lane & 15, kg = lane >> 4;
  bf16x8 qh[2], ql[2];
  {
    const float* qr = a.q + (size_t)(slot * kRows + min(n, kRows - 1)) * a.ldq + head * kHeadDim + 8 * kg;
    const float scale = n < kRows ? 0.125f : 0.f;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float4 x0 = *reinterpret_cast<const float4*>(qr + 32 * h);
      const float4 x1 = *reinterpret_cast<const float4*>(qr + 32 * h + 4);
      const float f[8] = {x0.x, x0.y, x0.z, x0.w, x1.x, x1.y, x1.z, x1.w};
      uint32_t hb[8], lb[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float v = f[j] * scale;
        hb[j] = __float_as_uint(v) >> 16;
        lb[j] = bf16_bits_rne(v - __uint_as_float(hb[j] << 16));
      }
      qh[h] = __builtin_bit_cast(bf16x8, make_uint4(hb[0] | hb[1] << 16, hb[2] | hb[3] << 16, hb[4] | hb[5] << 16,
                                                    hb[6] | hb[7] << 16));
      ql[h] = __builtin_bit_cast(bf16x8, make_uint4(lb[0] | lb[1] << 16, lb[2] | lb[3] << 16, lb[4] | lb[5] << 16,
                                                    lb[6] | lb[7] << 16));
    }
  }
  const int ntile = (nk + 15) >> 4;
  const int nst = ((ntile - w + kXrWaves - 1) / kXrWaves + kXrTiles - 1) / kXrTiles;  // load stages of this wave
  auto tile_of = [&](int st, int t) { return w + kXrWaves * (st * kXrTiles + t); };
  bf16x8 kt[2][kXrTiles][2];
  auto load = [&](int buf, int st) {  // frames past the end re-read the last one (not stored)
#pragma unroll
    for (int t = 0; t < kXrTiles; ++t) {
      const int f = min(tile_of(st, t) * 16 + n, nk - 1);
      const bf16x8* kp = reinterpret_cast<const bf16x8*>(Kx + (size_t)f * kHeadDim) + kg;
      kt[buf][t][0] = kp[0];
      kt[buf][t][1] = kp[4];
    }
  };
  auto scores = [&](int buf, int st) {
#pragma unroll
    for (int t = 0; t < kXrTiles; ++t) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[buf][t][0], qh[0], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[buf][t][0], ql[0], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[buf][t][1], qh[1], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[buf][t][1], ql[1], acc, 0, 0, 0);
      const int f0 = tile_of(st, t) * 16 + 4 * kg;
      if (n < kRows) {
#pragma unroll
        for (int v = 0; v < 4; ++v)
          if (f0 + v < nk) sc[(f0 + v) * kXrStride + n] = acc[v];
      }
    }
  };
  load(0, 0);
  for (int st = 0; st < nst; st += 2) {
    load(1, st + 1);
    scores(0, st);
    load(0, st + 2);
    scores(1, st + 1);
  }
}

template <typename S>
__global__ void __launch_bounds__(kXrThreads, 4) k_attn_cross_rows(CrossArgs a) {
  StampScope stamp_scope(a.stamp, kXrThreads);
  // key octets per vector load stage (the fp32 score pass and the value pass)
  constexpr int NW = kXrWaves, B = sizeof(S) == 2 ? 2 : 1;
  extern __shared__ float sc[];
  float(*wacc)[kRows][64] = reinterpret_cast<float(*)[kRows][64]>(sc);
  __shared__ float rmax[kRows], lsum[kRows];
  __shared__ float lpart[kXrSweepKeys * kRows];
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y, c = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, g = lane & 7, kl = lane >> 3;
  const int k0 = c * a.chunk, nk = min(a.n_frames - k0, a.chunk), noct = (nk + 7) >> 3;
  const int nst = ((noct - w + NW - 1) / NW + B - 1) / B;  // load stages of this wave
  const S* Kx = reinterpret_cast<const S*>(a.kv) +
                (((size_t)slot * 2 * a.n_head + head) * a.n_frames + k0) * kHeadDim;
  const S* Vx = Kx + (size_t)a.n_head * a.n_frames * kHeadDim;
  // key of lane group kl in octet b of stage st of this wave (may lie past the end)
  auto key_of = [&](int st, int b) { return (w + NW * (st * B + b)) * 8 + kl; };
  if constexpr (sizeof(S) == 2) {
    xr_scores_mfma(a, slot, head, reinterpret_cast<const bf16*>(Kx), nk, sc);
  } else {  // pass 1: scores
    float q8[kRows][8];
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const float* qr = a.q + (size_t)(slot * kRows + r) * a.ldq + head * kHeadDim + 8 * g;
#pragma unroll
      for (int e = 0; e < 8; ++e) q8[r][e] = qr[e] * 0.125f;
    }
    Raw8<S> kr[2][B];
    auto load = [&](int buf, int st) {  // keys past the end re-read the last one (not stored)
#pragma unroll
      for (int b = 0; b < B; ++b) kr[buf][b].load(Kx + (uint32_t)min(key_of(st, b), nk - 1) * kHeadDim + 8 * g);
    };
    auto scores = [&](int buf, int st) {
#pragma unroll
      for (int b = 0; b < B; ++b) {
        const int key = key_of(st, b);
        float k8[8];
        kr[buf][b].unpack(k8);
        float t[kRows];
#pragma unroll
        for (int r = 0; r < kRows; ++r) {
          float u = 0.f;
#pragma unroll
          for (int e = 0; e < 8; ++e) u = fmaf(q8[r][e], k8[e], u);
          t[r] = sum8(u);
        }
        if (g == 0 && key < nk) {
          float4* d = reinterpret_cast<float4*>(sc + key * kXrStride);
          d[0] = make_float4(t[0], t[1], t[2], t[3]);
          d[1] = make_float4(t[4], t[5], t[6], t[7]);
          d[2] = make_float4(t[8], 0.f, 0.f, 0.f);
        }
      }
    };
    load(0, 0);
    for (int st = 0; st < nst; st += 2) {
      load(1, st + 1);
      scores(0, st);
      load(0, st + 2);
      scores(1, st + 1);
    }
  }
  // pass 2's first value stages go out now, so their latency overlaps the sweeps
  constexpr int NB2 = sizeof(S) == 2 ? 3 : 2;  // value load stages in flight
  Raw8<S> vr[NB2][B];
  auto loadv = [&](int buf, int st) {  // keys past the end re-read the last one (weight 0)
#pragma unroll
    for (int b = 0; b < B; ++b) vr[buf][b].load(Vx + (uint32_t)min(key_of(st, b), nk - 1) * kHeadDim + 8 * g);
  };
#pragma unroll
  for (int i = 0; i < NB2 - 1; ++i) loadv(i, i);
  __syncthreads();
  // sweeps over the scores, one thread per (frame, row): row maxima, then
  // probabilities in place and the row sums; each row's 56 partials are then
  // reduced by one wave (rows 0..7 by waves 0..7, row 8 by wave 0)
  const bool sweeper = threadIdx.x < kXrSweepKeys * kRows;
  const int sr = threadIdx.x % kRows;
  constexpr int U = 4;  // sweep steps whose LDS reads are issued together
  if (sweeper) {
    float m = -INFINITY;
    for (int key0 = threadIdx.x / kRows; key0 < nk; key0 += U * kXrSweepKeys) {
      float x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = sc[min(key0 + u * kXrSweepKeys, nk - 1) * kXrStride + sr];
#pragma unroll
      for (int u = 0; u < U; ++u) m = fmaxf(m, x[u]);  // a clamped re-read repeats a present score
    }
    lpart[threadIdx.x] = m;
  }
  __syncthreads();
  {
    const float m = wave_max(lane < kXrSweepKeys ? lpart[lane * kRows + w] : -INFINITY);
    const float m8 = wave_max(lane < kXrSweepKeys && w == 0 ? lpart[lane * kRows + 8] : -INFINITY);
    if (lane == 0) {
      rmax[w] = m;
      if (w == 0) rmax[8] = m8;
    }
  }
  __syncthreads();
  if (sweeper) {
    const float M = rmax[sr];
    float lp = 0.f;
    for (int key0 = threadIdx.x / kRows; key0 < nk; key0 += U * kXrSweepKeys) {
      float x[U];
#pragma unroll
      for (int u = 0; u < U; ++u) x[u] = sc[min(key0 + u * kXrSweepKeys, nk - 1) * kXrStride + sr];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int key = key0 + u * kXrSweepKeys;
        const float p = __expf(x[u] - M);
        if (key < nk) {
          sc[key * kXrStride + sr] = p;
          lp += p;
        }
      }
    }
    lpart[threadIdx.x] = lp;
  }
  __syncthreads();
  {
    const float l = wave_sum(lane < kXrSweepKeys ? lpart[lane * kRows + w] : 0.f);
    const float l8 = wave_sum(lane < kXrSweepKeys && w == 0 ? lpart[lane * kRows + 8] : 0.f);
    if (lane == 0) {
      lsum[w] = l;
      if (w == 0) lsum[8] = l8;
    }
  }
  // pass 2: values
  float acc[kRows][8];
#pragma unroll
  for (int r = 0; r < kRows; ++r)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[r][e] = 0.f;
  {
    auto accumulate = [&](int buf, int st) {
#pragma unroll
      for (int b = 0; b < B; ++b) {
        const int key = key_of(st, b);
        const bool in = key < nk;
        const float4* d = reinterpret_cast<const float4*>(sc + min(key, nk - 1) * kXrStride);
        const float4 s0 = d[0], s1 = d[1], s2 = d[2];
        const float p[kRows] = {in ? s0.x : 0.f, in ? s0.y : 0.f, in ? s0.z : 0.f, in ? s0.w : 0.f, in ? s1.x : 0.f,
                                in ? s1.y : 0.f, in ? s1.z : 0.f, in ? s1.w : 0.f, in ? s2.x : 0.f};
        float v8[8];
        vr[buf][b].unpack(v8);
#pragma unroll
        for (int r = 0; r < kRows; ++r)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[r][e] = fmaf(p[r], v8[e], acc[r][e]);
      }
    };
    for (int st0 = 0; st0 < nst; st0 += NB2) {
#pragma unroll
      for (int i = 0; i < NB2; ++i) {
        loadv((i + NB2 - 1) % NB2, st0 + i + NB2 - 1);
        accumulate(i, st0 + i);
      }
    }
  }
  // sum the key lanes of each dim group and publish per wave: lane l holds the
  // nine rows of dim 8 (l % 8) + l / 8
  __syncthreads();  // every wave is done with the probabilities
  {
    float o9[kRows];
    scatter_key_lanes(acc, o9);
    const int dim = 8 * g + kl;
#pragma unroll
    for (int r = 0; r < kRows; ++r) wacc[w][r][dim] = o9[r];
  }
  __syncthreads();
  const int pair = blockIdx.y * a.n_head + head;
  float* part = a.part + (size_t)pair * a.nchunk * kXrPart;
  for (int t = threadIdx.x; t < kRows * 64; t += kXrThreads) {
    const int r = t >> 6, dim = t & 63;
    float o = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) o += wacc[i][r][dim];
    if (a.nchunk == 1) put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + r, head * kHeadDim + dim, o / lsum[r]);
    else part[c * kXrPart + 32 + t] = o;
  }
  if (a.nchunk > 1 && threadIdx.x < kRows) {
    part[c * kXrPart + threadIdx.x] = rmax[threadIdx.x];
    part[c * kXrPart + 16 + threadIdx.x] = lsum[threadIdx.x];
  }
}


// ---------------------------------------------------------------- fused attention output product (one slot)
// Group g of C = N / kOpGroups columns, C / 16 tiles of 16 on the matrix cores:
// wave w < C / 16 takes tile T = g C / 16 + w over the head's two 32-dim k-steps.
// op_load fetches the wave's two weight fragments (lane l: column 16 T + l % 16,
// k-group l / 16, in the weights' fragment order) and each lane's column bias at
// block start.  op_apply splits the head's output rows (fp32, in LDS) into three
// bf16 terms as a 27-row operand (two 16-row tiles, rows 9 e + r holding term e of
// row r, so the products are exact in fp32), multiplies, adds each row's three
// terms and adds the nine rows to h with one atomic per (row, column) (the bias
// once, by head 0).
struct OpPre {
  bf16x8 w[2];
  uint32_t b;
};
constexpr int kOpTerms = 3 * kRows;            // operand rows that hold terms
constexpr int kOpTiles = kOpMaxCols / 16;      // column tiles of a group at most
// OWNED: waves past the group's tiles load nothing (their registers get defined
// values from an empty asm, so no copy at the join waits for the other waves'
// loads); only for a kernel whose next waits also cover younger loads, since the
// compiler counts outstanding loads on the path without these.  Otherwise every
// wave loads (tile clamped), which keeps the count of younger loads exact.
template <bool OWNED>
__device__ __forceinline__ void op_load(const OprojArgs& op, int head, int g, int t, OpPre& pre) {
  const int nt = op.N / kOpGroups / 16, KS = op.K / 32, lane = t & 63;
  int w = t >> 6;
  if (!OWNED) w = min(w, nt - 1);
  if (!OWNED || w < nt) {
    const int T = g * nt + w;
    const bf16x8* wp = reinterpret_cast<const bf16x8*>(op.w) + ((size_t)T * KS + 2 * head) * 64 + lane;
    pre.w[0] = wp[0];
    pre.w[1] = wp[64];
    pre.b = reinterpret_cast<const uint16_t*>(op.bias)[16 * T + (lane & 15)];
  } else {
#pragma unroll
    for (int s = 0; s < 2; ++s) __asm__ volatile("" : "=v"(pre.w[s]));
    __asm__ volatile("" : "=v"(pre.b));
  }
}
// Every thread of the block (nt threads of 64 at least) calls it; it holds barriers.
// aop: the operand's 2 x 2 fragments; part: each wave's 27 x 16 products.
__device__ __forceinline__ void op_apply(const OprojArgs& op, int head, int g, int t, const OpPre& pre,
                                         const float (*Ob)[64], int row0, uint4 (*aop)[64],
                                         float (*part)[kOpTerms][16]) {
  const int nt = op.N / kOpGroups / 16, lane = t & 63, w = t >> 6;
  // fragment (tile mt, k-step s), lane l: operand row 16 mt + l % 16, dims 32 s + 8 (l / 16) .. + 7
  for (int i = t; i < 4 * 64; i += blockDim.x) {
    const int mt = i >> 7, st = (i >> 6) & 1, l = i & 63, R = 16 * mt + (l & 15), k0 = 32 * st + 8 * (l >> 4);
    uint32_t bits[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    if (R < kOpTerms) {
      const int e = R / kRows, r = R - e * kRows;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint32_t hi, mid, lo;
        split3_bits(Ob[r][k0 + j], hi, mid, lo);
        bits[j] = e == 0 ? hi : e == 1 ? mid : lo;
      }
    }
    aop[2 * mt + st][l] = pack8_bits(bits);
  }
  __syncthreads();
  if (w < nt) {
    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, aop[st][lane]), pre.w[st], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, aop[2 + st][lane]), pre.w[st], acc1, 0, 0,
                                                     0);
    }
    // lane l holds column l % 16 of operand rows 4 (l / 16) + v (and 16 + ...)
    const int col = lane & 15, kg = lane >> 4;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      part[w][4 * kg + v][col] = acc0[v];
      if (16 + 4 * kg + v < kOpTerms) part[w][16 + 4 * kg + v][col] = acc1[v];
    }
  }
  __syncthreads();
  if (w < nt) {
    // item i = lane + 64 j: row i / 16, column i % 16 (= lane % 16, whose bias the lane holds)
    const int T = g * nt + w;
    const float b = head == 0 ? __uint_as_float(pre.b << 16) : 0.f;
    for (int i = lane; i < kRows * 16; i += 64) {
      const int r = i >> 4, cc = i & 15;
      const float v = (part[w][r][cc] + part[w][kRows + r][cc]) + part[w][2 * kRows + r][cc];
      atomicAdd(op.h + (size_t)(row0 + r) * op.ldh + 16 * T + cc, v + b);
    }
  }
}

// ---------------------------------------------------------------- cross-attention, bf16, matrix cores
// Block (head, slot, chunk of 32 KS NW frames), NW waves of 32 KS frames each, all
// nine query rows, both products on the matrix cores.  Keys are row-major
// [frame][64]; values are stored transposed in 256-frame pieces [frame / 256]
// [dim][256] (zeros past the last frame), so both operands are 16-byte reads of
// consecutive elements.  Every load
// of the block is issued at its start (query rows, key tiles, value fragments),
// so the block waits for memory once.
//   scores       S^T = K q^T per 16-frame tile (v_mfma_f32_16x16x32_bf16, the query
//                rows as hi + lo bf16 planes): lane l gets row l % 16 of frames
//                4 (l / 16)..+3 of the tile.
//   softmax      the chunk's row maxima (lane swaps, then across waves in LDS);
//                p = exp(s - max) in place, row sums.
//   values       O^T = V^T P^T per 32-frame step: two lane swaps (half-wave, then
//                row pair) turn the two score tiles of the step into the B operand
//                (lane l: row l % 16, frames 8 (l / 16)..+7); P as hi + lo planes.
//   output       waves summed in LDS; one chunk: O / l, else the chunk's
//                (max, l, O) record for the merge kernel.

__device__ __forceinline__ bf16x8 pack_bf16x8(const uint32_t* b) {
  return __builtin_bit_cast(bf16x8, make_uint4(b[0] | b[1] << 16, b[2] | b[3] << 16, b[4] | b[5] << 16, b[6] | b[7] << 16));
}
// v = hi + lo: hi truncated to bf16, lo = RNE(v - hi) (2^-17 relative)
__device__ __forceinline__ void split_planes(const float* v, bf16x8& hi, bf16x8& lo) {
  uint32_t hb[8], lb[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    hb[j] = __float_as_uint(v[j]) >> 16;
    lb[j] = bf16_bits_rne(v[j] - __uint_as_float(hb[j] << 16));
  }
  hi = pack_bf16x8(hb);
  lo = pack_bf16x8(lb);
}

// The loads of one (head, slot, chunk) item: query row n (rows >= 9 re-read row 8,
// zeroed below), key tiles (frames past the end re-read the last one, masked
// below), value fragments (inside the padded rows).
template <int KS>
struct XKv {
  bf16x8 kt[2 * KS][2];
  bf16x8 vt[KS][4];
};
template <int KS>
struct XItem {
  float4 qx[2][2];
  XKv<KS> kv;
};

__device__ __forceinline__ void xq_load(const CrossArgs& a, int head, int slot, float4 (&qx)[2][2]) {
  const int lane = threadIdx.x & 63, n = lane & 15, kg = lane >> 4;
  const float* qr = a.q + (size_t)(slot * kRows + min(n, kRows - 1)) * a.ldq + head * kHeadDim + 8 * kg;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    qx[h][0] = *reinterpret_cast<const float4*>(qr + 32 * h);
    qx[h][1] = *reinterpret_cast<const float4*>(qr + 32 * h + 4);
  }
}

template <int KS, int NW>
__device__ __forceinline__ void xkv_load(const CrossArgs& a, int head, int slot, int c, XKv<KS>& it) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, n = lane & 15, kg = lane >> 4;
  const int F = a.n_frames, Fp = a.vt_frames;
  const int f0w = c * a.chunk + w * 32 * KS;  // first frame of this wave
  const bf16* base = reinterpret_cast<const bf16*>(a.kv) + (size_t)slot * a.d * (F + Fp);
  const bf16* Kh = base + (size_t)head * F * kHeadDim;
  const bf16* Vt = base + (size_t)a.n_head * F * kHeadDim + (size_t)head * kHeadDim * Fp;
#pragma unroll
  for (int t = 0; t < 2 * KS; ++t) {
    const int f = min(f0w + 16 * t + n, F - 1);
    const bf16x8* kp = reinterpret_cast<const bf16x8*>(Kh + (size_t)f * kHeadDim) + kg;
    it.kt[t][0] = kp[0];
    it.kt[t][1] = kp[4];
  }
#pragma unroll
  for (int st = 0; st < KS; ++st)
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      it.vt[st][dt] = *reinterpret_cast<const bf16x8*>(Vt + vt_index(16 * dt + n, f0w + 32 * st + 8 * kg));
}

template <int KS, int NW>
__device__ __forceinline__ void xitem_load(const CrossArgs& a, int head, int slot, int c, XItem<KS>& it) {
  xq_load(a, head, slot, it.qx);
  xkv_load<KS, NW>(a, head, slot, c, it.kv);
}

// The query planes of the nine rows scaled by 1/sqrt(64) (rows >= 9 zero).
__device__ __forceinline__ void xq_planes(const float4 (&qx)[2][2], bf16x8 (&qh)[2], bf16x8 (&ql)[2]) {
  const int n = threadIdx.x & 15;
  const float scale = n < kRows ? 0.125f : 0.f;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const float v[8] = {qx[h][0].x * scale, qx[h][0].y * scale, qx[h][0].z * scale, qx[h][0].w * scale,
                        qx[h][1].x * scale, qx[h][1].y * scale, qx[h][1].z * scale, qx[h][1].w * scale};
    split_planes(v, qh[h], ql[h]);
  }
}

// Block-wide barrier for LDS only: waits for this wave's LDS operations, not for
// its global loads in flight (a __syncthreads would wait for those too).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_s_waitcnt((63 & 15) | ((63 >> 4) << 14) | (7 << 4) | (0 << 8));  // lgkmcnt(0), vmcnt any
  __builtin_amdgcn_s_barrier();
}

// Scores, chunk softmax and values of chunk c whose keys and values are in `it`:
// leaves each wave's row maxima, row sums and unnormalised output rows in LDS
// (wmax / wsum / wo), readable by every thread of the block on return.
template <int KS, int NW>
__device__ __forceinline__ void xchunk_rows(const CrossArgs& a, int c, const XKv<KS>& it, const bf16x8 (&qh)[2],
                                            const bf16x8 (&ql)[2], float (*wmax)[16], float (*wsum)[16],
                                            float (*wo)[kRows][64]) {
  constexpr int NT = 2 * KS;  // 16-frame score tiles per wave
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, n = lane & 15, kg = lane >> 4;
  const int F = a.n_frames;
  const int f0w = c * a.chunk + w * 32 * KS;
  // scores and this wave's row maxima
  floatx4 sct[NT];
  float mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    floatx4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(it.kt[t][0], qh[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(it.kt[t][0], ql[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(it.kt[t][1], qh[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(it.kt[t][1], ql[1], acc, 0, 0, 0);
    sct[t] = acc;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (f0w + 16 * t + 4 * kg + i < F) mx = fmaxf(mx, acc[i]);
  }
  {
    const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    mx = fmaxf(__uint_as_float(x[0]), __uint_as_float(x[1]));
    const auto y = __builtin_amdgcn_permlane16_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
    mx = fmaxf(__uint_as_float(y[0]), __uint_as_float(y[1]));
    if (lane < 16) wmax[w][lane] = mx;
  }
  lds_barrier();
  float M = wmax[0][n];
#pragma unroll
  for (int i = 1; i < NW; ++i) M = fmaxf(M, wmax[i][n]);  // finite: frame c * chunk is present
  // probabilities and row sums
  float lsum = 0.f;
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float p = f0w + 16 * t + 4 * kg + i < F ? __expf(sct[t][i] - M) : 0.f;
      sct[t][i] = p;
      lsum += p;
    }
  // values: O^T[dim][row] over the wave's 32-frame steps
  floatx4 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int st = 0; st < KS; ++st) {
    float pb[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // tiles 2st (frames 4kg + i) and 2st + 1 (16 + 4kg + i) -> frames 8kg..8kg+7
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(sct[2 * st][i]), __float_as_uint(sct[2 * st + 1][i]),
                                                      false, false);
      const auto y = __builtin_amdgcn_permlane16_swap(x[0], x[1], false, false);
      pb[i] = __uint_as_float(y[0]);
      pb[4 + i] = __uint_as_float(y[1]);
    }
    bf16x8 ph, pl;
    split_planes(pb, ph, pl);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(it.vt[st][dt], ph, oacc[dt], 0, 0, 0);
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(it.vt[st][dt], pl, oacc[dt], 0, 0, 0);
    }
  }
  // this wave's row sums (over the four frame groups) and outputs to LDS
  {
    const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(lsum), __float_as_uint(lsum), false, false);
    lsum = __uint_as_float(x[0]) + __uint_as_float(x[1]);
    const auto y = __builtin_amdgcn_permlane16_swap(__float_as_uint(lsum), __float_as_uint(lsum), false, false);
    lsum = __uint_as_float(y[0]) + __uint_as_float(y[1]);
  }
  if (n < kRows) {
    if (lane < 16) wsum[w][n] = lsum;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) wo[w][n][16 * dt + 4 * kg + i] = oacc[dt][i];
  }
  lds_barrier();
}

// One (head, slot, chunk) item whose loads are in `it`: writes the chunk record
// (pair = slot index within the launch * H + head), or the output rows when the
// chunk is the only one and no output product is fused.
template <int KS, int NW>
__device__ __forceinline__ void xitem_compute(const CrossArgs& a, int head, int slot, int pair, int c, const XItem<KS>& it,
                                              float (*wmax)[16], float (*wsum)[16], float (*wo)[kRows][64]) {
  bf16x8 qh[2], ql[2];
  xq_planes(it.qx, qh, ql);
  xchunk_rows<KS, NW>(a, c, it.kv, qh, ql, wmax, wsum, wo);
  float* part = a.part + ((size_t)pair * a.nchunk + c) * kXrPart;
  for (int t = threadIdx.x; t < kRows * 64; t += NW * 64) {
    const int r = t >> 6, dim = t & 63;
    float o = 0.f, L = 0.f;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      o += wo[i][r][dim];
      L += wsum[i][r];
    }
    if (a.nchunk == 1 && a.op.w == nullptr) {
      put_op<bf16>(a.out, a.nsplit, a.R9, slot * kRows + r, head * kHeadDim + dim, o / L);
    } else {
      part[32 + t] = o;
      if (dim == 0) {
        float m = wmax[0][r];
#pragma unroll
        for (int i = 1; i < NW; ++i) m = fmaxf(m, wmax[i][r]);
        part[r] = m;
        part[16 + r] = L;
      }
    }
  }
}

template <int KS, int NW>
__global__ void __launch_bounds__(NW * 64) k_attn_cross_mx(CrossArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  __shared__ float wmax[NW][16];
  __shared__ float wsum[NW][16];
  __shared__ float wo[NW][kRows][64];
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y, c = blockIdx.z;
  XItem<KS> it;
  xitem_load<KS, NW>(a, head, slot, c, it);
  __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any use below
  xitem_compute<KS, NW>(a, head, slot, blockIdx.y * a.n_head + head, c, it, wmax, wsum, wo);
}

// Many (head, slot) pairs: one block per pair walks all NCH chunks of 32 KS NW
// frames, the next chunk's keys and values in flight while the current one is
// computed (two register sets used alternately: the chunk count is a
// compile-time constant, since a load under a runtime condition makes the
// compiler wait for every load in flight), and folds each chunk's rows into
// running maxima, sums and outputs with the merge's max-shifted rule.  The rows
// go straight into the next product's operand: no chunk records (their writes
// among the key and value reads cost about a tenth of the launch at 96 slots)
// and no merge launch.
template <int KS, int NW, int NCH>
__global__ void __launch_bounds__(NW * 64) k_attn_cross_pair(CrossArgs a) {
  constexpr int NI = (kRows * 64 + NW * 64 - 1) / (NW * 64);  // (row, dim) items per thread
  StampScope stamp_scope(a.stamp, NW * 64);
  // LDS partials alternate between chunks, so chunk c + 1 writes while slower
  // threads still fold chunk c
  __shared__ float wmax[2][NW][16];
  __shared__ float wsum[2][NW][16];
  __shared__ float wo[2][NW][kRows][64];
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y;
  float4 qx[2][2];
  XKv<KS> it[2];
  xq_load(a, head, slot, qx);
#pragma unroll
  for (int c = 0; c < 2 && c < NCH; ++c) xkv_load<KS, NW>(a, head, slot, c, it[c]);
  __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any use below
  bf16x8 qh[2], ql[2];
  xq_planes(qx, qh, ql);
  float rM[NI], rL[NI], rO[NI];
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    rM[i] = -INFINITY;
    rL[i] = 0.f;
    rO[i] = 0.f;
  }
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int b = c & 1;
    xchunk_rows<KS, NW>(a, c, it[b], qh, ql, wmax[b], wsum[b], wo[b]);
    if (c + 2 < NCH) {  // the set just used takes chunk c + 2
      __builtin_amdgcn_sched_barrier(0);
      xkv_load<KS, NW>(a, head, slot, c + 2, it[b]);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int t = threadIdx.x + i * NW * 64;
      if (t < kRows * 64) {
        const int r = t >> 6, dim = t & 63;
        float o = 0.f, L = 0.f, m = wmax[b][0][r];
#pragma unroll
        for (int j = 0; j < NW; ++j) {
          o += wo[b][j][r][dim];
          L += wsum[b][j][r];
          m = fmaxf(m, wmax[b][j][r]);
        }
        const float Mn = fmaxf(rM[i], m);  // finite: every chunk holds a frame
        const float f0 = __expf(rM[i] - Mn), f1 = __expf(m - Mn);  // f0 = 0 for the first chunk
        rO[i] = rO[i] * f0 + o * f1;
        rL[i] = rL[i] * f0 + L * f1;
        rM[i] = Mn;
      }
    }
  }
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int t = threadIdx.x + i * NW * 64;
    if (t < kRows * 64)
      put_op<bf16>(a.out, a.nsplit, a.R9, slot * kRows + (t >> 6), head * kHeadDim + (t & 63), rO[i] / rL[i]);
  }
}

// Merge of the chunk records of one (head, slot): one thread per (row, 4 dims).
// The records are read G chunks at a time with every load of a group issued
// together (indices clamped, chunks past the end weighted 0); groups combine with
// the same max-shifted rule.  With a fused output product (grid z = column group)
// the merged rows go to LDS and the block adds their product to h.
constexpr int kXmThreads = 640;  // a wave per column tile of the fused product's group
static_assert(kXmThreads / 64 >= kOpTiles, "merge blocks hold a wave per column tile");
template <typename S, bool FUSED, int G>
__global__ void __launch_bounds__(kXmThreads) k_attn_cross_merge(CrossArgs a) {
  StampScope stamp_scope(a.stamp, kXmThreads);
  __shared__ float Ob[kRows][64];
  __shared__ uint4 opa[FUSED ? 4 : 1][64];                          // fused output product: operand
  __shared__ float oppart[FUSED ? kOpTiles : 1][kOpTerms][16];     // and its products per wave
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y, g = blockIdx.z;
  // FUSED: the output product's weights are loaded unconditionally (a branch around
  // them would make the record loads below wait for them)
  OpPre opre;
  if constexpr (FUSED) op_load<true>(a.op, head, g, threadIdx.x, opre);
  const int t = threadIdx.x;
  // thread t < 9 * 16 merges row t / 16, dims 4 (t % 16) .. + 3 (one float4 of each
  // record), all the chunks of a group of G loaded before the first is used
  if (t < kRows * 16) {
    const int r = t >> 4, d4 = 4 * (t & 15);
    const float* part = a.part + (size_t)(blockIdx.y * a.n_head + head) * a.nchunk * kXrPart;
    float M = -INFINITY, L = 0.f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int c0 = 0; c0 < a.nchunk; c0 += G) {
      float m[G], l[G];
      float4 v[G];
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float* pc = part + (size_t)min(c0 + j, a.nchunk - 1) * kXrPart;
        m[j] = pc[r];
        l[j] = pc[16 + r];
        v[j] = *reinterpret_cast<const float4*>(pc + 32 + r * 64 + d4);
      }
      float Mg = M;
#pragma unroll
      for (int j = 0; j < G; ++j) Mg = fmaxf(Mg, m[j]);
      const float f0 = __expf(M - Mg);  // 0 before the first group
      L *= f0;
      o.x *= f0;
      o.y *= f0;
      o.z *= f0;
      o.w *= f0;
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const float f = c0 + j < a.nchunk ? __expf(m[j] - Mg) : 0.f;
        L = fmaf(f, l[j], L);
        o.x = fmaf(f, v[j].x, o.x);
        o.y = fmaf(f, v[j].y, o.y);
        o.z = fmaf(f, v[j].z, o.z);
        o.w = fmaf(f, v[j].w, o.w);
      }
      M = Mg;
    }
    const float ov[4] = {o.x / L, o.y / L, o.z / L, o.w / L};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if constexpr (FUSED) Ob[r][d4 + k] = ov[k];
      else put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + r, head * kHeadDim + d4 + k, ov[k]);
    }
  }
  if constexpr (FUSED) {
    __syncthreads();
    op_apply(a.op, head, g, t, opre, Ob, slot * kRows, opa, oppart);
  }
}

// Merge launch with a chunk group that covers the usual chunk counts in one pass.
template <typename S, bool FUSED>
static void launch_merge(const CrossArgs& a, int n, hipStream_t st) {
  const dim3 grid(a.n_head, n, FUSED ? kOpGroups : 1);
  if (a.nchunk <= 4) k_attn_cross_merge<S, FUSED, 4><<<grid, kXmThreads, 0, st>>>(a);
  else if (a.nchunk <= 12) k_attn_cross_merge<S, FUSED, 12><<<grid, kXmThreads, 0, st>>>(a);
  else k_attn_cross_merge<S, FUSED, 16><<<grid, kXmThreads, 0, st>>>(a);
}

// ---------------------------------------------------------------- causal self-attention
// Verify pass: row i < nv of slot s sits at position pos0 + i and attends to cached
// positions 0..pos0 + i (Section 3.1: one causal pass).  Rows i >= nv are padding
// and get zeros.  All keys of a row fit one batch (4 waves x 14 octets = 448).
constexpr int kSelfThreads = 256;
template <typename S>
__global__ void __launch_bounds__(kSelfThreads) k_attn_self(AttnArgs a) {
  StampScope stamp_scope(a.stamp, kSelfThreads);
  constexpr int NW = kSelfThreads / 64;
  static_assert(NW * 14 * 8 >= kMaxCtx, "one batch of key octets covers the context");
  __shared__ float part[NW][4][64];
  __shared__ float pm[NW], pl[NW];
  __shared__ int pts[kMaxCtx / kPage];
  int head, row;
  if (!head_row(blockIdx.x, a.n_head, head, row)) return;
  const int slot = a.slot0 + blockIdx.y;
  const int* st = a.state + slot * kStateInts;
  // state, page table and query are independent loads
  if (threadIdx.x < a.pages_per_slot) pts[threadIdx.x] = a.page_table[slot * a.pages_per_slot + threadIdx.x];
  const int pos0 = st[ST_POS0], nv = st[ST_NV];
  const int lane = threadIdx.x & 63, g = lane & 7;
  const float* qr = a.q + (size_t)(slot * kRows + row) * a.ldq + head * kHeadDim + 8 * g;
  float q8[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) q8[e] = qr[e] * 0.125f;
  __syncthreads();
  if (row >= nv) {
    if (threadIdx.x < kHeadDim) put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + row, head * kHeadDim + threadIdx.x, 0.f);
    return;
  }
  const int nk = pos0 + row + 1;
  const S* Kc = reinterpret_cast<const S*>(a.kcache);
  const S* Vc = reinterpret_cast<const S*>(a.vcache);
  const int H = a.n_head;
  float m, l, acc[8];
  attend_wave<S, NW, 14>(
      q8, nk, Kc, Vc, [&](int j) { return (((uint32_t)pts[j >> 4] * H + head) * kPage + (j & 15)) * kHeadDim; }, m, l,
      acc);
  const float o = merge_waves<NW>(m, l, acc, part, pm, pl);
  if (threadIdx.x < kHeadDim)
    put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + row, head * kHeadDim + threadIdx.x, o);
}

// ---------------------------------------------------------------- causal self-attention, bf16, matrix cores
// Block (head, slot): all nine rows of the pass over the slot's cached positions
// 0..pos0 + nv - 1 (the pass's own rows included); wave w takes positions
// 32w..32w+31 (logical pages 2w and 2w + 1), so kMaxCtx / 32 waves cover the
// context and waves past the last key only take part in the combine.  Values
// are stored transposed within a page ([page][head][64][16]).  A wave computes
// S^T = K q^T for its two 16-position tiles (query rows as hi + lo bf16 planes),
// applies the causal mask (row i sees positions <= pos0 + i), takes its own row
// maxima m_w, p = exp(s - m_w), the row sums l_w and O_w^T = V^T P^T as in the
// cross-attention; the waves' (m_w, l_w, O_w) are then combined max-shifted in
// LDS.  Rows i >= nv are padding and get zeros.
constexpr int kSxWaves = kMaxCtx / 32;
constexpr int kSxThreads = kSxWaves * 64;
static_assert(kSxWaves >= kOpTiles, "self-attention blocks hold a wave per column tile of the fused product");
template <bool FUSED>
__global__ void __launch_bounds__(kSxThreads) k_attn_self_mx(AttnArgs a) {
  StampScope stamp_scope(a.stamp, kSxThreads);
  __shared__ float wmax[kSxWaves][16];
  __shared__ float wsum[kSxWaves][16];
  __shared__ float wo[kSxWaves][kRows][64];
  __shared__ float Ob[kRows][64];
  __shared__ uint4 opa[FUSED ? 4 : 1][64];                          // fused output product: operand
  __shared__ float oppart[FUSED ? kOpTiles : 1][kOpTerms][16];     // and its products per wave
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y, g = blockIdx.z;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, n = lane & 15, kg = lane >> 4;
  const int* st = a.state + slot * kStateInts;
  // The wave's two page-table entries, the slot state and the query rows are
  // independent loads, issued first; the fused output product's weights (FUSED,
  // unconditional) follow, so the key and value loads wait for the page entries
  // alone (loads complete in issue order).
  const int* ptab = a.page_table + (size_t)slot * a.pages_per_slot;
  const int pe0 = ptab[min(2 * w, a.pages_per_slot - 1)], pe1 = ptab[min(2 * w + 1, a.pages_per_slot - 1)];
  const int pos0 = st[ST_POS0], nv = st[ST_NV];
  float4 qx[2][2];
  {
    const float* qr = a.q + (size_t)(slot * kRows + min(n, kRows - 1)) * a.ldq + head * kHeadDim + 8 * kg;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      qx[h][0] = *reinterpret_cast<const float4*>(qr + 32 * h);
      qx[h][1] = *reinterpret_cast<const float4*>(qr + 32 * h + 4);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  OpPre opre;
  if constexpr (FUSED) op_load<false>(a.op, head, g, threadIdx.x, opre);
  __builtin_amdgcn_sched_barrier(0);
  float mrow = -INFINITY, lrow = 0.f;
  floatx4 oacc[4];
#pragma unroll
  for (int dt = 0; dt < 4; ++dt) oacc[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  if (32 * w < pos0 + nv) {  // this wave holds keys (uniform)
    const int pg0 = pe0, pg1 = pe1;
    const bf16* Kc = reinterpret_cast<const bf16*>(a.kcache);
    const bf16* Vc = reinterpret_cast<const bf16*>(a.vcache);
    const int H = a.n_head;
    bf16x8 kt[2][2], vt[4];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const bf16x8* kp = reinterpret_cast<const bf16x8*>(Kc + (((size_t)(t ? pg1 : pg0) * H + head) * kPage + n) * kHeadDim) + kg;
      kt[t][0] = kp[0];
      kt[t][1] = kp[4];
    }
    const size_t vpage = (size_t)(kg < 2 ? pg0 : pg1) * H + head;
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
      vt[dt] = *reinterpret_cast<const bf16x8*>(Vc + (vpage * kHeadDim + 16 * dt + n) * kPage + 8 * (kg & 1));
    __builtin_amdgcn_sched_barrier(0);  // every load above is issued before any use below
    bf16x8 qh[2], ql[2];
    {
      const float scale = n < kRows ? 0.125f : 0.f;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const float v[8] = {qx[h][0].x * scale, qx[h][0].y * scale, qx[h][0].z * scale, qx[h][0].w * scale,
                            qx[h][1].x * scale, qx[h][1].y * scale, qx[h][1].z * scale, qx[h][1].w * scale};
        split_planes(v, qh[h], ql[h]);
      }
    }
    floatx4 sct[2];
    float mx = -INFINITY;
    const int last = pos0 + n;  // row n sees positions <= last
    const bool row_ok = n < nv;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      floatx4 acc = {0.f, 0.f, 0.f, 0.f};
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[t][0], qh[0], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[t][0], ql[0], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[t][1], qh[1], acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kt[t][1], ql[1], acc, 0, 0, 0);
      sct[t] = acc;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (row_ok && 32 * w + 16 * t + 4 * kg + i <= last) mx = fmaxf(mx, acc[i]);
    }
    {
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(x[0]), __uint_as_float(x[1]));
      const auto y = __builtin_amdgcn_permlane16_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
      mx = fmaxf(__uint_as_float(y[0]), __uint_as_float(y[1]));
    }
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool ok = row_ok && 32 * w + 16 * t + 4 * kg + i <= last;  // then mx is finite
        const float p = ok ? __expf(sct[t][i] - mx) : 0.f;
        sct[t][i] = p;
        ls += p;
      }
    float pb[8];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(sct[0][i]), __float_as_uint(sct[1][i]), false, false);
      const auto y = __builtin_amdgcn_permlane16_swap(x[0], x[1], false, false);
      pb[i] = __uint_as_float(y[0]);
      pb[4 + i] = __uint_as_float(y[1]);
    }
    bf16x8 ph, pl;
    split_planes(pb, ph, pl);
#pragma unroll
    for (int dt = 0; dt < 4; ++dt) {
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt[dt], ph, oacc[dt], 0, 0, 0);
      oacc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt[dt], pl, oacc[dt], 0, 0, 0);
    }
    {
      const auto x = __builtin_amdgcn_permlane32_swap(__float_as_uint(ls), __float_as_uint(ls), false, false);
      ls = __uint_as_float(x[0]) + __uint_as_float(x[1]);
      const auto y = __builtin_amdgcn_permlane16_swap(__float_as_uint(ls), __float_as_uint(ls), false, false);
      ls = __uint_as_float(y[0]) + __uint_as_float(y[1]);
    }
    mrow = mx;
    lrow = ls;
  }
  if (lane < 16) {
    wmax[w][lane] = mrow;
    wsum[w][lane] = lrow;
  }
  if (n < kRows) {
#pragma unroll
    for (int dt = 0; dt < 4; ++dt)
#pragma unroll
      for (int i = 0; i < 4; ++i) wo[w][n][16 * dt + 4 * kg + i] = oacc[dt][i];
  }
  __syncthreads();
  if (a.clear_q) {  // every wave that multiplies has used its query values by now
    for (int t = threadIdx.x; t < kRows * 64; t += kSxThreads)
      const_cast<float*>(a.q)[(size_t)(slot * kRows + (t >> 6)) * a.ldq + head * kHeadDim + (t & 63)] = 0.f;
  }
  for (int t = threadIdx.x; t < kRows * 64; t += kSxThreads) {
    const int r = t >> 6, dim = t & 63;
    float o = 0.f;
    if (r < nv) {
      float M = wmax[0][r];  // finite: wave 0 holds position 0
#pragma unroll
      for (int i = 1; i < kSxWaves; ++i) M = fmaxf(M, wmax[i][r]);
      float L = 0.f;
#pragma unroll
      for (int i = 0; i < kSxWaves; ++i) {
        const float f = __expf(wmax[i][r] - M);  // 0 for a wave without keys of this row
        L = fmaf(f, wsum[i][r], L);
        o = fmaf(f, wo[i][r][dim], o);
      }
      o /= L;
    }
    if constexpr (FUSED) Ob[r][dim] = o;
    else put_op<bf16>(a.out, a.nsplit, a.R9, slot * kRows + r, head * kHeadDim + dim, o);
  }
  if constexpr (FUSED) {
    __syncthreads();
    op_apply(a.op, head, g, threadIdx.x, opre, Ob, slot * kRows, opa, oppart);
  }
}

// ---------------------------------------------------------------- drafter attention
// Block row i (position t+i, t = anchor position) attends in one softmax to the
// history keys at positions 0..t-1 and to all nine block keys (Section 3.2:
// bidirectional inside the block).  The query and the block keys get RoPE here
// (rotate-half, pairs (j, j+32)); history keys were stored with RoPE at their own
// positions.  Ablation variants: without history the nine block keys are all the
// keys; with absolute positions nothing is rotated.
template <typename S>
__global__ void __launch_bounds__(kSelfThreads) k_attn_draft(AttnArgs a) {
  StampScope stamp_scope(a.stamp, kSelfThreads);
  constexpr int NT = kSelfThreads, NW = NT / 64;
  __shared__ float sc[kMaxCtx + 16];
  __shared__ float part[NW][64];
  __shared__ float red[NW];
  __shared__ float kb[kRows][kHeadDim];
  __shared__ float vb[kRows][kHeadDim];
  int head, row;
  if (!head_row(blockIdx.x, a.n_head, head, row)) return;
  const int slot = a.slot0 + blockIdx.y;
  const int t0 = a.state[slot * kStateInts + ST_L];
  const int nh = a.draft_hist ? t0 : 0;  // history keys attended
  const int d = a.d;
  const int lane = threadIdx.x & 63, g = lane & 7;
  // rotated block keys and their values
  for (int t = threadIdx.x; t < kRows * 32; t += NT) {
    const int jb = t >> 5, j = t & 31;
    const int pos = t0 + jb;
    const float c = a.draft_rope ? a.rope[(pos * 32 + j) * 2] : 1.f;
    const float sn = a.draft_rope ? a.rope[(pos * 32 + j) * 2 + 1] : 0.f;
    const float* kr = a.q + (size_t)(slot * kRows + jb) * a.ldq + d + head * kHeadDim;
    const float* vr = kr + d;
    const float k1 = kr[j], k2 = kr[j + 32];
    kb[jb][j] = k1 * c - k2 * sn;
    kb[jb][j + 32] = k1 * sn + k2 * c;
    vb[jb][j] = vr[j];
    vb[jb][j + 32] = vr[j + 32];
  }
  // this lane's 8 rotated query dims
  float q8[8];
  {
    const float* qr = a.q + (size_t)(slot * kRows + row) * a.ldq + head * kHeadDim;
    const int pos = t0 + row;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int dim = 8 * g + e, j = dim & 31;
      const float c = a.draft_rope ? a.rope[(pos * 32 + j) * 2] : 1.f;
      const float sn = a.draft_rope ? a.rope[(pos * 32 + j) * 2 + 1] : 0.f;
      const float u1 = qr[j], u2 = qr[j + 32];
      q8[e] = (dim < 32 ? u1 * c - u2 * sn : u1 * sn + u2 * c) * 0.125f;
    }
  }
  const S* Kh = reinterpret_cast<const S*>(a.kcache) + ((size_t)slot * a.n_head + head) * a.n_ctx * kHeadDim;
  const S* Vh = reinterpret_cast<const S*>(a.vcache) + ((size_t)slot * a.n_head + head) * a.n_ctx * kHeadDim;
  score_pass<S, NT, 14>(q8, nh, [&](int j) { return Kh + (size_t)j * kHeadDim; }, sc);
  __syncthreads();
  // the nine block keys: one wave, lane (key kl, dims 8g..), keys 0..7 then key 8
  if (threadIdx.x < 64) {
    const int kl = lane >> 3;
    for (int half = 0; half < 2; ++half) {
      const int jb = half * 8 + kl;
      float s = 0.f;
      if (jb < kRows) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s = fmaf(q8[e], kb[jb][8 * g + e], s);
      }
      s = key_sum(s);
      if (g == 0 && jb < kRows) sc[nh + jb] = s;
    }
  }
  __syncthreads();
  const int nk = nh + kRows;
  const float L = softmax_pass<NT>(sc, nk, red);
  __syncthreads();
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  value_pass<S, NT, 14>(acc, nh, [&](int j) { return Vh + (size_t)j * kHeadDim; }, sc);
  if (threadIdx.x < 64) {
    const int kl = lane >> 3;
    for (int half = 0; half < 2; ++half) {
      const int jb = half * 8 + kl;
      if (jb < kRows) {
        const float pk = sc[nh + jb];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] = fmaf(pk, vb[jb][8 * g + e], acc[e]);
      }
    }
  }
  reduce_out<NT>(acc, part);
  if (threadIdx.x < kHeadDim) {
    const float o = (part[0][threadIdx.x] + part[1][threadIdx.x]) + (part[2][threadIdx.x] + part[3][threadIdx.x]);
    put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + row, head * kHeadDim + threadIdx.x, o / L);
  }
}

// Drafter attention (Section 3.2, Eq. 2; Appendix A.2) with all nine block rows of
// a (head, slot) in one block: one softmax over the history positions before the
// anchor and the nine block rows (bidirectional inside the block), RoPE on the
// queries and the block keys (the history keys were stored rotated), scores / 8.
// Each history key and value is read once per block for all nine rows (a block per
// (head, row) read the slot's history nine times: 183 us per launch at 96 slots).
// Scores: thread t takes keys t, t + 256 (loaded together, both at once) and forms
// the nine rows' dot products against the rotated queries in LDS; softmax per row
// by one wave; values: wave w sums keys w, w + 4, ... for all rows and its lane's
// dim, eight keys' values in flight, and the four waves' partial sums are added in
// a fixed order.
constexpr int kDrThreads = 256;
constexpr int kDrKeys = (kMaxCtx + kRows + kDrThreads - 1) / kDrThreads;  // keys per thread in the score pass
constexpr int kDrSc = kMaxCtx + kRows + 3;                                // score row stride (floats)
constexpr int kDrMinBlocks = 160;  // (head, slot) blocks from which the all-rows kernel is used

template <typename S>
__global__ void __launch_bounds__(kDrThreads) k_attn_draft_rows(AttnArgs a) {
  StampScope stamp_scope(a.stamp, kDrThreads);
  constexpr int NW = kDrThreads / 64;
  static_assert(NW == 4, "the partial sums of four waves are added below");
  __shared__ float qs[kRows][kHeadDim];
  __shared__ float kb[kRows][kHeadDim];
  __shared__ float vb[kRows][kHeadDim];
  __shared__ float sc[kRows][kDrSc];
  __shared__ float part[NW][kRows][kHeadDim];
  __shared__ float rsum[kRows];
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int t0 = a.state[slot * kStateInts + ST_L];
  const int nh = a.draft_hist ? min(t0, a.n_ctx) : 0;  // history keys attended
  const int nk = nh + kRows;
  const int d = a.d;
  const S* Kh = reinterpret_cast<const S*>(a.kcache) + ((size_t)slot * a.n_head + head) * a.n_ctx * kHeadDim;
  const S* Vh = reinterpret_cast<const S*>(a.vcache) + ((size_t)slot * a.n_head + head) * a.n_ctx * kHeadDim;
  // this thread's history keys (clamped into the cache; keys past nh are not used),
  // issued before the block rows are staged
  float kv[kDrKeys][kHeadDim];
#pragma unroll
  for (int u = 0; u < kDrKeys; ++u) {
    const int j = min((int)threadIdx.x + u * kDrThreads, max(nh - 1, 0));
#pragma unroll
    for (int c = 0; c < kHeadDim; c += 8) ld8(Kh + (size_t)j * kHeadDim + c, &kv[u][c]);
  }
  // rotated, scaled queries; rotated block keys; block values
  for (int t = threadIdx.x; t < kRows * 32; t += kDrThreads) {
    const int r = t >> 5, j = t & 31, pos = t0 + r;
    const float c = a.draft_rope ? a.rope[(pos * 32 + j) * 2] : 1.f;
    const float sn = a.draft_rope ? a.rope[(pos * 32 + j) * 2 + 1] : 0.f;
    const float* qr = a.q + (size_t)(slot * kRows + r) * a.ldq + head * kHeadDim;
    const float* kr = qr + d;
    const float* vr = qr + 2 * d;
    const float q1 = qr[j], q2 = qr[j + 32], k1 = kr[j], k2 = kr[j + 32];
    qs[r][j] = (q1 * c - q2 * sn) * 0.125f;
    qs[r][j + 32] = (q1 * sn + q2 * c) * 0.125f;
    kb[r][j] = k1 * c - k2 * sn;
    kb[r][j + 32] = k1 * sn + k2 * c;
    vb[r][j] = vr[j];
    vb[r][j + 32] = vr[j + 32];
  }
  __syncthreads();
  // scores of keys t, t + 256: history keys from registers, block keys from LDS
#pragma unroll
  for (int u = 0; u < kDrKeys; ++u) {
    const int j = (int)threadIdx.x + u * kDrThreads;
    if (j >= nk) continue;
    if (j >= nh) {
#pragma unroll
      for (int e = 0; e < kHeadDim; ++e) kv[u][e] = kb[j - nh][e];
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < kHeadDim; ++e) s = fmaf(qs[r][e], kv[u][e], s);
      sc[r][j] = s;
    }
  }
  __syncthreads();
  // softmax numerators per row (max subtracted) and their sums
  for (int r = wv; r < kRows; r += NW) {
    float m = -INFINITY;
    for (int j = lane; j < nk; j += 64) m = fmaxf(m, sc[r][j]);
    m = wave_max(m);
    float sum = 0.f;
    for (int j = lane; j < nk; j += 64) {
      const float p = expf(sc[r][j] - m);
      sc[r][j] = p;
      sum += p;
    }
    sum = wave_sum(sum);
    if (lane == 0) rsum[r] = sum;
  }
  __syncthreads();
  // values: wave wv sums keys wv, wv + 4, ... (eight in flight) for its lane's dim
  float acc[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) acc[r] = 0.f;
  for (int j0 = wv; j0 < nh; j0 += 8 * NW) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = to_f(Vh[(size_t)min(j0 + u * NW, nh - 1) * kHeadDim + lane]);
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int j = j0 + u * NW;
      if (j < nh) {
#pragma unroll
        for (int r = 0; r < kRows; ++r) acc[r] = fmaf(sc[r][j], v[u], acc[r]);
      }
    }
  }
  for (int jb = wv; jb < kRows; jb += NW) {
    const float v = vb[jb][lane];
#pragma unroll
    for (int r = 0; r < kRows; ++r) acc[r] = fmaf(sc[r][nh + jb], v, acc[r]);
  }
#pragma unroll
  for (int r = 0; r < kRows; ++r) part[wv][r][lane] = acc[r];
  __syncthreads();
  for (int t = threadIdx.x; t < kRows * kHeadDim; t += kDrThreads) {
    const int r = t / kHeadDim, dim = t % kHeadDim;
    const float o = (part[0][r][dim] + part[1][r][dim]) + (part[2][r][dim] + part[3][r][dim]);
    put_op<S>(a.out, a.nsplit, a.R9, slot * kRows + r, head * kHeadDim + dim, o / rsum[r]);
  }
}

// ---------------------------------------------------------------- launchers
static inline unsigned row_blocks(int H) { return (unsigned)(8 * ((H + 7) / 8) * kRows); }

template <typename S>
void Ops<S>::attn_self(const AttnArgs& a, int n, hipStream_t st) {
  if constexpr (sizeof(S) == 2) {
    if (a.op.w != nullptr) k_attn_self_mx<true><<<dim3(a.n_head, n, kOpGroups), kSxThreads, 0, st>>>(a);
    else k_attn_self_mx<false><<<dim3(a.n_head, n, 1), kSxThreads, 0, st>>>(a);
  }
  else k_attn_self<S><<<dim3(row_blocks(a.n_head), n), kSelfThreads, 0, st>>>(a);
}
template <typename S>
void Ops<S>::attn_draft(const AttnArgs& a, int n, hipStream_t st) {
  // a few slots: a block per (head, row) fills more of the chip (20 all-rows blocks
  // at one slot took 13.3 us per launch against 8.6); with more slots the history is
  // read once per (head, slot)
  if (n * a.n_head >= kDrMinBlocks) k_attn_draft_rows<S><<<dim3(a.n_head, n), kDrThreads, 0, st>>>(a);
  else k_attn_draft<S><<<dim3(row_blocks(a.n_head), n), kSelfThreads, 0, st>>>(a);
}
// enough slots to fill the chip with (head, slot) blocks: all rows per block;
// otherwise one block per (head, row)
template <typename S>
void Ops<S>::attn_cross(const CrossArgs& a, int n, hipStream_t st) {
  if constexpr (sizeof(S) == 2) {  // transposed values, matrix cores, frame chunks + merge
    if (a.by_pair) {  // one block per (head, slot) over every chunk: no merge
      const dim3 grid(a.n_head, n);
      switch (a.nchunk) {
#define WF_XPAIR(N) \
  case N: k_attn_cross_pair<1, 4, N><<<grid, 256, 0, st>>>(a); break;
        WF_XPAIR(1) WF_XPAIR(2) WF_XPAIR(3) WF_XPAIR(4) WF_XPAIR(5) WF_XPAIR(6)
        WF_XPAIR(7) WF_XPAIR(8) WF_XPAIR(9) WF_XPAIR(10) WF_XPAIR(11) WF_XPAIR(12)
#undef WF_XPAIR
      }
      return;
    }
    if (a.chunk == 128) k_attn_cross_mx<1, 4><<<dim3(a.n_head, n, a.nchunk), 256, 0, st>>>(a);
    else k_attn_cross_mx<2, 8><<<dim3(a.n_head, n, a.nchunk), 512, 0, st>>>(a);
  } else {
    if (n == 1) {  // one slot: a block per (head, row) streams all frames (9 blocks per head share an L2)
      k_attn_cross<S><<<dim3(row_blocks(a.n_head), n), kCrossThreads, 0, st>>>(a);
      return;
    }
    k_attn_cross_rows<S><<<dim3(a.n_head, n, a.nchunk), kXrThreads, xr_lds_bytes(a.chunk), st>>>(a);
  }
  if (a.nchunk > 1 || a.op.w != nullptr) {
    if (a.op.w != nullptr) launch_merge<S, true>(a, n, st);
    else launch_merge<S, false>(a, n, st);
  }
}

template void Ops<float>::attn_self(const AttnArgs&, int, hipStream_t);
template void Ops<bf16>::attn_self(const AttnArgs&, int, hipStream_t);
template void Ops<float>::attn_draft(const AttnArgs&, int, hipStream_t);
template void Ops<bf16>::attn_draft(const AttnArgs&, int, hipStream_t);
template void Ops<float>::attn_cross(const CrossArgs&, int, hipStream_t);
template void Ops<bf16>::attn_cross(const CrossArgs&, int, hipStream_t);

}  // namespace wf
