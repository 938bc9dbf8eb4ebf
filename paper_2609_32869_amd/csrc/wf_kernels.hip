// HIP kernels of the Whisper-Flash draft-and-verify step (gfx950, wave64).
//
// Rows: a pass over slot s uses activation rows s*9 + i, i = 0..8 (anchor plus
// eight candidates, or eight masks for the drafter).  Every kernel computes a
// row's result the same way however many rows or slots share the launch, so a
// token's logits never depend on the batch composition.
#include "../../include/wf.h"
#include "wf_kernels.h"

namespace wf {

// ---------------------------------------------------------------- block reductions
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[w] = v;
  __syncthreads();
  float t = red[0] + red[1] + red[2] + red[3];
  return t;
}

// ---------------------------------------------------------------- LayerNorm
// y = g * (x - mean) / sqrt(var + 1e-5) + b over the d columns of each row
// (Whisper's pre-LN blocks and final LN).  One block of 256 threads per row.
template <typename S>
__global__ void __launch_bounds__(256) k_layernorm(const float* __restrict__ x, const S* __restrict__ g,
                                                   const S* __restrict__ b, float* __restrict__ y, int d,
                                                   int row0) {
  __shared__ float red[4];
  const int row = row0 + blockIdx.x;
  const float* xr = x + (size_t)row * d;
  float* yr = y + (size_t)row * d;
  float s = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) s += xr[i];
  const float mean = block_sum256(s, red) / (float)d;
  float v = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float c = xr[i] - mean;
    v += c * c;
  }
  const float var = block_sum256(v, red) / (float)d;
  const float inv = 1.0f / sqrtf(var + 1e-5f);
  for (int i = threadIdx.x; i < d; i += 256) yr[i] = (xr[i] - mean) * inv * to_f(g[i]) + to_f(b[i]);
}

// ---------------------------------------------------------------- GEMV (rows x W^T)
// y[row, n] = sum_k x[row, k] * W[n, k] for the 9 rows of every slot.
// Block: 256 threads = 4 waves, 16 output columns (4 per wave); lanes split K in
// 8-element chunks (16-byte loads of bf16 weights).  fp32 accumulation.
template <typename S, int EPI>
__global__ void __launch_bounds__(256) k_gemv(GemvArgs a) {
  __shared__ float sv[kRows][16];
  const S* __restrict__ W = reinterpret_cast<const S*>(a.w);
  const S* __restrict__ bias = reinterpret_cast<const S*>(a.bias);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int nb = blockIdx.x * 16;
  const int n0 = nb + wv * 4;
  const int K = a.K, N = a.N;
  for (int s = 0; s < a.nslots; ++s) {
    const int slot = a.slot0 + s;
    const float* __restrict__ xs = a.x + (size_t)slot * kRows * a.ldx;
    float acc[kRows][4];
#pragma unroll
    for (int r = 0; r < kRows; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) acc[r][c] = 0.f;
    for (int k = lane * 8; k < K; k += 512) {
      float w[4][8];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        if (n0 + c < N) {
          ld8(W + (size_t)(n0 + c) * K + k, w[c]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; ++e) w[c][e] = 0.f;
        }
      }
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        float xv[8];
        ld8(xs + (size_t)r * a.ldx + k, xv);
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[r][c] = fmaf(xv[e], w[c][e], acc[r][c]);
      }
    }
    float mine = 0.f;
#pragma unroll
    for (int r = 0; r < kRows; ++r)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float t = wave_sum(acc[r][c]);
        if (lane == r * 4 + c) mine = t;
      }
    const int r = lane >> 2, c = lane & 3;
    const int n = n0 + c;
    const bool act = lane < kRows * 4 && n < N;
    const int row = slot * kRows + r;
    float v = mine;
    if (act && bias != nullptr) v += to_f(bias[n]);
    if constexpr (EPI == EPI_STORE) {
      if (act) a.y[(size_t)row * a.ldy + n] = v;
    } else if constexpr (EPI == EPI_GELU) {
      if (act) a.y[(size_t)row * a.ldy + n] = gelu_erf(v);
    } else if constexpr (EPI == EPI_RESID) {
      if (act) {
        float* p = a.y + (size_t)row * a.ldy + n;
        float hn = *p + v;
        *p = hn;
        if (a.tap >= 0) a.taps[(((size_t)slot * kRows + r) * a.n_tap + a.tap) * N + n] = hn;
      }
    } else if constexpr (EPI == EPI_QKV) {
      // q -> y; k, v -> paged self-attention cache at position pos0 + r (valid rows only)
      if (act) {
        const int d = a.d;
        if (n < d) {
          a.y[(size_t)row * a.ldy + n] = v;
        } else {
          const int* st = a.state + slot * kStateInts;
          const int nv = st[ST_NV], pos = st[ST_POS0] + r;
          if (r < nv && pos < a.n_ctx) {
            const int kv = n >= 2 * d;
            const int col = n - d - kv * d, head = col >> 6, dim = col & 63;
            const int page = a.page_table[slot * a.pages_per_slot + (pos >> 4)];
            S* cache = reinterpret_cast<S*>(a.cache) + (size_t)kv * a.kv_stride;
            cache[(((size_t)page * a.n_head + head) * kPage + (pos & 15)) * kHeadDim + dim] = from_f<S>(v);
          }
        }
      }
    } else if constexpr (EPI == EPI_ARGMAX) {
      if (act && a.y != nullptr) a.y[(size_t)row * a.ldy + n] = v;
      __syncthreads();
      if (lane < kRows * 4) sv[r][wv * 4 + c] = (n < N) ? v : -INFINITY;
      __syncthreads();
      if (threadIdx.x < kRows) {
        const int rr = threadIdx.x;
        float bv = sv[rr][0];
        int bi = nb;
        for (int j = 1; j < 16; ++j) {
          if (nb + j >= N) break;
          if (better(sv[rr][j], nb + j, bv, bi)) { bv = sv[rr][j]; bi = nb + j; }
        }
        const size_t o = (size_t)(slot * kRows + rr) * a.nblk + blockIdx.x;
        a.hv[o] = bv;
        a.hi[o] = bi;
      }
    }
  }
}

// final argmax over the per-block partials of each row; flags non-finite maxima
__global__ void __launch_bounds__(256) k_argmax_final(const float* __restrict__ hv, const int* __restrict__ hi,
                                                      int nblk, int row0, int* __restrict__ g,
                                                      float* __restrict__ gmax, unsigned* status) {
  __shared__ float bvs[4];
  __shared__ int bis[4];
  const int row = row0 + blockIdx.x;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int j = threadIdx.x; j < nblk; j += 256) {
    float v = hv[(size_t)row * nblk + j];
    int i = hi[(size_t)row * nblk + j];
    if (better(v, i, bv, bi)) { bv = v; bi = i; }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    float ov = __shfl_xor(bv, o, 64);
    int oi = __shfl_xor(bi, o, 64);
    if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) { bvs[w] = bv; bis[w] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int j = 1; j < 4; ++j)
      if (better(bvs[j], bis[j], bvs[0], bis[0])) { bvs[0] = bvs[j]; bis[0] = bis[j]; }
    g[row] = bis[0];
    gmax[row] = bvs[0];
    if (!isfinite(bvs[0])) atomicOr(status, WF_STATUS_NONFINITE_LOGITS);
  }
}

// ---------------------------------------------------------------- causal self-attention
// Target verify pass: rows i < nv of slot s sit at positions pos0 + i and attend to
// cached positions 0..pos0 + i (Section 3.1: one causal pass).  One block per
// (head, slot); scores for all rows are kept in LDS.
template <typename S>
__global__ void __launch_bounds__(256) k_attn_self(AttnArgs a) {
  __shared__ float qs[kRows][kHeadDim];
  __shared__ float sc[kRows][kMaxCtx + 16];
  __shared__ float part[4][kRows][kHeadDim];
  __shared__ float rmax[kRows], rsum[kRows];
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y;
  const int* st = a.state + slot * kStateInts;
  const int pos0 = st[ST_POS0], nv = st[ST_NV];
  const int T = pos0 + nv;
  const int d = a.d;
  const float scale = 0.125f;
  for (int t = threadIdx.x; t < kRows * kHeadDim; t += 256) {
    int r = t >> 6, j = t & 63;
    qs[r][j] = a.q[(size_t)(slot * kRows + r) * a.ldq + head * kHeadDim + j] * scale;
  }
  __syncthreads();
  const S* Kc = reinterpret_cast<const S*>(a.kcache);
  const S* Vc = reinterpret_cast<const S*>(a.vcache);
  const int* pt = a.page_table + slot * a.pages_per_slot;
  for (int j = threadIdx.x; j < T; j += 256) {
    const int page = pt[j >> 4];
    const S* kp = Kc + (((size_t)page * a.n_head + head) * kPage + (j & 15)) * kHeadDim;
    float kv[kHeadDim];
#pragma unroll
    for (int e = 0; e < kHeadDim; e += 8) ld8(kp + e, kv + e);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < kHeadDim; ++e) s = fmaf(qs[r][e], kv[e], s);
      sc[r][j] = (j <= pos0 + r) ? s : -INFINITY;
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int r = w; r < kRows; r += 4) {
    float m = -INFINITY;
    for (int j = lane; j < T; j += 64) m = fmaxf(m, sc[r][j]);
    m = wave_max(m);
    float l = 0.f;
    for (int j = lane; j < T; j += 64) {
      float e = (sc[r][j] == -INFINITY) ? 0.f : __expf(sc[r][j] - m);
      sc[r][j] = e;
      l += e;
    }
    l = wave_sum(l);
    if (lane == 0) { rmax[r] = m; rsum[r] = l; }
  }
  __syncthreads();
  // P V: thread (w, dim) sums keys j = w, w+4, ...
  {
    const int dim = lane;
    float acc[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) acc[r] = 0.f;
    for (int j = w; j < T; j += 4) {
      const int page = pt[j >> 4];
      const float vv = to_f(Vc[(((size_t)page * a.n_head + head) * kPage + (j & 15)) * kHeadDim + dim]);
#pragma unroll
      for (int r = 0; r < kRows; ++r) acc[r] = fmaf(sc[r][j], vv, acc[r]);
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) part[w][r][dim] = acc[r];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < kRows * kHeadDim; t += 256) {
    int r = t >> 6, j = t & 63;
    float o = (part[0][r][j] + part[1][r][j]) + (part[2][r][j] + part[3][r][j]);
    float out = (r < nv) ? o / rsum[r] : 0.f;
    a.out[(size_t)(slot * kRows + r) * d + head * kHeadDim + j] = out;
  }
}

// ---------------------------------------------------------------- drafter attention
// Block rows (positions t..t+8, t = anchor position) attend in one softmax to
// the history keys at positions 0..t-1 and to all nine block keys (Section 3.2:
// bidirectional inside the block).  Queries and block keys get RoPE here; history
// keys were stored with RoPE at their own positions.
template <typename S>
__global__ void __launch_bounds__(256) k_attn_draft(AttnArgs a) {
  __shared__ float qs[kRows][kHeadDim];
  __shared__ float kb[kRows][kHeadDim];
  __shared__ float vb[kRows][kHeadDim];
  __shared__ float sc[kRows][kMaxCtx + 16];
  __shared__ float part[4][kRows][kHeadDim];
  __shared__ float rsum[kRows];
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y;
  const int* st = a.state + slot * kStateInts;
  const int t0 = st[ST_L];
  const int T = t0 + kRows;
  const int d = a.d;
  // RoPE on q (scaled by 1/8) and block k; pair (j, j+32)
  for (int t = threadIdx.x; t < kRows * 32; t += 256) {
    const int r = t >> 5, j = t & 31;
    const int pos = t0 + r;
    const float c = a.rope[(pos * 32 + j) * 2], sn = a.rope[(pos * 32 + j) * 2 + 1];
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
  const S* Kh = reinterpret_cast<const S*>(a.kcache) + ((size_t)slot * a.n_head + head) * a.n_ctx * kHeadDim;
  const S* Vh = reinterpret_cast<const S*>(a.vcache) + ((size_t)slot * a.n_head + head) * a.n_ctx * kHeadDim;
  for (int j = threadIdx.x; j < T; j += 256) {
    float kv[kHeadDim];
    if (j < t0) {
#pragma unroll
      for (int e = 0; e < kHeadDim; e += 8) ld8(Kh + (size_t)j * kHeadDim + e, kv + e);
    } else {
#pragma unroll
      for (int e = 0; e < kHeadDim; ++e) kv[e] = kb[j - t0][e];
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < kHeadDim; ++e) s = fmaf(qs[r][e], kv[e], s);
      sc[r][j] = s;
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int r = w; r < kRows; r += 4) {
    float m = -INFINITY;
    for (int j = lane; j < T; j += 64) m = fmaxf(m, sc[r][j]);
    m = wave_max(m);
    float l = 0.f;
    for (int j = lane; j < T; j += 64) {
      float e = __expf(sc[r][j] - m);
      sc[r][j] = e;
      l += e;
    }
    l = wave_sum(l);
    if (lane == 0) rsum[r] = l;
  }
  __syncthreads();
  {
    const int dim = lane;
    float acc[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) acc[r] = 0.f;
    for (int j = w; j < T; j += 4) {
      const float vv = (j < t0) ? to_f(Vh[(size_t)j * kHeadDim + dim]) : vb[j - t0][dim];
#pragma unroll
      for (int r = 0; r < kRows; ++r) acc[r] = fmaf(sc[r][j], vv, acc[r]);
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) part[w][r][dim] = acc[r];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < kRows * kHeadDim; t += 256) {
    int r = t >> 6, j = t & 63;
    float o = (part[0][r][j] + part[1][r][j]) + (part[2][r][j] + part[3][r][j]);
    a.out[(size_t)(slot * kRows + r) * d + head * kHeadDim + j] = o / rsum[r];
  }
}

// ---------------------------------------------------------------- cross-attention
// Nine rows of one slot against the 1500 acoustic frames of one head, split into
// chunks of kFrameSplit frames; each chunk writes (max, sum, unnormalised output)
// and k_attn_cross_comb merges the chunks in a fixed order.
template <typename S>
__global__ void __launch_bounds__(128) k_attn_cross_part(CrossArgs a) {
  __shared__ float qs[kRows][kHeadDim];
  __shared__ float sc[kRows][kFrameSplit];
  __shared__ float mx[kRows];
  __shared__ float part[2][kRows][kHeadDim];
  const int split = blockIdx.x, head = blockIdx.y, slot = a.slot0 + blockIdx.z;
  const int f0 = split * kFrameSplit;
  const int nf = min(kFrameSplit, a.n_frames - f0);
  for (int t = threadIdx.x; t < kRows * kHeadDim; t += 128) {
    int r = t >> 6, j = t & 63;
    qs[r][j] = a.q[(size_t)(slot * kRows + r) * a.ldq + head * kHeadDim + j] * 0.125f;
  }
  __syncthreads();
  const S* Kx = reinterpret_cast<const S*>(a.kv) + ((size_t)slot * 2 * a.n_head + head) * a.n_frames * kHeadDim;
  const S* Vx = Kx + (size_t)a.n_head * a.n_frames * kHeadDim;
  {
    const int f = threadIdx.x;
    if (f < nf) {
      float kv[kHeadDim];
#pragma unroll
      for (int e = 0; e < kHeadDim; e += 8) ld8(Kx + (size_t)(f0 + f) * kHeadDim + e, kv + e);
#pragma unroll
      for (int r = 0; r < kRows; ++r) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < kHeadDim; ++e) s = fmaf(qs[r][e], kv[e], s);
        sc[r][f] = s;
      }
    } else {
#pragma unroll
      for (int r = 0; r < kRows; ++r) sc[r][f] = -INFINITY;
    }
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int r = w; r < kRows; r += 2) {
    float m = fmaxf(sc[r][lane], sc[r][lane + 64]);
    m = wave_max(m);
    float e0 = (sc[r][lane] == -INFINITY) ? 0.f : __expf(sc[r][lane] - m);
    float e1 = (sc[r][lane + 64] == -INFINITY) ? 0.f : __expf(sc[r][lane + 64] - m);
    sc[r][lane] = e0;
    sc[r][lane + 64] = e1;
    float l = wave_sum(e0 + e1);
    if (lane == 0) {
      mx[r] = m;
      const size_t o = ((size_t)(slot * kRows + r) * a.n_head + head) * a.nsplit + split;
      a.pm[o] = m;
      a.pl[o] = l;
    }
  }
  __syncthreads();
  {
    const int dim = lane;
    float acc[kRows];
#pragma unroll
    for (int r = 0; r < kRows; ++r) acc[r] = 0.f;
    for (int f = w; f < nf; f += 2) {
      const float vv = to_f(Vx[(size_t)(f0 + f) * kHeadDim + dim]);
#pragma unroll
      for (int r = 0; r < kRows; ++r) acc[r] = fmaf(sc[r][f], vv, acc[r]);
    }
#pragma unroll
    for (int r = 0; r < kRows; ++r) part[w][r][dim] = acc[r];
  }
  __syncthreads();
  for (int t = threadIdx.x; t < kRows * kHeadDim; t += 128) {
    int r = t >> 6, j = t & 63;
    const size_t o = ((size_t)(slot * kRows + r) * a.n_head + head) * a.nsplit + split;
    a.po[o * kHeadDim + j] = part[0][r][j] + part[1][r][j];
  }
}

__global__ void __launch_bounds__(64) k_attn_cross_comb(CrossArgs a) {
  const int head = blockIdx.x, slot = a.slot0 + blockIdx.y, dim = threadIdx.x;
  for (int r = 0; r < kRows; ++r) {
    const size_t base = ((size_t)(slot * kRows + r) * a.n_head + head) * a.nsplit;
    float M = -INFINITY;
    for (int s = 0; s < a.nsplit; ++s) M = fmaxf(M, a.pm[base + s]);
    float L = 0.f, o = 0.f;
    for (int s = 0; s < a.nsplit; ++s) {
      const float c = __expf(a.pm[base + s] - M);
      L = fmaf(a.pl[base + s], c, L);
      o = fmaf(a.po[(base + s) * kHeadDim + dim], c, o);
    }
    a.out[(size_t)(slot * kRows + r) * a.d + head * kHeadDim + dim] = o / L;
  }
}

// ---------------------------------------------------------------- pass set-up
// Verify rows: [anchor, c_1..c_k] at positions L..L+k with the budget rule
// k = min(K, k_max, max_new - emitted - 1, n_ctx - L - 1) (Appendix A.1).
template <typename S>
__global__ void __launch_bounds__(256) k_verify_begin(BeginArgs a) {
  __shared__ int toks[kRows];
  __shared__ int pos0s, nvs;
  const int slot = a.slot0 + blockIdx.x;
  int* st = a.state + slot * kStateInts;
  if (threadIdx.x == 0) {
    const int L = st[ST_L], left = st[ST_MAX_NEW] - st[ST_EMITTED];
    int nv = 0;
    if (st[ST_LIVE] && !st[ST_DONE] && left > 0 && L < a.n_ctx) {
      int k = min(min(a.block_k, a.k_max), min(left - 1, a.n_ctx - L - 1));
      nv = k + 1;
    }
    st[ST_POS0] = L;
    st[ST_NV] = nv;
    pos0s = L;
    nvs = nv;
    const int anchor = st[ST_ANCHOR];
    for (int i = 0; i < kRows; ++i) {
      int t = (i == 0 || i >= nv) ? anchor : a.draft[(size_t)blockIdx.x * a.block_k + i - 1];
      t = min(max(t, 0), a.n_vocab - 1);
      toks[i] = t;
      a.tok[slot * kRows + i] = t;
    }
  }
  __syncthreads();
  const S* E = reinterpret_cast<const S*>(a.emb);
  const S* P = reinterpret_cast<const S*>(a.pos);
  for (int i = 0; i < kRows; ++i) {
    const int p = min(pos0s + i, a.n_ctx - 1);
    float* hr = a.h + (size_t)(slot * kRows + i) * a.d;
    for (int c = threadIdx.x; c < a.d; c += 256) hr[c] = to_f(E[(size_t)toks[i] * a.d + c]) + to_f(P[(size_t)p * a.d + c]);
  }
}

// Draft block X_t = [Emb(y_t), m, ..., m] (Eq. 2).
template <typename S>
__global__ void __launch_bounds__(256) k_draft_begin(BeginArgs a) {
  const int slot = a.slot0 + blockIdx.x;
  const int* st = a.state + slot * kStateInts;
  const int anchor = min(max(st[ST_ANCHOR], 0), a.n_vocab - 1);
  const S* E = reinterpret_cast<const S*>(a.emb);
  const S* m = reinterpret_cast<const S*>(a.pos);
  for (int i = 0; i < kRows; ++i) {
    float* hr = a.h + (size_t)(slot * kRows + i) * a.d;
    for (int c = threadIdx.x; c < a.d; c += 256)
      hr[c] = (i == 0) ? to_f(E[(size_t)anchor * a.d + c]) : to_f(m[c]);
  }
}

// Prefill chunk c: prompt positions 9c..9c+8 of each slot.
template <typename S>
__global__ void __launch_bounds__(256) k_prefill_begin(BeginArgs a) {
  __shared__ int toks[kRows];
  __shared__ int pos0s;
  const int slot = a.slot0 + blockIdx.x;
  int* st = a.state + slot * kStateInts;
  if (threadIdx.x == 0) {
    const int len = st[ST_LEN];
    const int pos0 = a.chunk * kRows;
    const int nv = max(0, min(kRows, len - pos0));
    st[ST_POS0] = pos0;
    st[ST_NV] = nv;
    st[ST_HPOS] = pos0;
    st[ST_HN] = nv;
    pos0s = pos0;
    for (int i = 0; i < kRows; ++i) {
      int t = (i < nv) ? a.draft[(size_t)blockIdx.x * a.pmax + pos0 + i] : 0;
      t = min(max(t, 0), a.n_vocab - 1);
      toks[i] = t;
      a.tok[slot * kRows + i] = t;
    }
  }
  __syncthreads();
  const S* E = reinterpret_cast<const S*>(a.emb);
  const S* P = reinterpret_cast<const S*>(a.pos);
  for (int i = 0; i < kRows; ++i) {
    const int p = min(pos0s + i, a.n_ctx - 1);
    float* hr = a.h + (size_t)(slot * kRows + i) * a.d;
    for (int c = threadIdx.x; c < a.d; c += 256) hr[c] = to_f(E[(size_t)toks[i] * a.d + c]) + to_f(P[(size_t)p * a.d + c]);
  }
}

// keep the final hidden row of each slot's last prompt position (row 0 of lasth)
__global__ void __launch_bounds__(256) k_save_last(const float* __restrict__ h, float* __restrict__ lasth,
                                                   const int* __restrict__ state, int slot0, int d, int chunk) {
  const int slot = slot0 + blockIdx.x;
  const int len = state[slot * kStateInts + ST_LEN];
  const int last = len - 1;
  if (last / kRows != chunk) return;
  const int r = last % kRows;
  for (int c = threadIdx.x; c < d; c += 256)
    lasth[(size_t)slot * kRows * d + c] = h[(size_t)(slot * kRows + r) * d + c];
}

// first anchor from the argmax of the last prompt row
__global__ void k_prefill_finish(int* __restrict__ state, const int* __restrict__ g, int slot0, int n, int eos,
                                 int n_ctx, int* __restrict__ first) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n) return;
  const int slot = slot0 + s;
  int* st = state + slot * kStateInts;
  const int tok = g[slot * kRows];
  st[ST_ANCHOR] = tok;
  st[ST_L] = st[ST_LEN];
  st[ST_EMITTED] = 1;
  st[ST_STEP] = 0;
  st[ST_HN] = 0;
  st[ST_DONE] = (tok == eos) || st[ST_MAX_NEW] <= 1 || st[ST_LEN] >= n_ctx;
  st[ST_LIVE] = 1;
  if (first) first[s] = tok;
}

// ---------------------------------------------------------------- history update
// Write the drafter history of pending rows: k gets RoPE at its own position, both
// k and v are rounded to the storage type (Appendix A.2).
template <typename S>
__global__ void __launch_bounds__(256) k_hist_write(HistArgs a) {
  const int slot = a.slot0 + blockIdx.y, r = blockIdx.x;
  const int* st = a.state + slot * kStateInts;
  const int hn = st[ST_HN], pos = st[ST_HPOS] + r;
  if (r >= hn || pos >= a.n_ctx) return;
  const float* kr = a.kv + (size_t)(slot * kRows + r) * 2 * a.d;
  const float* vr = kr + a.d;
  S* Kh = reinterpret_cast<S*>(a.kcache);
  S* Vh = reinterpret_cast<S*>(a.vcache);
  for (int t = threadIdx.x; t < a.n_head * 32; t += 256) {
    const int head = t >> 5, j = t & 31;
    const float c = a.rope[(pos * 32 + j) * 2], sn = a.rope[(pos * 32 + j) * 2 + 1];
    const float k1 = kr[head * kHeadDim + j], k2 = kr[head * kHeadDim + j + 32];
    const size_t base = (((size_t)slot * a.n_head + head) * a.n_ctx + pos) * kHeadDim;
    Kh[base + j] = from_f<S>(k1 * c - k2 * sn);
    Kh[base + j + 32] = from_f<S>(k1 * sn + k2 * c);
    Vh[base + j] = from_f<S>(vr[head * kHeadDim + j]);
    Vh[base + j + 32] = from_f<S>(vr[head * kHeadDim + j + 32]);
  }
}

__global__ void k_hist_done(int* state, int slot0, int n) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s < n) state[(slot0 + s) * kStateInts + ST_HN] = 0;
}

// ---------------------------------------------------------------- acceptance
// Greedy longest-prefix rule (Section 3.1) with the end-of-transcript rule and
// the cache/anchor update of Appendix A.1.  One thread per slot.
__global__ void k_accept_greedy(AcceptArgs a) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= a.n) return;
  const int slot = a.slot0 + s;
  int* st = a.state + slot * kStateInts;
  const int nv = st[ST_NV];
  const int K = a.block_k;
  int* out = a.out ? a.out + (size_t)s * (K + 1) : nullptr;
  if (nv == 0) {
    if (a.n_out) a.n_out[s] = 0;
    if (a.n_acc) a.n_acc[s] = 0;
    if (a.done) a.done[s] = st[ST_LIVE] ? 1 : 0;
    if (st[ST_LIVE]) st[ST_DONE] = 1;
    return;
  }
  const int k = nv - 1;
  const int* tok = a.tok + slot * kRows;
  const int* g = a.g + slot * kRows;
  int acc = 0;
  while (acc < k && tok[acc + 1] == g[acc]) ++acc;
  int nemit = 0;
  bool fin = false;
  for (int e = 0; e < acc; ++e) {
    const int c = tok[e + 1];
    if (out) out[nemit] = c;
    ++nemit;
    if (c == a.eos) { fin = true; break; }
  }
  int last;
  if (!fin) {
    last = g[acc];
    if (out) out[nemit] = last;
    ++nemit;
    fin = (last == a.eos);
  } else {
    last = tok[nemit];
    acc = nemit;
  }
  const int L = st[ST_L];
  st[ST_HPOS] = L;
  st[ST_HN] = nv;
  st[ST_L] = L + 1 + acc;
  st[ST_ANCHOR] = last;
  st[ST_EMITTED] += nemit;
  st[ST_STEP] += 1;
  st[ST_K] = k;
  st[ST_A] = acc;
  const bool done = fin || st[ST_EMITTED] >= st[ST_MAX_NEW] || st[ST_L] >= a.n_ctx;
  st[ST_DONE] = done;
  if (out)
    for (int j = nemit; j <= K; ++j) out[j] = -1;
  if (a.n_out) a.n_out[s] = nemit;
  if (a.n_acc) a.n_acc[s] = acc;
  if (a.done) a.done[s] = done;
}

// drafted tokens = argmax of mask rows 1..K
__global__ void k_draft_tokens(const int* __restrict__ g, int* __restrict__ dst, int* __restrict__ keep, int slot0,
                               int n, int K) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= n * K) return;
  const int s = t / K, j = t % K;
  const int v = g[(slot0 + s) * kRows + 1 + j];
  if (dst) dst[t] = v;
  keep[(size_t)(slot0 + s) * K + j] = v;
}

// ---------------------------------------------------------------- encode: cross K/V
// C[f, n] = sum_k A[f, k] W[n, k] + b[n] for the 2d key/value columns of one
// block, written to the per-head frame-major cross cache.  64x64 tiles, fp32
// accumulation.
template <typename S>
__global__ void __launch_bounds__(256) k_gemm_xkv(XkvArgs a) {
  __shared__ float As[16][64 + 4];
  __shared__ float Bs[16][64 + 4];
  const S* A = reinterpret_cast<const S*>(a.mem);
  const S* W = reinterpret_cast<const S*>(a.w);
  const S* bias = reinterpret_cast<const S*>(a.bias);
  const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  const int K = a.d, M = a.n_frames, N = 2 * a.d;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int t = threadIdx.x; t < 64 * 16; t += 256) {
      const int mm = t >> 4, kk = t & 15;
      As[kk][mm] = (m0 + mm < M) ? to_f(A[(size_t)(m0 + mm) * K + k0 + kk]) : 0.f;
      Bs[kk][mm] = to_f(W[(size_t)(n0 + mm) * K + k0 + kk]);
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = As[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) bv[j] = Bs[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
  S* out = reinterpret_cast<S*>(a.out);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int f = m0 + ty * 4 + i;
    if (f >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = n0 + tx * 4 + j;
      const int kv = n >= a.d, col = n - kv * a.d, head = col >> 6, dim = col & 63;
      const float v = acc[i][j] + to_f(bias[n]);
      out[(((size_t)kv * a.n_head + head) * M + f) * kHeadDim + dim] = from_f<S>(v);
    }
  }
}

// ---------------------------------------------------------------- launchers
template <typename S>
void Ops<S>::layernorm(const float* x, const void* g, const void* b, float* y, int d, int row0, int rows,
                       hipStream_t st) {
  k_layernorm<S><<<rows, 256, 0, st>>>(x, (const S*)g, (const S*)b, y, d, row0);
}
template <typename S>
void Ops<S>::gemv(int epi, const GemvArgs& a, hipStream_t st) {
  const int grid = (a.N + 15) / 16;
  switch (epi) {
    case EPI_STORE: k_gemv<S, EPI_STORE><<<grid, 256, 0, st>>>(a); break;
    case EPI_GELU: k_gemv<S, EPI_GELU><<<grid, 256, 0, st>>>(a); break;
    case EPI_RESID: k_gemv<S, EPI_RESID><<<grid, 256, 0, st>>>(a); break;
    case EPI_QKV: k_gemv<S, EPI_QKV><<<grid, 256, 0, st>>>(a); break;
    case EPI_ARGMAX: k_gemv<S, EPI_ARGMAX><<<grid, 256, 0, st>>>(a); break;
  }
}
template <typename S>
void Ops<S>::attn_self(const AttnArgs& a, int n, hipStream_t st) {
  k_attn_self<S><<<dim3(a.n_head, n), 256, 0, st>>>(a);
}
template <typename S>
void Ops<S>::attn_draft(const AttnArgs& a, int n, hipStream_t st) {
  k_attn_draft<S><<<dim3(a.n_head, n), 256, 0, st>>>(a);
}
template <typename S>
void Ops<S>::attn_cross(const CrossArgs& a, int n, hipStream_t st) {
  k_attn_cross_part<S><<<dim3(a.nsplit, a.n_head, n), 128, 0, st>>>(a);
  k_attn_cross_comb<<<dim3(a.n_head, n), 64, 0, st>>>(a);
}
template <typename S>
void Ops<S>::verify_begin(const BeginArgs& a, int n, hipStream_t st) { k_verify_begin<S><<<n, 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::draft_begin(const BeginArgs& a, int n, hipStream_t st) { k_draft_begin<S><<<n, 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::prefill_begin(const BeginArgs& a, int n, hipStream_t st) { k_prefill_begin<S><<<n, 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::hist_write(const HistArgs& a, int n, hipStream_t st) { k_hist_write<S><<<dim3(kRows, n), 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::gemm_xkv(const XkvArgs& a, hipStream_t st) {
  k_gemm_xkv<S><<<dim3((a.n_frames + 63) / 64, 2 * a.d / 64), 256, 0, st>>>(a);
}

void argmax_final(const float* hv, const int* hi, int nblk, int row0, int rows, int* g, float* gmax,
                  unsigned* status, hipStream_t st) {
  k_argmax_final<<<rows, 256, 0, st>>>(hv, hi, nblk, row0, g, gmax, status);
}
void save_last(const float* h, float* lasth, const int* state, int slot0, int n, int d, int chunk, hipStream_t st) {
  k_save_last<<<n, 256, 0, st>>>(h, lasth, state, slot0, d, chunk);
}
void prefill_finish(int* state, const int* g, int slot0, int n, int eos, int n_ctx, int* first, hipStream_t st) {
  k_prefill_finish<<<(n + 63) / 64, 64, 0, st>>>(state, g, slot0, n, eos, n_ctx, first);
}
void hist_done(int* state, int slot0, int n, hipStream_t st) { k_hist_done<<<(n + 63) / 64, 64, 0, st>>>(state, slot0, n); }
void accept_greedy(const AcceptArgs& a, hipStream_t st) { k_accept_greedy<<<(a.n + 63) / 64, 64, 0, st>>>(a); }
void draft_tokens(const int* g, int* dst, int* keep, int slot0, int n, int K, hipStream_t st) {
  k_draft_tokens<<<(n * K + 255) / 256, 256, 0, st>>>(g, dst, keep, slot0, n, K);
}

template struct Ops<float>;
template struct Ops<bf16>;

}  // namespace wf
