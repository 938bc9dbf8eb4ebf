// Kernels of the Whisper audio encoder (the acoustic memory the drafter and the
// target cross-attend to, Section 3.2) besides its matrix products, which run on
// k_mm: the log-mel frontend, the convolution stem's row gathering, row-wise
// LayerNorm and the fused self-attention.
#include <float.h>

#include "wf_common.h"
#include "wf_kernels.h"
#include "wf_operand.h"

namespace wf {

namespace {

// order-preserving map of fp32 values to signed ints (max over floats = max over keys)
__device__ __forceinline__ int f2key(float f) {
  const int b = __float_as_int(f);
  return b >= 0 ? b : b ^ 0x7fffffff;
}
__device__ __forceinline__ float key2f(int k) { return __int_as_float(k >= 0 ? k : k ^ 0x7fffffff); }

__device__ __forceinline__ float block_max(float v, float* red) {
  for (int o = 32; o; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = red[0];
  for (int i = 1; i < nw; ++i) r = fmaxf(r, red[i]);
  return r;
}

}  // namespace

// One block per frame f of one request: the frame's n_fft samples (reflect-padded
// signal, periodic Hann window), their power spectrum by a direct DFT in fp64,
// the mel filterbank (each filter summed over its nonzero bins) and log10 of
// max(mel, 1e-10), written to logmel[f][m]; the request's maximum goes to *gmax
// as an order-preserving int.
__global__ void __launch_bounds__(256) k_logmel(LogmelArgs a) {
  __shared__ double xw[kMaxFft];
  __shared__ double tw[2 * kMaxFft];
  __shared__ double pw[kMaxFft / 2 + 1];
  __shared__ float red[4];
  const int f = blockIdx.x, N = a.n_fft, nb = N / 2 + 1;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    int s = f * a.hop - N / 2 + i;
    s = s < 0 ? -s : s;
    s = s >= a.n_samples ? 2 * (a.n_samples - 1) - s : s;
    xw[i] = (double)a.audio[s] * a.window[i];
    tw[2 * i] = a.twiddle[2 * i];
    tw[2 * i + 1] = a.twiddle[2 * i + 1];
  }
  __syncthreads();
  for (int k = threadIdx.x; k < nb; k += blockDim.x) {
    double re = 0.0, im = 0.0;
    int idx = 0;
    for (int i = 0; i < N; ++i) {  // exp(-2 pi i k i / N): index (k i) mod N of the table
      re = fma(xw[i], tw[2 * idx], re);
      im = fma(xw[i], tw[2 * idx + 1], im);
      idx += k;
      if (idx >= N) idx -= N;
    }
    pw[k] = re * re + im * im;
  }
  __syncthreads();
  float mx = -FLT_MAX;
  for (int m = threadIdx.x; m < a.n_mels; m += blockDim.x) {
    const int lo = a.fband[2 * m], hi = a.fband[2 * m + 1];
    double s = 0.0;
    for (int k = lo; k < hi; ++k) s = fma(a.filters[(size_t)m * nb + k], pw[k], s);
    const float lg = (float)log10(fmax(s, 1e-10));
    a.logmel[(size_t)f * a.n_mels + m] = lg;
    mx = fmaxf(mx, lg);
  }
  mx = block_max(mx, red);
  if (threadIdx.x == 0) atomicMax(a.gmax, f2key(mx));
}

// the request's maximum starts below every value
__global__ void k_logmel_init(int* gmax) {
  if (threadIdx.x == 0) *gmax = f2key(-FLT_MAX);
}

// Clamp and scale the log-mel values ((max(x, max - 8) + 4) / 4) and gather the
// first convolution's rows: A[t][c * 3 + j] = x[t + j - 1][c] (zero outside the
// frames and in the padding columns up to ld), bf16.  Optionally the scaled
// features [n_mels][frames] fp32 for inspection.
__global__ void __launch_bounds__(256) k_logmel_rows(LogmelArgs a) {
  const float top = key2f(*a.gmax) - 8.f;
  const size_t total = (size_t)a.n_frames * a.ld1;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(e / a.ld1), k = (int)(e % a.ld1);
    float v = 0.f;
    if (k < 3 * a.n_mels) {
      const int c = k / 3, j = k - 3 * c, src = t + j - 1;
      if (src >= 0 && src < a.n_frames) v = (fmaxf(a.logmel[(size_t)src * a.n_mels + c], top) + 4.f) * 0.25f;
    }
    a.rows[e] = from_f<bf16>(v);
    if (a.mel_out && k < a.n_mels)
      a.mel_out[(size_t)k * a.n_frames + t] = (fmaxf(a.logmel[(size_t)t * a.n_mels + k], top) + 4.f) * 0.25f;
  }
}

// Rows of the strided second convolution: A[t][c * 3 + j] = z[2 t + j - 1][c]
// (zero outside), t < n_out, from z [n_in][d] bf16.
__global__ void __launch_bounds__(256) k_conv_rows_s2(const bf16* __restrict__ z, bf16* __restrict__ out, int n_in,
                                                      int n_out, int d) {
  const size_t total = (size_t)n_out * d;
  for (size_t e = (size_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (size_t)gridDim.x * blockDim.x) {
    const int t = (int)(e / d), c = (int)(e % d);
    bf16* o = out + (size_t)t * 3 * d + 3 * c;
#pragma unroll
    for (int j = 0; j < 3; ++j) {
      const int src = 2 * t + j - 1;
      bf16 v;
      v.u = 0;
      if (src >= 0 && src < n_in) v = z[(size_t)src * d + c];
      o[j] = v;
    }
  }
}

// LayerNorm of fp32 rows [rows][d] into bf16 rows [rows][ldo] (one wave per row,
// biased variance, eps 1e-5, two passes over the row held in registers; d a
// multiple of 4, each lane loading 16-byte runs of four columns).
__global__ void __launch_bounds__(256) k_ln_rows(const float* __restrict__ x, const bf16* __restrict__ g,
                                                 const bf16* __restrict__ b, bf16* __restrict__ out, int rows, int d,
                                                 long long ldo) {
  constexpr int kMax = kMaxEncD / 256;  // float4 runs per lane
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float4* xr = reinterpret_cast<const float4*>(x + (size_t)row * d);
  const int n4 = d >> 2;
  float4 v[kMax];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    v[i] = c < n4 ? xr[c] : make_float4(0.f, 0.f, 0.f, 0.f);
    s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  for (int o = 32; o; o >>= 1) s += __shfl_xor(s, o, 64);
  const float mean = s / d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    if (lane + 64 * i < n4) {
      const float a0 = v[i].x - mean, a1 = v[i].y - mean, a2 = v[i].z - mean, a3 = v[i].w - mean;
      q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
    }
  }
  for (int o = 32; o; o >>= 1) q += __shfl_xor(q, o, 64);
  const float r = 1.f / sqrtf(q / d + 1e-5f);
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    if (c < n4) {
      const int col = 4 * c;
      const float o0 = (v[i].x - mean) * r * to_f(g[col]) + to_f(b[col]);
      const float o1 = (v[i].y - mean) * r * to_f(g[col + 1]) + to_f(b[col + 1]);
      const float o2 = (v[i].z - mean) * r * to_f(g[col + 2]) + to_f(b[col + 2]);
      const float o3 = (v[i].w - mean) * r * to_f(g[col + 3]) + to_f(b[col + 3]);
      uint2 pk;
      pk.x = bf16_bits_rne(o0) | (bf16_bits_rne(o1) << 16);
      pk.y = bf16_bits_rne(o2) | (bf16_bits_rne(o3) << 16);
      *reinterpret_cast<uint2*>(out + (size_t)row * ldo + col) = pk;
    }
  }
}

// Bidirectional self-attention of one head over all positions, fused: one block
// per (128 queries, head), four waves of 32 queries.  Keys and transposed values
// stream through four LDS stages in tiles of 64 keys, copied straight from memory
// (global_load_lds_dwordx4) three tiles ahead of their use.  Two passes over the
// keys: the first keeps a running maximum and rescaled sum of exp per (lane,
// row), combined across lanes at its end into the row maximum M and sum L; the
// second forms p = exp(s - M) / L, rounds it to bf16 (the product's input, as an
// unfused softmax would store it) and accumulates O += p V on the matrix cores.
// Scores s = q.k / 8 from bf16 q, k (v_mfma_f32_32x32x16_bf16, fp32
// accumulation); the probability tile goes through per-wave LDS to become the
// next product's A operand.
namespace {
typedef __attribute__((address_space(3))) void lds_void;
constexpr int kAq = 128, kAk = 64, kAThreads = 256;
constexpr int kPld = kAk + 8;  // row stride of a wave's probability tile (bf16)
// stage layout (16-byte chunks): keys [key * 8 + chunk ^ (key & 7)] then
// transposed values [512 + dim * 8 + chunk ^ (dim & 7)]
constexpr int kStageChunks = 1024;
constexpr int kWaitK = (4 & 15) | (7 << 4) | (0 << 8);  // vmcnt <= 4: two later tiles' key copies
constexpr int kWaitKV = (8 & 15) | (7 << 4) | (0 << 8); // vmcnt <= 8: two later tiles' key + value copies
constexpr int kWaitAll = (0 & 15) | (7 << 4) | (15 << 8);
}  // namespace
__shared__ uint4 g_att0[kStageChunks], g_att1[kStageChunks], g_att2[kStageChunks], g_att3[kStageChunks];
__shared__ bf16 g_attp[4][32 * kPld];

// copies of key tile kt (its index clamped to the last tile) into a stage: wave w
// fills chunks (w * 2 + j) * 64 + lane of the keys (and, with values, 512 + ...)
template <bool V>
__device__ __forceinline__ void attn_copy(const EncAttnArgs& a, int head, int kt, int ntile, uint4* stage) {
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, k0 = min(kt, ntile - 1) * kAk;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int slot = (w * 2 + j) * 64 + lane, r = slot >> 3, ch = (slot & 7) ^ (r & 7);
    const bf16* src = a.qk + (size_t)min(k0 + r, a.n - 1) * a.ldqk + a.d + head * kHeadDim + 8 * ch;
    __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)&stage[(w * 2 + j) * 64], 16, 0, 0);
  }
  if (V) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int slot = (w * 2 + j) * 64 + lane, r = slot >> 3, ch = (slot & 7) ^ (r & 7);
      const bf16* src = a.vt + ((size_t)head * kHeadDim + r) * a.Tp + k0 + 8 * ch;
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)&stage[512 + (w * 2 + j) * 64], 16, 0, 0);
    }
  }
}

// scores of this wave's 32 queries against the tile's 64 keys (two 32-key halves)
__device__ __forceinline__ void attn_scores(const uint4* stage, const bf16x8* qf, floatx16* acc, int lr, int lk) {
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[kb][v] = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int row = kb * 32 + lr;
      const bf16x8 kf = __builtin_bit_cast(bf16x8, stage[row * 8 + ((2 * s + lk) ^ (row & 7))]);
      acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(qf[s], kf, acc[kb], 0, 0, 0);
    }
  }
}

__global__ void __launch_bounds__(kAThreads) k_enc_attn(EncAttnArgs a) {
  const int head = blockIdx.y, q0 = blockIdx.x * kAq;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 31, lk = lane >> 5;
  const int ntile = (a.n + kAk - 1) / kAk;
  bf16x8 qf[4];
  {
    const int qrow = min(q0 + w * 32 + lr, a.n - 1);
    const bf16* qp = a.qk + (size_t)qrow * a.ldqk + head * kHeadDim + 8 * lk;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = *reinterpret_cast<const bf16x8*>(qp + 16 * s);
  }
  floatx16 acc[2];

  // pass 1: running maximum and sum of exp per (lane, row)
  float m[16], l[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    m[v] = -FLT_MAX;
    l[v] = 0.f;
  }
  auto step1 = [&](int kt, const uint4* cur, uint4* nxt) {
    __builtin_amdgcn_s_waitcnt(kWaitK);
    __builtin_amdgcn_s_barrier();
    attn_copy<false>(a, head, kt + 3, ntile, nxt);  // every step issues its copies: exact wait counts
    if (kt < ntile) {
      attn_scores(cur, qf, acc, lr, lk);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bool ok = kt * kAk + kb * 32 + lr < a.n;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float sv = acc[kb][v] * 0.125f;
          const float mn = ok ? fmaxf(m[v], sv) : m[v];
          l[v] = ok ? l[v] * __expf(m[v] - mn) + __expf(sv - mn) : l[v];
          m[v] = mn;
        }
      }
    }
  };
  attn_copy<false>(a, head, 0, ntile, g_att0);
  attn_copy<false>(a, head, 1, ntile, g_att1);
  attn_copy<false>(a, head, 2, ntile, g_att2);
  for (int kt = 0; kt < ntile; kt += 4) {
    step1(kt, g_att0, g_att3);
    step1(kt + 1, g_att1, g_att0);
    step1(kt + 2, g_att2, g_att1);
    step1(kt + 3, g_att3, g_att2);
  }
  __builtin_amdgcn_s_waitcnt(kWaitAll);  // the surplus copies have landed before the stages are refilled
  // combine over the 32 lanes holding a row's columns (same half of the wave)
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    float mx = m[v];
    for (int o = 1; o < 32; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    float sm = l[v] * __expf(m[v] - mx);
    for (int o = 1; o < 32; o <<= 1) sm += __shfl_xor(sm, o, 64);
    m[v] = mx;
    l[v] = 1.f / sm;
  }
  __syncthreads();

  // pass 2: p = exp(s - M) / L in bf16, O += p V
  floatx16 o[2];
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[nt][v] = 0.f;
  bf16* pw = g_attp[w];
  auto step2 = [&](int kt, const uint4* cur, uint4* nxt) {
    __builtin_amdgcn_s_waitcnt(kWaitKV);
    __builtin_amdgcn_s_barrier();
    attn_copy<true>(a, head, kt + 3, ntile, nxt);
    if (kt < ntile) {
      attn_scores(cur, qf, acc, lr, lk);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const bool ok = kt * kAk + kb * 32 + lr < a.n;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float pv = ok ? __expf(acc[kb][v] * 0.125f - m[v]) * l[v] : 0.f;
          const int row = 8 * (v >> 2) + 4 * lk + (v & 3);
          pw[row * kPld + kb * 32 + lr] = from_f<bf16>(pv);
        }
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const bf16x8 pf = *reinterpret_cast<const bf16x8*>(pw + lr * kPld + 16 * s + 8 * lk);
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
          const int row = nt * 32 + lr;
          const bf16x8 vf = __builtin_bit_cast(bf16x8, cur[512 + row * 8 + ((2 * s + lk) ^ (row & 7))]);
          o[nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf, vf, o[nt], 0, 0, 0);
        }
      }
    }
  };
  attn_copy<true>(a, head, 0, ntile, g_att0);
  attn_copy<true>(a, head, 1, ntile, g_att1);
  attn_copy<true>(a, head, 2, ntile, g_att2);
  for (int kt = 0; kt < ntile; kt += 4) {
    step2(kt, g_att0, g_att3);
    step2(kt + 1, g_att1, g_att0);
    step2(kt + 2, g_att2, g_att1);
    step2(kt + 3, g_att3, g_att2);
  }
  __builtin_amdgcn_s_waitcnt(kWaitAll);  // no copy may land in LDS after the block has left
  // O rows: query 8 (v / 4) + 4 lk + v % 4 of the wave, dim nt * 32 + lr
#pragma unroll
  for (int nt = 0; nt < 2; ++nt)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int q = q0 + w * 32 + 8 * (v >> 2) + 4 * lk + (v & 3);
      if (q < a.n) a.o[(size_t)q * a.ldo + head * kHeadDim + nt * 32 + lr] = from_f<bf16>(o[nt][v]);
    }
}

void enc_attention(const EncAttnArgs& a, int n_head, hipStream_t st) {
  k_enc_attn<<<dim3((a.n + kAq - 1) / kAq, n_head), kAThreads, 0, st>>>(a);
}

void logmel(const LogmelArgs& a, hipStream_t st) {
  k_logmel_init<<<1, 64, 0, st>>>(a.gmax);
  k_logmel<<<a.n_frames, 256, 0, st>>>(a);
  const size_t total = (size_t)a.n_frames * a.ld1;
  k_logmel_rows<<<(unsigned)std::min<size_t>((total + 255) / 256, 4096), 256, 0, st>>>(a);
}
void conv_rows_s2(const bf16* z, bf16* out, int n_in, int n_out, int d, hipStream_t st) {
  const size_t total = (size_t)n_out * d;
  k_conv_rows_s2<<<(unsigned)std::min<size_t>((total + 255) / 256, 4096), 256, 0, st>>>(z, out, n_in, n_out, d);
}
void ln_rows(const float* x, const bf16* g, const bf16* b, bf16* out, int rows, int d, long long ldo, hipStream_t st) {
  k_ln_rows<<<(rows + 3) / 4, 256, 0, st>>>(x, g, b, out, rows, d, ldo);
}

}  // namespace wf
