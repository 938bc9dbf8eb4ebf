// Kernels of the Whisper audio encoder (the acoustic memory the drafter and the
// target cross-attend to, Section 3.2) besides its matrix products, which run on
// k_mm: the log-mel frontend, the convolution stem's row gathering, row-wise
// LayerNorm and the attention softmax.
#include <float.h>

#include "wf_common.h"
#include "wf_kernels.h"

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
__device__ __forceinline__ float block_sum(float v, float* red) {
  for (int o = 32; o; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  float r = 0.f;
  for (int i = 0; i < nw; ++i) r += red[i];
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
// biased variance, eps 1e-5, two passes over the row held in registers).
__global__ void __launch_bounds__(256) k_ln_rows(const float* __restrict__ x, const bf16* __restrict__ g,
                                                 const bf16* __restrict__ b, bf16* __restrict__ out, int rows, int d,
                                                 long long ldo) {
  constexpr int kMax = kMaxEncD / 64;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  const float* xr = x + (size_t)row * d;
  float v[kMax];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    v[i] = c < d ? xr[c] : 0.f;
    s += v[i];
  }
  for (int o = 32; o; o >>= 1) s += __shfl_xor(s, o, 64);
  const float mean = s / d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    const float dv = c < d ? v[i] - mean : 0.f;
    q += dv * dv;
  }
  for (int o = 32; o; o >>= 1) q += __shfl_xor(q, o, 64);
  const float r = 1.f / sqrtf(q / d + 1e-5f);
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = lane + 64 * i;
    if (c < d) out[(size_t)row * ldo + c] = from_f<bf16>((v[i] - mean) * r * to_f(g[c]) + to_f(b[c]));
  }
}

// Softmax of score rows [rows][ld] over their first n columns into bf16
// probabilities (columns n..ld-1 written as zeros); one block per row.
__global__ void __launch_bounds__(256) k_softmax_rows(const float* __restrict__ s, bf16* __restrict__ p, int n,
                                                      int ld) {
  __shared__ float red[4];
  constexpr int kMax = kMaxEncCtx / 256;
  const float* sr = s + (size_t)blockIdx.x * ld;
  bf16* pr = p + (size_t)blockIdx.x * ld;
  float v[kMax];
  float m = -FLT_MAX;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = threadIdx.x + 256 * i;
    v[i] = c < n ? sr[c] : -FLT_MAX;
    m = fmaxf(m, v[i]);
  }
  m = block_max(m, red);
  float sum = 0.f;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = threadIdx.x + 256 * i;
    v[i] = c < n ? expf(v[i] - m) : 0.f;
    sum += v[i];
  }
  sum = block_sum(sum, red);
  const float inv = 1.f / sum;
#pragma unroll
  for (int i = 0; i < kMax; ++i) {
    const int c = threadIdx.x + 256 * i;
    if (c < ld) pr[c] = from_f<bf16>(v[i] * inv);
  }
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
void softmax_rows(const float* s, bf16* p, int rows, int n, int ld, hipStream_t st) {
  k_softmax_rows<<<rows, 256, 0, st>>>(s, p, n, ld);
}

}  // namespace wf
