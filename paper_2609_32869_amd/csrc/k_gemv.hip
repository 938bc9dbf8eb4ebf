// Weight-streaming matrix products Y = X W^T for the 9 rows of each slot
// (gfx950).  Every parameter byte is read once per pass; the activation operand
// is tiny and stays in L2.
//
// bf16 storage: weights and operands are stored in matrix-core fragment order
// (wf_common.h) so every wave load is 1 KB of contiguous memory.  Two shapes:
//  * 16-column tiles, v_mfma_f32_16x16x32_bf16, two 16-row operand tiles per pass
//    (narrow matrices: more tiles, more blocks);
//  * 32-column tiles, v_mfma_f32_32x32x16_bf16, one 32-row operand tile per pass
//    (wide matrices: half the operand traffic per weight byte).
// A block streams one column tile; its waves split the k-steps and issue the loads
// of up to U steps before the first matrix instruction that consumes them; the
// wave partials are summed in LDS in a fixed order.
//
// fp32 storage (the small correctness configuration): row-major weights and
// operand, v_mfma_f32_16x16x4f32.
#include "../../include/wf.h"
#include "wf_operand.h"

namespace wf {

constexpr int kU = 10;  // k-steps whose loads a wave issues together (16-wave blocks: 5)

// ---------------------------------------------------------------- epilogue
// Everything the batch-1 epilogue reads from memory for its tile (9 rows x TC
// columns), loaded at kernel start so the epilogue does not wait on a global
// read.  Element it of a thread is tile entry threadIdx.x + it * NT, as in the
// epilogue loop.  The loads are unconditional (indexes clamped into the buffers,
// unused values discarded; also with several slots, whose epilogue does not use
// them) so no load waits for another and no branch joins a loaded value.
template <int TC, int NT, bool LN = false>
struct EpiPre {
  static constexpr int P = (kRows * TC + NT - 1) / NT;
  uint32_t bb[P];    // bf16 bias bits (converted when used, so nothing waits here)
  float r[P];
  float lc[LN ? P : 1], le[LN ? P : 1];  // LN folded in: the column sums c and e
  uint8_t sup[P];    // ARGMAX: suppressed
  int s0, s1, s2, s3;  // QKV: valid rows, first position, its page, the next page; ARGMAX: step

  template <typename S, int EPI>
  __device__ __forceinline__ void load(const GemvArgs& a, int nb) {
    const bool has_bias = a.bias != nullptr;  // without one, read the weights and discard
    const uint16_t* bias = reinterpret_cast<const uint16_t*>(has_bias ? a.bias : a.w);
    const int* st = a.state != nullptr ? a.state + a.slot0 * kStateInts : reinterpret_cast<const int*>(a.w);
#pragma unroll
    for (int it = 0; it < P; ++it) {
      const int idx = threadIdx.x + it * NT, ml = min(idx / TC, kRows - 1), n = min(nb + idx % TC, a.N - 1);
      bb[it] = bias[n];
      r[it] = EPI == EPI_RESID ? a.y[(size_t)(a.slot0 * kRows + ml) * a.ldy + n] : 0.f;
      if constexpr (LN) {
        lc[it] = a.lnc[n];
        le[it] = a.lne[n];
      }
      if constexpr (EPI == EPI_ARGMAX) {
        const uint8_t* sp = a.suppress != nullptr ? a.suppress : reinterpret_cast<const uint8_t*>(a.w);
        sup[it] = sp[n];
      }
    }
    if constexpr (EPI == EPI_QKV) {
      s0 = st[ST_NV];
      s1 = st[ST_POS0];
      s2 = st[ST_PG0];
      s3 = st[ST_PG1];
    } else if constexpr (EPI == EPI_ARGMAX) {
      s0 = st[a.state != nullptr ? ST_STEP : 0];
    }
  }
  __device__ __forceinline__ float bias(const GemvArgs& a, int it) const {
    return a.bias != nullptr ? __uint_as_float(bb[it] << 16) : 0.f;
  }
  // Called where the epilogue starts: returns a copy in which an empty asm
  // redefines every prefetched value, so no arithmetic on them (and no wait for
  // their loads) can be scheduled before the main loop.  The prefetched values
  // themselves stay unchanged: redefining them in place would carry them around a
  // tile loop, and the register copy at the loop entry would wait for the loads
  // before the first weight load is issued.
  __device__ __forceinline__ EpiPre arrived() const {
    EpiPre o = *this;
#pragma unroll
    for (int it = 0; it < P; ++it) {
      __asm__ volatile("" : "+v"(o.bb[it]));
      __asm__ volatile("" : "+v"(o.r[it]));
      if constexpr (LN) {
        __asm__ volatile("" : "+v"(o.lc[it]));
        __asm__ volatile("" : "+v"(o.le[it]));
      }
      uint32_t sp = o.sup[it];
      __asm__ volatile("" : "+v"(sp));
      o.sup[it] = (uint8_t)sp;
    }
    __asm__ volatile("" : "+v"(o.s0), "+v"(o.s1), "+v"(o.s2), "+v"(o.s3));
    return o;
  }
};

// Appends the k or v value v of column n (>= d) at cache page `page`, position pos.
// Keys are [page][head][16][64]; values too with fp32 storage, and transposed
// within the page, [page][head][64][16], with bf16 storage (the matrix-core
// self-attention reads 8 consecutive positions of one dim).
template <typename S>
__device__ __forceinline__ void qkv_append(const GemvArgs& a, int n, float v, int page, int pos) {
  const int d = a.d, kv = n >= 2 * d;
  const int cc = n - d - kv * d, head = cc >> 6, dim = cc & 63;
  S* cache = reinterpret_cast<S*>(a.cache) + (size_t)kv * a.kv_stride;
  const size_t ph = (size_t)page * a.n_head + head;
  const size_t i = sizeof(S) == 2 && kv ? (ph * kHeadDim + dim) * kPage + (pos & 15) : (ph * kPage + (pos & 15)) * kHeadDim + dim;
  cache[i] = from_f<S>(v);
}

// Bias and residual values of a multi-slot tile (TM rows x TC columns), loaded at
// kernel start like EpiPre so the epilogue starts without a global read.
template <int TM, int TC, int NT>
struct RowsPre {
  static constexpr int P = (TM * TC + NT - 1) / NT;
  uint32_t bb[P];  // bf16 bias bits
  float r[P];

  template <typename S, int EPI>
  __device__ __forceinline__ void load(const GemvArgs& a, int m0, int nb) {
    const bool has_bias = a.bias != nullptr;  // without one, read the weights and discard
    const uint16_t* bias = reinterpret_cast<const uint16_t*>(has_bias ? a.bias : a.w);
#pragma unroll
    for (int it = 0; it < P; ++it) {
      const int idx = threadIdx.x + it * NT;
      const int row = min(m0 + idx / TC, a.R9 - 1), n = min(nb + idx % TC, a.N - 1);
      bb[it] = bias[n];
      r[it] = EPI == EPI_RESID ? a.y[(size_t)row * a.ldy + n] : 0.f;
    }
  }
  __device__ __forceinline__ void arrive() {
#pragma unroll
    for (int it = 0; it < P; ++it) {
      __asm__ volatile("" : "+v"(bb[it]));
      __asm__ volatile("" : "+v"(r[it]));
    }
  }
};

// Output value v of (row, column n) for the store, GELU, residual and partial-sum
// epilogues; res = current residual value (EPI_RESID).  The k/v append and the
// head scores are written by the epilogue loops from prefetched values.
template <typename S, int EPI>
__device__ __forceinline__ void epi_one(const GemvArgs& a, int row, int n, float v, float res) {
  if constexpr (EPI == EPI_STORE) {
    a.y[(size_t)row * a.ldy + n] = v;
  } else if constexpr (EPI == EPI_GELU) {
    put_op<S>(a.aout, a.nsplit, a.R9, row, n, gelu_erf(v));
  } else if constexpr (EPI == EPI_RESID) {
    const float hn = res + v;
    a.y[(size_t)row * a.ldy + n] = hn;
    if (a.tap >= 0) put_op<S>(a.aout, a.nsplit, a.R9, row, a.tap * a.N + n, hn);
  } else if constexpr (EPI == EPI_PART) {
    a.y[blockIdx.y * a.pstride + (size_t)row * a.ldy + n] = v;
  } else if constexpr (EPI == EPI_ACC) {
    atomicAdd(a.y + (size_t)row * a.ldy + n, v);
  }
}

// Head score of (row, column n): the logit (greedy), or z = logit * inv_t plus the
// row's Gumbel noise when sampling; oz receives z for the softmax normaliser.
// step: the slot's step counter (read only when drawing noise; -1: read it here).
__device__ __forceinline__ void head_score(const GemvArgs& a, int row, int n, bool act, float v, float* ov, float* oz,
                                           int step = -1) {
  if (!act) {
    *ov = -INFINITY;
    *oz = -INFINITY;
    return;
  }
  if (a.inv_t > 0.f) {
    const float z = v * a.inv_t;
    *oz = z;
    if (a.rng_purpose != 0) {
      const int slot = row / kRows, pos = row - slot * kRows;
      if (step < 0) step = a.state[slot * kStateInts + ST_STEP];
      *ov = z + rng_gumbel(rng_word(a.seed, a.rng_purpose, slot, step, pos, n));
    } else {
      *ov = z;
    }
  } else {
    *ov = v;
    *oz = v;
  }
}

// sv holds the wave-summed tile: TM operand rows (split terms) x TC columns; ov and
// oz are the head's score and z buffers (EPI_ARGMAX).
// RP: rp holds the bias / residual of a multi-slot tile prefetched at kernel start
// (bf16); otherwise the epilogue loads them.
// LN: batch 1 with the LayerNorm folded in; sv holds (x*g) W^T and lnst the rows'
// means (lnst[r]) and 1/sqrt(var + eps) (lnst[9 + r]).
template <typename S, int EPI, int TM, int TC, int NT, bool RP = false, bool LN = false>
__device__ __forceinline__ void finish_tile(const GemvArgs& a, float (*sv)[TC + 1], float (*ov)[TC], float (*oz)[TC], int m0, int nb,
                            const EpiPre<TC, NT, LN>& pre, RowsPre<TM, TC, NT>& rp, const float* lnst = nullptr) {
  const bool split3 = a.nsplit == 3;
  const int R = a.slot0 * kRows, Rend = (a.slot0 + a.nslots) * kRows;
  const int nrows = split3 ? kRows : TM;
  if (split3) {
    const EpiPre<TC, NT, LN> pv = pre.arrived();
    // rows r, r + 9, r + 18 hold the three split terms of row r
#pragma unroll
    for (int it = 0; it < EpiPre<TC, NT>::P; ++it) {
      const int idx = threadIdx.x + it * NT;
      if (idx >= kRows * TC) break;
      const int ml = idx / TC, c = idx % TC, n = nb + c, row = R + ml;
      const bool act = n < a.N;
      const float bb = EPI == EPI_ACC && blockIdx.y != 0 ? 0.f : pv.bias(a, it);  // the bias once
      float v = (sv[ml][c] + sv[ml + 9][c]) + sv[ml + 18][c];
      if constexpr (LN) v = lnst[kRows + ml] * (v - lnst[ml] * pv.lc[it]) + pv.le[it];
      v += bb;
      if constexpr (EPI == EPI_ARGMAX) {
        if (a.suppress != nullptr && pv.sup[it]) v = -INFINITY;
        head_score(a, row, n, act, v, &ov[ml][c], &oz[ml][c], pv.s0);
        if (act && a.y != nullptr) a.y[(size_t)row * a.ldy + n] = v;
      } else if constexpr (EPI == EPI_QKV) {
        if (act) {
          const int pos = pv.s1 + ml;
          if (n < a.d) a.y[(size_t)row * a.ldy + n] = v;
          else if (ml < pv.s0 && pos < a.n_ctx)
            qkv_append<S>(a, n, v, ((pv.s1 & 15) + ml >= 16) ? pv.s3 : pv.s2, pos);
        }
      } else {
        if (act) epi_one<S, EPI>(a, row, n, v, pv.r[it]);
      }
    }
  } else if (EPI == EPI_GELU && TC % 8 == 0 && a.N % 8 == 0) {
    // GELU into the next product's operand: an item is 8 consecutive columns of
    // one row, contiguous in every operand order, so each split term is one
    // 16-byte store (scalar stores would write 2 bytes per lane)
    constexpr int NI = TM * TC / 8, PI = (NI + NT - 1) / NT;
#pragma unroll
    for (int it = 0; it < PI; ++it) {
      const int item = threadIdx.x + it * NT;
      const int ml = item / (TC / 8), c8 = 8 * (item % (TC / 8)), row = m0 + ml, n = nb + c8;
      if (item >= NI || row < R || row >= Rend || n >= a.N) continue;
      float b8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if (a.bias != nullptr) {
#pragma unroll
        for (int e = 0; e < 8; ++e) b8[e] = to_f(reinterpret_cast<const S*>(a.bias)[n + e]);
      }
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = gelu_erf(sv[ml][c8 + e] + b8[e]);
      put_op8<S>(a.aout, a.nsplit, a.R9, row, n, v);
    }
  } else {
    // Every global load of the epilogue is issued before any result is formed, and
    // unconditionally (indexes clamped into the buffers, unused values discarded),
    // so their latencies overlap instead of adding up element by element.
    constexpr int P = (TM * TC + NT - 1) / NT;
    if constexpr (RP) rp.arrive();
    // without one, read the weights and discard; split-K partial sums added to y
    // (EPI_ACC) take the bias from the first k-split only
    const bool has_bias = a.bias != nullptr && !(EPI == EPI_ACC && blockIdx.y != 0);
    const S* bias = reinterpret_cast<const S*>(has_bias ? a.bias : a.w);
    const int rmax = a.R9 - 1, nmax = a.N - 1;
    float bv[P], rv[P];
    int iv[P], pv[P];  // QKV: cache page (-1: no append) and position; ARGMAX: step, suppressed
#pragma unroll
    for (int it = 0; it < P; ++it) {
      const int idx = threadIdx.x + it * NT;
      const int ml = idx / TC, c = idx % TC, row = min(m0 + ml, rmax), n = min(nb + c, nmax);
      if constexpr (RP) {
        bv[it] = has_bias ? __uint_as_float(rp.bb[it] << 16) : 0.f;
        rv[it] = rp.r[it];
      } else {
        const float bb = to_f(bias[n]);
        bv[it] = has_bias ? bb : 0.f;
        rv[it] = EPI == EPI_RESID ? a.y[(size_t)row * a.ldy + n] : 0.f;
      }
      iv[it] = -1;
      pv[it] = 0;
      if constexpr (EPI == EPI_QKV) {
        const int* st = a.state + (row / kRows) * kStateInts;
        const int r = row - (row / kRows) * kRows, nv = st[ST_NV], pos0 = st[ST_POS0];
        const int pg0 = st[ST_PG0], pg1 = st[ST_PG1];
        iv[it] = r < nv ? ((pos0 & 15) + r >= 16 ? pg1 : pg0) : -1;
        pv[it] = pos0 + r;
      } else if constexpr (EPI == EPI_ARGMAX) {
        // absent state / suppression: read the weights instead and discard
        const int* stp = a.state != nullptr ? a.state : reinterpret_cast<const int*>(a.w);
        const uint8_t* sup = a.suppress != nullptr ? a.suppress : reinterpret_cast<const uint8_t*>(a.w);
        const int step = stp[a.state != nullptr ? (row / kRows) * kStateInts + ST_STEP : 0];
        const int supv = sup[n];
        iv[it] = a.inv_t > 0.f && a.rng_purpose != 0 ? step : -1;
        pv[it] = a.suppress != nullptr ? supv : 0;
      }
    }
#pragma unroll
    for (int it = 0; it < P; ++it) {
      const int idx = threadIdx.x + it * NT;
      const int ml = idx / TC, c = idx % TC, row = m0 + ml, n = nb + c;
      const bool act = idx < TM * TC && row >= R && row < Rend && n < a.N;
      if (idx >= TM * TC) break;
      float v = sv[ml][c] + bv[it];
      if constexpr (EPI == EPI_ARGMAX) {
        if (pv[it]) v = -INFINITY;
        head_score(a, row, n, act, v, &ov[ml][c], &oz[ml][c], iv[it]);
        if (act && a.y != nullptr) a.y[(size_t)row * a.ldy + n] = v;
      } else if constexpr (EPI == EPI_QKV) {
        if (act) {
          const int d = a.d;
          if (n < d) a.y[(size_t)row * a.ldy + n] = v;
          else if (iv[it] >= 0 && pv[it] < a.n_ctx) qkv_append<S>(a, n, v, iv[it], pv[it]);
        }
      } else {
        if (act) epi_one<S, EPI>(a, row, n, v, rv[it]);
      }
    }
  }
  if constexpr (EPI == EPI_ARGMAX) {
    // A row's TC scores are reduced by a group of TC consecutive lanes with
    // butterflies (ties to the lower column, as better() orders them; columns past
    // N hold -inf scores and add nothing to the normaliser).
    static_assert(TC <= 64 && (TC & (TC - 1)) == 0, "a tile row fits one lane group");
    constexpr int GPB = NT / TC;
    const int j = threadIdx.x % TC, grp = threadIdx.x / TC;
    __syncthreads();
    for (int ml0 = 0; ml0 < nrows; ml0 += GPB) {
      const int ml = ml0 + grp, mc = min(ml, nrows - 1);
      const int row = split3 ? R + ml : m0 + ml;
      float bv = ov[mc][j], zm = oz[mc][j];
      int bi = nb + j;
#pragma unroll
      for (int o = TC / 2; o > 0; o >>= 1) {
        const float v2 = __shfl_xor(bv, o, TC);
        const int i2 = __shfl_xor(bi, o, TC);
        if (better(v2, i2, bv, bi)) {
          bv = v2;
          bi = i2;
        }
        zm = fmaxf(zm, __shfl_xor(zm, o, TC));
      }
      float zs = 0.f;
      if (a.hm != nullptr) {
        zs = zm > -INFINITY ? expf(oz[mc][j] - zm) : 0.f;
#pragma unroll
        for (int o = TC / 2; o > 0; o >>= 1) zs += __shfl_xor(zs, o, TC);
      }
      if (j == 0 && ml < nrows && row >= R && row < Rend) {
        const size_t o = (size_t)row * a.nblk + nb / TC;  // column block of this tile
        a.hv[o] = bv;
        a.hi[o] = bi;
        if (a.hm != nullptr) {
          a.hm[o] = zm;
          a.hs[o] = zs;
        }
      }
    }
  }
}

// ---------------------------------------------------------------- bf16, 16-column tiles
template <int EPI, int NW>
__global__ void __launch_bounds__(NW * 64) k_gemv16(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  constexpr int U = NW >= 16 ? kU / 2 : kU;
  __shared__ float red[NW][32][17];
  __shared__ float sv[32][17];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][16];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][16];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<16, NW * 64> pre;
  pre.template load<bf16, EPI>(a, blockIdx.x * 16);
  const int col = lane & 15, kg = lane >> 4;
  const int KS = a.K / 32;
  const int spw = (KS + NW - 1) / NW;
  const int s0 = min(KS, wv * spw), s1 = min(KS, s0 + spw);
  const bf16x8* Wt = reinterpret_cast<const bf16x8*>(a.w) + (size_t)blockIdx.x * KS * 64 + lane;
  const bf16x8* Ab = reinterpret_cast<const bf16x8*>(a.a.p) + lane;
  const int MT = a.a.mt;
  for (int tile0 = a.mt0; tile0 < a.mt1; tile0 += 2) {
    const bool two = tile0 + 1 < a.mt1;
    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    for (int st = s0; st < s1; st += U) {
      bf16x8 bw[U], a0[U], a1[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ss = min(st + u, s1 - 1);
        bw[u] = Wt[(size_t)ss * 64];
        a0[u] = Ab[((size_t)ss * MT + tile0) * 64];
        if (two) a1[u] = Ab[((size_t)ss * MT + tile0 + 1) * 64];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (st + u < s1) {
          acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], bw[u], acc0, 0, 0, 0);
          if (two) acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[u], bw[u], acc1, 0, 0, 0);
        }
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      red[wv][kg * 4 + v][col] = acc0[v];
      red[wv][16 + kg * 4 + v][col] = acc1[v];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 32 * 16; idx += NW * 64) {
      const int ml = idx >> 4, c = idx & 15;
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w][ml][c];
      sv[ml][c] = s;
    }
    __syncthreads();
    {
      RowsPre<32, 16, NW * 64> none;
      finish_tile<bf16, EPI, 32, 16, NW * 64>(a, sv, ov, oz, tile0 * 16, blockIdx.x * 16, pre, none);
    }
    if (a.nsplit == 3) break;
  }
}

// ---------------------------------------------------------------- bf16, CT 16-column tiles, split-K
// A block covers CT adjacent 16-column tiles (the operand fragments loaded per
// k-step serve CT weight fragments) and one of gridDim.y contiguous k-ranges;
// with more than one k-range the epilogue must be EPI_PART.
template <int EPI, int NW, int CT>
__global__ void __launch_bounds__(NW * 64) k_gemv16w(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  constexpr int U = CT >= 4 ? 4 : 8;
  constexpr int TC = 16 * CT;
  __shared__ float red[NW][32][TC + 1];
  __shared__ float sv[32][TC + 1];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][TC];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][TC];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<TC, NW * 64> pre;
  pre.template load<bf16, EPI>(a, blockIdx.x * TC);
  const int col = lane & 15, kg = lane >> 4;
  const int KS = a.K / 32;
  const int ntile = (a.N + 15) / 16;
  const int kss = (KS + gridDim.y - 1) / gridDim.y;
  const int k0 = min(KS, (int)blockIdx.y * kss), k1 = min(KS, k0 + kss);
  const int spw = (k1 - k0 + NW - 1) / NW;
  const int s0 = min(k1, k0 + wv * spw), s1 = min(k1, s0 + spw);
  const bf16x8* Wt = reinterpret_cast<const bf16x8*>(a.w) + (size_t)blockIdx.x * CT * KS * 64 + lane;
  const bf16x8* Ab = reinterpret_cast<const bf16x8*>(a.a.p) + lane;
  const int MT = a.a.mt;
  bool tv[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) tv[c] = (int)blockIdx.x * CT + c < ntile;
  for (int tile0 = a.mt0; tile0 < a.mt1; tile0 += 2) {
    const bool two = tile0 + 1 < a.mt1;
    floatx4 acc0[CT], acc1[CT];
#pragma unroll
    for (int c = 0; c < CT; ++c) acc0[c] = acc1[c] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int st = s0; st < s1; st += U) {
      bf16x8 bw[U][CT], a0[U], a1[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ss = min(st + u, s1 - 1);
#pragma unroll
        for (int c = 0; c < CT; ++c)
          if (tv[c]) bw[u][c] = Wt[((size_t)c * KS + ss) * 64];
        a0[u] = Ab[((size_t)ss * MT + tile0) * 64];
        if (two) a1[u] = Ab[((size_t)ss * MT + tile0 + 1) * 64];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (st + u < s1) {
#pragma unroll
          for (int c = 0; c < CT; ++c)
            if (tv[c]) {
              acc0[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], bw[u][c], acc0[c], 0, 0, 0);
              if (two) acc1[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[u], bw[u][c], acc1[c], 0, 0, 0);
            }
        }
    }
    __syncthreads();
#pragma unroll
    for (int c = 0; c < CT; ++c)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        red[wv][kg * 4 + v][16 * c + col] = acc0[c][v];
        red[wv][16 + kg * 4 + v][16 * c + col] = acc1[c][v];
      }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 32 * TC; idx += NW * 64) {
      const int ml = idx / TC, c = idx % TC;
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w][ml][c];
      sv[ml][c] = s;
    }
    __syncthreads();
    {
      RowsPre<32, TC, NW * 64> none;
      finish_tile<bf16, EPI, 32, TC, NW * 64>(a, sv, ov, oz, tile0 * 16, blockIdx.x * TC, pre, none);
    }
    if (a.nsplit == 3) break;
  }
}

// Batch 1 (three split terms in row tiles mt0 and mt0 + 1), CT 16-column tiles,
// split-K as k_gemv16w, when every wave's k-steps fit one batch of U: the wave's
// loads are issued together and unconditionally (tiles and steps past the data
// re-read the last valid one and are not multiplied), with no loop or branch
// around them, so nothing waits before the last of them is in flight.
template <int EPI, int NW, int CT, int U>
__global__ void __launch_bounds__(NW * 64) k_gemv16k(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  constexpr int TC = 16 * CT;
  static_assert(EPI == EPI_ACC || EPI == EPI_PART, "split-K epilogues only");
  __shared__ float red[NW][32][TC + 1];
  __shared__ float sv[32][TC + 1];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<TC, NW * 64> pre;
  pre.template load<bf16, EPI>(a, blockIdx.x * TC);
  const int col = lane & 15, kg = lane >> 4;
  const int KS = a.K / 32;
  const int ntile = (a.N + 15) / 16;
  const int kss = (KS + gridDim.y - 1) / gridDim.y;
  const int k0 = min(KS, (int)blockIdx.y * kss), k1 = min(KS, k0 + kss);
  const int spw = (k1 - k0 + NW - 1) / NW;
  const int s0 = min(k1, k0 + wv * spw), s1 = min(k1, s0 + spw);
  const int cmax = min(CT, ntile - (int)blockIdx.x * CT) - 1;  // last tile of this block inside N
  const bf16x8* Wt = reinterpret_cast<const bf16x8*>(a.w) + (size_t)blockIdx.x * CT * KS * 64 + lane;
  const bf16x8* Ab = reinterpret_cast<const bf16x8*>(a.a.p) + lane;
  const int MT = a.a.mt;
  bf16x8 bw[U][CT], a0[U], a1[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int ss = min(s0 + u, KS - 1);
#pragma unroll
    for (int c = 0; c < CT; ++c) bw[u][c] = Wt[((size_t)min(c, cmax) * KS + ss) * 64];
    a0[u] = Ab[((size_t)ss * MT + a.mt0) * 64];
    a1[u] = Ab[((size_t)ss * MT + a.mt0 + 1) * 64];
  }
  __builtin_amdgcn_sched_barrier(0);  // every load issued before the first wait
  floatx4 acc0[CT], acc1[CT];
#pragma unroll
  for (int c = 0; c < CT; ++c) acc0[c] = acc1[c] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (s0 + u < s1) {
#pragma unroll
      for (int c = 0; c < CT; ++c) {
        acc0[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0[u], bw[u][c], acc0[c], 0, 0, 0);
        acc1[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1[u], bw[u][c], acc1[c], 0, 0, 0);
      }
    }
#pragma unroll
  for (int c = 0; c < CT; ++c)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      red[wv][kg * 4 + v][16 * c + col] = acc0[c][v];
      red[wv][16 + kg * 4 + v][16 * c + col] = acc1[c][v];
    }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * TC; idx += NW * 64) {
    const int ml = idx / TC, c = idx % TC;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[w][ml][c];
    sv[ml][c] = s;
  }
  __syncthreads();
  {
    RowsPre<32, TC, NW * 64> none;
    finish_tile<bf16, EPI, 32, TC, NW * 64>(a, sv, nullptr, nullptr, a.mt0 * 16, blockIdx.x * TC, pre, none);
  }
}

// ---------------------------------------------------------------- bf16 GEMM (batch >= 2)
// The rows of several slots (nine each) times W^T over 64 x 64 block tiles: each of
// the four waves computes a 32 x 32 sub-tile (2 x 2 fragments of
// v_mfma_f32_16x16x32_bf16), loading operand and weight fragments straight from
// their fragment orders (1 KB per wave load).  The operand holds each value as
// two bf16 planes (hi + lo, 2^-17 relative), both multiplied into one
// accumulator, so the product is accurate to fp32 rounding.  Loads are double-buffered: the
// fragments of the next kGemmU k-steps are in flight while the current ones
// multiply.  Grid y splits the k-steps (EPI_PART stores each split's partial
// sums).  Block b runs on XCD b % 8; the row blocks of one column block are
// numbered so they share an XCD and its L2 serves them the weight tile.
typedef __attribute__((address_space(3))) void lds_void;
constexpr int kGemmU = 2;
// From this many 64-row blocks (two-plane operand over ~2 MB) the XCDs split the
// rows in two halves and the columns in four quarters, so each XCD's L2 keeps its
// half of the operand while the weight tiles stream (weights are then read by two
// XCDs, the operand no longer cycles through all eight L2s).
constexpr int kGemmSplitRows = 6;
__host__ __device__ __forceinline__ unsigned gemm_grid(int nmb, int nnb) {
  return nmb >= kGemmSplitRows ? 8u * ((nmb + 1) / 2) * ((nnb + 3) / 4) : 8u * ((nnb + 7) / 8) * nmb;
}
template <int EPI>
__global__ void __launch_bounds__(256) k_gemm16(GemvArgs a, int mb0, int nmb, int nnb) {
  StampScope stamp_scope(a.stamp, 256);
  __shared__ float sv[64][65];
  __shared__ float ov[EPI == EPI_ARGMAX ? 64 : 1][64];
  __shared__ float oz[EPI == EPI_ARGMAX ? 64 : 1][64];
  const int x = blockIdx.x & 7, i = blockIdx.x >> 3;
  int nbk, mbk;
  if (nmb >= kGemmSplitRows) {  // XCD x: row half x & 1, column quarter x >> 1 (row blocks fastest)
    const int nrh = (nmb + 1) / 2, ncq = (nnb + 3) / 4, rb0 = (x & 1) * nrh;
    mbk = rb0 + i % nrh;
    nbk = (x >> 1) * ncq + i / nrh;
    if (mbk >= nmb || i / nrh >= ncq || nbk >= nnb) return;
  } else {  // XCD x: column blocks x, x + 8, ..., each with every row block
    nbk = x + 8 * (i / nmb);
    mbk = i % nmb;
    if (nbk >= nnb) return;
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int wm = wv >> 1, wn = wv & 1;
  const int KS = a.K / 32, MT = a.a.mt, ntile = (a.N + 15) / 16;
  const int kper = KS / gridDim.y, ks0 = blockIdx.y * kper, ks1 = ks0 + kper;
  const int mt0 = (mb0 + mbk) * 4 + wm * 2, nt0 = nbk * 4 + wn * 2;  // 16-row / 16-column tiles
  RowsPre<64, 64, 256> rp;
  rp.template load<bf16, EPI>(a, (mb0 + mbk) * 64, nbk * 64);
  const bf16x8* Ab = reinterpret_cast<const bf16x8*>(a.a.p) + lane;
  const bf16x8* Wb = reinterpret_cast<const bf16x8*>(a.w) + lane;
  // Tiles past the operand's rows or the matrix's columns re-read the last one:
  // their products only reach output rows / columns the epilogue skips, and the
  // loads stay unconditional, so the compiler can wait for one buffer at a time.
  const int ma0 = min(mt0, MT - 1), ma1 = min(mt0 + 1, MT - 1);
  const int na0 = min(nt0, ntile - 1), na1 = min(nt0 + 1, ntile - 1);
  floatx4 acc[2][2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int q = 0; q < 2; ++q) acc[p][q] = floatx4{0.f, 0.f, 0.f, 0.f};
  // the operand's two bf16 planes (hi, lo): both multiply the same weight fragment
  const size_t plane = (size_t)MT * KS * 64;
  bf16x8 af[2][kGemmU][2][2], wf[2][kGemmU][2];
  auto load = [&](int b, int st) {  // k-steps st.. (past the range: re-read the last one)
#pragma unroll
    for (int u = 0; u < kGemmU; ++u) {
      const int ss = min(st + u, ks1 - 1);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        af[b][u][0][h] = Ab[h * plane + ((size_t)ss * MT + ma0) * 64];
        af[b][u][1][h] = Ab[h * plane + ((size_t)ss * MT + ma1) * 64];
      }
      wf[b][u][0] = Wb[((size_t)na0 * KS + ss) * 64];
      wf[b][u][1] = Wb[((size_t)na1 * KS + ss) * 64];
    }
  };
  auto mul = [&](int b, int st) {
#pragma unroll
    for (int u = 0; u < kGemmU; ++u)
      if (st + u < ks1) {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
          for (int p = 0; p < 2; ++p)
#pragma unroll
            for (int q = 0; q < 2; ++q)
              acc[p][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[b][u][p][h], wf[b][u][q], acc[p][q], 0, 0, 0);
      }
  };
  load(0, ks0);
  for (int st = ks0; st < ks1; st += 2 * kGemmU) {
    load(1, st + kGemmU);
    mul(0, st);
    load(0, st + 2 * kGemmU);
    mul(1, st + kGemmU);
  }
  // result fragment: lane l holds column l % 16, rows 4 (l / 16) + v
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        sv[wm * 32 + p * 16 + 4 * (lane >> 4) + v][wn * 32 + q * 16 + (lane & 15)] = acc[p][q][v];
  __syncthreads();
  EpiPre<64, 256> pre;  // batch-1 prefetch, unused here
  finish_tile<bf16, EPI, 64, 64, 256, true>(a, sv, ov, oz, (mb0 + mbk) * 64, nbk * 64, pre, rp);
}

// The same GEMM with the fragments staged through LDS: each k-step's twelve
// distinct 1 KB fragments (four 16-row operand tiles x two planes, four 16-column
// weight tiles) are copied once per block straight from memory into one of four
// 12 KB LDS stages (global_load_lds_dwordx4, three per wave), three k-steps ahead,
// and every wave reads its six fragments from LDS.  The loads through each CU's
// address units halve (24 KB per k-step became 12 KB), the kernel's limit.  The
// stages are separate LDS objects and the loop is unrolled over them, so the
// compiler sees that a copy into one stage cannot alias reads of another and keeps
// the copies in flight; each step waits for its own stage's copies (vmcnt) and its
// earlier LDS reads (lgkmcnt) before a plain barrier.
__shared__ uint4 g_stage0[12][64], g_stage1[12][64], g_stage2[12][64], g_stage3[12][64];
constexpr unsigned kGemmStagedBlocks = 256;
constexpr int kStageWait = (6 & 15) | (7 << 4) | (0 << 8);  // vmcnt <= 6 (two later k-steps' copies), lgkmcnt 0

template <int EPI>
__global__ void __launch_bounds__(256) k_gemm16s(GemvArgs a, int mb0, int nmb, int nnb) {
  StampScope stamp_scope(a.stamp, 256);
  __shared__ float sv[64][65];
  if (a.pf.blocks > 0 && blockIdx.x >= gridDim.x - a.pf.blocks) {  // appended blocks: a later product's weights
    if (blockIdx.y == 0) touch_range(a.pf, blockIdx.x - (gridDim.x - a.pf.blocks));
    return;
  }
  const int x = blockIdx.x & 7, i = blockIdx.x >> 3;
  int nbk, mbk;
  if (nmb >= kGemmSplitRows) {
    const int nrh = (nmb + 1) / 2, ncq = (nnb + 3) / 4, rb0 = (x & 1) * nrh;
    mbk = rb0 + i % nrh;
    nbk = (x >> 1) * ncq + i / nrh;
    if (mbk >= nmb || i / nrh >= ncq || nbk >= nnb) return;
  } else {
    nbk = x + 8 * (i / nmb);
    mbk = i % nmb;
    if (nbk >= nnb) return;
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int wm = wv >> 1, wn = wv & 1;
  const int KS = a.K / 32, MT = a.a.mt, ntile = (a.N + 15) / 16;
  const int kper = KS / gridDim.y, ks0 = blockIdx.y * kper, ks1 = ks0 + kper;
  RowsPre<64, 64, 256> rp;
  rp.template load<bf16, EPI>(a, (mb0 + mbk) * 64, nbk * 64);
  // this wave's three fragments of every k-step: f < 8 operand tile f >> 1, plane
  // f & 1; f >= 8 weight tile f - 8 (tiles past the data re-read the last one)
  const bf16x8* src[3];
  size_t sstride[3];
  const size_t plane = (size_t)MT * KS * 64;
#pragma unroll
  for (int j = 0; j < 3; ++j) {
    const int f = 3 * wv + j;
    if (f < 8) {
      const int mt = min((mb0 + mbk) * 4 + (f >> 1), MT - 1);
      src[j] = reinterpret_cast<const bf16x8*>(a.a.p) + (f & 1) * plane + (size_t)mt * 64 + lane;
      sstride[j] = (size_t)MT * 64;
    } else {
      const int nt = min(nbk * 4 + f - 8, ntile - 1);
      src[j] = reinterpret_cast<const bf16x8*>(a.w) + (size_t)nt * KS * 64 + lane;
      sstride[j] = 64;
    }
  }
  auto copy = [&](int st, uint4 (*stg)[64]) {  // k-step st (past the range: the last one)
    const size_t ss = (size_t)min(st, ks1 - 1);
#pragma unroll
    for (int j = 0; j < 3; ++j)
      __builtin_amdgcn_global_load_lds((const void*)(src[j] + ss * sstride[j]), (lds_void*)&stg[3 * wv + j][0], 16, 0, 0);
  };
  floatx4 acc[2][2];
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int q = 0; q < 2; ++q) acc[p][q] = floatx4{0.f, 0.f, 0.f, 0.f};
  auto step = [&](int st, uint4 (*cur)[64], uint4 (*nxt)[64]) {
    __builtin_amdgcn_s_waitcnt(kStageWait);
    __builtin_amdgcn_s_barrier();
    copy(st + 3, nxt);  // every step issues three copies, so the wait count stays exact
    if (st < ks1) {
      bf16x8 af[2][2], wf[2];
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int h = 0; h < 2; ++h) af[p][h] = __builtin_bit_cast(bf16x8, cur[2 * (2 * wm + p) + h][lane]);
#pragma unroll
      for (int q = 0; q < 2; ++q) wf[q] = __builtin_bit_cast(bf16x8, cur[8 + 2 * wn + q][lane]);
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int q = 0; q < 2; ++q)
            acc[p][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[p][h], wf[q], acc[p][q], 0, 0, 0);
    }
  };
  copy(ks0, g_stage0);
  copy(ks0 + 1, g_stage1);
  copy(ks0 + 2, g_stage2);
  for (int st = ks0; st < ks1; st += 4) {
    step(st, g_stage0, g_stage3);
    step(st + 1, g_stage1, g_stage0);
    step(st + 2, g_stage2, g_stage1);
    step(st + 3, g_stage3, g_stage2);
  }
  // no copy may land in LDS after the block has left
  __builtin_amdgcn_s_waitcnt((0 & 15) | (7 << 4) | (15 << 8));
#pragma unroll
  for (int p = 0; p < 2; ++p)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int v = 0; v < 4; ++v)
        sv[wm * 32 + p * 16 + 4 * (lane >> 4) + v][wn * 32 + q * 16 + (lane & 15)] = acc[p][q][v];
  __syncthreads();
  EpiPre<64, 256> pre;  // batch-1 prefetch, unused here
  float ov[1][64], oz[1][64];  // (no argmax here)
  finish_tile<bf16, EPI, 64, 64, 256, true>(a, sv, ov, oz, (mb0 + mbk) * 64, nbk * 64, pre, rp);
}

// ---------------------------------------------------------------- several slots, wide tiles
// Products of many slots' rows (hundreds of rows) on v_mfma_f32_32x32x16_bf16,
// which issues twice the work per cycle of the 16x16x32 form here.  The data keep
// their 16x32 fragment order: the 32x32x16 operand of lane l is row l % 32 of a
// 32-row tile and k chunk 2 s + l / 32 of k-substep s, i.e. lane (l % 16) + 16 (2 s +
// l / 32) of 16-row fragment 2 j + (l % 32) / 16, so every load is 16 bytes from a
// 256-byte run.  Block tile 64 rows x 32 CN columns, four independent waves of 32 x
// 16 CN (no LDS in the main loop, no barrier): each wave loads its own operand and
// weight fragments straight into registers kWideD k-steps ahead (about 160 KB in
// flight per CU; LDS-staged copies behind a barrier per k-step stayed latency-bound
// at a third of that).  XCD x takes row half x & 1 and column quarter x >> 1, so the
// blocks sharing an L2 share their operand rows and weight columns.  The finished
// tile is staged in LDS and written 8 consecutive columns per item (16-byte stores).
constexpr int kWideD = 4;             // k-steps in flight per wave (the k-step count must be a multiple)
constexpr int kWideMinRowBlocks = 8;  // 64-row blocks from which the wide kernel is used (about 57 slots)
constexpr int kWideMaxCN = 10;        // widest tile: 32 kWideMaxCN columns

__host__ __device__ __forceinline__ unsigned wide_grid(int nmb, int nnb) {
  return 8u * ((nmb + 1) / 2) * ((nnb + 3) / 4);
}

template <int EPI, int CN>
__global__ void __launch_bounds__(256) k_gemm32r(GemvArgs a, int mb0, int nmb, int nnb) {
  static_assert(CN <= kWideMaxCN && CN % 2 == 0, "tile width");
  StampScope stamp_scope(a.stamp, 256);
  constexpr int WCT = CN / 2, TC = 32 * CN;
  __shared__ float sv[64][TC + 1];  // the finished tile
  if (a.pf.blocks > 0 && blockIdx.x >= gridDim.x - a.pf.blocks) {  // appended blocks: a later product's weights
    if (blockIdx.y == 0) touch_range(a.pf, blockIdx.x - (gridDim.x - a.pf.blocks));
    return;
  }
  int mbk, nbk;
  {
    const int x = blockIdx.x & 7, i = blockIdx.x >> 3;
    const int nrh = (nmb + 1) / 2, ncq = (nnb + 3) / 4;
    mbk = (x & 1) * nrh + i % nrh;
    nbk = (x >> 1) * ncq + i / nrh;
    if (i >= nrh * ncq || mbk >= nmb || nbk >= nnb) return;
  }
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, wm = wv >> 1, wn = wv & 1;
  const int KS = a.K / 32, MT = a.a.mt, ntile = (a.N + 15) / 16;
  const size_t plane = (size_t)MT * KS * 64;
  const int r32 = lane & 31, kh = lane >> 5, fsub = r32 >> 4, fl = (r32 & 15) + 16 * kh;
  // rows and columns past the data re-read the last tile; their results are not written
  const int mt = min((mb0 + mbk) * 4 + 2 * wm + fsub, MT - 1);
  const bf16x8* pa = reinterpret_cast<const bf16x8*>(a.a.p) + (size_t)mt * 64 + fl;
  const bf16x8* pb[WCT];
#pragma unroll
  for (int q = 0; q < WCT; ++q)
    pb[q] = reinterpret_cast<const bf16x8*>(a.w) + (size_t)min(2 * (nbk * CN + wn * WCT + q) + fsub, ntile - 1) * KS * 64 + fl;
  struct Frag {
    bf16x8 a[2][2], w[2][WCT];  // [k-substep][plane], [k-substep][column tile]
  };
  auto ld = [&](int st, Frag& f) {
    const size_t ss = (size_t)min(st, KS - 1);
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) {
#pragma unroll
      for (int h = 0; h < 2; ++h) f.a[sub][h] = pa[h * plane + ss * MT * 64 + 32 * sub];
#pragma unroll
      for (int q = 0; q < WCT; ++q) f.w[sub][q] = pb[q][ss * 64 + 32 * sub];
    }
  };
  floatx16 acc[WCT];
#pragma unroll
  for (int q = 0; q < WCT; ++q)
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[q][v] = 0.f;
  auto mul = [&](const Frag& f) {
#pragma unroll
    for (int sub = 0; sub < 2; ++sub)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int q = 0; q < WCT; ++q) acc[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[sub][h], f.w[sub][q], acc[q], 0, 0, 0);
  };
  // Each step multiplies the fragments loaded kWideD steps earlier and reloads their
  // registers kWideD steps ahead (past the end: the last k-step again, unused); the
  // scheduling barriers keep every load where it is issued (the scheduler otherwise
  // moves loads next to their use to shorten register lifetimes).
  // grid y splits the k-steps (EPI_PART: one partial-sum buffer per split)
  const int kper = KS / gridDim.y, kb = blockIdx.y * kper, ke = kb + kper;
  Frag fr[kWideD];
#pragma unroll
  for (int d = 0; d < kWideD; ++d) ld(kb + d, fr[d]);
  __builtin_amdgcn_sched_barrier(0);
  for (int st = kb; st < ke; st += kWideD) {
#pragma unroll
    for (int d = 0; d < kWideD; ++d) {
      mul(fr[d]);
      __builtin_amdgcn_sched_barrier(0);
      ld(st + d + kWideD, fr[d]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  // accumulator v of 32 x 32 tile q: row 8 (v / 4) + 4 (lane / 32) + v % 4, column lane % 32
#pragma unroll
  for (int q = 0; q < WCT; ++q)
#pragma unroll
    for (int v = 0; v < 16; ++v) sv[wm * 32 + 8 * (v >> 2) + 4 * kh + (v & 3)][(wn * WCT + q) * 32 + r32] = acc[q][v];
  __syncthreads();
  // epilogue items: 8 consecutive columns of one row
  const int m0 = (mb0 + mbk) * 64, n0 = nbk * TC;
  const int R = a.slot0 * kRows, Rend = (a.slot0 + a.nslots) * kRows;
  const uint4* bias8 = reinterpret_cast<const uint4*>(a.bias);
  for (int item = threadIdx.x; item < 64 * (TC / 8); item += 256) {
    const int ml = item / (TC / 8), c8 = 8 * (item % (TC / 8)), row = m0 + ml, n = n0 + c8;
    if (row < R || row >= Rend || n >= a.N) continue;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = sv[ml][c8 + e];
    if (bias8 != nullptr) {
      const uint4 bb = bias8[n / 8];
      const uint32_t bw[4] = {bb.x, bb.y, bb.z, bb.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += __uint_as_float(e & 1 ? bw[e >> 1] & 0xffff0000u : bw[e >> 1] << 16);
    }
    if constexpr (EPI == EPI_GELU) {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = gelu_erf(v[e]);
      put_op8<bf16>(a.aout, a.nsplit, a.R9, row, n, v);
    } else if constexpr (EPI == EPI_STORE || EPI == EPI_PART) {
      float* yb = EPI == EPI_PART ? a.y + blockIdx.y * a.pstride : a.y;
      float4* y = reinterpret_cast<float4*>(yb + (size_t)row * a.ldy + n);
      y[0] = make_float4(v[0], v[1], v[2], v[3]);
      y[1] = make_float4(v[4], v[5], v[6], v[7]);
    } else if constexpr (EPI == EPI_RESID) {
      float4* y = reinterpret_cast<float4*>(a.y + (size_t)row * a.ldy + n);
      const float4 r0 = y[0], r1 = y[1];
      v[0] += r0.x; v[1] += r0.y; v[2] += r0.z; v[3] += r0.w;
      v[4] += r1.x; v[5] += r1.y; v[6] += r1.z; v[7] += r1.w;
      y[0] = make_float4(v[0], v[1], v[2], v[3]);
      y[1] = make_float4(v[4], v[5], v[6], v[7]);
      if (a.tap >= 0) put_op8<bf16>(a.aout, a.nsplit, a.R9, row, a.tap * a.N + n, v);
    } else if constexpr (EPI == EPI_QKV) {
      if (n < a.d) {
        float4* y = reinterpret_cast<float4*>(a.y + (size_t)row * a.ldy + n);
        y[0] = make_float4(v[0], v[1], v[2], v[3]);
        y[1] = make_float4(v[4], v[5], v[6], v[7]);
      } else {
        const int* st = a.state + (row / kRows) * kStateInts;
        const int r = row - (row / kRows) * kRows, pos0 = st[ST_POS0];
        const int page = (pos0 & 15) + r >= 16 ? st[ST_PG1] : st[ST_PG0];
        if (r < st[ST_NV] && pos0 + r < a.n_ctx) {
#pragma unroll
          for (int e = 0; e < 8; ++e) qkv_append<bf16>(a, n + e, v[e], page, pos0 + r);
        }
      }
    }
  }
}

// ---------------------------------------------------------------- bf16, 32-column tiles
template <int EPI, int NW>
__global__ void __launch_bounds__(NW * 64) k_gemv32(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  constexpr int U = NW >= 16 ? kU / 2 : kU;
  __shared__ float red[NW][32][33];
  __shared__ float sv[32][33];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][32];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][32];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<32, NW * 64> pre;
  pre.template load<bf16, EPI>(a, blockIdx.x * 32);
  const int col = lane & 31, kg = lane >> 5;
  const int KS = a.K / 16;
  const int spw = (KS + NW - 1) / NW;
  const int s0 = min(KS, wv * spw), s1 = min(KS, s0 + spw);
  const bf16x8* Wt = reinterpret_cast<const bf16x8*>(a.w) + (size_t)blockIdx.x * KS * 64 + lane;
  const bf16x8* Ab = reinterpret_cast<const bf16x8*>(a.a.p) + lane;
  const int MT = a.a.mt;
  for (int tile0 = a.mt0; tile0 < a.mt1; ++tile0) {
    floatx16 acc = {};
    for (int st = s0; st < s1; st += U) {
      bf16x8 bw[U], av[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int ss = min(st + u, s1 - 1);
        bw[u] = Wt[(size_t)ss * 64];
        av[u] = Ab[((size_t)ss * MT + tile0) * 64];
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (st + u < s1) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[u], bw[u], acc, 0, 0, 0);
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) red[wv][8 * i + 4 * kg + j][col] = acc[4 * i + j];
    __syncthreads();
    for (int idx = threadIdx.x; idx < 32 * 32; idx += NW * 64) {
      const int ml = idx >> 5, c = idx & 31;
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w][ml][c];
      sv[ml][c] = s;
    }
    __syncthreads();
    {
      RowsPre<32, 32, NW * 64> none;
      finish_tile<bf16, EPI, 32, 32, NW * 64>(a, sv, ov, oz, tile0 * 32, blockIdx.x * 32, pre, none);
    }
    if (a.nsplit == 3) break;
  }
}

// ---------------------------------------------------------------- LayerNorm folded in (bf16, batch 1)
// The block stages its operand in LDS itself (LnFold below): three bf16 split
// terms per value (rows r, 9 + r, 18 + r; rows 27..31 zero) in the fragment order
// of its tile shape.

// LDS slot of operand chunk (row m, k..k+7): fragment order with the 16-byte slot
// inside each 256-byte group XOR-swizzled by the group index, so that both the
// staging writes (one row, many k) and the fragment reads (64 consecutive slots)
// spread over the banks.
__device__ __forceinline__ int lds_swz(int i) { return i ^ ((i >> 4) & 15); }
template <int TILE>
__device__ __forceinline__ int lds_frag(int m, int k) {
  if constexpr (TILE == 16) return lds_swz(((k >> 5) * 2 + (m >> 4)) * 64 + (m & 15) + 16 * ((k & 31) >> 3));
  else return lds_swz((k >> 4) * 64 + (m & 31) + 32 * ((k & 15) >> 3));
}

// Operand of a batch-1 product with its LayerNorm folded in.  For a row x with
// mean m and r = 1/sqrt(var + eps), LN(x) W^T = r ((x*g) W^T - m (g W^T)) + b W^T,
// so the block stages x*g alone (three split terms, no statistics needed) and
// the epilogue applies m and r with the column sums c = g W^T and e = b W^T
// precomputed per matrix.  The 9 x K/8 items (row, 8 consecutive columns) are
// spread over all the block's lanes, and every item leaves its sum and its sum of
// squared deviations from its own mean; after the staging barrier wave r merges
// row r's items (the pairwise update of Chan, Golub and LeVeque) in a fixed order
// while the weight loads are still in flight (with fewer than nine waves, wave w
// merges rows w, w + NW, ...).
template <int NW>
struct LnFold {
  static constexpr int NT = NW * 64;
  // Item t = lane + i S for i < I, with the stride S = NT - NT % (K/8) a multiple of
  // K/8: a lane's items share their 8 columns (one load of the gains) and lanes
  // >= S hold none.  K <= kLnFoldMaxK gives at most I items per lane.
  static constexpr int I = (kRows + NT / (kLnFoldMaxK / 8) - 1) / (NT / (kLnFoldMaxK / 8));
  static_assert(NT >= kLnFoldMaxK / 8, "a lane per column of the items");
  float x[I][8];
  uint4 g;

  // Only the items that exist are loaded; these loads are all issued before the
  // weights', so waiting for them never waits for the weights.
  __device__ __forceinline__ void load(const GemvArgs& a) {
    const int nch = a.K >> 3, ni = kRows * nch, S = NT - NT % nch;
    const int c = (int)threadIdx.x % nch;
    if ((int)threadIdx.x < S) g = reinterpret_cast<const uint4*>(a.lng)[c];
#pragma unroll
    for (int i = 0; i < I; ++i) {
      const int t = (int)threadIdx.x + i * S;
      if ((int)threadIdx.x < S && t < ni) ld8(a.lnx + (size_t)(t / nch) * a.K + 8 * c, x[i]);
    }
  }

  // Writes the operand x*g into aop (rows r, 9 + r and 18 + r hold the three split
  // terms of row r; rows 27..31 are zero) and the item statistics of row r into
  // ps + r * pstride: sums at [c], squared deviations at [K/8 + c].
  template <int TILE>
  __device__ __forceinline__ void stage(const GemvArgs& a, uint4* aop, float* ps, int pstride) const {
    const int nch = a.K >> 3, ni = kRows * nch, S = NT - NT % nch;
    const int c = (int)threadIdx.x % nch;
#pragma unroll
    for (int i = 0; i < I; ++i) {
      const int t = (int)threadIdx.x + i * S;
      if ((int)threadIdx.x < S && t < ni) {
        const int r = t / nch;
        const uint32_t gw[4] = {g.x, g.y, g.z, g.w};
        uint32_t th[8], tm[8], tl[8];
        float sum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float gv = __uint_as_float(e & 1 ? gw[e >> 1] & 0xffff0000u : gw[e >> 1] << 16);
          split3_bits(x[i][e] * gv, th[e], tm[e], tl[e]);
          sum += x[i][e];
        }
        const float m = sum * 0.125f;
        float dev = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float dx = x[i][e] - m;
          dev = fmaf(dx, dx, dev);
        }
        aop[lds_frag<TILE>(r, 8 * c)] = pack8_bits(th);
        aop[lds_frag<TILE>(kRows + r, 8 * c)] = pack8_bits(tm);
        aop[lds_frag<TILE>(2 * kRows + r, 8 * c)] = pack8_bits(tl);
        ps[r * pstride + c] = sum;
        ps[r * pstride + nch + c] = dev;
        if (a.tap >= 0 && t % (int)gridDim.x == (int)blockIdx.x) {
          // the drafter tap of the rows (the previous block's output, 16-row
          // fragment order, three split terms): each item written by one block
          uint32_t xh[8], xm[8], xl[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) split3_bits(x[i][e], xh[e], xm[e], xl[e]);
          uint4* T = reinterpret_cast<uint4*>(a.aout.p);
          const int row = a.slot0 * kRows + r, col = a.tap * a.K + 8 * c;
          T[afrag16_index(row, col, a.aout.mt) / 8] = pack8_bits(xh);
          T[afrag16_index(a.R9 + row, col, a.aout.mt) / 8] = pack8_bits(xm);
          T[afrag16_index(2 * a.R9 + row, col, a.aout.mt) / 8] = pack8_bits(xl);
        }
      }
    }
    for (int t = threadIdx.x; t < (32 - 3 * kRows) * nch; t += NT)
      aop[lds_frag<TILE>(3 * kRows + t / nch, 8 * (t % nch))] = make_uint4(0u, 0u, 0u, 0u);
  }

  // Merges row r's items into st[r] = mean and st[9 + r] = 1/sqrt(var + eps), row r
  // taken by wave r % NW.
  __device__ __forceinline__ static void row_stats(const GemvArgs& a, const float* ps, int pstride, float* st) {
    for (int r = (int)threadIdx.x >> 6; r < kRows; r += NW) row_stat(a, ps + r * pstride, r, st);
  }
  __device__ __forceinline__ static void row_stat(const GemvArgs& a, const float* p, int r, float* st) {
    const int lane = threadIdx.x & 63;
    constexpr int J = (kLnFoldMaxK / 8 + 63) / 64;
    const int nch = a.K >> 3;
    float sm[J], dv[J];
    float sum = 0.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int c = lane + 64 * j;
      sm[j] = c < nch ? p[c] : 0.f;
      dv[j] = c < nch ? p[nch + c] : 0.f;
      sum += sm[j];
    }
    const float mean = wave_sum(sum) / (float)a.K;
    float m2 = 0.f;
#pragma unroll
    for (int j = 0; j < J; ++j) {
      if (lane + 64 * j < nch) {
        const float dm = sm[j] * 0.125f - mean;
        m2 += fmaf(8.f * dm, dm, dv[j]);
      }
    }
    const float var = wave_sum(m2) / (float)a.K;
    if (lane == 0) {
      st[r] = mean;
      st[kRows + r] = 1.0f / sqrtf(var + 1e-5f);
    }
  }
};

// ---------------------------------------------------------------- batch-1 head, persistent
// Batch 1 (three split terms in one 32-row tile), 32-column tiles: a block walks
// the column tiles tile = blockIdx.x + i gridDim.x.  The operand fragments of a
// wave's k-steps are the same for every tile and stay in registers; the next
// tile's weight fragments and epilogue prefetch are in flight while the current
// tile is multiplied, reduced and finished.  The two sets of registers alternate
// (a copy from one to the other would wait for its loads); past the last tile a
// block re-reads its current one (from L2) instead of branching around the loads.
// LN: the final LayerNorm folded in; each block stages the rows (LnFold) before its
// first tile, behind its first weight loads, and the epilogue applies the rows'
// statistics with the column sums of that LayerNorm.
constexpr int kHeadBlocks = 256;
template <int EPI, int NW, int U, bool LN>
__global__ void __launch_bounds__(NW * 64) k_gemv32p(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  __shared__ float red[NW][32][33];
  __shared__ float sv[32][33];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][32];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][32];
  __shared__ uint4 aop[LN ? kLnFoldMaxK / 16 * 64 : 1];
  __shared__ float lnst[LN ? 2 * kRows : 1];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int col = lane & 31, kg = lane >> 5;
  const int KS = a.K / 16, ntile = (a.N + 31) / 32;
  const int spw = (KS + NW - 1) / NW;
  const int s0 = min(KS, wv * spw), s1 = min(KS, s0 + spw);
  const bf16x8* W0 = reinterpret_cast<const bf16x8*>(a.w) + lane;
  const bf16x8* Ab = reinterpret_cast<const bf16x8*>(a.a.p) + lane;
  typedef EpiPre<32, NW * 64, LN> Pre;
  auto fetch = [&](int tile, bf16x8* w, Pre& p) {
    p.template load<bf16, EPI>(a, tile * 32);
    const bf16x8* Wt = W0 + (size_t)tile * KS * 64;
#pragma unroll
    for (int u = 0; u < U; ++u) w[u] = Wt[(size_t)min(s0 + u, KS - 1) * 64];
  };
  bf16x8 av[U], wa[U], wb[U];
  Pre pa, pb;
  auto finish = [&](int tile, const bf16x8* w, const Pre& p) {
    floatx16 acc = {};
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (s0 + u < s1) acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[u], w[u], acc, 0, 0, 0);
    __syncthreads();  // the previous tile's epilogue is done with red, sv, ov and oz
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) red[wv][8 * i + 4 * kg + j][col] = acc[4 * i + j];
    __syncthreads();
    for (int idx = threadIdx.x; idx < 32 * 32; idx += NW * 64) {
      const int ml = idx >> 5, c = idx & 31;
      float sum = 0.f;
#pragma unroll
      for (int w8 = 0; w8 < NW; ++w8) sum += red[w8][ml][c];
      sv[ml][c] = sum;
    }
    __syncthreads();
    RowsPre<32, 32, NW * 64> none;
    finish_tile<bf16, EPI, 32, 32, NW * 64, false, LN>(a, sv, ov, oz, a.mt0 * 32, tile * 32, p, none, lnst);
  };
  const int G = gridDim.x;
  int tile = blockIdx.x;
  if constexpr (LN) {
    // rows first, then the first tile's weights, then the staging (which waits for
    // the rows alone); the item statistics of the nine rows sit packed in the
    // reduction buffer, which the first tile's epilogue takes only after a barrier
    constexpr int PS = 2 * (kLnFoldMaxK / 8);
    static_assert(kRows * PS <= NW * 32 * 33, "item statistics fit the reduction buffer");
    LnFold<NW> rows;
    rows.load(a);
    __builtin_amdgcn_sched_barrier(0);
    fetch(tile, wa, pa);
    __builtin_amdgcn_sched_barrier(0);
    rows.template stage<32>(a, aop, &red[0][0][0], PS);
    __syncthreads();
    LnFold<NW>::row_stats(a, &red[0][0][0], PS, lnst);
#pragma unroll
    for (int u = 0; u < U; ++u) av[u] = __builtin_bit_cast(bf16x8, aop[lds_swz(min(s0 + u, KS - 1) * 64 + lane)]);
  } else {
    fetch(tile, wa, pa);
#pragma unroll
    for (int u = 0; u < U; ++u) av[u] = Ab[((size_t)min(s0 + u, KS - 1) * a.a.mt + a.mt0) * 64];
  }
  for (;;) {
    fetch(tile + G < ntile ? tile + G : tile, wb, pb);
    __builtin_amdgcn_sched_barrier(0);
    finish(tile, wa, pa);
    tile += G;
    if (tile >= ntile) break;
    fetch(tile + G < ntile ? tile + G : tile, wa, pa);
    __builtin_amdgcn_sched_barrier(0);
    finish(tile, wb, pb);
    tile += G;
    if (tile >= ntile) break;
  }
}

// 16-column tiles; every wave's k-steps fit one batch of loads (K <= kLnFoldMaxK).
template <int EPI, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_gemv16_ln(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  __shared__ uint4 aop[kLnFoldMaxK / 32 * 2 * 64];
  __shared__ float red[NW][32][17];
  __shared__ float sv[32][17];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][16];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][16];
  __shared__ float lnst[2 * kRows];
  static_assert(2 * (kLnFoldMaxK / 8) <= 32 * 17, "item statistics of a row fit its wave's reduction slot");
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<16, NW * 64, true> pre;
  pre.template load<bf16, EPI>(a, blockIdx.x * 16);
  const int col = lane & 15, kg = lane >> 4;
  const int KS = a.K / 32;
  const int spw = (KS + NW - 1) / NW;
  const int s0 = min(KS, wv * spw), s1 = min(KS, s0 + spw);
  const bf16x8* Wt = reinterpret_cast<const bf16x8*>(a.w) + (size_t)blockIdx.x * KS * 64 + lane;
  LnFold<NW> rows;
  rows.load(a);
  // The weight loads are unconditional (steps past the wave's range re-read the
  // last one and are not multiplied) and kept after the rows' loads (scheduling
  // barriers), so the staging waits only for the rows, not for the weights.
  __builtin_amdgcn_sched_barrier(0);
  bf16x8 bw[U];
#pragma unroll
  for (int u = 0; u < U; ++u)
    bw[u] = Wt[(size_t)min(s0 + u, KS - 1) * 64];
  __builtin_amdgcn_sched_barrier(0);
  // the item statistics of row r go to wave r's reduction slot, which that wave
  // reads back before it writes its products there
  rows.template stage<16>(a, aop, &red[0][0][0], 32 * 17);
  __syncthreads();
  LnFold<NW>::row_stats(a, &red[0][0][0], 32 * 17, lnst);
  floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (s0 + u < s1) {
      const bf16x8 a0 = __builtin_bit_cast(bf16x8, aop[lds_swz(((s0 + u) * 2) * 64 + lane)]);
      const bf16x8 a1 = __builtin_bit_cast(bf16x8, aop[lds_swz(((s0 + u) * 2 + 1) * 64 + lane)]);
      acc0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a0, bw[u], acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a1, bw[u], acc1, 0, 0, 0);
    }
#pragma unroll
  for (int v = 0; v < 4; ++v) {
    red[wv][kg * 4 + v][col] = acc0[v];
    red[wv][16 + kg * 4 + v][col] = acc1[v];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * 16; idx += NW * 64) {
    const int ml = idx >> 4, c = idx & 15;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[w][ml][c];
    sv[ml][c] = s;
  }
  __syncthreads();
  {
      RowsPre<32, 16, NW * 64> none;
      finish_tile<bf16, EPI, 32, 16, NW * 64, false, true>(a, sv, ov, oz, 0, blockIdx.x * 16, pre, none, lnst);
    }
}

// 32-column tiles; every wave's k-steps fit one batch of loads (K <= kLnFoldMaxK).
template <int EPI, int NW, int U>
__global__ void __launch_bounds__(NW * 64) k_gemv32_ln(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  __shared__ uint4 aop[kLnFoldMaxK / 16 * 64];
  __shared__ float red[NW][32][33];
  __shared__ float sv[32][33];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][32];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][32];
  __shared__ float lnst[2 * kRows];
  static_assert(2 * (kLnFoldMaxK / 8) <= 32 * 33, "item statistics of a row fit its wave's reduction slot");
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<32, NW * 64, true> pre;
  pre.template load<bf16, EPI>(a, blockIdx.x * 32);
  const int col = lane & 31, kg = lane >> 5;
  const int KS = a.K / 16;
  const int spw = (KS + NW - 1) / NW;
  const int s0 = min(KS, wv * spw), s1 = min(KS, s0 + spw);
  const bf16x8* Wt = reinterpret_cast<const bf16x8*>(a.w) + (size_t)blockIdx.x * KS * 64 + lane;
  LnFold<NW> rows;
  rows.load(a);
  // The weight loads are unconditional (steps past the wave's range re-read the
  // last one and are not multiplied) and kept after the rows' loads (scheduling
  // barriers), so the staging waits only for the rows, not for the weights.
  __builtin_amdgcn_sched_barrier(0);
  bf16x8 bw[U];
#pragma unroll
  for (int u = 0; u < U; ++u)
    bw[u] = Wt[(size_t)min(s0 + u, KS - 1) * 64];
  __builtin_amdgcn_sched_barrier(0);
  rows.template stage<32>(a, aop, &red[0][0][0], 32 * 33);
  __syncthreads();
  LnFold<NW>::row_stats(a, &red[0][0][0], 32 * 33, lnst);
  floatx16 acc = {};
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (s0 + u < s1)
      acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, aop[lds_swz((s0 + u) * 64 + lane)]), bw[u],
                                                     acc, 0, 0, 0);
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) red[wv][8 * i + 4 * kg + j][col] = acc[4 * i + j];
  __syncthreads();
  for (int idx = threadIdx.x; idx < 32 * 32; idx += NW * 64) {
    const int ml = idx >> 5, c = idx & 31;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) s += red[w][ml][c];
    sv[ml][c] = s;
  }
  __syncthreads();
  {
      RowsPre<32, 32, NW * 64> none;
      finish_tile<bf16, EPI, 32, 32, NW * 64, false, true>(a, sv, ov, oz, 0, blockIdx.x * 32, pre, none, lnst);
    }
}

// ---------------------------------------------------------------- fp32, row-major
// Lane group kg supplies k = kg*4 + e at step e of each 16-wide slice (the sum over
// k does not depend on the order in which k is visited).
template <int EPI, int NW>
__global__ void __launch_bounds__(NW * 64) k_gemv_f32(GemvArgs a) {
  StampScope stamp_scope(a.stamp, NW * 64);
  constexpr int U = NW >= 16 ? kU / 2 : kU;
  __shared__ float red[NW][32][17];
  __shared__ float sv[32][17];
  __shared__ float ov[EPI == EPI_ARGMAX ? 32 : 1][16];
  __shared__ float oz[EPI == EPI_ARGMAX ? 32 : 1][16];
  const float* __restrict__ W = reinterpret_cast<const float*>(a.w);
  const float* __restrict__ A = reinterpret_cast<const float*>(a.a.p);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  EpiPre<16, NW * 64> pre;
  pre.template load<float, EPI>(a, blockIdx.x * 16);
  const int col = lane & 15, kg = lane >> 4;
  const int nb = blockIdx.x * 16;
  const int K = a.K, lda = a.a.ld;
  const int KS = K / 16;
  const int spw = (KS + NW - 1) / NW;
  const int s0 = min(KS, wv * spw), s1 = min(KS, s0 + spw);
  const float* wp = W + (size_t)min(nb + col, a.N - 1) * K + kg * 4;
  for (int tile0 = a.mt0; tile0 < a.mt1; tile0 += 2) {
    const bool two = tile0 + 1 < a.mt1;
    const float* ap0 = A + (size_t)(tile0 * 16 + col) * lda + kg * 4;
    const float* ap1 = ap0 + (size_t)16 * lda;
    floatx4 acc0 = {0.f, 0.f, 0.f, 0.f}, acc1 = {0.f, 0.f, 0.f, 0.f};
    for (int st = s0; st < s1; st += U) {
      float4 bw[U], a0[U], a1[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int k = min(st + u, s1 - 1) * 16;
        bw[u] = *reinterpret_cast<const float4*>(wp + k);
        a0[u] = *reinterpret_cast<const float4*>(ap0 + k);
        if (two) a1[u] = *reinterpret_cast<const float4*>(ap1 + k);
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (st + u < s1) {
          acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[u].x, bw[u].x, acc0, 0, 0, 0);
          acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[u].y, bw[u].y, acc0, 0, 0, 0);
          acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[u].z, bw[u].z, acc0, 0, 0, 0);
          acc0 = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[u].w, bw[u].w, acc0, 0, 0, 0);
          if (two) {
            acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[u].x, bw[u].x, acc1, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[u].y, bw[u].y, acc1, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[u].z, bw[u].z, acc1, 0, 0, 0);
            acc1 = __builtin_amdgcn_mfma_f32_16x16x4f32(a1[u].w, bw[u].w, acc1, 0, 0, 0);
          }
        }
    }
    __syncthreads();
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      red[wv][kg * 4 + v][col] = acc0[v];
      red[wv][16 + kg * 4 + v][col] = acc1[v];
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < 32 * 16; idx += NW * 64) {
      const int ml = idx >> 4, c = idx & 15;
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < NW; ++w) s += red[w][ml][c];
      sv[ml][c] = s;
    }
    __syncthreads();
    {
      RowsPre<32, 16, NW * 64> none;
      finish_tile<float, EPI, 32, 16, NW * 64>(a, sv, ov, oz, tile0 * 16, nb, pre, none);
    }
  }
}

// ---------------------------------------------------------------- weight repack
// Row-major [N][K] bf16 -> fragment order; columns beyond N are zero.
__global__ void __launch_bounds__(256) k_repack(const bf16* __restrict__ src, bf16* __restrict__ dst, int N, int K,
                                                int kind, size_t chunks) {
  const size_t c = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (c >= chunks) return;
  const int lane = (int)(c & 63);
  size_t rest = c >> 6;
  int n, k;
  if (kind == W_F16) {
    const int KS = K / 32;
    const int ks = (int)(rest % KS), tile = (int)(rest / KS);
    n = tile * 16 + (lane & 15);
    k = ks * 32 + 8 * (lane >> 4);
  } else {
    const int KS = K / 16;
    const int ks = (int)(rest % KS), tile = (int)(rest / KS);
    n = tile * 32 + (lane & 31);
    k = ks * 16 + 8 * (lane >> 5);
  }
  uint4 v = make_uint4(0u, 0u, 0u, 0u);
  if (n < N) v = *reinterpret_cast<const uint4*>(src + (size_t)n * K + k);
  *reinterpret_cast<uint4*>(dst + c * 8) = v;
}

// ---------------------------------------------------------------- LayerNorm column sums
// One wave per row n of w: c[n] = sum_k g[k] w[n][k], e[n] = sum_k b[k] w[n][k] in fp64.
__global__ void __launch_bounds__(256) k_ln_fold_cols(const bf16* __restrict__ w, const bf16* __restrict__ g,
                                                      const bf16* __restrict__ b, int N, int K, float* __restrict__ c,
                                                      float* __restrict__ e) {
  const int lane = threadIdx.x & 63, n = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (n >= N) return;
  double sc = 0.0, se = 0.0;
  for (int k = lane; k < K; k += 64) {
    const double wv = (double)to_f(w[(size_t)n * K + k]);
    sc += (double)to_f(g[k]) * wv;
    se += (double)to_f(b[k]) * wv;
  }
  for (int o = 32; o > 0; o >>= 1) {
    sc += __shfl_xor(sc, o);
    se += __shfl_xor(se, o);
  }
  if (lane == 0) {
    c[n] = (float)sc;
    e[n] = (float)se;
  }
}

void ln_fold_cols(const void* w, const void* g, const void* b, int N, int K, float* c, float* e, hipStream_t st) {
  k_ln_fold_cols<<<(N + 3) / 4, 256, 0, st>>>(reinterpret_cast<const bf16*>(w), reinterpret_cast<const bf16*>(g),
                                              reinterpret_cast<const bf16*>(b), N, K, c, e);
}

// ---------------------------------------------------------------- launchers
template <int EPI, int NW>
static void launch_bf16(const GemvArgs& a, hipStream_t st) {
  if (a.wkind == W_F32) {
    k_gemv32<EPI, NW><<<(a.N + 31) / 32, NW * 64, 0, st>>>(a);
  } else {
    k_gemv16<EPI, NW><<<(a.N + 15) / 16, NW * 64, 0, st>>>(a);
  }
}
template <int EPI, int NW>
static void launch_f32(const GemvArgs& a, hipStream_t st) {
  k_gemv_f32<EPI, NW><<<(a.N + 15) / 16, NW * 64, 0, st>>>(a);
}

// 16 waves: one row of the LayerNorm per wave; K <= kLnFoldMaxK gives at most
// kLnFoldMaxK / 16 / 16 = 5 k-steps per wave.
constexpr int kLnWaves = 16;
constexpr int kLnSteps = kLnFoldMaxK / 16 / kLnWaves;      // 32-column tiles: k-steps of 16 per wave
constexpr int kLnSteps16 = (kLnFoldMaxK / 32 + kLnWaves - 1) / kLnWaves;  // 16-column tiles: k-steps of 32
template <int EPI>
static void launch_ln(const GemvArgs& a, hipStream_t st) {
  if (a.wkind == W_F32) {
    k_gemv32_ln<EPI, kLnWaves, kLnSteps><<<(a.N + 31) / 32, kLnWaves * 64, 0, st>>>(a);
  } else {
    k_gemv16_ln<EPI, kLnWaves, kLnSteps16><<<(a.N + 15) / 16, kLnWaves * 64, 0, st>>>(a);
  }
}

// Batch 1, bf16, split-K (EPI_ACC or EPI_PART): 64-column blocks, k split over
// grid y; the straight-line kernel when each wave's k-steps fit one batch.
template <int EPI>
static void launch_splitk(const GemvArgs& a, hipStream_t st) {
  const int ntile = (a.N + 15) / 16, ks = a.ksplit > 1 ? a.ksplit : 1;
  const dim3 grid((ntile + 3) / 4, ks);
  const int KS = a.K / 32, kss = (KS + ks - 1) / ks, spw = (kss + 7) / 8;
  if (a.nsplit == 3 && a.mt1 - a.mt0 == 2) {
    if (spw <= 1) { k_gemv16k<EPI, 8, 4, 1><<<grid, 512, 0, st>>>(a); return; }
    if (spw <= 2) { k_gemv16k<EPI, 8, 4, 2><<<grid, 512, 0, st>>>(a); return; }
    if (spw <= 4) { k_gemv16k<EPI, 8, 4, 4><<<grid, 512, 0, st>>>(a); return; }
  }
  k_gemv16w<EPI, 8, 4><<<grid, 512, 0, st>>>(a);
}

// blocks appended to a staged several-slot GEMM launch for the weights it reads ahead
static unsigned pf_blocks(const GemvArgs& a) { return (unsigned)a.pf.blocks; }

template <typename S, int EPI>
static void launch_epi(const GemvArgs& a, hipStream_t st) {
  if constexpr (EPI == EPI_ACC) {  // bf16: split-K partial sums added to y
    if constexpr (sizeof(S) == 2) {
      if (a.nsplit == 2 && a.wkind == W_F16) {  // several slots: GEMM tiles, k split over grid y
        const int mb0 = a.slot0 * kRows / 64, mb1 = ((a.slot0 + a.nslots) * kRows + 63) / 64;
        const int nmb = mb1 - mb0, nnb = (a.N + 63) / 64, ks = a.ksplit > 1 ? a.ksplit : 1;
        const unsigned nb = gemm_grid(nmb, nnb);
        if (nb * (unsigned)ks >= kGemmStagedBlocks) k_gemm16s<EPI><<<dim3(nb + pf_blocks(a), ks), 256, 0, st>>>(a, mb0, nmb, nnb);
        else k_gemm16<EPI><<<dim3(nb, ks), 256, 0, st>>>(a, mb0, nmb, nnb);
      } else {
        launch_splitk<EPI_ACC>(a, st);  // batch 1
      }
    }
    return;
  } else {
  if constexpr (sizeof(S) == 2) {
    if constexpr (EPI == EPI_ARGMAX) {  // batch-1 vocabulary head: persistent blocks
      if (a.nsplit == 3 && a.wkind == W_F32 && a.mt1 - a.mt0 == 1 && (a.K / 16 + 7) / 8 <= kU) {
        const int ntile = (a.N + 31) / 32, per = (ntile + kHeadBlocks - 1) / kHeadBlocks;
        if (a.lnx != nullptr) k_gemv32p<EPI, 8, kU, true><<<(ntile + per - 1) / per, 512, 0, st>>>(a);
        else k_gemv32p<EPI, 8, kU, false><<<(ntile + per - 1) / per, 512, 0, st>>>(a);
        return;
      }
    }
    if (a.lnx != nullptr) {
      launch_ln<EPI>(a, st);
      return;
    }
    const int ks = a.ksplit > 1 ? a.ksplit : 1;
    if (a.nsplit == 2 && a.wkind == W_F16) {  // several slots: 64 x 64 GEMM tiles (k split over grid y)
      const int mb0 = a.slot0 * kRows / 64, mb1 = ((a.slot0 + a.nslots) * kRows + 63) / 64;
      const int nmb = mb1 - mb0, nnb = (a.N + 63) / 64;
      if constexpr (EPI == EPI_PART) {
        // many rows, k split into partial sums: wide tiles, grid y = the splits
        const int kss = a.K / 32;
        if (ks > 1 && nmb >= kWideMinRowBlocks && kss % (ks * kWideD) == 0 && a.N % 320 == 0 && a.a.kind == OP_F16) {
          k_gemm32r<EPI, 10><<<dim3(wide_grid(nmb, a.N / 320) + pf_blocks(a), ks), 256, 0, st>>>(a, mb0, nmb, a.N / 320);
          return;
        }
      }
      if constexpr (EPI == EPI_STORE || EPI == EPI_GELU || EPI == EPI_RESID || EPI == EPI_QKV) {
        // many rows: wide tiles on the 32x32x16 matrix instruction
        if (ks == 1 && nmb >= kWideMinRowBlocks && (a.K / 32) % kWideD == 0 && a.N % 8 == 0 && a.a.kind == OP_F16) {
          GemvArgs b = a;
          b.pf = Touch{nullptr, 0, 0};  // these launches append no reading blocks
          if (a.N % 320 == 0 && a.N / 320 >= 16) {
            k_gemm32r<EPI, 10><<<wide_grid(nmb, a.N / 320), 256, 0, st>>>(b, mb0, nmb, a.N / 320);
            return;
          }
          if (a.N % 256 == 0 && a.N >= 2560) {
            k_gemm32r<EPI, 8><<<wide_grid(nmb, a.N / 256), 256, 0, st>>>(b, mb0, nmb, a.N / 256);
            return;
          }
          // narrower products (1280 columns at 96 slots) measured slower in this kernel
          // (128-column tiles: 33 against 17.5 us per launch) and keep the 64 x 64 tiles
        }
      }
      // LDS-staged fragments once the launch has enough blocks to cover the
      // chip; with fewer, the per-k-step barrier costs more than the halved loads
      // save (measured: 72-240 blocks at 16 slots 12-15% slower, 280+ at 96
      // slots 6-32% faster)
      const unsigned nb = gemm_grid(nmb, nnb);
      if constexpr (EPI != EPI_ARGMAX) {
        if (nb * (unsigned)ks >= kGemmStagedBlocks) {
          k_gemm16s<EPI><<<dim3(nb + pf_blocks(a), ks), 256, 0, st>>>(a, mb0, nmb, nnb);
          return;
        }
      }
      k_gemm16<EPI><<<dim3(nb, ks), 256, 0, st>>>(a, mb0, nmb, nnb);
      return;
    }
    if constexpr (EPI == EPI_PART) {  // batch 1
      launch_splitk<EPI_PART>(a, st);
      return;
    }
  }
  // waves per block: enough that each wave's share of the k-steps fits one batch
  const int kstep = sizeof(S) == 4 ? 16 : (a.wkind == W_F32 ? 16 : 32);
  const int steps = a.K / kstep;
  if constexpr (sizeof(S) == 4) {
    if (steps <= 4 * kU) launch_f32<EPI, 4>(a, st);
    else if (steps <= 8 * kU || EPI == EPI_ARGMAX) launch_f32<EPI, 8>(a, st);  // the head's epilogue needs > 128 VGPRs
    else launch_f32<EPI, EPI == EPI_ARGMAX ? 8 : 16>(a, st);
  } else {
    if (steps <= 4 * kU) launch_bf16<EPI, 4>(a, st);
    else if (steps <= 8 * kU) launch_bf16<EPI, 8>(a, st);
    else launch_bf16<EPI, 16>(a, st);
  }
  }
}

template <typename S>
void Ops<S>::gemv(int epi, const GemvArgs& a0, hipStream_t st) {
  // the staged GEMM takes the last pf.blocks blocks of grid x as reading blocks
  // (other kernels ignore the request): a request with nothing to read appends none
  GemvArgs a = a0;
  if (a.pf.p == nullptr || a.pf.bytes < 16 || a.pf.blocks <= 0) a.pf = Touch{nullptr, 0, 0};
  switch (epi) {
    case EPI_STORE: launch_epi<S, EPI_STORE>(a, st); break;
    case EPI_GELU: launch_epi<S, EPI_GELU>(a, st); break;
    case EPI_RESID: launch_epi<S, EPI_RESID>(a, st); break;
    case EPI_QKV: launch_epi<S, EPI_QKV>(a, st); break;
    case EPI_ARGMAX: launch_epi<S, EPI_ARGMAX>(a, st); break;
    case EPI_PART: launch_epi<S, EPI_PART>(a, st); break;
    case EPI_ACC: launch_epi<S, EPI_ACC>(a, st); break;
  }
}

template <>
void repack<bf16>(const void* src, void* dst, int N, int K, int wkind, hipStream_t st) {
  const int tile = wkind == W_F32 ? 32 : 16;
  const size_t npad = (size_t)(N + tile - 1) / tile * tile;
  const size_t chunks = npad * K / 8;
  k_repack<<<(unsigned)((chunks + 255) / 256), 256, 0, st>>>(reinterpret_cast<const bf16*>(src),
                                                                reinterpret_cast<bf16*>(dst), N, K, wkind, chunks);
}
template <>
void repack<float>(const void*, void*, int, int, int, hipStream_t) {}

template void Ops<float>::gemv(int, const GemvArgs&, hipStream_t);
template void Ops<bf16>::gemv(int, const GemvArgs&, hipStream_t);

}  // namespace wf
