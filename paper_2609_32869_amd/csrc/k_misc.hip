// Small kernels of the draft-and-verify step (gfx950, wave64): LayerNorm into a
// matrix operand, pass set-up, argmax, acceptance, drafter-history write and the
// encode-time cross K/V product.
//
// Rows: a pass over slot s uses activation rows s*9 + i, i = 0..8 (anchor plus
// eight candidates, or eight masks for the drafter).  Every kernel here computes a
// row's result the same way however many rows or slots share the launch, except
// the LayerNorm operand launch, which sums a row's statistics in another order
// from kLnColMaxRows rows on (as the products' kernels and k-splits also change
// with the slot count).
#include "../../include/wf.h"
#include "wf_operand.h"

namespace wf {

// ---------------------------------------------------------------- LayerNorm -> operand
// y = g * (x - mean) / sqrt(var + 1e-5) + b over the d columns of a row (Whisper's
// pre-LN blocks and final LN), written as the operand of the next product.  One
// wave per row, four rows per block: a lane holds 8 consecutive columns of each of
// its chunks (lane, lane + 64, ...; d <= 2048), loaded and written 16 bytes at a
// time, and the statistics are wave sums (no barrier).
constexpr int kLnRowsPerBlock = 4;
template <typename S>
__global__ void __launch_bounds__(64 * kLnRowsPerBlock) k_ln_operand(LnArgs a) {
  StampScope stamp_scope(a.stamp, 64 * kLnRowsPerBlock);
  constexpr int J = 2048 / 8 / 64;
  const int lane = threadIdx.x & 63;
  const int row = a.row0 + blockIdx.x * kLnRowsPerBlock + (int)(threadIdx.x >> 6);
  if (row >= a.row0 + a.rows) return;
  const int nch = a.d >> 3;
  const float* xr = a.x + (size_t)row * a.d;
  // every load first and unconditionally (chunks past the row re-read the last one)
  float v[J][8], gv[J][8], bv[J][8];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = min(lane + 64 * j, nch - 1);
    ld8(xr + 8 * c, v[j]);
    ld8(reinterpret_cast<const S*>(a.g) + 8 * c, gv[j]);
    ld8(reinterpret_cast<const S*>(a.b) + 8 * c, bv[j]);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j)
    if (lane + 64 * j < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) s += v[j][e];
  const float mean = wave_sum(s) / (float)a.d;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j)
    if (lane + 64 * j < nch)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float c = v[j][e] - mean;
        q += c * c;
      }
  const float inv = 1.0f / sqrtf(wave_sum(q) / (float)a.d + 1e-5f);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = lane + 64 * j;
    if (c < nch) {
      float y[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = (v[j][e] - mean) * inv * gv[j][e] + bv[j][e];
      put_op8<S>(a.out, a.nsplit, a.R9, row, 8 * c, y);
    }
  }
}

// The same LayerNorm with one block of three waves per row (d <= 1536), a thread
// holding 8 consecutive columns, statistics as wave sums merged in LDS: for
// launches of fewer than kLnColMaxRows rows, which the wave-per-row kernel
// spreads over too few CUs (144 rows: 3.7 against 5.0 us; 864 rows: 7.8
// against 6.9, where the four-row blocks already cover the chip).
constexpr int kLnColThreads = 192;
constexpr int kLnColMaxRows = 512;
template <typename S>
__global__ void __launch_bounds__(kLnColThreads) k_ln_operand_cols(LnArgs a) {
  StampScope stamp_scope(a.stamp, kLnColThreads);
  constexpr int NW = kLnColThreads / 64;
  __shared__ float red[2][NW];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int row = a.row0 + blockIdx.x, nch = a.d >> 3, c = threadIdx.x, cc = min(c, nch - 1);
  const bool act = c < nch;
  float v[8], gv[8], bv[8];
  ld8(a.x + (size_t)row * a.d + 8 * cc, v);
  ld8(reinterpret_cast<const S*>(a.g) + 8 * cc, gv);
  ld8(reinterpret_cast<const S*>(a.b) + 8 * cc, bv);
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) s += act ? v[e] : 0.f;
  s = wave_sum(s);
  if (lane == 0) red[0][w] = s;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) tot += red[0][i];
  const float mean = tot / (float)a.d;
  float q = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float cd = v[e] - mean;
    q += act ? cd * cd : 0.f;
  }
  q = wave_sum(q);
  if (lane == 0) red[1][w] = q;
  __syncthreads();
  float qt = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) qt += red[1][i];
  const float inv = 1.0f / sqrtf(qt / (float)a.d + 1e-5f);
  if (act) {
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = (v[e] - mean) * inv * gv[e] + bv[e];
    put_op8<S>(a.out, a.nsplit, a.R9, row, 8 * c, y);
  }
}

// ---------------------------------------------------------------- streamed matrix-core GEMV
// Y[row, n] = sum_k X[row, k] W[n, k] for the 9 rows of each slot of the batch.
// Block = 4 waves and 16 output columns; wave w takes a contiguous quarter of K.
// Lane (col = lane % 16, kg = lane / 16) streams 16-byte chunks of weight row
// n0 + col (8 per round in flight) as the B operand of v_mfma_f32_16x16x32_bf16

// final argmax over the per-block partials of each row; flags non-finite maxima.
// Drafter pass (keep != null): rows 1..K of slot s are the drafted tokens, also
// stored to keep[s * K + j] and, if given, dst[(s - slot0) * K + j].
constexpr int kArgmaxLoads = 8;
__global__ void __launch_bounds__(256) k_argmax_final(const float* __restrict__ hv, const int* __restrict__ hi,
                                                      int nblk, int row0, int* __restrict__ g,
                                                      float* __restrict__ gmax, unsigned* status, int* keep, int* dst,
                                                      int slot0, int K, const float* __restrict__ hm,
                                                      const float* __restrict__ hs, float* rmax, float* rsum) {
  __shared__ float bvs[4];
  __shared__ int bis[4];
  __shared__ float ms[4], ss[4];
  const int row = row0 + blockIdx.x;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  float zm = -INFINITY, zs = 0.f;  // normaliser over this thread's blocks
  for (int j0 = threadIdx.x; j0 < nblk; j0 += 256 * kArgmaxLoads) {
    float v[kArgmaxLoads], bm[kArgmaxLoads], bs[kArgmaxLoads];
    int ix[kArgmaxLoads];
#pragma unroll
    for (int u = 0; u < kArgmaxLoads; ++u) {
      const int j = j0 + 256 * u;
      v[u] = j < nblk ? hv[(size_t)row * nblk + j] : -INFINITY;
      ix[u] = j < nblk ? hi[(size_t)row * nblk + j] : 0x7fffffff;
      bm[u] = (hm != nullptr && j < nblk) ? hm[(size_t)row * nblk + j] : -INFINITY;
      bs[u] = (hm != nullptr && j < nblk) ? hs[(size_t)row * nblk + j] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < kArgmaxLoads; ++u) {
      if (better(v[u], ix[u], bv, bi)) { bv = v[u]; bi = ix[u]; }
      if (bm[u] > -INFINITY) {
        const float mn = fmaxf(zm, bm[u]);
        zs = zs * expf(zm - mn) + bs[u] * expf(bm[u] - mn);
        zm = mn;
      }
    }
  }
  if (hm != nullptr) {
    // fixed-order combine: within the wave, then across the four waves
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float om = __shfl_xor(zm, o, 64), os = __shfl_xor(zs, o, 64);
      const float mn = fmaxf(zm, om);
      if (mn > -INFINITY) {
        zs = zs * expf(zm - mn) + os * expf(om - mn);
        zm = mn;
      }
    }
    if ((threadIdx.x & 63) == 0) {
      ms[threadIdx.x >> 6] = zm;
      ss[threadIdx.x >> 6] = zs;
    }
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
    if (hm != nullptr && rmax != nullptr) {
      float M = ms[0];
      for (int j = 1; j < 4; ++j) M = fmaxf(M, ms[j]);
      float Ssum = 0.f;
      for (int j = 0; j < 4; ++j) Ssum += ss[j] * expf(ms[j] - M);
      rmax[row] = M;
      rsum[row] = Ssum;
    }
    const int slot = row / kRows, i = row - slot * kRows;
    if (keep != nullptr && i >= 1 && i <= K) {
      keep[(size_t)slot * K + i - 1] = bis[0];
      if (dst != nullptr) dst[(size_t)(slot - slot0) * K + i - 1] = bis[0];
    }
  }
}

// ---------------------------------------------------------------- attention helpers


// ---------------------------------------------------------------- pass set-up
// Rows of a pass: h[slot * 9 + i] = E[toks[i]] + P[pos[i]] (target) or E[anchor] /
// mask vector (drafter).  A slot's rows are split over kBeginGroups blocks by
// 8-column chunks (block g takes chunks [g nch / G, (g + 1) nch / G)), every
// load of a thread issued before the first add; each block works out the pass's
// tokens and positions itself, and block 0 alone writes the slot's state.
constexpr int kBeginGroups = 8;
constexpr int kBeginTasks = 2;  // chunk tasks per thread: 9 rows * 2048 / 8 / 8 / 256, rounded up
struct BeginCols {
  int cb, ce;  // this block's 8-column chunks
  __device__ __forceinline__ BeginCols(int d) {
    const int nch = d >> 3;
    cb = (int)blockIdx.y * nch / kBeginGroups;
    ce = ((int)blockIdx.y + 1) * nch / kBeginGroups;
  }
};
template <typename S>
__device__ __forceinline__ void fill_rows(const BeginArgs& a, int slot, const int* toks, const int* poss, bool mask_rows,
                                          BeginCols bc) {
  const S* E = reinterpret_cast<const S*>(a.emb);
  const S* P = reinterpret_cast<const S*>(a.pos);
  const int nc = max(bc.ce - bc.cb, 1);
  float e8[kBeginTasks][8], p8[kBeginTasks][8];
  // every load unconditionally (tasks past the nine rows re-read row 8), so all
  // chunks are in flight together; rows that take no embedding / no position
  // read one anyway and zero it below
#pragma unroll
  for (int j = 0; j < kBeginTasks; ++j) {
    const int t = threadIdx.x + 256 * j, i = min(t / nc, kRows - 1), c = 8 * min(bc.cb + t % nc, (a.d >> 3) - 1);
    const int tok = toks[i];
    const size_t ei = a.emb_kind == W_F32   ? wfrag32_index(tok, c, a.d / 16)
                      : a.emb_kind == W_F16 ? wfrag16_index(tok, c, a.d / 32)
                                            : (size_t)tok * a.d + c;
    ld8(E + ei, e8[j]);
    ld8(mask_rows ? P + c : P + (size_t)poss[i] * a.d + c, p8[j]);
  }
#pragma unroll
  for (int j = 0; j < kBeginTasks; ++j) {
    const int t = threadIdx.x + 256 * j, i = t / nc;
    if (mask_rows) {  // draft block: row 0 is the anchor's embedding, rows 1.. the mask vector
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if (i > 0) e8[j][e] = 0.f;
        else p8[j][e] = 0.f;
      }
    }
  }
#pragma unroll
  for (int j = 0; j < kBeginTasks; ++j) {
    const int t = threadIdx.x + 256 * j, i = t / nc, c = 8 * (bc.cb + t % nc);
    if (i < kRows && bc.ce > bc.cb) {
      float* hr = a.h + (size_t)(slot * kRows + i) * a.d + c;
      *reinterpret_cast<float4*>(hr) = make_float4(e8[j][0] + p8[j][0], e8[j][1] + p8[j][1], e8[j][2] + p8[j][2], e8[j][3] + p8[j][3]);
      *reinterpret_cast<float4*>(hr + 4) =
          make_float4(e8[j][4] + p8[j][4], e8[j][5] + p8[j][5], e8[j][6] + p8[j][6], e8[j][7] + p8[j][7]);
    }
  }
}

// Pages of the nine rows of a pass starting at pos0 (they span at most two).
__device__ __forceinline__ void set_pass_pages(const BeginArgs& a, int slot, int* st, int pos0) {
  const int* pt = a.page_table + slot * a.pages_per_slot;
  const int p = min(max(pos0, 0) >> 4, a.pages_per_slot - 1);
  st[ST_PG0] = pt[p];
  st[ST_PG1] = pt[min(p + 1, a.pages_per_slot - 1)];
}

// Zeroes the block's columns of the slot's nine history-projection rows (a.hp).
__device__ __forceinline__ void clear_hp(const BeginArgs& a, int slot, BeginCols bc) {
  if (a.hp == nullptr) return;
  const int n4 = 2 * (bc.ce - bc.cb);  // float4 per row
  for (int t = threadIdx.x; t < kRows * n4; t += blockDim.x) {
    const int i = t / n4, q = t - i * n4;
    reinterpret_cast<float4*>(a.hp + (size_t)(slot * kRows + i) * a.d + 8 * bc.cb)[q] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// Verify rows: [anchor, c_1..c_k] at positions L..L+k with the budget rule
// k = min(K, k_max, max_new - emitted - 1, n_ctx - L - 1) (Appendix A.1).
template <typename S>
__global__ void __launch_bounds__(256) k_verify_begin(BeginArgs a) {
  __shared__ int toks[kRows], poss[kRows];
  const int slot = a.slot0 + blockIdx.x;
  const BeginCols bc(a.d);
  const bool lead = blockIdx.y == 0;  // writes the slot's state, tokens and status
  clear_hp(a, slot, bc);
  int* st = a.state + slot * kStateInts;
  const int L = st[ST_L], left = st[ST_MAX_NEW] - st[ST_EMITTED], anchor = st[ST_ANCHOR];
  const bool go = st[ST_LIVE] && !st[ST_DONE] && left > 0 && L < a.n_ctx;
  const int nv = go ? min(min(a.block_k, a.k_max), min(left - 1, a.n_ctx - L - 1)) + 1 : 0;
  // the acceptance marks a slot finished once its cache reaches n_ctx, so a live,
  // unfinished slot at or beyond it has an inconsistent state: its pass is refused
  if (lead && threadIdx.x == 0 && a.status && st[ST_LIVE] && !st[ST_DONE] && left > 0 && L >= a.n_ctx)
    atomicOr(a.status, WF_STATUS_POSITION_OVERFLOW);
  if (threadIdx.x < kRows) {
    const int i = threadIdx.x;
    int t = (i == 0 || i >= nv) ? anchor : a.draft[(size_t)blockIdx.x * a.block_k + i - 1];
    t = min(max(t, 0), a.n_vocab - 1);
    toks[i] = t;
    poss[i] = min(L + i, a.n_ctx - 1);
    if (lead) a.tok[slot * kRows + i] = t;
  }
  __syncthreads();  // every read of the slot's state is done before block 0 writes it
  if (lead && threadIdx.x == 0) {
    st[ST_POS0] = L;
    st[ST_NV] = nv;
    set_pass_pages(a, slot, st, L);
  }
  fill_rows<S>(a, slot, toks, poss, false, bc);
}

// Draft block X_t = [Emb(y_t), m, ..., m] (Eq. 2).  The drafter history already
// holds every verified position (it is written at the end of each verify).
template <typename S>
__global__ void __launch_bounds__(256) k_draft_begin(BeginArgs a) {
  __shared__ int toks[kRows];
  const int slot = a.slot0 + blockIdx.x;
  const BeginCols bc(a.d);
  int* st = a.state + slot * kStateInts;
  if (threadIdx.x < kRows) toks[threadIdx.x] = min(max(st[ST_ANCHOR], 0), a.n_vocab - 1);
  __syncthreads();
  fill_rows<S>(a, slot, toks, nullptr, true, bc);
  if (a.pos2 != nullptr) {  // absolute-position variant: + P[t + i] on row i
    __syncthreads();
    const S* P = reinterpret_cast<const S*>(a.pos2);
    const int L = st[ST_L], w = 8 * (bc.ce - bc.cb);
    for (int idx = threadIdx.x; idx < kRows * w; idx += 256) {
      const int i = idx / w, col = 8 * bc.cb + idx - i * w;
      a.h[(size_t)(slot * kRows + i) * a.d + col] += to_f(P[(size_t)min(L + i, a.n_ctx - 1) * a.d + col]);
    }
  }
}

// Prefill chunk c: prompt positions 9c..9c+8 of each slot.
template <typename S>
__global__ void __launch_bounds__(256) k_prefill_begin(BeginArgs a) {
  __shared__ int toks[kRows], poss[kRows];
  const int slot = a.slot0 + blockIdx.x;
  const BeginCols bc(a.d);
  const bool lead = blockIdx.y == 0;  // writes the slot's state and tokens
  clear_hp(a, slot, bc);
  int* st = a.state + slot * kStateInts;
  const int len = st[ST_LEN];
  const int pos0 = a.chunk * kRows;
  const int nv = max(0, min(kRows, len - pos0));
  if (threadIdx.x < kRows) {
    const int i = threadIdx.x;
    int t = (i < nv) ? a.draft[(size_t)blockIdx.x * a.pmax + pos0 + i] : 0;
    t = min(max(t, 0), a.n_vocab - 1);
    toks[i] = t;
    poss[i] = min(pos0 + i, a.n_ctx - 1);
    if (lead) a.tok[slot * kRows + i] = t;
  }
  __syncthreads();  // every read of the slot's state is done before block 0 writes it
  if (lead && threadIdx.x == 0) {
    st[ST_POS0] = pos0;
    st[ST_NV] = nv;
    st[ST_HPOS] = pos0;
    st[ST_HN] = nv;
    set_pass_pages(a, slot, st, pos0);
  }
  fill_rows<S>(a, slot, toks, poss, false, bc);
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
  if (r >= hn) return;
  if (pos >= a.n_ctx) {  // never reached by a consistent state (the budget keeps passes below n_ctx)
    if (threadIdx.x == 0 && a.status) atomicOr(a.status, WF_STATUS_POSITION_OVERFLOW);
    return;
  }
  const int layer = blockIdx.z;
  const float* kr = a.kv + layer * a.kv_stride + (size_t)(slot * kRows + r) * 2 * a.d;
  const float* vr = kr + a.d;
  S* Kh = reinterpret_cast<S*>(a.kcache) + layer * a.cache_stride;
  S* Vh = reinterpret_cast<S*>(a.vcache) + layer * a.cache_stride;
  for (int t = threadIdx.x; t < a.n_head * 32; t += 256) {
    const int head = t >> 5, j = t & 31;
    const float c = a.use_rope ? a.rope[(pos * 32 + j) * 2] : 1.f, sn = a.use_rope ? a.rope[(pos * 32 + j) * 2 + 1] : 0.f;
    const float k1 = kr[head * kHeadDim + j], k2 = kr[head * kHeadDim + j + 32];
    const size_t base = (((size_t)slot * a.n_head + head) * a.n_ctx + pos) * kHeadDim;
    Kh[base + j] = from_f<S>(k1 * c - k2 * sn);
    Kh[base + j + 32] = from_f<S>(k1 * sn + k2 * c);
    Vh[base + j] = from_f<S>(vr[head * kHeadDim + j]);
    Vh[base + j + 32] = from_f<S>(vr[head * kHeadDim + j + 32]);
  }
}

// ---------------------------------------------------------------- acceptance
// Greedy longest-prefix rule (Section 3.1) with the end-of-transcript rule and
// the cache/anchor update of Appendix A.1.  One thread per slot.
__global__ void k_accept_greedy(AcceptArgs a) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= a.n) return;
  const int slot = a.slot0 + s;
  int* st = a.state + slot * kStateInts;
  // every read before the first branch or store (the stores below may alias)
  const int nv = st[ST_NV], live = st[ST_LIVE], L = st[ST_L], emitted = st[ST_EMITTED];
  const int max_new = st[ST_MAX_NEW], step = st[ST_STEP];
  int tok[kRows], g[kRows];
#pragma unroll
  for (int i = 0; i < kRows; ++i) {
    tok[i] = a.tok[slot * kRows + i];
    g[i] = a.g[slot * kRows + i];
  }
  const int K = a.block_k;
  int* out = a.out ? a.out + (size_t)s * (K + 1) : nullptr;
  if (nv == 0) {
    if (a.n_out) a.n_out[s] = 0;
    if (a.n_acc) a.n_acc[s] = 0;
    if (a.done) a.done[s] = live ? 1 : 0;
    if (live) st[ST_DONE] = 1;
    st[ST_HN] = 0;
    return;
  }
  const int k = nv - 1;
  int acc = 0;
  while (acc < k && tok[acc + 1] == g[acc]) ++acc;
  // accepted candidates up to and including the first end-of-transcript one
  int nacc = acc;
  bool eos_acc = false;
  for (int e = 0; e < acc; ++e)
    if (tok[e + 1] == a.eos) {
      nacc = e + 1;
      eos_acc = true;
      break;
    }
  int nemit, last;
  bool fin;
  if (eos_acc) {  // the transcript ends inside the accepted prefix: no correction token
    nemit = nacc;
    acc = nacc;
    last = tok[nacc];
    fin = true;
  } else {
    nemit = acc + 1;
    last = g[acc];
    fin = last == a.eos;
  }
  st[ST_HPOS] = L;
  st[ST_HN] = nv;
  st[ST_L] = L + 1 + acc;
  st[ST_ANCHOR] = last;
  st[ST_EMITTED] = emitted + nemit;
  st[ST_STEP] = step + 1;
  st[ST_K] = k;
  st[ST_A] = acc;
  const bool done = fin || emitted + nemit >= max_new || L + 1 + acc >= a.n_ctx;
  st[ST_DONE] = done;
  if (out) {
#pragma unroll
    for (int j = 0; j < kRows; ++j)
      if (j <= K) out[j] = j < acc ? tok[j + 1] : j == acc && !eos_acc ? last : -1;
  }
  if (a.n_out) a.n_out[s] = nemit;
  if (a.n_acc) a.n_acc[s] = acc;
  if (a.done) a.done[s] = done;
}

// ---------------------------------------------------------------- sampling acceptance
// Speculative rejection rule (Section 3.1, Appendix A.4) with fp32 softmaxes of the
// scaled logits: candidate c_j (drafted from q_j = draft row j) is accepted iff
// u_j * q_j(c_j) < p_{j-1}(c_j), u_j the acceptance uniform of position j - 1.  At
// the first rejection a token is drawn from (p - q)_+ (from p if that set is
// empty), after k acceptances a bonus from target row k, and with k = 0 a plain
// draw from row 0; draws are Gumbel-max.  An accepted end-of-transcript
// candidate ends the transcript with no draw.
enum { SM_NONE = 0, SM_RES = 1, SM_BON = 2, SM_PLAIN = 3 };

__device__ __forceinline__ float prob_of(const float* logits, int V, float zmax, float zsum, float inv_t, int c) {
  return expf(logits[c] * inv_t - zmax) / zsum;
}

// one thread per slot: accepted count and the draw to make
__global__ void k_sample_scan(SampleArgs a) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= a.n) return;
  const int slot = a.slot0 + s;
  const int* st = a.state + slot * kStateInts;
  int* o = a.sst + slot * 4;
  const int nv = st[ST_NV];
  if (nv == 0) {
    o[0] = SM_NONE; o[1] = 0; o[2] = 0; o[3] = -1;  // nothing verified (finished slot)
    return;
  }
  const int k = nv - 1, step = st[ST_STEP];
  const int* tok = a.tok + slot * kRows;
  const size_t V = a.V;
  int mode = k == 0 ? SM_PLAIN : SM_BON, row = k == 0 ? 0 : k, acc = k, fin = 0;
  for (int j = 0; j < k; ++j) {
    const int c = tok[j + 1];
    const int tr = slot * kRows + j, dr = slot * kRows + j + 1;
    const float q = prob_of(a.lq + dr * V, a.V, a.dmax[dr], a.dsum[dr], a.inv_t, c);
    const float p = prob_of(a.lp + tr * V, a.V, a.tmax[tr], a.tsum[tr], a.inv_t, c);
    const float u = rng_uniform(rng_word(a.seed, RNG_ACC, slot, step, 0, j));
    if (!(u * q < p)) {
      mode = SM_RES;
      row = j;
      acc = j;
      break;
    }
    if (c == a.eos) {
      mode = SM_NONE;
      acc = j + 1;
      fin = 1;
      break;
    }
  }
  o[0] = mode; o[1] = row; o[2] = acc; o[3] = fin;
}

// grid (nsb, n): Gumbel-max partials of the slot's draw over a slice of the vocabulary
constexpr int kSampleThreads = 256;
__global__ void __launch_bounds__(kSampleThreads) k_sample_draw(SampleArgs a) {
  __shared__ float sb[4][4];
  __shared__ int si[4][4];
  const int slot = a.slot0 + blockIdx.y;
  const int* o = a.sst + slot * 4;
  const int mode = o[0], row = o[1];
  if (mode == SM_NONE) return;
  const int step = a.state[slot * kStateInts + ST_STEP];
  const int V = a.V;
  const int cs = (V + a.nsb - 1) / a.nsb;
  const int v0 = blockIdx.x * cs, v1 = min(V, v0 + cs);
  const int tr = slot * kRows + row, dr = slot * kRows + row + 1;
  const float* lp = a.lp + (size_t)tr * V;
  const float* lq = a.lq + (size_t)dr * V;
  float best = -INFINITY, fb = -INFINITY;
  int bi = 0x7fffffff, fi = 0x7fffffff;
  for (int v = v0 + threadIdx.x; v < v1; v += kSampleThreads) {
    float score, fscore = -INFINITY;
    if (mode == SM_RES) {
      const float g = rng_gumbel(rng_word(a.seed, RNG_RES, slot, step, row + 1, v));
      const float p = prob_of(lp, V, a.tmax[tr], a.tsum[tr], a.inv_t, v);
      const float q = prob_of(lq, V, a.dmax[dr], a.dsum[dr], a.inv_t, v);
      const float r = p - q;
      score = r > 0.f ? logf(r) + g : -INFINITY;
      fscore = p > 0.f ? logf(p) + g : -INFINITY;
    } else {
      const int purpose = mode == SM_BON ? RNG_BON : RNG_PLAIN;
      score = lp[v] * a.inv_t + rng_gumbel(rng_word(a.seed, purpose, slot, step, 0, v));
    }
    if (better(score, v, best, bi)) { best = score; bi = v; }
    if (better(fscore, v, fb, fi)) { fb = fscore; fi = v; }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float ob = __shfl_xor(best, off, 64), of = __shfl_xor(fb, off, 64);
    const int oi = __shfl_xor(bi, off, 64), oj = __shfl_xor(fi, off, 64);
    if (better(ob, oi, best, bi)) { best = ob; bi = oi; }
    if (better(of, oj, fb, fi)) { fb = of; fi = oj; }
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sb[w][0] = best; si[w][0] = bi; sb[w][1] = fb; si[w][1] = fi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int j = 1; j < 4; ++j) {
      if (better(sb[j][0], si[j][0], best, bi)) { best = sb[j][0]; bi = si[j][0]; }
      if (better(sb[j][1], si[j][1], fb, fi)) { fb = sb[j][1]; fi = si[j][1]; }
    }
    float* pp = a.part + ((size_t)slot * a.nsb + blockIdx.x) * 4;
    pp[0] = best;
    pp[1] = __int_as_float(bi);
    pp[2] = fb;
    pp[3] = __int_as_float(fi);
  }
}

// one thread per slot: the drawn token, emitted tokens and the state update
__global__ void k_sample_final(SampleArgs a) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= a.n) return;
  const int slot = a.slot0 + s;
  int* st = a.state + slot * kStateInts;
  const int* o = a.sst + slot * 4;
  const int K = a.block_k;
  int* out = a.out ? a.out + (size_t)s * (K + 1) : nullptr;
  const int nv = st[ST_NV];
  if (nv == 0) {
    if (a.n_out) a.n_out[s] = 0;
    if (a.n_acc) a.n_acc[s] = 0;
    if (a.done) a.done[s] = st[ST_LIVE] ? 1 : 0;
    if (st[ST_LIVE]) st[ST_DONE] = 1;
    st[ST_HN] = 0;
    return;
  }
  const int mode = o[0], acc = o[2];
  bool fin = o[3] != 0;
  const int* tok = a.tok + slot * kRows;
  int nemit = 0;
  for (int e = 0; e < acc; ++e) {
    if (out) out[nemit] = tok[e + 1];
    ++nemit;
  }
  int last = acc > 0 ? tok[acc] : -1;
  if (mode != SM_NONE) {
    float best = -INFINITY, fb = -INFINITY;
    int bi = 0x7fffffff, fi = 0x7fffffff;
    for (int b = 0; b < a.nsb; ++b) {
      const float* pp = a.part + ((size_t)slot * a.nsb + b) * 4;
      if (better(pp[0], __float_as_int(pp[1]), best, bi)) { best = pp[0]; bi = __float_as_int(pp[1]); }
      if (better(pp[2], __float_as_int(pp[3]), fb, fi)) { fb = pp[2]; fi = __float_as_int(pp[3]); }
    }
    last = (mode == SM_RES && best == -INFINITY) ? fi : bi;  // empty residual: draw from p
    if (out) out[nemit] = last;
    ++nemit;
    fin = last == a.eos;
  }
  const int L = st[ST_L];
  st[ST_HPOS] = L;
  st[ST_HN] = nv;
  st[ST_L] = L + 1 + acc;
  st[ST_ANCHOR] = last;
  st[ST_EMITTED] += nemit;
  st[ST_STEP] += 1;
  st[ST_K] = nv - 1;
  st[ST_A] = acc;
  const bool done = fin || st[ST_EMITTED] >= st[ST_MAX_NEW] || st[ST_L] >= a.n_ctx;
  st[ST_DONE] = done;
  if (out)
    for (int j = nemit; j <= K; ++j) out[j] = -1;
  if (a.n_out) a.n_out[s] = nemit;
  if (a.n_acc) a.n_acc[s] = acc;
  if (a.done) a.done[s] = done;
}

// raw generator words (test entry point)
__global__ void k_rng_words(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out) {
  const int v = blockIdx.x * blockDim.x + threadIdx.x;
  if (v < n) out[v] = rng_word(seed, purpose, slot, step, pos, v);
}
void rng_words_device(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out, hipStream_t st) {
  if (n > 0) k_rng_words<<<(n + 255) / 256, 256, 0, st>>>(seed, purpose, slot, step, pos, n, out);
}

void accept_sample(const SampleArgs& a, hipStream_t st) {
  k_sample_scan<<<(a.n + 63) / 64, 64, 0, st>>>(a);
  k_sample_draw<<<dim3(a.nsb, a.n), kSampleThreads, 0, st>>>(a);
  k_sample_final<<<(a.n + 63) / 64, 64, 0, st>>>(a);
}

// ---------------------------------------------------------------- encode: cross K/V
// C[f, n] = sum_k A[f, k] W[n, k] + b[n] for the 2d key/value columns of one
// block, written to the per-head cross cache: keys frame-major [head][frame][64];
// values frame-major too, or transposed in 256-frame pieces
// [head][frame / 256][dim][256] (vt_frames frames per head) when vt_frames > 0
// (bf16 storage, read by the matrix-core cross-attention).  64x64 tiles, fp32
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
  if (a.vt_frames > 0 && n0 >= a.d) {
    // value columns of one head, stored transposed in 256-frame pieces
    // [frame / 256][dim][256]: the tile goes through LDS so that consecutive
    // threads write consecutive frames; frames from n_frames to vt_frames are
    // written as zeros
    __shared__ float Ct[64][65];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) Ct[tx * 4 + j][ty * 4 + i] = acc[i][j] + to_f(bias[n0 + tx * 4 + j]);
    __syncthreads();
    const int head = (n0 - a.d) >> 6;
    S* vt = out + (size_t)a.n_head * M * kHeadDim + (size_t)head * kHeadDim * a.vt_frames;
    for (int t = threadIdx.x; t < 64 * 64; t += 256) {
      const int dim = t >> 6, fl = t & 63, f = m0 + fl;
      if (f < a.vt_frames) vt[vt_index(dim, f)] = from_f<S>(f < M ? Ct[dim][fl] : 0.f);
    }
    return;
  }
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


// ---------------------------------------------------------------- split-K reduction + LayerNorm
// h[row] += sum over the partial products (fixed order) + bias; the new h is also
// written as the drafter tap operand when requested; then, if a gain is given,
// LayerNorm(h[row]) as the operand of the next product (same formula as the
// separate LayerNorm).  One block per row; column c of the row is thread c % 1024.
constexpr int kRlnThreads = 1024;
constexpr int kRlnMaxParts = 16;
template <typename S>
__global__ void __launch_bounds__(kRlnThreads) k_reduce_ln(RlnArgs a) {
  StampScope stamp_scope(a.stamp, kRlnThreads);
  constexpr int NW = kRlnThreads / 64;
  constexpr int J = 2;  // d <= 2048
  __shared__ float red[2][NW];
  const int row = a.row0 + blockIdx.x;
  const int d = a.d;
  const S* bias = reinterpret_cast<const S*>(a.bias);
  float* hr = a.h + (size_t)row * d;
  float v[J];
  // every load of the row is issued before the first add, unconditionally
  // (columns past d and partials past nparts re-read valid ones, then discarded)
  const bool has_bias = bias != nullptr, has_ln = a.g != nullptr;
  const void* bp = has_bias ? a.bias : a.part;
  const void* gp = has_ln ? a.g : a.part;
  const void* lp = has_ln ? a.b : a.part;
  float x[J], pv[J][kRlnMaxParts];
  uint32_t bv[J], gv[J], lv[J];
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = min((int)threadIdx.x + j * kRlnThreads, d - 1);
    x[j] = hr[c];
    bv[j] = ld_bits<S>(bp, c);
    gv[j] = ld_bits<S>(gp, c);
    lv[j] = ld_bits<S>(lp, c);
#pragma unroll
    for (int p = 0; p < kRlnMaxParts; ++p)
      pv[j][p] = a.part[min(p, a.nparts - 1) * a.pstride + (size_t)row * d + c];
  }
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = threadIdx.x + j * kRlnThreads;
    float sum = 0.f;
#pragma unroll
    for (int p = 0; p < kRlnMaxParts; ++p) sum += p < a.nparts ? pv[j][p] : 0.f;
    const float bb = has_bias ? from_bits<S>(bv[j]) : 0.f;
    v[j] = c < d ? x[j] + (sum + bb) : 0.f;  // columns past d stay out of the statistics
    if (c < d) {
      hr[c] = v[j];
      if (a.tapcol >= 0) put_op<S>(a.tap, a.nsplit, a.R9, row, a.tapcol + c, v[j]);
    }
  }
  if (a.g == nullptr) return;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float s = wave_sum(v[0] + v[1]);
  if (lane == 0) red[0][w] = s;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) tot += red[0][i];
  const float mean = tot / (float)d;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = threadIdx.x + j * kRlnThreads;
    const float cdev = v[j] - mean;
    q += c < d ? cdev * cdev : 0.f;
  }
  q = wave_sum(q);
  if (lane == 0) red[1][w] = q;
  __syncthreads();
  float qt = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) qt += red[1][i];
  const float inv = 1.0f / sqrtf(qt / (float)d + 1e-5f);
#pragma unroll
  for (int j = 0; j < J; ++j) {
    const int c = threadIdx.x + j * kRlnThreads;
    if (c < d) put_op<S>(a.out, a.nsplit, a.R9, row, c, (v[j] - mean) * inv * from_bits<S>(gv[j]) + from_bits<S>(lv[j]));
  }
}

// The same update for several slots' rows with at most kRlnRowParts partial
// buffers and d <= 8 kRlnColThreads: one block per row, a thread holding 8
// consecutive columns, loaded and written 16 bytes at a time (h, the tap and the
// operand), statistics as wave sums merged in LDS.  The sums are formed in the
// order of k_reduce_ln: h + ((p0 + p1 + ...) + bias).
constexpr int kRlnRowParts = 4;
constexpr int kRlnColThreads = 192;
template <typename S>
__global__ void __launch_bounds__(kRlnColThreads) k_reduce_ln_rows(RlnArgs a) {
  StampScope stamp_scope(a.stamp, kRlnColThreads);
  constexpr int NW = kRlnColThreads / 64;
  __shared__ float red[2][NW];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int row = a.row0 + blockIdx.x;
  const int d = a.d, nch = d >> 3, c = threadIdx.x;
  const int cc = min(c, nch - 1);
  float* hr = a.h + (size_t)row * d;
  const bool has_bias = a.bias != nullptr, has_ln = a.g != nullptr, act = c < nch;
  // every load first and unconditionally (chunks past the row and partials past
  // nparts re-read valid ones, then discarded)
  float v[8], pv[kRlnRowParts][8], bv[8], gv[8], lv[8];
  ld8(hr + 8 * cc, v);
#pragma unroll
  for (int p = 0; p < kRlnRowParts; ++p) ld8(a.part + min(p, a.nparts - 1) * a.pstride + (size_t)row * d + 8 * cc, pv[p]);
  ld8(reinterpret_cast<const S*>(has_bias ? a.bias : a.part) + 8 * cc, bv);
  ld8(reinterpret_cast<const S*>(has_ln ? a.g : a.part) + 8 * cc, gv);
  ld8(reinterpret_cast<const S*>(has_ln ? a.b : a.part) + 8 * cc, lv);
  float s = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float sum = 0.f;
#pragma unroll
    for (int p = 0; p < kRlnRowParts; ++p) sum += p < a.nparts ? pv[p][e] : 0.f;
    v[e] = act ? v[e] + (sum + (has_bias ? bv[e] : 0.f)) : 0.f;
    s += v[e];
  }
  if (act) {
    float4* y = reinterpret_cast<float4*>(hr + 8 * c);
    y[0] = make_float4(v[0], v[1], v[2], v[3]);
    y[1] = make_float4(v[4], v[5], v[6], v[7]);
    if (a.tapcol >= 0) put_op8<S>(a.tap, a.nsplit, a.R9, row, a.tapcol + 8 * c, v);
  }
  if (!has_ln) return;
  s = wave_sum(s);
  if (lane == 0) red[0][w] = s;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) tot += red[0][i];
  const float mean = tot / (float)d;
  float q = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float cd = v[e] - mean;
    q += act ? cd * cd : 0.f;
  }
  q = wave_sum(q);
  if (lane == 0) red[1][w] = q;
  __syncthreads();
  float qt = 0.f;
#pragma unroll
  for (int i = 0; i < NW; ++i) qt += red[1][i];
  const float inv = 1.0f / sqrtf(qt / (float)d + 1e-5f);
  if (act) {
    float y[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) y[e] = (v[e] - mean) * inv * gv[e] + lv[e];
    put_op8<S>(a.out, a.nsplit, a.R9, row, 8 * c, y);
  }
}

// ---------------------------------------------------------------- launchers
template <typename S>
void Ops<S>::ln_operand(const LnArgs& a, int rows, hipStream_t st) {
  LnArgs b = a;
  b.rows = rows;
  if (rows < kLnColMaxRows && a.d <= 8 * kLnColThreads && a.d % 8 == 0) {
    k_ln_operand_cols<S><<<rows, kLnColThreads, 0, st>>>(b);
    return;
  }
  k_ln_operand<S><<<(rows + kLnRowsPerBlock - 1) / kLnRowsPerBlock, 64 * kLnRowsPerBlock, 0, st>>>(b);
}
template <typename S>
void Ops<S>::reduce_ln(const RlnArgs& a, int rows, hipStream_t st) {
  if (a.nparts <= kRlnRowParts && a.d <= 8 * kRlnColThreads && a.d % 8 == 0) {
    k_reduce_ln_rows<S><<<rows, kRlnColThreads, 0, st>>>(a);
    return;
  }
  k_reduce_ln<S><<<rows, kRlnThreads, 0, st>>>(a);
}
template <typename S>
void Ops<S>::verify_begin(const BeginArgs& a, int n, hipStream_t st) { k_verify_begin<S><<<dim3(n, kBeginGroups), 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::draft_begin(const BeginArgs& a, int n, hipStream_t st) { k_draft_begin<S><<<dim3(n, kBeginGroups), 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::prefill_begin(const BeginArgs& a, int n, hipStream_t st) { k_prefill_begin<S><<<dim3(n, kBeginGroups), 256, 0, st>>>(a); }
template <typename S>
void Ops<S>::hist_write(const HistArgs& a, int n, hipStream_t st) {
  k_hist_write<S><<<dim3(kRows, n, a.nlayer > 0 ? a.nlayer : 1), 256, 0, st>>>(a);
}
template <typename S>
void Ops<S>::gemm_xkv(const XkvArgs& a, hipStream_t st) {
  const int frames = a.vt_frames > a.n_frames ? a.vt_frames : a.n_frames;  // blocks past n_frames write value padding
  k_gemm_xkv<S><<<dim3((frames + 63) / 64, 2 * a.d / 64), 256, 0, st>>>(a);
}

void argmax_final(const float* hv, const int* hi, int nblk, int row0, int rows, int* g, float* gmax,
                  unsigned* status, int* keep, int* dst, int slot0, int K, const float* hm, const float* hs, float* rmax,
                  float* rsum, hipStream_t st) {
  k_argmax_final<<<rows, 256, 0, st>>>(hv, hi, nblk, row0, g, gmax, status, keep, dst, slot0, K, hm, hs, rmax, rsum);
}
void save_last(const float* h, float* lasth, const int* state, int slot0, int n, int d, int chunk, hipStream_t st) {
  k_save_last<<<n, 256, 0, st>>>(h, lasth, state, slot0, d, chunk);
}
void prefill_finish(int* state, const int* g, int slot0, int n, int eos, int n_ctx, int* first, hipStream_t st) {
  k_prefill_finish<<<(n + 63) / 64, 64, 0, st>>>(state, g, slot0, n, eos, n_ctx, first);
}
void accept_greedy(const AcceptArgs& a, hipStream_t st) { k_accept_greedy<<<(a.n + 63) / 64, 64, 0, st>>>(a); }

#define WF_MISC_INST(S)                                                     \
  template void Ops<S>::ln_operand(const LnArgs&, int, hipStream_t);        \
  template void Ops<S>::reduce_ln(const RlnArgs&, int, hipStream_t);        \
  template void Ops<S>::verify_begin(const BeginArgs&, int, hipStream_t);   \
  template void Ops<S>::draft_begin(const BeginArgs&, int, hipStream_t);    \
  template void Ops<S>::prefill_begin(const BeginArgs&, int, hipStream_t);  \
  template void Ops<S>::hist_write(const HistArgs&, int, hipStream_t);      \
  template void Ops<S>::gemm_xkv(const XkvArgs&, hipStream_t);
WF_MISC_INST(float)
WF_MISC_INST(bf16)

// ---------------------------------------------------------------- launch timing slots
__global__ void __launch_bounds__(256) k_stamp_init(unsigned long long* s, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;  // one (start, end) pair
  if (i < n) {
    s[2 * i] = ~0ull;
    s[2 * i + 1] = 0ull;
  }
}
void stamp_init(unsigned long long* s, int n, hipStream_t st) {
  const int pairs = n * kStampWords / 2;
  k_stamp_init<<<(unsigned)((pairs + 255) / 256), 256, 0, st>>>(s, pairs);
}

}  // namespace wf
