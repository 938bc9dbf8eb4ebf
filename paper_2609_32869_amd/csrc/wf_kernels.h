// Kernel argument blocks and launchers of libwf (internal).
#pragma once
#include <hip/hip_runtime.h>

#include "wf_common.h"

namespace wf {

enum { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_QKV = 3, EPI_ARGMAX = 4, EPI_PART = 5, EPI_ACC = 6 };
// EPI_PART: split-K partial sums (no bias) of k-split blockIdx.y stored to
// y + blockIdx.y * pstride, row-major [rows][ldy].
// EPI_ACC (bf16, one slot, split-K): each k-split adds its partial sums to y
// (the residual rows) with fp32 atomic adds, the bias by k-split 0.

// Matrix-operand rows: the activation rows of a pass are stored once per split
// term, row m = s * R9 + slot * 9 + i, s < nsplit (R9 = 9 * max_batch).  With
// bf16 storage and nsplit = 3 the three bf16 terms of an fp32 value sum to it
// (24 significant bits), so bf16 matrix cores reproduce fp32 products exactly;
// with nsplit = 1 the operand is the value rounded to the storage type.
// Operand orders: row-major [rows][ld] (fp32 storage), or bf16 fragment order for
// 16x16x32 (OP_F16) or 32x32x16 (OP_F32) matrix instructions with `mt` row tiles.
enum { OP_ROW = 0, OP_F16 = 1, OP_F32 = 2 };
struct Operand {
  void* p;
  int ld;    // row length K
  int kind;  // OP_ROW / OP_F16 / OP_F32
  int mt;    // row tiles held by the buffer (fragment orders)
};

// Reset n launch timing slots (start = max, end = 0).
void stamp_init(unsigned long long* s, int n, hipStream_t st);

// Weight orders: row-major [N][K] or bf16 fragment order (16- or 32-column tiles).
enum { W_ROW = 0, W_F16 = 1, W_F32 = 2 };

// Weights of a later product read ahead by extra blocks of an earlier launch.
// With many slots every weight product runs from HBM (a step reads far more
// weights than the memory-side cache holds), and the wide-tile GEMM, which loads
// its fragments straight into registers four k-steps ahead, stalls on those
// first reads; read once shortly before, it runs as if warm (864 rows, first MLP
// product: 41.5 -> 34.0 us standalone).  Non-temporal loads do not allocate in
// that cache and do not help.
struct Touch {
  const void* p;  // null: nothing to read
  size_t bytes;
  int blocks;     // extra blocks of the launch that read it
};
// Row blocks (64 rows) from which the step reads weights ahead (about 57 slots)
constexpr int kTouchMinRowBlocks = 8;

// Block b of the t.blocks reading blocks reads its share of bytes [0, t.bytes) of
// t.p, 16 bytes per thread and eight loads in flight, and discards the values (the
// empty asm keeps the loads).
__device__ inline void touch_range(const Touch& t, unsigned b) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  const u32x4* q = static_cast<const u32x4*>(t.p);
  const size_t n16 = t.bytes / 16, stride = (size_t)t.blocks * blockDim.x;
  for (size_t i = (size_t)b * blockDim.x + threadIdx.x; i < n16; i += 8 * stride) {
    unsigned x = 0;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const size_t j = min(i + u * stride, n16 - 1);
      const u32x4 v = q[j];
      x ^= v.x ^ v.w;
    }
    asm volatile("" ::"v"(x));
  }
}

struct GemvArgs {
  Operand a;         // input operand (unused when lnx is set)
  const void* w;     // [N, K] storage type, order wkind
  int wkind;
  const void* bias;  // [N] storage type or null
  int K, N;
  int slot0, nslots, nsplit, R9;
  int mt0, mt1;      // operand row tiles (16 or 32 rows by wkind) covering the batch, all split terms
  // LayerNorm folded into the product (bf16, one slot, three split terms): the
  // operand is LN(lnx rows) with gain lng and bias lnb, built in LDS by each block.
  const float* lnx;  // [9][K] fp32 rows, or null
  const void* lng;
  const void* lnb;
  // column sums of the weights scaled by the gain and by the bias of that
  // LayerNorm, c[n] = sum_k g[k] W[n][k] and e[n] = sum_k b[k] W[n][k] ([N] fp32)
  const float* lnc;
  const float* lne;
  // split-K (EPI_PART): number of k-splits (grid y) and the element stride between
  // their partial buffers
  int ksplit;
  size_t pstride;
  int ct;  // 16-column tiles per block (4: wide kernel, with split-K), else 1
  float* y;          // STORE: out; RESID: residual stream; QKV: q; ARGMAX: optional logits
  int ldy;
  Operand aout;      // GELU: operand of the next product; RESID: tap operand (column offset tap * N);
                     // LayerNorm folded in (batch 1): tap operand of the rows lnx (column offset tap * K)
  int tap;
  // QKV cache append
  const int* state;
  const int* page_table;
  void* cache;
  size_t kv_stride;
  int d, n_head, n_ctx, pages_per_slot;
  // ARGMAX partials: best score and its column per (row, block); with inv_t > 0
  // the scores are z = logit * inv_t, plus Gumbel noise of stream rng_purpose (if
  // nonzero; position = row within the slot), and hm/hs receive the block's max of z
  // and sum of exp(z - max) for the softmax normaliser
  float* hv;
  int* hi;
  int nblk;
  const uint8_t* suppress;  // [N] nonzero: column excluded (logit -inf), or null
  float inv_t;
  int rng_purpose;
  uint64_t seed;
  float* hm;
  float* hs;
  unsigned long long* stamp;  // launch timing slot (profiled calls), or null
  // weights of a later product, read by pf.blocks blocks appended to grid x (grid
  // y 0 only); the LDS-staged several-slot GEMM takes it, other kernels ignore it
  Touch pf;
};

// Attention output product fused into the attention kernel (bf16, one slot):
// h[row][c] += sum over the head's 64 dims of O[row][k] W[k][c] (+ b[c], added
// once), W in 16-column fragment order with K = d.  Each block takes one of
// kOpGroups column groups of its head; the partial sums of the heads reach h
// through fp32 atomic adds (their order varies from run to run).
constexpr int kOpGroups = 8;
constexpr int kOpMaxCols = 160;  // columns of one group of a fused output product (d_model <= 1280)
struct OprojArgs {
  const void* w;     // null: no fused product (the operand rows are written instead)
  const void* bias;  // [N]
  float* h;          // residual rows [rows][ldh]
  int ldh, N, K;
};

struct AttnArgs {
  const float* q;  // q at column head*64 of row slot*9+i (stride ldq); drafter: q | k | v
  int ldq;
  const void* kcache;
  const void* vcache;
  const int* state;
  const int* page_table;
  const float* rope;  // [pos][32][cos, sin]
  Operand out;        // operand rows of the following product
  int slot0, d, n_head, n_ctx, pages_per_slot, nsplit, R9;
  OprojArgs op;
  // nonzero: the block clears the query values it read (its head's 64 columns of
  // the slot's nine rows) once every wave has used them, so that the next product
  // can add split-K partial sums into those places
  int clear_q;
  // drafter attention: the history before the anchor is attended (else the nine
  // block rows only), and queries / keys carry RoPE (else no rotation)
  int draft_hist, draft_rope;
  unsigned long long* stamp;  // launch timing slot (profiled calls), or null
};

struct CrossArgs {
  const float* q;
  int ldq;
  const void* kv;  // block base: per slot the keys [head][frame][64], then the values
                   // [head][frame][64] (fp32) or transposed [head][dim][vt_frames] (bf16)
  Operand out;
  int slot0, d, n_head, n_frames, nsplit, R9;
  int vt_frames;  // padded frame count of the transposed values (bf16), else 0
  int nchunk, chunk;  // frame chunks per (head, slot) and frames per chunk (multiple of 8)
  float* part;        // [pair][nchunk][kXrPart] chunk partials (nchunk > 1 or op.w)
  OprojArgs op;       // fused output product (taken by the merge kernel)
  int by_pair;        // bf16: one block per (head, slot) walks every chunk (no records, no merge)
  unsigned long long* stamp;  // launch timing slot (profiled calls), or null
};
// Chunk partial record: max [9] at 0, sum [9] at 16, acc [9][64] at 32.
constexpr int kXrPart = 32 + kRows * 64;
constexpr int kXrMaxPairs = 128;      // chunking only below this many (head, slot) pairs
constexpr int kXrMaxPartials = 512;   // pair * chunk records of a chunked launch
// bf16 acoustic memory: values stored transposed in 256-frame pieces,
// [head][frame / 256][dim][256], with the frame count padded to a multiple of
// kMxChunkMax (zeros past n_frames), so every matrix-core chunk reads whole
// 16-byte groups of one contiguous region.  Cross-attention blocks take chunks of
// 128 frames (four waves) for one slot and 512 (eight waves) for several.
constexpr int kMxChunkMax = 512;
constexpr int kVtPiece = 256;
__host__ __device__ __forceinline__ size_t vt_index(int dim, int f) {
  return ((size_t)(f / kVtPiece) * 64 + dim) * kVtPiece + (f % kVtPiece);
}
inline int xkv_vt_frames(int n_frames) { return (n_frames + kMxChunkMax - 1) / kMxChunkMax * kMxChunkMax; }
inline size_t xkv_slot_elems(bool bf16, int n_frames, int d) {
  return bf16 ? (size_t)d * (n_frames + xkv_vt_frames(n_frames)) : (size_t)2 * n_frames * d;
}
inline int cross_mx_chunk(int n) { return n == 1 ? 128 : 512; }
inline int cross_mx_chunks(int n, int n_frames) { return (n_frames + cross_mx_chunk(n) - 1) / cross_mx_chunk(n); }
// bf16, many (head, slot) pairs: a block per pair takes every 128-frame chunk in
// turn (up to kXpMaxChunks); measured at 96 slots, 20 heads, 1500 frames: 142 us
// against 150 + 12 us for 512-frame chunk blocks and their merge
constexpr int kXpMinPairs = 1024;    // about 52 slots at 20 heads: at least four blocks per CU
constexpr int kXpChunk = 128;
constexpr int kXpMaxChunks = 12;     // 1536 frames
inline bool cross_by_pair(int n, int n_head, int n_frames) {
  return n * n_head >= kXpMinPairs && (n_frames + kXpChunk - 1) / kXpChunk <= kXpMaxChunks;
}
// Chunking of cross-attention over the frames for a few slots with fp32
// storage (2 to 6 at 20 heads): about 240 blocks, chunks of >= 64 frames.  nchunk <= want, so
// pairs * nchunk <= kXrMaxPartials.
inline void cross_chunks(int pairs, int n_frames, int& nchunk, int& chunk) {
  nchunk = 1;
  chunk = n_frames;
  if (pairs >= kXrMaxPairs) return;
  int want = (240 + pairs - 1) / pairs;
  if (want > kXrMaxPartials / pairs) want = kXrMaxPartials / pairs;
  int ch = (n_frames + want - 1) / want;
  ch = ch < 64 ? 64 : (ch + 7) / 8 * 8;
  if (ch >= n_frames) return;
  chunk = ch;
  nchunk = (n_frames + ch - 1) / ch;
}

struct LnArgs {
  const float* x;  // [rows][d]
  const void* g;
  const void* b;
  Operand out;
  int d, row0, nsplit, R9;
  int rows;  // rows row0 .. row0 + rows - 1 (set by the launcher)
  unsigned long long* stamp;  // launch timing slot (profiled calls), or null
};

// h[row] += sum_s part[s][row] + bias; optional tap operand of the new h; then,
// when g is set, LayerNorm(h[row]) (gain g, bias b) as the operand `out`.
struct RlnArgs {
  const float* part;  // [nparts][rows][d] partial sums
  int nparts;
  size_t pstride;     // elements between partial buffers
  const void* bias;   // producer bias [d] or null
  float* h;           // residual stream [rows][d]
  Operand tap;        // tap operand (column offset tapcol) when tapcol >= 0
  int tapcol;
  const void* g;
  const void* b;
  Operand out;
  int d, row0, nsplit, R9;
  unsigned long long* stamp;  // launch timing slot (profiled calls), or null
};

struct BeginArgs {
  int* state;
  const int* draft;  // verify: draft [n][block_k]; prefill: tokens [n][pmax]
  int* tok;
  const void* emb;  // token embedding, order emb_kind (W_ROW, W_F16 or W_F32)
  int emb_kind;
  const void* pos;  // positional table (target) or mask vector (drafter)
  float* h;
  const int* page_table;  // [slot][pages_per_slot] (target passes: sets ST_PG0 / ST_PG1)
  int pages_per_slot;
  int slot0, d, n_vocab, n_ctx, block_k, k_max, chunk, pmax;
  unsigned* status;  // sticky device status word (verify: position overflow), or null
  const void* pos2;  // drafter with absolute positions: position table added to row i at t + i, else null
  float* hp;  // target passes: history-projection rows [slot][9][d] cleared for the split-K
              // product at the pass's end (its k-splits add into them), or null
};

struct HistArgs {
  const float* kv;  // [rows][2d]: k (no RoPE yet) | v, of the first drafter block
  void* kcache;     // first drafter block base [slot][head][n_ctx][64]
  void* vcache;
  int nlayer;           // drafter blocks written (grid z), 1 if 0
  size_t kv_stride;     // floats from one block's kv rows to the next's
  size_t cache_stride;  // storage elements from one block's caches to the next's
  const int* state;
  const float* rope;
  int slot0, d, n_head, n_ctx;
  unsigned* status;  // sticky device status word (position overflow), or null
  int use_rope;      // keys rotated at their positions (RoPE drafter), else stored as projected
};

struct AcceptArgs {
  int* state;
  const int* tok;
  const int* g;
  int* out;
  int* n_out;
  int* n_acc;
  int* done;
  int slot0, n, block_k, eos, n_ctx;
};

struct XkvArgs {
  const void* mem;  // [n_frames][d] of one slot
  const void* w;    // [2d][d]
  const void* bias; // [2d]
  void* out;        // block base + slot offset
  int d, n_head, n_frames;
  int vt_frames;    // > 0: values stored transposed [head][dim][vt_frames], padding zero
};

// Request-time matrix-core GEMM (k_mm.hip): C = A B^T (+ bias) for bf16 A [M, K] and
// B [N, K] (row-major, k contiguous), fp32 accumulation, 128 x 128 tiles, k in steps
// of kMmK; grid z runs over `batch` independent products (element strides sA, sB,
// sBias, sO, sO2).
constexpr int kMmTile = 128, kMmK = 64;
enum {
  MM_F32 = 0,        // out fp32 [M][ldo] = scale * C + bias
  MM_BF16 = 1,       // out bf16 [M][ldo]
  MM_BF16_GELU = 2,  // out bf16 [M][ldo] = GELU(scale * C + bias)
  MM_RESID = 3,      // out fp32 [M][ldo] += scale * C + bias
  MM_XKV = 4,        // acoustic keys [head][frame][64] then values [head][frame / 256][dim][256]
  MM_QKV_ENC = 5,    // columns < 2d: out bf16 [M][ldo]; the rest: out2 bf16 [head][dim][vt_frames]
  MM_GELU_ADD_F32 = 6,  // out fp32 [M][ldo] = GELU(scale * C + bias) + add[M][ldadd]
};
struct MmArgs {
  const bf16* A;
  long long lda, sA;
  const bf16* B;
  long long ldb, sB;
  const bf16* bias;
  long long sBias;
  int M, N, K;
  void* out;
  long long ldo, sO;
  void* out2;
  long long sO2;
  int d, n_head, vt_frames;  // transposed epilogues: model width, heads, padded frame count
  float scale;
  const float* add;  // MM_GELU_ADD_F32: fp32 rows added after the activation
  long long ldadd;
  int nb;            // rows of B present (0: N); columns past them re-read its last row
};
int mm_check(const MmArgs& a, int ep);
void mm(const MmArgs& a, int ep, int batch, hipStream_t st);

// Audio encoder (k_enc.hip).  Largest frontend window, model width and output
// positions the kernels hold in registers / LDS.
constexpr int kMaxFft = 512, kMaxEncD = 2048, kMaxEncCtx = 2048;
struct LogmelArgs {
  const float* audio;     // [n_samples] fp32
  int n_samples, n_fft, hop, n_frames, n_mels;
  const double* window;   // [n_fft] periodic Hann
  const double* twiddle;  // [n_fft][2]: cos(2 pi i / n_fft), -sin(2 pi i / n_fft)
  const double* filters;  // [n_mels][n_fft / 2 + 1] mel filterbank
  const int* fband;       // [n_mels][2]: first and one-past-last nonzero bin of each filter
  float* logmel;          // [n_frames][n_mels] log10 values
  int* gmax;              // the request's largest log10 value (order-preserving int)
  bf16* rows;             // [n_frames][ld1] first-convolution rows
  int ld1;
  float* mel_out;         // [n_mels][n_frames] scaled features, or null
};
void logmel(const LogmelArgs& a, hipStream_t st);
void conv_rows_s2(const bf16* z, bf16* out, int n_in, int n_out, int d, hipStream_t st);
void ln_rows(const float* x, const bf16* g, const bf16* b, bf16* out, int rows, int d, long long ldo, hipStream_t st);
// fused bidirectional attention of the encoder: q | k rows [n][ldqk] (q at column
// head * 64, k at d + head * 64), values transposed per head [head][64][Tp] (zero
// past n), output rows [n][ldo] at column head * 64; Tp a multiple of 64
struct EncAttnArgs {
  const bf16* qk;
  int ldqk;
  const bf16* vt;
  int Tp;
  bf16* o;
  int ldo, n, d;
};
void enc_attention(const EncAttnArgs& a, int n_head, hipStream_t st);

template <typename S>
struct Ops {
  static void ln_operand(const LnArgs& a, int rows, hipStream_t st);
  static void gemv(int epi, const GemvArgs& a, hipStream_t st);
  static void attn_self(const AttnArgs& a, int n, hipStream_t st);
  static void attn_draft(const AttnArgs& a, int n, hipStream_t st);
  static void attn_cross(const CrossArgs& a, int n, hipStream_t st);
  static void reduce_ln(const RlnArgs& a, int rows, hipStream_t st);
  static void verify_begin(const BeginArgs& a, int n, hipStream_t st);
  static void draft_begin(const BeginArgs& a, int n, hipStream_t st);
  static void prefill_begin(const BeginArgs& a, int n, hipStream_t st);
  static void hist_write(const HistArgs& a, int n, hipStream_t st);
  static void gemm_xkv(const XkvArgs& a, hipStream_t st);
};

template <typename S>
void repack(const void* src, void* dst, int N, int K, int wkind, hipStream_t st);

// c[n] = sum_k g[k] w[n][k] and e[n] = sum_k b[k] w[n][k] of a row-major bf16
// matrix w [N][K] and a LayerNorm's gain g and bias b [K] (fp64 sums rounded to
// fp32): what a product with that LayerNorm folded in adds after its matrix pass.
void ln_fold_cols(const void* w, const void* g, const void* b, int N, int K, float* c, float* e, hipStream_t st);

constexpr int kRlnMaxPartsHost = 16;
constexpr int kSampleBlocks = 64;     // vocabulary slices of a sampling draw per slot  // most split-K partials a reduction sums

// largest row length K of a product with the LayerNorm folded in (its operand is
// staged whole in LDS)
constexpr int kLnFoldMaxK = 1280;

// Per-row final argmax over the head's block partials; with hm set also the
// softmax normaliser (rmax = max z, rsum = sum exp(z - rmax)).
void argmax_final(const float* hv, const int* hi, int nblk, int row0, int rows, int* g, float* gmax, unsigned* status,
                  int* keep, int* dst, int slot0, int K, const float* hm, const float* hs, float* rmax, float* rsum,
                  hipStream_t st);

// Sampling acceptance (rejection rule), three launches: per-slot scan of the
// candidates, a Gumbel-max pass over the vocabulary for the residual / bonus /
// plain draw, and the final token plus state update.
struct SampleArgs {
  int* state;
  const int* tok;       // [rows] verify tokens (anchor, c_1..c_k)
  const float* lp;      // target logits [rows][V]
  const float* lq;      // draft logits [rows][V] (row j holds mask j)
  const float* tmax;    // target row normalisers
  const float* tsum;
  const float* dmax;    // draft row normalisers
  const float* dsum;
  int* sst;             // per slot: mode, row, accepted count, finished
  float* part;          // [slot][nsb][4]: best, index, fallback best, fallback index
  int nsb;
  int* out;
  int* n_out;
  int* n_acc;
  int* done;
  int slot0, n, block_k, eos, n_ctx, V;
  float inv_t;
  uint64_t seed;
};
void accept_sample(const SampleArgs& a, hipStream_t st);
void rng_words_device(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out, hipStream_t st);
void save_last(const float* h, float* lasth, const int* state, int slot0, int n, int d, int chunk, hipStream_t st);
void prefill_finish(int* state, const int* g, int slot0, int n, int eos, int n_ctx, int* first, hipStream_t st);
void accept_greedy(const AcceptArgs& a, hipStream_t st);

}  // namespace wf
