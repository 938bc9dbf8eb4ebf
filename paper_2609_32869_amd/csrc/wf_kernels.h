// Kernel argument blocks and launchers of libwf (internal).
#pragma once
#include <hip/hip_runtime.h>

#include "wf_common.h"

namespace wf {

enum { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_QKV = 3, EPI_ARGMAX = 4 };

struct GemvArgs {
  const float* x;  // input rows [slot*9 + i][ldx], fp32
  int ldx;
  const void* w;     // [N, K] storage type
  const void* bias;  // [N] storage type or null
  int K, N;
  int slot0, nslots;
  float* y;  // output rows (EPI_STORE/GELU: out; RESID: residual stream; QKV: q; ARGMAX: optional logits)
  int ldy;
  // EPI_RESID tap copy
  float* taps;
  int tap, n_tap;
  // EPI_QKV cache append
  const int* state;
  const int* page_table;
  void* cache;
  size_t kv_stride;
  int d, n_head, n_ctx, pages_per_slot;
  // EPI_ARGMAX partials
  float* hv;
  int* hi;
  int nblk;
};

struct AttnArgs {
  const float* q;  // q at column head*64 of row slot*9+i (stride ldq); drafter: q | k | v
  int ldq;
  const void* kcache;
  const void* vcache;
  const int* state;
  const int* page_table;
  const float* rope;  // [pos][32][cos, sin]
  float* out;         // [rows][d]
  int slot0, d, n_head, n_ctx, pages_per_slot;
};

struct CrossArgs {
  const float* q;
  int ldq;
  const void* kv;  // layer base of [slot][2][head][frame][64]
  float *pm, *pl, *po;
  float* out;
  int slot0, d, n_head, n_frames, nsplit;
};

struct BeginArgs {
  int* state;
  const int* draft;  // verify: draft [n][block_k]; prefill: tokens [n][pmax]
  int* tok;
  const void* emb;
  const void* pos;  // positional table (target) or mask vector (drafter)
  float* h;
  int slot0, d, n_vocab, n_ctx, block_k, k_max, chunk, pmax;
};

struct HistArgs {
  const float* kv;  // [rows][2d]: k (no RoPE yet) | v
  void* kcache;     // layer base [slot][head][n_ctx][64]
  void* vcache;
  const int* state;
  const float* rope;
  int slot0, d, n_head, n_ctx;
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
  void* out;        // layer base + slot offset
  int d, n_head, n_frames;
};

template <typename S>
struct Ops {
  static void layernorm(const float* x, const void* g, const void* b, float* y, int d, int row0, int rows, hipStream_t st);
  static void gemv(int epi, const GemvArgs& a, hipStream_t st);
  static void attn_self(const AttnArgs& a, int n, hipStream_t st);
  static void attn_draft(const AttnArgs& a, int n, hipStream_t st);
  static void attn_cross(const CrossArgs& a, int n, hipStream_t st);
  static void verify_begin(const BeginArgs& a, int n, hipStream_t st);
  static void draft_begin(const BeginArgs& a, int n, hipStream_t st);
  static void prefill_begin(const BeginArgs& a, int n, hipStream_t st);
  static void hist_write(const HistArgs& a, int n, hipStream_t st);
  static void gemm_xkv(const XkvArgs& a, hipStream_t st);
};

void argmax_final(const float* hv, const int* hi, int nblk, int row0, int rows, int* g, float* gmax, unsigned* status,
                  hipStream_t st);
void save_last(const float* h, float* lasth, const int* state, int slot0, int n, int d, int chunk, hipStream_t st);
void prefill_finish(int* state, const int* g, int slot0, int n, int eos, int n_ctx, int* first, hipStream_t st);
void hist_done(int* state, int slot0, int n, hipStream_t st);
void accept_greedy(const AcceptArgs& a, hipStream_t st);
void draft_tokens(const int* g, int* dst, int* keep, int slot0, int n, int K, hipStream_t st);

}  // namespace wf
