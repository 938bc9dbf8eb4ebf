// Host runtime of libwf: configuration checks, workspace carve-up, parameter
// copy, and the enqueue sequences of encode / prefill / draft / verify / step.
// Every device buffer lives in the caller's workspace; nothing here allocates
// device memory.
#include <algorithm>
#include <cmath>
#include <type_traits>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "wf_internal.h"

using namespace wf;

// Static scratch of wf_step_noalloc: the per-call buffers of one step when the
// caller cannot allocate.  Every GPU the library runs on holds its own copy until
// the process ends; all wf_step_noalloc calls on that GPU share it.
constexpr size_t kScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

// Device address of `scratch` per device.  In host code the array's name is only
// a stand-in, so kernels and copies get this address, looked up once per device
// (with that device current) by hipGetSymbolAddress.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

hipError_t scratch_setup(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev]) return hipSuccess;
  void* p = nullptr;
  hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_ptr[dev] = static_cast<char*>(p);
  return hipSuccess;
}

char* scratch_of(int dev) {
  if (dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  return g_scratch_ptr[dev];
}

thread_local std::string g_err;

int fail(Handle* h, int code, const std::string& msg) {
  if (h) h->err = msg;
  g_err = msg;
  return code;
}

#define HIPCK(h, x)                                                                 \
  do {                                                                              \
    hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess) return fail(h, WF_EHIP, std::string(#x ": ") + hipGetErrorString(e_)); \
  } while (0)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

size_t elt_bytes(const wf_config& c) { return c.dtype == WF_BF16 ? 2 : 4; }

int check_config(const wf_config* c, std::string& why) {
  if (!c) { why = "null config"; return WF_EINVAL; }
  if (c->dtype != WF_F32 && c->dtype != WF_BF16) { why = "dtype must be WF_F32 or WF_BF16"; return WF_EINVAL; }
  if (c->n_head <= 0 || c->d_model != c->n_head * kHeadDim) { why = "head width must be 64"; return WF_EINVAL; }
  if (c->d_model > 2048) { why = "d_model must be <= 2048"; return WF_EINVAL; }
  if (c->n_layer <= 0 || c->n_draft_layer <= 0) { why = "layer counts must be positive"; return WF_EINVAL; }
  if (c->d_ff <= 0 || c->d_ff % 32) { why = "d_ff must be a positive multiple of 32"; return WF_EINVAL; }
  if (c->n_vocab < 2) { why = "n_vocab must be >= 2"; return WF_EINVAL; }
  if (c->n_ctx < 16 || c->n_ctx > kMaxCtx || c->n_ctx % kPage) { why = "n_ctx must be a multiple of 16 in [16, 448]"; return WF_EINVAL; }
  if (c->n_frames < 1 || c->n_frames > kMaxFrames) { why = "n_frames must be in [1, 2048]"; return WF_EINVAL; }
  if (c->block_k != kRows - 1) { why = "block_k must be 8"; return WF_EINVAL; }
  if (c->n_tap < 1 || c->n_tap > WF_MAX_TAPS) { why = "n_tap must be in [1, 8]"; return WF_EINVAL; }
  for (int i = 0; i < c->n_tap; ++i) {
    if (c->taps[i] < 0 || c->taps[i] >= c->n_layer || (i && c->taps[i] <= c->taps[i - 1])) {
      why = "taps must be strictly increasing block indices";
      return WF_EINVAL;
    }
  }
  if (c->max_batch < 1 || c->max_batch > 4096) { why = "max_batch must be in [1, 4096]"; return WF_EINVAL; }
  if (c->eos_id < -1 || c->eos_id >= c->n_vocab) { why = "eos_id out of range"; return WF_EINVAL; }
  if (c->draft_flags & ~(int32_t)(WF_DRAFT_NO_AUDIO | WF_DRAFT_NO_HISTORY | WF_DRAFT_ABS_POS)) {
    why = "unknown draft_flags bits";
    return WF_EINVAL;
  }
  return WF_OK;
}

// manifest entry -> (numel, destination element offset in the weight region, the
// streamed matrix it belongs to or -1)
struct ManEntry {
  size_t numel, dst;
  int mat;
};

// A streamed weight matrix [N][K]: with bf16 storage it is kept in matrix-core
// fragment order (kind W_F16 or W_F32); entries of the manifest that make it up
// are consecutive and hold consecutive row ranges.
struct Mat {
  size_t dst;
  int N, K, kind;
  // a product with this LayerNorm folded in (batch 1): gain and bias offsets in the
  // weight region and the fp32 offset of its column sums c, e; lng == kNoLn otherwise
  size_t lng, lnb, cols;
};
constexpr size_t kNoLn = ~(size_t)0;

std::vector<ManEntry> manifest(const wf_config& c, const Layout& L, std::vector<Mat>* mats = nullptr) {
  const size_t d = c.d_model, F = c.d_ff;
  const bool frag = c.dtype == WF_BF16;
  std::vector<ManEntry> m;
  std::vector<Mat> mm;
  // start a streamed matrix (bf16 storage only); returns its index for the entries
  auto mat = [&](size_t dst, size_t N, size_t K, int kind, size_t lng = kNoLn, size_t lnb = 0, size_t cols = 0) {
    if (!frag) return -1;
    mm.push_back({dst, (int)N, (int)K, kind, L.nsplit_op == 3 ? lng : kNoLn, lnb, cols});
    return (int)mm.size() - 1;
  };
  // 32-column tiles (W_1, head) only at batch 1; with several slots every matrix
  // uses 16-column tiles for the GEMM kernel
  const int wide = L.nsplit_op == 3 ? W_F32 : W_F16;
  const int emb = mat(L.tok_emb, c.n_vocab, d, wide);
  m.push_back({(size_t)c.n_vocab * d, L.tok_emb, emb});
  m.push_back({(size_t)c.n_ctx * d, L.pos_emb, -1});
  auto block = [&](const BlockW& b, bool cross) {
    m.push_back({d, b.ln1_g, -1}); m.push_back({d, b.ln1_b, -1});
    const int qkv = mat(b.w_qkv, 3 * d, d, W_F16, b.ln1_g, b.ln1_b, b.c_qkv);
    m.push_back({d * d, b.w_qkv, qkv}); m.push_back({d, b.b_qkv, -1});
    m.push_back({d * d, b.w_qkv + d * d, qkv});
    m.push_back({d * d, b.w_qkv + 2 * d * d, qkv}); m.push_back({d, b.b_qkv + 2 * d, -1});
    m.push_back({d * d, b.w_o, mat(b.w_o, d, d, W_F16)}); m.push_back({d, b.b_o, -1});
    if (cross) {
      m.push_back({d, b.ln2_g, -1}); m.push_back({d, b.ln2_b, -1});
      m.push_back({d * d, b.w_q2, mat(b.w_q2, d, d, W_F16, b.ln2_g, b.ln2_b, b.c_q2)}); m.push_back({d, b.b_q2, -1});
      m.push_back({d * d, b.w_kv2, -1});  // encode-time product: row-major
      m.push_back({d * d, b.w_kv2 + d * d, -1}); m.push_back({d, b.b_kv2 + d, -1});
      m.push_back({d * d, b.w_o2, mat(b.w_o2, d, d, W_F16)}); m.push_back({d, b.b_o2, -1});
    }
    m.push_back({d, b.ln3_g, -1}); m.push_back({d, b.ln3_b, -1});
    m.push_back({F * d, b.w_fc1, mat(b.w_fc1, F, d, wide, b.ln3_g, b.ln3_b, b.c_fc1)}); m.push_back({F, b.b_fc1, -1});
    m.push_back({d * F, b.w_fc2, mat(b.w_fc2, d, F, W_F16)}); m.push_back({d, b.b_fc2, -1});
  };
  for (auto& b : L.tb) block(b, true);
  m.push_back({d, L.lnf_g, -1}); m.push_back({d, L.lnf_b, -1});
  if (!(c.draft_flags & WF_DRAFT_NO_HISTORY)) {
    m.push_back({d * c.n_tap * d, L.hproj_w, mat(L.hproj_w, d, c.n_tap * d, W_F16)});
    m.push_back({d, L.hproj_b, -1});
  }
  m.push_back({d, L.mask, -1});
  for (auto& b : L.db) block(b, !(c.draft_flags & WF_DRAFT_NO_AUDIO));
  m.push_back({d, L.dlnf_g, -1}); m.push_back({d, L.dlnf_b, -1});
  if (mats) *mats = mm;
  return m;
}

}  // namespace

namespace wf {

int compute_layout(const wf_config& c, Layout& L) {
  const size_t d = c.d_model, F = c.d_ff, V = c.n_vocab, B = c.max_batch, H = c.n_head;
  const size_t R9 = B * kRows;
  const size_t eb = elt_bytes(c);
  // weight region (element offsets, 128-element aligned)
  size_t w = 0;
  auto take = [&](size_t n) { size_t o = w; w = align_up(w + n, 128); return o; };
  size_t cw = 0;  // fp32 LayerNorm column sums (c then e) of the folded products
  auto takec = [&](size_t n) { size_t o = cw; cw += 2 * n; return o; };
  L.tok_emb = take(align_up(V, 32) * d);  // padded to whole 32-column tiles
  L.pos_emb = take((size_t)c.n_ctx * d);
  auto block = [&]() {
    BlockW b;
    b.ln1_g = take(d); b.ln1_b = take(d);
    b.w_qkv = take(3 * d * d); b.b_qkv = take(3 * d);
    b.w_o = take(d * d); b.b_o = take(d);
    b.ln2_g = take(d); b.ln2_b = take(d);
    b.w_q2 = take(d * d); b.b_q2 = take(d);
    b.w_kv2 = take(2 * d * d); b.b_kv2 = take(2 * d);
    b.w_o2 = take(d * d); b.b_o2 = take(d);
    b.ln3_g = take(d); b.ln3_b = take(d);
    b.w_fc1 = take(F * d); b.b_fc1 = take(F);
    b.w_fc2 = take(d * F); b.b_fc2 = take(d);
    b.c_qkv = takec(3 * d); b.c_q2 = takec(d); b.c_fc1 = takec(F);
    return b;
  };
  L.tb.clear();
  L.db.clear();
  for (int l = 0; l < c.n_layer; ++l) L.tb.push_back(block());
  L.lnf_g = take(d); L.lnf_b = take(d);
  L.hproj_w = take(d * c.n_tap * d); L.hproj_b = take(d); L.mask = take(d);
  for (int l = 0; l < c.n_draft_layer; ++l) L.db.push_back(block());
  L.dlnf_g = take(d); L.dlnf_b = take(d);
  L.c_head = takec(V); L.c_dhead = takec(V);
  L.weight_elems = w;
  L.pages_per_slot = c.n_ctx / kPage;
  // column blocks of the vocabulary head: 32-column tiles (bf16, batch 1), 64-column
  // GEMM blocks (bf16, several slots) or 16-column tiles (fp32)
  L.nsplit_op = c.dtype != WF_BF16 ? 1 : c.max_batch == 1 ? 3 : 2;
  L.head_blocks = c.dtype != WF_BF16 ? (int)((V + 15) / 16) : L.nsplit_op == 3 ? (int)((V + 31) / 32) : (int)((V + 63) / 64);
  // raw bf16 matrices are staged at init in the cross K/V region before reordering
  L.stage_bytes = 0;
  if (c.dtype == WF_BF16) {
    const size_t big = std::max({V * d, 3 * d * d, F * d, (size_t)c.n_tap * d * d});
    L.stage_bytes = big * eb;
  }
  // byte regions
  size_t o = 0;
  auto region = [&](size_t bytes) { size_t r = o; o = align_up(o + bytes, 256); return r; };
  L.state = region(B * kStateInts * 4);
  L.page_table = region(B * L.pages_per_slot * 4);
  L.rope = region((size_t)(c.n_ctx + kRows + 1) * 32 * 2 * 4);
  L.status = region(256);
  L.aux = region(4 * B * 4);
  L.weights = region(w * eb);
  L.xkv = region(std::max((size_t)(c.n_layer + c.n_draft_layer) * B * xkv_slot_elems(c.dtype == WF_BF16, c.n_frames, (int)d) * eb,
                          L.stage_bytes));
  L.skv = region((size_t)c.n_layer * 2 * B * L.pages_per_slot * H * kPage * kHeadDim * eb);
  L.hkv = region((size_t)c.n_draft_layer * 2 * B * H * c.n_ctx * kHeadDim * eb);
  // matrix operands: 3 bf16 terms per fp32 value as extra rows at batch 1, 2 terms as
  // two planes with several slots (bf16 storage, set above)
  const size_t rows = (L.nsplit_op == 3 ? 3 : 1) * R9, planes = L.nsplit_op == 2 ? 2 : 1;
  L.mt16 = (int)((rows + 15) / 16);
  L.mt32 = (int)((rows + 31) / 32);
  const size_t M16 = (size_t)L.mt16 * 16, M32 = std::max((size_t)L.mt32 * 32, M16);
  L.a_d16 = region(planes * M16 * d * eb);
  L.a_d32 = region(planes * M32 * d * eb);
  L.a_f16 = region(planes * M16 * F * eb);
  L.a_tap16 = region(planes * M16 * c.n_tap * d * eb);
  L.h = region(R9 * d * 4);
  L.qkv = region(R9 * 3 * d * 4);
  L.hp = region(R9 * d * 4);
  L.kvh = region(R9 * 2 * d * 4 * std::max(c.n_draft_layer, 1));  // k | v rows of each drafter block
  L.hv = region(R9 * L.head_blocks * 4);
  L.hi = region(R9 * L.head_blocks * 4);
  L.hm = region(R9 * L.head_blocks * 4);
  L.hs = region(R9 * L.head_blocks * 4);
  L.tmax = region(R9 * 4);
  L.tsum = region(R9 * 4);
  L.dmax = region(R9 * 4);
  L.dsum = region(R9 * 4);
  L.sst = region(B * 4 * 4);
  L.spart = region(B * kSampleBlocks * 4 * 4);
  L.tok = region(R9 * 4);
  L.g = region(R9 * 4);
  L.gmax = region(R9 * 4);
  L.draft = region(B * c.block_k * 4);
  L.lasth = region(R9 * d * 4);
  L.logits = region(R9 * V * 4);
  L.dlogits = region(R9 * V * 4);
  // batch 1 with bf16 storage: the second MLP product is split over k into
  // partial sums that the residual update reduces (about 240 blocks of 64 columns)
  L.fc2_split = 0;
  if (c.dtype == WF_BF16 && L.nsplit_op == 3 && d <= (size_t)kLnFoldMaxK) {
    const int tiles64 = (int)((d + 63) / 64), ksteps = (int)(F / 32);
    L.fc2_split = std::max(1, std::min({kRlnMaxPartsHost, 240 / tiles64, ksteps}));
  }
  const int nparts = std::max({L.fc2_split, L.nsplit_op == 2 ? kFc2SplitBatch : 0, 1});
  L.part = region((size_t)nparts * R9 * d * 4);
  const size_t xrec = c.dtype == WF_BF16 ? B * H * (size_t)cross_mx_chunks(1, c.n_frames) : 0;  // 1 slot: the smallest chunks
  L.xpart = region(std::max((size_t)kXrMaxPartials, xrec) * kXrPart * 4);
  L.lncd = region(L.nsplit_op == 3 ? cw * 4 : 0);
  L.stamps = region((size_t)kStampSlots * kStampWords * 8);
  L.total = o;
  return WF_OK;
}

}  // namespace wf

namespace {

template <typename S>
struct Runner {
  Handle* h;
  hipStream_t st;
  const wf_config& c;
  const Layout& L;
  Runner(Handle* h_, hipStream_t s) : h(h_), st(s), c(h_->cfg), L(h_->lay) {}

  // The LayerNorm operand of the next product was already written by the
  // residual reduction (Ad16 for a block's first product, Ad32 for the head).
  bool ln_ready = false;
  int tap_next = -1;  // drafter tap the next folded q|k|v product writes from its rows (-1: none)

  // The LayerNorm that follows a block: the next block's first one, or the final
  // one before the vocabulary head (wide: its operand feeds 32-column tiles).
  struct LnNext {
    size_t g, b;
    bool wide;
    size_t wq, nq;  // weights of the next block's q|k|v product (offset, elements; 0: none)
  };

  // Several slots (kTouchMinRowBlocks row blocks or more, bf16 operands): the
  // weights of the wide-tile products (q|k|v, W_1) are read by extra blocks of
  // the product launched before them (W'_o, W_2 of the previous block), so they
  // come from the memory-side cache rather than HBM.  The 64 x 64 tile products
  // stage three k-steps ahead through LDS and gain nothing from it (measured).
  // touch_ holds the request for the next product launch, which takes it.
  Touch touch_{nullptr, 0, 0};
  bool touch_ahead(int slot0, int n) const {
    if (L.nsplit_op != 2) return false;
    const int mb0 = slot0 * kRows / 64, mb1 = ((slot0 + n) * kRows + 63) / 64;
    return mb1 - mb0 >= kTouchMinRowBlocks;
  }
  // blocks: extra blocks of the launch (64 beside a 64 x 64 tile product, which
  // holds two blocks per CU)
  void touch_next(int slot0, int n, size_t w, size_t elems, int blocks) {
    touch_ = touch_ahead(slot0, n) && elems > 0 ? Touch{W(w), elems * (size_t)eb(), blocks} : Touch{nullptr, 0, 0};
  }

  // Run one launch.  When profiling, the launch gets a timing slot (kernels that
  // take one record their first-wave start and last-wave end in it).
  template <typename F>
  void launch(const char* tag, double bytes, F&& f) {
    unsigned long long* stamp = nullptr;
    if (h->prof && h->nstamp < kStampSlots) {
      const int slot = h->nstamp++;
      stamp = h->at<unsigned long long>(L.stamps) + (size_t)kStampWords * slot;
      (h->capturing ? h->cap_recs : h->prof_recs).push_back(ProfRec{tag, bytes, slot});
    }
    f(stamp);
  }
  double eb() const { return c.dtype == WF_BF16 ? 2.0 : 4.0; }

  const S* W(size_t off) const { return h->at<const S>(L.weights) + off; }
  float* F32(size_t off) const { return h->at<float>(off); }
  int* I32(size_t off) const { return h->at<int>(off); }
  size_t xkv_slot() const { return xkv_slot_elems(c.dtype == WF_BF16, c.n_frames, c.d_model); }
  int vt_frames() const { return c.dtype == WF_BF16 ? xkv_vt_frames(c.n_frames) : 0; }
  S* xkv_layer(int l) const { return h->at<S>(L.xkv) + (size_t)l * c.max_batch * xkv_slot(); }
  S* skv_layer(int l) const {
    return h->at<S>(L.skv) + (size_t)l * 2 * kv_stride();
  }
  size_t kv_stride() const { return (size_t)c.max_batch * L.pages_per_slot * c.n_head * kPage * kHeadDim; }
  S* hkv(int dl, int kv) const {
    return h->at<S>(L.hkv) + ((size_t)dl * 2 + kv) * c.max_batch * c.n_head * c.n_ctx * kHeadDim;
  }

  bool frag() const { return c.dtype == WF_BF16; }
  // Operand buffer at `off` with row length K, in the order read by products whose
  // weights have 32-column (wide) or 16-column tiles.
  Operand op(size_t off, int K, bool wide) const {
    if (!frag()) return Operand{h->at<void>(off), K, OP_ROW, L.mt16};
    return wide && L.nsplit_op == 3 ? Operand{h->at<void>(off), K, OP_F32, L.mt32}
                                    : Operand{h->at<void>(off), K, OP_F16, L.mt16};
  }
  Operand Ad16() const { return op(L.a_d16, c.d_model, false); }
  Operand Ad32() const { return op(L.a_d32, c.d_model, true); }
  Operand Af16() const { return op(L.a_f16, c.d_ff, false); }
  Operand Atap16() const { return op(L.a_tap16, c.n_tap * c.d_model, false); }
  int wk(bool wide) const { return frag() ? (wide && L.nsplit_op == 3 ? W_F32 : W_F16) : W_ROW; }
  int R9() const { return c.max_batch * kRows; }

  GemvArgs gemv_base(int slot0, int n, int wkind) const {
    GemvArgs a{};
    a.slot0 = slot0;
    a.nslots = n;
    a.nsplit = L.nsplit_op;
    a.R9 = R9();
    a.wkind = wkind;
    const int T = wkind == W_F32 ? 32 : 16;  // operand rows per tile
    if (L.nsplit_op == 3) {
      a.mt0 = 0;
      a.mt1 = (3 * R9() + T - 1) / T;
    } else {
      a.mt0 = slot0 * kRows / T;
      a.mt1 = ((slot0 + n) * kRows + T - 1) / T;
    }
    a.tap = -1;
    a.state = I32(L.state);
    a.page_table = I32(L.page_table);
    a.d = c.d_model;
    a.n_head = c.n_head;
    a.n_ctx = c.n_ctx;
    a.pages_per_slot = L.pages_per_slot;
    return a;
  }

  // bytes a GEMV launch must move: weights + bias once, operand rows, outputs
  double gemv_bytes(int n, int K, int N, int epi) const {
    const double rows = (double)kRows * n;
    return (double)N * K * eb() + N * eb() + L.nsplit_op * rows * K * eb() +
           rows * N * 4.0 * (epi == EPI_RESID ? 2 : 1);
  }

  GemvArgs gemv_args(int slot0, int n, Operand x, size_t w, size_t b, int K, int N, float* y, int ldy,
                     Operand aout, int tap) const {
    GemvArgs a = gemv_base(slot0, n, wk(x.kind == OP_F32));
    a.a = x;
    a.w = W(w);
    a.bias = W(b);
    a.K = K;
    a.N = N;
    a.y = y;
    a.ldy = ldy;
    a.aout = aout;
    a.tap = tap;
    return a;
  }
  // Several slots whose 64 x 64 tiles of an N-column product cover fewer than 160
  // blocks: the product is split over k in kResidSplit (partial sums added).
  bool split_small(int slot0, int n, int K, int N) const {
    if (L.nsplit_op != 2) return false;
    const int mb0 = slot0 * kRows / 64, mb1 = ((slot0 + n) * kRows + 63) / 64;
    return (mb1 - mb0) * ((N + 63) / 64) < 160 && (K / 32) % kResidSplit == 0;
  }

  // h += x W^T + b.  With several slots whose 64 x 64 tiles cover fewer than 160
  // blocks, the k-steps are split kResidSplit ways and every split adds its
  // partial sums to h (the bias from the first), so the launch fills the chip.
  void resid(const char* tag, int slot0, int n, Operand x, size_t w, size_t b, int K, int N) {
    GemvArgs a = gemv_args(slot0, n, x, w, b, K, N, F32(L.h), c.d_model, Operand{nullptr, 0, OP_ROW, 0}, -1);
    if (split_small(slot0, n, K, N)) {
      a.ksplit = kResidSplit;
      run_gemv(tag, EPI_ACC, n, a);
      return;
    }
    run_gemv(tag, EPI_RESID, n, a);
  }

  // tag: the product's role in the step, for the eager profile
  void run_gemv(const char* tag, int epi, int n, const GemvArgs& a) {
    const Touch pf = touch_;
    touch_ = Touch{nullptr, 0, 0};
    launch(tag, gemv_bytes(n, a.K, a.N, epi), [&](unsigned long long* sp) {
      GemvArgs b = a;
      b.stamp = sp;
      b.pf = pf;
      Ops<S>::gemv(epi, b, st);
    });
  }

  void gemv(const char* tag, int epi, int slot0, int n, Operand x, size_t w, size_t b, int K, int N, float* y, int ldy,
            Operand aout = Operand{nullptr, 0, OP_ROW, 0}, int tap = -1) {
    run_gemv(tag, epi, n, gemv_args(slot0, n, x, w, b, K, N, y, ldy, aout, tap));
  }

  // LayerNorm folded into the product that consumes it: bf16 storage at batch 1
  // (three split terms) with rows short enough to stage in LDS.
  bool fold_ln() const { return frag() && L.nsplit_op == 3 && c.d_model <= kLnFoldMaxK; }

  // Batch 1 with bf16 storage: the attention output products are fused into the
  // attention kernels (h += O W + b through atomic adds); a group's d / kOpGroups
  // columns (two threads each) must fit the merge kernel's block.
  bool fuse_oproj() const {
    return frag() && L.nsplit_op == 3 && c.d_model / kOpGroups <= kOpMaxCols && (c.d_model / kOpGroups) % 16 == 0;
  }
  OprojArgs oproj(size_t w, size_t b) {
    if (!fuse_oproj()) return OprojArgs{};
    return OprojArgs{W(w), W(b), F32(L.h), (int)c.d_model, (int)c.d_model, (int)c.d_model};
  }

  // Make LayerNorm(rows x; gain g, bias b) the operand of product a: folded into
  // the product, or a separate launch that writes operand `op`.
  // The fold repeats the normalisation in every block, so products with many
  // column blocks (the vocabulary head) take the separate launch.
  // cols: fp32 offset of the matrix's column sums c (e follows after N values),
  // row0: first output column of the product within that matrix
  void ln_operand(GemvArgs& a, int slot0, int n, const float* x, size_t g, size_t b, Operand op, bool fold = true,
                  size_t cols = 0, size_t ncols = 0, size_t row0 = 0) {
    if (fold && fold_ln()) {
      a.lnx = x + (size_t)slot0 * kRows * c.d_model;
      a.lng = W(g);
      a.lnb = W(b);
      a.lnc = F32(L.lncd) + cols + row0;
      a.lne = F32(L.lncd) + cols + ncols + row0;
    } else {
      ln(slot0, n, x, g, b, op);
      a.a = op;
    }
  }

  // y = LN(x) W^T + bias with the LayerNorm operand in `op` when not folded
  // cols / ncols / row0: the LayerNorm column sums of the matrix w belongs to (see ln_operand)
  void gemv_ln(const char* tag, int epi, int slot0, int n, const float* x, size_t g, size_t gb, size_t cols, size_t ncols,
               size_t row0, Operand op, size_t w, size_t b, int K, int N, float* y, int ldy,
               Operand aout = Operand{nullptr, 0, OP_ROW, 0}) {
    GemvArgs a = gemv_args(slot0, n, op, w, b, K, N, y, ldy, aout, -1);
    ln_operand(a, slot0, n, x, g, gb, op, true, cols, ncols, row0);
    run_gemv(tag, epi, n, a);
  }

  void ln(int slot0, int n, const float* x, size_t g, size_t b, Operand out) {
    LnArgs la{};
    la.x = x; la.g = W(g); la.b = W(b); la.out = out; la.d = c.d_model; la.row0 = slot0 * kRows;
    la.nsplit = L.nsplit_op; la.R9 = R9();
    launch("layernorm", 4.0 * kRows * n * c.d_model * (1 + L.nsplit_op * eb() / 4.0),
           [&](unsigned long long* sp) {
             la.stamp = sp;
             Ops<S>::ln_operand(la, n * kRows, st);
           });
  }

  void cross(int slot0, int n, int layer, const OprojArgs& op) {
    CrossArgs a{};
    a.op = op;
    a.q = F32(L.qkv);
    a.ldq = 3 * c.d_model;
    a.kv = xkv_layer(layer);
    a.out = Ad16();
    a.slot0 = slot0;
    a.d = c.d_model;
    a.n_head = c.n_head;
    a.n_frames = c.n_frames;
    a.nsplit = L.nsplit_op;
    a.R9 = R9();
    a.vt_frames = vt_frames();
    if (c.dtype == WF_BF16 && op.w == nullptr && cross_by_pair(n, c.n_head, c.n_frames)) {
      a.by_pair = 1;
      a.chunk = kXpChunk;
      a.nchunk = (c.n_frames + kXpChunk - 1) / kXpChunk;
    } else if (c.dtype == WF_BF16) {
      a.chunk = cross_mx_chunk(n);
      a.nchunk = cross_mx_chunks(n, c.n_frames);
    } else {
      cross_chunks(n * c.n_head, c.n_frames, a.nchunk, a.chunk);
    }
    a.part = F32(L.xpart);
    const double wbytes = op.w ? (double)c.d_model * c.d_model * eb() : 0.0;  // fused output product
    launch("attn_cross", 2.0 * c.n_head * c.n_frames * kHeadDim * eb() * n + wbytes, [&](unsigned long long* sp) {
      a.stamp = sp;
      Ops<S>::attn_cross(a, n, st);
    });
  }

  // Several slots with bf16 operands: the second MLP product's k-steps split in
  // kFc2SplitBatch (partial sums reduced with the residual update and the next
  // LayerNorm), else 0.  Few slots: its 64 x 64 tiles alone would not fill the
  // chip; many slots: it runs on the wide tiles, which alone would give too few.
  int fc2_split_batch() const {
    if (L.nsplit_op != 2) return 0;
    return (c.d_ff / 32) % kFc2SplitBatch == 0 ? kFc2SplitBatch : 0;
  }

  // second half of a decoder block shared by target and drafter: cross-attention and MLP
  // q_clear: the self-attention before left the query places at zero, so a
  // split W'_q product may add its partial sums into them
  // cross: the block has its cross-attention sub-layer (every target block; drafter
  // blocks unless the variant drops it)
  void block_tail(int slot0, int n, const BlockW& b, int xlayer, int tap, const LnNext& nx, bool q_clear = false,
                  bool cross = true) {
    if (cross) cross_sublayer(slot0, n, b, xlayer, q_clear);
    mlp_sublayer(slot0, n, b, tap, nx);
  }

  void cross_sublayer(int slot0, int n, const BlockW& b, int xlayer, bool q_clear) {
    const int d = c.d_model;
    float *h_ = F32(L.h), *qkv = F32(L.qkv);
    if (q_clear) {
      GemvArgs a = gemv_args(slot0, n, Ad16(), b.w_q2, b.b_q2, d, d, qkv, 3 * d, Operand{nullptr, 0, OP_ROW, 0}, -1);
      ln_operand(a, slot0, n, h_, b.ln2_g, b.ln2_b, Ad16(), true, b.c_q2, d, 0);
      a.ksplit = kResidSplit;
      run_gemv("gemv_q2", EPI_ACC, n, a);
    } else {
      gemv_ln("gemv_q2", EPI_STORE, slot0, n, h_, b.ln2_g, b.ln2_b, b.c_q2, d, 0, Ad16(), b.w_q2, b.b_q2, d, d, qkv, 3 * d);
    }
    const OprojArgs op2 = oproj(b.w_o2, b.b_o2);
    cross(slot0, n, xlayer, op2);
    if (op2.w == nullptr) {
      touch_next(slot0, n, b.w_fc1, (size_t)c.d_ff * d, 64);
      resid("gemv_o", slot0, n, Ad16(), b.w_o2, b.b_o2, d, d);
    }
  }

  void mlp_sublayer(int slot0, int n, const BlockW& b, int tap, const LnNext& nx) {
    const int d = c.d_model;
    float* h_ = F32(L.h);
    gemv_ln("gemv_fc1", EPI_GELU, slot0, n, h_, b.ln3_g, b.ln3_b, b.c_fc1, c.d_ff, 0, Ad32(), b.w_fc1, b.b_fc1, d, c.d_ff,
            nullptr, 0, Af16());
    touch_next(slot0, n, nx.wq, nx.nq, 64);
    const int ksplit = L.fc2_split > 0 ? L.fc2_split : fc2_split_batch();
    // a tap block followed by a target block: that block's q|k|v product, which
    // folds its LayerNorm and so reads the rows anyway, writes the tap
    const bool tap_later = tap >= 0 && !nx.wide && fold_ln() && Atap16().kind == OP_F16;
    if (fuse_oproj() && L.fc2_split > 0 && (tap < 0 || tap_later)) {
      // batch 1 (bf16): the k-splits add their partial sums and the bias straight
      // to the residual rows; the next product folds its LayerNorm in (or the
      // head's LayerNorm runs on its own)
      GemvArgs a = gemv_args(slot0, n, Af16(), b.w_fc2, b.b_fc2, c.d_ff, d, h_, d, Operand{nullptr, 0, OP_ROW, 0}, -1);
      a.ct = 4;
      a.ksplit = L.fc2_split;
      run_gemv("gemv_fc2", EPI_ACC, n, a);
      ln_ready = false;
      tap_next = tap;
    } else if (ksplit > 0) {
      // k-split partial sums, then h += sum + bias, the tap, and the next LayerNorm
      GemvArgs a = gemv_args(slot0, n, Af16(), b.w_fc2, b.b_fc2, c.d_ff, d, F32(L.part), d, Operand{nullptr, 0, OP_ROW, 0}, -1);
      a.bias = nullptr;
      a.ct = 4;
      a.ksplit = ksplit;
      a.pstride = (size_t)R9() * d;
      run_gemv("gemv_fc2", EPI_PART, n, a);
      RlnArgs ra{};
      ra.part = F32(L.part); ra.nparts = ksplit; ra.pstride = (size_t)R9() * d; ra.bias = W(b.b_fc2); ra.h = h_;
      ra.tap = Atap16(); ra.tapcol = tap >= 0 ? tap * d : -1; ra.g = W(nx.g); ra.b = W(nx.b); ra.out = nx.wide ? Ad32() : Ad16();
      ra.d = d; ra.row0 = slot0 * kRows; ra.nsplit = L.nsplit_op; ra.R9 = R9();
      launch("reduce_ln", 4.0 * kRows * n * d * (ksplit + 3), [&](unsigned long long* sp) {
        ra.stamp = sp;
        Ops<S>::reduce_ln(ra, n * kRows, st);
      });
      ln_ready = true;
    } else {
      gemv("gemv_fc2", EPI_RESID, slot0, n, Af16(), b.w_fc2, b.b_fc2, c.d_ff, d, h_, d, Atap16(), tap);
    }
  }

  void target_forward(int slot0, int n) {
    const int d = c.d_model;
    float *h_ = F32(L.h), *qkv = F32(L.qkv);
    ln_ready = false;
    tap_next = -1;
    touch_ = Touch{nullptr, 0, 0};
    for (int l = 0; l < c.n_layer; ++l) {
      const BlockW& b = L.tb[l];
      int tap = -1;
      for (int i = 0; i < c.n_tap; ++i)
        if (c.taps[i] == l) tap = i;
      GemvArgs a = gemv_base(slot0, n, wk(false));
      a.w = W(b.w_qkv); a.bias = W(b.b_qkv); a.K = d; a.N = 3 * d;
      a.y = qkv; a.ldy = 3 * d; a.cache = skv_layer(l); a.kv_stride = kv_stride();
      if (ln_ready) a.a = Ad16();
      else ln_operand(a, slot0, n, h_, b.ln1_g, b.ln1_b, Ad16(), true, b.c_qkv, 3 * d);
      if (tap_next >= 0) {
        a.aout = Atap16();
        a.tap = tap_next;
        tap_next = -1;
      }
      ln_ready = false;
      run_gemv("gemv_qkv", EPI_QKV, n, a);
      AttnArgs at{};
      at.q = qkv; at.ldq = 3 * d; at.kcache = skv_layer(l); at.vcache = skv_layer(l) + kv_stride();
      at.state = I32(L.state); at.page_table = I32(L.page_table); at.rope = F32(L.rope); at.out = Ad16();
      at.slot0 = slot0; at.d = d; at.n_head = c.n_head; at.n_ctx = c.n_ctx; at.pages_per_slot = L.pages_per_slot;
      at.nsplit = L.nsplit_op; at.R9 = R9();
      at.op = oproj(b.w_o, b.b_o);
      // several slots with a small W'_q product: the attention clears the query
      // rows it read and W'_q is split over k into them (never with the fused
      // output product, whose column groups all read the same query rows)
      const bool q_clear = at.op.w == nullptr && split_small(slot0, n, d, d);
      at.clear_q = q_clear ? 1 : 0;
      // bytes: the fused output product's weights (the cache reads depend on the
      // device-side lengths and are not counted)
      launch("attn_self", at.op.w ? (double)d * d * eb() : 0.0, [&](unsigned long long* sp) {
        at.stamp = sp;
        Ops<S>::attn_self(at, n, st);
      });
      if (at.op.w == nullptr) resid("gemv_o", slot0, n, Ad16(), b.w_o, b.b_o, d, d);
      const LnNext nx = l + 1 < c.n_layer ? LnNext{L.tb[l + 1].ln1_g, L.tb[l + 1].ln1_b, false, L.tb[l + 1].w_qkv, (size_t)3 * d * d}
                                          : LnNext{L.lnf_g, L.lnf_b, true, 0, 0};
      block_tail(slot0, n, b, l, tap, nx, q_clear);
    }
  }

  bool sampling() const { return h->temperature > 0.f; }

  // vocabulary head: logits = LN_final(x) @ tok_emb^T, per-row argmax into g.
  // Drafter pass: keep/dst receive the drafted tokens (rows 1..K).  When sampling,
  // the rows' scores are logit / T plus Gumbel noise of stream `purpose` (none for
  // 0), the softmax normalisers go to rmax/rsum and the logits are kept.
  void head(int slot0, int n, const float* x, size_t g, size_t gb, float* logits, int* keep = nullptr,
            int* dst = nullptr, int purpose = 0, float* rmax = nullptr, float* rsum = nullptr) {
    GemvArgs a = gemv_base(slot0, n, wk(true));
    a.w = W(L.tok_emb); a.bias = nullptr; a.K = c.d_model; a.N = c.n_vocab;
    a.y = logits; a.ldy = c.n_vocab; a.hv = F32(L.hv); a.hi = I32(L.hi); a.nblk = L.head_blocks;
    a.suppress = h->suppress;
    if (sampling()) {
      a.inv_t = h->inv_t;
      a.rng_purpose = purpose;
      a.seed = h->seed;
      if (rmax != nullptr) {  // softmax normalisers only where acceptance needs them
        a.hm = F32(L.hm);
        a.hs = F32(L.hs);
      }
    }
    if (ln_ready) a.a = Ad32();
    else ln_operand(a, slot0, n, x, g, gb, Ad32(), true, g == L.lnf_g ? L.c_head : L.c_dhead, c.n_vocab, 0);
    ln_ready = false;
    run_gemv("head", EPI_ARGMAX, n, a);
    launch("argmax_final", kRows * n * L.head_blocks * 8.0, [&](unsigned long long*) {
      argmax_final(F32(L.hv), I32(L.hi), L.head_blocks, slot0 * kRows, n * kRows, I32(L.g), F32(L.gmax),
                   h->at<unsigned>(L.status), keep, dst, slot0, c.block_k, a.hm, a.hs, rmax, rsum, st);
    });
  }

  // Batch 1 (bf16): the history projection (K = n_tap d) split over k into about
  // 240 blocks of 64 columns whose partial sums add into the projection rows,
  // which the pass's set-up kernel cleared; 0 (one launch storing the rows) otherwise.
  int hproj_split() const {
    if (!fuse_oproj() || (c.draft_flags & WF_DRAFT_NO_HISTORY)) return 0;
    const int tiles64 = (c.d_model + 63) / 64, ksteps = c.n_tap * c.d_model / 32;
    return std::max(1, std::min(240 / tiles64, ksteps));
  }
  float* hp_clear() { return hproj_split() > 0 ? F32(L.hp) : nullptr; }

  // drafter history for pending rows (Appendix A.2): taps -> W_h -> per-block LN, k (RoPE), v
  void history_apply(int slot0, int n) {
    if (c.draft_flags & WF_DRAFT_NO_HISTORY) return;  // the variant keeps no history
    const int d = c.d_model;
    float *hp = F32(L.hp), *kvh = F32(L.kvh);
    if (const int ks = hproj_split()) {
      GemvArgs a = gemv_args(slot0, n, Atap16(), L.hproj_w, L.hproj_b, c.n_tap * d, d, hp, d,
                             Operand{nullptr, 0, OP_ROW, 0}, -1);
      a.ksplit = ks;
      run_gemv("gemv_hproj", EPI_ACC, n, a);
    } else {
      gemv("gemv_hproj", EPI_STORE, slot0, n, Atap16(), L.hproj_w, L.hproj_b, c.n_tap * d, d, hp, d);
    }
    // every block's k | v rows first (each block its own rows), then one launch
    // writes them all into the blocks' history caches
    const size_t kvs = (size_t)R9() * 2 * d;
    for (int dl = 0; dl < c.n_draft_layer; ++dl) {
      const BlockW& b = L.db[dl];
      // rows d..3d of the concatenated q|k|v matrix start d*d elements in, in either order
      gemv_ln("gemv_hist_kv", EPI_STORE, slot0, n, hp, b.ln1_g, b.ln1_b, b.c_qkv, 3 * d, d, Ad16(), b.w_qkv + (size_t)d * d,
              b.b_qkv + d, d, 2 * d, kvh + dl * kvs, 2 * d);
    }
    if (c.n_draft_layer > 0) {
      HistArgs ha{};
      ha.kv = kvh; ha.kcache = hkv(0, 0); ha.vcache = hkv(0, 1); ha.state = I32(L.state); ha.rope = F32(L.rope);
      ha.nlayer = c.n_draft_layer; ha.kv_stride = kvs;
      ha.cache_stride = (size_t)2 * c.max_batch * c.n_head * c.n_ctx * kHeadDim;  // hkv(dl + 1, .) - hkv(dl, .)
      ha.slot0 = slot0; ha.d = d; ha.n_head = c.n_head; ha.n_ctx = c.n_ctx;
      ha.status = h->at<unsigned>(L.status);
      ha.use_rope = !(c.draft_flags & WF_DRAFT_ABS_POS);
      launch("hist_write", 0, [&](unsigned long long*) { Ops<S>::hist_write(ha, n, st); });
    }
  }

  void drafter_forward(int slot0, int n, int* dst) {
    const int d = c.d_model;
    float *h_ = F32(L.h), *qkv = F32(L.qkv);
    BeginArgs ba{};
    ba.state = I32(L.state); ba.emb = W(L.tok_emb); ba.emb_kind = wk(true); ba.pos = W(L.mask); ba.h = h_;
    ba.slot0 = slot0; ba.d = d; ba.n_vocab = c.n_vocab; ba.n_ctx = c.n_ctx; ba.block_k = c.block_k;
    if (c.draft_flags & WF_DRAFT_ABS_POS) ba.pos2 = W(L.pos_emb);
    launch("begin", 0, [&](unsigned long long*) { Ops<S>::draft_begin(ba, n, st); });
    ln_ready = false;
    touch_ = Touch{nullptr, 0, 0};
    const bool xattn = !(c.draft_flags & WF_DRAFT_NO_AUDIO);
    for (int dl = 0; dl < c.n_draft_layer; ++dl) {
      const BlockW& b = L.db[dl];
      if (ln_ready) gemv("gemv_draft_qkv", EPI_STORE, slot0, n, Ad16(), b.w_qkv, b.b_qkv, d, 3 * d, qkv, 3 * d);
      else gemv_ln("gemv_draft_qkv", EPI_STORE, slot0, n, h_, b.ln1_g, b.ln1_b, b.c_qkv, 3 * d, 0, Ad16(), b.w_qkv, b.b_qkv,
                   d, 3 * d, qkv, 3 * d);
      ln_ready = false;
      AttnArgs at{};
      at.q = qkv; at.ldq = 3 * d; at.kcache = hkv(dl, 0); at.vcache = hkv(dl, 1);
      at.state = I32(L.state); at.rope = F32(L.rope); at.out = Ad16();
      at.slot0 = slot0; at.d = d; at.n_head = c.n_head; at.n_ctx = c.n_ctx;
      at.nsplit = L.nsplit_op; at.R9 = R9();
      at.draft_hist = !(c.draft_flags & WF_DRAFT_NO_HISTORY);
      at.draft_rope = !(c.draft_flags & WF_DRAFT_ABS_POS);
      launch("attn_draft", 0, [&](unsigned long long* sp) {
        at.stamp = sp;
        Ops<S>::attn_draft(at, n, st);
      });
      if (!xattn) touch_next(slot0, n, b.w_fc1, (size_t)c.d_ff * d, 64);  // the MLP follows directly
      resid("gemv_o", slot0, n, Ad16(), b.w_o, b.b_o, d, d);
      const LnNext nx = dl + 1 < c.n_draft_layer
                            ? LnNext{L.db[dl + 1].ln1_g, L.db[dl + 1].ln1_b, false, L.db[dl + 1].w_qkv, (size_t)3 * d * d}
                            : LnNext{L.dlnf_g, L.dlnf_b, true, 0, 0};
      block_tail(slot0, n, b, c.n_layer + dl, -1, nx, false, xattn);
    }
    touch_ = Touch{nullptr, 0, 0};
    head(slot0, n, h_, L.dlnf_g, L.dlnf_b, h->debug || sampling() ? F32(L.dlogits) : nullptr, I32(L.draft), dst,
         RNG_DRAFT, F32(L.dmax), F32(L.dsum));
  }

  void verify(int slot0, int n, const int* draft, int k_max, int* out, int* n_out, int* n_acc, int* done) {
    BeginArgs ba{};
    ba.state = I32(L.state); ba.draft = draft; ba.tok = I32(L.tok); ba.emb = W(L.tok_emb); ba.emb_kind = wk(true); ba.pos = W(L.pos_emb);
    ba.h = F32(L.h); ba.slot0 = slot0; ba.d = c.d_model; ba.n_vocab = c.n_vocab; ba.n_ctx = c.n_ctx;
    ba.block_k = c.block_k; ba.k_max = k_max;
    ba.page_table = I32(L.page_table); ba.pages_per_slot = L.pages_per_slot;
    ba.status = h->at<unsigned>(L.status);
    ba.hp = hp_clear();
    launch("begin", 0, [&](unsigned long long*) { Ops<S>::verify_begin(ba, n, st); });
    target_forward(slot0, n);
    head(slot0, n, F32(L.h), L.lnf_g, L.lnf_b, h->debug || sampling() ? F32(L.logits) : nullptr, nullptr, nullptr, 0,
         F32(L.tmax), F32(L.tsum));
    if (sampling()) {
      SampleArgs sa{};
      sa.state = I32(L.state); sa.tok = I32(L.tok); sa.lp = F32(L.logits); sa.lq = F32(L.dlogits);
      sa.tmax = F32(L.tmax); sa.tsum = F32(L.tsum); sa.dmax = F32(L.dmax); sa.dsum = F32(L.dsum);
      sa.sst = I32(L.sst); sa.part = F32(L.spart); sa.nsb = kSampleBlocks;
      sa.out = out; sa.n_out = n_out; sa.n_acc = n_acc; sa.done = done;
      sa.slot0 = slot0; sa.n = n; sa.block_k = c.block_k; sa.eos = c.eos_id; sa.n_ctx = c.n_ctx; sa.V = c.n_vocab;
      sa.inv_t = h->inv_t; sa.seed = h->seed;
      launch("accept", 0, [&](unsigned long long*) { accept_sample(sa, st); });
      history_apply(slot0, n);
      return;
    }
    AcceptArgs aa{};
    aa.state = I32(L.state); aa.tok = I32(L.tok); aa.g = I32(L.g); aa.out = out; aa.n_out = n_out; aa.n_acc = n_acc;
    aa.done = done; aa.slot0 = slot0; aa.n = n; aa.block_k = c.block_k; aa.eos = c.eos_id; aa.n_ctx = c.n_ctx;
    launch("accept", 0, [&](unsigned long long*) { accept_greedy(aa, st); });
    history_apply(slot0, n);
  }

  // The history already holds every verified position: each verify writes the
  // drafter history of its rows after the acceptance (Appendix A.2), so any
  // sequence of verify and draft calls sees a complete history.
  void draft(int slot0, int n, int* dst) { drafter_forward(slot0, n, dst); }

  void encode(int slot0, int n, const void* mem) {
    const size_t per = (size_t)c.n_frames * c.d_model;
    if (std::is_same<S, bf16>::value) {
      // bf16 storage: the keys and values of all blocks on the matrix cores, one
      // launch per slot for the target blocks (grid z = block) and one for the
      // drafter's (their weights sit at a fixed stride within each group)
      for (int s = 0; s < n; ++s) {
        const int slot = slot0 + s;
        auto group = [&](int first, int count, const std::vector<BlockW>& bw) {
          MmArgs a{};
          a.A = reinterpret_cast<const bf16*>(mem) + s * per;
          a.lda = c.d_model;
          a.B = reinterpret_cast<const bf16*>(W(bw[0].w_kv2));
          a.ldb = c.d_model;
          a.sB = count > 1 ? (long long)(bw[1].w_kv2 - bw[0].w_kv2) : 0;
          a.bias = reinterpret_cast<const bf16*>(W(bw[0].b_kv2));
          a.sBias = count > 1 ? (long long)(bw[1].b_kv2 - bw[0].b_kv2) : 0;
          a.M = c.n_frames;
          a.N = 2 * c.d_model;
          a.K = c.d_model;
          a.out = xkv_layer(first) + (size_t)slot * xkv_slot();
          a.sO = (long long)c.max_batch * xkv_slot();
          a.d = c.d_model;
          a.n_head = c.n_head;
          a.vt_frames = vt_frames();
          a.scale = 1.f;
          mm(a, MM_XKV, count, st);
        };
        group(0, c.n_layer, L.tb);
        if (!(c.draft_flags & WF_DRAFT_NO_AUDIO)) group(c.n_layer, c.n_draft_layer, L.db);
      }
      return;
    }
    for (int s = 0; s < n; ++s) {
      const int slot = slot0 + s;
      const int nblk = c.n_layer + ((c.draft_flags & WF_DRAFT_NO_AUDIO) ? 0 : c.n_draft_layer);
      for (int l = 0; l < nblk; ++l) {
        const BlockW& b = l < c.n_layer ? L.tb[l] : L.db[l - c.n_layer];
        XkvArgs a{};
        a.mem = reinterpret_cast<const S*>(mem) + s * per;
        a.w = W(b.w_kv2);
        a.bias = W(b.b_kv2);
        a.out = xkv_layer(l) + (size_t)slot * xkv_slot();
        a.d = c.d_model;
        a.n_head = c.n_head;
        a.n_frames = c.n_frames;
        a.vt_frames = vt_frames();
        Ops<S>::gemm_xkv(a, st);
      }
    }
  }

  void prefill(int slot0, int n, const int* tokens, int pmax, int max_len, int* first) {
    const int nchunks = (max_len + kRows - 1) / kRows;
    BeginArgs ba{};
    ba.state = I32(L.state); ba.draft = tokens; ba.tok = I32(L.tok); ba.emb = W(L.tok_emb); ba.emb_kind = wk(true); ba.pos = W(L.pos_emb);
    ba.h = F32(L.h); ba.slot0 = slot0; ba.d = c.d_model; ba.n_vocab = c.n_vocab; ba.n_ctx = c.n_ctx;
    ba.block_k = c.block_k; ba.pmax = pmax;
    ba.page_table = I32(L.page_table); ba.pages_per_slot = L.pages_per_slot;
    ba.hp = hp_clear();
    for (int ch = 0; ch < nchunks; ++ch) {
      ba.chunk = ch;
      Ops<S>::prefill_begin(ba, n, st);
      target_forward(slot0, n);
      save_last(F32(L.h), F32(L.lasth), I32(L.state), slot0, n, c.d_model, ch, st);
      history_apply(slot0, n);
    }
    ln_ready = false;  // the final LayerNorm applies to the saved last rows, not to h
    head(slot0, n, F32(L.lasth), L.lnf_g, L.lnf_b, nullptr, nullptr, nullptr, RNG_PREFILL);
    prefill_finish(I32(L.state), I32(L.g), slot0, n, c.eos_id, c.n_ctx, first, st);
  }
};

// Accumulate the durations of recorded launches (in launch order) from the stamp
// buffer; the stream must be synchronised.  Launches whose kernels take no slot
// are skipped.  Two durations per launch: the execution span (longest per-XCD
// first-wave-start to last-wave-end) and the share of the timeline, from the
// previous timed launch's last wave end to this launch's (dispatch and
// completion included, comparable to a profiler's per-dispatch duration).
int collect_stamps(Handle* h, const std::vector<ProfRec>& recs) {
  if (recs.empty()) return WF_OK;
  int top = 0;
  for (auto& r : recs) top = std::max(top, r.slot + 1);
  std::vector<unsigned long long> t((size_t)top * kStampWords);
  HIPCK(h, hipMemcpy(t.data(), h->at<unsigned long long>(h->lay.stamps), t.size() * 8, hipMemcpyDeviceToHost));
  unsigned long long prev_end = 0;
  for (auto& r : recs) {
    unsigned long long span = 0, end = 0;
    bool any = false;
    for (int x = 0; x < kStampXcds; ++x) {  // per XCD: earliest start and latest end over the residues
      unsigned long long a = ~0ull, b = 0;
      for (int j = 0; j < kStampSub; ++j) {
        const size_t w = (size_t)r.slot * kStampWords + 2 * (x * kStampSub + j);
        a = std::min(a, t[w]);
        b = std::max(b, t[w + 1]);
      }
      if (a == ~0ull || b < a) continue;
      any = true;
      span = std::max(span, b - a);
      end = std::max(end, b);
    }
    if (!any) continue;
    const unsigned long long share = prev_end && end > prev_end ? end - prev_end : span;
    prev_end = end;
    ProfAgg& g = h->prof_acc[r.tag];
    g.ms += (double)share / h->wall_khz;
    g.exec_ms += (double)span / h->wall_khz;
    g.bytes += r.bytes;
    g.n += 1;
  }
  return WF_OK;
}

// Run fn with the storage type of the handle.  When profiling, the timing slots
// are reset first (a fill kernel, so a capture records it) and an eager call
// synchronises and collects its launch durations.
template <typename Fn>
int dispatch(Handle* h, hipStream_t st, Fn&& fn) {
  const bool prof = h->prof;
  if (prof) {
    h->nstamp = 0;
    stamp_init(h->at<unsigned long long>(h->lay.stamps), kStampSlots, st);
  }
  if (h->cfg.dtype == WF_BF16) {
    fn(static_cast<bf16*>(nullptr));
  } else {
    fn(static_cast<float*>(nullptr));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(h, WF_EHIP, std::string("kernel launch: ") + hipGetErrorString(e));
  if (prof && !h->capturing) {
    HIPCK(h, hipStreamSynchronize(st));
    int r = collect_stamps(h, h->prof_recs);
    h->prof_recs.clear();
    if (r) return r;
  }
  return WF_OK;
}

int check_batch(Handle* h, int slot0, int n, bool need_live) {
  if (!h) return fail(nullptr, WF_EINVAL, "null handle");
  if (n < 1 || slot0 < 0 || slot0 + n > h->cfg.max_batch) return fail(h, WF_EINVAL, "slot range out of bounds");
  if (need_live)
    for (int s = slot0; s < slot0 + n; ++s)
      if (!h->live[s]) return fail(h, WF_ESTATE, "slot not prefilled");
  return WF_OK;
}

std::vector<float> rope_table(int n_pos) {
  std::vector<float> t((size_t)n_pos * 32 * 2);
  for (int p = 0; p < n_pos; ++p)
    for (int i = 0; i < 32; ++i) {
      const float omega = (float)std::pow(10000.0, -2.0 * i / 64.0);
      const float theta = (float)p * omega;  // fp32 product
      t[((size_t)p * 32 + i) * 2] = (float)std::cos((double)theta);
      t[((size_t)p * 32 + i) * 2 + 1] = (float)std::sin((double)theta);
    }
  return t;
}

}  // namespace

extern "C" {

int wf_workspace_bytes(const wf_config* cfg, size_t* bytes) {
  std::string why;
  if (int r = check_config(cfg, why)) return fail(nullptr, r, why);
  if (!bytes) return fail(nullptr, WF_EINVAL, "null bytes");
  Layout L;
  compute_layout(*cfg, L);
  *bytes = L.total;
  return WF_OK;
}

int wf_weight_count(const wf_config* cfg, int* n) {
  std::string why;
  if (int r = check_config(cfg, why)) return fail(nullptr, r, why);
  if (!n) return fail(nullptr, WF_EINVAL, "null n");
  Layout L;
  compute_layout(*cfg, L);
  *n = (int)manifest(*cfg, L).size();
  return WF_OK;
}

int wf_weight_numel(const wf_config* cfg, int i, int64_t* numel) {
  std::string why;
  if (int r = check_config(cfg, why)) return fail(nullptr, r, why);
  Layout L;
  compute_layout(*cfg, L);
  auto m = manifest(*cfg, L);
  if (!numel || i < 0 || i >= (int)m.size()) return fail(nullptr, WF_EINVAL, "index out of range");
  *numel = (int64_t)m[i].numel;
  return WF_OK;
}

int wf_init_weights(wf_handle** out, const wf_config* cfg, const void* const* weights, int n_weights, void* workspace,
                    size_t ws_bytes, void* stream) {
  std::string why;
  if (!out) return fail(nullptr, WF_EINVAL, "null handle pointer");
  if (int r = check_config(cfg, why)) return fail(nullptr, r, why);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) return fail(nullptr, WF_EINVAL, "workspace must be 256-byte aligned");
  Layout L;
  compute_layout(*cfg, L);
  if (ws_bytes < L.total) return fail(nullptr, WF_ESIZE, "workspace too small");
  auto man = manifest(*cfg, L);
  if (!weights || n_weights != (int)man.size()) return fail(nullptr, WF_EINVAL, "wrong number of weight tensors");
  for (int i = 0; i < n_weights; ++i)
    if (!weights[i]) return fail(nullptr, WF_EINVAL, "null weight pointer");
  Handle* h = new (std::nothrow) Handle();
  if (!h) return fail(nullptr, WF_EINVAL, "out of host memory");
  h->cfg = *cfg;
  h->lay = L;
  h->ws = static_cast<char*>(workspace);
  h->ws_bytes = ws_bytes;
  h->live.assign(cfg->max_batch, 0);
  hipStream_t st = static_cast<hipStream_t>(stream);
  auto cleanup = [&](int code, const std::string& msg) { delete h; return fail(nullptr, code, msg); };
  {
    int dev = 0, khz = 0;
    hipError_t e0 = hipGetDevice(&dev);
    if (e0 == hipSuccess) e0 = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (e0 != hipSuccess || khz <= 0) return cleanup(WF_EHIP, "wall clock rate unavailable");
    h->wall_khz = khz;
    h->device = dev;
    // the static scratch of wf_step_noalloc on this device (looked up once per device)
    e0 = scratch_setup(dev);
    if (e0 != hipSuccess) return cleanup(WF_EHIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e0));
  }
  hipError_t e = hipMemsetAsync(workspace, 0, L.total, st);
  if (e != hipSuccess) return cleanup(WF_EHIP, std::string("hipMemsetAsync: ") + hipGetErrorString(e));
  const size_t eb = elt_bytes(*cfg);
  char* wbase = h->at<char>(L.weights);
  char* stage = h->at<char>(L.xkv);
  std::vector<Mat> mats;
  manifest(*cfg, L, &mats);
  std::vector<int> last(mats.size(), -1);  // last manifest entry of each matrix
  for (int i = 0; i < n_weights; ++i)
    if (man[i].mat >= 0) last[man[i].mat] = i;
  for (int i = 0; i < n_weights; ++i) {
    const int mi = man[i].mat;
    char* dst = mi < 0 ? wbase + man[i].dst * eb : stage + (man[i].dst - mats[mi].dst) * eb;
    e = hipMemcpyAsync(dst, weights[i], man[i].numel * eb, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) return cleanup(WF_EHIP, std::string("hipMemcpyAsync: ") + hipGetErrorString(e));
    if (mi >= 0 && last[mi] == i) {
      // the whole matrix is staged: reorder it into its place
      const Mat& m = mats[mi];
      if (m.lng != kNoLn) {
        float* cols = h->at<float>(L.lncd) + m.cols;
        ln_fold_cols(stage, wbase + m.lng * eb, wbase + m.lnb * eb, m.N, m.K, cols, cols + m.N, st);
      }
      repack<bf16>(stage, wbase + m.dst * eb, m.N, m.K, m.kind, st);
      e = hipGetLastError();
      if (e != hipSuccess) return cleanup(WF_EHIP, std::string("repack: ") + hipGetErrorString(e));
    }
  }
  if (!mats.empty()) {
    e = hipMemsetAsync(stage, 0, L.stage_bytes, st);
    if (e != hipSuccess) return cleanup(WF_EHIP, std::string("hipMemsetAsync: ") + hipGetErrorString(e));
  }
  if (cfg->dtype == WF_BF16 && L.nsplit_op == 3 && (size_t)cfg->d_model <= (size_t)kLnFoldMaxK) {
    // the heads' column sums, from the caller's row-major embedding (manifest entry
    // 0), now that both final LayerNorms are in place
    float* cols = h->at<float>(L.lncd);
    const int V = cfg->n_vocab, d = cfg->d_model;
    ln_fold_cols(weights[0], wbase + L.lnf_g * eb, wbase + L.lnf_b * eb, V, d, cols + L.c_head, cols + L.c_head + V, st);
    ln_fold_cols(weights[0], wbase + L.dlnf_g * eb, wbase + L.dlnf_b * eb, V, d, cols + L.c_dhead, cols + L.c_dhead + V, st);
    e = hipGetLastError();
    if (e != hipSuccess) return cleanup(WF_EHIP, std::string("ln_fold_cols: ") + hipGetErrorString(e));
  }
  // page table: logical page j of slot s -> physical page j * max_batch + s
  std::vector<int> pt((size_t)cfg->max_batch * L.pages_per_slot);
  for (int s = 0; s < cfg->max_batch; ++s)
    for (int j = 0; j < L.pages_per_slot; ++j) pt[(size_t)s * L.pages_per_slot + j] = j * cfg->max_batch + s;
  std::vector<float> rope = rope_table(cfg->n_ctx + kRows + 1);
  e = hipMemcpyAsync(h->at<char>(L.page_table), pt.data(), pt.size() * 4, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipMemcpyAsync(h->at<char>(L.rope), rope.data(), rope.size() * 4, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return cleanup(WF_EHIP, std::string("init copy: ") + hipGetErrorString(e));
  *out = reinterpret_cast<wf_handle*>(h);
  return WF_OK;
}

int wf_encode_memory_set(wf_handle* hh, int slot0, int n, const void* mem, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (int r = check_batch(h, slot0, n, false)) return r;
  if (!mem) return fail(h, WF_EINVAL, "null memory");
  if (h->cfg.dtype == WF_BF16) {
    if (reinterpret_cast<uintptr_t>(mem) & 15) return fail(h, WF_EINVAL, "acoustic memory must be 16-byte aligned");
    MmArgs a{};
    a.M = h->cfg.n_frames; a.N = 2 * h->cfg.d_model; a.K = a.lda = a.ldb = h->cfg.d_model;
    a.d = h->cfg.d_model; a.vt_frames = xkv_vt_frames(h->cfg.n_frames);
    if (mm_check(a, MM_XKV)) return fail(h, WF_EINVAL, "acoustic K/V product: unsupported shape");
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  return dispatch(h, st, [&](auto* tag) {
    using S = std::remove_pointer_t<decltype(tag)>;
    Runner<S>(h, st).encode(slot0, n, mem);
  });
}

int wf_prefill(wf_handle* hh, int slot0, int n, const int32_t* tokens, int pmax, const int32_t* lens,
               const int32_t* max_new, int32_t* first, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (int r = check_batch(h, slot0, n, false)) return r;
  if (!tokens || !lens || !max_new || pmax < 1) return fail(h, WF_EINVAL, "null argument");
  int max_len = 0;
  for (int s = 0; s < n; ++s) {
    if (lens[s] < 1 || lens[s] > pmax || lens[s] > h->cfg.n_ctx) return fail(h, WF_EINVAL, "prompt length out of range");
    if (max_new[s] < 1) return fail(h, WF_EINVAL, "max_new must be >= 1");
    max_len = std::max(max_len, (int)lens[s]);
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  std::vector<int> init((size_t)n * kStateInts, 0);
  for (int s = 0; s < n; ++s) {
    init[(size_t)s * kStateInts + ST_LEN] = lens[s];
    init[(size_t)s * kStateInts + ST_MAX_NEW] = max_new[s];
  }
  HIPCK(h, hipMemcpyAsync(h->at<int>(h->lay.state) + (size_t)slot0 * kStateInts, init.data(), init.size() * 4,
                          hipMemcpyHostToDevice, st));
  int r = dispatch(h, st, [&](auto* tag) {
    using S = std::remove_pointer_t<decltype(tag)>;
    Runner<S>(h, st).prefill(slot0, n, tokens, pmax, max_len, first);
  });
  if (r) return r;
  HIPCK(h, hipStreamSynchronize(st));
  for (int s = slot0; s < slot0 + n; ++s) h->live[s] = 1;
  return WF_OK;
}

// Destroy every captured graph.
static void clear_graphs(Handle* h) {
  for (auto& kv : h->graphs) (void)hipGraphExecDestroy(kv.second);
  h->graphs.clear();
  h->graph_recs.clear();
}

int wf_set_sampling(wf_handle* hh, float temperature, uint64_t seed, const uint8_t* suppress) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h) return fail(nullptr, WF_EINVAL, "null handle");
  if (!(temperature >= 0.f) || std::isinf(temperature)) return fail(h, WF_EINVAL, "temperature must be finite and >= 0");
  h->temperature = temperature;
  h->inv_t = temperature > 0.f ? (float)(1.0 / (double)temperature) : 0.f;
  h->seed = seed;
  h->suppress = suppress;
  // captured steps bake the sampling parameters in
  clear_graphs(h);
  return WF_OK;
}

int wf_draft(wf_handle* hh, int slot0, int n, int32_t* draft, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (int r = check_batch(h, slot0, n, true)) return r;
  hipStream_t st = static_cast<hipStream_t>(stream);
  return dispatch(h, st, [&](auto* tag) {
    using S = std::remove_pointer_t<decltype(tag)>;
    Runner<S>(h, st).draft(slot0, n, draft);
  });
}

int wf_verify_accept(wf_handle* hh, int slot0, int n, const int32_t* draft, int k_max, int32_t* out, int32_t* n_out,
                     int32_t* n_acc, int32_t* done, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (int r = check_batch(h, slot0, n, true)) return r;
  if (!draft) return fail(h, WF_EINVAL, "null draft");
  if (k_max < 0 || k_max > h->cfg.block_k) return fail(h, WF_EINVAL, "k_max out of range");
  hipStream_t st = static_cast<hipStream_t>(stream);
  return dispatch(h, st, [&](auto* tag) {
    using S = std::remove_pointer_t<decltype(tag)>;
    Runner<S>(h, st).verify(slot0, n, draft, k_max, out, n_out, n_acc, done);
  });
}

static int step_enqueue(Handle* h, int slot0, int n, int k_max, const int32_t* ovr, int32_t* out, int32_t* n_out,
                        int32_t* n_acc, int32_t* done, hipStream_t st) {
  return dispatch(h, st, [&](auto* tag) {
    using S = std::remove_pointer_t<decltype(tag)>;
    Runner<S> R(h, st);
    // k_max = 0 verifies the anchor alone (plain decoding): no proposal is used,
    // so the drafter does not run
    if (k_max > 0) R.draft(slot0, n, nullptr);
    const int* d = ovr ? ovr : h->at<int>(h->lay.draft) + (size_t)slot0 * h->cfg.block_k;
    R.verify(slot0, n, d, k_max, out, n_out, n_acc, done);
  });
}

int wf_step(wf_handle* hh, int slot0, int n, int k_max, const int32_t* ovr, int32_t* out, int32_t* n_out,
            int32_t* n_acc, int32_t* done, int use_graph, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (int r = check_batch(h, slot0, n, true)) return r;
  if (k_max < 0 || k_max > h->cfg.block_k) return fail(h, WF_EINVAL, "k_max out of range");
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!use_graph) return step_enqueue(h, slot0, n, k_max, ovr, out, n_out, n_acc, done, st);
  if (!st) return fail(h, WF_EINVAL, "graph replay needs a non-null stream");
  GraphKey key{slot0, n, k_max, ovr, out, n_out, n_acc, done, h->prof};
  auto it = h->graphs.find(key);
  if (it == h->graphs.end()) {
    h->cap_recs.clear();
    HIPCK(h, hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
    h->capturing = true;
    int r = step_enqueue(h, slot0, n, k_max, ovr, out, n_out, n_acc, done, st);
    h->capturing = false;
    hipGraph_t g = nullptr;
    hipError_t e = hipStreamEndCapture(st, &g);
    auto drop_recs = [&] { h->cap_recs.clear(); };
    if (r) { if (g) (void)hipGraphDestroy(g); drop_recs(); return r; }
    if (e != hipSuccess) { drop_recs(); return fail(h, WF_EHIP, std::string("hipStreamEndCapture: ") + hipGetErrorString(e)); }
    hipGraphExec_t ex = nullptr;
    e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
    (void)hipGraphDestroy(g);
    if (e != hipSuccess) { drop_recs(); return fail(h, WF_EHIP, std::string("hipGraphInstantiate: ") + hipGetErrorString(e)); }
    it = h->graphs.emplace(key, ex).first;
    if (key.prof) h->graph_recs[key] = h->cap_recs;
    h->cap_recs.clear();
  }
  HIPCK(h, hipGraphLaunch(it->second, st));
  if (key.prof) {  // profiled replay: read this replay's launch durations now
    HIPCK(h, hipStreamSynchronize(st));
    return collect_stamps(h, h->graph_recs[key]);
  }
  return WF_OK;
}

int wf_step_noalloc(wf_handle* hh, int slot0, int n, int k_max, const int32_t* ovr, int32_t* out, int32_t* n_out,
                    int32_t* n_acc, int32_t* done, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (int r = check_batch(h, slot0, n, true)) return r;
  if (k_max < 0 || k_max > h->cfg.block_k) return fail(h, WF_EINVAL, "k_max out of range");
  if (h->capturing) return fail(h, WF_ESTATE, "wf_step_noalloc inside a wf_step capture");
  const size_t need = h->transient_bytes();
  if (need > kScratchBytes) {
    char msg[160];
    snprintf(msg, sizeof(msg), "per-call buffers need %zu bytes; the static scratch holds %zu (use wf_step)", need,
             kScratchBytes);
    return fail(h, WF_ESIZE, msg);
  }
  char* p = scratch_of(h->device);
  if (!p) return fail(h, WF_EHIP, "static scratch not set up on the handle's device");
  hipStream_t st = static_cast<hipStream_t>(stream);
  // the scratch keeps the previous call's contents (possibly of another handle and
  // layout): start from zeros, as the workspace does after wf_init_weights
  HIPCK(h, hipMemsetAsync(p, 0, need, st));
  const bool prof = h->prof;
  h->prof = false;  // timing stamps are not taken in this variant
  h->scratch = p;
  const int r = step_enqueue(h, slot0, n, k_max, ovr, out, n_out, n_acc, done, st);
  h->scratch = nullptr;
  h->prof = prof;
  return r;
}

int wf_debug_ptr(wf_handle* hh, int which, void** ptr) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h || !ptr) return fail(h, WF_EINVAL, "null argument");
  switch (which) {
    case 0: *ptr = h->at<void>(h->lay.logits); break;
    case 1: *ptr = h->at<void>(h->lay.dlogits); break;
    case 2: *ptr = h->at<void>(h->lay.state); break;
    case 3: *ptr = h->at<void>(h->lay.draft); break;
    default: return fail(h, WF_EINVAL, "unknown debug view");
  }
  return WF_OK;
}

int wf_set_debug(wf_handle* hh, int enable) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h) return fail(nullptr, WF_EINVAL, "null handle");
  if (h->debug != (enable != 0)) clear_graphs(h);
  h->debug = enable != 0;
  return WF_OK;
}

int wf_profile_enable(wf_handle* hh, int enable) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h) return fail(nullptr, WF_EINVAL, "null handle");
  h->prof = enable != 0;
  return WF_OK;
}

int wf_profile_summary(wf_handle* hh, char* buf, size_t len) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h || !buf || len == 0) return fail(h, WF_EINVAL, "null argument");
  std::map<std::string, ProfAgg> agg;
  agg.swap(h->prof_acc);
  std::string js = "{";
  bool first = true;
  for (auto& kv : agg) {
    char item[256];
    snprintf(item, sizeof(item), "%s\"%s\": {\"launches\": %ld, \"ms\": %.6f, \"exec_ms\": %.6f, \"bytes\": %.1f}",
             first ? "" : ", ", kv.first.c_str(), kv.second.n, kv.second.ms, kv.second.exec_ms, kv.second.bytes);
    js += item;
    first = false;
  }
  js += "}";
  if (js.size() + 1 > len) return fail(h, WF_ESIZE, "summary buffer too small");
  memcpy(buf, js.c_str(), js.size() + 1);
  return WF_OK;
}

int wf_status(wf_handle* hh, uint32_t* flags, void* stream) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h || !flags) return fail(h, WF_EINVAL, "null argument");
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t v = 0;
  HIPCK(h, hipMemcpyAsync(&v, h->at<char>(h->lay.status), 4, hipMemcpyDeviceToHost, st));
  HIPCK(h, hipStreamSynchronize(st));
  *flags = v;
  if (v) HIPCK(h, hipMemsetAsync(h->at<char>(h->lay.status), 0, 4, st));
  return WF_OK;
}

int wf_release(wf_handle* hh) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  if (!h) return fail(nullptr, WF_EINVAL, "null handle");
  clear_graphs(h);
  delete h;
  return WF_OK;
}

int wf_rng_words_host(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out) {
  if (!out || n < 0) return fail(nullptr, WF_EINVAL, "null output or negative count");
  for (int v = 0; v < n; ++v) out[v] = rng_word(seed, purpose, slot, step, pos, v);
  return WF_OK;
}

int wf_rng_words_device(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out, void* stream) {
  if (!out || n < 0) return fail(nullptr, WF_EINVAL, "null output or negative count");
  rng_words_device(seed, purpose, slot, step, pos, n, out, static_cast<hipStream_t>(stream));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(nullptr, WF_EHIP, std::string("kernel launch: ") + hipGetErrorString(e));
  return WF_OK;
}

const char* wf_strerror(int code) {
  switch (code) {
    case WF_OK: return "ok";
    case WF_EINVAL: return "invalid argument";
    case WF_ESTATE: return "invalid state";
    case WF_ESIZE: return "workspace too small";
    case WF_EHIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

const char* wf_last_error(wf_handle* hh) {
  Handle* h = reinterpret_cast<Handle*>(hh);
  return h ? h->err.c_str() : g_err.c_str();
}

}  // extern "C"
