// Host runtime of the Whisper audio encoder: configuration checks, workspace
// carve-up, parameter copy and the enqueue sequence from waveform to acoustic
// memory (the frozen encoder whose output A = E(x) both the target and the
// drafter read, Section 3.2; it runs once per request over a 30 s window).
// Every device buffer lives in the caller's workspace; nothing here allocates
// device memory.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/wf.h"
#include "wf_common.h"
#include "wf_kernels.h"

using namespace wf;

namespace {

thread_local std::string g_enc_err;

struct EncLayer {
  size_t ln1_g, ln1_b, wqkv, bqkv, wo, bo, ln2_g, ln2_b, w1, b1, w2, b2;  // bf16 element offsets
};

struct EncLayout {
  int T, Tp, Kp1, nb;  // mel frames, positions padded to 64, first-conv row length, FFT bins
  // bf16 weight element offsets
  size_t conv1, conv1_b, conv2, conv2_b, lnp_g, lnp_b, wtotal;
  std::vector<EncLayer> layers;
  // byte offsets
  size_t weights, pos, window, twiddle, filters, fband, gmax, logmel, rows1, z, rows2, x, a, qk, vt, o, u, total;
};

struct Enc {
  wf_encoder_config cfg;
  EncLayout lay;
  char* ws;
  std::string err;
  template <typename T>
  T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
  const bf16* W(size_t e) const { return at<const bf16>(lay.weights) + e; }
};

int efail(Enc* e, int code, const std::string& msg) {
  if (e) e->err = msg;
  g_enc_err = msg;
  return code;
}

size_t up(size_t v, size_t a) { return (v + a - 1) / a * a; }

int check(const wf_encoder_config* c, std::string& why) {
  if (!c) { why = "null config"; return WF_EINVAL; }
  if (c->n_head <= 0 || c->d_model != c->n_head * kHeadDim) { why = "head width must be 64"; return WF_EINVAL; }
  if (c->d_model > kMaxEncD) { why = "d_model must be <= 2048"; return WF_EINVAL; }
  if (c->n_layer < 1 || c->d_ff < kMmK || c->d_ff % kMmK) { why = "n_layer >= 1, d_ff a positive multiple of 64"; return WF_EINVAL; }
  if (c->n_ctx < 1 || up(c->n_ctx, 64) > (size_t)kMaxEncCtx) { why = "n_ctx must be in [1, 2048]"; return WF_EINVAL; }
  if (c->n_mels < 1 || c->n_fft < 2 || c->n_fft > kMaxFft || c->n_fft % 2 || c->hop < 1) {
    why = "n_mels >= 1, n_fft even and <= 512, hop >= 1";
    return WF_EINVAL;
  }
  if (2 * c->n_ctx * c->hop <= c->n_fft / 2) { why = "window longer than the signal"; return WF_EINVAL; }
  if (c->sample_rate < 1) { why = "sample_rate must be positive"; return WF_EINVAL; }
  return WF_OK;
}

void layout(const wf_encoder_config& c, EncLayout& L) {
  const size_t d = c.d_model, F = c.d_ff;
  L.T = 2 * c.n_ctx;
  L.Tp = (int)up(c.n_ctx, 64);
  L.Kp1 = (int)up(3 * (size_t)c.n_mels, kMmK);
  L.nb = c.n_fft / 2 + 1;
  size_t w = 0;
  auto take = [&](size_t n) { size_t o = w; w = up(w + n, 128); return o; };
  L.conv1 = take(d * L.Kp1); L.conv1_b = take(d);
  L.conv2 = take(d * 3 * d); L.conv2_b = take(d);
  L.layers.clear();
  for (int l = 0; l < c.n_layer; ++l) {
    EncLayer e;
    e.ln1_g = take(d); e.ln1_b = take(d);
    e.wqkv = take(3 * d * d); e.bqkv = take(3 * d);
    e.wo = take(d * d); e.bo = take(d);
    e.ln2_g = take(d); e.ln2_b = take(d);
    e.w1 = take(F * d); e.b1 = take(F);
    e.w2 = take(d * F); e.b2 = take(d);
    L.layers.push_back(e);
  }
  L.lnp_g = take(d); L.lnp_b = take(d);
  L.wtotal = w;
  size_t o = 0;
  auto region = [&](size_t bytes) { size_t r = o; o = up(o + bytes, 256); return r; };
  const size_t H = c.n_head, n = c.n_ctx, T = L.T;
  L.weights = region(w * 2);
  L.pos = region(n * d * 4);
  L.window = region((size_t)c.n_fft * 8);
  L.twiddle = region((size_t)c.n_fft * 16);
  L.filters = region((size_t)c.n_mels * L.nb * 8);
  L.fband = region((size_t)c.n_mels * 8);
  L.gmax = region(4);
  L.logmel = region(T * c.n_mels * 4);
  L.rows1 = region(T * L.Kp1 * 2);
  L.z = region(T * d * 2);
  L.rows2 = region(n * 3 * d * 2);
  L.x = region(n * d * 4);
  L.a = region(n * d * 2);
  L.qk = region(n * 2 * d * 2);
  L.vt = region(H * kHeadDim * L.Tp * 2);
  L.o = region(n * d * 2);
  L.u = region(n * F * 2);
  L.total = o;
}

// manifest entry i -> (element count, destination, row copy (rows, src row, dst row) or plain)
struct EncEntry {
  size_t numel, dst;
  size_t rows, src_row, dst_row;  // rows > 0: a matrix copied row by row into a wider destination
};

std::vector<EncEntry> manifest(const wf_encoder_config& c, const EncLayout& L) {
  const size_t d = c.d_model, F = c.d_ff, m = c.n_mels;
  std::vector<EncEntry> v;
  v.push_back({d * m * 3, L.conv1, d, 3 * m, (size_t)L.Kp1});  // [d, n_mels, 3] -> rows of Kp1
  v.push_back({d, L.conv1_b, 0, 0, 0});
  v.push_back({d * d * 3, L.conv2, 0, 0, 0});                  // [d, d, 3] = rows of 3 d
  v.push_back({d, L.conv2_b, 0, 0, 0});
  for (auto& e : L.layers) {
    v.push_back({d, e.ln1_g, 0, 0, 0}); v.push_back({d, e.ln1_b, 0, 0, 0});
    v.push_back({d * d, e.wqkv, 0, 0, 0}); v.push_back({d, e.bqkv, 0, 0, 0});          // q.w, q.b
    v.push_back({d * d, e.wqkv + d * d, 0, 0, 0});                                      // k.w (no bias)
    v.push_back({d * d, e.wqkv + 2 * d * d, 0, 0, 0}); v.push_back({d, e.bqkv + 2 * d, 0, 0, 0});  // v.w, v.b
    v.push_back({d * d, e.wo, 0, 0, 0}); v.push_back({d, e.bo, 0, 0, 0});
    v.push_back({d, e.ln2_g, 0, 0, 0}); v.push_back({d, e.ln2_b, 0, 0, 0});
    v.push_back({F * d, e.w1, 0, 0, 0}); v.push_back({F, e.b1, 0, 0, 0});
    v.push_back({d * F, e.w2, 0, 0, 0}); v.push_back({d, e.b2, 0, 0, 0});
  }
  v.push_back({d, L.lnp_g, 0, 0, 0}); v.push_back({d, L.lnp_b, 0, 0, 0});
  return v;
}

// Slaney mel scale: 200/3 Hz per mel below 1 kHz, a factor 6.4 per 27 mels above.
double hz2mel(double f) { return f < 1000.0 ? f * 3.0 / 200.0 : 15.0 + std::log(f / 1000.0) * 27.0 / std::log(6.4); }
double mel2hz(double m) { return m < 15.0 ? m * 200.0 / 3.0 : 1000.0 * std::exp((m - 15.0) * std::log(6.4) / 27.0); }

// Host tables: sinusoid positions, window, DFT twiddles, unit-area triangular mel filters.
void tables(const wf_encoder_config& c, const EncLayout& L, std::vector<float>& pos, std::vector<double>& win,
            std::vector<double>& tw, std::vector<double>& filt, std::vector<int>& band) {
  const int d = c.d_model, half = d / 2, N = c.n_fft;
  pos.assign((size_t)c.n_ctx * d, 0.f);
  const double inc = std::log(10000.0) / (half - 1);
  for (int t = 0; t < c.n_ctx; ++t)
    for (int i = 0; i < half; ++i) {
      const double a = t * std::exp(-inc * i);
      pos[(size_t)t * d + i] = (float)std::sin(a);
      pos[(size_t)t * d + half + i] = (float)std::cos(a);
    }
  win.resize(N);
  tw.resize(2 * N);
  const double pi = 3.14159265358979323846;
  for (int i = 0; i < N; ++i) {
    win[i] = 0.5 - 0.5 * std::cos(2 * pi * i / N);
    tw[2 * i] = std::cos(2 * pi * i / N);
    tw[2 * i + 1] = -std::sin(2 * pi * i / N);
  }
  const int nb = L.nb;
  filt.assign((size_t)c.n_mels * nb, 0.0);
  band.assign(2 * (size_t)c.n_mels, 0);
  const double top = hz2mel(c.sample_rate / 2.0);
  std::vector<double> corner(c.n_mels + 2);
  for (int i = 0; i < c.n_mels + 2; ++i) corner[i] = mel2hz(top * i / (c.n_mels + 1));
  for (int m = 0; m < c.n_mels; ++m) {
    const double lo = corner[m], ce = corner[m + 1], hi = corner[m + 2];
    int first = nb, last = 0;
    for (int k = 0; k < nb; ++k) {
      const double f = (double)k * c.sample_rate / N;
      const double w = std::max(0.0, std::min((f - lo) / (ce - lo), (hi - f) / (hi - ce))) * 2.0 / (hi - lo);
      filt[(size_t)m * nb + k] = w;
      if (w > 0) { first = std::min(first, k); last = k + 1; }
    }
    band[2 * m] = first < last ? first : 0;
    band[2 * m + 1] = first < last ? last : 0;
  }
}

}  // namespace

struct wf_encoder {
  Enc e;
};

extern "C" {

int wf_encoder_workspace_bytes(const wf_encoder_config* cfg, size_t* bytes) {
  std::string why;
  if (int r = check(cfg, why)) return efail(nullptr, r, why);
  if (!bytes) return efail(nullptr, WF_EINVAL, "null bytes");
  EncLayout L;
  layout(*cfg, L);
  *bytes = L.total;
  return WF_OK;
}

int wf_encoder_weight_count(const wf_encoder_config* cfg, int* n) {
  std::string why;
  if (int r = check(cfg, why)) return efail(nullptr, r, why);
  if (!n) return efail(nullptr, WF_EINVAL, "null n");
  EncLayout L;
  layout(*cfg, L);
  *n = (int)manifest(*cfg, L).size();
  return WF_OK;
}

int wf_encoder_weight_numel(const wf_encoder_config* cfg, int i, int64_t* numel) {
  std::string why;
  if (int r = check(cfg, why)) return efail(nullptr, r, why);
  EncLayout L;
  layout(*cfg, L);
  auto m = manifest(*cfg, L);
  if (!numel || i < 0 || i >= (int)m.size()) return efail(nullptr, WF_EINVAL, "index out of range");
  *numel = (int64_t)m[i].numel;
  return WF_OK;
}

int wf_encoder_init(wf_encoder** out, const wf_encoder_config* cfg, const void* const* weights, int n_weights,
                    void* workspace, size_t ws_bytes, void* stream) {
  std::string why;
  if (!out) return efail(nullptr, WF_EINVAL, "null handle pointer");
  if (int r = check(cfg, why)) return efail(nullptr, r, why);
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255)) return efail(nullptr, WF_EINVAL, "workspace must be 256-byte aligned");
  EncLayout L;
  layout(*cfg, L);
  if (ws_bytes < L.total) return efail(nullptr, WF_ESIZE, "workspace too small");
  auto man = manifest(*cfg, L);
  if (!weights || n_weights != (int)man.size()) return efail(nullptr, WF_EINVAL, "weight count does not match the manifest");
  for (int i = 0; i < n_weights; ++i)
    if (!weights[i]) return efail(nullptr, WF_EINVAL, "null weight pointer");
  wf_encoder* h = new (std::nothrow) wf_encoder();
  if (!h) return efail(nullptr, WF_EINVAL, "out of host memory");
  Enc& e = h->e;
  e.cfg = *cfg;
  e.lay = L;
  e.ws = static_cast<char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  auto bail = [&](hipError_t err, const char* what) {
    delete h;
    return efail(nullptr, WF_EHIP, std::string(what) + ": " + hipGetErrorString(err));
  };
  hipError_t err = hipMemsetAsync(workspace, 0, L.weights + L.wtotal * 2, st);  // weights incl. padding
  if (err != hipSuccess) return bail(err, "hipMemsetAsync");
  char* wb = e.at<char>(L.weights);
  for (int i = 0; i < n_weights; ++i) {
    const EncEntry& m = man[i];
    if (m.rows)
      err = hipMemcpy2DAsync(wb + m.dst * 2, m.dst_row * 2, weights[i], m.src_row * 2, m.src_row * 2, m.rows,
                             hipMemcpyDeviceToDevice, st);
    else
      err = hipMemcpyAsync(wb + m.dst * 2, weights[i], m.numel * 2, hipMemcpyDeviceToDevice, st);
    if (err != hipSuccess) return bail(err, "weight copy");
  }
  std::vector<float> pos;
  std::vector<double> win, tw, filt;
  std::vector<int> band;
  tables(*cfg, L, pos, win, tw, filt, band);
  err = hipMemcpyAsync(e.at<void>(L.pos), pos.data(), pos.size() * 4, hipMemcpyHostToDevice, st);
  if (err == hipSuccess) err = hipMemcpyAsync(e.at<void>(L.window), win.data(), win.size() * 8, hipMemcpyHostToDevice, st);
  if (err == hipSuccess) err = hipMemcpyAsync(e.at<void>(L.twiddle), tw.data(), tw.size() * 8, hipMemcpyHostToDevice, st);
  if (err == hipSuccess) err = hipMemcpyAsync(e.at<void>(L.filters), filt.data(), filt.size() * 8, hipMemcpyHostToDevice, st);
  if (err == hipSuccess) err = hipMemcpyAsync(e.at<void>(L.fband), band.data(), band.size() * 4, hipMemcpyHostToDevice, st);
  if (err == hipSuccess) err = hipStreamSynchronize(st);  // the host tables go out of scope
  if (err != hipSuccess) return bail(err, "table copy");
  *out = h;
  return WF_OK;
}

// The frontend of one waveform: log-mel features into the workspace (and
// optionally the scaled features [n_mels][frames] into mel_out).
static void enc_frontend(Enc& e, const float* audio, float* mel_out, hipStream_t st) {
  const EncLayout& L = e.lay;
  LogmelArgs a{};
  a.audio = audio;
  a.n_samples = L.T * e.cfg.hop;
  a.n_fft = e.cfg.n_fft;
  a.hop = e.cfg.hop;
  a.n_frames = L.T;
  a.n_mels = e.cfg.n_mels;
  a.window = e.at<double>(L.window);
  a.twiddle = e.at<double>(L.twiddle);
  a.filters = e.at<double>(L.filters);
  a.fband = e.at<int>(L.fband);
  a.logmel = e.at<float>(L.logmel);
  a.gmax = e.at<int>(L.gmax);
  a.rows = e.at<bf16>(L.rows1);
  a.ld1 = L.Kp1;
  a.mel_out = mel_out;
  logmel(a, st);
}

static MmArgs mm_args(const bf16* A, long long lda, const bf16* B, long long ldb, const bf16* bias, int M, int N, int K,
                      void* out, long long ldo) {
  MmArgs a{};
  a.A = A; a.lda = lda; a.B = B; a.ldb = ldb; a.bias = bias;
  a.M = M; a.N = N; a.K = K; a.out = out; a.ldo = ldo; a.scale = 1.f;
  return a;
}

// Waveform -> acoustic memory [n_ctx][d] (bf16) for one request.
static void enc_forward(Enc& e, const float* audio, bf16* mem, hipStream_t st) {
  const wf_encoder_config& c = e.cfg;
  const EncLayout& L = e.lay;
  const int d = c.d_model, F = c.d_ff, H = c.n_head, n = c.n_ctx;
  enc_frontend(e, audio, nullptr, st);
  bf16 *z = e.at<bf16>(L.z), *rows2 = e.at<bf16>(L.rows2), *a = e.at<bf16>(L.a), *qk = e.at<bf16>(L.qk);
  bf16 *vt = e.at<bf16>(L.vt), *o = e.at<bf16>(L.o), *u = e.at<bf16>(L.u);
  float* x = e.at<float>(L.x);
  // stem: conv1 + GELU, conv2 (stride 2) + GELU + positions
  mm(mm_args(e.at<bf16>(L.rows1), L.Kp1, e.W(L.conv1), L.Kp1, e.W(L.conv1_b), L.T, d, L.Kp1, z, d), MM_BF16_GELU, 1, st);
  conv_rows_s2(z, rows2, L.T, n, d, st);
  {
    MmArgs m = mm_args(rows2, 3 * d, e.W(L.conv2), 3 * d, e.W(L.conv2_b), n, d, 3 * d, x, d);
    m.add = e.at<float>(L.pos);
    m.ldadd = d;
    mm(m, MM_GELU_ADD_F32, 1, st);
  }
  for (const EncLayer& w : L.layers) {
    ln_rows(x, e.W(w.ln1_g), e.W(w.ln1_b), a, n, d, d, st);
    {  // q | k row-major, v transposed per head [head][dim][Tp]
      MmArgs m = mm_args(a, d, e.W(w.wqkv), d, e.W(w.bqkv), n, 3 * d, d, qk, 2 * d);
      m.out2 = vt;
      m.d = d;
      m.n_head = H;
      m.vt_frames = L.Tp;
      mm(m, MM_QKV_ENC, 1, st);
    }
    {  // softmax(q k^T / 8) v per head, fused (scores stay on chip)
      EncAttnArgs at{};
      at.qk = qk; at.ldqk = 2 * d; at.vt = vt; at.Tp = L.Tp; at.o = o; at.ldo = d; at.n = n; at.d = d;
      enc_attention(at, H, st);
    }
    mm(mm_args(o, d, e.W(w.wo), d, e.W(w.bo), n, d, d, x, d), MM_RESID, 1, st);
    ln_rows(x, e.W(w.ln2_g), e.W(w.ln2_b), a, n, d, d, st);
    mm(mm_args(a, d, e.W(w.w1), d, e.W(w.b1), n, F, d, u, F), MM_BF16_GELU, 1, st);
    mm(mm_args(u, F, e.W(w.w2), F, e.W(w.b2), n, d, F, x, d), MM_RESID, 1, st);
  }
  ln_rows(x, e.W(L.lnp_g), e.W(L.lnp_b), mem, n, d, d, st);
}

int wf_encoder_run(wf_encoder* h, int n, const float* audio, void* mem, void* stream) {
  if (!h) return efail(nullptr, WF_EINVAL, "null handle");
  Enc& e = h->e;
  if (n < 1 || !audio || !mem) return efail(&e, WF_EINVAL, "null argument or n < 1");
  if (reinterpret_cast<uintptr_t>(mem) & 15) return efail(&e, WF_EINVAL, "memory output must be 16-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const size_t ns = (size_t)e.lay.T * e.cfg.hop, per = (size_t)e.cfg.n_ctx * e.cfg.d_model;
  for (int r = 0; r < n; ++r) enc_forward(e, audio + r * ns, static_cast<bf16*>(mem) + r * per, st);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return efail(&e, WF_EHIP, std::string("kernel launch: ") + hipGetErrorString(err));
  return WF_OK;
}

int wf_encoder_logmel(wf_encoder* h, const float* audio, float* mel, void* stream) {
  if (!h) return efail(nullptr, WF_EINVAL, "null handle");
  Enc& e = h->e;
  if (!audio || !mel) return efail(&e, WF_EINVAL, "null argument");
  enc_frontend(e, audio, mel, static_cast<hipStream_t>(stream));
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return efail(&e, WF_EHIP, std::string("kernel launch: ") + hipGetErrorString(err));
  return WF_OK;
}

int wf_encoder_release(wf_encoder* h) {
  delete h;
  return WF_OK;
}

const char* wf_encoder_last_error(wf_encoder* h) { return h ? h->e.err.c_str() : g_enc_err.c_str(); }

}  // extern "C"
