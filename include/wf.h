/*
 * wf.h - C ABI of the Whisper-Flash draft-and-verify step for MI355X (gfx950).
 *
 * One speculative round of Whisper-Flash decoding (Section 3.1 and Figure 1
 * of the paper): a two-block drafter fills K = 8 mask positions after the
 * anchor (Section 3.2, Eq. 2), the frozen Whisper decoder verifies the anchor
 * plus the candidates in one causal pass, the longest agreeing prefix is kept
 * (or the rejection rule is applied when sampling), and the target cache,
 * drafter history and anchor advance (Appendix A.1).
 *
 * Conventions
 *  - Every function returns an int status: WF_OK (0) or a negative WF_E* code.
 *    wf_strerror() maps a code to text; wf_last_error() gives the message of
 *    the last failed call on a handle.  Host-side checks run before anything
 *    is enqueued; a call that fails them leaves all state untouched.
 *  - Pointers marked "device" are device memory owned by the caller.  The
 *    library never allocates device memory: all of its state lives in one
 *    caller-provided workspace of wf_workspace_bytes() bytes.
 *  - Work is enqueued on the caller's HIP stream (passed as void*, 0 = null
 *    stream) and is complete when that stream has synchronised.  Calls on one
 *    handle must be issued on one stream (or externally ordered).
 *  - A batch is a contiguous range of slots [slot0, slot0 + n); each slot is
 *    one request.  Per-slot decoding state (cache length, anchor, counters,
 *    done flag) lives on the device, so steps never synchronise with the host.
 *  - Storage type (wf_config.dtype): WF_F32 stores weights, acoustic memory and
 *    all caches in fp32; WF_BF16 stores them in bf16.  Activations, residual
 *    stream, LayerNorm, softmax, GELU, logits and all accumulation are fp32 in
 *    both.
 *  - Token ids are int32.
 */
#ifndef WF_H
#define WF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define WF_OK 0
#define WF_EINVAL (-1)   /* bad argument (null pointer, size, range, config) */
#define WF_ESTATE (-2)   /* call not valid in the current state (e.g. step before prefill) */
#define WF_ESIZE (-3)    /* workspace too small */
#define WF_EHIP (-4)     /* a HIP runtime call failed */

#define WF_F32 0
#define WF_BF16 1

/* Device status word bits (wf_status). */
#define WF_STATUS_NONFINITE_LOGITS 0x1u  /* a verified row's logits had NaN/Inf */
#define WF_STATUS_POSITION_OVERFLOW 0x2u /* a pass or history write at or beyond n_ctx was refused:
                                            a live, unfinished slot whose cache length reached n_ctx
                                            (the budget rule of Appendix A.1 never produces one; the
                                            bit reports a state corrupted from outside) */

#define WF_MAX_TAPS 8

/* Drafter variants of the paper's ablations (wf_config.draft_flags; Section 5.4
 * Table 3 and Appendix Table A4).  0 is the paper's drafter. */
#define WF_DRAFT_NO_AUDIO 0x1u   /* blocks without the cross-attention sub-layer (and its
                                    LayerNorm): the manifest omits those eight tensors */
#define WF_DRAFT_NO_HISTORY 0x2u /* no target history: the manifest omits hproj.w/b and
                                    the block attends to its own nine rows only */
#define WF_DRAFT_ABS_POS 0x4u    /* absolute positions: no RoPE; the target's position
                                    table (shared, like the embedding) is added to the
                                    block rows at positions t..t+8 */

/*
 * Model and batch shape.  The target is a Whisper decoder (Section 4: Whisper
 * large-v3 has n_layer 32, d_model 1280, n_head 20, d_ff 5120, n_vocab 51866,
 * n_ctx 448, n_frames 1500); the drafter has n_draft_layer blocks of the same
 * width (2 in the paper), a block of block_k mask positions (8, Eq. 2) and a
 * history memory from target blocks taps[0..n_tap) (zero-based, Appendix A.2:
 * 1, 8, 15, 22, 29).  Head width must be 64.
 */
typedef struct wf_config {
  int32_t n_layer;
  int32_t d_model;
  int32_t n_head;
  int32_t d_ff;
  int32_t n_vocab;
  int32_t n_ctx;
  int32_t n_frames;
  int32_t n_draft_layer;
  int32_t block_k;          /* must be 8 */
  int32_t n_tap;
  int32_t taps[WF_MAX_TAPS];
  int32_t eos_id;           /* end-of-transcript id, or -1 for none */
  int32_t dtype;            /* WF_F32 or WF_BF16 */
  int32_t max_batch;        /* number of slots */
  int32_t draft_flags;      /* WF_DRAFT_* bits (0: the paper's drafter); n_draft_layer
                               sets the depth (2 in the paper, 5 in Table A4) */
} wf_config;

typedef struct wf_handle wf_handle;

/* Number of workspace bytes a handle with this config needs. */
int wf_workspace_bytes(const wf_config* cfg, size_t* bytes);

/* Number of parameter tensors wf_init_weights expects, and the element count
 * of tensor i (in the manifest order below). */
int wf_weight_count(const wf_config* cfg, int* n);
int wf_weight_numel(const wf_config* cfg, int i, int64_t* numel);

/*
 * Create a handle over `workspace` (device, ws_bytes >= wf_workspace_bytes,
 * 256-byte aligned) and copy the parameters into it.
 *
 * weights: host array of n_weights device pointers, one per parameter in the
 * manifest order, each holding its tensor in the storage type, row-major,
 * linear weights as [out, in]:
 *   tok_emb [V,d]  pos_emb [n_ctx,d]
 *   per target block l: attn_ln.g/b [d]; attn.q.w [d,d] attn.q.b [d];
 *     attn.k.w [d,d]; attn.v.w [d,d] attn.v.b [d]; attn.o.w [d,d] attn.o.b [d];
 *     xattn_ln.g/b; xattn.q.w/b; xattn.k.w; xattn.v.w/b; xattn.o.w/b;
 *     mlp_ln.g/b; mlp.fc1.w [F,d] mlp.fc1.b [F]; mlp.fc2.w [d,F] mlp.fc2.b [d]
 *   ln_f.g/b
 *   drafter: hproj.w [d, n_tap*d] hproj.b [d] (absent with WF_DRAFT_NO_HISTORY);
 *     mask [d]; then n_draft_layer blocks with the target block layout (without
 *     the xattn_ln / xattn entries with WF_DRAFT_NO_AUDIO); ln_f.g/b
 * The caller's tensors are only read by work enqueued on `stream`; they may be
 * freed once that stream has synchronised.  Slots start empty.
 * Errors: WF_EINVAL (config, null, n_weights), WF_ESIZE, WF_EHIP.
 */
int wf_init_weights(wf_handle** h, const wf_config* cfg, const void* const* weights, int n_weights,
                    void* workspace, size_t ws_bytes, void* stream);

/*
 * Store the acoustic memory of slots [slot0, slot0+n) and compute their
 * cross-attention keys and values for every target and drafter block
 * (K = A W_k^T, V = A W_v^T + b_v; Appendix A.5: each request refreshes the
 * acoustic K/V of target and drafter).
 * mem: device, [n, n_frames, d_model] in the storage type.
 */
int wf_encode_memory_set(wf_handle* h, int slot0, int n, const void* mem, void* stream);

/*
 * Prefill (Appendix A.1): run the target over the prompt of each slot
 * (positions 0..len-1), fill its cache and the drafter history, and emit the
 * first transcript token, which becomes the first anchor (greedy argmax, or a
 * sample when temperature > 0).  emitted = 1.
 * tokens: device int32 [n, pmax] (row s holds len[s] ids); lens, max_new:
 * host int32 [n] with 1 <= len[s] <= min(pmax, n_ctx) and max_new[s] >= 1
 * (max_new counts emitted tokens including the first).
 * first_token: device int32 [n] or NULL.
 */
int wf_prefill(wf_handle* h, int slot0, int n, const int32_t* tokens, int pmax, const int32_t* lens,
               const int32_t* max_new, int32_t* first_token, void* stream);

/*
 * Sampling controls for later calls: temperature 0 selects greedy decoding;
 * T > 0 selects sampling at temperature T with the speculative rejection rule
 * (Section 3.1, Appendix A.4).  Random draws come from Philox4x64-10 keyed by
 * (seed, 0) with counter (purpose << 32 | slot, step, row, vocab >> 2).
 * suppress: device uint8 [n_vocab] (1 = token never produced, applied to
 * draft and target alike) or NULL.  Host-side only; takes effect for
 * subsequently enqueued work.
 */
int wf_set_sampling(wf_handle* h, float temperature, uint64_t seed, const uint8_t* suppress);

/*
 * Draft (Section 3.2): run the drafter for slots [slot0, slot0+n) from each
 * slot's anchor, history and acoustic memory.  The history already holds
 * every position before the anchor (prefill and each verify write it).
 * draft: device int32 [n, block_k] (greedy argmax or Gumbel-max samples).
 * Errors: WF_EINVAL (slot range), WF_ESTATE (a slot not prefilled), WF_EHIP.
 */
int wf_draft(wf_handle* h, int slot0, int n, int32_t* draft, void* stream);

/*
 * Verify and accept (Section 3.1, Appendix A.1): one causal target pass over
 * [anchor, draft[0..k)) at positions L..L+k with
 * k = min(block_k, k_max, max_new - emitted - 1, n_ctx - L - 1), then greedy
 * longest-prefix acceptance (or the rejection rule), then the state update
 * (L += 1 + a, anchor = last emitted token, emitted += a + 1, done on EOS,
 * budget or context end), then the drafter history of the verified rows
 * (Appendix A.2: the target taps of rows L..L+k projected and written at their
 * positions; rows at or beyond the new length are never read and are
 * overwritten later).  Finished slots are left unchanged and report
 * n_out = 0.  k_max in [0, block_k]; k_max = 0 is plain decoding.
 * draft: device int32 [n, block_k]. out: device int32 [n, block_k + 1];
 * n_out, n_acc, done: device int32 [n] (any may be NULL).
 */
int wf_verify_accept(wf_handle* h, int slot0, int n, const int32_t* draft, int k_max, int32_t* out,
                     int32_t* n_out, int32_t* n_acc, int32_t* done, void* stream);

/*
 * One full step: wf_draft followed by wf_verify_accept.  If draft_override
 * (device int32 [n, block_k]) is not NULL the drafter still runs but its
 * proposals are replaced by draft_override (planted drafts for benchmarks).
 * With k_max = 0 no proposal is verified and the drafter does not run (plain
 * decoding: one target pass per token).
 * use_graph != 0 captures the step into a HIP graph on first use (per
 * argument tuple) and replays it afterwards.
 */
int wf_step(wf_handle* h, int slot0, int n, int k_max, const int32_t* draft_override, int32_t* out,
            int32_t* n_out, int32_t* n_acc, int32_t* done, int use_graph, void* stream);

/*
 * wf_step (eager, use_graph = 0) for callers that cannot allocate device memory
 * or use a workspace of their own per call: code under HIP graph capture, tight
 * serving loops, harnesses that forbid allocation.  The per-call buffers of the
 * step (matrix operands, activation rows, partial sums, head partials, logits:
 * everything but the weights, caches and per-slot state of the workspace) live
 * in a static device array of the library, 16 MiB per GPU, held until the
 * process ends; nothing is allocated (no hipMalloc or hipFree, no allocating
 * library routine).  The array is cleared at the start of every call.  All calls
 * on one GPU share that array, so calls that overlap on one GPU (other streams,
 * other handles) race: issue them in order.  Same arguments and results as
 * wf_step; the debug views (wf_debug_ptr) and profiling are not written by it.
 * Errors: as wf_step, plus WF_ESIZE when this configuration's per-call buffers
 * exceed the array (large vocabularies times many slots; batch 1 at
 * Whisper-large-v3 shapes needs about 7 MiB).
 */
int wf_step_noalloc(wf_handle* h, int slot0, int n, int k_max, const int32_t* draft_override, int32_t* out,
                    int32_t* n_out, int32_t* n_acc, int32_t* done, void* stream);

/*
 * Debug views for tests: device pointers into the workspace (valid until
 * wf_release).  which: 0 = target logits of the last verify [max_batch,
 * block_k+1, n_vocab] fp32 (written when wf_set_debug(h, 1) or when
 * sampling), 1 = draft logits of the last draft [max_batch, block_k+1,
 * n_vocab] fp32 (row j >= 1 is mask j; same condition), 2 = per-slot state
 * int32 [max_batch, 16] (0 L, 1 anchor, 2 emitted, 3 max_new, 4 done,
 * 5 step), 3 = last drafted tokens int32 [max_batch, block_k].
 */
int wf_debug_ptr(wf_handle* h, int which, void** ptr);
int wf_set_debug(wf_handle* h, int enable);

/*
 * Profiling: while enabled, every launch of the weight products, attention,
 * LayerNorm and residual-reduction kernels records the wall-clock time at
 * which its first wave starts and its last wave ends (a device timing slot per
 * launch).  "exec_ms" sums those spans; "ms" sums each launch's share of the
 * timeline, from the previous timed launch's last wave end to its own (the
 * dispatch and completion between kernels included).  Eager calls synchronise
 * their stream and collect the durations before returning; wf_step with
 * use_graph captures a separate profiled graph and each replay of it
 * synchronises and collects.  wf_profile_summary writes a JSON object
 * {"<kernel class>": {"launches": n, "ms": total, "exec_ms": total, "bytes":
 * algorithmic bytes}} of everything collected since the previous summary into
 * buf (len bytes, including the terminating NUL), then forgets it (also when
 * buf is too small: WF_ESIZE).  Algorithmic bytes count parameters, caches and
 * activations each launch must move once.  Calls made while profiling is off
 * carry no timing.
 */
int wf_profile_enable(wf_handle* h, int enable);
int wf_profile_summary(wf_handle* h, char* buf, size_t len);

/* Read and clear the sticky device status word (synchronises `stream`). */
int wf_status(wf_handle* h, uint32_t* flags, void* stream);

/* Destroy the handle (does not touch the workspace). */
int wf_release(wf_handle* h);

const char* wf_strerror(int code);

/*
 * Test entry points for the sampling generator (Philox4x64-10, Salmon et al.,
 * SC'11, with the stream layout of wf_set_sampling): words v = 0..n-1 of
 * stream (seed, purpose, slot, step, pos), i.e. word v & 3 of the block with
 * counter (purpose << 32 | slot, step, pos, v >> 2) under key (seed, 0).
 * Purposes: 1 prefill, 2 plain, 3 draft, 4 acceptance, 5 residual, 6 bonus.
 * _host computes them on the CPU into host memory out[n]; _device enqueues a
 * kernel writing device memory out[n] on stream.  Both use the code the
 * sampling kernels use.
 */
int wf_rng_words_host(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out);
int wf_rng_words_device(uint64_t seed, int purpose, int slot, int step, int pos, int n, uint64_t* out, void* stream);
const char* wf_last_error(wf_handle* h);

/*
 * Whisper audio encoder: waveform -> acoustic memory A = E(x), the frozen
 * encoder output both the target and the drafter cross-attend to (Section 3.2;
 * it runs once per request over a 30 s window, Section 1).  The paper names the
 * model only as Whisper large-v3; these are that model's definitions:
 *  - log-mel frontend: 16 kHz samples, periodic Hann window of n_fft, hop
 *    samples apart, signal reflect-padded by n_fft / 2, |STFT|^2 with the last
 *    frame dropped (2 n_ctx frames), triangular filters on the Slaney mel scale
 *    normalised to unit area, log10 of max(mel, 1e-10), raised to at least
 *    (maximum - 8), then (x + 4) / 4;
 *  - stem: conv(n_mels -> d, kernel 3, padding 1) + GELU, conv(d -> d, kernel 3,
 *    stride 2, padding 1) + GELU, plus the sinusoid position table;
 *  - n_layer pre-LN blocks: bidirectional self-attention (no key bias, scores
 *    scaled by 1/8), GELU MLP; then the final LayerNorm.
 * Storage bf16 (weights, products' inputs); the residual stream, LayerNorm,
 * softmax, GELU and accumulation are fp32; the frontend is fp64.
 * Large-v3: n_mels 128, n_ctx 1500, d_model 1280, n_head 20, n_layer 32,
 * d_ff 5120, n_fft 400, hop 160, sample_rate 16000.
 */
typedef struct wf_encoder_config {
  int32_t n_mels;
  int32_t n_ctx;       /* output positions; the waveform holds 2 * n_ctx * hop samples */
  int32_t d_model;     /* 64 * n_head, <= 2048 */
  int32_t n_head;
  int32_t n_layer;
  int32_t d_ff;        /* multiple of 64 */
  int32_t n_fft;       /* even, <= 512 */
  int32_t hop;
  int32_t sample_rate;
} wf_encoder_config;

typedef struct wf_encoder wf_encoder;

/* Workspace bytes of an encoder handle (one request's activations). */
int wf_encoder_workspace_bytes(const wf_encoder_config* cfg, size_t* bytes);
/* Number of parameter tensors and the element count of tensor i, in manifest
 * order: conv1.w [d, n_mels, 3] conv1.b [d] conv2.w [d, d, 3] conv2.b [d]; per
 * block: attn_ln.g/b [d]; attn.q.w [d,d] attn.q.b; attn.k.w; attn.v.w attn.v.b;
 * attn.o.w attn.o.b; mlp_ln.g/b; mlp.fc1.w [d_ff,d] mlp.fc1.b; mlp.fc2.w [d,d_ff]
 * mlp.fc2.b; then ln_post.g/b. */
int wf_encoder_weight_count(const wf_encoder_config* cfg, int* n);
int wf_encoder_weight_numel(const wf_encoder_config* cfg, int i, int64_t* numel);
/* Create an encoder over `workspace` (device, 256-byte aligned, >= the bytes
 * above) and copy the bf16 parameters (device pointers in manifest order) into
 * it; the caller's tensors may be freed once `stream` has synchronised.
 * Errors: WF_EINVAL, WF_ESIZE, WF_EHIP. */
int wf_encoder_init(wf_encoder** e, const wf_encoder_config* cfg, const void* const* weights, int n_weights,
                    void* workspace, size_t ws_bytes, void* stream);
/* Encode n waveforms: audio device fp32 [n, 2 * n_ctx * hop]; mem device bf16
 * [n, n_ctx, d_model] (16-byte aligned), ready for wf_encode_memory_set.
 * Requests run one after another on `stream`. */
int wf_encoder_run(wf_encoder* e, int n, const float* audio, void* mem, void* stream);
/* The frontend alone: scaled log-mel features of one waveform into mel, device
 * fp32 [n_mels, 2 * n_ctx]. */
int wf_encoder_logmel(wf_encoder* e, const float* audio, float* mel, void* stream);
int wf_encoder_release(wf_encoder* e);
const char* wf_encoder_last_error(wf_encoder* e);

#ifdef __cplusplus
}
#endif

#endif /* WF_H */
