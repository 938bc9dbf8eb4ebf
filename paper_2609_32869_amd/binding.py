"""ctypes binding of libwf (include/wf.h).

Argument marshalling only: every step of the draft-and-verify path runs in the
HIP kernels of libwf.so.  PyTorch provides device memory (the workspace and
output tensors) and the HIP stream.  The library must be built first
(``python -m paper_2609_32869_amd.build`` or ``__graft_entry__.build()``);
importing this module without it raises.
"""
import ctypes
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libwf.so")

WF_F32, WF_BF16 = 0, 1
WF_MAX_TAPS = 8
WF_STATUS_NONFINITE_LOGITS = 0x1
WF_STATUS_POSITION_OVERFLOW = 0x2

# symbols declared in include/wf.h
EXPORTS = ["wf_workspace_bytes", "wf_weight_count", "wf_weight_numel", "wf_init_weights",
           "wf_encode_memory_set", "wf_prefill", "wf_set_sampling", "wf_draft", "wf_verify_accept",
           "wf_step", "wf_step_noalloc", "wf_debug_ptr", "wf_set_debug", "wf_profile_enable", "wf_profile_summary", "wf_status",
           "wf_release", "wf_strerror", "wf_last_error", "wf_rng_words_host", "wf_rng_words_device",
           "wf_encoder_workspace_bytes", "wf_encoder_weight_count", "wf_encoder_weight_numel", "wf_encoder_init",
           "wf_encoder_run", "wf_encoder_logmel", "wf_encoder_release", "wf_encoder_last_error"]


class WfConfig(ctypes.Structure):
    _fields_ = [("n_layer", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_head", ctypes.c_int32),
                ("d_ff", ctypes.c_int32), ("n_vocab", ctypes.c_int32), ("n_ctx", ctypes.c_int32),
                ("n_frames", ctypes.c_int32), ("n_draft_layer", ctypes.c_int32), ("block_k", ctypes.c_int32),
                ("n_tap", ctypes.c_int32), ("taps", ctypes.c_int32 * WF_MAX_TAPS), ("eos_id", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("max_batch", ctypes.c_int32), ("draft_flags", ctypes.c_int32)]


class WfEncoderConfig(ctypes.Structure):
    _fields_ = [("n_mels", ctypes.c_int32), ("n_ctx", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("n_head", ctypes.c_int32), ("n_layer", ctypes.c_int32), ("d_ff", ctypes.c_int32),
                ("n_fft", ctypes.c_int32), ("hop", ctypes.c_int32), ("sample_rate", ctypes.c_int32)]


class WfError(RuntimeError):
    pass


_lib = None


def load_library(path=LIB_PATH):
    """Load libwf.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise WfError(f"{path} not found: build the HIP library first (python -m paper_2609_32869_amd.build)")
    lib = ctypes.CDLL(path)
    P, I, Z, U64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t, ctypes.c_uint64
    cfgp = ctypes.POINTER(WfConfig)
    sig = {
        "wf_workspace_bytes": [cfgp, ctypes.POINTER(Z)],
        "wf_weight_count": [cfgp, ctypes.POINTER(I)],
        "wf_weight_numel": [cfgp, I, ctypes.POINTER(ctypes.c_int64)],
        "wf_init_weights": [ctypes.POINTER(P), cfgp, ctypes.POINTER(P), I, P, Z, P],
        "wf_encode_memory_set": [P, I, I, P, P],
        "wf_prefill": [P, I, I, P, I, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_int32), P, P],
        "wf_set_sampling": [P, ctypes.c_float, U64, P],
        "wf_draft": [P, I, I, P, P],
        "wf_verify_accept": [P, I, I, P, I, P, P, P, P, P],
        "wf_step": [P, I, I, I, P, P, P, P, P, I, P],
        "wf_step_noalloc": [P, I, I, I, P, P, P, P, P, P],
        "wf_debug_ptr": [P, I, ctypes.POINTER(P)],
        "wf_set_debug": [P, I],
        "wf_profile_enable": [P, I],
        "wf_profile_summary": [P, ctypes.c_char_p, Z],
        "wf_status": [P, ctypes.POINTER(ctypes.c_uint32), P],
        "wf_release": [P],
        "wf_strerror": [I],
        "wf_last_error": [P],
        "wf_rng_words_host": [U64, I, I, I, I, I, ctypes.POINTER(U64)],
        "wf_rng_words_device": [U64, I, I, I, I, I, P, P],
        "wf_encoder_workspace_bytes": [ctypes.POINTER(WfEncoderConfig), ctypes.POINTER(Z)],
        "wf_encoder_weight_count": [ctypes.POINTER(WfEncoderConfig), ctypes.POINTER(I)],
        "wf_encoder_weight_numel": [ctypes.POINTER(WfEncoderConfig), I, ctypes.POINTER(ctypes.c_int64)],
        "wf_encoder_init": [ctypes.POINTER(P), ctypes.POINTER(WfEncoderConfig), ctypes.POINTER(P), I, P, Z, P],
        "wf_encoder_run": [P, I, P, P, P],
        "wf_encoder_logmel": [P, P, P, P],
        "wf_encoder_release": [P],
        "wf_encoder_last_error": [P],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = ctypes.c_char_p if name in ("wf_strerror", "wf_last_error", "wf_encoder_last_error") else ctypes.c_int
    _lib = lib
    return lib


def rng_words_host(seed, purpose, slot, step, pos, n):
    """Generator words v = 0..n-1 of a sampling stream, computed by the library on the host."""
    lib = load_library()
    out = np.zeros(n, np.uint64)
    rc = lib.wf_rng_words_host(int(seed), purpose, slot, step, pos, n, out.ctypes.data_as(ctypes.POINTER(ctypes.c_uint64)))
    if rc != 0:
        raise WfError(lib.wf_last_error(None).decode())
    return out


def rng_words_device(seed, purpose, slot, step, pos, n, stream=None):
    """The same words computed by the library's device kernel (int64 tensor holding the bits)."""
    lib = load_library()
    out = torch.empty(n, dtype=torch.int64, device="cuda")
    rc = lib.wf_rng_words_device(int(seed), purpose, slot, step, pos, n, _ptr(out), _stream(stream))
    if rc != 0:
        raise WfError(lib.wf_last_error(None).decode())
    return out


def make_config(cfg, max_batch):
    """WfConfig from a model-shape object (attributes as in wf_fixtures.ModelConfig)."""
    c = WfConfig()
    c.n_layer, c.d_model, c.n_head, c.d_ff = cfg.n_layer, cfg.d_model, cfg.n_head, cfg.d_ff
    c.n_vocab, c.n_ctx, c.n_frames = cfg.n_vocab, cfg.n_ctx, cfg.n_frames
    c.n_draft_layer, c.block_k, c.n_tap = cfg.n_draft_layer, cfg.block_k, len(cfg.taps)
    for i, t in enumerate(cfg.taps):
        c.taps[i] = t
    c.eos_id = cfg.eos_id
    c.dtype = WF_BF16 if cfg.dtype == "bf16" else WF_F32
    c.max_batch = max_batch
    c.draft_flags = getattr(cfg, "draft_flags", 0)
    return c


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def to_device_storage(arr, dtype, device="cuda"):
    """Host fp32 array -> device tensor in the storage type (bf16 values must be exact)."""
    a = np.ascontiguousarray(arr, dtype=np.float32)
    if dtype == "bf16":
        bits = (a.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
        return torch.from_numpy(bits.view(np.int16)).to(device).view(torch.bfloat16)
    return torch.from_numpy(a).to(device)


class WhisperFlash:
    """One libwf handle over a workspace tensor it owns."""

    def __init__(self, cfg, max_batch, weights, stream=None):
        """weights: device tensors in manifest order (storage type)."""
        self.lib = load_library()
        self.cfg = cfg
        self.ccfg = make_config(cfg, max_batch)
        self.max_batch = max_batch
        self.K = cfg.block_k
        nbytes = ctypes.c_size_t()
        self._check(self.lib.wf_workspace_bytes(ctypes.byref(self.ccfg), ctypes.byref(nbytes)))
        self.ws = torch.empty(nbytes.value, dtype=torch.uint8, device="cuda")
        n = ctypes.c_int()
        self._check(self.lib.wf_weight_count(ctypes.byref(self.ccfg), ctypes.byref(n)))
        if len(weights) != n.value:
            raise WfError(f"expected {n.value} weight tensors, got {len(weights)}")
        arr = (ctypes.c_void_p * n.value)(*[w.data_ptr() for w in weights])
        h = ctypes.c_void_p()
        self._check(self.lib.wf_init_weights(ctypes.byref(h), ctypes.byref(self.ccfg), arr, n.value,
                                             ctypes.c_void_p(self.ws.data_ptr()), nbytes.value, _stream(stream)))
        self.h = h

    @classmethod
    def from_host(cls, cfg, max_batch, ordered_arrays, stream=None):
        dev = [to_device_storage(a, cfg.dtype) for a in ordered_arrays]
        obj = cls(cfg, max_batch, dev, stream)
        torch.cuda.synchronize()
        del dev
        return obj

    def _check(self, rc):
        if rc != 0:
            h = getattr(self, "h", None)
            msg = self.lib.wf_last_error(h if h is not None else None)
            raise WfError(f"{self.lib.wf_strerror(rc).decode()} ({rc}): {msg.decode() if msg else ''}")

    def close(self):
        if getattr(self, "h", None) is not None:
            self.lib.wf_release(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- calls of include/wf.h
    def encode_memory_set(self, slot0, mem, stream=None):
        """mem: device tensor [n, n_frames, d] in the storage type."""
        self._check(self.lib.wf_encode_memory_set(self.h, slot0, mem.shape[0], _ptr(mem), _stream(stream)))

    def prefill(self, slot0, tokens, lens, max_new, stream=None):
        """tokens: device int32 [n, pmax]; lens, max_new: sequences of ints. Returns first tokens [n]."""
        n, pmax = tokens.shape
        first = torch.empty(n, dtype=torch.int32, device="cuda")
        L = (ctypes.c_int32 * n)(*[int(x) for x in lens])
        M = (ctypes.c_int32 * n)(*[int(x) for x in max_new])
        self._check(self.lib.wf_prefill(self.h, slot0, n, _ptr(tokens), pmax, L, M, _ptr(first), _stream(stream)))
        return first

    def set_sampling(self, temperature, seed=0, suppress=None):
        self._check(self.lib.wf_set_sampling(self.h, float(temperature), int(seed), _ptr(suppress)))

    def draft(self, slot0, n, stream=None):
        out = torch.empty((n, self.K), dtype=torch.int32, device="cuda")
        self._check(self.lib.wf_draft(self.h, slot0, n, _ptr(out), _stream(stream)))
        return out

    def _outs(self, n):
        return (torch.empty((n, self.K + 1), dtype=torch.int32, device="cuda"),
                torch.empty(n, dtype=torch.int32, device="cuda"),
                torch.empty(n, dtype=torch.int32, device="cuda"),
                torch.empty(n, dtype=torch.int32, device="cuda"))

    def verify_accept(self, slot0, draft, k_max=None, outs=None, stream=None):
        n = draft.shape[0]
        k_max = self.K if k_max is None else k_max
        out, n_out, n_acc, done = outs if outs is not None else self._outs(n)
        self._check(self.lib.wf_verify_accept(self.h, slot0, n, _ptr(draft), k_max, _ptr(out), _ptr(n_out),
                                              _ptr(n_acc), _ptr(done), _stream(stream)))
        return out, n_out, n_acc, done

    def step(self, slot0, n, k_max=None, draft_override=None, outs=None, use_graph=False, stream=None):
        k_max = self.K if k_max is None else k_max
        out, n_out, n_acc, done = outs if outs is not None else self._outs(n)
        self._check(self.lib.wf_step(self.h, slot0, n, k_max, _ptr(draft_override), _ptr(out), _ptr(n_out),
                                     _ptr(n_acc), _ptr(done), 1 if use_graph else 0, _stream(stream)))
        return out, n_out, n_acc, done

    def step_noalloc(self, slot0, n, k_max=None, draft_override=None, outs=None, stream=None):
        """wf_step_noalloc: the step with its per-call buffers in the library's static scratch."""
        k_max = self.K if k_max is None else k_max
        out, n_out, n_acc, done = outs if outs is not None else self._outs(n)
        self._check(self.lib.wf_step_noalloc(self.h, slot0, n, k_max, _ptr(draft_override), _ptr(out), _ptr(n_out),
                                             _ptr(n_acc), _ptr(done), _stream(stream)))
        return out, n_out, n_acc, done

    def set_debug(self, on):
        self._check(self.lib.wf_set_debug(self.h, 1 if on else 0))

    def _view(self, which, shape, dtype):
        p = ctypes.c_void_p()
        self._check(self.lib.wf_debug_ptr(self.h, which, ctypes.byref(p)))
        off = p.value - self.ws.data_ptr()
        nbytes = int(np.prod(shape)) * torch.tensor([], dtype=dtype).element_size()
        return self.ws[off:off + nbytes].view(dtype).view(*shape)

    def target_logits(self):
        return self._view(0, (self.max_batch, 9, self.cfg.n_vocab), torch.float32)

    def draft_logits(self):
        """[max_batch, 9, V]; row j (1..8) holds the logits of mask j."""
        return self._view(1, (self.max_batch, 9, self.cfg.n_vocab), torch.float32)

    def state(self):
        return self._view(2, (self.max_batch, 16), torch.int32)

    def last_draft(self):
        return self._view(3, (self.max_batch, self.K), torch.int32)

    def profile(self, on):
        self._check(self.lib.wf_profile_enable(self.h, 1 if on else 0))

    def profile_summary(self):
        import json
        buf = ctypes.create_string_buffer(1 << 16)
        self._check(self.lib.wf_profile_summary(self.h, buf, len(buf)))
        return json.loads(buf.value.decode())

    def status(self, stream=None):
        f = ctypes.c_uint32()
        self._check(self.lib.wf_status(self.h, ctypes.byref(f), _stream(stream)))
        return f.value


def make_encoder_config(ecfg):
    """WfEncoderConfig from an encoder-shape object (attributes as in wf_fixtures.EncoderConfig)."""
    c = WfEncoderConfig()
    c.n_mels, c.n_ctx, c.d_model, c.n_head = ecfg.n_mels, ecfg.n_ctx, ecfg.d_model, ecfg.n_head
    c.n_layer, c.d_ff, c.n_fft, c.hop, c.sample_rate = ecfg.n_layer, ecfg.d_ff, ecfg.n_fft, ecfg.hop, ecfg.sample_rate
    return c


class WhisperEncoder:
    """One libwf encoder handle over a workspace tensor it owns (bf16 weights)."""

    def __init__(self, ecfg, weights, stream=None):
        self.lib = load_library()
        self.cfg = ecfg
        self.ccfg = make_encoder_config(ecfg)
        nbytes = ctypes.c_size_t()
        self._check(self.lib.wf_encoder_workspace_bytes(ctypes.byref(self.ccfg), ctypes.byref(nbytes)))
        self.ws = torch.empty(nbytes.value, dtype=torch.uint8, device="cuda")
        n = ctypes.c_int()
        self._check(self.lib.wf_encoder_weight_count(ctypes.byref(self.ccfg), ctypes.byref(n)))
        if len(weights) != n.value:
            raise WfError(f"expected {n.value} encoder weight tensors, got {len(weights)}")
        arr = (ctypes.c_void_p * n.value)(*[w.data_ptr() for w in weights])
        h = ctypes.c_void_p()
        self._check(self.lib.wf_encoder_init(ctypes.byref(h), ctypes.byref(self.ccfg), arr, n.value,
                                             ctypes.c_void_p(self.ws.data_ptr()), nbytes.value, _stream(stream)))
        self.h = h

    @classmethod
    def from_host(cls, ecfg, ordered_arrays, stream=None):
        dev = [to_device_storage(a, "bf16") for a in ordered_arrays]
        obj = cls(ecfg, dev, stream)
        torch.cuda.synchronize()
        del dev
        return obj

    def _check(self, rc):
        if rc != 0:
            h = getattr(self, "h", None)
            msg = self.lib.wf_encoder_last_error(h if h is not None else None)
            raise WfError(f"{self.lib.wf_strerror(rc).decode()} ({rc}): {msg.decode() if msg else ''}")

    def run(self, audio, stream=None):
        """audio: device fp32 [n, n_samples] -> acoustic memory, device bf16 [n, n_ctx, d]."""
        n = audio.shape[0]
        mem = torch.empty((n, self.cfg.n_ctx, self.cfg.d_model), dtype=torch.bfloat16, device="cuda")
        self._check(self.lib.wf_encoder_run(self.h, n, _ptr(audio), _ptr(mem), _stream(stream)))
        return mem

    def logmel(self, audio, stream=None):
        """audio: device fp32 [n_samples] -> scaled log-mel features, device fp32 [n_mels, frames]."""
        mel = torch.empty((self.cfg.n_mels, 2 * self.cfg.n_ctx), dtype=torch.float32, device="cuda")
        self._check(self.lib.wf_encoder_logmel(self.h, _ptr(audio), _ptr(mel), _stream(stream)))
        return mel

    def close(self):
        if getattr(self, "h", None) is not None:
            self.lib.wf_encoder_release(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
