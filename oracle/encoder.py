"""Whisper audio encoder and its log-mel frontend (test infrastructure only).

The paper's drafter reads the acoustic memory A = E(x), the output of the
frozen Whisper encoder (Section 3.2); the encoder runs once per request over a
30 s window (Section 1; Appendix B.2, Table A2 measures its share of request
time).  The architecture is Whisper's (large-v3 shapes: 128 mel bins, 32 blocks
of width 1280 with 20 heads, 1500 positions); the paper describes it only as
Whisper, so every definition below is that model's, written out plainly:

  log-mel   16 kHz waveform, periodic Hann window of 400 samples, hop 160, the
            signal reflect-padded by 200 on both sides, |STFT|^2 (the last frame
            dropped, 3000 frames for 30 s), Slaney-style mel filterbank with
            Slaney area normalisation, log10 of max(mel, 1e-10), values below
            (maximum - 8) raised to it, then (x + 4) / 4;
  stem      conv1d(n_mels -> d, kernel 3, padding 1) + GELU, conv1d(d -> d,
            kernel 3, stride 2, padding 1) + GELU, plus the sinusoidal position
            table;
  blocks    pre-LN bidirectional self-attention (biases on q, v, o, none on k;
            scores scaled by 1/8), pre-LN GELU MLP, each added to the residual;
  output    final LayerNorm (ln_post).

Precision: fp32 arithmetic; with ``opts.gemm_bf16`` every product input is
rounded to bf16 (the GPU's matrix-core operands): the convolution inputs, the
LayerNorm outputs, q, k, v, the attention probabilities and the attention and
MLP hidden activations.
"""
import numpy as np

from .numerics import layer_norm, gelu, linear, softmax, bf16


# ---------------------------------------------------------------- frontend

def hann_periodic(n):
    """w[i] = 0.5 - 0.5 cos(2 pi i / n), i = 0..n-1 (the periodic Hann window)."""
    i = np.arange(n, dtype=np.float64)
    return 0.5 - 0.5 * np.cos(2.0 * np.pi * i / n)


def stft_power(audio, n_fft=400, hop=160):
    """|STFT|^2 [frames, n_fft/2 + 1] of a 1-D signal (reflect padding n_fft/2,
    periodic Hann window); the last frame is dropped, as Whisper does."""
    x = np.asarray(audio, np.float64)
    pad = n_fft // 2
    xp = np.pad(x, (pad, pad), mode="reflect")
    n_frames = 1 + (len(xp) - n_fft) // hop
    idx = hop * np.arange(n_frames)[:, None] + np.arange(n_fft)[None, :]
    spec = np.fft.rfft(xp[idx] * hann_periodic(n_fft)[None, :], axis=1)
    return (np.abs(spec) ** 2)[:-1]


# Slaney's mel scale: linear below 1 kHz (200/3 Hz per mel), logarithmic above
# (a factor 6.4 per 27 mels).
_F_SP = 200.0 / 3.0
_MIN_LOG_HZ = 1000.0
_MIN_LOG_MEL = _MIN_LOG_HZ / _F_SP
_LOGSTEP = np.log(6.4) / 27.0


def hz_to_mel(f):
    f = np.asarray(f, np.float64)
    lin = f / _F_SP
    return np.where(f >= _MIN_LOG_HZ, _MIN_LOG_MEL + np.log(np.maximum(f, 1e-300) / _MIN_LOG_HZ) / _LOGSTEP, lin)


def mel_to_hz(m):
    m = np.asarray(m, np.float64)
    return np.where(m >= _MIN_LOG_MEL, _MIN_LOG_HZ * np.exp(_LOGSTEP * (m - _MIN_LOG_MEL)), _F_SP * m)


def mel_filters(sr=16000, n_fft=400, n_mels=128):
    """[n_mels, n_fft/2 + 1] triangular filters, their corners at n_mels + 2 points
    equally spaced on the Slaney mel scale from 0 Hz to sr/2, each scaled to unit
    area in Hz (2 / (upper corner - lower corner))."""
    fft_hz = np.linspace(0.0, sr / 2.0, n_fft // 2 + 1)
    corners = mel_to_hz(np.linspace(hz_to_mel(0.0), hz_to_mel(sr / 2.0), n_mels + 2))
    w = np.zeros((n_mels, len(fft_hz)))
    for i in range(n_mels):
        lo, c, hi = corners[i], corners[i + 1], corners[i + 2]
        rise = (fft_hz - lo) / (c - lo)
        fall = (hi - fft_hz) / (hi - c)
        w[i] = np.maximum(0.0, np.minimum(rise, fall)) * (2.0 / (hi - lo))
    return w


def log_mel(audio, n_mels=128, n_fft=400, hop=160, sr=16000):
    """Whisper's log-mel features [n_mels, frames] of one waveform, fp32."""
    power = stft_power(audio, n_fft, hop)                     # [frames, bins]
    mel = mel_filters(sr, n_fft, n_mels) @ power.T            # [n_mels, frames]
    lg = np.log10(np.maximum(mel, 1e-10))
    lg = np.maximum(lg, lg.max() - 8.0)
    return ((lg + 4.0) / 4.0).astype(np.float32)


def sinusoids(length, channels, max_timescale=10000.0):
    """Position table [length, channels]: sin in the first half, cos in the second,
    timescales geometric from 1 to max_timescale."""
    inc = np.log(max_timescale) / (channels // 2 - 1)
    inv = np.exp(-inc * np.arange(channels // 2))
    t = np.arange(length)[:, None] * inv[None, :]
    return np.concatenate([np.sin(t), np.cos(t)], axis=1)


# ---------------------------------------------------------------- encoder

def conv1d(x, w, b, stride, opts):
    """x [T, C_in], w [C_out, C_in, 3], padding 1: y[t] = sum_j w[:, :, j] x[stride t + j - 1] + b."""
    T, cin = x.shape
    xp = np.concatenate([np.zeros((1, cin), x.dtype), x, np.zeros((1, cin), x.dtype)])
    n_out = (T + 2 - 3) // stride + 1
    cols = np.stack([xp[stride * np.arange(n_out) + j] for j in range(3)], axis=2)  # [n_out, C_in, 3]
    return linear(cols.reshape(n_out, cin * 3), w.reshape(w.shape[0], -1), b, opts)


def _blk(W, prefix):
    return {k.split(".", 1)[1]: v for k, v in W.items() if k.startswith(prefix + ".")}


class Encoder:
    def __init__(self, ecfg, W, opts):
        self.cfg, self.opts = ecfg, opts
        self.W = W
        self.blocks = [_blk(W, f"e{l}") for l in range(ecfg.n_layer)]

    def _r(self, x):
        return bf16(x) if self.opts.gemm_bf16 else x

    def attend(self, b, a):
        """Bidirectional multi-head self-attention of rows a [T, d] (pre-LN applied)."""
        opts, dt, H = self.opts, self.opts.dtype, self.cfg.n_head
        T, d = a.shape
        hd = d // H
        q = self._r(linear(a, b["attn.q.w"], b["attn.q.b"], opts)).reshape(T, H, hd)
        k = self._r(linear(a, b["attn.k.w"], None, opts)).reshape(T, H, hd)
        v = self._r(linear(a, b["attn.v.w"], b["attn.v.b"], opts)).reshape(T, H, hd)
        o = np.zeros((T, H, hd), dt)
        for h in range(H):
            s = (q[:, h, :].astype(dt) @ k[:, h, :].astype(dt).T) * dt(1.0 / np.sqrt(hd))
            p = self._r(softmax(s, axis=-1).astype(dt))
            o[:, h, :] = p @ v[:, h, :].astype(dt)
        return linear(o.reshape(T, d), b["attn.o.w"], b["attn.o.b"], opts)

    def forward(self, mel):
        """Acoustic memory [n_ctx, d] from log-mel features [n_mels, 2 n_ctx]."""
        cfg, opts, dt, W = self.cfg, self.opts, self.opts.dtype, self.W
        x = mel.T.astype(dt)
        x = gelu(conv1d(x, W["conv1.w"], W["conv1.b"], 1, opts))
        x = gelu(conv1d(x, W["conv2.w"], W["conv2.b"], 2, opts))
        x = (x + sinusoids(x.shape[0], cfg.d_model)).astype(dt)
        for b in self.blocks:
            x = x + self.attend(b, layer_norm(x, b["attn_ln.g"], b["attn_ln.b"], dt))
            m = layer_norm(x, b["mlp_ln.g"], b["mlp_ln.b"], dt)
            x = x + linear(gelu(linear(m, b["mlp.fc1.w"], b["mlp.fc1.b"], opts)), b["mlp.fc2.w"], b["mlp.fc2.b"], opts)
        return layer_norm(x, W["ln_post.g"], W["ln_post.b"], dt)

    def encode(self, audio):
        return self.forward(log_mel(audio, self.cfg.n_mels))
