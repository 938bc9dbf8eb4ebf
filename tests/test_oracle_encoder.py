"""Pins of the oracle's Whisper encoder and log-mel frontend (CPU only).

Library special cases: the periodic Hann window against scipy's, the power
spectrum against torch.stft, the convolutions against torch's conv1d, and the
encoder blocks (pre-LN, exact GELU, no key bias) against torch's
TransformerEncoderLayer, all in fp64.  Closed forms: the Slaney mel scale's
fixed points, the filters' triangle corners and unit areas, a pure tone's
spectral peak and mel bin, the sinusoid table's values, the log-mel clamp.
"""
import numpy as np
import pytest
import scipy.signal
import torch

from wf_fixtures import MICRO_ENC, LARGE_V3_ENC, make_encoder_weights, make_audio, encoder_manifest, param_count
from oracle import OracleOpts
from oracle.encoder import (hann_periodic, stft_power, hz_to_mel, mel_to_hz, mel_filters, log_mel, sinusoids,
                            conv1d, Encoder)

F64 = OracleOpts(dtype=np.float64)


def test_hann_window_is_the_periodic_one():
    for n in (8, 400):
        np.testing.assert_allclose(hann_periodic(n), scipy.signal.get_window("hann", n, fftbins=True), atol=1e-15)


def test_power_spectrum_matches_torch_stft():
    x = make_audio(MICRO_ENC, 0).astype(np.float64)
    ref = torch.stft(torch.from_numpy(x), 400, 160, window=torch.hann_window(400, dtype=torch.float64),
                     center=True, pad_mode="reflect", return_complex=True).abs() ** 2
    got = stft_power(x)
    assert got.shape == (2 * MICRO_ENC.n_ctx, 201)
    np.testing.assert_allclose(got, ref.numpy()[:, :-1].T, rtol=1e-9, atol=1e-12)


def test_pure_tone_peak():
    """A sinusoid centred on FFT bin k: its power sits in bin k at (A N / 4)^2."""
    n, k, A = 400, 25, 0.3
    t = np.arange(16000)
    x = A * np.cos(2 * np.pi * k * t / n)
    p = stft_power(x)
    mid = p[len(p) // 2]
    assert int(np.argmax(mid)) == k
    np.testing.assert_allclose(mid[k], (A * n / 4) ** 2, rtol=1e-9)


def test_slaney_mel_scale():
    assert hz_to_mel(1000.0) == pytest.approx(15.0)
    assert hz_to_mel(500.0) == pytest.approx(7.5)           # linear part: 200/3 Hz per mel
    assert hz_to_mel(6400.0) == pytest.approx(15.0 + 27.0)  # a factor 6.4 per 27 mels
    f = np.array([0.0, 100.0, 999.0, 1000.0, 4000.0, 8000.0])
    np.testing.assert_allclose(mel_to_hz(hz_to_mel(f)), f, rtol=1e-12, atol=1e-9)


def test_mel_filters_are_unit_area_triangles():
    sr, n_fft = 16000, 400
    for n_mels in (80, 128):
        w = mel_filters(sr, n_fft, n_mels)
        assert w.shape == (n_mels, 201) and (w >= 0).all()
        corners = mel_to_hz(np.linspace(0.0, hz_to_mel(sr / 2), n_mels + 2))
        hz = np.linspace(0, sr / 2, 201)
        df = hz[1]
        for i in range(n_mels):
            lo, c, hi = corners[i], corners[i + 1], corners[i + 2]
            assert (w[i][(hz <= lo) | (hz >= hi)] == 0).all()
            # a bin exactly at the centre carries the peak 2 / (hi - lo)
            on = np.isclose(hz, c)
            if on.any():
                assert w[i][on][0] == pytest.approx(2.0 / (hi - lo))
            if hi - lo > 8 * df:  # wide filters: the bin sum approximates the unit area
                assert w[i].sum() * df == pytest.approx(1.0, rel=0.02)


def test_log_mel_clamp_and_scale():
    x = make_audio(MICRO_ENC, 1)
    m = log_mel(x, MICRO_ENC.n_mels)
    assert m.shape == (MICRO_ENC.n_mels, 2 * MICRO_ENC.n_ctx) and m.dtype == np.float32
    assert m.min() >= m.max() - 2.0 - 1e-6   # 8 decades below the maximum, divided by 4
    # a tone's energy lands in the filter around its frequency
    f = 2000.0
    t = np.arange(MICRO_ENC.n_samples) / 16000
    m = log_mel(0.2 * np.sin(2 * np.pi * f * t), 80)
    centres = mel_to_hz(np.linspace(0.0, hz_to_mel(8000.0), 82))[1:-1]
    band = int(np.argmax(m[:, m.shape[1] // 2]))
    assert abs(band - int(np.argmin(np.abs(centres - f)))) <= 1


def test_sinusoid_table():
    s = sinusoids(1500, 1280)
    assert s.shape == (1500, 1280)
    np.testing.assert_allclose(s[0], np.r_[np.zeros(640), np.ones(640)])
    np.testing.assert_allclose(s[:, 0], np.sin(np.arange(1500)))            # timescale 1
    np.testing.assert_allclose(s[:, 639], np.sin(np.arange(1500) / 1e4))    # timescale 10000
    np.testing.assert_allclose(s[:, :640] ** 2 + s[:, 640:] ** 2, 1.0, atol=1e-12)


def test_conv_stem_matches_torch_conv1d():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((20, 6))
    w = rng.standard_normal((5, 6, 3))
    b = rng.standard_normal(5)
    for stride in (1, 2):
        ref = torch.nn.functional.conv1d(torch.from_numpy(x.T[None]), torch.from_numpy(w), torch.from_numpy(b),
                                         stride=stride, padding=1)[0].numpy().T
        np.testing.assert_allclose(conv1d(x, w, b, stride, F64), ref, atol=1e-12)


def _torch_encoder(W, ecfg):
    d, H, F = ecfg.d_model, ecfg.n_head, ecfg.d_ff
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    layers = []
    for l in range(ecfg.n_layer):
        layer = torch.nn.TransformerEncoderLayer(d, H, F, dropout=0.0, activation="gelu", layer_norm_eps=1e-5,
                                                 batch_first=True, norm_first=True, dtype=torch.float64)
        p = f"e{l}."
        with torch.no_grad():
            layer.self_attn.in_proj_weight.copy_(t(np.concatenate([W[p + "attn.q.w"], W[p + "attn.k.w"], W[p + "attn.v.w"]])))
            layer.self_attn.in_proj_bias.copy_(t(np.concatenate([W[p + "attn.q.b"], np.zeros(d), W[p + "attn.v.b"]])))
            layer.self_attn.out_proj.weight.copy_(t(W[p + "attn.o.w"]))
            layer.self_attn.out_proj.bias.copy_(t(W[p + "attn.o.b"]))
            layer.linear1.weight.copy_(t(W[p + "mlp.fc1.w"]))
            layer.linear1.bias.copy_(t(W[p + "mlp.fc1.b"]))
            layer.linear2.weight.copy_(t(W[p + "mlp.fc2.w"]))
            layer.linear2.bias.copy_(t(W[p + "mlp.fc2.b"]))
            layer.norm1.weight.copy_(t(W[p + "attn_ln.g"]))
            layer.norm1.bias.copy_(t(W[p + "attn_ln.b"]))
            layer.norm2.weight.copy_(t(W[p + "mlp_ln.g"]))
            layer.norm2.bias.copy_(t(W[p + "mlp_ln.b"]))
        layers.append(layer.eval())
    return layers


def test_encoder_matches_torch_layers():
    """The whole encoder in fp64: torch's conv1d + GELU stem, the sinusoid table,
    chained TransformerEncoderLayer(norm_first, gelu) with a zero key bias, and
    the final LayerNorm."""
    ecfg = MICRO_ENC
    W = {k: np.asarray(v, np.float64) for k, v in make_encoder_weights(ecfg).values.items()}
    mel = log_mel(make_audio(ecfg, 0), ecfg.n_mels).astype(np.float64)
    got = Encoder(ecfg, W, F64).forward(mel)
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    g = torch.nn.functional.gelu
    with torch.no_grad():
        x = g(torch.nn.functional.conv1d(t(mel)[None], t(W["conv1.w"]), t(W["conv1.b"]), padding=1))
        x = g(torch.nn.functional.conv1d(x, t(W["conv2.w"]), t(W["conv2.b"]), stride=2, padding=1))
        x = x[0].T + t(sinusoids(ecfg.n_ctx, ecfg.d_model))
        for layer in _torch_encoder(W, ecfg):
            x = layer(x[None])[0]
        x = torch.nn.functional.layer_norm(x, (ecfg.d_model,), t(W["ln_post.g"]), t(W["ln_post.b"]), 1e-5)
    assert got.shape == (ecfg.n_ctx, ecfg.d_model)
    np.testing.assert_allclose(got, x.numpy(), atol=1e-9)


def test_bf16_operands_change_little():
    ecfg = MICRO_ENC
    W = make_encoder_weights(ecfg).values
    mel = log_mel(make_audio(ecfg, 0), ecfg.n_mels)
    a = Encoder(ecfg, W, OracleOpts(dtype=np.float32)).forward(mel)
    b = Encoder(ecfg, W, OracleOpts(dtype=np.float32, gemm_bf16=True)).forward(mel)
    d = np.abs(a - b)
    assert 0 < d.max() < 0.1 and d.mean() < 0.01


def test_large_v3_encoder_parameter_count():
    # Whisper large-v3's encoder: 635,048,960 parameters at these shapes (the position
    # table is fixed, not learned)
    assert param_count(encoder_manifest(LARGE_V3_ENC)) == 635_048_960
