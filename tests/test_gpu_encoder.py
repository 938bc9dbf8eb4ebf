"""The Whisper audio encoder on the HIP path (through the C ABI) against the oracle.

  * the log-mel frontend (fp64 on both sides) agrees to 1e-5;
  * the acoustic memory agrees with the oracle computed with the same bf16
    rounding of every product input (fp32 accumulation on both sides; the
    difference comes from accumulation order flipping bf16 roundings of
    intermediate values), at micro and large-v3 shapes;
  * end to end: waveform -> GPU encoder -> wf_encode_memory_set -> prefill ->
    draft + verify steps, against the oracle decoding from its own encoder
    output (logits within the decoder's bf16 tolerance, tokens identical
    wherever the margin exceeds it).
"""
import numpy as np
import pytest
import torch

from wf_fixtures import (MICRO, MICRO_ENC, LARGE_V3_ENC, make_encoder_weights, make_audio, make_weights,
                         make_prefix)
from oracle import OracleOpts
from oracle.encoder import Encoder, log_mel
from oracle.numerics import bf16

pytestmark = pytest.mark.gpu

ENC_OPTS = OracleOpts(dtype=np.float32, gemm_bf16=True, exact=False)
# acoustic memory: unit-scale LayerNorm output stored in bf16, whose ulp is 2^-7 = 7.8e-3
# for |A| in [1, 2): any element may differ by one stored ulp where an accumulation
# order flipped a rounding; the mean stays far below it
TOL_MEM_MAX, TOL_MEM_MEAN = 8e-3, 5e-4


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _encoder(ecfg):
    from paper_2609_32869_amd import WhisperEncoder
    W = make_encoder_weights(ecfg)
    return WhisperEncoder.from_host(ecfg, [W.values[n] for n, _ in W.order]), W


def test_logmel_frontend():
    ecfg = MICRO_ENC
    enc, _ = _encoder(ecfg)
    for slot in range(2):
        x = make_audio(ecfg, slot)
        got = enc.logmel(torch.from_numpy(x).cuda()).cpu().numpy()
        want = log_mel(x, ecfg.n_mels)
        print(f"log-mel slot {slot}: max |d| {np.abs(got - want).max():.2e}")
        np.testing.assert_allclose(got, want, rtol=0, atol=1e-5)
    enc.close()


def _compare_memory(ecfg, nreq):
    enc, W = _encoder(ecfg)
    audio = np.stack([make_audio(ecfg, s) for s in range(nreq)])
    got = enc.run(torch.from_numpy(audio).cuda()).float().cpu().numpy()
    E = Encoder(ecfg, W.values, ENC_OPTS)
    for s in range(nreq):
        want = bf16(E.encode(audio[s]))
        d = np.abs(got[s] - want)
        print(f"{ecfg.name} request {s}: max |dA| {d.max():.3e}, mean {d.mean():.3e}, "
              f"share > 1e-2 {np.mean(d > 1e-2):.2e}", flush=True)
        assert d.max() <= TOL_MEM_MAX and d.mean() <= TOL_MEM_MEAN
    enc.close()


def test_micro_encoder_matches_oracle():
    _compare_memory(MICRO_ENC, 2)


@pytest.mark.timeout(900)
def test_large_v3_encoder_matches_oracle():
    _compare_memory(LARGE_V3_ENC, 1)


def test_waveform_to_tokens_micro():
    """Waveform -> GPU encoder -> decoder steps, against the oracle decoding from its
    own encoder output (the decoder's acoustic memory is the only coupling)."""
    from lockstep import Lockstep
    ecfg, cfg = MICRO_ENC, MICRO.with_(name="micro-bf16-audio", dtype="bf16", n_vocab=501)
    assert cfg.n_frames == ecfg.n_ctx and cfg.d_model == ecfg.d_model
    enc, EW = _encoder(ecfg)
    audio = np.stack([make_audio(ecfg, s) for s in range(2)])
    mem_gpu = enc.run(torch.from_numpy(audio).cuda())
    E = Encoder(ecfg, EW.values, ENC_OPTS)
    mems = [bf16(E.encode(audio[s])).astype(np.float32) for s in range(2)]
    W = make_weights(cfg)
    prompts = [make_prefix(cfg, 0, 6), make_prefix(cfg, 1, 11)]
    ls = Lockstep(cfg, W, prompts, [30, 30], 2e-2, opts=OracleOpts(dtype=np.float32, kv_bf16=True), mems=mems)
    ls.eng.encode_memory_set(0, mem_gpu)          # the GPU decoder reads the GPU encoder's memory
    ls.eng.prefill(0, torch.from_numpy(np.stack([np.pad(p, (0, 11 - len(p))) for p in prompts]).astype(np.int32)).cuda(),
                   [len(p) for p in prompts], [30, 30])
    for _ in range(4):
        ls.step()
    print(f"waveform->tokens: max |dlogit| draft {ls.max_dlogit:.2e} target {ls.max_tlogit:.2e}, near ties {ls.near_ties}")
    ls.close()
    enc.close()
