"""Pins of the oracle's drafter ablation variants (CPU only).

The paper's ablations (Section 5.4 Table 3; Appendix Table A4) train drafters
without direct audio (47.5M parameters), without the target history (52.5M),
with absolute positions instead of RoPE, and with five layers.  Their
parameter counts pin the first two architectures; closed forms under
constructed weights pin what each variant computes:

  * no audio: removing the cross-attention sub-layer equals keeping it with a
    zero output projection;
  * no history: the drafter's output does not depend on the prompt's history,
    and a zero query averages the nine block values only;
  * absolute positions: with zero output projections mask row j gives
    LN_df(m + P[t + j]) E^T; a constant query and key (which RoPE would turn
    into a one-hot attention) give uniform attention (no rotation).
"""
import numpy as np
import torch

from wf_fixtures import MICRO, LARGE_V3, make_weights, make_memory, make_prefix
from wf_fixtures.manifest import drafter_manifest, param_count
from oracle import OracleOpts, Target, Drafter, Session

F64 = OracleOpts(dtype=np.float64)
PROMPT = 20


def _ln(x, g, b):
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    return torch.nn.functional.layer_norm(t(x), (x.shape[-1],), t(g), t(b), 1e-5).numpy()


def _values(cfg):
    W = make_weights(cfg)
    return {k: np.array(v, np.float64) for k, v in W.values.items()}


def _zero(V, name):
    V[name] = np.zeros_like(V[name])


def _zero_outputs(V, cfg, blocks, parts):
    for l in blocks:
        for p in parts:
            if f"d{l}.{p}.w" in V:
                _zero(V, f"d{l}.{p}.w")
                _zero(V, f"d{l}.{p}.b")


def _session(cfg, V, slot=0, prompt=None):
    T, D = Target(cfg, V, F64), Drafter(cfg, V, F64)
    prompt = make_prefix(cfg, slot, PROMPT) if prompt is None else prompt
    return Session(T, D, make_memory(cfg, slot).astype(np.float64), prompt, cfg.n_ctx)


def _head(V, x):
    return _ln(x, V["d.ln_f.g"], V["d.ln_f.b"]) @ V["tok_emb"].T


def test_variant_parameter_counts():
    """Trainable drafter parameters at large-v3 shapes: the paper's 60.7M / 47.5M /
    52.5M (Table 3 caption); the absolute-position variant adds none (it uses the
    target's frozen position table); five layers add three blocks."""
    full = param_count(drafter_manifest(LARGE_V3))
    assert full == 60_669_440
    assert param_count(drafter_manifest(LARGE_V3.with_(draft_audio=False))) == 47_549_440
    assert param_count(drafter_manifest(LARGE_V3.with_(draft_history=False))) == 52_476_160
    assert param_count(drafter_manifest(LARGE_V3.with_(draft_pos="abs"))) == full
    five = param_count(drafter_manifest(LARGE_V3.with_(n_draft_layer=5)))
    per_block = (full - param_count(drafter_manifest(LARGE_V3.with_(n_draft_layer=1))))
    assert five == full + 3 * per_block == 139_377_920


def test_no_audio_equals_zero_cross_output():
    full = MICRO
    cfg = MICRO.with_(name="micro-noaudio", draft_audio=False)
    V = _values(full)
    Vz = dict(V)
    _zero_outputs(Vz, full, range(full.n_draft_layer), ["xattn.o"])
    a = _session(full, Vz).draft_logits()
    Vn = {k: v for k, v in V.items() if not (k.startswith("d") and ".xattn" in k)}
    b = _session(cfg, Vn).draft_logits()
    np.testing.assert_allclose(b, a, rtol=0, atol=1e-9)
    # and it differs from the drafter that reads the audio
    assert np.abs(_session(full, V).draft_logits() - b).max() > 1e-3


def test_no_history_ignores_the_prompt_and_averages_block_values():
    cfg = MICRO.with_(name="micro-nohist", draft_history=False)
    V = {k: v for k, v in _values(cfg).items() if not k.startswith("d.hproj")}
    # two requests with different prompts of the same length and the same anchor
    s1 = _session(cfg, V, 0)
    p2 = make_prefix(cfg, 5, PROMPT)
    s2 = _session(cfg, V, 0, prompt=p2)
    s2.anchor = s1.anchor
    np.testing.assert_allclose(s1.draft_logits(), s2.draft_logits(), rtol=0, atol=1e-12)
    # zero query: uniform weights over the nine block rows only
    _zero(V, "d0.attn.q.w")
    _zero(V, "d0.attn.q.b")
    _zero_outputs(V, cfg, [0], ["xattn.o", "mlp.fc2"])
    _zero_outputs(V, cfg, range(1, cfg.n_draft_layer), ["attn.o", "xattn.o", "mlp.fc2"])
    s = _session(cfg, V)
    x0 = np.concatenate([V["tok_emb"][[s.anchor]], np.repeat(V["d.mask"][None], cfg.block_k, 0)])
    vb = _ln(x0, V["d0.attn_ln.g"], V["d0.attn_ln.b"]) @ V["d0.attn.v.w"].T + V["d0.attn.v.b"]
    x = x0 + vb.mean(axis=0) @ V["d0.attn.o.w"].T + V["d0.attn.o.b"]
    np.testing.assert_allclose(s.draft_logits(), _head(V, x[1:]), rtol=0, atol=1e-6)


def test_absolute_positions_add_the_position_table():
    cfg = MICRO.with_(name="micro-abs", draft_pos="abs")
    V = _values(cfg)
    _zero_outputs(V, cfg, range(cfg.n_draft_layer), ["attn.o", "xattn.o", "mlp.fc2"])
    s = _session(cfg, V)
    t = s.L
    x = V["d.mask"][None] + V["pos_emb"][t + 1:t + cfg.block_k + 1]
    got = s.draft_logits()
    np.testing.assert_allclose(got, _head(V, x), rtol=0, atol=1e-6)
    assert np.abs(got[1] - got[0]).max() > 1e-3  # rows differ through their positions


def test_absolute_positions_do_not_rotate():
    """Constant queries and keys (the construction that RoPE turns into a one-hot
    attention at a fixed offset) give equal scores without RoPE: every row takes
    the mean of all values (history < t and the block)."""
    cfg = MICRO.with_(name="micro-abs", draft_pos="abs")
    V = _values(cfg)
    d, hd = cfg.d_model, cfg.head_dim
    g, b = V["d0.attn_ln.g"], V["d0.attn_ln.b"]
    g[d // 2:] = 0.0
    b[d // 2:] = 0.0
    b[d // 2] = 1.0
    wk = np.zeros((d, d))
    wk[:hd // 2, d // 2] = 21.0
    V["d0.attn.k.w"] = wk
    V["d0.attn.q.w"] = np.zeros((d, d))
    bq = np.zeros(d)
    bq[:hd // 2] = 21.0
    V["d0.attn.q.b"] = bq
    _zero_outputs(V, cfg, [0], ["xattn.o", "mlp.fc2"])
    _zero_outputs(V, cfg, range(1, cfg.n_draft_layer), ["attn.o", "xattn.o", "mlp.fc2"])
    s = _session(cfg, V)
    t = s.L
    T = Target(cfg, V, F64)
    mem = make_memory(cfg, 0).astype(np.float64)
    _, taps = T.forward(T.new_cache(), make_prefix(cfg, 0, PROMPT), 0, T.cross_kv(mem))
    hp = taps.reshape(t, -1) @ V["d.hproj.w"].T + V["d.hproj.b"]
    x0 = np.concatenate([V["tok_emb"][[s.anchor]], np.repeat(V["d.mask"][None], cfg.block_k, 0)])
    x0 = x0 + V["pos_emb"][t:t + cfg.block_k + 1]
    vals = np.concatenate([_ln(hp, g, b), _ln(x0, g, b)]) @ V["d0.attn.v.w"].T + V["d0.attn.v.b"]
    x = x0 + vals.mean(axis=0) @ V["d0.attn.o.w"].T + V["d0.attn.o.b"]
    np.testing.assert_allclose(s.draft_logits(), _head(V, x[1:]), rtol=0, atol=1e-6)
