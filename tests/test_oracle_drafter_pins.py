"""Pins of the oracle's drafter forward with constructed weights (CPU only).

The drafter has no printed values to compare with, so these tests choose
weights for which the drafter's output has a closed form that follows from
its definition (Section 3.2, Eq. 2; Appendix A.2) by plain algebra, and
compare the oracle with that closed form.  Every test runs through
``Session`` (prefill of a real prompt through the target, history written
from the target's taps, then a draft), so the wiring between target taps,
history, acoustic memories and the drafter is covered as well.

  * zero outputs: with every drafter sub-layer's output projection and bias
    set to zero, each block passes its rows through unchanged, so the logits
    of every mask row j = 1..8 equal LN_df(m) E^T with the drafter's own final
    LayerNorm;
  * uniform self-attention: with W_q = 0 and b_q = 0 every score is zero, so
    each block row receives the plain mean of the values of all keys it may
    see: the projected history at positions < t passed through the block's
    pre-LN and W_v, and the nine block rows.  All mask rows then get the same
    output (the block is bidirectional);
  * uniform cross-attention: with W'_q = 0 and b'_q = 0 each row receives the
    mean over frames of the drafter's OWN acoustic values A W'_v^T + b'_v;
  * one-hot relative attention: with keys made constant before RoPE (a
    LayerNorm gain of zero on half of the width leaves only the shift there)
    and a constant query rotated by -D * omega_i per frequency, the score of
    a query at position p and a key at position p' is a^2 sum_i cos((p - p'
    - D) omega_i), which peaks only at p - p' = D; mask row j (text position
    t + j) then copies the value of the history row at position t + j - D.

The mistakes each test is meant to catch are listed in the design notes.
"""
import numpy as np
import torch

from wf_fixtures import MICRO, make_weights, make_memory, make_prefix
from oracle import OracleOpts, Target, Drafter, Session

F64 = OracleOpts(dtype=np.float64)
PROMPT = 20
D_OFFSET = 12    # row j at t + j reads history position t + j - 12 (all < t for t = 20)
A_SCALE = 21.0   # |q_i| = |k_i|; score gap a^2 (32 - 30.92) / 8 > 59 against the nearest offset


def _ln(x, g, b):
    """LayerNorm by torch's routine (independent of the oracle's numpy code), fp64."""
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    return torch.nn.functional.layer_norm(t(x), (x.shape[-1],), t(g), t(b), 1e-5).numpy()


def _values():
    cfg = MICRO
    W = make_weights(cfg)
    return cfg, {k: np.array(v, np.float64) for k, v in W.values.items()}


def _zero(V, name):
    V[name] = np.zeros_like(V[name])


def _zero_outputs(V, cfg, blocks, parts=("attn.o", "xattn.o", "mlp.fc2")):
    for l in blocks:
        for p in parts:
            _zero(V, f"d{l}.{p}.w")
            _zero(V, f"d{l}.{p}.b")


def _session(cfg, V, slot=0):
    T, D = Target(cfg, V, F64), Drafter(cfg, V, F64)
    mem = make_memory(cfg, slot).astype(np.float64)
    prompt = make_prefix(cfg, slot, PROMPT)
    s = Session(T, D, mem, prompt, cfg.n_ctx)
    return s, T, mem, prompt


def _block_rows(V, cfg, anchor):
    return np.concatenate([V["tok_emb"][[anchor]], np.repeat(V["d.mask"][None], cfg.block_k, 0)])


def _head_logits(V, x):
    return _ln(x, V["d.ln_f.g"], V["d.ln_f.b"]) @ V["tok_emb"].T


def _taps(T, mem, prompt):
    _, taps = T.forward(T.new_cache(), prompt, 0, T.cross_kv(mem))
    return taps


def test_zero_output_blocks_give_mask_logits_from_own_final_norm():
    cfg, V = _values()
    _zero_outputs(V, cfg, range(cfg.n_draft_layer))
    s, _, _, _ = _session(cfg, V)
    got = s.draft_logits()
    want = _head_logits(V, V["d.mask"][None])[0]
    assert got.shape == (cfg.block_k, cfg.n_vocab)
    for j in range(cfg.block_k):
        np.testing.assert_allclose(got[j], want, rtol=0, atol=1e-6)
    # the target's final norm differs (its gains are drawn separately)
    other = _ln(V["d.mask"][None], V["ln_f.g"], V["ln_f.b"])[0] @ V["tok_emb"].T
    assert np.abs(other - want).max() > 1e-3


def test_uniform_self_attention_is_mean_of_history_and_block_values():
    cfg, V = _values()
    _zero(V, "d0.attn.q.w")
    _zero(V, "d0.attn.q.b")
    _zero_outputs(V, cfg, [0], ("xattn.o", "mlp.fc2"))
    _zero_outputs(V, cfg, range(1, cfg.n_draft_layer))
    s, T, mem, prompt = _session(cfg, V)
    t = s.L
    assert t == PROMPT
    # history rows: taps of the prompt positions -> W_h -> block pre-LN -> W_v
    taps = _taps(T, mem, prompt)
    hp = taps.reshape(t, -1) @ V["d.hproj.w"].T + V["d.hproj.b"]
    g, b = V["d0.attn_ln.g"], V["d0.attn_ln.b"]
    v_hist = _ln(hp, g, b) @ V["d0.attn.v.w"].T + V["d0.attn.v.b"]
    x0 = _block_rows(V, cfg, s.anchor)
    v_blk = _ln(x0, g, b) @ V["d0.attn.v.w"].T + V["d0.attn.v.b"]
    mean_v = np.concatenate([v_hist, v_blk]).mean(axis=0)
    x = x0 + mean_v @ V["d0.attn.o.w"].T + V["d0.attn.o.b"]
    want = _head_logits(V, x[1:])
    got = s.draft_logits()
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-6)
    # bidirectional block: every mask row sees the same keys, so their logits agree
    assert np.abs(got - got[0]).max() < 1e-9


def test_uniform_cross_attention_reads_the_drafters_own_acoustic_values():
    cfg, V = _values()
    _zero_outputs(V, cfg, [0], ("attn.o", "mlp.fc2"))
    _zero(V, "d0.xattn.q.w")
    _zero(V, "d0.xattn.q.b")
    _zero_outputs(V, cfg, range(1, cfg.n_draft_layer))
    s, _, mem, _ = _session(cfg, V)
    x0 = _block_rows(V, cfg, s.anchor)
    mean_v = (mem @ V["d0.xattn.v.w"].T + V["d0.xattn.v.b"]).mean(axis=0)
    x = x0 + mean_v @ V["d0.xattn.o.w"].T + V["d0.xattn.o.b"]
    want = _head_logits(V, x[1:])
    np.testing.assert_allclose(s.draft_logits(), want, rtol=0, atol=1e-6)
    # the target block 0's acoustic values would give a different result
    mean_t = (mem @ V["t0.xattn.v.w"].T + V["t0.xattn.v.b"]).mean(axis=0)
    other = _head_logits(V, (x0 + mean_t @ V["d0.xattn.o.w"].T + V["d0.xattn.o.b"])[1:])
    assert np.abs(other - want).max() > 1e-3


def test_one_hot_relative_attention_reads_history_at_fixed_offset():
    cfg, V = _values()
    d, hd = cfg.d_model, cfg.head_dim
    half = hd // 2
    # block 0 pre-LN: gain 0 on columns d/2.., shift e_{d/2} there, so those LN
    # outputs are exactly (1, 0, ..., 0) for every row (history and block alike)
    g = V["d0.attn_ln.g"]
    b = V["d0.attn_ln.b"]
    g[d // 2:] = 0.0
    b[d // 2:] = 0.0
    b[d // 2] = 1.0
    # keys of head 0: k_i = a (i < 32), k_{i+32} = 0, from that constant column; head 1: 0
    wk = np.zeros((d, d))
    wk[:half, d // 2] = A_SCALE
    V["d0.attn.k.w"] = wk
    # queries: constant a * exp(-i D omega_i) per frequency pair of head 0; head 1: 0
    omega = np.array([10000.0 ** (-2.0 * i / hd) for i in range(half)], np.float64).astype(np.float32).astype(np.float64)
    V["d0.attn.q.w"] = np.zeros((d, d))
    bq = np.zeros(d)
    bq[:half] = A_SCALE * np.cos(D_OFFSET * omega)
    bq[half:hd] = -A_SCALE * np.sin(D_OFFSET * omega)
    V["d0.attn.q.b"] = bq
    # values of head 0: the first 64 LN outputs; head 1: zero (uniform over zeros)
    wv = np.zeros((d, d))
    wv[:hd, :hd] = np.eye(hd)
    V["d0.attn.v.w"] = wv
    V["d0.attn.v.b"] = np.zeros(d)
    _zero_outputs(V, cfg, [0], ("xattn.o", "mlp.fc2"))
    _zero_outputs(V, cfg, range(1, cfg.n_draft_layer))
    s, T, mem, prompt = _session(cfg, V)
    t = s.L
    taps = _taps(T, mem, prompt)
    hp = taps.reshape(t, -1) @ V["d.hproj.w"].T + V["d.hproj.b"]
    x0 = _block_rows(V, cfg, s.anchor)
    rows = []
    for j in range(1, cfg.block_k + 1):
        src = t + j - D_OFFSET
        assert 0 <= src < t
        o = np.zeros(d)
        o[:hd] = _ln(hp[src][None], g, b)[0, :hd]
        rows.append(x0[j] + o @ V["d0.attn.o.w"].T + V["d0.attn.o.b"])
    want = _head_logits(V, np.stack(rows))
    got = s.draft_logits()
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-6)
    # the rows read different history positions, so their logits differ
    assert np.abs(got[1] - got[0]).max() > 1e-3
