"""Pins of the oracle's target decoder and drafter (CPU only)."""
import numpy as np
import pytest
import torch

from wf_fixtures import MICRO, LARGE_V3, make_weights, make_memory, make_prefix
from wf_fixtures.manifest import drafter_manifest, param_count
from oracle import OracleOpts, Target, Drafter

F64 = OracleOpts(dtype=np.float64)
F32 = OracleOpts(dtype=np.float32)


def _torch_block(W, cfg, l):
    d, H, F = cfg.d_model, cfg.n_head, cfg.d_ff
    layer = torch.nn.TransformerDecoderLayer(d, H, F, dropout=0.0, activation="gelu", layer_norm_eps=1e-5,
                                             batch_first=True, norm_first=True, dtype=torch.float64)
    t = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    p = f"t{l}."
    with torch.no_grad():
        layer.self_attn.in_proj_weight.copy_(t(np.concatenate([W[p + "attn.q.w"], W[p + "attn.k.w"], W[p + "attn.v.w"]])))
        layer.self_attn.in_proj_bias.copy_(t(np.concatenate([W[p + "attn.q.b"], np.zeros(d), W[p + "attn.v.b"]])))
        layer.self_attn.out_proj.weight.copy_(t(W[p + "attn.o.w"]))
        layer.self_attn.out_proj.bias.copy_(t(W[p + "attn.o.b"]))
        layer.multihead_attn.in_proj_weight.copy_(t(np.concatenate([W[p + "xattn.q.w"], W[p + "xattn.k.w"], W[p + "xattn.v.w"]])))
        layer.multihead_attn.in_proj_bias.copy_(t(np.concatenate([W[p + "xattn.q.b"], np.zeros(d), W[p + "xattn.v.b"]])))
        layer.multihead_attn.out_proj.weight.copy_(t(W[p + "xattn.o.w"]))
        layer.multihead_attn.out_proj.bias.copy_(t(W[p + "xattn.o.b"]))
        layer.linear1.weight.copy_(t(W[p + "mlp.fc1.w"]))
        layer.linear1.bias.copy_(t(W[p + "mlp.fc1.b"]))
        layer.linear2.weight.copy_(t(W[p + "mlp.fc2.w"]))
        layer.linear2.bias.copy_(t(W[p + "mlp.fc2.b"]))
        for norm, name in ((layer.norm1, "attn_ln"), (layer.norm2, "xattn_ln"), (layer.norm3, "mlp_ln")):
            norm.weight.copy_(t(W[p + name + ".g"]))
            norm.bias.copy_(t(W[p + name + ".b"]))
    return layer.eval()


def test_target_blocks_match_torch_decoder_layer(micro):
    """A Whisper decoder block is a pre-LN transformer decoder layer with exact GELU and
    no key bias; chaining torch's layer reproduces the oracle's residual stream after
    every tapped block."""
    cfg, W = micro
    W = W.values
    mem = make_memory(cfg, 0)
    toks = make_prefix(cfg, 0, 13)
    T = Target(cfg, W, F64)
    logits, taps = T.forward(T.new_cache(), toks, 0, T.cross_kv(mem))
    h = torch.from_numpy(W["tok_emb"][toks].astype(np.float64) + W["pos_emb"][:13].astype(np.float64))[None]
    memt = torch.from_numpy(mem.astype(np.float64))[None]
    mask = torch.nn.Transformer.generate_square_subsequent_mask(13, dtype=torch.float64)
    with torch.no_grad():
        for l in range(cfg.n_layer):
            h = _torch_block(W, cfg, l)(h, memt, tgt_mask=mask)
            np.testing.assert_allclose(taps[:, cfg.taps.index(l)], h[0].numpy(), rtol=0, atol=1e-10)
        hf = torch.nn.functional.layer_norm(h, (cfg.d_model,), torch.from_numpy(W["ln_f.g"].astype(np.float64)),
                                            torch.from_numpy(W["ln_f.b"].astype(np.float64)), 1e-5)
        ref = hf[0] @ torch.from_numpy(W["tok_emb"].astype(np.float64)).T
    np.testing.assert_allclose(logits, ref.numpy(), rtol=0, atol=1e-5)  # logits are returned in fp32


def test_incremental_cache_equals_one_pass(micro):
    cfg, W = micro
    mem = make_memory(cfg, 1)
    toks = make_prefix(cfg, 1, 20)
    T = Target(cfg, W.values, F64)
    xkv = T.cross_kv(mem)
    full, taps_full = T.forward(T.new_cache(), toks, 0, xkv)
    cache = T.new_cache()
    a, ta = T.forward(cache, toks[:7], 0, xkv)
    b, tb = T.forward(cache, toks[7:9], 7, xkv)
    c, tc = T.forward(cache, toks[9:], 9, xkv)
    np.testing.assert_allclose(np.concatenate([a, b, c]), full, atol=1e-6)
    np.testing.assert_allclose(np.concatenate([ta, tb, tc]), taps_full, atol=1e-12)


def test_verify_is_causal(micro):
    """Row i of one causal pass does not depend on the tokens after it."""
    cfg, W = micro
    mem = make_memory(cfg, 2)
    toks = make_prefix(cfg, 2, 12)
    T = Target(cfg, W.values, F64)
    xkv = T.cross_kv(mem)
    base, _ = T.forward(T.new_cache(), toks, 0, xkv)
    alt = toks.copy()
    alt[8:] = (alt[8:] + 17) % cfg.n_vocab
    other, _ = T.forward(T.new_cache(), alt, 0, xkv)
    np.testing.assert_array_equal(base[:8], other[:8])
    assert np.abs(base[8:] - other[8:]).max() > 1e-3


def test_cross_attention_invariant_to_frame_order(micro):
    cfg, W = micro
    mem = make_memory(cfg, 3)
    toks = make_prefix(cfg, 3, 6)
    T = Target(cfg, W.values, F64)
    base, _ = T.forward(T.new_cache(), toks, 0, T.cross_kv(mem))
    perm = np.random.default_rng(0).permutation(cfg.n_frames)
    other, _ = T.forward(T.new_cache(), toks, 0, T.cross_kv(mem[perm]))
    np.testing.assert_allclose(base, other, atol=1e-9)


def _hist_from_teacher(cfg, W, mem, seq, opts):
    T, D = Target(cfg, W, opts), Drafter(cfg, W, opts)
    _, taps = T.forward(T.new_cache(), seq, 0, T.cross_kv(mem))
    hc = D.new_cache()
    D.history_update(hc, taps, 0)
    return D, hc


def test_draft_ignores_history_at_or_after_anchor(micro):
    """A mask position never sees history at or beyond its anchor (Appendix A.2)."""
    cfg, W = micro
    mem = make_memory(cfg, 4)
    seq = make_prefix(cfg, 4, 15)
    D, hc = _hist_from_teacher(cfg, W.values, mem, seq, F64)
    dxkv = D.cross_kv(mem)
    t = 10
    base = D.forward(hc, t, seq[t], dxkv)
    hc.K[:, t:] = np.nan
    hc.V[:, t:] = np.nan
    poisoned = D.forward(hc, t, seq[t], dxkv)
    assert np.all(np.isfinite(poisoned))
    np.testing.assert_array_equal(base, poisoned)
    # but history before the anchor does matter
    hc.K[:, 3] += 1.0
    assert np.abs(D.forward(hc, t, seq[t], dxkv) - base).max() > 1e-6


def test_mask_rows_see_each_other(micro):
    """Attention inside the draft block is bidirectional: mask row 1 depends on the
    mask vector content at rows after it only through the block attention, so
    changing the anchor changes every mask row."""
    cfg, W = micro
    mem = make_memory(cfg, 5)
    seq = make_prefix(cfg, 5, 9)
    D, hc = _hist_from_teacher(cfg, W.values, mem, seq, F64)
    dxkv = D.cross_kv(mem)
    a = D.forward(hc, 8, seq[8], dxkv)
    b = D.forward(hc, 8, (seq[8] + 1) % cfg.n_vocab, dxkv)
    assert np.all(np.abs(a - b).max(axis=1) > 1e-6)


def test_history_written_across_rounds_equals_teacher_forced(micro):
    """History K/V written round by round equal those from one teacher-forced pass."""
    cfg, W = micro
    mem = make_memory(cfg, 6)
    seq = make_prefix(cfg, 6, 20)
    D, hc_full = _hist_from_teacher(cfg, W.values, mem, seq, F64)
    T = Target(cfg, W.values, F64)
    xkv = T.cross_kv(mem)
    cache, hc = T.new_cache(), D.new_cache()
    for lo, hi in ((0, 5), (5, 6), (6, 14), (14, 20)):
        _, taps = T.forward(cache, seq[lo:hi], lo, xkv)
        D.history_update(hc, taps, lo)
    np.testing.assert_allclose(hc.K[:, :20], hc_full.K[:, :20], atol=1e-12)
    np.testing.assert_allclose(hc.V[:, :20], hc_full.V[:, :20], atol=1e-12)


def test_drafter_rope_relative_positions(micro):
    """History keys carry RoPE at their own text positions: writing the same history
    rows at positions shifted by 20 and rotating a query at a position shifted by 20
    leaves every query-key score unchanged up to fp32 phase rounding."""
    from oracle.numerics import rope
    cfg, W = micro
    mem = make_memory(cfg, 7)
    seq = make_prefix(cfg, 7, 12)
    T, D = Target(cfg, W.values, F64), Drafter(cfg, W.values, F64)
    _, taps = T.forward(T.new_cache(), seq, 0, T.cross_kv(mem))
    h0, h1 = D.new_cache(), D.new_cache()
    shift = 20
    D.history_update(h0, taps[:10], 0)
    D.history_update(h1, taps[:10], shift)
    q = np.random.default_rng(0).standard_normal((1, cfg.n_head, 64))
    qa = rope(q, [10], np.float64)[0]
    qb = rope(q, [10 + shift], np.float64)[0]
    for l in range(cfg.n_draft_layer):
        for hd in range(cfg.n_head):
            ka = h0.K[l, :10, hd * 64:(hd + 1) * 64]
            kb = h1.K[l, shift:shift + 10, hd * 64:(hd + 1) * 64]
            sa, sb = ka @ qa[hd], kb @ qb[hd]
            np.testing.assert_allclose(sa, sb, atol=1e-4 * (1 + np.abs(sa).max()))
            np.testing.assert_array_equal(h0.V[l, :10], h1.V[l, shift:shift + 10])


def test_drafter_parameter_counts_match_paper():
    """60.7M trainable drafter parameters (Section 3.2); 47.5M without the audio path and
    52.5M without the history projection (Table 3 caption)."""
    m = drafter_manifest(LARGE_V3)
    full = param_count(m)
    no_audio = param_count(m, ("d0.xattn", "d1.xattn"))
    no_hist = param_count(m, ("d.hproj",))
    assert round(full / 1e6, 1) == 60.7
    assert round(no_audio / 1e6, 1) == 47.5
    assert round(no_hist / 1e6, 1) == 52.5
    assert full == 60_669_440
