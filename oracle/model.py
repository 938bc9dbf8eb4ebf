"""Target decoder and drafter of the oracle (test infrastructure only).

Target: the frozen Whisper decoder the paper verifies with (Section 4,
Whisper large-v3).  A row at text position p starts from tok_emb[y_p] +
pos_emb[p]; each block is pre-LN self-attention (causal: position p sees
positions 0..p), pre-LN cross-attention to the acoustic memory A (all 1500
frames), and a pre-LN GELU MLP, each added to the residual stream.  The
key projections carry no bias.  The logits of position p are
LN_f(h_p) @ tok_emb^T and predict the token at p+1 (Section 3.1).

The cross-attention keys and values depend only on A, so they are computed
once per request (Appendix A.5: each request refreshes the acoustic K/V of
target and drafter).

Drafter (Section 3.2, Eq. 2, Appendix A.2):
  * history memory: for each verified position p, the residual streams after
    target blocks ``cfg.taps`` (taken before the final LN) are concatenated
    and projected to width d:  Hproj[p] = concat_s(T_s[p]) @ W_h^T + b_h;
  * the draft block X_t = [Emb(y_t), m, ..., m] has K+1 rows at text
    positions t..t+K (t is the anchor's position);
  * in each drafter block the block rows' queries attend, in ONE softmax, to
    keys/values of the projected history at positions < t and of the block
    itself (every block row sees every other block row); history and block
    rows go through the same pre-LN and the same W_k/W_v; queries and keys
    carry RoPE at their explicit text positions; then cross-attention to the
    drafter's own K/V of A and a GELU MLP;
  * mask row j (position t+j) predicts the token at t+j via the drafter's
    final LN and the shared output head.
Because history keys/values of a position never change once written, they
are cached per drafter block (``HistoryCache``).

Pin status.  The target block is pinned to torch's pre-LN decoder layer and
the decoding loop to plain greedy decoding.  The drafter is pinned by
properties (history at or beyond the anchor is never read, RoPE scores are
relative, history written round by round equals a teacher-forced pass, the
parameter count matches the paper's 60.7M / 47.5M / 52.5M) and by closed
forms under constructed weights (tests/test_oracle_drafter_pins.py): with
zero output projections every mask row's logits are LN_df(m) E^T; a zero
query makes each row the mean of the values of history < t (through the
block's pre-LN) and of the whole block; a zero cross-attention query gives
the mean of the drafter's own acoustic values; a constant pre-RoPE key and
a query rotated by -D omega make mask row j copy the history row at
position t + j - D.
"""
import numpy as np

from .numerics import layer_norm, gelu, linear, attention, rope, bf16


def _blk(W, prefix):
    return {k.split(".", 1)[1]: v for k, v in W.items() if k.startswith(prefix + ".")}


class TargetCache:
    """Self-attention K/V of every target block at text positions 0..n_ctx-1."""

    def __init__(self, cfg, dt):
        self.K = np.zeros((cfg.n_layer, cfg.n_ctx, cfg.d_model), dt)
        self.V = np.zeros((cfg.n_layer, cfg.n_ctx, cfg.d_model), dt)


class HistoryCache:
    """Drafter history K (after RoPE) and V per drafter block and text position."""

    def __init__(self, cfg, dt):
        self.K = np.zeros((cfg.n_draft_layer, cfg.n_ctx, cfg.d_model), dt)
        self.V = np.zeros((cfg.n_draft_layer, cfg.n_ctx, cfg.d_model), dt)


def _store(x, opts):
    return bf16(x) if opts.kv_bf16 else x


def _cross_kv(blocks, mem, prefix, opts):
    out = []
    for b in blocks:
        k = linear(mem, b[f"{prefix}.k.w"], None, opts)
        v = linear(mem, b[f"{prefix}.v.w"], b[f"{prefix}.v.b"], opts)
        out.append((_store(k, opts), _store(v, opts)))
    return out


def _cross_attend(b, x, kv, H, opts):
    dt = opts.dtype
    c = layer_norm(x, b["xattn_ln.g"], b["xattn_ln.b"], dt)
    q = linear(c, b["xattn.q.w"], b["xattn.q.b"], opts)
    K, V = kv
    R, d = q.shape
    hd = d // H
    allowed = np.ones((R, K.shape[0]), bool)
    o = attention(q.reshape(R, H, hd), K.reshape(-1, H, hd), V.reshape(-1, H, hd), allowed, dt)
    return linear(o, b["xattn.o.w"], b["xattn.o.b"], opts)


def _mlp(b, x, opts):
    dt = opts.dtype
    m = layer_norm(x, b["mlp_ln.g"], b["mlp_ln.b"], dt)
    u = gelu(linear(m, b["mlp.fc1.w"], b["mlp.fc1.b"], opts))
    return linear(u, b["mlp.fc2.w"], b["mlp.fc2.b"], opts)


class Target:
    def __init__(self, cfg, W, opts):
        self.cfg, self.opts = cfg, opts
        dt = opts.dtype
        self.E = W["tok_emb"].astype(dt)
        self.P = W["pos_emb"].astype(dt)
        self.blocks = [_blk(W, f"t{l}") for l in range(cfg.n_layer)]
        self.lnf = (W["ln_f.g"], W["ln_f.b"])

    def cross_kv(self, mem):
        return _cross_kv(self.blocks, mem, "xattn", self.opts)

    def new_cache(self):
        return TargetCache(self.cfg, self.opts.dtype)

    def forward(self, cache, tokens, pos0, xkv, suppress=None):
        """Causal pass over rows at text positions pos0..pos0+R-1.

        Writes their keys/values into ``cache`` and attends row i to cached
        positions 0..pos0+i.  Returns (logits [R, V], taps [R, n_tap, d]).
        """
        cfg, opts, dt = self.cfg, self.opts, self.opts.dtype
        tokens = np.asarray(tokens, dtype=np.int64)
        R, H, d = len(tokens), cfg.n_head, cfg.d_model
        hd = d // H
        assert pos0 + R <= cfg.n_ctx
        pos = np.arange(pos0, pos0 + R)
        h = self.E[tokens] + self.P[pos]
        T = pos0 + R
        allowed = np.arange(T)[None, :] <= pos[:, None]
        taps = []
        for l, b in enumerate(self.blocks):
            a = layer_norm(h, b["attn_ln.g"], b["attn_ln.b"], dt)
            q = linear(a, b["attn.q.w"], b["attn.q.b"], opts)
            k = linear(a, b["attn.k.w"], None, opts)
            v = linear(a, b["attn.v.w"], b["attn.v.b"], opts)
            cache.K[l, pos0:T] = _store(k, opts)
            cache.V[l, pos0:T] = _store(v, opts)
            o = attention(q.reshape(R, H, hd), cache.K[l, :T].reshape(T, H, hd),
                          cache.V[l, :T].reshape(T, H, hd), allowed, dt)
            h = h + linear(o, b["attn.o.w"], b["attn.o.b"], opts)
            h = h + _cross_attend(b, h, xkv[l], H, opts)
            h = h + _mlp(b, h, opts)
            if l in cfg.taps:
                taps.append(h.copy())
        hf = layer_norm(h, self.lnf[0], self.lnf[1], dt)
        logits = linear(hf, self.E, None, opts).astype(np.float32)
        if suppress is not None:
            logits[:, suppress] = -np.inf
        return logits, np.stack(taps, axis=1)


class Drafter:
    """The block drafter.  Ablation variants (Section 5.4 Table 3, Table A4) follow
    ``cfg.draft_audio`` (False: the blocks have no cross-attention sub-layer),
    ``cfg.draft_history`` (False: no history projection; the block attends to its
    own nine rows only) and ``cfg.draft_pos`` ("abs": no RoPE; the target's learned
    position table, shared and frozen like the token embedding, is added to the
    block rows at positions t..t+K)."""

    def __init__(self, cfg, W, opts):
        self.cfg, self.opts = cfg, opts
        dt = opts.dtype
        self.audio = getattr(cfg, "draft_audio", True)
        self.hist = getattr(cfg, "draft_history", True)
        self.use_rope = getattr(cfg, "draft_pos", "rope") == "rope"
        self.E = W["tok_emb"].astype(dt)          # shared embedding / output head
        self.P = W["pos_emb"].astype(dt)          # shared position table (absolute-position variant)
        if self.hist:
            self.Wh, self.bh = W["d.hproj.w"], W["d.hproj.b"]
        self.m = W["d.mask"].astype(dt)
        self.blocks = [_blk(W, f"d{l}") for l in range(cfg.n_draft_layer)]
        self.lnf = (W["d.ln_f.g"], W["d.ln_f.b"])

    def cross_kv(self, mem):
        if not self.audio:
            return None
        return _cross_kv(self.blocks, mem, "xattn", self.opts)

    def new_cache(self):
        return HistoryCache(self.cfg, self.opts.dtype)

    def history_proj(self, taps):
        """Hproj rows from taps [R, n_tap, d] (concatenated in ascending block order)."""
        R = taps.shape[0]
        return linear(taps.reshape(R, -1), self.Wh, self.bh, self.opts)

    def _block_kv(self, b, a, positions):
        H, d = self.cfg.n_head, self.cfg.d_model
        hd = d // H
        k = linear(a, b["attn.k.w"], None, self.opts)
        if self.use_rope:
            k = rope(k.reshape(-1, H, hd), positions, self.opts.dtype).reshape(-1, d)
        v = linear(a, b["attn.v.w"], b["attn.v.b"], self.opts)
        return k, v

    def history_update(self, hcache, taps, pos0):
        """Write history K/V of rows at positions pos0.. from their target taps."""
        if not self.hist:
            return
        dt = self.opts.dtype
        hp = self.history_proj(taps)
        pos = np.arange(pos0, pos0 + hp.shape[0])
        for l, b in enumerate(self.blocks):
            a = layer_norm(hp, b["attn_ln.g"], b["attn_ln.b"], dt)
            k, v = self._block_kv(b, a, pos)
            hcache.K[l, pos] = _store(k, self.opts)
            hcache.V[l, pos] = _store(v, self.opts)

    def forward(self, hcache, t, anchor, dxkv, suppress=None, return_hidden=False):
        """Draft logits [K, V] for mask rows 1..K of the block anchored at position t.

        History positions 0..t-1 of ``hcache`` are read; nothing at or beyond t.
        """
        cfg, opts, dt = self.cfg, self.opts, self.opts.dtype
        K, H, d = cfg.block_k, cfg.n_head, cfg.d_model
        hd = d // H
        x = np.concatenate([self.E[[int(anchor)]], np.repeat(self.m[None, :], K, axis=0)]).astype(dt)
        pos = np.arange(t, t + K + 1)
        if not self.use_rope:
            x = x + self.P[np.minimum(pos, cfg.n_ctx - 1)]
        nh = t if self.hist else 0
        for l, b in enumerate(self.blocks):
            a = layer_norm(x, b["attn_ln.g"], b["attn_ln.b"], dt)
            q = linear(a, b["attn.q.w"], b["attn.q.b"], opts).reshape(-1, H, hd)
            if self.use_rope:
                q = rope(q, pos, dt)
            kb, vb = self._block_kv(b, a, pos)
            Kall = np.concatenate([hcache.K[l, :nh], kb]).reshape(-1, H, hd)
            Vall = np.concatenate([hcache.V[l, :nh], vb]).reshape(-1, H, hd)
            allowed = np.ones((K + 1, nh + K + 1), bool)
            o = attention(q, Kall, Vall, allowed, dt)
            x = x + linear(o, b["attn.o.w"], b["attn.o.b"], opts)
            if self.audio:
                x = x + _cross_attend(b, x, dxkv[l], H, opts)
            x = x + _mlp(b, x, opts)
        hf = layer_norm(x[1:], self.lnf[0], self.lnf[1], dt)
        logits = linear(hf, self.E, None, opts).astype(np.float32)
        if suppress is not None:
            logits[:, suppress] = -np.inf
        if return_hidden:
            return logits, x
        return logits
