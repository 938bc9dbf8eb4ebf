"""Weight manifest: the fixed order and shapes in which parameters are
generated and handed to the C-ABI (``wf_init_weights`` takes one pointer per
entry, in this order).

Linear weights are stored ``[out, in]``; a projection computes x @ W.T + b.
Following Whisper's decoder block, the key projections of self- and
cross-attention carry no bias.

Target (frozen Whisper decoder, Section 4):
  tok_emb [V, d] (also the tied output head), pos_emb [n_ctx, d], then per
  block: self-attention pre-LN and q/k/v/o, cross-attention pre-LN and
  q/k/v/o, MLP pre-LN and fc1/fc2; final LN.

Drafter (Section 3.2 and Appendix A.2): the history projection from the
concatenated taps (n_tap*d -> d), the learned mask vector m of Eq. 2, two
blocks with the same layout as a target block (own acoustic key/value
projections), and a final LN before the shared output head.
"""


def _block(prefix, d, f):
    return [
        (f"{prefix}.attn_ln.g", (d,)), (f"{prefix}.attn_ln.b", (d,)),
        (f"{prefix}.attn.q.w", (d, d)), (f"{prefix}.attn.q.b", (d,)),
        (f"{prefix}.attn.k.w", (d, d)),
        (f"{prefix}.attn.v.w", (d, d)), (f"{prefix}.attn.v.b", (d,)),
        (f"{prefix}.attn.o.w", (d, d)), (f"{prefix}.attn.o.b", (d,)),
        (f"{prefix}.xattn_ln.g", (d,)), (f"{prefix}.xattn_ln.b", (d,)),
        (f"{prefix}.xattn.q.w", (d, d)), (f"{prefix}.xattn.q.b", (d,)),
        (f"{prefix}.xattn.k.w", (d, d)),
        (f"{prefix}.xattn.v.w", (d, d)), (f"{prefix}.xattn.v.b", (d,)),
        (f"{prefix}.xattn.o.w", (d, d)), (f"{prefix}.xattn.o.b", (d,)),
        (f"{prefix}.mlp_ln.g", (d,)), (f"{prefix}.mlp_ln.b", (d,)),
        (f"{prefix}.mlp.fc1.w", (f, d)), (f"{prefix}.mlp.fc1.b", (f,)),
        (f"{prefix}.mlp.fc2.w", (d, f)), (f"{prefix}.mlp.fc2.b", (d,)),
    ]


BLOCK_FIELDS = [n.split(".", 1)[1] for n, _ in _block("x", 1, 1)]


def target_manifest(cfg):
    d, f = cfg.d_model, cfg.d_ff
    m = [("tok_emb", (cfg.n_vocab, d)), ("pos_emb", (cfg.n_ctx, d))]
    for l in range(cfg.n_layer):
        m += _block(f"t{l}", d, f)
    m += [("ln_f.g", (d,)), ("ln_f.b", (d,))]
    return m


def drafter_manifest(cfg):
    """The drafter's parameters; the ablation variants drop the history projection
    (no target history) or every block's cross-attention sub-layer with its
    LayerNorm (no direct audio)."""
    d, f = cfg.d_model, cfg.d_ff
    m = []
    if getattr(cfg, "draft_history", True):
        m += [("d.hproj.w", (d, cfg.n_tap * d)), ("d.hproj.b", (d,))]
    m += [("d.mask", (d,))]
    for l in range(cfg.n_draft_layer):
        blk = _block(f"d{l}", d, f)
        if not getattr(cfg, "draft_audio", True):
            blk = [(n, s) for n, s in blk if ".xattn" not in n]
        m += blk
    m += [("d.ln_f.g", (d,)), ("d.ln_f.b", (d,))]
    return m


def full_manifest(cfg):
    return target_manifest(cfg) + drafter_manifest(cfg)


def param_count(manifest, exclude_prefixes=()):
    n = 0
    for name, shape in manifest:
        if any(name.startswith(p) for p in exclude_prefixes):
            continue
        k = 1
        for s in shape:
            k *= s
        n += k
    return n


def encoder_manifest(ecfg):
    """Whisper encoder parameters: the convolution stem (weights [out, in, 3]),
    n_layer blocks (self-attention without a key bias, GELU MLP) and ln_post."""
    d, f, m = ecfg.d_model, ecfg.d_ff, ecfg.n_mels
    out = [("conv1.w", (d, m, 3)), ("conv1.b", (d,)), ("conv2.w", (d, d, 3)), ("conv2.b", (d,))]
    for l in range(ecfg.n_layer):
        p = f"e{l}"
        out += [(f"{p}.attn_ln.g", (d,)), (f"{p}.attn_ln.b", (d,)),
                (f"{p}.attn.q.w", (d, d)), (f"{p}.attn.q.b", (d,)),
                (f"{p}.attn.k.w", (d, d)),
                (f"{p}.attn.v.w", (d, d)), (f"{p}.attn.v.b", (d,)),
                (f"{p}.attn.o.w", (d, d)), (f"{p}.attn.o.b", (d,)),
                (f"{p}.mlp_ln.g", (d,)), (f"{p}.mlp_ln.b", (d,)),
                (f"{p}.mlp.fc1.w", (f, d)), (f"{p}.mlp.fc1.b", (f,)),
                (f"{p}.mlp.fc2.w", (d, f)), (f"{p}.mlp.fc2.b", (d,))]
    out += [("ln_post.g", (d,)), ("ln_post.b", (d,))]
    return out
