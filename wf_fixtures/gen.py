"""Seeded generators for weights, acoustic memories, prompts and planted drafts.

Random initialisation: every matrix, embedding, bias and the mask vector is
drawn N(0, 0.02); LayerNorm gains are 1 + N(0, 0.02) and LayerNorm shifts
N(0, 0.02), so the affine path of every norm is exercised.  Draws come from
numpy's ``default_rng(seed)`` in manifest order, in fp32.  For bf16 shapes
each fp32 draw is rounded once to bf16 (round to nearest even) and both
sides use exactly those bf16 values.

The acoustic memory stands in for the encoder output of one 30 s window:
N(0, 1) of shape [1500, d].  Prompt tokens are uniform over the vocabulary
minus the end-of-transcript id.
"""
import numpy as np

from .manifest import full_manifest


def bf16_round_bits(x):
    """fp32 array -> uint16 bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bits_to_f32(b):
    """uint16 bf16 bit patterns -> fp32 values (exact)."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


class WeightSet:
    """Parameter values keyed by manifest name.

    ``values[name]`` is an fp32 array holding the exact parameter values
    (already bf16-representable for bf16 shapes).  ``bits(name)`` gives the
    uint16 bf16 pattern of a bf16 parameter.
    """

    def __init__(self, cfg, values, order):
        self.cfg = cfg
        self.values = values
        self.order = order

    def __getitem__(self, name):
        return self.values[name]

    def bits(self, name):
        v = self.values[name]
        return (v.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


def _is_ln_gain(name):
    return name.endswith("_ln.g") or name.endswith("ln_f.g")


def _is_drafter(name):
    return name.startswith("d.") or (name[0] == "d" and name[1].isdigit())


def _fill(out, seed, index, name, std):
    """Draw one parameter into ``out`` (a view of the flat buffer)."""
    rng = np.random.default_rng([seed, index])
    rng.standard_normal(out=out, dtype=np.float32)
    out *= np.float32(std)
    if _is_ln_gain(name):
        out += np.float32(1.0)


def _round_inplace(flat):
    """Round an fp32 buffer to bf16 values in place (round to nearest even)."""
    u = flat.view(np.uint32)
    step = 1 << 24
    tmp = np.empty(min(step, u.size), dtype=np.uint32)
    for i in range(0, u.size, step):
        blk = u[i:i + step]
        t = tmp[:blk.size]
        np.right_shift(blk, np.uint32(16), out=t)
        np.bitwise_and(t, np.uint32(1), out=t)
        np.add(t, np.uint32(0x7FFF), out=t)
        np.add(blk, t, out=blk)
        np.bitwise_and(blk, np.uint32(0xFFFF0000), out=blk)


def _draw_manifest(order, seed_of, dtype, threads, std):
    from concurrent.futures import ThreadPoolExecutor

    sizes = [int(np.prod(shape)) for _, shape in order]
    flat = np.empty(sum(sizes), dtype=np.float32)
    views, off = [], 0
    for (name, shape), n in zip(order, sizes):
        views.append(flat[off:off + n])
        off += n

    def work(i):
        name = order[i][0]
        _fill(views[i], seed_of(name), i, name, std)
        if dtype == "bf16":
            _round_inplace(views[i])

    idx = sorted(range(len(order)), key=lambda i: -sizes[i])
    with ThreadPoolExecutor(max_workers=threads) as ex:
        list(ex.map(work, idx))
    return flat, {name: v.reshape(shape) for (name, shape), v in zip(order, views)}


def make_encoder_weights(ecfg, seed=2, threads=8, std=0.02):
    """Whisper encoder parameters in manifest order, drawn as the decoder's are
    (N(0, std), LayerNorm gains 1 + N(0, std)), rounded to bf16 for bf16 shapes."""
    from .manifest import encoder_manifest
    order = encoder_manifest(ecfg)
    flat, values = _draw_manifest(order, lambda name: seed, ecfg.dtype, threads, std)
    ws = WeightSet(ecfg, values, order)
    ws.flat = flat
    return ws


def make_audio(ecfg, slot, seed_base=600):
    """Synthetic 16 kHz waveform of one request (n_samples long): a few harmonic
    tones with random fundamentals, a slow amplitude envelope and a little white
    noise, peak level about 0.3 (fp32)."""
    rng = np.random.default_rng(seed_base + slot)
    n = ecfg.n_samples
    t = np.arange(n) / ecfg.sample_rate
    x = np.zeros(n)
    for _ in range(3):
        f0 = rng.uniform(90.0, 300.0)
        env = 0.5 + 0.5 * np.sin(2 * np.pi * rng.uniform(0.5, 3.0) * t + rng.uniform(0, 2 * np.pi))
        for hmn in range(1, 6):
            x += (0.05 / hmn) * env * np.sin(2 * np.pi * f0 * hmn * t + rng.uniform(0, 2 * np.pi))
    x += 0.005 * rng.standard_normal(n)
    return x.astype(np.float32)


def make_weights(cfg, seed_target=0, seed_drafter=1, threads=8, std=0.02):
    """All target and drafter parameters for ``cfg``.

    ``std`` (0.02 for every workload) may be raised for the 64-token sampling
    check, where sharper distributions give the chi-square test its power.

    Parameter number i of the manifest (counting from 0) is drawn from
    ``default_rng([seed, i])`` with ``seed = seed_target`` for target
    parameters and ``seed_drafter`` for drafter parameters.  The draw does
    not depend on the thread count.
    """
    order = full_manifest(cfg)
    seed_of = lambda name: seed_drafter if _is_drafter(name) else seed_target
    flat, values = _draw_manifest(order, seed_of, cfg.dtype, threads, std)
    ws = WeightSet(cfg, values, order)
    ws.flat = flat
    return ws


def make_memory(cfg, slot, seed_base=100):
    """Acoustic memory stand-in for one request: N(0,1) of shape [n_frames, d]."""
    rng = np.random.default_rng(seed_base + slot)
    a = rng.standard_normal((cfg.n_frames, cfg.d_model), dtype=np.float32)
    if cfg.dtype == "bf16":
        a = bits_to_f32(bf16_round_bits(a)).reshape(a.shape)
    return a


def make_prefix(cfg, slot, length, seed_base=200):
    """Prompt token ids for one request: uniform over [0, V) minus the EOS id."""
    rng = np.random.default_rng(seed_base + slot)
    toks = rng.integers(0, cfg.n_vocab - 1, size=length, dtype=np.int64)
    if 0 <= cfg.eos_id < cfg.n_vocab:
        toks = np.where(toks >= cfg.eos_id, toks + 1, toks)
    return toks.astype(np.int32)


def make_prefix_lengths(n, lo, hi, seed=300):
    """n prompt lengths uniform on the integers [lo, hi]."""
    rng = np.random.default_rng(seed)
    return rng.integers(lo, hi + 1, size=n).astype(np.int32)


def plant_drafts(cont, r, n_vocab, rng):
    """Planted draft block from the target's own continuation ``cont`` (length K).

    Position r (0-based) is replaced by a different token, so a greedy
    verifier accepts exactly r candidates; r == K leaves the block intact.
    """
    d = np.array(cont, dtype=np.int32).copy()
    if r < len(d):
        d[r] = (int(d[r]) + 1 + int(rng.integers(0, n_vocab - 1))) % n_vocab
    return d
