"""Elementary operations of the oracle (test infrastructure only).

Every function is the textbook definition written out in numpy, with no
blocking or fusion:

  LayerNorm    y = g * (x - mean) / sqrt(var + 1e-5) + b, biased variance
               (Whisper's pre-LN blocks and final LN).
  GELU         0.5 * x * (1 + erf(x / sqrt(2))), the exact-erf form.
  attention    softmax(q k^T / sqrt(64)) v per head, max subtracted, in the
               working precision; masked keys get -inf.
  RoPE         rotate-half rotary embedding with base 10000 and fp32 phases
               (Appendix A.2): pair (i, i+32) of each 64-wide head is rotated
               by theta = fp32(p) * fp32(10000^(-2i/64)), the product taken
               in fp32; cos/sin of that fp32 angle are evaluated in fp64 and
               rounded to fp32.
  bf16         round-to-nearest-even to an 8-bit significand, the storage
               format of caches in the bf16 configuration.
"""
from dataclasses import dataclass

import numpy as np
from scipy.special import erf


@dataclass(frozen=True)
class OracleOpts:
    """Precision choices.

    dtype      working precision of all arithmetic (float32 by default).
    kv_bf16    round cross-attention K/V, the target's self-attention K/V cache
               and the drafter's history K/V to bf16 where they are stored.
    gemm_bf16  round the input rows of every weight product to bf16 (the
               large-batch matrix-core regime).
    exact      compute weight products one row at a time, so a row's result
               never depends on how many rows share the pass.
    """
    dtype: type = np.float32
    kv_bf16: bool = False
    gemm_bf16: bool = False
    exact: bool = True


def bf16(x):
    """Round to the nearest bf16 value (ties to even), returned in x's dtype."""
    x = np.asarray(x)
    m, e = np.frexp(x.astype(np.float64))
    r = np.ldexp(np.rint(m * 256.0) / 256.0, e)
    return r.astype(x.dtype)


def layer_norm(x, g, b, dt, eps=1e-5):
    x = x.astype(dt, copy=False)
    mu = np.mean(x, axis=-1, keepdims=True, dtype=dt)
    c = x - mu
    var = np.mean(c * c, axis=-1, keepdims=True, dtype=dt)
    return (c / np.sqrt(var + dt(eps))) * g.astype(dt) + b.astype(dt)


def gelu(x):
    dt = x.dtype.type
    return dt(0.5) * x * (dt(1.0) + erf(x / dt(np.sqrt(2.0))).astype(x.dtype))


def linear(x, w, b, opts):
    """x @ w.T + b for x [R, in], w [out, in]."""
    dt = opts.dtype
    x = x.astype(dt, copy=False)
    if opts.gemm_bf16:
        x = bf16(x)
    w = w.astype(dt, copy=False)
    if opts.exact:
        y = np.stack([w @ x[r] for r in range(x.shape[0])]) if x.shape[0] else np.zeros((0, w.shape[0]), dt)
    else:
        y = x @ w.T
    if b is not None:
        y = y + b.astype(dt)
    return y.astype(dt, copy=False)


def softmax(s, axis=-1):
    m = np.max(s, axis=axis, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=axis, keepdims=True)


def attention(q, k, v, allowed, dt):
    """Multi-head attention.

    q [R, H, hd], k/v [T, H, hd]; allowed [R, T] boolean (True = may attend).
    Returns [R, H*hd].  Scores are scaled by 1/sqrt(hd) once.
    """
    R, H, hd = q.shape
    scale = dt(1.0 / np.sqrt(hd))
    out = np.zeros((R, H, hd), dt)
    for h in range(H):
        s = (q[:, h, :].astype(dt) @ k[:, h, :].astype(dt).T) * scale
        s = np.where(allowed, s, dt(-np.inf))
        p = softmax(s, axis=-1).astype(dt)
        out[:, h, :] = p @ v[:, h, :].astype(dt)
    return out.reshape(R, H * hd)


def rope_tables(positions, hd=64):
    """cos/sin [len(positions), hd/2] for rotate-half RoPE with fp32 phases."""
    half = hd // 2
    omega = np.array([10000.0 ** (-2.0 * i / hd) for i in range(half)], dtype=np.float64).astype(np.float32)
    p = np.asarray(positions).astype(np.float32)
    theta = (p[:, None] * omega[None, :]).astype(np.float32)  # fp32 product
    c = np.cos(theta.astype(np.float64)).astype(np.float32)
    s = np.sin(theta.astype(np.float64)).astype(np.float32)
    return c, s


def rope(x, positions, dt):
    """Rotate-half RoPE on x [R, H, hd] at text positions [R]."""
    R, H, hd = x.shape
    half = hd // 2
    c, s = rope_tables(positions, hd)
    c = c.astype(dt)[:, None, :]
    s = s.astype(dt)[:, None, :]
    u1 = x[..., :half].astype(dt)
    u2 = x[..., half:].astype(dt)
    return np.concatenate([u1 * c - u2 * s, u1 * s + u2 * c], axis=-1).astype(dt)
