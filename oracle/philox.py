"""Philox4x64-10 counter-based generator (test infrastructure only).

Philox (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as
1, 2, 3", SC'11) maps a 256-bit counter and a 128-bit key to 256 random
bits through ten rounds.  One round with multipliers M0, M1 takes counter
(c0, c1, c2, c3) and key (k0, k1) to

    (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))

and the key advances by the Weyl constants (W0, W1) between rounds.

Stream layout used for the decoding randomness (one uniform per draw):
  key     = (seed, 0)
  counter = (purpose << 32 | slot, step, pos, v >> 2); word v & 3 of the output
where purpose names the decision (plain sample, draft sample, acceptance
test, residual sample, bonus sample, prefill sample), step is the slot's
verify-call counter, pos the row within the call and v the vocabulary index
(0 for scalar draws).
A 64-bit word x becomes the fp32 uniform ((x >> 41) + 0.5) * 2^-23 in (0, 1),
and a uniform u becomes Gumbel noise -log(-log(u)) in fp32.
"""
import numpy as np

M0 = np.uint64(0xD2E7470EE14C6C93)
M1 = np.uint64(0xCA5A826395121157)
W0 = np.uint64(0x9E3779B97F4A7C15)
W1 = np.uint64(0xBB67AE8584CAA73B)
_MASK32 = np.uint64(0xFFFFFFFF)
_S32 = np.uint64(32)


def _mulhilo(a, b):
    """Full 128-bit product of uint64 arrays, as (hi, lo)."""
    a = np.asarray(a, np.uint64)
    b = np.asarray(b, np.uint64)
    a0, a1 = a & _MASK32, a >> _S32
    b0, b1 = b & _MASK32, b >> _S32
    p00 = a0 * b0
    p01 = a0 * b1
    p10 = a1 * b0
    p11 = a1 * b1
    mid = (p00 >> _S32) + (p01 & _MASK32) + (p10 & _MASK32)
    lo = (p00 & _MASK32) | ((mid & _MASK32) << _S32)
    hi = p11 + (p01 >> _S32) + (p10 >> _S32) + (mid >> _S32)
    return hi, lo


def philox4x64(ctr, key, rounds=10):
    """ctr [..., 4] uint64, key (k0, k1) -> [..., 4] uint64."""
    c = np.array(ctr, dtype=np.uint64, copy=True)
    c0, c1, c2, c3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = np.uint64(key[0])
    k1 = np.uint64(key[1])
    with np.errstate(over="ignore"):
        for r in range(rounds):
            if r > 0:
                k0 = k0 + W0
                k1 = k1 + W1
            hi0, lo0 = _mulhilo(M0, c0)
            hi1, lo1 = _mulhilo(M1, c2)
            c0, c1, c2, c3 = hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0
    return np.stack([c0, c1, c2, c3], axis=-1)


def raw_words(seed, purpose, slot, step, pos, n):
    """n consecutive 64-bit words of the stream (purpose, slot, step, pos)."""
    nb = (n + 3) // 4
    ctr = np.zeros((nb, 4), np.uint64)
    ctr[:, 0] = (np.uint64(purpose) << _S32) | np.uint64(slot)
    ctr[:, 1] = np.uint64(step)
    ctr[:, 2] = np.uint64(pos)
    ctr[:, 3] = np.arange(nb, dtype=np.uint64)
    return philox4x64(ctr, (seed, 0)).reshape(-1)[:n]


def to_uniform(x):
    m = (np.asarray(x, np.uint64) >> np.uint64(41)).astype(np.float32)
    return (m + np.float32(0.5)) * np.float32(2.0 ** -23)


def uniforms(seed, purpose, slot, step, pos, n):
    return to_uniform(raw_words(seed, purpose, slot, step, pos, n))


def gumbel(u):
    u = np.asarray(u, np.float32)
    return -np.log(-np.log(u))
