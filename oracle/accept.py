"""Acceptance rules of the oracle (test infrastructure only).

Indices: a verify call processes rows 0..k at text positions L..L+k holding
[anchor, c_1, ..., c_k].  Target row i predicts the token at L+i+1, so
candidate c_j (position L+j) is checked against target row j-1.

Greedy (Section 3.1): keep candidates while they equal the target's argmax;
emit the target's token at the first disagreement, or a bonus token (the
argmax of row k) when all k agree.  An accepted end-of-transcript token ends
the transcript with no bonus (Appendix A.1).

Sampling (Section 3.1, Appendix A.4): candidate c_j, drawn from the draft
distribution q_j, is accepted with probability min(1, p_j(c_j)/q_j(c_j)),
where p_j is the target distribution of row j-1; this is decided as
u * q_j(c_j) < p_j(c_j) with a uniform u.  At the first rejection the token
is drawn from the normalised residual (p_j - q_j)_+; after a fully accepted
block a bonus is drawn from row k's target distribution.  Draws use the
Gumbel-max rule: argmax_v (log w_v + g_v) is a draw from w / sum(w).

Budget (Appendix A.1): with R output tokens left, at most R-1 candidates are
proposed; no position at or beyond n_ctx is ever processed.
"""
import numpy as np


def budget_k(block_k, k_max, max_new, emitted, n_ctx, L):
    """Number of candidates to verify this round, or -1 if the sequence is finished."""
    left = max_new - emitted
    if left <= 0 or L >= n_ctx:
        return -1
    return max(0, min(block_k, k_max, left - 1, n_ctx - L - 1))


def argmax_first(x):
    """Index of the maximum; ties go to the lowest index."""
    return int(np.argmax(x))


def greedy_accept(drafts, g, eos):
    """drafts: c_1..c_k; g: target argmax of rows 0..k.

    Returns (a, tokens, finished): a accepted candidates, emitted tokens,
    and whether an end-of-transcript token was emitted.
    """
    k = len(drafts)
    assert len(g) == k + 1
    a = 0
    while a < k and int(drafts[a]) == int(g[a]):
        a += 1
    for e in range(a):
        if int(drafts[e]) == eos:
            return e + 1, [int(t) for t in drafts[:e + 1]], True
    toks = [int(t) for t in drafts[:a]] + [int(g[a])]
    return a, toks, toks[-1] == eos


def softmax32(logits, inv_t):
    """fp32 softmax of logits * inv_t (inv_t an fp32 scalar); -inf entries get 0."""
    z = logits.astype(np.float32) * np.float32(inv_t)
    m = np.max(z, axis=-1, keepdims=True)
    e = np.exp(z - m)
    return (e / np.sum(e, axis=-1, keepdims=True)).astype(np.float32)


def gumbel_argmax(score, g):
    return argmax_first(score.astype(np.float32) + g.astype(np.float32))


def rejection_accept(drafts, q, p, u_acc, g_res, logits_p, inv_t, g_bon, eos):
    """Speculative rejection rule for one verify call.

    drafts [k]; q [k, V] draft probabilities of c_1..c_k; p [k+1, V] target
    probabilities of rows 0..k; u_acc [k] acceptance uniforms; g_res [k, V]
    Gumbel noise for a residual draw at candidate j; logits_p [k+1, V] target
    logits; g_bon [V] Gumbel noise for the bonus.
    Returns (a, tokens, finished).
    """
    k = len(drafts)
    for j in range(k):
        c = int(drafts[j])
        if not (np.float32(u_acc[j]) * q[j, c] < p[j, c]):
            r = p[j] - q[j]
            pos = r > 0
            if np.any(pos):
                with np.errstate(divide="ignore"):
                    score = np.where(pos, np.log(np.where(pos, r, 1.0)).astype(np.float32), np.float32(-np.inf))
            else:
                with np.errstate(divide="ignore"):
                    score = np.log(p[j]).astype(np.float32)
            tok = gumbel_argmax(score, g_res[j])
            toks = [int(t) for t in drafts[:j]] + [tok]
            return j, toks, tok == eos
        if c == eos:
            return j + 1, [int(t) for t in drafts[:j + 1]], True
    tok = gumbel_argmax(logits_p[k].astype(np.float32) * np.float32(inv_t), g_bon)
    toks = [int(t) for t in drafts] + [tok]
    return k, toks, tok == eos
