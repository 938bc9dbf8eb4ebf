"""Decoding loops of the oracle (test infrastructure only).

``Session`` holds one request (one slot) in the state the paper's execution
keeps (Appendix A.1): the target cache and the drafter history hold exactly
the text positions before the anchor; the anchor (the latest emitted token)
is not yet processed.  One ``step`` is one draft-and-verify round:

  1. draft: the drafter proposes K tokens from the anchor, the history and
     the acoustic memory (Section 3.2);
  2. verify: one causal target pass over [anchor, c_1..c_k] (Section 3.1);
  3. accept: greedy longest-prefix rule or the rejection rule (accept.py);
  4. update: the cache keeps L+1+a positions (old anchor + accepted
     candidates), the correction/bonus becomes the next anchor, and the
     history gains the states of those 1+a positions.

The history rows of all k+1 verified positions are written right after the
verify pass; positions at or beyond the new length are never read (the
drafter reads history strictly before its anchor) and are overwritten by a
later round.

``plain_greedy`` is Eq. 1 with a KV cache; ``brute_greedy`` recomputes the
whole sequence for every token (no cache).  With k_max = 0 a speculative
session performs exactly plain decoding.
"""
import numpy as np

from .accept import budget_k, greedy_accept, rejection_accept, softmax32, gumbel_argmax, argmax_first
from .philox import uniforms, gumbel

PREFILL, PLAIN, DRAFT, ACC, RES, BON = 1, 2, 3, 4, 5, 6


class Session:
    def __init__(self, target, drafter, mem, prompt, max_new, slot=0, temperature=0.0, seed=500,
                 suppress=None):
        self.t, self.d = target, drafter
        self.cfg = target.cfg
        self.slot = slot
        self.temperature = float(temperature)
        self.inv_t = np.float32(1.0 / temperature) if temperature > 0 else None
        self.seed = seed
        self.suppress = suppress
        self.max_new = int(max_new)
        self.xkv = target.cross_kv(mem)
        self.dxkv = drafter.cross_kv(mem) if drafter is not None else None
        self.cache = target.new_cache()
        self.hcache = drafter.new_cache() if drafter is not None else None
        self.step_no = 0
        self.out = []
        self.done = False
        self.history = []          # per step: dict(k, a, tokens)
        self._prefill(np.asarray(prompt, np.int64))

    # -- prefill (Appendix A.1): process the prompt, emit the first anchor
    def _prefill(self, prompt):
        P = len(prompt)
        logits, taps = self.t.forward(self.cache, prompt, 0, self.xkv, self.suppress)
        if self.d is not None:
            self.d.history_update(self.hcache, taps, 0)
        self.L = P
        self.last_logits = logits
        if self.inv_t is None:
            first = argmax_first(logits[-1])
        else:
            g = gumbel(uniforms(self.seed, PREFILL, self.slot, 0, 0, self.cfg.n_vocab))
            first = gumbel_argmax(logits[-1].astype(np.float32) * self.inv_t, g)
        self.anchor = first
        self.out = [first]
        self.done = (first == self.cfg.eos_id) or self.max_new <= 1 or self.L >= self.cfg.n_ctx

    @property
    def emitted(self):
        return len(self.out)

    def budget(self, k_max):
        return budget_k(self.cfg.block_k, k_max, self.max_new, self.emitted, self.cfg.n_ctx, self.L)

    # -- drafting (Section 3.2)
    def draft_logits(self):
        return self.d.forward(self.hcache, self.L, self.anchor, self.dxkv, self.suppress)

    def draft(self):
        """Drafted tokens c_1..c_K (greedy argmax, or Gumbel-max samples) and draft logits."""
        lq = self.draft_logits()
        K = self.cfg.block_k
        if self.inv_t is None:
            return np.array([argmax_first(lq[j]) for j in range(K)], np.int32), lq
        toks = []
        for j in range(K):
            g = gumbel(uniforms(self.seed, DRAFT, self.slot, self.step_no, j + 1, self.cfg.n_vocab))
            toks.append(gumbel_argmax(lq[j].astype(np.float32) * self.inv_t, g))
        return np.array(toks, np.int32), lq

    # -- verify + accept + update (Section 3.1, Appendix A.1)
    def verify_accept(self, drafts, k_max, draft_logits=None):
        if self.done:
            return None
        k = self.budget(k_max)
        if k < 0:
            self.done = True
            return None
        drafts = np.asarray(drafts, np.int64)[:k]
        rows = np.concatenate([[self.anchor], drafts]).astype(np.int64)
        logits, taps = self.t.forward(self.cache, rows, self.L, self.xkv, self.suppress)
        if self.d is not None:
            self.d.history_update(self.hcache, taps, self.L)
        self.last_logits = logits
        if self.inv_t is None:
            g = [argmax_first(logits[i]) for i in range(k + 1)]
            a, toks, fin = greedy_accept(drafts, g, self.cfg.eos_id)
        else:
            if k == 0:
                gp = gumbel(uniforms(self.seed, PLAIN, self.slot, self.step_no, 0, self.cfg.n_vocab))
                tok = gumbel_argmax(logits[0].astype(np.float32) * self.inv_t, gp)
                a, toks, fin = 0, [tok], tok == self.cfg.eos_id
            else:
                q = softmax32(draft_logits[:k], self.inv_t)
                p = softmax32(logits, self.inv_t)
                u = uniforms(self.seed, ACC, self.slot, self.step_no, 0, k)
                gres = np.stack([gumbel(uniforms(self.seed, RES, self.slot, self.step_no, j + 1, self.cfg.n_vocab))
                                 for j in range(k)])
                gbon = gumbel(uniforms(self.seed, BON, self.slot, self.step_no, 0, self.cfg.n_vocab))
                a, toks, fin = rejection_accept(drafts, q, p, u, gres, logits, self.inv_t, gbon, self.cfg.eos_id)
        self.out.extend(toks)
        self.L += 1 + a
        self.anchor = toks[-1]
        self.step_no += 1
        self.done = fin or self.emitted >= self.max_new or self.L >= self.cfg.n_ctx
        rec = dict(k=k, a=a, tokens=toks)
        self.history.append(rec)
        return rec

    def step(self, k_max=None, draft_override=None):
        """One draft-and-verify round.  ``draft_override`` replaces the drafted tokens."""
        if self.done:
            return None
        if k_max is None:
            k_max = self.cfg.block_k
        lq = None
        if self.d is not None and k_max > 0:
            drafts, lq = self.draft()
        else:
            drafts = np.zeros(self.cfg.block_k, np.int32)
        if draft_override is not None:
            drafts = np.asarray(draft_override, np.int32)
        return self.verify_accept(drafts, k_max, lq)

    def run(self, k_max=None, draft_fn=None, max_steps=100000):
        n = 0
        while not self.done and n < max_steps:
            ov = draft_fn(self) if draft_fn is not None else None
            self.step(k_max, ov)
            n += 1
        return list(self.out)


def plain_greedy(target, mem, prompt, max_new):
    """Eq. 1: y_{t+1} = argmax_v p(v | x, y_<=t), one token per target call, with a KV cache."""
    s = Session(target, None, mem, prompt, max_new)
    return s.run(k_max=0)


def brute_greedy(target, mem, prompt, max_new):
    """Eq. 1 without any cache: every token recomputes the whole sequence."""
    cfg = target.cfg
    xkv = target.cross_kv(mem)
    seq = [int(t) for t in prompt]
    out = []
    while True:
        cache = target.new_cache()
        logits, _ = target.forward(cache, seq, 0, xkv)
        tok = argmax_first(logits[-1])
        out.append(tok)
        seq.append(tok)
        if tok == cfg.eos_id or len(out) >= max_new or len(seq) > cfg.n_ctx:
            return out


def spec_greedy(target, drafter, mem, prompt, max_new, k_max=None, draft_fn=None):
    s = Session(target, drafter, mem, prompt, max_new)
    return s.run(k_max=k_max, draft_fn=draft_fn), s


def plain_sample(target, mem, prompt, max_new, temperature, seed=500, slot=0):
    s = Session(target, None, mem, prompt, max_new, slot=slot, temperature=temperature, seed=seed)
    return s.run(k_max=0)


def spec_sample(target, drafter, mem, prompt, max_new, temperature, seed=500, slot=0, k_max=None):
    s = Session(target, drafter, mem, prompt, max_new, slot=slot, temperature=temperature, seed=seed)
    return s.run(k_max=k_max), s
