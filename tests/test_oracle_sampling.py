"""Pins of the oracle's speculative sampling (CPU only).

The rejection rule (Section 3.1; Leviathan et al., Chen et al.) must leave the
target distribution unchanged.  Checked three ways:
  * the rule's exact output law, from its decision thresholds, equals p (closed form);
  * the oracle's rule, driven by random draws, reproduces p (chi-square), and a
    deliberately broken rule ("accept every draft") is rejected by the same test;
  * full speculative sampling sessions on a 64-token vocabulary produce the same
    token distribution as the exact autoregressive target law (chi-square).
"""
import numpy as np
import pytest
from scipy.stats import chi2 as chi2_dist

from wf_fixtures import VOCAB64, make_weights, make_memory, make_prefix
from oracle import OracleOpts, Target, Drafter, Session
import oracle.decode as odec
from oracle.accept import rejection_accept, softmax32

ALPHA = 1e-3


def chi2_pvalue(counts, expected):
    counts = np.asarray(counts, float)
    expected = np.asarray(expected, float)
    order = np.argsort(expected)
    c, e = counts[order], expected[order]
    # merge the smallest cells until each merged cell expects >= 5
    merged_c, merged_e, acc_c, acc_e = [], [], 0.0, 0.0
    for ci, ei in zip(c, e):
        acc_c += ci
        acc_e += ei
        if acc_e >= 5:
            merged_c.append(acc_c)
            merged_e.append(acc_e)
            acc_c = acc_e = 0.0
    if acc_e > 0 and merged_e:
        merged_c[-1] += acc_c
        merged_e[-1] += acc_e
    mc, me = np.array(merged_c), np.array(merged_e)
    stat = ((mc - me) ** 2 / me).sum()
    return chi2_dist.sf(stat, len(mc) - 1)


def _rule_law(p, q):
    """Exact law of the first emitted token under the rule: accept c~q w.p. min(1, p_c/q_c),
    else draw from (p-q)_+ normalised."""
    acc = np.minimum(p, q)
    rej = 1.0 - acc.sum()
    res = np.maximum(p - q, 0.0)
    return acc + (rej * res / res.sum() if res.sum() > 0 else 0.0)


def test_rule_closed_form_equals_p():
    rng = np.random.default_rng(0)
    for _ in range(50):
        V = int(rng.integers(2, 40))
        p = rng.dirichlet(np.ones(V) * rng.uniform(0.1, 3))
        q = rng.dirichlet(np.ones(V) * rng.uniform(0.1, 3))
        np.testing.assert_allclose(_rule_law(p, q), p, atol=1e-14)


def _sample_first_tokens(rule, n, V, rng, T=1.0):
    lp = rng.standard_normal(V).astype(np.float32) * 1.5
    lq = rng.standard_normal(V).astype(np.float32) * 1.5
    inv_t = np.float32(1.0 / T)
    p = softmax32(lp[None], inv_t)
    q = softmax32(lq[None], inv_t)
    out = np.zeros(V, int)
    for _ in range(n):
        gq = -np.log(-np.log(rng.uniform(size=V))).astype(np.float32)
        c = int(np.argmax(lq * inv_t + gq))
        g_res = -np.log(-np.log(rng.uniform(size=(1, V)))).astype(np.float32)
        g_bon = -np.log(-np.log(rng.uniform(size=V))).astype(np.float32)
        u = rng.uniform(size=1).astype(np.float32)
        a, toks, _ = rule(np.array([c]), q, np.concatenate([p, p]), u, g_res,
                          np.stack([lp, lp]), inv_t, g_bon, -1)
        out[toks[0]] += 1
    return out, p[0].astype(np.float64)


def test_rule_preserves_target_distribution():
    rng = np.random.default_rng(1)
    counts, p = _sample_first_tokens(rejection_accept, 20000, 12, rng)
    assert chi2_pvalue(counts, p * counts.sum()) > ALPHA


def _accept_all(drafts, q, p, u_acc, g_res, logits_p, inv_t, g_bon, eos):
    """A deliberately wrong rule: every draft is accepted (power control)."""
    k = len(drafts)
    tok = int(np.argmax(logits_p[k] * inv_t + g_bon))
    return k, [int(t) for t in drafts] + [tok], False


def test_power_control_accept_all_is_rejected():
    rng = np.random.default_rng(1)
    counts, p = _sample_first_tokens(_accept_all, 20000, 12, rng)
    assert chi2_pvalue(counts, p * counts.sum()) < ALPHA


@pytest.fixture(scope="module")
def v64():
    cfg = VOCAB64
    W = make_weights(cfg, seed_target=11, seed_drafter=12, std=0.25)
    opts = OracleOpts(dtype=np.float32)
    T, D = Target(cfg, W.values, opts), Drafter(cfg, W.values, opts)
    mem = make_memory(cfg, 0)
    prompt = make_prefix(cfg, 0, 6)
    return cfg, W, T, D, mem, prompt


def _exact_next(cfg, W, mem, seq, temperature):
    """Exact target law of the next token after ``seq`` (fp64 oracle)."""
    T64 = Target(cfg, W.values, OracleOpts(dtype=np.float64))
    logits, _ = T64.forward(T64.new_cache(), seq, 0, T64.cross_kv(mem))
    z = logits[-1].astype(np.float64) / temperature
    e = np.exp(z - z.max())
    return e / e.sum()


def _run_sessions(v64, temperature, n, rule=None, monkeypatch=None):
    cfg, W, T, D, mem, prompt = v64
    if rule is not None:
        monkeypatch.setattr(odec, "rejection_accept", rule)
    firsts, seconds = [], []
    for i in range(n):
        s = Session(T, D, mem, prompt, max_new=4, temperature=temperature, seed=1000 + i)
        s.step()
        firsts.append(s.out[0])
        seconds.append(s.out[1])
    return np.array(firsts), np.array(seconds)


@pytest.mark.parametrize("temperature", [0.7, 1.0])
def test_spec_sampling_matches_target_law(v64, temperature):
    cfg, W, T, D, mem, prompt = v64
    n = 1500
    firsts, seconds = _run_sessions(v64, temperature, n)
    # first token: prefill sample from p(. | prompt)
    p1 = _exact_next(cfg, W, mem, list(prompt), temperature)
    assert chi2_pvalue(np.bincount(firsts, minlength=64), p1 * n) > ALPHA
    # second token: first token of the speculative rule, conditional on the first
    counts, expected = [], []
    for t1 in np.unique(firsts):
        sel = seconds[firsts == t1]
        p2 = _exact_next(cfg, W, mem, list(prompt) + [int(t1)], temperature)
        counts.append(np.bincount(sel, minlength=64))
        expected.append(p2 * len(sel))
    assert chi2_pvalue(np.concatenate(counts), np.concatenate(expected)) > ALPHA


def test_spec_sampling_power_control(v64, monkeypatch):
    cfg, W, T, D, mem, prompt = v64
    n = 1500
    firsts, seconds = _run_sessions(v64, 1.0, n, rule=_accept_all, monkeypatch=monkeypatch)
    counts, expected = [], []
    for t1 in np.unique(firsts):
        sel = seconds[firsts == t1]
        p2 = _exact_next(cfg, W, mem, list(prompt) + [int(t1)], 1.0)
        counts.append(np.bincount(sel, minlength=64))
        expected.append(p2 * len(sel))
    assert chi2_pvalue(np.concatenate(counts), np.concatenate(expected)) < ALPHA
