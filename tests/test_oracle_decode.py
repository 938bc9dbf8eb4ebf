"""Pins of the oracle's decoding loop (CPU only): speculative greedy output equals
plain greedy decoding (Section 3.1 / Section 5.1), the worked example of Figure 1,
rollback (Appendix A.1), the budget and end-of-transcript rules."""
import json
import os

import numpy as np
import pytest

from wf_fixtures import MICRO, make_weights, make_memory, make_prefix, plant_drafts
from oracle import OracleOpts, Target, Drafter, Session, plain_greedy, brute_greedy, spec_greedy
from oracle.accept import greedy_accept, budget_k

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F32 = OracleOpts()


@pytest.fixture(scope="module")
def models(micro):
    cfg, W = micro
    return cfg, W, Target(cfg, W.values, F32), Drafter(cfg, W.values, F32)


def test_figure1_worked_example():
    ex = json.load(open(os.path.join(GOLDEN, "fig1_example.json")))
    ids = {w: i for i, w in enumerate(ex["vocab"])}
    drafts = [ids[w] for w in ex["drafts"]]
    # target argmax of the first rows as the figure gives them; later rows are irrelevant
    g = [ids[w] for w in ex["target_argmax_first_rows"]] + [ids["in"]] * 6
    a, toks, fin = greedy_accept(drafts, g, ids[ex["eos"]])
    exp = ex["expected"]
    assert a == exp["accepted"]
    assert toks == [ids[w] for w in exp["emitted"]]
    assert len(toks) == exp["tokens_advanced"] and not fin
    assert toks[-1] == ids[exp["next_anchor"]]
    # the anchor plus the accepted candidates enter the cache and history: 1 + a positions
    assert [ids[ex["anchor"]]] + drafts[:a] == [ids[w] for w in exp["history_extended_by"]]


def test_greedy_accept_edge_cases():
    eos = 9
    assert greedy_accept([], [4], eos) == (0, [4], False)                       # plain step
    assert greedy_accept([1, 2, 3], [1, 2, 3, 5], eos) == (3, [1, 2, 3, 5], False)  # bonus
    assert greedy_accept([7, 2, 3], [1, 2, 3, 5], eos) == (0, [1], False)          # first rejected
    assert greedy_accept([1, 9, 3], [1, 9, 3, 5], eos) == (2, [1, 9], True)        # accepted EOS, no bonus
    assert greedy_accept([1, 2], [1, 9, 4], eos) == (1, [1, 9], True)              # EOS as correction


def test_budget_rule():
    # R tokens left -> at most R-1 candidates; never a position >= n_ctx
    assert budget_k(8, 8, 64, 1, 448, 10) == 8
    assert budget_k(8, 8, 64, 60, 448, 10) == 3
    assert budget_k(8, 8, 64, 63, 448, 10) == 0
    assert budget_k(8, 8, 64, 64, 448, 10) == -1
    assert budget_k(8, 8, 1000, 1, 448, 440) == 7
    assert budget_k(8, 8, 1000, 1, 448, 447) == 0
    assert budget_k(8, 8, 1000, 1, 448, 448) == -1
    assert budget_k(8, 3, 1000, 1, 448, 10) == 3


@pytest.mark.parametrize("slot,plen", [(0, 5), (1, 17), (2, 30)])
def test_spec_equals_plain_equals_brute(models, slot, plen):
    cfg, W, T, D = models
    mem = make_memory(cfg, slot)
    prompt = make_prefix(cfg, slot, plen)
    n = 24
    pg = plain_greedy(T, mem, prompt, n)
    assert pg == brute_greedy(T, mem, prompt, n)
    sg, _ = spec_greedy(T, D, mem, prompt, n)
    assert sg == pg


def _continuation(T, mem, prompt, n):
    return plain_greedy(T, mem, prompt, n)


@pytest.mark.parametrize("seed", [0, 1])
def test_planted_drafts_accept_exactly_r(models, seed):
    cfg, W, T, D = models
    mem = make_memory(cfg, 3)
    prompt = make_prefix(cfg, 3, 9)
    ref = _continuation(T, mem, prompt, 40)
    rng = np.random.default_rng(seed)
    planted_r = []

    def fn(s):
        e = s.emitted
        cont = (ref + [0] * 16)[e:e + cfg.block_k]
        r = int(rng.integers(0, cfg.block_k + 1))
        planted_r.append((r, s.budget(cfg.block_k)))
        return plant_drafts(cont, r, cfg.n_vocab, rng)

    out, s = spec_greedy(T, D, mem, prompt, 40, draft_fn=fn)
    assert out == ref
    for (r, k), rec in zip(planted_r, s.history):
        assert rec["k"] == k
        assert rec["a"] == min(r, k)
        assert len(rec["tokens"]) == rec["a"] + 1


@pytest.mark.parametrize("k_max", [0, 1, 3, 8])
def test_k_max_keeps_tokens(models, k_max):
    cfg, W, T, D = models
    mem = make_memory(cfg, 4)
    prompt = make_prefix(cfg, 4, 6)
    ref = plain_greedy(T, mem, prompt, 20)
    out, s = spec_greedy(T, D, mem, prompt, 20, k_max=k_max, draft_fn=lambda s: (ref + [0] * 9)[s.emitted:s.emitted + 8])
    assert out == ref
    assert all(h["k"] <= k_max for h in s.history)


def test_adversarial_drafts(models):
    cfg, W, T, D = models
    mem = make_memory(cfg, 5)
    prompt = make_prefix(cfg, 5, 7)
    ref = plain_greedy(T, mem, prompt, 25)
    for fn in (lambda s: [cfg.eos_id] * 8, lambda s: [s.anchor] * 8, lambda s: list(range(8))):
        out, _ = spec_greedy(T, D, mem, prompt, 25, draft_fn=fn)
        assert out == ref


@pytest.mark.parametrize("as_candidate", [True, False])
def test_planted_eos_ends_decoding(models, as_candidate):
    """Make the token greedy emits at step s the EOS id; decoding must end exactly there,
    whether EOS arrives as an accepted candidate (no bonus) or as the correction."""
    cfg, W, T, D = models
    mem = make_memory(cfg, 6)
    prompt = make_prefix(cfg, 6, 8)
    ref = plain_greedy(T, mem, prompt, 30)
    s_idx = 11
    # choose an id that first appears at position s_idx
    eos = ref[s_idx]
    first = ref.index(eos)
    cfg2 = cfg.with_(eos_id=eos)
    T2, D2 = Target(cfg2, W.values, F32), Drafter(cfg2, W.values, F32)
    ref2 = plain_greedy(T2, mem, prompt, 30)
    assert ref2 == ref[:first + 1]

    def fn(s):
        cont = (ref + [0] * 16)[s.emitted:s.emitted + 8]
        if not as_candidate:
            cont = [(c + 1) % cfg.n_vocab for c in cont]
        return cont

    out, s = spec_greedy(T2, D2, mem, prompt, 30, draft_fn=fn)
    assert out == ref2 and s.done


def test_rollback_cache_equals_teacher_forced_prefill(models):
    """After a speculative run the target cache and drafter history for positions < L equal
    a teacher-forced prefill over the prompt and all emitted tokens but the last."""
    cfg, W, T, D = models
    mem = make_memory(cfg, 7)
    prompt = make_prefix(cfg, 7, 10)
    ref = plain_greedy(T, mem, prompt, 30)
    rng = np.random.default_rng(3)
    fn = lambda s: plant_drafts((ref + [0] * 16)[s.emitted:s.emitted + 8], int(rng.integers(0, 9)), cfg.n_vocab, rng)
    s = Session(T, D, mem, prompt, 30)
    s.run(draft_fn=fn)
    seq = list(prompt) + s.out[:-1]
    assert s.L == len(seq)
    s2 = Session(T, D, mem, seq, 30)
    np.testing.assert_allclose(s.cache.K[:, :s.L], s2.cache.K[:, :s.L], atol=1e-5)
    np.testing.assert_allclose(s.cache.V[:, :s.L], s2.cache.V[:, :s.L], atol=1e-5)
    np.testing.assert_allclose(s.hcache.K[:, :s.L], s2.hcache.K[:, :s.L], atol=1e-5)
    np.testing.assert_allclose(s.hcache.V[:, :s.L], s2.hcache.V[:, :s.L], atol=1e-5)


def test_context_limit_never_exceeded(models):
    cfg, W, T, D = models
    mem = make_memory(cfg, 8)
    prompt = make_prefix(cfg, 8, cfg.n_ctx - 12)
    ref = plain_greedy(T, mem, prompt, 1000)
    assert len(prompt) + len(ref) - 1 == cfg.n_ctx  # stops when the anchor cannot be processed
    out, s = spec_greedy(T, D, mem, prompt, 1000, draft_fn=lambda s: (ref + [0] * 16)[s.emitted:s.emitted + 8])
    assert out == ref and s.L == cfg.n_ctx
    assert all(h["k"] <= cfg.n_ctx - 1 for h in s.history)
