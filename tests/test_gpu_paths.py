"""Call sequences, status word and the timed path of the HIP library (through the
C ABI) against the oracle.

  * verify calls with no draft call between them, then a draft: the drafter
    history must hold every verified position (Appendix A.2);
  * the sticky status word: non-finite logits and a refused position;
  * WF_ESTATE for calls on a slot that was never prefilled;
  * the graph-replayed wf_step with planted drafts at Whisper-large-v3 shapes,
    batch 1 (the step the benchmark times), compared with the oracle on every
    step: draft and target logits, drafted tokens, emitted tokens, accepted
    counts and the done flag;
  * verification budgets k_max below K (micro shapes, and the graph-replayed step
    at large-v3 shapes);
  * a verify pass reaching the last context position at large-v3 shapes;
  * GPU speculative greedy decoding equals GPU plain greedy decoding over 200
    tokens at large-v3 shapes (Section 3.1: speculation keeps greedy's output).

Bar: logits within 2e-2 of the fp32 oracle (bf16 storage), tokens identical
wherever the deciding row's top-2 margin exceeds that tolerance.
"""
import numpy as np
import pytest
import torch

from wf_fixtures import MICRO, LARGE_V3, make_weights, make_memory, make_prefix, make_prefix_lengths, plant_drafts
from oracle import OracleOpts, Target, plain_greedy

pytestmark = pytest.mark.gpu

TOL_F32 = 1e-3
TOL_BF16 = 2e-2
MICRO_BF16 = MICRO.with_(name="micro-bf16", dtype="bf16", n_vocab=501, n_frames=45)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture
def side_stream():
    """Graph capture and replay need a stream other than the null stream; the
    whole test (weights, encode, prefill, steps) runs on it."""
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        yield s
    torch.cuda.synchronize()


def _plan(ref, emitted, K, r, V, rng):
    cont = (list(ref) + [0] * (K + 1))[emitted:emitted + K]
    return plant_drafts(cont, r, V, rng)


@pytest.mark.parametrize("cfg,tol", [(MICRO, TOL_F32), (MICRO_BF16, 2e-3)], ids=["f32", "bf16"])
def test_verify_calls_without_draft_keep_history(cfg, tol):
    """Several wf_verify_accept calls (plain, then planted candidates) with no
    wf_draft between them, then drafts: the draft logits match the oracle, whose
    history is written by every verify."""
    from lockstep import Lockstep
    W = make_weights(cfg)
    prompts = [make_prefix(cfg, 0, 9), make_prefix(cfg, 1, 14)]
    ls = Lockstep(cfg, W, prompts, [40, 40], tol)
    T = Target(cfg, W.values, OracleOpts(dtype=np.float32, kv_bf16=cfg.dtype == "bf16"))
    refs = [plain_greedy(T, make_memory(cfg, i), prompts[i], 40) for i in range(2)]
    rng = np.random.default_rng(11)
    for _ in range(3):
        ls.verify_only(k_max=0)
    ov = np.stack([_plan(refs[i], ls.sess[i].emitted, cfg.block_k, 5, cfg.n_vocab, rng) for i in range(2)])
    ls.verify_only(k_max=8, override=ov)
    ls.verify_only(k_max=0)
    for _ in range(3):
        ls.step()
    print(f"verify-verify-draft {cfg.name}: max |dlogit| draft {ls.max_dlogit:.2e} target {ls.max_tlogit:.2e}, "
          f"near ties {ls.near_ties}")
    assert all(ls.live), ls.near_ties
    ls.close()


def test_status_nonfinite_logits():
    """A NaN in the final LayerNorm gain makes every target logit NaN: the verify
    sets WF_STATUS_NONFINITE_LOGITS, and reading the word clears it."""
    from lockstep import build_engine
    from paper_2609_32869_amd.binding import WF_STATUS_NONFINITE_LOGITS
    cfg = MICRO
    W = make_weights(cfg)
    W.values["ln_f.g"][3] = np.nan
    eng = build_engine(cfg, W, 1)
    from paper_2609_32869_amd import to_device_storage
    eng.encode_memory_set(0, to_device_storage(make_memory(cfg, 0), cfg.dtype)[None])
    eng.prefill(0, torch.from_numpy(make_prefix(cfg, 0, 6)[None].copy()).cuda(), [6], [20])
    assert eng.status() & WF_STATUS_NONFINITE_LOGITS  # the prefill's head already saw them
    assert eng.status() == 0
    eng.verify_accept(0, torch.zeros((1, cfg.block_k), dtype=torch.int32, device="cuda"), 0)
    assert eng.status() & WF_STATUS_NONFINITE_LOGITS
    eng.close()


def test_status_position_overflow_on_inconsistent_state():
    """A live, unfinished slot whose cache length is n_ctx (a state the acceptance
    never produces; planted through the state view) is refused: nothing is
    emitted, the slot reports done and the status word carries the overflow bit."""
    from lockstep import build_engine
    from paper_2609_32869_amd import to_device_storage
    from paper_2609_32869_amd.binding import WF_STATUS_POSITION_OVERFLOW
    cfg = MICRO
    W = make_weights(cfg)
    eng = build_engine(cfg, W, 2)
    mem = torch.stack([to_device_storage(make_memory(cfg, s), cfg.dtype) for s in range(2)])
    eng.encode_memory_set(0, mem)
    toks = torch.from_numpy(np.stack([make_prefix(cfg, s, 6) for s in range(2)])).cuda()
    eng.prefill(0, toks, [6, 6], [30, 30])
    assert eng.status() == 0
    st = eng.state()
    st[1, 0] = cfg.n_ctx        # L of slot 1 at the context end, slot still live and unfinished
    st[1, 4] = 0
    torch.cuda.synchronize()
    out, n_out, n_acc, done = eng.verify_accept(0, torch.zeros((2, cfg.block_k), dtype=torch.int32, device="cuda"), 0)
    torch.cuda.synchronize()
    assert n_out.tolist() == [1, 0] and done.tolist()[1] == 1
    assert eng.status() == WF_STATUS_POSITION_OVERFLOW
    eng.close()


def test_calls_before_prefill_are_refused():
    from lockstep import build_engine
    from paper_2609_32869_amd.binding import WfError
    cfg = MICRO
    eng = build_engine(cfg, make_weights(cfg), 2)
    for call in (lambda: eng.draft(0, 1),
                 lambda: eng.verify_accept(0, torch.zeros((1, cfg.block_k), dtype=torch.int32, device="cuda")),
                 lambda: eng.step(0, 2, use_graph=True)):
        with pytest.raises(WfError, match=r"\(-2\)"):
            call()
    eng.close()


@pytest.mark.timeout(900)
def test_large_v3_b1_graph_step_planted_matches_oracle(side_stream):
    """The benchmark's timed path: wf_step replayed from a captured HIP graph with
    planted drafts (first-rejection index r ~ U{0..8}, r = 8 every fifth step) at large-v3 shapes, batch 1,
    for 20 steps: every step's drafter logits and drafted tokens, target logits,
    emitted tokens, accepted count and done flag against the oracle.  This runs the
    batch-1 kernels at full size: 12-chunk cross-attention merge, persistent head,
    12-way split of the second MLP product."""
    from lockstep import Lockstep
    cfg = LARGE_V3
    W = make_weights(cfg)
    L = int(make_prefix_lengths(1, 20, 200)[0])
    prompt = make_prefix(cfg, 0, L)
    ls = Lockstep(cfg, W, [prompt], [cfg.n_ctx], TOL_BF16)
    ls.eng.set_debug(True)
    T = ls.T
    steps = 20
    ref = plain_greedy(T, make_memory(cfg, 0), prompt, (cfg.block_k + 1) * steps + 2)
    print(f"large-v3 graph step: prefix {L}, reference of {len(ref)} tokens", flush=True)
    rng = np.random.default_rng(400)
    outs = ls.eng._outs(1)
    ovr = torch.zeros((1, cfg.block_k), dtype=torch.int32, device="cuda")
    accepted = []
    for n in range(steps):
        s = ls.sess[0]
        # every fifth step plants a block the target accepts whole (bonus token)
        r = cfg.block_k if n % 5 == 4 else int(rng.integers(0, cfg.block_k + 1))
        ov = _plan(ref, s.emitted, cfg.block_k, r, cfg.n_vocab, rng)[None]
        _, _, n_acc, _ = ls.graph_step(ov, outs, ovr)
        if not ls.live[0]:
            break
        accepted.append(int(n_acc[0]))
        assert accepted[-1] == min(r, cfg.block_k), (n, r, accepted[-1])
    print(f"large-v3 graph step: accepted {accepted}; max |dlogit| draft {ls.max_dlogit:.2e} "
          f"target {ls.max_tlogit:.2e}; near ties {ls.near_ties}", flush=True)
    assert len(accepted) >= 16 and max(accepted) == cfg.block_k
    ls.close()


@pytest.mark.parametrize("cfg,tol", [(MICRO, TOL_F32), (MICRO_BF16, 2e-3)], ids=["f32", "bf16"])
def test_verification_budget_sweep(cfg, tol):
    """The verification budget (Appendix A.1; Table A5 varies it): k_max = 1, 2, 4,
    5 and 7 on three slots whose planted drafts are the target's own greedy
    continuation (so a step accepts min(k_max, remaining budget) candidates unless
    EOS ends it), and the same budgets with the first rejection at r ~ U{0..8};
    drafts, target logits, emitted tokens, accepted counts and done against the
    oracle every step."""
    from lockstep import Lockstep
    W = make_weights(cfg)
    prompts = [make_prefix(cfg, 0, 5), make_prefix(cfg, 1, 17), make_prefix(cfg, 2, 30)]
    max_new = [60, 25, 60]
    ls = Lockstep(cfg, W, prompts, max_new, tol)
    refs = [plain_greedy(ls.T, make_memory(cfg, i), prompts[i], max_new[i]) for i in range(3)]
    rng = np.random.default_rng(12)
    K = cfg.block_k
    for rep in range(2):
        for k_max in (1, 2, 4, 5, 7):
            ov = np.stack([_plan(refs[i], ls.sess[i].emitted, K, K if rep == 0 else int(rng.integers(0, K + 1)),
                                 cfg.n_vocab, rng) for i in range(3)])
            ls.step(k_max=k_max, override=ov)
    print(f"budget sweep {cfg.name}: accepted {ls.accepted}; max |dlogit| draft {ls.max_dlogit:.2e} "
          f"target {ls.max_tlogit:.2e}; near ties {ls.near_ties}")
    assert ls.steps == 10 and max(ls.accepted) == 7
    ls.close()


@pytest.mark.timeout(900)
def test_large_v3_b1_graph_step_budgets(side_stream):
    """The timed path at budgets below K (Table A5's knob) at large-v3 shapes,
    batch 1: graph-replayed wf_step with k_max = 1, 2, 4 and 7 and the whole
    greedy continuation planted, so each step accepts exactly k_max candidates;
    logits, tokens and accepted counts against the oracle."""
    from lockstep import Lockstep
    cfg = LARGE_V3
    W = make_weights(cfg)
    prompt = make_prefix(cfg, 0, 60)
    ls = Lockstep(cfg, W, [prompt], [cfg.n_ctx], TOL_BF16)
    ls.eng.set_debug(True)
    budgets = (1, 2, 4, 7, 4, 1)
    ref = plain_greedy(ls.T, make_memory(cfg, 0), prompt, sum(budgets) + len(budgets) + 2)
    rng = np.random.default_rng(13)
    outs = ls.eng._outs(1)
    ovr = torch.zeros((1, cfg.block_k), dtype=torch.int32, device="cuda")
    accepted = []
    for k_max in budgets:
        ov = _plan(ref, ls.sess[0].emitted, cfg.block_k, cfg.block_k, cfg.n_vocab, rng)[None]
        _, _, n_acc, _ = ls.graph_step(ov, outs, ovr, k_max=k_max)
        if not ls.live[0]:
            break
        accepted.append(int(n_acc[0]))
    print(f"large-v3 budgets {budgets}: accepted {accepted}; max |dlogit| draft {ls.max_dlogit:.2e} "
          f"target {ls.max_tlogit:.2e}; near ties {ls.near_ties}", flush=True)
    assert accepted == list(budgets[:len(accepted)]) and len(accepted) >= 4
    ls.close()


@pytest.mark.timeout(900)
def test_large_v3_b1_verify_reaches_last_context_position():
    """A 439-token prompt leaves k = 8: one step verifies positions 439..447 (the
    last of the 448), accepts all eight planted candidates (the target's own greedy
    continuation), emits nine tokens and finishes with L = 448."""
    from lockstep import Lockstep
    cfg = LARGE_V3
    W = make_weights(cfg)
    prompt = make_prefix(cfg, 0, 439)
    ls = Lockstep(cfg, W, [prompt], [cfg.n_ctx], TOL_BF16)
    ref = plain_greedy(ls.T, make_memory(cfg, 0), prompt, cfg.block_k + 2)
    ov = np.array(ref[1:cfg.block_k + 1], np.int32)[None]
    out, n_out, n_acc, done = ls.step(override=ov)
    st = ls.eng.state()[0].cpu().numpy()
    print(f"last position: n_acc {n_acc[0]} n_out {n_out[0]} L {st[0]} done {done[0]}; near ties {ls.near_ties}; "
          f"max |dlogit| target {ls.max_tlogit:.2e}")
    assert ls.live[0], ls.near_ties
    assert (n_acc[0], n_out[0], st[0], done[0]) == (8, 9, cfg.n_ctx, 1)
    assert list(out[0, :9]) == ref[1:10]
    ls.close()


@pytest.mark.timeout(900)
def test_large_v3_b1_speculative_equals_plain_greedy_on_gpu(side_stream):
    """GPU speculative greedy decoding (graph-replayed wf_step, planted drafts from
    the plain run's own tokens, r ~ U{0..8}) emits the same 200 tokens as GPU plain
    greedy decoding (k_max = 0), and a second plain run repeats the first.  The
    batch-1 residual stream receives the attention output products through fp32
    atomic adds whose order varies, so logits may differ between runs in the last
    bits; token sequences are compared up to the first row whose top-2 margin is
    below 2e-2 (reported), and must agree up to there."""
    from lockstep import build_engine
    from paper_2609_32869_amd import to_device_storage
    cfg = LARGE_V3
    W = make_weights(cfg)
    eng = build_engine(cfg, W, 1)
    eng.set_debug(True)
    eng.encode_memory_set(0, to_device_storage(make_memory(cfg, 0), cfg.dtype)[None])
    P, N = 40, 200
    toks = torch.from_numpy(make_prefix(cfg, 0, P)[None].copy()).cuda()
    K = cfg.block_k
    outs = eng._outs(1)
    zero = torch.zeros((1, K), dtype=torch.int32, device="cuda")

    def plain():
        first = eng.prefill(0, toks, [P], [N])
        seq = [first[0:1].clone()]
        marg, top = [], []
        for _ in range(N - 1):
            eng.step(0, 1, 0, draft_override=zero, outs=outs, use_graph=True)
            seq.append(outs[0][0, 0:1].clone())
            v = torch.topk(eng.target_logits()[0, 0], 2)
            marg.append(v.values[0] - v.values[1])
            top.append(eng.target_logits()[0, 0].clone())
        torch.cuda.synchronize()
        return (torch.cat(seq).cpu().numpy(), np.array([0.0] + torch.stack(marg).cpu().tolist()),
                torch.stack(top))

    a, marg_a, la = plain()
    b, marg_b, lb = plain()
    run_diff = float((la - lb).abs().max())
    # speculative run with planted drafts from the plain tokens
    rng = np.random.default_rng(7)
    eng.prefill(0, toks, [P], [N])
    ovr = torch.zeros((1, K), dtype=torch.int32, device="cuda")
    spec = [int(a[0])]
    steps = 0
    while len(spec) < N:
        r = int(rng.integers(0, K + 1))
        cont = (list(a[len(spec):len(spec) + K]) + [0] * K)[:K]
        ovr.copy_(torch.from_numpy(plant_drafts(cont, r, cfg.n_vocab, rng)[None].copy()))
        eng.step(0, 1, K, draft_override=ovr, outs=outs, use_graph=True)
        torch.cuda.synchronize()
        n = int(outs[1][0])
        if n == 0:
            break
        spec += [int(x) for x in outs[0][0, :n].cpu().numpy()]
        steps += 1
    spec = np.array(spec[:N])

    def first_diff(x, y):
        d = np.nonzero(x[:len(y)] != y[:len(x)])[0]
        return int(d[0]) if len(d) else None

    near = [(i, float(marg_a[i])) for i in range(1, N) if marg_a[i] <= TOL_BF16]
    print(f"spec == plain: {steps} spec steps for {len(spec)} tokens; run-to-run max |dlogit| {run_diff:.2e}; "
          f"rows with margin <= 2e-2: {near[:5]}", flush=True)
    for x, y, what in ((a, b, "plain run 2"), (a, spec, "speculative")):
        i = first_diff(x, y)
        if i is not None:
            assert marg_a[i] <= TOL_BF16, f"{what} differs from plain greedy at token {i} (margin {marg_a[i]:.3e})"
            print(f"{what}: first difference at token {i}, a near tie (margin {marg_a[i]:.3e})")
    assert len(a) == N and len(spec) == N
    eng.close()
