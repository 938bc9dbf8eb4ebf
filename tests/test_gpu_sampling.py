"""Sampling on the GPU (rejection rule, Gumbel-max draws, Philox4x64-10).

* the device generator reproduces the host build bit-exactly (the host build is
  pinned to the oracle on the CPU);
* step by step against the oracle on the fp32 micro configuration: drafted
  tokens, accepted counts and emitted tokens identical, except where the oracle's
  own decision is within rounding of a tie (Gumbel top-2 gap < 1e-4, or
  |u q - p| < 1e-5 p), which is reported and ends the comparison of that slot;
* the emitted-token law on the 64-token vocabulary equals the exact target law
  (chi-square, alpha = 1e-3, about 2e5 samples per temperature), while the
  drafter's own proposals fail the same test (power control).
"""
import numpy as np
import pytest
import torch

from wf_fixtures import MICRO, VOCAB64, PURPOSE, make_weights, make_memory, make_prefix
from oracle import OracleOpts, Target, Drafter, Session
from oracle.accept import softmax32
from oracle.philox import uniforms, gumbel
from paper_2609_32869_amd import rng_words_host, rng_words_device, to_device_storage
from lockstep import build_engine
from test_oracle_sampling import chi2_pvalue, ALPHA

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def test_device_generator_equals_host():
    for seed, pur, slot, step, pos, n in [(500, "DRAFT", 0, 0, 1, 512), (7, "RES", 31, 9, 8, 1000),
                                         ((1 << 64) - 1, "BON", 2, 3, 0, 65), (500, "ACC", 5, 2, 0, 8)]:
        d = rng_words_device(seed, PURPOSE[pur], slot, step, pos, n).cpu().numpy().view(np.uint64)
        h = rng_words_host(seed, PURPOSE[pur], slot, step, pos, n)
        np.testing.assert_array_equal(d, h)


def _gap(scores):
    top = np.partition(scores.astype(np.float64), -2)[-2:]
    return float(top[1] - top[0])


def _sampling_lockstep(cfg, temperature, suppress=None, steps=10, plant_every=3, prompts=None, check=None,
                       opts=None, gap_tol=1e-4, margin_tol=1e-5):
    """Sampling decisions of the GPU vs the oracle for the slots in ``check``.  A
    disagreement is accepted only where the oracle's own decision is within
    gap_tol (Gumbel top-2 gap) or margin_tol (|u q - p| / p) of a tie."""
    W = make_weights(cfg)
    if prompts is None:
        prompts = [make_prefix(cfg, 0, 5), make_prefix(cfg, 1, 12)]
    n = len(prompts)
    max_new = [min(40, cfg.n_ctx)] * n
    check = set(range(n) if check is None else check)
    eng = build_engine(cfg, W, n)
    sup_dev = None
    if suppress is not None:
        sup_dev = torch.from_numpy(suppress.astype(np.uint8)).cuda()
    eng.set_sampling(temperature, seed=500, suppress=sup_dev)
    if opts is None:
        opts = OracleOpts(dtype=np.float32, exact=True)
    T, D = Target(cfg, W.values, opts), Drafter(cfg, W.values, opts)
    mems = [make_memory(cfg, s) for s in range(n)]
    eng.encode_memory_set(0, torch.stack([to_device_storage(m, cfg.dtype) for m in mems]))
    toks = np.zeros((n, max(len(p) for p in prompts)), np.int32)
    for i, p in enumerate(prompts):
        toks[i, :len(p)] = p
    sup_idx = np.nonzero(suppress)[0] if suppress is not None else None
    first = eng.prefill(0, torch.from_numpy(toks).cuda(), [len(p) for p in prompts], max_new).cpu().numpy()
    sess = [Session(T, D, mems[i], prompts[i], max_new[i], slot=i, temperature=temperature, seed=500,
                    suppress=sup_idx) if i in check else None for i in range(n)]
    live = [i in check for i in range(n)]
    ties = []
    for i, s in enumerate(sess):
        if s is None:
            continue
        if first[i] != s.out[0]:
            g = gumbel(uniforms(500, PURPOSE["PREFILL"], i, 0, 0, cfg.n_vocab))
            gap = _gap(s.last_logits[-1].astype(np.float32) * s.inv_t + g)
            assert gap < gap_tol, f"slot {i}: first token {first[i]} vs {s.out[0]} (gap {gap})"
            ties.append((i, "prefill", gap))
            live[i] = False
    rng = np.random.default_rng(3)
    decisions = 0
    for step in range(steps):
        drafts = eng.draft(0, n).cpu().numpy()
        used = drafts.copy()
        if step % plant_every == 1:
            used = rng.integers(0, cfg.n_vocab, size=drafts.shape).astype(np.int32)
            if sup_idx is not None:
                used[np.isin(used, sup_idx)] = int(np.setdiff1d(np.arange(cfg.n_vocab), sup_idx)[0])
        out, n_out, n_acc, done = (t.cpu().numpy() for t in eng.verify_accept(0, torch.from_numpy(used).cuda(), 8))
        for i, s in enumerate(sess):
            if not live[i] or s.done:
                continue
            otoks, lq = s.draft()
            if not np.array_equal(otoks, drafts[i]):
                j = int(np.nonzero(otoks != drafts[i])[0][0])
                g = gumbel(uniforms(500, PURPOSE["DRAFT"], i, s.step_no, j + 1, cfg.n_vocab))
                gap = _gap(lq[j].astype(np.float32) * s.inv_t + g)
                assert gap < gap_tol, f"slot {i} step {step}: draft {drafts[i]} vs {otoks} (gap {gap})"
                ties.append((i, f"draft {step}", gap))
                live[i] = False
                continue
            rec = s.verify_accept(used[i], 8, draft_logits=lq)
            gpu = list(out[i, :n_out[i]])
            decisions += rec["k"] + 1
            if gpu != rec["tokens"] or n_acc[i] != rec["a"]:
                margins = []
                # acceptance thresholds of this step, from the oracle's own quantities
                k = rec["k"]
                q = softmax32(lq[:k], s.inv_t) if k else None
                p = softmax32(s.last_logits, s.inv_t)
                u = uniforms(500, PURPOSE["ACC"], i, s.step_no - 1, 0, max(k, 1))
                for j in range(k):
                    c = int(used[i, j])
                    margins.append(abs(float(u[j]) * float(q[j, c]) - float(p[j, c])) / max(float(p[j, c]), 1e-30))
                assert margins and min(margins) < margin_tol, \
                    f"slot {i} step {step}: GPU {gpu} a={n_acc[i]} vs oracle {rec['tokens']} a={rec['a']}"
                ties.append((i, f"accept {step}", min(margins)))
                live[i] = False
                continue
            if sup_idx is not None:
                assert not np.isin(gpu, sup_idx).any()
            assert bool(done[i]) == s.done
    eng.close()
    return decisions, ties


@pytest.mark.parametrize("temperature", [0.75, 1.0])
def test_micro_sampling_lockstep(temperature):
    decisions, ties = _sampling_lockstep(MICRO, temperature)
    print(f"T={temperature}: {decisions} verified rows compared, near ties {ties}")
    assert decisions > 50


def test_micro_sampling_with_suppression():
    sup = np.zeros(MICRO.n_vocab, bool)
    sup[:40] = True
    sup[MICRO.eos_id] = False
    decisions, ties = _sampling_lockstep(MICRO, 1.0, suppress=sup, steps=6)
    print(f"suppressed: {decisions} verified rows compared, near ties {ties}")
    assert decisions > 20


@pytest.mark.parametrize("temperature", [0.75, 1.0])
def test_micro_bf16_b1_sampling(temperature):
    """bf16 storage at batch 1 (ragged vocabulary 501, 45 frames), sampling: the
    batch-1 kernels (folded LayerNorms, fused attention output products, split-K
    second MLP product, persistent head with the Gumbel scores and softmax
    normalisers) against the oracle; decisions compared where the oracle's margins
    exceed the bf16 bar."""
    cfg = MICRO.with_(name="micro-bf16", dtype="bf16", n_vocab=501, n_frames=45)
    opts = OracleOpts(dtype=np.float32, kv_bf16=True)
    decisions, ties = _sampling_lockstep(cfg, temperature, prompts=[make_prefix(cfg, 0, 11)], opts=opts,
                                         gap_tol=2e-3, margin_tol=2e-3)
    print(f"micro-bf16 b1 T={temperature}: {decisions} verified rows compared, near ties {ties}")
    assert decisions > 20


# ---------------------------------------------------------------- distribution on V = 64
def _exact_next(cfg, W, mem, seq, temperature):
    T64 = Target(cfg, W.values, OracleOpts(dtype=np.float64))
    logits, _ = T64.forward(T64.new_cache(), seq, 0, T64.cross_kv(mem))
    z = logits[-1].astype(np.float64) / temperature
    e = np.exp(z - z.max())
    return e / e.sum()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("temperature,k_max", [(0.75, 8), (1.0, 8), (1.0, 0)])
def test_v64_emitted_law_equals_target(temperature, k_max):
    cfg = VOCAB64
    W = make_weights(cfg, seed_target=11, seed_drafter=12, std=0.25)
    B, runs = 512, 400
    mem = make_memory(cfg, 0)
    prompt = make_prefix(cfg, 0, 6)
    eng = build_engine(cfg, W, B)
    eng.encode_memory_set(0, torch.stack([to_device_storage(mem, cfg.dtype)] * B))
    toks = torch.from_numpy(np.tile(np.asarray(prompt, np.int32), (B, 1))).cuda()
    firsts, seconds, drafted = [], [], []
    for r in range(runs):
        eng.set_sampling(temperature, seed=1000 + r)
        first = eng.prefill(0, toks, [len(prompt)] * B, [8] * B)
        d = eng.draft(0, B)
        out, n_out, _, _ = eng.verify_accept(0, d, k_max)
        firsts.append(first.cpu().numpy())
        seconds.append(out[:, 0].cpu().numpy())
        drafted.append(d[:, 0].cpu().numpy())
    eng.close()
    firsts, seconds, drafted = (np.concatenate(x) for x in (firsts, seconds, drafted))
    n = len(firsts)
    p1 = _exact_next(cfg, W, mem, list(prompt), temperature)
    pv1 = chi2_pvalue(np.bincount(firsts, minlength=64), p1 * n)
    counts, expected, dcounts = [], [], []
    for t1 in np.unique(firsts):
        sel = firsts == t1
        p2 = _exact_next(cfg, W, mem, list(prompt) + [int(t1)], temperature)
        counts.append(np.bincount(seconds[sel], minlength=64))
        dcounts.append(np.bincount(drafted[sel], minlength=64))
        expected.append(p2 * sel.sum())
    pv2 = chi2_pvalue(np.concatenate(counts), np.concatenate(expected))
    pv_power = chi2_pvalue(np.concatenate(dcounts), np.concatenate(expected))
    print(f"T={temperature} k_max={k_max}: n={n} p(first)={pv1:.3g} p(second)={pv2:.3g} power control p={pv_power:.3g}")
    assert pv1 > ALPHA and pv2 > ALPHA
    assert pv_power < ALPHA


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("temperature", [0.7, 1.0])
def test_large_v3_b8_sampling(temperature):
    """Large-v3 shapes, 8 slots, prefixes uniform in [4, 440]; the oracle follows two
    slots; decisions are compared where the oracle's margins exceed the bf16 bar."""
    from wf_fixtures import LARGE_V3, make_prefix_lengths
    cfg = LARGE_V3
    lens = [int(x) for x in make_prefix_lengths(8, 4, 440, seed=300)]
    prompts = [make_prefix(cfg, s, lens[s]) for s in range(8)]
    opts = OracleOpts(dtype=np.float32, kv_bf16=True, exact=False)
    decisions, ties = _sampling_lockstep(cfg, temperature, steps=3, prompts=prompts, check=[0, 5], opts=opts,
                                         gap_tol=2e-2, margin_tol=2e-2)
    print(f"large b8 T={temperature}: {decisions} verified rows compared, near ties {ties}", flush=True)
    assert decisions > 0
