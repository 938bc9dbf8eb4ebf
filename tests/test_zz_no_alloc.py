"""wf_step_noalloc (the step with its per-call buffers in the library's static
scratch) against wf_step on the same inputs, through the C ABI.

Two engines with identical weights, memories and prompts run the same calls:
one through wf_step (eager), the other through wf_step_noalloc.  Each case makes
two calls in a row, the second with a smaller input (fewer slots, or fewer
verified candidates), so the second call runs over scratch that still holds
the first call's contents.  Bar: emitted tokens, accepted counts, done flags and
per-slot state identical (fp32 storage); with bf16 storage at one slot the
residual stream receives fp32 atomic adds in varying order, so tokens are
compared with the margin rule of the parity tests (a difference is allowed only
at a row whose top-2 margin is at most the logit tolerance).
"""
import numpy as np
import pytest
import torch

from wf_fixtures import MICRO, make_weights, make_memory, make_prefix
from oracle import OracleOpts, Target, plain_greedy

pytestmark = pytest.mark.gpu

MICRO_BF16 = MICRO.with_(name="micro-bf16", dtype="bf16", n_vocab=501, n_frames=45)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _engine(cfg, W, prompts, max_new):
    from lockstep import build_engine
    from paper_2609_32869_amd import to_device_storage
    n = len(prompts)
    eng = build_engine(cfg, W, n)
    mem = torch.stack([to_device_storage(make_memory(cfg, s), cfg.dtype) for s in range(n)])
    eng.encode_memory_set(0, mem)
    pmax = max(len(p) for p in prompts)
    toks = np.zeros((n, pmax), np.int32)
    for i, p in enumerate(prompts):
        toks[i, :len(p)] = p
    eng.prefill(0, torch.from_numpy(toks).cuda(), [len(p) for p in prompts], max_new)
    return eng


def _planted(cfg, refs, emitted, rng):
    K = cfg.block_k
    ov = np.zeros((len(refs), K), np.int32)
    for i, ref in enumerate(refs):
        cont = (list(ref) + [0] * (K + 1))[emitted[i]:emitted[i] + K]
        r = int(rng.integers(0, K + 1))
        ov[i] = cont
        if r < K:
            ov[i, r] = (ov[i, r] + 1) % cfg.n_vocab
    return ov


def _pair_run(cfg, calls, tol):
    """calls: list of (n slots, k_max); returns the number of calls compared."""
    W = make_weights(cfg)
    nmax = max(n for n, _ in calls)
    prompts = [make_prefix(cfg, s, 5 + 7 * s) for s in range(nmax)]
    max_new = [40] * nmax
    a = _engine(cfg, W, prompts, max_new)
    b = _engine(cfg, W, prompts, max_new)
    a.set_debug(True)
    T = Target(cfg, W.values, OracleOpts(dtype=np.float32, kv_bf16=cfg.dtype == "bf16"))
    refs = [plain_greedy(T, make_memory(cfg, s), prompts[s], 40) for s in range(nmax)]
    rng = np.random.default_rng(3)
    exact = cfg.dtype != "bf16"
    for n, k_max in calls:
        emitted = a.state()[:n, 2].cpu().numpy()
        ov = torch.from_numpy(_planted(cfg, refs[:n], emitted, rng)).cuda()
        ra = [t.cpu().numpy() for t in a.step(0, n, k_max, draft_override=ov)]
        rb = [t.cpu().numpy() for t in b.step_noalloc(0, n, k_max, draft_override=ov)]
        torch.cuda.synchronize()
        sa, sb = a.state()[:n].cpu().numpy(), b.state()[:n].cpu().numpy()
        if exact:
            for x, y in zip(ra, rb):
                np.testing.assert_array_equal(x, y)
            np.testing.assert_array_equal(sa, sb)
        else:
            logits = a.target_logits()[:n].cpu().numpy()
            for i in range(n):
                if all(np.array_equal(x[i], y[i]) for x, y in zip(ra, rb)):
                    assert np.array_equal(sa[i], sb[i])
                    continue
                k = int(ra[2][i])
                top = np.sort(logits[i, k].astype(np.float64))[-2:]
                assert top[1] - top[0] <= tol, f"slot {i}: noalloc step differs at a clear row"
    a.close()
    b.close()
    return len(calls)


def test_noalloc_equals_step_several_slots_f32():
    # three slots, then two: the second call runs over the first call's scratch
    assert _pair_run(MICRO, [(3, 8), (2, 8)], 0.0) == 2


def test_noalloc_equals_step_one_slot_bf16():
    # the batch-1 kernels (three-term operands, fused output products); the second
    # call verifies fewer candidates
    assert _pair_run(MICRO_BF16, [(1, 8), (1, 3)], 2e-3) == 2


def test_noalloc_rejects_configuration_beyond_scratch():
    from lockstep import build_engine
    from paper_2609_32869_amd.binding import WfError
    cfg = MICRO.with_(name="micro-wide-vocab", n_vocab=120000)
    W = make_weights(cfg)
    eng = _engine(cfg, W, [make_prefix(cfg, s, 4) for s in range(2)], [8, 8])
    with pytest.raises(WfError, match=r"\(-3\).*static scratch"):
        eng.step_noalloc(0, 2)
    eng.close()
