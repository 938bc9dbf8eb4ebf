"""Drafter ablation variants on the HIP path (through the C ABI) against the oracle:
no direct audio, no target history, absolute positions instead of RoPE, and
five layers (Section 5.4 Table 3; Appendix Table A4).

Each variant runs the lockstep comparison of the parity tests: draft and target
logits within tolerance, drafted and emitted tokens, accepted counts and done
flags identical wherever the deciding row's top-2 margin exceeds the tolerance,
with natural and planted drafts; at fp32 storage with two slots, at bf16
storage with one slot (the batch-1 kernels), at bf16 storage with ten slots of
a wider micro model (the several-slot kernels), and at large-v3 shapes.
"""
import numpy as np
import pytest
import torch

from wf_fixtures import MICRO, LARGE_V3, make_weights, make_memory, make_prefix, make_prefix_lengths, plant_drafts
from oracle import OracleOpts, Target, plain_greedy

pytestmark = pytest.mark.gpu

VARIANTS = {
    "no-audio": dict(draft_audio=False),
    "no-history": dict(draft_history=False),
    "abs-pos": dict(draft_pos="abs"),
    "five-layers": dict(n_draft_layer=5),
}
MICRO_BF16 = MICRO.with_(name="micro-bf16", dtype="bf16", n_vocab=501, n_frames=45)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _planted(ls, refs, rng):
    K = ls.cfg.block_k
    ov = np.zeros((ls.n, K), np.int32)
    for i, s in enumerate(ls.sess):
        cont = (list(refs[i]) + [0] * (K + 1))[s.emitted:s.emitted + K]
        ov[i] = plant_drafts(cont, int(rng.integers(0, K + 1)), ls.cfg.n_vocab, rng)
    return ov


# d 1024 (16 heads) at 10 slots: 160 (head, slot) blocks, so the drafter attention
# takes its all-rows kernel (one block per (head, slot) for the nine block rows)
MICRO_WIDE = MICRO_BF16.with_(name="micro-wide", d_model=1024, n_head=16, d_ff=2560)


@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("base,tol,nslots", [(MICRO, 1e-3, 2), (MICRO_BF16, 2e-3, 1), (MICRO_WIDE, 2e-3, 10)],
                         ids=["f32-b2", "bf16-b1", "wide-b10"])
def test_micro_variant_lockstep(variant, base, tol, nslots):
    from lockstep import Lockstep
    cfg = base.with_(name=f"{base.name}-{variant}", **VARIANTS[variant])
    W = make_weights(cfg)
    prompts = [make_prefix(cfg, s, 7 + (9 * s) % 40) for s in range(nslots)]
    max_new = [40] * nslots
    opts = OracleOpts(dtype=np.float32, kv_bf16=cfg.dtype == "bf16")
    ls = Lockstep(cfg, W, prompts, max_new, tol, opts=opts)
    T = Target(cfg, W.values, opts)
    refs = [plain_greedy(T, make_memory(cfg, s), prompts[s], 40) for s in range(nslots)]
    rng = np.random.default_rng(12)
    for n in range(8):
        ls.step(override=None if n % 3 == 0 else _planted(ls, refs, rng))
    print(f"{cfg.name}: max |dlogit| draft {ls.max_dlogit:.2e} target {ls.max_tlogit:.2e}, near ties {ls.near_ties}")
    assert ls.steps == 8 and max(ls.accepted) > 0
    ls.close()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("variant", list(VARIANTS))
def test_large_v3_variant_lockstep_b1(variant):
    """Full shapes, bf16, one slot: two steps with the random drafter's own
    proposals (the drafter logits of every mask row are compared)."""
    from lockstep import Lockstep
    cfg = LARGE_V3.with_(name=f"large-v3-{variant}", **VARIANTS[variant])
    W = make_weights(cfg)
    L = int(make_prefix_lengths(1, 20, 200)[0])
    ls = Lockstep(cfg, W, [make_prefix(cfg, 0, L)], [cfg.n_ctx], 2e-2)
    for _ in range(2):
        ls.step()
    print(f"{cfg.name}: max |dlogit| draft {ls.max_dlogit:.2e} target {ls.max_tlogit:.2e}, near ties {ls.near_ties}")
    ls.close()
