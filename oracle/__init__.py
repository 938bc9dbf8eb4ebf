"""CPU oracle for the Whisper-Flash draft-and-verify step.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import or run
this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the
HIP path; both take inputs from ``wf_fixtures``.

The oracle is plain numpy, fp32 by default (the softmax and acceptance
probabilities are fp32 as the paper fixes in Appendix A.4; everything else
follows that precision), with an optional fp64 mode used by the pins.

Modules
  numerics   LayerNorm, exact-erf GELU, softmax attention, RoPE, bf16 rounding
  model      frozen Whisper decoder (target) and the two-block drafter
  accept     greedy longest-prefix acceptance and the rejection-sampling rule
  philox     Philox4x64-10 counter-based generator, uniforms and Gumbel noise
  decode     plain greedy / plain sampling loops and the speculative loop
"""
from .numerics import OracleOpts
from .model import Target, Drafter, TargetCache, HistoryCache
from .accept import greedy_accept, rejection_accept, budget_k
from .decode import (Session, plain_greedy, brute_greedy, spec_greedy, plain_sample, spec_sample)

__all__ = ["OracleOpts", "Target", "Drafter", "TargetCache", "HistoryCache",
           "greedy_accept", "rejection_accept", "budget_k", "Session",
           "plain_greedy", "brute_greedy", "spec_greedy", "plain_sample", "spec_sample"]
