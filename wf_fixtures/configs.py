"""Model shapes used by the tests and the benchmark.

``LARGE_V3`` is the target of the paper's experiments (Section 4: Whisper
large-v3; 32 decoder blocks of width 1280 with 20 heads of 64, a 5120-wide
GELU MLP and a 51866-token vocabulary).  ``TINY`` is a 4-block, width-384
Whisper-shaped decoder with fp32 weights used as the correctness workload.
``MICRO`` and ``VOCAB64`` are small shapes for brute-force and statistical
tests on the CPU (the 64-token vocabulary is the one the sampling
equivalence check runs on).

The drafter always has two blocks of the target's width (Section 3.2,
"a two-layer drafter") and a block of K = 8 mask positions (Eq. 2).
"""
from dataclasses import dataclass, field, replace


@dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layer: int          # target decoder blocks
    d_model: int          # residual width
    n_head: int           # attention heads (head width is d_model // n_head)
    d_ff: int             # MLP hidden width
    n_vocab: int          # vocabulary size (tied embedding / output head)
    taps: tuple           # zero-based target blocks whose outputs feed the history memory
    dtype: str            # "f32" or "bf16": storage type of weights, memory and caches
    n_ctx: int = 448      # learned text positions
    n_frames: int = 1500  # acoustic memory length (30 s window)
    n_draft_layer: int = 2
    block_k: int = 8      # mask positions per draft block
    eos_id: int = 50257   # end-of-transcript token id
    # drafter variants of the ablations (Section 5.4 Table 3; Table A4): without
    # its cross-attention to the acoustic memory, without the target history, and
    # with absolute positions (the target's learned position table added to the
    # block rows) instead of RoPE
    draft_audio: bool = True
    draft_history: bool = True
    draft_pos: str = "rope"   # "rope" or "abs"

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_head

    @property
    def n_tap(self) -> int:
        return len(self.taps)

    @property
    def draft_flags(self) -> int:
        """Variant bits of the C ABI (1 no audio, 2 no history, 4 absolute positions)."""
        return (0 if self.draft_audio else 1) | (0 if self.draft_history else 2) | (4 if self.draft_pos == "abs" else 0)

    def with_(self, **kw) -> "ModelConfig":
        return replace(self, **kw)


# Whisper large-v3 decoder shapes; drafter taps from Appendix A.2.
LARGE_V3 = ModelConfig(name="large-v3", n_layer=32, d_model=1280, n_head=20, d_ff=5120,
                       n_vocab=51866, taps=(1, 8, 15, 22, 29), dtype="bf16")

# Whisper-tiny-shaped decoder with fp32 weights: every block is tapped.
TINY = ModelConfig(name="tiny", n_layer=4, d_model=384, n_head=6, d_ff=1536,
                   n_vocab=51865, taps=(0, 1, 2, 3), dtype="f32")

# Small shapes for brute-force CPU tests.  Head width stays 64.
MICRO = ModelConfig(name="micro", n_layer=2, d_model=128, n_head=2, d_ff=256,
                    n_vocab=512, taps=(0, 1), dtype="f32", n_ctx=64, n_frames=48,
                    eos_id=7)

# The 64-token vocabulary variant for the sampling distribution check.
VOCAB64 = ModelConfig(name="vocab64", n_layer=2, d_model=128, n_head=2, d_ff=256,
                      n_vocab=64, taps=(0, 1), dtype="f32", n_ctx=64, n_frames=48,
                      eos_id=-1)

_BY_NAME = {c.name: c for c in (LARGE_V3, TINY, MICRO, VOCAB64)}


@dataclass(frozen=True)
class EncoderConfig:
    """Whisper audio encoder shapes (the acoustic memory the drafter and the target
    read): log-mel frontend of a 16 kHz waveform, two-convolution stem halving the
    frame rate, n_layer pre-LN blocks, n_ctx output positions (1500 for 30 s)."""
    name: str
    n_mels: int
    n_ctx: int            # output positions (half the mel frames)
    d_model: int
    n_head: int
    n_layer: int
    d_ff: int
    n_fft: int = 400
    hop: int = 160
    sample_rate: int = 16000
    dtype: str = "bf16"

    @property
    def n_samples(self) -> int:
        return 2 * self.n_ctx * self.hop

    @property
    def head_dim(self) -> int:
        return self.d_model // self.n_head

    def with_(self, **kw) -> "EncoderConfig":
        return replace(self, **kw)


# Whisper large-v3 encoder: 128 mel bins, 30 s windows (3000 mel frames, 1500
# positions), 32 blocks of width 1280 with 20 heads, MLP 5120.
LARGE_V3_ENC = EncoderConfig(name="large-v3-enc", n_mels=128, n_ctx=1500, d_model=1280, n_head=20, n_layer=32,
                             d_ff=5120)
# A small encoder for brute-force tests: 1.54 s of audio, 80 mel bins.
MICRO_ENC = EncoderConfig(name="micro-enc", n_mels=80, n_ctx=48, d_model=128, n_head=2, n_layer=2, d_ff=256)


def config_by_name(name: str) -> ModelConfig:
    return _BY_NAME[name]


# Philox stream purposes (counter word 0 carries purpose << 32 | slot).
PURPOSE = {"PREFILL": 1, "PLAIN": 2, "DRAFT": 3, "ACC": 4, "RES": 5, "BON": 6}
