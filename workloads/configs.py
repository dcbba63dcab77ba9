"""Synthetic workload descriptions for the Seer hot path (shapes, seeds, knobs).

Each workload is a batch of sequences laid out as [visual prefix ; prompt ;
generation window], the layout the method operates on (Sec. 3.1, the denoising
step equation: every step re-processes the whole window together with the
visual context).  The shapes mirror the paper's serving workloads: a LLaDA-8B
sized layer (d=4096, 32 heads of 128, SwiGLU intermediate 12288) with a
27x27-patch visual prefix, multi-crop and multi-frame prefixes, and generation
windows that are mostly padding.  The paper's datasets and trained weights are
not used; these seeded synthetic batches stand in for them.

This module holds only data (sizes, seeds, thresholds).  It contains none of
the method's arithmetic and is shared by the oracle and the GPU path.
"""
from dataclasses import dataclass, field
from fractions import Fraction
from typing import Optional, Tuple


@dataclass(frozen=True)
class LayerShape:
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int            # SwiGLU intermediate size I

    @property
    def gemm_flop_per_row(self) -> int:
        # QKV (3 d^2) + O (d^2) + gate/up (2 d I) + down (d I), two flop per MAC.
        d, i = self.d_model, self.d_ff
        return 2 * (4 * d * d + 3 * d * i)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: LayerShape
    n_layers: int
    l_det: int                 # layer whose MLP feeds the sparsity statistic (0-based)
    batch: int
    n_visual: int
    n_prompt: int
    window: int                # generation window length N
    dtype: str                 # "f32" or "bf16"
    boundary: Tuple            # ("fixed", b) | ("loguniform", lo, hi) | ("uniform", lo, hi)
    seed: int
    act_eps: float             # near-zero threshold on |SwiGLU activation| (strict <)
    trunc_steps: int = 1       # truncated denoising steps after step 0
    eos_amplitude: float = 16.0
    noise_std: float = 0.01    # std of the per-position noise added to the EOS vector
    weight_std: float = 0.02
    rms_eps: float = 1e-5
    # confounders for the detector-sensitivity sweeps: (runs per sequence, longest
    # run) of content positions replaced by EOS rows before the planted boundary
    dips: Tuple[int, int] = (0, 0)
    # layers whose gate/up weights define the planted EOS direction (None: l_det)
    eos_layers: Optional[Tuple[int, ...]] = None

    @property
    def prefix_len(self) -> int:
        return self.n_visual + self.n_prompt

    @property
    def seq_len_full(self) -> int:
        return self.prefix_len + self.window

    @property
    def rows_full(self) -> int:
        return self.batch * self.seq_len_full


# SNR detector defaults: tau_jump = 0.03, gamma = 0.6, look-ahead of three
# positions (Sec. 3.3; the defaults are the knee of the Pareto study in Sec. 4).
TAU_JUMP = Fraction(3, 100)
GAMMA = Fraction(3, 5)
LOOKAHEAD = 3
# Static-path admission threshold on the padding waste ratio (Sec. 3.4).
TAU_PAD = Fraction(1, 5)

LLADA8B = LayerShape(d_model=4096, n_heads=32, head_dim=128, d_ff=12288)
TINY = LayerShape(d_model=256, n_heads=4, head_dim=64, d_ff=688)
# Smallest shape the bf16 kernels take (head_dim 128): parity cases that
# still span several GEMM tiles and attention tiles with ragged tails.
SMALL_BF16 = LayerShape(d_model=512, n_heads=4, head_dim=128, d_ff=1024)


def act_eps_for(shape: LayerShape, weight_std: float = 0.02, kappa: float = 0.01) -> float:
    """Near-zero threshold: kappa times the variance of a gate pre-activation.

    With RMS-normalised inputs (unit mean square) and N(0, s^2) weights a gate
    pre-activation has variance s^2 * d; the threshold is 1% of that.
    """
    return kappa * weight_std * weight_std * shape.d_model


WORKLOADS = {
    "tiny_f32": Workload(
        name="tiny_f32", shape=TINY, n_layers=1, l_det=0, batch=1,
        n_visual=64, n_prompt=32, window=128, dtype="f32",
        boundary=("fixed", 40), seed=1234, act_eps=act_eps_for(TINY)),
    "llada_b1": Workload(
        name="llada_b1", shape=LLADA8B, n_layers=1, l_det=0, batch=1,
        n_visual=729, n_prompt=64, window=1024, dtype="bf16",
        boundary=("fixed", 96), seed=2002, act_eps=act_eps_for(LLADA8B)),
    "llada_b16_ragged": Workload(
        name="llada_b16_ragged", shape=LLADA8B, n_layers=1, l_det=0, batch=16,
        n_visual=729, n_prompt=64, window=1024, dtype="bf16",
        boundary=("loguniform", 16, 512), seed=3003, act_eps=act_eps_for(LLADA8B)),
    "llada32_multicrop_b8": Workload(
        name="llada32_multicrop_b8", shape=LLADA8B, n_layers=32, l_det=3, batch=8,
        n_visual=3645, n_prompt=64, window=512, dtype="bf16",
        boundary=("uniform", 32, 256), seed=4004, act_eps=act_eps_for(LLADA8B),
        trunc_steps=63),
    "llada32_video_b4": Workload(
        name="llada32_video_b4", shape=LLADA8B, n_layers=32, l_det=3, batch=4,
        n_visual=3136, n_prompt=128, window=2048, dtype="bf16",
        boundary=("uniform", 64, 1024), seed=5005, act_eps=act_eps_for(LLADA8B),
        trunc_steps=63),
}

# Parity-test workloads at reduced size (not benchmark lines).
WORKLOADS["small_bf16_ragged"] = Workload(
    name="small_bf16_ragged", shape=SMALL_BF16, n_layers=1, l_det=0, batch=5,
    n_visual=100, n_prompt=27, window=160, dtype="bf16",
    boundary=("uniform", 12, 140), seed=606, act_eps=act_eps_for(SMALL_BF16))
WORKLOADS["small_bf16_stack"] = Workload(
    name="small_bf16_stack", shape=SMALL_BF16, n_layers=3, l_det=1, batch=3,
    n_visual=150, n_prompt=20, window=200, dtype="bf16",
    boundary=("uniform", 20, 180), seed=707, act_eps=act_eps_for(SMALL_BF16))

# Detector-sensitivity sweeps (look-ahead, tau_jump x gamma, detection layer):
# six layers with the EOS direction planted at layer 3, EOS rows with strong
# per-position noise (a noisy padding plateau), and up to two runs of one or
# two EOS rows inside the content, which a look-ahead of 2 mistakes for the
# boundary.
WORKLOADS["sweep_small"] = Workload(
    name="sweep_small", shape=SMALL_BF16, n_layers=6, l_det=3, batch=64,
    n_visual=64, n_prompt=16, window=256, dtype="bf16",
    boundary=("uniform", 24, 224), seed=808, act_eps=act_eps_for(SMALL_BF16),
    noise_std=10.0, dips=(2, 2))
WORKLOADS["sweep_llada"] = Workload(
    name="sweep_llada", shape=LLADA8B, n_layers=6, l_det=3, batch=32,
    n_visual=256, n_prompt=32, window=512, dtype="bf16",
    boundary=("uniform", 32, 448), seed=909, act_eps=act_eps_for(LLADA8B),
    noise_std=10.0, dips=(2, 2))

WORKLOAD_ORDER = ["tiny_f32", "llada_b1", "llada_b16_ragged",
                  "llada32_multicrop_b8", "llada32_video_b4"]


def scaled(w: Workload, **changes) -> Workload:
    """A copy of a workload with some fields replaced (used for small test cases)."""
    from dataclasses import replace
    return replace(w, **changes)
