"""CPU oracle for the ES parameter path (test infrastructure, not product code).

This package is a plain, slow, obviously-correct NumPy implementation of what
the GPU library computes: the counter-based noise (Philox4x32-10 words, the
uniform map, the Box-Muller transform), in-place perturb/restore of bf16
parameters, the population z-score of rewards, the reward-weighted update, and
the cosine schedule of the perturbation radius.  Floating point work is done in
fp64 and rounded to bf16 exactly once, round-to-nearest-even (the update can
instead round stochastically, from binary32, with counter-based draws).

Only the test suite, the smoke check and the CPU-baseline leg of the benchmark
may import it.  It shares no code with the HIP library and imports nothing from
it; the two meet only through the seeded input generators, which hold none of
the method's arithmetic.

Paper sections followed (arXiv 2608.17310, "Agentic ESOpt"):
  * Section 3 (Methodology): Gaussian-smoothed objective, population z-score,
    the implemented update theta += (alpha/G) sum_i zhat_i eps_i, seed-only
    noise with in-place addition and subtraction.
  * Section 3.1: cosine decay of sigma.
  * Appendix C.1: canonical estimator with the explicit 1/(G sigma) factor.
  * Appendix D.6 (hyperparameter summary): perturb, evaluate, revert,
    regenerate the direction from its integer seed at update time.
The paper names no generator and no transform; Philox4x32-10 is the published
generator of Salmon, Moraes, Dror and Shaw (SC'11) and Box-Muller the textbook
transform of Box and Muller (1958).

checksum.py sums a 64-bit mix of every element's index, tensor id and bits
mod 2^64: the library's parameter checksum, used to check a replayed run.

The int8 path (quant.py) perturbs and updates symmetric int8 codes with
per-row scales in units of the quantum, rounding offsets stochastically; the
fp8 path (fp8.py) does the same on the grid of the E4M3 format, rounding the
scaled value stochastically onto it; the paper lists quantized ES as future
work (Appendix A.2).

Pin status of every function is listed in the module docstrings; all functions
are pinned (none is "parity unpinned").
"""

from .philox import philox4x32_10, philox4x32_10_bigint, MASK32
from .noise import (key_words, counter_words, uniform_from_word, angle_from_word,
                    box_muller, noise_words, normals, rounding_draws, spare_draws)
from .bf16 import bf16_to_f64, f64_to_bf16_rne, f64_to_bf16_sr, bf16_ulp
from .es import (perturb, restore, swap, zscore, update_coefficient, member_weights,
                 update, update_master, perturb_master, sigma_cosine, ES_UPDATE_DIV_SIGMA,
                 ES_REWARDS_ARE_WEIGHTS, ES_UPDATE_STOCHASTIC_ROUND, ES_UPDATE_MASTER)
from .quant import (QMAX, row_scales, round_offset, round_offset9, offset_values, qperturb,
                    qrestore, update_values, qupdate)
from .checksum import mix64, checksum, qchecksum, plan_checksum
from . import fp8
from .fp8 import (E4M3_MAX, e4m3_decode, e4m3_encode, grid_floor, round_onto_grid, f8perturb,
                  f8restore, f8update_values, f8update)

__all__ = [
    "philox4x32_10", "philox4x32_10_bigint", "MASK32",
    "key_words", "counter_words", "uniform_from_word", "angle_from_word", "box_muller",
    "noise_words", "normals", "rounding_draws", "spare_draws",
    "bf16_to_f64", "f64_to_bf16_rne", "f64_to_bf16_sr", "bf16_ulp",
    "perturb", "restore", "swap", "zscore", "update_coefficient", "member_weights",
    "update", "update_master", "perturb_master", "sigma_cosine", "ES_UPDATE_DIV_SIGMA", "ES_REWARDS_ARE_WEIGHTS",
    "ES_UPDATE_MASTER",
    "ES_UPDATE_STOCHASTIC_ROUND",
    "QMAX", "row_scales", "round_offset", "round_offset9", "offset_values", "qperturb", "qrestore", "update_values", "qupdate",
    "mix64", "checksum", "qchecksum", "plan_checksum",
    "fp8", "E4M3_MAX", "e4m3_decode", "e4m3_encode", "grid_floor", "round_onto_grid",
    "f8perturb", "f8restore", "f8update_values", "f8update",
]
