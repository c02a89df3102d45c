"""Seed-only Gaussian noise: which Philox words feed which parameter, the
uniform map and the Box-Muller transform (oracle; test-only).

The paper stores only an integer seed per perturbation and regenerates the
same full-parameter direction eps ~ N(0, I) from it at update time (Section 3,
the paragraph after the implemented update; Appendix D.6).  It does not say
how; the definition below is this library's reading, fixed once so that any
element of any tensor can be regenerated in isolation:

  key     = (seed mod 2^32, seed div 2^32)                 seed: 64-bit
  counter = (q mod 2^32, q div 2^32, tensor_id, domain)    q = j div 4
  element j of tensor `tensor_id` uses the pair (w0, w1) of the call at
  counter q when j mod 4 is 0 or 1, and the pair (w2, w3) when it is 2 or 3.
  domain is 0 for the perturbation noise and 1 for the draws of the update's
  stochastic rounding (other values are reserved).

  m(w) = w mod 2^23 (the low 23 bits of a word)
  radius uniform u(w) = (m(w) + 1/2) * 2^-23, in [2^-24, 1 - 2^-24]
  angle (in turns)  v(w) = m(w) * 2^-23,     in [0, 1)
  Both are exact in binary32 as well as binary64, and log(0) cannot occur.

  Box-Muller (G. E. P. Box, M. E. Muller, 1958) on a word pair (wa, wb):
      r   = sqrt(-2 ln u(wa)),  phi = 2 pi v(wb)
      first  element of the pair: r cos(phi)
      second element of the pair: r sin(phi)

Spare bits: the uniform map reads only the low 23 bits of a word, so each
word's top 9 bits are a free draw, independent of the normal it helps make.
Element j's spare draw is the top 9 bits of word (j mod 4) of the call at its
quad (the int8 path rounds perturbation offsets with it).

Stochastic-rounding draws (domain 1, key from the update's rounding seed):
one Philox call at counter (g mod 2^32, g div 2^32, tensor_id, 1), g = j div 8,
serves elements 8g .. 8g+7; element j takes word (j mod 8) div 2, its low 16
bits when j is even and its high 16 bits when j is odd.

Pins (tests/test_oracle_noise.py, tests/test_oracle_rounding.py): the word-to-element assignment against the
counter/offset API of PyTorch's and rocRAND's Philox engines; the uniform map's
closed-form endpoints; hand-worked Box-Muller values; the moments, the
Kolmogorov-Smirnov distance to N(0,1), the closed-form bound
|eps| <= sqrt(48 ln 2) and the pair correlation of the generated normals; the
rounding draws against the big-integer Philox and their uniformity.
"""

import numpy as np

from .philox import philox4x32_10, MASK32

DOMAIN_NOISE = 0
DOMAIN_ROUNDING = 1


def key_words(seed):
    """Split a 64-bit seed into the two 32-bit Philox key words."""
    seed = int(seed)
    if not 0 <= seed < (1 << 64):
        raise ValueError("seed must be in [0, 2^64)")
    return (seed & MASK32, seed >> 32)


def counter_words(q, tensor_id, domain=DOMAIN_NOISE):
    """Counter words (c0, c1, c2, c3) for quad index q (array) of a tensor."""
    q = np.asarray(q, dtype=np.uint64)
    return (q & np.uint64(MASK32), q >> np.uint64(32),
            np.full(q.shape, tensor_id, dtype=np.uint64),
            np.full(q.shape, domain, dtype=np.uint64))


def noise_words(seed, tensor_id, quads, domain=DOMAIN_NOISE):
    """The four Philox words of every quad in `quads`: a (4, n) uint64 array."""
    quads = np.atleast_1d(np.asarray(quads, dtype=np.uint64))
    return philox4x32_10(counter_words(quads, tensor_id, domain),
                         key_words(seed))


def low23(w):
    """m(w) = w mod 2^23."""
    return np.asarray(w, dtype=np.uint64) & np.uint64((1 << 23) - 1)


def uniform_from_word(w):
    """Radius uniform u(w) = (m(w) + 1/2) * 2^-23, exact in fp64."""
    return (low23(w).astype(np.float64) + 0.5) * 2.0 ** -23


def angle_from_word(w):
    """Angle in turns v(w) = m(w) * 2^-23, exact in fp64."""
    return low23(w).astype(np.float64) * 2.0 ** -23


def box_muller(wa, wb):
    """Box-Muller on word pairs; returns (r cos phi, r sin phi) in fp64."""
    r = np.sqrt(-2.0 * np.log(uniform_from_word(wa)))
    phi = 2.0 * np.pi * angle_from_word(wb)
    return r * np.cos(phi), r * np.sin(phi)


def normals(seed, tensor_id, elems):
    """eps_j for the given element indices j of one tensor, in fp64.

    Any element is computed from its own Philox call, independently of the
    others; a list of arbitrary (sampled) indices is fine.
    """
    elems = np.atleast_1d(np.asarray(elems, dtype=np.uint64))
    q = elems >> np.uint64(2)
    lane = (elems & np.uint64(3)).astype(np.int64)
    w = noise_words(seed, tensor_id, q)
    first_pair = lane < 2
    wa = np.where(first_pair, w[0], w[2])
    wb = np.where(first_pair, w[1], w[3])
    e_cos, e_sin = box_muller(wa, wb)
    return np.where(lane % 2 == 0, e_cos, e_sin)


def rounding_draws(round_seed, tensor_id, elems, domain=DOMAIN_ROUNDING):
    """The 16-bit stochastic-rounding draw of each element index j of one
    tensor (domain 1 by default): an int64 array with values in [0, 65535]."""
    elems = np.atleast_1d(np.asarray(elems, dtype=np.uint64))
    g = elems >> np.uint64(3)
    w = noise_words(round_seed, tensor_id, g, domain)
    word = (elems >> np.uint64(1)) & np.uint64(3)
    picked = np.choose(word.astype(np.int64), [w[0], w[1], w[2], w[3]])
    shift = (elems & np.uint64(1)) * np.uint64(16)
    return ((picked >> shift) & np.uint64(0xFFFF)).astype(np.int64)


def spare_draws(seed, tensor_id, elems):
    """The 9-bit spare draw of each element index j: word (j mod 4) of the
    noise call at quad j div 4, shifted right by 23 (int64 in [0, 511])."""
    elems = np.atleast_1d(np.asarray(elems, dtype=np.uint64))
    w = noise_words(seed, tensor_id, elems >> np.uint64(2))
    lane = (elems & np.uint64(3)).astype(np.int64)
    picked = np.choose(lane, [w[0], w[1], w[2], w[3]])
    return (picked >> np.uint64(23)).astype(np.int64)
