"""Parameter checksum (oracle; test-only).

The library's checksum of a set of bf16 tensors (or of int8 codes), written
out from its definition: every element contributes mix64(j K_J + id K_T + b K_B) and the
contributions are added mod 2^64, where j is the element's index in its
whole tensor, id the tensor's noise identity, b the element's 16 bits, and
mix64 the 64-bit finalizer of SplitMix64 (Steele, Lea and Flood, "Fast
splittable pseudorandom number generators", OOPSLA 2014).  The paper does not
define a checksum; the library provides one so that a run rebuilt from its
seed log (Section 3 and Appendix D.6 keep only seeds) can be checked against
values recorded during the run.

Pins (tests/test_oracle_checksum.py): the first outputs of SplitMix64 from
state 0 (tests/golden/splitmix64.txt) through this mix64; mix64 inverted by a
separately written inverse (modular inverses of the multipliers, xor-shifts
undone bit by bit) on random inputs; a pure-Python big-integer evaluation of
the sum on small tensors; additivity over split ranges (the property that
makes shard checksums add up); and sensitivity to every element's bits, its
position and the tensor id.
"""

import numpy as np

MASK64 = (1 << 64) - 1
K_J = 0x9E3779B97F4A7C15
K_T = 0xC2B2AE3D27D4EB4F
K_B = 0x165667B19E3779F9
MIX_M1 = 0xBF58476D1CE4E5B9
MIX_M2 = 0x94D049BB133111EB


def mix64(z):
    """SplitMix64's finalizer on uint64 values (array or scalar), wrapping
    mod 2^64."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * np.uint64(MIX_M1)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(MIX_M2)
        return z ^ (z >> np.uint64(31))


def checksum(bits, tensor_id, elem0=0, chunk=1 << 22):
    """Checksum (a Python int in [0, 2^64)) of the bf16 elements `bits`
    (uint16) that sit at whole-tensor indices elem0, elem0 + 1, ... of tensor
    `tensor_id`."""
    return _sum(np.asarray(bits, dtype=np.uint16).ravel(), tensor_id, elem0, chunk)


def qchecksum(codes, tensor_id, elem0=0, chunk=1 << 22):
    """Checksum of one-byte codes (int8 or E4M3) at whole-tensor indices
    elem0, elem0 + 1, ... of tensor `tensor_id`: the same sum with b the
    code's 8 bits read as an unsigned byte."""
    return _sum(np.asarray(codes, dtype=np.int8).ravel().view(np.uint8), tensor_id, elem0, chunk)


def _sum(b_all, tensor_id, elem0, chunk):
    salt = np.uint64((int(tensor_id) * K_T) & MASK64)
    total = 0
    for c0 in range(0, b_all.size, chunk):
        b = b_all[c0:c0 + chunk].astype(np.uint64)
        j = np.arange(b.size, dtype=np.uint64) + np.uint64(int(elem0) + c0)
        with np.errstate(over="ignore"):
            x = j * np.uint64(K_J) + salt + b * np.uint64(K_B)
        total = (total + int(mix64(x).sum(dtype=np.uint64))) & MASK64
    return total


def plan_checksum(parts):
    """Checksum of several tensors or shards: parts is a list of
    (bits, tensor_id, elem0)."""
    total = 0
    for bits, tid, elem0 in parts:
        total = (total + checksum(bits, tid, elem0)) & MASK64
    return total
