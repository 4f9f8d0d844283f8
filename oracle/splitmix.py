"""SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
generators", OOPSLA 2014), the counter-based generator used as the seeded
tie-break of the budgeted overlap sampling.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The generator keeps a 64-bit state, adds the odd constant GAMMA (the golden
ratio scaled to 2^64) on every call and returns the state passed through the
variant-13 finaliser: xor-shift 30, multiply, xor-shift 27, multiply,
xor-shift 31.  ``tiebreak(seed, gid)`` is the first output of a generator whose
initial state is seed XOR gid.
"""
import numpy as np

GAMMA = np.uint64(0x9E3779B97F4A7C15)
M1 = np.uint64(0xBF58476D1CE4E5B9)
M2 = np.uint64(0x94D049BB133111EB)


def mix(z: np.ndarray) -> np.ndarray:
    """Variant-13 finaliser, element-wise on uint64 (wrapping arithmetic)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * M1
        z = (z ^ (z >> np.uint64(27))) * M2
    return z ^ (z >> np.uint64(31))


def sequence(seed: int, count: int) -> np.ndarray:
    """The first ``count`` outputs of SplitMix64 started from state ``seed``."""
    with np.errstate(over="ignore"):
        states = np.uint64(seed) + GAMMA * np.arange(1, count + 1, dtype=np.uint64)
    return mix(states)


def tiebreak(seed: int, gid: np.ndarray) -> np.ndarray:
    """First SplitMix64 output from state (seed XOR gid), for each gid."""
    x = np.uint64(seed) ^ np.asarray(gid, dtype=np.int64).astype(np.uint64)
    with np.errstate(over="ignore"):
        return mix(x + GAMMA)
