"""Counter-based Gaussian projection maps (oracle side).

The paper (App. A.2, "Factor projection" and "Random maps") requires that the
two sides of a layer use distinct seeds derived from a per-layer base seed, held
fixed across every gradient that is compared, and that a dense Gaussian map be
available.  It does not name a generator.  This module fixes one, built only from
published algorithms:

* seed derivation with SplitMix64 (Steele, Lea & Flood, OOPSLA 2014; the
  64-bit finalizer constants of Vigna's reference ``splitmix64.c``);
* a counter-based stream with Philox4x32-10 (Salmon, Moraes, Dror & Shaw,
  "Parallel random numbers: as easy as 1, 2, 3", SC 2011);
* normal deviates with the Box-Muller transform (Box & Muller, 1958);
* Rademacher signs (Achlioptas, 2003, the map App. A.2 lists) from bit 31 of
  the first Philox output word of the same counter.

Definition (also implemented, independently, by the HIP library's host runtime):

    base            = SM(seed)
    s(layer, side)  = SM(base XOR (2*layer + side))     side 0 = P_in, 1 = P_out
    element (v, c) of a d x k map, flat e = v*k + c:
        (x0, x1, x2, x3) = Philox4x32-10(counter=(e mod 2^32, e div 2^32, 0, 0),
                                         key=(s mod 2^32, s div 2^32))
        u1 = ((x0*2^32 + x1) >> 11) + 1) * 2^-53          in (0, 1]
        u2 = ((x2*2^32 + x3) >> 11)      * 2^-53          in [0, 1)
        z  = sqrt(-2 ln u1) * cos(2 pi u2)
        P[v, c] = z / sqrt(k)          computed in float64
    stored value = round_to_compute_dtype(P[v, c]) with float64 -> float32 (RNE),
    then float32 -> bfloat16 (RNE) when the compute type is bfloat16.

The 1/sqrt(k) scale, with k the map's output dimension, follows the Rademacher
convention stated in App. A.2 (entries of magnitude 1/sqrt(d_out) of the map);
it makes E[P^T P] = I, so projected inner products are unbiased (pinned by a
Monte-Carlo test).  SM(x) is the output of one SplitMix64 step from state x.

Parity: the raw Philox and SplitMix64 streams are pinned to published
known-answer values (tests/golden); the seed/counter layout itself is this
library's reading and is "parity unpinned" with respect to the paper.
"""

import numpy as np

MASK32 = 0xFFFFFFFF
MASK64 = 0xFFFFFFFFFFFFFFFF

# SplitMix64 (Vigna's reference implementation of Steele et al.'s generator).
_SM_GAMMA = 0x9E3779B97F4A7C15
_SM_M1 = 0xBF58476D1CE4E5B9
_SM_M2 = 0x94D049BB133111EB

# Philox4x32 round multipliers and Weyl key increments (Salmon et al. 2011).
_PH_M0 = 0xD2511F53
_PH_M1 = 0xCD9E8D57
_PH_W0 = 0x9E3779B9
_PH_W1 = 0xBB67AE85


def splitmix64_next(state):
    """One SplitMix64 step. Returns (new_state, output) as Python ints."""
    state = (state + _SM_GAMMA) & MASK64
    z = state
    z = ((z ^ (z >> 30)) * _SM_M1) & MASK64
    z = ((z ^ (z >> 27)) * _SM_M2) & MASK64
    z = z ^ (z >> 31)
    return state, z


def sm(x):
    """Output of one SplitMix64 step taken from state ``x``."""
    return splitmix64_next(x & MASK64)[1]


def side_seed(global_seed, layer, side):
    """64-bit Philox key for one side (0 = input map, 1 = output map) of a layer."""
    if side not in (0, 1):
        raise ValueError("side must be 0 (input map) or 1 (output map)")
    return sm(sm(global_seed) ^ (2 * layer + side))


def philox4x32_10(c0, c1, c2, c3, k0, k1):
    """Philox4x32 with 10 rounds on uint32 numpy arrays (or scalars).

    Each round: (hi0, lo0) = M0 * c0, (hi1, lo1) = M1 * c2 (64-bit products),
    new counter = (hi1 ^ c1 ^ k0, lo1, hi0 ^ c3 ^ k1, lo0); the key is bumped by
    the Weyl constants between rounds.
    """
    c0 = np.asarray(c0, dtype=np.uint64)
    c1 = np.asarray(c1, dtype=np.uint64)
    c2 = np.asarray(c2, dtype=np.uint64)
    c3 = np.asarray(c3, dtype=np.uint64)
    k0 = np.uint64(k0)
    k1 = np.uint64(k1)
    m32 = np.uint64(MASK32)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + np.uint64(_PH_W0)) & m32
            k1 = (k1 + np.uint64(_PH_W1)) & m32
        p0 = np.uint64(_PH_M0) * c0
        p1 = np.uint64(_PH_M1) * c2
        hi0, lo0 = p0 >> np.uint64(32), p0 & m32
        hi1, lo1 = p1 >> np.uint64(32), p1 & m32
        c0, c1, c2, c3 = (hi1 ^ c1 ^ k0) & m32, lo1, (hi0 ^ c3 ^ k1) & m32, lo0
    return (c0.astype(np.uint32), c1.astype(np.uint32),
            c2.astype(np.uint32), c3.astype(np.uint32))


def box_muller(x0, x1, x2, x3):
    """Standard normal deviate from four uint32 words (see module docstring)."""
    a = (x0.astype(np.uint64) << np.uint64(32)) | x1.astype(np.uint64)
    b = (x2.astype(np.uint64) << np.uint64(32)) | x3.astype(np.uint64)
    u1 = ((a >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * 2.0 ** -53
    u2 = (b >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
    return np.sqrt(-2.0 * np.log(u1)) * np.cos(2.0 * np.pi * u2)


def gaussian_map_f64(seed64, d, k):
    """Unrounded d x k Gaussian map with N(0, 1/k) entries from one Philox key."""
    e = np.arange(d * k, dtype=np.uint64)
    x = philox4x32_10(e & np.uint64(MASK32), e >> np.uint64(32),
                      np.zeros_like(e), np.zeros_like(e),
                      seed64 & MASK32, seed64 >> 32)
    z = box_muller(*x)
    return (z / np.sqrt(float(k))).reshape(d, k)


def rademacher_map_f64(seed64, d, k):
    """Unrounded d x k Rademacher map with entries +-1/sqrt(k) (App. A.2
    "Random maps", k the map's output dimension) from the same Philox stream
    as the Gaussian map: element e = v*k + c takes the sign of bit 31 of the
    first output word x0 (set: negative)."""
    e = np.arange(d * k, dtype=np.uint64)
    x0, _, _, _ = philox4x32_10(e & np.uint64(MASK32), e >> np.uint64(32),
                                np.zeros_like(e), np.zeros_like(e),
                                seed64 & MASK32, seed64 >> 32)
    sign = np.where((x0 >> np.uint32(31)) != 0, -1.0, 1.0)
    return (sign / np.sqrt(float(k))).reshape(d, k)


MAPS = {"gaussian": gaussian_map_f64, "rademacher": rademacher_map_f64}


def round_bf16_from_f32(x32):
    """float32 -> bfloat16 round-to-nearest-even, returned as float32 values."""
    bits = np.ascontiguousarray(x32, dtype=np.float32).view(np.uint32)
    lsb = (bits >> np.uint32(16)) & np.uint32(1)
    rounded = (bits + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return rounded.view(np.float32)


def round_to_dtype(x64, dtype):
    """Round float64 values as the library stores them: f32 RNE, then bf16 RNE."""
    x32 = np.asarray(x64, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return x32.astype(np.float64)
    if dtype == "bf16":
        return round_bf16_from_f32(x32).astype(np.float64)
    raise ValueError("dtype must be 'f32' or 'bf16'")


def projection_pair(global_seed, layer, d_in, d_out, k_in, k_out, dtype, kind="gaussian"):
    """(P_in [d_in, k_in], P_out [d_out, k_out]) as float64 arrays holding the
    values the library stores for ``layer`` (registration index); ``kind`` is
    "gaussian" or "rademacher"."""
    gen = MAPS[kind]
    p_in = gen(side_seed(global_seed, layer, 0), d_in, k_in)
    p_out = gen(side_seed(global_seed, layer, 1), d_out, k_out)
    return round_to_dtype(p_in, dtype), round_to_dtype(p_out, dtype)
