"""Oracle of the integer/host rules of the tuning loop -- TEST INFRASTRUCTURE ONLY.

Plain Python, written from the stated definitions, sharing nothing with the
library. Each function names the rule it follows.

* Candidate selection with no history is random (paper, section 2.1, stage
  "select configurations"), per schedule template (kernel family), since a
  TVM-style tuner tunes each template as a task of its own. The rule fixed
  here: the ascending valid list is split by family; family quotas are equal
  shares of min(n, |V|), the remainder going to the first families, and a
  family smaller than its share hands the rest on, in rounds; within a family
  a partial Fisher-Yates shuffle driven by splitmix64 (Steele, Lea, Flood,
  OOPSLA 2014) from state
  seed ^ (GAMMA * (1 + config_id) mod 2^64) ^ (0xC0FFEE << 32) ^ layer_id
       ^ (0xD1B54A32D192ED03 * family mod 2^64),
  first output discarded, j = i + next() mod (|V_f| - i); the output takes
  the k-th pick of every family in family order, then the (k+1)-th.
* A configuration's latency is the median of its repeats (the profile stage
  measures execution time; the statistic is this build's reading).
* The best configuration is the one with the lowest latency (implied by the
  early-stop rule of section 2.2.1, which stops when new configurations no
  longer lower it). Screening keeps the t fastest by (latency, sample position);
  among the re-measured ones every latency within (1 + eps) of the minimum is
  a tie and the lowest sample position wins.
* A fixed GPU share per process (section 2.2) is a CU mask: m = round(n f) CUs,
  slot j = mask bits [j m, (j + 1) m).
* Knob grids are mixed-radix numbers, first knob most significant.

Pins (tests/test_oracle_host_pins.py): the published splitmix64 stream from
state 0, shuffles and a two-family interleave worked by hand from it, and
hand-worked quota, top-t, tie-band, mask, median and radix cases; planted
mistakes in copies of this file are each rejected by one of them.
"""
from __future__ import annotations

import math
from typing import List, Sequence

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15


class SplitMix64:
    """splitmix64: state += GAMMA; z = state; two xor-shift-multiply rounds; final xor-shift."""

    def __init__(self, state: int):
        self.state = state & MASK64

    def next(self) -> int:
        self.state = (self.state + GAMMA) & MASK64
        z = self.state
        z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
        z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
        return z ^ (z >> 31)


def sampler_state(seed: int, config_id: int, layer_id: int, family: int) -> int:
    return (seed ^ ((GAMMA * (1 + config_id)) & MASK64) ^ ((0xC0FFEE << 32) & MASK64)
            ^ (layer_id & 0xFFFFFFFF) ^ ((0xD1B54A32D192ED03 * family) & MASK64)) & MASK64


def partial_shuffle(size: int, take: int, state: int) -> List[int]:
    """The first `take` positions of a Fisher-Yates shuffle of range(size)."""
    rng = SplitMix64(state)
    rng.next()  # the first output is discarded
    v = list(range(size))
    out = []
    for i in range(min(take, size)):
        j = i + rng.next() % (size - i)
        v[i], v[j] = v[j], v[i]
        out.append(v[i])
    return out


def uniform_positions(size: int, n: int, seed: int, config_id: int, layer_id: int) -> List[int]:
    """The sample without family quotas: the first n positions of one partial
    shuffle of the whole valid list, from the state without the family term."""
    state = (seed ^ ((GAMMA * (1 + config_id)) & MASK64) ^ ((0xC0FFEE << 32) & MASK64)
             ^ (layer_id & 0xFFFFFFFF)) & MASK64
    return partial_shuffle(size, n, state)


def family_quotas(sizes: Sequence[int], n: int) -> List[int]:
    """Equal shares of min(n, total), the remainder to the first families; a
    family smaller than its share hands the rest on, round after round."""
    q = [0] * len(sizes)
    rem = min(n, sum(sizes))
    while rem > 0:
        act = [f for f in range(len(sizes)) if q[f] < sizes[f]]
        base, extra = divmod(rem, len(act))
        for i, f in enumerate(act):
            add = min(base + (1 if i < extra else 0), sizes[f] - q[f])
            q[f] += add
            rem -= add
    return q


def sample_positions(families: Sequence[int], sizes: Sequence[int], n: int, seed: int, config_id: int,
                     layer_id: int) -> List[int]:
    """Indices into the ascending valid list (families in order, family f
    holding sizes[f] entries), in sample order."""
    q = family_quotas(sizes, n)
    starts = [sum(sizes[:f]) for f in range(len(sizes))]
    picks = [partial_shuffle(sizes[f], q[f], sampler_state(seed, config_id, layer_id, families[f]))
             for f in range(len(sizes))]
    out = []
    for k in range(max(q, default=0)):
        for f in range(len(sizes)):
            if k < q[f]:
                out.append(starts[f] + picks[f][k])
    return out


def mixed_radix_decode(radices: Sequence[int], index: int) -> List[int]:
    """Digits of index, first digit most significant."""
    digits = []
    for r in reversed(radices):
        digits.append(index % r)
        index //= r
    return digits[::-1]


def mixed_radix_encode(radices: Sequence[int], digits: Sequence[int]) -> int:
    idx = 0
    for r, d in zip(radices, digits):
        idx = idx * r + d
    return idx


def cu_mask(num_cus: int, fraction: float, slot: int, words: int = 8) -> List[int]:
    m = int(math.floor(num_cus * fraction + 0.5))
    if m <= 0 or (slot + 1) * m > num_cus:
        raise ValueError("slot does not fit")
    bits = [0] * words
    for b in range(slot * m, (slot + 1) * m):
        bits[b // 32] |= 1 << (b % 32)
    return bits


def median(values) -> float:
    """Median of float32 values; an even count averages the two middle ones in fp64."""
    import numpy as np
    v = sorted(float(np.float32(x)) for x in values)
    n = len(v)
    if n % 2:
        return np.float32(v[n // 2])
    return np.float32((v[n // 2 - 1] + v[n // 2]) / 2.0)


def top_t(lat, status, t: int) -> List[int]:
    ok = [i for i in range(len(lat)) if status[i] == 0 and math.isfinite(lat[i])]
    ok.sort(key=lambda i: (float(lat[i]), i))
    return ok[:t]


def select_winner(lat, pos, eps: float) -> int:
    """Index (into lat) of the winner, or -1 if no latency is finite."""
    import numpy as np
    finite = [float(l) for l in lat if math.isfinite(l)]
    if not finite:
        return -1
    limit = min(finite) * (1.0 + float(np.float32(eps)))
    tied = [i for i in range(len(lat)) if math.isfinite(lat[i]) and float(lat[i]) <= limit]
    return min(tied, key=lambda i: pos[i])
