"""Hand-worked pins of the oracle's host rules (oracle/host_rules.py).

Every expected value here comes from outside the oracle: the published output
stream of splitmix64 from state 0 (the reference generator's first six values),
worked through the sampling rule by hand in the comments, or from selection,
mask, median and radix cases written out by hand from their definitions. The
mutant test plants plausible mistakes in copies of the oracle's source and
checks that these pins reject each one.
"""
import importlib.util
import math
import os

import numpy as np
import pytest

import oracle.host_rules as HR

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "host_rules.py")

# splitmix64 from state 0: its first six outputs (published with the generator)
PUBLISHED = [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F,
             0xF88BB8A8724C81EC, 0x1B39896A51A8749B, 0x53CB9F0C747EA2EA]
INF = float("inf")


def pin_stream(H):
    g = H.SplitMix64(0)
    return [g.next() for _ in range(6)] == PUBLISHED


def pin_shuffle(H):
    # size 5, take 3, state 0: the first output is discarded, then
    #   i=0: 0x6E789E6AA1B965F4 mod 5 = 0 -> j=0, v=[0,1,2,3,4] -> 0
    #   i=1: 0x06C45D188009454F mod 4 = 3 -> j=4, v=[0,4,2,3,1] -> 4
    #   i=2: 0xF88BB8A8724C81EC mod 3 = 1 -> j=3, v=[0,4,3,2,1] -> 3
    a = H.partial_shuffle(5, 3, 0) == [0, 4, 3]
    # size 7, take 5: mod 7 = 1 -> j=1 [1,0,2,3,4,5,6] -> 1; mod 6 = 1 -> j=2 [1,2,0,...] -> 2;
    #   mod 5 = 4 -> j=6 [1,2,6,3,4,5,0] -> 6; 0x1B39896A51A8749B mod 4 = 3 -> j=6
    #   [1,2,6,0,4,5,3] -> 0; 0x53CB9F0C747EA2EA mod 3 = 0 -> j=4 -> 4
    b = H.partial_shuffle(7, 5, 0) == [1, 2, 6, 0, 4]
    return a and b


def _seed_for_zero_state(family, config_id=0, layer_id=0):
    """The seed that makes the sampler stream of `family` start at state 0,
    from the documented state rule (seed ^ GAMMA (1 + config) ^ 0xC0FFEE << 32
    ^ layer ^ 0xD1B54A32D192ED03 family, all mod 2^64)."""
    m = (1 << 64) - 1
    return ((0x9E3779B97F4A7C15 * (1 + config_id)) & m) ^ (0xC0FFEE << 32) ^ layer_id ^ \
        ((0xD1B54A32D192ED03 * family) & m)


def pin_interleave(H):
    # families 1 and 2 of sizes 7 and 1, n = 6: equal shares 3 + 3, family 2
    # holds only 1 and hands 2 on, so the quotas are 5 and 1. Family 1's stream
    # starts at state 0 (the seed is chosen for that), so its picks are the size-7
    # shuffle above, [1, 2, 6, 0, 4]; family 2 has one schedule, at position 7.
    # Output: the k-th pick of each family in family order: 1, 7, 2, 6, 0, 4.
    got = H.sample_positions([1, 2], [7, 1], 6, _seed_for_zero_state(1), 0, 0)
    return got == [1, 7, 2, 6, 0, 4]


def pin_uniform(H):
    # the whole-space shuffle from state 0: seed = GAMMA (1 + 0) ^ 0xC0FFEE << 32 ^ 0
    # cancels the other terms, so positions follow the size-7 worked shuffle
    seed = 0x9E3779B97F4A7C15 ^ (0xC0FFEE << 32)
    return H.uniform_positions(7, 5, seed, 0, 0) == [1, 2, 6, 0, 4]


def pin_quotas(H):
    return (H.family_quotas([10, 2, 7], 12) == [5, 2, 5]      # 4+4+4, family 2 hands 2 on: 5, 2, 5
            and H.family_quotas([10, 10, 10], 10) == [4, 3, 3]
            and H.family_quotas([2, 1], 10) == [2, 1])


def pin_top_t(H):
    lat = [3.0, 1.0, 2.0, 1.0, INF, 0.5]
    st = [0, 0, 0, 0, 0, 1]  # the fastest one was not OK, one is infinite
    # OK and finite: 0 (3.0), 1 (1.0), 2 (2.0), 3 (1.0); by (latency, index): 1, 3, 2, 0
    return H.top_t(lat, st, 3) == [1, 3, 2] and H.top_t(lat, st, 10) == [1, 3, 2, 0]


def pin_winner(H):
    # min 8, eps 0.25 (both exact in fp32): the band is [8, 10] inclusive;
    # 10 + 2^-10 lies outside although its position is the lowest
    a = H.select_winner([8.0, 10.0, 10.0009765625, 9.0], [6, 2, 1, 7], 0.25) == 1
    b = H.select_winner([5.0, 5.0, 5.0], [9, 4, 7], 0.0) == 1           # equal latencies: lowest position
    c = H.select_winner([INF, 3.0, INF], [0, 5, 1], 0.5) == 1           # infinite entries never tie
    d = H.select_winner([INF, INF], [0, 1], 0.01) == -1
    return a and b and c and d


def pin_masks(H):
    a = H.cu_mask(256, 0.25, 1) == [0, 0, 0xFFFFFFFF, 0xFFFFFFFF, 0, 0, 0, 0]       # CUs 64..127
    # 0.3 of 256 = 76.8 -> 77 CUs; slot 2 = CUs 154..230
    b = H.cu_mask(256, 0.3, 2) == [0, 0, 0, 0, 0xFC000000, 0xFFFFFFFF, 0xFFFFFFFF, 0x7F]
    try:
        H.cu_mask(256, 0.3, 3)  # CUs 231..307 do not exist
        c = False
    except ValueError:
        c = True
    return a and b and c


def pin_median(H):
    return (H.median([3, 1, 2]) == 2 and H.median([4, 1, 3, 2]) == np.float32(2.5)
            and H.median([1, 2]) == np.float32(1.5))


def pin_radix(H):
    # 37 = 1*20 + 3*5 + 2 over radices (3, 4, 5), first digit most significant
    return H.mixed_radix_decode([3, 4, 5], 37) == [1, 3, 2] and H.mixed_radix_encode([3, 4, 5], [1, 3, 2]) == 37


PINS = [pin_stream, pin_shuffle, pin_interleave, pin_uniform, pin_quotas, pin_top_t, pin_winner, pin_masks, pin_median,
        pin_radix]


@pytest.mark.parametrize("pin", PINS, ids=lambda p: p.__name__)
def test_oracle_host_rules_hold_hand_worked_pins(pin):
    assert pin(HR)


# plausible mistakes, each a source edit of oracle/host_rules.py
MUTANTS = {
    "first output kept": ("    rng.next()  # the first output is discarded\n", ""),
    "shuffle range short by one": ("j = i + rng.next() % (size - i)", "j = i + rng.next() % max(size - i - 1, 1)"),
    "families interleaved backwards": ("        for f in range(len(sizes)):\n            if k < q[f]:",
                                       "        for f in reversed(range(len(sizes))):\n            if k < q[f]:"),
    "no hand-on of unused shares": ("    while rem > 0:", "    for _ in range(1):"),
    "remainder to the last families": ("add = min(base + (1 if i < extra else 0), sizes[f] - q[f])",
                                       "add = min(base + (1 if i >= len(act) - extra else 0), sizes[f] - q[f])"),
    "top_t ignores status": ("if status[i] == 0 and math.isfinite(lat[i])", "if math.isfinite(lat[i])"),
    "top_t ties to the higher index": ("ok.sort(key=lambda i: (float(lat[i]), i))",
                                       "ok.sort(key=lambda i: (float(lat[i]), -i))"),
    "band edge excluded": ("float(lat[i]) <= limit", "float(lat[i]) < limit"),
    "ties to the first index": ("return min(tied, key=lambda i: pos[i])", "return min(tied)"),
    "mask size truncated": ("int(math.floor(num_cus * fraction + 0.5))", "int(num_cus * fraction)"),
    "median without averaging": ("return np.float32((v[n // 2 - 1] + v[n // 2]) / 2.0)", "return np.float32(v[n // 2])"),
    "radix digits reversed": ("    return digits[::-1]", "    return digits"),
    "splitmix shift": ("z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64",
                       "z = ((z ^ (z >> 31)) * 0xBF58476D1CE4E5B9) & MASK64"),
}


def _load_variant(tmp_path, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, "mutation site not found once: %s" % name
    path = tmp_path / ("hr_%d.py" % abs(hash(name)))
    path.write_text(src.replace(old, new))
    spec = importlib.util.spec_from_file_location("hr_mutant", str(path))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistakes(tmp_path, name):
    old, new = MUTANTS[name]
    mod = _load_variant(tmp_path, name, old, new)
    failed = []
    for p in PINS:
        try:
            ok = p(mod)
        except Exception:
            ok = False
        if not ok:
            failed.append(p.__name__)
    assert failed, "no pin rejects the mutant %r" % name
