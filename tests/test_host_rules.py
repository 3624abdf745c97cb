"""Host logic of the library (no GPU needed), checked against oracle/host_rules.py.

Also checks that libconvtune.so loads and exports every function that
include/convtune.h declares (no compute call is made).
"""
import math
import random

import numpy as np
import pytest

import oracle.host_rules as HR
from paper_2008_03602_amd import _lib as L, synth, workloads as W


def test_library_exports_every_declared_function():
    names = L.header_functions()
    assert len(names) >= 20
    h = L.lib()
    missing = [n for n in names if not hasattr(h, n)]
    assert not missing, missing
    assert set(names) == set(L._SIGS), "binding and header disagree"


def test_uninitialised_device_calls_fail_cleanly():
    # nothing here initialises a device; entry points must return CT_E_NOINIT, not crash
    with pytest.raises(L.CtError) as e:
        L.ct_num_cus()
    assert e.value.code == L.CT_E_NOINIT
    op = W.config(1).ops[0]
    with pytest.raises(L.CtError):
        L.measure_candidates(op, L.ct_sample(op, 0, 1, 0, 2), 1.0, L.make_opts(), 1, 1, 1)


def test_splitmix64_matches_published_first_output_and_numpy_stream():
    # splitmix64 seeded with 0 starts 0xE220A8397B1DCDAF (the reference generator's first value)
    g = HR.SplitMix64(0)
    first = [g.next() for _ in range(5)]
    assert first[0] == 0xE220A8397B1DCDAF
    vec = synth.splitmix64_block(0, 5, skip=0)
    assert [int(v) for v in vec] == first


@pytest.mark.parametrize("family", [1, 2, 3, 4])
def test_grid_decode_encode_roundtrip(family):
    nk, size = L.ct_grid_info(family)
    vals = [L.ct_knob_values(family, k) for k in range(nk)]
    radices = [len(v) for v in vals]
    assert size == int(np.prod(radices))
    rng = random.Random(family)
    for idx in [0, size - 1] + [rng.randrange(size) for _ in range(200)]:
        s = L.ct_grid_decode(family, idx)
        digits = HR.mixed_radix_decode(radices, idx)
        assert [s.knob[k] for k in range(nk)] == [vals[k][d] for k, d in enumerate(digits)]
        assert L.ct_grid_encode(s) == idx == HR.mixed_radix_encode(radices, digits)
    with pytest.raises(L.CtError):
        L.ct_grid_decode(family, size)


@pytest.mark.parametrize("cfg,layer", [(1, 0), (2, 0), (2, 9), (4, 5), (5, 0), (5, 12)])
def test_sampler_is_bit_identical_to_oracle(cfg, layer):
    c = W.config(cfg)
    op = c.ops[layer]
    space = L.ct_valid_space(op)
    fams = sorted({s.family for s in space})
    sizes = [sum(1 for s in space if s.family == f) for f in fams]
    for seed in (0, 1, 12345):
        got = L.ct_sample(op, seed, cfg, layer, c.n_candidates)
        pos = HR.sample_positions(fams, sizes, c.n_candidates, seed, cfg, layer)
        assert len(got) == len(pos) == min(c.n_candidates, len(space))
        assert [L.schedule_tuple(s) for s in got] == [L.schedule_tuple(space[p]) for p in pos]
        assert len(set(pos)) == len(pos)


@pytest.mark.parametrize("cfg,layer", [(2, 1), (4, 5), (5, 12)])
def test_uniform_sampler_is_bit_identical_to_oracle(cfg, layer):
    c = W.config(cfg)
    op = c.ops[layer]
    space = L.ct_valid_space(op)
    for seed in (0, 7):
        got = L.ct_sample_uniform(op, seed, cfg, layer, 256)
        pos = HR.uniform_positions(len(space), 256, seed, cfg, layer)
        assert [L.schedule_tuple(s) for s in got] == [L.schedule_tuple(space[p]) for p in pos]


def test_family_quotas_by_hand():
    assert HR.family_quotas([5, 100], 20) == [5, 15]      # a small family hands its share on
    assert HR.family_quotas([3, 3], 10) == [3, 3]         # the whole space
    assert HR.family_quotas([10, 10, 10], 10) == [4, 3, 3]
    assert HR.family_quotas([1, 2, 50], 9) == [1, 2, 6]
    assert HR.family_quotas([], 5) == []


def test_sample_is_balanced_and_interleaved_across_families():
    op = W.config(2).ops[1]  # direct and fp32 MFMA families both apply
    got = L.ct_sample(op, 0, 2, 1, 256)
    fams = [s.family for s in got]
    assert fams.count(1) == fams.count(4) == 128
    assert fams[:6] == [1, 4, 1, 4, 1, 4]


def test_sampler_determinism_and_seed_sensitivity():
    op = W.config(1).ops[0]
    a = [L.schedule_tuple(s) for s in L.ct_sample(op, 0, 1, 0, 64)]
    b = [L.schedule_tuple(s) for s in L.ct_sample(op, 0, 1, 0, 64)]
    c = [L.schedule_tuple(s) for s in L.ct_sample(op, 1, 1, 0, 64)]
    assert a == b and a != c


def test_sampler_returns_whole_space_when_small():
    op = W.mobilenet_v2_pointwise(16)[0]  # 32 -> 16 channels: a tiny space
    space = L.ct_valid_space(op)
    got = L.ct_sample(op, 0, 5, 10, 1024)
    assert len(got) == len(space) < 1024
    assert sorted(L.schedule_tuple(s) for s in got) == sorted(L.schedule_tuple(s) for s in space)


def test_every_sampled_schedule_validates():
    for op in W.resnet18(1)[:3] + W.mobilenet_v2_depthwise(16)[:2] + W.mobilenet_v2_pointwise(16)[-2:]:
        for s in L.ct_sample(op, 7, 2, 0, 64):
            assert L.ct_validate(op, s) == 0
            shape = L.ct_launch_shape(op, s)
            assert 32 <= shape["threads"] <= 1024 and shape["lds_bytes"] <= 160 * 1024 and shape["blocks"] >= 1


@pytest.mark.parametrize("frac,slots", [(0.125, 8), (0.25, 4), (0.5, 2), (0.75, 1), (1.0, 1)])
def test_cu_masks_match_oracle_and_are_disjoint(frac, slots):
    union = 0
    for j in range(slots):
        m = L.ct_build_cu_mask(256, frac, j)
        assert list(m) == HR.cu_mask(256, frac, j)
        bits = sum(int(v) << (32 * i) for i, v in enumerate(m))
        assert bin(bits).count("1") == round(256 * frac)
        assert union & bits == 0
        union |= bits
    with pytest.raises(L.CtError):
        L.ct_build_cu_mask(256, frac, slots)


def test_top_t_and_winner_match_oracle_with_ties():
    rng = np.random.default_rng(3)
    for trial in range(200):
        n = int(rng.integers(1, 40))
        lat = rng.choice(np.array([1.0, 1.005, 1.02, 2.0, 3.5, np.inf], dtype=np.float32), size=n)
        st = rng.choice([0, 0, 0, 1, 3, 4], size=n).astype(np.int32)
        t = int(rng.integers(1, 10))
        top = L.ct_top_t(lat, st, t)
        assert list(top) == HR.top_t(lat, st, t)
        pos = rng.permutation(n).astype(np.int32)
        assert L.ct_select_winner(lat, pos, 0.01) == HR.select_winner(lat, pos, 0.01)


def test_validator_rejects_documented_cases():
    op = W.config(1).ops[0]
    # 8 x 8 x 8 threads = 1024 ok; a direct tile of 14 x 56 with mk=1, mw=1, tk=64 is 50176 threads
    bad_threads = L.make_schedule(1, [14, 56, 64, 1, 1, 0, 8, 1, 1])
    assert L.ct_validate(op, bad_threads) == L.S_INVALID
    assert "threads" in L.ct_last_error()
    # LDS: on a 7x7-filter op, a 14 x 32 output tile with 32-channel chunks needs
    # a 32 x 20 x 38 halo plus a 32 x 32 x 49 filter chunk: 297 KiB > 160 KiB
    big = W.Op("big7", 1, 64, 56, 56, 64, 7, 7, 1, 1, 3, 3)
    bad_lds = L.make_schedule(1, [14, 32, 32, 8, 4, 1, 32, 1, 1])
    assert L.ct_validate(big, bad_lds) == L.S_INVALID
    assert "LDS" in L.ct_last_error()
    # a bf16 family on an fp32 op
    assert L.ct_validate(op, L.make_schedule(3, [16, 1, 1, 1, 1, 32, 0, 1, 0])) == L.S_INVALID
    # a knob value outside the table
    assert L.ct_validate(op, L.make_schedule(1, [3, 8, 8, 1, 1, 0, 8, 1, 1])) == L.S_INVALID
    # split that leaves an empty channel range (64 channels, ct 32 -> 2 chunks, split 4)
    assert L.ct_validate(op, L.make_schedule(1, [4, 8, 16, 2, 1, 0, 32, 4, 1])) == L.S_INVALID
    # the MFMA families store through 32-bit buffer offsets: an output of 2^31
    # bytes or more is refused (here 2^29 + 2^21 fp32 elements, inputs small)
    big_y = W.Op("big_y", 1, 8, 363, 363, 4096, 1, 1, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC)
    assert L.ct_validate(big_y, L.make_schedule(3, [16, 1, 1, 1, 1, 32, 0, 1, 0])) == L.S_INVALID
    assert "output too large" in L.ct_last_error()
    big_y32 = W.Op("big_y32", 1, 16, 363, 363, 4096, 1, 1)
    assert L.ct_validate(big_y32, L.make_schedule(4, [16, 1, 1, 1, 4, 1, 32, 16, 1, 1])) == L.S_INVALID
    assert "output too large" in L.ct_last_error()
    # malformed op
    with pytest.raises(L.CtError):
        L.ct_validate(W.Op("bad", 1, 3, 4, 4, 5, 3, 3, groups=2), bad_threads)


def test_bf16_block_renumbering_is_a_bijection_into_xcd_bands():
    # the kernel's own function, through the library: every tile is taken by
    # exactly one block, and the blocks that run on one XCD (b mod 8) take one
    # contiguous band of tiles, in block order
    for tiles in (1, 7, 8, 9, 63, 64, 65, 196, 1000):
        got = L.ct_test_xcd_band(tiles)
        assert sorted(got.tolist()) == list(range(tiles))
        for x in range(8):
            band = got[x::8].tolist()
            assert band == list(range(band[0], band[0] + len(band))) if band else True


def test_median_rule():
    assert HR.median([3, 1, 2]) == 2
    assert HR.median([4, 1, 2, 3]) == np.float32(2.5)


def test_degenerate_ops_are_refused_at_the_boundary():
    """An op with no work (zero batch, an output with no pixels) or an
    impossible grouping is an argument error, not an empty candidate list."""
    some = L.ct_sample(W.conv("ok", 1, 4, 8, 8, 3, 1), 0, 0, 0, 1)[0]
    bad = [W.Op("n0", 0, 4, 8, 8, 4, 3, 3, 1, 1, 1, 1, 1, 1, 1, 0, 0),
           W.Op("c0", 1, 0, 8, 8, 4, 3, 3, 1, 1, 1, 1, 1, 1, 1, 0, 0),
           W.Op("no_output", 1, 4, 2, 2, 4, 5, 5, 1, 1, 0, 0, 1, 1, 1, 0, 0),
           W.Op("stride0", 1, 4, 8, 8, 4, 3, 3, 0, 1, 1, 1, 1, 1, 1, 0, 0),
           W.Op("groups", 1, 6, 8, 8, 4, 3, 3, 1, 1, 1, 1, 1, 1, 4, 0, 0)]
    for op in bad:
        with pytest.raises(L.CtError) as e:
            L.ct_validate(op, some)
        assert e.value.code == -1, op.name
        with pytest.raises(L.CtError):
            L.ct_valid_space(op)
