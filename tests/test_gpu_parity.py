"""GPU parity of every kernel family against the fp64 oracle, through the C ABI.

Shapes are small enough for the oracle to finish in seconds but span several
tiles with ragged tails (H, W, K and C not multiples of the tile sizes, C = 3,
stride 2, 7x7 filters). Each case runs a seeded sample of schedules from the
op's valid candidate space.
"""
import random

import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, workloads as W
from gpu_util import check_close, device_ready, make_inputs, note, reference, sched_str, to_device

pytestmark = pytest.mark.gpu

F32_OPS = [
    W.conv("odd3x3", 1, 5, 13, 11, 3, 1),
    W.conv("odd3x3s2", 2, 6, 15, 9, 3, 2),
    W.conv("stem7x7", 1, 3, 29, 10, 7, 2, 3),
    W.conv("pw_odd", 2, 19, 9, 21, 1, 1, 0),
    W.conv("pw_s2", 1, 24, 14, 40, 1, 2, 0),
    W.Op("rect5x3", 1, 7, 12, 17, 12, 5, 3, 1, 2, 2, 1, 1, 1, 1, 0, 0),
    W.Op("dilated", 1, 4, 11, 11, 6, 3, 3, 1, 1, 2, 2, 2, 2, 1, 0, 0),
]
DW_OPS = [
    W.conv("dw_odd", 2, 13, 15, 13, 3, 1, 1, groups=13),
    W.conv("dw_s2", 3, 24, 17, 24, 3, 2, 1, groups=24),
    W.Op("dw5x5", 1, 8, 10, 10, 8, 5, 5, 1, 1, 2, 2, 1, 1, 8, 0, 0),
]
# shapes where IGEMM_F32 copies 16 bytes per lane (W a multiple of 4), with ragged tiles
VEC_OPS = [
    W.conv("vec3x3", 1, 24, 20, 40, 3, 1),
    W.conv("vec3x3s2", 1, 16, 28, 24, 3, 2),
    W.conv("vec1x1", 2, 32, 12, 20, 1, 1, 0),
    W.Op("vec_rect", 2, 12, 9, 24, 20, 3, 3, 1, 1, 1, 1, 1, 1, 1, 0, 0),
]
BF_OPS = [
    W.conv("pwbf_odd", 2, 24, 9, 40, 1, 1, 0, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC),
    W.conv("pwbf_c96", 1, 96, 11, 24, 1, 1, 0, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC),
    W.conv("pwbf_s2", 1, 40, 13, 72, 1, 2, 0, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC),
]


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _run_sample(op, n_sched, seed, dist="uniform", int_range=2, exact=False, family=None):
    x, w = make_inputs(op, dist, seed=seed, int_range=int_range)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    if family is None:
        scheds = L.ct_sample(op, seed, 99, 0, n_sched)
    else:  # a seeded sample of one family's valid schedules
        space = [s for s in L.ct_valid_space(op) if s.family == family]
        scheds = random.Random(seed).sample(space, min(n_sched, len(space)))
    assert len(scheds) > 0
    fams = set()
    for s in scheds:
        tag = "%s %s" % (op.name, sched_str(s))
        note(tag)
        yd.fill_(float("nan"))
        L.conv2d_run(op, s, xd, wd, yd)
        y = yd.cpu().numpy()
        split = W.split_of(s)
        if exact:
            assert np.array_equal(y.astype(np.float64), ref), tag + ": not bit-exact on integer inputs"
        else:
            check_close(op, y, ref, a, tag, split=4 if split > 1 else 1)
        fams.add(s.family)
    return fams


@pytest.mark.parametrize("op", F32_OPS, ids=lambda o: o.name)
def test_fp32_families_match_oracle(op):
    fams = _run_sample(op, 24, seed=11)
    assert fams <= {W.FAM_DIRECT_F32, W.FAM_IGEMM_F32}


@pytest.mark.parametrize("op", F32_OPS + VEC_OPS, ids=lambda o: o.name)
def test_fp32_mfma_schedules_match_oracle(op):
    # 24 schedules of the MFMA family alone: both staging depths, 1- and
    # 16-byte copies, register double buffering, reduction groups and splits
    assert _run_sample(op, 24, seed=14, family=W.FAM_IGEMM_F32) == {W.FAM_IGEMM_F32}


def test_misaligned_tensors_are_refused_by_16_byte_schedules():
    op = VEC_OPS[0]
    x, w = make_inputs(op, "uniform", seed=3)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    buf = torch.empty(xd.numel() + 4, dtype=torch.float32, device=xd.device)
    xm = buf[1:1 + xd.numel()].view(op.x_shape())  # 4 bytes past a 16-byte boundary
    xm.copy_(xd)
    space = L.ct_valid_space(op)
    vec = next(s for s in space if s.family == W.FAM_IGEMM_F32)
    direct = next(s for s in space if s.family == W.FAM_DIRECT_F32)
    note("misaligned x: " + sched_str(vec))
    with pytest.raises(L.CtError) as e:
        L.conv2d_run(op, vec, xm, wd, yd)
    assert e.value.code == L.CT_E_ARG and "aligned" in str(e.value)
    lat, st = L.measure_candidates_mask(op, [vec, direct], L.ct_cu_mask(1.0, 0), L.make_opts(1, 1, 2, 2),
                                        xm, wd, yd)
    assert list(st) == [L.S_LAUNCH, L.S_OK]
    yd.fill_(float("nan"))
    L.conv2d_run(op, direct, xm, wd, yd)
    check_close(op, yd.cpu().numpy(), ref, a, "misaligned x, direct schedule")


@pytest.mark.parametrize("op", DW_OPS, ids=lambda o: o.name)
def test_depthwise_matches_oracle(op):
    _run_sample(op, 24, seed=12)


# 3x3 pad-1 depthwise shapes for the 4-columns-per-thread variant: 16-byte
# loads and stores (W a multiple of 4, W = stride * OW, OW a multiple of 4),
# and the word-by-word fallback (odd widths, W != 2 OW), with ragged tiles
Q4_OPS = [
    W.conv("dwq_s1", 2, 12, 20, 12, 3, 1, 1, groups=12),
    W.conv("dwq_s2", 3, 8, 24, 8, 3, 2, 1, groups=8),
    W.conv("dwq_odd", 2, 13, 15, 13, 3, 1, 1, groups=13),
    W.conv("dwq_s2odd", 1, 6, 17, 6, 3, 2, 1, groups=6),
    W.conv("dwq_s2w14", 2, 10, 14, 10, 3, 2, 1, groups=10),
]


def _q4_sample(op, n, seed):
    space = [s for s in L.ct_valid_space(op) if s.family == W.FAM_DEPTHWISE_F32 and s.knob[8] == 1]
    assert space, op.name
    return random.Random(seed).sample(space, min(n, len(space)))


@pytest.mark.parametrize("op", Q4_OPS, ids=lambda o: o.name)
def test_depthwise_q4_matches_oracle_and_is_exact_on_integers(op):
    x, w = make_inputs(op, "uniform", seed=31)
    ref, a = reference(op, x, w)
    xi, wi = make_inputs(op, "int", seed=32)
    refi, _ = reference(op, xi, wi)
    xd, wd, yd = to_device(op, x, w)
    xid, wid, yid = to_device(op, xi, wi)
    for s in _q4_sample(op, 16, seed=33):
        tag = "%s %s" % (op.name, sched_str(s))
        note(tag)
        yd.fill_(float("nan"))
        L.conv2d_run(op, s, xd, wd, yd)
        check_close(op, yd.cpu().numpy(), ref, a, tag)
        yid.fill_(float("nan"))
        L.conv2d_run(op, s, xid, wid, yid)
        assert np.array_equal(yid.cpu().numpy().astype(np.float64), refi), tag + ": not bit-exact on integers"


@pytest.mark.parametrize("op", BF_OPS, ids=lambda o: o.name)
def test_bf16_pointwise_matches_oracle(op):
    _run_sample(op, 24, seed=13)


@pytest.mark.parametrize("op", [F32_OPS[0], F32_OPS[3], DW_OPS[0]], ids=lambda o: o.name)
def test_integer_inputs_bit_exact_fp32(op):
    _run_sample(op, 16, seed=21, dist="int", int_range=2, exact=True)


@pytest.mark.parametrize("op", [BF_OPS[0], BF_OPS[1]], ids=lambda o: o.name)
def test_integer_inputs_bit_exact_bf16(op):
    _run_sample(op, 16, seed=22, dist="int", int_range=8, exact=True)


def test_every_family_covered_on_config1_shape():
    op = W.config(1).ops[0]
    x, w = make_inputs(op, "uniform", seed=0, config_id=1)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    scheds = L.ct_sample(op, 0, 1, 0, 64)
    for s in scheds:
        note("config1 " + sched_str(s))
        yd.fill_(float("nan"))
        L.conv2d_run(op, s, xd, wd, yd)
        check_close(op, yd.cpu().numpy(), ref, a, "config1 " + sched_str(s), split=4)


def _fixed_filter(op):
    """The 1x1 / 3x3 specialisations (stride 1 or 2, no dilation, 'same' padding)."""
    sq = op.r == op.s and op.stride_h == op.stride_w and op.stride_h in (1, 2) and op.dil_h == op.dil_w == 1
    return sq and ((op.r == 1 and op.pad_h == op.pad_w == 0) or (op.r == 3 and op.pad_h == op.pad_w == 1))


def _direct_class(op, s):
    """Which operand path a direct schedule takes (mirrors the kernel's choice)."""
    toh, tow, tk, mk, mw, lds, ct, split, unr = (s.knob[i] for i in range(9))
    cols = tow // mw
    threads = (tk // mk) * toh * cols
    if not lds:
        kind = "regs-fixed" if _fixed_filter(op) else "regs"
        return kind + ("-uniform-w" if (toh * cols) % 64 == 0 else "")
    ih = (toh - 1) * op.stride_h + (op.r - 1) * op.dil_h + 1
    iw = (tow - 1) * op.stride_w + (op.s - 1) * op.dil_w + 1
    xt, wt = ct * ih * iw, tk * ct * op.r * op.s
    n_stage = max(-(-xt // threads), -(-wt // threads))
    tile = mk * mw
    # deepest register prefetch the instance allows (launch bound 512 threads
    # from 16 accumulators up, else 1024)
    cap = 16 if tile >= 16 else (0 if unr == 2 and tile >= 8 else (4 if unr == 2 and tile >= 4 else 8))
    if cap and n_stage <= cap:
        return "prefetch-%d" % next(d for d in (2, 4, 8, 16) if n_stage <= d)
    return "batch16" if n_stage >= 16 else "batch4"


@pytest.mark.parametrize("op", [W.conv("deep3x3", 1, 48, 9, 72, 3, 1), F32_OPS[1], F32_OPS[4], F32_OPS[5]],
                         ids=lambda o: o.name)
def test_direct_staging_paths_match_oracle(op):
    # every way the direct family reads its operands: registers (per-tap
    # input offsets kept resident for a fixed 1x1 or 3x3 filter) with vector
    # or scalar filter loads, LDS chunks prefetched through registers at each
    # depth (2, 4, 8, 16 elements per thread; a last chunk shorter than CT
    # where C is not a multiple of it, split channel ranges), and LDS staging
    # in batches of four or sixteen loads
    x, w = make_inputs(op, "uniform", seed=31)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    by = {}
    for s in L.ct_valid_space(op):
        if s.family == W.FAM_DIRECT_F32:
            by.setdefault(_direct_class(op, s), []).append(s)
    rng = random.Random(5)
    seen = set()
    ragged = 0
    for cls in sorted(by):
        pool = by[cls]
        # prefer schedules whose channel chunks do not divide C, then split ones
        pick = rng.sample(pool, min(3, len(pool)))
        odd = [s for s in pool if op.c % s.knob[6] and s not in pick]
        spl = [s for s in pool if s.knob[7] > 1 and s not in pick]
        pick += rng.sample(odd, min(2, len(odd))) + rng.sample(spl, min(1, len(spl)))
        for s in pick:
            tag = "%s %s [%s]" % (op.name, sched_str(s), cls)
            note(tag)
            yd.fill_(float("nan"))
            L.conv2d_run(op, s, xd, wd, yd)
            split = W.split_of(s)
            check_close(op, yd.cpu().numpy(), ref, a, tag, split=4 if split > 1 else 1)
            seen.add(cls)
            ragged += bool(op.c % s.knob[6]) and cls.startswith("prefetch")
    print(op.name, "paths:", sorted(seen), "ragged prefetched chunks:", ragged)
    if op.name == "deep3x3":
        assert {"regs-fixed", "prefetch-2", "prefetch-4", "prefetch-8", "prefetch-16", "batch4",
                "batch16"} <= seen
        assert ragged > 0


# Degenerate shapes: a one-pixel image (only the centre tap of a padded 3x3
# filter sees data), a filter as large as the image (one output pixel),
# one input and one output channel, a stride larger than the filter, a batch
# of three, and a one-row bf16 image.
DEGENERATE_OPS = [
    W.conv("one_pixel", 1, 8, 1, 8, 3, 1),
    W.Op("filter_covers_image", 1, 5, 7, 7, 6, 7, 7, 1, 1, 0, 0, 1, 1, 1, 0, 0),
    W.conv("one_channel", 2, 1, 9, 1, 3, 1),
    W.conv("stride3_1x1", 1, 12, 10, 8, 1, 3, 0),
    W.conv("batch3", 3, 16, 6, 16, 3, 1),
    W.Op("pwbf_one_row", 2, 16, 1, 9, 24, 1, 1, 1, 1, 0, 0, 1, 1, 1, W.DT_BF16, W.LAYOUT_NHWC),
]


@pytest.mark.parametrize("op", DEGENERATE_OPS, ids=lambda o: o.name)
def test_degenerate_shapes_match_oracle(op):
    fams = _run_sample(op, 12, seed=11)
    assert fams, op.name
    # every family that has a schedule for the shape, including the MFMA ones
    space_fams = {s.family for s in L.ct_valid_space(op)}
    for fam in sorted(space_fams - fams):
        _run_sample(op, 4, seed=12, family=fam)


@pytest.mark.parametrize("op", DEGENERATE_OPS, ids=lambda o: o.name)
def test_degenerate_shapes_bit_exact_on_integers(op):
    bf16 = op.dtype == W.DT_BF16
    _run_sample(op, 8, seed=13, dist="int", int_range=8 if bf16 else 2, exact=True)
