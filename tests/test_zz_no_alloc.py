"""conv2d_run_noalloc against conv2d_run through the C ABI: the same schedules
give the same output bit for bit (same kernels, fixed-order split reduction),
on two calls in a row, the second on a smaller input; schedules whose split
partial sums exceed the static scratch array are refused."""
import numpy as np
import pytest
import torch

from paper_2008_03602_amd import _lib as L, workloads as W
from gpu_util import check_close, device_ready, make_inputs, note, reference, sched_str, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    device_ready()
    yield


def _split_and_plain(op, per_family=2):
    """Split-reduction schedules of every family that applies (they use the
    scratch array), plus one schedule without a split."""
    space = L.ct_valid_space(op)
    out, plain = [], None
    for fam in sorted({s.family for s in space}):
        split = [s for s in space if s.family == fam and W.split_of(s) > 1]
        out += split[::max(1, len(split) // per_family)][:per_family]
        if plain is None:
            plain = next(s for s in space if s.family == fam and W.split_of(s) == 1)
    return out + [plain]


def _run_pair(op, seed):
    x, w = make_inputs(op, "uniform", seed=seed)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    y2 = torch.full_like(yd, float("nan"))
    stream = torch.cuda.current_stream().cuda_stream
    scheds = _split_and_plain(op)
    assert any(W.split_of(s) > 1 for s in scheds)
    for s in scheds:
        tag = "%s %s" % (op.name, sched_str(s))
        note("noalloc " + tag)
        yd.fill_(float("nan"))
        L.conv2d_run(op, s, xd, wd, yd)
        y2.fill_(float("nan"))
        torch.cuda.synchronize()
        L.conv2d_run_noalloc(op, s, xd, wd, y2, stream)
        torch.cuda.synchronize()
        a1, a2 = yd.cpu().numpy(), y2.cpu().numpy()
        assert np.array_equal(a1.view(np.uint32), a2.view(np.uint32)), tag + ": outputs differ"
        check_close(op, a2, ref, a, tag, split=8)


def test_noalloc_matches_conv2d_run_then_on_a_smaller_input():
    _run_pair(W.conv("na_big", 1, 64, 56, 64, 3, 1), seed=21)   # partial sums up to 8 x 200704 floats
    _run_pair(W.conv("na_small", 1, 24, 13, 40, 3, 1), seed=22)  # the second call reads a smaller scratch range


def test_noalloc_on_the_null_stream():
    op = W.conv("na_null", 2, 128, 14, 48, 1, 1, 0, dtype=W.DT_BF16, layout=W.LAYOUT_NHWC)
    x, w = make_inputs(op, "uniform", seed=23)
    ref, a = reference(op, x, w)
    xd, wd, yd = to_device(op, x, w)
    for s in _split_and_plain(op, per_family=1):
        note("noalloc null stream " + sched_str(s))
        yd.fill_(float("nan"))
        torch.cuda.synchronize()
        L.conv2d_run_noalloc(op, s, xd, wd, yd, 0)
        torch.cuda.synchronize()
        check_close(op, yd.cpu().numpy(), ref, a, sched_str(s), split=8)


def test_noalloc_refuses_partials_beyond_the_scratch_array():
    # a 64 -> 64 3x3 layer at 300 x 300: 5.76M outputs, so a direct schedule
    # that splits the channels 4 ways needs 23M floats of partial sums, beyond
    # the array's 2^24 (the buffers are full size all the same)
    op = W.conv("na_huge", 1, 64, 300, 64, 3, 1)
    s = next(s for s in L.ct_valid_space(op) if s.family == W.FAM_DIRECT_F32 and s.knob[7] == 4)
    assert W.split_of(s) > 1
    assert 4 * 64 * 300 * 300 > L.SCRATCH_FLOATS
    xd = torch.zeros(op.x_shape(), dtype=torch.float32, device="cuda")
    wd = torch.zeros(op.w_shape(), dtype=torch.float32, device="cuda")
    yd = torch.zeros(op.y_shape(), dtype=torch.float32, device="cuda")
    with pytest.raises(L.CtError) as e:
        L.conv2d_run_noalloc(op, s, xd, wd, yd, 0)
    assert e.value.code == L.CT_E_ARG and "scratch" in str(e.value)
