"""Pins of the fp64 oracle against facts that do not come from the oracle itself.

* exact rational brute force in the scatter form (tiny shapes, all options),
* a library special case: torch's float64 CPU conv2d on every task shape,
* closed forms: delta filter, all-ones input (interior and border),
* linearity in x and in w, 1x1 = matrix product, integer exactness,
* layout consistency (NHWC = transposed NCHW), thread-count independence.
"""
import itertools
import random

import numpy as np
import pytest
import torch

import oracle
from oracle.brute import conv2d_scatter
from paper_2008_03602_amd import synth, workloads as W


def _tiny_cases(seed=1234, count=160):
    rng = random.Random(seed)
    cases = []
    while len(cases) < count:
        N = rng.choice([1, 2])
        C = rng.choice([1, 2, 3])
        groups = rng.choice([1, C])
        K = groups * rng.choice([1, 2]) if groups > 1 else rng.choice([1, 2, 3])
        H, Wd = rng.randint(1, 6), rng.randint(1, 6)
        R, S = rng.randint(1, 3), rng.randint(1, 3)
        st = (rng.choice([1, 2]), rng.choice([1, 2]))
        pd = (rng.choice([0, 1, 2]), rng.choice([0, 1, 2]))
        dl = (rng.choice([1, 1, 2]), rng.choice([1, 1, 2]))
        OH = (H + 2 * pd[0] - dl[0] * (R - 1) - 1) // st[0] + 1
        OW = (Wd + 2 * pd[1] - dl[1] * (S - 1) - 1) // st[1] + 1
        if OH <= 0 or OW <= 0:
            continue
        cases.append((N, C, H, Wd, K, R, S, st, pd, dl, groups))
    return cases


def _rand_dyadic(rng, shape):
    # multiples of 1/8 in [-2, 2]: every product and sum is exact in fp64
    return np.array([rng.randint(-16, 16) / 8.0 for _ in range(int(np.prod(shape)))]).reshape(shape)


@pytest.mark.parametrize("case", _tiny_cases())
def test_brute_force_exact(case):
    N, C, H, Wd, K, R, S, st, pd, dl, groups = case
    rng = random.Random(hash(case) & 0xFFFF)
    x = _rand_dyadic(rng, (N, C, H, Wd))
    w = _rand_dyadic(rng, (K, C // groups, R, S))
    ref = np.array(conv2d_scatter(x.tolist(), w.tolist(), N, C, H, Wd, K, R, S, st, pd, dl, groups),
                   dtype=np.float64)
    y = oracle.conv2d(x, w, st, pd, dl, groups)
    assert y.shape == ref.shape
    assert np.array_equal(y, ref)
    # the NHWC layout gives the same numbers, transposed
    y2 = oracle.conv2d(x.transpose(0, 2, 3, 1), w.transpose(0, 2, 3, 1), st, pd, dl, groups,
                       layout="nhwc")
    assert np.array_equal(y2, ref.transpose(0, 2, 3, 1))


def _task_ops():
    return W.resnet18(1) + W.resnet50(1)[:6] + W.mobilenet_v2_depthwise(1)[:4]


@pytest.mark.parametrize("op", _task_ops(), ids=lambda o: o.name)
def test_matches_torch_float64(op):
    x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), "uniform", 7, 2, 3)
    y = oracle.conv2d(x, w, (op.stride_h, op.stride_w), (op.pad_h, op.pad_w), (op.dil_h, op.dil_w),
                      op.groups, threads=8)
    t = torch.nn.functional.conv2d(torch.from_numpy(x.astype(np.float64)),
                                   torch.from_numpy(w.astype(np.float64)), None,
                                   (op.stride_h, op.stride_w), (op.pad_h, op.pad_w),
                                   (op.dil_h, op.dil_w), op.groups).numpy()
    assert y.shape == t.shape == op.y_shape()
    assert np.max(np.abs(y - t)) <= 1e-12 * max(np.max(np.abs(t)), 1.0)


@pytest.mark.parametrize("C,K,H,R,stride,groups", [(3, 6, 9, 3, 1, 1), (4, 4, 8, 3, 2, 4),
                                                   (2, 4, 7, 5, 1, 1), (5, 5, 6, 3, 1, 5),
                                                   (3, 3, 11, 7, 2, 1)])
def test_delta_filter_reproduces_input(C, K, H, R, stride, groups):
    x = synth.draw((2, C, H, H + 1), "uniform", 1, 0, 1, 0).astype(np.float64)
    Cg = C // groups
    w = np.zeros((K, Cg, R, R))
    for k in range(K):
        c_src = k % C
        if groups > 1:
            assert (c_src // Cg) == k // (K // groups)
        w[k, c_src % Cg, R // 2, R // 2] = 1.0
    y = oracle.conv2d(x, w, (stride, stride), (R // 2, R // 2), (1, 1), groups)
    for k in range(K):
        assert np.array_equal(y[:, k], x[:, k % C, ::stride, ::stride])


@pytest.mark.parametrize("H,Wd,R,S,pad,stride", [(8, 9, 3, 3, 1, 1), (10, 7, 3, 5, 2, 2),
                                                  (6, 6, 1, 1, 0, 1), (12, 12, 7, 7, 3, 2)])
def test_all_ones_input_closed_form(H, Wd, R, S, pad, stride):
    C, K = 3, 4
    x = np.ones((1, C, H, Wd))
    w = synth.draw((K, C, R, S), "uniform", 3, 0, 2, 0).astype(np.float64)
    y = oracle.conv2d(x, w, (stride, stride), (pad, pad))
    OH, OW = y.shape[2:]
    for p in range(OH):
        for q in range(OW):
            rows = [r for r in range(R) if 0 <= p * stride - pad + r < H]
            cols = [t for t in range(S) if 0 <= q * stride - pad + t < Wd]
            expect = w[:, :, rows][:, :, :, cols].sum(axis=(1, 2, 3))
            interior = len(rows) == R and len(cols) == S
            if interior:
                assert np.allclose(y[0, :, p, q], w.sum(axis=(1, 2, 3)), rtol=0, atol=1e-13)
            assert np.allclose(y[0, :, p, q], expect, rtol=0, atol=1e-13)


def test_linearity():
    op = W.resnet18(1)[3]  # 64->128 3x3 s2
    x1, w1 = (t.astype(np.float64) for t in synth.conv_inputs(op.x_shape(), op.w_shape(), "normal", 1, 9, 0))
    x2, w2 = (t.astype(np.float64) for t in synth.conv_inputs(op.x_shape(), op.w_shape(), "normal", 2, 9, 0))
    kw = dict(stride=(2, 2), pad=(1, 1), threads=8)
    a, b = 0.75, -1.5
    lhs = oracle.conv2d(a * x1 + b * x2, w1, **kw)
    rhs = a * oracle.conv2d(x1, w1, **kw) + b * oracle.conv2d(x2, w1, **kw)
    assert np.max(np.abs(lhs - rhs)) <= 1e-12 * np.max(np.abs(rhs))
    lhs = oracle.conv2d(x1, a * w1 + b * w2, **kw)
    rhs = a * oracle.conv2d(x1, w1, **kw) + b * oracle.conv2d(x1, w2, **kw)
    assert np.max(np.abs(lhs - rhs)) <= 1e-12 * np.max(np.abs(rhs))


@pytest.mark.parametrize("layout", ["nchw", "nhwc"])
def test_pointwise_is_matrix_product(layout):
    N, C, H, K = 2, 24, 7, 40
    x = synth.draw((N, C, H, H), "uniform", 5, 0, 1, 0).astype(np.float64)
    w = synth.draw((K, C, 1, 1), "uniform", 5, 0, 2, 0).astype(np.float64)
    ref = np.einsum("kc,nchw->nkhw", w[:, :, 0, 0], x)
    if layout == "nchw":
        y = oracle.conv2d(x, w)
    else:
        y = oracle.conv2d(x.transpose(0, 2, 3, 1), w.transpose(0, 2, 3, 1), layout="nhwc")
        y = y.transpose(0, 3, 1, 2)
    assert np.max(np.abs(y - ref)) <= 1e-13 * np.max(np.abs(ref))


def test_integer_inputs_give_exact_integers():
    op = W.resnet18(1)[10]  # 512->512 3x3 at 7x7: the longest reduction (4608 taps)
    x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), "int", 0, 1, 10, int_range=2)
    y = oracle.conv2d(x, w, (1, 1), (1, 1), threads=8)
    assert np.array_equal(y, np.round(y))
    # compare with exact integer arithmetic through int64 im2col
    xi = np.pad(x.astype(np.int64), ((0, 0), (0, 0), (1, 1), (1, 1)))
    cols = np.stack([xi[0, :, r:r + 7, t:t + 7] for r in range(3) for t in range(3)], axis=1)
    ref = np.einsum("kcj,cjpq->kpq", w.astype(np.int64).reshape(512, 512, 9), cols)
    assert np.array_equal(y[0].astype(np.int64), ref)


def test_thread_count_does_not_change_result():
    op = W.resnet50(1)[1]
    x, w = synth.conv_inputs(op.x_shape(), op.w_shape(), "normal", 0, 4, 1)
    y1 = oracle.conv2d(x, w, (1, 1), (1, 1), threads=1)
    y8 = oracle.conv2d(x, w, (1, 1), (1, 1), threads=8)
    assert np.array_equal(y1, y8)


def test_abs_bound_output():
    x = synth.draw((1, 5, 9, 9), "normal", 0, 0, 1, 0)
    w = synth.draw((6, 5, 3, 3), "normal", 0, 0, 2, 0)
    y, a = oracle.conv2d(x, w, (1, 1), (1, 1), with_abs=True)
    a2 = oracle.conv2d(np.abs(x), np.abs(w), (1, 1), (1, 1))
    assert np.array_equal(a, a2)
    assert np.all(a >= np.abs(y))


def test_out_size_and_rejects_bad_shapes():
    assert oracle.out_size(224, 3, 1, 7, 2) == 112
    assert oracle.out_size(56, 0, 1, 1, 2) == 28
    assert oracle.out_size(2, 0, 1, 3, 1) == 0
    with pytest.raises(ValueError):
        oracle.conv2d(np.zeros((1, 3, 4, 4)), np.zeros((4, 2, 3, 3)), groups=1)
