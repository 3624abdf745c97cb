"""Seeded synthetic inputs shared by the GPU path and the oracle's tests.

This module only *draws numbers*: it holds none of the convolution or tuning
arithmetic. Both sides of every parity check receive the arrays made here.

Generator: splitmix64 (Steele, Lea and Flood, "Fast splittable pseudorandom
number generators", OOPSLA 2014; Vigna's public-domain reference code).
One independent stream per (tensor, layer):

    state0 = seed ^ (GAMMA * (1 + config_id) mod 2^64) ^ (tag << 32) ^ layer_id

and the first output of the stream is discarded. Value recipes:

* ``uniform``  U(-1,1): u = (z >> 11) * 2^-53, v = 2u - 1, rounded to fp32.
* ``normal``   N(0,1): Box-Muller on two draws, v = sqrt(-2 ln(1-u1)) cos(2 pi u2).
* ``int``      integers in [-m, m]: v = (z >> 33) mod (2m+1) - m.

bf16 tensors are drawn in fp32 first and then rounded to nearest-even bf16.
Tensors are filled in the memory order of their layout.
"""
from __future__ import annotations

import numpy as np

GAMMA = 0x9E3779B97F4A7C15
_M1 = 0xBF58476D1CE4E5B9
_M2 = 0x94D049BB133111EB
MASK64 = (1 << 64) - 1

TAG_X = 1
TAG_W = 2


def stream_state(seed: int, config_id: int, tag: int, layer_id: int) -> int:
    """Initial splitmix64 state of the stream for (seed, config, tensor tag, layer)."""
    return (seed ^ ((GAMMA * (1 + config_id)) & MASK64) ^ ((tag << 32) & MASK64) ^ layer_id) & MASK64


def splitmix64_block(state0: int, count: int, skip: int = 1) -> np.ndarray:
    """Outputs skip+1 .. skip+count of the splitmix64 stream that starts at state0.

    The k-th call (k = 1, 2, ...) mixes state0 + k*GAMMA, so any window of the
    stream can be produced without a loop.
    """
    out = np.empty(count, dtype=np.uint64)
    chunk = 1 << 20  # in place, a chunk at a time: large tensors stay cache- and memory-friendly
    t = np.empty(min(chunk, max(count, 1)), dtype=np.uint64)
    with np.errstate(over="ignore"):
        for b in range(0, count, chunk):
            z = out[b:b + chunk]
            tt = t[:len(z)]
            z[:] = np.arange(skip + 1 + b, skip + 1 + b + len(z), dtype=np.uint64)
            z *= np.uint64(GAMMA)
            z += np.uint64(state0)
            np.right_shift(z, np.uint64(30), out=tt)
            z ^= tt
            z *= np.uint64(_M1)
            np.right_shift(z, np.uint64(27), out=tt)
            z ^= tt
            z *= np.uint64(_M2)
            np.right_shift(z, np.uint64(31), out=tt)
            z ^= tt
    return out


def _unit(z: np.ndarray) -> np.ndarray:
    return (z >> np.uint64(11)).astype(np.float64) * (2.0 ** -53)


def draw(shape, dist: str, seed: int, config_id: int, tag: int, layer_id: int,
         int_range: int = 2) -> np.ndarray:
    """An fp32 array of the given shape, filled in C order from its own stream."""
    count = int(np.prod(shape))
    s0 = stream_state(seed, config_id, tag, layer_id)
    if dist == "uniform":
        z = splitmix64_block(s0, count)
        z >>= np.uint64(11)
        v = z.astype(np.float64)
        del z
        v *= 2.0 ** -52  # 2 * (z >> 11) * 2^-53, exact
        v -= 1.0
    elif dist == "normal":
        z = splitmix64_block(s0, 2 * count)
        u1 = _unit(z[0::2])
        u2 = _unit(z[1::2])
        v = np.sqrt(-2.0 * np.log1p(-u1)) * np.cos(2.0 * np.pi * u2)
    elif dist == "int":
        m = int(int_range)
        z = splitmix64_block(s0, count)
        v = ((z >> np.uint64(33)) % np.uint64(2 * m + 1)).astype(np.int64) - m
        v = v.astype(np.float64)
    elif dist == "ones":
        v = np.ones(count, dtype=np.float64)
    else:
        raise ValueError(f"unknown distribution {dist!r}")
    return v.astype(np.float32).reshape(shape)


def round_to_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returned as fp32."""
    bits = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = np.uint64(0x7FFF) + ((bits >> np.uint64(16)) & np.uint64(1))
    r = ((bits + bias) >> np.uint64(16)) << np.uint64(16)
    return r.astype(np.uint32).view(np.float32).reshape(a.shape)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of already-bf16-valued fp32 data, as uint16 (the bf16 encoding)."""
    bits = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    return (bits >> np.uint32(16)).astype(np.uint16)


def conv_inputs(x_shape, w_shape, dist: str, seed: int, config_id: int, layer_id: int,
                bf16: bool = False, int_range: int = 2):
    """x and w for one layer, each from its own stream (tags 1 and 2)."""
    x = draw(x_shape, dist, seed, config_id, TAG_X, layer_id, int_range)
    w = draw(w_shape, dist, seed, config_id, TAG_W, layer_id, int_range)
    if bf16:
        x = round_to_bf16(x)
        w = round_to_bf16(w)
    return x, w
