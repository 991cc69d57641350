"""A second, independent implementation of the group quantizer, in NumPy
float32, used to pin the C oracle's quantizer bit for bit.

It shares nothing with ``oracle/jf_oracle.c``: fp16 rounding here is integer
arithmetic on the binary32 significand and exponent (the definition of
rounding a binary32 value to the binary16 grid), not a bisection over fp16
bit patterns, and min/max use an integer total-order key.  The arithmetic
steps are the encoding's: binary32 subtraction of the rounded bias, binary32
IEEE division by the rounded scale, round half to even, clamp to 0..15
(affine 4-bit with a scale and an offset per group: the paper's Introduction,
four-bit weights; the readings that fix each step are listed with the
oracle).
"""
from __future__ import annotations

import numpy as np

F16_MAX = 65504.0


def _bit_length(m: np.ndarray) -> np.ndarray:
    """Bit length of non-negative int64 values below 2^25 (0 for 0)."""
    out = np.zeros(m.shape, np.int64)
    v = m.copy()
    for sh in (16, 8, 4, 2, 1):
        big = v >= (np.int64(1) << sh)
        out += np.where(big, sh, 0)
        v = np.where(big, v >> sh, v)
    return out + (v > 0)


def round_f32_to_f16(f: np.ndarray, mode: str) -> np.ndarray:
    """Round finite binary32 values to binary16.

    mode "even": to nearest, ties to an even last bit; "down": toward -inf;
    "up": toward +inf.  Beyond the largest finite fp16 (65504) nearest
    rounding gives infinity from 65520 up, "up" gives infinity for anything
    above 65504, "down" stays at 65504 (mirrored for negative values)."""
    f = np.ascontiguousarray(f, np.float32)
    bits = f.view(np.uint32).astype(np.int64)
    neg = (bits >> 31) == 1
    e = (bits >> 23) & 0xFF
    frac = bits & 0x7FFFFF
    M = np.where(e > 0, frac | (1 << 23), frac)     # |f| = M * 2^E exactly
    E = np.maximum(e, 1) - 150
    top = E + _bit_length(M) - 1                     # floor(log2 |f|)
    Q = np.maximum(top - 10, -24)                    # fp16 quantum at |f|
    s = Q - E                                        # right shift to that quantum
    sp = np.clip(s, 0, 62)
    fl = np.where(s > 0, M >> sp, M << np.clip(-s, 0, 62))
    rem = np.where(s > 0, M - (fl << sp), 0)
    half = np.where(s > 0, np.int64(1) << np.clip(sp - 1, 0, 62), 1)
    # which way the magnitude goes
    if mode == "even":
        up = (rem > half) | ((rem == half) & (s > 0) & ((fl & 1) == 1))
        to_inf = np.ones(f.shape, bool)
    elif mode in ("down", "up"):
        mag_up = neg if mode == "down" else ~neg
        up = mag_up & (rem > 0)
        to_inf = mag_up
    else:
        raise ValueError(mode)
    mag = (fl + up).astype(np.float64) * np.exp2(Q.astype(np.float64))
    mag = np.where(mag > F16_MAX, np.where(to_inf, np.inf, F16_MAX), mag)
    mag = np.where(M == 0, 0.0, mag)
    out = np.where(neg, -mag, mag)
    return out.astype(np.float16)  # exact: every value here is on the fp16 grid


def _total_order_key(x32: np.ndarray) -> np.ndarray:
    """Integer key ordered like the values, with -0 below +0."""
    b = x32.view(np.int32).astype(np.int64)
    return np.where(b < 0, b ^ 0x7FFFFFFF, b)


def quantize_groups(x: np.ndarray):
    """x fp16 [n][G] -> (codes uint8 [n][G], scales fp16 [n], biases fp16 [n])."""
    x = np.ascontiguousarray(x, np.float16)
    x32 = x.astype(np.float32)                       # exact
    key = _total_order_key(x32)
    rows = np.arange(x.shape[0])
    mn = x32[rows, np.argmin(key, axis=1)]
    mx = x32[rows, np.argmax(key, axis=1)]
    bias = round_f32_to_f16(mn, "down")
    rng = (mx - mn).astype(np.float32)               # binary32 subtraction
    step = (rng / np.float32(15.0)).astype(np.float32)  # binary32 IEEE division
    scale = np.where(rng == 0, np.float16(0.0), round_f32_to_f16(step, "up"))
    s32 = scale.astype(np.float32)
    b32 = bias.astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        diff = (x32 - b32[:, None]).astype(np.float32)
        r = (diff / s32[:, None]).astype(np.float32)
    q = np.clip(np.rint(r), 0.0, 15.0)
    q = np.where((s32 == 0)[:, None], 0.0, q)
    return q.astype(np.uint8), scale.astype(np.float16), bias.astype(np.float16)
