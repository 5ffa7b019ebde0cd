"""Rounding of exact float64 values to the storage precision of the projections.

The paper does not fix the numeric precision of the selector.  The projected
keys, queries and values are stored in the workload's dtype (bfloat16 or
float32), rounded once to nearest with ties to even from the exact product;
this module states that rounding from the format definitions.

bfloat16: 1 sign bit, 8 exponent bits (bias 127, same range as float32), 7
stored fraction bits.  A finite x with 2^E <= |x| < 2^(E+1) and E >= -126 is a
multiple of 2^(E-7); below the normal range the spacing is 2^-133.  Values at
or beyond 2^128 after rounding overflow to infinity.
"""
import numpy as np


def _round_bf16_frexp(x):
    # frexp: x = m * 2**e with 0.5 <= |m| < 1, so 2**(e-1) <= |x| < 2**e
    # (zero gives e = 0, and infinities and NaN pass through the scaling).
    _, e = np.frexp(x)
    # 8 significant bits: spacing 2**(e-8); never finer than the subnormal spacing.
    q_exp = np.maximum(e - 8, -133).astype(np.int32)
    r = np.ldexp(np.round(np.ldexp(x, -q_exp)), q_exp)   # np.round: half to even
    return np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, r), r)


def round_bf16(x):
    """Round float64 values to the nearest bfloat16 (ties to even), as float64.

    Inside bfloat16's normal range, [2^-126, 2^128), this keeps 7 of float64's
    52 fraction bits: add half a unit of the last kept bit (minus one, plus the
    kept bit itself, which breaks ties to even) and clear the 45 dropped bits;
    a carry out of the fraction correctly bumps the exponent.  Values outside
    that range (zero, subnormal, overflow, inf, NaN) take the frexp form.
    """
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty_like(x)
    flat_x, flat_o = x.reshape(-1), out.reshape(-1)
    step = 1 << 20                      # chunks keep the temporaries cache-resident
    for i in range(0, flat_x.size, step):
        xc = flat_x[i:i + step]
        ax = np.abs(xc)
        normal = (ax >= 2.0 ** -126) & (ax < 2.0 ** 128)
        bits = xc.view(np.uint64)
        keep = (bits >> np.uint64(45)) & np.uint64(1)
        rounded = (bits + (np.uint64((1 << 44) - 1) + keep)) & ~np.uint64((1 << 45) - 1)
        r = rounded.view(np.float64)
        r = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, r), r)
        if not normal.all():
            r = np.where(normal, r, _round_bf16_frexp(np.where(normal, 0.0, xc)))
        flat_o[i:i + step] = r
    return out


def round_f32(x):
    """Round float64 values to the nearest float32 (ties to even), as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(x, dtype: str):
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "f32":
        return round_f32(x)
    raise ValueError(f"unknown storage dtype {dtype!r}")
