"""Number formats, decoded from their definitions (oracle; test infrastructure only).

* IEEE 754 binary16: 1 sign bit, 5 exponent bits (bias 15), 10 fraction bits.
  The fp16 block scale of the GGUF Q8_0 / Q4_0 formats is stored this way,
  little-endian.  Subnormals, signed zero and negative scales are legal.
* bfloat16: the upper half of a binary32 (8 exponent bits, 7 fraction bits);
  round-to-nearest-even from the real value.  Used only by the prefill
  variant, whose MFMA tiles hold bf16 operands.
"""
import numpy as np


def fp16_decode(bits):
    """Exact fp64 value of each binary16 bit pattern (uint16 array or int)."""
    b = np.asarray(bits, dtype=np.int64)
    sign = np.where((b >> 15) & 1, -1.0, 1.0)
    expo = (b >> 10) & 0x1F
    frac = (b & 0x3FF).astype(np.float64)
    normal = sign * np.ldexp(1.0 + frac / 1024.0, (expo - 15).astype(np.int64))
    subnormal = sign * np.ldexp(frac / 1024.0, -14)
    special = np.where(frac == 0, sign * np.inf, np.nan)
    out = np.where(expo == 0, subnormal, np.where(expo == 31, special, normal))
    return out if out.ndim else float(out)


def bf16_round(x):
    """Round each real value (fp64 array) to the nearest bfloat16, ties to even.

    Written from the format: a finite nonzero v = m * 2**e with 0.5 <= |m| < 1;
    bf16 keeps 8 significant bits, so v is rounded to a multiple of
    2**(e-8) (normal range), or of 2**-133 below the smallest normal 2**-126.
    Values past the largest finite bf16 round to +-inf.
    """
    v = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(v)
    e = np.maximum(e, -125)                   # subnormal bf16 spacing is 2**-133
    step = np.ldexp(1.0, e - 8)
    r = np.rint(v / step) * step              # np.rint rounds half to even
    big = np.abs(r) >= 2.0 ** 128
    r = np.where(big, np.copysign(np.inf, v), r)
    return np.where(np.isfinite(v), r, v)
