"""The decode kernels' in-place code extraction is exact (CPU check of the
arithmetic the dequantization relies on; no GPU).

A code q of `bits` bits masked at bit offset o of a 16-bit half, or'ed with
0x6400, is the fp16 value 1024 + 2^o q.  The kernel recovers q - z as
(1024 + 2^o q) * 2^-o + (-(1024 / 2^o + z)) with one fused multiply-add.  The
product is then 1024 / 2^o + q and the sum q - z, both exactly representable,
so the fused operation rounds nothing, and the result matches the plain
subtraction (1024 + q) - (1024 + z) used for o = 0.
"""
import itertools

import numpy as np
import pytest


def f16(bits: int) -> float:
    return float(np.array([bits], np.uint16).view(np.float16)[0])


def exact_f16(x: float) -> bool:
    return float(np.float16(x)) == x


@pytest.mark.parametrize("bits,offsets", [(4, (0, 4)), (2, (0, 2, 4, 6))])
def test_in_place_extraction_is_exact(bits, offsets):
    m = (1 << bits) - 1
    for o, q, z in itertools.product(offsets, range(m + 1), range(m + 1)):
        x = f16(0x6400 | (q << o))
        assert x == 1024 + (1 << o) * q                 # the masked pattern is the fp16 integer
        scale = 2.0 ** -o
        c = (1024.0 - 1024.0 / (1 << o)) - (1024.0 + z)  # the kernel forms -(1024/2^o + z) from 1024 + z
        assert exact_f16(scale) and exact_f16(1024.0 + z) and exact_f16(1024.0 - 1024.0 / (1 << o))
        assert exact_f16(c) and c == -(1024.0 / (1 << o) + z)
        prod = x * scale                                 # exact real product
        assert exact_f16(prod) and prod == 1024.0 / (1 << o) + q
        r = prod + c                                     # the fused result before rounding
        assert exact_f16(r) and r == q - z
        # the same value as the plain path, signed zero included
        plain = np.float16(f16(0x6400 | q)) - np.float16(1024.0 + z)
        assert float(plain) == r and np.signbit(plain) == np.signbit(np.float16(r))
