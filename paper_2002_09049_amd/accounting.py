"""Memory and operation counts of a quantized network (Sec. 3.4, Table 1,
and the OP convention of the experiments, Sec. 5).

Per output channel of d weights with N-bit codes (Table 1):

    naive       memory d N bits          multiplications d N^2 binary ops
    multipoint  memory n d N + 32 n bits multiplications n (d N^2 + 32^2)

(n points; each point has d codes and one 32-bit integer scale A_i, and each
output takes n dot products plus n 32-bit x 32-bit products with the A_i).
With weight bits w and activation bits a the dot product's binary ops are
d w a.  One OP is one 8-bit x 8-bit multiplication, 64 binary ops, so an
m-bit x n-bit product counts m n / 64 OPs; additions are not counted.  An
output channel of a conv layer produces hw outputs per image.

Host arithmetic only (no device work).  Sizes are returned in bytes; the
paper's "MB" are 2^20 bytes and its M / G of OPs are 10^6 / 10^9.
"""
from __future__ import annotations

from typing import Dict, Optional, Sequence, Tuple

import numpy as np

Layer = Tuple[int, int, int]   # (C_out, d, output positions per image)


def channel_memory_bits(d: int, wbits: int, n: Optional[int] = None) -> int:
    """Table 1, memory of one channel: d N (naive, n is None) or n d N + 32 n."""
    return d * wbits if n is None else n * d * wbits + 32 * n


def channel_mul_binops(d: int, wbits: int, abits: int, n: Optional[int] = None) -> int:
    """Table 1, binary ops of the multiplications of one output: d w a
    (naive) or n (d w a + 32^2) (multipoint)."""
    return d * wbits * abits if n is None else n * (d * wbits * abits + 32 * 32)


def network_cost(layers: Sequence[Layer], wbits: int, abits: int,
                 counts: Optional[Sequence[np.ndarray]] = None) -> Dict[str, float]:
    """Size and OPs per image of the listed layers.

    counts: None (naive quantization) or one int array of per-channel point
    counts per layer (multipoint).  Returns bytes of the quantized weights,
    bytes at fp32, and OPs (binary ops / 64)."""
    bits = 0
    fp_bits = 0
    binops = 0
    for li, (C, d, hw) in enumerate(layers):
        fp_bits += 32 * C * d
        if counts is None:
            bits += C * channel_memory_bits(d, wbits)
            binops += C * hw * channel_mul_binops(d, wbits, abits)
        else:
            n = np.asarray(counts[li], dtype=np.int64)
            assert n.shape == (C,)
            tot = int(n.sum())
            bits += tot * d * wbits + 32 * tot
            binops += hw * tot * (d * wbits * abits + 32 * 32)
    return {"bytes": bits / 8.0, "fp32_bytes": fp_bits / 8.0, "ops": binops / 64.0}
