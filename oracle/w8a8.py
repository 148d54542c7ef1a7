"""Oracle: W8A8 linear layers (test infrastructure).

Sec. 4 (efficiency, Fig. 7) combines ISPA with W8A8 quantisation of the
linear layers and reports it as quantisation-friendly, without stating the
scheme. Reading: symmetric int8 with one scale per row,
per token for activations [n, d_in] and per output channel for the linear
weight [d_out, d_in];

    scale = absmax(row) / 127   (1 for an all-zero row)
    code  = clamp(round_half_even(x / scale), -127, 127)

with the division and the rounding in float32. The product of codes is exact
in integers and is dequantised as float32(acc) * scale_a * scale_w, in that
order, one IEEE float32 operation at a time.
"""

import numpy as np


def quantize_rows(x):
    """int8 codes and float32 scales of each row of ``x`` (float32 values)."""
    x = np.asarray(x, dtype=np.float32)
    amax = np.max(np.abs(x), axis=1)
    scale = np.where(amax > 0, (amax / np.float32(127.0)).astype(np.float32), np.float32(1.0)).astype(np.float32)
    q = np.rint((x / scale[:, None]).astype(np.float32))
    q = np.clip(q, -127, 127).astype(np.int8)
    return q, scale


def dequantize_rows(q, scale):
    return np.asarray(q, dtype=np.float32) * np.asarray(scale, dtype=np.float32)[:, None]


def project_w8a8(qa, sa, qw, sw):
    """y = (q_a q_w^T) * s_a * s_w for codes q_a [n, d_in], q_w [d_out, d_in]."""
    acc = np.asarray(qa, dtype=np.int64) @ np.asarray(qw, dtype=np.int64).T
    y = acc.astype(np.float32) * np.asarray(sa, dtype=np.float32)[:, None]
    return (y * np.asarray(sw, dtype=np.float32)[None, :]).astype(np.float32)
