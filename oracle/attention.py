"""Decode attention over a (dequantized) KV cache (oracle).

One new query per sequence attends over all cached tokens of its KV head,
the quantized prefix dequantized and the residual window exact.  Grouped
query attention: query head j reads KV head j // (Hq / H) (contiguous
grouping; the paper only says its models use GQA, Sec. 4 setup).

    out_j = softmax(q_j . K_hat^T / sqrt(d)) V_hat      (fp64, max-subtracted)
"""
import math

import numpy as np


def decode_attention(q, keys, values, scale=None):
    """q: [G][d] queries sharing one KV head; keys, values: [T][d].
    Returns out [G][d] float64."""
    q = np.asarray(q, dtype=np.float64)
    keys = np.asarray(keys, dtype=np.float64)
    values = np.asarray(values, dtype=np.float64)
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    s = (q @ keys.T) * scale
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p = p / p.sum(axis=-1, keepdims=True)
    return p @ values
