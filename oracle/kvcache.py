"""FP8 KV-cache write: new keys and values as E4M3 codes at their cache slots.

Test infrastructure only (see the package docstring): the GPU path never
imports this module.

The paper stores the KV cache in FP8 (§3.2 FP8 Post-Training Quantization),
half the bytes of bf16.  The cache is read here as slot-major codes
[num_slots, H, D] (a paged [blocks, block_size, H, D] cache is that same
array with slot = block * block_size + offset).  For each new token t with
slot s = slot_mapping[t] in [0, num_slots) and each head h, the D values of
head h form one row that is quantized exactly like an activation row
(quantize.quantize_rows, or quantize.quantize_per_tensor with the static
scale) and stored at cache[s, h]; per-row scales go to scales[s, h].  A slot
outside [0, num_slots) skips the token.  Slots are taken to be distinct.
"""

from __future__ import annotations

import numpy as np

from . import quantize as q


def kv_cache_write(x_bits: np.ndarray, slot_mapping: np.ndarray, H: int, D: int, cache: np.ndarray,
                   scales: np.ndarray = None, static_scale: float = None):
    """Write the rows of x (bf16 bits [T, >= H*D]) into `cache` [num_slots, H, D] in place.

    Per-row mode (static_scale None): scales [num_slots, H] fp32 receives the
    stored rows' scales.  Per-tensor mode: every row uses static_scale.
    Returns (cache, scales).
    """
    num_slots = cache.shape[0]
    for t, s in enumerate(np.asarray(slot_mapping, np.int64)):
        if s < 0 or s >= num_slots:
            continue
        rows = np.asarray(x_bits[t, :H * D]).reshape(H, D)
        if static_scale is None:
            codes, sc = q.quantize_rows(rows)
            scales[s] = sc
        else:
            codes = q.quantize_per_tensor(rows, static_scale)
        cache[s] = codes
    return cache, scales
