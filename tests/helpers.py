"""Shared test helpers: device transfer, the parity metric, mask packing."""
from __future__ import annotations

import numpy as np


def parity_err(gpu, ref) -> float:
    """max_i |g_i - o_i| / max(|o_i|, rms(o)) -- the element-wise relative
    error with the reference's RMS as the floor."""
    g = np.asarray(gpu, dtype=np.float64)
    o = np.asarray(ref, dtype=np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    if o.size == 0:
        return 0.0
    rms = np.sqrt(np.mean(o * o))
    if rms == 0:
        return float(np.max(np.abs(g - o)))
    den = np.maximum(np.abs(o), rms)
    return float(np.max(np.abs(g - o) / den))


def pack_mask(mask_bool: np.ndarray) -> np.ndarray:
    """bool [n, d] -> int32 [n, d/32]: bit c%32 of word c/32 is mask[j, c]."""
    n, d = mask_bool.shape
    bits = mask_bool.reshape(n, d // 32, 32).astype(np.uint64)
    words = (bits << np.arange(32, dtype=np.uint64)).sum(axis=2).astype(np.uint32)
    return words.view(np.int32)


def unpack_mask(words: np.ndarray, d: int) -> np.ndarray:
    w = np.asarray(words).view(np.uint32).reshape(-1, d // 32)
    bits = (w[:, :, None] >> np.arange(32, dtype=np.uint32)) & 1
    return bits.reshape(w.shape[0], d).astype(bool)


def to_dev(x, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(device)


def graph_to_dev(g, device="cuda"):
    import torch
    return dict(src=to_dev(g.src, device), dst=to_dev(g.dst, device), rel=to_dev(g.rel, device),
                ntype=to_dev(g.ntype, device), part=to_dev(g.part, device))


def clear_relu_kinks(a, rows, margin_rel=1e-4):
    """Per-column shift of a bias that keeps every pre-activation a[rows, j]
    at least margin_rel * rms(a[rows]) away from the ReLU kink, so that a
    float32 and a float64 evaluation take the same decision there.  Returns
    the shift [d] (zero for a column that needs none); tests add it to the
    bias before either side runs."""
    a = np.asarray(a, dtype=np.float64)[rows]
    d = a.shape[1]
    if a.size == 0:
        return np.zeros(d)
    margin = margin_rel * np.sqrt(np.mean(a * a))
    delta = np.zeros(d)
    for j in range(d):
        for k in range(256):
            cand = ((k + 1) // 2) * (1 if k % 2 else -1) * 2.0 * margin   # 0, +2m, -2m, +4m, ...
            if np.min(np.abs(a[:, j] + cand)) > margin:
                delta[j] = cand
                break
        else:
            raise AssertionError(f"no bias shift clears column {j}")
    return delta
