"""Host-side (numpy) views of the library's device layouts.

Frame page of T tokens: keys [H][T][d], values transposed [H][d][T]; logical
token j of a stream lives in page page_ids[j // T] at offset j % T.  Text
keys/values of one stream: keys [H][L_x][d], values [H][d][L_x].  These are
pure index permutations used to fill and read the caller-owned buffers."""
from __future__ import annotations

import numpy as np


def pack_pages(k_tokens, v_tokens, page_ids, k_pages, v_pages):
    """Scatter logical [n, H, d] keys/values of one stream into page arrays
    k_pages [P, H, T, d] and v_pages [P, H, d, T] (modified in place)."""
    T = k_pages.shape[2]
    n = k_tokens.shape[0]
    for f in range((n + T - 1) // T):
        p = page_ids[f]
        j0, j1 = f * T, min(n, (f + 1) * T)
        k_pages[p, :, : j1 - j0, :] = np.transpose(k_tokens[j0:j1], (1, 0, 2))
        v_pages[p, :, :, : j1 - j0] = np.transpose(v_tokens[j0:j1], (1, 2, 0))


def unpack_pages(k_pages, v_pages, page_ids, n_tokens):
    """Gather logical [n, H, d] keys/values of one stream from page arrays."""
    T = k_pages.shape[2]
    H, d = k_pages.shape[1], k_pages.shape[3]
    k = np.empty((n_tokens, H, d), dtype=k_pages.dtype)
    v = np.empty((n_tokens, H, d), dtype=v_pages.dtype)
    for f in range((n_tokens + T - 1) // T):
        p = page_ids[f]
        j0, j1 = f * T, min(n_tokens, (f + 1) * T)
        k[j0:j1] = np.transpose(k_pages[p, :, : j1 - j0, :], (1, 0, 2))
        v[j0:j1] = np.transpose(v_pages[p, :, :, : j1 - j0], (2, 0, 1))
    return k, v


def ctx_to_device_layout(kc, vc, n_heads):
    """[L_x, D] text keys/values of one stream -> flat keys [H][L_x][d] and
    values [H][d][L_x] (each returned as a [L_x * D] array)."""
    Lx, D = kc.shape
    d = D // n_heads
    k = np.transpose(kc.reshape(Lx, n_heads, d), (1, 0, 2)).reshape(-1)
    v = np.transpose(vc.reshape(Lx, n_heads, d), (1, 2, 0)).reshape(-1)
    return k, v


def ctx_from_device_layout(k_flat, v_flat, Lx, n_heads, d):
    k = np.transpose(k_flat.reshape(n_heads, Lx, d), (1, 0, 2)).reshape(Lx, n_heads * d)
    v = np.transpose(v_flat.reshape(n_heads, d, Lx), (2, 0, 1)).reshape(Lx, n_heads * d)
    return k, v
