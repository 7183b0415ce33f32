"""Oracle: hybrid-mask block attention over a paged KV cache (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__``).

What is computed
----------------
One forward carries ``R = n_causal + n_mask`` query rows per sequence s at
absolute positions ``L_s + r`` (r = 0..R-1).  Positions ``[0, L_s)`` hold the
committed, causal KV in the cache; the R rows' own K/V are appended at
``[L_s, L_s + R)`` before attending (the verify pass writes its own KV into
the cache; appendix "Self-Speculative Decoding and KV-Cache Update", Verify
forward).

Visibility (the block-causal pattern of Preliminaries "Block Diffusion" and
Method "Joint AR-Diffusion Training"; the draft window of the appendix's
Draft forward item):

* causal rows r < n_causal see keys ``k <= L_s + r``  (token-level causal);
* mask rows r >= n_causal see the whole cache, every causal row of the
  window, and every mask row (bidirectional inside the mask block), i.e.
  ``k <= L_s + R - 1``.

For each visible key the score is ``scale * <q, k>``; the output is the
softmax-weighted sum of V (standard scaled dot-product attention).  Query head
h reads KV head ``h // (Hq / Hkv)`` (grouped-query attention with contiguous
groups).  Nothing is blocked, fused, or computed online: each row's full score
vector is formed, masked, exponentiated after subtracting its maximum,
normalised and contracted with V.
"""
from __future__ import annotations

import numpy as np


def visible_hi(L: int, n_causal: int, n_mask: int) -> np.ndarray:
    """Largest visible absolute key position for each window row (inclusive)."""
    R = n_causal + n_mask
    hi = np.empty(R, dtype=np.int64)
    for r in range(R):
        hi[r] = L + r if r < n_causal else L + R - 1
    return hi


def visible_mask(L: int, n_causal: int, n_mask: int, group: int = 0) -> np.ndarray:
    """Visibility [R, L + R] of the window rows over key positions, with the
    mask rows cut into groups of ``group`` rows (0: one group of n_mask).

    Causal row r sees keys <= L + r.  With G = n_mask / group groups, the
    rows of mask group g see the whole cache, the causal rows
    0 .. n_causal - G + g and the rows of their own group (bidirectionally).
    One group (G = 1) is the hybrid mask of ``visible_hi``.  With
    G = n_causal, group g is the draft block of the continuation that keeps
    the causal rows 0..g: the per-acceptance drafts of the structured-mask
    AR-diffusion hybrids the paper cites in its related work.
    """
    R = n_causal + n_mask
    group = n_mask if group == 0 else group
    vis = np.zeros((R, L + R), dtype=bool)
    vis[:, :L] = True
    for r in range(n_causal):
        vis[r, L:L + r + 1] = True
    if n_mask:
        n_groups = n_mask // group
        assert n_groups * group == n_mask and (n_groups == 1 or n_groups <= n_causal)
        for r in range(n_causal, R):
            g = (r - n_causal) // group
            vis[r, L:L + n_causal - n_groups + g + 1] = True
            lo = L + n_causal + g * group
            vis[r, lo:lo + group] = True
    return vis


def window_positions(L: int, n_causal: int, n_mask: int, group: int = 0) -> np.ndarray:
    """Sequence position of every window row: L + r for causal rows; row i of
    mask group g sits right after the last causal row the group sees, at
    L + (n_causal - G + g) + 1 + i (one group: L + r)."""
    R = n_causal + n_mask
    group = n_mask if group == 0 else max(group, 1)
    pos = np.empty(R, dtype=np.int64)
    pos[:n_causal] = L + np.arange(n_causal)
    if n_mask:
        n_groups = n_mask // group
        for r in range(n_causal, R):
            g, i = divmod(r - n_causal, group)
            pos[r] = L + (n_causal - n_groups + g) + 1 + i
    return pos


def gather_cache(pool: np.ndarray, page_row: np.ndarray, L: int, page_size: int,
                 slot_last: bool = False, decode=None) -> np.ndarray:
    """Dense [L, Hkv, D] view of a sequence's first L cached positions.

    Logical position p lives in physical page ``page_row[p // page_size]`` at
    slot ``p % page_size``.  K pools are laid out [pages, Hkv, page_size, D];
    V pools (``slot_last``) are laid out [pages, Hkv, D, page_size].
    ``decode`` (optional) maps stored elements to float64, e.g. bf16 bit
    patterns, so a large pool need not be expanded as a whole.
    """
    Hkv = pool.shape[1]
    D = pool.shape[2] if slot_last else pool.shape[3]
    out = np.empty((L, Hkv, D), dtype=np.float64)
    for p in range(L):
        page, slot = page_row[p // page_size], p % page_size
        v = pool[page, :, :, slot] if slot_last else pool[page, :, slot, :]
        out[p] = v if decode is None else decode(v)
    return out


def append_block(pool: np.ndarray, page_row: np.ndarray, L: int, block: np.ndarray,
                 page_size: int, slot_last: bool = False) -> None:
    """Write the window's R rows of K (or V), [R, Hkv, D], at positions [L, L+R)."""
    for r in range(block.shape[0]):
        p = L + r
        page, slot = page_row[p // page_size], p % page_size
        if slot_last:
            pool[page, :, :, slot] = block[r]
        else:
            pool[page, :, slot, :] = block[r]


def attend_rows(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, hi: np.ndarray,
                scale: float) -> np.ndarray:
    """Masked softmax attention for one sequence.

    q [R, Hq, D]; keys/vals [T, Hkv, D] at absolute positions 0..T-1;
    hi[r] = last visible position of row r.  Returns [R, Hq, D].
    """
    R, Hq, D = q.shape
    T, Hkv, _ = keys.shape
    G = Hq // Hkv
    pos = np.arange(T)
    out = np.zeros((R, Hq, D), dtype=np.float64)
    for r in range(R):
        vis = pos <= hi[r]
        for h in range(Hq):
            g = h // G
            s = scale * (keys[:, g, :] @ q[r, h, :])          # [T]
            s = np.where(vis, s, -np.inf)
            s = s - s.max()
            w = np.exp(s)
            w = w / w.sum()
            out[r, h, :] = w @ vals[:, g, :]
    return out


def attend_rows_vis(q: np.ndarray, keys: np.ndarray, vals: np.ndarray, vis: np.ndarray,
                    scale: float) -> np.ndarray:
    """attend_rows with an explicit visibility vis [R, T] over key positions."""
    R, Hq, D = q.shape
    T, Hkv, _ = keys.shape
    G = Hq // Hkv
    out = np.zeros((R, Hq, D), dtype=np.float64)
    for r in range(R):
        for h in range(Hq):
            g = h // G
            s = scale * (keys[:, g, :] @ q[r, h, :])
            s = np.where(vis[r], s, -np.inf)
            s = s - s.max()
            w = np.exp(s)
            w = w / w.sum()
            out[r, h, :] = w @ vals[:, g, :]
    return out


def attn_hybrid_block(q, k_new, v_new, k_pool, v_pool, page_table, kv_len,
                      n_causal: int, n_mask: int, scale: float, page_size: int = 16,
                      seqs=None, group: int = 0):
    """Append the window's K/V to the pools, then attend with the hybrid mask
    (``group`` > 0: the grouped mask of ``visible_mask``).

    All float inputs are float64 arrays: q [S,R,Hq,D], k_new/v_new [S,R,Hkv,D],
    k_pool [P,Hkv,page_size,D], v_pool [P,Hkv,D,page_size] (both modified in
    place by the append).
    Returns out [S,R,Hq,D] (rows of sequences not in ``seqs`` are left zero).
    """
    S, R = q.shape[0], q.shape[1]
    assert R == n_causal + n_mask
    out = np.zeros(q.shape, dtype=np.float64)
    for s in (range(S) if seqs is None else seqs):
        L = int(kv_len[s])
        append_block(k_pool, page_table[s], L, k_new[s], page_size)
        append_block(v_pool, page_table[s], L, v_new[s], page_size, slot_last=True)
        keys = gather_cache(k_pool, page_table[s], L + R, page_size)
        vals = gather_cache(v_pool, page_table[s], L + R, page_size, slot_last=True)
        if group and group != n_mask:
            out[s] = attend_rows_vis(q[s], keys, vals, visible_mask(L, n_causal, n_mask, group),
                                     scale)
        else:
            out[s] = attend_rows(q[s], keys, vals, visible_hi(L, n_causal, n_mask), scale)
    return out


def attn_sampled(q, k_new, v_new, k_pool, v_pool, page_table, kv_len, n_causal: int,
                 n_mask: int, scale: float, samples, page_size: int = 16, decode=None):
    """Outputs for selected (s, r, h) triples, without touching the pools.

    Keys at [L_s, L_s + R) are taken from the window's own K/V (what the
    append would have written).  q, k_new, v_new are float64; the pools may be
    stored in another format that ``decode`` maps to float64.
    Returns {(s, r, h): [D] float64}.
    """
    res = {}
    by_seq = {}
    for (s, r, h) in samples:
        by_seq.setdefault(int(s), []).append((int(r), int(h)))
    R = q.shape[1]
    Hq, Hkv = q.shape[2], k_new.shape[2]
    G = Hq // Hkv
    for s, rh in by_seq.items():
        L = int(kv_len[s])
        cache_k = gather_cache(k_pool, page_table[s], L, page_size, decode=decode)
        cache_v = gather_cache(v_pool, page_table[s], L, page_size, slot_last=True,
                               decode=decode)
        keys = np.concatenate([cache_k, k_new[s]], axis=0)
        vals = np.concatenate([cache_v, v_new[s]], axis=0)
        hi = visible_hi(L, n_causal, n_mask)
        pos = np.arange(L + R)
        for (r, h) in rh:
            g = h // G
            sc = scale * (keys[:, g, :] @ q[s, r, h, :])
            sc = np.where(pos <= hi[r], sc, -np.inf)
            w = np.exp(sc - sc.max())
            w /= w.sum()
            res[(s, r, h)] = w @ vals[:, g, :]
    return res
