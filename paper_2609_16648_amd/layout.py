"""Host-side view of the paged KV layout of libgm (gm.h, gm_kv_cache).

Each layer has a K pool and a V pool of shape [num_pages, n_kv, page_size *
head_dim].  Position t of sequence b lives in page block_table[b, t //
page_size] at offset t % page_size; offsets come in tiles of 16 tokens, and
inside a tile (token s, channel c):
    K at (c // 32) * 512 + ((c % 32) // 8) * 128 + s * 8 + c % 8
    V at (c // 32) * 512 + (s // 4) * 128 + (c % 16) * 8 + ((c // 16) % 2) * 4 + s % 4
These helpers scatter logical [tokens, n_kv, head_dim] entries into pools and
gather them back; they serve set-up and read-back, not the step itself.
"""
from __future__ import annotations

import numpy as np


def tile_offsets(head_dim: int):
    """(K offsets, V offsets), each [16, head_dim] int64."""
    s = np.arange(16)[:, None]
    c = np.arange(head_dim)[None, :]
    k = (c // 32) * 512 + ((c % 32) // 8) * 128 + s * 8 + c % 8
    v = (c // 32) * 512 + (s // 4) * 128 + (c % 16) * 8 + ((c // 16) % 2) * 4 + s % 4
    return k.astype(np.int64), v.astype(np.int64)


def element_index(positions: np.ndarray, pages_of_seq: np.ndarray, page_size: int, head_dim: int, which: str):
    """Flat index inside one (page, kv head) block and the page id, for every
    (position, channel): returns (page [T], elem [T, head_dim])."""
    positions = np.asarray(positions, dtype=np.int64)
    page = np.asarray(pages_of_seq, dtype=np.int64)[positions // page_size]
    off = positions % page_size
    k_off, v_off = tile_offsets(head_dim)
    tab = k_off if which == "k" else v_off
    elem = (off // 16 * 16 * head_dim)[:, None] + tab[off % 16]
    return page, elem


def scatter(pool: np.ndarray, entries: np.ndarray, positions, pages_of_seq, page_size: int, which: str):
    """pool [num_pages, n_kv, page_size*head_dim]; entries [T, n_kv, head_dim]."""
    n_kv, head_dim = entries.shape[1], entries.shape[2]
    page, elem = element_index(positions, pages_of_seq, page_size, head_dim, which)
    pool[page[:, None, None], np.arange(n_kv)[None, :, None], elem[:, None, :]] = entries


def gather(pool: np.ndarray, positions, pages_of_seq, page_size: int, n_kv: int, head_dim: int, which: str):
    page, elem = element_index(positions, pages_of_seq, page_size, head_dim, which)
    return pool[page[:, None, None], np.arange(n_kv)[None, :, None], elem[:, None, :]]


def block_table(pages_needed, max_pages: int, seed: int = 0):
    """A page table that deals sum(pages_needed) pages to the sequences in a
    shuffled order (as an allocator serving many sequences would); entries a
    sequence does not own are -1.  Returns (table [B, max_pages] int32, num_pages)."""
    pages_needed = np.asarray(pages_needed, dtype=np.int64)
    if (pages_needed > max_pages).any():
        raise ValueError("a sequence needs more than max_pages pages")
    num_pages = int(pages_needed.sum())
    perm = np.random.default_rng(seed).permutation(num_pages)
    table = np.full((len(pages_needed), max_pages), -1, dtype=np.int32)
    o = 0
    for b, n in enumerate(pages_needed):
        table[b, :n] = perm[o:o + n]
        o += n
    return table, num_pages


def tile_weight(w: np.ndarray) -> np.ndarray:
    """Row-major W [out, in] -> the tiled bf16 weight layout of gm.h: tiles of
    16 rows x 32 columns (element (n, c) of a tile at ((c % 32) // 8) * 128 +
    (n % 16) * 8 + c % 8), the tile of strip s = n // 16 and k-step c // 32 at
    ((s // 8) * (in / 32) + c // 32) * 8 + s % 8.  Returns a flat array."""
    n, k = w.shape
    if n % 128 or k % 32:
        raise ValueError(f"tiled weights need out % 128 == 0 and in % 32 == 0, got {w.shape}")
    # [group][strip in group][row][kstep][col block][col] -> [group][kstep][strip][col block][row][col]
    return np.ascontiguousarray(w.reshape(n // 128, 8, 16, k // 32, 4, 8).transpose(0, 3, 1, 4, 2, 5)).reshape(-1)


def untile_weight(flat: np.ndarray, n: int, k: int) -> np.ndarray:
    return np.ascontiguousarray(flat.reshape(n // 128, k // 32, 8, 4, 16, 8).transpose(0, 2, 4, 1, 3, 5)).reshape(n, k)
