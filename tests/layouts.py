"""GPU slot layouts written out from their definitions in include/wsk.h, for
tests that read slot bytes (GPU pool or load region).  Test code only."""
import numpy as np


def gqa_elements(off, head_dim, block_tokens, head):
    """Element indices (bf16 units, within one slot) of the K and V rows of
    positions with block offsets `off` for KV head `head` (WSK_LAYOUT_TILED64):
    two [len(off), head_dim] index arrays."""
    off = np.asarray(off)
    t = off % 64
    d = np.arange(head_dim)
    tile = (head * (block_tokens // 64) + off // 64) * 16384
    mt = 2 * (t // 32) + (t % 8) // 4
    nk = 4 * ((t % 32) // 8) + t % 4
    k_piece = (4 * mt[:, None] + d[None] // 32) * 64 + 16 * ((d[None] % 32) // 8) + nk[:, None]
    k_el = tile[:, None] + k_piece * 8 + d[None] % 8
    v_piece = (2 * (d[None] // 16) + t[:, None] // 32) * 64 + 16 * ((t[:, None] % 32) // 8) + d[None] % 16
    v_el = tile[:, None] + 8192 + v_piece * 8 + t[:, None] % 8
    return k_el, v_el


def mla_elements(off, row_elems):
    """Element indices (within one slot) of the rows of positions with block
    offsets `off` (WSK_LAYOUT_MLA32): a [len(off), row_elems] index array."""
    off = np.asarray(off)
    u = off % 32
    c = np.arange(row_elems // 8)
    base = (off // 32) * (32 * row_elems)
    piece = (2 * (c[None] // 4) + (u[:, None] // 4) % 2) * 64 + 16 * (c[None] % 4) + 4 * (u[:, None] // 8) \
        + u[:, None] % 4
    return (base[:, None, None] + piece[:, :, None] * 8 + np.arange(8)[None, None]).reshape(len(off), row_elems)
