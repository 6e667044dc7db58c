"""Packed code-stream layout, written plainly in Python (oracle; tiny inputs only).

Test infrastructure only: nothing in the product path may import this module.

The paper stores r codes of b bits per token per head with no per-token
metadata, i.e. exactly r*b/d bits per dimension (Appendix E, the paragraph on
the rotation-based methods), and dequantizes on the attention read (table step
8). It leaves the byte layout open; the layout below is this implementation's
definition, and the oracle packs to it independently of the GPU encoder.

* Tiles of 64 tokens. Tile t of a (unit, side) stream starts at byte
  code_off + t * 8 * r * b; a tile is 8*r*b bytes (r even, so a multiple of 16).
* A b-bit code is split into planes: b = 8 is one 8-bit plane; otherwise the
  binary expansion of b, widest plane first (7 -> 4,2,1). The widest plane
  holds the most significant bits. Plane of width p occupies 8*r*p bytes, the
  planes follow one another in that order.
* K side: slot phi in [0, 64 r) of a plane of width p holds its p bits at
  bits [p*phi, p*phi + p) of the plane, counting bit n as bit n % 8 of byte
  n // 8 (a plain little-endian bit stream). Slot of (token t in tile,
  coordinate i), with g16 = r // 16, rho = r % 16:
      i < 16 g16:  phi = (i // 16) * 1024 + t * 16 + i % 16
                   (groups of 16 coordinates, token-major inside a group)
      otherwise:   phi = 1024 g16 + t * rho + (i - 16 g16)   (the tail group)
* V side: fields of 16 codes. Field (n, c, q) holds coordinate 16 n + c
  (N-tile n, column c) for the 16 tokens of quarter q = t // 16 of the tile,
  token t at position pos_b(t % 16): p bits each at bits [p*pos, p*pos + p)
  of the field's 2p bytes. In a plane of width p the N-tiles form groups of
  g = 8 // p consecutive ones (g = 1 for p = 8), and the fields of the
  coordinates below r are stored one after another in the order
  (n // g, 4 c + q, n): group by group, inside a group by L = 4 c + q, then
  by N-tile. So the fields of one L in a group are 16 consecutive bytes
  (fewer in a short last group).
* pos_b(m) is the position inside a run of 16 items given to the m-th item:
  b = 8: m; b = 4: 8 (m // 8) + 2 (m % 4) + (m // 4) % 2; any other b:
  4 (m % 4) + m // 4 (a 4 x 4 transpose). It is an involution for b != 4.
* The bits of tokens past the end of the last tile hold zero.
"""
from __future__ import annotations

SIDE_K = 0
SIDE_V = 1
TILE = 64


def plane_widths(b: int) -> list[int]:
    if b == 8:
        return [8]
    return [p for p in (4, 2, 1) if b & p]


def plane_shifts(b: int) -> list[int]:
    widths = plane_widths(b)
    out = []
    for k in range(len(widths)):
        out.append(sum(widths[k + 1:]))
    return out


def tile_bytes(r: int, b: int) -> int:
    return 8 * r * b


def stream_bytes(n_tok: int, r: int, b: int) -> int:
    return ((n_tok + TILE - 1) // TILE) * tile_bytes(r, b)


def pos_b(b: int, m: int) -> int:
    if b == 8:
        return m
    if b == 4:
        return 8 * (m // 8) + 2 * (m % 4) + (m // 4) % 2
    return 4 * (m % 4) + m // 4


def slot_k(t: int, i: int, r: int) -> int:
    g16, rho = r // 16, r % 16
    if i < 16 * g16:
        return (i // 16) * 1024 + t * 16 + i % 16
    return 1024 * g16 + t * rho + (i - 16 * g16)


def v_field_bytes(r: int, p: int) -> dict:
    """Byte offset inside a V plane of width p of every field (n, c, q), by enumeration in the
    layout's order (group n // g, then 4 c + q, then n)."""
    g = 1 if p == 8 else 8 // p
    nvt = (r + 15) // 16
    order = sorted(((n // g, 4 * c + q, n), (n, c, q)) for n in range(nvt) for c in range(16) for q in range(4)
                   if 16 * n + c < r)
    return {key: 2 * p * k for k, (_, key) in enumerate(order)}


def plane_bit(side: int, t: int, i: int, r: int, b: int, p: int, vtab=None) -> int:
    """Bit of the code of (token t in tile, coordinate i) inside its plane of width p."""
    if side == SIDE_K:
        return p * slot_k(t, i, r)
    vtab = v_field_bytes(r, p) if vtab is None else vtab
    return 8 * vtab[(i // 16, i % 16, t // 16)] + p * pos_b(b, t % 16)


def pack(codes, r: int, b: int, side: int) -> bytes:
    """codes[t][i] for tokens 0..n-1 (n may be ragged) -> stream bytes."""
    n = len(codes)
    n_tiles = (n + TILE - 1) // TILE
    out = bytearray(n_tiles * tile_bytes(r, b))
    widths, shifts = plane_widths(b), plane_shifts(b)
    for tile in range(n_tiles):
        base = tile * tile_bytes(r, b)
        plane_off = 0
        for p, sh in zip(widths, shifts):
            vtab = v_field_bytes(r, p) if side == SIDE_V else None
            for t in range(TILE):
                tok = tile * TILE + t
                if tok >= n:
                    continue
                for i in range(r):
                    v = (int(codes[tok][i]) >> sh) & ((1 << p) - 1)
                    bit = plane_bit(side, t, i, r, b, p, vtab)
                    out[base + plane_off + bit // 8] |= v << (bit % 8)
            plane_off += 8 * r * p
    return bytes(out)


def unpack(stream: bytes, n: int, r: int, b: int, side: int) -> list[list[int]]:
    widths, shifts = plane_widths(b), plane_shifts(b)
    vtabs = [v_field_bytes(r, p) if side == SIDE_V else None for p in widths]
    codes = [[0] * r for _ in range(n)]
    for tok in range(n):
        tile, t = divmod(tok, TILE)
        base = tile * tile_bytes(r, b)
        plane_off = 0
        for p, sh, vtab in zip(widths, shifts, vtabs):
            for i in range(r):
                bit = plane_bit(side, t, i, r, b, p, vtab)
                codes[tok][i] |= ((stream[base + plane_off + bit // 8] >> (bit % 8)) & ((1 << p) - 1)) << sh
            plane_off += 8 * r * p
    return codes
