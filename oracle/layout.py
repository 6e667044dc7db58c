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
* Inside a plane: 2*r*p little-endian 32-bit words. Slot phi in [0, 64 r) lies
  in word phi // (32/p); with iota = phi % (32/p) its bits start at
  8 * (iota % 4) + p * (iota // 4).
* Slot of (token t in tile, coordinate i), with g16 = r // 16, rho = r % 16:
  K side: i < 16 g16:  phi = (i // 16) * 1024 + t * 16 + i % 16
                       (token-major inside each group of 16 coordinates)
          otherwise:   phi = 1024 g16 + t * rho + (i - 16 g16)   (the tail group)
  V side: phi = i * 64 + psi(t), psi(16 a + 4 c + e) = 16 c + 4 a + e
  (coordinate-major with a fixed 4x4 transpose of the token order).
* Slots of tokens past the end of the last tile hold zero.
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


def psi(t: int) -> int:
    a, c, e = t // 16, (t // 4) % 4, t % 4
    return 16 * c + 4 * a + e


def slot(side: int, t: int, i: int, r: int) -> int:
    if side == SIDE_V:
        return i * TILE + psi(t)
    g16, rho = r // 16, r % 16
    if i < 16 * g16:
        return (i // 16) * 1024 + t * 16 + i % 16
    return 1024 * g16 + t * rho + (i - 16 * g16)


def slot_bit(phi: int, p: int) -> tuple[int, int]:
    """(word index, bit offset) of slot phi in a plane of width p."""
    per_word = 32 // p
    iota = phi % per_word
    return phi // per_word, 8 * (iota % 4) + p * (iota // 4)


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
            words = [0] * (2 * r * p)
            for t in range(TILE):
                tok = tile * TILE + t
                if tok >= n:
                    continue
                for i in range(r):
                    v = (int(codes[tok][i]) >> sh) & ((1 << p) - 1)
                    w, bit = slot_bit(slot(side, t, i, r), p)
                    words[w] |= v << bit
            for w, val in enumerate(words):
                out[base + plane_off + 4 * w: base + plane_off + 4 * w + 4] = val.to_bytes(4, "little")
            plane_off += 8 * r * p
    return bytes(out)


def unpack(stream: bytes, n: int, r: int, b: int, side: int) -> list[list[int]]:
    widths, shifts = plane_widths(b), plane_shifts(b)
    codes = [[0] * r for _ in range(n)]
    for tok in range(n):
        tile, t = divmod(tok, TILE)
        base = tile * tile_bytes(r, b)
        plane_off = 0
        for p, sh in zip(widths, shifts):
            for i in range(r):
                w, bit = slot_bit(slot(side, t, i, r), p)
                word = int.from_bytes(stream[base + plane_off + 4 * w: base + plane_off + 4 * w + 4], "little")
                codes[tok][i] |= ((word >> bit) & ((1 << p) - 1)) << sh
            plane_off += 8 * r * p
    return codes
