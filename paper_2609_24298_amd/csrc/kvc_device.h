// Device-side helpers of libkvc shared by the HIP kernels: the packed-stream
// layout (see include/kvc.h) and fp16 bit decoding. CDNA4 / gfx950 only.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "kvc.h"
#include "kvc_internal.h"

namespace kvc {

// Per-side tables passed to kernels by value.
struct DevSide {
    const int32_t* r;
    const int32_t* b;
    const int64_t* code_off;
    const int64_t* basis_off;
    const float* delta;
    uint8_t* codes;
    const uint16_t* basis;
};

// Position inside a run of 16 slots given to the m-th item, and its inverse. The V side stores
// each quarter of 16 tokens in this order; in the decode kernels position j of a 16-slot run is
// operand byte kidx_b(j) (byte k of dword d at 4d + k), which is where the unpacking of a field of
// that width puts it. b = 8: identity; b = 4: nibble pairs; other b: 4 x 4 transpose.
__host__ __device__ constexpr int pos_b(int b, int m) {
    return b == 8 ? m : (b == 4 ? 8 * (m >> 3) + 2 * (m & 3) + ((m >> 2) & 1) : 4 * (m & 3) + (m >> 2));
}
__host__ __device__ constexpr int kidx_b(int b, int j) {
    return b == 8 ? j : (b == 4 ? 8 * (j >> 3) + 4 * (j & 1) + ((j & 7) >> 1) : 4 * (j & 3) + (j >> 2));
}

// Slot of (token t in tile, coordinate i) on the K side: token-major inside groups of 16
// coordinates (a token's 16 codes of a group are 16 consecutive slots), the r % 16 tail group
// token-major after them; slot phi of a plane of width p holds bits [p phi, p phi + p).
__device__ __forceinline__ int slot_k(int t, int i, int r) {
    const int g16 = r >> 4;
    if (i < 16 * g16) return ((i >> 4) << 10) + (t << 4) + (i & 15);
    return (g16 << 10) + t * (r & 15) + (i - 16 * g16);
}
// Inverse of slot_k: token and coordinate of slot phi.
__device__ __forceinline__ void unslot_k(int phi, int r, int& t, int& i) {
    const int g16 = r >> 4;
    if (phi < (g16 << 10)) { t = (phi >> 4) & 63; i = ((phi >> 10) << 4) + (phi & 15); return; }
    const int rho = r & 15, q = phi - (g16 << 10);
    t = q / rho;
    i = 16 * g16 + (q - t * rho);
}
// V fields: the 16 codes of coordinate 16 n + c (N-tile n, column c) for the tokens of quarter q of
// the tile, token t at position pos_b(t % 16), p bits each: 2p bytes. In a plane of width p the
// N-tiles form groups of g = 8 / p (g = 1 for p = 8), group Q at byte 1024 Q of the plane, and a
// group stores its fields ordered by L = 4 c + q, then n (the fields of coordinates below r only):
// a lane's fields of a whole group are 16 consecutive bytes. Byte offset of field (n, c, q) in the
// plane: 2p (g L + j), j = n - g Q, in a group of g N-tiles; in the last group, of m N-tiles whose
// last holds ct coordinates, 2p (m L - A + j) with A = 4 max(0, c - ct) + [c >= ct] q fields of
// the coordinates c' >= ct (one field fewer each) ahead of L.
__host__ __device__ constexpr int v_group_ntiles(int p) { return p == 8 ? 1 : 8 / p; }
__host__ __device__ inline int v_field_off(int p, int r, int n, int c, int q) {
    const int g = v_group_ntiles(p), nvt = (r + 15) >> 4;
    const int Q = n / g, j = n - g * Q, ql = (nvt - 1) / g, L = 4 * c + q;
    if (Q < ql) return 1024 * Q + 2 * p * (g * L + j);
    const int m = nvt - g * ql, ct = r - 16 * (nvt - 1);
    const int A = c >= ct ? 4 * (c - ct) + q : 0;
    return 1024 * Q + 2 * p * (m * L - A + j);
}
// Bit of the code of (token t in tile, coordinate i) in the V plane of width p.
__host__ __device__ inline int v_plane_bit(int t, int i, int r, int b, int p) {
    return 8 * v_field_off(p, r, i >> 4, i & 15, t >> 4) + p * pos_b(b, t & 15);
}

// Code stored in K slot phi of the tile starting at `tile`: the p bits of each plane
// (widest first) sit at bits [p phi, p phi + p) of the plane.
__device__ __forceinline__ uint32_t load_code(const uint8_t* __restrict__ tile, int r, int b, int phi) {
    if (b == 8) return tile[phi];
    uint32_t c = 0;
    int rem = b;
    int off = 0;
#pragma unroll
    for (int p = 4; p >= 1; p >>= 1) {
        if (b & p) {
            const int bit = p * phi;
            rem -= p;
            c |= ((uint32_t)(tile[off + (bit >> 3)] >> (bit & 7)) & ((1u << p) - 1u)) << rem;
            off += 8 * r * p;
        }
    }
    return c;
}

// Code of (token t in tile, coordinate i) on the V side.
__device__ __forceinline__ uint32_t load_code_v(const uint8_t* __restrict__ tile, int r, int b, int t, int i) {
    if (b == 8) return tile[v_plane_bit(t, i, r, 8, 8) >> 3];
    uint32_t c = 0;
    int rem = b;
    int off = 0;
#pragma unroll
    for (int p = 4; p >= 1; p >>= 1) {
        if (b & p) {
            const int bit = v_plane_bit(t, i, r, b, p);
            rem -= p;
            c |= ((uint32_t)(tile[off + (bit >> 3)] >> (bit & 7)) & ((1u << p) - 1u)) << rem;
            off += 8 * r * p;
        }
    }
    return c;
}

// Planes of a b-bit code, widest first (b = 8: one plane): width of plane k, its bit
// shift inside the code and its offset in units of 8*r bytes. Fragment extraction is
// instantiated per b, so these fold to constants.
__host__ __device__ constexpr int n_planes(int b) { return b == 8 ? 1 : ((b & 4) ? 1 : 0) + ((b & 2) ? 1 : 0) + (b & 1); }
__host__ __device__ constexpr int plane_w(int b, int k) {
    return b == 8 ? 8 : (k == 0 ? ((b & 4) ? 4 : ((b & 2) ? 2 : 1))
                               : (k == 1 ? ((b & 4) ? ((b & 2) ? 2 : 1) : 1) : 1));
}
// Bits below plane k (its shift) and plane widths before it (its offset): closed forms, so that
// they fold to constants even where k is an unrolled loop index.
__host__ __device__ constexpr int plane_sh(int b, int k) { return b == 8 ? 0 : (b & (plane_w(b, k) - 1)); }
__host__ __device__ constexpr int plane_off(int b, int k) { return b == 8 ? 0 : (b & ~(2 * plane_w(b, k) - 1)); }

// Runs CALL with the compile-time bit width B_ equal to the runtime value b.
#define KVC_SWITCH_B(b, CALL)                                \
    switch (b) {                                             \
        case 1: { constexpr int B_ = 1; CALL; } break;       \
        case 2: { constexpr int B_ = 2; CALL; } break;       \
        case 3: { constexpr int B_ = 3; CALL; } break;       \
        case 4: { constexpr int B_ = 4; CALL; } break;       \
        case 5: { constexpr int B_ = 5; CALL; } break;       \
        case 6: { constexpr int B_ = 6; CALL; } break;       \
        case 7: { constexpr int B_ = 7; CALL; } break;       \
        default: { constexpr int B_ = 8; CALL; } break;      \
    }

// fp16 bits -> fp32 (exact).
__device__ __forceinline__ float h2f(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }

// fp16 bits -> signed integer mantissa m and exponent e with value m * 2^e
// (finite inputs; e in [-24, 5]).
__device__ __forceinline__ void half_parts(uint16_t h, int32_t& m, int& e) {
    const int ex = (h >> 10) & 31, fr = h & 1023;
    if (ex == 0) { m = fr; e = -24; }
    else { m = 1024 + fr; e = ex - 25; }
    if (h & 0x8000) m = -m;
}

// ---------------------------------------------------------------- host helpers

inline DevSide dev_side(const kvc_stream_desc* s) {
    return DevSide{s->r, s->b, s->code_off, s->basis_off, s->delta, s->codes, s->basis};
}

inline int check_launch(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(KVC_EDEVICE, "%s: %s", what, hipGetErrorString(e));
    return KVC_OK;
}

}  // namespace kvc
