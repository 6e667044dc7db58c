// Device functions of the few-token append (a decode step's new token), shared by the encode
// kernels (kvc_kernels.hip) and the fused decode step (kvc_decode.hip): exact and bounded code
// decisions, and the per-unit append that decides the codes of 1-4 new tokens and writes them into
// their tiles. CDNA4 / gfx950 only. Each including source gets its own copy (internal linkage).
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kvc_device.h"

namespace kvc {
namespace {

// Exact code: y = sum_j P_ij x_j as an integer N = y 2^48 (|y| < 2^88); the code
// clamp(floor(y / step) + 2^(b-1), 0, 2^b - 1) equals the number of thresholds
// j step, j in [1 - 2^(b-1), 2^(b-1) - 1], that y reaches, found by bisection with
// exact 128-bit comparisons N >= j step 2^48 (no division). Used only for
// elements the floating-point paths cannot decide.
__device__ __forceinline__ uint32_t exact_code(const uint16_t* __restrict__ Prow, const uint16_t* __restrict__ xrow,
                                               float step, int b) {
    __int128 N = 0;
    for (int j = 0; j < KVC_HEAD_DIM; ++j) {
        int32_t mp, mx;
        int ep, ex;
        half_parts(Prow[j], mp, ep);
        half_parts(xrow[j], mx, ex);
        N += (__int128)((int64_t)mp * mx) << (ep + ex + 48);
    }
    const uint32_t u = __float_as_uint(step);
    const int64_t m = 0x800000 | (u & 0x7fffff);
    const int sD = (int)((u >> 23) & 255) - 150 + 48;  // >= 1 for step >= 2^-24
    const int h = 1 << (b - 1);
    // count = #{j in [lo, hi] : N >= j m 2^sD}; thresholds increase with j
    int lo = 1 - h, hi = h - 1;  // the answer is lo + (number passed) - ... kept as a half-open search
    int first_fail = hi + 1;     // smallest j with N < j D (hi + 1 if none)
    while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        if (N >= ((__int128)((int64_t)mid * m) << sD)) lo = mid + 1;
        else { first_fail = mid; hi = mid - 1; }
    }
    return (uint32_t)(first_fail - (1 - h));
}

// Code from the fp32 projection `acc` whose error is at most `err` (|acc - y| <= err), when no
// quantizer threshold j * step, j in [1 - 2^(b-1), 2^(b-1) - 1], lies within that error: returns
// false (undecided) otherwise.
__device__ __forceinline__ bool fast_code(float acc, float err, float step, int b, uint32_t& code) {
    const int h = 1 << (b - 1);
    const double st = step, yd = acc, ed = err;
    const double t = yd / st;
    if (!(ed < 0.25 * st)) return false;
    const double jn = rint(t);
    if (jn >= 1 - h && jn <= h - 1 && !(fabs(yd - jn * st) > ed + 0x1p-45 * fabs(yd))) return false;
    code = (uint32_t)fmin(fmax(floor(t) + h, 0.0), (double)((1 << b) - 1));
    return true;
}

// v moved across the lanes of each row of 16 by a DPP row rotation (both halves of the double).
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double v) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)u, CTRL, 0xf, 0xf, true);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_mov_dpp((int)(uint32_t)(u >> 32), CTRL, 0xf, 0xf, true);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
    const uint64_t u = __builtin_bit_cast(uint64_t, v);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, l);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), l);
    return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Sum over the wavefront, the same value in every lane: row sums by row rotations (8, 4, 2, 1), then
// the four row sums. The order of the additions is fixed but not that of a sequential sum; the
// callers' error bounds hold for any order.
__device__ __forceinline__ double wave_sum(double v) {
    v += dpp_f64<0x128>(v);
    v += dpp_f64<0x124>(v);
    v += dpp_f64<0x122>(v);
    v += dpp_f64<0x121>(v);
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// Code from y ~ P_c . x (an fp64 sum of the 128 exact fp16 products, any order): true when y is far
// enough from every threshold for the code to be certain. jn is a threshold index near y / step;
// the sign of y - jn step is certain when |y - jn step| exceeds the bound, and then (for
// e < step / 4) y lies between the jn - 1 and jn + 1 thresholds.
__device__ __forceinline__ bool certain_code(double y, float step, int b, float pn, float xn, uint32_t& code) {
    const double e = 0x1p-45 * (double)pn * (double)xn * 1.01;
    const int h = 1 << (b - 1);
    const double st = step;
    const double jn = rint(y * (1.0 / st));
    const double d = fma(-jn, st, y);
    if (e < 0.25 * st && fabs(d) > e + 0x1p-50 * fabs(y) && fabs(d) < 0.75 * st) {
        code = (uint32_t)fmin(fmax(jn - (d < 0.0 ? 1.0 : 0.0) + h, 0.0), (double)((1 << b) - 1));
        return true;
    }
    return false;
}

// Code of coordinate c for token row `xrow`, decided by the whole wavefront: fp64 sum of the 128
// exact products (lane takes j = 2 lane, 2 lane + 1), then the exact path if still undecided.
// Uniform across the wavefront.
__device__ uint32_t resolve_code_wave(const uint16_t* __restrict__ Pl_row, const uint16_t* __restrict__ Pg_row,
                                      const uint16_t* __restrict__ xrow, float step, int b, float pn, float xn,
                                      int lane) {
    const uint32_t pw = *reinterpret_cast<const uint32_t*>(Pl_row + 2 * lane);
    const uint32_t xw = *reinterpret_cast<const uint32_t*>(xrow + 2 * lane);
    const double s = (double)h2f((uint16_t)(pw & 0xffff)) * (double)h2f((uint16_t)(xw & 0xffff)) +
                     (double)h2f((uint16_t)(pw >> 16)) * (double)h2f((uint16_t)(xw >> 16));
    const double y = wave_sum(s);
    uint32_t code;
    if (certain_code(y, step, b, pn, xn, code)) return code;
    return exact_code(Pg_row, xrow, step, b);
}

// Sum over the 16 lanes of a DPP row, returned in every lane of the row (row rotations).
__device__ __forceinline__ float row_sum16(float v) {
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x128, 0xf, 0xf, true));
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x124, 0xf, 0xf, true));
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x122, 0xf, 0xf, true));
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x121, 0xf, 0xf, true));
    return v;
}

// Appending a few tokens (a decode step adds one per unit): one block per unit; coordinate i of
// every new token is projected from basis row i, its code decided against the fp32 error bound
// (the wavefront settles the rare undecided ones as the bulk encoder does), and the new codes are
// written into their tiles.
constexpr int kAppThreads = KVC_HEAD_DIM;
constexpr int kAppMaxTok = 4;

__device__ __forceinline__ void append_unit(const DevSide& s, int side, const uint16_t* __restrict__ x,
                                            int64_t x_stride, int t0, int n_tok, int u) {
    __shared__ float xs[kAppMaxTok][KVC_HEAD_DIM];
    __shared__ float red[kAppMaxTok][kAppThreads / 64];
    __shared__ uint8_t cs[kAppMaxTok][KVC_HEAD_DIM];
    __shared__ float ys[kAppMaxTok][KVC_HEAD_DIM];
    __shared__ float pns[KVC_HEAD_DIM];
    const int i = threadIdx.x;
    const int r = s.r[u], b = s.b[u];
    const float step = s.delta[u];
    const uint16_t* __restrict__ P = s.basis + s.basis_off[u];
    const uint16_t* __restrict__ xu = x + (int64_t)u * x_stride;
    for (int t = 0; t < n_tok; ++t) {
        const float v = h2f(xu[(int64_t)t * KVC_HEAD_DIM + i]);
        xs[t][i] = v;
        float s2 = v * v;
        for (int o = 32; o > 0; o >>= 1) s2 += __shfl_xor(s2, o);
        if ((i & 63) == 0) red[t][i >> 6] = s2;
    }
    __syncthreads();
    {
        // Coalesced projection: in pass k, the 16 lanes (rr, c) of a row group read 16 bytes each of
        // basis row 8 k + rr (the whole 256-byte row), form partial dot products over their 8 columns
        // and sum them across the group with row rotations. Every row's loads are issued up front.
        const int c = i & 15, rr = i >> 4;
        float xr[kAppMaxTok][8];
#pragma unroll
        for (int t = 0; t < kAppMaxTok; ++t)
#pragma unroll
            for (int e = 0; e < 8; ++e) xr[t][e] = t < n_tok ? xs[t][8 * c + e] : 0.f;
        uint4 w[KVC_HEAD_DIM / 8];
#pragma unroll
        for (int k = 0; k < KVC_HEAD_DIM / 8; ++k) {
            const int row = 8 * k + rr;
            w[k] = row < r ? reinterpret_cast<const uint4*>(P + (int64_t)row * KVC_HEAD_DIM)[c] : uint4{0u, 0u, 0u, 0u};
        }
#pragma unroll
        for (int k = 0; k < KVC_HEAD_DIM / 8; ++k) {
            const uint32_t w4[4] = {w[k].x, w[k].y, w[k].z, w[k].w};
            float pn = 0.f, acc[kAppMaxTok] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const float pv = h2f((uint16_t)(w4[e >> 1] >> (16 * (e & 1))));
                pn = fmaf(pv, pv, pn);
#pragma unroll
                for (int t = 0; t < kAppMaxTok; ++t) acc[t] = fmaf(pv, xr[t][e], acc[t]);
            }
            pn = row_sum16(pn);
#pragma unroll
            for (int t = 0; t < kAppMaxTok; ++t)
                if (t < n_tok) acc[t] = row_sum16(acc[t]);
            if (c == 0) {
                const int row = 8 * k + rr;
                pns[row] = pn;
#pragma unroll
                for (int t = 0; t < kAppMaxTok; ++t) ys[t][row] = acc[t];
            }
        }
    }
    __syncthreads();
    {
        // Codes decided in fp32 where the error bound allows; each undecided element is then
        // resolved by its whole wavefront (fp64, then exact), one element at a time.
        const int lane = i & 63;
        const float pn = i < r ? sqrtf(pns[i]) : 0.f;
        for (int t = 0; t < n_tok; ++t) {
            // |acc - y| <= 2^-17 ||P_i|| ||x|| for a 128-term fp32 sum in any order, used with a 4x margin
            const float xn = sqrtf(red[t][0] + red[t][1]);
            uint32_t code = 0;
            const bool amb = i < r && !fast_code(ys[t][i], 0x1p-15f * pn * xn, step, b, code);
            uint64_t m = __ballot(amb);
            while (m) {
                const int l = __builtin_ctzll(m);
                m &= m - 1;
                const int il = (i & ~63) + l;
                const uint16_t* Prow = P + (int64_t)il * KVC_HEAD_DIM;
                const uint32_t cl = resolve_code_wave(Prow, Prow, xu + (int64_t)t * KVC_HEAD_DIM, step, b, sqrtf(pns[il]), xn, lane);
                if (lane == l) code = cl;
            }
            if (i < r) cs[t][i] = (uint8_t)code;
        }
    }
    __syncthreads();
    if (i >= r) return;
    // Merge, per new token and plane. K: a token's 16 codes of a full coordinate group are 16
    // consecutive slots, i.e. whole 16-bit (p = 1) or 32-bit words that belong to this token alone:
    // the group's lanes OR their fields together and one lane per word stores it. The tail group's
    // fields, and every V code (p bits of a field of 16 tokens shared with other tokens), are written
    // in place with an atomic clear and set of its bits (they never straddle a word).
    // One thread owns each coordinate, so the new tokens of a call are written in order.
    uint8_t* __restrict__ stream = s.codes + s.code_off[u];
    const int g16 = r >> 4, rho = r & 15;
    for (int t = 0; t < n_tok; ++t) {
        const int tok = t0 + t, tile = tok / KVC_TILE_TOKENS, tt = tok % KVC_TILE_TOKENS;
        uint8_t* __restrict__ tbase = stream + (int64_t)tile * 8 * r * b;
        const uint32_t c = cs[t][i];
        for (int k = 0; k < 4; ++k) {
            const int p = b == 8 ? (k == 0 ? 8 : 0) : (k == 0 ? 4 : (k == 1 ? 2 : (k == 2 ? 1 : 0)));
            if (p == 0 || (b != 8 && !(b & p))) continue;
            const int sh = b == 8 ? 0 : (b & (p - 1));
            const int off = b == 8 ? 0 : (b & ~(2 * p - 1));
            const uint32_t pb = p == 8 ? c : (c >> sh) & ((1u << p) - 1u);
            uint8_t* __restrict__ base = tbase + 8 * r * off;
            if (side == KVC_SIDE_K && i < 16 * g16) {
                const int lpw = p >= 4 ? 32 / p : 16;  // lanes whose fields share one stored word
                const int fb = p * (i & 15);            // field bit within the group's run
                uint32_t v = pb << (fb & 31);
                for (int o = 1; o < lpw; o <<= 1) v |= __shfl_xor(v, o);
                if ((i & (lpw - 1)) == 0) {
                    uint8_t* w = base + p * (128 * (i >> 4) + 2 * tt) + (fb >> 3);
                    if (p == 1) *reinterpret_cast<uint16_t*>(w) = (uint16_t)v;
                    else *reinterpret_cast<uint32_t*>(w) = v;
                }
            } else {
                const int bit = side == KVC_SIDE_K ? p * (1024 * g16 + tt * rho + (i - 16 * g16)) : v_plane_bit(tt, i, r, b, p);
                if (p == 8) {
                    base[bit >> 3] = (uint8_t)pb;
                } else {
                    uint32_t* wp = reinterpret_cast<uint32_t*>(base) + (bit >> 5);
                    const uint32_t m = ((1u << p) - 1u) << (bit & 31);
                    atomicAnd(wp, ~m);
                    atomicOr(wp, pb << (bit & 31));
                }
            }
        }
    }
}

}  // namespace
}  // namespace kvc
