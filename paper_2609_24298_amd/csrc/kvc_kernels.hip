// Device half of libkvc, compression side: HIP kernels for CDNA4 (gfx950) and
// their C-ABI launchers (kvc_encode, kvc_reconstruct). Decode attention lives
// in kvc_decode.hip.
//
// Kernels
//  encode_kernel        one (unit, 64-token tile) per 256-thread block: the
//                       fp16 basis is staged in LDS as fp32, each thread
//                       projects one token onto a quarter of the coordinates
//                       in fp32 with a rigorous error bound, undecided codes
//                       are settled exactly in 128-bit integers, and the tile
//                       is bit-packed from LDS with one thread per output word.
//  reconstruct_kernel   x_hat = P^T z for a 64-token block of one unit.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kvc_device.h"
#include "kvc_internal.h"

namespace kvc {

constexpr int kD = KVC_HEAD_DIM;
constexpr int kTile = KVC_TILE_TOKENS;

// ---------------------------------------------------------------- encode

// Exact code: y = sum_j P_ij x_j as an integer multiple of 2^-48 (|y| < 2^88),
// k = clamp(floor(y / step) + 2^(b-1), 0, 2^b - 1) with floor division in
// 128-bit integers. Used only for elements the fp32 path cannot decide.
__device__ __noinline__ uint32_t exact_code(const uint16_t* __restrict__ Prow, const uint16_t* __restrict__ xrow,
                                            float step, int b) {
    __int128 N = 0;
    for (int j = 0; j < kD; ++j) {
        int32_t mp, mx;
        int ep, ex;
        half_parts(Prow[j], mp, ep);
        half_parts(xrow[j], mx, ex);
        N += (__int128)((int64_t)mp * mx) * ((__int128)1 << (ep + ex + 48));
    }
    const uint32_t u = __float_as_uint(step);
    const int64_t m = 0x800000 | (u & 0x7fffff);
    const int sD = (int)((u >> 23) & 255) - 150 + 48;  // >= 1 for step >= 2^-24
    const __int128 D = (__int128)m << sD;
    __int128 q = N / D;
    if (N % D != 0 && N < 0) q -= 1;
    const __int128 k = q + (1 << (b - 1));
    const __int128 kmax = (1 << b) - 1;
    return (uint32_t)(k < 0 ? 0 : (k > kmax ? kmax : k));
}

// Code from the fp32 projection `acc` whose error is at most `err`
// (|acc - y| <= err). Falls back to exact_code when a quantizer threshold
// j * step, j in [1 - 2^(b-1), 2^(b-1) - 1], is not clearly separated.
__device__ __forceinline__ uint32_t decide_code(float acc, float err, float step, int b,
                                                const uint16_t* Prow, const uint16_t* xrow) {
    const int h = 1 << (b - 1);
    const double st = step, yd = acc, ed = err;
    const double t = yd / st;
    bool amb = !(ed < 0.25 * st);
    if (!amb) {
        const double jn = rint(t);
        if (jn >= 1 - h && jn <= h - 1) amb = !(fabs(yd - jn * st) > ed + 0x1p-45 * fabs(yd));
    }
    if (!amb) {
        const double kd = fmin(fmax(floor(t) + h, 0.0), (double)((1 << b) - 1));
        return (uint32_t)kd;
    }
    return exact_code(Prow, xrow, step, b);
}

// Plane of output word w of a tile: width p, bit shift in the code, word index in the plane.
__device__ __forceinline__ void word_plane(int w, int r, int b, int& p, int& shift, int& lw) {
    if (b == 8) { p = 8; shift = 0; lw = w; return; }
    int rem = b;
#pragma unroll
    for (int q = 4; q >= 1; q >>= 1) {
        if (b & q) {
            rem -= q;
            const int nw = 2 * r * q;
            if (w < nw) { p = q; shift = rem; lw = w; return; }
            w -= nw;
        }
    }
    p = 1; shift = 0; lw = w;  // not reached for w < 2*r*b
}

constexpr int kEncThreads = 256;

__global__ __launch_bounds__(kEncThreads) void encode_kernel(DevSide s, int side, const uint16_t* __restrict__ x,
                                                             int64_t x_stride, int t0, int n_tok, int tile_first) {
    extern __shared__ float smem[];
    const int u = blockIdx.y;
    const int tile = tile_first + blockIdx.x;
    const int r = s.r[u], b = s.b[u];
    const float step = s.delta[u];
    const uint16_t* __restrict__ P = s.basis + s.basis_off[u];
    float* Ps = smem;                                   // [r][128] fp32 basis
    float* pn = Ps + r * kD;                            // [r] row norms
    uint8_t* cs = reinterpret_cast<uint8_t*>(pn + kD);  // [64][128] codes

    for (int k = threadIdx.x; k < r * kD; k += kEncThreads) Ps[k] = h2f((P[k]));
    __syncthreads();
    if (threadIdx.x < r) {
        float s2 = 0.f;
        for (int j = 0; j < kD; ++j) s2 = fmaf(Ps[threadIdx.x * kD + j], Ps[threadIdx.x * kD + j], s2);
        pn[threadIdx.x] = sqrtf(s2);
    }

    const int t = threadIdx.x & 63, grp = threadIdx.x >> 6;
    const int tok = tile * kTile + t;
    const bool active = tok >= t0 && tok < t0 + n_tok;
    const uint16_t* xrow = x + (int64_t)u * x_stride + (int64_t)(tok - t0) * kD;
    float xv[kD];
    float xn2 = 0.f;
    if (active) {
        const uint4* xr4 = reinterpret_cast<const uint4*>(xrow);
#pragma unroll
        for (int q = 0; q < kD / 8; ++q) {
            const uint4 v = xr4[q];
            const uint32_t w4[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                xv[8 * q + 2 * e] = h2f(((uint16_t)(w4[e] & 0xffff)));
                xv[8 * q + 2 * e + 1] = h2f(((uint16_t)(w4[e] >> 16)));
            }
        }
#pragma unroll
        for (int j = 0; j < kD; ++j) xn2 = fmaf(xv[j], xv[j], xn2);
    }
    // |acc - y| <= gamma_128 * sum_j |P_ij x_j| <= 2^-17 * ||P_i|| ||x||; 2^-15 leaves a 4x margin
    // for the rounding of the norms themselves.
    const float xn = sqrtf(xn2);
    __syncthreads();
    if (active) {
        for (int i = grp; i < r; i += 4) {
            const float4* Pr = reinterpret_cast<const float4*>(Ps + i * kD);
            float acc = 0.f;
#pragma unroll
            for (int q = 0; q < kD / 4; ++q) {
                const float4 pv = Pr[q];
                acc = fmaf(pv.x, xv[4 * q], acc);
                acc = fmaf(pv.y, xv[4 * q + 1], acc);
                acc = fmaf(pv.z, xv[4 * q + 2], acc);
                acc = fmaf(pv.w, xv[4 * q + 3], acc);
            }
            const float err = 0x1p-15f * pn[i] * xn;
            cs[t * kD + i] = (uint8_t)decide_code(acc, err, step, b, P + (int64_t)i * kD, xrow);
        }
    }
    __syncthreads();

    // Pack: one thread per 32-bit output word; partial tiles keep the other tokens' bits.
    uint32_t* tw = reinterpret_cast<uint32_t*>(s.codes + s.code_off[u] + (int64_t)tile * 8 * r * b);
    const int tok0 = tile * kTile;
    const bool full = tok0 >= t0 && tok0 + kTile <= t0 + n_tok;
    const int n_words = 2 * r * b;
    for (int w = threadIdx.x; w < n_words; w += kEncThreads) {
        int p, shift, lw;
        word_plane(w, r, b, p, shift, lw);
        const int per_word = 32 / p;
        const uint32_t vmask = (1u << p) - 1u;
        uint32_t val = 0, msk = 0;
        for (int iota = 0; iota < per_word; ++iota) {
            const int phi = lw * per_word + iota;
            int tt, i;
            if (side == KVC_SIDE_K) unslot_k(phi, r, tt, i);
            else { i = phi >> 6; tt = psi(phi & 63); }
            const int tk = tok0 + tt;
            if (tk >= t0 && tk < t0 + n_tok) {
                const int bit = 8 * (iota & 3) + p * (iota >> 2);
                val |= ((uint32_t)(cs[tt * kD + i] >> shift) & vmask) << bit;
                msk |= vmask << bit;
            }
        }
        tw[w] = full ? val : ((tw[w] & ~msk) | val);
    }
}

// ---------------------------------------------------------------- append

// Appending a few tokens (a decode step adds one per unit): one block per unit, thread i
// computes coordinate i of every new token from its basis row, decides the code as
// encode_kernel does, and the new codes are merged into the packed words of their tiles.
constexpr int kAppThreads = kD;
constexpr int kAppMaxTok = 4;

__global__ __launch_bounds__(kAppThreads) void append_kernel(DevSide s, int side, const uint16_t* __restrict__ x,
                                                             int64_t x_stride, int t0, int n_tok) {
    __shared__ float xs[kAppMaxTok][kD];
    __shared__ float red[kAppMaxTok][kAppThreads / 64];
    __shared__ uint8_t cs[kAppMaxTok][kD];
    const int u = blockIdx.x, i = threadIdx.x;
    const int r = s.r[u], b = s.b[u];
    const float step = s.delta[u];
    const uint16_t* __restrict__ P = s.basis + s.basis_off[u];
    const uint16_t* __restrict__ xu = x + (int64_t)u * x_stride;
    for (int t = 0; t < n_tok; ++t) {
        const float v = h2f(xu[(int64_t)t * kD + i]);
        xs[t][i] = v;
        float s2 = v * v;
        for (int o = 32; o > 0; o >>= 1) s2 += __shfl_xor(s2, o);
        if ((i & 63) == 0) red[t][i >> 6] = s2;
    }
    __syncthreads();
    if (i < r) {
        float acc[kAppMaxTok] = {0.f, 0.f, 0.f, 0.f};
        float pn2 = 0.f;
        const uint4* Pr = reinterpret_cast<const uint4*>(P + (int64_t)i * kD);
#pragma unroll 4
        for (int q = 0; q < kD / 8; ++q) {
            const uint4 w = Pr[q];
            const uint32_t w4[4] = {w.x, w.y, w.z, w.w};
            float pv[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                pv[2 * e] = h2f((uint16_t)(w4[e] & 0xffff));
                pv[2 * e + 1] = h2f((uint16_t)(w4[e] >> 16));
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                pn2 = fmaf(pv[e], pv[e], pn2);
#pragma unroll
                for (int t = 0; t < kAppMaxTok; ++t)
                    if (t < n_tok) acc[t] = fmaf(pv[e], xs[t][8 * q + e], acc[t]);
            }
        }
        const float pn = sqrtf(pn2);
#pragma unroll
        for (int t = 0; t < kAppMaxTok; ++t)
            if (t < n_tok) {
                // same bound as encode_kernel: |acc - y| <= 2^-17 ||P_i|| ||x||, used with a 4x margin
                const float xn = sqrtf(red[t][0] + red[t][1]);
                cs[t][i] = (uint8_t)decide_code(acc[t], 0x1p-15f * pn * xn, step, b, P + (int64_t)i * kD,
                                                xu + (int64_t)t * kD);
            }
    }
    __syncthreads();
    if (i >= r) return;
    // Merge: thread (t, i) visits the word holding slot (t, i) in each plane. The word's first slot
    // that belongs to a new token elects one thread per word, which rewrites the new tokens' bits
    // of that word and keeps every other bit.
    uint8_t* __restrict__ stream = s.codes + s.code_off[u];
    for (int t = 0; t < n_tok; ++t) {
        const int tok = t0 + t, tile = tok / kTile, tt = tok % kTile;
        const int phi = side == KVC_SIDE_K ? slot_k(tt, i, r) : slot_v(tt, i);
        uint8_t* __restrict__ tbase = stream + (int64_t)tile * 8 * r * b;
        for (int p = 8; p >= 1; p >>= 1) {
            if (b == 8 ? p != 8 : (p == 8 || !(b & p))) continue;
            const int sh = b == 8 ? 0 : (b & (p - 1));
            const int off = b == 8 ? 0 : (b & ~(2 * p - 1));
            const int ppw = 32 / p;
            const uint32_t vmask = p == 8 ? 0xffu : ((1u << p) - 1u);
            const int lw = phi / ppw;
            uint32_t val = 0, msk = 0;
            bool first = true, leader = false;
            for (int iota = 0; iota < ppw; ++iota) {
                const int ph = lw * ppw + iota;
                int t2, i2;
                if (side == KVC_SIDE_K) unslot_k(ph, r, t2, i2);
                else { i2 = ph >> 6; t2 = psi(ph & 63); }
                const int tk = tile * kTile + t2 - t0;
                if (tk >= 0 && tk < n_tok) {
                    if (first) { leader = tk == t && i2 == i; first = false; }
                    const int bit = 8 * (iota & 3) + p * (iota >> 2);
                    val |= ((uint32_t)(cs[tk][i2] >> sh) & vmask) << bit;
                    msk |= vmask << bit;
                }
            }
            if (leader) {
                uint32_t* wp = reinterpret_cast<uint32_t*>(tbase + 8 * r * off) + lw;
                *wp = (*wp & ~msk) | val;
            }
        }
    }
}

// ---------------------------------------------------------------- reconstruct

constexpr int kRecThreads = 256;

__global__ __launch_bounds__(kRecThreads) void reconstruct_kernel(DevSide s, int side, int t0, int n_tok, float* __restrict__ out) {
    extern __shared__ float smem[];
    const int u = blockIdx.y;
    const int blk0 = t0 + blockIdx.x * kTile;  // first token of this block
    const int r = s.r[u], b = s.b[u];
    const float step = s.delta[u];
    const float half = (float)(1 << (b - 1)) - 0.5f;
    const uint16_t* __restrict__ P = s.basis + s.basis_off[u];
    const uint8_t* __restrict__ stream = s.codes + s.code_off[u];
    float* Ps = smem;            // [r][128]
    float* zh = Ps + r * kD;     // [64][r + 1]
    const int zs = r + 1;
    for (int k = threadIdx.x; k < r * kD; k += kRecThreads) Ps[k] = h2f((P[k]));
    for (int k = threadIdx.x; k < kTile * r; k += kRecThreads) {
        const int tt = k / r, i = k - tt * r;
        const int tok = blk0 + tt;
        float z = 0.f;
        if (tok < t0 + n_tok) {
            const uint8_t* tile = stream + (int64_t)(tok / kTile) * 8 * r * b;
            const int tl = tok % kTile;
            const int phi = side == KVC_SIDE_K ? slot_k(tl, i, r) : slot_v(tl, i);
            z = ((float)load_code(tile, r, b, phi) - half) * step;
        }
        zh[tt * zs + i] = z;
    }
    __syncthreads();
    const int j = threadIdx.x & (kD - 1);
    for (int tt = threadIdx.x >> 7; tt < kTile; tt += kRecThreads / kD) {
        const int tok = blk0 + tt;
        if (tok >= t0 + n_tok) break;
        float o = 0.f;
        for (int i = 0; i < r; ++i) o = fmaf(Ps[i * kD + j], zh[tt * zs + i], o);
        out[((int64_t)u * n_tok + (tok - t0)) * kD + j] = o;
    }
}

// ---------------------------------------------------------------- host side

namespace {

int max_r(const kvc_stream_desc* s) {
    int m = 2;
    for (int u = 0; u < s->n_units; ++u) m = s->r_host[u] > m ? s->r_host[u] : m;
    return m;
}

int set_smem_limit(const void* fn, size_t bytes) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return set_error(KVC_EDEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

using namespace kvc;

extern "C" int kvc_encode(const kvc_stream_desc* s, const uint16_t* x, int64_t x_unit_stride, int32_t t0, int32_t n_tok,
                          void* stream) {
    clear_error();
    if (int e = validate_desc(s, "kvc_encode")) return e;
    if (t0 < 0 || n_tok < 0) return set_error(KVC_EINVAL, "kvc_encode: negative t0 or n_tok");
    if ((int64_t)t0 + n_tok > s->capacity) return set_error(KVC_ENOSPACE, "kvc_encode: t0 + n_tok > capacity");
    if (n_tok == 0 || s->n_units == 0) return KVC_OK;
    if (!x || (reinterpret_cast<uintptr_t>(x) & 15) || (x_unit_stride & 7) || x_unit_stride < (int64_t)n_tok * kD)
        return set_error(KVC_EINVAL, "kvc_encode: x must be 16-byte aligned with stride a multiple of 8 and >= n_tok*d");
    if (n_tok <= kAppMaxTok) {
        hipLaunchKernelGGL(append_kernel, dim3(s->n_units), dim3(kAppThreads), 0, (hipStream_t)stream, dev_side(s),
                           s->side, x, x_unit_stride, t0, n_tok);
        return check_launch("kvc_encode");
    }
    const int tile_first = t0 / kTile;
    const int tile_last = (t0 + n_tok - 1) / kTile;
    const size_t smem = (size_t)max_r(s) * kD * 4 + kD * 4 + kTile * kD;
    if (int e = set_smem_limit((const void*)encode_kernel, smem)) return e;
    dim3 grid(tile_last - tile_first + 1, s->n_units);
    hipLaunchKernelGGL(encode_kernel, grid, dim3(kEncThreads), smem, (hipStream_t)stream, dev_side(s), s->side, x,
                       x_unit_stride, t0, n_tok, tile_first);
    return check_launch("kvc_encode");
}

extern "C" int kvc_reconstruct(const kvc_stream_desc* s, int32_t t0, int32_t n_tok, float* out, void* stream) {
    clear_error();
    if (int e = validate_desc(s, "kvc_reconstruct")) return e;
    if (t0 < 0 || n_tok < 0) return set_error(KVC_EINVAL, "kvc_reconstruct: negative t0 or n_tok");
    if ((int64_t)t0 + n_tok > s->capacity) return set_error(KVC_ENOSPACE, "kvc_reconstruct: t0 + n_tok > capacity");
    if (n_tok == 0 || s->n_units == 0) return KVC_OK;
    if (!out) return set_error(KVC_EINVAL, "kvc_reconstruct: null output");
    const int r = max_r(s);
    const size_t smem = (size_t)r * kD * 4 + (size_t)kTile * (r + 1) * 4;
    if (int e = set_smem_limit((const void*)reconstruct_kernel, smem)) return e;
    dim3 grid((n_tok + kTile - 1) / kTile, s->n_units);
    hipLaunchKernelGGL(reconstruct_kernel, grid, dim3(kRecThreads), smem, (hipStream_t)stream, dev_side(s), s->side, t0,
                       n_tok, out);
    return check_launch("kvc_reconstruct");
}
