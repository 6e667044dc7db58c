// Decode attention over the packed KV-COBRA cache on CDNA4 (gfx950): kernels
// and the kvc_decode_attn launcher (table step 8; App. I, "Wall-clock at the
// primitive level").
//
// The logits and the probability-weighted sum of values are dense contractions
// in the rank space: S = Qt (G x r_K) . C_K^T (r_K x tokens) and
// A = P (G x tokens) . C_V (tokens x r_V). Both run on int8 matrix cores
// (v_mfma_i32_16x16x64_i8) with exact int32 accumulation:
//  * codes enter as int8 (raw codes for b <= 7; c - 128 for b = 8);
//  * the rank-space query q~ = P_K q is split into three balanced base-254
//    int8 limbs with a per-query scale (relative error ~1e-7 of max|q~|);
//  * the softmax weights p in [0, 2^6] (relative to the chunk's running max) are
//    quantised to P < 2^31 - 2^24 and split into four byte limbs,
//    P = S0 + 2^8 S1 + 2^16 S2 + 2^24 S3 (S0..S2 signed, S3 in [0, 127]). The
//    quantum is 2^-25 of the running max, so a chunk of n tokens loses at most
//    n 2^-26 of its mass to rounding (<= 2^-12 at the longest chunk, 2^14
//    tokens), whatever the shape of the attention;
//  * centring (c - 2^(b-1)) is exact in integers: the logits subtract
//    2^(b-1) sum_i Q_i, and the value accumulator carries an all-ones virtual
//    coordinate whose column gives sum_t P_t (also the softmax denominator).
//
// One wavefront per work item = (unit, context chunk) walks the chunk in
// 64-token tiles. Each lane loads the packed fields its operand fragments need
// straight into registers with buffer loads at loop-invariant offsets (the
// stream layout puts a token's codes of a group of 16 coordinates, and a
// quarter of 16 tokens of one value coordinate, in one bit field whose
// unpacking lands directly in MFMA operand order); the next tile's loads are in
// flight while the current one is computed. Only the K-step holding the tail
// group (r_K % 16 coordinates, token fields that are not word aligned) is staged
// through LDS and read back with funnel shifts. The logit lane (query head,
// column) receives the three limbs of one (head, token) logit and forms it alone;
// the online softmax keeps a lazily raised running max per head; probability
// limbs go through LDS into the A operand of the PV products, whose int32
// accumulators hold every limb of one (head, coordinate) in one lane, so a raise
// of the max rescales them exactly in place. A second kernel merges the chunks
// and applies step_V and the V basis.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>
#include <utility>

#include "kvc_append.h"
#include "kvc_device.h"
#include "kvc_internal.h"

namespace kvc {

constexpr int kD = KVC_HEAD_DIM;
constexpr int kTile = KVC_TILE_TOKENS;
constexpr int kPartStride = 132;  // floats per (item, query head): m, l, pad, pad, acc[128]
constexpr int kLimbs = 3;
constexpr float kLazy = 6.f;              // the running max is raised only when a tile beats it by > 2^6
constexpr float kPScale = 33292288.f;     // (2^31 - 2^24) / 2^6: p <= 2^6 maps to P <= 2^31 - 2^24
constexpr float kPBias = 8421504.f;       // 0x808080, the offsets of the three signed low limbs; the fma's
                                          // result is >= 2^23, so its rounding to nearest is the rounding of P
// Tiles per chunk at most: |S_l c| <= 2^15 per token keeps the int32 accumulators below 2^31
// (2^29 per chunk, plus at most 2^24 carried into a limb by a rescale), and bounds the rounding
// loss of a chunk's softmax mass (see kPScale).
constexpr int kMaxChunkTiles = 256;
constexpr int kPRowBytes = 80;            // LDS row of the probability limbs (64 tokens + pad)
constexpr uint32_t kLaneOOB = 0x10000000u;  // lane offset (in plane-width units) past any stream
constexpr int kRsrcWord3 = 0x00020000;    // raw buffer, 32-bit data format (gfx9 family)

typedef int32_t v4i __attribute__((ext_vector_type(4)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t perm(uint32_t hi, uint32_t lo, uint32_t sel) {
    return __builtin_amdgcn_perm(hi, lo, sel);
}
__device__ __forceinline__ uint32_t funnel(uint32_t hi, uint32_t lo, uint32_t sh) {
    return __builtin_amdgcn_alignbit(hi, lo, sh);
}

// Maximum over the 16 lanes of a DPP row (row rotations).
template <int N>
__device__ __forceinline__ float row_ror(float v) {
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), 0x120 + N, 0xf, 0xf, true));
}
__device__ __forceinline__ float row_max(float m) {
    m = fmaxf(m, row_ror<8>(m));
    m = fmaxf(m, row_ror<4>(m));
    m = fmaxf(m, row_ror<2>(m));
    return fmaxf(m, row_ror<1>(m));
}

// The partial kernel's work-group is one wavefront, whose LDS accesses execute in program order:
// between an LDS write and a read of the same bytes only the compiler's reordering of memory
// operations has to be stopped, which a wavefront-scope fence does without any wait.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// ---------------------------------------------------------------- field unpacking

// One token's field (16 codes) of one plane: up to four 32-bit words, bit 0 aligned.
struct Fld {
    uint32_t w0, w1, w2, w3;
};

// The 16 codes of a field as int8 operand bytes: byte k of dword d holds the code at position
// kidx_b^-1(4 d + k) of the field, i.e. operand index 4 d + k <-> position pos_b(4 d + k).
// f[k] is plane k's field (widest first); hi1 selects the upper 16 bits of the word of a 1-bit
// plane (two tokens share a word there). b = 8 codes come out centred (c - 128).
template <int B>
__device__ __forceinline__ v4i unpack16(const Fld (&f)[3], bool hi1) {
    uint32_t D[4];
    if constexpr (B == 8) {
        D[0] = f[0].w0 ^ 0x80808080u;
        D[1] = f[0].w1 ^ 0x80808080u;
        D[2] = f[0].w2 ^ 0x80808080u;
        D[3] = f[0].w3 ^ 0x80808080u;
    } else if constexpr (B == 4) {  // nibble order
        constexpr uint32_t M = 0x0f0f0f0fu;
        D[0] = f[0].w0 & M;
        D[1] = (f[0].w0 >> 4) & M;
        D[2] = f[0].w1 & M;
        D[3] = (f[0].w1 >> 4) & M;
    } else {  // position 4 k + d -> byte k of dword d, for every plane
        D[0] = D[1] = D[2] = D[3] = 0u;
#pragma unroll
        for (int k = 0; k < n_planes(B); ++k) {
            const int P = plane_w(B, k), SH = plane_sh(B, k);
            uint32_t E[4];
            if (P == 4) {
                constexpr uint32_t M = 0x0f0f0f0fu;
                const uint32_t t02 = perm(f[k].w1, f[k].w0, 0x06040200u), t13 = perm(f[k].w1, f[k].w0, 0x07050301u);
                E[0] = t02 & M;
                E[1] = (t02 >> 4) & M;
                E[2] = t13 & M;
                E[3] = (t13 >> 4) & M;
            } else if (P == 2) {
                constexpr uint32_t M = 0x03030303u;
#pragma unroll
                for (int d = 0; d < 4; ++d) E[d] = (f[k].w0 >> (2 * d)) & M;
            } else {
                constexpr uint32_t M = 0x01010101u;
                const uint32_t x = perm(f[k].w0 >> 4, f[k].w0, hi1 ? 0x07030602u : 0x05010400u);
#pragma unroll
                for (int d = 0; d < 4; ++d) E[d] = (x >> d) & M;
            }
#pragma unroll
            for (int d = 0; d < 4; ++d) D[d] |= E[d] << SH;
        }
    }
    return v4i{(int)D[0], (int)D[1], (int)D[2], (int)D[3]};
}

// Words of a K-step held per lane: 8 p bytes per plane of width p, either the fields of the lane's
// four tokens (direct) or its share of the staged region (the K-step holding the tail group: the
// plane's bytes from 512 p ks on, at most 496 p of them, 8 p bytes per lane).
__host__ __device__ constexpr int k_step_words(int b) { return 2 * b; }
__host__ __device__ constexpr int plane_stage_off(int b, int k) { return 512 * plane_off(b, k); }  // LDS bytes
constexpr int kKBufWords = 16;  // prefetch registers per side
// K-steps' words kept in the prefetch registers: both K-steps of the widths where they fit, also for the
// structure taken at run time (KM < 0); the one K-step of ranks <= 64 (KM >= 2) for every width.
__host__ __device__ constexpr bool k_prefetch_on(int b, int km) {
    return 2 * k_step_words(b) <= kKBufWords || (km >= 2 && k_step_words(b) <= kKBufWords);
}
// The second K-step's load is issued (absent K-steps read past the stream and return zero) wherever
// its words fit the registers, so that every tile issues the same loads.
__host__ __device__ constexpr bool k_second_load(int b) { return 2 * k_step_words(b) <= kKBufWords; }
constexpr int kVBufWords = 16;  // value prefetch registers
constexpr int kPrefetchDepth = 2;  // tiles of K and V loads in flight ahead of the one being processed (the
                                    // general path keeps one: its per-tile width switches need the registers)

// Value groups (v_field_off): a plane of width p keeps the fields of v_group(p) = 8 / p consecutive
// N-tiles of a lane together (16 bytes), so a lane reads a group of one plane with one 16-byte load.
__host__ __device__ constexpr int v_group(int p) { return v_group_ntiles(p); }
__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }
// Prefetch registers taken by the groups of the first n N-tiles, plane k's groups starting at word
// v_pf_base(b, k, n), and the N-tiles prefetched for a rank bound of NV N-tiles (whole groups that
// fit kVBufWords; the groups past them are loaded while the tile is processed).
__host__ __device__ constexpr int v_pf_base(int b, int k, int n) {
    int w = 0;
    for (int j = 0; j < k; ++j) w += 4 * cdiv(n, v_group(plane_w(b, j)));
    return w;
}
__host__ __device__ constexpr int v_pf_words(int b, int n) { return v_pf_base(b, n_planes(b), n); }
__host__ __device__ constexpr int v_pf_tiles(int b, int nv) {
    int n = nv;
    while (n > 0 && v_pf_words(b, n) > kVBufWords) --n;
    return n;
}

// Direct loads of one K-step's fields into w[0 .. 2B).
template <int B>
__device__ __forceinline__ void k_load_direct(const __amdgpu_buffer_rsrc_t rs, int r, uint32_t lk, uint32_t* w) {
    int o = 0;
#pragma unroll
    for (int k = 0; k < n_planes(B); ++k) {
        const int P = plane_w(B, k);
        const int voff = (int)(P * lk) + 8 * r * plane_off(B, k);
        if (P == 1) {
            const v2u v = __builtin_amdgcn_raw_buffer_load_b64(rs, voff, 0, 0);
            w[o] = v[0];
            w[o + 1] = v[1];
        } else {
#pragma unroll
            for (int q = 0; q < P / 2; ++q) {
                const v4u v = __builtin_amdgcn_raw_buffer_load_b128(rs, voff + 16 * q, 0, 0);
                w[o + 4 * q] = v[0];
                w[o + 4 * q + 1] = v[1];
                w[o + 4 * q + 2] = v[2];
                w[o + 4 * q + 3] = v[3];
            }
        }
        o += 2 * P;
    }
}

// The lane's share of the staged region goes to LDS at 8 p lane of the plane's area.
template <int B>
__device__ __forceinline__ void k_write_stage(const uint32_t* w, uint8_t* __restrict__ stage, int lane) {
    int o = 0;
#pragma unroll
    for (int k = 0; k < n_planes(B); ++k) {
        const int P = plane_w(B, k);
        uint8_t* dst = stage + plane_stage_off(B, k) + 8 * P * lane;
        if (P == 1) {
            *reinterpret_cast<v2u*>(dst) = v2u{w[o], w[o + 1]};
        } else {
#pragma unroll
            for (int q = 0; q < P / 2; ++q)
                *reinterpret_cast<v4u*>(dst + 16 * q) = v4u{w[o + 4 * q], w[o + 4 * q + 1], w[o + 4 * q + 2], w[o + 4 * q + 3]};
        }
        o += 2 * P;
    }
}

// Operand fragment of token st (0..3 of the lane's four) from one K-step's directly loaded fields.
template <int B>
__device__ __forceinline__ v4i k_frag_direct(const uint32_t* w, int st) {
    Fld f[3];
    int o = 0;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        if (k < n_planes(B)) {
            const int P = plane_w(B, k);
            if (P == 1) f[k] = Fld{w[o + (st >> 1)], 0u, 0u, 0u};
            else if (P == 2) f[k] = Fld{w[o + st], 0u, 0u, 0u};
            else if (P == 4) f[k] = Fld{w[o + 2 * st], w[o + 2 * st + 1], 0u, 0u};
            else f[k] = Fld{w[o + 4 * st], w[o + 4 * st + 1], w[o + 4 * st + 2], w[o + 4 * st + 3]};
            o += 2 * P;
        } else {
            f[k] = Fld{0u, 0u, 0u, 0u};
        }
    }
    return unpack16<B>(f, (st & 1) != 0);
}

// Operand fragment of a token from the staged K-step: its field of plane k starts at bit p * x of the
// plane's staged region.
template <int B>
__device__ __forceinline__ v4i k_frag_staged(const uint8_t* __restrict__ stage, uint32_t x) {
    Fld f[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        if (k < n_planes(B)) {
            const int P = plane_w(B, k);
            const uint32_t bit = x * (uint32_t)P;
            const uint32_t* s32 = reinterpret_cast<const uint32_t*>(stage + plane_stage_off(B, k)) + (bit >> 5);
            const uint32_t d0 = s32[0], d1 = s32[1];
            if (P <= 2) {
                f[k] = Fld{funnel(d1, d0, bit), 0u, 0u, 0u};
            } else if (P == 4) {
                const uint32_t d2 = s32[2];
                f[k] = Fld{funnel(d1, d0, bit), funnel(d2, d1, bit), 0u, 0u};
            } else {
                const uint32_t d2 = s32[2], d3 = s32[3], d4 = s32[4];
                f[k] = Fld{funnel(d1, d0, bit), funnel(d2, d1, bit), funnel(d3, d2, bit), funnel(d4, d3, bit)};
            }
        } else {
            f[k] = Fld{0u, 0u, 0u, 0u};
        }
    }
    return unpack16<B>(f, false);
}

template <int B>
__device__ __forceinline__ void k_fetch(uint32_t* w, const __amdgpu_buffer_rsrc_t rs, int rk, uint32_t lk) {
    k_load_direct<B>(rs, rk, lk, w);
}

// Prefetch of a unit's first tile (both K-steps, for the widths whose two K-steps fit the prefetch
// registers; wider codes are loaded when their tile is processed).
template <int B, int KM>
__device__ __forceinline__ void k_prefetch(uint32_t (&kb)[kKBufWords], const __amdgpu_buffer_rsrc_t rs, int rk, int nk,
                                           int ks_t, const uint32_t (&LK)[2], int lane) {
    constexpr int W0 = k_step_words(B);
    (void)nk;
    if constexpr (k_prefetch_on(B, KM)) {
        k_fetch<B>(kb, rs, rk, LK[0]);
        if constexpr (k_second_load(B)) k_fetch<B>(kb + W0, rs, rk, LK[1]);
    }
}

// Logit of token 4 col + st for the lane's heads: three int32 limb sums -> log2-domain value + off.
template <int LM>
__device__ __forceinline__ void logit_of(const v4i (&acc)[LM], const float (&k0)[LM], const float (&k1)[LM],
                                         const float (&k2)[LM], const float (&off)[LM], float (&s)[LM][4], int st) {
#pragma unroll
    for (int lm = 0; lm < LM; ++lm) {
        float v = fmaf((float)acc[lm][2], k2[lm], off[lm]);
        v = fmaf((float)acc[lm][1], k1[lm], v);
        s[lm][st] = fmaf((float)acc[lm][0], k0[lm], v);
    }
}

// Logits of one tile: s[lm][st] = logit + off for the lane's four tokens. The K-step holding the tail
// group (if any) is staged in LDS; its token fields start at plane-width units xb + st xs. For the
// widths whose two K-steps are prefetched, each token column is finished right after its MFMAs and
// the next tile's fields are loaded into the freed registers; wider codes load each K-step here.
template <int B, int LM, int KM>
__device__ __forceinline__ void k_tile(uint32_t (&kb)[kKBufWords], uint32_t (&kb_next)[kKBufWords], bool stage_next,
                                       const __amdgpu_buffer_rsrc_t rs,
                                       const __amdgpu_buffer_rsrc_t rs_n, int rk, int nk_rt, int ks_t_rt,
                                       const uint32_t (&LK)[2], uint32_t xb, uint32_t xs, int lane,
                                       uint8_t* __restrict__ stage, const v4i (&qa)[2][LM], const float (&k0)[LM],
                                       const float (&k1)[LM], const float (&k2)[LM], const float (&off)[LM],
                                       float (&s)[LM][4]) {
    constexpr int W0 = k_step_words(B);
    // K-step structure fixed at compile time when KM >= 0 (see k_mode), else taken at run time
    const int nk = KM >= 0 ? (KM < 2 ? 2 : 1) : nk_rt;
    const int ks_t = KM >= 0 ? (KM == 1 ? 1 : (KM == 3 ? 0 : 2)) : ks_t_rt;
    if constexpr (k_prefetch_on(B, KM)) {
        // The staged K-step goes to LDS first (constant indices into kb: a runtime one would move the
        // array to scratch memory). Every load below is issued unconditionally, in the same order on
        // every tile (absent K-steps read past the stream and return zero), so that the wait for a
        // tile's data counts exactly the younger loads still in flight.
        // The staged K-step of this tile is already in LDS when the caller staged it one tile ahead
        // (stage_next on the previous tile); otherwise it is written now.
        // Widths whose second K-step does not fit are prefetched only with one K-step (KM >= 2), and
        // their code below never forms the second K-step's registers.
        constexpr bool kTwo = k_second_load(B);
        if (!stage_next) {
            if (ks_t == 0) {
                k_write_stage<B>(kb, stage, lane);
                wave_lds_sync();
            } else if constexpr (kTwo) {
                if (ks_t == 1 && nk > 1) {
                    k_write_stage<B>(kb + W0, stage, lane);
                    wave_lds_sync();
                }
            }
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            v4i acc[LM];
            {
                const v4i bk = ks_t == 0 ? k_frag_staged<B>(stage, xb + st * xs) : k_frag_direct<B>(kb, st);
#pragma unroll
                for (int lm = 0; lm < LM; ++lm) acc[lm] = mfma_i8(qa[0][lm], bk, v4i{0, 0, 0, 0});
            }
            if constexpr (kTwo) {
                if (nk > 1) {
                    const v4i bk = ks_t == 1 ? k_frag_staged<B>(stage, xb + st * xs) : k_frag_direct<B>(kb + W0, st);
#pragma unroll
                    for (int lm = 0; lm < LM; ++lm) acc[lm] = mfma_i8(qa[1][lm], bk, acc[lm]);
                }
            }
            logit_of<LM>(acc, k0, k1, k2, off, s, st);
        }
        k_load_direct<B>(rs_n, rk, LK[0], kb);
        if constexpr (kTwo) k_load_direct<B>(rs_n, rk, LK[1], kb + W0);
        // stage the next tile's K-step (loaded into the other register set one tile ago) now, away from
        // the loop head
        if (stage_next) {
            wave_lds_sync();
            if (ks_t == 0) k_write_stage<B>(kb_next, stage, lane);
            else if constexpr (kTwo) {
                if (ks_t == 1 && nk > 1) k_write_stage<B>(kb_next + W0, stage, lane);
            }
            wave_lds_sync();
        }
    } else {
        v4i S[LM][4];
#pragma unroll
        for (int lm = 0; lm < LM; ++lm)
#pragma unroll
            for (int st = 0; st < 4; ++st) S[lm][st] = v4i{0, 0, 0, 0};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            if (ks >= nk) break;
            k_fetch<B>(kb, rs, rk, LK[ks]);
            if (ks == ks_t) {
                k_write_stage<B>(kb, stage, lane);
                wave_lds_sync();
            }
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                const v4i bk = ks == ks_t ? k_frag_staged<B>(stage, xb + st * xs) : k_frag_direct<B>(kb, st);
#pragma unroll
                for (int lm = 0; lm < LM; ++lm) S[lm][st] = mfma_i8(qa[ks][lm], bk, S[lm][st]);
            }
            if (ks == ks_t) wave_lds_sync();
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            v4i acc[LM];
#pragma unroll
            for (int lm = 0; lm < LM; ++lm) acc[lm] = S[lm][st];
            logit_of<LM>(acc, k0, k1, k2, off, s, st);
        }
    }
}

// Group Q of plane k for this lane: field index L = 4 col + grp of every N-tile in the group, the
// lane's fields in N-tile order. Groups before the last hold g N-tiles (16 bytes per lane, lanes in
// order); the last holds the remaining m N-tiles, the lanes of coordinates col >= ct (the coordinates
// of a partial last N-tile) one field fewer, so lane L starts A = 4 max(0, col - ct) + [col >= ct] grp
// fields before L m. Groups past the rank read beyond it (bounded by the stream) into accumulator
// columns that are never output.
template <int B>
__device__ __forceinline__ v4u v_group_load(const __amdgpu_buffer_rsrc_t rs, int k, int Q, int r, uint32_t L,
                                            uint32_t A) {
    const int P = plane_w(B, k), g = v_group(P);
    const int nvt = (r + 15) >> 4;
    const int ql = (nvt - 1) / g, m = nvt - g * ql;
    const uint32_t in = Q == ql ? (uint32_t)(2 * P) * (L * (uint32_t)m - A) : 16u * L;
    const int voff = 8 * r * plane_off(B, k) + 1024 * Q + (int)in;
    // A multiple of 4 bytes, except for 1-bit planes, whose last group (the only one, r <= 128) may start
    // a lane's fields at 2 mod 4 bytes: the load takes the dword-aligned 16 bytes below (the lane's
    // fields, at most 14 bytes in that case, stay inside them) and v_tile shifts them into place.
    return __builtin_amdgcn_raw_buffer_load_b128(rs, voff & ~3, 0, 0);
}

// A of the lane (col, grp) for rank r.
__device__ __forceinline__ uint32_t v_lane_adj(int r, int col, int grp) {
    const int ct = r - 16 * (((r + 15) >> 4) - 1);
    return col >= ct ? (uint32_t)(4 * (col - ct) + grp) : 0u;
}

// Loads of the prefetched groups whose last N-tile (below NV) is nt, plane by plane: the prefetch of a
// tile issues them for nt = 0, 1, .. in the same order as the processing of a tile refills them.
template <int B, int NV>
__device__ __forceinline__ void v_refill(uint32_t* vb, const __amdgpu_buffer_rsrc_t rs, int r, uint32_t L, uint32_t A,
                                         int nt) {
    constexpr int NPF = v_pf_tiles(B, NV);
#pragma unroll
    for (int k = 0; k < n_planes(B); ++k) {
        const int g = v_group(plane_w(B, k)), Q = nt / g;
        const int last = (Q + 1) * g < NV ? (Q + 1) * g - 1 : NV - 1;
        if (Q < cdiv(NPF, g) && nt == last) {
            const v4u v = v_group_load<B>(rs, k, Q, r, L, A);
            uint32_t* w = vb + v_pf_base(B, k, NPF) + 4 * Q;
            w[0] = v[0];
            w[1] = v[1];
            w[2] = v[2];
            w[3] = v[3];
        }
    }
}

template <int B, int NV>
__device__ __forceinline__ void v_prefetch(uint32_t (&vb)[kVBufWords], const __amdgpu_buffer_rsrc_t rs, int r,
                                           uint32_t L, uint32_t A) {
#pragma unroll
    for (int nt = 0; nt < NV; ++nt) v_refill<B, NV>(vb, rs, r, L, A, nt);
}

// PV MFMAs of one tile (N-tiles nt < NV, a compile-time bound on the rank's N-tiles; the prefetched
// groups come from vb, the rest are loaded here as their first N-tile comes), then the next tile's
// prefetch (rs_next; a zero-sized descriptor when there is none).
template <int B, int LM, int NV>
__device__ __forceinline__ void v_tile(uint32_t* vb, const __amdgpu_buffer_rsrc_t rs, const __amdgpu_buffer_rsrc_t rs_next,
                                       int r, uint32_t L, uint32_t A, const v4i (&ap)[LM], v4i (&C)[LM][9]) {
    constexpr int NPF = v_pf_tiles(B, NV);
    // Every N-tile below NV is processed, also those past the rank: no branches, and every tile issues
    // the same loads in the same order, so the waits for a tile's data stay exact.
    uint32_t gw[3][4], w1[4];
#pragma unroll
    for (int nt = 0; nt < NV; ++nt) {
        Fld f[3];
        bool hi = false;
#pragma unroll
        for (int k = 0; k < 3; ++k) {
            if (k < n_planes(B)) {
                const int P = plane_w(B, k), g = v_group(P), Q = nt / g, j = nt % g;
                const bool pf = Q < cdiv(NPF, g);
                if (!pf && j == 0) {
                    const v4u v = v_group_load<B>(rs, k, Q, r, L, A);
                    gw[k][0] = v[0];
                    gw[k][1] = v[1];
                    gw[k][2] = v[2];
                    gw[k][3] = v[3];
                }
                const uint32_t* w = pf ? vb + v_pf_base(B, k, NPF) + 4 * Q : gw[k];
                if (P == 1) {
                    // one group of m = ceil(r / 16) N-tiles: the lane's fields start at bit 16 (m L - A)
                    // mod 32 of the dword-aligned words; they are shifted down once, on the group's
                    // first N-tile, where the words are used (a shift right after the load would wait
                    // for it)
                    if (j == 0) {
                        const uint32_t sh = ((L * (uint32_t)((r + 15) >> 4) - A) & 1u) << 4;
                        w1[0] = funnel(w[1], w[0], sh);
                        w1[1] = funnel(w[2], w[1], sh);
                        w1[2] = funnel(w[3], w[2], sh);
                        w1[3] = w[3] >> sh;
                    }
                    f[k] = Fld{w1[j >> 1], 0u, 0u, 0u};
                    hi = (j & 1) != 0;
                } else if (P == 2) {
                    f[k] = Fld{w[j], 0u, 0u, 0u};
                } else if (P == 4) {
                    f[k] = Fld{w[2 * j], w[2 * j + 1], 0u, 0u};
                } else {
                    f[k] = Fld{w[0], w[1], w[2], w[3]};
                }
            } else {
                f[k] = Fld{0u, 0u, 0u, 0u};
            }
        }
        const v4i bv = unpack16<B>(f, hi);
#pragma unroll
        for (int pm = 0; pm < LM; ++pm) C[pm][nt] = mfma_i8(ap[pm], bv, C[pm][nt]);
        v_refill<B, NV>(vb, rs_next, r, L, A, nt);
    }
}

// ---------------------------------------------------------------- q~ limbs

// Per unit: q~_g = (step_K log2(e) / sqrt(d)) P_K q_g, sigma_g = max|q~_g| / 127 and three int8
// limbs with q~ ~ sigma (L0 + L1/254 + L2/254^2). The limbs are written as the logit MFMA's A
// operand of every lane: qa[u][ks][lm][lane] = 16 bytes, lane (grp, row = 4 (h % 4) + limb), lm = h / 4,
// operand byte m <-> coordinate 16 (4 ks + grp) + pos_b(m) (zero outside the rank, for limb 3 and for
// heads >= G). qk[u][h] = (sigma, sigma / 254, sigma / 254^2, bias) with
// bias = -2^(b-1) sum_limb k_limb sum_i L_limb,i (0 for b = 8, whose codes are centred on load).
typedef _Float16 qp_h8 __attribute__((ext_vector_type(8)));
typedef float qp_f4 __attribute__((ext_vector_type(4)));

// NW wavefronts per unit (1 when the units fill the device, 8 for a few units), wavefront w taking
// row blocks [w 8/NW, (w + 1) 8/NW). The projection Y = P_K Q (rank rows x query-head columns) runs on
// v_mfma_f32_16x16x32_f16 (exact fp16 products, fp32 accumulation): A = 16 basis rows x 32
// coordinates, B = 32 coordinates x 16 heads, four k-steps per row block, every operand loaded
// straight from global memory with up to four row blocks' loads in flight. Lane (kq, col) then holds
// rows 16 rb + 4 kq + v of head col; a head's max and limb sums reduce over its four lanes, then over
// the wavefronts through LDS.
template <int NW>
__device__ __forceinline__ void qprep_unit(const DevSide& K, const uint16_t* __restrict__ q, int G, int LM,
                                           v4i* __restrict__ qa, float4* __restrict__ qk, const int u) {
    constexpr int RB = 8 / NW;                 // row blocks per wavefront
    constexpr int HALF = RB > 4 ? 2 : 1;       // rounds of at most four row blocks' loads
    constexpr int RQ = RB / HALF;
    extern __shared__ uint8_t img[];  // [2][LM][64][16] operand image
    __shared__ float red_m[NW][16];
    __shared__ int red_l[NW][16][kLimbs];
    const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63, col = lane & 15, kq = lane >> 4;
    const int r = K.r[u], b = K.b[u];
    const uint16_t* __restrict__ P = K.basis + K.basis_off[u];
    const int img_words = 2 * LM * 64 * 4;
    for (int k = threadIdx.x; k < img_words; k += 64 * NW) reinterpret_cast<uint32_t*>(img)[k] = 0u;
    __syncthreads();
    qp_f4 C[RB];
#pragma unroll
    for (int j = 0; j < RB; ++j) C[j] = qp_f4{0.f, 0.f, 0.f, 0.f};
    for (int h0 = 0; h0 < G; h0 += 16) {  // heads in groups of 16 columns
        const int g = h0 + col;
        qp_h8 B[4];
#pragma unroll
        for (int k4 = 0; k4 < 4; ++k4) {
            const uint4 w = g < G ? reinterpret_cast<const uint4*>(q + ((int64_t)u * G + g) * kD + 32 * k4 + 8 * kq)[0]
                                  : uint4{0u, 0u, 0u, 0u};
            B[k4] = __builtin_bit_cast(qp_h8, w);
        }
#pragma unroll
        for (int half = 0; half < HALF; ++half) {
            uint4 A[RQ][4];
#pragma unroll
            for (int rq = 0; rq < RQ; ++rq)
#pragma unroll
                for (int k4 = 0; k4 < 4; ++k4) {
                    const int row = 16 * (RB * wv + RQ * half + rq) + col;
                    A[rq][k4] = row < r ? reinterpret_cast<const uint4*>(P + (int64_t)row * kD + 32 * k4 + 8 * kq)[0]
                                        : uint4{0u, 0u, 0u, 0u};
                }
#pragma unroll
            for (int rq = 0; rq < RQ; ++rq) {
                qp_f4 c = qp_f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int k4 = 0; k4 < 4; ++k4)
                    c = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(qp_h8, A[rq][k4]), B[k4], c, 0, 0, 0);
                C[RQ * half + rq] = c;
            }
        }
        const int hk = b == 8 ? 0 : (1 << (b - 1));
        const float scale0 = K.delta[u] * 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)
        float m = 0.f;
#pragma unroll
        for (int j = 0; j < RB; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                C[j][v] *= scale0;
                m = fmaxf(m, fabsf(C[j][v]));
            }
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        if constexpr (NW > 1) {
            if (kq == 0) red_m[wv][col] = m;
            __syncthreads();
#pragma unroll
            for (int w = 0; w < NW; ++w) m = fmaxf(m, red_m[w][col]);
        }
        const float sigma = m > 0.f ? m / 127.f : 1.f;
        const int g16 = r >> 4;
        int lsum[kLimbs] = {0, 0, 0};
#pragma unroll
        for (int j = 0; j < RB; ++j)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int i = 16 * (RB * wv + j) + 4 * kq + v;  // rank coordinate
                if (i < r && g < G) {
                    const float x = C[j][v] / sigma;
                    const float l0 = fminf(fmaxf(rintf(x), -127.f), 127.f);
                    const float r1 = (x - l0) * 254.f;
                    const float l1 = fminf(fmaxf(rintf(r1), -127.f), 127.f);
                    const float r2 = (r1 - l1) * 254.f;
                    const float l2 = fminf(fmaxf(rintf(r2), -127.f), 127.f);
                    const int L[kLimbs] = {(int)l0, (int)l1, (int)l2};
                    // destination of coordinate i in the operand image
                    const int cg = i < 16 * g16 ? (i >> 4) : g16;
                    const int jpos = i - 16 * cg;
                    const int ks = cg >> 2, grp = cg & 3;
                    const int kidx = kidx_b(b, jpos);
#pragma unroll
                    for (int k = 0; k < kLimbs; ++k) {
                        img[(((ks * LM + (g >> 2)) * 64 + 16 * grp + 4 * (g & 3) + k) << 4) + kidx] = (uint8_t)(int8_t)L[k];
                        lsum[k] += L[k];
                    }
                }
            }
#pragma unroll
        for (int k = 0; k < kLimbs; ++k) {
            lsum[k] += __shfl_xor(lsum[k], 16);
            lsum[k] += __shfl_xor(lsum[k], 32);
        }
        if constexpr (NW > 1) {
            if (kq == 0)
#pragma unroll
                for (int k = 0; k < kLimbs; ++k) red_l[wv][col][k] = lsum[k];
            __syncthreads();
#pragma unroll
            for (int k = 0; k < kLimbs; ++k) {
                lsum[k] = 0;
#pragma unroll
                for (int w = 0; w < NW; ++w) lsum[k] += red_l[w][col][k];
            }
        }
        if (wv == 0 && kq == 0 && g < G) {
            const float k0 = sigma, k1 = sigma * (1.f / 254.f), k2 = sigma * (1.f / 64516.f);
            const float bias = -(float)hk * ((float)lsum[0] * k0 + (float)lsum[1] * k1 + (float)lsum[2] * k2);
            qk[(int64_t)u * G + g] = float4{k0, k1, k2, bias};
        }
        if constexpr (NW > 1) __syncthreads();  // red_m, red_l are rewritten by the next head group
    }
    __syncthreads();
    v4i* dst = qa + (int64_t)u * 2 * LM * 64;
    for (int k = threadIdx.x; k < 2 * LM * 64; k += 64 * NW) dst[k] = reinterpret_cast<const v4i*>(img)[k];
}

template <int NW>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2, 2))) void qprep_kernel(
    DevSide K, const uint16_t* __restrict__ q, int G, int LM, v4i* __restrict__ qa, float4* __restrict__ qk) {
    qprep_unit<NW>(K, q, G, LM, qa, qk, blockIdx.x);
}

// The first launch of a fused decode step (kvc_decode_step): block (u, 0) projects unit u's queries
// (two wavefronts, four row blocks each), blocks (u, 1) and (u, 2) append the new token's key and
// value to unit u's streams (the append of kvc_encode_kv). The decode partials, launched next on the
// same stream, read the appended codes.
constexpr int kStepPrepThreads = 128;
static_assert(kStepPrepThreads == kAppThreads, "the append uses one thread per coordinate");
// Three wavefronts per SIMD (166 registers, none spilled): 1.5 times the resident blocks of the
// unconstrained allocation, so the 3 x units blocks run in fewer rounds.
#ifndef KVC_DECODE_PARTIALS_UNIT
__global__ __launch_bounds__(kStepPrepThreads) __attribute__((amdgpu_waves_per_eu(3, 3))) void step_prep_kernel(
    DevSide K, DevSide V, const uint16_t* __restrict__ q, int G, int LM, v4i* __restrict__ qa, float4* __restrict__ qk,
    const uint16_t* __restrict__ xk, int64_t xk_stride, const uint16_t* __restrict__ xv, int64_t xv_stride, int t_new) {
    if (blockIdx.y == 0) qprep_unit<2>(K, q, G, LM, qa, qk, blockIdx.x);
    else if (blockIdx.y == 1) append_unit(K, KVC_SIDE_K, xk, xk_stride, t_new, 1, blockIdx.x);
    else append_unit(V, KVC_SIDE_V, xv, xv_stride, t_new, 1, blockIdx.x);
}
#endif

// ---------------------------------------------------------------- partials

template <int G> struct Shape {
    static constexpr int LM = (G + 3) / 4;  // M-tiles of 16 rows = 4 heads x 4 limb slots (logits and PV)
    // Wavefronts per SIMD the register budget is cut for (512 / W registers per lane, no spills).
    static constexpr int W = G <= 4 ? 3 : (G == 8 ? 2 : 1);
};

// Runs a KVC_SWITCH_B-style CALL with B_ = the compile-time width BKc (BVc), or switches on the
// runtime width when it is 0.
#define KVC_SW_K(CALL)                                          \
    if constexpr (BKc != 0) {                                   \
        constexpr int B_ = BKc;                                 \
        CALL;                                                   \
    } else {                                                    \
        KVC_SWITCH_B(bk, CALL);                                 \
    }
#define KVC_SW_V(CALL)                                          \
    if constexpr (BVc != 0) {                                   \
        constexpr int B_ = BVc;                                 \
        CALL;                                                   \
    } else {                                                    \
        KVC_SWITCH_B(bv, CALL);                                 \
    }

// One work item (unit u, context chunk [start, end)) with the K and V bit widths fixed at compile
// time (BKc in 1..8, BVc in 1..4), or switched per tile (0: the general path for values wider than 4).
extern __shared__ __attribute__((aligned(16))) uint8_t kvc_dsm[];

// K-step structure of a rank: 0: two K-steps, no tail group; 1: two K-steps, the tail group in the
// second; 2: one K-step, no tail group; 3: one K-step holding the tail group.
__host__ __device__ constexpr int k_mode(int r) {
    return r > 64 ? ((r & 15) ? 1 : 0) : ((r & 15) ? 3 : 2);
}

// Wave-uniform copies of values the compiler cannot prove uniform (kept in scalar registers).
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ const uint8_t* uni(const uint8_t* p) {
    const uint64_t a = reinterpret_cast<uint64_t>(p);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a), hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return reinterpret_cast<const uint8_t*>(((uint64_t)hi << 32) | lo);
}

// Inlined into the kernel: each instantiation is a disjoint branch of the dispatch, so registers
// are allocated per branch, and no call frame saves registers to scratch memory on every item.
template <int G, int BKc, int BVc, int KM, int NVc>
__device__ __attribute__((always_inline)) void run_item(const DevSide& K, const DevSide& V, const v4i* __restrict__ qa_ws,
                                         const float4* __restrict__ qk_ws, int k_cap_tiles, int v_cap_tiles, int u,
                                         int start, int end, float* __restrict__ out, int lane) {
    constexpr int LM = Shape<G>::LM;
    constexpr int kDepth = KM >= 0 ? kPrefetchDepth : 1;
    uint8_t* pmat = kvc_dsm;                            // [16 LM][kPRowBytes] probability limbs
    uint8_t* stage = kvc_dsm + 16 * LM * kPRowBytes;    // staged tail K-step
    const int col = lane & 15, grp = lane >> 4;
    u = uni(u);
    start = uni(start);
    end = uni(end);
    k_cap_tiles = uni(k_cap_tiles);
    v_cap_tiles = uni(v_cap_tiles);
    const int rk = uni(K.r[u]), bk = uni(K.b[u]), rv = uni(V.r[u]), bv = uni(V.b[u]);
    const int hv = bv == 8 ? 0 : (1 << (bv - 1));
    const int nk = (rk + 63) >> 6, nv = (rv + 15) >> 4;
    const int g16 = rk >> 4, rho = rk & 15;
    const int ks_t = rho ? (g16 >> 2) : 2;  // K-step holding the tail group (2: none)
    const int ktb = 8 * rk * bk, vtb = 8 * rv * bv;
    const int tile0 = start / kTile, tile_last = (end - 1) / kTile;
    const uint8_t* kstream = uni(K.codes + K.code_off[u]);
    const uint8_t* vstream = uni(V.codes + V.code_off[u]);
    // Descriptor of tile t of a stream (bounds: the stream's end); none past the chunk.
    auto k_rs = [&](int t) {
        const bool ok = t <= tile_last;
        return __builtin_amdgcn_make_buffer_rsrc((void*)(kstream + (int64_t)t * ktb), (short)0,
                                                 ok ? (k_cap_tiles - t) * ktb : 0, kRsrcWord3);
    };
    auto v_rs = [&](int t) {
        const bool ok = t <= tile_last;
        return __builtin_amdgcn_make_buffer_rsrc((void*)(vstream + (int64_t)t * vtb), (short)0,
                                                 ok ? (v_cap_tiles - t) * vtb : 0, kRsrcWord3);
    };

    // lane constants (plane-width units): direct K fields of K-step ks (group 4 ks + grp, tokens 4 col ..),
    // value fields (coordinate col of the N-tile, quarter grp), staged tail positions.
    uint32_t LK[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int cg = 4 * ks + grp;
        LK[ks] = ks == ks_t ? (uint32_t)(512 * ks + 8 * lane) : (cg < g16 ? (uint32_t)(128 * cg + 8 * col) : kLaneOOB);
    }
    const uint32_t LV = (uint32_t)(4 * col + grp), VA = v_lane_adj(rv, col, grp);
    uint32_t XB = 0, XS = 0;  // staged token fields start at plane-width units XB + st XS
    {
        const int nf = g16 - 4 * (ks_t < 2 ? ks_t : 0);  // full groups in the staged K-step
        if (grp < nf) { XB = (uint32_t)((64 * grp + 4 * col) * 16); XS = 16; }
        else if (grp == nf) { XB = (uint32_t)(nf * 1024 + 4 * col * rho); XS = (uint32_t)rho; }
    }

    // q~ limbs (A operands of the logits) and per-head scale factors
    v4i qa[2][LM];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int lm = 0; lm < LM; ++lm) qa[ks][lm] = qa_ws[(((int64_t)u * 2 + ks) * LM + lm) * 64 + lane];
    float k0[LM], k1[LM], k2[LM], bias[LM], mrun[LM], mb[LM];
#pragma unroll
    for (int lm = 0; lm < LM; ++lm) {
        const int h = 4 * lm + grp;
        const float4 v = h < G ? qk_ws[(int64_t)u * G + h] : float4{0.f, 0.f, 0.f, 0.f};
        k0[lm] = v.x; k1[lm] = v.y; k2[lm] = v.z; bias[lm] = v.w;
        mrun[lm] = -INFINITY;
        mb[lm] = 0.f;  // bias - mrun once the first tile has set mrun
    }
    for (int k = lane; k < 16 * LM * kPRowBytes / 4; k += 64) reinterpret_cast<uint32_t*>(pmat)[k] = 0u;
    wave_lds_sync();

    v4i C[LM][9];
#pragma unroll
    for (int pm = 0; pm < LM; ++pm)
#pragma unroll
        for (int nt = 0; nt < 9; ++nt) C[pm][nt] = v4i{0, 0, 0, 0};
    const uint32_t one = col == 0 ? 0x01010101u : 0u;
    const v4i ones = v4i{(int)one, (int)one, (int)one, (int)one};

    // Prefetch registers: with a depth of 2, tile t is processed from set t % 2 while the loads of
    // tile t + 1 (the other set) are in flight, and set t % 2 is refilled with tile t + 2 as it is
    // consumed; with a depth of 1 there is one set, refilled with tile t + 1.
    uint32_t kbA[kKBufWords], vbA[kVBufWords], kbB[kKBufWords], vbB[kVBufWords];
#pragma unroll
    for (int k = 0; k < kKBufWords; ++k) kbA[k] = kbB[k] = 0u;
#pragma unroll
    for (int k = 0; k < kVBufWords; ++k) vbA[k] = vbB[k] = 0u;
    {
        // issued in the loop's own order (K-steps, then value N-tiles, per set), so that the waits at
        // the loop head count the same younger loads on entry as on the back edge
        const auto krs = k_rs(tile0), vrs = v_rs(tile0);
        KVC_SW_K((k_prefetch<B_, KM>(kbA, krs, rk, nk, ks_t, LK, lane)));
        __builtin_amdgcn_sched_barrier(0);
        KVC_SW_V((v_prefetch<B_, NVc>(vbA, vrs, rv, LV, VA)));
        __builtin_amdgcn_sched_barrier(0);
        if constexpr (kDepth == 2) {
            const auto krs1 = k_rs(tile0 + 1), vrs1 = v_rs(tile0 + 1);
            KVC_SW_K((k_prefetch<B_, KM>(kbB, krs1, rk, nk, ks_t, LK, lane)));
            __builtin_amdgcn_sched_barrier(0);
            KVC_SW_V((v_prefetch<B_, NVc>(vbB, vrs1, rv, LV, VA)));
            __builtin_amdgcn_sched_barrier(0);
        }
    }

    auto step = [&](const int tile, uint32_t (&kb)[kKBufWords], uint32_t (&vb)[kVBufWords],
                    uint32_t (&kb_next)[kKBufWords], const bool stage_next) {
        const int tok0 = tile * kTile;
        const bool first = tile == tile0;
        const auto krs = k_rs(tile), vrs = v_rs(tile);
        const auto krs_n = k_rs(tile + kDepth), vrs_n = v_rs(tile + kDepth);
        // Opaque per-tile copies of the lane and rank constants: the offsets every bit width derives
        // from them are recomputed inside the loop instead of being hoisted and kept live across it
        // for all eight widths at once.
        uint32_t LKt[2] = {LK[0], LK[1]}, XBt = XB, XSt = XS, LVt = LV, VAt = VA;
        int rkt = rk, rvt = rv;
        if constexpr (BKc == 0 || BVc == 0) {
            asm volatile("" : "+v"(LKt[0]), "+v"(LKt[1]), "+v"(LVt), "+v"(VAt), "+v"(XBt), "+v"(XSt));
            asm volatile("" : "+s"(rkt), "+s"(rvt));
        }
        const int nkt = nk, kst = ks_t;

        // ---- logits, log2 domain, less the running max (the raw logits on the first tile)
        float s[LM][4];
        {
            float off[LM];
#pragma unroll
            for (int lm = 0; lm < LM; ++lm) off[lm] = first ? bias[lm] : mb[lm];
            KVC_SW_K((k_tile<B_, LM, KM>(kb, kb_next, stage_next, krs, krs_n, rkt, nkt, kst, LKt, XBt, XSt, lane, stage, qa, k0, k1, k2, off, s)));
        }

        // ---- online softmax
        const bool last = tok0 + kTile > end;
        bool raise = first;
        if (last) {  // tokens past the end of the chunk
#pragma unroll
            for (int lm = 0; lm < LM; ++lm)
#pragma unroll
                for (int st = 0; st < 4; ++st)
                    if (tok0 + 4 * col + st >= end) s[lm][st] = -INFINITY;
        }
        if constexpr (G % 4 != 0) {  // rows of heads past G
#pragma unroll
            for (int lm = 0; lm < LM; ++lm)
                if (4 * lm + grp >= G) s[lm][0] = s[lm][1] = s[lm][2] = s[lm][3] = -INFINITY;
        }
        // A head's row max beats kLazy exactly when one of its lanes' own maxima does: the common
        // path tests the lane maxima only and takes the cross-lane row max inside the rare branch.
        float ml[LM];
#pragma unroll
        for (int lm = 0; lm < LM; ++lm) {
            ml[lm] = fmaxf(fmaxf(s[lm][0], s[lm][1]), fmaxf(s[lm][2], s[lm][3]));
            raise = raise || ml[lm] > kLazy;
        }
        if (__any(raise)) {
            float mx[LM];
#pragma unroll
            for (int lm = 0; lm < LM; ++lm) mx[lm] = row_max(ml[lm]);
            // Raise the max of each head whose tile beats it by more than 2^kLazy (every head on the
            // first tile) to the tile's own max, and rescale that head's accumulators (every limb of a
            // (head, coordinate) sits in this lane): value = C0 + 2^8 C1 + 2^16 C2 + 2^24 C3 (exact in
            // fp64: |value| <= 2^53) -> rint(value alpha), split again into C3 and three bytes.
#pragma unroll
            for (int lm = 0; lm < LM; ++lm) {
                if ((first && mx[lm] > -INFINITY) || mx[lm] > kLazy) {
                    const float mold = mrun[lm];
                    const float shift = first ? 0.f : mold;  // s + shift = the raw logit
                    const float mnew = mx[lm] + shift;
                    const float alpha = first ? 0.f : exp2f(mold - mnew);
                    mrun[lm] = mnew;
                    mb[lm] = bias[lm] - mnew;
#pragma unroll
                    for (int st = 0; st < 4; ++st) s[lm][st] = (s[lm][st] + shift) - mnew;
                    if (!first) {
                        const double a = (double)alpha;
#pragma unroll
                        for (int nt = 0; nt < 9; ++nt) {
                            const double v = ((double)C[lm][nt][0] + 256.0 * (double)C[lm][nt][1]) +
                                             (65536.0 * (double)C[lm][nt][2] + 16777216.0 * (double)C[lm][nt][3]);
                            const double vs = rint(v * a);
                            const double c3 = floor(vs * (1.0 / 16777216.0));
                            const double r3 = vs - 16777216.0 * c3;  // [0, 2^24): exact from here on
                            const double c2 = floor(r3 * (1.0 / 65536.0));
                            const double r2 = r3 - 65536.0 * c2;
                            const double c1 = floor(r2 * (1.0 / 256.0));
                            C[lm][nt][3] = (int)c3;
                            C[lm][nt][2] = (int)c2;
                            C[lm][nt][1] = (int)c1;
                            C[lm][nt][0] = (int)(r2 - 256.0 * c1);
                        }
                    }
                }
            }
        }

        // ---- probability limbs: P'' = round(p kPScale) + 0x808080; bytes 0, 1, 2 (xor 0x80) and 3 are
        // the limbs S0..S3 with P = S0 + 2^8 S1 + 2^16 S2 + 2^24 S3. Row 4 h + limb, bytes 4 col + st.
#pragma unroll
        for (int lm = 0; lm < LM; ++lm) {
            uint32_t P[4];
#pragma unroll
            for (int st = 0; st < 4; ++st)
                P[st] = (uint32_t)fmaf(__builtin_amdgcn_exp2f(s[lm][st]), kPScale, kPBias);
            const uint32_t q01 = perm(P[1], P[0], 0x05010400u), q23 = perm(P[3], P[2], 0x05010400u);
            const uint32_t r01 = perm(P[1], P[0], 0x07030602u), r23 = perm(P[3], P[2], 0x07030602u);
            const uint32_t L0 = perm(q23, q01, 0x05040100u) ^ 0x80808080u;
            const uint32_t L1 = perm(q23, q01, 0x07060302u) ^ 0x80808080u;
            const uint32_t L2 = perm(r23, r01, 0x05040100u) ^ 0x80808080u;
            const uint32_t L3 = perm(r23, r01, 0x07060302u);
            // every lane writes (heads past G have -inf logits, so zero limbs): no divergent LDS writes
            uint8_t* row = pmat + (16 * lm + 4 * grp) * kPRowBytes + 4 * col;
            *reinterpret_cast<uint32_t*>(row) = L0;
            *reinterpret_cast<uint32_t*>(row + kPRowBytes) = L1;
            *reinterpret_cast<uint32_t*>(row + 2 * kPRowBytes) = L2;
            *reinterpret_cast<uint32_t*>(row + 3 * kPRowBytes) = L3;
        }
        wave_lds_sync();
        v4i ap[LM];
#pragma unroll
        for (int pm = 0; pm < LM; ++pm)
            ap[pm] = *reinterpret_cast<const v4i*>(pmat + (16 * pm + col) * kPRowBytes + 16 * grp);

        // ---- PV (value N-tiles, then the all-ones column)
        KVC_SW_V((v_tile<B_, LM, NVc>(vb, vrs, vrs_n, rvt, LVt, VAt, ap, C)));
#pragma unroll
        for (int pm = 0; pm < LM; ++pm) C[pm][8] = mfma_i8(ap[pm], ones, C[pm][8]);
        wave_lds_sync();  // pmat is rewritten by the next tile
    };
    if constexpr (kDepth == 2) {
        // pairs of tiles in a straight-line body (the load-wait counts stay exact across the back edge)
        // The staged (tail) K-step of tile t + 1 goes to LDS at the end of tile t's logits (the first
        // tile's before the loop); the general path stages each tile itself.
        constexpr bool kAhead = KM >= 0 && k_prefetch_on(BKc, KM);
        if constexpr (kAhead) {
            if (ks_t == 0) k_write_stage<BKc>(kbA, stage, lane);
            else if constexpr (k_second_load(BKc)) {
                if (ks_t == 1) k_write_stage<BKc>(kbA + k_step_words(BKc), stage, lane);
            }
            wave_lds_sync();
        }
        int tile = tile0;
        for (; tile + 1 <= tile_last; tile += 2) {
            step(tile, kbA, vbA, kbB, kAhead);
            step(tile + 1, kbB, vbB, kbA, kAhead);
        }
        if (tile <= tile_last) step(tile, kbA, vbA, kbB, kAhead);
    } else {
        for (int tile = tile0; tile <= tile_last; ++tile) step(tile, kbA, vbA, kbA, false);
    }

    // Partial of each head: m, l = sum of P (all-ones column), centred accumulator. Lane (grp, col)
    // holds every limb of head 4 pm + grp at coordinate 16 nt + col; the all-ones column is col 0.
#pragma unroll
    for (int pm = 0; pm < LM; ++pm) {
        const int h = 4 * pm + grp;
        const int o0 = __shfl(C[pm][8][0], lane & 48), o1 = __shfl(C[pm][8][1], lane & 48),
                  o2 = __shfl(C[pm][8][2], lane & 48), o3 = __shfl(C[pm][8][3], lane & 48);
        if (G % 4 == 0 || h < G) {
            float* o = out + h * kPartStride;
            if (col == 0) {
                o[0] = mrun[pm];
                o[1] = ((float)o0 + 256.f * (float)o1) + (65536.f * (float)o2 + 16777216.f * (float)o3);
            }
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) {
                const int cc = 16 * nt + col;
                if (nt < nv) {
                    const int a0 = C[pm][nt][0] - hv * o0, a1 = C[pm][nt][1] - hv * o1, a2 = C[pm][nt][2] - hv * o2,
                              a3 = C[pm][nt][3] - hv * o3;
                    o[4 + cc] = cc < rv ? ((float)a0 + 256.f * (float)a1) + (65536.f * (float)a2 + 16777216.f * (float)a3)
                                        : 0.f;
                }
            }
        }
    }
}

#undef KVC_SW_K
#undef KVC_SW_V

// Token of logit column col in sub-tile st is 4 col + st: a lane's four tokens are consecutive, so
// its K fields are one contiguous load, and its probability limbs are one dword per limb in LDS.
template <int G>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(Shape<G>::W, Shape<G>::W))) void decode_partial_kernel(
    DevSide K, DevSide V, const v4i* __restrict__ qa_ws, const float4* __restrict__ qk_ws,
    const int32_t* __restrict__ seq_len, int max_seq, int chunk, int n_chunks, int k_cap_tiles, int v_cap_tiles,
    float* __restrict__ part) {
    constexpr int LM = Shape<G>::LM;

    const int u = blockIdx.y, c = blockIdx.x, lane = threadIdx.x;
    const int col = lane & 15, grp = lane >> 4;
    int T = seq_len[u];
    T = T < 0 ? 0 : (T > max_seq ? max_seq : T);
    const int start = c * chunk;
    const int end = min(T, start + chunk);
    float* __restrict__ out = part + ((int64_t)u * n_chunks + c) * G * kPartStride;
    if (start >= end) {
        if (lane < G) { out[lane * kPartStride] = -INFINITY; out[lane * kPartStride + 1] = 0.f; }
        return;
    }
    const int bk = K.b[u], bv = V.b[u];
    // Compiled per (b_K, b_V, K-step structure) for value widths up to 4 and the common group sizes;
    // the general path switches on the widths per tile.
    if constexpr (G == 4 || G == 8) {
        if (bv <= 4) {
            // Value ranks <= 64 (four N-tiles) at 1-3 bits with keys up to 4 bits, and 3-bit values at
            // rank <= 96 (six N-tiles), have instantiations of their own.
            const int rv = V.r[u];
            const int nvc = rv <= 64 && bk <= 4 && bv <= 3 ? 2 : (bv == 3 && rv <= 96 ? 1 : 0);
            switch ((((bk - 1) * 4 + (bv - 1)) * 4 + k_mode(K.r[u])) * 3 + nvc) {
#define KVC_ITEM(BK, BV, KM, NV)                                                                                  \
    case (((BK - 1) * 4 + (BV - 1)) * 4 + KM) * 3 + (NV == 6 ? 1 : (NV == 4 ? 2 : 0)):                          \
        run_item<G, BK, BV, KM, NV>(K, V, qa_ws, qk_ws, k_cap_tiles, v_cap_tiles, u, start, end, out, lane);    \
        return;
#define KVC_ITEM4(BK, BV) KVC_ITEM(BK, BV, 0, 8) KVC_ITEM(BK, BV, 1, 8) KVC_ITEM(BK, BV, 2, 8) KVC_ITEM(BK, BV, 3, 8)
#define KVC_ITEM4N(BK, BV, NV) KVC_ITEM(BK, BV, 0, NV) KVC_ITEM(BK, BV, 1, NV) KVC_ITEM(BK, BV, 2, NV) KVC_ITEM(BK, BV, 3, NV)
#define KVC_ITEM4S(BK) KVC_ITEM4(BK, 3) KVC_ITEM4N(BK, 3, 6)
#define KVC_ITEMN4(BK) KVC_ITEM4N(BK, 1, 4) KVC_ITEM4N(BK, 2, 4) KVC_ITEM4N(BK, 3, 4)
                KVC_ITEM4(1, 1) KVC_ITEM4(1, 2) KVC_ITEM4S(1) KVC_ITEM4(1, 4) KVC_ITEMN4(1)
                KVC_ITEM4(2, 1) KVC_ITEM4(2, 2) KVC_ITEM4S(2) KVC_ITEM4(2, 4) KVC_ITEMN4(2)
                KVC_ITEM4(3, 1) KVC_ITEM4(3, 2) KVC_ITEM4S(3) KVC_ITEM4(3, 4) KVC_ITEMN4(3)
                KVC_ITEM4(4, 1) KVC_ITEM4(4, 2) KVC_ITEM4S(4) KVC_ITEM4(4, 4) KVC_ITEMN4(4)
                KVC_ITEM4(5, 1) KVC_ITEM4(5, 2) KVC_ITEM4S(5) KVC_ITEM4(5, 4)
                KVC_ITEM4(6, 1) KVC_ITEM4(6, 2) KVC_ITEM4S(6) KVC_ITEM4(6, 4)
                KVC_ITEM4(7, 1) KVC_ITEM4(7, 2) KVC_ITEM4S(7) KVC_ITEM4(7, 4)
                KVC_ITEM4(8, 1) KVC_ITEM4(8, 2) KVC_ITEM4S(8) KVC_ITEM4(8, 4)
#undef KVC_ITEMN4
#undef KVC_ITEM4N
#undef KVC_ITEM4S
#undef KVC_ITEM4
#undef KVC_ITEM
                default: break;
            }
        }
    }
    run_item<G, 0, 0, -1, 8>(K, V, qa_ws, qk_ws, k_cap_tiles, v_cap_tiles, u, start, end, out, lane);
}

// The instantiations for 4 and 8 query heads per KV head are compiled in translation units of their
// own (kvc_decode_g4.hip, kvc_decode_g8.hip), in parallel with this one.
#ifndef KVC_DECODE_PARTIALS_UNIT
extern template __global__ void decode_partial_kernel<4>(DevSide, DevSide, const v4i*, const float4*, const int32_t*, int,
                                                         int, int, int, int, float*);
extern template __global__ void decode_partial_kernel<8>(DevSide, DevSide, const v4i*, const float4*, const int32_t*, int,
                                                         int, int, int, int, float*);
#endif

// ---------------------------------------------------------------- RoPE-aware partials

// Keys are cached before the rotary position embedding (Sec. 5, scope), so a model with RoPE scores the
// rotated query q' against each reconstructed key rotated at its own position; that depends on the
// position and cannot be folded into a rank-space query. Per 64-token tile, in four blocks of 16 tokens:
//  1. the block's centred K codes (c - 2^(b-1) + 1/2, exact in fp16) go to LDS, token-major;
//  2. K^T (128 features x 16 tokens) = P_K^T Z^T on v_mfma_f32_16x16x32_f16, with P_K^T staged in LDS once
//     per block of four wavefronts (the four context chunks of one unit share it); lane (col, kq) then
//     holds features 16 rb + 4 kq + v of token col, so both members of every rotation pair (j, j + 64)
//     sit in the same lane;
//  3. each pair is rotated by the angle p theta_j, the position's turns computed as the tile's start
//     (fp64, one frequency per lane) plus the offset inside the tile (fp32);
//  4. the logits q' . K_rot on the same matrix instruction, K_rot split into fp16 hi + lo and q' permuted
//     to the lane's feature order (the order of the k index of a dot product is free);
// then the online softmax and the rank-space PV products exactly as in the partials kernel (int8 value
// codes, probability limbs through LDS, int32 accumulators), writing the same partials, which the
// combine kernel merges.
constexpr int kRopeWaves = 4;
constexpr int kPtPitch = 136;   // halves per feature row of the staged P_K^T (coordinates 0..127 + pad)
constexpr int kZPitch = 136;    // halves per token row of a staged 16-token block of centred K codes
constexpr int kRopeKTile = 8 * kD * 8;  // bytes of the widest K tile (r = 128, b = 8)
constexpr int kRopeShared = kD * kPtPitch * 2 + 64 * 8;  // LDS shared by a block's wavefronts: P_K^T, E16
constexpr int kRopeKChunks = kRopeKTile / 16 / 64;  // 16-byte loads per lane for one K tile
// Blocks of 16 tokens processed together (their chains are independent and share each P_K^T operand
// read): as many as the register file allows for the group size.
__host__ __device__ constexpr int rope_blocks(int G) { return G <= 8 ? 2 : 1; }
__host__ __device__ constexpr int rope_wave_lds(int G) {
    return kRopeKTile + rope_blocks(G) * 16 * kZPitch * 2 + 16 * ((G + 3) / 4) * kPRowBytes + 64 * 4;
}

typedef _Float16 rp_h8 __attribute__((ext_vector_type(8)));
typedef float rp_f4 __attribute__((ext_vector_type(4)));

// Position of coordinate i in a staged row of centred K codes (and in the staged P_K^T): inside each
// group of 16, coordinates m and m + 8 (m < 8) are neighbours, at 2 m and 2 m + 1, so that a pair of
// codes converts to fp16 as one packed dword. The k order of the reconstruction's products is free.
__host__ __device__ constexpr int zpos(int i) { return (i & ~15) | ((i & 7) << 1) | ((i >> 3) & 1); }

// A 16-code field of one plane of width p (codes 16 g + m at bits p m), aligned at bit 0 in f[0 .. p / 2)
// (f[0] low 16 bits for p = 1), as the pairs (m, m + 8): bits [0, p) and [16, 16 + p) of pr[m], the rest
// of each half zero.
template <int P>
__device__ __forceinline__ void plane_pairs(const uint32_t (&f)[4], uint32_t (&pr)[8]) {
    if constexpr (P == 1) {
        const uint32_t y = (f[0] & 0xffu) | ((f[0] & 0xff00u) << 8);  // code m + 8 at bit 16 + m
#pragma unroll
        for (int m = 0; m < 8; ++m) pr[m] = (y >> m) & 0x00010001u;
    } else if constexpr (P == 2) {
#pragma unroll
        for (int m = 0; m < 8; ++m) pr[m] = (f[0] >> (2 * m)) & 0x00030003u;
    } else if constexpr (P == 4) {
        const uint32_t y01 = perm(f[1], f[0], 0x05040100u), y23 = perm(f[1], f[0], 0x07060302u);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
            pr[m] = (y01 >> (4 * m)) & 0x000f000fu;
            pr[m + 4] = (y23 >> (4 * m)) & 0x000f000fu;
        }
    } else {
#pragma unroll
        for (int m = 0; m < 8; ++m)  // byte m % 4 of dwords m / 4 and m / 4 + 2, zero bytes between
            pr[m] = perm(f[(m >> 2) + 2], f[m >> 2], 0x0c040c00u + 0x00010001u * (uint32_t)(m & 3));
    }
}

// The fields of group g of token t of a K tile, aligned: a whole group's field of a plane of width p is
// 16 p bits at bit p (1024 g + 16 t) of the plane; the tail group's (rho = r % 16 codes) starts at
// bit p (1024 g16 + t rho) and is aligned with funnel shifts over five words (codes past rho are other
// tokens' codes: finite, and they meet zero basis entries).
template <int P>
__device__ __forceinline__ void group_field(const uint8_t* __restrict__ plane, bool tail, int g, int g16, int rho, int t,
                                            uint32_t (&f)[4]) {
    if (!tail) {
        const uint8_t* base = plane + P * (128 * g + 2 * t);
        if constexpr (P == 1) {
            f[0] = *reinterpret_cast<const uint16_t*>(base);
        } else if constexpr (P == 2) {
            f[0] = *reinterpret_cast<const uint32_t*>(base);
        } else if constexpr (P == 4) {
            const uint2 v2 = *reinterpret_cast<const uint2*>(base);
            f[0] = v2.x; f[1] = v2.y;
        } else {
            const uint4 v4 = *reinterpret_cast<const uint4*>(base);
            f[0] = v4.x; f[1] = v4.y; f[2] = v4.z; f[3] = v4.w;
        }
    } else {
        const uint32_t bit0 = (uint32_t)(P * (1024 * g16 + t * rho));
        const uint32_t* w = reinterpret_cast<const uint32_t*>(plane) + (bit0 >> 5);
        const uint32_t d0 = w[0], d1 = w[1];
        f[0] = funnel(d1, d0, bit0);
        if constexpr (P >= 4) {
            const uint32_t d2 = w[2];
            f[1] = funnel(d2, d1, bit0);
            if constexpr (P == 8) {
                const uint32_t d3 = w[3], d4 = w[4];
                f[2] = funnel(d3, d2, bit0);
                f[3] = funnel(d4, d3, bit0);
            }
        }
    }
}

// Stage the centred K codes (c - 2^(b-1) + 1/2, exact in fp16) of token t for the lane's two groups
// 2 kq, 2 kq + 1 into its row of ZT, in zpos order: per code pair, the planes' bits are combined one
// bit up, under the fp16 exponent of 512 (512 + c, exact: the spacing there is 1/2), and moved by one
// packed add of -512 - 2^(b-1) + 1/2 (also exact).
template <int B>
__device__ __forceinline__ void rope_stage_codes(const uint8_t* __restrict__ ktile, int rk, int g16, int rho, int kq,
                                                 int t, uint16_t* __restrict__ zrow) {
    typedef _Float16 h2v __attribute__((ext_vector_type(2)));
    const _Float16 sh = (_Float16)(-512.f - ((float)(1 << (B - 1)) - 0.5f));
    const h2v sh2 = h2v{sh, sh};
#pragma unroll
    for (int gg = 0; gg < 2; ++gg) {
        const int g = 2 * kq + gg;
        const bool tail = g >= g16;
        uint32_t pc[8];
#pragma unroll
        for (int m = 0; m < 8; ++m) pc[m] = 0u;
#pragma unroll
        for (int k = 0; k < n_planes(B); ++k) {
            const int P = plane_w(B, k), SH = plane_sh(B, k), OFF = plane_off(B, k);
            uint32_t f[4] = {0u, 0u, 0u, 0u}, pr[8];
            const uint8_t* plane = ktile + 8 * rk * OFF;
            if (P == 1) { group_field<1>(plane, tail, g, g16, rho, t, f); plane_pairs<1>(f, pr); }
            else if (P == 2) { group_field<2>(plane, tail, g, g16, rho, t, f); plane_pairs<2>(f, pr); }
            else if (P == 4) { group_field<4>(plane, tail, g, g16, rho, t, f); plane_pairs<4>(f, pr); }
            else { group_field<8>(plane, tail, g, g16, rho, t, f); plane_pairs<8>(f, pr); }
#pragma unroll
            for (int m = 0; m < 8; ++m) pc[m] |= pr[m] << (SH + 1);
        }
        uint32_t hw[8];
#pragma unroll
        for (int m = 0; m < 8; ++m)
            hw[m] = __builtin_bit_cast(uint32_t, __builtin_bit_cast(h2v, pc[m] | 0x60006000u) + sh2);
        *reinterpret_cast<uint4*>(zrow + 16 * g) = uint4{hw[0], hw[1], hw[2], hw[3]};
        *reinterpret_cast<uint4*>(zrow + 16 * g + 8) = uint4{hw[4], hw[5], hw[6], hw[7]};
    }
}

template <int G>
__global__ __launch_bounds__(64 * kRopeWaves) void decode_rope_kernel(
    DevSide K, DevSide V, const uint16_t* __restrict__ q, const int32_t* __restrict__ seq_len, int max_seq, int chunk,
    int n_chunks, int v_cap_tiles, float log2_base, float* __restrict__ part) {
    constexpr int LM = Shape<G>::LM;
    extern __shared__ __attribute__((aligned(16))) uint8_t rope_sm[];
    const int u = blockIdx.y, wv = uni((int)(threadIdx.x >> 6)), lane = threadIdx.x & 63;
    const int col = lane & 15, kq = lane >> 4, grp = kq;
    const int rk = uni(K.r[u]), bk = uni(K.b[u]);
    uint16_t* PT = reinterpret_cast<uint16_t*>(rope_sm);  // [128 features][kPtPitch]
    float2* E16 = reinterpret_cast<float2*>(rope_sm + kRopeShared - 64 * 8);  // [64 pairs] rotation by 16 positions
    if (threadIdx.x < 64) {
        // cos, sin of the rotation of pair j by 16 positions (turns reduced in fp64)
        const int j = threadIdx.x;
        const double w = exp2(-(double)j / 64.0 * (double)log2_base) * 0.15915494309189535;
        const float t16 = (float)(6.283185307179586 * (16.0 * w - floor(16.0 * w)));
        E16[j] = float2{cosf(t16), sinf(t16)};
    }
    {
        // stage P_K^T: zero it (coordinates past the rank take part in the last 32-wide k-step), then
        // transpose the basis rows in
        for (int e = threadIdx.x; e < kD * kPtPitch / 8; e += 64 * kRopeWaves)
            reinterpret_cast<uint4*>(PT)[e] = uint4{0u, 0u, 0u, 0u};
        __syncthreads();
        const uint16_t* __restrict__ P = K.basis + K.basis_off[u];
        for (int e = threadIdx.x; e < rk * (kD / 8); e += 64 * kRopeWaves) {
            const int i = e / (kD / 8), f0 = 8 * (e % (kD / 8));
            const uint4 w = reinterpret_cast<const uint4*>(P + (int64_t)i * kD)[f0 / 8];
            const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int k = 0; k < 8; ++k) PT[(f0 + k) * kPtPitch + zpos(i)] = (uint16_t)(ww[k >> 1] >> (16 * (k & 1)));
        }
        __syncthreads();
    }
    const int c = blockIdx.x * kRopeWaves + wv;
    if (c >= n_chunks) return;  // no block-wide barrier follows
    constexpr int NB = rope_blocks(G);
    uint8_t* wbase = rope_sm + kRopeShared + wv * rope_wave_lds(G);
    uint8_t* KS = wbase;                                               // the K tile being processed
    uint16_t* ZT = reinterpret_cast<uint16_t*>(wbase + kRopeKTile);     // [NB blocks][16 tokens][kZPitch]
    uint8_t* pmat = wbase + kRopeKTile + NB * 16 * kZPitch * 2;        // [16 LM][kPRowBytes]
    float* rho0 = reinterpret_cast<float*>(pmat + 16 * LM * kPRowBytes);  // [64] tile start, turns

    int T = uni(seq_len[u]);
    T = T < 0 ? 0 : (T > max_seq ? max_seq : T);
    const int start = uni(c * chunk);
    const int end = uni(min(T, start + chunk));
    float* __restrict__ out = part + ((int64_t)u * n_chunks + c) * G * kPartStride;
    if (start >= end) {
        if (lane < G) { out[lane * kPartStride] = -INFINITY; out[lane * kPartStride + 1] = 0.f; }
        return;
    }
    const int rv = uni(V.r[u]), bv = uni(V.b[u]);
    const int hv = bv == 8 ? 0 : (1 << (bv - 1));
    const int nks = (rk + 31) >> 5, nv = (rv + 15) >> 4, g16 = rk >> 4, rho = rk & 15;
    const int ktb = 8 * rk * bk, vtb = 8 * rv * bv;
    const int tile0 = uni(start / kTile), tile_last = uni((end - 1) / kTile);
    const uint8_t* kstream = uni(K.codes + K.code_off[u]);
    const uint8_t* vstream = uni(V.codes + V.code_off[u]);
    v_cap_tiles = uni(v_cap_tiles);
    auto v_rs = [&](int t) {
        const bool ok = t <= tile_last;
        return __builtin_amdgcn_make_buffer_rsrc((void*)(vstream + (int64_t)t * vtb), (short)0,
                                                 ok ? (v_cap_tiles - t) * vtb : 0, kRsrcWord3);
    };
    // K tile t as one range-checked descriptor (reads past the tile return zero; none past the chunk)
    auto k_rs = [&](int t) {
        return __builtin_amdgcn_make_buffer_rsrc((void*)(kstream + (int64_t)t * ktb), (short)0, t <= tile_last ? ktb : 0,
                                                 kRsrcWord3);
    };
    // the K tile's bytes, 16 per lane and load, in flight one tile ahead
    v4u kpf[kRopeKChunks];
    auto k_fetch = [&](int t) {
        const auto rs = k_rs(t);
#pragma unroll
        for (int m = 0; m < kRopeKChunks; ++m) kpf[m] = __builtin_amdgcn_raw_buffer_load_b128(rs, 16 * (lane + 64 * m), 0, 0);
    };
    // q' as the logits' A operand: row = head (col), k-step ks, element e <-> feature 16 (2 ks + e / 4) + 4 kq + e % 4
    rp_h8 qa[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int f = 16 * (2 * ks + (e >> 2)) + 4 * kq + (e & 3);
            qa[ks][e] = col < G ? __builtin_bit_cast(_Float16, q[((int64_t)u * G + col) * kD + f]) : (_Float16)0.f;
        }
    // rotation frequencies of the lane's pairs j = 16 rb + 4 kq + v (rb < 4), in turns per position
    float om[4][4];
#pragma unroll
    for (int rb = 0; rb < 4; ++rb)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int j = 16 * rb + 4 * kq + v;
            om[rb][v] = (float)(exp2(-(double)j / 64.0 * (double)log2_base) * 0.15915494309189535);
        }
    const double om_lane = exp2(-(double)lane / 64.0 * (double)log2_base) * 0.15915494309189535;  // frequency j = lane
    const float scale = K.delta[u] * 1.4426950408889634f * 0.08838834764831845f;  // step_K log2(e) / sqrt(128)

    float mrun[4];  // running max of heads 4 kq + v (log2 domain), replicated over the group's 16 lanes
#pragma unroll
    for (int v = 0; v < 4; ++v) mrun[v] = -INFINITY;
    for (int k = lane; k < 16 * LM * kPRowBytes / 4; k += 64) reinterpret_cast<uint32_t*>(pmat)[k] = 0u;
    v4i C[LM][9];
#pragma unroll
    for (int pm = 0; pm < LM; ++pm)
#pragma unroll
        for (int nt = 0; nt < 9; ++nt) C[pm][nt] = v4i{0, 0, 0, 0};
    const uint32_t one = col == 0 ? 0x01010101u : 0u;
    const v4i ones = v4i{(int)one, (int)one, (int)one, (int)one};
    uint32_t vb[kVBufWords];
#pragma unroll
    for (int k = 0; k < kVBufWords; ++k) vb[k] = 0u;
    const uint32_t LV = (uint32_t)(4 * col + grp), VA = v_lane_adj(rv, col, grp);
    {
        const auto vrs = v_rs(tile0);
        KVC_SWITCH_B(bv, (v_prefetch<B_, 8>(vb, vrs, rv, LV, VA)));
    }
    k_fetch(tile0);

    for (int tile = tile0; tile <= tile_last; ++tile) {
        // the K tile to LDS, then the next tile's loads go out
#pragma unroll
        for (int m = 0; m < kRopeKChunks; ++m)
            if (16 * (lane + 64 * m) < ktb) *reinterpret_cast<v4u*>(KS + 16 * (lane + 64 * m)) = kpf[m];
        k_fetch(tile + 1);
        const int tok0 = tile * kTile;
        // Opaque per-tile copies of the widths, ranks and lane offsets: the addresses every width's branch
        // derives from them are recomputed inside the loop, not hoisted and kept live for all widths.
        int rkt = rk, bkt = bk, rvt = rv, bvt = bv, nvt = nv, g16t = g16, rhot = rho, nkst = nks;
        uint32_t LVt = LV, VAt = VA;
        int colt = col, kqt = kq;
        asm volatile("" : "+v"(LVt), "+v"(VAt), "+v"(colt), "+v"(kqt));
        asm volatile("" : "+s"(rkt), "+s"(bkt), "+s"(rvt), "+s"(bvt), "+s"(nvt), "+s"(g16t), "+s"(rhot), "+s"(nkst));
        const uint8_t* ktile = KS;
        {
            // turns of the tile's first position for frequency j = lane (fp64, then reduced)
            const double t0 = (double)tok0 * om_lane;
            rho0[lane] = (float)(t0 - floor(t0));
        }
        // rotation of the lane's token in block 0 (position tok0 + col) for each of its pairs, as cos, sin;
        // block tb's follows by tb rotations of 16 positions
        float wc[4][4], ws[4][4];
        wave_lds_sync();  // rho0 written above
#pragma unroll
        for (int rb = 0; rb < 4; ++rb)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                float tr = fmaf((float)col, om[rb][v], rho0[16 * rb + 4 * kq + v]);
                tr -= floorf(tr);
                wc[rb][v] = __cosf(6.283185307179586f * tr);
                ws[rb][v] = __sinf(6.283185307179586f * tr);
            }
        float s[4][4];  // [token block][head v], log2 domain
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int v = 0; v < 4; ++v) s[a][v] = -INFINITY;
        // The tile's four blocks of 16 tokens in groups of NB (tb = NB tp + h): the blocks' chains are
        // independent and share each P_K^T operand read.
#pragma unroll 1
        for (int tp = 0; tp < 4 / NB; ++tp) {
#pragma unroll
            for (int h = 0; h < NB; ++h) {
                // stage the centred codes of tokens 16 tb .. 16 tb + 15: lane (token col, part kq) takes
                // coordinates 32 kq .. 32 kq + 31 (zero past the rank, within the 32-wide k-steps)
                const int t = 16 * (NB * tp + h) + colt;
                KVC_SWITCH_B(bkt, (rope_stage_codes<B_>(ktile, rkt, g16t, rhot, kqt, t, ZT + (16 * h + colt) * kZPitch)));
            }
            wave_lds_sync();
            // K^T blocks: rows 16 rb + 4 kq + v, column token col
            rp_f4 Cr[NB][8];
#pragma unroll
            for (int h = 0; h < NB; ++h)
#pragma unroll
                for (int rb = 0; rb < 8; ++rb) Cr[h][rb] = rp_f4{0.f, 0.f, 0.f, 0.f};
            for (int ks = 0; ks < nkst; ++ks) {
                rp_h8 bz[NB];
#pragma unroll
                for (int h = 0; h < NB; ++h)
                    bz[h] = *reinterpret_cast<const rp_h8*>(ZT + (16 * h + col) * kZPitch + 32 * ks + 8 * kq);
#pragma unroll
                for (int rb = 0; rb < 8; ++rb) {
                    const rp_h8 ap = *reinterpret_cast<const rp_h8*>(PT + (16 * rb + col) * kPtPitch + 32 * ks + 8 * kq);
#pragma unroll
                    for (int h = 0; h < NB; ++h) Cr[h][rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ap, bz[h], Cr[h][rb], 0, 0, 0);
                }
            }
            wave_lds_sync();  // ZT is rewritten by the next group of blocks
#pragma unroll
            for (int h = 0; h < NB; ++h) {
                const int tb = NB * tp + h;
                // rotate each pair (j, j + 64) of token 16 tb + col at its position, then advance the
                // rotation by 16 positions for the next block
#pragma unroll
                for (int rb = 0; rb < 4; ++rb)
#pragma unroll
                    for (int v = 0; v < 4; ++v) {
                        const float cs = wc[rb][v], sn = ws[rb][v];
                        const float a = Cr[h][rb][v], b = Cr[h][rb + 4][v];
                        Cr[h][rb][v] = fmaf(a, cs, -b * sn);
                        Cr[h][rb + 4][v] = fmaf(a, sn, b * cs);
                        const float2 e = E16[16 * rb + 4 * kq + v];
                        wc[rb][v] = fmaf(cs, e.x, -sn * e.y);
                        ws[rb][v] = fmaf(cs, e.y, sn * e.x);
                    }
                // logits: sum over features of q' times (hi + lo) of the rotated key
                rp_f4 S = rp_f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    rp_h8 bh, bl;
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        const float x = Cr[h][2 * ks + (e >> 2)][e & 3];
                        const _Float16 hx = (_Float16)x;
                        bh[e] = hx;
                        bl[e] = (_Float16)(x - (float)hx);
                    }
                    S = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa[ks], bh, S, 0, 0, 0);
                    S = __builtin_amdgcn_mfma_f32_16x16x32_f16(qa[ks], bl, S, 0, 0, 0);
                }
                const bool valid_tok = tok0 + 16 * tb + col < end;
#pragma unroll
                for (int a = 0; a < 4; ++a)  // s[tb] without a run-time register index
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        if (a == tb) s[a][v] = (valid_tok && 4 * kq + v < G) ? S[v] * scale : -INFINITY;
            }
        }

        // ---- online softmax of the tile: heads 4 kq + v live in the 16 lanes of group kq
        float mx[4];
        bool raise = false;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            mx[v] = row_max(fmaxf(fmaxf(s[0][v], s[1][v]), fmaxf(s[2][v], s[3][v])));
            raise = raise || (mx[v] > -INFINITY && (mrun[v] == -INFINITY || mx[v] - mrun[v] > kLazy));
        }
        if (__any(raise)) {
            float alpha[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                alpha[v] = 1.f;
                if (mx[v] > -INFINITY && (mrun[v] == -INFINITY || mx[v] - mrun[v] > kLazy)) {
                    alpha[v] = mrun[v] == -INFINITY ? 0.f : exp2f(mrun[v] - mx[v]);
                    mrun[v] = mx[v];
                }
            }
            // accumulators of head 4 pm + grp: its factor lives in lane 16 pm, element grp
#pragma unroll
            for (int pm = 0; pm < LM; ++pm) {
                float al = 1.f;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float t = __shfl(alpha[v], 16 * pm);
                    if (grp == v) al = t;
                }
                if (al != 1.f) {
                    const double a = (double)al;
#pragma unroll
                    for (int nt = 0; nt < 9; ++nt) {
                        const double vv = ((double)C[pm][nt][0] + 256.0 * (double)C[pm][nt][1]) +
                                          (65536.0 * (double)C[pm][nt][2] + 16777216.0 * (double)C[pm][nt][3]);
                        const double vs = rint(vv * a);
                        const double c3 = floor(vs * (1.0 / 16777216.0));
                        const double r3 = vs - 16777216.0 * c3;
                        const double c2 = floor(r3 * (1.0 / 65536.0));
                        const double r2 = r3 - 65536.0 * c2;
                        const double c1 = floor(r2 * (1.0 / 256.0));
                        C[pm][nt][3] = (int)c3;
                        C[pm][nt][2] = (int)c2;
                        C[pm][nt][1] = (int)c1;
                        C[pm][nt][0] = (int)(r2 - 256.0 * c1);
                    }
                }
            }
        }
        // ---- probability limbs of heads 4 kq + v, token 16 tb + col: row 16 kq + 4 v + limb, byte = token
        if (kq < LM) {
#pragma unroll
            for (int tb = 0; tb < 4; ++tb)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const float pr = s[tb][v] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(s[tb][v] - mrun[v]);
                    const uint32_t P = (uint32_t)fmaf(pr, kPScale, kPBias);
                    uint8_t* row = pmat + (16 * kq + 4 * v) * kPRowBytes + 16 * tb + col;
                    row[0] = (uint8_t)((P & 255u) ^ 0x80u);
                    row[kPRowBytes] = (uint8_t)(((P >> 8) & 255u) ^ 0x80u);
                    row[2 * kPRowBytes] = (uint8_t)(((P >> 16) & 255u) ^ 0x80u);
                    row[3 * kPRowBytes] = (uint8_t)(P >> 24);
                }
        }
        wave_lds_sync();
        v4i ap[LM];
#pragma unroll
        for (int pm = 0; pm < LM; ++pm)
            ap[pm] = *reinterpret_cast<const v4i*>(pmat + (16 * pm + col) * kPRowBytes + 16 * grp);
        {
            const auto vrs = v_rs(tile), vrs_n = v_rs(tile + 1);
            KVC_SWITCH_B(bvt, (v_tile<B_, LM, 8>(vb, vrs, vrs_n, rvt, LVt, VAt, ap, C)));
        }
#pragma unroll
        for (int pm = 0; pm < LM; ++pm) C[pm][8] = mfma_i8(ap[pm], ones, C[pm][8]);
        wave_lds_sync();  // pmat and rho0 are rewritten by the next tile
    }

    // partials: m of head 4 pm + grp (lane 16 pm, element grp), l and the centred accumulator
#pragma unroll
    for (int pm = 0; pm < LM; ++pm) {
        const int h = 4 * pm + grp;
        float mh = -INFINITY;
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float t = __shfl(mrun[v], 16 * pm);
            if (grp == v) mh = t;
        }
        const int o0 = __shfl(C[pm][8][0], lane & 48), o1 = __shfl(C[pm][8][1], lane & 48),
                  o2 = __shfl(C[pm][8][2], lane & 48), o3 = __shfl(C[pm][8][3], lane & 48);
        if (G % 4 == 0 || h < G) {
            float* o = out + h * kPartStride;
            if (col == 0) {
                o[0] = mh;
                o[1] = ((float)o0 + 256.f * (float)o1) + (65536.f * (float)o2 + 16777216.f * (float)o3);
            }
#pragma unroll
            for (int nt = 0; nt < 8; ++nt) {
                const int cc = 16 * nt + col;
                if (nt < nv) {
                    const int a0 = C[pm][nt][0] - hv * o0, a1 = C[pm][nt][1] - hv * o1, a2 = C[pm][nt][2] - hv * o2,
                              a3 = C[pm][nt][3] - hv * o3;
                    o[4 + cc] = cc < rv ? ((float)a0 + 256.f * (float)a1) + (65536.f * (float)a2 + 16777216.f * (float)a3)
                                        : 0.f;
                }
            }
        }
    }
}

// ---------------------------------------------------------------- combine

// One block of WC wavefronts per unit (one for a few chunks, more when the context is split into
// many). Lane l handles rank coordinates l and l + 64 of the merge and output columns 2 l, 2 l + 1.
// The chunks' partials merge in the log2 domain (M = max m_c, L = sum l_c 2^(m_c - M),
// A_j = sum acc_c,j 2^(m_c - M)): wavefront w merges chunks w, w + WC, ... (a batch of chunks in
// flight at once, the running sums rescaled when a batch raises M), the wavefronts' merges meet in
// LDS, and z_j = step_V (A_j / L + 1/2) is the dequantised rank-space average. Then o = P_V^T z (the
// V reconstruction of Lemma lem:head-dist applied after the softmax average, which is linear), with
// the heads shared among the wavefronts (G / WC each, at least one), each loading its two columns
// of every basis row at the start.
constexpr int kCombMaxRed = 32;  // WC x G at most (LDS of the cross-wavefront merge)
template <int G, int WC>
__global__ __launch_bounds__(64 * WC) __attribute__((amdgpu_waves_per_eu(2, 2)))
void combine_kernel(DevSide V, int n_chunks, const float* __restrict__ part, float* __restrict__ out) {
    static_assert(WC * G <= kCombMaxRed || WC == 1, "combine_kernel: cross-wavefront merge exceeds its LDS");
    constexpr int Wc = WC;
    constexpr int GH = G / WC > 0 ? G / WC : 1;          // heads whose output one wavefront computes
    constexpr int kCombBatch = 16 / G > 0 ? 16 / G : 1;  // chunks whose partials are in flight together (per wavefront)
    __shared__ float zs[G][kD];
    extern __shared__ float comb_dsm[];  // [WC * G][kPartStride] per (wavefront, head): M, L, -, -, A[128]
    const int u = blockIdx.x, lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int gb = wv * GH;  // first head of this wavefront's output (none when gb >= G)
    float(*red)[kPartStride] = reinterpret_cast<float(*)[kPartStride]>(comb_dsm);
    const int rv = V.r[u];
    const float step = V.delta[u];
    // the lane's two columns of every basis row, in flight while the chunks merge
    const uint32_t* __restrict__ P32 = reinterpret_cast<const uint32_t*>(V.basis + V.basis_off[u]);
    uint32_t pw[kD];
#pragma unroll
    for (int i = 0; i < kD; ++i) pw[i] = (gb < G && i < rv) ? P32[i * (kD / 2) + lane] : 0u;
    const float* __restrict__ pu = part + (int64_t)u * n_chunks * G * kPartStride;
    float M[G], L[G], A0[G], A1[G];
#pragma unroll
    for (int g = 0; g < G; ++g) { M[g] = -INFINITY; L[g] = A0[g] = A1[g] = 0.f; }
    for (int c0 = wv; c0 < n_chunks; c0 += kCombBatch * Wc) {
        float mc[kCombBatch][G], lc[kCombBatch][G], a0[kCombBatch][G], a1[kCombBatch][G];
#pragma unroll
        for (int k = 0; k < kCombBatch; ++k) {
            const int ck = c0 + k * Wc;
            const int c = min(ck, n_chunks - 1);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const float* pc = pu + ((int64_t)c * G + g) * kPartStride;
                mc[k][g] = pc[0];
                lc[k][g] = ck < n_chunks ? pc[1] : 0.f;
                a0[k][g] = pc[4 + lane];
                a1[k][g] = pc[4 + 64 + lane];
            }
        }
#pragma unroll
        for (int g = 0; g < G; ++g) {
            float mb = M[g];
#pragma unroll
            for (int k = 0; k < kCombBatch; ++k)
                if (lc[k][g] > 0.f) mb = fmaxf(mb, mc[k][g]);
            if (mb > M[g]) {  // M[g] = -inf before the first non-empty chunk: the sums are still zero
                const float sc = M[g] == -INFINITY ? 0.f : exp2f(M[g] - mb);
                L[g] *= sc; A0[g] *= sc; A1[g] *= sc;
                M[g] = mb;
            }
#pragma unroll
            for (int k = 0; k < kCombBatch; ++k) {
                if (lc[k][g] > 0.f) {  // an empty chunk (or a batch slot past the last) has l = 0 and no accumulator
                    const float w = exp2f(mc[k][g] - M[g]);
                    L[g] = fmaf(lc[k][g], w, L[g]);
                    A0[g] = fmaf(a0[k][g], w, A0[g]);
                    A1[g] = fmaf(a1[k][g], w, A1[g]);
                }
            }
        }
    }
#pragma unroll
    for (int g = 0; g < G; ++g) {
        float* rd = red[wv * G + g];
        if (lane == 0) { rd[0] = M[g]; rd[1] = L[g]; }
        rd[4 + lane] = A0[g];
        rd[4 + 64 + lane] = A1[g];
    }
    __syncthreads();
    for (int g = wv; g < G; g += Wc) {  // the wavefronts' merges of head g, then z
        float Mg = -INFINITY;
        for (int w = 0; w < Wc; ++w)
            if (red[w * G + g][1] > 0.f) Mg = fmaxf(Mg, red[w * G + g][0]);
        float Lg = 0.f, B0 = 0.f, B1 = 0.f;
        for (int w = 0; w < Wc; ++w) {
            const float* rd = red[w * G + g];
            if (rd[1] > 0.f) {
                const float sc = exp2f(rd[0] - Mg);
                Lg = fmaf(rd[1], sc, Lg);
                B0 = fmaf(rd[4 + lane], sc, B0);
                B1 = fmaf(rd[4 + 64 + lane], sc, B1);
            }
        }
        const float inv = Lg > 0.f ? 1.f / Lg : 0.f;
        zs[g][lane] = (Lg > 0.f && lane < rv) ? step * fmaf(B0, inv, 0.5f) : 0.f;
        zs[g][lane + 64] = (Lg > 0.f && lane + 64 < rv) ? step * fmaf(B1, inv, 0.5f) : 0.f;
    }
    __syncthreads();
    if (gb < G) {
        float o0[GH], o1[GH];
#pragma unroll
        for (int j = 0; j < GH; ++j) o0[j] = o1[j] = 0.f;
#pragma unroll
        for (int i = 0; i < kD; ++i) {
            const float p0 = h2f((uint16_t)(pw[i] & 0xffffu)), p1 = h2f((uint16_t)(pw[i] >> 16));
#pragma unroll
            for (int j = 0; j < GH; ++j) {
                const float z = zs[gb + j][i];  // zero past the rank
                o0[j] = fmaf(p0, z, o0[j]);
                o1[j] = fmaf(p1, z, o1[j]);
            }
        }
#pragma unroll
        for (int j = 0; j < GH; ++j)
            reinterpret_cast<float2*>(out + ((int64_t)u * G + gb + j) * kD)[lane] = float2{o0[j], o1[j]};
    }
}

// Wavefronts of a combine block (1, 2, 4 or 8): enough that each merges about 8 chunks, within the
// LDS of the cross-wavefront merge, and few enough that every block is resident at once (the
// kernel's register budget leaves two wavefronts per SIMD, eight per CU).
inline int combine_waves(int G, int n_chunks, int U, int ncu) {
    const int cap = std::min(std::min(std::max(kCombMaxRed / G, 1), 8), std::max(1, 8 * ncu / std::max(U, 1)));
    int w = 1;
    while (2 * w <= cap && 8 * w < n_chunks) w *= 2;
    return w;
}

// ---------------------------------------------------------------- host side

// Combine launch with cw (a power of two that combine_waves chose for this G) wavefronts per block.
template <int G>
void launch_combine(int cw, dim3 grid, dim3 blk, size_t smem, hipStream_t st, const DevSide& V, int n_chunks,
                    const float* part, float* out) {
    switch (cw) {
        case 8:
            if constexpr (8 * G <= kCombMaxRed) {
                hipLaunchKernelGGL((combine_kernel<G, 8>), grid, blk, smem, st, V, n_chunks, part, out);
                return;
            }
            break;
        case 4:
            if constexpr (4 * G <= kCombMaxRed) {
                hipLaunchKernelGGL((combine_kernel<G, 4>), grid, blk, smem, st, V, n_chunks, part, out);
                return;
            }
            break;
        case 2:
            if constexpr (2 * G <= kCombMaxRed) {
                hipLaunchKernelGGL((combine_kernel<G, 2>), grid, blk, smem, st, V, n_chunks, part, out);
                return;
            }
            break;
        default:
            break;
    }
    hipLaunchKernelGGL((combine_kernel<G, 1>), grid, dim3(64), (size_t)G * kPartStride * 4, st, V, n_chunks, part, out);
}

#ifndef KVC_DECODE_PARTIALS_UNIT
// ---------------------------------------------------------------- read probe

// Streaming read of n16 16-byte words (non-temporal loads, grid-stride). The words fold into one
// value per lane, stored to sink only when it equals a constant, so that the loads stay live.
__global__ __launch_bounds__(256) void read_probe_kernel(const v4u* __restrict__ p, size_t n16, uint32_t* __restrict__ sink) {
    uint32_t acc = 0u;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (size_t)gridDim.x * 256) {
        const v4u v = __builtin_nontemporal_load(p + i);
        acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    if (acc == 0x9e3779b9u) sink[0] = acc;
}

namespace {


// LDS bytes of the staged tail K-step: the largest over units whose rank has a tail group.
int stage_lds_bytes(const kvc_stream_desc* k) {
    int m = 0;
    for (int u = 0; u < k->n_units; ++u)
        if (k->r_host[u] & 15) m = std::max(m, 512 * k->b_host[u]);
    return m == 0 ? 0 : m + 32;  // funnel reads may look one word past a plane's region
}

size_t partial_smem(int G, int stage_bytes_) {
    const int LM = (G + 3) / 4;
    return (size_t)16 * LM * kPRowBytes + (size_t)stage_bytes_;
}

template <int G>
int resident_blocks(size_t smem) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, decode_partial_kernel<G>, 64, smem) != hipSuccess || nb <= 0) {
        (void)hipGetLastError();
        nb = 16;
    }
    return nb;
}

// Compute units of the current device (256, the MI355X figure, without a device).
int device_cus() {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        ncu <= 0) {
        (void)hipGetLastError();
        ncu = 256;
    }
    return ncu;
}

// Work items (wavefronts) the device holds at once for this launch.
int64_t resident_slots(int G, size_t smem) {
    const int ncu = device_cus();
    int nb;
    switch (G) {
        case 1: nb = resident_blocks<1>(smem); break;
        case 2: nb = resident_blocks<2>(smem); break;
        case 4: nb = resident_blocks<4>(smem); break;
        case 8: nb = resident_blocks<8>(smem); break;
        default: nb = resident_blocks<16>(smem); break;
    }
    return (int64_t)ncu * nb;
}

// Split of each unit's context into n_chunks equal chunks of whole tiles (at most kMaxChunkTiles
// each). The count minimises
//   rounds x (tiles per item + per-item overhead) + (straggler share) x tiles per item,
// rounds = ceil(items / resident slots): whole rounds with no short remainder, and no more items
// than that (one round of longer items can beat two rounds of items half as long that would fill
// every slot). The two constants are fitted to the partials kernel's times on the 8B-shaped 32k
// workload at 3, 6 and 9 chunks per unit (2, 4 and 6 rounds): about four tiles of work per item,
// and a small straggler share, as the hardware hands each freed slot the next item.
constexpr int kItemOverheadTiles = 4;
constexpr double kStragglerShare = 0.1;

struct WsLayout {
    int chunk, n_chunks, stage_bytes;
    int64_t qa, qk, part, total;  // byte offsets
};

WsLayout ws_layout(const kvc_stream_desc* k, int G, int max_seq) {
    WsLayout L;
    const int U = k->n_units;
    const int LM = (G + 3) / 4;
    L.stage_bytes = stage_lds_bytes(k);
    const int64_t slots = resident_slots(G, partial_smem(G, L.stage_bytes));
    const int tpu = (max_seq + kTile - 1) / kTile;
    double best_cost = -1.0;
    L.chunk = std::min(tpu, kMaxChunkTiles) * kTile;
    L.n_chunks = (tpu + kMaxChunkTiles - 1) / kMaxChunkTiles;
    for (int n = 1; n <= tpu && n <= 4096; ++n) {
        const int c = (tpu + n - 1) / n;
        if ((tpu + c - 1) / c != n || c > kMaxChunkTiles) continue;
        const int64_t items = (int64_t)U * n;
        const int64_t rounds = (items + slots - 1) / slots;
        const double cost = (double)rounds * (c + kItemOverheadTiles) + kStragglerShare * c;
        if (best_cost < 0.0 || cost < best_cost) {
            best_cost = cost;
            L.chunk = c * kTile;
            L.n_chunks = n;
        }
    }
    auto up = [](int64_t x) { return (x + 255) / 256 * 256; };
    L.qa = 0;
    L.qk = up(L.qa + (int64_t)U * 2 * LM * 64 * 16);
    L.part = up(L.qk + (int64_t)U * G * 16);
    L.total = L.part + (int64_t)U * L.n_chunks * G * kPartStride * 4;
    return L;
}

int decode_check(const kvc_stream_desc* k, const kvc_stream_desc* v, int32_t G, int32_t max_seq_len) {
    if (int e = validate_desc(k, "kvc_decode_attn(k)")) return e;
    if (int e = validate_desc(v, "kvc_decode_attn(v)")) return e;
    if (k->side != KVC_SIDE_K || v->side != KVC_SIDE_V) return set_error(KVC_EINVAL, "kvc_decode_attn: descriptor sides");
    if (k->n_units != v->n_units) return set_error(KVC_EINVAL, "kvc_decode_attn: K and V unit counts differ");
    if (G != 1 && G != 2 && G != 4 && G != 8 && G != 16)
        return set_error(KVC_EUNSUPPORTED, "kvc_decode_attn: G = %d (1, 2, 4, 8 or 16)", G);
    if (max_seq_len < 1) return set_error(KVC_EINVAL, "kvc_decode_attn: max_seq_len < 1");
    if (max_seq_len > k->capacity || max_seq_len > v->capacity)
        return set_error(KVC_ENOSPACE, "kvc_decode_attn: max_seq_len exceeds capacity");
    // per-unit streams must lie inside their arenas (the kernels bound their loads by the stream)
    const int64_t kct = ((int64_t)k->capacity + kTile - 1) / kTile, vct = ((int64_t)v->capacity + kTile - 1) / kTile;
    for (int u = 0; u < k->n_units; ++u) {
        if (kct * 8 * k->r_host[u] * k->b_host[u] > INT32_MAX || vct * 8 * v->r_host[u] * v->b_host[u] > INT32_MAX)
            return set_error(KVC_EUNSUPPORTED, "kvc_decode_attn: a unit's stream exceeds 2 GiB");
    }
    return KVC_OK;
}

template <int G>
int launch_partials(dim3 grid, hipStream_t st, const DevSide& K, const DevSide& V, const v4i* qa, const float4* qk,
                    const int32_t* seq_len, int max_seq, int chunk, int n_chunks, int kct, int vct, float* part,
                    int stage_bytes_) {
    const size_t smem = partial_smem(G, stage_bytes_);
    if (smem > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute((const void*)decode_partial_kernel<G>,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return set_error(KVC_EDEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    hipLaunchKernelGGL(decode_partial_kernel<G>, grid, dim3(64), smem, st, K, V, qa, qk, seq_len, max_seq, chunk,
                       n_chunks, kct, vct, part);
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

using namespace kvc;

extern "C" size_t kvc_decode_attn_workspace(const kvc_stream_desc* k, const kvc_stream_desc* v, int32_t G,
                                            int32_t max_seq_len) {
    clear_error();
    if (decode_check(k, v, G, max_seq_len)) return 0;
    return (size_t)ws_layout(k, G, max_seq_len).total;
}

namespace kvc {
namespace {

// The new token of a fused decode step (none for a plain decode call).
struct StepAppend {
    const uint16_t* xk = nullptr;
    int64_t xk_stride = 0;
    const uint16_t* xv = nullptr;
    int64_t xv_stride = 0;
    int t_new = -1;
};

// Launches of one decode step into the workspace ws (validated by the caller, of layout L); with an
// append, the query projection and the append share the first launch.
int decode_launch(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q, int32_t G,
                  const int32_t* seq_len, int32_t max_seq_len, float* out, void* ws, const WsLayout& L, void* stream,
                  const StepAppend& app = StepAppend()) {
    const int U = k->n_units;
    char* w = reinterpret_cast<char*>(ws);
    v4i* qa = reinterpret_cast<v4i*>(w + L.qa);
    float4* qk = reinterpret_cast<float4*>(w + L.qk);
    float* part = reinterpret_cast<float*>(w + L.part);
    hipStream_t st = (hipStream_t)stream;
    const DevSide K = dev_side(k), V = dev_side(v);
    const int LM = (G + 3) / 4;
    const size_t qsm = (size_t)2 * LM * 64 * 16;
    if (app.t_new >= 0)
        hipLaunchKernelGGL(step_prep_kernel, dim3(U, 3), dim3(kStepPrepThreads), qsm, st, K, V, q, G, LM, qa, qk, app.xk,
                           app.xk_stride, app.xv, app.xv_stride, app.t_new);
    // one wavefront per unit while the units fill the device, eight (one per row block) for a few units
    else if ((int64_t)U * 4 >= (int64_t)device_cus() * 8)
        hipLaunchKernelGGL(qprep_kernel<1>, dim3(U), dim3(64), qsm, st, K, q, G, LM, qa, qk);
    else
        hipLaunchKernelGGL(qprep_kernel<8>, dim3(U), dim3(512), qsm, st, K, q, G, LM, qa, qk);
    const int kct = (k->capacity + kTile - 1) / kTile, vct = (v->capacity + kTile - 1) / kTile;
    const dim3 grid(L.n_chunks, U);
    int e = KVC_OK;
    switch (G) {
        case 1: e = launch_partials<1>(grid, st, K, V, qa, qk, seq_len, max_seq_len, L.chunk, L.n_chunks, kct, vct, part, L.stage_bytes); break;
        case 2: e = launch_partials<2>(grid, st, K, V, qa, qk, seq_len, max_seq_len, L.chunk, L.n_chunks, kct, vct, part, L.stage_bytes); break;
        case 4: e = launch_partials<4>(grid, st, K, V, qa, qk, seq_len, max_seq_len, L.chunk, L.n_chunks, kct, vct, part, L.stage_bytes); break;
        case 8: e = launch_partials<8>(grid, st, K, V, qa, qk, seq_len, max_seq_len, L.chunk, L.n_chunks, kct, vct, part, L.stage_bytes); break;
        default: e = launch_partials<16>(grid, st, K, V, qa, qk, seq_len, max_seq_len, L.chunk, L.n_chunks, kct, vct, part, L.stage_bytes); break;
    }
    if (e) return e;
    const int cw = combine_waves(G, L.n_chunks, U, device_cus());
    const dim3 cblk(64 * cw);
    const size_t csm = (size_t)cw * G * kPartStride * 4;
    switch (G) {
        case 1: launch_combine<1>(cw, dim3(U), cblk, csm, st, V, L.n_chunks, part, out); break;
        case 2: launch_combine<2>(cw, dim3(U), cblk, csm, st, V, L.n_chunks, part, out); break;
        case 4: launch_combine<4>(cw, dim3(U), cblk, csm, st, V, L.n_chunks, part, out); break;
        case 8: launch_combine<8>(cw, dim3(U), cblk, csm, st, V, L.n_chunks, part, out); break;
        default: launch_combine<16>(cw, dim3(U), cblk, csm, st, V, L.n_chunks, part, out); break;
    }
    return check_launch("kvc_decode_attn");
}

// Checks shared by both decode entry points (pointers and alignment; the descriptors are checked by
// decode_check).
int decode_args(const char* fn, const uint16_t* q, const int32_t* seq_len, const float* out) {
    if (!q || !seq_len || !out) return set_error(KVC_EINVAL, "%s: null pointer", fn);
    if (reinterpret_cast<uintptr_t>(q) & 15) return set_error(KVC_EINVAL, "%s: q not 16-byte aligned", fn);
    return KVC_OK;
}

// The no-allocation variant's workspace: one file-scope array per device (each GPU holds its own copy
// at its own address, from the library's load until the process ends). Host code never passes the
// array's name to a kernel: its device address comes from hipGetSymbolAddress, taken once per device
// with that device current.
__device__ __align__(256) uint8_t scratch[KVC_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_of_current_device(void** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return set_error(KVC_EDEVICE, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return set_error(KVC_EUNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return set_error(KVC_EDEVICE, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

extern "C" int kvc_decode_attn(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q, int32_t G,
                               const int32_t* seq_len, int32_t max_seq_len, float* out, void* ws, size_t ws_bytes,
                               void* stream) {
    clear_error();
    if (int e = decode_check(k, v, G, max_seq_len)) return e;
    if (k->n_units == 0) return KVC_OK;
    if (int e = decode_args("kvc_decode_attn", q, seq_len, out)) return e;
    if (!ws) return set_error(KVC_EINVAL, "kvc_decode_attn: null workspace");
    if (reinterpret_cast<uintptr_t>(ws) & 255) return set_error(KVC_EINVAL, "kvc_decode_attn: workspace not 256-byte aligned");
    const WsLayout L = ws_layout(k, G, max_seq_len);
    if ((int64_t)ws_bytes < L.total)
        return set_error(KVC_ENOSPACE, "kvc_decode_attn: workspace %zu < %lld bytes", ws_bytes, (long long)L.total);
    return decode_launch(k, v, q, G, seq_len, max_seq_len, out, ws, L, stream);
}

extern "C" int kvc_decode_step(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* xk,
                               int64_t xk_unit_stride, const uint16_t* xv, int64_t xv_unit_stride, int32_t t_new,
                               const uint16_t* q, int32_t G, const int32_t* seq_len, int32_t max_seq_len, float* out,
                               void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (int e = decode_check(k, v, G, max_seq_len)) return e;
    if (t_new < 0) return set_error(KVC_EINVAL, "kvc_decode_step: negative t_new");
    if ((int64_t)t_new + 1 > k->capacity || (int64_t)t_new + 1 > v->capacity)
        return set_error(KVC_ENOSPACE, "kvc_decode_step: t_new + 1 > capacity");
    if (k->n_units == 0) return KVC_OK;
    for (const auto& xs : {std::make_pair(xk, xk_unit_stride), std::make_pair(xv, xv_unit_stride)})
        if (!xs.first || (reinterpret_cast<uintptr_t>(xs.first) & 15) || (xs.second & 7) || xs.second < (int64_t)kD)
            return set_error(KVC_EINVAL, "kvc_decode_step: xk, xv must be 16-byte aligned with stride a multiple of 8 and >= d");
    if (int e = decode_args("kvc_decode_step", q, seq_len, out)) return e;
    if (!ws) return set_error(KVC_EINVAL, "kvc_decode_step: null workspace");
    if (reinterpret_cast<uintptr_t>(ws) & 255) return set_error(KVC_EINVAL, "kvc_decode_step: workspace not 256-byte aligned");
    const WsLayout L = ws_layout(k, G, max_seq_len);
    if ((int64_t)ws_bytes < L.total)
        return set_error(KVC_ENOSPACE, "kvc_decode_step: workspace %zu < %lld bytes", ws_bytes, (long long)L.total);
    StepAppend app;
    app.xk = xk;
    app.xk_stride = xk_unit_stride;
    app.xv = xv;
    app.xv_stride = xv_unit_stride;
    app.t_new = t_new;
    return decode_launch(k, v, q, G, seq_len, max_seq_len, out, ws, L, stream, app);
}

namespace kvc {
namespace {

template <int G>
int launch_rope(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q, const int32_t* seq_len,
                int32_t max_seq_len, float log2_base, float* out, const WsLayout& L, float* part, hipStream_t st) {
    const size_t smem = (size_t)kRopeShared + (size_t)kRopeWaves * rope_wave_lds(G);
    if (smem > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute((const void*)decode_rope_kernel<G>,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return set_error(KVC_EDEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    const int U = k->n_units;
    const int vct = (v->capacity + kTile - 1) / kTile;
    const DevSide K = dev_side(k), V = dev_side(v);
    hipLaunchKernelGGL(decode_rope_kernel<G>, dim3((L.n_chunks + kRopeWaves - 1) / kRopeWaves, U),
                       dim3(64 * kRopeWaves), smem, st, K, V, q, seq_len, max_seq_len, L.chunk, L.n_chunks, vct,
                       log2_base, part);
    const int cw = combine_waves(G, L.n_chunks, U, device_cus());
    launch_combine<G>(cw, dim3(U), dim3(64 * cw), (size_t)cw * G * kPartStride * 4, st, V, L.n_chunks, part, out);
    return check_launch("kvc_decode_attn_rope");
}

}  // namespace
}  // namespace kvc

extern "C" int kvc_decode_attn_rope(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q, int32_t G,
                                    const int32_t* seq_len, int32_t max_seq_len, float rope_base, float* out,
                                    void* ws, size_t ws_bytes, void* stream) {
    clear_error();
    if (int e = decode_check(k, v, G, max_seq_len)) return e;
    if (!(rope_base > 1.f) || !std::isfinite(rope_base))
        return set_error(KVC_EINVAL, "kvc_decode_attn_rope: rope_base must be finite and > 1");
    if (k->n_units == 0) return KVC_OK;
    if (int e = decode_args("kvc_decode_attn_rope", q, seq_len, out)) return e;
    if (!ws) return set_error(KVC_EINVAL, "kvc_decode_attn_rope: null workspace");
    if (reinterpret_cast<uintptr_t>(ws) & 255) return set_error(KVC_EINVAL, "kvc_decode_attn_rope: workspace not 256-byte aligned");
    const WsLayout L = ws_layout(k, G, max_seq_len);
    if ((int64_t)ws_bytes < L.total)
        return set_error(KVC_ENOSPACE, "kvc_decode_attn_rope: workspace %zu < %lld bytes", ws_bytes, (long long)L.total);
    float* part = reinterpret_cast<float*>(reinterpret_cast<char*>(ws) + L.part);
    const float lb = (float)std::log2((double)rope_base);
    hipStream_t st = (hipStream_t)stream;
    switch (G) {
        case 1: return launch_rope<1>(k, v, q, seq_len, max_seq_len, lb, out, L, part, st);
        case 2: return launch_rope<2>(k, v, q, seq_len, max_seq_len, lb, out, L, part, st);
        case 4: return launch_rope<4>(k, v, q, seq_len, max_seq_len, lb, out, L, part, st);
        case 8: return launch_rope<8>(k, v, q, seq_len, max_seq_len, lb, out, L, part, st);
        default: return launch_rope<16>(k, v, q, seq_len, max_seq_len, lb, out, L, part, st);
    }
}

extern "C" int kvc_decode_attn_noalloc(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q,
                                       int32_t G, const int32_t* seq_len, int32_t max_seq_len, float* out,
                                       void* stream) {
    clear_error();
    if (int e = decode_check(k, v, G, max_seq_len)) return e;
    if (k->n_units == 0) return KVC_OK;
    if (int e = decode_args("kvc_decode_attn_noalloc", q, seq_len, out)) return e;
    const WsLayout L = ws_layout(k, G, max_seq_len);
    if (L.total > (int64_t)KVC_NOALLOC_SCRATCH_BYTES)
        return set_error(KVC_ENOSPACE, "kvc_decode_attn_noalloc: needs %lld bytes of workspace, the scratch holds %lld",
                         (long long)L.total, (long long)KVC_NOALLOC_SCRATCH_BYTES);
    void* ws = nullptr;
    if (int e = scratch_of_current_device(&ws)) return e;
    return decode_launch(k, v, q, G, seq_len, max_seq_len, out, ws, L, stream);
}

extern "C" int kvc_read_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream) {
    clear_error();
    if (!buf || !sink || (reinterpret_cast<uintptr_t>(buf) & 15) || (bytes & 15) || (reinterpret_cast<uintptr_t>(sink) & 3))
        return set_error(KVC_EINVAL, "kvc_read_probe: buf and bytes must be multiples of 16 bytes, sink a 4-byte aligned word");
    if (bytes == 0) return KVC_OK;
    const size_t n16 = bytes / 16;
    const size_t blocks = std::min<size_t>((n16 + 255) / 256, (size_t)64 * device_cus());
    hipLaunchKernelGGL(read_probe_kernel, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream,
                       reinterpret_cast<const v4u*>(buf), n16, sink);
    return check_launch("kvc_read_probe");
}
#else
}  // namespace kvc
#endif  // KVC_DECODE_PARTIALS_UNIT
