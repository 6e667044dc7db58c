// Device half of libkvc, compression side: HIP kernels for CDNA4 (gfx950) and
// their C-ABI launchers (kvc_encode, kvc_reconstruct). Decode attention lives
// in kvc_decode.hip.
//
// Kernels
//  encode_mfma_kernel   bulk encode: per (unit, run of 64-token tiles), the
//                       projection on fp16 matrix cores with fp32 accumulation,
//                       codes decided against a rigorous error bound (undecided
//                       elements settled in fp64, then exactly in 128-bit
//                       integers), bit-packed from LDS group by group.
//  append_kernel        1-4 new tokens per unit (a decode step's append): basis
//                       rows read coalesced, the same bounded decision (undecided
//                       elements settled by their wavefront), and the new fields
//                       written in place (whole words where a token owns them).
//  reconstruct_kernel   x_hat = P^T z for a 64-token block of one unit.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <utility>

#include "kvc_append.h"
#include "kvc_device.h"
#include "kvc_internal.h"

namespace kvc {

constexpr int kD = KVC_HEAD_DIM;
constexpr int kTile = KVC_TILE_TOKENS;

// ---------------------------------------------------------------- encode

// ---------------------------------------------------------------- bulk encode on matrix cores

// Bulk encode (any token count above the append path's): one 256-thread block per (unit, run of
// tiles); each wavefront encodes whole 64-token tiles. The projection y = P x runs on
// v_mfma_f32_16x16x32_f16 (exact fp16 products, fp32 accumulation) with the basis staged in LDS
// and the tile's tokens held as operand fragments in registers. Codes are decided in fp32 against
// the bound |y_mma - y| <= 2^-16 ||P_i|| ||x|| (twice the bound for 128 terms summed with fp32
// round-to-nearest, so it also holds for truncating additions) plus the rounding of y / step; the rare undecided elements are re-evaluated by the whole
// wavefront in fp64 (exact products, a 2^-45 ||P_i|| ||x|| sum bound) and, if still undecided,
// exactly in 128-bit integers. Each group of 16 coordinates fills 1024 consecutive slots of the
// stream layout (K: coordinate group; V: 16 coordinate rows), which are bit-packed from LDS as
// soon as the group is decided.
constexpr int kEncMmaThreads = 256;
constexpr int kEncMmaTilesPerBlock = 32;
constexpr int kPRow = kD + 8;  // LDS row stride of the staged basis, in halves

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef float f4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ f4 mfma_f16(h8 a, h8 b, f4 c) { return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0); }

// Four slots (one code per byte of v, already masked to P bits) packed into 4 P consecutive bits.
template <int P>
__device__ __forceinline__ uint32_t compact4(uint32_t v) {
    if constexpr (P == 4) {
        v = (v | (v >> 4)) & 0x00ff00ffu;
        return (v | (v >> 8)) & 0xffffu;
    } else if constexpr (P == 2) {
        v = (v | (v >> 6)) & 0x000f000fu;
        return (v | (v >> 12)) & 0xffu;
    } else if constexpr (P == 1) {
        v = (v | (v >> 7)) & 0x00030003u;
        return (v | (v >> 14)) & 0xfu;
    } else {
        return v;
    }
}

// The codes of one slot group (1024 slots) wait in LDS in slot order, except that on the V side each
// 64-slot coordinate row starts kVRow bytes after the previous one: the 16 extra bytes spread the
// rows' dword writes (lane (col, grp) writes row col at 4 grp + 16 nt) over the banks.
constexpr int kVRow = 80;
constexpr int kSlotBufBytes = 16 * kVRow;
template <int side>
__device__ __forceinline__ int sb_off(int slot) {
    return side == KVC_SIDE_K ? slot : (slot >> 6) * kVRow + (slot & 63);
}

// Codes of the PPW slots [PPW w, PPW w + PPW) of the group, four per dword, read with one LDS access
// (two for 1-bit planes).
template <int side, int PPW>
__device__ __forceinline__ void slot_words(const uint8_t* __restrict__ sb, int w, uint32_t (&v)[PPW / 4]) {
    const uint8_t* src = sb + sb_off<side>(w * PPW);
    if constexpr (PPW == 4) {
        v[0] = *reinterpret_cast<const uint32_t*>(src);
    } else if constexpr (PPW == 8) {
        const uint2 a = *reinterpret_cast<const uint2*>(src);
        v[0] = a.x; v[1] = a.y;
    } else if constexpr (PPW == 16) {
        const uint4 a = *reinterpret_cast<const uint4*>(src);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    } else {
        const uint4 a = *reinterpret_cast<const uint4*>(src), c = *reinterpret_cast<const uint4*>(src + 16);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = c.x; v[5] = c.y; v[6] = c.z; v[7] = c.w;
    }
}

// Packs slots [sl0, sl0 + n_sl) of a tile (the group's codes in sb, see sb_off) into every bit plane
// of a B-bit code: slot phi of a plane of width p takes bits [p phi, p phi + p), so word w of the
// plane holds slots [w 32/p, (w + 1) 32/p) in order.
template <int side, int B, int K>
__device__ __forceinline__ void pack_plane(const uint8_t* __restrict__ sb, uint8_t* __restrict__ tbase, int r, int sl0,
                                           int n_sl, int lane) {
    if constexpr (K < n_planes(B)) {
        constexpr int P = plane_w(B, K), SH = plane_sh(B, K), PPW = 32 / P;
        constexpr uint32_t PM = (P == 8 ? 0xffu : ((1u << P) - 1u)) * 0x01010101u;
        uint32_t* __restrict__ pw = reinterpret_cast<uint32_t*>(tbase + 8 * r * plane_off(B, K)) + sl0 / PPW;
        const int nw = n_sl / PPW;
        for (int wi = lane; wi < nw; wi += 64) {
            uint32_t src[PPW / 4];
            slot_words<side, PPW>(sb, wi, src);
            uint32_t word = 0;
#pragma unroll
            for (int m = 0; m < PPW / 4; ++m) word |= compact4<P>((src[m] >> SH) & PM) << (4 * P * m);
            pw[wi] = word;
        }
    }
}

// One plane of the V field of this lane (see v_field_off): its 16 codes, in position order, as four
// dwords of four bytes -> 2p bytes at the field's offset.
template <int B, int K>
__device__ __forceinline__ void pack_vfield_plane(const uint32_t (&src)[4], uint8_t* __restrict__ tbase, int r, int n,
                                                  int c, int q) {
    if constexpr (K < n_planes(B)) {
        constexpr int P = plane_w(B, K), SH = plane_sh(B, K);
        constexpr uint32_t PM = (P == 8 ? 0xffu : ((1u << P) - 1u)) * 0x01010101u;
        uint8_t* __restrict__ dst = tbase + 8 * r * plane_off(B, K) + v_field_off(P, r, n, c, q);
        uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int m = 0; m < 4; ++m) w[(4 * P * m) >> 5] |= compact4<P>((src[m] >> SH) & PM) << ((4 * P * m) & 31);
        if constexpr (P == 1) *reinterpret_cast<uint16_t*>(dst) = (uint16_t)w[0];
        else if constexpr (P == 2) *reinterpret_cast<uint32_t*>(dst) = w[0];
        else if constexpr (P == 4) *reinterpret_cast<uint2*>(dst) = uint2{w[0], w[1]};
        else *reinterpret_cast<uint4*>(dst) = uint4{w[0], w[1], w[2], w[3]};
    }
}

// The wavefront's LDS accesses execute in program order: between a write and a read of the same
// bytes by other lanes only the compiler's reordering has to be stopped.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// Value fields of a plane narrower than 8 bits are gathered per group in LDS (kVGroupBytes per plane
// and wavefront) and the finished group goes out as whole 16-byte rows of the plane, instead of one
// scattered 2p-byte store per field.
constexpr int kVGroupBytes = 1024;
constexpr int kVStageBytes = 3 * kVGroupBytes;

template <int B, int K>
__device__ __forceinline__ void pack_vfield_staged(const uint32_t (&src)[4], bool has, uint8_t* __restrict__ vst,
                                                   uint8_t* __restrict__ tbase, int r, int n, int n_last, int c, int q,
                                                   int lane) {
    if constexpr (K < n_planes(B)) {
        constexpr int P = plane_w(B, K), SH = plane_sh(B, K), G = v_group_ntiles(P);
        if constexpr (P == 8) {
            if (has) pack_vfield_plane<B, K>(src, tbase, r, n, c, q);
        } else {
            constexpr uint32_t PM = ((1u << P) - 1u) * 0x01010101u;
            const int Q = n / G;
            uint8_t* __restrict__ gst = vst + K * kVGroupBytes;
            if (has) {
                uint32_t w[2] = {0u, 0u};
#pragma unroll
                for (int m = 0; m < 4; ++m) w[(4 * P * m) >> 5] |= compact4<P>((src[m] >> SH) & PM) << ((4 * P * m) & 31);
                uint8_t* dst = gst + (v_field_off(P, r, n, c, q) - 1024 * Q);
                if constexpr (P == 1) *reinterpret_cast<uint16_t*>(dst) = (uint16_t)w[0];
                else if constexpr (P == 2) *reinterpret_cast<uint32_t*>(dst) = w[0];
                else *reinterpret_cast<uint2*>(dst) = uint2{w[0], w[1]};
            }
            if (n - G * Q == G - 1 || n == n_last) {  // the group is complete: 8 p bytes per coordinate
                const int gbytes = 8 * P * min(16 * G, r - 16 * G * Q);  // a multiple of 16 (r even)
                wave_lds_sync();
                uint8_t* __restrict__ pbase = tbase + 8 * r * plane_off(B, K) + 1024 * Q;
                if (16 * lane < gbytes)
                    *reinterpret_cast<uint4*>(pbase + 16 * lane) = *reinterpret_cast<const uint4*>(gst + 16 * lane);
                wave_lds_sync();
            }
        }
    }
}

// Packs the V fields of N-tile n (its codes in sb: coordinate row c at kVRow c, quarter q at 16 q,
// in position order) into every plane: lane 4 c + q owns field (n, c, q).
template <int B>
__device__ __forceinline__ void pack_vfields(const uint8_t* __restrict__ sb, uint8_t* __restrict__ vst,
                                             uint8_t* __restrict__ tbase, int r, int n, int n_last, int lane) {
    const int c = lane >> 2, q = lane & 3;
    const bool has = 16 * n + c < r;
    uint32_t src[4] = {0u, 0u, 0u, 0u};
    if (has) {
        const uint4 a = *reinterpret_cast<const uint4*>(sb + kVRow * c + 16 * q);
        src[0] = a.x; src[1] = a.y; src[2] = a.z; src[3] = a.w;
    }
    pack_vfield_staged<B, 0>(src, has, vst, tbase, r, n, n_last, c, q, lane);
    pack_vfield_staged<B, 1>(src, has, vst, tbase, r, n, n_last, c, q, lane);
    pack_vfield_staged<B, 2>(src, has, vst, tbase, r, n, n_last, c, q, lane);
}

template <int side, int B>
__device__ __forceinline__ void pack_group(const uint8_t* __restrict__ sb, uint8_t* __restrict__ tbase, int r, int sl0,
                                           int n_sl, int lane) {
    pack_plane<side, B, 0>(sb, tbase, r, sl0, n_sl, lane);
    pack_plane<side, B, 1>(sb, tbase, r, sl0, n_sl, lane);
    pack_plane<side, B, 2>(sb, tbase, r, sl0, n_sl, lane);
}

template <int side>
__global__ __launch_bounds__(kEncMmaThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void encode_mfma_kernel(DevSide s, const uint16_t* __restrict__ x,
                                                                    int64_t x_stride, int t0, int n_tok, int tile_first,
                                                                    int n_tiles) {
    extern __shared__ uint8_t esm[];
    uint16_t* Pl = reinterpret_cast<uint16_t*>(esm);                   // [128][kPRow] fp16 basis, rows >= r zero
    float* tolc = reinterpret_cast<float*>(Pl + kD * kPRow);           // [128] 2^-16 1.01 ||P_i|| / step (NaN for i >= r)
    float* pnrm = tolc + kD;                                           // [128] ||P_i||
    float* etoks = pnrm + kD;                                          // [4 waves][64] token norms
    uint8_t* slots = reinterpret_cast<uint8_t*>(etoks + 4 * kTile);    // [4 waves][kSlotBufBytes] codes of one slot group
    const int u = blockIdx.y, tid = threadIdx.x;
    const int r = s.r[u], b = s.b[u];
    const float step = s.delta[u];
    const uint16_t* __restrict__ Pg = s.basis + s.basis_off[u];
    for (int q = tid; q < kD * (kD / 8); q += kEncMmaThreads) {
        const int row = q >> 4, c8 = q & 15;
        uint4 v = {0u, 0u, 0u, 0u};
        if (row < r) v = reinterpret_cast<const uint4*>(Pg + (int64_t)row * kD)[c8];
        *reinterpret_cast<uint4*>(Pl + row * kPRow + 8 * c8) = v;
    }
    __syncthreads();
    if (tid < kD) {
        float s2 = 0.f;
        for (int j = 0; j < kD; ++j) {
            const float p = h2f(Pl[tid * kPRow + j]);
            s2 = fmaf(p, p, s2);
        }
        pnrm[tid] = sqrtf(s2);
        tolc[tid] = tid < r ? 0x1p-16f * 1.01f * sqrtf(s2) / step : __builtin_nanf("");
    }
    __syncthreads();

    const int wv = tid >> 6, lane = tid & 63, col = lane & 15, grp = lane >> 4;
    uint8_t* __restrict__ sb = slots + wv * kSlotBufBytes;
    // [4 waves][kVStageBytes] value groups being gathered (value side only)
    uint8_t* __restrict__ vst = slots + (kEncMmaThreads / 64) * kSlotBufBytes + wv * kVStageBytes;
    float* __restrict__ etok = etoks + wv * kTile;
    const int h = 1 << (b - 1);
    const float fh = (float)h, fmax_code = (float)(2 * h - 1), inv = 1.f / step;
    const float fh_lo = fh - 0.5f;                                       // t' = t - 1/2
    const float half_amb = 0.5f - (float)(3 * h + 4) * 0x1p-22f;         // 1/2 - c_amb (exact in fp32)
    const int g16 = r >> 4, rho = r & 15, n_mc = (r + 15) >> 4;
    uint8_t* __restrict__ stream = s.codes + s.code_off[u];
    const uint16_t* __restrict__ xu = x + (int64_t)u * x_stride;

    // Token fragments: operand row 16 nt + col, dims 32 ks + 8 grp + [0, 8). The row holds token
    // 16 nt + col for K; for V, token 16 nt + kidx_b(col), the token whose slot in the quarter is
    // position col (pos_b o kidx_b = identity), so that a lane's four results (rows 4 grp + i) are
    // four consecutive slot bytes. Tokens outside the range read a valid token and never reach the
    // stream. The fragments of a wavefront's next tile are loaded as soon as the last products of the
    // current one have read them, so that the loads overlap the tile's last decisions and packing.
    const int trow = side == KVC_SIDE_K ? col : kidx_b(b, col);
    h8 xf[4][4];
    auto load_x = [&](int tl) {
        const int tok0n = (tile_first + tl) * kTile;
        const int lon = max(t0, tok0n), hin = min(t0 + n_tok, tok0n + kTile);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int tk = tok0n + 16 * nt + trow;
            const h8* row = reinterpret_cast<const h8*>(xu + (int64_t)((tk >= lon && tk < hin ? tk : lon) - t0) * kD);
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) xf[nt][ks] = row[4 * ks + grp];
        }
    };
    if (blockIdx.x * kEncMmaTilesPerBlock + wv < n_tiles) load_x(blockIdx.x * kEncMmaTilesPerBlock + wv);

#pragma unroll 1
    for (int tt = wv; tt < kEncMmaTilesPerBlock; tt += kEncMmaThreads / 64) {
        const int tl_idx = blockIdx.x * kEncMmaTilesPerBlock + tt;
        if (tl_idx >= n_tiles) break;
        const int tile = tile_first + tl_idx, tok0 = tile * kTile;
        const int lo = max(t0, tok0), hi = min(t0 + n_tok, tok0 + kTile);
        const bool full = lo == tok0 && hi == tok0 + kTile;
        uint8_t* __restrict__ tbase = stream + (int64_t)tile * 8 * r * b;
        const int tl_next = tl_idx + kEncMmaThreads / 64;
        const bool has_next = tt + kEncMmaThreads / 64 < kEncMmaTilesPerBlock && tl_next < n_tiles;

        // etok is indexed by operand row.
        float et[4];  // ||x|| of the lane's token (NaN outside the range: such elements are never undecided)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) {
            const int tk = tok0 + 16 * nt + trow;
            const bool ok = tk >= lo && tk < hi;
            float s2 = 0.f;
#pragma unroll
            for (int ks = 0; ks < 4; ++ks) {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const h2 v = {xf[nt][ks][2 * e], xf[nt][ks][2 * e + 1]};
                    s2 = __builtin_amdgcn_fdot2(v, v, s2, false);
                }
            }
            s2 += __shfl_xor(s2, 16);
            s2 += __shfl_xor(s2, 32);
            et[nt] = ok ? sqrtf(s2) : __builtin_nanf("");
            if (grp == 0) etok[16 * nt + col] = et[nt];
        }
        __builtin_amdgcn_wave_barrier();
#pragma unroll 1
        for (int mc = 0; mc < n_mc; ++mc) {
            h8 pf[4];
#pragma unroll
            for (int ks = 0; ks < 4; ++ks)
                pf[ks] = *reinterpret_cast<const h8*>(Pl + (16 * mc + col) * kPRow + 32 * ks + 8 * grp);
            f4 acc[4];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                acc[nt] = f4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    acc[nt] = side == KVC_SIDE_K ? mfma_f16(pf[ks], xf[nt][ks], acc[nt]) : mfma_f16(xf[nt][ks], pf[ks], acc[nt]);
            }
            if (mc == n_mc - 1 && has_next) load_x(tl_next);
            // K: lane holds coordinates 16 mc + 4 grp + i of token 16 nt + col.
            // V: lane holds tokens 16 nt + 4 grp + i of coordinate 16 mc + col.
            // t = y / step + 2^(b-1): its floor, clamped, is the code. With t' = t - 1/2 (one fused
            // multiply-add) the floor is rint(t') wherever t is not within the error bound eps of an
            // integer, i.e. wherever |t' - rint(t')| < 1/2 - eps; the other elements are undecided.
            // eps = (the basis-product bound tb) + c_amb, c_amb covering the rounding of 1 / step and
            // of the multiply-add, (|t| + 2^(b-1) + 1) 2^-22, for every |t| <= 2^b + 1 (beyond, the
            // code is clamped to 0 or 2^b - 1 whatever the error).
            bool any_amb = false;
            uint32_t cw[4];
#pragma unroll
            for (int nt = 0; nt < 4; ++nt) {
                uint32_t w = 0;
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float thr = side == KVC_SIDE_K ? fmaf(-et[nt], tolc[16 * mc + 4 * grp + i], half_amb)
                                                         : fmaf(-etok[16 * nt + 4 * grp + i], tolc[16 * mc + col], half_amb);
                    const float tp = fmaf(acc[nt][i], inv, fh_lo);
                    const float m = __builtin_rintf(tp);
                    any_amb |= fabsf(tp - m) >= thr;
                    w = __builtin_amdgcn_cvt_pk_u8_f32(__builtin_amdgcn_fmed3f(m, 0.f, fmax_code), i, w);
                }
                cw[nt] = w;
            }
            // place the codes in the group's 1024 slots
            const bool tailg = mc == g16;  // K tail group (rho > 0)
            if constexpr (side == KVC_SIDE_K) {
                if (!tailg) {
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt)
                        *reinterpret_cast<uint32_t*>(sb + 16 * (16 * nt + col) + 4 * grp) = cw[nt];
                } else {
#pragma unroll
                    for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            if (4 * grp + i < rho) sb[(16 * nt + col) * rho + 4 * grp + i] = (uint8_t)(cw[nt] >> (8 * i));
                }
            } else if (16 * mc + col < r) {
                // operand rows 16 nt + 4 grp + i of coordinate row col: slot positions 4 grp + i of quarter nt
#pragma unroll
                for (int nt = 0; nt < 4; ++nt) *reinterpret_cast<uint32_t*>(sb + kVRow * col + 16 * nt + 4 * grp) = cw[nt];
            }
            // undecided elements (rare): flag them again per lane, then the whole wavefront settles
            // them one by one
            if (__any(any_amb)) {
                uint32_t ambm = 0;
#pragma unroll
                for (int nt = 0; nt < 4; ++nt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const float thr = side == KVC_SIDE_K ? fmaf(-et[nt], tolc[16 * mc + 4 * grp + i], half_amb)
                                                             : fmaf(-etok[16 * nt + 4 * grp + i], tolc[16 * mc + col], half_amb);
                        const float tp = fmaf(acc[nt][i], inv, fh_lo);
                        if (fabsf(tp - __builtin_rintf(tp)) >= thr) ambm |= 1u << (4 * nt + i);
                    }
                uint64_t pend = __ballot(ambm != 0);
                while (pend) {
                    const int L = __builtin_ctzll(pend);
                    pend &= pend - 1;
                    uint32_t m = (uint32_t)__builtin_amdgcn_readlane((int)ambm, L);
                    const int Lcol = L & 15, Lgrp = L >> 4;
                    while (m) {
                        const int bit = __builtin_ctz(m);
                        m &= m - 1;
                        const int nt = bit >> 2, i = bit & 3;
                        int tkn, c, sl, row;  // token, coordinate, slot, operand row of the element
                        if constexpr (side == KVC_SIDE_K) {
                            tkn = 16 * nt + Lcol;
                            row = tkn;
                            c = 16 * mc + 4 * Lgrp + i;
                            sl = tailg ? tkn * rho + 4 * Lgrp + i : 16 * tkn + 4 * Lgrp + i;
                        } else {
                            row = 16 * nt + 4 * Lgrp + i;
                            tkn = 16 * nt + kidx_b(b, 4 * Lgrp + i);
                            c = 16 * mc + Lcol;
                            sl = 64 * Lcol + row;
                        }
                        const uint16_t* xrow = xu + (int64_t)(tok0 + tkn - t0) * kD;
                        const uint32_t code = resolve_code_wave(Pl + c * kPRow, Pg + (int64_t)c * kD, xrow, step, b,
                                                                pnrm[c], etok[row], lane);
                        if (lane == 0) sb[sb_off<side>(sl)] = (uint8_t)code;
                    }
                }
            }
            __builtin_amdgcn_wave_barrier();
            // pack the group's slots [1024 mc, 1024 mc + n_sl) (K) or fields of N-tile mc (V) into every plane
            const int n_sl = (rho && mc == n_mc - 1) ? 64 * rho : 1024;  // K tail group
            const int sl0 = 1024 * mc;
            if constexpr (side == KVC_SIDE_V) {
                if (full) {
                    KVC_SWITCH_B(b, (pack_vfields<B_>(sb, vst, tbase, r, mc, n_mc - 1, lane)));
                } else {
                    // partial tile: rewrite only the codes of tokens in [lo, hi), byte by byte (a code
                    // never straddles a byte); lane 4 c + q owns field (mc, c, q)
                    const int c = lane >> 2, q = lane & 3;
                    if (16 * mc + c < r) {
                        for (int p = 8, off = 0; p >= 1; p >>= 1) {
                            if (b == 8 ? p != 8 : (p == 8 || !(b & p))) continue;
                            const int sh = b == 8 ? 0 : (b & (p - 1));
                            const uint32_t vm = p == 8 ? 0xffu : ((1u << p) - 1u);
                            uint8_t* __restrict__ dst = tbase + 8 * r * off + v_field_off(p, r, mc, c, q);
                            for (int m = 0; m < 16; ++m) {
                                const int tk = tok0 + 16 * q + kidx_b(b, m);
                                if (tk >= lo && tk < hi) {
                                    const uint32_t v = ((uint32_t)sb[kVRow * c + 16 * q + m] >> sh) & vm;
                                    const int bit = p * m;
                                    dst[bit >> 3] = (uint8_t)((dst[bit >> 3] & ~(vm << (bit & 7))) | (v << (bit & 7)));
                                }
                            }
                            off += p;
                        }
                    }
                }
            } else if (full) {
                KVC_SWITCH_B(b, (pack_group<side, B_>(sb, tbase, r, sl0, n_sl, lane)));
            } else {
                // partial tile: rewrite only the slots of tokens in [lo, hi)
                for (int p = 8, off = 0; p >= 1; p >>= 1) {
                    if (b == 8 ? p != 8 : (p == 8 || !(b & p))) continue;
                    const int sh = b == 8 ? 0 : (b & (p - 1));
                    const int ppw = 32 / p, nw = n_sl / ppw;
                    const uint32_t vm = p == 8 ? 0xffu : ((1u << p) - 1u);
                    uint32_t* __restrict__ pw = reinterpret_cast<uint32_t*>(tbase + 8 * r * off) + sl0 / ppw;
                    for (int wi = lane; wi < nw; wi += 64) {
                        uint32_t word = 0, msk = 0;
                        for (int io = 0; io < ppw; ++io) {
                            const int ph = sl0 + wi * ppw + io;
                            int t2, i2;
                            unslot_k(ph, r, t2, i2);
                            const int tk = tok0 + t2;
                            if (tk >= lo && tk < hi) {
                                const int bit = p * io;
                                word |= (((uint32_t)sb[sb_off<side>(wi * ppw + io)] >> sh) & vm) << bit;
                                msk |= vm << bit;
                            }
                        }
                        pw[wi] = (pw[wi] & ~msk) | word;
                    }
                    off += p;
                }
            }
            __builtin_amdgcn_wave_barrier();
        }
    }
}

// ---------------------------------------------------------------- append

// One side: one block per unit.
__global__ __launch_bounds__(kAppThreads) void append_kernel(DevSide s, int side, const uint16_t* __restrict__ x,
                                                             int64_t x_stride, int t0, int n_tok) {
    append_unit(s, side, x, x_stride, t0, n_tok, blockIdx.x);
}

// Both sides in one launch: block (u, 0) appends unit u's keys, block (u, 1) its values.
__global__ __launch_bounds__(kAppThreads) void append_kv_kernel(DevSide k, DevSide v, const uint16_t* __restrict__ xk,
                                                                int64_t xk_stride, const uint16_t* __restrict__ xv,
                                                                int64_t xv_stride, int t0, int n_tok) {
    if (blockIdx.y == 0) append_unit(k, KVC_SIDE_K, xk, xk_stride, t0, n_tok, blockIdx.x);
    else append_unit(v, KVC_SIDE_V, xv, xv_stride, t0, n_tok, blockIdx.x);
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
            const uint32_t code = side == KVC_SIDE_K ? load_code(tile, r, b, slot_k(tl, i, r)) : load_code_v(tile, r, b, tl, i);
            z = ((float)code - half) * step;
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
    const int n_tiles = (t0 + n_tok - 1) / kTile - tile_first + 1;
    const size_t smem = (size_t)kD * kPRow * 2 + 2 * kD * 4 + (kEncMmaThreads / 64) * (kTile * 4 + kSlotBufBytes) +
                        (s->side == KVC_SIDE_V ? (kEncMmaThreads / 64) * kVStageBytes : 0);
    dim3 grid((n_tiles + kEncMmaTilesPerBlock - 1) / kEncMmaTilesPerBlock, s->n_units);
    if (s->side == KVC_SIDE_K)
        hipLaunchKernelGGL(encode_mfma_kernel<KVC_SIDE_K>, grid, dim3(kEncMmaThreads), smem, (hipStream_t)stream,
                           dev_side(s), x, x_unit_stride, t0, n_tok, tile_first, n_tiles);
    else
        hipLaunchKernelGGL(encode_mfma_kernel<KVC_SIDE_V>, grid, dim3(kEncMmaThreads), smem, (hipStream_t)stream,
                           dev_side(s), x, x_unit_stride, t0, n_tok, tile_first, n_tiles);
    return check_launch("kvc_encode");
}

extern "C" int kvc_encode_kv(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* xk,
                             int64_t xk_unit_stride, const uint16_t* xv, int64_t xv_unit_stride, int32_t t0,
                             int32_t n_tok, void* stream) {
    clear_error();
    if (int e = validate_desc(k, "kvc_encode_kv(k)")) return e;
    if (int e = validate_desc(v, "kvc_encode_kv(v)")) return e;
    if (k->side != KVC_SIDE_K || v->side != KVC_SIDE_V) return set_error(KVC_EINVAL, "kvc_encode_kv: descriptor sides");
    if (k->n_units != v->n_units) return set_error(KVC_EINVAL, "kvc_encode_kv: K and V unit counts differ");
    if (n_tok > kAppMaxTok) {  // runs of tiles: the bulk encoder, one launch per side
        if (int e = kvc_encode(k, xk, xk_unit_stride, t0, n_tok, stream)) return e;
        return kvc_encode(v, xv, xv_unit_stride, t0, n_tok, stream);
    }
    if (t0 < 0 || n_tok < 0) return set_error(KVC_EINVAL, "kvc_encode_kv: negative t0 or n_tok");
    if ((int64_t)t0 + n_tok > k->capacity || (int64_t)t0 + n_tok > v->capacity)
        return set_error(KVC_ENOSPACE, "kvc_encode_kv: t0 + n_tok > capacity");
    if (n_tok == 0 || k->n_units == 0) return KVC_OK;
    for (const auto& xs : {std::make_pair(xk, xk_unit_stride), std::make_pair(xv, xv_unit_stride)})
        if (!xs.first || (reinterpret_cast<uintptr_t>(xs.first) & 15) || (xs.second & 7) || xs.second < (int64_t)n_tok * kD)
            return set_error(KVC_EINVAL, "kvc_encode_kv: x must be 16-byte aligned with stride a multiple of 8 and >= n_tok*d");
    hipLaunchKernelGGL(append_kv_kernel, dim3(k->n_units, 2), dim3(kAppThreads), 0, (hipStream_t)stream, dev_side(k),
                       dev_side(v), xk, xk_unit_stride, xv, xv_unit_stride, t0, n_tok);
    return check_launch("kvc_encode_kv");
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
