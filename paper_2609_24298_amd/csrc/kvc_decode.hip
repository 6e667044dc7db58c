// Decode attention over the packed KV-COBRA cache on CDNA4 (gfx950): kernels
// and the kvc_decode_attn launcher.
//
// The logits and the probability-weighted sum of values are dense contractions
// in the rank space: S = Qt (G x r_K) . C_K^T (r_K x tokens) and
// A = P (G x tokens) . C_V (tokens x r_V). Both run on int8 matrix cores
// (v_mfma_i32_16x16x64_i8) with exact int32 accumulation:
//  * codes enter as int8 (raw codes for b <= 7; c - 128 for b = 8);
//  * the rank-space query q~ = P_K q is split into three balanced base-254
//    int8 limbs with a per-query scale (relative error ~1e-7 of max|q~|);
//  * the softmax weights p in [0, 1] are quantised to 21 bits,
//    P = round(p (2^21 - 1)), and split into three 7-bit limbs;
//  * centring (c - 2^(b-1)) is exact in integers: the logits subtract
//    2^(b-1) sum_i Q_i, and the value accumulator carries an all-ones virtual
//    coordinate whose column gives sum_t P_t (also the softmax denominator).
// Per work item = (unit, context chunk) one wavefront walks the chunk in 64-token
// tiles. Each packed K and V tile is staged in LDS with coalesced 16-byte loads
// (the next tile's loads are in flight while the current one is computed);
// operand fragments are extracted from LDS by code instantiated per bit width
// (one switch per tile and side). The logits take the q~ limbs as the A operand
// (rows = head x limb) and the K codes as B (columns = tokens), so each lane
// receives the three limbs of one (head, token) pair and forms the logit alone.
// The online softmax keeps a lazily raised running max per query head; the
// probabilities are split into limbs and written to LDS in the token order of the
// V layout, where they are read back as the A operand of the PV products. Those
// accumulate in int32 MFMA accumulators across the whole chunk and are rescaled in
// place when a head's max grows. Centring and the limb sum happen once at the end
// of the chunk. A second kernel merges the chunks and applies step_V and the V basis.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>

#include "kvc_device.h"
#include "kvc_internal.h"

namespace kvc {

constexpr int kD = KVC_HEAD_DIM;
constexpr int kTile = KVC_TILE_TOKENS;
constexpr int kPartStride = 132;  // floats per (item, query head): m, l, pad, pad, acc[128]
constexpr int kAccStride = 132;   // LDS fp32 accumulator row: coordinates 0..127, 128 = all-ones column
constexpr int kLimbs = 3;
constexpr float kLazy = 6.f;               // the running max is raised only when a tile beats it by > 2^6
constexpr float kPScale = 32767.984375f;   // (2^21 - 1) / 2^6: p <= 2^6 maps to P < 2^21

typedef int32_t v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i mfma_i8(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// Value of lane (lane + n) mod 16 within each row of 16 lanes (DPP row rotate).
template <int N>
__device__ __forceinline__ float row_ror(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x120 + N, 0xf, 0xf, false));
}

__device__ __forceinline__ constexpr uint32_t plane_mask(int p) {
    return p == 8 ? 0xffffffffu : (p == 4 ? 0x0f0f0f0fu : (p == 2 ? 0x03030303u : 0x01010101u));
}

// 16 slots [phi0, phi0 + 16) of one plane of width P, phi0 a multiple of 16:
// dword d, byte j holds the plane value of slot phi0 + 4d + j.
template <int P>
__device__ __forceinline__ void plane_frag16(const uint8_t* __restrict__ plane, int phi0, uint32_t d[4]) {
    constexpr uint32_t M = plane_mask(P);
    if constexpr (P == 8) {
        const uint4 w = *reinterpret_cast<const uint4*>(plane + phi0);
        d[0] = w.x; d[1] = w.y; d[2] = w.z; d[3] = w.w;
    } else if constexpr (P == 4) {
        const uint2 w = *reinterpret_cast<const uint2*>(plane + (phi0 >> 1));
        d[0] = w.x & M; d[1] = (w.x >> 4) & M; d[2] = w.y & M; d[3] = (w.y >> 4) & M;
    } else if constexpr (P == 2) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(plane + (phi0 >> 2));
        d[0] = w & M; d[1] = (w >> 2) & M; d[2] = (w >> 4) & M; d[3] = (w >> 6) & M;
    } else {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(plane + ((phi0 >> 5) << 2)) >> ((phi0 & 16) >> 2);
        d[0] = w & M; d[1] = (w >> 1) & M; d[2] = (w >> 2) & M; d[3] = (w >> 3) & M;
    }
}

template <int B, int K>
__device__ __forceinline__ void add_plane16(const uint8_t* __restrict__ tile, int r, int phi0, uint32_t acc[4]) {
    if constexpr (K < n_planes(B)) {
        uint32_t f[4];
        plane_frag16<plane_w(B, K)>(tile + 8 * r * plane_off(B, K), phi0, f);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[j] |= f[j] << plane_sh(B, K);
    }
}

// Codes of 16 aligned slots of a tile (rank r, B bits), one byte each; b = 8 codes are
// returned centred (c - 128) so that they fit int8.
template <int B>
__device__ __forceinline__ v4i code_frag16(const uint8_t* __restrict__ tile, int r, int phi0) {
    uint32_t acc[4] = {0, 0, 0, 0};
    add_plane16<B, 0>(tile, r, phi0, acc);
    add_plane16<B, 1>(tile, r, phi0, acc);
    add_plane16<B, 2>(tile, r, phi0, acc);
    constexpr uint32_t X = B == 8 ? 0x80808080u : 0u;
    return v4i{(int)(acc[0] ^ X), (int)(acc[1] ^ X), (int)(acc[2] ^ X), (int)(acc[3] ^ X)};
}

template <int B, int K>
__device__ __forceinline__ uint32_t plane_subdword(const uint8_t* __restrict__ tile, int r, int sd) {
    if constexpr (K < n_planes(B)) {
        constexpr int P = plane_w(B, K);
        constexpr int SPW = 8 / P;  // sub-dwords per word
        const uint32_t w = reinterpret_cast<const uint32_t*>(tile + 8 * r * plane_off(B, K))[sd / SPW];
        return ((w >> (P * (sd % SPW))) & plane_mask(P)) << plane_sh(B, K);
    } else {
        return 0u;
    }
}

// Codes of the 4 slots of sub-dword sd of a tile (any alignment), one byte each (b = 8 centred).
template <int B>
__device__ __forceinline__ uint32_t code_subdword(const uint8_t* __restrict__ tile, int r, int sd) {
    return (plane_subdword<B, 0>(tile, r, sd) | plane_subdword<B, 1>(tile, r, sd) | plane_subdword<B, 2>(tile, r, sd)) ^
           (B == 8 ? 0x80808080u : 0u);
}

// ---------------------------------------------------------------- q~ limbs

// Per unit and query head: q~ = (step_K log2(e) / sqrt(d)) P_K q, its scale
// sigma = max|q~| / 127 and three int8 limbs with q~ ~ sigma (L0 + L1/254 + L2/254^2);
// corr[limb][g] = 2^(b_K - 1) sum_i L_limb,i (0 for b_K = 8, whose codes are centred on load).
__global__ __launch_bounds__(kD) void qprep_kernel(DevSide K, const uint16_t* __restrict__ q, int G,
                                                   int8_t* __restrict__ qlimb, float* __restrict__ qscale,
                                                   int32_t* __restrict__ qcorr) {
    __shared__ float qsh[16][kD];
    __shared__ float fred[kD / 64];
    __shared__ int ired[kLimbs][kD / 64];
    const int u = blockIdx.x, i = threadIdx.x, lane = i & 63, wv = i >> 6;
    for (int g = 0; g < G; ++g) qsh[g][i] = h2f(q[((int64_t)u * G + g) * kD + i]);
    __syncthreads();
    const int r = K.r[u], b = K.b[u];
    const int hk = b == 8 ? 0 : (1 << (b - 1));
    const float scale0 = K.delta[u] * 1.4426950408889634f * 0.08838834764831845f;  // log2(e) / sqrt(128)
    // basis row i, read once with 16-byte loads
    float prow[kD];
    {
        const uint4* P4 = reinterpret_cast<const uint4*>(K.basis + K.basis_off[u] + (int64_t)(i < r ? i : 0) * kD);
#pragma unroll
        for (int c = 0; c < kD / 8; ++c) {
            const uint4 w = P4[c];
            const uint32_t w4[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                prow[8 * c + 2 * e] = i < r ? h2f((uint16_t)(w4[e] & 0xffff)) : 0.f;
                prow[8 * c + 2 * e + 1] = i < r ? h2f((uint16_t)(w4[e] >> 16)) : 0.f;
            }
        }
    }
    for (int g = 0; g < G; ++g) {
        float acc = 0.f;
#pragma unroll
        for (int j = 0; j < kD; ++j) acc = fmaf(prow[j], qsh[g][j], acc);
        const float qt = acc * scale0;
        float m = fabsf(qt);
        for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
        if (lane == 0) fred[wv] = m;
        __syncthreads();
        const float amax = fmaxf(fred[0], fred[1]);
        const float sigma = amax > 0.f ? amax / 127.f : 1.f;
        const float x = qt / sigma;
        const float l0 = fminf(fmaxf(rintf(x), -127.f), 127.f);
        const float r1 = (x - l0) * 254.f;
        const float l1 = fminf(fmaxf(rintf(r1), -127.f), 127.f);
        const float r2 = (r1 - l1) * 254.f;
        const float l2 = fminf(fmaxf(rintf(r2), -127.f), 127.f);
        const int L[kLimbs] = {(int)l0, (int)l1, (int)l2};
#pragma unroll
        for (int k = 0; k < kLimbs; ++k) {
            qlimb[(((int64_t)u * kLimbs + k) * G + g) * kD + i] = (int8_t)L[k];
            int s = L[k];
            for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o);
            if (lane == 0) ired[k][wv] = s;
        }
        __syncthreads();
        if (i < kLimbs) qcorr[((int64_t)u * kLimbs + i) * G + g] = hk * (ired[i][0] + ired[i][1]);
        if (i == 0) qscale[(int64_t)u * G + g] = sigma;
        __syncthreads();
    }
}

// ---------------------------------------------------------------- partials

template <int G> struct Shape {
    static constexpr int LM = (4 * G + 15) / 16;       // logit M-tiles: row 4 h + limb (limb 3 is zero)
    static constexpr int PM = (kLimbs * G + 15) / 16;  // PV M-tiles: row limb * G + h
    static constexpr int NV = kD / 16 + 1;             // V N-tiles incl. the all-ones coordinate
    // Wavefronts per SIMD the register budget is cut for (512 / W registers per lane, no spills).
    static constexpr int W = G == 1 || G == 4 ? 4 : (G == 2 ? 3 : (G == 8 ? 2 : 1));
};

// Token of logit column col in sub-tile st. With this order a lane's four tokens (st = 0..3) sit at
// the consecutive V slots 4 col + st of the token permutation psi, so its probability limbs go to
// LDS as one dword per limb.
__device__ __forceinline__ int tok_of(int st, int col) { return 16 * (col & 3) + 4 * (col >> 2) + st; }

// K tail group (r_K % 16 coordinates) of the staged tile, transposed to [token][16] bytes in LDS.
template <int BK>
__device__ __forceinline__ void k_tail(const uint8_t* __restrict__ ktile, int rk, uint8_t* __restrict__ tail, int lane) {
    const int g16 = rk >> 4, rho = rk & 15;
    const float inv_rho = 1.f / (float)rho;
    const int base_sd = g16 << 8;  // first sub-dword of the tail (slot 1024 g16)
    for (int sd = lane; sd < 16 * rho; sd += 64) {
        const uint32_t cw = code_subdword<BK>(ktile, rk, base_sd + sd);
        const int q0 = 4 * sd, q1 = q0 + 2;
        // q / rho for q < 64 rho: (q + 1/2) / rho sits >= 1/(2 rho) away from an integer, far above fp32 error
        const int t0i = (int)(((float)q0 + 0.5f) * inv_rho), t1i = (int)(((float)q1 + 0.5f) * inv_rho);
        *reinterpret_cast<uint16_t*>(tail + t0i * 16 + (q0 - t0i * rho)) = (uint16_t)(cw & 0xffff);
        *reinterpret_cast<uint16_t*>(tail + t1i * 16 + (q1 - t1i * rho)) = (uint16_t)(cw >> 16);
    }
}

// K operand fragments of K-step ks for the 4 sub-tiles (logit B operand): lane (grp, col) = token
// tok_of(st, col), coordinates 64 ks + 16 grp + [0, 16), read in the grouped layout without bounds:
// groups past r_K read stale LDS bytes, which meet zero q~ limbs, and the lanes of the tail group are
// replaced from the transposed tail by the caller. All reads stay below 1024 b_K bytes.
template <int BK>
__device__ __forceinline__ void k_frags(const uint8_t* __restrict__ ktile, int rk, int ks, int lane, v4i (&Bk)[4]) {
    const int col = lane & 15, grp = lane >> 4;
    const int cg = 4 * ks + grp;
#pragma unroll
    for (int st = 0; st < 4; ++st) Bk[st] = code_frag16<BK>(ktile, rk, (cg << 10) + (tok_of(st, col) << 4));
}

// V operand fragments of N-tiles nt0 .. nt0 + 4: lane (grp, col) = coordinate 16 nt + col, tokens
// 16 st + 4 grp + i at slot 4 st + i. Coordinates >= r_V read stale LDS bytes (below 1024 b_V bytes
// past the tile start) into accumulator columns that are never used; N-tile 8 is the all-ones column.
template <int BV>
__device__ __forceinline__ void v_frags(const uint8_t* __restrict__ vtile, int rv, int nt0, int lane, v4i ones,
                                        v4i (&Bf)[5]) {
    const int col = lane & 15, grp = lane >> 4;
#pragma unroll
    for (int k = 0; k < 5; ++k) {
        const int nt = nt0 + k;
        Bf[k] = nt == kD / 16 ? ones : code_frag16<BV>(vtile, rv, ((16 * nt + col) << 6) + (grp << 4));
    }
}

template <int G>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(Shape<G>::W, Shape<G>::W))) void decode_mfma_kernel(DevSide K, DevSide V, const int8_t* __restrict__ qlimb,
                                                         const float* __restrict__ qscale,
                                                         const int32_t* __restrict__ qcorr,
                                                         const int32_t* __restrict__ seq_len, int max_seq, int chunk,
                                                         int n_chunks, float* __restrict__ part, int raw_bytes) {
    constexpr int LM = Shape<G>::LM, PM = Shape<G>::PM, NV = Shape<G>::NV;
    extern __shared__ float smem[];
    float* accs = smem;                                                   // [G][kAccStride] fp32: coords 0..127, 128 = sum P
    float* alph = smem + G * kAccStride;                                  // [16] per-head rescale factors
    uint8_t* pmat = reinterpret_cast<uint8_t*>(alph + 16);               // [16 PM][64] probability limbs, V slot order
    uint8_t* tail = pmat + 16 * PM * kTile;                               // [64][16] K tail codes
    uint4* raw = reinterpret_cast<uint4*>(tail + kTile * 16);            // raw K tile, then V tile

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
    const int rk = K.r[u], bk = K.b[u], rv = V.r[u], bv = V.b[u];
    const int hv = bv == 8 ? 0 : (1 << (bv - 1));
    const int nk = (rk + 63) >> 6;
    const int nv = (rv + 15) >> 4;  // V N-tiles holding coordinates (N-tile 8 = all-ones column)
    const uint8_t* __restrict__ kstream = K.codes + K.code_off[u];
    const uint8_t* __restrict__ vstream = V.codes + V.code_off[u];

    // Logit A operands: lane (grp, col) = row 16 lm + col = (head 4 lm + col / 4, limb col % 4),
    // coordinates 64 ks + 16 grp + [0, 16). The logit of (head 4 lm + grp, token) is
    // sum_limb S_limb kq[lm][limb] + bq[lm] in the log2 domain (bq holds the centring correction).
    v4i qA[2][LM];
    float kq[LM][kLimbs], bq[LM];
#pragma unroll
    for (int lm = 0; lm < LM; ++lm) {
        const int h = 4 * lm + (col >> 2), limb = col & 3;
        const bool ok = h < G && limb < kLimbs;
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            v4i v = {0, 0, 0, 0};
            if (ok && ks < nk)
                v = *reinterpret_cast<const v4i*>(qlimb + (((int64_t)u * kLimbs + limb) * G + h) * kD + 64 * ks + 16 * grp);
            qA[ks][lm] = v;
        }
        const int hs = 4 * lm + grp;
        float bsum = 0.f;
#pragma unroll
        for (int l = 0; l < kLimbs; ++l) {
            const float ls = l == 0 ? 1.f : (l == 1 ? (1.f / 254.f) : (1.f / 64516.f));
            kq[lm][l] = hs < G ? qscale[(int64_t)u * G + hs] * ls : 0.f;
            if (hs < G) bsum = fmaf(-(float)qcorr[((int64_t)u * kLimbs + l) * G + hs], kq[lm][l], bsum);
        }
        bq[lm] = bsum;
    }
    for (int k = lane; k < G * kAccStride; k += 64) accs[k] = 0.f;
    for (int k = lane; k < 16 * PM * kTile / 4; k += 64) reinterpret_cast<uint32_t*>(pmat)[k] = 0u;
    __syncthreads();

    v4i Cpv[PM][NV];
#pragma unroll
    for (int pm = 0; pm < PM; ++pm)
#pragma unroll
        for (int nt = 0; nt < NV; ++nt) Cpv[pm][nt] = v4i{0, 0, 0, 0};
    float m_run[LM];  // running max (log2 domain) of head 4 lm + grp
#pragma unroll
    for (int lm = 0; lm < LM; ++lm) m_run[lm] = -INFINITY;

    // When a head's running max grows (by more than 2^kLazy, so alpha <= 2^-kLazy) its int32
    // accumulator rows are rescaled in place: C <- rint(C alpha). The rounding adds at most about one
    // quantum of P per rescale, the size of one token's quantisation error; rows of heads that kept
    // their max are left untouched. Rare (a few tiles per chunk), so it is written for size.
    auto rescale = [&](const float (&alpha)[LM]) {
        int ln = threadIdx.x;
        asm volatile("" : "+v"(ln));
        const int gr = ln >> 4;
#pragma unroll
        for (int lm = 0; lm < LM; ++lm)
            if ((ln & 15) == 0 && 4 * lm + gr < G) alph[4 * lm + gr] = alpha[lm];
        __syncthreads();
#pragma unroll
        for (int pm = 0; pm < PM; ++pm)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = 16 * pm + 4 * gr + i;
                const float a = row < kLimbs * G ? alph[row % G] : 1.f;
                const bool keep = a == 1.f;
#pragma unroll
                for (int nt = 0; nt < NV; ++nt) {
                    const int cur = Cpv[pm][nt][i];
                    const int scaled = (int)rintf((float)cur * a);
                    Cpv[pm][nt][i] = keep ? cur : scaled;
                }
            }
        __syncthreads();
    };

    const v4i ones = col == 0 ? v4i{0x01010101, 0x01010101, 0x01010101, 0x01010101} : v4i{0, 0, 0, 0};
    const int kch = (8 * rk * bk) >> 4, vch = (8 * rv * bv) >> 4;  // 16-byte chunks per K / V tile
    const uint8_t* ktile = reinterpret_cast<const uint8_t*>(raw);
    const uint8_t* vtile = reinterpret_cast<const uint8_t*>(raw + kch);
    // The packed K and V tiles are staged in LDS with coalesced 16-byte loads: chunk cc < kch of
    // the K tile, then the V tile's, 64 chunks per round. The first 4 rounds of the next tile are
    // loaded into registers while the current tile is computed; further rounds (tiles of more than
    // 4 KiB) are loaded when their tile is staged. Lanes past the last chunk reload the V tile's last.
    const int nch = kch + vch;
    const int64_t ktb = 8 * rk * bk, vtb = 8 * rv * bv;  // tile bytes
    auto chunk_src = [&](int tile, int cc) -> const uint4* {
        const uint4* kb = reinterpret_cast<const uint4*>(kstream + tile * ktb);
        const uint4* vb = reinterpret_cast<const uint4*>(vstream + tile * vtb) - kch;
        return (cc < kch ? kb : vb) + min(cc, nch - 1);
    };
    uint4 pf0, pf1, pf2, pf3;
    {
        const int tile = start / kTile;
        pf0 = *chunk_src(tile, lane);
        pf1 = *chunk_src(tile, 64 + lane);
        pf2 = *chunk_src(tile, 128 + lane);
        pf3 = *chunk_src(tile, 192 + lane);
    }
    for (int tok0 = start; tok0 < end; tok0 += kTile) {
        // An opaque per-tile copy of the lane id: lane-dependent fragment offsets are recomputed
        // inside the loop instead of being hoisted and kept live in registers across it.
        int lane_it = lane;
        asm volatile("" : "+v"(lane_it));
        const int col_it = lane_it & 15, grp_it = lane_it >> 4;
        const int tile = tok0 / kTile;
        if (lane_it < nch) raw[lane_it] = pf0;
        if (64 + lane_it < nch) raw[64 + lane_it] = pf1;
        if (128 + lane_it < nch) raw[128 + lane_it] = pf2;
        if (192 + lane_it < nch) raw[192 + lane_it] = pf3;
        for (int c0 = 256; c0 < nch; c0 += 64)
            if (c0 + lane_it < nch) raw[c0 + lane_it] = *chunk_src(tile, c0 + lane_it);
        __syncthreads();
        if (tok0 + kTile < end) {
            pf0 = *chunk_src(tile + 1, lane_it);
            pf1 = *chunk_src(tile + 1, 64 + lane_it);
            pf2 = *chunk_src(tile + 1, 128 + lane_it);
            pf3 = *chunk_src(tile + 1, 192 + lane_it);
        }
        // Logits: S[lm][st] = q~ limbs (rows) . codes (64 coords x 16 tokens), summed over K-steps.
        if (rk & 15) {
            KVC_SWITCH_B(bk, k_tail<B_>(ktile, rk, tail, lane_it));
            __syncthreads();
        }
        v4i S[LM][4];
#pragma unroll
        for (int lm = 0; lm < LM; ++lm)
#pragma unroll
            for (int st = 0; st < 4; ++st) S[lm][st] = v4i{0, 0, 0, 0};
        // All MFMAs are issued unconditionally (absent coordinates contribute zero fragments), which
        // keeps the accumulator code straight-line.
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            v4i Bk[4];
            KVC_SWITCH_B(bk, k_frags<B_>(ktile, rk, ks, lane_it, Bk));
            if ((rk & 15) && (rk >> 6) == ks) {  // this K-step holds the tail group: its lanes read the transposed copy
#pragma unroll
                for (int st = 0; st < 4; ++st) {
                    const v4i tv = *reinterpret_cast<const v4i*>(tail + tok_of(st, col_it) * 16);
                    if (grp_it == ((rk >> 4) & 3)) Bk[st] = tv;
                }
            }
#pragma unroll
            for (int st = 0; st < 4; ++st)
#pragma unroll
                for (int lm = 0; lm < LM; ++lm) S[lm][st] = mfma_i8(qA[ks][lm], Bk[st], S[lm][st]);
        }
        // Lane (grp, col) holds the three limbs of head 4 lm + grp for token tok_of(st, col).
        float s[LM][4];
#pragma unroll
        for (int lm = 0; lm < LM; ++lm)
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                float v = fmaf((float)S[lm][st][0], kq[lm][0], bq[lm]);
                v = fmaf((float)S[lm][st][1], kq[lm][1], v);
                s[lm][st] = fmaf((float)S[lm][st][2], kq[lm][2], v);
            }
        if (tok0 + kTile > end) {  // last tile of the chunk: tokens past the end get zero weight
#pragma unroll
            for (int st = 0; st < 4; ++st)
                if (tok0 + tok_of(st, col_it) >= end) {
#pragma unroll
                    for (int lm = 0; lm < LM; ++lm) s[lm][st] = -INFINITY;
                }
        }

        // Online softmax: running max per head over the 16 lanes of its row; the int32
        // accumulators are rescaled when it grows past the lazy margin.
        float alpha[LM];
        bool grow = false;
#pragma unroll
        for (int lm = 0; lm < LM; ++lm) {
            float m = fmaxf(fmaxf(s[lm][0], s[lm][1]), fmaxf(s[lm][2], s[lm][3]));
            m = fmaxf(m, row_ror<8>(m));
            m = fmaxf(m, row_ror<4>(m));
            m = fmaxf(m, row_ror<2>(m));
            m = fmaxf(m, row_ror<1>(m));
            // lazy: keep the stale max while the tile stays within 2^kLazy of it (p <= 2^kLazy then)
            const float mn = m > m_run[lm] + kLazy ? m : m_run[lm];
            alpha[lm] = mn > m_run[lm] ? __builtin_amdgcn_exp2f(m_run[lm] - mn) : 1.f;
            grow = grow || (mn > m_run[lm] && m_run[lm] > -INFINITY);
            m_run[lm] = mn;
        }
        if (__any(grow)) rescale(alpha);

        // Probability limbs: P = round(p (2^21 - 1) / 2^kLazy) = L0 2^14 + L1 2^7 + L2 (p <= 2^kLazy).
        // Row limb * G + h of pmat, bytes 4 col .. 4 col + 3 = tokens tok_of(0..3, col).
#pragma unroll
        for (int lm = 0; lm < LM; ++lm) {
            const int h = 4 * lm + grp_it;
            uint32_t P[4];
#pragma unroll
            for (int st = 0; st < 4; ++st)
                P[st] = (uint32_t)fmaf(__builtin_amdgcn_exp2f(s[lm][st] - m_run[lm]), kPScale, 0.5f);
            if (G >= 4 * (lm + 1) || h < G) {
#pragma unroll
                for (int l = 0; l < kLimbs; ++l) {
                    const uint32_t sh = 14 - 7 * l;
                    uint32_t w = (P[0] >> sh) & 0x7fu;
#pragma unroll
                    for (int st = 1; st < 4; ++st) w |= ((P[st] >> sh) & 0x7fu) << (8 * st);
                    *reinterpret_cast<uint32_t*>(pmat + (l * G + h) * kTile + 4 * col_it) = w;
                }
            }
        }
        __syncthreads();
        v4i Ap[PM];
#pragma unroll
        for (int pm = 0; pm < PM; ++pm)
            Ap[pm] = *reinterpret_cast<const v4i*>(pmat + (16 * pm + col_it) * kTile + 16 * grp_it);

        // PV: Cpv[pm][nt] += P limbs (rows x 64 tokens) . V codes (64 tokens x 16 coords).
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int nt0 = 5 * half;
            v4i Bf[5];
            KVC_SWITCH_B(bv, v_frags<B_>(vtile, rv, nt0, lane_it, ones, Bf));
#pragma unroll
            for (int k = 0; k < 5; ++k)
                if (nt0 + k < NV)
#pragma unroll
                    for (int pm = 0; pm < PM; ++pm) Cpv[pm][nt0 + k] = mfma_i8(Ap[pm], Bf[k], Cpv[pm][nt0 + k]);
        }
        __syncthreads();  // raw and pmat are rewritten by the next tile
    }
    // Centre (exact, in integers, with the all-ones column O) and combine the three P limbs of each
    // head into the fp32 LDS accumulator: accs[g][c] = sum_limb ls (C - 2^(b-1) O), accs[g][128] = sum_limb ls O.
    {
#pragma unroll
        for (int pm = 0; pm < PM; ++pm)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int row = 16 * pm + 4 * grp + i;
                const int plimb = row / G, g = row - plimb * G;
                const int O = __shfl(Cpv[pm][NV - 1][i], lane & 48);
                const float ls = plimb == 0 ? 16384.f : (plimb == 1 ? 128.f : 1.f);
                float* arow = accs + g * kAccStride;
                if (plimb < kLimbs) {
#pragma unroll
                    for (int nt = 0; nt < NV - 1; ++nt) {
                        const int coord = 16 * nt + col;
                        if (nt < nv && coord < rv) atomicAdd(arow + coord, (float)(Cpv[pm][nt][i] - hv * O) * ls);
                    }
                    if (col == 0) atomicAdd(arow + kD, (float)O * ls);
                }
            }
    }
    __syncthreads();

    // Partial of each head: m, l = sum of P (all-ones column), centred accumulator.
#pragma unroll
    for (int g = 0; g < G; ++g) {
        const float mg = __shfl(m_run[g / 4], 16 * (g % 4));
        float* o = out + g * kPartStride;
        const float* arow = accs + g * kAccStride;
        if (lane == 0) { o[0] = mg; o[1] = arow[kD]; }
        o[4 + lane] = lane < rv ? arow[lane] : 0.f;
        o[4 + 64 + lane] = lane + 64 < rv ? arow[lane + 64] : 0.f;
    }
}

// ---------------------------------------------------------------- combine

__global__ __launch_bounds__(kD) void combine_kernel(DevSide V, int G, int n_chunks, const float* __restrict__ part,
                                                     float* __restrict__ out) {
    constexpr int kMaxG = 16;
    __shared__ float zs[kMaxG][kD];
    __shared__ float lsum[kMaxG];
    const int u = blockIdx.x, j = threadIdx.x;
    const int rv = V.r[u];
    const float step = V.delta[u];
    const float* __restrict__ pu = part + (int64_t)u * n_chunks * G * kPartStride;
    for (int g = 0; g < G; ++g) {
        const float* pg = pu + g * kPartStride;
        float M = -INFINITY;
        for (int c = 0; c < n_chunks; ++c) M = fmaxf(M, pg[(int64_t)c * G * kPartStride]);
        float L = 0.f, A = 0.f;
        for (int c = 0; c < n_chunks; ++c) {
            const float* pc = pg + (int64_t)c * G * kPartStride;
            const float lc = pc[1];
            if (lc > 0.f) {
                const float w = exp2f(pc[0] - M);
                L = fmaf(lc, w, L);
                if (j < rv) A = fmaf(pc[4 + j], w, A);
            }
        }
        zs[g][j] = (L > 0.f && j < rv) ? step * (A / L + 0.5f) : 0.f;
        if (j == 0) lsum[g] = L;
    }
    __syncthreads();
    // o_g = P_V^T z_g for every head in one pass over the basis (coalesced rows of P)
    const uint16_t* __restrict__ P = V.basis + V.basis_off[u];
    float o[kMaxG];
#pragma unroll
    for (int g = 0; g < kMaxG; ++g) o[g] = 0.f;
    for (int i = 0; i < rv; ++i) {
        const float p = h2f(P[(int64_t)i * kD + j]);
#pragma unroll
        for (int g = 0; g < kMaxG; ++g)
            if (g < G) o[g] = fmaf(p, zs[g][i], o[g]);
    }
#pragma unroll
    for (int g = 0; g < kMaxG; ++g)
        if (g < G) out[((int64_t)u * G + g) * kD + j] = lsum[g] > 0.f ? o[g] : 0.f;
}

// ---------------------------------------------------------------- host side

namespace {

// Raw LDS bytes for the staged tiles: fragment reads run past the staged tiles (up to 1024 b bytes
// from each tile start), so the region covers max(1024 b_K, 8 r_K b_K + 1024 b_V) over the units.
int raw_tile_bytes(const kvc_stream_desc* k, const kvc_stream_desc* v) {
    int raw = 16;
    for (int u = 0; u < k->n_units; ++u) {
        const int kb = 8 * k->r_host[u] * k->b_host[u];
        raw = std::max(raw, std::max(1024 * k->b_host[u], kb + 1024 * v->b_host[u]));
    }
    return raw;
}

size_t partial_smem(int G, int raw_bytes) {
    const int PM = (kLimbs * G + 15) / 16;
    return (size_t)G * kAccStride * 4 + 16 * 4 + (size_t)16 * PM * kTile + kTile * 16 + (size_t)raw_bytes;
}

template <int G>
int resident_blocks(size_t smem) {
    int nb = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, decode_mfma_kernel<G>, 64, smem) != hipSuccess || nb <= 0) {
        (void)hipGetLastError();
        nb = 8;
    }
    return nb;
}

// Work items (wavefronts) the device holds at once for this launch; without a device, the
// MI355X figures (256 CUs, 8 resident wavefronts each).
int64_t resident_slots(int G, size_t smem) {
    int dev = 0, ncu = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        ncu <= 0) {
        (void)hipGetLastError();
        ncu = 256;
    }
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

// Split of each unit's context into n_chunks equal chunks of whole tiles. Among counts that give
// at least one work item per resident slot, the count minimises
//   rounds x (tiles per item + per-item overhead) + (straggler share) x tiles per item,
// rounds = ceil(items / resident slots): whole rounds with no short remainder, and items short
// enough that units of different cost even out (measured on the 32-layer 32k-token workload:
// 9 chunks of 57 tiles beat 3 chunks of 171 by 11 % and 24 chunks of 22 by 12 %).
constexpr int kItemOverheadTiles = 4;
constexpr double kStragglerShare = 0.5;

struct WsLayout {
    int chunk, n_chunks, raw_bytes;
    int64_t qlimb, qscale, qcorr, part, total;  // byte offsets
};

WsLayout ws_layout(const kvc_stream_desc* k, const kvc_stream_desc* v, int G, int max_seq) {
    WsLayout L;
    const int U = k->n_units;
    L.raw_bytes = raw_tile_bytes(k, v);
    const int64_t slots = resident_slots(G, partial_smem(G, L.raw_bytes));
    const int tpu = (max_seq + kTile - 1) / kTile;
    // Candidates that fill every resident slot rank by cost; if none can (few units, short
    // contexts), the one with the most items wins.
    bool best_full = false;
    double best_cost = 0.0;
    int64_t best_items = -1;
    L.chunk = tpu * kTile;
    L.n_chunks = 1;
    for (int n = 1; n <= tpu && n <= 1024; ++n) {
        const int c = (tpu + n - 1) / n;
        if ((tpu + c - 1) / c != n) continue;
        const int64_t items = (int64_t)U * n;
        const bool full = items >= slots;
        const int64_t rounds = (items + slots - 1) / slots;
        const double cost = (double)rounds * (c + kItemOverheadTiles) + kStragglerShare * c;
        const bool better = best_items < 0 || (full && !best_full) ||
                            (full && best_full && cost < best_cost) || (!full && !best_full && items > best_items);
        if (better) {
            best_full = full;
            best_cost = cost;
            best_items = items;
            L.chunk = c * kTile;
            L.n_chunks = n;
        }
    }
    auto up = [](int64_t x) { return (x + 255) / 256 * 256; };
    L.qlimb = 0;
    L.qscale = up(L.qlimb + (int64_t)U * kLimbs * G * kD);
    L.qcorr = up(L.qscale + (int64_t)U * G * 4);
    L.part = up(L.qcorr + (int64_t)U * kLimbs * G * 4);
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
    return KVC_OK;
}

template <int G>
int launch_partials(dim3 grid, hipStream_t st, const DevSide& K, const DevSide& V, const int8_t* ql, const float* qs,
                    const int32_t* qc, const int32_t* seq_len, int max_seq, int chunk, int n_chunks, float* part,
                    int raw_bytes) {
    const size_t smem = partial_smem(G, raw_bytes);
    if (smem > 64 * 1024) {
        const hipError_t e = hipFuncSetAttribute((const void*)decode_mfma_kernel<G>,
                                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem);
        if (e != hipSuccess) return set_error(KVC_EDEVICE, "hipFuncSetAttribute: %s", hipGetErrorString(e));
    }
    hipLaunchKernelGGL(decode_mfma_kernel<G>, grid, dim3(64), smem, st, K, V, ql, qs, qc, seq_len, max_seq, chunk,
                       n_chunks, part, raw_bytes);
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

using namespace kvc;

extern "C" size_t kvc_decode_attn_workspace(const kvc_stream_desc* k, const kvc_stream_desc* v, int32_t G,
                                            int32_t max_seq_len) {
    clear_error();
    if (decode_check(k, v, G, max_seq_len)) return 0;
    return (size_t)ws_layout(k, v, G, max_seq_len).total;
}

extern "C" int kvc_decode_attn(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q, int32_t G,
                               const int32_t* seq_len, int32_t max_seq_len, float* out, void* ws, size_t ws_bytes,
                               void* stream) {
    clear_error();
    if (int e = decode_check(k, v, G, max_seq_len)) return e;
    if (k->n_units == 0) return KVC_OK;
    if (!q || !seq_len || !out || !ws) return set_error(KVC_EINVAL, "kvc_decode_attn: null pointer");
    if (reinterpret_cast<uintptr_t>(ws) & 255) return set_error(KVC_EINVAL, "kvc_decode_attn: workspace not 256-byte aligned");
    const int U = k->n_units;
    const WsLayout L = ws_layout(k, v, G, max_seq_len);
    if ((int64_t)ws_bytes < L.total)
        return set_error(KVC_ENOSPACE, "kvc_decode_attn: workspace %zu < %lld bytes", ws_bytes, (long long)L.total);
    char* w = reinterpret_cast<char*>(ws);
    int8_t* ql = reinterpret_cast<int8_t*>(w + L.qlimb);
    float* qs = reinterpret_cast<float*>(w + L.qscale);
    int32_t* qc = reinterpret_cast<int32_t*>(w + L.qcorr);
    float* part = reinterpret_cast<float*>(w + L.part);
    hipStream_t st = (hipStream_t)stream;
    const DevSide K = dev_side(k), V = dev_side(v);
    hipLaunchKernelGGL(qprep_kernel, dim3(U), dim3(kD), 0, st, K, q, G, ql, qs, qc);
    const int raw_bytes = L.raw_bytes;
    const dim3 grid(L.n_chunks, U);
    int e = KVC_OK;
    switch (G) {
        case 1: e = launch_partials<1>(grid, st, K, V, ql, qs, qc, seq_len, max_seq_len, L.chunk, L.n_chunks, part, raw_bytes); break;
        case 2: e = launch_partials<2>(grid, st, K, V, ql, qs, qc, seq_len, max_seq_len, L.chunk, L.n_chunks, part, raw_bytes); break;
        case 4: e = launch_partials<4>(grid, st, K, V, ql, qs, qc, seq_len, max_seq_len, L.chunk, L.n_chunks, part, raw_bytes); break;
        case 8: e = launch_partials<8>(grid, st, K, V, ql, qs, qc, seq_len, max_seq_len, L.chunk, L.n_chunks, part, raw_bytes); break;
        default: e = launch_partials<16>(grid, st, K, V, ql, qs, qc, seq_len, max_seq_len, L.chunk, L.n_chunks, part, raw_bytes); break;
    }
    if (e) return e;
    hipLaunchKernelGGL(combine_kernel, dim3(U), dim3(kD), 0, st, V, G, L.n_chunks, part, out);
    return check_launch("kvc_decode_attn");
}
