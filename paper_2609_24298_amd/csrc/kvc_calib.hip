// Calibration statistics on the device (table step 1): per-head covariance of calibration
// activations, its eigendecomposition, and the query variance along each key eigendirection, for
// many heads at once (CDNA4 / gfx950). The allocator (kvc_allocate, host) and the basis builder
// (kvc_make_basis, host) consume the results.
//
//  * covariance_kernel: C = (1/n) X^T X - mu mu^T per head on fp16 matrix cores
//    (v_mfma_f32_16x16x32_f16, exact fp16 products, fp32 accumulation). One block of four
//    wavefronts per head walks the tokens in tiles of 128 staged in LDS; each wavefront owns a
//    64 x 64 quadrant of the output (16 tiles of 16 x 16).
//  * eigh_kernel: fp32 parallel cyclic Jacobi (the precision the paper states for its
//    eigendecomposition). One block per head holds A and the accumulated rotations V in LDS
//    (2 x 128 x 129 floats). A sweep is 127 rounds of the round-robin ordering; each round
//    annihilates 64 disjoint off-diagonal pairs at once (the rotations commute), applied as
//    A <- A J, V <- V J (column pass) then A <- J^T A (row pass), each 2 x 2 pivot block set by the
//    exact formulas (a_pp - t a_pq, a_qq + t a_pq, 0) and the other entries rotated in the
//    x - s (y + tau x) form (Rutishauser), which keeps the rounding of the diagonal small.
//  * query_variance_kernel: sigma^2_Q,i = (1/G) sum_g u_i^T Sigma_Q,g u_i, U and Sigma_Q,g staged
//    in LDS, one thread per (column i, half of the rows).
//  * measured_quant_kernel: the quantization term of the measured distortion tables (Appendix D,
//    exact DP over measured distortion) for every candidate rank and width.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "kvc.h"
#include "kvc_internal.h"

namespace kvc {
namespace {

constexpr int kD = KVC_HEAD_DIM;
constexpr int kLd = kD + 1;  // padded LDS row (floats)

typedef _Float16 cv_h8 __attribute__((ext_vector_type(8)));
typedef float cv_f4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------- covariance

constexpr int kCovTok = 128;         // tokens staged per step
constexpr int kCovPitch = kD + 8;    // LDS row pitch of the staged tokens (halves)

__global__ __launch_bounds__(256) void covariance_kernel(const uint16_t* __restrict__ x, int64_t head_stride, int n_tok,
                                                         int centered, float* __restrict__ cov) {
    __shared__ __attribute__((aligned(16))) _Float16 xs[kCovTok * kCovPitch];
    __shared__ float msum[16][kD];
    const int h = blockIdx.x, tid = threadIdx.x, wv = tid >> 6, lane = tid & 63, col = lane & 15, kq = lane >> 4;
    const uint16_t* __restrict__ X = x + (int64_t)h * head_stride;
    const int I0 = 4 * (wv >> 1), J0 = 4 * (wv & 1);  // the wavefront's 4 x 4 block of 16 x 16 tiles
    cv_f4 C[4][4];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b) C[a][b] = cv_f4{0.f, 0.f, 0.f, 0.f};
    // partial feature sums: thread handles features 8 (tid % 16) .. + 7 of tokens tid / 16 + 16 k
    float fs[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const int fb = tid & 15, tr = tid >> 4;
    for (int t0 = 0; t0 < n_tok; t0 += kCovTok) {
        // stage 128 tokens (zero past n_tok): 16-byte loads, 8 features of one token each
#pragma unroll
        for (int k = 0; k < kCovTok / 16; ++k) {
            const int t = tr + 16 * k;
            uint4 w = uint4{0u, 0u, 0u, 0u};
            if (t0 + t < n_tok) w = reinterpret_cast<const uint4*>(X + (int64_t)(t0 + t) * kD)[fb];
            *reinterpret_cast<uint4*>(&xs[t * kCovPitch + 8 * fb]) = w;
            const cv_h8 v = __builtin_bit_cast(cv_h8, w);
#pragma unroll
            for (int e = 0; e < 8; ++e) fs[e] += (float)v[e];
        }
        __syncthreads();
        // four k-steps of 32 tokens; lane (col, kq) takes tokens 8 kq .. 8 kq + 7 of the step for
        // feature 16 I + col (A operand, rows = features) and 16 J + col (B operand, columns = features)
#pragma unroll
        for (int ks = 0; ks < kCovTok / 32; ++ks) {
            cv_h8 fa[4], fbv[4];
#pragma unroll
            for (int a = 0; a < 4; ++a) {
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int t = 32 * ks + 8 * kq + e;
                    fa[a][e] = xs[t * kCovPitch + 16 * (I0 + a) + col];
                    fbv[a][e] = xs[t * kCovPitch + 16 * (J0 + a) + col];
                }
            }
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int b = 0; b < 4; ++b) C[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_f16(fa[a], fbv[b], C[a][b], 0, 0, 0);
        }
        __syncthreads();
    }
    // feature means
#pragma unroll
    for (int e = 0; e < 8; ++e) msum[tr][8 * fb + e] = fs[e];
    __syncthreads();
    __shared__ float mu[kD];
    if (tid < kD) {
        float m = 0.f;
        for (int r = 0; r < 16; ++r) m += msum[r][tid];
        mu[tid] = m / (float)n_tok;
    }
    __syncthreads();
    const float inv_n = 1.f / (float)n_tok;
    float* __restrict__ out = cov + (int64_t)h * kD * kD;
    // lane (col, kq) holds rows 16 I + 4 kq + v, column 16 J + col of tile (I, J)
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int i = 16 * (I0 + a) + 4 * kq + v, j = 16 * (J0 + b) + col;
                float c = C[a][b][v] * inv_n;
                if (centered) c -= mu[i] * mu[j];
                out[i * kD + j] = c;
            }
}

// ---------------------------------------------------------------- eigendecomposition

constexpr int kEighThreads = 512;
constexpr int kMaxSweeps = 30;

// Pair k of round m of the round-robin ordering of 128 indices: (m, 127) and ((m + k) mod 127,
// (m - k) mod 127) for k = 1..63 cover every index once.
__device__ __forceinline__ void rr_pair(int m, int k, int& p, int& q) {
    if (k == 0) { p = m; q = kD - 1; return; }
    const int a = (m + k) % (kD - 1), b = (m - k + (kD - 1)) % (kD - 1);
    p = a < b ? a : b;
    q = a < b ? b : a;
}

__global__ __launch_bounds__(kEighThreads) void eigh_kernel(const float* __restrict__ S, float* __restrict__ lam,
                                                            float* __restrict__ U, int32_t* __restrict__ sweeps_out) {
    extern __shared__ float eig_sm[];
    float* A = eig_sm;            // [128][129]
    float* V = eig_sm + kD * kLd;  // [128][129]
    __shared__ float sn[kD / 2], tau[kD / 2], dlt[kD / 2];
    __shared__ int pp[kD / 2], qq[kD / 2];
    __shared__ float red[kEighThreads / 64];
    __shared__ int rotated;
    __shared__ int rank_of[kD];
    __shared__ float inv_norm[kD];
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* __restrict__ Sh = S + (int64_t)h * kD * kD;
    float f2 = 0.f;
    for (int e = tid; e < kD * kD; e += kEighThreads) {
        const int i = e >> 7, j = e & (kD - 1);
        const float a = Sh[e];
        A[i * kLd + j] = a;
        V[i * kLd + j] = i == j ? 1.f : 0.f;
        f2 += a * a;
    }
    for (int o = 32; o > 0; o >>= 1) f2 += __shfl_xor(f2, o);
    if ((tid & 63) == 0) red[tid >> 6] = f2;
    __syncthreads();
    float fro2 = 0.f;
    for (int w = 0; w < kEighThreads / 64; ++w) fro2 += red[w];
    // a rotation is skipped when |a_pq| is below the fp32 resolution of its diagonal pair, or below
    // 2^-40 of the matrix norm (entries that small no longer move any eigenvalue in fp32)
    const float floor_abs = ldexpf(sqrtf(fro2), -40);
    int sweep = 0;
    for (; sweep < kMaxSweeps; ++sweep) {
        if (tid == 0) rotated = 0;
        __syncthreads();
        for (int m = 0; m < kD - 1; ++m) {
            if (tid < kD / 2) {
                int p, q;
                rr_pair(m, tid, p, q);
                const float apq = A[p * kLd + q], app = A[p * kLd + p], aqq = A[q * kLd + q];
                float s = 0.f, ta = 0.f, t = 0.f;
                if (fabsf(apq) > fmaxf(ldexpf(sqrtf(fabsf(app) * fabsf(aqq)), -24), floor_abs)) {
                    const float theta = (aqq - app) / (2.f * apq);
                    t = copysignf(1.f, theta) / (fabsf(theta) + sqrtf(fmaf(theta, theta, 1.f)));
                    const float c = 1.f / sqrtf(fmaf(t, t, 1.f));
                    s = t * c;
                    ta = s / (1.f + c);
                    rotated = 1;
                }
                sn[tid] = s;
                tau[tid] = ta;
                dlt[tid] = t * apq;  // the pivot block becomes diag(a_pp - t a_pq, a_qq + t a_pq)
                pp[tid] = p;
                qq[tid] = q;
            }
            __syncthreads();
            // Columns p, q of A (rows outside the pivot block) and of V, in the form
            // x_p' = x_p - s (x_q + tau x_p), x_q' = x_q + s (x_p - tau x_q) (consecutive threads take
            // consecutive rows)
            for (int e = tid; e < kD * (kD / 2); e += kEighThreads) {
                const int i = e & (kD - 1), k = e >> 7;
                const float s = sn[k];
                if (s == 0.f) continue;
                const float ta = tau[k];
                const int p = pp[k], q = qq[k];
                if (i != p && i != q) {
                    const float aip = A[i * kLd + p], aiq = A[i * kLd + q];
                    A[i * kLd + p] = aip - s * (aiq + ta * aip);
                    A[i * kLd + q] = aiq + s * (aip - ta * aiq);
                }
                const float vip = V[i * kLd + p], viq = V[i * kLd + q];
                V[i * kLd + p] = vip - s * (viq + ta * vip);
                V[i * kLd + q] = viq + s * (vip - ta * viq);
            }
            __syncthreads();
            // rows p, q of A (columns outside the pivot block)
            for (int e = tid; e < kD * (kD / 2); e += kEighThreads) {
                const int j = e & (kD - 1), k = e >> 7;
                const float s = sn[k];
                if (s == 0.f) continue;
                const float ta = tau[k];
                const int p = pp[k], q = qq[k];
                if (j == p || j == q) continue;
                const float apj = A[p * kLd + j], aqj = A[q * kLd + j];
                A[p * kLd + j] = apj - s * (aqj + ta * apj);
                A[q * kLd + j] = aqj + s * (apj - ta * aqj);
            }
            __syncthreads();
            if (tid < kD / 2 && sn[tid] != 0.f) {  // the pivot block, by the exact 2 x 2 formulas
                const int p = pp[tid], q = qq[tid];
                A[p * kLd + p] -= dlt[tid];
                A[q * kLd + q] += dlt[tid];
                A[p * kLd + q] = 0.f;
                A[q * kLd + p] = 0.f;
            }
            __syncthreads();
        }
        const int any = rotated;  // every thread reads the flag before thread 0 clears it again
        __syncthreads();
        if (!any) break;
    }
    // eigenvalues in descending order (ties by diagonal index), eigenvectors as columns with their
    // largest-magnitude entry positive
    if (tid < kD) {
        const float li = A[tid * kLd + tid];
        int r = 0;
        for (int j = 0; j < kD; ++j) {
            const float lj = A[j * kLd + j];
            r += (lj > li || (lj == li && j < tid)) ? 1 : 0;
        }
        rank_of[tid] = r;
        lam[(int64_t)h * kD + r] = fmaxf(li, 0.f);
    }
    __syncthreads();
    if (tid < kD) {
        // each column is renormalised (the rotations' rounding moves the norms by a few 1e-5 over a
        // full decomposition) and its largest entry made positive
        int jm = 0;
        float am = fabsf(V[tid]), n2 = V[tid] * V[tid];
        for (int j = 1; j < kD; ++j) {
            const float v = V[j * kLd + tid], a = fabsf(v);
            n2 = fmaf(v, v, n2);
            if (a > am) { am = a; jm = j; }
        }
        inv_norm[tid] = (V[jm * kLd + tid] < 0.f ? -1.f : 1.f) / sqrtf(n2);
    }
    __syncthreads();
    // coalesced output: consecutive threads write consecutive columns k = rank of diagonal index
    float* __restrict__ Uh = U + (int64_t)h * kD * kD;
    for (int e = tid; e < kD * kD; e += kEighThreads) {
        const int j = e >> 7, src = e & (kD - 1);
        Uh[j * kD + rank_of[src]] = inv_norm[src] * V[j * kLd + src];
    }
    if (tid == 0 && sweeps_out) sweeps_out[h] = sweep < kMaxSweeps ? sweep + 1 : -1;
}

// ---------------------------------------------------------------- query variance

__global__ __launch_bounds__(256) void query_variance_kernel(const float* __restrict__ U, const float* __restrict__ Sq,
                                                             int G, float* __restrict__ sig) {
    extern __shared__ float qv_sm[];
    float* Us = qv_sm;             // [128][129]
    float* Ss = qv_sm + kD * kLd;  // [128][129]
    __shared__ float part[2][kD];
    const int h = blockIdx.x, tid = threadIdx.x, i = tid & (kD - 1), half = tid >> 7;
    const float* __restrict__ Uh = U + (int64_t)h * kD * kD;
    for (int e = tid; e < kD * kD; e += 256) Us[(e >> 7) * kLd + (e & (kD - 1))] = Uh[e];
    float acc = 0.f;
    for (int g = 0; g < G; ++g) {
        const float* __restrict__ Sg = Sq + ((int64_t)h * G + g) * kD * kD;
        __syncthreads();
        for (int e = tid; e < kD * kD; e += 256) Ss[(e >> 7) * kLd + (e & (kD - 1))] = Sg[e];
        __syncthreads();
        // rows j of this half: y_j = sum_k S_jk u_ki, acc += u_ji y_j
        for (int j = 64 * half; j < 64 * half + 64; ++j) {
            float y = 0.f;
            for (int k = 0; k < kD; ++k) y = fmaf(Ss[j * kLd + k], Us[k * kLd + i], y);
            acc = fmaf(Us[j * kLd + i], y, acc);
        }
    }
    part[half][i] = acc;
    __syncthreads();
    if (tid < kD) sig[(int64_t)h * kD + tid] = (part[0][tid] + part[1][tid]) / (float)G;
}

// ---------------------------------------------------------------- measured quantization error

// Quantization term of the measured distortion table, one block per (rank on the grid, head): the
// candidate basis P_r (fp16, staged in LDS) projects every calibration token (fp32 accumulation of
// the exact fp16 products, v_dot2_f32_f16), each projected coordinate is quantized at every width
// b = 1..8 with its step, and c_k (z - zhat)^2 accumulates per width; the block's sums over its
// tokens give mean_t sum_k c_k (z_tk - zhat_tk)^2.
constexpr int kMqThreads = 256;
typedef _Float16 mq_h2 __attribute__((ext_vector_type(2)));

__global__ __launch_bounds__(kMqThreads) void measured_quant_kernel(
    const uint16_t* __restrict__ x, int64_t x_head_stride, int n_tok, const uint16_t* __restrict__ P_all,
    int64_t P_head_stride, const float* __restrict__ delta_all, const float* __restrict__ row_w_all,
    int64_t rw_head_stride, int r_min, int r_step, int n_r, float* __restrict__ quant) {
    __shared__ __attribute__((aligned(16))) uint16_t Ps[kD * kD];
    __shared__ float cw[kD];
    __shared__ float red[8][kMqThreads / 64];
    const int ri = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const int r = r_min + ri * r_step;
    // offset of rank r's records: sum of the ranks before it
    const int64_t before = (int64_t)ri * r_min + (int64_t)r_step * ri * (ri - 1) / 2;
    const uint16_t* __restrict__ P = P_all + (int64_t)h * P_head_stride + before * kD;
    const float* __restrict__ c = row_w_all + (int64_t)h * rw_head_stride + before;
    for (int e = tid; e < r * kD / 8; e += kMqThreads)
        reinterpret_cast<uint4*>(Ps)[e] = reinterpret_cast<const uint4*>(P)[e];
    for (int k = tid; k < r; k += kMqThreads) cw[k] = c[k];
    float st[8], inv[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        st[b] = delta_all[((int64_t)h * n_r + ri) * 8 + b];
        inv[b] = 1.f / st[b];
    }
    __syncthreads();
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    const uint16_t* __restrict__ xh = x + (int64_t)h * x_head_stride;
    for (int t = tid; t < n_tok; t += kMqThreads) {
        mq_h2 xv[kD / 2];
#pragma unroll
        for (int q = 0; q < kD / 8; ++q) {
            const uint4 w = reinterpret_cast<const uint4*>(xh + (int64_t)t * kD)[q];
            xv[4 * q] = __builtin_bit_cast(mq_h2, w.x);
            xv[4 * q + 1] = __builtin_bit_cast(mq_h2, w.y);
            xv[4 * q + 2] = __builtin_bit_cast(mq_h2, w.z);
            xv[4 * q + 3] = __builtin_bit_cast(mq_h2, w.w);
        }
        for (int k = 0; k < r; ++k) {
            float z = 0.f;
            const uint4* Pk = reinterpret_cast<const uint4*>(Ps + k * kD);
#pragma unroll
            for (int q = 0; q < kD / 8; ++q) {
                const uint4 w = Pk[q];
                z = __builtin_amdgcn_fdot2(__builtin_bit_cast(mq_h2, w.x), xv[4 * q], z, false);
                z = __builtin_amdgcn_fdot2(__builtin_bit_cast(mq_h2, w.y), xv[4 * q + 1], z, false);
                z = __builtin_amdgcn_fdot2(__builtin_bit_cast(mq_h2, w.z), xv[4 * q + 2], z, false);
                z = __builtin_amdgcn_fdot2(__builtin_bit_cast(mq_h2, w.w), xv[4 * q + 3], z, false);
            }
            const float ck = cw[k];
#pragma unroll
            for (int b = 0; b < 8; ++b) {
                const float hb = (float)(1 << b);  // 2^(b+1-1) for width b + 1
                const float code = fminf(fmaxf(floorf(z * inv[b]) + hb, 0.f), 2.f * hb - 1.f);
                const float e = z - (code - hb + 0.5f) * st[b];
                acc[b] = fmaf(ck * e, e, acc[b]);
            }
        }
    }
#pragma unroll
    for (int b = 0; b < 8; ++b) {
        float v = acc[b];
        for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
        if ((tid & 63) == 0) red[b][tid >> 6] = v;
    }
    __syncthreads();
    if (tid < 8) {
        float v = 0.f;
        for (int w = 0; w < kMqThreads / 64; ++w) v += red[tid][w];
        quant[((int64_t)h * n_r + ri) * 8 + tid] = v / (float)n_tok;
    }
}

int check_launch_calib(const char* what) {
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return set_error(KVC_EDEVICE, "%s: %s", what, hipGetErrorString(e));
    return KVC_OK;
}

int set_big_lds(const void* fn, size_t bytes, const char* what) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return set_error(KVC_EDEVICE, "%s: hipFuncSetAttribute: %s", what, hipGetErrorString(e));
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

using namespace kvc;

extern "C" int kvc_covariance(const uint16_t* x, int64_t x_head_stride, int32_t n_heads, int32_t n_tok,
                              int32_t centered, float* cov, void* stream) {
    clear_error();
    if (n_heads < 0 || n_tok < 1) return set_error(KVC_EINVAL, "kvc_covariance: n_heads < 0 or n_tok < 1");
    if (n_heads == 0) return KVC_OK;
    if (!x || !cov) return set_error(KVC_EINVAL, "kvc_covariance: null pointer");
    if ((reinterpret_cast<uintptr_t>(x) & 15) || (x_head_stride & 7))
        return set_error(KVC_EINVAL, "kvc_covariance: x must be 16-byte aligned and the head stride a multiple of 8");
    if (x_head_stride < (int64_t)n_tok * kD) return set_error(KVC_EINVAL, "kvc_covariance: head stride < n_tok * d");
    if (centered != 0 && centered != 1) return set_error(KVC_EINVAL, "kvc_covariance: centered must be 0 or 1");
    hipLaunchKernelGGL(covariance_kernel, dim3(n_heads), dim3(256), 0, (hipStream_t)stream, x, x_head_stride, n_tok,
                       centered, cov);
    return check_launch_calib("kvc_covariance");
}

extern "C" int kvc_eigh(const float* S, int32_t n, float* lambda, float* U, int32_t* sweeps, void* stream) {
    clear_error();
    if (n < 0) return set_error(KVC_EINVAL, "kvc_eigh: n < 0");
    if (n == 0) return KVC_OK;
    if (!S || !lambda || !U) return set_error(KVC_EINVAL, "kvc_eigh: null pointer");
    const size_t smem = (size_t)2 * kD * kLd * sizeof(float);
    if (int e = set_big_lds((const void*)eigh_kernel, smem, "kvc_eigh")) return e;
    hipLaunchKernelGGL(eigh_kernel, dim3(n), dim3(kEighThreads), smem, (hipStream_t)stream, S, lambda, U, sweeps);
    return check_launch_calib("kvc_eigh");
}

extern "C" int kvc_measured_quant(const uint16_t* x, int64_t x_head_stride, int32_t n_heads, int32_t n_tok,
                                  const uint16_t* P_all, int64_t P_head_stride, const float* delta_all,
                                  const float* row_w_all, int64_t rw_head_stride, int32_t r_min, int32_t r_step,
                                  float* quant, void* stream) {
    clear_error();
    if (n_heads < 0 || n_tok < 1) return set_error(KVC_EINVAL, "kvc_measured_quant: n_heads < 0 or n_tok < 1");
    if (n_heads == 0) return KVC_OK;
    if (!x || !P_all || !delta_all || !row_w_all || !quant) return set_error(KVC_EINVAL, "kvc_measured_quant: null pointer");
    if (r_min < 2 || r_step < 2 || (r_min & 1) || (r_step & 1) || r_min > kD)
        return set_error(KVC_EUNSUPPORTED, "kvc_measured_quant: rank grid (%d, %d) must be even, r_min <= d", r_min, r_step);
    const int n_r = (kD - r_min) / r_step + 1;
    const int64_t sum_r = (int64_t)n_r * r_min + (int64_t)r_step * n_r * (n_r - 1) / 2;
    if ((reinterpret_cast<uintptr_t>(x) & 15) || (x_head_stride & 7) || x_head_stride < (int64_t)n_tok * kD)
        return set_error(KVC_EINVAL, "kvc_measured_quant: x must be 16-byte aligned, head stride a multiple of 8 and >= n_tok * d");
    if ((reinterpret_cast<uintptr_t>(P_all) & 15) || (P_head_stride & 7) || P_head_stride < sum_r * kD)
        return set_error(KVC_EINVAL, "kvc_measured_quant: P_all must be 16-byte aligned, its head stride a multiple of 8 "
                                     "and >= the candidate bases of one head");
    if (rw_head_stride < sum_r) return set_error(KVC_EINVAL, "kvc_measured_quant: row-weight head stride too small");
    hipLaunchKernelGGL(measured_quant_kernel, dim3(n_r, n_heads), dim3(kMqThreads), 0, (hipStream_t)stream, x,
                       x_head_stride, n_tok, P_all, P_head_stride, delta_all, row_w_all, rw_head_stride, r_min, r_step,
                       n_r, quant);
    return check_launch_calib("kvc_measured_quant");
}

extern "C" int kvc_query_variance(const float* U, const float* S_q, int32_t n_heads, int32_t G, float* sigma2_q,
                                  void* stream) {
    clear_error();
    if (n_heads < 0 || G < 1) return set_error(KVC_EINVAL, "kvc_query_variance: n_heads < 0 or G < 1");
    if (n_heads == 0) return KVC_OK;
    if (!U || !S_q || !sigma2_q) return set_error(KVC_EINVAL, "kvc_query_variance: null pointer");
    const size_t smem = (size_t)2 * kD * kLd * sizeof(float);
    if (int e = set_big_lds((const void*)query_variance_kernel, smem, "kvc_query_variance")) return e;
    hipLaunchKernelGGL(query_variance_kernel, dim3(n_heads), dim3(256), smem, (hipStream_t)stream, U, S_q, G, sigma2_q);
    return check_launch_calib("kvc_query_variance");
}
