/*
 * KV-COBRA oracle, exact integer part: per-token encode and the packed layout.
 *
 * Test infrastructure only. Nothing in the product path may link or load
 * this file; it shares no code with the GPU library.
 *
 * Passages followed: calibration/inference table, steps 7-8 (a token's code is
 * quantize(P x) with the Hadamard rotation folded into P; codes are cached and
 * dequantized on read); Section 3.4 (one uniform b-bit quantizer per head).
 *
 * Definition computed (readings stated in oracle/quant.py and oracle/layout.py):
 *   y_i = sum_j P_ij x_j, exactly (P and x are fp16, so every product is an
 *         integer multiple of 2^-48 and the sum fits a 128-bit integer);
 *   k_i = clamp(floor(y_i / step) + 2^(b-1), 0, 2^b - 1), exactly.
 * The packed layout is the one documented in oracle/layout.py.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -fPIC -shared (no fast-math).
 */
#include <stdint.h>
#include <string.h>

typedef __int128 i128;

/* fp16 bits -> signed integer mantissa and power-of-two exponent. Returns -1 for inf/nan. */
static int half_parts(uint16_t h, int64_t *m, int *e) {
    int s = h >> 15, ex = (h >> 10) & 31, fr = h & 1023;
    if (ex == 31) return -1;
    if (ex == 0) { *m = fr; *e = -24; }
    else { *m = 1024 + fr; *e = ex - 25; }
    if (s) *m = -*m;
    return 0;
}

/* step as an exact integer multiple of 2^-48; returns -1 if out of the supported range. */
static int step_units(float step, i128 *D) {
    uint32_t u;
    memcpy(&u, &step, 4);
    int ex = (u >> 23) & 255;
    if ((u >> 31) || ex == 0 || ex == 255) return -1;  /* positive normal only */
    int64_t m = 0x800000 | (u & 0x7fffff);
    int e = ex - 150;           /* step = m * 2^e */
    int s = e + 48;
    if (s < 0 || s > 60) return -1;
    *D = ((i128)m) << s;
    return 0;
}

/* Exact codes: codes[t*r + i] for tokens t < n. Returns 0, or -1 on a non-finite input / bad step. */
int oracle_encode_codes(const uint16_t *P, int r, int d, float step, int b,
                        const uint16_t *x, int n, uint8_t *codes) {
    i128 D;
    if (step_units(step, &D)) return -1;
    const int64_t h = (int64_t)1 << (b - 1);
    const int64_t kmax = ((int64_t)1 << b) - 1;
    int bad = 0;
    /* tokens are independent: spread over threads (no effect on any value) */
#pragma omp parallel for schedule(static) reduction(|: bad)
    for (int t = 0; t < n; ++t) {
        const uint16_t *xt = x + (int64_t)t * d;
        for (int i = 0; i < r; ++i) {
            const uint16_t *Pi = P + (int64_t)i * d;
            i128 N = 0;
            for (int j = 0; j < d; ++j) {
                int64_t mp, mx; int ep, exx;
                if (half_parts(Pi[j], &mp, &ep) || half_parts(xt[j], &mx, &exx)) { bad = 1; mp = mx = 0; ep = exx = -24; }
                int s = ep + exx + 48;              /* 0 .. 58 */
                N += (i128)(mp * mx) * ((i128)1 << s);  /* exact, no overflow */
            }
            i128 q = N / D;
            if ((N % D) != 0 && N < 0) q -= 1;      /* floor division (D > 0) */
            i128 k = q + h;
            if (k < 0) k = 0;
            if (k > kmax) k = kmax;
            codes[(int64_t)t * r + i] = (uint8_t)k;
        }
    }
    return bad ? -1 : 0;
}

static int n_planes(int b, int *w) {
    if (b == 8) { w[0] = 8; return 1; }
    int n = 0;
    if (b & 4) w[n++] = 4;
    if (b & 2) w[n++] = 2;
    if (b & 1) w[n++] = 1;
    return n;
}

/* Position inside a run of 16 slots of the m-th item (V side token order; see oracle/layout.py). */
static int pos_b(int b, int m) {
    if (b == 8) return m;
    if (b == 4) return 8 * (m / 8) + 2 * (m % 4) + (m / 4) % 2;
    return 4 * (m % 4) + m / 4;
}

static int slot_k(int t, int i, int r) {
    int g16 = r / 16, rho = r % 16;
    if (i < 16 * g16) return (i / 16) * 1024 + t * 16 + i % 16;
    return 1024 * g16 + t * rho + (i - 16 * g16);
}

/* Byte offset of every V field (n, c, q) inside a plane of width p, by enumeration in the layout's
 * order: group n / g (g = 8 / p, 1 for p = 8), then L = 4 c + q, then n; fields of coordinates >= r
 * are absent. off[64 n + 4 c + q]. */
static void v_field_table(int r, int p, int *off) {
    int g = p == 8 ? 1 : 8 / p, nvt = (r + 15) / 16, k = 0;
    for (int n0 = 0; n0 < nvt; n0 += g)
        for (int L = 0; L < 64; ++L)
            for (int n = n0; n < n0 + g && n < nvt; ++n)
                if (16 * n + L / 4 < r) off[64 * n + L] = 2 * p * k++;
}

/* Bit of the code of (token t in tile, coordinate i) inside its plane of width p (vtab: the plane's
 * v_field_table on the V side). */
static int64_t plane_bit(int side, int t, int i, int r, int b, int p, const int *vtab) {
    if (side == 0) return (int64_t)p * slot_k(t, i, r);
    return 8LL * vtab[64 * (i / 16) + 4 * (i % 16) + t / 16] + (int64_t)p * pos_b(b, t % 16);
}

/* codes[t*r+i] (t < n) -> stream of ceil(n/64) tiles (zero-filled by this function). */
void oracle_pack(const uint8_t *codes, int n, int r, int b, int side, uint8_t *out) {
    int w[3];
    int np = n_planes(b, w);
    int n_tiles = (n + 63) / 64;
    int64_t tb = 8LL * r * b;
    int vtab[512];
    memset(out, 0, (size_t)(n_tiles * tb));
    for (int tile = 0; tile < n_tiles; ++tile) {
        uint8_t *base = out + tile * tb;
        int64_t plane_off = 0;
        for (int k = 0; k < np; ++k) {
            int p = w[k];
            int sh = 0;
            for (int k2 = k + 1; k2 < np; ++k2) sh += w[k2];
            if (side != 0) v_field_table(r, p, vtab);
            for (int t = 0; t < 64; ++t) {
                int tok = tile * 64 + t;
                if (tok >= n) continue;
                for (int i = 0; i < r; ++i) {
                    uint32_t v = (codes[(int64_t)tok * r + i] >> sh) & ((1u << p) - 1);
                    int64_t bitpos = plane_bit(side, t, i, r, b, p, vtab);
                    base[plane_off + bitpos / 8] |= (uint8_t)(v << (bitpos % 8));
                }
            }
            plane_off += 8LL * r * p;
        }
    }
}

/* stream -> codes[t*r+i] for tokens t < n. */
void oracle_unpack(const uint8_t *stream, int n, int r, int b, int side, uint8_t *codes) {
    int w[3];
    int np = n_planes(b, w);
    int64_t tb = 8LL * r * b;
    int vtab[3][512];
    if (side != 0)
        for (int k = 0; k < np; ++k) v_field_table(r, w[k], vtab[k]);
    for (int tok = 0; tok < n; ++tok) {
        int tile = tok / 64, t = tok % 64;
        const uint8_t *base = stream + tile * tb;
        for (int i = 0; i < r; ++i) {
            uint32_t c = 0;
            int64_t plane_off = 0;
            for (int k = 0; k < np; ++k) {
                int p = w[k];
                int sh = 0;
                for (int k2 = k + 1; k2 < np; ++k2) sh += w[k2];
                int64_t bitpos = plane_bit(side, t, i, r, b, p, vtab[k]);
                c |= ((uint32_t)(base[plane_off + bitpos / 8] >> (bitpos % 8)) & ((1u << p) - 1)) << sh;
                plane_off += 8LL * r * p;
            }
            codes[(int64_t)tok * r + i] = (uint8_t)c;
        }
    }
}

/*
 * Calibration, table step 1: eigendecomposition of a symmetric d x d matrix S
 * (row-major, fp64) by the cyclic-by-row Jacobi method (Golub and Van Loan,
 * Matrix Computations, Sec. 8.5: the symmetric Schur decomposition of each
 * 2 x 2 pivot block annihilates a_pq; A <- J^T A J, V <- V J).
 * A rotation is skipped when |a_pq| <= 2^-60 sqrt(|a_pp a_qq|) (or a_pq = 0);
 * the iteration ends after a sweep with no rotation, or after 60 sweeps.
 * Outputs, in the calibration reading of the oracle: eigenvalues in descending
 * order (ties keep the diagonal index order), negative ones clamped to 0;
 * U[j*d + k] = component j of eigenvector k; each eigenvector's entry of
 * largest magnitude (the first such) made positive.
 * Returns the number of sweeps, or -1 if it did not converge.
 */
#include <math.h>
#include <stdlib.h>

static int jacobi_one(const double *S, int d, double *lam, double *U, double *A, double *V, int *idx) {
    for (int i = 0; i < d * d; ++i) A[i] = S[i];
    for (int i = 0; i < d; ++i)
        for (int j = 0; j < d; ++j) V[i * d + j] = (i == j) ? 1.0 : 0.0;
    int sweeps = 0, converged = 0;
    while (sweeps < 60) {
        int rotated = 0;
        for (int p = 0; p < d - 1; ++p) {
            for (int q = p + 1; q < d; ++q) {
                const double apq = A[p * d + q];
                if (apq == 0.0 || fabs(apq) <= ldexp(sqrt(fabs(A[p * d + p]) * fabs(A[q * d + q])), -60)) continue;
                rotated = 1;
                const double theta = (A[q * d + q] - A[p * d + p]) / (2.0 * apq);
                const double t = (theta >= 0.0 ? 1.0 : -1.0) / (fabs(theta) + sqrt(1.0 + theta * theta));
                const double c = 1.0 / sqrt(1.0 + t * t);
                const double s = t * c;
                for (int k = 0; k < d; ++k) {  /* columns p, q: A <- A J */
                    const double akp = A[k * d + p], akq = A[k * d + q];
                    A[k * d + p] = c * akp - s * akq;
                    A[k * d + q] = s * akp + c * akq;
                }
                for (int k = 0; k < d; ++k) {  /* rows p, q: A <- J^T A */
                    const double apk = A[p * d + k], aqk = A[q * d + k];
                    A[p * d + k] = c * apk - s * aqk;
                    A[q * d + k] = s * apk + c * aqk;
                }
                A[p * d + q] = A[q * d + p] = 0.0;
                for (int k = 0; k < d; ++k) {  /* V <- V J */
                    const double vkp = V[k * d + p], vkq = V[k * d + q];
                    V[k * d + p] = c * vkp - s * vkq;
                    V[k * d + q] = s * vkp + c * vkq;
                }
            }
        }
        ++sweeps;
        if (!rotated) { converged = 1; break; }
    }
    /* descending order, stable (insertion sort on the diagonal index) */
    for (int i = 0; i < d; ++i) idx[i] = i;
    for (int i = 1; i < d; ++i) {
        const int v = idx[i];
        int j = i - 1;
        while (j >= 0 && A[idx[j] * d + idx[j]] < A[v * d + v]) { idx[j + 1] = idx[j]; --j; }
        idx[j + 1] = v;
    }
    for (int k = 0; k < d; ++k) {
        const int src = idx[k];
        const double l = A[src * d + src];
        lam[k] = l > 0.0 ? l : 0.0;
        int jm = 0;
        for (int j = 1; j < d; ++j)
            if (fabs(V[j * d + src]) > fabs(V[jm * d + src])) jm = j;
        const double sg = V[jm * d + src] < 0.0 ? -1.0 : 1.0;
        for (int j = 0; j < d; ++j) U[j * d + k] = sg * V[j * d + src];
    }
    return converged ? sweeps : -1;
}

/* n matrices S[n][d][d] -> lam[n][d], U[n][d][d]; sweeps[n] as jacobi_one returns. Matrices are
 * independent: spread over threads. Returns 0, or -1 if any did not converge. */
int oracle_jacobi_eigh(const double *S, int n, int d, double *lam, double *U, int *sweeps) {
    int bad = 0;
#pragma omp parallel for schedule(dynamic) reduction(|: bad)
    for (int h = 0; h < n; ++h) {
        double *A = (double *)malloc(sizeof(double) * d * d);
        double *V = (double *)malloc(sizeof(double) * d * d);
        int *idx = (int *)malloc(sizeof(int) * d);
        const int s = jacobi_one(S + (int64_t)h * d * d, d, lam + (int64_t)h * d, U + (int64_t)h * d * d, A, V, idx);
        sweeps[h] = s;
        if (s < 0) bad = 1;
        free(A); free(V); free(idx);
    }
    return bad ? -1 : 0;
}
