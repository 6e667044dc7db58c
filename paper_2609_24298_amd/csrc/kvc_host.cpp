// Host half of libkvc: the (r, b) allocator, the fused-basis builder,
// descriptor validation and the error state. Pure C++17, no HIP.
//
// Built with -ffp-contract=off and without fast-math: the allocator's fp64
// evaluation order is part of its definition (every sum is left to right in
// the order stated below), so its tables are reproducible bit for bit.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <limits>
#include <string>
#include <vector>

#include "kvc_internal.h"

namespace kvc {

static thread_local std::string g_error;

int set_error(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_error = buf;
    return code;
}

void clear_error() { g_error.clear(); }

int validate_desc(const kvc_stream_desc* s, const char* name) {
    if (!s) return set_error(KVC_EINVAL, "%s: null descriptor", name);
    if (s->d != KVC_HEAD_DIM) return set_error(KVC_EUNSUPPORTED, "%s: d = %d, only 128 is supported", name, s->d);
    if (s->n_units < 0 || s->capacity < 0) return set_error(KVC_EINVAL, "%s: negative n_units or capacity", name);
    if (s->side != KVC_SIDE_K && s->side != KVC_SIDE_V) return set_error(KVC_EINVAL, "%s: side must be K or V", name);
    if (s->n_units == 0) return KVC_OK;
    if (!s->r_host || !s->b_host || !s->code_off_host || !s->basis_off_host || !s->delta_host || !s->r || !s->b || !s->code_off ||
        !s->basis_off || !s->delta || !s->codes || !s->basis)
        return set_error(KVC_EINVAL, "%s: null table or arena pointer", name);
    if ((reinterpret_cast<uintptr_t>(s->codes) & 15) != 0)
        return set_error(KVC_EINVAL, "%s: code arena must be 16-byte aligned", name);
    for (int u = 0; u < s->n_units; ++u) {
        const int r = s->r_host[u], b = s->b_host[u];
        if (r < 2 || r > s->d || (r & 1)) return set_error(KVC_EUNSUPPORTED, "%s: unit %d has r = %d (even, 2..d)", name, u, r);
        if (b < 1 || b > 8) return set_error(KVC_EUNSUPPORTED, "%s: unit %d has b = %d (1..8)", name, u, b);
        const int64_t off = s->code_off_host[u];
        if (off < 0 || (off & 15)) return set_error(KVC_EINVAL, "%s: unit %d code_off %lld not a multiple of 16", name, u, (long long)off);
        if (off + stream_bytes(s->capacity, r, b) > s->codes_bytes)
            return set_error(KVC_ENOSPACE, "%s: unit %d stream exceeds the code arena", name, u);
        const int64_t boff = s->basis_off_host[u];
        if (boff < 0 || boff + (int64_t)r * s->d > s->basis_elems)
            return set_error(KVC_ENOSPACE, "%s: unit %d basis exceeds the basis arena", name, u);
        const float st = s->delta_host[u];
        if (!(st >= std::ldexp(1.0f, -24) && st <= std::ldexp(1.0f, 24)))
            return set_error(KVC_EUNSUPPORTED, "%s: unit %d step %g outside [2^-24, 2^24]", name, u, (double)st);
    }
    return KVC_OK;
}

// ------------------------------------------------------------------ allocator

namespace {

// q(b) = 2^(-2b) / 12, Eq. (eq:q).
inline double q_of_b(int b) { return std::ldexp(1.0, -2 * b) / 12.0; }

// One head's weights in importance order with its head and tail sums:
// S[k] = w_0 + ... + w_{k-1} (left to right), T[k] = w_{d-1} + ... + w_k
// (accumulated from the end). D(r, b) = T[r] + q(b) * S[r].
struct Head {
    std::vector<double> S, T;
    double dist(int r, int b) const { return T[r] + q_of_b(b) * S[r]; }
};

struct C1Result {
    int r, b;
    double D;
};

// C1 (Section 3.2): r = r_min, r_min + r_step, ... <= min(d, floor(B / b_min)),
// b = min(b_max, floor(B / r)), argmin D with ties kept at the smallest r.
C1Result c1(const Head& h, double B, const kvc_alloc_opts& o) {
    const int d = o.d;
    const double rb = std::floor(B / (double)o.b_min);
    const int r_hi = rb < (double)d ? (int)rb : d;
    C1Result best{-1, -1, 0.0};
    for (int r = o.r_min; r <= r_hi; r += o.r_step) {
        const double fb = std::floor(B / (double)r);
        const int b = fb < (double)o.b_max ? (int)fb : o.b_max;
        const double D = h.dist(r, b);
        if (best.r < 0 || D < best.D) best = {r, b, D};
    }
    if (best.r < 0) best = {o.r_min, o.b_min, h.dist(o.r_min, o.b_min)};
    return best;
}

// Exact DP (Appendix D) over integer budgets beta_h in [ceil(B_min), floor(B_max)], sum <= floor(B_tot),
// for a per-head optimum opt(h, beta) that is non-increasing in beta. The running table is
// non-increasing in the total, so only the budgets where D*_h drops (plus the lowest one) can be the
// smallest minimiser: scanning those in ascending order with a strict comparison picks the same beta_h
// as scanning all.
template <class Opt>
int dp_solve(int N, const kvc_alloc_opts& o, double B_tot, Opt opt, kvc_head_alloc* out, const char* fn) {
    const int64_t lo = (int64_t)std::ceil(o.B_min), hi = (int64_t)std::floor(o.B_max);
    const int64_t cap = (int64_t)std::floor(B_tot);
    if (lo < 0 || hi < lo) return set_error(KVC_EINVAL, "%s: empty DP budget range", fn);
    if (cap > (int64_t)1 << 26) return set_error(KVC_EINVAL, "%s: DP budget too large", fn);
    if ((int64_t)N * lo > cap) return set_error(KVC_EINVAL, "%s: B_tot below n_heads * B_min", fn);
    const double INF = std::numeric_limits<double>::infinity();
    std::vector<std::vector<int32_t>> bp_beta(N);
    std::vector<std::vector<double>> bp_D(N);
    for (int h = 0; h < N; ++h) {
        double prevD = 0.0;
        for (int64_t beta = lo; beta <= hi; ++beta) {
            const double D = opt(h, (double)beta).D;
            if (beta == lo || D < prevD) {
                bp_beta[h].push_back((int32_t)beta);
                bp_D[h].push_back(D);
            }
            prevD = D;
        }
    }
    std::vector<double> prev(cap + 1, 0.0), cur(cap + 1);
    std::vector<int32_t> choice((size_t)N * (cap + 1));
    for (int h = 0; h < N; ++h) {
        const int32_t* bb = bp_beta[h].data();
        const double* bd = bp_D[h].data();
        const int nb = (int)bp_beta[h].size();
        int32_t* ch = choice.data() + (size_t)h * (cap + 1);
        for (int64_t tot = 0; tot <= cap; ++tot) {
            double best = INF;
            int32_t arg = -1;
            for (int k = 0; k < nb && bb[k] <= tot; ++k) {
                const double base = prev[tot - bb[k]];
                if (base == INF) continue;
                const double v = base + bd[k];
                if (v < best) { best = v; arg = bb[k]; }
            }
            cur[tot] = best;
            ch[tot] = arg;
        }
        std::swap(prev, cur);
    }
    if (prev[cap] == INF) return set_error(KVC_EINVAL, "%s: DP found no feasible allocation", fn);
    int64_t tot = cap;
    for (int h = N - 1; h >= 0; --h) {
        const int32_t beta = choice[(size_t)h * (cap + 1) + tot];
        C1Result a = opt(h, (double)beta);
        out[h] = {a.r, a.b, (double)beta, a.D};
        tot -= beta;
    }
    return KVC_OK;
}

// Per-head optimum over a table D[ri][bi] (r = r_min + ri r_step, b = b_min + bi): the smallest D
// over every grid pair with r b <= B, ties at the smallest r, then the smallest b; below the smallest
// pair, (r_min, b_min).
C1Result c1_table(const double* D, int n_r, int n_b, double B, const kvc_alloc_opts& o) {
    C1Result best{-1, -1, 0.0};
    for (int ri = 0; ri < n_r; ++ri) {
        const int r = o.r_min + ri * o.r_step;
        for (int bi = 0; bi < n_b; ++bi) {
            const int b = o.b_min + bi;
            if ((double)r * b <= B && (best.r < 0 || D[ri * n_b + bi] < best.D)) best = {r, b, D[ri * n_b + bi]};
        }
    }
    if (best.r < 0) best = {o.r_min, o.b_min, D[0]};
    return best;
}

int check_opts(const kvc_alloc_opts* o) {
    if (!o) return set_error(KVC_EINVAL, "kvc_allocate: null options");
    if (o->d < 2 || o->d > 4096) return set_error(KVC_EINVAL, "kvc_allocate: d = %d", o->d);
    if (o->r_min < 1 || o->r_step < 1 || o->r_min > o->d)
        return set_error(KVC_EINVAL, "kvc_allocate: bad rank grid (r_min %d, r_step %d)", o->r_min, o->r_step);
    if (o->b_min < 1 || o->b_max > 8 || o->b_min > o->b_max)
        return set_error(KVC_EINVAL, "kvc_allocate: bad bit range [%d, %d]", o->b_min, o->b_max);
    if (!(o->bpd > 0.0) || !std::isfinite(o->bpd)) return set_error(KVC_EINVAL, "kvc_allocate: bpd must be > 0");
    if (o->solver < KVC_SOLVER_DAMPED || o->solver > KVC_SOLVER_C1_ONLY)
        return set_error(KVC_EINVAL, "kvc_allocate: unknown solver %d", o->solver);
    if (o->rounds < 0 || !std::isfinite(o->eta) || !std::isfinite(o->B_min) || !std::isfinite(o->B_max))
        return set_error(KVC_EINVAL, "kvc_allocate: bad rounds / eta / budget bounds");
    if (o->B_min > o->B_max) return set_error(KVC_EINVAL, "kvc_allocate: B_min > B_max");
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

using namespace kvc;

extern "C" int kvc_alloc_opts_default(kvc_alloc_opts* o, double bpd) {
    if (!o) return set_error(KVC_EINVAL, "kvc_alloc_opts_default: null");
    o->d = KVC_HEAD_DIM;
    o->r_min = 2;
    o->r_step = 2;
    o->b_min = 1;
    o->b_max = 8;
    o->solver = KVC_SOLVER_DAMPED;
    o->rounds = 5;
    o->reorder = 1;
    o->bpd = bpd;
    o->eta = 0.3;
    o->B_min = (double)(o->r_min * o->b_min);
    o->B_max = (double)(o->d * o->b_max);
    return KVC_OK;
}

extern "C" int kvc_allocate(const double* lambda, const double* sigma2_q, int32_t n_heads,
                            const kvc_alloc_opts* opts, kvc_head_alloc* out, int32_t* order_out) {
    clear_error();
    if (int e = check_opts(opts)) return e;
    const kvc_alloc_opts& o = *opts;
    if (n_heads <= 0 || !lambda || !out) return set_error(KVC_EINVAL, "kvc_allocate: null input or n_heads <= 0");
    const int N = n_heads, d = o.d;

    // Weights (Proposition prop:kl-bound) and importance order (table step 2).
    std::vector<Head> heads(N);
    std::vector<int32_t> idx(d);
    std::vector<double> w(d);
    for (int h = 0; h < N; ++h) {
        for (int i = 0; i < d; ++i) {
            const double l = lambda[(int64_t)h * d + i];
            w[i] = sigma2_q ? sigma2_q[(int64_t)h * d + i] * l : l;
            if (!std::isfinite(w[i])) return set_error(KVC_EINVAL, "kvc_allocate: non-finite weight (head %d)", h);
            idx[i] = i;
        }
        if (o.reorder) std::stable_sort(idx.begin(), idx.end(), [&](int a, int b) { return w[a] > w[b]; });
        if (order_out) std::copy(idx.begin(), idx.end(), order_out + (int64_t)h * d);
        Head& H = heads[h];
        H.S.assign(d + 1, 0.0);
        H.T.assign(d + 1, 0.0);
        for (int k = 0; k < d; ++k) H.S[k + 1] = H.S[k] + w[idx[k]];
        for (int k = d - 1; k >= 0; --k) H.T[k] = H.T[k + 1] + w[idx[k]];
    }

    const double bmin = o.B_min;
    if (o.solver == KVC_SOLVER_C1_ONLY) {
        const double B = o.bpd * (double)d;
        for (int h = 0; h < N; ++h) {
            C1Result a = c1(heads[h], B, o);
            out[h] = {a.r, a.b, B, a.D};
        }
        return KVC_OK;
    }

    const double B_tot = o.bpd * (double)((int64_t)N * d);
    if (o.solver == KVC_SOLVER_DAMPED) {
        // Table steps 3-4 and Eq. (eq:c2-update): damped proportional update,
        // clamp at B_min, renormalise to B_tot; a final C1 emits the table.
        const double B_bar = B_tot / N;
        const double step = o.eta * B_bar;
        std::vector<double> B(N, o.bpd * (double)d), Bp(N), D(N);
        for (int round = 0; round < o.rounds; ++round) {
            double D_sum = 0.0;
            for (int h = 0; h < N; ++h) {
                D[h] = c1(heads[h], B[h], o).D;
                D_sum = D_sum + D[h];
            }
            const double D_bar = D_sum / N;
            if (!(D_bar > 0.0)) break;
            double S = 0.0;
            for (int h = 0; h < N; ++h) {
                Bp[h] = std::max(bmin, B[h] + step * (std::sqrt(D[h] / D_bar) - 1.0));
                S = S + Bp[h];
            }
            const double f = B_tot / S;
            for (int h = 0; h < N; ++h) B[h] = Bp[h] * f;
        }
        for (int h = 0; h < N; ++h) {
            C1Result a = c1(heads[h], B[h], o);
            out[h] = {a.r, a.b, B[h], a.D};
        }
        return KVC_OK;
    }

    // Exact DP (Appendix D).
    return dp_solve(N, o, B_tot, [&](int h, double beta) { return c1(heads[h], beta, o); }, out, "kvc_allocate");
}

extern "C" int kvc_allocate_measured(const double* quant, const double* trunc_w, const int32_t* order,
                                     int32_t n_heads, const kvc_alloc_opts* opts, kvc_head_alloc* out) {
    clear_error();
    if (int e = check_opts(opts)) return e;
    const kvc_alloc_opts& o = *opts;
    if (n_heads <= 0 || !quant || !trunc_w || !order || !out)
        return set_error(KVC_EINVAL, "kvc_allocate_measured: null input or n_heads <= 0");
    const int N = n_heads, d = o.d;
    const int n_r = (d - o.r_min) / o.r_step + 1, n_b = o.b_max - o.b_min + 1;
    // D[h][ri][bi] = T[r] + quant[h][ri][bi], T[r] the measured truncation term summed from the last
    // importance position down
    std::vector<double> D((size_t)N * n_r * n_b);
    std::vector<double> T(d + 1);
    for (int h = 0; h < N; ++h) {
        T[d] = 0.0;
        for (int p = d - 1; p >= 0; --p) {
            const int i = order[(int64_t)h * d + p];
            if (i < 0 || i >= d) return set_error(KVC_EINVAL, "kvc_allocate_measured: order out of range (head %d)", h);
            T[p] = T[p + 1] + trunc_w[(int64_t)h * d + i];
        }
        for (int ri = 0; ri < n_r; ++ri)
            for (int bi = 0; bi < n_b; ++bi) {
                const double q = quant[((int64_t)h * n_r + ri) * n_b + bi];
                const double v = T[o.r_min + ri * o.r_step] + q;
                if (!std::isfinite(v)) return set_error(KVC_EINVAL, "kvc_allocate_measured: non-finite table (head %d)", h);
                D[((size_t)h * n_r + ri) * n_b + bi] = v;
            }
    }
    const double B_tot = o.bpd * (double)((int64_t)N * d);
    return dp_solve(N, o, B_tot,
                    [&](int h, double beta) { return c1_table(D.data() + (size_t)h * n_r * n_b, n_r, n_b, beta, o); },
                    out, "kvc_allocate_measured");
}

// ------------------------------------------------------------------ basis

namespace {

// MSE-optimal step of the 2^b-level uniform mid-rise quantizer for a unit
// Gaussian (exact Gaussian MSE minimised over the step), to four significant
// digits; b = 1..5 are the classical values of J. Max (1960).
const double kStep[9] = {0.0, 1.596, 0.9957, 0.5860, 0.3352, 0.1881, 0.1041, 0.05687, 0.03076};

// Round to nearest even fp16, returned as raw bits.
uint16_t to_half_bits(double x) {
    const uint16_t sign = std::signbit(x) ? 0x8000 : 0;
    const double a = std::fabs(x);
    if (std::isnan(x)) return 0x7e00;
    if (a >= 65520.0) return sign | 0x7c00;  // halfway to 2^16 and beyond round to infinity
    int e;
    std::frexp(a, &e);                        // a = m 2^e, m in [0.5, 1)
    int E = e - 1;                            // a = 1.f 2^E
    const int qexp = (E < -14 ? -14 : E) - 10;
    double n = std::nearbyint(std::ldexp(a, -qexp));  // exact scaling, ties to even
    if (a == 0.0) return sign;
    if (E < -14) return sign | (uint16_t)n;   // subnormal (n == 1024 encodes the smallest normal)
    if (n == 2048.0) { n = 1024.0; ++E; }
    if (E > 15) return sign | 0x7c00;
    return sign | (uint16_t)(((E + 15) << 10) | ((int)n - 1024));
}

// Binary expansion of r, largest power first.
std::vector<int> block_sizes(int r) {
    std::vector<int> s;
    for (int bit = 1 << 30; bit; bit >>= 1)
        if (r & bit) s.push_back(bit);
    return s;
}

}  // namespace

namespace kvc {
namespace {

// Importance positions 0..r-1 dealt to the Hadamard blocks (binary expansion of r, largest first): position
// i goes to the block with the largest remaining quota (i + 1) n_j - r count_j, ties to the larger block.
std::vector<std::vector<int>> deal_blocks(int r, const std::vector<int>& sizes) {
    const int nblk = (int)sizes.size();
    std::vector<std::vector<int>> members(nblk);
    std::vector<int> count(nblk, 0);
    for (int i = 0; i < r; ++i) {
        int best = -1;
        int64_t best_v = 0;
        for (int j = 0; j < nblk; ++j) {
            if (count[j] >= sizes[j]) continue;
            const int64_t v = (int64_t)(i + 1) * sizes[j] - (int64_t)r * count[j];
            if (best < 0 || v > best_v) { best = j; best_v = v; }
        }
        members[best].push_back(i);
        ++count[best];
    }
    return members;
}

int check_basis_args(const char* fn, const double* U, const int32_t* order, const double* lambda, int32_t d, int32_t r,
                     const int8_t* sign) {
    if (!U || !order || !lambda || !sign) return set_error(KVC_EINVAL, "%s: null pointer", fn);
    if (d < 2 || r < 2 || r > d || (r & 1)) return set_error(KVC_EUNSUPPORTED, "%s: r = %d, d = %d", fn, r, d);
    for (int i = 0; i < r; ++i) {
        if (order[i] < 0 || order[i] >= d) return set_error(KVC_EINVAL, "%s: order[%d] = %d", fn, i, order[i]);
        if (sign[i] != 1 && sign[i] != -1) return set_error(KVC_EINVAL, "%s: sign[%d] not +-1", fn, i);
    }
    return KVC_OK;
}

// P rows of block j: (1/sqrt(n)) sum_c H_n[a][c] sign[i_c] u_{order[i_c]}, c ascending, rounded to fp16.
void build_basis(const double* U, const int32_t* order, int32_t d, int32_t r, const int8_t* sign,
                 const std::vector<int>& sizes, const std::vector<std::vector<int>>& members, uint16_t* P) {
    int row0 = 0;
    for (size_t j = 0; j < sizes.size(); ++j) {
        const int n = sizes[j];
        const double inv = 1.0 / std::sqrt((double)n);
        for (int a = 0; a < n; ++a) {
            for (int col = 0; col < d; ++col) {
                double acc = 0.0;
                for (int c = 0; c < n; ++c) {
                    const int i = members[j][c];
                    const double hv = (__builtin_popcount((unsigned)(a & c)) & 1) ? -1.0 : 1.0;
                    acc = acc + hv * ((double)sign[i] * U[(int64_t)col * d + order[i]]);
                }
                P[(int64_t)(row0 + a) * d + col] = to_half_bits(acc * inv);
            }
        }
        row0 += n;
    }
}

// Step: sqrt of the mean retained variance times delta_b (Appendix A.1).
int step_of(const double* lambda, const int32_t* order, int32_t r, int32_t b, float* delta, const char* fn) {
    double s = 0.0;
    for (int i = 0; i < r; ++i) s = s + lambda[order[i]];
    const double sigma2 = s / r;
    const float st = (float)(std::sqrt(sigma2) * kStep[b]);
    if (!(st >= std::ldexp(1.0f, -24) && st <= std::ldexp(1.0f, 24)))
        return set_error(KVC_EUNSUPPORTED, "%s: step %g outside [2^-24, 2^24]", fn, (double)st);
    *delta = st;
    return KVC_OK;
}

}  // namespace
}  // namespace kvc

extern "C" int kvc_make_basis(const double* U, const int32_t* order, const double* lambda, int32_t d,
                              int32_t r, int32_t b, const int8_t* sign, uint16_t* P, float* delta) {
    clear_error();
    if (!P || !delta) return set_error(KVC_EINVAL, "kvc_make_basis: null pointer");
    if (int e = check_basis_args("kvc_make_basis", U, order, lambda, d, r, sign)) return e;
    if (b < 1 || b > 8) return set_error(KVC_EUNSUPPORTED, "kvc_make_basis: b = %d", b);
    const std::vector<int> sizes = block_sizes(r);
    build_basis(U, order, d, r, sign, sizes, deal_blocks(r, sizes), P);
    return step_of(lambda, order, r, b, delta, "kvc_make_basis");
}

extern "C" int kvc_make_candidates(const double* U, const int32_t* order, const double* lambda, const double* wt,
                                   int32_t d, const int8_t* sign, int32_t r_min, int32_t r_step, uint16_t* P_all,
                                   float* delta_all, float* row_w_all) {
    clear_error();
    if (!wt || !P_all || !delta_all || !row_w_all) return set_error(KVC_EINVAL, "kvc_make_candidates: null pointer");
    if (r_min < 2 || r_step < 2 || (r_min & 1) || (r_step & 1) || r_min > d)
        return set_error(KVC_EUNSUPPORTED, "kvc_make_candidates: rank grid (%d, %d) must be even", r_min, r_step);
    if (int e = check_basis_args("kvc_make_candidates", U, order, lambda, d, d - (d - r_min) % r_step, sign)) return e;
    int64_t po = 0, wo = 0;
    for (int r = r_min, ri = 0; r <= d; r += r_step, ++ri) {
        const std::vector<int> sizes = block_sizes(r);
        const std::vector<std::vector<int>> members = deal_blocks(r, sizes);
        build_basis(U, order, d, r, sign, sizes, members, P_all + po);
        for (int b = 1; b <= 8; ++b)
            if (int e = step_of(lambda, order, r, b, delta_all + (int64_t)ri * 8 + (b - 1), "kvc_make_candidates")) return e;
        int row = 0;
        for (size_t j = 0; j < sizes.size(); ++j) {
            double s = 0.0;
            for (int i : members[j]) s = s + wt[order[i]];
            const float c = (float)(s / sizes[j]);
            for (int a = 0; a < sizes[j]; ++a) row_w_all[wo + row + a] = c;
            row += sizes[j];
        }
        po += (int64_t)r * d;
        wo += r;
    }
    return KVC_OK;
}

extern "C" const char* kvc_last_error(void) { return g_error.c_str(); }

extern "C" int32_t kvc_version(void) { return 1; }
