/*
 * kvc.h - C ABI of the KV-COBRA hot path on AMD Instinct MI355X (gfx950).
 *
 * KV-COBRA compresses each attention head's keys and values by projecting
 * them onto a per-head truncated eigenbasis with a folded Walsh-Hadamard
 * rotation, quantizing the r retained coordinates to b bits and bit-packing
 * them; the per-head (r, b) comes from a rate-distortion allocator. Decode
 * attention reads the packed codes directly.
 *
 * Conventions for every entry point
 *  - Return value: KVC_OK (0) or a positive KVC_E* code; on error a message is
 *    available from kvc_last_error() (thread-local), and no output has been
 *    written by a kernel (validation happens on the host before any launch).
 *  - "device" pointers are HIP device memory (e.g. torch tensors on cuda:0);
 *    "host" pointers are ordinary CPU memory. The library never allocates,
 *    frees or keeps any caller array; the caller owns every buffer.
 *  - Asynchronous calls enqueue kernels on `stream` (a hipStream_t; NULL is
 *    the null stream) and return without synchronising. Faults inside a
 *    kernel surface at the caller's next synchronisation.
 *  - d (head dimension) is 128; r is even in [2, d]; b is in [1, 8].
 *  - Every floating-point input must be finite.
 *
 * Packed code stream of one (unit, side), defined by this library (the
 * paper fixes only its size: exactly r*b bits per token, no metadata,
 * Appendix E):
 *  - tiles of 64 tokens, tile t at byte code_off + t * 8*r*b;
 *  - a b-bit code is split into planes (b = 8: one 8-bit plane; otherwise the
 *    binary expansion of b, widest first, widest = most significant bits);
 *    the plane of width p is 8*r*p bytes, planes in that order;
 *  - K side: inside a plane of width p, slot phi holds its p bits at bits
 *    [p*phi, p*phi + p) of the plane (a little-endian bit stream); slot of
 *    (token t in the tile, coordinate i), g16 = r/16, rho = r%16:
 *      i < 16*g16: phi = (i/16)*1024 + t*16 + i%16 (token-major in groups of
 *      16 coordinates); else phi = 1024*g16 + t*rho + (i - 16*g16);
 *  - V side: field (n, c, q) holds coordinate 16n + c for the 16 tokens of
 *    quarter q = t/16 of the tile, token t at position pos_b(t%16), p bits
 *    each (2p bytes), with pos_b(m) = m (b = 8), 8*(m/8) + 2*(m%4) + (m/4)%2
 *    (b = 4), 4*(m%4) + m/4 (other b). In a plane of width p the N-tiles n
 *    form groups of g = 8/p (1 for p = 8), and the fields of coordinates
 *    below r follow one another in the order (n/g, 4c + q, n), so the
 *    fields of one (c, q) in a group are 16 consecutive bytes (fewer in a
 *    short last group);
 *  - so a token's codes of a group of 16 coordinates (K) and a quarter of 16
 *    tokens of one coordinate (V) are one bit field of 16p bits, unpacked by
 *    the decode kernels straight into matrix-core operands, and a lane of the
 *    decode reads a V group of one plane with one 16-byte load;
 *  - kvc_encode writes only the bits of the tokens it encodes; bits of
 *    tokens never encoded keep the arena's contents (zero if the caller
 *    zeroed the arena, which the reference packing assumes).
 */
#ifndef KVC_H
#define KVC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KVC_OK 0
#define KVC_EINVAL 1        /* null pointer, bad size, inconsistent arguments */
#define KVC_EUNSUPPORTED 2  /* odd r, r > d, b outside 1..8, d != 128, step out of range */
#define KVC_ENOSPACE 3      /* token range beyond capacity, arena or workspace too small */
#define KVC_EDEVICE 4       /* a HIP runtime call failed */

#define KVC_SIDE_K 0
#define KVC_SIDE_V 1

#define KVC_SOLVER_DAMPED 0   /* C1 + damped C2 (the paper's default) */
#define KVC_SOLVER_DP 1       /* C1 + exact integer DP over per-head budgets */
#define KVC_SOLVER_C1_ONLY 2  /* C1 at the uniform budget bpd*d (V side; "w/o C2" ablation) */

#define KVC_TILE_TOKENS 64
#define KVC_HEAD_DIM 128

/* Allocator options (Sections 3.2-3.3; Appendices B-D, F). */
typedef struct kvc_alloc_opts {
    int32_t d;        /* head dimension (128) */
    int32_t r_min;    /* smallest rank on the grid (2) */
    int32_t r_step;   /* rank grid step (2) */
    int32_t b_min;    /* smallest bit width (1) */
    int32_t b_max;    /* largest bit width (8) */
    int32_t solver;   /* KVC_SOLVER_* */
    int32_t rounds;   /* C2 rounds (5) */
    int32_t reorder;  /* 1: sort directions by weight, descending (stable) */
    double bpd;       /* target bits per dimension of this side */
    double eta;       /* C2 damping (0.3) */
    double B_min;     /* per-head budget floor in bits (r_min * b_min) */
    double B_max;     /* per-head budget cap for the DP (d * b_max) */
} kvc_alloc_opts;

/* Per-head result of the allocator. */
typedef struct kvc_head_alloc {
    int32_t r;   /* retained rank */
    int32_t b;   /* bits per retained coordinate */
    double B;    /* final per-head budget in bits (real for C2, integer for DP) */
    double D;    /* modelled distortion D(r, b) */
} kvc_head_alloc;

/* One side (K or V) of a compressed cache: n_units streams plus their bases.
 * A unit is one (layer, sequence, KV head). Units may share a basis. */
typedef struct kvc_stream_desc {
    int32_t n_units;
    int32_t d;              /* 128 */
    int32_t capacity;       /* tokens each unit's stream can hold */
    int32_t side;           /* KVC_SIDE_K or KVC_SIDE_V */
    /* host mirrors, used for validation and launch planning */
    const int32_t* r_host;         /* [n_units] */
    const int32_t* b_host;         /* [n_units] */
    const int64_t* code_off_host;  /* [n_units] byte offset of the stream, multiple of 16 */
    const int64_t* basis_off_host; /* [n_units] element offset of the unit's basis */
    const float* delta_host;       /* [n_units] quantizer step, in [2^-24, 2^24] */
    /* device copies of the same tables */
    const int32_t* r;
    const int32_t* b;
    const int64_t* code_off;
    const int64_t* basis_off;      /* [n_units] element offset of the unit's r x d fp16 basis */
    const float* delta;
    /* device arenas */
    uint8_t* codes;                /* code arena */
    int64_t codes_bytes;           /* its size */
    const uint16_t* basis;         /* fp16 basis arena */
    int64_t basis_elems;           /* its size in elements */
} kvc_stream_desc;

/* Defaults listed above with the given bits per dimension. Host only. */
int kvc_alloc_opts_default(kvc_alloc_opts* o, double bpd);

/*
 * kvc_allocate - per-head rank and bit width under a total bit budget.
 * Paper: global problem Eq. (eq:global); table steps 2-4; C1 Section 3.2 and
 * Appendix B; C2 damped update Eq. (eq:c2-update), Appendix C; exact DP
 * Appendix D; V side C1 only, Appendix F.
 *
 *  lambda     host, [n_heads][d]: eigenvalues of each head's covariance in
 *             descending order (eigen index order).
 *  sigma2_q   host, [n_heads][d] or NULL: query variance along each
 *             eigendirection. Non-NULL selects the attention-KL weights
 *             w = sigma2_q * lambda (Proposition prop:kl-bound); NULL selects
 *             the MSE weights w = lambda.
 *  out        host, [n_heads]: result per head.
 *  order      host, [n_heads][d] or NULL: importance order (eigen indices
 *             sorted by w descending, ties in eigen order; identity when
 *             o->reorder == 0). The first r entries are the retained directions.
 * Budget B_tot = bpd * n_heads * d. fp64 throughout, deterministic; C1 ties
 * keep the smallest r; an infeasible budget (below r_min*b_min) yields
 * (r_min, b_min). Synchronous, host only, reentrant.
 */
int kvc_allocate(const double* lambda, const double* sigma2_q, int32_t n_heads,
                 const kvc_alloc_opts* o, kvc_head_alloc* out, int32_t* order);

/*
 * kvc_allocate_measured - the exact DP of Appendix D over measured distortion tables ("exact DP over
 * measured distortion": the calibration activations quantized once per candidate (r, b) replace the
 * Bennett model). Per head, D(r, b) = T[r] + quant[r][b] with the measured truncation term
 * T[r] = sum over importance positions p >= r of trunc_w[order[p]] (summed from the last position
 * down, fp64); the per-head optimum at budget beta is the smallest D over the grid pairs with
 * r b <= beta (ties: smallest r, then smallest b), and the budgets beta_h are the exact integer
 * knapsack of kvc_allocate's DP (same B_min, B_max, B_tot = bpd n_heads d).
 *  quant     host, [n_heads][n_r][n_b]: measured quantization term (kvc_measured_quant), rank
 *            r = r_min + ri r_step (n_r = (d - r_min) / r_step + 1), width b = b_min + bi.
 *  trunc_w   host, [n_heads][d]: weight times the measured variance along each eigendirection, by eigen
 *            index (sigma2_q * lambda_hat for the attention-KL objective, lambda_hat for MSE).
 *  order     host, [n_heads][d]: the importance order the candidate bases were built with.
 *  out       host, [n_heads]: (r, b, integer budget, D). o->solver is ignored.
 * Synchronous, host only, deterministic.
 */
int kvc_allocate_measured(const double* quant, const double* trunc_w, const int32_t* order, int32_t n_heads,
                          const kvc_alloc_opts* o, kvc_head_alloc* out);

/*
 * kvc_make_candidates - the records of every candidate rank of one head, for the measured tables:
 * for r = r_min, r_min + r_step, ..., <= d (even grid) the fused basis P_r exactly as kvc_make_basis
 * builds it, its step for every b = 1..8, and per row k of P_r the weight
 * c_k = (sum of wt over the importance positions dealt to row k's Hadamard block) / (block size),
 * which spreads a rotated coordinate's quantization error evenly over its block's eigendirections.
 *  wt         host, [d]: weight per eigen index (sigma2_q for the attention-KL objective, 1 for MSE).
 *  P_all      host out: the bases one after another, sum of r*d fp16 values.
 *  delta_all  host out, [n_r][8]: steps, b = 1..8.
 *  row_w_all  host out: sum of r floats, the row weights of each rank in turn.
 * Other arguments as kvc_make_basis. Host only.
 */
int kvc_make_candidates(const double* U, const int32_t* order, const double* lambda, const double* wt,
                        int32_t d, const int8_t* sign, int32_t r_min, int32_t r_step, uint16_t* P_all,
                        float* delta_all, float* row_w_all);

/*
 * kvc_make_basis - the stored per-head record: fused basis and quantizer step.
 * Paper: Section 3.4 and table steps 5-6 (P = H_r diag(s) U_r^T), Appendix A.1
 * (after the rotation every channel has the mean retained variance).
 *
 *  U        host, [d][d] row-major; column k is the eigenvector of eigen index k.
 *  order    host, [>= r]: importance order; order[0..r) are the retained directions.
 *  lambda   host, [d]: eigenvalues by eigen index (variances, not KL weights).
 *  sign     host, [r]: +1/-1 per importance position (the random sign flip).
 *  P        host out, [r][d]: fp16 bits of P = blockdiag(H_n/sqrt(n)) diag(sign) U_r^T.
 *           H_n are Sylvester-Hadamard blocks over the binary expansion of r,
 *           largest first; position i goes to the block with the largest
 *           remaining quota (i+1)*n_j - r*count_j (ties: larger block). For
 *           r = 2^k this is the r x r Walsh-Hadamard matrix of the paper.
 *           Entries are accumulated in fp64 over block columns in order, scaled
 *           by 1/sqrt(n) and rounded to nearest even fp16.
 *  delta    host out: f32(sqrt(mean(lambda[order[0..r)])) * delta_b), delta_b the
 *           MSE-optimal step of the 2^b-level uniform mid-rise quantizer of a
 *           unit Gaussian, to four significant digits.
 * Returns KVC_EUNSUPPORTED if the step falls outside [2^-24, 2^24].
 */
int kvc_make_basis(const double* U, const int32_t* order, const double* lambda, int32_t d,
                   int32_t r, int32_t b, const int8_t* sign, uint16_t* P, float* delta);

/*
 * kvc_encode - compress tokens [t0, t0 + n_tok) of every unit into its stream.
 * Paper: table step 7 (quantize(P k_t, b): projection and rotation in one
 * multiply), step 8 (cache the codes).
 *
 *  x            device fp16 [n_units][...]: unit u's tokens start at
 *               x + u * x_unit_stride elements, n_tok rows of d.
 *  Code of coordinate i: k = clamp(floor(y_i / delta) + 2^(b-1), 0, 2^b - 1)
 *  with y_i = sum_j P_ij x_j taken exactly (the GPU computes y in fp32 with a
 *  rigorous error bound and settles every undecided element with exact
 *  integer arithmetic), so the stream is bit-identical to the definition.
 *  Codes of tokens of the same tiles outside [t0, t0 + n_tok) are preserved
 *  (read-modify-write of the partial tiles), so a cache grows by appending.
 *  Requires t0 >= 0, n_tok >= 0, t0 + n_tok <= capacity; x must be 16-byte
 *  aligned and x_unit_stride a multiple of 8 elements, >= n_tok * d.
 *  Async on `stream`. Calls on one stream are ordered; concurrent calls that
 *  touch the same tiles race.
 */
int kvc_encode(const kvc_stream_desc* s, const uint16_t* x, int64_t x_unit_stride,
               int32_t t0, int32_t n_tok, void* stream);

/*
 * kvc_decode_attn - one decode step of attention over the compressed cache.
 * Paper: table step 8 (dequantize on read); Section 4 (logits <q,k>/sqrt(d),
 * softmax); Appendix I "Wall-clock at the primitive level" (dequantize and
 * undo the rotation in one fused pass).
 *
 *  k, v         descriptors of the K and V sides; same n_units, unit u pairs.
 *  q            device fp16 [n_units][G][d], 16-byte aligned: the G query
 *               heads sharing unit u's KV head (KVC_EINVAL if misaligned).
 *  seq_len      device int32 [n_units]: tokens attended per unit (each in
 *               [1, max_seq_len]). Being device data it is not validated:
 *               values are clamped to [0, max_seq_len] on the device, and a
 *               unit with 0 tokens gets an all-zero output.
 *  max_seq_len  host: upper bound of seq_len, <= both capacities.
 *  out          device f32 [n_units][G][d]:
 *               out[u][g] = P_V^T sum_t p_t z_V,t,
 *               p = softmax_t((P_K q_g) . z_K,t / sqrt(d)),
 *               z = (k - 2^(b-1) + 1/2) * delta (dequantized codes).
 *  ws           device workspace of >= kvc_decode_attn_workspace(...) bytes,
 *               256-byte aligned; contents on entry are ignored.
 * Split over the context (flash-decoding): each (unit, chunk) writes a
 * partial (max, sum, rank-space accumulator); a second kernel merges them and
 * applies the V basis. No atomics: results are deterministic. Async.
 */
int kvc_decode_attn(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q,
                    int32_t G, const int32_t* seq_len, int32_t max_seq_len, float* out,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * kvc_decode_step - one serving decode step in one call: append the new token's key and value to
 * every unit, then attend. Paper: table steps 7-8 (each new token is compressed and cached; attention
 * reads the cache). Equivalent to kvc_encode_kv(k, v, xk, .., xv, .., t_new, 1) followed by
 * kvc_decode_attn(k, v, q, G, seq_len, max_seq_len, out, ws, ..), with identical codes and outputs,
 * but the append runs in the same launch as the query projection (three launches instead of four).
 *  xk, xv        device fp16 [n_units][...], the new token of unit u at xk + u * xk_unit_stride (one
 *                row of d); 16-byte aligned, strides multiples of 8 elements and >= d.
 *  t_new         host: the new token's position in every unit's stream (t_new + 1 <= capacities).
 *  seq_len       as kvc_decode_attn; a step that attends to the new token passes t_new + 1.
 * Other arguments, workspace (kvc_decode_attn_workspace) and errors as kvc_decode_attn and
 * kvc_encode_kv. Async on `stream`.
 */
int kvc_decode_step(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* xk,
                    int64_t xk_unit_stride, const uint16_t* xv, int64_t xv_unit_stride, int32_t t_new,
                    const uint16_t* q, int32_t G, const int32_t* seq_len, int32_t max_seq_len, float* out,
                    void* ws, size_t ws_bytes, void* stream);

/*
 * kvc_decode_attn_rope - decode attention for a model with rotary position embeddings. Paper: Sec. 5
 * (keys are compressed before RoPE) with the rotary embedding of the Llama family.
 *  q          device fp16 [n_units][G][d], 16-byte aligned: the queries already rotated at their
 *             own positions.
 *  rope_base  host: the rotary base (e.g. 10000 or 500000), finite and > 1.
 *  out[u][g] = P_V^T sum_t p_t z_V,t,  p = softmax_t(q_g . rope(P_K^T z_K,t, t) / sqrt(d)),
 *  where rope(x, t) rotates each coordinate pair (j, j + d/2), j < d/2, by the angle
 *  t * rope_base^(-2j/d): the key of stream index t sits at position t and is rotated after its
 *  reconstruction (its codes hold the pre-RoPE key).
 * Other arguments, workspace (kvc_decode_attn_workspace) and errors as kvc_decode_attn. Async.
 */
int kvc_decode_attn_rope(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q, int32_t G,
                         const int32_t* seq_len, int32_t max_seq_len, float rope_base, float* out,
                         void* ws, size_t ws_bytes, void* stream);

/* Workspace bytes kvc_decode_attn needs for these descriptors (host only). */
size_t kvc_decode_attn_workspace(const kvc_stream_desc* k, const kvc_stream_desc* v,
                                 int32_t G, int32_t max_seq_len);

/* Size of the library's own decode workspace (see kvc_decode_attn_noalloc): 64 MiB per GPU. */
#define KVC_NOALLOC_SCRATCH_BYTES (64ll << 20)

/*
 * kvc_decode_attn_noalloc - kvc_decode_attn without a caller workspace and without any allocation.
 * For callers that cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same kernels, arguments, results and errors as kvc_decode_attn,
 * except that the workspace is a fixed array inside the library: KVC_NOALLOC_SCRATCH_BYTES bytes of
 * device memory on each GPU the library runs on, held from the library's load until the process ends
 * (its address is looked up once per device, on the first call with that device current).
 *  - KVC_ENOSPACE if these descriptors need more workspace than that (kvc_decode_attn_workspace gives
 *    the need; the measured workloads need at most ~45 MiB).
 *  - Calls no hipMalloc, hipFree or allocating library routine.
 *  - Every call on one GPU uses the same array: calls that overlap on one GPU (two streams, or two
 *    host threads without ordering) race and give undefined results. Calls ordered on one stream are
 *    safe. The array's contents on entry are ignored (every byte a call reads it wrote first).
 * Async on `stream`.
 */
int kvc_decode_attn_noalloc(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* q,
                            int32_t G, const int32_t* seq_len, int32_t max_seq_len, float* out,
                            void* stream);

/*
 * kvc_encode_kv - kvc_encode of the keys and the values of the same tokens in one call.
 * Paper: table step 7-8 (a decode step caches the new token's key and value). For
 * n_tok <= 4 (appending a decode step's tokens) both sides run in one launch; longer
 * runs take the bulk encoder, one launch per side. Codes are those kvc_encode writes.
 *  k, v          descriptors of the K (side 0) and V (side 1) streams, same n_units.
 *  xk, xv        device fp16 tokens of each side, laid out as kvc_encode's x.
 * Same requirements and errors as kvc_encode for each side, plus KVC_EINVAL for
 * swapped sides or differing unit counts. Async on `stream`.
 */
int kvc_encode_kv(const kvc_stream_desc* k, const kvc_stream_desc* v, const uint16_t* xk, int64_t xk_unit_stride,
                  const uint16_t* xv, int64_t xv_unit_stride, int32_t t0, int32_t n_tok, void* stream);

/*
 * kvc_reconstruct - x_hat_t = P^T z_t for tokens [t0, t0 + n_tok) of every unit.
 * Paper: Appendix A, Lemma lem:head-dist (x_hat = U_r H_r^T Q(H_r U_r^T x)).
 *  out   device f32 [n_units][n_tok][d]. Async.
 */
int kvc_reconstruct(const kvc_stream_desc* s, int32_t t0, int32_t n_tok, float* out, void* stream);

/*
 * kvc_read_probe - measurement utility, not a step of the method: streams `bytes` bytes of device
 * memory with 16-byte non-temporal loads over the whole device. Its rate is the achievable HBM read
 * bandwidth that the decode kernels are compared against (the paper's premise, Sec. 1, is that decode
 * is bound by reading the KV cache).
 *  buf    device memory, 16-byte aligned; bytes a multiple of 16 (0: no launch).
 *  sink   one device uint32, 4-byte aligned, owned by the caller; written only when the folded value
 *         of every loaded word equals a fixed constant (it exists to keep the loads live).
 * KVC_EINVAL on a null or misaligned argument. Async on `stream`.
 */
int kvc_read_probe(const void* buf, size_t bytes, uint32_t* sink, void* stream);

/*
 * Calibration on the device (table step 1; Section 2 for the query variance; the paper computes the
 * eigendecomposition in fp32). Batched over heads; every array is device memory owned by the caller;
 * async on `stream`. The results feed kvc_allocate (lambda, sigma2_q) and kvc_make_basis (U) on the host.
 *
 * kvc_covariance - cov[h] = (1/n) sum_t x_t x_t^T - mu mu^T (centered = 1) or without the mean term
 * (centered = 0), mu = (1/n) sum_t x_t, for the n_tok calibration activations of each head.
 *  x      device fp16 [n_heads][...]: head h's tokens start at x + h * x_head_stride elements, n_tok
 *         rows of d = 128. 16-byte aligned; x_head_stride a multiple of 8, >= n_tok * d.
 *  cov    device f32 [n_heads][d][d], row-major. fp32 accumulation of exact fp16 products.
 */
int kvc_covariance(const uint16_t* x, int64_t x_head_stride, int32_t n_heads, int32_t n_tok,
                   int32_t centered, float* cov, void* stream);

/*
 * kvc_eigh - eigendecomposition S = U diag(lambda) U^T of n symmetric d x d matrices (fp32 Jacobi).
 *  S        device f32 [n][d][d] (read only; only symmetric input is meaningful).
 *  lambda   device f32 [n][d] out: eigenvalues in descending order (negative ones clamped to 0).
 *  U        device f32 [n][d][d] out, row-major: column k (U[j*d + k]) is the eigenvector of
 *           lambda[k], its largest-magnitude entry made positive.
 *  sweeps   device int32 [n] out, or NULL: Jacobi sweeps used per matrix (-1: not converged in 30).
 * Ties in lambda keep the order of the converged diagonal.
 */
int kvc_eigh(const float* S, int32_t n, float* lambda, float* U, int32_t* sweeps, void* stream);

/*
 * kvc_query_variance - sigma2_q[h][i] = (1/G) sum_g u_i^T S_q[h][g] u_i: the query variance along each
 * eigendirection u_i (column i of U[h]), averaged over the G query heads sharing KV head h.
 *  U        device f32 [n_heads][d][d] as kvc_eigh writes it.
 *  S_q      device f32 [n_heads][G][d][d]: query covariances.
 *  sigma2_q device f32 [n_heads][d] out.
 */
int kvc_query_variance(const float* U, const float* S_q, int32_t n_heads, int32_t G, float* sigma2_q,
                       void* stream);

/*
 * kvc_measured_quant - the quantization term of the measured distortion tables on the device: for every
 * head h, candidate rank r (grid r_min, r_min + r_step, ..., <= d) and width b = 1..8,
 *   quant[h][ri][b-1] = (1/n_tok) sum_t sum_k c_k (z_tk - zhat_tk)^2,  z_t = P_r x_t,
 * zhat the dequantized b-bit code of z with the candidate's step (fp32 projection of the exact fp16
 * products; a measurement, so codes are decided in fp32).
 *  x          device fp16 [n_heads][...] calibration activations, head h at x + h * x_head_stride, n_tok
 *             rows of d; 16-byte aligned, stride a multiple of 8 and >= n_tok * d.
 *  P_all, delta_all, row_w_all  device copies of kvc_make_candidates' outputs, one head after another
 *             (P_head_stride elements, a multiple of 8, between heads' bases; delta [n_heads][n_r][8];
 *             rw_head_stride floats between heads' row weights).
 *  quant      device f32 [n_heads][n_r][8] out.
 * Async on `stream`.
 */
int kvc_measured_quant(const uint16_t* x, int64_t x_head_stride, int32_t n_heads, int32_t n_tok,
                       const uint16_t* P_all, int64_t P_head_stride, const float* delta_all,
                       const float* row_w_all, int64_t rw_head_stride, int32_t r_min, int32_t r_step,
                       float* quant, void* stream);

/* Message of the last failing call on this thread ("" if none). */
const char* kvc_last_error(void);

/* Library version, for the binding's load check. */
int32_t kvc_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KVC_H */
