/*
 * fm.h -- C ABI of libfm: low-precision (FP8) evaluation of bilinear fast
 * matrix multiplication schemes on AMD Instinct MI355X (gfx950), across
 * batches of gauge-transformed copies of a scheme.
 *
 * The method (Xie et al., "Beyond Accuracy: Prefix-Invariant Realizations of
 * Low-Precision Fast Matrix Multiplication"):
 *   eq. (1), Sec. 2.1 -- A is split into an m x k grid of blocks A_il and B
 *     into a k x n grid B_lj; R products of block sums
 *       M_r = (sum_il u_{r,il} A_il)(sum_lj v_{r,lj} B_lj)
 *     are combined as C_ij = sum_r w_{r,ij} M_r;
 *   Sec. 2.1 -- sign variants: running the scheme on DAE and EBF and flipping
 *     back gives coefficients d_i e_l u, e_l f_j v, d_i f_j w; the same exact
 *     product;
 *   App. B.1 -- the FP8 schedule: block sums rounded to FP8 (e4m3) before
 *     multiplying, products combined in fp32; relative Frobenius error
 *     against a float64 reference (App. F).
 *
 * Conventions for every call:
 *   - Return value: FM_OK (0) or a negative FM_E_* code; no call throws or
 *     aborts across the ABI (a host allocation that fails inside a call
 *     returns FM_E_NOMEM; the size queries then return 0).  fm_last_error()
 *     gives a thread-local message describing the most recent failure on
 *     the calling thread.
 *   - Host arrays are row-major doubles and are copied; the library never
 *     keeps a caller's host pointer.
 *   - Device arrays are caller-owned, row-major, and must be device memory
 *     of the current HIP device.  No call allocates device memory: scratch
 *     space comes from the caller's workspace.
 *   - `hip_stream` is a hipStream_t passed as void* (NULL = default stream).
 *     Calls marked "async" only enqueue work on it; calls marked
 *     "synchronizes" wait for the stream before returning.
 *   - Grid index flattening: (i,l) -> i*k + l, (l,j) -> l*n + j,
 *     (i,j) -> i*n + j.  Blocks are contiguous: block (i,l) of A covers rows
 *     [i*M/m, (i+1)*M/m) and columns [l*K/k, (l+1)*K/k).
 *   - A scheme flattened to L levels (the scheme applied recursively inside
 *     its own blocks, Sec. 1: "two-level Strassen") has grid m^L x k^L x n^L
 *     and R^L products, product index r = r1*R^(L-1) + ... + rL and block
 *     index i = i1*m^(L-1) + ... + iL (outer level first).
 */
#ifndef FM_H
#define FM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---------------------------------------------------------------- errors */
#define FM_OK 0
#define FM_E_ARG (-1)        /* null pointer, non-positive size, bad enum   */
#define FM_E_SHAPE (-2)      /* M, N, K not divisible by the block grid, or */
                             /* a dimension beyond the supported range      */
#define FM_E_BRENT (-3)      /* coefficients do not compute AB (residual of */
                             /* the Brent equations above 1e-9)             */
#define FM_E_SINGULAR (-4)   /* a gauge matrix is not invertible            */
#define FM_E_NONFINITE (-5)  /* an Inf/NaN reached a block sum              */
#define FM_E_WORKSPACE (-6)  /* workspace NULL, misaligned or too small     */
#define FM_E_HIP (-7)        /* the HIP runtime reported an error           */
#define FM_E_MISMATCH (-8)   /* schemes of one orbit differ in shape        */
#define FM_E_NOMEM (-9)      /* host allocation failed                      */
#define FM_E_UNSUPPORTED (-10) /* no kernel for this grid size              */
#define FM_E_RANGE (-11)       /* a block sum of integer codes left int8:
                                  codes beyond the certified bound          */
#define FM_E_UNCERTIFIED (-12) /* the scheme, code bounds and tiling do not
                                  meet Prop. 1's conditions                 */

typedef struct fm_scheme fm_scheme; /* opaque, immutable, library-owned     */

typedef enum { FM_E4M3 = 0, FM_E5M2 = 1 } fm_fmt; /* OCP E4M3FN, OCP E5M2  */

/* Arithmetic of the block products (fm_set_block_product_arithmetic). */
typedef enum { FM_ACC_BF16 = 0, FM_ACC_FP8 = 1 } fm_accum;

/* Scale granularity of the FP8 rounding of block sums.
 *   FM_SCALE_TENSOR: one scale per block-sum tensor (per product and side);
 *     scale arrays hold R values per gauge and side.
 *   FM_SCALE_ROWCOL: one scale per row of every block sum of A and per
 *     column of every block sum of B, the form the paper uses on synthetic
 *     matrices (App. B.1); scale arrays hold R x Mb values (A side) and
 *     R x Nb values (B side) per gauge.
 *   FM_SCALE_GROUP: the models' schedule (App. B.1): one scale per row of
 *     A's block sums and 128 consecutive inner entries; B's block sums are
 *     first rounded to bf16, then get one scale per 128 x 128 block; block
 *     products are returned in bf16 (as fp32 values).  Scale arrays hold
 *     R x (Kb/128) x Mb (A) and R x (Kb/128) x (Nb/128) (B) per gauge. */
/* Repairs (App. C, the repair rules), OR-ed into the fm_scale_mode argument
 * of the *_scaled calls (except fm_block_products_scaled), with
 * FM_SCALE_GROUP only (FM_E_ARG otherwise):
 *   FM_REPAIR_ROWS: every row t of A is divided by d_t = 2^k_t before the
 *     block sums and the output row t multiplied by d_t afterwards, k_t the
 *     least integer with 4^k_t >= m2_t and k_t >= -9, where m2_t is the
 *     float64 mean of the squares of the row (partial sums over the indices
 *     mod 64 in ascending order, combined pairwise as v[l] + v[l ^ off] for
 *     off = 32, ..., 1, then divided by K): 2^k_t is the least power of two
 *     at least max(RMS, 1e-3);
 *   FM_REPAIR_WEIGHTS: the FP8 codes of B's bf16 block sums are chosen
 *     jointly at every position: each product's two codes whose values
 *     bracket s q (its block's scales q, d), starting at the value nearer s
 *     (fp32 distances), then sweeps r = 0..R-1 taking the other code when
 *     fl(fl(2 delta) g_r) + fl(fl(delta delta) H_rr) < 0, where e_r =
 *     fl(fl(code value * d) - s), g = H e (fmaf, ascending), updated by
 *     g_t = fmaf(H_tr, delta, g_t) on each change, and H_rs =
 *     fl32(<w_r, w_s> <u_r, u_s>) in float64; at most 12 sweeps, stopping
 *     after one with no change.  Built for R <= 64 (FM_E_UNSUPPORTED
 *     otherwise). */
typedef enum {
  FM_SCALE_TENSOR = 0,
  FM_SCALE_ROWCOL = 1,
  FM_SCALE_GROUP = 2,
  FM_REPAIR_ROWS = 0x100,
  FM_REPAIR_WEIGHTS = 0x200
} fm_scale_mode;

typedef struct {
  double rel_fro; /* ||C - C_ref||_F / ||C_ref||_F (0 if C_ref = 0)         */
  double err_sq;  /* sum (C - C_ref)^2, float64                             */
  double ref_sq;  /* sum C_ref^2, float64                                   */
  double max_abs; /* max |C - C_ref|                                        */
} fm_stats;

/* Text for an FM_E_* code (static storage). */
const char* fm_strerror(int code);
/* Message for the last failure on this thread ("" if none). */
const char* fm_last_error(void);
/* Library version string. */
const char* fm_version(void);

/* ------------------------------------------------------- scheme (host) */

/* Load a scheme from its coefficients, eq. (1) of Sec. 2.1.
 * U: R x (m*k), V: R x (k*n), W: R x (m*n), row-major float64, copied.
 * The scheme is accepted only if it computes AB: the largest residual of the
 * Brent equations sum_r u_{r,il} v_{r,l'j} w_{r,i'j'} = [i=i'][l=l'][j=j']
 * must be <= 1e-9 (FM_E_BRENT otherwise).  On success *out owns a new scheme
 * that the caller releases with fm_scheme_free.  Sizes: 1 <= m,n,k <= 16,
 * 1 <= R <= 4096. */
int fm_scheme_load(const double* U, const double* V, const double* W, int m,
                   int n, int k, int R, fm_scheme** out);

/* Gauge-transformed copy of a scheme (the sign variants of Sec. 2.1,
 * generalized to invertible P (m x m), Q (k x k), S (n x n), row-major
 * float64): the scheme run on P A Q and Q^-1 B S and undone with
 * P^-1 . S^-1, i.e.
 *   U'_r = (P^T U_r) Q^T,   V'_r = (Q^-T V_r) S^T,   W'_r = (P^-1 W_r) S^-1,
 * computed in float64 (each matrix product summed over its inner index in
 * ascending order; inverses of order <= 3 by adjugate / determinant, larger
 * ones by Gauss-Jordan elimination with partial pivoting).  Diagonal +-1
 * P, Q, S give exactly the paper's sign variants.  FM_E_SINGULAR if P, Q or
 * S has zero determinant (or a zero pivot), or if X X^-1 differs from the
 * identity by more than 1e-12 n max|X| max|X^-1| for X = P, Q, S (the base
 * scheme passed the Brent check, so accurate inverses keep it exact). */
int fm_gauge_apply(const fm_scheme* s, const double* P, const double* Q,
                   const double* S, fm_scheme** out);

/* fm_gauge_apply for G gauge elements at once (one call for a whole orbit):
 * P is G x m x m, Q is G x k x k, S is G x n x n (row-major float64,
 * element g at offset g*m*m, ...); out receives G new schemes.  On failure
 * no scheme is returned (every out[g] is NULL) and the code is that of the
 * first failing element. */
int fm_gauge_apply_batch(const fm_scheme* s, int G, const double* P,
                         const double* Q, const double* S, fm_scheme** out);

/* The scheme applied recursively `levels` times and flattened to one level
 * (Kronecker power, outer level first; coefficients multiplied in float64
 * from the outer level in).  levels = 1 returns a copy.  Two-level Strassen
 * is fm_scheme_kron(strassen, 2): grid 4 x 4 x 4, 49 products. */
int fm_scheme_kron(const fm_scheme* s, int levels, fm_scheme** out);

/* Grid and rank of a scheme (any pointer may be NULL). */
int fm_scheme_dims(const fm_scheme* s, int* m, int* n, int* k, int* R);

/* Float64 coefficients (U: R x m*k, V: R x k*n, W: R x m*n). */
int fm_scheme_coeffs(const fm_scheme* s, double* U, double* V, double* W);

/* Coefficients of the scheme flattened to `levels` levels, each rounded once
 * from float64 to fp32 (round to nearest even): exactly the tables the
 * kernels use.  Sizes R^L x (mk)^L, R^L x (kn)^L, R^L x (mn)^L. */
int fm_scheme_coeffs_f32(const fm_scheme* s, int levels, float* U, float* V,
                         float* W);

void fm_scheme_free(fm_scheme* s);

/* ------------------------------------------------------ workspace sizing */

/* Bytes of device workspace needed to evaluate G gauged copies of `s`
 * (flattened to `levels`) at M x K times K x N, `chunk` copies at a time
 * (chunk <= 0 means all G at once).  0 if the arguments are invalid.
 * With chunk < G the size includes a second set of a chunk's block
 * products, maxima and scales, so that fm_orbit_eval can reconstruct one
 * chunk while the next is formed (and, with one scale per tensor, form a
 * chunk's maxima one chunk ahead).
 * fm_matmul_lowp and fm_form_operands need fm_workspace_size(s,M,N,K,L,1,1).
 * The workspace must be 256-byte aligned. */
size_t fm_workspace_size(const fm_scheme* s, int M, int N, int K, int levels,
                         int G, int chunk);

/* Bytes of workspace fm_error_stats needs for an M x N output. */
size_t fm_error_workspace_size(int M, int N);

/* --------------------------------------------------- the FP8 schedule */

/* Operand formation only (steps: block sums, one scale per block-sum
 * tensor, FP8 codes), for checking.  Async.
 * For every product r of the scheme flattened to `levels` (grid gm x gk x gn):
 *   T_r = sum over nonzero u_{r,il}, ascending row-major (i,l), of
 *         u * A_il, formed in fp32 as a chain of fused multiply-adds
 *         starting from +0;   S_r likewise from v_{r,lj} and B_lj, (l,j)
 *         ascending row-major;
 *   amax = max |T_r| over the whole tensor; d = amax / FMAX and
 *         q = FMAX / amax (each a correctly rounded fp32 division;
 *         d = q = 1 if amax = 0); FMAX = 448 (E4M3) or 57344 (E5M2);
 *   code = FP8(fl(x * q)), round to nearest even, saturating (no overflow
 *         can occur since |x * q| <= FMAX (1 + 2^-23)^2).
 * Outputs (device, caller-owned):
 *   Tq: R^L x (M/gm) x (K/gk) bytes (row-major per product),
 *   Sq: R^L x (N/gn) x (K/gk) bytes -- S_r TRANSPOSED (inner dimension
 *       contiguous), i.e. Sq[r][z][y] is the code of S_r[y][z],
 *   dT, dS: R^L floats.
 * A non-finite block sum makes the next synchronizing call on this
 * workspace (fm_error_stats, fm_orbit_eval, fm_status) return
 * FM_E_NONFINITE. */
int fm_form_operands(const fm_scheme* s, int levels, const float* A,
                     const float* B, int M, int N, int K, fm_fmt fmt,
                     uint8_t* Tq, uint8_t* Sq, float* dT, float* dS,
                     void* workspace, size_t ws_bytes, void* hip_stream);

/* Block products (step M_r of eq. (1) on FP8 operands), batched.  Async.
 * For b in [0, batch): Mout[b] = ((Tq[b] * Sq[b]^T accumulated in fp32 by
 * the matrix cores) * dT[b]) * dS[b], two fp32 multiplications.  The
 * products are exact and summed in fp32 (FM_ACC_BF16, the default), or
 * formed by the FP8 matrix instructions (FM_ACC_FP8); see
 * fm_set_block_product_arithmetic.
 * Tq: batch x Mb x Kb, Sq: batch x Nb x Kb (inner dimension contiguous),
 * dT, dS: batch floats, Mout: batch x Mb x Nb fp32.  Mb, Nb, Kb >= 1; Kb a
 * multiple of 16. */
int fm_block_products(const uint8_t* Tq, const uint8_t* Sq, const float* dT,
                      const float* dS, int batch, int Mb, int Nb, int Kb,
                      fm_fmt fmt, float* Mout, void* hip_stream);

/* Reconstruction C_ij = sum_r w_{r,ij} M_r (eq. (1)), fp32 fused
 * multiply-adds over nonzero w in ascending r, starting from +0.  Async.
 * Mprod: R^L x (M/gm) x (N/gn) fp32; C: M x N fp32. */
int fm_reconstruct(const fm_scheme* s, int levels, const float* Mprod, int M,
                   int N, float* C, void* workspace, size_t ws_bytes,
                   void* hip_stream);

/* The whole FP8 schedule for one scheme: C (M x N fp32, device) from
 * A (M x K) and B (K x N) fp32 device arrays.  Async.  Workspace:
 * fm_workspace_size(s, M, N, K, levels, 1, 1) bytes.  The classical FP8
 * baseline is this call with the 1 x 1 x 1 rank-1 scheme. */
int fm_matmul_lowp(const fm_scheme* s, const float* A, const float* B,
                   float* C, int M, int N, int K, int levels, fm_fmt fmt,
                   void* workspace, size_t ws_bytes, void* hip_stream);

/* Float64 reference C_ref = A B from fp32 A (M x K) and B (K x N), device
 * arrays (App. F: a float64 reference).  Async. */
int fm_reference_f64(const float* A, const float* B, double* C_ref, int M,
                     int N, int K, void* hip_stream);

/* Relative Frobenius error of C against C_ref (App. B.1), float64 sums in a
 * fixed order (bit-reproducible run to run).  Synchronizes; writes *out. */
int fm_error_stats(const float* C, const double* C_ref, int M, int N,
                   fm_stats* out, void* workspace, size_t ws_bytes,
                   void* hip_stream);

/* fm_error_stats without a workspace, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the same kernels, sums and result,
 * with the reduction's partial sums in a static device array of the
 * library (32768 bytes per device, held until the process ends) instead of
 * a caller's workspace.  Allocates nothing (no hipMalloc, hipFree or pinned
 * host memory; the 24-byte result is copied straight into a host local).
 * Every output size fits the array (the reduction uses at most 1024
 * workgroups); FM_E_WORKSPACE would report one that did not.  All calls on
 * one device share that device's array: calls that overlap in time on one
 * device (several host threads, or several streams) race and must be
 * serialized by the caller.  Synchronizes; writes *out. */
int fm_error_stats_noalloc(const float* C, const double* C_ref, int M, int N,
                           fm_stats* out, void* hip_stream);

/* Orbit evaluation: for each of G gauged schemes (same grid and rank after
 * flattening to `levels`), the whole FP8 schedule on A, B and the float64
 * relative Frobenius error against C_ref (M x N float64, device), reduced on
 * the device; rel_fro_out (host, G doubles) receives the errors.  C is not
 * materialized.  Works through the gauges in chunks that fit `ws_bytes`
 * (fm_workspace_size(.., G, chunk)): the largest chunk reached by halving G
 * that fits.  With several chunks and room for two product buffers, each
 * chunk's reconstruction runs on a second stream of the library's (one per
 * device, default priority), ordered by events against the caller's stream,
 * beside the next chunk's formation; concurrent calls on one device share
 * that stream (their reconstructions then run one after another).  The
 * results are the bits of the one-buffer schedule; within a chunk the
 * products may be stored in a tiled order internally (when they are whole
 * tiles of the block-product kernel, 512 x 128 or 256 x 128, with tensor
 * scales).  Synchronizes. */
int fm_orbit_eval(const fm_scheme* const* gauged, int G, const float* A,
                  const float* B, const double* C_ref, int M, int N, int K,
                  int levels, fm_fmt fmt, double* rel_fro_out,
                  void* workspace, size_t ws_bytes, void* hip_stream);

/* ------------------------------------------- finer scale granularity
 * The same calls with an explicit fm_scale_mode.  FM_SCALE_TENSOR gives
 * exactly the calls above.  FM_SCALE_ROWCOL follows App. B.1's synthetic
 * form: every row x of every A-side block sum T_r has its own amax, d and q
 * (same rule as a whole tensor: correctly rounded fp32 divisions, d = q = 1
 * for an all-zero row), and so does every column z of every B-side block
 * sum S_r (a row of the transposed Sq).  Block products are then
 * M_r[x][z] = ((sum_k Tq_r[x][k] Sq_r[z][k]) * dT_r[x]) * dS_r[z].
 * Scale arrays: dT holds R^L x Mb floats ([r][x]), dS holds R^L x Nb floats
 * ([r][z]); fm_block_products_scaled takes batch x Mb and batch x Nb.
 * FM_SCALE_GROUP (App. B.1, the models' schedule): every group of 128
 * consecutive inner entries of a row of T_r has its own scale, and S_r,
 * rounded to bf16 (nearest even) first, one per 128 x 128 block (128
 * columns z by 128 inner entries); then for every group kg in ascending
 * order acc = fmaf(P_kg, dT_r[kg][x] * dS_r[kg][z / 128], acc) from +0,
 * where P_kg is the group's sum of code products, and M_r = bf16(acc).
 * Needs Kb and Nb multiples of 128 and Mb of 4 (FM_E_SHAPE otherwise).
 * Scale arrays: dT [r][kg][x] (R^L x Kb/128 x Mb), dS [r][kg][zb]
 * (R^L x Kb/128 x Nb/128); fm_block_products_scaled takes them per batch
 * entry in that layout.
 * FM_E_ARG for an unknown mode; otherwise errors as in the calls above. */

/* Workspace bytes for fm_orbit_eval_scaled / fm_matmul_lowp_scaled /
 * fm_form_operands_scaled (0 on a bad argument). */
size_t fm_workspace_size_scaled(const fm_scheme* s, int M, int N, int K,
                                int levels, int G, int chunk,
                                fm_scale_mode scale_mode);

/* fm_form_operands with a scale granularity.  Async. */
int fm_form_operands_scaled(const fm_scheme* s, int levels, const float* A,
                            const float* B, int M, int N, int K, fm_fmt fmt,
                            fm_scale_mode scale_mode, uint8_t* Tq,
                            uint8_t* Sq, float* dT, float* dS,
                            void* workspace, size_t ws_bytes,
                            void* hip_stream);

/* fm_block_products with a scale granularity.  Async.  The kernels read the
 * scale arrays in aligned 16-byte chunks: with FM_SCALE_ROWCOL dS must be
 * 16-byte aligned; with FM_SCALE_GROUP dT and dS must be 16-byte aligned
 * and readable up to the next multiple of 4 floats past their last entry
 * (pad the allocation).  FM_E_ARG for a misaligned scale array. */
int fm_block_products_scaled(const uint8_t* Tq, const uint8_t* Sq,
                             const float* dT, const float* dS, int batch,
                             int Mb, int Nb, int Kb, fm_fmt fmt,
                             fm_scale_mode scale_mode, float* Mout,
                             void* hip_stream);

/* fm_matmul_lowp with a scale granularity.  Async. */
int fm_matmul_lowp_scaled(const fm_scheme* s, const float* A, const float* B,
                          float* C, int M, int N, int K, int levels,
                          fm_fmt fmt, fm_scale_mode scale_mode,
                          void* workspace, size_t ws_bytes,
                          void* hip_stream);

/* fm_orbit_eval with a scale granularity.  Synchronizes. */
int fm_orbit_eval_scaled(const fm_scheme* const* gauged, int G,
                         const float* A, const float* B, const double* C_ref,
                         int M, int N, int K, int levels, fm_fmt fmt,
                         fm_scale_mode scale_mode, double* rel_fro_out,
                         void* workspace, size_t ws_bytes, void* hip_stream);

/* ------------------------------------------------------ integer path
 * The quantization specification of Sec. 2.2 / App. D and the two operators
 * of Sec. 4.2 on it.  Codes are int8; groups of g consecutive entries along
 * the inner dimension share a scale per row of A and per column of B.
 * Scale arrays are group-major: dA[gi * M + t], dB[gi * N + j].
 * B always enters transposed (N x K codes), so both operands have the
 * inner dimension contiguous. */

/* Integer codes of X (rows x K fp32, device): for every row t and group gi,
 * d = max|x| / b over the group's g entries (one correctly rounded fp32
 * division; d = 1 for an all-zero group) and code = x / d (one fp32
 * division) rounded to the nearest integer, ties to even, no clipping
 * (|code| <= b).  codes: rows x K int8; d: (K/g) x rows fp32 (group-major).
 * A group holding Inf or NaN ORs 1 into *flag (device, may be NULL).
 * g a multiple of 64 and at most 512, K a multiple of g, 1 <= b <= 127.
 * Quantize A directly and B through its transpose.  Async. */
int fm_int8_quantize(const float* X, int rows, int K, int g, int b,
                     int8_t* codes, float* d, uint32_t* flag,
                     void* hip_stream);

/* The classical int8 operator at the specification (Sec. 2.2): for every
 * group gi in ascending order, the exact integer product P of the group's
 * codes (int32 on the matrix cores, exact since |P| <= g b^2 < 2^24) is
 * converted to fp32 and added as out += (P * dA) * dB, each step a
 * separate fp32 operation, to an output starting at +0.  Ac: M x K, BTc:
 * N x K codes; dA: (K/g) x M, dB: (K/g) x N; out: M x N fp32 (device).
 * g a multiple of 128; M, N multiples of 4.  Async. */
int fm_int8_matmul_classical(const int8_t* Ac, const float* dA,
                             const int8_t* BTc, const float* dB, int M,
                             int N, int K, int g, float* out,
                             void* hip_stream);

/* Prop. 1's certificate for the scheme flattened to `levels`, code bounds
 * b_A, b_B, blocks of inner length h and groups of g (int32 accumulation):
 *   (i)   L_A b_A <= 127 and L_B b_B <= 127,
 *   (ii)  max(L_W h (L_A b_A)(L_B b_B), g b_A b_B) < 2^31,
 *   (iii) a call (k^levels blocks of length h) lies within one group.
 * conditions (host, 3 ints) receive 1/0 per condition; L (host, 3 doubles)
 * receives L_A, L_B, L_W (largest coefficient 1-norms of the block sums and
 * largest total weight of an output block).  FM_E_ARG if the coefficients
 * are not integers. */
int fm_int8_certify(const fm_scheme* s, int levels, int b_A, int b_B, int h,
                    int g, int* conditions, double* L);

/* Workspace bytes for fm_int8_matmul_fast (0 on a bad argument). */
size_t fm_int8_workspace_size(const fm_scheme* s, int levels, int M, int N,
                              int K, int g, int h);

/* The certified fast realization (Sec. 4.2): the classical operator's
 * quantization, rescaling and fp32 order, with every group's integer
 * product computed call by call by the scheme: for each call (k^levels
 * consecutive blocks of inner length h within one group) the block sums of
 * the codes T_r, S_r (exact int8 under the certificate), and every output
 * block C_ij = sum_r w_{r,ij} T_r S_r on the matrix cores in int32.  Output
 * bits equal fm_int8_matmul_classical's on every input whose codes are
 * within b_A, b_B.  FM_E_UNCERTIFIED if (i)-(iii) fail or the combination
 * weights are not in {-1, 0, 1}; a block sum outside int8 (codes beyond the
 * bounds) is reported as FM_E_RANGE by the next fm_status on the
 * workspace.  h a multiple of 16 dividing 128; M, N multiples of 4 m^levels
 * and 4 n^levels.  Async. */
int fm_int8_matmul_fast(const fm_scheme* s, int levels, const int8_t* Ac,
                        const float* dA, const int8_t* BTc, const float* dB,
                        int M, int N, int K, int g, int h, int b_A, int b_B,
                        float* out, void* workspace, size_t ws_bytes,
                        void* hip_stream);

/* The overflow correction (Sec. 4.3, eq. (2); App. D, the corrected
 * computation's certificate): every exact block sum s of codes is split as
 * s = s0 + 256 q, q = floor((s + 128) / 256), s0 in [-128, 127], and each
 * block product as A0 B0 + 256 (R_A B0 + A0 R_B) + 256^2 R_A R_B on the
 * int8 matrix cores, all in one exact int32 accumulator; the result is
 * classical int8's at the same specification bit for bit, up to code bound
 * 127.  fm_int8_certify_corrected: conditions[0] the split parts q fit int8
 * (|q| <= qmax = floor((L b + 128) / 256)), [1] the sum of the absolute
 * weighted terms per output entry, L_W h (128 + 256 qmax_A)(128 + 256
 * qmax_B), and g b_A b_B stay below 2^31, [2] a call lies within one group;
 * bounds[0] that sum, bounds[1..2] qmax_A, qmax_B (two-level Strassen at 127
 * with h = 32: 16 * 13,107,200 and 2, 2).  The kernel needs one call per
 * group (g = k^levels h), else FM_E_UNSUPPORTED; a split part beyond qmax
 * (codes beyond the bounds) is FM_E_RANGE at the next fm_status.  Async. */
int fm_int8_certify_corrected(const fm_scheme* s, int levels, int b_A, int b_B,
                              int h, int g, int* conditions, double* bounds);
size_t fm_int8_workspace_size_corrected(const fm_scheme* s, int levels, int M,
                                        int N, int K, int g, int h);
int fm_int8_matmul_corrected(const fm_scheme* s, int levels, const int8_t* Ac,
                             const float* dA, const int8_t* BTc,
                             const float* dB, int M, int N, int K, int g,
                             int h, int b_A, int b_B, float* out,
                             void* workspace, size_t ws_bytes,
                             void* hip_stream);

/* A fast call prepared once: fm_int8_plan_create validates and certifies
 * exactly as fm_int8_matmul_fast (correct = 0) or fm_int8_matmul_corrected
 * (correct = 1) does, then writes the scheme's tables and the tile schedule
 * into the caller's workspace (async on hip_stream, which orders them before
 * any later work on it; sized by the matching workspace-size call).  The
 * plan records the workspace; keep it alive and unchanged while the plan is
 * used.  fm_int8_plan_run performs the call on new codes and scales of the
 * planned shapes, with the same result and errors as the one-shot call;
 * runs that share a plan on different streams race on its workspace.
 * Library-owned handle, freed by fm_int8_plan_free (null is ignored). */
typedef struct fm_int8_plan fm_int8_plan;
int fm_int8_plan_create(const fm_scheme* s, int levels, int M, int N, int K,
                        int g, int h, int b_A, int b_B, int correct,
                        void* workspace, size_t ws_bytes, void* hip_stream,
                        fm_int8_plan** out);
int fm_int8_plan_run(const fm_int8_plan* p, const int8_t* Ac, const float* dA,
                     const int8_t* BTc, const float* dB, float* out,
                     void* hip_stream);
void fm_int8_plan_free(fm_int8_plan* p);

/* Selects, process-wide, how the block products are multiplied (the App. B
 * schedule multiplies FP8 block sums and combines the products in fp32):
 *   FM_ACC_BF16 (default): every FP8 value is widened exactly to bf16 and
 *     multiplied on the bf16 matrix cores with fp32 accumulation (within
 *     about 2e-7 of the exact sums rounded once);
 *   FM_ACC_FP8: the gfx950 FP8 matrix instructions, at twice the rate, which
 *     truncate small products summed beside large ones (about 5e-5 relative
 *     on random FP8 data).
 * FM_E_ARG for any other value. */
int fm_set_block_product_arithmetic(fm_accum a);

/* ------------------------------------------------------------ diagnostics */

/* FP8 codes of n fp32 device values x, written to out (device, n bytes):
 * impl 0 = the encoder the formation kernels use, 1 = the gfx950 conversion
 * instructions (v_cvt_pk_fp8_f32 / v_cvt_pk_bf8_f32), 2 = the integer
 * encoder.  Round to nearest even; values beyond the largest finite value
 * saturate (impl 2) -- the schedule never produces such values.  Async. */
int fm_fp8_encode(const float* x, int64_t n, fm_fmt fmt, int impl, uint8_t* out,
                  void* hip_stream);

/* The bf16 rounding of the group schedule (App. B.1: B's block sums are
 * rounded to bf16 before their scales and codes) applied to n fp32 device
 * values x; out (device, n floats) holds the bf16 values as fp32:
 * impl 0 = the rounding the formation kernels use, 1 = the gfx950
 * conversion instruction (v_cvt_pk_bf16_f32), 2 = the integer rounding
 * (add 0x7fff plus the kept low bit, truncate).  Nearest, ties to even;
 * finite inputs (the formation flags non-finite ones).  Async. */
int fm_bf16_round(const float* x, int64_t n, int impl, float* out, void* hip_stream);

/* Name of the kernel family that evaluates `s` flattened to `levels`
 * ("Strassen2", "DenseR7G2", ... or "generic"): families have formation and
 * reconstruction kernels compiled for their nonzero structure.  Static
 * string; "" on error. */
const char* fm_scheme_kernel_family(const fm_scheme* s, int levels);

/* Whether `s` flattened to `levels` is a sign variant of its kernel family's
 * base scheme on operand side `side` (0: A's block sums, 1: B's): every
 * coefficient equal to the family's base coefficient times a sign that
 * depends only on its operand block (the case the family's formation
 * kernels take with compile-time coefficients, Sec. 2.1's sign orbit
 * flattened).  *is_sign (host) gets 1 or 0; when 1, *neg_mask (host) gets
 * bit b set for each block b (row-major over the side's grid of blocks, B's
 * transposed) whose sign is -1.  Returns FM_E_ARG for null pointers, a side
 * other than 0 or 1, or levels outside [1, 8]. */
int fm_scheme_sign_variant(const fm_scheme* s, int levels, int side, int* is_sign,
                           uint64_t* neg_mask);

/* Kernel timing for measurement.  While enabled (on != 0), every launch of
 * the kernel classes below made by this library is bracketed by two HIP
 * events recorded on the launch's own stream:
 *   "form_amax", "form_quant" (operand formation, both operands),
 *   "block_gemm" (FP8 block products), "recon" (reconstruction + error),
 *   "reference" (float64 reference).
 * fm_timing_read synchronizes on the recorded events and returns the number
 * of launches and their summed duration in milliseconds for one class;
 * fm_timing_reset drops all records.  Process-wide, not thread-safe; costs
 * two event records per launch while enabled. */
int fm_timing_enable(int on);
int fm_timing_reset(void);
int fm_timing_read(const char* kernel_class, int* launches, double* total_ms);

/* Waits for `hip_stream` and reports a deferred device-side error recorded
 * in `workspace` by earlier async calls (FM_E_NONFINITE), then clears it. */
int fm_status(void* workspace, size_t ws_bytes, void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* FM_H */
