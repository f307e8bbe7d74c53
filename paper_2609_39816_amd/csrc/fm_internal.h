// Internal declarations shared by the host code and the HIP kernels of
// libfm.  Not part of the public ABI (include/fm.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <string>
#include <vector>

#include "fm.h"

struct fm_scheme {
  int m = 0, n = 0, k = 0, R = 0;
  std::vector<double> U, V, W;  // R x (m*k), R x (k*n), R x (m*n)
};

// A prepared fast integer call (fm_int8_plan_create): shapes, the scheme's
// block grid and the workspace offsets of its tables and block sums.
struct fm_int8_plan {
  int M = 0, N = 0, K = 0, g = 0, h = 0, gm = 0, gn = 0, gk = 0, R = 0;
  int calls_per_group = 0, nsegs = 0, grid = 0, sa = 0, sb = 0;
  bool corr = false;          // the overflow correction (eq. (2))
  int qmax_a = 0, qmax_b = 0;  // bounds on the split parts q of the block sums
  char* ws = nullptr;
  size_t ws_bytes = 0;
  size_t flags = 0, zero = 0, coefa = 0, coefb = 0, segs = 0, segoff = 0, order = 0,
         order_off = 0, phase = 0, t = 0, s = 0, sn = 0, tr = 0, sr = 0, snr = 0;
};

namespace fm {

// ---------------------------------------------------------------- errors
int fail(int code, const std::string& msg);  // records msg, returns code
int host_failure() noexcept;                  // records a host failure, returns FM_E_NOMEM
void clear_error();
int hip_check(hipError_t e, const char* what);

// ------------------------------------------------------- scheme (host)
double brent_residual(const fm_scheme& s);
fm_scheme kron(const fm_scheme& a, const fm_scheme& b);
fm_scheme power(const fm_scheme& s, int levels);
// Inverse of an n x n row-major matrix (false if singular).
bool invert(const std::vector<double>& P, int n, std::vector<double>& out);

// Coefficient lists of one flattened scheme, in the orders the kernels use
// (struct of arrays: offsets, block indices, fp32 coefficients):
//   a: per product r, nonzero u in ascending row-major (i,l); idx = i*gk + l
//      (block index in A's gm x gk grid);
//   b: per product r, nonzero v in ascending row-major (l,j); idx = j*gk + l
//      (block index in B^T's gn x gk grid, where the kernels read B);
//   w: per product r, nonzero w with idx = i*gn + j, r-major (so every
//      output block receives its terms in ascending r).
struct Side {
  std::vector<int32_t> off;  // R + 1
  std::vector<int32_t> idx;
  std::vector<float> coef;
};
struct Lists {
  Side a, b, w;
};
void build_lists(const fm_scheme& flat, Lists& out);

// Pattern family of one side of a list (compiled specializations), or -1.
int match_pattern(int side, const Side& s, int R, int NB);
// Sign variants of a family with prefix-shared chains: true if every
// coefficient of one scheme's side list (A: 0, B: 1) of family `pattern` is
// the family's base coefficient times a sign that depends on its block
// alone (NB <= 64 blocks); *mask gets bit b set where block b's sign is -1.
// The shared chains then give every product's own chain (a shared entry has
// one block and one base value, hence one coefficient).
bool block_signs(int pattern, int side, const Side& s, int NB, uint64_t* mask);
// Family whose H pattern (pairs of products sharing a block of A and a
// block of C) equals one gauge's H support in compressed rows, or -1.
int match_h_pattern(const int32_t* rowptr, const uint16_t* cols, int R);
// Number of pattern families, and the name of family `id`.
int pattern_count();
const char* pattern_name(int id);

// Geometry of one evaluation.
struct Geometry {
  int gm, gk, gn, R;       // flattened grid and rank
  int M, N, K;             // full sizes
  int Mb, Nb, Kb;          // block sizes
  int NBa() const { return gm * gk; }
  int NBb() const { return gn * gk; }
  int NC() const { return gm * gn; }
};

// ------------------------------------------------------ kernel timing
// Kernel classes timed by fm_timing_*; timing_begin/timing_end bracket one
// launch with events on its stream when timing is enabled.
enum TimedClass { T_FORM_AMAX = 0, T_FORM_QUANT, T_BLOCK_GEMM, T_RECON, T_REFERENCE, T_COUNT };
void timing_begin(int cls, hipStream_t st);
void timing_end(int cls, hipStream_t st);

// ----------------------------------------------------- kernel launchers
// All launchers enqueue on `st` and return FM_OK or FM_E_HIP /
// FM_E_UNSUPPORTED.

// Fill n 32-bit words with `value`.
int launch_fill_u32(uint32_t* p, size_t n, uint32_t value, hipStream_t st);

// Bt (cols x rows) = X^T for X rows x cols, fp32.
int launch_transpose(const float* X, float* Xt, int rows, int cols, hipStream_t st);

// Operand formation over a chunk of gauges (G gauges, lists already on the
// device).  X: rows x cols fp32, grid gr x gc; off: G*(R+1) offsets into ent.
// mode 0: amax[g*R + r] = max(amax, bits(|T|)) (atomic max on uint bits);
// mode 1: codes[(g*R + r)*br*bc + ...] = FP8(T * q[g*R + r]).
struct FormArgs {
  const float* X;
  int rows, cols, gr, gc, br, bc;
  const int32_t* off;  // G*(R+1), absolute indices into idx/coef
  const int32_t* idx;
  const float* coef;
  int R, G;
  uint32_t* amax;   // mode 0
  const float* q;   // mode 1
  uint8_t* codes;   // mode 1
  int fmt;
  int per_row;      // 0: one amax/scale per (gauge, product); 1: one per
                    // group of entries, gran below, folded by atomics
  int gran = 1;     // with per_row: 1 one per row of the block-sum tensor as
                    // stored, at [(g R + r) br + x]; 2 one per row and 128
                    // consecutive entries, at [((g R + r) (bc/128) + y/128) br + x];
                    // 3 the same values rounded to bf16 first, one per 128 x 128
                    // block, at [((g R + r) (bc/128) + y/128) (br/128) + x/128]
  int trie = 0;     // every gauge is a sign variant of the family's base
                    // scheme (block_signs), so the prefix-shared chains apply
  const uint64_t* sgn = nullptr;  // with trie: per gauge, bit b set where the
                                  // coefficients of block b are the base's negated
};
// pattern: family id from match_pattern (side A or B), or -1 for the
// generic kernel.
int launch_form(const FormArgs& a, int mode, int pattern, int side, hipStream_t st);
// One side's FP8 codes of one chunk (aq, scales known) and per-tensor maxima
// of the next (am) in one pass; both of the family `pattern` (no generic
// form).  Returns 1, launching nothing, when the pair does not fit the
// merged kernel.
int launch_form_merged(const FormArgs& aq, const FormArgs& am, int pattern, int side,
                       hipStream_t st);
// Repairs: row exponents of A (As = A 2^-k row by row, up = 2^k), and the
// joint rounding of B's bf16 block sums (a is B's FormArgs with gran 3;
// codes into a.codes; qS, dS the block scales; H of every gauge in
// compressed rows: hv values, hc columns (G x R x R each), hp pointers
// (G x (R + 1)); pattern: the family id shared by all three sides of every
// gauge, or -1 for the generic kernel).
int launch_row_repair(const float* A, int M, int K, float* As, float* up, hipStream_t st);
int launch_joint_round(const FormArgs& a, const float* qS, const float* dS, const float* hv,
                       const uint16_t* hc, const int32_t* hp, int pattern, hipStream_t st);

// Scales from amax: for i < n: q[i] = FMAX/amax, d[i] = amax/FMAX (1, 1 for
// amax = 0); a non-finite amax sets *flag |= 1.
int launch_scales(const uint32_t* amax, float* q, float* d, int n, int fmt, uint32_t* flag,
                  hipStream_t st);

// Process-wide arithmetic of the block products (FM_ACC_BF16 / FM_ACC_FP8).
int set_block_product_arith(int a);

// Batched FP8 block products: Mout[b] = ((Tq[b] Sq[b]^T) * dT) * dS with
// dT = dT[b], dS = dS[b] (FM_SCALE_TENSOR) or dT[b*Mb + x], dS[b*Nb + z]
// (FM_SCALE_ROWCOL).
// out_bf16 (group scales only): the products, bf16 values, are stored as
// bf16 (2 bytes each, uint16_t at Mout) instead of fp32.
// tiled (tensor scales, whole tiles of the kernel that runs, see
// block_gemm_tile_rows): each product is stored tile by tile
// (tile_layout_position below) instead of row by row.
int launch_block_gemm(const uint8_t* Tq, const uint8_t* Sq, const float* dT, const float* dS,
                      float* Mout, int batch, int Mb, int Nb, int Kb, int fmt, int scale_mode,
                      hipStream_t st, bool out_bf16 = false, bool tiled = false);

// Rows of the output tile of the block-product kernel launch_block_gemm
// runs for these arguments: 512 (gemm_wide_kernel: bf16 arithmetic, tensor
// or row/column scales, fp32 products, Mb a multiple of 512, Nb of 128, Kb
// of 64), 256 (gemm_dma_kernel: Kb a multiple of 128), 0 otherwise.  Tiles
// are 128 columns wide.
int block_gemm_tile_rows(int Mb, int Nb, int Kb, int scale_mode, bool out_bf16);

// The tiled layout of a product block (Mb x Nb, whole TR x 128 tiles, TR =
// 256 or 512): the 16-byte piece p (4 consecutive columns of one row) sits
// at byte 16 p, t being the tile (row-major over the block's tiles).  For
// TR = 256, p = (((t 8 + w) 4 + i) 4 + j) 64 + 4 l + c with the 64 x 64
// quarter w = 2 (row / 64 % 4) + (column / 64 % 2), i = row / 16 % 4, j =
// column / 16 % 4, l = row % 16 and c = column / 4 % 4.  For TR = 512, p =
// ((((t 4 + w) 4 + i) 4 + j) 4 + g) 64 + 32 h + r with the 128-row quarter
// w = row / 128 % 4, i = row / 32 % 4, r = row % 32, j = column / 32 % 4,
// g = column / 8 % 4 and h = column / 4 % 2.  The block-product kernel
// stores each wave's piece of a tile as one contiguous kilobyte; the
// reconstruction reads pieces in this order.
__host__ __device__ inline void tile_layout_position(int p, int Nb, int TR, int& row, int& col) {
  const int tn = Nb / 128;
  if (TR == 512) {
    const int r = p & 31, h = (p >> 5) & 1, g = (p >> 6) & 3, j = (p >> 8) & 3;
    const int i = (p >> 10) & 3, w = (p >> 12) & 3;
    const int t = p >> 14, tm = t / tn;
    row = tm * 512 + w * 128 + i * 32 + r;
    col = (t - tm * tn) * 128 + j * 32 + 8 * g + 4 * h;
  } else {
    const int l = (p >> 2) & 15, c = p & 3;
    const int j = (p >> 6) & 3, i = (p >> 8) & 3, w = (p >> 10) & 7;
    const int t = p >> 13, tm = t / tn;
    row = tm * 256 + (w >> 1) * 64 + i * 16 + l;
    col = (t - tm * tn) * 128 + (w & 1) * 64 + j * 16 + 4 * c;
  }
}

// Reconstruction + error: for gauge g < G, C_g = sum_r w M_{g,r}; if C is not
// null it is written (G must be 1); if Cref is not null, partial sums of
// (C - Cref)^2 go to partial[g*nblk + blk].  Returns nblk through *nblk_out.
struct ReconArgs {
  const float* Mprod;  // G x R x Mb x Nb (fp32, or bf16 when prod_bf16)
  const int32_t* off;  // G*(R+1)
  const int32_t* idx;
  const float* coef;
  int R, G, gm, gn, Mb, Nb, N;
  float* C;            // optional
  const double* Cref;  // optional
  double* partial;     // G x nblk (if Cref)
  const float* rowscale = nullptr;  // optional: output row i*Mb + x times rowscale[i*Mb + x]
  int prod_bf16 = 0;  // products stored as bf16 (uint16_t at Mprod; group scales)
  int tiled = 0;      // products in the tiled layout of tiles of this many rows
                      // (256 or 512; fp32, 4 positions per thread), or 0
};
// Positions per thread in the reconstruction kernels (4 or 1) and the
// number of workgroups per gauge (one position group per thread).
inline int recon_width(const ReconArgs& a) {
  return (a.gm * a.gn <= 16 && a.Nb % 4 == 0 && a.N % 4 == 0) ? 4 : 1;
}
int recon_blocks(const ReconArgs& a);
int launch_recon(const ReconArgs& a, int pattern, hipStream_t st);

// out[g] = sum_{b < nblk} partial[g*nblk + b] (fixed order), g < G.
int launch_reduce_rows(const double* partial, int nblk, int G, double* out, hipStream_t st);

// Integer path (fm_int8.hip).
int launch_i8_quantize(const float* X, int rows, int K, int g, int b, int8_t* codes, float* d,
                       uint32_t* flag, hipStream_t st);
int launch_i8_form(const int8_t* X, int rows, int K, int gp, int gk, int h, int R,
                   const int8_t* coef, int stride, int8_t* out, int8_t* outn, int8_t* outR,
                   int8_t* outnR, int qmax, uint32_t* flag, hipStream_t st);
// Tiles of the fast integer kernel, and their longest-first assignment to
// workgroups (returns the grid; order holds every workgroup's tiles, off its
// grid + 1 offsets).
long long i8_fast_tiles(int gm, int gn, int Mb, int Nb);
int i8_fast_schedule(int gm, int gn, int Mb, int Nb, const std::vector<int>& block_steps,
                     std::vector<int32_t>& order, std::vector<int32_t>& off);
int launch_i8_gemm(bool fast, const int8_t* A, const int8_t* B, const int8_t* Bn,
                   const int8_t* zero, const float* dA, const float* dB, float* out,
                   const int32_t* segs, const int32_t* seg_off, int nsegs, const int32_t* order,
                   const int32_t* order_off, int grid, int M, int N, int K, int g, int gm, int gn,
                   int R, int h, int calls_per_group, const int8_t* AR, const int8_t* BR,
                   const int8_t* BnR, const int32_t* phase, hipStream_t st);

// Float64 reference C = A B.
int launch_reference_f64(const float* A, const float* B, double* C, int M, int N, int K,
                         hipStream_t st);

// Error statistics partials over n elements: per block (err_sq, ref_sq,
// max_abs) into partial[3*blk...]; nblk blocks.
int error_stats_blocks(size_t n);
int launch_error_stats(const float* C, const double* Cref, size_t n, double* partial,
                       hipStream_t st);
int launch_error_finalize(const double* partial, int nblk, double* out3, hipStream_t st);

// Diagnostic encoder: codes for n fp32 values with the kernels' encoder.
int launch_fp8_encode(const float* x, uint8_t* out, size_t n, int fmt, int impl, hipStream_t st);
int launch_bf16_round(const float* x, float* out, size_t n, int impl, hipStream_t st);

}  // namespace fm
