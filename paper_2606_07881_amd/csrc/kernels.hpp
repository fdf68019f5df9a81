// Host-side launchers of the stage kernels. Every pointer is device memory;
// every launcher enqueues on `st` and returns the launch status.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace paci {

enum DType { DT_F32 = 0, DT_BF16 = 1 };

// Dropout at one site of one micro-batch: key (seed, mb), site word
// (block << 2) | site (0 embedding, 1 attention probabilities, 2 projection
// output, 3 FFN output); an element is kept when its 16-bit Philox value is
// >= thr (thr 0: no dropout) and then scaled by `scale` = 1 / (1 - p).
struct DropArgs {
  uint32_t seed = 0, mb = 0, word = 0, thr = 0;
  float scale = 1.f;
};

// ---- GEMM: C[m][n] = sum_k A(m, k) B(k, n) -------------------------------------------
// Operand layouts (ld in elements):
//   GEMM_NT (forward, y = x W^T):      A(m,k) = A[m*lda + k], B(k,n) = B[n*ldb + k]
//   GEMM_NN (input gradient, dX = dY W): A(m,k) = A[m*lda + k], B(k,n) = B[k*ldb + n]
//   GEMM_TN (weight gradient, dW = dY^T X): A(m,k) = A[k*lda + m], B(k,n) = B[k*ldb + n]
enum GemmLayout { GEMM_NT = 0, GEMM_NN = 1, GEMM_TN = 2 };
// Fused epilogues (acc is the fp32 sum for one (m, n)):
//   EPI_STORE      C = acc
//   EPI_BIAS       C = acc + bias[n]
//   EPI_BIAS_RES   C = acc + bias[n] + aux[m*ld_aux + n]        (residual add)
//   EPI_BIAS_GELU  u = acc + bias[n];  C = gelu'(u);  C2 = gelu(u)  (FFN up-projection)
//   EPI_GELU_GRAD  C = acc * aux[m*ld_aux + n]  (aux = gelu'(u); FFN down-projection dgrad)
//   EPI_ACC        Cf32 += acc  (plain read-modify-write; one split only)
//   EPI_ATOMIC     Cf32 += acc  (atomic add; any number of splits)
// Softmax cross-entropy over the output columns (bf16 GEMM_NT only, one split):
//   EPI_CE_STATS   nothing stored in C; per row m and 64-column group g (columns
//                  64g .. 64g+63 below N): ce_part[2 (m ld_part + g) + {0, 1}] =
//                  {max, sum exp(acc - max)}; ce_zt[m] = acc at column row_tgt[m]
//   EPI_CE_GRAD    C = alpha * (exp(acc - row_lse[m]) - [n == row_tgt[m]])  (bf16)
enum GemmEpi { EPI_STORE = 0, EPI_BIAS, EPI_BIAS_RES, EPI_BIAS_GELU, EPI_GELU_GRAD, EPI_ACC, EPI_ATOMIC, EPI_CE_STATS,
               EPI_CE_GRAD };

// Grouped weight gradients (bf16, one launch): problem p adds
// C_p[M_p, N_p] (fp32, row stride N_p) += A_p^T B_p over K contracted rows, with
// A_p [K, M_p] and B_p [K, N_p] bf16 row-major (the layer's output gradient and
// its input, GEMM_TN). Every output tile belongs to one workgroup, so the sum is
// a plain read-modify-write (no split, no atomics). `probs` is device memory
// holding n problems; tile0 is the problem's first workgroup, a multiple of 8
// (wgrad_group_tiles gives each problem's count; workgroups past a problem's
// tiles exit). M_p, N_p, K multiples of 8 and 16-byte aligned operands.
// xcd_m: 0, or the number of row bands of the problem's tile grid when it is
// split into 8 equal blocks (xcd_m bands x 8 / xcd_m column bands), one per XCD
// (see wgrad_group_xcd_m).
struct WgradProblem {
  const void* A;
  const void* B;
  float* C;
  int M, N, tile0, xcd_m;
};
struct GemmArgs {
  const void* A; int64_t lda;
  const void* B; int64_t ldb;
  int M, N, K;
  void* C; int64_t ldc;
  const float* bias;
  const void* aux; int64_t ld_aux;
  void* C2;
  const void* zeros;  // >= 16 bytes of device zeros (bf16 path: source of out-of-range tile slots)
  float* colsum = nullptr;  // optional: += column sums of the output C (non-accumulating epilogues, bf16 path)
  // optional (TN layout, bf16 path): operand B's contracted rows come in segments of
  // seg_rows rows (a multiple of 64); segment s starts at B + seg_stride elements
  // times ((seg_first + s) % seg_count), each with row stride ldb
  int64_t seg_rows = 0, seg_stride = 0;
  int seg_first = 0, seg_count = 1;
  // cross-entropy epilogues (see GemmEpi)
  const int32_t* row_tgt = nullptr;
  const float* row_lse = nullptr;
  float* ce_part = nullptr;
  int64_t ld_part = 0;
  float* ce_zt = nullptr;
  float alpha = 1.f;
  // grouped weight gradients (gemm_wgrad_grouped): device problem table
  const WgradProblem* group = nullptr;
  int group_n = 0;
  int* nonfinite = nullptr;   // fp32 EPI_ACC / EPI_STORE: set to 1 if an element written is not finite
};
// bf16 operands: K-major vectors that straddle K read the memory just past K,
// which must hold zeros (true when K % 8 == 0, or for zero-padded rows).

// Two tile shapes: wide = 256 x 256 (eight 128 x 64 wave tiles), else 256 x 128.
// overwrite: C_p = A_p^T B_p instead of +=; nonfinite (nullable): set to 1 (a plain
// store) if any element written is NaN or infinite.
int wgrad_group_tiles(int M, int N, bool wide);
// Workgroup w of a problem runs on XCD w % 8. Each XCD streams the operand
// panels of the tiles it runs through its own L2, so the launch gives each XCD
// one block of the tile grid: the split of the grid into 8 equal blocks (xcd_m
// row bands) that reads the fewest panel bytes per XCD, or 0 if the grid does
// not split evenly (then the generic XCD-aware order applies). K contracted rows.
int wgrad_group_xcd_m(int M, int N, int K, bool wide);
// How many leading problems (of n, shapes M[p] x N[p]) go on wide tiles, the rest
// in a second launch on 256 x 128 tiles: the split with the fewest rounds of
// workgroups over the CUs, a wide tile costing 1.8 narrow ones (measured); the
// whole list on narrow tiles when no split does better.
int wgrad_group_wide(const int* M, const int* N, int n);
hipError_t gemm_wgrad_grouped(const WgradProblem* probs, int n, int total_tiles, int K, const void* zeros,
                              bool overwrite, bool wide, int* nonfinite, hipStream_t st);

// dtype: element type of A, B, aux and of C/C2 unless out_f32 (then C is float).
// splits > 1 is only valid with EPI_ATOMIC.
hipError_t gemm(DType dt, bool out_f32, GemmLayout lay, GemmEpi epi, const GemmArgs& a, int splits, hipStream_t st);
// Tile edge used by gemm(); callers size split-K against it.
// Split-K count the fp32-accumulating TN product (weight gradients) should use.
int gemm_acc_splits(DType dt, int M, int N, int K);
// Testing hook: force one kernel configuration for bf16 calls (0: register-staged 128x128;
// direct-to-LDS pipelines 10: 256x128 x 3 stages (the default), 11: 128x128 x 4, 12: 128x256 x 3).
void gemm_set_tile_override(int cfg);

// ---- causal attention over the fused projection qkv [T, 3d] --------------------------
// Forward: o [T, d]; lse2 [mu*H*S] = log2-sum-exp2 of the scaled scores in log2 units.
hipError_t attn_fwd(DType dt, const void* qkv, void* o, float* lse2, int mu, int S, int H, int dh, const DropArgs& drop,
                    hipStream_t st);
// Backward: D = rowsum(dO * O) per (b, h, query), then dK, dV and dQ into dqkv [T, 3d].
// Dbuf is workspace of attn_bwd_workspace_floats() floats. gbias (optional, fp32 [3d]):
// += the column sums of dqkv, i.e. the gradient of the qkv projection's bias.
int64_t attn_bwd_workspace_floats(DType dt, int mu, int S, int H);
hipError_t attn_bwd(DType dt, const void* qkv, const void* o, const void* dO, const float* lse2, float* Dbuf,
                    void* dqkv, float* gbias, int mu, int S, int H, int dh, const DropArgs& drop, hipStream_t st);

// ---- LayerNorm -----------------------------------------------------------------------
// n = (x - mean) * rstd * gamma + beta, per row of d; xcopy (optional) receives x.
hipError_t layernorm_fwd(DType dt, const void* x, void* n, float* mean, float* rstd, const float* gamma,
                         const float* beta, void* xcopy, int rows, int d, float eps, hipStream_t st);
// dx = res + rstd * (g - mean(g) - xhat * mean(g * xhat)), g = dn * gamma (res optional);
// Ggamma += sum_rows dn * xhat, Gbeta += sum_rows dn and, if Gdx is not null,
// Gdx += sum_rows dx (fp32 atomics; the column sums are one pass after dx).
hipError_t layernorm_bwd(DType dt, const void* dn, const void* x, const float* mean, const float* rstd,
                         const float* gamma, const void* res, void* dx, float* Ggamma, float* Gbeta, float* Gdx,
                         int rows, int d, hipStream_t st);

// ---- dropout at the element-wise sites ----------------------------------------------------
// out = res + z * keep * scale over rows x cols (cols % 8 == 0; res nullable:
// out = z * keep * scale; out may alias z). Element e = r * cols + c.
hipError_t dropout_fwd(DType dt, const void* z, const void* res, void* out, int rows, int cols, const DropArgs& drop,
                       hipStream_t st);

// ---- column sums accumulated into fp32 (bias gradients) ---------------------------------
// G[c] += sum_r Y[r*ld + c], c < ncols (fp32 atomics).
hipError_t colsum_acc(DType dt, const void* Y, int64_t ld, int rows, int ncols, float* G, hipStream_t st);

// ---- first stage: token + position embedding ----------------------------------------------
// x[b*S + s] = wte[ids[b*S + s]] + wpe[s] (fp32 tables, x in the stage dtype).
hipError_t embed_fwd(DType dt, const int32_t* ids, const float* wte, const float* wpe, void* x, int mu, int S, int d,
                     int V, hipStream_t st);
// Gwte[ids[t]] += dx[t] (atomic; repeated ids add), Gwpe[s] += sum_b dx[b*S + s].
// Ids outside [0, V) read as a zero row and receive no gradient.
hipError_t embed_bwd(DType dt, const int32_t* ids, const void* dx, float* Gwte, float* Gwpe, int mu, int S, int d,
                     int V, hipStream_t st);

// ---- last stage: softmax cross-entropy over fp32 logits z [T, ldz] (V valid columns) --------
// lse[t] = logsumexp(z[t, :V]); loss_out (one float) = mean_t (lse[t] - z[t, tgt[t]]).
// `part` needs ce_part_floats(T) floats.
hipError_t ce_fwd(const float* z, int64_t ldz, const int32_t* tgt, float* lse, float* loss_out, float* part, int T,
                  int V, hipStream_t st);
int64_t ce_part_floats(int T);
// From the EPI_CE_STATS partials of a [T, V] logit product (ngroups = ceil(V / 64)
// groups of 64 columns per row, row stride ld_part float2): lse[t] and the mean
// loss over t of lse[t] - zt[t] into loss_out (a target outside [0, V) gives NaN).
// `part_loss` needs ce_part_floats(T) floats.
hipError_t ce_combine(const float* ce_part, int64_t ld_part, int ngroups, const float* zt, const int32_t* tgt, int V,
                      float* lse, float* loss_out, float* part_loss, int T, hipStream_t st);
// dz[t, v] = scale * (exp(z[t, v] - lse[t]) - [v == tgt[t]]) in the stage dtype; columns
// V .. ldz-1 are written as zero.
hipError_t ce_bwd(DType dt, const float* z, int64_t ldz, const int32_t* tgt, const float* lse, void* dz, int T, int V,
                  float scale, hipStream_t st);

// ---- AdamW over the flat parameter arena --------------------------------------------------
// ctl: 4 device ints {G not finite, updates applied, updates skipped, unused}.
// adamw_guard: ctl[0] = 1 if any of the n values of G is not finite (else ctl[0]
// is left as is); adamw_guard_ranges: the same over ranges[i] = {begin, end}
// (elements, multiples of 4), one workgroup per range.
// adamw: one launch over every parameter, one workgroup per table entry:
//   {begin, end, flags, 0}: the elements [begin, end) of one tensor (multiples of 4);
//   {offset, r0 << 16 | c0, flags | ADAMW_TILE, rows << 16 | cols}: the 64 x 64 tile at
//   (r0, c0) of the matrix [rows, cols] at offset (rows, cols multiples of 8), whose
//   bf16 values also go transposed into theta_bf16T ([cols, rows] at the same offset).
// Unless ctl[0] is set: with t = ctl[1] + 1, theta <- theta * (1 - lr_t * wd) where
// ADAMW_DECAY, then the Adam direction with bias correction of step t; m, v updated;
// theta_bf16 (nullable) rewritten. G is cleared either way where ADAMW_CLEAR_G.
// lr_t follows the schedule (lr_total = 0: lr).
// adamw_ctl: mode 0 clears ctl[0]; 1 counts the update (ctl[1] or ctl[2]) and clears
// ctl[0]; 2 clears all of ctl.
enum { ADAMW_DECAY = 1, ADAMW_CLEAR_G = 2, ADAMW_TILE = 4 };
struct AdamwArgs { float lr, beta1, beta2, eps, weight_decay, lr_min_ratio; int lr_warmup, lr_total; };
hipError_t adamw_guard(const float* G, int64_t n, int* ctl, hipStream_t st);
hipError_t adamw_guard_ranges(const float* G, const int2* ranges, int nranges, int* ctl, hipStream_t st);
hipError_t adamw(float* theta, float* G, float* m, float* v, void* theta_bf16, void* theta_bf16T, const int4* chunks,
                 int nchunks, const AdamwArgs& a, const int* ctl, hipStream_t st);
hipError_t adamw_ctl(int* ctl, int mode, hipStream_t st);
// p[i] = v for i < n (a kernel: no memset node when the stream is captured).
hipError_t fill_f32(float* p, int64_t n, float v, hipStream_t st);
// dst (bf16) = round-to-nearest-even(src), n elements.
hipError_t f32_to_bf16(const float* src, void* dst, int64_t n, hipStream_t st);
// dst [cols, rows] = src [rows, cols]^T for 16-bit elements; rows, cols multiples of 8.
hipError_t transpose16(const void* src, void* dst, int rows, int cols, hipStream_t st);

}  // namespace paci
