/*
 * patchkv.h - C ABI of the PatchKV context-loading path on one MI355X (gfx950).
 *
 * PatchKV (weight-space compensation of a compressed KV cache) builds, for every
 * transformer block, a closed-form weight patch that makes the block's output
 * under a compressed cache match its output under the full cache on a set of
 * context-derived reference queries (Sec. 2.2-2.3, Alg. 1 of the paper). Per
 * block the path is:
 *
 *   attend_full        reference queries attend over the full cache     (Alg. 1, teacher forward)
 *   attend_compressed  the same queries over the compressed cache       (Alg. 1, student forward)
 *   compute_targets    T = (O_f - O_c) W + rho (O_f - O_c)              (Eq. 5)
 *   accumulate_normal_eq  G (+)= Xc^T Xc, C (+)= Xc^T (Yf - Yc)          (Eq. 9)
 *   solve_patch        (G + lambda I) dW = C by blocked Cholesky         (Eq. 6, 8; Eq. 7 adaptive lambda)
 *   compute_layer_patch   all of the above for one block
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Orientation: activations are rows (one token per row). With X = the
 *   compressed-cache features (the paper's H') and T the targets, G = X^T X is the
 *   paper's S_H, C = X^T T is the transpose of its S_T, and the returned
 *   dW [d_in][d_out] is the transpose of its column-vector Delta W; the patched
 *   projection is X (W + dW).
 * - All tensor pointers are DEVICE pointers to contiguous row-major arrays owned
 *   by the caller. The library never allocates device memory and never frees
 *   caller memory; scratch space is the caller's `workspace` (size from the
 *   matching *_workspace_bytes query, 256-byte aligned start recommended; at least
 *   `workspace_bytes` bytes must be valid).
 * - Calls are asynchronous: kernels are enqueued on `stream` (a hipStream_t; NULL
 *   means the default stream) and the call returns. Outputs are valid once the
 *   stream has completed. Inputs must stay valid and unmodified until then.
 * - bf16 data are raw bfloat16 values (uint16 bit patterns); f32 are IEEE floats;
 *   f64 are IEEE doubles.
 * - Every argument is validated on the host before anything is enqueued. On any
 *   error nothing is enqueued and a non-zero patchkv_status is returned.
 *   PATCHKV_E_HIP means a HIP launch reported an error (work enqueued earlier in
 *   the same call may have run).
 * - Calls that share a workspace, or write the same outputs, race unless they are
 *   ordered on one stream.
 */
#ifndef PATCHKV_H
#define PATCHKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PATCHKV_OK = 0,
  PATCHKV_E_NULL = 1,        /* a required pointer is NULL */
  PATCHKV_E_SHAPE = 2,       /* a size is <= 0, too large, or inconsistent (e.g. Hq % Hkv != 0) */
  PATCHKV_E_DTYPE = 3,       /* unknown or unsupported dtype code for this argument */
  PATCHKV_E_VALUE = 4,       /* a scalar is out of range (lambda <= 0, scale <= 0, rho not 0/1, ...) */
  PATCHKV_E_WORKSPACE = 5,   /* workspace NULL or smaller than the matching *_workspace_bytes */
  PATCHKV_E_UNSUPPORTED = 6, /* head_dim other than 64 or 128 */
  PATCHKV_E_HIP = 7,         /* the HIP runtime reported an error */
  PATCHKV_E_SCRATCH = 8      /* more scratch needed than the fixed buffer of a *_noalloc call holds */
} patchkv_status;

typedef enum {
  PATCHKV_F32 = 0,
  PATCHKV_BF16 = 1,
  PATCHKV_F64 = 2
} patchkv_dtype;

typedef enum {
  PATCHKV_RIDGE_ABSOLUTE = 0, /* lambda is the ridge coefficient itself (Eq. 6) */
  PATCHKV_RIDGE_ADAPTIVE = 1, /* lambda is lambda_0; ridge = lambda_0 ||G||_F^2 / tr(G) (Eq. 7) */
  /* lambda is lambda_0; ridge = lambda_0 tr(G) / d_in, the mean eigenvalue: the
   * trace-mean scaling that the paper's ridge-scaling ablation compares with Eq. 7 */
  PATCHKV_RIDGE_TRACE_MEAN = 2,
  /* Flags OR-ed into any mode, used by the F32 solve only (F64 ignores them), at most
   * one of them. By default the F32 solve keeps the paper's FP32 patch construction
   * (App. B.1): every fp32 operand of a block product is split into three bf16 pieces
   * and six bf16 MFMA products are summed in fp32, as exact as an fp32 multiply
   * (about 2^-24 relative per product). */
  PATCHKV_SOLVE_EXACT_F32 = 16, /* exact fp32 products on fp32 MFMA (slower) */
  PATCHKV_SOLVE_FAST_BF16 = 32  /* two bf16 pieces, three products: about 2^-16 relative
                                   per product, faster; below FP32 grade */
} patchkv_ridge_mode;

/* Index sets of an eviction-style compressed cache (the `idx_mode` argument).    */
/* KVzip, the paper's eviction method, scores KV pairs with global head scoring  */
/* (App. B.1; Sec. 3.1), so each KV head keeps its own tokens, and not           */
/* necessarily as many as the others.                                          */
typedef enum {
  PATCHKV_IDX_SHARED = 0,  /* idx [B] int32: one set of cache rows for every KV head */
  PATCHKV_IDX_PER_HEAD = 1 /* idx [Hkv][B] int32: KV head g keeps rows idx[g][0..B) */
} patchkv_idx_mode;

/* Shared by the compressed-cache calls (attend_compressed, attend_chunk,
 * attend_cache, compute_layer_patch):
 *  - counts (optional, device int32 [Hkv], 4-byte aligned): KV head g's compressed
 *    cache is only its first counts[g] entries (idx[g][0..counts[g]) per head, the
 *    first counts[g] entries of a shared set, or of the rows of a contiguous cache);
 *    NULL means B for every head. Each count must lie in [1, B]; a count outside is
 *    clamped into that range and reported through info.
 *  - Every index entry a head uses must lie in [0, N). An entry outside reads as a
 *    zero row (no memory outside the cache is touched) and is reported.
 *  - info (device int32, 4-byte aligned; optional for the attend_* calls): written 0
 *    when every used entry and every count is in range; otherwise -(1 + c) for the
 *    smallest offending code c, where an entry at flat position q of idx (q = b for
 *    a shared set, g * B + b per head) has code q and the count of head g has code
 *    E + g, E being the number of entries in idx (B shared, Hkv * B per head, 0 with
 *    no idx). compute_layer_patch reports such an input error in its info word in
 *    place of the solve's result.                                              */

/* Storage of a cache's keys and values (patchkv_attend_cache). */
typedef enum {
  PATCHKV_KV_PLAIN = 0,  /* K, V in the call's dtype */
  PATCHKV_KV_MXINT8 = 1, /* int8 q and one int8 power-of-two exponent e per 32 channels: q * 2^e */
  PATCHKV_KV_MXINT4 = 2  /* the same with int4 q in [-8, 7], two per byte, even channel low */
} patchkv_kv_format;

/* Human-readable name of a status code (static string, never NULL). */
const char* patchkv_status_string(int status);

/* Library version as 10000*major + 100*minor + patch. */
int patchkv_version(void);

/* ------------------------------------------------------------------------- */
/* Attention of reference queries over a cache (Sec. 2.2 teacher/student       */
/* forward passes; Alg. 1).                                                    */
/*                                                                           */
/* O[m, h*dh + j] = sum_n softmax_n(scale * <Q[m,h,:], K[g,n,:]>) V[g,n,j],    */
/* g = floor(h / (Hq/Hkv)) (grouped-query attention), over all cache entries   */
/* n, with no mask (rotary embeddings already applied to Q and K).             */
/*                                                                           */
/* dtype: PATCHKV_BF16 (bf16 MFMA products, fp32 softmax and accumulation) or  */
/*        PATCHKV_F32 (fp32 throughout).                                       */
/* Q  [M][Hq][dh]      queries (dtype)                                          */
/* K, V [Hkv][N][dh]   full cache (dtype)                                       */
/* O  [M][Hq*dh]       float output, written (not accumulated)                  */
/* Limits: 1 <= Hkv <= Hq, Hq % Hkv == 0, dh in {64, 128}, M >= 1, N >= 1,      */
/*         M*Hq and N below 2^31, and for bf16 N*dh*2 below 2^32 (N < 2^24 at   */
/*         dh = 128); scale > 0 and finite.                                    */
/* Workspace: bf16 needs a transposed copy of V (Hkv*N*dh bf16, laid out in     */
/*   32-key tiles) plus a few bytes per work item; both dtypes need partial     */
/*   results when the key range is split (small M).                             */
/* ------------------------------------------------------------------------- */
size_t patchkv_attend_workspace_bytes(int dtype, int64_t M, int64_t N, int Hq, int Hkv, int dh);

int patchkv_attend_full(int dtype, const void* Q, const void* K, const void* V,
                        int64_t M, int64_t N, int Hq, int Hkv, int dh, float scale,
                        float* O, void* workspace, size_t workspace_bytes, void* stream);

/* The same attention over a compressed cache of B entries (Alg. 1, student     */
/* forward; Sec. 2.1 compressed cache C_b).                                     */
/*  - idx != NULL: eviction subset. K, V are the FULL cache [Hkv][N][dh]; the    */
/*    compressed cache of KV head g is rows idx[b] (PATCHKV_IDX_SHARED, idx [B]) */
/*    or idx[g][b] (PATCHKV_IDX_PER_HEAD, idx [Hkv][B]) of K[g], V[g], gathered  */
/*    on the fly.                                                              */
/*  - idx == NULL: synthesized cache. K, V are [Hkv][B][dh]; N is ignored;       */
/*    idx_mode must be PATCHKV_IDX_SHARED.                                     */
/* counts and info as described above patchkv_kv_format (info may be NULL).     */
/* The workspace size is patchkv_attend_workspace_bytes(dtype, M, B, ...).       */
int patchkv_attend_compressed(int dtype, const void* Q, const void* K, const void* V,
                              const int32_t* idx, int idx_mode, const int32_t* counts,
                              int64_t M, int64_t N, int64_t B, int Hq, int Hkv, int dh,
                              float scale, float* O, int32_t* info, void* workspace,
                              size_t workspace_bytes, void* stream);

/* Allocation-free variant of patchkv_attend_compressed, for callers that       */
/* cannot allocate device memory or bring a workspace: code under HIP graph     */
/* capture, tight serving loops (e.g. re-patching after each online compaction  */
/* of the cache), harnesses that forbid hipMalloc. Same arguments and results   */
/* as patchkv_attend_compressed, without the workspace: the scratch (V^T tiles, */
/* fast-path flags, split-key partials) lives in one fixed device buffer of     */
/* PATCHKV_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on */
/* until the process ends. The call allocates nothing (no hipMalloc, no         */
/* allocating library routine). A shape whose scratch                           */
/* (patchkv_attend_workspace_bytes(dtype, M, B, ...)) exceeds the buffer returns */
/* PATCHKV_E_SCRATCH before anything is enqueued. Every call on one GPU shares  */
/* that GPU's buffer: calls that overlap on one GPU (other streams, other host  */
/* threads) race; calls ordered on one stream do not. The first call on a       */
/* device looks up the buffer's device address (PATCHKV_E_HIP if that fails).   */
#define PATCHKV_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
int patchkv_attend_compressed_noalloc(int dtype, const void* Q, const void* K, const void* V,
                                      const int32_t* idx, int idx_mode, const int32_t* counts,
                                      int64_t M, int64_t N, int64_t B, int Hq, int Hkv, int dh,
                                      float scale, float* O, int32_t* info, void* stream);

/* ------------------------------------------------------------------------- */
/* Attention of one reference chunk over a cache plus the chunk's own causal    */
/* prefix (Sec. 2.3, chunked query encoding; Alg. 1, loop over reference       */
/* chunks). The chunk's M tokens are the queries; token m attends over every    */
/* cache entry and over the chunk's own entries 0..m (itself included), never   */
/* over other chunks:                                                          */
/*   O[m, h*dh + j] = sum_e softmax_e(scale * <Q[m,h,:], key_e>) value_e[j],    */
/*   e over the n_cache cache entries of KV head g = floor(h / (Hq/Hkv)) and    */
/*   the own entries Ks[g, 0..m, :] / Vs[g, 0..m, :].                           */
/* The cache:                                                                  */
/*  - idx != NULL: K, V [Hkv][n_src][dh] and the cache is rows idx[0..n_cache)  */
/*    (idx_mode SHARED) or idx[g][0..n_cache) (PER_HEAD) of head g (eviction    */
/*    subset, gathered on the fly; entries in [0, n_src)).                      */
/*  - idx == NULL: rows 0..n_cache of K, V [Hkv][n_src][dh] (n_cache <= n_src); */
/*    n_cache = n_src is the full cache, a synthesized cache is passed as is.   */
/* counts and info as described above patchkv_kv_format, with B = n_cache and  */
/* N = n_src (info may be NULL).                                               */
/* Ks, Vs [Hkv][M][dh] (dtype): the chunk's own keys and values.                */
/* p_terms: 1 = P enters the P V product rounded to bf16 (as attend_full),      */
/*          2 = as a two-term bf16 split (as attend_compressed); f32 ignores it.*/
/* Limits as patchkv_attend_full with N = n_cache, plus n_src and M within the  */
/* same row limits. When the cache is split into key ranges (small M), the own  */
/* entries go with the last range.                                             */
/* Workspace: patchkv_attend_chunk_workspace_bytes(dtype, M, n_cache, ...):     */
/*   that of patchkv_attend_full for (M, n_cache) plus, for bf16, a transposed  */
/*   copy of the own values (Hkv*ceil(M/32)*32*dh bf16).                        */
/* ------------------------------------------------------------------------- */
size_t patchkv_attend_chunk_workspace_bytes(int dtype, int64_t M, int64_t n_cache, int Hq, int Hkv,
                                            int dh);

int patchkv_attend_chunk(int dtype, const void* Q, const void* K, const void* V,
                         const int32_t* idx, int idx_mode, const int32_t* counts, int64_t n_src,
                         int64_t n_cache, const void* Ks, const void* Vs, int64_t M, int Hq,
                         int Hkv, int dh, float scale, int p_terms, float* O, int32_t* info,
                         void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Attention over a compressed cache in the storage formats of Sec. 3.1 and     */
/* App. C (attention-matching logit bias; quantized KV caches):              */
/*   O[m, h*dh + j] = sum_n softmax_n(scale <Q[m,h,:], K_n> + bias[g, n]) V_n[j] */
/* over the n_cache entries of KV head g = floor(h / (Hq/Hkv)).                 */
/*  - kv_format PATCHKV_KV_PLAIN: K, V [Hkv][n_src][dh] in dtype; Ke, Ve NULL.   */
/*  - PATCHKV_KV_MXINT8: K, V int8 [Hkv][n_src][dh]; Ke, Ve int8                */
/*    [Hkv][n_src][dh/32]; entry value q * 2^e (exact in bf16).                 */
/*  - PATCHKV_KV_MXINT4: K, V uint8 [Hkv][n_src][dh/2], two int4 per byte, the  */
/*    even channel in the low nibble; Ke, Ve as for MXINT8.                     */
/*  - idx != NULL: the cache is rows idx[0..n_cache) (idx_mode SHARED) or      */
/*    idx[g][0..n_cache) of head g (PER_HEAD) (eviction subset); idx == NULL:  */
/*    rows 0..n_cache. counts and info as described above patchkv_kv_format,    */
/*    with B = n_cache and N = n_src (info may be NULL).                       */
/*  - bias [Hkv][n_cache] float (natural-log units, indexed by cache entry) or  */
/*    NULL for none.                                                           */
/*  - p_terms as for patchkv_attend_chunk (1: P rounded to bf16; 2: two terms). */
/* Quantized entries, exact in bf16: the bf16 kernels read them as stored and  */
/* expand them on the way into LDS (no copy of the cache); with dtype F32 they */
/* are first expanded into f32 rows in the workspace.                          */
/* Limits as patchkv_attend_compressed with B = n_cache; dh a multiple of 32.  */
/* Workspace: patchkv_attend_cache_workspace_bytes(...).                       */
/* ------------------------------------------------------------------------- */
size_t patchkv_attend_cache_workspace_bytes(int dtype, int kv_format, int64_t M, int64_t n_cache,
                                            int Hq, int Hkv, int dh);

int patchkv_attend_cache(int dtype, const void* Q, const void* K, const void* V, int kv_format,
                         const int8_t* Ke, const int8_t* Ve, const int32_t* idx, int idx_mode,
                         const int32_t* counts, int64_t n_src, int64_t n_cache, const float* bias,
                         int64_t M, int Hq, int Hkv, int dh, float scale, int p_terms, float* O,
                         int32_t* info, void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Per-token targets, Eq. 5 in row form with h = z = the attention output:      */
/*   T = (O_f - O_c) W + rho (O_f - O_c)                                        */
/* Of, Oc [M][d_in] float; W [d_in][d_out] (w_dtype PATCHKV_BF16 or F32);        */
/* rho in {0, 1}; rho = 1 requires d_in == d_out. T [M][d_out] float, written.   */
/* The product is formed from a two-term bf16 split of (O_f - O_c) (and of W     */
/* when W is f32) on bf16 MFMA with fp32 accumulation (relative error ~1e-5).   */
/* ------------------------------------------------------------------------- */
size_t patchkv_targets_workspace_bytes(int w_dtype, int64_t M, int64_t d_in, int64_t d_out);

int patchkv_compute_targets(int w_dtype, const float* Of, const float* Oc, const void* W,
                            int64_t M, int64_t d_in, int64_t d_out, int rho, float* T,
                            void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* The MLP-shaped block (Sec. 2.2, "MLP activation matching"; Alg. 1). The      */
/* block output is y = h W + z: z [M][d] is the attention output, h [M][d_ff]   */
/* the post-activation SwiGLU intermediate, W [d_ff][d] the down-projection     */
/* that the patch corrects. The MLP reads z through an RMS norm with unit gain.  */
/*                                                                           */
/* patchkv_mlp_features:  H = silu(u Wg) * (u Wu), u = z / sqrt(mean(z^2)+eps)  */
/*   per row, silu(x) = x / (1 + e^-x). Z [M][d] float; Wg, Wu [d][d_ff]        */
/*   (w_dtype); H [M][d_ff] float, written. u enters the MFMA products as a      */
/*   two-term bf16 split (and W too when f32): relative error ~1e-5.            */
/* patchkv_compute_block_targets:  Eq. 5, T = (Hf - Hc) W + (Zf - Zc).          */
/*   Hf, Hc [M][d_ff] float; W [d_ff][d] (w_dtype); Zf, Zc [M][d] float;        */
/*   T [M][d] float, written.                                                  */
/* patchkv_propagate_student:  student-state propagation of Alg. 1, the patched */
/*   block's output Y = Hc (W + dW) + Zc. Hc [M][d_ff], dW [d_ff][d], Zc [M][d] */
/*   float; W [d_ff][d] (w_dtype); Y [M][d] float, written.                     */
/* The patch itself is patchkv_accumulate_normal_eq on (Hc, T) with d_in = d_ff */
/* and patchkv_solve_patch (d_in = d_ff, d_out = d).                           */
/* Limits: M >= 1 (M below 2^31), 1 <= d, d_ff <= 65536, d_ff a multiple of 4; */
/*   eps >= 0 and finite; every pointer 16-byte aligned.                       */
/* ------------------------------------------------------------------------- */
size_t patchkv_mlp_features_workspace_bytes(int w_dtype, int64_t M, int64_t d, int64_t d_ff);

int patchkv_mlp_features(int w_dtype, const float* Z, const void* Wg, const void* Wu, int64_t M,
                         int64_t d, int64_t d_ff, float eps, float* H, void* workspace,
                         size_t workspace_bytes, void* stream);

size_t patchkv_block_targets_workspace_bytes(int w_dtype, int64_t M, int64_t d_ff, int64_t d);

int patchkv_compute_block_targets(int w_dtype, const float* Hf, const float* Hc, const void* W,
                                  const float* Zf, const float* Zc, int64_t M, int64_t d_ff,
                                  int64_t d, float* T, void* workspace, size_t workspace_bytes,
                                  void* stream);

size_t patchkv_propagate_workspace_bytes(int w_dtype, int64_t M, int64_t d_ff, int64_t d);

int patchkv_propagate_student(int w_dtype, const float* Hc, const void* W, const float* dW,
                              const float* Zc, int64_t M, int64_t d_ff, int64_t d, float* Y,
                              void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Sufficient statistics, Eq. 9 (row form; Alg. 1 accumulation over chunks):    */
/*   G (+)= Xc^T Xc              [d_in][d_in]                                   */
/*   C (+)= Xc^T (Yf - Yc)       [d_in][d_out]                                  */
/* Xc [rows][d_in], Yf [rows][d_out] float; Yc NULL means zero (Yf is then the   */
/* target T itself). accumulate = 0 overwrites G and C, 1 adds to them (running */
/* sums over reference chunks start from zero: call with 0 first).              */
/* acc_dtype: PATCHKV_F32 -> G, C are float*, products from a split-bf16 MFMA   */
/*   scheme (error ~1e-5 relative) accumulated in fp32;                        */
/*   PATCHKV_F64 -> G, C are double*, fp64 products and accumulation.           */
/* G is written in full (both triangles).                                       */
/* ------------------------------------------------------------------------- */
size_t patchkv_normal_eq_workspace_bytes(int acc_dtype, int64_t rows, int64_t d_in, int64_t d_out);

int patchkv_accumulate_normal_eq(int acc_dtype, const float* Xc, const float* Yf,
                                 const float* Yc, int64_t rows, int64_t d_in, int64_t d_out,
                                 int accumulate, void* G, void* C,
                                 void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* Ridge patch, Eq. 8 (row form): dW = (G + lambda I)^{-1} C, by a blocked      */
/* Cholesky factorisation (G + lambda I = L L^T) and two triangular solves.     */
/* G [d_in][d_in] (only the lower triangle is read), C [d_in][d_out], both of   */
/* acc_dtype (F32: float, F64: double); they are not modified.                  */
/* ridge_mode ABSOLUTE: lambda is the ridge coefficient (> 0).                  */
/* ridge_mode ADAPTIVE: lambda is lambda_0 (> 0) and the coefficient is         */
/*   lambda_0 ||G||_F^2 / tr(G) (Eq. 7), computed on the device in fp64.        */
/* ridge_mode TRACE_MEAN: lambda is lambda_0 (> 0) and the coefficient is       */
/*   lambda_0 tr(G) / d_in, computed on the device in fp64.                     */
/* ridge_mode | PATCHKV_SOLVE_EXACT_F32 or | PATCHKV_SOLVE_FAST_BF16: the F32    */
/*   solve's block products (see patchkv_ridge_mode; default FP32-grade). Both   */
/*   flags, or any other bit set in ridge_mode: PATCHKV_E_VALUE.                */
/* dW [d_in][d_out] float, written.                                             */
/* info: device int32, written: 0 on success, else the 1-based column of the    */
/*   first non-positive (or NaN) pivot, LAPACK style (dW is then meaningless).  */
/* ------------------------------------------------------------------------- */
size_t patchkv_solve_workspace_bytes(int acc_dtype, int64_t d_in, int64_t d_out);

int patchkv_solve_patch(int acc_dtype, const void* G, const void* C, int64_t d_in, int64_t d_out,
                        double lambda, int ridge_mode, float* dW, int32_t* info,
                        void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* The same ridge patch from the data, for few rows and a wide d_in (the       */
/* MLP-shaped patch: one block of M reference tokens, d_in = d_ff > M). Eq. 8  */
/* through the push-through identity:                                        */
/*   dW = (X^T X + lambda I)^{-1} X^T T = X^T (X X^T + lambda I)^{-1} T,        */
/* so the factored system is rows x rows: K = X X^T (split-bf16 MFMA, all four  */
/* term pairs, fp32), the solve of patchkv_solve_patch on (K, T), then X^T Y.    */
/* X [rows][d_in], T [rows][d_out] float (the statistics' inputs, not G and C); */
/* dW [d_in][d_out] float, written. ridge_mode as for patchkv_solve_patch, and  */
/* every mode gives the primal system's lambda: ||X^T X||_F = ||X X^T||_F and   */
/* tr X^T X = tr X X^T, and the trace mean stays a mean over d_in. info as for  */
/* the solve (first failing pivot of K + lambda I, 1-based).                   */
/* Limits: 1 <= rows, d_in, d_out <= 65536;                                  */
/* every pointer 16-byte aligned, info 4-byte aligned.                         */
/* ------------------------------------------------------------------------- */
size_t patchkv_solve_patch_dual_workspace_bytes(int64_t rows, int64_t d_in, int64_t d_out);

int patchkv_solve_patch_dual(const float* X, const float* T, int64_t rows, int64_t d_in,
                             int64_t d_out, double lambda, int ridge_mode, float* dW,
                             int32_t* info, void* workspace, size_t workspace_bytes,
                             void* stream);

/* ------------------------------------------------------------------------- */
/* Reduced-rank patch (App. C, low-rank weight patches; reduced-rank regression):*/
/* the ridge patch projected onto its top-r output subspace. In row form,       */
/*   dW_r = dW U_r U_r^T,  U_r [d_out][r] = top-r eigenvectors of dW^T G dW,    */
/* stored as the factors A = dW U_r [d_in][r] and U_r, (d_in + d_out) r floats. */
/* G [d_in][d_in] float (the statistic without the ridge), dW [d_in][d_out]      */
/* float. Outputs: A, U written; dW_r [d_in][d_out] written when non-NULL.       */
/* Method: subspace iteration with a block of b = min(64, d_out) (rounded down  */
/* to even) columns for `iters` steps, then Rayleigh-Ritz (fp64 Jacobi on the   */
/* b x b projection). Where eigenvalue r and r+1 of dW^T G dW nearly coincide,  */
/* the subspace is ill-determined and only its captured energy is.             */
/* Limits: 1 <= r <= b, 1 <= iters <= 1000, d_in, d_out <= 65536, d_out >= 2.   */
/* ------------------------------------------------------------------------- */
size_t patchkv_low_rank_workspace_bytes(int64_t d_in, int64_t d_out, int r);

int patchkv_low_rank_patch(const float* G, const float* dW, int64_t d_in, int64_t d_out, int r,
                           int iters, float* A, float* U, float* dW_r, void* workspace,
                           size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* One block's patch (Alg. 1, one block and one reference chunk):               */
/*   O_f = attend_full(Q, K, V); O_c = attend over the compressed cache;        */
/*   T = (O_f - O_c) W + rho (O_f - O_c); G = O_c^T O_c, C = O_c^T T;           */
/*   dW = (G + lambda I)^{-1} C.                                                */
/* dtype: input type of Q, K, V, Kc, Vc and W (PATCHKV_BF16 or PATCHKV_F32).     */
/* acc_dtype: statistics and solve precision (PATCHKV_F32 or PATCHKV_F64).      */
/* Compressed cache: idx != NULL -> eviction subset of (K, V), idx [B] or      */
/*   [Hkv][B] by idx_mode (Kc, Vc ignored); idx == NULL -> synthesized Kc, Vc   */
/*   [Hkv][B][dh]. counts as described above patchkv_kv_format.                */
/* W [d][d] with d = Hq*dh. dW [d][d] float. info (required): as in solve_patch, */
/*   except that an out-of-range index entry or count is reported in its place  */
/*   (negative code, as described above patchkv_kv_format).                    */
/* ------------------------------------------------------------------------- */
size_t patchkv_layer_workspace_bytes(int dtype, int acc_dtype, int64_t M, int64_t N, int64_t B,
                                     int Hq, int Hkv, int dh);

int patchkv_compute_layer_patch(int dtype, int acc_dtype, const void* Q, const void* K,
                                const void* V, const int32_t* idx, int idx_mode,
                                const int32_t* counts, const void* Kc, const void* Vc,
                                const void* W, int64_t M, int64_t N, int64_t B, int Hq, int Hkv,
                                int dh, float scale, int rho, double lambda, int ridge_mode,
                                float* dW, int32_t* info, void* workspace,
                                size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PATCHKV_H */
