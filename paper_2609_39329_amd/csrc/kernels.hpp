// Internal launcher interface between the C ABI (capi.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pkv {

// ---------------------------------------------------------------- attention
struct AttnShape {
  int64_t M;         // reference queries
  int64_t Nk;        // cache entries attended
  int Hq, Hkv, dh;
  bool bf16;         // input dtype: bf16 (MFMA path) or f32
  int64_t Ms = 0;    // own entries of a reference chunk (0, or M: query m sees own 0..m)
};

struct AttnPlan {
  int n_split;         // number of key ranges (1 = no partial outputs)
  int keys_per_split;  // multiple of the key tile
  int row_tiles;       // query-row tiles per KV head
  int total_items;     // Hkv * n_split * row_tiles
  int per_xcd;         // work items per XCD
  int grid;            // launched workgroups (multiple of the XCD count)
  size_t ws_bytes;     // workspace: partial outputs and (m, l) pairs
};

AttnPlan plan_attention(const AttnShape& s);

// Which rows of K, V form the cache. idx null: rows 0..Nk of every KV head. Otherwise
// entry n of KV head g is row idx[g * stride + n] (stride 0: one set for every head);
// entries outside [0, src_rows) read as zero rows. counts non-null: head g keeps only
// its first counts[g] entries (clamped into [1, Nk]).
struct CacheIndex {
  const int32_t* idx = nullptr;
  int64_t stride = 0;
  const int32_t* counts = nullptr;
};

// Block-scaled integer storage of a cache's K and V (bf16 path): bits 8 (int8 values)
// or 4 (int4, two per byte, even channel in the low nibble), Ke / Ve one int8 exponent
// per 32 channels ([Hkv][src_rows][dh / 32]); an entry's value is q * 2^e. bits 0: K
// and V are plain bf16 / f32 rows.
struct KvQuant {
  int bits = 0;
  const int8_t* Ke = nullptr;
  const int8_t* Ve = nullptr;
};

// Q [M][Hq][dh]; K, V rows of KV head g start at (g * src_rows) * dh; the cache's
// entries are selected by ci.
// psplit: form P V from a two-term bf16 split of P (bf16 path only).
// s.Ms > 0: Ks, Vs [Hkv][Ms][dh] are the chunk's own entries (causal, after the cache).
// bias [Hkv][Nk]: per-entry logit bias (natural-log units), added to entry n's logit.
// kq.bits != 0 (bf16, no own entries): K, V are block-scaled integers, expanded to
// bf16 inside the kernels (keys at the LDS store of each tile, values by the V^T
// pre-pass).
hipError_t launch_attention(const AttnShape& s, const void* Q, const void* K, const void* V,
                            const CacheIndex& ci, int64_t src_rows, int64_t src_valid,
                            float scale, bool psplit, float* O, void* ws, hipStream_t st,
                            const void* Ks = nullptr, const void* Vs = nullptr,
                            const float* bias = nullptr, const KvQuant& kq = KvQuant{});
// Block-scaled integer cache rows -> [Hkv][n_cache][dh] bf16 (bf16) or f32: value
// q * 2^e, q int8 (bits 8) or int4 packed two per byte (bits 4, even channel in the
// low nibble), e int8 per 32 channels; entry n of head g is row idx[g * stride + n]
// (or n) of n_src rows; entries past a head's count are zero rows.
hipError_t launch_mx_dequant(bool bf16, int bits, const void* q, const int8_t* e,
                             const CacheIndex& ci, int64_t n_src, int64_t n_cache, int Hkv, int dh,
                             void* out, hipStream_t st);
// *info = 0 when every index entry lies in [0, n_src) and every count in [1, B], else
// the negative code of the first offending entry or count (see patchkv.h).
hipError_t launch_idx_check(const CacheIndex& ci, int heads, int64_t B, int64_t n_src,
                            int32_t* info, hipStream_t st);
// *info = *status where *status is non-zero.
hipError_t launch_info_merge(const int32_t* status, int32_t* info, hipStream_t st);

// The allocation-free attention's fixed scratch: its size, and its device address on
// the current device (looked up on the first call per device).
constexpr size_t kNoallocScratchBytes = (size_t)64 << 20;
constexpr int kMaxDevices = 64;
hipError_t noalloc_scratch(void** ptr);

// ---------------------------------------------------------------- statistics (fp32 acc)
size_t targets_ws_bytes(int64_t M, int64_t din, int64_t dout);
// T = (Of - Oc) W + rho (Of - Oc); W bf16 (w_bf16) or f32. With Zf non-null the
// residual is (Zf - Zc) [M][dout] instead (the MLP-shaped block).
hipError_t launch_targets(const float* Of, const float* Oc, const void* W, bool w_bf16,
                          int64_t M, int64_t din, int64_t dout, int rho, float* T, void* ws,
                          hipStream_t st, const float* Zf = nullptr, const float* Zc = nullptr);
// H [M][d_ff] = silu(u Wg) * (u Wu), u = rms_norm(Z) (unit gain), Wg, Wu [d][d_ff].
size_t mlp_features_ws_bytes(int64_t M, int64_t d, int64_t d_ff);
hipError_t launch_mlp_features(const float* Z, const void* Wg, const void* Wu, bool w_bf16,
                               int64_t M, int64_t d, int64_t d_ff, float eps, float* H, void* ws,
                               hipStream_t st);
// Y [M][d] = Hc (W + dW) + Zc, W [d_ff][d] (bf16 or f32), dW fp32.
size_t propagate_ws_bytes(int64_t M, int64_t d_ff, int64_t d);
hipError_t launch_propagate(const float* Hc, const void* W, bool w_bf16, const float* dW,
                            const float* Zc, int64_t M, int64_t d_ff, int64_t d, float* Y, void* ws,
                            hipStream_t st);
size_t normal_eq_ws_bytes(int64_t rows, int64_t din, int64_t dout);
// G (+)= X^T X, C (+)= X^T (Yf - Yc) with split-bf16 MFMA, fp32 accumulation.
hipError_t launch_normal_eq_f32(const float* X, const float* Yf, const float* Yc, int64_t rows,
                                int64_t din, int64_t dout, bool accumulate, float* G, float* C,
                                void* ws, hipStream_t st);

// Dual-form statistics (few rows, wide d_in): K [rows][rows] = X X^T (exactly
// symmetric) and Out [din][dout] = X^T Y, X [rows][din], Y [rows][dout], split-bf16
// MFMA with all four term pairs, fp32 accumulation.
size_t dual_stats_ws_bytes(int64_t rows, int64_t din, int64_t dout);
hipError_t launch_gram_rows(const float* X, int64_t rows, int64_t din, float* K, void* ws,
                            hipStream_t st);
hipError_t launch_xt_y(const float* X, const float* Y, int64_t rows, int64_t din, int64_t dout,
                       float* Out, void* ws, hipStream_t st);

// ---------------------------------------------------------------- statistics (fp64 acc)
hipError_t launch_targets_f64(const float* Of, const float* Oc, const void* W, bool w_bf16,
                              int64_t M, int64_t din, int64_t dout, int rho, double* T,
                              hipStream_t st);
// G (+)= X^T X, C (+)= X^T Y with Y = Yf - Yc (floats) or Yd (doubles, when non-null).
hipError_t launch_normal_eq_f64(const float* X, const float* Yf, const float* Yc, const double* Yd,
                                int64_t rows, int64_t din, int64_t dout, bool accumulate,
                                double* G, double* C, hipStream_t st);

// ---------------------------------------------------------------- ridge solve
// Reduced-rank patch: A [din][r], U [dout][r] with dW_r = A U^T the projection of dW
// onto the top-r eigenvectors of dW^T G dW; dWr [din][dout] written when non-null.
// r <= min(dout, 64) rounded down to even; iters subspace iterations.
size_t low_rank_ws_bytes(int64_t din, int64_t dout);
hipError_t launch_low_rank(const float* G, const float* dW, int64_t din, int64_t dout, int r,
                           int iters, float* A, float* U, float* dWr, void* ws, hipStream_t st);
size_t solve_ws_bytes(bool f64, int64_t din, int64_t dout);
// ridge: 0 the coefficient is lambda; 1 lambda ||G||_F^2 / tr G (Eq. 7); 2 lambda tr G / d.
// products (fp32 solve): how block products are formed; the fp64 solve always uses
// fp64 arithmetic.
constexpr int kProductsSplit6 = 0;  // three bf16 pieces per operand, six MFMA terms (FP32-grade)
constexpr int kProductsExact = 1;   // fp32 MFMA (exact fp32 products)
constexpr int kProductsSplit3 = 2;  // two bf16 pieces, three MFMA terms (about 2^-16)
hipError_t launch_solve(bool f64, const void* G, const void* C, int64_t din, int64_t dout,
                        double lambda, int ridge, int products, float* dW, int32_t* info,
                        void* ws, hipStream_t st);

// Small helpers.
inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

}  // namespace pkv
