// C ABI of the PatchKV context-loading path: argument validation, workspace
// carving and kernel dispatch. Every check runs on the host before anything is
// enqueued; the kernels themselves assume validated arguments.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>

#include "../../include/patchkv.h"
#include "kernels.hpp"

using namespace pkv;

namespace {

constexpr int64_t kMaxDim = 1 << 16;           // d_in, d_out
static_assert(PATCHKV_NOALLOC_SCRATCH_BYTES == kNoallocScratchBytes,
              "the header states the size of the allocation-free call's fixed scratch");
constexpr int64_t kMaxRows = (int64_t)1 << 31;  // M*Hq, N, B, rows

bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }
bool al4(const void* p) { return ((uintptr_t)p & 3) == 0; }

// The index set of an eviction-style compressed cache: mode and pointer alignment
// (its values are checked on the device, see idx_check).
int check_index(const int32_t* idx, int idx_mode, const int32_t* counts) {
  if (idx_mode != PATCHKV_IDX_SHARED && idx_mode != PATCHKV_IDX_PER_HEAD) return PATCHKV_E_VALUE;
  if (idx_mode == PATCHKV_IDX_PER_HEAD && !idx) return PATCHKV_E_NULL;
  if (!al4(idx) || !al4(counts)) return PATCHKV_E_VALUE;
  return PATCHKV_OK;
}

CacheIndex cache_index(const int32_t* idx, int idx_mode, const int32_t* counts, int64_t B) {
  CacheIndex ci;
  ci.idx = idx;
  ci.stride = idx && idx_mode == PATCHKV_IDX_PER_HEAD ? B : 0;
  ci.counts = counts;
  return ci;
}

int status_of(hipError_t e) { return e == hipSuccess ? PATCHKV_OK : PATCHKV_E_HIP; }

// The bf16 kernels address one KV head's rows (and its V^T tiles) with 32-bit
// buffer offsets: rows * dh * 2 bytes must stay below 2^32.
bool src_rows_ok(int dtype, int64_t rows, int dh) {
  return rows >= 1 && rows < kMaxRows && (dtype != PATCHKV_BF16 || rows * dh * 2 < ((int64_t)1 << 32));
}

int check_attn_shape(int dtype, int64_t M, int64_t Nk, int Hq, int Hkv, int dh) {
  if (dtype != PATCHKV_F32 && dtype != PATCHKV_BF16) return PATCHKV_E_DTYPE;
  if (M < 1 || Nk < 1 || Hq < 1 || Hkv < 1 || Hq % Hkv != 0) return PATCHKV_E_SHAPE;
  if (dh != 64 && dh != 128) return PATCHKV_E_UNSUPPORTED;
  if (M * Hq >= kMaxRows || !src_rows_ok(dtype, Nk, dh)) return PATCHKV_E_SHAPE;
  return PATCHKV_OK;
}

AttnShape attn_shape(int dtype, int64_t M, int64_t Nk, int Hq, int Hkv, int dh) {
  AttnShape s{};
  s.M = M;
  s.Nk = Nk;
  s.Hq = Hq;
  s.Hkv = Hkv;
  s.dh = dh;
  s.bf16 = dtype == PATCHKV_BF16;
  return s;
}

int check_ws(const void* ws, size_t have, size_t need) {
  if (need == 0) return PATCHKV_OK;
  if (!ws || have < need || !al16(ws)) return PATCHKV_E_WORKSPACE;
  return PATCHKV_OK;
}

bool finite_pos(double x) { return isfinite(x) && x > 0.0; }
constexpr int kProductFlags = PATCHKV_SOLVE_EXACT_F32 | PATCHKV_SOLVE_FAST_BF16;
bool valid_ridge_mode(int m) {
  const int base = m & ~kProductFlags;
  if ((m & kProductFlags) == kProductFlags) return false;  // one product mode at most
  return base == PATCHKV_RIDGE_ABSOLUTE || base == PATCHKV_RIDGE_ADAPTIVE ||
         base == PATCHKV_RIDGE_TRACE_MEAN;
}
// 0: absolute, 1: Eq. 7, 2: trace mean (the solve's ridge selector)
int ridge_kind(int m) { return m & ~kProductFlags; }
// the F32 solve's block products
int products(int m) {
  if (m & PATCHKV_SOLVE_EXACT_F32) return kProductsExact;
  if (m & PATCHKV_SOLVE_FAST_BF16) return kProductsSplit3;
  return kProductsSplit6;
}

int check_stats_dims(int64_t rows, int64_t din, int64_t dout) {
  if (rows < 1 || din < 1 || dout < 1) return PATCHKV_E_SHAPE;
  if (rows >= kMaxRows || din > kMaxDim || dout > kMaxDim) return PATCHKV_E_SHAPE;
  return PATCHKV_OK;
}

// Layer-patch workspace layout.
struct LayerWs {
  size_t Of, Oc, T, G, C, attn, solve, stat, total;
};

LayerWs layer_ws(int dtype, int acc, int64_t M, int64_t N, int64_t B, int Hq, int Hkv, int dh) {
  LayerWs L{};
  const int64_t d = (int64_t)Hq * dh;
  const size_t accb = acc == PATCHKV_F64 ? sizeof(double) : sizeof(float);
  size_t o = 0;
  L.Of = o; o += align_up(sizeof(float) * M * d);
  L.Oc = o; o += align_up(sizeof(float) * M * d);
  L.T = o; o += align_up(accb * M * d);
  L.G = o; o += align_up(accb * d * d);
  L.C = o; o += align_up(accb * d * d);
  // scratch shared by the two attention passes, then by the targets and statistics
  // pre-passes (all ordered on one stream)
  L.attn = o;
  size_t scratch = std::max(plan_attention(attn_shape(dtype, M, N, Hq, Hkv, dh)).ws_bytes,
                            plan_attention(attn_shape(dtype, M, B, Hq, Hkv, dh)).ws_bytes);
  if (acc == PATCHKV_F32)
    scratch = std::max({scratch, targets_ws_bytes(M, d, d), normal_eq_ws_bytes(M, d, d)});
  o += align_up(scratch);
  L.solve = o; o += align_up(solve_ws_bytes(acc == PATCHKV_F64, d, d));
  L.stat = o; o += align_up(sizeof(int32_t));  // index-set check, merged into info at the end
  L.total = o;
  return L;
}

}  // namespace

extern "C" {

const char* patchkv_status_string(int status) {
  switch (status) {
    case PATCHKV_OK: return "ok";
    case PATCHKV_E_NULL: return "null pointer argument";
    case PATCHKV_E_SHAPE: return "invalid or inconsistent shape";
    case PATCHKV_E_DTYPE: return "unsupported dtype";
    case PATCHKV_E_VALUE: return "scalar argument out of range or misaligned pointer";
    case PATCHKV_E_WORKSPACE: return "workspace missing, misaligned or too small";
    case PATCHKV_E_UNSUPPORTED: return "unsupported head_dim (64 or 128 only)";
    case PATCHKV_E_HIP: return "HIP runtime error";
    case PATCHKV_E_SCRATCH:
      return "the call needs more scratch than the fixed buffer of the allocation-free entry point";
    default: return "unknown status";
  }
}

int patchkv_version(void) { return 10000; }

size_t patchkv_attend_workspace_bytes(int dtype, int64_t M, int64_t N, int Hq, int Hkv, int dh) {
  if (check_attn_shape(dtype, M, N, Hq, Hkv, dh) != PATCHKV_OK) return 0;
  return plan_attention(attn_shape(dtype, M, N, Hq, Hkv, dh)).ws_bytes;
}

int patchkv_attend_full(int dtype, const void* Q, const void* K, const void* V, int64_t M,
                        int64_t N, int Hq, int Hkv, int dh, float scale, float* O, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (!Q || !K || !V || !O) return PATCHKV_E_NULL;
  int s = check_attn_shape(dtype, M, N, Hq, Hkv, dh);
  if (s) return s;
  if (!finite_pos(scale)) return PATCHKV_E_VALUE;
  if (!al16(Q) || !al16(K) || !al16(V) || !al16(O)) return PATCHKV_E_VALUE;
  const AttnShape sh = attn_shape(dtype, M, N, Hq, Hkv, dh);
  s = check_ws(workspace, workspace_bytes, plan_attention(sh).ws_bytes);
  if (s) return s;
  return status_of(launch_attention(sh, Q, K, V, CacheIndex{}, N, N, scale, false, O, workspace,
                                    (hipStream_t)stream));
}

}  // extern "C"

namespace {

// attend_compressed with the scratch from the caller's workspace, or (noalloc) from the
// library's fixed device buffer.
int attend_compressed_impl(int dtype, const void* Q, const void* K, const void* V,
                           const int32_t* idx, int idx_mode, const int32_t* counts, int64_t M,
                           int64_t N, int64_t B, int Hq, int Hkv, int dh, float scale, float* O,
                           int32_t* info, void* workspace, size_t workspace_bytes, bool noalloc,
                           void* stream) {
  if (!Q || !K || !V || !O) return PATCHKV_E_NULL;
  int s = check_attn_shape(dtype, M, B, Hq, Hkv, dh);
  if (s) return s;
  if (idx && !src_rows_ok(dtype, N, dh)) return PATCHKV_E_SHAPE;
  s = check_index(idx, idx_mode, counts);
  if (s) return s;
  if (!finite_pos(scale)) return PATCHKV_E_VALUE;
  if (!al16(Q) || !al16(K) || !al16(V) || !al16(O) || !al4(info)) return PATCHKV_E_VALUE;
  const AttnShape sh = attn_shape(dtype, M, B, Hq, Hkv, dh);
  const size_t need = plan_attention(sh).ws_bytes;
  if (noalloc) {
    if (need > kNoallocScratchBytes) return PATCHKV_E_SCRATCH;
    workspace = nullptr;
    if (need > 0 && noalloc_scratch(&workspace) != hipSuccess) return PATCHKV_E_HIP;
  } else {
    s = check_ws(workspace, workspace_bytes, need);
    if (s) return s;
  }
  const int64_t src = idx ? N : B;
  const CacheIndex ci = cache_index(idx, idx_mode, counts, B);
  const hipStream_t st = (hipStream_t)stream;
  if (info && launch_idx_check(ci, Hkv, B, src, info, st) != hipSuccess) return PATCHKV_E_HIP;
  return status_of(launch_attention(sh, Q, K, V, ci, src, src, scale, true, O, workspace, st));
}

}  // namespace

extern "C" {

int patchkv_attend_compressed(int dtype, const void* Q, const void* K, const void* V,
                              const int32_t* idx, int idx_mode, const int32_t* counts, int64_t M,
                              int64_t N, int64_t B, int Hq, int Hkv, int dh, float scale, float* O,
                              int32_t* info, void* workspace, size_t workspace_bytes,
                              void* stream) {
  return attend_compressed_impl(dtype, Q, K, V, idx, idx_mode, counts, M, N, B, Hq, Hkv, dh,
                                scale, O, info, workspace, workspace_bytes, false, stream);
}

int patchkv_attend_compressed_noalloc(int dtype, const void* Q, const void* K, const void* V,
                                      const int32_t* idx, int idx_mode, const int32_t* counts,
                                      int64_t M, int64_t N, int64_t B, int Hq, int Hkv, int dh,
                                      float scale, float* O, int32_t* info, void* stream) {
  return attend_compressed_impl(dtype, Q, K, V, idx, idx_mode, counts, M, N, B, Hq, Hkv, dh,
                                scale, O, info, nullptr, 0, true, stream);
}

size_t patchkv_attend_chunk_workspace_bytes(int dtype, int64_t M, int64_t n_cache, int Hq, int Hkv,
                                            int dh) {
  if (check_attn_shape(dtype, M, n_cache, Hq, Hkv, dh) != PATCHKV_OK) return 0;
  if (!src_rows_ok(dtype, M, dh)) return 0;
  AttnShape sh = attn_shape(dtype, M, n_cache, Hq, Hkv, dh);
  sh.Ms = M;
  return plan_attention(sh).ws_bytes;
}

int patchkv_attend_chunk(int dtype, const void* Q, const void* K, const void* V,
                         const int32_t* idx, int idx_mode, const int32_t* counts, int64_t n_src,
                         int64_t n_cache, const void* Ks, const void* Vs, int64_t M, int Hq,
                         int Hkv, int dh, float scale, int p_terms, float* O, int32_t* info,
                         void* workspace, size_t workspace_bytes, void* stream) {
  if (!Q || !K || !V || !Ks || !Vs || !O) return PATCHKV_E_NULL;
  int s = check_attn_shape(dtype, M, n_cache, Hq, Hkv, dh);
  if (s) return s;
  if (!src_rows_ok(dtype, n_src, dh) || !src_rows_ok(dtype, M, dh)) return PATCHKV_E_SHAPE;
  if (!idx && n_cache > n_src) return PATCHKV_E_SHAPE;
  s = check_index(idx, idx_mode, counts);
  if (s) return s;
  if (p_terms != 1 && p_terms != 2) return PATCHKV_E_VALUE;
  if (!finite_pos(scale)) return PATCHKV_E_VALUE;
  if (!al16(Q) || !al16(K) || !al16(V) || !al16(Ks) || !al16(Vs) || !al16(O) || !al4(info))
    return PATCHKV_E_VALUE;
  AttnShape sh = attn_shape(dtype, M, n_cache, Hq, Hkv, dh);
  sh.Ms = M;
  s = check_ws(workspace, workspace_bytes, plan_attention(sh).ws_bytes);
  if (s) return s;
  const CacheIndex ci = cache_index(idx, idx_mode, counts, n_cache);
  const hipStream_t st = (hipStream_t)stream;
  if (info && launch_idx_check(ci, Hkv, n_cache, n_src, info, st) != hipSuccess)
    return PATCHKV_E_HIP;
  return status_of(launch_attention(sh, Q, K, V, ci, n_src, n_src, scale, p_terms == 2, O,
                                    workspace, st, Ks, Vs));
}

namespace {
bool valid_kv_format(int f) {
  return f == PATCHKV_KV_PLAIN || f == PATCHKV_KV_MXINT8 || f == PATCHKV_KV_MXINT4;
}
// dequantized cache rows (quantized formats, f32 path), carved after the attention
// workspace; the bf16 kernels expand block-scaled entries themselves
size_t dequant_bytes(int dtype, int kv_format, int64_t n_cache, int Hkv, int dh) {
  if (kv_format == PATCHKV_KV_PLAIN || dtype == PATCHKV_BF16) return 0;
  const size_t e = dtype == PATCHKV_BF16 ? 2 : 4;
  return 2 * ((size_t)Hkv * n_cache * dh * e + 255) / 256 * 256;
}
}  // namespace

size_t patchkv_attend_cache_workspace_bytes(int dtype, int kv_format, int64_t M, int64_t n_cache,
                                            int Hq, int Hkv, int dh) {
  if (!valid_kv_format(kv_format)) return 0;
  if (check_attn_shape(dtype, M, n_cache, Hq, Hkv, dh) != PATCHKV_OK) return 0;
  const size_t a = (plan_attention(attn_shape(dtype, M, n_cache, Hq, Hkv, dh)).ws_bytes + 255) / 256 * 256;
  return a + dequant_bytes(dtype, kv_format, n_cache, Hkv, dh);
}

int patchkv_attend_cache(int dtype, const void* Q, const void* K, const void* V, int kv_format,
                         const int8_t* Ke, const int8_t* Ve, const int32_t* idx, int idx_mode,
                         const int32_t* counts, int64_t n_src, int64_t n_cache, const float* bias,
                         int64_t M, int Hq, int Hkv, int dh, float scale, int p_terms, float* O,
                         int32_t* info, void* workspace, size_t workspace_bytes, void* stream) {
  if (!Q || !K || !V || !O) return PATCHKV_E_NULL;
  if (!valid_kv_format(kv_format)) return PATCHKV_E_VALUE;
  const bool quant = kv_format != PATCHKV_KV_PLAIN;
  if (quant && (!Ke || !Ve)) return PATCHKV_E_NULL;
  int s = check_attn_shape(dtype, M, n_cache, Hq, Hkv, dh);
  if (s) return s;
  if (!src_rows_ok(dtype, n_src, dh)) return PATCHKV_E_SHAPE;
  if (!idx && n_cache > n_src) return PATCHKV_E_SHAPE;
  s = check_index(idx, idx_mode, counts);
  if (s) return s;
  if (p_terms != 1 && p_terms != 2) return PATCHKV_E_VALUE;
  if (!finite_pos(scale)) return PATCHKV_E_VALUE;
  if (!al16(Q) || !al16(K) || !al16(V) || !al16(O) || (bias && !al16(bias)) || !al4(info))
    return PATCHKV_E_VALUE;
  const AttnShape sh = attn_shape(dtype, M, n_cache, Hq, Hkv, dh);
  const size_t a = (plan_attention(sh).ws_bytes + 255) / 256 * 256;
  s = check_ws(workspace, workspace_bytes, a + dequant_bytes(dtype, kv_format, n_cache, Hkv, dh));
  if (s) return s;
  const CacheIndex ci = cache_index(idx, idx_mode, counts, n_cache);
  const hipStream_t st = (hipStream_t)stream;
  if (info && launch_idx_check(ci, Hkv, n_cache, n_src, info, st) != hipSuccess)
    return PATCHKV_E_HIP;
  if (!quant)
    return status_of(launch_attention(sh, Q, K, V, ci, n_src, n_src, scale, p_terms == 2, O,
                                      workspace, st, nullptr, nullptr, bias));
  const int bits = kv_format == PATCHKV_KV_MXINT8 ? 8 : 4;
  if (dtype == PATCHKV_BF16) {  // the kernels read the block-scaled entries themselves
    KvQuant kq;
    kq.bits = bits;
    kq.Ke = Ke;
    kq.Ve = Ve;
    return status_of(launch_attention(sh, Q, K, V, ci, n_src, n_src, scale, p_terms == 2, O,
                                      workspace, st, nullptr, nullptr, bias, kq));
  }
  // f32: expand the quantized entries (gathered through idx) into f32 rows, then attend
  const size_t half = dequant_bytes(dtype, kv_format, n_cache, Hkv, dh) / 2;
  char* kx = (char*)workspace + a;
  char* vx = kx + half;
  hipError_t e = launch_mx_dequant(dtype == PATCHKV_BF16, bits, K, Ke, ci, n_src, n_cache, Hkv,
                                   dh, kx, st);
  if (e == hipSuccess)
    e = launch_mx_dequant(dtype == PATCHKV_BF16, bits, V, Ve, ci, n_src, n_cache, Hkv, dh, vx, st);
  if (e != hipSuccess) return PATCHKV_E_HIP;
  CacheIndex dense;
  dense.counts = counts;  // the expanded rows are dense; a head still keeps only its count
  return status_of(launch_attention(sh, Q, kx, vx, dense, n_cache, n_cache, scale, p_terms == 2,
                                    O, workspace, st, nullptr, nullptr, bias));
}

size_t patchkv_targets_workspace_bytes(int w_dtype, int64_t M, int64_t d_in, int64_t d_out) {
  if (w_dtype != PATCHKV_BF16 && w_dtype != PATCHKV_F32) return 0;
  if (check_stats_dims(M, d_in, d_out)) return 0;
  return targets_ws_bytes(M, d_in, d_out);
}

int patchkv_compute_targets(int w_dtype, const float* Of, const float* Oc, const void* W,
                            int64_t M, int64_t d_in, int64_t d_out, int rho, float* T,
                            void* workspace, size_t workspace_bytes, void* stream) {
  if (!Of || !Oc || !W || !T) return PATCHKV_E_NULL;
  if (w_dtype != PATCHKV_BF16 && w_dtype != PATCHKV_F32) return PATCHKV_E_DTYPE;
  int s = check_stats_dims(M, d_in, d_out);
  if (s) return s;
  if (rho != 0 && rho != 1) return PATCHKV_E_VALUE;
  if (rho == 1 && d_in != d_out) return PATCHKV_E_SHAPE;
  s = check_ws(workspace, workspace_bytes, targets_ws_bytes(M, d_in, d_out));
  if (s) return s;
  return status_of(launch_targets(Of, Oc, W, w_dtype == PATCHKV_BF16, M, d_in, d_out, rho, T,
                                  workspace, (hipStream_t)stream));
}

namespace {
int check_mlp(int w_dtype, int64_t M, int64_t d, int64_t d_ff) {
  if (w_dtype != PATCHKV_BF16 && w_dtype != PATCHKV_F32) return PATCHKV_E_DTYPE;
  int s = check_stats_dims(M, d, d_ff);
  if (s) return s;
  if (d_ff % 4 != 0) return PATCHKV_E_SHAPE;
  return PATCHKV_OK;
}
}  // namespace

size_t patchkv_mlp_features_workspace_bytes(int w_dtype, int64_t M, int64_t d, int64_t d_ff) {
  if (check_mlp(w_dtype, M, d, d_ff)) return 0;
  return mlp_features_ws_bytes(M, d, d_ff);
}

int patchkv_mlp_features(int w_dtype, const float* Z, const void* Wg, const void* Wu, int64_t M,
                         int64_t d, int64_t d_ff, float eps, float* H, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (!Z || !Wg || !Wu || !H) return PATCHKV_E_NULL;
  int s = check_mlp(w_dtype, M, d, d_ff);
  if (s) return s;
  if (!(isfinite(eps) && eps >= 0.f)) return PATCHKV_E_VALUE;
  if (!al16(Z) || !al16(Wg) || !al16(Wu) || !al16(H)) return PATCHKV_E_VALUE;
  s = check_ws(workspace, workspace_bytes, mlp_features_ws_bytes(M, d, d_ff));
  if (s) return s;
  return status_of(launch_mlp_features(Z, Wg, Wu, w_dtype == PATCHKV_BF16, M, d, d_ff, eps, H,
                                       workspace, (hipStream_t)stream));
}

size_t patchkv_block_targets_workspace_bytes(int w_dtype, int64_t M, int64_t d_ff, int64_t d) {
  if (check_mlp(w_dtype, M, d, d_ff)) return 0;
  return targets_ws_bytes(M, d_ff, d);
}

int patchkv_compute_block_targets(int w_dtype, const float* Hf, const float* Hc, const void* W,
                                  const float* Zf, const float* Zc, int64_t M, int64_t d_ff,
                                  int64_t d, float* T, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  if (!Hf || !Hc || !W || !Zf || !Zc || !T) return PATCHKV_E_NULL;
  int s = check_mlp(w_dtype, M, d, d_ff);
  if (s) return s;
  if (!al16(Hf) || !al16(Hc) || !al16(W) || !al16(Zf) || !al16(Zc) || !al16(T))
    return PATCHKV_E_VALUE;
  s = check_ws(workspace, workspace_bytes, targets_ws_bytes(M, d_ff, d));
  if (s) return s;
  return status_of(launch_targets(Hf, Hc, W, w_dtype == PATCHKV_BF16, M, d_ff, d, 0, T, workspace,
                                  (hipStream_t)stream, Zf, Zc));
}

size_t patchkv_propagate_workspace_bytes(int w_dtype, int64_t M, int64_t d_ff, int64_t d) {
  if (check_mlp(w_dtype, M, d, d_ff)) return 0;
  return propagate_ws_bytes(M, d_ff, d);
}

int patchkv_propagate_student(int w_dtype, const float* Hc, const void* W, const float* dW,
                              const float* Zc, int64_t M, int64_t d_ff, int64_t d, float* Y,
                              void* workspace, size_t workspace_bytes, void* stream) {
  if (!Hc || !W || !dW || !Zc || !Y) return PATCHKV_E_NULL;
  int s = check_mlp(w_dtype, M, d, d_ff);
  if (s) return s;
  if (!al16(Hc) || !al16(W) || !al16(dW) || !al16(Zc) || !al16(Y)) return PATCHKV_E_VALUE;
  s = check_ws(workspace, workspace_bytes, propagate_ws_bytes(M, d_ff, d));
  if (s) return s;
  return status_of(launch_propagate(Hc, W, w_dtype == PATCHKV_BF16, dW, Zc, M, d_ff, d, Y,
                                    workspace, (hipStream_t)stream));
}

size_t patchkv_normal_eq_workspace_bytes(int acc_dtype, int64_t rows, int64_t d_in,
                                         int64_t d_out) {
  if (acc_dtype != PATCHKV_F32 && acc_dtype != PATCHKV_F64) return 0;
  if (check_stats_dims(rows, d_in, d_out)) return 0;
  return acc_dtype == PATCHKV_F32 ? normal_eq_ws_bytes(rows, d_in, d_out) : 0;
}

int patchkv_accumulate_normal_eq(int acc_dtype, const float* Xc, const float* Yf, const float* Yc,
                                 int64_t rows, int64_t d_in, int64_t d_out, int accumulate,
                                 void* G, void* C, void* workspace, size_t workspace_bytes,
                                 void* stream) {
  if (!Xc || !Yf || !G || !C) return PATCHKV_E_NULL;
  if (acc_dtype != PATCHKV_F32 && acc_dtype != PATCHKV_F64) return PATCHKV_E_DTYPE;
  int s = check_stats_dims(rows, d_in, d_out);
  if (s) return s;
  if (accumulate != 0 && accumulate != 1) return PATCHKV_E_VALUE;
  s = check_ws(workspace, workspace_bytes,
               acc_dtype == PATCHKV_F32 ? normal_eq_ws_bytes(rows, d_in, d_out) : 0);
  if (s) return s;
  hipStream_t st = (hipStream_t)stream;
  if (acc_dtype == PATCHKV_F32)
    return status_of(launch_normal_eq_f32(Xc, Yf, Yc, rows, d_in, d_out, accumulate != 0,
                                          (float*)G, (float*)C, workspace, st));
  return status_of(launch_normal_eq_f64(Xc, Yf, Yc, nullptr, rows, d_in, d_out, accumulate != 0,
                                        (double*)G, (double*)C, st));
}

size_t patchkv_solve_workspace_bytes(int acc_dtype, int64_t d_in, int64_t d_out) {
  if (acc_dtype != PATCHKV_F32 && acc_dtype != PATCHKV_F64) return 0;
  if (d_in < 1 || d_out < 1 || d_in > kMaxDim || d_out > kMaxDim) return 0;
  return solve_ws_bytes(acc_dtype == PATCHKV_F64, d_in, d_out);
}

int patchkv_solve_patch(int acc_dtype, const void* G, const void* C, int64_t d_in, int64_t d_out,
                        double lambda, int ridge_mode, float* dW, int32_t* info, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (!G || !C || !dW || !info) return PATCHKV_E_NULL;
  if (acc_dtype != PATCHKV_F32 && acc_dtype != PATCHKV_F64) return PATCHKV_E_DTYPE;
  if (d_in < 1 || d_out < 1 || d_in > kMaxDim || d_out > kMaxDim) return PATCHKV_E_SHAPE;
  if (!finite_pos(lambda)) return PATCHKV_E_VALUE;
  if (!valid_ridge_mode(ridge_mode)) return PATCHKV_E_VALUE;
  int s = check_ws(workspace, workspace_bytes, solve_ws_bytes(acc_dtype == PATCHKV_F64, d_in, d_out));
  if (s) return s;
  return status_of(launch_solve(acc_dtype == PATCHKV_F64, G, C, d_in, d_out, lambda,
                                ridge_kind(ridge_mode), products(ridge_mode), dW, info, workspace,
                                (hipStream_t)stream));
}

namespace {
// Dual-form solve workspace: K = X X^T, Y = (K + lambda I)^{-1} T, the solve's own
// workspace, the statistics' split planes.
struct DualSolveWs {
  size_t K, Y, solve, stats, total;
};
DualSolveWs dual_solve_layout(int64_t rows, int64_t din, int64_t dout) {
  DualSolveWs L{};
  size_t o = 0;
  L.K = o; o += align_up(sizeof(float) * rows * rows);
  L.Y = o; o += align_up(sizeof(float) * rows * dout);
  L.solve = o; o += align_up(solve_ws_bytes(false, rows, dout));
  L.stats = o; o += align_up(dual_stats_ws_bytes(rows, din, dout));
  L.total = o;
  return L;
}
int check_dual_dims(int64_t rows, int64_t din, int64_t dout) {
  int s = check_stats_dims(rows, din, dout);
  if (s) return s;
  return rows > kMaxDim ? PATCHKV_E_SHAPE : PATCHKV_OK;
}
}  // namespace

size_t patchkv_solve_patch_dual_workspace_bytes(int64_t rows, int64_t d_in, int64_t d_out) {
  if (check_dual_dims(rows, d_in, d_out)) return 0;
  return dual_solve_layout(rows, d_in, d_out).total;
}

int patchkv_solve_patch_dual(const float* X, const float* T, int64_t rows, int64_t d_in,
                             int64_t d_out, double lambda, int ridge_mode, float* dW,
                             int32_t* info, void* workspace, size_t workspace_bytes,
                             void* stream) {
  if (!X || !T || !dW || !info) return PATCHKV_E_NULL;
  int s = check_dual_dims(rows, d_in, d_out);
  if (s) return s;
  if (!finite_pos(lambda)) return PATCHKV_E_VALUE;
  if (!valid_ridge_mode(ridge_mode)) return PATCHKV_E_VALUE;
  if (!al16(X) || !al16(T) || !al16(dW) || !al4(info)) return PATCHKV_E_VALUE;
  const DualSolveWs L = dual_solve_layout(rows, d_in, d_out);
  s = check_ws(workspace, workspace_bytes, L.total);
  if (s) return s;
  char* w = (char*)workspace;
  float* K = (float*)(w + L.K);
  float* Y = (float*)(w + L.Y);
  const hipStream_t st = (hipStream_t)stream;
  // The solve takes the trace mean over its own side (rows); the primal system's mean
  // is over d_in, with the same trace.
  const double lam = ridge_kind(ridge_mode) == PATCHKV_RIDGE_TRACE_MEAN
                         ? lambda * (double)rows / (double)d_in
                         : lambda;
  hipError_t e = launch_gram_rows(X, rows, d_in, K, w + L.stats, st);
  if (e == hipSuccess)
    e = launch_solve(false, K, T, rows, d_out, lam, ridge_kind(ridge_mode), products(ridge_mode),
                     Y, info, w + L.solve, st);
  if (e == hipSuccess) e = launch_xt_y(X, Y, rows, d_in, d_out, dW, w + L.stats, st);
  return status_of(e);
}

namespace {
int check_low_rank(int64_t din, int64_t dout, int r, int iters) {
  if (din < 1 || dout < 2 || din > kMaxDim || dout > kMaxDim) return PATCHKV_E_SHAPE;
  const int b = (int)std::min<int64_t>(64, dout) & ~1;
  if (r < 1 || r > b || iters < 1 || iters > 1000) return PATCHKV_E_VALUE;
  return PATCHKV_OK;
}
}  // namespace

size_t patchkv_low_rank_workspace_bytes(int64_t d_in, int64_t d_out, int r) {
  if (check_low_rank(d_in, d_out, r, 1)) return 0;
  return low_rank_ws_bytes(d_in, d_out);
}

int patchkv_low_rank_patch(const float* G, const float* dW, int64_t d_in, int64_t d_out, int r,
                           int iters, float* A, float* U, float* dW_r, void* workspace,
                           size_t workspace_bytes, void* stream) {
  if (!G || !dW || !A || !U) return PATCHKV_E_NULL;
  int s = check_low_rank(d_in, d_out, r, iters);
  if (s) return s;
  if (!al16(G) || !al16(dW) || !al16(A) || !al16(U) || (dW_r && !al16(dW_r)))
    return PATCHKV_E_VALUE;
  s = check_ws(workspace, workspace_bytes, low_rank_ws_bytes(d_in, d_out));
  if (s) return s;
  return status_of(launch_low_rank(G, dW, d_in, d_out, r, iters, A, U, dW_r, workspace,
                                   (hipStream_t)stream));
}

size_t patchkv_layer_workspace_bytes(int dtype, int acc_dtype, int64_t M, int64_t N, int64_t B,
                                     int Hq, int Hkv, int dh) {
  if (acc_dtype != PATCHKV_F32 && acc_dtype != PATCHKV_F64) return 0;
  if (check_attn_shape(dtype, M, N, Hq, Hkv, dh) || check_attn_shape(dtype, M, B, Hq, Hkv, dh))
    return 0;
  if ((int64_t)Hq * dh > kMaxDim) return 0;
  return layer_ws(dtype, acc_dtype, M, N, B, Hq, Hkv, dh).total;
}

int patchkv_compute_layer_patch(int dtype, int acc_dtype, const void* Q, const void* K,
                                const void* V, const int32_t* idx, int idx_mode,
                                const int32_t* counts, const void* Kc, const void* Vc,
                                const void* W, int64_t M, int64_t N, int64_t B, int Hq, int Hkv,
                                int dh, float scale, int rho, double lambda, int ridge_mode,
                                float* dW, int32_t* info, void* workspace, size_t workspace_bytes,
                                void* stream) {
  if (!Q || !K || !V || !W || !dW || !info) return PATCHKV_E_NULL;
  if (!idx && (!Kc || !Vc)) return PATCHKV_E_NULL;
  {
    const int si = check_index(idx, idx_mode, counts);
    if (si) return si;
  }
  if (!al4(info)) return PATCHKV_E_VALUE;
  if (acc_dtype != PATCHKV_F32 && acc_dtype != PATCHKV_F64) return PATCHKV_E_DTYPE;
  int s = check_attn_shape(dtype, M, N, Hq, Hkv, dh);
  if (s) return s;
  s = check_attn_shape(dtype, M, B, Hq, Hkv, dh);
  if (s) return s;
  const int64_t d = (int64_t)Hq * dh;
  if (d > kMaxDim) return PATCHKV_E_SHAPE;
  if (!finite_pos(scale) || !finite_pos(lambda)) return PATCHKV_E_VALUE;
  if (rho != 0 && rho != 1) return PATCHKV_E_VALUE;
  if (!valid_ridge_mode(ridge_mode)) return PATCHKV_E_VALUE;
  if (!al16(Q) || !al16(K) || !al16(V) || !al16(W) || (!idx && (!al16(Kc) || !al16(Vc))))
    return PATCHKV_E_VALUE;
  const LayerWs L = layer_ws(dtype, acc_dtype, M, N, B, Hq, Hkv, dh);
  s = check_ws(workspace, workspace_bytes, L.total);
  if (s) return s;

  hipStream_t st = (hipStream_t)stream;
  char* w = (char*)workspace;
  float* Of = (float*)(w + L.Of);
  float* Oc = (float*)(w + L.Oc);
  void* T = w + L.T;
  void* G = w + L.G;
  void* C = w + L.C;
  void* wa = w + L.attn;
  void* wsv = w + L.solve;
  int32_t* stat = (int32_t*)(w + L.stat);

  const CacheIndex ci = cache_index(idx, idx_mode, counts, B);
  hipError_t e = launch_idx_check(ci, Hkv, B, idx ? N : B, stat, st);
  if (e != hipSuccess) return PATCHKV_E_HIP;
  e = launch_attention(attn_shape(dtype, M, N, Hq, Hkv, dh), Q, K, V, CacheIndex{}, N, N, scale,
                       false, Of, wa, st);
  if (e != hipSuccess) return PATCHKV_E_HIP;
  if (idx)
    e = launch_attention(attn_shape(dtype, M, B, Hq, Hkv, dh), Q, K, V, ci, N, N, scale, true, Oc,
                         wa, st);
  else
    e = launch_attention(attn_shape(dtype, M, B, Hq, Hkv, dh), Q, Kc, Vc, ci, B, B, scale, true,
                         Oc, wa, st);
  if (e != hipSuccess) return PATCHKV_E_HIP;
  const bool wbf = dtype == PATCHKV_BF16;
  if (acc_dtype == PATCHKV_F32) {
    e = launch_targets(Of, Oc, W, wbf, M, d, d, rho, (float*)T, wa, st);
    if (e == hipSuccess)
      e = launch_normal_eq_f32(Oc, (const float*)T, nullptr, M, d, d, false, (float*)G, (float*)C,
                               wa, st);
  } else {
    e = launch_targets_f64(Of, Oc, W, wbf, M, d, d, rho, (double*)T, st);
    if (e == hipSuccess)
      e = launch_normal_eq_f64(Oc, nullptr, nullptr, (const double*)T, M, d, d, false, (double*)G,
                               (double*)C, st);
  }
  if (e != hipSuccess) return PATCHKV_E_HIP;
  e = launch_solve(acc_dtype == PATCHKV_F64, G, C, d, d, lambda, ridge_kind(ridge_mode),
                   products(ridge_mode), dW, info, wsv, st);
  if (e == hipSuccess) e = launch_info_merge(stat, info, st);
  return status_of(e);
}

}  // extern "C"
