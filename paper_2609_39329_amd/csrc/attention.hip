// Attention launchers: the work plan, the V^T pre-pass and the kernel choice (kernels
// in attention_kernels.hpp), the block-scaled expansion for the f32 path, the index
// check and the fixed scratch of the allocation-free entry point.
#include <math.h>

#include <mutex>

#include "attention_kernels.hpp"

namespace pkv {

namespace {

// Block-scaled integer cache -> rows [Hkv][n_cache][dh] of OUT (bf16 or f32). Entry n
// of head g is source row idx[g * idx_stride + n] (or n); rows outside [0, n_src), and
// entries at or past the head's count, read as zeros. Exact: an int8 or int4 value
// times a power of two is a bf16 number. One thread per 8 channels.
template <class OUT, int BITS>
__global__ __launch_bounds__(256) void mx_dequant_kernel(const uint8_t* __restrict__ q,
                                                         const int8_t* __restrict__ e,
                                                         const int32_t* __restrict__ idx,
                                                         int idx_stride,
                                                         const int32_t* __restrict__ counts,
                                                         int64_t n_src, int n_cache, int dh,
                                                         OUT* __restrict__ out) {
  const int g = blockIdx.y;
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per_row = dh / 8;
  if (t >= (int64_t)n_cache * per_row) return;
  const int n = (int)(t / per_row), c0 = (int)(t % per_row) * 8;
  const int nk = counts ? min(max(counts[g], 1), n_cache) : n_cache;
  const int64_t src = n >= nk ? -1 : idx ? (int64_t)idx[(int64_t)g * idx_stride + n] : (int64_t)n;
  float v[8] = {};
  if (src >= 0 && src < n_src) {
    const int64_t row = (int64_t)g * n_src + src;
    const int ex = e[row * (dh / 32) + c0 / 32];
    if constexpr (BITS == 8) {
      const uint2 w = *(const uint2*)(q + row * dh + c0);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const uint32_t word = i < 4 ? w.x : w.y;
        v[i] = ldexpf((float)(int8_t)(word >> (8 * (i & 3))), ex);
      }
    } else {
      const uint32_t w = *(const uint32_t*)(q + row * (dh / 2) + c0 / 2);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int nib = (int)((w >> (4 * i)) & 0xF);
        v[i] = ldexpf((float)(nib >= 8 ? nib - 16 : nib), ex);
      }
    }
  }
  OUT* o = out + ((int64_t)g * n_cache + n) * dh + c0;
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = (OUT)v[i];
}

}  // namespace

AttnPlan plan_attention(const AttnShape& s) {
  AttnPlan pl{};
  const int64_t rows = s.M * (s.Hq / s.Hkv);
  const int rows_wg = s.bf16 ? kRowsBf16 : kRowsF32;
  pl.row_tiles = (int)((rows + rows_wg - 1) / rows_wg);
  const int kt = s.bf16 ? kKeyTile : kKeyTileF32;
  const int64_t ntiles = (s.Nk + kt - 1) / kt;
  const int64_t items = (int64_t)s.Hkv * pl.row_tiles;
  // Pick the number of key ranges that minimises (rounds of workgroups) x (tiles
  // per workgroup) plus the merge traffic, on 256 CUs.
  const double slots = 256.0 * (s.bf16 ? kWgPerCu : 1);
  // one bf16 tile-iteration of a workgroup ~ 64 x rows x dh x 4 flops at ~4 TFLOP/s per CU
  // (shared by the workgroups resident on the CU)
  const double tile_s = (double)kt * rows_wg * s.dh * 4.0 / (s.bf16 ? 4e12 / kWgPerCu : 0.45e12);
  double best = 1e300;
  int best_s = 1;
  for (int sp = 1; sp <= 64 && sp <= ntiles; ++sp) {
    const int64_t tps = (ntiles + sp - 1) / sp;
    const int64_t waves = (items * sp + (int64_t)slots - 1) / (int64_t)slots;
    double cost = (double)waves * tps * tile_s;
    if (sp > 1) cost += (double)s.Hkv * rows * (s.dh + 2) * 4.0 * sp * 2 / 4e12 + 4e-6;
    if (cost < best * 0.98) {
      best = cost;
      best_s = sp;
    }
  }
  const int64_t tps = (ntiles + best_s - 1) / best_s;
  pl.keys_per_split = (int)(tps * kt);
  pl.n_split = (int)((s.Nk + pl.keys_per_split - 1) / pl.keys_per_split);
  pl.total_items = (int)(items * pl.n_split);
  pl.per_xcd = (pl.total_items + kXcds - 1) / kXcds;
  pl.grid = pl.per_xcd * kXcds;
  pl.ws_bytes = pl.n_split > 1
                    ? align_up((size_t)s.Hkv * pl.n_split * rows * s.dh * sizeof(float)) +
                          align_up((size_t)s.Hkv * pl.n_split * rows * 2 * sizeof(float))
                    : 0;
  if (s.bf16) {
    pl.ws_bytes += align_up((size_t)pl.total_items * sizeof(int));
    pl.ws_bytes += align_up((size_t)s.Hkv * ntiles * 32 * s.dh * 2);  // V^T tiles
    if (s.Ms > 0)  // V^T tiles of the own entries
      pl.ws_bytes += align_up((size_t)s.Hkv * ((s.Ms + kKeyTile - 1) / kKeyTile) * 32 * s.dh * 2);
  }
  return pl;
}

hipError_t launch_attention(const AttnShape& s, const void* Q, const void* K, const void* V,
                            const CacheIndex& ci, int64_t src_rows, int64_t src_valid,
                            float scale, bool psplit, float* O, void* ws, hipStream_t st,
                            const void* Ks, const void* Vs, const float* bias, const KvQuant& kq) {
  if (kq.bits != 0 && ((kq.bits != 8 && kq.bits != 4) || !s.bf16 || s.Ms > 0 || !kq.Ke || !kq.Ve))
    return hipErrorInvalidValue;
  const AttnPlan pl = plan_attention(s);
  AttnParams p{};
  p.idx = ci.idx;
  p.idx_stride = (int)ci.stride;
  p.counts = ci.counts;
  p.bias = bias;
  p.bias_mul = s.bf16 ? 1.0f / scale : 1.0f;
  p.Q = Q;
  p.K = K;
  p.V = V;
  p.Ke = kq.Ke;
  p.Ve = kq.Ve;
  p.O = O;
  p.Ks = Ks;
  p.Vs = Vs;
  p.Ms = (int)s.Ms;
  size_t off = 0;
  if (pl.n_split > 1) {
    const size_t n = (size_t)s.Hkv * pl.n_split * s.M * (s.Hq / s.Hkv);
    p.Opart = (float*)ws;
    off += align_up(n * s.dh * sizeof(float));
    p.ML = (float*)((char*)ws + off);
    off += align_up(n * 2 * sizeof(float));
  }
  const int64_t vt_tiles = (s.Nk + kKeyTile - 1) / kKeyTile;
  if (s.bf16) {
    p.flags = (int*)((char*)ws + off);
    off += align_up((size_t)pl.total_items * sizeof(int));
    p.Vt = (const __bf16*)((char*)ws + off);  // V^T tiles of the cache
    p.vt_tiles = (int)vt_tiles;
    if (s.Ms > 0) {  // then those of the chunk's own entries
      off += align_up((size_t)s.Hkv * vt_tiles * 32 * s.dh * 2);
      p.Vts = (const __bf16*)((char*)ws + off);
      p.own_tiles = (int)((s.Ms + kKeyTile - 1) / kKeyTile);
    }
  }
  p.Hq = s.Hq;
  p.G = s.Hq / s.Hkv;
  p.src_rows = src_rows;
  p.src_valid = (int)src_valid;
  p.Nk = (int)s.Nk;
  p.n_split = pl.n_split;
  p.keys_per_split = pl.keys_per_split;
  p.rows = (int)(s.M * p.G);
  p.row_tiles = pl.row_tiles;
  p.total_items = pl.total_items;
  p.per_xcd = pl.per_xcd;
  p.c = s.bf16 ? scale * 1.4426950408889634f : scale;
  const bool gather = ci.idx != nullptr;
  if (kq.bits) return run_attention_mx(s, pl, p, kq.bits, gather, psplit, st);
  if (s.dh == 128) return run_attention<128, 0>(s, pl, p, gather, psplit, st);
  return run_attention<64, 0>(s, pl, p, gather, psplit, st);
}

}  // namespace pkv

namespace pkv {

hipError_t launch_mx_dequant(bool bf16, int bits, const void* q, const int8_t* e,
                             const CacheIndex& ci, int64_t n_src, int64_t n_cache, int Hkv, int dh,
                             void* out, hipStream_t st) {
  const int64_t n = n_cache * (dh / 8);
  const dim3 grid((unsigned)((n + 255) / 256), (unsigned)Hkv), block(256);
  const uint8_t* qb = (const uint8_t*)q;
  const int is = (int)ci.stride;
  if (bf16) {
    if (bits == 8)
      hipLaunchKernelGGL((mx_dequant_kernel<__bf16, 8>), grid, block, 0, st, qb, e, ci.idx, is,
                         ci.counts, n_src, (int)n_cache, dh, (__bf16*)out);
    else
      hipLaunchKernelGGL((mx_dequant_kernel<__bf16, 4>), grid, block, 0, st, qb, e, ci.idx, is,
                         ci.counts, n_src, (int)n_cache, dh, (__bf16*)out);
  } else {
    if (bits == 8)
      hipLaunchKernelGGL((mx_dequant_kernel<float, 8>), grid, block, 0, st, qb, e, ci.idx, is,
                         ci.counts, n_src, (int)n_cache, dh, (float*)out);
    else
      hipLaunchKernelGGL((mx_dequant_kernel<float, 4>), grid, block, 0, st, qb, e, ci.idx, is,
                         ci.counts, n_src, (int)n_cache, dh, (float*)out);
  }
  return hipGetLastError();
}

namespace {

// Validity of a compressed cache's index set, one workgroup. Codes: an entry at flat
// position q of idx (q = b for a shared set, g * B + b per head; only b below the
// head's count is looked at) outside [0, n_src) has code q; a count outside [1, B] has
// code E + g, E = the number of entries of idx (0 without idx). info = 0 if nothing
// is out of range, else -(1 + the smallest code). Deterministic; needs no cleared
// memory.
__global__ __launch_bounds__(1024) void idx_check_kernel(const int32_t* __restrict__ idx,
                                                         int64_t stride,
                                                         const int32_t* __restrict__ counts,
                                                         int heads, int64_t B, int64_t n_src,
                                                         int32_t* __restrict__ info) {
  __shared__ long long red[1024 / kWave];
  const long long none = 1ll << 62;
  const long long E = idx ? (stride ? (long long)heads * B : (long long)B) : 0;
  long long best = none;
  for (int g = 0; g < heads; ++g) {
    const long long cnt = counts ? (long long)counts[g] : (long long)B;
    if (cnt < 1 || cnt > B) best = min(best, E + g);
    if (!idx || (stride == 0 && g > 0 && !counts)) continue;
    const long long n = min(max(cnt, 1ll), (long long)B);
    const int32_t* ig = idx + g * stride;
    for (long long b = threadIdx.x; b < n; b += blockDim.x) {
      const int32_t v = ig[b];
      if (v < 0 || (long long)v >= n_src) best = min(best, (long long)g * stride + b);
    }
  }
  for (int o = kWave / 2; o > 0; o >>= 1) best = min(best, (long long)__shfl_xor(best, o));
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = best;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 1; i < (int)(blockDim.x / kWave); ++i) best = min(best, red[i]);
    *info = best == none ? 0 : (int32_t)-(min(best, (long long)INT32_MAX - 1) + 1);
  }
}

// info <- status when status is non-zero (an input error outranks a later result)
__global__ void info_merge_kernel(const int32_t* __restrict__ status, int32_t* __restrict__ info) {
  if (threadIdx.x == 0 && *status != 0) *info = *status;
}

}  // namespace

hipError_t launch_idx_check(const CacheIndex& ci, int heads, int64_t B, int64_t n_src,
                            int32_t* info, hipStream_t st) {
  hipLaunchKernelGGL(idx_check_kernel, dim3(1), dim3(1024), 0, st, ci.idx, ci.stride, ci.counts,
                     heads, B, n_src, info);
  return hipGetLastError();
}

hipError_t launch_info_merge(const int32_t* status, int32_t* info, hipStream_t st) {
  hipLaunchKernelGGL(info_merge_kernel, dim3(1), dim3(64), 0, st, status, info);
  return hipGetLastError();
}

// Fixed scratch of the allocation-free compressed-cache attention: a file-scope
// device array (zero-initialised, held by every GPU the library runs on until the
// process ends). Host code never passes the array's name to a kernel: that name is a
// host-side stand-in. Its device address is looked up once per device.
static __device__ __align__(256) unsigned char scratch[kNoallocScratchBytes];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** ptr) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace pkv
