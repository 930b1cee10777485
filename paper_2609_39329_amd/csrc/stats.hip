// Targets and sufficient statistics (Eq. 5 and Eq. 9, row form):
//   T = (O_f - O_c) W + rho (O_f - O_c)
//   G (+)= X^T X,   C (+)= X^T (Yf - Yc)
//
// fp32-accumulate path (split_gemm_kernel): gfx950 has no fp32-input MFMA faster
// than 157 TFLOP/s and no xf32 mode, so every fp32 operand x is split into
// x_hi = bf16(x) and x_lo = bf16(x - x_hi) while it is staged from HBM into LDS,
// and the product is formed on bf16 MFMA 32x32x16 with fp32 accumulation:
//   x y ~ x_hi y_hi + x_hi y_lo + x_lo y_hi (+ x_lo y_lo for the Gram matrix).
// Dropping x_lo y_lo in G would subtract a PSD matrix L^T L whose diagonal grows
// with the number of rows (a systematic shift of the ridge), so G keeps all four
// products; C keeps three (its lo x lo cross term has no such bias). A bf16
// operand (W) has no low part. Operands whose contraction index is contiguous
// in memory are stored [i][k] in LDS and read with 16-byte reads; operands whose
// output index is contiguous (X^T for the Gram, W for the targets) are stored
// [k][i] and read with the LDS transpose instruction. G is computed on the upper
// block triangle only and mirrored.
//
// fp64-accumulate path (f64_gemm_kernel): plain fp64 FMA tiles through LDS.
#include "common.hpp"
#include "kernels.hpp"

namespace pkv {

namespace {

constexpr int BM = 128, BN = 128, KC = 32;

struct SplitParams {
  const float* A1;   // A(i,k) = A1 - A2 (A2 may be null)
  const float* A2;
  int64_t lda;
  const void* B1;    // B(j,k) = B1 - B2 (B2 may be null; B1 float or bf16)
  const float* B2;
  int64_t ldb;
  float* Out;
  int64_t ldo;
  const float* E1;   // epilogue: + rho (E1 - E2)[i][j]
  const float* E2;
  int64_t lde;
  float rho;
  int I, J, K;
  int accumulate;
  int tiles_j;
  int ntiles;
  bool vecA, vecB;   // 16-byte loads allowed (strides and bases aligned)
};

// AK: A(i,k) at A[i*lda + k] (else A[k*lda + i]); BK likewise for B(j,k).
template <bool AK, bool BK, bool B_BF16, bool SYM, int NTERMS>
__global__ __launch_bounds__(256, 1) void split_gemm_kernel(SplitParams p) {
  // LDS tiles, hi and lo parts. [i][k] layout pitch KC+8, [k][i] layout pitch BM+16.
  constexpr int PA = AK ? (KC + 8) : (BM + 16);
  constexpr int PB = BK ? (KC + 8) : (BN + 16);
  constexpr int SA = AK ? BM * PA : KC * PA;
  constexpr int SB = BK ? BN * PB : KC * PB;
  __shared__ __attribute__((aligned(16))) __bf16 Ah[SA];
  __shared__ __attribute__((aligned(16))) __bf16 Al[SA];
  __shared__ __attribute__((aligned(16))) __bf16 Bh[SB];
  __shared__ __attribute__((aligned(16))) __bf16 Bl[B_BF16 ? 8 : SB];

  int ti, tj;
  {
    const int t = xcd_item((p.ntiles + kXcds - 1) / kXcds);
    if (t >= p.ntiles) return;
    if constexpr (SYM) {
      // upper block triangle, row-major enumeration
      int r = 0, rem = t;
      while (rem >= p.tiles_j - r) {
        rem -= p.tiles_j - r;
        ++r;
      }
      ti = r;
      tj = r + rem;
    } else {
      ti = t / p.tiles_j;
      tj = t % p.tiles_j;
    }
  }
  const int i0 = ti * BM, j0 = tj * BN;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int h32 = lane >> 5, l32 = lane & 31;
  const int wi = (wid >> 1) * 64, wj = (wid & 1) * 64;

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  // staging registers: A and B tiles of 128 x 32 floats (4 float4 per thread).
  // The 4 (or 8) elements one thread loads are contiguous in memory.
  f32x4 ra[4], rb[4];
  u32x4 rbw[2];
  auto ld4 = [](const float* s1, const float* s2, int nvalid, bool vec) -> f32x4 {
    f32x4 v = {};
    if (nvalid >= 4 && vec) {
      v = *(const f32x4*)s1;
      if (s2) v -= *(const f32x4*)s2;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (e < nvalid) v[e] = s1[e] - (s2 ? s2[e] : 0.f);
    }
    return v;
  };
  auto fetch = [&](int k0) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = u * 256 + tid;
      int i, k;
      if constexpr (AK) { i = c / (KC / 4); k = (c % (KC / 4)) * 4; }
      else { k = c / (BM / 4); i = (c % (BM / 4)) * 4; }
      const int gi = i0 + i, gk = k0 + k;
      const int64_t off = AK ? (int64_t)gi * p.lda + gk : (int64_t)gk * p.lda + gi;
      const int nvalid = AK ? (gi < p.I ? p.K - gk : 0) : (gk < p.K ? p.I - gi : 0);
      ra[u] = nvalid > 0 ? ld4(p.A1 + off, p.A2 ? p.A2 + off : nullptr, nvalid, p.vecA)
                         : f32x4{};
    }
    if constexpr (B_BF16) {
      // B(j,k) = W[k][j], bf16, [k][j] layout: 32 x 128 bf16 = 512 chunks of 16 B
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = u * 256 + tid;
        const int k = c / (BN / 8), j = (c % (BN / 8)) * 8;
        const int gk = k0 + k, gj = j0 + j;
        const int nvalid = gk < p.K ? p.J - gj : 0;
        u32x4 v = {};
        if (nvalid > 0) {
          const __bf16* s = (const __bf16*)p.B1 + (int64_t)gk * p.ldb + gj;
          if (nvalid >= 8 && p.vecB) {
            v = *(const u32x4*)s;
          } else {
            bf16x8 t8 = __builtin_bit_cast(bf16x8, v);
#pragma unroll
            for (int e = 0; e < 8; ++e)
              if (e < nvalid) t8[e] = s[e];
            v = __builtin_bit_cast(u32x4, t8);
          }
        }
        rbw[u] = v;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = u * 256 + tid;
        int j, k;
        if constexpr (BK) { j = c / (KC / 4); k = (c % (KC / 4)) * 4; }
        else { k = c / (BN / 4); j = (c % (BN / 4)) * 4; }
        const int gj = j0 + j, gk = k0 + k;
        const int64_t off = BK ? (int64_t)gj * p.ldb + gk : (int64_t)gk * p.ldb + gj;
        const int nvalid = BK ? (gj < p.J ? p.K - gk : 0) : (gk < p.K ? p.J - gj : 0);
        rb[u] = nvalid > 0 ? ld4((const float*)p.B1 + off, p.B2 ? p.B2 + off : nullptr, nvalid,
                                 p.vecB)
                           : f32x4{};
      }
    }
  };
  auto split_store = [&](__bf16* hi, __bf16* lo, int off, f32x4 v) {
    bf16x4 h, l;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      h[e] = to_bf16(v[e]);
      l[e] = to_bf16(v[e] - (float)h[e]);
    }
    *(bf16x4*)(hi + off) = h;
    *(bf16x4*)(lo + off) = l;
  };
  auto stash = [&]() {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = u * 256 + tid;
      if constexpr (AK) split_store(Ah, Al, (c / (KC / 4)) * PA + (c % (KC / 4)) * 4, ra[u]);
      else split_store(Ah, Al, (c / (BM / 4)) * PA + (c % (BM / 4)) * 4, ra[u]);
    }
    if constexpr (B_BF16) {
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        const int c = u * 256 + tid;
        *(u32x4*)(Bh + (c / (BN / 8)) * PB + (c % (BN / 8)) * 8) = rbw[u];
      }
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = u * 256 + tid;
        if constexpr (BK) split_store(Bh, Bl, (c / (KC / 4)) * PB + (c % (KC / 4)) * 4, rb[u]);
        else split_store(Bh, Bl, (c / (BN / 4)) * PB + (c % (BN / 4)) * 4, rb[u]);
      }
    }
  };

  // operand fragment (32 rows x 16 k) at row offset r0 and k offset k0 of an LDS tile
  const int tr_k = 8 * h32 + ((lane & 15) >> 2);
  const int tr_i = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
  auto frag = [&](const __bf16* base, int pitch, bool kcontig, int r0, int k0) -> bf16x8 {
    if (kcontig) return *(const bf16x8*)(base + (r0 + l32) * pitch + k0 + h32 * 8);
    const PKV_LDS __bf16* q = (const PKV_LDS __bf16*)(base + (k0 + tr_k) * pitch + r0 + tr_i);
    return cat8(lds_read_tr16(q), lds_read_tr16(q + 4 * pitch));
  };

  fetch(0);
  for (int k0 = 0; k0 < p.K; k0 += KC) {
    __syncthreads();
    stash();
    __syncthreads();
    if (k0 + KC < p.K) fetch(k0 + KC);
#pragma unroll
    for (int ks = 0; ks < KC; ks += 16) {
      bf16x8 ah[2], al[2], bh[2], bl[2];
#pragma unroll
      for (int a = 0; a < 2; ++a) {
        ah[a] = frag(Ah, PA, AK, wi + 32 * a, ks);
        al[a] = frag(Al, PA, AK, wi + 32 * a, ks);
      }
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        bh[b] = frag(Bh, PB, BK, wj + 32 * b, ks);
        if constexpr (!B_BF16) bl[b] = frag(Bl, PB, BK, wj + 32 * b, ks);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) {
          acc[a][b] = mfma32(ah[a], bh[b], acc[a][b]);
          acc[a][b] = mfma32(al[a], bh[b], acc[a][b]);
          if constexpr (!B_BF16) {
            acc[a][b] = mfma32(ah[a], bl[b], acc[a][b]);
            if constexpr (NTERMS == 4) acc[a][b] = mfma32(al[a], bl[b], acc[a][b]);
          }
        }
    }
  }

  // epilogue
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = i0 + wi + 32 * a + 8 * (e >> 2) + 4 * h32 + (e & 3);
        const int j = j0 + wj + 32 * b + l32;
        if (i >= p.I || j >= p.J) continue;
        // diagonal tiles of G: keep the i <= j triangle and mirror it, so G is
        // exactly symmetric (the two triangles accumulate their terms in
        // different orders)
        if (SYM && ti == tj && i > j) continue;
        float v = acc[a][b][e];
        if (p.E1) v += p.rho * (p.E1[(int64_t)i * p.lde + j] - p.E2[(int64_t)i * p.lde + j]);
        float* o = p.Out + (int64_t)i * p.ldo + j;
        *o = p.accumulate ? *o + v : v;
        if constexpr (SYM) {
          if (i != j) {
            float* o2 = p.Out + (int64_t)j * p.ldo + i;
            *o2 = p.accumulate ? *o2 + v : v;
          }
        }
      }
}

// ---------------------------------------------------------------- fp64 path

template <class T>
__device__ __forceinline__ double ld64(const T* p, int64_t i) {
  return (double)p[i];
}
template <>
__device__ __forceinline__ double ld64<__bf16>(const __bf16* p, int64_t i) {
  return (double)(float)p[i];
}

template <class TA, class TB>
struct F64Params {
  const TA* A1;
  const TA* A2;
  int64_t sai, sak;
  const TB* B1;
  const TB* B2;
  int64_t sbj, sbk;
  double* Out;
  int64_t ldo;
  const float* E1;
  const float* E2;
  int64_t lde;
  double rho;
  int I, J, K;
  int accumulate;
  int tiles_j;
};

// Out[i][j] (+)= sum_k A(i,k) B(j,k) (+ rho E), all products and sums in fp64.
template <class TA, class TB>
__global__ __launch_bounds__(256) void f64_gemm_kernel(F64Params<TA, TB> p) {
  constexpr int T = 64, KC2 = 16;
  __shared__ double As[KC2][T + 1];
  __shared__ double Bs[KC2][T + 1];
  const int i0 = (blockIdx.x / p.tiles_j) * T, j0 = (blockIdx.x % p.tiles_j) * T;
  const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
  double acc[4][4] = {};
  for (int k0 = 0; k0 < p.K; k0 += KC2) {
    for (int e = tid; e < T * KC2; e += 256) {
      int i, k;
      if (p.sak == 1) { i = e / KC2; k = e % KC2; } else { k = e / T; i = e % T; }
      double v = 0.0;
      const int gi = i0 + i, gk = k0 + k;
      if (gi < p.I && gk < p.K) {
        const int64_t o = (int64_t)gi * p.sai + (int64_t)gk * p.sak;
        v = ld64(p.A1, o) - (p.A2 ? ld64(p.A2, o) : 0.0);
      }
      As[k][i] = v;
      int j, kb;
      if (p.sbk == 1) { j = e / KC2; kb = e % KC2; } else { kb = e / T; j = e % T; }
      double w = 0.0;
      const int gj = j0 + j, gkb = k0 + kb;
      if (gj < p.J && gkb < p.K) {
        const int64_t o = (int64_t)gj * p.sbj + (int64_t)gkb * p.sbk;
        w = ld64(p.B1, o) - (p.B2 ? ld64(p.B2, o) : 0.0);
      }
      Bs[kb][j] = w;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < KC2; ++k) {
      double a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = As[k][ty * 4 + u];
        b[u] = Bs[k][tx * 4 + u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[u][v] = fma(a[u], b[v], acc[u][v]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int i = i0 + ty * 4 + u, j = j0 + tx * 4 + v;
      if (i >= p.I || j >= p.J) continue;
      double r = acc[u][v];
      if (p.E1)
        r += p.rho * ((double)p.E1[(int64_t)i * p.lde + j] - (double)p.E2[(int64_t)i * p.lde + j]);
      double* o = p.Out + (int64_t)i * p.ldo + j;
      *o = p.accumulate ? *o + r : r;
    }
}

template <class TA, class TB>
hipError_t run_f64(F64Params<TA, TB> p, hipStream_t st) {
  p.tiles_j = (p.J + 63) / 64;
  const int ti = (p.I + 63) / 64;
  hipLaunchKernelGGL((f64_gemm_kernel<TA, TB>), dim3(ti * p.tiles_j), dim3(256), 0, st, p);
  return hipGetLastError();
}

SplitParams base_params(int I, int J, int K) {
  SplitParams p{};
  p.I = I;
  p.J = J;
  p.K = K;
  return p;
}

bool al16(const void* q) { return ((uintptr_t)q & 15) == 0; }

void set_vec(SplitParams& p, bool b_bf16) {
  p.vecA = p.lda % 4 == 0 && al16(p.A1) && al16(p.A2);
  p.vecB = p.ldb % (b_bf16 ? 8 : 4) == 0 && al16(p.B1) && al16(p.B2);
}

}  // namespace

size_t targets_ws_bytes(int64_t, int64_t, int64_t) { return 0; }
size_t normal_eq_ws_bytes(int64_t, int64_t, int64_t) { return 0; }

hipError_t launch_targets(const float* Of, const float* Oc, const void* W, bool w_bf16, int64_t M,
                          int64_t din, int64_t dout, int rho, float* T, void*, hipStream_t st) {
  SplitParams p = base_params((int)M, (int)dout, (int)din);
  p.A1 = Of;
  p.A2 = Oc;
  p.lda = din;
  p.B1 = W;
  p.ldb = dout;
  p.Out = T;
  p.ldo = dout;
  if (rho) {
    p.E1 = Of;
    p.E2 = Oc;
    p.lde = din;
    p.rho = (float)rho;
  }
  p.tiles_j = (int)((dout + BN - 1) / BN);
  p.ntiles = (int)((M + BM - 1) / BM) * p.tiles_j;
  set_vec(p, w_bf16);
  dim3 grid((p.ntiles + kXcds - 1) / kXcds * kXcds), block(256);
  if (w_bf16)
    hipLaunchKernelGGL((split_gemm_kernel<true, false, true, false, 2>), grid, block, 0, st, p);
  else
    hipLaunchKernelGGL((split_gemm_kernel<true, false, false, false, 3>), grid, block, 0, st, p);
  return hipGetLastError();
}

hipError_t launch_normal_eq_f32(const float* X, const float* Yf, const float* Yc, int64_t rows,
                                int64_t din, int64_t dout, bool accumulate, float* G, float* C,
                                void*, hipStream_t st) {
  {  // G = X^T X on the upper block triangle, mirrored
    SplitParams p = base_params((int)din, (int)din, (int)rows);
    p.A1 = X;
    p.lda = din;
    p.B1 = X;
    p.ldb = din;
    p.Out = G;
    p.ldo = din;
    p.accumulate = accumulate;
    p.tiles_j = (int)((din + BN - 1) / BN);
    p.ntiles = p.tiles_j * (p.tiles_j + 1) / 2;
    set_vec(p, false);
    dim3 grid((p.ntiles + kXcds - 1) / kXcds * kXcds), block(256);
    hipLaunchKernelGGL((split_gemm_kernel<false, false, false, true, 4>), grid, block, 0, st, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  SplitParams p = base_params((int)din, (int)dout, (int)rows);
  p.A1 = X;
  p.lda = din;
  p.B1 = Yf;
  p.B2 = Yc;
  p.ldb = dout;
  p.Out = C;
  p.ldo = dout;
  p.accumulate = accumulate;
  p.tiles_j = (int)((dout + BN - 1) / BN);
  p.ntiles = (int)((din + BM - 1) / BM) * p.tiles_j;
  set_vec(p, false);
  dim3 grid((p.ntiles + kXcds - 1) / kXcds * kXcds), block(256);
  hipLaunchKernelGGL((split_gemm_kernel<false, false, false, false, 3>), grid, block, 0, st, p);
  return hipGetLastError();
}

hipError_t launch_targets_f64(const float* Of, const float* Oc, const void* W, bool w_bf16,
                              int64_t M, int64_t din, int64_t dout, int rho, double* T,
                              hipStream_t st) {
  if (w_bf16) {
    F64Params<float, __bf16> p{};
    p.A1 = Of; p.A2 = Oc; p.sai = din; p.sak = 1;
    p.B1 = (const __bf16*)W; p.sbj = 1; p.sbk = dout;
    p.Out = T; p.ldo = dout;
    if (rho) { p.E1 = Of; p.E2 = Oc; p.lde = din; p.rho = rho; }
    p.I = (int)M; p.J = (int)dout; p.K = (int)din;
    return run_f64(p, st);
  }
  F64Params<float, float> p{};
  p.A1 = Of; p.A2 = Oc; p.sai = din; p.sak = 1;
  p.B1 = (const float*)W; p.sbj = 1; p.sbk = dout;
  p.Out = T; p.ldo = dout;
  if (rho) { p.E1 = Of; p.E2 = Oc; p.lde = din; p.rho = rho; }
  p.I = (int)M; p.J = (int)dout; p.K = (int)din;
  return run_f64(p, st);
}

hipError_t launch_normal_eq_f64(const float* X, const float* Yf, const float* Yc, const double* Yd,
                                int64_t rows, int64_t din, int64_t dout, bool accumulate,
                                double* G, double* C, hipStream_t st) {
  {
    F64Params<float, float> p{};
    p.A1 = X; p.sai = 1; p.sak = din;
    p.B1 = X; p.sbj = 1; p.sbk = din;
    p.Out = G; p.ldo = din; p.accumulate = accumulate;
    p.I = (int)din; p.J = (int)din; p.K = (int)rows;
    hipError_t e = run_f64(p, st);
    if (e != hipSuccess) return e;
  }
  if (Yd) {
    F64Params<float, double> p{};
    p.A1 = X; p.sai = 1; p.sak = din;
    p.B1 = Yd; p.sbj = 1; p.sbk = dout;
    p.Out = C; p.ldo = dout; p.accumulate = accumulate;
    p.I = (int)din; p.J = (int)dout; p.K = (int)rows;
    return run_f64(p, st);
  }
  F64Params<float, float> p{};
  p.A1 = X; p.sai = 1; p.sak = din;
  p.B1 = Yf; p.B2 = Yc; p.sbj = 1; p.sbk = dout;
  p.Out = C; p.ldo = dout; p.accumulate = accumulate;
  p.I = (int)din; p.J = (int)dout; p.K = (int)rows;
  return run_f64(p, st);
}

}  // namespace pkv
