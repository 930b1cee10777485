// Ridge patch, Eq. 8 in row form: dW = (G + lambda I)^{-1} C.
//
// Right-looking blocked Cholesky with block size NB, fused with the forward
// substitution of the right-hand side:
//   for each block column k:
//     potrf_inv_kernel   A_kk = L_kk L_kk^T in LDS, then L_kk^{-1} in place (1 WG)
//     grouped GEMM       L_ik = A_ik L_kk^{-T} (i > k);  Z_k = L_kk^{-1} R_k
//     grouped GEMM       A_ij -= L_ik L_jk^T (lower blocks);  R_i -= L_ik Z_k (i > k)
//   then backward:  X_k = L_kk^{-T} Z_k;  Z_i -= L_ki^T X_k (i < k), k descending.
// Triangular solves against a diagonal block use that block's explicit inverse (a
// GEMM instead of a substitution); its condition number is at most the square root
// of that of G + lambda I.
// fp32 (acc F32) GEMM tiles run on MFMA 32x32x2 f32; fp64 (acc F64) on fp64 FMA.
// The adaptive ridge of Eq. 7, lambda_0 ||G||_F^2 / tr G, is reduced on the device
// in fp64 in a fixed order (deterministic).
#include <math.h>

#include <algorithm>

#include "common.hpp"
#include "kernels.hpp"

namespace pkv {

namespace {

constexpr int NB = 128;      // Cholesky block size
constexpr int GT = 64;       // GEMM tile
constexpr int GK = 32;       // GEMM k chunk
constexpr int kRedBlocks = 256;

template <class T>
struct GemmDesc {
  const T* A;      // A(i,k) = A[i*sai + k*sak]
  int64_t sai, sak;
  const T* B;      // B(k,j) = B[k*sbk + j*sbj]
  int64_t sbk, sbj;
  T* C;            // C[i*ldc + j] = beta C + alpha sum_k A(i,k) B(k,j)
  int64_t ldc;
  int M, N, K;
  T alpha, beta;
  int lower;       // only tiles with tile_row >= tile_col
  int tiles_n;
  int ntiles;
};

template <class T>
struct GemmGroup {
  GemmDesc<T> d[2];
  int n;
};

template <class T>
__global__ __launch_bounds__(256) void solve_gemm_kernel(GemmGroup<T> grp) {
  __shared__ T As[GK][GT + 4];
  __shared__ T Bs[GK][GT + 4];
  int t = blockIdx.x;
  int which = 0;
  if (t >= grp.d[0].ntiles) {
    t -= grp.d[0].ntiles;
    which = 1;
    if (which >= grp.n || t >= grp.d[1].ntiles) return;
  }
  const GemmDesc<T>& g = grp.d[which];
  const int ti = t / g.tiles_n, tj = t % g.tiles_n;
  if (g.lower && tj > ti) return;
  const int i0 = ti * GT, j0 = tj * GT;
  const int tid = threadIdx.x;

  f32x16 acc32 = {};
  double acc64[4][4] = {};
  const int lane = tid & 63, wid = tid >> 6;
  const int wi = (wid >> 1) * 32, wj = (wid & 1) * 32;
  const int ty = tid / 16, tx = tid % 16;

  for (int k0 = 0; k0 < g.K; k0 += GK) {
    for (int e = tid; e < GT * GK; e += 256) {
      int i, k;
      if (g.sak == 1) { i = e / GK; k = e % GK; } else { k = e / GT; i = e % GT; }
      const int gi = i0 + i, gk = k0 + k;
      As[k][i] = (gi < g.M && gk < g.K) ? g.A[(int64_t)gi * g.sai + (int64_t)gk * g.sak] : T(0);
      int j, kb;
      if (g.sbj == 1) { kb = e / GT; j = e % GT; } else { j = e / GK; kb = e % GK; }
      const int gj = j0 + j, gkb = k0 + kb;
      Bs[kb][j] = (gj < g.N && gkb < g.K) ? g.B[(int64_t)gkb * g.sbk + (int64_t)gj * g.sbj] : T(0);
    }
    __syncthreads();
    if constexpr (sizeof(T) == 4) {
#pragma unroll
      for (int kk = 0; kk < GK; kk += 2) {
        const float a = As[kk + (lane >> 5)][wi + (lane & 31)];
        const float b = Bs[kk + (lane >> 5)][wj + (lane & 31)];
        acc32 = mfma32_f32(a, b, acc32);
      }
    } else {
#pragma unroll 4
      for (int kk = 0; kk < GK; ++kk) {
        double a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          a[u] = As[kk][ty * 4 + u];
          b[u] = Bs[kk][tx * 4 + u];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
#pragma unroll
          for (int v = 0; v < 4; ++v) acc64[u][v] = fma(a[u], b[v], acc64[u][v]);
      }
    }
    __syncthreads();
  }

  if constexpr (sizeof(T) == 4) {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int i = i0 + wi + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      const int j = j0 + wj + (lane & 31);
      if (i < g.M && j < g.N) {
        T* c = g.C + (int64_t)i * g.ldc + j;
        const T v = g.alpha * (T)acc32[e];
        *c = g.beta != T(0) ? g.beta * *c + v : v;
      }
    }
  } else {
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const int i = i0 + ty * 4 + u, j = j0 + tx * 4 + v;
        if (i < g.M && j < g.N) {
          T* c = g.C + (int64_t)i * g.ldc + j;
          const T r = g.alpha * (T)acc64[u][v];
          *c = g.beta != T(0) ? g.beta * *c + r : r;
        }
      }
  }
}

// Factor the bs x bs diagonal block at (kb, kb) of A (lower) and replace it by the
// inverse of its Cholesky factor (upper part of the block zeroed).
template <class T>
__global__ __launch_bounds__(512) void potrf_inv_kernel(T* A, int64_t lda, int kb, int bs,
                                                        int32_t* info) {
  constexpr int P = NB + 1;
  __shared__ T L[NB * P];
  __shared__ T colbuf[NB];
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int e = tid; e < bs * bs; e += nt) {
    const int i = e / bs, j = e % bs;
    L[i * P + j] = j <= i ? A[(int64_t)(kb + i) * lda + kb + j] : T(0);
  }
  __syncthreads();
  // right-looking unblocked Cholesky
  for (int j = 0; j < bs; ++j) {
    const T ajj = L[j * P + j];
    const bool bad = !(ajj > T(0));
    const T d = sqrt(ajj);
    __syncthreads();
    if (tid == 0) {
      L[j * P + j] = d;
      if (bad && *info == 0) *info = kb + j + 1;
    }
    for (int i = j + 1 + tid; i < bs; i += nt) L[i * P + j] /= d;
    __syncthreads();
    const int n = bs - j - 1;  // trailing block; only its lower triangle is updated
    for (int e = tid; e < n * n; e += nt) {
      const int r = e / n, c = e % n;
      if (c <= r) {
        const int gi = j + 1 + r, gc = j + 1 + c;
        L[gi * P + gc] -= L[gi * P + j] * L[gc * P + j];
      }
    }
    __syncthreads();
  }
  // in-place inverse of the lower-triangular factor, last column first:
  // column j below the diagonal becomes -(Linv_trailing * L[j+1:, j]) / L[j][j].
  for (int j = bs - 1; j >= 0; --j) {
    const T inv = T(1) / L[j * P + j];
    for (int i = j + 1 + tid; i < bs; i += nt) {
      T s = T(0);
      for (int t = j + 1; t <= i; ++t) s += L[i * P + t] * L[t * P + j];
      colbuf[i] = -s * inv;
    }
    __syncthreads();
    for (int i = j + 1 + tid; i < bs; i += nt) L[i * P + j] = colbuf[i];
    if (tid == 0) L[j * P + j] = inv;
    __syncthreads();
  }
  for (int e = tid; e < bs * bs; e += nt) {
    const int i = e / bs, j = e % bs;
    A[(int64_t)(kb + i) * lda + kb + j] = j <= i ? L[i * P + j] : T(0);
  }
}

// A = G + lambda I (full copy), R = C, info = 0.
template <class T>
__global__ __launch_bounds__(256) void init_kernel(const T* __restrict__ G, const T* __restrict__ C,
                                                   T* __restrict__ A, T* __restrict__ R, int64_t d,
                                                   int64_t dout, double lambda,
                                                   const double* lam_dev, int32_t* info) {
  const int64_t nA = d * d, nR = d * dout;
  const double lam = lam_dev ? *lam_dev : lambda;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < nA + nR;
       e += (int64_t)gridDim.x * blockDim.x) {
    if (e < nA) {
      const int64_t i = e / d, j = e % d;
      A[e] = G[e] + (i == j ? (T)lam : T(0));
    } else {
      R[e - nA] = C[e - nA];
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *info = 0;
}

// Stage 1 of the adaptive ridge: per-block partial sums of G_ij^2 and G_ii.
template <class T>
__global__ __launch_bounds__(256) void ridge_partial_kernel(const T* __restrict__ G, int64_t d,
                                                            double* part) {
  __shared__ double s2[256], st[256];
  double a = 0.0, b = 0.0;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < d * d; e += (int64_t)kRedBlocks * 256) {
    const double v = (double)G[e];
    a += v * v;
    if (e / d == e % d) b += v;
  }
  s2[threadIdx.x] = a;
  st[threadIdx.x] = b;
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) {
      s2[threadIdx.x] += s2[threadIdx.x + s];
      st[threadIdx.x] += st[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = s2[0];
    part[2 * blockIdx.x + 1] = st[0];
  }
}

// Stage 2: lambda = lambda_0 * sum(G^2) / tr(G)  (Eq. 7).
__global__ __launch_bounds__(256) void ridge_final_kernel(const double* part, double lam0,
                                                          double* lam_out) {
  __shared__ double s2[256], st[256];
  s2[threadIdx.x] = part[2 * threadIdx.x];
  st[threadIdx.x] = part[2 * threadIdx.x + 1];
  __syncthreads();
  for (int s = 128; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) {
      s2[threadIdx.x] += s2[threadIdx.x + s];
      st[threadIdx.x] += st[threadIdx.x + s];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) lam_out[0] = lam0 * s2[0] / st[0];
}

template <class T>
__global__ __launch_bounds__(256) void to_float_kernel(const T* __restrict__ X, float* __restrict__ Y,
                                                       int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    Y[e] = (float)X[e];
}

template <class T>
GemmDesc<T> desc(const T* A, int64_t sai, int64_t sak, const T* B, int64_t sbk, int64_t sbj, T* C,
                 int64_t ldc, int M, int N, int K, T alpha, T beta, int lower = 0) {
  GemmDesc<T> g{};
  g.A = A; g.sai = sai; g.sak = sak;
  g.B = B; g.sbk = sbk; g.sbj = sbj;
  g.C = C; g.ldc = ldc;
  g.M = M; g.N = N; g.K = K;
  g.alpha = alpha; g.beta = beta;
  g.lower = lower;
  g.tiles_n = (N + GT - 1) / GT;
  g.ntiles = (M > 0 && N > 0 && K > 0) ? ((M + GT - 1) / GT) * g.tiles_n : 0;
  return g;
}

template <class T>
hipError_t run_group(const GemmDesc<T>* ds, int n, hipStream_t st) {
  GemmGroup<T> grp{};
  int total = 0;
  int m = 0;
  for (int i = 0; i < n; ++i)
    if (ds[i].ntiles > 0) {
      grp.d[m++] = ds[i];
      total += ds[i].ntiles;
    }
  if (m == 0) return hipSuccess;
  grp.n = m;
  hipLaunchKernelGGL((solve_gemm_kernel<T>), dim3(total), dim3(256), 0, st, grp);
  return hipGetLastError();
}

struct SolveLayout {
  size_t A, Lm, R, Z, X, part, lam, total;
};

template <class T>
SolveLayout layout(int64_t d, int64_t dout) {
  SolveLayout L{};
  size_t o = 0;
  L.A = o; o += align_up(sizeof(T) * d * d);
  L.Lm = o; o += align_up(sizeof(T) * d * d);
  L.R = o; o += align_up(sizeof(T) * d * dout);
  L.Z = o; o += align_up(sizeof(T) * d * dout);
  L.X = o; o += align_up(sizeof(T) * d * dout);
  L.part = o; o += align_up(sizeof(double) * 2 * kRedBlocks);
  L.lam = o; o += align_up(sizeof(double));
  L.total = o;
  return L;
}

#define PKV_TRY(x)                           \
  do {                                       \
    hipError_t e_ = (x);                     \
    if (e_ != hipSuccess) return e_;         \
  } while (0)

template <class T>
hipError_t solve_t(const T* G, const T* C, int64_t d64, int64_t dout64, double lambda,
                   bool adaptive, float* dW, int32_t* info, void* ws, hipStream_t st) {
  const SolveLayout L = layout<T>(d64, dout64);
  char* w = (char*)ws;
  T* A = (T*)(w + L.A);
  T* Lm = (T*)(w + L.Lm);
  T* R = (T*)(w + L.R);
  T* Z = (T*)(w + L.Z);
  T* X = (T*)(w + L.X);
  double* part = (double*)(w + L.part);
  double* lam = (double*)(w + L.lam);
  const int d = (int)d64, dout = (int)dout64;

  if (adaptive) {
    hipLaunchKernelGGL((ridge_partial_kernel<T>), dim3(kRedBlocks), dim3(256), 0, st, G, d64, part);
    PKV_TRY(hipGetLastError());
    hipLaunchKernelGGL(ridge_final_kernel, dim3(1), dim3(256), 0, st, part, lambda, lam);
    PKV_TRY(hipGetLastError());
  }
  {
    const int64_t n = d64 * d64 + d64 * dout64;
    const int blocks = (int)std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL((init_kernel<T>), dim3(blocks), dim3(256), 0, st, G, C, A, R, d64, dout64,
                       lambda, adaptive ? lam : (const double*)nullptr, info);
    PKV_TRY(hipGetLastError());
  }
  const T one = T(1), zero = T(0), mone = T(-1);
  const int nblk = (d + NB - 1) / NB;
  for (int k = 0; k < nblk; ++k) {
    const int kb = k * NB, bs = std::min(NB, d - kb);
    const int rest = d - kb - bs;
    hipLaunchKernelGGL((potrf_inv_kernel<T>), dim3(1), dim3(512), 0, st, A, d64, kb, bs, info);
    PKV_TRY(hipGetLastError());
    const T* Linv = A + (int64_t)kb * d + kb;  // Linv(i,t) = Linv[i*d + t]
    {
      GemmDesc<T> g[2];
      // L_ik = A_ik Linv^T : (rest x bs) = (rest x bs) * (bs x bs)^T
      g[0] = desc<T>(A + (int64_t)(kb + bs) * d + kb, d, 1, Linv, 1, d,
                     Lm + (int64_t)(kb + bs) * d + kb, d, rest, bs, bs, one, zero);
      // Z_k = Linv R_k : (bs x dout)
      g[1] = desc<T>(Linv, d, 1, R + (int64_t)kb * dout, dout, 1, Z + (int64_t)kb * dout, dout, bs,
                     dout, bs, one, zero);
      PKV_TRY(run_group(g, 2, st));
    }
    if (rest > 0) {
      GemmDesc<T> g[2];
      const T* Lp = Lm + (int64_t)(kb + bs) * d + kb;  // panel rows kb+bs.., cols kb..kb+bs
      // A_ij -= L_ik L_jk^T over the trailing lower blocks
      g[0] = desc<T>(Lp, d, 1, Lp, 1, d, A + (int64_t)(kb + bs) * d + kb + bs, d, rest, rest, bs, mone,
                     one, 1);
      // R_i -= L_ik Z_k
      g[1] = desc<T>(Lp, d, 1, Z + (int64_t)kb * dout, dout, 1, R + (int64_t)(kb + bs) * dout, dout,
                     rest, dout, bs, mone, one);
      PKV_TRY(run_group(g, 2, st));
    }
  }
  for (int k = nblk - 1; k >= 0; --k) {
    const int kb = k * NB, bs = std::min(NB, d - kb);
    const T* Linv = A + (int64_t)kb * d + kb;
    {
      // X_k = Linv^T Z_k : X(i,n) = sum_t Linv[t][i] Z[kb+t][n]
      GemmDesc<T> g = desc<T>(Linv, 1, d, Z + (int64_t)kb * dout, dout, 1, X + (int64_t)kb * dout,
                              dout, bs, dout, bs, one, zero);
      PKV_TRY(run_group(&g, 1, st));
    }
    if (kb > 0) {
      // Z_i -= L_ki^T X_k for i < kb : Z(i,n) -= sum_t Lm[kb+t][i] X[kb+t][n]
      GemmDesc<T> g = desc<T>(Lm + (int64_t)kb * d, 1, d, X + (int64_t)kb * dout, dout, 1, Z, dout, kb,
                              dout, bs, mone, one);
      PKV_TRY(run_group(&g, 1, st));
    }
  }
  {
    const int64_t n = d64 * dout64;
    const int blocks = (int)std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL((to_float_kernel<T>), dim3(blocks), dim3(256), 0, st, X, dW, n);
    PKV_TRY(hipGetLastError());
  }
  return hipSuccess;
}

}  // namespace

size_t solve_ws_bytes(bool f64, int64_t din, int64_t dout) {
  return f64 ? layout<double>(din, dout).total : layout<float>(din, dout).total;
}

hipError_t launch_solve(bool f64, const void* G, const void* C, int64_t din, int64_t dout,
                        double lambda, bool adaptive, float* dW, int32_t* info, void* ws,
                        hipStream_t st) {
  if (f64)
    return solve_t<double>((const double*)G, (const double*)C, din, dout, lambda, adaptive, dW, info,
                           ws, st);
  return solve_t<float>((const float*)G, (const float*)C, din, dout, lambda, adaptive, dW, info, ws,
                        st);
}

}  // namespace pkv
