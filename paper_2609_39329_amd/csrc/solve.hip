// Ridge patch, Eq. 8 in row form: dW = (G + lambda I)^{-1} C.
//
// Right-looking blocked Cholesky with block size NB (128 for fp32, 64 for fp64),
// fused with the forward substitution of the right-hand side:
//   for each block column k:
//     diagonal kernel    L_kk^{-1} (1 WG)
//     grouped GEMM       L_ik = A_ik L_kk^{-T} (i > k);  Z_k = L_kk^{-1} R_k
//     grouped GEMM       A_ij -= L_ik L_jk^T (lower blocks);  R_i -= L_ik Z_k (i > k)
// The updates outside a group of eight block columns (an outer block, OB = 8 NB) are
// deferred to the end of the group (K = OB), see solve_t. Backward substitution runs
// per outer block: X_O = L_OO^{-T} Z_O;  Z_i -= L_Oi^T X_O (i before O).
// Triangular solves against a diagonal block use that block's explicit inverse (a
// GEMM instead of a substitution); its condition number is at most the square root
// of that of G + lambda I. The OB-wide inverses are assembled from the NB-wide ones
// by batched GEMMs.
// fp32 block products split both operands into three bf16 pieces and sum six bf16
// MFMA products, as exact as fp32 products (128 x 128 tiles; 64 x 64 with the whole K
// range staged at once for the latency-bound K <= 128 updates); on request they split
// into two pieces and three products (about 2^-16 relative, faster) or run on MFMA
// 32x32x2 f32 (exact fp32 products). fp64 tiles run on fp64 FMA. The adaptive ridge of Eq. 7, lambda_0 ||G||_F^2 / tr G, and
// the trace-mean scaling lambda_0 tr G / d are reduced on the device in fp64 in a fixed
// order (deterministic).
#include <math.h>

#include <algorithm>
#include <utility>

#include "common.hpp"
#include "kernels.hpp"

namespace pkv {

namespace {

template <class T>
struct Blk;
template <>
struct Blk<float> {
  static constexpr int NB = 128;  // block size
};
template <>
struct Blk<double> {
  static constexpr int NB = 64;
};

constexpr int kRedBlocks = 1024;  // workgroups of the adaptive-ridge reduction

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
  int vecA, vecB;  // 16-byte loads along the contiguous dimension are allowed
  // batch of equal-shaped problems: item b uses A + b bA, B + b bB, C + b bC
  int batch, tiles_b;  // items, tiles per item (ntiles = batch * tiles_b)
  int64_t bA, bB, bC;
};

// the problem of tile t of a batched descriptor (t becomes the tile within it)
template <class D>
__device__ __forceinline__ D batch_item(const D& g, int& t) {
  D h = g;
  if (g.batch > 1) {
    const int b = t / g.tiles_b;
    t -= b * g.tiles_b;
    h.A += b * g.bA;
    h.B += b * g.bB;
    h.C += b * g.bC;
  }
  return h;
}

// ---- fp32: BM x BM output tile (128 or 64), 4 waves, MFMA 32x32x2 f32 ---------------
constexpr int F_KC = 32;

template <int BM>
__device__ __forceinline__ void gemm_f32_body(const GemmDesc<float>& g, int t) {
  constexpr int P = BM + 4;
  constexpr int WT = BM / 64;                 // MFMA tiles per wave and dimension
  constexpr int NU = BM * F_KC / 4 / 256;     // float4 per thread per operand and chunk
  __shared__ float As[2][F_KC][P];
  __shared__ float Bs[2][F_KC][P];
  const int ti = t / g.tiles_n, tj = t % g.tiles_n;
  if (g.lower && tj > ti) return;
  const int i0 = ti * BM, j0 = tj * BM;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int wi = (wid >> 1) * (BM / 2), wj = (wid & 1) * (BM / 2);

  f32x16 acc[WT][WT];
#pragma unroll
  for (int a = 0; a < WT; ++a)
#pragma unroll
    for (int b = 0; b < WT; ++b) acc[a][b] = f32x16{};

  f32x4 ra[NU], rb[NU];
  const bool a_k = g.sak == 1;  // A contiguous along k (else along i)
  const bool b_j = g.sbj == 1;  // B contiguous along j (else along k)
  auto fetch = [&](int k0) {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int c = u * 256 + tid;
      int i, k;
      if (a_k) { i = c / (F_KC / 4); k = (c % (F_KC / 4)) * 4; }
      else { k = c / (BM / 4); i = (c % (BM / 4)) * 4; }
      const int gi = i0 + i, gk = k0 + k;
      f32x4 v = {};
      if (a_k) {
        if (gi < g.M) {
          const float* s = g.A + (int64_t)gi * g.sai + gk;
          if (g.vecA && gk + 3 < g.K) v = *(const f32x4*)s;
          else
            for (int e = 0; e < 4; ++e) v[e] = gk + e < g.K ? s[e] : 0.f;
        }
      } else {
        if (gk < g.K) {
          const float* s = g.A + (int64_t)gk * g.sak + gi;
          if (g.vecA && gi + 3 < g.M) v = *(const f32x4*)s;
          else
            for (int e = 0; e < 4; ++e) v[e] = gi + e < g.M ? s[(int64_t)e * g.sai] : 0.f;
        }
      }
      ra[u] = v;
      int j, kb;
      if (b_j) { kb = c / (BM / 4); j = (c % (BM / 4)) * 4; }
      else { j = c / (F_KC / 4); kb = (c % (F_KC / 4)) * 4; }
      const int gj = j0 + j, gkb = k0 + kb;
      f32x4 w = {};
      if (b_j) {
        if (gkb < g.K) {
          const float* s = g.B + (int64_t)gkb * g.sbk + gj;
          if (g.vecB && gj + 3 < g.N) w = *(const f32x4*)s;
          else
            for (int e = 0; e < 4; ++e) w[e] = gj + e < g.N ? s[(int64_t)e * g.sbj] : 0.f;
        }
      } else {
        if (gj < g.N) {
          const float* s = g.B + (int64_t)gj * g.sbj + gkb;
          if (g.vecB && gkb + 3 < g.K) w = *(const f32x4*)s;
          else
            for (int e = 0; e < 4; ++e) w[e] = gkb + e < g.K ? s[(int64_t)e * g.sbk] : 0.f;
        }
      }
      rb[u] = w;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int c = u * 256 + tid;
      if (a_k) {
        const int i = c / (F_KC / 4), k = (c % (F_KC / 4)) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) As[buf][k + e][i] = ra[u][e];
      } else {
        *(f32x4*)&As[buf][c / (BM / 4)][(c % (BM / 4)) * 4] = ra[u];
      }
      if (b_j) {
        *(f32x4*)&Bs[buf][c / (BM / 4)][(c % (BM / 4)) * 4] = rb[u];
      } else {
        const int j = c / (F_KC / 4), k = (c % (F_KC / 4)) * 4;
#pragma unroll
        for (int e = 0; e < 4; ++e) Bs[buf][k + e][j] = rb[u][e];
      }
    }
  };

  const int nk = (g.K + F_KC - 1) / F_KC;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int buf = kc & 1;
    if (kc + 1 < nk) fetch((kc + 1) * F_KC);
#pragma unroll
    for (int ks = 0; ks < F_KC; ks += 2) {
      float av[WT], bv[WT];
#pragma unroll
      for (int a = 0; a < WT; ++a) av[a] = As[buf][ks + (lane >> 5)][wi + 32 * a + (lane & 31)];
#pragma unroll
      for (int b = 0; b < WT; ++b) bv[b] = Bs[buf][ks + (lane >> 5)][wj + 32 * b + (lane & 31)];
#pragma unroll
      for (int a = 0; a < WT; ++a)
#pragma unroll
        for (int b = 0; b < WT; ++b) acc[a][b] = mfma32_f32(av[a], bv[b], acc[a][b]);
    }
    if (kc + 1 < nk) stash(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int a = 0; a < WT; ++a)
#pragma unroll
    for (int b = 0; b < WT; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int i = i0 + wi + 32 * a + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int j = j0 + wj + 32 * b + (lane & 31);
        if (i < g.M && j < g.N) {
          float* c = g.C + (int64_t)i * g.ldc + j;
          const float v = g.alpha * acc[a][b][e];
          *c = g.beta != 0.f ? g.beta * *c + v : v;
        }
      }
}

// ---- fp32 via bf16 MFMA terms: 128 x 128 output tile, 4 waves -------------------------
//
// Each fp32 operand x is split into bf16 pieces while it is staged into LDS and the
// product is formed from bf16 MFMA 32x32x16 products with fp32 accumulation:
//  TERMS = 6 (FP32-grade): x = h + m + l, h = bf16(x), m = bf16(x - h),
//    l = bf16(x - h - m), which represents x to about 2^-27; a b ~ hh + hm + mh + mm +
//    hl + lh, the dropped ml, lm, ll about 2^-27 relative: the products are as exact as
//    fp32 multiplication (2^-24) and the sums are fp32.
//  TERMS = 3: x = h + l, a b ~ hh + hl + lh, about 2^-16 relative per product.
// The MFMA computes the transposed tile (rows = output columns), so every lane owns 4
// consecutive output columns of one output row and the read-modify-write of C uses
// 16-byte accesses. The C tile is fetched before the K loop so its latency hides
// behind the products.
struct SGemm {
  const float* A;  // A(i,k) = AK ? A[i*sa + k] : A[k*sa + i]
  int64_t sa;
  const float* B;  // B(k,j) = BJ ? B[k*sb + j] : B[j*sb + k]
  int64_t sb;
  float* C;        // C[i*ldc + j] = beta C + alpha sum_k A(i,k) B(k,j)
  int64_t ldc;
  int M, N, K;
  float alpha, beta;
  int lower;       // only tiles with tile_row >= tile_col (enumerated triangularly)
  int tiles_n, ntiles;
  int vecA, vecB, vecC;
  int batch, tiles_b;  // as in GemmDesc
  int64_t bA, bB, bC;
};

// bf16 pieces of each operand, and the K chunk staged per round (the six-term products
// stage half the chunk, so two workgroups still fit in a CU's LDS)
template <int TERMS>
struct Split {
  static_assert(TERMS == 3 || TERMS == 6, "three or six product terms");
  static constexpr int P = TERMS == 6 ? 3 : 2;     // pieces per operand
  static constexpr int KC = TERMS == 6 ? 16 : 32;  // K chunk
};

// x -> bf16 pieces (two elements per conversion), stored at off of each piece's plane
template <int NP>
__device__ __forceinline__ void split_store(__bf16* const (&pl)[NP], int off, f32x4 v) {
  f32x4 r = v;
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    const unsigned h01 = pack_bf16(r[0], r[1]), h23 = pack_bf16(r[2], r[3]);
    *(u32x2*)(pl[q] + off) = u32x2{h01, h23};
    if (q + 1 < NP) {
      r[0] -= __builtin_bit_cast(float, h01 << 16);
      r[1] -= __builtin_bit_cast(float, h01 & 0xffff0000u);
      r[2] -= __builtin_bit_cast(float, h23 << 16);
      r[3] -= __builtin_bit_cast(float, h23 & 0xffff0000u);
    }
  }
}

// acc += b a over the kept piece pairs: fb[q] / fa[q] are the pieces of the B / A
// fragments (transposed tile: MFMA rows are output columns)
template <int TERMS>
__device__ __forceinline__ f32x16 split_mfma(const bf16x8 (&fb)[Split<TERMS>::P],
                                             const bf16x8 (&fa)[Split<TERMS>::P], f32x16 acc) {
  if constexpr (TERMS == 6) {
    // the smallest terms first
    acc = mfma32(fb[2], fa[0], acc);
    acc = mfma32(fb[0], fa[2], acc);
    acc = mfma32(fb[1], fa[1], acc);
    acc = mfma32(fb[1], fa[0], acc);
    acc = mfma32(fb[0], fa[1], acc);
    acc = mfma32(fb[0], fa[0], acc);
  } else {
    acc = mfma32(fb[0], fa[0], acc);
    acc = mfma32(fb[0], fa[1], acc);
    acc = mfma32(fb[1], fa[0], acc);
  }
  return acc;
}

constexpr int S_BM = 128;
template <int TERMS>
struct SLayout {
  static constexpr int KC = Split<TERMS>::KC;
  static constexpr int PK = KC + 8;    // pitch of a [row][k] LDS tile (bf16)
  static constexpr int PR = S_BM + 16;   // pitch of a [k][row] LDS tile (bf16)
  static constexpr int TILE = S_BM * PK > KC * PR ? S_BM * PK : KC * PR;  // bf16 per plane
  static constexpr int LDS = 2 * 2 * Split<TERMS>::P * TILE;  // 2 buffers x {A, B} x pieces
};

// CHECK: bounds-checked staging loads (edge tiles); without it the tile must lie
// inside M x N, K must be a multiple of the chunk and both operands vector-aligned,
// and the loads are plain 16-byte loads from pointers advanced once per chunk.
template <int TERMS, bool AK, bool BJ, bool CHECK>
__device__ __forceinline__ void sgemm3_tile(const SGemm& g, int i0, int j0, __bf16* lds);

// tile t of g (lower: the triangle's tiles in row order)
template <int TERMS, bool AK, bool BJ>
__device__ __forceinline__ void sgemm3_body(const SGemm& g, int t, __bf16* lds) {
  int ti, tj;
  if (g.lower) {
    ti = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
    while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
    while (ti * (ti + 1) / 2 > t) --ti;
    tj = t - ti * (ti + 1) / 2;
  } else {
    ti = t / g.tiles_n;
    tj = t % g.tiles_n;
  }
  const int i0 = ti * S_BM, j0 = tj * S_BM;
  const bool interior = i0 + S_BM <= g.M && j0 + S_BM <= g.N && g.K % SLayout<TERMS>::KC == 0 &&
                        g.vecA && g.vecB;
  if (interior) sgemm3_tile<TERMS, AK, BJ, false>(g, i0, j0, lds);
  else sgemm3_tile<TERMS, AK, BJ, true>(g, i0, j0, lds);
}

template <int TERMS, bool AK, bool BJ, bool CHECK>
__device__ __forceinline__ void sgemm3_tile(const SGemm& g, int i0, int j0, __bf16* lds) {
  using LY = SLayout<TERMS>;
  constexpr int KC = LY::KC, NP = Split<TERMS>::P;
  constexpr int NU = S_BM * KC / 4 / 256;  // float4 runs per thread, operand and chunk
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int h32 = lane >> 5, l32 = lane & 31;
  const int wi = (wid >> 1) * 64, wj = (wid & 1) * 64;
  // [row][k] when the contraction index is contiguous in memory, else [k][row]
  constexpr bool a_rk = AK, b_rk = !BJ;
  constexpr int PA = a_rk ? LY::PK : LY::PR, PB = b_rk ? LY::PK : LY::PR;

  // C tile prefetch: lane owns C[i0+wi+32a+l32][j0+wj+32b+8q+4h32 .. +3]
  f32x4 cpre[2][2][4];
  const bool use_c = g.beta != 0.f;
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        f32x4 v = {};
        const int i = i0 + wi + 32 * a + l32, j = j0 + wj + 32 * b + 8 * q + 4 * h32;
        if (use_c && i < g.M && j < g.N) {
          const float* s = g.C + (int64_t)i * g.ldc + j;
          if (g.vecC && j + 3 < g.N) v = *(const f32x4*)s;
          else
            for (int e = 0; e < 4; ++e) v[e] = j + e < g.N ? s[e] : 0.f;
        }
        cpre[a][b][q] = v;
      }

  f32x16 acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b) acc[a][b] = f32x16{};

  // staging: 128 x KC floats per operand and chunk = NU float4 per thread, each a run
  // of 4 elements contiguous in memory
  f32x4 ra[NU], rb[NU];
  // unchecked staging: this thread's runs of the first chunk, advanced by one chunk
  // per fetch (fetches are issued in chunk order)
  const float* pa[NU];
  const float* pb[NU];
  const int64_t stepA = AK ? KC : (int64_t)KC * g.sa, stepB = BJ ? (int64_t)KC * g.sb : KC;
  if constexpr (!CHECK) {
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int c = u * 256 + tid;
      if constexpr (AK) pa[u] = g.A + (int64_t)(i0 + c / (KC / 4)) * g.sa + (c % (KC / 4)) * 4;
      else pa[u] = g.A + (int64_t)(c / (S_BM / 4)) * g.sa + i0 + (c % (S_BM / 4)) * 4;
      if constexpr (BJ) pb[u] = g.B + (int64_t)(c / (S_BM / 4)) * g.sb + j0 + (c % (S_BM / 4)) * 4;
      else pb[u] = g.B + (int64_t)(j0 + c / (KC / 4)) * g.sb + (c % (KC / 4)) * 4;
    }
  }
  auto fetch = [&](int k0) {
    if constexpr (!CHECK) {
#pragma unroll
      for (int u = 0; u < NU; ++u) {
        ra[u] = *(const f32x4*)pa[u];
        rb[u] = *(const f32x4*)pb[u];
        pa[u] += stepA;
        pb[u] += stepB;
      }
      return;
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int c = u * 256 + tid;
      {
        int i, k;
        if constexpr (AK) { i = c / (KC / 4); k = (c % (KC / 4)) * 4; }
        else { k = c / (S_BM / 4); i = (c % (S_BM / 4)) * 4; }
        const int gi = i0 + i, gk = k0 + k;
        const int nvalid = AK ? (gi < g.M ? g.K - gk : 0) : (gk < g.K ? g.M - gi : 0);
        const float* s = g.A + (AK ? (int64_t)gi * g.sa + gk : (int64_t)gk * g.sa + gi);
        f32x4 v = {};
        if (nvalid >= 4 && g.vecA) v = *(const f32x4*)s;
        else
          for (int e = 0; e < 4; ++e)
            if (e < nvalid) v[e] = s[e];
        ra[u] = v;
      }
      {
        int j, k;
        if constexpr (BJ) { k = c / (S_BM / 4); j = (c % (S_BM / 4)) * 4; }
        else { j = c / (KC / 4); k = (c % (KC / 4)) * 4; }
        const int gj = j0 + j, gk = k0 + k;
        const int nvalid = BJ ? (gk < g.K ? g.N - gj : 0) : (gj < g.N ? g.K - gk : 0);
        const float* s = g.B + (BJ ? (int64_t)gk * g.sb + gj : (int64_t)gj * g.sb + gk);
        f32x4 v = {};
        if (nvalid >= 4 && g.vecB) v = *(const f32x4*)s;
        else
          for (int e = 0; e < 4; ++e)
            if (e < nvalid) v[e] = s[e];
        rb[u] = v;
      }
    }
  };
  // plane of operand X (0: A, 1: B), piece q, in buffer buf
  auto plane = [&](int buf, int x, int q) { return lds + ((buf * 2 + x) * NP + q) * LY::TILE; };
  auto stash = [&](int buf) {
    __bf16* pa_[NP];
    __bf16* pb_[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      pa_[q] = plane(buf, 0, q);
      pb_[q] = plane(buf, 1, q);
    }
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int c = u * 256 + tid;
      split_store<NP>(pa_, a_rk ? (c / (KC / 4)) * PA + (c % (KC / 4)) * 4
                                : (c / (S_BM / 4)) * PA + (c % (S_BM / 4)) * 4, ra[u]);
      split_store<NP>(pb_, b_rk ? (c / (KC / 4)) * PB + (c % (KC / 4)) * 4
                                : (c / (S_BM / 4)) * PB + (c % (S_BM / 4)) * 4, rb[u]);
    }
  };
  // 32 rows x 8 k fragment (row r0 + l32, k k0 + 8 h32 ..) of an LDS tile
  const int tr_k = 8 * h32 + ((lane & 15) >> 2);
  const int tr_r = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
  auto frag = [&](const __bf16* base, int pitch, bool rk, int r0, int k0) -> bf16x8 {
    if (rk) return *(const bf16x8*)(base + (r0 + l32) * pitch + k0 + h32 * 8);
    const PKV_LDS __bf16* q = (const PKV_LDS __bf16*)(base + (k0 + tr_k) * pitch + r0 + tr_r);
    return cat8(lds_read_tr16(q), lds_read_tr16(q + 4 * pitch));
  };

  const int nk = (g.K + KC - 1) / KC;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int kc = 0; kc < nk; ++kc) {
    const int buf = kc & 1;
    if (kc + 1 < nk) fetch((kc + 1) * KC);
#pragma unroll
    for (int ks = 0; ks < KC; ks += 16) {
      bf16x8 fa[2][NP], fb[2][NP];
#pragma unroll
      for (int q = 0; q < NP; ++q) {
#pragma unroll
        for (int a = 0; a < 2; ++a) fa[a][q] = frag(plane(buf, 0, q), PA, a_rk, wi + 32 * a, ks);
#pragma unroll
        for (int b = 0; b < 2; ++b) fb[b][q] = frag(plane(buf, 1, q), PB, b_rk, wj + 32 * b, ks);
      }
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = split_mfma<TERMS>(fb[b], fa[a], acc[a][b]);
    }
    if (kc + 1 < nk) stash(buf ^ 1);
    __syncthreads();
  }

#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int i = i0 + wi + 32 * a + l32, j = j0 + wj + 32 * b + 8 * q + 4 * h32;
        if (i >= g.M || j >= g.N) continue;
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = g.alpha * acc[a][b][4 * q + e];
        if (use_c) v += g.beta * cpre[a][b][q];
        float* d = g.C + (int64_t)i * g.ldc + j;
        if (g.vecC && j + 3 < g.N) *(f32x4*)d = v;
        else
          for (int e = 0; e < 4; ++e)
            if (j + e < g.N) d[e] = v[e];
      }
}

// Up to two problems per launch, each with its own operand layout; work items are
// spread so that consecutive tiles of one problem share an XCD (and its L2).
template <int TERMS, bool AK0, bool BJ0, bool AK1, bool BJ1>
__global__ __launch_bounds__(256, 2) void sgemm3_kernel(SGemm d0, SGemm d1) {
  __shared__ __attribute__((aligned(16))) __bf16 lds[SLayout<TERMS>::LDS];
  const int total = d0.ntiles + d1.ntiles;
  const int t = xcd_item((total + kXcds - 1) / kXcds);
  if (t >= total) return;
  if (t < d0.ntiles) {
    int u = t;
    const SGemm g = batch_item(d0, u);
    sgemm3_body<TERMS, AK0, BJ0>(g, u, lds);
  } else {
    int u = t - d0.ntiles;
    const SGemm g = batch_item(d1, u);
    sgemm3_body<TERMS, AK1, BJ1>(g, u, lds);
  }
}

// ---- the same split products for K <= 128: 64 x 64 tiles, one staging round ----------
//
// The small updates of the factorisation (K = one block column) are latency bound:
// with 128 x 128 tiles a launch has few workgroups and every chunk waits for its loads.
// Here each workgroup (4 waves of 32 x 32) loads its whole K range in one round (K
// padded to 16 with zeros, bounds-checked), splits it into bf16 planes in LDS and runs
// the MFMAs with no further waits.
constexpr int T_BM = 64, T_KMAX = 128;
constexpr int T_PK = T_KMAX + 8;  // pitch of a [row][k] LDS tile (bf16)
constexpr int T_PR = T_BM + 16;   // pitch of a [k][row] LDS tile (bf16)
constexpr int T_TILE = T_BM * T_PK > T_KMAX * T_PR ? T_BM * T_PK : T_KMAX * T_PR;  // bf16 per plane

template <int TERMS, bool AK, bool BJ>
__device__ __forceinline__ void sgemm3s_body(const SGemm& g, int t, __bf16* lds) {
  constexpr int NP = Split<TERMS>::P;
  int ti, tj;
  if (g.lower) {
    ti = (int)((sqrtf(8.f * (float)t + 1.f) - 1.f) * 0.5f);
    while ((ti + 1) * (ti + 2) / 2 <= t) ++ti;
    while (ti * (ti + 1) / 2 > t) --ti;
    tj = t - ti * (ti + 1) / 2;
  } else {
    ti = t / g.tiles_n;
    tj = t % g.tiles_n;
  }
  const int i0 = ti * T_BM, j0 = tj * T_BM;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int h32 = lane >> 5, l32 = lane & 31;
  const int wi = (wid >> 1) * 32, wj = (wid & 1) * 32;
  constexpr bool a_rk = AK, b_rk = !BJ;
  constexpr int PA = a_rk ? T_PK : T_PR, PB = b_rk ? T_PK : T_PR;
  const int Kp = (g.K + 15) & ~15;

  // C prefetch: lane owns C[i0+wi+l32][j0+wj+8q+4h32 .. +3]
  f32x4 cpre[4];
  const bool use_c = g.beta != 0.f;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    f32x4 v = {};
    const int i = i0 + wi + l32, j = j0 + wj + 8 * q + 4 * h32;
    if (use_c && i < g.M && j < g.N) {
      const float* c = g.C + (int64_t)i * g.ldc + j;
      if (g.vecC && j + 3 < g.N) v = *(const f32x4*)c;
      else
        for (int e = 0; e < 4; ++e)
          if (j + e < g.N) v[e] = c[e];
    }
    cpre[q] = v;
  }

  // the whole K range: 64 x Kp per operand = up to 8 runs of 4 floats per thread
  constexpr int NU = T_BM * T_KMAX / 4 / 256;
  f32x4 ra[NU], rb[NU];
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int c = u * 256 + tid;
    {
      int i, k;
      if constexpr (AK) { i = c / (T_KMAX / 4); k = (c % (T_KMAX / 4)) * 4; }
      else { k = c / (T_BM / 4); i = (c % (T_BM / 4)) * 4; }
      const int gi = i0 + i;
      const int nvalid = AK ? (gi < g.M ? g.K - k : 0) : (k < g.K ? g.M - gi : 0);
      const float* src = g.A + (AK ? (int64_t)gi * g.sa + k : (int64_t)k * g.sa + gi);
      f32x4 v = {};
      if (k < Kp) {
        if (nvalid >= 4 && g.vecA) v = *(const f32x4*)src;
        else
          for (int e = 0; e < 4; ++e)
            if (e < nvalid) v[e] = src[e];
      }
      ra[u] = v;
    }
    {
      int j, k;
      if constexpr (BJ) { k = c / (T_BM / 4); j = (c % (T_BM / 4)) * 4; }
      else { j = c / (T_KMAX / 4); k = (c % (T_KMAX / 4)) * 4; }
      const int gj = j0 + j;
      const int nvalid = BJ ? (k < g.K ? g.N - gj : 0) : (gj < g.N ? g.K - k : 0);
      const float* src = g.B + (BJ ? (int64_t)k * g.sb + gj : (int64_t)gj * g.sb + k);
      f32x4 v = {};
      if (k < Kp) {
        if (nvalid >= 4 && g.vecB) v = *(const f32x4*)src;
        else
          for (int e = 0; e < 4; ++e)
            if (e < nvalid) v[e] = src[e];
      }
      rb[u] = v;
    }
  }
  __bf16* pa_[NP];
  __bf16* pb_[NP];
#pragma unroll
  for (int q = 0; q < NP; ++q) {
    pa_[q] = lds + q * T_TILE;
    pb_[q] = lds + (NP + q) * T_TILE;
  }
#pragma unroll
  for (int u = 0; u < NU; ++u) {
    const int c = u * 256 + tid;
    const int ka = AK ? (c % (T_KMAX / 4)) * 4 : c / (T_BM / 4);
    const int kb = BJ ? c / (T_BM / 4) : (c % (T_KMAX / 4)) * 4;
    if (ka < Kp)
      split_store<NP>(pa_, a_rk ? (c / (T_KMAX / 4)) * PA + (c % (T_KMAX / 4)) * 4
                                : (c / (T_BM / 4)) * PA + (c % (T_BM / 4)) * 4, ra[u]);
    if (kb < Kp)
      split_store<NP>(pb_, b_rk ? (c / (T_KMAX / 4)) * PB + (c % (T_KMAX / 4)) * 4
                                : (c / (T_BM / 4)) * PB + (c % (T_BM / 4)) * 4, rb[u]);
  }
  __syncthreads();
  // 32 rows x 8 k fragment (row r0 + l32, k k0 + 8 h32 ..) of an LDS tile
  const int tr_k = 8 * h32 + ((lane & 15) >> 2);
  const int tr_r = ((lane >> 4) & 1) * 16 + 4 * (lane & 3);
  auto frag = [&](const __bf16* base, int pitch, bool rk, int r0, int k0) -> bf16x8 {
    if (rk) return *(const bf16x8*)(base + (r0 + l32) * pitch + k0 + h32 * 8);
    const PKV_LDS __bf16* q = (const PKV_LDS __bf16*)(base + (k0 + tr_k) * pitch + r0 + tr_r);
    return cat8(lds_read_tr16(q), lds_read_tr16(q + 4 * pitch));
  };
  f32x16 acc = {};
  for (int ks = 0; ks < Kp; ks += 16) {
    bf16x8 fa[NP], fb[NP];
#pragma unroll
    for (int q = 0; q < NP; ++q) {
      fa[q] = frag(pa_[q], PA, a_rk, wi, ks);
      fb[q] = frag(pb_[q], PB, b_rk, wj, ks);
    }
    acc = split_mfma<TERMS>(fb, fa, acc);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = i0 + wi + l32, j = j0 + wj + 8 * q + 4 * h32;
    if (i >= g.M || j >= g.N) continue;
    f32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = g.alpha * acc[4 * q + e];
    if (use_c) v += g.beta * cpre[q];
    float* d = g.C + (int64_t)i * g.ldc + j;
    if (g.vecC && j + 3 < g.N) *(f32x4*)d = v;
    else
      for (int e = 0; e < 4; ++e)
        if (j + e < g.N) d[e] = v[e];
  }
}

// (six-term planes take 120 KB of LDS: one workgroup per CU; these launches are few
// workgroups anyway)
template <int TERMS, bool AK0, bool BJ0, bool AK1, bool BJ1>
__global__ __launch_bounds__(256, TERMS == 6 ? 1 : 2) void sgemm3s_kernel(SGemm d0, SGemm d1) {
  __shared__ __attribute__((aligned(16))) __bf16 lds[2 * Split<TERMS>::P * T_TILE];
  const int total = d0.ntiles + d1.ntiles;
  const int t = xcd_item((total + kXcds - 1) / kXcds);
  if (t >= total) return;
  if (t < d0.ntiles) {
    int u = t;
    const SGemm g = batch_item(d0, u);
    sgemm3s_body<TERMS, AK0, BJ0>(g, u, lds);
  } else {
    int u = t - d0.ntiles;
    const SGemm g = batch_item(d1, u);
    sgemm3s_body<TERMS, AK1, BJ1>(g, u, lds);
  }
}

// ---- fp64: 64 x 64 output tile, fp64 FMA, 4 x 4 outputs per thread ----------------
constexpr int D_T = 64, D_KC = 32;

__device__ __forceinline__ void gemm_f64_body(const GemmDesc<double>& g, int t) {
  __shared__ double As[D_KC][D_T + 1];
  __shared__ double Bs[D_KC][D_T + 1];
  const int ti = t / g.tiles_n, tj = t % g.tiles_n;
  if (g.lower && tj > ti) return;
  const int i0 = ti * D_T, j0 = tj * D_T;
  const int tid = threadIdx.x, ty = tid / 16, tx = tid % 16;
  double acc[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += D_KC) {
    for (int e = tid; e < D_T * D_KC; e += 256) {
      int i, k;
      if (g.sak == 1) { i = e / D_KC; k = e % D_KC; } else { k = e / D_T; i = e % D_T; }
      const int gi = i0 + i, gk = k0 + k;
      As[k][i] = (gi < g.M && gk < g.K) ? g.A[(int64_t)gi * g.sai + (int64_t)gk * g.sak] : 0.0;
      int j, kb;
      if (g.sbj == 1) { kb = e / D_T; j = e % D_T; } else { j = e / D_KC; kb = e % D_KC; }
      const int gj = j0 + j, gkb = k0 + kb;
      Bs[kb][j] = (gj < g.N && gkb < g.K) ? g.B[(int64_t)gkb * g.sbk + (int64_t)gj * g.sbj] : 0.0;
    }
    __syncthreads();
#pragma unroll 4
    for (int kk = 0; kk < D_KC; ++kk) {
      double a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = As[kk][ty * 4 + u];
        b[u] = Bs[kk][tx * 4 + u];
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
      if (i < g.M && j < g.N) {
        double* c = g.C + (int64_t)i * g.ldc + j;
        const double r = g.alpha * acc[u][v];
        *c = g.beta != 0.0 ? g.beta * *c + r : r;
      }
    }
}

// Up to two independent GEMM problems per launch: blocks [0, d0.ntiles) work on d0,
// the rest on d1. Each problem is its own by-value argument so no descriptor is
// ever indexed dynamically.
template <int BM>
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmDesc<float> d0, GemmDesc<float> d1) {
  const int t = blockIdx.x;
  if (t < d0.ntiles) {
    int u = t;
    const GemmDesc<float> g = batch_item(d0, u);
    gemm_f32_body<BM>(g, u);
  } else if (t - d0.ntiles < d1.ntiles) {
    int u = t - d0.ntiles;
    const GemmDesc<float> g = batch_item(d1, u);
    gemm_f32_body<BM>(g, u);
  }
}

__global__ __launch_bounds__(256) void gemm_f64_kernel(GemmDesc<double> d0, GemmDesc<double> d1) {
  const int t = blockIdx.x;
  if (t < d0.ntiles) {
    int u = t;
    const GemmDesc<double> g = batch_item(d0, u);
    gemm_f64_body(g, u);
  } else if (t - d0.ntiles < d1.ntiles) {
    int u = t - d0.ntiles;
    const GemmDesc<double> g = batch_item(d1, u);
    gemm_f64_body(g, u);
  }
}

// ---- diagonal block, blocked: sub-blocks of 16 ----------------------------------------
//
// The NB x NB block A (128 fp32 or 64 fp64; lower triangle read; zero-padded with an
// identity past bs) and E = L^{-1} live in LDS. For each sub-block column k:
//   leaf (one wave):  A_kk = L_kk L_kk^T and X_kk = L_kk^{-1}, in registers;
//   phase B:          L_ik = A_ik X_kk^T (i > k);  E_km = X_kk E_km (m < k);  E_kk = X_kk
//   phase C:          A_ij -= L_ik L_jk^T (k < j <= i);  E_im -= L_ik E_km (i > k, m <= k)
// i.e. right-looking blocked Cholesky with the forward substitution of the identity
// carried along; phases B and C are independent 16 x 16 x 16 products (fp32: MFMA
// 16x16x4 with exact fp32 products; fp64: fp64 FMA), spread over eight waves, one
// barrier between phases. The leaf of step k + 1 needs only the first product of
// phase C of step k (its own diagonal block), so wave 0 does that product and then
// the leaf while the other seven waves do the rest of phase C: the single-wave leaf,
// the longest serial part (its cost grows with the square of its width), overlaps
// the trailing products.

// LDS pitch (elements): lane-per-row reads of one column hit distinct banks
template <class T>
constexpr int diag_pitch() { return Blk<T>::NB + 2; }

// 1 / x and 1 / sqrt(x) in fp64: the native approximations and one Newton step each
__device__ __forceinline__ double rcp64(double x) {
  const double r = __builtin_amdgcn_rcp(x);
  return fma(r, fma(-x, r, 1.0), r);
}
__device__ __forceinline__ double rsq64(double x) {
  const double r = __builtin_amdgcn_rsq(x);
  return fma(0.5 * r, fma(-x * r, r, 1.0), r);
}

// D = sgn * P Q' (+ C), 16 x 16 blocks in LDS (pitch PT); Q' = Q^T if QT else Q. One
// wave; lane l holds D[4 (l / 16) + e][l % 16]. fp32: MFMA 16x16x4, lane l supplying
// row l % 16 of P and column l % 16 of Q' at k = 4 ks + l / 16; fp64: FMA over k in
// order. D may alias P, Q or C (every operand is read before D is written).
template <bool QT, class T>
__device__ __forceinline__ void mm16(T* D, const T* P, const T* Q, const T* C, T sgn, int lane) {
  constexpr int PT = diag_pitch<T>();
  const int g = lane >> 4, l16 = lane & 15;
  if constexpr (sizeof(T) == 4) {
    f32x4 acc;
#pragma unroll
    for (int e = 0; e < 4; ++e) acc[e] = C ? C[(4 * g + e) * PT + l16] : 0.f;
    float a[4], b[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      const int k = 4 * ks + g;
      a[ks] = sgn * P[l16 * PT + k];
      b[ks] = QT ? Q[l16 * PT + k] : Q[k * PT + l16];
    }
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[ks], b[ks], acc, 0, 0, 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) D[(4 * g + e) * PT + l16] = acc[e];
  } else {
    T acc[4], q[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) q[k] = QT ? Q[l16 * PT + k] : Q[k * PT + l16];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const T* prow = P + (4 * g + e) * PT;
      T a = 0;
#pragma unroll
      for (int k = 0; k < 16; ++k) a = fma(prow[k], q[k], a);
      acc[e] = C ? fma(sgn, a, C[(4 * g + e) * PT + l16]) : sgn * a;
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) D[(4 * g + e) * PT + l16] = acc[e];
  }
}

__device__ __forceinline__ float bcast(float x, int src_lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, x), src_lane));
}
__device__ __forceinline__ double bcast(double x, int src_lane) {
  const u32x2 w = __builtin_bit_cast(u32x2, x);
  const u32x2 r = {(unsigned)__builtin_amdgcn_readlane((int)w[0], src_lane),
                   (unsigned)__builtin_amdgcn_readlane((int)w[1], src_lane)};
  return __builtin_bit_cast(double, r);
}
__device__ __forceinline__ float rsq_of(float x) { return __builtin_amdgcn_rsqf(x); }
__device__ __forceinline__ double rsq_of(double x) { return rsq64(x); }

// Row G's value at each lane's position in its 16-lane row: permlane16_swap gives rows
// (0, 0, 2, 2) and (1, 1, 3, 3), permlane32_swap of that gives its lower (or upper) half
// twice.
template <int G>
__device__ __forceinline__ float from_row(float x) {
  const unsigned u = __builtin_bit_cast(unsigned, x);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const unsigned y = (G & 1) ? a[1] : a[0];
  const auto b = __builtin_amdgcn_permlane32_swap(y, y, false, false);
  return __builtin_bit_cast(float, (G & 2) ? b[1] : b[0]);
}
// lane J of each 16-lane row, to the whole row (DPP row_newbcast)
template <int J>
__device__ __forceinline__ float row_lane(float x) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), 0x150 + J, 0xF, 0xF, false));
}

// The fp32 16-wide leaf on all 64 lanes: lane 16 q + r holds columns 4 k + q (k < 4) of
// row r of the trailing matrix (v) and of Y (x), the block symmetrised from its lower
// triangle on load. Step j, with pivot p = A_jj and u_r = A_rj / p (r > j, else 0):
//   A_rc -= u_r A_jc for c > j (A_jc = A_cj: the trailing matrix stays symmetric), row j
//     of the lane's column group through a DPP broadcast of lane j;
//   Y_rm -= u_r Y_jm for m <= j, the same way;
// A_rj itself comes from column group j % 4 through two lane-row swaps, the pivot through
// one readlane. A lane updates its 4 - j/4 (and j/4 + 1) columns instead of all 16; with
// the broadcasts (separate DPP moves, not fused into the FMAs) and their wait states a
// step takes about 30 instructions against 36 for the row-per-lane sweep below.
__device__ __forceinline__ void leaf16_groups(float* S, float* Xo, int lane, int col0, int bs,
                                              int32_t* info, bool& failed) {
  constexpr int PT = diag_pitch<float>();
  int q = lane >> 4, r = lane & 15;
  asm volatile("" : "+v"(q), "+v"(r));
  float v[4], x[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int c = 4 * k + q;
    v[k] = c > r ? S[c * PT + r] : S[r * PT + c];
    x[k] = c == r ? 1.f : 0.f;
  }
  float rs_own = 0.f;
  static_for<16>([&](auto j_t) {
    constexpr int j = decltype(j_t)::value, jq = j % 4, jk = j / 4;
    const float rs = rsq_of(bcast(v[jk], 16 * jq + j));
    const float a = from_row<jq>(v[jk]);  // on every lane: the swaps are wave-wide
    const float u = r > j ? a * (rs * rs) : 0.f;  // A[r][j] / p
    if (r == j) rs_own = rs;
    static_for<4 - jk>([&](auto kk_t) {  // columns 4 k + q > j
      constexpr int k = jk + decltype(kk_t)::value;
      const float uk = (k > jk || q > jq) ? u : 0.f;
      v[k] = fmaf(-uk, row_lane<j>(v[k]), v[k]);
    });
    static_for<jk + 1>([&](auto k_t) {  // columns 4 k + q <= j
      constexpr int k = decltype(k_t)::value;
      const float uk = (k < jk || q <= jq) ? u : 0.f;
      x[k] = fmaf(-uk, row_lane<j>(x[k]), x[k]);
    });
    if (q == jq) v[jk] *= rs;  // column j of L
  });
  // first failing pivot (padding pivots past bs are 1): row r's diagonal sits in group r % 4
  float dg = v[0];
#pragma unroll
  for (int k = 1; k < 4; ++k)
    if (k == (r >> 2)) dg = v[k];
  const uint64_t bad = __ballot(q == (r & 3) && col0 + r < bs && !(dg > 0.f));
  const unsigned rows = (unsigned)(bad | bad >> 16 | bad >> 32 | bad >> 48) & 0xFFFFu;
  if (rows != 0 && !failed) {
    failed = true;
    if (lane == 0 && *info == 0) *info = col0 + __builtin_ctz(rows) + 1;
  }
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int c = 4 * k + q;
    S[r * PT + c] = v[k];             // row r of L (upper part unused)
    Xo[r * PT + c] = x[k] * rs_own;   // row r of X (zeros above the diagonal)
  }
}

// One wave: factor the SPD N x N block S (lower triangle read) and write
// X = L^{-1} (lower, zeros above) to Xo, in one right-looking sweep.
// Lane r (and its copies r + N, r + 2N, .., which repeat the same work so the wave
// never diverges) holds row r of the trailing matrix (v) and row r of Y, the identity
// under forward substitution (x). Step j, with pivot p = A_jj and u_r = A_rj / p for
// rows r > j (0 otherwise):
//   A_rc -= u_r A_cj     (c > j: column j of every lane, read through readlane)
//   Y_rm -= u_r Y_jm     (m <= j: row j of Y, read from lane j)
// and column j of L is A_rj / sqrt(p). Row r of X is row r of Y over L_rr, applied at
// the end (Y's row r is final after step r - 1). Each step reads N values across
// lanes, in groups of up to 8 held in distinct scalar registers, so that a readlane
// is not directly followed by its consumer. A pivot that is not positive (or NaN)
// makes its L_jj, and every later one, NaN: the first NaN on the diagonal is the
// failing column.
template <int N, class T>
__device__ __forceinline__ void leaf_rows(T* S, T* Xo, int lane, int col0, int bs, int32_t* info,
                                          bool& failed) {
  static_assert(N == 16 || N == 32, "leaf width");
  constexpr int PT = diag_pitch<T>();
  int r = lane & (N - 1);
  // opaque per call: keeps the per-step lane comparisons inside the call instead of
  // hoisting them into scalar registers for the whole kernel
  asm volatile("" : "+v"(r));
  T v[N], x[N];
#pragma unroll
  for (int c = 0; c < N; ++c) {
    v[c] = S[r * PT + c];
    x[c] = c == r ? T(1) : T(0);
  }
  T rs_own = 0;
  // w[c0 .. c0+n) -= u * src(c), the n <= 8 values read first (the empty asm makes
  // them live at once, in distinct registers)
  auto group = [&](T (&w)[N], auto c0_t, auto n_t, auto src, T u) {
    constexpr int c0 = decltype(c0_t)::value, n = decltype(n_t)::value;
    T t[8];
#pragma unroll
    for (int q = 0; q < n; ++q) t[q] = src(c0 + q);
#pragma unroll
    for (int q = n; q < 8; ++q) t[q] = t[0];
    asm volatile("" ::"s"(t[0]), "s"(t[1]), "s"(t[2]), "s"(t[3]), "s"(t[4]), "s"(t[5]), "s"(t[6]),
                 "s"(t[7]));
#pragma unroll
    for (int q = 0; q < n; ++q) w[c0 + q] = fma(-u, t[q], w[c0 + q]);
    __builtin_amdgcn_sched_barrier(0);
  };
  static_for<N>([&](auto j_t) {
    constexpr int j = decltype(j_t)::value;
    const T rs = rsq_of(bcast(v[j], j));
    const T u = r > j ? v[j] * (rs * rs) : T(0);  // A[r][j] / p
    if (r == j) rs_own = rs;
    // A_rc -= u_r A_cj, c = j+1..N-1 (A_cj is lane c's v[j])
    static_for<(N - 1 - j + 7) / 8>([&](auto g_t) {
      constexpr int c0 = j + 1 + 8 * decltype(g_t)::value;
      constexpr int n = N - c0 < 8 ? N - c0 : 8;
      group(v, std::integral_constant<int, c0>{}, std::integral_constant<int, n>{},
            [&](int c) { return bcast(v[j], c); }, u);
    });
    // Y_rm -= u_r Y_jm, m = 0..j (lane j's x[m])
    static_for<(j + 1 + 7) / 8>([&](auto g_t) {
      constexpr int m0 = 8 * decltype(g_t)::value;
      constexpr int n = j + 1 - m0 < 8 ? j + 1 - m0 : 8;
      group(x, std::integral_constant<int, m0>{}, std::integral_constant<int, n>{},
            [&](int m) { return bcast(x[m], j); }, u);
    });
    v[j] *= rs;
  });
  // first failing pivot of this block (padding pivots past bs are 1)
  T diag = 0;
#pragma unroll
  for (int c = 0; c < N; ++c)
    if (c == r) diag = v[c];
  const uint64_t bad = __ballot(lane < N && col0 + r < bs && !(diag > T(0)));
  if (bad != 0 && !failed) {
    failed = true;
    if (lane == 0 && *info == 0) *info = col0 + __builtin_ctzll(bad) + 1;
  }
  if (lane < N) {
#pragma unroll
    for (int c = 0; c < N; ++c) {
      S[r * PT + c] = v[c];            // row r of L (upper part unused)
      Xo[r * PT + c] = x[c] * rs_own;  // row r of X (zeros above the diagonal)
    }
  }
}

// the fp32 16-wide leaf on four column groups, every other on the row-per-lane sweep
template <int N, class T>
__device__ __forceinline__ void leaf(T* S, T* Xo, int lane, int col0, int bs, int32_t* info,
                                     bool& failed) {
  if constexpr (N == 16 && sizeof(T) == 4) leaf16_groups(S, Xo, lane, col0, bs, info, failed);
  else leaf_rows<N>(S, Xo, lane, col0, bs, info, failed);
}

constexpr int kPotrfWaves = 8;  // 8 waves: the next leaf overlaps the trailing products
constexpr int kLeaf = 16;       // leaf width

// The diagonal block at (kb, kb) of A (lda): L^{-1} (lower, zeros above) over it,
// info = first failing column (1-based) if the block is not positive definite.
template <class T>
__global__ __launch_bounds__(64 * kPotrfWaves) void potrf_blk_kernel(T* A, int64_t lda, int kb, int bs,
                                                                    int32_t* info) {
  constexpr int NB = Blk<T>::NB, PT = diag_pitch<T>(), NT = 64 * kPotrfWaves;
  constexpr int EV = 16 / sizeof(T), NL = NB * NB / EV / NT;  // 16-byte pieces per thread
  constexpr int NLV = NB / kLeaf, NL1 = NLV - 1;
  typedef T V16 __attribute__((ext_vector_type(EV)));
  __shared__ __attribute__((aligned(16))) T As[NB * PT];
  __shared__ __attribute__((aligned(16))) T Es[NB * PT];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  // 16-byte accesses when every row start is 16-byte aligned (kb is a multiple of NB)
  const bool vec = (lda * (int64_t)sizeof(T)) % 16 == 0 && (((uintptr_t)A) & 15) == 0;
  T* Ab = A + (int64_t)kb * lda + kb;
  {
    // every load in flight before the first LDS write; both triangles are copied
    // (the leaf reads whole rows of its diagonal block), identity past bs
    V16 buf[NL];
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const int e = (u * NT + tid) * EV;  // EV consecutive columns of one row
      const int i = e / NB, j0 = e % NB;
      const T* src = Ab + (int64_t)i * lda + j0;
      if (i < bs && vec && j0 + EV - 1 < bs) {
        buf[u] = *(const V16*)src;
      } else {
#pragma unroll
        for (int t = 0; t < EV; ++t)
          buf[u][t] = (i < bs && j0 + t < bs) ? src[t] : (i == j0 + t ? T(1) : T(0));
      }
    }
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const int e = (u * NT + tid) * EV;
      const int i = e / NB, j0 = e % NB;
      // E = L^{-1} starts at zero in its strictly lower kLeaf-blocks (the diagonal
      // blocks are written whole by the leaf; the upper ones are never read)
      const bool ez = i / kLeaf > j0 / kLeaf;
      if constexpr (sizeof(T) == 4) {  // the row pitch keeps 8-byte alignment only
        *(f32x2*)&As[i * PT + j0] = f32x2{buf[u][0], buf[u][1]};
        *(f32x2*)&As[i * PT + j0 + 2] = f32x2{buf[u][2], buf[u][3]};
        if (ez) {
          *(f32x2*)&Es[i * PT + j0] = f32x2{0.f, 0.f};
          *(f32x2*)&Es[i * PT + j0 + 2] = f32x2{0.f, 0.f};
        }
      } else {
        *(V16*)&As[i * PT + j0] = buf[u];
        if (ez) *(V16*)&Es[i * PT + j0] = V16{};
      }
    }
  }
  __syncthreads();
  auto blk = [](T* base, int i, int j) { return base + (kLeaf * i) * PT + kLeaf * j; };
  bool failed = false;
  if (wid == 0) leaf<kLeaf>(blk(As, 0, 0), blk(Es, 0, 0), lane, kb, kb + bs, info, failed);
  __syncthreads();
  for (int k = 0; k < NLV; ++k) {
    // phase B: (NL1 - k) panel products, k products of the identity's row block k
    for (int q = wid; q < NL1; q += kPotrfWaves) {
      if (q < NL1 - k) {
        const int i = k + 1 + q;
        mm16<true>(blk(As, i, k), blk(As, i, k), blk(Es, k, k), (const T*)nullptr, T(1), lane);
      } else {
        const int m = q - (NL1 - k);
        mm16<false>(blk(Es, k, m), blk(Es, k, k), blk(Es, k, m), (const T*)nullptr, T(1), lane);
      }
    }
    __syncthreads();
    if (k == NL1) break;
    // phase C: trailing lower blocks (k < j <= i), then E_im for i > k, m <= k. Job 0
    // is the next diagonal block: wave 0 updates it and factors it (the next leaf)
    // while the other waves share the remaining jobs.
    const int ntr = (NL1 - k) * (NL1 - k + 1) / 2;
    const int njobs = ntr + (NL1 - k) * (k + 1);
    auto job = [&](int q) {
      if (q < ntr) {
        int i = k + 1, t = q;
        while (t > i - k - 1) {  // row i holds i - k blocks (j = k+1..i)
          t -= i - k;
          ++i;
        }
        const int j = k + 1 + t;
        mm16<true>(blk(As, i, j), blk(As, i, k), blk(As, j, k), (const T*)blk(As, i, j), T(-1), lane);
      } else {
        const int t = q - ntr;
        const int i = k + 1 + t / (k + 1), m = t % (k + 1);
        mm16<false>(blk(Es, i, m), blk(As, i, k), blk(Es, k, m), (const T*)blk(Es, i, m), T(-1), lane);
      }
    };
    if (wid == 0) {
      job(0);
      leaf<kLeaf>(blk(As, k + 1, k + 1), blk(Es, k + 1, k + 1), lane, kb + kLeaf * (k + 1), kb + bs,
                  info, failed);
    } else {
      for (int q = wid; q < njobs; q += kPotrfWaves - 1) job(q);
    }
    __syncthreads();
  }
  // recompute the store's bounds masks here rather than keep the load's alive
  int tid2 = tid;
  asm volatile("" : "+v"(tid2));
#pragma unroll
  for (int u = 0; u < NL; ++u) {
    const int e = (u * NT + tid2) * EV;
    const int i = e / NB, j0 = e % NB;
    if (i >= bs) continue;
    V16 v;
#pragma unroll
    for (int t = 0; t < EV; ++t) v[t] = j0 + t <= i ? Es[i * PT + j0 + t] : T(0);
    T* dst = Ab + (int64_t)i * lda + j0;
    if (vec && j0 + EV - 1 < bs) *(V16*)dst = v;
    else
      for (int t = 0; t < EV; ++t)
        if (j0 + t < bs) dst[t] = v[t];
  }
}

// Zeros above the nb x nb diagonal blocks inside each ob x ob diagonal block of A:
// A[i][j] = 0 for (i / nb + 1) nb <= j < min((i / ob + 1) ob, d).
template <class T>
__global__ __launch_bounds__(256) void zero_upper_kernel(T* A, int64_t d, int nb, int ob) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < d * ob;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = e / ob, j = (i / ob) * ob + e % ob;
    if (j < d && j >= (i / nb + 1) * nb) A[i * d + j] = T(0);
  }
}

// A = G + lambda I (full copy), R = C, info = 0. A workgroup copies whole rows (rows
// of A first, then of R) in 16-byte runs when source and destination allow it; the
// thread whose run holds A's diagonal element adds lambda to it.
template <class T>
__global__ __launch_bounds__(256) void init_kernel(const T* __restrict__ G, const T* __restrict__ C,
                                                   T* __restrict__ A, T* __restrict__ R, int64_t d,
                                                   int64_t dout, double lambda,
                                                   const double* lam_dev, int32_t* info) {
  constexpr int EV = 16 / sizeof(T);
  typedef T V16 __attribute__((ext_vector_type(EV)));
  const T lam = (T)(lam_dev ? *lam_dev : lambda);
  for (int64_t i = blockIdx.x; i < d + d; i += gridDim.x) {
    const bool isA = i < d;
    const int64_t r = isA ? i : i - d, n = isA ? d : dout;
    const T* src = isA ? G + r * d : C + r * dout;
    T* dst = isA ? A + r * d : R + r * dout;
    const int64_t diag = isA ? r : -1;
    if ((((uintptr_t)src | (uintptr_t)dst) & 15) == 0) {
      const int64_t nv = n / EV;
      for (int64_t v = threadIdx.x; v < nv; v += blockDim.x) {
        V16 x = *(const V16*)(src + v * EV);
        const int64_t t = diag - v * EV;
        if (t >= 0 && t < EV) x[t] += lam;
        *(V16*)(dst + v * EV) = x;
      }
      for (int64_t j = nv * EV + threadIdx.x; j < n; j += blockDim.x) dst[j] = src[j] + (j == diag ? lam : T(0));
    } else {
      for (int64_t j = threadIdx.x; j < n; j += blockDim.x) dst[j] = src[j] + (j == diag ? lam : T(0));
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *info = 0;
}

// Stage 1 of the scaled ridge: per-block partial sums of G_ij^2 and G_ii, in fp64
// and in a fixed order (each thread strides over the matrix, then the diagonal).
template <class T>
__global__ __launch_bounds__(256) void ridge_partial_kernel(const T* __restrict__ G, int64_t d,
                                                            double* part) {
  __shared__ double s2[256], st[256];
  double a = 0.0, b = 0.0;
  const int64_t first = (int64_t)blockIdx.x * 256 + threadIdx.x, stride = (int64_t)kRedBlocks * 256;
  for (int64_t e = first; e < d * d; e += stride) {
    const double v = (double)G[e];
    a = fma(v, v, a);
  }
  for (int64_t i = first; i < d; i += stride) b += (double)G[i * d + i];
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

// Stage 2: lambda = lambda_0 * sum(G^2) / tr(G) (Eq. 7, ridge 1) or lambda_0 * tr(G) / d
// (trace mean, ridge 2).
__global__ __launch_bounds__(256) void ridge_final_kernel(const double* part, double lam0, int ridge,
                                                          double d, double* lam_out) {
  __shared__ double s2[256], st[256];
  double a = 0.0, b = 0.0;
  for (int i = threadIdx.x; i < kRedBlocks; i += 256) {
    a += part[2 * i];
    b += part[2 * i + 1];
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
  if (threadIdx.x == 0) lam_out[0] = ridge == 1 ? lam0 * s2[0] / st[0] : lam0 * st[0] / d;
}

template <class T>
__global__ __launch_bounds__(256) void to_float_kernel(const T* __restrict__ X, float* __restrict__ Y,
                                                       int64_t n) {
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x)
    Y[e] = (float)X[e];
}

bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

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
  g.batch = 1;
  // vector loads along the contiguous dimension: the other stride and the base must
  // keep every 4-element group 16-byte aligned
  g.vecA = al16(A) && ((sak == 1 && sai % 4 == 0) || (sai == 1 && sak % 4 == 0));
  g.vecB = al16(B) && ((sbj == 1 && sbk % 4 == 0) || (sbk == 1 && sbj % 4 == 0));
  return g;
}

// g repeated over `count` problems, item b offset by (b bA, b bB, b bC) elements
template <class T>
GemmDesc<T> batched(GemmDesc<T> g, int count, int64_t bA, int64_t bB, int64_t bC) {
  g.batch = count;
  g.bA = bA;
  g.bB = bB;
  g.bC = bC;
  if (bA % 4 != 0) g.vecA = 0;
  if (bB % 4 != 0) g.vecB = 0;
  return g;
}

template <class T>
void set_tiles(GemmDesc<T>& g, int tile) {
  g.tiles_n = (g.N + tile - 1) / tile;
  g.tiles_b = (g.M > 0 && g.N > 0 && g.K > 0) ? ((g.M + tile - 1) / tile) * g.tiles_n : 0;
  g.ntiles = g.batch * g.tiles_b;
}

// One launch for up to two problems. fp32 uses 128 x 128 tiles unless that would
// leave most of the 256 CUs idle, then 64 x 64.
template <class T>
hipError_t run_group(const GemmDesc<T>* ds, int n, hipStream_t st) {
  GemmDesc<T> d[2] = {};
  int m = 0;
  for (int i = 0; i < n; ++i)
    if (ds[i].M > 0 && ds[i].N > 0 && ds[i].K > 0) d[m++] = ds[i];
  if (m == 0) return hipSuccess;
  if constexpr (sizeof(T) == 4) {
    for (int i = 0; i < m; ++i) set_tiles(d[i], 128);
    const bool small = d[0].ntiles + d[1].ntiles < 256;
    if (small)
      for (int i = 0; i < m; ++i) set_tiles(d[i], 64);
    const int total = d[0].ntiles + d[1].ntiles;
    if (small)
      hipLaunchKernelGGL(gemm_f32_kernel<64>, dim3(total), dim3(256), 0, st, d[0], d[1]);
    else
      hipLaunchKernelGGL(gemm_f32_kernel<128>, dim3(total), dim3(256), 0, st, d[0], d[1]);
  } else {
    for (int i = 0; i < m; ++i) set_tiles(d[i], D_T);
    const int total = d[0].ntiles + d[1].ntiles;
    hipLaunchKernelGGL(gemm_f64_kernel, dim3(total), dim3(256), 0, st, d[0], d[1]);
  }
  return hipGetLastError();
}

SGemm to_sgemm(const GemmDesc<float>& g, bool& ak, bool& bj, int tile) {
  SGemm s{};
  ak = g.sak == 1;
  bj = g.sbj == 1;
  s.A = g.A; s.sa = ak ? g.sai : g.sak;
  s.B = g.B; s.sb = bj ? g.sbk : g.sbj;
  s.C = g.C; s.ldc = g.ldc;
  s.M = g.M; s.N = g.N; s.K = g.K;
  s.alpha = g.alpha; s.beta = g.beta;
  s.lower = g.lower;
  const int tm = (g.M + tile - 1) / tile, tn = (g.N + tile - 1) / tile;
  s.tiles_n = tn;
  s.tiles_b = g.lower ? tm * (tm + 1) / 2 : tm * tn;  // a lower-triangle update is square
  s.batch = g.batch;
  s.ntiles = s.batch * s.tiles_b;
  s.bA = g.bA; s.bB = g.bB; s.bC = g.bC;
  s.vecA = g.vecA; s.vecB = g.vecB;
  s.vecC = al16(g.C) && g.ldc % 4 == 0 && g.bC % 4 == 0;
  return s;
}

// fp32 products on three bf16 MFMA terms, up to two problems per launch. The
// operand layouts the solve uses: A contiguous along k with B along k or j, or A
// contiguous along i with B along j.
template <int TERMS>
hipError_t run_group_split(const GemmDesc<float>* ds, int n, hipStream_t st) {
  SGemm s[2] = {};
  bool ak[2] = {true, true}, bj[2] = {true, true};
  // K <= 128 everywhere (the factorisation's block-column updates) and too few 128 x 128
  // tiles to fill the CUs: the small-K kernel (latency rather than throughput)
  int kmax = 0, tiles128 = 0;
  for (int i = 0; i < n; ++i)
    if (ds[i].M > 0 && ds[i].N > 0 && ds[i].K > 0) {
      bool a, b;
      kmax = std::max(kmax, ds[i].K);
      tiles128 += to_sgemm(ds[i], a, b, S_BM).ntiles;
    }
  const bool small = kmax <= T_KMAX && tiles128 < 256;
  int m = 0;
  for (int i = 0; i < n; ++i)
    if (ds[i].M > 0 && ds[i].N > 0 && ds[i].K > 0) {
      s[m] = to_sgemm(ds[i], ak[m], bj[m], small ? T_BM : S_BM);
      ++m;
    }
  if (m == 0) return hipSuccess;
  if (m == 1) {
    ak[1] = ak[0];
    bj[1] = bj[0];
  }
  const int total = s[0].ntiles + s[1].ntiles;
  const dim3 grid((total + kXcds - 1) / kXcds * kXcds), block(256);
  const int key = (ak[0] << 3) | (bj[0] << 2) | (ak[1] << 1) | (int)bj[1];
#define PKV_SG(A0, B0, A1, B1)                                                                  \
  do {                                                                                          \
    if (small)                                                                                  \
      hipLaunchKernelGGL((sgemm3s_kernel<TERMS, A0, B0, A1, B1>), grid, block, 0, st, s[0], s[1]); \
    else                                                                                        \
      hipLaunchKernelGGL((sgemm3_kernel<TERMS, A0, B0, A1, B1>), grid, block, 0, st, s[0], s[1]);  \
  } while (0)
  switch (key) {
    case 0b1011: PKV_SG(true, false, true, true); break;
    case 0b1010: PKV_SG(true, false, true, false); break;
    case 0b1111: PKV_SG(true, true, true, true); break;
    case 0b0101: PKV_SG(false, true, false, true); break;
    default: return hipErrorInvalidValue;
  }
#undef PKV_SG
  return hipGetLastError();
}

// Column blocks of NB are grouped into outer blocks of kSolveNBO * NB (1024 wide in fp32;
// solve at d = 4096: 2.46 ms, 4 column blocks: 2.53, 16: 2.59)
constexpr int kSolveNBO = 8;

struct SolveLayout {
  size_t A, Lm, R, Z, X, Tw, part, lam, total;
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
  // products of the backward's block inversion: at most (d / 2s + 1) s^2 for s <= OB / 2
  {
    const int64_t ob = (int64_t)kSolveNBO * Blk<T>::NB;
    L.Tw = o; o += align_up(sizeof(T) * (d + ob) * ob / 2);
  }
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
                   int ridge, int products, float* dW, int32_t* info, void* ws, hipStream_t st) {
  constexpr int NB = Blk<T>::NB;
  const SolveLayout L = layout<T>(d64, dout64);
  char* w = (char*)ws;
  T* A = (T*)(w + L.A);
  T* Lm = (T*)(w + L.Lm);
  T* R = (T*)(w + L.R);
  T* Z = (T*)(w + L.Z);
  // the backward substitution's result: in fp32 directly the caller's dW (G and C are
  // read only before it is written), in fp64 a workspace matrix converted at the end
  T* X = sizeof(T) == 4 ? (T*)dW : (T*)(w + L.X);
  double* part = (double*)(w + L.part);
  double* lam = (double*)(w + L.lam);
  const int d = (int)d64, dout = (int)dout64;

  const bool scaled = ridge != 0;  // the coefficient is lambda times a statistic of G
  if (scaled) {
    hipLaunchKernelGGL((ridge_partial_kernel<T>), dim3(kRedBlocks), dim3(256), 0, st, G, d64, part);
    PKV_TRY(hipGetLastError());
    hipLaunchKernelGGL(ridge_final_kernel, dim3(1), dim3(256), 0, st, part, lambda, ridge, (double)d64,
                       lam);
    PKV_TRY(hipGetLastError());
  }
  {
    const int blocks = (int)std::min<int64_t>(2 * d64, 4096);
    hipLaunchKernelGGL((init_kernel<T>), dim3(blocks), dim3(256), 0, st, G, C, A, R, d64, dout64,
                       lambda, scaled ? lam : (const double*)nullptr, info);
    PKV_TRY(hipGetLastError());
  }
  const T one = T(1), zero = T(0), mone = T(-1);
  auto run = [&](const GemmDesc<T>* g, int n) -> hipError_t {
    if constexpr (sizeof(T) == 4) {
      if (products == kProductsSplit6) return run_group_split<6>(g, n, st);
      if (products == kProductsSplit3) return run_group_split<3>(g, n, st);
    }
    return run_group(g, n, st);
  };
  // Column blocks of NB are grouped into outer blocks of OB = NBO * NB. Within an
  // outer block only its own remaining column blocks (and their rows of R) are
  // updated after each panel; the rest of the trailing matrix and of R is updated
  // once per outer block with K = OB, which divides the read-modify-write traffic
  // of the large updates by NBO. The backward substitution is grouped the same way.
  constexpr int NBO = kSolveNBO;
  const int OB = NBO * NB;
  for (int K0 = 0; K0 < d; K0 += OB) {
    const int W = std::min(OB, d - K0);  // width of this outer block
    for (int kb = K0; kb < K0 + W; kb += NB) {
      const int bs = std::min(NB, d - kb);
      const int rest = d - kb - bs;
      hipLaunchKernelGGL((potrf_blk_kernel<T>), dim3(1), dim3(64 * kPotrfWaves), 0, st, A, d64, kb, bs,
                         info);
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
        PKV_TRY(run(g, 2));
      }
      const int kb1 = kb + bs;
      if (kb1 < K0 + W) {
        // the remaining column blocks of this outer block (columns kb1..K0+W, all rows
        // from kb1): A[kb1.., kb1..K0+W] -= L[kb1.., k] L[kb1..K0+W, k]^T, and their rows
        // of R: R[kb1..K0+W] -= L[kb1..K0+W, k] Z_k
        const int wr = K0 + W - kb1;
        const T* Lr = Lm + (int64_t)kb1 * d + kb;  // rows kb1.., cols of block k
        GemmDesc<T> g[2];
        g[0] = desc<T>(Lr, d, 1, Lr, 1, d, A + (int64_t)kb1 * d + kb1, d, d - kb1, wr, bs, mone, one);
        g[1] = desc<T>(Lr, d, 1, Z + (int64_t)kb * dout, dout, 1, R + (int64_t)kb1 * dout, dout, wr,
                       dout, bs, mone, one);
        PKV_TRY(run(g, 2));
      }
    }
    const int T0 = K0 + W, restT = d - T0;
    if (restT > 0) {
      GemmDesc<T> g[2];
      const T* Lp = Lm + (int64_t)T0 * d + K0;  // panel rows T0.., cols K0..K0+W
      // A_ij -= L_iK L_jK^T over the trailing lower blocks (K = W)
      g[0] = desc<T>(Lp, d, 1, Lp, 1, d, A + (int64_t)T0 * d + T0, d, restT, restT, W, mone, one, 1);
      // R_i -= L_iK Z_K
      g[1] = desc<T>(Lp, d, 1, Z + (int64_t)K0 * dout, dout, 1, R + (int64_t)T0 * dout, dout, restT,
                     dout, W, mone, one);
      PKV_TRY(run(g, 2));
    }
  }
  // Backward substitution, X = L^{-T} Z, one outer block at a time on the inverse
  // M = L_OO^{-1} of its OB x OB diagonal block of L. M is assembled in place of that
  // block of A from the NB x NB inverses the factorisation left there, by doubling:
  // for s = NB, 2 NB, .., OB / 2, every pair of adjacent s-wide blocks (aligned to 2s)
  // gets [[M_1, 0], [L_21, M_2]]^{-1} = [[M_1, 0], [-M_2 L_21 M_1, M_2]], all pairs
  // of a level in one batched launch per product (the last pair, which may be short,
  // as a second problem). Each outer block then takes two launches instead of two
  // per column block.
  T* Tw = (T*)(w + L.Tw);
  {
    const int blocks = (int)std::min<int64_t>((d64 * OB + 255) / 256, 4096);
    hipLaunchKernelGGL((zero_upper_kernel<T>), dim3(blocks), dim3(256), 0, st, A, d64, NB, OB);
    PKV_TRY(hipGetLastError());
  }
  for (int s = NB; s < OB && s < d; s *= 2) {
    const int full = d / (2 * s);                // pairs with both halves s wide
    const int q_r = full * 2 * s, s2_r = d - q_r - s;  // the short last pair, if s2_r > 0
    const int64_t step = (int64_t)2 * s * (d + 1);    // diagonal offset between pairs
    GemmDesc<T> g[2];
    int n = 0;
    // Tw_p = L_21 M_1
    if (full > 0)
      g[n++] = batched(desc<T>(Lm + (int64_t)s * d, d, 1, A, d, 1, Tw, s, s, s, s, one, zero), full, step,
                       step, (int64_t)s * s);
    if (s2_r > 0)
      g[n++] = desc<T>(Lm + (int64_t)(q_r + s) * d + q_r, d, 1, A + (int64_t)q_r * d + q_r, d, 1,
                       Tw + (int64_t)full * s * s, s, s2_r, s, s, one, zero);
    PKV_TRY(run(g, n));
    n = 0;
    // M_21 = -M_2 Tw_p, into the lower-left block of the pair
    if (full > 0)
      g[n++] = batched(desc<T>(A + (int64_t)s * d + s, d, 1, Tw, s, 1, A + (int64_t)s * d, d, s, s, s, mone,
                               zero),
                       full, step, (int64_t)s * s, step);
    if (s2_r > 0)
      g[n++] = desc<T>(A + (int64_t)(q_r + s) * d + q_r + s, d, 1, Tw + (int64_t)full * s * s, s, 1,
                       A + (int64_t)(q_r + s) * d + q_r, d, s2_r, s, s2_r, mone, zero);
    PKV_TRY(run(g, n));
  }
  const int nout = (d + OB - 1) / OB;
  for (int ko = nout - 1; ko >= 0; --ko) {
    const int K0 = ko * OB, W = std::min(OB, d - K0);
    {
      // X_O = M^T Z_O : X(i,n) = sum_t M[t][i] Z[K0+t][n]
      GemmDesc<T> g = desc<T>(A + (int64_t)K0 * d + K0, 1, d, Z + (int64_t)K0 * dout, dout, 1,
                              X + (int64_t)K0 * dout, dout, W, dout, W, one, zero);
      PKV_TRY(run(&g, 1));
    }
    if (K0 > 0) {
      // Z_i -= L_Ki^T X_K for i < K0 : Z(i,n) -= sum_t Lm[K0+t][i] X[K0+t][n] (K = W)
      GemmDesc<T> g = desc<T>(Lm + (int64_t)K0 * d, 1, d, X + (int64_t)K0 * dout, dout, 1, Z, dout, K0,
                              dout, W, mone, one);
      PKV_TRY(run(&g, 1));
    }
  }
  if constexpr (sizeof(T) == 8) {
    const int64_t n = d64 * dout64;
    const int blocks = (int)std::min<int64_t>((n + 255) / 256, 4096);
    hipLaunchKernelGGL((to_float_kernel<T>), dim3(blocks), dim3(256), 0, st, X, dW, n);
    PKV_TRY(hipGetLastError());
  }
  return hipSuccess;
}

// ---------------------------------------------------------------- reduced-rank patch
//
// dW_r = dW U_r U_r^T with U_r the top-r eigenvectors of S = dW^T G dW (d_out x d_out),
// found by subspace iteration on MFMA GEMMs: Q <- orth(S' Q) with a block of
// kRrrBlock >= r columns, S' = S + mu I with mu = 1e-5 trace(S) >= 1e-5 lambda_max
// (the same eigenvectors; S' Q keeps full column rank, to fp32 accuracy, when S has
// a low numerical rank). orth is Cholesky QR with the Gram matrix Z^T Z formed and
// factored in fp64 (its condition number is that of Z squared, up to 1e10), then
// Q = Z L^-T on fp32 MFMA; two more passes at the end make Q orthonormal to
// rounding. Rayleigh-Ritz: the kRrrBlock x kRrrBlock matrix Q^T S' Q is
// diagonalised by parallel Jacobi in fp64 in one workgroup and its top-r
// eigenvectors map back through Q.

constexpr int kRrrBlock = 64;   // subspace width (r <= it)
static_assert(kRrrBlock <= 64, "the tall-skinny products take at most 64 columns");
constexpr int kJacobiSweeps = 14;

// M[i][i] += rel * trace(M) / n (one workgroup; the trace in fp64, fixed order)
__global__ __launch_bounds__(256) void diag_shift_kernel(float* M, int64_t n, int64_t ld, float rel) {
  __shared__ double part[256];
  double t = 0.0;
  for (int64_t i = threadIdx.x; i < n; i += 256) t += (double)M[i * ld + i];
  part[threadIdx.x] = t;
  __syncthreads();
  for (int s2 = 128; s2 > 0; s2 >>= 1) {
    if ((int)threadIdx.x < s2) part[threadIdx.x] += part[threadIdx.x + s2];
    __syncthreads();
  }
  const float mu = (float)(rel * part[0] / (double)n);
  for (int64_t i = threadIdx.x; i < n; i += 256) M[i * ld + i] += mu;
}

// Tall-skinny products of the subspace iteration: C [rows][nc] = A [rows][K] B [K][nc]
// (nc <= kRrrBlock), row-major with leading dimensions lda, ldb, ldc. One workgroup
// per 16 rows of C; its eight waves take interleaved 16-wide chunks of K (wave w:
// chunks w, w + 8, ...), so the waves of a workgroup read adjacent 64-byte segments of
// the same rows of A. Each wave keeps a 16 x 16 tile per 16 columns of C on fp32 MFMA
// 16x16x4 (exact fp32 products, fp32 accumulation) with the next chunk's operands
// loaded while the current one is multiplied; the eight partial tiles are summed in
// LDS in wave order (deterministic). Lane l holds row l % 16 of the A chunk, columns
// 4 (l / 16) .. +3, and the matching rows of B for column l % 16 of each tile.
constexpr int kTsWaves = 8;
__device__ __forceinline__ f32x4 mfma16_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
template <int NCT>
__global__ __launch_bounds__(64 * kTsWaves) void tsgemm_kernel(const float* __restrict__ A, int64_t lda,
                                                               const float* __restrict__ B, int64_t ldb,
                                                               int64_t rows, int K, int nc,
                                                               float* __restrict__ C, int64_t ldc) {
  __shared__ float red[kTsWaves][NCT][4][64];
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6, l16 = lane & 15, g = lane >> 4;
  const int64_t r0 = (int64_t)blockIdx.x * 16;
  const int64_t row = r0 + l16;
  const bool va = (lda & 3) == 0 && (((uintptr_t)A) & 15) == 0;
  f32x4 a_cur, a_nxt;
  float b_cur[NCT][4], b_nxt[NCT][4];
  auto load = [&](int k0, f32x4& a, float (&b)[NCT][4]) {
    const int k = k0 + 4 * g;
    if (row < rows && va && k + 3 < K) {
      a = *(const f32x4*)(A + row * lda + k);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) a[t] = (row < rows && k + t < K) ? A[row * lda + k + t] : 0.f;
    }
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
      const int c = 16 * ct + l16;
#pragma unroll
      for (int t = 0; t < 4; ++t) b[ct][t] = (k + t < K && c < nc) ? B[(int64_t)(k + t) * ldb + c] : 0.f;
    }
  };
  f32x4 acc[NCT];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
  constexpr int step = 16 * kTsWaves;
  int k0 = 16 * wid;
  if (k0 < K) load(k0, a_cur, b_cur);
  for (; k0 < K; k0 += step) {
    if (k0 + step < K) load(k0 + step, a_nxt, b_nxt);
#pragma unroll
    for (int t = 0; t < 4; ++t)
#pragma unroll
      for (int ct = 0; ct < NCT; ++ct) acc[ct] = mfma16_f32(a_cur[t], b_cur[ct][t], acc[ct]);
    a_cur = a_nxt;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
      for (int t = 0; t < 4; ++t) b_cur[ct][t] = b_nxt[ct][t];
  }
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[wid][ct][e][lane] = acc[ct][e];
  __syncthreads();
  // element (ct, e, lane) of the tile is C[r0 + 4 (lane / 16) + e][16 ct + lane % 16]
  for (int q = tid; q < NCT * 4 * 64; q += 64 * kTsWaves) {
    const int ct = q / 256, e = (q / 64) % 4, ln = q % 64;
    float v = 0.f;
#pragma unroll
    for (int w = 0; w < kTsWaves; ++w) v += red[w][ct][e][ln];
    const int64_t rr = r0 + 4 * (ln >> 4) + e;
    const int c = 16 * ct + (ln & 15);
    if (rr < rows && c < nc) C[rr * ldc + c] = v;
  }
}

// Partial sums of X^T Y in fp64 (X, Y [rows][b] fp32, b <= kRrrBlock) over slice z of
// the rows: part[z][i][j]; one workgroup per 16 x 16 tile and slice.
constexpr int kGramSlices = 16;
__global__ __launch_bounds__(256) void gram_partial_kernel(const float* __restrict__ X,
                                                           const float* __restrict__ Y, int64_t rows,
                                                           int b, double* __restrict__ part) {
  __shared__ float xs[64][17], ys[64][17];
  const int i0 = blockIdx.y * 16, j0 = blockIdx.x * 16, z = blockIdx.z, tid = threadIdx.x;
  const int ti = tid / 16, tj = tid % 16;
  const int64_t per = (rows + kGramSlices - 1) / kGramSlices;
  const int64_t lo = z * per, hi = std::min<int64_t>(rows, lo + per);
  double acc = 0.0;
  for (int64_t k0 = lo; k0 < hi; k0 += 64) {
    for (int e = tid; e < 64 * 16; e += 256) {
      const int kk = e / 16, c = e % 16;
      const int64_t k = k0 + kk;
      xs[kk][c] = (k < hi && i0 + c < b) ? X[k * b + i0 + c] : 0.f;
      ys[kk][c] = (k < hi && j0 + c < b) ? Y[k * b + j0 + c] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int kk = 0; kk < 64; ++kk) acc = fma((double)xs[kk][ti], (double)ys[kk][tj], acc);
    __syncthreads();
  }
  if (i0 + ti < b && j0 + tj < b) part[((int64_t)z * b + i0 + ti) * b + j0 + tj] = acc;
}

// W = sum over the slices, in slice order (fp64)
__global__ __launch_bounds__(256) void gram_reduce_kernel(const double* __restrict__ part, int b,
                                                          double* __restrict__ W) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= b * b) return;
  double s = 0.0;
  for (int z = 0; z < kGramSlices; ++z) s += part[(int64_t)z * b * b + e];
  W[e] = s;
}

// Wt[k][j] = (float) L^-1[j][k]: the transposed inverse factor, row-major, for tsgemm
__global__ __launch_bounds__(256) void linv_t_kernel(const double* __restrict__ Linv, int b,
                                                     float* __restrict__ Wt) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= b * b) return;
  const int k = e / b, j = e % b;
  Wt[e] = (float)Linv[j * b + k];
}

// Q[i][j] = a counter-based pseudo-random value in [-1, 1) of (i, j)
__global__ __launch_bounds__(256) void rrr_init_kernel(float* Q, int64_t rows, int b, int* info) {
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (e == 0) *info = 0;
  if (e >= rows * b) return;
  uint32_t h = (uint32_t)e * 0x9E3779B9u + 0x7F4A7C15u;
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  Q[e] = (float)(h >> 8) * (2.0f / 16777216.0f) - 1.0f;
}

// Eigenvectors of the symmetric b x b matrix (T + T^T) / 2 (b even, <= kRrrBlock) by
// parallel cyclic Jacobi in fp64: each step rotates NB/2 disjoint index pairs of a
// round-robin schedule, columns then rows. The matrix is padded with zeros to
// NB = kRrrBlock (a padded index never couples, so its rotations are the identity,
// and it never enters the ranking), so all index arithmetic is compile-time. Thread
// tid takes row (column update) or column (row update) tid % 64 of pairs tid / 64 + 4u:
// the lanes of a wave read one pair's entries down a column or along a row, which
// spreads them over the LDS banks. Vr [b][r] receives the
// eigenvectors of the r largest eigenvalues, in descending order (ties: lower index
// first); w [b] all eigenvalues by index.
__global__ __launch_bounds__(256) void jacobi_top_kernel(const double* __restrict__ T, int b, int r,
                                                         float* __restrict__ Vr,
                                                         double* __restrict__ w) {
  constexpr int NB = kRrrBlock, P = NB + 1, HALF = NB / 2;
  static_assert(NB == 64, "thread mapping assumes a 64-wide block and 256 threads");
  __shared__ double A[NB * P], V[NB * P];
  __shared__ double cs[HALF][2];
  __shared__ int pq[HALF][2];
  __shared__ double red[2][256];
  __shared__ int done;
  const int tid = threadIdx.x;
  for (int e = tid; e < NB * NB; e += 256) {
    const int i = e / NB, j = e % NB;
    double a = 0.0;
    if (i < b && j < b) a = 0.5 * (T[i * b + j] + T[j * b + i]);
    A[i * P + j] = a;
    V[i * P + j] = i == j ? 1.0 : 0.0;
  }
  __syncthreads();
  const int kk = tid % NB, t0 = tid / NB;  // this thread's row / column and first pair
  for (int sweep = 0; sweep < kJacobiSweeps; ++sweep) {
    // stop once the off-diagonal mass is below 1e-24 of the diagonal's: an eigenvector
    // is then off by about 1e-12 ||A|| / gap, far below the fp32 output's precision
    double off = 0.0, dia = 0.0;
    for (int e = tid; e < NB * NB; e += 256) {
      const int i = e / NB, j = e % NB;
      if (i >= b || j >= b) continue;
      const double v = A[i * P + j] * A[i * P + j];
      if (i == j) dia += v; else off += v;
    }
    red[0][tid] = off;
    red[1][tid] = dia;
    __syncthreads();
    for (int s2 = 128; s2 > 0; s2 >>= 1) {
      if (tid < s2) {
        red[0][tid] += red[0][tid + s2];
        red[1][tid] += red[1][tid + s2];
      }
      __syncthreads();
    }
    if (tid == 0) done = red[0][0] <= 1e-24 * red[1][0];
    __syncthreads();
    if (done) break;
#pragma unroll 1
    for (int step = 0; step < NB - 1; ++step) {
      if (tid < HALF) {
        // round robin: position 0 fixed, the others rotate by `step`
        auto at = [&](int k) { return k == 0 ? 0 : (k - 1 + step) % (NB - 1) + 1; };
        int p = at(tid), q = at(NB - 1 - tid);
        if (p > q) { const int t = p; p = q; q = t; }
        const double apq = A[p * P + q];
        double c = 1.0, s = 0.0;
        if (fabs(apq) > 1e-300) {
          // t = tan of the rotation angle, the root of t^2 + 2 th t - 1 of smaller
          // magnitude; native fp64 reciprocal and reciprocal square root, each with one
          // Newton step, so that c^2 + s^2 = 1 to fp64 rounding
          const double th = (A[q * P + q] - A[p * P + p]) * rcp64(2.0 * apq);
          const double ath = fabs(th);
          double t;
          if (ath < 1e150) {
            const double y = fma(th, th, 1.0);
            t = rcp64(ath + y * rsq64(y));
          } else {
            t = 0.5 * rcp64(ath);
          }
          if (th < 0.0) t = -t;
          c = rsq64(fma(t, t, 1.0));
          s = t * c;
        }
        pq[tid][0] = p;
        pq[tid][1] = q;
        cs[tid][0] = c;
        cs[tid][1] = s;
      }
      __syncthreads();
      // this thread's 8 pairs, read once for both halves of the step
      int pp[HALF / 4], qq[HALF / 4];
      double cc[HALF / 4], ss[HALF / 4];
#pragma unroll
      for (int u = 0; u < HALF / 4; ++u) {
        const int t = t0 + 4 * u;
        pp[u] = pq[t][0];
        qq[u] = pq[t][1];
        cc[u] = cs[t][0];
        ss[u] = cs[t][1];
      }
      // columns: A <- A J, V <- V J
#pragma unroll
      for (int u = 0; u < HALF / 4; ++u) {
        const int p = pp[u], q = qq[u];
        const double c = cc[u], s = ss[u];
        const double akp = A[kk * P + p], akq = A[kk * P + q];
        A[kk * P + p] = c * akp - s * akq;
        A[kk * P + q] = s * akp + c * akq;
        const double vkp = V[kk * P + p], vkq = V[kk * P + q];
        V[kk * P + p] = c * vkp - s * vkq;
        V[kk * P + q] = s * vkp + c * vkq;
      }
      __syncthreads();
      // rows: A <- J^T A
#pragma unroll
      for (int u = 0; u < HALF / 4; ++u) {
        const int p = pp[u], q = qq[u];
        const double c = cc[u], s = ss[u];
        const double apk = A[p * P + kk], aqk = A[q * P + kk];
        A[p * P + kk] = c * apk - s * aqk;
        A[q * P + kk] = s * apk + c * aqk;
      }
      __syncthreads();
    }
  }
  if (tid < b) {
    const double wi = A[tid * P + tid];
    w[tid] = wi;
    int rank = 0;
    for (int j = 0; j < b; ++j) {
      const double wj = A[j * P + j];
      rank += (wj > wi || (wj == wi && j < tid)) ? 1 : 0;
    }
    if (rank < r)
      for (int k = 0; k < b; ++k) Vr[k * r + rank] = (float)V[k * P + tid];
  }
}

struct RrrWs {
  size_t X, S, Q, Z, Y, W, W64, part, T, Vr, w, info, total;
};
RrrWs rrr_layout(int64_t din, int64_t dout, int b) {
  RrrWs L{};
  size_t o = 0;
  auto take = [&](size_t n) { const size_t at = o; o += align_up(n); return at; };
  L.X = take((size_t)din * dout * 4);
  L.S = take((size_t)dout * dout * 4);
  L.Q = take((size_t)dout * b * 4);
  L.Z = take((size_t)dout * b * 4);
  L.Y = take((size_t)dout * b * 4);
  L.W = take((size_t)b * b * 4);
  L.W64 = take((size_t)b * b * 8);
  L.part = take((size_t)kGramSlices * b * b * 8);
  L.T = take((size_t)b * b * 8);
  L.Vr = take((size_t)b * b * 4);
  L.w = take((size_t)b * 8);
  L.info = take(16);
  L.total = o;
  return L;
}
int rrr_block(int64_t dout) { return (int)std::min<int64_t>(kRrrBlock, dout) & ~1; }

}  // namespace

size_t low_rank_ws_bytes(int64_t din, int64_t dout) {
  return rrr_layout(din, dout, rrr_block(dout)).total;
}

hipError_t launch_low_rank(const float* G, const float* dW, int64_t din, int64_t dout, int r,
                           int iters, float* A, float* U, float* dWr, void* ws, hipStream_t st) {
  const int b = rrr_block(dout);
  const RrrWs L = rrr_layout(din, dout, b);
  char* w = (char*)ws;
  float *X = (float*)(w + L.X), *S = (float*)(w + L.S), *Q = (float*)(w + L.Q);
  float *Z = (float*)(w + L.Z), *Y = (float*)(w + L.Y), *W = (float*)(w + L.W);
  float* Vr = (float*)(w + L.Vr);
  double *W64 = (double*)(w + L.W64), *part = (double*)(w + L.part), *T = (double*)(w + L.T);
  double* ev = (double*)(w + L.w);
  int32_t* info = (int32_t*)(w + L.info);
  const int din_i = (int)din, dout_i = (int)dout;
  // S = dW^T (G dW): the two large products on the split-bf16 path
  {
    GemmDesc<float> g = desc<float>(G, din, 1, dW, dout, 1, X, dout, din_i, dout_i, din_i, 1.f, 0.f);
    PKV_TRY(run_group_split<6>(&g, 1, st));
    g = desc<float>(dW, 1, dout, X, dout, 1, S, dout, dout_i, dout_i, din_i, 1.f, 0.f);
    PKV_TRY(run_group_split<6>(&g, 1, st));
  }
  hipLaunchKernelGGL(diag_shift_kernel, dim3(1), dim3(256), 0, st, S, dout, dout,
                     (float)(1e-5 * (double)dout));
  PKV_TRY(hipGetLastError());
  {
    const int64_t n = dout * b;
    hipLaunchKernelGGL(rrr_init_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, Q, dout,
                       b, info);
    PKV_TRY(hipGetLastError());
  }
  // C [rows][nc] = A [rows][K] B [K][nc] (tall-skinny, fp32)
  auto ts = [&](const float* Am, int64_t lda, const float* Bm, int64_t ldb, int64_t rows, int K,
                int nc, float* Cm, int64_t ldc) -> hipError_t {
    const dim3 grid((unsigned)((rows + 15) / 16)), block(64 * kTsWaves);
    switch ((nc + 15) / 16) {
      case 1: hipLaunchKernelGGL(tsgemm_kernel<1>, grid, block, 0, st, Am, lda, Bm, ldb, rows, K, nc, Cm, ldc); break;
      case 2: hipLaunchKernelGGL(tsgemm_kernel<2>, grid, block, 0, st, Am, lda, Bm, ldb, rows, K, nc, Cm, ldc); break;
      case 3: hipLaunchKernelGGL(tsgemm_kernel<3>, grid, block, 0, st, Am, lda, Bm, ldb, rows, K, nc, Cm, ldc); break;
      case 4: hipLaunchKernelGGL(tsgemm_kernel<4>, grid, block, 0, st, Am, lda, Bm, ldb, rows, K, nc, Cm, ldc); break;
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  };
  // fp64 X^T Y [b][b]
  auto gram = [&](const float* Xm, const float* Ym, double* out) -> hipError_t {
    const dim3 gg((unsigned)((b + 15) / 16), (unsigned)((b + 15) / 16), kGramSlices);
    hipLaunchKernelGGL(gram_partial_kernel, gg, dim3(256), 0, st, Xm, Ym, dout, b, part);
    PKV_TRY(hipGetLastError());
    hipLaunchKernelGGL(gram_reduce_kernel, dim3((b * b + 255) / 256), dim3(256), 0, st, part, b, out);
    return hipGetLastError();
  };
  // src (dout x b) -> dst = src L^-T with src^T src = L L^T (Gram and factor in fp64)
  auto orth = [&](const float* src, float* dst) -> hipError_t {
    PKV_TRY(gram(src, src, W64));
    hipLaunchKernelGGL((potrf_blk_kernel<double>), dim3(1), dim3(64 * kPotrfWaves), 0, st, W64,
                       (int64_t)b, 0, b, info);
    PKV_TRY(hipGetLastError());
    hipLaunchKernelGGL(linv_t_kernel, dim3((b * b + 255) / 256), dim3(256), 0, st, W64, b, W);
    PKV_TRY(hipGetLastError());
    return ts(src, b, W, b, dout, b, b, dst, b);
  };
  // one power step per orthonormalisation: cond(Z) <= lambda_max / mu <= 1e5, so the
  // fp64 Gram matrix (its square) stays factorable
  for (int it = 0; it < iters; ++it) {
    PKV_TRY(ts(S, dout, Q, b, dout, dout_i, b, Z, b));
    PKV_TRY(orth(Z, Q));
  }
  PKV_TRY(orth(Q, Y));  // two more passes: orthonormal to rounding
  PKV_TRY(orth(Y, Z));
  // Rayleigh-Ritz: T = Z^T S Z (fp64), its top-r eigenvectors, U = Z Vr
  PKV_TRY(ts(S, dout, Z, b, dout, dout_i, b, Y, b));
  PKV_TRY(gram(Z, Y, T));
  hipLaunchKernelGGL(jacobi_top_kernel, dim3(1), dim3(256), 0, st, T, b, r, Vr, ev);
  PKV_TRY(hipGetLastError());
  PKV_TRY(ts(Z, b, Vr, r, dout, b, r, U, r));
  PKV_TRY(ts(dW, dout, U, r, din, dout_i, r, A, r));
  if (dWr) {
    GemmDesc<float> g = desc<float>(A, r, 1, U, 1, r, dWr, dout, din_i, dout_i, r, 1.f, 0.f);
    PKV_TRY(run_group(&g, 1, st));
  }
  return hipSuccess;
}

size_t solve_ws_bytes(bool f64, int64_t din, int64_t dout) {
  return f64 ? layout<double>(din, dout).total : layout<float>(din, dout).total;
}

hipError_t launch_solve(bool f64, const void* G, const void* C, int64_t din, int64_t dout,
                        double lambda, int ridge, int products, float* dW, int32_t* info,
                        void* ws, hipStream_t st) {
  if (f64)
    return solve_t<double>((const double*)G, (const double*)C, din, dout, lambda, ridge,
                           kProductsExact, dW, info, ws, st);
  return solve_t<float>((const float*)G, (const float*)C, din, dout, lambda, ridge, products, dW,
                        info, ws, st);
}

}  // namespace pkv
