// Targets and sufficient statistics (Eq. 5 and Eq. 9, row form):
//   T = (O_f - O_c) W + rho (O_f - O_c)
//   G (+)= X^T X,   C (+)= X^T (Yf - Yc)
// and the MLP-shaped block (Sec. 2.2; Alg. 1): SwiGLU features of the RMS-normed
// attention output, targets through the down-projection plus the attention
// residual, and the student state through the patched block.
//
// fp32-accumulate path: split pre-passes + bgemm_kernel (bf16 MFMA, fp32 accumulation).
// fp64-accumulate path (f64_gemm_kernel): plain fp64 FMA tiles through LDS.
#include <algorithm>
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace pkv {

namespace {

// ---------------------------------------------------------------- fp32 path
//
// Every fp32 operand x is first split, once, into x_hi = bf16(x) and
// x_lo = bf16(x - x_hi) by a memory-bound pre-pass that also lays it out with the
// contraction index contiguous and zero-pads both dimensions (rows to 128, the
// contraction to 64). The products then run on one bf16 MFMA GEMM kernel that sums
// several (A_t, B_t) term pairs with fp32 accumulation:
//   x y ~ x_hi y_hi + x_hi y_lo + x_lo y_hi (+ x_lo y_lo for the Gram matrix).
// Dropping x_lo y_lo in G would subtract a PSD matrix L^T L whose diagonal grows
// with the number of rows (a systematic shift of the ridge), so G keeps all four
// products; C keeps three (its lo x lo cross term has no such bias). A bf16 operand
// (W) has no low part.

constexpr int G_BM = 256, G_KC = 64;  // row and contraction padding of the split planes

inline int64_t pad_to(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// dst[r][c] (r < rows_p, c < cols_p), hi and lo planes, = split(S1 - S2)[r][c] inside
// rows x cols, zero outside. One thread per 8 consecutive columns.
__global__ __launch_bounds__(256) void split_rows_kernel(const float* __restrict__ S1,
                                                         const float* __restrict__ S2, int rows,
                                                         int cols, int64_t ld, __bf16* __restrict__ hi,
                                                         __bf16* __restrict__ lo, int rows_p,
                                                         int cols_p) {
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per_row = cols_p / 8;
  if (g >= (int64_t)rows_p * per_row) return;
  const int r = (int)(g / per_row), c0 = (int)(g % per_row) * 8;
  float v[8];
  const bool vec = (ld & 3) == 0 && (((uintptr_t)S1 | (uintptr_t)S2) & 15) == 0;
  if (r < rows && c0 + 7 < cols && vec) {
    const f32x4* p1 = (const f32x4*)(S1 + (int64_t)r * ld + c0);
    f32x4 a = p1[0], b = p1[1];
    if (S2) {
      const f32x4* p2 = (const f32x4*)(S2 + (int64_t)r * ld + c0);
      a -= p2[0];
      b -= p2[1];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      v[e] = a[e];
      v[4 + e] = b[e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int c = c0 + e;
      v[e] = (r < rows && c < cols)
                 ? S1[(int64_t)r * ld + c] - (S2 ? S2[(int64_t)r * ld + c] : 0.f)
                 : 0.f;
    }
  }
  bf16x8 h, l;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    h[e] = to_bf16(v[e]);
    l[e] = to_bf16(v[e] - (float)h[e]);
  }
  const int64_t o = (int64_t)r * cols_p + c0;
  *(bf16x8*)(hi + o) = h;
  *(bf16x8*)(lo + o) = l;
}

// dst[c][r] (c < cols_p, r < rows_p) = split(S1 + s2 S2)[r][c] inside rows x cols,
// zero outside: the transpose, through a 128 x 64 LDS tile (s2 = -1: a difference,
// +1: a bf16 weight plus an fp32 patch). SRC float (hi and lo planes,
// lo may be null for a bf16 source) or bf16 (hi plane only). Each thread reads 4
// consecutive source columns (one vector load when vec is set: S1, S2 and ld allow
// it), and 16 threads write one 256-byte run of a destination row.
template <class SRC>
__global__ __launch_bounds__(256) void split_transpose_kernel(const SRC* __restrict__ S1,
                                                              const float* __restrict__ S2, float s2,
                                                              int rows, int cols, int64_t ld,
                                                              __bf16* __restrict__ hi,
                                                              __bf16* __restrict__ lo, int rows_p,
                                                              int cols_p, int vec) {
  constexpr int TR = 128, TC = 64;
  __shared__ float tile[TR][TC + 1];
  const int r0 = blockIdx.y * TR, c0 = blockIdx.x * TC;
  const int tid = threadIdx.x;
#pragma unroll
  for (int u = 0; u < TR * TC / 4 / 256; ++u) {
    const int e = u * 256 + tid;
    const int rr = e / 16, cc = (e % 16) * 4;
    const int r = r0 + rr, c = c0 + cc;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
    if (r < rows) {
      const int64_t o = (int64_t)r * ld + c;
      if (vec && c + 3 < cols) {
        if constexpr (std::is_same<SRC, float>::value) {
          const f32x4 x = *(const f32x4*)(S1 + o);
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = x[t];
        } else {
          const bf16x4 x = *(const bf16x4*)(S1 + o);
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = (float)x[t];
        }
        if (S2) {
          const f32x4 y = *(const f32x4*)(S2 + o);
#pragma unroll
          for (int t = 0; t < 4; ++t) v[t] = fmaf(s2, y[t], v[t]);
        }
      } else {
#pragma unroll
        for (int t = 0; t < 4; ++t)
          if (c + t < cols) {
            v[t] = (float)S1[o + t];
            if (S2) v[t] = fmaf(s2, S2[o + t], v[t]);
          }
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) tile[rr][cc + t] = v[t];
  }
  __syncthreads();
  // row c of dst: 128 consecutive r as 16 chunks of 8 bf16
#pragma unroll
  for (int u = 0; u < TR * TC / 8 / 256; ++u) {
    const int e = u * 256 + tid;
    const int cc = e / 16, rr0 = (e % 16) * 8;
    const int c = c0 + cc;
    if (c >= cols_p || r0 + rr0 >= rows_p) continue;
    bf16x8 h, l;
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float v = tile[rr0 + t][cc];
      h[t] = to_bf16(v);
      l[t] = to_bf16(v - (float)h[t]);
    }
    const int64_t o = (int64_t)c * rows_p + r0 + rr0;
    *(bf16x8*)(hi + o) = h;
    if (lo) *(bf16x8*)(lo + o) = l;
  }
}

// Out[i][j] (+)= sum_t sum_k A_{a(t)}[i][k] B_{b(t)}[j][k] (+ rho (E1 - E2)[i][j]).
// The operands are up to two bf16 planes per side (hi, lo), each [rows_p][Kp] with
// the contraction index contiguous and zero padding (rows_p a multiple of G_BM, Kp of
// 64), so the main loop has no bounds checks. Each K chunk loads every plane once and
// applies all term products to it: term t multiplies plane a(t) = bit t of TA with
// plane b(t) = bit t of TB. The MFMA computes the transposed tile (rows = output
// columns), so a lane owns 4 consecutive output columns and the epilogue uses 16-byte
// accesses. SYM: only tiles with tile_i <= tile_j; the diagonal tiles keep their i <= j
// half and every tile is mirrored, so the result is exactly symmetric.
//
// Two tile shapes (BgTile<T>):
//   T = 256: 8 waves of 128 x 64, two LDS stages; one 256-tile per CU fills the chip
//     for a 4096 x 4096 output (16 x 16 tiles).
//   T = 192: 8 waves, two per 96 x 96 quadrant (nine accumulators each): wave w takes
//     the first 16 k of every 32-k chunk, wave w + 4 (on the same SIMD) the second 16,
//     and the two partial tiles are summed once at the end through LDS. Three LDS
//     stages; waves 0-3 load the A planes, waves 4-7 the B planes. The symmetric
//     products use it: a 4096-wide triangle is 253 tiles of 192 (one round on 256 CUs)
//     against 136 of 256.
// A tile's K chunk goes from HBM straight into LDS (buffer_load ... lds; no staging
// registers) while earlier chunks are multiplied. Rows past a plane's end (the last
// 192-tile reaches past a 256-padded plane) read as zeros through the buffer range.
struct BGemm {
  const __bf16* A[2];  // planes of A [Ip][Kp]
  const __bf16* B[2];  // planes of B [Jp][Kp]
  int64_t ld;          // Kp
  float* Out;
  int64_t ldo;
  const float* E1;
  const float* E2;
  int64_t lde;
  float rho;
  int I, J, Kp;
  int accumulate;
  int tiles_j, ntiles;
  int vec_out;
};

constexpr int BG_KC = 32;    // contraction chunk per LDS stage
constexpr int BG_GROUP = 4;  // tile rows per group of the non-symmetric tile order
template <int T>
struct BgTile;
template <>
struct BgTile<256> {
  static constexpr int WM = 128, WN = 64, STAGES = 2, KSPLIT = 1;
};
template <>
struct BgTile<192> {
  static constexpr int WM = 96, WN = 96, STAGES = 3, KSPLIT = 2;
};
template <int T>
constexpr int bg_threads() {
  return (T / BgTile<T>::WM) * (T / BgTile<T>::WN) * BgTile<T>::KSPLIT * 64;
}

template <int T, int NA, int NB, int NT, int TA, int TB, bool SYM>
__global__ __launch_bounds__(bg_threads<T>(), 1) void bgemm_kernel(BGemm p) {
  constexpr int WM = BgTile<T>::WM, WN = BgTile<T>::WN, S = BgTile<T>::STAGES;
  constexpr int KSP = BgTile<T>::KSPLIT;
  constexpr int NTH = bg_threads<T>();
  constexpr int ROWS = (NA + NB) * T;              // stacked plane rows per stage
  // KSP = 1: all threads load every plane; KSP = 2: threads [0, NTH/2) the A planes,
  // [NTH/2, NTH) the B planes
  constexpr int LTH = KSP == 1 ? NTH : NTH / 2;    // threads loading one plane
  constexpr int RPU = LTH / 4;                     // rows per load round (4 chunks per row)
  constexpr int PPR = T / RPU;                     // load rounds per plane
  constexpr int LPT = ROWS * (BG_KC / 8) / NTH;    // 16-byte loads per thread per stage
  constexpr int MA = WM / 32, MB = WN / 32;
  static_assert(KSP == 1 || (KSP == 2 && NA == NB), "split loads: as many A as B planes");
  static_assert(T % RPU == 0 && LPT == PPR * (KSP == 1 ? NA + NB : NA), "whole load rounds per plane");
  static_assert(BG_KC == 32 && (KSP == 1 || KSP == 2), "one or two 16-k halves per chunk");
  static_assert(WM % 16 == 0 && WN % 16 == 0 && T % 16 == 0, "fragment rows aligned to the swizzle");
  __shared__ __attribute__((aligned(16))) __bf16 lds[S][ROWS * BG_KC];
  int ti, tj;
  {
    const int t = xcd_item((p.ntiles + kXcds - 1) / kXcds);
    if (t >= p.ntiles) return;
    if constexpr (SYM) {
      int r = 0, rem = t;
      while (rem >= p.tiles_j - r) {
        rem -= p.tiles_j - r;
        ++r;
      }
      ti = r;
      tj = r + rem;
    } else {
      // groups of BG_GROUP tile rows, column by column inside a group: the run of items
      // one XCD takes covers few tile rows and few tile columns, so its L2 serves more
      // of the operand re-reads
      const int tiles_i = p.ntiles / p.tiles_j;
      const int per_group = BG_GROUP * p.tiles_j;
      const int first = (t / per_group) * BG_GROUP;
      const int rows = min(BG_GROUP, tiles_i - first);
      const int r = t % per_group;
      ti = first + r % rows;
      tj = r / rows;
    }
  }
  const int i0 = ti * T, j0 = tj * T;
  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int h32 = lane >> 5, l32 = lane & 31;
  constexpr int NQW = (T / WM) * (T / WN);  // waves per k half
  const int wq = wid % NQW, kh = wid / NQW;  // output block, k half (KSP = 2)
  const int wi = (wq / (T / WN)) * WM, wj = (wq % (T / WN)) * WN;
  const int nq = p.Kp / BG_KC;

  f32x16 acc[MA][MB];
#pragma unroll
  for (int a = 0; a < MA; ++a)
#pragma unroll
    for (int b = 0; b < MB; ++b) acc[a][b] = f32x16{};

  // Stages of unpadded [stacked row][32 k] tiles. LDS position c of a stage (16 bytes)
  // holds stacked row c / 4, k chunk (c % 4) ^ ((row / 4) % 4): the 16 consecutive rows
  // an MFMA fragment read takes at one k chunk land in 16 different bank groups. Load u
  // (u < LPT) of thread tid fills row (u % PPR) * RPU + lt / 4 of plane u / PPR (KSP =
  // 1; lt = tid) or of plane (tid < NTH/2 ? 0 : NA) + u / PPR (KSP = 2; lt = tid % (NTH/2)).
  // buffer descriptors of the planes' rows of this tile (unused ones repeat plane 0;
  // plain variables: the host pass drops the kernel if a descriptor is a temporary);
  // the planes hold pad(I) and pad(J) rows, pad = G_BM
  const int ip = (p.I + G_BM - 1) / G_BM * G_BM, jp = (p.J + G_BM - 1) / G_BM * G_BM;
  auto plane_base = [&](int pl) {
    return pl < NA ? p.A[pl] + (int64_t)i0 * p.ld : p.B[pl - NA] + (int64_t)j0 * p.ld;
  };
  auto plane_bytes = [&](int pl) {
    return (uint32_t)(min(T, pl < NA ? ip - i0 : jp - j0) * p.ld * 2);
  };
  const __amdgpu_buffer_rsrc_t rs0 =
      __builtin_amdgcn_make_buffer_rsrc((void*)plane_base(0), 0, plane_bytes(0), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs1 = __builtin_amdgcn_make_buffer_rsrc(
      (void*)plane_base(NA + NB > 1 ? 1 : 0), 0, plane_bytes(NA + NB > 1 ? 1 : 0), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs2 = __builtin_amdgcn_make_buffer_rsrc(
      (void*)plane_base(NA + NB > 2 ? 2 : 0), 0, plane_bytes(NA + NB > 2 ? 2 : 0), 0x00020000);
  const __amdgpu_buffer_rsrc_t rs3 = __builtin_amdgcn_make_buffer_rsrc(
      (void*)plane_base(NA + NB > 3 ? 3 : 0), 0, plane_bytes(NA + NB > 3 ? 3 : 0), 0x00020000);
  static_assert(NA + NB <= 4, "at most four planes");
  const int lt = tid % LTH, lw = lt / 64;  // thread and wave within the loading group
  const uint32_t voff0 = (uint32_t)(((lt / 4) * p.ld + (((lt % 4) ^ ((lt / 16) % 4)) * 8)) * 2);
  auto issue = [&](int q, int buf) {
    const uint32_t k0b = (uint32_t)(q * BG_KC * 2);
    static_for<LPT>([&](auto u_t) {
      constexpr int u = decltype(u_t)::value;
      const uint32_t vo = voff0 + (uint32_t)((u % PPR) * RPU * p.ld * 2);
      if constexpr (KSP == 1) {
        constexpr int pl = u / PPR;
        PKV_LDS void* dst = (PKV_LDS void*)&lds[buf][(u * NTH + wid * 64) * 8];
        if constexpr (pl == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs0, dst, 16, vo, k0b, 0, 0);
        else if constexpr (pl == 1) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs1, dst, 16, vo, k0b, 0, 0);
        else if constexpr (pl == 2) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs2, dst, 16, vo, k0b, 0, 0);
        else __builtin_amdgcn_raw_ptr_buffer_load_lds(rs3, dst, 16, vo, k0b, 0, 0);
      } else {
        // a wave's 64 lanes fill 16 rows (1 KB) of one plane; which plane is wave-uniform
        constexpr int pu = u / PPR;  // plane within the side (hi or lo)
        const int row = (u % PPR) * RPU + lw * 16;
        if (__builtin_amdgcn_readfirstlane(wid) < NTH / 128) {
          PKV_LDS void* dst = (PKV_LDS void*)&lds[buf][(pu * T + row) * BG_KC];
          if constexpr (pu == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs0, dst, 16, vo, k0b, 0, 0);
          else __builtin_amdgcn_raw_ptr_buffer_load_lds(rs1, dst, 16, vo, k0b, 0, 0);
        } else {
          PKV_LDS void* dst = (PKV_LDS void*)&lds[buf][((NA + pu) * T + row) * BG_KC];
          if constexpr (pu == 0) __builtin_amdgcn_raw_ptr_buffer_load_lds(rs2, dst, 16, vo, k0b, 0, 0);
          else __builtin_amdgcn_raw_ptr_buffer_load_lds(rs3, dst, 16, vo, k0b, 0, 0);
        }
      }
    });
  };
  // at most N of this wave's loads still in flight (the chunks issued after the one
  // needed next), then a plain barrier (the workgroup fence of __syncthreads adds
  // nothing here)
  auto landed = [&](auto n_t) {
    constexpr int N = decltype(n_t)::value;
    asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
  };
  const int sw = (l32 / 4) % 4;

  // chunk q in stage q % S; S - 1 chunks in flight ahead of the one multiplied
#pragma unroll
  for (int q = 0; q < S - 1; ++q)
    if (q < nq) issue(q, q);
  if (S == 3 && nq > 1) landed(std::integral_constant<int, LPT>{});
  else landed(std::integral_constant<int, 0>{});
  for (int q = 0; q < nq; ++q) {
    const int buf = q % S;
    // the stage of chunk q + S - 1 was last read in step q - 1 (a barrier ago)
    if (q + S - 1 < nq) issue(q + S - 1, (q + S - 1) % S);
    const __bf16* L0 = lds[buf];
#pragma unroll
    for (int kk = 0; kk < BG_KC / KSP; kk += 16) {
      const int ks = KSP == 1 ? kk : 16 * kh;
      const int ch = ((2 * (ks / 16) + h32) ^ sw) * 8;  // k chunk of this lane, swizzled
      bf16x8 fa[NA][MA], fb[NB][MB];
#pragma unroll
      for (int pa = 0; pa < NA; ++pa)
#pragma unroll
        for (int a = 0; a < MA; ++a)
          fa[pa][a] = *(const bf16x8*)(L0 + (pa * T + wi + 32 * a + l32) * BG_KC + ch);
#pragma unroll
      for (int pb = 0; pb < NB; ++pb)
#pragma unroll
        for (int b = 0; b < MB; ++b)
          fb[pb][b] = *(const bf16x8*)(L0 + ((NA + pb) * T + wj + 32 * b + l32) * BG_KC + ch);
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int a = 0; a < MA; ++a)
#pragma unroll
          for (int b = 0; b < MB; ++b)
            acc[a][b] = mfma32(fb[(TB >> t) & 1][b], fa[(TA >> t) & 1][a], acc[a][b]);
    }
    // chunk q + 1 has landed (with three stages, chunk q + 2 may still be in flight)
    if (S == 3 && q + 2 < nq) landed(std::integral_constant<int, LPT>{});
    else landed(std::integral_constant<int, 0>{});
  }
  // KSP = 2: the second k half's partial tile goes through the (now idle) stages,
  // lane-major per register (a wave's 64 lanes write and read 256 consecutive bytes),
  // and is added in the epilogue, four values at a time
  static_assert(KSP == 1 || NQW * MA * MB * 16 * 64 * 4 <= (int)sizeof(lds), "partial tiles fit the stages");
  const float* part = (const float*)&lds[0][0] + wq * (MA * MB * 16 * 64);
  if constexpr (KSP == 2) {
    if (kh == 1) {
      float* pw = (float*)&lds[0][0] + wq * (MA * MB * 16 * 64);
#pragma unroll
      for (int a = 0; a < MA; ++a)
#pragma unroll
        for (int b = 0; b < MB; ++b)
#pragma unroll
          for (int e = 0; e < 16; ++e) pw[((a * MB + b) * 16 + e) * 64 + lane] = acc[a][b][e];
    }
    __syncthreads();
    if (kh == 1) return;
  }

  // lane owns Out[i0+wi+32a+l32][j0+wj+32b+8g+4h32 .. +3]
#pragma unroll
  for (int a = 0; a < MA; ++a)
#pragma unroll
    for (int b = 0; b < MB; ++b)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int i = i0 + wi + 32 * a + l32, j = j0 + wj + 32 * b + 8 * g + 4 * h32;
        if (i >= p.I || j >= p.J) continue;
        f32x4 v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[a][b][4 * g + e];
        if constexpr (KSP == 2) {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[e] += part[((a * MB + b) * 16 + 4 * g + e) * 64 + lane];
        }
        if (p.E1) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (j + e < p.J)
              v[e] += p.rho * (p.E1[(int64_t)i * p.lde + j + e] -
                               (p.E2 ? p.E2[(int64_t)i * p.lde + j + e] : 0.f));
        }
        float* o = p.Out + (int64_t)i * p.ldo + j;
        const bool diag = SYM && ti == tj;
        if (p.vec_out && j + 3 < p.J && !diag) {
          // v stays this call's contribution: the mirror below adds it again
          *(f32x4*)o = p.accumulate ? v + *(const f32x4*)o : v;
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (j + e < p.J && !(diag && i > j + e)) o[e] = p.accumulate ? o[e] + v[e] : v[e];
        }
        if constexpr (SYM) {
          // mirror to (j + e, i): the 32 lanes of a half write 32 consecutive floats
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int jj = j + e;
            if (jj >= p.J || i >= jj) continue;
            float* o2 = p.Out + (int64_t)jj * p.ldo + i;
            *o2 = p.accumulate ? *o2 + v[e] : v[e];
          }
        }
      }
}

// symmetric products on 192-tiles, the others on 256-tiles
template <int NA, int NB, int NT, int TA, int TB, bool SYM>
hipError_t run_bgemm(BGemm p, hipStream_t st) {
  constexpr int T = SYM ? 192 : 256;
  p.tiles_j = (int)((p.J + T - 1) / T);
  p.ntiles = SYM ? p.tiles_j * (p.tiles_j + 1) / 2 : (int)((p.I + T - 1) / T) * p.tiles_j;
  p.vec_out = (p.ldo & 3) == 0 && ((uintptr_t)p.Out & 15) == 0;
  const dim3 grid((p.ntiles + kXcds - 1) / kXcds * kXcds), block(bg_threads<T>());
  hipLaunchKernelGGL((bgemm_kernel<T, NA, NB, NT, TA, TB, SYM>), grid, block, 0, st, p);
  return hipGetLastError();
}

hipError_t run_split_rows(const float* S1, const float* S2, int64_t rows, int64_t cols, int64_t ld,
                          __bf16* hi, __bf16* lo, int64_t rows_p, int64_t cols_p, hipStream_t st) {
  const int64_t n = rows_p * (cols_p / 8);
  hipLaunchKernelGGL(split_rows_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, S1, S2,
                     (int)rows, (int)cols, ld, hi, lo, (int)rows_p, (int)cols_p);
  return hipGetLastError();
}

template <class SRC>
hipError_t run_split_transpose(const SRC* S1, const float* S2, int64_t rows, int64_t cols,
                               int64_t ld, __bf16* hi, __bf16* lo, int64_t rows_p, int64_t cols_p,
                               hipStream_t st, float s2 = -1.f) {
  // rows_p is a multiple of 8 (every caller pads it to 64): whole 16-byte chunks
  const dim3 grid((unsigned)((cols_p + 63) / 64), (unsigned)((rows_p + 127) / 128));
  const int vec = ld % 4 == 0 && (uintptr_t)S1 % (4 * sizeof(SRC)) == 0 &&
                  (S2 == nullptr || (uintptr_t)S2 % 16 == 0);
  hipLaunchKernelGGL((split_transpose_kernel<SRC>), grid, dim3(256), 0, st, S1, S2, s2, (int)rows,
                     (int)cols, ld, hi, lo, (int)rows_p, (int)cols_p, vec);
  return hipGetLastError();
}

// u = z / sqrt(mean(z^2) + eps) per row, split into hi and lo planes [rows_p][cols_p]
// (zero outside rows x cols). One workgroup per row; the mean square in fp32.
__global__ __launch_bounds__(256) void rmsnorm_split_kernel(const float* __restrict__ Z, int rows,
                                                            int cols, float eps,
                                                            __bf16* __restrict__ hi,
                                                            __bf16* __restrict__ lo, int cols_p) {
  __shared__ float part[8];
  const int r = blockIdx.x, tid = threadIdx.x;
  float inv = 0.f;
  if (r < rows) {
    const float* z = Z + (int64_t)r * cols;
    float ss = 0.f;
    for (int c = tid; c < cols; c += 256) ss = fmaf(z[c], z[c], ss);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) ss += __shfl_xor(ss, o);
    if ((tid & 63) == 0) part[tid >> 6] = ss;
    __syncthreads();
    if (tid == 0) part[4] = 1.0f / sqrtf((part[0] + part[1] + part[2] + part[3]) / (float)cols + eps);
    __syncthreads();
    inv = part[4];
  }
  for (int c0 = tid * 8; c0 < cols_p; c0 += 256 * 8) {
    bf16x8 h, l;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int c = c0 + e;
      const float v = (r < rows && c < cols) ? Z[(int64_t)r * cols + c] * inv : 0.f;
      h[e] = to_bf16(v);
      l[e] = to_bf16(v - (float)h[e]);
    }
    *(bf16x8*)(hi + (int64_t)r * cols_p + c0) = h;
    *(bf16x8*)(lo + (int64_t)r * cols_p + c0) = l;
  }
}

// H[m][j] = silu(GU[m][j]) * GU[m][up + j], silu(g) = g / (1 + e^-g), for j < d_ff.
__global__ __launch_bounds__(256) void swiglu_kernel(const float* __restrict__ GU, int64_t ldgu,
                                                     int64_t up, int rows, int d_ff,
                                                     float* __restrict__ H) {
  const int64_t g = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int per_row = d_ff / 4;
  if (g >= (int64_t)rows * per_row) return;
  const int r = (int)(g / per_row), j = (int)(g % per_row) * 4;
  const f32x4 a = *(const f32x4*)(GU + (int64_t)r * ldgu + j);
  const f32x4 b = *(const f32x4*)(GU + (int64_t)r * ldgu + up + j);
  f32x4 h;
#pragma unroll
  for (int e = 0; e < 4; ++e) h[e] = a[e] / (1.0f + expf(-a[e])) * b[e];
  *(f32x4*)(H + (int64_t)r * d_ff + j) = h;
}

struct TargetsWs {
  size_t Dh, Dl, Wh, Wl, total;
};
TargetsWs targets_layout(int64_t M, int64_t din, int64_t dout) {
  const int64_t Mp = pad_to(M, G_BM), Kp = pad_to(din, G_KC), Jp = pad_to(dout, G_BM);
  TargetsWs L{};
  size_t o = 0;
  L.Dh = o; o += align_up((size_t)Mp * Kp * 2);
  L.Dl = o; o += align_up((size_t)Mp * Kp * 2);
  L.Wh = o; o += align_up((size_t)Jp * Kp * 2);
  L.Wl = o; o += align_up((size_t)Jp * Kp * 2);
  L.total = o;
  return L;
}
struct NormalEqWs {
  size_t Xh, Xl, Yh, Yl, total;
};
NormalEqWs normal_eq_layout(int64_t rows, int64_t din, int64_t dout) {
  const int64_t Kp = pad_to(rows, G_KC), Ip = pad_to(din, G_BM), Jp = pad_to(dout, G_BM);
  NormalEqWs L{};
  size_t o = 0;
  L.Xh = o; o += align_up((size_t)Ip * Kp * 2);
  L.Xl = o; o += align_up((size_t)Ip * Kp * 2);
  L.Yh = o; o += align_up((size_t)Jp * Kp * 2);
  L.Yl = o; o += align_up((size_t)Jp * Kp * 2);
  L.total = o;
  return L;
}

struct MlpWs {
  size_t Uh, Ul, Wh, Wl, GU, total;
  int64_t Mp, Kp, Jh;  // padded rows, padded d, padded d_ff (one half of the gate|up planes)
};
MlpWs mlp_layout(int64_t M, int64_t d, int64_t d_ff) {
  MlpWs L{};
  L.Mp = pad_to(M, G_BM);
  L.Kp = pad_to(d, G_KC);
  L.Jh = pad_to(d_ff, G_BM);
  size_t o = 0;
  L.Uh = o; o += align_up((size_t)L.Mp * L.Kp * 2);
  L.Ul = o; o += align_up((size_t)L.Mp * L.Kp * 2);
  L.Wh = o; o += align_up((size_t)2 * L.Jh * L.Kp * 2);
  L.Wl = o; o += align_up((size_t)2 * L.Jh * L.Kp * 2);
  L.GU = o; o += align_up((size_t)M * 2 * L.Jh * 4);
  L.total = o;
  return L;
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

}  // namespace

size_t targets_ws_bytes(int64_t M, int64_t din, int64_t dout) {
  return targets_layout(M, din, dout).total;
}
size_t mlp_features_ws_bytes(int64_t M, int64_t d, int64_t d_ff) {
  return mlp_layout(M, d, d_ff).total;
}

hipError_t launch_mlp_features(const float* Z, const void* Wg, const void* Wu, bool w_bf16,
                               int64_t M, int64_t d, int64_t d_ff, float eps, float* H, void* ws,
                               hipStream_t st) {
  const MlpWs L = mlp_layout(M, d, d_ff);
  char* w = (char*)ws;
  __bf16 *Uh = (__bf16*)(w + L.Uh), *Ul = (__bf16*)(w + L.Ul);
  __bf16 *Wh = (__bf16*)(w + L.Wh), *Wl = (__bf16*)(w + L.Wl);
  float* GU = (float*)(w + L.GU);
  hipLaunchKernelGGL(rmsnorm_split_kernel, dim3((unsigned)L.Mp), dim3(256), 0, st, Z, (int)M, (int)d,
                     eps, Uh, Ul, (int)L.Kp);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  // [Wg | Wu] transposed: rows [0, d_ff) gate, rows [Jh, Jh + d_ff) up
  const int64_t off = L.Jh * L.Kp;
  for (int h = 0; h < 2; ++h) {
    const void* Wx = h ? Wu : Wg;
    if (w_bf16)
      e = run_split_transpose((const __bf16*)Wx, nullptr, d, d_ff, d_ff, Wh + h * off, nullptr, L.Kp,
                              L.Jh, st);
    else
      e = run_split_transpose((const float*)Wx, nullptr, d, d_ff, d_ff, Wh + h * off,
                              Wl + h * off, L.Kp, L.Jh, st);
    if (e != hipSuccess) return e;
  }
  BGemm p{};
  p.ld = L.Kp;
  p.Out = GU;
  p.ldo = 2 * L.Jh;
  p.I = (int)M;
  p.J = (int)(2 * L.Jh);
  p.Kp = (int)L.Kp;
  p.A[0] = Uh; p.A[1] = Ul;
  p.B[0] = Wh; p.B[1] = Wl;
  e = w_bf16 ? run_bgemm<2, 1, 2, 0b10, 0b00, false>(p, st)
             : run_bgemm<2, 2, 3, 0b010, 0b100, false>(p, st);
  if (e != hipSuccess) return e;
  const int64_t n = M * (d_ff / 4);
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, GU, 2 * L.Jh,
                     L.Jh, (int)M, (int)d_ff, H);
  return hipGetLastError();
}

size_t propagate_ws_bytes(int64_t M, int64_t d_ff, int64_t d) {
  return targets_layout(M, d_ff, d).total;
}

hipError_t launch_propagate(const float* Hc, const void* W, bool w_bf16, const float* dW,
                            const float* Zc, int64_t M, int64_t d_ff, int64_t d, float* Y, void* ws,
                            hipStream_t st) {
  const TargetsWs L = targets_layout(M, d_ff, d);
  const int64_t Mp = pad_to(M, G_BM), Kp = pad_to(d_ff, G_KC), Jp = pad_to(d, G_BM);
  char* w = (char*)ws;
  __bf16 *Hh = (__bf16*)(w + L.Dh), *Hl = (__bf16*)(w + L.Dl);
  __bf16 *Wh = (__bf16*)(w + L.Wh), *Wl = (__bf16*)(w + L.Wl);
  hipError_t e = run_split_rows(Hc, nullptr, M, d_ff, d_ff, Hh, Hl, Mp, Kp, st);
  if (e != hipSuccess) return e;
  // (W + dW) [d_ff][d] -> transposed [d][d_ff], split
  if (w_bf16)
    e = run_split_transpose((const __bf16*)W, dW, d_ff, d, d, Wh, Wl, Kp, Jp, st, 1.f);
  else
    e = run_split_transpose((const float*)W, dW, d_ff, d, d, Wh, Wl, Kp, Jp, st, 1.f);
  if (e != hipSuccess) return e;
  BGemm p{};  // Y = Hc (W + dW) + Zc: terms (0,0) (0,1) (1,0)
  p.ld = Kp;
  p.Out = Y;
  p.ldo = d;
  p.E1 = Zc;
  p.lde = d;
  p.rho = 1.f;
  p.I = (int)M;
  p.J = (int)d;
  p.Kp = (int)Kp;
  p.A[0] = Hh; p.A[1] = Hl;
  p.B[0] = Wh; p.B[1] = Wl;
  return run_bgemm<2, 2, 3, 0b100, 0b010, false>(p, st);
}
size_t normal_eq_ws_bytes(int64_t rows, int64_t din, int64_t dout) {
  return normal_eq_layout(rows, din, dout).total;
}

// ---------------------------------------------------------------- dual-form statistics
//
// For the ridge patch through the push-through identity (few rows, wide d_in):
// K = X X^T over the rows, and dW = X^T Y. Both sum all four hi/lo term pairs (the
// split of both operands loses only the lo x lo cross term otherwise; X^T Y's result
// can be much smaller than |X||Y| when the ridge is small, so it keeps every term).
struct DualWs {
  size_t Ah, Al, Bh, Bl, total;
};
DualWs dual_layout(int64_t rows, int64_t din, int64_t dout) {
  // K: planes of X [rows_p][din_p] (contraction d_in); X^T Y: planes of X^T and Y^T
  // [*][rows_p] (contraction rows)
  const int64_t rK = pad_to(rows, G_BM), cK = pad_to(din, G_KC);
  const int64_t kY = pad_to(rows, G_KC), iY = pad_to(din, G_BM), jY = pad_to(dout, G_BM);
  const size_t a = std::max((size_t)rK * cK, (size_t)iY * kY) * 2;
  const size_t b = (size_t)jY * kY * 2;
  DualWs L{};
  size_t o = 0;
  L.Ah = o; o += align_up(a);
  L.Al = o; o += align_up(a);
  L.Bh = o; o += align_up(b);
  L.Bl = o; o += align_up(b);
  L.total = o;
  return L;
}

hipError_t launch_gram_rows(const float* X, int64_t rows, int64_t din, float* K, void* ws,
                            hipStream_t st) {
  const DualWs L = dual_layout(rows, din, 1);
  const int64_t rK = pad_to(rows, G_BM), cK = pad_to(din, G_KC);
  char* w = (char*)ws;
  __bf16 *Xh = (__bf16*)(w + L.Ah), *Xl = (__bf16*)(w + L.Al);
  hipError_t e = run_split_rows(X, nullptr, rows, din, din, Xh, Xl, rK, cK, st);
  if (e != hipSuccess) return e;
  BGemm g{};
  g.ld = cK;
  g.Out = K;
  g.ldo = rows;
  g.I = (int)rows;
  g.J = (int)rows;
  g.Kp = (int)cK;
  g.A[0] = Xh; g.A[1] = Xl;
  g.B[0] = Xh; g.B[1] = Xl;
  return run_bgemm<2, 2, 4, 0b1100, 0b1010, true>(g, st);
}

hipError_t launch_xt_y(const float* X, const float* Y, int64_t rows, int64_t din, int64_t dout,
                       float* Out, void* ws, hipStream_t st) {
  const DualWs L = dual_layout(rows, din, dout);
  const int64_t kY = pad_to(rows, G_KC), iY = pad_to(din, G_BM), jY = pad_to(dout, G_BM);
  char* w = (char*)ws;
  __bf16 *Xh = (__bf16*)(w + L.Ah), *Xl = (__bf16*)(w + L.Al);
  __bf16 *Yh = (__bf16*)(w + L.Bh), *Yl = (__bf16*)(w + L.Bl);
  // X [rows][din] -> X^T [din][rows]; Y [rows][dout] -> Y^T [dout][rows]
  hipError_t e = run_split_transpose(X, (const float*)nullptr, rows, din, din, Xh, Xl, kY, iY, st);
  if (e != hipSuccess) return e;
  e = run_split_transpose(Y, (const float*)nullptr, rows, dout, dout, Yh, Yl, kY, jY, st);
  if (e != hipSuccess) return e;
  BGemm p{};
  p.ld = kY;
  p.Out = Out;
  p.ldo = dout;
  p.I = (int)din;
  p.J = (int)dout;
  p.Kp = (int)kY;
  p.A[0] = Xh; p.A[1] = Xl;
  p.B[0] = Yh; p.B[1] = Yl;
  return run_bgemm<2, 2, 4, 0b1100, 0b1010, false>(p, st);
}

size_t dual_stats_ws_bytes(int64_t rows, int64_t din, int64_t dout) {
  return dual_layout(rows, din, dout).total;
}

hipError_t launch_targets(const float* Of, const float* Oc, const void* W, bool w_bf16, int64_t M,
                          int64_t din, int64_t dout, int rho, float* T, void* ws, hipStream_t st,
                          const float* Zf, const float* Zc) {
  const TargetsWs L = targets_layout(M, din, dout);
  const int64_t Mp = pad_to(M, G_BM), Kp = pad_to(din, G_KC), Jp = pad_to(dout, G_BM);
  char* w = (char*)ws;
  __bf16 *Dh = (__bf16*)(w + L.Dh), *Dl = (__bf16*)(w + L.Dl);
  __bf16 *Wh = (__bf16*)(w + L.Wh), *Wl = (__bf16*)(w + L.Wl);
  hipError_t e = run_split_rows(Of, Oc, M, din, din, Dh, Dl, Mp, Kp, st);
  if (e != hipSuccess) return e;
  // W [din][dout] -> W^T [dout][din] (rows j, contraction k contiguous)
  if (w_bf16)
    e = run_split_transpose((const __bf16*)W, nullptr, din, dout, dout, Wh, nullptr, Kp, Jp, st);
  else
    e = run_split_transpose((const float*)W, nullptr, din, dout, dout, Wh, Wl, Kp, Jp, st);
  if (e != hipSuccess) return e;
  BGemm p{};
  p.ld = Kp;
  p.Out = T;
  p.ldo = dout;
  if (Zf) {  // residual pair of its own (width dout)
    p.E1 = Zf;
    p.E2 = Zc;
    p.lde = dout;
    p.rho = 1.f;
  } else if (rho) {
    p.E1 = Of;
    p.E2 = Oc;
    p.lde = din;
    p.rho = (float)rho;
  }
  p.I = (int)M;
  p.J = (int)dout;
  p.Kp = (int)Kp;
  p.A[0] = Dh; p.A[1] = Dl;
  p.B[0] = Wh; p.B[1] = Wl;
  // terms (a, b): bf16 W (0,0) (1,0); fp32 W (0,0) (1,0) (0,1)
  if (w_bf16) return run_bgemm<2, 1, 2, 0b10, 0b00, false>(p, st);
  return run_bgemm<2, 2, 3, 0b010, 0b100, false>(p, st);
}

hipError_t launch_normal_eq_f32(const float* X, const float* Yf, const float* Yc, int64_t rows,
                                int64_t din, int64_t dout, bool accumulate, float* G, float* C,
                                void* ws, hipStream_t st) {
  const NormalEqWs L = normal_eq_layout(rows, din, dout);
  const int64_t Kp = pad_to(rows, G_KC), Ip = pad_to(din, G_BM), Jp = pad_to(dout, G_BM);
  char* w = (char*)ws;
  __bf16 *Xh = (__bf16*)(w + L.Xh), *Xl = (__bf16*)(w + L.Xl);
  __bf16 *Yh = (__bf16*)(w + L.Yh), *Yl = (__bf16*)(w + L.Yl);
  // X [rows][din] -> X^T [din][rows]; (Yf - Yc) [rows][dout] -> [dout][rows]
  hipError_t e = run_split_transpose(X, (const float*)nullptr, rows, din, din, Xh, Xl, Kp, Ip, st);
  if (e != hipSuccess) return e;
  e = run_split_transpose(Yf, Yc, rows, dout, dout, Yh, Yl, Kp, Jp, st);
  if (e != hipSuccess) return e;
  {  // G = X^T X: terms (0,0) (0,1) (1,0) (1,1), upper block triangle, mirrored
    BGemm g{};
    g.ld = Kp;
    g.Out = G;
    g.ldo = din;
    g.I = (int)din;
    g.J = (int)din;
    g.Kp = (int)Kp;
    g.accumulate = accumulate;
    g.A[0] = Xh; g.A[1] = Xl;
    g.B[0] = Xh; g.B[1] = Xl;
    e = run_bgemm<2, 2, 4, 0b1100, 0b1010, true>(g, st);
    if (e != hipSuccess) return e;
  }
  BGemm p{};  // C = X^T (Yf - Yc): terms (0,0) (0,1) (1,0)
  p.ld = Kp;
  p.Out = C;
  p.ldo = dout;
  p.I = (int)din;
  p.J = (int)dout;
  p.Kp = (int)Kp;
  p.accumulate = accumulate;
  p.A[0] = Xh; p.A[1] = Xl;
  p.B[0] = Yh; p.B[1] = Yl;
  return run_bgemm<2, 2, 3, 0b100, 0b010, false>(p, st);
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
