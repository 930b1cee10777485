// Attention kernels (device code) shared by attention.hip (plain bf16 and f32 caches)
// and attention_mx.hip (block-scaled integer caches), and their templated launchers.
//
// Reference-query attention over a KV cache (the teacher and student forward
// passes of Alg. 1): O[m, h*dh:(h+1)*dh] = softmax(scale q_{m,h} K_g^T) V_g,
// g = floor(h / (Hq/Hkv)), every query against every cache entry.
//
// bf16 path (attn_bf16_kernel): one workgroup = 8 waves x 32 query rows of one KV
// head (two waves per SIMD, so one wave's softmax runs under the other's MFMAs).
// The query heads of a GQA group are packed into the row dimension (row r <->
// query r / G, head g*G + r % G), so one K/V tile in LDS serves all of them.
// Each wave keeps its rows of Q in registers and computes S^T = K Q^T on bf16 MFMA
// 32x32x16 (keys along the MFMA rows, queries along its columns), so a lane owns
// one query and softmax statistics need only one cross-lane exchange (lane l with
// l^32). P stays in registers and feeds O^T += V^T P^T directly. A contiguous cache's
// V tiles go to LDS as stored, in 64-byte rows of 32 channels, and each V operand is
// two transposing LDS reads (ds_read_b64_tr_b16) over four consecutive rows (a chunk's
// own entries likewise). Gathered, block-scaled and biased caches are first rewritten by
// vt_kernel into 32-key tiles of V^T whose key order matches the P fragments' k-slots,
// so there the V operand is one 16-byte LDS read. The online softmax runs in
// fp32 in the exp2 domain with a fixed per-row offset (fast path) and falls back
// to a lazily rescaled pass for work items whose scores outgrow it. On the main
// path K and V (or V^T) tiles go from HBM straight into eight LDS slots (buffer_load ... lds, no
// register staging; issued by waves 0-3 only), six tiles ahead, with XOR-swizzled
// 16-byte chunks in place of row padding and one barrier per two tiles (also with a
// two-term P; block-scaled and gathered keys come through registers into the same
// slots, V^T by DMA); the biased variants and the fixup stage through registers into
// four padded slots. The workgroup -> work-item
// map keeps all row tiles of one KV head (and key range) on one XCD so its L2
// serves the K/V re-reads.
//
// f32 path (attn_f32_kernel): exact fp32 products on MFMA 32x32x2 f32 (32 rows per
// wave, as in the bf16 kernel), K/V tiles in their natural layout in LDS, online
// softmax with expf and rescaling whenever a row's maximum grows.
//
// Both paths can split the cache into key ranges (more workgroups for small M);
// attn_combine_kernel then merges the partial (O, m, l) triples.
//
// Per-entry logit bias (BIAS = true; an attention-matching compressed cache carries
// one per entry): bias[g][n] is added to the logit of cache entry n. The bf16 path
// stores each tile's 32 biases (divided by the softmax scale) in LDS with the K
// tile and starts the score MFMA accumulator from them, so the steady-state loop
// gains four 16-byte LDS reads per tile and no VALU work.
//
// Chunked reference sets (OWN = true): the queries are one chunk's tokens, and
// token m also attends to the chunk's own entries 0..m (its causal prefix), which
// follow the cache in the key order: a work item's first key tiles are its range
// of the cache, and the work item of the last key range then takes the own
// entries' tiles, masked per query. Every range keeps at least one cache key, so
// every row of every partial result has a finite maximum.
//
// Block-scaled integer caches (KQ = 8 or 4; App. C, quantized KV caches): K and V
// hold int8 (or packed int4) values with one power-of-two exponent per 32 channels.
// Register loads fetch the stored K bytes and expand each 8-channel chunk to bf16 when
// the tile is stored to LDS; vt_kernel expands V on its way into the V^T tiles. The
// expansion is exact, so the arithmetic after it is that of a bf16 cache.
#pragma once

#include <math.h>

#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace pkv {

struct AttnParams {
  const void* Q;
  const void* K;
  const void* V;
  const __bf16* Vt;  // bf16 path: V transposed into 32-key tiles (see vt_kernel)
  int vt_tiles;      // tiles per KV head in Vt
  const int32_t* idx;
  int idx_stride;         // 0: one index set for every KV head; else head g's set is idx + g * idx_stride
  const int32_t* counts;  // per-head entry counts [Hkv] (clamped into [1, Nk]) or null: Nk for every head
  float* O;
  float* Opart;
  float* ML;
  int* flags;  // bf16 path: per work item, 1 = the fast path left it to the fixup
  int Hq, G;
  int64_t src_rows;
  int src_valid;
  int Nk;
  int n_split, keys_per_split;
  int rows;
  int row_tiles;
  int total_items, per_xcd;
  float c;  // bf16: scale * log2(e); f32: scale
  // own entries of a reference chunk (OWN kernels): Ks, Vs [Hkv][Ms][dh]; Vts their
  // V^T tiles (bf16)
  const void* Ks;
  const void* Vs;
  const __bf16* Vts;
  int Ms, own_tiles;
  // per-entry logit bias [Hkv][Nk] (BIAS kernels; natural-log units) and the factor
  // that puts it in the units of the raw score q.k (bf16: 1 / scale; f32: 1)
  const float* bias;
  float bias_mul;
  // block-scaled integer K / V (KQ kernels): one int8 exponent per 32 channels of a row,
  // [Hkv][src_rows][dh / 32]; K and V then hold the int8 (or packed int4) values
  const int8_t* Ke;
  const int8_t* Ve;
};

namespace {

constexpr float kTau = 8.0f;   // lazy-rescale threshold of the fixup path (log2 units)
constexpr float kBigSum = 0x1p64f;  // fast path: largest trusted partial row sum (2^kBig, kBig = 64)

// A partial row sum the fast path cannot trust: above kBigSum, infinite or NaN (an
// overflowing weight gives inf, and inf - inf = NaN in a two-term P's low piece). The
// test is on the bit pattern: these kernels are built without NaN semantics, and a
// floating-point !(l <= kBigSum) compiled to kBigSum < l, which NaN passes. Sums are
// non-negative, so a larger pattern is a larger value, inf or NaN (a sign bit, which no
// sum has, counts as untrusted too).
__device__ __forceinline__ bool untrusted_sum(float l) {
  return __builtin_bit_cast(uint32_t, l) > __builtin_bit_cast(uint32_t, kBigSum);
}
constexpr int kKeyTile = 32;  // keys per iteration, bf16 path
constexpr int kRowsBf16 = 256;  // query rows per workgroup, bf16 path
constexpr int kRowsF32 = 256;   // query rows per workgroup, f32 path (32 per wave)
constexpr int kWgPerCu = 1;     // bf16 workgroups resident per CU (launch bound)
// bf16 path: 32-row query tiles per wave (1: eight waves of 32 rows per workgroup,
// two waves per SIMD, everything in VGPRs; 2: four waves of 64 rows, one per SIMD,
// accumulators in AGPRs) and register staging sets of the K/V tile loads
// (prefetch depth kLoadSets - 1 steps; 2 or 4).
constexpr int kQT = 1;
constexpr int kThreadsBf16 = kRowsBf16 / (32 * kQT) * 64;
constexpr int kLoadSets = 2;
constexpr int kKeyTileF32 = 32;
constexpr int kF32Waves = 8;  // f32 path: waves per workgroup (32 rows each)
// bf16 fast path without gather, bias or two-term P: K / V^T tiles are loaded straight
// into LDS (buffer_load ... lds) through kDmaSlots slots, each tile's loads issued
// kDmaAhead steps before the step that scores it, one barrier per kDmaSteps steps
constexpr bool kAttnDma = true;
constexpr int kDmaSlots = 8, kDmaAhead = 6, kDmaSteps = 2;
static_assert(kDmaAhead <= kDmaSlots - kDmaSteps && kDmaAhead >= kDmaSteps + 1,
              "a slot is refilled only after its last read");
static_assert(kDmaSlots % (2 * kDmaSteps) == 0, "whole barrier groups per unrolled pass");
// Waves 0 .. kDmaWaves-1 issue all of a tile's loads (the others only compute): with
// the loads spread over all eight waves the kernel took 5 % more cycles
constexpr int kDmaWaves = 4;
constexpr int kDmaLpdMax = 4;  // 16-byte chunks of one K (or V^T) tile per issuing lane, at most


// Eight channels of a block-scaled integer cache row as bf16, q * 2^ex: q the signed
// bytes of w0 (channels 0-3) and w1 (4-7) for KQ = 8, the signed nibbles of w0 for
// KQ = 4 (channel i in bits 4i .. 4i+3). Exact while q * 2^ex is a normal bf16 number;
// otherwise rounded to nearest even, as the conversion of the fp32 value ldexp(q, ex).
template <int KQ>
__device__ __forceinline__ bf16x8 mx_expand8(uint32_t w0, uint32_t w1, int ex) {
  static_assert(KQ == 8 || KQ == 4, "int8 or int4 values");
  bf16x8 v;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int q;
    if constexpr (KQ == 8) q = (int)((i < 4 ? w0 : w1) << (24 - 8 * (i & 3))) >> 24;
    else q = (int)(w0 << (28 - 4 * i)) >> 28;
    v[i] = (__bf16)ldexpf((float)q, ex);
  }
  return v;
}

// V -> V^T in 32-key tiles, so that the P V product reads V with plain 16-byte LDS
// reads: Vt[g][tile][d][pos] (bf16). Within a tile the keys are stored in the
// k-slot order of the P fragments: key 16b + r (r < 16) sits at position
// 16b + 8((r % 8) / 4) + 4(r / 8) + r % 4, so the 8 keys one lane feeds into an MFMA
// (keys 16b + 4h + {0..3} and 16b + 8 + 4h + {0..3}) are 8 consecutive positions.
// Keys at or past the head's entry count (and gathered rows outside the cache) are
// zero. GATHER: key n of head g is row idx[g * idx_stride + n] of V. KQ = 8 or 4: V
// holds block-scaled integers (exponents in Ve), expanded to bf16 on the way.
template <int DH, bool GATHER, int KQ>
__global__ __launch_bounds__(256) void vt_kernel(const void* __restrict__ V,
                                                 const int8_t* __restrict__ Ve,
                                                 const int32_t* __restrict__ idx, int idx_stride,
                                                 const int32_t* __restrict__ counts,
                                                 int64_t src_rows, int Nk, int ntiles,
                                                 __bf16* __restrict__ Vt) {
  constexpr int CH = DH / 8;     // 16-byte chunks per V row
  constexpr int SP = DH + 2;     // LDS pitch (elements) of the [key][d] staging tile
  __shared__ __bf16 sm[32 * SP];
  const int tile = blockIdx.x, g = blockIdx.y, tid = threadIdx.x;
  constexpr int RB = DH * (KQ ? KQ : 16) / 8;  // bytes of one stored V row
  const char* Vg = (const char*)V + (int64_t)g * src_rows * RB;
  const int nk = counts ? min(max(counts[g], 1), Nk) : Nk;
  const int32_t* ig = GATHER ? idx + (int64_t)g * idx_stride : nullptr;
  for (int c = tid; c < 32 * CH; c += 256) {
    const int key = c / CH, col = (c % CH) * 8;
    const int n = tile * 32 + key;
    bf16x8 v = {};
    if (n < nk) {
      const int64_t src = GATHER ? (int64_t)ig[n] : (int64_t)n;
      if (src >= 0 && src < src_rows) {
        const char* row = Vg + src * RB;
        if constexpr (KQ == 0) {
          v = load_bf16x8((const __bf16*)row + col);
        } else {
          const int ex = Ve[((int64_t)g * src_rows + src) * (DH / 32) + col / 32];
          if constexpr (KQ == 8) {
            const u32x2 w = *(const u32x2*)(row + col);
            v = mx_expand8<8>(w[0], w[1], ex);
          } else {
            v = mx_expand8<4>(*(const uint32_t*)(row + col / 2), 0u, ex);
          }
        }
      }
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sm[key * SP + col + e] = v[e];
  }
  __syncthreads();
  __bf16* out = Vt + ((int64_t)g * ntiles + tile) * DH * 32;
  for (int c = tid; c < DH * 4; c += 256) {
    const int d = c / 4, q = c % 4;  // positions 8q .. 8q+7 of row d
    bf16x8 v;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int key = 16 * (q / 2) + 8 * (e / 4) + 4 * (q % 2) + (e % 4);
      v[e] = sm[key * SP + d];
    }
    *(u32x4*)(out + d * 32 + 8 * q) = __builtin_bit_cast(u32x4, v);
  }
}

// SAFE = false (fast path): each row's exponent offset is fixed to the exact max of
// its first key tile, so O is never rescaled and only MFMA touches it, and the
// steady-state loop takes no row maxima at all. Every weight P a lane adds is at most
// that lane's partial row sum, so a row whose partial sums all stay at or below
// 2^kBig never met a score more than about kBig (log2 units) above its offset: P, l and O stay far from fp32
// overflow. A work item with a larger (or non-finite) partial sum in any row is
// marked in p.flags at the end and its outputs are not trusted. SAFE = true (fixup,
// launched right after on the same stream): the lazy-rescale online softmax, run
// only for marked work items, overwriting their outputs.
// KQ = 8 or 4: K holds block-scaled integers (exponents in p.Ke), loaded as such and
// expanded to bf16 when the tile is stored to LDS (through registers on either
// pipeline); V was expanded by vt_kernel into the V^T tiles.
// VNAT (contiguous bf16 cache, every row of it used; own entries, if any, as stored):
// no V^T tiles; V tiles arrive in their stored [key][d] order and the P V product reads
// its V operand with transposing LDS reads (see vfrag).
template <int DH, bool GATHER, bool PSPLIT, bool PARTIAL, bool SAFE, bool OWN, bool BIAS, int KQ,
          bool VNAT>
__global__ __launch_bounds__(kThreadsBf16, kWgPerCu) void attn_bf16_kernel(AttnParams p) {
  static_assert(!(OWN && BIAS), "own entries carry no bias");
  static_assert(KQ == 0 || KQ == 8 || KQ == 4, "bf16, int8 or int4 keys");
  static_assert(!VNAT || (!GATHER && !BIAS && KQ == 0), "V tiles of a contiguous bf16 cache");
  static_assert(!(OWN && KQ), "own entries are bf16");
  constexpr int KT = kKeyTile;
  constexpr int NKT = KT / 32;  // 32-key MFMA tiles per iteration
  constexpr int KP = DH + 8;   // K tile pitch (elements): conflict-free 16-byte row reads
  constexpr int VTP = 40;      // V^T tile pitch (elements): 32 keys + 8, conflict-free 16-byte reads
  constexpr int NS = DH / 16;  // MFMA k-steps over head_dim
  constexpr int ND = DH / 32;  // 32-wide head_dim tiles of O
  constexpr int CH = DH / 8;   // 16-byte chunks per K/V row
  constexpr int QT = kQT;        // 32-row query tiles per wave
  constexpr int NT = kThreadsBf16;
  constexpr int NCH = KT * CH;             // 16-byte chunks per K tile (= per V^T tile)
  constexpr int LPT = (NCH + NT - 1) / NT;  // chunks per thread
  // DMA: the fast path over contiguous bf16 K (one- or two-term P) streams K / V^T
  // tiles straight into LDS (no register staging), through kDmaSlots unpadded slots
  // whose 16-byte chunks are XOR-swizzled so that the MFMA operand reads stay
  // conflict-free
  constexpr bool DMA = kAttnDma && !SAFE && !BIAS;
  // K through registers on the DMA pipeline: block-scaled values, or gathered rows
  constexpr bool KREG = KQ != 0 || GATHER;
  // stored K rows: bf16, or int8 / packed int4 values (KRB bytes per row, KCB bytes per
  // 8-channel chunk) with DH / 32 exponent bytes
  constexpr int KCB = KQ ? KQ : 16;
  constexpr int KRB = CH * KCB;
  constexpr int NSL = kDmaSlots;
  __shared__ __attribute__((aligned(16))) __bf16 Ks[DMA ? 1 : 4][KT * KP];
  __shared__ __attribute__((aligned(16))) __bf16 Vs[DMA ? 1 : 4][DH * VTP];
  __shared__ __attribute__((aligned(16))) __bf16 Kd[DMA ? NSL : 1][DMA ? KT * DH : 8];
  __shared__ __attribute__((aligned(16))) __bf16 Vd[DMA ? NSL : 1][DMA ? DH * KT : 8];
  __shared__ __attribute__((aligned(16))) float Bs[BIAS ? 4 : 1][BIAS ? KT : 4];
  __shared__ int overflow;

  // work-item coordinates are workgroup-uniform; readfirstlane keeps them (and the
  // buffer descriptors and offsets built from them) in scalar registers
  const int w = __builtin_amdgcn_readfirstlane(xcd_item(p.per_xcd));
  if (w >= p.total_items) return;
  if constexpr (SAFE) {
    if (p.flags[w] == 0) return;
  }
  const int rt = __builtin_amdgcn_readfirstlane(w % p.row_tiles);
  const int t2 = __builtin_amdgcn_readfirstlane(w / p.row_tiles);
  const int split = __builtin_amdgcn_readfirstlane(t2 % p.n_split);
  const int g = __builtin_amdgcn_readfirstlane(t2 / p.n_split);
  // entries of this KV head's cache (a per-head index set may keep fewer than Nk)
  const int nk = p.counts ? __builtin_amdgcn_readfirstlane(min(max(p.counts[g], 1), p.Nk)) : p.Nk;
  const int k_begin = split * p.keys_per_split;
  const int k_end = max(k_begin, min(nk, k_begin + p.keys_per_split));
  // cache tiles [0, ct) of this key range, then (OWN, last range) the own tiles up
  // to this workgroup's last query
  // (tiles past ntiles are masked like keys past k_end, also in the other ranges)
  const int ct = (k_end - k_begin + KT - 1) / KT;
  const bool own_range = OWN && split == p.n_split - 1;
  if constexpr (PARTIAL) {
    // a key range past the end of a shorter head's cache (and without own entries):
    // an empty partial result, weight zero in the merge
    if (ct == 0 && !own_range) {
      if constexpr (!SAFE) {
        if (threadIdx.x == 0) p.flags[w] = 0;
      }
      for (int i = threadIdx.x; i < kRowsBf16; i += blockDim.x) {
        const int r = rt * kRowsBf16 + i;
        if (r >= p.rows) break;
        const int64_t rid = ((int64_t)(g * p.n_split + split)) * p.rows + r;
        f32x4* op = (f32x4*)(p.Opart + rid * DH);
#pragma unroll
        for (int c4 = 0; c4 < DH / 4; ++c4) op[c4] = f32x4{};
        p.ML[2 * rid] = -INFINITY;
        p.ML[2 * rid + 1] = 0.f;
      }
      return;
    }
  }
  int ntiles = ct;
  if (own_range) {
    const int last_q = min(p.rows - 1, rt * kRowsBf16 + kRowsBf16 - 1) / p.G;
    ntiles = ct + last_q / KT + 1;
  }

  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6;
  const int h32 = lane >> 5, l32 = lane & 31;
  const __bf16* Qb = (const __bf16*)p.Q;
  const char* Kb = (const char*)p.K + (int64_t)g * p.src_rows * KRB;
  const int row_base = rt * kRowsBf16 + wid * (32 * QT);

  bf16x8 qf[QT][NS];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const int r = min(row_base + qt * 32 + l32, p.rows - 1);
    const int m = r / p.G, j = r - m * p.G;
    const __bf16* qp = Qb + ((int64_t)m * p.Hq + g * p.G + j) * DH + h32 * 8;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[qt][s] = load_bf16x8(qp + s * 16);
  }

  // K/V are read with buffer loads whose per-lane offset carries every term (the
  // buffer range check leaves the scalar offset out), so rows past the end of this KV
  // head's buffer read as zeros (such keys are masked anyway).
  // Two register staging sets: a tile's loads are issued one step before its LDS
  // store, so their latency hides behind a whole step of MFMA work.
  const uint32_t head_bytes = (uint32_t)(p.src_rows * KRB);
  const __amdgpu_buffer_rsrc_t krs =
      __builtin_amdgcn_make_buffer_rsrc((void*)Kb, 0, head_bytes, 0x00020000);
  // V^T tiles of this KV head, or (VNAT) its V rows as stored
  const __amdgpu_buffer_rsrc_t vrs =
      VNAT ? __builtin_amdgcn_make_buffer_rsrc((void*)((const char*)p.V + (int64_t)g * p.src_rows * (DH * 2)),
                                               0, head_bytes, 0x00020000)
           : __builtin_amdgcn_make_buffer_rsrc((void*)(p.Vt + (int64_t)g * p.vt_tiles * DH * 32), 0,
                                               (uint32_t)p.vt_tiles * (DH * 32 * 2), 0x00020000);
  // A V tile in LDS (VNAT) is DH / 32 sub-tiles [dt][key][32 channels], 64-byte rows:
  // 16-byte chunk c of the stored tile (key c / CH, channels 8 (c % CH) ..) sits at
  // chunk position vnat_pos(c). The P V product's operand for channels dt * 32 + l32 and
  // the 8 keys of a P fragment (16 p2 + 4 h32 + {0..3}, then + 8) is two transposing
  // reads: in each 16-lane group, lane 4r + q points at key row r, channels 4q .. 4q + 3
  // of a 4 x 16 block, and lane j receives channel j of the block's 4 keys. A half-wave
  // reads 4 consecutive 64-byte rows (256 contiguous bytes): no bank conflicts.
  auto vnat_pos = [](int c) { return ((c % CH) / 4) * (KT * 4) + (c / CH) * 4 + c % 4; };
  const int vn_lane = (4 * h32 + ((lane & 15) >> 2)) * 32 + ((lane >> 4) & 1) * 16 + (lane & 3) * 4;
  auto vfrag = [&](const __bf16* tile, int p2, int dt) -> bf16x8 {
    const PKV_LDS __bf16* q = (const PKV_LDS __bf16*)(tile + dt * (KT * 32) + 16 * p2 * 32 + vn_lane);
    return cat8(lds_read_tr16(q), lds_read_tr16(q + 8 * 32));
  };
  const __amdgpu_buffer_rsrc_t irs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.idx + (int64_t)g * p.idx_stride), 0, (uint32_t)(p.Nk * 4), 0x00020000);
  // own entries (OWN): rows past Ms and tiles past the last read as zeros; their V^T
  // tiles, or (VNAT) their V rows as stored
  const __amdgpu_buffer_rsrc_t ksrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)((const __bf16*)p.Ks + (int64_t)g * p.Ms * DH), 0, (uint32_t)(p.Ms * DH * 2), 0x00020000);
  const __amdgpu_buffer_rsrc_t vtsrs =
      VNAT ? __builtin_amdgcn_make_buffer_rsrc((void*)((const __bf16*)p.Vs + (int64_t)g * p.Ms * DH), 0,
                                               (uint32_t)(p.Ms * DH * 2), 0x00020000)
           : __builtin_amdgcn_make_buffer_rsrc((void*)(p.Vts + (int64_t)g * p.own_tiles * DH * 32), 0,
                                               (uint32_t)p.own_tiles * (DH * 64), 0x00020000);
  // logit bias of this KV head's entries (BIAS): entries past Nk read as 0
  const __amdgpu_buffer_rsrc_t brs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.bias + (int64_t)g * p.Nk), 0, (uint32_t)(p.Nk * 4), 0x00020000);
  // exponents of this KV head's block-scaled keys (KQ)
  const __amdgpu_buffer_rsrc_t kers = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(p.Ke + (int64_t)g * p.src_rows * (DH / 32)), 0, (uint32_t)(p.src_rows * (DH / 32)),
      0x00020000);
  // one 8-channel chunk of a stored K row at byte offset off (exponent byte eoff):
  // bf16 as is; KQ: the raw values in .x (.y) and the exponent in .z, expanded at the
  // LDS store
  auto kload = [&](uint32_t off, uint32_t eoff) -> u32x4 {
    if constexpr (KQ == 0) {
      return __builtin_amdgcn_raw_buffer_load_b128(krs, off, 0, 0);
    } else {
      u32x4 r = {};
      if constexpr (KQ == 8) {
        const u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(krs, off, 0, 0);
        r[0] = w[0];
        r[1] = w[1];
      } else {
        r[0] = __builtin_amdgcn_raw_buffer_load_b32(krs, off, 0, 0);
      }
      r[2] = __builtin_amdgcn_raw_buffer_load_b8(kers, eoff, 0, 0);
      return r;
    }
  };
  auto kexpand = [&](const u32x4& r) -> u32x4 {
    if constexpr (KQ == 0) {
      return r;
    } else {
      return __builtin_bit_cast(u32x4, mx_expand8<KQ>(r[0], r[1], (int)(int8_t)(r[2] & 0xffu)));
    }
  };
  constexpr int NSET = kLoadSets;
  u32x4 kreg[NSET][LPT], vreg[NSET][LPT];
  float breg[NSET];
  auto load_tile_to = [&](int tile, int set) {
    if constexpr (BIAS) {
      if (tid < KT) breg[set] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                   brs, (k_begin + tile * KT + tid) * 4, 0, 0));
    }
    if constexpr (OWN) {
      if (own_range && tile >= ct) {
        const int j0 = (tile - ct) * KT;  // first own entry of the tile
#pragma unroll
        for (int i = 0; i < LPT; ++i) {
          const int c = i * NT + tid;
          if (NCH % NT != 0 && c >= NCH) break;
          kreg[set][i] = __builtin_amdgcn_raw_buffer_load_b128(ksrs, (uint32_t)j0 * (DH * 2) + c * 16, 0, 0);
          vreg[set][i] = __builtin_amdgcn_raw_buffer_load_b128(
              vtsrs, VNAT ? (uint32_t)j0 * (DH * 2) + c * 16 : (uint32_t)(j0 / 32) * (DH * 64) + c * 16,
              0, 0);
        }
        return;
      }
    }
    const int kb0 = k_begin + tile * KT;
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int c = i * NT + tid;  // 16-byte chunk: row c / CH, column c % CH
      if (NCH % NT != 0 && c >= NCH) break;
      if constexpr (GATHER) {
        // entries past the index array read as 0; an entry outside the cache is checked
        // before any offset is formed from it, and its row reads as zeros
        const int src = (int)__builtin_amdgcn_raw_buffer_load_b32(irs, (kb0 + c / CH) * 4, 0, 0);
        const bool in = (uint32_t)src < (uint32_t)p.src_rows;
        const uint32_t row = in ? (uint32_t)src : 0u;
        const u32x4 kv = kload(row * KRB + (c % CH) * KCB, row * (DH / 32) + (c % CH) / 4);
        kreg[set][i] = in ? kv : u32x4{};
      } else {
        // chunk c of the tile: byte c * KCB past its first row, exponent byte c / 4
        kreg[set][i] = kload((uint32_t)kb0 * KRB + c * KCB, (uint32_t)kb0 * (DH / 32) + c / 4);
      }
      // V^T tile kb0 / 32 (already gathered), or (VNAT) V rows kb0 ..; tiles past the end
      // read as 0
      vreg[set][i] = __builtin_amdgcn_raw_buffer_load_b128(
          vrs, VNAT ? (uint32_t)kb0 * (DH * 2) + c * 16 : (uint32_t)(kb0 / 32) * (DH * 64) + c * 16, 0, 0);
    }
  };
  auto store_tile_from = [&](int buf, int set) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      const int c = i * NT + tid;
      if (NCH % NT != 0 && c >= NCH) break;
      const int row = c / CH, col = c % CH;
      *(u32x4*)(&Ks[buf][row * KP + col * 8]) = kexpand(kreg[set][i]);
      if constexpr (VNAT) *(u32x4*)(&Vs[buf][vnat_pos(c) * 8]) = vreg[set][i];
      else *(u32x4*)(&Vs[buf][(c / 4) * VTP + (c % 4) * 8]) = vreg[set][i];
    }
    if constexpr (BIAS) {
      if (tid < KT) Bs[buf][tid] = breg[set] * p.bias_mul;
    }
  };
  auto load_tile = [&](int tile) { load_tile_to(tile, 0); };
  auto store_tile = [&](int buf) { store_tile_from(buf, 0); };

  f32x16 o[QT][ND];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt)
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) o[qt][dt] = f32x16{};
  float m_run[QT], l_part[QT];
#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    m_run[qt] = -INFINITY;
    l_part[qt] = 0.f;
  }
  const float c = p.c;


  // S^T = K Q^T (+ init) for the tile in LDS slot `buf`
  auto scores_init = [&](f32x16 (&s)[NKT][QT], int buf, const f32x16 (&init)[NKT]) {
    const __bf16* ks = Ks[buf];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) s[kt][qt] = init[kt];
#pragma unroll
    for (int st = 0; st < NS; ++st) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const bf16x8 a = *(const bf16x8*)(ks + (kt * 32 + l32) * KP + st * 16 + h32 * 8);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) s[kt][qt] = mfma32(a, qf[qt][st], s[kt][qt]);
      }
    }
  };
  // keys >= k_end of tile t set to -inf; own entries j > m of query m set to -inf
  auto mask = [&](f32x16 (&s)[NKT][QT], int t) {
    if constexpr (OWN) {
      if (own_range && t >= ct) {
        const int j0 = (t - ct) * KT;
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          const int mq = min(row_base + qt * 32 + l32, p.rows - 1) / p.G;
#pragma unroll
          for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
              const int j = j0 + kt * 32 + 8 * (e >> 2) + 4 * h32 + (e & 3);
              if (j > mq) s[kt][qt][e] = -INFINITY;
            }
        }
        return;
      }
    }
    const int tb = k_begin + t * KT;
    if (tb + KT > k_end) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int key = tb + kt * 32 + 8 * (e >> 2) + 4 * h32 + (e & 3);
          if (key >= k_end) {
#pragma unroll
            for (int qt = 0; qt < QT; ++qt) s[kt][qt][e] = -INFINITY;
          }
        }
    }
  };
  // the accumulator's starting value: zero, or (BIAS) the tile's biases; element
  // 4j + i of a lane's fragment is key 8j + 4 h32 + i of the 32-key tile
  auto start = [&](int buf, f32x16 (&init)[NKT]) {
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt) {
      if constexpr (BIAS) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const f32x4 b = *(const f32x4*)(&Bs[buf][kt * 32 + 8 * j + 4 * h32]);
#pragma unroll
          for (int i = 0; i < 4; ++i) init[kt][4 * j + i] = b[i];
        }
      } else {
        init[kt] = f32x16{};
      }
    }
  };
  auto scores = [&](f32x16 (&s)[NKT][QT], int buf, int t) {
    f32x16 init[NKT];
    start(buf, init);
    scores_init(s, buf, init);
    mask(s, t);
  };
  // scaled row max of the tile (both halves of the 64-lane wave)
  auto row_max = [&](f32x16 (&s)[NKT][QT], float (&mt)[QT]) {
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) {
      float mx = s[0][qt][0];
#pragma unroll
      for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s[0][qt][e]);
#pragma unroll
      for (int kt = 1; kt < NKT; ++kt)
#pragma unroll
        for (int e = 0; e < 16; ++e) mx = fmaxf(mx, s[kt][qt][e]);
      mt[qt] = pair_max(mx) * c;
    }
  };
  // P = exp2(S c - m_run) as bf16 MFMA operands (two-term split when PSPLIT). The row
  // sums add up the bf16 values the MFMA actually uses (v_dot2 with (1, 1)), from the
  // same packed pairs: one v_cvt_pk_bf16_f32 per pair serves both (converted element by
  // element, the compiler repacked the pairs for the sums with extra conversions and
  // permutes).
  auto softmax = [&](f32x16 (&s)[NKT][QT], bf16x8 (&pb)[NKT][QT][2], bf16x8 (&pl)[NKT][QT][2]) {
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) {
        const float nm = -m_run[qt];
#pragma unroll
        for (int e = 0; e < 16; ++e) s[kt][qt][e] = fast_exp2(fmaf(s[kt][qt][e], c, nm));
        float sum0 = 0.f, sum1 = 0.f;
#pragma unroll
        for (int p2 = 0; p2 < 2; ++p2) {
          u32x4 hw, lw = {};
#pragma unroll
          for (int e = 0; e < 8; e += 2) {
            const float v0 = s[kt][qt][8 * p2 + e], v1 = s[kt][qt][8 * p2 + e + 1];
            const unsigned hp = pack_bf16(v0, v1);
            hw[e / 2] = hp;
            sum0 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, hp), ones, sum0,
                                                   false);
            if constexpr (PSPLIT) {
              const float h0 = __builtin_bit_cast(float, hp << 16);
              const float h1 = __builtin_bit_cast(float, hp & 0xffff0000u);
              const unsigned lp = pack_bf16(v0 - h0, v1 - h1);
              lw[e / 2] = lp;
              sum1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, lp), ones, sum1,
                                                     false);
            }
          }
          pb[kt][qt][p2] = __builtin_bit_cast(bf16x8, hw);
          if constexpr (PSPLIT) pl[kt][qt][p2] = __builtin_bit_cast(bf16x8, lw);
        }
        // (sum1 only with a two-term P: sum0 + 0 would cost an add the compiler keeps)
        if constexpr (PSPLIT) l_part[qt] += sum0 + sum1;
        else l_part[qt] += sum0;
      }
  };
  // O^T += V^T P^T with the V^T tile of LDS slot `buf`: the A operand (32 rows of d,
  // 8 keys) is one 16-byte read, in the P fragments' key order
  auto pv = [&](bf16x8 (&pb)[NKT][QT][2], bf16x8 (&pl)[NKT][QT][2], int buf) {
    const __bf16* vs = Vs[buf];
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int p2 = 0; p2 < 2; ++p2) {
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
          const bf16x8 a = VNAT ? vfrag(vs, p2, dt)
                                : *(const bf16x8*)(vs + (dt * 32 + l32) * VTP + kt * 32 + 16 * p2 + 8 * h32);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            o[qt][dt] = mfma32(a, pb[kt][qt][p2], o[qt][dt]);
            if constexpr (PSPLIT) o[qt][dt] = mfma32(a, pl[kt][qt][p2], o[qt][dt]);
          }
        }
      }
  };
  auto accumulate = [&](f32x16 (&s)[NKT][QT], int buf) {
    bf16x8 pb[NKT][QT][2];
    bf16x8 pl[NKT][QT][2];
    softmax(s, pb, pl);
    pv(pb, pl, buf);
  };

  if (tid == 0) overflow = 0;
  if constexpr (!DMA) {
    load_tile_to(0, 0);
    store_tile_from(0, 0);
  }

  if constexpr (DMA) {
    // LDS position c of a slot holds K row c / CH, chunk (c % CH) ^ swk(row), and
    // V^T row c / 4, chunk (c % 4) ^ ((row / 4) % 4): for every 16 consecutive rows read
    // at one chunk index the 16-byte reads land in 16 different bank groups.
    constexpr int RPB = 16 / CH;  // K rows per 256 bytes of LDS
    constexpr int D = kDmaAhead;
    // the issuing waves' lanes each move LPD 16-byte chunks of the K tile and LPD of the
    // V^T tile; chunk c = i * DT + tid of round i (with K through registers, all eight
    // waves issuing a share of the V tile measured slower: 14.0 against 13.5 ms for an
    // MXINT8 pass of 4,096 queries x 32 heads over 172,032 entries)
    constexpr int DW = kDmaWaves;
    constexpr int DT = DW * kWave;
    constexpr int LPD = NCH / DT;
    static_assert(NCH % DT == 0 && LPD >= 1 && LPD <= kDmaLpdMax && DW <= NT / kWave,
                  "whole DMA rounds of the issuing waves");
    // (sized by a namespace-scope constant: an array sized by the local constexpr and
    // captured by the lambdas below made the host pass drop these kernels' launch stubs)
    uint32_t koff[kDmaLpdMax], voff[kDmaLpdMax];
#pragma unroll
    for (int i = 0; i < LPD; ++i) {
      const int c = i * DT + tid % DT;
      const int krow = c / CH, kch = (c % CH) ^ ((krow / RPB) % CH);
      koff[i] = (uint32_t)(krow * DH * 2 + kch * 16);
      if constexpr (VNAT) {
        // LDS chunk position c holds channels 8 (4 dt + cq) .. of key (c / 4) % KT
        const int dt = c / (KT * 4), key = (c / 4) % KT, cq = c % 4;
        voff[i] = (uint32_t)(key * (DH * 2) + (4 * dt + cq) * 16);
      } else {
        const int vrow = c / 4, vch = (c % 4) ^ ((vrow / 4) % 4);
        voff[i] = (uint32_t)(vrow * 64 + vch * 16);
      }
    }
    // the tile offset goes into the per-lane offset, so the buffer range check covers it
    // (OWN: the tiles after the cache range of the last key range are the chunk's own
    // entries, from their own buffers)
    auto issue = [&](int tile, auto slot_t) {
      constexpr int SL = decltype(slot_t)::value;
      // a scalar branch (wid is wave-uniform)
      if (__builtin_amdgcn_readfirstlane(wid) >= DW) return;
#pragma unroll
      for (int i = 0; i < LPD; ++i) {
        // a wave's DMA instruction writes its 64 lanes' chunks to 1 KB of consecutive LDS
        PKV_LDS void* kd = (PKV_LDS void*)&Kd[SL][(i * DT + wid * 64) * 8];
        PKV_LDS void* vd = (PKV_LDS void*)&Vd[SL][(i * DT + wid * 64) * 8];
        if (OWN && own_range && tile >= ct) {
          const uint32_t j0 = (uint32_t)((tile - ct) * KT);
          if constexpr (!KREG)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ksrs, kd, 16, koff[i] + j0 * (DH * 2), 0, 0, 0);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              vtsrs, vd, 16, voff[i] + (VNAT ? j0 * (DH * 2) : (j0 / 32) * (DH * 64)), 0, 0, 0);
        } else {
          const uint32_t kb0 = (uint32_t)(k_begin + tile * KT);
          // (block-scaled and gathered keys come through registers, kq_load / kq_store)
          if constexpr (!KREG)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(krs, kd, 16, koff[i] + kb0 * (DH * 2), 0, 0, 0);
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              vrs, vd, 16, voff[i] + (VNAT ? kb0 * (DH * 2) : (kb0 / 32) * (DH * 64)), 0, 0, 0);
        }
      }
    };
    // wait until at most N of this wave's loads are in flight (waves that issue none pass
    // at once), then a plain barrier (no fence: it would wait for every load in flight)
    auto sync_slots = [&](auto n_t) {
      constexpr int N = decltype(n_t)::value;
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(N) : "memory");
    };
    const int swk = (l32 / RPB) % CH, swv = (l32 / 4) % 4;
    auto scores_d = [&](f32x16 (&s)[NKT][QT], auto slot_t) {
      constexpr int SL = decltype(slot_t)::value;
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) s[0][qt] = f32x16{};
#pragma unroll
      for (int st = 0; st < NS; ++st) {
        const bf16x8 a = *(const bf16x8*)(&Kd[SL][l32 * DH + (((2 * st + h32) ^ swk) * 8)]);
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) s[0][qt] = mfma32(a, qf[qt][st], s[0][qt]);
      }
    };
    auto pv_d = [&](bf16x8 (&pb)[NKT][QT][2], bf16x8 (&pl)[NKT][QT][2], auto slot_t) {
      constexpr int SL = decltype(slot_t)::value;
#pragma unroll
      for (int p2 = 0; p2 < 2; ++p2)
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) {
          const bf16x8 a =
              VNAT ? vfrag(&Vd[SL][0], p2, dt)
                   : *(const bf16x8*)(&Vd[SL][(dt * 32 + l32) * 32 + (((2 * p2 + h32) ^ swv) * 8)]);
#pragma unroll
          for (int qt = 0; qt < QT; ++qt) {
            o[qt][dt] = mfma32(a, pb[0][qt][p2], o[qt][dt]);
            if constexpr (PSPLIT) o[qt][dt] = mfma32(a, pl[0][qt][p2], o[qt][dt]);
          }
        }
    };
    static_assert(NKT == 1, "DMA path: one 32-key MFMA tile");
    // Block-scaled keys (KQ) and gathered keys (GATHER): V^T tiles (expanded or gathered
    // by vt_kernel) still arrive by DMA; the stored K chunks are loaded by every thread
    // (chunk c = u * NT + tid) three steps before their LDS store, in four register sets,
    // and expanded (KQ) at the store into the slot's swizzled layout. Step t stores K tile
    // t + 3 (read at step t + 2, after a barrier) and loads tile t + 6. A gathered row's
    // index is loaded three steps before its K chunk (step t loads the indices of tile
    // t + 9) into a ring of four, so no load waits on another one issued in the same step.
    constexpr int LPK = (NCH + NT - 1) / NT;
    constexpr int KSETS = 4, KLEAD = 3;
    static_assert(!KREG || (NSL % KSETS == 0 && KLEAD + 3 <= D + 1), "K register sets");
    static_assert(!GATHER || LPK == 1, "one gathered K chunk per thread and tile");
    u32x4 kq[KREG ? KSETS : 1][LPK];
    uint32_t kidx[GATHER ? KSETS : 1];
    bool kin[GATHER ? KSETS : 1];  // the gathered row is inside the cache
    // the index of the row of this thread's chunk in tile `tile` (entries past the index
    // array read as 0; own tiles load a placeholder, so every step issues the same loads)
    auto kidx_load = [&](int tile, auto set_t) {
      if constexpr (GATHER) {
        constexpr int SET = decltype(set_t)::value;
        kidx[SET] = __builtin_amdgcn_raw_buffer_load_b32(irs, (k_begin + tile * KT + tid / CH) * 4, 0, 0);
      }
    };
    auto kq_load = [&](int tile, auto set_t) {
      if constexpr (KREG) {
        constexpr int SET = decltype(set_t)::value;
        const int kb0 = k_begin + tile * KT;
#pragma unroll
        for (int u = 0; u < LPK; ++u) {
          const int cc = u * NT + tid;
          if (NCH % NT != 0 && cc >= NCH) break;
          if constexpr (GATHER) {
            if (OWN && own_range && tile >= ct) {
              kq[SET][u] = __builtin_amdgcn_raw_buffer_load_b128(
                  ksrs, (uint32_t)((tile - ct) * KT) * (DH * 2) + cc * 16, 0, 0);
              kin[SET] = true;
            } else {
              // an entry outside the cache is checked before any offset is formed from it,
              // and its row is stored as zeros (the select waits until the store, so the
              // load need not have landed here)
              const int src = (int)kidx[SET];
              const bool in = (uint32_t)src < (uint32_t)p.src_rows;
              const uint32_t row = in ? (uint32_t)src : 0u;
              kq[SET][u] = kload(row * KRB + (cc % CH) * KCB, row * (DH / 32) + (cc % CH) / 4);
              kin[SET] = in;
            }
          } else {
            kq[SET][u] = kload((uint32_t)kb0 * KRB + cc * KCB, (uint32_t)kb0 * (DH / 32) + cc / 4);
          }
        }
      }
    };
    auto kq_store = [&](auto set_t, auto slot_t) {
      if constexpr (KREG) {
        constexpr int SET = decltype(set_t)::value, SL = decltype(slot_t)::value;
#pragma unroll
        for (int u = 0; u < LPK; ++u) {
          const int cc = u * NT + tid;
          if (NCH % NT != 0 && cc >= NCH) break;
          const int row = cc / CH, pos = row * CH + ((cc % CH) ^ ((row / RPB) % CH));
          u32x4 v = kexpand(kq[SET][u]);
          if constexpr (GATHER) v = kin[SET] ? v : u32x4{};
          *(u32x4*)(&Kd[SL][pos * 8]) = v;
        }
      }
    };
    // loads a wave may leave in flight at a barrier (V^T tiles t + 4 .. t + 6 and, with
    // K through registers, the K loads issued after V^T tile t + 3)
    // loads per step besides the V^T tile's: values and exponent (KQ), or index and row
    // (GATHER)
    constexpr int KLI = KREG ? 2 : 0;
    constexpr int INFL = KREG ? KLI + 3 * (LPD + KLI) : 2 * LPD * (D - kDmaSteps - 1);
    static_for<D>([&](auto j_t) { issue(decltype(j_t)::value, j_t); });
    if constexpr (KREG) {
      static_assert(D == 6 && kDmaSteps == 2, "the K schedule assumes six tiles ahead");
      kidx_load(0, std::integral_constant<int, 0>{});
      kidx_load(1, std::integral_constant<int, 1>{});
      kidx_load(2, std::integral_constant<int, 2>{});
      kq_load(0, std::integral_constant<int, 0>{});
      kq_load(1, std::integral_constant<int, 1>{});
      kq_load(2, std::integral_constant<int, 2>{});
      kq_store(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});
      kq_store(std::integral_constant<int, 1>{}, std::integral_constant<int, 1>{});
      kq_store(std::integral_constant<int, 2>{}, std::integral_constant<int, 2>{});
      kidx_load(3, std::integral_constant<int, 3>{});
      kidx_load(4, std::integral_constant<int, 0>{});
      kidx_load(5, std::integral_constant<int, 1>{});
      kq_load(3, std::integral_constant<int, 3>{});
      kq_load(4, std::integral_constant<int, 0>{});
      kq_load(5, std::integral_constant<int, 1>{});
      kidx_load(6, std::integral_constant<int, 2>{});
      kidx_load(7, std::integral_constant<int, 3>{});
      kidx_load(8, std::integral_constant<int, 0>{});
    }
    // tiles 0 .. kDmaSteps resident
    sync_slots(std::integral_constant<int, INFL>{});
    f32x16 sa[NKT][QT], sb[NKT][QT];
    scores_d(sa, std::integral_constant<int, 0>{});
    mask(sa, 0);  // a key range shorter than one tile
    {
      float mt[QT];
      row_max(sa, mt);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) m_run[qt] = mt[qt];
    }
    bool over = false;
    // step t (I = t % NSL): issue tile t + D; S_{t+1} = K_{t+1} Q^T; P_t; O += V_t P_t;
    // then tile t + 2 must be resident (2 (D - 2) loads of later tiles may be in flight)
    auto step = [&](auto i_t, auto masked_t, f32x16 (&sc)[NKT][QT], f32x16 (&sn)[NKT][QT], int t) {
      constexpr int I = decltype(i_t)::value;
      constexpr bool MASKED = decltype(masked_t)::value;
      issue(t + D, std::integral_constant<int, (I + D) % NSL>{});
      kq_store(std::integral_constant<int, (I + 3) % KSETS>{}, std::integral_constant<int, (I + 3) % NSL>{});
      kq_load(t + 3 + KLEAD, std::integral_constant<int, (I + 3 + KLEAD) % KSETS>{});
      kidx_load(t + 6 + KLEAD, std::integral_constant<int, (I + 6 + KLEAD) % KSETS>{});
      scores_d(sn, std::integral_constant<int, (I + 1) % NSL>{});
      if constexpr (MASKED) mask(sn, t + 1);
      bf16x8 pb[NKT][QT][2];
      bf16x8 pl[NKT][QT][2];
      softmax(sc, pb, pl);
      pv_d(pb, pl, std::integral_constant<int, I % NSL>{});
      // the row sums are complete at the end of each step: left free, the compiler sank
      // every step's sums to the end of the unrolled loop, holding all eight tiles' P
      // registers live (256 VGPRs against 202, 4 % slower)
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) asm volatile("" : "+v"(l_part[qt]));
      // a barrier after every kDmaSteps steps: the next group reads up to tile
      // t + kDmaSteps + 1, and 2 (D - kDmaSteps - 1) loads of later tiles may be in flight
      if constexpr (I % kDmaSteps == kDmaSteps - 1) sync_slots(std::integral_constant<int, INFL>{});
    };
    auto steps = [&](auto masked_t, int t) {
      static_for<NSL / 2>([&](auto h_t) {
        constexpr int H = decltype(h_t)::value;
        step(std::integral_constant<int, 2 * H>{}, masked_t, sa, sb, t + 2 * H);
        step(std::integral_constant<int, 2 * H + 1>{}, masked_t, sb, sa, t + 2 * H + 1);
      });
    };
    const int t_full = (k_end - k_begin) / KT;
    int t = 0;
    for (; t + NSL < t_full; t += NSL) steps(std::false_type{}, t);
    for (; t < ntiles; t += NSL) steps(std::true_type{}, t);
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) over |= untrusted_sum(l_part[qt]);
    if (__ballot(over) != 0) overflow = 1;
    // every load has landed before the slots are given up
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
  } else if constexpr (!SAFE) {
    // Software pipeline over four LDS slots (tile t in slot t % 4) and NSET register
    // staging sets (tile j is loaded into set j % NSET). Step t:
    //   issue the loads of tile t + NSET + 1;
    //   MFMA S_{t+1} = K_{t+1} Q^T  while the VALU forms P_t from S_t;
    //   MFMA O += V_t P_t           while the VALU takes S_{t+1}'s row max;
    //   store tile t+2 (loaded in step t - NSET + 1) into its slot, last read in
    //   step t-2; one barrier.
    // A tile's loads thus have NSET - 1 whole steps to arrive: the workgroups of an
    // XCD stream the same K/V rows at about the same time, so most loads wait for
    // one shared miss and see close to the full memory latency.
    // The loop runs a multiple of UNR steps; tiles past the key range are fully
    // masked (they contribute nothing), so every step has the same shape.
    constexpr int UNR = NSET > 2 ? NSET : 2;
    load_tile_to(1, 0);
    store_tile_from(1, 0);
#pragma unroll
    for (int j = 2; j <= NSET; ++j) load_tile_to(j, j % NSET);
    __syncthreads();
    f32x16 sa[NKT][QT], sb[NKT][QT];
    scores(sa, 0, 0);
    {
      float mt[QT];
      row_max(sa, mt);
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) m_run[qt] = mt[qt];
    }
    bool over = false;
    // I: step index modulo UNR (compile time); MASKED: the tile scored in this step
    // may reach past k_end
    auto step = [&](auto i_t, auto masked_t, f32x16 (&sc)[NKT][QT], f32x16 (&sn)[NKT][QT], int t) {
      constexpr int I = decltype(i_t)::value;
      constexpr bool MASKED = decltype(masked_t)::value;
      load_tile_to(t + NSET + 1, (I + NSET + 1) % NSET);
      if constexpr (MASKED) {
        scores(sn, (t + 1) & 3, t + 1);
      } else {
        f32x16 init[NKT];
        start((t + 1) & 3, init);
        scores_init(sn, (t + 1) & 3, init);
      }
      bf16x8 pb[NKT][QT][2];
      bf16x8 pl[NKT][QT][2];
      softmax(sc, pb, pl);
      pv(pb, pl, t & 3);
      store_tile_from((t + 2) & 3, (I + 2) % NSET);
      __syncthreads();
    };
    auto steps = [&](auto masked_t, int t) {
      step(std::integral_constant<int, 0>{}, masked_t, sa, sb, t);
      step(std::integral_constant<int, 1>{}, masked_t, sb, sa, t + 1);
      if constexpr (UNR == 4) {
        step(std::integral_constant<int, 2>{}, masked_t, sa, sb, t + 2);
        step(std::integral_constant<int, 3>{}, masked_t, sb, sa, t + 3);
      }
    };
    static_assert(UNR == 2 || UNR == 4, "pipeline unroll");
    // tiles [0, t_full) lie entirely inside the key range; step t scores tile t+1
    const int t_full = (k_end - k_begin) / KT;
    int t = 0;
    for (; t + UNR < t_full; t += UNR) steps(std::false_type{}, t);
    for (; t < ntiles; t += UNR) steps(std::true_type{}, t);
    // a lane's partial sum bounds every weight it added
#pragma unroll
    for (int qt = 0; qt < QT; ++qt) over |= untrusted_sum(l_part[qt]);
    if (__ballot(over) != 0) overflow = 1;
    __syncthreads();
  } else {
    // lazy rescale: when a row's running max would grow by more than 2^kTau the
    // wave rescales O first (m_run = -inf on the first tile: alpha = 0)
    __syncthreads();
    for (int t = 0; t < ntiles; ++t) {
      const int cur = t & 1;
      if (t + 1 < ntiles) load_tile(t + 1);
      f32x16 s[NKT][QT];
      scores(s, cur, t);
      float mt[QT];
      row_max(s, mt);
      bool need = false;
#pragma unroll
      for (int qt = 0; qt < QT; ++qt) need |= mt[qt] > m_run[qt] + kTau;
      if (__ballot(need) != 0) {
#pragma unroll
        for (int qt = 0; qt < QT; ++qt) {
          const float mn = fmaxf(m_run[qt], mt[qt]);
          const float alpha = fast_exp2(m_run[qt] - mn);
          m_run[qt] = mn;
          l_part[qt] *= alpha;
#pragma unroll
          for (int dt = 0; dt < ND; ++dt) o[qt][dt] *= alpha;
        }
      }
      accumulate(s, cur);
      if (t + 1 < ntiles) store_tile(cur ^ 1);
      __syncthreads();
    }
  }

#pragma unroll
  for (int qt = 0; qt < QT; ++qt) {
    const float l = pair_sum(l_part[qt]);
    const int r = row_base + qt * 32 + l32;
    if (r >= p.rows) continue;
    if constexpr (!PARTIAL) {
      const float inv = 1.0f / l;
      const int m = r / p.G, j = r - m * p.G;
      float* op = p.O + ((int64_t)m * p.Hq + g * p.G + j) * DH + 4 * h32;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          f32x4 v = {o[qt][dt][4 * jj] * inv, o[qt][dt][4 * jj + 1] * inv,
                     o[qt][dt][4 * jj + 2] * inv, o[qt][dt][4 * jj + 3] * inv};
          *(f32x4*)(op + dt * 32 + 8 * jj) = v;
        }
    } else {
      const int64_t rid = ((int64_t)(g * p.n_split + split)) * p.rows + r;
      float* op = p.Opart + rid * DH + 4 * h32;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt)
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          f32x4 v = {o[qt][dt][4 * jj], o[qt][dt][4 * jj + 1], o[qt][dt][4 * jj + 2],
                     o[qt][dt][4 * jj + 3]};
          *(f32x4*)(op + dt * 32 + 8 * jj) = v;
        }
      if (h32 == 0) {
        p.ML[2 * rid] = m_run[qt];
        p.ML[2 * rid + 1] = l;
      }
    }
  }
  if constexpr (!SAFE) {
    if (tid == 0) p.flags[w] = overflow;
  }
}

// fp32 inputs: exact fp32 products on MFMA 32x32x2 f32, fp32 online softmax with expf.
// A workgroup of kF32Waves waves owns kRowsF32 rows of one KV head, 32 per wave, as in
// the bf16 kernel. K and V tiles of 32 keys are staged through registers into two LDS
// slots (natural [key][d] layout: an fp32 operand is one value per lane, so V needs no
// transposed copy). The contraction orders are chosen so that every operand read is a
// 16-byte (or 8-byte) LDS read:
//   scores S^T = K Q^T: step s pairs channel h * DH/2 + s of lane half h, so a lane
//     reads 4 consecutive channels of its key for 4 steps;
//   O^T += V^T P^T: step s takes key 8 (s / 4) + 4 h + s % 4 on lane half h, which is
//     where element s of the score accumulator already holds that key's weight, and
//     output row rho of MFMA tile dt is channel ND * rho + dt, so one read fetches a
//     key's ND channels for all ND tiles.
template <int DH, bool GATHER, bool PARTIAL, bool OWN, bool BIAS>
__global__ __launch_bounds__(kF32Waves * 64) void attn_f32_kernel(AttnParams p) {
  static_assert(!(OWN && BIAS), "own entries carry no bias");
  static_assert(DH == 64 || DH == 128, "head_dim 64 or 128");
  static_assert(kRowsF32 == 32 * kF32Waves, "32 rows per wave");
  constexpr int KT = kKeyTileF32;  // 32 keys per tile
  constexpr int HALF = DH / 2;     // score steps (two channels per MFMA)
  constexpr int ND = DH / 32;      // 32-row output tiles of O^T
  constexpr int KPF = DH + 4;      // K tile pitch (floats): conflict-free 16-byte reads
  constexpr int C4 = DH / 4;       // 16-byte chunks per row
  constexpr int NT = kF32Waves * 64;
  constexpr int LPT = KT * C4 / NT;  // chunks per thread per tile, K and V each
  static_assert(KT == 32 && KT * C4 % NT == 0 && LPT >= 1, "whole staging rounds");
  typedef float VN __attribute__((ext_vector_type(ND)));
  __shared__ __attribute__((aligned(16))) float Ks[2][KT * KPF];
  __shared__ __attribute__((aligned(16))) float Vs[2][KT * DH];
  __shared__ float Bs[2][BIAS ? KT : 1];

  const int w = xcd_item(p.per_xcd);
  if (w >= p.total_items) return;
  const int rt = w % p.row_tiles;
  const int t2 = w / p.row_tiles;
  const int split = t2 % p.n_split;
  const int g = t2 / p.n_split;
  const int nk = p.counts ? min(max(p.counts[g], 1), p.Nk) : p.Nk;
  const int k_begin = split * p.keys_per_split;
  const int k_end = min(nk, k_begin + p.keys_per_split);  // empty range: (O, m, l) = (0, -inf, 0)
  const int32_t* ig = GATHER ? p.idx + (int64_t)g * p.idx_stride : nullptr;
  const int ct = k_end > k_begin ? (k_end - k_begin + KT - 1) / KT : 0;  // cache tiles
  const bool own_range = OWN && split == p.n_split - 1;
  int ntiles = ct;
  if (own_range) {
    const int last_q = min(p.rows - 1, rt * kRowsF32 + kRowsF32 - 1) / p.G;
    ntiles = ct + last_q / KT + 1;
  }

  const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
  const int h = lane >> 5, l32 = lane & 31;
  const int r = rt * kRowsF32 + wid * 32 + l32;
  const int rr = min(r, p.rows - 1);
  const int mq = rr / p.G, jq = rr - mq * p.G;
  const float* Kb = (const float*)p.K + (int64_t)g * p.src_rows * DH;
  const float* Vb = (const float*)p.V + (int64_t)g * p.src_rows * DH;
  const float* Ksb = OWN ? (const float*)p.Ks + (int64_t)g * p.Ms * DH : nullptr;
  const float* Vsb = OWN ? (const float*)p.Vs + (int64_t)g * p.Ms * DH : nullptr;

  // B operand of the score steps: channels h * HALF .. h * HALF + HALF - 1 of this row
  float qv[HALF];
  {
    const f32x4* qp =
        (const f32x4*)((const float*)p.Q + ((int64_t)mq * p.Hq + g * p.G + jq) * DH + h * HALF);
#pragma unroll
    for (int i = 0; i < HALF / 4; ++i) {
      const f32x4 v = qp[i];
#pragma unroll
      for (int u = 0; u < 4; ++u) qv[4 * i + u] = v[u];
    }
  }
  f32x16 o[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) o[dt] = f32x16{};
  float m_run = -INFINITY, l_part = 0.f;

  // staging: chunk c = u * NT + tid of a tile is key row c / C4, channels 4 (c % C4)..
  f32x4 kst[LPT], vst[LPT];
  float bst = 0.f;
  auto load_tile = [&](int t) {
#pragma unroll
    for (int u = 0; u < LPT; ++u) {
      const int c = u * NT + tid, row = c / C4, col = c % C4;
      f32x4 kv = {}, vv = {};
      if (!OWN || t < ct) {
        const int key = k_begin + t * KT + row;
        if (key < k_end) {
          int src = key;
          bool in = true;
          if constexpr (GATHER) {
            // an entry outside the cache reads as a zero row (no offset is formed from it)
            src = ig[key];
            in = (uint32_t)src < (uint32_t)p.src_valid;
          }
          if (in) {
            kv = *((const f32x4*)(Kb + (int64_t)src * DH) + col);
            vv = *((const f32x4*)(Vb + (int64_t)src * DH) + col);
          }
        }
      } else {
        const int j = (t - ct) * KT + row;  // own entry
        if (j < p.Ms) {
          kv = *((const f32x4*)(Ksb + (int64_t)j * DH) + col);
          vv = *((const f32x4*)(Vsb + (int64_t)j * DH) + col);
        }
      }
      kst[u] = kv;
      vst[u] = vv;
    }
    if constexpr (BIAS) {
      if (tid < KT) {
        const int key = k_begin + t * KT + tid;
        bst = key < k_end ? p.bias[(int64_t)g * p.Nk + key] : 0.f;
      }
    }
  };
  auto store_tile = [&](int buf) {
#pragma unroll
    for (int u = 0; u < LPT; ++u) {
      const int c = u * NT + tid, row = c / C4, col = c % C4;
      *(f32x4*)&Ks[buf][row * KPF + 4 * col] = kst[u];
      *(f32x4*)&Vs[buf][row * DH + 4 * col] = vst[u];
    }
    if constexpr (BIAS) {
      if (tid < KT) Bs[buf][tid] = bst;
    }
  };

  auto compute_tile = [&](int t, int buf) {
    // S^T: element e of this lane is key 8 (e / 4) + 4 h + e % 4 of the tile, row l32
    f32x16 sc = {};
    const float* kr = &Ks[buf][l32 * KPF + h * HALF];
#pragma unroll
    for (int s4 = 0; s4 < HALF / 4; ++s4) {
      const f32x4 kv = *(const f32x4*)(kr + 4 * s4);
#pragma unroll
      for (int u = 0; u < 4; ++u) sc = mfma32_f32(kv[u], qv[4 * s4 + u], sc);
    }
    const bool own_tile = OWN && t >= ct;
    float mx = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int kk = 8 * (e >> 2) + 4 * h + (e & 3);
      float v;
      if (own_tile) {
        const int j = (t - ct) * KT + kk;
        v = (j <= mq && j < p.Ms) ? sc[e] * p.c : -INFINITY;
      } else {
        const int key = k_begin + t * KT + kk;
        v = key < k_end ? fmaf(sc[e], p.c, BIAS ? Bs[buf][kk] : 0.f) : -INFINITY;
      }
      sc[e] = v;
      mx = fmaxf(mx, v);
    }
    const float m_new = fmaxf(m_run, pair_max(mx));
    if (m_new == -INFINITY) {  // every key so far masked (or a -inf bias): no weight
#pragma unroll
      for (int e = 0; e < 16; ++e) sc[e] = 0.f;
    } else {
      if (m_new > m_run) {
        const float a = expf(m_run - m_new);
        l_part *= a;
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) o[dt] *= a;
        m_run = m_new;
      }
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        sc[e] = expf(sc[e] - m_run);
        l_part += sc[e];
      }
    }
    // O^T += V^T P^T
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int kk = 8 * (s >> 2) + 4 * h + (s & 3);
      const VN vv = *(const VN*)&Vs[buf][kk * DH + ND * l32];
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) o[dt] = mfma32_f32(vv[dt], sc[s], o[dt]);
    }
  };

  // two slots: tile t + 1's loads are in flight while tile t is multiplied
  if (ntiles > 0) {
    load_tile(0);
    store_tile(0);
    __syncthreads();
  }
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) load_tile(t + 1);
    compute_tile(t, buf);
    if (t + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  if (r >= p.rows) return;
  const float l = pair_sum(l_part);
  // element e of tile dt is channel ND (8 (e / 4) + 4 h + e % 4) + dt
  if constexpr (!PARTIAL) {
    const float inv = 1.0f / l;
    float* op = p.O + ((int64_t)mq * p.Hq + g * p.G + jq) * DH;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      VN v;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) v[dt] = o[dt][e] * inv;
      *(VN*)(op + ND * (8 * (e >> 2) + 4 * h + (e & 3))) = v;
    }
  } else {
    const int64_t rid = ((int64_t)(g * p.n_split + split)) * p.rows + r;
    float* op = p.Opart + rid * DH;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      VN v;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) v[dt] = o[dt][e];
      *(VN*)(op + ND * (8 * (e >> 2) + 4 * h + (e & 3))) = v;
    }
    if (h == 0) {
      p.ML[2 * rid] = m_run;
      p.ML[2 * rid + 1] = l;
    }
  }
}

// Merge split-key partials: O = sum_s e^(m_s - m*) O_s / sum_s e^(m_s - m*) l_s.
template <int DH, bool LOG2>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ Opart,
                                                           const float* __restrict__ ML,
                                                           float* __restrict__ O, int rows,
                                                           int n_split, int Hkv, int G, int Hq) {
  constexpr int C4 = DH / 4;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)Hkv * rows * C4;
  if (gid >= total) return;
  const int c4 = (int)(gid % C4);
  const int64_t t = gid / C4;
  const int r = (int)(t % rows);
  const int g = (int)(t / rows);
  float mx = -INFINITY;
  for (int s = 0; s < n_split; ++s) mx = fmaxf(mx, ML[2 * (((int64_t)g * n_split + s) * rows + r)]);
  f32x4 acc = {};
  float l = 0.f;
  for (int s = 0; s < n_split; ++s) {
    const int64_t rid = ((int64_t)g * n_split + s) * rows + r;
    const float ms = ML[2 * rid];
    const float wgt = LOG2 ? exp2f(ms - mx) : expf(ms - mx);
    l += wgt * ML[2 * rid + 1];
    const f32x4 v = *((const f32x4*)(Opart + rid * DH) + c4);
    acc += wgt * v;
  }
  const int m = r / G, j = r - m * G;
  *((f32x4*)(O + ((int64_t)m * Hq + g * G + j) * DH) + c4) = acc * (1.0f / l);
}

// The V^T pre-pass (bf16), the kernels (fast path then fixup, or the f32 kernel) and,
// with split key ranges, the merge. p is complete (plan fields, buffers, Vt / Vts
// workspace pointers). KQ = 8 or 4 (bf16 only, no own entries): block-scaled K / V.
// A contiguous bf16 cache without bias or per-head counts, whose every row is an entry,
// needs no V^T tiles (nor do a chunk's own entries beside it): its kernels read V as
// stored (VNAT).
template <int DH, int KQ>
hipError_t run_attention(const AttnShape& s, const AttnPlan& pl, AttnParams& p, bool gather,
                         bool psplit, hipStream_t st) {
  if (KQ != 0 && (!s.bf16 || s.Ms > 0)) return hipErrorInvalidValue;
  const bool part = pl.n_split > 1;
  const bool own = s.Ms > 0;
  const bool bias = p.bias != nullptr;
  const bool vnat = KQ == 0 && s.bf16 && !gather && !bias && !p.counts && p.src_rows == p.Nk;
  dim3 grid(pl.grid), block(256);
  if (s.bf16) {
    const dim3 vg((unsigned)p.vt_tiles, (unsigned)s.Hkv);
    if (gather)
      hipLaunchKernelGGL((vt_kernel<DH, true, KQ>), vg, block, 0, st, p.V, p.Ve, p.idx,
                         p.idx_stride, p.counts, p.src_rows, p.Nk, p.vt_tiles, (__bf16*)p.Vt);
    else if (!vnat)
      hipLaunchKernelGGL((vt_kernel<DH, false, KQ>), vg, block, 0, st, p.V, p.Ve, p.idx,
                         p.idx_stride, p.counts, p.src_rows, p.Nk, p.vt_tiles, (__bf16*)p.Vt);
    if constexpr (KQ == 0) {
      if (own && !vnat) {  // V^T tiles of the chunk's own entries
        const dim3 og((unsigned)p.own_tiles, (unsigned)s.Hkv);
        hipLaunchKernelGGL((vt_kernel<DH, false, 0>), og, block, 0, st, p.Vs, nullptr, nullptr, 0,
                           nullptr, (int64_t)p.Ms, p.Ms, p.own_tiles, (__bf16*)p.Vts);
      }
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const dim3 bblock(kThreadsBf16);
    // fast path, then the lazy-rescale fixup for any work item it handed back
#define PKV_LB(G_, P_, S_, O_, B_)                                                                           \
  do {                                                                                                       \
    hipLaunchKernelGGL((attn_bf16_kernel<DH, G_, P_, S_, false, O_, B_, KQ, false>), grid, bblock, 0, st, p); \
    hipLaunchKernelGGL((attn_bf16_kernel<DH, G_, P_, S_, true, O_, B_, KQ, false>), grid, bblock, 0, st, p);  \
  } while (0)
#define PKV_LV(P_, S_, O_)                                                                                 \
  do {                                                                                                     \
    hipLaunchKernelGGL((attn_bf16_kernel<DH, false, P_, S_, false, O_, false, 0, true>), grid, bblock, 0, st, p); \
    hipLaunchKernelGGL((attn_bf16_kernel<DH, false, P_, S_, true, O_, false, 0, true>), grid, bblock, 0, st, p);  \
  } while (0)
#define PKV_L(G_, P_, S_, O_)                      \
  do {                                             \
    if (bias) PKV_LB(G_, P_, S_, false, true);     \
    else PKV_LB(G_, P_, S_, O_, false);            \
  } while (0)
    bool done = false;
    if constexpr (KQ == 0) {
      if (vnat) {
        done = true;
        if (own) {
          if (psplit) { if (part) PKV_LV(true, true, true); else PKV_LV(true, false, true); }
          else { if (part) PKV_LV(false, true, true); else PKV_LV(false, false, true); }
        } else {
          if (psplit) { if (part) PKV_LV(true, true, false); else PKV_LV(true, false, false); }
          else { if (part) PKV_LV(false, true, false); else PKV_LV(false, false, false); }
        }
      } else if (own) {
        done = true;
        if (gather) {
          if (psplit) { if (part) PKV_L(true, true, true, true); else PKV_L(true, true, false, true); }
          else { if (part) PKV_L(true, false, true, true); else PKV_L(true, false, false, true); }
        } else {
          if (psplit) { if (part) PKV_L(false, true, true, true); else PKV_L(false, true, false, true); }
          else { if (part) PKV_L(false, false, true, true); else PKV_L(false, false, false, true); }
        }
      }
    }
    if (done) {
    } else if (gather) {
      if (psplit) { if (part) PKV_L(true, true, true, false); else PKV_L(true, true, false, false); }
      else { if (part) PKV_L(true, false, true, false); else PKV_L(true, false, false, false); }
    } else {
      if (psplit) { if (part) PKV_L(false, true, true, false); else PKV_L(false, true, false, false); }
      else { if (part) PKV_L(false, false, true, false); else PKV_L(false, false, false, false); }
    }
#undef PKV_L
#undef PKV_LV
#undef PKV_LB
  } else if constexpr (KQ == 0) {
    const dim3 fblock(kF32Waves * 64);
#define PKV_L(G_, S_, O_)                                                                         \
  do {                                                                                            \
    if (bias) hipLaunchKernelGGL((attn_f32_kernel<DH, G_, S_, false, true>), grid, fblock, 0, st, p); \
    else hipLaunchKernelGGL((attn_f32_kernel<DH, G_, S_, O_, false>), grid, fblock, 0, st, p);       \
  } while (0)
    if (own) {
      if (gather) { if (part) PKV_L(true, true, true); else PKV_L(true, false, true); }
      else { if (part) PKV_L(false, true, true); else PKV_L(false, false, true); }
    }
    else if (gather) { if (part) PKV_L(true, true, false); else PKV_L(true, false, false); }
    else { if (part) PKV_L(false, true, false); else PKV_L(false, false, false); }
#undef PKV_L
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !part) return e;
  const int64_t total = (int64_t)s.Hkv * p.rows * (DH / 4);
  dim3 cg((unsigned)((total + 255) / 256));
  if (s.bf16)
    hipLaunchKernelGGL((attn_combine_kernel<DH, true>), cg, block, 0, st, p.Opart, p.ML, p.O,
                       p.rows, pl.n_split, s.Hkv, p.G, s.Hq);
  else
    hipLaunchKernelGGL((attn_combine_kernel<DH, false>), cg, block, 0, st, p.Opart, p.ML, p.O,
                       p.rows, pl.n_split, s.Hkv, p.G, s.Hq);
  return hipGetLastError();
}

}  // namespace

// Block-scaled integer caches (attention_mx.hip): run_attention<dh, bits>.
hipError_t run_attention_mx(const AttnShape& s, const AttnPlan& pl, AttnParams& p, int bits,
                            bool gather, bool psplit, hipStream_t st);

}  // namespace pkv
