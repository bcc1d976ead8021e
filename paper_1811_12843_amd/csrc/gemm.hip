// Grouped fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_16x16x4f32) with fused
// epilogues.  One launch computes every (cell, slot) problem of one dependent
// phase of a generation: each cell's networks are small (M = 100..600 rows,
// K = 64..784), so they are only worth a GPU when all of them run side by side.
// Problems of one launch are described in device memory (GemmProb) and grouped
// by shape and depth (GemmGroups, passed as scalar kernel arguments that the
// hardware preloads); blockIdx is remapped so that each group is split into
// eight contiguous shares, one per XCD: the tiles of one problem share an L2
// and the long tiles of a launch are spread over every XCD.
//
// Stores: a template parameter WT selects device-scope (write-through) buffer
// stores for the epilogues' outputs, or write-back; the library picks one per
// grid, by the size of its state.
//
// Tiling: a 256-thread workgroup (4 wave64) owns a BM x 64 output tile
// (BM = 32 or 64).  Three kernels share the tile and the epilogue:
//
// * gemm_fast_kernel (16-byte aligned operands): wave w owns the (BM/2) x 32
//   block (w / 2, w % 2) as (BM/32) x 2 MFMA 16x16 accumulators.  K advances
//   in BK-deep slices through an LDS ring: buffer loads (bounded by the
//   operand's extent, so no branches on the edges) of the next slices are in
//   registers while the MFMAs of the current one run, one barrier per slice.
//   Each operand keeps its global layout in LDS (no transposing stores):
//   k-contiguous operands (A row-major, B = W^T) are read as 4 consecutive k
//   per lane with ds_read_b128; m/n-contiguous operands are read one k per
//   MFMA.  Within a 16-deep k block, MFMA sub-step s of lane group g = l / 16
//   uses k = 4 g + s for both operands, so the two layouts mix freely.  Row
//   strides are padded to 4 (mod 16) floats, which puts the four lane groups
//   of one read on disjoint LDS banks.
// * gemm_wave_kernel (deep K): split-K across the four waves, no LDS in the
//   main loop (described at its definition).
// * gemm_generic_kernel: any alignment, per-element bounds checks.
//
// Epilogues: plain store; bias + activation (forward), optionally with the
// tile's partial dot product against a 1-wide output layer; activation
// derivative (input gradient); Adam on the weight gradient in registers.
//
// MFMA 16x16x4 f32 operand layout (wave64): lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; accumulator register r of lane l is
// D[4 (l / 16) + r][l % 16].
#include <string.h>

#include <hip/hip_ext.h>

#include "lipz_internal.h"

namespace lipz {

typedef float v4f __attribute__((ext_vector_type(4)));

namespace {

#ifndef LIPZ_GEMM_STAGES
#define LIPZ_GEMM_STAGES 2      // slices of A/B loads in flight per workgroup
#endif
#ifndef LIPZ_GEMM_WG32
#define LIPZ_GEMM_WG32 4        // occupancy target of the fast kernel, 32-row tiles
#endif
#ifndef LIPZ_GEMM_WG64
#define LIPZ_GEMM_WG64 2        // occupancy target of the fast kernel, 64-row tiles
#endif
#ifndef LIPZ_GEMM_TILE64_MIN
#define LIPZ_GEMM_TILE64_MIN 100000  // phases with at least this many 64x64 tiles use 64-row tiles
#endif

#ifndef LIPZ_GEMM_BK
#define LIPZ_GEMM_BK 32         // K depth of one LDS slice
#endif
#ifndef LIPZ_GEMM_WAVE_SPLIT
#define LIPZ_GEMM_WAVE_SPLIT 1  // allow the wave-split (split-K in the workgroup) kernel
#endif
#ifndef LIPZ_GEMM_WAVE_MIN_K
#define LIPZ_GEMM_WAVE_MIN_K 512  // ... for phases whose deepest problem has K >= this
#endif

constexpr int BN = GEMM_BN;
constexpr int BK = LIPZ_GEMM_BK;
constexpr int KQ = BK / 4;    // float4 per row of a k-contiguous slice
constexpr int NT = 256;
constexpr int S_K = BK + 4;   // row stride of k-contiguous LDS tiles ([m][k], [n][k])


template <int BM>
struct Tile {
  static constexpr int S_M = BM + 4;                        // row stride of [k][m] tiles
  static constexpr int S_N = BN + 4;                        // row stride of [k][n] tiles
  static constexpr int A_FLOATS = (BK * S_M > BM * S_K) ? BK * S_M : BM * S_K;
  static constexpr int B_FLOATS = (BK * S_N > BN * S_K) ? BK * S_N : BN * S_K;
  static constexpr int A_VEC = BM * BK / 4 / NT;            // float4 of A per thread per slice
  static constexpr int B_VEC = BN * BK / 4 / NT;
  static constexpr int WM = BM / 2;                         // rows per wave
  static constexpr int TI = WM / 16;                        // accumulator tiles along M per wave
};

template <int BM>
struct Regs {
  float4 a[Tile<BM>::A_VEC];
  float4 b[Tile<BM>::B_VEC];
};

__device__ __forceinline__ float4 ld4(const LIPZ_GLOBAL float* p) {
  const v4f v = *reinterpret_cast<const LIPZ_GLOBAL v4f*>(p);
  return make_float4(v[0], v[1], v[2], v[3]);
}

// Global -> registers: this thread's share of the A and B slices at k0.
template <int BM>
__device__ __forceinline__ void load_slices(const GemmProb& P, int m0, int n0, int k0, int tid,
                                            Regs<BM>& f) {
  using T = Tile<BM>;
  const LIPZ_GLOBAL float* gA = as_global(P.A);
  const LIPZ_GLOBAL float* gB = as_global(P.B);
#pragma unroll
  for (int rep = 0; rep < T::A_VEC; ++rep) {
    const int q = tid + NT * rep;
    float4 v;
    if (!P.a_trans) {  // [M][K]: row q / KQ, k 4 (q % KQ)
      const int gm = m0 + q / KQ, gk = k0 + ((q % KQ) << 2);
      if ((P.vec & 1) && gm < P.a_rows && gk + 3 < P.K) {
        v = ld4(gA + (size_t)gm * P.lda + gk);
      } else {
        const bool r = gm < P.a_rows;
        const LIPZ_GLOBAL float* s = gA + (size_t)gm * P.lda;
        v.x = (r && gk + 0 < P.K) ? s[gk + 0] : 0.f;
        v.y = (r && gk + 1 < P.K) ? s[gk + 1] : 0.f;
        v.z = (r && gk + 2 < P.K) ? s[gk + 2] : 0.f;
        v.w = (r && gk + 3 < P.K) ? s[gk + 3] : 0.f;
      }
    } else {  // [K][M]: k q / (BM/4), m 4 (q % (BM/4))
      constexpr int PER_K = BM / 4;
      const int gk = k0 + q / PER_K, gm = m0 + ((q % PER_K) << 2);
      if ((P.vec & 1) && gk < P.K && gm + 3 < P.a_rows) {
        v = ld4(gA + (size_t)gk * P.lda + gm);
      } else {
        float e[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int m = gm + u;
          float x = 0.f;
          if (gk < P.K) {
            if (m < P.a_rows) x = gA[(size_t)gk * P.lda + m];
            else if (m == P.ones_row) x = 1.f;
          }
          e[u] = x;
        }
        v = make_float4(e[0], e[1], e[2], e[3]);
      }
    }
    f.a[rep] = v;
  }
#pragma unroll
  for (int rep = 0; rep < T::B_VEC; ++rep) {
    const int q = tid + NT * rep;
    float4 v;
    if (!P.b_trans) {  // [K][N]: k q / 16, n 4 (q % 16)
      const int gk = k0 + (q >> 4), gn = n0 + ((q & 15) << 2);
      if ((P.vec & 2) && gk < P.K && gn + 3 < P.N) {
        v = ld4(gB + (size_t)gk * P.ldb + gn);
      } else {
        const bool r = gk < P.K;
        const LIPZ_GLOBAL float* s = gB + (size_t)gk * P.ldb;
        v.x = (r && gn + 0 < P.N) ? s[gn + 0] : 0.f;
        v.y = (r && gn + 1 < P.N) ? s[gn + 1] : 0.f;
        v.z = (r && gn + 2 < P.N) ? s[gn + 2] : 0.f;
        v.w = (r && gn + 3 < P.N) ? s[gn + 3] : 0.f;
      }
    } else {  // [N][K]: n q / KQ, k 4 (q % KQ)
      const int gn = n0 + q / KQ, gk = k0 + ((q % KQ) << 2);
      if ((P.vec & 2) && gn < P.N && gk + 3 < P.K) {
        v = ld4(gB + (size_t)gn * P.ldb + gk);
      } else {
        const bool r = gn < P.N;
        const LIPZ_GLOBAL float* s = gB + (size_t)gn * P.ldb;
        v.x = (r && gk + 0 < P.K) ? s[gk + 0] : 0.f;
        v.y = (r && gk + 1 < P.K) ? s[gk + 1] : 0.f;
        v.z = (r && gk + 2 < P.K) ? s[gk + 2] : 0.f;
        v.w = (r && gk + 3 < P.K) ? s[gk + 3] : 0.f;
      }
    }
    f.b[rep] = v;
  }
}

// Registers -> LDS, in the operand's own layout.
template <int BM>
__device__ __forceinline__ void store_slices(const GemmProb& P, int tid, const Regs<BM>& f, float* As,
                                             float* Bs) {
  using T = Tile<BM>;
#pragma unroll
  for (int rep = 0; rep < T::A_VEC; ++rep) {
    const int q = tid + NT * rep;
    float* d;
    if (!P.a_trans) d = As + (q / KQ) * S_K + ((q % KQ) << 2);
    else d = As + (q / (BM / 4)) * T::S_M + ((q % (BM / 4)) << 2);
    *reinterpret_cast<float4*>(d) = f.a[rep];
  }
#pragma unroll
  for (int rep = 0; rep < T::B_VEC; ++rep) {
    const int q = tid + NT * rep;
    float* d;
    if (!P.b_trans) d = Bs + (q >> 4) * T::S_N + ((q & 15) << 2);
    else d = Bs + (q / KQ) * S_K + ((q % KQ) << 2);
    *reinterpret_cast<float4*>(d) = f.b[rep];
  }
}

typedef unsigned int v4u __attribute__((ext_vector_type(4)));

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float* p, uint32_t bytes) {
  // dword 3 = 0x00020000: raw 32-bit data format on gfx9-family parts
  return __builtin_amdgcn_make_buffer_rsrc((void*)p, (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ float4 bload4(__amdgpu_buffer_rsrc_t r, uint32_t off_bytes) {
  const v4u v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off_bytes, 0, 0);
  return make_float4(__uint_as_float(v[0]), __uint_as_float(v[1]), __uint_as_float(v[2]),
                     __uint_as_float(v[3]));
}


// One element through a buffer resource: the epilogues address C, the Adam
// moments and the auxiliary operand with 32-bit element offsets from the
// descriptor's base (no 64-bit address per element).
//
// Store policy (WT, a template parameter of the kernels, chosen per grid).
// With WT the epilogues' element stores (outputs, Adam's p, m, v), the head
// partials and the minibatch rows are device-scope stores (cache policy
// sc1): written through the XCD's L2 towards memory, so that the next
// dependent launch, which reads them from whichever XCD its tiles run on,
// does not wait for an end-of-kernel writeback of dirty L2 lines.  Without
// it they are write-back stores.  (The folded loss head's per-row side
// outputs and partial dot products are write-back stores in either case.)
constexpr uint32_t kWholeBuffer = 0x7FFFFFFFu;  // element offsets of a problem stay below 2^31 (planning checks)
constexpr int kStoreDevice = 16;                // buffer-store cache policy: sc1 (device scope)
__device__ __forceinline__ float bld1(__amdgpu_buffer_rsrc_t r, uint32_t off_elems) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)(off_elems * 4u), 0, 0));
}
template <bool WT>
__device__ __forceinline__ void bst1(__amdgpu_buffer_rsrc_t r, uint32_t off_elems, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)(off_elems * 4u), 0, WT ? kStoreDevice : 0);
}

// The loss head's dL/da of this lane's epilogue rows (rows m0 + wm + 16 i +
// 4 (lane / 16) + r), from the partial logits, formed as the separate head
// kernel forms it.  With four partial sums per row (a 129..256-wide last
// hidden layer) the loads are issued together with the epilogue's other
// loads, so they add no round trip.
template <int BM>
__device__ __forceinline__ void head_rows_dl(const GemmProb& P, int m0, float (&dl)[Tile<BM>::TI][4]) {
  using T = Tile<BM>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * T::WM, lg = lane >> 4;
  const float invB = 1.f / (float)P.rs_B;
#pragma unroll
  for (int i = 0; i < T::TI; ++i) {
    // lane r of each 16-lane group forms row r's value, then the group shares them
    const int row = m0 + wm + 16 * i + 4 * lg + (lane & 3);
    const LIPZ_GLOBAL float* pr = as_global(P.rs_part) + (size_t)(row < P.M ? row : 0) * P.rs_tn;
    float a;
    if (P.rs_tn == 4) {  // a 129..256-wide last hidden layer: the row's four partial sums in one load
      const float4 v = ld4(pr);
      a = ((v.x + v.y) + v.z) + v.w;
    } else {
      a = 0.f;
      for (int t = 0; t < P.rs_tn; ++t) a += pr[t];
    }
    const float mine = head_dl(P.loss_kind, a, P.rs_mode == 2 || row < P.rs_B, invB);
#pragma unroll
    for (int r = 0; r < 4; ++r) dl[i][r] = __shfl(mine, (lane & ~15) | r, 64);
  }
}

// Workgroup q of a sampling job: SAMPLE_ROWS minibatch rows of one unit,
// drawn exactly as sample_kernel draws them.
template <bool WT>
__device__ __forceinline__ void sample_rows(const SampleJob& sj, int q) {
  const int per = (sj.B + SAMPLE_ROWS - 1) / SAMPLE_ROWS;
  const int u = sj.u0 + q / per, b0 = (q % per) * SAMPLE_ROWS;
  const int nr = sj.B - b0 < SAMPLE_ROWS ? sj.B - b0 : SAMPLE_ROWS;
  const int tid = threadIdx.x;
  for (int rr = 0; rr < nr; ++rr) {
    const int b = b0 + rr;
    const uint4 wi = stream_block(sj.key, (uint32_t)(b >> 2), (uint32_t)u, sj.gen, sj.sf, LIPZ_TAG_IDX);
    const int64_t row = (int64_t)(((uint64_t)word_of(wi, b & 3) * (uint64_t)sj.N) >> 32);
    const float* src = sj.data + row * sj.xd;
    const __amdgpu_buffer_rsrc_t rd = make_rsrc(sj.X + u * sj.x_stride + (int64_t)b * sj.xd, kWholeBuffer);
    if ((sj.xd & 3) == 0) {
      for (int k = tid; k < (sj.xd >> 2); k += NT) {
        const float4 v = reinterpret_cast<const float4*>(src)[k];
        __builtin_amdgcn_raw_buffer_store_b128(
            v4u{__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)}, rd,
            k * 16, 0, WT ? kStoreDevice : 0);
      }
    } else {
      for (int k = tid; k < sj.xd; k += NT) bst1<WT>(rd, (uint32_t)k, src[k]);
    }
  }
  const __amdgpu_buffer_rsrc_t rz = make_rsrc(sj.Z + u * sj.z_stride + (int64_t)b0 * sj.zd, kWholeBuffer);
  for (int k = tid; k < nr * sj.zd; k += NT) {
    const int64_t e = (int64_t)b0 * sj.zd + k;
    const uint4 w = stream_block(sj.key, (uint32_t)(e >> 2), (uint32_t)u, sj.gen, sj.sf, LIPZ_TAG_Z);
    bst1<WT>(rz, (uint32_t)k, (float)normal_of(w, (int)(e & 3)));
  }
}

// The output layer's weight gradient of the discriminator step, in pieces:
// this tile's column sums of dL/da[i] * hsrc[i][j] over its rows (and, in
// column 0, of dL/da[i]), summed over the lane groups and then over the two
// waves that share the tile's columns, in a fixed order.  Rows past M and
// columns past hp_w add nothing.
template <int BM, bool WT>
__device__ __forceinline__ void head_partials(const GemmProb& P, const float (&dl)[Tile<BM>::TI][4], int m0,
                                              int n0, int tile_n, float (*red)[BM]) {
  using T = Tile<BM>;
  __shared__ float dsum;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * T::WM, wn = (wave & 1) * 32;
  const int li = lane & 15, lg = lane >> 4;
  const bool wgan = P.loss_kind == LIPZ_LOSS_WASSERSTEIN;
  const __amdgpu_buffer_rsrc_t rH = make_rsrc(P.hsrc, kWholeBuffer);
  float hv[T::TI][2][4];
#pragma unroll
  for (int i = 0; i < T::TI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + 16 * i + 4 * lg + r, col = n0 + wn + 16 * j + li;
        const bool in = row < P.M && col < P.hp_w;
        const float x = bld1(rH, in ? (uint32_t)(row * P.hp_w + col) : 0u);
        hv[i][j][r] = in ? x : 0.f;
      }
  float cs[2] = {0.f, 0.f}, ds = 0.f;
#pragma unroll
  for (int i = 0; i < T::TI; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = m0 + wm + 16 * i + 4 * lg + r;
      const float d = row < P.M ? (wgan ? (row < P.rs_B ? -1.f : 1.f) : dl[i][r]) : 0.f;
      ds += d;
#pragma unroll
      for (int j = 0; j < 2; ++j) cs[j] += d * hv[i][j][r];
    }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    cs[j] += __shfl_xor(cs[j], 16, 64);
    cs[j] += __shfl_xor(cs[j], 32, 64);
  }
  ds += __shfl_xor(ds, 16, 64);
  ds += __shfl_xor(ds, 32, 64);
  if (wm != 0 && lane < 16) {
    red[wave & 1][li] = cs[0];
    red[wave & 1][16 + li] = cs[1];
    if (wn == 0 && lane == 0) dsum = ds;
  }
  __syncthreads();
  if (wm == 0 && lane < 16) {
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(P.hpart + (size_t)(m0 / BM) * P.hp_ld, kWholeBuffer);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn + 16 * j + li;
      if (col < P.hp_w) bst1<WT>(ro, (uint32_t)col, cs[j] + red[wave & 1][16 * j + li]);
    }
    if (tile_n == 0 && wn == 0 && lane == 0) bst1<WT>(ro, (uint32_t)P.hp_w, ds + dsum);
  }
}

// Kernel arguments of the three GEMM kernels.  The descriptor pointer, the
// tile groups of the launch and the step index come first, as 14 scalar
// words that the hardware preloads into scalar registers (the library is
// built with -mllvm -amdgpu-kernarg-preload-count=14), so that a GEMM
// workgroup's first memory access is its problem descriptor; only the
// sampling workgroups read their SampleJob from kernel-argument memory.
// Group q of the launch: tiles first_tile[q] .. (first_tile[q + 1] or
// total) - 1, problems first_prob[q] on, tiles_per_prob[q] tiles each;
// first_tile[0] = first_prob[0] = 0, and a group past the launch's last one
// has first_tile = total.
#define LIPZ_GEMM_ARGS                                                                              \
  const GemmProb *__restrict__ probs, int32_t g_total, int32_t g_ft1, int32_t g_ft2, int32_t g_ft3, \
      int32_t g_fp1, int32_t g_fp2, int32_t g_fp3, int32_t g_tp0, int32_t g_tp1, int32_t g_tp2,     \
      int32_t g_tp3, int32_t step_local, SampleJob sj
#define LIPZ_GEMM_GROUPS g_total, g_ft1, g_ft2, g_ft3, g_fp1, g_fp2, g_fp3, g_tp0, g_tp1, g_tp2, g_tp3

// This workgroup's problem (index pi into the launch's descriptors) and tile
// of it (lt), from the XCD-balanced block-to-tile map.  No array is indexed
// at run time, so the groups stay in scalar registers.
__device__ __forceinline__ void locate_tile(int total, int ft1, int ft2, int ft3, int fp1, int fp2, int fp3, int tp0,
                                            int tp1, int tp2, int tp3, int& pi, int& lt) {
  GemmGroups grp;
  grp.n = 1 + (ft1 < total) + (ft2 < total) + (ft3 < total);
  grp.total = total;
  grp.first_tile[0] = 0;
  grp.first_tile[1] = ft1;
  grp.first_tile[2] = ft2;
  grp.first_tile[3] = ft3;
  const int t = xcd_group_tile(blockIdx.x, total, grp);
  int ft = 0, fp = 0, tp = tp0;
  if (t >= ft1) ft = ft1, fp = fp1, tp = tp1;
  if (t >= ft2) ft = ft2, fp = fp2, tp = tp2;
  if (t >= ft3) ft = ft3, fp = fp3, tp = tp3;
  pi = fp + (t - ft) / tp;
  lt = (t - ft) % tp;
}

// Epilogue shared by both kernel variants: bias + activation (optionally
// with the per-tile partial dot product of the next 1-wide layer), the
// activation-derivative product, or the fused Adam update; then stores.
// All of a lane's loads are issued before any of them is used, so their
// latencies overlap (out-of-range elements read element 0 and are dropped).
template <int BM, bool WT>
__device__ __forceinline__ void epilogue(const GemmProb& P, v4f (&acc)[Tile<BM>::TI][2], int m0, int n0,
                                         int tile_n, int step_local, float (*red)[BM]) {
  using T = Tile<BM>;
  constexpr int NE = T::TI * 2 * 4;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * T::WM, wn = (wave & 1) * 32;
  const int li = lane & 15, lg = lane >> 4;
  const float slope = P.slope;
  const __amdgpu_buffer_rsrc_t rC = make_rsrc(P.C, kWholeBuffer);
  uint32_t off[NE];
  bool ok[NE];
#pragma unroll
  for (int i = 0; i < T::TI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = (i * 2 + j) * 4 + r;
        const int row = m0 + wm + 16 * i + 4 * lg + r;
        const int col = n0 + wn + 16 * j + li;
        ok[e] = row < P.M && col < P.N;
        off[e] = ok[e] ? (uint32_t)(row * P.ldc + col) : 0u;
      }
  if (P.epi == EPI_ADAM) {
    const AdamConsts& ac = P.ac;
    const __amdgpu_buffer_rsrc_t rM = make_rsrc(P.m, kWholeBuffer);
    const __amdgpu_buffer_rsrc_t rV = make_rsrc(P.v, kWholeBuffer);
    const float lr = *as_global(P.lr);
    const int tt = *as_global(P.t) + step_local + 1;
    const float bc1 = (float)(1.0 - pow((double)ac.beta1, (double)tt));
    const float bc2 = (float)(1.0 - pow((double)ac.beta2, (double)tt));
    float pp[NE], mm[NE], vv[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) {
      pp[e] = bld1(rC, off[e]);
      mm[e] = bld1(rM, off[e]);
      vv[e] = bld1(rV, off[e]);
    }
#pragma unroll
    for (int i = 0; i < T::TI; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = (i * 2 + j) * 4 + r;
          const float g = P.gscale != 0.f ? acc[i][j][r] * P.gscale : acc[i][j][r];
          const float m = ac.beta1 * mm[e] + ac.one_minus_beta1 * g;
          const float v = ac.beta2 * vv[e] + ac.one_minus_beta2 * g * g;
          float p = pp[e] - lr * (m / bc1) / (sqrtf(v / bc2) + ac.eps);
          if (P.clip > 0.f) p = p > P.clip ? P.clip : (p < -P.clip ? -P.clip : p);  // keeps NaN
          if (ok[e]) {
            bst1<WT>(rM, off[e], m);
            bst1<WT>(rV, off[e], v);
            bst1<WT>(rC, off[e], p);
          }
        }
    return;
  }
  if (P.epi == EPI_DACT) {
    const __amdgpu_buffer_rsrc_t rAux = make_rsrc(P.aux, kWholeBuffer);
    float ax[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) ax[e] = bld1(rAux, off[e]);
    if (P.rs_mode == 0) {
#pragma unroll
      for (int i = 0; i < T::TI; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int e = (i * 2 + j) * 4 + r;
            if (ok[e]) bst1<WT>(rC, off[e], acc[i][j][r] * act_deriv_from_out(P.act, ax[e], slope));
          }
      return;
    }
    float dl[T::TI][4];
    head_rows_dl<BM>(P, m0, dl);
    LIPZ_GLOBAL float* gSide = as_global(P.side);
#pragma unroll
    for (int i = 0; i < T::TI; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = (i * 2 + j) * 4 + r;
          if (ok[e]) {
            bst1<WT>(rC, off[e], dl[i][r] * (acc[i][j][r] * act_deriv_from_out(P.act, ax[e], slope)));
            if (P.side) {
              const int row = m0 + wm + 16 * i + 4 * lg + r, col = n0 + wn + 16 * j + li;
              gSide[(size_t)row * P.side_ld + col] = dl[i][r] * ax[e];
            }
          }
        }
    if (P.rs_mode == 1 && P.hpart) head_partials<BM, WT>(P, dl, m0, n0, tile_n, red);
    // column 0 of the problem: the per-row extras
    if (P.side && tile_n == 0 && wn == 0 && li == 0) {
      LIPZ_GLOBAL float* gDl = as_global(P.dlout);
#pragma unroll
      for (int i = 0; i < T::TI; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int row = m0 + wm + 16 * i + 4 * lg + r;
          if (row < P.M) {
            LIPZ_GLOBAL float* sr = gSide + (size_t)row * P.side_ld + P.N;
            sr[0] = dl[i][r];
            sr[1] = 0.f;
            sr[2] = 0.f;
            sr[3] = 0.f;
            LIPZ_GLOBAL float* o = gDl + (size_t)row * 4;
            o[0] = P.loss_kind == LIPZ_LOSS_WASSERSTEIN ? (row < P.rs_B ? -1.f : 1.f) : dl[i][r];
            o[1] = 0.f;
            o[2] = 0.f;
            o[3] = 0.f;
          }
        }
    }
    return;
  }
  if (P.epi != EPI_BIAS_ACT) {
#pragma unroll
    for (int i = 0; i < T::TI; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int e = (i * 2 + j) * 4 + r;
          if (ok[e]) bst1<WT>(rC, off[e], acc[i][j][r]);
        }
    return;
  }
  // bias + activation, optional partial dot product with the next layer's weights
  const bool dot = P.dot_out != nullptr;
  float bias[2] = {0.f, 0.f}, dw[2] = {0.f, 0.f};
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int col = n0 + wn + 16 * j + li;
    const int c = col < P.N ? col : 0;
    if (P.bias) bias[j] = as_global(P.bias)[c];
    if (dot) dw[j] = col < P.N ? as_global(P.dotw)[c] : 0.f;
  }
#pragma unroll
  for (int i = 0; i < T::TI; ++i) {
    float rowdot[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int e = (i * 2 + j) * 4 + r;
        const float y = act_fwd(P.act, acc[i][j][r] + bias[j], slope);
        if (ok[e]) {
          bst1<WT>(rC, off[e], y);
          rowdot[r] += y * dw[j];
          if (P.gout) bst1<WT>(make_rsrc(P.gout, kWholeBuffer), off[e], dw[j] * act_deriv_from_out(P.act, y, slope));
        }
      }
    if (dot) {
      // sum over the 16 lanes that hold one row's columns, then over the two
      // column halves of the tile (waves wn = 0 and 32) in a fixed order
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float v = rowdot[r];
        v += __shfl_xor(v, 1, 64);
        v += __shfl_xor(v, 2, 64);
        v += __shfl_xor(v, 4, 64);
        v += __shfl_xor(v, 8, 64);
        rowdot[r] = v;
      }
      if (li == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) red[wave & 1][wm + 16 * i + 4 * lg + r] = rowdot[r];
      }
    }
  }
  if (dot) {
    __syncthreads();
    const float b = (tile_n == 0 && P.dot_bias) ? *as_global(P.dot_bias) : 0.f;
    for (int r = tid; r < BM; r += NT) {
      const int row = m0 + r;
      if (row < P.M) as_global(P.dot_out)[(size_t)row * P.dot_ld + tile_n] = (red[0][r] + red[1][r]) + b;
    }
  }
}

// Generic variant: any alignment, per-element bounds checks.  Used for
// phases whose rows are not 16-byte aligned (tiny widths such as 2-D data).
template <int BM, bool WT>
__global__ __launch_bounds__(NT, 2) void gemm_generic_kernel(LIPZ_GEMM_ARGS) {
  using T = Tile<BM>;
  if ((int)blockIdx.x >= g_total) {
    sample_rows<WT>(sj, (int)blockIdx.x - g_total);
    return;
  }
  int pi, lt;
  locate_tile(LIPZ_GEMM_GROUPS, pi, lt);
  const GemmProb P = probs[pi];
  const int tile_n = lt % P.tiles_n;
  const int m0 = (lt / P.tiles_n) * BM;
  const int n0 = tile_n * BN;

  __shared__ __align__(16) float As[2][T::A_FLOATS];
  __shared__ __align__(16) float Bs[2][T::B_FLOATS];
  __shared__ float red[2][BM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * T::WM, wn = (wave & 1) * 32;
  const int li = lane & 15, lg = lane >> 4;

  v4f acc[T::TI][2];
#pragma unroll
  for (int i = 0; i < T::TI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  Regs<BM> f;
  const int n_it = (P.K + BK - 1) / BK;
  load_slices<BM>(P, m0, n0, 0, tid, f);
  store_slices<BM>(P, tid, f, As[0], Bs[0]);
  __syncthreads();
  for (int it = 0; it < n_it; ++it) {
    const int s = it & 1;
    if (it + 1 < n_it) load_slices<BM>(P, m0, n0, (it + 1) * BK, tid, f);
    const float* as = As[s];
    const float* bs = Bs[s];
#pragma unroll
    for (int kb = 0; kb < BK; kb += 16) {
      float a[T::TI][4], b[2][4];
      const int kq = kb + 4 * lg;  // this lane group's 4 k values: kq .. kq + 3
#pragma unroll
      for (int i = 0; i < T::TI; ++i) {
        const int m = wm + 16 * i + li;
        if (!P.a_trans) {
          const float4 v = *reinterpret_cast<const float4*>(as + m * S_K + kq);
          a[i][0] = v.x; a[i][1] = v.y; a[i][2] = v.z; a[i][3] = v.w;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) a[i][u] = as[(kq + u) * T::S_M + m];
        }
      }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int n = wn + 16 * j + li;
        if (P.b_trans) {
          const float4 v = *reinterpret_cast<const float4*>(bs + n * S_K + kq);
          b[j][0] = v.x; b[j][1] = v.y; b[j][2] = v.z; b[j][3] = v.w;
        } else {
#pragma unroll
          for (int u = 0; u < 4; ++u) b[j][u] = bs[(kq + u) * T::S_N + n];
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int i = 0; i < T::TI; ++i) {
          acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][u], b[0][u], acc[i][0], 0, 0, 0);
          acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][u], b[1][u], acc[i][1], 0, 0, 0);
        }
    }
    if (it + 1 < n_it) store_slices<BM>(P, tid, f, As[s ^ 1], Bs[s ^ 1]);
    __syncthreads();
  }

  epilogue<BM, WT>(P, acc, m0, n0, tile_n, step_local, red);
}

// ---------------------------------------------------------------------------
// Fast variant: every operand row 16-byte aligned, each operand's extent in
// the descriptor.  Loads are buffer loads bounded by that extent (reads
// past it return 0), so the main loop has no per-element bounds branches;
// the operand layouts are template parameters chosen once per workgroup.
// The K tail of the last slice and the bias "ones" row are set by selects
// when the slice is written to LDS.  Loads run two slices ahead of the
// MFMAs (two register sets, two LDS stages, one barrier per slice).
// ---------------------------------------------------------------------------
template <int BM, int AT, int BT>
struct FastRegs {
  float4 a[Tile<BM>::A_VEC];
  float4 b[Tile<BM>::B_VEC];
};

template <int BM, int AT, int BT>
__device__ __forceinline__ void fast_load(const GemmProb& P, __amdgpu_buffer_rsrc_t ra,
                                          __amdgpu_buffer_rsrc_t rb, int m0, int n0, int k0, int tid,
                                          FastRegs<BM, AT, BT>& f) {
  using T = Tile<BM>;
#pragma unroll
  for (int rep = 0; rep < T::A_VEC; ++rep) {
    const int q = tid + NT * rep;
    uint32_t off;
    if (AT == 0) off = (uint32_t)((m0 + q / KQ) * P.lda + k0 + ((q % KQ) << 2)) * 4u;
    else off = (uint32_t)((k0 + q / (BM / 4)) * P.lda + m0 + ((q % (BM / 4)) << 2)) * 4u;
    f.a[rep] = bload4(ra, off);
  }
#pragma unroll
  for (int rep = 0; rep < T::B_VEC; ++rep) {
    const int q = tid + NT * rep;
    uint32_t off;
    if (BT == 0) off = (uint32_t)((k0 + (q >> 4)) * P.ldb + n0 + ((q & 15) << 2)) * 4u;
    else off = (uint32_t)((n0 + q / KQ) * P.ldb + k0 + ((q % KQ) << 2)) * 4u;
    f.b[rep] = bload4(rb, off);
  }
}

// Registers -> LDS with the K tail (k >= kvalid) zeroed and, for a [K][M]
// operand, rows past a_rows zeroed except the ones row.
template <int BM, int AT, int BT>
__device__ __forceinline__ void fast_store(const GemmProb& P, int m0, int kvalid, int tid,
                                           const FastRegs<BM, AT, BT>& f, float* As, float* Bs) {
  using T = Tile<BM>;
#pragma unroll
  for (int rep = 0; rep < T::A_VEC; ++rep) {
    const int q = tid + NT * rep;
    float4 v = f.a[rep];
    float* d;
    if (AT == 0) {
      const int kq = (q % KQ) << 2;
      v.x = kq + 0 < kvalid ? v.x : 0.f;
      v.y = kq + 1 < kvalid ? v.y : 0.f;
      v.z = kq + 2 < kvalid ? v.z : 0.f;
      v.w = kq + 3 < kvalid ? v.w : 0.f;
      d = As + (q / KQ) * S_K + kq;
    } else {
      const int kk = q / (BM / 4), mq = (q % (BM / 4)) << 2;
      const bool kok = kk < kvalid;
      const int gm = m0 + mq;
      const float one = kok ? 1.f : 0.f;
      v.x = gm + 0 < P.a_rows ? (kok ? v.x : 0.f) : (gm + 0 == P.ones_row ? one : 0.f);
      v.y = gm + 1 < P.a_rows ? (kok ? v.y : 0.f) : (gm + 1 == P.ones_row ? one : 0.f);
      v.z = gm + 2 < P.a_rows ? (kok ? v.z : 0.f) : (gm + 2 == P.ones_row ? one : 0.f);
      v.w = gm + 3 < P.a_rows ? (kok ? v.w : 0.f) : (gm + 3 == P.ones_row ? one : 0.f);
      d = As + kk * T::S_M + mq;
    }
    *reinterpret_cast<float4*>(d) = v;
  }
#pragma unroll
  for (int rep = 0; rep < T::B_VEC; ++rep) {
    const int q = tid + NT * rep;
    float4 v = f.b[rep];
    float* d;
    if (BT == 0) {
      const int kk = q >> 4;
      if (kk >= kvalid) v = make_float4(0.f, 0.f, 0.f, 0.f);
      d = Bs + kk * T::S_N + ((q & 15) << 2);
    } else {
      const int kq = (q % KQ) << 2;
      v.x = kq + 0 < kvalid ? v.x : 0.f;
      v.y = kq + 1 < kvalid ? v.y : 0.f;
      v.z = kq + 2 < kvalid ? v.z : 0.f;
      v.w = kq + 3 < kvalid ? v.w : 0.f;
      d = Bs + (q / KQ) * S_K + kq;
    }
    *reinterpret_cast<float4*>(d) = v;
  }
}

template <int BM>
struct Frag {
  float a[Tile<BM>::TI][4];
  float b[2][4];
};

// MFMA fragments of one 16-deep k block kb of the slice in LDS.
template <int BM, int AT, int BT>
__device__ __forceinline__ void read_frag(const float* as, const float* bs, int kb, int wm, int wn,
                                          int li, int lg, Frag<BM>& F) {
  using T = Tile<BM>;
  const int kq = 16 * kb + 4 * lg;
#pragma unroll
  for (int i = 0; i < T::TI; ++i) {
    const int m = wm + 16 * i + li;
    if (AT == 0) {
      const float4 v = *reinterpret_cast<const float4*>(as + m * S_K + kq);
      F.a[i][0] = v.x; F.a[i][1] = v.y; F.a[i][2] = v.z; F.a[i][3] = v.w;
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) F.a[i][u] = as[(kq + u) * T::S_M + m];
    }
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = wn + 16 * j + li;
    if (BT == 1) {
      const float4 v = *reinterpret_cast<const float4*>(bs + n * S_K + kq);
      F.b[j][0] = v.x; F.b[j][1] = v.y; F.b[j][2] = v.z; F.b[j][3] = v.w;
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) F.b[j][u] = bs[(kq + u) * T::S_N + n];
    }
  }
}

template <int BM>
__device__ __forceinline__ void mfma_frag(const Frag<BM>& F, v4f (&acc)[Tile<BM>::TI][2]) {
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int i = 0; i < Tile<BM>::TI; ++i) {
      acc[i][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(F.a[i][u], F.b[0][u], acc[i][0], 0, 0, 0);
      acc[i][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(F.a[i][u], F.b[1][u], acc[i][1], 0, 0, 0);
    }
}

// One slice: write registers R (slice it) to LDS stage (as, bs), barrier,
// start the loads of slice it + NS into R, then the MFMAs of the slice's two
// 16-deep k blocks, with the LDS reads of the second block issued ahead of
// the MFMAs of the first.
template <int BM, int AT, int BT, int NS, bool LOAD_ALWAYS>
__device__ __forceinline__ void fast_slice(const GemmProb& P, __amdgpu_buffer_rsrc_t ra,
                                           __amdgpu_buffer_rsrc_t rb, int m0, int n0, int it, int n_it,
                                           FastRegs<BM, AT, BT>& R, float* as, float* bs,
                                           v4f (&acc)[Tile<BM>::TI][2]) {
  using T = Tile<BM>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * T::WM, wn = (wave & 1) * 32;
  const int li = lane & 15, lg = lane >> 4;
  fast_store<BM, AT, BT>(P, m0, P.K - it * BK, tid, R, as, bs);
  __syncthreads();
  if (LOAD_ALWAYS || it + NS < n_it) fast_load<BM, AT, BT>(P, ra, rb, m0, n0, (it + NS) * BK, tid, R);
  // A wave whose rows all lie past M, or a 16-deep k block wholly past K
  // (zeros in both operands), has no MFMA work: skip it (wave-uniform).
  static_assert(BK == 32, "the k-block skip is written for two 16-deep blocks per slice");
  if (m0 + wm >= P.M) return;
  const bool two = P.K - it * BK > 16;
  Frag<BM> F0, F1;
  read_frag<BM, AT, BT>(as, bs, 0, wm, wn, li, lg, F0);
  if (two) read_frag<BM, AT, BT>(as, bs, 1, wm, wn, li, lg, F1);
  __builtin_amdgcn_sched_barrier(0);
  mfma_frag<BM>(F0, acc);
  __builtin_amdgcn_sched_barrier(0);
  if (two) mfma_frag<BM>(F1, acc);
  __builtin_amdgcn_sched_barrier(0);
}

// K loop: NS register sets hold the loads of the next NS slices; the loop is
// unrolled by NS so each set (and each of the two LDS stages) has a fixed
// role.  Its steady state issues every prefetch without a branch, so the
// compiler counts the outstanding loads exactly and a slice's stores wait
// for that slice's loads only (with a branch around the prefetch, the stores
// also waited for the loads of the slices after it).
template <int BM, int AT, int BT>
__device__ __forceinline__ void fast_mainloop(const GemmProb& P, int m0, int n0, float* As0,
                                              float* Bs0, v4f (&acc)[Tile<BM>::TI][2]) {
  using T = Tile<BM>;
  constexpr int NS = LIPZ_GEMM_STAGES;
  static_assert(NS % 2 == 0, "an even number of register stages maps onto the two LDS stages");
  const int tid = threadIdx.x;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(P.A, P.a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(P.B, P.b_bytes);
  FastRegs<BM, AT, BT> R[NS];
  const int n_it = (P.K + BK - 1) / BK;
  // the first NS slices' loads, all issued (past K they read zeros or
  // data the K-tail selects drop), so that the steady-state loop below
  // starts from the same outstanding loads on every path
#pragma unroll
  for (int s = 0; s < NS; ++s) fast_load<BM, AT, BT>(P, ra, rb, m0, n0, s * BK, tid, R[s]);
  int it = 0;
  // steady state: every slice's prefetch is needed, no branch on the loads,
  // so each store waits for its own slice's loads and no later ones
  for (; it + 2 * NS <= n_it; it += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      fast_slice<BM, AT, BT, NS, true>(P, ra, rb, m0, n0, it + s, n_it, R[s], As0 + (s & 1) * T::A_FLOATS,
                                       Bs0 + (s & 1) * T::B_FLOATS, acc);
  }
  // the last NS .. 2 NS - 1 slices
  for (; it < n_it; it += NS) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      if (it + s < n_it)
        fast_slice<BM, AT, BT, NS, false>(P, ra, rb, m0, n0, it + s, n_it, R[s], As0 + (s & 1) * T::A_FLOATS,
                                          Bs0 + (s & 1) * T::B_FLOATS, acc);
  }
}

template <int BM, bool WT>
__global__ __launch_bounds__(NT, BM == 32 ? LIPZ_GEMM_WG32 : LIPZ_GEMM_WG64) void gemm_fast_kernel(LIPZ_GEMM_ARGS) {
  using T = Tile<BM>;
  if ((int)blockIdx.x >= g_total) {
    sample_rows<WT>(sj, (int)blockIdx.x - g_total);
    return;
  }
  int pi, lt;
  locate_tile(LIPZ_GEMM_GROUPS, pi, lt);
  const GemmProb P = probs[pi];
  const int tile_n = lt % P.tiles_n;
  const int m0 = (lt / P.tiles_n) * BM;
  const int n0 = tile_n * BN;

  __shared__ __align__(16) float As[2 * T::A_FLOATS];
  __shared__ __align__(16) float Bs[2 * T::B_FLOATS];
  __shared__ float red[2][BM];

  v4f acc[T::TI][2];
#pragma unroll
  for (int i = 0; i < T::TI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  if (P.a_trans) fast_mainloop<BM, 1, 0>(P, m0, n0, As, Bs, acc);
  else if (P.b_trans) fast_mainloop<BM, 0, 1>(P, m0, n0, As, Bs, acc);
  else fast_mainloop<BM, 0, 0>(P, m0, n0, As, Bs, acc);
  epilogue<BM, WT>(P, acc, m0, n0, tile_n, step_local, red);
}

// ---------------------------------------------------------------------------
// Wave-split variant: the four waves of a workgroup each compute the whole
// BM x 64 tile over every fourth 16-deep k block (split-K inside the
// workgroup).  Each wave streams its operands from global memory (L2)
// straight into registers in the MFMA fragment layout, PD k blocks ahead of
// its MFMAs, so the main loop has no LDS traffic and no barriers, and a
// tile's dependent chain is a quarter of K.  No operand element is loaded
// twice, exactly as with an LDS-shared tile.  At the end the four partial
// tiles are summed through LDS in a fixed order and handed to the shared
// epilogue.
// ---------------------------------------------------------------------------
#ifndef LIPZ_WAVE_PD
#define LIPZ_WAVE_PD 2
#endif

template <int BM>
struct WFrag {
  float a[BM / 16][4];   // A rows 16 i + (l % 16), k = kb + 4 (l / 16) + s
  float b[4][4];         // B cols 16 j + (l % 16), same k
};

template <int BM, int AT, int BT>
__device__ __forceinline__ void wave_load(const GemmProb& P, __amdgpu_buffer_rsrc_t ra,
                                          __amdgpu_buffer_rsrc_t rb, int m0, int n0, int kb, int li,
                                          int lg, WFrag<BM>& F) {
  const int k = kb + 4 * lg;
#pragma unroll
  for (int i = 0; i < BM / 16; ++i) {
    const int m = m0 + 16 * i + li;
    if (AT == 0) {
      const float4 v = bload4(ra, (uint32_t)(m * P.lda + k) * 4u);
      F.a[i][0] = v.x; F.a[i][1] = v.y; F.a[i][2] = v.z; F.a[i][3] = v.w;
    } else {
#pragma unroll
      for (int s = 0; s < 4; ++s)
        F.a[i][s] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(ra, (int)((uint32_t)((k + s) * P.lda + m) * 4u), 0, 0));
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int n = n0 + 16 * j + li;
    if (BT == 1) {
      const float4 v = bload4(rb, (uint32_t)(n * P.ldb + k) * 4u);
      F.b[j][0] = v.x; F.b[j][1] = v.y; F.b[j][2] = v.z; F.b[j][3] = v.w;
    } else {
#pragma unroll
      for (int s = 0; s < 4; ++s)
        F.b[j][s] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rb, (int)((uint32_t)((k + s) * P.ldb + n) * 4u), 0, 0));
    }
  }
}

// MFMAs of one k block.  TAIL: zero k >= K (the problem's last, partial
// block).  ONES: the tile holds the bias row of a [K][M] operand: set row
// ones_row to 1 (0 past K) and the other rows past a_rows to 0.
template <int BM, bool TAIL, bool ONES>
__device__ __forceinline__ void wave_mma(const GemmProb& P, int m0, int kb, int li, int lg, WFrag<BM>& F,
                                         v4f (&acc)[BM / 16][4]) {
  const int k = kb + 4 * lg;
  if (TAIL) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const bool ok = k + s < P.K;
#pragma unroll
      for (int i = 0; i < BM / 16; ++i) F.a[i][s] = ok ? F.a[i][s] : 0.f;
#pragma unroll
      for (int j = 0; j < 4; ++j) F.b[j][s] = ok ? F.b[j][s] : 0.f;
    }
  }
  if (ONES) {
#pragma unroll
    for (int i = 0; i < BM / 16; ++i) {
      const int m = m0 + 16 * i + li;
#pragma unroll
      for (int s = 0; s < 4; ++s) {
        const float one = (TAIL && k + s >= P.K) ? 0.f : 1.f;
        F.a[i][s] = m < P.a_rows ? F.a[i][s] : (m == P.ones_row ? one : 0.f);
      }
    }
  }
  // a 16-row block wholly past M has no MFMA work (uniform); each
  // accumulator still takes its four k steps in order
#pragma unroll
  for (int i = 0; i < BM / 16; ++i)
    if (i == 0 || m0 + 16 * i < P.M)
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(F.a[i][s], F.b[j][s], acc[i][j], 0, 0, 0);
}

template <int BM, int AT, int BT, bool ONES>
__device__ __forceinline__ void wave_mainloop(const GemmProb& P, int m0, int n0, v4f (&acc)[BM / 16][4]) {
  constexpr int PD = LIPZ_WAVE_PD;
  // the wave index is uniform across the wave: keep it (and every k-block
  // index and loop bound derived from it) in scalar registers
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, lg = lane >> 4;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(P.A, P.a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(P.B, P.b_bytes);
  const int nkb = (P.K + 15) / 16;                          // k blocks of the problem
  const int mine = nkb > wave ? (nkb - wave + 3) / 4 : 0;   // blocks wave, wave + 4, ...
  WFrag<BM> F[PD];
  // every prologue load issued (past the wave's blocks they read zeros or
  // values no MFMA uses), so that the steady-state loop below starts from
  // the same outstanding loads on every path
#pragma unroll
  for (int p = 0; p < PD; ++p) wave_load<BM, AT, BT>(P, ra, rb, m0, n0, 16 * (wave + 4 * p), li, lg, F[p]);
  // steady state: every block full, every prefetch needed, no branches on
  // the loads, so the compiler can count outstanding loads exactly
  int q = 0;
  for (; q + 2 * PD <= mine; q += PD) {
#pragma unroll
    for (int p = 0; p < PD; ++p) {
      wave_mma<BM, false, ONES>(P, m0, 16 * (wave + 4 * (q + p)), li, lg, F[p], acc);
      wave_load<BM, AT, BT>(P, ra, rb, m0, n0, 16 * (wave + 4 * (q + p + PD)), li, lg, F[p]);
    }
  }
  // drain: the last PD .. 2 PD - 1 blocks, the problem's partial block among them
  for (; q < mine; q += PD) {
#pragma unroll
    for (int p = 0; p < PD; ++p) {
      if (q + p < mine) {
        const int kb = 16 * (wave + 4 * (q + p));
        if (kb + 16 > P.K) wave_mma<BM, true, ONES>(P, m0, kb, li, lg, F[p], acc);
        else wave_mma<BM, false, ONES>(P, m0, kb, li, lg, F[p], acc);
        if (q + p + PD < mine)
          wave_load<BM, AT, BT>(P, ra, rb, m0, n0, 16 * (wave + 4 * (q + p + PD)), li, lg, F[p]);
      }
    }
  }
}

template <int BM, bool WT>
__global__ __launch_bounds__(NT, BM == 32 ? 2 : 1) void gemm_wave_kernel(LIPZ_GEMM_ARGS) {
  using T = Tile<BM>;
  constexpr int RS = BN + 4;  // row stride of the partial tiles in LDS
  if ((int)blockIdx.x >= g_total) {
    sample_rows<WT>(sj, (int)blockIdx.x - g_total);
    return;
  }
  int pi, lt;
  locate_tile(LIPZ_GEMM_GROUPS, pi, lt);
  const GemmProb P = probs[pi];
  const int tile_n = lt % P.tiles_n;
  const int m0 = (lt / P.tiles_n) * BM;
  const int n0 = tile_n * BN;

  __shared__ __align__(16) float part[4][BM * RS];
  __shared__ float red[2][BM];

  v4f pacc[BM / 16][4];
#pragma unroll
  for (int i = 0; i < BM / 16; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) pacc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};
  if (P.a_trans) {
    if (m0 + BM > P.a_rows) wave_mainloop<BM, 1, 0, true>(P, m0, n0, pacc);
    else wave_mainloop<BM, 1, 0, false>(P, m0, n0, pacc);
  } else if (P.b_trans) {
    wave_mainloop<BM, 0, 1, false>(P, m0, n0, pacc);
  } else {
    wave_mainloop<BM, 0, 0, false>(P, m0, n0, pacc);
  }

  // partial tiles to LDS (MFMA D layout: row 16 i + 4 (l / 16) + r, col 16 j + l % 16)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int li = lane & 15, lg = lane >> 4;
  float* mine = part[wave];
#pragma unroll
  for (int i = 0; i < BM / 16; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) mine[(16 * i + 4 * lg + r) * RS + 16 * j + li] = pacc[i][j][r];
  __syncthreads();
  // each wave takes its quadrant of the tile in the layout the epilogue expects
  const int wm = (wave >> 1) * T::WM, wn = (wave & 1) * 32;
  v4f acc[T::TI][2];
#pragma unroll
  for (int i = 0; i < T::TI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int o = (wm + 16 * i + 4 * lg + r) * RS + wn + 16 * j + li;
        acc[i][j][r] = (part[0][o] + part[1][o]) + (part[2][o] + part[3][o]);
      }
  epilogue<BM, WT>(P, acc, m0, n0, tile_n, step_local, red);
}

}  // namespace

int gemm_tile_rows(int tiles64) { return tiles64 < LIPZ_GEMM_TILE64_MIN ? 32 : 64; }

void gemm_set_extents(GemmProb& p) {
  const uint64_t a = (uint64_t)(p.a_trans ? p.K : p.a_rows) * (uint64_t)p.lda * 4u;
  const uint64_t b = (uint64_t)(p.b_trans ? p.N : p.K) * (uint64_t)p.ldb * 4u;
  p.a_bytes = a < 0x7FFFFFF0u ? (uint32_t)a : 0u;
  p.b_bytes = b < 0x7FFFFFF0u ? (uint32_t)b : 0u;
}

bool gemm_fast_ok(const GemmProb& p) {
  // the fast kernel instantiates the three operand layouts the library uses:
  // (A, B) = (row, row) forward, (row, W^T) input gradient, (X^T, row) weight gradient
  return !(p.a_trans && p.b_trans) && p.vec == 3 && p.a_bytes > 0 && p.b_bytes > 0 && p.a_bytes < 0x7FFFFFF0u &&
         p.b_bytes < 0x7FFFFFF0u;
}

bool gemm_wave_ok(int max_k) { return LIPZ_GEMM_WAVE_SPLIT && max_k >= LIPZ_GEMM_WAVE_MIN_K; }

hipError_t launch_gemm_grouped(const GemmProb* d_probs, const GemmGroups& grp, int total_tiles,
                               int tile_rows, int kernel, int step_local, bool write_through, hipStream_t s,
                               hipEvent_t ev_start, hipEvent_t ev_stop, const SampleJob* job) {
  if (grp.n <= 0 || total_tiles <= 0) return hipSuccess;
  SampleJob sj;
  memset(&sj, 0, sizeof(sj));
  if (job) sj = *job;
  // the groups as the kernels take them (see LIPZ_GEMM_ARGS)
  if (grp.n > GEMM_MAX_GROUPS || grp.first_tile[0] != 0 || grp.first_prob[0] != 0) return hipErrorInvalidValue;
  int ft[GEMM_MAX_GROUPS], fp[GEMM_MAX_GROUPS];
  for (int q = 0; q < GEMM_MAX_GROUPS; ++q) {
    ft[q] = q < grp.n ? grp.first_tile[q] : total_tiles;
    fp[q] = q < grp.n ? grp.first_prob[q] : 0;
    if (q > 0 && q < grp.n && !(ft[q - 1] < ft[q] && ft[q] < total_tiles)) return hipErrorInvalidValue;
  }
  const dim3 g(total_tiles + sj.blocks), b(NT);
  // the events (may be null) are stamped by the kernel's own dispatch packet,
  // so their difference is the kernel's execution time alone
#define LIPZ_LAUNCH(K)                                                                                          \
  hipExtLaunchKernelGGL(K, g, b, 0, s, ev_start, ev_stop, 0, d_probs, total_tiles, ft[1], ft[2], ft[3], fp[1], \
                        fp[2], fp[3], grp.tiles_per_prob[0], grp.tiles_per_prob[1], grp.tiles_per_prob[2],    \
                        grp.tiles_per_prob[3], step_local, sj)
#define LIPZ_LAUNCH_WT(KN, BMV) \
  if (write_through) LIPZ_LAUNCH((KN<BMV, true>)); else LIPZ_LAUNCH((KN<BMV, false>))
  const bool r32 = tile_rows == 32;
  switch (kernel) {
    case GEMM_K_WAVE:
      if (r32) { LIPZ_LAUNCH_WT(gemm_wave_kernel, 32); } else { LIPZ_LAUNCH_WT(gemm_wave_kernel, 64); }
      break;
    case GEMM_K_FAST:
      if (r32) { LIPZ_LAUNCH_WT(gemm_fast_kernel, 32); } else { LIPZ_LAUNCH_WT(gemm_fast_kernel, 64); }
      break;
    default:
      if (r32) { LIPZ_LAUNCH_WT(gemm_generic_kernel, 32); } else { LIPZ_LAUNCH_WT(gemm_generic_kernel, 64); }
  }
#undef LIPZ_LAUNCH_WT
#undef LIPZ_LAUNCH
  return hipGetLastError();
}

int gemm_choose_kernel(bool fast, int max_k) {
  if (!fast) return GEMM_K_GENERIC;
  return gemm_wave_ok(max_k) ? GEMM_K_WAVE : GEMM_K_FAST;
}

}  // namespace lipz
