// Grouped fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_16x16x4f32) with fused
// epilogues.  One launch computes every (cell, slot) problem of one dependent
// phase of a generation: each cell's networks are small (M = 100..600 rows,
// K = 64..784), so they are only worth a GPU when all of them run side by side.
//
// Tiling: a 256-thread workgroup (4 wave64) owns a BM x 64 output tile
// (BM = 64 or 32, chosen per phase so that small phases still spread over the
// 256 CUs).  Wave w owns the (BM/2) x 32 block (w / 2, w % 2) as (BM/32) x 2
// MFMA 16x16 accumulators.  K advances in 64-deep slices through a
// double-buffered LDS ring: the global loads of slice k+1 are in flight while
// the MFMAs of slice k run, one barrier per slice.
//
// Each operand keeps its global layout in LDS (no transposing stores):
//   k-contiguous operands (A row-major, B = W^T) are read as 4 consecutive k
//   per lane with ds_read_b128; m/n-contiguous operands are read one k per
//   MFMA.  Within a 16-deep k block, MFMA sub-step s of lane group g = l / 16
//   uses k = 4 g + s for both operands, so the two layouts mix freely.  Row
//   strides are padded to 4 (mod 16) floats, which puts the four lane groups
//   of one read on disjoint LDS banks.
//
// MFMA 16x16x4 f32 operand layout (wave64): lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; accumulator register r of lane l is
// D[4 (l / 16) + r][l % 16].
#include "lipz_internal.h"

namespace lipz {

typedef float v4f __attribute__((ext_vector_type(4)));

namespace {

constexpr int BN = GEMM_BN;
constexpr int BK = 64;
constexpr int NT = 256;
constexpr int S_K = BK + 4;   // row stride of k-contiguous LDS tiles ([m][k], [n][k])

// Blocks are dispatched round-robin over the 8 XCDs (block b -> XCD b % 8).
// Give each XCD a contiguous range of logical tiles so that tiles of one
// problem (which share A rows and B columns) meet in the same L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, i = b >> 3;
  return x * q + (x < r ? x : r) + i;
}

template <int BM>
struct Tile {
  static constexpr int S_M = BM + 4;                        // row stride of [k][m] tiles
  static constexpr int S_N = BN + 4;                        // row stride of [k][n] tiles
  static constexpr int A_FLOATS = (BK * S_M > BM * S_K) ? BK * S_M : BM * S_K;
  static constexpr int B_FLOATS = BK * S_N;                 // == BN * S_K
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
    if (!P.a_trans) {  // [M][K]: row q / 16, k 4 (q % 16)
      const int gm = m0 + (q >> 4), gk = k0 + ((q & 15) << 2);
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
    } else {  // [N][K]: n q / 16, k 4 (q % 16)
      const int gn = n0 + (q >> 4), gk = k0 + ((q & 15) << 2);
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
    if (!P.a_trans) d = As + (q >> 4) * S_K + ((q & 15) << 2);
    else d = As + (q / (BM / 4)) * T::S_M + ((q % (BM / 4)) << 2);
    *reinterpret_cast<float4*>(d) = f.a[rep];
  }
#pragma unroll
  for (int rep = 0; rep < T::B_VEC; ++rep) {
    const int q = tid + NT * rep;
    float* d;
    if (!P.b_trans) d = Bs + (q >> 4) * T::S_N + ((q & 15) << 2);
    else d = Bs + (q >> 4) * S_K + ((q & 15) << 2);
    *reinterpret_cast<float4*>(d) = f.b[rep];
  }
}

// Epilogue shared by both kernel variants: bias + activation (optionally
// with the per-tile partial dot product of the next 1-wide layer), the
// activation-derivative product, or the fused Adam update; then stores.
template <int BM>
__device__ __forceinline__ void epilogue(const GemmProb& P, v4f (&acc)[Tile<BM>::TI][2], int m0, int n0,
                                         int tile_n, int step_local, float slope, const AdamConsts& ac,
                                         float (*red)[BM]) {
  using T = Tile<BM>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * T::WM, wn = (wave & 1) * 32;
  const int li = lane & 15, lg = lane >> 4;
  float lr = 0.f, bc1 = 1.f, bc2 = 1.f;
  if (P.epi == EPI_ADAM) {
    lr = *as_global(P.lr);
    const int tt = *as_global(P.t) + step_local + 1;
    bc1 = (float)(1.0 - pow((double)ac.beta1, (double)tt));
    bc2 = (float)(1.0 - pow((double)ac.beta2, (double)tt));
  }
  const bool dot = P.dot_out != nullptr;
  LIPZ_GLOBAL float* gC = as_global(P.C);
  LIPZ_GLOBAL float* gM = as_global(P.m);
  LIPZ_GLOBAL float* gV = as_global(P.v);
  const LIPZ_GLOBAL float* gBias = as_global(P.bias);
  const LIPZ_GLOBAL float* gAux = as_global(P.aux);
  const LIPZ_GLOBAL float* gDotw = as_global(P.dotw);
#pragma unroll
  for (int i = 0; i < T::TI; ++i) {
    float rowdot[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn + 16 * j + li;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + 16 * i + 4 * lg + r;
        if (row >= P.M || col >= P.N) continue;
        float x = acc[i][j][r];
        const size_t o = (size_t)row * P.ldc + col;
        switch (P.epi) {
          case EPI_BIAS_ACT: {
            if (P.bias) x += gBias[col];
            const float y = act_fwd(P.act, x, slope);
            gC[o] = y;
            if (dot) rowdot[r] += y * gDotw[col];
            break;
          }
          case EPI_DACT:
            gC[o] = x * act_deriv_from_out(P.act, gAux[o], slope);
            break;
          case EPI_ADAM: {
            const float m = ac.beta1 * gM[o] + ac.one_minus_beta1 * x;
            const float v = ac.beta2 * gV[o] + ac.one_minus_beta2 * x * x;
            gM[o] = m;
            gV[o] = v;
            const float mhat = m / bc1, vhat = v / bc2;
            gC[o] = gC[o] - lr * mhat / (sqrtf(vhat) + ac.eps);
            break;
          }
          default:
            gC[o] = x;
        }
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
    const float bias = (tile_n == 0 && P.dot_bias) ? *as_global(P.dot_bias) : 0.f;
    for (int r = tid; r < BM; r += NT) {
      const int row = m0 + r;
      if (row < P.M) as_global(P.dot_out)[(size_t)row * P.dot_ld + tile_n] = (red[0][r] + red[1][r]) + bias;
    }
  }
}

// Generic variant: any alignment, per-element bounds checks.  Used for
// phases whose rows are not 16-byte aligned (tiny widths such as 2-D data).
template <int BM>
__global__ __launch_bounds__(NT, 2) void gemm_generic_kernel(const GemmProb* __restrict__ probs,
                                                             GemmGroups grp, int step_local,
                                                             float slope, AdamConsts ac) {
  using T = Tile<BM>;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  int gi = 0;
#pragma unroll
  for (int q = 1; q < GEMM_MAX_GROUPS; ++q)
    if (q < grp.n && t >= grp.first_tile[q]) gi = q;
  const int rel = t - grp.first_tile[gi];
  const int pi = grp.first_prob[gi] + rel / grp.tiles_per_prob[gi];
  const int lt = rel % grp.tiles_per_prob[gi];
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

  epilogue<BM>(P, acc, m0, n0, tile_n, step_local, slope, ac, red);
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
    if (AT == 0) off = (uint32_t)((m0 + (q >> 4)) * P.lda + k0 + ((q & 15) << 2)) * 4u;
    else off = (uint32_t)((k0 + q / (BM / 4)) * P.lda + m0 + ((q % (BM / 4)) << 2)) * 4u;
    f.a[rep] = bload4(ra, off);
  }
#pragma unroll
  for (int rep = 0; rep < T::B_VEC; ++rep) {
    const int q = tid + NT * rep;
    uint32_t off;
    if (BT == 0) off = (uint32_t)((k0 + (q >> 4)) * P.ldb + n0 + ((q & 15) << 2)) * 4u;
    else off = (uint32_t)((n0 + (q >> 4)) * P.ldb + k0 + ((q & 15) << 2)) * 4u;
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
      const int kq = (q & 15) << 2;
      v.x = kq + 0 < kvalid ? v.x : 0.f;
      v.y = kq + 1 < kvalid ? v.y : 0.f;
      v.z = kq + 2 < kvalid ? v.z : 0.f;
      v.w = kq + 3 < kvalid ? v.w : 0.f;
      d = As + (q >> 4) * S_K + kq;
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
      const int kq = (q & 15) << 2;
      v.x = kq + 0 < kvalid ? v.x : 0.f;
      v.y = kq + 1 < kvalid ? v.y : 0.f;
      v.z = kq + 2 < kvalid ? v.z : 0.f;
      v.w = kq + 3 < kvalid ? v.w : 0.f;
      d = Bs + (q >> 4) * S_K + kq;
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
// start the loads of slice it + 2 into R, then the MFMAs of the slice with
// the LDS reads of k block kb + 1 issued ahead of the MFMAs of block kb.
template <int BM, int AT, int BT>
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
  if (it + 2 < n_it) fast_load<BM, AT, BT>(P, ra, rb, m0, n0, (it + 2) * BK, tid, R);
  Frag<BM> F0, F1;
  read_frag<BM, AT, BT>(as, bs, 0, wm, wn, li, lg, F0);
#pragma unroll
  for (int kb = 0; kb < BK / 16; kb += 2) {
    read_frag<BM, AT, BT>(as, bs, kb + 1, wm, wn, li, lg, F1);
    __builtin_amdgcn_sched_barrier(0);
    mfma_frag<BM>(F0, acc);
    __builtin_amdgcn_sched_barrier(0);
    if (kb + 2 < BK / 16) read_frag<BM, AT, BT>(as, bs, kb + 2, wm, wn, li, lg, F0);
    __builtin_amdgcn_sched_barrier(0);
    mfma_frag<BM>(F1, acc);
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int BM, int AT, int BT>
__device__ __forceinline__ void fast_mainloop(const GemmProb& P, int m0, int n0, float* As0,
                                              float* Bs0, v4f (&acc)[Tile<BM>::TI][2]) {
  using T = Tile<BM>;
  const int tid = threadIdx.x;
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(P.A, P.a_bytes);
  const __amdgpu_buffer_rsrc_t rb = make_rsrc(P.B, P.b_bytes);
  FastRegs<BM, AT, BT> R0, R1;
  const int n_it = (P.K + BK - 1) / BK;
  fast_load<BM, AT, BT>(P, ra, rb, m0, n0, 0, tid, R0);
  if (n_it > 1) fast_load<BM, AT, BT>(P, ra, rb, m0, n0, BK, tid, R1);
  // unrolled by two so that R0 / R1 and the LDS stages have fixed roles
  for (int it = 0; it < n_it; it += 2) {
    fast_slice<BM, AT, BT>(P, ra, rb, m0, n0, it, n_it, R0, As0, Bs0, acc);
    if (it + 1 < n_it)
      fast_slice<BM, AT, BT>(P, ra, rb, m0, n0, it + 1, n_it, R1, As0 + T::A_FLOATS,
                             Bs0 + T::B_FLOATS, acc);
  }
}

template <int BM>
__global__ __launch_bounds__(NT, 2) void gemm_fast_kernel(const GemmProb* __restrict__ probs,
                                                          GemmGroups grp, int step_local, float slope,
                                                          AdamConsts ac) {
  using T = Tile<BM>;
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  int gi = 0;
#pragma unroll
  for (int q = 1; q < GEMM_MAX_GROUPS; ++q)
    if (q < grp.n && t >= grp.first_tile[q]) gi = q;
  const int rel = t - grp.first_tile[gi];
  const int pi = grp.first_prob[gi] + rel / grp.tiles_per_prob[gi];
  const int lt = rel % grp.tiles_per_prob[gi];
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
  epilogue<BM>(P, acc, m0, n0, tile_n, step_local, slope, ac, red);
}
}  // namespace

int gemm_tile_rows(int tiles64) { return tiles64 < 512 ? 32 : 64; }

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

hipError_t launch_gemm_grouped(const GemmProb* d_probs, const GemmGroups& grp, int total_tiles,
                               int tile_rows, bool fast, int step_local, float slope, AdamConsts ac,
                               hipStream_t s) {
  if (grp.n <= 0 || total_tiles <= 0) return hipSuccess;
  const dim3 g(total_tiles), b(NT);
  if (fast) {
    if (tile_rows == 32)
      hipLaunchKernelGGL(gemm_fast_kernel<32>, g, b, 0, s, d_probs, grp, step_local, slope, ac);
    else
      hipLaunchKernelGGL(gemm_fast_kernel<64>, g, b, 0, s, d_probs, grp, step_local, slope, ac);
  } else {
    if (tile_rows == 32)
      hipLaunchKernelGGL(gemm_generic_kernel<32>, g, b, 0, s, d_probs, grp, step_local, slope, ac);
    else
      hipLaunchKernelGGL(gemm_generic_kernel<64>, g, b, 0, s, d_probs, grp, step_local, slope, ac);
  }
  return hipGetLastError();
}

}  // namespace lipz
