// Grouped fp32 GEMM on CDNA4 matrix cores (v_mfma_f32_16x16x4f32) with fused
// epilogues.  One launch covers every (cell, slot) problem of one dependent
// phase of the generation: the per-cell networks of the grid are small
// (M = 100..600 rows, K = 64..784), so they are only worth a GPU when all of
// them run side by side.
//
// Tiling: a 256-thread workgroup (4 wave64) owns a 64x64 output tile; wave w
// owns the 32x32 quadrant (w / 2, w % 2) as 2x2 MFMA 16x16 accumulators.  The
// K loop stages 64x16 slices of A and 16x64 slices of B through LDS (k-major,
// padded rows), double-buffered in registers: the global loads of slice k+1
// are issued before the MFMAs of slice k.
//
// MFMA 16x16x4 f32 operand layout (wave64): lane l supplies A[l % 16][l / 16]
// and B[l / 16][l % 16]; accumulator register r of lane l is
// D[4 (l / 16) + r][l % 16].
#include "lipz_internal.h"

namespace lipz {

typedef float v4f __attribute__((ext_vector_type(4)));

namespace {

constexpr int BM = GEMM_BM;
constexpr int BN = GEMM_BN;
constexpr int BK = 16;
constexpr int LDS_STRIDE = BM + 16;  // 80 floats: the four k-rows a wave reads hit distinct banks
constexpr int NT = 256;

// Blocks are dispatched round-robin over the 8 XCDs (block b -> XCD b % 8).
// Give each XCD a contiguous range of logical tiles so that tiles of one
// problem (which share A rows and B columns) meet in the same L2.
__device__ __forceinline__ int xcd_remap(int b, int nb) {
  const int q = nb >> 3, r = nb & 7;
  const int x = b & 7, i = b >> 3;
  return x * q + (x < r ? x : r) + i;
}

struct Frag {
  float a[4];
  float b[4];
};

// Load this thread's share of the A and B slices starting at k0 into registers.
__device__ __forceinline__ void load_slices(const GemmProb& P, int m0, int n0, int k0, int tid,
                                            Frag& f) {
  // ---- A ----
  if (!P.a_trans) {
    const int row = tid >> 2, kq = (tid & 3) << 2;
    const int gm = m0 + row, gk = k0 + kq;
    if ((P.vec & 1) && gm < P.a_rows && gk + 3 < P.K) {
      const float4 v = *reinterpret_cast<const float4*>(P.A + (size_t)gm * P.lda + gk);
      f.a[0] = v.x; f.a[1] = v.y; f.a[2] = v.z; f.a[3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        f.a[e] = (gm < P.a_rows && gk + e < P.K) ? P.A[(size_t)gm * P.lda + gk + e] : 0.f;
    }
  } else {
    const int kk = tid >> 4, mq = (tid & 15) << 2;
    const int gk = k0 + kk, gm = m0 + mq;
    if ((P.vec & 1) && gk < P.K && gm + 3 < P.a_rows) {
      const float4 v = *reinterpret_cast<const float4*>(P.A + (size_t)gk * P.lda + gm);
      f.a[0] = v.x; f.a[1] = v.y; f.a[2] = v.z; f.a[3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int m = gm + e;
        float x = 0.f;
        if (gk < P.K) {
          if (m < P.a_rows) x = P.A[(size_t)gk * P.lda + m];
          else if (m == P.ones_row) x = 1.f;
        }
        f.a[e] = x;
      }
    }
  }
  // ---- B ----
  if (!P.b_trans) {
    const int kk = tid >> 4, nq = (tid & 15) << 2;
    const int gk = k0 + kk, gn = n0 + nq;
    if ((P.vec & 2) && gk < P.K && gn + 3 < P.N) {
      const float4 v = *reinterpret_cast<const float4*>(P.B + (size_t)gk * P.ldb + gn);
      f.b[0] = v.x; f.b[1] = v.y; f.b[2] = v.z; f.b[3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        f.b[e] = (gk < P.K && gn + e < P.N) ? P.B[(size_t)gk * P.ldb + gn + e] : 0.f;
    }
  } else {
    const int n = tid >> 2, kq = (tid & 3) << 2;
    const int gn = n0 + n, gk = k0 + kq;
    if ((P.vec & 2) && gn < P.N && gk + 3 < P.K) {
      const float4 v = *reinterpret_cast<const float4*>(P.B + (size_t)gn * P.ldb + gk);
      f.b[0] = v.x; f.b[1] = v.y; f.b[2] = v.z; f.b[3] = v.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        f.b[e] = (gn < P.N && gk + e < P.K) ? P.B[(size_t)gn * P.ldb + gk + e] : 0.f;
    }
  }
}

// Write the register slices to LDS in k-major order.
__device__ __forceinline__ void store_slices(const GemmProb& P, int tid, const Frag& f,
                                             float (*As)[LDS_STRIDE], float (*Bs)[LDS_STRIDE]) {
  if (!P.a_trans) {
    const int row = tid >> 2, kq = (tid & 3) << 2;
#pragma unroll
    for (int e = 0; e < 4; ++e) As[kq + e][row] = f.a[e];
  } else {
    const int kk = tid >> 4, mq = (tid & 15) << 2;
    *reinterpret_cast<float4*>(&As[kk][mq]) = make_float4(f.a[0], f.a[1], f.a[2], f.a[3]);
  }
  if (!P.b_trans) {
    const int kk = tid >> 4, nq = (tid & 15) << 2;
    *reinterpret_cast<float4*>(&Bs[kk][nq]) = make_float4(f.b[0], f.b[1], f.b[2], f.b[3]);
  } else {
    const int n = tid >> 2, kq = (tid & 3) << 2;
#pragma unroll
    for (int e = 0; e < 4; ++e) Bs[kq + e][n] = f.b[e];
  }
}

__global__ __launch_bounds__(NT) void gemm_grouped_kernel(const GemmProb* __restrict__ probs,
                                                          int nprob, int step_local, float slope,
                                                          AdamConsts ac) {
  const int t = xcd_remap(blockIdx.x, gridDim.x);
  int lo = 0, hi = nprob - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (probs[mid].tile_begin <= t) lo = mid; else hi = mid - 1;
  }
  const GemmProb P = probs[lo];
  const int lt = t - P.tile_begin;
  const int m0 = (lt / P.tiles_n) * BM;
  const int n0 = (lt % P.tiles_n) * BN;

  __shared__ float As[BK][LDS_STRIDE];
  __shared__ float Bs[BK][LDS_STRIDE];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = (wave >> 1) * 32, wn = (wave & 1) * 32;
  const int lr_ = lane & 15, lk = lane >> 4;

  v4f acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = v4f{0.f, 0.f, 0.f, 0.f};

  Frag f;
  load_slices(P, m0, n0, 0, tid, f);
  for (int k0 = 0; k0 < P.K; k0 += BK) {
    __syncthreads();
    store_slices(P, tid, f, As, Bs);
    __syncthreads();
    if (k0 + BK < P.K) load_slices(P, m0, n0, k0 + BK, tid, f);
#pragma unroll
    for (int kk = 0; kk < BK; kk += 4) {
      const float a0 = As[kk + lk][wm + lr_];
      const float a1 = As[kk + lk][wm + 16 + lr_];
      const float b0 = Bs[kk + lk][wn + lr_];
      const float b1 = Bs[kk + lk][wn + 16 + lr_];
      acc[0][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(a1, b1, acc[1][1], 0, 0, 0);
    }
  }

  // ---- epilogue ----
  float lr = 0.f, bc1 = 1.f, bc2 = 1.f;
  if (P.epi == EPI_ADAM) {
    lr = *P.lr;
    const int tt = *P.t + step_local + 1;
    bc1 = (float)(1.0 - pow((double)ac.beta1, (double)tt));
    bc2 = (float)(1.0 - pow((double)ac.beta2, (double)tt));
  }
#pragma unroll
  for (int i = 0; i < 2; ++i) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = n0 + wn + 16 * j + lr_;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = m0 + wm + 16 * i + 4 * lk + r;
        if (row >= P.M || col >= P.N) continue;
        float x = acc[i][j][r];
        const size_t o = (size_t)row * P.ldc + col;
        switch (P.epi) {
          case EPI_BIAS_ACT:
            if (P.bias) x += P.bias[col];
            P.C[o] = act_fwd(P.act, x, slope);
            break;
          case EPI_DACT:
            P.C[o] = x * act_deriv_from_out(P.act, P.aux[o], slope);
            break;
          case EPI_ADAM: {
            const float m = ac.beta1 * P.m[o] + ac.one_minus_beta1 * x;
            const float v = ac.beta2 * P.v[o] + ac.one_minus_beta2 * x * x;
            P.m[o] = m;
            P.v[o] = v;
            const float mhat = m / bc1, vhat = v / bc2;
            P.C[o] = P.C[o] - lr * mhat / (sqrtf(vhat) + ac.eps);
            break;
          }
          default:
            P.C[o] = x;
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm_grouped(const GemmProb* d_probs, int nprob, int total_tiles, int step_local,
                               float slope, AdamConsts ac, hipStream_t s) {
  if (nprob <= 0 || total_tiles <= 0) return hipSuccess;
  hipLaunchKernelGGL(gemm_grouped_kernel, dim3(total_tiles), dim3(NT), 0, s, d_probs, nprob,
                     step_local, slope, ac);
  return hipGetLastError();
}

}  // namespace lipz
