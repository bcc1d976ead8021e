// Test hook of include/lipz_testing.h: one grouped-GEMM problem.
#include <string.h>

#include "lipz_internal.h"
#include "lipz_testing.h"

using namespace lipz;

extern "C" lipz_status lipz_test_gemm(void* hip_stream, void* d_desc, int32_t M, int32_t N,
                                      int32_t K, const float* d_A, int32_t lda, int32_t a_trans,
                                      int32_t ones_row, const float* d_B, int32_t ldb,
                                      int32_t b_trans, float* d_C, int32_t ldc, int32_t epi,
                                      int32_t act, float slope, const float* d_bias,
                                      const float* d_aux, float* d_m, float* d_v,
                                      const float* d_lr, const int32_t* d_t, int32_t step_local,
                                      float beta1, float beta2, float eps, int32_t tile_rows,
                                      int32_t variant) {
  static_assert(sizeof(GemmProb) <= 256, "the caller's descriptor scratch is 256 bytes");
  if (!d_desc || !d_A || !d_B || !d_C || M < 1 || N < 1 || K < 1) return LIPZ_E_INVAL;
  if (epi < EPI_STORE || epi > EPI_ADAM || act < LIPZ_ACT_LINEAR || act > LIPZ_ACT_TANH)
    return LIPZ_E_INVAL;
  if (ones_row >= 0 && (!a_trans || ones_row != M - 1)) return LIPZ_E_INVAL;
  if (epi == EPI_DACT && !d_aux) return LIPZ_E_INVAL;
  if (tile_rows != 0 && tile_rows != 32 && tile_rows != 64) return LIPZ_E_INVAL;
  if (variant < 0 || variant > 6 || (variant & 3) == 3) return LIPZ_E_INVAL;
  if (epi == EPI_ADAM && (!d_m || !d_v || !d_lr || !d_t)) return LIPZ_E_INVAL;
  const int a_rows = ones_row >= 0 ? ones_row : M;
  if (lda < (a_trans ? a_rows : K) || ldb < (b_trans ? K : N) || ldc < N) return LIPZ_E_INVAL;
  GemmProb p;
  memset(&p, 0, sizeof(p));
  p.A = d_A;
  p.B = d_B;
  p.C = d_C;
  p.bias = d_bias;
  p.aux = d_aux;
  p.m = d_m;
  p.v = d_v;
  p.lr = d_lr;
  p.t = d_t;
  p.M = M;
  p.N = N;
  p.K = K;
  p.lda = lda;
  p.ldb = ldb;
  p.ldc = ldc;
  p.a_trans = a_trans;
  p.b_trans = b_trans;
  p.a_rows = a_rows;
  p.ones_row = ones_row;
  p.epi = epi;
  p.act = act;
  p.vec = ((((uintptr_t)d_A & 15) == 0 && (lda & 3) == 0) ? 1 : 0) |
          ((((uintptr_t)d_B & 15) == 0 && (ldb & 3) == 0) ? 2 : 0);
  p.tiles_n = (N + GEMM_BN - 1) / GEMM_BN;
  p.tile_begin = 0;
  if (tile_rows == 0) tile_rows = gemm_tile_rows(((M + 63) / 64) * p.tiles_n);
  const int tiles = ((M + tile_rows - 1) / tile_rows) * p.tiles_n;
  p.slope = slope;
  p.ac.beta1 = beta1;
  p.ac.beta2 = beta2;
  p.ac.one_minus_beta1 = (float)(1.0 - (double)beta1);
  p.ac.one_minus_beta2 = (float)(1.0 - (double)beta2);
  p.ac.eps = eps;
  GemmGroups grp;
  memset(&grp, 0, sizeof(grp));
  grp.n = 1;
  grp.tiles_per_prob[0] = tiles;
  gemm_set_extents(p);
  if (hipMemcpy(d_desc, &p, sizeof(p), hipMemcpyHostToDevice) != hipSuccess) return LIPZ_E_HIP;
  // variant & 3 = 0: the kernel a phase of this one problem runs on; 1 / 2:
  // the register-staged or the wave-split kernel (aligned operands only);
  // variant & 4: write-back stores (else device-scope)
  const int kv = variant & 3;
  int kernel = gemm_choose_kernel(gemm_fast_ok(p), K);
  if (kv != 0) {
    if (!gemm_fast_ok(p)) return LIPZ_E_INVAL;
    kernel = kv == 1 ? GEMM_K_FAST : GEMM_K_WAVE;
  }
  if (launch_gemm_grouped((const GemmProb*)d_desc, grp, tiles, tile_rows, kernel, step_local, (variant & 4) == 0,
                          (hipStream_t)hip_stream) != hipSuccess)
    return LIPZ_E_HIP;
  return LIPZ_OK;
}

extern "C" lipz_status lipz_test_es_select(void* hip_stream, const float* d_fit, const float* d_sets,
                                           float* d_params, int32_t n_units, int32_t n_pairs, int64_t P,
                                           int64_t stride, float clip) {
  if (!d_fit || !d_sets || !d_params || n_units < 1 || n_units > 65535 || n_pairs < 1 || n_pairs > 64 || P < 1 ||
      stride < P || !(clip >= 0.f))
    return LIPZ_E_INVAL;
  NesArgs a;
  memset(&a, 0, sizeof(a));
  a.p = d_params;
  a.sets = (float*)d_sets;
  a.fit = (float*)d_fit;
  a.stride = stride;
  a.P = P;
  a.n = n_pairs;
  a.c0 = 0;
  a.C = n_units;
  a.clip = clip;
  return launch_es_select(a, (hipStream_t)hip_stream) == hipSuccess ? LIPZ_OK : LIPZ_E_HIP;
}

extern "C" lipz_status lipz_test_tile_map(int32_t n_groups, const int32_t* first_tile, int32_t n_blocks,
                                          int32_t* tiles) {
  if (n_groups < 1 || n_groups > lipz::GEMM_MAX_GROUPS || !first_tile || !tiles || n_blocks < 1 ||
      first_tile[0] != 0)
    return LIPZ_E_INVAL;
  lipz::GemmGroups grp{};
  grp.n = n_groups;
  for (int g = 0; g < n_groups; ++g) {
    if (g > 0 && first_tile[g] <= first_tile[g - 1]) return LIPZ_E_INVAL;
    if (first_tile[g] >= n_blocks) return LIPZ_E_INVAL;
    grp.first_tile[g] = first_tile[g];
  }
  for (int32_t b = 0; b < n_blocks; ++b) tiles[b] = lipz::xcd_group_tile(b, n_blocks, grp);
  return LIPZ_OK;
}
