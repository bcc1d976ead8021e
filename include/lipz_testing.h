/*
 * lipz_testing.h -- test hook of liblipz.so: runs the grouped fp32-MFMA GEMM
 * kernel that every generation phase uses on ONE problem, so the kernel can
 * be checked against a plain matrix product on ragged shapes.  Not needed to
 * run the method (include/lipz.h).
 *
 *   C(i,j) <- epilogue( sum_k A(i,k) B(k,j) ),  0 <= i < M, 0 <= j < N, 0 <= k < K
 *   A(i,k) = d_A[i*lda + k] (a_trans 0) or d_A[k*lda + i] (a_trans 1); with
 *            ones_row >= 0 (a_trans 1 only) A has ones_row data rows and row
 *            ones_row is all ones (appends a bias row to a weight gradient)
 *   B(k,j) = d_B[k*ldb + j] (b_trans 0) or d_B[j*ldb + k] (b_trans 1)
 *   epi 0: C = acc; 1: C = act(acc + bias[j]) (bias may be NULL);
 *   epi 2: C = acc * act'(aux[i*ldc + j]) with act' taken from the output
 *          value aux (relu: [aux > 0]; lrelu: 1 or slope; tanh: 1 - aux^2);
 *   epi 3: acc is the gradient of parameter C[i*ldc + j]: one bias-corrected
 *          Adam step with step count t = *d_t + step_local + 1 and learning
 *          rate *d_lr on C, d_m, d_v (same indexing as C).
 * tile_rows: 32 or 64 output rows per workgroup tile, 0 = the choice the
 * library makes for a phase of this size.  variant: 0 = the kernel the
 * library runs such a phase on; 1 = the register-staged LDS kernel, 2 = the
 * wave-split kernel (1-2 need 16-byte aligned operand rows, else
 * LIPZ_E_INVAL); plus 4: the kernel's write-back stores instead of its
 * device-scope ones (the store policy of grids whose state exceeds 128 MB;
 * the results are the same).  Other values: LIPZ_E_INVAL.
 * d_desc: device scratch of at least 256 bytes for the problem descriptor
 * (caller-owned).  The call copies the descriptor synchronously, enqueues the
 * kernel on hip_stream and returns; LIPZ_E_INVAL on bad sizes.
 */
#ifndef LIPZ_TESTING_H
#define LIPZ_TESTING_H

#include "lipz.h"

#ifdef __cplusplus
extern "C" {
#endif

lipz_status lipz_test_gemm(void* hip_stream, void* d_desc, int32_t M, int32_t N, int32_t K,
                           const float* d_A, int32_t lda, int32_t a_trans, int32_t ones_row,
                           const float* d_B, int32_t ldb, int32_t b_trans, float* d_C, int32_t ldc,
                           int32_t epi, int32_t act, float slope, const float* d_bias,
                           const float* d_aux, float* d_m, float* d_v, const float* d_lr,
                           const int32_t* d_t, int32_t step_local, float beta1, float beta2,
                           float eps, int32_t tile_rows, int32_t variant);

/*
 * Host-only check of a configuration's launch plan (no GPU, no device
 * memory): the library lays the plan out over placeholder addresses and
 * recomputes, for every GEMM, convolution, batch-norm, reduction and dot
 * descriptor, the first and last element each kernel can read or write,
 * using the kernels' own index formulas.  *n_bad = the number of accesses
 * that fall outside the workspace or the dataset; msg (msg_len bytes,
 * NUL-terminated, may be NULL) names the first of them.  LIPZ_E_INVAL for an
 * invalid configuration.
 */
lipz_status lipz_test_plan_bounds(const lipz_config* cfg, int64_t n_samples, char* msg, int32_t msg_len,
                                  int32_t* n_bad);

/*
 * The ES trainer's plus-selection (paper Section 3: gradient-free trainers;
 * the selection rule of the mixture step's (1+1)-ES) on caller-given losses:
 * for each of n_units units u, d_fit[u][0 .. 2n] holds the losses of the 2n
 * mutants and, last, of the parent.  The kept candidate is the first mutant
 * of lowest loss if that loss is strictly lower than the parent's, else the
 * parent; a NaN loss ranks as +infinity.  Its P values are written over
 * d_params[u][0 .. P) (row stride `stride` floats): mutant q's are
 * d_sets[(u * 2n + q) * stride ...], the parent's the row itself.  clip > 0
 * clips every kept value to [-clip, clip].  Device pointers, caller-owned;
 * enqueued on hip_stream; LIPZ_E_INVAL on bad sizes.
 */
lipz_status lipz_test_es_select(void* hip_stream, const float* d_fit, const float* d_sets, float* d_params,
                                int32_t n_units, int32_t n_pairs, int64_t P, int64_t stride, float clip);

/*
 * Host-only: the logical tile that each of the n_blocks workgroups of a
 * grouped GEMM launch computes (tiles[b] for block b), for a launch whose
 * n_groups (1..4) groups of problems start at tiles first_tile[0] = 0 <
 * first_tile[1] < ... < n_blocks.  The kernels dispatch block b to XCD b % 8
 * and give each XCD a contiguous chunk of every group.  Caller-owned host
 * arrays; LIPZ_E_INVAL on a bad group layout.
 */
lipz_status lipz_test_tile_map(int32_t n_groups, const int32_t* first_tile, int32_t n_blocks, int32_t* tiles);

#ifdef __cplusplus
}
#endif
#endif /* LIPZ_TESTING_H */
