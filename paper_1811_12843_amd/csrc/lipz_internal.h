// Internal declarations shared by the HIP kernels and the host runtime of
// liblipz.so.  Not part of the public interface (include/lipz.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "lipz.h"

namespace lipz {

// Pointers read from a descriptor in memory have no known address space, so
// the compiler would access them with flat instructions, which share the
// LDS wait counter and serialise a prefetch behind every LDS read.  Device
// code casts them to the global address space before use.
#define LIPZ_GLOBAL __attribute__((address_space(1)))
template <class T>
__device__ __forceinline__ LIPZ_GLOBAL T* as_global(T* p) {
  return (LIPZ_GLOBAL T*)p;
}

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC 2011): ten rounds of
//   (c0,c1,c2,c3) -> (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0))
// with the key advanced by the Weyl constants between rounds.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint2 k) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k.x += 0x9E3779B9u;
      k.y += 0xBB67AE85u;
    }
    const uint32_t hi0 = __umulhi(0xD2511F53u, c.x), lo0 = 0xD2511F53u * c.x;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c.z), lo1 = 0xCD9E8D57u * c.z;
    c = make_uint4(hi1 ^ c.y ^ k.x, lo1, hi0 ^ c.w ^ k.y, lo0);
  }
  return c;
}

// Word `e % 4` of block e / 4 of the stream (cell, gen, step_field, tag).
__device__ __forceinline__ uint4 stream_block(uint2 key, uint32_t blk, uint32_t cell, uint32_t gen,
                                              uint32_t step_field, uint32_t tag) {
  return philox4x32_10(make_uint4(blk, cell, (gen << 16) | step_field, tag), key);
}

__device__ __forceinline__ uint32_t word_of(uint4 w, int i) {
  return i == 0 ? w.x : i == 1 ? w.y : i == 2 ? w.z : w.w;
}

// ((w >> 9) + 0.5) * 2^-23: exact in fp32, in (0, 1).
__device__ __forceinline__ double uniform_of(uint32_t w) {
  return ((double)(w >> 9) + 0.5) * (1.0 / 8388608.0);
}

// Normal number q (0..3) of a block by Box-Muller on (u0, u1) and (u2, u3), in fp64.
__device__ __forceinline__ double normal_of(uint4 w, int q) {
  const double ua = uniform_of(q < 2 ? w.x : w.z);
  const double ub = uniform_of(q < 2 ? w.y : w.w);
  const double r = sqrt(-2.0 * log(ua));
  double s, c;
  sincos(2.0 * 3.141592653589793 * ub, &s, &c);
  return (q & 1) ? r * s : r * c;
}

// ---------------------------------------------------------------------------
// Activations (LIPZ_ACT_*) and their derivatives expressed through the output
// y = act(x): relu' = [y > 0], lrelu' = [y > 0] + slope [y <= 0], tanh' = 1 - y^2.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float act_fwd(int act, float x, float slope) {
  switch (act) {
    case 1: return x > 0.f ? x : 0.f;
    case 2: return x > 0.f ? x : slope * x;
    case 3: return tanhf(x);
    default: return x;
  }
}
__device__ __forceinline__ float act_deriv_from_out(int act, float y, float slope) {
  switch (act) {
    case 1: return y > 0.f ? 1.f : 0.f;
    case 2: return y > 0.f ? 1.f : slope;
    case 3: return 1.f - y * y;
    default: return 1.f;
  }
}
// softplus(x) = log(1 + e^x), stable form.
__device__ __forceinline__ float softplus_f(float x) {
  return fmaxf(x, 0.f) + log1pf(expf(-fabsf(x)));
}
__device__ __forceinline__ float sigmoid_f(float x) { return 1.f / (1.f + expf(-x)); }
// Per-row loss terms of a logit / critic output a, for a row whose target is
// "real" (data rows in the D step; every row of the G step) or "fake".
// BCE: softplus(-a) and softplus(a); Wasserstein: -a and a.
__device__ __forceinline__ float real_term(int loss_kind, float a) {
  return loss_kind == LIPZ_LOSS_WASSERSTEIN ? -a : softplus_f(-a);
}
__device__ __forceinline__ float fake_term(int loss_kind, float a) {
  return loss_kind == LIPZ_LOSS_WASSERSTEIN ? a : softplus_f(a);
}
// dL/da of one row (the mean over B rows included): BCE (sigmoid(a) - target) / B;
// Wasserstein -1 / B for a real target, +1 / B for a fake one.
__device__ __forceinline__ float head_dl(int loss_kind, float a, bool real_target, float invB) {
  if (loss_kind == LIPZ_LOSS_WASSERSTEIN) return real_target ? -invB : invB;
  return (sigmoid_f(a) - (real_target ? 1.f : 0.f)) * invB;
}

// ---------------------------------------------------------------------------
// Grouped GEMM: one launch computes many independent problems
//   C[M][N] (+)= epilogue( sum_k A(i,k) B(k,j) )
// A(i,k) = A[i*lda + k] (a_trans 0) or A[k*lda + i] (a_trans 1);
// rows i >= a_rows of A are zero, except row ones_row which is all ones (this
// appends the bias row to a weight gradient: [X | 1]^T dY = (dW; db)).
// B(k,j) = B[k*ldb + j] (b_trans 0) or B[j*ldb + k] (b_trans 1).
// ---------------------------------------------------------------------------
enum Epi : int32_t {
  EPI_STORE = 0,     // C = acc
  EPI_BIAS_ACT = 1,  // C = act(acc + bias[j])
  EPI_DACT = 2,      // C = acc * act'(aux) with aux the forward output at the same index
  EPI_ADAM = 3       // acc is the gradient of parameter C[i][j]; Adam update of C, m, v
};

struct AdamConsts {
  float beta1, beta2, one_minus_beta1, one_minus_beta2, eps;
};

struct GemmProb {
  const float* A;
  const float* B;
  float* C;
  const float* bias;
  const float* aux;
  // Fields that only some epilogues use share storage (the descriptor is held
  // in scalar registers by every workgroup, so it is kept small).
  union {
    float* m;          // EPI_ADAM: the first moment
    float* gout;       // EPI_BIAS_ACT with dot_out: see the loss head below
    float* side;       // EPI_DACT with rs_mode: see the loss head below
  };
  union {
    float* v;          // EPI_ADAM: the second moment
    float* dlout;      // EPI_DACT with side
  };
  union {
    const float* lr;   // EPI_ADAM: the cell's learning rate
    const float* hsrc; // EPI_DACT with hpart: see the loss head below
  };
  union {
    const int32_t* t;  // EPI_ADAM: the cell's Adam step count before this call
    struct {
      int32_t hp_w;    // EPI_DACT with hpart: columns of hsrc (its row stride)
      int32_t hp_ld;   // EPI_DACT with hpart: row stride of hpart
    };
  };
  // EPI_BIAS_ACT only: when dot_out is set, the tile also writes
  //   dot_out[i*dot_ld + tile_n] = sum over its columns j of C[i][j] * dotw[j]
  // (+ *dot_bias in tile column 0): the next layer's 1-wide output, split
  // into per-tile partial sums that a later kernel adds in a fixed order.
  union {
    const float* dotw;
    const float* rs_part;  // EPI_DACT with rs_mode
  };
  const float* dot_bias;
  union {
    float* dot_out;
    float* hpart;      // EPI_DACT with rs_mode 1: see the loss head below
  };
  int32_t M, N, K;
  int32_t lda, ldb, ldc;
  int32_t a_trans, b_trans;
  int32_t a_rows, ones_row;
  int32_t epi, act;
  int32_t vec;         // bit 0: A rows 16-byte aligned; bit 1: B rows 16-byte aligned
  int32_t tiles_n;
  int32_t tile_begin;
  union {
    int32_t dot_ld;
    int32_t rs_tn;     // EPI_DACT with rs_mode
  };
  uint32_t a_bytes;    // extent of A from its base: a_rows * lda (a_trans 0) or K * lda floats
  uint32_t b_bytes;    // extent of B: K * ldb (b_trans 0) or N * ldb floats
  union {
    float clip;        // EPI_ADAM: when > 0 the updated parameter is clipped to [-clip, clip]
    int32_t side_ld;   // EPI_DACT with side
  };
  union {
    float gscale;      // EPI_ADAM: the gradient is acc * gscale (0 stands for 1: descriptors start zeroed)
    int32_t rs_B;      // EPI_DACT with rs_mode
  };
  // The discriminator's loss head, folded into the launches around it (a
  // 1-wide output layer a = h w + b over the last hidden layer h):
  //  * EPI_BIAS_ACT with dot_out: gout (when set) receives w[j] * act'(C[i][j]),
  //    indexed like C, so that dL/dh = (dL/da)[i] * gout[i][j];
  //  * EPI_DACT with rs_mode != 0: the product of the input gradient takes the
  //    per-row factor dL/da[i] of the head, formed from the partial logits
  //    rs_part[i * rs_tn + t] (t in order) as the separate head kernel forms it:
  //    rs_mode 1 rows i < rs_B have the "real" target, the others "fake"
  //    (discriminator step); rs_mode 2 every row "real" (generator step).
  //    side (when set) receives dL/da[i] * aux[i][j] (ld side_ld), and the
  //    tiles of column 0 also write side[i * side_ld + N] = dL/da[i], zeros
  //    at N + 1 .. N + 3, and dlout[4 i] = dL/da[i] (Wasserstein: the exact
  //    +-1 of the separate head, scaled by 1 / rs_B later), dlout[4 i + 1 .. 3] = 0.
  //  * EPI_DACT with rs_mode 1 and hpart set (hp_w <= N): the output layer's
  //    weight gradient in per-row-tile pieces.  The tile of rows m0 .. m0+BM-1
  //    writes, for its columns j < hp_w, hpart[(m0 / BM) * hp_ld + j] = sum
  //    over its rows i of dL/da[i] * hsrc[i * hp_w + j] (hsrc: the last hidden
  //    layer's activations), and the tile of column 0 also
  //    hpart[(m0 / BM) * hp_ld + hp_w] = sum over its rows of dL/da[i]
  //    (Wasserstein: the +-1 of dlout in both).
  int16_t rs_mode, loss_kind;
  // The grid's constants of the epilogues, the same in every descriptor:
  // the leaky-ReLU slope and Adam's constants.  Carried here so that a GEMM
  // workgroup reads nothing from kernel-argument memory.
  float slope;
  AdamConsts ac;
};

constexpr int GEMM_BN = 64;
constexpr int GEMM_MAX_GROUPS = 4;

// A phase's problems form up to 4 groups of consecutive problems with the
// same tile count, so a workgroup finds its problem from kernel arguments
// alone: group g covers tiles [first_tile[g], first_tile[g+1]) and problem
// first_prob[g] + (tile - first_tile[g]) / tiles_per_prob[g].
struct GemmGroups {
  int32_t n;
  int32_t total;  // GEMM tiles of the launch (set at launch); workgroups past them run its SampleJob
  int32_t first_tile[GEMM_MAX_GROUPS];
  int32_t first_prob[GEMM_MAX_GROUPS];
  int32_t tiles_per_prob[GEMM_MAX_GROUPS];
};

// Blocks are dispatched round-robin over the 8 XCDs (block b -> XCD b % 8).
// Each group of problems (tiles of one shape) is split into 8 contiguous
// chunks, one per XCD, whose sizes differ by at most one tile (the larger
// chunks rotate over the XCDs from group to group), and an XCD runs its
// chunks group after group.  Tiles of one problem (which share A rows and B
// columns) meet in the same L2, and every group is spread evenly over the
// XCDs, so a launch that mixes short and long tiles does not pile the long
// ones onto a few XCDs.  The per-XCD totals equal the number of blocks the
// round-robin dispatch gives each XCD.
__host__ __device__ inline int xcd_group_tile(int b, int nb, const GemmGroups& grp) {
  const int x = b & 7;
  int i = b >> 3, s = 0, t = 0;
#pragma unroll
  for (int g = 0; g < GEMM_MAX_GROUPS; ++g) {
    if (g < grp.n) {
      const int last = g + 1 == grp.n;
      const int tg = (last ? nb : grp.first_tile[g + 1]) - grp.first_tile[g];
      const int q = tg >> 3, r = tg & 7;
      const int cnt = q + (((x - s) & 7) < r ? 1 : 0);
      if (i >= 0 && (i < cnt || last)) {
        // chunks before x that hold one extra tile: XCDs s .. s + r - 1 (mod 8)
        const int e = s + r;
        int ext = x > s ? (x < e ? x : e) - s : 0;
        if (e > 8) ext += x < e - 8 ? x : e - 8;
        t = grp.first_tile[g] + x * q + ext + i;
      }
      i -= cnt;
      s = (s + r) & 7;
    }
  }
  return t;
}

// Tile height (32 or 64 rows) for a phase that has `tiles64` tiles of 64x64.
int gemm_tile_rows(int tiles64);

// True when a problem can use the fast kernel: one of the three operand
// layouts it instantiates, 16-byte aligned rows of both operands and extents
// below 2 GiB (buffer-load offsets are 32-bit).
bool gemm_fast_ok(const GemmProb& p);
// Fill a_bytes / b_bytes from the problem's shape (0 if they do not fit 32 bits).
void gemm_set_extents(GemmProb& p);

// True when a phase whose deepest problem has K = max_k runs faster on the
// wave-split kernel (each wave takes every fourth k block of the whole tile,
// operands straight from L2 into registers) than on the LDS-staged kernel.
bool gemm_wave_ok(int max_k);

// Kernel variants of the grouped GEMM (gemm.hip).
enum GemmKernel : int32_t {
  GEMM_K_GENERIC = 0,  // any alignment, per-element bounds checks
  GEMM_K_FAST = 1,     // register-staged LDS slices
  GEMM_K_WAVE = 2      // split-K across the four waves, operands from L2 into registers
};
// The kernel a phase runs on: its problems all fast-path eligible (fast), its
// deepest K (max_k).
int gemm_choose_kernel(bool fast, int max_k);

// A training minibatch drawn by extra workgroups of a GEMM launch (the
// draws of sample_kernel, written to other buffers than the launch's GEMMs
// read): units u0 .. u0 + units - 1, B rows each; workgroup q (of
// `blocks` = units * ceil(B / SAMPLE_ROWS)) takes rows SAMPLE_ROWS * (q %
// ceil(B / SAMPLE_ROWS)) .. of unit u0 + q / ceil(B / SAMPLE_ROWS): data row
// floor(w N / 2^32) of stream (u, gen, sf, IDX) to X[u][b][:] and latent row
// z[u][b][:] from stream (u, gen, sf, Z).  blocks == 0: no sampling.
constexpr int SAMPLE_ROWS = 4;
struct SampleJob {
  const float* data;
  float* X;
  float* Z;
  int64_t N, x_stride, z_stride;  // dataset rows; per-unit strides of X and Z (floats)
  uint2 key;
  uint32_t gen, sf;
  int32_t xd, zd, B, u0, blocks;
};

// Launch the grouped GEMM over the problems stored at d_probs (device),
// covering `total_tiles` tiles of tile_rows x 64 outputs on kernel variant
// `kernel`, plus the sampling workgroups of *job (may be null).  With
// write_through the kernels' stores are device-scope (written through L2).
// ev_start / ev_stop (or null) are recorded around the kernel itself.
hipError_t launch_gemm_grouped(const GemmProb* d_probs, const GemmGroups& grp, int total_tiles,
                               int tile_rows, int kernel, int step_local, bool write_through, hipStream_t s,
                               hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr, const SampleJob* job = nullptr);

// ---------------------------------------------------------------------------
// Convolutions as implicit GEMMs (conv.hip)
//
// Activations are NHWC.  A "position" is p = (img, y, x) of a grid
// [NI][2^gh][2^gw]; p = (img << (gh + gw)) | (y << gw) | x.  A position map
// sends p to the element ((img * 2^h + y * sy + y0) * 2^w + x * sx + x0) * ld
// of a tensor [NI][2^h][2^w][ld].  A tap t = (a, b) of a tw x tw tap grid
// (tw = 2^tw_log, t = a * tw + b) shifts the source row by a * tys + ty0 and the column by
// b * tys + tx0; it uses the weight tap (kh, kw) = (a * khs + kh0,
// b * khs + kw0) of a kw_full-wide kernel.  Source positions outside the
// tensor read 0 (zero padding).
//
// CONV_FWD: rows are the grid positions, columns the output channels:
//   C(p, n) = sum over taps t and channels c < cs of
//             S[map(p) shifted by t][c] * W[(tap(t) * cs + c) * wsc + n * wsn]
//   (wsc, wsn) = (N, 1): forward weights [taps][cs][N];
//   (wsc, wsn) = (1, cs): the transposed weights of an input gradient.
//   The output goes through the output position map; epilogues EPI_STORE,
//   EPI_BIAS_ACT and EPI_DACT (aux at the output's own address).
// CONV_WG: weight gradient, rows m = (t, c) of the tap-expanded input,
//   columns the output channels, reduced over the grid positions:
//   C(m, n) = sum over p of S[map(p) shifted by t][c] * P[pmap(p)][n],
//   plus row ones_row (if >= 0) = sum over p of P[pmap(p)][n] (a bias).
//   Row m = (t, c) is stored at weight-block row tap(t) * cs + c, the ones
//   row at brow.  K (positions) is cut into splits of ksplit positions;
//   split s writes its partial sums to C + s * split_stride.
// ---------------------------------------------------------------------------
enum ConvMode : int32_t { CONV_FWD = 0, CONV_WG = 1 };

struct PosMap {
  int32_t h_log, w_log;    // target spatial size (log2)
  int32_t sy, y0, sx, x0;  // grid -> target coordinates
  int32_t ld;              // floats per target position
};

struct ConvProb {
  int32_t mode;
  int32_t M, N, K;
  int32_t gh_log, gw_log;  // grid of positions (per image)
  int32_t taps, tw_log, cs;  // taps = 4^tw_log (0 for a bias-only problem), channels per tap
  int32_t cs_log;          // log2 cs, or -1 when taps == 1 (then k = c)
  int32_t tys, ty0, tx0;   // tap shifts
  int32_t khs, kh0, kw0, kw_full;
  int32_t gen;             // 1: element-wise (unaligned) operand loads
  const float* S;          // the tap-gathered operand
  PosMap smap;             // grid -> S (before the tap shift; sy/sx are the strides)
  uint32_t s_bytes;        // extent of S
  // CONV_FWD
  const float* W;
  int32_t wsc, wsn;
  uint32_t w_bytes;
  PosMap omap;             // grid -> C
  // CONV_WG
  const float* P;          // the plain operand (output gradient)
  PosMap pmap;
  uint32_t p_bytes;
  int32_t ones_row, brow;
  int32_t ksplit, splits;
  int64_t split_stride;
  int32_t ldc;             // CONV_WG: floats per partial row
  // output
  float* C;
  int32_t epi, act;
  const float* bias;
  const float* aux;
  int32_t tn;              // tile columns: 64, or 16 when N <= 16
  int32_t tiles_m, tiles_n, tile_begin;
  // Column taps (0 = off; element-wise loads only): column n is (tap n /
  // n_inner, channel n % n_inner).  CONV_FWD: B(k, n) = W[k-part +
  // (n / n_inner) * n_tap_stride + (n % n_inner) * wsn].  CONV_WG: output
  // (m, n) goes to row-block n / n_inner: C + (n / n_inner) * n_tap_stride +
  // row(m) * ldc + n % n_inner.
  int32_t n_inner, n_tap_stride;
};

// Patches of a 4x4, stride-2, pad-1 window (im2col): for every position
// (img, y, x) of a [NI][2^(h-1)]^2 grid,
//   dst[p][(kh * 4 + kw) * ch + c] = src[img][2y - 1 + kh][2x - 1 + kw][c] (0 outside).
// Its inverse gather (col2im) sums, for every element (img, Y, X, c) of a
// [NI][2^h]^2[ch] map, the 4 column entries that land on it:
//   out = sum over kh = (Y + 1) mod 2 + {0, 2}, kw likewise, with
//         (iy, ix) = ((Y + 1 - kh) / 2, (X + 1 - kw) / 2) inside the grid, of
//         cols[(img, iy, ix)][(kh * 4 + kw) * ch + c]
// in the order kh, kw ascending, then the epilogue: act(out + bias[c])
// (EPI_BIAS_ACT) or out * act'(aux at the output's index) (EPI_DACT).  The
// first is a stride-2 transposed convolution's output from its 16-tap
// columns; the second a stride-2 convolution's input gradient.
struct ColProb {
  const float* src;        // im2col: the map; col2im: the columns
  float* dst;              // im2col: the columns; col2im: the map
  const float* bias;
  const float* aux;
  int32_t n_img, h_log, ch;  // map [n_img][2^h][2^h][ch]
  int32_t epi, act;
};
// max_pairs: the largest (position, tap) count of the descriptors (n_img *
// 2^(2h-2) * 16); max_elems: the largest map (n_img * 2^(2h) * ch).
hipError_t launch_im2col(const ColProb* d_probs, int n_probs, int64_t max_pairs, hipStream_t s);
hipError_t launch_col2im(const ColProb* d_probs, int n_probs, int64_t max_elems, float slope, hipStream_t s);

// A convolution phase's problems in up to 4 groups of consecutive problems
// with equal tile counts (tiles_m * tiles_n * splits).  Each group starts at
// a block index that is a multiple of 8 and spans a multiple of 8 blocks
// (blocks past its real_tiles exit at once), so every XCD receives an equal,
// contiguous share of every group: groups of long tiles (deep K) are not
// piled onto a few XCDs.
struct ConvGroups {
  int32_t n;
  int32_t first_block[GEMM_MAX_GROUPS];
  int32_t blocks[GEMM_MAX_GROUPS];
  int32_t real_tiles[GEMM_MAX_GROUPS];
  int32_t first_prob[GEMM_MAX_GROUPS];
  int32_t tiles_per_prob[GEMM_MAX_GROUPS];
};

// Launch every problem of one phase (problems in device memory).
hipError_t launch_conv_grouped(const ConvProb* d_probs, const ConvGroups& grp, int total_blocks, float slope,
                               hipStream_t s, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// Sum of the split partial sums of a weight gradient, in split order, then
// the Adam step of the parameters (W and its bias row laid out as the
// partial rows).  One descriptor per (cell, layer).
struct RedProb {
  const float* part;
  int64_t split_stride;
  int32_t splits;
  int64_t n;               // parameters (rows * cols)
  float* p;
  float* m;
  float* v;
  const float* lr;
  const int32_t* t;
  float clip;              // > 0: clip every updated parameter to [-clip, clip] (the Wasserstein critic)
};
hipError_t launch_reduce_adam(const RedProb* d_probs, int n_probs, int64_t max_n, int step_local, AdamConsts ac,
                              hipStream_t s);

// Batch norm over the rows of x [rows][ch] of each instance, statistics of
// the batch itself (biased variance, eps), in a fixed order: per chunk of
// BN_CHUNK rows a two-pass mean and sum of squared deviations, then the
// chunks merged in order (Chan, Golub and LeVeque's pairwise update).
constexpr int BN_CHUNK = 256;
struct BnProb {
  const float* x;          // conv output [rows][ch]
  float* y;                // forward: act(gamma xhat + beta); backward: gradient in / out
  const float* aux;        // backward: unused
  int64_t rows;
  int32_t ch;
  float* part;             // [chunks][2][ch] scratch
  float* stats;            // [2][ch]: mean, rstd  (backward: + [3][ch] coefficients)
  float* gamma;            // parameters of the cell; beta = gamma + ch
  float* gm;               // Adam m, v of gamma (beta follows)
  float* gv;
  const float* lr;
  const int32_t* t;
  int32_t act;
  int32_t first_block;     // prefix of chunks * channel groups over preceding instances
};
hipError_t launch_bn_stats(const BnProb* d_probs, int n_probs, int total_blocks, float eps, hipStream_t s);
hipError_t launch_bn_apply(const BnProb* d_probs, int n_probs, int64_t max_elems, float slope, hipStream_t s);
// Backward: y holds dL/d(bn output); becomes dL/dx.  gamma, beta take an Adam step.
hipError_t launch_bn_backward(const BnProb* d_probs, int n_probs, int total_blocks, int64_t max_elems,
                              int step_local, AdamConsts ac, hipStream_t s);

// out[r * ld_out] = dot(x[r][0..H), w) + *bias for each row r of each instance.
struct DotProb {
  const float* x;
  const float* w;          // weights, bias at w[H]
  float* out;
  int32_t rows, H, ld_out;
  int32_t first_row;       // prefix of rows over preceding instances
};
hipError_t launch_dot_rows(const DotProb* d_probs, int n_probs, int total_rows, hipStream_t s);

// Initial DCGAN parameters of C cells (rows of `stride` floats): element e of
// a row is normal number e of the stream (cell, 0, 0, tag); weights get
// 0.02 n, batch-norm gammas 1 + 0.02 n, biases and betas 0.
struct ConvInitLayout {
  int32_t n;
  int64_t off_w[8], n_w[8], off_b[8], off_g[8];
  int32_t n_b[8], n_g[8];
};
hipError_t launch_init_conv_params(float* p, int64_t stride, int64_t P, int C, const ConvInitLayout& L, uint2 key,
                                   uint32_t tag, hipStream_t s);

// ---------------------------------------------------------------------------
// Other kernels (kernels.hip)
// ---------------------------------------------------------------------------
struct NetLayers {
  int32_t n;             // number of layers
  int64_t off[8];        // offset of W_l in the parameter row
  int32_t fan_in[8];
  int32_t fan_out[8];
};

hipError_t launch_init_params(float* p, int64_t stride, int64_t P, int C, NetLayers L, uint2 key,
                              uint32_t tag, hipStream_t s);
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s);
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s);
hipError_t launch_normals(float* out, int64_t n, double scale, uint2 key, uint32_t cell, uint32_t gen,
                          uint32_t step_field, uint32_t tag, hipStream_t s);
// Cells c0 .. c0 + C - 1.
hipError_t launch_sample(const float* data, int64_t N, int xd, int zd, int B, int c0, int C, uint2 key,
                         uint32_t gen, uint32_t step_field, float* X, int64_t x_cell_stride,
                         float* Z, int64_t z_cell_stride, hipStream_t s);

struct HeadArgs {
  int loss_only;         // only the per-cell losses (the loss head is folded into the GEMM launches)
  const float* part;     // per-tile partial logits [C][rows][tn] (bias included)
  int tn;
  const float* act;      // last hidden activations [C][rows][H] (cell stride act_cell_stride)
  int64_t act_cell_stride;
  float* delta;          // out: gradient w.r.t. the last hidden pre-activation, same layout
  const float* w;        // output-layer weights of cell 0; cell c at w + c * p_stride
  int64_t p_stride;
  float* dlbuf;          // D step: out dL/da as [C][2B][4] (column 0), else null;
                         // Wasserstein: B dL/da = -1 / +1, exact, so its sum over rows is exactly 0
  float* losses;         // [cells][2] slice for this step, or null
  int H, B;
  int c0, C;             // the launch covers cells c0 .. c0 + C - 1
  int hidden_act;
  float slope;
  int loss_kind;         // LIPZ_LOSS_BCE or LIPZ_LOSS_WASSERSTEIN
};
// Discriminator step head: logits of 2B rows (B real then B fake), BCE, its
// gradient dL/da into dlbuf and delta.
hipError_t launch_head_d(const HeadArgs& a, hipStream_t s);
// Generator step head: logits of B fake rows, non-saturating loss, delta.
hipError_t launch_head_g(const HeadArgs& a, hipStream_t s);
// The losses alone (a.losses) of the discriminator / generator step.
hipError_t launch_loss_d(const HeadArgs& a, hipStream_t s);
hipError_t launch_loss_g(const HeadArgs& a, hipStream_t s);

struct EvalHeadArgs {
  const float* part;     // partial logits [C][nn][(1 + nn) B][tn] (bias included)
  int tn;
  float* L;              // [C][nn][nn]
  float* Lg;
  float* rmean;          // [C][nn] real-row term means, or null
  int B, C, nn;
  int loss_kind;         // LIPZ_LOSS_BCE or LIPZ_LOSS_WASSERSTEIN
};
hipError_t launch_head_eval(const EvalHeadArgs& a, hipStream_t s);

// NES trainer (one role): perturbed parameter sets, their losses, and the
// estimate + Adam step.  Set q < n holds theta + sigma eps_q, set n + k holds
// theta - sigma eps_k, set 2n holds theta; eps_k[e] is normal k P + e of
// stream (cell, gen, sf, tag).
struct NesArgs {
  float* p;              // the role's parameters, cell c at p + c * stride (updated in place)
  float* m;
  float* v;
  const float* lr;       // [C]
  const int32_t* t;      // [C] Adam step count before this call
  float* sets;           // [C][2n][stride]: theta + sigma eps_k (k < n), theta - sigma eps_(k-n)
  float* eps;            // [C][n][eps_stride]: the directions eps_k in fp32 (null: not kept)
  const float* part;     // partial logits: D role [C][Q][2B][tn], G role [C][Q B][tn]
  float* fit;            // [C][Q] loss of each set
  float* losses;         // [C][2] slice of this step, or null
  int64_t stride, P, eps_stride;
  int n, tn, B, c0, C;   // training units c0 .. c0 + C - 1
  int role;              // LIPZ_ROLE_G / LIPZ_ROLE_D
  int loss_kind;
  float sigma, clip;     // clip > 0: clip the updated parameters (Wasserstein critic)
  uint2 key;
  uint32_t gen, sf, tag;
  int step_local;
  AdamConsts ac;
};
hipError_t launch_nes_perturb(const NesArgs& a, hipStream_t s);
hipError_t launch_nes_head(const NesArgs& a, hipStream_t s);
hipError_t launch_nes_update(const NesArgs& a, hipStream_t s);
hipError_t launch_es_select(const NesArgs& a, hipStream_t s);
hipError_t launch_fitness(const float* L, const float* Lg, int C, int nn, int mode, float* fit_g, float* fit_d,
                          int32_t* flags, float* out_L, float* out_Lg, float* out_fg, float* out_fd,
                          hipStream_t s);

struct SelectArgs {
  const float* fit_g;
  const float* fit_d;
  const int32_t* nbr;
  const int32_t* forced;   // [U][2] source individuals, or null
  int32_t* sel;            // internal [U][2]
  int32_t* flags;          // bit 1 set when a forced source individual is out of range
  int32_t* sel_out;        // or null
  float* lr_out;           // or null
  const int32_t* t_src[2]; // current buffer Gt, Dt
  const float* lr_src[2];
  int32_t* t_dst[2];       // next buffer
  float* lr_dst[2];
  int c0, C, s, U, tsize, mutate;  // cells c0 .. c0 + C - 1; individuals per role and cell; all individuals
  float mut_std, mut_prob;
  uint2 key;
  uint32_t gen;
};
hipError_t launch_select(const SelectArgs& a, hipStream_t s);

// Post-training re-evaluation (elitism).  Block (j, c), j < nn: previous
// discriminator j of the cell's neighbourhood on the s B rows of the trained
// generators (part2 [C][nn][s B][tn]); block (nn + j, c), j < s: trained
// discriminator j on the (1 + nn) B evaluation rows (part3 [C][s][(1+nn)B][tn]).
//   L2[c][i][j] = rmean[c][j] + mean fake term of G'_i under D_j, Lg2 its
//   generator term; M3[c][0][j] the real-row mean of D'_j, M3[c][1 + k][j]
//   its fake mean on G_k's rows (L(G_k, D'_j) = M3[c][0][j] + M3[c][1+k][j]).
// The merge (one thread per cell and role) forms fit2 = -mean_j L2 (or
// mean_j Lg2) and mean_k L3 in a fixed order, keeps the s best of the 2 s,
// writes src (previous individual or -1) and the step counts and learning
// rates of the slots given back.
struct EliteArgs {
  const float* part2;
  const float* part3;
  const float* rmean;    // [C][nn]
  float* L2;             // [C][s][nn]
  float* Lg2;            // [C][s][nn]
  float* M3;             // [C][1 + nn][s]
  const float* fit_g;    // [C][nn] fitness of the previous neighbourhood (evaluation)
  const float* fit_d;
  float* fit2_g;         // [C][s]
  float* fit2_d;
  int32_t* src;          // [U][2] internal: previous individual or -1
  int32_t* src_out;      // [U][2] previous member or -1, or null
  float* fit2_g_out;     // or null
  float* fit2_d_out;
  int32_t* flags;        // bit 0 on a non-finite value
  const int32_t* t_old[2];
  const float* lr_old[2];
  int32_t* t_new[2];
  float* lr_new[2];
  int tn, B, c0, C, s, nn, mode, loss_kind;  // cells c0 .. c0 + C - 1
};
hipError_t launch_elite(const EliteArgs& a, hipStream_t s);

struct CopyArgs {
  const int32_t* sel;      // [U][2] source individual of each destination, < 0: no copy
  const float* src[2][3];  // role, (p, m, v)
  float* dst[2][3];
  int64_t stride[2];       // floats per row, multiple of 4
  const float* w_src;      // mixture weights [C][5] copied along, or null
  float* w_dst;
  int U, C;
};
hipError_t launch_copy_winners(const CopyArgs& a, hipStream_t s);
hipError_t launch_add_i32(int32_t* p, int n, int32_t v, hipStream_t s);

// Feature moments in fp64 (mean f and mean f^2 per cell and feature: their
// difference, the variance, cancels when the mean dominates).
// part: scratch of C * ceil(S / 64) * 2 * F doubles.
hipError_t launch_moments(const float* feats, int C, int S, int F, double* part, double* mu, double* s2,
                          hipStream_t s);
hipError_t launch_col_stats(const float* feats, int64_t N, int F, double* mu, double* sd, hipStream_t s);

struct EsArgs {
  const double* mu;       // [cells][F]
  const double* s2;
  const double* mu_r;
  const double* sd_r;
  const int32_t* nbr;
  float* w;               // [C][5] in place
  float* w_out;
  float* score_out;
  int32_t* acc_out;
  int c0, C, F;            // cells c0 .. c0 + C - 1
  float sigma;
  uint2 key;
  uint32_t gen;
};
hipError_t launch_es(const EsArgs& a, hipStream_t s);

}  // namespace lipz
