// Element-wise, sampling, loss-head, selection and mixture kernels of the grid
// coevolution.  Every reduction runs in a fixed order, so results are
// bit-reproducible run to run (no floating-point atomics).
#include "lipz_internal.h"

namespace lipz {

namespace {

constexpr int NT = 256;

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Sum of one value per thread over a 256-thread block in a fixed order.
__device__ float block_sum(float x, float* red) {
  x = wave_sum(x);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) red[wave] = x;
  __syncthreads();
  const float r = (red[0] + red[1]) + (red[2] + red[3]);
  __syncthreads();
  return r;
}

// ---------------------------------------------------------------------------
// Step 1 initialisation: element e of a cell's parameter row, in layer l,
// is (2u - 1) / sqrt(fan_in_l) with u from word e of stream (cell, 0, 0, tag).
// ---------------------------------------------------------------------------
__global__ void init_params_kernel(float* p, int64_t stride, int64_t P, int C, NetLayers L,
                                   uint2 key, uint32_t tag) {
  const int64_t total = (int64_t)C * P;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i / P);
    const int64_t e = i - (int64_t)c * P;
    int l = 0;
    while (l + 1 < L.n && e >= L.off[l + 1]) ++l;
    const uint4 w = stream_block(key, (uint32_t)(e >> 2), (uint32_t)c, 0, 0, tag);
    const double u = uniform_of(word_of(w, (int)(e & 3)));
    p[(int64_t)c * stride + e] = (float)((2.0 * u - 1.0) / sqrt((double)L.fan_in[l]));
  }
}

__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}
__global__ void fill_i32_kernel(int32_t* p, int64_t n, int32_t v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}
__global__ void add_i32_kernel(int32_t* p, int n, int32_t v) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] += v;
}

__global__ void normals_kernel(float* out, int64_t n, double scale, uint2 key, uint32_t cell,
                               uint32_t gen, uint32_t sf, uint32_t tag) {
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < n;
       e += (int64_t)gridDim.x * blockDim.x) {
    const uint4 w = stream_block(key, (uint32_t)(e >> 2), cell, gen, sf, tag);
    out[e] = (float)(scale * normal_of(w, (int)(e & 3)));
  }
}

// ---------------------------------------------------------------------------
// Minibatch sampling: block (b, c) draws data row floor(w_b N / 2^32) of
// stream (c, gen, sf, IDX) and copies it to X[c][b]; it also writes the
// latent row z[c][b][:] from stream (c, gen, sf, Z), element b * zd + k.
// ---------------------------------------------------------------------------
__global__ void sample_kernel(const float* __restrict__ data, int64_t N, int xd, int zd, int c0,
                              uint2 key, uint32_t gen, uint32_t sf, float* __restrict__ X,
                              int64_t x_cell_stride, float* __restrict__ Z, int64_t z_cell_stride) {
  const int b = blockIdx.x, c = c0 + blockIdx.y;
  const uint4 wi = stream_block(key, (uint32_t)(b >> 2), (uint32_t)c, gen, sf, LIPZ_TAG_IDX);
  const int64_t row = (int64_t)(((uint64_t)word_of(wi, b & 3) * (uint64_t)N) >> 32);
  const float* src = data + row * xd;
  float* dst = X + c * x_cell_stride + (int64_t)b * xd;
  if ((xd & 3) == 0) {
    for (int q = threadIdx.x; q < (xd >> 2); q += blockDim.x)
      reinterpret_cast<float4*>(dst)[q] = reinterpret_cast<const float4*>(src)[q];
  } else {
    for (int q = threadIdx.x; q < xd; q += blockDim.x) dst[q] = src[q];
  }
  for (int k = threadIdx.x; k < zd; k += blockDim.x) {
    const int64_t e = (int64_t)b * zd + k;
    const uint4 w = stream_block(key, (uint32_t)(e >> 2), (uint32_t)c, gen, sf, LIPZ_TAG_Z);
    Z[c * z_cell_stride + e] = (float)normal_of(w, (int)(e & 3));
  }
}

// ---------------------------------------------------------------------------
// Output layer of D (H -> 1) for block (cell, 64-column block cb, 32-row
// chunk rs).  Logits come from the per-tile partial sums (bias included):
//   D step rows: B real (target 1) then B fake (target 0); G step: B fake
//   rows with the non-saturating target 1.  dL/da = (sigmoid(a) - target) / B,
//   delta[r][n] = dL/da_r * w_n * act'(act[r][n]) for the block's cells.
// Block (cb 0, rs 0) also writes the loss (mean softplus(-a_real) + mean
// softplus(a_fake), or mean softplus(-a_fake)).  In the D step, blocks with
// cb 0 write dL/da into dlbuf[r][0] (columns 1..3 zero): the gradient of the
// output layer, [act | 1]^T dL/da, and its Adam step run as a GEMM problem
// of the next phase, so nothing here reads and writes w in one launch.
// When the head is folded into the GEMM epilogues (D with two or more hidden
// layers) the same kernel runs with loss_only: grid (C, 1, 1), the loss alone.
// ---------------------------------------------------------------------------
constexpr int HEAD_ROWS = 32;


template <bool D_STEP>
__global__ __launch_bounds__(NT) void head_kernel(HeadArgs A) {
  __shared__ float dl[HEAD_ROWS];
  __shared__ float red[4];
  const int c = A.c0 + blockIdx.x, cb = blockIdx.y, rs = blockIdx.z;
  const int rows = D_STEP ? 2 * A.B : A.B;
  const int r0 = rs * HEAD_ROWS;
  const int nr = min(HEAD_ROWS, rows - r0);
  const int tn = A.tn;
  const float* part = A.part + (int64_t)c * rows * tn;
  const float invB = 1.f / (float)A.B;
  if (!A.loss_only && (int)threadIdx.x < nr) {
    const int r = r0 + threadIdx.x;
    float a = 0.f;
    for (int t = 0; t < tn; ++t) a += part[(int64_t)r * tn + t];
    const float d = head_dl(A.loss_kind, a, !D_STEP || r < A.B, invB);
    dl[threadIdx.x] = d;
    if (D_STEP && cb == 0) {
      float* o = A.dlbuf + ((int64_t)c * rows + r) * 4;
      // the Wasserstein critic's output bias has a zero gradient: store the
      // exact +-1 (the weight-gradient GEMM scales by 1 / B afterwards)
      o[0] = A.loss_kind == LIPZ_LOSS_WASSERSTEIN ? (r < A.B ? -1.f : 1.f) : d;
      o[1] = 0.f;
      o[2] = 0.f;
      o[3] = 0.f;
    }
  }
  if (cb == 0 && rs == 0) {
    float lr_ = 0.f, lf = 0.f;
    for (int r = threadIdx.x; r < rows; r += NT) {
      float a = 0.f;
      for (int t = 0; t < tn; ++t) a += part[(int64_t)r * tn + t];
      if (D_STEP && r >= A.B) lf += fake_term(A.loss_kind, a);
      else lr_ += real_term(A.loss_kind, a);
    }
    lr_ = block_sum(lr_, red);
    lf = block_sum(lf, red);
    if (threadIdx.x == 0 && A.losses)
      A.losses[c * 2 + (D_STEP ? 0 : 1)] = D_STEP ? lr_ * invB + lf * invB : lr_ * invB;
  }
  if (A.loss_only) return;
  __syncthreads();
  const int H = A.H;
  const int n = cb * 64 + (threadIdx.x & 63);
  if (n >= H) return;
  const int rg = threadIdx.x >> 6;
  const float w = A.w[(int64_t)c * A.p_stride + n];
  const float* act = A.act + c * A.act_cell_stride;
  float* delta = A.delta + c * A.act_cell_stride;
  float y[HEAD_ROWS / 4];
#pragma unroll
  for (int k = 0; k < HEAD_ROWS / 4; ++k) {
    const int rr = rg + 4 * k;
    y[k] = rr < nr ? act[(int64_t)(r0 + rr) * H + n] : 0.f;
  }
#pragma unroll
  for (int k = 0; k < HEAD_ROWS / 4; ++k) {
    const int rr = rg + 4 * k;
    if (rr < nr) delta[(int64_t)(r0 + rr) * H + n] = dl[rr] * w * act_deriv_from_out(A.hidden_act, y[k], A.slope);
  }
}

// ---------------------------------------------------------------------------
// Evaluation head for block (j, c): logits of the (1 + nn) B rows
// [x_c; G_0(z_c); ...; G_(nn-1)(z_c)] under discriminator j (from the partial
// sums), then
//   L[c][i][j] = mean softplus(-a_real) + mean softplus(a_fake_i)
//   Lg[c][i][j] = mean softplus(-a_fake_i)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(NT) void head_eval_kernel(EvalHeadArgs A) {
  extern __shared__ float mean[];  // [1 + 2 nn]
  const int j = blockIdx.x, c = blockIdx.y, nn = A.nn;
  const int rows = (1 + nn) * A.B;
  const float* part = A.part + (int64_t)(c * nn + j) * rows * A.tn;
  // one wave per mean: mean 0 is the real rows' term, 1 .. nn the fake
  // block i = q - 1, nn + 1 .. 2 nn the generator term of block q - nn; each
  // sums its B terms lane-strided (a row's logit is its partial sums in
  // order), then a fixed shuffle tree
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int q = wave; q <= 2 * nn; q += NT / 64) {
    const int blk = q <= nn ? q : q - nn;
    const bool fake = q >= 1 && q <= nn;
    float s = 0.f;
    for (int b = lane; b < A.B; b += 64) {
      const float* pr = part + (int64_t)(blk * A.B + b) * A.tn;
      float a = 0.f;
      for (int t = 0; t < A.tn; ++t) a += pr[t];
      s += fake ? fake_term(A.loss_kind, a) : real_term(A.loss_kind, a);
    }
    s = wave_sum(s);
    if (lane == 0) mean[q] = s / (float)A.B;
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nn; i += NT) {
    A.L[(c * nn + i) * nn + j] = mean[0] + mean[1 + i];
    A.Lg[(c * nn + i) * nn + j] = mean[1 + nn + i];
  }
  if (A.rmean && threadIdx.x == 0) A.rmean[c * nn + j] = mean[0];
}

// ---------------------------------------------------------------------------
// NES trainer (Section 3 lists NES among the trainers; reading: antithetic
// estimate + Adam).  eps_k[e] = normal k P + e of stream (cell, gen, sf, tag).
// ---------------------------------------------------------------------------
// Thread b of cell c draws Philox block b of the cell's direction stream:
// normals i = 4b .. 4b+3 of the n P (direction k = i / P, element e = i % P).
// The workgroup's 4 NT normals pass through LDS so that each store writes NT
// consecutive elements.  Every normal is drawn once; it goes to eps and to
// the sets theta + sigma eps_k and theta - sigma eps_k.  n P < 2^31.
__global__ __launch_bounds__(NT) void nes_perturb_kernel(NesArgs A) {
  __shared__ float4 zs4[NT];
  const int c = A.c0 + blockIdx.y;
  const uint32_t P = (uint32_t)A.P, total = (uint32_t)A.n * P;
  const uint32_t b0 = blockIdx.x * NT, b = b0 + threadIdx.x;
  if (4u * b < total) {
    const uint4 w = stream_block(A.key, b, (uint32_t)c, A.gen, A.sf, A.tag);
    const double r01 = sqrt(-2.0 * log(uniform_of(w.x)));
    const double r23 = sqrt(-2.0 * log(uniform_of(w.z)));
    double s01, c01, s23, c23;
    // the angle 2 pi u as sincospi(2 u): no argument reduction by 2 pi
    sincospi(2.0 * uniform_of(w.y), &s01, &c01);
    sincospi(2.0 * uniform_of(w.w), &s23, &c23);
    zs4[threadIdx.x] = make_float4((float)(r01 * c01), (float)(r01 * s01), (float)(r23 * c23), (float)(r23 * s23));
  }
  __syncthreads();
  const float* zs = reinterpret_cast<const float*>(zs4);
  const float* th = A.p + c * A.stride;
  float* sets = A.sets + (int64_t)c * 2 * A.n * A.stride;
  float* dir = A.eps ? A.eps + (int64_t)c * A.n * A.eps_stride : nullptr;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t i = 4u * b0 + threadIdx.x + j * NT;
    if (i >= total) break;
    const float z = zs[threadIdx.x + j * NT];
    const uint32_t k = i / P, e = i - k * P;
    const float se = A.sigma * z;
    const float t = th[e];
    sets[(int64_t)k * A.stride + e] = t + se;
    sets[(int64_t)(A.n + k) * A.stride + e] = t - se;
    if (A.eps) dir[(int64_t)k * A.eps_stride + e] = z;
  }
}

// block (q, c): the loss of set q from the partial logits, in a fixed order.
// D role: rows [x; G(z)] (2B); G role: the B rows generated by set q.
__global__ __launch_bounds__(NT) void nes_head_kernel(NesArgs A) {
  __shared__ float red[4];
  const int q = blockIdx.x, c = A.c0 + blockIdx.y, Q = 2 * A.n + 1;
  const bool d_role = A.role == LIPZ_ROLE_D;
  const int rows = d_role ? 2 * A.B : A.B;
  const float* part = A.part + ((int64_t)c * Q + q) * rows * A.tn;
  float s = 0.f;
  for (int r = threadIdx.x; r < rows; r += NT) {
    float a = 0.f;
    for (int t = 0; t < A.tn; ++t) a += part[(int64_t)r * A.tn + t];
    s += (d_role && r >= A.B) ? fake_term(A.loss_kind, a) : real_term(A.loss_kind, a);
  }
  s = block_sum(s, red);
  if (threadIdx.x == 0) {
    const float f = s / (float)A.B;
    A.fit[c * Q + q] = f;
    if (q == 2 * A.n && A.losses) A.losses[c * 2 + (d_role ? 0 : 1)] = f;
  }
}

// block (x, c): g[e] = sum_k (F_k+ - F_k-) eps_k[e] / (2 n sigma), then one
// bias-corrected Adam step of parameter e (and the clip, when set)
__global__ __launch_bounds__(NT) void nes_update_kernel(NesArgs A) {
  __shared__ float bc[2];
  const int c = A.c0 + blockIdx.y, Q = 2 * A.n + 1;
  const AdamConsts& ac = A.ac;
  if (threadIdx.x == 0) {
    const int tt = A.t[c] + A.step_local + 1;
    bc[0] = (float)(1.0 - pow((double)ac.beta1, (double)tt));
    bc[1] = (float)(1.0 - pow((double)ac.beta2, (double)tt));
  }
  __syncthreads();
  const int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (e >= A.P) return;
  const float* f = A.fit + c * Q;
  const float* dir = A.eps + (int64_t)c * A.n * A.eps_stride + e;
  // eight directions' loads in flight at once; the sum keeps the order k = 0, 1, ...
  float g = 0.f;
  int k = 0;
  for (; k + 8 <= A.n; k += 8) {
    float d[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) d[j] = dir[(int64_t)(k + j) * A.eps_stride];
#pragma unroll
    for (int j = 0; j < 8; ++j) g += (f[k + j] - f[A.n + k + j]) * d[j];
  }
  for (; k < A.n; ++k) g += (f[k] - f[A.n + k]) * dir[(int64_t)k * A.eps_stride];
  g /= 2.f * (float)A.n * A.sigma;
  const int64_t o = c * A.stride + e;
  const float lr = A.lr[c];
  const float m = ac.beta1 * A.m[o] + ac.one_minus_beta1 * g;
  const float v = ac.beta2 * A.v[o] + ac.one_minus_beta2 * g * g;
  float p = A.p[o] - lr * (m / bc[0]) / (sqrtf(v / bc[1]) + ac.eps);
  if (A.clip > 0.f) p = p > A.clip ? A.clip : (p < -A.clip ? -A.clip : p);
  A.m[o] = m;
  A.v[o] = v;
  A.p[o] = p;
}

// block (x, c): the ES trainer's plus-selection.  Set q of cell c (q < 2n the
// mutants, q = 2n the parent) has loss fit[c][q]; the first mutant of lowest
// loss replaces the parent only if that loss is strictly lower.  Then the
// critic clip, on whichever set was kept.
// Ordering key of a loss or fitness value: NaN sorts as +infinity (it loses).
__device__ __forceinline__ float fit_key(float f) { return f != f ? INFINITY : f; }

// Plus-selection over the 2n + 1 losses of a unit (parent last), NaN as
// +infinity: the first mutant of lowest key replaces the parent only when
// its key is strictly lower.
__global__ __launch_bounds__(NT) void es_select_kernel(NesArgs A) {
  __shared__ int win;
  const int c = A.c0 + blockIdx.y, parent = 2 * A.n;
  if (threadIdx.x == 0) {
    const float* f = A.fit + c * (parent + 1);
    int q = 0;
    for (int j = 1; j < parent; ++j)
      if (fit_key(f[j]) < fit_key(f[q])) q = j;
    win = fit_key(f[q]) < fit_key(f[parent]) ? q : parent;
  }
  __syncthreads();
  const int64_t e = (int64_t)blockIdx.x * NT + threadIdx.x;
  if (e >= A.P) return;
  const int64_t o = c * A.stride + e;
  float p = win == parent ? A.p[o] : A.sets[((int64_t)c * parent + win) * A.stride + e];
  if (A.clip > 0.f) p = p > A.clip ? A.clip : (p < -A.clip ? -A.clip : p);
  A.p[o] = p;
}

// fit_d[c][j] = mean_i L[c][i][j]; fit_g[c][i] = -mean_j L[c][i][j] (mode 0)
// or mean_j Lg[c][i][j] (mode 1).  Flags bit 0 on any non-finite value.
__global__ void fitness_kernel(const float* L, const float* Lg, int C, int nn, int mode, float* fit_g,
                               float* fit_d, int32_t* flags, float* oL, float* oLg, float* ofg,
                               float* ofd) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  const int nn2 = nn * nn;
  if (i < C * nn2) {
    if (oL) oL[i] = L[i];
    if (oLg) oLg[i] = Lg[i];
    if (!isfinite(L[i]) || !isfinite(Lg[i])) atomicOr(flags, 1);
  }
  if (i >= C * nn) return;
  const int c = i / nn, k = i % nn;
  const float* Lc = L + (int64_t)c * nn2;
  float sd = 0.f;
  for (int a = 0; a < nn; ++a) sd += Lc[a * nn + k];
  float sg = 0.f;
  if (mode == 0) {
    for (int b = 0; b < nn; ++b) sg += Lc[k * nn + b];
    sg = -(sg / (float)nn);
  } else {
    for (int b = 0; b < nn; ++b) sg += Lg[(int64_t)c * nn2 + k * nn + b];
    sg = sg / (float)nn;
  }
  sd = sd / (float)nn;
  fit_d[i] = sd;
  fit_g[i] = sg;
  if (ofd) ofd[i] = sd;
  if (ofg) ofg[i] = sg;
}

// ---------------------------------------------------------------------------
// Tournament + learning-rate mutation, one thread per (cell, role).
// ---------------------------------------------------------------------------
// Thread (cell c, member i, role): tournament i of the cell over its nn
// neighbourhood individuals, words 8 i .. 8 i + 7 of the cell's stream
// (Philox blocks 2 i, 2 i + 1); the copy's learning-rate mutation from words
// 4 i .. 4 i + 3 (block i) of the mutation stream.
__global__ void select_kernel(SelectArgs A) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  const int nn = LIPZ_SLOTS * A.s;
  if (t >= 2 * A.C * A.s) return;
  const int u = A.c0 * A.s + (t >> 1), role = t & 1, c = u / A.s, i = u % A.s;
  int src;
  if (A.forced) {
    src = A.forced[u * 2 + role];
    if (src < 0 || src >= A.U) {
      atomicOr(A.flags, 2);
      src = u;
    }
  } else {
    const float* fit = (role == 0 ? A.fit_g : A.fit_d) + c * nn;
    const uint32_t tag = role == 0 ? LIPZ_TAG_TOURN_G : LIPZ_TAG_TOURN_D;
    const uint4 w0 = stream_block(A.key, 2 * i, (uint32_t)c, A.gen, 0, tag);
    const uint4 w1 = stream_block(A.key, 2 * i + 1, (uint32_t)c, A.gen, 0, tag);
    int remaining[LIPZ_SLOTS * 4];
    for (int q = 0; q < nn; ++q) remaining[q] = q;
    int n_rem = nn;
    int best = -1;
    const int draws = A.tsize < nn - 1 ? A.tsize : nn - 1;
    for (int j = 0; j < A.tsize; ++j) {
      int pos = 0;
      if (j < draws) pos = (int)(((uint64_t)word_of(j < 4 ? w0 : w1, j & 3) * (uint64_t)(nn - j)) >> 32);
      const int k = remaining[pos];
      for (int q = pos; q + 1 < n_rem; ++q) remaining[q] = remaining[q + 1];
      --n_rem;
      if (best < 0 || fit_key(fit[k]) < fit_key(fit[best])) best = k;
    }
    src = A.nbr[c * LIPZ_SLOTS + best / A.s] * A.s + best % A.s;
  }
  A.sel[u * 2 + role] = src;
  if (A.sel_out) A.sel_out[u * 2 + role] = src;
  A.t_dst[role][u] = A.t_src[role][src];
  float lr = A.lr_src[role][src];
  if (A.mutate) {
    const uint4 w = stream_block(A.key, i, (uint32_t)c, A.gen, 0,
                                 role == 0 ? LIPZ_TAG_LRMUT_G : LIPZ_TAG_LRMUT_D);
    if (uniform_of(w.x) < (double)A.mut_prob) {
      const double nv = (double)lr + (double)A.mut_std * normal_of(w, 2);
      lr = (float)(nv > 0.0 ? nv : 0.0);
    }
  }
  A.lr_dst[role][u] = lr;
  if (A.lr_out) A.lr_out[u * 2 + role] = lr;
}
// means of one block of B rows of partial logits, one wave per mean (see
// head_eval_kernel): q < nq means, mean q over rows [row0(q), row0(q) + B)
__global__ __launch_bounds__(NT) void elite_means_kernel(EliteArgs A) {
  const int c = A.c0 + blockIdx.y, nn = A.nn, s = A.s;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const bool prev = (int)blockIdx.x < nn;
  const int j = prev ? blockIdx.x : blockIdx.x - nn;
  // previous D_j: s fake means then s generator terms; trained D'_j: real
  // mean then nn fake means
  const int nq = prev ? 2 * s : 1 + nn;
  const float* part = prev ? A.part2 + (int64_t)(c * nn + j) * s * A.B * A.tn
                           : A.part3 + (int64_t)(c * s + j) * (1 + nn) * A.B * A.tn;
  for (int q = wave; q < nq; q += NT / 64) {
    const int blk = prev ? (q < s ? q : q - s) : q;
    const bool fake = prev ? q < s : q > 0;
    float acc = 0.f;
    for (int b = lane; b < A.B; b += 64) {
      const float* pr = part + (int64_t)(blk * A.B + b) * A.tn;
      float a = 0.f;
      for (int t = 0; t < A.tn; ++t) a += pr[t];
      acc += fake ? fake_term(A.loss_kind, a) : real_term(A.loss_kind, a);
    }
    acc = wave_sum(acc);
    if (lane == 0) {
      const float m = acc / (float)A.B;
      if (prev) {
        if (q < s) A.L2[(c * s + q) * nn + j] = A.rmean[c * nn + j] + m;
        else A.Lg2[(c * s + q - s) * nn + j] = m;
      } else {
        A.M3[(c * (1 + nn) + q) * s + j] = m;  // q = 0: real rows; 1 + k: G_k's rows
      }
    }
  }
}

// thread (cell c, role): the elitist truncation of the cell's s previous and
// s trained individuals of the role
__global__ void elite_merge_kernel(EliteArgs A) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= 2 * A.C) return;
  const int c = A.c0 + (t >> 1), role = t & 1, s = A.s, nn = A.nn;
  float fo[4], fn[4];
  bool bad = false;
  for (int i = 0; i < s; ++i) {
    float acc = 0.f;
    if (role == 0) {
      const float* row = (A.mode == 0 ? A.L2 : A.Lg2) + (c * s + i) * nn;
      for (int j = 0; j < nn; ++j) acc += row[j];
      acc = A.mode == 0 ? -(acc / (float)nn) : acc / (float)nn;
      fo[i] = A.fit_g[c * nn + i];
    } else {
      const float* m = A.M3 + (int64_t)c * (1 + nn) * s;
      for (int k = 0; k < nn; ++k) acc += m[i] + m[(1 + k) * s + i];
      acc = acc / (float)nn;
      fo[i] = A.fit_d[c * nn + i];
    }
    fn[i] = acc;
    bad |= !isfinite(acc);
    float* out = role == 0 ? A.fit2_g : A.fit2_d;
    out[c * s + i] = acc;
    float* ext = role == 0 ? A.fit2_g_out : A.fit2_d_out;
    if (ext) ext[c * s + i] = acc;
  }
  if (bad) atomicOr(A.flags, 1);
  // rank of each of the 2 s candidates in the order (fitness, NaN last;
  // trained before previous; lower member first); the first s are kept
  int rank_new[4], rank_old[4];
  for (int r = 0; r < 2 * s; ++r) {
    const bool rn = r < s;
    const int ri = rn ? r : r - s;
    const float f = fit_key(rn ? fn[ri] : fo[ri]);
    int rank = 0;
    for (int q = 0; q < 2 * s; ++q) {
      const bool qn = q < s;
      const int qi = qn ? q : q - s;
      const float g = fit_key(qn ? fn[qi] : fo[qi]);
      rank += g < f || (g == f && (qn != rn ? qn : qi < ri));
    }
    if (rn) rank_new[ri] = rank;
    else rank_old[ri] = rank;
  }
  int kept_old[4], n_old = 0;
  for (int r = 0; r < s; ++r)
    for (int i = 0; i < s; ++i)
      if (rank_old[i] == r) kept_old[n_old++] = i;
  // the dropped trained slots, in slot order, take the kept previous members
  // in rank order
  int k = 0;
  for (int i = 0; i < s; ++i) {
    const int u = c * s + i;
    const int src = rank_new[i] < s ? -1 : c * s + kept_old[k++];
    A.src[u * 2 + role] = src;
    if (A.src_out) A.src_out[u * 2 + role] = src < 0 ? -1 : src - c * s;
    if (src >= 0) {
      A.t_new[role][u] = A.t_old[role][src];
      A.lr_new[role][u] = A.lr_old[role][src];
    }
  }
}

// block (x, u, role): p, m, v of individual sel[u][role] into individual u
__global__ void copy_winners_kernel(CopyArgs A) {
  const int u = blockIdx.y, role = blockIdx.z;
  const int src = A.sel[u * 2 + role];
  if (A.w_dst && role == 0 && u < A.C && blockIdx.x == 0 && threadIdx.x < 5)
    A.w_dst[u * 5 + threadIdx.x] = A.w_src[u * 5 + threadIdx.x];
  if (src < 0) return;
  const int64_t n4 = A.stride[role] >> 2;
  for (int a = 0; a < 3; ++a) {
    const float4* s = reinterpret_cast<const float4*>(A.src[role][a] + src * A.stride[role]);
    float4* d = reinterpret_cast<float4*>(A.dst[role][a] + u * A.stride[role]);
    for (int64_t q = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; q < n4;
         q += (int64_t)gridDim.x * blockDim.x)
      d[q] = s[q];
  }
}

// Per-cell feature moments over S samples: mu = mean f, s2 = mean f^2, summed
// in fp64 in a fixed order.  Stage 1, block (chunk, cell): 4 row lanes x 64
// features sum MOM_ROWS rows of a chunk, combined in lane order; stage 2,
// thread (cell, f) (grid-stride): the chunk sums in chunk order.
constexpr int MOM_ROWS = 64;

__global__ __launch_bounds__(NT) void moments_chunk_kernel(const float* feats, int S, int F, double* part) {
  __shared__ double red[2][4][64];
  const int chunk = blockIdx.x, c = blockIdx.y, n_chunks = gridDim.x;
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  for (int f0 = 0; f0 < F; f0 += 64) {
    const int f = f0 + l;
    double s = 0.0, q = 0.0;
    if (f < F) {
      const int r1 = min(S, (chunk + 1) * MOM_ROWS);
      for (int r = chunk * MOM_ROWS + w; r < r1; r += 4) {
        const double v = (double)feats[((int64_t)c * S + r) * F + f];
        s += v;
        q += v * v;
      }
    }
    __syncthreads();
    red[0][w][l] = s;
    red[1][w][l] = q;
    __syncthreads();
    if (w == 0 && f < F) {
      double* o = part + (((int64_t)c * n_chunks + chunk) * 2) * F;
      o[f] = (red[0][0][l] + red[0][1][l]) + (red[0][2][l] + red[0][3][l]);
      o[F + f] = (red[1][0][l] + red[1][1][l]) + (red[1][2][l] + red[1][3][l]);
    }
  }
}

__global__ void moments_final_kernel(const double* part, int n_chunks, int C, int S, int F, double* mu,
                                     double* s2) {
  const int64_t n = (int64_t)C * F;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = i / F, f = i - c * F;
    double s = 0.0, q = 0.0;
    for (int k = 0; k < n_chunks; ++k) {
      const double* o = part + ((c * n_chunks + k) * 2) * F;
      s += o[f];
      q += o[F + f];
    }
    mu[i] = s / (double)S;
    s2[i] = q / (double)S;
  }
}

// Column mean and (biased, two-pass) standard deviation over N rows, fp64.
__device__ double block_sum_f64(double v, double* red) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__global__ __launch_bounds__(NT) void col_stats_kernel(const float* feats, int64_t N, int F,
                                                       double* mu, double* sd) {
  __shared__ double red[4];
  const int f = blockIdx.x;
  double s = 0.0;
  for (int64_t r = threadIdx.x; r < N; r += NT) s += feats[r * F + f];
  const double mean = block_sum_f64(s, red) / (double)N;
  double q = 0.0;
  for (int64_t r = threadIdx.x; r < N; r += NT) {
    const double d = (double)feats[r * F + f] - mean;
    q += d * d;
  }
  const double var = block_sum_f64(q, red) / (double)N;
  if (threadIdx.x == 0) {
    mu[f] = mean;
    sd[f] = sqrt(var);
  }
}

// score(w) = sum_f (mu_w - mu_r)^2 + (sqrt(var_w) - sd_r)^2 with the mixture's
// mean mu_w = sum_k w_k mu_k and variance var_w = sum_k w_k s2_k - mu_w^2, in fp64.
__device__ double mixture_score(const double* w, const int32_t* ks, const double* mu, const double* s2,
                                const double* mu_r, const double* sd_r, int F) {
  double sc = 0.0;
  for (int f = 0; f < F; ++f) {
    double mw = 0.0, sw = 0.0;
    for (int k = 0; k < 5; ++k) {
      mw += w[k] * mu[(int64_t)ks[k] * F + f];
      sw += w[k] * s2[(int64_t)ks[k] * F + f];
    }
    const double var = fmax(sw - mw * mw, 0.0);
    const double dm = mw - mu_r[f], ds = sqrt(var) - sd_r[f];
    sc += dm * dm + ds * ds;
  }
  return sc;
}

// (1+1)-ES on the mixture weights of cell i.  The weights are stored in
// fp32; the proposal, both scores and the comparison are formed in fp64.
__global__ void es_kernel(EsArgs A) {
  const int c = A.c0 + blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= A.c0 + A.C) return;
  const int32_t* ks = A.nbr + c * 5;
  float w[5];
  double wd[5], wpd[5];
  for (int k = 0; k < 5; ++k) {
    w[k] = A.w[c * 5 + k];
    wd[k] = (double)w[k];
  }
  const uint4 w0 = stream_block(A.key, 0, (uint32_t)c, A.gen, 0, LIPZ_TAG_MIXN);
  const uint4 w1 = stream_block(A.key, 1, (uint32_t)c, A.gen, 0, LIPZ_TAG_MIXN);
  double tot = 0.0;
  for (int k = 0; k < 5; ++k) {
    const double n = k < 4 ? normal_of(w0, k) : normal_of(w1, 0);
    const double x = wd[k] + (double)A.sigma * n;
    wpd[k] = x > 0.0 ? x : 0.0;
    tot += wpd[k];
  }
  double cur = mixture_score(wd, ks, A.mu, A.s2, A.mu_r, A.sd_r, A.F);
  int acc = 0;
  if (tot > 0.0) {
    for (int k = 0; k < 5; ++k) wpd[k] /= tot;
    const double nw = mixture_score(wpd, ks, A.mu, A.s2, A.mu_r, A.sd_r, A.F);
    if (nw < cur) {
      cur = nw;
      acc = 1;
      for (int k = 0; k < 5; ++k) w[k] = (float)wpd[k];
    }
  }
  for (int k = 0; k < 5; ++k) {
    A.w[c * 5 + k] = w[k];
    if (A.w_out) A.w_out[c * 5 + k] = w[k];
  }
  if (A.score_out) A.score_out[c] = (float)cur;
  if (A.acc_out) A.acc_out[c] = acc;
}

int grid_for(int64_t n, int threads = NT, int cap = 8192) {
  int64_t b = (n + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

}  // namespace

hipError_t launch_init_params(float* p, int64_t stride, int64_t P, int C, NetLayers L, uint2 key,
                              uint32_t tag, hipStream_t s) {
  hipLaunchKernelGGL(init_params_kernel, dim3(grid_for((int64_t)C * P)), dim3(NT), 0, s, p, stride,
                     P, C, L, key, tag);
  return hipGetLastError();
}
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_f32_kernel, dim3(grid_for(n)), dim3(NT), 0, s, p, n, v);
  return hipGetLastError();
}
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(grid_for(n)), dim3(NT), 0, s, p, n, v);
  return hipGetLastError();
}
hipError_t launch_add_i32(int32_t* p, int n, int32_t v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(add_i32_kernel, dim3(grid_for(n)), dim3(NT), 0, s, p, n, v);
  return hipGetLastError();
}
hipError_t launch_normals(float* out, int64_t n, double scale, uint2 key, uint32_t cell,
                          uint32_t gen, uint32_t sf, uint32_t tag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(normals_kernel, dim3(grid_for(n)), dim3(NT), 0, s, out, n, scale, key, cell,
                     gen, sf, tag);
  return hipGetLastError();
}
hipError_t launch_sample(const float* data, int64_t N, int xd, int zd, int B, int c0, int C, uint2 key,
                         uint32_t gen, uint32_t sf, float* X, int64_t x_cell_stride, float* Z,
                         int64_t z_cell_stride, hipStream_t s) {
  hipLaunchKernelGGL(sample_kernel, dim3(B, C), dim3(NT), 0, s, data, N, xd, zd, c0, key, gen, sf, X,
                     x_cell_stride, Z, z_cell_stride);
  return hipGetLastError();
}
hipError_t launch_head_d(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(head_kernel<true>, dim3(a.C, (a.H + 63) / 64, (2 * a.B + HEAD_ROWS - 1) / HEAD_ROWS),
                     dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_head_g(const HeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(head_kernel<false>, dim3(a.C, (a.H + 63) / 64, (a.B + HEAD_ROWS - 1) / HEAD_ROWS),
                     dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_loss_d(const HeadArgs& a, hipStream_t s) {
  HeadArgs b = a;
  b.loss_only = 1;
  hipLaunchKernelGGL(head_kernel<true>, dim3(a.C, 1, 1), dim3(NT), 0, s, b);
  return hipGetLastError();
}
hipError_t launch_loss_g(const HeadArgs& a, hipStream_t s) {
  HeadArgs b = a;
  b.loss_only = 1;
  hipLaunchKernelGGL(head_kernel<false>, dim3(a.C, 1, 1), dim3(NT), 0, s, b);
  return hipGetLastError();
}
hipError_t launch_nes_perturb(const NesArgs& a, hipStream_t s) {
  const int64_t blocks = ((int64_t)a.n * a.P + 3) / 4;
  hipLaunchKernelGGL(nes_perturb_kernel, dim3((unsigned)((blocks + NT - 1) / NT), a.C), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_nes_head(const NesArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(nes_head_kernel, dim3(2 * a.n + 1, a.C), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_nes_update(const NesArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(nes_update_kernel, dim3((unsigned)((a.P + NT - 1) / NT), a.C), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_es_select(const NesArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(es_select_kernel, dim3((unsigned)((a.P + NT - 1) / NT), a.C), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_elite(const EliteArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(elite_means_kernel, dim3(a.nn + a.s, a.C), dim3(NT), 0, s, a);
  hipLaunchKernelGGL(elite_merge_kernel, dim3(grid_for(2 * a.C)), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_head_eval(const EvalHeadArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(head_eval_kernel, dim3(a.nn, a.C), dim3(NT), (1 + 2 * a.nn) * sizeof(float), s, a);
  return hipGetLastError();
}
hipError_t launch_fitness(const float* L, const float* Lg, int C, int nn, int mode, float* fit_g,
                          float* fit_d, int32_t* flags, float* oL, float* oLg, float* ofg,
                          float* ofd, hipStream_t s) {
  hipLaunchKernelGGL(fitness_kernel, dim3(grid_for((int64_t)C * nn * nn)), dim3(NT), 0, s, L, Lg, C, nn,
                     mode, fit_g, fit_d, flags, oL, oLg, ofg, ofd);
  return hipGetLastError();
}
hipError_t launch_select(const SelectArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(select_kernel, dim3(grid_for(2 * a.C * a.s)), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_copy_winners(const CopyArgs& a, hipStream_t s) {
  const int64_t n4 = (a.stride[0] > a.stride[1] ? a.stride[0] : a.stride[1]) >> 2;
  hipLaunchKernelGGL(copy_winners_kernel, dim3(grid_for(n4, NT, 64), a.U, 2), dim3(NT), 0, s, a);
  return hipGetLastError();
}
hipError_t launch_moments(const float* feats, int C, int S, int F, double* part, double* mu, double* s2,
                          hipStream_t s) {
  const int n_chunks = (S + MOM_ROWS - 1) / MOM_ROWS;
  hipLaunchKernelGGL(moments_chunk_kernel, dim3(n_chunks, C), dim3(NT), 0, s, feats, S, F, part);
  hipLaunchKernelGGL(moments_final_kernel, dim3(grid_for((int64_t)C * F)), dim3(NT), 0, s, part, n_chunks, C, S, F,
                     mu, s2);
  return hipGetLastError();
}
hipError_t launch_col_stats(const float* feats, int64_t N, int F, double* mu, double* sd,
                            hipStream_t s) {
  hipLaunchKernelGGL(col_stats_kernel, dim3(F), dim3(NT), 0, s, feats, N, F, mu, sd);
  return hipGetLastError();
}
hipError_t launch_es(const EsArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(es_kernel, dim3(grid_for(a.C, 64)), dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace lipz
