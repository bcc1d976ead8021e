// Host runtime of liblipz.so: configuration checks, workspace carving, the
// per-phase grouped-GEMM problem tables, and the C ABI of include/lipz.h.
//
// A generation of the grid is a fixed sequence of dependent phases (paper
// Section 3, steps 2-4).  Every phase is one kernel launch that covers all
// cells of the grid.  The GEMM problems of every phase are built once at
// create time, for both state buffers (generations are double-buffered), and
// uploaded into the workspace; a call only enqueues launches.
#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "grid.h"
#include "lipz_testing.h"

using namespace lipz;

#ifndef LIPZ_FUSED_SAMPLE
#define LIPZ_FUSED_SAMPLE 1  // draw the next step's minibatch inside a launch of the current one
#endif
#ifndef LIPZ_FUSED_HEAD
#define LIPZ_FUSED_HEAD 1
#endif

namespace {

// Workspace of lipz_grid_create_static: one array per device, held for the
// life of the process.  Host code never uses its name as an address: each
// device's copy is looked up once with hipGetSymbolAddress (that device
// current) and kept in g_static_ptr.
constexpr size_t kStaticWorkspaceBytes = LIPZ_STATIC_WORKSPACE_BYTES;
constexpr int kMaxStaticDevices = 64;
static __device__ __align__(256) char scratch[kStaticWorkspaceBytes];
std::mutex g_static_mu;
void* g_static_ptr[kMaxStaticDevices] = {};
bool g_static_busy[kMaxStaticDevices] = {};  // a live grid uses the device's array

}  // namespace

namespace lipz {

lipz_status fail(lipz_grid* g, lipz_status s, const std::string& msg) {
  if (g) g->last_err = msg;
  return s;
}

lipz_status check_hip(lipz_grid* g, hipError_t e, const char* what) {
  if (e == hipSuccess) return LIPZ_OK;
  g->sticky = LIPZ_E_HIP;
  g->last_err = std::string(what) + ": " + hipGetErrorString(e);
  return LIPZ_E_HIP;
}

bool valid_act(int a) { return a >= LIPZ_ACT_LINEAR && a <= LIPZ_ACT_TANH; }

// Validate a configuration; fills the network descriptions.  Returns "" if ok.
std::string validate(const lipz_config* c, int64_t n_samples, Net* Gn, Net* Dn) {
  if (!c) return "null config";
  if (c->abi_version != LIPZ_ABI_VERSION) return "abi_version mismatch";
  if (c->net != LIPZ_NET_MLP && c->net != LIPZ_NET_DCGAN) return "unknown net";
  if (c->rows < 1 || c->cols < 1 || (int64_t)c->rows * c->cols > 4096) return "grid size out of range";
  if (c->z_dim < 1 || c->x_dim < 1 || c->z_dim > 65536 || c->x_dim > (1 << 20)) return "bad z_dim / x_dim";
  if (c->batch < 1 || c->batch > 2048) return "batch must be in [1, 2048]";
  if (c->n_g_hidden < 1 || c->n_g_hidden > LIPZ_MAX_HIDDEN) return "n_g_hidden must be in [1, 4]";
  if (c->n_d_hidden < 1 || c->n_d_hidden > LIPZ_MAX_HIDDEN) return "n_d_hidden must be in [1, 4]";
  for (int i = 0; i < c->n_g_hidden; ++i)
    if (c->g_hidden[i] < 1 || c->g_hidden[i] > 65536) return "bad g_hidden width";
  for (int i = 0; i < c->n_d_hidden; ++i)
    if (c->d_hidden[i] < 1 || c->d_hidden[i] > 65536) return "bad d_hidden width";
  if (!valid_act(c->g_hidden_act) || !valid_act(c->g_out_act) || !valid_act(c->d_hidden_act))
    return "bad activation code";
  if (!(c->lrelu_slope > 0.f) || c->lrelu_slope >= 1.f) return "lrelu_slope must be in (0, 1)";
  if (c->tournament_size < 1 || c->tournament_size > 5) return "tournament_size must be in [1, 5]";
  if (c->fitness_mode != 0 && c->fitness_mode != 1) return "fitness_mode must be 0 or 1";
  if (c->loss_kind != LIPZ_LOSS_BCE && c->loss_kind != LIPZ_LOSS_WASSERSTEIN) return "unknown loss_kind";
  if (c->trainer != LIPZ_TRAINER_GRADIENT && c->trainer != LIPZ_TRAINER_NES && c->trainer != LIPZ_TRAINER_ES)
    return "unknown trainer";
  if (c->trainer != LIPZ_TRAINER_GRADIENT) {
    if (c->net != LIPZ_NET_MLP) return "the gradient-free trainers are implemented for the MLP networks";
    if (c->nes_pairs < 1 || c->nes_pairs > 64) return "nes_pairs must be in [1, 64]";
    if (!(c->nes_sigma > 0.f && c->nes_sigma < 1e30f)) return "nes_sigma must be a positive finite scale";
  }
  if (c->loss_kind == LIPZ_LOSS_WASSERSTEIN && !(c->wgan_clip > 0.f && c->wgan_clip < 1e30f))
    return "wgan_clip must be a positive finite bound";
  if (!(c->beta1 >= 0.f && c->beta1 < 1.f && c->beta2 >= 0.f && c->beta2 < 1.f && c->eps > 0.f))
    return "bad Adam constants";
  if (!(c->lr0_g >= 0.f && c->lr0_d >= 0.f)) return "learning rates must be >= 0";
  if (!(c->lr_mut_prob >= 0.f && c->lr_mut_prob <= 1.f && c->lr_mut_std >= 0.f))
    return "bad learning-rate mutation";
  if (c->mix_enable) {
    if (c->mix_samples < 1 || c->mix_samples > (1 << 20)) return "bad mix_samples";
    if (c->mix_feat_dim < 1 || c->mix_feat_dim > 4096) return "bad mix_feat_dim";
    if (!(c->mix_sigma >= 0.f)) return "bad mix_sigma";
  }
  if (c->pop_size < 1 || c->pop_size > 4) return "pop_size must be in [1, 4]";
  if (c->elitism != 0 && c->elitism != 1) return "elitism must be 0 or 1";
  if ((c->pop_size > 1 || c->elitism) && c->net != LIPZ_NET_MLP)
    return "sub-populations and elitism are implemented for the MLP networks";
  if (c->pop_size > 1 && c->mix_enable) return "the mixture step needs pop_size 1";
  if (c->bands < 0 || c->bands > LIPZ_MAX_BANDS || (c->bands > 1 && c->bands > c->rows))
    return "bands must be in [0, 8] and at most rows";
  if (c->bands > 1 && c->net != LIPZ_NET_MLP) return "row bands are implemented for the MLP networks";
  if ((int64_t)c->rows * c->cols * c->pop_size > 4096) return "grid size x pop_size out of range";
  if (n_samples < 1 || n_samples > ((int64_t)1 << 31) - 1) return "n_samples must be in [1, 2^31)";
  if (c->net == LIPZ_NET_DCGAN) return dc_validate(c, Gn, Dn);
  auto build = [](Net* n, int in, int nh, const int32_t* hid, int out, int hact, int oact) {
    int64_t off = 0;
    n->nl = nh + 1;
    for (int l = 0; l <= nh; ++l) {
      n->fi[l] = l == 0 ? in : hid[l - 1];
      n->fo[l] = l == nh ? out : hid[l];
      n->act[l] = l == nh ? oact : hact;
      n->off[l] = off;
      off += (int64_t)(n->fi[l] + 1) * n->fo[l];
    }
    n->P = off;
    n->stride = (int64_t)align_up((size_t)off, 64);
  };
  build(Gn, c->z_dim, c->n_g_hidden, c->g_hidden, c->x_dim, c->g_hidden_act, c->g_out_act);
  build(Dn, c->x_dim, c->n_d_hidden, c->d_hidden, 1, c->d_hidden_act, LIPZ_ACT_LINEAR);
  if (c->trainer != LIPZ_TRAINER_GRADIENT &&
      (int64_t)c->nes_pairs * (Gn->P > Dn->P ? Gn->P : Dn->P) >= ((int64_t)1 << 31))
    return "nes_pairs x parameters of a network must stay below 2^31";
  return "";
}

// The two state buffers in the documented blob layout.
void carve_state(lipz_grid* g, Carver& cv, char* base) {
  const int C = g->C, U = g->U;
  const Net &G = g->G, &D = g->D;
  for (int b = 0; b < 2; ++b) {
    StateBuf sb;
    const size_t start = align_up(cv.off, kAlign);
    cv.off = start;
    int64_t* so = g->state_off;
    auto take_f = [&](int k, size_t n) {
      cv.off = align_up(cv.off, kAlign);
      so[k] = (int64_t)(cv.off - start);
      return cv.take<float>(n);
    };
    auto take_i = [&](int k, size_t n) {
      cv.off = align_up(cv.off, kAlign);
      so[k] = (int64_t)(cv.off - start);
      return cv.take<int32_t>(n);
    };
    sb.base = base + start;
    sb.Gp = take_f(0, (size_t)U * G.stride);
    sb.Gm = take_f(1, (size_t)U * G.stride);
    sb.Gv = take_f(2, (size_t)U * G.stride);
    sb.Dp = take_f(3, (size_t)U * D.stride);
    sb.Dm = take_f(4, (size_t)U * D.stride);
    sb.Dv = take_f(5, (size_t)U * D.stride);
    sb.Gt = take_i(6, U);
    sb.Dt = take_i(7, U);
    sb.Glr = take_f(8, U);
    sb.Dlr = take_f(9, U);
    sb.w = take_f(10, (size_t)C * LIPZ_SLOTS);
    cv.off = align_up(cv.off, kAlign);
    so[11] = (int64_t)(cv.off - start);
    g->state_bytes = (size_t)so[11];
    g->gemm_wt = g->state_bytes <= ((size_t)128 << 20);
    g->st[b] = sb;
  }
}

// Carve every buffer; with base == nullptr only the size is computed.
void carve(lipz_grid* g, char* base, size_t* total) {
  Carver cv{base};
  const int C = g->C, B = g->B, zd = g->zd, xd = g->xd;
  const Net &G = g->G, &D = g->D;
  carve_state(g, cv, base);
  if (g->dc) {
    // grid-level buffers shared with the MLP path
    g->nbr = cv.take<int32_t>((size_t)C * 5);
    g->sel = cv.take<int32_t>((size_t)C * 2);
    g->flags = cv.take<int32_t>(4);
    g->L = cv.take<float>((size_t)C * 25);
    g->Lg = cv.take<float>((size_t)C * 25);
    g->fit_g = cv.take<float>((size_t)C * 5);
    g->fit_d = cv.take<float>((size_t)C * 5);
    dc_carve(g, cv);
    g->probs_d = cv.take<GemmProb>(g->probs_h.size());
    dc_carve_tables(g, cv);
    *total = align_up(cv.off, kAlign);
    return;
  }
  const int U = g->U, s = g->s, nn = g->nn, er = 1 + nn;  // er: evaluation row blocks per cell
  g->nbr = cv.take<int32_t>((size_t)C * 5);
  g->sel = cv.take<int32_t>((size_t)U * 2);
  g->flags = cv.take<int32_t>(4);
  g->L = cv.take<float>((size_t)C * nn * nn);
  g->Lg = cv.take<float>((size_t)C * nn * nn);
  g->fit_g = cv.take<float>((size_t)C * nn);
  g->fit_d = cv.take<float>((size_t)C * nn);
  // training (one unit per individual pair)
  g->z = cv.take<float>((size_t)U * B * zd);
  g->Xtr = cv.take<float>((size_t)U * 2 * B * xd);
  if (g->fused_sample) {
    g->z_alt = cv.take<float>((size_t)U * B * zd);
    g->Xtr_alt = cv.take<float>((size_t)U * 2 * B * xd);
  }
  for (int l = 0; l + 1 < G.nl; ++l) g->h[l] = cv.take<float>((size_t)U * B * G.fo[l]);
  for (int l = 0; l < G.nl; ++l) g->dG[l] = cv.take<float>((size_t)U * B * G.fo[l]);
  g->part_tr = cv.take<float>((size_t)U * 2 * B * g->tn);
  g->dlbuf = cv.take<float>((size_t)U * 2 * B * 4);
  g->part_g = cv.take<float>((size_t)U * B * g->tn);
  g->part_e = cv.take<float>((size_t)C * nn * er * B * g->tn);
  for (int l = 0; l + 1 < D.nl; ++l) {
    g->a[l] = cv.take<float>((size_t)U * 2 * B * D.fo[l]);
    g->dD[l] = cv.take<float>((size_t)U * 2 * B * D.fo[l]);
    g->ag[l] = cv.take<float>((size_t)U * B * D.fo[l]);
    g->dDg[l] = cv.take<float>((size_t)U * B * D.fo[l]);
  }
  if (g->fused_head) g->aS = cv.take<float>((size_t)U * 2 * B * g->aS_ld);
  if (g->hp_rows) g->hpart = cv.take<float>((size_t)U * g->hp_rows * g->hp_ld);
  // evaluation: rows [x_c; G_0(z_c); ...; G_(nn-1)(z_c)] per cell
  g->ze = cv.take<float>((size_t)C * B * zd);
  g->Xe = cv.take<float>((size_t)C * er * B * xd);
  for (int l = 0; l + 1 < G.nl; ++l) g->he[l] = cv.take<float>((size_t)C * nn * B * G.fo[l]);
  for (int l = 0; l + 1 < D.nl; ++l) g->ae[l] = cv.take<float>((size_t)C * nn * er * B * D.fo[l]);
  if (g->cfg.elitism) {
    g->rmean = cv.take<float>((size_t)C * nn);
    for (int l = 0; l + 1 < G.nl; ++l) g->he2[l] = cv.take<float>((size_t)C * s * B * G.fo[l]);
    g->xe2 = cv.take<float>((size_t)C * s * B * xd);
    for (int l = 0; l + 1 < D.nl; ++l) {
      g->ae2[l] = cv.take<float>((size_t)C * nn * s * B * D.fo[l]);
      g->ae3[l] = cv.take<float>((size_t)C * s * er * B * D.fo[l]);
    }
    g->part_e2 = cv.take<float>((size_t)C * nn * s * B * g->tn);
    g->part_e3 = cv.take<float>((size_t)C * s * er * B * g->tn);
    g->fit2_g = cv.take<float>((size_t)C * s);
    g->fit2_d = cv.take<float>((size_t)C * s);
    g->el_L2 = cv.take<float>((size_t)C * s * nn);
    g->el_Lg2 = cv.take<float>((size_t)C * s * nn);
    g->el_M3 = cv.take<float>((size_t)C * (1 + nn) * s);
    g->esrc = cv.take<int32_t>((size_t)U * 2);
  }
  // mixture
  if (g->cfg.mix_enable) {
    const int S = g->S, F = g->F;
    g->zeta = cv.take<float>((size_t)(g->n_bands > 1 ? g->n_bands : 1) * S * zd);  // one copy per row band
    for (int l = 0; l + 1 < G.nl; ++l) g->hm[l] = cv.take<float>((size_t)C * S * G.fo[l]);
    g->xm = cv.take<float>((size_t)C * S * xd);
    g->fm = cv.take<float>((size_t)C * S * F);
    g->mu_k = cv.take<double>((size_t)C * F);
    g->s2_k = cv.take<double>((size_t)C * F);
    g->mom_part = cv.take<double>((size_t)C * ((S + 63) / 64) * 2 * F);
    g->P = cv.take<float>((size_t)xd * F);
    g->mu_r = cv.take<double>(F);
    g->sd_r = cv.take<double>(F);
    g->realfeat = cv.take<float>((size_t)g->N * F);
  }
  if (g->cfg.trainer != LIPZ_TRAINER_GRADIENT) {
    const int Q = g->nes_q = 2 * g->cfg.nes_pairs + 1;
    // the perturbed sets (the unperturbed one is the parameters themselves),
    // and one direction buffer shared by the two roles, which run one after
    // the other on the stream
    g->nes_pd = cv.take<float>((size_t)U * (Q - 1) * D.stride);
    g->nes_pg = cv.take<float>((size_t)U * (Q - 1) * G.stride);
    if (g->cfg.trainer == LIPZ_TRAINER_NES) {  // the ES trainer keeps no directions
      g->nes_eps_stride = D.stride > G.stride ? D.stride : G.stride;
      g->nes_eps = cv.take<float>((size_t)U * g->cfg.nes_pairs * g->nes_eps_stride);
    }
    for (int l = 0; l + 1 < D.nl; ++l) {
      g->nes_aq[l] = cv.take<float>((size_t)U * Q * 2 * B * D.fo[l]);
      g->nes_agq[l] = cv.take<float>((size_t)U * Q * B * D.fo[l]);
    }
    for (int l = 0; l + 1 < G.nl; ++l) g->nes_hq[l] = cv.take<float>((size_t)U * Q * B * G.fo[l]);
    g->nes_xq = cv.take<float>((size_t)U * Q * B * xd);
    g->nes_part_d = cv.take<float>((size_t)U * Q * 2 * B * g->tn);
    g->nes_part_g = cv.take<float>((size_t)U * Q * B * g->tn);
    g->nes_fd = cv.take<float>((size_t)U * Q);
    g->nes_fg = cv.take<float>((size_t)U * Q);
  }
  g->probs_d = cv.take<GemmProb>(g->probs_h.size());
  *total = align_up(cv.off, kAlign);
}

int ceil_div(int a, int b) { return (a + b - 1) / b; }

int vec_flag(const float* p, int ld) {
  return (((uintptr_t)p & 15) == 0 && (ld & 3) == 0) ? 1 : 0;
}

GemmProb base_prob(const float* A, int lda, int a_trans, const float* Bm, int ldb, int b_trans,
                   float* C, int ldc, int M, int N, int K) {
  GemmProb p;
  memset(&p, 0, sizeof(p));
  p.A = A;
  p.B = Bm;
  p.C = C;
  p.M = M;
  p.N = N;
  p.K = K;
  p.lda = lda;
  p.ldb = ldb;
  p.ldc = ldc;
  p.a_trans = a_trans;
  p.b_trans = b_trans;
  p.a_rows = M;
  p.ones_row = -1;
  p.vec = vec_flag(A, lda) | (vec_flag(Bm, ldb) << 1);
  return p;
}

// y = act(x W + b): x [M][fi] (ld fi), Wb = W [fi][fo] then b [fo].
GemmProb fwd_prob(const float* x, int M, const float* Wb, int fi, int fo, float* y, int act) {
  GemmProb p = base_prob(x, fi, 0, Wb, fo, 0, y, fo, M, fo, fi);
  p.bias = Wb + (size_t)fi * fo;
  p.epi = EPI_BIAS_ACT;
  p.act = act;
  return p;
}

// Attach D's output layer (H -> 1, weights w then bias) to the forward
// problem of its last hidden layer: per-tile partial logits into part [M][tn].
GemmProb with_head(GemmProb p, const float* head, float* part, int tn) {
  p.dotw = head;
  p.dot_bias = head + p.N;
  p.dot_out = part;
  p.dot_ld = tn;
  return p;
}

// dx = (dy W^T) * act'(xfwd): dy [M][fo], W [fi][fo], dx and xfwd [M][fi].
GemmProb dgrad_prob(const float* dy, int M, const float* W, int fi, int fo, float* dx,
                    const float* xfwd, int act) {
  GemmProb p = base_prob(dy, fo, 0, W, fo, 1, dx, fi, M, fi, fo);
  p.aux = xfwd;
  p.epi = EPI_DACT;
  p.act = act;
  return p;
}

// (dW; db) = [x | 1]^T dy over `rows` samples, applied by Adam to (W; b).
GemmProb wgrad_adam_prob(const float* x, int rows, int fi, const float* dy, int fo, float* Wb,
                         float* m, float* v, const float* lr, const int32_t* t) {
  GemmProb p = base_prob(x, fi, 1, dy, fo, 0, Wb, fo, fi + 1, fo, rows);
  p.a_rows = fi;
  p.ones_row = fi;
  p.m = m;
  p.v = v;
  p.lr = lr;
  p.t = t;
  p.epi = EPI_ADAM;
  return p;
}

double prob_bytes(const GemmProb& p) {
  const double mn = (double)p.M * p.N;
  double b = (double)p.a_rows * p.K + (double)p.K * p.N;  // operands
  if (p.epi == EPI_ADAM) b += 6.0 * mn;                    // read p, m, v; write p, m, v
  else b += mn;                                            // write C
  if (p.epi == EPI_DACT) b += mn;                          // read the forward output
  if (p.epi == EPI_BIAS_ACT && p.bias) b += p.N;
  if (p.epi == EPI_BIAS_ACT && p.dot_out) b += (double)p.M * ((p.N + GEMM_BN - 1) / GEMM_BN) + p.N;
  if (p.epi == EPI_BIAS_ACT && p.dot_out && p.gout) b += mn;  // write w * act'
  if (p.epi == EPI_DACT && p.rs_mode) {
    b += (double)p.M * p.rs_tn;                                // read the partial logits
    if (p.side) b += mn + 8.0 * p.M;                           // scaled activations, dL/da, dlout
    if (p.rs_mode == 1 && p.hpart)                             // output layer's gradient pieces
      b += (double)p.M * p.hp_w + (double)((p.M + 31) / 32) * (p.hp_w + 1);
  }
  return 4.0 * b;
}

double prob_flops(const GemmProb& p) {
  const double rows = p.ones_row >= 0 ? (double)p.a_rows : (double)p.M;
  return 2.0 * rows * p.N * p.K;
}

int add_phase(lipz_grid* g, const std::vector<GemmProb>& ps) {
  Phase ph;
  ph.first = (int)g->probs_h.size();
  ph.count = (int)ps.size();
  int tiles64 = 0;
  for (const GemmProb& p : ps) tiles64 += ceil_div(p.M, 64) * ceil_div(p.N, GEMM_BN);
  ph.tile_rows = gemm_tile_rows(tiles64);
  int max_k = 0;
  for (const GemmProb& p : ps) max_k = p.K > max_k ? p.K : max_k;
  int tiles = 0;
  memset(&ph.grp, 0, sizeof(ph.grp));
  int prev_tpp = -1, prev_k = -1;
  for (size_t k = 0; k < ps.size(); ++k) {
    GemmProb p = ps[k];
    p.slope = g->slope;
    p.ac = g->ac;
    // the epilogue addresses C (and aux, m, v) through buffer resources with
    // 32-bit byte offsets 4 (row * ldc + col) below 2^31: a problem whose
    // output reaches 2^29 elements (2 GiB) is not planned (the configuration
    // is rejected as invalid)
    if ((int64_t)(p.M - 1) * p.ldc + p.N >= ((int64_t)1 << 29)) {
      g->plan_ok = false;
      break;
    }
    gemm_set_extents(p);
    ph.fast = ph.fast && gemm_fast_ok(p);
    p.tiles_n = ceil_div(p.N, GEMM_BN);
    p.tile_begin = tiles;
    const int tpp = ceil_div(p.M, ph.tile_rows) * p.tiles_n;
    // a new group at every change of tile count (needed) and, while groups
    // are left, of depth K (tiles of different cost are then spread over the
    // XCDs separately)
    if (tpp != prev_tpp || (p.K != prev_k && ph.grp.n < GEMM_MAX_GROUPS)) {
      // the problem lists built here have at most 3 tile counts per phase
      if (ph.grp.n == GEMM_MAX_GROUPS) {  // a plan this library builds never gets here
        g->plan_ok = false;
        break;
      }
      ph.grp.first_tile[ph.grp.n] = tiles;
      ph.grp.first_prob[ph.grp.n] = (int)k;
      ph.grp.tiles_per_prob[ph.grp.n] = tpp;
      ++ph.grp.n;
      prev_tpp = tpp;
    }
    prev_k = p.K;
    tiles += tpp;
    ph.flops += prob_flops(p);
    ph.bytes += prob_bytes(p);
    g->probs_h.push_back(p);
  }
  ph.tiles = tiles;
  ph.kernel = gemm_choose_kernel(ph.fast, max_k);
  g->phases.push_back(ph);
  return (int)g->phases.size() - 1;
}

// The backward schedule shared by both networks: the weight gradient of
// layer l + 1 (which rewrites W_{l+1}) runs beside the input gradient of
// layer l (which reads W_l), never beside the one of its own layer.
template <class Dgrad, class Wgrad>
void backward_phases(lipz_grid* g, int top, Dgrad dgrad, Wgrad wgrad, std::vector<Op>* ops,
                     const std::vector<GemmProb>& extra_first = {}) {
  std::vector<GemmProb> pending;
  for (int l = top; l >= 0; --l) {
    std::vector<GemmProb> ph;
    if (l >= 1) dgrad(l, &ph);
    if (l == top) ph.insert(ph.end(), extra_first.begin(), extra_first.end());
    ph.insert(ph.end(), pending.begin(), pending.end());
    pending.clear();
    wgrad(l, &pending);
    if (l == 0) ph.insert(ph.end(), pending.begin(), pending.end());
    ops->push_back({OP_GEMM, add_phase(g, ph)});
  }
}


void setup_groups(lipz_grid* g) {
  if (g->cfg.bands >= 2) {
    // row bands: rows split as evenly as possible; the training groups are
    // the bands' individuals
    const int R = g->cfg.rows, Q = g->cfg.cols, nb = g->cfg.bands;
    g->n_bands = nb;
    for (int b = 0; b <= nb; ++b) g->band_c0[b] = (int)((int64_t)R * b / nb) * Q;
    for (int b = 0; b < nb; ++b) {
      uint32_t m = 0;
      for (int c = g->band_c0[b]; c < g->band_c0[b + 1]; ++c)
        for (int k = 0; k < LIPZ_SLOTS; ++k) {
          const int cn = g->nbr_h[c * LIPZ_SLOTS + k];
          for (int b2 = 0; b2 < nb; ++b2)
            if (cn >= g->band_c0[b2] && cn < g->band_c0[b2 + 1]) m |= 1u << b2;
        }
      g->band_wait[b] = m;
    }
    g->n_groups = nb;
    for (int b = 0; b <= nb; ++b) g->group_c0[b] = g->band_c0[b] * g->s;
    return;
  }
  // Measured on the 4x4 MNIST-shaped grid: 1, 2 and 4 groups are within a
  // few percent of each other, so by default one stream keeps the phases
  // in a single dependency chain.
  int n = LIPZ_CELL_GROUPS;
  if (n <= 0) n = 1;
  if (n > 4) n = 4;
  if (n > g->U) n = g->U;
  g->n_groups = n;
  for (int i = 0; i <= n; ++i) g->group_c0[i] = (int)((int64_t)g->U * i / n);
}

// The gradient-free trainers' step (reading of Section 3's NES and ES
// trainers; the ES trainer's last op of each role is the plus-selection):
// sample; G forward (its samples score the critic's perturbations); the
// discriminator's Q parameter sets, each D forward over the 2B rows, their
// losses, the estimate + Adam; then the generator's Q sets, each G forward,
// the updated D over all Q B generated rows, their losses, estimate + Adam.
// Training units u0 .. u1 - 1 of state buffer par.
void build_nes_ops_range(lipz_grid* g, int par, int u0, int u1, std::vector<Op>& ops) {
  const int B = g->B, zd = g->zd, xd = g->xd, Q = g->nes_q;
  const Net &G = g->G, &D = g->D;
  const int LG = G.nl, LD = D.nl;
  const size_t sG = G.stride, sD = D.stride;
  {
    const StateBuf& S = g->st[par];
    ops.clear();
    ops.push_back({OP_SAMPLE, -1});
    for (int l = 0; l < LG; ++l) {
      std::vector<GemmProb> ps;
      for (int c = u0; c < u1; ++c) {
        const float* x = l == 0 ? g->z + (size_t)c * B * zd : g->h[l - 1] + (size_t)c * B * G.fi[l];
        float* y = l + 1 < LG ? g->h[l] + (size_t)c * B * G.fo[l]
                              : g->Xtr + (size_t)c * 2 * B * xd + (size_t)B * xd;
        ps.push_back(fwd_prob(x, B, S.Gp + c * sG + G.off[l], G.fi[l], G.fo[l], y, G.act[l]));
      }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    ops.push_back({OP_NES_PERTURB, LIPZ_ROLE_D});
    for (int l = 0; l + 1 < LD; ++l) {
      std::vector<GemmProb> ps;
      for (int c = u0; c < u1; ++c)
        for (int q = 0; q < Q; ++q) {
          const size_t cq = (size_t)c * Q + q;
          const float* W = q + 1 < Q ? g->nes_pd + ((size_t)c * (Q - 1) + q) * sD : S.Dp + c * sD;
          const float* x = l == 0 ? g->Xtr + (size_t)c * 2 * B * xd : g->nes_aq[l - 1] + cq * 2 * B * D.fi[l];
          GemmProb p = fwd_prob(x, 2 * B, W + D.off[l], D.fi[l], D.fo[l], g->nes_aq[l] + cq * 2 * B * D.fo[l],
                                D.act[l]);
          if (l == LD - 2) p = with_head(p, W + D.off[LD - 1], g->nes_part_d + cq * 2 * B * g->tn, g->tn);
          ps.push_back(p);
        }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    ops.push_back({OP_NES_HEAD, LIPZ_ROLE_D});
    ops.push_back({OP_NES_UPDATE, LIPZ_ROLE_D});
    ops.push_back({OP_NES_PERTURB, LIPZ_ROLE_G});
    for (int l = 0; l < LG; ++l) {
      std::vector<GemmProb> ps;
      for (int c = u0; c < u1; ++c)
        for (int q = 0; q < Q; ++q) {
          const size_t cq = (size_t)c * Q + q;
          const float* x = l == 0 ? g->z + (size_t)c * B * zd : g->nes_hq[l - 1] + cq * B * G.fi[l];
          float* y = l + 1 < LG ? g->nes_hq[l] + cq * B * G.fo[l] : g->nes_xq + cq * B * xd;
          const float* W = q + 1 < Q ? g->nes_pg + ((size_t)c * (Q - 1) + q) * sG : S.Gp + c * sG;
          ps.push_back(fwd_prob(x, B, W + G.off[l], G.fi[l], G.fo[l], y, G.act[l]));
        }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    for (int l = 0; l + 1 < LD; ++l) {
      std::vector<GemmProb> ps;
      for (int c = u0; c < u1; ++c) {
        const float* x = l == 0 ? g->nes_xq + (size_t)c * Q * B * xd : g->nes_agq[l - 1] + (size_t)c * Q * B * D.fi[l];
        GemmProb p = fwd_prob(x, Q * B, S.Dp + c * sD + D.off[l], D.fi[l], D.fo[l],
                              g->nes_agq[l] + (size_t)c * Q * B * D.fo[l], D.act[l]);
        if (l == LD - 2)
          p = with_head(p, S.Dp + c * sD + D.off[LD - 1], g->nes_part_g + (size_t)c * Q * B * g->tn, g->tn);
        ps.push_back(p);
      }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    ops.push_back({OP_NES_HEAD, LIPZ_ROLE_G});
    ops.push_back({OP_NES_UPDATE, LIPZ_ROLE_G});
  }
}

void build_nes_ops(lipz_grid* g) {
  for (int par = 0; par < 2; ++par) {
    build_nes_ops_range(g, par, 0, g->U, g->nes_ops[par]);
    for (int b = 0; b < g->n_bands; ++b)
      build_nes_ops_range(g, par, g->band_c0[b] * g->s, g->band_c0[b + 1] * g->s, g->nes_band_ops[par][b]);
  }
}

void build_tables(lipz_grid* g) {
  g->probs_h.clear();
  g->phases.clear();
  const int C = g->C, B = g->B, zd = g->zd, xd = g->xd;
  const Net &G = g->G, &D = g->D;
  const int LG = G.nl, LD = D.nl;
  const size_t sG = G.stride, sD = D.stride;
  // the Wasserstein critic's parameters are clipped after every update
  const float d_clip = g->cfg.loss_kind == LIPZ_LOSS_WASSERSTEIN ? g->cfg.wgan_clip : 0.f;
  const bool fused = g->fused_head;
  for (int par = 0; par < 2; ++par) {
    const StateBuf& S = g->st[par];
    for (int grp = 0; grp < g->n_groups; ++grp)
    // with the minibatch drawn one step ahead, steps alternate between two
    // buffers of minibatch and latents: the odd steps have their own tables
    for (int sp = 0; sp < (g->fused_sample ? 2 : 1); ++sp) {
    const int cb = g->group_c0[grp], ce = g->group_c0[grp + 1];
    std::vector<Op>& ops = sp ? g->train_ops_odd[par][grp] : g->train_ops[par][grp];
    float* const Zb = sp ? g->z_alt : g->z;
    float* const Xb = sp ? g->Xtr_alt : g->Xtr;
    ops.clear();
    // ---- training step ----
    ops.push_back({OP_SAMPLE, -1});
    for (int l = 0; l < LG; ++l) {
      std::vector<GemmProb> ps;
      for (int c = cb; c < ce; ++c) {
        const float* x = l == 0 ? Zb + (size_t)c * B * zd : g->h[l - 1] + (size_t)c * B * G.fi[l];
        float* y = l + 1 < LG ? g->h[l] + (size_t)c * B * G.fo[l]
                              : Xb + (size_t)c * 2 * B * xd + (size_t)B * xd;
        ps.push_back(fwd_prob(x, B, S.Gp + c * sG + G.off[l], G.fi[l], G.fo[l], y, G.act[l]));
      }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    for (int l = 0; l + 1 < LD; ++l) {
      std::vector<GemmProb> ps;
      for (int c = cb; c < ce; ++c) {
        const float* x = l == 0 ? Xb + (size_t)c * 2 * B * xd
                                : g->a[l - 1] + (size_t)c * 2 * B * D.fi[l];
        GemmProb p = fwd_prob(x, 2 * B, S.Dp + c * sD + D.off[l], D.fi[l], D.fo[l],
                              g->a[l] + (size_t)c * 2 * B * D.fo[l], D.act[l]);
        if (l == LD - 2) {
          p = with_head(p, S.Dp + c * sD + D.off[LD - 1], g->part_tr + (size_t)c * 2 * B * g->tn, g->tn);
          if (fused) p.gout = g->dD[LD - 2] + (size_t)c * 2 * B * D.fo[l];
        }
        ps.push_back(p);
      }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    if (!fused) ops.push_back({OP_HEAD_D, -1});
    // output layer of D: ([act | 1]^T dL/da) and its Adam step, as GEMM problems
    std::vector<GemmProb> head_grad;
    for (int c = cb; c < ce; ++c) {
      const int H = D.fi[LD - 1];
      const size_t o = c * sD + D.off[LD - 1];
      GemmProb p = base_prob(g->a[LD - 2] + (size_t)c * 2 * B * H, H, 1, g->dlbuf + (size_t)c * 2 * B * 4, 4,
                             0, S.Dp + o, 1, H + 1, 1, 2 * B);
      p.a_rows = H;
      p.ones_row = H;
      p.m = S.Dm + o;
      p.v = S.Dv + o;
      p.lr = S.Dlr + c;
      p.t = S.Dt + c;
      p.epi = EPI_ADAM;
      p.clip = d_clip;
      if (g->cfg.loss_kind == LIPZ_LOSS_WASSERSTEIN) p.gscale = 1.f / (float)B;  // dL/da stored as exact +-1
      head_grad.push_back(p);
    }
    auto d_dgrad = [&](int l, std::vector<GemmProb>* ph) {
      for (int c = cb; c < ce; ++c)
        ph->push_back(dgrad_prob(g->dD[l] + (size_t)c * 2 * B * D.fo[l], 2 * B,
                                 S.Dp + c * sD + D.off[l], D.fi[l], D.fo[l],
                                 g->dD[l - 1] + (size_t)c * 2 * B * D.fi[l],
                                 g->a[l - 1] + (size_t)c * 2 * B * D.fi[l], D.act[l - 1]));
    };
    auto d_wgrad = [&](int l, std::vector<GemmProb>* ph) {
      for (int c = cb; c < ce; ++c) {
        const float* x = l == 0 ? Xb + (size_t)c * 2 * B * xd
                                : g->a[l - 1] + (size_t)c * 2 * B * D.fi[l];
        const size_t o = c * sD + D.off[l];
        GemmProb p = wgrad_adam_prob(x, 2 * B, D.fi[l], g->dD[l] + (size_t)c * 2 * B * D.fo[l],
                                     D.fo[l], S.Dp + o, S.Dm + o, S.Dv + o, S.Dlr + c, S.Dt + c);
        p.clip = d_clip;
        ph->push_back(p);
      }
    };
    if (!fused) {
      backward_phases(g, LD - 2, d_dgrad, d_wgrad, &ops, head_grad);
    } else {
      // The loss head inside the launches: with g = w (.) act'(h) (written by the
      // last hidden layer's forward) the head's delta of that layer is the row
      // scaling diag(dL/da) g, so
      //   input gradient  (diag(dL/da) g) W^T (.) act'(a) = diag(dL/da) (g W^T) (.) act'(a)
      //   weight gradient [a | 1]^T diag(dL/da) g = [diag(dL/da) a | dL/da]^T g
      // the first launch forms dL/da from the partial logits, the scaled
      // activations aS and the output layer's dL/da; the next one takes both
      // weight gradients (that layer's and the output layer's).
      const int t = LD - 2, Hs = D.fi[t], H = D.fo[t];
      std::vector<GemmProb> ph;
      for (int c = cb; c < ce; ++c) {
        GemmProb p = dgrad_prob(g->dD[t] + (size_t)c * 2 * B * H, 2 * B, S.Dp + c * sD + D.off[t], Hs, H,
                                g->dD[t - 1] + (size_t)c * 2 * B * Hs, g->a[t - 1] + (size_t)c * 2 * B * Hs,
                                D.act[t - 1]);
        p.rs_part = g->part_tr + (size_t)c * 2 * B * g->tn;
        p.rs_tn = g->tn;
        p.rs_mode = 1;
        p.rs_B = B;
        p.loss_kind = g->cfg.loss_kind;
        p.side = g->aS + (size_t)c * 2 * B * g->aS_ld;
        p.side_ld = g->aS_ld;
        p.dlout = g->dlbuf + (size_t)c * 2 * B * 4;
        if (g->hpart) {
          p.hpart = g->hpart + (size_t)c * g->hp_rows * g->hp_ld;
          p.hsrc = g->a[t] + (size_t)c * 2 * B * H;
          p.hp_w = H;
          p.hp_ld = g->hp_ld;
        }
        ph.push_back(p);
      }
      const int dgrad_phase = add_phase(g, ph);
      ops.push_back({OP_GEMM, dgrad_phase});
      if (g->hpart) {
        // the output layer's weight gradient from the per-row-tile column
        // sums: [w | b] = 1^T hpart over the launch's row tiles (a 1-row
        // product whose A is the all-ones row), and its Adam step
        const int rt = ceil_div(2 * B, g->phases[dgrad_phase].tile_rows);
        head_grad.clear();
        for (int c = cb; c < ce; ++c) {
          const size_t o = c * sD + D.off[LD - 1];
          float* hp = g->hpart + (size_t)c * g->hp_rows * g->hp_ld;
          GemmProb p = base_prob(hp, g->hp_ld, 1, hp, g->hp_ld, 0, S.Dp + o, H + 1, 1, H + 1, rt);
          p.a_rows = 0;
          p.ones_row = 0;
          p.m = S.Dm + o;
          p.v = S.Dv + o;
          p.lr = S.Dlr + c;
          p.t = S.Dt + c;
          p.epi = EPI_ADAM;
          p.clip = d_clip;
          if (g->cfg.loss_kind == LIPZ_LOSS_WASSERSTEIN) p.gscale = 1.f / (float)B;  // sums of exact +-1
          head_grad.push_back(p);
        }
      }
      std::vector<GemmProb> pending;
      for (int c = cb; c < ce; ++c) {
        const size_t o = c * sD + D.off[t];
        GemmProb p = base_prob(g->aS + (size_t)c * 2 * B * g->aS_ld, g->aS_ld, 1, g->dD[t] + (size_t)c * 2 * B * H,
                               H, 0, S.Dp + o, H, Hs + 1, H, 2 * B);
        p.a_rows = Hs + 1;  // the dL/da column is the bias row
        p.m = S.Dm + o;
        p.v = S.Dv + o;
        p.lr = S.Dlr + c;
        p.t = S.Dt + c;
        p.epi = EPI_ADAM;
        p.clip = d_clip;
        pending.push_back(p);
      }
      for (int l = t - 1; l >= 0; --l) {
        std::vector<GemmProb> q;
        if (l >= 1) d_dgrad(l, &q);
        q.insert(q.end(), pending.begin(), pending.end());
        pending.clear();
        d_wgrad(l, &pending);
        if (l == 0) q.insert(q.end(), pending.begin(), pending.end());
        ops.push_back({OP_GEMM, add_phase(g, q)});
      }
    }
    // generator step: D forward on the fake rows with the updated D
    for (int l = 0; l + 1 < LD; ++l) {
      std::vector<GemmProb> ps;
      // with the head folded in, the output layer's weight gradient + Adam
      // (it needs the dL/da of the input-gradient launch) runs beside the
      // first layer's forward on the fakes, before the output layer is read
      if (fused && l == 0) ps = head_grad;
      for (int c = cb; c < ce; ++c) {
        const float* x = l == 0 ? Xb + (size_t)c * 2 * B * xd + (size_t)B * xd
                                : g->ag[l - 1] + (size_t)c * B * D.fi[l];
        GemmProb p = fwd_prob(x, B, S.Dp + c * sD + D.off[l], D.fi[l], D.fo[l],
                              g->ag[l] + (size_t)c * B * D.fo[l], D.act[l]);
        if (l == LD - 2) {
          p = with_head(p, S.Dp + c * sD + D.off[LD - 1], g->part_g + (size_t)c * B * g->tn, g->tn);
          if (fused) p.gout = g->dDg[LD - 2] + (size_t)c * B * D.fo[l];
        }
        ps.push_back(p);
      }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
    }
    if (!fused) ops.push_back({OP_HEAD_G, -1});
    for (int l = LD - 2; l >= 0; --l) {
      std::vector<GemmProb> ps;
      for (int c = cb; c < ce; ++c) {
        if (l >= 1) {
          GemmProb p = dgrad_prob(g->dDg[l] + (size_t)c * B * D.fo[l], B, S.Dp + c * sD + D.off[l],
                                  D.fi[l], D.fo[l], g->dDg[l - 1] + (size_t)c * B * D.fi[l],
                                  g->ag[l - 1] + (size_t)c * B * D.fi[l], D.act[l - 1]);
          if (fused && l == LD - 2) {  // the generator step's head: every row has the "real" target
            p.rs_part = g->part_g + (size_t)c * B * g->tn;
            p.rs_tn = g->tn;
            p.rs_mode = 2;
            p.rs_B = B;
            p.loss_kind = g->cfg.loss_kind;
          }
          ps.push_back(p);
        } else {
          // into the generator output: delta of G's last layer
          ps.push_back(dgrad_prob(g->dDg[0] + (size_t)c * B * D.fo[0], B, S.Dp + c * sD + D.off[0],
                                  D.fi[0], D.fo[0], g->dG[LG - 1] + (size_t)c * B * xd,
                                  Xb + (size_t)c * 2 * B * xd + (size_t)B * xd, G.act[LG - 1]));
        }
      }
      ops.push_back({OP_GEMM, add_phase(g, ps)});
      // this launch (832 tiles at the 4x4 grid's shapes, about 450 workgroup
      // slots free) also draws the next step's minibatch
      if (l == 0 && g->fused_sample) ops.back().sample_next = 1;
    }
    backward_phases(
        g, LG - 1,
        [&](int l, std::vector<GemmProb>* ph) {
          for (int c = cb; c < ce; ++c)
            ph->push_back(dgrad_prob(g->dG[l] + (size_t)c * B * G.fo[l], B, S.Gp + c * sG + G.off[l],
                                     G.fi[l], G.fo[l], g->dG[l - 1] + (size_t)c * B * G.fi[l],
                                     g->h[l - 1] + (size_t)c * B * G.fi[l], G.act[l - 1]));
        },
        [&](int l, std::vector<GemmProb>* ph) {
          for (int c = cb; c < ce; ++c) {
            const float* x = l == 0 ? Zb + (size_t)c * B * zd : g->h[l - 1] + (size_t)c * B * G.fi[l];
            const size_t o = c * sG + G.off[l];
            ph->push_back(wgrad_adam_prob(x, B, G.fi[l], g->dG[l] + (size_t)c * B * G.fo[l], G.fo[l],
                                          S.Gp + o, S.Gm + o, S.Gv + o, S.Glr + c, S.Gt + c));
          }
        },
        &ops);
    // with the head folded in, the step's losses (when asked for) come from a
    // small kernel over the partial logits at the end of the step
    if (fused) {
      ops.push_back({OP_LOSS_D, -1});
      ops.push_back({OP_LOSS_G, -1});
    }
    }  // groups and step parities

    // ---- evaluation: rows [x_c; G_0(z_c); ...; G_(nn-1)(z_c)] per cell ----
    const int s = g->s, nn = g->nn, er = 1 + nn;
    auto owner_of = [&](int c, int i) { return g->nbr_h[c * 5 + i / s] * s + i % s; };
    auto eval_phases = [&](int cb, int ce, std::vector<int>& ev) {
      ev.clear();
      for (int l = 0; l < LG; ++l) {
        std::vector<GemmProb> ps;
        for (int c = cb; c < ce; ++c)
          for (int i = 0; i < nn; ++i) {
            const int owner = owner_of(c, i);
            const float* x = l == 0 ? g->ze + (size_t)c * B * zd
                                    : g->he[l - 1] + (size_t)(c * nn + i) * B * G.fi[l];
            float* y = l + 1 < LG ? g->he[l] + (size_t)(c * nn + i) * B * G.fo[l]
                                  : g->Xe + (size_t)c * er * B * xd + (size_t)(1 + i) * B * xd;
            ps.push_back(fwd_prob(x, B, S.Gp + owner * sG + G.off[l], G.fi[l], G.fo[l], y, G.act[l]));
          }
        ev.push_back(add_phase(g, ps));
      }
      for (int l = 0; l + 1 < LD; ++l) {
        std::vector<GemmProb> ps;
        for (int c = cb; c < ce; ++c)
          for (int j = 0; j < nn; ++j) {
            const int owner = owner_of(c, j);
            const float* x = l == 0 ? g->Xe + (size_t)c * er * B * xd
                                    : g->ae[l - 1] + (size_t)(c * nn + j) * er * B * D.fi[l];
            GemmProb p = fwd_prob(x, er * B, S.Dp + owner * sD + D.off[l], D.fi[l], D.fo[l],
                                  g->ae[l] + (size_t)(c * nn + j) * er * B * D.fo[l], D.act[l]);
            if (l == LD - 2)
              p = with_head(p, S.Dp + owner * sD + D.off[LD - 1],
                            g->part_e + (size_t)(c * nn + j) * er * B * g->tn, g->tn);
            ps.push_back(p);
          }
        ev.push_back(add_phase(g, ps));
      }
    };
    // ---- post-training re-evaluation (elitism): this buffer holds the trained
    // individuals, the other one the previous state ----
    auto elite_phases = [&](int cb, int ce, std::vector<int>& el) {
      el.clear();
      const StateBuf& O = g->st[1 - par];
      for (int l = 0; l < LG; ++l) {  // trained G'_i on the cell's evaluation latents
        std::vector<GemmProb> ps;
        for (int c = cb; c < ce; ++c)
          for (int i = 0; i < s; ++i) {
            const size_t ci = (size_t)c * s + i;
            const float* x = l == 0 ? g->ze + (size_t)c * B * zd : g->he2[l - 1] + ci * B * G.fi[l];
            float* y = l + 1 < LG ? g->he2[l] + ci * B * G.fo[l] : g->xe2 + ci * B * xd;
            ps.push_back(fwd_prob(x, B, S.Gp + ci * sG + G.off[l], G.fi[l], G.fo[l], y, G.act[l]));
          }
        el.push_back(add_phase(g, ps));
      }
      for (int l = 0; l + 1 < LD; ++l) {
        // one phase, two problem shapes (all cells' first kind, then the second)
        std::vector<GemmProb> ps;
        for (int c = cb; c < ce; ++c)
          for (int j = 0; j < nn; ++j) {  // previous D_j on the s B rows of the trained generators
            const int owner = owner_of(c, j);
            const size_t cj = (size_t)c * nn + j;
            const float* x = l == 0 ? g->xe2 + (size_t)c * s * B * xd : g->ae2[l - 1] + cj * s * B * D.fi[l];
            GemmProb p = fwd_prob(x, s * B, O.Dp + owner * sD + D.off[l], D.fi[l], D.fo[l],
                                  g->ae2[l] + cj * s * B * D.fo[l], D.act[l]);
            if (l == LD - 2)
              p = with_head(p, O.Dp + owner * sD + D.off[LD - 1], g->part_e2 + cj * s * B * g->tn, g->tn);
            ps.push_back(p);
          }
        for (int c = cb; c < ce; ++c)
          for (int j = 0; j < s; ++j) {  // trained D'_j on the evaluation rows
            const size_t cj = (size_t)c * s + j;
            const float* x = l == 0 ? g->Xe + (size_t)c * er * B * xd : g->ae3[l - 1] + cj * er * B * D.fi[l];
            GemmProb p = fwd_prob(x, er * B, S.Dp + cj * sD + D.off[l], D.fi[l], D.fo[l],
                                  g->ae3[l] + cj * er * B * D.fo[l], D.act[l]);
            if (l == LD - 2)
              p = with_head(p, S.Dp + cj * sD + D.off[LD - 1], g->part_e3 + cj * er * B * g->tn, g->tn);
            ps.push_back(p);
          }
        el.push_back(add_phase(g, ps));
      }
    };
    eval_phases(0, C, g->eval_phases[par]);
    g->elite_phases[par].clear();
    if (g->cfg.elitism) elite_phases(0, C, g->elite_phases[par]);
    for (int b = 0; b < g->n_bands; ++b) {  // the same plans per row band
      eval_phases(g->band_c0[b], g->band_c0[b + 1], g->band_eval_phases[par][b]);
      g->band_elite_phases[par][b].clear();
      if (g->cfg.elitism) elite_phases(g->band_c0[b], g->band_c0[b + 1], g->band_elite_phases[par][b]);
    }
    // ---- mixture ----
    auto mix_phases = [&](int cb, int ce, const float* zeta, std::vector<int>& mx) {
      mx.clear();
      const int Sm = g->S, F = g->F;
      for (int l = 0; l < LG; ++l) {
        std::vector<GemmProb> ps;
        for (int c = cb; c < ce; ++c) {
          const float* x = l == 0 ? zeta : g->hm[l - 1] + (size_t)c * Sm * G.fi[l];
          float* y = l + 1 < LG ? g->hm[l] + (size_t)c * Sm * G.fo[l] : g->xm + (size_t)c * Sm * xd;
          ps.push_back(fwd_prob(x, Sm, S.Gp + c * sG + G.off[l], G.fi[l], G.fo[l], y, G.act[l]));
        }
        mx.push_back(add_phase(g, ps));
      }
      std::vector<GemmProb> ps;
      for (int c = cb; c < ce; ++c)
        ps.push_back(base_prob(g->xm + (size_t)c * Sm * xd, xd, 0, g->P, F, 0,
                               g->fm + (size_t)c * Sm * F, F, Sm, F, xd));
      mx.push_back(add_phase(g, ps));
    };
    g->mix_phases[par].clear();
    if (g->cfg.mix_enable) {
      mix_phases(0, C, g->zeta, g->mix_phases[par]);
      for (int b = 0; b < g->n_bands; ++b)
        mix_phases(g->band_c0[b], g->band_c0[b + 1], g->zeta + (size_t)b * g->S * zd, g->band_mix_phases[par][b]);
    }
  }
  if (g->cfg.mix_enable) {
    std::vector<GemmProb> ps;
    ps.push_back(base_prob(g->data, g->xd, 0, g->P, g->F, 0, g->realfeat, g->F, (int)g->N, g->F, g->xd));
    g->real_phase = add_phase(g, ps);
  }
  if (g->cfg.trainer != LIPZ_TRAINER_GRADIENT) build_nes_ops(g);
}

// With timing on: a start / stop event pair for the next matrix-core launch.
hipError_t timing_events(lipz_grid* g, hipEvent_t* e0, hipEvent_t* e1) {
  *e0 = *e1 = nullptr;
  if (!g->timing) return hipSuccess;
  if (g->ev_pool.size() < 2) {
    hipEvent_t a, b;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return hipErrorOutOfMemory;
    g->ev_pool.push_back(a);
    g->ev_pool.push_back(b);
  }
  *e1 = g->ev_pool.back();
  g->ev_pool.pop_back();
  *e0 = g->ev_pool.back();
  g->ev_pool.pop_back();
  return hipSuccess;
}

void timing_record(lipz_grid* g, hipEvent_t e0, hipEvent_t e1, double flops, double bytes) {
  if (!g->timing) return;
  g->ev_live.push_back({e0, e1});
  g->ev_flops.push_back(flops);
  g->ev_bytes.push_back(bytes);
}

hipError_t run_gemm_phase(lipz_grid* g, int phase, int step_local, hipStream_t stream, const SampleJob* job) {
  const Phase& ph = g->phases[phase];
  hipEvent_t e0, e1;
  hipError_t e = timing_events(g, &e0, &e1);
  if (e != hipSuccess) return e;
  e = launch_gemm_grouped(g->probs_d + ph.first, ph.grp, ph.tiles, ph.tile_rows, ph.kernel, step_local, g->gemm_wt,
                          stream, e0, e1, job);
  timing_record(g, e0, e1, ph.flops, ph.bytes);
  return e;
}

lipz_status pre_call(lipz_grid* g) {
  if (!g) return LIPZ_E_INVAL;
  g->last_err.clear();
  if (g->sticky != LIPZ_OK) {
    g->last_err = "a previous HIP error is pending";
    return g->sticky;
  }
  return LIPZ_OK;
}

// A grid handle with its configuration, neighbour table, carved buffers
// (from `base`; nullptr only sizes them) and plan tables; no HIP calls.
lipz_grid* plan_grid(const lipz_config* cfg, int64_t n_samples, char* base, const float* data, size_t* total) {
  Net Gn, Dn;
  if (!validate(cfg, n_samples, &Gn, &Dn).empty()) return nullptr;
  lipz_grid* g = new (std::nothrow) lipz_grid();
  if (!g) return nullptr;
  g->cfg = *cfg;
  g->C = cfg->rows * cfg->cols;
  g->s = cfg->pop_size;
  g->U = g->C * g->s;
  g->nn = LIPZ_SLOTS * g->s;
  g->B = cfg->batch;
  g->zd = cfg->z_dim;
  g->xd = cfg->x_dim;
  g->S = cfg->mix_samples;
  g->F = cfg->mix_feat_dim;
  g->N = n_samples;
  g->G = Gn;
  g->D = Dn;
  if (cfg->net == LIPZ_NET_DCGAN) {
    g->dc = dc_new(cfg);
    if (!g->dc) {
      delete g;
      return nullptr;
    }
  } else {
    g->tn = ceil_div(Dn.fi[Dn.nl - 1], GEMM_BN);
    // the loss head folds into the launches around it when D has two or more
    // hidden layers (the discriminator step needs the layer below the last)
    g->fused_head = LIPZ_FUSED_HEAD && cfg->trainer == LIPZ_TRAINER_GRADIENT && Dn.nl >= 3;
    g->fused_sample = LIPZ_FUSED_SAMPLE && cfg->trainer == LIPZ_TRAINER_GRADIENT;
    if (g->fused_head) g->aS_ld = (Dn.fi[Dn.nl - 2] + 4 + 3) / 4 * 4;
    if (g->fused_head && Dn.fi[Dn.nl - 1] <= Dn.fi[Dn.nl - 2]) {
      g->hp_rows = (2 * g->B + 31) / 32;  // row tiles of the input-gradient launch (at most, 32-row tiles)
      g->hp_ld = (Dn.fi[Dn.nl - 1] + 1 + 3) / 4 * 4;
    }
  }
  g->data = data;
  g->key = make_uint2((uint32_t)(cfg->seed & 0xFFFFFFFFull), (uint32_t)(cfg->seed >> 32));
  g->slope = cfg->lrelu_slope;
  g->ac.beta1 = cfg->beta1;
  g->ac.beta2 = cfg->beta2;
  g->ac.one_minus_beta1 = (float)(1.0 - (double)cfg->beta1);
  g->ac.one_minus_beta2 = (float)(1.0 - (double)cfg->beta2);
  g->ac.eps = cfg->eps;

  // neighbour table: slots centre, north, south, west, east on the torus
  const int R = cfg->rows, Q = cfg->cols;
  g->nbr_h.resize((size_t)g->C * 5);
  for (int r = 0; r < R; ++r)
    for (int q = 0; q < Q; ++q) {
      int32_t* n = &g->nbr_h[(size_t)(r * Q + q) * 5];
      n[0] = r * Q + q;
      n[1] = ((r - 1 + R) % R) * Q + q;
      n[2] = ((r + 1) % R) * Q + q;
      n[3] = r * Q + (q - 1 + Q) % Q;
      n[4] = r * Q + (q + 1) % Q;
    }

  setup_groups(g);
  // The plan tables are carved last, so building them after the first carve
  // already sees the final buffer addresses; the second carve sizes them.
  carve(g, base, total);
  if (g->dc) dc_build(g);
  else build_tables(g);
  carve(g, base, total);
  if (!g->plan_ok || (g->dc && !dc_plan_ok(g->dc))) {
    dc_delete(g->dc);
    delete g;
    return nullptr;
  }
  return g;
}

// ---- enqueue helpers shared by the entry points and the row-band executor ----

// Evaluation of cells c0 .. c0 + nc - 1 of the current plan `phases`.
lipz_status enq_eval(lipz_grid* g, int gen, int c0, int nc, const std::vector<int>& phases, hipStream_t s,
                     float* d_L, float* d_Lg, float* d_fit_g, float* d_fit_d) {
  const int B = g->B, nn = g->nn, er = 1 + nn;
  const size_t n2 = (size_t)nn * nn;
  lipz_status st;
  hipError_t e = launch_sample(g->data, g->N, g->xd, g->zd, B, c0, nc, g->key, (uint32_t)gen, 0, g->Xe,
                               (int64_t)er * B * g->xd, g->ze, (int64_t)B * g->zd, s);
  if ((st = check_hip(g, e, "eval sample"))) return st;
  for (int ph : phases)
    if ((st = check_hip(g, run_gemm_phase(g, ph, 0, s), "eval forward"))) return st;
  EvalHeadArgs ha;
  memset(&ha, 0, sizeof(ha));
  ha.part = g->part_e + (size_t)c0 * nn * er * B * g->tn;
  ha.tn = g->tn;
  ha.L = g->L + c0 * n2;
  ha.Lg = g->Lg + c0 * n2;
  ha.rmean = g->rmean ? g->rmean + (size_t)c0 * nn : nullptr;
  ha.B = B;
  ha.C = nc;
  ha.nn = nn;
  ha.loss_kind = g->cfg.loss_kind;
  if ((st = check_hip(g, launch_head_eval(ha, s), "eval head"))) return st;
  e = launch_fitness(g->L + c0 * n2, g->Lg + c0 * n2, nc, nn, g->cfg.fitness_mode, g->fit_g + (size_t)c0 * nn,
                     g->fit_d + (size_t)c0 * nn, g->flags, d_L, d_Lg, d_fit_g, d_fit_d, s);
  return check_hip(g, e, "fitness");
}

// Tournaments and copies of cells c0 .. c0 + nc - 1 from buffer par into 1 - par.
lipz_status enq_select(lipz_grid* g, int gen, int par, int c0, int nc, const int32_t* d_forced, int32_t* d_sel,
                       float* d_lr, hipStream_t s) {
  const StateBuf& A = g->st[par];
  const StateBuf& Bn = g->st[1 - par];
  const int sp = g->s;
  lipz_status st;
  SelectArgs sa;
  memset(&sa, 0, sizeof(sa));
  sa.fit_g = g->fit_g;
  sa.fit_d = g->fit_d;
  sa.nbr = g->nbr;
  sa.forced = d_forced;
  sa.sel = g->sel;
  sa.flags = g->flags;
  sa.sel_out = d_sel;
  sa.lr_out = d_lr;
  sa.t_src[0] = A.Gt;
  sa.t_src[1] = A.Dt;
  sa.lr_src[0] = A.Glr;
  sa.lr_src[1] = A.Dlr;
  sa.t_dst[0] = Bn.Gt;
  sa.t_dst[1] = Bn.Dt;
  sa.lr_dst[0] = Bn.Glr;
  sa.lr_dst[1] = Bn.Dlr;
  sa.c0 = c0;
  sa.C = nc;
  sa.s = sp;
  sa.U = g->U;
  sa.tsize = g->cfg.tournament_size;
  sa.mutate = g->cfg.lr_mutation;
  sa.mut_std = g->cfg.lr_mut_std;
  sa.mut_prob = g->cfg.lr_mut_prob;
  sa.key = g->key;
  sa.gen = (uint32_t)gen;
  if ((st = check_hip(g, launch_select(sa, s), "tournament"))) return st;
  CopyArgs ca;
  memset(&ca, 0, sizeof(ca));
  const size_t u0 = (size_t)c0 * sp;
  ca.sel = g->sel + u0 * 2;
  ca.src[0][0] = A.Gp;
  ca.src[0][1] = A.Gm;
  ca.src[0][2] = A.Gv;
  ca.src[1][0] = A.Dp;
  ca.src[1][1] = A.Dm;
  ca.src[1][2] = A.Dv;
  ca.dst[0][0] = Bn.Gp + u0 * g->G.stride;
  ca.dst[0][1] = Bn.Gm + u0 * g->G.stride;
  ca.dst[0][2] = Bn.Gv + u0 * g->G.stride;
  ca.dst[1][0] = Bn.Dp + u0 * g->D.stride;
  ca.dst[1][1] = Bn.Dm + u0 * g->D.stride;
  ca.dst[1][2] = Bn.Dv + u0 * g->D.stride;
  ca.stride[0] = g->G.stride;
  ca.stride[1] = g->D.stride;
  ca.w_src = A.w + (size_t)c0 * LIPZ_SLOTS;
  ca.w_dst = Bn.w + (size_t)c0 * LIPZ_SLOTS;
  ca.U = nc * sp;
  ca.C = nc;
  return check_hip(g, launch_copy_winners(ca, s), "replace");
}

// Post-training re-evaluation and elitist truncation of cells c0 .. c0 + nc - 1:
// trained individuals in buffer par, the previous state in 1 - par.
lipz_status enq_elite(lipz_grid* g, int par, int c0, int nc, const std::vector<int>& phases, hipStream_t s,
                      int32_t* d_src, float* d_fit2_g, float* d_fit2_d) {
  lipz_status st;
  for (int ph : phases)
    if ((st = check_hip(g, run_gemm_phase(g, ph, 0, s), "re-evaluation"))) return st;
  const StateBuf& O = g->st[1 - par];
  const StateBuf& N = g->st[par];
  const int sp = g->s;
  EliteArgs ea;
  memset(&ea, 0, sizeof(ea));
  ea.part2 = g->part_e2;
  ea.part3 = g->part_e3;
  ea.rmean = g->rmean;
  ea.L2 = g->el_L2;
  ea.Lg2 = g->el_Lg2;
  ea.M3 = g->el_M3;
  ea.fit_g = g->fit_g;
  ea.fit_d = g->fit_d;
  ea.fit2_g = g->fit2_g;
  ea.fit2_d = g->fit2_d;
  ea.src = g->esrc;
  ea.src_out = d_src;
  ea.fit2_g_out = d_fit2_g;
  ea.fit2_d_out = d_fit2_d;
  ea.flags = g->flags;
  ea.t_old[0] = O.Gt;
  ea.t_old[1] = O.Dt;
  ea.lr_old[0] = O.Glr;
  ea.lr_old[1] = O.Dlr;
  ea.t_new[0] = N.Gt;
  ea.t_new[1] = N.Dt;
  ea.lr_new[0] = N.Glr;
  ea.lr_new[1] = N.Dlr;
  ea.tn = g->tn;
  ea.B = g->B;
  ea.c0 = c0;
  ea.C = nc;
  ea.s = sp;
  ea.nn = g->nn;
  ea.mode = g->cfg.fitness_mode;
  ea.loss_kind = g->cfg.loss_kind;
  if ((st = check_hip(g, launch_elite(ea, s), "elitist truncation"))) return st;
  CopyArgs ca;
  memset(&ca, 0, sizeof(ca));
  const size_t u0 = (size_t)c0 * sp;
  ca.sel = g->esrc + u0 * 2;
  ca.src[0][0] = O.Gp;
  ca.src[0][1] = O.Gm;
  ca.src[0][2] = O.Gv;
  ca.src[1][0] = O.Dp;
  ca.src[1][1] = O.Dm;
  ca.src[1][2] = O.Dv;
  ca.dst[0][0] = N.Gp + u0 * g->G.stride;
  ca.dst[0][1] = N.Gm + u0 * g->G.stride;
  ca.dst[0][2] = N.Gv + u0 * g->G.stride;
  ca.dst[1][0] = N.Dp + u0 * g->D.stride;
  ca.dst[1][1] = N.Dm + u0 * g->D.stride;
  ca.dst[1][2] = N.Dv + u0 * g->D.stride;
  ca.stride[0] = g->G.stride;
  ca.stride[1] = g->D.stride;
  ca.U = nc * sp;
  ca.C = nc;
  return check_hip(g, launch_copy_winners(ca, s), "elitist copy");
}

// The training heads of buffer par (all units; a group narrows c0, C).
void train_heads(lipz_grid* g, int par, HeadArgs* hd, HeadArgs* hg) {
  const StateBuf& S = g->st[par];
  const int B = g->B, LD = g->D.nl;
  memset(hd, 0, sizeof(*hd));
  hd->part = g->part_tr;
  hd->tn = g->tn;
  hd->act = g->a[LD - 2];
  hd->act_cell_stride = (int64_t)2 * B * g->D.fi[LD - 1];
  hd->delta = g->dD[LD - 2];
  hd->w = S.Dp + g->D.off[LD - 1];
  hd->p_stride = g->D.stride;
  hd->dlbuf = g->dlbuf;
  hd->H = g->D.fi[LD - 1];
  hd->B = B;
  hd->c0 = 0;
  hd->C = g->U;
  hd->hidden_act = g->D.act[LD - 2];
  hd->slope = g->slope;
  hd->loss_kind = g->cfg.loss_kind;
  *hg = *hd;
  hg->part = g->part_g;
  hg->act = g->ag[LD - 2];
  hg->act_cell_stride = (int64_t)B * g->D.fi[LD - 1];
  hg->delta = g->dDg[LD - 2];
  hg->dlbuf = nullptr;
}

// Gradient-trainer step k (training step `step`) of group grp of buffer par.
// One training step of cell group grp.  first: the step's minibatch is not
// drawn yet (the first step of a sequence); last: no further step follows,
// so the next minibatch is not drawn.
lipz_status enq_train_group_step(lipz_grid* g, int gen, int par, int grp, int k, int step, bool first, bool last,
                                 float* d_losses, const HeadArgs& hd, const HeadArgs& hg, hipStream_t gs) {
  const int B = g->B;
  const int c0 = g->group_c0[grp], nc = g->group_c0[grp + 1] - c0;
  HeadArgs gd = hd, gg = hg;
  gd.c0 = gg.c0 = c0;
  gd.C = gg.C = nc;
  gd.losses = gg.losses = d_losses ? d_losses + (size_t)k * g->U * 2 : nullptr;
  const bool odd = g->fused_sample && (step & 1);
  // the draw of step + 1 for the other buffer pair
  SampleJob job;
  memset(&job, 0, sizeof(job));
  if (g->fused_sample && !last) {
    job.data = g->data;
    job.N = g->N;
    job.X = odd ? g->Xtr : g->Xtr_alt;
    job.Z = odd ? g->z : g->z_alt;
    job.x_stride = (int64_t)2 * B * g->xd;
    job.z_stride = (int64_t)B * g->zd;
    job.key = g->key;
    job.gen = (uint32_t)gen;
    job.sf = (uint32_t)(step + 2);
    job.xd = g->xd;
    job.zd = g->zd;
    job.B = B;
    job.u0 = c0;
    job.blocks = nc * ((B + SAMPLE_ROWS - 1) / SAMPLE_ROWS);
  }
  lipz_status st;
  for (const Op& op : odd ? g->train_ops_odd[par][grp] : g->train_ops[par][grp]) {
    hipError_t e = hipSuccess;
    switch (op.kind) {
      case OP_SAMPLE:
        if (!g->fused_sample || first)
          e = launch_sample(g->data, g->N, g->xd, g->zd, B, c0, nc, g->key, (uint32_t)gen, (uint32_t)(step + 1),
                            odd ? g->Xtr_alt : g->Xtr, (int64_t)2 * B * g->xd, odd ? g->z_alt : g->z,
                            (int64_t)B * g->zd, gs);
        break;
      case OP_GEMM: e = run_gemm_phase(g, op.phase, k, gs, op.sample_next && job.blocks ? &job : nullptr); break;
      case OP_HEAD_D: e = launch_head_d(gd, gs); break;
      case OP_HEAD_G: e = launch_head_g(gg, gs); break;
      case OP_LOSS_D: if (d_losses) e = launch_loss_d(gd, gs); break;
      case OP_LOSS_G: if (d_losses) e = launch_loss_g(gg, gs); break;
      default: e = hipErrorInvalidValue; break;
    }
    if ((st = check_hip(g, e, "train step"))) return st;
  }
  return LIPZ_OK;
}

// The gradient-free trainers' per-role arguments for state buffer par.
void nes_args(lipz_grid* g, int gen, int par, NesArgs* na) {
  const StateBuf& S = g->st[par];
  for (int role = 0; role < 2; ++role) {
    NesArgs& a = na[role];
    memset(&a, 0, sizeof(a));
    const bool d = role == LIPZ_ROLE_D;
    a.p = d ? S.Dp : S.Gp;
    a.m = d ? S.Dm : S.Gm;
    a.v = d ? S.Dv : S.Gv;
    a.lr = d ? S.Dlr : S.Glr;
    a.t = d ? S.Dt : S.Gt;
    a.sets = d ? g->nes_pd : g->nes_pg;
    a.eps = g->nes_eps;
    a.eps_stride = g->nes_eps_stride;
    a.part = d ? g->nes_part_d : g->nes_part_g;
    a.fit = d ? g->nes_fd : g->nes_fg;
    a.stride = d ? g->D.stride : g->G.stride;
    a.P = d ? g->D.P : g->G.P;
    a.n = g->cfg.nes_pairs;
    a.tn = g->tn;
    a.B = g->B;
    a.c0 = 0;
    a.C = g->U;
    a.role = role;
    a.loss_kind = g->cfg.loss_kind;
    a.sigma = g->cfg.nes_sigma;
    a.clip = (d && g->cfg.loss_kind == LIPZ_LOSS_WASSERSTEIN) ? g->cfg.wgan_clip : 0.f;
    a.key = g->key;
    a.gen = (uint32_t)gen;
    a.tag = d ? LIPZ_TAG_NES_D : LIPZ_TAG_NES_G;
    a.ac = g->ac;
  }
}

// Gradient-free step k (training step `step`) of training units u0 .. u0 + nu - 1
// with their plan `ops`.
lipz_status enq_nes_step(lipz_grid* g, int gen, const std::vector<Op>& ops, const NesArgs* na, int u0, int nu,
                         int k, int step, float* d_losses, hipStream_t s) {
  const bool es = g->cfg.trainer == LIPZ_TRAINER_ES;
  const int B = g->B;
  lipz_status st;
  for (const Op& op : ops) {
    hipError_t e = hipSuccess;
    NesArgs a = op.kind >= OP_NES_PERTURB ? na[op.phase] : na[0];
    a.c0 = u0;
    a.C = nu;
    a.sf = (uint32_t)(step + 1);
    a.step_local = k;
    a.losses = d_losses ? d_losses + (size_t)k * g->U * 2 : nullptr;
    switch (op.kind) {
      case OP_SAMPLE:
        e = launch_sample(g->data, g->N, g->xd, g->zd, B, u0, nu, g->key, (uint32_t)gen, (uint32_t)(step + 1),
                          g->Xtr, (int64_t)2 * B * g->xd, g->z, (int64_t)B * g->zd, s);
        break;
      case OP_GEMM: e = run_gemm_phase(g, op.phase, k, s); break;
      case OP_NES_PERTURB: e = launch_nes_perturb(a, s); break;
      case OP_NES_HEAD: e = launch_nes_head(a, s); break;
      case OP_NES_UPDATE: e = es ? launch_es_select(a, s) : launch_nes_update(a, s); break;
      default: e = hipErrorInvalidValue; break;
    }
    if ((st = check_hip(g, e, es ? "ES step" : "NES step"))) return st;
  }
  return LIPZ_OK;
}

}  // namespace lipz

namespace lipz {

lipz_status create_grid(const lipz_config* cfg, void* d_workspace, size_t workspace_bytes,
                        const float* d_dataset, int64_t n_samples, void* hip_stream, lipz_grid** out) {
  if (!out) return LIPZ_E_INVAL;
  *out = nullptr;
  Net Gn, Dn;
  if (!validate(cfg, n_samples, &Gn, &Dn).empty()) return LIPZ_E_INVAL;
  if (!d_workspace || !d_dataset) return LIPZ_E_INVAL;
  if (((uintptr_t)d_workspace & (kAlign - 1)) != 0) return LIPZ_E_WORKSPACE;
  const size_t need = lipz_workspace_bytes(cfg, n_samples);
  if (need == 0 || workspace_bytes < need) return LIPZ_E_WORKSPACE;
  size_t total = 0;
  lipz_grid* g = plan_grid(cfg, n_samples, (char*)d_workspace, d_dataset, &total);
  if (!g) return LIPZ_E_INVAL;
  if (total > workspace_bytes) {
    dc_delete(g->dc);
    delete g;
    return LIPZ_E_WORKSPACE;
  }
  g->stream = (hipStream_t)hip_stream;

  hipStream_t s = g->stream;
  lipz_status st = LIPZ_OK;
  auto ck = [&](hipError_t e, const char* what) {
    if (st == LIPZ_OK) st = check_hip(g, e, what);
  };
  g->gstream[0] = s;
  if (g->n_groups > 1 || g->n_bands > 0) ck(hipEventCreateWithFlags(&g->fork_ev, hipEventDisableTiming), "create event");
  for (int i = 1; i < g->n_groups; ++i) {
    ck(hipStreamCreateWithFlags(&g->gstream[i], hipStreamNonBlocking), "create stream");
    ck(hipEventCreateWithFlags(&g->join_ev[i], hipEventDisableTiming), "create event");
  }
  for (int b = 0; b < g->n_bands; ++b) {
    ck(hipEventCreateWithFlags(&g->band_ev[b], hipEventDisableTiming), "create event");
    ck(hipEventCreateWithFlags(&g->mom_ev[b], hipEventDisableTiming), "create event");
  }
  ck(hipMemcpyAsync(g->nbr, g->nbr_h.data(), g->nbr_h.size() * sizeof(int32_t), hipMemcpyHostToDevice, s),
     "upload neighbours");
  ck(hipMemcpyAsync(g->probs_d, g->probs_h.data(), g->probs_h.size() * sizeof(GemmProb),
                    hipMemcpyHostToDevice, s),
     "upload GEMM tables");
  if (g->dc) ck(dc_upload_tables(g, s), "upload convolution tables");
  const StateBuf& S0 = g->st[0];
  const int C = g->C, U = g->U;
  // both state buffers, padding included, start at zero so saved blobs are deterministic
  for (int b = 0; b < 2; ++b)
    ck(launch_fill_i32(reinterpret_cast<int32_t*>(g->st[b].base), (int64_t)(g->state_bytes / 4), 0, s),
       "zero state");
  if (g->dc) {
    ck(dc_init_params(g, S0, s), "init");
  } else {
    // individual u from stream (cell field) u
    ck(launch_init_params(S0.Gp, g->G.stride, g->G.P, U, g->G.layers(), g->key, LIPZ_TAG_INIT_G, s), "init G");
    ck(launch_init_params(S0.Dp, g->D.stride, g->D.P, U, g->D.layers(), g->key, LIPZ_TAG_INIT_D, s), "init D");
  }
  ck(launch_fill_f32(S0.Gm, (int64_t)U * g->G.stride, 0.f, s), "zero");
  ck(launch_fill_f32(S0.Gv, (int64_t)U * g->G.stride, 0.f, s), "zero");
  ck(launch_fill_f32(S0.Dm, (int64_t)U * g->D.stride, 0.f, s), "zero");
  ck(launch_fill_f32(S0.Dv, (int64_t)U * g->D.stride, 0.f, s), "zero");
  ck(launch_fill_i32(S0.Gt, U, 0, s), "zero");
  ck(launch_fill_i32(S0.Dt, U, 0, s), "zero");
  ck(launch_fill_f32(S0.Glr, U, cfg->lr0_g, s), "fill");
  ck(launch_fill_f32(S0.Dlr, U, cfg->lr0_d, s), "fill");
  ck(launch_fill_f32(S0.w, (int64_t)C * 5, 1.f / 5.f, s), "fill");
  ck(launch_fill_i32(g->flags, 4, 0, s), "zero");
  if (cfg->mix_enable) {
    ck(launch_normals(g->P, (int64_t)g->xd * g->F, 1.0 / sqrt((double)g->xd), g->key, 0, 0, 0,
                      LIPZ_TAG_PROJ, s),
       "projection");
    ck(run_gemm_phase(g, g->real_phase, 0, s), "project dataset");
    ck(launch_col_stats(g->realfeat, g->N, g->F, g->mu_r, g->sd_r, s), "dataset feature stats");
  }
  ck(hipStreamSynchronize(s), "create sync");
  if (st != LIPZ_OK) {
    lipz_grid_destroy(g);
    return st;
  }
  *out = g;
  return LIPZ_OK;
}

}  // namespace lipz

extern "C" {

size_t lipz_workspace_bytes(const lipz_config* cfg, int64_t n_samples) {
  size_t total = 0;
  lipz_grid* g = plan_grid(cfg, n_samples, nullptr, nullptr, &total);
  if (!g) return 0;
  dc_delete(g->dc);
  delete g;
  return total;
}

lipz_status lipz_grid_create(const lipz_config* cfg, void* d_workspace, size_t workspace_bytes,
                             const float* d_dataset, int64_t n_samples, void* hip_stream,
                             lipz_grid** out) {
  return create_grid(cfg, d_workspace, workspace_bytes, d_dataset, n_samples, hip_stream, out);
}

lipz_status lipz_grid_create_static(const lipz_config* cfg, const float* d_dataset, int64_t n_samples,
                                    void* hip_stream, lipz_grid** out) {
  if (!out) return LIPZ_E_INVAL;
  *out = nullptr;
  Net Gn, Dn;
  if (!validate(cfg, n_samples, &Gn, &Dn).empty() || !d_dataset) return LIPZ_E_INVAL;
  // row bands create streams and events of their own
  if (cfg->bands >= 2) return LIPZ_E_UNSUPPORTED;
  const size_t need = lipz_workspace_bytes(cfg, n_samples);
  if (need == 0) return LIPZ_E_INVAL;
  if (need > kStaticWorkspaceBytes) return LIPZ_E_WORKSPACE;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return LIPZ_E_HIP;
  if (dev >= kMaxStaticDevices) return LIPZ_E_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (g_static_busy[dev]) return LIPZ_E_ORDER;
  if (!g_static_ptr[dev]) {
    // the device's own copy of the array (the name itself is a host-side stand-in)
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return LIPZ_E_HIP;
    g_static_ptr[dev] = p;
  }
  lipz_status st = create_grid(cfg, g_static_ptr[dev], kStaticWorkspaceBytes, d_dataset, n_samples, hip_stream, out);
  if (st == LIPZ_OK) {
    g_static_busy[dev] = true;
    (*out)->static_dev = dev;
  }
  return st;
}


lipz_status lipz_grid_destroy(lipz_grid* g) {
  if (!g) return LIPZ_E_INVAL;
  if (g->static_dev >= 0) {
    // the static array goes back to the device once the grid's work is done
    hipStreamSynchronize(g->stream);
    std::lock_guard<std::mutex> lock(g_static_mu);
    g_static_busy[g->static_dev] = false;
  }
  for (int i = 1; i < g->n_groups; ++i) {
    if (g->gstream[i]) {
      hipStreamSynchronize(g->gstream[i]);
      hipStreamDestroy(g->gstream[i]);
    }
    if (g->join_ev[i]) hipEventDestroy(g->join_ev[i]);
  }
  if (g->fork_ev) hipEventDestroy(g->fork_ev);
  for (int b = 0; b < g->n_bands; ++b) {
    if (g->band_ev[b]) hipEventDestroy(g->band_ev[b]);
    if (g->mom_ev[b]) hipEventDestroy(g->mom_ev[b]);
  }
  for (auto& e : g->ev_pool) hipEventDestroy(e);
  for (auto& p : g->ev_live) {
    hipEventDestroy(p.first);
    hipEventDestroy(p.second);
  }
  dc_delete(g->dc);
  delete g;
  return LIPZ_OK;
}

lipz_status lipz_eval_neighborhoods(lipz_grid* g, int32_t gen, float* d_L, float* d_Lg,
                                    float* d_fit_g, float* d_fit_d) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (gen < 0 || gen > 65535) return fail(g, LIPZ_E_INVAL, "gen must be in [0, 65535]");
  hipStream_t s = g->stream;
  if (g->dc) {
    if ((st = dc_eval(g, gen))) return st;
    hipError_t e = launch_fitness(g->L, g->Lg, g->C, g->nn, g->cfg.fitness_mode, g->fit_g, g->fit_d, g->flags,
                                  d_L, d_Lg, d_fit_g, d_fit_d, s);
    if ((st = check_hip(g, e, "fitness"))) return st;
  } else if ((st = enq_eval(g, gen, 0, g->C, g->eval_phases[g->cur], s, d_L, d_Lg, d_fit_g, d_fit_d))) {
    return st;
  }
  g->fitness_valid = true;
  g->elite_state = 1;
  g->elite_gen = gen;
  return LIPZ_OK;
}

lipz_status lipz_select_replace(lipz_grid* g, int32_t gen, const int32_t* d_forced, int32_t* d_sel,
                                float* d_lr) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (gen < 0 || gen > 65535) return fail(g, LIPZ_E_INVAL, "gen must be in [0, 65535]");
  if (!d_forced && !g->fitness_valid)
    return fail(g, LIPZ_E_ORDER, "select_replace needs an evaluation of the current state");
  if ((st = enq_select(g, gen, g->cur, 0, g->C, d_forced, d_sel, d_lr, g->stream))) return st;
  g->cur = 1 - g->cur;
  g->fitness_valid = false;
  g->elite_state = g->elite_state == 1 ? 2 : 0;
  return LIPZ_OK;
}

lipz_status lipz_elitist_replace(lipz_grid* g, int32_t gen, int32_t* d_src, float* d_fit2_g, float* d_fit2_d) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (!g->cfg.elitism) return fail(g, LIPZ_E_ORDER, "grid created with elitism = 0");
  if (g->elite_state != 2 || gen != g->elite_gen)
    return fail(g, LIPZ_E_ORDER, "elitist_replace needs eval_neighborhoods(gen), select_replace, training");
  // the current buffer holds the trained individuals; the other one the state selection read
  if ((st = enq_elite(g, g->cur, 0, g->C, g->elite_phases[g->cur], g->stream, d_src, d_fit2_g, d_fit2_d)))
    return st;
  g->elite_state = 0;
  g->fitness_valid = false;
  return LIPZ_OK;
}

lipz_status lipz_train_step(lipz_grid* g, int32_t gen, int32_t step0, int32_t n_steps,
                            float* d_losses) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (gen < 0 || gen > 65535) return fail(g, LIPZ_E_INVAL, "gen must be in [0, 65535]");
  if (step0 < 0 || n_steps < 0 || (int64_t)step0 + n_steps > 65535)
    return fail(g, LIPZ_E_INVAL, "steps must satisfy 0 <= step0, step0 + n_steps <= 65535");
  if (n_steps == 0) return LIPZ_OK;
  hipStream_t s = g->stream;
  if (g->dc) {
    if ((st = dc_train(g, gen, step0, n_steps, d_losses))) return st;
    const StateBuf& S = g->st[g->cur];
    hipError_t e = launch_add_i32(S.Gt, g->C, n_steps, s);
    if (e == hipSuccess) e = launch_add_i32(S.Dt, g->C, n_steps, s);
    if ((st = check_hip(g, e, "step count"))) return st;
    g->fitness_valid = false;
    return LIPZ_OK;
  }
  const int par = g->cur;
  const StateBuf& S = g->st[par];
  const int C = g->U, B = g->B;  // C: training units
  HeadArgs hd, hg;
  train_heads(g, par, &hd, &hg);
  if (g->cfg.trainer != LIPZ_TRAINER_GRADIENT) {
    NesArgs na[2];
    nes_args(g, gen, par, na);
    for (int k = 0; k < n_steps; ++k)
      if ((st = enq_nes_step(g, gen, g->nes_ops[par], na, 0, C, k, step0 + k, d_losses, s))) return st;
    hipError_t e = launch_add_i32(S.Gt, C, n_steps, s);
    if (e == hipSuccess) e = launch_add_i32(S.Dt, C, n_steps, s);
    if ((st = check_hip(g, e, "step count"))) return st;
    g->fitness_valid = false;
    return LIPZ_OK;
  }
  // fork: every group stream waits for the work already on the caller's stream
  if (g->n_groups > 1) {
    if ((st = check_hip(g, hipEventRecord(g->fork_ev, s), "fork"))) return st;
    for (int i = 1; i < g->n_groups; ++i)
      if ((st = check_hip(g, hipStreamWaitEvent(g->gstream[i], g->fork_ev, 0), "fork"))) return st;
  }
  // enqueue step by step across the groups so every stream has work early
  for (int k = 0; k < n_steps; ++k)
    for (int grp = 0; grp < g->n_groups; ++grp)
      if ((st = enq_train_group_step(g, gen, par, grp, k, step0 + k, k == 0, k + 1 == n_steps, d_losses, hd, hg,
                                     g->gstream[grp])))
        return st;
  // join: the caller's stream waits for every group
  for (int i = 1; i < g->n_groups; ++i) {
    if ((st = check_hip(g, hipEventRecord(g->join_ev[i], g->gstream[i]), "join"))) return st;
    if ((st = check_hip(g, hipStreamWaitEvent(s, g->join_ev[i], 0), "join"))) return st;
  }
  hipError_t e = launch_add_i32(S.Gt, C, n_steps, s);
  if (e == hipSuccess) e = launch_add_i32(S.Dt, C, n_steps, s);
  if ((st = check_hip(g, e, "step count"))) return st;
  g->fitness_valid = false;
  return LIPZ_OK;
}

// The generations of lipz_run_generations on the row bands' streams (the
// caller forks before and joins after, also when this stops on an error).
static lipz_status enq_band_generations(lipz_grid* g, int gen0, int n_gens, int n_steps) {
  const int nb = g->n_bands, sp = g->s;
  lipz_status st;
  for (int i = 0; i < n_gens; ++i) {
    const int gen = gen0 + i, par = g->cur;
    HeadArgs hd, hg;
    train_heads(g, 1 - par, &hd, &hg);
    // each band: wait for its neighbour bands' previous generation, then
    // evaluate and select its cells
    for (int b = 0; b < nb; ++b) {
      hipStream_t bs = g->gstream[b];
      if (i > 0)
        for (int b2 = 0; b2 < nb; ++b2)
          if (b2 != b && (g->band_wait[b] >> b2 & 1u))
            if ((st = check_hip(g, hipStreamWaitEvent(bs, g->band_ev[b2], 0), "band wait"))) return st;
      const int c0 = g->band_c0[b], nc = g->band_c0[b + 1] - c0;
      if ((st = enq_eval(g, gen, c0, nc, g->band_eval_phases[par][b], bs, nullptr, nullptr, nullptr, nullptr)))
        return st;
      if ((st = enq_select(g, gen, par, c0, nc, nullptr, nullptr, nullptr, bs))) return st;
    }
    // training, step by step across the bands so every stream has work early
    NesArgs na[2];
    if (g->cfg.trainer != LIPZ_TRAINER_GRADIENT) nes_args(g, gen, 1 - par, na);
    for (int k = 0; k < n_steps; ++k)
      for (int b = 0; b < nb; ++b) {
        if (g->cfg.trainer != LIPZ_TRAINER_GRADIENT) {
          const int u0 = g->band_c0[b] * sp, nu = g->band_c0[b + 1] * sp - u0;
          if ((st = enq_nes_step(g, gen, g->nes_band_ops[1 - par][b], na, u0, nu, k, k, nullptr, g->gstream[b])))
            return st;
        } else if ((st = enq_train_group_step(g, gen, 1 - par, b, k, k, k == 0, k + 1 == n_steps, nullptr, hd, hg,
                                              g->gstream[b]))) {
          return st;
        }
      }
    for (int b = 0; b < nb; ++b) {
      hipStream_t bs = g->gstream[b];
      const int c0 = g->band_c0[b], nc = g->band_c0[b + 1] - c0;
      const StateBuf& N = g->st[1 - par];
      if (n_steps > 0) {
        hipError_t e = launch_add_i32(N.Gt + (size_t)c0 * sp, nc * sp, n_steps, bs);
        if (e == hipSuccess) e = launch_add_i32(N.Dt + (size_t)c0 * sp, nc * sp, n_steps, bs);
        if ((st = check_hip(g, e, "step count"))) return st;
      }
      if (g->cfg.elitism &&
          (st = enq_elite(g, 1 - par, c0, nc, g->band_elite_phases[1 - par][b], bs, nullptr, nullptr, nullptr)))
        return st;
      if (g->cfg.mix_enable) {  // the band's generators' feature moments
        float* zeta = g->zeta + (size_t)b * g->S * g->zd;
        hipError_t e = launch_normals(zeta, (int64_t)g->S * g->zd, 1.0, g->key, 0, (uint32_t)gen, 0, LIPZ_TAG_MIXZ, bs);
        if ((st = check_hip(g, e, "mixture latents"))) return st;
        for (int ph : g->band_mix_phases[1 - par][b])
          if ((st = check_hip(g, run_gemm_phase(g, ph, 0, bs), "mixture forward"))) return st;
        const int nch = (g->S + 63) / 64;
        e = launch_moments(g->fm + (size_t)c0 * g->S * g->F, nc, g->S, g->F,
                           g->mom_part + (size_t)c0 * nch * 2 * g->F, g->mu_k + (size_t)c0 * g->F,
                           g->s2_k + (size_t)c0 * g->F, bs);
        if ((st = check_hip(g, e, "mixture moments"))) return st;
        if ((st = check_hip(g, hipEventRecord(g->mom_ev[b], bs), "moments ready"))) return st;
      } else if ((st = check_hip(g, hipEventRecord(g->band_ev[b], bs), "band ready"))) {
        return st;
      }
    }
    if (g->cfg.mix_enable) {
      // the ES step of a cell scores the moments of its neighbours' generators
      for (int b = 0; b < nb; ++b) {
        hipStream_t bs = g->gstream[b];
        for (int b2 = 0; b2 < nb; ++b2)
          if (b2 != b && (g->band_wait[b] >> b2 & 1u))
            if ((st = check_hip(g, hipStreamWaitEvent(bs, g->mom_ev[b2], 0), "moments wait"))) return st;
        EsArgs ea;
        memset(&ea, 0, sizeof(ea));
        ea.mu = g->mu_k;
        ea.s2 = g->s2_k;
        ea.mu_r = g->mu_r;
        ea.sd_r = g->sd_r;
        ea.nbr = g->nbr;
        ea.w = g->st[1 - par].w;
        ea.c0 = g->band_c0[b];
        ea.C = g->band_c0[b + 1] - g->band_c0[b];
        ea.F = g->F;
        ea.sigma = g->cfg.mix_sigma;
        ea.key = g->key;
        ea.gen = (uint32_t)gen;
        if ((st = check_hip(g, launch_es(ea, bs), "mixture ES"))) return st;
        if ((st = check_hip(g, hipEventRecord(g->band_ev[b], bs), "band ready"))) return st;
      }
    }
    g->cur = 1 - par;
  }
  return LIPZ_OK;
}

lipz_status lipz_run_generations(lipz_grid* g, int32_t gen0, int32_t n_gens, int32_t n_steps) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (gen0 < 0 || n_gens < 0 || (int64_t)gen0 + n_gens > 65536)
    return fail(g, LIPZ_E_INVAL, "generations must lie in [0, 65535]");
  if (n_steps < 0 || n_steps > 65535) return fail(g, LIPZ_E_INVAL, "n_steps must be in [0, 65535]");
  if (g->n_bands < 2) {  // one batch: the entry points in order
    for (int i = 0; i < n_gens; ++i) {
      const int gen = gen0 + i;
      if ((st = lipz_eval_neighborhoods(g, gen, nullptr, nullptr, nullptr, nullptr))) return st;
      if ((st = lipz_select_replace(g, gen, nullptr, nullptr, nullptr))) return st;
      if ((st = lipz_train_step(g, gen, 0, n_steps, nullptr))) return st;
      if (g->cfg.elitism && (st = lipz_elitist_replace(g, gen, nullptr, nullptr, nullptr))) return st;
      if (g->cfg.mix_enable && (st = lipz_mixture_update(g, gen, nullptr, nullptr, nullptr))) return st;
    }
    return LIPZ_OK;
  }
  const int nb = g->n_bands;
  hipStream_t s = g->stream;
  // fork: every band waits for the work already on the caller's stream
  if ((st = check_hip(g, hipEventRecord(g->fork_ev, s), "fork"))) return st;
  for (int b = 1; b < nb; ++b)
    if ((st = check_hip(g, hipStreamWaitEvent(g->gstream[b], g->fork_ev, 0), "fork"))) return st;
  st = enq_band_generations(g, gen0, n_gens, n_steps);
  // join: the caller's stream waits for everything enqueued on the bands
  for (int b = 1; b < nb; ++b) {
    lipz_status sj = check_hip(g, hipEventRecord(g->join_ev[b], g->gstream[b]), "join");
    if (!sj) sj = check_hip(g, hipStreamWaitEvent(s, g->join_ev[b], 0), "join");
    if (!st) st = sj;
  }
  g->fitness_valid = false;
  g->elite_state = 0;
  return st;
}

lipz_status lipz_mixture_update(lipz_grid* g, int32_t gen, float* d_w, float* d_score,
                                int32_t* d_accepted) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (!g->cfg.mix_enable) return fail(g, LIPZ_E_ORDER, "grid created with mix_enable = 0");
  if (gen < 0 || gen > 65535) return fail(g, LIPZ_E_INVAL, "gen must be in [0, 65535]");
  hipStream_t s = g->stream;
  const int par = g->cur;
  hipError_t e = launch_normals(g->zeta, (int64_t)g->S * g->zd, 1.0, g->key, 0, (uint32_t)gen, 0,
                                LIPZ_TAG_MIXZ, s);
  if ((st = check_hip(g, e, "mixture latents"))) return st;
  for (int ph : g->mix_phases[par])
    if ((st = check_hip(g, run_gemm_phase(g, ph, 0, s), "mixture forward"))) return st;
  e = launch_moments(g->fm, g->C, g->S, g->F, g->mom_part, g->mu_k, g->s2_k, s);
  if ((st = check_hip(g, e, "mixture moments"))) return st;
  EsArgs ea;
  ea.mu = g->mu_k;
  ea.s2 = g->s2_k;
  ea.mu_r = g->mu_r;
  ea.sd_r = g->sd_r;
  ea.nbr = g->nbr;
  ea.w = g->st[par].w;
  ea.w_out = d_w;
  ea.score_out = d_score;
  ea.acc_out = d_accepted;
  ea.c0 = 0;
  ea.C = g->C;
  ea.F = g->F;
  ea.sigma = g->cfg.mix_sigma;
  ea.key = g->key;
  ea.gen = (uint32_t)gen;
  return check_hip(g, launch_es(ea, s), "mixture ES");
}

lipz_status lipz_get_neighbors(const lipz_grid* g, int32_t* h_nbr) {
  if (!g || !h_nbr) return LIPZ_E_INVAL;
  memcpy(h_nbr, g->nbr_h.data(), g->nbr_h.size() * sizeof(int32_t));
  return LIPZ_OK;
}

lipz_status lipz_param_layout(const lipz_grid* g, int32_t role, int64_t* h_offsets, int32_t* h_n) {
  if (!g || !h_n || (role != LIPZ_ROLE_G && role != LIPZ_ROLE_D)) return LIPZ_E_INVAL;
  if (g->dc) return dc_param_layout(g, role, h_offsets, h_n);
  const Net& n = role == LIPZ_ROLE_G ? g->G : g->D;
  *h_n = n.nl;
  if (h_offsets)
    for (int l = 0; l < n.nl; ++l) {
      h_offsets[3 * l + 0] = n.off[l];
      h_offsets[3 * l + 1] = n.fi[l];
      h_offsets[3 * l + 2] = n.fo[l];
    }
  return LIPZ_OK;
}

lipz_status lipz_state_layout(const lipz_grid* g, int64_t* h_offsets, int64_t* h_strides) {
  if (!g) return LIPZ_E_INVAL;
  if (h_offsets) memcpy(h_offsets, g->state_off, sizeof(g->state_off));
  if (h_strides) {
    h_strides[0] = g->G.stride;
    h_strides[1] = g->D.stride;
  }
  return LIPZ_OK;
}

size_t lipz_state_bytes(const lipz_grid* g) { return g ? g->state_bytes : 0; }

lipz_status lipz_save_state(lipz_grid* g, void* d_dst) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (!d_dst) return fail(g, LIPZ_E_INVAL, "null destination");
  return check_hip(g, hipMemcpyAsync(d_dst, g->st[g->cur].base, g->state_bytes, hipMemcpyDeviceToDevice,
                                     g->stream),
                   "save state");
}

lipz_status lipz_load_state(lipz_grid* g, const void* d_src) {
  lipz_status st = pre_call(g);
  if (st) return st;
  if (!d_src) return fail(g, LIPZ_E_INVAL, "null source");
  g->fitness_valid = false;
  g->elite_state = 0;
  return check_hip(g, hipMemcpyAsync(g->st[g->cur].base, d_src, g->state_bytes, hipMemcpyDeviceToDevice,
                                     g->stream),
                   "load state");
}

lipz_status lipz_sync(lipz_grid* g) {
  if (!g) return LIPZ_E_INVAL;
  if (g->sticky != LIPZ_OK) return g->sticky;
  hipError_t e = hipStreamSynchronize(g->stream);
  if (e != hipSuccess) return check_hip(g, e, "stream sync");
  int32_t flags = 0;
  e = hipMemcpy(&flags, g->flags, sizeof(flags), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return check_hip(g, e, "read flags");
  if (flags & 2) {
    g->last_err = "a forced source individual was out of range (the individual kept itself)";
    return LIPZ_E_INVAL;
  }
  if (flags & 1) {
    g->last_err = "non-finite loss or fitness";
    return LIPZ_E_NONFINITE;
  }
  return LIPZ_OK;
}

const char* lipz_error_string(lipz_status s) {
  switch (s) {
    case LIPZ_OK: return "ok";
    case LIPZ_E_INVAL: return "invalid argument";
    case LIPZ_E_WORKSPACE: return "workspace too small or misaligned";
    case LIPZ_E_HIP: return "HIP runtime error";
    case LIPZ_E_ORDER: return "call out of order";
    case LIPZ_E_NONFINITE: return "non-finite loss or fitness";
    case LIPZ_E_UNSUPPORTED: return "unsupported configuration";
    default: return "unknown status";
  }
}

const char* lipz_last_error(const lipz_grid* g) { return g ? g->last_err.c_str() : ""; }

lipz_status lipz_set_gemm_timing(lipz_grid* g, int32_t enable) {
  if (!g) return LIPZ_E_INVAL;
  g->timing = enable != 0;
  return LIPZ_OK;
}

lipz_status lipz_gemm_timing(lipz_grid* g, double* h_ms, int64_t* h_launches, double* h_flops,
                             double* h_bytes) {
  if (!g) return LIPZ_E_INVAL;
  hipError_t e = hipStreamSynchronize(g->stream);
  if (e != hipSuccess) return check_hip(g, e, "timing sync");
  for (size_t i = 0; i < g->ev_live.size(); ++i) {
    float ms = 0.f;
    hipEventElapsedTime(&ms, g->ev_live[i].first, g->ev_live[i].second);
    g->gemm_ms += ms;
    g->gemm_flops += g->ev_flops[i];
    g->gemm_bytes += g->ev_bytes[i];
    g->gemm_launches += 1;
    g->ev_pool.push_back(g->ev_live[i].first);
    g->ev_pool.push_back(g->ev_live[i].second);
  }
  g->ev_live.clear();
  g->ev_flops.clear();
  g->ev_bytes.clear();
  if (h_ms) *h_ms = g->gemm_ms;
  if (h_launches) *h_launches = g->gemm_launches;
  if (h_flops) *h_flops = g->gemm_flops;
  if (h_bytes) *h_bytes = g->gemm_bytes;
  g->gemm_ms = 0.0;
  g->gemm_flops = 0.0;
  g->gemm_bytes = 0.0;
  g->gemm_launches = 0;
  return LIPZ_OK;
}

lipz_status lipz_test_plan_bounds(const lipz_config* cfg, int64_t n_samples, char* msg, int32_t msg_len,
                                  int32_t* n_bad) {
  if (!n_bad) return LIPZ_E_INVAL;
  *n_bad = 0;
  // Placeholder addresses, never dereferenced: the plan is only inspected.
  char* const base = reinterpret_cast<char*>((uintptr_t)1 << 40);
  const float* const data = reinterpret_cast<const float*>((uintptr_t)1 << 44);
  size_t total = 0;
  lipz_grid* g = plan_grid(cfg, n_samples, base, data, &total);
  if (!g) return LIPZ_E_INVAL;
  const char* lo[2] = {base, (const char*)data};
  const char* hi[2] = {base + total, (const char*)data + (size_t)n_samples * g->xd * 4};
  std::string text;
  int bad = 0;
  auto inside = [&](const void* p, int64_t first, int64_t last) {
    if (!p || first < 0) return false;
    const char* a = (const char*)p + 4 * first;
    const char* b = (const char*)p + 4 * (last + 1);
    for (int i = 0; i < 2; ++i)
      if (a >= lo[i] && b <= hi[i]) return true;
    return false;
  };
  auto note = [&](const char* what, size_t i) {
    ++bad;
    if (text.size() < 2000) text += std::string(what) + " #" + std::to_string(i) + "; ";
  };
  for (size_t i = 0; i < g->probs_h.size(); ++i) {
    const GemmProb& p = g->probs_h[i];
    const int64_t a_last = p.a_trans ? (int64_t)(p.K - 1) * p.lda + p.a_rows - 1 : (int64_t)(p.a_rows - 1) * p.lda + p.K - 1;
    const int64_t b_last = p.b_trans ? (int64_t)(p.N - 1) * p.ldb + p.K - 1 : (int64_t)(p.K - 1) * p.ldb + p.N - 1;
    const int64_t c_last = (int64_t)(p.M - 1) * p.ldc + p.N - 1;
    if (!inside(p.A, 0, a_last)) note("gemm A", i);
    if (!inside(p.B, 0, b_last)) note("gemm B", i);
    if (!inside(p.C, 0, c_last)) note("gemm C", i);
    if (c_last >= ((int64_t)1 << 29)) note("gemm C byte offset", i);
    if (p.epi == EPI_ADAM && (!inside(p.m, 0, c_last) || !inside(p.v, 0, c_last) || !inside(p.lr, 0, 0) ||
                              !inside(p.t, 0, 0)))
      note("gemm Adam state", i);
    if (p.epi == EPI_DACT && !inside(p.aux, 0, c_last)) note("gemm aux", i);
    if (p.epi == EPI_BIAS_ACT && p.bias && !inside(p.bias, 0, p.N - 1)) note("gemm bias", i);
    if (p.epi == EPI_BIAS_ACT && p.dot_out &&
        (!inside(p.dot_out, 0, (int64_t)(p.M - 1) * p.dot_ld + (p.N + GEMM_BN - 1) / GEMM_BN - 1) ||
         !inside(p.dotw, 0, p.N - 1)))
      note("gemm dot", i);
    // fields that share storage with others are checked under the epilogue that reads them
    if (p.epi == EPI_BIAS_ACT && p.dot_out && p.gout && !inside(p.gout, 0, c_last)) note("gemm head factor", i);
    if (p.epi == EPI_DACT && p.rs_mode) {
      if (p.rs_tn < 1 || !inside(p.rs_part, 0, (int64_t)p.M * p.rs_tn - 1)) note("gemm head logits", i);
      if (p.side && (p.side_ld < p.N + 4 || !inside(p.side, 0, (int64_t)(p.M - 1) * p.side_ld + p.N + 3) ||
                     !inside(p.dlout, 0, (int64_t)p.M * 4 - 1)))
        note("gemm head side outputs", i);
      // row tile m0 / BM (BM >= 32) of the output layer's gradient pieces
      if (p.rs_mode == 1 && p.hpart &&
          (p.hp_w < 1 || p.hp_w > p.N || p.hp_ld < p.hp_w + 1 ||
           !inside(p.hpart, 0, (int64_t)((p.M - 1) / 32) * p.hp_ld + p.hp_w) ||
           !inside(p.hsrc, 0, (int64_t)p.M * p.hp_w - 1)))
        note("gemm head gradient pieces", i);
    }
  }
  // every GEMM launch's block -> tile map covers each tile exactly once and
  // spreads each group over the 8 XCDs within one tile
  for (size_t k = 0; k < g->phases.size(); ++k) {
    const Phase& ph = g->phases[k];
    std::vector<int> seen((size_t)ph.tiles, 0), per((size_t)ph.grp.n * 8, 0);
    bool ok = ph.grp.n >= 1;
    for (int b = 0; ok && b < ph.tiles; ++b) {
      const int t = xcd_group_tile(b, ph.tiles, ph.grp);
      if (t < 0 || t >= ph.tiles || seen[(size_t)t]++) {
        ok = false;
        break;
      }
      int gi = 0;
      for (int q = 1; q < ph.grp.n; ++q)
        if (t >= ph.grp.first_tile[q]) gi = q;
      ++per[(size_t)gi * 8 + (b & 7)];
    }
    for (int gi = 0; ok && gi < ph.grp.n; ++gi) {
      const auto mm = std::minmax_element(per.begin() + gi * 8, per.begin() + gi * 8 + 8);
      ok = *mm.second - *mm.first <= 1;
    }
    if (!ok) note("gemm tile map", k);
  }
  if (!g->dc) {
    // the sample, evaluation-head, fitness, selection and re-evaluation
    // kernels' extents (cells C, individuals U, neighbourhood nn)
    const int64_t C = g->C, U = g->U, B = g->B, tn = g->tn, nn = g->nn, s = g->s, er = 1 + nn;
    if (!inside(g->Xe, 0, C * er * B * g->xd - 1) || !inside(g->ze, 0, C * B * g->zd - 1)) note("eval sample", 0);
    if (!inside(g->Xtr, 0, U * 2 * B * g->xd - 1) || !inside(g->z, 0, U * B * g->zd - 1)) note("train sample", 0);
    if (g->fused_sample &&
        (!inside(g->Xtr_alt, 0, U * 2 * B * g->xd - 1) || !inside(g->z_alt, 0, U * B * g->zd - 1)))
      note("train sample, odd steps", 0);
    if (!inside(g->part_e, 0, C * nn * er * B * tn - 1)) note("eval logits", 0);
    if (!inside(g->L, 0, C * nn * nn - 1) || !inside(g->Lg, 0, C * nn * nn - 1)) note("eval losses", 0);
    if (!inside(g->fit_g, 0, C * nn - 1) || !inside(g->fit_d, 0, C * nn - 1)) note("fitness", 0);
    if (!inside(g->sel, 0, U * 2 - 1) || !inside(g->nbr, 0, C * 5 - 1)) note("selection", 0);
    if (!inside(g->dlbuf, 0, U * 2 * B * 4 - 1) || !inside(g->part_tr, 0, U * 2 * B * tn - 1) ||
        !inside(g->part_g, 0, U * B * tn - 1))
      note("train heads", 0);
    if (g->cfg.elitism) {
      if (!inside(g->part_e2, 0, C * nn * s * B * tn - 1) || !inside(g->part_e3, 0, C * s * er * B * tn - 1))
        note("re-evaluation logits", 0);
      if (!inside(g->rmean, 0, C * nn - 1) || !inside(g->el_L2, 0, C * s * nn - 1) ||
          !inside(g->el_Lg2, 0, C * s * nn - 1) || !inside(g->el_M3, 0, C * (1 + nn) * s - 1))
        note("re-evaluation means", 0);
      if (!inside(g->fit2_g, 0, C * s - 1) || !inside(g->fit2_d, 0, C * s - 1) || !inside(g->esrc, 0, U * 2 - 1))
        note("elitist truncation", 0);
    }
  }
  if (g->cfg.mix_enable) {
    // the mixture kernels' fp64 moments [C][F] x 2, chunk sums
    // [C][ceil(S / 64)][2][F] and data statistics [F] x 2 (in floats: 2 per double)
    const int64_t C = g->C, F = g->F, nch = (g->S + 63) / 64;
    if (!inside(g->mu_k, 0, 2 * C * F - 1) || !inside(g->s2_k, 0, 2 * C * F - 1) ||
        !inside(g->mom_part, 0, 2 * C * nch * 2 * F - 1))
      note("mixture moments", 0);
    if (!inside(g->mu_r, 0, 2 * F - 1) || !inside(g->sd_r, 0, 2 * F - 1)) note("mixture data statistics", 0);
    if (!inside(g->fm, 0, C * g->S * F - 1) || !inside(g->realfeat, 0, g->N * F - 1)) note("mixture features", 0);
  }
  if (g->cfg.trainer != LIPZ_TRAINER_GRADIENT) {
    // the NES / ES kernels' extents: sets [C][2n][stride] and directions
    // [C][n][eps_stride] (elements e < P), partial logits [C][Q][rows][tn],
    // losses [C][Q]
    const int64_t Q = g->nes_q, C = g->U, B = g->B, tn = g->tn, n = g->cfg.nes_pairs;
    if (g->D.P > g->D.stride || g->G.P > g->G.stride) note("nes parameter row", 0);
    if (g->cfg.trainer == LIPZ_TRAINER_NES && (g->D.P > g->nes_eps_stride || g->G.P > g->nes_eps_stride))
      note("nes direction row", 0);
    if (!inside(g->nes_pd, 0, C * 2 * n * g->D.stride - 1)) note("nes sets D", 0);
    if (!inside(g->nes_pg, 0, C * 2 * n * g->G.stride - 1)) note("nes sets G", 0);
    if (g->cfg.trainer == LIPZ_TRAINER_NES && !inside(g->nes_eps, 0, C * n * g->nes_eps_stride - 1))
      note("nes directions", 0);
    if (!inside(g->nes_part_d, 0, C * Q * 2 * B * tn - 1)) note("nes logits D", 0);
    if (!inside(g->nes_part_g, 0, C * Q * B * tn - 1)) note("nes logits G", 0);
    if (!inside(g->nes_fd, 0, C * Q - 1) || !inside(g->nes_fg, 0, C * Q - 1)) note("nes losses", 0);
  }
  if (g->dc) bad += dc_check_bounds(g, lo, hi, 2, &text);
  *n_bad = bad;
  if (msg && msg_len > 0) {
    const size_t n = text.size() < (size_t)msg_len - 1 ? text.size() : (size_t)msg_len - 1;
    memcpy(msg, text.data(), n);
    msg[n] = 0;
  }
  dc_delete(g->dc);
  delete g;
  return LIPZ_OK;
}

}  // extern "C"
