// Plans of the DCGAN-style networks (the CelebA network of the paper's
// experiment settings, Section 4): buffers, the per-phase problem tables of
// one training step and one evaluation for both state buffers, and their
// execution.
//
// Networks (n stride-2 stages, image side 4 * 2^n, NHWC):
//   G: dense z -> 4x4xg0, BN, act | n-1 x [4x4 transposed conv s2 p1, BN,
//      act] | 4x4 transposed conv s2 p1 to the image channels + bias, out act
//   D: n x [4x4 conv s2 p1 + bias, act] | dense 4x4xd(n-1) -> 1 + bias
// Parameter row of a layer: weights [(taps * c_in)][c_out] with rows
// (kh, kw, c_in), then the bias [c_out] if any, then gamma and beta.
// Batch norm always normalises with the statistics of the batch it sees.
//
// A training step (Section 3 step 3) runs, for all cells at once:
//   sample | G forward (dense GEMM, BN, 4-phase transposed convs, BN, ...)
//   | D forward on the 2B real+fake images | logits | BCE head, output-layer
//   gradient + Adam | D input gradients (4-phase) beside D weight gradients
//   (split-K partial sums) | reduce + Adam of D | D forward on the fakes with
//   the updated D | logits | non-saturating head | D input gradients down to
//   the image | G weight and input gradients layer by layer with BN backward
//   (gamma, beta Adam) | G dense weight gradient + Adam | reduce + Adam of G.
#include <math.h>
#include <string.h>

#include "grid.h"

namespace lipz {

namespace {

enum LayerKind { LK_DENSE = 0, LK_CONV = 1, LK_CONVT = 2 };

struct DcLayer {
  int kind;
  int cin, cout;           // channels (dense: fan_in, fan_out)
  int in_log, out_log;     // log2 of the input / output side
  int bias, bn, act;
  int64_t off_w, n_w, off_b, off_g;
  int nb;                  // batch-norm channels
};

struct DcNet {
  int nl = 0;
  DcLayer L[LIPZ_MAX_HIDDEN + 1];
  int64_t P = 0;
};

struct ConvPhase {
  int first = 0, count = 0, tiles = 0;  // tiles: blocks of the launch
  ConvGroups grp;
  double flops = 0.0;
  double bytes = 0.0;  // algorithmic: each tensor read or written once
};
struct BnOp {
  int first, count, blocks;
  int64_t max_elems;
};
struct RedOp {
  int first, count;
  int64_t max_n;
};
struct DotOp {
  int first, count, rows;
};
struct ColOp {
  int first, count;
  int64_t max_work;  // im2col: (position, tap) pairs; col2im: map elements (per descriptor, the largest)
};

enum DcOpKind {
  DC_SAMPLE, DC_GEMM, DC_CONV, DC_BN_FWD, DC_BN_BWD, DC_REDUCE, DC_DOT, DC_HEAD_D, DC_HEAD_G, DC_IM2COL, DC_COL2IM
};
struct DcOp {
  DcOpKind kind;
  int idx;
};

#ifndef LIPZ_CONV_KSPLIT
#define LIPZ_CONV_KSPLIT 1024
#endif
constexpr int KSPLIT = LIPZ_CONV_KSPLIT;  // positions per split of a weight gradient

int ilog2(int v) {
  int l = 0;
  while ((1 << l) < v) ++l;
  return (1 << l) == v ? l : -1;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

PosMap posmap(int h_log, int w_log, int sy, int y0, int sx, int x0, int ld) {
  PosMap m;
  m.h_log = h_log;
  m.w_log = w_log;
  m.sy = sy;
  m.y0 = y0;
  m.sx = sx;
  m.x0 = x0;
  m.ld = ld;
  return m;
}

uint32_t extent(int64_t floats) {
  const int64_t b = floats * 4;
  return b < 0x7FFFFFF0ll ? (uint32_t)b : 0u;
}

ConvProb conv_base(int mode) {
  ConvProb p;
  memset(&p, 0, sizeof(p));
  p.mode = mode;
  p.ones_row = -1;
  p.brow = -1;
  p.cs_log = -1;
  p.kw_full = 4;
  return p;
}

void set_taps(ConvProb& p, int tw_log, int cs, int tys, int ty0, int tx0, int khs, int kh0, int kw0) {
  p.tw_log = tw_log;
  p.taps = 1 << (2 * tw_log);
  p.cs = cs;
  p.cs_log = ilog2(cs);
  p.tys = tys;
  p.ty0 = ty0;
  p.tx0 = tx0;
  p.khs = khs;
  p.kh0 = kh0;
  p.kw0 = kw0;
}

// 4x4 convolution, stride 2, pad 1: in [NI][2^h][2^h][cin] -> out [NI][2^(h-1)]^2[cout].
ConvProb conv_fwd(const float* in, int NI, int h, int cin, const float* W, int cout, float* out, int epi, int act,
                  const float* bias) {
  ConvProb p = conv_base(CONV_FWD);
  p.gh_log = p.gw_log = h - 1;
  p.M = NI << (2 * (h - 1));
  p.N = cout;
  p.K = 16 * cin;
  set_taps(p, 2, cin, 1, -1, -1, 1, 0, 0);
  p.S = in;
  p.smap = posmap(h, h, 2, 0, 2, 0, cin);
  p.s_bytes = extent(((int64_t)NI << (2 * h)) * cin);
  p.W = W;
  p.wsc = cout;
  p.wsn = 1;
  p.w_bytes = extent((int64_t)16 * cin * cout);
  p.omap = posmap(h - 1, h - 1, 1, 0, 1, 0, cout);
  p.C = out;
  p.epi = epi;
  p.act = act;
  p.bias = bias;
  p.gen = !(cin % 4 == 0 && cout % 4 == 0 && aligned16(in) && aligned16(W));
  return p;
}

// Phase (r, q) of the 4x4 transposed convolution, stride 2, pad 1:
// in [NI][2^h]^2[cin] -> out [NI][2^(h+1)]^2[cout] at (2y + r, 2x + q).
ConvProb convT_phase(const float* in, int NI, int h, int cin, const float* W, int cout, float* out, int r, int q,
                     int epi, int act, const float* bias) {
  ConvProb p = conv_base(CONV_FWD);
  p.gh_log = p.gw_log = h;
  p.M = NI << (2 * h);
  p.N = cout;
  p.K = 4 * cin;
  set_taps(p, 1, cin, -1, r, q, 2, 1 - r, 1 - q);
  p.S = in;
  p.smap = posmap(h, h, 1, 0, 1, 0, cin);
  p.s_bytes = extent(((int64_t)NI << (2 * h)) * cin);
  p.W = W;
  p.wsc = cout;
  p.wsn = 1;
  p.w_bytes = extent((int64_t)16 * cin * cout);
  p.omap = posmap(h + 1, h + 1, 2, r, 2, q, cout);
  p.C = out;
  p.epi = epi;
  p.act = act;
  p.bias = bias;
  p.gen = !(cin % 4 == 0 && cout % 4 == 0 && aligned16(in) && aligned16(W));
  return p;
}

// Phase (r, q) of the input gradient of conv_fwd: dout [NI][2^(h-1)]^2[cout]
// -> din [NI][2^h]^2[cin] at (2y + r, 2x + q), times act'(aux) (aux = the
// forward input, same layout as din).
ConvProb conv_dgrad_phase(const float* dout, int NI, int h, int cin, int cout, const float* W, float* din,
                          const float* aux, int act, int r, int q) {
  ConvProb p = conv_base(CONV_FWD);
  p.gh_log = p.gw_log = h - 1;
  p.M = NI << (2 * (h - 1));
  p.N = cin;
  p.K = 4 * cout;
  set_taps(p, 1, cout, -1, r, q, 2, 1 - r, 1 - q);
  p.S = dout;
  p.smap = posmap(h - 1, h - 1, 1, 0, 1, 0, cout);
  p.s_bytes = extent(((int64_t)NI << (2 * (h - 1))) * cout);
  p.W = W;
  p.wsc = 1;
  p.wsn = cout;
  p.w_bytes = extent((int64_t)16 * cin * cout);
  p.omap = posmap(h, h, 2, r, 2, q, cin);
  p.C = din;
  p.epi = EPI_DACT;
  p.act = act;
  p.aux = aux;
  p.gen = !(cin % 4 == 0 && cout % 4 == 0 && aligned16(dout) && aligned16(W));
  return p;
}

// Input gradient of convT_phase (all phases): dout [NI][2^(h+1)]^2[cout] ->
// din [NI][2^h]^2[cin], a stride-2 convolution with the transposed weights,
// times act'(aux).
ConvProb convT_dgrad(const float* dout, int NI, int h, int cin, int cout, const float* W, float* din,
                     const float* aux, int act) {
  ConvProb p = conv_base(CONV_FWD);
  p.gh_log = p.gw_log = h;
  p.M = NI << (2 * h);
  p.N = cin;
  p.K = 16 * cout;
  set_taps(p, 2, cout, 1, -1, -1, 1, 0, 0);
  p.S = dout;
  p.smap = posmap(h + 1, h + 1, 2, 0, 2, 0, cout);
  p.s_bytes = extent(((int64_t)NI << (2 * (h + 1))) * cout);
  p.W = W;
  p.wsc = 1;
  p.wsn = cout;
  p.w_bytes = extent((int64_t)16 * cin * cout);
  p.omap = posmap(h, h, 1, 0, 1, 0, cin);
  p.C = din;
  p.epi = EPI_DACT;
  p.act = act;
  p.aux = aux;
  p.gen = !(cin % 4 == 0 && cout % 4 == 0 && aligned16(dout) && aligned16(W));
  return p;
}

void set_split(ConvProb& p, int ksplit, int rows_total) {
  p.ksplit = ksplit;
  p.splits = (p.K + ksplit - 1) / ksplit;
  p.ldc = p.N;
  p.split_stride = (int64_t)rows_total * p.N;
}

int splits_for(int K) { return (K + KSPLIT - 1) / KSPLIT; }

// Weight gradient of conv_fwd (+ bias row): partial sums [splits][16 cin + 1][cout].
ConvProb conv_wgrad(const float* in, int NI, int h, int cin, const float* dout, int cout, float* part) {
  ConvProb p = conv_base(CONV_WG);
  p.gh_log = p.gw_log = h - 1;
  p.M = 16 * cin + 1;
  p.N = cout;
  p.K = NI << (2 * (h - 1));
  set_taps(p, 2, cin, 1, -1, -1, 1, 0, 0);
  p.S = in;
  p.smap = posmap(h, h, 2, 0, 2, 0, cin);
  p.s_bytes = extent(((int64_t)NI << (2 * h)) * cin);
  p.P = dout;
  p.pmap = posmap(h - 1, h - 1, 1, 0, 1, 0, cout);
  p.p_bytes = extent((int64_t)p.K * cout);
  p.ones_row = 16 * cin;
  p.brow = 16 * cin;
  p.C = part;
  set_split(p, KSPLIT, 16 * cin + 1);
  p.gen = !(cin % 4 == 0 && cout % 4 == 0 && aligned16(in) && aligned16(dout));
  return p;
}

// Weight-gradient rows of the 4 taps of phase (r, q) of convT_phase, reduced
// over the input positions: partial sums in [splits][rows_total][cout].
ConvProb convT_wgrad_phase(const float* in, int NI, int h, int cin, const float* dout, int cout, float* part,
                           int rows_total, int r, int q) {
  ConvProb p = conv_base(CONV_WG);
  p.gh_log = p.gw_log = h;
  p.M = 4 * cin;
  p.N = cout;
  p.K = NI << (2 * h);
  set_taps(p, 1, cin, -1, r, q, 2, 1 - r, 1 - q);
  p.S = in;
  p.smap = posmap(h, h, 1, 0, 1, 0, cin);
  p.s_bytes = extent((int64_t)p.K * cin);
  p.P = dout;
  p.pmap = posmap(h + 1, h + 1, 2, r, 2, q, cout);
  p.p_bytes = extent(((int64_t)NI << (2 * (h + 1))) * cout);
  p.C = part;
  set_split(p, KSPLIT, rows_total);
  p.gen = !(cin % 4 == 0 && cout % 4 == 0 && aligned16(in) && aligned16(dout));
  return p;
}

// Bias gradient of a transposed convolution: the sum of dout over every
// output position, as the ones row of a 1-row weight-gradient problem, in
// the same split layout as its phases (4x the positions per split).
ConvProb convT_bias_grad(const float* dout, int NI, int h_out, int cout, float* part, int rows_total, int brow) {
  ConvProb p = conv_base(CONV_WG);
  p.gh_log = p.gw_log = h_out;
  p.M = 1;
  p.N = cout;
  p.K = NI << (2 * h_out);
  p.taps = 0;
  p.cs = 0;
  p.S = dout;
  p.smap = posmap(h_out, h_out, 1, 0, 1, 0, cout);
  p.s_bytes = extent((int64_t)p.K * cout);
  p.P = dout;
  p.pmap = posmap(h_out, h_out, 1, 0, 1, 0, cout);
  p.p_bytes = p.s_bytes;
  p.ones_row = 0;
  p.brow = brow;
  p.C = part;
  set_split(p, 4 * KSPLIT, rows_total);
  p.gen = !(cout % 4 == 0 && aligned16(dout));
  return p;
}

// Rows = the positions of a [NI][2^g]^2 grid of a position-major matrix
// S[p][0..cs) (a 1-tap convolution): out[p][n] = sum_k S[p][k] W(k, n) with
// W row-major [cs][N], or transposed [N][cs].
ConvProb dense_rows(const float* S, int NI, int g, int cs, const float* W, int N, bool w_transposed, float* out,
                    int epi, int act, const float* bias) {
  ConvProb p = conv_base(CONV_FWD);
  p.gh_log = p.gw_log = g;
  p.M = NI << (2 * g);
  p.N = N;
  p.K = cs;
  set_taps(p, 0, cs, 0, 0, 0, 0, 0, 0);
  p.S = S;
  p.smap = posmap(g, g, 1, 0, 1, 0, cs);
  p.s_bytes = extent((int64_t)p.M * cs);
  p.W = W;
  p.wsc = w_transposed ? 1 : N;
  p.wsn = w_transposed ? cs : 1;
  p.w_bytes = extent((int64_t)cs * N);
  p.omap = posmap(g, g, 1, 0, 1, 0, N);
  p.C = out;
  p.epi = epi;
  p.act = act;
  p.bias = bias;
  p.gen = !(cs % 4 == 0 && N % 4 == 0 && aligned16(S) && aligned16(W));
  return p;
}

// Weight gradient of dense_rows (row-major weights, + bias row when
// with_bias): partial sums of S^T dY over the positions.
ConvProb dense_rows_wgrad(const float* S, int NI, int g, int cs, const float* dY, int N, float* part, int rows_total,
                          bool with_bias) {
  ConvProb p = conv_base(CONV_WG);
  p.gh_log = p.gw_log = g;
  p.K = NI << (2 * g);
  p.M = cs + (with_bias ? 1 : 0);
  p.N = N;
  set_taps(p, 0, cs, 0, 0, 0, 0, 0, 0);
  p.S = S;
  p.smap = posmap(g, g, 1, 0, 1, 0, cs);
  p.s_bytes = extent((int64_t)p.K * cs);
  p.P = dY;
  p.pmap = posmap(g, g, 1, 0, 1, 0, N);
  p.p_bytes = extent((int64_t)p.K * N);
  p.ones_row = with_bias ? cs : -1;
  p.brow = cs;
  p.C = part;
  set_split(p, KSPLIT, rows_total);
  p.gen = !(cs % 4 == 0 && N % 4 == 0 && aligned16(S) && aligned16(dY));
  return p;
}

// Columns of a stride-2 transposed convolution [c_in][16 taps x c_out]
// (weights [tap][c_in][c_out] read with column taps): out = S W.
ConvProb convT_cols(const float* S, int NI, int g, int cin, const float* W, int cout, float* cols) {
  ConvProb p = dense_rows(S, NI, g, cin, W, 16 * cout, false, cols, EPI_STORE, 0, nullptr);
  p.wsc = cout;
  p.wsn = 1;
  p.n_inner = cout;
  p.n_tap_stride = cin * cout;
  p.w_bytes = extent((int64_t)16 * cin * cout);
  p.gen = 1;
  return p;
}

double conv_flops(const ConvProb& p) {
  const double rows = p.mode == CONV_WG ? (double)p.taps * p.cs : (double)p.M;
  return 2.0 * rows * p.N * p.K;
}

// Each input tensor element read once, each output element written once
// (weight-gradient partial sums: written once per split).
double conv_bytes(const ConvProb& p) {
  if (p.mode == CONV_FWD) {
    const int NI = p.M >> (p.gh_log + p.gw_log);
    double b = (double)(((int64_t)NI << p.smap.h_log) << p.smap.w_log) * p.smap.ld;  // source
    b += (double)p.taps * p.cs * p.N;                                              // weights
    b += (double)p.M * p.N * (p.epi == EPI_DACT ? 2.0 : 1.0);                      // output (+ aux)
    return 4.0 * b;
  }
  const int NI = p.K >> (p.gh_log + p.gw_log);
  double b = p.taps ? (double)(((int64_t)NI << p.smap.h_log) << p.smap.w_log) * p.smap.ld : 0.0;
  b += (double)p.K * p.N;                                 // output gradient at the grid positions
  b += (double)p.splits * p.M * p.N;                      // partial sums
  return 4.0 * b;
}

}  // namespace

struct DcPlan {
  DcNet G, D;
  bool plan_ok = true;  // false if a phase exceeded the launch descriptor's shape groups
  int n = 0, img_log = 0, ic = 0;
  // training (per cell)
  float *z = nullptr, *Xtr = nullptr, *gdimg = nullptr;
  float *gx[LIPZ_MAX_HIDDEN] = {}, *gy[LIPZ_MAX_HIDDEN] = {}, *gdz[LIPZ_MAX_HIDDEN] = {};
  float *dy[LIPZ_MAX_HIDDEN] = {}, *ddel[LIPZ_MAX_HIDDEN] = {}, *dyg[LIPZ_MAX_HIDDEN] = {},
        *ddelg[LIPZ_MAX_HIDDEN] = {};
  float *part_tr = nullptr, *part_g = nullptr, *dlbuf = nullptr;
  float *bn_part[LIPZ_MAX_HIDDEN] = {}, *bn_stats[LIPZ_MAX_HIDDEN] = {};
  int64_t bn_part_cell[LIPZ_MAX_HIDDEN] = {};
  float *gpart[LIPZ_MAX_HIDDEN + 1] = {}, *dpart[LIPZ_MAX_HIDDEN] = {};
  int64_t gpart_cell[LIPZ_MAX_HIDDEN + 1] = {}, dpart_cell[LIPZ_MAX_HIDDEN] = {};
  // evaluation (per (cell, slot))
  float *patch = nullptr, *cols = nullptr;  // image patches [2B][..][16 ic]; 16-tap columns [B][..][16 ic]
  float *ze = nullptr, *Xe = nullptr, *part_e = nullptr;
  float *epatch = nullptr, *ecols = nullptr;
  float *gex[LIPZ_MAX_HIDDEN] = {}, *dey[2] = {};
  float *bne_part[LIPZ_MAX_HIDDEN] = {}, *bne_stats[LIPZ_MAX_HIDDEN] = {};
  // tables
  std::vector<ConvProb> conv_h;
  std::vector<BnProb> bn_h;
  std::vector<RedProb> red_h;
  std::vector<DotProb> dot_h;
  std::vector<ColProb> col_h;
  ConvProb* conv_d = nullptr;
  BnProb* bn_d = nullptr;
  RedProb* red_d = nullptr;
  DotProb* dot_d = nullptr;
  ColProb* col_d = nullptr;
  std::vector<ConvPhase> cph;
  std::vector<BnOp> bnops;
  std::vector<RedOp> redops;
  std::vector<DotOp> dotops;
  std::vector<ColOp> colops;
  std::vector<DcOp> train_ops[2], eval_ops[2];
};

namespace {

int64_t side_sq(int log) { return (int64_t)1 << (2 * log); }

void describe(const lipz_config* c, DcNet& G, DcNet& D, int* n_out, int* img_log_out) {
  const int n = c->n_g_hidden;
  const int img_log = 2 + n;
  auto add = [](DcNet& N, int kind, int cin, int cout, int in_log, int out_log, int bias, int bn, int act) {
    DcLayer& L = N.L[N.nl++];
    L.kind = kind;
    L.cin = cin;
    L.cout = cout;
    L.in_log = in_log;
    L.out_log = out_log;
    L.bias = bias;
    L.bn = bn;
    L.act = act;
    const int taps = kind == LK_DENSE ? 1 : 16;
    L.off_w = N.P;
    L.n_w = (int64_t)taps * cin * cout;
    N.P += L.n_w;
    L.off_b = bias ? N.P : -1;
    N.P += bias ? cout : 0;
    L.nb = bn ? (kind == LK_DENSE ? cout / 16 : cout) : 0;
    L.off_g = bn ? N.P : -1;
    N.P += 2 * L.nb;
  };
  G = DcNet();
  D = DcNet();
  add(G, LK_DENSE, c->z_dim, 16 * c->g_hidden[0], 0, 2, 0, 1, c->g_hidden_act);
  for (int k = 1; k < n; ++k) add(G, LK_CONVT, c->g_hidden[k - 1], c->g_hidden[k], 1 + k, 2 + k, 0, 1, c->g_hidden_act);
  add(G, LK_CONVT, c->g_hidden[n - 1], c->img_c, 1 + n, 2 + n, 1, 0, c->g_out_act);
  int cin = c->img_c;
  for (int k = 0; k < n; ++k) {
    add(D, LK_CONV, cin, c->d_hidden[k], img_log - k, img_log - k - 1, 1, 0, c->d_hidden_act);
    cin = c->d_hidden[k];
  }
  add(D, LK_DENSE, 16 * cin, 1, 2, 0, 1, 0, LIPZ_ACT_LINEAR);
  *n_out = n;
  *img_log_out = img_log;
}

}  // namespace

std::string dc_validate(const lipz_config* c, Net* Gn, Net* Dn) {
  const int n = c->n_g_hidden;
  if (c->n_d_hidden != n) return "DCGAN: n_g_hidden and n_d_hidden must both be the number of stride-2 stages";
  if (c->img_h != c->img_w || c->img_h != (4 << n)) return "DCGAN: images must be square with side 4 * 2^n";
  if (c->img_c < 1 || c->img_c > 64) return "DCGAN: img_c must be in [1, 64]";
  if ((int64_t)c->img_h * c->img_w * c->img_c != c->x_dim) return "DCGAN: x_dim must be img_h * img_w * img_c";
  for (int k = 0; k < n; ++k) {
    if (c->g_hidden[k] < 4 || c->g_hidden[k] > 1024 || c->g_hidden[k] % 4) return "DCGAN: channel widths must be multiples of 4 in [4, 1024]";
    if (c->d_hidden[k] < 4 || c->d_hidden[k] > 1024 || c->d_hidden[k] % 4) return "DCGAN: channel widths must be multiples of 4 in [4, 1024]";
  }
  if (c->mix_enable) return "DCGAN: the mixture step is defined for the MLP networks only";
  // every per-instance operand must stay below 2 GiB (32-bit buffer offsets)
  const int64_t lim = 0x7FFFFFF0ll / 4;
  if ((int64_t)6 * c->batch * c->x_dim >= lim) return "DCGAN: batch too large for the image size";
  for (int k = 0; k < n; ++k) {
    if ((int64_t)6 * c->batch * side_sq(1 + n - k) * c->d_hidden[k] >= lim)
      return "DCGAN: batch too large for the discriminator widths";
    if ((int64_t)c->batch * side_sq(2 + k) * c->g_hidden[k] >= lim) return "DCGAN: batch too large for the generator widths";
  }
  DcNet G, D;
  int nn, il;
  describe(c, G, D, &nn, &il);
  Gn->nl = G.nl;
  Gn->P = G.P;
  Gn->stride = (int64_t)align_up((size_t)G.P, 64);
  Dn->nl = D.nl;
  Dn->P = D.P;
  Dn->stride = (int64_t)align_up((size_t)D.P, 64);
  return "";
}

DcPlan* dc_new(const lipz_config* c) {
  DcPlan* p = new (std::nothrow) DcPlan();
  if (!p) return nullptr;
  describe(c, p->G, p->D, &p->n, &p->img_log);
  p->ic = c->img_c;
  return p;
}

bool dc_plan_ok(const DcPlan* p) { return p->plan_ok; }

void dc_delete(DcPlan* p) { delete p; }

void dc_carve(lipz_grid* g, Carver& cv) {
  DcPlan& P = *g->dc;
  const int C = g->C, B = g->B, zd = g->zd, xd = g->xd, n = P.n;
  auto tf = [&](int64_t k) { return cv.take<float>((size_t)k); };
  // training
  P.z = tf((int64_t)C * B * zd);
  P.Xtr = tf((int64_t)C * 2 * B * xd);
  P.gdimg = tf((int64_t)C * B * xd);
  for (int k = 0; k < n; ++k) {
    const DcLayer& L = P.G.L[k];
    const int64_t per = (int64_t)B * side_sq(L.out_log) * L.nb;
    P.gx[k] = tf(C * per);
    P.gy[k] = tf(C * per);
    P.gdz[k] = tf(C * per);
    const int64_t chunks = (B * side_sq(L.out_log) + BN_CHUNK - 1) / BN_CHUNK;
    P.bn_part_cell[k] = chunks * 2 * L.nb;
    P.bn_part[k] = tf(C * P.bn_part_cell[k]);
    P.bn_stats[k] = tf((int64_t)C * 5 * L.nb);
  }
  for (int k = 0; k < n; ++k) {
    const DcLayer& L = P.D.L[k];
    const int64_t per = side_sq(L.out_log) * L.cout;
    P.dy[k] = tf((int64_t)C * 2 * B * per);
    P.ddel[k] = tf((int64_t)C * 2 * B * per);
    P.dyg[k] = tf((int64_t)C * B * per);
    P.ddelg[k] = tf((int64_t)C * B * per);
    const int K = (2 * B) << (2 * L.out_log);
    P.dpart_cell[k] = (int64_t)splits_for(K) * (16 * L.cin + 1) * L.cout;
    P.dpart[k] = tf(C * P.dpart_cell[k]);
  }
  for (int k = 1; k <= n; ++k) {
    const DcLayer& L = P.G.L[k];
    const int K = B << (2 * L.in_log);
    P.gpart_cell[k] = (int64_t)splits_for(K) * (16 * L.cin + L.bias) * L.cout;
    P.gpart[k] = tf(C * P.gpart_cell[k]);
  }
  const int64_t pcols = ((int64_t)1 << (2 * (P.img_log - 1))) * 16 * P.ic;  // patch / column floats per image
  P.patch = tf((int64_t)C * 2 * B * pcols);
  P.cols = tf((int64_t)C * B * pcols);
  P.part_tr = tf((int64_t)C * 2 * B);
  P.part_g = tf((int64_t)C * B);
  P.dlbuf = tf((int64_t)C * 2 * B * 4);
  // evaluation
  P.ze = tf((int64_t)C * B * zd);
  P.Xe = tf((int64_t)C * 6 * B * xd);
  P.part_e = tf((int64_t)C * 5 * 6 * B);
  P.epatch = tf((int64_t)C * 6 * B * pcols);
  P.ecols = tf((int64_t)C * 5 * B * pcols);
  for (int k = 0; k < n; ++k) {
    const DcLayer& L = P.G.L[k];
    const int64_t rows = (int64_t)B * side_sq(L.out_log);
    P.gex[k] = tf((int64_t)C * 5 * rows * L.nb);
    P.bne_part[k] = tf((int64_t)C * 5 * ((rows + BN_CHUNK - 1) / BN_CHUNK) * 2 * L.nb);
    P.bne_stats[k] = tf((int64_t)C * 5 * 5 * L.nb);
  }
  int64_t pp[2] = {0, 0};
  for (int k = 0; k < n; ++k) {
    const DcLayer& L = P.D.L[k];
    const int64_t sz = (int64_t)C * 5 * 6 * B * side_sq(L.out_log) * L.cout;
    if (sz > pp[k & 1]) pp[k & 1] = sz;
  }
  P.dey[0] = tf(pp[0]);
  P.dey[1] = tf(pp[1] > 0 ? pp[1] : 4);
}

void dc_carve_tables(lipz_grid* g, Carver& cv) {
  DcPlan& P = *g->dc;
  P.conv_d = cv.take<ConvProb>(P.conv_h.size());
  P.bn_d = cv.take<BnProb>(P.bn_h.size());
  P.red_d = cv.take<RedProb>(P.red_h.size());
  P.dot_d = cv.take<DotProb>(P.dot_h.size());
  P.col_d = cv.take<ColProb>(P.col_h.size());
}

namespace {

int add_conv_phase(DcPlan& P, const std::vector<ConvProb>& ps) {
  ConvPhase ph;
  ph.first = (int)P.conv_h.size();
  ph.count = (int)ps.size();
  memset(&ph.grp, 0, sizeof(ph.grp));
  auto round8 = [](int v) { return (v + 7) & ~7; };
  int blocks = 0, prev = -1;
  for (size_t k = 0; k < ps.size(); ++k) {
    ConvProb p = ps[k];
    p.tn = p.N <= 16 ? 16 : 64;
    p.tiles_m = (p.M + 63) / 64;
    p.tiles_n = (p.N + p.tn - 1) / p.tn;
    if (p.mode != CONV_WG) p.splits = 1;
    const int tpp = p.tiles_m * p.tiles_n * p.splits;
    if (tpp != prev) {
      if (ph.grp.n == GEMM_MAX_GROUPS) {  // a plan this library builds never gets here
        P.plan_ok = false;
        break;
      }
      if (ph.grp.n > 0) blocks += round8(ph.grp.real_tiles[ph.grp.n - 1]);
      ph.grp.first_block[ph.grp.n] = blocks;
      ph.grp.first_prob[ph.grp.n] = (int)k;
      ph.grp.tiles_per_prob[ph.grp.n] = tpp;
      ++ph.grp.n;
      prev = tpp;
    }
    p.tile_begin = ph.grp.real_tiles[ph.grp.n - 1];
    ph.grp.real_tiles[ph.grp.n - 1] += tpp;
    ph.flops += conv_flops(p);
    ph.bytes += conv_bytes(p);
    P.conv_h.push_back(p);
  }
  for (int gi = 0; gi < ph.grp.n; ++gi) ph.grp.blocks[gi] = round8(ph.grp.real_tiles[gi]);
  ph.tiles = ph.grp.n ? ph.grp.first_block[ph.grp.n - 1] + ph.grp.blocks[ph.grp.n - 1] : 0;
  P.cph.push_back(ph);
  return (int)P.cph.size() - 1;
}

int add_bn_op(DcPlan& P, const std::vector<BnProb>& bs) {
  BnOp op;
  op.first = (int)P.bn_h.size();
  op.count = (int)bs.size();
  op.blocks = 0;
  op.max_elems = 0;
  for (BnProb b : bs) {
    b.first_block = op.blocks;
    op.blocks += (int)((b.rows + BN_CHUNK - 1) / BN_CHUNK) * ((b.ch + 63) / 64);
    const int64_t e = b.rows * b.ch;
    if (e > op.max_elems) op.max_elems = e;
    P.bn_h.push_back(b);
  }
  P.bnops.push_back(op);
  return (int)P.bnops.size() - 1;
}

int add_red_op(DcPlan& P, const std::vector<RedProb>& rs) {
  RedOp op;
  op.first = (int)P.red_h.size();
  op.count = (int)rs.size();
  op.max_n = 0;
  for (const RedProb& r : rs) {
    if (r.n > op.max_n) op.max_n = r.n;
    P.red_h.push_back(r);
  }
  P.redops.push_back(op);
  return (int)P.redops.size() - 1;
}

// im2col (to_cols) or col2im descriptors.
int add_col_op(DcPlan& P, const std::vector<ColProb>& cs, bool to_cols) {
  ColOp op;
  op.first = (int)P.col_h.size();
  op.count = (int)cs.size();
  op.max_work = 0;
  for (const ColProb& c : cs) {
    const int64_t w = to_cols ? ((int64_t)c.n_img << (2 * (c.h_log - 1))) * 16 : ((int64_t)c.n_img << (2 * c.h_log)) * c.ch;
    if (w > op.max_work) op.max_work = w;
    P.col_h.push_back(c);
  }
  P.colops.push_back(op);
  return (int)P.colops.size() - 1;
}

ColProb col_prob(const float* src, float* dst, int n_img, int h_log, int ch, int epi, int act, const float* bias,
                 const float* aux) {
  ColProb c;
  memset(&c, 0, sizeof(c));
  c.src = src;
  c.dst = dst;
  c.n_img = n_img;
  c.h_log = h_log;
  c.ch = ch;
  c.epi = epi;
  c.act = act;
  c.bias = bias;
  c.aux = aux;
  return c;
}

int add_dot_op(DcPlan& P, const std::vector<DotProb>& ds) {
  DotOp op;
  op.first = (int)P.dot_h.size();
  op.count = (int)ds.size();
  op.rows = 0;
  for (DotProb d : ds) {
    d.first_row = op.rows;
    op.rows += d.rows;
    P.dot_h.push_back(d);
  }
  P.dotops.push_back(op);
  return (int)P.dotops.size() - 1;
}

BnProb bn_prob(const float* x, float* y, int64_t rows, int ch, float* part, float* stats, float* gamma, float* gm,
               float* gv, const float* lr, const int32_t* t, int act) {
  BnProb b;
  memset(&b, 0, sizeof(b));
  b.x = x;
  b.y = y;
  b.rows = rows;
  b.ch = ch;
  b.part = part;
  b.stats = stats;
  b.gamma = gamma;
  b.gm = gm;
  b.gv = gv;
  b.lr = lr;
  b.t = t;
  b.act = act;
  return b;
}

}  // namespace

void dc_build(lipz_grid* g) {
  DcPlan& P = *g->dc;
  // the Wasserstein critic's parameters are clipped after every update
  const float d_clip = g->cfg.loss_kind == LIPZ_LOSS_WASSERSTEIN ? g->cfg.wgan_clip : 0.f;
  P.conv_h.clear();
  P.bn_h.clear();
  P.red_h.clear();
  P.dot_h.clear();
  P.col_h.clear();
  P.cph.clear();
  P.bnops.clear();
  P.redops.clear();
  P.dotops.clear();
  P.colops.clear();
  const int C = g->C, B = g->B, zd = g->zd, xd = g->xd, n = P.n;
  const int64_t sG = g->G.stride, sD = g->D.stride;
  const DcNet &G = P.G, &D = P.D;
  const DcLayer& H = D.L[n];  // D's dense output layer
  const int Hw = H.cin;
  for (int par = 0; par < 2; ++par) {
    const StateBuf& S = g->st[par];
    std::vector<DcOp>& ops = P.train_ops[par];
    ops.clear();
    auto gemm = [&](const std::vector<GemmProb>& ps) { ops.push_back({DC_GEMM, add_phase(g, ps)}); };
    auto conv = [&](const std::vector<ConvProb>& ps) { ops.push_back({DC_CONV, add_conv_phase(P, ps)}); };
    auto Gw = [&](int c, int l) { return S.Gp + c * sG + G.L[l].off_w; };
    auto Dw = [&](int c, int l) { return S.Dp + c * sD + D.L[l].off_w; };
    auto gsz = [&](int k) { return (int64_t)B * side_sq(G.L[k].out_log) * G.L[k].nb; };
    auto dsz = [&](int k) { return side_sq(D.L[k].out_log) * D.L[k].cout; };  // per image
    const int gimg = P.img_log - 1;                                    // grid side log2 of the image layers
    const int64_t pcols = side_sq(gimg) * 16 * P.ic;                   // patch / column floats per image
    const DcLayer& Lg = G.L[n];                                        // G's output layer
    const DcLayer& L0 = D.L[0];                                        // D's input layer
    auto im2col = [&](std::vector<DcOp>& o, const std::vector<ColProb>& cs) {
      o.push_back({DC_IM2COL, add_col_op(P, cs, true)});
    };
    auto col2im = [&](std::vector<DcOp>& o, const std::vector<ColProb>& cs) {
      o.push_back({DC_COL2IM, add_col_op(P, cs, false)});
    };
    ops.push_back({DC_SAMPLE, -1});
    // ---- G forward ----
    {
      std::vector<GemmProb> ps;
      for (int c = 0; c < C; ++c)
        ps.push_back(base_prob(P.z + (size_t)c * B * zd, zd, 0, Gw(c, 0), G.L[0].cout, 0, P.gx[0] + c * gsz(0),
                               G.L[0].cout, B, G.L[0].cout, zd));
      gemm(ps);
    }
    auto bn_fwd = [&](int k) {
      const DcLayer& L = G.L[k];
      std::vector<BnProb> bs;
      for (int c = 0; c < C; ++c) {
        const int64_t o = c * sG + L.off_g;
        bs.push_back(bn_prob(P.gx[k] + c * gsz(k), P.gy[k] + c * gsz(k), (int64_t)B * side_sq(L.out_log), L.nb,
                             P.bn_part[k] + c * P.bn_part_cell[k], P.bn_stats[k] + (int64_t)c * 5 * L.nb, S.Gp + o,
                             S.Gm + o, S.Gv + o, S.Glr + c, S.Gt + c, L.act));
      }
      ops.push_back({DC_BN_FWD, add_bn_op(P, bs)});
    };
    bn_fwd(0);
    for (int k = 1; k < n; ++k) {
      const DcLayer& L = G.L[k];
      std::vector<ConvProb> ps;
      for (int c = 0; c < C; ++c)
        for (int r = 0; r < 2; ++r)
          for (int q = 0; q < 2; ++q)
            ps.push_back(convT_phase(P.gy[k - 1] + c * gsz(k - 1), B, L.in_log, L.cin, Gw(c, k), L.cout,
                                     P.gx[k] + c * gsz(k), r, q, EPI_STORE, 0, nullptr));
      conv(ps);
      bn_fwd(k);
    }
    {
      // the image layer: 16-tap columns (one GEMM that reads the map once),
      // then their gather into the fake images with bias and the output act
      std::vector<ConvProb> ps;
      std::vector<ColProb> cs;
      for (int c = 0; c < C; ++c) {
        ps.push_back(convT_cols(P.gy[n - 1] + c * gsz(n - 1), B, Lg.in_log, Lg.cin, Gw(c, n), Lg.cout,
                                P.cols + c * B * pcols));
        cs.push_back(col_prob(P.cols + c * B * pcols, P.Xtr + (size_t)c * 2 * B * xd + (size_t)B * xd, B, P.img_log,
                              P.ic, EPI_BIAS_ACT, Lg.act, S.Gp + c * sG + Lg.off_b, nullptr));
      }
      conv(ps);
      col2im(ops, cs);
    }
    // ---- D forward on [real; fake] ----
    auto d_forward = [&](int rows_img, bool fake_only, float* const* acts, float* logits_base) {
      if (!fake_only) {
        // patches of the 2B real and fake images; the G step reuses the fake half
        std::vector<ColProb> cs;
        for (int c = 0; c < C; ++c)
          cs.push_back(col_prob(P.Xtr + (size_t)c * 2 * B * xd, P.patch + c * 2 * B * pcols, 2 * B, P.img_log, P.ic,
                                0, 0, nullptr, nullptr));
        im2col(ops, cs);
      }
      for (int k = 0; k < n; ++k) {
        const DcLayer& L = D.L[k];
        std::vector<ConvProb> ps;
        for (int c = 0; c < C; ++c) {
          if (k == 0)
            ps.push_back(dense_rows(P.patch + c * 2 * B * pcols + (fake_only ? B * pcols : 0), rows_img, gimg,
                                    16 * P.ic, Dw(c, 0), L.cout, false, acts[0] + c * rows_img * dsz(0), EPI_BIAS_ACT,
                                    L.act, S.Dp + c * sD + L.off_b));
          else
            ps.push_back(conv_fwd(acts[k - 1] + c * rows_img * dsz(k - 1), rows_img, L.in_log, L.cin, Dw(c, k),
                                  L.cout, acts[k] + c * rows_img * dsz(k), EPI_BIAS_ACT, L.act,
                                  S.Dp + c * sD + L.off_b));
        }
        conv(ps);
      }
      std::vector<DotProb> ds;
      for (int c = 0; c < C; ++c) {
        DotProb d;
        memset(&d, 0, sizeof(d));
        d.x = acts[n - 1] + c * rows_img * dsz(n - 1);
        d.w = Dw(c, n);
        d.out = logits_base + (size_t)c * rows_img;
        d.rows = rows_img;
        d.H = Hw;
        d.ld_out = 1;
        ds.push_back(d);
      }
      ops.push_back({DC_DOT, add_dot_op(P, ds)});
    };
    d_forward(2 * B, false, P.dy, P.part_tr);
    ops.push_back({DC_HEAD_D, -1});
    {
      std::vector<GemmProb> ps;
      for (int c = 0; c < C; ++c) {
        const size_t o = c * sD + H.off_w;
        GemmProb p = base_prob(P.dy[n - 1] + c * 2 * B * dsz(n - 1), Hw, 1, P.dlbuf + (size_t)c * 2 * B * 4, 4, 0,
                               S.Dp + o, 1, Hw + 1, 1, 2 * B);
        p.a_rows = Hw;
        p.ones_row = Hw;
        p.m = S.Dm + o;
        p.v = S.Dv + o;
        p.lr = S.Dlr + c;
        p.t = S.Dt + c;
        p.epi = EPI_ADAM;
        p.clip = d_clip;
        if (g->cfg.loss_kind == LIPZ_LOSS_WASSERSTEIN) p.gscale = 1.f / (float)B;  // dL/da stored as exact +-1
        ps.push_back(p);
      }
      gemm(ps);
    }
    // ---- D backward: input gradients beside weight gradients ----
    for (int k = n - 1; k >= 0; --k) {
      const DcLayer& L = D.L[k];
      std::vector<ConvProb> ps;
      if (k >= 1)
        for (int c = 0; c < C; ++c)
          for (int r = 0; r < 2; ++r)
            for (int q = 0; q < 2; ++q)
              ps.push_back(conv_dgrad_phase(P.ddel[k] + c * 2 * B * dsz(k), 2 * B, L.in_log, L.cin, L.cout, Dw(c, k),
                                            P.ddel[k - 1] + c * 2 * B * dsz(k - 1),
                                            P.dy[k - 1] + c * 2 * B * dsz(k - 1), D.L[k - 1].act, r, q));
      for (int c = 0; c < C; ++c) {
        if (k == 0)
          ps.push_back(dense_rows_wgrad(P.patch + c * 2 * B * pcols, 2 * B, gimg, 16 * P.ic, P.ddel[0] + c * 2 * B * dsz(0),
                                        L.cout, P.dpart[0] + c * P.dpart_cell[0], 16 * P.ic + 1, true));
        else
          ps.push_back(conv_wgrad(P.dy[k - 1] + c * 2 * B * dsz(k - 1), 2 * B, L.in_log, L.cin,
                                  P.ddel[k] + c * 2 * B * dsz(k), L.cout, P.dpart[k] + c * P.dpart_cell[k]));
      }
      conv(ps);
    }
    {
      std::vector<RedProb> rs;
      for (int c = 0; c < C; ++c)
        for (int k = 0; k < n; ++k) {
          const DcLayer& L = D.L[k];
          RedProb r;
          memset(&r, 0, sizeof(r));
          r.part = P.dpart[k] + c * P.dpart_cell[k];
          r.n = (int64_t)(16 * L.cin + 1) * L.cout;
          r.split_stride = r.n;
          r.splits = splits_for((2 * B) << (2 * L.out_log));
          const int64_t o = c * sD + L.off_w;
          r.p = S.Dp + o;
          r.m = S.Dm + o;
          r.v = S.Dv + o;
          r.lr = S.Dlr + c;
          r.t = S.Dt + c;
          r.clip = d_clip;
          rs.push_back(r);
        }
      ops.push_back({DC_REDUCE, add_red_op(P, rs)});
    }
    // ---- G step: D on the fakes with the updated D ----
    d_forward(B, true, P.dyg, P.part_g);
    ops.push_back({DC_HEAD_G, -1});
    for (int k = n - 1; k >= 1; --k) {
      const DcLayer& L = D.L[k];
      std::vector<ConvProb> ps;
      for (int c = 0; c < C; ++c)
        for (int r = 0; r < 2; ++r)
          for (int q = 0; q < 2; ++q)
            ps.push_back(conv_dgrad_phase(P.ddelg[k] + c * B * dsz(k), B, L.in_log, L.cin, L.cout, Dw(c, k),
                                          P.ddelg[k - 1] + c * B * dsz(k - 1), P.dyg[k - 1] + c * B * dsz(k - 1),
                                          D.L[k - 1].act, r, q));
      conv(ps);
    }
    {
      // into the image: 16-tap columns with D's input weights transposed, then
      // their gather into dL/d(G's output pre-activation) (times act')
      std::vector<ConvProb> ps;
      std::vector<ColProb> cs;
      for (int c = 0; c < C; ++c) {
        ps.push_back(dense_rows(P.ddelg[0] + c * B * dsz(0), B, gimg, L0.cout, Dw(c, 0), 16 * P.ic, true,
                                P.cols + c * B * pcols, EPI_STORE, 0, nullptr));
        cs.push_back(col_prob(P.cols + c * B * pcols, P.gdimg + (size_t)c * B * xd, B, P.img_log, P.ic, EPI_DACT, Lg.act,
                              nullptr, P.Xtr + (size_t)c * 2 * B * xd + (size_t)B * xd));
      }
      conv(ps);
      col2im(ops, cs);
    }
    // ---- G backward ----
    for (int k = n; k >= 1; --k) {
      const DcLayer& L = G.L[k];
      const float* dout = k == n ? P.gdimg : P.gdz[k];
      const int64_t dout_cell = k == n ? (int64_t)B * xd : gsz(k);
      const int rows_total = 16 * L.cin + L.bias;
      // The input gradient (K = 16 c_out, the deepest tiles) and the weight
      // gradient run as two launches: sharing one launch, the deep tiles of the
      // first layer ran at less than half their separate speed (measured).
      std::vector<ConvProb> pd, ps;
      for (int c = 0; c < C; ++c)
        pd.push_back(convT_dgrad(dout + c * dout_cell, B, L.in_log, L.cin, L.cout, Gw(c, k),
                                 P.gdz[k - 1] + c * gsz(k - 1), P.gy[k - 1] + c * gsz(k - 1), G.L[k - 1].act));
      conv(pd);
      if (k == n) {
        // patches of the image gradient: the 16 taps x c_out columns of every input position
        std::vector<ColProb> cs;
        for (int c = 0; c < C; ++c)
          cs.push_back(col_prob(P.gdimg + (size_t)c * B * xd, P.cols + c * B * pcols, B, P.img_log, P.ic, 0, 0, nullptr,
                                nullptr));
        im2col(ops, cs);
        for (int c = 0; c < C; ++c) {
          ConvProb p = dense_rows_wgrad(P.gy[k - 1] + c * gsz(k - 1), B, L.in_log, L.cin, P.cols + c * B * pcols,
                                        16 * L.cout, P.gpart[k] + c * P.gpart_cell[k], rows_total, false);
          // column n = (tap, c_out) lands on weight row tap * c_in + c_in index
          p.ldc = L.cout;
          p.n_inner = L.cout;
          p.n_tap_stride = L.cin * L.cout;
          p.split_stride = (int64_t)rows_total * L.cout;
          ps.push_back(p);
        }
      } else {
        for (int c = 0; c < C; ++c)
          for (int r = 0; r < 2; ++r)
            for (int q = 0; q < 2; ++q)
              ps.push_back(convT_wgrad_phase(P.gy[k - 1] + c * gsz(k - 1), B, L.in_log, L.cin, dout + c * dout_cell,
                                             L.cout, P.gpart[k] + c * P.gpart_cell[k], rows_total, r, q));
      }
      if (L.bias)
        for (int c = 0; c < C; ++c)
          ps.push_back(convT_bias_grad(dout + c * dout_cell, B, L.out_log, L.cout, P.gpart[k] + c * P.gpart_cell[k],
                                       rows_total, 16 * L.cin));
      conv(ps);
      // batch-norm backward of layer k - 1 (its dz is complete now)
      const DcLayer& Lb = G.L[k - 1];
      std::vector<BnProb> bs;
      for (int c = 0; c < C; ++c) {
        const int64_t o = c * sG + Lb.off_g;
        bs.push_back(bn_prob(P.gx[k - 1] + c * gsz(k - 1), P.gdz[k - 1] + c * gsz(k - 1),
                             (int64_t)B * side_sq(Lb.out_log), Lb.nb, P.bn_part[k - 1] + c * P.bn_part_cell[k - 1],
                             P.bn_stats[k - 1] + (int64_t)c * 5 * Lb.nb, S.Gp + o, S.Gm + o, S.Gv + o, S.Glr + c,
                             S.Gt + c, Lb.act));
      }
      ops.push_back({DC_BN_BWD, add_bn_op(P, bs)});
    }
    {
      // dense layer 0: [z]^T dx0, no bias, Adam
      std::vector<GemmProb> ps;
      for (int c = 0; c < C; ++c) {
        const size_t o = c * sG + G.L[0].off_w;
        GemmProb p = base_prob(P.z + (size_t)c * B * zd, zd, 1, P.gdz[0] + c * gsz(0), G.L[0].cout, 0, S.Gp + o,
                               G.L[0].cout, zd, G.L[0].cout, B);
        p.m = S.Gm + o;
        p.v = S.Gv + o;
        p.lr = S.Glr + c;
        p.t = S.Gt + c;
        p.epi = EPI_ADAM;
        ps.push_back(p);
      }
      gemm(ps);
    }
    {
      std::vector<RedProb> rs;
      for (int c = 0; c < C; ++c)
        for (int k = 1; k <= n; ++k) {
          const DcLayer& L = G.L[k];
          RedProb r;
          memset(&r, 0, sizeof(r));
          r.part = P.gpart[k] + c * P.gpart_cell[k];
          r.n = (int64_t)(16 * L.cin + L.bias) * L.cout;
          r.split_stride = r.n;
          r.splits = splits_for(B << (2 * L.in_log));
          const int64_t o = c * sG + L.off_w;
          r.p = S.Gp + o;
          r.m = S.Gm + o;
          r.v = S.Gv + o;
          r.lr = S.Glr + c;
          r.t = S.Gt + c;
          rs.push_back(r);
        }
      ops.push_back({DC_REDUCE, add_red_op(P, rs)});
    }

    // ---- evaluation: G_i(z_c) for the 5 generator slots, D_j on the 6B images ----
    std::vector<DcOp>& ev = P.eval_ops[par];
    ev.clear();
    const int NIe = 6 * B;
    auto egsz = [&](int k) { return (int64_t)B * side_sq(G.L[k].out_log) * G.L[k].nb; };
    {
      std::vector<GemmProb> ps;
      for (int c = 0; c < C; ++c)
        for (int i = 0; i < 5; ++i) {
          const int own = g->nbr_h[c * 5 + i];
          ps.push_back(base_prob(P.ze + (size_t)c * B * zd, zd, 0, Gw(own, 0), G.L[0].cout, 0,
                                 P.gex[0] + (c * 5 + i) * egsz(0), G.L[0].cout, B, G.L[0].cout, zd));
        }
      ev.push_back({DC_GEMM, add_phase(g, ps)});
    }
    auto ebn = [&](int k) {
      const DcLayer& L = G.L[k];
      const int64_t rows = (int64_t)B * side_sq(L.out_log);
      const int64_t pc = ((rows + BN_CHUNK - 1) / BN_CHUNK) * 2 * L.nb;
      std::vector<BnProb> bs;
      for (int c = 0; c < C; ++c)
        for (int i = 0; i < 5; ++i) {
          const int own = g->nbr_h[c * 5 + i];
          float* x = P.gex[k] + (c * 5 + i) * egsz(k);
          bs.push_back(bn_prob(x, x, rows, L.nb, P.bne_part[k] + (c * 5 + i) * pc,
                               P.bne_stats[k] + (int64_t)(c * 5 + i) * 5 * L.nb, S.Gp + own * sG + L.off_g, nullptr,
                               nullptr, nullptr, nullptr, L.act));
        }
      ev.push_back({DC_BN_FWD, add_bn_op(P, bs)});
    };
    ebn(0);
    for (int k = 1; k < n; ++k) {
      const DcLayer& L = G.L[k];
      std::vector<ConvProb> ps;
      for (int c = 0; c < C; ++c)
        for (int i = 0; i < 5; ++i) {
          const int own = g->nbr_h[c * 5 + i];
          for (int r = 0; r < 2; ++r)
            for (int q = 0; q < 2; ++q)
              ps.push_back(convT_phase(P.gex[k - 1] + (c * 5 + i) * egsz(k - 1), B, L.in_log, L.cin, Gw(own, k), L.cout,
                                       P.gex[k] + (c * 5 + i) * egsz(k), r, q, EPI_STORE, 0, nullptr));
        }
      ev.push_back({DC_CONV, add_conv_phase(P, ps)});
      ebn(k);
    }
    {
      std::vector<ConvProb> ps;
      std::vector<ColProb> cs;
      for (int c = 0; c < C; ++c)
        for (int i = 0; i < 5; ++i) {
          const int own = g->nbr_h[c * 5 + i];
          float* cols = P.ecols + (c * 5 + i) * B * pcols;
          ps.push_back(convT_cols(P.gex[n - 1] + (c * 5 + i) * egsz(n - 1), B, Lg.in_log, Lg.cin, Gw(own, n), Lg.cout,
                                  cols));
          cs.push_back(col_prob(cols, P.Xe + (size_t)c * 6 * B * xd + (size_t)(1 + i) * B * xd, B, P.img_log, P.ic,
                                EPI_BIAS_ACT, Lg.act, S.Gp + own * sG + Lg.off_b, nullptr));
        }
      ev.push_back({DC_CONV, add_conv_phase(P, ps)});
      col2im(ev, cs);
    }
    {
      // patches of each cell's 6B images, shared by its 5 discriminator slots
      std::vector<ColProb> cs;
      for (int c = 0; c < C; ++c)
        cs.push_back(col_prob(P.Xe + (size_t)c * 6 * B * xd, P.epatch + c * NIe * pcols, NIe, P.img_log, P.ic, 0, 0,
                              nullptr, nullptr));
      im2col(ev, cs);
    }
    for (int k = 0; k < n; ++k) {
      const DcLayer& L = D.L[k];
      std::vector<ConvProb> ps;
      for (int c = 0; c < C; ++c)
        for (int j = 0; j < 5; ++j) {
          const int own = g->nbr_h[c * 5 + j];
          float* out = P.dey[k & 1] + (c * 5 + j) * NIe * dsz(k);
          if (k == 0)
            ps.push_back(dense_rows(P.epatch + c * NIe * pcols, NIe, gimg, 16 * P.ic, Dw(own, 0), L.cout, false, out,
                                    EPI_BIAS_ACT, L.act, S.Dp + own * sD + L.off_b));
          else
            ps.push_back(conv_fwd(P.dey[(k - 1) & 1] + (c * 5 + j) * NIe * dsz(k - 1), NIe, L.in_log, L.cin, Dw(own, k),
                                  L.cout, out, EPI_BIAS_ACT, L.act, S.Dp + own * sD + L.off_b));
        }
      ev.push_back({DC_CONV, add_conv_phase(P, ps)});
    }
    {
      std::vector<DotProb> ds;
      for (int c = 0; c < C; ++c)
        for (int j = 0; j < 5; ++j) {
          const int own = g->nbr_h[c * 5 + j];
          DotProb d;
          memset(&d, 0, sizeof(d));
          d.x = P.dey[(n - 1) & 1] + (c * 5 + j) * NIe * dsz(n - 1);
          d.w = Dw(own, n);
          d.out = P.part_e + (size_t)(c * 5 + j) * NIe;
          d.rows = NIe;
          d.H = Hw;
          d.ld_out = 1;
          ds.push_back(d);
        }
      ev.push_back({DC_DOT, add_dot_op(P, ds)});
    }
  }
}

hipError_t dc_upload_tables(lipz_grid* g, hipStream_t s) {
  DcPlan& P = *g->dc;
  hipError_t e = hipSuccess;
  if (!P.conv_h.empty())
    e = hipMemcpyAsync(P.conv_d, P.conv_h.data(), P.conv_h.size() * sizeof(ConvProb), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !P.bn_h.empty())
    e = hipMemcpyAsync(P.bn_d, P.bn_h.data(), P.bn_h.size() * sizeof(BnProb), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !P.red_h.empty())
    e = hipMemcpyAsync(P.red_d, P.red_h.data(), P.red_h.size() * sizeof(RedProb), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !P.col_h.empty())
    e = hipMemcpyAsync(P.col_d, P.col_h.data(), P.col_h.size() * sizeof(ColProb), hipMemcpyHostToDevice, s);
  if (e == hipSuccess && !P.dot_h.empty())
    e = hipMemcpyAsync(P.dot_d, P.dot_h.data(), P.dot_h.size() * sizeof(DotProb), hipMemcpyHostToDevice, s);
  return e;
}

hipError_t dc_init_params(lipz_grid* g, const StateBuf& S, hipStream_t s) {
  DcPlan& P = *g->dc;
  auto layout = [](const DcNet& N) {
    ConvInitLayout L;
    memset(&L, 0, sizeof(L));
    L.n = N.nl;
    for (int l = 0; l < N.nl; ++l) {
      L.off_w[l] = N.L[l].off_w;
      L.n_w[l] = N.L[l].n_w;
      L.off_b[l] = N.L[l].off_b;
      L.n_b[l] = N.L[l].bias ? N.L[l].cout : 0;
      L.off_g[l] = N.L[l].off_g;
      L.n_g[l] = N.L[l].nb;
    }
    return L;
  };
  hipError_t e = launch_init_conv_params(S.Gp, g->G.stride, P.G.P, g->C, layout(P.G), g->key, LIPZ_TAG_INIT_G, s);
  if (e == hipSuccess)
    e = launch_init_conv_params(S.Dp, g->D.stride, P.D.P, g->C, layout(P.D), g->key, LIPZ_TAG_INIT_D, s);
  return e;
}

namespace {

hipError_t run_conv_phase(lipz_grid* g, int idx, hipStream_t s) {
  DcPlan& P = *g->dc;
  const ConvPhase& ph = P.cph[idx];
  hipEvent_t e0, e1;
  hipError_t e = timing_events(g, &e0, &e1);
  if (e != hipSuccess) return e;
  e = launch_conv_grouped(P.conv_d + ph.first, ph.grp, ph.tiles, g->slope, s, e0, e1);
  timing_record(g, e0, e1, ph.flops, ph.bytes);
  return e;
}

hipError_t run_op(lipz_grid* g, const DcOp& op, int step_local, hipStream_t s) {
  DcPlan& P = *g->dc;
  switch (op.kind) {
    case DC_GEMM: return run_gemm_phase(g, op.idx, step_local, s);
    case DC_CONV: return run_conv_phase(g, op.idx, s);
    case DC_BN_FWD: {
      const BnOp& b = P.bnops[op.idx];
      hipError_t e = launch_bn_stats(P.bn_d + b.first, b.count, b.blocks, 1e-5f, s);
      if (e == hipSuccess) e = launch_bn_apply(P.bn_d + b.first, b.count, b.max_elems, g->slope, s);
      return e;
    }
    case DC_BN_BWD: {
      const BnOp& b = P.bnops[op.idx];
      return launch_bn_backward(P.bn_d + b.first, b.count, b.blocks, b.max_elems, step_local, g->ac, s);
    }
    case DC_REDUCE: {
      const RedOp& r = P.redops[op.idx];
      return launch_reduce_adam(P.red_d + r.first, r.count, r.max_n, step_local, g->ac, s);
    }
    case DC_IM2COL: {
      const ColOp& c = P.colops[op.idx];
      return launch_im2col(P.col_d + c.first, c.count, c.max_work, s);
    }
    case DC_COL2IM: {
      const ColOp& c = P.colops[op.idx];
      return launch_col2im(P.col_d + c.first, c.count, c.max_work, g->slope, s);
    }
    case DC_DOT: {
      const DotOp& d = P.dotops[op.idx];
      return launch_dot_rows(P.dot_d + d.first, d.count, d.rows, s);
    }
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

lipz_status dc_eval(lipz_grid* g, int gen) {
  DcPlan& P = *g->dc;
  hipStream_t s = g->stream;
  const int C = g->C, B = g->B;
  lipz_status st;
  hipError_t e = launch_sample(g->data, g->N, g->xd, g->zd, B, 0, C, g->key, (uint32_t)gen, 0, P.Xe,
                               (int64_t)6 * B * g->xd, P.ze, (int64_t)B * g->zd, s);
  if ((st = check_hip(g, e, "eval sample"))) return st;
  for (const DcOp& op : P.eval_ops[g->cur])
    if ((st = check_hip(g, run_op(g, op, 0, s), "eval forward"))) return st;
  EvalHeadArgs ha;
  ha.part = P.part_e;
  ha.tn = 1;
  ha.L = g->L;
  ha.Lg = g->Lg;
  ha.B = B;
  ha.C = C;
  ha.nn = LIPZ_SLOTS;
  ha.rmean = nullptr;
  ha.loss_kind = g->cfg.loss_kind;
  return check_hip(g, launch_head_eval(ha, s), "eval head");
}

lipz_status dc_train(lipz_grid* g, int gen, int step0, int n_steps, float* d_losses) {
  DcPlan& P = *g->dc;
  hipStream_t s = g->stream;
  const int C = g->C, B = g->B, n = P.n;
  const StateBuf& S = g->st[g->cur];
  const DcLayer& H = P.D.L[n];
  HeadArgs hd;
  memset(&hd, 0, sizeof(hd));
  hd.part = P.part_tr;
  hd.tn = 1;
  hd.act = P.dy[n - 1];
  hd.act_cell_stride = (int64_t)2 * B * H.cin;
  hd.delta = P.ddel[n - 1];
  hd.w = S.Dp + H.off_w;
  hd.p_stride = g->D.stride;
  hd.dlbuf = P.dlbuf;
  hd.H = H.cin;
  hd.B = B;
  hd.c0 = 0;
  hd.C = C;
  hd.hidden_act = P.D.L[n - 1].act;
  hd.slope = g->slope;
  hd.loss_kind = g->cfg.loss_kind;
  HeadArgs hg = hd;
  hg.part = P.part_g;
  hg.act = P.dyg[n - 1];
  hg.act_cell_stride = (int64_t)B * H.cin;
  hg.delta = P.ddelg[n - 1];
  hg.dlbuf = nullptr;
  lipz_status st;
  for (int k = 0; k < n_steps; ++k) {
    const int step = step0 + k;
    hd.losses = hg.losses = d_losses ? d_losses + (size_t)k * C * 2 : nullptr;
    for (const DcOp& op : P.train_ops[g->cur]) {
      hipError_t e;
      switch (op.kind) {
        case DC_SAMPLE:
          e = launch_sample(g->data, g->N, g->xd, g->zd, B, 0, C, g->key, (uint32_t)gen, (uint32_t)(step + 1), P.Xtr,
                            (int64_t)2 * B * g->xd, P.z, (int64_t)B * g->zd, s);
          break;
        case DC_HEAD_D: e = launch_head_d(hd, s); break;
        case DC_HEAD_G: e = launch_head_g(hg, s); break;
        default: e = run_op(g, op, k, s); break;
      }
      if ((st = check_hip(g, e, "train step"))) return st;
    }
  }
  return LIPZ_OK;
}

lipz_status dc_param_layout(const lipz_grid* g, int role, int64_t* h_offsets, int32_t* h_n) {
  const DcNet& N = role == LIPZ_ROLE_G ? g->dc->G : g->dc->D;
  *h_n = N.nl;
  if (h_offsets)
    for (int l = 0; l < N.nl; ++l) {
      const int taps = N.L[l].kind == LK_DENSE ? 1 : 16;
      h_offsets[3 * l + 0] = N.L[l].off_w;
      h_offsets[3 * l + 1] = (int64_t)taps * N.L[l].cin;
      h_offsets[3 * l + 2] = N.L[l].cout;
    }
  return LIPZ_OK;
}

// ---------------------------------------------------------------------------
// Host-side bounds check of every descriptor of the plan (no GPU needed): the
// extreme addresses each kernel can touch, computed with the kernels' own
// index formulas, must lie inside one of the regions [lo[i], hi[i]).
// ---------------------------------------------------------------------------
namespace {

struct Checker {
  const char* const* lo;
  const char* const* hi;
  int nreg;
  int bad = 0;
  std::string* msg;
  void range(const void* p, int64_t first_float, int64_t last_float, const char* what, int idx) {
    if (!p) {
      fail_(what, idx, "null pointer");
      return;
    }
    const char* a = (const char*)p + 4 * first_float;
    const char* b = (const char*)p + 4 * (last_float + 1);
    for (int i = 0; i < nreg; ++i)
      if (a >= lo[i] && b <= hi[i] && first_float >= 0) return;
    fail_(what, idx, "outside the workspace");
  }
  void fail_(const char* what, int idx, const char* why) {
    ++bad;
    if (msg && msg->size() < 2000) *msg += std::string(what) + " #" + std::to_string(idx) + ": " + why + "; ";
  }
};

int64_t map_last(const PosMap& m, int NI, int gh, int gw, int N) {
  const int64_t y = (int64_t)((1 << gh) - 1) * m.sy + m.y0, x = (int64_t)((1 << gw) - 1) * m.sx + m.x0;
  return ((((int64_t)(NI - 1) << m.h_log) + y) << m.w_log) * m.ld + x * m.ld + N - 1;
}
int64_t map_first(const PosMap& m) { return (((int64_t)m.y0 << m.w_log) + m.x0) * m.ld; }

// True when column descriptor i belongs to an im2col op.
bool col_is_im2col(const DcPlan& P, int i) {
  for (int par = 0; par < 2; ++par)
    for (const auto* ops : {&P.train_ops[par], &P.eval_ops[par]})
      for (const DcOp& op : *ops)
        if (op.kind == DC_IM2COL || op.kind == DC_COL2IM) {
          const ColOp& c = P.colops[op.idx];
          if (i >= c.first && i < c.first + c.count) return op.kind == DC_IM2COL;
        }
  return false;
}

}  // namespace

int dc_check_bounds(const lipz_grid* g, const char* const* lo, const char* const* hi, int nreg, std::string* msg) {
  const DcPlan& P = *g->dc;
  Checker ck{lo, hi, nreg, 0, msg};
  for (size_t i = 0; i < P.conv_h.size(); ++i) {
    const ConvProb& p = P.conv_h[i];
    const int idx = (int)i;
    const int NI = p.M >> (p.gh_log + p.gw_log);
    if (p.s_bytes == 0 || (p.mode == CONV_FWD && p.w_bytes == 0) || (p.mode == CONV_WG && p.p_bytes == 0))
      ck.fail_("conv", idx, "operand extent does not fit 32 bits");
    ck.range(p.S, 0, p.s_bytes / 4 - 1, "conv S", idx);
    if (p.mode == CONV_FWD) {
      if (NI << (p.gh_log + p.gw_log) != p.M) ck.fail_("conv", idx, "M is not a whole number of images");
      ck.range(p.W, 0, p.w_bytes / 4 - 1, "conv W", idx);
      // largest weight offset the kernel forms
      int64_t wmax = 0;
      for (int t = 0; t < p.taps; ++t) {
        const int a = t >> p.tw_log, b = t & ((1 << p.tw_log) - 1);
        const int64_t wt = (int64_t)(a * p.khs + p.kh0) * p.kw_full + (b * p.khs + p.kw0);
        if (wt < 0) ck.fail_("conv", idx, "negative weight tap");
        const int64_t ncol = p.n_inner ? (int64_t)(p.N / p.n_inner - 1) * p.n_tap_stride + (int64_t)(p.n_inner - 1) * p.wsn
                                       : (int64_t)(p.N - 1) * p.wsn;
        if (p.n_inner && (p.N % p.n_inner || !p.gen)) ck.fail_("conv", idx, "column taps need element-wise loads");
        const int64_t o = wt * p.cs * p.N + (int64_t)(p.cs - 1) * p.wsc + ncol;
        if (o > wmax) wmax = o;
      }
      if (wmax >= (int64_t)p.w_bytes / 4) ck.fail_("conv", idx, "weights beyond their extent");
      // largest source position
      const int64_t smax = (((int64_t)NI << p.smap.h_log) << p.smap.w_log) * p.smap.ld;
      if (smax > (int64_t)p.s_bytes / 4) ck.fail_("conv", idx, "source images beyond their extent");
      if (map_first(p.omap) < 0) ck.fail_("conv", idx, "negative output offset");
      const int64_t last = map_last(p.omap, NI, p.gh_log, p.gw_log, p.N);
      ck.range(p.C, map_first(p.omap), last, "conv C", idx);
      if (p.epi == EPI_DACT) ck.range(p.aux, map_first(p.omap), last, "conv aux", idx);
      if (p.epi == EPI_BIAS_ACT && p.bias) ck.range(p.bias, 0, p.N - 1, "conv bias", idx);
    } else {
      const int NIk = p.K >> (p.gh_log + p.gw_log);
      if (NIk << (p.gh_log + p.gw_log) != p.K) ck.fail_("conv", idx, "K is not a whole number of images");
      ck.range(p.P, 0, p.p_bytes / 4 - 1, "conv P", idx);
      if (map_last(p.pmap, NIk, p.gh_log, p.gw_log, p.N) >= (int64_t)p.p_bytes / 4)
        ck.fail_("conv", idx, "output-gradient positions beyond their extent");
      int64_t crow_max = p.ones_row >= 0 ? p.brow : -1;
      for (int t = 0; t < p.taps; ++t) {
        const int a = t >> p.tw_log, b = t & ((1 << p.tw_log) - 1);
        const int64_t wt = (int64_t)(a * p.khs + p.kh0) * p.kw_full + (b * p.khs + p.kw0);
        const int64_t r = wt * p.cs + p.cs - 1;
        if (wt < 0) ck.fail_("conv", idx, "negative weight tap");
        if (r > crow_max) crow_max = r;
      }
      const int64_t col_last = p.n_inner ? (int64_t)(p.N / p.n_inner - 1) * p.n_tap_stride + p.n_inner - 1 : p.N - 1;
      if (p.n_inner && (p.N % p.n_inner || p.ldc < p.n_inner)) ck.fail_("conv", idx, "bad column taps");
      if (crow_max * p.ldc + col_last >= p.split_stride) ck.fail_("conv", idx, "partial rows overlap the next split");
      if (p.splits < 1 || (int64_t)(p.splits - 1) * p.ksplit >= p.K) ck.fail_("conv", idx, "bad split count");
      ck.range(p.C, 0, (int64_t)(p.splits - 1) * p.split_stride + crow_max * p.ldc + col_last, "conv partial", idx);
    }
  }
  for (size_t i = 0; i < P.bn_h.size(); ++i) {
    const BnProb& b = P.bn_h[i];
    const int idx = (int)i;
    const int64_t n = b.rows * b.ch;
    const int64_t chunks = (b.rows + BN_CHUNK - 1) / BN_CHUNK;
    if (b.ch % 4) ck.fail_("bn", idx, "channels not a multiple of 4");
    ck.range(b.x, 0, n - 1, "bn x", idx);
    ck.range(b.y, 0, n - 1, "bn y", idx);
    ck.range(b.part, 0, chunks * 2 * b.ch - 1, "bn part", idx);
    ck.range(b.stats, 0, 5 * b.ch - 1, "bn stats", idx);
    ck.range(b.gamma, 0, 2 * b.ch - 1, "bn gamma", idx);
    if (b.gm) ck.range(b.gm, 0, 2 * b.ch - 1, "bn adam m", idx);
    if (b.gv) ck.range(b.gv, 0, 2 * b.ch - 1, "bn adam v", idx);
  }
  for (size_t i = 0; i < P.red_h.size(); ++i) {
    const RedProb& r = P.red_h[i];
    const int idx = (int)i;
    ck.range(r.part, 0, (int64_t)(r.splits - 1) * r.split_stride + r.n - 1, "reduce part", idx);
    ck.range(r.p, 0, r.n - 1, "reduce p", idx);
    ck.range(r.m, 0, r.n - 1, "reduce m", idx);
    ck.range(r.v, 0, r.n - 1, "reduce v", idx);
    ck.range(r.lr, 0, 0, "reduce lr", idx);
    ck.range(r.t, 0, 0, "reduce t", idx);
  }
  for (size_t i = 0; i < P.col_h.size(); ++i) {
    const ColProb& c = P.col_h[i];
    const int idx = (int)i;
    const int64_t map = ((int64_t)c.n_img << (2 * c.h_log)) * c.ch;
    const bool to_cols = col_is_im2col(P, (int)i);
    ck.range(c.src, 0, (to_cols ? map : 4 * map) - 1, "col src", idx);
    ck.range(c.dst, 0, (to_cols ? 4 * map : map) - 1, "col dst", idx);
    if (!to_cols && c.epi == EPI_BIAS_ACT && c.bias) ck.range(c.bias, 0, c.ch - 1, "col bias", idx);
    if (!to_cols && c.epi == EPI_DACT) ck.range(c.aux, 0, map - 1, "col aux", idx);
  }
  for (size_t i = 0; i < P.dot_h.size(); ++i) {
    const DotProb& d = P.dot_h[i];
    const int idx = (int)i;
    ck.range(d.x, 0, (int64_t)d.rows * d.H - 1, "dot x", idx);
    ck.range(d.w, 0, d.H, "dot w", idx);
    ck.range(d.out, 0, (int64_t)(d.rows - 1) * d.ld_out, "dot out", idx);
  }
  return ck.bad;
}

}  // namespace lipz
