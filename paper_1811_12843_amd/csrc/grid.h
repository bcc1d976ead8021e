// The grid handle and the host-side helpers shared by the runtime files of
// liblipz.so (api.hip: configuration, workspace, MLP plans and the C ABI;
// dcgan.hip: the plans of the convolutional networks).
#pragma once

#include <string>
#include <vector>

#include "lipz_internal.h"

namespace lipz {

constexpr size_t kAlign = 256;
#define LIPZ_MAX_GROUPS 8
#ifndef LIPZ_CELL_GROUPS
#define LIPZ_CELL_GROUPS 0  // 0: choose from the grid size
#endif

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Bump allocator over the caller's workspace.  With base == nullptr it only
// measures, so sizing and carving share one code path.
struct Carver {
  char* base;
  size_t off = 0;
  template <class T>
  T* take(size_t count) {
    off = align_up(off, kAlign);
    T* p = reinterpret_cast<T*>(base + off);
    off += count * sizeof(T);
    return p;
  }
};

struct Net {
  int nl = 0;            // layers, the last one is the output layer
  int64_t off[LIPZ_MAX_HIDDEN + 1];
  int fi[LIPZ_MAX_HIDDEN + 1], fo[LIPZ_MAX_HIDDEN + 1];
  int act[LIPZ_MAX_HIDDEN + 1];
  int64_t P = 0, stride = 0;
  NetLayers layers() const {
    NetLayers L{};
    L.n = nl;
    for (int l = 0; l < nl; ++l) {
      L.off[l] = off[l];
      L.fan_in[l] = fi[l];
      L.fan_out[l] = fo[l];
    }
    return L;
  }
};

struct StateBuf {
  char* base;
  float *Gp, *Gm, *Gv, *Dp, *Dm, *Dv;
  int32_t *Gt, *Dt;
  float *Glr, *Dlr, *w;
};

struct Phase {
  int first = 0, count = 0, tiles = 0, tile_rows = 64;
  bool fast = true;             // every problem eligible for the aligned kernels
  int kernel = GEMM_K_FAST;     // GemmKernel variant
  GemmGroups grp;
  double flops = 0.0;
  double bytes = 0.0;  // algorithmic: each operand read once, each output written once
};

// A training-step op: a GEMM phase, or a kernel of the step; for the NES ops
// `phase` holds the role (LIPZ_ROLE_G / LIPZ_ROLE_D).
enum OpKind { OP_SAMPLE, OP_GEMM, OP_HEAD_D, OP_HEAD_G, OP_LOSS_D, OP_LOSS_G, OP_NES_PERTURB, OP_NES_HEAD,
              OP_NES_UPDATE };
struct Op {
  OpKind kind;
  int phase;
  int sample_next = 0;  // OP_GEMM: the launch also draws the next step's minibatch
};

struct DcPlan;  // the convolutional networks' plan (dcgan.hip)

}  // namespace lipz

// The opaque handle of include/lipz.h.
struct lipz_grid {
  typedef lipz::Net Net;
  typedef lipz::StateBuf StateBuf;
  typedef lipz::Op Op;
  typedef lipz::Phase Phase;
  typedef lipz::AdamConsts AdamConsts;
  typedef lipz::GemmProb GemmProb;
  lipz_config cfg;
  int C = 0, B = 0, zd = 0, xd = 0, S = 0, F = 0;
  // sub-populations: s individuals per role and cell, U = C s individuals
  // (training units), nn = 5 s individuals per neighbourhood
  int s = 1, U = 0, nn = LIPZ_SLOTS;
  Net G, D;
  hipStream_t stream = nullptr;
  const float* data = nullptr;
  int64_t N = 0;
  uint2 key;
  float slope = 0.f;
  AdamConsts ac;
  // GEMM launches store write-through (device scope) when the grid's state
  // (parameters and Adam moments of every individual) is at most 128 MB,
  // half the 256 MB last-level cache: measured faster for such grids (4x4
  // and 3x3 MNIST-shaped), slower for larger ones (4x4 with two individuals
  // per cell, 8x8), which store write-back.
  bool gemm_wt = false;

  StateBuf st[2];
  int cur = 0;
  size_t state_bytes = 0;
  int64_t state_off[12];
  std::vector<int32_t> nbr_h;

  int32_t *nbr = nullptr, *sel = nullptr, *flags = nullptr;
  float *L = nullptr, *Lg = nullptr, *fit_g = nullptr, *fit_d = nullptr;
  // training buffers
  float *z = nullptr, *Xtr = nullptr;
  // The gradient trainer draws step k + 1's minibatch inside step k's first
  // launch: steps alternate between (z, Xtr) (even) and (z_alt, Xtr_alt) (odd).
  bool fused_sample = false;
  float *z_alt = nullptr, *Xtr_alt = nullptr;
  float *h[LIPZ_MAX_HIDDEN] = {}, *a[LIPZ_MAX_HIDDEN] = {}, *dD[LIPZ_MAX_HIDDEN] = {};
  float *ag[LIPZ_MAX_HIDDEN] = {}, *dDg[LIPZ_MAX_HIDDEN] = {}, *dG[LIPZ_MAX_HIDDEN + 1] = {};
  float *part_tr = nullptr, *part_g = nullptr, *part_e = nullptr;  // partial logits
  float* dlbuf = nullptr;  // D-step dL/d(logit) [C][2B][4]
  // The loss head folded into the GEMM launches (reading 8's training step
  // with at least two hidden layers in D): aS [U][2B][aS_ld] holds dL/da-scaled
  // activations of the layer below D's last hidden layer, then dL/da.
  bool fused_head = false;
  float* aS = nullptr;
  int aS_ld = 0;
  // ... and, when D's last hidden layer is at most as wide as the one below
  // it, the output layer's weight gradient in per-row-tile column sums
  // hpart [U][hp_rows][hp_ld] written by the input-gradient launch
  float* hpart = nullptr;
  int hp_rows = 0, hp_ld = 0;
  int tn = 1;  // column tiles of D's last hidden layer
  // evaluation buffers
  float *ze = nullptr, *Xe = nullptr;
  float *he[LIPZ_MAX_HIDDEN] = {}, *ae[LIPZ_MAX_HIDDEN] = {};
  // mixture buffers
  float *zeta = nullptr, *xm = nullptr, *fm = nullptr;
  double *mu_k = nullptr, *s2_k = nullptr, *mom_part = nullptr;  // generator feature moments, fp64
  float *hm[LIPZ_MAX_HIDDEN] = {};
  float *P = nullptr, *realfeat = nullptr;
  double *mu_r = nullptr, *sd_r = nullptr;  // dataset feature mean and standard deviation, fp64

  GemmProb* probs_d = nullptr;
  std::vector<GemmProb> probs_h;
  std::vector<Phase> phases;
  // Cells are split into groups whose training phases run on separate
  // streams (group 0 on the caller's stream), so that one group's
  // latency-bound launches overlap another group's work.
  int n_groups = 1;
  int group_c0[LIPZ_MAX_GROUPS + 1] = {};
  hipStream_t gstream[LIPZ_MAX_GROUPS] = {};
  hipEvent_t fork_ev = nullptr, join_ev[LIPZ_MAX_GROUPS] = {};
  std::vector<Op> train_ops[2][LIPZ_MAX_GROUPS];
  std::vector<Op> train_ops_odd[2][LIPZ_MAX_GROUPS];  // odd steps when fused_sample
  // Row bands of lipz_run_generations (config bands >= 2): band b holds cells
  // band_c0[b] .. band_c0[b + 1] - 1 (whole rows); the training groups are
  // the bands' individuals, and each band has its own evaluation and
  // re-evaluation plans and a readiness event
  int n_bands = 0;
  int band_c0[LIPZ_MAX_GROUPS + 1] = {};
  uint32_t band_wait[LIPZ_MAX_GROUPS] = {};  // bit b': band b' holds a neighbour row of the band
  std::vector<int> band_eval_phases[2][LIPZ_MAX_GROUPS], band_elite_phases[2][LIPZ_MAX_GROUPS];
  std::vector<int> band_mix_phases[2][LIPZ_MAX_GROUPS];  // on the band's own copy of the mixture latents
  hipEvent_t band_ev[LIPZ_MAX_GROUPS] = {};   // the band finished its generation
  hipEvent_t mom_ev[LIPZ_MAX_GROUPS] = {};    // the band's generator moments of the generation are ready
  std::vector<int> eval_phases[2], mix_phases[2];
  int real_phase = -1;

  // post-training re-evaluation and elitist replacement
  float *rmean = nullptr;                                   // [C][nn] real-row term means of the evaluation
  float *he2[LIPZ_MAX_HIDDEN] = {}, *xe2 = nullptr;          // trained G' on the evaluation latents [C][s][B]
  float *ae2[LIPZ_MAX_HIDDEN] = {}, *part_e2 = nullptr;      // previous D_j on those rows [C][nn][sB]
  float *ae3[LIPZ_MAX_HIDDEN] = {}, *part_e3 = nullptr;      // trained D'_j on the evaluation rows [C][s][(1+nn)B]
  float *fit2_g = nullptr, *fit2_d = nullptr;                // [C][s]
  float *el_L2 = nullptr, *el_Lg2 = nullptr, *el_M3 = nullptr; // [C][s][nn] x2, [C][1 + nn][s]
  int32_t* esrc = nullptr;                                   // [U][2]
  std::vector<int> elite_phases[2];
  int elite_state = 0;  // 1: evaluated; 2: selected after that evaluation (training allowed)
  int32_t elite_gen = -1;

  bool plan_ok = true;  // false if a phase exceeded the launch descriptor's shape groups
  bool fitness_valid = false;
  lipz_status sticky = LIPZ_OK;
  std::string last_err;

  bool timing = false;
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev_live;
  std::vector<double> ev_flops, ev_bytes;
  double gemm_ms = 0.0, gemm_flops = 0.0, gemm_bytes = 0.0;
  int64_t gemm_launches = 0;

  lipz::DcPlan* dc = nullptr;  // set for LIPZ_NET_DCGAN
  int static_dev = -1;         // lipz_grid_create_static: the device whose static workspace it holds

  // NES trainer: Q = 2 nes_pairs + 1 parameter sets per role and cell (the
  // + and - perturbations, then the unperturbed parameters)
  int nes_q = 0;
  float *nes_pd = nullptr, *nes_pg = nullptr;                         // [C][2n][stride]
  float* nes_eps = nullptr;                                           // [C][n][nes_eps_stride]
  int64_t nes_eps_stride = 0;
  float *nes_aq[LIPZ_MAX_HIDDEN] = {}, *nes_part_d = nullptr;         // D per set on the 2B rows
  float *nes_hq[LIPZ_MAX_HIDDEN] = {}, *nes_xq = nullptr;             // G per set
  float *nes_agq[LIPZ_MAX_HIDDEN] = {}, *nes_part_g = nullptr;        // D on the Q B generated rows
  float *nes_fd = nullptr, *nes_fg = nullptr;                         // losses per set [C][Q]
  std::vector<Op> nes_ops[2];
  std::vector<Op> nes_band_ops[2][LIPZ_MAX_GROUPS];  // the same per row band
};

namespace lipz {

// api.hip
lipz_status create_grid(const lipz_config* cfg, void* d_workspace, size_t workspace_bytes,
                        const float* d_dataset, int64_t n_samples, void* hip_stream, lipz_grid** out);
lipz_status fail(lipz_grid* g, lipz_status s, const std::string& msg);
lipz_status check_hip(lipz_grid* g, hipError_t e, const char* what);
void carve_state(lipz_grid* g, Carver& cv, char* base);
GemmProb base_prob(const float* A, int lda, int a_trans, const float* Bm, int ldb, int b_trans, float* C, int ldc,
                   int M, int N, int K);
int add_phase(lipz_grid* g, const std::vector<GemmProb>& ps);
hipError_t run_gemm_phase(lipz_grid* g, int phase, int step_local, hipStream_t stream,
                          const SampleJob* job = nullptr);
hipError_t timing_events(lipz_grid* g, hipEvent_t* e0, hipEvent_t* e1);
void timing_record(lipz_grid* g, hipEvent_t e0, hipEvent_t e1, double flops, double bytes);
int ceil_div(int a, int b);

// dcgan.hip
std::string dc_validate(const lipz_config* c, Net* Gn, Net* Dn);
DcPlan* dc_new(const lipz_config* c);
void dc_delete(DcPlan* p);
void dc_carve(lipz_grid* g, Carver& cv);
void dc_build(lipz_grid* g);
bool dc_plan_ok(const DcPlan* p);
void dc_carve_tables(lipz_grid* g, Carver& cv);
hipError_t dc_upload_tables(lipz_grid* g, hipStream_t s);
hipError_t dc_init_params(lipz_grid* g, const StateBuf& S, hipStream_t s);
lipz_status dc_eval(lipz_grid* g, int gen);
lipz_status dc_train(lipz_grid* g, int gen, int step0, int n_steps, float* d_losses);
lipz_status dc_param_layout(const lipz_grid* g, int role, int64_t* h_offsets, int32_t* h_n);
int dc_check_bounds(const lipz_grid* g, const char* const* lo, const char* const* hi, int nreg, std::string* msg);

}  // namespace lipz
