/*
 * lipz.h -- C ABI of liblipz.so: one generation of spatial coevolutionary GAN
 * training (Lipizzaner, arXiv 1811.12843) with every cell of the toroidal grid
 * batched on one AMD Instinct MI355X (gfx950).
 *
 * The method (paper Section 3, "Coevolutionary GAN Training", steps 1-5):
 *   1. every cell holds one generator (params u, learning rate delta) and one
 *      discriminator (params v, learning rate gamma), randomly initialised
 *                                                       -> lipz_grid_create
 *   2. each generator of a cell's 5-cell von Neumann neighbourhood (Section 2)
 *      is evaluated against each discriminator of it; the losses of a
 *      discriminator are averaged and those of a generator negative-averaged
 *      to give fitness                                  -> lipz_eval_neighborhoods
 *   3. tournament selection of one generator and one discriminator per
 *      neighbourhood, Gaussian mutation of their learning rates
 *                                                       -> lipz_select_replace
 *      and gradient-based training of the selected pair -> lipz_train_step
 *   4. the generator-mixture weights of each neighbourhood evolve by a
 *      (1+1)-ES                                          -> lipz_mixture_update
 *   5. go to 2.
 * Hyper-parameter defaults follow the paper's experiment settings table
 * (population size 1 per cell, tournament size 2, Adam, learning rate 2e-4,
 * mutation rate 1e-4 with probability 0.5, mixture mutation scale 0.01).
 *
 * Readings where the paper is silent are fields of lipz_config; they are:
 * synchronous double-buffered generations; BCE loss in logit form (mean over
 * the minibatch), lower fitness wins; one evaluation minibatch per cell and
 * generation; tournaments draw distinct slots, ties go to the first drawn,
 * NaN fitness loses; the winner's parameters, Adam state and learning rate
 * are copied, then the learning rate mutates; per training step one
 * discriminator step then one non-saturating generator step on the same
 * latent batch; the mixture score is a diagonal Frechet distance in a fixed
 * random feature space (the paper's FID needs a pretrained network).
 *
 * Sub-populations (pop_size s > 1; the paper's experiments use 1 per cell)
 * and elitist replacement, a reading of step 3 for more than one individual
 * per cell: cell c holds the individuals u = c s + i, i < s, of each role; its
 * neighbourhood population is the n = 5 s individuals nbr[c][k] s + i at
 * neighbourhood index k s + i; evaluation scores all n x n pairs;
 * selection runs s tournaments per role (member i from words 8 i .. 8 i + 7 of
 * the cell's tournament stream, learning-rate mutation from words
 * 4 i .. 4 i + 3); member i of cell c trains as unit u on the streams of cell
 * field u.  With s = 1 every draw is the one described below.  Elitism: see
 * lipz_elitist_replace.
 *
 * Random numbers: Philox4x32-10 (Salmon et al., SC 2011) with key = seed and
 * counter = (element / 4, cell, (gen << 16) | step_field, tag), word
 * element % 4; step_field = 0 for evaluation, s + 1 for training step s.
 * Uniform u = ((w >> 9) + 0.5) * 2^-23; normals by Box-Muller on (u0, u1) and
 * (u2, u3); indices floor(w * n / 2^32).  Tags are the LIPZ_TAG_* values.
 *
 * Conventions for every call:
 *  - Memory: the caller allocates ALL device memory (the workspace sized by
 *    lipz_workspace_bytes, the dataset, every output).  The library never
 *    allocates device memory; it owns only the small host handle.
 *  - Pointers named d_* are device pointers, h_* host pointers.
 *  - Streams: every call enqueues its kernels on the stream given at create
 *    (a hipStream_t passed as void*) and returns without synchronising,
 *    except create (which waits for its initialisation to finish), the state
 *    layout queries and lipz_sync.  Outputs are valid after a stream sync.
 *  - Errors: argument and call-order checks run on the host before anything
 *    is enqueued and return a negative lipz_status.  HIP launch errors are
 *    sticky on the handle and returned by the next call and by lipz_sync.
 *    No C++ exception crosses this interface.
 *  - A handle is not thread-safe; separate handles are independent.
 */
#ifndef LIPZ_H
#define LIPZ_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LIPZ_ABI_VERSION 3
#define LIPZ_SLOTS 5          /* centre, north, south, west, east */
#define LIPZ_MAX_HIDDEN 4
#define LIPZ_MAX_BANDS 8      /* row bands of lipz_run_generations */

typedef int32_t lipz_status;
enum {
  LIPZ_OK = 0,
  LIPZ_E_INVAL = -1,        /* bad argument or configuration */
  LIPZ_E_WORKSPACE = -2,    /* workspace too small or misaligned */
  LIPZ_E_HIP = -3,          /* a HIP runtime call or kernel launch failed */
  LIPZ_E_ORDER = -4,        /* call out of order (e.g. select before eval) */
  LIPZ_E_NONFINITE = -5,    /* a loss or fitness value was NaN or Inf */
  LIPZ_E_UNSUPPORTED = -6   /* configuration not implemented */
};

enum { LIPZ_NET_MLP = 0, LIPZ_NET_DCGAN = 1 };
enum { LIPZ_ACT_LINEAR = 0, LIPZ_ACT_RELU = 1, LIPZ_ACT_LRELU = 2, LIPZ_ACT_TANH = 3 };
enum { LIPZ_ROLE_G = 0, LIPZ_ROLE_D = 1 };
/* The trainer's GAN objective.  BCE: the paper's minimax objective with a
 * sigmoid discriminator (Section 3).  WASSERSTEIN: the WGAN trainer the
 * paper names as the next one to add (Section 5): a linear critic, critic
 * loss mean D(fake) - mean D(real), generator loss -mean D(fake), and every
 * critic parameter clipped to [-wgan_clip, wgan_clip] after its update. */
enum { LIPZ_LOSS_BCE = 0, LIPZ_LOSS_WASSERSTEIN = 1 };
/* How lipz_train_step updates a cell's pair.  GRADIENT: backpropagation and
 * Adam (the paper's experiments, Section 4).  NES: the gradient-free Natural
 * Evolution Strategies trainer the system also offers (Section 3,
 * "Implementation and Distribution"): per step and role, nes_pairs antithetic
 * Gaussian directions eps_k (normal k P + e of stream (cell, gen, s + 1,
 * NES_G / NES_D)), the role's loss F at theta +- nes_sigma eps_k on the
 * step's minibatch, g = sum_k (F_k+ - F_k-) eps_k / (2 nes_pairs nes_sigma),
 * one Adam step of theta on g.  ES: the gradient-free evolution-strategies
 * trainer of the same passage, read as a (1+lambda)-ES like the mixture
 * step's (1+1)-ES: per step and role the same 2 nes_pairs mutants
 * theta +- nes_sigma eps_k and the parent theta are scored on the step's
 * minibatch; the mutant of lowest loss replaces theta only if its loss is
 * strictly lower (among equal mutants the first in the order +eps_0 ..
 * +eps_(n-1), -eps_0 .. -eps_(n-1)); Adam's moments are not used.  Both
 * gradient-free trainers: MLP networks only, nes_pairs x (parameters of a
 * network) < 2^31. */
enum { LIPZ_TRAINER_GRADIENT = 0, LIPZ_TRAINER_NES = 1, LIPZ_TRAINER_ES = 2 };
enum {
  LIPZ_TAG_IDX = 1, LIPZ_TAG_Z = 2, LIPZ_TAG_TOURN_G = 3, LIPZ_TAG_TOURN_D = 4,
  LIPZ_TAG_LRMUT_G = 5, LIPZ_TAG_LRMUT_D = 6, LIPZ_TAG_MIXN = 7, LIPZ_TAG_MIXZ = 8,
  LIPZ_TAG_PROJ = 9, LIPZ_TAG_INIT_G = 10, LIPZ_TAG_INIT_D = 11, LIPZ_TAG_NES_G = 12, LIPZ_TAG_NES_D = 13
};

/* Experiment configuration (the paper's single configuration file, Section 3,
 * "Configuration").  Plain data; abi_version must be LIPZ_ABI_VERSION. */
typedef struct {
  int32_t abi_version;
  int32_t rows, cols;               /* toroidal grid; cells = rows * cols, cell id = r * cols + c */
  int32_t net;                      /* LIPZ_NET_MLP or LIPZ_NET_DCGAN (see below) */
  int32_t z_dim, x_dim;             /* latent width, flat sample width */
  int32_t img_h, img_w, img_c;      /* DCGAN only; 0 for MLP */
  int32_t n_g_hidden, g_hidden[LIPZ_MAX_HIDDEN];  /* G: z_dim -> g_hidden... -> x_dim */
  int32_t n_d_hidden, d_hidden[LIPZ_MAX_HIDDEN];  /* D: x_dim -> d_hidden... -> 1 (logit) */
  /* LIPZ_NET_DCGAN (Section 4's CelebA network): n = n_g_hidden = n_d_hidden
   * stride-2 stages, square NHWC images of side img_h = img_w = 4 * 2^n,
   * x_dim = img_h * img_w * img_c; g_hidden / d_hidden are channel widths
   * (multiples of 4, at most 1024).
   *   G: dense z -> 4x4 x g_hidden[0] (no bias), batch norm, g_hidden_act;
   *      n - 1 x [4x4 transposed conv, stride 2, pad 1 (no bias), batch
   *      norm, g_hidden_act]; 4x4 transposed conv to img_c + bias, g_out_act.
   *   D: n x [4x4 conv, stride 2, pad 1 + bias, d_hidden_act]; dense over
   *      the 4x4 x d_hidden[n-1] map to 1 logit + bias.
   * Batch norm uses the statistics of the batch it normalises (biased
   * variance, eps 1e-5).  Parameter row of a layer: the weight block
   * [(taps * c_in)][c_out] with rows (kh, kw, c_in) (taps = 16; 1 for the
   * dense layers), the bias [c_out] if any, then gamma and beta [c_out].
   * Init: weights N(0, 0.02^2), gamma N(1, 0.02^2), biases and betas 0.
   * mix_enable must be 0. */
  int32_t g_hidden_act, g_out_act, d_hidden_act;  /* LIPZ_ACT_* */
  float lrelu_slope;
  int32_t batch;                    /* minibatch rows for evaluation and training */
  int32_t tournament_size;          /* 1..5 */
  int32_t fitness_mode;             /* 0: fit_D = mean_i L, fit_G = -mean_j L (paper);
                                       1: fit_G = mean_j Lg (non-saturating G loss) */
  int32_t lr_mutation;              /* 1: mutate learning rates after replacement */
  float lr0_g, lr0_d;               /* initial learning rates */
  float beta1, beta2, eps;          /* Adam */
  float lr_mut_std, lr_mut_prob;    /* Gaussian learning-rate mutation */
  int32_t mix_enable;               /* 1: allocate and allow lipz_mixture_update */
  int32_t mix_samples;              /* shared latents per generation for the mixture score */
  int32_t mix_feat_dim;             /* random feature width F */
  float mix_sigma;                  /* (1+1)-ES mutation scale */
  uint64_t seed;
  int32_t loss_kind;                /* LIPZ_LOSS_BCE (paper) or LIPZ_LOSS_WASSERSTEIN (MLP only) */
  float wgan_clip;                  /* critic clipping bound (> 0) for LIPZ_LOSS_WASSERSTEIN */
  int32_t trainer;                  /* LIPZ_TRAINER_GRADIENT (paper's experiments), _NES or _ES */
  int32_t nes_pairs;                /* NES / ES: antithetic direction (mutant) pairs, 1..64 */
  float nes_sigma;                  /* NES / ES: perturbation (mutation) scale (> 0) */
  int32_t pop_size;                 /* s: individuals per role and cell, 1..4 (1 in the paper) */
  int32_t elitism;                  /* 1: allow lipz_elitist_replace (MLP only) */
  int32_t bands;                    /* lipz_run_generations: 0 or 1 one batch; b >= 2 row bands */
} lipz_config;

typedef struct lipz_grid lipz_grid;  /* opaque host handle */

/* Bytes of device workspace a grid with this configuration and dataset size
 * needs (0 if the configuration is invalid).  The workspace must be 256-byte
 * aligned. */
size_t lipz_workspace_bytes(const lipz_config* cfg, int64_t n_samples);

/* Step 1 (Section 3): carve the workspace, build the neighbour table, and
 * initialise every cell on the device: MLP weights and biases of layer l are
 * U(-1/sqrt(fan_in), 1/sqrt(fan_in)) from tag INIT_G / INIT_D, Adam m = v = 0,
 * t = 0, learning rates lr0_g / lr0_d, mixture weights 1/5.  With mix_enable
 * the projection P and the dataset's feature mean / std are computed here.
 * d_dataset: [n_samples][x_dim] fp32 row-major, borrowed (must outlive the
 * grid).  hip_stream: hipStream_t or NULL for the null stream.  Waits for
 * the initialisation to finish. */
lipz_status lipz_grid_create(const lipz_config* cfg, void* d_workspace, size_t workspace_bytes,
                             const float* d_dataset, int64_t n_samples, void* hip_stream,
                             lipz_grid** out);
lipz_status lipz_grid_destroy(lipz_grid* g);

/* For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, harnesses that forbid hipMalloc): lipz_grid_create
 * with the workspace taken from a static device array of
 * LIPZ_STATIC_WORKSPACE_BYTES that the library holds on every GPU it runs on
 * until the process ends; the grid lives on the current device.  It calls no
 * hipMalloc / hipFree and creates no stream or event; initialisation,
 * results and the other calls are those of lipz_grid_create.  The array
 * keeps whatever the last grid left in it; the create clears what must
 * start at zero.  One such grid per device at a time: a second create on the
 * same device returns LIPZ_E_ORDER until lipz_grid_destroy (which waits for
 * the grid's stream) releases the array; work enqueued on it from other
 * threads or streams after that races with the next grid.  Errors:
 * LIPZ_E_WORKSPACE when lipz_workspace_bytes(cfg, n_samples) exceeds
 * LIPZ_STATIC_WORKSPACE_BYTES (e.g. the 2x2 ring-of-Gaussians grid needs
 * 6.4 MiB, the 3x3 MNIST-shaped grid 214 MiB), LIPZ_E_UNSUPPORTED for row
 * bands (bands >= 2: they create streams) or a device index >= 64,
 * LIPZ_E_INVAL for an invalid configuration, LIPZ_E_HIP when the array
 * cannot be located on the device. */
#define LIPZ_STATIC_WORKSPACE_BYTES ((size_t)64 << 20)
lipz_status lipz_grid_create_static(const lipz_config* cfg, const float* d_dataset, int64_t n_samples,
                                    void* hip_stream, lipz_grid** out);

/* Step 2 (Section 3): for every cell c, draw one minibatch (B data rows,
 * B latents; step_field 0) and evaluate each generator slot i against each
 * discriminator slot j of its neighbourhood:
 *   L [c][i][j] = mean_b softplus(-D_j(x_b)) + mean_b softplus(D_j(G_i(z_b)))
 *   Lg[c][i][j] = mean_b softplus(-D_j(G_i(z_b)))
 *   (LIPZ_LOSS_WASSERSTEIN: L = mean_b D_j(G_i(z_b)) - mean_b D_j(x_b),
 *    Lg = -mean_b D_j(G_i(z_b)))
 *   fit_d[c][j] = mean_i L[c][i][j];  fit_g[c][i] = -mean_j L[c][i][j]
 *   (fitness_mode 1: fit_g[c][i] = mean_j Lg[c][i][j]).  Lower is better.
 * Outputs fp32 [C][n][n] / [C][n] (n = 5 pop_size, neighbourhood index
 * k s + i); any may be NULL.  A non-finite value sets the sticky
 * LIPZ_E_NONFINITE flag reported by lipz_sync. */
lipz_status lipz_eval_neighborhoods(lipz_grid* g, int32_t gen, float* d_L, float* d_Lg,
                                    float* d_fit_g, float* d_fit_d);

/* Step 3, selection (Section 3): per cell, member i < s and role, a
 * tournament of tournament_size distinct neighbourhood indices on the
 * fitness of the last evaluation (draw j picks position
 * floor(w_(8i+j) (n - j) / 2^32) among the undrawn indices; lowest fitness
 * wins, NaN loses, ties go to the first drawn).  The winner's parameters,
 * Adam m, v, t and learning rate are copied into individual c s + i (the
 * next state buffer becomes current), then with probability lr_mut_prob the
 * learning rate gets + N(0, lr_mut_std^2), clamped at 0 (words 4i / 4i+2,
 * 4i+3 of tag LRMUT_G / LRMUT_D).  d_forced [U][2] int32 (source
 * individuals for G, D; U = C pop_size) replaces the tournaments when not
 * NULL (an id outside [0, U) keeps the individual and is reported by
 * lipz_sync).  d_sel [U][2] int32 receives the source individuals, d_lr
 * [U][2] fp32 the new learning rates; either may be NULL.
 * Without d_forced, requires a preceding lipz_eval_neighborhoods since the
 * last state change (else LIPZ_E_ORDER). */
lipz_status lipz_select_replace(lipz_grid* g, int32_t gen, const int32_t* d_forced,
                                int32_t* d_sel, float* d_lr);

/* Step 3, training (Section 3): n_steps training steps s = step0 ..
 * step0 + n_steps - 1 of every cell's own pair.  Per step: minibatch and
 * latents from step_field s + 1; discriminator Adam step on
 * mean softplus(-D(x)) + mean softplus(D(G(z))) with G(z) detached; then
 * generator Adam step on mean softplus(-D'(G(z))) against the updated
 * discriminator D' and the same z.  Adam: bias-corrected, per-cell learning
 * rate and step count.  LIPZ_LOSS_WASSERSTEIN: the critic minimises
 * mean D(G(z)) - mean D(x), then every critic parameter is clipped to
 * [-wgan_clip, wgan_clip]; the generator minimises -mean D'(G(z)).
 * LIPZ_TRAINER_NES: the same two losses, each minimised by one Adam step on
 * the NES estimate of its gradient (see LIPZ_TRAINER_NES); the losses
 * reported are those at the unperturbed parameters.  LIPZ_TRAINER_ES: the
 * same two losses, each by one plus-selection (see LIPZ_TRAINER_ES), then
 * the critic clip; losses at the parents; step counts advance by n_steps.
 * Every individual pair u < U = C pop_size trains (its minibatches and
 * latents from cell field u).
 * d_losses [n_steps][U][2] fp32 (L_D, L_G before each update) may be NULL. */
lipz_status lipz_train_step(lipz_grid* g, int32_t gen, int32_t step0, int32_t n_steps,
                            float* d_losses);

/* Post-training re-evaluation and elitist replacement (a reading of step 3
 * for elitism = 1; the paper's experiments replace unconditionally).  Scores
 * each cell's s trained generators against the n discriminators of the
 * previous state's neighbourhood, and its s trained discriminators against
 * the n previous generators, on the minibatch of generation gen's
 * evaluation (step_field 0), the opponents and rows that gave the cell's own
 * s previous individuals their fitness:
 *   fit2_g[c][i] = -mean_j L(G'_i, D_j)  (fitness_mode 1: mean_j Lg),
 *   fit2_d[c][j] = mean_k L(G_k, D'_j).
 * Of the 2 s per role the s of lowest fitness are kept (NaN last; ties to
 * the trained individual, then the lower member): a kept trained individual
 * stays in its slot; the kept previous ones, best first, take the slots of
 * the dropped trained ones in slot order, with their parameters, Adam state,
 * step count and learning rate.  Requires lipz_eval_neighborhoods(gen), then
 * lipz_select_replace (the previous state is the buffer it read), then any
 * number of lipz_train_step calls; another evaluation, selection, state load
 * or elitist replacement in between gives LIPZ_E_ORDER.  Outputs (any
 * may be NULL): d_src [U][2] int32 (-1: the trained individual stays, else
 * the previous member j < s whose individual c s + j took the slot),
 * d_fit2_g / d_fit2_d [C][s] fp32.  LIPZ_E_ORDER if elitism = 0. */
lipz_status lipz_elitist_replace(lipz_grid* g, int32_t gen, int32_t* d_src, float* d_fit2_g,
                                 float* d_fit2_d);

/* Steps 2-3 for n_gens generations gen0 .. gen0 + n_gens - 1, each of them
 * lipz_eval_neighborhoods, lipz_select_replace, lipz_train_step(gen, 0,
 * n_steps) and (elitism = 1) lipz_elitist_replace, and, with mix_enable,
 * lipz_mixture_update, with the same results bit for bit.
 *
 * bands >= 2 (MLP networks, every trainer, with or without the mixture
 * step, whose ES also waits for the neighbour bands' moments): the paper's
 * cells run asynchronously (Section 3, step 1 and its Figure 1), and this is
 * that scheduling on one device.  The grid's rows are split into `bands` row
 * bands, each on its own stream, and nothing waits for the whole grid: a
 * band starts generation g + 1 as soon as the bands holding its cells'
 * neighbour rows have finished generation g (a readiness event per band),
 * so bands that are not neighbours drift apart by up to the grid's band
 * distance in generations, and neighbours by at most one.  That rule keeps
 * every read of a neighbour's individuals and every overwrite of a state
 * buffer ordered as in the synchronous schedule.  Returns after enqueuing;
 * the caller's stream waits for every band at the end. */
lipz_status lipz_run_generations(lipz_grid* g, int32_t gen0, int32_t n_gens, int32_t n_steps);

/* Step 4 (Section 3): one (1+1)-ES step on every cell's mixture weights over
 * the generators of its neighbourhood (current state).  Features f = x P,
 * P [x_dim][F] ~ N(0, 1/x_dim) (tag PROJ); generator moments over
 * mix_samples shared latents (tag MIXZ, step_field 0);
 *   score(w) = ||mu_w - mu_r||^2 + ||sqrt(max(s_w - mu_w^2, 0)) - sd_r||^2,
 *   mu_w = sum_k w_k mean(f_k), s_w = sum_k w_k mean(f_k^2);
 * proposal w' = max(w + mix_sigma n, 0) / sum (n: tag MIXN), accepted iff
 * score(w') < score(w).  Outputs (any may be NULL): d_w [C][5] fp32,
 * d_score [C] fp32 (score of the kept w), d_accepted [C] int32.
 * LIPZ_E_ORDER if the grid was created with mix_enable = 0 (which
 * pop_size > 1 requires). */
lipz_status lipz_mixture_update(lipz_grid* g, int32_t gen, float* d_w, float* d_score,
                                int32_t* d_accepted);

/* ---- inspection, checkpoint and teacher forcing ---- */

/* Neighbour table [C][5] int32 into host memory. */
lipz_status lipz_get_neighbors(const lipz_grid* g, int32_t* h_nbr);

/* Parameter layout of one role's network: *h_n = number of layers; for
 * layer l, h_offsets[3l + 0] = float offset of W_l in the cell's parameter
 * row, [3l + 1] = fan_in, [3l + 2] = fan_out.  W_l is [fan_in][fan_out]
 * row-major and its bias [fan_out] follows it directly (DCGAN: fan_in =
 * taps * c_in, and a layer without bias is followed by its batch-norm gamma
 * and beta instead).  h_offsets may be
 * NULL to query *h_n; it must hold 3 * (LIPZ_MAX_HIDDEN + 1) entries. */
lipz_status lipz_param_layout(const lipz_grid* g, int32_t role, int64_t* h_offsets, int32_t* h_n);

/* State blob: the current population, in this layout (byte offsets written
 * to h_offsets[0..11] by lipz_state_layout; h_offsets[11] = total bytes):
 *   [0] Gp float [U][stride_G]  [1] Gm  [2] Gv     (U = C pop_size)
 *   [3] Dp float [U][stride_D]  [4] Dm  [5] Dv
 *   [6] Gt int32 [U]  [7] Dt int32 [U]  [8] Glr float [U]  [9] Dlr float [U]
 *   [10] w float [C][5]
 * h_strides[0] = stride_G, h_strides[1] = stride_D (floats per cell row,
 * >= the role's parameter count; the padding is ignored). */
lipz_status lipz_state_layout(const lipz_grid* g, int64_t* h_offsets, int64_t* h_strides);
size_t lipz_state_bytes(const lipz_grid* g);
/* Device-to-device copies of the current state, enqueued on the grid's
 * stream.  lipz_load_state invalidates the last evaluation. */
lipz_status lipz_save_state(lipz_grid* g, void* d_dst);
lipz_status lipz_load_state(lipz_grid* g, const void* d_src);

/* Synchronise the grid's stream; returns a sticky HIP error, then
 * LIPZ_E_INVAL if a forced source individual of lipz_select_replace was
 * outside [0, U) (that individual kept itself), then LIPZ_E_NONFINITE if any
 * evaluation produced a non-finite value.  Both flags are sticky. */
lipz_status lipz_sync(lipz_grid* g);
const char* lipz_error_string(lipz_status s);
/* Last error message of this handle ("" if none); valid until the next call. */
const char* lipz_last_error(const lipz_grid* g);

/* ---- kernel timing (for roofline measurement) ----
 * When enabled, every launch of the matrix-core kernels (the grouped GEMM
 * and, for LIPZ_NET_DCGAN, the implicit-GEMM convolution) is bracketed by
 * HIP events that the launch's own dispatch stamps.  lipz_gemm_timing
 * synchronises and returns, since the previous call: the summed kernel
 * milliseconds, the launch count, the algorithmic FLOPs (2 per multiply-add
 * of the GEMM and convolution problems, bias rows excluded) and the
 * algorithmic bytes (each operand element read once, each output element
 * written once, Adam's p, m, v read and written).  Any output pointer may be
 * NULL. */
lipz_status lipz_set_gemm_timing(lipz_grid* g, int32_t enable);
lipz_status lipz_gemm_timing(lipz_grid* g, double* h_ms, int64_t* h_launches, double* h_flops,
                             double* h_bytes);

#ifdef __cplusplus
}
#endif
#endif /* LIPZ_H */
