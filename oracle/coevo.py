"""One generation of the grid coevolution, in fp64, in the order of Section 3
("Coevolutionary GAN Training", steps 1-5):

 1. random initialisation of every cell's generator (u_i, delta_i) and
    discriminator (v_j, gamma_j);                                   -> create
 2. every generator is evaluated against every discriminator of its
    neighbourhood; the loss values of a discriminator are averaged and those
    of a generator negative-averaged to give fitness;               -> evaluate
 3. tournament selection of one generator and one discriminator per
    neighbourhood, Gaussian update of their hyper-parameters (learning rate),
    gradient (Adam) training of the selected pair;        -> select_replace,
                                                              train_step
 4. the generator-mixture weights w of each neighbourhood evolve by a
    (1+1)-ES (module ``mixture``);
 5. repeat from 2.

Readings where the paper is silent (each is a workload field):
 * synchronous, double-buffered generations (state g is read, g+1 written);
 * the loss L(u_i, v_j) is the discriminator's binary cross-entropy,
   mean over the minibatch of softplus(-a_real) + mean of softplus(a_fake),
   a = logit; lower fitness wins for both roles (fitness_mode 0);
 * one evaluation minibatch per cell per generation, shared by its 25 pairs;
 * tournament draws distinct slots; ties go to the first drawn; NaN loses;
 * replacement is unconditional (population size 1 per cell): the winner's
   parameters and Adam state (m, v, t) and learning rate are copied;
 * learning-rate mutation after copying: with the given probability add
   N(0, std^2), clamp at 0;
 * training: per step one discriminator step (real vs detached fake), then
   one non-saturating generator step against the updated discriminator on
   the same latent batch; Adam with beta1, beta2, eps, bias-corrected.

Sub-populations (workload pop_size s; Table 1 fixes 1 per cell) and elitist
replacement (workload elitism), a reading of step 3 for more than one
individual per cell:
 * cell c holds s generators and s discriminators, individuals c s + i
   (i < s); its neighbourhood population is the 5 s individuals of its 5
   slots, neighbourhood index k s + i for member i of slot k; evaluation
   scores all 5s x 5s pairs on the cell's minibatch;
 * s tournaments per role and cell: tournament i draws from words
   8 i .. 8 i + 7 of the cell's tournament stream and fills member i of the
   new sub-population, whose learning rate mutates with words 4 i .. 4 i + 3
   of the cell's mutation stream;
 * member i of cell c trains on the minibatches and latents of stream
   c s + i (a training unit); with s = 1 every draw is the one above;
 * elitism 1: after training, the cell's s trained generators are scored
   against the 5 s discriminators of the previous state (and its trained
   discriminators against the 5 s previous generators) on step 2's
   minibatch, the same opponents and rows that gave the cell's own s
   previous individuals their fitness; of those 2 s per role the s of lowest
   fitness are kept (NaN last; ties to the trained one, then the lower
   member): a kept trained individual stays in its slot, and the kept
   previous ones, best first, take the slots of the dropped trained ones in
   slot order, with their Adam state and learning rate (elitist_replace).

The Wasserstein trainer (workload loss "wasserstein"; the paper names WGAN as
the next trainer to add, Section 5, and its trainers differ only in the weight
update and the fitness evaluation, Section 3): D is a critic with a linear
output a; L(u_i, v_j) = mean a_fake - mean a_real (the critic's loss, lower is
better for it), the generator's own loss is -mean a_fake; training minimises
those two losses with the same Adam steps, and after every discriminator
update each of its parameters is clipped to [-c, c] (weight clipping of the
original WGAN, c = wgan_clip).
"""
import numpy as np
from scipy.special import expit

from . import dcgan, grid, mlp, rng


def softplus(x):
    return np.logaddexp(0.0, x)


class MlpNet:
    """One role's fully connected network (module ``mlp``)."""

    def __init__(self, role, sizes, acts, slope):
        self.role, self.sizes, self.acts, self.slope = role, sizes, acts, slope
        self.P = mlp.layout(sizes)[1]

    def init(self, seed, cell, tag):
        return mlp.init(self.sizes, seed, cell, tag)

    def forward(self, p, x):
        """(cache, out): out = G's samples [N, x_dim] or D's logits [N]."""
        pre, post = mlp.forward(p, self.sizes, self.acts, x, self.slope)
        return (pre, post), (post[-1] if self.role == "G" else post[-1][:, 0])

    def backward(self, p, cache, d_out, want_input_grad=False):
        d = d_out if self.role == "G" else d_out[:, None]
        return mlp.backward(p, self.sizes, self.acts, cache[0], cache[1], d, self.slope,
                            want_input_grad)


class ConvNet:
    """One role's DCGAN-style network (module ``dcgan``)."""

    def __init__(self, role, wl):
        self.arch = dcgan.Arch(role, wl["z_dim"], tuple(wl["img"]), wl["g_hidden"], wl["d_hidden"])
        self.role, self.slope, self.P = role, wl["lrelu_slope"], self.arch.P

    def init(self, seed, cell, tag):
        return dcgan.init(self.arch, seed, cell, tag)

    def forward(self, p, x):
        return dcgan.forward(self.arch, p, x, self.slope)

    def backward(self, p, cache, d_out, want_input_grad=False):
        return dcgan.backward(self.arch, p, cache, d_out, self.slope, want_input_grad)


class Setup:
    """Static description derived from a workload dict and the dataset."""

    def __init__(self, wl, n_samples):
        if wl["net"] not in ("mlp", "dcgan"):
            raise ValueError(f"unknown network kind {wl['net']!r}")
        self.wl = wl
        self.rows, self.cols = wl["rows"], wl["cols"]
        self.C = self.rows * self.cols
        self.nbr = grid.neighbours(self.rows, self.cols)
        self.B = wl["batch"]
        self.zd, self.xd = wl["z_dim"], wl["x_dim"]
        self.g_sizes = [self.zd] + list(wl["g_hidden"]) + [self.xd]
        self.g_acts = [wl["g_hidden_act"]] * len(wl["g_hidden"]) + [wl["g_out_act"]]
        self.d_sizes = [self.xd] + list(wl["d_hidden"]) + [1]
        self.d_acts = [wl["d_hidden_act"]] * len(wl["d_hidden"]) + ["linear"]
        self.slope = wl["lrelu_slope"]
        self.seed = wl["seed"]
        self.N = int(n_samples)
        if wl["net"] == "mlp":
            self.Gnet = MlpNet("G", self.g_sizes, self.g_acts, self.slope)
            self.Dnet = MlpNet("D", self.d_sizes, self.d_acts, self.slope)
        else:
            if wl["mix_enable"]:
                raise ValueError("the mixture step is defined for the MLP workloads only")
            self.Gnet, self.Dnet = ConvNet("G", wl), ConvNet("D", wl)
        self.PG, self.PD = self.Gnet.P, self.Dnet.P
        self.loss = wl.get("loss", "bce")
        if self.loss not in ("bce", "wasserstein"):
            raise ValueError(f"unknown loss {self.loss!r}")
        self.clip = float(wl.get("wgan_clip", 0.01))
        self.trainer = wl.get("trainer", "gradient")
        if self.trainer not in ("gradient", "nes", "es"):
            raise ValueError(f"unknown trainer {self.trainer!r}")
        if self.trainer in ("nes", "es") and wl["net"] != "mlp":
            raise ValueError("the gradient-free trainers are defined for the MLP workloads")
        self.s = int(wl.get("pop_size", 1))
        self.elitism = int(wl.get("elitism", 0))
        if not 1 <= self.s <= 4 or self.elitism not in (0, 1):
            raise ValueError("pop_size must be in [1, 4] and elitism 0 or 1")
        if (self.s > 1 or self.elitism) and wl["net"] != "mlp":
            raise ValueError("sub-populations and elitism are defined for the MLP workloads")
        if self.s > 1 and wl["mix_enable"]:
            raise ValueError("the mixture step is defined for one generator per cell")
        self.U = self.C * self.s            # individuals (training units) per role
        self.n = grid.N_SLOTS * self.s      # neighbourhood population per role
        # pool[c, k s + i] = individual of member i of slot k
        self.pool = (self.nbr[:, :, None] * self.s + np.arange(self.s)[None, None, :]).reshape(self.C, self.n)


class State:
    """Per-cell individuals: params, Adam m, v, step t and learning rate per role; mixture w."""

    FIELDS = ("Gp", "Gm", "Gv", "Gt", "Glr", "Dp", "Dm", "Dv", "Dt", "Dlr", "w")

    def __init__(self, **kw):
        for k in self.FIELDS:
            setattr(self, k, kw[k])

    def copy(self):
        return State(**{k: np.array(getattr(self, k), copy=True) for k in self.FIELDS})


def create(S):
    """Step 1: random initial individuals (individual u from stream u), zero Adam
    state, initial learning rates, w = 1/5."""
    wl = S.wl
    Gp = np.stack([S.Gnet.init(S.seed, u, "INIT_G") for u in range(S.U)])
    Dp = np.stack([S.Dnet.init(S.seed, u, "INIT_D") for u in range(S.U)])
    return State(Gp=Gp, Gm=np.zeros_like(Gp), Gv=np.zeros_like(Gp),
                 Gt=np.zeros(S.U, dtype=np.int64), Glr=np.full(S.U, float(wl["lr0_g"])),
                 Dp=Dp, Dm=np.zeros_like(Dp), Dv=np.zeros_like(Dp),
                 Dt=np.zeros(S.U, dtype=np.int64), Dlr=np.full(S.U, float(wl["lr0_d"])),
                 w=np.full((S.C, grid.N_SLOTS), 1.0 / grid.N_SLOTS))


def sample(S, data, cell, gen, step_field):
    """Minibatch rows drawn uniformly with replacement and a latent batch z ~ N(0, 1)."""
    idx = rng.indices(S.seed, S.B, S.N, cell, gen, step_field)
    z = rng.normals(S.seed, S.B * S.zd, cell, gen, step_field, "Z").reshape(S.B, S.zd)
    return idx, np.asarray(data[idx], dtype=np.float64), z


def g_forward(S, p, z):
    """(cache, G(z)) with G(z) [N, x_dim]."""
    return S.Gnet.forward(p, z)


def d_logits(S, p, x):
    """(cache, logits [N])."""
    return S.Dnet.forward(p, x)


def pair_losses(S, a_r, a_f):
    """(L, Lg) of one (generator, discriminator) pair from the critic outputs
    on the real and the fake rows: the discriminator's loss and the
    generator's own loss."""
    if S.loss == "wasserstein":
        return a_f.mean() - a_r.mean(), -a_f.mean()
    return softplus(-a_r).mean() + softplus(a_f).mean(), softplus(-a_f).mean()


def d_loss_grads(S, a_r, a_f):
    """dL_D/da for the real and the fake rows of a discriminator step."""
    B = len(a_r)
    if S.loss == "wasserstein":
        return np.full(B, -1.0 / B), np.full(len(a_f), 1.0 / len(a_f))
    return (expit(a_r) - 1.0) / B, expit(a_f) / len(a_f)


def g_loss_grad(S, a_f):
    """dL_G/da for the fake rows of a generator step."""
    if S.loss == "wasserstein":
        return np.full(len(a_f), -1.0 / len(a_f))
    return (expit(a_f) - 1.0) / len(a_f)


def evaluate(S, st, data, gen):
    """Step 2: all n x n pairs of each neighbourhood (n = 5 s), then fitness.

    Returns L[C,n,n] (discriminator BCE), Lg[C,n,n] (non-saturating generator
    loss), fit_g[C,n], fit_d[C,n], indexed by neighbourhood index k s + i.
    """
    C, n = S.C, S.n
    L = np.zeros((C, n, n))
    Lg = np.zeros((C, n, n))
    for c in range(C):
        L[c], Lg[c] = evaluate_cell(S, st, data, gen, c)
    fit_d = L.mean(axis=1)
    if S.wl["fitness_mode"] == 0:
        fit_g = -L.mean(axis=2)
    else:
        fit_g = Lg.mean(axis=2)
    return L, Lg, fit_g, fit_d


def evaluate_cell(S, st, data, gen, c):
    """The n x n pair losses (L, Lg) of cell c's neighbourhood on its
    evaluation minibatch (one cell of evaluate)."""
    n = S.n
    L = np.zeros((n, n))
    Lg = np.zeros((n, n))
    _, x, z = sample(S, data, c, gen, 0)
    fakes = [g_forward(S, st.Gp[S.pool[c, i]], z)[1] for i in range(n)]
    for j in range(n):
        dp = st.Dp[S.pool[c, j]]
        a_r = d_logits(S, dp, x)[1]
        for i in range(n):
            L[i, j], Lg[i, j] = pair_losses(S, a_r, d_logits(S, dp, fakes[i])[1])
    return L, Lg


def tournament_draw(S, cell, gen, tag, member=0):
    """Distinct neighbourhood indices in draw order for tournament `member`:
    draw j picks position floor(w_(8 member + j) * (n - j) / 2^32) among the
    indices not yet drawn (kept in order); a tournament of all n takes the
    last one without a draw."""
    size, n = S.wl["tournament_size"], S.n
    w = rng.raw_words(S.seed, 8 * (member + 1), cell, gen, 0, tag)[8 * member:]
    remaining = list(range(n))
    drawn = []
    for j in range(min(size, n - 1)):
        pos = int((int(w[j]) * (n - j)) >> 32)
        drawn.append(remaining.pop(pos))
    if size == n:
        drawn.append(remaining.pop(0))
    return drawn


def tournament_winner(fit_row, drawn):
    """Lowest fitness wins; NaN counts as +inf; ties go to the earliest drawn slot."""
    def key(f):
        return np.inf if np.isnan(f) else f
    best = drawn[0]
    for k in drawn[1:]:
        if key(fit_row[k]) < key(fit_row[best]):
            best = k
    return best


def mutate_lr(S, lr, cell, gen, tag, member=0):
    """Gaussian hyper-parameter update of member `member`'s copy: with
    probability p, lr += std * n; clamp at 0 (words 4 member .. 4 member + 3)."""
    wl = S.wl
    if not wl["lr_mutation"]:
        return lr
    u = rng.to_uniform(rng.raw_words(S.seed, 4 * (member + 1), cell, gen, 0, tag)[4 * member:])
    if u[0] < wl["lr_mut_prob"]:
        n = rng.box_muller(u)[2]
        lr = max(lr + wl["lr_mut_std"] * n, 0.0)
    return lr


def select_replace(S, st, fit_g, fit_d, gen, forced=None):
    """Step 3 (selection part): returns (state g+1, sel[U,2] source individuals (G, D))."""
    new = st.copy()
    sel = np.zeros((S.U, 2), dtype=np.int64)
    for c in range(S.C):
        for i in range(S.s):
            u = c * S.s + i
            for r, (fit, ttag, mtag, pre) in enumerate(((fit_g, "TOURN_G", "LRMUT_G", "G"),
                                                         (fit_d, "TOURN_D", "LRMUT_D", "D"))):
                if forced is not None:
                    src = int(forced[u, r])
                else:
                    src = int(S.pool[c, tournament_winner(fit[c], tournament_draw(S, c, gen, ttag, i))])
                sel[u, r] = src
                for f in ("p", "m", "v", "t"):
                    getattr(new, pre + f)[u] = getattr(st, pre + f)[src]
                getattr(new, pre + "lr")[u] = mutate_lr(S, getattr(st, pre + "lr")[src], c, gen, mtag, i)
    return new, sel


def adam(S, p, m, v, t, lr, g):
    """One bias-corrected Adam step in place; returns the new step count."""
    b1, b2, eps = S.wl["beta1"], S.wl["beta2"], S.wl["eps"]
    t = t + 1
    m *= b1
    m += (1.0 - b1) * g
    v *= b2
    v += (1.0 - b2) * g * g
    mhat = m / (1.0 - b1 ** t)
    vhat = v / (1.0 - b2 ** t)
    p -= lr * mhat / (np.sqrt(vhat) + eps)
    return t


def train_step(S, st, data, gen, step):
    """Step 3 (training part): one discriminator and one generator Adam step for
    every training unit (individual pair) c, in place.  Returns losses[U, 2] =
    (L_D, L_G) before the updates."""
    losses = np.zeros((S.U, 2))
    for c in range(S.U):
        losses[c] = train_unit(S, st, data, gen, step, c)
    return losses


def train_unit(S, st, data, gen, step, c):
    """Training step `step` of unit c alone (one iteration of train_step), in
    place on st's row c; returns (L_D, L_G) before the updates."""
    losses = np.zeros(2)
    _, x, z = sample(S, data, c, gen, step + 1)
    gcache, xf = g_forward(S, st.Gp[c], z)
    # discriminator step on real and detached fake
    cache_r, a_r = d_logits(S, st.Dp[c], x)
    cache_f, a_f = d_logits(S, st.Dp[c], xf)
    losses[0] = pair_losses(S, a_r, a_f)[0]
    d_r, d_f = d_loss_grads(S, a_r, a_f)
    g_r, _ = S.Dnet.backward(st.Dp[c], cache_r, d_r)
    g_f, _ = S.Dnet.backward(st.Dp[c], cache_f, d_f)
    st.Dt[c] = adam(S, st.Dp[c], st.Dm[c], st.Dv[c], st.Dt[c], st.Dlr[c], g_r + g_f)
    if S.loss == "wasserstein":
        np.clip(st.Dp[c], -S.clip, S.clip, out=st.Dp[c])
    # generator step (non-saturating) against the updated discriminator, same z
    cache2, a2 = d_logits(S, st.Dp[c], xf)
    losses[1] = pair_losses(S, a2, a2)[1]
    _, dxf = S.Dnet.backward(st.Dp[c], cache2, g_loss_grad(S, a2), want_input_grad=True)
    gG, _ = S.Gnet.backward(st.Gp[c], gcache, dxf)
    st.Gt[c] = adam(S, st.Gp[c], st.Gm[c], st.Gv[c], st.Gt[c], st.Glr[c], gG)
    return losses


def merge_elite(f_old, f_new):
    """Elitist truncation of one role of one cell: f_old[s] the previous
    members' fitness, f_new[s] the trained ones'.  Returns src[s]: -1 where the
    trained member stays, else the previous member that takes the slot."""
    s = len(f_old)

    def key(f):
        return np.inf if np.isnan(f) else float(f)
    ranked = sorted([(key(f_new[i]), 0, i) for i in range(s)] + [(key(f_old[i]), 1, i) for i in range(s)])[:s]
    kept_new = {i for _, kind, i in ranked if kind == 0}
    kept_old = [i for _, kind, i in ranked if kind == 1]  # best first
    free = [i for i in range(s) if i not in kept_new]
    src = np.full(s, -1, dtype=np.int64)
    for slot, i in zip(free, kept_old):
        src[slot] = i
    return src


def elitist_replace(S, old, new, data, gen, fit_g, fit_d, forced=None):
    """Post-training re-evaluation and elitist replacement (elitism 1): returns
    (state, info) with info = dict(fit_g2[C,s], fit_d2[C,s], src[U,2]);
    src[c s + i, r] = -1 (trained member stays) or the previous member j whose
    individual c s + j of `old` took the slot.  forced [U,2], in the same
    form, replaces the truncation's choice (a caller replaying another
    implementation's decisions on near-ties)."""
    s, n = S.s, S.n
    out = new.copy()
    fg2, fd2 = np.zeros((S.C, s)), np.zeros((S.C, s))
    src = np.full((S.U, 2), -1, dtype=np.int64)
    for c in range(S.C):
        _, x, z = sample(S, data, c, gen, 0)
        pool = S.pool[c]
        for i in range(s):
            xf = g_forward(S, new.Gp[c * s + i], z)[1]
            L2, Lg2 = np.zeros(n), np.zeros(n)
            for j in range(n):
                dp = old.Dp[pool[j]]
                L2[j], Lg2[j] = pair_losses(S, d_logits(S, dp, x)[1], d_logits(S, dp, xf)[1])
            fg2[c, i] = -L2.mean() if S.wl["fitness_mode"] == 0 else Lg2.mean()
        fakes = [g_forward(S, old.Gp[pool[k]], z)[1] for k in range(n)]
        for j in range(s):
            dp = new.Dp[c * s + j]
            a_r = d_logits(S, dp, x)[1]
            fd2[c, j] = np.mean([pair_losses(S, a_r, d_logits(S, dp, fakes[k])[1])[0] for k in range(n)])
        for r, (f_old, f_new, pre) in enumerate(((fit_g[c, :s], fg2[c], "G"), (fit_d[c, :s], fd2[c], "D"))):
            src[c * s:(c + 1) * s, r] = merge_elite(f_old, f_new) if forced is None else forced[c * s:(c + 1) * s, r]
            for i in range(s):
                j = src[c * s + i, r]
                if j >= 0:
                    for f in ("p", "m", "v", "t", "lr"):
                        getattr(out, pre + f)[c * s + i] = getattr(old, pre + f)[c * s + j]
    return out, dict(fit_g2=fg2, fit_d2=fd2, src=src)


def generation(S, st, data, gen, mix_stats=None):
    """Steps 2-4 for one generation; returns (new state, record dict)."""
    from . import es, mixture, nes
    L, Lg, fg, fd = evaluate(S, st, data, gen)
    st2, sel = select_replace(S, st, fg, fd, gen)
    step_fn = {"nes": nes.train_step, "es": es.train_step}.get(S.trainer, train_step)
    losses = [step_fn(S, st2, data, gen, s) for s in range(S.wl["steps"])]
    rec = dict(L=L, Lg=Lg, fit_g=fg, fit_d=fd, sel=sel, losses=np.array(losses))
    if S.elitism:
        st2, info = elitist_replace(S, st, st2, data, gen, fg, fd)
        rec.update(info)
    if S.wl["mix_enable"]:
        w, score, acc = mixture.update(S, st2, mix_stats, gen)
        st2.w[...] = w
        rec.update(w=w, score=score, accepted=acc)
    return st2, rec
