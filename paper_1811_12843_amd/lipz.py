"""ctypes binding of liblipz.so: same names as the C ABI (include/lipz.h),
argument marshalling only.  Device pointers are passed as Python ints (for a
torch tensor: ``t.data_ptr()``), streams as ints (``stream.cuda_stream``).

Importing this module does not need a GPU.  Loading the library fails loudly
if it has not been built (``python -m paper_1811_12843_amd.build``).
"""
import ctypes
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("LIPZ_LIBRARY") or os.path.join(_PKG, "liblipz.so")

LIPZ_ABI_VERSION = 3
LIPZ_MAX_HIDDEN = 4
LIPZ_OK, LIPZ_E_INVAL, LIPZ_E_WORKSPACE, LIPZ_E_HIP, LIPZ_E_ORDER, LIPZ_E_NONFINITE, \
    LIPZ_E_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
LIPZ_NET_MLP, LIPZ_NET_DCGAN = 0, 1
LIPZ_ACT_LINEAR, LIPZ_ACT_RELU, LIPZ_ACT_LRELU, LIPZ_ACT_TANH = 0, 1, 2, 3
LIPZ_ROLE_G, LIPZ_ROLE_D = 0, 1
LIPZ_LOSS_BCE, LIPZ_LOSS_WASSERSTEIN = 0, 1
LOSSES = {"bce": LIPZ_LOSS_BCE, "wasserstein": LIPZ_LOSS_WASSERSTEIN}
LIPZ_TRAINER_GRADIENT, LIPZ_TRAINER_NES, LIPZ_TRAINER_ES = 0, 1, 2
LIPZ_STATIC_WORKSPACE_BYTES = 64 << 20
TRAINERS = {"gradient": LIPZ_TRAINER_GRADIENT, "nes": LIPZ_TRAINER_NES, "es": LIPZ_TRAINER_ES}
ACTS = {"linear": LIPZ_ACT_LINEAR, "relu": LIPZ_ACT_RELU, "lrelu": LIPZ_ACT_LRELU, "tanh": LIPZ_ACT_TANH}

_i32, _i64, _f32, _u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_uint64
_vp, _sz = ctypes.c_void_p, ctypes.c_size_t


class lipz_config(ctypes.Structure):
    _fields_ = [
        ("abi_version", _i32), ("rows", _i32), ("cols", _i32), ("net", _i32),
        ("z_dim", _i32), ("x_dim", _i32), ("img_h", _i32), ("img_w", _i32), ("img_c", _i32),
        ("n_g_hidden", _i32), ("g_hidden", _i32 * LIPZ_MAX_HIDDEN),
        ("n_d_hidden", _i32), ("d_hidden", _i32 * LIPZ_MAX_HIDDEN),
        ("g_hidden_act", _i32), ("g_out_act", _i32), ("d_hidden_act", _i32),
        ("lrelu_slope", _f32),
        ("batch", _i32), ("tournament_size", _i32), ("fitness_mode", _i32), ("lr_mutation", _i32),
        ("lr0_g", _f32), ("lr0_d", _f32), ("beta1", _f32), ("beta2", _f32), ("eps", _f32),
        ("lr_mut_std", _f32), ("lr_mut_prob", _f32),
        ("mix_enable", _i32), ("mix_samples", _i32), ("mix_feat_dim", _i32), ("mix_sigma", _f32),
        ("seed", _u64),
        ("loss_kind", _i32), ("wgan_clip", _f32),
        ("trainer", _i32), ("nes_pairs", _i32), ("nes_sigma", _f32),
        ("pop_size", _i32), ("elitism", _i32), ("bands", _i32),
    ]


def config_from_dict(d):
    """Build a lipz_config from a plain dict with the field names of the
    struct (layer widths as lists, activations as names)."""
    c = lipz_config()
    c.abi_version = LIPZ_ABI_VERSION
    c.rows, c.cols = d["rows"], d["cols"]
    c.net = LIPZ_NET_DCGAN if d.get("net", "mlp") == "dcgan" else LIPZ_NET_MLP
    c.z_dim, c.x_dim = d["z_dim"], d["x_dim"]
    img = d.get("img") or (0, 0, 0)
    c.img_h, c.img_w, c.img_c = img
    gh, dh = list(d["g_hidden"]), list(d["d_hidden"])
    if len(gh) > LIPZ_MAX_HIDDEN or len(dh) > LIPZ_MAX_HIDDEN:
        raise ValueError("at most %d hidden layers" % LIPZ_MAX_HIDDEN)
    c.n_g_hidden, c.n_d_hidden = len(gh), len(dh)
    for i, v in enumerate(gh):
        c.g_hidden[i] = v
    for i, v in enumerate(dh):
        c.d_hidden[i] = v
    c.g_hidden_act = ACTS[d["g_hidden_act"]]
    c.g_out_act = ACTS[d["g_out_act"]]
    c.d_hidden_act = ACTS[d["d_hidden_act"]]
    c.lrelu_slope = d["lrelu_slope"]
    c.batch = d["batch"]
    c.tournament_size = d["tournament_size"]
    c.fitness_mode = d["fitness_mode"]
    c.lr_mutation = d["lr_mutation"]
    c.lr0_g, c.lr0_d = d["lr0_g"], d["lr0_d"]
    c.beta1, c.beta2, c.eps = d["beta1"], d["beta2"], d["eps"]
    c.lr_mut_std, c.lr_mut_prob = d["lr_mut_std"], d["lr_mut_prob"]
    c.mix_enable = d["mix_enable"]
    c.mix_samples, c.mix_feat_dim, c.mix_sigma = d["mix_samples"], d["mix_feat_dim"], d["mix_sigma"]
    c.seed = d["seed"]
    c.loss_kind = LOSSES[d.get("loss", "bce")]
    c.wgan_clip = d.get("wgan_clip", 0.01)
    c.trainer = TRAINERS[d.get("trainer", "gradient")]
    c.nes_pairs = d.get("nes_pairs", 8)
    c.nes_sigma = d.get("nes_sigma", 0.01)
    c.pop_size = d.get("pop_size", 1)
    c.elitism = d.get("elitism", 0)
    c.bands = d.get("bands", 0)
    return c


_SIGS = {
    "lipz_workspace_bytes": (_sz, [ctypes.POINTER(lipz_config), _i64]),
    "lipz_grid_create": (_i32, [ctypes.POINTER(lipz_config), _vp, _sz, _vp, _i64, _vp,
                                ctypes.POINTER(_vp)]),
    "lipz_grid_create_static": (_i32, [ctypes.POINTER(lipz_config), _vp, _i64, _vp, ctypes.POINTER(_vp)]),
    "lipz_grid_destroy": (_i32, [_vp]),
    "lipz_eval_neighborhoods": (_i32, [_vp, _i32, _vp, _vp, _vp, _vp]),
    "lipz_select_replace": (_i32, [_vp, _i32, _vp, _vp, _vp]),
    "lipz_train_step": (_i32, [_vp, _i32, _i32, _i32, _vp]),
    "lipz_elitist_replace": (_i32, [_vp, _i32, _vp, _vp, _vp]),
    "lipz_run_generations": (_i32, [_vp, _i32, _i32, _i32]),
    "lipz_mixture_update": (_i32, [_vp, _i32, _vp, _vp, _vp]),
    "lipz_get_neighbors": (_i32, [_vp, ctypes.POINTER(_i32)]),
    "lipz_param_layout": (_i32, [_vp, _i32, ctypes.POINTER(_i64), ctypes.POINTER(_i32)]),
    "lipz_state_layout": (_i32, [_vp, ctypes.POINTER(_i64), ctypes.POINTER(_i64)]),
    "lipz_state_bytes": (_sz, [_vp]),
    "lipz_save_state": (_i32, [_vp, _vp]),
    "lipz_load_state": (_i32, [_vp, _vp]),
    "lipz_sync": (_i32, [_vp]),
    "lipz_error_string": (ctypes.c_char_p, [_i32]),
    "lipz_last_error": (ctypes.c_char_p, [_vp]),
    "lipz_set_gemm_timing": (_i32, [_vp, _i32]),
    "lipz_gemm_timing": (_i32, [_vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i64),
                                ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "lipz_test_plan_bounds": (_i32, [ctypes.POINTER(lipz_config), _i64, ctypes.c_char_p, _i32,
                                     ctypes.POINTER(_i32)]),
    "lipz_test_gemm": (_i32, [_vp, _vp, _i32, _i32, _i32, _vp, _i32, _i32, _i32, _vp, _i32, _i32,
                              _vp, _i32, _i32, _i32, _f32, _vp, _vp, _vp, _vp, _vp, _vp, _i32,
                              _f32, _f32, _f32, _i32, _i32]),
    "lipz_test_es_select": (_i32, [_vp, _vp, _vp, _vp, _i32, _i32, _i64, _i64, _f32]),
    "lipz_test_tile_map": (_i32, [_i32, _vp, _i32, _vp]),
}

_lib = None


def load_library(path=LIB_PATH):
    """Load liblipz.so and declare every exported function; raises if missing."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run `python -m paper_1811_12843_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in _SIGS.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib


class LipzError(RuntimeError):
    def __init__(self, status, where, detail=""):
        self.status = status
        msg = f"{where}: {lipz_error_string(status)} ({status})"
        if detail:
            msg += f": {detail}"
        super().__init__(msg)


def _check(status, where, grid=None):
    if status != LIPZ_OK:
        detail = lipz_last_error(grid) if grid else ""
        raise LipzError(status, where, detail)
    return status


def _p(x):
    return None if x is None or x == 0 else ctypes.c_void_p(int(x))


# ---- C ABI, same names ----

def lipz_workspace_bytes(cfg, n_samples):
    return load_library().lipz_workspace_bytes(ctypes.byref(cfg), n_samples)


def lipz_grid_create(cfg, d_workspace, workspace_bytes, d_dataset, n_samples, stream):
    out = _vp()
    st = load_library().lipz_grid_create(ctypes.byref(cfg), _p(d_workspace), workspace_bytes,
                                         _p(d_dataset), n_samples, _p(stream), ctypes.byref(out))
    _check(st, "lipz_grid_create")
    return out.value


def lipz_grid_create_static(cfg, d_dataset, n_samples, stream):
    """lipz_grid_create on the library's static per-device workspace (no device allocation)."""
    out = _vp()
    st = load_library().lipz_grid_create_static(ctypes.byref(cfg), _p(d_dataset), n_samples, _p(stream),
                                                ctypes.byref(out))
    _check(st, "lipz_grid_create_static")
    return out.value


def lipz_grid_destroy(g):
    return _check(load_library().lipz_grid_destroy(_p(g)), "lipz_grid_destroy")


def lipz_eval_neighborhoods(g, gen, d_L=None, d_Lg=None, d_fit_g=None, d_fit_d=None):
    return _check(load_library().lipz_eval_neighborhoods(_p(g), gen, _p(d_L), _p(d_Lg),
                                                         _p(d_fit_g), _p(d_fit_d)),
                  "lipz_eval_neighborhoods", g)


def lipz_select_replace(g, gen, d_forced=None, d_sel=None, d_lr=None):
    return _check(load_library().lipz_select_replace(_p(g), gen, _p(d_forced), _p(d_sel), _p(d_lr)),
                  "lipz_select_replace", g)


def lipz_train_step(g, gen, step0, n_steps, d_losses=None):
    return _check(load_library().lipz_train_step(_p(g), gen, step0, n_steps, _p(d_losses)),
                  "lipz_train_step", g)


def lipz_elitist_replace(g, gen, d_src=None, d_fit2_g=None, d_fit2_d=None):
    return _check(load_library().lipz_elitist_replace(_p(g), gen, _p(d_src), _p(d_fit2_g), _p(d_fit2_d)),
                  "lipz_elitist_replace", g)


def lipz_run_generations(g, gen0, n_gens, n_steps):
    return _check(load_library().lipz_run_generations(_p(g), gen0, n_gens, n_steps), "lipz_run_generations", g)


def lipz_mixture_update(g, gen, d_w=None, d_score=None, d_accepted=None):
    return _check(load_library().lipz_mixture_update(_p(g), gen, _p(d_w), _p(d_score),
                                                     _p(d_accepted)),
                  "lipz_mixture_update", g)


def lipz_get_neighbors(g, n_cells):
    buf = (_i32 * (5 * n_cells))()
    _check(load_library().lipz_get_neighbors(_p(g), buf), "lipz_get_neighbors", g)
    return [list(buf[5 * c:5 * c + 5]) for c in range(n_cells)]


def lipz_param_layout(g, role):
    n = _i32()
    offs = (_i64 * (3 * (LIPZ_MAX_HIDDEN + 1)))()
    _check(load_library().lipz_param_layout(_p(g), role, offs, ctypes.byref(n)), "lipz_param_layout", g)
    return [(offs[3 * l], offs[3 * l + 1], offs[3 * l + 2]) for l in range(n.value)]


def lipz_state_layout(g):
    offs = (_i64 * 12)()
    strides = (_i64 * 2)()
    _check(load_library().lipz_state_layout(_p(g), offs, strides), "lipz_state_layout", g)
    return list(offs), list(strides)


def lipz_state_bytes(g):
    return load_library().lipz_state_bytes(_p(g))


def lipz_save_state(g, d_dst):
    return _check(load_library().lipz_save_state(_p(g), _p(d_dst)), "lipz_save_state", g)


def lipz_load_state(g, d_src):
    return _check(load_library().lipz_load_state(_p(g), _p(d_src)), "lipz_load_state", g)


def lipz_sync(g):
    """Returns the status (does not raise for LIPZ_E_NONFINITE)."""
    st = load_library().lipz_sync(_p(g))
    if st not in (LIPZ_OK, LIPZ_E_NONFINITE):
        _check(st, "lipz_sync", g)
    return st


def lipz_error_string(status):
    return load_library().lipz_error_string(status).decode()


def lipz_last_error(g):
    r = load_library().lipz_last_error(_p(g))
    return r.decode() if r else ""


def lipz_set_gemm_timing(g, enable):
    return _check(load_library().lipz_set_gemm_timing(_p(g), int(bool(enable))), "lipz_set_gemm_timing", g)


def lipz_gemm_timing(g):
    """(milliseconds, launches, algorithmic FLOPs, algorithmic bytes) since the last call."""
    ms, n, fl, by = ctypes.c_double(), _i64(), ctypes.c_double(), ctypes.c_double()
    _check(load_library().lipz_gemm_timing(_p(g), ctypes.byref(ms), ctypes.byref(n), ctypes.byref(fl),
                                           ctypes.byref(by)),
           "lipz_gemm_timing", g)
    return ms.value, n.value, fl.value, by.value


def lipz_test_gemm(stream, d_desc, M, N, K, d_A, lda, a_trans, ones_row, d_B, ldb, b_trans, d_C, ldc,
                   epi, act, slope=0.2, d_bias=None, d_aux=None, d_m=None, d_v=None, d_lr=None,
                   d_t=None, step_local=0, beta1=0.9, beta2=0.999, eps=1e-8, tile_rows=0, variant=0):
    return _check(load_library().lipz_test_gemm(_p(stream), _p(d_desc), M, N, K, _p(d_A), lda, a_trans,
                                                ones_row, _p(d_B), ldb, b_trans, _p(d_C), ldc, epi, act,
                                                slope, _p(d_bias), _p(d_aux), _p(d_m), _p(d_v), _p(d_lr),
                                                _p(d_t), step_local, beta1, beta2, eps, tile_rows, variant),
                  "lipz_test_gemm")


def lipz_test_es_select(stream, d_fit, d_sets, d_params, n_units, n_pairs, P, stride, clip=0.0):
    return _check(load_library().lipz_test_es_select(_p(stream), _p(d_fit), _p(d_sets), _p(d_params), n_units,
                                                     n_pairs, P, stride, clip), "lipz_test_es_select")


def lipz_test_plan_bounds(cfg, n_samples):
    """(number of out-of-bounds accesses in the launch plan, message)."""
    buf = ctypes.create_string_buffer(4096)
    bad = _i32()
    _check(load_library().lipz_test_plan_bounds(ctypes.byref(cfg), n_samples, buf, 4096, ctypes.byref(bad)),
           "lipz_test_plan_bounds")
    return bad.value, buf.value.decode()


def lipz_test_tile_map(first_tile, n_blocks):
    """Logical tile of each block of a grouped GEMM launch (host only)."""
    ft = (_i32 * len(first_tile))(*first_tile)
    out = (_i32 * n_blocks)()
    _check(load_library().lipz_test_tile_map(len(first_tile), ft, n_blocks, out), "lipz_test_tile_map")
    return list(out)
