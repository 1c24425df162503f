"""Python binding of the TADM reverse-diffusion step for MI355X (gfx950).

Argument marshalling only: every function below forwards to the C ABI of
``libtadm.so`` (declared in ``include/tadm.h``) with the same name.  PyTorch is
used by callers for device memory and streams; tensors are passed by
``data_ptr()``.  Importing this package fails loudly when the library has not
been built: there is no fallback implementation.
"""
import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtadm.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                      "(or python paper_2609_37924_amd/csrc/build.py)")

lib = C.CDLL(LIB_PATH)

# ----------------------------------------------------------------- constants
TADM_OK, TADM_ERR_INVALID, TADM_ERR_OOM, TADM_ERR_DEVICE, TADM_ERR_STATE, TADM_ERR_UNSUPPORTED = range(6)
DTYPE = {"f32": 0, "bf16": 1}
FFN = {"gelu": 0, "swiglu": 1, "geglu": 2}
FUSION = {"gated_mlp": 0, "paired": 1}
CACHE_H, CACHE_C, CACHE_A = 0, 1, 2
TAP_EMBED, TAP_FUSED, TAP_FINAL, TAP_CHOICE, TAP_CONF = 0, 1, 2, 3, 4
STAGES = ["embed", "anchor", "fusion", "denoise", "head", "sample", "select", "context",
          "qkv", "attn", "oproj", "ffn_up", "ffn_down", "fusion1", "fusion2", "selfcond"]


class tadm_config(C.Structure):
    _fields_ = [(n, C.c_int32) for n in
                ("vocab", "d_model", "n_heads", "n_kv_heads", "head_dim", "d_ffn", "ffn_kind",
                 "n_shared", "n_anchor", "n_denoise", "fusion_kind", "fusion_rank", "paired_heads",
                 "dtype", "max_batch", "max_seq")] + [
        ("rms_eps", C.c_float), ("ln_eps", C.c_float), ("rope_theta", C.c_float)]


class tadm_step_args(C.Structure):
    _fields_ = [("i", C.c_int32), ("T", C.c_int32), ("n_unmask", C.c_int32),
                ("step_id", C.c_uint32), ("seed", C.c_uint64), ("inv_temp", C.c_float),
                ("n_unmask_rows", C.c_void_p), ("mode", C.c_int32), ("p_unmask", C.c_float),
                ("sigma", C.c_float), ("top_p", C.c_float), ("entropy_eta", C.c_float),
                ("sc_in", C.c_void_p), ("sc_out", C.c_void_p)]


class tadm_sampler(C.Structure):
    _fields_ = [("kind", C.c_int32), ("eta", C.c_float), ("top_p", C.c_float),
                ("t_on", C.c_double), ("t_off", C.c_double), ("alpha_on", C.c_double),
                ("tau_max", C.c_float), ("tau_min", C.c_float)]


STEP_RANKED, STEP_REMASK, STEP_ENTROPY = 0, 1, 2
SAMPLER_LOOP, SAMPLER_ENTROPY = 2, 3


class TadmError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"tadm status {status}: {msg}")
        self.status = status


_P = C.c_void_p
_I = C.c_int32
_SIGS = {
    "tadm_weight_count": (_I, [_P]),
    "tadm_weight_info": (_I, [_P, _I, C.POINTER(C.c_int64), C.POINTER(C.c_int64)]),
    "tadm_model_create": (_I, [_P, C.POINTER(_P)]),
    "tadm_model_load_weight": (_I, [_P, _I, _P, C.c_size_t, _I]),
    "tadm_model_destroy": (_I, [_P]),
    "tadm_set_stream": (_I, [_P, _P]),
    "tadm_cache_create": (_I, [_P, _I, _I, C.POINTER(_P)]),
    "tadm_cache_destroy": (_I, [_P]),
    "tadm_cache_read": (_I, [_P, _I, _P, C.c_size_t]),
    "tadm_cache_refresh_step": (_I, [_P]),
    "tadm_context_create": (_I, [_P, _I, _I, C.POINTER(_P)]),
    "tadm_context_append": (_I, [_P, _P, _P, _I, _I]),
    "tadm_context_length": (_I, [_P]),
    "tadm_context_reset": (_I, [_P]),
    "tadm_context_destroy": (_I, [_P]),
    "tadm_anchor_forward": (_I, [_P, _P, _P, _I, _I, _I, _I, _P]),
    "tadm_anchor_forward_sc": (_I, [_P, _P, _P, _I, _I, _I, _I, _P, _I, _P]),
    "tadm_entropy_inv_temp": (C.c_float, [_I, _I, C.c_float, C.c_float]),
    "tadm_train_loss": (_I, [_P, _P, _I, _I, _P, _P, C.c_float, C.c_uint64, C.c_uint32, _P, _P, _P, _P]),
    "tadm_stale_times": (None, [_I, C.c_uint64, C.c_uint32, C.c_float, _P, _P, _P, _P, _P]),
    "tadm_denoise_step": (_I, [_P, _P, _P, _I, _I, _I, _P, C.POINTER(tadm_step_args), _P, _P]),
    "tadm_sample": (_I, [_P, _P, _P, _I, _I, _I, _I, C.POINTER(tadm_step_args), _P, _P, _P]),
    "tadm_sample_noalloc": (_I, [_P, _P, _P, _I, _I, _I, _I, C.POINTER(tadm_step_args), _P, _P, _P]),
    "tadm_generate": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, C.c_uint64, C.c_float, _P]),
    "tadm_generate_sampler": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, C.c_uint64, C.c_float,
                                   C.POINTER(tadm_sampler), _P]),
    "tadm_unmask_count": (_I, [_I, _I, _I]),
    "tadm_remask_probs": (None, [_I, _I, C.c_float, C.POINTER(C.c_float), C.POINTER(C.c_float)]),
    "tadm_loop_probs": (None, [_I, _I, C.c_float, C.c_double, C.c_double, C.c_double, C.POINTER(C.c_float),
                               C.POINTER(C.c_float)]),
    "tadm_debug_read": (_I, [_P, _I, _P, C.c_size_t]),
    "tadm_debug_taps": (_I, [_P, _I]),
    "tadm_debug_layers": (_I, [_P, _P, C.c_size_t]),
    "tadm_context_read": (_I, [_P, _I, _P, _P, C.c_size_t]),
    "tadm_context_capacity": (_I, [_P]),
    "tadm_profile_enable": (_I, [_P, _I]),
    "tadm_profile_read": (_I, [_P, _I, C.POINTER(C.c_double), C.POINTER(C.c_int64)]),
    "tadm_profile_reset": (_I, [_P]),
    "tadm_last_error": (C.c_char_p, []),
}
for _name, (_res, _args) in _SIGS.items():
    _f = getattr(lib, _name)
    _f.restype, _f.argtypes = _res, _args

EXPORTED = sorted(_SIGS)
NOALLOC_MAX_POSITIONS = 65536  # TADM_NOALLOC_MAX_POSITIONS


def last_error():
    return lib.tadm_last_error().decode()


def check(status):
    if status != TADM_OK:
        raise TadmError(status, last_error())
    return status


def ptr(t):
    """Device pointer of a tensor (or None)."""
    return None if t is None else C.c_void_p(t.data_ptr())


# ------------------------------------------------------------------ config
def make_config(cfg, max_batch=None, max_seq=None):
    return tadm_config(
        vocab=cfg["vocab"], d_model=cfg["d_model"], n_heads=cfg["n_heads"],
        n_kv_heads=cfg["n_kv_heads"], head_dim=cfg["head_dim"], d_ffn=cfg["d_ffn"],
        ffn_kind=FFN[cfg["ffn_kind"]], n_shared=cfg["n_shared"], n_anchor=cfg["n_anchor"],
        n_denoise=cfg["n_denoise"], fusion_kind=FUSION[cfg["fusion_kind"]],
        fusion_rank=cfg.get("fusion_rank", 0), paired_heads=cfg.get("paired_heads", 4),
        dtype=DTYPE[cfg["dtype"]],
        max_batch=cfg["batch"] if max_batch is None else max_batch,
        max_seq=(cfg["prompt_len"] + cfg["gen_len"]) if max_seq is None else max_seq,
        rms_eps=cfg["rms_eps"], ln_eps=cfg["ln_eps"], rope_theta=cfg["rope_theta"])


# --------------------------------------------------------- thin wrappers
def tadm_weight_count(c):
    return lib.tadm_weight_count(C.byref(c))


def tadm_weight_info(c, index):
    r, k = C.c_int64(), C.c_int64()
    check(lib.tadm_weight_info(C.byref(c), index, C.byref(r), C.byref(k)))
    return r.value, k.value


def tadm_model_create(c):
    m = C.c_void_p()
    check(lib.tadm_model_create(C.byref(c), C.byref(m)))
    return m


def tadm_model_load_weight(m, index, tensor):
    on_dev = 1 if tensor.is_cuda else 0
    t = tensor.contiguous()
    check(lib.tadm_model_load_weight(m, index, C.c_void_p(t.data_ptr()),
                                     t.numel() * t.element_size(), on_dev))


def tadm_model_destroy(m):
    check(lib.tadm_model_destroy(m))


def tadm_set_stream(m, stream_ptr):
    check(lib.tadm_set_stream(m, C.c_void_p(stream_ptr)))


def tadm_cache_create(m, B, L):
    c = C.c_void_p()
    check(lib.tadm_cache_create(m, B, L, C.byref(c)))
    return c


def tadm_cache_destroy(c):
    check(lib.tadm_cache_destroy(c))


def tadm_cache_read(c, field, dst):
    check(lib.tadm_cache_read(c, field, ptr(dst), dst.numel() * dst.element_size()))


def tadm_cache_refresh_step(c):
    return lib.tadm_cache_refresh_step(c)


def tadm_context_create(m, B, max_ctx):
    c = C.c_void_p()
    check(lib.tadm_context_create(m, B, max_ctx, C.byref(c)))
    return c


def tadm_context_append(m, ctx, tokens, B, n):
    check(lib.tadm_context_append(m, ctx, ptr(tokens), B, n))


def tadm_context_length(ctx):
    return lib.tadm_context_length(ctx)


def tadm_context_reset(ctx):
    check(lib.tadm_context_reset(ctx))


def tadm_context_destroy(ctx):
    check(lib.tadm_context_destroy(ctx))


def tadm_anchor_forward(m, ctx, canvas, B, L, i, T, cache):
    check(lib.tadm_anchor_forward(m, ctx, ptr(canvas), B, L, i, T, cache))


def step_args(i, T, n_unmask, step_id, seed, inv_temp, n_unmask_rows=None, remask=None, top_p=0.0,
              entropy_eta=None, sc_in=None, sc_out=None):
    """n_unmask_rows: optional device int32 tensor [B] of per-row counts (kept alive by
    the caller until the step has run).  remask: optional (p_unmask, sigma) selecting the
    remasking posterior instead of confidence-ranked unmasking.  entropy_eta selects the
    entropy-bound step of the uniform-state sampler, with the optional self-conditioning
    tensors sc_in / sc_out (device float32 [B, Lc, d])."""
    a = tadm_step_args(i=i, T=T, n_unmask=n_unmask, step_id=step_id, seed=seed,
                       inv_temp=inv_temp, n_unmask_rows=ptr(n_unmask_rows), top_p=top_p)
    if remask is not None:
        a.mode, a.p_unmask, a.sigma = STEP_REMASK, remask[0], remask[1]
    if entropy_eta is not None:
        a.mode, a.entropy_eta, a.sc_in, a.sc_out = STEP_ENTROPY, entropy_eta, ptr(sc_in), ptr(sc_out)
    return a


def tadm_anchor_forward_sc(m, ctx, canvas, B, L, i, T, sc, canvas_off, cache):
    check(lib.tadm_anchor_forward_sc(m, ctx, ptr(canvas), B, L, i, T, ptr(sc), canvas_off, cache))


def tadm_entropy_inv_temp(n, T, tau_max, tau_min):
    return lib.tadm_entropy_inv_temp(n, T, tau_max, tau_min)


def tadm_train_loss(m, x, B, L, t, t_stale, eps, seed, step, loss, n_masked=None, zt=None, zs=None):
    """Training objective forward pass (device tensors: x int32 [B, L], t / t_stale /
    loss float32 [B], optional n_masked int32 [B], zt / zs int32 [B, L])."""
    check(lib.tadm_train_loss(m, ptr(x), B, L, ptr(t), ptr(t_stale), eps, seed, step, ptr(loss), ptr(n_masked),
                              ptr(zt), ptr(zs)))


def tadm_stale_times(B, seed, step, eps):
    """(t, t', K, T, k) of a training batch as numpy arrays, computed by the library."""
    import numpy as np
    t, ts = np.zeros(B, np.float32), np.zeros(B, np.float32)
    K, T, k = (np.zeros(B, np.int32) for _ in range(3))
    lib.tadm_stale_times(B, seed, step, eps, *(C.c_void_p(a.ctypes.data) for a in (t, ts, K, T, k)))
    return t, ts, K, T, k


def tadm_denoise_step(m, ctx, canvas, B, L, canvas_off, cache, args, logits, next_canvas):
    check(lib.tadm_denoise_step(m, ctx, ptr(canvas), B, L, canvas_off, cache, C.byref(args),
                                ptr(logits), ptr(next_canvas)))


def tadm_sample(m, logits, canvas, B, L, canvas_off, pos0, args, next_canvas, choice=None, conf=None):
    check(lib.tadm_sample(m, ptr(logits), ptr(canvas), B, L, canvas_off, pos0, C.byref(args),
                          ptr(next_canvas), ptr(choice), ptr(conf)))


def tadm_sample_noalloc(m, logits, canvas, B, L, canvas_off, pos0, args, next_canvas, choice=None, conf=None):
    check(lib.tadm_sample_noalloc(m, ptr(logits), ptr(canvas), B, L, canvas_off, pos0, C.byref(args),
                                  ptr(next_canvas), ptr(choice), ptr(conf)))


def tadm_generate(m, prompt, B, P, gen_len, T, K, block_len, seed, temperature, tokens):
    check(lib.tadm_generate(m, ptr(prompt), B, P, gen_len, T, K, block_len, seed, temperature,
                            ptr(tokens)))


def tadm_generate_sampler(m, prompt, B, P, gen_len, T, K, block_len, seed, temperature, sampler, tokens):
    """sampler: None (confidence-ranked) or a tadm_sampler."""
    check(lib.tadm_generate_sampler(m, ptr(prompt), B, P, gen_len, T, K, block_len, seed, temperature,
                                    C.byref(sampler) if sampler is not None else None, ptr(tokens)))


def remask_sampler(eta, top_p=0.0):
    return tadm_sampler(kind=STEP_REMASK, eta=eta, top_p=top_p)


def entropy_sampler(eta=0.1, tau_max=0.8, tau_min=0.4):
    """Entropy-bound sampler of uniform-state diffusion (defaults: the paper's settings)."""
    return tadm_sampler(kind=SAMPLER_ENTROPY, eta=eta, tau_max=tau_max, tau_min=tau_min)


def loop_sampler(eta=0.02, t_on=0.55, t_off=0.05, alpha_on=0.9, top_p=0.0):
    """ReMDM-Loop remasking sampler (defaults: the paper's settings for T >= L)."""
    return tadm_sampler(kind=SAMPLER_LOOP, eta=eta, top_p=top_p, t_on=t_on, t_off=t_off, alpha_on=alpha_on)


def tadm_unmask_count(M0, i, T):
    return lib.tadm_unmask_count(M0, i, T)


def tadm_remask_probs(i, T, eta):
    """(sigma, p_unmask) as float32 values computed by the library."""
    sg, pu = C.c_float(), C.c_float()
    lib.tadm_remask_probs(i, T, eta, C.byref(sg), C.byref(pu))
    return sg.value, pu.value


def tadm_loop_probs(i, T, eta, t_on, t_off, alpha_on):
    """(sigma, p_unmask) of the ReMDM-Loop schedule as float32 values computed by the library."""
    sg, pu = C.c_float(), C.c_float()
    lib.tadm_loop_probs(i, T, eta, t_on, t_off, alpha_on, C.byref(sg), C.byref(pu))
    return sg.value, pu.value


def tadm_debug_read(m, tap, dst):
    check(lib.tadm_debug_read(m, tap, ptr(dst), dst.numel() * 4))


def tadm_debug_taps(m, enable):
    check(lib.tadm_debug_taps(m, int(enable)))


def tadm_profile_enable(m, stage_mask):
    """stage_mask: bit s records stage s (STAGES order); -1 records all, 0 none."""
    check(lib.tadm_profile_enable(m, int(stage_mask)))


def tadm_profile_reset(m):
    check(lib.tadm_profile_reset(m))


def tadm_profile_read(m, stage):
    ms, n = C.c_double(), C.c_int64()
    check(lib.tadm_profile_read(m, stage, C.byref(ms), C.byref(n)))
    return ms.value, n.value


# ------------------------------------------------------- model construction
def load_model(cfg, tensors, max_batch=None, max_seq=None, stream=None):
    """Create a model for the config dict ``cfg`` and upload ``tensors`` (ABI order).

    ``stream`` is a hipStream_t as an int (e.g. torch.cuda.current_stream().cuda_stream).
    """
    c = make_config(cfg, max_batch, max_seq)
    n = tadm_weight_count(c)
    if n != len(tensors):
        raise ValueError(f"config needs {n} tensors, got {len(tensors)}")
    m = tadm_model_create(c)
    try:
        for i, t in enumerate(tensors):
            tadm_model_load_weight(m, i, t)
        if stream is not None:
            tadm_set_stream(m, stream)
    except Exception:
        tadm_model_destroy(m)
        raise
    return m


def tadm_debug_layers(m, dst):
    """dst: device float32 tensor of 2 * n_layers slots [B, L, d] (None turns capture off)."""
    check(lib.tadm_debug_layers(m, ptr(dst), 0 if dst is None else dst.numel() * 4))


def tadm_context_read(ctx, layer, k, vt):
    check(lib.tadm_context_read(ctx, layer, ptr(k), ptr(vt), k.numel() * k.element_size()))


def tadm_context_capacity(ctx):
    return lib.tadm_context_capacity(ctx)
