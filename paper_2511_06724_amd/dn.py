"""ctypes binding of ``libargus_dn.so`` (the C ABI in include/argus_dn.h).

Argument marshalling only: every step of the denoise loop and of the cache
lookup runs in the library's HIP kernels. PyTorch tensors serve as device
buffers (``data_ptr()``) and PyTorch streams as HIP streams. Importing this
module raises if the library has not been built: there is no fallback.
"""

import ctypes as C
import os

import numpy as np

from .workloads import DnConfig, VaeConfig

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libargus_dn.so")

DN_OK, DN_EINVAL, DN_ENOMEM, DN_EHIP, DN_EUNSUPPORTED = 0, -1, -2, -3, -4
DN_FP32, DN_BF16, DN_FP8 = 0, 1, 2
DN_WEIGHTS_HOST, DN_WEIGHTS_DEVICE = 0, 1
ABI_VERSION = 1
MAX_LEVELS = 4

EXPORTED = ("dn_weight_count", "dn_weight_table", "dn_create", "dn_denoise", "dn_denoise_capture", "dn_unet_eps", "ac_lookup",
            "ac_lookup_batch", "ac_lookup_batch_k", "ac_lookup_batch_noalloc", "ac_fetch_latent", "dn_packed_weight_elems", "dn_pack_weight", "dn_op_linear", "dn_op_conv3x3",
            "dn_op_attention", "dn_op_groupnorm", "dn_op_layernorm", "dn_op_layernorm_slabs", "dn_op_linear_vt",
            "dn_probe_mfma_rate",
            "dn_destroy", "dn_last_error", "dn_vae_weight_count", "dn_vae_weight_table", "dn_vae_create",
            "dn_vae_decode", "dn_vae_destroy", "argus_oda", "argus_route", "argus_select_worker", "argus_last_error")


AC_MAX_K_LEVELS = 16


class _KTable(C.Structure):
    _fields_ = [("n_thresholds", C.c_int32), ("threshold", C.c_float * (AC_MAX_K_LEVELS - 1)),
                ("level", C.c_int32 * AC_MAX_K_LEVELS)]


class DnError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"[{code}] {msg}")
        self.code = code


class _Level(C.Structure):
    _fields_ = [("channels", C.c_int32), ("depth", C.c_int32), ("heads", C.c_int32), ("head_dim", C.c_int32)]


class _Config(C.Structure):
    _fields_ = [
        ("abi_version", C.c_int32), ("dtype", C.c_int32), ("batch", C.c_int32),
        ("latent_c", C.c_int32), ("latent_h", C.c_int32), ("latent_w", C.c_int32),
        ("model_channels", C.c_int32), ("n_levels", C.c_int32), ("level", _Level * MAX_LEVELS),
        ("layers_per_block", C.c_int32), ("mid_depth", C.c_int32), ("tiny_topology", C.c_int32),
        ("ctx_len", C.c_int32), ("ctx_dim", C.c_int32), ("ff_mult", C.c_int32), ("gn_groups", C.c_int32),
        ("gn_eps", C.c_float), ("tx_gn_eps", C.c_float), ("ln_eps", C.c_float),
        ("n_train_steps", C.c_int32), ("beta_start", C.c_float), ("beta_end", C.c_float),
        ("beta_schedule", C.c_int32),
    ]


class _VaeConfig(C.Structure):
    _fields_ = [
        ("abi_version", C.c_int32), ("dtype", C.c_int32), ("batch", C.c_int32),
        ("latent_c", C.c_int32), ("latent_h", C.c_int32), ("latent_w", C.c_int32),
        ("n_levels", C.c_int32), ("channels", C.c_int32 * MAX_LEVELS), ("layers_per_block", C.c_int32),
        ("gn_groups", C.c_int32), ("gn_eps", C.c_float), ("scaling_factor", C.c_float), ("out_c", C.c_int32),
    ]


def _load():
    # One HIP runtime per process: PyTorch bundles its own libamdhip64 with the
    # same soname as ROCm's. Importing torch first makes the library bind to that
    # already-loaded runtime, so torch's streams and allocations are the library's.
    import torch  # noqa: F401
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is missing: build it with __graft_entry__.build() "
                          "(python -c 'import __graft_entry__ as g; g.build()')")
    lib = C.CDLL(_LIB_PATH)
    P, I32, I64, F32, SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_size_t
    sig = {
        "dn_weight_count": [C.POINTER(_Config), C.POINTER(SZ)],
        "dn_weight_table": [C.POINTER(_Config), P, P, P, SZ, C.POINTER(SZ)],
        "dn_create": [C.POINTER(_Config), P, SZ, I32, C.POINTER(P)],
        "dn_denoise": [P, P, P, P, I32, I32, I32, F32, P],
        "dn_denoise_capture": [P, P, P, P, I32, I32, I32, F32, P, I32, P, P],
        "dn_unet_eps": [P, P, I32, P, F32, P, P, P],
        "ac_lookup": [P, P, I64, I32, C.POINTER(I64), C.POINTER(F32)],
        "ac_lookup_batch": [P, I32, P, I64, I32, C.POINTER(I64), C.POINTER(F32)],
        "ac_lookup_batch_k": [P, I32, P, I64, I32, C.POINTER(_KTable), P, P, P],
        "ac_lookup_batch_noalloc": [P, I32, P, I64, I32, P, P, P],
        "ac_fetch_latent": [P, I64, I64, I64, P, P],
        "dn_packed_weight_elems": [I32, I32, I32, C.POINTER(I64)],
        "dn_pack_weight": [I32, P, I32, I32, P, P],
        "dn_op_linear": [I32, P, P, P, P, I32, P, I32, I64, I32, I32, I32, P],
        "dn_op_conv3x3": [I32, P, I32, I32, I32, I32, I32, I32, P, P, P, P, P, I32, I32, P],
        "dn_op_attention": [I32, P, I32, P, I32, P, I32, P, I32, I32, I32, I32, I32, I32, F32, P],
        "dn_op_linear_vt": [I32, P, P, P, P, I64, I32, I32, I32, P, I32, I32, I32, I32, P],
        "dn_op_groupnorm": [I32, P, P, I32, I32, I32, I32, P, P, F32, I32, P],
        "dn_op_layernorm": [I32, P, P, I64, I32, P, P, F32, P],
        "dn_op_layernorm_slabs": [I32, P, P, I64, I32, P, P, F32, P, I32, P, I32, P],
        "dn_probe_mfma_rate": [I32, C.POINTER(C.c_double), C.POINTER(C.c_double)],
        "argus_oda": [P, P, I32, P],
        "argus_route": [P, I32, I32, C.c_double, C.POINTER(I32)],
        "argus_select_worker": [P, P, P, I32, I32, C.POINTER(I32)],
        "argus_last_error": [],
        "dn_vae_weight_count": [C.POINTER(_VaeConfig), C.POINTER(SZ)],
        "dn_vae_weight_table": [C.POINTER(_VaeConfig), P, P, P, SZ, C.POINTER(SZ)],
        "dn_vae_create": [C.POINTER(_VaeConfig), P, SZ, I32, C.POINTER(P)],
        "dn_vae_decode": [P, P, P, P],
        "dn_vae_destroy": [P],
        "dn_destroy": [P],
        "dn_last_error": [],
    }
    for name, args in sig.items():
        f = getattr(lib, name)
        f.argtypes = args
        f.restype = C.c_int
    lib.dn_destroy.restype = None
    lib.dn_vae_destroy.restype = None
    lib.dn_last_error.restype = C.c_char_p
    lib.argus_last_error.restype = C.c_char_p
    return lib


lib = _load()


def _check(code):
    if code != DN_OK:
        raise DnError(code, lib.dn_last_error().decode())


def _ptr(t):
    """Device (or host numpy) address of a buffer; None -> NULL."""
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        return t.ctypes.data
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def to_c_config(cfg: DnConfig) -> _Config:
    c = _Config()
    c.abi_version = ABI_VERSION
    c.dtype = cfg.dtype
    c.batch = cfg.batch
    c.latent_c, c.latent_h, c.latent_w = cfg.latent_c, cfg.latent_h, cfg.latent_w
    c.model_channels = cfg.model_channels
    c.n_levels = len(cfg.levels)
    for i, lv in enumerate(cfg.levels):
        c.level[i] = _Level(*lv)
    c.layers_per_block = cfg.layers_per_block
    c.mid_depth = cfg.mid_depth
    c.tiny_topology = cfg.tiny_topology
    c.ctx_len, c.ctx_dim, c.ff_mult, c.gn_groups = cfg.ctx_len, cfg.ctx_dim, cfg.ff_mult, cfg.gn_groups
    c.gn_eps, c.tx_gn_eps, c.ln_eps = cfg.gn_eps, cfg.tx_gn_eps, cfg.ln_eps
    c.n_train_steps = cfg.n_train_steps
    c.beta_start, c.beta_end = cfg.beta_start, cfg.beta_end
    c.beta_schedule = cfg.beta_schedule
    return c


def weight_count(cfg):
    n = C.c_size_t()
    _check(lib.dn_weight_count(C.byref(to_c_config(cfg)), C.byref(n)))
    return n.value


def weight_table(cfg):
    """[(numel, fan_in, kind)] with kind as in the C header (0 w, 1 b, 2 scale, 3 shift)."""
    c = to_c_config(cfg)
    n = C.c_size_t()
    _check(lib.dn_weight_table(C.byref(c), None, None, None, 0, C.byref(n)))
    numel = np.zeros(n.value, np.int64)
    fan = np.zeros(n.value, np.int32)
    kind = np.zeros(n.value, np.int32)
    _check(lib.dn_weight_table(C.byref(c), numel.ctypes.data, fan.ctypes.data, kind.ctypes.data, n.value,
                               C.byref(n)))
    return list(zip(numel.tolist(), fan.tolist(), kind.tolist()))


class Denoiser:
    """Owns a dn_handle. ``weights``: fp32 numpy array (host) or CUDA tensor (device)."""

    def __init__(self, cfg: DnConfig, weights):
        self.cfg = cfg
        self._h = C.c_void_p()
        on_dev = not isinstance(weights, np.ndarray)
        if on_dev:
            n = weights.numel()
        else:
            weights = np.ascontiguousarray(weights, dtype=np.float32)
            n = weights.size
        _check(lib.dn_create(C.byref(to_c_config(cfg)), _ptr(weights), n,
                             DN_WEIGHTS_DEVICE if on_dev else DN_WEIGHTS_HOST, C.byref(self._h)))

    def close(self):
        if self._h:
            lib.dn_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def denoise(self, latent, text_ctx, timesteps, start_step, n_steps, cfg_scale, stream=None):
        ts = np.ascontiguousarray(timesteps, dtype=np.int32)
        _check(lib.dn_denoise(self._h, _ptr(latent), _ptr(text_ctx), ts.ctypes.data, ts.size, start_step, n_steps,
                              cfg_scale, _stream(stream)))

    def denoise_capture(self, latent, text_ctx, timesteps, start_step, n_steps, cfg_scale, capture_at, out_latents,
                        stream=None):
        """dn_denoise that also writes the latent after each iteration count in capture_at
        (bf16) to out_latents [len(capture_at), B, C, H, W] (a bf16 CUDA tensor)."""
        ts = np.ascontiguousarray(timesteps, dtype=np.int32)
        cap = np.ascontiguousarray(capture_at, dtype=np.int32)
        _check(lib.dn_denoise_capture(self._h, _ptr(latent), _ptr(text_ctx), ts.ctypes.data, ts.size, start_step,
                                      n_steps, cfg_scale, cap.ctypes.data if cap.size else None, cap.size,
                                      _ptr(out_latents), _stream(stream)))

    def unet_eps(self, x, t, text_ctx, cfg_scale, out_raw, out_guided=None, stream=None):
        _check(lib.dn_unet_eps(self._h, _ptr(x), int(t), _ptr(text_ctx), cfg_scale, _ptr(out_raw),
                               _ptr(out_guided), _stream(stream)))


def to_c_vae_config(cfg: VaeConfig) -> _VaeConfig:
    c = _VaeConfig()
    c.abi_version = ABI_VERSION
    c.dtype, c.batch = cfg.dtype, cfg.batch
    c.latent_c, c.latent_h, c.latent_w = cfg.latent_c, cfg.latent_h, cfg.latent_w
    c.n_levels = len(cfg.block_channels)
    for i, ch in enumerate(cfg.block_channels):
        c.channels[i] = ch
    c.layers_per_block, c.gn_groups, c.gn_eps = cfg.layers_per_block, cfg.gn_groups, cfg.gn_eps
    c.scaling_factor, c.out_c = cfg.scaling_factor, cfg.out_c
    return c


def vae_weight_table(cfg):
    """[(numel, fan_in, kind)] of the decoder's canonical blob."""
    c = to_c_vae_config(cfg)
    n = C.c_size_t()
    _check(lib.dn_vae_weight_table(C.byref(c), None, None, None, 0, C.byref(n)))
    numel = np.zeros(n.value, np.int64)
    fan = np.zeros(n.value, np.int32)
    kind = np.zeros(n.value, np.int32)
    _check(lib.dn_vae_weight_table(C.byref(c), numel.ctypes.data, fan.ctypes.data, kind.ctypes.data, n.value,
                                   C.byref(n)))
    return list(zip(numel.tolist(), fan.tolist(), kind.tolist()))


class Decoder:
    """Owns a dn_vae. ``weights``: fp32 numpy array (host) or CUDA tensor (device)."""

    def __init__(self, cfg: VaeConfig, weights):
        self.cfg = cfg
        self._h = C.c_void_p()
        on_dev = not isinstance(weights, np.ndarray)
        if on_dev:
            n = weights.numel()
        else:
            weights = np.ascontiguousarray(weights, dtype=np.float32)
            n = weights.size
        _check(lib.dn_vae_create(C.byref(to_c_vae_config(cfg)), _ptr(weights), n,
                                 DN_WEIGHTS_DEVICE if on_dev else DN_WEIGHTS_HOST, C.byref(self._h)))

    def decode(self, latent, image, stream=None):
        _check(lib.dn_vae_decode(self._h, _ptr(latent), _ptr(image), _stream(stream)))

    def close(self):
        if self._h:
            lib.dn_vae_destroy(self._h)
            self._h = C.c_void_p()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def ac_lookup(query, cache):
    """(index, cosine) of the nearest cache row; query [dim], cache [n, dim] fp16 CUDA tensors."""
    idx = C.c_int64(-7)
    score = C.c_float()
    n, dim = (cache.shape[0], cache.shape[1]) if cache.dim() == 2 else (cache.shape[0], 1)
    _check(lib.ac_lookup(_ptr(query), _ptr(cache), n, dim, C.byref(idx), C.byref(score)))
    return idx.value, score.value


def ac_lookup_raw(query_ptr, cache_ptr, n, dim):
    idx = C.c_int64(-7)
    score = C.c_float()
    code = lib.ac_lookup(query_ptr, cache_ptr, n, dim, C.byref(idx), C.byref(score))
    return code, idx.value, score.value


def ac_lookup_batch(queries, cache):
    """(indices, cosines) of the nearest cache row for every query: queries [nq, dim],
    cache [n, dim] fp16 CUDA tensors. Lists of length nq; index -1 for a zero query."""
    nq, dim = queries.shape
    n = cache.shape[0]
    if cache.shape[1] != dim:
        raise ValueError("ac_lookup_batch: query and cache widths differ")
    idx = (C.c_int64 * nq)()
    score = (C.c_float * nq)()
    _check(lib.ac_lookup_batch(_ptr(queries), nq, _ptr(cache), n, dim, idx, score))
    return list(idx), list(score)


def k_table(thresholds, levels):
    """ac_k_table from thresholds [L] and levels [L + 1] (no checks: the library checks)."""
    t = _KTable()
    t.n_thresholds = len(thresholds)
    for i, v in enumerate(thresholds):
        t.threshold[i] = v
    for i, v in enumerate(levels):
        t.level[i] = v
    return t


def ac_lookup_batch_k(queries, cache, thresholds, levels):
    """(indices, cosines, levels K) for every query: ac_lookup_batch plus the approximation
    level chosen from the retrieved cosine by the threshold table (thresholds [L],
    levels [L + 1])."""
    nq, dim = queries.shape
    if cache.shape[1] != dim:
        raise ValueError("ac_lookup_batch_k: query and cache widths differ")
    if len(thresholds) >= AC_MAX_K_LEVELS or len(levels) > AC_MAX_K_LEVELS:
        raise ValueError("ac_lookup_batch_k: at most 15 thresholds")
    idx = (C.c_int64 * nq)()
    score = (C.c_float * nq)()
    k = (C.c_int32 * nq)()
    tab = k_table(thresholds, levels)
    _check(lib.ac_lookup_batch_k(_ptr(queries), nq, _ptr(cache), cache.shape[0], dim, C.byref(tab), idx, score, k))
    return list(idx), list(score), list(k)


def ac_lookup_batch_noalloc(queries, cache, out_idx, out_score=None, stream=None):
    """ac_lookup_batch on a stream with device outputs and no allocation in the library:
    queries [nq, dim], cache [n, dim] fp16 CUDA tensors; out_idx int64 [nq] and out_score
    float32 [nq] (or None) CUDA tensors receive the results."""
    nq, dim = queries.shape
    if cache.shape[1] != dim:
        raise ValueError("ac_lookup_batch_noalloc: query and cache widths differ")
    _check(lib.ac_lookup_batch_noalloc(_ptr(queries), nq, _ptr(cache), cache.shape[0], dim, _ptr(out_idx),
                                       _ptr(out_score), _stream(stream)))


def ac_fetch_latent(cache_latents, idx, latent, stream=None):
    n = cache_latents.shape[0]
    numel = cache_latents[0].numel()
    _check(lib.ac_fetch_latent(_ptr(cache_latents), n, numel, idx, _ptr(latent), _stream(stream)))


def packed_weight_elems(dtype, N, K):
    n = C.c_int64()
    _check(lib.dn_packed_weight_elems(dtype, N, K, C.byref(n)))
    return n.value


def pack_weight(dtype, w, N, K, stream=None):
    """Row-major device weight [N][K] (dtype elements; fp32 for DN_FP8) -> a new tensor in
    the GEMM's packed layout (for DN_FP8 a uint8 tensor: codes, then N fp32 scales)."""
    import torch
    out = torch.empty(packed_weight_elems(dtype, N, K), device=w.device,
                      dtype=torch.uint8 if dtype == DN_FP8 else w.dtype)
    _check(lib.dn_pack_weight(dtype, _ptr(w), N, K, _ptr(out), _stream(stream)))
    return out


def op_linear(dtype, x, w, bias, y, M, N, K, resid=None, resid_f32=False, y_f32=False, geglu=False, stream=None):
    _check(lib.dn_op_linear(dtype, _ptr(x), _ptr(w), _ptr(bias), _ptr(resid), int(resid_f32), _ptr(y), int(y_f32),
                            M, N, K, int(geglu), _stream(stream)))


def op_conv3x3(dtype, x, n, H, W, Cin, w, bias, y, Cout, up=0, stride=1, temb=None, resid=None, y_f32=False,
               stream=None):
    _check(lib.dn_op_conv3x3(dtype, _ptr(x), n, H, W, Cin, up, stride, _ptr(w), _ptr(bias), _ptr(temb),
                             _ptr(resid), _ptr(y), Cout, int(y_f32), _stream(stream)))


def op_attention(dtype, q, ldq, k, ldk, vt, vt_ld, o, ldo, B, heads, Sq, Skv, head_stride, scale, stream=None):
    _check(lib.dn_op_attention(dtype, _ptr(q), ldq, _ptr(k), ldk, _ptr(vt), vt_ld, _ptr(o), ldo, B, heads, Sq, Skv,
                               head_stride, scale, _stream(stream)))


def op_linear_vt(dtype, x, w, bias, y, M, N, K, vt_col0, vt, heads, head_stride, seq, vt_ld, stream=None):
    _check(lib.dn_op_linear_vt(dtype, _ptr(x), _ptr(w), _ptr(bias), _ptr(y), M, N, K, vt_col0, _ptr(vt), heads,
                               head_stride, seq, vt_ld, _stream(stream)))


def op_groupnorm(dtype, x, y, n, HW, Cc, G, gamma, beta, eps, silu, stream=None):
    _check(lib.dn_op_groupnorm(dtype, _ptr(x), _ptr(y), n, HW, Cc, G, _ptr(gamma), _ptr(beta), eps, int(silu),
                               _stream(stream)))


def op_layernorm(dtype, x, y, M, Cc, gamma, beta, eps, stream=None):
    _check(lib.dn_op_layernorm(dtype, _ptr(x), _ptr(y), M, Cc, _ptr(gamma), _ptr(beta), eps, _stream(stream)))


def op_layernorm_slabs(dtype, x, y, M, Cc, gamma, beta, eps, slabs, nsplit, bias=None, resid=True, stream=None):
    _check(lib.dn_op_layernorm_slabs(dtype, _ptr(x), _ptr(y), M, Cc, _ptr(gamma), _ptr(beta), eps, _ptr(slabs), nsplit,
                                     _ptr(bias), int(resid), _stream(stream)))


def probe_mfma_rate(iters=4000):
    """(TFLOP/s, GHz): the bf16 matrix-core rate the device sustains and its clock
    meanwhile (dn_probe_mfma_rate; a measurement, not a step of the method)."""
    tf, ghz = C.c_double(0.0), C.c_double(0.0)
    _check(lib.dn_probe_mfma_rate(iters, C.byref(tf), C.byref(ghz)))
    return tf.value, ghz.value


# ----------------------------------------------------------------------------- routing control plane (host)

def _check_ctl(code):
    if code != DN_OK:
        raise DnError(code, lib.argus_last_error().decode())


def oda(H, F):
    """PASM [n, n] (numpy fp64) from the demand histogram H and the load split F."""
    H = np.ascontiguousarray(H, dtype=np.float64)
    F = np.ascontiguousarray(F, dtype=np.float64)
    if H.shape != F.shape or H.ndim != 1:
        raise ValueError("oda: H and F must be 1-D of the same length")
    out = np.zeros((H.size, H.size), np.float64)
    _check_ctl(lib.argus_oda(H.ctypes.data, F.ctypes.data, H.size, out.ctypes.data))
    return out


def route(pasm, level, u):
    pasm = np.ascontiguousarray(pasm, dtype=np.float64)
    out = C.c_int32()
    _check_ctl(lib.argus_route(pasm.ctypes.data, pasm.shape[0], level, u, C.byref(out)))
    return out.value


def select_worker(queue_len, t_proc, worker_level, level):
    q = np.ascontiguousarray(queue_len, dtype=np.int32)
    t = np.ascontiguousarray(t_proc, dtype=np.float64)
    lv = np.ascontiguousarray(worker_level, dtype=np.int32)
    out = C.c_int32()
    _check_ctl(lib.argus_select_worker(q.ctypes.data, t.ctypes.data, lv.ctypes.data, q.size, level, C.byref(out)))
    return out.value
