"""ctypes binding of the synerdiff C ABI (argument marshalling only).

Device buffers are torch tensors on the current HIP device; streams are
torch streams.  Every computation runs in libsynerdiff.so.
"""
import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsynerdiff.so")
_LIB = None

SD_F32, SD_BF16 = 0, 1
SCHEDULES = {"linear": 0, "scaled_linear": 1}
STATUS = {0: "SD_OK", -1: "SD_ERR_INVALID_ARG", -2: "SD_ERR_UNSUPPORTED", -3: "SD_ERR_CAPACITY",
          -4: "SD_ERR_WORKSPACE", -5: "SD_ERR_HIP"}


class SynerDiffError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class UNetConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("latent_c", "latent_h", "latent_w", "n_levels")] + \
               [("ch", ctypes.c_int32 * 4), ("n_res", ctypes.c_int32), ("tx_depth", ctypes.c_int32 * 4)] + \
               [(n, ctypes.c_int32) for n in ("mid_tx_depth", "heads", "head_dim", "gn_groups", "ctx_len",
                                               "ctx_dim", "temb_in", "temb_dim", "add_in", "pooled_dim",
                                               "time_id_dim", "n_time_ids", "max_requests", "dtype")]


class KernelStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 24), ("launches", ctypes.c_int64), ("ms", ctypes.c_double),
                ("flop", ctypes.c_double), ("bytes", ctypes.c_double)]


class LayerStat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 64), ("launches", ctypes.c_int64), ("ms", ctypes.c_double),
                ("flop", ctypes.c_double), ("bytes", ctypes.c_double)]


class VAEConfig(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("latent_c", "latent_h", "latent_w", "n_levels")] + \
               [("ch", ctypes.c_int32 * 4)] + \
               [(n, ctypes.c_int32) for n in ("n_res", "gn_groups", "out_c", "max_images", "dtype")] + \
               [("scaling", ctypes.c_float)]


_P = ctypes.c_void_p
_SIG = {
    "synerdiff_abi_version": (ctypes.c_int32, []),
    "synerdiff_last_error": (ctypes.c_char_p, []),
    "synerdiff_config_check": (ctypes.c_int, [ctypes.POINTER(UNetConfig)]),
    "synerdiff_param_count": (ctypes.c_int64, [ctypes.POINTER(UNetConfig)]),
    "synerdiff_param_info": (ctypes.c_int, [ctypes.POINTER(UNetConfig), ctypes.c_int64, ctypes.c_char_p,
                                            ctypes.c_size_t, ctypes.POINTER(ctypes.c_int64),
                                            ctypes.POINTER(ctypes.c_int32)]),
    "synerdiff_weights_bytes": (ctypes.c_size_t, [ctypes.POINTER(UNetConfig)]),
    "synerdiff_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(UNetConfig)]),
    "synerdiff_unet_create": (ctypes.c_int, [ctypes.POINTER(UNetConfig), _P, ctypes.c_size_t, _P,
                                             ctypes.c_size_t, ctypes.POINTER(_P)]),
    "synerdiff_load_weights": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P]),
    "synerdiff_unet_step": (ctypes.c_int, [_P, ctypes.c_int32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P,
                                           _P, _P]),
    "synerdiff_row_plan": (ctypes.c_int, [ctypes.c_int32, _P, _P, _P, _P, _P]),
    "synerdiff_alphas_cumprod": (ctypes.c_int, [ctypes.c_int32, _P]),
    "synerdiff_ddim_coef": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P]),
    "synerdiff_unet_destroy": (None, [_P]),
    "synerdiff_ddim_coef_v": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P]),
    "synerdiff_unet_create_shared": (ctypes.c_int, [ctypes.POINTER(UNetConfig), _P, _P, ctypes.c_size_t,
                                                    ctypes.POINTER(_P)]),
    "synerdiff_profile": (ctypes.c_int, [_P, ctypes.c_int32]),
    "synerdiff_profile_read": (ctypes.c_int, [_P, ctypes.POINTER(KernelStat), ctypes.c_int32,
                                              ctypes.POINTER(ctypes.c_int32), ctypes.c_int32]),
    "synerdiff_profile_read_layers": (ctypes.c_int, [_P, ctypes.POINTER(LayerStat), ctypes.c_int32,
                                                     ctypes.POINTER(ctypes.c_int32), ctypes.c_int32]),
    "synerdiff_vae_config_check": (ctypes.c_int, [ctypes.POINTER(VAEConfig)]),
    "synerdiff_vae_param_count": (ctypes.c_int64, [ctypes.POINTER(VAEConfig)]),
    "synerdiff_vae_param_info": (ctypes.c_int, [ctypes.POINTER(VAEConfig), ctypes.c_int64, ctypes.c_char_p,
                                                ctypes.c_size_t, ctypes.POINTER(ctypes.c_int64),
                                                ctypes.POINTER(ctypes.c_int32)]),
    "synerdiff_vae_weights_bytes": (ctypes.c_size_t, [ctypes.POINTER(VAEConfig)]),
    "synerdiff_vae_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(VAEConfig)]),
    "synerdiff_vae_create": (ctypes.c_int, [ctypes.POINTER(VAEConfig), _P, ctypes.c_size_t, _P, ctypes.c_size_t,
                                            ctypes.POINTER(_P)]),
    "synerdiff_vae_load_weights": (ctypes.c_int, [_P, _P, ctypes.c_size_t, _P]),
    "synerdiff_vae_stage_count": (ctypes.c_int32, [_P]),
    "synerdiff_vae_stage_name": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_char_p, ctypes.c_size_t]),
    "synerdiff_vae_stage_flops": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)]),
    "synerdiff_vae_run": (ctypes.c_int, [_P, ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_int32, _P, _P]),
    "synerdiff_vae_destroy": (None, [_P]),
    "synerdiff_vae_activation": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int64)] +
                                 [ctypes.POINTER(ctypes.c_int32)] * 3),
    "synerdiff_vae_chunk_plan": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P]),
    "synerdiff_chunk_cost": (ctypes.c_int, [_P, _P, ctypes.c_int32, ctypes.c_double, ctypes.c_double,
                                            ctypes.c_double, ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "synerdiff_plan_sequence": (ctypes.c_int, [ctypes.c_int32] * 4 + [_P, _P, ctypes.c_double, ctypes.c_int32,
                                               ctypes.c_int32, _P, ctypes.POINTER(ctypes.c_int32),
                                               ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)]),
    "synerdiff_op_conv": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, _P] + [ctypes.c_int32] * 7 +
                          [_P, _P, ctypes.c_int32, _P, ctypes.c_int32, _P, _P, _P, ctypes.c_int32, _P,
                           ctypes.c_int64, _P]),
    "synerdiff_op_conv_scratch_floats": (ctypes.c_int64, [ctypes.c_int32] * 10),
    "synerdiff_op_attention": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int64, ctypes.c_int64, _P,
                                              ctypes.c_int64, ctypes.c_int64, _P, ctypes.c_int64, ctypes.c_int64,
                                              ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_int64] +
                               [ctypes.c_int32] * 5 + [ctypes.c_float, ctypes.c_int32, _P]),
    "synerdiff_op_groupnorm_scratch_floats": (ctypes.c_size_t, [ctypes.c_int32] * 3),
    "synerdiff_op_groupnorm_stats": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, _P] + [ctypes.c_int32] * 4 +
                                     [ctypes.c_float, _P, _P, _P, _P, _P, _P]),
    "synerdiff_op_conv_out_cfg_ddim": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_int32,
                                                      ctypes.c_int32, _P, _P, ctypes.c_int32, _P, _P, _P, _P, _P,
                                                      _P]),
    "synerdiff_op_groupnorm_stats_noalloc": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, _P] +
                                             [ctypes.c_int32] * 4 + [ctypes.c_float, _P, _P, _P, _P, _P]),
    "synerdiff_op_groupnorm_fused": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, _P] + [ctypes.c_int32] * 4 +
                                     [ctypes.c_float, _P, _P, ctypes.c_int32, _P, _P]),
    "synerdiff_op_layernorm": (ctypes.c_int, [ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_int32, _P, _P,
                                              ctypes.c_float, _P]),
    "synerdiff_op_layernorm_rstd": (ctypes.c_int, [ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_int32,
                                                    ctypes.c_float, _P]),
    "synerdiff_op_geglu": (ctypes.c_int, [ctypes.c_int32, _P, _P, ctypes.c_int64, ctypes.c_int32, _P]),
    "synerdiff_op_upconv": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_int32, _P, ctypes.c_int32, _P, _P, _P]),
    "synerdiff_op_linear_rows": (ctypes.c_int, [ctypes.c_int32, _P, ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P,
                                                ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P]),
}


def lib():
    """The loaded HIP library; raises if it has not been built."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2605_08835_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIG.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _LIB = L
    return _LIB


def _check(status):
    if status != 0:
        raise SynerDiffError(status, lib().synerdiff_last_error().decode())


def _ptr(a):
    """Data pointer of a numpy array or torch tensor (None -> NULL)."""
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    return a.data_ptr()


def config_from_dict(unet, max_requests):
    c = UNetConfig()
    c.latent_c, c.latent_h, c.latent_w = unet["latent_c"], unet["latent_h"], unet["latent_w"]
    c.n_levels = len(unet["ch"])
    for i, v in enumerate(unet["ch"]):
        c.ch[i] = v
    for i, v in enumerate(unet["tx_depth"]):
        c.tx_depth[i] = v
    c.n_res, c.mid_tx_depth = unet["n_res"], unet["mid_tx_depth"]
    c.heads, c.head_dim, c.gn_groups = unet["heads"], unet["head_dim"], unet["gn_groups"]
    c.ctx_len, c.ctx_dim = unet["ctx_len"], unet["ctx_dim"]
    c.temb_in, c.temb_dim, c.add_in = unet["temb_in"], unet["temb_dim"], unet["add_in"]
    c.pooled_dim, c.time_id_dim, c.n_time_ids = unet["pooled_dim"], unet["time_id_dim"], unet["n_time_ids"]
    c.max_requests = max_requests
    c.dtype = SD_BF16 if unet["dtype"] == "bf16" else SD_F32
    return c


def manifest(cfg):
    """[(name, shape)] of the parameters the library expects, in load order."""
    L = lib()
    n = L.synerdiff_param_count(ctypes.byref(cfg))
    if n < 0:
        raise SynerDiffError(-2, L.synerdiff_last_error().decode())
    out = []
    name = ctypes.create_string_buffer(256)
    shape = (ctypes.c_int64 * 4)()
    nd = ctypes.c_int32()
    for i in range(n):
        _check(L.synerdiff_param_info(ctypes.byref(cfg), i, name, 256, shape, ctypes.byref(nd)))
        out.append((name.value.decode(), tuple(shape[k] for k in range(nd.value))))
    return out


def row_plan(cfg_on):
    cfg_on = np.ascontiguousarray(cfg_on, np.uint8)
    n = len(cfg_on)
    rr, rb = np.zeros(2 * n, np.int32), np.zeros(2 * n, np.int32)
    ru, nr = np.zeros(n, np.int32), np.zeros(1, np.int32)
    _check(lib().synerdiff_row_plan(n, _ptr(cfg_on), _ptr(rr), _ptr(rb), _ptr(ru), _ptr(nr)))
    k = int(nr[0])
    return dict(row_req=rr[:k], row_branch=rb[:k], req_row_u=ru, n_rows=k)


def alphas_cumprod(schedule):
    out = np.zeros(1000, np.float64)
    _check(lib().synerdiff_alphas_cumprod(SCHEDULES[schedule], _ptr(out)))
    return out


def ddim_coef(abar, t, t_prev, prediction="eps"):
    """(A, B) of x' = A x + B out for an eps- or v-prediction UNet."""
    abar = np.ascontiguousarray(abar, np.float64)
    out = np.zeros(2, np.float32)
    f = lib().synerdiff_ddim_coef_v if prediction == "v" else lib().synerdiff_ddim_coef
    _check(f(_ptr(abar), int(t), int(t_prev), _ptr(out)))
    return float(out[0]), float(out[1])


class UNet:
    """One UNet handle over torch-allocated device buffers."""

    def __init__(self, unet, max_requests, device=None, share_weights_with=None):
        """share_weights_with: another UNet of the same architecture (any
        latent size); this handle then uses its packed weights."""
        import torch
        self.torch = torch
        self.unet = unet
        self.cfg = config_from_dict(unet, max_requests)
        L = lib()
        _check(L.synerdiff_config_check(ctypes.byref(self.cfg)))
        self.device = torch.device(device or "cuda")
        self.act_dtype = torch.bfloat16 if unet["dtype"] == "bf16" else torch.float32
        wb = L.synerdiff_weights_bytes(ctypes.byref(self.cfg))
        wsb = L.synerdiff_workspace_bytes(ctypes.byref(self.cfg))
        self.ws = torch.empty(wsb + 256, dtype=torch.uint8, device=self.device)
        sp = _align(self.ws.data_ptr())
        h = ctypes.c_void_p()
        if share_weights_with is not None:
            self.wbuf = share_weights_with.wbuf  # keeps the shared buffer alive
            self._shared_from = share_weights_with
            _check(L.synerdiff_unet_create_shared(ctypes.byref(self.cfg), share_weights_with.h, sp, wsb,
                                                  ctypes.byref(h)))
        else:
            self.wbuf = torch.empty(wb + 256, dtype=torch.uint8, device=self.device)
            wp = _align(self.wbuf.data_ptr())
            _check(L.synerdiff_unet_create(ctypes.byref(self.cfg), wp, wb, sp, wsb, ctypes.byref(h)))
        self.h = h
        self.weights_bytes, self.workspace_bytes = wb, wsb
        self.schedule_abar = {}

    def load_weights(self, weights):
        """weights: {name: float32 array}; laid out in the library's manifest order."""
        man = manifest(self.cfg)
        flat = np.concatenate([np.ascontiguousarray(weights[n], np.float32).ravel() for n, _ in man])
        _check(lib().synerdiff_load_weights(self.h, _ptr(flat), flat.size, self._stream()))

    def _stream(self, stream=None):
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        return s.cuda_stream

    def coefficients(self, schedule, timesteps, t_prev):
        if schedule not in self.schedule_abar:
            self.schedule_abar[schedule] = alphas_cumprod(schedule)
        ab = self.schedule_abar[schedule]
        pred = self.unet.get("prediction", "eps")
        return np.array([ddim_coef(ab, t, tp, pred) for t, tp in zip(timesteps, t_prev)], np.float32)

    def step(self, latents, timesteps, cfg_on, guidance, ctx_cond, ctx_uncond, coef, out=None,
             eps_out=None, pooled_cond=None, pooled_uncond=None, time_ids=None, stream=None):
        """Enqueue one step.  latents, ctx_*, pooled_*, out and eps_out are
        device tensors; timesteps, cfg_on, guidance, coef and time_ids are
        host arrays.  Returns out."""
        n = int(latents.shape[0]) if hasattr(latents, "shape") and len(latents.shape) else -1
        u = self.unet
        lat_shape = (n, u["latent_c"], u["latent_h"], u["latent_w"])
        L, D = u["ctx_len"], u["ctx_dim"]
        f32 = self.torch.float32
        self._check_dev("latents", latents, lat_shape, f32)
        ts = self._host("timesteps", timesteps, np.int32, (n,))
        cf = self._host("cfg_on", cfg_on, np.uint8, (n,))
        gd = self._host("guidance", guidance, np.float32, (n,))
        cc = self._host("coef", coef, np.float32, (n, 2)).reshape(-1)
        self._check_dev("ctx_cond", ctx_cond, (n, L, D), self.act_dtype)
        if ctx_uncond is not None:
            shp = tuple(ctx_uncond.shape) if hasattr(ctx_uncond, "shape") else None
            self._check_dev("ctx_uncond", ctx_uncond, (1, L, D) if shp and len(shp) == 3 else (L, D),
                            self.act_dtype)
        if u["add_in"]:
            P = u["pooled_dim"]
            self._check_dev("pooled_cond", pooled_cond, (n, P), f32)
            if pooled_uncond is not None:
                shp = tuple(pooled_uncond.shape) if hasattr(pooled_uncond, "shape") else None
                self._check_dev("pooled_uncond", pooled_uncond, (1, P) if shp and len(shp) == 2 else (P,), f32)
            ti = self._host("time_ids", time_ids, np.float32, (u["n_time_ids"],))
        else:
            if pooled_cond is not None or pooled_uncond is not None or time_ids is not None:
                raise ValueError("pooled inputs / time_ids given but the UNet has no added embedding")
            ti = None
        if out is None:
            out = self.torch.empty_like(latents)
        else:
            self._check_dev("out", out, lat_shape, f32)
        if eps_out is not None:
            self._check_dev("eps_out", eps_out, lat_shape, f32)
        _check(lib().synerdiff_unet_step(self.h, n, _ptr(latents), _ptr(ts), _ptr(cf), _ptr(gd), _ptr(ctx_cond),
                                         _ptr(ctx_uncond), _ptr(pooled_cond), _ptr(pooled_uncond), _ptr(ti),
                                         _ptr(cc), _ptr(out), _ptr(eps_out), self._stream(stream)))
        return out

    def _check_dev(self, name, t, shape, dtype):
        """A device tensor the C ABI reads or writes through a raw pointer:
        the library cannot see its size, so shape, dtype, device and layout
        are checked here before the call."""
        torch = self.torch
        if not isinstance(t, torch.Tensor):
            raise ValueError(f"{name}: expected a torch tensor, got {type(t).__name__}")
        if t.device.type != self.device.type or (self.device.index is not None and t.device.index != self.device.index):
            raise ValueError(f"{name}: must live on {self.device}, got {t.device}")
        if t.dtype != dtype:
            raise ValueError(f"{name}: dtype {t.dtype}, expected {dtype}")
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
        if not t.is_contiguous():
            raise ValueError(f"{name}: must be contiguous")

    @staticmethod
    def _host(name, a, dtype, shape):
        """A host array the C ABI reads n entries of: converted to a
        contiguous array of `dtype` and checked against `shape`."""
        if a is None:
            raise ValueError(f"{name}: required")
        if hasattr(a, "device") and getattr(a.device, "type", "cpu") != "cpu":
            raise ValueError(f"{name}: must be a host array")
        arr = np.ascontiguousarray(np.asarray(a), dtype)
        if arr.shape != tuple(shape):
            raise ValueError(f"{name}: shape {arr.shape}, expected {tuple(shape)}")
        return arr

    def profile(self, enable=True):
        _check(lib().synerdiff_profile(self.h, int(enable)))

    def profile_read(self, reset=True):
        """{kernel class: dict(launches, ms, flop, bytes)} since the last reset."""
        arr = (KernelStat * 16)()
        n = ctypes.c_int32()
        _check(lib().synerdiff_profile_read(self.h, arr, 16, ctypes.byref(n), int(reset)))
        return {arr[i].name.decode(): dict(launches=arr[i].launches, ms=arr[i].ms, flop=arr[i].flop,
                                           bytes=arr[i].bytes) for i in range(min(n.value, 16))}

    def profile_read_layers(self, reset=True):
        """{layer name: dict(launches, ms, flop, bytes)} since the last reset,
        in first-launch order."""
        n = ctypes.c_int32()
        _check(lib().synerdiff_profile_read_layers(self.h, None, 0, ctypes.byref(n), 0))
        cap = max(n.value, 1)
        arr = (LayerStat * cap)()
        _check(lib().synerdiff_profile_read_layers(self.h, arr, cap, ctypes.byref(n), int(reset)))
        return {arr[i].name.decode(): dict(launches=arr[i].launches, ms=arr[i].ms, flop=arr[i].flop,
                                           bytes=arr[i].bytes) for i in range(min(n.value, cap))}

    def close(self):
        if getattr(self, "h", None):
            lib().synerdiff_unet_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _align(p):
    return (p + 255) & ~255


def vae_config_from_dict(vae, max_images):
    c = VAEConfig()
    c.latent_c, c.latent_h, c.latent_w = vae["latent_c"], vae["latent_h"], vae["latent_w"]
    c.n_levels = len(vae["ch"])
    for i, v in enumerate(vae["ch"]):
        c.ch[i] = v
    c.n_res, c.gn_groups, c.out_c = vae["n_res"], vae["gn_groups"], vae["out_c"]
    c.max_images = max_images
    c.dtype = SD_BF16 if vae["dtype"] == "bf16" else SD_F32
    c.scaling = vae["scaling"]
    return c


def vae_manifest(cfg):
    """[(name, shape)] of the decoder parameters the library expects, in load order."""
    L = lib()
    n = L.synerdiff_vae_param_count(ctypes.byref(cfg))
    if n < 0:
        raise SynerDiffError(-2, L.synerdiff_last_error().decode())
    out = []
    name = ctypes.create_string_buffer(256)
    shape = (ctypes.c_int64 * 4)()
    nd = ctypes.c_int32()
    for i in range(n):
        _check(L.synerdiff_vae_param_info(ctypes.byref(cfg), i, name, 256, shape, ctypes.byref(nd)))
        out.append((name.value.decode(), tuple(shape[k] for k in range(nd.value))))
    return out


def vae_chunk_plan(stage_cost, c):
    """Boundaries b_0 = 0 < ... < b_c = len(stage_cost) of the c contiguous
    chunks with the smallest largest-chunk cost."""
    cost = np.ascontiguousarray(stage_cost, np.float64)
    out = np.zeros(c + 1, np.int32)
    _check(lib().synerdiff_vae_chunk_plan(_ptr(cost), len(cost), int(c), _ptr(out)))
    return [int(x) for x in out]


def chunk_cost(t_u, t_v, T_u0, T_v0, lam):
    """Eq. (2) cumulative latencies and the Eq. (1) cost: (T_u(c), T_v(c), L(c))."""
    tu = np.ascontiguousarray(t_u, np.float64)
    tv = np.ascontiguousarray(t_v, np.float64)
    a, b, l = ctypes.c_double(), ctypes.c_double(), ctypes.c_double()
    _check(lib().synerdiff_chunk_cost(_ptr(tu), _ptr(tv), len(tu), float(T_u0), float(T_v0), float(lam),
                                      ctypes.byref(a), ctypes.byref(b), ctypes.byref(l)))
    return a.value, b.value, l.value


class VAE:
    """One VAE-decoder handle over torch-allocated device buffers."""

    def __init__(self, vae, max_images, device=None):
        import torch
        self.torch = torch
        self.vae = vae
        self.cfg = vae_config_from_dict(vae, max_images)
        L = lib()
        _check(L.synerdiff_vae_config_check(ctypes.byref(self.cfg)))
        self.device = torch.device(device or "cuda")
        wb = L.synerdiff_vae_weights_bytes(ctypes.byref(self.cfg))
        wsb = L.synerdiff_vae_workspace_bytes(ctypes.byref(self.cfg))
        self.wbuf = torch.empty(wb + 256, dtype=torch.uint8, device=self.device)
        self.ws = torch.empty(wsb + 256, dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        _check(L.synerdiff_vae_create(ctypes.byref(self.cfg), _align(self.wbuf.data_ptr()), wb,
                                      _align(self.ws.data_ptr()), wsb, ctypes.byref(h)))
        self.h = h
        self.max_images = max_images
        self.up = 2 ** (len(vae["ch"]) - 1)
        n = L.synerdiff_vae_stage_count(self.h)
        name = ctypes.create_string_buffer(64)
        self.stages, self.stage_flops = [], []
        f = ctypes.c_double()
        for i in range(n):
            _check(L.synerdiff_vae_stage_name(self.h, i, name, 64))
            _check(L.synerdiff_vae_stage_flops(self.h, i, ctypes.byref(f)))
            self.stages.append(name.value.decode())
            self.stage_flops.append(f.value)

    def load_weights(self, weights):
        man = vae_manifest(self.cfg)
        flat = np.concatenate([np.ascontiguousarray(weights[n], np.float32).ravel() for n, _ in man])
        _check(lib().synerdiff_vae_load_weights(self.h, _ptr(flat), flat.size, self._stream()))

    def _stream(self, stream=None):
        s = stream if stream is not None else self.torch.cuda.current_stream(self.device)
        return s.cuda_stream

    def image_shape(self, n):
        v = self.vae
        return (n, v["out_c"], v["latent_h"] * self.up, v["latent_w"] * self.up)

    def run(self, latents, begin, end, image=None, stream=None):
        """Enqueue stages [begin, end) for the batch of latents [n, C, H, W]
        (fp32 device tensor); returns the image tensor (written when end is
        the last stage)."""
        torch = self.torch
        v = self.vae
        n = int(latents.shape[0])
        want = (n, v["latent_c"], v["latent_h"], v["latent_w"])
        if tuple(latents.shape) != want or latents.dtype != torch.float32 or not latents.is_contiguous() \
                or latents.device.type != self.device.type:
            raise ValueError(f"latents: expected a contiguous float32 device tensor of shape {want}")
        if image is None:
            image = torch.empty(self.image_shape(n), device=latents.device, dtype=torch.float32)
        elif tuple(image.shape) != self.image_shape(n) or image.dtype != torch.float32 or not image.is_contiguous():
            raise ValueError(f"image: expected a contiguous float32 tensor of shape {self.image_shape(n)}")
        _check(lib().synerdiff_vae_run(self.h, n, _ptr(latents), int(begin), int(end), _ptr(image),
                                       self._stream(stream)))
        return image

    def activation(self, i, n):
        """View of the activation after stage i ([n, H, W, C], channels-last)
        inside the workspace; valid after a run that ended at stage i + 1."""
        off = ctypes.c_int64()
        H, W, C = ctypes.c_int32(), ctypes.c_int32(), ctypes.c_int32()
        _check(lib().synerdiff_vae_activation(self.h, int(i), ctypes.byref(off), ctypes.byref(H), ctypes.byref(W),
                                              ctypes.byref(C)))
        dt = self.torch.bfloat16 if self.vae["dtype"] == "bf16" else self.torch.float32
        esz = 2 if self.vae["dtype"] == "bf16" else 4
        base = _align(self.ws.data_ptr()) - self.ws.data_ptr()
        nbytes = n * H.value * W.value * C.value * esz
        raw = self.ws[base + off.value: base + off.value + nbytes]
        return raw.view(dt).reshape(n, H.value, W.value, C.value)

    def decode(self, latents, image=None, stream=None):
        return self.run(latents, 0, len(self.stages), image=image, stream=stream)

    def close(self):
        if getattr(self, "h", None):
            lib().synerdiff_vae_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def plan_sequence(M, N, K, tau, delta, T_lim, exact=False, max_stages=None):
    """Stage sequence of the inter-concurrency scheduler (Alg. 1, or the exact
    optimum of Problem P with exact=True).  tau, delta: arrays [B][B][B]
    (B = bmax + 1) indexed [m][n][k].  Returns (list of (m, n, k), cost, time);
    raises SynerDiffError when no sequence meets T_lim."""
    tau = np.ascontiguousarray(tau, np.float64)
    delta = np.ascontiguousarray(delta, np.float64)
    B = tau.shape[0]
    if tau.shape != (B, B, B) or delta.shape != (B, B, B):
        raise ValueError("tau and delta must be [bmax + 1]^3 arrays")
    cap = max_stages if max_stages is not None else max(M, 1)
    seq = np.zeros(3 * cap, np.int32)
    ns, cost, tm = ctypes.c_int32(), ctypes.c_double(), ctypes.c_double()
    _check(lib().synerdiff_plan_sequence(int(M), int(N), int(K), B - 1, _ptr(tau), _ptr(delta), float(T_lim),
                                         int(bool(exact)), cap, _ptr(seq), ctypes.byref(ns), ctypes.byref(cost),
                                         ctypes.byref(tm)))
    return [tuple(int(x) for x in seq[3 * t:3 * t + 3]) for t in range(ns.value)], cost.value, tm.value
