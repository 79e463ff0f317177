"""ctypes binding of libparagan (include/paragan.h).

Argument marshalling only: every function here forwards to the C ABI of the
same name; torch tensors supply device memory and the stream.  There is no
fallback: if the in-tree libparagan.so is missing, loading raises.
"""
import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libparagan.so")

OK, EINVAL, EUNSUPPORTED, EWORKSPACE, EHIP, ENONFINITE, ETIMEOUT = 0, -1, -2, -3, -4, -5, -6
F32, BF16 = 0, 1
ADAM, ADABELIEF = 0, 1


class ParaganError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__("paragan error %d: %s" % (code, msg))
        self.code = code


class TensorInfo(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("ndim", C.c_int32), ("shape", C.c_int64 * 4),
                ("offset", C.c_int64), ("u_offset", C.c_int64)]


class GBlockDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("H", C.c_int32), ("W", C.c_int32), ("cin", C.c_int32),
                ("cout", C.c_int32), ("dc", C.c_int32), ("dtype", C.c_int32),
                ("n_power_iter", C.c_int32), ("bn_eps", C.c_float), ("sn_eps", C.c_float)]


class DBlockDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("H", C.c_int32), ("W", C.c_int32), ("cin", C.c_int32),
                ("cout", C.c_int32), ("preact", C.c_int32), ("downsample", C.c_int32),
                ("learnable_sc", C.c_int32), ("dtype", C.c_int32), ("n_power_iter", C.c_int32),
                ("sn_eps", C.c_float)]


class AttnDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("H", C.c_int32), ("W", C.c_int32), ("C", C.c_int32),
                ("n_power_iter", C.c_int32), ("sn_eps", C.c_float)]


class GoutDesc(C.Structure):
    _fields_ = [("B", C.c_int32), ("H", C.c_int32), ("W", C.c_int32), ("C", C.c_int32),
                ("n_power_iter", C.c_int32), ("bn_eps", C.c_float), ("sn_eps", C.c_float)]


class Optim(C.Structure):
    _fields_ = [("kind", C.c_int32), ("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float),
                ("eps", C.c_float)]


class BigganDesc(C.Structure):
    _fields_ = [("img", C.c_int32), ("ch", C.c_int32), ("n_g", C.c_int32), ("g_mult", C.c_int32 * 10),
                ("n_d", C.c_int32), ("d_mult", C.c_int32 * 10), ("d_down", C.c_int32 * 10),
                ("attn_res", C.c_int32), ("n_classes", C.c_int32), ("dz", C.c_int32),
                ("shared_dim", C.c_int32), ("B", C.c_int32), ("n_power_iter", C.c_int32),
                ("bn_eps", C.c_float), ("sn_eps", C.c_float), ("opt_g", Optim), ("opt_d", Optim)]


class NetState(C.Structure):
    _fields_ = [("params", C.c_void_p), ("u", C.c_void_p), ("grads", C.c_void_p),
                ("opt_m", C.c_void_p), ("opt_v", C.c_void_p), ("opt_t", C.c_int64)]


class StepInputs(C.Structure):
    _fields_ = [("x_real", C.POINTER(C.c_void_p)), ("y_real", C.POINTER(C.c_void_p)),
                ("z_fake", C.POINTER(C.c_void_p)), ("y_fake", C.POINTER(C.c_void_p)),
                ("z_g", C.c_void_p), ("y_g", C.c_void_p)]


class AsyncInputs(C.Structure):
    _fields_ = [("x_real", C.POINTER(C.c_void_p)), ("y_real", C.POINTER(C.c_void_p)),
                ("z", C.c_void_p), ("y", C.c_void_p), ("img_buff", C.c_void_p),
                ("lab_buff", C.c_void_p), ("pred_buff", C.c_void_p)]


class PipelineCfg(C.Structure):
    _fields_ = [("min_threads", C.c_int32), ("max_threads", C.c_int32), ("min_depth", C.c_int32),
                ("max_depth", C.c_int32), ("window", C.c_int32), ("threshold_ms", C.c_double)]


class PipelineStats(C.Structure):
    _fields_ = [("threads", C.c_int32), ("depth", C.c_int32), ("window_mean_ms", C.c_double),
                ("fetched", C.c_int64), ("delivered", C.c_int64), ("grows", C.c_int64), ("shrinks", C.c_int64),
                ("consumer_wait_ms", C.c_double)]


class SynthSource(C.Structure):
    _fields_ = [("seed", C.c_uint64), ("B", C.c_int32), ("img", C.c_int32), ("n_classes", C.c_int32),
                ("latency_ms", C.c_void_p), ("n_latency", C.c_int64)]


# int fetch(void* user, int64_t seq, void* slot, size_t slot_bytes)
FETCH_FN = C.CFUNCTYPE(C.c_int, C.c_void_p, C.c_int64, C.c_void_p, C.c_size_t)


class KernelStat(C.Structure):
    _fields_ = [("name", C.c_char * 64), ("launches", C.c_int64), ("total_ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_P = C.c_void_p
_SIGS = {
    "paragan_profile": (C.c_int, [_P, C.c_int]),
    "paragan_profile_read": (C.c_int, [_P, _P, C.c_int32, C.POINTER(C.c_int32)]),
    "paragan_create": (C.c_int, [C.POINTER(_P), _P]),
    "paragan_destroy": (None, [_P]),
    "paragan_last_error": (C.c_char_p, [_P]),
    "paragan_sync": (C.c_int, [_P]),
    "paragan_set_overlap_wgrad": (C.c_int, [_P, C.c_int]),
    "paragan_cpad": (C.c_int64, [C.c_int64]),
    "paragan_sn_ws_size": (C.c_int, [C.c_int64, C.c_int64, C.POINTER(C.c_size_t)]),
    "paragan_sn_power_iter": (C.c_int, [_P, _P, C.c_int64, C.c_int64, _P, _P, _P, C.c_int, C.c_float, _P]),
    "paragan_sn_check": (C.c_int, [C.c_int64, C.c_int64, C.c_int, C.c_float]),
    "paragan_gblock_layout": (C.c_int, [_P, _P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int64),
                                        C.POINTER(C.c_int64)]),
    "paragan_gblock_sizes": (C.c_int, [_P, C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "paragan_gblock_check": (C.c_int, [_P]),
    "paragan_gblock_fwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_gblock_bwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_dblock_layout": (C.c_int, [_P, _P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int64),
                                        C.POINTER(C.c_int64)]),
    "paragan_dblock_sizes": (C.c_int, [_P, C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "paragan_dblock_check": (C.c_int, [_P]),
    "paragan_dblock_fwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_dblock_bwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_attn_layout": (C.c_int, [_P, _P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int64),
                                      C.POINTER(C.c_int64)]),
    "paragan_attn_sizes": (C.c_int, [_P, C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "paragan_attn_check": (C.c_int, [_P]),
    "paragan_attn_fwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_attn_bwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_gout_layout": (C.c_int, [_P, _P, C.c_int32, C.POINTER(C.c_int32), C.POINTER(C.c_int64),
                                      C.POINTER(C.c_int64)]),
    "paragan_gout_sizes": (C.c_int, [_P, C.POINTER(C.c_size_t), C.POINTER(C.c_size_t)]),
    "paragan_gout_check": (C.c_int, [_P]),
    "paragan_gout_fwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_gout_bwd": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_net_layout": (C.c_int, [_P, C.c_int32, _P, C.c_int32, C.POINTER(C.c_int32),
                                     C.POINTER(C.c_int64), C.POINTER(C.c_int64)]),
    "paragan_biggan_check": (C.c_int, [_P]),
    "paragan_train_step_ws_size": (C.c_int, [_P, C.POINTER(C.c_size_t)]),
    "paragan_train_step": (C.c_int, [_P, _P, _P, _P, _P, C.c_int32, _P, _P]),
    "paragan_g_sample": (C.c_int, [_P, _P, _P, _P, _P, _P, _P]),
    "paragan_d_step": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_g_step": (C.c_int, [_P, _P, _P, _P, _P, _P, _P, _P]),
    "paragan_sn_power_iter_noalloc": (C.c_int, [_P, _P, C.c_int64, C.c_int64, _P, _P, _P, C.c_int, C.c_float]),
    "paragan_pipeline_create": (C.c_int, [_P, _P, _P, _P, _P, C.c_int32, C.c_size_t]),
    "paragan_pipeline_next": (C.c_int, [_P, C.POINTER(C.c_int64), C.POINTER(C.c_int32), C.c_int32]),
    "paragan_pipeline_release": (C.c_int, [_P, C.c_int32]),
    "paragan_pipeline_get_stats": (C.c_int, [_P, _P]),
    "paragan_pipeline_error": (C.c_char_p, [_P]),
    "paragan_pipeline_destroy": (None, [_P]),
    "paragan_synth_batch_bytes": (C.c_size_t, [_P]),
    "paragan_synth_fetch": (C.c_int, [_P, C.c_int64, _P, C.c_size_t]),
    "paragan_async_ws_size": (C.c_int, [_P, C.c_int32, C.POINTER(C.c_size_t)]),
    "paragan_async_step": (C.c_int, [_P, _P, _P, _P, _P, C.c_int32, _P, _P]),
}

_lib = None


def load():
    """Load the in-tree libparagan.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libparagan.so not built: run __graft_entry__.build() "
                              "or python -m paragan_2411_03999_amd.build")
        lib = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _lib = lib
    return _lib


def exported_symbols():
    return list(_SIGS)


def _ref(x):
    return C.byref(x) if x is not None else None


def _ptr(t):
    """Device pointer of a torch tensor (or None -> NULL)."""
    if t is None:
        return None
    return C.c_void_p(t.data_ptr())


class Context:
    """A libparagan context bound to a torch CUDA (HIP) stream."""

    def __init__(self, stream=None):
        import torch
        lib = load()
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        h = C.c_void_p()
        rc = lib.paragan_create(C.byref(h), C.c_void_p(stream.cuda_stream))
        if rc != OK:
            raise ParaganError(rc, lib.paragan_last_error(None).decode())
        self.h = h

    def check(self, rc):
        if rc != OK:
            raise ParaganError(rc, load().paragan_last_error(self.h).decode())
        return rc

    def set_overlap_wgrad(self, on):
        """Run the block backwards' weight gradients of the step calls on a
        further stream beside their data gradients (bit-identical results)."""
        return self.check(load().paragan_set_overlap_wgrad(self.h, int(on)))

    def close(self):
        if self.h:
            load().paragan_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _check_static(rc):
    if rc != OK:
        raise ParaganError(rc, load().paragan_last_error(None).decode())


def cpad(c):
    return int(load().paragan_cpad(c))


def _layout(fn, *args):
    cnt, npar, nu = C.c_int32(), C.c_int64(), C.c_int64()
    _check_static(fn(*args, None, 0, C.byref(cnt), C.byref(npar), C.byref(nu)))
    arr = (TensorInfo * cnt.value)()
    _check_static(fn(*args, arr, cnt.value, C.byref(cnt), C.byref(npar), C.byref(nu)))
    ents = [dict(name=a.name.decode(), shape=tuple(a.shape[:a.ndim]), offset=a.offset,
                 u_offset=a.u_offset) for a in arr]
    return ents, npar.value, nu.value


def _sizes(fn, desc):
    s, w = C.c_size_t(), C.c_size_t()
    _check_static(fn(C.byref(desc), C.byref(s), C.byref(w)))
    return s.value, w.value


# ---------------------------------------------------------------- entry points
def paragan_sn_ws_size(rows, cols):
    n = C.c_size_t()
    _check_static(load().paragan_sn_ws_size(rows, cols, C.byref(n)))
    return n.value


def paragan_sn_power_iter(ctx, W, rows, cols, u, v, sigma, n_iter, eps, ws):
    return ctx.check(load().paragan_sn_power_iter(ctx.h, _ptr(W), rows, cols, _ptr(u), _ptr(v), _ptr(sigma),
                                                  n_iter, eps, _ptr(ws)))


def paragan_gblock_layout(desc):
    return _layout(load().paragan_gblock_layout, C.byref(desc))


def paragan_gblock_sizes(desc):
    return _sizes(load().paragan_gblock_sizes, desc)


def paragan_gblock_check(desc):
    return load().paragan_gblock_check(C.byref(desc))


def paragan_gblock_fwd(ctx, desc, params, u, x, cond, y, saved, ws):
    return ctx.check(load().paragan_gblock_fwd(ctx.h, C.byref(desc), _ptr(params), _ptr(u), _ptr(x), _ptr(cond),
                                               _ptr(y), _ptr(saved), _ptr(ws)))


def paragan_gblock_bwd(ctx, desc, params, x, cond, saved, dy, dx, dcond, grads, ws):
    return ctx.check(load().paragan_gblock_bwd(ctx.h, C.byref(desc), _ptr(params), _ptr(x), _ptr(cond),
                                               _ptr(saved), _ptr(dy), _ptr(dx), _ptr(dcond), _ptr(grads),
                                               _ptr(ws)))


def paragan_dblock_layout(desc):
    return _layout(load().paragan_dblock_layout, C.byref(desc))


def paragan_dblock_sizes(desc):
    return _sizes(load().paragan_dblock_sizes, desc)


def paragan_dblock_check(desc):
    return load().paragan_dblock_check(C.byref(desc))


def paragan_dblock_fwd(ctx, desc, params, u, x, y, saved, ws):
    return ctx.check(load().paragan_dblock_fwd(ctx.h, C.byref(desc), _ptr(params), _ptr(u), _ptr(x), _ptr(y),
                                               _ptr(saved), _ptr(ws)))


def paragan_dblock_bwd(ctx, desc, params, x, saved, dy, dx, grads, ws):
    return ctx.check(load().paragan_dblock_bwd(ctx.h, C.byref(desc), _ptr(params), _ptr(x), _ptr(saved),
                                               _ptr(dy), _ptr(dx), _ptr(grads), _ptr(ws)))


def paragan_attn_layout(desc):
    return _layout(load().paragan_attn_layout, C.byref(desc))


def paragan_attn_sizes(desc):
    return _sizes(load().paragan_attn_sizes, desc)


def paragan_attn_check(desc):
    return load().paragan_attn_check(C.byref(desc))


def paragan_attn_fwd(ctx, desc, params, u, x, y, saved, ws):
    return ctx.check(load().paragan_attn_fwd(ctx.h, C.byref(desc), _ptr(params), _ptr(u), _ptr(x), _ptr(y),
                                             _ptr(saved), _ptr(ws)))


def paragan_attn_bwd(ctx, desc, params, x, saved, dy, dx, grads, ws):
    return ctx.check(load().paragan_attn_bwd(ctx.h, C.byref(desc), _ptr(params), _ptr(x), _ptr(saved),
                                             _ptr(dy), _ptr(dx), _ptr(grads), _ptr(ws)))


def paragan_gout_layout(desc):
    return _layout(load().paragan_gout_layout, C.byref(desc))


def paragan_gout_sizes(desc):
    return _sizes(load().paragan_gout_sizes, desc)


def paragan_gout_check(desc):
    return load().paragan_gout_check(C.byref(desc))


def paragan_gout_fwd(ctx, desc, params, u, x, img, saved, ws):
    return ctx.check(load().paragan_gout_fwd(ctx.h, C.byref(desc), _ptr(params), _ptr(u), _ptr(x), _ptr(img),
                                             _ptr(saved), _ptr(ws)))


def paragan_gout_bwd(ctx, desc, params, x, img, saved, dimg, dx, grads, ws):
    return ctx.check(load().paragan_gout_bwd(ctx.h, C.byref(desc), _ptr(params), _ptr(x), _ptr(img),
                                             _ptr(saved), _ptr(dimg), _ptr(dx), _ptr(grads), _ptr(ws)))


def paragan_net_layout(desc, which):
    return _layout(load().paragan_net_layout, C.byref(desc), which)


def paragan_biggan_check(desc):
    return load().paragan_biggan_check(C.byref(desc))


def paragan_train_step_ws_size(desc):
    n = C.c_size_t()
    _check_static(load().paragan_train_step_ws_size(C.byref(desc), C.byref(n)))
    return n.value


def paragan_train_step(ctx, desc, G, D, inputs, n_D, ws, losses):
    """G, D: NetState; inputs: StepInputs; losses: ctypes float array (n_D+1)."""
    return load().paragan_train_step(ctx.h, C.byref(desc), C.byref(G), C.byref(D), C.byref(inputs), n_D,
                                     _ptr(ws), losses)


def paragan_g_sample(ctx, desc, G, z, y, img, ws):
    """G: NetState; z, y, img, ws: device tensors.  Returns the status."""
    return load().paragan_g_sample(ctx.h, C.byref(desc), C.byref(G), _ptr(z), _ptr(y), _ptr(img), _ptr(ws))


def paragan_d_step(ctx, desc, D, x_real, y_real, x_fake, y_fake, ws, loss):
    """loss: ctypes float array (1).  Returns the status."""
    return load().paragan_d_step(ctx.h, C.byref(desc), C.byref(D), _ptr(x_real), _ptr(y_real), _ptr(x_fake),
                                 _ptr(y_fake), _ptr(ws), loss)


def paragan_g_step(ctx, desc, G, D, z, y, ws, loss):
    """loss: ctypes float array (1).  Returns the status."""
    return load().paragan_g_step(ctx.h, C.byref(desc), C.byref(G), C.byref(D), _ptr(z), _ptr(y), _ptr(ws), loss)


def paragan_sn_power_iter_noalloc(ctx, W, rows, cols, u, v, sigma, n_iter, eps):
    """As paragan_sn_power_iter, with the library's own scratch (no
    workspace argument).  Returns the status."""
    return load().paragan_sn_power_iter_noalloc(ctx.h, _ptr(W), rows, cols, _ptr(u), _ptr(v), _ptr(sigma), n_iter,
                                                eps)


def paragan_async_ws_size(desc, n_D):
    n = C.c_size_t()
    _check_static(load().paragan_async_ws_size(C.byref(desc), int(n_D), C.byref(n)))
    return n.value


def paragan_async_step(ctx, desc, G, D, inputs, n_D, ws, losses):
    """inputs: AsyncInputs; losses: ctypes float array (n_D+1).  Returns the status."""
    return load().paragan_async_step(ctx.h, C.byref(desc), C.byref(G), C.byref(D), C.byref(inputs), n_D,
                                     _ptr(ws), losses)


class Pipeline:
    """paragan_pipeline_* over host slot buffers.  fetch: a FETCH_FN (kept
    alive here) or None for the library's synthetic source `synth`."""

    def __init__(self, cfg, slots, slot_bytes, fetch=None, user=None, synth=None):
        lib = load()
        self._keep = [cfg, slots, fetch, synth]
        if fetch is None:
            fn = C.cast(lib.paragan_synth_fetch, C.c_void_p)
            user = C.cast(C.pointer(synth), C.c_void_p)
        else:
            fn = C.cast(fetch, C.c_void_p)
        arr = (C.c_void_p * len(slots))(*slots)
        self._keep.append(arr)
        h = C.c_void_p()
        rc = lib.paragan_pipeline_create(C.byref(h), C.byref(cfg), fn, user, arr, len(slots), slot_bytes)
        if rc != OK:
            raise ParaganError(rc, lib.paragan_pipeline_error(None).decode())
        self.h = h

    def next(self, timeout_ms=-1):
        """(status, seq, slot)."""
        seq, slot = C.c_int64(), C.c_int32()
        rc = load().paragan_pipeline_next(self.h, C.byref(seq), C.byref(slot), int(timeout_ms))
        return rc, seq.value, slot.value

    def release(self, slot):
        return load().paragan_pipeline_release(self.h, int(slot))

    def stats(self):
        st = PipelineStats()
        if load().paragan_pipeline_get_stats(self.h, C.byref(st)) != OK:
            raise ParaganError(EINVAL, self.error())
        return {k: getattr(st, k) for k, _ in PipelineStats._fields_}

    def error(self):
        return load().paragan_pipeline_error(self.h).decode()

    def close(self):
        if self.h:
            load().paragan_pipeline_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def paragan_profile(ctx, enable):
    """enable: 0 off, 1 on, 2 on with per-launch GEMM shapes in the names."""
    return ctx.check(load().paragan_profile(ctx.h, int(enable)))


def paragan_profile_read(ctx, cap=1024):
    """Per-kernel launch statistics since the last read (list of dicts);
    the records are consumed."""
    arr = (KernelStat * cap)()
    n = C.c_int32()
    ctx.check(load().paragan_profile_read(ctx.h, arr, cap, C.byref(n)))
    return [dict(name=a.name.decode(), launches=a.launches, total_ms=a.total_ms, flops=a.flops, bytes=a.bytes)
            for a in arr[:min(n.value, cap)]]


# ---------------------------------------------------------- tensor marshalling
def flat_from_named(layout, n_params, named, device="cuda"):
    """Pack {name: array} into the flat fp32 buffer order of `layout`."""
    import torch
    flat = np.zeros(n_params, dtype=np.float32)
    for e in layout:
        a = np.asarray(named[e["name"]], dtype=np.float32)
        assert a.shape == tuple(e["shape"]), (e["name"], a.shape, e["shape"])
        flat[e["offset"]:e["offset"] + a.size] = a.reshape(-1)
    return torch.from_numpy(flat).to(device)


def u_from_named(layout, n_u, named, device="cuda"):
    import torch
    flat = np.zeros(max(n_u, 1), dtype=np.float32)
    for e in layout:
        if e["u_offset"] >= 0:
            flat[e["u_offset"]:e["u_offset"] + e["shape"][0]] = np.asarray(named[e["name"]], np.float32)
    return torch.from_numpy(flat).to(device)


def named_from_flat(layout, flat):
    f = flat.detach().cpu().numpy().astype(np.float64)
    return {e["name"]: f[e["offset"]:e["offset"] + int(np.prod(e["shape"]))].reshape(e["shape"])
            for e in layout}


def named_u_from_flat(layout, flat):
    f = flat.detach().cpu().numpy().astype(np.float64)
    return {e["name"]: f[e["u_offset"]:e["u_offset"] + e["shape"][0]] for e in layout if e["u_offset"] >= 0}


def to_device_nhwc(x, dtype, device="cuda"):
    """(N,H,W,C) array -> padded NHWC device tensor (C rounded up to 32)."""
    import torch
    n, h, w, c = x.shape
    buf = np.zeros((n, h, w, cpad(c)), dtype=np.float32)
    buf[..., :c] = x
    t = torch.from_numpy(buf).to(device)
    return t.to(torch.bfloat16) if dtype == BF16 else t


def from_device_nhwc(t, c):
    import torch
    return t.detach().to(torch.float32).cpu().numpy()[..., :c].astype(np.float64)


def empty_nhwc(n, h, w, c, dtype, device="cuda"):
    import torch
    return torch.zeros((n, h, w, cpad(c)), dtype=torch.bfloat16 if dtype == BF16 else torch.float32,
                       device=device)


def workspace(nbytes, device="cuda"):
    """A 256-byte aligned device byte buffer of at least nbytes."""
    import torch
    t = torch.empty(max(int(nbytes), 1) + 256, dtype=torch.uint8, device=device)
    off = (-t.data_ptr()) % 256
    return t[off:off + max(int(nbytes), 1)]
