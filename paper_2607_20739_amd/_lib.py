"""ctypes binding of libpgc.so, one Python function per C entry point of include/pgc.h.

Argument marshalling only: every device computation runs in the library's HIP
kernels.  Device arguments accept a torch tensor (its data_ptr is passed after
checking device, dtype and contiguity) or a raw integer address.  A nonzero
status raises PGCError carrying the library's message.
"""

import ctypes
import os

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpgc.so")

PGC_FR, PGC_CR, PGC_CR_REAL, PGC_IS_SGD = 0, 1, 2, 3
PGC_LOGISTIC, PGC_LSQ, PGC_MLP = 0, 1, 2
PGC_OK, PGC_EINVAL, PGC_ESTRAGGLERS, PGC_ESINGULAR, PGC_EDEVICE, PGC_ESTATE = 0, -1, -2, -3, -4, -5
PGC_POLICY_EXACT, PGC_POLICY_UNIFORM_COUNT, PGC_POLICY_BERNOULLI, PGC_POLICY_SLOWEST = 0, 1, 2, 3
PGC_KERNEL_GRADIENT, PGC_KERNEL_REDUCE, PGC_KERNEL_CODE = 0, 1, 2
PGC_KERNEL_MLP_CAST, PGC_KERNEL_MLP_FORWARD, PGC_KERNEL_MLP_HEAD, PGC_KERNEL_MLP_WGRAD = 3, 4, 5, 6
PGC_MAX_N = 256
PGC_NOALLOC_SCRATCH_BYTES = 32 << 20
PGC_MLP_MAX_D_IN = 1 << 20

SCHEMES = {"FR": PGC_FR, "CR": PGC_CR, "CR_REAL": PGC_CR_REAL, "IS_SGD": PGC_IS_SGD}
MODELS = {"logistic": PGC_LOGISTIC, "lsq": PGC_LSQ, "mlp": PGC_MLP}


class PGCError(RuntimeError):
    def __init__(self, status, message):
        super().__init__("%s (status %d)" % (message, status))
        self.status = status


class pgc_config(ctypes.Structure):
    _fields_ = [("model", ctypes.c_int32), ("d_in", ctypes.c_int32), ("N", ctypes.c_int64),
                ("hidden", ctypes.c_int32), ("classes", ctypes.c_int32), ("code_seed", ctypes.c_uint64)]


_lib = None
_P = ctypes.c_void_p
_I32P = ctypes.POINTER(ctypes.c_int32)
_I64P = ctypes.POINTER(ctypes.c_int64)
_F64P = ctypes.POINTER(ctypes.c_double)
_U8P = ctypes.POINTER(ctypes.c_uint8)

_SIGNATURES = {
    "pgc_init": (ctypes.c_int, [ctypes.POINTER(_P), ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int64]),
    "pgc_configure": (ctypes.c_int, [_P, ctypes.POINTER(pgc_config)]),
    "pgc_set_pipelining": (ctypes.c_int, [_P, ctypes.c_int]),
    "pgc_set_stream": (ctypes.c_int, [_P, _P]),
    "pgc_workspace_bytes": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "pgc_bind_workspace": (ctypes.c_int, [_P, _P, ctypes.c_size_t]),
    "pgc_step": (ctypes.c_int, [_P, _P, _P, _P, _U8P, ctypes.c_float]),
    "pgc_step_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _U8P, ctypes.c_float]),
    "pgc_decode_coeffs": (ctypes.c_int, [_P, _U8P, _F64P, _F64P, _I32P, _I32P]),
    "pgc_placement": (ctypes.c_int, [_P, _I32P]),
    "pgc_schedule": (ctypes.c_int, [_P, ctypes.c_int64, _I32P]),
    "pgc_encoding_matrix": (ctypes.c_int, [_P, _F64P]),
    "pgc_num_coded": (ctypes.c_int, [_P, _I32P]),
    "pgc_make_mask": (ctypes.c_int, [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                     ctypes.c_int, ctypes.c_double, _U8P]),
    "pgc_delay_step": (ctypes.c_int, [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int, ctypes.c_int,
                                      ctypes.c_double, ctypes.c_double, _U8P, _F64P, _F64P]),
    "pgc_splitmix64": (ctypes.c_int, [ctypes.c_uint64, ctypes.c_uint64, ctypes.POINTER(ctypes.c_uint64)]),
    "pgc_read_ring": (ctypes.c_int, [_P, ctypes.c_int, ctypes.c_int, _P]),
    "pgc_read_coded": (ctypes.c_int, [_P, ctypes.c_int, _P]),
    "pgc_read_decoded": (ctypes.c_int, [_P, _P]),
    "pgc_state_bytes": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "pgc_save_state": (ctypes.c_int, [_P, _P, ctypes.c_size_t]),
    "pgc_load_state": (ctypes.c_int, [_P, _P, ctypes.c_size_t]),
    "pgc_get_step": (ctypes.c_int, [_P, _I64P]),
    "pgc_set_timing": (ctypes.c_int, [_P, ctypes.c_int]),
    "pgc_kernel_time": (ctypes.c_int, [_P, ctypes.c_int, _F64P, _I64P]),
    "pgc_set_timing_period": (ctypes.c_int, [_P, ctypes.c_int64]),
    "pgc_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "pgc_last_error": (ctypes.c_char_p, [_P]),
    "pgc_destroy": (ctypes.c_int, [_P]),
}


def lib():
    """The loaded library; raises if it has not been built (there is no fallback)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libpgc.so is not built (python -m paper_2607_20739_amd.build); "
                               "the PGC step has no other implementation")
        handle = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(handle, name)
            fn.restype = res
            fn.argtypes = args
        _lib = handle
    return _lib


def exported_symbols():
    return list(_SIGNATURES)


def _check(status, ctx=None):
    if status != PGC_OK:
        msg = lib().pgc_last_error(ctx).decode() if ctx is not None else ""
        if not msg:
            msg = lib().pgc_strerror(status).decode()
        raise PGCError(status, msg)


def _dev(x, dtype=None, numel=None):
    """Device address of a torch tensor (checked) or an integer address."""
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError("expected a GPU tensor")
    if not x.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    if dtype is not None and x.dtype != dtype:
        raise ValueError("expected dtype %s, got %s" % (dtype, x.dtype))
    if numel is not None and x.numel() < numel:
        raise ValueError("tensor holds %d elements, need %d" % (x.numel(), numel))
    return x.data_ptr()


def _mask_arg(mask, n):
    m = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    if m.shape != (n,):
        raise ValueError("straggler mask must have n = %d entries" % n)
    return m, m.ctypes.data_as(_U8P)


def pgc_init(scheme, n, c, d):
    ctx = _P()
    scheme = SCHEMES.get(scheme, scheme)
    _check(lib().pgc_init(ctypes.byref(ctx), int(scheme), int(n), int(c), int(d)))
    return ctx


def pgc_configure(ctx, model, N, d_in, hidden=0, classes=0, code_seed=0):
    cfg = pgc_config(MODELS.get(model, model), int(d_in), int(N), int(hidden), int(classes), int(code_seed))
    _check(lib().pgc_configure(ctx, ctypes.byref(cfg)), ctx)


def pgc_set_pipelining(ctx, enabled):
    """True: pipelined gradient coding (default); False: gradient coding."""
    _check(lib().pgc_set_pipelining(ctx, 1 if enabled else 0), ctx)


def pgc_set_stream(ctx, stream):
    """stream: a hipStream_t address (e.g. torch.cuda.current_stream().cuda_stream) or 0."""
    _check(lib().pgc_set_stream(ctx, _P(int(stream))), ctx)


def pgc_workspace_bytes(ctx):
    out = ctypes.c_size_t()
    _check(lib().pgc_workspace_bytes(ctx, ctypes.byref(out)), ctx)
    return out.value


def pgc_bind_workspace(ctx, workspace, nbytes=None):
    if nbytes is None:
        nbytes = workspace.numel() * workspace.element_size()
    _check(lib().pgc_bind_workspace(ctx, _P(_dev(workspace)), int(nbytes)), ctx)


def pgc_step(ctx, X, y, w, straggler_mask, lr, n):
    import torch
    _, mp = _mask_arg(straggler_mask, n)
    _check(lib().pgc_step(ctx, _P(_dev(X)), _P(_dev(y)), _P(_dev(w, torch.float32)), mp,
                          ctypes.c_float(lr)), ctx)


def pgc_step_noalloc(ctx, X, y, w, straggler_mask, lr, n):
    """pgc_step with the partial sums in the library's fixed device array."""
    import torch
    _, mp = _mask_arg(straggler_mask, n)
    _check(lib().pgc_step_noalloc(ctx, _P(_dev(X)), _P(_dev(y)), _P(_dev(w, torch.float32)), mp,
                                  ctypes.c_float(lr)), ctx)


def pgc_decode_coeffs(ctx, straggler_mask, n):
    """(survivors int32[|J|], d float64[|J|], scale)."""
    m, mp = _mask_arg(straggler_mask, n)
    d = np.zeros(n, dtype=np.float64)
    surv = np.zeros(n, dtype=np.int32)
    scale = ctypes.c_double()
    nj = ctypes.c_int32()
    _check(lib().pgc_decode_coeffs(ctx, mp, d.ctypes.data_as(_F64P), ctypes.byref(scale),
                                   surv.ctypes.data_as(_I32P), ctypes.byref(nj)), ctx)
    return surv[:nj.value].copy(), d[:nj.value].copy(), scale.value


def pgc_placement(ctx, n, c):
    out = np.zeros(n * c, dtype=np.int32)
    _check(lib().pgc_placement(ctx, out.ctypes.data_as(_I32P)), ctx)
    return out.reshape(n, c)


def pgc_schedule(ctx, t, n):
    out = np.zeros(n, dtype=np.int32)
    _check(lib().pgc_schedule(ctx, int(t), out.ctypes.data_as(_I32P)), ctx)
    return out


def pgc_encoding_matrix(ctx, n):
    out = np.zeros(n * n, dtype=np.float64)
    _check(lib().pgc_encoding_matrix(ctx, out.ctypes.data_as(_F64P)), ctx)
    return out.reshape(n, n)


def pgc_num_coded(ctx):
    out = ctypes.c_int32()
    _check(lib().pgc_num_coded(ctx, ctypes.byref(out)), ctx)
    return out.value


def pgc_make_mask(seed, t, policy, n, cap, p=0.0):
    out = np.zeros(n, dtype=np.uint8)
    _check(lib().pgc_make_mask(int(seed), int(t), int(policy), int(n), int(cap), float(p),
                               out.ctypes.data_as(_U8P)))
    return out


def pgc_delay_step(seed, t, n, s, mean_delay, compute_seconds=0.0):
    """Simulated straggler step: (mask uint8[n], delays float64[n], step_seconds)."""
    mask = np.zeros(n, dtype=np.uint8)
    delays = np.zeros(n, dtype=np.float64)
    step = ctypes.c_double()
    _check(lib().pgc_delay_step(int(seed), int(t), int(n), int(s), float(mean_delay),
                                float(compute_seconds), mask.ctypes.data_as(_U8P),
                                delays.ctypes.data_as(_F64P), ctypes.byref(step)))
    return mask, delays, step.value


def pgc_splitmix64(seed, index):
    out = ctypes.c_uint64()
    _check(lib().pgc_splitmix64(int(seed), int(index), ctypes.byref(out)))
    return out.value


def pgc_state_bytes(ctx):
    out = ctypes.c_size_t()
    _check(lib().pgc_state_bytes(ctx, ctypes.byref(out)), ctx)
    return out.value


def pgc_save_state(ctx, out, nbytes=None):
    if nbytes is None:
        nbytes = out.numel() * out.element_size()
    _check(lib().pgc_save_state(ctx, _P(_dev(out)), int(nbytes)), ctx)


def pgc_load_state(ctx, state, nbytes=None):
    if nbytes is None:
        nbytes = state.numel() * state.element_size()
    _check(lib().pgc_load_state(ctx, _P(_dev(state)), int(nbytes)), ctx)


def pgc_read_ring(ctx, worker, slot, out):
    _check(lib().pgc_read_ring(ctx, int(worker), int(slot), _P(_dev(out))), ctx)


def pgc_read_coded(ctx, index, out):
    _check(lib().pgc_read_coded(ctx, int(index), _P(_dev(out))), ctx)


def pgc_read_decoded(ctx, out):
    _check(lib().pgc_read_decoded(ctx, _P(_dev(out))), ctx)


def pgc_get_step(ctx):
    out = ctypes.c_int64()
    _check(lib().pgc_get_step(ctx, ctypes.byref(out)), ctx)
    return out.value


def pgc_set_timing(ctx, kernels):
    """Time the listed kernels (PGC_KERNEL_* ids); an empty list disables timing,
    True times every kernel."""
    if kernels is True:
        mask = -1
    else:
        mask = 0
        for k in (kernels or ()):
            mask |= 1 << int(k)
    _check(lib().pgc_set_timing(ctx, mask), ctx)


def pgc_set_timing_period(ctx, period):
    """Time one launch in `period` of each selected kernel."""
    _check(lib().pgc_set_timing_period(ctx, int(period)), ctx)


def pgc_kernel_time(ctx, kernel):
    """(total milliseconds, launches) of `kernel` since timing was enabled."""
    ms = ctypes.c_double()
    count = ctypes.c_int64()
    _check(lib().pgc_kernel_time(ctx, int(kernel), ctypes.byref(ms), ctypes.byref(count)), ctx)
    return ms.value, count.value


def pgc_strerror(status):
    return lib().pgc_strerror(int(status)).decode()


def pgc_last_error(ctx):
    return lib().pgc_last_error(ctx).decode()


def pgc_destroy(ctx):
    _check(lib().pgc_destroy(ctx))
