"""Python binding of libeigenpro: argument marshalling over the C ABI only.

Every function has the name and meaning of its C counterpart in
``include/eigenpro.h``; device arguments may be torch tensors (checked for
dtype, device and contiguity, then passed by pointer) or raw integer device
addresses. All computation happens in the HIP library: if ``libeigenpro.so``
is missing this module raises at import, it never falls back.
"""

import ctypes
import os
import re

_HERE = os.path.dirname(os.path.abspath(__file__))
# EIGENPRO_LIB selects another build of the same library (e.g. to compare
# kernel variants); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("EIGENPRO_LIB") or os.path.join(_HERE, "libeigenpro.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "eigenpro.h")

EP_OK, EP_EINVAL, EP_ENOMEM, EP_EDEVICE, EP_ENUMERIC, EP_EINDEX = 0, -1, -2, -3, -4, -5
EP_GAUSSIAN, EP_LAPLACIAN = 0, 1
EP_SOLVER_AUTO, EP_SOLVER_DENSE, EP_SOLVER_SUBSPACE = 0, 1, 2
EP_CONTRACT_AUTO, EP_CONTRACT_FUSED, EP_CONTRACT_BLOCKED = 0, 1, 2
CONTRACTIONS = {"auto": EP_CONTRACT_AUTO, "fused": EP_CONTRACT_FUSED,
                "blocked": EP_CONTRACT_BLOCKED}
SOLVERS = {"auto": EP_SOLVER_AUTO, "dense": EP_SOLVER_DENSE, "subspace": EP_SOLVER_SUBSPACE}
KERNELS = {"gaussian": EP_GAUSSIAN, "laplacian": EP_LAPLACIAN}
_CODES = {EP_EINVAL: "EP_EINVAL", EP_ENOMEM: "EP_ENOMEM", EP_EDEVICE: "EP_EDEVICE",
          EP_ENUMERIC: "EP_ENUMERIC", EP_EINDEX: "EP_EINDEX"}


class EpInfo(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("d", ctypes.c_int64), ("l", ctypes.c_int64),
                ("s", ctypes.c_int64), ("k", ctypes.c_int64),
                ("sigma_1", ctypes.c_double), ("sigma_k1", ctypes.c_double),
                ("lambda_k1", ctypes.c_double), ("beta", ctypes.c_double),
                ("m_star", ctypes.c_double), ("m", ctypes.c_int64),
                ("eta", ctypes.c_double), ("setup_ms", ctypes.c_double),
                ("k_max", ctypes.c_int64), ("accel", ctypes.c_double),
                ("solver", ctypes.c_int64), ("solver_iters", ctypes.c_int64),
                ("solver_matvecs", ctypes.c_int64), ("eig_residual", ctypes.c_double)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class EpSetupOpts(ctypes.Structure):
    _fields_ = [("solver", ctypes.c_int32), ("max_degree", ctypes.c_int32),
                ("max_iters", ctypes.c_int32), ("no_fallback", ctypes.c_int32),
                ("guard", ctypes.c_int64), ("tol", ctypes.c_double)]


class EpTiming(ctypes.Structure):
    _fields_ = [("kmv_ms", ctypes.c_double), ("kmv_launches", ctypes.c_int64),
                ("step_ms", ctypes.c_double), ("steps", ctypes.c_int64),
                ("kblock_ms", ctypes.c_double), ("kblock_launches", ctypes.c_int64),
                ("gemm_ms", ctypes.c_double), ("gemm_launches", ctypes.c_int64)]


class EigenProError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{_CODES.get(code, code)}: {msg}")
        self.code = code


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "or python paper_1806_06144_amd/build.py")
    # torch ships its own HIP runtime under the same soname; loading torch
    # first makes the library bind to that one, so the process holds a
    # single runtime (two copies would not see each other's devices).
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I, F = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    sig = {
        "ep_setup": (I, [ctypes.POINTER(P), P, I64, I64, I64, I, F, I64, I64, P,
                         ctypes.c_uint64, P, ctypes.POINTER(EpInfo)]),
        "ep_setup_ex": (I, [ctypes.POINTER(P), P, I64, I64, I64, I, F, I64, I64, P,
                            ctypes.c_uint64, P, ctypes.POINTER(EpSetupOpts),
                            ctypes.POINTER(EpInfo)]),
        "ep_restore": (I, [ctypes.POINTER(P), P, I64, I64, I64, I, F, I64, I64, P, P, P, P,
                           ctypes.POINTER(EpInfo)]),
        "ep_step": (I, [P, P, I64, P, P]),
        "ep_predict": (I, [P, P, I64, P]),
        "ep_predict_noalloc": (I, [P, P, I64, P]),
        "ep_get_alpha": (I, [P, P]),
        "ep_set_alpha": (I, [P, P]),
        "ep_get_preconditioner": (I, [P, P, P, P, P]),
        "ep_get_info": (I, [P, ctypes.POINTER(EpInfo)]),
        "ep_set_checks": (I, [P, I]),
        "ep_set_rank": (I, [P, I64]),
        "ep_set_contraction": (I, [P, I, I64]),
        "ep_adapt": (I, [P, I64, ctypes.POINTER(EpInfo)]),
        "ep_batch_sweep": (I, [P, P, I, I, P]),
        "ep_resource_batch": (I, [P, ctypes.c_double, ctypes.POINTER(I64), ctypes.POINTER(I64),
                                  ctypes.POINTER(I64)]),
        "ep_batch_knee": (I, [P, P, I, ctypes.c_double, ctypes.POINTER(I64),
                              ctypes.POINTER(ctypes.c_double)]),
        "ep_timing_enable": (I, [P, I]),
        "ep_timing_read": (I, [P, ctypes.POINTER(EpTiming)]),
        "ep_sync": (I, [P]),
        "ep_device_probe": (I, [P, P]),
        "ep_destroy": (None, [P]),
        "ep_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()


def declared_symbols():
    """Names of the functions declared in include/eigenpro.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ep_[a-z_0-9]+)\s*\(", text)))


def _check(rc):
    if rc != EP_OK:
        raise EigenProError(rc, _lib.ep_last_error().decode())
    return rc


def _ptr(x, dtype=None, allow_none=False):
    """Device address of a tensor (validated) or an integer address."""
    if x is None:
        if allow_none:
            return None
        raise ValueError("a device buffer is required")
    if isinstance(x, int):
        return x
    if not x.is_cuda:
        raise ValueError("expected a device tensor")
    if dtype is not None and x.dtype != dtype:
        raise TypeError(f"expected {dtype}, got {x.dtype}")
    if not x.is_contiguous():
        raise ValueError("expected a contiguous tensor")
    return x.data_ptr()


def _torch():
    import torch
    return torch


def _stream_handle(stream):
    if stream is None:
        return _torch().cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def ep_last_error():
    return _lib.ep_last_error().decode()


def ep_setup(X, n, d, l, kernel, bandwidth, s, k, sub_idx=None, seed=0, stream=None):
    """Returns (ctx, EpInfo). X: device float32 n x d (borrowed: keep it
    alive until ep_destroy). sub_idx: host int64 sequence of s indices or
    None."""
    return ep_setup_ex(X, n, d, l, kernel, bandwidth, s, k, sub_idx, seed, stream, None)


def ep_setup_ex(X, n, d, l, kernel, bandwidth, s, k, sub_idx=None, seed=0, stream=None,
                opts=None):
    """ep_setup with setup options: ``opts`` is an EpSetupOpts, a dict of its
    fields (``solver`` may be "auto", "dense" or "subspace"), or None."""
    torch = _torch()
    if isinstance(kernel, str):
        kernel = KERNELS[kernel]
    xp = _ptr(X, torch.float32)
    sub_ptr = None
    keep = None
    if sub_idx is not None:
        import numpy as np
        keep = np.ascontiguousarray(np.asarray(sub_idx, dtype=np.int64))
        if keep.shape != (s,):
            raise ValueError("sub_idx must hold s indices")
        sub_ptr = keep.ctypes.data
    if isinstance(opts, dict):
        o = dict(opts)
        if isinstance(o.get("solver"), str):
            o["solver"] = SOLVERS[o["solver"]]
        opts = EpSetupOpts(**o)
    ctx = ctypes.c_void_p()
    info = EpInfo()
    if opts is None:
        _check(_lib.ep_setup(ctypes.byref(ctx), xp, n, d, l, kernel, bandwidth, s, k, sub_ptr,
                             seed, _stream_handle(stream), ctypes.byref(info)))
    else:
        _check(_lib.ep_setup_ex(ctypes.byref(ctx), xp, n, d, l, kernel, bandwidth, s, k,
                                sub_ptr, seed, _stream_handle(stream), ctypes.byref(opts),
                                ctypes.byref(info)))
    return ctx, info


def ep_restore(X, n, d, l, kernel, bandwidth, s, k, sub_idx, sigma, V, stream=None):
    """Rebuild a context from a saved setup (sub_idx, sigma[k+1], V[s, k] as
    returned by ep_get_preconditioner). Returns (ctx, EpInfo)."""
    import numpy as np
    torch = _torch()
    if isinstance(kernel, str):
        kernel = KERNELS[kernel]
    r = np.ascontiguousarray(np.asarray(sub_idx, dtype=np.int64))
    sg = np.ascontiguousarray(np.asarray(sigma, dtype=np.float64))
    if r.shape != (s,) or sg.shape != (k + 1,):
        raise ValueError("sub_idx must hold s entries and sigma k+1")
    Vh = np.ascontiguousarray(np.asarray(V, dtype=np.float32).reshape(s, k)) if k else None
    ctx = ctypes.c_void_p()
    info = EpInfo()
    _check(_lib.ep_restore(ctypes.byref(ctx), _ptr(X, torch.float32), n, d, l, kernel,
                           bandwidth, s, k, r.ctypes.data, sg.ctypes.data,
                           Vh.ctypes.data if Vh is not None else None,
                           _stream_handle(stream), ctypes.byref(info)))
    return ctx, info


def ep_step(ctx, t, m, y_b, f_out=None):
    torch = _torch()
    return _check(_lib.ep_step(ctx, _ptr(t, torch.int64), m, _ptr(y_b, torch.float32),
                               _ptr(f_out, torch.float32, allow_none=True)))


def ep_predict(ctx, Z, n_z, out):
    torch = _torch()
    return _check(_lib.ep_predict(ctx, _ptr(Z, torch.float32), n_z, _ptr(out, torch.float32)))


def ep_predict_noalloc(ctx, Z, n_z, out):
    torch = _torch()
    return _check(_lib.ep_predict_noalloc(ctx, _ptr(Z, torch.float32), n_z,
                                          _ptr(out, torch.float32)))


def ep_get_alpha(ctx, out):
    return _check(_lib.ep_get_alpha(ctx, _ptr(out, _torch().float32)))


def ep_set_alpha(ctx, alpha):
    return _check(_lib.ep_set_alpha(ctx, _ptr(alpha, _torch().float32)))


def ep_get_preconditioner(ctx, info):
    """Returns numpy (sigma[k+1], D[k], V[s, k] float32, r[s])."""
    import numpy as np
    k, s = info.k, info.s
    sigma = np.zeros(k + 1, dtype=np.float64)
    D = np.zeros(max(k, 1), dtype=np.float64)
    V = np.zeros((s, max(k, 1)), dtype=np.float32)
    r = np.zeros(s, dtype=np.int64)
    _check(_lib.ep_get_preconditioner(ctx, sigma.ctypes.data, D.ctypes.data, V.ctypes.data,
                                      r.ctypes.data))
    return sigma, D[:k], V[:, :k], r


def ep_get_info(ctx):
    info = EpInfo()
    _check(_lib.ep_get_info(ctx, ctypes.byref(info)))
    return info


def ep_set_rank(ctx, k):
    return _check(_lib.ep_set_rank(ctx, k))


def ep_set_contraction(ctx, mode, block_bytes=0):
    """mode: EP_CONTRACT_* or "auto" / "fused" / "blocked"; block_bytes: cap
    of the blocked form's kernel-block buffer (0: 2 GiB)."""
    if isinstance(mode, str):
        mode = CONTRACTIONS[mode]
    return _check(_lib.ep_set_contraction(ctx, mode, block_bytes))


def ep_adapt(ctx, m_G):
    info = EpInfo()
    _check(_lib.ep_adapt(ctx, m_G, ctypes.byref(info)))
    return info


def ep_batch_sweep(ctx, ms, reps=3):
    """ms per fused step-2 pass for each batch size in ms."""
    import numpy as np
    arr = np.ascontiguousarray(np.asarray(ms, dtype=np.int64))
    out = np.zeros(arr.shape[0], dtype=np.float64)
    _check(_lib.ep_batch_sweep(ctx, arr.ctypes.data, arr.shape[0], reps, out.ctypes.data))
    return out


def ep_resource_batch(ctx, tol=0.1):
    """(m_C, m_S, m_G) of Section 3 Step 1."""
    mc, ms, mg = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.ep_resource_batch(ctx, tol, ctypes.byref(mc), ctypes.byref(ms), ctypes.byref(mg)))
    return mc.value, ms.value, mg.value


def ep_batch_knee(ms, ms_per_pass, tol=0.1):
    """(m_C, knee) of a time-per-iteration curve (host only)."""
    import numpy as np
    m = np.ascontiguousarray(np.asarray(ms, dtype=np.int64))
    t = np.ascontiguousarray(np.asarray(ms_per_pass, dtype=np.float64))
    if m.shape != t.shape:
        raise ValueError("ms and ms_per_pass differ in length")
    mc, kn = ctypes.c_int64(), ctypes.c_double()
    _check(_lib.ep_batch_knee(m.ctypes.data, t.ctypes.data, m.shape[0], tol, ctypes.byref(mc),
                              ctypes.byref(kn)))
    return mc.value, kn.value


def ep_set_checks(ctx, on):
    return _check(_lib.ep_set_checks(ctx, 1 if on else 0))


def ep_timing_enable(ctx, on):
    return _check(_lib.ep_timing_enable(ctx, 1 if on else 0))


def ep_timing_read(ctx):
    t = EpTiming()
    _check(_lib.ep_timing_read(ctx, ctypes.byref(t)))
    return t


def ep_device_probe():
    """(sustained fp32 MFMA TFLOP/s, shader clock MHz) of the current device."""
    tf = ctypes.c_double()
    mhz = ctypes.c_double()
    _check(_lib.ep_device_probe(ctypes.byref(tf), ctypes.byref(mhz)))
    return tf.value, mhz.value


def ep_sync(ctx):
    return _check(_lib.ep_sync(ctx))


def ep_destroy(ctx):
    _lib.ep_destroy(ctx)


def raw_call(name, *args):
    """Call a C entry point with already-marshalled arguments and return its
    integer status (used to exercise error paths)."""
    return getattr(_lib, name)(*args)
