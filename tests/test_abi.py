"""The C ABI library loads and exports every symbol its header declares, and
argument validation answers with error codes before any device work (so
these run without a GPU)."""

import ctypes
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_1806_06144_amd", "libeigenpro.so")

if not os.path.exists(LIB):
    import importlib.util
    _spec = importlib.util.spec_from_file_location(
        "_eigenpro_build", os.path.join(ROOT, "paper_1806_06144_amd", "build.py"))
    _b = importlib.util.module_from_spec(_spec)
    _spec.loader.exec_module(_b)
    _b.build()

import paper_1806_06144_amd as ep  # noqa: E402


def test_exports_every_declared_symbol():
    names = ep.declared_symbols()
    assert len(names) >= 12
    lib = ctypes.CDLL(LIB)
    for name in names:
        assert hasattr(lib, name), name


def _setup_rc(**kw):
    args = dict(ctx=ctypes.byref(ctypes.c_void_p()), X=1, n=100, d=8, l=3, kernel=0,
                bw=1.0, s=10, k=2, sub=None, seed=0, stream=None, info=None)
    args.update(kw)
    return ep.raw_call("ep_setup", args["ctx"], args["X"], args["n"], args["d"], args["l"],
                       args["kernel"], args["bw"], args["s"], args["k"], args["sub"],
                       args["seed"], args["stream"], args["info"])


@pytest.mark.parametrize("kw", [
    dict(ctx=None), dict(X=None), dict(n=0), dict(d=0), dict(l=0),
    dict(k=10), dict(k=-1), dict(s=101), dict(kernel=2), dict(bw=0.0), dict(d=(1 << 20) + 1),
    dict(bw=float("nan")), dict(bw=float("inf")), dict(bw=-1.0),
])
def test_setup_rejects_bad_arguments(kw):
    assert _setup_rc(**kw) == ep.EP_EINVAL
    assert ep.ep_last_error() != ""


def test_calls_on_null_context():
    assert ep.raw_call("ep_step", None, 1, 4, 1, None) == ep.EP_EINVAL
    assert ep.raw_call("ep_predict", None, 1, 4, 1) == ep.EP_EINVAL
    assert ep.raw_call("ep_get_alpha", None, 1) == ep.EP_EINVAL
    assert ep.raw_call("ep_set_alpha", None, 1) == ep.EP_EINVAL
    assert ep.raw_call("ep_sync", None) == ep.EP_EINVAL
    assert ep.raw_call("ep_set_checks", None, 1) == ep.EP_EINVAL
    assert ep.raw_call("ep_timing_enable", None, 1) == ep.EP_EINVAL
    ep.raw_call("ep_destroy", None)


@pytest.mark.parametrize("opts", [
    dict(solver=3), dict(solver=-1), dict(max_degree=-1), dict(max_iters=-2),
    dict(guard=-5), dict(tol=-1e-9), dict(tol=float("nan")), dict(tol=float("inf")),
])
def test_setup_ex_rejects_bad_options(opts):
    o = ep.EpSetupOpts(**opts)
    rc = ep.raw_call("ep_setup_ex", ctypes.byref(ctypes.c_void_p()), 1, 100, 8, 3, 0, 1.0, 10, 2,
                     None, 0, None, ctypes.byref(o), None)
    assert rc == ep.EP_EINVAL
    assert "solver" in ep.ep_last_error() or "option" in ep.ep_last_error()
