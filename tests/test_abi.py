"""The C-ABI library loads and exports every entry point include/hieravg.h
declares; host-side argument checks fail cleanly (no GPU needed: validation
runs before any HIP call)."""

import ctypes
import os
import re

import pytest

from paper_1903_05133_amd import native

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "hieravg.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(hieravg_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = native.lib()
    names = declared_functions()
    assert len(names) >= 14
    for name in names:
        assert hasattr(L, name), name
    assert set(names) == set(native.SIGNATURES)


def test_config_struct_matches_header():
    text = open(HEADER).read()
    body = text[text.index("typedef struct hieravg_config"):text.index("} hieravg_config;")]
    fields = re.findall(r"^\s*(?:int32_t|int64_t|float|uint64_t)\s+(\w+);", body, flags=re.M)
    assert fields == [f for f, _ in native.Config._fields_]


@pytest.mark.parametrize("args,msg", [
    ((0, 1, 1, 1, 1, 0.1, 8, 0), "P must be"),
    ((4, 3, 1, 1, 1, 0.1, 8, 0), "S must divide P"),
    ((4, 2, 0, 1, 1, 0.1, 8, 0), "K1"),
    ((4, 2, 1, 0, 1, 0.1, 8, 0), "K2"),
    ((4, 2, 1, 1, 1, 0.1, 0, 0), "B must be"),
    ((4, 2, 1, 1, 1, 0.1, 65536, 0), "B must be"),
    ((65536, 1, 1, 1, 1, 0.1, 8, 0), "P must be"),
    ((4, 2, 1, 1, 1, float("nan"), 8, 0), "lr"),
    ((4, 2, 1, 1, 1, -0.5, 8, 0), "lr"),
    ((4, 2, 1, 1, 7, 0.1, 8, 0), "unknown model"),
])
def test_invalid_arguments_rejected(args, msg):
    L = native.lib()
    assert not L.hieravg_create(*args)
    assert msg in L.hieravg_last_error().decode()


def test_invalid_config_rejected():
    from paper_1903_05133_amd import config
    L = native.lib()
    c = config(1, 4, 2, 1, 1, B=8, in_dim=10, hidden=0, classes=3, n_samples=10)
    assert not L.hieravg_create_config(ctypes.byref(c))
    assert "hidden" in L.hieravg_last_error().decode()
    c = config(2, 4, 2, 1, 1, in_dim=100, momentum=1.0)
    assert not L.hieravg_create_config(ctypes.byref(c))
    assert "momentum" in L.hieravg_last_error().decode()
    assert not L.hieravg_create_config(None)
    c = config(1, 4, 2, 1, 1, B=8, in_dim=10, hidden=5, classes=3, n_samples=10, update_mode=3)
    assert not L.hieravg_create_config(ctypes.byref(c))
    assert "update_mode" in L.hieravg_last_error().decode()
    # delayed first-layer updates: MLP with B <= 32, K1 <= 8
    for kw in (dict(classes=3, B=33, K1=1), dict(classes=3, B=8, K1=9)):
        c = config(1, 4, 2, kw["K1"], 1, B=kw["B"], in_dim=10, hidden=5, classes=kw["classes"], n_samples=10,
                   update_mode=2)
        assert not L.hieravg_create_config(ctypes.byref(c))
        assert "delayed" in L.hieravg_last_error().decode()
    c = config(0, 4, 2, 1, 1, B=8, in_dim=10, classes=3, n_samples=10, update_mode=2)
    assert not L.hieravg_create_config(ctypes.byref(c))
    # the optimizer fields, for every kind; delayed updates leave the momentum buffers out of the means
    for kw, msg in ((dict(momentum=-0.1), "momentum"), (dict(momentum=1.0), "momentum"),
                    (dict(weight_decay=-1.0), "weight_decay"), (dict(weight_decay=float("inf")), "weight_decay"),
                    (dict(avg_momentum=2), "avg_momentum"),
                    (dict(momentum=0.9, weight_decay=0.1, update_mode=2, avg_momentum=1), "delayed")):
        kw = dict(kw)
        avg_momentum = kw.pop("avg_momentum", None)
        c = config(1, 4, 2, 2, 1, B=8, in_dim=10, hidden=5, classes=3, n_samples=10, **kw)
        if avg_momentum is not None:
            c.avg_momentum = avg_momentum
        assert not L.hieravg_create_config(ctypes.byref(c))
        assert msg in L.hieravg_last_error().decode()
    # momentum and weight decay with unaveraged buffers pass validation in delayed mode
    c = config(1, 4, 2, 2, 1, B=8, in_dim=10, hidden=5, classes=3, n_samples=10, momentum=0.9, weight_decay=0.1,
               update_mode=2)
    h = L.hieravg_create_config(ctypes.byref(c))
    if h:
        L.hieravg_destroy(h)
    else:
        assert "delayed" not in L.hieravg_last_error().decode()


def test_kernel_class_names():
    L = native.lib()
    n = L.hieravg_kernel_classes()
    names = [L.hieravg_kernel_class_name(i) for i in range(n)]
    assert all(names) and len(set(names)) == n
    assert L.hieravg_kernel_class_name(n) == b""


def test_null_handles_are_safe():
    L = native.lib()
    L.hieravg_destroy(None)
    assert L.hieravg_round(None) == native.EINVAL
    assert L.hieravg_dim(None) == native.EINVAL
    assert L.hieravg_params(None, None, 0) == native.EINVAL
    assert L.hieravg_sync(None) == native.EINVAL
    assert L.hieravg_kernel_class_name(-1) == b""
