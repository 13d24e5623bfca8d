"""The C-ABI boundary on the CPU (no GPU needed): the library loads, exports every entry
point that include/gs.h declares, rejects invalid configurations before touching the
device, and the product package never touches the oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2108_06004_amd as gs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gs.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gs_[a-z_]+)\s*\(", text)))


def test_header_declares_the_five_steps_and_helpers():
    names = declared_functions()
    for n in ("gs_accumulate", "gs_sketch", "gs_merge", "gs_unsketch_topk", "gs_gather_reset", "gs_step",
              "gs_create", "gs_destroy", "gs_status_string", "gs_last_error"):
        assert n in names
    assert set(names) == set(gs.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = gs.load_library()
    for n in declared_functions():
        assert hasattr(lib, n), n


def test_status_strings():
    lib = gs.load_library()
    for st in range(5):
        assert lib.gs_status_string(st)
    assert lib.gs_status_string(99) == b"unknown status"


def _cfg(**over):
    hp = {"a": [1, 2, 3], "b": [0, 5, 7], "a2": [9, 10, 11], "b2": [1, 1, 1]}
    kw = dict(d=1000, P=4, r=3, c=50, k_max=10, rho=0.9, reset_momentum=1, state_layout=0, options=0)
    kw.update({k: v for k, v in over.items() if k in kw})
    hp.update({k: v for k, v in over.items() if k in hp})
    keep = [np.ascontiguousarray(hp[k], dtype=np.uint32) for k in ("a", "b", "a2", "b2")]
    u32p = ctypes.POINTER(ctypes.c_uint32)
    cfg = gs.gs_config(kw["d"], kw["P"], kw["r"], kw["c"], kw["k_max"], kw["rho"], kw["reset_momentum"],
                       *(a.ctypes.data_as(u32p) for a in keep), kw["state_layout"], kw["options"])
    return cfg, keep


P31 = (1 << 31) - 1


@pytest.mark.parametrize("over", [
    dict(d=0), dict(d=P31), dict(P=0), dict(P=65), dict(r=0), dict(r=17, a=[1] * 17, b=[0] * 17, a2=[1] * 17,
                                                                         b2=[0] * 17),
    dict(c=0), dict(c=P31), dict(k_max=0), dict(k_max=1001), dict(rho=float("nan")), dict(rho=float("inf")),
    dict(a=[0, 2, 3]), dict(a=[1, P31, 3]), dict(b=[0, P31, 0]), dict(a2=[1, 0, 1]), dict(b2=[P31, 0, 0]),
    dict(state_layout=2), dict(state_layout=-1), dict(options=2), dict(options=-1),
])
def test_create_rejects_invalid_config_before_any_device_call(over):
    lib = gs.load_library()
    cfg, keep = _cfg(**over)
    out = ctypes.c_void_p(12345)
    st = lib.gs_create(ctypes.byref(cfg), ctypes.byref(out))
    assert st == gs.GS_ERR_INVALID_ARG
    assert out.value is None
    assert lib.gs_last_error(None)


def test_create_rejects_null_pointers():
    lib = gs.load_library()
    out = ctypes.c_void_p()
    assert lib.gs_create(None, ctypes.byref(out)) == gs.GS_ERR_INVALID_ARG
    cfg, keep = _cfg()
    assert lib.gs_create(ctypes.byref(cfg), None) == gs.GS_ERR_INVALID_ARG
    cfg.hash_b = None
    assert lib.gs_create(ctypes.byref(cfg), ctypes.byref(out)) == gs.GS_ERR_INVALID_ARG


def test_calls_reject_null_context():
    lib = gs.load_library()
    assert lib.gs_accumulate(None, None, None, None, None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_sketch(None, None, None, None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_merge(None, None, None, None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_unsketch_topk(None, None, None, 1, None, None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_gather_reset(None, None, None, 1, None, None, None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_step(None, None, None, None, None, 1, None, None, None) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_destroy(None) == gs.GS_OK


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(gs, "LIB_PATH", os.path.join(ROOT, "does-not-exist", "libgs.so"))
    monkeypatch.setattr(gs, "_lib", None)
    with pytest.raises(gs.GsLibraryMissing):
        gs.load_library()


def test_product_never_touches_the_oracle():
    pkg = os.path.join(ROOT, "paper_2108_06004_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".hpp", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"\boracle\b|gs_oracle|\bora_", text), os.path.join(dirpath, f)


def test_state_layout_conversions():
    # the binding's [P][d] <-> state-layout helpers (pure tensor rearrangement, CPU tensors)
    torch = pytest.importorskip("torch")
    for P, layout, shape in [(3, "interleaved", (7, 4)), (8, "interleaved", (7, 8)), (3, "worker_major", (3, 7))]:
        ctx = gs.GsContext.__new__(gs.GsContext)
        ctx.d, ctx.P, ctx.state_layout, ctx.handle = 7, P, layout, None
        assert ctx.state_shape == shape and ctx.state_numel() == shape[0] * shape[1]
        x = torch.arange(P * 7, dtype=torch.float32).reshape(P, 7)
        st = ctx.to_state(x)
        assert tuple(st.shape) == shape
        if layout == "interleaved":
            assert st[2, 1] == x[1, 2] and torch.all(st[:, P:] == 0)
        assert torch.equal(ctx.from_state(st), x)
    assert gs.state_stride(1) == 4 and gs.state_stride(8) == 8 and gs.state_stride(17) == 20


def test_static_selection_rejects_invalid_arguments_before_any_device_call():
    lib = gs.load_library()
    fake = ctypes.c_void_p(256)  # never dereferenced: the checks fail first
    cfg, keep = _cfg(d=gs.GS_STATIC_MAX_D + 1)
    assert lib.gs_unsketch_topk_static(ctypes.byref(cfg), None, fake, 1, None, fake) == gs.GS_ERR_INVALID_ARG
    assert b"GS_STATIC_MAX_D" in lib.gs_last_error(None)
    cfg, keep = _cfg(d=1000)
    assert lib.gs_unsketch_topk_static(ctypes.byref(cfg), None, fake, 1001, None, fake) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_unsketch_topk_static(ctypes.byref(cfg), None, None, 1, None, fake) == gs.GS_ERR_INVALID_ARG
    assert lib.gs_unsketch_topk_static(None, None, fake, 1, None, fake) == gs.GS_ERR_INVALID_ARG
    cfg, keep = _cfg(a=[0, 2, 3])
    assert lib.gs_unsketch_topk_static(ctypes.byref(cfg), None, fake, 1, None, fake) == gs.GS_ERR_INVALID_ARG
