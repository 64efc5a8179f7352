"""CPU checks of libaep: the library loads, exports every declared entry point,
and its host-side validation / queue accounting / layer picking behave as
documented -- none of these calls touches a GPU."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "aep.h")


def _lib():
    from paper_2505_08944_amd import _lib as L
    if not os.path.exists(L.LIB_PATH):
        pytest.skip("libaep.so not built (run __graft_entry__.build())")
    return L, L.lib()


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+(aep_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported():
    L, lib = _lib()
    names = _declared()
    assert len(names) >= 17
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(L._SIG), "binding and header disagree"


def _cfg(L, **kw):
    base = dict(n_layers=2, n_experts=8, n_shared=0, d_model=256, d_ffn=512, top_k=2, renorm=1,
                act_dtype=L.AEP_BF16, w_dtype=L.AEP_BF16, max_tokens_per_layer=1024)
    base.update(kw)
    return L.Config(**base)


def _create(L, lib, **kw):
    h = ctypes.c_void_p()
    st = lib.aep_create(ctypes.byref(_cfg(L, **kw)), ctypes.byref(h))
    return st, h


def test_status_strings():
    L, lib = _lib()
    for code, name in L.STATUS_NAMES.items():
        assert lib.aep_status_string(code).decode() == name
    assert lib.aep_status_string(99).decode() == "AEP_ERR_UNKNOWN"


@pytest.mark.parametrize("kw,status", [
    (dict(n_layers=0), 1), (dict(n_experts=0), 1), (dict(top_k=0), 1), (dict(top_k=9, n_experts=16), 1),
    (dict(top_k=9), 1), (dict(renorm=2), 1), (dict(max_tokens_per_layer=0), 1),
    (dict(max_tokens_per_layer=1 << 24), 1), (dict(d_model=100), 6), (dict(d_ffn=96), 6),
    (dict(act_dtype=0, w_dtype=1), 6), (dict(act_dtype=1, w_dtype=0), 6), (dict(act_dtype=2), 6),
    (dict(act_dtype=7), 1), (dict(n_experts=1000, n_shared=30), 1),
    # bf16 / fp8 kernels: 32-bit byte offsets into a weight matrix and a group's rows
    (dict(d_model=65536, d_ffn=32768), 6), (dict(d_model=32768, d_ffn=65536, w_dtype=2), 6),
    (dict(max_tokens_per_layer=1 << 22), 6),
])
def test_create_rejects_bad_configs(kw, status):
    L, lib = _lib()
    st, h = _create(L, lib, **kw)
    assert st == status, (kw, st)
    assert not h.value


@pytest.mark.parametrize("kw", [
    dict(d_model=65536, d_ffn=32704), dict(max_tokens_per_layer=(1 << 22) - 1),
    dict(d_model=65536, d_ffn=32768, act_dtype=0, w_dtype=0),  # f32 kernels: no such bound
])
def test_create_accepts_sizes_below_the_offset_bound(kw):
    L, lib = _lib()
    st, h = _create(L, lib, **kw)
    assert st == 0, (kw, st)
    assert lib.aep_destroy(h) == 0


def test_workspace_accounting_and_unbound_state():
    L, lib = _lib()
    st, h = _create(L, lib)
    assert st == 0
    try:
        n1 = ctypes.c_size_t()
        assert lib.aep_workspace_size(h, ctypes.byref(n1)) == 0 and n1.value > 0
        st2, h2 = _create(L, lib, max_tokens_per_layer=2048)
        n2 = ctypes.c_size_t()
        lib.aep_workspace_size(h2, ctypes.byref(n2))
        lib.aep_destroy(h2)
        assert n2.value > n1.value
        # every device-facing call refuses to run without a bound workspace
        b = L.Batch()
        assert lib.aep_route_enqueue(h, 0, 1, 1, 4, None, None, None) == L.AEP_ERR_STATE
        assert lib.aep_rebatch(h, 0, ctypes.byref(b), None) == L.AEP_ERR_STATE
        assert lib.aep_set_expert_weights(h, 0, 0, 1, 1, 1, None, None, None) == L.AEP_ERR_STATE
        assert lib.aep_sync(h, None) == L.AEP_ERR_STATE
        assert lib.aep_expert_ffn(h, ctypes.byref(b), 1, None) == L.AEP_ERR_STATE
        # argument checks come first
        assert lib.aep_route_enqueue(None, 0, 1, 1, 4, None, None, None) == L.AEP_ERR_INVALID_ARG
        assert lib.aep_bind_workspace(h, 0x1001, n1.value, None) == L.AEP_ERR_INVALID_ARG  # misaligned
        assert lib.aep_bind_workspace(h, 0x1000, n1.value - 1, None) == L.AEP_ERR_CAPACITY
        t, r = ctypes.c_int64(-1), ctypes.c_int64(-1)
        assert lib.aep_queue_depth(h, 1, ctypes.byref(t), ctypes.byref(r)) == 0 and (t.value, r.value) == (0, 0)
        assert lib.aep_queue_depth(h, 2, ctypes.byref(t), ctypes.byref(r)) == L.AEP_ERR_INVALID_ARG
        lay = ctypes.c_int32(-1)
        for pol in (0, 1, 2):
            assert lib.aep_pick_layer(h, pol, 0.5, 2, ctypes.byref(lay)) == L.AEP_ERR_EMPTY
        assert lib.aep_pick_layer(h, 7, 0.5, 2, ctypes.byref(lay)) == L.AEP_ERR_INVALID_ARG
        assert lib.aep_pick_layer(h, 2, -1.0, 2, ctypes.byref(lay)) == L.AEP_ERR_INVALID_ARG
        assert lib.aep_fp8_e4m3_to_bf16(None, None, 0, None) == 0
        assert lib.aep_fp8_e4m3_to_bf16(None, None, -1, None) == L.AEP_ERR_INVALID_ARG
    finally:
        assert lib.aep_destroy(h) == 0
    assert lib.aep_destroy(None) == 0


def test_static_workspace_capacity():
    """The static workspace (AEP_STATIC_WORKSPACE_BYTES) holds a Mixtral-shaped
    layer (d=4096, ffn=14336, 8 experts, top-2, bf16) with 900 queued tokens,
    the split-K partial sums included, and not one with 1000; an f32 layer has
    no split-K area (its launches are never split)."""
    L, lib = _lib()

    def need(**kw):
        st, h = _create(L, lib, **kw)
        assert st == 0, (kw, st)
        n = ctypes.c_size_t()
        assert lib.aep_workspace_size(h, ctypes.byref(n)) == 0
        lib.aep_destroy(h)
        return n.value

    mix = dict(n_layers=1, d_model=4096, d_ffn=14336)
    assert need(max_tokens_per_layer=900, **mix) <= L.AEP_STATIC_WORKSPACE_BYTES
    assert need(max_tokens_per_layer=1000, **mix) > L.AEP_STATIC_WORKSPACE_BYTES
    small = dict(n_layers=1, d_model=256, d_ffn=512, max_tokens_per_layer=64)
    bf16 = need(**small)
    f32 = need(act_dtype=L.AEP_F32, w_dtype=L.AEP_F32, **small)
    # a tiny bf16 layer's workspace is mostly its 32 MiB of partial sums; the
    # f32 one has none
    assert bf16 >= 32 << 20 and f32 < 4 << 20, (bf16, f32)
