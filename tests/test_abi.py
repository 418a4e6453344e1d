"""C-ABI checks that run without a GPU: the library loads, exports every
function include/caee.h declares, and rejects bad arguments on the host
before launching anything."""
import ctypes
import os
import re

import pytest

from paper_2606_29982_amd import caee

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = 0x10000   # aligned, never dereferenced: every call below fails validation or has T = 0


def _declared():
    with open(os.path.join(ROOT, "include", "caee.h")) as fh:
        text = fh.read()
    return sorted(set(re.findall(r"\b(caee_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    names = _declared()
    assert "caee_moe_layer" in names and "caee_route_prune" in names and "caee_expert_ffn" in names
    lib = ctypes.CDLL(caee.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(caee.EXPORTED)
    assert caee.abi_version() == 8


def _layer(**kw):
    base = dict(T=32, d=7168, f=2048, E=256, n_group=8, topk_group=4, k=8, n_shared=1,
                routed_scaling=2.5, tau=0.05, n_bins=8)
    base.update(kw)
    return caee.Layer(**base)


def _ws_status(layer):
    n = ctypes.c_size_t(0)
    d = layer.desc()
    return caee.lib.caee_workspace_size(ctypes.byref(d), ctypes.byref(n)), n.value


@pytest.mark.parametrize("kw,status", [
    (dict(), caee.CAEE_OK),
    (dict(T=-1), caee.CAEE_ERR_INVALID_ARG),
    (dict(d=7000), caee.CAEE_ERR_INVALID_ARG),
    (dict(f=0), caee.CAEE_ERR_INVALID_ARG),
    (dict(E=257), caee.CAEE_ERR_INVALID_ARG),
    (dict(n_group=7), caee.CAEE_ERR_INVALID_ARG),
    (dict(topk_group=9), caee.CAEE_ERR_INVALID_ARG),
    (dict(k=17), caee.CAEE_ERR_INVALID_ARG),
    (dict(k=8, topk_group=1, n_group=64), caee.CAEE_ERR_INVALID_ARG),   # 4 experts per group < k
    (dict(n_shared=5), caee.CAEE_ERR_INVALID_ARG),
    (dict(routed_scaling=0.0), caee.CAEE_ERR_INVALID_ARG),
    (dict(routed_scaling=float("inf")), caee.CAEE_ERR_INVALID_ARG),
    (dict(tau=-0.1), caee.CAEE_ERR_INVALID_ARG),
    (dict(tau=float("nan")), caee.CAEE_ERR_INVALID_ARG),
    (dict(n_bins=0), caee.CAEE_ERR_INVALID_ARG),
    (dict(n_bins=300), caee.CAEE_ERR_INVALID_ARG),
    (dict(x_dtype="f32"), caee.CAEE_ERR_INVALID_ARG),
    (dict(y_dtype="fp8"), caee.CAEE_ERR_INVALID_ARG),
    (dict(T=65537), caee.CAEE_ERR_UNSUPPORTED),
    (dict(E=192, n_group=8), caee.CAEE_ERR_UNSUPPORTED),      # 24 per group, 4 per lane: 6 lanes
])
def test_descriptor_validation(kw, status):
    st, n = _ws_status(_layer(**kw))
    assert st == status, caee.lib.caee_last_error().decode()
    if st != caee.CAEE_OK:
        assert caee.lib.caee_last_error().decode()


def test_keep_top1_must_be_a_flag():
    d = _layer().desc()
    n = ctypes.c_size_t(0)
    for v, status in ((0, caee.CAEE_OK), (1, caee.CAEE_OK), (2, caee.CAEE_ERR_INVALID_ARG),
                      (-1, caee.CAEE_ERR_INVALID_ARG)):
        d.keep_top1 = v
        assert caee.lib.caee_workspace_size(ctypes.byref(d), ctypes.byref(n)) == status


def test_workspace_size_monotone_in_T():
    sizes = [_ws_status(_layer(T=t))[1] for t in (0, 1, 8, 32, 128)]
    assert sizes == sorted(sizes) and sizes[0] > 0


def _route(layer, logits=FAKE, cost=FAKE, bins=FAKE, out=True, ws=FAKE, ws_bytes=None, bias=None):
    d = layer.desc()
    n = _ws_status(layer)[1] if ws_bytes is None else ws_bytes
    ro = caee.RouteOut(FAKE, FAKE, None, None, None, None) if out else None
    return caee.lib.caee_route_prune(ctypes.byref(d), logits, bias, cost, bins,
                                     ctypes.byref(ro) if ro is not None else None, ws, n, None)


def test_route_prune_host_checks():
    L = _layer()
    assert _route(L, logits=None) == caee.CAEE_ERR_INVALID_ARG
    assert _route(L, cost=None) == caee.CAEE_ERR_INVALID_ARG
    assert _route(L, logits=FAKE + 4) == caee.CAEE_ERR_INVALID_ARG        # misaligned
    assert _route(L, bins=None) == caee.CAEE_ERR_INVALID_ARG              # n_bins=8 needs a bin map
    assert _route(L, out=False) == caee.CAEE_ERR_INVALID_ARG
    assert _route(L, ws=None) == caee.CAEE_ERR_WORKSPACE
    assert _route(L, ws=FAKE + 16) == caee.CAEE_ERR_WORKSPACE             # not 256-aligned
    assert _route(L, ws_bytes=_ws_status(L)[1] - 1) == caee.CAEE_ERR_WORKSPACE
    # an empty batch is valid and launches nothing
    assert _route(_layer(T=0)) == caee.CAEE_OK


def test_ffn_and_layer_host_checks():
    L = _layer()
    d = L.desc()
    n = _ws_status(L)[1]
    W = caee.ExpertWeights(FAKE, FAKE, None, None, FAKE, FAKE, None, None)
    ffn = lambda desc, w, x=FAKE: caee.lib.caee_expert_ffn(  # noqa: E731
        ctypes.byref(desc), x, FAKE, FAKE, ctypes.byref(w) if w is not None else None, FAKE, FAKE, n, None)
    assert ffn(d, None) == caee.CAEE_ERR_INVALID_ARG
    assert ffn(d, W, x=None) == caee.CAEE_ERR_INVALID_ARG
    no_sh = caee.ExpertWeights(FAKE, FAKE, None, None, None, None, None, None)
    assert ffn(d, no_sh) == caee.CAEE_ERR_INVALID_ARG                     # n_shared=1 needs shared weights
    scaled = caee.ExpertWeights(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, None)
    assert ffn(d, scaled) == caee.CAEE_ERR_INVALID_ARG                    # scales only for fp8
    d0 = _layer(T=0).desc()
    assert ffn(d0, W) == caee.CAEE_OK
    layer_call = caee.lib.caee_moe_layer(ctypes.byref(d0), FAKE, FAKE, None, FAKE, FAKE, ctypes.byref(W),
                                         FAKE, None, FAKE, n, None)
    assert layer_call == caee.CAEE_OK
    layer_call = caee.lib.caee_moe_layer(ctypes.byref(d), FAKE, FAKE, None, FAKE, FAKE, ctypes.byref(W),
                                         None, None, FAKE, n, None)
    assert layer_call == caee.CAEE_ERR_INVALID_ARG                        # y missing


def test_status_strings_and_timing_kinds():
    for s in range(5):
        assert caee.lib.caee_status_str(s)
    ms, cnt = ctypes.c_double(), ctypes.c_int64()
    assert caee.lib.caee_timing_query(9, ctypes.byref(ms), ctypes.byref(cnt)) == caee.CAEE_ERR_INVALID_ARG
    assert caee.lib.caee_timing_query(0, ctypes.byref(ms), ctypes.byref(cnt)) == caee.CAEE_OK


def test_pack_matrix_host_checks():
    pk = caee.lib.caee_pack_matrix
    assert pk(9, FAKE, FAKE * 16, 32, 64, 1, None) == caee.CAEE_ERR_INVALID_ARG
    assert pk(caee.CAEE_BF16, FAKE, FAKE * 16, 24, 64, 1, None) == caee.CAEE_ERR_INVALID_ARG    # rows % 16
    assert pk(caee.CAEE_BF16, FAKE, FAKE * 16, 32, 16, 1, None) == caee.CAEE_ERR_INVALID_ARG    # 32-byte rows
    assert pk(caee.CAEE_BF16, None, FAKE * 16, 32, 64, 1, None) == caee.CAEE_ERR_INVALID_ARG
    assert pk(caee.CAEE_BF16, FAKE, FAKE + 1024, 32, 64, 1, None) == caee.CAEE_ERR_INVALID_ARG  # overlap
    assert pk(caee.CAEE_BF16, FAKE, FAKE * 16, 32, 64, 0, None) == caee.CAEE_OK                 # nothing to do
    W = caee.ExpertWeights(FAKE, FAKE, None, None, FAKE, FAKE, None, None, 7)
    d = _layer().desc()
    n = _ws_status(_layer())[1]
    assert caee.lib.caee_expert_ffn(ctypes.byref(d), FAKE, FAKE, FAKE, ctypes.byref(W), FAKE, FAKE, n,
                                    None) == caee.CAEE_ERR_INVALID_ARG                          # unknown layout


def test_quantize_rows_host_checks():
    qr = caee.lib.caee_quantize_rows
    assert qr(caee.CAEE_FP8_E4M3, FAKE, 4, 128, FAKE, FAKE, None) == caee.CAEE_ERR_INVALID_ARG
    assert qr(caee.CAEE_BF16, FAKE, 4, 100, FAKE, FAKE, None) == caee.CAEE_ERR_INVALID_ARG
    assert qr(caee.CAEE_BF16, None, 4, 128, FAKE, FAKE, None) == caee.CAEE_ERR_INVALID_ARG
    assert qr(caee.CAEE_F32, FAKE, 0, 128, FAKE, FAKE, None) == caee.CAEE_OK


def _offload_status(layer=None, **kw):
    layer = layer or _layer(T=0, n_bins=1)
    E = layer.E
    arr = (ctypes.c_void_p * E)(*([FAKE] * E))
    fields = dict(host_w13=ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)),
                  host_w2=ctypes.cast(arr, ctypes.POINTER(ctypes.c_void_p)),
                  slot_w13=FAKE, slot_w2=FAKE, sh_w13=FAKE, sh_w2=FAKE, layout=1, n_cache=4, n_stage=2,
                  fetch_batch=2, miss_cost=1.0)
    fields.update(kw)
    od = caee.OffloadDesc(**fields)
    d = layer.desc()
    h = ctypes.c_void_p(None)
    st = caee.lib.caee_offload_create(ctypes.byref(d), ctypes.byref(od), ctypes.byref(h))
    assert not h.value
    return st


@pytest.mark.parametrize("kw", [dict(n_cache=0, n_stage=0), dict(n_cache=-1), dict(fetch_batch=0),
                                dict(miss_cost=0.0), dict(miss_cost=float("nan")), dict(layout=7),
                                dict(slot_w13=None), dict(slot_w2=FAKE + 4), dict(sh_w13=None),
                                dict(host_w13=None)])
def test_offload_create_rejects_bad_arguments(kw):
    assert _offload_status(**kw) == caee.CAEE_ERR_INVALID_ARG


def test_offload_create_rejects_fp8_and_bad_layer():
    assert _offload_status(_layer(T=0, n_bins=1, w_dtype="fp8")) == caee.CAEE_ERR_UNSUPPORTED
    assert _offload_status(_layer(T=0, n_bins=1, E=192)) == caee.CAEE_ERR_UNSUPPORTED
    assert _offload_status(_layer(T=0, n_bins=1, k=0)) == caee.CAEE_ERR_INVALID_ARG


def test_offload_null_handle():
    d = _layer(T=4, n_bins=1).desc()
    st = caee.lib.caee_offload_layer(None, ctypes.byref(d), FAKE, FAKE, None, FAKE, None, FAKE, 1 << 20, None,
                                     None)
    assert st == caee.CAEE_ERR_INVALID_ARG
    caee.lib.caee_offload_destroy(None)
    assert caee.lib.caee_offload_reset(None) == caee.CAEE_ERR_INVALID_ARG


def test_noalloc_refuses_oversize_and_empty_calls_on_the_host():
    # a batch whose workspace exceeds the library's scratch array is refused
    # before any launch; an empty batch does nothing (no GPU needed for either)
    w = caee.ExpertWeights(FAKE, FAKE, None, None, FAKE, FAKE, None, None, 1)
    for T, status in ((256, caee.CAEE_ERR_UNSUPPORTED), (0, caee.CAEE_OK)):
        layer = _layer(T=T)
        d = layer.desc()
        st = caee.lib.caee_moe_layer_noalloc(ctypes.byref(d), FAKE, FAKE, None, FAKE, FAKE, ctypes.byref(w),
                                             FAKE, None, None)
        assert st == status, caee.lib.caee_last_error().decode()
    assert caee.workspace_size(_layer(T=128)) <= caee.SCRATCH_BYTES < caee.workspace_size(_layer(T=256))
    # invalid arguments are rejected as by caee_moe_layer
    d = _layer(k=17).desc()
    assert caee.lib.caee_moe_layer_noalloc(ctypes.byref(d), FAKE, FAKE, None, FAKE, FAKE, ctypes.byref(w), FAKE,
                                           None, None) == caee.CAEE_ERR_INVALID_ARG
