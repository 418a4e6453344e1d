"""ctypes binding of the CAEE C ABI (include/caee.h).

Argument marshalling only: every step of the layer runs in the HIP kernels
of ``libcaee.so``.  Tensors are torch CUDA tensors (device memory); the
current torch stream of the tensors' device is passed to the library.
Importing this module fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
# CAEE_LIBRARY names another build of the library (e.g. the host-sanitized one).
LIB_PATH = os.environ.get("CAEE_LIBRARY") or os.path.join(HERE, "libcaee.so")

CAEE_OK, CAEE_ERR_INVALID_ARG, CAEE_ERR_UNSUPPORTED, CAEE_ERR_WORKSPACE, CAEE_ERR_HIP, CAEE_ERR_CAPACITY = range(6)
CAEE_F32, CAEE_BF16, CAEE_FP8_E4M3 = 0, 1, 2
KERNEL_KINDS = {"route": 0, "gate_up": 1, "down": 2, "combine": 3, "quant": 4}
DTYPE_CODE = {"f32": CAEE_F32, "bf16": CAEE_BF16, "fp8": CAEE_FP8_E4M3}
IMPORTANCE_CODE = {"max": 0, "sum": 1, "cir": 2}
REFILL_CODE = {"score": 0, "none": 1, "random": 2, "literal": 3}


class CaeeError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"caee status {status}: {message}")
        self.status = status


class LayerDesc(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("T", "d", "f", "E", "n_group", "topk_group", "k", "n_shared")] + [
        ("routed_scaling", ctypes.c_float), ("tau", ctypes.c_float),
        ("n_bins", ctypes.c_int32), ("importance", ctypes.c_int32),
        ("x_dtype", ctypes.c_int32), ("w_dtype", ctypes.c_int32), ("y_dtype", ctypes.c_int32),
        ("refill", ctypes.c_int32), ("seed", ctypes.c_uint32), ("keep_top1", ctypes.c_int32)]


class ExpertWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("w13", "w2", "w13_scale", "w2_scale", "sh_w13", "sh_w2", "sh_w13_scale", "sh_w2_scale")] + [
        ("layout", ctypes.c_int32)]


LAYOUT_ROWMAJOR, LAYOUT_TILED = 0, 1
STATS = 9   # entries of caee_route_out_t.stats


class OffloadDesc(ctypes.Structure):
    _fields_ = [("host_w13", ctypes.POINTER(ctypes.c_void_p)), ("host_w2", ctypes.POINTER(ctypes.c_void_p)),
                ("slot_w13", ctypes.c_void_p), ("slot_w2", ctypes.c_void_p),
                ("sh_w13", ctypes.c_void_p), ("sh_w2", ctypes.c_void_p),
                ("layout", ctypes.c_int32), ("n_cache", ctypes.c_int32), ("n_stage", ctypes.c_int32),
                ("fetch_batch", ctypes.c_int32), ("miss_cost", ctypes.c_float)]


class OffloadStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in
                ("calls", "needed", "hits", "misses", "staged", "evictions", "bytes_h2d")] + [
        ("passes", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class RouteOut(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in
                ("topk_ids", "topk_w", "orig_ids", "masks", "stats", "bin_loads")]


def _load(path: str = LIB_PATH):
    if not os.path.exists(path):
        raise ImportError(f"{path} is missing: build it with __graft_entry__.build() "
                          "(python -c 'import __graft_entry__ as g; g.build()')")
    # torch ships its own HIP runtime; importing it first makes the library
    # bind to that same runtime (one HIP runtime per process) instead of
    # loading a second copy that would not see the device torch opened.
    import torch  # noqa: F401
    lib = ctypes.CDLL(path)
    st = ctypes.c_int
    P = ctypes.c_void_p
    desc_p = ctypes.POINTER(LayerDesc)
    sig = {
        "caee_workspace_size": (st, [desc_p, ctypes.POINTER(ctypes.c_size_t)]),
        "caee_route_prune": (st, [desc_p, P, P, P, P, ctypes.POINTER(RouteOut), P, ctypes.c_size_t, P]),
        "caee_expert_ffn": (st, [desc_p, P, P, P, ctypes.POINTER(ExpertWeights), P, P, ctypes.c_size_t, P]),
        "caee_moe_layer": (st, [desc_p, P, P, P, P, P, ctypes.POINTER(ExpertWeights), P,
                                ctypes.POINTER(RouteOut), P, ctypes.c_size_t, P]),
        "caee_moe_layer_noalloc": (st, [desc_p, P, P, P, P, P, ctypes.POINTER(ExpertWeights), P,
                                        ctypes.POINTER(RouteOut), P]),
        "caee_pack_matrix": (st, [ctypes.c_int32, P, P, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, P]),
        "caee_quantize_rows": (st, [ctypes.c_int32, P, ctypes.c_int64, ctypes.c_int64, P, P, P]),
        "caee_offload_create": (st, [desc_p, ctypes.POINTER(OffloadDesc), ctypes.POINTER(P)]),
        "caee_offload_destroy": (None, [P]),
        "caee_offload_layer": (st, [P, desc_p, P, P, P, P, ctypes.POINTER(RouteOut), P, ctypes.c_size_t, P, P]),
        "caee_offload_stats": (st, [P, ctypes.POINTER(OffloadStats)]),
        "caee_offload_residency": (st, [P, P]),
        "caee_offload_reset": (st, [P]),
        "caee_lru_step": (st, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, P, P, P, ctypes.c_int64, P, P, P, P]),
        "caee_status_str": (ctypes.c_char_p, [st]),
        "caee_last_error": (ctypes.c_char_p, []),
        "caee_abi_version": (ctypes.c_int, []),
        "caee_timing_enable": (st, [ctypes.c_int]),
        "caee_timing_reset": (st, []),
        "caee_timing_query": (st, [ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_int64)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


lib = _load()


def load_library(path: str) -> None:
    """Bind this module to another build of the library (e.g. one compiled
    with different kernel tuning knobs)."""
    global lib
    lib = _load(path)


EXPORTED = ("caee_workspace_size", "caee_route_prune", "caee_expert_ffn", "caee_moe_layer", "caee_moe_layer_noalloc",
            "caee_pack_matrix", "caee_quantize_rows", "caee_offload_create", "caee_offload_destroy",
            "caee_offload_layer", "caee_offload_stats", "caee_offload_residency", "caee_offload_reset",
            "caee_lru_step", "caee_status_str", "caee_last_error", "caee_abi_version",
            "caee_timing_enable", "caee_timing_reset", "caee_timing_query")


def _check(status: int):
    if status != CAEE_OK:
        raise CaeeError(status, lib.caee_last_error().decode())


def abi_version() -> int:
    return lib.caee_abi_version()


@dataclass
class Layer:
    """Descriptor fields of one MoE layer call (see caee_layer_desc_t)."""

    T: int
    d: int
    f: int
    E: int
    n_group: int
    topk_group: int
    k: int
    n_shared: int
    routed_scaling: float
    tau: float = 0.0
    n_bins: int = 1
    w_dtype: str = "bf16"
    x_dtype: str = "bf16"
    y_dtype: str = "bf16"
    importance: str = "max"     # "max" | "sum" | "cir" (caee_importance_t)
    refill: str = "score"       # "score" | "none" | "random" | "literal" (caee_refill_t)
    seed: int = 0               # random refill keys
    keep_top1: bool = False     # each token's top expert mandatory in every call (not the paper's step 1)

    def desc(self) -> LayerDesc:
        return LayerDesc(self.T, self.d, self.f, self.E, self.n_group, self.topk_group, self.k,
                         self.n_shared, self.routed_scaling, self.tau, self.n_bins,
                         IMPORTANCE_CODE[self.importance],
                         DTYPE_CODE[self.x_dtype], DTYPE_CODE[self.w_dtype], DTYPE_CODE[self.y_dtype],
                         REFILL_CODE[self.refill], self.seed & 0xFFFFFFFF, 1 if self.keep_top1 else 0)

    @classmethod
    def from_shape(cls, shape, **over) -> "Layer":
        kw = dict(T=shape.T, d=shape.d, f=shape.f, E=shape.E, n_group=shape.n_group,
                  topk_group=shape.topk_group, k=shape.k, n_shared=shape.n_shared,
                  routed_scaling=shape.routed_scaling, tau=shape.tau, n_bins=shape.n_bins,
                  w_dtype=shape.w_dtype, x_dtype=shape.x_dtype, y_dtype=shape.y_dtype)
        kw.update(over)
        return cls(**kw)


def workspace_size(layer: Layer) -> int:
    n = ctypes.c_size_t(0)
    d = layer.desc()
    _check(lib.caee_workspace_size(ctypes.byref(d), ctypes.byref(n)))
    return int(n.value)


def _ptr(t) -> Optional[int]:
    return None if t is None else int(t.data_ptr())


def _stream(*tensors) -> Optional[int]:
    import torch
    for t in tensors:
        if t is not None:
            return int(torch.cuda.current_stream(t.device).cuda_stream)
    return None


def _weights(w: dict) -> ExpertWeights:
    g = lambda n: _ptr(w.get(n))  # noqa: E731
    return ExpertWeights(g("w13"), g("w2"), g("w13_scale"), g("w2_scale"),
                         g("sh_w13"), g("sh_w2"), g("sh_w13_scale"), g("sh_w2_scale"),
                         int(w.get("layout", LAYOUT_ROWMAJOR)))


def pack_matrix(w_dtype: str, src, dst, rows: int, cols: int, count: int):
    """Repack `count` row-major [rows][cols] matrices into the tiled layout."""
    _check(lib.caee_pack_matrix(DTYPE_CODE[w_dtype], _ptr(src), _ptr(dst), rows, cols, count, _stream(src)))
    return dst


def quantize_rows(src, q, scale):
    """E4M3 codes and per-128-column fp32 scales of a bf16/fp32 [rows][cols] tensor."""
    import torch
    dt = {torch.bfloat16: CAEE_BF16, torch.float32: CAEE_F32}[src.dtype]
    _check(lib.caee_quantize_rows(dt, _ptr(src), src.shape[0], src.shape[1], _ptr(q), _ptr(scale), _stream(src)))
    return q, scale


def pack_weights(weights: dict, w_dtype: str) -> dict:
    """Tiled copy of a row-major expert weight dict (scales are shared)."""
    import torch
    out = {k: v for k, v in weights.items() if k.endswith("_scale")}
    for name in ("w13", "w2", "sh_w13", "sh_w2"):
        src = weights.get(name)
        if src is None:
            continue
        dst = torch.empty_like(src)
        if src.numel():
            pack_matrix(w_dtype, src, dst, src.shape[1], src.shape[2], src.shape[0])
        out[name] = dst
    out["layout"] = LAYOUT_TILED
    return out


def pin_host_weights(weights: dict) -> dict:
    """Page-locked host copies of the routed expert matrices (``w13``, ``w2``)
    of a device weight dict, in its layout: the host side of an offloaded
    layer.  Shared experts stay on the device."""
    import torch
    out = {"layout": int(weights.get("layout", LAYOUT_ROWMAJOR))}
    for name in ("w13", "w2"):
        src = weights[name]
        dst = torch.empty(src.shape, dtype=src.dtype, pin_memory=True)
        dst.copy_(src)
        out[name] = dst
    return out


def alloc_slots(layer: Layer, n_slots: int, device) -> tuple:
    """Device buffers for ``n_slots`` experts of ``layer`` (w13, w2)."""
    import torch
    dt = {"f32": torch.float32, "bf16": torch.bfloat16}[layer.w_dtype]
    return (torch.empty((n_slots, 2 * layer.f, layer.d), dtype=dt, device=device),
            torch.empty((n_slots, layer.d, layer.f), dtype=dt, device=device))


def _route_out(out: Optional[dict]) -> Optional[RouteOut]:
    if out is None:
        return None
    g = lambda n: _ptr(out.get(n))  # noqa: E731
    return RouteOut(g("topk_ids"), g("topk_w"), g("orig_ids"), g("masks"), g("stats"), g("bin_loads"))


def alloc_workspace(layer: Layer, device):
    import torch
    return torch.empty(max(workspace_size(layer), 256), dtype=torch.uint8, device=device)


def alloc_route_out(layer: Layer, device, full: bool = True) -> dict:
    """Device buffers for the routing results of ``layer``."""
    import torch
    T, k = layer.T, layer.k
    out = {"topk_ids": torch.empty((T, k), dtype=torch.int32, device=device),
           "topk_w": torch.empty((T, k), dtype=torch.float32, device=device)}
    if full:
        words = (layer.E + 31) // 32
        out["orig_ids"] = torch.empty((T, k), dtype=torch.int32, device=device)
        out["masks"] = torch.empty((4, words), dtype=torch.int32, device=device)
        out["stats"] = torch.empty(STATS, dtype=torch.int32, device=device)
        out["bin_loads"] = torch.empty((3, layer.n_bins), dtype=torch.float64, device=device)
    return out


def route_prune(layer: Layer, logits, bias, cost, bins, out: dict, ws) -> dict:
    d = layer.desc()
    ro = _route_out(out)
    _check(lib.caee_route_prune(ctypes.byref(d), _ptr(logits), _ptr(bias), _ptr(cost), _ptr(bins),
                                ctypes.byref(ro), _ptr(ws), ws.numel(), _stream(logits)))
    return out


def expert_ffn(layer: Layer, x, topk_ids, topk_w, weights: dict, y, ws):
    d = layer.desc()
    w = _weights(weights)
    _check(lib.caee_expert_ffn(ctypes.byref(d), _ptr(x), _ptr(topk_ids), _ptr(topk_w), ctypes.byref(w),
                               _ptr(y), _ptr(ws), ws.numel(), _stream(x)))
    return y


def moe_layer(layer: Layer, x, logits, bias, cost, bins, weights: dict, y, ws, out: Optional[dict] = None):
    d = layer.desc()
    w = _weights(weights)
    ro = _route_out(out)
    _check(lib.caee_moe_layer(ctypes.byref(d), _ptr(x), _ptr(logits), _ptr(bias), _ptr(cost), _ptr(bins),
                              ctypes.byref(w), _ptr(y), None if ro is None else ctypes.byref(ro),
                              _ptr(ws), ws.numel(), _stream(x)))
    return y


SCRATCH_BYTES = 48 << 20   # CAEE_SCRATCH_BYTES: the library's own scratch array per GPU


def moe_layer_noalloc(layer: Layer, x, logits, bias, cost, bins, weights: dict, y, out: Optional[dict] = None):
    """caee_moe_layer_noalloc: the whole layer in the library's scratch array
    (no workspace argument; allocates nothing)."""
    d = layer.desc()
    w = _weights(weights)
    ro = _route_out(out)
    _check(lib.caee_moe_layer_noalloc(ctypes.byref(d), _ptr(x), _ptr(logits), _ptr(bias), _ptr(cost), _ptr(bins),
                                      ctypes.byref(w), _ptr(y), None if ro is None else ctypes.byref(ro),
                                      _stream(x)))
    return y


def timing_enable(on: bool = True):
    _check(lib.caee_timing_enable(1 if on else 0))


def timing_reset():
    _check(lib.caee_timing_reset())


def timing_query(kind: str):
    ms = ctypes.c_double(0)
    n = ctypes.c_int64(0)
    _check(lib.caee_timing_query(KERNEL_KINDS[kind], ctypes.byref(ms), ctypes.byref(n)))
    return float(ms.value), int(n.value)


def lru_step(E: int, n_cache: int, n_stage: int, slot_of, slot_expert, slot_used, call: int, need):
    """One residency plan on host numpy arrays (caee_lru_step); the state
    arrays are updated in place.  Returns (fetch, fetch_slot, counts) with
    counts = (hits, misses, staged, evictions)."""
    import numpy as np
    for a, dt in ((slot_of, np.int32), (slot_expert, np.int32), (slot_used, np.int64)):
        if a.dtype != dt or not a.flags.c_contiguous:
            raise TypeError("state arrays must be contiguous int32/int32/int64")
    need = np.ascontiguousarray(need, dtype=np.uint8)
    fetch = np.zeros(E, np.int32)
    fetch_slot = np.zeros(E, np.int32)
    counts = np.zeros(4, np.int32)
    p = lambda a: a.ctypes.data_as(ctypes.c_void_p)  # noqa: E731
    _check(lib.caee_lru_step(E, n_cache, n_stage, p(slot_of), p(slot_expert), p(slot_used), call, p(need),
                             p(fetch), p(fetch_slot), p(counts)))
    n = int(counts[1])
    return fetch[:n].copy(), fetch_slot[:n].copy(), tuple(int(c) for c in counts)


class Offload:
    """Offload residency handle (caee_offload_t) of one layer.

    ``host_w13``/``host_w2``: per-expert page-locked host tensors (or one
    pinned tensor [E][...] each); ``slot_w13``/``slot_w2``: device tensors
    with ``n_cache + n_stage`` expert slots; ``sh_w13``/``sh_w2``: device
    shared-expert weights (or None).  Every tensor must stay alive while the
    handle is used; the handle keeps references to them."""

    def __init__(self, layer: Layer, host_w13, host_w2, slot_w13, slot_w2, sh_w13, sh_w2, n_cache: int,
                 n_stage: int, miss_cost: float, fetch_batch: int = 4, layout: int = LAYOUT_TILED):
        E = layer.E
        h13 = list(host_w13) if isinstance(host_w13, (list, tuple)) else [host_w13[e] for e in range(E)]
        h2 = list(host_w2) if isinstance(host_w2, (list, tuple)) else [host_w2[e] for e in range(E)]
        if len(h13) != E or len(h2) != E:
            raise ValueError("one host tensor per routed expert is needed")
        self._keep = (host_w13, host_w2, h13, h2, slot_w13, slot_w2, sh_w13, sh_w2)
        self._h13 = (ctypes.c_void_p * E)(*[int(t.data_ptr()) for t in h13])
        self._h2 = (ctypes.c_void_p * E)(*[int(t.data_ptr()) for t in h2])
        self.od = OffloadDesc(ctypes.cast(self._h13, ctypes.POINTER(ctypes.c_void_p)),
                              ctypes.cast(self._h2, ctypes.POINTER(ctypes.c_void_p)),
                              _ptr(slot_w13), _ptr(slot_w2), _ptr(sh_w13), _ptr(sh_w2),
                              int(layout), int(n_cache), int(n_stage), int(fetch_batch), float(miss_cost))
        self.layer = layer
        self.E = E
        d = layer.desc()
        h = ctypes.c_void_p(None)
        _check(lib.caee_offload_create(ctypes.byref(d), ctypes.byref(self.od), ctypes.byref(h)))
        self.handle = h

    def __call__(self, layer: Layer, x, logits, bias, y, ws, out: Optional[dict] = None, copy_stream=None):
        """One layer call.  ``copy_stream``: a torch stream for the host-to-device
        copies (default: a dedicated stream of the handle)."""
        import torch
        if copy_stream is None:
            if getattr(self, "_copy_stream", None) is None:
                self._copy_stream = torch.cuda.Stream(device=x.device)
            copy_stream = self._copy_stream
        d = layer.desc()
        ro = _route_out(out)
        _check(lib.caee_offload_layer(self.handle, ctypes.byref(d), _ptr(x), _ptr(logits), _ptr(bias), _ptr(y),
                                      None if ro is None else ctypes.byref(ro), _ptr(ws), ws.numel(), _stream(x),
                                      int(copy_stream.cuda_stream)))
        return y

    def stats(self) -> dict:
        st = OffloadStats()
        _check(lib.caee_offload_stats(self.handle, ctypes.byref(st)))
        return {n: int(getattr(st, n)) for n, _ in OffloadStats._fields_ if n != "reserved"}

    def residency(self):
        import numpy as np
        a = np.zeros(self.E, np.int32)
        _check(lib.caee_offload_residency(self.handle, a.ctypes.data_as(ctypes.c_void_p)))
        return a

    def reset(self):
        _check(lib.caee_offload_reset(self.handle))

    def close(self):
        if getattr(self, "handle", None) is not None and self.handle.value:
            lib.caee_offload_destroy(self.handle)
        self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
