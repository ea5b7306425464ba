"""Python binding of libcardan.so (argument marshalling only).

Every function here checks dtypes, shapes, devices and contiguity of torch
tensors, turns them into raw device pointers and calls the C ABI declared in
``include/cardan.h``; all arithmetic runs in the library's HIP kernels.
Importing this module loads the library and raises ``ImportError`` when it is
missing: there is no fallback path.

bf16 arrays are passed as ``torch.bfloat16`` tensors (their storage is the
raw bf16 bit pattern the ABI expects).
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# CARDAN_LIB names another build of the library (the tests' sanitizer build)
LIB_PATH = os.environ.get("CARDAN_LIB") or os.path.join(HERE, "libcardan.so")

LAYER_FIELDS = (
    "router_w", "router_bias", "cb_gate", "cb_up", "cb_down",
    "codes_gate", "codes_up", "codes_down", "U_gate", "U_up",
    "V_gate", "V_up", "A_down", "B_down",
)

DENSE_LAYER_FIELDS = ("router_w", "router_bias", "W_gate", "W_up", "W_down")

KERNEL_KINDS = ("route", "expert", "rmsnorm")

ERRORS = {-1: "NULL_PTR", -2: "BAD_SHAPE", -3: "UNSUPPORTED", -4: "WORKSPACE", -5: "HIP",
          -6: "ALIGN"}


class CardanError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"cardan error {code} ({ERRORS.get(code, '?')}): {msg}")
        self.code = code


class Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("H", "I", "E", "top_k", "d", "K", "r")]


class LayerStruct(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in LAYER_FIELDS]


class DenseLayerStruct(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in DENSE_LAYER_FIELDS]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing; build it with `python -m paper_2609_21137_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
    sp = ctypes.POINTER(Shape)
    lp = ctypes.POINTER(LayerStruct)
    dp = ctypes.POINTER(DenseLayerStruct)
    sig = {
        "cardan_abi_version": ([], ctypes.c_int),
        "cardan_last_error": ([], ctypes.c_char_p),
        "cardan_workspace_bytes": ([sp, i32, ctypes.POINTER(sz)], ctypes.c_int),
        "cardan_route_topk": ([sp, i32, vp, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_shared_proj": ([sp, i32, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_vq_lr_expert_ffn": ([sp, i32, vp, vp, vp, vp, lp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_moe_layer": ([sp, i32, vp, lp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_moe_layer_noalloc": ([sp, i32, vp, lp, vp, vp, vp, vp], ctypes.c_int),
        "cardan_moe_layer_relu2": ([sp, i32, vp, lp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_moe_decode_step": ([sp, i32, i32, vp, lp, ctypes.c_float, vp, vp, vp, vp, vp, sz, vp],
                                   ctypes.c_int),
        "cardan_moe_layer_dense_down": ([sp, i32, vp, lp, vp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_dense_moe_layer": ([sp, i32, vp, dp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_dense_moe_layer_relu2": ([sp, i32, vp, dp, vp, vp, vp, vp, sz, vp], ctypes.c_int),
        "cardan_rmsnorm_bf16": ([i32, i32, vp, ctypes.c_float, vp, vp], ctypes.c_int),
        "cardan_profile_begin": ([i32], ctypes.c_int),
        "cardan_profile_end": ([ctypes.POINTER(ctypes.c_float), ctypes.POINTER(i32)], ctypes.c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _load()

EXPORTED = (
    "cardan_abi_version", "cardan_last_error", "cardan_workspace_bytes", "cardan_route_topk",
    "cardan_shared_proj", "cardan_vq_lr_expert_ffn", "cardan_moe_layer", "cardan_moe_layer_noalloc",
    "cardan_moe_decode_step", "cardan_moe_layer_relu2",
    "cardan_moe_layer_dense_down", "cardan_dense_moe_layer", "cardan_dense_moe_layer_relu2",
    "cardan_rmsnorm_bf16",
    "cardan_profile_begin", "cardan_profile_end",
)


def lib():
    return _lib


def _check(rc: int):
    if rc != 0:
        raise CardanError(rc, _lib.cardan_last_error().decode())


def abi_version() -> int:
    return _lib.cardan_abi_version()


def make_shape(H, I, E, top_k, d, K, r) -> Shape:
    return Shape(H, I, E, top_k, d, K, r)


def shape_of(w) -> Shape:
    """Shape struct of a workload from ``configs``."""
    return Shape(w.H, w.I, w.E, w.top_k, w.d, w.K, w.r)


def workspace_bytes(shape: Shape, B: int) -> int:
    out = ctypes.c_size_t(0)
    _check(_lib.cardan_workspace_bytes(ctypes.byref(shape), B, ctypes.byref(out)))
    return out.value


def workspace_status(ws: torch.Tensor) -> int:
    """Number of in-kernel waits that gave up (0 unless an invariant broke)."""
    return int(ws[:4].view(torch.int32).item())


def new_workspace(shape: Shape, B: int, device="cuda") -> torch.Tensor:
    """Zero-filled workspace (the library needs zeros before the first use)."""
    return torch.zeros(workspace_bytes(shape, B), dtype=torch.uint8, device=device)


def _ptr(t, dtype, name, shape=None, optional=False):
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must live on a GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    return ctypes.c_void_p(t.data_ptr())


def _stream(dev) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)


def bf16_tensor(bits: np.ndarray, device="cuda") -> torch.Tensor:
    """Raw bf16 bit patterns (uint16) to a bfloat16 tensor on ``device``."""
    arr = np.ascontiguousarray(bits, dtype=np.uint16).view(np.int16)
    return torch.from_numpy(arr).view(torch.bfloat16).to(device)


def bf16_bits(t: torch.Tensor) -> np.ndarray:
    """bfloat16 tensor back to raw uint16 bit patterns on the host."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


@dataclass
class DeviceLayer:
    """One layer's weights as device tensors (field names of ``cardan_layer``)."""
    tensors: dict

    @classmethod
    def from_numpy(cls, L: dict, device="cuda") -> "DeviceLayer":
        T = {}
        for key in LAYER_FIELDS:
            v = L.get(key)
            if v is None:
                T[key] = None
            elif key == "U_up" and L.get("U_up") is L.get("U_gate"):
                T[key] = T["U_gate"]
            elif v.dtype == np.uint16:
                T[key] = bf16_tensor(v, device)
            elif v.dtype == np.uint8:
                T[key] = torch.from_numpy(np.ascontiguousarray(v)).to(device)
            else:
                T[key] = torch.from_numpy(np.ascontiguousarray(v, dtype=np.float32)).to(device)
        return cls(T)

    def struct(self) -> LayerStruct:
        vals = []
        for key in LAYER_FIELDS:
            t = self.tensors.get(key)
            if t is None:
                vals.append(None)
            else:
                if not t.is_contiguous() or t.device.type != "cuda":
                    raise ValueError(f"{key} must be a contiguous GPU tensor")
                vals.append(t.data_ptr())
        return LayerStruct(*vals)

    def nbytes(self) -> int:
        seen, tot = set(), 0
        for t in self.tensors.values():
            if t is not None and t.data_ptr() not in seen:
                seen.add(t.data_ptr())
                tot += t.numel() * t.element_size()
        return tot


def route_topk(shape: Shape, x, router_w, router_bias=None, ws=None):
    """Router logits, top-k (descending, ties to the lower index) and softmax
    gating. Returns ``(topk_idx int32 [B, k], topk_w float32 [B, k])``."""
    B = x.shape[0]
    dev = x.device
    idx = torch.empty((B, shape.top_k), dtype=torch.int32, device=dev)
    w = torch.empty((B, shape.top_k), dtype=torch.float32, device=dev)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    _check(_lib.cardan_route_topk(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)),
        _ptr(router_w, torch.bfloat16, "router_w", (shape.H, shape.E)),
        _ptr(router_bias, torch.float32, "router_bias", (shape.E,), optional=True),
        _ptr(idx, torch.int32, "topk_idx"), _ptr(w, torch.float32, "topk_w"),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return idx, w


def shared_proj(shape: Shape, x, U_gate, U_up=None, ws=None):
    """Shared projections ``z[2, B, r]`` (gate, up) of every token."""
    B = x.shape[0]
    dev = x.device
    U_up = U_gate if U_up is None else U_up
    z = torch.empty((2, B, shape.r), dtype=torch.float32, device=dev)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    _check(_lib.cardan_shared_proj(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)),
        _ptr(U_gate, torch.bfloat16, "U_gate", (shape.H, shape.r)),
        _ptr(U_up, torch.bfloat16, "U_up", (shape.H, shape.r)),
        _ptr(z, torch.float32, "z"), _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return z


def vq_lr_expert_ffn(shape: Shape, x, topk_idx, topk_w, z, layer: DeviceLayer, ws=None, out=None):
    """Grouped expert computation and weighted combine for a given routing."""
    B = x.shape[0]
    dev = x.device
    y = out if out is not None else torch.empty((B, shape.H), dtype=torch.float32, device=dev)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    st = layer.struct()
    _check(_lib.cardan_vq_lr_expert_ffn(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)),
        _ptr(topk_idx, torch.int32, "topk_idx", (B, shape.top_k)),
        _ptr(topk_w, torch.float32, "topk_w", (B, shape.top_k)),
        _ptr(z, torch.float32, "z", (2, B, shape.r), optional=shape.r == 0),
        ctypes.byref(st), _ptr(y, torch.float32, "y", (B, shape.H)),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return y


def moe_layer(shape: Shape, x, layer: DeviceLayer, ws=None, out=None, idx=None, w=None):
    """The whole layer. Returns ``(y float32 [B, H], topk_idx, topk_w)``."""
    B = x.shape[0]
    dev = x.device
    y = out if out is not None else torch.empty((B, shape.H), dtype=torch.float32, device=dev)
    idx = idx if idx is not None else torch.empty((B, shape.top_k), dtype=torch.int32, device=dev)
    w = w if w is not None else torch.empty((B, shape.top_k), dtype=torch.float32, device=dev)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    st = layer.struct()
    _check(_lib.cardan_moe_layer(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)), ctypes.byref(st),
        _ptr(y, torch.float32, "y", (B, shape.H)),
        _ptr(idx, torch.int32, "topk_idx", (B, shape.top_k)),
        _ptr(w, torch.float32, "topk_w", (B, shape.top_k)),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return y, idx, w


def moe_layer_relu2(shape: Shape, x, layer: DeviceLayer, ws=None, out=None, idx=None, w=None):
    """The whole layer with up-only squared-ReLU experts (the layer's gate
    fields are not read). Returns ``(y float32 [B, H], topk_idx, topk_w)``."""
    B = x.shape[0]
    dev = x.device
    y, idx, w = _outputs(shape, x, out, idx, w)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    st = layer.struct()
    _check(_lib.cardan_moe_layer_relu2(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)), ctypes.byref(st),
        _ptr(y, torch.float32, "y", (B, shape.H)),
        _ptr(idx, torch.int32, "topk_idx", (B, shape.top_k)),
        _ptr(w, torch.float32, "topk_w", (B, shape.top_k)),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return y, idx, w


def moe_decode_step(shape: Shape, x0, layers, eps: float = 1e-6, ws=None, out=None, x_norm=None,
                    idx=None, w=None):
    """``len(layers)`` stacked layers, each output RMS-normalised (bf16) into
    the next layer's input. Returns ``(y [B, H] of the last layer,
    topk_idx [L, B, k], topk_w [L, B, k])``; ``x_norm`` (optional,
    ``[L - 1, B, H]`` bf16) receives the normalised inputs of layers 1..L-1."""
    B = x0.shape[0]
    L = len(layers)
    dev = x0.device
    y = out if out is not None else torch.empty((B, shape.H), dtype=torch.float32, device=dev)
    idx = idx if idx is not None else torch.empty((L, B, shape.top_k), dtype=torch.int32, device=dev)
    w = w if w is not None else torch.empty((L, B, shape.top_k), dtype=torch.float32, device=dev)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    structs = (LayerStruct * L)(*[dl.struct() for dl in layers])
    xn = (_ptr(x_norm, torch.bfloat16, "x_norm", (L - 1, B, shape.H)) if x_norm is not None and L > 1
          else None)
    _check(_lib.cardan_moe_decode_step(
        ctypes.byref(shape), B, L, _ptr(x0, torch.bfloat16, "x0", (B, shape.H)), structs,
        ctypes.c_float(eps), _ptr(y, torch.float32, "y", (B, shape.H)), xn,
        _ptr(idx, torch.int32, "topk_idx", (L, B, shape.top_k)),
        _ptr(w, torch.float32, "topk_w", (L, B, shape.top_k)),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return y, idx, w


def moe_layer_noalloc(shape: Shape, x, layer: DeviceLayer, out=None, idx=None, w=None):
    """The whole layer on the library's own scratch array (no workspace, no
    device allocation inside the call). Returns ``(y, topk_idx, topk_w)``."""
    B = x.shape[0]
    dev = x.device
    y, idx, w = _outputs(shape, x, out, idx, w)
    st = layer.struct()
    _check(_lib.cardan_moe_layer_noalloc(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)), ctypes.byref(st),
        _ptr(y, torch.float32, "y", (B, shape.H)),
        _ptr(idx, torch.int32, "topk_idx", (B, shape.top_k)),
        _ptr(w, torch.float32, "topk_w", (B, shape.top_k)), _stream(dev)))
    return y, idx, w


def _outputs(shape: Shape, x, out, idx, w):
    B = x.shape[0]
    dev = x.device
    y = out if out is not None else torch.empty((B, shape.H), dtype=torch.float32, device=dev)
    idx = idx if idx is not None else torch.empty((B, shape.top_k), dtype=torch.int32, device=dev)
    w = w if w is not None else torch.empty((B, shape.top_k), dtype=torch.float32, device=dev)
    return y, idx, w


def moe_layer_dense_down(shape: Shape, x, layer: DeviceLayer, W_down, ws=None, out=None, idx=None,
                         w=None):
    """The layer with compressed gate/up and a dense bf16 ``W_down [E, I, H]``
    (the layer's compressed down fields are not read). Returns
    ``(y float32 [B, H], topk_idx, topk_w)``."""
    B = x.shape[0]
    dev = x.device
    y, idx, w = _outputs(shape, x, out, idx, w)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    st = layer.struct()
    _check(_lib.cardan_moe_layer_dense_down(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)), ctypes.byref(st),
        _ptr(W_down, torch.bfloat16, "W_down", (shape.E, shape.I, shape.H)),
        _ptr(y, torch.float32, "y", (B, shape.H)),
        _ptr(idx, torch.int32, "topk_idx", (B, shape.top_k)),
        _ptr(w, torch.float32, "topk_w", (B, shape.top_k)),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return y, idx, w


@dataclass
class DenseLayer:
    """An uncompressed layer's device tensors (fields of ``cardan_dense_layer``):
    router_w [H, E] bf16, router_bias [E] f32 or None, W_gate / W_up [E, H, I]
    and W_down [E, I, H] bf16."""
    tensors: dict

    def struct(self, shape: Shape, up_only: bool = False) -> DenseLayerStruct:
        H, I, E = shape.H, shape.I, shape.E
        want = {"router_w": (torch.bfloat16, (H, E)), "router_bias": (torch.float32, (E,)),
                "W_gate": (torch.bfloat16, (E, H, I)), "W_up": (torch.bfloat16, (E, H, I)),
                "W_down": (torch.bfloat16, (E, I, H))}
        vals = []
        for key in DENSE_LAYER_FIELDS:
            dt, shp = want[key]
            optional = key == "router_bias" or (up_only and key == "W_gate")
            p = _ptr(self.tensors.get(key), dt, key, shp, optional=optional)
            vals.append(None if p is None else p.value)
        return DenseLayerStruct(*vals)


def dense_moe_layer(shape: Shape, x, layer: DenseLayer, ws=None, out=None, idx=None, w=None,
                    relu2: bool = False):
    """The uncompressed MoE layer (only H, I, E, top_k of ``shape`` are read);
    ``relu2``: up-only squared-ReLU experts (``W_gate`` not read).
    Returns ``(y float32 [B, H], topk_idx, topk_w)``."""
    B = x.shape[0]
    dev = x.device
    y, idx, w = _outputs(shape, x, out, idx, w)
    if ws is None:
        ws = new_workspace(shape, B, dev)
    st = layer.struct(shape, up_only=relu2)
    fn = _lib.cardan_dense_moe_layer_relu2 if relu2 else _lib.cardan_dense_moe_layer
    _check(fn(
        ctypes.byref(shape), B, _ptr(x, torch.bfloat16, "x", (B, shape.H)), ctypes.byref(st),
        _ptr(y, torch.float32, "y", (B, shape.H)),
        _ptr(idx, torch.int32, "topk_idx", (B, shape.top_k)),
        _ptr(w, torch.float32, "topk_w", (B, shape.top_k)),
        _ptr(ws, torch.uint8, "ws"), ws.numel(), _stream(dev)))
    return y, idx, w


def rmsnorm_bf16(y, eps: float = 1e-6, out=None):
    """``bf16_rne(y / sqrt(mean(y^2) + eps))`` per row, as a bfloat16 tensor."""
    B, H = y.shape
    xn = out if out is not None else torch.empty((B, H), dtype=torch.bfloat16, device=y.device)
    _check(_lib.cardan_rmsnorm_bf16(B, H, _ptr(y, torch.float32, "y", (B, H)), eps,
                                    _ptr(xn, torch.bfloat16, "x_next", (B, H)), _stream(y.device)))
    return xn


def profile_begin(max_calls: int):
    _check(_lib.cardan_profile_begin(max_calls))


def profile_end() -> dict:
    """``{kind: (total_ms, launches)}`` for the calls since ``profile_begin``."""
    n = len(KERNEL_KINDS)
    ms = (ctypes.c_float * n)()
    cnt = (ctypes.c_int32 * n)()
    _check(_lib.cardan_profile_end(ms, cnt))
    return {k: (ms[i], cnt[i]) for i, k in enumerate(KERNEL_KINDS)}
