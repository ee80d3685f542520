"""Python binding of the C ABI in include/spear.h (argument marshalling only).

Every step of the layer runs in libspear.so's HIP kernels; this module only
turns torch tensors into pointers, the problem description into the C
structs, and status codes into exceptions. If the library is not built it
raises at import time: there is no fallback.

Functions mirror the C entry points: dispatch_plan, w4_linear, w4ec_linear,
w4_dequant, plus allocate_workspace (the caller-owned scratch buffer).
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libspear.so")

F16, BF16 = 0, 1
GATE_ONE, GATE_SIGMOID_LINEAR, GATE_TANH_MLP = 0, 1, 2
PATH_AUTO, PATH_FUSED_GEMV, PATH_FUSED_MFMA, PATH_UNFUSED_CHAIN, PATH_UNFUSED_2K = 0, 1, 2, 3, 4
PATH_FUSED_LOCAL = 5
PATH_OVERLAP_2K = 6
PATH_NAMES = {PATH_AUTO: "auto", PATH_FUSED_GEMV: "fused_gemv", PATH_FUSED_MFMA: "fused_mfma",
              PATH_UNFUSED_CHAIN: "unfused_chain", PATH_UNFUSED_2K: "unfused_2k",
              PATH_FUSED_LOCAL: "fused_local", PATH_OVERLAP_2K: "overlap_2k"}

STATUS = {0: "SPEAR_OK", -1: "SPEAR_E_NULL", -2: "SPEAR_E_SHAPE", -3: "SPEAR_E_DTYPE",
          -4: "SPEAR_E_ALIGN", -5: "SPEAR_E_WORKSPACE", -6: "SPEAR_E_UNSUPPORTED",
          -7: "SPEAR_E_HIP", -8: "SPEAR_E_ALIAS"}

EXPORTED = ("spear_dispatch_plan", "spear_w4_linear", "spear_w4ec_linear", "spear_w4_dequant",
            "spear_w4ec_linear_tail", "spear_group_workspace", "spear_w4ec_linear_group",
            "spear_group_launches", "spear_set_wait_polls", "spear_set_gemv_shape",
            "spear_set_gemm_slices",
            "spear_set_gemm_tile", "spear_set_gemm_roles", "spear_workspace_regions",
            "spear_w4ec_linear_noalloc",
            "spear_set_gemv_stages",
            "spear_status_string", "spear_version", "spear_sched_latency", "spear_sched_chunk")


class Problem(ctypes.Structure):
    _fields_ = [("M", ctypes.c_int64), ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("group_size", ctypes.c_int32), ("act_dtype", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("gate_kind", ctypes.c_int32),
                ("gate_hidden", ctypes.c_int32), ("force_path", ctypes.c_int32),
                ("weight_bits", ctypes.c_int32)]


class W4(ctypes.Structure):
    _fields_ = [("qweight", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("zeros", ctypes.c_void_p)]


AB_ACT, AB_INT8 = 0, 1


class EC(ctypes.Structure):
    _fields_ = [("A", ctypes.c_void_p), ("B", ctypes.c_void_p), ("alpha", ctypes.c_float),
                ("w_g", ctypes.c_void_p), ("b_g", ctypes.c_float),
                ("W1", ctypes.c_void_p), ("b1", ctypes.c_void_p),
                ("W2", ctypes.c_void_p), ("b2", ctypes.c_void_p),
                ("ab_format", ctypes.c_int32), ("a_scale", ctypes.c_void_p),
                ("b_scale", ctypes.c_void_p)]


class Tail(ctypes.Structure):
    _fields_ = [("residual", ctypes.c_void_p), ("norm_w", ctypes.c_void_p),
                ("eps", ctypes.c_float), ("y_norm", ctypes.c_void_p)]


class LayerCall(ctypes.Structure):
    _fields_ = [("prob", ctypes.POINTER(Problem)), ("x", ctypes.c_void_p),
                ("w", ctypes.POINTER(W4)), ("ec", ctypes.POINTER(EC)), ("y", ctypes.c_void_p)]


GROUP_MAX = 4


class Plan(ctypes.Structure):
    _fields_ = [("path", ctypes.c_int32), ("split_k", ctypes.c_int32),
                ("ec_splits", ctypes.c_int32), ("tile_m", ctypes.c_int32),
                ("tile_n", ctypes.c_int32), ("num_launches", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("workspace_bytes", ctypes.c_size_t)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "reserved"}


class Lut(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("M", ctypes.POINTER(ctypes.c_int64)),
                ("lat_w4", ctypes.POINTER(ctypes.c_double)),
                ("lat_ec", ctypes.POINTER(ctypes.c_double))]


class ModelLat(ctypes.Structure):
    _fields_ = [("layers", ctypes.c_int32), ("modules", ctypes.c_int32),
                ("luts", ctypes.POINTER(Lut)), ("selection", ctypes.POINTER(ctypes.c_uint8)),
                ("extra", ctypes.POINTER(Lut))]


class SpearError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {STATUS.get(status, status)}")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2606_11244_amd.build.build()")
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    lib.spear_dispatch_plan.argtypes = [P(Problem), ctypes.c_int32, P(Plan)]
    lib.spear_w4_linear.argtypes = [P(Problem), ctypes.c_void_p, P(W4), ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.spear_w4ec_linear.argtypes = [P(Problem), ctypes.c_void_p, P(W4), P(EC), ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.spear_w4_dequant.argtypes = [P(Problem), P(W4), ctypes.c_void_p, ctypes.c_void_p]
    lib.spear_w4ec_linear_noalloc.argtypes = [P(Problem), ctypes.c_void_p, P(W4), P(EC),
                                              ctypes.c_void_p, ctypes.c_void_p]
    lib.spear_w4ec_linear_tail.argtypes = [P(Problem), ctypes.c_void_p, P(W4), P(EC), P(Tail),
                                           ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                           ctypes.c_void_p]
    lib.spear_group_workspace.argtypes = [ctypes.c_int32, P(LayerCall), P(ctypes.c_size_t)]
    lib.spear_group_launches.argtypes = [ctypes.c_int32, P(LayerCall), P(ctypes.c_int32)]
    lib.spear_w4ec_linear_group.argtypes = [ctypes.c_int32, P(LayerCall), ctypes.c_void_p,
                                            ctypes.c_size_t, ctypes.c_void_p]
    lib.spear_set_wait_polls.argtypes = [ctypes.c_int32]
    lib.spear_workspace_regions.argtypes = [P(Problem), ctypes.c_int32] + [P(ctypes.c_size_t)] * 4
    lib.spear_set_gemv_shape.argtypes = [ctypes.c_int32] * 3
    lib.spear_set_gemv_shape.restype = None
    lib.spear_set_gemm_slices.argtypes = [ctypes.c_int32]
    lib.spear_set_gemm_slices.restype = None
    lib.spear_set_gemm_tile.argtypes = [ctypes.c_int32]
    lib.spear_set_gemm_tile.restype = None
    lib.spear_set_gemm_roles.argtypes = [ctypes.c_int32]
    lib.spear_set_gemm_roles.restype = None
    lib.spear_set_gemv_stages.argtypes = [ctypes.c_int32]
    lib.spear_set_gemv_stages.restype = None
    lib.spear_sched_latency.argtypes = [P(ModelLat), ctypes.c_int64, P(ctypes.c_double)]
    lib.spear_sched_chunk.argtypes = [P(ModelLat), ctypes.c_int64, ctypes.c_double,
                                      ctypes.c_int64, ctypes.c_int64, P(ctypes.c_int64)]
    lib.spear_sched_latency.restype = ctypes.c_int32
    lib.spear_sched_chunk.restype = ctypes.c_int32
    lib.spear_status_string.argtypes = [ctypes.c_int32]
    lib.spear_status_string.restype = ctypes.c_char_p
    lib.spear_version.restype = ctypes.c_char_p
    for f in ("spear_dispatch_plan", "spear_w4_linear", "spear_w4ec_linear", "spear_w4_dequant",
              "spear_w4ec_linear_tail", "spear_group_workspace", "spear_w4ec_linear_group",
              "spear_group_launches", "spear_set_wait_polls", "spear_workspace_regions",
              "spear_w4ec_linear_noalloc"):
        getattr(lib, f).restype = ctypes.c_int32
    return lib


LIB = _load()


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float16:
        return F16
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported activation dtype {t.dtype}")


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def problem(M, N, K, group_size=0, act_dtype=F16, rank=0, gate_kind=GATE_SIGMOID_LINEAR,
            gate_hidden=0, force_path=PATH_AUTO, weight_bits=0) -> Problem:
    return Problem(int(M), int(N), int(K), int(group_size), int(act_dtype), int(rank),
                   int(gate_kind), int(gate_hidden), int(force_path), int(weight_bits))


def dispatch_plan(prob: Problem, with_ec: bool = True) -> Plan:
    out = Plan()
    st = LIB.spear_dispatch_plan(ctypes.byref(prob), 1 if with_ec else 0, ctypes.byref(out))
    if st != 0:
        raise SpearError(st, "spear_dispatch_plan")
    return out


def workspace_regions(prob: Problem, with_ec: bool = True):
    """((tag_begin, tag_end), (data_begin, data_end)) of a planned call's
    workspace (the fused path's tagged words; every other scratch region)."""
    v = [ctypes.c_size_t(0) for _ in range(4)]
    st = LIB.spear_workspace_regions(ctypes.byref(prob), 1 if with_ec else 0,
                                     *[ctypes.byref(a) for a in v])
    if st != 0:
        raise SpearError(st, "spear_workspace_regions")
    return (v[0].value, v[1].value), (v[2].value, v[3].value)


def allocate_workspace(prob: Problem, with_ec: bool = True, device="cuda") -> torch.Tensor:
    """Zero-filled workspace of the size the plan asks for (at least 256 B)."""
    nbytes = max(256, dispatch_plan(prob, with_ec).workspace_bytes)
    return torch.zeros(nbytes, dtype=torch.uint8, device=device)


def w4_linear(prob: Problem, x, qweight, scales, zeros, y, workspace=None, stream=None):
    w = W4(_ptr(qweight).value, _ptr(scales).value, _ptr(zeros).value)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = LIB.spear_w4_linear(ctypes.byref(prob), _ptr(x), ctypes.byref(w), _ptr(y),
                             _ptr(workspace), ws_bytes, _stream(stream))
    if st != 0:
        raise SpearError(st, "spear_w4_linear")
    return y


def w4ec_linear(prob: Problem, x, qweight, scales, zeros, A, B, y, *, alpha=1.0, w_g=None,
                b_g=0.0, W1=None, b1=None, W2=None, b2=None, a_scale=None, b_scale=None,
                ab_format=None, workspace=None, stream=None):
    """A and B in the activation dtype, or int8 codes with fp32 per-channel
    a_scale [r] and b_scale [N] (format SPEAR_AB_INT8, taken when the scales
    are given unless ab_format says otherwise)."""
    w = W4(_ptr(qweight).value, _ptr(scales).value, _ptr(zeros).value)

    def p(t):
        return None if t is None else t.data_ptr()

    fmt = (AB_INT8 if a_scale is not None else AB_ACT) if ab_format is None else int(ab_format)
    ec = EC(p(A), p(B), float(alpha), p(w_g), float(b_g), p(W1), p(b1), p(W2), p(b2),
            fmt, p(a_scale), p(b_scale))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = LIB.spear_w4ec_linear(ctypes.byref(prob), _ptr(x), ctypes.byref(w), ctypes.byref(ec),
                               _ptr(y), _ptr(workspace), ws_bytes, _stream(stream))
    if st != 0:
        raise SpearError(st, "spear_w4ec_linear")
    return y


SCRATCH_BYTES = 16 << 20  # SPEAR_SCRATCH_BYTES: the library's own scratch per GPU


def w4ec_linear_noalloc(prob: Problem, x, qweight, scales, zeros, A, B, y, *, alpha=1.0,
                        w_g=None, b_g=0.0, W1=None, b1=None, W2=None, b2=None, a_scale=None,
                        b_scale=None, ab_format=None, stream=None):
    """spear_w4ec_linear_noalloc: as w4ec_linear, with the library's own
    scratch instead of a workspace (nothing is allocated)."""
    w = W4(_ptr(qweight).value, _ptr(scales).value, _ptr(zeros).value)

    def p(t):
        return None if t is None else t.data_ptr()

    fmt = (AB_INT8 if a_scale is not None else AB_ACT) if ab_format is None else int(ab_format)
    ec = EC(p(A), p(B), float(alpha), p(w_g), float(b_g), p(W1), p(b1), p(W2), p(b2),
            fmt, p(a_scale), p(b_scale))
    st = LIB.spear_w4ec_linear_noalloc(ctypes.byref(prob), _ptr(x), ctypes.byref(w),
                                       ctypes.byref(ec), _ptr(y), _stream(stream))
    if st != 0:
        raise SpearError(st, "spear_w4ec_linear_noalloc")
    return y


def w4ec_linear_tail(prob: Problem, x, qweight, scales, zeros, y, *, ec_args=None, residual=None,
                     norm_w=None, eps=1e-5, y_norm=None, workspace=None, stream=None):
    """The layer plus the post-EC tail (include/spear.h): y gets the residual
    added before its rounding, y_norm = RMSNorm(y) * norm_w. ec_args: the
    keyword arguments of w4ec_linear for A, B and the gate (with "A" and
    "B"), or None for the 4-bit layer alone."""
    w = W4(_ptr(qweight).value, _ptr(scales).value, _ptr(zeros).value)

    def p(t):
        return None if t is None else t.data_ptr()

    ec = None
    if ec_args is not None:
        a = dict(ec_args)
        fmt = AB_INT8 if a.get("a_scale") is not None else AB_ACT
        ec = EC(p(a["A"]), p(a["B"]), float(a.get("alpha", 1.0)), p(a.get("w_g")),
                float(a.get("b_g", 0.0)), p(a.get("W1")), p(a.get("b1")), p(a.get("W2")),
                p(a.get("b2")), fmt, p(a.get("a_scale")), p(a.get("b_scale")))
    tail = Tail(p(residual), p(norm_w), float(eps), p(y_norm))
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = LIB.spear_w4ec_linear_tail(ctypes.byref(prob), _ptr(x), ctypes.byref(w),
                                    ctypes.byref(ec) if ec is not None else None,
                                    ctypes.byref(tail), _ptr(y), _ptr(workspace), ws_bytes,
                                    _stream(stream))
    if st != 0:
        raise SpearError(st, "spear_w4ec_linear_tail")
    return y


def _ec_from_args(a):
    def p(t):
        return None if t is None else t.data_ptr()
    fmt = AB_INT8 if a.get("a_scale") is not None else AB_ACT
    return EC(p(a["A"]), p(a["B"]), float(a.get("alpha", 1.0)), p(a.get("w_g")),
              float(a.get("b_g", 0.0)), p(a.get("W1")), p(a.get("b1")), p(a.get("W2")),
              p(a.get("b2")), fmt, p(a.get("a_scale")), p(a.get("b_scale")))


def _group_array(members):
    """ctypes array of spear_layer_call_t for members = [dict(prob, x,
    qweight, scales, zeros, y, ec_args or None)], plus the structs it points
    to (kept alive by the caller)."""
    n = len(members)
    arr = (LayerCall * max(n, 1))()
    keep = []
    for i, m in enumerate(members):
        w = W4(_ptr(m["qweight"]).value, _ptr(m["scales"]).value, _ptr(m["zeros"]).value)
        ec = _ec_from_args(m["ec_args"]) if m.get("ec_args") is not None else None
        keep += [m["prob"], w, ec]
        arr[i].prob = ctypes.pointer(m["prob"])
        arr[i].x = m["x"].data_ptr()
        arr[i].w = ctypes.pointer(w)
        arr[i].ec = ctypes.pointer(ec) if ec is not None else None
        arr[i].y = m["y"].data_ptr()
    return arr, keep


def group_workspace(members) -> int:
    """Workspace bytes of a grouped call (include/spear.h)."""
    arr, keep = _group_array(members)
    out = ctypes.c_size_t(0)
    st = LIB.spear_group_workspace(len(members), arr, ctypes.byref(out))
    if st != 0:
        raise SpearError(st, "spear_group_workspace")
    return out.value


def group_launches(members) -> int:
    """Kernel launches a grouped call with these members makes (include/spear.h)."""
    arr, keep = _group_array(members)
    out = ctypes.c_int32(0)
    st = LIB.spear_group_launches(len(members), arr, ctypes.byref(out))
    if st != 0:
        raise SpearError(st, "spear_group_launches")
    return out.value


def w4ec_linear_group(members, workspace=None, stream=None):
    """Up to GROUP_MAX independent layer calls; those of one kernel variant
    share one launch (include/spear.h); members as in group_workspace."""
    arr, keep = _group_array(members)
    ws_bytes = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = LIB.spear_w4ec_linear_group(len(members), arr, _ptr(workspace), ws_bytes,
                                     _stream(stream))
    if st != 0:
        raise SpearError(st, "spear_w4ec_linear_group")


def w4_dequant(prob: Problem, qweight, scales, zeros, w_out, stream=None):
    w = W4(_ptr(qweight).value, _ptr(scales).value, _ptr(zeros).value)
    st = LIB.spear_w4_dequant(ctypes.byref(prob), ctypes.byref(w), _ptr(w_out), _stream(stream))
    if st != 0:
        raise SpearError(st, "spear_w4_dequant")
    return w_out


def set_wait_polls(polls: int) -> int:
    return int(LIB.spear_set_wait_polls(int(polls)))


def set_gemv_shape(row_tiles=0, k_slices=0, waves=0) -> None:
    """Tuning override of the decode GEMV launch shape (0 = automatic)."""
    LIB.spear_set_gemv_shape(int(row_tiles), int(k_slices), int(waves))


def set_gemm_slices(k_slices=0) -> None:
    """Tuning override of the prefill GEMM's K-slices (0 = automatic)."""
    LIB.spear_set_gemm_slices(int(k_slices))


def set_gemv_stages(stages=0) -> None:
    """Decode GEMV pipeline depth (2, 4, 8; 0 = the planner's choice)."""
    LIB.spear_set_gemv_stages(int(stages))


def set_gemm_tile(tokens=0) -> None:
    """Tuning override of the prefill GEMM's token tile (128, 256; 0 = automatic)."""
    LIB.spear_set_gemm_tile(int(tokens))


def set_gemm_roles(roles=0) -> None:
    """Tuning override of the prefill GEMM's wave roles (1 = every wave both,
    2 = loading and multiplying waves; 0 = automatic)."""
    LIB.spear_set_gemm_roles(int(roles))


class LatencyModel:
    """Latency tables and an EC selection for the scheduler of
    include/spear_sched.h. `luts` is a list (one per module type) of
    (M list, 4-bit latency list, W4+EC latency list) in microseconds;
    `selection` a layers x modules list of 0/1; `extra` an optional
    (M list, latency list) of the other per-layer work."""

    def __init__(self, luts, selection, extra=None):
        self._keep = []
        arr = (Lut * len(luts))()
        for j, (M, lw, le) in enumerate(luts):
            arr[j] = self._lut(M, lw, le)
        layers, modules = len(selection), len(luts)
        flat = (ctypes.c_uint8 * (layers * modules))(*[int(bool(v)) for row in selection for v in row])
        self._keep += [arr, flat]
        ex = None
        if extra is not None:
            ex = ctypes.pointer(self._lut(extra[0], extra[1], extra[1]))
            self._keep.append(ex)
        self.c = ModelLat(layers, modules, arr, flat, ex)

    def _lut(self, M, lw, le):
        n = len(M)
        a = (ctypes.c_int64 * n)(*[int(v) for v in M])
        b = (ctypes.c_double * n)(*[float(v) for v in lw])
        c = (ctypes.c_double * n)(*[float(v) for v in le])
        self._keep += [a, b, c]
        return Lut(n, a, b, c)


def sched_latency(model: LatencyModel, m: int) -> float:
    """Estimated iteration latency (us) at m tokens (SPEAR section 4.3)."""
    out = ctypes.c_double()
    st = LIB.spear_sched_latency(ctypes.byref(model.c), int(m), ctypes.byref(out))
    if st != 0:
        raise SpearError(st, "spear_sched_latency")
    return out.value


def sched_chunk(model: LatencyModel, d: int, t_slo_us: float, c_min: int, c_max: int) -> int:
    """Largest prefill chunk c in [c_min, c_max] with T(d) + T(c) <= t_slo_us (0: none)."""
    out = ctypes.c_int64()
    st = LIB.spear_sched_chunk(ctypes.byref(model.c), int(d), float(t_slo_us), int(c_min),
                               int(c_max), ctypes.byref(out))
    if st != 0:
        raise SpearError(st, "spear_sched_chunk")
    return out.value


def version() -> str:
    return LIB.spear_version().decode()


# ---------------------------------------------------------------------------
# device tensors of a generated layer (synth.Layer) and one call on them
# ---------------------------------------------------------------------------

_TORCH_DT = {F16: torch.float16, BF16: torch.bfloat16}


class DeviceLayer:
    """The stored tensors of one layer, resident on the GPU."""

    def __init__(self, layer, device="cuda"):
        import numpy as np
        dt = _TORCH_DT[layer.act_dtype]

        def act(a, shape=None):
            t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(dt)
            return t.reshape(shape).to(device) if shape else t.to(device)

        self.layer = layer
        self.M, self.N, self.K = layer.M, layer.N, layer.K
        self.dtype = dt
        self.qweight = torch.from_numpy(layer.qweight.view(np.int32)).to(device)
        self.scales = torch.from_numpy(layer.scales.view(np.int16)).to(device)
        self.zeros = torch.from_numpy(layer.zeros).to(device)
        self.x = act(layer.x)
        self.ab_int8 = bool(getattr(layer, "ab_int8", False)) and layer.rank > 0
        if self.ab_int8:
            self.A = torch.from_numpy(np.ascontiguousarray(layer.A_q)).to(device)
            self.B = torch.from_numpy(np.ascontiguousarray(layer.B_q)).to(device)
            self.a_scale = torch.from_numpy(np.ascontiguousarray(layer.a_scale)).to(device)
            self.b_scale = torch.from_numpy(np.ascontiguousarray(layer.b_scale)).to(device)
        else:
            self.A = act(layer.A) if layer.rank > 0 else None
            self.B = act(layer.B) if layer.rank > 0 else None
            self.a_scale = self.b_scale = None
        self.w_g = act(layer.w_g)
        self.W1, self.b1 = act(layer.W1), act(layer.b1)
        self.W2, self.b2 = act(layer.W2), act(layer.b2)
        self.y = torch.empty((layer.M, layer.N), dtype=dt, device=device)

    def problem(self, force_path=PATH_AUTO, rank=None, gate_kind=None):
        L = self.layer
        return problem(L.M, L.N, L.K, L.group_size, L.act_dtype,
                       L.rank if rank is None else rank,
                       L.gate_kind if gate_kind is None else gate_kind,
                       L.gate_hidden if L.rank > 0 else 0, force_path,
                       getattr(L, "weight_bits", 4))

    def run_ec(self, prob, workspace, stream=None, y=None):
        L = self.layer
        y = self.y if y is None else y
        return w4ec_linear(prob, self.x, self.qweight, self.scales, self.zeros, self.A, self.B, y,
                           alpha=L.alpha, w_g=self.w_g, b_g=L.b_g, W1=self.W1, b1=self.b1,
                           W2=self.W2, b2=self.b2, a_scale=self.a_scale, b_scale=self.b_scale,
                           workspace=workspace, stream=stream)

    def run_noalloc(self, prob, stream=None, y=None):
        L = self.layer
        y = self.y if y is None else y
        return w4ec_linear_noalloc(prob, self.x, self.qweight, self.scales, self.zeros, self.A,
                                   self.B, y, alpha=L.alpha, w_g=self.w_g, b_g=L.b_g, W1=self.W1,
                                   b1=self.b1, W2=self.W2, b2=self.b2, a_scale=self.a_scale,
                                   b_scale=self.b_scale, stream=stream)

    def run_tail(self, prob, workspace, residual=None, norm_w=None, eps=1e-5, y_norm=None,
                 with_ec=True, stream=None, y=None):
        L = self.layer
        y = self.y if y is None else y
        ec_args = None
        if with_ec:
            ec_args = dict(A=self.A, B=self.B, alpha=L.alpha, w_g=self.w_g, b_g=L.b_g,
                           W1=self.W1, b1=self.b1, W2=self.W2, b2=self.b2,
                           a_scale=self.a_scale, b_scale=self.b_scale)
        return w4ec_linear_tail(prob, self.x, self.qweight, self.scales, self.zeros, y,
                                ec_args=ec_args, residual=residual, norm_w=norm_w, eps=eps,
                                y_norm=y_norm, workspace=workspace, stream=stream)

    def member(self, prob, with_ec=True, y=None):
        """This layer as a member of a grouped call."""
        L = self.layer
        ec_args = None
        if with_ec and prob.rank > 0:
            ec_args = dict(A=self.A, B=self.B, alpha=L.alpha, w_g=self.w_g, b_g=L.b_g,
                           W1=self.W1, b1=self.b1, W2=self.W2, b2=self.b2,
                           a_scale=self.a_scale, b_scale=self.b_scale)
        return dict(prob=prob, x=self.x, qweight=self.qweight, scales=self.scales,
                    zeros=self.zeros, y=self.y if y is None else y, ec_args=ec_args)

    def run_w4(self, prob, workspace, stream=None, y=None):
        y = self.y if y is None else y
        return w4_linear(prob, self.x, self.qweight, self.scales, self.zeros, y,
                         workspace=workspace, stream=stream)
