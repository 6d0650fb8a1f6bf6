"""Python binding of libd2moe (ctypes).  Argument marshalling only: every step
of the MoE layer runs in the HIP library; torch provides device memory and the
current stream.  The names mirror the C ABI in include/d2moe.h.

The library is loaded from this package directory (or from the path in the
D2MOE_LIB environment variable); if it is missing the call fails loudly (run
``paper_2504_15299_amd.build.build()`` first).
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("D2MOE_LIB") or os.path.join(_HERE, "libd2moe.so")

D2MOE_F32, D2MOE_BF16 = 0, 1
OK, EINVAL, EUNSUPPORTED, EHIP, EWORKSPACE, ESCRATCH = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 32 << 20   # D2MOE_NOALLOC_SCRATCH_BYTES

_P = ctypes.c_void_p
_I = ctypes.c_int32


class _Mwq(ctypes.Structure):
    _fields_ = [("n_experts", _I), ("rows", _I), ("cols", _I), ("group", _I), ("b_min", _I),
                ("b_max", _I), ("planes", _P), ("scales", _P), ("zeros", _P)]


class _Unit(ctypes.Structure):
    _fields_ = [("expert", _I), ("bits", _I), ("load_from", _I), ("load_to", _I), ("count", _I)]


class _BudgetAction(ctypes.Structure):
    _fields_ = [("action", _I), ("layer", _I), ("expert", _I), ("level", _I)]


class _Routing(ctypes.Structure):
    _fields_ = [("logits", _P), ("topk_idx", _P), ("topk_w", _P), ("topk_bits", _P),
                ("hist", _P), ("offsets", _P), ("perm", _P), ("slot_of", _P),
                ("expert_maxbit", _P), ("flags", _P)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing "
                               "(call paper_2504_15299_amd.build.build())")
        L = ctypes.CDLL(LIB_PATH)
        sz = ctypes.POINTER(ctypes.c_size_t)
        L.d2moe_status_string.argtypes = [_I]
        L.d2moe_status_string.restype = ctypes.c_char_p
        L.d2moe_mwq_size.argtypes = [_I, _I, _I, _I, _I, _I, sz, sz, sz]
        L.d2moe_pack_mwq.argtypes = [_P, _I, ctypes.POINTER(_Mwq), _P]
        L.d2moe_debug_unpack.argtypes = [ctypes.POINTER(_Mwq), _I, _I, _P, _P, _P]
        L.d2moe_mwq_calib_factor_workspace.argtypes = [_I, sz]
        L.d2moe_mwq_calib_factor.argtypes = [_P, _I, _I, ctypes.c_double, _P, _P, _P,
                                             ctypes.c_size_t, _P]
        L.d2moe_pack_mwq_calibrated_workspace.argtypes = [_I, _I, _I, sz]
        L.d2moe_pack_mwq_calibrated.argtypes = [_P, _I, _P, _I, ctypes.POINTER(_Mwq), _P,
                                                ctypes.c_size_t, _P]
        L.d2moe_route.argtypes = [_P, _I, _I, _I, _P, _P, _I, _I, _P, _P, _I, _I, _I,
                                  ctypes.POINTER(_Routing), _P]
        L.d2moe_route_learned.argtypes = [_P, _I, _I, _I, _P, _P, _I, _I, _P, _P, _I, _I, _P,
                                          ctypes.POINTER(_Routing), _P]
        L.d2moe_moe_forward_workspace.argtypes = [_I, _I, _I, _I, _I, _I, sz]
        L.d2moe_moe_forward.argtypes = [_P, _I, _I, _I, _I, _I, _I, ctypes.POINTER(_Mwq),
                                        ctypes.POINTER(_Mwq), ctypes.POINTER(_Routing),
                                        ctypes.POINTER(_Mwq), ctypes.POINTER(_Mwq), _I, _I, _P,
                                        _P, ctypes.c_size_t, _P]
        L.d2moe_moe_forward_profiled.argtypes = L.d2moe_moe_forward.argtypes + [_P]
        L.d2moe_moe_forward_noalloc.argtypes = [_P, _I, _I, _I, _I, _I, _I,
                                                ctypes.POINTER(_Mwq), ctypes.POINTER(_Mwq),
                                                ctypes.POINTER(_Routing), ctypes.POINTER(_Mwq),
                                                ctypes.POINTER(_Mwq), _I, _I, _P, _P]
        L.d2moe_stream_read.argtypes = [_P, ctypes.c_size_t, _P, _I, _P]
        L.d2moe_hebf_order.argtypes = [_P, _I, _I, _I, _P, _P, _P]
        L.d2moe_budget_plan.argtypes = [_P, _I, _I, _P, _I, ctypes.c_int64, _P, _P, _I, _P]
        L.d2moe_moe_forward_streamed.argtypes = [
            _P, _I, _I, _I, _I, _I, _I, ctypes.POINTER(_Mwq), ctypes.POINTER(_Mwq),
            ctypes.POINTER(_Mwq), ctypes.POINTER(_Mwq), _P, ctypes.POINTER(_Routing), _P, _P, _I,
            _P, _P, ctypes.c_size_t, _P, _P, _P]
        L.d2moe_residual_rmsnorm.argtypes = [_P, _P, _I, _I, _I, ctypes.c_float, _P, _I, _P]
        for name in ("d2moe_mwq_size", "d2moe_pack_mwq", "d2moe_debug_unpack", "d2moe_route",
                     "d2moe_mwq_calib_factor_workspace", "d2moe_mwq_calib_factor",
                     "d2moe_pack_mwq_calibrated_workspace", "d2moe_pack_mwq_calibrated",
                     "d2moe_route_learned",
                     "d2moe_moe_forward_workspace", "d2moe_moe_forward",
                     "d2moe_moe_forward_profiled", "d2moe_moe_forward_noalloc",
                     "d2moe_residual_rmsnorm", "d2moe_stream_read", "d2moe_hebf_order",
                     "d2moe_budget_plan", "d2moe_moe_forward_streamed"):
            getattr(L, name).restype = _I
        _lib = L
    return _lib


class D2MoEError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn} failed: {status} ({status_string(status)})")
        self.status = status


def status_string(s: int) -> str:
    return lib().d2moe_status_string(int(s)).decode()


def _check(fn, rc):
    if rc != OK:
        raise D2MoEError(fn, rc)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return D2MOE_F32
    if t.dtype == torch.bfloat16:
        return D2MOE_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


# ---- packed weights ---------------------------------------------------------

def mwq_size(n_experts, rows, cols, group, b_min=2, b_max=8):
    a, b, c = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check("d2moe_mwq_size", lib().d2moe_mwq_size(n_experts, rows, cols, group, b_min, b_max,
                                                  ctypes.byref(a), ctypes.byref(b),
                                                  ctypes.byref(c)))
    return a.value, b.value, c.value


@dataclass
class MWQ:
    """Device buffers of packed MWQ weights (canonical tiled bit-plane layout)."""
    n_experts: int
    rows: int
    cols: int
    group: int
    b_min: int
    b_max: int
    planes: torch.Tensor   # uint32 words, stored as int32
    scales: torch.Tensor   # binary16 bit patterns, stored as int16
    zeros: torch.Tensor    # uint8

    @staticmethod
    def empty(n_experts, rows, cols, group, b_min=2, b_max=8, device="cuda"):
        pb, sb, zb = mwq_size(n_experts, rows, cols, group, b_min, b_max)
        return MWQ(n_experts, rows, cols, group, b_min, b_max,
                   torch.empty(pb // 4, dtype=torch.int32, device=device),
                   torch.empty(sb // 2, dtype=torch.int16, device=device),
                   torch.empty(zb, dtype=torch.uint8, device=device))

    def _c(self) -> _Mwq:
        return _Mwq(self.n_experts, self.rows, self.cols, self.group, self.b_min, self.b_max,
                    self.planes.data_ptr(), self.scales.data_ptr(), self.zeros.data_ptr())

    def nbytes(self):
        return self.planes.numel() * 4 + self.scales.numel() * 2 + self.zeros.numel()

    def expert(self, e: int) -> "MWQ":
        """View of expert e as a one-expert MWQ (experts are outermost)."""
        np_, ns, nz = (t.numel() // self.n_experts for t in (self.planes, self.scales, self.zeros))
        return MWQ(1, self.rows, self.cols, self.group, self.b_min, self.b_max,
                   self.planes.narrow(0, e * np_, np_), self.scales.narrow(0, e * ns, ns),
                   self.zeros.narrow(0, e * nz, nz))


def pack_mwq(W: torch.Tensor, out: MWQ, stream=None) -> MWQ:
    """Quantize + pack W [n_experts][rows][cols] (fp32, device) into ``out``."""
    assert W.is_cuda and W.is_contiguous()
    c = out._c()
    _check("d2moe_pack_mwq", lib().d2moe_pack_mwq(_ptr(W), _dtype_code(W), ctypes.byref(c),
                                                  _stream(stream)))
    return out


def mwq_calib_factor(X: torch.Tensor, lam: float, stream=None):
    """``d2moe_mwq_calib_factor``: X [tokens][h] float (device) ->
    (U [h][h] float, info int32 tensor of one element)."""
    T, h = X.shape
    n = ctypes.c_size_t()
    _check("d2moe_mwq_calib_factor_workspace",
           lib().d2moe_mwq_calib_factor_workspace(h, ctypes.byref(n)))
    ws = torch.empty(n.value, dtype=torch.uint8, device=X.device)
    U = torch.empty((h, h), dtype=torch.float32, device=X.device)
    info = torch.empty(1, dtype=torch.int32, device=X.device)
    _check("d2moe_mwq_calib_factor",
           lib().d2moe_mwq_calib_factor(_ptr(X), T, h, float(lam), _ptr(U), _ptr(info), _ptr(ws),
                                        n.value, _stream(stream)))
    return U, info


def pack_mwq_calibrated(W: torch.Tensor, U: torch.Tensor, gamma: int, out: MWQ,
                        stream=None) -> MWQ:
    """``d2moe_pack_mwq_calibrated``: W [n_experts][rows][cols] float and the
    factor U [cols][cols] float, both on the device."""
    assert W.is_cuda and W.is_contiguous() and U.is_contiguous()
    n = ctypes.c_size_t()
    _check("d2moe_pack_mwq_calibrated_workspace",
           lib().d2moe_pack_mwq_calibrated_workspace(out.rows, out.cols, gamma, ctypes.byref(n)))
    ws = torch.empty(n.value, dtype=torch.uint8, device=W.device)
    c = out._c()
    _check("d2moe_pack_mwq_calibrated",
           lib().d2moe_pack_mwq_calibrated(_ptr(W), _dtype_code(W), _ptr(U), gamma,
                                           ctypes.byref(c), _ptr(ws), n.value, _stream(stream)))
    return out


def debug_unpack(w: MWQ, expert: int, bits: int, stream=None):
    """(q1 [rows][cols] uint8, signs [bits-b_min][rows][cols] int8 or None)."""
    dev = w.planes.device
    q1 = torch.empty((w.rows, w.cols), dtype=torch.uint8, device=dev)
    signs = (torch.empty((bits - w.b_min, w.rows, w.cols), dtype=torch.int8, device=dev)
             if bits > w.b_min else None)
    c = w._c()
    _check("d2moe_debug_unpack", lib().d2moe_debug_unpack(ctypes.byref(c), expert, bits,
                                                          _ptr(q1), _ptr(signs),
                                                          _stream(stream)))
    return q1, signs


# ---- routing ----------------------------------------------------------------

@dataclass
class Routing:
    logits: torch.Tensor
    topk_idx: torch.Tensor
    topk_w: torch.Tensor
    topk_bits: torch.Tensor
    hist: torch.Tensor
    offsets: torch.Tensor
    perm: torch.Tensor
    slot_of: torch.Tensor
    expert_maxbit: torch.Tensor
    flags: torch.Tensor

    @staticmethod
    def empty(T, E, k, b_min=2, b_max=8, device="cuda"):
        L = b_max - b_min + 1
        i32, dev = torch.int32, device
        return Routing(torch.empty((T, E), dtype=torch.float32, device=dev),
                       torch.empty((T, k), dtype=i32, device=dev),
                       torch.empty((T, k), dtype=torch.float32, device=dev),
                       torch.empty((T, k), dtype=torch.uint8, device=dev),
                       torch.empty((E, L), dtype=i32, device=dev),
                       torch.empty(E * L + 1, dtype=i32, device=dev),
                       torch.empty(T * k, dtype=i32, device=dev),
                       torch.empty(T * k, dtype=i32, device=dev),
                       torch.empty(E, dtype=torch.uint8, device=dev),
                       torch.empty(1, dtype=i32, device=dev))

    def _c(self) -> _Routing:
        return _Routing(*[getattr(self, f).data_ptr() for f, _ in _Routing._fields_])


def route(x: torch.Tensor, Wg: torch.Tensor, bias, k: int, token_req, bit_table: torch.Tensor,
          b_min=2, b_max=8, out: Routing | None = None, stream=None) -> Routing:
    T, d = x.shape
    E = Wg.shape[0]
    if out is None:
        out = Routing.empty(T, E, k, b_min, b_max, device=x.device)
    c = out._c()
    _check("d2moe_route", lib().d2moe_route(_ptr(x), _dtype_code(x), T, d, _ptr(Wg), _ptr(bias),
                                            E, k, _ptr(token_req), _ptr(bit_table),
                                            bit_table.shape[0], b_min, b_max, ctypes.byref(c),
                                            _stream(stream)))
    return out


def route_learned(x: torch.Tensor, Wg: torch.Tensor, bias, k: int, Wr: torch.Tensor, br,
                  b_min=2, b_max=8, out: Routing | None = None,
                  bit_logits: torch.Tensor | None = None, stream=None):
    """Dual routing with learned bit-width routers (``d2moe_route_learned``):
    Wr [E][L][d] float, br [E][L] float or None, L = b_max - b_min + 1.
    Returns (routing, bit_logits [T][E][L])."""
    T, d = x.shape
    E = Wg.shape[0]
    L_ = b_max - b_min + 1
    if tuple(Wr.shape) != (E, L_, d):
        raise ValueError(f"Wr must be [E][L][d] = {(E, L_, d)}, got {tuple(Wr.shape)}")
    if out is None:
        out = Routing.empty(T, E, k, b_min, b_max, device=x.device)
    if bit_logits is None:
        bit_logits = torch.empty((T, E, L_), dtype=torch.float32, device=x.device)
    c = out._c()
    _check("d2moe_route_learned",
           lib().d2moe_route_learned(_ptr(x), _dtype_code(x), T, d, _ptr(Wg), _ptr(bias), E, k,
                                     _ptr(Wr), _ptr(br), b_min, b_max, _ptr(bit_logits),
                                     ctypes.byref(c), _stream(stream)))
    return out, bit_logits


# ---- forward ----------------------------------------------------------------

def moe_forward_workspace(T, d, d_ff, E, k, shared_d_ff=0) -> int:
    n = ctypes.c_size_t()
    _check("d2moe_moe_forward_workspace",
           lib().d2moe_moe_forward_workspace(T, d, d_ff, E, k, shared_d_ff, ctypes.byref(n)))
    return n.value


def moe_forward(x: torch.Tensor, w13: MWQ, w2: MWQ, r: Routing, k: int, shared=None,
                out: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                stream=None, events=None) -> torch.Tensor:
    """``shared`` is None or (shared_w13: MWQ, shared_w2: MWQ, shared_bits).
    ``events``: optional 4 torch.cuda.Event (created with enable_timing) that
    are recorded around the W1/W3 and the W2 expert kernels."""
    T, d = x.shape
    E = w13.n_experts
    d_ff = w2.cols
    sw13 = sw2 = None
    sbits = sff = 0
    if shared is not None:
        sw13, sw2, sbits = shared
        sff = sw2.cols
    if out is None:
        out = torch.empty_like(x)
    need = moe_forward_workspace(T, d, d_ff, E, k, sff)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    c13, c2, cr = w13._c(), w2._c(), r._c()
    cs13 = ctypes.byref(sw13._c()) if sw13 is not None else None
    cs2 = ctypes.byref(sw2._c()) if sw2 is not None else None
    args = (_ptr(x), _dtype_code(x), T, d, d_ff, E, k, ctypes.byref(c13), ctypes.byref(c2),
            ctypes.byref(cr), cs13, cs2, sbits, sff, _ptr(out), _ptr(workspace),
            workspace.numel(), _stream(stream))
    if events is None:
        _check("d2moe_moe_forward", lib().d2moe_moe_forward(*args))
    else:
        arr = (ctypes.c_void_p * 4)(*[ev.cuda_event for ev in events])
        _check("d2moe_moe_forward_profiled", lib().d2moe_moe_forward_profiled(*args, arr))
    return out


def moe_forward_noalloc(x: torch.Tensor, w13: MWQ, w2: MWQ, r: Routing, k: int, shared=None,
                        out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """``d2moe_moe_forward_noalloc``: the forward with the library's fixed
    per-GPU scratch array as workspace (nothing is allocated by the call;
    ``out`` is allocated here only when not given)."""
    T, d = x.shape
    sw13 = sw2 = None
    sbits = sff = 0
    if shared is not None:
        sw13, sw2, sbits = shared
        sff = sw2.cols
    if out is None:
        out = torch.empty_like(x)
    c13, c2, cr = w13._c(), w2._c(), r._c()
    cs13 = ctypes.byref(sw13._c()) if sw13 is not None else None
    cs2 = ctypes.byref(sw2._c()) if sw2 is not None else None
    _check("d2moe_moe_forward_noalloc",
           lib().d2moe_moe_forward_noalloc(_ptr(x), _dtype_code(x), T, d, w2.cols,
                                           w13.n_experts, k, ctypes.byref(c13),
                                           ctypes.byref(c2), ctypes.byref(cr), cs13, cs2, sbits,
                                           sff, _ptr(out), _stream(stream)))
    return out


def residual_rmsnorm(x: torch.Tensor, y: torch.Tensor | None, eps: float = 1e-5,
                     h: torch.Tensor | None = None, h_dtype=torch.bfloat16,
                     stream=None) -> torch.Tensor:
    """x [T][d] float32 (updated in place: x += y); returns h = x / rms(x)
    (h_dtype).  y is None or [T][d] bfloat16 / float32."""
    T, d = x.shape
    if x.dtype != torch.float32 or not x.is_contiguous():
        raise ValueError("x must be a contiguous float32 tensor")
    if y is not None and (y.shape != x.shape or not y.is_contiguous()):
        raise ValueError("y must match x")
    if h is None:
        h = torch.empty((T, d), dtype=h_dtype, device=x.device)
    _check("d2moe_residual_rmsnorm",
           lib().d2moe_residual_rmsnorm(_ptr(x), _ptr(y) if y is not None else None,
                                        _dtype_code(y) if y is not None else D2MOE_F32, T, d,
                                        float(eps), _ptr(h), _dtype_code(h), _stream(stream)))
    return h


def stream_read(buf: torch.Tensor, sink: torch.Tensor, stream=None) -> None:
    """``d2moe_stream_read``: read all of ``buf`` once (plain HBM read
    kernel, a measurement helper); ``sink`` is a device int32 tensor with one
    word per workgroup."""
    _check("d2moe_stream_read",
           lib().d2moe_stream_read(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink),
                                   sink.numel(), _stream(stream)))


# ---- streamed weights: HEBF order, memory budget, streamed forward -------------

def hebf_order(hist, b_min=2, b_max=8, resident=None):
    """``d2moe_hebf_order`` on host arrays: hist [E][L] int -> list of units
    (expert, bits, load_from, load_to, count) in I/O order."""
    import numpy as np
    h = np.ascontiguousarray(hist, dtype=np.int32)
    E = h.shape[0]
    res = None if resident is None else np.ascontiguousarray(resident, dtype=np.uint8)
    units = (_Unit * max(1, h.size))()
    n = ctypes.c_int32()
    _check("d2moe_hebf_order",
           lib().d2moe_hebf_order(h.ctypes.data_as(_P), E, b_min, b_max,
                                  None if res is None else res.ctypes.data_as(_P), units,
                                  ctypes.byref(n)))
    return [(u.expert, u.bits, u.load_from, u.load_to, u.count) for u in units[:n.value]]


def budget_plan(want, level_bytes, budget, resident):
    """``d2moe_budget_plan`` on host arrays: want [n_layers][E] level counts,
    level_bytes [K], resident [n_layers][E] uint8 (updated in place).
    Returns the actions as (action, layer, expert, level) tuples."""
    import numpy as np
    w = np.ascontiguousarray(want, dtype=np.uint8)
    lb = np.ascontiguousarray(level_bytes, dtype=np.int64)
    assert resident.dtype == np.uint8 and resident.flags["C_CONTIGUOUS"]
    nl, E = w.shape
    n = ctypes.c_int32()
    cap = 64
    while True:
        acts = (_BudgetAction * cap)()
        rc = lib().d2moe_budget_plan(w.ctypes.data_as(_P), nl, E, lb.ctypes.data_as(_P), lb.size,
                                     int(budget), resident.ctypes.data_as(_P), acts, cap,
                                     ctypes.byref(n))
        if rc == EINVAL and n.value > cap:
            cap = n.value
            continue
        _check("d2moe_budget_plan", rc)
        return [(a.action, a.layer, a.expert, a.level) for a in acts[:n.value]]


def moe_forward_streamed(x, host_w13: MWQ, host_w2: MWQ, w13: MWQ, w2: MWQ, resident, r: Routing,
                         k: int, hist_host, units, events, io_stream, out=None, workspace=None,
                         stream=None):
    """``d2moe_moe_forward_streamed``: host_w13 / host_w2 hold pinned host
    tensors, w13 / w2 the device copy; resident is a host uint8 numpy array
    [E] (updated in place); units as returned by hebf_order; events: one
    torch.cuda.Event per unit; io_stream: a torch.cuda.Stream."""
    import numpy as np
    T, d = x.shape
    E, d_ff = w13.n_experts, w2.cols
    if out is None:
        out = torch.empty_like(x)
    need = moe_forward_workspace(T, d, d_ff, E, k)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=x.device)
    h = np.ascontiguousarray(hist_host, dtype=np.int32)
    assert resident.dtype == np.uint8 and resident.flags["C_CONTIGUOUS"]
    arr_u = (_Unit * max(1, len(units)))(*[_Unit(*u) for u in units])
    for ev in events:
        if ev.cuda_event == 0:
            ev.record(io_stream)          # torch creates the HIP event at its first record
    arr_e = (ctypes.c_void_p * max(1, len(units)))(*[ev.cuda_event for ev in events])
    c_h13, c_h2, c13, c2, cr = host_w13._c(), host_w2._c(), w13._c(), w2._c(), r._c()
    _check("d2moe_moe_forward_streamed",
           lib().d2moe_moe_forward_streamed(
               _ptr(x), _dtype_code(x), T, d, d_ff, E, k, ctypes.byref(c_h13), ctypes.byref(c_h2),
               ctypes.byref(c13), ctypes.byref(c2), resident.ctypes.data_as(_P), ctypes.byref(cr),
               h.ctypes.data_as(_P), arr_u, len(units), _ptr(out), _ptr(workspace),
               workspace.numel(), _stream(stream), ctypes.c_void_p(io_stream.cuda_stream), arr_e))
    return out
