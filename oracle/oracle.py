"""Python face of the CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by ``__graft_entry__.smoke()``
and by the CPU-baseline leg of ``bench.py``; the product package never imports
it.  It shares no code with the GPU path: the C file is compiled here with gcc
and driven through ctypes, and this module only marshals numpy arrays.

Every routine follows a passage of the paper (D^2MoE, arXiv 2504.15299):
  * ``mwq_quantize``   -- Sec. 3.3.1, Eq. 2-5, Algorithm 1 read with X = I;
  * ``mwq_dequant``    -- the nested dequantized weight defined under Eq. 5;
  * ``mwq_hessian`` / ``mwq_inv_chol_upper`` / ``mwq_quantize_calibrated``
                       -- calibration-aware MWQ: the regularised Hessian of
                          Algorithm 1, the upper Cholesky factor of its
                          inverse, and MWQ with Algorithm 1's block-level
                          error compensation (Eq. 3 and Eq. 5 with X);
  * ``mwq_pack``       -- the canonical bit-plane layout (planes 0..b-1 are a
                          b-bit read; Sec. 3.4 nested reuse of low bit-widths);
  * ``gate_logits`` / ``route_from_logits`` -- dual routing (Fig. 1): top-k
                          expert IDs plus a bit-width per activated expert, and
                          the selection counts B_{j,k} of Sec. 3.4.3;
  * ``bit_router_probs`` / ``bit_router_choice`` / ``route_learned`` -- the
                          token-adaptive bit-width routers of Sec. 3.2 (one
                          per expert, a probability over the nest's widths,
                          the most probable width used at inference);
  * ``expert_ffn`` / ``combine`` / ``moe_layer`` -- a SwiGLU expert FFN at the
                          selected bit-width and the weighted combine;
  * ``hebf_order`` / ``budget_plan`` -- the Hottest-Expert-Bit-First I/O order
                          of Sec. 3.4.3 and the memory-budget scheduler of
                          Algorithm 2 (Sec. 3.4.1), host-side planning.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c with gcc (no FMA contraction, no fast math)."""
    stale = (not os.path.exists(_LIB_PATH)) or (
        os.path.getmtime(_LIB_PATH) < max(os.path.getmtime(_SRC),
                                          os.path.getmtime(os.path.join(_HERE, "oracle.h"))))
    if force or stale:
        tmp = _LIB_PATH + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math",
                               "-shared", "-fPIC", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _L():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB_PATH)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.oracle_f32_to_f16.argtypes = [ctypes.c_float]
        lib.oracle_f32_to_f16.restype = ctypes.c_uint16
        lib.oracle_f16_to_f32.argtypes = [ctypes.c_uint16]
        lib.oracle_f16_to_f32.restype = ctypes.c_float
        lib.oracle_round_bf16.argtypes = [ctypes.c_float]
        lib.oracle_round_bf16.restype = ctypes.c_float
        lib.oracle_mwq_quantize.argtypes = [P, I, I, I, I, I, P, P, P, P, P]
        lib.oracle_mwq_dequant.argtypes = [I, I, I, I, I, I, P, P, P, P, P]
        lib.oracle_mwq_quantize_calibrated.argtypes = [P, I, I, I, I, I, P, I, P, P, P, P, P]
        lib.oracle_mwq_pack.argtypes = [I, I, I, I, I, P, P, P, P, P, P, P]
        lib.oracle_gate_logits.argtypes = [P, I, I, P, P, I, P]
        lib.oracle_route_from_logits.argtypes = [P, I, I, I, P, P, I, I, I, P, P, P, P, P, P, P, P]
        lib.oracle_expert_ffn.argtypes = [I, I, I, I, I, I, I, I, P, P, P, P, P, P, P, P, P, I, P]
        lib.oracle_combine.argtypes = [I, I, I, P, P, P]
        lib.oracle_rmsnorm.argtypes = [I, I, ctypes.c_double, P, P]
        for name in ("oracle_mwq_quantize", "oracle_mwq_dequant", "oracle_mwq_pack",
                     "oracle_mwq_quantize_calibrated",
                     "oracle_gate_logits", "oracle_route_from_logits", "oracle_expert_ffn",
                     "oracle_combine", "oracle_rmsnorm"):
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
    return _lib


def _p(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _ok(rc: int, what: str):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with code {rc}")


# ---- number formats --------------------------------------------------------

def f32_to_f16_bits(values) -> np.ndarray:
    L = _L()
    v = np.asarray(values, dtype=np.float32).ravel()
    return np.array([L.oracle_f32_to_f16(float(x)) for x in v], dtype=np.uint16)


def f16_bits_to_f32(bits) -> np.ndarray:
    L = _L()
    v = np.asarray(bits, dtype=np.uint16).ravel()
    return np.array([L.oracle_f16_to_f32(int(x)) for x in v], dtype=np.float32)


def round_bf16(values) -> np.ndarray:
    L = _L()
    v = np.asarray(values, dtype=np.float32).ravel()
    return np.array([L.oracle_round_bf16(float(x)) for x in v], dtype=np.float32)


# ---- MWQ -------------------------------------------------------------------

class MWQCodes:
    """Logical MWQ codes of one [rows][cols] matrix."""

    def __init__(self, rows, cols, group, b_min, b_max, q1, zeros, scales, signs, resid_sq):
        self.rows, self.cols, self.group = rows, cols, group
        self.b_min, self.b_max = b_min, b_max
        self.q1, self.zeros, self.scales, self.signs = q1, zeros, scales, signs
        self.resid_sq = resid_sq

    @property
    def levels(self):
        return self.b_max - self.b_min + 1


def mwq_quantize(W: np.ndarray, group: int, b_min: int = 2, b_max: int = 8) -> MWQCodes:
    W = np.ascontiguousarray(W, dtype=np.float32)
    rows, cols = W.shape
    ng = cols // group
    L = b_max - b_min + 1
    q1 = np.zeros((rows, cols), np.uint8)
    zeros = np.zeros((rows, ng), np.uint8)
    scales = np.zeros((L, rows, ng), np.uint16)
    signs = np.zeros((max(b_max - b_min, 1), rows, cols), np.uint8)
    resid = np.zeros((L, rows, ng), np.float64)
    _ok(_L().oracle_mwq_quantize(_p(W), rows, cols, group, b_min, b_max, _p(q1), _p(zeros),
                                 _p(scales), _p(signs), _p(resid)), "mwq_quantize")
    return MWQCodes(rows, cols, group, b_min, b_max, q1, zeros, scales,
                    signs[: b_max - b_min], resid)


# ---- calibration-aware MWQ (Sec. 3.3.1, Algorithm 1) ---------------------

def mwq_hessian(X: np.ndarray, lam: float) -> np.ndarray:
    """H = 2 X X^T + lambda I of Algorithm 1, binary64.  X is given as
    [tokens][features] (the paper's X^T), so H = 2 X^T X + lambda I here."""
    X = np.asarray(X, dtype=np.float64)
    return 2.0 * (X.T @ X) + lam * np.eye(X.shape[1])


def mwq_inv_chol_upper(H: np.ndarray) -> np.ndarray:
    """The H^c of Algorithm 1: the upper-triangular Cholesky factor U of
    H^-1 (H^-1 = U^T U), binary64, from numpy's inverse and Cholesky."""
    L = np.linalg.cholesky(np.linalg.inv(np.asarray(H, dtype=np.float64)))
    return np.ascontiguousarray(L.T)


def mwq_quantize_calibrated(W: np.ndarray, U: np.ndarray, group: int, gamma: int = 128,
                            b_min: int = 2, b_max: int = 8, with_targets: bool = False):
    """MWQ with Algorithm 1's block compensation (oracle.c documents the
    steps).  U: [cols][cols] upper factor, used in binary32.  Returns the
    codes, and with ``with_targets`` also the per-level values each column
    had when its block was quantized ([levels][rows][cols] float32)."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    U32 = np.ascontiguousarray(U, dtype=np.float32)
    rows, cols = W.shape
    ng = cols // group
    L = b_max - b_min + 1
    q1 = np.zeros((rows, cols), np.uint8)
    zeros = np.zeros((rows, ng), np.uint8)
    scales = np.zeros((L, rows, ng), np.uint16)
    signs = np.zeros((max(b_max - b_min, 1), rows, cols), np.uint8)
    targets = np.zeros((L, rows, cols), np.float32) if with_targets else None
    _ok(_L().oracle_mwq_quantize_calibrated(_p(W), rows, cols, group, b_min, b_max, _p(U32),
                                            gamma, _p(q1), _p(zeros), _p(scales), _p(signs),
                                            _p(targets)), "mwq_quantize_calibrated")
    c = MWQCodes(rows, cols, group, b_min, b_max, q1, zeros, scales, signs[: b_max - b_min],
                 None)
    return (c, targets) if with_targets else c


def mwq_dequant(c: MWQCodes, b: int) -> np.ndarray:
    out = np.zeros((c.rows, c.cols), np.float64)
    signs = c.signs if c.signs.size else np.zeros((1, c.rows, c.cols), np.uint8)
    _ok(_L().oracle_mwq_dequant(c.rows, c.cols, c.group, c.b_min, c.b_max, b, _p(c.q1),
                                _p(c.zeros), _p(c.scales), _p(np.ascontiguousarray(signs)),
                                _p(out)), "mwq_dequant")
    return out


def mwq_sizes(rows: int, cols: int, group: int, b_min: int, b_max: int):
    """(plane words, scale entries, zero entries) of one packed matrix."""
    return rows * cols // 32 * b_max, rows * (cols // group) * (b_max - b_min + 1), \
        rows * (cols // group)


def mwq_pack(c: MWQCodes):
    nw, ns, nz = mwq_sizes(c.rows, c.cols, c.group, c.b_min, c.b_max)
    planes = np.zeros(nw, np.uint32)
    scales = np.zeros(ns, np.uint16)
    zeros = np.zeros(nz, np.uint8)
    signs = c.signs if c.signs.size else np.zeros((1, c.rows, c.cols), np.uint8)
    _ok(_L().oracle_mwq_pack(c.rows, c.cols, c.group, c.b_min, c.b_max, _p(c.q1), _p(c.zeros),
                             _p(c.scales), _p(np.ascontiguousarray(signs)), _p(planes),
                             _p(scales), _p(zeros)), "mwq_pack")
    return planes, scales, zeros


# ---- routing ---------------------------------------------------------------

def gate_logits(x: np.ndarray, Wg: np.ndarray, bias: np.ndarray | None = None) -> np.ndarray:
    x = np.ascontiguousarray(x, dtype=np.float32)
    Wg = np.ascontiguousarray(Wg, dtype=np.float32)
    T, d = x.shape
    E = Wg.shape[0]
    out = np.zeros((T, E), np.float64)
    b = None if bias is None else np.ascontiguousarray(bias, dtype=np.float32)
    _ok(_L().oracle_gate_logits(_p(x), T, d, _p(Wg), _p(b), E, _p(out)), "gate_logits")
    return out


def route_from_logits(logits: np.ndarray, k: int, token_req: np.ndarray | None,
                      bit_table: np.ndarray, b_min: int = 2, b_max: int = 8) -> dict:
    logits = np.ascontiguousarray(logits, dtype=np.float64)
    T, E = logits.shape
    bit_table = np.ascontiguousarray(bit_table, dtype=np.uint8)
    R = bit_table.shape[0]
    req = None if token_req is None else np.ascontiguousarray(token_req, dtype=np.int32)
    L = b_max - b_min + 1
    o = dict(topk_idx=np.zeros((T, k), np.int32), topk_w=np.zeros((T, k), np.float64),
             topk_bits=np.zeros((T, k), np.uint8), hist=np.zeros((E, L), np.int32),
             offsets=np.zeros(E * L + 1, np.int32), perm=np.zeros(T * k, np.int32),
             slot_of=np.zeros(T * k, np.int32), maxbit=np.zeros(E, np.uint8))
    rc = _L().oracle_route_from_logits(
        _p(logits), T, E, k, _p(req), _p(bit_table), R, b_min, b_max, _p(o["topk_idx"]),
        _p(o["topk_w"]), _p(o["topk_bits"]), _p(o["hist"]), _p(o["offsets"]), _p(o["perm"]),
        _p(o["slot_of"]), _p(o["maxbit"]))
    _ok(rc, "route_from_logits")
    return o


# ---- learned bit-width routers (Sec. 3.2) -----------------------------------

def bit_router_probs(bit_logits: np.ndarray) -> np.ndarray:
    """Sec. 3.2: each expert's bit-width router assigns the token a probability
    over the nest's candidate widths b_min..b_max, the softmax of its scores
    (the p_k of Eq. 1).  bit_logits [..., L] -> probabilities [..., L],
    binary64."""
    z = np.asarray(bit_logits, dtype=np.float64)
    e = np.exp(z - z.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def bit_router_choice(bit_logits: np.ndarray, b_min: int) -> np.ndarray:
    """The width each router selects at inference: its most probable
    candidate, i.e. the largest score (the softmax is increasing), the lowest
    width when scores are equal.  bit_logits [T][E][L] -> uint8 [T][E]."""
    z = np.asarray(bit_logits, dtype=np.float64)
    T, E, L = z.shape
    out = np.zeros((T, E), np.uint8)
    for t in range(T):
        for e in range(E):
            best = 0
            for l in range(1, L):
                if z[t, e, l] > z[t, e, best]:
                    best = l
            out[t, e] = b_min + best
    return out


def route_learned(logits: np.ndarray, k: int, bit_logits: np.ndarray, b_min: int = 2,
                  b_max: int = 8) -> dict:
    """Dual routing with the learned routers: the top-k experts of
    ``route_from_logits``, each activated expert at its router's choice for
    the token.  The choices form a per-(token, expert) width table, i.e. one
    request per token."""
    choice = bit_router_choice(bit_logits, b_min)
    T = choice.shape[0]
    return route_from_logits(logits, k, np.arange(T, dtype=np.int32), choice, b_min, b_max)


# ---- expert FFN, combine, whole layer --------------------------------------

def expert_ffn(c13: MWQCodes, c2: MWQCodes, b: int, x: np.ndarray) -> np.ndarray:
    """y = W2_b (silu(W1_b x) * W3_b x) for each row of x, binary64.  ``c2``
    may hold a subset of W2's rows (codes are per row); y has c2.rows
    columns."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    n, d = x.shape
    f = c2.cols
    assert c13.rows == 2 * f and c13.cols == d
    y = np.zeros((n, c2.rows), np.float64)
    s13 = c13.signs if c13.signs.size else np.zeros((1, c13.rows, c13.cols), np.uint8)
    s2 = c2.signs if c2.signs.size else np.zeros((1, c2.rows, c2.cols), np.uint8)
    _ok(_L().oracle_expert_ffn(d, f, c2.rows, c13.group, c2.group, c13.b_min, c13.b_max, b,
                               _p(c13.q1),
                               _p(c13.zeros), _p(c13.scales), _p(np.ascontiguousarray(s13)),
                               _p(c2.q1), _p(c2.zeros), _p(c2.scales),
                               _p(np.ascontiguousarray(s2)), _p(x), n, _p(y)), "expert_ffn")
    return y


def combine(topk_w: np.ndarray, y_slot: np.ndarray) -> np.ndarray:
    topk_w = np.ascontiguousarray(topk_w, dtype=np.float64)
    T, k = topk_w.shape
    d = y_slot.shape[-1]
    y_slot = np.ascontiguousarray(y_slot.reshape(T * k, d), dtype=np.float64)
    out = np.zeros((T, d), np.float64)
    _ok(_L().oracle_combine(T, k, d, _p(topk_w), _p(y_slot), _p(out)), "combine")
    return out


def moe_layer(x: np.ndarray, route: dict, codes13: list, codes2: list, tokens=None,
              shared=None) -> np.ndarray:
    """MoE layer output for the listed tokens (all if None), binary64.

    ``route`` is the output of ``route_from_logits``; ``codes13[e]`` and
    ``codes2[e]`` are the logical codes of expert e; ``shared`` is None or
    (codes13, codes2, bits) of an always-on expert added with weight 1.
    Expert outputs are computed per (expert, bit-width) group of slots."""
    x = np.asarray(x, dtype=np.float32)
    T, d = x.shape
    idx, bits, w = route["topk_idx"], route["topk_bits"], route["topk_w"]
    k = idx.shape[1]
    toks = np.arange(T) if tokens is None else np.asarray(tokens)
    y_slot = np.zeros((len(toks), k, d), np.float64)
    for e in range(len(codes13)):
        for b in sorted(set(int(v) for v in bits[toks][idx[toks] == e])):
            sel = [(j, i) for j, t in enumerate(toks) for i in range(k)
                   if idx[t, i] == e and bits[t, i] == b]
            if not sel:
                continue
            xs = np.stack([x[toks[j]] for j, _ in sel]).astype(np.float64)
            ys = expert_ffn(codes13[e], codes2[e], b, xs)
            for (j, i), yv in zip(sel, ys):
                y_slot[j, i] = yv
    out = combine(w[toks], y_slot)
    if shared is not None:
        s13, s2, sb = shared
        out = out + expert_ffn(s13, s2, sb, x[toks].astype(np.float64))
    return out


# ---- decoder stack of MoE layers ---------------------------------------------

def rmsnorm(x: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """x / sqrt(mean(x^2) + eps) per row, binary64 (unit normalisation weight)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    T, d = x.shape
    h = np.zeros_like(x)
    _ok(_L().oracle_rmsnorm(T, d, float(eps), _p(x), _p(h)), "rmsnorm")
    return h


def moe_stack(x0: np.ndarray, layers: list, k: int, token_req, bit_table, eps: float = 1e-5,
              b_min: int = 2, b_max: int = 8):
    """A stack of MoE blocks x <- x + MoE_l(rmsnorm(x)) (attention absent).
    The MoE layer sees bf16 activations and returns bf16 outputs, as the
    layer does for bf16 inputs; the residual stream is binary64.
    ``layers[l]`` = (Wg, codes13, codes2).  Returns the final stream and, per
    layer, the layer's binary64 logits (to tell near-tied tokens)."""
    x = np.asarray(x0, dtype=np.float64).copy()
    logits_per_layer = []
    for Wg, c13, c2 in layers:
        h = round_bf16(rmsnorm(x, eps).astype(np.float32)).reshape(x.shape)
        logits = gate_logits(h, Wg)
        logits_per_layer.append(logits)
        route = route_from_logits(logits, k, token_req, bit_table, b_min, b_max)
        y = moe_layer(h, route, c13, c2)
        x = x + round_bf16(y.astype(np.float32)).reshape(y.shape).astype(np.float64)
    return x, logits_per_layer


# ---- bit-width-aware I/O-compute planning (Sec. 3.4) -----------------------

def hebf_order(B: np.ndarray, b_min: int, resident=None):
    """Hottest-Expert-Bit-First (Sec. 3.4.3).  B[j][k]: how many requests
    selected bit-width b_min + k of expert j (the B_{j,k} of the planning
    problem).  resident[j]: the bit-width whose planes are already on the
    device (0: none).
      1. a queue per expert of its requested bit-widths, ascending;
      2. repeatedly take, among the heads of all queues, the one with the
         highest count B_{j,k} (ties: lower expert index) and append it to
         the I/O queue;
      3. (execution) load the units in that order, computing each once its
         load is done.
    A unit is (expert, bit-width, loaded from, loaded to, count): its
    computation is the requests at that bit-width, and its load brings the
    expert's planes from the width already present up to the unit's, the
    nested delta that this width adds to the lower ones (nothing when the
    width is already present)."""
    B = np.asarray(B)
    E, L = B.shape
    res = [0] * E if resident is None else [int(v) for v in resident]
    queues = [[b_min + k for k in range(L) if B[j][k] > 0] for j in range(E)]
    have = list(res)
    out = []
    while any(queues):
        best = None
        for j in range(E):
            if not queues[j]:
                continue
            c = int(B[j][queues[j][0] - b_min])
            if best is None or c > best[1]:
                best = (j, c)
        j = best[0]
        b = queues[j].pop(0)
        frm = have[j]
        out.append((j, b, frm, max(frm, b), int(B[j][b - b_min])))
        have[j] = max(frm, b)
    return out


def budget_plan(want, unit_bytes, budget, resident=None):
    """Memory-budget scheduler of Algorithm 2 (Sec. 3.4.1) over one pass of
    the layers.  want[j][e]: how many levels layer j's expert e needs (0:
    unused; a bit-width b is b - b_min + 1 levels);
    unit_bytes[l]: bytes one expert's level l occupies (level 0: the base
    planes with their scale and zero points, level l >= 1: one residual
    plane with its scales); budget: bytes available for expert weights;
    resident[j][e]: the level count already on the device (0: none).
    For each layer j: if loading what it needs (the levels above the
    resident ones) exceeds the free budget, free levels of the layers before
    it, the previous layer first (j-1, then j-2, ...), highest levels first
    (one level of every expert of that layer at a time, experts ascending),
    the base level last, until the load fits; then load.  The layer itself
    is never freed.  Returns (actions, resident): actions is a list of
    ("free" | "load", layer, expert, level) in order, resident the final
    level counts."""
    want = np.asarray(want)
    nl, E = want.shape
    K = len(unit_bytes)
    res = np.zeros((nl, E), np.int64) if resident is None else np.array(resident, np.int64)
    used = int(sum(sum(unit_bytes[l] for l in range(res[j][e])) for j in range(nl)
                   for e in range(E)))
    free = budget - used
    actions = []
    for j in range(nl):
        need = 0
        for e in range(E):
            for l in range(res[j][e], want[j][e]):
                need += unit_bytes[l]
        for jj in range(j - 1, -1, -1):
            if need <= free:
                break
            for l in range(K - 1, -1, -1):
                if need <= free:
                    break
                for e in range(E):
                    if res[jj][e] == l + 1:
                        actions.append(("free", jj, e, l))
                        res[jj][e] = l
                        free += unit_bytes[l]
        for e in range(E):
            for l in range(res[j][e], want[j][e]):
                actions.append(("load", j, e, l))
                free -= unit_bytes[l]
            res[j][e] = max(res[j][e], want[j][e])
    return actions, res
