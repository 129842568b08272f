"""CPU oracle for mixed-policy KV attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never does; the two
share no code.  The arithmetic lives in ``ucref.cpp`` (plain C++, fp64
attention and scoring, binary32 quantizer); this module only marshals numpy
arrays into it and assembles the logical sequence the paper's reference
formulation attends over (App. E: masks for evicted rows, fake quantization
for quantised rows).

Parity status of each function is recorded in its docstring: every function
here is pinned by tests in ``tests/test_oracle_*.py`` against closed forms,
brute force or library routines; none is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.environ.get("UCREF_LIB") or os.path.join(HERE, "libucref.so")  # override: sanitized builds
_lib = None

DT = {"f32": 0, "f16": 1, "bf16": 2}
ELEM = {"f32": 4, "f16": 2, "bf16": 2}


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64, dbl = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_double
        sig = {
            "ucref_widen": (None, [vp, i32, i64, vp]),
            "ucref_round_value": (None, [vp, i32, i64, vp]),
            "ucref_quantize": (i32, [i32, i32, i32, i32, vp, i32, vp, vp, vp, vp, vp,
                                     vp, vp, vp, vp, vp, vp]),
            "ucref_dequant": (i32, [i32, i32, i32, i32, vp, i32, vp, vp, vp, vp, vp,
                                    vp, vp, vp, vp, vp, vp]),
            "ucref_score": (None, [i32, i32, i32, i32, i32, i64, vp, vp, vp, i32, dbl,
                                   vp, vp]),
            "ucref_select": (i32, [i32, i32, vp, i32, i32, vp]),
            "ucref_attend": (None, [i32, i32, i32, i32, i32, i64, vp, vp, vp, vp, vp,
                                    i32, dbl, vp, vp, vp, vp]),
            "ucref_dense_bytes": (i64, [i64, i32, i32]),
            "ucref_evicted_bytes": (i64, [i64, i32, i32]),
            "ucref_packed_bytes": (i64, [i64, i32, i32, i32, i32]),
            "ucref_evict_rows": (i64, [dbl, dbl, i64, i32, i32]),
            "ucref_assign_bits": (i32, [i32, vp, i64, i32, i32, i32, dbl, dbl, vp]),
            "ucref_type_budget": (i32, [i32, vp, vp, dbl, vp]),
            "ucref_quant_config": (i32, [dbl, i64, i32, i32, i32, i32]),
            "ucref_topk_mass": (i32, [i32, i32, vp, i32, vp]),
            "ucref_retention_next": (dbl, [dbl, dbl, dbl, dbl, dbl]),
            "ucref_set_threads": (i32, [i32]),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype=None):
    return np.ascontiguousarray(a, dtype=dtype) if a is not None else None


def set_threads(n: int) -> int:
    return int(lib().ucref_set_threads(n))


# ---- element types --------------------------------------------------------

def widen(x: np.ndarray, dtype: str) -> np.ndarray:
    """Stored elements (bf16 as uint16 bits) -> exact float64."""
    x = np.ascontiguousarray(x)
    out = np.empty(x.shape, np.float64)
    lib().ucref_widen(x.ctypes.data, DT[dtype], x.size, out.ctypes.data)
    return out


def round_value(x: np.ndarray, dtype: str) -> np.ndarray:
    """binary32 values after round-to-nearest-even into dtype, as float64."""
    x = np.ascontiguousarray(x, np.float32)
    out = np.empty(x.shape, np.float64)
    lib().ucref_round_value(x.ctypes.data, DT[dtype], x.size, out.ctypes.data)
    return out


# ---- quantization ---------------------------------------------------------

def packed_layout(BH: int, N: int, D: int, G: int, bits: Sequence[int]):
    """Per-(b,h) byte offsets of the codes (heads laid out back to back)."""
    n_full = G * (N // G)
    sizes = [n_full * D * int(b) // 8 for b in bits]
    off = np.zeros(BH, np.int64)
    off[1:] = np.cumsum(sizes)[:-1]
    return off, int(sum(sizes))


def quantize(k: np.ndarray, v: np.ndarray, dtype: str, G: int,
             bits: Sequence[int], code_off: Optional[np.ndarray] = None,
             codes_bytes: Optional[int] = None) -> Dict[str, np.ndarray]:
    """Group-wise asymmetric quantization of k, v [BH, N, D] (stored dtype).

    Pinned by: ramp and constant groups, |x - x_hat| <= s/2 bound, code range
    and min/max mapping, brute-force re-derivation on tiny groups."""
    k = np.ascontiguousarray(k)
    v = np.ascontiguousarray(v)
    BH, N, D = k.shape
    bits = np.ascontiguousarray(np.broadcast_to(np.asarray(bits, np.int32), (BH,)))
    off, total = packed_layout(BH, N, D, G, bits)
    if code_off is not None:
        off = np.ascontiguousarray(code_off, np.int64)
        total = codes_bytes
    n_full = G * (N // G)
    tail = N - n_full
    out = {
        "codes_k": np.zeros(max(total, 1), np.uint8),
        "codes_v": np.zeros(max(total, 1), np.uint8),
        "code_off": off,
        "bits": bits,
        "scale_k": np.zeros((BH, n_full // G, D), np.float32),
        "min_k": np.zeros((BH, n_full // G, D), np.float32),
        "scale_v": np.zeros((BH, n_full, D // G), np.float32),
        "min_v": np.zeros((BH, n_full, D // G), np.float32),
        "tail_k": np.zeros((BH, tail, D), k.dtype),
        "tail_v": np.zeros((BH, tail, D), k.dtype),
    }
    rc = lib().ucref_quantize(BH, N, D, G, bits.ctypes.data, DT[dtype], k.ctypes.data,
                              v.ctypes.data, out["codes_k"].ctypes.data,
                              out["codes_v"].ctypes.data, off.ctypes.data,
                              out["scale_k"].ctypes.data, out["min_k"].ctypes.data,
                              out["scale_v"].ctypes.data, out["min_v"].ctypes.data,
                              out["tail_k"].ctypes.data, out["tail_v"].ctypes.data)
    if rc != 0:
        raise ValueError("ucref_quantize: invalid arguments")
    return out


def dequant(pk: Dict[str, np.ndarray], N: int, D: int, G: int, dtype: str):
    """Logical (dequantised, dtype-rounded) K and V [BH, N, D] in float64."""
    BH = pk["bits"].shape[0]
    kh = np.empty((BH, N, D), np.float64)
    vh = np.empty((BH, N, D), np.float64)
    rc = lib().ucref_dequant(BH, N, D, G, pk["bits"].ctypes.data, DT[dtype],
                             pk["codes_k"].ctypes.data, pk["codes_v"].ctypes.data,
                             pk["code_off"].ctypes.data, pk["scale_k"].ctypes.data,
                             pk["min_k"].ctypes.data, pk["scale_v"].ctypes.data,
                             pk["min_v"].ctypes.data, _p(_c(pk["tail_k"])),
                             _p(_c(pk["tail_v"])), kh.ctypes.data, vh.ctypes.data)
    if rc != 0:
        raise ValueError("ucref_dequant: invalid arguments")
    return kh, vh


# ---- scoring, selection, attention ----------------------------------------

def score(q: np.ndarray, k: np.ndarray, seg_of_row: np.ndarray, n_segs: int,
          sm_scale: float) -> Tuple[np.ndarray, np.ndarray]:
    """q [B,Hq,W,D] float64, k [B,Hkv,N,D] float64 -> (score f32 [B,Hkv,N],
    mass f32 [B,Hkv,n_segs]), accumulated in double, rounded once.

    Pinned by: rows of P sum to one (sum of scores = G*W), q = 0 gives a
    uniform score, a dominant logit concentrates the mass, brute force."""
    q = _c(q, np.float64)
    k = _c(k, np.float64)
    B, Hq, W, D = q.shape
    _, Hkv, N, _ = k.shape
    seg = _c(seg_of_row, np.int32)
    sc = np.empty((B, Hkv, N), np.float64)
    ms = np.empty((B, Hkv, n_segs), np.float64)
    lib().ucref_score(B, Hq, Hkv, D, W, N, q.ctypes.data, k.ctypes.data, seg.ctypes.data,
                      n_segs, float(sm_scale), sc.ctypes.data, ms.ctypes.data)
    return sc.astype(np.float32), ms.astype(np.float32)


def score64(q, k, seg_of_row, n_segs, sm_scale):
    """As score() but returning the double-precision sums (for tie analysis)."""
    q = _c(q, np.float64)
    k = _c(k, np.float64)
    B, Hq, W, D = q.shape
    _, Hkv, N, _ = k.shape
    seg = _c(seg_of_row, np.int32)
    sc = np.empty((B, Hkv, N), np.float64)
    ms = np.empty((B, Hkv, n_segs), np.float64)
    lib().ucref_score(B, Hq, Hkv, D, W, N, q.ctypes.data, k.ctypes.data, seg.ctypes.data,
                      n_segs, float(sm_scale), sc.ctypes.data, ms.ctypes.data)
    return sc, ms


def select(scores: np.ndarray, k: int, n_recent: int = 0) -> np.ndarray:
    """scores [BH, N] f32 -> kept positions [BH, k] int32 ascending.

    Pinned by: brute-force sort, count, ascending order, kept >= evicted,
    lower index wins exact ties, k = N / k = 0, recent rows always kept."""
    s = _c(scores, np.float32)
    BH, N = s.shape
    out = np.empty((BH, k), np.int32)
    if lib().ucref_select(BH, N, s.ctypes.data, k, n_recent, out.ctypes.data) != 0:
        raise ValueError("ucref_select: invalid arguments")
    return out


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray,
           present: Optional[np.ndarray], seg_of_row: np.ndarray, n_segs: int,
           sm_scale: float):
    """q [B,Hq,M,D], k/v [B,Hkv,N,D] float64; present [B,Hkv,N] (1 = attended)
    or None.  Returns float64 (o [B,Hq,M,D], lse [B,Hq,M],
    seg_lse [B,Hq,M,n_segs], seg_mass [B,Hq,M,n_segs]).

    Pinned by: brute-force softmax(QK^T/sqrt(d))V, q = 0 gives the mean of V,
    one row gives v, chunked LSE merge equals one pass, segment order
    invariance, masked == compacted."""
    q = _c(q, np.float64)
    k = _c(k, np.float64)
    v = _c(v, np.float64)
    B, Hq, M, D = q.shape
    _, Hkv, N, _ = k.shape
    pr = _c(present, np.uint8)
    seg = _c(seg_of_row, np.int32)
    o = np.empty((B, Hq, M, D))
    lse = np.empty((B, Hq, M))
    sl = np.empty((B, Hq, M, n_segs))
    sm = np.empty((B, Hq, M, n_segs))
    lib().ucref_attend(B, Hq, Hkv, D, M, N, q.ctypes.data, k.ctypes.data, v.ctypes.data,
                       _p(pr), seg.ctypes.data, n_segs, float(sm_scale), o.ctypes.data,
                       lse.ctypes.data, sl.ctypes.data, sm.ctypes.data)
    return o, lse, sl, sm


# ---- accounting and budgets -----------------------------------------------

def dense_bytes(rows: int, D: int, dtype: str) -> int:
    return int(lib().ucref_dense_bytes(rows, D, DT[dtype]))


def evicted_bytes(rows: int, D: int, dtype: str) -> int:
    return int(lib().ucref_evicted_bytes(rows, D, DT[dtype]))


def packed_bytes(N: int, D: int, G: int, bits: int, dtype: str) -> int:
    return int(lib().ucref_packed_bytes(N, D, G, bits, DT[dtype]))


def evict_rows(budget: float, fixed: float, N: int, D: int, dtype: str) -> int:
    return int(lib().ucref_evict_rows(budget, fixed, N, D, DT[dtype]))


def assign_bits(mass: Sequence[float], N: int, D: int, G: int, dtype: str,
                budget: float, fixed: float) -> np.ndarray:
    m = np.ascontiguousarray(mass, np.float64)
    out = np.empty(m.shape[0], np.int32)
    if lib().ucref_assign_bits(m.shape[0], m.ctypes.data, N, D, G, DT[dtype], budget,
                               fixed, out.ctypes.data) != 0:
        raise ValueError("ucref_assign_bits: invalid arguments")
    return out


def type_budget(mass: Sequence[float], b_prev: Sequence[float], B_total: float) -> np.ndarray:
    m = np.ascontiguousarray(mass, np.float64)
    bp = np.ascontiguousarray(b_prev, np.float64)
    out = np.empty(m.shape[0])
    if lib().ucref_type_budget(m.shape[0], m.ctypes.data, bp.ctypes.data, B_total,
                               out.ctypes.data) != 0:
        raise ValueError("ucref_type_budget: invalid arguments")
    return out


def topk_mass(scores: np.ndarray, k: int) -> np.ndarray:
    """scores [BH, N] f32 -> fraction of each row's sum on its k largest
    entries (float64).

    Pinned by: uniform rows give k/N, one dominant entry gives ~1, k = N gives
    1, k = 0 gives 0, brute force against numpy's sort."""
    s = _c(scores, np.float32)
    BH, N = s.shape
    out = np.empty(BH)
    if lib().ucref_topk_mass(BH, N, s.ctypes.data, k, out.ctypes.data) != 0:
        raise ValueError("ucref_topk_mass: invalid arguments")
    return out


def quant_config(budget: float, N: int, D: int, dtype: str, n_heads: int,
                 first: int = 0) -> Tuple[int, int, int]:
    """(index, bits, group) of the most faithful quantization configuration at
    or after `first` whose n_heads packed segments fit the budget (the last
    one if none fits).  Configurations: widths 8, 4, 2; groups 32 ... D.

    Pinned by: hand-computed byte counts at the boundaries of each
    configuration, monotone in the budget, never before `first`."""
    i = int(lib().ucref_quant_config(float(budget), N, D, DT[dtype], n_heads, first))
    if i < 0:
        raise ValueError("ucref_quant_config: invalid arguments")
    ng = int(math.log2(D // 32)) + 1
    return i, 8 >> (i // ng), 32 << (i % ng)


def retention_next(rho, rho_init, rho_min, M_c, M_0) -> float:
    return float(lib().ucref_retention_next(rho, rho_init, rho_min, M_c, M_0))
