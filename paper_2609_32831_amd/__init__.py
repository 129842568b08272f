"""Python binding of libunicache (mixed-policy KV attention for MI355X).

Argument marshalling only: every function forwards to the C ABI declared in
``include/unicache.h`` under the same name; all device work runs in the
library's HIP kernels.  PyTorch supplies device memory and the stream.  There
is no fallback: importing this module fails if ``libunicache.so`` is missing,
and a call raises ``UcError`` when the library returns an error status.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import List, Optional, Sequence

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# UNICACHE_LIB: another build of the same library (the host-sanitized one
# the CPU tests can run against)
LIB_PATH = os.environ.get("UNICACHE_LIB") or os.path.join(HERE, "libunicache.so")

UC_OK, UC_E_INVALID, UC_E_UNSUPPORTED, UC_E_WORKSPACE, UC_E_DEVICE = range(5)
UC_F32, UC_F16, UC_BF16 = 0, 1, 2
UC_SEG_DENSE, UC_SEG_PACKED = 0, 1
UC_MAX_SEGMENTS = 8
UC_PATH_AUTO, UC_PATH_VALU = 0, 1

TORCH_DT = {torch.float32: UC_F32, torch.float16: UC_F16, torch.bfloat16: UC_BF16}
DT_TORCH = {v: k for k, v in TORCH_DT.items()}
NAME_DT = {"f32": UC_F32, "f16": UC_F16, "bf16": UC_BF16}


class UcError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        super().__init__(f"{where}: status {status} ({detail})")
        self.status = status


class uc_shape(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int32), ("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32),
                ("D", ctypes.c_int32)]


class uc_segment(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("n_rows", ctypes.c_int32),
                ("row_stride", ctypes.c_int32), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("idx", ctypes.c_void_p), ("group", ctypes.c_int32), ("bits", ctypes.c_int32),
                ("head_bits", ctypes.c_void_p), ("code_off", ctypes.c_void_p),
                ("codes_bytes", ctypes.c_uint64), ("codes_k", ctypes.c_void_p),
                ("codes_v", ctypes.c_void_p), ("scale_k", ctypes.c_void_p),
                ("min_k", ctypes.c_void_p), ("scale_v", ctypes.c_void_p),
                ("min_v", ctypes.c_void_p), ("tail_k", ctypes.c_void_p),
                ("tail_v", ctypes.c_void_p)]


class uc_budget_params(ctypes.Structure):
    _fields_ = [("Hq", ctypes.c_int32), ("Hkv", ctypes.c_int32), ("D", ctypes.c_int32),
                ("M", ctypes.c_int32), ("n_segs", ctypes.c_int32), ("ev", ctypes.c_int32),
                ("qt", ctypes.c_int32), ("n_ev", ctypes.c_int32), ("n_qt", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("rho_init", ctypes.c_double),
                ("rho_min", ctypes.c_double)]


class uc_budget_state(ctypes.Structure):
    _fields_ = [("rho", ctypes.c_double), ("B", ctypes.c_double), ("M0", ctypes.c_double),
                ("m", ctypes.c_double * 2), ("b", ctypes.c_double * 2),
                ("k", ctypes.c_int32), ("cfg", ctypes.c_int32), ("bits", ctypes.c_int32),
                ("group", ctypes.c_int32), ("k_prev", ctypes.c_int32),
                ("cfg_prev", ctypes.c_int32), ("n_boundaries", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2609_32831_amd/build.py "
                          "(or __graft_entry__.build())")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64, dbl, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                                  ctypes.c_uint64, ctypes.c_double, ctypes.c_size_t)
    shp, segp = ctypes.POINTER(uc_shape), ctypes.POINTER(uc_segment)
    sigs = {
        "uc_score_importance": (i32, [shp, segp, i32, vp, i32, i32, ctypes.c_float, vp, vp, vp,
                                      sz, vp]),
        "uc_score_workspace_size": (sz, [shp, segp, i32, i32]),
        "uc_score_columns": (i32, [shp, segp, i32, vp, i64, i32, i32, ctypes.c_float, vp, i64,
                                   vp, vp, vp, sz, vp]),
        "uc_select_keep": (i32, [vp, i32, i32, i32, i32, vp, vp, vp, vp, vp, i32, i32, vp, sz,
                                 vp]),
        "uc_select_workspace_size": (sz, [i32, i32]),
        "uc_evict_step": (i32, [shp, vp, segp, vp, segp, vp]),
        "uc_quantize_segment": (i32, [shp, vp, vp, i32, i32, segp, vp]),
        "uc_attend_mixed": (i32, [shp, segp, i32, vp, i32, i32, ctypes.c_float, vp, vp, vp, vp,
                                  sz, vp]),
        "uc_attend_workspace_size": (sz, [shp, segp, i32, i32, i32]),
        "uc_attend_mixed_noalloc": (i32, [shp, segp, i32, vp, i32, i32, ctypes.c_float, vp, vp,
                                          vp, vp]),
        "uc_segment_mass": (i32, [shp, i32, i32, vp, vp, vp, vp]),
        "uc_append_rows": (i32, [shp, vp, vp, i32, segp, i32, vp]),
        "uc_attend_append": (i32, [shp, segp, i32, i32, vp, vp, i32, vp, i32, i32,
                                   ctypes.c_float, vp, vp, vp, vp, sz, vp]),
        "uc_dense_bytes": (i64, [i64, i32, i32]),
        "uc_evicted_bytes": (i64, [i64, i32, i32]),
        "uc_packed_bytes": (i64, [i64, i32, i32, i32, i32]),
        "uc_evict_rows_for_budget": (i64, [dbl, dbl, i64, i32, i32]),
        "uc_assign_bits": (i32, [i32, vp, i64, i32, i32, i32, dbl, dbl, vp]),
        "uc_type_budget": (i32, [i32, vp, vp, dbl, vp]),
        "uc_retention_next": (dbl, [dbl, dbl, dbl, dbl, dbl]),
        "uc_status_string": (ctypes.c_char_p, [i32]),
        "uc_last_error": (ctypes.c_char_p, []),
        "uc_last_kernel": (ctypes.c_char_p, []),
        "uc_set_path": (i32, [i32]),
        "uc_set_kernel_events": (i32, [vp, vp]),
        "uc_dequantize_segment": (i32, [shp, segp, vp, vp, vp]),
        "uc_attend_batch": (i32, [shp, vp, vp, vp, i32, i32, ctypes.c_float, vp, vp, vp, sz, vp]),
        "uc_attend_batch_workspace_size": (sz, [shp, vp, vp, i32, i32]),
        "uc_stream_append": (i32, [shp, segp, vp, vp, i32, vp]),
        "uc_compose_index": (i32, [vp, i32, vp, i32, i32, vp, vp]),
        "uc_topk_mass": (i32, [vp, i32, i32, i32, vp, vp, sz, vp]),
        "uc_topk_mass_workspace_size": (sz, [i32, i32]),
        "uc_quant_config": (i32, [dbl, i64, i32, i32, i32, i32, vp, vp]),
        "uc_budget_step": (i32, [ctypes.POINTER(uc_budget_params), vp, i32, vp, vp]),
        "uc_calibrate_policy": (i32, [vp, i32, i32, dbl, vp, vp, vp]),
        "uc_plan_create": (i32, [shp, segp, i32, i32, i32, i32, ctypes.c_float,
                                 ctypes.POINTER(vp)]),
        "uc_plan_workspace_size": (sz, [vp]),
        "uc_plan_tail_rows": (i32, [vp]),
        "uc_plan_attend_append": (i32, [vp, vp, vp, i32, vp, vp, vp, vp, sz, vp]),
        "uc_plan_destroy": (i32, [vp]),
        "uc_plan_attend": (i32, [vp, vp, vp, vp, vp, vp, sz, vp]),
        "uc_plan_invalidate": (i32, [vp]),
        "uc_read_probe_unit": (sz, []),
        "uc_read_probe_sink_bytes": (sz, []),
        "uc_read_probe": (i32, [vp, sz, i32, vp, vp]),
    }
    for name, (res, args) in sigs.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


lib = _load()


def _check(status: int, where: str):
    if status != UC_OK:
        raise UcError(status, where, lib.uc_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        if torch.cuda.is_available():
            return torch.cuda.current_stream().cuda_stream
        return None
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def make_shape(B: int, Hq: int, Hkv: int, D: int) -> uc_shape:
    return uc_shape(B, Hq, Hkv, D)


class Segment:
    """One segment of the logical KV sequence plus the tensors it points into
    (kept alive with the descriptor)."""

    def __init__(self, desc: uc_segment, tensors: dict):
        self.desc = desc
        self.t = tensors

    @property
    def n_rows(self) -> int:
        return self.desc.n_rows

    @n_rows.setter
    def n_rows(self, n: int):
        self.desc.n_rows = n


def dense_segment(k: torch.Tensor, v: torch.Tensor, n_rows: Optional[int] = None,
                  idx: Optional[torch.Tensor] = None) -> Segment:
    """k, v [B, Hkv, row_stride, D] (contiguous); rows 0..n_rows-1 live."""
    assert k.is_contiguous() and v.is_contiguous() and k.shape == v.shape and k.dtype == v.dtype
    stride = k.shape[2]
    d = uc_segment(kind=UC_SEG_DENSE, dtype=TORCH_DT[k.dtype],
                   n_rows=stride if n_rows is None else n_rows, row_stride=stride,
                   k=k.data_ptr(), v=v.data_ptr(), idx=_ptr(idx))
    return Segment(d, {"k": k, "v": v, "idx": idx})


def packed_layout(BH: int, N: int, D: int, G: int, head_bits: Sequence[int]):
    """Back-to-back per-head code offsets (16-byte aligned) and total bytes."""
    n_full = G * (N // G)
    off, pos = [], 0
    for b in head_bits:
        off.append(pos)
        pos += (n_full * D * int(b) // 8 + 15) // 16 * 16
    return off, pos


def packed_storage(B: int, Hkv: int, N: int, D: int, dtype: torch.dtype, device="cuda") -> dict:
    """Flat buffers that hold a packed segment of N rows in any uniform
    configuration (codes up to 8 bits, groups down to 8 rows), for
    packed_segment(..., storage=...)."""
    BH = B * Hkv
    return {"codes_k": torch.empty(max(BH * N * D, 16), dtype=torch.uint8, device=device),
            "codes_v": torch.empty(max(BH * N * D, 16), dtype=torch.uint8, device=device),
            "scale_k": torch.empty(BH * (N // 8) * D, dtype=torch.float32, device=device),
            "min_k": torch.empty(BH * (N // 8) * D, dtype=torch.float32, device=device),
            "scale_v": torch.empty(BH * N * (D // 8), dtype=torch.float32, device=device),
            "min_v": torch.empty(BH * N * (D // 8), dtype=torch.float32, device=device),
            "tail_k": torch.empty(BH * 127 * D, dtype=dtype, device=device),
            "tail_v": torch.empty(BH * 127 * D, dtype=dtype, device=device)}


def packed_segment(B: int, Hkv: int, N: int, D: int, G: int, dtype: torch.dtype,
                   bits: int = 4, head_bits: Optional[Sequence[int]] = None,
                   device="cuda", capacity: int = 0, zero: bool = True,
                   storage: Optional[dict] = None) -> Segment:
    """Allocate the buffers of a packed segment of N rows (to be filled by
    uc_quantize_segment).  head_bits: optional per-(b, h_kv) code widths.
    capacity > 0: room for that many rows per head (a segment that grows by
    uc_stream_append; strides follow the capacity).  zero=False leaves the
    buffers uninitialised (for a segment that uc_quantize_segment fills
    whole before anything reads it).  storage: buffers from packed_storage
    to lay the segment out in instead of allocating (uniform widths, no
    capacity; contents left as they are)."""
    def take(name, shape, dt):
        if storage is None:
            return (torch.zeros if zero else torch.empty)(*shape, dtype=dt, device=device)
        return storage[name][:math.prod(shape)].view(*shape)
    BH = B * Hkv
    n_full = G * (N // G)
    tail = N - n_full
    cap_full = G * (capacity // G) if capacity else n_full
    tail_rows = G if capacity else tail
    t = {}
    if head_bits is not None:
        off, total = packed_layout(BH, cap_full, D, G, head_bits)
        t["head_bits"] = torch.tensor(list(head_bits), dtype=torch.uint8, device=device)
        t["code_off"] = torch.tensor(off, dtype=torch.int64, device=device)
    else:
        total = BH * cap_full * D * bits // 8
    assert storage is None or (head_bits is None and not capacity)
    shapes = {"codes_k": (max(total, 16),), "codes_v": (max(total, 16),),
              "scale_k": (B, Hkv, cap_full // G, D), "min_k": (B, Hkv, cap_full // G, D),
              "scale_v": (B, Hkv, cap_full, D // G), "min_v": (B, Hkv, cap_full, D // G),
              "tail_k": (B, Hkv, tail_rows, D), "tail_v": (B, Hkv, tail_rows, D)}
    for name, shp in shapes.items():
        dt = torch.uint8 if name.startswith("codes") else dtype if name.startswith("tail") \
            else torch.float32
        t[name] = take(name, shp, dt)
    d = uc_segment(kind=UC_SEG_PACKED, dtype=TORCH_DT[dtype], n_rows=N, row_stride=capacity,
                   group=G, bits=bits if head_bits is None else int(max(head_bits)),
                   head_bits=_ptr(t.get("head_bits")), code_off=_ptr(t.get("code_off")),
                   codes_bytes=total, codes_k=t["codes_k"].data_ptr(),
                   codes_v=t["codes_v"].data_ptr(), scale_k=t["scale_k"].data_ptr(),
                   min_k=t["min_k"].data_ptr(), scale_v=t["scale_v"].data_ptr(),
                   min_v=t["min_v"].data_ptr(),
                   tail_k=t["tail_k"].data_ptr() if tail_rows else None,
                   tail_v=t["tail_v"].data_ptr() if tail_rows else None)
    return Segment(d, t)


def _seg_array(segs: Sequence[Segment]):
    arr = (uc_segment * len(segs))()
    for i, s in enumerate(segs):
        arr[i] = s.desc
    return arr


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---- the C ABI, one function per entry point -------------------------------

def uc_attend_workspace_size(shape: uc_shape, segs: Sequence[Segment], q_dt: int, M: int) -> int:
    return int(lib.uc_attend_workspace_size(ctypes.byref(shape), _seg_array(segs), len(segs),
                                            q_dt, M))


def uc_attend_mixed(shape: uc_shape, segs: Sequence[Segment], q: torch.Tensor, M: int,
                    sm_scale: float, o: torch.Tensor, lse: Optional[torch.Tensor] = None,
                    seg_lse: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                    stream=None):
    arr = _seg_array(segs)
    q_dt = TORCH_DT[q.dtype]
    if ws is None:
        ws = _ws(lib.uc_attend_workspace_size(ctypes.byref(shape), arr, len(segs), q_dt, M),
                 q.device)
    _check(lib.uc_attend_mixed(ctypes.byref(shape), arr, len(segs), q.data_ptr(), q_dt, M,
                               ctypes.c_float(sm_scale), o.data_ptr(), _ptr(lse), _ptr(seg_lse),
                               ws.data_ptr(), ws.numel(), _stream(stream)), "uc_attend_mixed")
    return o


class AttendPlan:
    """An execution plan over a frozen layout (uc_plan_create): the segments
    are validated once and every call passes only pointers.  segs[tail] is
    the dense segment decode steps append to (its Segment's n_rows is kept
    in step with the plan); tail=None freezes every segment, and attend()
    then reuses its workspace preparation across calls (see
    uc_plan_attend).  Pointers may be given as tensors or as raw device
    addresses (ints); the stream is the current one at creation unless a
    call names another."""

    def __init__(self, shape: uc_shape, segs: Sequence[Segment], tail: Optional[int],
                 q_dtype: torch.dtype,
                 M: int, sm_scale: float, ws: Optional[torch.Tensor] = None, stream=None,
                 device="cuda"):
        h = ctypes.c_void_p()
        tail = -1 if tail is None else tail
        _check(lib.uc_plan_create(ctypes.byref(shape), _seg_array(segs), len(segs), tail,
                                  TORCH_DT[q_dtype], M, ctypes.c_float(sm_scale),
                                  ctypes.byref(h)), "uc_plan_create")
        self._h = h
        self.segs, self.tail = segs, tail
        need = int(lib.uc_plan_workspace_size(h))
        if ws is None:
            ws = _ws(need, device)
        assert ws.numel() >= need, f"workspace {ws.numel()} < {need} bytes"
        self.ws = ws
        self._ws_ptr, self._ws_n = ws.data_ptr(), ws.numel()
        self._stream = _stream(stream)
        self._fn = lib.uc_plan_attend_append

    @property
    def tail_rows(self) -> int:
        return int(lib.uc_plan_tail_rows(self._h))

    def attend_append(self, k_new, v_new, n_new: int, q, o, lse=None, stream=None):
        """One decode step: k_new / v_new [B, Hkv, n_new, D] join the tail and
        q [B, Hq, M, D] attends over every segment into o (and lse)."""
        a = [t if t is None or isinstance(t, int) else t.data_ptr()
             for t in (k_new, v_new, q, o, lse)]
        _check(self._fn(self._h, a[0], a[1], n_new, a[2], a[3], a[4], self._ws_ptr, self._ws_n,
                        self._stream if stream is None else _stream(stream)),
               "uc_plan_attend_append")
        self.segs[self.tail].n_rows += n_new
        return o

    def attend(self, q, o, lse=None, seg_lse=None, stream=None):
        """Attention of q [B, Hq, M, D] over the plan's segments into o (and
        lse, seg_lse)."""
        a = [t if t is None or isinstance(t, int) else t.data_ptr() for t in (q, o, lse, seg_lse)]
        _check(lib.uc_plan_attend(self._h, a[0], a[1], a[2], a[3], self._ws_ptr, self._ws_n,
                                  self._stream if stream is None else _stream(stream)),
               "uc_plan_attend")
        return o

    def invalidate(self):
        """The segments' contents changed: prepare the workspace again."""
        _check(lib.uc_plan_invalidate(self._h), "uc_plan_invalidate")

    def close(self):
        if self._h:
            lib.uc_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


UC_SCRATCH_BYTES = 16 << 20


def uc_attend_mixed_noalloc(shape: uc_shape, segs: Sequence[Segment], q: torch.Tensor, M: int,
                            sm_scale: float, o: torch.Tensor, lse: Optional[torch.Tensor] = None,
                            seg_lse: Optional[torch.Tensor] = None, stream=None):
    """uc_attend_mixed with the library's static scratch array as workspace
    (no device allocation by the library or here)."""
    arr = _seg_array(segs)
    _check(lib.uc_attend_mixed_noalloc(ctypes.byref(shape), arr, len(segs), q.data_ptr(),
                                       TORCH_DT[q.dtype], M, ctypes.c_float(sm_scale),
                                       o.data_ptr(), _ptr(lse), _ptr(seg_lse), _stream(stream)),
           "uc_attend_mixed_noalloc")
    return o


def uc_score_workspace_size(shape: uc_shape, segs: Sequence[Segment], W: int) -> int:
    return int(lib.uc_score_workspace_size(ctypes.byref(shape), _seg_array(segs), len(segs), W))


def uc_score_importance(shape: uc_shape, segs: Sequence[Segment], q_obs: torch.Tensor, W: int,
                        sm_scale: float, scores_out: Sequence[Optional[torch.Tensor]],
                        mass_out: Optional[torch.Tensor] = None,
                        ws: Optional[torch.Tensor] = None, stream=None):
    arr = _seg_array(segs)
    if ws is None:
        ws = _ws(lib.uc_score_workspace_size(ctypes.byref(shape), arr, len(segs), W),
                 q_obs.device)
    ptrs = (ctypes.c_void_p * len(segs))(*[_ptr(t) for t in scores_out])
    _check(lib.uc_score_importance(ctypes.byref(shape), arr, len(segs), q_obs.data_ptr(),
                                   TORCH_DT[q_obs.dtype], W, ctypes.c_float(sm_scale),
                                   ctypes.cast(ptrs, ctypes.c_void_p), _ptr(mass_out),
                                   ws.data_ptr(), ws.numel(), _stream(stream)),
           "uc_score_importance")


def uc_score_columns(shape: uc_shape, segs: Sequence[Segment], q_obs: torch.Tensor, W: int,
                     sm_scale: float, row_lse, lse_ld: int,
                     scores_out: Sequence[Optional[torch.Tensor]],
                     mass_out: Optional[torch.Tensor] = None,
                     ws: Optional[torch.Tensor] = None, stream=None, q_ld: Optional[int] = None):
    """uc_score_importance with the row log-sum-exps given: row_lse is a
    float tensor (or a raw device address) whose element (b*Hq + h)*lse_ld + w
    is observation row (b, h, w)'s normaliser.  q_obs [B, Hq, W, D], or with
    q_ld the window starting at q_obs's first element with q_ld rows between
    query heads (q_obs then may be the whole [B, Hq, M, D] block and W its
    last rows: pass q_obs[:, :, M - W:] as a view)."""
    arr = _seg_array(segs)
    if ws is None:
        ws = _ws(lib.uc_score_workspace_size(ctypes.byref(shape), arr, len(segs), W),
                 q_obs.device)
    ptrs = (ctypes.c_void_p * len(segs))(*[_ptr(t) for t in scores_out])
    lp = row_lse if isinstance(row_lse, int) else row_lse.data_ptr()
    _check(lib.uc_score_columns(ctypes.byref(shape), arr, len(segs), q_obs.data_ptr(),
                                W if q_ld is None else q_ld, TORCH_DT[q_obs.dtype], W,
                                ctypes.c_float(sm_scale), lp, lse_ld,
                                ctypes.cast(ptrs, ctypes.c_void_p), _ptr(mass_out),
                                ws.data_ptr(), ws.numel(), _stream(stream)),
           "uc_score_columns")


def uc_select_keep(scores: torch.Tensor, k: int, n_recent: int, keep_idx: torch.Tensor,
                   k_src: Optional[torch.Tensor] = None, v_src: Optional[torch.Tensor] = None,
                   k_dst: Optional[torch.Tensor] = None, v_dst: Optional[torch.Tensor] = None,
                   stream=None):
    """scores [BH, N] -> keep_idx [BH, k]; optional gather of [BH, N, D] rows."""
    BH, N = scores.shape[0], scores.shape[-1]
    dt = TORCH_DT[k_src.dtype] if k_src is not None else UC_BF16
    D = k_src.shape[-1] if k_src is not None else 128
    ws = _ws(lib.uc_select_workspace_size(BH, N), scores.device)
    _check(lib.uc_select_keep(scores.data_ptr(), BH, N, k, n_recent, keep_idx.data_ptr(),
                              _ptr(k_src), _ptr(v_src), _ptr(k_dst), _ptr(v_dst), dt, D,
                              ws.data_ptr(), ws.numel(), _stream(stream)), "uc_select_keep")
    return keep_idx


def uc_evict_step(shape: uc_shape, scores, cur: Segment, k_dev, out: Segment, stream=None):
    """Keep the best k = *k_dev rows of cur (scores [B*Hkv, cur.n_rows]) in
    out, composing logical indices; k >= cur.n_rows writes nothing.  scores
    and k_dev: tensors or raw device addresses."""
    sp = scores if isinstance(scores, int) else scores.data_ptr()
    kp = k_dev if isinstance(k_dev, int) else k_dev.data_ptr()
    _check(lib.uc_evict_step(ctypes.byref(shape), sp, ctypes.byref(cur.desc), kp,
                             ctypes.byref(out.desc), _stream(stream)), "uc_evict_step")


def uc_quantize_segment(shape: uc_shape, k: torch.Tensor, v: torch.Tensor, N: int,
                        out: Segment, stream=None):
    _check(lib.uc_quantize_segment(ctypes.byref(shape), k.data_ptr(), v.data_ptr(),
                                   TORCH_DT[k.dtype], N, ctypes.byref(out.desc),
                                   _stream(stream)), "uc_quantize_segment")


def _batch_arrays(reqs: Sequence[Sequence[Segment]]):
    arrs = [_seg_array(r) for r in reqs]
    ptrs = (ctypes.c_void_p * len(reqs))(*[ctypes.cast(a, ctypes.c_void_p) for a in arrs])
    counts = (ctypes.c_int * len(reqs))(*[len(r) for r in reqs])
    return arrs, ptrs, counts


def uc_attend_batch_workspace_size(shape: uc_shape, reqs: Sequence[Sequence[Segment]], q_dt: int,
                                   M: int) -> int:
    arrs, ptrs, counts = _batch_arrays(reqs)
    return int(lib.uc_attend_batch_workspace_size(ctypes.byref(shape), ptrs, counts, q_dt, M))


def uc_attend_batch(shape: uc_shape, reqs: Sequence[Sequence[Segment]], q: torch.Tensor, M: int,
                    sm_scale: float, o: torch.Tensor, lse: Optional[torch.Tensor] = None,
                    ws: Optional[torch.Tensor] = None, stream=None):
    """Requests of different segment layouts (each a list of one-request
    segments) attended in one call; q / o / lse as for len(reqs) batch
    elements."""
    arrs, ptrs, counts = _batch_arrays(reqs)
    if ws is None:
        ws = _ws(lib.uc_attend_batch_workspace_size(ctypes.byref(shape), ptrs, counts,
                                                    TORCH_DT[q.dtype], M), q.device)
    _check(lib.uc_attend_batch(ctypes.byref(shape), ptrs, counts, q.data_ptr(), TORCH_DT[q.dtype],
                               M, ctypes.c_float(sm_scale), o.data_ptr(), _ptr(lse),
                               ws.data_ptr(), ws.numel(), _stream(stream)), "uc_attend_batch")


def uc_dequantize_segment(shape: uc_shape, seg: Segment, k_out: torch.Tensor,
                          v_out: torch.Tensor, stream=None):
    """Packed segment -> dense rows [B, Hkv, n_rows, D] in its dtype."""
    _check(lib.uc_dequantize_segment(ctypes.byref(shape), ctypes.byref(seg.desc), k_out.data_ptr(),
                                     v_out.data_ptr(), _stream(stream)), "uc_dequantize_segment")


def uc_stream_append(shape: uc_shape, seg: Segment, k_new: torch.Tensor, v_new: torch.Tensor,
                     n_new: int, stream=None):
    """Append n_new rows [B, Hkv, n_new, D] to a packed segment with a row
    capacity; full row groups of the tail are quantised.  Advances
    seg.n_rows."""
    _check(lib.uc_stream_append(ctypes.byref(shape), ctypes.byref(seg.desc), k_new.data_ptr(),
                                v_new.data_ptr(), n_new, _stream(stream)), "uc_stream_append")
    seg.n_rows = seg.n_rows + n_new


def uc_topk_mass(scores: torch.Tensor, k: int, frac_out: torch.Tensor, stream=None):
    """scores [BH, N] -> frac_out [BH]: share of each row's sum on its k
    largest entries."""
    BH, N = scores.shape[0], scores.shape[-1]
    ws = _ws(lib.uc_topk_mass_workspace_size(BH, k), scores.device)
    _check(lib.uc_topk_mass(scores.data_ptr(), BH, N, k, frac_out.data_ptr(), ws.data_ptr(),
                            ws.numel(), _stream(stream)), "uc_topk_mass")
    return frac_out


def uc_compose_index(outer: torch.Tensor, inner: torch.Tensor, out: torch.Tensor, stream=None):
    """out[bh, j] = outer[bh, inner[bh, j]] (int32 tensors [BH, n_outer],
    [BH, k], [BH, k])."""
    BH, n_outer = outer.shape[0], outer.shape[-1]
    k = inner.shape[-1]
    _check(lib.uc_compose_index(outer.data_ptr(), n_outer, inner.data_ptr(), BH, k,
                                out.data_ptr(), _stream(stream)), "uc_compose_index")
    return out


def uc_quant_config(budget: float, N: int, D: int, dt: int, n_heads: int, first: int = 0):
    """(index, bits, group) of the most faithful configuration at or after
    `first` that fits the budget (the last one if none does)."""
    bits, group = ctypes.c_int(), ctypes.c_int()
    i = int(lib.uc_quant_config(float(budget), N, D, dt, n_heads, first, ctypes.byref(bits),
                                ctypes.byref(group)))
    if i < 0:
        raise UcError(UC_E_INVALID, "uc_quant_config", "invalid arguments")
    return i, bits.value, group.value


def uc_append_rows(shape: uc_shape, k_new: torch.Tensor, v_new: torch.Tensor, n_new: int,
                   seg: Segment, pos: int, stream=None):
    _check(lib.uc_append_rows(ctypes.byref(shape), k_new.data_ptr(), v_new.data_ptr(), n_new,
                              ctypes.byref(seg.desc), pos, _stream(stream)), "uc_append_rows")


def uc_attend_append(shape: uc_shape, segs: Sequence[Segment], tail: int, k_new: torch.Tensor,
                     v_new: torch.Tensor, n_new: int, q: torch.Tensor, M: int, sm_scale: float,
                     o: torch.Tensor, lse: Optional[torch.Tensor] = None,
                     seg_lse: Optional[torch.Tensor] = None, ws: Optional[torch.Tensor] = None,
                     stream=None):
    """One decode step: k_new / v_new join segs[tail] and the queries attend
    over every segment; segs[tail].n_rows is raised by n_new on success."""
    arr = _seg_array(segs)
    q_dt = TORCH_DT[q.dtype]
    if ws is None:  # sized for the segments as they stand after the append
        arr[tail].n_rows += n_new
        ws = _ws(lib.uc_attend_workspace_size(ctypes.byref(shape), arr, len(segs), q_dt, M),
                 q.device)
        arr[tail].n_rows -= n_new
    _check(lib.uc_attend_append(ctypes.byref(shape), arr, len(segs), tail, _ptr(k_new),
                                _ptr(v_new), n_new, q.data_ptr(), q_dt, M,
                                ctypes.c_float(sm_scale), o.data_ptr(), _ptr(lse), _ptr(seg_lse),
                                ws.data_ptr(), ws.numel(), _stream(stream)), "uc_attend_append")
    segs[tail].n_rows += n_new
    return o


def uc_segment_mass(shape: uc_shape, M: int, n_segs: int, lse: torch.Tensor,
                    seg_lse: torch.Tensor, mass_out: torch.Tensor, stream=None):
    _check(lib.uc_segment_mass(ctypes.byref(shape), M, n_segs, lse.data_ptr(),
                               seg_lse.data_ptr(), mass_out.data_ptr(), _stream(stream)),
           "uc_segment_mass")


def uc_dense_bytes(rows: int, D: int, dt: int) -> int:
    return int(lib.uc_dense_bytes(rows, D, dt))


def uc_evicted_bytes(rows: int, D: int, dt: int) -> int:
    return int(lib.uc_evicted_bytes(rows, D, dt))


def uc_packed_bytes(N: int, D: int, G: int, bits: int, dt: int) -> int:
    return int(lib.uc_packed_bytes(N, D, G, bits, dt))


def uc_evict_rows_for_budget(budget: float, fixed: float, N: int, D: int, dt: int) -> int:
    return int(lib.uc_evict_rows_for_budget(budget, fixed, N, D, dt))


def uc_assign_bits(mass: Sequence[float], N: int, D: int, G: int, dt: int, budget: float,
                   fixed: float) -> List[int]:
    import numpy as np
    m = np.ascontiguousarray(mass, np.float32)
    out = np.zeros(m.shape[0], np.uint8)
    _check(lib.uc_assign_bits(m.shape[0], m.ctypes.data, N, D, G, dt, budget, fixed,
                              out.ctypes.data), "uc_assign_bits")
    return [int(x) for x in out]


def uc_type_budget(mass: Sequence[float], b_prev: Sequence[float], B_total: float):
    import numpy as np
    m = np.ascontiguousarray(mass, np.float64)
    bp = np.ascontiguousarray(b_prev, np.float64)
    out = np.zeros(m.shape[0])
    _check(lib.uc_type_budget(m.shape[0], m.ctypes.data, bp.ctypes.data, B_total,
                              out.ctypes.data), "uc_type_budget")
    return out


def uc_retention_next(rho: float, rho_init: float, rho_min: float, M_c: float,
                      M_0: float) -> float:
    return float(lib.uc_retention_next(rho, rho_init, rho_min, M_c, M_0))


def budget_state_tensor(device="cuda") -> torch.Tensor:
    """Zero-filled device storage for one uc_budget_state (before the first
    boundary)."""
    return torch.zeros(ctypes.sizeof(uc_budget_state), dtype=torch.uint8, device=device)


def budget_state_read(state: torch.Tensor, host: Optional[torch.Tensor] = None,
                      stream=None) -> uc_budget_state:
    """Copy a device uc_budget_state to the host (waits for the stream);
    host: an optional pinned uint8 buffer of the same size to copy through."""
    if host is None:
        return uc_budget_state.from_buffer_copy(bytes(state.cpu().numpy()))
    s = torch.cuda.current_stream() if stream is None else stream
    with torch.cuda.stream(s):
        host.copy_(state, non_blocking=True)
    s.synchronize()
    return uc_budget_state.from_buffer_copy(host.numpy().tobytes())


def uc_budget_step(params: uc_budget_params, mass: torch.Tensor, n_steps: int,
                   state: torch.Tensor, stream=None) -> None:
    """mass: device float [n_steps, Hkv, n_segs] (contiguous)."""
    assert mass.dtype == torch.float32 and mass.is_contiguous()
    assert mass.numel() == n_steps * params.Hkv * params.n_segs
    assert state.numel() == ctypes.sizeof(uc_budget_state)
    _check(lib.uc_budget_step(ctypes.byref(params), mass.data_ptr(), n_steps, state.data_ptr(),
                              _stream(stream)), "uc_budget_step")


def uc_calibrate_policy(frac: torch.Tensor, threshold: float, conc_out: torch.Tensor,
                        evict_out: torch.Tensor, stream=None) -> None:
    """frac: device float [rows, n_types]; conc_out double [n_types], evict_out
    int32 [n_types]."""
    rows, n_types = frac.shape
    assert frac.dtype == torch.float32 and frac.is_contiguous()
    assert conc_out.dtype == torch.float64 and evict_out.dtype == torch.int32
    assert conc_out.numel() == evict_out.numel() == n_types
    _check(lib.uc_calibrate_policy(frac.data_ptr(), rows, n_types, threshold, conc_out.data_ptr(),
                                   evict_out.data_ptr(), _stream(stream)), "uc_calibrate_policy")


def uc_status_string(s: int) -> str:
    return lib.uc_status_string(s).decode()


def uc_last_error() -> str:
    return lib.uc_last_error().decode()


def uc_last_kernel() -> str:
    """Main kernel of this thread's last attention or scoring launch."""
    return lib.uc_last_kernel().decode()


def uc_set_kernel_events(start, stop) -> None:
    """Bracket the attention kernel of the next attention call (uc_attend_mixed,
    uc_attend_append, uc_attend_batch) on this thread with two events (torch.cuda.Event objects that have been recorded
    once, so that their handles exist; or raw hipEvent_t values; or None)."""
    def handle(ev):
        if ev is None:
            return None
        return ctypes.c_void_p(ev.cuda_event if hasattr(ev, "cuda_event") else int(ev))
    _check(lib.uc_set_kernel_events(handle(start), handle(stop)), "uc_set_kernel_events")


UC_PROBE_LINES = 0
UC_PROBE_OPERAND = 1


def uc_read_probe_unit() -> int:
    """Byte granularity of uc_read_probe's buffer (4 KB per workgroup)."""
    return lib.uc_read_probe_unit()


def uc_read_probe_sink_bytes() -> int:
    return lib.uc_read_probe_sink_bytes()


def uc_read_probe(buf: torch.Tensor, pattern: int, sink: torch.Tensor, stream=None) -> None:
    """Stream buf once (instrumentation; see the header): whole-line loads
    (UC_PROBE_LINES) or the matrix-core operand pattern (UC_PROBE_OPERAND);
    sink receives each wave's XOR of the words it read."""
    _check(lib.uc_read_probe(_ptr(buf), buf.numel() * buf.element_size(), pattern, _ptr(sink),
                             _stream(stream)), "uc_read_probe")


def uc_set_path(path: int) -> int:
    """UC_PATH_AUTO (matrix cores where eligible) or UC_PATH_VALU; returns the
    previous setting."""
    return int(lib.uc_set_path(path))
