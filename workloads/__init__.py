"""Seeded synthetic workloads for mixed-policy KV attention.

The paper measures on BAGEL-7B-MoT contexts (understanding, text-to-image,
image editing; Sec. 4.1, Sec. 4.4).  Neither the model nor its benchmarks are
available, so every input here is synthetic: seeded Gaussian K/V/Q with the
head shapes of a 7B model (28 query heads, 4 KV heads, head dim 128), 4096
tokens per image, and outlier key channels.  This module holds only input
recipes and the raw parameters of each workload; it contains none of the
method's arithmetic (no scoring, selection, quantization, budgets or
attention).  Budget-derived quantities (rows kept, bit widths) are computed
by the oracle and by the library's host helpers independently.

Random numbers come from ``libucgen.so`` (counter-based SplitMix64 +
Box-Muller, see ``ucgen.c``), so each tensor is a pure function of
(seed, config, tensor, segment, row-block, element index) and any slice can be
generated without the rest.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Tuple

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.environ.get("UCGEN_LIB") or os.path.join(HERE, "libucgen.so")  # override: sanitized builds
_lib = None

DTYPE_CODE = {"f32": 0, "f16": 1, "bf16": 2}
NP_STORAGE = {"f32": np.float32, "f16": np.float16, "bf16": np.uint16}
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2}

# tensor ids used in stream keys
T_K, T_V, T_QOBS, T_QDEC, T_KDEC, T_VDEC, T_QPRE = 1, 2, 3, 4, 5, 6, 7
T_OUTLIER, T_UDIR, T_TAU, T_DRIFT_Q, T_DRIFT_K, T_SELFDIR = 8, 9, 10, 11, 12, 13


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = ctypes.CDLL(_LIB_PATH)
        u64, i64, i32, dp, vp = (ctypes.c_uint64, ctypes.c_int64, ctypes.c_int,
                                 ctypes.POINTER(ctypes.c_double), ctypes.c_void_p)
        L.ucgen_raw.restype = u64
        L.ucgen_raw.argtypes = [u64, u64]
        L.ucgen_uniform.restype = ctypes.c_double
        L.ucgen_uniform.argtypes = [u64, u64]
        L.ucgen_stream.restype = u64
        L.ucgen_stream.argtypes = [u64, ctypes.POINTER(u64), i32]
        L.ucgen_normal_at.restype = ctypes.c_double
        L.ucgen_normal_at.argtypes = [u64, u64]
        L.ucgen_normal.restype = None
        L.ucgen_normal.argtypes = [u64, u64, i64, vp]
        L.ucgen_uniform_fill.restype = None
        L.ucgen_uniform_fill.argtypes = [u64, u64, i64, vp]
        L.ucgen_round.restype = None
        L.ucgen_round.argtypes = [vp, i64, i32, vp]
        L.ucgen_rows.restype = None
        L.ucgen_rows.argtypes = [u64, i64, i32, i64, i32, i64, vp, vp, vp, i32, vp, vp]
        L.ucgen_drift.restype = None
        L.ucgen_drift.argtypes = [u64, u64, ctypes.c_double, i64, i64, vp, i32, vp]
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def stream(base: int, *ids: int) -> int:
    arr = (ctypes.c_uint64 * len(ids))(*[int(i) & 0xFFFFFFFFFFFFFFFF for i in ids])
    return int(lib().ucgen_stream(ctypes.c_uint64(base), arr, len(ids)))


def normal(seed: int, start: int, n: int) -> np.ndarray:
    out = np.empty(n, np.float64)
    lib().ucgen_normal(seed, start, n, out.ctypes.data)
    return out


def uniform(seed: int, start: int, n: int) -> np.ndarray:
    out = np.empty(n, np.float64)
    lib().ucgen_uniform_fill(seed, start, n, out.ctypes.data)
    return out


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 -> storage dtype (fp32 RNE, then bf16/fp16 RNE); bf16 as uint16 bits."""
    x = np.ascontiguousarray(x, np.float64)
    out = np.empty(x.shape, NP_STORAGE[dtype])
    lib().ucgen_round(x.ctypes.data, x.size, DTYPE_CODE[dtype], out.ctypes.data)
    return out


# --------------------------------------------------------------------------
# Workload descriptions


@dataclass(frozen=True)
class SegSpec:
    """One typed segment of the context (Sec. 3.1).

    policy: "keep"    candidate kept at its stored precision,
            "evict"   eviction-managed (top-k by importance),
            "quant"   quantization-managed (group-wise low-bit),
            "protect" protected segment (decode-time tail; excluded from budget).
    keep_ratio: eviction by a fixed fraction of the segment (else the segment's
            rows follow from the shared storage budget).
    """
    name: str
    n: int
    policy: str
    dtype: str
    keep_ratio: Optional[float] = None
    bits: Optional[int] = None          # fixed code width, None = per-head by budget
    group: Optional[int] = None
    heavy_tail: bool = False            # Student-t heavy hitters on its keys
    self_align: float = 0.0             # keys += self_align * (the head's self direction)


@dataclass(frozen=True)
class Workload:
    name: str
    recipe_id: int                      # first id of every input stream of the workload
    B: int
    Hq: int
    Hkv: int
    D: int
    q_dtype: str
    segments: Tuple[SegSpec, ...]
    W: int                       # observation queries per query head for scoring
    mode: str                    # "decode" or "prefill"
    steps: int                   # decode steps or denoising timesteps
    M: int                       # queries per step and query head
    budget_ratio: Optional[float] = None   # overall compression target (x)
    n_outlier: int = 0           # outlier key channels per KV head
    outlier_scale: float = 1.0
    drift_sigma: float = 0.0
    rescore_every: int = 0
    tail_capacity: int = 0       # protected decode tail rows (decode append)
    stream_tail: bool = False    # decode rows join the quantised segment's residual tail
    # dynamic budget (Sec. 3.3 Eq. 1-3): timesteps per statistics chunk, the
    # initial and minimum retention ratios, and the observation rows per query
    # head that re-score an evicting type at a chunk boundary
    chunk_steps: int = 0
    rho_init: float = 0.0
    rho_min: float = 0.0
    obs_window: int = 0
    # prefill queries of timestep t are pulled along their KV head's self
    # direction by self_pull * min(1, t / self_ramp) (attention moving to the
    # current latent's own tokens as denoising proceeds)
    self_pull: float = 0.0
    self_ramp: int = 1
    # target average compression (1 - stored / original bytes of the cached
    # segments) that the minimum retention ratio is calibrated to
    target_compression: Optional[float] = None
    seed: int = 0
    notes: str = ""

    @property
    def group_size(self) -> int:
        return self.Hq // self.Hkv

    @property
    def n_context(self) -> int:
        return sum(s.n for s in self.segments)


TINY_UNDERSTANDING = Workload(
    name="tiny_understanding", recipe_id=1, B=1, Hq=4, Hkv=1, D=64, q_dtype="f32",
    segments=(SegSpec("text", 64, "keep", "f16"),
              SegSpec("vit", 256, "evict", "f32", keep_ratio=0.2),
              SegSpec("vae", 256, "quant", "f32", bits=4, group=32)),
    W=16, mode="decode", steps=1, M=1, n_outlier=4, outlier_scale=10.0,
    notes="1 layer, batch 1, 4 query heads on 1 KV head, head dim 64, fp32")

UNDERSTANDING_7B = Workload(
    name="understanding_7b", recipe_id=2, B=4, Hq=28, Hkv=4, D=128, q_dtype="bf16",
    segments=(SegSpec("text", 512, "keep", "bf16"),
              SegSpec("vit", 4096, "evict", "bf16")),
    W=32, mode="decode", steps=256, M=1, budget_ratio=5.0,
    n_outlier=2, outlier_scale=8.0, tail_capacity=256,
    notes="512 text + 4096 ViT, 5x budget, 256 decode steps")

IMAGE_EDITING = Workload(
    name="image_editing", recipe_id=3, B=2, Hq=28, Hkv=4, D=128, q_dtype="bf16",
    segments=(SegSpec("text", 1024, "keep", "bf16"),
              SegSpec("vit", 4096, "evict", "bf16", keep_ratio=0.25),
              SegSpec("vae", 4096, "quant", "bf16", bits=4, group=64)),
    W=4096, mode="prefill", steps=25, M=4096, budget_ratio=5.0,
    n_outlier=2, outlier_scale=8.0,
    notes="1024 text + 4096 ViT + 4096 VAE; 4096-query prefill x 25 timesteps")

TEXT_TO_IMAGE = Workload(
    name="text_to_image", recipe_id=4, B=8, Hq=28, Hkv=4, D=128, q_dtype="bf16",
    segments=(SegSpec("text", 768, "keep", "bf16"),
              SegSpec("latent", 4096, "quant", "bf16", bits=None, group=64)),
    W=4096, mode="prefill", steps=50, M=4096, budget_ratio=2.5,
    n_outlier=2, outlier_scale=8.0, drift_sigma=0.05, rescore_every=10,
    notes="768 text + 4096 latent int2/int4 per head, 2.5x; 50 x 4096-query "
          "prefill, rescoring every 10 steps, random-walk drift sigma 0.05")

LONG_CONTEXT_64K = Workload(
    name="long_context_64k", recipe_id=5, B=16, Hq=28, Hkv=4, D=128, q_dtype="bf16",
    segments=(SegSpec("text", 4096, "quant", "bf16", bits=4, group=64),
              SegSpec("vit", 15 * 4096, "evict", "bf16", heavy_tail=True)),
    W=32, mode="decode", steps=512, M=1, budget_ratio=5.0,
    n_outlier=2, outlier_scale=8.0, tail_capacity=512,
    notes="65536-token context (4096 text + 15x4096 ViT), 5x budget, "
          "512 decode steps")

# The editing workload under the dynamic budget: the same inputs (same stream
# ids), the ViT row count and VAE code width set by Eq. 2 at every chunk
# boundary instead of the fixed 25 % / int4 policies.
IMAGE_EDITING_DYNAMIC = Workload(
    **{**IMAGE_EDITING.__dict__,
       "name": "image_editing_dynamic",
       "segments": (SegSpec("text", 1024, "keep", "bf16"),
                    SegSpec("vit", 4096, "evict", "bf16"),
                    SegSpec("vae", 4096, "quant", "bf16", bits=None, group=None),
                    SegSpec("self", 1024, "protect", "bf16", self_align=6.0)),
       "budget_ratio": None, "chunk_steps": 5, "rho_init": 0.30, "rho_min": 0.15,
       "obs_window": 32, "self_pull": 10.0, "self_ramp": 10, "target_compression": 0.75,
       "notes": "editing with Eq. 1-3: chunks of 5 timesteps, rho from 0.30 down to at "
                "least rho_min with the candidate mass, Eq. 2 type budgets; a protected "
                "self segment (the current latent's own tokens) draws attention away "
                "from the cached conditioning as the timesteps advance; rho_min "
                "calibrated to 75 % average compression (the first chunk at rho_init "
                "and the kept text bound what this cache can reach)"})

# The 64k decode workload with a streaming residual tail: each decode step's
# K/V row enters the int4 text segment's bf16 tail, and every 64 rows form a
# new quantised group (no separate protected dense tail).
LONG_CONTEXT_64K_STREAMING = Workload(
    **{**LONG_CONTEXT_64K.__dict__, "name": "long_context_64k_streaming", "tail_capacity": 0,
       "stream_tail": True,
       "notes": "long_context_64k with decode rows streamed into the int4 g64 text segment"})

WORKLOADS = {w.name: w for w in (TINY_UNDERSTANDING, UNDERSTANDING_7B, IMAGE_EDITING,
                                 TEXT_TO_IMAGE, LONG_CONTEXT_64K, IMAGE_EDITING_DYNAMIC,
                                 LONG_CONTEXT_64K_STREAMING)}


def scaled(w: Workload, **kw) -> Workload:
    """A copy of a workload with some fields replaced (smaller parity cases)."""
    d = dict(w.__dict__)
    d.update(kw)
    return Workload(**d)


# --------------------------------------------------------------------------
# Input recipes


def outlier_channels(w: Workload, bh: int) -> np.ndarray:
    """Outlier key channels of KV row-block bh: the n_outlier channels with the
    smallest seeded uniforms (a seeded random choice)."""
    if w.n_outlier == 0:
        return np.zeros(0, np.int64)
    u = uniform(stream(w.seed, w.recipe_id, T_OUTLIER, bh), 0, w.D)
    return np.sort(np.argsort(u, kind="stable")[: w.n_outlier])


def key_channel_scale(w: Workload, bh0: int, nbh: int) -> np.ndarray:
    s = np.ones((nbh, w.D), np.float64)
    for i in range(nbh):
        s[i, outlier_channels(w, bh0 + i)] = w.outlier_scale
    return s


def heavy_dir(w: Workload, bh0: int, nbh: int) -> np.ndarray:
    """Unit direction u per KV row-block for heavy-tailed logits."""
    u = np.empty((nbh, w.D))
    for i in range(nbh):
        z = normal(stream(w.seed, w.recipe_id, T_UDIR, bh0 + i), 0, w.D)
        u[i] = z / np.sqrt(np.sum(z * z))
    return u


def heavy_coef(w: Workload, seg_index: int, bh0: int, nbh: int, row0: int,
               n: int) -> np.ndarray:
    """(sqrt(D)/2) * tau_j with tau_j ~ Student-t(3) = z / sqrt(chi2_3 / 3)."""
    out = np.empty((nbh, n))
    for i in range(nbh):
        z = normal(stream(w.seed, w.recipe_id, T_TAU, seg_index, bh0 + i), 4 * row0, 4 * n)
        z = z.reshape(n, 4)
        chi2 = np.sum(z[:, 1:] ** 2, axis=1)
        out[i] = (math.sqrt(w.D) / 2.0) * z[:, 0] / np.sqrt(chi2 / 3.0)
    return out


def _rows(base: int, bh0: int, nbh: int, n: int, D: int, row0: int, dtype: str,
          chan_scale=None, add_dir=None, row_coef=None, master=False):
    out = np.empty((nbh, n, D), NP_STORAGE[dtype])
    m = np.empty((nbh, n, D), np.float64) if master else None
    cs = None if chan_scale is None else np.ascontiguousarray(chan_scale, np.float64)
    ad = None if add_dir is None else np.ascontiguousarray(add_dir, np.float64)
    rc = None if row_coef is None else np.ascontiguousarray(row_coef, np.float64)
    lib().ucgen_rows(base, bh0, nbh, n, D, row0, _ptr(cs), _ptr(ad), _ptr(rc),
                     DTYPE_CODE[dtype], out.ctypes.data, _ptr(m))
    return (out, m) if master else out


def segment_kv(w: Workload, seg_index: int, which: str, bh0: int = 0,
               nbh: Optional[int] = None, row0: int = 0, n: Optional[int] = None,
               master: bool = False):
    """Stored K or V rows [nbh, n, D] of segment seg_index (pre-compression).

    Keys: N(0,1), outlier channels scaled, plus a heavy-tailed rank-1 term on
    segments marked heavy_tail.  Values: N(0,1)."""
    seg = w.segments[seg_index]
    nbh = w.B * w.Hkv if nbh is None else nbh
    n = seg.n - row0 if n is None else n
    tensor = T_K if which == "k" else T_V
    base = stream(w.seed, w.recipe_id, tensor, seg_index)
    if which == "v":
        return _rows(base, bh0, nbh, n, w.D, row0, seg.dtype, master=master)
    cs = key_channel_scale(w, bh0, nbh)
    ad = rc = None
    if seg.heavy_tail:
        ad = heavy_dir(w, bh0, nbh)
        rc = heavy_coef(w, seg_index, bh0, nbh, row0, n)
    elif seg.self_align:
        ad = seg.self_align * self_dir(w, bh0, nbh)
    return _rows(base, bh0, nbh, n, w.D, row0, seg.dtype, cs, ad, rc, master=master)


def self_dir(w: Workload, bh0: int, nbh: int) -> np.ndarray:
    """Unit direction per KV row-block shared by a self segment's keys and
    the pulled prefill queries of that KV head."""
    u = np.empty((nbh, w.D))
    for i in range(nbh):
        z = normal(stream(w.seed, w.recipe_id, T_SELFDIR, bh0 + i), 0, w.D)
        u[i] = z / np.sqrt(np.sum(z * z))
    return u


def _query_dir(w: Workload, bh0q: int, nbhq: int, tensor: int = 0,
               step: int = 0) -> Optional[np.ndarray]:
    heavy = any(s.heavy_tail for s in w.segments)
    pull = w.self_pull * min(1.0, step / w.self_ramp) if tensor == T_QPRE else 0.0
    if not heavy and pull == 0.0:
        return None
    out = np.zeros((nbhq, w.D))
    for i in range(nbhq):
        bq = bh0q + i
        b, h = divmod(bq, w.Hq)
        bh = b * w.Hkv + h // w.group_size
        if heavy:
            out[i] += 2.0 * heavy_dir(w, bh, 1)[0]
        if pull:
            out[i] += pull * self_dir(w, bh, 1)[0]
    return out


def queries(w: Workload, tensor: int, n: int, row0: int = 0, bh0: int = 0,
            nbh: Optional[int] = None, step: int = 0, master: bool = False):
    """Query rows [nbh, n, D] (row-blocks are (b, h_q)) for a query tensor id:
    T_QOBS observation window, T_QDEC decode steps (row = step),
    T_QPRE prefill block of timestep `step`."""
    nbh = w.B * w.Hq if nbh is None else nbh
    base = stream(w.seed, w.recipe_id, tensor, step)
    return _rows(base, bh0, nbh, n, w.D, row0, w.q_dtype,
                 add_dir=_query_dir(w, bh0, nbh, tensor, step), master=master)


def decode_kv(w: Workload, which: str, row0: int, n: int, bh0: int = 0,
              nbh: Optional[int] = None) -> np.ndarray:
    """New K or V rows produced by decode steps row0..row0+n-1 [nbh, n, D],
    stored in the protected tail (bf16 for the 7B-shaped workloads)."""
    nbh = w.B * w.Hkv if nbh is None else nbh
    tensor = T_KDEC if which == "k" else T_VDEC
    base = stream(w.seed, w.recipe_id, tensor)
    dt = "bf16" if w.q_dtype == "bf16" else w.q_dtype
    cs = key_channel_scale(w, bh0, nbh) if which == "k" else None
    return _rows(base, bh0, nbh, n, w.D, row0, dt, cs)


class Drift:
    """Random walk X_t = X_{t-1} + sigma * eps_t on an fp64 master copy, rounded
    to the storage dtype after every step (text-to-image timesteps).  The
    master holds elements start .. start + size - 1 of the whole tensor (a
    slice drifts exactly as inside the whole tensor)."""

    def __init__(self, w: Workload, tensor: int, master: np.ndarray, dtype: str, start: int = 0):
        self.w, self.tensor, self.dtype, self.start = w, tensor, dtype, start
        self.master = np.ascontiguousarray(master, np.float64)
        self.t = 0

    def step(self) -> np.ndarray:
        self.t += 1
        out = np.empty(self.master.shape, NP_STORAGE[self.dtype])
        base = stream(self.w.seed, self.w.recipe_id, self.tensor)
        lib().ucgen_drift(base, self.t, self.w.drift_sigma, self.start, self.master.size,
                          self.master.ctypes.data, DTYPE_CODE[self.dtype], out.ctypes.data)
        return out


# --------------------------------------------------------------------------
# plain-numpy twin of the generator's core, used only to pin libucgen.so

_G = np.uint64(0x9E3779B97F4A7C15)


def _mix64_np(z: np.ndarray) -> np.ndarray:
    z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
    z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
    return z ^ (z >> np.uint64(31))


def normal_np(seed: int, start: int, n: int) -> np.ndarray:
    with np.errstate(over="ignore"):
        i = np.arange(start, start + n, dtype=np.uint64)
        p = i >> np.uint64(1)
        s = np.uint64(seed)
        u1 = (_mix64_np(s + (np.uint64(2) * p + np.uint64(1)) * _G) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
        u2 = (_mix64_np(s + (np.uint64(2) * p + np.uint64(2)) * _G) >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
    r = np.sqrt(-2.0 * np.log1p(-u1))
    a = 2.0 * np.pi * u2
    return np.where((i & np.uint64(1)) == 0, r * np.cos(a), r * np.sin(a))
