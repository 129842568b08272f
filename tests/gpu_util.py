"""Helpers shared by the GPU parity tests: moving generator bytes to the GPU,
building segments from oracle outputs, and the numeric bars."""
import math

import numpy as np
import torch

import oracle as ref
import paper_2609_32831_amd as uc
import workloads as gen

TORCH = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}
UCDT = {"f32": uc.UC_F32, "f16": uc.UC_F16, "bf16": uc.UC_BF16}

# attention bar: fp32 accumulation over bf16 I/O, output compared in fp32
ATOL_MAX = 2e-3
REL_L2 = 1e-3


def dev(a: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    """Stored numpy bytes (bf16 as uint16) -> device tensor of that dtype."""
    a = np.ascontiguousarray(a)
    if dtype == "bf16":
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(a).to(device)


def host_bytes(t: torch.Tensor) -> np.ndarray:
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def rand_rows(seed: int, BH: int, N: int, D: int, dtype: str, scale=1.0, outliers=()):
    x = gen.normal(gen.stream(seed, BH, N, D), 0, BH * N * D).reshape(BH, N, D) * scale
    for c in outliers:
        x[:, :, c] *= 8.0
    return gen.round_to(x, dtype)


def packed_from_oracle(B, Hkv, N, D, G, dtype, pk, device="cuda", per_head=False):
    """A GPU packed segment holding exactly the oracle's codes/scales/tail."""
    bits = [int(b) for b in pk["bits"]]
    seg = uc.packed_segment(B, Hkv, N, D, G, TORCH[dtype], bits=bits[0],
                            head_bits=bits if per_head else None, device=device)
    t = seg.t
    n = pk["codes_k"].shape[0]
    t["codes_k"][:n].copy_(torch.from_numpy(pk["codes_k"]))
    t["codes_v"][:n].copy_(torch.from_numpy(pk["codes_v"]))
    for name in ("scale_k", "min_k", "scale_v", "min_v"):
        t[name].copy_(torch.from_numpy(pk[name]).reshape(t[name].shape))
    if pk["tail_k"].shape[1] > 0:
        t["tail_k"].copy_(dev(pk["tail_k"], dtype).reshape(t["tail_k"].shape))
        t["tail_v"].copy_(dev(pk["tail_v"], dtype).reshape(t["tail_v"].shape))
    return seg


def check_attention(o_gpu: np.ndarray, o_ref: np.ndarray, what=""):
    o_gpu = np.asarray(o_gpu, np.float64)
    err = np.abs(o_gpu - o_ref)
    rel = np.linalg.norm(o_gpu - o_ref) / max(np.linalg.norm(o_ref), 1e-30)
    assert np.all(np.isfinite(o_gpu)), what
    assert err.max() <= ATOL_MAX, f"{what}: max-abs {err.max():.3g} > {ATOL_MAX}"
    assert rel <= REL_L2, f"{what}: rel-L2 {rel:.3g} > {REL_L2}"
    return err.max(), rel


def sm_scale(D: int) -> float:
    return float(np.float32(1.0 / math.sqrt(D)))
