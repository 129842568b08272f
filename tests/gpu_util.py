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


def mixed_case(B, Hq, Hkv, D, dtype, sizes, seed=0, G=64, bits=4, per_head=False):
    """Segments: dense 'text', compacted 'vit' (rows chosen at random, with
    their logical positions), packed 'vae' with tail, dense tail segment with
    spare capacity.  Returns GPU segments and the oracle's logical K/V."""
    n_text, n_vit_full, n_vit_keep, n_pack, n_tail, cap = sizes
    BH = B * Hkv
    segs, kh, vh, seg_id = [], [], [], []
    # text (dense)
    kt = rand_rows(seed + 1, BH, n_text, D, dtype, outliers=(5,))
    vt = rand_rows(seed + 2, BH, n_text, D, dtype)
    segs.append(uc.dense_segment(dev(kt, dtype).reshape(B, Hkv, n_text, D),
                                 dev(vt, dtype).reshape(B, Hkv, n_text, D)))
    kh.append(ref.widen(kt, dtype)); vh.append(ref.widen(vt, dtype))
    # compacted eviction survivors
    kv_full = rand_rows(seed + 3, BH, n_vit_full, D, dtype, outliers=(5,))
    vv_full = rand_rows(seed + 4, BH, n_vit_full, D, dtype)
    rng = np.random.default_rng(seed)
    idx = np.sort(np.stack([rng.choice(n_vit_full, n_vit_keep, replace=False) for _ in range(BH)]), 1)
    kc = np.stack([kv_full[i][idx[i]] for i in range(BH)])
    vc = np.stack([vv_full[i][idx[i]] for i in range(BH)])
    segs.append(uc.dense_segment(dev(kc, dtype).reshape(B, Hkv, n_vit_keep, D),
                                 dev(vc, dtype).reshape(B, Hkv, n_vit_keep, D),
                                 idx=torch.from_numpy(idx.astype(np.int32)).cuda()))
    kh.append(ref.widen(kc, dtype)); vh.append(ref.widen(vc, dtype))
    # packed
    kp = rand_rows(seed + 5, BH, n_pack, D, dtype, 2.0, outliers=(5,))
    vp = rand_rows(seed + 6, BH, n_pack, D, dtype)
    hb = [bits] * BH if not per_head else [4 if (i % 3) else 2 for i in range(BH)]
    pk = ref.quantize(kp, vp, dtype, G, hb)
    segs.append(packed_from_oracle(B, Hkv, n_pack, D, G, dtype, pk, per_head=per_head))
    khp, vhp = ref.dequant(pk, n_pack, D, G, dtype)
    kh.append(khp); vh.append(vhp)
    # dense tail with spare capacity
    ktl = rand_rows(seed + 7, BH, cap, D, dtype)
    vtl = rand_rows(seed + 8, BH, cap, D, dtype)
    segs.append(uc.dense_segment(dev(ktl, dtype).reshape(B, Hkv, cap, D),
                                 dev(vtl, dtype).reshape(B, Hkv, cap, D), n_rows=n_tail))
    kh.append(ref.widen(ktl[:, :n_tail], dtype)); vh.append(ref.widen(vtl[:, :n_tail], dtype))
    for a, n in enumerate([n_text, n_vit_keep, n_pack, n_tail]):
        seg_id += [a] * n
    K = np.concatenate(kh, axis=1).reshape(B, Hkv, -1, D)
    V = np.concatenate(vh, axis=1).reshape(B, Hkv, -1, D)
    return segs, K, V, np.asarray(seg_id, np.int32)
