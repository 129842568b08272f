"""GPU parity of batched attention over requests of different segment layouts
(App. E, "Batched attention and CFG execution"): one uc_attend_batch call
against the oracle's attention of every request on its own."""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import oracle as ref  # noqa: E402
import paper_2609_32831_amd as uc  # noqa: E402
from gpu_util import TORCH, check_attention, dev, packed_from_oracle, rand_rows, sm_scale  # noqa: E402

Hq, Hkv, D = 28, 4, 128


def _request(seed, parts, dt="bf16"):
    """One request's segments (one-request layouts) and its logical K/V.
    parts: ("dense", n) | ("tail", n, cap) | ("packed", n, G, bits) |
    ("grown", n, G, bits, capacity)."""
    segs, kh, vh = [], [], []
    for j, p in enumerate(parts):
        s = seed * 10 + j
        if p[0] in ("dense", "tail"):
            n = p[1]
            cap = p[2] if p[0] == "tail" else n
            k = rand_rows(s, Hkv, cap, D, dt, outliers=(5,))
            v = rand_rows(s + 500, Hkv, cap, D, dt)
            segs.append(uc.dense_segment(dev(k, dt).reshape(1, Hkv, cap, D),
                                         dev(v, dt).reshape(1, Hkv, cap, D), n_rows=n))
            kh.append(ref.widen(k[:, :n], dt))
            vh.append(ref.widen(v[:, :n], dt))
        else:
            n, G, bits = p[1], p[2], p[3]
            k = rand_rows(s, Hkv, n, D, dt, 2.0, outliers=(5,))
            v = rand_rows(s + 500, Hkv, n, D, dt)
            pk = ref.quantize(k, v, dt, G, [bits] * Hkv)
            if p[0] == "packed":
                segs.append(packed_from_oracle(1, Hkv, n, D, G, dt, pk))
            else:  # a segment with room to grow, quantised on the GPU
                seg = uc.packed_segment(1, Hkv, n, D, G, TORCH[dt], bits=bits, capacity=p[4])
                uc.uc_quantize_segment(uc.make_shape(1, Hq, Hkv, D), dev(k, dt).reshape(1, Hkv, n, D),
                                       dev(v, dt).reshape(1, Hkv, n, D), n, seg)
                segs.append(seg)
            a, b = ref.dequant(pk, n, D, G, dt)
            kh.append(a)
            vh.append(b)
    seg_id = np.concatenate([np.full(x.shape[1], i, np.int32) for i, x in enumerate(kh)])
    K = np.concatenate(kh, axis=1)[None]
    V = np.concatenate(vh, axis=1)[None]
    return segs, K, V, seg_id


REQUESTS = [
    [("dense", 100), ("dense", 1000), ("packed", 300, 64, 4), ("tail", 3, 8)],
    [("packed", 130, 32, 2), ("dense", 17)],
    [("dense", 5000)],
    [("grown", 4100, 64, 4, 4200), ("tail", 1, 4)],
    [("dense", 1)],
    [("tail", 0, 4), ("packed", 64, 64, 4)],
]


@pytest.mark.parametrize("M", [1, 2])
def test_attend_batch_matches_each_request(M):
    print("CASE attend_batch M", M, flush=True)
    reqs, refs = [], []
    for r, parts in enumerate(REQUESTS):
        segs, K, V, seg_id = _request(r + 1, parts)
        reqs.append(segs)
        refs.append((K, V, seg_id, len(parts)))
    B = len(reqs)
    q = rand_rows(99, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    shape = uc.make_shape(B, Hq, Hkv, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    sm = sm_scale(D)
    uc.uc_attend_batch(shape, reqs, dev(q, "bf16"), M, sm, o, lse)
    assert uc.uc_last_kernel() == "decode_batch"
    torch.cuda.synchronize()
    og, lg = o.cpu().numpy(), lse.cpu().numpy()
    for r, (K, V, seg_id, ns) in enumerate(refs):
        o_ref, lse_ref, _, _ = ref.attend(ref.widen(q[r:r + 1], "bf16"), K, V, None, seg_id, ns, sm)
        check_attention(og[r:r + 1], o_ref, f"request {r}")
        assert np.allclose(lg[r:r + 1], lse_ref, rtol=1e-5, atol=1e-4), r
        # and the single-request call agrees far inside the bar
        o1 = torch.empty(1, Hq, M, D, device="cuda")
        uc.uc_attend_mixed(uc.make_shape(1, Hq, Hkv, D), reqs[r], dev(q[r:r + 1], "bf16"), M, sm, o1)
        torch.cuda.synchronize()
        assert np.abs(o1.cpu().numpy() - og[r:r + 1]).max() < 5e-4, r


def test_attend_batch_many_requests():
    """More requests than the launch can give a pair of workgroups per KV
    head (70 > 2 * 256 / 4 / 2): each gets single workgroups by its share of
    the bytes; every request still matches the oracle."""
    print("CASE attend_batch 70 requests", flush=True)
    reqs, refs = [], []
    for r in range(70):
        parts = [("dense", 20 + 37 * (r % 9))] + ([("packed", 64, 64, 4)] if r % 3 == 0 else [])
        segs, K, V, seg_id = _request(200 + r, parts)
        reqs.append(segs)
        refs.append((K, V, seg_id, len(parts)))
    B, M = len(reqs), 1
    q = rand_rows(98, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    sm = sm_scale(D)
    uc.uc_attend_batch(uc.make_shape(B, Hq, Hkv, D), reqs, dev(q, "bf16"), M, sm, o)
    assert uc.uc_last_kernel() == "decode_batch"
    torch.cuda.synchronize()
    og = o.cpu().numpy()
    for r, (K, V, seg_id, ns) in enumerate(refs):
        o_ref, _, _, _ = ref.attend(ref.widen(q[r:r + 1], "bf16"), K, V, None, seg_id, ns, sm)
        check_attention(og[r:r + 1], o_ref, f"request {r}")


@pytest.mark.parametrize("M", [1, 2])
def test_attend_batch_short_line(M):
    """A batch with a few tiles in all: requests shorter than a tile (most
    of their workgroups get empty shares), a packed segment with residual
    rows, M = 2 query rows per head."""
    print("CASE attend_batch short line M", M, flush=True)
    parts = [[("dense", 5)], [("dense", 40), ("tail", 2, 4)], [("packed", 70, 32, 2), ("dense", 70)],
             [("tail", 1, 1)]]
    reqs, refs = [], []
    for r, pr in enumerate(parts):
        segs, K, V, seg_id = _request(300 + r, pr)
        reqs.append(segs)
        refs.append((K, V, seg_id, len(pr)))
    B = len(reqs)
    q = rand_rows(97, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    lse = torch.empty(B, Hq, M, device="cuda")
    sm = sm_scale(D)
    uc.uc_attend_batch(uc.make_shape(B, Hq, Hkv, D), reqs, dev(q, "bf16"), M, sm, o, lse)
    assert uc.uc_last_kernel() == "decode_batch"
    torch.cuda.synchronize()
    og, lg = o.cpu().numpy(), lse.cpu().numpy()
    for r, (K, V, seg_id, ns) in enumerate(refs):
        o_ref, lse_ref, _, _ = ref.attend(ref.widen(q[r:r + 1], "bf16"), K, V, None, seg_id, ns, sm)
        check_attention(og[r:r + 1], o_ref, f"request {r}")
        assert np.allclose(lg[r:r + 1], lse_ref, rtol=1e-5, atol=1e-4), r


@pytest.mark.parametrize("n_req", [32, 33])
def test_attend_batch_descriptor_capacity(n_req):
    """32 requests of two segments fill the descriptors that travel in the
    attention kernel's arguments exactly (32 requests, 64 segments); 33 go
    through the workspace instead.  Both match the oracle."""
    print("CASE attend_batch capacity", n_req, flush=True)
    reqs, refs = [], []
    for r in range(n_req):
        parts = [("dense", 40 + 29 * (r % 7)), ("packed", 64, 32, 2 if r % 2 else 4)]
        segs, K, V, seg_id = _request(400 + r, parts)
        reqs.append(segs)
        refs.append((K, V, seg_id, len(parts)))
    B, M = len(reqs), 1
    q = rand_rows(96, B * Hq, M, D, "bf16").reshape(B, Hq, M, D)
    o = torch.empty(B, Hq, M, D, device="cuda")
    sm = sm_scale(D)
    uc.uc_attend_batch(uc.make_shape(B, Hq, Hkv, D), reqs, dev(q, "bf16"), M, sm, o)
    assert uc.uc_last_kernel() == "decode_batch"
    torch.cuda.synchronize()
    og = o.cpu().numpy()
    for r, (K, V, seg_id, ns) in enumerate(refs):
        o_ref, _, _, _ = ref.attend(ref.widen(q[r:r + 1], "bf16"), K, V, None, seg_id, ns, sm)
        check_attention(og[r:r + 1], o_ref, f"request {r}")


def test_attend_batch_falls_back_per_request():
    """A request outside the batched kernel's range (fp32 rows) sends every
    request through its own call; results are the same as each call's."""
    print("CASE attend_batch fallback", flush=True)
    r0, K0, V0, s0 = _request(7, [("dense", 300)], dt="f32")
    r1, K1, V1, s1 = _request(8, [("dense", 200), ("packed", 128, 64, 4)], dt="f32")
    q = rand_rows(5, 2 * Hq, 1, D, "f32").reshape(2, Hq, 1, D)
    o = torch.empty(2, Hq, 1, D, device="cuda")
    sm = sm_scale(D)
    uc.uc_attend_batch(uc.make_shape(2, Hq, Hkv, D), [r0, r1], dev(q, "f32"), 1, sm, o)
    torch.cuda.synchronize()
    for r, (K, V, sid, ns) in enumerate([(K0, V0, s0, 1), (K1, V1, s1, 2)]):
        o_ref, _, _, _ = ref.attend(ref.widen(q[r:r + 1], "f32"), K, V, None, sid, ns, sm)
        check_attention(o.cpu().numpy()[r:r + 1], o_ref, f"request {r}")
