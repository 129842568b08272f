"""Decode steps captured in a HIP graph: the library enqueues only kernels on
the caller's stream (no allocation, no synchronisation, no memset nodes), so
a captured run of fused decode steps replays the same work.  Each replay,
with eager work and synchronisations between replays, must reproduce the
outputs of the steps issued one by one bit for bit."""
import pytest
import torch

if not torch.cuda.is_available():
    pytest.skip("needs a GPU", allow_module_level=True)

import paper_2609_32831_amd as uc  # noqa: E402
import workloads as gen  # noqa: E402
from paper_2609_32831_amd.runner import Run  # noqa: E402
from workloads.device import device_inputs  # noqa: E402

pytestmark = pytest.mark.gpu


def test_decode_steps_replayed_from_graph():
    print("CASE test=graph workload=understanding_7b steps=16", flush=True)
    w = gen.UNDERSTANDING_7B
    T = 16
    inp = device_inputs(w, "cuda", steps=T)
    run = Run(w, inp)
    o = torch.empty(T, w.B, w.Hq, 1, w.D, device="cuda")

    def steps():
        for t in range(T):
            uc.uc_attend_append(run.shape, run.mixed, len(run.mixed) - 1, inp["k_dec"][t],
                                inp["v_dec"][t], 1, inp["q_dec"][t], 1, run.sm, o[t],
                                ws=run.ws_attend)

    run.compress()
    steps()
    torch.cuda.synchronize()
    o_eager = o.clone()
    run.tail.n_rows = 0
    stream = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    side.wait_stream(stream)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=side):
        steps()
    torch.cuda.synchronize()
    other = torch.empty(w.B, w.Hq, 1, w.D, device="cuda")
    for rep in range(3):
        o.zero_()
        # eager work between replays: an attention call over the same cache
        uc.uc_attend_mixed(run.shape, run.mixed[:-1], inp["q_dec"][rep], 1, run.sm, other,
                           ws=run.ws_attend)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, o_eager), f"replay {rep} differs from the steps issued one by one"
