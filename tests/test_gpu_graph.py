"""The routing and forward entry points can be captured in a HIP graph: they
allocate nothing, never synchronize with the host and clear what must start
at zero with kernels (no memset nodes).  A captured decode step is replayed
several times, with eager work of other shapes between the replays, and every
replay must reproduce the eager outputs bit for bit (the kernels are
deterministic: no floating-point atomics on outputs)."""
import numpy as np
import pytest
import torch

from layer_cases import DEV, Layer
from paper_2504_15299_amd import api
from paper_2504_15299_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _snapshot(r: api.Routing, out):
    names = ("logits", "topk_idx", "topk_w", "topk_bits", "hist", "offsets", "perm", "slot_of",
             "expert_maxbit", "flags")
    return {n: getattr(r, n).clone() for n in names} | {"out": out.clone()}


GRAPH_SPECS = {
    "decode_T4": wl.scaled(wl.mixtral_decode(T=4), d=512, f=384),
    "decode_T16": wl.scaled(wl.mixtral_decode(T=16), d=512, f=384),
    # the grouped-GEMM path: chunk tables built on the device, wide and narrow
    # chunks, and a shared expert whose W2 reduction is split in parts
    "prefill_small": wl.scaled(wl.mixtral_prefill(), d=256, f=384, T=600),
    "fine_shared_split": wl.scaled(wl.fine_grained(), d=256, f=64, T=200, shared_f=1024),
}


@pytest.mark.parametrize("name", list(GRAPH_SPECS))
def test_captured_step_replays_exactly(name):
    L = Layer(GRAPH_SPECS[name]).pack()
    s = L.spec
    x = L.x_dev()
    Wg = torch.from_numpy(L.Wg).to(DEV)
    bias = None if L.bias is None else torch.from_numpy(L.bias).to(DEV)
    req = torch.from_numpy(L.req).to(DEV)
    table = torch.from_numpy(L.table).to(DEV)
    r = api.Routing.empty(s.T, s.E, s.k, s.b_min, s.b_max, device=DEV)
    out = torch.empty_like(x)
    ws = torch.empty(api.moe_forward_workspace(s.T, s.d, s.f, s.E, s.k,
                                               shared_d_ff=s.shared_f or 0),
                     dtype=torch.uint8, device=DEV)

    def step():
        api.route(x, Wg, bias, s.k, req, table, s.b_min, s.b_max, out=r)
        api.moe_forward(x, L.w13, L.w2, r, s.k, shared=L.shared, out=out, workspace=ws)

    step()
    torch.cuda.synchronize()
    want = _snapshot(r, out)

    # other eager work between replays: a different batch through the same layer
    other = Layer(wl.scaled(s, T=3))
    other.w13, other.w2, other.shared = L.w13, L.w2, L.shared
    other.route()

    g = torch.cuda.CUDAGraph()
    s_cap = torch.cuda.Stream()
    s_cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s_cap):
        step()  # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(s_cap)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        out.zero_()
        r.perm.fill_(-7)
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(r, out)
        for name, ref in want.items():
            assert torch.equal(got[name], ref), f"replay {rep}: {name} differs"
        other.forward()  # eager work between replays
        torch.cuda.synchronize()
