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


@pytest.mark.parametrize("T", [4, 16])
def test_captured_decode_step_replays_exactly(T):
    L = Layer(wl.scaled(wl.mixtral_decode(T=T), d=512, f=384)).pack()
    s = L.spec
    x = L.x_dev()
    Wg = torch.from_numpy(L.Wg).to(DEV)
    req = torch.from_numpy(L.req).to(DEV)
    table = torch.from_numpy(L.table).to(DEV)
    r = api.Routing.empty(s.T, s.E, s.k, s.b_min, s.b_max, device=DEV)
    out = torch.empty_like(x)
    ws = torch.empty(api.moe_forward_workspace(s.T, s.d, s.f, s.E, s.k), dtype=torch.uint8,
                     device=DEV)

    def step():
        api.route(x, Wg, None, s.k, req, table, s.b_min, s.b_max, out=r)
        api.moe_forward(x, L.w13, L.w2, r, s.k, out=out, workspace=ws)

    step()
    torch.cuda.synchronize()
    want = _snapshot(r, out)

    # other eager work between replays: a different batch through the same layer
    other = Layer(wl.scaled(wl.mixtral_decode(T=3), d=512, f=384))
    other.w13, other.w2, other.shared = L.w13, L.w2, None
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
