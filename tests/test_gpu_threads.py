"""The forward runs the shared expert and the small routed experts on side
streams of the calling host thread.  Two host threads, each on its own stream
with its own buffers, run the same layers at the same time and must reproduce
the single-thread outputs bit for bit (the kernels are deterministic), and a
layer on the default stream must as well."""
import threading

import pytest
import torch

from layer_cases import DEV, Layer
from paper_2504_15299_amd import api
from paper_2504_15299_amd import workloads as wl

pytestmark = pytest.mark.gpu

SPEC = wl.scaled(wl.fine_grained(), d=256, f=64, T=200, shared_f=1024)


def _setup(seed_layer):
    L = Layer(SPEC, layer=seed_layer).pack()
    s = L.spec
    x = L.x_dev()
    Wg = torch.from_numpy(L.Wg).to(DEV)
    bias = None if L.bias is None else torch.from_numpy(L.bias).to(DEV)
    req = torch.from_numpy(L.req).to(DEV)
    table = torch.from_numpy(L.table).to(DEV)
    ws = torch.empty(api.moe_forward_workspace(s.T, s.d, s.f, s.E, s.k, shared_d_ff=s.shared_f),
                     dtype=torch.uint8, device=DEV)
    return L, x, Wg, bias, req, table, ws


def _run(case, stream, reps):
    L, x, Wg, bias, req, table, ws = case
    s = L.spec
    outs = []
    with torch.cuda.stream(stream):
        for _ in range(reps):
            r = api.route(x, Wg, bias, s.k, req, table, s.b_min, s.b_max)
            outs.append(api.moe_forward(x, L.w13, L.w2, r, s.k, shared=L.shared, workspace=ws))
    stream.synchronize()
    return outs


def test_two_host_threads_and_default_stream():
    cases = [_setup(0), _setup(1)]
    want = [_run(c, torch.cuda.Stream(), 1)[0] for c in cases]
    results = [None, None]

    def worker(i):
        results[i] = _run(cases[i], torch.cuda.Stream(), 6)

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
        assert not t.is_alive(), "worker thread did not finish"
    for i in range(2):
        for rep, got in enumerate(results[i]):
            assert torch.equal(got, want[i]), f"thread {i} call {rep} differs"
    # the legacy default stream (the fork and join events work on it too)
    got = _run(cases[0], torch.cuda.default_stream(), 2)
    for rep, g in enumerate(got):
        assert torch.equal(g, want[0]), f"default stream call {rep} differs"
