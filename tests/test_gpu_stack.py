"""Decoder stack of MoE layers on the device against the oracle: the residual
update + RMS normalisation entry point on its own, and a small stack (3
layers, 8 sequences, 2 decode steps, the 64-sequence stack's recipe at
reduced width) run end to end, each step starting from the previous step's
final hidden state.  Tokens whose expert set is decided within the logit
rounding error at any layer may legitimately diverge and are left out (the
count is reported)."""
import numpy as np
import pytest
import torch

from layer_cases import DEV, FWD_TOL, ambiguous_tokens, logit_error_bound, row_max_abs_rel
from oracle import oracle as O
from paper_2504_15299_amd import api
from paper_2504_15299_amd import workloads as wl

pytestmark = pytest.mark.gpu


# widths that take each register-array size of the kernel (values per
# thread 4, 8, 16, 32, 64), ragged and whole
@pytest.mark.parametrize("d,y_dtype,h_dtype", [(4096, torch.bfloat16, torch.bfloat16),
                                               (300, torch.float32, torch.float32),
                                               (2048, torch.float32, torch.bfloat16),
                                               (5000, torch.bfloat16, torch.float32),
                                               (16384, None, torch.bfloat16)])
def test_residual_rmsnorm(d, y_dtype, h_dtype):
    rng = np.random.default_rng(d)
    T = 7
    x0 = (rng.standard_normal((T, d)) * np.array([[1e-3], [1], [3], [50], [0.2], [1], [2]])
          ).astype(np.float32)
    y = None if y_dtype is None else wl.round_to_bf16(rng.standard_normal((T, d), dtype=np.float32))
    x = torch.from_numpy(x0).to(DEV)
    yt = None if y is None else torch.from_numpy(y).to(DEV).to(y_dtype)
    h = api.residual_rmsnorm(x, yt, 1e-5, h_dtype=h_dtype)
    torch.cuda.synchronize()
    xs = x0.astype(np.float64) + (0 if y is None else y.astype(np.float64))
    np.testing.assert_allclose(x.cpu().numpy(), xs.astype(np.float32), rtol=0, atol=0)
    ref = O.rmsnorm(xs, 1e-5)
    got = h.float().cpu().numpy()
    tol = 2.0 ** -8 if h_dtype == torch.bfloat16 else 1e-5
    assert np.abs(got - ref).max() <= tol * np.abs(ref).max()


def test_residual_rmsnorm_rejects_bad_width():
    x = torch.zeros((2, 16385), dtype=torch.float32, device=DEV)
    with pytest.raises(api.D2MoEError):
        api.residual_rmsnorm(x, None)


def test_small_stack_two_steps():
    spec = wl.scaled(wl.mixtral_stack(), d=256, f=256, T=8, n_requests=8)
    L, steps, eps = 3, 2, spec.extra["eps"]
    req = wl.token_requests(spec)
    table = wl.bit_table(spec)
    layers_cpu, layers_gpu = [], []
    for l in range(L):
        Wg, _ = wl.gate(spec, l)
        W13 = np.stack([wl.expert_w13(spec, e, l) for e in range(spec.E)])
        W2 = np.stack([wl.expert_w2(spec, e, l) for e in range(spec.E)])
        layers_cpu.append((Wg, [O.mwq_quantize(w, spec.group) for w in W13],
                           [O.mwq_quantize(w, spec.group) for w in W2]))
        w13 = api.MWQ.empty(spec.E, 2 * spec.f, spec.d, spec.group, device=DEV)
        w2 = api.MWQ.empty(spec.E, spec.d, spec.f, spec.group, device=DEV)
        api.pack_mwq(torch.from_numpy(W13).to(DEV), w13)
        api.pack_mwq(torch.from_numpy(W2).to(DEV), w2)
        layers_gpu.append((torch.from_numpy(Wg).to(DEV), w13, w2))
    x0 = wl.activations(spec).astype(np.float64)

    x = torch.from_numpy(x0.astype(np.float32)).to(DEV)
    reqt, tablet = torch.from_numpy(req).to(DEV), torch.from_numpy(table).to(DEV)
    h = api.residual_rmsnorm(x, None, eps)
    xr = x0
    for step in range(steps):
        for Wg, w13, w2 in layers_gpu:
            r = api.route(h, Wg, None, spec.k, reqt, tablet)
            y = api.moe_forward(h, w13, w2, r, spec.k)
            h = api.residual_rmsnorm(x, y, eps)
        torch.cuda.synchronize()
        xr, logits = O.moe_stack(xr, layers_cpu, spec.k, req, table, eps)
        amb = np.zeros(spec.T, bool)
        for lg, (Wg, _, _) in zip(logits, layers_cpu):
            hb = np.ones((spec.T, spec.d), np.float32)  # |h| <= sqrt(d) after normalisation
            amb |= ambiguous_tokens(lg, spec.k, 4 * logit_error_bound(hb * np.sqrt(spec.d),
                                                                      Wg, None))
        err = row_max_abs_rel(x.cpu().numpy()[~amb], xr[~amb])
        print(f"stack step {step}: worst row {err.max():.3e}, near-tied tokens {int(amb.sum())}")
        assert amb.sum() <= 2
        assert err.max() <= FWD_TOL
