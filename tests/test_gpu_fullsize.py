"""Full-size parity at the Mixtral-8x7B-shaped decode layer, in the launch
configuration the benchmark times: d_model 4096, d_ff 14336, 8 SwiGLU
experts, top-2, a batch of 16 tokens, group 128, 8-bit nest, bits per
(request, expert) from {2,3,4,8}.

Routing is compared on every token.  The layer output is compared on sampled
outputs that the oracle computes one by one: for two tokens chosen to cover
as many bit-widths as possible, 256 of the 4096 output rows (one in every
16-row block, at every position within a block).
The oracle quantizes the full W1/W3 of each expert those tokens use and only
the sampled rows of W2 (MWQ codes of a row depend on that row alone).  The
remaining experts get seeded weights drawn on the device; no sampled output
depends on them."""
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

from layer_cases import (DEV, FWD_TOL, Layer, ambiguous_tokens, logit_error_bound,
                         row_max_abs_rel)
from oracle import oracle as O
from paper_2504_15299_amd import api
from paper_2504_15299_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _say(t0, msg):
    print(f"[{time.time() - t0:6.1f} s] {msg}", flush=True)


def test_mixtral_decode_full_size_sampled():
    t0 = time.time()
    s = wl.mixtral_decode(T=16)
    x = wl.activations(s)
    Wg, bias = wl.gate(s)
    req = wl.token_requests(s)
    table = wl.bit_table(s)
    ref_logits = O.gate_logits(x, Wg, bias)
    ref = O.route_from_logits(ref_logits, s.k, req, table, s.b_min, s.b_max)
    amb = ambiguous_tokens(ref_logits, s.k, logit_error_bound(x, Wg, bias))
    decided = [t for t in range(s.T) if not amb[t]]
    # the first decided token, and the one that adds the most bit-widths to it
    seen = set(int(b) for b in ref["topk_bits"][decided[0]])
    second = max(decided[1:], key=lambda t: (len(set(int(b) for b in ref["topk_bits"][t]) - seen),
                                             -t))
    tokens = [decided[0], second]
    need = sorted({int(e) for t in tokens for e in ref["topk_idx"][t]})
    rows = np.arange(0, s.d, 16) + np.arange(s.d // 16) % 16  # one per 16-row block
    _say(t0, f"tokens {tokens}, experts {need}, bits "
             f"{[list(map(int, ref['topk_bits'][t])) for t in tokens]}, near-tied {int(amb.sum())}")

    w13 = api.MWQ.empty(s.E, 2 * s.f, s.d, s.group, s.b_min, s.b_max, device=DEV)
    w2 = api.MWQ.empty(s.E, s.d, s.f, s.group, s.b_min, s.b_max, device=DEV)
    gen = torch.Generator(device=DEV)
    gen.manual_seed(2024)
    cpu_weights = {}
    for e in range(s.E):
        if e in need:
            W13, W2 = wl.expert_w13(s, e), wl.expert_w2(s, e)
            cpu_weights[e] = (W13, np.ascontiguousarray(W2[rows]))
            a, b = torch.from_numpy(W13[None]).to(DEV), torch.from_numpy(W2[None]).to(DEV)
        else:
            a = torch.randn((1, 2 * s.f, s.d), generator=gen, device=DEV) * 0.02
            b = torch.randn((1, s.d, s.f), generator=gen, device=DEV) * 0.02
        api.pack_mwq(a, w13.expert(e))
        api.pack_mwq(b, w2.expert(e))
        torch.cuda.synchronize()
        del a, b
    _say(t0, "weights packed on the device")

    xt = torch.from_numpy(x).to(DEV).to(torch.bfloat16)
    r = api.route(xt, torch.from_numpy(Wg).to(DEV), None, s.k, torch.from_numpy(req).to(DEV),
                  torch.from_numpy(table).to(DEV), s.b_min, s.b_max)
    ws = torch.empty(api.moe_forward_workspace(s.T, s.d, s.f, s.E, s.k), dtype=torch.uint8,
                     device=DEV)
    out = api.moe_forward(xt, w13, w2, r, s.k, workspace=ws)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    _say(t0, "route + forward done on the device")

    gi, gb = r.topk_idx.cpu().numpy(), r.topk_bits.cpu().numpy()
    assert np.array_equal(gi[~amb], ref["topk_idx"][~amb])
    assert np.array_equal(gb[~amb], ref["topk_bits"][~amb])
    if not amb.any():
        for name in ("hist", "offsets", "perm", "slot_of"):
            assert np.array_equal(getattr(r, name).cpu().numpy().ravel(),
                                  np.asarray(ref[name]).ravel()), name
        assert np.array_equal(r.expert_maxbit.cpu().numpy(), ref["maxbit"])
    assert np.isfinite(got).all()

    def oracle_expert(e):
        W13, W2s = cpu_weights[e]
        c13 = O.mwq_quantize(W13, s.group, s.b_min, s.b_max)
        c2 = O.mwq_quantize(W2s, s.group, s.b_min, s.b_max)
        ys = {}
        for t in tokens:
            for i in range(s.k):
                if int(ref["topk_idx"][t, i]) == e:
                    ys[(t, i)] = O.expert_ffn(c13, c2, int(ref["topk_bits"][t, i]),
                                              x[t:t + 1].astype(np.float64))[0]
        return ys

    with ThreadPoolExecutor(len(need)) as ex:
        y_slot = {}
        for ys in ex.map(oracle_expert, need):
            y_slot.update(ys)
    _say(t0, "oracle done")

    ysl = np.stack([np.stack([y_slot[(t, i)] for i in range(s.k)]) for t in tokens])
    want = O.combine(np.asarray(ref["topk_w"])[tokens], ysl)
    err = row_max_abs_rel(got[tokens][:, rows], want)
    print(f"full-size decode: tokens {tokens} worst row {err.max():.3e}", flush=True)
    assert err.max() <= FWD_TOL


def _bucket_cover(idx, bits, candidates, per_group=None, groups=None):
    """Tokens from `candidates` chosen greedily so that every (expert, bit)
    bucket that any candidate uses holds at least one chosen slot; with
    `groups` (a group id per token) at least `per_group` tokens per group."""
    need = {(int(e), int(b)) for t in candidates for e, b in zip(idx[t], bits[t])}
    chosen, have = [], set()
    while need - have:
        t = max(candidates, key=lambda u: (len({(int(e), int(b)) for e, b in zip(idx[u], bits[u])}
                                               - have), -u))
        chosen.append(t)
        have |= {(int(e), int(b)) for e, b in zip(idx[t], bits[t])}
        candidates = [u for u in candidates if u != t]
    if groups is not None:
        for gid in np.unique(groups):
            mine = [t for t in chosen if groups[t] == gid]
            extra = [t for t in candidates if groups[t] == gid][:max(0, per_group - len(mine))]
            chosen += extra
    return sorted(set(chosen))


def _sampled_full_layer(spec, t0, rows, per_group=None):
    """Route + forward the full layer on the device; compare routing on every
    token and the output on a sample of tokens (every (expert, bit) bucket
    covered) and of output columns against the oracle."""
    L = Layer(spec)
    _say(t0, "inputs drawn")
    L.pack()
    L.route()
    got = L.forward()
    _say(t0, "route + forward done on the device")
    amb = ambiguous_tokens(L.ref_logits, spec.k, logit_error_bound(L.x, L.Wg, L.bias))
    gi, gb = L.r.topk_idx.cpu().numpy(), L.r.topk_bits.cpu().numpy()
    assert np.array_equal(gi[~amb], L.ref_route["topk_idx"][~amb])
    assert np.array_equal(gb[~amb], L.ref_route["topk_bits"][~amb])
    assert amb.sum() <= max(1, spec.T // 50)
    assert np.isfinite(got).all()
    decided = [t for t in range(spec.T) if not amb[t]]
    groups = L.req if per_group else None
    toks = _bucket_cover(L.ref_route["topk_idx"], L.ref_route["topk_bits"], decided,
                         per_group, groups)
    idx, bits = L.ref_route["topk_idx"], L.ref_route["topk_bits"]
    need = sorted({int(e) for t in toks for e in idx[t]})
    _say(t0, f"{len(toks)} sampled tokens, {len(need)} experts, near-tied {int(amb.sum())}")

    def codes(e):
        return (O.mwq_quantize(L.W13[e], spec.group, spec.b_min, spec.b_max),
                O.mwq_quantize(np.ascontiguousarray(L.W2[e][rows]), spec.group, spec.b_min,
                               spec.b_max))

    with ThreadPoolExecutor(16) as ex:
        cs = dict(zip(need, ex.map(codes, need)))
        work = [(e, b) for e in need for b in sorted({int(bits[t, i]) for t in toks
                                                      for i in range(spec.k) if idx[t, i] == e})]

        def ffn(eb):
            e, b = eb
            sel = [(j, i) for j, t in enumerate(toks) for i in range(spec.k)
                   if idx[t, i] == e and bits[t, i] == b]
            xs = np.stack([L.x[toks[j]] for j, _ in sel]).astype(np.float64)
            return sel, O.expert_ffn(cs[e][0], cs[e][1], b, xs)

        y_slot = np.zeros((len(toks), spec.k, len(rows)), np.float64)
        for sel, ys in ex.map(ffn, work):
            for (j, i), yv in zip(sel, ys):
                y_slot[j, i] = yv
        want = O.combine(L.ref_route["topk_w"][toks], y_slot)
        if spec.shared_f:
            sc13 = O.mwq_quantize(L.SW13, spec.group, spec.b_min, spec.b_max)
            sc2 = O.mwq_quantize(np.ascontiguousarray(L.SW2[rows]), spec.group, spec.b_min,
                                 spec.b_max)
            want = want + O.expert_ffn(sc13, sc2, spec.shared_bits,
                                       L.x[toks].astype(np.float64))
    _say(t0, "oracle done")
    err = row_max_abs_rel(got[toks][:, rows], want)
    print(f"{spec.name} full size: {len(toks)} tokens, worst row {err.max():.3e}, "
          f"median {np.median(err):.3e}", flush=True)
    assert err.max() <= FWD_TOL


@pytest.mark.parametrize("T", [1, 4, 32])
def test_mixtral_decode_other_batches_full_size_sampled(T):
    """Decode batches of 1 and 4 tokens (their W2 grids are too small for the
    row-block-pair kernel: one 4-wave workgroup per W2 row block) and of 32
    (more than 7 positions per expert: two 8-token column blocks per work
    item) at the full Mixtral layer: routing on every token, the output on
    tokens covering every (expert, bit) bucket, 256 of the 4096 columns."""
    t0 = time.time()
    s = wl.mixtral_decode(T=T)
    rows = np.arange(0, s.d, 16) + np.arange(s.d // 16) % 16
    _sampled_full_layer(s, t0, rows)


def test_mixtral_prefill_full_size_sampled():
    """2048 tokens from 4 requests (Zipf(1.1) expert load, bits from {2,4,8}
    per request and expert): routing on every token, the output on at least
    16 tokens per request covering every (expert, bit) bucket, 256 of the
    4096 output columns (one per 16-row block, every offset within a block)."""
    t0 = time.time()
    s = wl.mixtral_prefill()
    rows = np.arange(0, s.d, 16) + np.arange(s.d // 16) % 16
    _sampled_full_layer(s, t0, rows, per_group=16)


def test_fine_grained_full_size_sampled():
    """512 tokens, 64 routed experts (top-6, bits hottest-first 8/4/3/2) plus
    the shared expert at 8 bits: routing on every token, the output on tokens
    covering every (expert, bit) bucket, 256 of the 2048 output columns."""
    t0 = time.time()
    s = wl.fine_grained()
    rows = np.arange(0, s.d, 8) + np.arange(s.d // 8) % 8
    _sampled_full_layer(s, t0, rows)


def test_mixtral_v2_decode_full_size_sampled():
    """Batch-16 decode of the full Mixtral layer under the paper's second
    nest (b_min 5, b_max 8): routing on every token, the output on tokens
    covering every (expert, bit) bucket, 256 of the 4096 output columns."""
    t0 = time.time()
    s = wl.mixtral_decode_v2(T=16)
    rows = np.arange(0, s.d, 16) + np.arange(s.d // 16) % 16
    _sampled_full_layer(s, t0, rows)


def test_dense_full_size_sampled():
    """LLaMA2-13B-shaped dense SwiGLU FFN (one expert, top-1), batch 16 at
    bits {2,3,4}: every token's output on 320 of the 5120 columns."""
    t0 = time.time()
    s = wl.dense_decode(T=16)
    rows = np.arange(0, s.d, 16) + np.arange(s.d // 16) % 16
    _sampled_full_layer(s, t0, rows)
