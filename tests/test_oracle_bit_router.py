"""Pins of the oracle's learned bit-width routing (Sec. 3.2): the selected
width is the router's most probable one, ties go to the lowest width, each
expert uses its own router, and with fixed choices the routing is exactly
the table routing of the same widths."""
import numpy as np

from oracle import oracle as O


def test_choice_is_most_probable_width():
    rng = np.random.default_rng(0)
    z = rng.standard_normal((9, 5, 4))
    ch = O.bit_router_choice(z, 5)
    p = O.bit_router_probs(z)
    assert np.allclose(p.sum(-1), 1.0)
    assert np.all(p > 0)
    for t in range(9):
        for e in range(5):
            assert p[t, e, ch[t, e] - 5] == p[t, e].max()
    assert ch.min() >= 5 and ch.max() <= 8


def test_ties_go_to_lowest_width():
    z = np.zeros((2, 3, 7))
    z[1, 0, 2] = z[1, 0, 5] = 1.0   # two equal maxima
    z[1, 1, 6] = 0.5
    ch = O.bit_router_choice(z, 2)
    assert ch[0].tolist() == [2, 2, 2]           # all scores equal -> b_min
    assert ch[1].tolist() == [4, 8, 2]


def test_each_expert_uses_its_own_router():
    """E != L and a different preferred width per expert: a transposed or
    shared router layout would pick other widths."""
    T, E, L = 4, 6, 3
    z = np.full((T, E, L), -1.0)
    for e in range(E):
        z[:, e, (e * 2) % L] = 1.0 + e
    ch = O.bit_router_choice(z, 1)
    assert ch.tolist() == [[1 + (e * 2) % L for e in range(E)]] * T


def test_fixed_choices_equal_table_routing():
    """Routers that prefer one width per expert whatever the token route
    exactly like a one-request table of those widths."""
    rng = np.random.default_rng(1)
    T, E, k, b_min, b_max = 30, 8, 2, 2, 8
    L = b_max - b_min + 1
    logits = rng.standard_normal((T, E))
    widths = rng.integers(b_min, b_max + 1, size=E).astype(np.uint8)
    z = rng.standard_normal((T, E, L)) * 0.1
    z[:, np.arange(E), widths - b_min] += 10.0
    got = O.route_learned(logits, k, z, b_min, b_max)
    want = O.route_from_logits(logits, k, None, widths[None, :], b_min, b_max)
    for key in ("topk_idx", "topk_bits", "topk_w", "hist", "offsets", "perm", "slot_of",
                "maxbit"):
        assert np.array_equal(got[key], want[key]), key


def test_bits_follow_the_token():
    """Per-token choices: the same expert runs at different widths for
    different tokens, and the counts B_{j,k} split accordingly."""
    T, E, k = 4, 2, 1
    logits = np.array([[1.0, 0.0]] * T)          # every token picks expert 0
    z = np.zeros((T, E, 3))
    for t in range(T):
        z[t, 0, t % 3] = 1.0
    r = O.route_learned(logits, k, z, 2, 4)
    assert r["topk_idx"].ravel().tolist() == [0] * T
    assert r["topk_bits"].ravel().tolist() == [2, 3, 4, 2]
    assert r["hist"][0].tolist() == [2, 1, 1] and r["hist"][1].tolist() == [0, 0, 0]
    assert r["maxbit"].tolist() == [4, 0]
