"""Pins of oracle.model (MoE layer of Section 2.1 / Eq. 1) against closed forms,
brute force and invariants -- never against a retyped copy of itself."""
import math

import numpy as np
import pytest

from oracle import model
from oracle.numerics import identity, round_bf16


def _selection(rows, cols, rng):
    """A [rows][cols] matrix with one nonzero per row: (matrix, picked col, value)."""
    pick = rng.integers(0, cols, size=rows)
    val = rng.uniform(0.5, 2.0, size=rows) * rng.choice([-1, 1], size=rows)
    Mx = np.zeros((rows, cols))
    Mx[np.arange(rows), pick] = val
    return Mx, pick, val


def _silu_scalar(v):
    return v / (1.0 + math.exp(-v))


def test_expert_ffn_selection_matrices_closed_form():
    """With one nonzero per weight row every output element has a closed form,
    so a dropped term, a transposed operand or a wrong index changes it."""
    rng = np.random.default_rng(3)
    M, H, F = 5, 7, 11
    a = rng.normal(size=(M, H))
    Wg, pg, cg = _selection(F, H, rng)
    Wu, pu, cu = _selection(F, H, rng)
    Wd, pd, cd = _selection(H, F, rng)
    h, o = model.expert_ffn(a, Wg, Wu, Wd, identity)
    for i in range(M):
        for f in range(F):
            want = _silu_scalar(cg[f] * a[i, pg[f]]) * cu[f] * a[i, pu[f]]
            assert h[i, f] == pytest.approx(want, rel=1e-14, abs=1e-300)
        for n in range(H):
            assert o[i, n] == pytest.approx(cd[n] * h[i, pd[n]], rel=1e-14, abs=1e-300)


def test_expert_ffn_bf16_rounds_h_and_o():
    rng = np.random.default_rng(4)
    a = round_bf16(rng.normal(size=(3, 16)))
    Wg, Wu, Wd = (round_bf16(rng.normal(size=s) * 0.3) for s in [(8, 16), (8, 16), (16, 8)])
    h, o = model.expert_ffn(a, Wg, Wu, Wd, round_bf16)
    assert np.array_equal(round_bf16(h), h) and np.array_equal(round_bf16(o), o)
    h32, _ = model.expert_ffn(a, Wg, Wu, Wd, identity)
    assert np.array_equal(h, round_bf16(h32))


def test_rmsnorm_closed_form():
    c, eps = -3.0, 1e-6
    x = np.full((2, 64), c)
    g = np.linspace(0.5, 1.5, 64)
    a = model.rmsnorm_cast(x, g, eps, identity)
    assert np.allclose(a, c / math.sqrt(c * c + eps) * g, rtol=1e-15)
    # one nonzero entry: mean(x^2) = v^2 / H
    x = np.zeros((1, 16)); x[0, 3] = 2.0
    a = model.rmsnorm_cast(x, np.ones(16), 0.0, identity)
    assert a[0, 3] == pytest.approx(2.0 / math.sqrt(4.0 / 16)) and np.count_nonzero(a) == 1


def _topk_brute(z, k):
    out = []
    for row in z:
        left = list(range(len(row)))
        pick = []
        for _ in range(k):
            best = left[0]
            for e in left[1:]:
                if row[e] > row[best]:      # strict: equal logits keep the lower id
                    best = e
            pick.append(best)
            left.remove(best)
        out.append(pick)
    return np.array(out)


def test_topk_brute_force_with_ties():
    rng = np.random.default_rng(5)
    for E, k in [(8, 2), (60, 4), (64, 6), (5, 5), (1, 1)]:
        z = rng.integers(-3, 3, size=(40, E)).astype(np.float64)   # many ties
        assert np.array_equal(model.topk_indices(z, k), _topk_brute(z, k))
    z = np.array([[0.0, -0.0, 0.0]])
    assert list(model.topk_indices(z, 2)[0]) == [0, 1]


def test_gate_weights_properties():
    rng = np.random.default_rng(6)
    z = rng.normal(size=(30, 8))
    idx = model.topk_indices(z, 8)
    w = model.gate_weights(z, idx)
    assert np.allclose(w.sum(1), 1.0)                         # k = E: full softmax
    assert np.all(np.diff(w, axis=1) <= 0)                    # picked in decreasing order
    idx2 = model.topk_indices(z, 2)
    w2 = model.gate_weights(z, idx2)
    assert np.all(w2.sum(1) < 1.0)                            # literal Eq. 1: no renormalisation
    w2n = model.gate_weights(z, idx2, norm_topk=1)
    assert np.allclose(w2n.sum(1), 1.0)
    assert np.allclose(w2n[:, 0] / w2n[:, 1], np.exp(z[np.arange(30), idx2[:, 0]] - z[np.arange(30), idx2[:, 1]]))


def test_device_loads_contiguous_blocks():
    counts = np.arange(8)
    assert list(model.device_loads(counts, 4)) == [1, 5, 9, 13]
    assert list(model.device_loads(counts, 1)) == [28]
    assert list(model.device_loads(counts, 8)) == list(range(8))


def _rand_weights(L, H, F, E, S, rng, scale=0.2):
    router = [rng.normal(size=(E, H)) / math.sqrt(H) for _ in range(L)]
    bias = [rng.normal(size=E) for _ in range(L)]
    gu = {(l, e): (rng.normal(size=(F, H)) * scale, rng.normal(size=(F, H)) * scale)
          for l in range(L) for e in range(E + S)}
    dn = {(l, e): rng.normal(size=(H, F)) * scale for l in range(L) for e in range(E + S)}
    return model.Weights(gain=lambda l: np.ones(H), router=lambda l: router[l],
                         bias=lambda l: bias[l], gate_up=lambda l, e: gu[(l, e)],
                         down=lambda l, e: dn[(l, e)]), router, bias, gu, dn


def test_moe_layer_single_expert_is_dense_ffn():
    """E = 1, k = 1: the softmax weight is 1 and the layer is x + FFN(RMSNorm(x))
    with the closed-form selection-matrix FFN."""
    rng = np.random.default_rng(7)
    H, F, T = 6, 9, 4
    Wg, pg, cg = _selection(F, H, rng)
    Wu, pu, cu = _selection(F, H, rng)
    Wd, pd, cd = _selection(H, F, rng)
    P = model.Weights(gain=lambda l: np.ones(H), router=lambda l: rng.normal(size=(1, H)),
                      bias=lambda l: np.zeros(1), gate_up=lambda l, e: (Wg, Wu),
                      down=lambda l, e: Wd)
    x = rng.normal(size=(T, H))
    out = model.moe_layer(x, 0, P, E=1, k=1, S=0, eps=1e-6, dtype="f32")
    assert np.all(out.w == 1.0)
    for t in range(T):
        a = x[t] / math.sqrt(np.mean(x[t] ** 2) + 1e-6)
        hv = [_silu_scalar(cg[f] * a[pg[f]]) * cu[f] * a[pu[f]] for f in range(F)]
        for n in range(H):
            assert out.x_out[t, n] == pytest.approx(x[t, n] + cd[n] * hv[pd[n]], rel=1e-12)


def test_moe_layer_every_expert_is_the_dense_softmax_mixture():
    """k = E: top-k keeps every expert, so the layer is x + sum_e p_e FFN_e(a)
    with p the softmax of all E logits -- a dense mixture, written here with
    scalar loops and the closed-form selection-matrix experts."""
    rng = np.random.default_rng(11)
    H, F, T, E = 5, 7, 3, 4
    experts = [tuple(_selection(r, c, rng) for r, c in ((F, H), (F, H), (H, F))) for _ in range(E)]
    Wr = rng.normal(size=(E, H))
    b = rng.normal(size=E)
    P = model.Weights(gain=lambda l: np.ones(H), router=lambda l: Wr, bias=lambda l: b,
                      gate_up=lambda l, e: (experts[e][0][0], experts[e][1][0]),
                      down=lambda l, e: experts[e][2][0])
    x = rng.normal(size=(T, H))
    out = model.moe_layer(x, 0, P, E=E, k=E, S=0, eps=1e-6, dtype="f32")
    for t in range(T):
        a = x[t] / math.sqrt(np.mean(x[t] ** 2) + 1e-6)
        z = [sum(a[i] * Wr[e, i] for i in range(H)) + b[e] for e in range(E)]
        den = sum(math.exp(v) for v in z)
        for n in range(H):
            want = x[t, n]
            for e in range(E):
                (_, pg, cg), (_, pu, cu), (_, pd, cd) = experts[e]
                f = pd[n]
                want += math.exp(z[e]) / den * cd[n] * _silu_scalar(cg[f] * a[pg[f]]) * cu[f] * a[pu[f]]
            assert out.x_out[t, n] == pytest.approx(want, rel=1e-10, abs=1e-12)


def test_moe_layer_invariants():
    rng = np.random.default_rng(8)
    L, H, F, E, S, k, T = 1, 16, 12, 6, 2, 2, 10
    P, router, bias, gu, dn = _rand_weights(L, H, F, E, S, rng)
    x = rng.normal(size=(T, H))
    base = model.moe_layer(x, 0, P, E=E, k=k, S=S, eps=1e-6, dtype="f32")
    # 1) per-token independence: a token alone gives the same output
    for t in [0, 7]:
        solo = model.moe_layer(x[t:t + 1], 0, P, E=E, k=k, S=S, eps=1e-6, dtype="f32")
        assert np.allclose(solo.x_out[0], base.x_out[t], rtol=1e-13, atol=1e-13)
    # 2) relabelling experts consistently changes nothing
    pi = rng.permutation(E)
    P2 = model.Weights(gain=P.gain, router=lambda l: router[l][pi], bias=lambda l: bias[l][pi],
                       gate_up=lambda l, e: gu[(l, int(pi[e]) if e < E else e)],
                       down=lambda l, e: dn[(l, int(pi[e]) if e < E else e)])
    re = model.moe_layer(x, 0, P2, E=E, k=k, S=S, eps=1e-6, dtype="f32")
    assert np.allclose(re.x_out, base.x_out, rtol=1e-12, atol=1e-12)
    assert np.array_equal(pi[re.idx], base.idx)
    # 3) zero routed-expert down weights: only shared experts contribute;
    #    zero everything: residual only
    P3 = model.Weights(gain=P.gain, router=P.router, bias=P.bias, gate_up=P.gate_up,
                       down=lambda l, e: dn[(l, e)] * (e >= E))
    only_shared = model.moe_layer(x, 0, P3, E=E, k=k, S=S, eps=1e-6, dtype="f32")
    a = model.rmsnorm_cast(x, np.ones(H), 1e-6, identity)
    shared = sum(model.expert_ffn(a, *gu[(0, E + s)], dn[(0, E + s)], identity)[1] for s in range(S))
    assert np.allclose(only_shared.x_out, x + shared, rtol=1e-12, atol=1e-12)
    P4 = model.Weights(gain=P.gain, router=P.router, bias=P.bias, gate_up=P.gate_up,
                       down=lambda l, e: dn[(l, e)] * 0.0)
    assert np.array_equal(model.moe_layer(x, 0, P4, E=E, k=k, S=S, eps=1e-6, dtype="f32").x_out, x)
    # 4) the k picked experts are the only ones whose weights matter
    t = 3
    unused = [e for e in range(E) if e not in base.idx[t]][0]
    P5 = model.Weights(gain=P.gain, router=P.router, bias=P.bias, gate_up=P.gate_up,
                       down=lambda l, e: dn[(l, e)] * (100.0 if e == unused else 1.0))
    out5 = model.moe_layer(x[t:t + 1], 0, P5, E=E, k=k, S=S, eps=1e-6, dtype="f32")
    assert np.allclose(out5.x_out[0], base.x_out[t], rtol=1e-13, atol=1e-13)


def test_moe_layer_weighted_sum_two_experts_closed_form():
    """k = 2 of E = 2 with diagonal experts: x + p0 * o0 + p1 * o1 exactly (Eq. 1)."""
    H = F = 3
    rng = np.random.default_rng(9)
    diag = {0: (np.diag([1.0, 2.0, 3.0]), np.diag([0.5, 0.5, 0.5]), np.diag([1.0, -1.0, 2.0])),
            1: (np.diag([-1.0, 1.0, 0.5]), np.diag([2.0, 1.0, 1.0]), np.diag([0.25, 4.0, 1.0]))}
    Wr = rng.normal(size=(2, H))
    P = model.Weights(gain=lambda l: np.ones(H), router=lambda l: Wr, bias=lambda l: np.zeros(2),
                      gate_up=lambda l, e: diag[e][:2], down=lambda l, e: diag[e][2])
    x = rng.normal(size=(5, H))
    out = model.moe_layer(x, 0, P, E=2, k=2, S=0, eps=0.0, dtype="f32")
    for t in range(5):
        a = x[t] / math.sqrt(np.mean(x[t] ** 2))
        z = Wr @ a
        p = np.exp(z - z.max()); p /= p.sum()
        for n in range(H):
            o = [diag[e][2][n, n] * _silu_scalar(diag[e][0][n, n] * a[n]) * diag[e][1][n, n] * a[n]
                 for e in range(2)]
            assert out.x_out[t, n] == pytest.approx(x[t, n] + p[0] * o[0] + p[1] * o[1], rel=1e-12)


def test_run_plain_counts_and_loads():
    rng = np.random.default_rng(10)
    L, H, F, E, S, k, T, N, D = 3, 8, 8, 8, 1, 2, 20, 3, 4
    P, *_ = _rand_weights(L, H, F, E, S, rng)
    run = model.run_plain(rng.normal(size=(N, T, H)), P, L=L, E=E, k=k, S=S, D=D,
                          eps=1e-6, dtype="bf16")
    assert run.counts.sum(axis=-1).tolist() == [[T * k] * L] * N
    assert run.loads.sum(axis=-1).tolist() == [[T * k] * L] * N
    for j in range(N):
        for l in range(L):
            assert np.array_equal(run.counts[j, l], np.bincount(run.idx[j, l].ravel(), minlength=E))
    # layers run in order: x after layer l is the layer-l output of x before it
    out = model.moe_layer(run.x[1, 2], 1, P, E=E, k=k, S=S, eps=1e-6, dtype="bf16")
    assert np.array_equal(out.x_out, run.x[2, 2])


def test_router_logits_bias_closed_form():
    """One nonzero per router row: z[t, e] = c_e * a[t, p_e] + b_e, so a dropped,
    negated, scaled or misindexed bias term (or a transposed router) changes z."""
    rng = np.random.default_rng(11)
    T, H, E = 6, 10, 7
    Wg, pick, c = _selection(E, H, rng)
    b = rng.normal(size=E) * 3.0
    a = rng.normal(size=(T, H))
    z = model.router_logits(a, Wg, b)
    assert z.shape == (T, E)
    for t in range(T):
        for e in range(E):
            assert z[t, e] == pytest.approx(c[e] * a[t, pick[e]] + b[e], rel=1e-15, abs=1e-15)
    # a zero router leaves exactly the bias, in expert order, for every token
    z0 = model.router_logits(a, np.zeros((E, H)), b)
    assert np.array_equal(z0, np.broadcast_to(b, (T, E)))


def test_routing_decided_by_the_bias_alone():
    """Equal router rows give every expert the same a.Wg term, so the bias alone
    orders the experts (Section 2.1: W, I = topk(G(h'))): the picks are the
    experts of largest bias for every token, ties to the lower id, and the
    weights are the softmax of the bias (a common shift cancels)."""
    rng = np.random.default_rng(12)
    T, H, E, k = 9, 16, 6, 3
    row = rng.normal(size=H)
    b = np.array([0.5, 2.0, -1.0, 2.0, 1.5, -3.0])      # experts 1 and 3 tie
    P = model.Weights(gain=lambda l: np.ones(H), router=lambda l: np.tile(row, (E, 1)),
                      bias=lambda l: b, gate_up=None, down=None)
    x = rng.normal(size=(T, H))
    a, z, idx, w, counts = model.route(x, 0, P, k=k, eps=1e-6, dtype="f32")
    want = [1, 3, 4]                                    # 2.0 (id 1), 2.0 (id 3), 1.5
    assert idx.tolist() == [want] * T
    ez = [math.exp(v - 2.0) for v in b]
    for t in range(T):
        for r, e in enumerate(want):
            assert w[t, r] == pytest.approx(ez[e] / sum(ez), rel=1e-12)
    assert counts.tolist() == [0, T, 0, T, T, 0]
    # with the bias dropped every expert ties and the picks would be 0, 1, 2
    _, _, idx0, _, _ = model.route(x, 0, model.Weights(P.gain, P.router, lambda l: np.zeros(E),
                                                       None, None), k=k, eps=1e-6, dtype="f32")
    assert idx0.tolist() == [[0, 1, 2]] * T


def test_topk_nan_logits_rank_last_and_stay_distinct():
    """NaN logits sort after every number (stable argsort of -z), so a token
    whose remaining logits are all NaN takes the lowest ids not yet picked and
    its k picks are always distinct experts."""
    z = np.array([[np.nan, 1.0, np.nan, -np.inf, np.nan],
                  [np.nan] * 5,
                  [-np.inf, -np.inf, np.nan, 0.0, np.nan]])
    idx = model.topk_indices(z, 4)
    assert idx.tolist() == [[1, 3, 0, 2], [0, 1, 2, 3], [3, 0, 1, 2]]
    assert all(len(set(r)) == 4 for r in idx.tolist())


def test_placed_device_loads_hand_worked():
    """E = 3 on D = 2: expert 0 on both devices, 1 on device 0, 2 on device 1.
    Counts (5, 2, 4): expert 0 splits 3 + 2 (the first copy takes the odd
    pair), so device 0 carries 3 + 2 = 5 and device 1 carries 2 + 4 = 6."""
    got = model.placed_device_loads(np.array([5, 2, 4]), [[0, 1], [0], [1]], 2)
    assert got.tolist() == [5, 6]
    # three copies of 7 pairs: 3, 2, 2
    got = model.placed_device_loads(np.array([7, 0]), [[0, 2, 3], [1]], 4)
    assert got.tolist() == [3, 0, 2, 2]


def test_placed_device_loads_reduces_to_contiguous_blocks_and_brute_force():
    rng = np.random.default_rng(13)
    # one copy per expert at e // (E/D): the contiguous mapping exactly
    for E, D in [(8, 4), (60, 4), (64, 8), (256, 32)]:
        counts = rng.integers(0, 50, size=(3, 5, E))
        contig = [[e // (E // D)] for e in range(E)]
        assert np.array_equal(model.placed_device_loads(counts, contig, D), model.device_loads(counts, D))
    # random placements: dealing each expert's pairs one at a time round-robin
    # over its copies gives the same split; total work is conserved
    for trial in range(200):
        E, D = int(rng.integers(1, 9)), int(rng.integers(1, 6))
        copies = [sorted(rng.choice(D, size=int(rng.integers(1, D + 1)), replace=False).tolist())
                  for _ in range(E)]
        counts = rng.integers(0, 20, size=E)
        want = np.zeros(D, dtype=np.int64)
        for e in range(E):
            for p in range(int(counts[e])):
                want[copies[e][p % len(copies[e])]] += 1
        got = model.placed_device_loads(counts, copies, D)
        assert np.array_equal(got, want), (copies, counts)
        assert got.sum() == counts.sum()
