"""Pins of oracle.permute: brute force on tiny steps (Python's stable ``sorted``
on (key, enumeration index)), and the invariants a stable grouping must hold."""
import numpy as np

from oracle import permute


def _brute(run, E, S):
    pairs = []
    q = 0
    for rho, (layer, idx) in enumerate(run):
        for t in range(idx.shape[0]):
            slots = list(idx[t]) + [E + s for s in range(S)]
            for e in slots:
                pairs.append((layer * (E + S) + int(e), q))
                q += 1
    order = [qq for _, qq in sorted(pairs)]        # key, then enumeration index
    return [k for k, _ in pairs], order


def test_permutation_matches_brute_force():
    rng = np.random.default_rng(20)
    for trial in range(200):
        E = int(rng.integers(1, 9))
        k = int(rng.integers(1, E + 1))
        S = int(rng.integers(0, 3))
        L = int(rng.integers(1, 5))
        run = []
        for _ in range(int(rng.integers(1, 5))):
            T = int(rng.integers(0, 6))
            idx = np.array([rng.choice(E, size=k, replace=False) for _ in range(T)],
                           dtype=np.int64).reshape(T, k)
            run.append((int(rng.integers(0, L)), idx))
        keys = permute.step_keys(run, E, S)
        bkeys, border = _brute(run, E, S)
        assert keys.tolist() == bkeys
        perm, inv, offsets = permute.stable_permutation(keys, L * (E + S))
        assert perm.tolist() == border
        assert np.array_equal(perm[inv], np.arange(keys.size))
        assert offsets[0] == 0 and offsets[-1] == keys.size
        for key in range(L * (E + S)):
            seg = perm[offsets[key]:offsets[key + 1]]
            assert np.all(keys[seg] == key) and np.all(np.diff(seg) > 0)


def test_source_rows():
    run = [(0, np.array([[1, 2], [0, 3]])), (2, np.array([[3, 0]]))]
    src = permute.source_rows(run, S=1)
    assert src.tolist() == [[0, 0]] * 3 + [[0, 1]] * 3 + [[1, 0]] * 3
