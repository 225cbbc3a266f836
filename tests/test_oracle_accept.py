"""Pins of the oracle's greedy acceptance (Section 2.4, parallel verification
read at temperature 0): a hand-worked tree, the extreme cases, and a brute
force over every node's root path that uses the parent links instead of the
retrieve rows."""
import numpy as np
import pytest


def _tree(feo, N, k, rng, B):
    roots = rng.integers(0, 1000, B).astype(np.int32)
    ids = np.stack([np.stack([rng.choice(1000, k, replace=False) for _ in range(N)])
                    for _ in range(B)]).astype(np.int32)
    return feo.build_tree(N, k, roots, ids, np.zeros(B, np.int32))


def test_hand_worked(feo):
    # root 7; level candidates (1,2,3), (4,5,6), (8,9,10): nodes 1..9
    tr = feo.build_tree(3, 3, np.array([7], np.int32),
                        np.array([[[1, 2, 3], [4, 5, 6], [8, 9, 10]]], np.int32),
                        np.array([5], np.int32))
    nx = np.full((1, 10), -5, np.int32)
    nx[0, 0], nx[0, 1], nx[0, 4] = 1, 4, 9        # root -> 1 -> 4 -> 9 (node 8)
    out = feo.accept_greedy(3, 3, tr["tokens"], tr["retrieve"], nx)
    assert out["accept_len"][0] == 3
    assert list(tr["retrieve"][0, out["accept_path"][0]]) == [0, 1, 4, 8]
    assert list(out["accepted"][0]) == [1, 4, 9, -5]  # three drafts, then the target's token


def test_nothing_accepted(feo):
    rng = np.random.default_rng(1)
    tr = _tree(feo, 5, 8, rng, 2)
    nx = np.full((2, 41), 5000, np.int32)            # a token no node carries
    out = feo.accept_greedy(5, 8, tr["tokens"], tr["retrieve"], nx)
    np.testing.assert_array_equal(out["accept_len"], [0, 0])
    np.testing.assert_array_equal(out["accept_path"], [0, 0])  # first path on the tie
    np.testing.assert_array_equal(out["accepted"][:, 0], [5000, 5000])
    assert (out["accepted"][:, 1:] == -1).all()


def test_whole_backbone(feo):
    rng = np.random.default_rng(2)
    N, k = 7, 8
    tr = _tree(feo, N, k, rng, 1)
    par, tok = tr["parents"][0], tr["tokens"][0]
    nx = np.full((1, 1 + N * k), -1, np.int32)
    for n in range(1, 1 + N * k):
        if (n - 1) % k == 0:                           # rank-0 node of its level: the backbone
            nx[0, par[n]] = tok[n]
    nx[0, 1 + (N - 1) * k] = 12345                     # the target's token after the last one
    out = feo.accept_greedy(N, k, tr["tokens"], tr["retrieve"], nx)
    assert out["accept_len"][0] == N
    assert out["accepted"][0, N] == 12345


@pytest.mark.parametrize("N,k", [(1, 1), (2, 3), (5, 8), (7, 8), (4, 1), (3, 16)])
def test_brute_force_over_parent_paths(feo, N, k):
    rng = np.random.default_rng(100 * N + k)
    B, T = 6, 1 + N * k
    tr = _tree(feo, N, k, rng, B)
    # plant matches: for each sequence follow a random walk that matches for a
    # random number of steps, then random predictions elsewhere
    nx = rng.integers(0, 1000, (B, T)).astype(np.int32)
    for b in range(B):
        cur = 0
        for _ in range(rng.integers(0, N + 1)):
            kids = [n for n in range(T) if tr["parents"][b, n] == cur]
            if not kids:
                break
            c = kids[rng.integers(0, len(kids))]
            nx[b, cur] = tr["tokens"][b, c]
            cur = c
    out = feo.accept_greedy(N, k, tr["tokens"], tr["retrieve"], nx)
    for b in range(B):
        par, tok = tr["parents"][b], tr["tokens"][b]
        best, best_node = -1, 0
        for n in range(T):
            path = []
            cur = n
            while cur >= 0:
                path.append(cur)
                cur = par[cur]
            path = path[::-1]
            ok = all(tok[path[t]] == nx[b, path[t - 1]] for t in range(1, len(path)))
            if ok and len(path) - 1 > best:
                best, best_node = len(path) - 1, n
        assert out["accept_len"][b] == best
        path = []
        cur = best_node
        while cur >= 0:
            path.append(cur)
            cur = par[cur]
        path = path[::-1]
        want = [int(tok[n]) for n in path[1:]] + [int(nx[b, best_node])]
        want += [-1] * (N + 1 - len(want))
        assert list(out["accepted"][b]) == want
        row = tr["retrieve"][b, out["accept_path"][b]]
        assert list(row[:best + 1]) == path             # the winning row starts with that path
