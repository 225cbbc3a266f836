"""Structural checks of a Backbone Expansion tree (Section 2.2), shared by the
oracle pins and the GPU parity tests.  Pure properties: nothing here builds a
tree."""
import numpy as np


def check_tree(tr, b, N, k, root, topk_ids, P):
    T, NL = 1 + N * k, N * (k - 1) + 1
    tok, par, dep, pos = (tr[x][b] for x in ("tokens", "parents", "depth", "positions"))
    mask, ret = tr["mask"][b], tr["retrieve"][b]
    assert tok.shape == (T,) and mask.shape == (T, T) and ret.shape == (NL, N + 1)
    assert tok[0] == root and par[0] == -1 and dep[0] == 0
    levels = [[n for n in range(T) if dep[n] == l] for l in range(N + 1)]
    assert [len(x) for x in levels] == [1] + [k] * N
    backbone = [0]
    for l in range(1, N + 1):
        nodes = levels[l]
        assert len({int(par[n]) for n in nodes}) == 1          # one parent per level
        assert par[nodes[0]] == backbone[-1]                   # ... the previous backbone node
        assert list(tok[nodes]) == list(topk_ids[l - 1])       # rank order within the level
        backbone.append(nodes[0])                              # most probable extends the backbone
    for n in range(1, T):
        assert dep[n] == dep[par[n]] + 1
        assert par[n] in backbone                              # side branches are leaves
    assert (pos == P + dep).all()
    # exactly one backbone path of length N: the nodes with children form it
    has_child = np.zeros(T, bool)
    has_child[par[1:]] = True
    assert sorted(np.nonzero(has_child)[0].tolist()) == backbone[:-1]
    # ancestor-or-self mask
    assert (mask.sum(1) == dep + 1).all()
    for a in range(T):
        assert mask[a, a] == 1
        for c in range(T):
            if c != a:
                assert mask[a, c] == (mask[par[a], c] if par[a] >= 0 else 0)
    # root->leaf paths of every leaf, in node order
    leaves = [n for n in range(T) if not has_child[n]]
    assert len(leaves) == NL
    for r, leaf in enumerate(leaves):
        path = [int(x) for x in ret[r] if x >= 0]
        assert (ret[r][len(path):] == -1).all()
        assert path[0] == 0 and path[-1] == leaf and len(path) == dep[leaf] + 1
        for u, v in zip(path, path[1:]):
            assert par[v] == u
    if k == 1:
        assert (mask == np.tril(np.ones((T, T), np.uint8))).all()
