"""Pins for the oracle's tree verification (CPU only).

Appendix "Tree-decoder implementation check": the target verifies all nodes of a fixed
candidate tree in one pass with a tree attention mask, and a one-branch tree reproduces
the linear decoder token for token.
* One-branch trees against linear verification (bit-identical).
* Every root-to-leaf path of an 11-node tree against linear verification of that path
  (the already pinned one-pass verify): node logits, greedy tokens, and the walk's
  accepted length = the longest path acceptance.
* Losslessness: emitted tokens and the committed cache against autoregressive decoding.
"""
import numpy as np
import pytest

from oracle import decoder as od
from paper_2608_12703_amd import synth

# an 11-node tree: root 0 with children 1, 2, 3; 1 -> 4, 5; 2 -> 6; 4 -> 7, 8; 6 -> 9; 7 -> 10
TREE = [-1, 0, 0, 0, 1, 1, 2, 4, 4, 6, 7]


def _paths(parents):
    leaves = [i for i in range(len(parents)) if i not in parents[1:]]
    out = []
    for leaf in leaves:
        p, j = [], leaf
        while j != 0:
            p.append(j)
            j = parents[j]
        out.append([0] + p[::-1])
    return out


@pytest.fixture(scope="module")
def tiny(tiny_cfg):
    cfg = tiny_cfg.with_(vocab=97, n_layers=2)
    params = synth.make_params(cfg)
    model = od.Model(cfg, params)
    cross = od.cross_kv(model, synth.make_encoder(cfg, 0, 33))
    return cfg, model, cross


def test_tree_helpers():
    assert od.tree_depths(TREE) == [0, 1, 1, 1, 2, 2, 2, 3, 3, 3, 4]
    vis = od.tree_visibility(TREE, 2)
    assert vis.shape == (11, 13) and vis[:, :2].all()
    assert np.flatnonzero(vis[10, 2:]).tolist() == [0, 1, 4, 7, 10]
    assert np.flatnonzero(vis[9, 2:]).tolist() == [0, 2, 6, 9]
    chain = [-1, 0, 1, 2]
    np.testing.assert_array_equal(od.tree_visibility(chain, 0), np.tril(np.ones((4, 4), bool)))


def test_one_branch_tree_is_linear_verification(tiny):
    cfg, model, cross = tiny
    g = np.random.default_rng(0)
    for n in (0, 5):
        st = od.new_state(model, cross, 7, synth.make_prefix_kv(cfg, 1, n))
        y, _, _ = od.ar_decode(model, st, 5)
        for drafts in ([], y[:2], y[:2] + [(y[2] + 1) % 97], list(g.integers(0, 97, 5))):
            lin = od.verify(model, st, drafts)
            tr = od.verify_tree(model, st, [7] + list(drafts), [-1] + list(range(len(drafts))))
            assert (tr.greedy, tr.accepted, tr.emitted) == (lin.greedy, lin.accepted, lin.emitted)
            assert tr.path == list(range(lin.accepted + 1))
            for (K1, V1), (K2, V2) in zip(tr.state.self_kv, lin.state.self_kv):
                np.testing.assert_array_equal(K1, K2)
                np.testing.assert_array_equal(V1, V2)


def test_tree_paths_against_linear_verification(tiny):
    cfg, model, cross = tiny
    st = od.new_state(model, cross, 11, synth.make_prefix_kv(cfg, 2, 4))
    y, _, _ = od.ar_decode(model, st, 5)
    g = np.random.default_rng(3)
    for trial in range(4):
        tokens = [11] + [int(t) for t in g.integers(0, 97, len(TREE) - 1)]
        # plant the greedy continuation along one path, to a trial-dependent depth
        path = _paths(TREE)[trial % len(_paths(TREE))]
        for j, u in enumerate(path[1:][: trial + 1]):
            tokens[u] = y[j]
        out = od.forward_block(model, st, tokens, parents=TREE)
        tr = od.verify_tree(model, st, tokens, TREE)
        best = -1
        for p in _paths(TREE):
            lin = od.forward_block(model, st, [tokens[u] for u in p])
            np.testing.assert_allclose(out.logits[p], lin.logits, rtol=0, atol=1e-11)
            lv = od.verify(model, st, [tokens[u] for u in p[1:]])
            best = max(best, lv.accepted)
        assert tr.accepted == best
        assert tr.emitted == y[: tr.accepted + 1]


def test_tree_commit_equals_autoregressive_cache(tiny):
    cfg, model, cross = tiny
    st = od.new_state(model, cross, 3, synth.make_prefix_kv(cfg, 4, 6))
    y, _, _ = od.ar_decode(model, st, 4)
    tokens = [3] + [0] * (len(TREE) - 1)
    tokens[2], tokens[6], tokens[9] = y[0], y[1], y[2]         # the greedy path 0-2-6-9
    tokens[1], tokens[3] = (y[0] + 1) % 97, (y[0] + 2) % 97
    tr = od.verify_tree(model, st, tokens, TREE)
    assert tr.path == [0, 2, 6, 9] and tr.accepted == 3 and tr.emitted == y[:4]
    _, _, st_ar = od.ar_decode(model, st, 4)
    assert tr.state.n == st_ar.n == st.n + 4 and tr.state.t0 == st_ar.t0
    for (K1, V1), (K2, V2) in zip(tr.state.self_kv, st_ar.self_kv):
        np.testing.assert_allclose(K1, K2, rtol=2 ** -7, atol=1e-12)
        np.testing.assert_allclose(V1, V2, rtol=2 ** -7, atol=1e-12)
