"""GPU parity of draft-tree verification against the oracle.

Paper, appendix "Tree-decoder implementation check": every node of a candidate tree is
verified in one target pass under a tree attention mask, and a one-branch tree
reproduces the linear decoder token for token.  The step places node i at position
n + depth(i) with its keys / values at slot n + i, walks the tree from the root, and
ad_kv_commit_tree moves the accepted path's keys / values to slots n .. n + a.
* A chain given as a tree is bit-identical to the linear step (every output, the cache,
  the commit).
* Trees of 1 to 40 nodes (several 16-row query groups, nodes whose ancestors lie in an
  earlier group) against the oracle's tree pass: node logits, greedy tokens, the walk,
  the anchor at the path's last node, the written cache; the commit's moves are byte
  work, checked bit-exact.
* Lossless decoding with trees (including a decoy sibling that shadows the right one)
  against autoregressive decoding on the GPU.
* Bad parents, and the packed layout against the padded one.
* The bench's tree step at the large-v3 shape (the 11-node tree at all 32 sequences),
  one planted sequence against the oracle.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as od
from paper_2608_12703_amd import ad, synth
from paper_2608_12703_amd.configs import Config
from paper_2608_12703_amd.harness import Session

from gpu_common import (LOGIT_TOL, MARGIN_EXCLUDE, compare_anchor, device_session, kv_close,
                        kv_report, layer_input_errors, oracle_model, oracle_state, step_taps)

pytestmark = pytest.mark.gpu

UNIT = Config(name="unit_tree", n_layers=3, d_model=128, n_heads=2, d_ffn=256, vocab=1000,
              dtype="bf16", batch=5, k=4, k_min=0, frames=300, frames_min=40, kv_max=60,
              geo_p=0.3, seed=9)
ANCHOR_LAYER = 1
# an 11-node tree: root 0 with children 1, 2, 3; 1 -> 4, 5; 2 -> 6; 4 -> 7, 8; 6 -> 9; 7 -> 10
TREE = [-1, 0, 0, 0, 1, 1, 2, 4, 4, 6, 7]


def random_tree(rng, r):
    """Parents of an r-node tree: each node continues its predecessor half of the time,
    else hangs from a uniformly chosen earlier node."""
    return [-1] + [int(i - 1 if rng.random() < 0.5 else rng.integers(0, i)) for i in range(1, r)]


def path_to(parents, leaf):
    p = [leaf]
    while p[-1] != 0:
        p.append(parents[p[-1]])
    return p[::-1]


def tree_blocks(cfg, model, wl, trees, rng):
    """Tokens per sequence: the greedy continuation planted along the path to the tree's
    last node, to a depth that varies with the sequence; random tokens elsewhere."""
    blocks = []
    for b, par in enumerate(trees):
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        tok = [int(wl.t0[b])] + [int(t) for t in rng.integers(0, cfg.vocab, len(par) - 1)]
        path = path_to(par, len(par) - 1)
        if len(path) > 1:
            y, _, _ = od.ar_decode(model, st, len(path) - 1)
            for j, u in enumerate(path[1:][: 1 + b % len(path)]):
                tok[u] = y[j]
        blocks.append(np.array(tok, np.int64))
    return blocks


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_chain_as_tree_is_bit_identical_to_linear(dtype):
    cfg = UNIT.with_(dtype=dtype)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]).astype(np.int64) for b in range(wl.batch)]
    model = oracle_model(cfg, params)
    for b in (0, 2):      # plant the greedy continuation in two sequences
        st = oracle_state(cfg, model, b, int(wl.n[b]), int(wl.T[b]), int(wl.t0[b]))
        y, _, _ = od.ar_decode(model, st, len(blocks[b]) - 1)
        blocks[b][1:] = y
    out = []
    for tree in (False, True):
        s = device_session(cfg, params, wl)
        s.anchor_layer = ANCHOR_LAYER
        par = [[-1] + list(range(len(blk) - 1)) for blk in blocks] if tree else None
        s.step(blocks, parents=par)
        res = s.results()
        kv = [s.export_prefix(b, int(wl.n[b]) + len(blocks[b])) for b in range(wl.batch)]
        s.commit()
        res_c = s.results()
        kv_c = [s.export_prefix(b, int(res_c["kv_len"][b])) for b in range(wl.batch)]
        out.append((res, kv, res_c, kv_c))
    (r0, kv0, c0, kc0), (r1, kv1, c1, kc1) = out
    assert r0["err"] == 0 and r1["err"] == 0
    print(f"  accept {r0['accept_len'].tolist()}")
    for key in ("accept_len", "out_tokens", "anchor"):
        np.testing.assert_array_equal(r0[key], r1[key])
    np.testing.assert_array_equal(r0["anchor_peak"].view(np.uint32), r1["anchor_peak"].view(np.uint32))
    # every row of every block (padding rows past a sequence's block hold no result)
    rows = [b * (wl.k.max() + 1) + i for b in range(wl.batch) for i in range(len(blocks[b]))]
    np.testing.assert_array_equal(r0["greedy"][rows], r1["greedy"][rows])
    for key in ("logits", "hidden", "margin"):
        np.testing.assert_array_equal(r0[key][rows].view(np.uint32), r1[key][rows].view(np.uint32))
    for b in range(wl.batch):
        a = int(r1["accept_len"][b])
        assert r1["path"][b][: a + 1].tolist() == list(range(a + 1))
        assert np.all(r1["path"][b][a + 1:] == -1)
        np.testing.assert_array_equal(kv0[b].view(np.uint32), kv1[b].view(np.uint32))
        np.testing.assert_array_equal(kc0[b].view(np.uint32), kc1[b].view(np.uint32))
    np.testing.assert_array_equal(c0["kv_len"], c1["kv_len"])


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_tree_step_and_commit_match_oracle(dtype):
    cfg = UNIT.with_(dtype=dtype)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    rng = np.random.default_rng(11)
    trees = [TREE, random_tree(rng, 40), [-1], random_tree(rng, 17), [-1, 0, 1, 2, 3]]
    blocks = tree_blocks(cfg, model, wl, trees, rng)
    sess = device_session(cfg, params, wl, k_max=max(len(t) for t in trees) - 1)
    sess.anchor_layer = ANCHOR_LAYER
    sess.step(blocks, parents=trees)
    res = sess.results()
    assert res["err"] == 0
    gpu_taps = step_taps(sess, blocks, parents=trees)
    kv_pre = [sess.export_prefix(b, int(wl.n[b]) + len(trees[b])) for b in range(wl.batch)]
    sess.commit()
    res_c = sess.results()
    compared = 0
    for b, par in enumerate(trees):
        n, r = int(wl.n[b]), len(par)
        st = oracle_state(cfg, model, b, n, int(wl.T[b]), int(wl.t0[b]))
        out = od.forward_block(model, st, blocks[b], parents=par, probe_layer=ANCHOR_LAYER,
                               taps=list(range(cfg.n_layers - 1)))
        ref = od.verify_tree(model, st, blocks[b], par)
        rows = [sess.row_of(b, i) for i in range(r)]
        err = float(np.max(np.abs(res["logits"][rows] - out.logits)))
        print(f"  seq {b}: {r} nodes, depth {max(od.tree_depths(par))}, path {ref.path}, "
              f"gpu path {res['path'][b][: int(res['accept_len'][b]) + 1].tolist()}, logit error {err:.2e}")
        assert err <= LOGIT_TOL[dtype]
        g = res["greedy"][rows]
        for i in range(r):
            if ref.margins[i] >= MARGIN_EXCLUDE:
                assert g[i] == ref.greedy[i], f"seq {b} node {i}"
        # the cache the step wrote: node i at slot n + i
        eps = layer_input_errors(gpu_taps, out.taps, rows, cfg.n_layers)
        for layer, (kb, vb) in enumerate(out.new_kv):
            kv_close(kv_pre[b][layer, 0, n:], kb, f"seq {b} layer {layer} K", dtype, layer, eps[layer])
            kv_close(kv_pre[b][layer, 1, n:], vb, f"seq {b} layer {layer} V", dtype, layer, eps[layer])
        a = int(res["accept_len"][b])
        path = res["path"][b][: a + 1].tolist()
        # the walk reads the greedy tokens at the path's nodes
        if all(ref.margins[u] >= MARGIN_EXCLUDE for u in ref.path):
            assert path == ref.path and a == ref.accepted
            assert res["out_tokens"][b][: a + 1].tolist() == ref.emitted
            assert np.all(res["out_tokens"][b][a + 1:] == -1) and np.all(res["path"][b][a + 1:] == -1)
            compare_anchor(cfg, res, b, ref, od.anchor_of(out.xattn[ref.path[-1]]))
            compared += 1
        # the commit: path node j's slot moved to n + j, byte for byte; the length
        assert int(res_c["kv_len"][b]) == n + a + 1
        kv_post = sess.export_prefix(b, n + a + 1)
        np.testing.assert_array_equal(kv_post[:, :, n:].view(np.uint32),
                                      kv_pre[b][:, :, [n + u for u in path]].view(np.uint32))
        np.testing.assert_array_equal(kv_post[:, :, :n].view(np.uint32), kv_pre[b][:, :, :n].view(np.uint32))
        assert res["out_tokens"][b][: a + 1].tolist() == [int(g[u]) for u in path]
    assert compared >= wl.batch - 1


def test_tree_decoding_is_lossless():
    cfg = UNIT.with_(kv_max=0)
    params = synth.make_params(cfg)
    B, T, n_tokens, k_max = 3, 250, 30, 14
    encs = [synth.make_encoder(cfg, b, T) for b in range(B)]

    def session():
        s = Session(cfg, params, B, k_max, [T] * B)
        s.prefill_encoder(encs)
        s.set_kv_len(np.zeros(B, np.int64))
        return s

    start = 17
    ar = session()
    ref = [[] for _ in range(B)]
    pend = [start] * B
    for _ in range(n_tokens + k_max):
        ar.step([np.array([p], np.int64) for p in pend], commit=True)
        r = ar.results()
        for b in range(B):
            pend[b] = int(r["out_tokens"][b][0])
            ref[b].append(pend[b])
    # trees built from the true continuation: a right chain of random length, a wrong
    # sibling, sometimes a decoy with the right token (lower index) and a wrong child
    rng = np.random.default_rng(5)
    tr = session()
    got = [[] for _ in range(B)]
    pend = [start] * B
    rounds = 0
    while min(len(g) for g in got) < n_tokens:
        blocks, parents = [], []
        for b in range(B):
            fut = ref[b][len(got[b]):]      # (past the reference: a root alone)
            tok, par = [pend[b]], [-1]
            if len(fut) >= 2:
                if rng.random() < 0.5:
                    tok += [fut[0], (fut[1] + 1) % cfg.vocab]
                    par += [0, 1]
                tok.append((fut[0] + 3) % cfg.vocab)
                par.append(0)
            prev = 0
            for j in range(min(int(rng.integers(0, 8)), len(fut) if len(fut) >= 2 else 0)):
                tok.append(fut[j])
                par.append(prev)
                prev = len(tok) - 1
            blocks.append(np.array(tok, np.int64))
            parents.append(par)
        tr.step(blocks, parents=parents, commit=True)
        r = tr.results()
        assert r["err"] == 0
        for b in range(B):
            a = int(r["accept_len"][b])
            em = r["out_tokens"][b][: a + 1].tolist()
            got[b] += em
            pend[b] = em[-1]
        rounds += 1
    print(f"[tree loop] {rounds} rounds for {n_tokens} tokens per sequence")
    for b in range(B):
        assert got[b][:n_tokens] == ref[b][:n_tokens]
    assert rounds < n_tokens
    torch.cuda.synchronize()


def test_bad_parents_skip_only_their_sequence_and_packed_trees_agree():
    cfg = UNIT
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    rng = np.random.default_rng(4)
    trees = [TREE, random_tree(rng, 9), [-1, 0, 1], random_tree(rng, 14), [-1, 0, 0, 1]]
    blocks = tree_blocks(cfg, model, wl, trees, rng)
    k_max = max(len(t) for t in trees) - 1
    # the same trees in the padded and the packed layout: identical results
    out = {}
    for layout in (ad.AD_PADDED, ad.AD_PACKED):
        s = device_session(cfg, params, wl, layout=layout, k_max=k_max)
        s.step(blocks, parents=trees)
        r = s.results()
        assert r["err"] == 0
        rows = [s.row_of(b, i) for b in range(wl.batch) for i in range(len(trees[b]))]
        out[layout] = (r, rows, [s.export_prefix(b, int(wl.n[b]) + len(trees[b])) for b in range(wl.batch)])
    (rp, rowp, kvp), (rk, rowk, kvk) = out[ad.AD_PADDED], out[ad.AD_PACKED]
    for key in ("accept_len", "out_tokens", "path"):
        np.testing.assert_array_equal(rp[key], rk[key])
    np.testing.assert_array_equal(rp["logits"][rowp].view(np.uint32), rk["logits"][rowk].view(np.uint32))
    for b in range(wl.batch):
        np.testing.assert_array_equal(kvp[b].view(np.uint32), kvk[b].view(np.uint32))
    # a parent that is not an earlier row: AD_ERR_TREE, that sequence skipped, others unchanged
    bad = [list(t) for t in trees]
    bad[1][3] = 3                                  # its own row
    bad[3][5] = 9                                  # a later row
    s = device_session(cfg, params, wl, k_max=k_max)
    s.step(blocks, parents=bad)
    r = s.results()
    assert r["err"] == ad.AD_ERR_TREE
    assert r["accept_len"][1] == -1 and r["accept_len"][3] == -1
    assert np.all(r["out_tokens"][[1, 3]] == -1) and np.all(r["path"][[1, 3]] == -1)
    for b in (0, 2, 4):
        assert r["accept_len"][b] == rp["accept_len"][b]
        np.testing.assert_array_equal(r["path"][b], rp["path"][b])
        rows = [s.row_of(b, i) for i in range(len(trees[b]))]
        np.testing.assert_array_equal(r["logits"][rows].view(np.uint32),
                                      rp["logits"][[rowp[sum(len(t) for t in trees[:b]) + i]
                                                    for i in range(len(trees[b]))]].view(np.uint32))


def test_large_v3_tree_step_sampled():
    """The bench's tree step (the 11-node tree at every sequence of the large-v3 batch,
    anchor at three quarters of the depth) with one sequence planted and checked against
    the oracle's tree pass: node logits, greedy tokens, the walk, the anchor, the written
    cache of every layer, and the commit's moves."""
    from paper_2608_12703_amd.configs import CONFIGS
    cfg = CONFIGS["large_v3_bf16"]
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    model = oracle_model(cfg, params)
    b_s = int(np.argmax(wl.n))
    n = int(wl.n[b_s])
    st = oracle_state(cfg, model, b_s, n, int(wl.T[b_s]), int(wl.t0[b_s]))
    y, _, _ = od.ar_decode(model, st, 3)
    blocks = []
    for b in range(wl.batch):
        fill = list(wl.fill_any[b]) * 2
        tok = [int(wl.t0[b])] + [int(t) for t in fill[: len(TREE) - 1]]
        if b == b_s:
            for j, u in enumerate((1, 4, 7)):        # the greedy continuation along 0-1-4-7
                tok[u] = y[j]
        blocks.append(np.array(tok, np.int64))
    layer = 3 * cfg.n_layers // 4
    sess = device_session(cfg, params, wl, k_max=len(TREE) - 1)
    sess.anchor_layer = layer
    sess.step(blocks, parents=[TREE] * wl.batch)
    res = sess.results()
    assert res["err"] == 0
    gpu_taps = step_taps(sess, blocks, parents=[TREE] * wl.batch)
    kv_pre = sess.export_prefix(b_s, n + len(TREE))
    sess.commit()
    res_c = sess.results()
    out = od.forward_block(model, st, blocks[b_s], parents=TREE, probe_layer=layer,
                           taps=list(range(cfg.n_layers - 1)))
    ref = od.verify_tree(model, st, blocks[b_s], TREE)
    rows = [sess.row_of(b_s, i) for i in range(len(TREE))]
    err = float(np.max(np.abs(res["logits"][rows] - out.logits)))
    print(f"  seq {b_s}: n={n}, path {ref.path}, gpu path "
          f"{res['path'][b_s][: int(res['accept_len'][b_s]) + 1].tolist()}, logit error {err:.2e}")
    assert err <= LOGIT_TOL["bf16"]
    for i in range(len(TREE)):
        if ref.margins[i] >= MARGIN_EXCLUDE:
            assert res["greedy"][rows[i]] == ref.greedy[i]
    eps = layer_input_errors(gpu_taps, out.taps, rows, cfg.n_layers)
    for lay, (kb, vb) in enumerate(out.new_kv):
        kv_close(kv_pre[lay, 0, n:], kb, f"layer {lay} K", "bf16", lay, eps[lay])
        kv_close(kv_pre[lay, 1, n:], vb, f"layer {lay} V", "bf16", lay, eps[lay])
    kv_report("tree large-v3")
    assert all(ref.margins[u] >= MARGIN_EXCLUDE for u in ref.path)
    a = int(res["accept_len"][b_s])
    path = res["path"][b_s][: a + 1].tolist()
    assert path == ref.path and a == ref.accepted >= 3
    assert res["out_tokens"][b_s][: a + 1].tolist() == ref.emitted
    compare_anchor(cfg, res, b_s, ref, od.anchor_of(out.xattn[ref.path[-1]]))
    kv_post = sess.export_prefix(b_s, n + a + 1)
    np.testing.assert_array_equal(kv_post[:, :, n:].view(np.uint32),
                                  kv_pre[:, :, [n + u for u in path]].view(np.uint32))
    assert int(res_c["kv_len"][b_s]) == n + a + 1
