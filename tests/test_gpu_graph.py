"""The verify step and its commit captured into a HIP graph (torch.cuda.CUDAGraph over the
C-ABI calls) and replayed several times, with the program's own eager work and
synchronisations between the replays (the caller restores the committed length,
poisons the outputs and runs unrelated kernels).  Every replay must give the eager
step's results bit for bit: accept lengths, tokens, greedy tokens, logits, hidden rows,
margins, the committed lengths and the cache bytes the step writes."""
import numpy as np
import pytest
import torch

from paper_2608_12703_amd import synth
from paper_2608_12703_amd.configs import Config

from gpu_common import device_session

pytestmark = pytest.mark.gpu

UNIT = Config(name="unit_graph", n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=1000,
              dtype="bf16", batch=5, k=5, k_min=0, frames=150, frames_min=1, kv_max=80,
              geo_p=0.3, seed=3)


def _snapshot(sess, wl, blocks):
    r = sess.results()
    kv = [sess.export_prefix(b, int(wl.n[b]) + len(blocks[b])) for b in range(wl.batch)]
    return r, kv


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_step_graph_replays_equal_the_eager_step(dtype):
    cfg = UNIT.with_(dtype=dtype)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    sess = device_session(cfg, params, wl, want_logits=True)
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]).astype(np.int64) for b in range(wl.batch)]
    sess.prepare(blocks)
    kv0 = sess.kv_len.clone()
    outs = (sess.out_hidden, sess.out_logits, sess.out_margin)

    def poison():
        for t in outs:
            t.fill_(float("nan"))
        sess.accept_len.fill_(-7)
        sess.out_tokens.fill_(-7)
        sess.out_greedy.fill_(-7)
        sess.kv_len.copy_(kv0)

    poison()
    sess.run()
    sess.commit()
    want, kv_want = _snapshot(sess, wl, blocks)
    assert want["err"] == 0
    np.testing.assert_array_equal(want["kv_len"], wl.n + want["accept_len"] + 1)

    poison()
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sess.run()
        sess.commit()
    scratch = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        poison()
        scratch.mul_(1.0001).add_(0.5)          # the program's own eager work in between
        torch.cuda.synchronize()
        graph.replay()
        got, kv_got = _snapshot(sess, wl, blocks)
        assert got["err"] == 0
        for key in ("accept_len", "out_tokens", "greedy", "kv_len"):
            np.testing.assert_array_equal(got[key], want[key], err_msg=f"replay {rep}: {key}")
        for key in ("hidden", "logits", "margin"):
            np.testing.assert_array_equal(got[key].view(np.uint32), want[key].view(np.uint32),
                                          err_msg=f"replay {rep}: {key}")
        for b in range(wl.batch):
            np.testing.assert_array_equal(kv_got[b].view(np.uint32), kv_want[b].view(np.uint32))
    del graph
