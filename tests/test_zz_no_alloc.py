"""ad_verify_step_static (the step in the library's static scratch, no caller workspace)
against ad_verify_step with a workspace: two calls in a row through the C-ABI, the second
with a smaller block, each compared bit for bit with the workspace entry point on the
same inputs (same kernels, so the results must be identical).  Outputs of the static
call start poisoned, so a call that wrote nothing cannot pass."""
import numpy as np
import pytest

from paper_2608_12703_amd import ad, synth
from paper_2608_12703_amd.configs import Config

from gpu_common import device_session

pytestmark = pytest.mark.gpu

UNIT = Config(name="unit_static", n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=1000,
              dtype="bf16", batch=5, k=5, k_min=0, frames=150, frames_min=1, kv_max=80,
              geo_p=0.3, seed=3)


def _run(cfg, params, wl, static: bool):
    sess = device_session(cfg, params, wl, want_logits=True)
    blocks = [np.concatenate([[wl.t0[b]], wl.fill_any[b]]).astype(np.int64) for b in range(wl.batch)]
    sess.prepare(blocks)
    for t in (sess.out_hidden, sess.out_logits, sess.out_margin):
        t.fill_(float("nan"))
    sess.accept_len.fill_(-7)
    sess.out_tokens.fill_(-7)
    sess.out_greedy.fill_(-7)
    if static:
        sess.step_struct.workspace = None          # ignored by the static entry point
        sess.step_struct.workspace_bytes = 0
        ad.verify_step_static(sess.model, sess.step_struct)
    else:
        ad.verify_step(sess.model, sess.step_struct)
    res = sess.results()
    kv = [sess.export_prefix(b, int(wl.n[b]) + len(blocks[b])) for b in range(wl.batch)]
    return res, kv


@pytest.mark.parametrize("batch,k", [(5, 5), (2, 2)])   # a second, smaller call
def test_static_scratch_step_equals_workspace_step(batch, k):
    cfg = UNIT.with_(batch=batch, k=k)
    params = synth.make_params(cfg)
    wl = synth.make_step_workload(cfg)
    want, kv_want = _run(cfg, params, wl, static=False)
    got, kv_got = _run(cfg, params, wl, static=True)
    assert want["err"] == 0 and got["err"] == 0
    for key in ("accept_len", "out_tokens", "greedy"):
        np.testing.assert_array_equal(got[key], want[key], err_msg=key)
    for key in ("hidden", "logits", "margin"):
        np.testing.assert_array_equal(got[key].view(np.uint32), want[key].view(np.uint32), err_msg=key)
    for b in range(batch):
        np.testing.assert_array_equal(kv_got[b].view(np.uint32), kv_want[b].view(np.uint32))
