"""Host-only checks of libad.so: it loads, exports every entry point include/ad.h
declares, and rejects bad arguments before touching the GPU (CPU only)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ad.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ad_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def ad():
    from paper_2608_12703_amd import ad as mod
    return mod


def test_every_declared_function_is_exported(ad):
    declared = _declared()
    assert "ad_verify_step" in declared and "ad_kv_commit" in declared and "ad_draft_heads" in declared
    for name in declared:
        assert hasattr(ad.LIB, name), f"{name} declared in ad.h but not exported"
    assert sorted(ad.EXPORTS) == declared


def _tiny():
    from paper_2608_12703_amd.configs import Config
    return Config(name="t", n_layers=2, d_model=128, n_heads=2, d_ffn=256, vocab=100, dtype="bf16",
                  batch=2, k=3)


def test_param_count_and_model_validation(ad):
    cfg = _tiny()
    assert ad.param_count(cfg) == 4 + 20 * 2
    desc = ad.model_desc(cfg)
    h = ctypes.c_void_p()
    fake = (ctypes.c_void_p * 44)(*([0x1000] * 44))
    assert ad.LIB.ad_model_create(ctypes.byref(desc), fake, 43, ctypes.byref(h)) == -1
    bad = ad.model_desc(cfg.with_(d_model=100))
    assert ad.LIB.ad_model_create(ctypes.byref(bad), fake, 44, ctypes.byref(h)) == -5
    assert b"64 * n_heads" in ad.LIB.ad_last_error()
    f32 = ad.model_desc(cfg.with_(dtype="f32"))
    h32 = ctypes.c_void_p()
    assert ad.LIB.ad_model_create(ctypes.byref(f32), fake, 44, ctypes.byref(h32)) == 0
    n32 = ctypes.c_size_t()
    assert ad.LIB.ad_model_pack_size(h32, ctypes.byref(n32)) == -5
    ad.LIB.ad_model_destroy(h32)
    bad = ad.model_desc(cfg.with_(vocab=0))
    assert ad.LIB.ad_model_create(ctypes.byref(bad), fake, 44, ctypes.byref(h)) == -2
    desc.dtype = 7
    assert ad.LIB.ad_model_create(ctypes.byref(desc), fake, 44, ctypes.byref(h)) == -1
    misaligned = (ctypes.c_void_p * 44)(*([0x1000] * 43 + [0x1008]))
    assert ad.LIB.ad_model_create(ctypes.byref(ad.model_desc(cfg)), misaligned, 44, ctypes.byref(h)) == -1
    assert b"aligned" in ad.LIB.ad_last_error()
    wide = ad.model_desc(cfg.with_(d_model=64 * 65, n_heads=65))
    assert ad.LIB.ad_model_create(ctypes.byref(wide), fake, 44, ctypes.byref(h)) == -5
    nulls = (ctypes.c_void_p * 44)(*([0x1000] * 43 + [0]))
    assert ad.LIB.ad_model_create(ctypes.byref(ad.model_desc(cfg)), nulls, 44, ctypes.byref(h)) == -1
    assert ad.LIB.ad_model_create(ctypes.byref(ad.model_desc(cfg)), fake, 44, ctypes.byref(h)) == 0
    n = ctypes.c_size_t()
    assert ad.LIB.ad_model_pack_size(h, ctypes.byref(n)) == 0
    # per layer 7 tiled matrices (QKV, O, cross-Q, cross-O, FFN up and down, encoder K/V),
    # then the LM head: N rounded up to 128 columns
    want = 2 * (2 * (384 * 128 + 128 * 128 * 3 + 256 * 128 + 128 * 256 + 256 * 128) + 128 * 128)
    assert n.value == want
    assert ad.LIB.ad_model_pack(h, 0x1008, n.value, None) == -1      # misaligned
    assert ad.LIB.ad_model_pack(h, 0x1000, n.value - 1, None) == -3  # too small
    assert ad.LIB.ad_model_pack(h, None, 0, None) == 0               # back to row-major
    assert ad.LIB.ad_workspace_size(h, 8, 2, 3, ctypes.byref(n)) == 0 and n.value > 0
    assert ad.LIB.ad_workspace_size(h, 0, 2, 3, ctypes.byref(n)) == -2
    assert ad.LIB.ad_workspace_size(h, 8, 2, -1, ctypes.byref(n)) == -2
    ad.LIB.ad_model_destroy(h)


def _step(ad, **over):
    kv = ad.KV(0x1000, 56, 28, 0x1000, 0x1000)
    cross = ad.Cross(0x1000, 1504 * 2, 0x1000, 0x1000)
    s = ad.Step(2, ad.AD_PADDED, 3, 8, 0x1000, 0x1000, None, kv, cross, 0x1000, 0x1000, None, None,
                None, None, 0x1000, 0x1000, 1 << 40, -1, None, None, None, None,
                (ctypes.c_int32 * 3)(-1, -1, -1), None, None, None, None)
    for k, v in over.items():
        setattr(s, k, v)
    return s


def test_verify_step_rejects_before_enqueue(ad):
    cfg = _tiny()
    fake = (ctypes.c_void_p * 44)(*([0x1000] * 44))
    h = ctypes.c_void_p()
    assert ad.LIB.ad_model_create(ctypes.byref(ad.model_desc(cfg)), fake, 44, ctypes.byref(h)) == 0
    run = lambda s: ad.LIB.ad_verify_step(h, ctypes.byref(s), None)
    assert run(_step(ad, tokens=None)) == -1
    assert run(_step(ad, layout=5)) == -1
    assert run(_step(ad, layout=ad.AD_PACKED)) == -1               # packed without cu_rows
    assert run(_step(ad, batch=0)) == -2
    assert run(_step(ad, k_max=448)) == -2
    assert run(_step(ad, rows=7)) == -2                             # padded rows != B (k_max+1)
    assert run(_step(ad, layout=ad.AD_PACKED, cu_rows=0x1000, rows=9)) == -2
    s = _step(ad)
    s.cross.frames_cap = 20
    assert run(s) == -2
    assert run(_step(ad, anchor_layer=-2)) == -2
    assert run(_step(ad, anchor_layer=cfg.n_layers)) == -2
    assert run(_step(ad, anchor_layer=0)) == -1                     # readout without out_anchor
    assert run(_step(ad, tap_layers=(ctypes.c_int32 * 3)(-1, -1, cfg.n_layers))) == -2
    assert run(_step(ad, tap_layers=(ctypes.c_int32 * 3)(0, -1, -1))) == -1   # taps without out_taps
    assert run(_step(ad, k_max=64, rows=130)) == -5                 # 64-bit row masks: k_max <= 63
    assert run(_step(ad, parents=0x1000)) == -1                     # a tree without out_path
    assert run(_step(ad, out_xq=0x1000)) == -1                      # out_xq without anchor_layer
    # the AnchorDraft objective: argument checks before anything is enqueued
    lw = ctypes.c_size_t()
    assert ad.LIB.ad_anchordraft_loss_workspace_size(h, 2, 5, ctypes.byref(lw)) == 0
    assert ad.LIB.ad_anchordraft_loss_workspace_size(h, 0, 5, ctypes.byref(lw)) == -2
    cr = ad.Cross(0x1000, 1504 * 2, 0x1000, 0x1000)
    loss = lambda **o: ad.LIB.ad_anchordraft_loss(
        h, ctypes.byref(o.get("cross", cr)), o.get("layer", 0), o.get("batch", 2), 5,
        o.get("xq", 0x1000), o.get("center", 0x1000), o.get("sigma", 5.0), o.get("lam", 0.1),
        o.get("logits", None), o.get("targets", None), o.get("feat", None), None, 0x1000,
        None, o.get("dxq", None), None, None, 0x1000, o.get("wsp", 0x1000), o.get("ws", lw.value), None)
    assert loss(center=None) == -1                                  # xq without centres
    assert loss(logits=0x1000) == -1                                # logits without targets
    assert loss(feat=0x1000, targets=0x1000) == -1                  # feat without feat_target
    assert loss(xq=None, dxq=0x1000) == -1                          # a query gradient without xq
    assert loss(batch=0) == -2 and loss(layer=cfg.n_layers) == -2
    assert loss(sigma=0.0) == -2 and loss(lam=-1.0) == -2
    assert loss(ws=lw.value - 1) == -3
    assert loss(wsp=0x1010) == -1                                   # misaligned workspace
    ws = ctypes.c_size_t()
    assert ad.LIB.ad_draft_input_workspace_size(h, 2, ctypes.byref(ws)) == 0
    assert ws.value >= 7 * cfg.d_model * 2 * 4
    di = lambda **o: ad.LIB.ad_draft_input(
        h, o.get("w_fuse", 0x1000), 0x1000, 0x1000, 0x1000, o.get("batch", 2), o.get("taps", 0x1000),
        0x1000, o.get("layout", ad.AD_PADDED), 3, None, 0x1000, o.get("rows", 8), None, 0x1000,
        o.get("stride", 4), 0x1000, o.get("anchor", None), 0x1000, o.get("half", 20), 0x1000,
        0x1000, o.get("wsp", 0x1000), o.get("ws", ws.value), None)
    assert di(w_fuse=None) == -1
    assert di(layout=7) == -1
    assert di(layout=ad.AD_PACKED) == -1                            # packed without cu_rows
    assert di(taps=None) == -1                                      # neither taps nor feature
    assert di(batch=0) == -2 and di(stride=0) == -2 and di(rows=1) == -2
    assert di(anchor=0x1000, half=-1) == -2
    assert di(ws=ws.value - 1) == -3
    assert di(wsp=0x1010) == -1                                     # misaligned workspace
    assert run(_step(ad, workspace_bytes=100)) == -3
    assert b"workspace" in ad.LIB.ad_last_error()
    assert run(_step(ad, workspace=0x1010)) == -1                   # misaligned workspace
    assert b"aligned" in ad.LIB.ad_last_error()
    assert run(_step(ad, in_rows=0x1004)) == -1                     # misaligned input rows
    assert b"aligned" in ad.LIB.ad_last_error()
    assert ad.LIB.ad_kv_commit(None, None, 2, None) == -1
    assert ad.LIB.ad_kv_commit(0x1000, 0x1000, 0, None) == -2
    kv = ad.KV(0x1000, 56, 28, 0x1000, 0x1000)
    assert ad.LIB.ad_kv_commit_tree(h, ctypes.byref(kv), 0x1000, None, 4, 2, None) == -1
    assert ad.LIB.ad_kv_commit_tree(h, ctypes.byref(kv), 0x1000, 0x1000, 4, 0, None) == -2
    assert ad.LIB.ad_kv_commit_tree(h, ctypes.byref(kv), 0x1000, 0x1000, 0, 2, None) == -2
    assert ad.LIB.ad_kv_import(h, ctypes.byref(kv), 0, 0x1000, 449, 0x1000, None) == -2
    assert ad.LIB.ad_kv_export(h, ctypes.byref(kv), -1, 0x1000, 3, 0x1000, None) == -2
    cross = ad.Cross(0x1000, 17, 0x1000, 0x1000)
    assert ad.LIB.ad_cross_kv_prefill(h, 0x1000, ctypes.byref(cross), None) == -2
    # encoder states inside the last layer's slots (its prefill scratch) are refused
    cross = ad.Cross(0x100000, 64, 0x1000, 0x1000)
    last = 0x100000 + (cfg.n_layers - 1) * 2 * cfg.n_heads * 64 * 64 * 2
    assert ad.LIB.ad_cross_kv_prefill(h, last + 256, ctypes.byref(cross), None) == -1
    assert b"overlaps" in ad.LIB.ad_last_error()
    ws = ctypes.c_size_t()
    assert ad.LIB.ad_draft_heads_workspace_size(h, 4, 1, ctypes.byref(ws)) == 0
    assert ad.LIB.ad_draft_heads(h, 0x1000, 4, 0x1000, 0, 4, None, 0x1000, 0x1000, 1, 0x1000,
                                 0x1000, ws.value - 1, None) == -3
    assert ad.LIB.ad_draft_heads(h, 0x1000, 0, 0x1000, 0, 4, None, 0x1000, 0x1000, 1, 0x1000,
                                 0x1000, ws.value, None) == -2
    assert ad.LIB.ad_draft_heads(h, 0x1000, 4, 0x1000, 0, 4, None, 0x1000, 0x1000, 1, 0x1000,
                                 0x1010, ws.value, None) == -1      # misaligned workspace
    ad.LIB.ad_model_destroy(h)


def test_static_scratch_step_rejects_a_step_past_its_size(ad):
    """ad_verify_step_static refuses a step whose scratch exceeds its static buffer
    (the ragged batch of 64 at the large-v3 shape needs about 120 MiB) before anything is
    enqueued, with a message naming the buffer."""
    from paper_2608_12703_amd.configs import CONFIGS
    cfg = CONFIGS["ragged_large_v3"]
    n = ad.param_count(cfg)
    fake = (ctypes.c_void_p * n)(*[256 * (i + 1) for i in range(n)])   # never dereferenced
    h = ctypes.c_void_p()
    assert ad.LIB.ad_model_create(ctypes.byref(ad.model_desc(cfg)), fake, n, ctypes.byref(h)) == 0
    need = ctypes.c_size_t()
    assert ad.LIB.ad_workspace_size(h, 576, 64, 8, ctypes.byref(need)) == 0
    assert need.value > 64 << 20
    step = ad.Step()
    step.batch, step.layout, step.k_max, step.rows = 64, ad.AD_PADDED, 8, 576
    assert ad.LIB.ad_verify_step_static(h, ctypes.byref(step), None) == -3
    assert b"static scratch" in ad.LIB.ad_last_error()
    assert ad.LIB.ad_verify_step_static(None, ctypes.byref(step), None) == -1
    ad.LIB.ad_model_destroy(h)
