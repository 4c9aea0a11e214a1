"""ctypes binding over libad.so (the C-ABI declared in include/ad.h).

Argument marshalling only: every computation of the verify step runs in the library's
HIP kernels.  torch supplies device memory and the current stream.  Importing this
module loads the library; a missing library is an error, never a fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libad.so")

AD_F32, AD_BF16 = 0, 1
AD_PADDED, AD_PACKED = 0, 1
AD_ERR_LENGTH, AD_ERR_PAGE, AD_ERR_TOKEN, AD_ERR_FRAMES, AD_ERR_NONFINITE = 1, 2, 4, 8, 16
AD_ERR_TREE = 32
STATUS = {0: "AD_OK", -1: "AD_EINVAL", -2: "AD_ERANGE", -3: "AD_ENOSPACE", -4: "AD_EHIP",
          -5: "AD_EUNSUPPORTED"}

_i32 = ctypes.c_int32
_ptr = ctypes.c_void_p
_size = ctypes.c_size_t


class ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", _i32), ("d_model", _i32), ("n_heads", _i32), ("d_ffn", _i32),
                ("vocab", _i32), ("max_pos", _i32), ("max_frames", _i32), ("dtype", _i32)]


class KV(ctypes.Structure):
    _fields_ = [("pool", _ptr), ("num_pages", _i32), ("pages_per_seq", _i32),
                ("kv_len", _ptr), ("block_table", _ptr)]


class Cross(ctypes.Structure):
    _fields_ = [("data", _ptr), ("frames_cap", _i32), ("enc_len", _ptr), ("enc_off", _ptr)]


class Step(ctypes.Structure):
    _fields_ = [("batch", _i32), ("layout", _i32), ("k_max", _i32), ("rows", _i32),
                ("tokens", _ptr), ("k", _ptr), ("cu_rows", _ptr), ("kv", KV), ("cross", Cross),
                ("accept_len", _ptr), ("out_tokens", _ptr), ("out_greedy", _ptr),
                ("out_logits", _ptr), ("out_hidden", _ptr), ("out_margin", _ptr),
                ("err_flag", _ptr), ("workspace", _ptr), ("workspace_bytes", _size),
                ("anchor_layer", _i32), ("out_anchor", _ptr), ("out_anchor_peak", _ptr),
                ("in_rows", _ptr), ("cross_window", _ptr), ("tap_layers", _i32 * 3),
                ("out_taps", _ptr), ("parents", _ptr), ("out_path", _ptr),
                ("out_xq", _ptr)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run paper_2608_12703_amd.build.build()")
    lib = ctypes.CDLL(LIB_PATH)
    sig = {
        "ad_last_error": (ctypes.c_char_p, []),
        "ad_model_param_count": (_i32, [ctypes.POINTER(ModelDesc)]),
        "ad_model_create": (_i32, [ctypes.POINTER(ModelDesc), ctypes.POINTER(_ptr), _i32,
                                   ctypes.POINTER(_ptr)]),
        "ad_model_destroy": (_i32, [_ptr]),
        "ad_model_pack_size": (_i32, [_ptr, ctypes.POINTER(_size)]),
        "ad_model_pack": (_i32, [_ptr, _ptr, _size, _ptr]),
        "ad_workspace_size": (_i32, [_ptr, _i32, _i32, _i32, ctypes.POINTER(_size)]),
        "ad_cross_kv_prefill": (_i32, [_ptr, _ptr, ctypes.POINTER(Cross), _ptr]),
        "ad_verify_step": (_i32, [_ptr, ctypes.POINTER(Step), _ptr]),
        "ad_verify_step_static": (_i32, [_ptr, ctypes.POINTER(Step), _ptr]),
        "ad_kv_commit": (_i32, [_ptr, _ptr, _i32, _ptr]),
        "ad_kv_commit_tree": (_i32, [_ptr, _ptr, _ptr, _ptr, _i32, _i32, _ptr]),
        "ad_anchordraft_loss_workspace_size": (_i32, [_ptr, _i32, _i32, ctypes.POINTER(_size)]),
        "ad_anchordraft_loss": (_i32, [_ptr, _ptr, _i32, _i32, _i32, _ptr, _ptr, ctypes.c_float,
                                       ctypes.c_float, _ptr, _ptr, _ptr, _ptr, _ptr, _ptr, _ptr,
                                       _ptr, _ptr, _ptr, _ptr, _size, _ptr]),
        "ad_draft_heads_workspace_size": (_i32, [_ptr, _i32, _i32, ctypes.POINTER(_size)]),
        "ad_draft_heads": (_i32, [_ptr, _ptr, _i32, _ptr, _i32, _i32, _ptr, _ptr, _ptr, _i32,
                                  _ptr, _ptr, _size, _ptr]),
        "ad_kv_import": (_i32, [_ptr, ctypes.POINTER(KV), _i32, _ptr, _i32, _ptr, _ptr]),
        "ad_draft_input_workspace_size": (_i32, [_ptr, _i32, ctypes.POINTER(_size)]),
        "ad_draft_input": (_i32, [_ptr, _ptr, _ptr, _ptr, _ptr, _i32, _ptr, _ptr, _i32, _i32, _ptr,
                                  _ptr, _i32, _ptr, _ptr, _i32, _ptr, _ptr, _ptr, _i32, _ptr, _ptr,
                                  _ptr, _size, _ptr]),
        "ad_kv_export": (_i32, [_ptr, ctypes.POINTER(KV), _i32, _ptr, _i32, _ptr, _ptr]),
        "ad_profile_enable": (_i32, [_ptr, _i32, _i32]),
        "ad_profile_read": (_i32, [_ptr, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_i32)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


LIB = _load()
EXPORTS = ("ad_last_error", "ad_model_param_count", "ad_model_create", "ad_model_destroy",
           "ad_model_pack_size", "ad_model_pack",
           "ad_workspace_size", "ad_cross_kv_prefill", "ad_verify_step", "ad_verify_step_static",
           "ad_kv_commit", "ad_kv_commit_tree",
           "ad_draft_heads_workspace_size", "ad_draft_heads", "ad_kv_import", "ad_kv_export",
           "ad_draft_input_workspace_size", "ad_draft_input",
           "ad_anchordraft_loss_workspace_size", "ad_anchordraft_loss",
           "ad_profile_enable", "ad_profile_read")
PROF_CROSS_ATTN, PROF_SELF_ATTN, PROF_GEMM, PROF_LM_HEAD, PROF_XQ_CROSS, PROF_XQ, PROF_ANCHOR = 1, 2, 3, 4, 5, 6, 7


class ADError(RuntimeError):
    def __init__(self, what: str, status: int):
        self.status = status
        msg = LIB.ad_last_error().decode()
        super().__init__(f"{what}: {STATUS.get(status, status)}: {msg}")


def check(status: int, what: str):
    if status != 0:
        raise ADError(what, status)


def ptr(t) -> int | None:
    """Device address of a tensor (None for None)."""
    return None if t is None else t.data_ptr()


def stream_handle(stream=None) -> int:
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def model_desc(cfg, max_pos=448, max_frames=1500) -> ModelDesc:
    return ModelDesc(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.d_ffn, cfg.vocab, max_pos,
                     max_frames, AD_BF16 if cfg.dtype == "bf16" else AD_F32)


def param_count(cfg) -> int:
    return LIB.ad_model_param_count(ctypes.byref(model_desc(cfg)))


class Model:
    """A model handle over caller-owned device parameters (kept alive here)."""

    def __init__(self, cfg, params: list, max_frames: int = 1500):
        self.cfg = cfg
        self.params = params
        self.desc = model_desc(cfg, max_pos=cfg.max_pos, max_frames=max_frames)
        arr = (_ptr * len(params))(*[p.data_ptr() for p in params])
        h = _ptr()
        check(LIB.ad_model_create(ctypes.byref(self.desc), arr, len(params), ctypes.byref(h)),
              "ad_model_create")
        self.handle = h

    def workspace_size(self, rows: int, batch: int, k_max: int) -> int:
        n = _size()
        check(LIB.ad_workspace_size(self.handle, rows, batch, k_max, ctypes.byref(n)),
              "ad_workspace_size")
        return n.value

    def pack_size(self) -> int:
        n = _size()
        check(LIB.ad_model_pack_size(self.handle, ctypes.byref(n)), "ad_model_pack_size")
        return n.value

    def pack(self, buffer, stream=None):
        """Tile the weights into `buffer` (a device tensor of at least pack_size() bytes,
        kept alive here), or return to the row-major parameters with buffer=None."""
        check(LIB.ad_model_pack(self.handle, ptr(buffer), 0 if buffer is None else
                                buffer.numel() * buffer.element_size(), stream_handle(stream)),
              "ad_model_pack")
        self.packed = buffer

    def draft_heads_workspace_size(self, n_heads: int, batch: int) -> int:
        n = _size()
        check(LIB.ad_draft_heads_workspace_size(self.handle, n_heads, batch, ctypes.byref(n)),
              "ad_draft_heads_workspace_size")
        return n.value

    def close(self):
        if getattr(self, "handle", None):
            LIB.ad_model_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def cross_kv_prefill(model: Model, enc, cross: Cross, stream=None):
    check(LIB.ad_cross_kv_prefill(model.handle, ptr(enc), ctypes.byref(cross),
                                  stream_handle(stream)), "ad_cross_kv_prefill")


def verify_step(model: Model, step: Step, stream=None):
    check(LIB.ad_verify_step(model.handle, ctypes.byref(step), stream_handle(stream)),
          "ad_verify_step")


def verify_step_static(model: Model, step: Step, stream=None):
    """ad_verify_step in the library's static scratch (step.workspace is ignored)."""
    check(LIB.ad_verify_step_static(model.handle, ctypes.byref(step), stream_handle(stream)),
          "ad_verify_step_static")


def kv_commit(kv_len, accept_len, batch: int, stream=None):
    check(LIB.ad_kv_commit(ptr(kv_len), ptr(accept_len), batch, stream_handle(stream)),
          "ad_kv_commit")


def kv_commit_tree(model: Model, kv: KV, accept_len, path, path_stride: int, batch: int,
                   stream=None):
    check(LIB.ad_kv_commit_tree(model.handle, ctypes.byref(kv), ptr(accept_len), ptr(path),
                                path_stride, batch, stream_handle(stream)), "ad_kv_commit_tree")


def anchordraft_loss_workspace_size(model: Model, batch: int, rows_per_seq: int) -> int:
    n = _size()
    check(LIB.ad_anchordraft_loss_workspace_size(model.handle, batch, rows_per_seq, ctypes.byref(n)),
          "ad_anchordraft_loss_workspace_size")
    return n.value


def anchordraft_loss(model: Model, cross, layer: int, batch: int, rows_per_seq: int, xq, center,
                     sigma: float, lam: float, logits, targets, feat, feat_target, out_terms,
                     out_row, out_dxq, out_dlogits, out_dfeat, err_flag, workspace, stream=None):
    """The AnchorDraft objective (ad.h: ad_anchordraft_loss); cross is a Cross struct or
    None, array arguments are device tensors or None."""
    check(LIB.ad_anchordraft_loss(
        model.handle, None if cross is None else ctypes.byref(cross), layer, batch, rows_per_seq,
        ptr(xq), ptr(center), sigma, lam, ptr(logits), ptr(targets), ptr(feat), ptr(feat_target),
        ptr(out_terms), ptr(out_row), ptr(out_dxq), ptr(out_dlogits), ptr(out_dfeat), ptr(err_flag),
        ptr(workspace), 0 if workspace is None else workspace.numel() * workspace.element_size(),
        stream_handle(stream)), "ad_anchordraft_loss")


def draft_heads(model: Model, heads_w, n_heads: int, hidden, layout: int, k_max: int, cu_rows,
                accept_len, out_tokens, batch: int, next_tokens, workspace, stream=None):
    check(LIB.ad_draft_heads(model.handle, ptr(heads_w), n_heads, ptr(hidden), layout, k_max,
                             ptr(cu_rows), ptr(accept_len), ptr(out_tokens), batch,
                             ptr(next_tokens), ptr(workspace), workspace.numel(),
                             stream_handle(stream)), "ad_draft_heads")


def draft_input_workspace_size(model: Model, batch: int) -> int:
    n = _size()
    check(LIB.ad_draft_input_workspace_size(model.handle, batch, ctypes.byref(n)),
          "ad_draft_input_workspace_size")
    return n.value


def draft_input(model: Model, w_fuse, b_fuse, w_in, b_in, batch: int, taps, hidden, layout: int,
                k_max: int, cu_rows, accept_len, rows: int, feature, tokens, token_stride: int,
                token_index, anchor, enc_len, half_window: int, window, out, workspace, stream=None):
    check(LIB.ad_draft_input(model.handle, ptr(w_fuse), ptr(b_fuse), ptr(w_in), ptr(b_in), batch,
                             ptr(taps), ptr(hidden), layout, k_max, ptr(cu_rows), ptr(accept_len),
                             rows, ptr(feature), ptr(tokens), token_stride, ptr(token_index),
                             ptr(anchor), ptr(enc_len), half_window, ptr(window), ptr(out),
                             ptr(workspace), workspace.numel(), stream_handle(stream)),
          "ad_draft_input")


def kv_import(model: Model, kv: KV, b: int, src, n: int, err_flag, stream=None):
    check(LIB.ad_kv_import(model.handle, ctypes.byref(kv), b, ptr(src), n, ptr(err_flag),
                           stream_handle(stream)), "ad_kv_import")


def kv_export(model: Model, kv: KV, b: int, dst, n: int, err_flag, stream=None):
    check(LIB.ad_kv_export(model.handle, ctypes.byref(kv), b, ptr(dst), n, ptr(err_flag),
                           stream_handle(stream)), "ad_kv_export")


def profile_enable(model: Model, kernel: int, max_launches: int):
    check(LIB.ad_profile_enable(model.handle, kernel, max_launches), "ad_profile_enable")


def profile_read(model: Model):
    """(summed milliseconds, number of timed launches) since the last read."""
    t, n = ctypes.c_double(), _i32()
    check(LIB.ad_profile_read(model.handle, ctypes.byref(t), ctypes.byref(n)), "ad_profile_read")
    return t.value, n.value
