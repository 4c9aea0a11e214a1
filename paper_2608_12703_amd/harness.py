"""Device buffers of one batch of sequences, driven through the C-ABI.

A Session owns (through torch) everything a verify step reads and writes: parameters,
the paged self-KV pool and its block table, the encoder K/V, the step's token block and
outputs, and the workspace.  It only moves data and calls libad entry points.
"""
from __future__ import annotations

import ctypes

import numpy as np
import torch

from . import ad, synth
from .configs import MAX_FRAMES, MAX_POS, PAGE, Config


def _ceil32(x: int) -> int:
    """Encoder slots are allotted in 32-frame blocks."""
    return (x + 31) // 32 * 32


def torch_dtype(cfg: Config):
    return torch.bfloat16 if cfg.dtype == "bf16" else torch.float32


def upload(a: np.ndarray, dtype, device="cuda") -> torch.Tensor:
    """Host float32 array -> device tensor of `dtype` (exact for bf16-representable values)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dtype).to(device)


def upload_params(cfg: Config, params: dict, device="cuda") -> list:
    dt = torch_dtype(cfg)
    return [upload(params[name], dt, device) for name, _ in synth.param_specs(cfg)]


class Session:
    def __init__(self, cfg: Config, params, batch: int, k_max: int, frames, *,
                 layout: int = ad.AD_PADDED, packed_encoder: bool = False,
                 page_seed: int | None = 0, want_logits: bool = False, device: str = "cuda",
                 extra_pages: int = 0, pack_weights: bool = True, max_frames: int = MAX_FRAMES):
        self.cfg, self.B, self.k_max, self.layout = cfg, batch, k_max, layout
        self.device = device
        self.dt = torch_dtype(cfg)
        L, d, H = cfg.n_layers, cfg.d_model, cfg.n_heads
        self.params = params if isinstance(params, list) else upload_params(cfg, params, device)
        self.model = ad.Model(cfg, self.params, max_frames=max_frames)
        if pack_weights and cfg.dtype == "bf16":   # tiled weights for the matrix-core GEMMs
            self.model.pack(torch.empty(self.model.pack_size(), dtype=torch.uint8, device=device))
        i32 = dict(dtype=torch.int32, device=device)

        # paged self-KV: every sequence may reach the last position
        self.pages_per_seq = (cfg.max_pos + PAGE - 1) // PAGE
        self.num_pages = batch * self.pages_per_seq + extra_pages
        order = np.arange(self.num_pages)
        if page_seed is not None:
            order = np.random.default_rng(page_seed).permutation(self.num_pages)
        table = order[: batch * self.pages_per_seq].reshape(batch, self.pages_per_seq)
        self.block_table = torch.tensor(table, **i32)
        self.pool = torch.empty(L * 2 * self.num_pages * H * PAGE * 64, dtype=self.dt, device=device)
        self.kv_len = torch.zeros(batch, **i32)

        # encoder K/V slots
        frames = [int(t) for t in frames]
        assert len(frames) == batch and all(1 <= t <= max_frames for t in frames)
        self.frames = frames
        if packed_encoder:
            off = np.concatenate([[0], np.cumsum([_ceil32(t) for t in frames])])
        else:
            tmax = _ceil32(max(frames))
            off = np.arange(batch + 1) * tmax
        self.frames_cap = int(off[-1])
        self.enc_off = torch.tensor(off[:-1], **i32)
        self.enc_len = torch.tensor(frames, **i32)
        self.cross = torch.empty(L * 2 * H * self.frames_cap * 64, dtype=self.dt, device=device)

        # step outputs and workspace (sized for the padded row count)
        self.max_rows = batch * (k_max + 1)
        self.accept_len = torch.zeros(batch, **i32)
        self.out_tokens = torch.zeros(batch, k_max + 1, **i32)
        self.out_greedy = torch.zeros(self.max_rows, **i32)
        self.out_hidden = torch.zeros(self.max_rows, d, dtype=torch.float32, device=device)
        self.out_margin = torch.zeros(self.max_rows, dtype=torch.float32, device=device)
        self.out_logits = (torch.zeros(self.max_rows, cfg.vocab, dtype=torch.float32, device=device)
                           if want_logits else None)
        self.err_flag = torch.zeros(1, **i32)
        # verification-attention anchor readout (anchor_layer -1: off)
        self.anchor_layer = -1
        self.out_anchor = torch.full((batch,), -1, **i32)
        self.out_anchor_peak = torch.zeros(batch, dtype=torch.float32, device=device)
        # draft-block use: input rows replacing the token embedding, a per-sequence
        # cross-attention window, and residual taps (tap_layers -1: none)
        self.in_rows = None
        self.cross_window = None
        self.tap_layers = (-1, -1, -1)
        self.out_taps = None
        # draft trees: per-row parents of the current block (None: chains) and the path
        self.parents = None
        self.out_xq = None      # anchor_layer's cross-attention queries [rows][d] (optional)
        self.out_path = torch.full((batch, k_max + 1), -1, **i32)
        self.workspace = torch.empty(self.model.workspace_size(self.max_rows, batch, k_max),
                                     dtype=torch.uint8, device=device)
        self.step_struct = None

    # ------------------------------------------------------------------ structs
    def kv_struct(self) -> ad.KV:
        return ad.KV(self.pool.data_ptr(), self.num_pages, self.pages_per_seq,
                     self.kv_len.data_ptr(), self.block_table.data_ptr())

    def cross_struct(self) -> ad.Cross:
        return ad.Cross(self.cross.data_ptr(), self.frames_cap, self.enc_len.data_ptr(),
                        self.enc_off.data_ptr())

    # ------------------------------------------------------------------ setup
    def upload_encoder(self, encs) -> torch.Tensor:
        """Encoder states (list of [T_b, d] arrays) in the session's encoder slots."""
        enc = torch.zeros(self.frames_cap, self.cfg.d_model, dtype=self.dt, device=self.device)
        offs = self.enc_off.cpu().numpy()
        for b, e in enumerate(encs):
            enc[offs[b]: offs[b] + len(e)] = upload(e, self.dt, self.device)
        return enc

    def prefill_encoder(self, encs):
        """Upload encoder states (list of [T_b, d] arrays) and build the encoder K/V."""
        enc = self.upload_encoder(encs)
        ad.cross_kv_prefill(self.model, enc, self.cross_struct())
        del enc

    def import_prefix(self, b: int, kv: np.ndarray):
        """Committed prefix of sequence b from a [L, 2, n, H, 64] array."""
        n = kv.shape[2]
        src = upload(kv, self.dt, self.device) if n else None
        ad.kv_import(self.model, self.kv_struct(), b, src, n, self.err_flag)

    def export_prefix(self, b: int, n: int) -> np.ndarray:
        """Positions 0..n-1 of sequence b as a float32 [L, 2, n, H, 64] array."""
        cfg = self.cfg
        dst = torch.empty(cfg.n_layers, 2, n, cfg.n_heads, 64, dtype=self.dt, device=self.device)
        ad.kv_export(self.model, self.kv_struct(), b, dst, n, self.err_flag)
        torch.cuda.synchronize()
        return dst.float().cpu().numpy()

    def set_kv_len(self, n):
        self.kv_len.copy_(torch.tensor(np.asarray(n), dtype=torch.int32))

    # ------------------------------------------------------------------ step
    def prepare(self, blocks, layout: int | None = None, parents=None):
        """Upload the token blocks ([t0, d_1..d_k] per sequence) and build the step struct.
        parents: per sequence, the parent row of each block row (entry 0 ignored) for a
        draft-tree step, or None for chains."""
        layout = self.layout if layout is None else layout
        ks = [len(b) - 1 for b in blocks]
        assert len(blocks) == self.B and max(ks) <= self.k_max
        i32 = dict(dtype=torch.int32, device=self.device)
        if layout == ad.AD_PADDED:
            tok = np.zeros((self.B, self.k_max + 1), np.int64)
            for b, blk in enumerate(blocks):
                tok[b, : len(blk)] = blk
            tok = tok.reshape(-1)
            cu = None
            if parents is not None:
                par = np.full((self.B, self.k_max + 1), -1, np.int64)
                for b, p in enumerate(parents):
                    par[b, : len(p)] = p
                par = par.reshape(-1)
        else:
            tok = np.concatenate([np.asarray(b, np.int64) for b in blocks])
            cu = torch.tensor(np.concatenate([[0], np.cumsum([k + 1 for k in ks])]), **i32)
            if parents is not None:
                par = np.concatenate([np.asarray(p, np.int64) for p in parents])
        self.parents = None if parents is None else torch.tensor(par, **i32)
        self.tokens = torch.tensor(tok, **i32)
        self.k = torch.tensor(ks, **i32)
        self.cu_rows = cu
        self.rows = len(tok)
        self.step_struct = ad.Step(
            self.B, layout, self.k_max, self.rows, self.tokens.data_ptr(), self.k.data_ptr(),
            ad.ptr(cu), self.kv_struct(), self.cross_struct(), self.accept_len.data_ptr(),
            self.out_tokens.data_ptr(), self.out_greedy.data_ptr(), ad.ptr(self.out_logits),
            self.out_hidden.data_ptr(), self.out_margin.data_ptr(), self.err_flag.data_ptr(),
            self.workspace.data_ptr(), self.workspace.numel(), int(self.anchor_layer),
            self.out_anchor.data_ptr(), self.out_anchor_peak.data_ptr(), ad.ptr(self.in_rows),
            ad.ptr(self.cross_window), (ctypes.c_int32 * 3)(*self.tap_layers), ad.ptr(self.out_taps),
            ad.ptr(self.parents), self.out_path.data_ptr(), ad.ptr(self.out_xq))
        self.cur_layout = layout
        return self.step_struct

    def run(self):
        ad.verify_step(self.model, self.step_struct)

    def commit(self):
        if self.parents is not None:
            ad.kv_commit_tree(self.model, self.kv_struct(), self.accept_len, self.out_path,
                              self.k_max + 1, self.B)
        else:
            ad.kv_commit(self.kv_len, self.accept_len, self.B)

    def step(self, blocks, layout: int | None = None, commit: bool = False, parents=None):
        self.prepare(blocks, layout, parents)
        self.run()
        if commit:
            self.commit()

    # ------------------------------------------------------------------ results
    def row_of(self, b: int, i: int) -> int:
        if self.cur_layout == ad.AD_PADDED:
            return b * (self.k_max + 1) + i
        return int(self.cu_rows[b].item()) + i

    def results(self, keys=None) -> dict:
        """The step's outputs on the host; keys limits the copies to the named ones (a
        decode loop needs only accept_len, out_tokens and err)."""
        torch.cuda.synchronize()
        if keys is not None:
            src = {"accept_len": self.accept_len, "out_tokens": self.out_tokens,
                   "kv_len": self.kv_len, "greedy": self.out_greedy[: self.rows]}
            out = {k: src[k].cpu().numpy() for k in keys if k != "err"}
            if "err" in keys:
                out["err"] = int(self.err_flag.item())
            return out
        out = {"accept_len": self.accept_len.cpu().numpy(),
               "out_tokens": self.out_tokens.cpu().numpy(),
               "greedy": self.out_greedy[: self.rows].cpu().numpy(),
               "hidden": self.out_hidden[: self.rows].cpu().numpy(),
               "margin": self.out_margin[: self.rows].cpu().numpy(),
               "kv_len": self.kv_len.cpu().numpy(),
               "err": int(self.err_flag.item())}
        if self.out_logits is not None:
            out["logits"] = self.out_logits[: self.rows].cpu().numpy()
        if self.parents is not None:
            out["path"] = self.out_path.cpu().numpy()
        if self.anchor_layer >= 0:
            out["anchor"] = self.out_anchor.cpu().numpy()
            out["anchor_peak"] = self.out_anchor_peak.cpu().numpy()
        return out
