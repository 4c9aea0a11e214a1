"""Audio-conditioned draft step (test infrastructure only).

Sources: section 3, paragraph "Models and Protocol" (an EAGLE-3 style drafter that
predicts tokens directly from features of several target layers, extended so that
every draft step also attends to the frozen encoder output); appendix "Draft
architecture" (the drafter's input mixes four target feature vectors with the embedding
of the current token and feeds a single causal decoder block made of self-attention,
audio cross-attention and a feed-forward sublayer); appendix "Window geometry" (when the
audio attention is restricted, it covers 400 ms on each side of its centre).

The paper fixes the shape, not the wiring; the readings used here:
* The four target representations are the residual stream after target layers L/4,
  L/2 and 3L/4 (tap_layers) and the target's final LayerNorm output, all at block row
  a_b, the last verified position.
* At a round's first draft step the feature is f = W_fuse [r1; r2; r3; h] + b_fuse; every
  later step uses the draft block's own output of the previous step (EAGLE-3).
* The block's input u = W_in [f; E_tok[t]] + b_in replaces the token embedding; the
  position embedding of the step's index within the round is added.  The draft's
  self-attention spans the current round's steps: its cache restarts every round.
* The block is a pre-LN decoder layer of the target's form with its own final
  LayerNorm, whose output feeds the target's tied LM head (d = argmax of the
  float32-rounded logits, lowest index) and is the next step's feature.
* Cross-attention uses the draft's own key/value projection of the encoder states,
  restricted to frames c - 20 .. c + 20 around the anchor c (20 ms per encoder frame, so
  400 ms is 20 frames), clipped to the audio.  The first token fed is the round's
  pending token (the bonus token of the verification), at step index 0.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import decoder as od
from .numerics import round_f32

HALF_WINDOW = 20   # frames: 400 ms at 20 ms per encoder frame


def tap_layers(n_layers: int):
    """Target layers whose output residual stream the draft reads (L/4, L/2, 3L/4)."""
    return [max(0, n_layers * i // 4 - 1) for i in (1, 2, 3)]


def window(center: int, T: int, half: int = HALF_WINDOW):
    """Frames [lo, hi) within half frames of the centre, clipped to 0..T-1."""
    return max(0, center - half), min(T, center + half + 1)


def block_model(dcfg, target_params: dict, draft_params: dict, kv_dtype: str | None = None) -> od.Model:
    """The draft block as a one-layer decoder: its own layer and final LayerNorm, the
    target's token (LM head) and position tables.  Its caches are stored like the
    target's (kv_dtype defaults to the model dtype)."""
    p = dict(draft_params)
    p["tok_emb"], p["pos_emb"] = target_params["tok_emb"], target_params["pos_emb"]
    return od.Model(dcfg, p, kv_dtype)


def fuse(draft_params: dict, taps3: np.ndarray, hidden: np.ndarray) -> np.ndarray:
    """f = W_fuse [r1; r2; r3; h] + b_fuse."""
    z = np.concatenate([np.asarray(taps3, np.float64).reshape(-1), np.asarray(hidden, np.float64)])
    return np.asarray(draft_params["w_fuse"], np.float64) @ z + np.asarray(draft_params["b_fuse"], np.float64)


def block_input(draft_params: dict, tok_emb, feature: np.ndarray, token: int) -> np.ndarray:
    """u = W_in [f; E_tok[t]] + b_in."""
    z = np.concatenate([np.asarray(feature, np.float64), np.asarray(tok_emb[int(token)], np.float64)])
    return np.asarray(draft_params["w_in"], np.float64) @ z + np.asarray(draft_params["b_in"], np.float64)


@dataclass
class DraftRound:
    drafts: list        # d_1..d_K
    margins: list       # top-1 minus top-2 of each step's float32-rounded logits
    hidden: list        # each step's output feature [d]
    inputs: list        # each step's block input u [d]


def draft_round(bmodel: od.Model, draft_params: dict, dcross, taps3, hidden, token: int,
                anchor: int, T: int, K: int) -> DraftRound:
    """K draft steps from the pending token, conditioned on the target's representations
    at the last verified row and on the audio around the anchor frame."""
    state = od.new_state(bmodel, dcross, int(token))
    lo, hi = window(int(anchor), int(T))
    f = fuse(draft_params, taps3, hidden)
    t = int(token)
    out = DraftRound([], [], [], [])
    for _ in range(K):
        u = block_input(draft_params, bmodel.params["tok_emb"], f, t)
        blk = od.forward_block(bmodel, state, [t], in_rows=u[None], cross_window=(lo, hi))
        logits = round_f32(blk.logits[0])
        d = od.argmax_lowest(logits)
        out.drafts.append(d)
        out.margins.append(od.top2_margin(logits))
        out.hidden.append(blk.hidden[0])
        out.inputs.append(u)
        state = od.commit(state, blk, 0, d)
        f, t = blk.hidden[0], d
    return out
