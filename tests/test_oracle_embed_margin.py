"""Pins of the oracle's Embed step and of the top-2 margin behind the near-tie window.

Embed (Alg. 1, Eq. (1)): a packed row is either an embedding-table row selected by its token
id (the instruction tokens of a prefill, the fed-back token of a decode stage) or a row given
by the caller (the vision rows).  The HF decoder looks ids up in its own ``nn.Embedding``, so
running it on ``input_ids`` pins the oracle's lookup without going through
``OracleModel.embed``; a hand-built three-row table pins the id / given-row selection.

top2_margin: the gap between the largest and the second-largest logit of a row, which sets
the window inside which two greedy tokens may legitimately differ.  Pinned by hand values
and by a brute-force loop.

Planted mistakes (a swapped selection, a table indexed by packed row instead of token id, an
off-by-one in the margin) must each break a pin.
"""
import numpy as np
import pytest
import torch

import oracle
import workload as wl
from oracle.pipeline import sequential_generate, top2_margin
from tests.helpers import oracle_model, tiny_prefill_fn
from tests.test_oracle_model import MAX_POS, SHAPE, _hf_model

L_P = 32


@pytest.fixture(scope="module")
def weights():
    return wl.model_weights(SHAPE, seed=0, random_gains=True)


# ----------------------------------------------------------------------------- embed
HAND_SHAPE = wl.ModelShape(n_layers=0, d_model=2, n_heads=1, head_dim=2, d_ff=2, vocab=3, dtype="f32")
HAND_TABLE = np.array([[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]])


def _hand_check(storage):
    """ids (2, -1, 0, 1, -1) over the table rows (1,2), (3,4), (5,6) and given rows; the
    given rows at id positions are decoys that must not show up."""
    model = oracle.OracleModel(HAND_SHAPE, {"embed": HAND_TABLE, "final_norm": np.ones(2),
                                            "lm_head": HAND_TABLE}, [], storage=storage)
    ids = np.array([2, -1, 0, 1, -1])
    given = np.array([[9.0, 9.0], [7.0, 8.0], [-9.0, 9.0], [9.0, -9.0], [0.5, -0.25]])
    want = np.array([[5.0, 6.0], [7.0, 8.0], [1.0, 2.0], [3.0, 4.0], [0.5, -0.25]])
    got = model.embed(ids, given)
    return got.shape == want.shape and np.array_equal(got, want)


def _hf_ids_check(model, weights, n_tokens=4):
    """Max |oracle - HF| over the logits of every generated position, for an all-id prompt
    (HF looks the ids up itself) and for a prompt of 8 given rows + 24 ids (HF looks the 24
    ids up with its own embedding module and takes the 8 rows as given)."""
    hf = _hf_model(weights)
    worst = 0.0
    # all-id prompt
    fn = tiny_prefill_fn(SHAPE, L_P, seed=3)
    ids, emb = fn(0)
    assert np.all(ids >= 0)
    seq = sequential_generate(model, ids, emb, n_tokens)
    all_ids = torch.from_numpy(np.concatenate([ids, seq["tokens"][:-1]]))[None]
    with torch.no_grad():
        z = hf(input_ids=all_ids).logits[0, L_P - 1:].numpy()
    worst = max(worst, float(np.abs(z - seq["logits"]).max()))
    # given rows followed by ids
    fn = tiny_prefill_fn(SHAPE, L_P, seed=4, n_vision=8)
    ids, emb = fn(1)
    seq = sequential_generate(model, ids, emb, n_tokens)
    text = torch.from_numpy(np.concatenate([ids[8:], seq["tokens"][:-1]]))
    with torch.no_grad():
        rows = torch.cat([torch.from_numpy(emb[:8]), hf.model.embed_tokens(text)])
        z = hf(inputs_embeds=rows[None]).logits[0, L_P - 1:].numpy()
    worst = max(worst, float(np.abs(z - seq["logits"]).max()))
    return worst


def test_embed_hand_table():
    assert _hand_check(None)
    assert _hand_check("f32")
    assert _hand_check("bf16")   # every value is exact in bf16


def test_embed_matches_hf_lookup(weights):
    model = oracle_model(SHAPE, *weights, storage=None)
    # HF keeps RMSNorm and the rotary angles in fp32 even in a float64 model
    assert _hf_ids_check(model, weights) < 2e-5


def _embed_swapped(self, ids, embeds):          # given row where an id is, and vice versa
    ids = np.asarray(ids)
    out = np.zeros((ids.shape[0], self.shape.d_model))
    for r, t in enumerate(ids):
        out[r] = np.asarray(embeds[r]) if t >= 0 else self.g["embed"][t]
    return self.rs(out)


def _embed_by_row(self, ids, embeds):           # table indexed by packed row, not by token id
    ids = np.asarray(ids)
    out = np.zeros((ids.shape[0], self.shape.d_model))
    for r, t in enumerate(ids):
        out[r] = self.g["embed"][r] if t >= 0 else np.asarray(embeds[r])
    return self.rs(out)


def _embed_off_by_one(self, ids, embeds):       # id t takes table row t + 1 (mod V)
    ids = np.asarray(ids)
    out = np.zeros((ids.shape[0], self.shape.d_model))
    for r, t in enumerate(ids):
        out[r] = self.g["embed"][(t + 1) % self.shape.vocab] if t >= 0 else np.asarray(embeds[r])
    return self.rs(out)


@pytest.mark.parametrize("bad", [_embed_swapped, _embed_by_row, _embed_off_by_one])
def test_planted_embed_mistakes_break_a_pin(weights, monkeypatch, bad):
    monkeypatch.setattr(oracle.OracleModel, "embed", bad)
    try:
        hand_ok = _hand_check(None)
    except Exception:
        hand_ok = False
    model = oracle_model(SHAPE, *weights, storage=None)
    try:
        hf_ok = _hf_ids_check(model, weights, n_tokens=2) < 2e-5
    except Exception:
        hf_ok = False
    # each pin alone catches each of them
    assert not hand_ok, bad.__name__
    assert not hf_ok, bad.__name__


# ----------------------------------------------------------------------------- top-2 margin
def _margin_hand_check(fn):
    z = np.array([[1.0, 5.0, 3.0, 0.0],      # 5 - 3
                  [4.0, 4.0, 1.0, 0.0],      # a tie at the top: 0
                  [-3.0, -1.0, -2.0, -7.0],  # -1 - (-2)
                  [9.0, 0.0, 8.5, 8.75]])    # 9 - 8.75
    if not np.array_equal(fn(z), [2.0, 0.0, 1.0, 0.25]):
        return False
    # a single row (1-d input) gives a scalar
    return float(fn(np.array([0.5, -2.0, 0.25]))) == 0.25


def _margin_brute(z):
    out = []
    for row in z:
        row = [float(v) for v in row]
        i = max(range(len(row)), key=lambda j: row[j])
        rest = row[:i] + row[i + 1:]
        out.append(row[i] - max(rest))
    return np.array(out)


def test_top2_margin_hand_values():
    assert _margin_hand_check(top2_margin)


def test_top2_margin_brute_force():
    rng = np.random.default_rng(7)
    z = rng.standard_normal((200, 37))
    z[::5, 3] = z[::5].max(axis=1)             # exact ties in every fifth row
    z[1::7] = np.round(z[1::7], 1)             # coarse values: more ties
    assert np.array_equal(top2_margin(z), _margin_brute(z))


def _srt(z):
    return np.sort(np.asarray(z, dtype=np.float64), axis=-1)


def _margin_distinct(z):                        # ties at the top ignored: next distinct value
    z = np.asarray(z, dtype=np.float64)
    out = np.array([np.unique(r)[-1] - np.unique(r)[-2] for r in np.atleast_2d(z)])
    return out if z.ndim > 1 else out[0]


@pytest.mark.parametrize("bad", [
    lambda z: _srt(z)[..., -1] - _srt(z)[..., -3],   # skips the runner-up
    lambda z: _srt(z)[..., -2] - _srt(z)[..., -3],   # off by one position
    lambda z: _srt(z)[..., -1] - _srt(z)[..., 0],    # max - min
    _margin_distinct,
])
def test_planted_margin_mistakes_break_a_pin(bad):
    try:
        ok = _margin_hand_check(bad)
    except Exception:
        ok = False
    assert not ok
