"""Model-level pins of the oracle.

* The plain definition (``sequential_generate``) equals the HF Transformers Llama
  decoder run on the same weights (an independent implementation of the standard
  block the paper's backbone uses).
* The method (``PipelineOracle``, Alg. 1 + Alg. 2) equals the plain definition row for
  row and token for token (the paper's losslessness claim, Sec. 4.4).
* The ring slot of every live request equals that request's linear cache (Sec. 3.3:
  logically partitioned per request).
* Planted mistakes in the oracle (on the CPU) break these pins.
"""
import copy

import numpy as np
import pytest
import torch

import oracle
import workload as wl
from oracle.pipeline import PipelineOracle, sequential_generate
from tests.helpers import oracle_model, tiny_prefill_fn, to_np

SHAPE = wl.TINY
K, L_P, N_SLOTS, MAX_POS = 3, 32, 4, 64


@pytest.fixture(scope="module")
def weights():
    return wl.model_weights(SHAPE, seed=0, random_gains=True)


def _hf_model(weights):
    from transformers import LlamaConfig, LlamaForCausalLM
    g, layers = weights
    cfg = LlamaConfig(vocab_size=SHAPE.vocab, hidden_size=SHAPE.d_model, intermediate_size=SHAPE.d_ff,
                      num_hidden_layers=SHAPE.n_layers, num_attention_heads=SHAPE.n_heads,
                      num_key_value_heads=SHAPE.n_heads, head_dim=SHAPE.head_dim, rms_norm_eps=SHAPE.rms_eps,
                      rope_theta=SHAPE.rope_theta, max_position_embeddings=MAX_POS, attention_bias=False,
                      mlp_bias=False, tie_word_embeddings=False)
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).to(torch.float64).eval()
    sd = {"model.embed_tokens.weight": g["embed"], "model.norm.weight": g["final_norm"], "lm_head.weight": g["lm_head"]}
    names = dict(attn_norm="input_layernorm.weight", wq="self_attn.q_proj.weight", wk="self_attn.k_proj.weight",
                 wv="self_attn.v_proj.weight", wo="self_attn.o_proj.weight", mlp_norm="post_attention_layernorm.weight",
                 w_gate="mlp.gate_proj.weight", w_up="mlp.up_proj.weight", w_down="mlp.down_proj.weight")
    for l, lw in enumerate(layers):
        for k, v in lw.items():
            sd[f"model.layers.{l}.{names[k]}"] = v
    m.load_state_dict({k: v.to(torch.float64) for k, v in sd.items()}, strict=True)
    return m


def _hf_pin(model, weights, n_tokens=5):
    """Max |oracle - HF| over logits of every generated position and the layer-0 output."""
    fn = tiny_prefill_fn(SHAPE, L_P, seed=0, n_vision=8)
    ids, emb = fn(0)
    seq = sequential_generate(model, ids, emb, n_tokens)
    hf = _hf_model(weights)
    toks = seq["tokens"]
    x0 = model.embed(ids, emb)
    rows = np.concatenate([x0, np.stack([model.g["embed"][t] for t in toks[:-1]])])
    with torch.no_grad():
        out = hf(inputs_embeds=torch.from_numpy(rows)[None], output_hidden_states=True)
    hf_logits = out.logits[0, L_P - 1:].numpy()
    d_logits = np.abs(hf_logits - seq["logits"]).max()
    # hidden_states[1] is the output of layer 0 for every row
    ref1 = np.zeros_like(seq["hidden"])
    x = x0
    ck = np.zeros((len(rows), model.H, model.hd)); cv = np.zeros_like(ck)
    from oracle.pipeline import _block_linear_cache
    ref1 = _block_linear_cache(model, 0, rows, np.arange(len(rows)), ck, cv)
    d_h1 = np.abs(out.hidden_states[1][0].numpy() - ref1).max()
    return d_logits, d_h1, toks, hf_logits


def test_sequential_definition_matches_hf_llama(weights):
    model = oracle_model(SHAPE, *weights, storage=None)
    d_logits, d_h1, toks, hf_logits = _hf_pin(model, weights)
    # HF keeps RMSNorm and the rotary angles in fp32 even in a float64 model
    assert d_h1 < 2e-5, d_h1
    assert d_logits < 2e-5, d_logits
    assert toks == [int(np.argmax(z)) for z in hf_logits]


def test_planted_mistakes_break_the_hf_pin(weights, monkeypatch):
    """Each plausible slip in the oracle's math must move it far from HF."""
    import oracle.model as om
    import oracle.pipeline as op
    good_rope, good_silu, good_rms = om.rope, om.silu, om.rmsnorm

    def rope_sign(u, pos, theta):      # rotation in the wrong direction
        return good_rope(u, -np.asarray(pos), theta)

    def rope_interleaved(u, pos, theta):  # pairs (2j, 2j+1) instead of (j, j + hd/2)
        hd = u.shape[-1]
        perm = np.stack([np.arange(hd // 2), np.arange(hd // 2) + hd // 2], -1).reshape(-1)
        v = good_rope(u[..., perm], pos, theta)
        out = np.empty_like(v)
        out[..., perm] = v
        return out

    def silu_as_sigmoid(z):
        return 1.0 / (1.0 + np.exp(-np.asarray(z)))

    def rms_no_gain(x, g, eps):
        return good_rms(x, np.ones_like(g), eps)

    # (a uniform shift of every position is not a mistake: scores depend only on m - n)
    cases = [("rope", rope_sign), ("rope", rope_interleaved), ("silu", silu_as_sigmoid),
             ("rmsnorm", rms_no_gain)]
    model = oracle_model(SHAPE, *weights, storage=None)
    for name, bad in cases:
        with monkeypatch.context() as mp:
            mp.setattr(om, name, bad)
            mp.setattr(op, name, bad)
            d_logits, d_h1, _, _ = _hf_pin(model, weights, n_tokens=2)
        assert max(d_logits, d_h1) > 1e-3, (name, bad.__name__, d_logits, d_h1)


def _run_pipeline(model, n_steps, k=K):
    fn = tiny_prefill_fn(SHAPE, L_P, seed=0, n_vision=8)
    pipe = PipelineOracle(model, k, N_SLOTS, MAX_POS, fn)
    steps = [pipe.step() for _ in range(n_steps)]
    return pipe, steps, fn


@pytest.mark.parametrize("storage", [None, "f32", "bf16"])
def test_packed_equals_sequential(weights, storage):
    model = oracle_model(SHAPE, *weights, storage=storage)
    pipe, steps, fn = _run_pipeline(model, 7)
    finished = {}
    for st in steps:
        finished.update(st["done"])
    assert sorted(finished) == [0, 1, 2, 3, 4]
    tol = 1e-10 if storage is None else 0.0
    for r, toks in finished.items():
        ids, emb = fn(r)
        seq = sequential_generate(model, ids, emb, K)
        assert toks == seq["tokens"], (r, toks, seq["tokens"])
        # every row the pipeline computed for request r equals the sequential row
        for st in steps:
            for sg in st["segments"]:
                if sg.request_id != r:
                    continue
                got = st["hidden"][sg.q_start:sg.q_start + sg.q_len]
                want = seq["hidden"][sg.pos0:sg.pos0 + sg.q_len]
                assert np.abs(got - want).max() <= tol * max(1.0, np.abs(want).max()), (r, st["t"])


def test_step2_is_the_34_row_configured_step(weights):
    """Cold start, K = 3, L_P = 32: step 2 packs 32 prefill rows + decodes at contexts 33, 34."""
    model = oracle_model(SHAPE, *weights)
    _, steps, _ = _run_pipeline(model, 3)
    segs = steps[2]["segments"]
    assert [(s.q_start, s.q_len, s.slot, s.pos0, s.kv_len) for s in segs] == \
        [(0, 32, 2, 0, 32), (32, 1, 1, 32, 33), (33, 1, 0, 33, 34)]


def test_ring_slot_equals_linear_cache(weights):
    model = oracle_model(SHAPE, *weights, storage="bf16")
    pipe, steps, fn = _run_pipeline(model, 6)
    # live after step 5: requests 4 (1 token) and 5 (0 tokens... prefill done, 1 token)
    for r in (4, 5):
        slot = pipe.ring.slot_of(r)
        n = pipe.ring.length[slot]
        ids, emb = fn(r)
        forced = pipe.seqs[r]
        seq = sequential_generate(model, ids, emb, len(forced) + 1, forced=forced)
        assert np.array_equal(pipe.kv.k[:, slot, :n], seq["cache_k"][:, :n])
        assert np.array_equal(pipe.kv.v[:, slot, :n], seq["cache_v"][:, :n])


def test_planted_mask_mistake_breaks_packed_equals_sequential(weights, monkeypatch):
    """A packed attention that lets a prefill row see later rows must fail the pin."""
    import oracle.model as om
    good = om.attend_segment

    def leaky(q, pos, keys, values, scale):
        return good(q, np.full_like(np.asarray(pos), keys.shape[0] - 1), keys, values, scale)

    model = oracle_model(SHAPE, *weights, storage=None)
    monkeypatch.setattr(om, "attend_segment", leaky)
    pipe, steps, fn = _run_pipeline(model, 1)
    ids, emb = fn(0)
    seq = sequential_generate(model, ids, emb, 1)
    assert np.abs(steps[0]["hidden"] - seq["hidden"][:L_P]).max() > 1e-3


def test_planted_slot_mistake_breaks_ring_pin(weights, monkeypatch):
    """Reading a decode's history from the wrong slot must fail packed == sequential."""
    import oracle.model as om
    model = oracle_model(SHAPE, *weights, storage=None)
    good_layer = om.OracleModel.layer_packed

    def wrong_slot(self, l, x, segs, ring, trace=None):
        segs = [copy.copy(s) for s in segs]
        if len(segs) > 1:
            segs[1].slot = (segs[1].slot + 1) % ring.n_slots
        return good_layer(self, l, x, segs, ring, trace)

    monkeypatch.setattr(om.OracleModel, "layer_packed", wrong_slot)
    pipe, steps, fn = _run_pipeline(model, 3)
    ids, emb = fn(1)
    forced = [steps[1]["used"][0]]
    seq = sequential_generate(model, ids, emb, 2, forced=forced)
    row = steps[2]["segments"][1].q_start
    assert np.abs(steps[2]["hidden"][row] - seq["hidden"][L_P]).max() > 1e-3


def test_planted_decode_position_mistake_breaks_packed_equals_sequential(weights, monkeypatch):
    """Rotating a stage-s decode row at L_P + s (one past its KV index) instead of
    L_P + s - 1 shifts its distance to the history and must fail the pin."""
    import oracle.model as om
    good = om.rope

    def shifted(u, pos, theta):
        pos = np.asarray(pos)
        return good(u, np.where(pos >= L_P, pos + 1, pos), theta)

    model = oracle_model(SHAPE, *weights, storage=None)
    monkeypatch.setattr(om, "rope", shifted)   # packed path only; the definition keeps the true rope
    pipe, steps, fn = _run_pipeline(model, 2)
    ids, emb = fn(0)
    seq = sequential_generate(model, ids, emb, 2, forced=[steps[0]["used"][0]])
    row = steps[1]["segments"][1].q_start
    assert np.abs(steps[1]["hidden"][row] - seq["hidden"][L_P]).max() > 1e-3
