"""The oracle's target forward pinned against transformers' Qwen3 (CPU, fp64)
with identical weights, and the drafter's layer pinned against the same
library layer run with a bidirectional mask over [context; block]."""
import numpy as np
import pytest
import torch

from oracle import Mode, OracleDFlow, OracleModel
from workload import get_config
from workload.synth import make_prompts, make_weights

transformers = pytest.importorskip("transformers")


def _hf_model(dm, w, prefix="layers", final_norm="final_norm"):
    from transformers import Qwen3Config, Qwen3ForCausalLM
    cfg = Qwen3Config(vocab_size=dm.vocab, hidden_size=dm.d, intermediate_size=dm.ffn,
                      num_hidden_layers=dm.n_layers if prefix == "layers" else dm.n_draft_layers,
                      num_attention_heads=dm.n_heads, num_key_value_heads=dm.n_kv_heads, head_dim=dm.head_dim,
                      rms_norm_eps=dm.rms_eps, rope_parameters={"rope_type": "default", "rope_theta": dm.rope_theta},
                      tie_word_embeddings=False, attention_bias=False, max_position_embeddings=4096,
                      attn_implementation="eager")
    model = Qwen3ForCausalLM(cfg).double().eval()
    f = lambda a: torch.from_numpy(np.asarray(a, np.float64))
    sd = {"model.embed_tokens.weight": f(w["embed"]), "model.norm.weight": f(w[final_norm]),
          "lm_head.weight": f(w["lm_head"])}
    n = cfg.num_hidden_layers
    for l in range(n):
        p = f"{prefix}.{l}"
        q = f"model.layers.{l}"
        sd.update({f"{q}.input_layernorm.weight": f(w[f"{p}.attn_norm"]),
                   f"{q}.post_attention_layernorm.weight": f(w[f"{p}.ffn_norm"]),
                   f"{q}.self_attn.q_proj.weight": f(w[f"{p}.wq"]), f"{q}.self_attn.k_proj.weight": f(w[f"{p}.wk"]),
                   f"{q}.self_attn.v_proj.weight": f(w[f"{p}.wv"]), f"{q}.self_attn.o_proj.weight": f(w[f"{p}.wo"]),
                   f"{q}.self_attn.q_norm.weight": f(w[f"{p}.q_norm"]),
                   f"{q}.self_attn.k_norm.weight": f(w[f"{p}.k_norm"]),
                   f"{q}.mlp.gate_proj.weight": f(w[f"{p}.w_gate"]), f"{q}.mlp.up_proj.weight": f(w[f"{p}.w_up"]),
                   f"{q}.mlp.down_proj.weight": f(w[f"{p}.w_down"])})
    missing, unexpected = model.load_state_dict(sd, strict=False)
    assert not unexpected and all("rotary" in k for k in missing), (missing, unexpected)
    return model


@pytest.fixture(scope="module")
def tiny():
    wl = get_config("tiny-f32")
    w = make_weights(wl.dims, wl.seed_w)
    return wl, w


def test_target_logits_match_hf_qwen3(tiny):
    wl, w = tiny
    dm = wl.dims
    prompt = make_prompts(wl)[0][:96]
    hf = _hf_model(dm, w)
    with torch.no_grad():
        out = hf(torch.from_numpy(prompt.astype(np.int64))[None], output_hidden_states=True)
    ref = out.logits[0].numpy()
    m = OracleModel(dm, w, Mode("fp64"))
    o = OracleDFlow(m, wl.block)
    lg = o.full_logits(prompt)
    rel = np.linalg.norm(lg - ref, axis=1) / np.linalg.norm(ref, axis=1)
    # transformers evaluates RoPE angles in fp32 even for a float64 model, so
    # agreement is bounded near 1e-7; a dropped gain, a sign or an index error
    # moves the logits by more than 1e-3.
    assert rel.max() < 1e-5, rel.max()
    np.testing.assert_allclose(hf.model.rotary_emb.inv_freq.double().numpy(), m.inv_freq, rtol=1e-6)
    # residual stream after layer 0 (hidden_states[1] is not final-normed for l < L-1)
    e = lambda: np.zeros((0, dm.n_kv_heads, dm.head_dim))
    _, _, _, hid = m.target_block(list(prompt), 0, [e() for _ in range(dm.n_layers)], [e() for _ in range(dm.n_layers)])
    np.testing.assert_allclose(hid[0], out.hidden_states[1][0].numpy(), rtol=1e-5, atol=1e-6)


def test_fp32_oracle_agrees_with_fp64(tiny):
    wl, w = tiny
    prompt = make_prompts(wl)[0][:64]
    l64 = OracleDFlow(OracleModel(wl.dims, w, Mode("fp64")), wl.block).full_logits(prompt)
    l32 = OracleDFlow(OracleModel(wl.dims, w, Mode("fp32")), wl.block).full_logits(prompt)
    rel = np.linalg.norm(l32 - l64, axis=1) / np.linalg.norm(l64, axis=1)
    assert rel.max() < 1e-5, rel.max()


def test_bf16_oracle_close_to_fp64(tiny):
    wl, w = tiny
    prompt = make_prompts(wl)[0][:64]
    l64 = OracleDFlow(OracleModel(wl.dims, w, Mode("fp64")), wl.block).full_logits(prompt)
    lb = OracleDFlow(OracleModel(wl.dims, w, Mode("bf16")), wl.block).full_logits(prompt)
    rel = np.linalg.norm(lb - l64, axis=1) / np.linalg.norm(l64, axis=1)
    assert 1e-5 < rel.max() < 3e-2, rel.max()     # rounding is really applied, and bounded


def test_drafter_layer_matches_hf_with_bidirectional_mask(tiny):
    """With an empty context, the drafter is a Qwen3 decoder stack whose block
    rows all see each other: pin it against transformers' Qwen3 run on the
    drafter's weights with an all-visible attention mask at positions
    pos0..pos0+B-1 (context attention is pinned separately through the SDPA
    test of the attention primitive)."""
    wl, w = tiny
    dm = wl.dims
    m = OracleModel(dm, w, Mode("fp64"))
    rng = np.random.default_rng(11)
    B = wl.block
    x = m.w("embed")[rng.integers(0, dm.vocab, B)]
    e = lambda: np.zeros((0, dm.n_kv_heads, dm.head_dim))
    pos0 = 37
    lg = m.drafter_block(x, pos0, [e()], [e()])
    # HF drafter stand-in: one Qwen3 layer + drafter final norm + shared LM head,
    # run with an all-visible 4D mask at positions pos0..pos0+B-1
    hf = _hf_model(dm, w, prefix="draft.layers", final_norm="draft.final_norm")
    with torch.no_grad():
        pos = torch.arange(pos0, pos0 + B)[None]
        mask = torch.zeros(1, 1, B, B, dtype=torch.float64)
        out = hf(inputs_embeds=torch.from_numpy(x)[None], position_ids=pos, attention_mask=mask)
    ref = out.logits[0].numpy()
    rel = np.linalg.norm(lg - ref, axis=1) / np.linalg.norm(ref, axis=1)
    assert rel.max() < 1e-5, rel.max()
    with torch.no_grad():   # the library honoured the mask: causal results differ
        causal = hf(inputs_embeds=torch.from_numpy(x)[None], position_ids=pos).logits[0].numpy()
    assert np.abs(causal[:-1] - ref[:-1]).max() > 1e-3


def test_fuse_matches_torch(tiny):
    """f = RMSNorm(W_c [H^l1; ...; H^lm]) with torch's linear and rms_norm."""
    wl, w = tiny
    dm = wl.dims
    m = OracleModel(dm, w, Mode("fp64"))
    h = np.random.default_rng(12).standard_normal((5, dm.m * dm.d))
    ref = torch.nn.functional.rms_norm(torch.from_numpy(h) @ torch.from_numpy(m.w("draft.w_c")).T, (dm.d,),
                                       torch.from_numpy(m.w("draft.g_c")), eps=dm.rms_eps).numpy()
    np.testing.assert_allclose(m.fuse(h), ref, rtol=1e-12, atol=1e-13)


def test_capture_order_matches_hf_layer_outputs(tiny):
    """Verify captures the raw residual output of each capture layer, concatenated
    in increasing layer order (hooks on transformers' decoder layers)."""
    wl, w = tiny
    dm = wl.dims
    hf = _hf_model(dm, w)
    outs = {}
    hooks = [hf.model.layers[l].register_forward_hook(
        lambda mod, inp, out, l=l: outs.__setitem__(l, (out[0] if isinstance(out, tuple) else out)[0].numpy()))
        for l in range(dm.n_layers)]
    prompt = make_prompts(wl)[0][:40]
    m = OracleModel(dm, w, Mode("fp64"))
    o = OracleDFlow(m, wl.block)
    s = o.prefill(prompt[:32])
    block = prompt[32:32 + wl.block]
    block[0] = s.anchor
    _, _, hcat, _, _ = o.verify(s, block)
    with torch.no_grad():
        hf(torch.from_numpy(np.concatenate([prompt[:32], block]).astype(np.int64))[None])
    for h in hooks:
        h.remove()
    ref = np.concatenate([outs[l][32:] for l in dm.capture_layers], axis=1)
    np.testing.assert_allclose(hcat, ref, rtol=1e-5, atol=1e-6)


def test_drafter_with_context_matches_hf_cache(tiny):
    """The drafter block attends to context keys/values made from the fused
    features by each draft layer's own key/value projections (k-norm and RoPE
    on keys, no input norm) plus every block key.  Pin: build those context
    entries with transformers' own k_proj / k_norm / v_proj / rotary modules,
    load them as the layer's cache, and run transformers' drafter stack with an
    all-visible mask over [context; block]."""
    from transformers import DynamicCache
    from transformers.models.qwen3.modeling_qwen3 import apply_rotary_pos_emb
    wl, w = tiny
    dm = wl.dims
    m = OracleModel(dm, w, Mode("fp64"))
    o = OracleDFlow(m, wl.block)
    s = o.prefill(make_prompts(wl)[0][:45])
    t, B = s.t, wl.block
    x, _ = o.draft_inputs(s, carry_on=False)
    lg = m.drafter_block(x, t, s.ck, s.cv)
    hf = _hf_model(dm, w, prefix="draft.layers", final_norm="draft.final_norm")
    cache = DynamicCache()
    F = torch.from_numpy(s.F)[None]
    with torch.no_grad():
        for l, layer in enumerate(hf.model.layers):
            at = layer.self_attn
            k = at.k_norm(at.k_proj(F).view(1, t, dm.n_kv_heads, dm.head_dim)).transpose(1, 2)
            v = at.v_proj(F).view(1, t, dm.n_kv_heads, dm.head_dim).transpose(1, 2)
            cos, sin = hf.model.rotary_emb(k, torch.arange(t)[None])
            _, k = apply_rotary_pos_emb(k, k, cos, sin)
            cache.update(k, v, l)
            np.testing.assert_allclose(k[0].transpose(0, 1).numpy(), s.ck[l], rtol=1e-5, atol=1e-6)
            np.testing.assert_allclose(v[0].transpose(0, 1).numpy(), s.cv[l], rtol=1e-12, atol=1e-13)
        mask = torch.zeros(1, 1, B, t + B, dtype=torch.float64)
        out = hf(inputs_embeds=torch.from_numpy(x)[None], position_ids=torch.arange(t, t + B)[None],
                 attention_mask=mask, past_key_values=cache, use_cache=True)
    ref = out.logits[0].numpy()
    rel = np.linalg.norm(lg - ref, axis=1) / np.linalg.norm(ref, axis=1)
    assert rel.max() < 1e-5, rel.max()
