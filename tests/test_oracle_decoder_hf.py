"""Pins of the oracle decoder as a whole (layer wiring, not just its parts).

* Against an independent implementation of the Llama layer: ``transformers``'
  ``LlamaForCausalLM`` run in float64 on the CPU, with the oracle's weights
  mapped into it (q / k / v rows of wqkv, gate / up rows of w_gate_up).  The
  paper's models are Llama / Qwen-family decoders (Section 4.1; Table 10),
  which the Llama layer stands in for.  Transformers' RMSNorm computes in
  float32 whatever the model dtype, which limits agreement to ~1e-7 relative;
  a mis-wired layer (dropped residual, norm in the wrong place, gate and up
  swapped, wrong GQA head map or rotary convention) is off by O(1).
* Closed forms that hold for any decoder built from the Llama layer: with the
  attention output and down projections zeroed the residual stream is the
  embedding, so the logits are RMSNorm(E[x]) W_lm^T; with wqkv zeroed the
  attention contributes nothing and one layer is a pure MLP residual.

Norm weights are drawn away from 1 and the init scale raised so that every
sub-layer moves the logits; one case has a vocabulary above 8192 so that the
oracle's blocked LM-head product runs.
"""

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decoder as D
from workloads import ModelShape, model_weights
from workloads.gen import bf16_u16_to_f32

transformers = pytest.importorskip("transformers")


def _f64(w):
    w = np.asarray(w)
    if w.dtype == np.uint16:
        return torch.from_numpy(bf16_u16_to_f32(w).astype(np.float64))
    return torch.from_numpy(w.astype(np.float64))


def _weights(sh, seed):
    """Model weights with norm vectors drawn from U(0.5, 1.5) (same storage dtype)."""
    w = model_weights(sh, seed)
    g = np.random.default_rng(seed + 1)

    def norm_vec():
        x = g.uniform(0.5, 1.5, sh.d_model).astype(np.float32)
        if sh.dtype == "bf16":
            from workloads import bf16_round_u16
            return bf16_round_u16(x)
        return x

    w["final_norm"] = norm_vec()
    for lw in w["layers"]:
        lw["attn_norm"] = norm_vec()
        lw["mlp_norm"] = norm_vec()
    return w


def _hf_model(sh, w):
    from transformers import LlamaConfig, LlamaForCausalLM
    cfg = LlamaConfig(vocab_size=sh.vocab, hidden_size=sh.d_model, intermediate_size=sh.ffn_dim,
                      num_hidden_layers=len(w["layers"]), num_attention_heads=sh.n_heads,
                      num_key_value_heads=sh.n_kv_heads, head_dim=sh.head_dim, rope_theta=sh.rope_theta,
                      rms_norm_eps=sh.rms_eps, tie_word_embeddings=False, attention_bias=False,
                      mlp_bias=False, max_position_embeddings=4096, hidden_act="silu")
    cfg._attn_implementation = "eager"
    torch.manual_seed(0)
    m = LlamaForCausalLM(cfg).double().eval()
    hq, hkv, hd, f = sh.n_heads * sh.head_dim, sh.n_kv_heads * sh.head_dim, sh.head_dim, sh.ffn_dim
    del hd
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(_f64(w["embed"]))
        m.model.norm.weight.copy_(_f64(w["final_norm"]))
        m.lm_head.weight.copy_(_f64(w["lm_head"]))
        for L, lw in zip(m.model.layers, w["layers"]):
            qkv = _f64(lw["wqkv"])
            L.self_attn.q_proj.weight.copy_(qkv[:hq])
            L.self_attn.k_proj.weight.copy_(qkv[hq:hq + hkv])
            L.self_attn.v_proj.weight.copy_(qkv[hq + hkv:])
            L.self_attn.o_proj.weight.copy_(_f64(lw["wo"]))
            gu = _f64(lw["w_gate_up"])
            L.mlp.gate_proj.weight.copy_(gu[:f])
            L.mlp.up_proj.weight.copy_(gu[f:])
            L.mlp.down_proj.weight.copy_(_f64(lw["w_down"]))
            L.input_layernorm.weight.copy_(_f64(lw["attn_norm"]))
            L.post_attention_layernorm.weight.copy_(_f64(lw["mlp_norm"]))
    return m


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / np.max(np.abs(b)))


CASES = {
    "mha-f32": ModelShape("pin-hf-mha", 2, 64, 4, 4, 16, 96, 300, 1e4, dtype="f32", init_std=0.15),
    "gqa-bf16": ModelShape("pin-hf-gqa", 2, 64, 8, 2, 16, 96, 300, 5e5, dtype="bf16", init_std=0.15),
    "gqa-hd32-f32": ModelShape("pin-hf-hd32", 3, 128, 4, 1, 32, 160, 500, 5e5, dtype="f32", init_std=0.1),
    "bigvocab-f32": ModelShape("pin-hf-bigv", 1, 32, 4, 2, 8, 48, 9000, 1e4, dtype="f32", init_std=0.15),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_decoder_matches_transformers_llama(case):
    sh = CASES[case]
    w = _weights(sh, 21)
    toks = np.random.default_rng(3).integers(0, sh.vocab, size=23)
    ours = D.Decoder(sh, w).full_logits(toks)
    with torch.no_grad():
        ref = _hf_model(sh, w)(torch.from_numpy(toks)[None]).logits[0].numpy()
    assert ours.shape == ref.shape
    err = _rel(ours, ref)
    print(f"{case}: max rel err vs transformers {err:.2e}")
    assert err < 1e-5, err
    # the comparison is sharp: the layers move the logits by O(1) relative
    e = _f64(w["embed"])[torch.from_numpy(toks)]
    skip = F.rms_norm(e, (sh.d_model,), _f64(w["final_norm"]), eps=sh.rms_eps) @ _f64(w["lm_head"]).T
    assert _rel(skip.numpy(), ref) > 0.1


def test_decoder_cached_rows_match_transformers():
    """Incremental rows through the oracle's KV list at positions 17..22 equal
    the matching rows of transformers' full forward."""
    sh = CASES["gqa-bf16"]
    w = _weights(sh, 5)
    toks = np.random.default_rng(4).integers(0, sh.vocab, size=23)
    dec = D.Decoder(sh, w)
    kv = dec.new_kv()
    dec.forward(kv, toks[:17], np.arange(17), logits=False)
    z = dec.forward(kv, toks[17:], np.arange(17, 23))
    with torch.no_grad():
        ref = _hf_model(sh, w)(torch.from_numpy(toks)[None]).logits[0].numpy()
    assert _rel(z, ref[17:]) < 1e-5


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_zero_output_projections_give_embedding_logits(dtype):
    """wo = w_down = 0: every layer adds zero, so logits = RMSNorm(E[x]) W_lm^T."""
    sh = ModelShape("pin-id", 2, 48, 4, 2, 12, 64, 10000, 1e4, dtype=dtype, init_std=0.2)
    w = _weights(sh, 8)
    for lw in w["layers"]:
        lw["wo"] = np.zeros_like(lw["wo"])
        lw["w_down"] = np.zeros_like(lw["w_down"])
    toks = np.random.default_rng(9).integers(0, sh.vocab, size=11)
    e = _f64(w["embed"])[torch.from_numpy(toks)]
    y = F.rms_norm(e, (sh.d_model,), _f64(w["final_norm"]), eps=sh.rms_eps)
    ref = (y @ _f64(w["lm_head"]).T).numpy()
    assert _rel(D.Decoder(sh, w).full_logits(toks), ref) < 1e-12


def test_zero_qkv_gives_mlp_residual():
    """wqkv = 0: values are zero, attention adds nothing, and one layer is
    h = e + W_down (silu(W_gate y) * (W_up y)) with y = RMSNorm(e) w_mlp."""
    sh = ModelShape("pin-mlp", 1, 40, 5, 5, 8, 72, 200, 1e4, dtype="f32", init_std=0.2)
    w = _weights(sh, 12)
    lw = w["layers"][0]
    lw["wqkv"] = np.zeros_like(lw["wqkv"])
    toks = np.random.default_rng(13).integers(0, sh.vocab, size=9)
    e = _f64(w["embed"])[torch.from_numpy(toks)]
    y = F.rms_norm(e, (sh.d_model,), _f64(lw["mlp_norm"]), eps=sh.rms_eps)
    gu = _f64(lw["w_gate_up"])
    h = e + (F.silu(y @ gu[:sh.ffn_dim].T) * (y @ gu[sh.ffn_dim:].T)) @ _f64(lw["w_down"]).T
    z = F.rms_norm(h, (sh.d_model,), _f64(w["final_norm"]), eps=sh.rms_eps) @ _f64(w["lm_head"]).T
    assert _rel(D.Decoder(sh, w).full_logits(toks), z.numpy()) < 1e-12
