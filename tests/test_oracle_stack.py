"""Pins of the decoder-stack oracle (CPU).

* P9: a query with one fragment (prefix, fragment, cross) is plain causal
  attention over S at every layer, so the stack is an ordinary causal decoder.
  Checked against transformers' LlamaForCausalLM, an independently written
  decoder, in float64 with the same weights: hidden states after each layer and
  the logits of the last row.
* After one layer the cross rows of a many-fragment query equal that decoder's
  rows over S (their keys and values are projections of embeddings, and a cross
  row sees every earlier token at its final position); fragment rows equal the
  decoder over prefix | fragment (section 5.6 mask, canonical positions).
* At any depth a fragment's rows depend only on the prefix and the fragment.
* The bf16 rounding helper against torch's conversion and the workloads' bit
  rounding; argmax ties go to the lowest id.
"""
import numpy as np
import pytest

import workloads as W
from oracle import attention as OA
from oracle import stack as OS

torch = pytest.importorskip("torch")
transformers = pytest.importorskip("transformers")

HQ, HKV, D, HIDDEN, FFN, VOCAB = 4, 2, 16, 64, 96, 100
THETA, EPS = 1e4, 1e-5


def _weights(n_layers, seed=0, hidden=HIDDEN, hq=HQ, hkv=HKV, d=D, ffn=FFN, vocab=VOCAB, std=0.2):
    sw = W.stack_weights(seed, n_layers, hidden, hq, hkv, d, ffn, vocab, std=std, norm_std=0.1, threads=2)
    f = lambda a: W.bf16_bits_to_f32(a).astype(np.float64)  # noqa: E731
    return OS.Weights(embed=f(sw.embed), attn_norm=[f(a) for a in sw.attn_norm], w_qkv=[f(a) for a in sw.w_qkv],
                      w_o=[f(a) for a in sw.w_o], ffn_norm=[f(a) for a in sw.ffn_norm],
                      w_gate_up=[f(a) for a in sw.w_gate_up], w_down=[f(a) for a in sw.w_down],
                      final_norm=f(sw.final_norm), lm_head=f(sw.lm_head), n_q_heads=hq, n_kv_heads=hkv, head_dim=d)


def _llama(Wt, n_layers):
    from transformers import LlamaConfig, LlamaForCausalLM
    hq, hkv, d = Wt.n_q_heads, Wt.n_kv_heads, Wt.head_dim
    hidden = Wt.embed.shape[1]
    ffn = Wt.w_down[0].shape[0]
    cfg = LlamaConfig(vocab_size=Wt.embed.shape[0], hidden_size=hidden, intermediate_size=ffn,
                      num_hidden_layers=n_layers, num_attention_heads=hq, num_key_value_heads=hkv, head_dim=d,
                      rms_norm_eps=EPS, rope_theta=THETA, max_position_embeddings=4096, tie_word_embeddings=False,
                      attention_bias=False, mlp_bias=False)
    cfg._attn_implementation = "eager"
    m = LlamaForCausalLM(cfg).to(torch.float64).eval()
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.float64))  # noqa: E731
    with torch.no_grad():
        m.model.embed_tokens.weight.copy_(t(Wt.embed))
        m.model.norm.weight.copy_(t(Wt.final_norm))
        m.lm_head.weight.copy_(t(Wt.lm_head.T))
        for l, blk in enumerate(m.model.layers):
            qkv = Wt.w_qkv[l]
            blk.input_layernorm.weight.copy_(t(Wt.attn_norm[l]))
            blk.self_attn.q_proj.weight.copy_(t(qkv[:, : hq * d].T))
            blk.self_attn.k_proj.weight.copy_(t(qkv[:, hq * d: (hq + hkv) * d].T))
            blk.self_attn.v_proj.weight.copy_(t(qkv[:, (hq + hkv) * d:].T))
            blk.self_attn.o_proj.weight.copy_(t(Wt.w_o[l].T))
            blk.post_attention_layernorm.weight.copy_(t(Wt.ffn_norm[l]))
            blk.mlp.gate_proj.weight.copy_(t(Wt.w_gate_up[l][:, :ffn].T))
            blk.mlp.up_proj.weight.copy_(t(Wt.w_gate_up[l][:, ffn:].T))
            blk.mlp.down_proj.weight.copy_(t(Wt.w_down[l].T))
    return m


def _hf(m, tokens):
    """Hidden states after each layer (the last one before the final norm, taken from
    the layer hook) and the logits of every row."""
    outs = []
    hooks = [blk.register_forward_hook(lambda mod, inp, out: outs.append(
        (out[0] if isinstance(out, tuple) else out)[0].detach().numpy().copy())) for blk in m.model.layers]
    with torch.no_grad():
        r = m(input_ids=torch.tensor([list(tokens)]))
    for h in hooks:
        h.remove()
    return outs, r.logits[0].numpy()


def _close(a, b, rel=1e-5):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    assert np.max(np.abs(a - b)) <= rel * max(1.0, np.max(np.abs(b))), np.max(np.abs(a - b))


@pytest.mark.parametrize("prefix_len,frag_len,cross_len", [(7, 20, 5), (0, 33, 0), (16, 1, 17)])
def test_one_fragment_stack_is_a_causal_decoder(prefix_len, frag_len, cross_len):
    n_layers = 3
    Wt = _weights(n_layers)
    rng = np.random.default_rng(1)
    pre, frag, cross = (rng.integers(0, VOCAB, n).tolist() for n in (prefix_len, frag_len, cross_len))
    toks = OS.query_tokens(pre, [frag], cross)
    lay = OA.layout(prefix_len, [frag_len], cross_len)
    mine = OS.stack_forward(toks, lay, Wt, n_layers, THETA, EPS, storage="f64", keep=[1, 2, 3])
    ref_layers, ref_logits = _hf(_llama(Wt, n_layers), toks)
    for l in (1, 2, 3):
        _close(mine[l], ref_layers[l - 1])
    logits = OS.final_logits(mine[3][-1], Wt, EPS, storage="f64")
    _close(logits, ref_logits[-1])
    assert OS.first_token(logits) == int(np.argmax(ref_logits[-1]))


def test_first_layer_rows_reduce_to_causal_decoder_rows():
    Wt = _weights(1, seed=3)
    rng = np.random.default_rng(2)
    P, Ls, Q = 9, [13, 4, 21], 6
    pre = rng.integers(0, VOCAB, P).tolist()
    frags = [rng.integers(0, VOCAB, n).tolist() for n in Ls]
    cross = rng.integers(0, VOCAB, Q).tolist()
    toks = OS.query_tokens(pre, frags, cross)
    lay = OA.layout(P, Ls, Q)
    mine = OS.stack_forward(toks, lay, Wt, 1, THETA, EPS, storage="f64")
    m = _llama(Wt, 1)
    whole, _ = _hf(m, toks)
    _close(mine[-Q:], whole[0][-Q:])                    # cross rows: causal over all of S
    at = P
    for f, L in zip(frags, Ls):                           # fragment rows: causal over prefix | fragment
        alone, _ = _hf(m, pre + f)
        _close(mine[at: at + L], alone[0][P:])
        at += L
    _close(mine[:P], whole[0][:P])


@pytest.mark.parametrize("storage", ["f64", "bf16"])
def test_fragment_rows_depend_only_on_prefix_and_fragment(storage):
    n_layers = 3
    Wt = _weights(n_layers, seed=5)
    rng = np.random.default_rng(4)
    P, Ls, Q = 12, [19, 7, 30], 9
    pre = rng.integers(0, VOCAB, P).tolist()
    frags = [rng.integers(0, VOCAB, n).tolist() for n in Ls]
    cross = rng.integers(0, VOCAB, Q).tolist()
    full = OS.stack_forward(OS.query_tokens(pre, frags, cross), OA.layout(P, Ls, Q), Wt, n_layers, THETA, EPS,
                            storage=storage)
    order = [2, 0, 1]
    perm = OS.stack_forward(OS.query_tokens(pre, [frags[i] for i in order], cross),
                            OA.layout(P, [Ls[i] for i in order], Q), Wt, n_layers, THETA, EPS, storage=storage)
    starts = np.cumsum([P] + Ls[:-1])
    pstarts = dict(zip(order, np.cumsum([P] + [Ls[i] for i in order][:-1])))
    tol = 1e-12 if storage == "f64" else 0.0
    for i, (f, L) in enumerate(zip(frags, Ls)):
        alone = OS.stack_forward(OS.query_tokens(pre, [f], []), OA.layout(P, [L], 0), Wt, n_layers, THETA, EPS,
                                 storage=storage)
        a = full[starts[i]: starts[i] + L]
        if storage == "f64":
            _close(a, alone[P:], rel=tol)
            _close(perm[pstarts[i]: pstarts[i] + L], a, rel=tol)
        else:
            # bf16 storage: equal up to rare one-unit roundings where float64 sums over
            # differently sized operands differ in the last bits
            assert np.mean(a == alone[P:]) > 0.99
            assert np.max(np.abs(a - alone[P:])) <= 2.0 ** -6 * max(1.0, np.max(np.abs(a)))


def test_round_bf16_against_torch_and_bit_rounding():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(200_000).astype(np.float32) * np.float32(10.0) ** rng.integers(-3, 3, 200_000)
    # exact halfway cases between neighbouring bf16 values: both neighbours' parities
    mant = rng.integers(128, 256, 2000).astype(np.float32)
    half = (mant + np.float32(0.5)) * np.float32(2.0) ** rng.integers(-20, 10, 2000).astype(np.float32)
    x = np.concatenate([x, half, -half, np.float32([0.0, 1.0, -1.0, 3.0])])
    mine = OS.round_bf16(x.astype(np.float64))
    t = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mine, t)
    assert np.array_equal(mine, W.bf16_bits_to_f32(W.round_to_bf16_bits(x)).astype(np.float64))


def test_first_token_lowest_id_on_ties():
    assert OS.first_token(np.array([0.5, 2.0, -1.0, 2.0])) == 1
    assert OS.first_token(np.array([3.0])) == 0


def test_rms_norm_closed_form():
    x = np.full((1, 8), -3.0)
    g = np.arange(1.0, 9.0)
    np.testing.assert_allclose(OS.rms_norm(x, g, 0.0), -g[None, :], rtol=1e-15)
    np.testing.assert_allclose(OS.rms_norm(x, g, 7.0), -3.0 / 4.0 * g[None, :], rtol=1e-15)
