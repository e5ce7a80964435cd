"""A decoder stack around span attention, written out from its definition (CPU, float64).

Test infrastructure only (see the package docstring).

The span query's model input S = p | F_s1 | ... | F_sn | c runs through a
pre-norm decoder whose attention is the span attention of ``attention`` (the
mask of section 5.6 with the positions of section 5.5): a fragment token's hidden
state depends only on the prefix and its own fragment, at every layer, which is
what lets the cache of section 5.5 hold a fragment's keys and values once for any
query.  The layer itself is not the paper's subject (it names no architecture for
its latency experiments); this one is the Llama-shaped block the workloads use:

    n  = RMSNorm(x) * g_attn                  RMSNorm(x) = x / sqrt(mean(x^2) + eps)
    q, k, v = n W_q, n W_k, n W_v             (W_qkv holds the three side by side)
    o  = span attention(q, k, v)              query head h reads kv head floor(h Hkv / Hq)
    h  = x + o W_o
    n2 = RMSNorm(h) * g_ffn
    x' = h + (silu(n2 W_gate) * (n2 W_up)) W_down      silu(z) = z / (1 + e^-z)

then a final RMSNorm and the LM head on the last cross row; the first token is
the argmax of those logits, the lowest token id on ties.

Precision.  Arithmetic is float64.  With ``storage="bf16"`` every tensor the
model stores between operations (the norms' outputs, q/k/v, the attention output,
the residual stream after each addition, the gate/up product and the SwiGLU
output) is rounded to bfloat16, round to nearest even, as a bf16 model stores it;
the logits stay float64.  ``storage="f64"`` rounds nothing.

Pins (tests/test_oracle_stack.py): one fragment with its prefix and cross segment
is plain causal attention, so the whole stack reduces to an ordinary causal
decoder, checked against an independently written Llama decoder (transformers'
LlamaForCausalLM in float64) layer by layer and at the logits; after one layer
the cross rows of any query equal that decoder's rows over S; fragment rows of a
many-fragment query equal the stack over the prefix and that fragment alone.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

from . import attention as A


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits), ties to even, of finite float64 values."""
    x = np.asarray(x, np.float64)
    m, e = np.frexp(x)                       # x = m 2^e, 0.5 <= |m| < 1
    scale = np.ldexp(1.0, e - 8)             # one unit in the 8th significant bit
    return np.where(x == 0, 0.0, np.round(x / scale) * scale)


def rms_norm(x: np.ndarray, gain: np.ndarray, eps: float) -> np.ndarray:
    x = np.asarray(x, np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * np.asarray(gain, np.float64)


def silu(z: np.ndarray) -> np.ndarray:
    return z / (1.0 + np.exp(-z))


@dataclass
class Weights:
    """Float64 views of a stack's weights (x @ W convention: W is [in, out])."""
    embed: np.ndarray                 # [vocab, hidden]
    attn_norm: Sequence[np.ndarray]   # per layer [hidden]
    w_qkv: Sequence[np.ndarray]       # per layer [hidden, (Hq + 2 Hkv) d]: q | k | v columns
    w_o: Sequence[np.ndarray]         # per layer [Hq d, hidden]
    ffn_norm: Sequence[np.ndarray]    # per layer [hidden]
    w_gate_up: Sequence[np.ndarray]   # per layer [hidden, 2 F]: gate | up columns
    w_down: Sequence[np.ndarray]      # per layer [F, hidden]
    final_norm: np.ndarray            # [hidden]
    lm_head: np.ndarray               # [hidden, vocab]
    n_q_heads: int
    n_kv_heads: int
    head_dim: int


def layer(x: np.ndarray, lay: A.Layout, W: Weights, l: int, theta: float, eps: float,
          storage: str = "bf16") -> np.ndarray:
    """One decoder layer over every token of S (rows in S order)."""
    rnd = round_bf16 if storage == "bf16" else (lambda a: a)
    hq, hkv, d = W.n_q_heads, W.n_kv_heads, W.head_dim
    n_tok = x.shape[0]
    n = rnd(rms_norm(x, W.attn_norm[l], eps))
    qkv = rnd(n @ np.asarray(W.w_qkv[l], np.float64))
    q = qkv[:, : hq * d].reshape(n_tok, hq, d)
    k = qkv[:, hq * d: (hq + hkv) * d].reshape(n_tok, hkv, d)
    v = qkv[:, (hq + hkv) * d:].reshape(n_tok, hkv, d)
    o = rnd(A.span_attention(q, k, v, lay, theta)).reshape(n_tok, hq * d)
    h = rnd(x + o @ np.asarray(W.w_o[l], np.float64))
    n2 = rnd(rms_norm(h, W.ffn_norm[l], eps))
    gu = rnd(n2 @ np.asarray(W.w_gate_up[l], np.float64))
    f = gu.shape[1] // 2
    act = rnd(silu(gu[:, :f]) * gu[:, f:])
    return rnd(h + act @ np.asarray(W.w_down[l], np.float64))


def stack_forward(tokens: Sequence[int], lay: A.Layout, W: Weights, n_layers: int, theta: float,
                  eps: float, storage: str = "bf16", keep: Optional[Sequence[int]] = None):
    """Hidden states of every token of S after ``n_layers`` layers (float64 [N, hidden]).
    With ``keep``, returns {layer count: hidden states} for each count in keep (0 = the
    embeddings)."""
    x = np.asarray(np.asarray(W.embed)[np.asarray(tokens, np.int64)], np.float64)
    kept = {}
    if keep is not None and 0 in keep:
        kept[0] = x.copy()
    for l in range(n_layers):
        x = layer(x, lay, W, l, theta, eps, storage)
        if keep is not None and (l + 1) in keep:
            kept[l + 1] = x.copy()
    return kept if keep is not None else x


def final_logits(x_row: np.ndarray, W: Weights, eps: float, storage: str = "bf16") -> np.ndarray:
    """LM-head logits (float64) of one hidden state: RMSNorm with the final gain, then W_lm."""
    rnd = round_bf16 if storage == "bf16" else (lambda a: a)
    n = rnd(rms_norm(np.asarray(x_row, np.float64)[None, :], W.final_norm, eps))
    return (n @ np.asarray(W.lm_head, np.float64))[0]


def first_token(logits: np.ndarray) -> int:
    """Argmax with ties to the lowest token id."""
    logits = np.asarray(logits)
    return int(np.flatnonzero(logits == logits.max())[0])


def query_tokens(prefix: Sequence[int], frags: Sequence[Sequence[int]], cross: Sequence[int]) -> List[int]:
    """Tokens of S = prefix | fragments in this query's order | cross."""
    out = [int(t) for t in prefix]
    for f in frags:
        out += [int(t) for t in f]
    return out + [int(t) for t in cross]
