"""Pins of the attention oracle against facts it does not define itself.

* Textbook reduction (single layer): a fragment's rows are ordinary causal
  attention over (prefix | fragment) at positions 0..P+L-1; cross rows are
  ordinary causal attention over the whole sequence at positions 0..N-1;
  with one fragment the whole output is ordinary causal attention.  The
  reference is torch's scaled_dot_product_attention with the rotary encoding
  of the transformers Llama implementation (library routines).
* Closed forms: with q = 0 every allowed key has equal weight, so with
  one-hot segment values the output is the exact fraction of allowed keys in
  each segment.
* Rotary identities: R(a)^T R(b) = R(b - a).
* Brute force: on tiny inputs, a pure-Python loop over (row, key, dim) that
  applies the visibility and position rules pair by pair agrees to 1e-12.
* Invariants from the paper: permuting commuting children leaves each child's
  cached KV bit-identical; cached-then-repositioned keys equal keys encoded
  at their final positions.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as A


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _llama_rope(x, pos, theta):
    """Rotary encoding via transformers' Llama implementation (x: [N, H, d] float64)."""
    from transformers import LlamaConfig
    from transformers.models.llama import modeling_llama as m
    d = x.shape[-1]
    cfg = LlamaConfig(hidden_size=d * 2, num_attention_heads=2, num_key_value_heads=2, head_dim=d,
                      rope_theta=theta)
    rot = m.LlamaRotaryEmbedding(cfg)
    t = torch.from_numpy(np.ascontiguousarray(x)).permute(1, 0, 2)[None]      # [1, H, N, d]
    cos, sin = rot(t, torch.as_tensor(pos)[None])
    out, _ = m.apply_rotary_pos_emb(t, t, cos, sin)
    return out[0].permute(1, 0, 2).numpy()


def _causal_sdpa(q, k, v, theta):
    """Ordinary causal attention over a whole sequence at positions 0..N-1."""
    n = q.shape[0]
    pos = np.arange(n)
    qr = torch.from_numpy(_llama_rope(q, pos, theta)).permute(1, 0, 2)[None]
    kr = torch.from_numpy(_llama_rope(k, pos, theta)).permute(1, 0, 2)[None]
    vv = torch.from_numpy(np.ascontiguousarray(v)).permute(1, 0, 2)[None]
    o = torch.nn.functional.scaled_dot_product_attention(qr, kr, vv, is_causal=True,
                                                         enable_gqa=q.shape[1] != k.shape[1])
    return o[0].permute(1, 0, 2).numpy()


CASES = [
    # prefix, fragment lengths, cross, Hq, Hkv, d
    (5, (7, 3, 9), 4, 4, 2, 8),
    (0, (6, 1, 4), 3, 2, 2, 4),
    (3, (1, 1), 0, 4, 1, 8),
    (8, (17,), 5, 4, 4, 6),
    (4, (), 6, 2, 1, 4),
]


@pytest.mark.parametrize("P,Ls,Q,hq,hkv,d", CASES)
def test_single_layer_reduces_to_causal_attention(P, Ls, Q, hq, hkv, d):
    theta = 1e4
    lay = A.layout(P, Ls, Q)
    n = lay.n
    q, k, v = _rand((n, hq, d), 1), _rand((n, hkv, d), 2), _rand((n, hkv, d), 3)
    out = A.span_attention(q, k, v, lay, theta)
    # prefix rows: causal attention over the prefix alone
    if P:
        ref = _causal_sdpa(q[:P], k[:P], v[:P], theta)
        np.testing.assert_allclose(out[:P], ref, atol=1e-5, rtol=0)
    # fragment i rows: causal attention over (prefix | F_i) at positions 0..P+L_i-1
    for i, L in enumerate(Ls):
        sel = np.concatenate([np.arange(P), np.nonzero(lay.seg == i)[0]])
        ref = _causal_sdpa(q[sel], k[sel], v[sel], theta)
        np.testing.assert_allclose(out[sel[P:]], ref[P:], atol=1e-5, rtol=0)
    # cross rows: causal attention over the whole sequence in query order
    if Q:
        ref = _causal_sdpa(q, k, v, theta)
        np.testing.assert_allclose(out[n - Q:], ref[n - Q:], atol=1e-5, rtol=0)


def test_one_fragment_is_plain_causal_attention():
    theta = 1e4
    lay = A.layout(6, (11,), 5)
    n = lay.n
    q, k, v = _rand((n, 4, 8), 4), _rand((n, 2, 8), 5), _rand((n, 2, 8), 6)
    np.testing.assert_allclose(A.span_attention(q, k, v, lay, theta), _causal_sdpa(q, k, v, theta),
                               atol=1e-5, rtol=0)


@pytest.mark.parametrize("P,Ls,Q", [(5, (7, 3, 9), 4), (0, (2, 5), 3), (16, (16, 32, 1), 16)])
def test_uniform_weights_closed_form(P, Ls, Q):
    """q = 0: weights are uniform over allowed keys; V one-hot by segment."""
    lay = A.layout(P, Ls, Q)
    n, nf = lay.n, len(Ls)
    d = 2 * ((nf + 3) // 2)   # even, at least nf + 2 channels
    q = np.zeros((n, 2, d))
    k = _rand((n, 1, d), 7)
    v = np.zeros((n, 1, d))
    for c in range(n):
        s = lay.seg[c]
        v[c, 0, 0 if s == A.SEG_PREFIX else (nf + 1 if s == A.SEG_CROSS else 1 + s)] = 1.0
    out = A.span_attention(q, k, v, lay, 1e4)
    for r in range(n):
        s, j = lay.seg[r], lay.idx[r]
        want = np.zeros(d)
        if s == A.SEG_PREFIX:
            want[0] = 1.0
        elif s == A.SEG_CROSS:
            tot = P + sum(Ls) + j + 1
            want[0] = P / tot
            for i, L in enumerate(Ls):
                want[1 + i] = L / tot
            want[nf + 1] = (j + 1) / tot
        else:
            tot = P + j + 1
            want[0] = P / tot
            want[1 + s] = (j + 1) / tot
        for h in range(2):
            np.testing.assert_allclose(out[r, h], want, atol=1e-14, rtol=0)


def test_mask_cardinality_and_dense_ratio():
    # C2-shaped query: prefix 256, 16 x 512 fragments, cross 128
    lay = A.layout(256, (512,) * 16, 128)
    n = lay.n
    pairs = A.allowed_pairs(lay)
    # 256*257/2 + 16*(512*256 + 512*513/2) + 128*8448 + 128*129/2
    assert pairs == 32_896 + 16 * 262_400 + 1_089_600 == 5_320_896
    assert n * (n + 1) // 2 == 36_778_176
    small = A.layout(5, (7, 3, 9), 4)
    assert int(A.span_mask(small).sum()) == A.allowed_pairs(small)


def test_rotary_relative_identity():
    theta = 1e4
    x = _rand((1, 1, 16), 8)[0]
    y = _rand((1, 1, 16), 9)[0]
    for a, b, c in [(0, 5, 100), (3, 17, 9000), (250, 260, -240)]:
        lhs = (A.rope(x[None], np.array([a]), theta)[0] * A.rope(y[None], np.array([b]), theta)[0]).sum()
        rhs = (A.rope(x[None], np.array([a + c]), theta)[0] * A.rope(y[None], np.array([b + c]), theta)[0]).sum()
        np.testing.assert_allclose(lhs, rhs, rtol=0, atol=1e-10)
    # rotation composes: R(b) applied to R(a) x equals R(a + b) x
    r1 = A.rope(A.rope(x[None], np.array([37]), theta), np.array([1200]), theta)
    r2 = A.rope(x[None], np.array([1237]), theta)
    np.testing.assert_allclose(r1, r2, atol=1e-12, rtol=0)


def test_rotary_matches_llama_convention():
    theta = 5e5
    x = _rand((9, 3, 16), 10)
    pos = np.array([0, 1, 2, 7, 31, 100, 555, 1000, 4095])
    np.testing.assert_allclose(A.rope(x, pos, theta), _llama_rope(x, pos, theta), atol=2e-4, rtol=0)


def test_permuted_children_keep_cached_kv_bit_identical():
    theta = 1e4
    P, Ls, Q = 6, (5, 9, 3), 4
    rng = np.random.default_rng(11)
    # per-content activations: fragment f has fixed rows wherever it lands
    pre_k, pre_v = rng.standard_normal((P, 2, 8)), rng.standard_normal((P, 2, 8))
    fk = [rng.standard_normal((L, 2, 8)) for L in Ls]
    fv = [rng.standard_normal((L, 2, 8)) for L in Ls]
    outs = {}
    for order in [(0, 1, 2), (2, 0, 1), (1, 2, 0)]:
        lay = A.layout(P, [Ls[i] for i in order], Q)
        k = np.concatenate([pre_k] + [fk[i] for i in order] + [np.zeros((Q, 2, 8))])
        v = np.concatenate([pre_v] + [fv[i] for i in order] + [np.zeros((Q, 2, 8))])
        for child, f in enumerate(order):
            kc, vc = A.cached_fragment_kv(k, v, lay, child, theta)
            if f in outs:
                assert np.array_equal(outs[f][0], kc) and np.array_equal(outs[f][1], vc)
            else:
                outs[f] = (kc, vc)


def test_fragment_rows_do_not_depend_on_order_or_other_fragments():
    theta = 1e4
    P, Ls, Q = 4, (6, 3, 5), 3
    rng = np.random.default_rng(12)
    pre = [rng.standard_normal((P, h, 8)) for h in (4, 2, 2)]
    fr = [[rng.standard_normal((L, h, 8)) for h in (4, 2, 2)] for L in Ls]
    cr = [rng.standard_normal((Q, h, 8)) for h in (4, 2, 2)]
    res = {}
    for order in [(0, 1, 2), (2, 1, 0)]:
        lay = A.layout(P, [Ls[i] for i in order], Q)
        q, k, v = (np.concatenate([pre[t]] + [fr[i][t] for i in order] + [cr[t]]) for t in range(3))
        out = A.span_attention(q, k, v, lay, theta)
        for child, f in enumerate(order):
            rows = out[lay.seg == child]
            if f in res:
                # same terms, summed by BLAS in a position-dependent order
                np.testing.assert_allclose(res[f], rows, atol=1e-13, rtol=0)
            else:
                res[f] = rows


def test_repositioned_cache_equals_encoding_at_final_positions():
    """Section 5.5: a cached block, rotated by (new - old) position, equals the
    block encoded at its new position."""
    theta = 1e4
    P, Ls, Q = 8, (16, 7, 12), 5
    lay = A.layout(P, Ls, Q)
    k = _rand((lay.n, 2, 8), 13)
    for child in range(len(Ls)):
        sel = np.nonzero(lay.seg == child)[0]
        kc, _ = A.cached_fragment_kv(k, k, lay, child, theta)
        delta = lay.pos_final[sel] - lay.pos_canon[sel]
        moved = A.rope(kc, delta, theta)
        np.testing.assert_allclose(moved, A.rope(k[sel], lay.pos_final[sel], theta), atol=1e-12, rtol=0)


def _brute_force(q, k, v, P, Ls, Q, theta):
    """Span attention from the rules alone, one (row, key, dim) at a time in plain
    Python floats: who may see whom (prefix causal; fragment rows see the prefix and
    their own fragment causally; cross rows see everything before them), at which
    positions (canonical for prefix/fragment rows, index in the sequence for cross
    rows), rotate-half rotary, softmax with math.exp."""
    seg, idx = [], []
    for t in range(P):
        seg.append(("p", 0)); idx.append(t)
    for i, L in enumerate(Ls):
        for j in range(L):
            seg.append(("f", i)); idx.append(j)
    for t in range(Q):
        seg.append(("c", 0)); idx.append(t)
    n = len(seg)
    hq, hkv, d = q.shape[1], k.shape[1], q.shape[2]
    half = d // 2

    def sees(r, c):
        (kr, ir), (kc, ic) = seg[r], seg[c]
        if kr == "c":
            return c <= r
        if kr == "p":
            return kc == "p" and c <= r
        return kc == "p" or (kc == "f" and ic == ir and idx[c] <= idx[r])

    def canon(t):
        return idx[t] if seg[t][0] == "p" else P + idx[t] if seg[t][0] == "f" else P + sum(Ls) + idx[t]

    def rot(x, pos):
        out = [0.0] * d
        for i in range(half):
            a = pos * theta ** (-2.0 * i / d)
            out[i] = x[i] * math.cos(a) - x[i + half] * math.sin(a)
            out[i + half] = x[i + half] * math.cos(a) + x[i] * math.sin(a)
        return out

    out = np.zeros((n, hq, d))
    for r in range(n):
        for h in range(hq):
            g = h * hkv // hq
            pos = (lambda t: t) if seg[r][0] == "c" else canon
            qr = rot([float(x) for x in q[r, h]], pos(r))
            keys = [c for c in range(n) if sees(r, c)]
            s = []
            for c in keys:
                kc = rot([float(x) for x in k[c, g]], pos(c))
                s.append(sum(qr[i] * kc[i] for i in range(d)) / math.sqrt(d))
            mx = max(s)
            w = [math.exp(x - mx) for x in s]
            z = sum(w)
            for e in range(d):
                out[r, h, e] = sum(w[j] * float(v[c, g, e]) for j, c in enumerate(keys)) / z
    return out


@pytest.mark.parametrize("P,Ls,Q,hq,hkv,d", [
    (3, (4, 1, 2), 3, 2, 1, 4),     # three fragments, one of length 1
    (0, (5, 3), 2, 2, 2, 2),        # no prefix
    (2, (6,), 0, 4, 2, 4),          # one fragment, no cross segment
    (4, (), 5, 2, 1, 6),            # no fragment
    (1, (2, 2, 2, 2), 4, 2, 1, 4),  # equal lengths (order-sensitive index errors)
])
def test_brute_force_agrees_on_tiny_inputs(P, Ls, Q, hq, hkv, d):
    n = P + sum(Ls) + Q
    q, k, v = _rand((n, hq, d), 11), _rand((n, hkv, d), 12), _rand((n, hkv, d), 13)
    lay = A.layout(P, Ls, Q)
    got = A.span_attention(q, k, v, lay, 10000.0)
    ref = _brute_force(q, k, v, P, Ls, Q, 10000.0)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-12)
