"""The span-query front-end: tree IR, high-level rewrites, lowering, serialization.

Definitions from the paper: the span query is an expression tree over C, R, F,
Plus, Cross, S, U, A, G (Def. 2 and the operator table, section 4.1); the
high-level optimizer applies its rules to a fixed point (section 5.1): C
desugaring, R desugaring through Prepare (G with max_tokens 1), plus
simplification and plus distribution; serialization parenthesises the join with
special tokens aligned to block starts, the closing token carrying the position
of its sub-tree's start (section 5.2, Def. 4, section 5.3).  Each rule is checked
on its own, then the optimizer on the paper's use cases (chat, RAG, nested
generation), then the serializer against the library's parser and the lowered
query against the planner.
"""
import random

import numpy as np
import pytest

from oracle.pool import PoolReplay
from paper_2511_02749_amd import spanquery as sq
from tests.helpers import assert_tables_match, replay_queries

spanq = pytest.importorskip("paper_2511_02749_amd")


def _lib():
    try:
        return spanq.load()
    except FileNotFoundError:
        pytest.skip("libspanq.so not built")


S1, S2, U1, U2, U3 = sq.S([1, 2, 3]), sq.S([4, 5]), sq.U([6, 7]), sq.U([8]), sq.U([9, 10, 11])
F1, F2, F3 = sq.F([20, 21]), sq.F([30, 31, 32]), sq.F([40])


def _ops(n):
    yield n
    for c in n.children:
        yield from _ops(c)


# ---- one rule at a time ------------------------------------------------------

def test_c_desugar():
    assert sq.rule_c_desugar(sq.C(S1, U1)) == sq.G(sq.Cross(S1, U1))
    assert sq.rule_c_desugar(sq.Cross(S1)) is None


def test_r_desugar_prepares_each_fragment():
    out = sq.rule_r_desugar(sq.R(F1, F2))
    assert out == sq.Plus(sq.Prepare(F1), sq.Prepare(F2))
    assert all(sq.is_prepare(c) and c.max_tokens == 1 for c in out.children)
    assert sq.rule_r_desugar(sq.Plus(F1)) is None


def test_plus_simplification():
    assert sq.rule_plus_flatten(sq.Plus(F1, sq.Plus(F2, F3))) == sq.Plus(F1, F2, F3)
    assert sq.rule_plus_flatten(sq.Plus(F1, F2)) is None
    assert sq.rule_plus_single(sq.Plus(F1)) == F1
    deep = sq.Plus(sq.Plus(F1, sq.Plus(F2)), sq.Plus(sq.Plus(F3)))
    assert sq.optimize(deep, rules=(sq.rule_plus_flatten, sq.rule_plus_single)) == sq.Plus(F1, F2, F3)


def test_cross_flattening():
    assert sq.rule_cross_flatten(sq.Cross(S1, sq.Cross(U1, U2))) == sq.Cross(S1, U1, U2)
    assert sq.rule_cross_flatten(sq.Cross(S1, U1)) is None


def test_plus_distribution():
    g1, g2 = sq.G(sq.Cross(S1, U1), 64), sq.G(sq.Cross(S1, U2), 64)
    assert sq.rule_plus_distribution(sq.Plus(g1, g2)) == sq.G(sq.Plus(sq.Cross(S1, U1), sq.Cross(S1, U2)), 64)
    # not across generates of different lengths, not over prepares, not over a lone child
    assert sq.rule_plus_distribution(sq.Plus(g1, sq.G(U2, 8))) is None
    assert sq.rule_plus_distribution(sq.Plus(sq.Prepare(F1), sq.Prepare(F2))) is None
    assert sq.rule_plus_distribution(sq.Plus(g1)) is None


# ---- the optimizer on the paper's use cases -------------------------------------

def _fixed_point(tree):
    out = sq.optimize(tree)
    assert sq.optimize(out) == out
    assert all(rule(n) is None for n in _ops(out) for rule in sq.RULES)
    return out


def test_chat_query():
    out = _fixed_point(sq.C(S1, sq.A([50, 51]), U1))
    assert out == sq.G(sq.Cross(S1, sq.A([50, 51]), U1))
    sp = sq.to_spans(out)
    assert sp.prefix == [] and sp.fragments == [] and sp.cross == [1, 2, 3, 50, 51, 6, 7]


def test_rag_query_becomes_prefix_fragments_cross():
    out = _fixed_point(sq.C(S1, sq.R(F1, F2, F3), U1))
    assert out == sq.G(sq.Cross(S1, sq.Plus(sq.Prepare(F1), sq.Prepare(F2), sq.Prepare(F3)), U1))
    sp = sq.to_spans(out)
    assert (sp.prefix, sp.fragments, sp.cross) == ([1, 2, 3], [[20, 21], [30, 31, 32], [40]], [6, 7])


def test_nested_generation_with_commutativity_hint():
    """Judge over two generated candidates (section 3.2 with the hint of section 4.3):
    plus distribution puts the join inside the inner generate, so the judge reads each
    candidate prefixed by the input that produced it, which is what the cache holds."""
    tree = sq.C(S2, sq.Plus(sq.C(S1, U1), sq.C(S1, U2)), U3)
    out = _fixed_point(tree)
    inner = sq.G(sq.Plus(sq.Cross(S1, U1), sq.Cross(S1, U2)))
    assert out == sq.G(sq.Cross(S2, inner, U3))
    calls = []

    def generate(tokens, max_tokens):
        calls.append(list(tokens))
        return [1000 + len(calls), 2000 + len(calls)]

    ex = sq.expand_generates(out, generate)
    assert calls == [[1, 2, 3, 6, 7], [1, 2, 3, 8]]
    sp = sq.to_spans(ex)
    assert sp.prefix == [4, 5] and sp.cross == [9, 10, 11]
    assert sp.fragments == [[1, 2, 3, 6, 7, 1001, 2001], [1, 2, 3, 8, 1002, 2002]]


def test_optimizer_converges_on_random_trees():
    rnd = random.Random(0)

    def tree(depth):
        if depth == 0 or rnd.random() < 0.3:
            k = rnd.randrange(4)
            return [sq.S, sq.U, sq.A, sq.F][k]([rnd.randrange(100) for _ in range(rnd.randrange(1, 4))])
        op = rnd.choice(["C", "Plus", "Cross", "G", "R"])
        if op == "R":
            return sq.R(*[sq.F([rnd.randrange(100)]) for _ in range(rnd.randrange(1, 4))])
        kids = [tree(depth - 1) for _ in range(rnd.randrange(1, 4))]
        if op == "G":
            return sq.G(kids[0], rnd.choice([1, 8, 16]))
        return sq.Node(op, children=tuple(kids))

    for _ in range(300):
        out = _fixed_point(tree(4))
        assert not any(n.op in ("C", "R") for n in _ops(out))


# ---- serialization and the library's parser -------------------------------------

def test_serialization_is_block_aligned():
    sp = sq.Spans(prefix=[1, 2, 3], fragments=[[10, 11], [20, 21, 22], []], cross=[5, 6])
    specials = sq.SpecialTokens()
    for block in (1, 2, 4, 16):
        seq = sq.serialize(sp, block, specials)
        marks = [i for i, t in enumerate(seq) if t in (specials.open, specials.sep, specials.close)]
        assert marks and all(i % block == 0 for i in marks)
        open_at = seq.index(specials.open)
        assert seq[seq.index(specials.close) + 1] == open_at
        # pads only fill the ends of blocks before a special token
        for i, t in enumerate(seq):
            if t == specials.pad:
                j = i
                while seq[j] == specials.pad:
                    j += 1
                assert seq[j] in (specials.open, specials.sep, specials.close) and j % block == 0


@pytest.mark.parametrize("block", [1, 2, 3, 16])
def test_library_parser_round_trip(block):
    _lib()
    rnd = random.Random(block)
    for _ in range(200):
        sp = sq.Spans(prefix=[rnd.randrange(500) for _ in range(rnd.randrange(0, 40))],
                      fragments=[[rnd.randrange(500) for _ in range(rnd.randrange(0, 40))]
                                 for _ in range(rnd.randrange(0, 6))],
                      cross=[rnd.randrange(500) for _ in range(rnd.randrange(0, 20))])
        if not sp.fragments:
            sp.cross = sp.prefix + sp.cross
            sp.prefix = []
        got = sq.parse(sq.serialize(sp, block), block)
        assert (got.prefix, got.fragments, got.cross) == (sp.prefix, sp.fragments, sp.cross)


def test_library_parser_rejects_malformed_streams():
    _lib()
    sp = sq.SpecialTokens()
    P, O, E, X = sp.pad, sp.open, sp.sep, sp.close
    good = [1, 2, P, P, O, 5, 6, 7, E, 8, P, P, X, 4, 9]
    assert sq.parse(good, 4).fragments == [[5, 6, 7], [8]]
    bad = {
        "OPEN not at a block start": [1, 2, P, O, 5, 6, 7, P, E, 8, P, P, X, 3, 9],
        "points to": [1, 2, P, P, O, 5, 6, 7, E, 8, P, P, X, 0, 9],
        "nested join": [1, 2, P, P, O, 5, 6, 7, O, 8, P, P, X, 4, 9],
        "not closed": [1, 2, P, P, O, 5, 6, 7, E, 8, 9],
        "inside the fragment": [1, 2, P, P, O, 5, P, 7, E, 8, P, P, X, 4, 9],
        "after the join": [1, 2, P, P, O, 5, 6, 7, E, 8, P, P, X, 4, E],
        "without the position": [1, 2, P, P, O, 5, 6, 7, E, 8, P, P, X],
    }
    for msg, seq in bad.items():
        with pytest.raises(spanq.SpanError) as e:
            sq.parse(seq, 4)
        assert msg in str(e.value), (msg, str(e.value))


# ---- down to the planner ---------------------------------------------------------

def test_rag_through_front_end_and_planner():
    """The paper's RAG example (section 3.1): the same retrieved fragments in the
    reverse order.  Through the front-end and the library's parser, span hashing
    finds every fragment again; block tables equal the oracle's replay."""
    _lib()
    rng = np.random.default_rng(0)
    frags = [sq.F(rng.integers(0, 1000, n).tolist()) for n in (37, 64, 5)]
    system, question = sq.S(rng.integers(0, 1000, 20).tolist()), sq.U(rng.integers(0, 1000, 9).tolist())
    q1 = sq.C(system, sq.R(*frags), question)
    q2 = sq.C(system, sq.R(*frags[::-1]), question)
    pool = spanq.Pool(num_q_heads=8, num_kv_heads=2, head_dim=128, num_pages=64, device=-1)
    replay = PoolReplay(64)
    for i, tree in enumerate((q1, q2)):
        wire = sq.serialize(sq.to_spans(sq.optimize(tree)), 16)
        query = sq.to_query(sq.parse(wire, 16))
        plan = pool.plan([query])
        res = replay.plan(replay_queries([query]))
        assert_tables_match(plan, res, [query])
        st = plan.stats()
        if i == 1:
            assert st["tokens_new"] == 0 and st["tokens_hit"] == 20 + 37 + 64 + 5
        plan.commit()
        replay.commit(res)
    pool.close()


def _judge_tree(n, gen_tokens=3, judge_tokens=2):
    """A judge over n generated candidates (section 6's judge/generator), at the fixed
    point of the rewrite rules: G(Cross(S, G(Plus(Cross(S1, U_i)..)), U))."""
    cands = [sq.C(S1, sq.U([100 + i])) for i in range(n)]
    tree = sq.C(S2, sq.Plus(*[sq.G(sq.Cross(*c.children), gen_tokens) for c in cands]), U3)
    tree = sq.G(tree.children[0] if tree.op == "G" else sq.Cross(*tree.children), judge_tokens)
    return _fixed_point(tree)


def test_attention_locality_eight_way_judge_becomes_three_two_way_plies():
    tree = _judge_tree(8)
    assert tree.op == "G" and sq.plies(tree) == 2          # the judge, then the distributed candidates
    out = sq.attention_locality(tree, 2)
    assert sq.plies(out) == 4                               # 3 judge plies over the candidates' generate
    # every judge reads at most two candidates or judgments, with the judge's own messages around them
    judges = []

    def walk(n, depth):
        if n.op == "G" and n.children[0].op == "Cross":
            parts = n.children[0].children
            assert parts[0] == S2 and parts[-1] == U3 and len(parts) == 3
            join = parts[1]
            kids = join.children[0].children if join.op == "G" else join.children
            assert 1 <= len(kids) <= 2
            judges.append(depth)
        for c in n.children:
            walk(c, depth + 1)
    walk(out, 0)
    assert len(judges) == 4 + 2 + 1
    # the candidates keep their order across the ply-1 judges
    leaves = []

    def cand(n):
        if n.op == "U" and n.tokens[0] >= 100:
            leaves.append(n.tokens[0])
        for c in n.children:
            cand(c)
    cand(out)
    assert leaves == [100 + i for i in range(8)]


@pytest.mark.parametrize("n,k,expect", [(8, 2, 3), (8, 3, 2), (9, 3, 2), (10, 3, 3), (24, 2, 5), (24, 24, 1)])
def test_attention_locality_plies(n, k, expect):
    out = sq.attention_locality(_judge_tree(n), k)
    assert sq.plies(out) - 1 == expect                      # judge plies (the candidates' generate aside)
    if n <= k:
        assert out == _judge_tree(n)


def test_attention_locality_runs_judges_on_outputs_alone():
    """Executed with expand_generates: 8 candidate generates (each read as input then
    output), then 4 + 2 judges as span queries of their own whose fragments are, in
    ply 1, the candidates' input and output and, in ply 2, the ply-1 judgments alone;
    the root lowers to a query over the two ply-2 judgments."""
    out = sq.attention_locality(_judge_tree(8), 2)
    gens, joins = [], []

    def generate(tokens, max_tokens):
        gens.append((list(tokens), max_tokens))
        return [500 + len(gens)] * max_tokens

    def generate_join(spans, max_tokens):
        joins.append(spans)
        return [900 + len(joins)] * max_tokens

    ex = sq.expand_generates(out, generate, generate_join)
    assert len(gens) == 8 and all(m == 3 for _, m in gens)
    assert [g[0] for g in gens] == [[1, 2, 3, 100 + i] for i in range(8)]
    assert len(joins) == 6
    # innermost first, one sub-tree after the other: ply-1 judges 0 and 1, the ply-2
    # judge over them, ply-1 judges 2 and 3, the ply-2 judge over those
    ply1 = [joins[0], joins[1], joins[3], joins[4]]
    for j, sp in enumerate(ply1):
        assert sp.prefix == [4, 5] and sp.cross == [9, 10, 11]
        assert sp.fragments == [[1, 2, 3, 100 + 2 * j] + [501 + 2 * j] * 3, [1, 2, 3, 101 + 2 * j] + [502 + 2 * j] * 3]
    assert joins[2].fragments == [[901, 901], [902, 902]] and joins[5].fragments == [[904, 904], [905, 905]]
    root = sq.to_spans(ex)
    assert root.fragments == [[903, 903], [906, 906]] and root.max_tokens == 2


def test_attention_locality_leaves_other_shapes_alone():
    chat = _fixed_point(sq.C(S1, U1))
    assert sq.attention_locality(chat, 2) == chat
    rag = _fixed_point(sq.C(S1, sq.R(F1, F2, F3), U1))
    out = sq.attention_locality(rag, 2)                     # plain fragments: judged two at a time
    assert sq.plies(out) == 2 and sq.attention_locality(rag, 3) == rag   # ceil(log2 3) judge plies
    with pytest.raises(ValueError):
        sq.attention_locality(rag, 1)
