"""Span queries: the expression-tree front-end (client side).

A span query (Def. 2 and the operator table of section 4.1) is an expression tree
over
    C   chat completion            (sugar)
    R   corpus retrieval           (sugar; its children are fragments F)
    F   corpus fragment            (sugar)
    Plus   commutative join of its children's messages
    Cross  non-commutative join (concatenation in order)
    S, U, A   system, user, assistant messages (token lists)
    G   generate new tokens (``max_tokens``); Prepare = G with max_tokens 1

The high-level optimizer (section 5.1) rewrites a tree to a fixed point, applying
the first rule that matches, splicing in its right-hand side and starting over:
    C(x..)                 -> G(Cross(x..))                    C desugaring
    R(F1..Fn)              -> Plus(Prepare(F1) .. Prepare(Fn))   R desugaring
    Plus(.. Plus(y..) ..)  -> Plus(.. y.. ..)                   plus simplification
    Plus(x)                -> x                                 (a join of one child)
    Cross(.. Cross(y..) ..) -> Cross(.. y.. ..)                 (concatenation is associative)
    Plus(G(x1) .. G(xn))   -> G(Plus(x1 .. xn))                 plus distribution
The last rule moves the commutative join inside the generate: the generate then
runs once per child, and its output is presented prefixed by that child's input
(the "dual output" of section 2: what the cache holds is input followed by
output), so a later reader of the outputs reads exactly what is cached.

Attention locality (section 6, ``attention_locality``): a judge over n candidates
becomes a tree reduction of k-way judges, so that no generate attends to more than k
candidates at once.

Lowering (``to_spans``) maps an optimized RAG / judge-shaped tree
G(Cross(before.., Plus(children..), after..)) to the library's span query:
the messages before the join are the shared prefix, each child of the join is a
fragment (a Prepare or a message list; a fragment's tokens are its messages'
tokens), the messages after it are the cross segment.

Serialization (section 5.2, Def. 4, and block alignment of section 5.3): the
parenthesised token stream
    before..  OPEN child1..  SEP child2..  ...  CLOSE n  after..
where every special token starts a block (PAD tokens fill the rest of the block
before it) and n, the token after CLOSE, is the sequence position of the OPEN
that began the sub-tree (the variant the paper uses so that the server needs no
parsing stack).  The library parses such a stream with
``span_parse_serialized``.
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

from . import _lib

MESSAGE_KINDS = ("S", "U", "A")


@dataclass(frozen=True)
class Node:
    op: str                                   # C R F Plus Cross S U A G
    children: Tuple["Node", ...] = ()
    tokens: Tuple[int, ...] = ()              # messages and fragments
    max_tokens: int = 0                       # G

    def __post_init__(self):
        if self.op not in ("C", "R", "F", "Plus", "Cross", "S", "U", "A", "G"):
            raise ValueError(f"unknown operator {self.op}")
        if self.op in MESSAGE_KINDS + ("F",) and self.children:
            raise ValueError(f"{self.op} is a leaf")
        if self.op == "R" and any(c.op != "F" for c in self.children):
            raise ValueError("R retrieves fragments F")
        if self.op == "G" and len(self.children) != 1:
            raise ValueError("G takes one child")


def msg(kind: str, tokens: Sequence[int]) -> Node:
    return Node(kind, tokens=tuple(int(t) for t in tokens))


def S(tokens):
    return msg("S", tokens)


def U(tokens):
    return msg("U", tokens)


def A(tokens):
    return msg("A", tokens)


def F(tokens):
    return Node("F", tokens=tuple(int(t) for t in tokens))


def R(*frags: Node) -> Node:
    return Node("R", children=tuple(frags))


def C(*children: Node) -> Node:
    return Node("C", children=tuple(children))


def Plus(*children: Node) -> Node:
    return Node("Plus", children=tuple(children))


def Cross(*children: Node) -> Node:
    return Node("Cross", children=tuple(children))


def G(child: Node, max_tokens: int = 0) -> Node:
    return Node("G", children=(child,), max_tokens=int(max_tokens))


def Prepare(child: Node) -> Node:
    return G(child, max_tokens=1)


def is_prepare(n: Node) -> bool:
    return n.op == "G" and n.max_tokens == 1


# ---------------------------------------------------------------- rewrites

def rule_c_desugar(n: Node) -> Optional[Node]:
    if n.op == "C":
        return G(Cross(*n.children))
    return None


def rule_r_desugar(n: Node) -> Optional[Node]:
    if n.op == "R":
        return Plus(*[Prepare(f) for f in n.children])
    return None


def rule_plus_flatten(n: Node) -> Optional[Node]:
    if n.op == "Plus" and any(c.op == "Plus" for c in n.children):
        out = []
        for c in n.children:
            out.extend(c.children if c.op == "Plus" else (c,))
        return Plus(*out)
    return None


def rule_plus_single(n: Node) -> Optional[Node]:
    if n.op == "Plus" and len(n.children) == 1:
        return n.children[0]
    return None


def rule_cross_flatten(n: Node) -> Optional[Node]:
    if n.op == "Cross" and any(c.op == "Cross" for c in n.children):
        out = []
        for c in n.children:
            out.extend(c.children if c.op == "Cross" else (c,))
        return Cross(*out)
    return None


def rule_plus_distribution(n: Node) -> Optional[Node]:
    # every child a generate of the same kind (max_tokens), at least two of them;
    # Prepare children are left alone: their output is discarded, not read
    if (n.op == "Plus" and len(n.children) >= 2 and all(c.op == "G" for c in n.children)
            and len({c.max_tokens for c in n.children}) == 1 and not is_prepare(n.children[0])):
        return G(Plus(*[c.children[0] for c in n.children]), max_tokens=n.children[0].max_tokens)
    return None


RULES = (rule_c_desugar, rule_r_desugar, rule_plus_flatten, rule_plus_single, rule_cross_flatten,
         rule_plus_distribution)


def _rewrite_once(n: Node, rules) -> Optional[Node]:
    """Apply the first rule that matches anywhere in the tree (pre-order, node before
    its children, rules in order); None if nothing matches."""
    for rule in rules:
        out = rule(n)
        if out is not None:
            return out
    for i, c in enumerate(n.children):
        out = _rewrite_once(c, rules)
        if out is not None:
            kids = list(n.children)
            kids[i] = out
            return Node(n.op, children=tuple(kids), tokens=n.tokens, max_tokens=n.max_tokens)
    return None


def optimize(n: Node, rules=RULES, max_steps: int = 10_000) -> Node:
    """The high-level optimizer: rewrite to a fixed point."""
    for _ in range(max_steps):
        out = _rewrite_once(n, rules)
        if out is None:
            return n
        n = out
    raise RuntimeError("the rewrite did not converge")


# ---------------------------------------------------------------- attention locality

def _is_join(n: Node) -> bool:
    """A commutative join, plain or inside a distributed generate G(Plus(..))."""
    return n.op == "Plus" or (n.op == "G" and not is_prepare(n) and n.children[0].op == "Plus")


def attention_locality(tree: Node, k: int = 2) -> Node:
    """Section 6: a judge over n candidates, G(Cross(before.., join, after..)), becomes
    a tree reduction of k-way judges: the candidates are judged k at a time (each
    judge G(Cross(before.., join of k candidates, after..)) with the root's
    max_tokens), then the judgments k at a time, and so on, ceil(log_k n) plies in
    all, the last one being the root.  A judge reads the judgments of the ply below
    as plain outputs (A(out) once the generates have run), so every generate attends
    to at most k candidates.  A group of one judgment passes through unjudged.
    Apply it to a tree at the fixed point of the section 5.1 rules and do not
    optimize the result again: plus distribution would turn the judgments' join back
    into one generate.  Trees of another shape, or with at most k candidates, come
    back unchanged."""
    if k < 2:
        raise ValueError("k must be at least 2")
    if tree.op != "G" or is_prepare(tree):
        return tree
    body = tree.children[0]
    parts = list(body.children) if body.op == "Cross" else [body]
    joins = [i for i, c in enumerate(parts) if _is_join(c)]
    if len(joins) != 1:
        return tree
    j = joins[0]
    before, join, after = parts[:j], parts[j], parts[j + 1:]
    if join.op == "G":  # the candidates are generated: each group stays one distributed generate
        items = list(join.children[0].children)
        group = lambda xs: G(Plus(*xs), max_tokens=join.max_tokens)  # noqa: E731
    else:
        items = list(join.children)
        group = lambda xs: Plus(*xs)  # noqa: E731
    if len(items) <= k:
        return tree
    judge = lambda inner: G(Cross(*before, inner, *after), max_tokens=tree.max_tokens)  # noqa: E731
    level = [judge(group(items[i:i + k])) for i in range(0, len(items), k)]
    while len(level) > k:
        level = [judge(Plus(*level[i:i + k])) if len(level[i:i + k]) > 1 else level[i]
                 for i in range(0, len(level), k)]
    return judge(Plus(*level)) if len(level) > 1 else level[0]


def plies(tree: Node) -> int:
    """Generates on the longest root-to-leaf path (the root counts; Prepare does not)."""
    own = 1 if tree.op == "G" and not is_prepare(tree) else 0
    return own + max((plies(c) for c in tree.children), default=0)


# ---------------------------------------------------------------- inner generates

def expand_generates(tree: Node, generate, generate_join=None) -> Node:
    """Run the generates nested inside the root (innermost first) with
    ``generate(tokens, max_tokens) -> output tokens`` and splice in what their readers
    see: for a distributed G(Plus(x1..xn)), Plus(Cross(x1, A(out1)) .. Cross(xn,
    A(outn))), each child's output prefixed by its input; for any other inner G(x),
    A(out) alone.  An inner generate whose body holds a join (a judge of a tree
    reduction) is a span query of its own: it runs as
    ``generate_join(spans, max_tokens)`` on its lowering, or, without that callback,
    through ``generate`` on its tokens in sequence order.  Prepare nodes are left for
    the lowering (their output is never read)."""
    def walk(n: Node, root: bool) -> Node:
        kids = tuple(walk(c, False) for c in n.children)
        n = Node(n.op, children=kids, tokens=n.tokens, max_tokens=n.max_tokens)
        if root or n.op != "G" or is_prepare(n):
            return n
        body = n.children[0]
        if body.op == "Plus":
            return Plus(*[Cross(c, A(generate(_message_tokens(c), n.max_tokens))) for c in body.children])
        if body.op == "Cross" and any(c.op == "Plus" for c in body.children):
            sp = to_spans(n)
            if generate_join is not None:
                return A(generate_join(sp, n.max_tokens))
            return A(generate(sp.prefix + [t for f in sp.fragments for t in f] + sp.cross, n.max_tokens))
        return A(generate(_message_tokens(body), n.max_tokens))
    return walk(tree, True)


# ---------------------------------------------------------------- lowering

def _message_tokens(n: Node) -> List[int]:
    """Tokens of a message-valued sub-tree: messages, fragments, their Cross, and the
    input of a Prepare (whose generated token is discarded)."""
    if n.op in MESSAGE_KINDS + ("F",):
        return list(n.tokens)
    if n.op == "Cross":
        return [t for c in n.children for t in _message_tokens(c)]
    if is_prepare(n):
        return _message_tokens(n.children[0])
    raise ValueError(f"{n.op} is not a message sub-tree here")


@dataclass
class Spans:
    """A lowered span query: shared prefix, commuting fragments (in this query's
    order), cross segment; max_tokens of the outer generate."""
    prefix: List[int]
    fragments: List[List[int]]
    cross: List[int]
    max_tokens: int = 0


def to_spans(tree: Node) -> Spans:
    """Lower an optimized tree of the form G(Cross(before.., Plus(..), after..)) (or a
    G over a single Cross with no join: no fragments) to spans."""
    if tree.op != "G":
        raise ValueError("the root of a span query to run is a generate")
    body = tree.children[0]
    parts = list(body.children) if body.op == "Cross" else [body]
    joins = [i for i, c in enumerate(parts) if c.op == "Plus"]
    if len(joins) > 1:
        raise ValueError("one commutative join per query")
    if not joins:
        return Spans(prefix=[], fragments=[], cross=[t for c in parts for t in _message_tokens(c)],
                     max_tokens=tree.max_tokens)
    j = joins[0]
    return Spans(prefix=[t for c in parts[:j] for t in _message_tokens(c)],
                 fragments=[_message_tokens(c) for c in parts[j].children],
                 cross=[t for c in parts[j + 1:] for t in _message_tokens(c)], max_tokens=tree.max_tokens)


# ---------------------------------------------------------------- serialization

@dataclass(frozen=True)
class SpecialTokens:
    """Token ids of the special tokens (section 5.2 table): PAD (block alignment),
    OPEN "(", SEP ")(", CLOSE ")" (followed by the position of its OPEN)."""
    pad: int = -1
    open: int = -2
    sep: int = -3
    close: int = -4


def _pad_to_block(seq: List[int], block: int, pad: int):
    while len(seq) % block:
        seq.append(pad)


def serialize(spans: Spans, block: int, sp: SpecialTokens = SpecialTokens()) -> List[int]:
    """Block-aligned parenthesised stream of a lowered span query."""
    seq = list(spans.prefix)
    if spans.fragments:
        _pad_to_block(seq, block, sp.pad)
        open_at = len(seq)
        for i, f in enumerate(spans.fragments):
            seq.append(sp.open if i == 0 else sp.sep)
            seq.extend(f)
            _pad_to_block(seq, block, sp.pad)
        seq.extend([sp.close, open_at])
    seq.extend(spans.cross)
    return seq


@dataclass
class SpanTokens:
    tokens: np.ndarray
    row: int

    @property
    def n(self) -> int:
        return int(self.tokens.shape[0])


@dataclass
class Query:
    """A query in the form span_plan takes (prefix, fragments, cross; caller rows)."""
    prefix: SpanTokens
    frags: List[SpanTokens]
    cross: SpanTokens


def to_query(spans: Spans, row0: int = 0) -> Query:
    """The planner's form of lowered spans, rows numbered from row0 in sequence order."""
    at = row0
    out = []
    for toks in [spans.prefix, *spans.fragments, spans.cross]:
        out.append(SpanTokens(tokens=np.asarray(toks, np.int32), row=at))
        at += len(toks)
    return Query(prefix=out[0], frags=out[1:-1], cross=out[-1])


def parse(tokens: Sequence[int], block: int, sp: SpecialTokens = SpecialTokens()) -> Spans:
    """Parse a serialized stream with the library (span_parse_serialized)."""
    lib = _lib.load()
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    special = (ctypes.c_int32 * 4)(sp.pad, sp.open, sp.sep, sp.close)
    n_frags = ctypes.c_int32()
    prefix, cross = _lib.SpanRange(), _lib.SpanRange()
    _lib._check(lib.span_parse_serialized(_lib._i32p(t), t.size, block, special, None, 0, ctypes.byref(n_frags),
                                          ctypes.byref(prefix), ctypes.byref(cross)))
    frags = (_lib.SpanRange * max(1, n_frags.value))()
    _lib._check(lib.span_parse_serialized(_lib._i32p(t), t.size, block, special, frags, n_frags.value,
                                          ctypes.byref(n_frags), ctypes.byref(prefix), ctypes.byref(cross)))
    cut = lambda r: [int(x) for x in t[r.begin: r.begin + r.n]]  # noqa: E731
    return Spans(prefix=cut(prefix), fragments=[cut(frags[i]) for i in range(n_frags.value)], cross=cut(cross))
