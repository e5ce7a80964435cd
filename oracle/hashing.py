"""Chained page hashes with accumulation suspended at commuting children.

Section 2: the cache works on fixed-size pages ("blocks", 16 tokens by
default); the hash of page i folds in the hash of page i-1, so a page is keyed
by everything before it, and a lookup returns only the longest cached prefix.

Section 5.4: at the start of an independent sub-tree the running hash is no
longer folded in, and folding resumes after it.  Here a fragment's chain starts
from a seed derived from the shared prefix's final hash only (the fragment
attends to the prefix and to itself, so its cached KV depends on exactly those
two), never from the fragments that happen to precede it in a query.

Mixing function: SplitMix64 (Steele, Lea and Flood, "Fast splittable
pseudorandom number generators", OOPSLA 2014): add the golden-ratio increment,
then the xor-shift-multiply finaliser.

Per page (tokens t_0..t_{n-1}, index i inside its span, previous value h):
    h <- mix(h xor t)            for each token (token as unsigned 32-bit)
    h <- mix(h xor (n << 32) xor i)
A tail page shorter than the page size is hashed with its true n.

Parity unpinned: nothing here; pinned against SplitMix64's published output
stream and the paper's chat example.
"""
from __future__ import annotations

from typing import List, Sequence

MASK64 = (1 << 64) - 1
GOLDEN_GAMMA = 0x9E3779B97F4A7C15
ROOT_SEED = 0x243F6A8885A308D3      # first 64 fraction bits of pi
FRAG_TAG = 0x13198A2E03707344       # next 64 fraction bits of pi


def splitmix64(x: int) -> int:
    z = (x + GOLDEN_GAMMA) & MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & MASK64
    return z ^ (z >> 31)


def page_hash(prev: int, tokens: Sequence[int], page_idx: int) -> int:
    h = prev
    for t in tokens:
        h = splitmix64(h ^ (int(t) & 0xFFFFFFFF))
    return splitmix64(h ^ ((len(tokens) << 32) & MASK64) ^ (page_idx & MASK64))


def chain(seed: int, tokens: Sequence[int], page_size: int, include_partial: bool = True) -> List[int]:
    """Hashes of the pages of one span, chained from ``seed``."""
    out, h = [], seed
    n = len(tokens)
    for p in range((n + page_size - 1) // page_size):
        page = tokens[p * page_size: (p + 1) * page_size]
        if len(page) < page_size and not include_partial:
            break
        h = page_hash(h, page, p)
        out.append(h)
    return out


def fragment_seed(prefix_hashes: Sequence[int]) -> int:
    """Seed of every fragment chain under a given prefix."""
    last = prefix_hashes[-1] if len(prefix_hashes) else ROOT_SEED
    return splitmix64(last ^ FRAG_TAG)


def query_hashes(prefix: Sequence[int], frags: Sequence[Sequence[int]], page_size: int):
    """(prefix page hashes, [page hashes of each fragment]) of one query."""
    ph = chain(ROOT_SEED, prefix, page_size)
    fs = fragment_seed(ph)
    return ph, [chain(fs, f, page_size) for f in frags]
