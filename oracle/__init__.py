"""Oracle for span-query attention and its page cache (test infrastructure).

A plain, slow, deliberately literal CPU implementation of what the span-query
hot path computes, written from the paper (Castro et al., "Using Span Queries
to Optimize for Cache and Attention Locality"):

* ``attention``: the span attention mask (prefix, commuting fragments, cross
  segment), the canonical and final position rules, rotary encoding and the
  masked softmax, in float64 (sections 4.3, 5.5 and 5.6).
* ``hashing``: the chained page hash with accumulation suspended at each
  commuting child (sections 2 and 5.4).
* ``pool``: a replay of the page cache's lookup, deduplication, allocation
  and LRU eviction rules.
* ``stack``: a Llama-shaped decoder around span attention (RMSNorm, q/k/v and
  output projections, SwiGLU, residuals, final norm, LM head, first-token
  argmax), with the bf16 storage rounding of a bf16 model as an option.

Only the test suite, the smoke check and the benchmark's CPU baseline may
import this package.  It shares no code with the HIP library and never imports
it; the product path never calls it.
"""
