"""Oracle for automatic prefix caching — TEST INFRASTRUCTURE ONLY.

Only ``tests/`` may import this module; the product (``libmetro.so``,
``metro_seq_open_cached`` in ``include/metro.h``) never uses it.

The serving engine of AI Metropolis can reuse the KV cache of a prompt prefix
that an earlier request already computed (§4.1: the paper turns this common
prefix cache off for stable measurements and reports about 20% more throughput
with it on).  Reuse never changes a result -- the K/V of a position depend
only on the tokens up to it -- so what the cache decides is how many leading
prompt tokens a new request takes over instead of recomputing.  Its plain
definition, for a cache that has evicted nothing:

* a *known prefix* is the first ``16 j`` tokens of a sequence (one page is 16
  positions) that a prefill has computed while every token before them came
  from prefills too (a decode step's tokens are produced on the device, so a
  sequence adds no known prefix after its first decode step; a forked
  sequence adds none);
* a prompt of ``n`` tokens takes over the largest multiple ``k`` of 16 with
  ``k <= n - 1`` (one token is always left to compute, the one whose logits
  the prefill returns) such that its first ``k`` tokens form a known prefix.

Known prefixes outlive the sequences that computed them (the cache holds the
pages).  Here they are kept as plain tuples of token ids in a set and matched
by comparing whole prefixes; there is no page chain, no hashing and no
eviction.
"""

from __future__ import annotations

PAGE = 16


class OraclePrefixCache:
    def __init__(self, page: int = PAGE):
        self.page = page
        self.known: set[tuple] = set()
        self.seqs: dict[int, list | None] = {}   # tokens known so far, or None

    def open(self, sid: int) -> None:
        self.seqs[sid] = []

    def open_cached(self, sid: int, prompt) -> int:
        prompt = [int(t) for t in prompt]
        n = len(prompt)
        k = 0
        for j in range(1, n // self.page + 1):
            if j * self.page <= n - 1 and tuple(prompt[:j * self.page]) in self.known:
                k = max(k, j * self.page)
        self.seqs[sid] = prompt[:k]
        return k

    def prefill(self, sid: int, tokens) -> None:
        s = self.seqs[sid]
        if s is None:
            return
        s.extend(int(t) for t in tokens)
        for j in range(1, len(s) // self.page + 1):
            self.known.add(tuple(s[:j * self.page]))

    def decode(self, sid: int) -> None:
        self.seqs[sid] = None

    def fork(self, sid: int) -> None:
        self.seqs[sid] = None

    def close(self, sid: int) -> None:
        del self.seqs[sid]
