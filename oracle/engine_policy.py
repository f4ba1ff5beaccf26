"""Admission rule of mixed continuous batching -- TEST INFRASTRUCTURE ONLY.

The plain definition of which requests a forward pass carries, written from
the paper's priority rule (§3.5: every request carries its agent's step, and
requests with smaller steps run first; no request is preempted during
inference) and the chunked prefill it cites as prior art (§5):

1. every running request (its prompt is in, outputs remain) gets its next
   token as a one-token item, in priority order, while items remain;
2. the tokens left of the forward's budget go to waiting requests in priority
   order, at most ``chunk`` prompt tokens each, until the items or the budget
   run out;
3. priority order: lowest step first, ties by submission order (or
   submission order alone without priority).

A request becomes running once its last prompt chunk has been prefilled (that
forward yields its first output token) and is retired after ``n_out`` tokens.
"""

from __future__ import annotations


class Request:
    def __init__(self, rid, step, arrival, n_prompt, n_out):
        self.rid, self.step, self.arrival = rid, step, arrival
        self.n_prompt, self.n_out = n_prompt, n_out
        self.off = 0
        self.produced = 0

    @property
    def running(self):
        return self.off == self.n_prompt and self.produced < self.n_out

    @property
    def waiting(self):
        return self.off < self.n_prompt


def order_key(r: Request, priority: bool):
    return (r.step, r.arrival) if priority else (r.arrival,)


def plan(requests, max_tokens: int, chunk: int, max_items: int, priority: bool):
    """[(request id, tokens, is a decode token)] of the next forward."""
    items = []
    for r in sorted([r for r in requests if r.running], key=lambda r: order_key(r, priority)):
        if len(items) == max_items:
            break
        items.append((r.rid, 1, True))
    budget = max_tokens - len(items)
    for r in sorted([r for r in requests if r.waiting], key=lambda r: order_key(r, priority)):
        if len(items) == max_items or budget <= 0:
            break
        take = min(chunk, r.n_prompt - r.off, budget)
        items.append((r.rid, take, False))
        budget -= take
    return items


def apply(requests, items):
    """Advance the requests by one forward's items; return the ids retired."""
    by_id = {r.rid: r for r in requests}
    done = []
    for rid, take, is_decode in items:
        r = by_id[rid]
        if is_decode:
            r.produced += 1
        else:
            r.off += take
            if r.off < r.n_prompt:
                continue
            r.produced += 1
        if r.produced == r.n_out:
            done.append(rid)
    return done
