"""The four KV-cache regions of the decode phase and attention over them.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper: Sec. "Decode Phase" / "Buffer Update".  The cache is kept as four
contiguous regions: Sink (a few early tokens, attended densely), Retrieval
(historical tokens, indexed and searched), Local (the most recent
``local`` tokens, attended densely) and the Update Buffer (newly generated
tokens).  Each new token goes to the Update Buffer; when the buffer holds
``m`` tokens, the oldest ``m`` tokens of Local are evicted into Retrieval
(and encoded), and the buffered tokens are promoted into Local so that
Local again holds the most recent ``local`` tokens.  Sec. "Experiments"
(setup) uses sink 128, local 512 and updates every 256 or 512 steps.

This module replays that update rule token by token with explicit lists of
token positions (no closed form), so it can be read against the paper:

  * ``Regions`` holds the position lists of the four regions;
  * ``after_prefill`` lays out a prompt of P tokens: the first ``sink``
    tokens are Sink, the last ``local`` tokens (of those not in Sink) are
    Local, the rest is Retrieval, the buffer is empty;
  * ``decode_step`` appends one token and, when the buffer is full,
    performs the eviction / promotion.

Readings (where the paper leaves a detail open):
  * a prompt shorter than ``sink + local`` puts as many tokens as fit into
    Sink, then Local; Retrieval starts empty;
  * when Local holds fewer than ``m`` tokens at an update, every token of
    Local plus the oldest buffered tokens beyond the ``local`` most recent
    ones move to Retrieval, i.e. Local becomes exactly the most recent
    ``local`` tokens of Local + Buffer;
  * the attention of a decode step covers Sink, the retrieved tokens, Local
    and the Update Buffer (buffered tokens are recent context and are
    attended densely before their promotion).

``window_attention`` is the float64 softmax attention over the union of
the dense rows and the retrieved rows (Eqs. approx_weight, approx_output
with C(q) = Sink + retrieved + Local + Buffer).
"""

from dataclasses import dataclass, field

import numpy as np

from .attention import sparse_attention


@dataclass
class Regions:
    sink: list = field(default_factory=list)
    retrieval: list = field(default_factory=list)
    local: list = field(default_factory=list)
    buffer: list = field(default_factory=list)
    sink_size: int = 128
    local_size: int = 512
    update_every: int = 256

    @property
    def length(self):
        return len(self.sink) + len(self.retrieval) + len(self.local) + len(self.buffer)


def after_prefill(P, sink=128, local=512, m=256):
    """Regions right after a prompt of P tokens (positions 0 .. P-1)."""
    R = Regions(sink_size=sink, local_size=local, update_every=m)
    tokens = list(range(P))
    R.sink = tokens[:sink]
    rest = tokens[sink:]
    n_local = min(local, len(rest))
    R.local = rest[len(rest) - n_local:]
    R.retrieval = rest[:len(rest) - n_local]
    return R


def decode_step(R):
    """Append the next token; run the buffer update when the buffer is full.

    Returns the list of positions moved into Retrieval by this step (the keys
    to encode and index), empty when no update happened."""
    R.buffer.append(R.length)
    if len(R.buffer) < R.update_every:
        return []
    # (i) the oldest tokens of Local go to Retrieval, (ii) the buffered tokens
    # are promoted so that Local keeps the most recent `local_size` tokens.
    merged = R.local + R.buffer
    keep = min(R.local_size, len(merged))
    evicted = merged[:len(merged) - keep]
    R.retrieval = R.retrieval + evicted
    R.local = merged[len(merged) - keep:]
    R.buffer = []
    return evicted


def dense_rows(R):
    """Positions attended densely at this step: Sink, Local and the Update Buffer."""
    return R.sink + R.local + R.buffer


def window_attention(q, K, V, dense, retrieved, scale=1.0):
    """Softmax attention over dense + retrieved rows (float64).

    ``retrieved`` are K/V row positions; -1 entries are ignored.  The two
    lists must not share a position (each row is counted once per entry)."""
    retrieved = [int(r) for r in np.asarray(retrieved).ravel() if r >= 0]
    rows = list(dense) + retrieved
    return sparse_attention(q, K, V, np.asarray(rows, dtype=np.int64), scale)
