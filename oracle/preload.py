"""Oracle of the SSD -> DRAM tier: the two-level DRAM cache and the layer-wise
preloader (Sec. 5.4 "Pattern-Aware Preloading for SSD", Fig. 8).

TEST INFRASTRUCTURE ONLY (tests/ and the benchmark's CPU leg use it; the
library never does). Plain Python, one decision at a time, written from the
passage:

  * every layer's neurons live in a file (the SSD);
  * the DRAM cache has a fixed area holding the first n layers, loaded once
    and never evicted (so a new token does not reload them), and a dynamic
    area of layer slots that changes as inference moves through the layers;
  * the preloader loads whole layers (no per-neuron bookkeeping, no accuracy
    impact) two or more layers ahead of the layer being computed, since one
    layer's load takes longer than one layer's compute.

Readings where the passage is silent (the library follows the same ones):
  * Decode visits layers 0, 1, ..., L-1, 0, 1, ... (one token after another).
  * When layer l is used, the window W(l) = l, l+1, ..., l+a (mod L) must be
    in DRAM or on its way: l itself is loaded first if missing (the consumer
    waits for it), then l+1 ... l+a are queued (a = look-ahead depth >= 1).
  * A missing layer takes the lowest-numbered empty dynamic slot; with none
    empty, the victim is the dynamic slot whose layer is not in W(l) and
    whose next use is furthest away, i.e. the largest (layer - l) mod L.
    With the cyclic order this is the optimal (furthest next use) choice: a
    layer just computed is evicted before one that is about to be needed.
  * If no slot can be given up, a look-ahead load is skipped (it is retried
    at the next layer); this needs at least a + 1 dynamic slots.
"""
from __future__ import annotations


class TwoLevelDram:
    """Decisions of the two-level DRAM cache for a sequence of layer uses."""

    def __init__(self, n_layers: int, fixed: int, slots: int, lookahead: int):
        if not (0 <= fixed <= n_layers and lookahead >= 1):
            raise ValueError("bad configuration")
        if fixed < n_layers and slots < lookahead + 1:
            raise ValueError("the dynamic area needs at least lookahead + 1 slots")
        self.L, self.fixed, self.a = n_layers, fixed, lookahead
        self.slot_layer = [-1] * slots
        self.log = []  # (used layer, loaded layer, slot, evicted layer or -1)

    def resident(self, m: int) -> bool:
        return m < self.fixed or m in self.slot_layer

    def use(self, l: int):
        """Layer l is about to be computed: ensure W(l) in order."""
        window = [(l + j) % self.L for j in range(self.a + 1)]
        for m in window:
            if self.resident(m):
                continue
            empty = [s for s, v in enumerate(self.slot_layer) if v < 0]
            if empty:
                s, old = empty[0], -1
            else:
                cand = [s for s, v in enumerate(self.slot_layer) if v not in window]
                if not cand:
                    if m == l:
                        raise RuntimeError("no slot for the layer in use")
                    continue
                s = max(cand, key=lambda q: (self.slot_layer[q] - l) % self.L)
                old = self.slot_layer[s]
            self.slot_layer[s] = m
            self.log.append((l, m, s, old))

    def run_tokens(self, tokens: int):
        for _ in range(tokens):
            for l in range(self.L):
                self.use(l)
        return self.log
