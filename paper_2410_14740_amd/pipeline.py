"""Decode schedule of a stack of FFN layers over three HIP streams.

Sec. 6.1 of the paper runs the neuron transfers on dedicated streams so that
they overlap computation, and Sec. 5.4 prepares layers ahead of the one being
computed. Here every layer-step is the four calls of the C ABI:

    aux stream   m2c_predict_rank, m2c_cache_plan
    copy stream  m2c_cache_fill          (waits for the plan)
    main stream  m2c_sparse_ffn          (waits for the fill)

and the aux stream of layer-step f waits for the FFN of layer-step f - lag, so
the plan and fill of a layer run while the FFN of the layer before it runs.

Ordering argument (what the events guarantee, and what the pipeline test
checks with held streams and poisoned slots):
  * a fill starts after its plan (copy waits for the plan event);
  * an FFN starts after its fill (main waits for the fill event), so it never
    reads a slot before the bytes are there;
  * the plan of layer l at step t + 1 waits for the FFN of layer-step
    f - lag with lag <= n_layers, and the main stream runs FFNs in order, so
    the FFN of layer l at step t (layer-step f - n_layers) is complete: the
    plan neither rewrites the plan buffer that FFN reads nor lets a fill
    overwrite a slot it reads (fills follow their plan).
Everything is enqueued from the host without synchronization.
"""
from __future__ import annotations


class StackSchedule:
    """Enqueues decode steps of `layers` (m2c.Layer objects) on three streams.

    k, n16, n8: top-k and tier counts for every layer. tiers: a uint8 device
    tensor [n_layers][d_ff] (batch 1) or [n_layers][batch][d_ff] for the tier
    maps. lag: how many layer-steps behind the FFN the aux stream may run (1
    or 2; at most the layer count). batch: decode rows per step (each layer
    created with max_batch >= batch); x_of / y_of then give [batch][d] rows.
    """

    def __init__(self, torch, layers, k, n16, n8, tiers, lag=2, streams=None, batch=1):
        self.torch = torch
        self.layers = layers
        self.k, self.n16, self.n8 = k, n16, n8
        self.tiers = tiers
        self.batch = batch
        n = len(layers)
        self.lag = max(1, min(lag, n))
        if streams is None:
            streams = (torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream())
        self.main, self.aux, self.copy = streams
        self.ev_plan = [torch.cuda.Event() for _ in range(n)]
        self.ev_fill = [torch.cuda.Event() for _ in range(n)]
        self.ev_ffn = [torch.cuda.Event() for _ in range(n)]
        self.enqueued = 0  # layer-steps enqueued so far

    def step(self, t, x_of, y_of, hooks=None, plan_of=None):
        """Enqueue decode step t of every layer. x_of(l) -> fp16 device rows
        [batch][d] (the tokens' inputs of layer l), y_of(l) -> fp32 device rows
        [batch][d] that the FFN adds into. plan_of(l) -> plan buffer, or None for the
        layer's own. hooks: an object whose optional methods
        before_predict / after_plan / before_fill / after_fill / before_ffn /
        after_ffn (l, t, stream) run at those points (timing events, held
        streams, poisoning, plan archiving)."""
        n = len(self.layers)

        def hook(name, l, s):
            if hooks is not None:
                fn = getattr(hooks, name, None)
                if fn is not None:
                    fn(l, t, s)

        for l in range(n):
            L = self.layers[l]
            f = self.enqueued
            if f - self.lag >= 0:
                self.aux.wait_event(self.ev_ffn[(f - self.lag) % n])
            x = x_of(l)
            plan = None if plan_of is None else plan_of(l)
            hook("before_predict", l, self.aux)
            B = self.batch
            L.predict_rank(x, B, self.k, self.n16, self.n8, None, self.tiers[l], stream=self.aux)
            L.cache_plan(self.tiers[l], B, t, stream=self.aux, plan=plan)
            hook("after_plan", l, self.aux)
            self.ev_plan[l].record(self.aux)
            self.copy.wait_event(self.ev_plan[l])
            hook("before_fill", l, self.copy)
            L.cache_fill(stream=self.copy, plan=plan)
            hook("after_fill", l, self.copy)
            self.ev_fill[l].record(self.copy)
            self.main.wait_event(self.ev_fill[l])
            hook("before_ffn", l, self.main)
            L.sparse_ffn(x, B, y_of(l), stream=self.main, plan=plan)
            hook("after_ffn", l, self.main)
            self.ev_ffn[l].record(self.main)
            self.enqueued += 1
