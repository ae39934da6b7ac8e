"""Seeded synthetic workloads shaped like the paper's LLaMA-2 FFN layers.

This module only draws random inputs and turns configuration fractions into
integer counts; it holds none of the method's arithmetic, so both the HIP
path and the CPU oracle can consume what it produces.

The paper measures on LLaMA-2 7B/13B/70B with trained Deja Vu predictors and
wikitext prompts (Sec. 6.2-6.3). None of that is available, so these stand in:
  * weights W_gate, W_up [d_ff][d], W_down [d][d_ff] ~ N(0, sigma_w) in fp16;
  * a random rank-r linear predictor A [r][d], B [d_ff][r] ~ N(0, sigma_p);
  * decode inputs: per layer and per batch row an AR(1) process
    x_t = rho x_{t-1} + sqrt(1 - rho^2) eps_t with N(0, 1) marginals,
    drawn in fp64 and stored as fp16, so consecutive tokens share most of
    their active neurons as in the paper's inter-token overlap (Sec. 5.3);
  * for the batched workload, a skewed neuron popularity: a score bias
    b_i = -1.1 * sigma_s * ln(pi(i) + 1) with pi a seeded permutation and
    sigma_s = sigma_p^2 sqrt(r d) the score standard deviation (a log-Zipf
    profile with exponent 1.1).
Random streams: numpy Philox, one SeedSequence([seed, layer, tensor]) per
tensor, so any layer can be drawn alone.
"""
from __future__ import annotations

import concurrent.futures as cf
from dataclasses import dataclass, field
from fractions import Fraction as F

import numpy as np

SEED_BASE = 0x4D32430

# tensor ids inside a layer's seed sequence
_T_GATE, _T_UP, _T_DOWN, _T_PA, _T_PB, _T_X, _T_PERM = range(7)


@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    d_model: int
    d_ff: int
    pred_rank: int
    n_layers: int
    steps: int
    batch: int
    rhos: tuple
    sigma_w: float
    sigma_p: float
    k_frac: F
    fp16_frac: F
    int8_frac: F
    cache_frac: F
    zipf_bias: bool = False
    description: str = ""

    @property
    def seed(self) -> int:
        return SEED_BASE + self.index

    def counts(self):
        """(k, n_fp16, n_int8): k = floor(d_ff * k_frac); the tier boundaries are
        cumulative floors of k times the tier fractions, in exact arithmetic."""
        return tier_counts(self.d_ff, self.k_frac, self.fp16_frac, self.int8_frac)

    def cache_slots(self) -> int:
        return int(self.d_ff * self.cache_frac // 1)


def tier_counts(d_ff: int, k_frac, fp16_frac, int8_frac):
    k = int(F(d_ff) * F(k_frac) // 1)
    n16 = int(F(k) * F(fp16_frac) // 1)
    n16_8 = int(F(k) * (F(fp16_frac) + F(int8_frac)) // 1)
    return k, n16, n16_8 - n16


WORKLOADS = {
    "tiny": Workload(
        "tiny", 0, 1024, 2752, 128, 1, 16, 1, (0.9,), 0.02, 0.05,
        F(1, 4), F(1, 3), F(1, 3), F(1, 2),
        description="tiny single layer, d 1024, d_ff 2752, rank 128, top 25%, thirds, cache 50%"),
    "llama2-7b": Workload(
        "llama2-7b", 1, 4096, 11008, 256, 32, 128, 1, (0.9,), 0.02, 0.05,
        F(1, 5), F(1, 10), F(2, 5), F(3, 10),
        description="LLaMA-2-7B-shaped FFN stack, 32 layers, top 20%, tiers 10/40/50, cache 30%"),
    "llama2-13b": Workload(
        "llama2-13b", 2, 5120, 13824, 256, 40, 128, 1, (0.8,), 0.02, 0.05,
        F(3, 20), F(1, 5), F(3, 10), F(1, 5),
        description="LLaMA-2-13B-shaped FFN stack, 40 layers, top 15%, tiers 20/30/50, cache 20%"),
    "llama2-70b": Workload(
        "llama2-70b", 3, 8192, 28672, 512, 80, 64, 1, (0.9,), 0.015, 0.05,
        F(1, 10), F(1, 10), F(3, 10), F(1, 10),
        description="LLaMA-2-70B-shaped FFN stack, 80 layers, top 10%, tiers 10/30/60, "
                    "cache = 10% of the layer's fp16 FFN bytes in FP16-sized slots"),
    "llama2-7b-b8": Workload(
        "llama2-7b-b8", 4, 4096, 11008, 256, 1, 64, 8, (0.5, 0.95), 0.02, 0.05,
        F(1, 5), F(1, 10), F(2, 5), F(3, 10), zipf_bias=True,
        description="batched decode on the 7B layer, batch 8, rho 0.5/0.95 alternating, "
                    "log-Zipf neuron popularity"),
}


def _rng(seed: int, layer: int, tensor: int) -> np.random.Generator:
    return np.random.Generator(np.random.Philox(np.random.SeedSequence([seed, layer, tensor])))


def _normal_f16(rng: np.random.Generator, shape, sigma: float) -> np.ndarray:
    a = rng.standard_normal(shape, dtype=np.float32)
    a *= np.float32(sigma)
    return a.astype(np.float16)


def layer_weights(seed: int, layer: int, d: int, d_ff: int, sigma_w: float):
    """(w_gate [d_ff][d], w_up [d_ff][d], w_down [d][d_ff]) fp16. The three
    matrices come from independent streams and are drawn in parallel threads
    (numpy releases the GIL while filling large arrays)."""
    jobs = ((_T_GATE, (d_ff, d)), (_T_UP, (d_ff, d)), (_T_DOWN, (d, d_ff)))
    with cf.ThreadPoolExecutor(3) as ex:
        return tuple(ex.map(lambda j: _normal_f16(_rng(seed, layer, j[0]), j[1], sigma_w), jobs))


def layer_predictor(seed: int, layer: int, d: int, d_ff: int, r: int, sigma_p: float,
                    zipf_bias: bool = False):
    """(A [r][d] fp16, B [d_ff][r] fp16, bias fp32 [d_ff] or None)."""
    A = _normal_f16(_rng(seed, layer, _T_PA), (r, d), sigma_p)
    B = _normal_f16(_rng(seed, layer, _T_PB), (d_ff, r), sigma_p)
    bias = None
    if zipf_bias:
        perm = _rng(seed, layer, _T_PERM).permutation(d_ff)
        sigma_s = sigma_p * sigma_p * np.sqrt(float(r) * float(d))
        bias = (-1.1 * sigma_s * np.log(perm.astype(np.float64) + 1.0)).astype(np.float32)
    return A, B, bias


def layer_inputs(seed: int, layer: int, d: int, steps: int, rhos) -> np.ndarray:
    """x [steps][batch][d] fp16: row b is an AR(1) stream with rho = rhos[b]."""
    rng = _rng(seed, layer, _T_X)
    B = len(rhos)
    rho = np.asarray(rhos, np.float64)[:, None]
    out = np.empty((steps, B, d), np.float16)
    x = rng.standard_normal((B, d))
    out[0] = x.astype(np.float16)
    c = np.sqrt(1.0 - rho * rho)
    for t in range(1, steps):
        x = rho * x + c * rng.standard_normal((B, d))
        out[t] = x.astype(np.float16)
    return out


def batch_rhos(wl: Workload, batch: int | None = None) -> tuple:
    """rho of every batch row (the listed values repeat across rows)."""
    b = wl.batch if batch is None else batch
    return tuple(wl.rhos[i % len(wl.rhos)] for i in range(b))


@dataclass
class LayerData:
    """Everything one layer needs, for tests and the benchmark."""
    d_model: int
    d_ff: int
    pred_rank: int
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray
    pred_a: np.ndarray
    pred_b: np.ndarray
    bias: np.ndarray | None
    x: np.ndarray = field(repr=False)  # [steps][batch][d] fp16


def make_layer(seed: int, layer: int, d: int, d_ff: int, r: int, steps: int, rhos=(0.9,),
               sigma_w: float = 0.02, sigma_p: float = 0.05, zipf_bias: bool = False,
               weight_layer: int | None = None, draw_weights: bool = True) -> LayerData:
    """Draw one layer. `weight_layer` selects whose weights to draw (to let
    several layers of a stack share one weight set); default: this layer.
    With draw_weights=False the weight fields are None (a layer that will read
    another layer's neuron store)."""
    wl = layer if weight_layer is None else weight_layer
    if draw_weights:
        wg, wu, wd = layer_weights(seed, wl, d, d_ff, sigma_w)
    else:
        wg = wu = wd = None
    A, Bm, bias = layer_predictor(seed, layer, d, d_ff, r, sigma_p, zipf_bias)
    x = layer_inputs(seed, layer, d, steps, rhos)
    return LayerData(d, d_ff, r, wg, wu, wd, A, Bm, bias, x)


def workload_layer(wl: Workload, layer: int, steps: int | None = None, batch: int | None = None,
                   weight_layer: int | None = None, draw_weights: bool = True) -> LayerData:
    return make_layer(wl.seed, layer, wl.d_model, wl.d_ff, wl.pred_rank,
                      wl.steps if steps is None else steps, batch_rhos(wl, batch),
                      wl.sigma_w, wl.sigma_p, wl.zipf_bias, weight_layer, draw_weights)
