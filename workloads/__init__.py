"""Seeded synthetic inputs for MKOR's hot path.

This module holds no arithmetic of the method: it only draws the inputs that
both the HIP path and the float64 oracle consume (layer shapes, the rank-1
mean vectors a and g, the layer gradient G, the initial inverse factors), so
that both sides see exactly the same bits.

Seeds: every tensor has its own ``numpy.random.SeedSequence`` with entropy
230601685 and spawn key (config, layer, step, kind), kind 0 = a, 1 = g,
2 = G, 3 = Q of the left initial factor, 4 = Q of the right initial factor,
5 = activation token rows, 6 = output-gradient token rows, so any subset can be
regenerated on its own.

The layer sets stand in for the paper's BERT-Large pre-training and fine-tuning
runs (Wikipedia/BookCorpus, SQuAD, GLUE), which are not available here: only
the layer shapes of those models are used; values are random.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

ENTROPY = 2306_01685

KIND_A, KIND_G, KIND_GRAD, KIND_QL, KIND_QR = 0, 1, 2, 3, 4
KIND_AROWS, KIND_GROWS = 5, 6


@dataclass(frozen=True)
class Workload:
    cid: int
    name: str
    shapes: tuple            # ((d_in, d_out), ...)
    grad_dtype: str          # "fp32" or "bf16"
    gamma: float
    steps: int
    rows: int                # token rows the means a, g average over
    act_dist: str = "normal"  # "normal" or "student_t4"
    act_std: float = 1.0
    grad_row_std: float = 1e-3
    G_std: float = 1e-3
    init: str = "identity"   # "identity" or "perturbed"
    blocks: int = 1
    block_shapes: tuple = field(default=())

    @property
    def n_layers(self) -> int:
        return len(self.shapes)

    @property
    def factor_elems(self) -> int:
        return sum(i * i + o * o for i, o in self.shapes)

    @property
    def precond_flops(self) -> int:
        return sum(2 * i * o * (i + o) for i, o in self.shapes)


def _blockset(blocks, block_shapes):
    return tuple(s for _ in range(blocks) for s in block_shapes)


def _mk(cid, name, blocks, block_shapes, **kw):
    return Workload(cid=cid, name=name, shapes=_blockset(blocks, block_shapes),
                    blocks=blocks, block_shapes=tuple(block_shapes), **kw)


SINGLE_64 = _mk(1, "single-64x64", 1, [(64, 64)], grad_dtype="fp32", gamma=0.9, steps=20, rows=32)
BERT_BASE = _mk(2, "bert-base-72", 12, [(768, 768)] * 4 + [(768, 3072), (3072, 768)],
                grad_dtype="fp32", gamma=0.9, steps=50, rows=8192)
BERT_LARGE = _mk(3, "bert-large-144", 24, [(1024, 1024)] * 4 + [(1024, 4096), (4096, 1024)],
                 grad_dtype="bf16", gamma=0.9, steps=50, rows=16384)
SINGLE_8192 = _mk(4, "single-8192x8192", 1, [(8192, 8192)], grad_dtype="fp32", gamma=0.95,
                  steps=20, rows=8192, init="perturbed")
GPT2_XL = _mk(5, "gpt2-xl-192", 48, [(1600, 4800), (1600, 1600), (1600, 6400), (6400, 1600)],
              grad_dtype="bf16", gamma=0.9, steps=50, rows=32768, act_dist="student_t4")

# by workload number (bench.py --config N; the number also keys the seeded streams)
WORKLOADS = {w.cid: w for w in (SINGLE_64, BERT_BASE, BERT_LARGE, SINGLE_8192, GPT2_XL)}


def rng(cid: int, layer: int, step: int, kind: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=ENTROPY, spawn_key=(cid, layer, step, kind))
    return np.random.Generator(np.random.PCG64(ss))


def _row_mean(gen, n_rows, d, dist, std, chunk=1024):
    """Mean over n_rows rows drawn explicitly (float64 accumulation)."""
    acc = np.zeros(d, dtype=np.float64)
    done = 0
    while done < n_rows:
        m = min(chunk, n_rows - done)
        if dist == "student_t4":
            rows = gen.standard_t(4.0, size=(m, d))
        else:
            rows = gen.standard_normal(size=(m, d))
        acc += rows.sum(axis=0)
        done += m
    return (acc * (std / n_rows)).astype(np.float32)


def _mean_shortcut(gen, n_rows, d, dist, std):
    """Same distribution as the explicit row mean, drawn directly: the mean of
    n iid rows with variance v per entry has variance v / n (Student-t with 4
    degrees of freedom has variance 2; the mean is close to normal at these n).
    """
    var = 2.0 if dist == "student_t4" else 1.0
    return (gen.standard_normal(d) * (std * np.sqrt(var / n_rows))).astype(np.float32)


def rank1_vectors(w: Workload, layer: int, step: int, explicit: bool = False):
    """The rank-1 means (a, g) of one layer at one step, float32."""
    d_in, d_out = w.shapes[layer]
    ga, gg = rng(w.cid, layer, step, KIND_A), rng(w.cid, layer, step, KIND_G)
    if explicit:
        a = _row_mean(ga, w.rows, d_in, w.act_dist, w.act_std)
        g = _row_mean(gg, w.rows, d_out, "normal", w.grad_row_std)
    else:
        a = _mean_shortcut(ga, w.rows, d_in, w.act_dist, w.act_std)
        g = _mean_shortcut(gg, w.rows, d_out, "normal", w.grad_row_std)
    return a, g


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned
    as float32 holding exactly representable bf16 values (storage format of
    the bf16 gradients; NaN stays NaN)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    lsb = (b >> 16) & 1
    r = ((b + 0x7FFF + lsb) >> 16) << 16
    r = r.astype(np.uint32)
    nan = np.isnan(x)
    out = r.view(np.float32).copy()
    out[nan] = np.float32("nan")
    return out


def gradient(w: Workload, layer: int, step: int) -> np.ndarray:
    """Layer gradient G (d_in x d_out, row-major), float32 values; for bf16
    workloads the values are already rounded to bf16."""
    d_in, d_out = w.shapes[layer]
    G = rng(w.cid, layer, step, KIND_GRAD).standard_normal((d_in, d_out), dtype=np.float32)
    G *= np.float32(w.G_std)
    if w.grad_dtype == "bf16":
        G = round_to_bf16(G)
    return G


def initial_factors(w: Workload, layer: int):
    """Initial (Linv, Rinv), float32.  Identity (the paper initialises the
    factors with I), or for the perturbed init I + 0.01 Q Q^T / d with
    Q ~ N(0,1)^{d x 64} drawn independently for each factor."""
    d_in, d_out = w.shapes[layer]
    if w.init == "identity":
        return np.eye(d_in, dtype=np.float32), np.eye(d_out, dtype=np.float32)
    out = []
    for d, kind in ((d_in, KIND_QL), (d_out, KIND_QR)):
        Q = rng(w.cid, layer, 0, kind).standard_normal((d, 64))
        P = np.eye(d) + 0.01 * (Q @ Q.T) / d
        P = 0.5 * (P + P.T)
        out.append(P.astype(np.float32))
    return out[0], out[1]


def token_rows(w: Workload, layer: int, step: int, rows: int = None, dtype: str = "fp32"):
    """The token rows a layer's rank-1 means are formed from: activations
    (rows x d_in, N(0, act_std^2) or Student-t(4) scaled by act_std) and output
    gradients (rows x d_out, N(0, grad_row_std^2)), float32; for dtype "bf16"
    the values are rounded to bf16 (the storage format of such rows)."""
    d_in, d_out = w.shapes[layer]
    n = w.rows if rows is None else rows
    ga, gg = rng(w.cid, layer, step, KIND_AROWS), rng(w.cid, layer, step, KIND_GROWS)
    if w.act_dist == "student_t4":
        A = ga.standard_t(4.0, size=(n, d_in)).astype(np.float32)
    else:
        A = ga.standard_normal((n, d_in), dtype=np.float32)
    A *= np.float32(w.act_std)
    Go = gg.standard_normal((n, d_out), dtype=np.float32) * np.float32(w.grad_row_std)
    if dtype == "bf16":
        A, Go = round_to_bf16(A), round_to_bf16(Go)
    return A, Go


def custom(shapes, grad_dtype="fp32", gamma=0.9, rows=32, cid=100, steps=1, **kw) -> Workload:
    """A workload with explicit layer shapes (tests: ragged and degenerate sizes)."""
    return Workload(cid=cid, name=f"custom-{cid}", shapes=tuple(tuple(s) for s in shapes),
                    grad_dtype=grad_dtype, gamma=gamma, steps=steps, rows=rows,
                    block_shapes=tuple(tuple(s) for s in shapes), **kw)
