"""Seeded synthetic inputs for the NVFP4 W4A4 + RAC MoE layer.

This module only draws random numbers and casts them to the storage dtypes
(float32 -> bfloat16 with round-to-nearest-even); it holds none of the
layer's arithmetic.  Both the GPU library's tests and the CPU oracle's tests
take their inputs from here.

Five workloads, each a stand-in for the paper's MoE rollout activations
(Sec. 4.1 trains an MoE 25B-A2.8B model whose layer sizes the paper does not
give):

  dense_t16_k256_n128        one dense W4A4+RAC GEMM: 16 tokens, K=256,
                             N=128, X ~ N(0,1) with 4 channels x30,
                             W ~ N(0, 0.02), K_s = 8
  moe_decode_t256_h2048      256 tokens, H=2048, E=128, top-8, I=768,
                             router logits N(0,1), X ~ N(0,1) with 1% of the
                             channels x20, W ~ N(0, 0.02), K_s = 64
  moe_prefill_t8192_h2048    as above with 8192 tokens
  moe_prefill_t4096_h4096    4096 tokens, H=4096, I=1536, 1% channels x50,
                             K_s = 128
  moe_zipf_decode_t64_h4096  64 tokens, H=4096, I=1536, expert popularity
                             Zipf(1.2) (Gumbel-top-k sampling without
                             replacement), X ~ Student-t(3), K_s = 128, and
                             injected edge cases: one all-zero token, all-zero
                             16-blocks, all-equal blocks, blocks whose E4M3
                             scale is subnormal or underflows to zero.

Random streams: SeedSequence(2607158100 + index).spawn(6) ->
(logits, X, outlier channels, W13, W2, edge cases).  Expert e's weights come
from the W13 (W2) sequence with spawn key e appended, so a test can draw any
subset of the experts on its own and leave the rest zero.
"""

from dataclasses import dataclass, field

import numpy as np
import torch

BASE_SEED = 2607158100


@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    T: int
    H: int
    E: int = 1
    k: int = 1
    I: int = 0          # expert intermediate size (MoE); 0 for the dense GEMM
    N: int = 0          # output width of the dense GEMM
    Ks: int = 0
    outlier_frac: float = 0.0
    outlier_count: int = 0
    outlier_scale: float = 1.0
    routing: str = "normal"      # "normal" | "zipf" | "none"
    zipf_s: float = 1.2
    acts: str = "normal"         # "normal" | "student_t3"
    edge_cases: bool = False
    w_std: float = 0.02

    @property
    def dense(self):
        return self.routing == "none"

    @property
    def n_outliers(self):
        if self.outlier_count:
            return self.outlier_count
        return int(round(self.outlier_frac * self.H))


WORKLOADS = {
    w.name: w for w in [
        Workload("dense_t16_k256_n128", 0, T=16, H=256, N=128, Ks=8,
                 outlier_count=4, outlier_scale=30.0, routing="none"),
        Workload("moe_decode_t256_h2048", 1, T=256, H=2048, E=128, k=8, I=768,
                 Ks=64, outlier_frac=0.01, outlier_scale=20.0),
        Workload("moe_prefill_t8192_h2048", 2, T=8192, H=2048, E=128, k=8,
                 I=768, Ks=64, outlier_frac=0.01, outlier_scale=20.0),
        Workload("moe_prefill_t4096_h4096", 3, T=4096, H=4096, E=128, k=8,
                 I=1536, Ks=128, outlier_frac=0.01, outlier_scale=50.0),
        Workload("moe_zipf_decode_t64_h4096", 4, T=64, H=4096, E=128, k=8,
                 I=1536, Ks=128, routing="zipf", acts="student_t3",
                 edge_cases=True),
    ]
}
ORDER = list(WORKLOADS)


def to_bf16(a):
    """float32 numpy -> torch.bfloat16 (round to nearest even)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)


def _seeds(index):
    return np.random.SeedSequence(BASE_SEED + index).spawn(6)


def _streams(index):
    return [np.random.default_rng(s) for s in _seeds(index)]


def make_logits(wl, rng, T=None):
    T = wl.T if T is None else T
    if wl.routing == "zipf":
        p = np.arange(1, wl.E + 1, dtype=np.float64) ** (-wl.zipf_s)
        p /= p.sum()
        perm = rng.permutation(wl.E)
        base = np.empty(wl.E, dtype=np.float64)
        base[perm] = np.log(p)          # expert perm[r] has popularity rank r
        g = rng.gumbel(size=(T, wl.E))
        return (base[None, :] + g).astype(np.float32)
    return rng.standard_normal((T, wl.E), dtype=np.float32)


def make_acts(wl, rng_x, rng_o, rng_edge, T=None, H=None):
    T = wl.T if T is None else T
    H = wl.H if H is None else H
    if wl.acts == "student_t3":
        x = rng_x.standard_t(3, size=(T, H)).astype(np.float32)
    else:
        x = rng_x.standard_normal((T, H), dtype=np.float32)
    n_out = wl.n_outliers if H == wl.H else max(1, int(round(wl.n_outliers * H / wl.H)))
    if n_out:
        ch = rng_o.choice(H, size=n_out, replace=False)
        x[:, ch] *= np.float32(wl.outlier_scale)
    if wl.edge_cases:
        amax = float(np.max(np.abs(x)))
        nb = H // 16
        x[rng_edge.integers(T)] = 0.0                                # zero token
        cells = rng_edge.choice(T * nb, size=16, replace=False)
        zero_b, equal_b, sub_b, under_b = cells[:4], cells[4:8], cells[8:12], cells[12:16]
        for c in zero_b:
            t, b = divmod(int(c), nb)
            x[t, b * 16:(b + 1) * 16] = 0.0
        for c in equal_b:
            t, b = divmod(int(c), nb)
            x[t, b * 16:(b + 1) * 16] = np.float32(rng_edge.standard_normal())
        for c in sub_b:        # block scale lands in the E4M3 subnormal range
            t, b = divmod(int(c), nb)
            x[t, b * 16:(b + 1) * 16] = (rng_edge.standard_normal(16) * amax * 1e-5).astype(np.float32)
        for c in under_b:      # block scale underflows to zero
            t, b = divmod(int(c), nb)
            x[t, b * 16:(b + 1) * 16] = (rng_edge.standard_normal(16) * amax * 1e-8).astype(np.float32)
    return x


def expert_weights(seed_seq, e, N, K, std):
    """Expert e's [N][K] float32 weights from its own stream (the bank's seed
    sequence with spawn key e), so any subset of experts can be drawn alone."""
    ss = np.random.SeedSequence(seed_seq.entropy, spawn_key=tuple(seed_seq.spawn_key) + (e,))
    return np.random.default_rng(ss).standard_normal((N, K), dtype=np.float32) * np.float32(std)


def make_bank(seed_seq, E, N, K, std, experts=None, threads=None):
    """[E][N][K] bfloat16 weights.  experts: the experts to draw (default all);
    the others are zero (full-size tests that check a sample of experts).
    Each expert has its own stream, so drawing them on a pool of threads
    gives the same bank as drawing them in order."""
    import concurrent.futures as cf
    import os
    out = torch.zeros((E, N, K), dtype=torch.bfloat16)
    todo = list(range(E)) if experts is None else [int(e) for e in experts]

    def one(e):
        out[e] = to_bf16(expert_weights(seed_seq, e, N, K, std))

    n = threads or min(16, os.cpu_count() or 1)
    if n <= 1 or len(todo) <= 1:
        for e in todo:
            one(e)
    else:
        with cf.ThreadPoolExecutor(n) as ex:
            list(ex.map(one, todo))
    return out


@dataclass
class Inputs:
    wl: Workload
    x: torch.Tensor                  # bf16 [T][H]
    logits: torch.Tensor = None      # f32 [T][E] (MoE)
    w13: torch.Tensor = None         # bf16 [E][2I][H] (MoE) or [1][N][H] dense
    w2: torch.Tensor = None          # bf16 [E][H][I]
    extra: dict = field(default_factory=dict)


def generate(name, T=None, with_weights=True, experts=None):
    """Generate a workload's inputs on the CPU.  T overrides the token count
    (same distributions, smaller batch) for oracle-sized parity cases;
    experts restricts the drawn expert weights (others zero)."""
    wl = WORKLOADS[name]
    r_logit, r_x, r_o, _r_w13, _r_w2, r_edge = _streams(wl.index)
    s_w13, s_w2 = _seeds(wl.index)[3:5]
    T = wl.T if T is None else T
    x = to_bf16(make_acts(wl, r_x, r_o, r_edge, T=T))
    if wl.dense:
        w = make_bank(s_w13, 1, wl.N, wl.H, wl.w_std) if with_weights else None
        return Inputs(wl, x, w13=w)
    logits = torch.from_numpy(make_logits(wl, r_logit, T=T))
    w13 = w2 = None
    if with_weights:
        w13 = make_bank(s_w13, wl.E, 2 * wl.I, wl.H, wl.w_std, experts)
        w2 = make_bank(s_w2, wl.E, wl.H, wl.I, wl.w_std, experts)
    return Inputs(wl, x, logits=logits, w13=w13, w2=w2)


def small_moe(name, T, H, E, k, I, Ks, seed=0, acts="normal", routing="normal",
              outlier_frac=0.01, outlier_scale=20.0, edge_cases=False):
    """A reduced MoE case with a workload's distributions at oracle size."""
    wl = Workload(f"{name}_T{T}_H{H}_E{E}_k{k}_I{I}", 100 + seed, T=T, H=H, E=E,
                  k=k, I=I, Ks=Ks, outlier_frac=outlier_frac,
                  outlier_scale=outlier_scale, routing=routing, acts=acts,
                  edge_cases=edge_cases)
    r_logit, r_x, r_o, _r_w13, _r_w2, r_edge = _streams(wl.index)
    s_w13, s_w2 = _seeds(wl.index)[3:5]
    x = to_bf16(make_acts(wl, r_x, r_o, r_edge))
    logits = torch.from_numpy(make_logits(wl, r_logit))
    w13 = make_bank(s_w13, E, 2 * I, H, wl.w_std)
    w2 = make_bank(s_w2, E, H, I, wl.w_std)
    return Inputs(wl, x, logits=logits, w13=w13, w2=w2)


def block_params(H, E, seed=0, gamma_std=0.1, router_std=0.02):
    """The block input path's parameters: the RMSNorm gain gamma [H] (about
    1, N(1, gamma_std)) and the router weights [E][H] (N(0, router_std)),
    both bf16, from their own seeded stream (the hidden state h is drawn
    like a workload's activations)."""
    rng = np.random.default_rng(np.random.SeedSequence([BASE_SEED, 7919, seed, H, E]))
    gamma = to_bf16(1.0 + gamma_std * rng.standard_normal(H))
    w_router = to_bf16(router_std * rng.standard_normal((E, H)))
    return gamma, w_router
