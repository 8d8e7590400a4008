"""Seeded synthetic inputs for Radar's decode path.

This module only draws random tensors (torch generators, fixed seeds); it holds
none of the method's arithmetic. Both the HIP path (through the binding) and the
CPU oracle consume the tensors it returns, so the two sides always see the same
inputs. Omega, the Gaussian projection the method samples once (Alg. 1,
initialisation), is drawn here and passed in as an input.

The workloads stand in for the paper's long-context decoding setups (the
16K-token prefill of the PG-19 perplexity runs, Llama-2 MHA and Llama-3 /
Mistral GQA head shapes, prompts up to 32K and beyond); none of the paper's
datasets or weights are used.
"""
from __future__ import annotations

import dataclasses
import math

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    t0: int             # context length when decoding starts
    seg_len: int        # c
    top_k: int          # k segments per query head
    n_features: int     # n random features
    window: int         # w, recent window
    dtype: str          # "f32" or "bf16" (q, K, V, out)
    steps: int          # decode steps (one append + one decode each)
    keys: str           # "gauss" | "gauss_scaled" | "clustered"
    planted: int        # planted keys per query for the "gauss*" generators

    @property
    def capacity(self) -> int:
        return self.t0 + self.steps

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def scaled(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # Tiny single-layer decode, fp32.
    "tiny": Workload("tiny", 1, 4, 4, 64, 4096, 64, 4, 128, 64, "f32", 32,
                     "gauss", 2),
    # Llama-2-7B-shaped MHA layer at 16K context.
    "llama2_16k": Workload("llama2_16k", 1, 32, 32, 128, 16384, 128, 16, 256,
                           128, "bf16", 256, "gauss_scaled", 4),
    # Long-context MHA at 128K context (the throughput workload).
    "mha_128k": Workload("mha_128k", 8, 32, 32, 128, 131072, 256, 16, 256, 256,
                         "bf16", 512, "clustered", 0),
    # Llama-3-8B-shaped GQA layer at 64K context.
    "gqa_64k": Workload("gqa_64k", 16, 32, 8, 128, 65536, 256, 16, 256, 256,
                        "bf16", 512, "clustered", 0),
    # 512K context, c close to sqrt(t), with a full index build.
    "gqa_512k": Workload("gqa_512k", 1, 32, 8, 128, 524288, 724, 32, 512, 724,
                         "bf16", 1024, "clustered", 0),
    # The paper's own Radar settings at its 16K-token prefill (n = 2048
    # features, k = 64 segments, a 1024-token window, c = sqrt(16384)) on a
    # Llama-3 / Mistral-shaped GQA layer; context only.
    "paper_16k": Workload("paper_16k", 1, 32, 8, 128, 16384, 128, 64, 2048, 1024,
                          "bf16", 256, "clustered", 0),
}

# Seeds: Omega = 1234 + index, data = 1000 * index + {0 keys, 1 values,
# 2 queries, 3 query plants}; index is the workload's 1-based position.
WORKLOAD_INDEX = {name: i + 1 for i, name in enumerate(WORKLOADS)}

N_CLUSTERS = 64          # mixture components per (batch, kv head)
CENTRE_STD = 0.73        # centre ~ N(0, CENTRE_STD^2 I)
KEY_NOISE = 0.25         # key = centre + KEY_NOISE * N(0, I)
QUERY_NOISE = 0.1        # N(0, 0.1): standard deviation 0.1
MEAN_RUN = 64            # mean run length of one mixture label


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _round(x, dtype):
    return x.to(dtype) if dtype != torch.float32 else x


def make_omega(n: int, d: int, seed: int, dtype: str, device="cpu"):
    """Omega [n][d], i.i.d. N(0,1) drawn in fp32. For bf16 workloads the values
    are rounded to bf16 (round to nearest even) and those rounded values are
    Omega for every consumer; the tensor stays fp32."""
    om = torch.randn(n, d, generator=_gen(device, seed), device=device,
                     dtype=torch.float32)
    if dtype == "bf16":
        om = om.to(torch.bfloat16).to(torch.float32)
    return om


def _clustered_slice(T, d, gen, device):
    """Keys of one (batch, kv head): a 64-component Gaussian mixture whose
    labels come in runs (each token after the first starts a new run with
    probability 1/MEAN_RUN; a run's label is uniform)."""
    centres = torch.randn(N_CLUSTERS, d, generator=gen, device=device) \
        * CENTRE_STD
    starts = torch.rand(T, generator=gen, device=device) < 1.0 / MEAN_RUN
    starts[0] = True
    run_id = torch.cumsum(starts.to(torch.long), 0) - 1
    n_runs = int(run_id[-1].item()) + 1
    run_label = torch.randint(0, N_CLUSTERS, (n_runs,), generator=gen,
                              device=device)
    keys = centres[run_label[run_id]] + KEY_NOISE * torch.randn(
        T, d, generator=gen, device=device)
    return keys, centres


@dataclasses.dataclass
class Inputs:
    """All tensors of one run.

    K, V       [B][H_kv][capacity][d]; rows [0, t0) hold the prefilled cache,
               rows at and after t0 are zero until appended.
    k_new, v_new [steps][B][H_kv][d]; the token appended at step i sits at
               position t0 + i.
    q          [steps][B][H_q][d]; the query of step i (context length
               t0 + i + 1 once the step's token is appended).
    omega      [n][d] fp32.
    """
    wl: Workload
    K: torch.Tensor
    V: torch.Tensor
    k_new: torch.Tensor
    v_new: torch.Tensor
    q: torch.Tensor
    omega: torch.Tensor

    def keys_at(self, step: int, b: int, h: int):
        """Rows [0, t0 + step) of head (b, h): the cache after `step` appends."""
        t0 = self.wl.t0
        return torch.cat([self.K[b, h, :t0], self.k_new[:step, b, h]], 0)

    def values_at(self, step: int, b: int, h: int):
        t0 = self.wl.t0
        return torch.cat([self.V[b, h, :t0], self.v_new[:step, b, h]], 0)


def make_inputs(wl: Workload, device="cpu", steps: int | None = None,
                seed_index: int | None = None) -> Inputs:
    """Draw one run's inputs for workload `wl` on `device`.

    steps overrides wl.steps (fewer pre-generated decode steps; the capacity
    of K and V is then t0 + steps)."""
    if steps is not None:
        wl = wl.scaled(steps=steps)
    idx = seed_index if seed_index is not None else WORKLOAD_INDEX.get(wl.name, 9)
    B, Hq, Hkv, d, T = wl.batch, wl.n_q_heads, wl.n_kv_heads, wl.head_dim, \
        wl.capacity
    S, t0, G = wl.steps, wl.t0, wl.group
    dt = wl.torch_dtype()
    gk, gv, gq, gp = (_gen(device, 1000 * idx + j) for j in range(4))
    omega = make_omega(wl.n_features, d, 1234 + idx, wl.dtype, device)

    K = torch.zeros(B, Hkv, T, d, device=device, dtype=dt)
    V = torch.zeros(B, Hkv, T, d, device=device, dtype=dt)
    k_new = torch.empty(S, B, Hkv, d, device=device, dtype=dt)
    v_new = torch.empty(S, B, Hkv, d, device=device, dtype=dt)
    scale = 1.0 / math.sqrt(d) if wl.keys == "gauss_scaled" else 1.0
    centres = torch.empty(B, Hkv, N_CLUSTERS, d, device=device)
    for b in range(B):
        for h in range(Hkv):
            if wl.keys == "clustered":
                keys, centres[b, h] = _clustered_slice(T, d, gk, device)
            else:
                keys = torch.randn(T, d, generator=gk, device=device) * scale
            vals = torch.randn(T, d, generator=gv, device=device) * scale
            keys = _round(keys, dt)
            vals = _round(vals, dt)
            K[b, h, :t0] = keys[:t0]
            V[b, h, :t0] = vals[:t0]
            k_new[:, b, h] = keys[t0:]
            v_new[:, b, h] = vals[t0:]
            del keys, vals

    noise = QUERY_NOISE * torch.randn(S, B, Hq, d, generator=gq, device=device)
    kv_of_q = torch.arange(Hq, device=device) // G
    if wl.keys == "clustered":
        # query = a random mixture centre of its kv head + noise; the centre
        # is drawn independently per (step, q head).
        m = torch.randint(0, N_CLUSTERS, (S, B, Hq), generator=gp,
                          device=device)
        bidx = torch.arange(B, device=device)[None, :, None]
        qf = centres[bidx, kv_of_q[None, None, :], m] + noise
    else:
        # query = sum of `planted` keys of its kv head, each from a different
        # segment that is a decode candidate from the first step on, + noise.
        c = wl.seg_len
        n_cand0 = max(1, max(0, t0 + 1 - wl.window) // c)
        npl = min(wl.planted, n_cand0)
        segs = torch.rand(S, B, Hq, n_cand0, generator=gp,
                          device=device).argsort(-1)[..., :npl]
        # (a context shorter than one segment plants on its own tokens)
        offs = torch.randint(0, min(c, t0), (S, B, Hq, npl), generator=gp,
                             device=device)
        pos = segs * c + offs                                  # < t0
        bidx = torch.arange(B, device=device)[None, :, None, None]
        hidx = kv_of_q[None, None, :, None]
        qf = K[bidx, hidx, pos].float().sum(-2) + noise
    q = _round(qf, dt).contiguous()
    return Inputs(wl, K, V, k_new, v_new, q, omega)


def small(wl: Workload, **kw) -> Workload:
    """A scaled-down copy of a workload (same generator, smaller sizes) for
    tests that must also run the oracle over every head."""
    return wl.scaled(**kw)
