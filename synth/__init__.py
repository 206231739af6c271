"""Seeded synthetic inputs for the DBLast head + verification workloads.

Shared by the tests, the benchmark and the smoke check, which hand the same bytes to the HIP
library and to the CPU oracle. This module holds random draws only (and the softmax that turns
synthetic *target* logits into the target's log-probabilities); it computes nothing of the
drafter head, the sampler or the verifier.

The paper evaluates Qwen3-4B and Qwen3-8B targets (hidden sizes 2560 and 4096, vocabulary
151,936; Table "Parameter overhead"), drafted blocks of 15 tokens, 4 categories and target
sampling temperatures 0.7 to 1.5 on GSM8K, MT-Bench and HumanEval prompts. No weights or prompts
are available here, so the workloads below stand in for them with random inputs of those
shapes:

* h[b, k, r, :]  branch hidden states; for the Qwen3 shapes h = sqrt(1/2) eps + sqrt(1/2) P_{b,r}
  with eps ~ N(0, 1) and a rank-8 perturbation P_{b,r} = 8^-1/2 sum_l c_{b,r,l} u_{b,l} shared
  by every position of block b (c, u ~ N(0, 1));
* w[v, :]        LM-head rows ~ N(0, 0.02^2) (N(0, 1/d) for the tiny case), the lm_head.weight
                 layout [V, d];
* ell[b, :]      category logits ~ N(0, 1);
* target logits  g[b, k, v]: N(0, 2^2) (tiny); 3 eps + zipf(v) with
                 zipf(v) = -1.1 ln(1 + perm(v)) for one fixed random permutation perm of [0, V)
                 (Qwen3 shapes and the objective workload); 4 t_3 with t_3 Student-t with 3
                 degrees of freedom (stress); the target log-probabilities are
                 log_softmax(g / T) at sampling temperature T, computed in binary64 and stored
                 binary32; T = 0 is the greedy target (0 at the first argmax, -inf elsewhere).
"""
from __future__ import annotations

import dataclasses
import math

import torch


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    B: int            # blocks (sequences) in one step
    K: int            # drafted positions per block
    R: int            # latent categories
    d: int            # hidden size
    V: int            # vocabulary size
    dtype: str        # "f32" or "bf16" for h and w
    w_std: float      # standard deviation of the LM-head weights
    target: str       # "normal", "zipf" or "student_t"
    target_scale: float
    temperature: float
    low_rank: int     # rank of the shared per-block perturbation of h (0: none)
    seed_in: int      # seed of the input streams
    z_temp: float = 1.0
    philox_seed: int = 0

    @property
    def M(self) -> int:
        return self.B * self.K * self.R

    @property
    def positions(self) -> int:
        return self.B * self.K

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


QWEN_V = 151936

WORKLOADS = {
    # Tiny fp32 case, small enough for brute-force enumeration.
    "tiny": Workload("tiny", B=1, K=4, R=2, d=64, V=256, dtype="f32", w_std=1.0 / math.sqrt(64),
                     target="normal", target_scale=2.0, temperature=1.0, low_rank=0, seed_in=1001),
    # Qwen3-4B-shaped head.
    "qwen3_4b": Workload("qwen3_4b", B=8, K=16, R=8, d=2560, V=QWEN_V, dtype="bf16", w_std=0.02,
                         target="zipf", target_scale=3.0, temperature=0.6, low_rank=8,
                         seed_in=1002),
    # Qwen3-8B-shaped head (the benchmark workload; swept over T in {0, 0.6, 1.0, 1.5}).
    "qwen3_8b": Workload("qwen3_8b", B=16, K=16, R=8, d=4096, V=QWEN_V, dtype="bf16", w_std=0.02,
                         target="zipf", target_scale=3.0, temperature=1.0, low_rank=8,
                         seed_in=1003),
    # Training-objective reduction: 64 sequences x 32 blocks.
    "objective": Workload("objective", B=2048, K=16, R=16, d=4096, V=QWEN_V, dtype="bf16",
                          w_std=0.02, target="zipf", target_scale=3.0, temperature=1.0,
                          low_rank=8, seed_in=1004),
    # High-throughput batched decode stress.
    "stress": Workload("stress", B=256, K=8, R=4, d=4096, V=QWEN_V, dtype="bf16", w_std=0.02,
                       target="student_t", target_scale=4.0, temperature=1.0, low_rank=8,
                       seed_in=1005),
}

QWEN3_8B_TEMPERATURES = (0.0, 0.6, 1.0, 1.5)

_STREAM_H, _STREAM_W, _STREAM_ELL, _STREAM_TARGET, _STREAM_PERM, _STREAM_TRAJ = range(6)


def torch_dtype(wl: Workload):
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def _gen(wl: Workload, stream: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed_in * 16 + stream)
    return g


def make_h(wl: Workload, device="cpu", blocks=None) -> torch.Tensor:
    """Branch hidden states [B, K, R, d] in the workload dtype (rows m = (b K + k) R + r).

    ``blocks`` (a range) generates only those blocks; block b's values do not depend on which
    other blocks are generated.
    """
    blocks = range(wl.B) if blocks is None else blocks
    out = torch.empty((len(blocks), wl.K, wl.R, wl.d), dtype=torch_dtype(wl), device=device)
    for i, b in enumerate(blocks):
        g = torch.Generator(device=device)
        g.manual_seed((wl.seed_in * 16 + _STREAM_H) * 1_000_003 + b)
        eps = torch.randn((wl.K, wl.R, wl.d), generator=g, device=device, dtype=torch.float64)
        if wl.low_rank:
            c = torch.randn((wl.R, wl.low_rank), generator=g, device=device, dtype=torch.float64)
            u = torch.randn((wl.low_rank, wl.d), generator=g, device=device, dtype=torch.float64)
            P = (c @ u) / math.sqrt(wl.low_rank)
            x = math.sqrt(0.5) * eps + math.sqrt(0.5) * P[None]
        else:
            x = eps
        out[i] = x.to(torch.float32).to(torch_dtype(wl))
    return out


def make_w(wl: Workload, device="cpu") -> torch.Tensor:
    """LM-head weights [V, d] in the workload dtype."""
    g = _gen(wl, _STREAM_W, device)
    w = torch.randn((wl.V, wl.d), generator=g, device=device, dtype=torch.float32)
    return (w * wl.w_std).to(torch_dtype(wl))


def make_ell(wl: Workload, device="cpu") -> torch.Tensor:
    """Category logits [B, R] float32."""
    g = _gen(wl, _STREAM_ELL, device)
    return torch.randn((wl.B, wl.R), generator=g, device=device, dtype=torch.float32)


def _zipf_bias(wl: Workload, device) -> torch.Tensor:
    g = _gen(wl, _STREAM_PERM, device)
    perm = torch.randperm(wl.V, generator=g, device=device)
    return -1.1 * torch.log1p(perm.to(torch.float64))


def make_target_logits(wl: Workload, rows: int, device="cpu", blocks=None) -> torch.Tensor:
    """Raw target logits g [nb, rows, V] (binary64) for ``rows`` positions per block."""
    blocks = range(wl.B) if blocks is None else blocks
    bias = _zipf_bias(wl, device) if wl.target == "zipf" else None
    out = torch.empty((len(blocks), rows, wl.V), dtype=torch.float64, device=device)
    for i, b in enumerate(blocks):
        g = torch.Generator(device=device)
        g.manual_seed((wl.seed_in * 16 + _STREAM_TARGET) * 1_000_003 + b)
        if wl.target == "student_t":
            z = torch.randn((rows, wl.V), generator=g, device=device, dtype=torch.float64)
            chi = torch.randn((3, rows, wl.V), generator=g, device=device, dtype=torch.float64)
            chi2 = (chi * chi).sum(0)
            out[i] = wl.target_scale * z / torch.sqrt(chi2 / 3.0)
        else:
            e = torch.randn((rows, wl.V), generator=g, device=device, dtype=torch.float64)
            out[i] = wl.target_scale * e + (bias if bias is not None else 0.0)
    return out


def target_logprobs(g: torch.Tensor, temperature: float) -> torch.Tensor:
    """log_softmax(g / T) over the last axis in binary64, stored binary32; T = 0 is greedy."""
    if temperature == 0.0:
        top = torch.argmax(g, dim=-1, keepdim=True)
        out = torch.full(g.shape, -math.inf, dtype=torch.float32, device=g.device)
        out.scatter_(-1, top, 0.0)
        return out
    return torch.log_softmax(g.to(torch.float64) / temperature, dim=-1).to(torch.float32)


def make_logp(wl: Workload, rows: int | None = None, device="cpu", blocks=None,
              temperature: float | None = None) -> torch.Tensor:
    """Target log-probabilities [nb, rows, V] float32 (rows = K, or K + 1 with a bonus row)."""
    rows = wl.K if rows is None else rows
    blocks = range(wl.B) if blocks is None else blocks
    T = wl.temperature if temperature is None else temperature
    out = torch.empty((len(blocks), rows, wl.V), dtype=torch.float32, device=device)
    for i, b in enumerate(blocks):
        out[i] = target_logprobs(make_target_logits(wl, rows, device, blocks=[b])[0], T)
    return out


def make_trajectory(wl: Workload, logp: torch.Tensor, blocks=None) -> torch.Tensor:
    """A target trajectory x*_k ~ p_k for every block of ``logp`` [nb, K, V]: int32 [nb, K]."""
    blocks = range(logp.shape[0]) if blocks is None else blocks
    out = torch.empty((logp.shape[0], wl.K), dtype=torch.int32, device=logp.device)
    for i, b in enumerate(blocks):
        g = torch.Generator(device=logp.device)
        g.manual_seed((wl.seed_in * 16 + _STREAM_TRAJ) * 1_000_003 + b)
        probs = torch.exp(logp[i, :wl.K].to(torch.float64))
        out[i] = torch.multinomial(probs, 1, generator=g)[:, 0].to(torch.int32)
    return out


def make_uniform_logits(shape, seed: int, scale: float = 1.0, device="cpu") -> torch.Tensor:
    """N(0, scale^2) binary64 values of any shape (synthetic logits for small test cases)."""
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return scale * torch.randn(shape, generator=g, device=device, dtype=torch.float64)
