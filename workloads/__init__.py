"""Seeded synthetic inputs for the speculative-verification step.

This module only draws random numbers and lays them out; it holds none of the
method's arithmetic (no softmax, KL, acceptance or draw).  Both the HIP path
and the CPU oracle consume what it produces: inputs are generated once (on the
GPU when one is present) and copied to the host for the oracle, never
regenerated there.

Workloads (stand-ins for the paper's datasets and model pairs, whose logits
are not available here):

  tiny    B=4, SL=4 each, V=32000 fp32, target z ~ N(0, 3^2) + Zipf(1.1) rank bias,
          draft = z + N(0, 1); T=1; ring W=8 pre-filled.
  b64     B=64, SL ~ U{1..8}, V=32000 bf16, per-sequence draft noise sigma ~ U[0.3, 3];
          T=1; W=16.
  b256    B=256, SL ~ U{1..8}, V=128256 bf16 (the LLaMA-3 vocabulary of the paper's main
          pair), z ~ N(0, 4^2) + Zipf(1.05), sigma ~ U[0.2, 4]; T=0.7 for even and
          1.0 for odd sequences; W=32.
  lowacc  B=512, SL ~ U{1..16}, V=152064 bf16, draft = 0.5 z + N(0, 3^2) (a weakly
          correlated drafter: acceptance well below 0.4); T=1; W=32; SL_max=16.
  greedy  b64 with T=0 (greedy verification; drafts are the draft argmax) for even
          and T=1 for odd sequences.
  b256g   b256 with T=0 for every sequence (the temperature-0.0 setting of the
          paper's experiments).
  loop    B=1024, V=128256 bf16, 200 steps; per-sequence sigma follows a reflected
          random walk in [0.2, 4]; SL chosen each step by the controller; W=32,
          empty ring at the start; fresh logits every step.
  spread  B=256, SL ~ U{1..8}, V=32000 bf16, close drafts (sigma ~ U[0.05, 0.6]) and a
          per-sequence SL_max ~ U[4, 16] with next-step bound 16: small penalties
          SF * WVIR, so the SL rule's decisions spread over many lengths instead of
          collapsing onto SL_min.

Zipf bias: row r gets b(v) = -s * ln(rank_r(v)) with rank_r(v) = ((a_r v + c_r) mod V) + 1
and a_r coprime to V, a seeded bijection of the vocabulary, so exp(b) ~ rank^-s.
Drafted tokens are sampled from the tempered draft distribution by Gumbel-max.
Uniforms come from torch.rand (values in [0, 1)).
"""
import math
from dataclasses import dataclass, field

import numpy as np
import torch

CONFIGS = {
    "tiny": dict(B=4, sl=("fixed", 4), V=32000, dtype="fp32", sigma_z=3.0, zipf=1.1,
                 draft=("noise", 1.0, 1.0), temp=("all", 1.0), W=8, sl_max=8.0, k_max=4, prefill=True),
    "b64": dict(B=64, sl=("uniform", 1, 8), V=32000, dtype="bf16", sigma_z=3.0, zipf=1.1,
                draft=("noise", 0.3, 3.0), temp=("all", 1.0), W=16, sl_max=8.0, k_max=8, prefill=True),
    "b256": dict(B=256, sl=("uniform", 1, 8), V=128256, dtype="bf16", sigma_z=4.0, zipf=1.05,
                 draft=("noise", 0.2, 4.0), temp=("alternate", 0.7, 1.0), W=32, sl_max=8.0, k_max=8,
                 prefill=True),
    "lowacc": dict(B=512, sl=("uniform", 1, 16), V=152064, dtype="bf16", sigma_z=4.0, zipf=1.05,
                   draft=("weak", 0.5, 3.0), temp=("all", 1.0), W=32, sl_max=16.0, k_max=16,
                   prefill=True),
    "greedy": dict(B=64, sl=("uniform", 1, 8), V=32000, dtype="bf16", sigma_z=3.0, zipf=1.1,
                   draft=("noise", 0.3, 3.0), temp=("alternate", 0.0, 1.0), W=16, sl_max=8.0, k_max=8,
                   prefill=True),
    "b256g": dict(B=256, sl=("uniform", 1, 8), V=128256, dtype="bf16", sigma_z=4.0, zipf=1.05,
                  draft=("noise", 0.2, 4.0), temp=("all", 0.0), W=32, sl_max=8.0, k_max=8, prefill=True),
    # one GPU's share of b256 with the batch split eight ways (32 sequences)
    "batch8": dict(B=32, sl=("uniform", 1, 8), V=128256, dtype="bf16", sigma_z=4.0, zipf=1.05,
                   draft=("noise", 0.2, 4.0), temp=("alternate", 0.7, 1.0), W=32, sl_max=8.0, k_max=8,
                   prefill=True),
    "spread": dict(B=256, sl=("uniform", 1, 8), V=32000, dtype="bf16", sigma_z=3.0, zipf=1.1,
                   draft=("noise", 0.05, 0.6), temp=("all", 1.0), W=32, sl_max=("uniform", 4.0, 16.0),
                   sl_hi=16, k_max=8, prefill=True),
    "loop": dict(B=1024, sl=("uniform", 2, 8), V=128256, dtype="bf16", sigma_z=4.0, zipf=1.05,
                 draft=("walk", 0.2, 4.0), temp=("all", 1.0), W=32, sl_max=8.0, k_max=8, prefill=False,
                 steps=200),
}

# stream tags: each random quantity has its own generator so that changing one
# never shifts another
_TAGS = {"sl": 1, "zipf": 2, "target": 3, "draft": 4, "tokens": 5, "uacc": 6, "ures": 7, "hist": 8,
         "sigma": 9, "walk": 10, "slmax": 11}


def _seed(seed, tag, step=0):
    return (int(seed) * 1_000_003 + _TAGS[tag] * 7_919 + int(step) * 104_729) % (2 ** 63 - 1)


def _gen(device, seed, tag, step=0):
    g = torch.Generator(device=device)
    g.manual_seed(_seed(seed, tag, step))
    return g


def _np_rng(seed, tag, step=0):
    return np.random.default_rng(_seed(seed, tag, step))


@dataclass
class Step:
    """One verification step's inputs, packed as the library expects."""
    target: torch.Tensor        # [N+B, V] bf16 or fp32; rows cu_sl[b]+b+j, j = 0..SL_b (last = bonus)
    draft: torch.Tensor         # [N, V]; rows cu_sl[b]+j, j < SL_b
    sl: torch.Tensor            # [B] int32
    cu_sl: torch.Tensor         # [B+1] int32
    draft_tokens: torch.Tensor  # [N] int32
    temperature: torch.Tensor   # [B] float32
    u_acc: torch.Tensor         # [N] float32 in [0, 1)
    u_res: torch.Tensor         # [B] float32 in [0, 1)
    k_max: int
    meta: dict = field(default_factory=dict)

    @property
    def B(self):
        return int(self.sl.shape[0])

    @property
    def N(self):
        return int(self.draft.shape[0])

    @property
    def V(self):
        return int(self.target.shape[1])


@dataclass
class SignalState:
    hist: torch.Tensor    # [B, W] float32 ring of per-step mean KLD
    head: torch.Tensor    # [B] int32: slot of the next write
    count: torch.Tensor   # [B] int32: entries held (<= W)
    sl_max: torch.Tensor  # [B] float32


def sample_sl(cfg, seed, step=0):
    kind = cfg["sl"]
    B = cfg["B"]
    if kind[0] == "fixed":
        return np.full(B, kind[1], np.int32)
    lo, hi = kind[1], kind[2]
    return _np_rng(seed, "sl", step).integers(lo, hi + 1, B).astype(np.int32)


def initial_sigma(cfg, seed):
    kind = cfg["draft"]
    B = cfg["B"]
    if kind[0] == "noise" and kind[1] == kind[2]:
        return np.full(B, kind[1], np.float64)
    if kind[0] == "weak":
        return np.full(B, kind[2], np.float64)
    return _np_rng(seed, "sigma").uniform(kind[1], kind[2], B)


def walk_sigma(sigma, cfg, seed, step):
    """Reflected Gaussian random walk of the per-sequence draft noise."""
    lo, hi = cfg["draft"][1], cfg["draft"][2]
    s = sigma + 0.2 * _np_rng(seed, "walk", step).standard_normal(sigma.shape[0])
    for _ in range(4):
        s = np.where(s < lo, 2 * lo - s, s)
        s = np.where(s > hi, 2 * hi - s, s)
    return np.clip(s, lo, hi)


def temperatures(cfg):
    kind = cfg["temp"]
    B = cfg["B"]
    if kind[0] == "all":
        return np.full(B, kind[1], np.float32)
    t = np.full(B, kind[2], np.float32)
    t[0::2] = kind[1]
    return t


def _zipf_bias(rows, V, s, seed, step, device, row_offset=0):
    rng = _np_rng(seed, "zipf", step)
    a = np.empty(rows, np.int64)
    c = rng.integers(0, V, rows).astype(np.int64)
    for i in range(rows):
        while True:
            x = int(rng.integers(1, max(V, 2)))
            if math.gcd(x, V) == 1:
                a[i] = x
                break
    v = torch.arange(V, device=device, dtype=torch.int64)
    a_t = torch.as_tensor(a, device=device)[:, None]
    c_t = torch.as_tensor(c, device=device)[:, None]
    rank = (a_t * v[None, :] + c_t) % V + 1
    return -s * torch.log(rank.to(torch.float32))


def make_step(cfg, seed=0, device="cpu", step=0, sl=None, sigma=None, V=None, B=None):
    """Inputs of one step.  ``sl`` and ``sigma`` override the configured draws
    (the controller loop passes its own SLs and its walked sigmas)."""
    V = int(V or cfg["V"])
    B = int(B or cfg["B"])
    sl = np.asarray(sample_sl(cfg, seed, step) if sl is None else sl, np.int32)[:B]
    sigma = np.asarray(initial_sigma(cfg, seed) if sigma is None else sigma, np.float64)[:B]
    cu = np.zeros(B + 1, np.int32)
    cu[1:] = np.cumsum(sl)
    N = int(cu[-1])
    temp = temperatures(dict(cfg, B=B))
    dt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32

    # target logits, one sequence block after another (SL_b + 1 rows each)
    g_t = _gen(device, seed, "target", step)
    z = torch.randn((N + B, V), generator=g_t, device=device, dtype=torch.float32)
    z.mul_(cfg["sigma_z"])
    CH = 256
    for r0 in range(0, N + B, CH):
        r1 = min(N + B, r0 + CH)
        z[r0:r1] += _zipf_bias(r1 - r0, V, cfg["zipf"], seed * 131 + r0, step, device)

    # draft rows: drafted position j of sequence b pairs with target row cu[b] + b + j
    seq_of_pos = np.repeat(np.arange(B), sl)
    tgt_row = (np.arange(N) + seq_of_pos).astype(np.int64)
    g_d = _gen(device, seed, "draft", step)
    noise = torch.randn((N, V), generator=g_d, device=device, dtype=torch.float32)
    zt_rows = z[torch.as_tensor(tgt_row, device=device)]
    kind = cfg["draft"]
    sig = torch.as_tensor(sigma[seq_of_pos], device=device, dtype=torch.float32)[:, None]
    if kind[0] == "weak":
        y = kind[1] * zt_rows + sig * noise
    else:
        y = zt_rows + sig * noise
    del noise, zt_rows
    target = z.to(dt)
    del z
    draft = y.to(dt)
    del y

    # drafted tokens ~ softmax(draft / T) by Gumbel-max, row by row block; at
    # T = 0 (greedy drafting) the draft row's argmax
    g_k = _gen(device, seed, "tokens", step)
    temp_pos = torch.as_tensor(temp[seq_of_pos], device=device)[:, None]
    sampled = (temp_pos != 0).to(torch.float32)
    t_div = torch.where(temp_pos != 0, temp_pos, torch.ones_like(temp_pos))
    toks = torch.empty(N, dtype=torch.int64, device=device)
    for r0 in range(0, N, CH):
        r1 = min(N, r0 + CH)
        u = torch.rand((r1 - r0, V), generator=g_k, device=device, dtype=torch.float32)
        u.clamp_(min=1e-30)
        gumbel = -torch.log(-torch.log(u))
        toks[r0:r1] = torch.argmax(draft[r0:r1].float() / t_div[r0:r1] + gumbel * sampled[r0:r1], dim=1)

    u_acc = torch.rand(N, generator=_gen(device, seed, "uacc", step), device=device, dtype=torch.float32)
    u_res = torch.rand(B, generator=_gen(device, seed, "ures", step), device=device, dtype=torch.float32)
    return Step(target=target, draft=draft,
                sl=torch.as_tensor(sl, device=device), cu_sl=torch.as_tensor(cu, device=device),
                draft_tokens=toks.to(torch.int32), temperature=torch.as_tensor(temp, device=device),
                u_acc=u_acc, u_res=u_res, k_max=int(cfg["k_max"]),
                meta=dict(seed=seed, step=step, sigma=sigma))


def make_signal_state(cfg, seed=0, device="cpu", B=None):
    """Ring of per-step mean KLD values and SL_max.  Pre-filled rings hold W entries
    h = kappa_b * exp(0.5 g) with kappa_b log-uniform in [0.02, 2]; for every
    fourth sequence the newest five entries are tripled (a recent burst of
    disagreement, which pushes WVIR above 1)."""
    B = int(B or cfg["B"])
    W = int(cfg["W"])
    hist = np.zeros((B, W), np.float32)
    head = np.zeros(B, np.int32)
    count = np.zeros(B, np.int32)
    if cfg["prefill"]:
        rng = _np_rng(seed, "hist")
        kappa = np.exp(rng.uniform(math.log(0.02), math.log(2.0), B))
        vals = kappa[:, None] * np.exp(0.5 * rng.standard_normal((B, W)))  # oldest first
        vals[3::4, -5:] *= 3.0
        head = rng.integers(0, W, B).astype(np.int32)
        for b in range(B):
            for i in range(W):
                hist[b, (head[b] - W + i) % W] = vals[b, i]
        count[:] = W
    if isinstance(cfg["sl_max"], tuple):  # ("uniform", lo, hi): one SL_max per sequence
        sl_max = _np_rng(seed, "slmax").uniform(cfg["sl_max"][1], cfg["sl_max"][2], B).astype(np.float32)
    else:
        sl_max = np.full(B, float(cfg["sl_max"]), np.float32)
    return SignalState(hist=torch.as_tensor(hist, device=device),
                       head=torch.as_tensor(head, device=device),
                       count=torch.as_tensor(count, device=device),
                       sl_max=torch.as_tensor(sl_max, device=device))


def host_arrays(step: Step):
    """numpy copies of a step for the CPU oracle (bf16 as uint16 bit patterns)."""
    def logits(t):
        t = t.detach().cpu().contiguous()
        if t.dtype == torch.bfloat16:
            return t.view(torch.int16).numpy().view(np.uint16)
        return t.numpy()
    return dict(target=logits(step.target), draft=logits(step.draft), V=step.V,
                sl=step.sl.cpu().numpy(), cu_sl=step.cu_sl.cpu().numpy(),
                draft_tokens=step.draft_tokens.cpu().numpy(),
                temperature=step.temperature.cpu().numpy(), u_acc=step.u_acc.cpu().numpy(),
                u_res=step.u_res.cpu().numpy(), k_max=step.k_max)
