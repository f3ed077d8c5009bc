"""Seeded synthetic inputs for the MoE expert stage.

This module only draws inputs: token activations, expert weights, routing
(expert ids and combine weights) and micro-batch lengths.  It performs none of
the stage's arithmetic (no dispatch, no FFN, no combine) and is the one piece of
code shared by the HIP path and the CPU oracle.

Shapes follow the DeepSeek-V3 layer the paper evaluates (hidden size 7168,
256 routed experts, top-8 routing plus one shared expert; Table 1 and the
evaluation methodology).  The paper's production length trace and model
weights are not available, so lognormal lengths, Zipf or uniform routing and
Gaussian weights stand in for them.

Random streams.  A ``numpy.random.SeedSequence(seed)`` is split into eight
children, in this order: lengths, routing, logits, x, W_gate, W_up, W_down,
shared.  Routing, logits and lengths are drawn with numpy on the host.  Large
float tensors (activations and weights) are drawn with ``torch.randn`` from a
``torch.Generator`` on the requested device, seeded from the matching child;
values are drawn in fp32, scaled, and rounded to bf16 (round to nearest even).
On a given device the inputs are therefore a pure function of (config, seed).

fp8 weights (the fp8 variant) are prepared offline, as a model checkpoint
would be: each 128x128 block of a bf16 weight gets an fp32 scale
amax/448 and is cast to OCP e4m3 with torch's conversion.  Activation
quantisation is *not* done here: it is a step of the stage (the sender-side
quantiser) and both the HIP path and the oracle implement it themselves.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional

import numpy as np
import torch

__all__ = [
    "MoEConfig", "CONFIGS", "MicroBatch", "ExpertWeights",
    "make_config_inputs", "make_weights", "make_microbatches",
    "draw_lengths", "draw_routing",
]

_STREAMS = ("lengths", "routing", "logits", "x", "w_gate", "w_up", "w_down", "shared")


@dataclasses.dataclass(frozen=True)
class MoEConfig:
    """One synthetic workload of the expert stage.

    ``lengths`` fixes the micro-batch token counts; when it is None,
    ``n_micro`` lengths are drawn from clip(rint(exp(mu + sigma z)), lo, hi).
    """
    name: str
    d: int                     # hidden size (paper: H)
    f: int                     # expert intermediate size
    E: int                     # routed experts in the model (paper: E_total)
    e0: int                    # first local expert id
    E_loc: int                 # local experts on this device
    k: int                     # top-k
    lengths: Optional[tuple] = None
    n_micro: int = 1
    lognormal: tuple = (7.0, 1.0, 16, 8192)
    routing: str = "uniform"   # "uniform" | "zipf"
    zipf_s: float = 1.2
    dead_local: tuple = ()     # local expert ids that receive no token (zipf)
    has_shared: bool = False
    dtype: str = "bf16"        # "bf16" | "fp8"
    x_std: float = 1.0
    w_std: float = 0.02
    seed: int = 0

    @property
    def max_tokens(self) -> int:
        if self.lengths is not None:
            return max(self.lengths) if self.lengths else 0
        return self.lognormal[3]


CONFIGS = {
    # Tiny layer: 8 experts, 0-3 local, top-2.
    "c0": MoEConfig("c0", d=256, f=128, E=8, e0=0, E_loc=4, k=2, lengths=(64,)),
    # DeepSeek-V3 EP32 share: 8 of 256 experts local, top-8, T=4096.
    "c1": MoEConfig("c1", d=7168, f=2048, E=256, e0=0, E_loc=8, k=8, lengths=(4096,)),
    # Same share at T=32768 (the paper's maximum batch S), i.e. about 1024
    # token-slots per local expert.
    "c1p": MoEConfig("c1p", d=7168, f=2048, E=256, e0=0, E_loc=8, k=8, lengths=(32768,)),
    # Skewed ragged routing: 4 lognormal micro-batches, Zipf(1.2) expert choice,
    # local experts 6 and 7 receive nothing.
    "c2": MoEConfig("c2", d=7168, f=2048, E=256, e0=0, E_loc=8, k=8, n_micro=4,
                    routing="zipf", dead_local=(6, 7)),
    # EP8 share: 32 local experts plus an always-on shared expert, T=16384.
    "c3": MoEConfig("c3", d=7168, f=2048, E=256, e0=0, E_loc=32, k=8, lengths=(16384,),
                    has_shared=True),
    # fp8 (e4m3, 128-block scales) variant of c2.
    "c4": MoEConfig("c4", d=7168, f=2048, E=256, e0=0, E_loc=8, k=8, n_micro=4,
                    routing="zipf", dead_local=(6, 7), dtype="fp8"),
    # fp8 variants of the MFMA-bound shapes, for the fp8 kernel's own rates.
    "c1p_fp8": MoEConfig("c1p_fp8", d=7168, f=2048, E=256, e0=0, E_loc=8, k=8, lengths=(32768,),
                         dtype="fp8"),
    "c3_fp8": MoEConfig("c3_fp8", d=7168, f=2048, E=256, e0=0, E_loc=32, k=8, lengths=(16384,),
                        has_shared=True, dtype="fp8"),
}


@dataclasses.dataclass
class MicroBatch:
    x: torch.Tensor         # [T, d] bf16 (on the generation device)
    ids: np.ndarray         # [T, k] int32, -1 = masked slot
    w: np.ndarray           # [T, k] float32 combine weights


@dataclasses.dataclass
class ExpertWeights:
    """Local expert weights as the checkpoint stores them.

    bf16: w_gate/w_up [E_loc, f, d], w_down [E_loc, d, f] bf16.
    fp8:  the same shapes as uint8 e4m3 codes, plus fp32 block scales
          s_gate/s_up [E_loc, f/128, d/128], s_down [E_loc, d/128, f/128].
    The shared expert (if any) uses the same layout with E_loc = 1.
    """
    w_gate: torch.Tensor
    w_up: torch.Tensor
    w_down: torch.Tensor
    s_gate: Optional[torch.Tensor] = None
    s_up: Optional[torch.Tensor] = None
    s_down: Optional[torch.Tensor] = None
    sh_gate: Optional[torch.Tensor] = None
    sh_up: Optional[torch.Tensor] = None
    sh_down: Optional[torch.Tensor] = None
    sh_s_gate: Optional[torch.Tensor] = None
    sh_s_up: Optional[torch.Tensor] = None
    sh_s_down: Optional[torch.Tensor] = None


def _children(seed: int):
    kids = np.random.SeedSequence(seed).spawn(len(_STREAMS))
    return dict(zip(_STREAMS, kids))


def _torch_gen(child: np.random.SeedSequence, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(child.generate_state(1, dtype=np.uint64)[0] & 0x7FFF_FFFF_FFFF_FFFF))
    return g


def _randn_bf16(shape, std, gen, device) -> torch.Tensor:
    t = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(torch.bfloat16)


def draw_lengths(cfg: MoEConfig, rng: np.random.Generator) -> List[int]:
    if cfg.lengths is not None:
        return list(cfg.lengths)
    mu, sigma, lo, hi = cfg.lognormal
    z = rng.standard_normal(cfg.n_micro)
    return [int(min(max(np.rint(np.exp(mu + sigma * zi)), lo), hi)) for zi in z]


def _zipf_logp(cfg: MoEConfig, perm_rng: np.random.Generator) -> np.ndarray:
    """log-probabilities over the E experts for Zipf routing.

    Rank 1 goes to the first local expert; ranks 2..E go to the other ids in a
    seeded random order; p(rank r) is proportional to r^-s.  The local experts
    listed in ``dead_local`` get probability 0, so some local experts receive
    no token at all.
    """
    E = cfg.E
    ranks = np.empty(E, dtype=np.float64)
    ranks[cfg.e0] = 1.0
    others = [e for e in range(E) if e != cfg.e0]
    order = perm_rng.permutation(len(others))
    for pos, idx in enumerate(order):
        ranks[others[idx]] = pos + 2.0
    logp = -cfg.zipf_s * np.log(ranks)
    for dl in cfg.dead_local:
        logp[cfg.e0 + dl] = -np.inf
    return logp


def draw_routing(cfg: MoEConfig, T: int, rng: np.random.Generator,
                 logit_rng: np.random.Generator, logp: Optional[np.ndarray]):
    """Top-k distinct expert ids per token and their softmax weights.

    ids: k distinct experts per token, drawn without replacement by
    Gumbel-top-k over log p (uniform p for "uniform" routing), listed in the
    order they were drawn.  Weights: k logits ~ N(0,1), sorted descending,
    softmax over the k logits in fp64, stored as fp32 (slot 0 has the largest
    weight).
    """
    E, k = cfg.E, cfg.k
    if T == 0:
        return np.zeros((0, k), np.int32), np.zeros((0, k), np.float32)
    u = rng.random((T, E))
    gumbel = -np.log(-np.log(np.clip(u, 1e-300, None)))
    keys = gumbel if logp is None else gumbel + logp[None, :]
    ids = np.argsort(-keys, axis=1, kind="stable")[:, :k].astype(np.int32)
    logits = np.sort(logit_rng.standard_normal((T, k)), axis=1)[:, ::-1]
    z = np.exp(logits - logits[:, :1])
    w = (z / z.sum(axis=1, keepdims=True)).astype(np.float32)
    return np.ascontiguousarray(ids), np.ascontiguousarray(w)


def make_microbatches(cfg: MoEConfig, device="cpu", check_skew: bool = True) -> List[MicroBatch]:
    kids = _children(cfg.seed)
    len_rng = np.random.default_rng(kids["lengths"])
    route_rng = np.random.default_rng(kids["routing"])
    logit_rng = np.random.default_rng(kids["logits"])
    xgen = _torch_gen(kids["x"], device)
    lengths = draw_lengths(cfg, len_rng)
    logp = _zipf_logp(cfg, route_rng) if cfg.routing == "zipf" else None
    mbs = []
    for T in lengths:
        ids, w = draw_routing(cfg, T, route_rng, logit_rng, logp)
        x = _randn_bf16((T, cfg.d), cfg.x_std, xgen, device)
        if cfg.routing == "zipf" and check_skew and T > 0:
            cnt = np.bincount(ids.ravel(), minlength=cfg.E)[cfg.e0:cfg.e0 + cfg.E_loc]
            assert all(cnt[dl] == 0 for dl in cfg.dead_local), cnt
            assert cnt.max() > 4 * cnt.mean(), cnt
        mbs.append(MicroBatch(x=x, ids=ids, w=w))
    return mbs


def _fp8_block_quant(w_bf16: torch.Tensor):
    """Checkpoint-style fp8 weights: per 128x128 block scale amax/448 (fp32),
    codes = e4m3(w / scale) via torch's round-to-nearest-even cast."""
    E_, R, C = w_bf16.shape
    wf = w_bf16.float().reshape(E_, R // 128, 128, C // 128, 128)
    amax = wf.abs().amax(dim=(2, 4))
    scale = torch.where(amax > 0, amax / 448.0, torch.ones_like(amax))
    q = (wf / scale[:, :, None, :, None]).clamp_(-448.0, 448.0)
    codes = q.reshape(E_, R, C).to(torch.float8_e4m3fn).view(torch.uint8)
    return codes.contiguous(), scale.contiguous()


def make_weights(cfg: MoEConfig, device="cpu") -> ExpertWeights:
    kids = _children(cfg.seed)
    E_loc, d, f, s = cfg.E_loc, cfg.d, cfg.f, cfg.w_std
    wg = _randn_bf16((E_loc, f, d), s, _torch_gen(kids["w_gate"], device), device)
    wu = _randn_bf16((E_loc, f, d), s, _torch_gen(kids["w_up"], device), device)
    wd = _randn_bf16((E_loc, d, f), s, _torch_gen(kids["w_down"], device), device)
    out = ExpertWeights(wg, wu, wd)
    if cfg.has_shared:
        sg = _torch_gen(kids["shared"], device)
        out.sh_gate = _randn_bf16((1, f, d), s, sg, device)
        out.sh_up = _randn_bf16((1, f, d), s, sg, device)
        out.sh_down = _randn_bf16((1, d, f), s, sg, device)
    if cfg.dtype == "fp8":
        out.w_gate, out.s_gate = _fp8_block_quant(wg)
        out.w_up, out.s_up = _fp8_block_quant(wu)
        out.w_down, out.s_down = _fp8_block_quant(wd)
        if cfg.has_shared:
            out.sh_gate, out.sh_s_gate = _fp8_block_quant(out.sh_gate)
            out.sh_up, out.sh_s_up = _fp8_block_quant(out.sh_up)
            out.sh_down, out.sh_s_down = _fp8_block_quant(out.sh_down)
    return out


def make_config_inputs(name_or_cfg, device="cpu"):
    cfg = CONFIGS[name_or_cfg] if isinstance(name_or_cfg, str) else name_or_cfg
    return cfg, make_weights(cfg, device), make_microbatches(cfg, device)


def scaled(cfg: MoEConfig, **kw) -> MoEConfig:
    """A copy of ``cfg`` with some fields replaced (used for reduced-size cases)."""
    return dataclasses.replace(cfg, **kw)

