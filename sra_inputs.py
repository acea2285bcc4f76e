"""Seeded synthetic inputs for Sparse Reference Attention (SRA).

This module is the only code shared by the GPU path's tests/benchmark and the CPU
oracle. It holds geometry descriptions and random-number draws; it computes nothing
that belongs to the attention method itself.

Token layout (both streams): packed along tokens, sample after sample, frame-major
inside a sample (frame, row, column), tensors shaped [tokens, heads, head_dim].

Workload recipes (the paper gives no SRA workload; these mirror its video shapes):
  * tiny    : 1 sample, gen 2x8x8 = 128 tokens, ref 4x8x8 = 256 tokens, H=1, d=64, seed 0.
  * 480p    : gen 21x30x52 = 32,760, ref 9x30x52 = 14,040, H=40, d=128, seed 1, RMS-normalised Q/K.
  * sweep_n : 480p gen stream, ref n x 30x52 for n in {4,16,64,256}, H=40, d=128, seed 2, RMS Q/K.
  * 720p    : gen 21x45x80 = 75,600, ref 21x45x80 = 75,600, H=40, d=128, seed 3.
  * varlen  : 4 samples, gen 5x68x120 = 40,800 each, ref {4,2,8,4} x 68x120 frames, H=24,
              d=128, seed 4, RMS Q/K. The reference lengths are drawn once from
              numpy default_rng(13872).choice([2, 4, 8, 12], 4).
  * varlen_window : the varlen batch with a +-1 latent-frame window on gen-gen attention
              (the refiner's sparse temporal attention), seed 5.
  * varlen_tokens : the varlen batch with a reference token mask per sample from
              box_token_mask(r, 68, 120, 13872 + i) (invalid boxes and frames), seed 6.
Every value is an iid N(0,1) fp32 draw rounded to bf16 (round-to-nearest-even).
Draw order: q_gen, k_gen, v_gen, q_ref, k_ref, v_ref, do_gen, do_ref.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np


@dataclass(frozen=True)
class SampleGeom:
    """Geometry of one packed sample: a generation clip and a reference clip.

    gen_frames x gen_h x gen_w generation tokens, ref_frames x ref_h x ref_w reference
    tokens. group_frames consecutive reference latent frames form one self-attention
    group of reference queries. frame_valid (None = all valid) marks reference frames
    that take part at all (e.g. frames where the face is visible). gen_window (None = no
    window) limits which generation keys a generation query sees to the latent frames within
    that many frames of its own (the refiner's sparse temporal attention). ref_token_valid
    (None = every token of a valid frame) marks single reference tokens, frame-major, one
    entry per reference token; a token takes part when its frame and its own entry are valid.
    """

    gen_frames: int
    gen_h: int
    gen_w: int
    ref_frames: int
    ref_h: int
    ref_w: int
    group_frames: int = 1
    frame_valid: Optional[Sequence[int]] = field(default=None)
    gen_window: Optional[int] = None
    ref_token_valid: Optional[Sequence[int]] = field(default=None)

    @property
    def n_gen(self) -> int:
        return self.gen_frames * self.gen_h * self.gen_w

    @property
    def n_ref(self) -> int:
        return self.ref_frames * self.ref_h * self.ref_w


@dataclass
class Workload:
    name: str
    samples: List[SampleGeom]
    heads: int
    head_dim: int
    seed: int
    rms_norm_qk: bool


VARLEN_REF_FRAMES = [int(x) for x in np.random.default_rng(13872).choice([2, 4, 8, 12], size=4)]


def box_token_mask(ref_frames: int, ref_h: int, ref_w: int, seed: int, p_frame_invalid: float = 0.1,
                   p_box: float = 0.6, box_area=(0.1, 0.4)) -> tuple:
    """A reference token mask with the structure of invalid regions in video: per frame, the
    whole frame is invalid with probability p_frame_invalid, else with probability p_box one
    axis-aligned box covering box_area (fraction range) of the frame is invalid, else the
    frame is fully valid. Frame-major, 1 = valid. Drawn from numpy default_rng(seed)."""
    rng = np.random.default_rng(seed)
    m = np.ones((ref_frames, ref_h, ref_w), dtype=np.uint8)
    for f in range(ref_frames):
        u = rng.random()
        if u < p_frame_invalid:
            m[f] = 0
        elif u < p_frame_invalid + p_box:
            area = rng.uniform(*box_area)
            aspect = rng.uniform(0.5, 2.0)
            bh = int(np.clip(round(np.sqrt(area * ref_h * ref_w * aspect)), 1, ref_h))
            bw = int(np.clip(round(area * ref_h * ref_w / bh), 1, ref_w))
            y0 = int(rng.integers(0, ref_h - bh + 1))
            x0 = int(rng.integers(0, ref_w - bw + 1))
            m[f, y0:y0 + bh, x0:x0 + bw] = 0
    return tuple(int(x) for x in m.reshape(-1))


def workload(name: str) -> Workload:
    """The named workload; "<name>@h<N>" is that workload with N heads (a GPU's share of the
    heads when the layer is split across GPUs by head), same geometry and seed."""
    if "@h" in name:
        base, heads = name.split("@h", 1)
        w = workload(base)
        return Workload(name, w.samples, int(heads), w.head_dim, w.seed, w.rms_norm_qk)
    if name == "tiny":
        return Workload(name, [SampleGeom(2, 8, 8, 4, 8, 8)], 1, 64, 0, False)
    if name == "480p":
        return Workload(name, [SampleGeom(21, 30, 52, 9, 30, 52)], 40, 128, 1, True)
    if name.startswith("sweep_"):
        n = int(name.split("_", 1)[1])
        return Workload(name, [SampleGeom(21, 30, 52, n, 30, 52)], 40, 128, 2, True)
    if name == "720p":
        return Workload(name, [SampleGeom(21, 45, 80, 21, 45, 80)], 40, 128, 3, False)
    if name == "720p_whole_ref":
        # the 720p layer with one self-attention group over the whole reference (g = T_r): the
        # other reading of the reference groups, which the reference K/V cache also keeps linear
        return Workload(name, [SampleGeom(21, 45, 80, 21, 45, 80, group_frames=21)], 40, 128, 8, False)
    if name == "varlen":
        return Workload(name, [SampleGeom(5, 68, 120, r, 68, 120) for r in VARLEN_REF_FRAMES],
                        24, 128, 4, True)
    if name == "varlen_window":
        # the same packed batch with the refiner's temporal window: +-1 latent frame
        return Workload(name, [SampleGeom(5, 68, 120, r, 68, 120, gen_window=1) for r in VARLEN_REF_FRAMES],
                        24, 128, 5, True)
    if name == "varlen_tokens":
        # the varlen batch with token-level validity: invalid boxes and frames in the reference
        return Workload(name, [SampleGeom(5, 68, 120, r, 68, 120,
                                          ref_token_valid=box_token_mask(r, 68, 120, 13872 + i))
                               for i, r in enumerate(VARLEN_REF_FRAMES)], 24, 128, 6, True)
    raise KeyError(name)


SWEEP_POINTS = (4, 16, 64, 256)
TENSOR_NAMES = ("q_gen", "k_gen", "v_gen", "q_ref", "k_ref", "v_ref", "do_gen", "do_ref")


def _rms_normalise(x):
    import torch

    xf = x.float()
    return xf * torch.rsqrt(xf.pow(2).mean(dim=-1, keepdim=True) + 1e-6)


def make_inputs(samples: Sequence[SampleGeom], heads: int, head_dim: int, seed: int,
                rms_norm_qk: bool = False, device="cpu", grads: bool = True):
    """Draws the eight bf16 tensors of one SRA problem in the fixed order.

    Returns a dict name -> torch.bfloat16 tensor [tokens, heads, head_dim], contiguous, on
    `device`. Values are fp32 N(0,1) draws from torch.Generator(device).manual_seed(seed),
    optionally RMS-normalised per (token, head) for Q and K, then rounded to bf16.
    """
    import torch

    n_gen = sum(s.n_gen for s in samples)
    n_ref = sum(s.n_ref for s in samples)
    gen = torch.Generator(device=device).manual_seed(seed)
    out = {}
    names = TENSOR_NAMES if grads else TENSOR_NAMES[:6]
    for name in names:
        rows = n_gen if name.endswith("_gen") else n_ref
        x = torch.randn((rows, heads, head_dim), generator=gen, device=device, dtype=torch.float32)
        if rms_norm_qk and name[0] in "qk":
            x = _rms_normalise(x)
        out[name] = x.to(torch.bfloat16).contiguous()
    return out


def to_numpy64(t) -> np.ndarray:
    """Exact float64 copy of a bf16 tensor (bf16 -> fp32 is exact, fp32 -> fp64 is exact)."""
    return t.detach().float().cpu().numpy().astype(np.float64)
