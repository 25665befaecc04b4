"""Seeded synthetic inputs for joint text-video attention.

Shared by the oracle's tests, the GPU parity tests and the benchmark. It
holds only shapes and random draws, none of the attention arithmetic.

Workload shapes follow the paper: 24 heads (Sec. VI-D, training throughput
paragraph), 720p frames at 16x spatial token downsampling, i.e. a 45x80 token
grid per frame (implied by the 1.16M-token figure quoted for a
144x1920x1080 input in the same paragraph), multi-second clips (Sec. VI-A,
final training stages) and captions of 100-200 tokens (Sec. IV), hence a
256-token text slot. Values are i.i.d. standard normal; attention time
depends on shapes and the mask, not on values, so these stand in for the
paper's video latents, which are not available.

Draw order (numpy PCG64, seed = 1000 + workload id): q, k, v, do, each
standard_normal float32 [B, N, H, D]; then, for the ragged workload,
text_len = integers(8, 257, size=B) (uniform on [8, 256]).
"""
from __future__ import annotations

from dataclasses import dataclass, asdict

import numpy as np


@dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    batch: int
    heads: int
    head_dim: int
    text_slot: int
    frames: int
    grid_h: int
    grid_w: int
    q_prescale: float = 1.0     # data transform applied to q before the bf16 cast
    ragged_text: bool = False   # draw per-sample text lengths in [8, text_slot]

    @property
    def video_tokens(self) -> int:
        return self.frames * self.grid_h * self.grid_w

    @property
    def tokens(self) -> int:
        return self.text_slot + self.video_tokens

    @property
    def shape(self):
        return (self.batch, self.tokens, self.heads, self.head_dim)

    def describe(self) -> dict:
        d = asdict(self)
        d["tokens"] = self.tokens
        return d


WORKLOADS = {
    1: Workload(1, "tiny", 1, 2, 64, 16, 2, 8, 8),
    2: Workload(2, "medium", 2, 16, 64, 128, 8, 32, 32, q_prescale=1.0 / 8.0),
    3: Workload(3, "long-720p", 1, 24, 128, 256, 16, 45, 80),
    4: Workload(4, "ragged-text", 4, 16, 128, 256, 8, 30, 40, ragged_text=True),
    5: Workload(5, "max-720p", 1, 24, 128, 256, 32, 48, 80),
}

HEADLINE = 3

# Shapes measured by the benchmark's branch modes only (not parity workloads of the five
# configurations): a 144-frame clip, the longest input length in frames the paper quotes
# (Sec. VI-D), at the 720p token grid. Their inputs are drawn on the device
# (make_inputs_device): a host draw of 6.4e9 values would take minutes.
EXTRA = {
    6: Workload(6, "clip-144f-720p", 1, 24, 128, 256, 144, 45, 80),
}


def get(wid: int) -> Workload:
    return WORKLOADS[wid] if wid in WORKLOADS else EXTRA[wid]


def make_inputs(w: Workload | int, seed: int | None = None, with_do: bool = True) -> dict:
    """Float32 q, k, v, do (numpy, [B,N,H,D]) and int32 text_len (or None)."""
    if isinstance(w, int):
        w = WORKLOADS[w]
    seed = 1000 + w.wid if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    shp = w.shape
    q = rng.standard_normal(shp, dtype=np.float32)
    if w.q_prescale != 1.0:
        q *= np.float32(w.q_prescale)
    k = rng.standard_normal(shp, dtype=np.float32)
    v = rng.standard_normal(shp, dtype=np.float32)
    do = rng.standard_normal(shp, dtype=np.float32) if with_do else None
    text_len = None
    if w.ragged_text:
        text_len = rng.integers(min(8, w.text_slot), w.text_slot + 1, size=w.batch).astype(np.int32)
    return {"q": q, "k": k, "v": v, "do": do, "text_len": text_len}


def make_inputs_device(w: Workload, seed: int | None = None, device="cuda") -> dict:
    """bf16 q, k, v, do ([B,N,H,D], standard normal) drawn with torch's generator on the
    device (seed = 1000 + workload id), in that order; text_len as make_inputs draws it."""
    import torch
    seed = 1000 + w.wid if seed is None else seed
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    out = {}
    for name in ("q", "k", "v", "do"):
        x = torch.randn(w.shape, generator=gen, device=device, dtype=torch.float32)
        if name == "q" and w.q_prescale != 1.0:
            x *= w.q_prescale
        out[name] = x.to(torch.bfloat16).contiguous()
        del x
    text_len = None
    if w.ragged_text:
        rng = np.random.Generator(np.random.PCG64(seed))
        text_len = rng.integers(min(8, w.text_slot), w.text_slot + 1, size=w.batch).astype(np.int32)
    out["text_len"] = text_len
    return out


def custom(batch, heads, head_dim, text_slot, frames, grid_h, grid_w, wid=0, name="custom",
           ragged_text=False, q_prescale=1.0) -> Workload:
    return Workload(wid, name, batch, heads, head_dim, text_slot, frames, grid_h, grid_w,
                    q_prescale=q_prescale, ragged_text=ragged_text)


def random_key_mask(w: Workload, seed: int, keep: float = 0.9) -> np.ndarray:
    """uint8 [B, N] mask with roughly `keep` of the keys kept."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return (rng.random((w.batch, w.tokens)) < keep).astype(np.uint8)
