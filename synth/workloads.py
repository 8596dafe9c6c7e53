"""Seeded synthetic inputs with the shapes and value distributions of the five
benchmark workloads of the modality-aware quantized linear.

Stand-in for the paper's real activations (Qwen2.5-VL / Qwen2.5-Omni decoder
linears, Sec. 5.1), which are not available: visual tokens are drawn about
30x larger than text tokens, matching the 10-100x range the paper reports in
the introduction, with a small set of outlier channels (Sec. 4.1, "Smoothing
Misalignment").

Recipe (all draws from ``numpy.random.default_rng`` seeded by
``SeedSequence([config index, crc32(stream name)])``):

* text rows   ~ N(0, 1),       outlier channel set O scaled x20
* vision rows ~ N(0, 1) * 30,  the same set O scaled x20
* audio rows  ~ N(0, 1) * 2,   a disjoint set O_a (same size) scaled x10
* |O| = 8 for the 512-wide layer, round(0.01 * C_in) otherwise
* float weight W ~ N(0, 1/C_in), paper layout [C_in][C_out]
* bf16 workloads round X once (round-to-nearest-even) after drawing in fp32
* modality layout: contiguous (text rows first) or interleaved runs whose
  lengths are drawn from U{64..512}, ordered so that adjacent runs differ in
  modality whenever possible.

Nothing here quantizes, smooths or factorizes: those are the method's steps
and live separately in the oracle and in the GPU package.
"""
from __future__ import annotations

import zlib
from dataclasses import dataclass, field

import numpy as np

TEXT, VISION, AUDIO = 0, 1, 2

# (row scale, outlier multiplier, which outlier set) per modality id.
_MODALITY_STATS = {
    TEXT: (1.0, 20.0, "shared"),
    VISION: (30.0, 20.0, "shared"),
    AUDIO: (2.0, 10.0, "audio"),
}


@dataclass(frozen=True)
class Projection:
    name: str
    c_in: int
    c_out: int
    input_key: str  # projections with the same key read the same activations


@dataclass(frozen=True)
class Config:
    index: int
    name: str
    T: int
    counts: tuple            # tokens per modality id (text, vision[, audio])
    projections: tuple
    rank: int
    act_dtype: str           # "f32" or "bf16": X and Y
    lr_dtype: str            # "f32" or "bf16": low-rank factors
    layout: str              # "contiguous" or "runs"
    n_outlier: int = -1      # -1: round(0.01 * C_in)
    description: str = ""

    @property
    def n_mod(self) -> int:
        return len(self.counts)

    def outliers_for(self, c_in: int) -> int:
        return self.n_outlier if self.n_outlier > 0 else int(round(0.01 * c_in))


def _single(name, c_in, c_out):
    return (Projection(name, c_in, c_out, "x"),)


_DECODER_STACK = (
    Projection("q_proj", 3584, 3584, "x_attn_in"),
    Projection("k_proj", 3584, 512, "x_attn_in"),
    Projection("v_proj", 3584, 512, "x_attn_in"),
    Projection("o_proj", 3584, 3584, "x_attn_out"),
    Projection("gate_proj", 3584, 18944, "x_mlp_in"),
    Projection("up_proj", 3584, 18944, "x_mlp_in"),
    Projection("down_proj", 18944, 3584, "x_mlp_mid"),
)

CONFIGS = (
    Config(0, "linear_fp32_t256_k512_n512_r16", 256, (192, 64),
           _single("linear", 512, 512), 16, "f32", "f32", "contiguous", 8,
           "single fp32 linear, 192 text + 64 vision tokens"),
    Config(1, "prefill_bf16_t4096_k3584_n18944_r64", 4096, (1024, 3072),
           _single("gate_up_proj", 3584, 18944), 64, "bf16", "bf16", "contiguous",
           description="7B-class gate/up projection, prefill, 1024 text + 3072 vision"),
    Config(2, "decode_bf16_t16_k18944_n3584_r64", 16, (8, 8),
           _single("down_proj", 18944, 3584), 64, "bf16", "bf16", "contiguous",
           description="7B-class down projection, decode batch 8 text + 8 vision"),
    Config(3, "trimodal_bf16_t8192_k3584_n3584_r64", 8192, (2048, 4096, 2048),
           _single("q_o_proj", 3584, 3584), 64, "bf16", "bf16", "runs",
           description="tri-modal prefill, runs of 64-512 tokens"),
    Config(4, "decoder_stack_bf16_t2048_r64", 2048, (512, 1280, 256),
           _DECODER_STACK, 64, "bf16", "bf16", "runs",
           description="seven projections of a 7B-class decoder layer, tri-modal"),
)


def config_by_name(name: str) -> Config:
    for c in CONFIGS:
        if c.name == name or str(c.index) == str(name):
            return c
    raise KeyError(name)


def _rng(cfg_index: int, stream: str, extra: int = 0) -> np.random.Generator:
    ss = np.random.SeedSequence([int(cfg_index), zlib.crc32(stream.encode()), int(extra)])
    return np.random.default_rng(ss)


def _split_runs(count: int, rng: np.random.Generator, lo: int = 64, hi: int = 512):
    """Split ``count`` tokens into runs with lengths in [lo, hi]."""
    if count <= 0:
        return []
    if count <= hi:
        return [count]
    runs = []
    rem = count
    while rem > hi:
        length = int(rng.integers(lo, hi + 1))
        if rem - length < lo:          # keep the final run within bounds
            length = rem - lo
        runs.append(length)
        rem -= length
    runs.append(rem)
    return runs


def make_modality_layout(counts, layout: str, cfg_index: int = 0, seed_extra: int = 0) -> np.ndarray:
    """Per-token modality ids (int32), 0 = text."""
    counts = [int(c) for c in counts]
    if layout == "contiguous":
        return np.concatenate([np.full(c, m, np.int32) for m, c in enumerate(counts)]).astype(np.int32)
    if layout == "alternating":
        T = sum(counts)
        out = np.empty(T, np.int32)
        rem = list(counts)
        last = -1
        for t in range(T):
            cands = [m for m in range(len(rem)) if rem[m] > 0 and m != last] or \
                    [m for m in range(len(rem)) if rem[m] > 0]
            m = max(cands, key=lambda k: rem[k])
            out[t] = m
            rem[m] -= 1
            last = m
        return out
    if layout != "runs":
        raise ValueError(layout)
    rng = _rng(cfg_index, "layout", seed_extra)
    pools = {m: _split_runs(c, rng) for m, c in enumerate(counts)}
    for m in pools:
        rng.shuffle(pools[m])
    seq = []
    last = -1
    while any(pools.values()):
        cands = [m for m, p in pools.items() if p and m != last] or [m for m, p in pools.items() if p]
        most = max(len(pools[m]) for m in cands)
        top = [m for m in cands if len(pools[m]) == most]
        m = top[int(rng.integers(len(top)))]
        seq.append(np.full(pools[m].pop(), m, np.int32))
        last = m
    return np.concatenate(seq).astype(np.int32)


def _outlier_sets(cfg: Config, c_in: int, seed_extra: int = 0):
    rng = _rng(cfg.index, f"outliers{c_in}", seed_extra)
    n = cfg.outliers_for(c_in)
    perm = rng.permutation(c_in)
    return np.sort(perm[:n]), np.sort(perm[n:2 * n])


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Input preparation: fp32 values rounded once to the nearest bf16 (ties to
    even), returned as fp32.  Uses torch's CPU cast, which is an independent
    implementation from anything in the oracle or the kernels."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def make_activations(cfg: Config, key: str, c_in: int, modality: np.ndarray,
                     seed_extra: int = 0) -> np.ndarray:
    """X [T][c_in] float32 (bf16-representable for bf16 workloads)."""
    rng = _rng(cfg.index, f"x:{key}:{c_in}", seed_extra)
    T = modality.shape[0]
    x = rng.standard_normal((T, c_in), dtype=np.float32)
    shared, audio = _outlier_sets(cfg, c_in, seed_extra)
    for m, (scale, mult, which) in _MODALITY_STATS.items():
        rows = modality == m
        if not rows.any():
            continue
        cols = shared if which == "shared" else audio
        block = x[rows] * np.float32(scale)
        block[:, cols] *= np.float32(mult)
        x[rows] = block
    if cfg.act_dtype == "bf16":
        x = round_to_bf16(x)
    return np.ascontiguousarray(x, dtype=np.float32)


def make_weight(cfg: Config, proj: Projection, seed_extra: int = 0) -> np.ndarray:
    """Float weight W [c_in][c_out] ~ N(0, 1/c_in), float32 (paper layout)."""
    rng = _rng(cfg.index, f"w:{proj.name}", seed_extra)
    w = rng.standard_normal((proj.c_in, proj.c_out), dtype=np.float32)
    w *= np.float32(1.0 / np.sqrt(proj.c_in))
    return w


@dataclass
class LayerInputs:
    cfg: Config
    modality: np.ndarray                      # int32 [T]
    x: dict = field(default_factory=dict)     # input_key -> float32 [T][c_in]
    w: dict = field(default_factory=dict)     # projection name -> float32 [c_in][c_out]


def make_layer_inputs(cfg: Config, seed_extra: int = 0, projections=None,
                      layout: str | None = None) -> LayerInputs:
    """All seeded inputs of a workload: modality ids, activations, float weights."""
    mod = make_modality_layout(cfg.counts, layout or cfg.layout, cfg.index, seed_extra)
    out = LayerInputs(cfg, mod)
    names = None if projections is None else set(projections)
    for p in cfg.projections:
        if names is not None and p.name not in names:
            continue
        if p.input_key not in out.x:
            out.x[p.input_key] = make_activations(cfg, p.input_key, p.c_in, mod, seed_extra)
        out.w[p.name] = make_weight(cfg, p, seed_extra)
    return out
