"""Synthetic benchmark layers: seeded inputs plus their calibrated artifacts.

Combines the seeded input generator (``synth``) with the offline calibration
(``calibrate``) for one projection of one of the five benchmark workloads.
The result can be cached on disk (``MASQ_CACHE_DIR``) because calibrating a
3584 x 18944 layer takes several seconds of host time.
"""
from __future__ import annotations

import os

import numpy as np

import synth

from . import calibrate

_KEYS = ("x", "modality", "inv_smooth", "wq", "w_scale", "l_down", "r_up")


METHODS = ("masquant", "smoothquant", "mas")


def _cache_path(cfg, proj, seed_extra, weight_bits, method):
    d = os.environ.get("MASQ_CACHE_DIR")
    if not d:
        return None
    os.makedirs(d, exist_ok=True)
    tag = ("" if weight_bits == 8 else f"__w{weight_bits}") + \
          ("" if method == "masquant" else f"__{method}")
    return os.path.join(d, f"{cfg.name}__{proj.name}__{seed_extra}{tag}.npz")


def layer(cfg, proj_name: str | None = None, seed_extra: int = 0, weight_bits: int = 8,
          method: str = "masquant") -> dict:
    """Inputs and artifacts of one projection: x [T][K] f32 (bf16-exact for
    bf16 workloads), modality [T] int32, and the calibration arrays; with
    weight_bits=4 the shared weight is quantised to 4-bit codes (kept as
    int8 codes here; the device copy is packed).  method="smoothquant" gives
    the comparator with the unified smoothing factor for every token and no
    compensation (rank 0); method="mas" the MAS-only comparator, one weight
    per modality (wq [M][N][K], w_scale [M][N]) and no compensation."""
    if method not in METHODS:
        raise ValueError(f"method must be one of {METHODS}")
    if isinstance(cfg, (int, str)):
        cfg = synth.config_by_name(str(cfg))
    proj = cfg.projections[0] if proj_name is None else \
        next(p for p in cfg.projections if p.name == proj_name)
    path = _cache_path(cfg, proj, seed_extra, weight_bits, method)
    if path and os.path.exists(path):
        with np.load(path, allow_pickle=False) as f:
            out = {k: f[k] for k in _KEYS}
    else:
        li = synth.make_layer_inputs(cfg, seed_extra, projections=[proj.name])
        x = li.x[proj.input_key]
        if method == "smoothquant":
            art = calibrate.calibrate_smoothquant(x, li.w[proj.name], cfg.n_mod, cfg.lr_dtype,
                                                  weight_bits=weight_bits)
        elif method == "mas":
            if weight_bits != 8:
                raise ValueError("the MAS-only comparator is built for 8-bit weights")
            art = calibrate.calibrate_mas_only(x, li.modality, li.w[proj.name], cfg.n_mod,
                                               cfg.lr_dtype)
        else:
            art = calibrate.calibrate_layer(x, li.modality, li.w[proj.name], cfg.n_mod,
                                            cfg.rank, cfg.lr_dtype, weight_bits=weight_bits)
        out = dict(x=x, modality=li.modality, **{k: art[k] for k in _KEYS[2:]})
        if path:
            tmp = path + ".tmp.npz"
            np.savez(tmp, **out)
            os.replace(tmp, path)
    out.update(cfg=cfg, proj=proj, n_mod=cfg.n_mod,
               rank=cfg.rank if method == "masquant" else 0, method=method,
               act_dtype=cfg.act_dtype, lr_dtype=cfg.lr_dtype, weight_bits=weight_bits)
    return out


def to_device(layer_arrays: dict, device="cuda"):
    """(x, modality, ops.Linear) on the device; imports the HIP binding."""
    import torch

    from . import ops
    act = torch.bfloat16 if layer_arrays["act_dtype"] == "bf16" else torch.float32
    x = torch.from_numpy(layer_arrays["x"]).to(device=device, dtype=act).contiguous()
    mod = torch.from_numpy(layer_arrays["modality"]).to(device=device).contiguous()
    if layer_arrays.get("method") == "mas":
        lin = ops.MasOnlyLinear.from_arrays(layer_arrays, device)
    else:
        lin = ops.Linear.from_arrays(layer_arrays, device)
    return x, mod, lin
