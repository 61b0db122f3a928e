"""Device-side draws of the synthetic KV caches, for whole model stacks.

The recipe is the one of ``synth.py`` (see its docstring): per (layer, KV head, sequence),
keys k_t = M_g (sigma * xi_t) with two outlier channels scaled by 10 and a planted 5% of the
coded tokens shifted along u_g by a ~ U(6, 10); values A_g eta + 0.1 eps.  The head models
(M_g, u_g, A_g, outlier channels), the window and decode queries and the calibration bases
are exactly those of ``synth.py`` (host numpy, same seeds).  Only the per-token Gaussian and
uniform draws come from torch's device generator (Philox), seeded from the same SplitMix64
stream seeds, so that a 32-layer x 131072-token stack is drawn in seconds on the GPU.  These
draws are therefore not bit-identical to ``make_layer``'s: parity tests use ``make_layer``;
this module feeds the stack benchmarks.

Nothing here computes salience, ranks, projections or attention.
"""
from __future__ import annotations

import dataclasses

import numpy as np

from .synth import (OUTLIER_SCALE, PLANT_FRACTION, PLANT_LOGIT_HI, PLANT_LOGIT_LO, VALUE_NOISE,
                    VALUE_RANK, _S_KEYS, _S_QWIN, _S_VALS, _rng, _window_law_queries,
                    calibration_basis, decode_queries, make_head_model, seed_for)


@dataclasses.dataclass
class DeviceLayer:
    K: "torch.Tensor"    # [n, G, d] storage dtype, on the device
    V: "torch.Tensor"
    Qw: np.ndarray       # [w, H, d] float32 (host)
    q: np.ndarray        # [Q, H, d] float32 (host)
    PK: np.ndarray       # [G, d, d] float32 (host)
    PV: np.ndarray


def _gen(device, seed: int):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed & ((1 << 63) - 1))
    return g


def make_layer_device(cfg: dict, layer: int = 0, seq: int = 0, n_queries: int = 1,
                      query_law: str = "aware", device="cuda", with_basis: bool = True,
                      head_models=None) -> DeviceLayer:
    """Draw one layer of one sequence with the per-token draws on ``device``."""
    import torch
    G, H, d, w, n = cfg["G"], cfg["H"], cfg["d"], cfg["w"], cfg["n"]
    base = cfg["seed"]
    N = n - w
    dt = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    hms = head_models or [make_head_model(base, layer, g, d) for g in range(G)]
    sigma = torch.tensor(1.0 / np.arange(1, d + 1), dtype=torch.float32, device=device)
    K = torch.empty((n, G, d), dtype=dt, device=device)
    V = torch.empty((n, G, d), dtype=dt, device=device)
    n_plant = int(round(PLANT_FRACTION * N))
    for g in range(G):
        hm = hms[g]
        gk = _gen(device, seed_for(base, layer, g, seq, _S_KEYS))
        M = torch.tensor(hm.M, dtype=torch.float32, device=device)
        k = (torch.randn((n, d), generator=gk, device=device) * sigma) @ M.T
        k[:, torch.as_tensor(hm.outliers, device=device)] *= OUTLIER_SCALE
        if n_plant:
            planted = torch.randperm(N, generator=gk, device=device)[:n_plant]
            a = torch.rand(n_plant, generator=gk, device=device) * (PLANT_LOGIT_HI - PLANT_LOGIT_LO) + PLANT_LOGIT_LO
            u = torch.tensor(hm.u, dtype=torch.float32, device=device)
            k[planted] += a[:, None] * u[None, :]
        K[:, g, :] = k.to(dt)
        gv = _gen(device, seed_for(base, layer, g, seq, _S_VALS))
        if cfg["values"] == "lowrank":
            A = torch.tensor(hm.A, dtype=torch.float32, device=device)
            v = torch.randn((n, VALUE_RANK), generator=gv, device=device) @ A.T + \
                VALUE_NOISE * torch.randn((n, d), generator=gv, device=device)
        else:
            Mv = torch.tensor(hm.Mv, dtype=torch.float32, device=device)
            v = (torch.randn((n, d), generator=gv, device=device) * sigma) @ Mv.T
            v[:, torch.as_tensor(hm.outliers_v, device=device)] *= OUTLIER_SCALE
        V[:, g, :] = v.to(dt)
    hm_of_head = [hms[h // (H // G)] for h in range(H)]
    Qw = _window_law_queries(_rng(base, layer, 0, seq, _S_QWIN), hm_of_head, w, H, d)
    if query_law == "agnostic":
        q = decode_queries(cfg, layer, seq, n_queries, "agnostic", hms, K.float().cpu().numpy())
    else:
        q = decode_queries(cfg, layer, seq, n_queries, query_law, hms)
    if with_basis:
        PK = np.empty((G, d, d), np.float32)
        PV = np.empty((G, d, d), np.float32)
        for g in range(G):
            PK[g], PV[g] = calibration_basis(base, layer, g, hms[g], d, cfg["values"])
    else:
        PK = PV = None
    return DeviceLayer(K, V, Qw.astype(np.float32), q.astype(np.float32), PK, PV)
