"""The no-allocation decode entry point (varrate_decode_attn_noalloc) against the workspace
entry point (varrate_decode_attn): same kernels and plan, so the outputs must agree bit for
bit, and both stay within the decode bound of the oracle.  Two calls in a row, the second on
a smaller input (fewer sequences, shorter prompt, fewer heads), so the second reuses the
fixed scratch the first one filled."""
import sys

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

DEC_TOL_BF16 = 2e-2


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def _case(vr, oracle_lib, n, G, H, S, Q, seed):
    import torch
    from workloads import CONFIGS, make_layer
    cfg = dict(CONFIGS["llama_32k"])
    cfg.update(n=n, G=G, H=H, seed=seed)
    shape = vr.Shape(n=n, G=G, H=H, w=32, r_min=16, kappa_pct=20, dtype="bf16")
    caches, qs, refs = [], [], []
    for s in range(S):
        li = make_layer(cfg, seq=s, n_queries=Q)
        oc = oracle_lib.compress(li.K, li.V, li.Qw, li.PK, li.PV, H, 20, 16, "bf16")
        dev = lambda a, t=torch.bfloat16: torch.from_numpy(np.ascontiguousarray(a)).to(t).cuda()
        PK, PV = dev(li.PK, torch.float32), dev(li.PV, torch.float32)
        cache = vr.new_cache(shape)
        vr.allocate(shape, dev(oc.sbar, torch.float32), cache)
        vr.project(shape, dev(li.K), dev(li.V), PK, PV, cache)
        caches.append(cache)
        qs.append(li.q)
        refs.append([oracle_lib.decode(oc.coefK, oc.coefV, oc.alloc.rank, oc.Kx, oc.Vx, li.PK, li.PV,
                                       li.q[i], H) for i in range(Q)])
    q = torch.from_numpy(np.stack(qs)).to(torch.bfloat16).cuda()
    return shape, caches, q, PK, PV, refs


def test_noalloc_decode_matches_workspace_decode_twice(oracle_lib):
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU tests need a visible MI355X")
    import paper_2607_15498_amd as vr
    vr.library()
    for (n, G, H, S, Q, seed) in ((4000, 4, 16, 3, 2, 71), (900, 2, 8, 1, 1, 72)):
        say(f"[noalloc] n={n} G={G} H={H} S={S} Q={Q}")
        shape, caches, q, PK, PV, refs = _case(vr, oracle_lib, n, G, H, S, Q, seed)
        need = int(vr.library().varrate_decode_scratch_need(__import__("ctypes").byref(shape.c()), S, Q))
        assert 0 < need <= (8 << 20)
        out_ws = vr.decode(shape, caches, q, PK, PV)
        out_na = torch.full_like(q, float("nan"))
        vr.decode_noalloc(shape, caches, q, PK, PV, out_na)
        torch.cuda.synchronize()
        a = out_ws.float().cpu().numpy()
        b = out_na.float().cpu().numpy()
        assert np.array_equal(a, b), "no-allocation decode differs from the workspace decode"
        worst = 0.0
        for s in range(S):
            for i in range(Q):
                o = b[s, i]
                r = refs[s][i]
                worst = max(worst, max(np.abs(o[h] - r[h]).max() / np.abs(r[h]).max() for h in range(H)))
        say(f"  bit-identical to the workspace decode; worst rel err vs oracle {worst:.3e}")
        assert worst <= DEC_TOL_BF16
