"""The meta-gradient call recorded in a HIP graph and replayed: the library
launches only kernels on the caller's stream (no allocation, copy, memset or
synchronisation inside a call), so one mfmg_meta_grad call can be captured and
replayed.  Every replay is checked bit for bit against the eager result (all
reductions run in a fixed order), with eager work between the replays."""
import numpy as np
import pytest
import torch

import workloads as W
from helpers import desc_of, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_00793_amd import _lib
    _lib.lib()


def _call(P, cfg, dev, d_eta, vloss, ws):
    if cfg.kind == W.KIND_TRANSFORMER:
        dummy = dev["dummy"]
        return P.mfmg_meta_grad(dev["theta0"], None, dev["eta"], dev["xs"], [dummy] * len(dev["xs"]),
                                dev["vx"], dummy, d_eta, vloss, ws=ws)
    return P.mfmg_meta_grad(dev["theta0"], None, dev["eta"], dev["xs"], dev["ys"], dev["vx"],
                            dev["vy"], d_eta, vloss, ws=ws)


@pytest.mark.parametrize("name", ["c1_small", "c2_small", "c3_small", "c5_small", "c4_small",
                                  "c4_fused"])
def test_meta_grad_graph_replay(name):
    from paper_2505_00793_amd import _lib as M
    cfg = W.SMALL[name]
    inp = W.make_inputs(cfg)
    dev = to_device(inp)
    dev["dummy"] = torch.zeros(1, dtype=torch.int32, device="cuda")
    P = M.Problem(desc_of(cfg))
    ws = P.workspace(P.mfmg_query_sizes(cfg.T).workspace_bytes)
    n = W.n_eta(cfg)
    print(f"\n[graph] {name}", flush=True)
    ref = torch.empty(n, device="cuda")
    ref_v = torch.empty(1, device="cuda")
    _call(P, cfg, dev, ref, ref_v, ws)
    torch.cuda.synchronize()

    out = torch.full((n,), float("nan"), device="cuda")
    out_v = torch.full((1,), float("nan"), device="cuda")
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _call(P, cfg, dev, out, out_v, ws)          # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        _call(P, cfg, dev, out, out_v, ws)
    other = torch.empty(n, device="cuda")
    other_v = torch.empty(1, device="cuda")
    for k in range(3):
        out.fill_(float("nan"))
        out_v.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, ref) and torch.equal(out_v, ref_v), f"replay {k} differs"
        _call(P, cfg, dev, other, other_v, ws)      # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(other, ref)
    print(f"  3 replays bit-identical to the eager call ({n} entries)", flush=True)
    assert np.all(np.isfinite(ref.cpu().numpy()))
