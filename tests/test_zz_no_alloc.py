"""mfmg_meta_grad_noalloc (the library's static scratch instead of a caller
workspace) against mfmg_meta_grad with a torch-allocated workspace, through the
C ABI: two calls in a row, the second on a smaller problem, each compared with
the workspace entry point's result on the same inputs."""
import numpy as np
import pytest

import workloads as W
from helpers import desc_of, to_device

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2505_00793_amd import _lib
    _lib.lib()


def _run(cfg, noalloc):
    from paper_2505_00793_amd import _lib as M
    P = M.Problem(desc_of(cfg))
    dev = to_device(W.make_inputs(cfg))
    d = torch.full((W.n_eta(cfg),), float("nan"), device="cuda")
    vl = torch.full((1,), float("nan"), device="cuda")
    args = (dev["theta0"], dev["opt_state0"], dev["eta"], dev["xs"], dev["ys"], dev["vx"],
            dev["vy"], d, vl)
    peak = P.mfmg_meta_grad_noalloc(*args) if noalloc else P.mfmg_meta_grad(*args)
    torch.cuda.synchronize()
    return d.cpu().numpy(), float(vl.item()), peak, P.mfmg_query_sizes(cfg.T).workspace_bytes


def test_noalloc_matches_workspace_entry_point():
    from paper_2505_00793_amd import _lib as M
    big = W.get("c5_small")             # bf16 MLP, 3 inner steps
    small = W.get("c5_small").with_(T=2, rows=90, val_rows=50)
    cases = [big, small, W.get("c4_small"), W.get("c2_small")]
    sizes = []
    for cfg in cases:
        print(f"\n[noalloc] {cfg.name} T={cfg.T} rows={cfg.rows}", flush=True)
        got, V, peak, need = _run(cfg, noalloc=True)
        ref, Vr, peak_r, _ = _run(cfg, noalloc=False)
        sizes.append(need)
        print(f"  workspace {need} bytes; bit-identical {np.array_equal(got, ref)}", flush=True)
        assert need <= M.NOALLOC_SCRATCH_BYTES
        assert np.all(np.isfinite(got))
        assert np.array_equal(got, ref) and V == Vr
        assert peak == peak_r
    assert sizes[1] < sizes[0]


def test_noalloc_rejects_problems_beyond_the_scratch():
    from paper_2505_00793_amd import _lib as M
    cfg = W.get("c5_mid")
    assert M.Problem(desc_of(cfg)).mfmg_query_sizes(cfg.T).workspace_bytes > M.NOALLOC_SCRATCH_BYTES
    with pytest.raises(M.MfmgError) as e:
        _run(cfg, noalloc=True)
    assert e.value.status == M.ERR_WORKSPACE
