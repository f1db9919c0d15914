"""pair_audit_noalloc, the audit whose workspace is the library's static
device scratch, against pair_audit with a caller workspace: two calls in a
row through the C ABI, the audit workload at full size (B=256, G=16,
D=65536, R=4096: four prompt chunks of the 64 MiB scratch) and then a
smaller ragged batch with up to 64 candidates and a logged rho block.  Every
output must be bitwise that of pair_audit (the same kernels, prompt by
prompt), whatever the previous call left in the scratch."""
import numpy as np
import pytest
import torch

import paper_2608_11368_amd as pair
import workloads as wl
from tests.gpu_util import DEV, log, upload_meta

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    pair.lib()
    yield
    torch.cuda.synchronize()


def _outputs(B, R):
    return {"mse": torch.empty(B, dtype=torch.float64, device=DEV),
            "bias_norm": torch.empty(B, dtype=torch.float64, device=DEV),
            "rep_sqerr": torch.empty((B, R), dtype=torch.float32, device=DEV),
            "edge_count": torch.empty((B, R), dtype=torch.int32, device=DEV),
            "status": torch.zeros(1, dtype=torch.int32, device=DEV)}


def _compare(w, meta, R, rep0, pi_w=None):
    dm = upload_meta(meta)
    s = wl.device_scores(w, meta.nv, DEV)
    ref = pair.audit(dm["offsets"], s, dm["rewards"], dm["p"], w.design_seed, rep0, R, meta.gmax,
                     pi_w=pi_w, nv=meta.nv)
    got = _outputs(meta.B, R)
    torch.cuda.synchronize()
    pair.pair_audit_noalloc(meta.B, meta.nv, meta.gmax, dm["offsets"], s, dm["rewards"], dm["p"],
                            pi_w, w.design_seed, rep0, R, got["mse"], got["bias_norm"],
                            got["rep_sqerr"], got["edge_count"], got["status"])
    torch.cuda.synchronize()
    assert int(ref["status"].item()) == 0 and int(got["status"].item()) == 0
    for k in ("mse", "bias_norm", "rep_sqerr", "edge_count"):
        assert torch.equal(got[k], ref[k]), f"{k} differs from pair_audit"
    assert float(got["mse"].max()) > 0.0


def test_noalloc_audit_equals_pair_audit_twice():
    w = wl.WORKLOADS["audit"]
    meta = wl.host_meta(w)
    ws = pair.pair_audit_workspace_bytes(meta.B, meta.gmax, w.D, w.R)
    log(f"no-alloc audit, full workload B={meta.B} D={w.D} R={w.R}: "
        f"workspace {ws / 2**20:.0f} MiB against {pair.AUDIT_SCRATCH_BYTES / 2**20:.0f} MiB")
    assert ws > pair.AUDIT_SCRATCH_BYTES      # the call runs in several prompt chunks
    _compare(w, meta, w.R, 0)
    wr = wl.WORKLOADS["ragged"].replace(B=5, D=1504, dtype=wl.BF16)
    mr = wl.host_meta(wr)
    log(f"no-alloc audit, second call: ragged B={mr.B} gmax={mr.gmax} D={wr.D} R=200 rep0=17")
    pi_w = torch.rand((mr.B, mr.gmax, mr.gmax), device=DEV) * 0.9 + 0.1
    _compare(wr, mr, 200, 17, pi_w=pi_w)


def test_noalloc_audit_replays_from_a_graph():
    """The callers this entry point is for include code under HIP graph
    capture: the call is captured once (after an eager call has looked up
    the scratch's address) and replayed three times, with new rewards and
    continuation probabilities copied into the captured buffers between
    replays; every replay must equal an eager pair_audit with a workspace
    bitwise, and the audit runs in two prompt chunks."""
    w = wl.WORKLOADS["audit"].replace(B=100, D=65536 + 2048, R=4096)
    meta = wl.host_meta(w)
    dm = upload_meta(meta)
    s = wl.device_scores(w, meta.nv, DEV)
    ws_bytes = pair.pair_audit_workspace_bytes(meta.B, meta.gmax, w.D, w.R)
    log(f"no-alloc audit under graph capture: B={meta.B} D={w.D} R={w.R}, "
        f"workspace {ws_bytes / 2**20:.0f} MiB against {pair.AUDIT_SCRATCH_BYTES / 2**20:.0f} MiB")
    assert ws_bytes > pair.AUDIT_SCRATCH_BYTES
    got = _outputs(meta.B, w.R)

    def call():
        pair.pair_audit_noalloc(meta.B, meta.nv, meta.gmax, dm["offsets"], s, dm["rewards"],
                                dm["p"], None, w.design_seed, 11, w.R, got["mse"],
                                got["bias_norm"], got["rep_sqerr"], got["edge_count"],
                                got["status"])

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        call()                                # eager: the scratch address is looked up here
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    rng = np.random.default_rng(8)
    for k in range(3):
        dm["rewards"].copy_(torch.from_numpy(rng.permutation(meta.rewards)).to(DEV))
        dm["p"].copy_(torch.from_numpy(rng.uniform(0.1, 1.0, meta.nv).astype(np.float32)).to(DEV))
        got["status"].zero_()
        g.replay()
        torch.cuda.synchronize()
        ref = pair.audit(dm["offsets"], s, dm["rewards"], dm["p"], w.design_seed, 11, w.R,
                         meta.gmax, nv=meta.nv)
        torch.cuda.synchronize()
        assert int(got["status"].item()) == 0 and int(ref["status"].item()) == 0
        for key in ("mse", "bias_norm", "rep_sqerr", "edge_count"):
            assert torch.equal(got[key], ref[key]), f"replay {k}: {key} differs"
        log(f"  replay {k}: bitwise equal to pair_audit (mean mse {float(ref['mse'].mean()):.4e})")
