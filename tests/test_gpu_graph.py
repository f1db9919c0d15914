"""A whole step of the hot path captured once in a HIP graph and replayed.

The entry points allocate nothing, clear nothing with hipMemsetAsync and
never synchronise with the host, so the step (design draw and coefficient
fold, weighted gradient, audit) can be recorded with torch.cuda.CUDAGraph
and replayed.  Between replays the inputs are changed by eager copies and
the status word is cleared by an eager fill kernel; every replay must equal
the same calls made eagerly, bitwise.
"""
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


def _outputs(meta, w, meta_a, wa):
    return {
        "coeff": torch.empty(meta.nv, device=DEV),
        "mask": torch.empty(meta.nv, dtype=torch.uint8, device=DEV),
        "pi": torch.empty((meta.B, meta.gmax, meta.gmax), device=DEV),
        "ec": torch.empty(meta.B, dtype=torch.int32, device=DEV),
        "comp": torch.empty(meta.B, dtype=torch.int32, device=DEV),
        "out": torch.empty((meta.B, w.D), device=DEV),
        "mse": torch.empty(meta_a.B, dtype=torch.float64, device=DEV),
        "bias": torch.empty(meta_a.B, dtype=torch.float64, device=DEV),
        "reps": torch.empty((meta_a.B, wa.R), device=DEV),
        "ec_a": torch.empty((meta_a.B, wa.R), dtype=torch.int32, device=DEV),
        "ws": torch.empty(pair.pair_audit_workspace_bytes(meta_a.B, meta_a.gmax, wa.D, wa.R),
                          dtype=torch.uint8, device=DEV),
        "st": torch.zeros(1, dtype=torch.int32, device=DEV),
    }


def test_step_replays_from_a_graph():
    w = wl.WORKLOADS["b128"].replace(B=16, D=3 * 4096 + 100)
    wa = wl.WORKLOADS["audit"].replace(B=8, D=2048 + 64, R=300)
    meta, meta_a = wl.host_meta(w), wl.host_meta(wa)
    dm, da = upload_meta(meta), upload_meta(meta_a)
    s = wl.device_scores(w, meta.nv, DEV, ld=(w.D + 7) // 8 * 8)[:, :w.D]
    sa = wl.device_scores(wa, meta_a.nv, DEV)
    log(f"graph step: chain B={meta.B} D={w.D}, audit B={meta_a.B} D={wa.D} R={wa.R}")

    def step(o):
        pair.pair_design_coeffs(meta.B, meta.nv, meta.gmax, dm["offsets"], dm["p"], dm["rewards"],
                                w.design_seed, 2, o["coeff"], o["mask"], o["pi"], o["ec"],
                                o["comp"], o["st"])
        pair.pair_weighted_grad(meta.B, meta.nv, dm["offsets"], s, o["coeff"], o["out"], 0,
                                o["st"])
        pair.pair_audit(meta_a.B, meta_a.nv, meta_a.gmax, da["offsets"], sa, da["rewards"],
                        da["p"], None, wa.design_seed, 7, wa.R, o["mse"], o["bias"], o["reps"],
                        o["ec_a"], o["ws"], o["st"])

    graph_out = _outputs(meta, w, meta_a, wa)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step(graph_out)                      # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step(graph_out)

    rng = np.random.default_rng(3)
    for k in range(3):
        # New rewards and continuation probabilities in the captured buffers.
        dm["rewards"].copy_(torch.from_numpy(
            rng.permutation(meta.rewards).astype(np.float32)).to(DEV))
        da["p"].copy_(torch.from_numpy(
            np.clip(rng.uniform(0.1, 1.0, meta_a.nv), 0.1, 1.0).astype(np.float32)).to(DEV))
        graph_out["st"].zero_()
        g.replay()
        torch.cuda.synchronize()
        eager = _outputs(meta, w, meta_a, wa)
        step(eager)
        torch.cuda.synchronize()
        assert int(graph_out["st"].item()) == 0 and int(eager["st"].item()) == 0
        for key in ("coeff", "mask", "pi", "ec", "comp", "out", "mse", "bias", "reps", "ec_a"):
            assert torch.equal(graph_out[key], eager[key]), f"replay {k}: {key} differs"
        log(f"  replay {k}: bitwise equal to the eager step "
            f"(mean mse {float(eager['mse'].mean()):.4e})")
