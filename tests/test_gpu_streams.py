"""The allocating helpers given an explicit side stream.

Each helper allocates its outputs, status word and (for the audits) a
temporary workspace with torch, and zero-fills the status word, before the
library's kernels run on the stream it was given.  With that stream as
torch's current stream during the call, the fills are ordered before the
kernels and the temporary workspace returns to the caching allocator only
behind them.  Every helper called on a side stream, while the default stream
is kept busy, must give bitwise the results of the same call on the default
stream.
"""
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


def _busy(n=8):
    # Queue some work on the default stream so that anything wrongly ordered
    # against it would overlap the side-stream calls.
    x = torch.randn(2048, 2048, device=DEV)
    for _ in range(n):
        x = x @ x
        x = x / x.norm()
    return x


def _equal(a, b):
    if a is None or b is None:
        return a is None and b is None
    return torch.equal(a, b)


def test_helpers_on_a_side_stream_equal_default_stream():
    w = wl.WORKLOADS["b128"].replace(B=12, D=3 * 4096 + 40)
    wa = wl.WORKLOADS["audit"].replace(B=6, D=2048 + 200, R=333)
    meta, meta_a = wl.host_meta(w), wl.host_meta(wa)
    meta_a.rewards[:16] = 1.0           # one audit prompt with equal rewards (not swept)
    dm, da = upload_meta(meta), upload_meta(meta_a)
    s = wl.device_scores(w, meta.nv, DEV)
    sa = wl.device_scores(wa, meta_a.nv, DEV)
    log(f"side stream: chain B={meta.B} D={w.D}, audit B={meta_a.B} D={wa.D} R={wa.R}")

    def run(stream):
        out = {}
        d = pair.design_inclusion(dm["offsets"], dm["p"], w.design_seed, 5, 2, meta.gmax,
                                  nv=meta.nv, stream=stream)
        c = pair.edge_coeffs(dm["offsets"], dm["rewards"], d["mask"][1], d["pi"], meta.gmax,
                             nv=meta.nv, stream=stream)
        g = pair.weighted_grad(dm["offsets"], s, c["coeff"], nv=meta.nv, stream=stream)
        gm = pair.weighted_grad(dm["offsets"], s, c["coeff"], nv=meta.nv, reduce=True,
                                stream=stream)
        dc = pair.design_coeffs(dm["offsets"], dm["p"], dm["rewards"], w.design_seed, 6,
                                meta.gmax, nv=meta.nv, stream=stream)
        a = pair.audit(da["offsets"], sa, da["rewards"], da["p"], wa.design_seed, 7, wa.R,
                       meta_a.gmax, nv=meta_a.nv, stream=stream)
        ad = pair.audit_direction(da["offsets"], sa, da["rewards"], da["p"], wa.design_seed, 7,
                                  wa.R, meta_a.gmax, nv=meta_a.nv, stream=stream)
        ax = pair.audit_exact(da["offsets"], sa, da["rewards"], da["p"], meta_a.gmax,
                              nv=meta_a.nv, stream=stream)
        for name, res in (("design", d), ("coeffs", c), ("grad", g), ("mean", gm),
                          ("design_coeffs", dc), ("audit", a), ("direction", ad), ("exact", ax)):
            for k, v in res.items():
                out[f"{name}.{k}"] = v
        return out

    ref = run(None)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    busy = _busy()
    got = run(side)
    side.synchronize()
    torch.cuda.synchronize()
    del busy
    assert set(got) == set(ref)
    for k in sorted(ref):
        if ref[k] is not None and k.endswith("status"):
            assert int(ref[k].item()) == 0, k
        assert _equal(got[k], ref[k]), f"{k} differs on the side stream"
    assert float(ref["audit.mse"][0]) == 0.0
