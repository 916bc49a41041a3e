"""The forward and backward captured in a HIP graph.

The library allocates, clears and synchronizes nothing and launches only
kernels on the caller's stream, so a training step (forward, then backward
with the forward's states) can be captured once and replayed.  Each replay,
with other eager work and synchronizations between replays, must reproduce
the eager step bit for bit (the library is deterministic)."""
import pytest

import workloads as W
from tests.gpu_util import to_device, desc_of

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def F():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2606_27748_amd as F
    F.load()
    return F


# (64, 128): one kernel per pass; (128, 80): two frequency groups, the first
# padded; d_v != d: the zero-padded copies and the cropped results in the graph
@pytest.mark.parametrize("d,m,dv", [(64, 128, 64), (128, 80, 128), (64, 128, 32), (32, 64, 128)])
def test_fwd_bwd_graph_replays(F, d, m, dv):
    import torch
    wl = W.Workload("graph", 2, 3, 700, d, m, "nonstationary", True, "bf16", True, 51, value_dim=dv)
    t = to_device(W.generate(wl))
    desc = desc_of(wl)
    dev = t["Q"].device
    f32 = torch.float32
    B, H, N = wl.B, wl.H, wl.N
    wsf = torch.empty(F.workspace_size(desc, F.FLEX_PASS_FWD), dtype=torch.uint8, device=dev)
    wsb = torch.empty(F.workspace_size(desc, F.FLEX_PASS_BWD), dtype=torch.uint8, device=dev)
    out = dict(O=torch.empty_like(t["V"]), den=torch.empty(B, H, N, dtype=f32, device=dev),
               dQ=torch.empty(B, H, N, d, dtype=f32, device=dev), dK=torch.empty(B, H, N, d, dtype=f32, device=dev),
               dV=torch.empty(B, H, N, dv, dtype=f32, device=dev), dW1=torch.empty(H, m, d, dtype=f32, device=dev),
               dW2=torch.empty(H, m, d, dtype=f32, device=dev), dtau=torch.empty(H, dtype=f32, device=dev))

    def step():
        F.flex_linattn_fwd(desc, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"],
                           O=out["O"], den=out["den"], ws=wsf)
        F.flex_linattn_bwd(desc, t["Q"], t["K"], t["V"], t["W1"], t["W2"], t["tau"], out["O"], out["den"],
                           t["dO"], dQ=out["dQ"], dK=out["dK"], dV=out["dV"], dW1=out["dW1"], dW2=out["dW2"],
                           dtau=out["dtau"], ws=wsb, fwd_ws=wsf)

    step()
    torch.cuda.synchronize()
    ref = {k: v.clone() for k, v in out.items()}

    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()   # default priority
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step()
    torch.cuda.synchronize()

    other = torch.empty_like(t["V"])
    for rep in range(3):
        for v in out.values():
            v.fill_(float("nan"))
        # eager work between replays: a forward with the roles of Q and K swapped
        F.flex_linattn_fwd(desc, t["K"], t["Q"], t["V"], t["W1"], t["W2"], t["tau"], O=other, ws=wsf)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for k, v in ref.items():
            assert torch.equal(out[k], v), (rep, k)
