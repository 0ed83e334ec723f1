"""GPU: the compute entry points replayed from a captured HIP graph.

The compute calls launch kernels only on the caller's stream (no allocation,
memset or synchronisation), so a caller may capture them.  The graph is
replayed several times, each time on new values written into the captured
input buffers by eager work between the replays, and every replay must equal
the eager result bit for bit (the kernels are deterministic: no atomics, a
fixed reduction order).
"""
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("cfg", [2, 3])
def test_graph_replays_match_eager(gpu_lib, cfg):
    splat = gpu_lib
    w = workloads.get(cfg)
    a = splat.Acsr(splat.Pattern.named(w.kind, w.params, w.L))
    inputs = [tuple(x.cuda() for x in workloads.make_qkv(w.with_(seed=w.seed + 100 * r)))
              for r in range(4)]
    Q, K, V = (x.clone() for x in inputs[0])
    S = torch.empty((w.B, w.H, a.nnz), dtype=torch.float32, device="cuda")
    P = torch.empty_like(S)
    O = torch.empty_like(Q)
    Ou = torch.empty_like(Q)

    def step():
        splat.sparse_mhsa_fwd(a, Q, K, V, w.scale, O=O)
        splat.rsddmm(a, Q, K, w.scale, S=S)
        splat.row_softmax(a, S, P)
        splat.rspmm(a, P, V, O=Ou)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()                      # first calls (one-time kernel attributes) outside capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()

    for r in (1, 2, 3, 0):
        q, k, v = inputs[r]
        Q.copy_(q), K.copy_(k), V.copy_(v)
        O.zero_(), Ou.zero_(), S.zero_(), P.zero_()
        g.replay()
        torch.cuda.synchronize()
        got = (O.clone(), S.clone(), P.clone(), Ou.clone())
        e_O = splat.sparse_mhsa_fwd(a, q, k, v, w.scale)
        e_S = splat.rsddmm(a, q, k, w.scale)
        e_P = splat.row_softmax(a, e_S)
        e_Ou = splat.rspmm(a, e_P, v, out_dtype=v.dtype)
        torch.cuda.synchronize()
        for name, x, y in zip(("fused O", "S", "P", "unfused O"), got, (e_O, e_S, e_P, e_Ou)):
            assert torch.equal(x, y), f"replay with inputs {r}: {name} differs from the eager call"
