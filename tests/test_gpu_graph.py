"""Training steps captured as a HIP graph (torch.cuda.CUDAGraph on the
stream the library launches on) and replayed: every replay equals, bit for
bit, the same epoch run eagerly from the same weights.  The graph is
replayed three times with the program's own eager work and synchronisations
between replays, and each replay is checked (the step records no memset
node: every buffer it clears is cleared by a kernel)."""
import numpy as np
import pytest

import pmlp_workloads as wl

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    torch.cuda.set_device(0)
    return torch


@pytest.fixture(scope="module")
def pm(torch):
    import paper_2206_08369_amd as pm
    pm.load_library()
    return pm


@pytest.mark.parametrize("wname", ["w60_f10", "w1k_f50"])
def test_graph_replays_equal_eager_epochs(pm, torch, wname):
    w = wl.WORKLOADS[wname]
    hs, acts = w.model_grid()
    X, y = wl.workload_dataset(w)
    Xd = torch.from_numpy(X).cuda()
    yd = torch.from_numpy(y).cuda()
    batches = w.batches()
    g_net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed)
    e_net = pm.PackedMLP(w.F, w.O, hs, acts, seed=w.init_seed)

    def epoch(net):
        for s, n in batches:
            net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)

    # workspaces grown before capture (the full batch comes first)
    W1, W2 = g_net.get_params()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        s, n = batches[0]
        g_net.train_step(Xd[s:s + n], yd[s:s + n], w.lr)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g_net.set_params(W1, W2)               # back to the initial weights
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, capture_error_mode="relaxed"):
        epoch(g_net)
    torch.cuda.synchronize()
    g_net.set_params(W1, W2)               # capture does not run the kernels; reset anyway
    e_net.set_params(W1, W2)
    scratch = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        graph.replay()
        scratch.add_(1.0)                  # eager work between replays
        epoch(e_net)
        torch.cuda.synchronize()
        a1, a2 = g_net.get_params()
        b1, b2 = e_net.get_params()
        assert np.array_equal(a1, b1) and np.array_equal(a2, b2), rep
        assert np.array_equal(g_net.losses(), e_net.losses()), rep
    g_net.close()
    e_net.close()
