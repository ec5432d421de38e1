"""The allocation-free training step (pmlp_train_step_noalloc) against
pmlp_train_step: same kernels, so the same losses and weights bit for bit,
on two calls in a row, the second with a smaller batch (the static
workspace keeps the first call's contents)."""
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


def dev(torch, a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# (hidden sizes, F, O, first batch, second batch): the three-piece kernels
# with segments wider than the M3 tile (logits cleared before the split
# halves add into them), and the matrix-core M3 kernels at O = 10
SHAPES = {
    "f100_split": (np.array([1300, 3, 700, 1, 1024, 40, 513, 2] * 3, np.int32), 100, 2, 200, 70),
    "f32_o10": (np.random.default_rng(4).integers(1, 300, 60).astype(np.int32), 32, 10, 64, 29),
}


@pytest.mark.parametrize("name", sorted(SHAPES))
def test_noalloc_step_equals_train_step(pm, torch, name):
    hs, F, O, B1, B2 = SHAPES[name]
    acts = np.arange(len(hs), dtype=np.int32) % 10
    X, y = wl.make_dataset(F, O, B1 + B2, seed=77)
    ref = pm.PackedMLP(F, O, hs, acts, seed=5)
    net = pm.PackedMLP(F, O, hs, acts, seed=5)
    Xd, yd = dev(torch, X), dev(torch, y)
    for s, n in ((0, B1), (B1, B2)):
        Xb, yb = Xd[s:s + n], yd[s:s + n]
        ref._stream()
        pm.pmlp_train_step(ref.handle, Xb, yb, n, 0.05)
        net._stream()
        pm.pmlp_train_step_noalloc(net.handle, Xb, yb, n, 0.05)
        assert np.array_equal(net.losses(), ref.losses())
        a1, a2 = net.get_params()
        r1, r2 = ref.get_params()
        assert np.array_equal(a1, r1) and np.array_equal(a2, r2)
    net.close()
    ref.close()


def test_noalloc_step_rejects_what_does_not_fit(pm, torch):
    hs = np.full(300, 1000, np.int32)           # 300,000 units: 293 MiB of Z at 256 samples
    net = pm.PackedMLP(8, 2, hs, np.zeros(300, np.int32), seed=1)
    X = dev(torch, np.ones((256, 8), np.float32))
    y = dev(torch, np.zeros(256, np.int32))
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_train_step_noalloc(net.handle, X, y, 256, 0.1)
    assert e.value.code == pm.PMLP_EINVAL and "256 MiB" in str(e.value)
    pm.pmlp_train_step_noalloc(net.handle, X[:64], y[:64], 64, 0.1)   # 73 MiB fits
    assert np.all(np.isfinite(net.losses()))
    net.set_precision(pm.PMLP_BF16_GEMM)
    with pytest.raises(pm.PmlpError) as e:
        pm.pmlp_train_step_noalloc(net.handle, X[:64], y[:64], 64, 0.1)
    assert e.value.code == pm.PMLP_ESTATE
    net.close()
