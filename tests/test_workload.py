"""The shared seeded input generator: host and device backends agree bit for
bit, and the draws have the intended shapes and moments."""
import numpy as np
import pytest
import torch

from paper_2607_11185_amd import workload as WL


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_numpy_and_torch_backends_identical(dtype):
    idx = np.arange(1000, 9000)
    a = WL.normal_np(3, 1, idx, 0.02, dtype)
    b = WL.normal_torch(3, 1, 1000, 8000, 0.02, dtype, device="cpu", chunk=3000)
    assert np.array_equal(a, b.to(torch.float64).numpy())
    ti = WL.uniform_int_np(3, 5, idx, 151936)
    tt = WL.uniform_int_torch(3, 5, 1000, 8000, 151936, device="cpu")
    assert np.array_equal(ti, tt.numpy())


def test_moments_and_ranges():
    z = WL.normal_np(0, 1, np.arange(200000), 1.0, "f32")
    assert abs(z.mean()) < 0.01 and abs(z.var() - 1.0) < 0.01
    t = WL.uniform_int_np(0, 5, np.arange(100000), 1024)
    assert t.min() >= 0 and t.max() < 1024


def test_large_index_counters_differ():
    a = WL.normal_np(0, 1, np.array([5, (1 << 32) + 5]), 1.0, "f32")
    assert a[0] != a[1]


def test_spans_of_configs():
    sp = WL.make_spans(WL.SEVEN_B)
    assert sp.num_traj == 8 and sp.num_steps == 240
    assert sp.text_len.min() >= 150 and sp.text_len.max() <= 400
    assert (sp.action_len == 32).all() and (sp.img_len == 2691).all()
    lg = WL.make_spans(WL.LONG)
    T = np.diff(lg.step_offsets)
    assert T.min() >= 10 and T.max() <= 50


def test_layer_generators_host_and_device_identical():
    a = WL.layer_weights_np(3, 40, 24, 2, 1, 64)
    b = WL.layer_weights_torch(3, 40, 24, 2, 1, 64, device="cpu")
    for n, shp in WL.layer_shapes(40, 24, 2, 1, 64).items():
        assert a[n].shape == shp and tuple(b[n].shape) == shp
        assert np.array_equal(a[n], b[n].to(torch.float64).numpy()), n
    # projections have unit-variance rows after the 1/sqrt(fan_in) scale
    assert abs(a["wg"].std() * np.sqrt(40) - 1.0) < 0.1
    assert abs(a["g1"].mean() - 1.0) < 0.1
    x = WL.layer_rows_np(3, "x", np.array([4, 0, 6]), 40)
    xt = WL.layer_rows_torch(3, "x", 7, 40, device="cpu")
    assert np.array_equal(x, xt.to(torch.float64).numpy()[[4, 0, 6]])


def test_spans_subset():
    sp = WL.make_spans(WL.SMALL)
    a, b = sp.subset(0, 2), sp.subset(2, 4)
    assert a.num_traj == 2 and b.num_traj == 2 and a.num_steps + b.num_steps == sp.num_steps
    assert np.array_equal(np.concatenate([a.traj_tokens(), b.traj_tokens()]), sp.traj_tokens())
    assert np.array_equal(np.concatenate([a.text_len, b.text_len]), sp.text_len)
