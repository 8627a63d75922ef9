"""The seeded checkpoint generator gives the same bits through torch and numpy,
and has the stated distribution."""

import numpy as np
import torch

import synthetic_checkpoint as sc


def test_torch_and_numpy_agree():
    for t, (r, c) in [(0, (3, 7)), (17, (64, 33)), (12351, (5, 4096))]:
        for dt in ("f32", "bf16"):
            x = sc.values_torch(t, r, c, dt).reshape(-1)
            bits = x.view(torch.int32 if dt == "f32" else torch.int16).numpy()
            bits = bits.view(np.uint32 if dt == "f32" else np.uint16)
            assert np.array_equal(bits, sc.values_numpy(t, np.arange(r * c), dt))
            part = sc.values_torch(t, r, c, dt, start=5, count=11)
            assert torch.equal(part, x[5:16])


def test_distribution_and_distinct_tensors():
    x = sc.values_torch(3, 512, 512, "f32")
    assert abs(float(x.mean())) < 1e-3 and abs(float(x.std()) - 0.02) < 2e-4
    y = sc.values_torch(4, 512, 512, "f32")
    assert not torch.equal(x, y)
    b = sc.values_torch(3, 512, 512, "bf16")
    # bf16 values are the upper halves of the fp32 values
    assert torch.equal(b.view(torch.int16), (x.view(torch.int32) >> 16).to(torch.int16))
