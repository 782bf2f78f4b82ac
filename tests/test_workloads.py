"""Properties of the seeded synthetic inputs (shapes, distributions, plant)."""
import math

import numpy as np
import torch

from workloads import gen

D = 128


def test_planted_mass_is_eighty_percent():
    s = gen.spec("c3", ctx=(8192, 8192), num_seqs=2, hkv=2)
    lay = gen.make_layer(s, 0)
    q = lay["queries"]
    for b in range(2):
        for h in range(2):
            k = lay["k"][b, h].double()
            qg = q[b, h * s.group:(h + 1) * s.group].double()
            z = (qg @ k.T) / math.sqrt(D)
            p = torch.softmax(z, dim=1)
            m = lay["planted"][(b, h)]
            assert int(m.sum()) == 64 * max(1, (8192 // 64) * 5 // 100)
            mass = float(p[:, m].sum(1).mean())
            assert abs(mass - 0.80) < 0.005


def test_shapes_ragged_and_rotations_orthogonal():
    s = gen.spec("c5", ctx=(300, 77, 129), appends=4)
    lay = gen.make_layer(s, 0)
    assert lay["k"].shape == (3, 4, 300, D) and lay["k"].dtype == torch.bfloat16
    assert float(lay["k"][1, :, 77:].abs().sum()) == 0.0
    R = lay["rot_k"][0, 1, 0].double()
    assert torch.allclose(R @ R.T, torch.eye(D, dtype=torch.float64), atol=1e-5)
    # rows ordered by descending eigenvalue of the window's X^T X
    X = lay["k"][0, 1, :300].double()
    ev = ((X @ R.T) ** 2).sum(0)
    assert bool((ev[:-1] >= ev[1:] * (1 - 1e-6)).all())


def test_outlier_heads_fixed_across_sequences():
    s = gen.spec("c1", ctx=(2048, 2048))
    lay = gen.make_layer(s, 0)
    for h in range(2):
        var0 = lay["k"][0, h].float().pow(2).mean(0)
        var1 = lay["k"][1, h].float().pow(2).mean(0)
        top0 = set(torch.topk(var0, 4).indices.tolist())
        top1 = set(torch.topk(var1, 4).indices.tolist())
        assert top0 == top1 and float(var0[list(top0)].min()) > 30
