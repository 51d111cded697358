"""Host-side checks of the synthetic workload definitions (shapes, counts,
kept-count rounding, seeded determinism)."""
import numpy as np

from workloads import (CHANNEL, ELEMENT, FILTER, SHAPE, WORKLOADS, alexnet_layers, get_workload,
                       input_nchw, kept_count, layer_tensors, resnet50_layers)


def test_resnet50_has_53_convs():
    L = resnet50_layers()
    assert len(L) == 53
    assert sum(l.n for l in L) == 23_454_912
    # output sizes of the stem and of the stride-2 3x3 / downsample convs
    assert (L[0].P, L[0].Q) == (112, 112)
    strided = [l for l in L if l.stride == 2][1:]
    assert sorted({(l.H, l.P) for l in strided}) == [(14, 7), (28, 14), (56, 28)]
    assert sorted({l.A for l in L}) == [64, 128, 256, 512, 1024, 2048]


def test_alexnet_geometry():
    L = alexnet_layers()
    assert [l.P for l in L] == [55, 27, 13, 13, 13]
    assert [l.in_channels for l in L] == [3, 96, 256, 384, 384]
    # each layer's input channels are the previous layer's filters (chain)
    assert all(L[i].in_channels == L[i - 1].A for i in range(1, 5))


def test_kept_counts():
    a = get_workload("alexnet_shape30")
    assert [a.k_for(i, SHAPE, 30) for i in range(5)] == [109, 360, 691, 518, 518]
    c = get_workload("alexnet_chain_f50c50")
    assert [c.k_for(i, FILTER, 50) for i in range(5)] == [48, 128, 192, 192, 128]
    r = get_workload("resnet50_filter60")
    assert sorted({r.k_for(i, FILTER, 60) for i in range(53)}) == [38, 77, 154, 307, 614, 1229]
    s = get_workload("resnet50_s3_sweep")
    assert [s.k_for(0, FILTER, p) for p in (10, 25, 50)] == [26, 64, 128]
    assert [s.k_for(0, SHAPE, p) for p in (10, 25, 50)] == [230, 576, 1152]
    assert [s.k_for(0, ELEMENT, p) for p in (10, 25, 50)] == [58982, 147456, 294912]
    assert get_workload("cifar_conv64").k_for(0, FILTER, 50) == 32
    assert kept_count(50, 3) == 2 and kept_count(50, 1) == 1 and kept_count(0, 10) == 0


def test_generators_are_seeded_and_distinct():
    wl = WORKLOADS["cifar_conv64"]
    W1, U1 = layer_tensors(wl, 0)
    W2, _ = layer_tensors(wl, 0)
    assert W1.dtype == np.float32 and W1.shape == (64, 64, 3, 3)
    assert np.array_equal(W1, W2) and not np.any(U1)
    assert abs(float(W1.std()) - 0.05) < 0.002
    X = input_nchw(wl, 0)
    assert X.shape == (8, 64, 32, 32) and X.dtype == np.float32
    wl2 = WORKLOADS["alexnet_shape30"]
    W, U = layer_tensors(wl2, 2)
    assert abs(float(U.std()) - 1e-4) < 1e-5
    assert not np.array_equal(W[:1], layer_tensors(wl2, 3)[0][:1])
