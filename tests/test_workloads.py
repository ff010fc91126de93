"""Workload shapes against Table 1 and the layout rules; seeded generator."""
import numpy as np
import pytest

from workloads import gen, tables

# Table 1 ("Volumes of data and computation"), weight_size |W| column, in MB.
# Eq. 1 counts conv + FC weights only, 4 bytes each.  AlexNet's row matches
# the ungrouped network and GoogLeNet's the one with its two auxiliary
# classifiers; the benchmark workloads use the grouped AlexNet and GoogLeNet
# without auxiliary heads (both shapes are built here).
TABLE1_MB = {"nin": 30, "alexnet_ungrouped": 249, "googlenet_aux": 54, "vgg19": 575}


@pytest.mark.parametrize("name,mb", sorted(TABLE1_MB.items()))
def test_eq1_matches_table1(name, mb):
    wl = tables.get(name)
    assert abs(tables.eq1_weight_bytes(wl.layers) / 1e6 - mb) <= 1.0


@pytest.mark.parametrize("name,nseg,nparams,minseg", [
    ("flat", 1, 1 << 20, 1 << 20), ("nin", 24, 7_595_176, 96), ("googlenet", 116, 6_998_552, 16),
    ("vgg19", 38, 143_667_240, 64), ("alexnet", 16, 60_965_224, 96)])
def test_shapes(name, nseg, nparams, minseg):
    wl = tables.get(name)
    assert len(wl.segments) == nseg and wl.n_params == nparams
    assert min(s.length for s in wl.segments) == minseg


@pytest.mark.parametrize("name", ["flat", "nin", "googlenet", "googlenet_aux", "googlenet_caffe_bias", "vgg19",
                                  "alexnet", "alexnet_ungrouped"])
def test_layout_rules(name):
    wl = tables.get(name)
    end = 0
    for s in wl.segments:
        assert s.offset % tables.ALIGN == 0 and s.offset >= end and s.length > 0
        end = s.offset + s.length
    assert end <= wl.padded and wl.padded % tables.ALIGN == 0
    googlenet_convs = sum(1 for L in tables.googlenet_layers() if "classifier" not in L.name)
    assert googlenet_convs == 57


def test_host_generator_is_seeded_and_pads_with_zero():
    wl = tables.nin()
    segs = wl.segments[:3]
    a = gen.host_inputs(wl, 11, K=3, segments=segs)
    b = gen.host_inputs(wl, 11, K=3, segments=segs)
    c = gen.host_inputs(wl, 12, K=3, segments=segs)
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    assert not np.array_equal(a[0], c[0])
    reps = a[0]
    inside = np.zeros(reps.shape[1], bool)
    for s in segs:
        inside[s.offset:s.offset + s.length] = True
    assert np.all(reps[:, ~inside] == 0)
    # per-layer spread follows 1e-3/sqrt(fan_in)
    s0 = segs[0]
    sd = reps[:, s0.offset:s0.offset + s0.length].std()
    assert abs(sd / (1e-3 / np.sqrt(s0.fan_in)) - 1) < 0.05


def test_algorithmic_bytes():
    wl = tables.googlenet()
    assert wl.algorithmic_bytes() == wl.n_params * (128 * 4 + 16)
    assert wl.algorithmic_bytes(out=True, bcast=True) == wl.n_params * (128 * 4 + 16 + 4 + 4 * 128)
    assert tables.alexnet().algorithmic_bytes() == 60_965_224 * (128 * 2 + 16)


def test_caffe_bias_variant():
    """GoogLeNet with Caffe's bias multipliers: the layout of GoogLeNet, every
    bias segment (2, 0), every weight segment (1, 1)."""
    a, b = tables.googlenet(), tables.get("googlenet_caffe_bias")
    assert [(s.offset, s.length) for s in a.segments] == [(s.offset, s.length) for s in b.segments]
    assert b.name == "googlenet_caffe_bias" and b.n_params == a.n_params
    for s in b.segments:
        assert (s.lr_mult, s.decay_mult) == ((2.0, 0.0) if s.is_bias else (1.0, 1.0))
    assert sum(1 for s in b.segments if s.is_bias) == 58
