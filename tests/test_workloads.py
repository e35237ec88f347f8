"""The synthetic-input generator and the model shapes."""
import numpy as np

from workloads import configs, models, rng


def test_splitmix64_published_outputs():
    # first three outputs of SplitMix64 seeded with 0 (Vigna's reference implementation)
    outs = rng.mix((np.arange(1, 4, dtype=np.uint64) * rng.GAMMA))
    assert [int(v) for v in outs] == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_counter_access_equals_sequential_stream():
    key = 7
    s = int(rng.stream_seed(key))
    g = 0x9E3779B97F4A7C15
    seq = []
    x = s
    for _ in range(12):
        x = (x + g) % (1 << 64)
        seq.append(int(rng.mix(np.array([x], dtype=np.uint64))[0]))
    got = [int(rng.draw(key, np.array([i]), j)[0]) for i in range(3) for j in range(4)]
    assert got == seq


def test_uniform_values_are_cell_midpoints():
    u = rng.uniform(3, np.arange(200000))
    assert u.dtype == np.float32
    assert np.all(np.abs(u) < 1)
    k = (u.astype(np.float64) * 2 ** 24 + 2 ** 24 - 1) / 2
    assert np.all(k == np.round(k))  # (2k + 1 - 2^24) * 2^-24 exactly
    assert abs(u.mean()) < 0.01 and abs(u.var() - 1 / 3) < 0.01


def test_normal_moments_and_grid():
    x = rng.normal(0, np.arange(400000), 0.01)
    assert x.dtype == np.float32
    assert abs(x.mean()) < 1e-4
    assert abs(x.std() - 0.01) < 1e-4
    assert np.max(np.abs(x)) <= 6 * 0.01 * (1 + 1e-6)
    # about 0.3% of the mass lies beyond 3 sigma for a normal distribution
    assert 0.001 < np.mean(np.abs(x) > 0.03) < 0.006
    # the fraction that falls below binary16's normal range (gradual underflow matters)
    sub = np.mean(np.abs(x) < 2.0 ** -14)
    assert 0.002 < sub < 0.008


def test_keys_and_indices_give_different_streams():
    a = rng.normal(0, np.arange(1000))
    b = rng.normal(1, np.arange(1000))
    c = rng.normal(0, np.arange(1, 1001))
    assert np.array_equal(a[1:], c[:-1])  # counter-based: index i is the same value anywhere
    assert np.mean(a == b) < 0.01


def test_model_totals():
    # parameter totals of the architectures as specified (He et al. 2015 ResNet-50 with
    # batch-norm scale and shift; Inception-V3 without the auxiliary head; VGG-16 D)
    want = {"tiny": (8, 20388), "resnet50": (161, 25557032), "inceptionv3": (284, 23834568), "vgg16": (32, 138357544)}
    for name, (nt, total) in want.items():
        t = models.MODELS[name]()
        assert len(t) == nt and sum(models.numel_list(t)) == total
    inc = models.inception_v3()
    assert sum(1 for n, _ in inc if n.endswith("/w") and not n.startswith("fc")) == 94
    assert sum(int(np.prod(s)) for n, s in inc if n.endswith("bn_gamma")) == 17216
    vgg = dict(models.vgg16())
    assert int(np.prod(vgg["fc6/w"])) == 102760448


def test_workloads_ready_order_and_bytes():
    w = configs.get("tiny")
    assert w.numel() == [10000, 513, 4096, 4608, 1000, 100, 64, 7]
    assert w.prefix()[:3] == [0, 10000, 10513]
    assert configs.get("vgg16").rank_bytes == 553430176
    assert configs.get("resnet50").rank_bytes == 102228128
    assert [configs.get(n).nranks for n in configs.WORKLOADS] == [4, 8, 16, 32, 64]
