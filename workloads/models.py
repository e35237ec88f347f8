"""Gradient-tensor shapes of the benchmark models.

Only the element count of each trainable tensor matters to the allreduce, so each
model is a list of (name, shape) in *definition order* (input layer first).  The
order in which a backward pass produces gradients is the reverse of that;
`ready_order` gives it.  Shapes follow the architecture papers:

* ResNet-50: He, Zhang, Ren, Sun, "Deep Residual Learning for Image Recognition"
  (2015), Table 1, 50-layer column; bottleneck blocks; batch norm (scale + shift)
  after every convolution; convolutions without bias; 1x1 projection shortcut in
  the first block of each stage.
* Inception-V3: Szegedy, Vanhoucke, Ioffe, Shlens, Wojna, "Rethinking the Inception
  Architecture for Computer Vision" (2016), Table 1 with the module figures 5, 6
  and 7; 299x299 input; bias-free convolutions, each followed by batch norm
  (scale + shift); no auxiliary classifier.
* VGG-16: Simonyan & Zisserman, "Very Deep Convolutional Networks for Large-Scale
  Image Recognition" (2014), Table 1, configuration D; every layer has a bias.

Convolution weights are written (kh, kw, cin, cout).  The element counts are what
the paper under study calls the model size: its section on benchmarks explains
VGG-16's communication cost by its many fully connected parameters.
"""
from __future__ import annotations

from math import prod

__all__ = ["tiny", "resnet50", "inception_v3", "vgg16", "MODELS", "ready_order", "numel_list"]


def tiny():
    """The 8-tensor toy model: sizes {7, 64, 100, 1000, 3x3x16x32, 4096, 513, 10000}."""
    shapes = [(7,), (64,), (100,), (1000,), (3, 3, 16, 32), (4096,), (513,), (10000,)]
    return [(f"t{i}", s) for i, s in enumerate(shapes)]


def _conv_bn(out, name, kh, kw, cin, cout):
    out.append((f"{name}/w", (kh, kw, cin, cout)))
    out.append((f"{name}/bn_gamma", (cout,)))
    out.append((f"{name}/bn_beta", (cout,)))


def resnet50():
    """ResNet-50 trainable tensors (161 tensors)."""
    t = []
    _conv_bn(t, "conv1", 7, 7, 3, 64)
    cin = 64
    for stage, (width, blocks) in enumerate(zip((64, 128, 256, 512), (3, 4, 6, 3)), start=2):
        for b in range(blocks):
            p = f"conv{stage}_{b + 1}"
            _conv_bn(t, f"{p}/a", 1, 1, cin, width)
            _conv_bn(t, f"{p}/b", 3, 3, width, width)
            _conv_bn(t, f"{p}/c", 1, 1, width, 4 * width)
            if b == 0:
                _conv_bn(t, f"{p}/proj", 1, 1, cin, 4 * width)
            cin = 4 * width
    t.append(("fc/w", (2048, 1000)))
    t.append(("fc/b", (1000,)))
    return t


def inception_v3():
    """Inception-V3 trainable tensors (94 convolutions + batch norms, fc; 284 tensors)."""
    t = []
    c = lambda name, kh, kw, cin, cout: _conv_bn(t, name, kh, kw, cin, cout)  # noqa: E731
    # stem: 299x299x3 -> 35x35x192
    c("stem/1a", 3, 3, 3, 32)
    c("stem/2a", 3, 3, 32, 32)
    c("stem/2b", 3, 3, 32, 64)
    c("stem/3b", 1, 1, 64, 80)
    c("stem/4a", 3, 3, 80, 192)
    # three 35x35 modules (figure 5 with the 5x5 factored into two 3x3)
    cin = 192
    for name, pool in (("5b", 32), ("5c", 64), ("5d", 64)):
        m = f"mixed_{name}"
        c(f"{m}/b1x1", 1, 1, cin, 64)
        c(f"{m}/b5x5_1", 1, 1, cin, 48)
        c(f"{m}/b5x5_2", 5, 5, 48, 64)
        c(f"{m}/b3x3dbl_1", 1, 1, cin, 64)
        c(f"{m}/b3x3dbl_2", 3, 3, 64, 96)
        c(f"{m}/b3x3dbl_3", 3, 3, 96, 96)
        c(f"{m}/pool", 1, 1, cin, pool)
        cin = 64 + 64 + 96 + pool
    # grid reduction 35 -> 17
    c("mixed_6a/b3x3", 3, 3, cin, 384)
    c("mixed_6a/b3x3dbl_1", 1, 1, cin, 64)
    c("mixed_6a/b3x3dbl_2", 3, 3, 64, 96)
    c("mixed_6a/b3x3dbl_3", 3, 3, 96, 96)
    cin = 384 + 96 + cin  # 768
    # four 17x17 modules (figure 6, n = 7)
    for name, c7 in (("6b", 128), ("6c", 160), ("6d", 160), ("6e", 192)):
        m = f"mixed_{name}"
        c(f"{m}/b1x1", 1, 1, cin, 192)
        c(f"{m}/b7x7_1", 1, 1, cin, c7)
        c(f"{m}/b7x7_2", 1, 7, c7, c7)
        c(f"{m}/b7x7_3", 7, 1, c7, 192)
        c(f"{m}/b7x7dbl_1", 1, 1, cin, c7)
        c(f"{m}/b7x7dbl_2", 7, 1, c7, c7)
        c(f"{m}/b7x7dbl_3", 1, 7, c7, c7)
        c(f"{m}/b7x7dbl_4", 7, 1, c7, c7)
        c(f"{m}/b7x7dbl_5", 1, 7, c7, 192)
        c(f"{m}/pool", 1, 1, cin, 192)
        cin = 4 * 192
    # grid reduction 17 -> 8
    c("mixed_7a/b3x3_1", 1, 1, cin, 192)
    c("mixed_7a/b3x3_2", 3, 3, 192, 320)
    c("mixed_7a/b7x7x3_1", 1, 1, cin, 192)
    c("mixed_7a/b7x7x3_2", 1, 7, 192, 192)
    c("mixed_7a/b7x7x3_3", 7, 1, 192, 192)
    c("mixed_7a/b7x7x3_4", 3, 3, 192, 192)
    cin = 320 + 192 + cin  # 1280
    # two 8x8 modules (figure 7, expanded filter bank)
    for name in ("7b", "7c"):
        m = f"mixed_{name}"
        c(f"{m}/b1x1", 1, 1, cin, 320)
        c(f"{m}/b3x3_1", 1, 1, cin, 384)
        c(f"{m}/b3x3_2a", 1, 3, 384, 384)
        c(f"{m}/b3x3_2b", 3, 1, 384, 384)
        c(f"{m}/b3x3dbl_1", 1, 1, cin, 448)
        c(f"{m}/b3x3dbl_2", 3, 3, 448, 384)
        c(f"{m}/b3x3dbl_3a", 1, 3, 384, 384)
        c(f"{m}/b3x3dbl_3b", 3, 1, 384, 384)
        c(f"{m}/pool", 1, 1, cin, 192)
        cin = 320 + 768 + 768 + 192  # 2048
    t.append(("fc/w", (2048, 1000)))
    t.append(("fc/b", (1000,)))
    return t


def vgg16():
    """VGG-16 (configuration D) trainable tensors (32 tensors)."""
    t = []
    cin = 3
    for i, cout in enumerate((64, 64, 128, 128, 256, 256, 256, 512, 512, 512, 512, 512, 512)):
        t.append((f"conv{i + 1}/w", (3, 3, cin, cout)))
        t.append((f"conv{i + 1}/b", (cout,)))
        cin = cout
    for name, (fin, fout) in (("fc6", (7 * 7 * 512, 4096)), ("fc7", (4096, 4096)), ("fc8", (4096, 1000))):
        t.append((f"{name}/w", (fin, fout)))
        t.append((f"{name}/b", (fout,)))
    return t


MODELS = {"tiny": tiny, "resnet50": resnet50, "inceptionv3": inception_v3, "vgg16": vgg16}


def ready_order(tensors):
    """Gradients become ready in reverse definition order during backpropagation."""
    return list(reversed(tensors))


def numel_list(tensors):
    return [prod(shape) for _, shape in tensors]
