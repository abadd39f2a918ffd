"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no FGQ arithmetic: it only draws fp32 weights and fp32
activations with the shapes and value distributions of the paper's workloads
(ResNet-50/101 and AlexNet on 224x224 ImageNet images, Sec. 4), and lists the
layer shapes.  The oracle and the HIP library receive the same bytes.

Recipe (the paper's trained weights and ImageNet images are not available):
  * weights   He-Gaussian N(0, 2/fan_in), fan_in = C*R*S, layout [O][C][R][S]
  * acts      ReLU(N(0, 1)), NHWC float32 (about half exact zeros, like
              post-ReLU feature maps)
  * generator numpy PCG64 seeded from SeedSequence(170501462, spawn_key=key)
              where key is derived from a textual tag, so every tensor has its
              own reproducible stream.
"""
import zlib

import numpy as np

SEED = 170501462


def rng(*tags):
    key = tuple(zlib.crc32(str(t).encode()) for t in tags)
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(SEED, spawn_key=key)))


def he_weights(O, C, R, S, *tags):
    std = np.sqrt(2.0 / (C * R * S))
    return (rng("w", O, C, R, S, *tags).standard_normal((O, C, R, S)) * std).astype(np.float32)


def gauss_weights(O, K, std, *tags):
    return (rng("wg", O, K, std, *tags).standard_normal((O, K)) * std).astype(np.float32)


def relu_gauss(shape, *tags):
    x = rng("x", *shape, *tags).standard_normal(shape).astype(np.float32)
    return np.maximum(x, np.float32(0.0))


def laplace_weights(O, K, scale, *tags):
    """Heavy-tailed weights (|w| exponential), as the paper reports for early
    layers of trained networks (Sec. 3.1, Fig. 1 discussion)."""
    return rng("wl", O, K, scale, *tags).laplace(0.0, scale, (O, K)).astype(np.float32)


def conv_out(H, W, R, S, stride, pad):
    return (H + 2 * pad - R) // stride + 1, (W + 2 * pad - S) // stride + 1


# ---------------------------------------------------------------------------
# Workload shapes.  A conv layer is (name, B, H, W, C, O, R, S, stride, pad).
# ---------------------------------------------------------------------------

GEMM_SMALL = dict(M=64, K=256, O=128, G=4, bits=8, wstd=0.05)  # single FGQ GEMM

CONV3X3_C128 = dict(name="conv3_x 3x3 128->128", B=32, H=28, W=28, C=128, O=128,
                    R=3, S=3, stride=1, pad=1)
CONV1X1_C256 = dict(name="conv 1x1 256->64", B=32, H=56, W=56, C=256, O=64,
                    R=1, S=1, stride=1, pad=0)


def resnet_convs(depth, batch, hw=224):
    """torchvision v1.5 bottleneck ResNet conv shapes (stride on the 3x3) for
    hw x hw input images (224 is the standard size).

    conv1 has its 3 input channels zero-padded to 4 so that a group of 4
    input channels exists; the stem's 3x3 max pooling (stride 2, pad 1)
    follows it.  Returns a list of dicts, then the FC as a 1x1 conv on a
    1x1 map.
    """
    blocks = {50: [3, 4, 6, 3], 101: [3, 4, 23, 3]}[depth]
    layers = [dict(name="conv1", B=batch, H=hw, W=hw, C=4, O=64, R=7, S=7, stride=2, pad=3)]
    H = ((hw + 6 - 7) // 2 + 1 + 2 - 3) // 2 + 1  # conv1 (7x7, stride 2, pad 3), then the max pooling
    cin = 64
    for li, (nb, width) in enumerate(zip(blocks, [64, 128, 256, 512])):
        for bi in range(nb):
            stride = 2 if (bi == 0 and li > 0) else 1
            Ho = (H - 1) // stride + 1
            p = f"l{li + 1}.{bi}"
            layers.append(dict(name=p + ".c1", B=batch, H=H, W=H, C=cin, O=width, R=1, S=1, stride=1, pad=0))
            layers.append(dict(name=p + ".c2", B=batch, H=H, W=H, C=width, O=width, R=3, S=3, stride=stride, pad=1))
            layers.append(dict(name=p + ".c3", B=batch, H=Ho, W=Ho, C=width, O=4 * width, R=1, S=1, stride=1, pad=0))
            if bi == 0:
                layers.append(dict(name=p + ".ds", B=batch, H=H, W=H, C=cin, O=4 * width, R=1, S=1, stride=stride, pad=0))
            cin = 4 * width
            H = Ho
    layers.append(dict(name="fc", B=batch, H=1, W=1, C=2048, O=1000, R=1, S=1, stride=1, pad=0))
    return layers


def alexnet_layers(batch):
    """AlexNet shapes (single tower, 227x227 input; the 3 image channels
    zero-padded to 4; pooling between layers is not part of the FGQ layer).
    The fully-connected layers are GEMMs with M = batch."""
    return [
        dict(name="conv1", B=batch, H=227, W=227, C=4, O=96, R=11, S=11, stride=4, pad=0),
        dict(name="conv2", B=batch, H=27, W=27, C=96, O=256, R=5, S=5, stride=1, pad=2),
        dict(name="conv3", B=batch, H=13, W=13, C=256, O=384, R=3, S=3, stride=1, pad=1),
        dict(name="conv4", B=batch, H=13, W=13, C=384, O=384, R=3, S=3, stride=1, pad=1),
        dict(name="conv5", B=batch, H=13, W=13, C=384, O=256, R=3, S=3, stride=1, pad=1),
        dict(name="fc6", B=batch, H=1, W=1, C=9216, O=4096, R=1, S=1, stride=1, pad=0),
        dict(name="fc7", B=batch, H=1, W=1, C=4096, O=4096, R=1, S=1, stride=1, pad=0),
        dict(name="fc8", B=batch, H=1, W=1, C=4096, O=1000, R=1, S=1, stride=1, pad=0),
    ]
