"""Seeded synthetic inputs shaped like the paper's workloads.

This module holds no ESB arithmetic: it only draws fp32 tensors and the caller's
candidate grids for the scale search, so that the GPU path and the CPU oracle
are fed the same bytes.  Inputs come from NumPy's PCG64 stream seeded with
``[config_id, seed]``; weights are drawn first, then activations, each as
float64 normals, scaled, passed through the activation function and cast to
float32.

The paper's own data (ImageNet images and trained AlexNet / ResNet18 /
MobileNetV2 weights, Sec. 5.1) is not available; these tensors stand in for it
with the same layer shapes and the bell-shaped / rectified distributions the
paper assumes for weights and activations (Sec. 3.4).

Layouts: activations NHWC, convolution weights KRSC (K output channels,
R x S window, C input channels per group), matrices row-major.
"""
import numpy as np

GRID_POINTS = 64


def rng(config_id, seed):
    return np.random.default_rng([int(config_id), int(seed)])


def normal(r, shape, std):
    return (r.standard_normal(shape) * std).astype(np.float32)


def relu_normal(r, shape):
    return np.maximum(r.standard_normal(shape), 0.0).astype(np.float32)


def relu6_normal(r, shape):
    return np.clip(r.standard_normal(shape), 0.0, 6.0).astype(np.float32)


def scale_grid(s, points=GRID_POINTS):
    """Candidate scales s * 3 (j+1) / points, j = 0..points-1, in fp32.

    The paper searches alpha over (0, 3] for unit-variance data (Sec. 3.4);
    s is the spread of the data the grid is meant for (the generating standard
    deviation for weights, 1 for rectified unit-normal activations).
    """
    j = np.arange(1, points + 1, dtype=np.float64)
    return (np.float64(s) * (3.0 * j / points)).astype(np.float32)


def maxabs_grid_factors(cmax, points=GRID_POINTS):
    """Factors c_j = fl32((j+1) / (points * cmax)), j = 0..points-1, for the data-driven grid
    alpha_j = 2^E c_j of the ResNet18 stack, E the binary exponent of max|x|
    (2^(E-1) <= max|x| < 2^E; cmax: the largest set value, so the grid spans (0, 2^E / cmax]).
    Multiplying by a power of two is exact: the grid is the same on any device."""
    j = np.arange(1, points + 1, dtype=np.float64)
    return (j / (points * float(cmax))).astype(np.float32)


def tiny_gemm(seed=0):
    """64x576 weights N(0, 0.05) times 576x64 activations ReLU(N(0,1)); ESB n=4, k_sig=2."""
    r = rng(0, seed)
    W = normal(r, (64, 576), 0.05)
    A = relu_normal(r, (576, 64))
    return dict(name="tiny_gemm_64x576x64", W=W, A=A, nW=4, ksW=2, nA=4, ksA=2,
                gridW=scale_grid(0.05), gridA=scale_grid(1.0))


def resnet_conv3x3(seed=0):
    """ResNet18 layer1 3x3 conv, 64->64, 56x56, stride 1, pad 1, batch 1; ESB n=4, k_sig=2."""
    r = rng(1, seed)
    std = float(np.sqrt(2.0 / 576.0))
    w = normal(r, (64, 3, 3, 64), std)
    x = relu_normal(r, (1, 56, 56, 64))
    return dict(name="resnet18_conv3x3_64x56x56_b1", w=w, x=x, nW=4, ksW=2, nX=4, ksX=2,
                stride=(1, 1), pad=(1, 1), groups=1,
                gridW=scale_grid(std), gridX=scale_grid(1.0))


def alexnet_fc(seed=0):
    """AlexNet FC 9216->4096 at batch 128: W N(0, 0.01) ESB(3, k_sig=1), X ReLU(N(0,1)) ESB(3, k_sig=2)."""
    r = rng(2, seed)
    W = normal(r, (4096, 9216), 0.01)
    X = relu_normal(r, (128, 9216))
    return dict(name="alexnet_fc_9216x4096_b128", W=W, X=X, nW=3, ksW=1, nX=3, ksX=2,
                gridW=scale_grid(0.01), gridX=scale_grid(1.0))


def mobilenetv2_block(seed=0, batch=32):
    """MobileNetV2 inverted residual at 56x56: 1x1 24->144, dw 3x3 on 144, 1x1 144->24; ESB n=5, k_sig=3."""
    r = rng(3, seed)
    w_exp = normal(r, (144, 1, 1, 24), 0.1)
    w_dw = normal(r, (144, 3, 3, 1), 0.1)
    w_prj = normal(r, (24, 1, 1, 144), 0.1)
    x_exp = relu6_normal(r, (batch, 56, 56, 24))
    x_dw = relu6_normal(r, (batch, 56, 56, 144))
    x_prj = relu6_normal(r, (batch, 56, 56, 144))
    return dict(name="mobilenetv2_block_56x56_b%d" % batch, n=5, ks=3,
                layers=[dict(name="expand_1x1", w=w_exp, x=x_exp, stride=(1, 1), pad=(0, 0), groups=1),
                        dict(name="dw_3x3", w=w_dw, x=x_dw, stride=(1, 1), pad=(1, 1), groups=144),
                        dict(name="project_1x1", w=w_prj, x=x_prj, stride=(1, 1), pad=(0, 0), groups=1)],
                gridW=scale_grid(0.1), gridX=scale_grid(1.0))


# ResNet18 (He et al. 2016) convolution stack: (name, Cin, Cout, R, stride, pad).
RESNET18_CONVS = [
    ("conv1", 3, 64, 7, 2, 3),
    ("l1.0.c1", 64, 64, 3, 1, 1), ("l1.0.c2", 64, 64, 3, 1, 1),
    ("l1.1.c1", 64, 64, 3, 1, 1), ("l1.1.c2", 64, 64, 3, 1, 1),
    ("l2.0.c1", 64, 128, 3, 2, 1), ("l2.0.c2", 128, 128, 3, 1, 1), ("l2.0.ds", 64, 128, 1, 2, 0),
    ("l2.1.c1", 128, 128, 3, 1, 1), ("l2.1.c2", 128, 128, 3, 1, 1),
    ("l3.0.c1", 128, 256, 3, 2, 1), ("l3.0.c2", 256, 256, 3, 1, 1), ("l3.0.ds", 128, 256, 1, 2, 0),
    ("l3.1.c1", 256, 256, 3, 1, 1), ("l3.1.c2", 256, 256, 3, 1, 1),
    ("l4.0.c1", 256, 512, 3, 2, 1), ("l4.0.c2", 512, 512, 3, 1, 1), ("l4.0.ds", 256, 512, 1, 2, 0),
    ("l4.1.c1", 512, 512, 3, 1, 1), ("l4.1.c2", 512, 512, 3, 1, 1),
]


def resnet18_weights(seed=0):
    """He-init fp32 weights (std sqrt(2 / (R*S*Cin))) for every ResNet18 conv and the FC."""
    r = rng(4, seed)
    ws = {}
    for name, cin, cout, k, _, _ in RESNET18_CONVS:
        ws[name] = normal(r, (cout, k, k, cin), float(np.sqrt(2.0 / (k * k * cin))))
    ws["fc"] = normal(r, (1000, 512), float(np.sqrt(2.0 / 512)))
    return ws


def resnet18_input(seed=0, batch=64):
    r = rng(4, 1000 + seed)
    return normal(r, (batch, 224, 224, 3), 1.0)


def random_codes(seed, shape, n):
    """Uniform random n-bit codes (for contraction parity tests independent of projection)."""
    r = rng(99, seed)
    return r.integers(0, 1 << n, size=shape, dtype=np.uint8)
