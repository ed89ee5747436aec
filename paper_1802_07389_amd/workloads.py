"""Seeded synthetic inputs for the 3LC path.

This module only draws random numbers; it holds none of the method's
arithmetic, so both the HIP path and the CPU oracle consume exactly the same
fp32 bytes from it.  Every generator uses numpy's PCG64 (``default_rng``).

The workloads stand in for the state changes of the paper's evaluation
(ResNet-110 on CIFAR-10, Section 5.2), which need a dataset, trained weights
and a training cluster; none of those are used here.

Distributions: ``N(0, sigma)`` draws have standard deviation ``sigma``;
``Laplace(0, b)`` draws have scale ``b``.
"""
import numpy as np

F32 = np.float32


# ---------------------------------------------------------------- C1
C1_N = 1 << 20
C1_S = 1.0


def c1_tensor():
    """2^20 values ~ N(0, 1e-3) from seed 0; the residual starts at zero."""
    rng = np.random.default_rng(0)
    return rng.standard_normal(C1_N, dtype=F32) * F32(1e-3)


# ---------------------------------------------------------------- C2
C2_S = 1.75
C2_STEPS = 10


def resnet110_cifar_shapes():
    """Parameter tensors of ResNet-110 for CIFAR-10, in network order.

    Returns a list of (name, shape, kind) with kind in {"conv", "bn", "fc"}.
    3x3 conv 3->16, then three stages (16, 32, 64 channels) of 18 basic
    blocks with two 3x3 convs each; a 1x1 projection where the channel count
    changes; batch-norm gamma and beta after every conv and projection; a
    64x10 fully connected layer with bias.  335 tensors, 1,730,714 values.
    """
    out = []

    def conv(name, k, cin, cout):
        out.append((name + ".w", (k, k, cin, cout), "conv"))
        out.append((name + ".bn.gamma", (cout,), "bn"))
        out.append((name + ".bn.beta", (cout,), "bn"))

    conv("conv1", 3, 3, 16)
    cin = 16
    for stage, width in enumerate((16, 32, 64)):
        for block in range(18):
            pre = f"s{stage}.b{block}"
            conv(pre + ".a", 3, cin, width)
            conv(pre + ".b", 3, width, width)
            if cin != width:
                conv(pre + ".proj", 1, cin, width)
            cin = width
    out.append(("fc.w", (64, 10), "fc"))
    out.append(("fc.b", (10,), "fc"))
    return out


def c2_sizes():
    return [int(np.prod(shape)) for _, shape, _ in resnet110_cifar_shapes()]


def c2_sigma(t):
    """sigma_t = 10^U(-4, -2), drawn once per tensor t."""
    rng = np.random.default_rng([2, 0, t])
    return F32(10.0 ** rng.uniform(-4.0, -2.0))


def c2_gradient(step, t, n):
    """Step ``step`` (0-based) gradient of tensor t: N(0, sigma_t)."""
    rng = np.random.default_rng([2, step + 1, t])
    return rng.standard_normal(n, dtype=F32) * c2_sigma(t)


# ---------------------------------------------------------------- C3
C3_N = 1 << 26
C3_S = (1.0, 1.5, 1.9)
C3_ZERO_RUN_P = 1.0 / 40.0   # zero runs ~ Geometric(1/40), mean 40
C3_NZ_RUN_P = 7.0 / 120.0    # non-zero runs ~ Geometric(7/120), mean 17.14


def c3_tensor(n=C3_N):
    """Laplace(0, 1e-3) values with 70% of positions exactly +0.0 in runs.

    Runs alternate between zero and non-zero; the first run is a zero run
    with probability 0.7.  Run lengths are geometric on {1, 2, ...}.
    """
    rng = np.random.default_rng([3, 0, 0])
    zero_first = rng.random() < 0.7
    lens = []
    total = 0
    # draw run pairs in batches until they cover n positions
    while total < n:
        k = max(1024, int((n - total) / 57.0 * 1.1) + 1)
        z = rng.geometric(C3_ZERO_RUN_P, size=k)
        nz = rng.geometric(C3_NZ_RUN_P, size=k)
        pair = np.empty(2 * k, dtype=np.int64)
        if zero_first:
            pair[0::2], pair[1::2] = z, nz
        else:
            pair[0::2], pair[1::2] = nz, z
        lens.append(pair)
        total += int(pair.sum())
    lens = np.concatenate(lens)
    is_zero = np.zeros(lens.size, dtype=bool)
    is_zero[0 if zero_first else 1::2] = True
    mask = np.repeat(is_zero, lens)[:n]
    vals = np.random.default_rng([3, 0, 1]).laplace(0.0, 1e-3, n).astype(F32)
    vals[mask] = F32(0.0)
    return vals


# ---------------------------------------------------------------- C4
C4_N = 1 << 28
C4_S = 1.75
C4_STEPS = 5


def c4_tensor(step, n=C4_N):
    """Step ``step`` input: 2^28 values ~ N(0, 1e-3) (1 GiB of fp32)."""
    rng = np.random.default_rng([4, step, 0])
    return rng.standard_normal(n, dtype=F32) * F32(1e-3)


# ---------------------------------------------------------------- C5
C5_N = 25_600_000
C5_PAYLOADS = 16
C5_S = 1.75


def c5_tensor(p, n=C5_N):
    """Worker p's input (p = 0..15): N(0, 1e-3)."""
    rng = np.random.default_rng([5, p, 0])
    return rng.standard_normal(n, dtype=F32) * F32(1e-3)


# ---------------------------------------------------------------- misc
def normal(seed, n, sigma=1e-3):
    """Generic N(0, sigma) test tensor from an integer-sequence seed."""
    rng = np.random.default_rng(seed)
    return rng.standard_normal(n, dtype=F32) * F32(sigma)


def runs_tensor(seed, n, zero_frac=0.7, mean_zero_run=40.0, b=1e-3):
    """Small C3-style tensor: alternating zero / Laplace runs."""
    rng = np.random.default_rng(seed)
    p_zero = 1.0 / mean_zero_run
    mean_nz = mean_zero_run * (1.0 - zero_frac) / zero_frac
    p_nz = 1.0 / max(mean_nz, 1.0)
    k = n // 2 + 2
    z = rng.geometric(p_zero, size=k)
    nz = rng.geometric(p_nz, size=k)
    lens = np.empty(2 * k, dtype=np.int64)
    lens[0::2], lens[1::2] = z, nz
    is_zero = np.zeros(2 * k, dtype=bool)
    is_zero[0::2] = True
    mask = np.repeat(is_zero, lens)[:n]
    vals = rng.laplace(0.0, b, n).astype(F32)
    vals[mask] = F32(0.0)
    return vals
