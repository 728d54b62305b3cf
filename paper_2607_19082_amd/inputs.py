"""Seeded synthetic inputs and workload shapes.

This module holds no part of the method's arithmetic: it only draws random
arrays of the shapes and value distributions of the paper's workloads, and it
is the one piece shared by the GPU path's tests/benchmark and the CPU oracle.

The paper evaluates pre-trained CompressAI models on Kodak (768x512 images,
a 48x32 latent at /16), Tecnick and CLIC (Sec. IV-A).  Neither the datasets
nor the trained weights are used here; seeded draws stand in for them:

* weights ~ N(0, 1/fan_in), drawn with seed 0 in the order ctx_w, ctx_b, w1,
  b1, w2, b2, w3, b3 (biases from the same law, so a dropped bias shows);
  ctx_w is drawn for all 25 positions of the 5x5 kernel and fan_in counts the
  12 causal taps; the method ignores the masked positions;
* hyperprior parameters psi ~ N(0, 1), NHWC [B][H][W][2M], seed 1;
* symbols: continuous Laplace(0, b) rounded half-to-even and clipped to
  [-clip, clip], int32 NHWC [B][H][W][M], seed 2;
* encoder noise u ~ U(-0.5 + g, 0.5 - g), seed 3 (the encoder input is
  symbol + u + mean of the matching decode);
* the scale table: 64 levels spaced evenly in log between 0.11 and 256,
  computed in fp64 and rounded to fp32 once;
* transform weights (hyper-decoder and synthesis, for timing only), seed 4:
  conv weights ~ N(0, 1/fan_in), biases from the same law, GDN beta ~
  1 + U(0, 0.1) and gamma = 0.1 I + U(0, 0.01 / N) (positive, as GDN needs);
* the quantised hyper-latent z_hat: N(0, 2) rounded half-to-even, seed 5.
"""
import numpy as np

# Workloads.  d1 = floor(10M/3), d2 = floor(8M/3); n3 = 2M (mean, scale) or
# 9M (weight, mean, scale of 3 mixture components).
WORKLOADS = {
    "minnen-16x16-m192": dict(H=16, W=16, M=192, B=1, K=1, relaxed=False, lap_b=2.0, clip=32),
    "minnen-kodak-48x32-m192": dict(H=32, W=48, M=192, B=1, K=1, relaxed=False, lap_b=2.0, clip=32),
    "cheng-gmm3-1080p-120x68-m192": dict(H=68, W=120, M=192, B=1, K=3, relaxed=False, lap_b=3.0, clip=64),
    "minnen-relaxed-b8-120x68-m192": dict(H=68, W=120, M=192, B=8, K=1, relaxed=True, lap_b=2.0, clip=32),
    "minnen-hr-4k-240x135-m320": dict(H=135, W=240, M=320, B=1, K=1, relaxed=False, lap_b=4.0, clip=128),
}

ENCODE_GUARD = 1e-3


def widths(M, K):
    """(d1, d2, n3) of the entropy-parameter network for M channels."""
    return (10 * M) // 3, (8 * M) // 3, (2 if K == 1 else 9) * M


def scale_table(levels=64, lo=0.11, hi=256.0):
    """Log-spaced scale levels (fp64 -> fp32 once)."""
    k = np.arange(levels, dtype=np.float64)
    t = np.exp(np.log(lo) + k * (np.log(hi) - np.log(lo)) / (levels - 1))
    return t.astype(np.float32)


def make_weights(M, K, seed=0, radius=2):
    """Random weights of the context model and the parameter network, in
    PyTorch layouts: ctx_w [2M][M][2R+1][2R+1] (R = radius; 5x5 by default),
    w1 [d1][4M], w2 [d2][d1], w3 [n3][d2].  fan_in of the conv is its number
    of causal taps (2R^2 + 2R) times M."""
    d1, d2, n3 = widths(M, K)
    rng = np.random.default_rng(seed)

    def draw(shape, fan_in):
        return (rng.standard_normal(shape) / np.sqrt(fan_in)).astype(np.float32)

    w = {}
    k, taps = 2 * radius + 1, 2 * radius * radius + 2 * radius
    w["ctx_w"] = draw((2 * M, M, k, k), taps * M)
    w["ctx_b"] = draw((2 * M,), taps * M)
    w["w1"] = draw((d1, 4 * M), 4 * M)
    w["b1"] = draw((d1,), 4 * M)
    w["w2"] = draw((d2, d1), d1)
    w["b2"] = draw((d2,), d1)
    w["w3"] = draw((n3, d2), d2)
    w["b3"] = draw((n3,), d2)
    return w


def make_psi(B, H, W, M, seed=1):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((B, H, W, 2 * M), dtype=np.float32)


def make_symbols(B, H, W, M, lap_b, clip, seed=2):
    rng = np.random.default_rng(seed)
    v = rng.laplace(0.0, lap_b, size=(B, H, W, M))
    return np.clip(np.rint(v), -clip, clip).astype(np.int32)


def make_noise(B, H, W, M, guard=ENCODE_GUARD, seed=3):
    rng = np.random.default_rng(seed)
    return rng.uniform(-0.5 + guard, 0.5 - guard, size=(B, H, W, M)).astype(np.float32)


def encoder_input(sym, noise, mean):
    """y = symbol + noise + mean, in fp32."""
    return (sym.astype(np.float32) + noise) + mean.astype(np.float32)


def workload(name):
    """Shape and distribution parameters of a named workload."""
    cfg = dict(WORKLOADS[name])
    cfg["d1"], cfg["d2"], cfg["n3"] = widths(cfg["M"], cfg["K"])
    cfg["name"] = name
    return cfg


def make_inputs(name, H=None, W=None, B=None):
    """Weights, table, psi and symbols of a named workload; H, W, B may be
    overridden to draw a smaller grid with the same distributions."""
    cfg = workload(name)
    if H is not None:
        cfg["H"] = H
    if W is not None:
        cfg["W"] = W
    if B is not None:
        cfg["B"] = B
    w = make_weights(cfg["M"], cfg["K"])
    psi = make_psi(cfg["B"], cfg["H"], cfg["W"], cfg["M"])
    sym = make_symbols(cfg["B"], cfg["H"], cfg["W"], cfg["M"], cfg["lap_b"], cfg["clip"])
    return cfg, w, scale_table(), psi, sym


def make_transform_weights(N, M, seed=4):
    """Random weights of the hyper-decoder (hs1..hs3) and the synthesis
    transform (gs1..gs4 with GDN parameters gdn1..gdn3), PyTorch layouts:
    transposed convs [in][out][5][5], the 3x3 conv [out][in][3][3]."""
    rng = np.random.default_rng(seed)

    def draw(shape, fan_in):
        return (rng.standard_normal(shape) / np.sqrt(fan_in)).astype(np.float32)

    w = {}
    c = M * 3 // 2
    for name, cin, cout in (("hs1", N, M), ("hs2", M, c)):
        w[name + "_w"] = draw((cin, cout, 5, 5), cin * 25 // 4)
        w[name + "_b"] = draw((cout,), cin * 25 // 4)
    w["hs3_w"] = draw((2 * M, c, 3, 3), c * 9)
    w["hs3_b"] = draw((2 * M,), c * 9)
    for k, (cin, cout) in enumerate(((M, N), (N, N), (N, N), (N, 3)), start=1):
        w[f"gs{k}_w"] = draw((cin, cout, 5, 5), cin * 25 // 4)
        w[f"gs{k}_b"] = draw((cout,), cin * 25 // 4)
        if k < 4:
            w[f"gdn{k}_beta"] = (1.0 + 0.1 * rng.random(cout)).astype(np.float32)
            w[f"gdn{k}_gamma"] = (0.1 * np.eye(cout) + (0.01 / cout) * rng.random((cout, cout))).astype(np.float32)
    return w


def make_zhat(B, Hz, Wz, N, seed=5):
    """Quantised hyper-latent [B][Hz][Wz][N] (integer values as fp32)."""
    rng = np.random.default_rng(seed)
    return np.rint(rng.normal(scale=2.0, size=(B, Hz, Wz, N))).astype(np.float32)
