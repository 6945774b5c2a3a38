"""Seeded synthetic inputs for the MXFP4 backward hot path.

This module serves both the CPU oracle (in tests) and the GPU path; it holds
none of the method's arithmetic: only shapes, value distributions and the
float -> bf16 conversion of the generated data.

The paper trains GPT models on GPT2-Wikipedia (Sec. 4); that data and the
trained models are not available, so gradients, activations and weights are
drawn from distributions of the same shape and character:

* dY (output gradient): heavy tailed, 1e-3 * t_3 / sqrt(3) (Student t with 3
  degrees of freedom, rescaled to standard deviation 1e-3), sparse large
  outliers for the 6.7B shape (Sec. 3.2 mentions sparse gradients and
  block-level outliers).
* x (activations): N(0, 1).
* W (weights): N(0, 0.02^2), the usual GPT initialisation scale.
* Block outliers: whole 32-element row-major blocks picked i.i.d. with
  probability p and multiplied by a factor, after drawing.

Every value is drawn in float64 from numpy's PCG64 generator, rounded to
float32 (round to nearest even) and then to bf16 (round to nearest even).
Chunk c of 2^22 consecutive elements draws from its own stream,
PCG64(SeedSequence(seed).spawn(n)[c]), so chunks can be drawn in parallel
threads with a result independent of the thread count; block outliers are
picked (one draw per block, before any value) from the stream of
SeedSequence(seed) itself.
Sizes follow the paper's GPT configurations (Appendix B table): hidden 1024 /
2048 / 4096 for 345M / 1.3B / 6.7B, MLP width 4x hidden.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

BLOCK = 32


def fp32_to_bf16_bits(x):
    """Round finite float32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    b = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    # b + 0x7FFF + lsb stays below 2^32 for every finite float32
    rounded = (b + np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_float(bits):
    """uint16 bf16 bit patterns -> float32 values."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


CHUNK = 1 << 22
_THREADS = max(1, min(16, os.cpu_count() or 1))


def matrix(shape, seed, dist="normal", scale=1.0, outlier_p=0.0, outlier_factor=1.0):
    """One seeded bf16 matrix (uint16 bit patterns), row-major, of the given shape.

    The number of elements must be a multiple of 32 when outliers are used.
    """
    n = int(np.prod(shape))
    seq = np.random.SeedSequence(seed)
    hit = None
    if outlier_p > 0:
        if n % BLOCK:
            raise ValueError("outliers need a multiple of 32 elements")
        hit = np.random.Generator(np.random.PCG64(seq)).random(n // BLOCK) < outlier_p
    out = np.empty(n, dtype=np.uint16)
    nchunks = max(1, -(-n // CHUNK))
    children = seq.spawn(nchunks)

    def fill(c):
        rng = np.random.Generator(np.random.PCG64(children[c]))
        i = c * CHUNK
        m = min(CHUNK, n - i)
        if dist == "normal":
            v = rng.standard_normal(m)
        elif dist == "t3":
            v = rng.standard_t(3, m) / np.sqrt(3.0)
        else:
            raise ValueError(dist)
        v = (v * scale).astype(np.float32)
        if hit is not None:
            blocks = v.reshape(-1, BLOCK)
            blocks[hit[i // BLOCK:(i + m) // BLOCK]] *= np.float32(outlier_factor)
        out[i:i + m] = fp32_to_bf16_bits(v)

    if nchunks == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(max_workers=_THREADS) as pool:
            list(pool.map(fill, range(nchunks)))
    return out.reshape(shape)


# ---------------------------------------------------------------------------
# Workload configurations. Linear layers are (name, in_features, out_features);
# a transformer block has QKV h->3h, attention output projection h->h and the
# MLP h->4h, 4h->h.

def _gpt_block(h):
    return [("qkv", h, 3 * h), ("proj", h, h), ("fc1", h, 4 * h), ("fc2", 4 * h, h)]


CONFIGS = {
    # Single linear layer, small enough for the oracle to run in seconds.
    "tiny": dict(tokens=256, linears=[("linear", 256, 256)], g=[64], data_seed=0,
                 dy=dict(dist="normal", scale=1.0, outlier_p=0.01, outlier_factor=100.0),
                 x=dict(dist="normal", scale=1.0, outlier_p=0.01, outlier_factor=100.0),
                 w=dict(dist="normal", scale=1.0, outlier_p=0.01, outlier_factor=100.0)),
    # GPT-345M-shaped block: batch 2 x sequence 2048 tokens, hidden 1024.
    "gpt345m": dict(tokens=4096, linears=_gpt_block(1024), g=[64], data_seed=2,
                    dy=dict(dist="t3", scale=1e-3), x=dict(dist="normal", scale=1.0),
                    w=dict(dist="normal", scale=0.02)),
    # GPT-1.3B-shaped block: 8192 tokens, hidden 2048, MLP 8192; g swept.
    "gpt1.3b": dict(tokens=8192, linears=_gpt_block(2048), g=[32, 64, 128, 256], data_seed=3,
                    dy=dict(dist="t3", scale=1e-3), x=dict(dist="normal", scale=1.0),
                    w=dict(dist="normal", scale=0.02)),
    # GPT-6.7B-shaped block: 16384 tokens, hidden 4096, MLP 16384; 0.5% of dY
    # blocks are x1000 outliers.
    "gpt6.7b": dict(tokens=16384, linears=_gpt_block(4096), g=[64], data_seed=4,
                    dy=dict(dist="t3", scale=1e-3, outlier_p=0.005, outlier_factor=1000.0),
                    x=dict(dist="normal", scale=1.0), w=dict(dist="normal", scale=0.02)),
}

# Standalone quantiser sweep: N(0,1) matrices, row-major and transposed reads.
QUANT_SWEEP = dict(shapes=[(4096, 4096), (8192, 8192), (16384, 16384), (32768, 16384)],
                   g=[64, 256], data_seed=5)

# RHT overhead on a plain GEMM C = A B^T, A [n, k], B [m, k] (both bf16, N(0,1)),
# transformed and quantised along k: the 7B- and 70B-sized (m, n, k) of the
# paper's overhead estimate (Sec. 4.2), g = 64.
RHT_OVERHEAD = dict(shapes=[(32768, 8192, 8192), (16384, 28672, 28672)], g=64, data_seed=6)


# Sample vectors of the variance study (the figure of Sec. 3.2): A, B in R^b,
# A = z + m o with z ~ N(0, I), m ~ Bernoulli(p) per element and o ~ N(0, 5 I)
# (read as variance 5); n samples as the rows of an [n, b] matrix.
FIG2 = dict(n=4096, b=[32, 64, 128, 256, 512, 1024, 2048, 4096], p=[0.0, 0.01, 0.05], outlier_var=5.0,
            data_seed=7)


def mixture_vectors(n, b, p, seed, outlier_var=5.0):
    """[n, b] bf16 bit patterns: N(0, 1) entries plus, with probability p per
    entry, an independent N(0, outlier_var) term; float64 draws rounded to
    float32, then to bf16."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed)))
    z = rng.standard_normal((n, b))
    m = rng.random((n, b)) < p
    o = rng.standard_normal((n, b)) * np.sqrt(outlier_var)
    return fp32_to_bf16_bits((z + np.where(m, o, 0.0)).astype(np.float32))


def linear_inputs(config, linear):
    """(dY [T, out], x [T, in], W [out, in]) bf16 bit patterns for one linear of a config."""
    cfg = CONFIGS[config]
    names = [l[0] for l in cfg["linears"]]
    idx = names.index(linear)
    _, fin, fout = cfg["linears"][idx]
    t = cfg["tokens"]
    base = cfg["data_seed"]
    dy = matrix((t, fout), [base, idx, 0], **cfg["dy"])
    x = matrix((t, fin), [base, idx, 1], **cfg["x"])
    w = matrix((fout, fin), [base, idx, 2], **cfg["w"])
    return dy, x, w


def gemm_flops(config):
    """Algorithmic FLOPs of the two backward GEMMs of every linear: 4 * T * in * out each."""
    cfg = CONFIGS[config]
    return sum(4 * cfg["tokens"] * fin * fout for _, fin, fout in cfg["linears"])
