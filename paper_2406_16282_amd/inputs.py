"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module draws numbers and lays them out in storage formats; it holds none of
the method's arithmetic. Both the HIP path and the CPU oracle receive the exact
bytes produced here.

Recipe: ``numpy.random.Generator(PCG64(SeedSequence([seed, block, tensor_id])))``,
``standard_normal`` in float64, scaled, rounded to fp32 (round to nearest even),
then for bf16 rounded again from the fp32 bits to 16 bits (round to nearest even).
tensor_id: 0 = norm input x, 1 = norm upstream gradient dz, 2 = activation input
x (the gate g of a SwiGLU product), 3 = activation upstream gradient dy (dh),
4 = the SwiGLU "up" input u, drawn N(0, 1).

The workloads mirror the activation shapes of the paper's fine-tuning runs
(ViT-B/16 at 224 px: 197 tokens, width 768, MLP 3072; LLaMA-7B: width 4096,
FFN 11008; LLaMA-13B: 5120 / 13824). No dataset or pretrained weight is used:
i.i.d. draws stand in for the activations those models would produce.
"""

from dataclasses import dataclass, field

import numpy as np

SEED = 0
NORM_X, NORM_DZ, ACT_X, ACT_DY, ACT_U = 0, 1, 2, 3, 4
LIN_X, LIN_W, LIN_B = 5, 6, 7


def rng(seed, block, tensor_id):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, block, tensor_id])))


def f32_to_bf16_bits(a32):
    """Round float32 values to bf16 (nearest, ties to even); returns uint16 patterns.

    Inputs are finite, so the NaN case of the usual bit trick does not arise.
    """
    u = np.ascontiguousarray(a32, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def to_storage(a64, dtype):
    """float64 draws -> fp32 array or bf16 uint16 patterns."""
    a32 = np.asarray(a64, dtype=np.float64).astype(np.float32)
    if dtype == "fp32":
        return a32
    if dtype == "bf16":
        return f32_to_bf16_bits(a32)
    raise ValueError(f"unknown dtype {dtype!r}")


def normal(shape, std, dtype, seed=SEED, block=0, tensor_id=0, mean=0.0):
    g = rng(seed, block, tensor_id)
    return to_storage(mean + std * g.standard_normal(size=shape), dtype)


def dyadic(shape, exponent, seed=SEED, block=0, tensor_id=0, span=8):
    """Integers in [-span, span] times 2^exponent, as bf16 patterns. Products and sums
    of such values stay exactly representable in fp32 for moderate sizes, so any
    summation order gives the exact result."""
    g = rng(seed, block, tensor_id)
    v = g.integers(-span, span + 1, size=shape).astype(np.float64) * 2.0 ** exponent
    return to_storage(v, "bf16")


def outlier_mixture(shape, dtype, seed=SEED, block=0, tensor_id=0,
                    p_outlier=0.01, std_in=1.0, std_out=30.0):
    """Per element: N(0, std_out^2) with probability p_outlier, else N(0, std_in^2)."""
    g = rng(seed, block, tensor_id)
    base = g.standard_normal(size=shape)
    mask = g.random(size=shape) < p_outlier
    return to_storage(np.where(mask, std_out, std_in) * base, dtype)


# ---------------------------------------------------------------- edge cases

def _neighbours(value, dtype, radius=3):
    """The storage values nearest ``value``: its rounding and +-radius steps of the
    bit pattern (a bit-pattern step is one ulp for finite same-sign values)."""
    if dtype == "fp32":
        b = int(np.array([value], dtype=np.float32).view(np.uint32)[0])
        pats = np.array([b + k for k in range(-radius, radius + 1)], dtype=np.uint32)
        return pats.view(np.float32).astype(np.float64)
    b = int(f32_to_bf16_bits(np.array([value], dtype=np.float32))[0])
    pats = np.array([b + k for k in range(-radius, radius + 1)], dtype=np.uint32) << np.uint32(16)
    return pats.view(np.float32).astype(np.float64)


def edge_activation(shape, dtype, thresholds, seed=SEED, tensor_id=ACT_X):
    """Stress input for a ReLU-combination activation.

    40% of the elements are the storage neighbours (down to 3 ulps on either side)
    of the given thresholds, 10% are extremes (+-1e4 rounded to the format,
    log-uniform magnitudes in [10, 1e4], signed zeros, fp32 subnormals), the rest
    N(0, 1); the order is shuffled. ``thresholds`` are plain numbers supplied by the
    caller; nothing about how they are used lives here.
    """
    g = rng(seed, 99, tensor_id)
    n = int(np.prod(shape))
    near = np.concatenate([_neighbours(t, dtype) for t in thresholds])
    n_near = int(0.4 * n)
    n_ext = int(0.1 * n)
    vals = np.empty(n, dtype=np.float64)
    vals[:n_near] = g.choice(near, size=n_near)
    k = n_near
    special = np.array([1e4, -1e4, 0.0, -0.0, 1e-40, -1e-40, 1.4e-45, -1.4e-45, 1e-39])
    n_special = min(n_ext // 2, 4 * special.size)
    vals[k:k + n_special] = np.resize(special, n_special)
    k += n_special
    n_log = n_ext - n_special
    mags = 10.0 ** g.uniform(1.0, 4.0, size=n_log)
    vals[k:k + n_log] = mags * g.choice([-1.0, 1.0], size=n_log)
    k += n_log
    vals[k:] = g.standard_normal(size=n - k)
    g.shuffle(vals)
    return to_storage(vals.reshape(shape), dtype)


def edge_norm_rows(shape, dtype, seed=SEED, tensor_id=NORM_X):
    """Rows of N(0,1) with special rows interleaved: constant, all zero, mean 1e4 plus
    N(0,1), a single +-1e4 spike, all +-1e4 with random signs."""
    rows, p = shape
    g = rng(seed, 98, tensor_id)
    x = g.standard_normal(size=shape)
    kinds = 6
    for r in range(rows):
        kind = r % (2 * kinds)
        if kind == 1:
            x[r] = 3.0
        elif kind == 3:
            x[r] = 0.0
        elif kind == 5:
            x[r] = 1e4 + g.standard_normal(size=p)
        elif kind == 7:
            x[r, g.integers(p)] = 1e4 * g.choice([-1.0, 1.0])
        elif kind == 9:
            x[r] = 1e4 * g.choice([-1.0, 1.0], size=p)
    return to_storage(x, dtype)


# ---------------------------------------------------------------- large tensors

HASH_MUL = 2654435761  # Knuth's multiplicative hash constant


def hash_values(index, scale=8.0, salt=0):
    """Closed-form pseudo-random values for flat element indices (an integer hash of
    index + salt mapped to [-scale, scale)), as float64. Used for tensors too large to
    draw on the host: the device computes the same formula for every element, the host
    only for the sampled indices it checks. Different salts give unrelated tensors."""
    i = np.asarray(index, dtype=np.int64) + np.int64(salt)
    hsh = (i * HASH_MUL) & 0xFFFFFFFF
    return ((hsh >> 8).astype(np.float64) / float(1 << 24) * 2.0 - 1.0) * scale


def hash_tensor(n, dtype, device, scale=8.0, salt=0, chunk=1 << 27):
    """The values of ``hash_values(range(n), scale, salt)`` rounded to ``dtype``, built on
    ``device`` with torch integer arithmetic in chunks (no host copy of the tensor)."""
    import torch
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    out = torch.empty(n, dtype=tdt, device=device)
    for s in range(0, n, chunk):
        e = min(n, s + chunk)
        i = torch.arange(s + salt, e + salt, dtype=torch.int64, device=device)
        hsh = (i * HASH_MUL) & 0xFFFFFFFF
        v = ((hsh >> 8).to(torch.float64) / float(1 << 24) * 2.0 - 1.0) * scale
        out[s:e] = v.to(torch.float32).to(tdt)
    return out


def hash_storage(index, dtype, scale=8.0, salt=0):
    """Host storage values (fp32 array or bf16 patterns) of ``hash_tensor`` at ``index``:
    the same float64 -> fp32 -> dtype rounding chain."""
    return to_storage(hash_values(index, scale, salt), dtype)


# ---------------------------------------------------------------- workloads

@dataclass(frozen=True)
class NormSpec:
    op: str            # "msln" or "msrms"
    rows: int
    cols: int
    dtype: str
    eps: float
    x_std: float
    dz_std: float
    mixture: bool = False


@dataclass(frozen=True)
class ActSpec:
    op: str            # "regelu2" or "resilu2"
    rows: int
    cols: int
    dtype: str
    x_std: float
    dy_std: float
    mixture: bool = False


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    norm: NormSpec
    act: ActSpec
    blocks: int = 1
    timed: bool = True
    extra: dict = field(default_factory=dict)

    def norm_x(self, block=0, seed=SEED):
        s = self.norm
        if s.mixture:
            return outlier_mixture((s.rows, s.cols), s.dtype, seed, block, NORM_X)
        return normal((s.rows, s.cols), s.x_std, s.dtype, seed, block, NORM_X)

    def norm_dz(self, block=0, seed=SEED):
        s = self.norm
        return normal((s.rows, s.cols), s.dz_std, s.dtype, seed, block, NORM_DZ)

    def act_x(self, block=0, seed=SEED):
        s = self.act
        if s.mixture:
            return outlier_mixture((s.rows, s.cols), s.dtype, seed, block, ACT_X)
        return normal((s.rows, s.cols), s.x_std, s.dtype, seed, block, ACT_X)

    def act_dy(self, block=0, seed=SEED):
        s = self.act
        return normal((s.rows, s.cols), s.dy_std, s.dtype, seed, block, ACT_DY)

    def act_u(self, block=0, seed=SEED):
        """The "up" projection u of a SwiGLU product h = SiLU(g) * u (same shape as g)."""
        s = self.act
        return normal((s.rows, s.cols), 1.0, s.dtype, seed, block, ACT_U)


WORKLOADS = {
    "vit_b_fp32": Workload(
        "vit_b_fp32",
        "ViT-B block nonlinearities, fp32: MS-LN on [8*197, 768], ReGELU2 on [8*197, 3072]",
        NormSpec("msln", 8 * 197, 768, "fp32", 1e-6, 1.0, 1.0),
        ActSpec("regelu2", 8 * 197, 3072, "fp32", 1.0, 1.0)),
    "vit_b_bs64_bf16_x12": Workload(
        "vit_b_bs64_bf16_x12",
        "ViT-B fine-tuning batch 64, bf16: MS-LN on [64*197, 768], ReGELU2 on [64*197, 3072], 12 blocks",
        NormSpec("msln", 64 * 197, 768, "bf16", 1e-6, 1.5, 1e-2),
        ActSpec("regelu2", 64 * 197, 3072, "bf16", 1.5, 1e-2),
        blocks=12),
    "llama7b_swiglu_bf16": Workload(
        "llama7b_swiglu_bf16",
        "LLaMA-7B-shaped, bf16: MS-RMSNorm on [4*2048, 4096], ReSiLU2 on the gate [4*2048, 11008]",
        NormSpec("msrms", 4 * 2048, 4096, "bf16", 1e-5, 1.0, 1e-3),
        ActSpec("resilu2", 4 * 2048, 11008, "bf16", 2.0, 1e-3)),
    "llama13b_outliers_bf16": Workload(
        "llama13b_outliers_bf16",
        "LLaMA-13B-shaped, bf16, 1% N(0,30^2) outliers: MS-RMSNorm on [2*4096, 5120], ReSiLU2 on [2*4096, 13824]",
        NormSpec("msrms", 2 * 4096, 5120, "bf16", 1e-5, 1.0, 1e-3, mixture=True),
        ActSpec("resilu2", 2 * 4096, 13824, "bf16", 1.0, 1e-3, mixture=True)),
}

# Edge shapes: widths that are not multiples of 64 (rows chosen so each tensor holds
# about 2.5e6 elements; element counts are not multiples of 16).
EDGE_SHAPES = ((2501, 1000), (2445, 1023), (2439, 1025), (305, 8191))
EDGE_EPS = {"msln": 1e-6, "msrms": 1e-5}


def storage_to_torch(arr, device):
    """Host storage array -> torch tensor on ``device`` with the same bytes."""
    import torch
    a = np.ascontiguousarray(arr)
    if a.dtype == np.float32:
        return torch.from_numpy(a).to(device)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(device)
    if a.dtype == np.uint32:
        return torch.from_numpy(a.view(np.int32)).to(device)
    raise TypeError(f"unsupported storage dtype {a.dtype}")


def torch_to_storage(t):
    """torch tensor (any device) -> host storage array with the same bytes."""
    import torch
    t = t.detach().contiguous().cpu()
    if t.dtype == torch.float32:
        return t.numpy()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype == torch.int32:
        return t.numpy().view(np.uint32)
    raise TypeError(f"unsupported tensor dtype {t.dtype}")
