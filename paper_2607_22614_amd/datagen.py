"""Seeded synthetic training state for the staging workloads.

Input generation only: it writes fp32 weights, norms and Adam moments in the
flat training layout (model-order tensors, row-major, zero tail padding to a
multiple of W*256) and holds no part of the staging arithmetic (no cast, no
rollout layout, no chunking, no checksum).  Both the HIP path and the CPU
oracle consume what it produces.

Value recipe: weights N(0, 0.02); norms 1 + N(0, 0.01); optionally a fraction
of positions replaced by values that stress a bf16 cast (exact rounding ties,
fp32 subnormals, +-Inf, quiet NaN, +-0).  Adam moments m ~ N(0, 1e-3) and
v = |N(0, 1)| * 1e-6 over the whole padded buffer.

Host generation uses numpy PCG64 with one stream per tensor spawned from
``SeedSequence(seed)``; device generation (the 8B/32B shapes) uses torch's
device generator seeded per tensor, so it depends on the torch/ROCm build.
"""
from __future__ import annotations

import numpy as np

_LAYER = (("ln1", "norm"), ("q", "w"), ("k", "w"), ("v", "w"), ("o", "w"),
          ("ln2", "norm"), ("gate", "w"), ("up", "w"), ("down", "w"))


def tensor_list(model) -> list[tuple[str, int, str]]:
    """(name, numel, kind) of each training tensor in flat-layout order; kind is 'w' or 'norm'."""
    L, H, Hq, Hkv, D, F, V = model
    sizes = {"ln1": H, "q": Hq * D * H, "k": Hkv * D * H, "v": Hkv * D * H, "o": H * Hq * D,
             "ln2": H, "gate": F * H, "up": F * H, "down": H * F}
    out = [("embed", V * H, "w")]
    for layer in range(L):
        out += [(f"layers.{layer}.{n}", sizes[n], kind) for n, kind in _LAYER]
    out += [("final_norm", H, "norm"), ("lm_head", V * H, "w")]
    return out


def flat_sizes(model, w: int) -> tuple[int, int]:
    """(N, Npad): element count and the count padded to a multiple of W*256."""
    n = sum(numel for _, numel, _ in tensor_list(model))
    unit = 256 * w
    return n, -(-n // unit) * unit


# ----------------------------------------------------------------------------- host (numpy)
def special_values(rng: np.random.Generator, k: int) -> np.ndarray:
    """k fp32 bit patterns drawn uniformly from seven cast-stressing categories.

    0: rounding ties (low 16 bits 0x8000, random sign/exponent 1..254/top mantissa bits)
    1: subnormals (exponent 0, nonzero mantissa; half of them ties)
    2: +Inf   3: -Inf   4: quiet NaN 0x7FC00000   5: +0   6: -0
    """
    cat = rng.integers(0, 7, size=k)
    sign = rng.integers(0, 2, size=k, dtype=np.uint32) << np.uint32(31)
    exp = rng.integers(1, 255, size=k, dtype=np.uint32) << np.uint32(23)
    top7 = rng.integers(0, 128, size=k, dtype=np.uint32) << np.uint32(16)
    tie = sign | exp | top7 | np.uint32(0x8000)
    sub_rand = rng.integers(1, 1 << 23, size=k, dtype=np.uint32)
    sub_tie = top7 | np.uint32(0x8000)
    sub = sign | np.where(rng.integers(0, 2, size=k) == 1, sub_tie, sub_rand).astype(np.uint32)
    fixed = np.array([0, 0, 0x7F800000, 0xFF800000, 0x7FC00000, 0x00000000, 0x80000000], dtype=np.uint32)
    out = fixed[cat]
    out = np.where(cat == 0, tie, out)
    out = np.where(cat == 1, sub, out)
    return out.astype(np.uint32)


def make_flat_numpy(model, w: int, seed: int, specials_frac: float = 0.0) -> np.ndarray:
    """Padded flat fp32 training buffer (float32 array of Npad elements) on the host."""
    tensors = tensor_list(model)
    n, npad = flat_sizes(model, w)
    flat = np.zeros(npad, dtype=np.float32)
    children = np.random.SeedSequence(seed).spawn(len(tensors) + 1)
    off = 0
    for (name, numel, kind), child in zip(tensors, children):
        rng = np.random.Generator(np.random.PCG64(child))
        x = rng.standard_normal(numel, dtype=np.float32)
        if kind == "norm":
            flat[off:off + numel] = np.float32(1.0) + np.float32(0.01) * x
        else:
            flat[off:off + numel] = np.float32(0.02) * x
        off += numel
    if specials_frac > 0:
        rng = np.random.Generator(np.random.PCG64(children[-1]))
        k = int(round(specials_frac * n))
        pos = _distinct_positions(rng, n, k)
        flat.view(np.uint32)[pos] = special_values(rng, k)
    return flat


def make_tensors_numpy(model, seed: int, names, workers: int = 1) -> dict[str, np.ndarray]:
    """Named training tensors (flat float32 arrays), each equal to its slice of
    make_flat_numpy(model, w, seed) without specials: the same per-tensor streams, generated
    only for the tensors asked for, on up to `workers` host threads."""
    tensors = tensor_list(model)
    index = {name: i for i, (name, _, _) in enumerate(tensors)}
    children = np.random.SeedSequence(seed).spawn(len(tensors) + 1)

    def one(name):
        i = index[name]
        _, numel, kind = tensors[i]
        x = np.random.Generator(np.random.PCG64(children[i])).standard_normal(numel, dtype=np.float32)
        if kind == "norm":
            x *= np.float32(0.01)
            x += np.float32(1.0)
        else:
            x *= np.float32(0.02)
        return name, x

    names = list(dict.fromkeys(names))
    if workers <= 1:
        return dict(one(n) for n in names)
    from concurrent.futures import ThreadPoolExecutor
    with ThreadPoolExecutor(workers) as ex:
        return dict(ex.map(one, names))


def _distinct_positions(rng: np.random.Generator, n: int, k: int) -> np.ndarray:
    """k distinct positions in [0, n), uniform without replacement (sequential draws, repeats dropped)."""
    picked = np.empty(0, dtype=np.int64)
    while picked.size < k:
        draw = rng.integers(0, n, size=int((k - picked.size) * 1.25) + 16)
        cand = np.concatenate([picked, draw])
        _, first = np.unique(cand, return_index=True)
        picked = cand[np.sort(first)]
    return picked[:k]


def make_moments_numpy(npad: int, seed: int) -> tuple[np.ndarray, np.ndarray]:
    """Adam moments (m, v) as padded flat fp32 buffers on the host."""
    a, b = np.random.SeedSequence(seed).spawn(2)
    m = np.random.Generator(np.random.PCG64(a)).standard_normal(npad, dtype=np.float32) * np.float32(1e-3)
    v = np.abs(np.random.Generator(np.random.PCG64(b)).standard_normal(npad, dtype=np.float32)) * np.float32(1e-6)
    return m, v


def tagged_flat(model, w: int) -> np.ndarray:
    """Padded flat buffer whose element e holds the bf16-exact pattern (e+1) << 16 (e < 32639).

    Every weight is unique, so a staged output word names the element it came from.
    """
    n, npad = flat_sizes(model, w)
    assert n < 0x7F7F, "tagging needs fewer than 32639 elements"
    bits = np.zeros(npad, dtype=np.uint32)
    bits[:n] = (np.arange(n, dtype=np.uint32) + np.uint32(1)) << np.uint32(16)
    return bits.view(np.float32)


# ----------------------------------------------------------------------------- device (torch)
def make_flat_torch(model, w: int, seed: int, device="cuda"):
    """Padded flat fp32 training buffer generated on the device, one generator seed per tensor."""
    import torch

    tensors = tensor_list(model)
    n, npad = flat_sizes(model, w)
    flat = torch.empty(npad, dtype=torch.float32, device=device)
    flat[n:].zero_()
    g = torch.Generator(device=device)
    off = 0
    for idx, (_, numel, kind) in enumerate(tensors):
        g.manual_seed(seed * 1_000_003 + idx)
        view = flat[off:off + numel]
        if kind == "norm":
            view.normal_(1.0, 0.01, generator=g)
        else:
            view.normal_(0.0, 0.02, generator=g)
        off += numel
    return flat


def make_moments_torch(npad: int, seed: int, device="cuda"):
    """Adam moments (m, v) as padded flat fp32 buffers generated on the device."""
    import torch

    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + 999_001)
    m = torch.empty(npad, dtype=torch.float32, device=device).normal_(0.0, 1e-3, generator=g)
    g.manual_seed(seed * 1_000_003 + 999_002)
    v = torch.empty(npad, dtype=torch.float32, device=device).normal_(0.0, 1.0, generator=g)
    v.abs_().mul_(1e-6)
    return m, v


# ----------------------------------------------------------------------------- stage-time traces
def stage_time_trace(seed: int, steps: int, enter: float = 0.2, noise: float = 0.05,
                     shift_at: int | None = None, shift_to: float = 0.5) -> list[tuple[float, float]]:
    """Open-loop (rollout time, training time) pairs: training ~10 s, rollout around it with
    multiplicative noise, optionally shifted to a sustained imbalance from step `shift_at`
    (rollout = training * (1 + shift_to) / (1 - shift_to) on average, i.e. r ~ shift_to)."""
    rng = np.random.default_rng(seed)
    out = []
    for k in range(steps):
        tt = 10.0 * float(np.exp(rng.normal(0.0, noise)))
        base = (1 + shift_to) / (1 - shift_to) if (shift_at is not None and k >= shift_at) else 1.0
        tr = 10.0 * base * float(np.exp(rng.normal(0.0, noise)))
        out.append((tr, tt))
    return out


def rollout_work_trace(seed: int, steps: int, shift_at: int, heavy: float = 2.5) -> np.ndarray:
    """Rollout work per step (GPU-seconds) with long-tail noise (lognormal) and a shift to a
    heavier, reasoning-style prompt mix from step `shift_at`."""
    rng = np.random.default_rng(seed)
    base = np.where(np.arange(steps) >= shift_at, heavy, 1.0) * 40.0
    return base * np.exp(rng.normal(0.0, 0.15, size=steps))
