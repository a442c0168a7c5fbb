"""Plain CPU oracle of bounded state staging (DynaResize, Training->Rollout role switch).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import, call or run anything in this
package.  The product path (the HIP library and its Python binding) never
imports it, and it never imports the product path: the two share no code, no
tables and no constants.  Inputs are handed in as numpy arrays by the caller.

What it computes.  During a role switch the paper moves a GPU's training state
(weights and optimizer moments, sharded as FSDP/Megatron keep them) into the
layout the new role consumes, through bounded host-memory chunks (Sec. 3.3,
"Staged State Reloading"), with the optimizer reload deferred (Sec. 3.3, last
paragraph) and the rollout role fed by weight synchronization (Sec. 3.2).  The
paper does not spell out the layouts, the cast or the chunk record; this module
writes out the fixed convention used for them:

* O1  training layout: tensors in model order, row-major [out, in] fp32, packed
      densely, zero-padded at the tail to a multiple of W*256, cut into W equal
      contiguous shards;
* O2  fp32 -> bf16 by IEEE 754 roundTiesToEven on the bit pattern (no flush of
      subnormals, overflow to infinity), NaN kept NaN with sign and the top
      payload bits, quiet bit set;
* O3  rollout layout of TP rank r: embed/lm_head vocab rows r*V/T.., q/k/v rows
      of that rank's heads fused as [q; k; v], gate/up rows fused as [gate; up],
      o and down column-sliced, norms replicated; ranks packed one after
      another (rank-major);
* O4  chunks: the rollout byte stream cut every B bytes;
* O5  per-chunk checksum (s1, s2) over little-endian u32 words, mod 2^64;
* O6  moment stream m_0 .. m_{W-1} v_0 .. v_{W-1} (padding included).

Parity pins: every function here is checked in ``tests/test_oracle_*.py``
against closed forms, a library cast, exact rational rounding, conservation
counts, a tagged brute-force index formula and the round-trip inverse.  The
conventions themselves (tensor order, fused-row order, rank-major packing, NaN
payload rule, the checksum function) are not fixed by the paper: for them the
parity is "unpinned by the paper" and pinned only by this convention.
"""
from __future__ import annotations

from collections import namedtuple

import numpy as np

Model = namedtuple("Model", "n_layers hidden n_q_heads n_kv_heads head_dim ffn vocab")

_LAYER_NAMES = ("ln1", "q", "k", "v", "o", "ln2", "gate", "up", "down")


# --------------------------------------------------------------------------- O1
def training_tensors(m: Model) -> list[tuple[str, tuple[int, ...]]]:
    """O1: (name, shape) of every training tensor, in packing order.

    Shapes are [out, in] for matrices (row-major) and [hidden] for norms.
    """
    H = m.hidden
    qd = m.n_q_heads * m.head_dim
    kd = m.n_kv_heads * m.head_dim
    per_layer = {
        "ln1": (H,),
        "q": (qd, H),
        "k": (kd, H),
        "v": (kd, H),
        "o": (H, qd),
        "ln2": (H,),
        "gate": (m.ffn, H),
        "up": (m.ffn, H),
        "down": (H, m.ffn),
    }
    out = [("embed", (m.vocab, H))]
    for layer in range(m.n_layers):
        for name in _LAYER_NAMES:
            out.append((f"layers.{layer}.{name}", per_layer[name]))
    out.append(("final_norm", (H,)))
    out.append(("lm_head", (m.vocab, H)))
    return out


def training_offsets(m: Model) -> tuple[dict[str, tuple[int, tuple[int, ...]]], int]:
    """O1: element offset and shape of each training tensor, and N (unpadded count)."""
    table = {}
    off = 0
    for name, shape in training_tensors(m):
        table[name] = (off, shape)
        off += int(np.prod(shape))
    return table, off


def padded_elems(n: int, w: int) -> int:
    """O1: the flat buffer is zero-padded at its tail to a multiple of W*256 elements."""
    unit = w * 256
    return -(-n // unit) * unit


def training_views(flat: np.ndarray, m: Model) -> dict[str, np.ndarray]:
    """O1: name -> view of the flat buffer with that tensor's shape (no copy)."""
    table, n = training_offsets(m)
    assert flat.ndim == 1 and flat.size >= n
    return {name: flat[off:off + int(np.prod(shape))].reshape(shape) for name, (off, shape) in table.items()}


def shards(flat: np.ndarray, w: int) -> list[np.ndarray]:
    """O1: W equal contiguous shards of the padded flat buffer."""
    assert flat.size % w == 0
    s = flat.size // w
    return [flat[i * s:(i + 1) * s] for i in range(w)]


# --------------------------------------------------------------------------- O2
def rne_bf16(bits: np.ndarray) -> np.ndarray:
    """O2: fp32 bit patterns (uint32) -> bf16 bit patterns (uint16).

    IEEE 754 roundTiesToEven from 24 to 8 significand bits, done on the
    encoding: the upper half ``t`` is the value truncated toward zero, the lower
    half ``r`` is the discarded remainder in units of 2^-16 ulp.  The magnitude
    is rounded up (``t + 1``) when ``r`` is more than half an ulp, or exactly
    half and ``t`` is odd.  Because the encoding is monotone in the magnitude,
    ``t + 1`` carries into the exponent when the significand overflows and turns
    the largest finite values into infinity, for either sign.  Subnormals round
    like any other value (nothing is flushed).  A NaN keeps its sign and top
    payload bits and gets the quiet bit (bit 6 of the bf16 significand).
    """
    u = np.asarray(bits, dtype=np.uint32)
    t = u >> np.uint32(16)
    r = u & np.uint32(0xFFFF)
    half = np.uint32(0x8000)
    odd = (t & np.uint32(1)) == 1
    round_up = (r > half) | ((r == half) & odd)
    out = t + round_up.astype(np.uint32)
    is_nan = (u & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
    out = np.where(is_nan, t | np.uint32(0x0040), out)
    return out.astype(np.uint16)


def widen_bf16(bits16: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> the fp32 bit patterns of the same values (exact)."""
    return np.asarray(bits16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)


# --------------------------------------------------------------------------- O3
def _per_rank(m: Model, t: int) -> tuple[int, int, int, int]:
    assert m.n_q_heads % t == 0 and m.n_kv_heads % t == 0 and m.ffn % t == 0 and m.vocab % t == 0
    return m.n_q_heads // t, m.n_kv_heads // t, m.ffn // t, m.vocab // t


def rollout_tensors(m: Model, t: int) -> list[tuple[str, tuple[int, ...]]]:
    """O3: (name, shape) of one TP rank's rollout tensors, in packing order."""
    qh, kh, fr, vr = _per_rank(m, t)
    H, D = m.hidden, m.head_dim
    out = [("embed", (vr, H))]
    for layer in range(m.n_layers):
        out += [
            (f"layers.{layer}.ln1", (H,)),
            (f"layers.{layer}.qkv", ((qh + 2 * kh) * D, H)),
            (f"layers.{layer}.o", (H, qh * D)),
            (f"layers.{layer}.ln2", (H,)),
            (f"layers.{layer}.gate_up", (2 * fr, H)),
            (f"layers.{layer}.down", (H, fr)),
        ]
    out += [("final_norm", (H,)), ("lm_head", (vr, H))]
    return out


def rollout_table(m: Model, t: int) -> list[tuple[int, str, int, tuple[int, ...]]]:
    """O3: (rank, name, element offset in the rank-major stream, shape) for every rollout tensor."""
    table = []
    off = 0
    for r in range(t):
        for name, shape in rollout_tensors(m, t):
            table.append((r, name, off, shape))
            off += int(np.prod(shape))
    return table


def rollout_tensor(src: dict[str, np.ndarray], m: Model, t: int, r: int, name: str) -> np.ndarray:
    """O3: one rollout tensor of TP rank ``r`` (name as in ``rollout_tensors``) as bf16 bits (uint16).

    ``src`` maps training tensor names to their fp32 bit patterns (uint32,
    training shape), e.g. ``training_views(flat, m)``; only the tensors this
    output reads are looked up.  Head h of rank r is global head r*qh+h (kv:
    r*kh+h); rank r owns vocab rows [r*V/T, (r+1)*V/T) and FFN units
    [r*F/T, (r+1)*F/T).
    """
    qh, kh, fr, vr = _per_rank(m, t)
    D = m.head_dim
    q_rows = slice(r * qh * D, (r + 1) * qh * D)
    kv_rows = slice(r * kh * D, (r + 1) * kh * D)
    f_rows = slice(r * fr, (r + 1) * fr)
    v_rows = slice(r * vr, (r + 1) * vr)
    base = name.split(".")[-1]
    p = name[: -len(base)]
    if base in ("embed", "lm_head"):
        return rne_bf16(src[name][v_rows, :])
    if base in ("ln1", "ln2", "final_norm"):
        return rne_bf16(src[name])
    if base == "qkv":
        return rne_bf16(np.concatenate([src[p + "q"][q_rows, :], src[p + "k"][kv_rows, :], src[p + "v"][kv_rows, :]],
                                       axis=0))
    if base == "o":
        return rne_bf16(src[p + "o"][:, q_rows])
    if base == "gate_up":
        return rne_bf16(np.concatenate([src[p + "gate"][f_rows, :], src[p + "up"][f_rows, :]], axis=0))
    if base == "down":
        return rne_bf16(src[p + "down"][:, f_rows])
    raise KeyError(name)


def rollout_rank(src: dict[str, np.ndarray], m: Model, t: int, r: int) -> list[tuple[str, np.ndarray]]:
    """O3: every rollout tensor of TP rank ``r``, in packing order, as (name, bf16 bits)."""
    return [(name, rollout_tensor(src, m, t, r, name)) for name, _ in rollout_tensors(m, t)]


def rollout_stream(src: dict[str, np.ndarray], m: Model, t: int) -> np.ndarray:
    """O3: the whole rollout byte stream R_0 || ... || R_{T-1}, as uint16 (bf16 bits)."""
    parts = []
    for r in range(t):
        parts += [a.ravel() for _, a in rollout_rank(src, m, t, r)]
    return np.concatenate(parts)


def split_stream(stream: np.ndarray, m: Model, t: int) -> list[dict[str, np.ndarray]]:
    """Cut a rank-major rollout stream (uint16) back into per-rank named tensors."""
    ranks: list[dict[str, np.ndarray]] = [dict() for _ in range(t)]
    for r, name, off, shape in rollout_table(m, t):
        ranks[r][name] = stream[off:off + int(np.prod(shape))].reshape(shape)
    return ranks


def inverse(ranks: list[dict[str, np.ndarray]], m: Model, t: int) -> dict[str, np.ndarray]:
    """Inverse of O3: rebuild every training tensor (bf16 bits) from the T ranks.

    Row slices are stacked back along rows, column slices along columns; the
    fused tensors are cut at the q/k/v and gate/up row boundaries.  Replicated
    norms must be identical on every rank (asserted).
    """
    qh, kh, fr, _ = _per_rank(m, t)
    D = m.head_dim
    out = {}

    def same_on_all(name):
        first = ranks[0][name]
        for r in range(1, t):
            assert np.array_equal(ranks[r][name], first), name
        return first

    out["embed"] = np.concatenate([ranks[r]["embed"] for r in range(t)], axis=0)
    for layer in range(m.n_layers):
        p = f"layers.{layer}."
        qkv = [ranks[r][p + "qkv"] for r in range(t)]
        out[p + "ln1"] = same_on_all(p + "ln1")
        out[p + "q"] = np.concatenate([x[: qh * D] for x in qkv], axis=0)
        out[p + "k"] = np.concatenate([x[qh * D:(qh + kh) * D] for x in qkv], axis=0)
        out[p + "v"] = np.concatenate([x[(qh + kh) * D:] for x in qkv], axis=0)
        out[p + "o"] = np.concatenate([ranks[r][p + "o"] for r in range(t)], axis=1)
        out[p + "ln2"] = same_on_all(p + "ln2")
        gu = [ranks[r][p + "gate_up"] for r in range(t)]
        out[p + "gate"] = np.concatenate([x[:fr] for x in gu], axis=0)
        out[p + "up"] = np.concatenate([x[fr:] for x in gu], axis=0)
        out[p + "down"] = np.concatenate([ranks[r][p + "down"] for r in range(t)], axis=1)
    out["final_norm"] = same_on_all("final_norm")
    out["lm_head"] = np.concatenate([ranks[r]["lm_head"] for r in range(t)], axis=0)
    return out


# --------------------------------------------------------------------------- O4
def chunk_spans(total_bytes: int, budget: int) -> list[tuple[int, int]]:
    """O4: byte ranges [c*B, min((c+1)*B, total)) of every chunk of a stream."""
    return [(c, min(c + budget, total_bytes)) for c in range(0, total_bytes, budget)]


# --------------------------------------------------------------------------- O5
def checksum(chunk: np.ndarray) -> tuple[int, int]:
    """O5: (s1, s2) of one chunk, both mod 2^64.

    w_j is the little-endian u32 at bytes [4j, 4j+4) of the chunk;
    s1 = sum_j w_j and s2 = sum_j (j+1) w_j.  numpy uint64 arithmetic wraps
    modulo 2^64, which is exactly the reduction the definition asks for.
    """
    raw = np.ascontiguousarray(chunk).view(np.uint8).ravel()
    assert raw.size % 4 == 0
    w = raw.view("<u4").astype(np.uint64)
    j1 = np.arange(1, w.size + 1, dtype=np.uint64)
    s1 = int(w.sum(dtype=np.uint64))
    s2 = int((j1 * w).sum(dtype=np.uint64))
    return s1, s2


def chunk_checksums(stream: np.ndarray, budget: int) -> list[tuple[int, int]]:
    """O4 + O5: checksum of every chunk of a stream (uint16 / uint8 / any dtype)."""
    raw = np.ascontiguousarray(stream).view(np.uint8).ravel()
    return [checksum(raw[a:b]) for a, b in chunk_spans(raw.size, budget)]


# --------------------------------------------------------------------------- reshard
def reshard(flat: np.ndarray, n: int, w2: int) -> np.ndarray:
    """Training -> training move to W' shards: the same N training elements, bit for bit,
    followed by the padding of a W'-shard layout (+0.0 up to a multiple of W'*256).

    ``flat`` is the source flat buffer (any padding); the result is the destination flat
    buffer, whose W' equal contiguous pieces are the new shards (``shards(result, w2)``).
    Its bytes, cut every B bytes, are the chunks; each chunk's checksum is O5 over them.
    """
    out = np.zeros(padded_elems(n, w2), dtype=flat.dtype)
    out[:n] = flat[:n]
    return out


# --------------------------------------------------------------------------- O6
def moment_stream(m_shards: list[np.ndarray], v_shards: list[np.ndarray]) -> np.ndarray:
    """O6: bytes of m_0 || ... || m_{W-1} || v_0 || ... || v_{W-1} (padding included)."""
    parts = [np.ascontiguousarray(a).view(np.uint8).ravel() for a in list(m_shards) + list(v_shards)]
    return np.concatenate(parts)
