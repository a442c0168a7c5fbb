"""ctypes binding of libdr.so: the C ABI of include/dr.h with the same names.

Argument marshalling only: every step of staging runs in the HIP library.
Device buffers are passed as torch tensors (or raw integer addresses), streams
as torch streams (default: the current stream).  Importing this module loads
the library and raises ImportError when it has not been built, so nothing can
silently fall back to another implementation.

The C ABI carries pointers without sizes.  For tensor and array arguments the
binding checks, before calling the library, what the library would otherwise
trust: the number of shard pointers equals the plan's, every buffer is dense,
device arguments are device tensors and the host store is host memory, and each
buffer holds the bytes the plan will touch (ValueError otherwise).  Raw integer
addresses are passed through unchecked.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdr.so")
if not os.path.exists(_LIB_PATH):
    raise ImportError(f"{_LIB_PATH} is missing: build it with `python -m paper_2607_22614_amd.build` "
                      "(or __graft_entry__.build())")
_lib = ctypes.CDLL(_LIB_PATH)

DR_OK, DR_EINVAL, DR_ERANGE, DR_ENOMEM, DR_EHIP = 0, -1, -2, -3, -4
DR_MAX_SHARDS = 64
DR_SEG_VEC4 = 1
DR_OP_CAST_BF16, DR_OP_COPY_F32, DR_OP_ZERO_F32 = 0, 1, 2
DR_PLAN_ROLLOUT, DR_PLAN_RESHARD = 0, 1
DR_TILE_DEPTH_AUTO = 0
_CODES = {DR_EINVAL: "DR_EINVAL", DR_ERANGE: "DR_ERANGE", DR_ENOMEM: "DR_ENOMEM", DR_EHIP: "DR_EHIP"}


class dr_model(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("n_layers", "hidden", "n_q_heads", "n_kv_heads", "head_dim", "ffn", "vocab")]


class dr_layout(ctypes.Structure):
    _fields_ = [("train_shards", ctypes.c_int32), ("tp", ctypes.c_int32),
                ("chunk_bytes", ctypes.c_uint64), ("moment_chunk_bytes", ctypes.c_uint64),
                ("tile_depth", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class dr_checksum(ctypes.Structure):
    _fields_ = [("s1", ctypes.c_uint64), ("s2", ctypes.c_uint64)]


class dr_plan_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint64) for n in
                ("n_elems", "padded_elems", "shard_elems", "norm_elems", "rank_elems", "rollout_bytes",
                 "num_chunks", "last_chunk_bytes", "moment_bytes", "num_moment_chunks", "num_segments",
                 "num_tiles", "device_table_bytes", "pinned_bytes")] + \
              [("device", ctypes.c_int32), ("kind", ctypes.c_int32), ("dst_shard_elems", ctypes.c_uint64),
               ("tile_elems", ctypes.c_uint64), ("train_shards", ctypes.c_int32), ("tp", ctypes.c_int32),
               ("dst_shards", ctypes.c_int32), ("reserved", ctypes.c_int32), ("chunk_bytes", ctypes.c_uint64),
               ("moment_chunk_bytes", ctypes.c_uint64), ("deep_tile_elems", ctypes.c_uint64),
               ("deep_num_tiles", ctypes.c_uint64), ("last_tile_depth", ctypes.c_int32),
               ("reserved2", ctypes.c_int32)]


class dr_tensor_desc(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("rank", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("byte_offset", ctypes.c_uint64), ("rows", ctypes.c_int64), ("cols", ctypes.c_int64)]


class dr_segment(ctypes.Structure):
    _fields_ = [("dst_elem", ctypes.c_uint64), ("src_elem", ctypes.c_uint64),
                ("shard", ctypes.c_uint32), ("chunk", ctypes.c_uint32),
                ("rows", ctypes.c_uint32), ("cols", ctypes.c_uint32),
                ("src_row_stride", ctypes.c_uint32), ("flags", ctypes.c_uint32),
                ("dst_shard", ctypes.c_uint32), ("op", ctypes.c_uint32)]


class dr_hyst_params(ctypes.Structure):
    _fields_ = [("num_configs", ctypes.c_int32), ("initial", ctypes.c_int32),
                ("train_gpus", ctypes.POINTER(ctypes.c_int32)), ("rollout_gpus", ctypes.POINTER(ctypes.c_int32)),
                ("enter", ctypes.c_double), ("exit", ctypes.c_double), ("consecutive", ctypes.c_int32),
                ("dwell", ctypes.c_int32), ("cooldown", ctypes.c_int32), ("horizon_steps", ctypes.c_int32),
                ("switch_cost_s", ctypes.c_double)]


class dr_hyst_decision(ctypes.Structure):
    _fields_ = [("config", ctypes.c_int32), ("action", ctypes.c_int32), ("reason", ctypes.c_int32),
                ("run", ctypes.c_int32), ("imbalance", ctypes.c_double), ("predicted_gain_s", ctypes.c_double)]


DR_HYST_BALANCED, DR_HYST_PERSISTENCE, DR_HYST_COOLDOWN, DR_HYST_DWELL, DR_HYST_EDGE, DR_HYST_AMORTIZE, \
    DR_HYST_RESIZE = range(7)

_P = ctypes.c_void_p
_PP = ctypes.POINTER(ctypes.c_void_p)
_SIGS = {
    "dr_plan_create": ([ctypes.POINTER(dr_model), ctypes.POINTER(dr_layout), ctypes.POINTER(_P)], ctypes.c_int),
    "dr_plan_create_host": ([ctypes.POINTER(dr_model), ctypes.POINTER(dr_layout), ctypes.POINTER(_P)], ctypes.c_int),
    "dr_reshard_plan_create": ([ctypes.POINTER(dr_model), ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64,
                                ctypes.POINTER(_P)], ctypes.c_int),
    "dr_reshard_plan_create_host": ([ctypes.POINTER(dr_model), ctypes.c_int32, ctypes.c_int32, ctypes.c_uint64,
                                     ctypes.POINTER(_P)], ctypes.c_int),
    "dr_plan_destroy": ([_P], None),
    "dr_plan_get_info": ([_P, ctypes.POINTER(dr_plan_info)], ctypes.c_int),
    "dr_plan_tensor": ([_P, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(dr_tensor_desc)], ctypes.c_int),
    "dr_plan_segment": ([_P, ctypes.c_uint64, ctypes.POINTER(dr_segment)], ctypes.c_int),
    "dr_stage_chunk": ([_P, ctypes.c_uint64, _PP, _P, _P, _P], ctypes.c_int),
    "dr_stage_chunk_noalloc": ([_P, ctypes.c_uint64, _PP, _P, _P, _P], ctypes.c_int),
    "dr_stage_all": ([_P, _PP, _P, _P, _P], ctypes.c_int),
    "dr_stage_through_host": ([_P, _PP, _P, _P, _P], ctypes.c_int),
    "dr_reshard": ([_P, _PP, _PP, _P, _P], ctypes.c_int),
    "dr_offload_moments": ([_P, _PP, _PP, _P, _P], ctypes.c_int),
    "dr_restore_moments": ([_P, _P, _PP, _PP, _P], ctypes.c_int),
    "dr_reshard_through_host": ([_P, _PP, _PP, _P, _P], ctypes.c_int),
    "dr_offload_moments_range": ([_P, _PP, _PP, _P, ctypes.c_uint64, ctypes.c_uint64, _P], ctypes.c_int),
    "dr_restore_moments_range": ([_P, _P, _PP, _PP, ctypes.c_uint64, ctypes.c_uint64, _P], ctypes.c_int),
    "dr_restore_moments_begin": ([_P, _P, _PP, _PP, _P], ctypes.c_int),
    "dr_restore_moments_end": ([_P], ctypes.c_int),
    "dr_moment_checksums": ([_P, _PP, _PP, _P, _P], ctypes.c_int),
    "dr_hyst_create": ([ctypes.POINTER(dr_hyst_params), ctypes.POINTER(_P)], ctypes.c_int),
    "dr_hyst_step": ([_P, ctypes.c_double, ctypes.c_double, ctypes.POINTER(dr_hyst_decision)], ctypes.c_int),
    "dr_hyst_destroy": ([_P], None),
    "dr_break_even_steps": ([ctypes.c_double, ctypes.c_double, ctypes.c_double], ctypes.c_double),
    "dr_last_error": ([], ctypes.c_char_p),
}
for _name, (_args, _res) in _SIGS.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res

EXPORTED = tuple(_SIGS)


class DrError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        msg = _lib.dr_last_error().decode(errors="replace")
        super().__init__(f"{where}: {_CODES.get(code, code)}: {msg}")


def _check(rc: int, where: str) -> None:
    if rc != DR_OK:
        raise DrError(rc, where)


def _addr(x) -> int:
    """Device/host address of a tensor, numpy array or integer."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    if hasattr(x, "data_ptr"):
        return x.data_ptr()
    if hasattr(x, "ctypes"):
        return x.ctypes.data
    raise TypeError(f"cannot take the address of {type(x)!r}")


def _buf(x, nbytes: int, where: str, device: bool) -> int:
    """Address of a buffer the library will access as `nbytes` dense bytes.

    The C ABI carries no sizes, so a tensor or array argument is checked here: dense
    (contiguous), on the right side (device tensor for device arguments, host memory for the
    host store) and at least nbytes long.  A plain integer address is passed through unchecked.
    """
    if x is None or isinstance(x, int):
        return _addr(x)
    if hasattr(x, "data_ptr"):  # torch tensor
        if not x.is_contiguous():
            raise ValueError(f"{where}: tensor is not contiguous")
        if bool(x.is_cuda) != device:
            raise ValueError(f"{where}: expected a {'device' if device else 'host'} tensor, got one on {x.device}")
        have = x.numel() * x.element_size()
    elif hasattr(x, "ctypes"):  # numpy array: host memory
        if device:
            raise ValueError(f"{where}: a numpy array is host memory; a device buffer is needed")
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError(f"{where}: array is not contiguous")
        have = x.nbytes
    else:
        raise TypeError(f"{where}: cannot take the address of {type(x)!r}")
    if have < nbytes:
        raise ValueError(f"{where}: {have} bytes, the plan needs {nbytes}")
    return _addr(x)


def _ptr_array(xs: Sequence) -> ctypes.Array:
    return (ctypes.c_void_p * len(xs))(*[_addr(x) for x in xs])


def _shards(xs: Sequence, count: int, nbytes: int, where: str) -> ctypes.Array:
    """Host array of `count` device pointers; the library reads exactly `count` of them.
    count None: a call on the wrong kind of plan, passed through for the library to reject."""
    if count is None:
        return _ptr_array(xs)
    if len(xs) != count:
        raise ValueError(f"{where}: {len(xs)} shard buffers given, the plan has {count}")
    return (ctypes.c_void_p * count)(*[_buf(x, nbytes, f"{where}[{i}]", True) for i, x in enumerate(xs)])


def _stream(stream) -> int:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Plan:
    """Owns a dr_plan*; destroyed with the object (after the caller has synchronized)."""

    def __init__(self, handle: int):
        self._h = handle
        # buffers a deferred restore reads and writes from a library thread: held until it ends
        self._restore_refs = None
        info = dr_plan_info()
        _check(_lib.dr_plan_get_info(handle, ctypes.byref(info)), "dr_plan_get_info")
        self.info = {n: getattr(info, n) for n, _ in dr_plan_info._fields_}

    @property
    def handle(self) -> int:
        return self._h

    def close(self) -> None:
        if self._h:
            _lib.dr_plan_destroy(self._h)  # joins a deferred restore still in flight
            self._h = None
        self._restore_refs = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def _model(model) -> dr_model:
    if isinstance(model, dr_model):
        return model
    return dr_model(*[int(v) for v in model])


def _layout(train_shards, tp, chunk_bytes, moment_chunk_bytes=0, tile_depth=DR_TILE_DEPTH_AUTO) -> dr_layout:
    return dr_layout(int(train_shards), int(tp), int(chunk_bytes), int(moment_chunk_bytes), int(tile_depth), 0)


def dr_plan_create(model, train_shards: int, tp: int, chunk_bytes: int, moment_chunk_bytes: int = 0,
                   tile_depth: int = DR_TILE_DEPTH_AUTO) -> Plan:
    """model: (n_layers, hidden, n_q_heads, n_kv_heads, head_dim, ffn, vocab) or dr_model."""
    h = ctypes.c_void_p()
    _check(_lib.dr_plan_create(ctypes.byref(_model(model)),
                               ctypes.byref(_layout(train_shards, tp, chunk_bytes, moment_chunk_bytes, tile_depth)),
                               ctypes.byref(h)), "dr_plan_create")
    return Plan(h.value)


def dr_plan_create_host(model, train_shards: int, tp: int, chunk_bytes: int, moment_chunk_bytes: int = 0,
                        tile_depth: int = DR_TILE_DEPTH_AUTO) -> Plan:
    h = ctypes.c_void_p()
    _check(_lib.dr_plan_create_host(ctypes.byref(_model(model)),
                                    ctypes.byref(_layout(train_shards, tp, chunk_bytes, moment_chunk_bytes,
                                                         tile_depth)),
                                    ctypes.byref(h)), "dr_plan_create_host")
    return Plan(h.value)


def dr_reshard_plan_create(model, from_shards: int, to_shards: int, chunk_bytes: int) -> Plan:
    h = ctypes.c_void_p()
    _check(_lib.dr_reshard_plan_create(ctypes.byref(_model(model)), int(from_shards), int(to_shards),
                                       int(chunk_bytes), ctypes.byref(h)), "dr_reshard_plan_create")
    return Plan(h.value)


def dr_reshard_plan_create_host(model, from_shards: int, to_shards: int, chunk_bytes: int) -> Plan:
    h = ctypes.c_void_p()
    _check(_lib.dr_reshard_plan_create_host(ctypes.byref(_model(model)), int(from_shards), int(to_shards),
                                            int(chunk_bytes), ctypes.byref(h)), "dr_reshard_plan_create_host")
    return Plan(h.value)


def dr_plan_get_info(plan: Plan) -> dict:
    info = dr_plan_info()
    _check(_lib.dr_plan_get_info(plan.handle, ctypes.byref(info)), "dr_plan_get_info")
    return {n: getattr(info, n) for n, _ in dr_plan_info._fields_}


def dr_plan_tensor(plan: Plan, rank: int, index: int) -> dict:
    d = dr_tensor_desc()
    _check(_lib.dr_plan_tensor(plan.handle, rank, index, ctypes.byref(d)), "dr_plan_tensor")
    return {"name": d.name.decode(), "rank": d.rank, "ndim": d.ndim, "byte_offset": d.byte_offset,
            "rows": d.rows, "cols": d.cols}


def dr_plan_segment(plan: Plan, index: int) -> dict:
    s = dr_segment()
    _check(_lib.dr_plan_segment(plan.handle, index, ctypes.byref(s)), "dr_plan_segment")
    return {n: getattr(s, n) for n, _ in dr_segment._fields_}


def _rollout(plan: Plan) -> bool:
    return plan.info["kind"] == DR_PLAN_ROLLOUT


def _chunk_len(i: dict, chunk: int) -> int:
    if 0 <= chunk < i["num_chunks"] - 1:
        return i["chunk_bytes"]
    return i["last_chunk_bytes"] if chunk == i["num_chunks"] - 1 else 0


def dr_stage_chunk(plan: Plan, chunk: int, shards: Sequence, dst_chunk, d_ck, stream=None) -> None:
    """shards: W device tensors/addresses; dst_chunk: device buffer; d_ck: device dr_checksum slot."""
    i = plan.info
    arr = _shards(shards, i["train_shards"] if _rollout(plan) else None, 4 * i["shard_elems"], "dr_stage_chunk shards")
    _check(_lib.dr_stage_chunk(plan.handle, int(chunk), ctypes.cast(arr, _PP),
                               _buf(dst_chunk, _chunk_len(i, int(chunk)), "dr_stage_chunk dst_chunk", True),
                               _buf(d_ck, 16, "dr_stage_chunk d_ck", True), _stream(stream)), "dr_stage_chunk")


def dr_stage_chunk_noalloc(plan: Plan, chunk: int, shards: Sequence, dst_chunk, d_ck, stream=None) -> None:
    """dr_stage_chunk without any device allocation: the checksum accumulators are the library's
    static per-GPU array.  Calls on one GPU must not overlap."""
    i = plan.info
    arr = _shards(shards, i["train_shards"] if _rollout(plan) else None, 4 * i["shard_elems"],
                  "dr_stage_chunk_noalloc shards")
    _check(_lib.dr_stage_chunk_noalloc(plan.handle, int(chunk), ctypes.cast(arr, _PP),
                                       _buf(dst_chunk, _chunk_len(i, int(chunk)), "dr_stage_chunk_noalloc dst_chunk",
                                            True),
                                       _buf(d_ck, 16, "dr_stage_chunk_noalloc d_ck", True), _stream(stream)),
           "dr_stage_chunk_noalloc")


def dr_stage_all(plan: Plan, shards: Sequence, dst, d_cks, stream=None) -> None:
    i = plan.info
    arr = _shards(shards, i["train_shards"] if _rollout(plan) else None, 4 * i["shard_elems"], "dr_stage_all shards")
    _check(_lib.dr_stage_all(plan.handle, ctypes.cast(arr, _PP), _buf(dst, i["rollout_bytes"], "dr_stage_all dst", True),
                             _buf(d_cks, 16 * i["num_chunks"], "dr_stage_all d_cks", True), _stream(stream)),
           "dr_stage_all")


def dr_stage_through_host(plan: Plan, shards: Sequence, dst, d_cks, stream=None) -> None:
    i = plan.info
    arr = _shards(shards, i["train_shards"] if _rollout(plan) else None, 4 * i["shard_elems"], "dr_stage_through_host shards")
    _check(_lib.dr_stage_through_host(plan.handle, ctypes.cast(arr, _PP),
                                      _buf(dst, i["rollout_bytes"], "dr_stage_through_host dst", True),
                                      _buf(d_cks, 16 * i["num_chunks"], "dr_stage_through_host d_cks", True),
                                      _stream(stream)), "dr_stage_through_host")


def dr_reshard(plan: Plan, src_shards: Sequence, dst_shards: Sequence, d_cks, stream=None) -> None:
    i = plan.info
    ok = i["kind"] == DR_PLAN_RESHARD
    a = _shards(src_shards, i["train_shards"] if ok else None, 4 * i["shard_elems"], "dr_reshard src_shards")
    b = _shards(dst_shards, i["dst_shards"] if ok else None, 4 * i["dst_shard_elems"], "dr_reshard dst_shards")
    _check(_lib.dr_reshard(plan.handle, ctypes.cast(a, _PP), ctypes.cast(b, _PP),
                           _buf(d_cks, 16 * i["num_chunks"], "dr_reshard d_cks", True), _stream(stream)), "dr_reshard")


def dr_reshard_through_host(plan: Plan, src_shards: Sequence, dst_shards: Sequence, d_cks, stream=None) -> None:
    i = plan.info
    ok = i["kind"] == DR_PLAN_RESHARD
    a = _shards(src_shards, i["train_shards"] if ok else None, 4 * i["shard_elems"], "dr_reshard_through_host src_shards")
    b = _shards(dst_shards, i["dst_shards"] if ok else None, 4 * i["dst_shard_elems"],
                "dr_reshard_through_host dst_shards")
    _check(_lib.dr_reshard_through_host(plan.handle, ctypes.cast(a, _PP), ctypes.cast(b, _PP),
                                        _buf(d_cks, 16 * i["num_chunks"], "dr_reshard_through_host d_cks", True),
                                        _stream(stream)), "dr_reshard_through_host")


def _moment_args(plan: Plan, m_shards: Sequence, v_shards: Sequence, host_store, where: str):
    i = plan.info
    m = _shards(m_shards, i["train_shards"], 4 * i["shard_elems"], f"{where} m_shards")
    v = _shards(v_shards, i["train_shards"], 4 * i["shard_elems"], f"{where} v_shards")
    return m, v, _buf(host_store, i["moment_bytes"], f"{where} host_store", False)


def dr_offload_moments(plan: Plan, m_shards: Sequence, v_shards: Sequence, host_store, side_stream) -> None:
    m, v, store = _moment_args(plan, m_shards, v_shards, host_store, "dr_offload_moments")
    _check(_lib.dr_offload_moments(plan.handle, ctypes.cast(m, _PP), ctypes.cast(v, _PP), store,
                                   _stream(side_stream)), "dr_offload_moments")


def dr_restore_moments(plan: Plan, host_store, m_shards: Sequence, v_shards: Sequence, side_stream) -> None:
    m, v, store = _moment_args(plan, m_shards, v_shards, host_store, "dr_restore_moments")
    _check(_lib.dr_restore_moments(plan.handle, store, ctypes.cast(m, _PP), ctypes.cast(v, _PP),
                                   _stream(side_stream)), "dr_restore_moments")


def dr_offload_moments_range(plan: Plan, m_shards: Sequence, v_shards: Sequence, host_store, first_chunk: int,
                             num_chunks: int, side_stream) -> None:
    m, v, store = _moment_args(plan, m_shards, v_shards, host_store, "dr_offload_moments_range")
    _check(_lib.dr_offload_moments_range(plan.handle, ctypes.cast(m, _PP), ctypes.cast(v, _PP), store,
                                         int(first_chunk), int(num_chunks), _stream(side_stream)),
           "dr_offload_moments_range")


def dr_restore_moments_range(plan: Plan, host_store, m_shards: Sequence, v_shards: Sequence, first_chunk: int,
                             num_chunks: int, side_stream) -> None:
    m, v, store = _moment_args(plan, m_shards, v_shards, host_store, "dr_restore_moments_range")
    _check(_lib.dr_restore_moments_range(plan.handle, store, ctypes.cast(m, _PP), ctypes.cast(v, _PP),
                                         int(first_chunk), int(num_chunks), _stream(side_stream)),
           "dr_restore_moments_range")


def dr_restore_moments_begin(plan: Plan, host_store, m_shards: Sequence, v_shards: Sequence, side_stream) -> None:
    """Starts the deferred restore on a library thread.  The plan keeps references to the host
    store, the shard tensors and the side stream until dr_restore_moments_end (or close), so
    none of them is freed while the thread still copies."""
    m, v, store = _moment_args(plan, m_shards, v_shards, host_store, "dr_restore_moments_begin")
    refs = (host_store, tuple(m_shards), tuple(v_shards), side_stream)
    _check(_lib.dr_restore_moments_begin(plan.handle, store, ctypes.cast(m, _PP), ctypes.cast(v, _PP),
                                         _stream(side_stream)), "dr_restore_moments_begin")
    plan._restore_refs = refs


def dr_restore_moments_end(plan: Plan) -> None:
    try:
        _check(_lib.dr_restore_moments_end(plan.handle), "dr_restore_moments_end")
    finally:
        plan._restore_refs = None  # the thread has been joined, whatever it returned


def dr_moment_checksums(plan: Plan, m_shards: Sequence, v_shards: Sequence, d_cks, stream=None) -> None:
    """Checksum of every moment chunk (num_moment_chunks dr_checksum slots in d_cks)."""
    i = plan.info
    m = _shards(m_shards, i["train_shards"], 4 * i["shard_elems"], "dr_moment_checksums m_shards")
    v = _shards(v_shards, i["train_shards"], 4 * i["shard_elems"], "dr_moment_checksums v_shards")
    _check(_lib.dr_moment_checksums(plan.handle, ctypes.cast(m, _PP), ctypes.cast(v, _PP),
                                    _buf(d_cks, 16 * i["num_moment_chunks"], "dr_moment_checksums d_cks", True),
                                    _stream(stream)), "dr_moment_checksums")


class Hysteresis:
    """Owns a dr_hyst*."""

    def __init__(self, handle: int):
        self._h = handle

    @property
    def handle(self) -> int:
        return self._h

    def close(self) -> None:
        if self._h:
            _lib.dr_hyst_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def dr_hyst_create(train_gpus: Sequence[int], rollout_gpus: Sequence[int], initial: int, enter: float, exit: float,
                   consecutive: int, dwell: int, cooldown: int, switch_cost_s: float = 0.0,
                   horizon_steps: int = 0) -> Hysteresis:
    """train_gpus/rollout_gpus: the pre-specified splits, most training GPUs first."""
    n = len(train_gpus)
    tg = (ctypes.c_int32 * max(n, 1))(*[int(x) for x in train_gpus])
    rg = (ctypes.c_int32 * max(len(rollout_gpus), 1))(*[int(x) for x in rollout_gpus])
    p = dr_hyst_params(int(n) if len(rollout_gpus) == n else -1, int(initial), tg, rg, float(enter), float(exit),
                       int(consecutive), int(dwell), int(cooldown), int(horizon_steps), float(switch_cost_s))
    h = ctypes.c_void_p()
    _check(_lib.dr_hyst_create(ctypes.byref(p), ctypes.byref(h)), "dr_hyst_create")
    return Hysteresis(h.value)


def dr_hyst_step(h: Hysteresis, t_rollout: float, t_train: float) -> dict:
    d = dr_hyst_decision()
    _check(_lib.dr_hyst_step(h.handle, float(t_rollout), float(t_train), ctypes.byref(d)), "dr_hyst_step")
    return {"config": d.config, "action": d.action, "reason": d.reason, "run": d.run, "imbalance": d.imbalance,
            "predicted_gain_s": d.predicted_gain_s}


def dr_break_even_steps(switch_cost_s: float, step_before_s: float, step_after_s: float) -> float:
    return _lib.dr_break_even_steps(float(switch_cost_s), float(step_before_s), float(step_after_s))


def dr_last_error() -> str:
    return _lib.dr_last_error().decode(errors="replace")


def library_path() -> str:
    return _LIB_PATH
