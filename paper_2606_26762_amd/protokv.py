"""Thin ctypes binding of libprotokv (argument marshalling only).

Every step of the hot path runs in the HIP library; this module converts
Python/torch arguments into the C-ABI's pointers and sizes, and raises
``ProtoKVError`` on a non-OK status.  Loading fails loudly if the library has
not been built (``python -m paper_2606_26762_amd.build``).
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libprotokv.so")

ROW_BYTES = 3200
KV_BF16, KV_FP32 = 0, 1
FLAG_PQ, FLAG_MASS_BIAS, FLAG_MAINTENANCE, FLAG_EMA_CENTRES, FLAG_MAH_SQUARED, FLAG_VAR_ALLOC = 1, 2, 4, 8, 16, 32

STATUS = {0: "OK", 1: "E_INVALID", 2: "E_UNSUPPORTED", 3: "E_WORKSPACE", 4: "E_STATE", 5: "E_DEVICE"}

EXPORTED = [
    "protokv_default_config", "protokv_validate_config", "protokv_workspace_size", "protokv_init",
    "protokv_destroy", "protokv_append_frame", "protokv_fold", "protokv_synthesize", "protokv_attend",
    "protokv_stream_info_get", "protokv_get_counters", "protokv_read_assignments", "protokv_read_bank",
    "protokv_read_pseudo", "protokv_read_codebooks", "protokv_profile", "protokv_profile_read",
    "protokv_state_size", "protokv_get_state", "protokv_set_state", "protokv_attend_static",
    "protokv_read_pseudo_counts",
    "protokv_last_error",
]

STATE_MAGIC, STATE_VERSION = 0x53564B50, 1
MAX_EVICTED_TOKENS = 16777214
STATIC_SCRATCH_BYTES = 64 << 20

KERNELS = ["ring_insert", "seed", "screen", "aggregate", "decode", "attend", "attend_merge", "pq_encode",
           "materialize", "maintain", "rope_ring", "rope_q", "warm_collect", "warm_kmeans", "alloc"]


class ProtoKVError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [
        ("num_streams", ctypes.c_int32), ("num_layers", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32), ("num_q_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
        ("window_frames", ctypes.c_int32), ("capacity", ctypes.c_int32),
        ("pseudo_per_proto", ctypes.c_int32), ("pq_subspaces", ctypes.c_int32),
        ("pq_codewords", ctypes.c_int32), ("beam", ctypes.c_int32), ("t_idle", ctypes.c_int32),
        ("max_query_tokens", ctypes.c_int32), ("kv_dtype", ctypes.c_int32),
        ("flags", ctypes.c_uint32), ("eta", ctypes.c_float), ("pq_eps", ctypes.c_float),
        ("lambda_sp", ctypes.c_double), ("lambda_idle", ctypes.c_double), ("ridge", ctypes.c_double),
        ("gamma", ctypes.c_double), ("eps_k", ctypes.c_double), ("eps_v", ctypes.c_double),
        ("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("rope_theta", ctypes.c_double),
        ("warm_frames", ctypes.c_int32), ("warm_tokens", ctypes.c_int32),
        ("kmeans_epochs", ctypes.c_int32), ("kmeans_batch", ctypes.c_int32), ("pseudo_max", ctypes.c_int32),
    ]


class StreamInfo(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_uint64), ("evicted_tokens", ctypes.c_uint64),
                ("active_slots", ctypes.c_int32), ("pending", ctypes.c_int32)]


class Counters(ctypes.Structure):
    _fields_ = [("folds", ctypes.c_uint64), ("tokens_assigned", ctypes.c_uint64),
                ("tokens_seeded", ctypes.c_uint64), ("refined", ctypes.c_uint64),
                ("refined_full", ctypes.c_uint64), ("near_ties", ctypes.c_uint64),
                ("touched", ctypes.c_uint64), ("aged", ctypes.c_uint64), ("merged", ctypes.c_uint64),
                ("recycled", ctypes.c_uint64)]


class StateHeader(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_uint32), ("version", ctypes.c_uint32), ("units", ctypes.c_uint32),
                ("capacity", ctypes.c_uint32), ("tokens_per_frame", ctypes.c_uint32),
                ("window_frames", ctypes.c_uint32), ("kv_bytes", ctypes.c_uint32),
                ("codewords", ctypes.c_uint32), ("warm_tokens", ctypes.c_uint32), ("rotated", ctypes.c_uint32),
                ("frames", ctypes.c_uint64), ("evicted_tokens", ctypes.c_uint64),
                ("active_slots", ctypes.c_int32), ("folds", ctypes.c_int32),
                ("reservoir_rows", ctypes.c_int32), ("pad", ctypes.c_int32),
                ("off_ring_k", ctypes.c_uint64), ("off_ring_v", ctypes.c_uint64), ("off_bank", ctypes.c_uint64),
                ("off_codebooks", ctypes.c_uint64), ("off_reservoir", ctypes.c_uint64),
                ("off_ring_kr", ctypes.c_uint64), ("total_bytes", ctypes.c_uint64)]


class KernelTimes(ctypes.Structure):
    _fields_ = [("ms", ctypes.c_double * 16), ("launches", ctypes.c_uint64 * 16)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built: run `python -m paper_2606_26762_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        P = ctypes.POINTER
        L.protokv_default_config.argtypes = [P(Config)]
        L.protokv_validate_config.argtypes = [P(Config)]
        L.protokv_workspace_size.argtypes = [P(Config), P(sz)]
        L.protokv_init.argtypes = [P(Config), vp, vp, sz, vp, P(vp)]
        L.protokv_destroy.argtypes = [vp]
        L.protokv_append_frame.argtypes = [vp, P(i32), i32, vp, vp, vp]
        L.protokv_fold.argtypes = [vp, vp]
        L.protokv_synthesize.argtypes = [vp, i32, vp]
        L.protokv_attend.argtypes = [vp, i32, vp, i32, vp, vp, vp]
        L.protokv_attend_static.argtypes = [vp, i32, vp, i32, vp, vp, vp]
        L.protokv_stream_info_get.argtypes = [vp, i32, P(StreamInfo)]
        L.protokv_get_counters.argtypes = [vp, P(Counters), vp]
        L.protokv_read_assignments.argtypes = [vp, i32, vp, sz, vp]
        L.protokv_read_bank.argtypes = [vp, i32, vp, sz, vp]
        L.protokv_read_pseudo.argtypes = [vp, vp, vp, vp, vp]
        L.protokv_read_codebooks.argtypes = [vp, i32, vp, sz, vp]
        L.protokv_read_pseudo_counts.argtypes = [vp, vp, sz, vp]
        L.protokv_profile.argtypes = [vp, ctypes.c_uint32]
        L.protokv_profile_read.argtypes = [vp, P(KernelTimes)]
        L.protokv_state_size.argtypes = [vp, P(sz)]
        L.protokv_get_state.argtypes = [vp, i32, vp, sz, vp]
        L.protokv_set_state.argtypes = [vp, i32, vp, sz, vp]
        L.protokv_last_error.argtypes = [vp]
        L.protokv_last_error.restype = ctypes.c_char_p
        for name in EXPORTED:
            if name != "protokv_last_error":
                getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int, handle=None):
    if status != 0:
        msg = lib().protokv_last_error(handle)
        raise ProtoKVError(status, msg.decode() if msg else "")


def default_config(**overrides) -> Config:
    cfg = Config()
    _check(lib().protokv_default_config(ctypes.byref(cfg)))
    for k, v in overrides.items():
        if not hasattr(cfg, k):
            raise AttributeError(k)
        setattr(cfg, k, v)
    return cfg


def workspace_size(cfg: Config) -> int:
    n = ctypes.c_size_t()
    _check(lib().protokv_workspace_size(ctypes.byref(cfg), ctypes.byref(n)))
    return n.value


def _stream_ptr(stream) -> Optional[int]:
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def decode_bank(raw: np.ndarray, units: int, capacity: int) -> Dict[str, np.ndarray]:
    """Views of the documented bank row layout (uint8 [units*capacity*3200])."""
    rows = raw.reshape(units, capacity, ROW_BYTES)
    f32 = lambda a, b: rows[:, :, a:b].copy().view(np.float32)
    u32 = lambda a, b: rows[:, :, a:b].copy().view(np.uint32)
    meta = rows[:, :, 3072:3104].copy()
    return {
        "sum_k": f32(0, 512), "sum_v": f32(512, 1024), "sq_k": f32(1024, 1536), "sq_v": f32(1536, 2048),
        "hist_k": u32(2048, 2560).reshape(units, capacity, 8, 16),
        "hist_v": u32(2560, 3072).reshape(units, capacity, 8, 16),
        "n": meta[:, :, 0:4].view(np.uint32)[..., 0], "n_res": meta[:, :, 4:8].view(np.uint32)[..., 0],
        "mu": meta[:, :, 8:16].view(np.float32), "sigma": meta[:, :, 16:28].view(np.float32),
        "tau": meta[:, :, 28:32].view(np.int32)[..., 0],
    }


def encode_bank(bank: Dict[str, np.ndarray], units: int, capacity: int) -> np.ndarray:
    """The documented bank row layout (uint8 [units*capacity*3200]) from arrays
    shaped as decode_bank returns them (histograms [units][K][G][C], C <= 16)."""
    rows = np.zeros((units, capacity, ROW_BYTES), dtype=np.uint8)

    def put(a, b, arr, dt):
        rows[:, :, a:b] = np.ascontiguousarray(np.asarray(arr, dtype=dt).reshape(units, capacity, -1)).view(np.uint8)
    put(0, 512, bank["sum_k"], np.float32)
    put(512, 1024, bank["sum_v"], np.float32)
    put(1024, 1536, bank["sq_k"], np.float32)
    put(1536, 2048, bank["sq_v"], np.float32)
    for name, a in (("hist_k", 2048), ("hist_v", 2560)):
        h = np.zeros((units, capacity, 8, 16), dtype=np.uint32)
        src = np.asarray(bank[name])
        h[..., :src.shape[-1]] = src
        put(a, a + 512, h, np.uint32)
    put(3072, 3076, bank["n"], np.uint32)
    put(3076, 3080, bank["n_res"], np.uint32)
    put(3080, 3088, bank["mu"], np.float32)
    put(3088, 3100, bank["sigma"], np.float32)
    put(3100, 3104, bank["tau"], np.int32)
    return rows.reshape(-1)


class State:
    """One stream's state blob (protokv.h) with views of its sections."""

    def __init__(self, blob: np.ndarray, kv_dtype: str):
        self.blob = blob
        self.header = StateHeader.from_buffer_copy(blob[:ctypes.sizeof(StateHeader)].tobytes())
        h = self.header
        if h.magic != STATE_MAGIC:
            raise ValueError("not a protokv state blob")
        self.kv_dtype = kv_dtype
        T, W, U = h.tokens_per_frame, h.window_frames, h.units
        ring = U * (W + 1) * T * 128 * h.kv_bytes
        self._ring_shape = (U, W + 1, T, 128)
        self._ring_bytes = ring

    def _section(self, off, nbytes):
        return self.blob[off:off + nbytes]

    def ring(self, which: str = "k") -> np.ndarray:
        """The ring as float32 [units][W+1][T][D] (a copy)."""
        off = {"k": self.header.off_ring_k, "v": self.header.off_ring_v, "kr": self.header.off_ring_kr}[which]
        raw = self._section(off, self._ring_bytes)
        if self.header.kv_bytes == 4:
            return raw.view(np.float32).reshape(self._ring_shape).copy()
        return (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32).reshape(self._ring_shape)

    def bank(self) -> Dict[str, np.ndarray]:
        h = self.header
        return decode_bank(self._section(h.off_bank, h.units * h.capacity * ROW_BYTES), h.units, h.capacity)

    def set_bank_rows(self, unit: int, rows: np.ndarray):
        """Replace the rows of one unit (uint8 [capacity * 3200])."""
        h = self.header
        n = h.capacity * ROW_BYTES
        self.blob[h.off_bank + unit * n:h.off_bank + (unit + 1) * n] = rows

    def set_active_slots(self, n: int):
        self.header.active_slots = n
        self.blob[:ctypes.sizeof(StateHeader)] = np.frombuffer(bytes(self.header), dtype=np.uint8)

    def codebooks(self) -> np.ndarray:
        h = self.header
        n = h.units * 2 * 8 * h.codewords * 16
        return self._section(h.off_codebooks, n * 4).view(np.float32).reshape(h.units, 2, 8, h.codewords, 16)


class ProtoKV:
    """One libprotokv handle with its workspace held as a torch uint8 tensor."""

    def __init__(self, cfg: Config, codebooks: np.ndarray, device="cuda", stream=None):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.units = cfg.num_layers * cfg.num_kv_heads
        self.T = cfg.grid_h * cfg.grid_w
        self.kv_dtype = torch.float32 if cfg.kv_dtype == KV_FP32 else torch.bfloat16
        cb = np.ascontiguousarray(codebooks, dtype=np.float32)
        expect = (cfg.num_streams * self.units * 2 * cfg.pq_subspaces * cfg.pq_codewords
                  * (cfg.head_dim // cfg.pq_subspaces))
        if cb.size != expect:
            raise ValueError(f"codebooks: expected {expect} floats, got {cb.size}")
        self.workspace = torch.empty(workspace_size(cfg), dtype=torch.uint8, device=device)
        h = ctypes.c_void_p()
        _check(lib().protokv_init(ctypes.byref(cfg), cb.ctypes.data, self.workspace.data_ptr(),
                                  self.workspace.numel(), _stream_ptr(stream), ctypes.byref(h)))
        self.h = h

    def close(self):
        if getattr(self, "h", None) is not None and self.h.value:
            lib().protokv_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- hot path --------------------------------------------------------
    def append_frame(self, stream_ids: Sequence[int], k, v, stream=None):
        ids = (ctypes.c_int32 * len(stream_ids))(*stream_ids)
        self._check_tensor(k, (len(stream_ids), self.cfg.num_layers, self.cfg.num_kv_heads, self.T,
                               self.cfg.head_dim))
        self._check_tensor(v, tuple(k.shape))
        _check(lib().protokv_append_frame(self.h, ids, len(stream_ids), k.data_ptr(), v.data_ptr(),
                                          _stream_ptr(stream)), self.h)

    def fold(self, stream=None):
        _check(lib().protokv_fold(self.h, _stream_ptr(stream)), self.h)

    def synthesize(self, stream_id: int, stream=None):
        _check(lib().protokv_synthesize(self.h, stream_id, _stream_ptr(stream)), self.h)

    def attend(self, stream_id: int, q, out=None, lse=None, stream=None):
        torch = self.torch
        tq = q.shape[1]
        self._check_tensor(q, (self.cfg.num_layers, tq, self.cfg.num_q_heads, self.cfg.head_dim))
        if out is None:
            out = torch.empty_like(q)
        if lse is None:
            lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        _check(lib().protokv_attend(self.h, stream_id, q.data_ptr(), tq, out.data_ptr(),
                                    lse.data_ptr() if lse is not False else None,
                                    _stream_ptr(stream)), self.h)
        return out, lse

    def attend_static(self, stream_id: int, q, out=None, lse=None, stream=None):
        """protokv_attend_static: the readout with its scratch in the library's
        fixed device array (no allocation by the library)."""
        torch = self.torch
        tq = q.shape[1]
        self._check_tensor(q, (self.cfg.num_layers, tq, self.cfg.num_q_heads, self.cfg.head_dim))
        if out is None:
            out = torch.empty_like(q)
        if lse is None:
            lse = torch.empty(q.shape[:3], dtype=torch.float32, device=q.device)
        _check(lib().protokv_attend_static(self.h, stream_id, q.data_ptr(), tq, out.data_ptr(),
                                           lse.data_ptr() if lse is not False else None,
                                           _stream_ptr(stream)), self.h)
        return out, lse

    # -- introspection -----------------------------------------------------
    def stream_info(self, stream_id: int) -> StreamInfo:
        info = StreamInfo()
        _check(lib().protokv_stream_info_get(self.h, stream_id, ctypes.byref(info)), self.h)
        return info

    def counters(self, stream=None) -> Counters:
        c = Counters()
        _check(lib().protokv_get_counters(self.h, ctypes.byref(c), _stream_ptr(stream)), self.h)
        return c

    def read_assignments(self, stream_id: int, stream=None) -> np.ndarray:
        out = np.zeros((self.units, self.T), dtype=np.int32)
        _check(lib().protokv_read_assignments(self.h, stream_id, out.ctypes.data, out.size,
                                              _stream_ptr(stream)), self.h)
        return out

    def read_bank(self, stream_id: int, stream=None) -> Dict[str, np.ndarray]:
        raw = np.zeros(self.units * self.cfg.capacity * ROW_BYTES, dtype=np.uint8)
        _check(lib().protokv_read_bank(self.h, stream_id, raw.ctypes.data, raw.size,
                                       _stream_ptr(stream)), self.h)
        return decode_bank(raw, self.units, self.cfg.capacity)

    def read_codebooks(self, stream_id: int, stream=None) -> np.ndarray:
        """-> float32 [units][2][G][C][D/G]: the stream's PQ codebooks (given, or learned by the warm-up)."""
        c = self.cfg
        out = np.zeros((self.units, 2, c.pq_subspaces, c.pq_codewords, c.head_dim // c.pq_subspaces),
                       dtype=np.float32)
        _check(lib().protokv_read_codebooks(self.h, stream_id, out.ctypes.data, out.size, _stream_ptr(stream)),
               self.h)
        return out

    def read_pseudo(self, stream=None):
        """-> keys, values float32 [units][K*S][D] and bias [units][K]."""
        n = self.units * self.cfg.capacity * self.cfg.pseudo_per_proto * self.cfg.head_dim
        bits = 32 if self.cfg.kv_dtype == KV_FP32 else 16
        raw_k = np.zeros(n, dtype=np.uint32 if bits == 32 else np.uint16)
        raw_v = np.zeros_like(raw_k)
        bias = np.zeros(self.units * self.cfg.capacity, dtype=np.float32)
        _check(lib().protokv_read_pseudo(self.h, raw_k.ctypes.data, raw_v.ctypes.data, bias.ctypes.data,
                                         _stream_ptr(stream)), self.h)
        conv = (lambda r: r.view(np.float32)) if bits == 32 else \
            (lambda r: (r.astype(np.uint32) << 16).view(np.float32))
        shape = (self.units, self.cfg.capacity * self.cfg.pseudo_per_proto, self.cfg.head_dim)
        return conv(raw_k).reshape(shape), conv(raw_v).reshape(shape), bias.reshape(self.units, -1)

    def state_size(self) -> int:
        n = ctypes.c_size_t()
        _check(lib().protokv_state_size(self.h, ctypes.byref(n)), self.h)
        return n.value

    def get_state(self, stream_id: int, stream=None) -> State:
        blob = np.zeros(self.state_size(), dtype=np.uint8)
        _check(lib().protokv_get_state(self.h, stream_id, blob.ctypes.data, blob.size, _stream_ptr(stream)), self.h)
        return State(blob, "fp32" if self.cfg.kv_dtype == KV_FP32 else "bf16")

    def set_state(self, stream_id: int, state, stream=None):
        blob = np.ascontiguousarray(state.blob if isinstance(state, State) else state, dtype=np.uint8)
        _check(lib().protokv_set_state(self.h, stream_id, blob.ctypes.data, blob.size, _stream_ptr(stream)), self.h)

    def read_pseudo_counts(self, stream=None) -> np.ndarray:
        """-> int32 [units][K]: pseudo-tokens per slot of the current synthesis."""
        out = np.zeros((self.units, self.cfg.capacity), dtype=np.int32)
        _check(lib().protokv_read_pseudo_counts(self.h, out.ctypes.data, out.size, _stream_ptr(stream)), self.h)
        return out

    def profile(self, enable, kernels=None):
        """Time every launch (enable=True), only the named kernels, or stop (False)."""
        mask = 0
        if enable:
            mask = 0xFFFFFFFF if kernels is None else sum(1 << KERNELS.index(k) for k in kernels)
        _check(lib().protokv_profile(self.h, mask), self.h)

    def profile_read(self) -> Dict[str, dict]:
        """-> {kernel: {"ms": total, "launches": n, "avg_us": mean}} for timed kernels."""
        kt = KernelTimes()
        _check(lib().protokv_profile_read(self.h, ctypes.byref(kt)), self.h)
        out = {}
        for i, name in enumerate(KERNELS):
            n = int(kt.launches[i])
            if n:
                out[name] = {"ms": kt.ms[i], "launches": n, "avg_us": 1000.0 * kt.ms[i] / n}
        return out

    def _check_tensor(self, t, shape):
        if tuple(t.shape) != tuple(shape):
            raise ValueError(f"expected shape {tuple(shape)}, got {tuple(t.shape)}")
        if t.dtype != self.kv_dtype or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"expected a contiguous {self.kv_dtype} CUDA tensor")
