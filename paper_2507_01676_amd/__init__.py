"""Python binding of libembx (ctypes): argument marshalling only.

Every step of the lookup runs in the library's HIP kernels; PyTorch provides
device memory and streams.  Names follow include/embx.h.  Importing this
package fails loudly if the native library has not been built.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.environ.get("EMBX_LIBRARY") or os.path.join(_HERE, "libembx.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"embx native library missing: {LIB_PATH} (build it with: python paper_2507_01676_amd/build.py)")

# PyTorch ships its own HIP runtime under the same soname as the system one; it must be
# the one in the process (loaded first), so that torch's device pointers and streams
# and the library's kernels live in one runtime.
try:
    import torch  # noqa: F401
except ImportError:
    pass

_lib = ctypes.CDLL(LIB_PATH)

# ---------------------------------------------------------------- constants (include/embx.h)
OK, ERR_INVALID_ARGUMENT, ERR_UNSUPPORTED, ERR_OUT_OF_MEMORY, ERR_DEVICE, ERR_NOT_BOUND, \
    ERR_INDEX_OUT_OF_RANGE, ERR_BUFFER_TOO_SMALL = range(8)
DTYPE_F32, DTYPE_F16 = 0, 1
STRAT_AUTO, STRAT_LDS, STRAT_HOT, STRAT_DEDUP, STRAT_GATHER = -1, 0, 1, 2, 3
STRATEGY_NAMES = {0: "LDS", 1: "HOT", 2: "DEDUP", 3: "GATHER", 4: "STREAM"}
POOL_SUM, POOL_MEAN = 0, 1
POOLING_CODES = {"sum": POOL_SUM, "mean": POOL_MEAN}
BETA_COUNT = 11
MAX_HOT_STATS = 4096

EXPORTED = ["emb_plan_create", "emb_plan_create_noalloc", "emb_plan_bind_weights", "emb_lookup", "emb_lookup_weighted", "emb_plan_check_errors",
            "emb_plan_serialize", "emb_plan_get_info", "emb_plan_destroy", "emb_plan_text",
            "emb_status_string", "emb_debug_dedup_tile", "emb_debug_hot_probe", "embx_fill_table",
            "emb_plan_set_trace", "emb_default_beta", "emb_debug_check_input"]


class EmbxError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(f"{what}: {status_string(code)} ({code})")


class _Stats(ctypes.Structure):
    _fields_ = [("mean_pooling", ctypes.c_double), ("max_pooling", ctypes.c_int32), ("n_hot", ctypes.c_int32),
                ("hot_rows", ctypes.POINTER(ctypes.c_int64)), ("hot_freq", ctypes.POINTER(ctypes.c_double)),
                ("unique_frac", ctypes.c_double)]


class _Opts(ctypes.Structure):
    _fields_ = [("wg_per_cu", ctypes.c_int32), ("lds_budget_bytes", ctypes.c_int32), ("lif_milli", ctypes.c_int32),
                ("order_mode", ctypes.c_int32), ("chunk_max_bytes", ctypes.c_int64),
                ("beta", ctypes.POINTER(ctypes.c_double)), ("force_strategy", ctypes.POINTER(ctypes.c_int32)),
                ("num_workers", ctypes.c_int32), ("sym_max_gather", ctypes.c_int32),
                ("pooling", ctypes.POINTER(ctypes.c_int32)), ("no_replication", ctypes.c_int32),
                ("gather_lookup_ps", ctypes.POINTER(ctypes.c_double))]


class _Info(ctypes.Structure):
    _fields_ = [("num_tables", ctypes.c_int32), ("embedding_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("row_bytes", ctypes.c_int32), ("num_workers", ctypes.c_int32), ("block_threads", ctypes.c_int32),
                ("lds_bytes", ctypes.c_int32), ("num_items", ctypes.c_int32), ("max_batch", ctypes.c_int32),
                ("lds_budget_bytes", ctypes.c_int32), ("max_load_ps", ctypes.c_int64),
                ("sum_load_ps", ctypes.c_int64), ("lif_milli", ctypes.c_int32), ("r_symmetric", ctypes.c_int32),
                ("n_strategy", ctypes.c_int32 * 5), ("gather_runs", ctypes.c_int32 * 3), ("kernel", ctypes.c_int32),
                ("debug_checks", ctypes.c_int32), ("gather_steps", ctypes.c_int32)]


_vp, _i32, _i64, _sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
_lib.emb_status_string.restype = ctypes.c_char_p
_lib.emb_status_string.argtypes = [_i32]
_lib.emb_plan_create.argtypes = [ctypes.POINTER(_vp), _i32, ctypes.POINTER(_i64), _i32, _i32,
                                 ctypes.POINTER(_Stats), _i32, ctypes.POINTER(_Opts)]
_lib.emb_plan_create_noalloc.argtypes = _lib.emb_plan_create.argtypes
_lib.emb_plan_bind_weights.argtypes = [_vp, ctypes.POINTER(_vp)]
_lib.emb_lookup.argtypes = [_vp, _vp, _vp, _i32, _vp, _vp]
_lib.emb_lookup_weighted.argtypes = [_vp, _vp, _vp, _vp, _i32, _vp, _vp]
_lib.emb_plan_check_errors.argtypes = [_vp, _vp, ctypes.POINTER(_i64)]
_lib.emb_plan_serialize.argtypes = [_vp, ctypes.c_char_p, _sz, ctypes.POINTER(_sz)]
_lib.emb_plan_get_info.argtypes = [_vp, ctypes.POINTER(_Info)]
_lib.emb_plan_destroy.argtypes = [_vp]
_lib.emb_plan_text.argtypes = [_i32, ctypes.POINTER(_i64), _i32, _i32, ctypes.POINTER(_Stats), _i32, _i32,
                               ctypes.POINTER(_Opts), ctypes.c_char_p, _sz, ctypes.POINTER(_sz)]
_lib.emb_plan_set_trace.argtypes = [_vp, _vp, _sz, ctypes.POINTER(_sz)]
_lib.emb_default_beta.argtypes = [_i32, ctypes.POINTER(ctypes.c_double), _i32]
_lib.emb_debug_dedup_tile.argtypes = [_vp, _i32, _vp, _vp, _vp, _vp]
_lib.emb_debug_hot_probe.argtypes = [_vp, _i32, _vp, _i32, _vp, _vp]
_lib.emb_debug_check_input.argtypes = [_vp, _vp, _vp, _vp, _i32, _vp]
_lib.embx_fill_table.argtypes = [_vp, _i64, _i64, _i32, _i32, _i32, ctypes.c_uint64, ctypes.c_double,
                                 ctypes.c_double, _i32, _vp]
for _f in EXPORTED:
    if _f != "emb_status_string":
        getattr(_lib, _f).restype = _i32


def status_string(code: int) -> str:
    return _lib.emb_status_string(int(code)).decode()


def _check(code: int, what: str):
    if code != OK:
        raise EmbxError(code, what)


def _dtype_code(dtype) -> int:
    if dtype in ("f32", "fp32", "float32", DTYPE_F32):
        return DTYPE_F32
    if dtype in ("f16", "fp16", "float16", DTYPE_F16):
        return DTYPE_F16
    try:
        import torch
        if dtype == torch.float32:
            return DTYPE_F32
        if dtype == torch.float16:
            return DTYPE_F16
    except ImportError:
        pass
    raise ValueError(f"unsupported dtype {dtype!r}")


def _get(s, name, default=None):
    if isinstance(s, dict):
        return s.get(name, default)
    return getattr(s, name, default)


class _Marshal:
    """Holds the ctypes views of the statistics and options for one call."""

    def __init__(self, rows, stats, opts: dict, T: int):
        self.rows = (ctypes.c_int64 * T)(*[int(r) for r in rows])
        self.stats = (_Stats * T)()
        self.keep = []
        for t, s in enumerate(stats):
            hr = np.ascontiguousarray(np.asarray(_get(s, "hot_rows", []), dtype=np.int64)[:MAX_HOT_STATS])
            hf = np.ascontiguousarray(np.asarray(_get(s, "hot_freq", []), dtype=np.float64)[:MAX_HOT_STATS])
            n = min(hr.size, hf.size)
            self.keep += [hr, hf]
            st = self.stats[t]
            st.mean_pooling = float(_get(s, "mean_pooling", 1.0))
            st.max_pooling = int(_get(s, "max_pooling", 0) or 0)
            st.n_hot = n
            st.hot_rows = hr.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)) if n else None
            st.hot_freq = hf.ctypes.data_as(ctypes.POINTER(ctypes.c_double)) if n else None
            uf = _get(s, "unique_frac", -1.0)
            st.unique_frac = float(-1.0 if uf is None else uf)
        o = _Opts()
        o.wg_per_cu = int(opts.get("wg_per_cu", 0))
        o.lds_budget_bytes = int(opts.get("lds_budget", 0))
        o.lif_milli = int(opts.get("lif_milli", 0))
        o.order_mode = int(opts.get("order_mode", 0))
        o.chunk_max_bytes = int(opts.get("chunk_max_bytes", 0))
        o.num_workers = int(opts.get("num_workers", 0))
        o.sym_max_gather = int(opts.get("sym_max", 0))
        o.no_replication = 1 if opts.get("no_replication", False) else 0
        beta = opts.get("beta")
        if beta is not None:
            b = np.ascontiguousarray(np.asarray(beta, dtype=np.float64))
            if b.size != BETA_COUNT:
                raise ValueError(f"beta needs {BETA_COUNT} coefficients, got {b.size}")
            self.keep.append(b)
            o.beta = b.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
        force = opts.get("force")
        if force is not None:
            f = np.ascontiguousarray(np.asarray(force, dtype=np.int32))
            if f.size != T:
                raise ValueError(f"force needs one strategy per table ({T}), got {f.size}")
            self.keep.append(f)
            o.force_strategy = f.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        pooling = opts.get("pooling")
        if pooling is not None:
            if isinstance(pooling, (str, int)):
                pooling = [pooling] * T
            pc = np.ascontiguousarray(np.asarray([POOLING_CODES.get(x, x) for x in pooling], dtype=np.int32))
            if pc.size != T:
                raise ValueError(f"pooling needs one reduction per table ({T}), got {pc.size}")
            self.keep.append(pc)
            o.pooling = pc.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        g1 = opts.get("gather_lookup_ps")
        if g1 is not None:
            g = np.ascontiguousarray(np.asarray(g1, dtype=np.float64))
            if g.size != T:
                raise ValueError(f"gather_lookup_ps needs one cost per table ({T}), got {g.size}")
            self.keep.append(g)
            o.gather_lookup_ps = g.ctypes.data_as(ctypes.POINTER(ctypes.c_double))
        self.opts = o


def _stream_ptr(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def default_beta(row_bytes: int) -> List[float]:
    """The built-in cost coefficients (picoseconds, layout of ``include/embx.h``) the
    planner uses for rows of ``row_bytes`` bytes when no beta is given."""
    out = (ctypes.c_double * BETA_COUNT)()
    _check(_lib.emb_default_beta(int(row_bytes), out, BETA_COUNT), "emb_default_beta")
    return [float(x) for x in out]


def plan_text(rows: Sequence[int], E: int, dtype, stats, max_batch: int, num_workers: int, **opts) -> str:
    """The planner alone (host only): the canonical text of the plan for ``num_workers`` workers."""
    T = len(rows)
    m = _Marshal(rows, stats, opts, T)
    n = _sz(0)
    code = _lib.emb_plan_text(T, m.rows, int(E), _dtype_code(dtype), m.stats, int(max_batch), int(num_workers),
                              ctypes.byref(m.opts), None, 0, ctypes.byref(n))
    if code not in (OK, ERR_BUFFER_TOO_SMALL):
        raise EmbxError(code, "emb_plan_text")
    buf = ctypes.create_string_buffer(n.value + 1)
    _check(_lib.emb_plan_text(T, m.rows, int(E), _dtype_code(dtype), m.stats, int(max_batch), int(num_workers),
                              ctypes.byref(m.opts), buf, n.value + 1, ctypes.byref(n)), "emb_plan_text")
    return buf.value.decode()


class Plan:
    """A lookup plan on the current HIP device (emb_plan_create .. emb_plan_destroy)."""

    def __init__(self, rows: Sequence[int], E: int, dtype, stats, max_batch: int, noalloc: bool = False, **opts):
        """``noalloc``: emb_plan_create_noalloc (device data in the library's fixed per-GPU
        array; a later such plan on the device replaces this one)."""
        self.T = len(rows)
        self.E = int(E)
        self.dtype = _dtype_code(dtype)
        self.max_batch = int(max_batch)
        m = _Marshal(rows, stats, opts, self.T)
        h = _vp()
        fn = _lib.emb_plan_create_noalloc if noalloc else _lib.emb_plan_create
        _check(fn(ctypes.byref(h), self.T, m.rows, self.E, self.dtype, m.stats, self.max_batch,
                  ctypes.byref(m.opts)), "emb_plan_create_noalloc" if noalloc else "emb_plan_create")
        self._h = h
        self._weights = None

    def bind(self, weights: List) -> "Plan":
        import torch
        if len(weights) != self.T:
            raise ValueError(f"bind needs one table per plan table ({self.T}), got {len(weights)}")
        want = torch.float16 if self.dtype == DTYPE_F16 else torch.float32
        for w in weights:
            if not (w.is_cuda and w.dtype == want and w.dim() == 2 and w.shape[1] == self.E and w.is_contiguous()):
                raise ValueError("weights must be contiguous [rows, E] device tensors of the plan's dtype")
        arr = (_vp * self.T)(*[w.data_ptr() for w in weights])
        _check(_lib.emb_plan_bind_weights(self._h, arr), "emb_plan_bind_weights")
        self._weights = list(weights)
        return self

    def lookup(self, indices, offsets, batch: int, out=None, stream=None, weights=None):
        """One batch (emb_lookup); with ``weights`` (fp32 device tensor aligned with
        ``indices``) each lookup's row is scaled by its weight (emb_lookup_weighted)."""
        import torch
        if out is None:
            out = torch.empty((batch, self.T, self.E), dtype=torch.float32, device=indices.device)
        for name, x, dt in (("indices", indices, torch.int64), ("offsets", offsets, torch.int64),
                            ("out", out, torch.float32)):
            if not (x.is_cuda and x.dtype == dt and x.is_contiguous()):
                raise ValueError(f"{name} must be a contiguous {dt} device tensor")
        if out.numel() < batch * self.T * self.E:
            raise ValueError(f"out holds {out.numel()} elements, the batch needs {batch * self.T * self.E}")
        if offsets.numel() < self.T * batch + 1:
            raise ValueError(f"offsets holds {offsets.numel()} entries, the batch needs {self.T * batch + 1}")
        if weights is None:
            _check(_lib.emb_lookup(self._h, indices.data_ptr(), offsets.data_ptr(), int(batch), out.data_ptr(),
                                   _stream_ptr(stream)), "emb_lookup")
        else:
            if not (weights.is_cuda and weights.dtype == torch.float32 and weights.is_contiguous()
                    and weights.numel() >= indices.numel()):
                raise ValueError("weights must be a contiguous fp32 device tensor with one weight per index")
            _check(_lib.emb_lookup_weighted(self._h, indices.data_ptr(), offsets.data_ptr(), weights.data_ptr(),
                                            int(batch), out.data_ptr(), _stream_ptr(stream)), "emb_lookup_weighted")
        return out

    def lookup_ptr(self, indices_ptr: int, offsets_ptr: int, batch: int, out_ptr: int, stream_ptr,
                   weights_ptr: int = 0) -> None:
        """Raw-pointer launch (benchmark loop); weights_ptr != 0 -> emb_lookup_weighted."""
        if weights_ptr:
            _check(_lib.emb_lookup_weighted(self._h, indices_ptr, offsets_ptr, weights_ptr, int(batch), out_ptr,
                                            stream_ptr), "emb_lookup_weighted")
        else:
            _check(_lib.emb_lookup(self._h, indices_ptr, offsets_ptr, int(batch), out_ptr, stream_ptr), "emb_lookup")

    def set_trace(self, buf) -> int:
        """Records per-slice timers into device uint64/int64 tensor ``buf`` (None: off).
        Returns the number of entries the plan needs."""
        n = _sz(0)
        if buf is None:
            _check(_lib.emb_plan_set_trace(self._h, None, 0, ctypes.byref(n)), "emb_plan_set_trace")
            self._trace = None
            return int(n.value)
        _check(_lib.emb_plan_set_trace(self._h, buf.data_ptr(), buf.numel(), ctypes.byref(n)), "emb_plan_set_trace")
        self._trace = buf
        return int(n.value)

    def trace_size(self) -> int:
        n = _sz(0)
        _lib.emb_plan_set_trace(self._h, None, 0, ctypes.byref(n))
        return int(n.value)

    def check_errors(self, stream=None) -> int:
        n = _i64(0)
        code = _lib.emb_plan_check_errors(self._h, _stream_ptr(stream), ctypes.byref(n))
        if code not in (OK, ERR_INDEX_OUT_OF_RANGE):
            raise EmbxError(code, "emb_plan_check_errors")
        return int(n.value)

    def serialize(self) -> str:
        n = _sz(0)
        _lib.emb_plan_serialize(self._h, None, 0, ctypes.byref(n))
        buf = ctypes.create_string_buffer(n.value + 1)
        _check(_lib.emb_plan_serialize(self._h, buf, n.value + 1, ctypes.byref(n)), "emb_plan_serialize")
        return buf.value.decode()

    def info(self) -> dict:
        i = _Info()
        _check(_lib.emb_plan_get_info(self._h, ctypes.byref(i)), "emb_plan_get_info")
        d = {k: getattr(i, k) for k, _ in _Info._fields_ if k not in ("n_strategy", "gather_runs")}
        d["n_strategy"] = {STRATEGY_NAMES[s]: i.n_strategy[s] for s in range(5)}
        d["gather_runs"] = {"wave": i.gather_runs[0], "single": i.gather_runs[1], "sw": i.gather_runs[2]}
        d["kernel"] = "gather_kernel" if i.kernel == 1 else "lookup_kernel"
        return d

    def check_input(self, indices, offsets, batch: int, weights=None, stream=None):
        """The input checks of EMBX_DEBUG_CHECKS on one launch's input (launches nothing)."""
        _check(_lib.emb_debug_check_input(self._h, indices.data_ptr(), offsets.data_ptr(),
                                          weights.data_ptr() if weights is not None else None, int(batch),
                                          _stream_ptr(stream)), "emb_debug_check_input")

    def hot_probe(self, table: int, idx, stream=None):
        import torch
        slot = torch.empty(idx.numel(), dtype=torch.int32, device=idx.device)
        _check(_lib.emb_debug_hot_probe(self._h, int(table), idx.data_ptr(), idx.numel(), slot.data_ptr(),
                                        _stream_ptr(stream)), "emb_debug_hot_probe")
        return slot

    def close(self):
        if getattr(self, "_h", None):
            _check(_lib.emb_plan_destroy(self._h), "emb_plan_destroy")
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def fill_table(w, table_id: int, seed: int, lo: float = -0.05, hi: float = 0.05, mode: int = 0,
               row_begin: int = 0, stream=None):
    """Fills device tensor ``w`` [n, E] with rows [row_begin, row_begin+n) of the synthetic table."""
    import torch
    if not (w.is_cuda and w.is_contiguous() and w.dim() == 2 and w.dtype in (torch.float16, torch.float32)):
        raise ValueError("fill_table needs a contiguous 2-D fp16 or fp32 device tensor")
    dt = DTYPE_F16 if w.dtype == torch.float16 else DTYPE_F32
    _check(_lib.embx_fill_table(w.data_ptr(), int(row_begin), int(w.shape[0]), int(w.shape[1]), dt, int(table_id),
                                int(seed) & ((1 << 64) - 1), float(lo), float(hi), int(mode), _stream_ptr(stream)),
           "embx_fill_table")
    return w


def fill_table_ptr(ptr: int, row_begin: int, n_rows: int, E: int, dtype_code: int, table_id: int, seed: int,
                   lo: float, hi: float, mode: int, stream_ptr) -> None:
    """Raw-pointer form of fill_table for timing loops (as thin as Plan.lookup_ptr: ctypes
    converts the arguments): rows [row_begin, row_begin + n_rows) of the synthetic table
    into device memory at ptr; dtype_code DTYPE_F32 or DTYPE_F16, seed < 2**64."""
    _check(_lib.embx_fill_table(ptr, row_begin, n_rows, E, dtype_code, table_id, seed, lo, hi, mode, stream_ptr),
           "embx_fill_table")


def dedup_tile(idx, stream=None):
    """Device tile sort/dedup of up to 2048 row ids: (sorted distinct ids, slot of each input)."""
    import torch
    n = idx.numel()
    uniq = torch.empty(max(n, 1), dtype=torch.int32, device=idx.device)
    inv = torch.empty(max(n, 1), dtype=torch.int32, device=idx.device)
    nu = torch.zeros(1, dtype=torch.int32, device=idx.device)
    _check(_lib.emb_debug_dedup_tile(idx.data_ptr(), n, uniq.data_ptr(), inv.data_ptr(), nu.data_ptr(),
                                     _stream_ptr(stream)), "emb_debug_dedup_tile")
    k = int(nu.item())
    return uniq[:k], inv[:n]
