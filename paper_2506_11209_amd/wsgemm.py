"""ctypes binding of libwsgemm.so (declared in include/ws_gemm.h and
include/ws_model.h).

Functions carry the C names and only marshal arguments; every step of the
GEMM runs in the library's HIP kernels.  Importing this module raises if the
library has not been built (``python -m paper_2506_11209_amd.build``): there
is no fallback path.

``WsGemm`` is a convenience wrapper over torch device tensors and streams.
"""
from __future__ import annotations

import ctypes
import os

# torch ships its own HIP runtime.  It must be the one loaded first: the
# library's libamdhip64 dependency then resolves to that same copy, and the
# process holds a single runtime (two copies do not share the device).
import torch  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(_HERE, "libwsgemm.so")

if not os.path.exists(LIBRARY):
    raise ImportError("%s is not built; run `python -m paper_2506_11209_amd.build`" % LIBRARY)

_lib = ctypes.CDLL(LIBRARY)

WS_F16, WS_BF16 = 0, 1
WS_LOAD_REGISTERS, WS_LOAD_DMA = 0, 1
LOAD_PATHS = {"registers": WS_LOAD_REGISTERS, "dma": WS_LOAD_DMA}
DTYPE_CODES = {"f16": WS_F16, "bf16": WS_BF16}

WS_OK = 0
WS_ERR_INVALID_ARG = 1
WS_ERR_UNSUPPORTED = 2
WS_ERR_LDS_OVERFLOW = 3
WS_ERR_HIP = 4
WS_ERR_TIMEOUT = 5
WS_ERR_NOT_DIVISIBLE = 6

# ws_calib_kind: calibration kernels of the performance model
WS_CALIB_NONE, WS_CALIB_EMPTY, WS_CALIB_LOAD_A, WS_CALIB_LOAD_B, WS_CALIB_MATH, WS_CALIB_EPILOGUE = \
    -1, 0, 1, 2, 3, 4
WS_CALIB_LOAD_AB = 5
CALIB_KINDS = {"empty": WS_CALIB_EMPTY, "load_a": WS_CALIB_LOAD_A, "load_b": WS_CALIB_LOAD_B,
               "math": WS_CALIB_MATH, "epilogue": WS_CALIB_EPILOGUE, "load_ab": WS_CALIB_LOAD_AB}


class ws_gemm_config(ctypes.Structure):
    _fields_ = [("tile_m", ctypes.c_int32), ("tile_n", ctypes.c_int32), ("tile_k", ctypes.c_int32),
                ("producer_waves", ctypes.c_int32), ("consumer_waves", ctypes.c_int32),
                ("stages", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("load_path", ctypes.c_int32), ("split", ctypes.c_int32)]


class ws_gemm_plan_info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "grid", "block", "lds_bytes", "tiles_m", "tiles_n", "tiles", "rounds", "iters", "split",
        "group_m", "xcd_remap", "ragged", "general")]

    def as_dict(self) -> dict:
        return {n: getattr(self, n) for n, _ in self._fields_}


# ws_out_dtype: element type of C
WS_OUT_F32, WS_OUT_BF16, WS_OUT_F16 = 0, 1, 2
OUT_DTYPES = {"f32": WS_OUT_F32, "bf16": WS_OUT_BF16, "f16": WS_OUT_F16}


class ws_gemm_epilogue(ctypes.Structure):
    _fields_ = [("alpha", ctypes.c_float), ("beta", ctypes.c_float), ("out_dtype", ctypes.c_int32)]


class ws_gemm_debug(ctypes.Structure):
    _fields_ = [("spin_limit", ctypes.c_int32), ("producer_delay", ctypes.c_int32),
                ("consumer_delay", ctypes.c_int32)]


class ws_model_params(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in (
        "t_init", "t_epilogue", "compute_throughput", "compute_latency", "load_throughput",
        "load_latency")]


class ws_model_options(ctypes.Structure):
    _fields_ = [("two_dma", ctypes.c_int32), ("persistent", ctypes.c_int32),
                ("finish_math", ctypes.c_int32)]


class ws_model_result(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in (
        "total_us", "round_us", "t_math", "t_load_a", "t_load_b", "wait_us")] + [
        ("rounds", ctypes.c_int32), ("iters", ctypes.c_int32)]

    def as_dict(self) -> dict:
        return {n: getattr(self, n) for n, _ in self._fields_}


_h = ctypes.c_void_p
_p = ctypes.c_void_p
_i64, _i32 = ctypes.c_int64, ctypes.c_int32

_lib.ws_gemm_abi_version.argtypes = []
_lib.ws_gemm_abi_version.restype = _i32
_lib.ws_gemm_status_str.argtypes = [_i32]
_lib.ws_gemm_status_str.restype = ctypes.c_char_p
_lib.ws_gemm_last_error.argtypes = []
_lib.ws_gemm_last_error.restype = ctypes.c_char_p
_lib.ws_gemm_plan.argtypes = [_i64, _i64, _i64, ctypes.POINTER(ws_gemm_config), _i32, _i32,
                              ctypes.POINTER(ws_gemm_plan_info)]
_lib.ws_gemm_plan.restype = _i32
_lib.ws_gemm_schedule.argtypes = [ctypes.POINTER(ws_gemm_plan_info), _i32, _i32,
                                  ctypes.POINTER(_i32), ctypes.POINTER(_i32)]
_lib.ws_gemm_schedule.restype = _i32
_lib.ws_gemm_create.argtypes = [_i64, _i64, _i64, ctypes.POINTER(ws_gemm_config),
                                ctypes.POINTER(_h)]
_lib.ws_gemm_create.restype = _i32
_lib.ws_gemm_create_calibration.argtypes = [_i64, _i64, _i64, ctypes.POINTER(ws_gemm_config), _i32,
                                            ctypes.POINTER(_h)]
_lib.ws_gemm_create_calibration.restype = _i32
_lib.ws_gemm_run.argtypes = [_h, _p, _p, _p, _p]
_lib.ws_gemm_run.restype = _i32
_lib.ws_gemm_sync_status.argtypes = [_h, _p]
_lib.ws_gemm_sync_status.restype = _i32
_u64p = ctypes.POINTER(ctypes.c_uint64)
_lib.ws_gemm_clock.argtypes = [_h, _p, _u64p, _u64p, ctypes.POINTER(_i64)]
_lib.ws_gemm_clock.restype = _i32
_lib.ws_gemm_query.argtypes = [_h, ctypes.POINTER(ws_gemm_plan_info)]
_lib.ws_gemm_query.restype = _i32
_lib.ws_gemm_set_debug.argtypes = [_h, ctypes.POINTER(ws_gemm_debug)]
_lib.ws_gemm_set_debug.restype = _i32
_lib.ws_gemm_set_epilogue.argtypes = [_h, ctypes.POINTER(ws_gemm_epilogue)]
_lib.ws_gemm_set_epilogue.restype = _i32
_lib.ws_gemm_set_trace.argtypes = [_h, _p, _i64, _i32, _i32]
_lib.ws_gemm_set_trace.restype = _i32
_lib.ws_gemm_run_noalloc.argtypes = [_i64, _i64, _i64, ctypes.POINTER(ws_gemm_config), _p, _p, _p, _p]
_lib.ws_gemm_run_noalloc.restype = _i32
_lib.ws_gemm_destroy.argtypes = [_h]
_lib.ws_gemm_destroy.restype = _i32
_lib.ws_model_predict.argtypes = [_i64, _i64, _i64, _i32, _i32, _i32, _i32, _i32,
                                  ctypes.POINTER(ws_model_params), ctypes.POINTER(ws_model_options),
                                  ctypes.POINTER(ws_model_result)]
_lib.ws_model_predict.restype = _i32
_lib.ws_model_predict_costs.argtypes = [_i64, _i64, _i64, _i32, _i32, _i32, _i32, _i32, ctypes.c_double,
                                        ctypes.c_double, ctypes.c_double,
                                        ctypes.POINTER(ws_model_params), ctypes.POINTER(ws_model_options),
                                        ctypes.POINTER(ws_model_result)]
_lib.ws_model_predict_costs.restype = _i32
_dp = ctypes.POINTER(ctypes.c_double)
_lib.ws_model_events.argtypes = [_i32, _i32, _i32, ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                 ctypes.c_double, ctypes.POINTER(ws_model_options), _dp, _dp, _dp]
_lib.ws_model_events.restype = _i32


def library() -> ctypes.CDLL:
    return _lib


def config(tile=(128, 128, 32), stages=3, producer_waves=4, consumer_waves=4, dtype="bf16",
           load_path="registers", split=0):
    """split: DMA warps per MATH warp (1 or 2); 0 derives it from the wave counts."""
    tm, tn, tk = tile
    return ws_gemm_config(tm, tn, tk, producer_waves, consumer_waves, stages, DTYPE_CODES[dtype],
                          LOAD_PATHS[load_path], split)


# -- C names -----------------------------------------------------------------

def ws_gemm_abi_version() -> int:
    return _lib.ws_gemm_abi_version()


def ws_gemm_status_str(status: int) -> str:
    return _lib.ws_gemm_status_str(status).decode()


def ws_gemm_last_error() -> str:
    return _lib.ws_gemm_last_error().decode()


def ws_gemm_plan(M, N, K, cfg: ws_gemm_config, num_cus: int, wgs_per_cu: int = 0):
    info = ws_gemm_plan_info()
    s = _lib.ws_gemm_plan(M, N, K, ctypes.byref(cfg), num_cus, wgs_per_cu, ctypes.byref(info))
    return s, info


def ws_gemm_schedule(info: ws_gemm_plan_info, wg: int, rnd: int):
    ti, tj = _i32(-1), _i32(-1)
    s = _lib.ws_gemm_schedule(ctypes.byref(info), wg, rnd, ctypes.byref(ti), ctypes.byref(tj))
    return s, ti.value, tj.value


def ws_gemm_create(M, N, K, cfg: ws_gemm_config):
    h = _h()
    s = _lib.ws_gemm_create(M, N, K, ctypes.byref(cfg), ctypes.byref(h))
    return s, h


def ws_gemm_create_calibration(M, N, K, cfg: ws_gemm_config, kind: int):
    h = _h()
    s = _lib.ws_gemm_create_calibration(M, N, K, ctypes.byref(cfg), kind, ctypes.byref(h))
    return s, h


def ws_gemm_run(h, A_ptr: int, B_ptr: int, C_ptr: int, stream_ptr: int = 0) -> int:
    return _lib.ws_gemm_run(h, _p(A_ptr), _p(B_ptr), _p(C_ptr), _p(stream_ptr))


def ws_gemm_sync_status(h, stream_ptr: int = 0) -> int:
    return _lib.ws_gemm_sync_status(h, _p(stream_ptr))


def ws_gemm_clock(h, stream_ptr: int = 0):
    """(status, shader_cycles, ref_ticks, launches); clears the accumulators."""
    c, r, n = ctypes.c_uint64(0), ctypes.c_uint64(0), _i64(0)
    s = _lib.ws_gemm_clock(h, _p(stream_ptr), ctypes.byref(c), ctypes.byref(r), ctypes.byref(n))
    return s, c.value, r.value, n.value


def ws_gemm_query(h):
    info = ws_gemm_plan_info()
    s = _lib.ws_gemm_query(h, ctypes.byref(info))
    return s, info


def ws_gemm_set_debug(h, dbg: ws_gemm_debug | None) -> int:
    return _lib.ws_gemm_set_debug(h, ctypes.byref(dbg) if dbg is not None else None)


def ws_gemm_set_epilogue(h, epi: ws_gemm_epilogue | None) -> int:
    return _lib.ws_gemm_set_epilogue(h, ctypes.byref(epi) if epi is not None else None)


def ws_gemm_set_trace(h, buf_ptr: int | None, nbytes: int = 0, wgs: int = 0, iters: int = 0) -> int:
    return _lib.ws_gemm_set_trace(h, _p(buf_ptr) if buf_ptr else None, nbytes, wgs, iters)


def ws_gemm_run_noalloc(M, N, K, cfg: ws_gemm_config, A_ptr: int, B_ptr: int, C_ptr: int,
                        stream_ptr: int = 0) -> int:
    return _lib.ws_gemm_run_noalloc(M, N, K, ctypes.byref(cfg), _p(A_ptr), _p(B_ptr), _p(C_ptr),
                                    _p(stream_ptr))


def ws_gemm_destroy(h) -> int:
    return _lib.ws_gemm_destroy(h)


# -- convenience over torch ----------------------------------------------------

class WsGemmError(RuntimeError):
    def __init__(self, where: str, status: int):
        detail = (" [%s]" % ws_gemm_last_error()) if status == WS_ERR_HIP else ""
        super().__init__("%s: %s (status %d)%s" % (where, ws_gemm_status_str(status), status, detail))
        self.status = status


class WsGemm:
    """A created plan for one (M, N, K, configuration); call it on torch tensors."""

    def __init__(self, M, N, K, tile=(128, 128, 32), stages=3, producer_waves=4,
                 consumer_waves=4, dtype="bf16", load_path="registers", calibration=None, split=0):
        """calibration: None for the GEMM, else a key of CALIB_KINDS (the
        calibration kernels of the performance model, same launch).  split:
        DMA warps per MATH warp (1 or 2; 0 derives it from the wave counts)."""
        self.M, self.N, self.K = M, N, K
        self.dtype = dtype
        self.out_dtype = "f32"
        self.cfg = config(tile, stages, producer_waves, consumer_waves, dtype, load_path, split)
        if calibration is None:
            s, self._h = ws_gemm_create(M, N, K, self.cfg)
            where = "ws_gemm_create"
        else:
            s, self._h = ws_gemm_create_calibration(M, N, K, self.cfg, CALIB_KINDS[calibration])
            where = "ws_gemm_create_calibration"
        if s != WS_OK:
            self._h = None
            raise WsGemmError(where, s)
        s, self.info = ws_gemm_query(self._h)
        if s != WS_OK:
            raise WsGemmError("ws_gemm_query", s)

    def _check(self, t, shape, dtype_name):
        import torch
        want = {"f16": torch.float16, "bf16": torch.bfloat16, "f32": torch.float32}[dtype_name]
        if t.device.type != "cuda" or t.dtype != want or tuple(t.shape) != shape or not t.is_contiguous():
            raise ValueError("expected a contiguous %s cuda tensor of shape %s, got %s %s %s" % (
                dtype_name, shape, t.dtype, tuple(t.shape), t.device))

    def __call__(self, A, B, C=None, stream=None):
        import torch
        self._check(A, (self.M, self.K), self.dtype)
        self._check(B, (self.K, self.N), self.dtype)
        if C is None:
            want = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}[self.out_dtype]
            C = torch.empty((self.M, self.N), dtype=want, device=A.device)
        self._check(C, (self.M, self.N), self.out_dtype)
        st = stream if stream is not None else torch.cuda.current_stream(A.device)
        s = ws_gemm_run(self._h, A.data_ptr(), B.data_ptr(), C.data_ptr(), st.cuda_stream)
        if s != WS_OK:
            raise WsGemmError("ws_gemm_run", s)
        return C

    def set_epilogue(self, alpha=1.0, beta=0.0, out_dtype="f32"):
        """C <- alpha (A B) + beta C, stored as out_dtype ("f32", "bf16", "f16")."""
        s = ws_gemm_set_epilogue(self._h, ws_gemm_epilogue(alpha, beta, OUT_DTYPES[out_dtype]))
        if s != WS_OK:
            raise WsGemmError("ws_gemm_set_epilogue", s)
        self.out_dtype = out_dtype
        s, self.info = ws_gemm_query(self._h)
        if s != WS_OK:
            raise WsGemmError("ws_gemm_query", s)

    def run_ptrs(self, A_ptr, B_ptr, C_ptr, stream_ptr=0):
        s = ws_gemm_run(self._h, A_ptr, B_ptr, C_ptr, stream_ptr)
        if s != WS_OK:
            raise WsGemmError("ws_gemm_run", s)

    def sync_status(self, stream=None) -> int:
        import torch
        st = stream if stream is not None else torch.cuda.current_stream()
        return ws_gemm_sync_status(self._h, st.cuda_stream)

    def clock_mhz(self, stream=None):
        """Average shader clock (MHz) of the launches since the last call, and
        their count (see ws_gemm_clock); (None, 0) when none took part."""
        import torch
        st = stream if stream is not None else torch.cuda.current_stream()
        s, cyc, ticks, n = ws_gemm_clock(self._h, st.cuda_stream)
        if s != WS_OK:
            raise WsGemmError("ws_gemm_clock", s)
        return (100.0 * cyc / ticks if ticks else None), n

    def set_debug(self, spin_limit=0, producer_delay=0, consumer_delay=0):
        s = ws_gemm_set_debug(self._h, ws_gemm_debug(spin_limit, producer_delay, consumer_delay))
        if s != WS_OK:
            raise WsGemmError("ws_gemm_set_debug", s)

    def close(self):
        if self._h is not None:
            ws_gemm_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# -- performance model (include/ws_model.h) ----------------------------------

def model_options(two_dma=False, persistent=False, finish_math=False) -> ws_model_options:
    return ws_model_options(int(two_dma), int(persistent), int(finish_math))


def ws_model_predict(M, N, K, tile_m, tile_n, tile_k, stages, slots, params: ws_model_params,
                     opts: ws_model_options | None = None):
    r = ws_model_result()
    s = _lib.ws_model_predict(M, N, K, tile_m, tile_n, tile_k, stages, slots, ctypes.byref(params),
                              ctypes.byref(opts) if opts is not None else None, ctypes.byref(r))
    return s, r


def ws_model_predict_costs(M, N, K, tile_m, tile_n, tile_k, stages, slots, t_math, t_load_a, t_load_b,
                           params: ws_model_params, opts: ws_model_options | None = None):
    r = ws_model_result()
    s = _lib.ws_model_predict_costs(M, N, K, tile_m, tile_n, tile_k, stages, slots, t_math, t_load_a,
                                    t_load_b, ctypes.byref(params),
                                    ctypes.byref(opts) if opts is not None else None, ctypes.byref(r))
    return s, r


def ws_model_events(iters, rounds, stages, t_math, t_load_a, t_load_b, t_epilogue,
                    opts: ws_model_options | None = None):
    """Returns (status, s_a, s_b, s_m) as lists; entry j is the paper's j + 1."""
    persistent = opts is not None and opts.persistent
    n = iters * rounds if persistent else iters
    if n <= 0:
        return WS_ERR_INVALID_ARG, [], [], []
    arrs = [(ctypes.c_double * n)() for _ in range(3)]
    s = _lib.ws_model_events(iters, rounds, stages, t_math, t_load_a, t_load_b, t_epilogue,
                             ctypes.byref(opts) if opts is not None else None, *arrs)
    return s, [list(a) for a in arrs][0], list(arrs[1]), list(arrs[2])
