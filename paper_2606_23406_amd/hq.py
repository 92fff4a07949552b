"""Python binding of libhq.so: argument marshalling only.

Every entry point has the name of the C function it calls (include/hq.h).
PyTorch provides device memory and the current HIP stream; all codec work
runs in the library's gfx950 kernels.  There is no fallback: if libhq.so is
missing or fails to load, every call raises.
"""
import ctypes as C
import os

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libhq.so")

HQ_OK = 0
HQ_E8, HQ_D4, HQ_A2, HQ_Z = 0, 1, 2, 3
HQ_BF16, HQ_FP32, HQ_FP16, HQ_INT8 = 0, 1, 2, 3
HQ_ROT_NONE, HQ_ROT_SIGNS, HQ_ROT_QJL = 0, 1, 2
LATTICES = {"E8": HQ_E8, "D4": HQ_D4, "A2": HQ_A2, "Z": HQ_Z}
STATUS = {0: "HQ_OK", -1: "HQ_ERR_INVALID_ARG", -2: "HQ_ERR_UNSUPPORTED", -3: "HQ_ERR_CAPACITY",
          -4: "HQ_ERR_OVERFLOW", -5: "HQ_ERR_HIP", -6: "HQ_ERR_CORRUPT",
          -7: "HQ_ERR_NO_CALIBRATION"}


class HQError(RuntimeError):
    def __init__(self, fn, status):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)}")
        self.status = status


class Options(C.Structure):
    _fields_ = [("rotation", C.c_int32), ("dither", C.c_int32), ("rot_seed", C.c_uint64),
                ("dither_seed", C.c_uint64), ("norm_dtype", C.c_int32), ("substream", C.c_int32),
                ("use_snr", C.c_int32), ("reserved0", C.c_int32), ("snr_db", C.c_double),
                ("qjl", C.c_void_p)]


class PlanInfo(C.Structure):
    _fields_ = [("alpha", C.c_float), ("snr_db", C.c_float), ("tile", C.c_int32),
                ("lattice", C.c_int32), ("substream", C.c_int32), ("rice_k", C.c_int32),
                ("cols", C.c_int64), ("tiles_per_row", C.c_int64), ("subs_per_row", C.c_int64),
                ("max_words_per_substream", C.c_int64), ("max_words_per_row", C.c_int64)]


class Stats(C.Structure):
    _fields_ = [("payload_bits", C.c_uint64), ("pad_bits", C.c_uint64), ("status", C.c_uint32),
                ("overflow_tiles", C.c_uint32), ("corrupt_substreams", C.c_uint32),
                ("clamps", C.c_uint32)]


STATS_BYTES = C.sizeof(Stats)


class StreamStruct(C.Structure):
    _fields_ = [("payload", C.c_void_p), ("capacity_words", C.c_int64), ("offsets", C.c_void_p),
                ("kparam", C.c_void_p), ("norms", C.c_void_p), ("rows_capacity", C.c_int64),
                ("rows", C.c_int64), ("scan", C.c_void_p), ("scan_bytes", C.c_int64),
                ("stats", C.c_void_p)]


_lib = None


def lib():
    """Load libhq.so (built in-tree by paper_2606_23406_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2606_23406_amd.build`")
    L = C.CDLL(LIB_PATH)
    p, i32, i64, u64, f32 = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_float
    L.hq_plan.restype = i32
    L.hq_plan.argtypes = [i32, i32, f32, u64, i32, i64, p, p, p]
    L.hq_plan_destroy.restype = i32
    L.hq_plan_destroy.argtypes = [p]
    L.hq_plan_get_info.restype = i32
    L.hq_plan_get_info.argtypes = [p, p]
    L.hq_scan_bytes.restype = C.c_size_t
    L.hq_scan_bytes.argtypes = [p, i64]
    L.hq_encode.restype = i32
    L.hq_encode.argtypes = [p, p, i32, i64, i64, p, i32, p]
    L.hq_encode_noalloc.restype = i32
    L.hq_encode_noalloc.argtypes = [p, p, i32, i64, i64, p, i32, p]
    L.hq_decode.restype = i32
    L.hq_decode.argtypes = [p, p, i64, i64, p, i32, i64, p]
    L.hq_encode_group.restype = i32
    L.hq_encode_group.argtypes = [p, p, i32, p, p, p, i32, p]
    L.hq_decode_group.restype = i32
    L.hq_decode_group.argtypes = [p, p, p, i32, p, i32, p]
    L.hq_decode_int8.restype = i32
    L.hq_decode_int8.argtypes = [p, p, i64, i64, p, i64, p, p]
    L.hq_act_prep.restype = i32
    L.hq_act_prep.argtypes = [p, p, i64, i64, p, p, p]
    L.hq_gemm_int8_blockscaled.restype = i32
    L.hq_gemm_int8_blockscaled.argtypes = [p, p, p, i64, p, p, i64, p, i32, p]
    L.hq_decode_fp8.restype = i32
    L.hq_decode_fp8.argtypes = [p, p, i64, i64, p, i64, p, p]
    L.hq_act_prep_fp8.restype = i32
    L.hq_act_prep_fp8.argtypes = [p, p, i64, i64, p, p, p]
    L.hq_gemm_fp8_blockscaled.restype = i32
    L.hq_gemm_fp8_blockscaled.argtypes = [p, p, p, i64, p, p, i64, p, i32, p]
    L.hq_decode_mxfp4.restype = i32
    L.hq_decode_mxfp4.argtypes = [p, p, i64, i64, p, p, p]
    L.hq_act_prep_mxfp4.restype = i32
    L.hq_act_prep_mxfp4.argtypes = [p, p, i64, i64, p, p, p]
    L.hq_gemm_mxfp4_blockscaled.restype = i32
    L.hq_gemm_mxfp4_blockscaled.argtypes = [p, p, p, i64, p, p, i64, p, i32, p]
    L.hq_gemm_workspace_bytes.restype = C.c_size_t
    L.hq_gemm_workspace_bytes.argtypes = [p, i64, i64]
    L.hq_dequant_gemm_int8.restype = i32
    L.hq_dequant_gemm_int8.argtypes = [p, p, i64, p, i64, p, i32, p, C.c_size_t, p]
    L.hq_gemv_workspace_bytes.restype = C.c_size_t
    L.hq_gemv_workspace_bytes.argtypes = [p]
    L.hq_decode_gemv.restype = i32
    L.hq_decode_gemv.argtypes = [p, p, i64, i64, p, i32, p, i32, p, C.c_size_t, p]
    L.hq_attention_workspace_bytes.restype = C.c_size_t
    L.hq_attention_workspace_bytes.argtypes = [p, i64, i32, i64]
    L.hq_decode_attention.restype = i32
    L.hq_decode_attention.argtypes = [p, p, p, p, p, i32, i64, i32, C.c_float, p, i32, i32, p, p,
                                      p, i32, i32, p, i32, p, C.c_size_t, p]
    L.hq_rice_kstar.restype = i32
    L.hq_rice_kstar.argtypes = [i64, i64]
    L.hq_calibrated_snr.restype = i32
    L.hq_calibrated_snr.argtypes = [i32, i32, f32, C.POINTER(C.c_double)]
    L.hq_status_string.restype = C.c_char_p
    L.hq_status_string.argtypes = [i32]
    _lib = L
    return L


def _check(fn, status):
    if status != HQ_OK:
        raise HQError(fn, status)


def _stream_handle(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _dtype_code(dt):
    if dt == torch.bfloat16:
        return HQ_BF16
    if dt == torch.float32:
        return HQ_FP32
    raise ValueError(f"unsupported dtype {dt}")


class Plan:
    """An hq_plan handle and its derived values."""

    def __init__(self, handle, info: PlanInfo, options: Options):
        self.handle = handle
        self.info = info
        self.options = options

    @property
    def cols(self):
        return self.info.cols

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.hq_plan_destroy(self.handle)
            self.handle = None


def hq_plan(tile=128, lattice=HQ_E8, bps=4.0, rht_seed=0, rice_k=-1, cols=4096, *, rotation=0,
            dither=False, rot_seed=0, dither_seed=0, norm_fp16=False, snr_db=None, substream=0,
            qjl=None):
    """hq_plan of include/hq.h; snr_db bypasses the calibration table; qjl: the
    tile x tile orthogonal S of rotation HQ_ROT_QJL (host array, copied)."""
    L = lib()
    S = None
    if qjl is not None:
        S = np.ascontiguousarray(np.asarray(qjl, dtype=np.float32))
        assert S.shape == (tile, tile)
    o = Options(rotation, int(bool(dither)), rot_seed & (2**64 - 1), dither_seed & (2**64 - 1),
                HQ_FP16 if norm_fp16 else HQ_FP32, substream, 0 if snr_db is None else 1, 0,
                0.0 if snr_db is None else float(snr_db),
                None if S is None else S.ctypes.data_as(C.c_void_p))
    h = C.c_void_p()
    info = PlanInfo()
    st = L.hq_plan(tile, lattice, C.c_float(bps), rht_seed & (2**64 - 1), rice_k, cols, C.byref(o),
                   C.byref(h), C.byref(info))
    _check("hq_plan", st)
    o.qjl = None  # the plan holds its own device copy of S
    plan = Plan(h, info, o)
    plan.qjl = S
    return plan


class EncodedStream:
    """Device buffers of one encoded matrix (hq_stream), allocated with torch."""

    def __init__(self, plan: Plan, rows_capacity: int, device="cuda", capacity_words=None,
                 stats=True):
        info = plan.info
        self.plan = plan
        self.device = torch.device(device)
        cap = capacity_words if capacity_words is not None else rows_capacity * info.max_words_per_row
        self.payload = torch.zeros(max(int(cap), 1), dtype=torch.int32, device=device)
        nsub = rows_capacity * info.subs_per_row
        self.offsets = torch.zeros(nsub + 1, dtype=torch.int32, device=device)
        self.kparam = torch.zeros(max(nsub, 1), dtype=torch.uint8, device=device)
        ndt = torch.float16 if plan.options.norm_dtype == HQ_FP16 else torch.float32
        self.norms = torch.zeros(max(rows_capacity * info.tiles_per_row, 1), dtype=ndt,
                                 device=device)
        scan_bytes = lib().hq_scan_bytes(plan.handle, rows_capacity)
        self.scan = torch.zeros((scan_bytes + 7) // 8, dtype=torch.int64, device=device)
        self.stats = torch.zeros(STATS_BYTES // 4, dtype=torch.int32, device=device) if stats else None
        self.c = StreamStruct(self.payload.data_ptr(), int(cap), self.offsets.data_ptr(),
                              self.kparam.data_ptr(), self.norms.data_ptr(), rows_capacity, 0,
                              self.scan.data_ptr(), self.scan.numel() * 8,
                              self.stats.data_ptr() if stats else None)

    @property
    def rows(self):
        return self.c.rows

    def read_stats(self):
        if self.stats is None:
            return None
        raw = self.stats.cpu().numpy().tobytes()
        s = Stats.from_buffer_copy(raw)
        return {f: getattr(s, f) for f, _ in Stats._fields_}

    def reset_stats(self):
        if self.stats is not None:
            self.stats.zero_()

    def end_words(self):
        return int(self.offsets[self.rows * self.plan.info.subs_per_row].item()) & 0xFFFFFFFF


def hq_encode(plan: Plan, x: torch.Tensor, s: EncodedStream, append=False, stream=None):
    assert x.dim() == 2 and x.is_cuda
    rows = x.shape[0]
    ld = x.stride(0)
    assert x.stride(1) == 1
    st = lib().hq_encode(plan.handle, C.c_void_p(x.data_ptr()), _dtype_code(x.dtype), rows, ld,
                         C.byref(s.c), int(bool(append)), _stream_handle(stream))
    _check("hq_encode", st)
    return s


def hq_encode_noalloc(plan: Plan, x: torch.Tensor, s: EncodedStream, append=False, stream=None):
    """hq_encode_noalloc: hq_encode with the library's fixed look-back scratch
    (s.scan is not used)."""
    assert x.dim() == 2 and x.is_cuda
    rows = x.shape[0]
    ld = x.stride(0)
    assert x.stride(1) == 1
    st = lib().hq_encode_noalloc(plan.handle, C.c_void_p(x.data_ptr()), _dtype_code(x.dtype), rows,
                                 ld, C.byref(s.c), int(bool(append)), _stream_handle(stream))
    _check("hq_encode_noalloc", st)
    return s


def hq_decode(plan: Plan, s: EncodedStream, row0=0, rows=None, out_dtype=torch.bfloat16, out=None,
              stream=None):
    rows = s.rows - row0 if rows is None else rows
    if out is None:
        out = torch.empty((rows, plan.cols), dtype=out_dtype, device=s.device)
    st = lib().hq_decode(plan.handle, C.byref(s.c), row0, rows, C.c_void_p(out.data_ptr()),
                         _dtype_code(out.dtype), out.stride(0), _stream_handle(stream))
    _check("hq_decode", st)
    return out


def hq_encode_group(plans, xs, streams, stream=None):
    """hq_encode_group: encode xs[i] with plans[i] into streams[i] (whole
    matrices, as hq_encode with append = 0), several per launch."""
    n = len(plans)
    assert len(xs) == n and len(streams) == n and n > 0
    dt = _dtype_code(xs[0].dtype)
    for x in xs:
        assert x.dim() == 2 and x.is_cuda and x.stride(1) == 1 and _dtype_code(x.dtype) == dt
    ph = (C.c_void_p * n)(*[pl.handle for pl in plans])
    xp = (C.c_void_p * n)(*[x.data_ptr() for x in xs])
    rows = (C.c_int64 * n)(*[x.shape[0] for x in xs])
    lds = (C.c_int64 * n)(*[x.stride(0) for x in xs])
    sp = (C.c_void_p * n)(*[C.addressof(s.c) for s in streams])
    st = lib().hq_encode_group(ph, xp, dt, rows, lds, sp, n, _stream_handle(stream))
    _check("hq_encode_group", st)
    return streams


def hq_decode_group(plans, streams, outs, stream=None):
    """hq_decode_group: decode every row of streams[i] with plans[i] into
    outs[i] (bf16 or fp32, one dtype for the group), several per launch."""
    n = len(plans)
    assert len(streams) == n and len(outs) == n and n > 0
    dt = _dtype_code(outs[0].dtype)
    for y in outs:
        assert y.is_cuda and y.stride(1) == 1 and _dtype_code(y.dtype) == dt
    ph = (C.c_void_p * n)(*[pl.handle for pl in plans])
    sp = (C.c_void_p * n)(*[C.addressof(s.c) for s in streams])
    yp = (C.c_void_p * n)(*[y.data_ptr() for y in outs])
    lds = (C.c_int64 * n)(*[y.stride(0) for y in outs])
    st = lib().hq_decode_group(ph, sp, yp, dt, lds, n, _stream_handle(stream))
    _check("hq_decode_group", st)
    return outs


def hq_decode_int8(plan: Plan, s: EncodedStream, row0=0, rows=None, stream=None):
    rows = s.rows - row0 if rows is None else rows
    codes = torch.empty((rows, plan.cols), dtype=torch.int8, device=s.device)
    g = torch.empty((rows, plan.info.tiles_per_row), dtype=torch.float32, device=s.device)
    st = lib().hq_decode_int8(plan.handle, C.byref(s.c), row0, rows, C.c_void_p(codes.data_ptr()),
                              codes.stride(0), C.c_void_p(g.data_ptr()), _stream_handle(stream))
    _check("hq_decode_int8", st)
    return codes, g


def hq_decode_mxfp4(plan: Plan, s: EncodedStream, row0=0, rows=None, stream=None):
    """hq_decode_mxfp4: E2M1 code pairs (uint8, cols / 2 per row) and E8M0
    scale bytes (cols / 32 per row) of the reconstruction."""
    rows = s.rows - row0 if rows is None else rows
    codes = torch.empty((rows, plan.cols // 2), dtype=torch.uint8, device=s.device)
    scales = torch.empty((rows, plan.cols // 32), dtype=torch.uint8, device=s.device)
    st = lib().hq_decode_mxfp4(plan.handle, C.byref(s.c), row0, rows, C.c_void_p(codes.data_ptr()),
                               C.c_void_p(scales.data_ptr()), _stream_handle(stream))
    _check("hq_decode_mxfp4", st)
    return codes, scales


def hq_act_prep_mxfp4(plan: Plan, a: torch.Tensor, stream=None):
    """hq_act_prep_mxfp4: MXFP4 of the rotated activations (codes, scales)."""
    assert a.dim() == 2 and a.dtype == torch.bfloat16 and a.stride(1) == 1
    M = a.shape[0]
    xq = torch.empty((M, plan.cols // 2), dtype=torch.uint8, device=a.device)
    xs = torch.empty((M, plan.cols // 32), dtype=torch.uint8, device=a.device)
    st = lib().hq_act_prep_mxfp4(plan.handle, C.c_void_p(a.data_ptr()), M, a.stride(0),
                                 C.c_void_p(xq.data_ptr()), C.c_void_p(xs.data_ptr()),
                                 _stream_handle(stream))
    _check("hq_act_prep_mxfp4", st)
    return xq, xs


def hq_gemm_mxfp4_blockscaled(plan: Plan, xq, xs, codes, ws, out_dtype=torch.bfloat16, out=None,
                              stream=None):
    M, N = xq.shape[0], codes.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=xq.device)
    st = lib().hq_gemm_mxfp4_blockscaled(plan.handle, C.c_void_p(xq.data_ptr()),
                                         C.c_void_p(xs.data_ptr()), M, C.c_void_p(codes.data_ptr()),
                                         C.c_void_p(ws.data_ptr()), N, C.c_void_p(out.data_ptr()),
                                         _dtype_code(out.dtype), _stream_handle(stream))
    _check("hq_gemm_mxfp4_blockscaled", st)
    return out


def hq_decode_fp8(plan: Plan, s: EncodedStream, row0=0, rows=None, stream=None):
    """hq_decode_fp8: E4M3 code bytes (uint8) and the per-tile factors."""
    rows = s.rows - row0 if rows is None else rows
    codes = torch.empty((rows, plan.cols), dtype=torch.uint8, device=s.device)
    g = torch.empty((rows, plan.info.tiles_per_row), dtype=torch.float32, device=s.device)
    st = lib().hq_decode_fp8(plan.handle, C.byref(s.c), row0, rows, C.c_void_p(codes.data_ptr()),
                             codes.stride(0), C.c_void_p(g.data_ptr()), _stream_handle(stream))
    _check("hq_decode_fp8", st)
    return codes, g


def hq_act_prep_fp8(plan: Plan, a: torch.Tensor, stream=None):
    assert a.dtype == torch.bfloat16 and a.stride(1) == 1
    M = a.shape[0]
    xq = torch.empty((M, plan.cols), dtype=torch.uint8, device=a.device)
    sx = torch.empty((M,), dtype=torch.float32, device=a.device)
    st = lib().hq_act_prep_fp8(plan.handle, C.c_void_p(a.data_ptr()), M, a.stride(0),
                               C.c_void_p(xq.data_ptr()), C.c_void_p(sx.data_ptr()),
                               _stream_handle(stream))
    _check("hq_act_prep_fp8", st)
    return xq, sx


def hq_gemm_fp8_blockscaled(plan: Plan, xq, sx, codes, g, out_dtype=torch.bfloat16, out=None,
                            stream=None):
    M, N = xq.shape[0], codes.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=xq.device)
    st = lib().hq_gemm_fp8_blockscaled(plan.handle, C.c_void_p(xq.data_ptr()),
                                       C.c_void_p(sx.data_ptr()), M,
                                       C.c_void_p(codes.data_ptr()), C.c_void_p(g.data_ptr()), N,
                                       C.c_void_p(out.data_ptr()), _dtype_code(out.dtype),
                                       _stream_handle(stream))
    _check("hq_gemm_fp8_blockscaled", st)
    return out


def hq_act_prep(plan: Plan, a: torch.Tensor, stream=None):
    assert a.dtype == torch.bfloat16 and a.stride(1) == 1
    M = a.shape[0]
    xq = torch.empty((M, plan.cols), dtype=torch.int8, device=a.device)
    sx = torch.empty((M,), dtype=torch.float32, device=a.device)
    st = lib().hq_act_prep(plan.handle, C.c_void_p(a.data_ptr()), M, a.stride(0),
                           C.c_void_p(xq.data_ptr()), C.c_void_p(sx.data_ptr()),
                           _stream_handle(stream))
    _check("hq_act_prep", st)
    return xq, sx


def hq_gemm_int8_blockscaled(plan: Plan, xq, sx, codes, g, out_dtype=torch.bfloat16, out=None,
                             stream=None):
    M, N = xq.shape[0], codes.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=xq.device)
    st = lib().hq_gemm_int8_blockscaled(plan.handle, C.c_void_p(xq.data_ptr()),
                                        C.c_void_p(sx.data_ptr()), M,
                                        C.c_void_p(codes.data_ptr()), C.c_void_p(g.data_ptr()), N,
                                        C.c_void_p(out.data_ptr()), _dtype_code(out.dtype),
                                        _stream_handle(stream))
    _check("hq_gemm_int8_blockscaled", st)
    return out


def hq_gemm_workspace_bytes(plan: Plan, M, N):
    return lib().hq_gemm_workspace_bytes(plan.handle, M, N)


def hq_dequant_gemm_int8(plan: Plan, w: EncodedStream, a: torch.Tensor, out_dtype=torch.bfloat16,
                         workspace=None, out=None, stream=None):
    M, N = a.shape[0], w.rows
    nbytes = hq_gemm_workspace_bytes(plan, M, N)
    if workspace is None:
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=a.device)
    if out is None:
        out = torch.empty((M, N), dtype=out_dtype, device=a.device)
    st = lib().hq_dequant_gemm_int8(plan.handle, C.byref(w.c), N, C.c_void_p(a.data_ptr()), M,
                                    C.c_void_p(out.data_ptr()), _dtype_code(out.dtype),
                                    C.c_void_p(workspace.data_ptr()), workspace.numel(),
                                    _stream_handle(stream))
    _check("hq_dequant_gemm_int8", st)
    return out


def hq_gemv_workspace_bytes(plan: Plan):
    return lib().hq_gemv_workspace_bytes(plan.handle)


def hq_decode_gemv(plan: Plan, s: EncodedStream, x: torch.Tensor, row0=0, rows=None,
                   out_dtype=torch.float32, workspace=None, out=None, stream=None):
    """hq_decode_gemv: y[r] = sum_k W^[row0 + r, k] x[k], the decoded rows
    never materialized.  x: plan.cols values (bf16 or fp32) on the device."""
    rows = s.rows - row0 if rows is None else rows
    assert x.is_cuda and x.dim() == 1 and x.stride(0) == 1 and x.numel() == plan.cols
    if workspace is None:
        workspace = torch.empty(hq_gemv_workspace_bytes(plan), dtype=torch.uint8, device=x.device)
    if out is None:
        out = torch.empty((rows,), dtype=out_dtype, device=x.device)
    st = lib().hq_decode_gemv(plan.handle, C.byref(s.c), row0, rows, C.c_void_p(x.data_ptr()),
                              _dtype_code(x.dtype), C.c_void_p(out.data_ptr()),
                              _dtype_code(out.dtype), C.c_void_p(workspace.data_ptr()),
                              workspace.numel(), _stream_handle(stream))
    _check("hq_decode_gemv", st)
    return out


def hq_attention_workspace_bytes(k_plan: Plan, batch, heads_q, max_tokens):
    return lib().hq_attention_workspace_bytes(k_plan.handle, batch, heads_q, max_tokens)


def hq_decode_attention(k_plan: Plan, k: EncodedStream, v_plan: Plan, v: EncodedStream,
                        q: torch.Tensor, block_table: torch.Tensor, seq_lens: torch.Tensor,
                        block_tokens, scale=None, out_dtype=torch.float32, workspace=None,
                        out=None, stream=None, window_k=None, window_v=None):
    """hq_decode_attention: q [batch, heads_q, 128] (bf16 or fp32) attends
    over the coded cache; block_table int32 [batch, max_blocks] and seq_lens
    int32 [batch] on the device.  window_k / window_v: optional residual
    window rings [batch, W, H_kv * 128] (bf16 or fp32, token t in slot t % W).
    Returns [batch, heads_q, 128]."""
    assert q.is_cuda and q.dim() == 3 and q.shape[2] == 128 and q.is_contiguous()
    assert block_table.dtype == torch.int32 and block_table.is_contiguous() and block_table.dim() == 2
    assert seq_lens.dtype == torch.int32 and seq_lens.is_contiguous()
    batch, heads_q = q.shape[0], q.shape[1]
    max_blocks = block_table.shape[1]
    scale = 128 ** -0.5 if scale is None else scale
    if workspace is None:
        nb = hq_attention_workspace_bytes(k_plan, batch, heads_q, max_blocks * block_tokens)
        workspace = torch.empty(max(nb, 16), dtype=torch.uint8, device=q.device)
    if out is None:
        out = torch.empty((batch, heads_q, 128), dtype=out_dtype, device=q.device)
    window, wk, wv, wt = 0, None, None, 0
    if window_k is not None:
        assert window_v is not None and window_k.shape == window_v.shape and window_k.dim() == 3
        assert window_k.is_contiguous() and window_v.is_contiguous() and window_k.dtype == window_v.dtype
        window, wt = window_k.shape[1], _dtype_code(window_k.dtype)
        wk, wv = C.c_void_p(window_k.data_ptr()), C.c_void_p(window_v.data_ptr())
    st = lib().hq_decode_attention(k_plan.handle, C.byref(k.c), v_plan.handle, C.byref(v.c),
                                   C.c_void_p(q.data_ptr()), _dtype_code(q.dtype), batch, heads_q,
                                   C.c_float(scale), C.c_void_p(block_table.data_ptr()),
                                   max_blocks, block_tokens, C.c_void_p(seq_lens.data_ptr()),
                                   wk, wv, wt, window,
                                   C.c_void_p(out.data_ptr()), _dtype_code(out.dtype),
                                   C.c_void_p(workspace.data_ptr()), workspace.numel(),
                                   _stream_handle(stream))
    _check("hq_decode_attention", st)
    return out


def hq_rice_kstar(count, total):
    return lib().hq_rice_kstar(int(count), int(total))


def hq_calibrated_snr(lattice, rice_k, bps):
    v = C.c_double()
    st = lib().hq_calibrated_snr(lattice, rice_k, C.c_float(bps), C.byref(v))
    _check("hq_calibrated_snr", st)
    return v.value


EXPORTED = ["hq_plan", "hq_plan_destroy", "hq_plan_get_info", "hq_scan_bytes", "hq_encode",
            "hq_encode_noalloc",
            "hq_decode", "hq_encode_group", "hq_decode_group", "hq_decode_int8", "hq_act_prep", "hq_gemm_int8_blockscaled",
            "hq_gemm_workspace_bytes", "hq_dequant_gemm_int8", "hq_gemv_workspace_bytes",
            "hq_decode_gemv", "hq_attention_workspace_bytes", "hq_decode_attention",
            "hq_decode_fp8", "hq_act_prep_fp8", "hq_gemm_fp8_blockscaled",
            "hq_decode_mxfp4", "hq_act_prep_mxfp4", "hq_gemm_mxfp4_blockscaled",
            "hq_rice_kstar",
            "hq_calibrated_snr", "hq_status_string"]
