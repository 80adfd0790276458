"""fp8q: FP8 scaled quantization (paper Sec. 2.2, Eq. 3) and the scaled FP8
GEMM of the FP8 linear layer, as hand-written HIP kernels for MI355X (gfx950).

This module is a thin ctypes binding over the C-ABI of ``libfp8q.so``
(declared in ``include/fp8q.h``): it only marshals arguments.  PyTorch is
used for device memory and the current HIP stream; every step of the
computation runs in the library's kernels.  There is no fallback: if the
library is missing, every call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfp8q.so")

# fp8q_granularity
TENSOR, ROW, COL, BLOCK_1x128, BLOCK_128x1, BLOCK_128x128 = range(6)
OUT_TRANSPOSED = 1
POW2_SCALE = 2
E5M2 = 4                      # quantize flag: E5M2 codes (F_max = 57344)
A_E5M2, B_E5M2 = 1, 2         # gemm_formats operand formats
_STATUS = {0: "FP8Q_OK", -1: "FP8Q_ERR_INVAL", -2: "FP8Q_ERR_UNSUPPORTED",
           -3: "FP8Q_ERR_ALIGN", -4: "FP8Q_ERR_HIP"}
# the entry points of include/fp8q.h
EXPORTS = ("fp8q_scales_count", "fp8q_quantize", "fp8q_quantize_dual",
           "fp8q_gemm", "fp8q_gemm_grouped", "fp8q_gemm_formats", "fp8q_gemm_pow2", "fp8q_gemm_quantized",
           "fp8q_gemm_splitk_workspace", "fp8q_gemm_splitk",
           "fp8q_calibrate_clip_workspace", "fp8q_calibrate_clip", "fp8q_calibrate_clip_noalloc",
           "fp8q_cast_f32",
           "fp8q_cast_f32_e5m2", "fp8q_status_string")


MAX_GROUP = 8


class GemmProblem(ctypes.Structure):
    """fp8q_gemm_problem of include/fp8q.h."""
    _fields_ = [("A", ctypes.c_void_p), ("sA", ctypes.c_void_p), ("lda", ctypes.c_int64),
                ("B", ctypes.c_void_p), ("sB", ctypes.c_void_p), ("ldb", ctypes.c_int64),
                ("C", ctypes.c_void_p), ("ldc", ctypes.c_int64),
                ("M", ctypes.c_int64), ("N", ctypes.c_int64)]


class ClipConfig(ctypes.Structure):
    """fp8q_clip_config (include/fp8q.h)."""
    _fields_ = [(n, ctypes.c_double) for n in ("c_low_ref", "c_high_ref", "l_min", "l_max",
                                                "h_min", "h_max", "step", "delta_l", "delta_h")]


class ClipResult(ctypes.Structure):
    """fp8q_clip_result (include/fp8q.h)."""
    _fields_ = ([(n, ctypes.c_double) for n in ("l_new", "h_new", "l_star", "h_star", "alpha_low",
                                                 "rho_bf16", "rho_fp8")]
                + [("n_neg", ctypes.c_int64), ("n_pos", ctypes.c_int64),
                   ("l_updated", ctypes.c_int32), ("h_updated", ctypes.c_int32)])


# Sec. 4 settings, with the GRPO experiments' reference bounds (Sec. 5.1).
PAPER_CLIP_CONFIG = dict(c_low_ref=0.8, c_high_ref=1.24, l_min=0.5, l_max=0.9, h_min=1.2,
                         h_max=2.0, step=0.02, delta_l=0.05, delta_h=0.1)


class Fp8qError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__("%s: %s" % (what, status_string(status)))


_lib = None


def lib():
    """Load libfp8q.so (built by __graft_entry__.build()); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libfp8q.so is not built (%s); run "
                              "__graft_entry__.build()" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        p, i64, i32, u32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_uint
        L.fp8q_scales_count.argtypes = [i64, i64, i32, u32]
        L.fp8q_scales_count.restype = i64
        L.fp8q_quantize.argtypes = [p, i64, i64, i64, i32, u32, p, i64, p, p]
        L.fp8q_quantize.restype = i32
        L.fp8q_quantize_dual.argtypes = [p, i64, i64, i64, u32, p, i64, p, p, i64, p, p]
        L.fp8q_quantize_dual.restype = i32
        L.fp8q_gemm.argtypes = [p, p, i32, i64, p, p, i32, i64, i64, i64, i64,
                                p, i64, p]
        L.fp8q_gemm.restype = i32
        L.fp8q_gemm_grouped.argtypes = [ctypes.POINTER(GemmProblem), i32, i32, i32, i64, p]
        L.fp8q_gemm_grouped.restype = i32
        L.fp8q_gemm_formats.argtypes = [p, p, i32, i64, p, p, i32, i64, i64, i64, i64, u32, p, i64, p]
        L.fp8q_gemm_formats.restype = i32
        L.fp8q_gemm_pow2.argtypes = [p, p, i32, i64, p, p, i32, i64, i64, i64, i64, p, i64, p]
        L.fp8q_gemm_pow2.restype = i32
        L.fp8q_gemm_quantized.argtypes = [p, p, i32, i64, p, p, i32, i64, i64,
                                          i64, i64, p, i64, p, p]
        L.fp8q_gemm_quantized.restype = i32
        L.fp8q_gemm_splitk_workspace.argtypes = [i64, i64, i64]
        L.fp8q_gemm_splitk_workspace.restype = i64
        L.fp8q_gemm_splitk.argtypes = [p, p, i32, i64, p, p, i32, i64, i64, i64, i64,
                                       p, i64, p, i64, p]
        L.fp8q_gemm_splitk.restype = i32
        L.fp8q_calibrate_clip_workspace.argtypes = [i64]
        L.fp8q_calibrate_clip_workspace.restype = i64
        d = ctypes.c_double
        L.fp8q_calibrate_clip.argtypes = [p, p, p, p, p, i64, d, d, ctypes.POINTER(ClipConfig),
                                          p, i64, p, p]
        L.fp8q_calibrate_clip.restype = i32
        L.fp8q_calibrate_clip_noalloc.argtypes = [p, p, p, p, p, i64, d, d, ctypes.POINTER(ClipConfig), p, p]
        L.fp8q_calibrate_clip_noalloc.restype = i32
        L.fp8q_cast_f32.argtypes = [p, i64, ctypes.c_float, p, p]
        L.fp8q_cast_f32_e5m2.argtypes = [p, i64, ctypes.c_float, p, p]
        L.fp8q_cast_f32_e5m2.restype = i32
        L.fp8q_cast_f32.restype = i32
        L.fp8q_status_string.argtypes = [i32]
        L.fp8q_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(status):
    try:
        return lib().fp8q_status_string(status).decode()
    except ImportError:
        return _STATUS.get(status, str(status))


def _check(status, what):
    if status != 0:
        raise Fp8qError(status, what)


def _stream(t):
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ld(t):
    """Leading dimension of a row-major 2-D tensor (unit column stride)."""
    if t.dim() != 2 or t.stride(1) != 1:
        raise ValueError("expected a row-major 2-D tensor")
    return t.stride(0)


def _matrix(t, dtype, what, shape=None, device=None):
    """t as a row-major 2-D CUDA tensor of dtype (and of shape / on device
    when given): the kernels read and write exactly that region, so a
    tensor of another shape would be read or written past its end."""
    if not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda or t.dim() != 2:
        raise ValueError("%s must be a 2-D %s CUDA tensor" % (what, dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s must have shape %s, not %s" % (what, tuple(shape), tuple(t.shape)))
    if device is not None and t.device != device:
        raise ValueError("%s must be on %s" % (what, device))
    _ld(t)
    return t


def _vector(t, dtype, n, what, device):
    """t as a contiguous CUDA tensor of dtype with at least n elements."""
    if (not isinstance(t, torch.Tensor) or t.dtype != dtype or not t.is_cuda or not t.is_contiguous()
            or t.device != device):
        raise ValueError("%s must be a contiguous %s tensor on %s" % (what, dtype, device))
    if t.numel() < n:
        raise ValueError("%s holds %d elements, %d needed" % (what, t.numel(), n))
    return t


def _operands(a, sa, ga, b, sb, gb):
    """The checks shared by the GEMM entry points: FP8 codes a [M, K] and b
    [N, K] on one device, and scale arrays holding at least the counts
    their granularities give for those shapes; returns M, N, K."""
    _matrix(a, torch.uint8, "a")
    _matrix(b, torch.uint8, "b", device=a.device)
    M, K = a.shape
    N, K2 = b.shape
    if K != K2:
        raise ValueError("contraction sizes differ")
    _vector(sa, torch.float32, max(scales_count(M, K, ga), 0), "sa", a.device)
    _vector(sb, torch.float32, max(scales_count(N, K, gb), 0), "sb", a.device)
    return M, N, K


def scales_count(rows, cols, granularity, transposed=False):
    n = lib().fp8q_scales_count(rows, cols, granularity, OUT_TRANSPOSED if transposed else 0)
    if n < 0:
        raise ValueError("invalid quantization shape or granularity")
    return n


def quantize(x, granularity, transposed=False, codes=None, scales=None, pow2=False, e5m2=False):
    """Eq. 3 per scaling unit on a bf16 CUDA tensor x[rows, cols].

    Returns (codes, scales): codes uint8 (OCP E4M3 bytes) [rows, cols], or
    [cols, rows] when `transposed`; scales fp32 1-D in the layout of
    include/fp8q.h.  pow2: power-of-two scales (FP8Q_POW2_SCALE); e5m2:
    E5M2 codes (FP8Q_E5M2).
    """
    _matrix(x, torch.bfloat16, "x")
    rows, cols = x.shape
    oshape = (cols, rows) if transposed else (rows, cols)
    n = scales_count(rows, cols, granularity, transposed)
    if codes is None:
        codes = torch.empty(oshape, dtype=torch.uint8, device=x.device)
    _matrix(codes, torch.uint8, "codes", oshape, x.device)
    if scales is None:
        scales = torch.empty(n, dtype=torch.float32, device=x.device)
    _vector(scales, torch.float32, n, "scales", x.device)
    st = lib().fp8q_quantize(x.data_ptr(), rows, cols, _ld(x), granularity,
                             (OUT_TRANSPOSED if transposed else 0) | (POW2_SCALE if pow2 else 0)
                             | (E5M2 if e5m2 else 0),
                             codes.data_ptr(), _ld(codes), scales.data_ptr(),
                             _stream(x))
    _check(st, "fp8q_quantize")
    return codes, scales


def quantize_dual(x, codes_r=None, scales_r=None, codes_t=None, scales_t=None, pow2=False, e5m2=False):
    """Both backward-pass layouts of a bf16 CUDA tensor x[rows, cols] from
    one read: (codes_r, scales_r) = quantize(x, BLOCK_1x128) and
    (codes_t, scales_t) = quantize(x, BLOCK_128x1, transposed=True), with
    the same pow2 / e5m2 options."""
    _matrix(x, torch.bfloat16, "x")
    rows, cols = x.shape
    nr, nt = scales_count(rows, cols, BLOCK_1x128), scales_count(rows, cols, BLOCK_128x1, True)
    if codes_r is None:
        codes_r = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    if scales_r is None:
        scales_r = torch.empty(nr, dtype=torch.float32, device=x.device)
    if codes_t is None:
        codes_t = torch.empty((cols, rows), dtype=torch.uint8, device=x.device)
    if scales_t is None:
        scales_t = torch.empty(nt, dtype=torch.float32, device=x.device)
    _matrix(codes_r, torch.uint8, "codes_r", (rows, cols), x.device)
    _matrix(codes_t, torch.uint8, "codes_t", (cols, rows), x.device)
    _vector(scales_r, torch.float32, nr, "scales_r", x.device)
    _vector(scales_t, torch.float32, nt, "scales_t", x.device)
    st = lib().fp8q_quantize_dual(x.data_ptr(), rows, cols, _ld(x),
                                  (POW2_SCALE if pow2 else 0) | (E5M2 if e5m2 else 0),
                                  codes_r.data_ptr(), _ld(codes_r),
                                  scales_r.data_ptr(), codes_t.data_ptr(),
                                  _ld(codes_t), scales_t.data_ptr(), _stream(x))
    _check(st, "fp8q_quantize_dual")
    return codes_r, scales_r, codes_t, scales_t


def gemm(a, sa, ga, b, sb, gb, out=None):
    """C[M, N] = dequant(a)[M, K] @ dequant(b)[N, K]^T in bf16.

    a, b: uint8 E4M3 codes, K contiguous; sa, sb: fp32 scales for the
    granularities ga, gb (pairs listed in include/fp8q.h).
    """
    M, N, K = _operands(a, sa, ga, b, sb, gb)
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    _matrix(out, torch.bfloat16, "out", (M, N), a.device)
    st = lib().fp8q_gemm(a.data_ptr(), sa.data_ptr(), ga, _ld(a),
                         b.data_ptr(), sb.data_ptr(), gb, _ld(b), M, N, K,
                         out.data_ptr(), _ld(out), _stream(a))
    _check(st, "fp8q_gemm")
    return out


def gemm_splitk_workspace(M, N, K):
    """Bytes of workspace gemm_splitk needs for an M x N x K problem (0 when
    it does not split K)."""
    need = lib().fp8q_gemm_splitk_workspace(M, N, K)
    if need < 0:
        raise ValueError("invalid GEMM size")
    return need


def gemm_splitk(a, sa, ga, b, sb, gb, out=None, workspace=None):
    """gemm for skinny problems with each output tile's K blocks split over
    several workgroups (fp8q_gemm_splitk).  workspace: a uint8 CUDA tensor
    of at least gemm_splitk_workspace(M, N, K) bytes, zero-filled before its
    first use (a new zero-filled one when None); calls sharing it must be
    ordered (one stream)."""
    M, N, K = _operands(a, sa, ga, b, sb, gb)
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    _matrix(out, torch.bfloat16, "out", (M, N), a.device)
    need = gemm_splitk_workspace(M, N, K)
    if workspace is None:
        workspace = torch.zeros(max(need, 16), dtype=torch.uint8, device=a.device)
    _vector(workspace, torch.uint8, need, "workspace", a.device)
    st = lib().fp8q_gemm_splitk(a.data_ptr(), sa.data_ptr(), ga, _ld(a),
                                b.data_ptr(), sb.data_ptr(), gb, _ld(b), M, N, K,
                                out.data_ptr(), _ld(out), workspace.data_ptr(),
                                workspace.numel(), _stream(a))
    _check(st, "fp8q_gemm_splitk")
    return out


def gemm_grouped(problems, ga, gb, outs=None):
    """Several gemm() problems in one launch (fp8q_gemm_grouped).

    problems: list of (a, sa, b, sb) with one K and the granularities ga,
    gb for all (the a's may be the same tensor); returns the bf16 outputs
    (or fills `outs`)."""
    if not 1 <= len(problems) <= MAX_GROUP:
        raise ValueError("1 .. %d problems" % MAX_GROUP)
    K = problems[0][0].shape[1]
    dev = problems[0][0].device
    for a, sa, b, sb in problems:
        _operands(a, sa, ga, b, sb, gb)
        if a.shape[1] != K or a.device != dev:
            raise ValueError("every problem must have the same K and device")
    if outs is None:
        outs = [torch.empty((a.shape[0], b.shape[0]), dtype=torch.bfloat16, device=a.device)
                for a, _, b, _ in problems]
    if len(outs) != len(problems):
        raise ValueError("one output per problem")
    arr = (GemmProblem * len(problems))()
    for i, ((a, sa, b, sb), c) in enumerate(zip(problems, outs)):
        _matrix(c, torch.bfloat16, "outs[%d]" % i, (a.shape[0], b.shape[0]), dev)
        arr[i] = GemmProblem(a.data_ptr(), sa.data_ptr(), _ld(a), b.data_ptr(), sb.data_ptr(), _ld(b),
                             c.data_ptr(), _ld(c), a.shape[0], b.shape[0])
    st = lib().fp8q_gemm_grouped(arr, len(problems), ga, gb, K, _stream(problems[0][0]))
    _check(st, "fp8q_gemm_grouped")
    return outs


def gemm_formats(a, sa, ga, b, sb, gb, formats, out=None):
    """gemm() with E5M2 codes for A (formats & A_E5M2) and/or B (formats &
    B_E5M2): the backward pairs (1x128, 128x128) and (1x128, 1x128)."""
    M, N, K = _operands(a, sa, ga, b, sb, gb)
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    _matrix(out, torch.bfloat16, "out", (M, N), a.device)
    st = lib().fp8q_gemm_formats(a.data_ptr(), sa.data_ptr(), ga, _ld(a),
                                 b.data_ptr(), sb.data_ptr(), gb, _ld(b), M, N, K,
                                 formats, out.data_ptr(), _ld(out), _stream(a))
    _check(st, "fp8q_gemm_formats")
    return out


def gemm_pow2(a, sa, ga, b, sb, gb, out=None):
    """gemm() for operands quantized with power-of-two scales (pow2=True):
    the block scales enter the matrix instruction as exponents."""
    M, N, K = _operands(a, sa, ga, b, sb, gb)
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=a.device)
    _matrix(out, torch.bfloat16, "out", (M, N), a.device)
    st = lib().fp8q_gemm_pow2(a.data_ptr(), sa.data_ptr(), ga, _ld(a),
                              b.data_ptr(), sb.data_ptr(), gb, _ld(b), M, N, K,
                              out.data_ptr(), _ld(out), _stream(a))
    _check(st, "fp8q_gemm_pow2")
    return out


def gemm_quantized(a, sa, ga, b, sb, gb, codes=None, scales=None):
    """The GEMM of gemm() with its bf16 output quantized per 1x128 block
    (the next layer's activation operand), in one kernel.  Returns (codes
    uint8 [M, N], scales fp32 in the 1x128 layout), exactly
    quantize(gemm(a, sa, ga, b, sb, gb), BLOCK_1x128)."""
    M, N, K = _operands(a, sa, ga, b, sb, gb)
    n = scales_count(M, N, BLOCK_1x128)
    if codes is None:
        codes = torch.empty((M, N), dtype=torch.uint8, device=a.device)
    if scales is None:
        scales = torch.empty(n, dtype=torch.float32, device=a.device)
    _matrix(codes, torch.uint8, "codes", (M, N), a.device)
    _vector(scales, torch.float32, n, "scales", a.device)
    st = lib().fp8q_gemm_quantized(a.data_ptr(), sa.data_ptr(), ga, _ld(a),
                                   b.data_ptr(), sb.data_ptr(), gb, _ld(b), M, N, K,
                                   codes.data_ptr(), _ld(codes), scales.data_ptr(),
                                   _stream(a))
    _check(st, "fp8q_gemm_quantized")
    return codes, scales


def calibrate_clip(adv, w_tis, pi_sampler, r_bf16, r_fp8, l_old, h_old, config=None,
                   workspace=None, result=None, read=True):
    """Calibrated Clipping (Alg. 1) on the GPU.  The five per-token inputs
    are contiguous float32 CUDA tensors of one batch; config maps the
    fields of ClipConfig (default: the paper's).  Returns the result as a
    dict (reading it back waits for the kernels); `result` may be a uint8
    CUDA tensor of ctypes.sizeof(ClipResult) bytes to write into, and with
    read=False nothing is read back (the call returns None)."""
    ts = (adv, w_tis, pi_sampler, r_bf16, r_fp8)
    n = adv.numel()
    for t in ts:
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous() or t.numel() != n:
            raise ValueError("inputs must be contiguous float32 CUDA tensors of one length")
    cfg = ClipConfig(**(config or PAPER_CLIP_CONFIG))
    need = lib().fp8q_calibrate_clip_workspace(n)
    if need < 0:
        raise ValueError("empty batch")
    if workspace is None:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=adv.device)
    if result is None:
        result = torch.empty(ctypes.sizeof(ClipResult), dtype=torch.uint8, device=adv.device)
    _vector(workspace, torch.uint8, need, "workspace", adv.device)
    _vector(result, torch.uint8, ctypes.sizeof(ClipResult), "result", adv.device)
    st = lib().fp8q_calibrate_clip(*(t.data_ptr() for t in ts), n, float(l_old), float(h_old),
                                   ctypes.byref(cfg), workspace.data_ptr(), workspace.numel(),
                                   result.data_ptr(), _stream(adv))
    _check(st, "fp8q_calibrate_clip")
    if not read:
        return None
    r = ClipResult.from_buffer_copy(result.cpu().numpy().tobytes())
    return {name: getattr(r, name) for name, _ in ClipResult._fields_}


def calibrate_clip_noalloc(adv, w_tis, pi_sampler, r_bf16, r_fp8, l_old, h_old, config=None,
                           result=None, read=True):
    """calibrate_clip() through fp8q_calibrate_clip_noalloc: no workspace,
    the partial sums go to the library's own device array (calls on one
    device must not overlap).  `result` and `read` as for calibrate_clip."""
    ts = (adv, w_tis, pi_sampler, r_bf16, r_fp8)
    n = adv.numel()
    for t in ts:
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous() or t.numel() != n:
            raise ValueError("inputs must be contiguous float32 CUDA tensors of one length")
    cfg = ClipConfig(**(config or PAPER_CLIP_CONFIG))
    if result is None:
        result = torch.empty(ctypes.sizeof(ClipResult), dtype=torch.uint8, device=adv.device)
    _vector(result, torch.uint8, ctypes.sizeof(ClipResult), "result", adv.device)
    st = lib().fp8q_calibrate_clip_noalloc(*(t.data_ptr() for t in ts), n, float(l_old), float(h_old),
                                           ctypes.byref(cfg), result.data_ptr(), _stream(adv))
    _check(st, "fp8q_calibrate_clip_noalloc")
    if not read:
        return None
    r = ClipResult.from_buffer_copy(result.cpu().numpy().tobytes())
    return {name: getattr(r, name) for name, _ in ClipResult._fields_}


def cast_f32(x, scale, codes=None, e5m2=False):
    """Q_FP8(RN32(x / scale)) elementwise on an fp32 CUDA tensor (E4M3, or
    E5M2 codes)."""
    if x.dtype != torch.float32 or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous fp32 CUDA tensor")
    if codes is None:
        codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device)
    _vector(codes, torch.uint8, x.numel(), "codes", x.device)
    fn = lib().fp8q_cast_f32_e5m2 if e5m2 else lib().fp8q_cast_f32
    st = fn(x.data_ptr(), x.numel(), float(scale), codes.data_ptr(), _stream(x))
    _check(st, "fp8q_cast_f32_e5m2" if e5m2 else "fp8q_cast_f32")
    return codes
