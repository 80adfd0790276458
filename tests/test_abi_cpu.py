"""The C-ABI library loads without a GPU, exports every entry point that
include/fp8q.h declares, and rejects bad arguments on the host before any
HIP call (so no GPU is touched here)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fp8q.h")

fp8q = pytest.importorskip("paper_2609_22870_amd")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(fp8q.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    return fp8q.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fp8q_\w+)\s*\(", text)))


def test_header_declares_the_abi():
    assert declared_functions() == sorted(fp8q.EXPORTS)


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name
    out = os.popen("nm -D --defined-only %s" % fp8q.LIB_PATH).read()
    for name in declared_functions():
        assert re.search(r"\bT %s\b" % name, out), name


def test_status_strings(L):
    for s in (0, -1, -2, -3, -4):
        assert fp8q.status_string(s).startswith("FP8Q_")


@pytest.mark.parametrize("rows,cols,g,t,want", [
    (256, 384, fp8q.TENSOR, False, 1),
    (256, 384, fp8q.ROW, False, 256),
    (256, 384, fp8q.ROW, True, 256),
    (256, 384, fp8q.COL, False, 384),
    (256, 384, fp8q.BLOCK_1x128, False, 256 * 3),
    (256, 384, fp8q.BLOCK_1x128, True, 256 * 3),
    (256, 384, fp8q.BLOCK_128x1, False, 2 * 384),
    (256, 384, fp8q.BLOCK_128x1, True, 2 * 384),
    (256, 384, fp8q.BLOCK_128x128, False, 6),
    (256, 384, fp8q.BLOCK_128x128, True, 6),
    (0, 384, fp8q.TENSOR, False, -1),
    (256, 384, 9, False, -1),
])
def test_scales_count(L, rows, cols, g, t, want):
    assert L.fp8q_scales_count(rows, cols, g, 1 if t else 0) == want


FAKE = 0x10000  # never dereferenced: every case below fails validation


def quant(L, x=FAKE, rows=256, cols=256, ldx=256, g=3, flags=0, codes=FAKE,
          ldc=256, scales=FAKE):
    return L.fp8q_quantize(x, rows, cols, ldx, g, flags, codes, ldc, scales, None)


def test_quantize_rejections(L):
    assert quant(L, x=None) == -1
    assert quant(L, codes=None) == -1
    assert quant(L, scales=None) == -1
    assert quant(L, rows=0) == -1
    assert quant(L, cols=-5) == -1
    assert quant(L, g=6) == -1
    assert quant(L, flags=8) == -1                           # unknown flag bit
    assert quant(L, ldx=128) == -1
    assert quant(L, ldc=128) == -1
    assert quant(L, cols=200, ldx=200, ldc=208) == -2        # cols % 16
    assert quant(L, cols=272, ldx=272, ldc=272) == -2        # 1x128 needs cols % 128
    assert quant(L, rows=200, g=4) == -2                     # 128x1 needs rows % 128
    assert quant(L, rows=200, g=5) == -2
    assert quant(L, rows=200, g=1, flags=1, ldc=208) == -2   # transposed: rows % 16
    assert quant(L, rows=65535 * 128 + 128, g=5) == -2       # row limit
    assert quant(L, rows=65535 * 128 + 128, g=3) == -2
    assert quant(L, x=FAKE + 2) == -3
    assert quant(L, codes=FAKE + 8) == -3
    assert quant(L, scales=FAKE + 2) == -3
    assert quant(L, ldx=260) == -3
    assert quant(L, ldc=264) == -3


def gemm(L, A=FAKE, sA=FAKE, gA=3, lda=256, B=FAKE, sB=FAKE, gB=5, ldb=256,
         M=256, N=256, K=256, C=FAKE, ldc=256):
    return L.fp8q_gemm(A, sA, gA, lda, B, sB, gB, ldb, M, N, K, C, ldc, None)


def test_gemm_rejections(L):
    assert gemm(L, A=None) == -1
    assert gemm(L, sB=None) == -1
    assert gemm(L, C=None) == -1
    assert gemm(L, M=0) == -1
    assert gemm(L, lda=128) == -1
    assert gemm(L, ldc=100) == -1
    assert gemm(L, gA=7) == -1
    assert gemm(L, gA=0, gB=1) == -2
    assert gemm(L, gA=5, gB=5) == -2
    assert gemm(L, gA=3, gB=4) == -2
    assert gemm(L, K=200, lda=256, ldb=256) == -2
    assert gemm(L, N=200, ldc=256) == -2                     # 128x128 B needs N % 128
    assert gemm(L, A=FAKE + 4) == -3
    assert gemm(L, lda=264) == -3
    assert gemm(L, C=FAKE + 2) == -3
    assert gemm(L, ldc=258) == -3


def gemm_sk(L, ws=FAKE, ws_bytes=1 << 30, **kw):
    args = dict(A=FAKE, sA=FAKE, gA=3, lda=12288, B=FAKE, sB=FAKE, gB=5, ldb=12288, M=256, N=4096, K=12288,
                C=FAKE, ldc=4096)
    args.update(kw)
    return L.fp8q_gemm_splitk(*args.values(), ws, ws_bytes, None)


def test_gemm_splitk_workspace_sizes(L):
    """Split counts: the largest power of two up to 8 with tiles x S <= 256
    and at least four K blocks per split; the workspace is one counter per
    tile padded to 256 bytes, then S fp32 128 x 128 partial tiles per tile."""
    ws = L.fp8q_gemm_splitk_workspace
    assert ws(256, 4096, 12288) == 256 + 64 * 4 * 128 * 128 * 4       # decode down: 64 tiles, S = 4
    assert ws(256, 12288, 4096) == 0                                   # 192 tiles: not split
    assert ws(200, 384, 1024) == 256 + 6 * 2 * 65536                   # 8 K blocks: S = 2
    assert ws(200, 384, 2048) == 256 + 6 * 4 * 65536
    assert ws(200, 384, 4096) == 256 + 6 * 8 * 65536
    assert ws(128, 128, 384) == 0                                      # 3 K blocks
    assert ws(128, 128, 200) == 0                                      # K not whole blocks
    assert ws(0, 128, 1024) == -1 and ws(128, -1, 1024) == -1 and ws(128, 128, 1 << 31) == -1


def test_gemm_splitk_rejections(L):
    assert gemm_sk(L, A=None) == -1
    assert gemm_sk(L, gA=3, gB=4) == -2
    assert gemm_sk(L, ws=None) == -1                                  # splits and needs one
    assert gemm_sk(L, ws_bytes=L.fp8q_gemm_splitk_workspace(256, 4096, 12288) - 1) == -1
    assert gemm_sk(L, ws=FAKE + 8) == -3
    assert gemm_sk(L, C=FAKE + 2) == -3


def test_gemm_pow2_rejections(L):
    def gp(**kw):
        args = dict(A=FAKE, sA=FAKE, gA=3, lda=256, B=FAKE, sB=FAKE, gB=5, ldb=256, M=256, N=256, K=256,
                    C=FAKE, ldc=256)
        args.update(kw)
        return L.fp8q_gemm_pow2(*args.values(), None)
    assert gp(A=None) == -1
    assert gp(M=0) == -1
    assert gp(gA=0, gB=0) == -2                              # only 1x128 x 128x128
    assert gp(gA=3, gB=3) == -2
    assert gp(N=200, ldc=256) == -2
    assert gp(K=200) == -2
    assert gp(A=FAKE + 4) == -3
    assert gp(ldc=258) == -3


def test_scales_count_pow2_and_e5m2_flags(L):
    assert L.fp8q_scales_count(256, 384, fp8q.BLOCK_1x128, 2) == 256 * 3
    assert L.fp8q_scales_count(256, 384, fp8q.BLOCK_1x128, 3) == 256 * 3
    assert L.fp8q_scales_count(256, 384, fp8q.BLOCK_1x128, 4) == 256 * 3    # E5M2
    assert L.fp8q_scales_count(256, 384, fp8q.BLOCK_1x128, 7) == 256 * 3
    assert L.fp8q_scales_count(256, 384, fp8q.BLOCK_1x128, 8) == -1


def grouped(L, probs, gA=3, gB=5, K=256, count=None):
    arr = (fp8q.GemmProblem * max(1, len(probs)))()
    for i, kw in enumerate(probs):
        d = dict(A=FAKE, sA=FAKE, lda=256, B=FAKE, sB=FAKE, ldb=256, C=FAKE, ldc=512, M=256, N=512)
        d.update(kw)
        arr[i] = fp8q.GemmProblem(**d)
    return L.fp8q_gemm_grouped(arr, len(probs) if count is None else count, gA, gB, K, None)


def test_gemm_grouped_rejections(L):
    assert L.fp8q_gemm_grouped(None, 1, 3, 5, 256, None) == -1
    assert grouped(L, [{}], count=0) == -1
    assert grouped(L, [{}] * 9) == -1                        # more than FP8Q_MAX_GROUP
    assert grouped(L, [{}, dict(B=None)]) == -1              # a bad second problem
    assert grouped(L, [{}, dict(M=0)]) == -1
    assert grouped(L, [{}, dict(ldc=256)]) == -1             # ldc < N
    assert grouped(L, [{}], gA=3, gB=3) == -2                # the wgrad pair is not grouped
    assert grouped(L, [{}], K=200) == -2
    assert grouped(L, [{}, dict(N=200, ldc=256)]) == -2      # 128x128 B needs N % 128
    assert grouped(L, [dict(M=1 << 24, lda=256)]) == -2      # A spans 4 GiB
    assert grouped(L, [{}, dict(C=FAKE + 2)]) == -3


def gemm_f(L, formats, **kw):
    args = dict(A=FAKE, sA=FAKE, gA=3, lda=256, B=FAKE, sB=FAKE, gB=5, ldb=256, M=256, N=256, K=256)
    args.update(kw)
    return L.fp8q_gemm_formats(*args.values(), formats, FAKE, 256, None)


def test_gemm_formats_rejections(L):
    assert gemm_f(L, 4) == -1                                # unknown format bit
    assert gemm_f(L, 1, A=None) == -1
    assert gemm_f(L, 1, gA=0, gB=0) == -2                    # E5M2 only for the blockwise pairs
    assert gemm_f(L, 2, gA=1, gB=1) == -2
    assert gemm_f(L, 3, N=200) == -2
    assert gemm_f(L, 1, A=FAKE + 4) == -3
    assert gemm_f(L, 1, gA=3, gB=3, lda=264) == -3


@pytest.mark.parametrize("name", ["fp8q_cast_f32", "fp8q_cast_f32_e5m2"])
def test_cast_rejections(L, name):
    fn = getattr(L, name)
    assert fn(None, 10, 1.0, FAKE, None) == -1
    assert fn(FAKE, 0, 1.0, FAKE, None) == -1
    assert fn(FAKE, 10, 0.0, FAKE, None) == -1
    assert fn(FAKE + 1, 10, 1.0, FAKE, None) == -3


def test_cast_rejections_e4m3(L):
    assert L.fp8q_cast_f32(None, 10, 1.0, FAKE, None) == -1
    assert L.fp8q_cast_f32(FAKE, 0, 1.0, FAKE, None) == -1
    assert L.fp8q_cast_f32(FAKE, 10, 0.0, FAKE, None) == -1
    assert L.fp8q_cast_f32(FAKE, 10, -1.0, FAKE, None) == -1
    assert L.fp8q_cast_f32(FAKE + 1, 10, 1.0, FAKE, None) == -3


def test_no_cpu_fallback_when_library_missing(monkeypatch, tmp_path):
    """Without the built library the binding raises instead of computing."""
    monkeypatch.setattr(fp8q, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(fp8q, "_lib", None)
    with pytest.raises(ImportError):
        fp8q.lib()


def dual(L, x=FAKE, rows=256, cols=256, ldx=256, flags=0, cr=FAKE, ldr=256, sr=FAKE,
         ct=FAKE, ldt=256, st=FAKE):
    return L.fp8q_quantize_dual(x, rows, cols, ldx, flags, cr, ldr, sr, ct, ldt, st, None)


def test_quantize_dual_rejections(L):
    assert dual(L, x=None) == -1
    assert dual(L, flags=1) == -1                            # transposition is implied, not a flag
    assert dual(L, flags=8) == -1
    assert dual(L, flags=6, rows=272, ldt=272) == -2         # pow2 | E5M2 accepted, shape checked
    assert dual(L, cr=None) == -1
    assert dual(L, st=None) == -1
    assert dual(L, rows=0) == -1
    assert dual(L, ldx=128) == -1
    assert dual(L, ldr=128) == -1
    assert dual(L, rows=384, ldt=256) == -1                  # ldt < rows
    assert dual(L, rows=272, ldt=272) == -2                  # rows % 128
    assert dual(L, cols=400, ldx=400, ldr=400) == -2         # cols % 128
    assert dual(L, x=FAKE + 2) == -3
    assert dual(L, ct=FAKE + 8) == -3
    assert dual(L, sr=FAKE + 1) == -3
    assert dual(L, ldx=260) == -3
    assert dual(L, ldt=264) == -3


def gemm_q(L, A=FAKE, sA=FAKE, gA=3, lda=256, B=FAKE, sB=FAKE, gB=5, ldb=256,
           M=256, N=256, K=256, q=FAKE, ldq=256, s=FAKE):
    return L.fp8q_gemm_quantized(A, sA, gA, lda, B, sB, gB, ldb, M, N, K, q, ldq, s, None)


def test_gemm_quantized_rejections(L):
    assert gemm_q(L, A=None) == -1
    assert gemm_q(L, q=None) == -1
    assert gemm_q(L, s=None) == -1
    assert gemm_q(L, M=0) == -1
    assert gemm_q(L, ldq=128) == -1
    assert gemm_q(L, gA=0, gB=0) == -2                       # only 1x128 x 128x128
    assert gemm_q(L, gA=3, gB=3) == -2
    assert gemm_q(L, K=200, lda=256, ldb=256) == -2
    assert gemm_q(L, N=200, ldq=256) == -2
    assert gemm_q(L, q=FAKE + 8) == -3
    assert gemm_q(L, ldq=264) == -3
    assert gemm_q(L, s=FAKE + 2) == -3


def calib(L, ptrs=(FAKE,) * 5, n=4096, cfg=None, ws=FAKE, ws_bytes=1 << 30, res=FAKE):
    import ctypes
    c = fp8q.ClipConfig(**(cfg or fp8q.PAPER_CLIP_CONFIG))
    return L.fp8q_calibrate_clip(*ptrs, n, 0.6, 1.8, ctypes.byref(c), ws, ws_bytes, res, None)


def test_calibrate_clip_workspace_and_rejections(L):
    assert L.fp8q_calibrate_clip_workspace(0) == -1
    assert L.fp8q_calibrate_clip_workspace(1) > 0
    assert L.fp8q_calibrate_clip_workspace(1 << 30) >= L.fp8q_calibrate_clip_workspace(1 << 20)
    P = fp8q.PAPER_CLIP_CONFIG
    assert calib(L, ptrs=(None,) + (FAKE,) * 4) == -1
    assert calib(L, ws=None) == -1
    assert calib(L, res=None) == -1
    assert calib(L, n=0) == -1
    assert calib(L, cfg=dict(P, step=0.0)) == -1
    assert calib(L, cfg=dict(P, l_max=0.4)) == -1                 # inverted interval
    assert calib(L, cfg=dict(P, l_max=0.91)) == -1                # not whole steps
    assert calib(L, ws_bytes=8) == -1
    assert calib(L, cfg=dict(P, l_min=0.42)) == -2                # 25 lower points
    assert calib(L, cfg=dict(P, h_max=2.16)) == -2                # 49 upper points
    assert calib(L, ptrs=(FAKE + 4,) + (FAKE,) * 4) == -3
    assert calib(L, ws=FAKE + 4) == -3
    assert calib(L, res=FAKE + 4) == -3


def test_calibrate_clip_batch_limit(L):
    """Every batch's partials take at most 256 blocks of sums; batches past
    2^52 tokens are refused."""
    for n in (1, 4096, 1 << 20, 1 << 40, 1 << 52):
        assert 0 < L.fp8q_calibrate_clip_workspace(n) <= 212992
    assert L.fp8q_calibrate_clip_workspace((1 << 52) + 1) == -1
    assert calib(L, n=(1 << 52) + 1) == -2


def calib_na(L, ptrs=(FAKE,) * 5, n=4096, cfg=None, res=FAKE):
    import ctypes
    c = fp8q.ClipConfig(**(cfg or fp8q.PAPER_CLIP_CONFIG))
    return L.fp8q_calibrate_clip_noalloc(*ptrs, n, 0.6, 1.8, ctypes.byref(c), res, None)


def test_calibrate_clip_noalloc_rejections(L):
    """The allocation-free form takes the same checks, before it looks up
    its array (no HIP call is made for a rejected call)."""
    P = fp8q.PAPER_CLIP_CONFIG
    assert calib_na(L, ptrs=(FAKE,) * 4 + (None,)) == -1
    assert calib_na(L, res=None) == -1
    assert calib_na(L, n=0) == -1
    assert calib_na(L, n=-3) == -1
    assert calib_na(L, cfg=dict(P, step=-0.02)) == -1
    assert calib_na(L, cfg=dict(P, h_max=1.1)) == -1
    assert calib_na(L, cfg=dict(P, l_min=0.42)) == -2
    assert calib_na(L, ptrs=(FAKE,) * 2 + (FAKE + 8,) + (FAKE,) * 2) == -3
    assert calib_na(L, res=FAKE + 4) == -3
    # every batch's partials fit the array: the largest workspace any n needs
    for n in (1, 4096, 1 << 20, 1 << 40, 1 << 52):
        assert 0 < L.fp8q_calibrate_clip_workspace(n) <= 212992
    assert L.fp8q_calibrate_clip_workspace((1 << 52) + 1) == -1
    assert calib_na(L, n=(1 << 52) + 1) == -2


def test_binding_rejects_short_or_misshapen_buffers():
    """The Python binding checks caller-supplied outputs and scale arrays
    before any call: the kernels read and write exactly the sizes the shapes
    give, so a smaller tensor would be read or written past its end.  (CPU
    tensors fail the same checks; no kernel runs.)"""
    import torch
    import paper_2609_22870_amd as fp8q
    x = torch.zeros((256, 256), dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        fp8q.quantize(x, fp8q.BLOCK_1x128)                      # not a CUDA tensor
    a = torch.zeros((256, 256), dtype=torch.uint8)
    s = torch.zeros(512, dtype=torch.float32)
    with pytest.raises(ValueError):
        fp8q.gemm(a, s, fp8q.BLOCK_1x128, a, s, fp8q.BLOCK_128x128)
    with pytest.raises(ValueError):
        fp8q.cast_f32(torch.zeros(16), 1.0)
