"""C-ABI tests that need no GPU: the library loads, exports every function the
header declares, and rejects bad arguments before launching anything."""
import ctypes
import os
import re

import pytest

import paper_2006_03555_amd as fv
from paper_2006_03555_amd import _lib

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for fn in os.listdir(inc):
        if fn.endswith(".h"):
            text = open(os.path.join(inc, fn)).read()
            names |= set(re.findall(r"FAVOR_API\s+[\w\s\*]+?\b(favor_\w+)\s*\(", text))
    return sorted(names)


@pytest.fixture(scope="module")
def L():
    return fv.lib()


def test_header_declares_the_boundary():
    names = _declared_functions()
    for required in ("favor_orf_draw", "favor_feature_map", "favor_attn_bidir",
                     "favor_attn_causal", "favor_workspace_size", "favor_last_error"):
        assert required in names


def test_library_exports_every_declared_symbol(L):
    for name in _declared_functions():
        assert hasattr(L, name), name


def test_abi_version_and_strings(L):
    assert L.favor_abi_version() == 7
    assert fv.status_string(0) == "FAVOR_OK"
    assert fv.status_string(3) == "FAVOR_ERR_WORKSPACE_TOO_SMALL"


def _desc(**kw):
    base = dict(B=2, H=4, L=1000, d=64, M=256, in_dtype=fv.BF16, out_dtype=fv.BF16,
                input_scale=64 ** -0.25, denom_eps=0.0, segment=0)
    base.update(kw)
    return fv.make_desc(**base)


@pytest.mark.parametrize("kw,status", [
    (dict(), 0),
    (dict(L=0), 0),
    (dict(B=0), 0),
    (dict(L=-1), 1),
    (dict(d=0), 1),
    (dict(d=32), 2),
    (dict(M=100), 2),
    (dict(M=272), 2),
    (dict(M=48), 0),
    (dict(M=16), 0),
    (dict(M=208), 0),
    (dict(M=0), 1),
    (dict(in_dtype=7), 1),
    (dict(out_dtype=-1), 1),
    (dict(input_scale=float("nan")), 1),
    (dict(denom_eps=-1.0), 1),
    (dict(segment=100), 1),
    (dict(segment=-64), 1),
    (dict(chunk=-1), 1),
    (dict(chunk=64), 0),         # the chunk length T of the scan: 64 or 32 (bf16 inputs)
    (dict(chunk=32), 0),
    (dict(chunk=128), 2),
    (dict(chunk=48), 2),
    (dict(B=300, H=300), 2),
    (dict(kernel=fv.KERNEL_RELU), 0),
    (dict(kernel=fv.KERNEL_RELU, kernel_eps=0.0), 0),
    (dict(renormalize=False), 0),
    (dict(kernel=2), 1),
    (dict(kernel=-1), 1),
    (dict(kernel=fv.KERNEL_RELU, kernel_eps=-1e-3), 1),
    (dict(kernel=fv.KERNEL_RELU, kernel_eps=float("inf")), 1),
    (dict(kernel_eps=-1.0), 0),   # kernel_eps is not read for softmax features
    (dict(L=1 << 30), 0),         # the longest sequence per head
    (dict(L=(1 << 30) + 1), 2),
    (dict(segment=1 << 30), 0),
    (dict(segment=(1 << 30) + 64), 2),
])
def test_validate_desc(kw, status):
    for op in (fv.OP_FEATURE_MAP, fv.OP_BIDIR, fv.OP_CAUSAL, fv.OP_BOTH):
        assert fv.validate_desc(_desc(**kw), op) == status
        if status:
            assert fv.last_error() != ""


def test_chunk_32_needs_bf16_inputs_for_the_scan():
    """T = 32 is a variant of the bf16 chunked scan; fp32 inputs take T = 64, and
    the calls without a scan ignore the field."""
    g = _desc(in_dtype=fv.F32, out_dtype=fv.F32, chunk=32)
    for op in (fv.OP_CAUSAL, fv.OP_BOTH, fv.OP_CAUSAL_BACKWARD):
        assert fv.validate_desc(g, op) == 2
        assert "bf16" in fv.last_error()
    for op in (fv.OP_FEATURE_MAP, fv.OP_BIDIR, fv.OP_BIDIR_BACKWARD):
        assert fv.validate_desc(g, op) == 0
    assert fv.validate_desc(_desc(chunk=32), fv.OP_CAUSAL_BACKWARD) == 0


def test_default_chunk_and_segments():
    """chunk = 0 scans bf16 inputs with M <= 128 in 32-token chunks, whose
    workgroups share a compute unit two by two, so the default segments are
    halved (twice the segment aggregates in the workspace); M = 256 and fp32
    inputs default to 64-token chunks and one workgroup per compute unit."""
    def ws(op=1, **kw):
        return fv.workspace_size(_desc(B=1, H=2, L=65536, **kw), op)
    for op in (1, 2):
        for M in (64, 128):
            assert ws(op, M=M) == ws(op, M=M, chunk=32)
            assert ws(op, M=M) > ws(op, M=M, chunk=64)
        assert ws(op, M=256) == ws(op, M=256, chunk=64)
        assert ws(op, M=256) < ws(op, M=256, chunk=32)
        f32 = dict(in_dtype=fv.F32, out_dtype=fv.F32, M=128)
        assert ws(op, **f32) == ws(op, **f32, chunk=64)
    # segment aggregates: M x 65 fp32 per segment; with an explicit segment
    # length the chunk does not change the plan
    assert ws(M=128, chunk=32) - ws(M=128, chunk=64) == 256 * 128 * 65 * 4
    assert ws(M=128, segment=1024) == ws(M=128, segment=1024, chunk=64)


def test_fp32_causal_takes_every_m():
    """fp32 causal at M > 128 runs as two feature-half passes, which need a
    [B*H][L][68] fp32 area of workspace more than M = 128."""
    g = _desc(in_dtype=fv.F32, out_dtype=fv.F32, M=256)
    for op in (fv.OP_CAUSAL, fv.OP_BOTH, fv.OP_BIDIR, fv.OP_BOTH_BACKWARD):
        assert fv.validate_desc(g, op) == 0
    assert fv.validate_desc(g, 7) == 1
    half = -(-2 * 4 * 1000 * 68 * 4 // 256) * 256
    # bf16 at M = 256 runs in one pass; fp32 W'' fragments take 16 more bytes per lane
    plain = fv.workspace_size(_desc(M=256), 1) + 4 * (256 // 16) * 2 * 64 * 16
    for M in (144, 256):
        n = fv.workspace_size(_desc(in_dtype=fv.F32, out_dtype=fv.F32, M=M), 1)
        assert n == plain + half
    assert fv.workspace_size(_desc(in_dtype=fv.F32, out_dtype=fv.F32, M=128), 1) < plain


def test_backward_validation():
    for op in (fv.OP_BIDIR_BACKWARD, fv.OP_CAUSAL_BACKWARD):
        assert fv.validate_desc(_desc(), op) == 0
        assert fv.validate_desc(_desc(out_dtype=fv.F32), op) == 2   # out dtype = in dtype
        # fp32 at every M (feature slices)
        for M in (64, 128, 208, 256):
            assert fv.validate_desc(_desc(in_dtype=fv.F32, out_dtype=fv.F32, M=M), op) == 0
    for op in (fv.OP_BIDIR_BACKWARD, fv.OP_CAUSAL_BACKWARD):
        assert fv.validate_desc(_desc(kernel=fv.KERNEL_RELU, renormalize=False), op) == 0


def test_backward_workspace_size():
    g = _desc()
    nb = fv.backward_workspace_size(g, False)
    nc = fv.backward_workspace_size(g, True)
    assert nb > fv.workspace_size(g, 0) and nb % 256 == 0
    assert nc > fv.workspace_size(g, 1) and nc % 256 == 0
    assert fv.backward_workspace_size(_desc(L=0), True) == 0
    assert fv.backward_workspace_size(_desc(out_dtype=fv.F32), False) == 0


def test_backward_calls_fail_before_launch(L):
    g = _desc()
    null = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    f6 = [fake] * 6
    nf = [null, 0]          # no forward workspace
    st = L.favor_attn_bidir_backward(ctypes.byref(g), *f6, null, null, *nf, null, fake, fake,
                                     fake, 1 << 40, null)
    assert st == 1 and "dQ" in fv.last_error()
    st = L.favor_attn_bidir_backward(ctypes.byref(g), *f6, null, null, *nf, fake, fake, fake,
                                     fake, 16, null)
    assert st == 3
    # out and row_scale come together or not at all
    st = L.favor_attn_bidir_backward(ctypes.byref(g), *f6, fake, null, *nf, fake, fake, fake,
                                     fake, 1 << 40, null)
    assert st == 1 and "together" in fv.last_error()
    st = L.favor_attn_causal_backward(ctypes.byref(g), *([fake] * 5), null, fake, null, null,
                                      *nf, null, fake, fake, fake, null, fake, 16, null)
    assert st == 3
    odd = ctypes.c_void_p((1 << 20) + 4)
    st = L.favor_attn_causal_backward(ctypes.byref(g), *([fake] * 5), odd, fake, null, null,
                                      *nf, null, fake, fake, fake, null, fake, 1 << 40, null)
    assert st == 1 and "state_in" in fv.last_error()
    bad = _desc(out_dtype=fv.F32)
    st = L.favor_attn_bidir_backward(ctypes.byref(bad), *f6, null, null, *nf, fake, fake, fake,
                                     fake, 1 << 40, null)
    assert st == 2
    # a forward workspace names the forward call that left it, and only calls
    # whose workspace holds what the backward reads are accepted
    for fptr, fop, ok in ((fake, 1, True), (fake, 3, True), (fake, 2, False), (fake, 0, False),
                          (null, 1, False), (odd, 1, False), (fake, 7, False)):
        st = L.favor_attn_bidir_backward(ctypes.byref(g), *f6, null, null, fptr, fop, fake,
                                         fake, fake, fake, 16, null)
        assert st == (3 if ok else 1), (fop, fv.last_error())
    for fptr, fop, ok in ((fake, 2, True), (fake, 3, True), (fake, 1, False), (null, 3, False)):
        st = L.favor_attn_causal_backward(ctypes.byref(g), *([fake] * 5), null, fake, null, null,
                                          fptr, fop, null, fake, fake, fake, null, fake, 16, null)
        assert st == (3 if ok else 1), (fop, fv.last_error())
    # a forward row_scale needs out dtype = in dtype
    st = L.favor_attn_bidir_save(ctypes.byref(bad), fake, fake, fake, fake, fake, fake, fake,
                                 fake, 1 << 40, null)
    assert st == 2 and "row_scale" in fv.last_error()
    st = L.favor_attn_causal_save(ctypes.byref(bad), fake, fake, fake, fake, fake, fake, null,
                                  null, fake, fake, 1 << 40, null)
    assert st == 2 and "row_scale" in fv.last_error()


def test_workspace_size():
    g = _desc()
    nb = fv.workspace_size(g, 0)
    nc = fv.workspace_size(g, 1)
    assert nb > 0 and nc > 0 and nb % 256 == 0 and nc % 256 == 0
    nboth = fv.workspace_size(g, 2)
    assert nboth > nc and nboth % 256 == 0
    assert fv.workspace_size(_desc(L=0), 0) == 0
    assert fv.workspace_size(_desc(M=100), 0) == 0
    # M is padded to the kernels' 64, 128 or 256 rows inside the workspace
    for op in (0, 1, 2):
        assert fv.workspace_size(_desc(M=48), op) == fv.workspace_size(_desc(M=64), op)
        assert fv.workspace_size(_desc(M=144), op) == fv.workspace_size(_desc(M=256), op)
    # causal segment length is honoured: more segments need more workspace
    assert fv.workspace_size(_desc(segment=128), 1) > fv.workspace_size(_desc(segment=512), 1)


def test_calls_fail_before_launch(L):
    g = _desc()
    null = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    # NULL tensors
    st = L.favor_attn_bidir(ctypes.byref(g), null, null, null, null, null, null, null, 0, null)
    assert st == 1 and "NULL" in fv.last_error()
    # misaligned tensor
    odd = ctypes.c_void_p((1 << 20) + 2)
    st = L.favor_attn_bidir(ctypes.byref(g), odd, fake, fake, fake, fake, fake, fake, 1 << 30,
                            null)
    assert st == 1 and "aligned" in fv.last_error()
    # workspace too small
    st = L.favor_attn_bidir(ctypes.byref(g), fake, fake, fake, fake, fake, fake, fake, 16, null)
    assert st == 3
    st = L.favor_attn_causal(ctypes.byref(g), fake, fake, fake, fake, fake, fake, null, null,
                             fake, 16, null)
    assert st == 3
    st = L.favor_attn_both(ctypes.byref(g), fake, fake, fake, fake, fake, fake, null, null, null,
                           null, null, fake, 1 << 30, null)
    assert st == 1 and "out_causal" in fv.last_error()
    st = L.favor_attn_both(ctypes.byref(g), fake, fake, fake, fake, fake, fake, fake, null, null,
                           null, null, fake, 16, null)
    assert st == 3
    # bad descriptor
    bad = _desc(M=100)
    assert L.favor_feature_map(ctypes.byref(bad), fake, fake, fake, fake, null) == 2
    assert L.favor_feature_map(None, fake, fake, fake, fake, null) == 1


def test_orf_draw_argument_errors(L):
    null = ctypes.c_void_p(0)
    fake = ctypes.c_void_p(1 << 20)
    assert L.favor_orf_draw(1, -1, 256, 64, 0, fake, fake, null) == 1
    assert L.favor_orf_draw(1, 4, 256, 32, 0, fake, fake, null) == 2
    assert L.favor_orf_draw(1, 4, 256, 64, 9, fake, fake, null) == 1
    assert L.favor_orf_draw(1, 4, 256, 64, 0, null, fake, null) == 1
    assert L.favor_orf_draw(1, 4, 256, 64, 0, ctypes.c_void_p((1 << 20) + 4), fake, null) == 1
    assert "16-byte" in fv.last_error()
    assert L.favor_orf_draw(1, 4, 8192, 64, 0, fake, fake, null) == 2
    assert L.favor_orf_draw(1, 0, 256, 64, 0, null, null, null) == 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(_lib, "_LIB", None)
    monkeypatch.setenv("FAVOR_LIBRARY", str(tmp_path / "nope.so"))
    with pytest.raises(fv.FavorLibraryMissing):
        fv.lib()


def test_binding_checks_tensor_shapes_and_dtypes():
    """A caller-supplied tensor of the wrong shape or dtype is refused before any
    launch (the kernels size their writes from the descriptor)."""
    import torch
    bf = torch.bfloat16
    Q = torch.zeros((1, 2, 64, 64), dtype=bf)
    W = torch.zeros((2, 128, 64))
    b = torch.zeros((2, 128))
    cases = [
        (lambda: fv.feature_map(Q, W, b, 0.35, out_dtype=bf, out=torch.zeros((1, 2, 64, 128))),
         "out"),
        (lambda: fv.feature_map(Q, W, b, 0.35, out=torch.zeros((1, 2, 64, 64), dtype=bf)), "out"),
        (lambda: fv.attn_bidir(Q, Q[:, :, :32], Q, W, b, 0.35), "K"),
        (lambda: fv.attn_bidir(Q, Q, Q.float(), W, b, 0.35), "V"),
        (lambda: fv.attn_bidir(Q, Q, Q, W, b[:1], 0.35), "b"),
        (lambda: fv.attn_causal(Q, Q, Q, W, b, 0.35, state_in=torch.zeros((1, 2, 128, 64))),
         "state_in"),
        (lambda: fv.attn_both(Q, Q, Q, W, b, 0.35, out_causal=torch.zeros((1, 2, 64, 64))),
         "out_causal"),
        (lambda: fv.orf_draw(1, 2, 128, 64, W=torch.zeros((2, 128, 32)), b=b), "W"),
    ]
    for call, name in cases:
        with pytest.raises(fv.FavorError) as e:
            call()
        assert name in str(e.value), (name, str(e.value))


def test_noalloc_rejects_a_workspace_beyond_its_scratch(L):
    """favor_attn_both_noalloc checks the workspace the call needs against its
    static scratch before any device call (placeholder pointers: nothing runs)."""
    assert L.favor_noalloc_scratch_bytes() == 32 << 20
    # fp32 causal passes at M > 128 keep [B][H][L][68] fp32 rows in the workspace
    g = _desc(B=8, H=8, L=8192, M=256, in_dtype=fv.F32, out_dtype=fv.F32)
    assert fv.workspace_size(g, 2) > L.favor_noalloc_scratch_bytes()
    p = ctypes.c_void_p(1 << 20)
    st = L.favor_attn_both_noalloc(ctypes.byref(g), p, p, p, p, p, p, p, None, None, None,
                                   None, None)
    assert st == 3, fv.last_error()
    assert "static scratch" in fv.last_error()
    bad = _desc(d=32)
    assert L.favor_attn_both_noalloc(ctypes.byref(bad), p, p, p, p, p, p, p, None, None, None,
                                     None, None) == 2


def test_header_compiles_as_c_and_after_the_hip_runtime(tmp_path):
    """include/favor.h is a C header: it compiles as C11 on its own and as C++
    after hip/hip_runtime_api.h (whose hipStream_t it declares identically)."""
    import shutil
    import subprocess
    inc = os.path.join(ROOT, "include")
    rocm = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "include")
    c = tmp_path / "a.c"
    c.write_text('#include "favor.h"\nint main(void) { favor_desc g = {0}; hipStream_t s = 0;\n'
                 '  (void)s; return (int)favor_workspace_size(&g, 0); }\n')
    cxx = tmp_path / "b.cpp"
    cxx.write_text('#include <hip/hip_runtime_api.h>\n#include "favor.h"\n'
                   'int f(hipStream_t s) { return s == nullptr; }\n')
    if shutil.which("gcc") is None:
        pytest.skip("needs gcc")
    r = subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-fsyntax-only", "-I", inc, str(c)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    if os.path.isdir(os.path.join(rocm, "hip")):
        r = subprocess.run(["g++", "-std=c++17", "-Wall", "-Werror", "-fsyntax-only",
                            "-D__HIP_PLATFORM_AMD__", "-I", rocm, "-I", inc, str(cxx)],
                           capture_output=True, text=True)
        assert r.returncode == 0, r.stderr


def test_probe_arguments_and_work(L):
    """favor_probe validates its arguments before any launch; favor_probe_work is
    linear in the iteration count."""
    sink = ctypes.c_void_p(0x1000)   # never dereferenced: every call below fails validation
    for kind, iters, s in ((3, 1, sink), (-1, 1, sink), (0, 0, sink), (1, -5, sink),
                           (2, 1, ctypes.c_void_p(0))):
        assert L.favor_probe(kind, iters, s, None) == 1, (kind, iters)
        assert "favor_probe" in fv.last_error()
    for kind in (0, 1, 2):
        w1, w3 = L.favor_probe_work(kind, 1), L.favor_probe_work(kind, 3)
        assert w1 > 0 and w3 == 3 * w1, kind


def test_timing_table(L):
    """Kernel ids 0 .. n-1 carry distinct names; reads outside the table fail."""
    n = L.favor_timing_num_kernels()
    assert n >= 10
    names = [L.favor_timing_kernel_name(k).decode() for k in range(n)]
    assert len(set(names)) == n and all(x.startswith("k_") for x in names)
    ms, cnt = ctypes.c_double(), ctypes.c_int64()
    for k in (-1, n):
        assert L.favor_timing_read(k, ctypes.byref(ms), ctypes.byref(cnt)) == 1
