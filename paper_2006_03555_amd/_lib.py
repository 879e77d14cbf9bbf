"""ctypes declarations of libfavor's C ABI (include/favor.h)."""
import ctypes
import os

F32 = 0
BF16 = 1
RF_ORTHO_CHI = 0
RF_ORTHO_FIXED = 1
RF_IID = 2
RF_HADAMARD = 3
RF_GIVENS = 4
OP_FEATURE_MAP = 0
OP_BIDIR = 1
OP_CAUSAL = 2
OP_BOTH = 3
OP_BIDIR_BACKWARD = 4
OP_CAUSAL_BACKWARD = 5
OP_BOTH_BACKWARD = 6

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None


class FavorLibraryMissing(ImportError):
    pass


class FavorError(RuntimeError):
    def __init__(self, status, message):
        self.status = status
        super().__init__(f"{status_string(status) if _LIB else status}: {message}")


class FavorDesc(ctypes.Structure):
    _fields_ = [
        ("B", ctypes.c_int32), ("H", ctypes.c_int32), ("L", ctypes.c_int32),
        ("d", ctypes.c_int32), ("M", ctypes.c_int32),
        ("in_dtype", ctypes.c_int), ("out_dtype", ctypes.c_int),
        ("input_scale", ctypes.c_float), ("denom_eps", ctypes.c_float),
        ("chunk", ctypes.c_int32),
        ("kernel", ctypes.c_int32), ("no_renormalize", ctypes.c_int32),
        ("kernel_eps", ctypes.c_float),
        ("segment", ctypes.c_int32),
    ]


def lib_path():
    return os.environ.get("FAVOR_LIBRARY", os.path.join(_HERE, "libfavor.so"))


def lib():
    """Load libfavor.so once; raise FavorLibraryMissing if it has not been built."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = lib_path()
    if not os.path.exists(path):
        raise FavorLibraryMissing(
            f"{path} not found: build it with `python -m paper_2006_03555_amd.build`")
    L = ctypes.CDLL(path)
    vp, i32, u64, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    dp = ctypes.POINTER(FavorDesc)
    sig = {
        "favor_orf_draw": (ctypes.c_int, [u64, i32, i32, i32, ctypes.c_int, vp, vp, vp]),
        "favor_feature_map": (ctypes.c_int, [dp, vp, vp, vp, vp, vp]),
        "favor_workspace_size": (sz, [dp, ctypes.c_int]),
        "favor_attn_bidir": (ctypes.c_int, [dp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "favor_attn_bidir_save": (ctypes.c_int, [dp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "favor_attn_causal": (ctypes.c_int,
                              [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "favor_attn_causal_save": (ctypes.c_int,
                                   [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "favor_attn_both": (ctypes.c_int,
                            [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]),
        "favor_attn_both_noalloc": (ctypes.c_int,
                                    [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]),
        "favor_noalloc_scratch_bytes": (sz, []),
        "favor_probe": (ctypes.c_int, [i32, i32, vp, vp]),
        "favor_probe_work": (ctypes.c_double, [i32, i32]),
        "favor_backward_workspace_size": (sz, [dp, ctypes.c_int]),
        "favor_attn_bidir_backward": (ctypes.c_int, [dp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                     vp, i32, vp, vp, vp, vp, sz, vp]),
        "favor_attn_causal_backward": (ctypes.c_int, [dp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                      vp, vp, i32, vp, vp, vp, vp, vp, vp, sz,
                                                      vp]),
        "favor_attn_both_backward": (ctypes.c_int, [dp, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                                    vp, vp, vp, vp, i32, vp, vp, vp, vp, vp,
                                                    vp, sz, vp]),
        "favor_validate_desc": (ctypes.c_int, [dp, ctypes.c_int]),
        "favor_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "favor_last_error": (ctypes.c_char_p, []),
        "favor_abi_version": (i32, []),
        "favor_timing_enable": (ctypes.c_int, [ctypes.c_int]),
        "favor_timing_reset": (ctypes.c_int, []),
        "favor_timing_num_kernels": (i32, []),
        "favor_timing_kernel_name": (ctypes.c_char_p, [i32]),
        "favor_timing_read": (ctypes.c_int, [i32, ctypes.POINTER(ctypes.c_double),
                                             ctypes.POINTER(ctypes.c_int64)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    if L.favor_abi_version() != ABI_VERSION:
        raise FavorLibraryMissing(f"{path}: ABI version {L.favor_abi_version()} != {ABI_VERSION}")
    _LIB = L
    return L


def status_string(s):
    return lib().favor_status_string(int(s)).decode()


def last_error():
    return lib().favor_last_error().decode()


KERNEL_SOFTMAX = 0
KERNEL_RELU = 1
ABI_VERSION = 7   # the backward of both directions in one call


def make_desc(B, H, L, d, M, in_dtype, out_dtype, input_scale, denom_eps=0.0, segment=0,
              kernel=KERNEL_SOFTMAX, renormalize=True, kernel_eps=1e-3, chunk=0):
    """Descriptor; segment = causal rows per segment (0 = library default),
    chunk = causal chunk length T (0 = the library's choice: 32 for bf16 inputs
    with M <= 128, else 64)."""
    return FavorDesc(B, H, L, d, M, in_dtype, out_dtype, float(input_scale), float(denom_eps),
                     chunk, int(kernel), 0 if renormalize else 1, float(kernel_eps), segment)


def validate_desc(g, op):
    return lib().favor_validate_desc(ctypes.byref(g), op)


def backward_workspace_size(g, causal):
    """causal: False/0 bidirectional, True/1 causal, 2 both directions in one call."""
    return lib().favor_backward_workspace_size(ctypes.byref(g),
                                               2 if causal == 2 else (1 if causal else 0))


def workspace_size(g, causal):
    """causal: False/0 bidirectional, True/1 causal, 2 both directions."""
    return lib().favor_workspace_size(ctypes.byref(g), 2 if causal == 2 else (1 if causal else 0))


def timing_enable(on=True):
    lib().favor_timing_enable(1 if on else 0)


def timing_reset():
    st = lib().favor_timing_reset()
    if st != 0:
        raise FavorError(st, "timing reset failed")


def timing_read():
    """{kernel name: (total ms, launches)} since the last reset (waits for the events)."""
    L = lib()
    out = {}
    for k in range(L.favor_timing_num_kernels()):
        ms = ctypes.c_double()
        n = ctypes.c_int64()
        st = L.favor_timing_read(k, ctypes.byref(ms), ctypes.byref(n))
        if st != 0:
            raise FavorError(st, "timing read failed")
        out[L.favor_timing_kernel_name(k).decode()] = (ms.value, n.value)
    return out
