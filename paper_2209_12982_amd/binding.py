"""ctypes binding of libwinof4 (include/winof4.h).  Argument marshalling only:
device buffers are torch tensors (their ``data_ptr()``), host tables are numpy
arrays, and the stream defaults to torch's current stream.  Every step of the
convolution runs in the library's HIP kernels."""
import ctypes
import os

import numpy as np

TAPS = 36
NCHW, NHWC = 0, 1
SPLIT, FUSED = 0, 1
TAP_AUTO, TAP_RESIDENT, TAP_ROWS = 0, 1, 2
TAP_RESIDENT_64X32, TAP_RESIDENT_32X32, TAP_RESIDENT_16X16 = 3, 4, 5
TAP_WAVES = 6
TAP_ROWS_STREAMK = 7
NOALLOC_SCRATCH_BYTES = 64 << 20   # WINO_NOALLOC_SCRATCH_BYTES
ALGO_DIRECT, ALGO_F2, ALGO_F4 = 0, 2, 4

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

EXPORTS = [
    "wino_f4_plan", "wino_f4_plan_tables", "wino_f4_plan_destroy", "wino_f4_plan_info",
    "wino_f2_plan", "wino_f2_plan_tables", "wino_f2_calibrate_input",
    "wino_f4_plan_device", "wino_f2_plan_device", "wino_f4_plan_int8", "wino_f2_plan_int8",
    "wino_f4_plan_i10", "wino_f2_plan_i10", "wino_f4_plan_tables_i10", "wino_f2_plan_tables_i10",
    "wino_f4_calibrate_input_i10", "wino_f2_calibrate_input_i10",
    "wino_f4_plan_set_tap_kernel", "wino_f4_tap_kernel_choice", "wino_select_algorithm",
    "wino_f4_workspace_bytes",
    "wino_f4_conv_int8", "wino_f4_conv_int8_noalloc", "wino_f4_input_transform", "wino_f4_tap_gemm", "wino_f4_calibrate_input", "wino_f4_calibrate_output",
    "wino_f4_debug_input_transform", "wino_f4_debug_tap_gemm",
    "direct_conv_quantize_weights", "direct_conv_int8", "wino_f4_conv_float", "wino_strerror",
]
# include/winof4_probe.h: the measurement probe, outside the method's interface.
PROBE_EXPORTS = ["wino_probe_mfma_int8"]


class LibraryNotBuilt(RuntimeError):
    pass


class WinoError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {wino_strerror(status)} ({status})")


def library_path():
    return os.path.join(_HERE, "libwinof4.so")


def load_library():
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        raise LibraryNotBuilt(f"{path} is missing; run __graft_entry__.build() or "
                              "python paper_2209_12982_amd/build.py")
    # PyTorch ships its own HIP runtime and loads it under a name that does
    # not match the runtime's soname.  Loaded first, it satisfies this
    # library's dependency as well and the process has one HIP runtime;
    # loaded after this library, it would start a second one next to the
    # system runtime this library bound to, and the library's HIP calls fail.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(path)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    sig = {
        "wino_f4_plan": (I32, [P, P, I32, I32, P, P, P, I32, I32, P]),
        "wino_f4_plan_tables": (I32, [P, I32, I32, P, P, P, I32, P, P, P, P, P]),
        "wino_f2_plan": (I32, [P, P, I32, I32, P, P, P, I32, I32, P]),
        "wino_f2_plan_tables": (I32, [P, I32, I32, P, P, P, I32, P, P, P, P, P]),
        "wino_f2_calibrate_input": (I32, [P, I32, I32, I32, I32, I32, P, P, P]),
        "wino_f4_plan_i10": (I32, [P, P, I32, I32, P, P, P, I32, I32, P]),
        "wino_f2_plan_i10": (I32, [P, P, I32, I32, P, P, P, I32, I32, P]),
        "wino_f4_plan_tables_i10": (I32, [P, I32, I32, P, P, P, I32, P, P, P, P, P]),
        "wino_f2_plan_tables_i10": (I32, [P, I32, I32, P, P, P, I32, P, P, P, P, P]),
        "wino_f4_calibrate_input_i10": (I32, [P, I32, I32, I32, I32, I32, P, P, P]),
        "wino_f2_calibrate_input_i10": (I32, [P, I32, I32, I32, I32, I32, P, P, P]),
        "wino_f4_plan_device": (I32, [P, P, I32, I32, P, P, P, I32, I32, P]),
        "wino_f2_plan_device": (I32, [P, P, I32, I32, P, P, P, I32, I32, P]),
        "wino_f4_plan_int8": (I32, [P, P, I32, I32, I32, P, P, P, I32, I32, P]),
        "wino_f2_plan_int8": (I32, [P, P, I32, I32, I32, P, P, P, I32, I32, P]),
        "wino_f4_plan_destroy": (None, [P]),
        "wino_f4_plan_info": (I32, [P, P, P, P, P, P, P, P]),
        "wino_f4_plan_set_tap_kernel": (I32, [P, I32]),
        "wino_f4_tap_kernel_choice": (I32, [P, I32, I32, I32, P]),
        "wino_select_algorithm": (I32, [I32, I32, I32, I32, I32, I32, P]),
        "wino_f4_workspace_bytes": (SZ, [P, I32, I32, I32, I32]),
        "wino_f4_conv_int8": (I32, [P, P, P, I32, I32, I32, I32, I32, P, SZ, P]),
        "wino_f4_conv_int8_noalloc": (I32, [P, P, P, I32, I32, I32, I32, P]),
        "wino_f4_input_transform": (I32, [P, P, I32, I32, I32, I32, P, SZ, P]),
        "wino_f4_tap_gemm": (I32, [P, P, SZ, P, I32, I32, I32, I32, P]),
        "wino_f4_calibrate_input": (I32, [P, I32, I32, I32, I32, I32, P, P, P]),
        "wino_f4_calibrate_output": (I32, [P, P, I32, I32, I32, I32, P, SZ, P, P, P]),
        "wino_f4_debug_input_transform": (I32, [P, P, I32, I32, I32, I32, P, P, SZ, P]),
        "wino_f4_debug_tap_gemm": (I32, [P, P, I32, I32, I32, I32, P, P, SZ, P]),
        "direct_conv_quantize_weights": (I32, [P, I32, I32, P, P]),
        "direct_conv_int8": (I32, [P, P, P, P, I32, I32, I32, I32, I32, I32, I32, I32, P]),
        "wino_f4_conv_float": (I32, [P, P, P, I32, I32, I32, I32, I32, I32, P]),
        "wino_probe_mfma_int8": (I32, [I32, I32, I32, P, P, P]),
        "wino_strerror": (ctypes.c_char_p, [I32]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def exported_symbols():
    """Names from EXPORTS that the built library resolves."""
    lib = load_library()
    return [n for n in EXPORTS if hasattr(lib, n)]


def wino_strerror(status):
    try:
        return load_library().wino_strerror(int(status)).decode()
    except LibraryNotBuilt:
        return f"status {status}"


def _check(status, where):
    if status != 0:
        raise WinoError(status, where)


def _ptr(t):
    """Device pointer of a torch tensor (or None)."""
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def _dptr(t, dtype, need=0, what="tensor"):
    """Device pointer of a contiguous torch GPU tensor of `dtype` (any dtype
    if None) holding at least `need` elements, or None for None.  The C ABI
    takes plain pointers and cannot tell a host array or a short buffer from
    device memory; a kernel reading either would fault, so the binding checks
    before passing the pointer on."""
    if t is None:
        return None
    import torch
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{what}: expected a torch tensor on the GPU, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{what}: must be a GPU tensor (the kernels read and write device memory)")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{what}: expected {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{what}: must be contiguous")
    if need > 0 and t.numel() < need:
        raise ValueError(f"{what}: holds {t.numel()} elements, the call reads or writes {need}")
    return ctypes.c_void_p(t.data_ptr())


def _tiles(n, h, w, m):
    """Number of m x m output tiles of a batch, 0 for empty or negative sizes."""
    if min(n, h, w) <= 0:
        return 0
    return int(n) * ((int(h) + m - 1) // m) * ((int(w) + m - 1) // m)


def _elems(*dims):
    """Product of the sizes, 0 if any is negative (the C ABI rejects those)."""
    p = 1
    for d in dims:
        if d < 0:
            return 0
        p *= int(d)
    return p


def _stream(stream):
    if stream is None:
        import torch
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return ctypes.c_void_p(stream)
    return ctypes.c_void_p(stream.cuda_stream)


def _nbytes(t):
    """Size in bytes of a device tensor, 0 for None."""
    return 0 if t is None else t.numel() * t.element_size()


def _host(a, dtype, n=None):
    a = np.ascontiguousarray(np.asarray(a, dtype=dtype))
    if n is not None and a.size != n:
        raise ValueError(f"expected {n} values, got {a.size}")
    return a


class WinoF4Plan:
    """Owns a wino_f4_plan_t (from wino_f4_plan, m = 4, or wino_f2_plan,
    m = 2; bits = 10 for the int8/10 plans); destroyed with the object or by
    close()."""

    def __init__(self, handle, cin, cout, m=4, bits=8):
        self.handle = handle
        self.cin = cin
        self.cout = cout
        self.m = m
        self.bits = bits
        self.ntap = (m + 2) * (m + 2)

    def close(self):
        if self.handle:
            load_library().wino_f4_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _make_plan(fn, m, w_oihw, in_exp, w_exp, bias, out_shift, relu, stream, bits=8):
    ntap = (m + 2) * (m + 2)
    w = _host(w_oihw, np.float32)
    cout, cin = w.shape[:2]
    eb = _host(in_exp, np.int8, ntap)
    eg = None if w_exp is None else _host(w_exp, np.int8, ntap)
    b = None if bias is None else _host(bias, np.int32, cout)
    h = ctypes.c_void_p()
    st = getattr(load_library(), fn)(ctypes.byref(h), w.ctypes.data, cin, cout, eb.ctypes.data,
                                     None if eg is None else eg.ctypes.data,
                                     None if b is None else b.ctypes.data, int(out_shift), int(bool(relu)),
                                     _stream(stream))
    _check(st, fn)
    return WinoF4Plan(h, cin, cout, m, bits)


def wino_f4_plan(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    return _make_plan("wino_f4_plan", 4, w_oihw, in_exp, w_exp, bias, out_shift, relu, stream)


def wino_f2_plan(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    """F(2x2, 3x3) plan: 16-entry in_exp / w_exp."""
    return _make_plan("wino_f2_plan", 2, w_oihw, in_exp, w_exp, bias, out_shift, relu, stream)


def wino_f4_plan_i10(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    """int8/10 plan: 10-bit Winograd-domain integers (Vq, Uq in [-512, 511])."""
    return _make_plan("wino_f4_plan_i10", 4, w_oihw, in_exp, w_exp, bias, out_shift, relu, stream, bits=10)


def wino_f2_plan_i10(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    return _make_plan("wino_f2_plan_i10", 2, w_oihw, in_exp, w_exp, bias, out_shift, relu, stream, bits=10)


def _device_weights(w, dtype):
    """Shape and pointer of a contiguous device weight tensor [cout][cin][3][3]."""
    import torch
    if not (isinstance(w, torch.Tensor) and w.is_cuda and w.dtype == dtype and w.dim() == 4
            and tuple(w.shape[2:]) == (3, 3) and w.is_contiguous()):
        raise ValueError(f"expected a contiguous {dtype} device tensor [cout][cin][3][3]")
    return int(w.shape[0]), int(w.shape[1]), _ptr(w)


def _make_plan_device(fn, m, w_dev, e_f, in_exp, w_exp, bias, out_shift, relu, stream):
    import torch
    ntap = (m + 2) * (m + 2)
    int8 = e_f is not None
    cout, cin, wp = _device_weights(w_dev, torch.int8 if int8 else torch.float32)
    eb = _host(in_exp, np.int8, ntap)
    eg = None if w_exp is None else _host(w_exp, np.int8, ntap)
    b = None if bias is None else _host(bias, np.int32, cout)
    h = ctypes.c_void_p()
    args = [ctypes.byref(h), wp] + ([int(e_f)] if int8 else []) + [
        cin, cout, eb.ctypes.data, None if eg is None else eg.ctypes.data,
        None if b is None else b.ctypes.data, int(out_shift), int(bool(relu)), _stream(stream)]
    _check(getattr(load_library(), fn)(*args), fn)
    return WinoF4Plan(h, cin, cout, m)


def wino_f4_plan_device(w_dev, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    """Plan whose weight transform and tap calibration run on the GPU; w_dev:
    contiguous fp32 device tensor [cout][cin][3][3].  Same tables as
    wino_f4_plan on the same weights."""
    return _make_plan_device("wino_f4_plan_device", 4, w_dev, None, in_exp, w_exp, bias, out_shift, relu, stream)


def wino_f2_plan_device(w_dev, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    return _make_plan_device("wino_f2_plan_device", 2, w_dev, None, in_exp, w_exp, bias, out_shift, relu, stream)


def wino_f4_plan_int8(w_dev, w_scale_exp, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    """Plan from int8 spatial weights w * 2^w_scale_exp (w_dev: contiguous
    int8 device tensor [cout][cin][3][3]), transformed in integers on the GPU."""
    return _make_plan_device("wino_f4_plan_int8", 4, w_dev, w_scale_exp, in_exp, w_exp, bias, out_shift, relu,
                             stream)


def wino_f2_plan_int8(w_dev, w_scale_exp, in_exp, w_exp=None, bias=None, out_shift=0, relu=False, stream=None):
    return _make_plan_device("wino_f2_plan_int8", 2, w_dev, w_scale_exp, in_exp, w_exp, bias, out_shift, relu,
                             stream)


def _plan_tables(fn, m, w_oihw, in_exp, w_exp, bias, out_shift, qbits=8):
    ntap = (m + 2) * (m + 2)
    w = _host(w_oihw, np.float32)
    cout, cin = w.shape[:2]
    eb = _host(in_exp, np.int8, ntap)
    eg_in = None if w_exp is None else _host(w_exp, np.int8, ntap)
    b = None if bias is None else _host(bias, np.int32, cout)
    eg = np.zeros(ntap, np.int8)
    sh = np.zeros(ntap, np.int8)
    eo = ctypes.c_int32()
    bits = ctypes.c_int32()
    uq = np.zeros((ntap, cin, cout), np.int16 if qbits == 10 else np.int8)
    st = getattr(load_library(), fn)(w.ctypes.data, cin, cout, eb.ctypes.data,
                                     None if eg_in is None else eg_in.ctypes.data,
                                     None if b is None else b.ctypes.data, int(out_shift),
                                     eg.ctypes.data, sh.ctypes.data, ctypes.byref(eo), ctypes.byref(bits),
                                     uq.ctypes.data)
    _check(st, fn)
    return dict(e_g=eg.astype(int).tolist(), sh=sh.astype(int).tolist(), e_o=eo.value,
                epilogue_bits=bits.value, uq=uq)


def wino_f4_plan_tables(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0):
    """Host-only plan arithmetic (no GPU): dict with e_g, sh, e_o,
    epilogue_bits and uq [36][cin][cout]."""
    return _plan_tables("wino_f4_plan_tables", 4, w_oihw, in_exp, w_exp, bias, out_shift)


def wino_f2_plan_tables(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0):
    """The same for F(2x2, 3x3): 16 taps."""
    return _plan_tables("wino_f2_plan_tables", 2, w_oihw, in_exp, w_exp, bias, out_shift)


def wino_f4_plan_tables_i10(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0):
    """Host-only int8/10 plan arithmetic; uq is int16 [36][cin][cout]."""
    return _plan_tables("wino_f4_plan_tables_i10", 4, w_oihw, in_exp, w_exp, bias, out_shift, qbits=10)


def wino_f2_plan_tables_i10(w_oihw, in_exp, w_exp=None, bias=None, out_shift=0):
    return _plan_tables("wino_f2_plan_tables_i10", 2, w_oihw, in_exp, w_exp, bias, out_shift, qbits=10)


def wino_f4_plan_info(plan, with_uq=False):
    lib = load_library()
    eg = np.zeros(plan.ntap, np.int8)
    sh = np.zeros(plan.ntap, np.int8)
    eo = ctypes.c_int32()
    bits = ctypes.c_int32()
    uq = np.zeros((plan.ntap, plan.cin, plan.cout), np.int8) if with_uq else None
    st = lib.wino_f4_plan_info(plan.handle, eg.ctypes.data, sh.ctypes.data, ctypes.byref(eo),
                               ctypes.byref(bits), None if uq is None else uq.ctypes.data, None, None)
    _check(st, "wino_f4_plan_info")
    return dict(e_g=eg.astype(int).tolist(), sh=sh.astype(int).tolist(), e_o=eo.value,
                epilogue_bits=bits.value, uq=uq)


def wino_f4_plan_set_tap_kernel(plan, kind):
    """TAP_AUTO, TAP_RESIDENT, TAP_ROWS, TAP_ROWS_STREAMK, TAP_WAVES or a TAP_RESIDENT_*
    block shape: the tap-GEMM kernel of later SPLIT convolutions with this plan."""
    _check(load_library().wino_f4_plan_set_tap_kernel(plan.handle, int(kind)), "wino_f4_plan_set_tap_kernel")


def wino_f4_tap_kernel_choice(plan, n, h, w):
    """TAP_WAVES, TAP_ROWS, TAP_ROWS_STREAMK or a TAP_RESIDENT_* shape: the tap-GEMM kernel a
    SPLIT convolution runs."""
    kind = ctypes.c_int32()
    _check(load_library().wino_f4_tap_kernel_choice(plan.handle, n, h, w, ctypes.byref(kind)),
           "wino_f4_tap_kernel_choice")
    return kind.value


def wino_select_algorithm(n, cin, cout, h, w, layout=NHWC):
    """ALGO_DIRECT, ALGO_F2 or ALGO_F4 for a 3x3 layer of this shape and layout."""
    algo = ctypes.c_int32()
    _check(load_library().wino_select_algorithm(n, cin, cout, h, w, layout, ctypes.byref(algo)),
           "wino_select_algorithm")
    return algo.value


def wino_f4_workspace_bytes(plan, n, h, w, variant=SPLIT):
    return int(load_library().wino_f4_workspace_bytes(plan.handle, n, h, w, variant))


def wino_f4_conv_int8(plan, x, y, n, h, w, layout=NCHW, variant=SPLIT, workspace=None, stream=None):
    lib = load_library()
    ws_bytes = _nbytes(workspace)
    import torch
    st = lib.wino_f4_conv_int8(plan.handle, _dptr(x, torch.int8, _elems(n, plan.cin, h, w), "x"),
                               _dptr(y, torch.int8, _elems(n, plan.cout, h, w), "y"), n, h, w, layout, variant,
                               _dptr(workspace, None, 0, "workspace"), ws_bytes, _stream(stream))
    _check(st, "wino_f4_conv_int8")


def wino_f4_conv_int8_noalloc(plan, x, y, n, h, w, layout=NCHW, stream=None):
    """SPLIT convolution with the library's own device scratch (allocates
    nothing; workspace up to NOALLOC_SCRATCH_BYTES)."""
    lib = load_library()
    import torch
    st = lib.wino_f4_conv_int8_noalloc(plan.handle, _dptr(x, torch.int8, _elems(n, plan.cin, h, w), "x"),
                                       _dptr(y, torch.int8, _elems(n, plan.cout, h, w), "y"), n, h, w, layout,
                                       _stream(stream))
    _check(st, "wino_f4_conv_int8_noalloc")


def wino_f4_input_transform(plan, x, n, h, w, layout, workspace, stream=None):
    lib = load_library()
    ws_bytes = _nbytes(workspace)
    import torch
    _check(lib.wino_f4_input_transform(plan.handle, _dptr(x, torch.int8, _elems(n, plan.cin, h, w), "x"), n, h, w,
                                       layout, _dptr(workspace, None, 0, "workspace"), ws_bytes, _stream(stream)),
           "wino_f4_input_transform")


def wino_f4_tap_gemm(plan, workspace, y, n, h, w, layout, stream=None):
    lib = load_library()
    ws_bytes = _nbytes(workspace)
    import torch
    _check(lib.wino_f4_tap_gemm(plan.handle, _dptr(workspace, None, 0, "workspace"), ws_bytes,
                                _dptr(y, torch.int8, _elems(n, plan.cout, h, w), "y"), n, h, w, layout,
                                _stream(stream)), "wino_f4_tap_gemm")


def _calibrate_input(fn, m, x, n, cin, h, w, layout, stream):
    ntap = (m + 2) * (m + 2)
    amax = np.zeros(ntap, np.int32)
    eb = np.zeros(ntap, np.int8)
    import torch
    st = getattr(load_library(), fn)(_dptr(x, torch.int8, _elems(n, cin, h, w), "x"), n, cin, h, w, layout,
                                     amax.ctypes.data, eb.ctypes.data, _stream(stream))
    _check(st, fn)
    return eb.astype(int).tolist(), amax.astype(int).tolist()


def wino_f4_calibrate_input(x, n, cin, h, w, layout=NCHW, stream=None):
    return _calibrate_input("wino_f4_calibrate_input", 4, x, n, cin, h, w, layout, stream)


def wino_f2_calibrate_input(x, n, cin, h, w, layout=NCHW, stream=None):
    return _calibrate_input("wino_f2_calibrate_input", 2, x, n, cin, h, w, layout, stream)


def wino_f4_calibrate_input_i10(x, n, cin, h, w, layout=NCHW, stream=None):
    return _calibrate_input("wino_f4_calibrate_input_i10", 4, x, n, cin, h, w, layout, stream)


def wino_f2_calibrate_input_i10(x, n, cin, h, w, layout=NCHW, stream=None):
    return _calibrate_input("wino_f2_calibrate_input_i10", 2, x, n, cin, h, w, layout, stream)


def wino_f4_calibrate_output(plan, x, n, h, w, layout=NCHW, workspace=None, stream=None):
    lib = load_library()
    ws_bytes = _nbytes(workspace)
    zmax = ctypes.c_int64()
    shift = ctypes.c_int32()
    import torch
    st = lib.wino_f4_calibrate_output(plan.handle, _dptr(x, torch.int8, _elems(n, plan.cin, h, w), "x"), n, h, w,
                                      layout, _dptr(workspace, None, 0, "workspace"), ws_bytes,
                                      ctypes.byref(zmax), ctypes.byref(shift), _stream(stream))
    _check(st, "wino_f4_calibrate_output")
    return shift.value, zmax.value


def wino_f4_debug_input_transform(plan, x, n, h, w, layout, vq, workspace, stream=None):
    lib = load_library()
    ws_bytes = _nbytes(workspace)
    import torch
    st = lib.wino_f4_debug_input_transform(plan.handle, _dptr(x, torch.int8, _elems(n, plan.cin, h, w), "x"),
                                           n, h, w, layout,
                                           _dptr(vq, torch.float16 if plan.bits == 10 else torch.int8,
                                                 plan.ntap * _tiles(n, h, w, plan.m) * plan.cin, "vq"),
                                           _dptr(workspace, None, 0, "workspace"), ws_bytes, _stream(stream))
    _check(st, "wino_f4_debug_input_transform")


def wino_f4_debug_tap_gemm(plan, x, n, h, w, layout, m, workspace, stream=None):
    lib = load_library()
    ws_bytes = _nbytes(workspace)
    import torch
    st = lib.wino_f4_debug_tap_gemm(plan.handle, _dptr(x, torch.int8, _elems(n, plan.cin, h, w), "x"),
                                    n, h, w, layout,
                                    _dptr(m, torch.int32, plan.ntap * _tiles(n, h, w, plan.m) * plan.cout, "m"),
                                    _dptr(workspace, None, 0, "workspace"), ws_bytes, _stream(stream))
    _check(st, "wino_f4_debug_tap_gemm")


def direct_conv_quantize_weights(w_oihw):
    """Returns (int8 weights [cout][3][3][cin], exponent e)."""
    lib = load_library()
    w = _host(w_oihw, np.float32)
    cout, cin = w.shape[:2]
    out = np.zeros((cout, 3, 3, cin), np.int8)
    e = ctypes.c_int32()
    _check(lib.direct_conv_quantize_weights(w.ctypes.data, cout, cin, out.ctypes.data, ctypes.byref(e)),
           "direct_conv_quantize_weights")
    return out, e.value


def direct_conv_int8(x, w_ohwi, bias, y, n, cin, cout, h, w, layout=NCHW, out_shift=0, relu=False,
                     stream=None):
    lib = load_library()
    import torch
    st = lib.direct_conv_int8(_dptr(x, torch.int8, _elems(n, cin, h, w), "x"),
                              _dptr(w_ohwi, torch.int8, _elems(9, cin, cout), "w_ohwi"),
                              _dptr(bias, torch.int32, _elems(cout), "bias"),
                              _dptr(y, torch.int8, _elems(n, cout, h, w), "y"), n, cin, cout, h, w, layout,
                              int(out_shift), int(bool(relu)), _stream(stream))
    _check(st, "direct_conv_int8")


def wino_f4_conv_float(x, w_oihw, y, n, cin, cout, h, w, layout=NCHW, stream=None):
    """Unquantized fp32 Winograd F(4x4,3x3) (reference stage): x int8, w_oihw
    fp32 [cout][cin][3][3], y fp32 in x's layout, all torch device tensors."""
    lib = load_library()
    import torch
    st = lib.wino_f4_conv_float(_dptr(x, torch.int8, _elems(n, cin, h, w), "x"),
                                _dptr(w_oihw, torch.float32, _elems(cout, cin, 9), "w_oihw"),
                                _dptr(y, torch.float32, _elems(n, cout, h, w), "y"), n, cin, cout, h, w, layout,
                                _stream(stream))
    _check(st, "wino_f4_conv_float")


def wino_probe_mfma_int8(shape, iters, blocks, sink, stream=None):
    """Launch the int8 matrix-core rate probe (measurement only); returns the
    launch's operation count.  sink: a device int32 tensor of >= 1 element."""
    ops = ctypes.c_int64()
    import torch
    st = load_library().wino_probe_mfma_int8(int(shape), int(iters), int(blocks), _dptr(sink, torch.int32, 1, "sink"),
                                             ctypes.byref(ops), _stream(stream))
    _check(st, "wino_probe_mfma_int8")
    return ops.value
