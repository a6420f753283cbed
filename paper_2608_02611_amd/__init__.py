"""Python binding of the MI355X candidate-screening library (libkb.so).

Argument marshalling only: every step of generation and screening runs in the
library's HIP kernels; torch provides device memory, tensor metadata and the
current stream.  The names mirror the C interface in include/kb.h:

    kb_policy_check, kb_screen_workspace_bytes, kb_screen_launch, kb_screen,
    kb_screen_stats, kb_gen_inputs, kb_last_error, kb_version

plus `screen(...)`, which chains the gate, the kernel and the readback for the
common case.  The pass/fail verdict of each record comes from the library
(kb_summarize / kb_screen_stats); this module only copies it into the record
dicts.  Loading fails loudly (KbError) when libkb.so has not been built;
there is no fallback implementation.
"""
import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libkb.so")

# Codes shared with include/kb.h.
KB_F32, KB_F16, KB_BF16, KB_U32 = 0, 1, 2, 3
KB_DIST_U32, KB_DIST_UNIFORM, KB_DIST_NORMAL, KB_DIST_STUDENT_T3 = 0, 1, 2, 3
(KB_PERTURB_ADD_UNIFORM, KB_PERTURB_REL_UNIFORM, KB_PERTURB_ADD_NORMAL, KB_PERTURB_SCALE_WHERE,
 KB_PERTURB_FLIP_LSB_WHERE, KB_PERTURB_SPECIALS, KB_PERTURB_ZERO_SUBNORMAL_REL) = range(1, 8)
KB_SCATTER_NAN, KB_SCATTER_INF_SIGN_OF_REF = 1, 2
KB_MAX_INDICES = 4096
KB_OK = 0
KB_ERR_INVALID_ARG, KB_ERR_DTYPE, KB_ERR_WORKSPACE, KB_ERR_ALIGNMENT, KB_ERR_HIP = -1, -2, -3, -4, -5
KB_STATUS_OK, KB_REJECT_NULL, KB_REJECT_DTYPE, KB_REJECT_SHAPE, KB_REJECT_LAYOUT = 0, 1, 2, 3, 4
KB_EQUAL_NAN = 1
KB_FAIL_FAST = 2
KB_MAX_DIMS = 8

ERROR_NAMES = {KB_ERR_INVALID_ARG: "KB_ERR_INVALID_ARG", KB_ERR_DTYPE: "KB_ERR_DTYPE",
               KB_ERR_WORKSPACE: "KB_ERR_WORKSPACE", KB_ERR_ALIGNMENT: "KB_ERR_ALIGNMENT",
               KB_ERR_HIP: "KB_ERR_HIP"}


class KbError(RuntimeError):
    def __init__(self, code, message):
        super().__init__("%s (%d): %s" % (ERROR_NAMES.get(code, "KB_ERR"), code, message))
        self.code = code


class KbTensor(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("dtype", ctypes.c_int32), ("ndim", ctypes.c_int32),
                ("shape", ctypes.c_int64 * KB_MAX_DIMS), ("strides", ctypes.c_int64 * KB_MAX_DIMS)]


class KbStats(ctypes.Structure):
    _fields_ = [("numel", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
                ("nan_count", ctypes.c_uint64), ("pos_inf_count", ctypes.c_uint64),
                ("neg_inf_count", ctypes.c_uint64), ("sum_sq_diff", ctypes.c_double),
                ("sum_sq_ref", ctypes.c_double), ("rel_l2", ctypes.c_double),
                ("max_abs_err", ctypes.c_float), ("max_rel_err", ctypes.c_float),
                ("bitwise_equal", ctypes.c_int32), ("status", ctypes.c_int32)]

    def as_dict(self, passed=None):
        """The record's fields; `passed`, the library's verdict for it (from
        kb_summarize or kb_screen_stats), is added when given."""
        d = {name: getattr(self, name) for name, _ in self._fields_}
        if passed is not None:
            d["passed"] = int(passed)
        return d


class KbSummary(ctypes.Structure):
    _fields_ = [("n_candidates", ctypes.c_int32), ("n_passed", ctypes.c_int32),
                ("n_rejected", ctypes.c_int32), ("n_failed", ctypes.c_int32),
                ("first_passed", ctypes.c_int32), ("first_failed", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class KbScreenOpts(ctypes.Structure):
    _fields_ = [("host_table", ctypes.c_void_p), ("host_table_bytes", ctypes.c_size_t),
                ("d_loc", ctypes.c_void_p)]


KB_INLINE_CANDS = 128


class KbLaunch(ctypes.Structure):
    _fields_ = [("group_size", ctypes.c_int32), ("n_groups", ctypes.c_int32),
                ("blocks_per_group", ctypes.c_int32), ("threads", ctypes.c_int32),
                ("grid", ctypes.c_int64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class KbLocate(ctypes.Structure):
    _fields_ = [("first_mismatch", ctypes.c_int64), ("max_abs_index", ctypes.c_int64),
                ("max_rel_index", ctypes.c_int64), ("reserved", ctypes.c_int64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_ if name != "reserved"}


class KbSampleStats(ctypes.Structure):
    _fields_ = [("mean_us", ctypes.c_double), ("p50_us", ctypes.c_double),
                ("p90_us", ctypes.c_double), ("p95_us", ctypes.c_double),
                ("p99_us", ctypes.c_double), ("p90_over_p50", ctypes.c_double),
                ("p95_over_p50", ctypes.c_double), ("p99_over_p50", ctypes.c_double),
                ("speedup_vs_base", ctypes.c_double), ("n_samples", ctypes.c_int32),
                ("valid", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class KbRungScore(ctypes.Structure):
    _fields_ = [("latency_us", ctypes.c_double), ("score", ctypes.c_double),
                ("speedup_vs_base", ctypes.c_double), ("valid", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_ if name != "reserved"}


assert ctypes.sizeof(KbSampleStats) == 80
assert ctypes.sizeof(KbRungScore) == 32
assert ctypes.sizeof(KbStats) == 80
assert ctypes.sizeof(KbLocate) == 32
assert ctypes.sizeof(KbTensor) == 144

EXPORTS = ("kb_policy_check", "kb_screen_workspace_bytes", "kb_screen_positions_workspace_bytes",
           "kb_screen_workspace_init",
           "kb_screen_launch", "kb_screen", "kb_screen_ex", "kb_screen_host_table_bytes",
           "kb_screen_stats", "kb_summarize", "kb_gen_inputs",
           "kb_screen_locate", "kb_rung_stats", "kb_rung_promote", "kb_rung_survival", "kb_screen_multi",
           "kb_screen_multi_workspace_bytes", "kb_screen_multi_host_table_bytes", "kb_summarize_multi",
           "kb_screen_noalloc", "kb_gen_softmax_rows", "kb_gen_indices", "kb_gen_perturb", "kb_gen_scatter",
           "kb_last_error", "kb_version")

_lib = None


def lib():
    """The loaded libkb.so; raises KbError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise KbError(KB_ERR_HIP, "%s is not built (run __graft_entry__.build())" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, u32, u64, f32 = (ctypes.c_void_p, ctypes.c_int, ctypes.c_uint32, ctypes.c_uint64,
                                  ctypes.c_float)
        L.kb_policy_check.argtypes = [ctypes.POINTER(KbTensor), ctypes.POINTER(KbTensor), i32,
                                      ctypes.POINTER(ctypes.c_int32)]
        L.kb_policy_check.restype = i32
        L.kb_screen_workspace_bytes.argtypes = [i32, u64, i32]
        L.kb_screen_workspace_bytes.restype = ctypes.c_size_t
        L.kb_screen_positions_workspace_bytes.argtypes = [i32, u64, i32]
        L.kb_screen_positions_workspace_bytes.restype = ctypes.c_size_t
        L.kb_screen_workspace_init.argtypes = [vp, ctypes.c_size_t, vp]
        L.kb_screen_workspace_init.restype = i32
        L.kb_summarize.argtypes = [ctypes.POINTER(KbStats), i32, ctypes.POINTER(KbSummary),
                                   ctypes.POINTER(ctypes.c_int32)]
        L.kb_summarize.restype = i32
        L.kb_screen_launch.argtypes = [i32, u64, i32, ctypes.POINTER(KbLaunch)]
        L.kb_screen_launch.restype = i32
        L.kb_screen.argtypes = [ctypes.POINTER(KbTensor), ctypes.POINTER(KbTensor), i32, f32, f32,
                                u32, vp, ctypes.c_size_t, vp, vp]
        L.kb_screen.restype = i32
        L.kb_screen_ex.argtypes = [ctypes.POINTER(KbTensor), ctypes.POINTER(KbTensor), i32, f32, f32,
                                   u32, vp, ctypes.c_size_t, vp, ctypes.POINTER(KbScreenOpts), vp]
        L.kb_screen_ex.restype = i32
        L.kb_screen_noalloc.argtypes = [ctypes.POINTER(KbTensor), ctypes.POINTER(KbTensor), i32, f32, f32,
                                        u32, vp, vp]
        L.kb_screen_noalloc.restype = i32
        L.kb_screen_host_table_bytes.argtypes = [i32]
        L.kb_screen_host_table_bytes.restype = ctypes.c_size_t
        L.kb_screen_stats.argtypes = [vp, i32, ctypes.POINTER(KbStats), ctypes.POINTER(KbSummary),
                                      ctypes.POINTER(ctypes.c_int32), vp]
        L.kb_screen_stats.restype = i32
        L.kb_screen_locate.argtypes = [ctypes.POINTER(KbTensor), ctypes.POINTER(KbTensor), i32, f32,
                                       f32, u32, vp, vp, vp]
        L.kb_screen_locate.restype = i32
        f64 = ctypes.c_double
        L.kb_rung_stats.argtypes = [vp, i32, i32, i32, i32, i32, f64, f64, f64, vp, vp, vp]
        L.kb_rung_stats.restype = i32
        L.kb_rung_promote.argtypes = [vp, i32, i32, i32, i32, vp, vp, vp, vp]
        L.kb_rung_promote.restype = i32
        L.kb_rung_survival.argtypes = [vp, vp, vp, i32, i32, vp, vp]
        L.kb_rung_survival.restype = i32
        L.kb_screen_multi_workspace_bytes.argtypes = [ctypes.POINTER(KbTensor), i32, i32]
        L.kb_screen_multi_workspace_bytes.restype = ctypes.c_size_t
        L.kb_screen_multi.argtypes = [ctypes.POINTER(KbTensor), i32, ctypes.POINTER(KbTensor), i32,
                                      ctypes.POINTER(f32), ctypes.POINTER(f32), u32, vp,
                                      ctypes.c_size_t, vp, ctypes.POINTER(KbScreenOpts), vp]
        L.kb_screen_multi.restype = i32
        L.kb_screen_multi_host_table_bytes.argtypes = [i32, i32]
        L.kb_screen_multi_host_table_bytes.restype = ctypes.c_size_t
        L.kb_summarize_multi.argtypes = [ctypes.POINTER(KbStats), i32, i32, ctypes.POINTER(KbSummary),
                                         ctypes.POINTER(ctypes.c_int32)]
        L.kb_summarize_multi.restype = i32
        L.kb_gen_inputs.argtypes = [vp, i32, u64, i32, f32, f32, u64, u32, u32, u64, vp]
        L.kb_gen_inputs.restype = i32
        L.kb_gen_softmax_rows.argtypes = [vp, i32, u64, u64, f32, u64, u32, u32, vp]
        L.kb_gen_softmax_rows.restype = i32
        L.kb_gen_indices.argtypes = [vp, u32, u64, u64, u32, u32, vp]
        L.kb_gen_indices.restype = i32
        L.kb_gen_perturb.argtypes = [vp, vp, i32, u64, i32, f32, f32, f32, u64, u32, u32, u64, vp]
        L.kb_gen_perturb.restype = i32
        L.kb_gen_scatter.argtypes = [vp, vp, i32, u64, vp, u32, i32, vp]
        L.kb_gen_scatter.restype = i32
        L.kb_last_error.argtypes = []
        L.kb_last_error.restype = ctypes.c_char_p
        L.kb_version.argtypes = []
        L.kb_version.restype = i32
        _lib = L
    return _lib


def kb_last_error():
    return lib().kb_last_error().decode()


def kb_version():
    return lib().kb_version()


def _check(rc):
    if rc != KB_OK:
        raise KbError(rc, kb_last_error())
    return rc


# ------------------------------------------------------------ marshalling ---

def _torch():
    import torch
    return torch


def dtype_code(t):
    torch = _torch()
    m = {torch.float32: KB_F32, torch.float16: KB_F16, torch.bfloat16: KB_BF16,
         torch.int32: KB_U32}
    if hasattr(torch, "uint32"):
        m[torch.uint32] = KB_U32
    if t.dtype not in m:
        return -1
    return m[t.dtype]


def describe(t, dtype=None):
    """kb_tensor descriptor of a torch tensor (or None -> a NULL candidate)."""
    d = KbTensor()
    if t is None:
        d.data = None
        d.dtype = -1 if dtype is None else dtype
        d.ndim = 0
        return d
    if t.dim() > KB_MAX_DIMS:
        raise ValueError("more than %d dimensions" % KB_MAX_DIMS)
    d.data = t.data_ptr() if t.numel() > 0 or t.data_ptr() else None
    d.dtype = dtype_code(t) if dtype is None else dtype
    d.ndim = t.dim()
    for i in range(t.dim()):
        d.shape[i] = t.shape[i]
        d.strides[i] = t.stride(i)
    return d


def _stream_handle(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


# ------------------------------------------------------------- interface ---

def kb_policy_check(ref, cands):
    """Per-candidate policy status (list of ints) for torch tensors / None."""
    r = describe(ref)
    arr = (KbTensor * max(1, len(cands)))(*[describe(c) for c in cands])
    status = (ctypes.c_int32 * max(1, len(cands)))()
    _check(lib().kb_policy_check(ctypes.byref(r), arr, len(cands), status))
    return list(status)[:len(cands)]


def kb_screen_workspace_bytes(n_cands, numel, dtype):
    return lib().kb_screen_workspace_bytes(n_cands, numel, dtype)


def kb_screen_positions_workspace_bytes(n_cands, numel, dtype):
    return lib().kb_screen_positions_workspace_bytes(n_cands, numel, dtype)


def kb_screen_launch(n_cands, numel, dtype):
    out = KbLaunch()
    _check(lib().kb_screen_launch(n_cands, numel, dtype, ctypes.byref(out)))
    return out.as_dict()


def kb_screen_workspace_init(workspace, stream=None):
    """Zero-fill a workspace tensor with the library's fill kernel."""
    _check(lib().kb_screen_workspace_init(ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                          _stream_handle(stream)))
    return workspace


def alloc_workspace(n_cands, numel, dtype, device, stream=None, positions=False):
    """A workspace for these sizes (for calls with positions if `positions`),
    zero-filled by the library."""
    torch = _torch()
    nbytes = (kb_screen_positions_workspace_bytes if positions else kb_screen_workspace_bytes)(n_cands, numel,
                                                                                              dtype)
    if nbytes == 0:
        raise KbError(KB_ERR_INVALID_ARG, "no workspace size for these arguments")
    ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    return kb_screen_workspace_init(ws, stream)


def alloc_stats(n_cands, device):
    torch = _torch()
    return torch.empty(n_cands * ctypes.sizeof(KbStats), dtype=torch.uint8, device=device)


def alloc_locate(n_cands, device):
    torch = _torch()
    return torch.empty(n_cands * ctypes.sizeof(KbLocate), dtype=torch.uint8, device=device)


def _sync_stream(stream):
    """Wait for `stream` (torch's current stream when None)."""
    torch = _torch()
    (torch.cuda.current_stream() if stream is None else stream).synchronize()


def read_locate(buf, n):
    """Position dicts from a kb_locate buffer (copies a device buffer back on
    torch's current stream: the caller has waited for the writing stream)."""
    host = buf.cpu() if buf.device.type != "cpu" else buf
    locs = (KbLocate * max(1, n)).from_buffer_copy(host.numpy().tobytes())
    return [locs[k].as_dict() for k in range(n)]


class HostTables:
    """The caller-owned pinned launch tables of calls with more than
    KB_INLINE_CANDS candidates: a ring of `count` pinned host buffers of
    `nbytes` each.  A buffer is handed out again only once the stream has
    passed the call that last used it (an event recorded after each call),
    because the kernels read their table from it."""

    def __init__(self, nbytes, count=2):
        torch = _torch()
        self.nbytes = int(nbytes)
        self.bufs = [torch.empty(max(1, self.nbytes), dtype=torch.uint8, pin_memory=True)
                     for _ in range(count)]
        self.events = [None] * count
        self.opts = [KbScreenOpts(t.data_ptr(), self.nbytes) for t in self.bufs]
        self.next = 0

    def acquire(self):
        """(index, opts) of the next buffer, after its previous call has passed."""
        i = self.next
        self.next = (i + 1) % len(self.bufs)
        if self.events[i] is not None:
            self.events[i].synchronize()
            self.events[i] = None
        return i, self.opts[i]

    def release(self, i, stream=None):
        """Record that the call just enqueued on `stream` reads buffer i."""
        torch = _torch()
        e = torch.cuda.Event()
        e.record(torch.cuda.current_stream() if stream is None else stream)
        self.events[i] = e


# Host tables of function-style calls, kept alive until their calls have passed.
_pending_tables = []


def _one_off_opts(nbytes, stream):
    """(opts, keep) for one call that needs a host table, or (None, None)."""
    global _pending_tables
    if nbytes == 0:
        return None, None
    _pending_tables = [(t, e) for t, e in _pending_tables if not e.query()]
    tables = HostTables(nbytes, count=1)
    i, opts = tables.acquire()
    return opts, (tables, i)


def _after_one_off(keep, stream):
    if keep is not None:
        tables, i = keep
        tables.release(i, stream)
        _pending_tables.append((tables, tables.events[i]))


def kb_screen(ref, cands, atol, rtol, flags=0, workspace=None, d_stats=None, stream=None, d_loc=None):
    """Enqueue the screen of `cands` (torch tensors or None) against `ref`.

    Returns (d_stats, workspace) device buffers; read the records with
    kb_screen_stats.  More than KB_INLINE_CANDS candidates go through
    kb_screen_ex with a pinned host table, kept alive here until the call
    has passed.  d_loc (a buffer of len(cands) kb_locate, see alloc_locate)
    asks for the positions in the same pass (read them with read_locate).
    """
    n = len(cands)
    r = describe(ref)
    arr = (KbTensor * max(1, n))(*[describe(c) for c in cands])
    if workspace is None:
        workspace = alloc_workspace(max(1, n), ref.numel(), r.dtype if r.dtype >= 0 else 0,
                                    ref.device, stream, positions=d_loc is not None)
    if d_stats is None:
        d_stats = alloc_stats(max(1, n), ref.device)
    opts, keep = _one_off_opts(lib().kb_screen_host_table_bytes(n), stream)
    if d_loc is not None:
        opts = opts if opts is not None else KbScreenOpts(None, 0, None)
        opts.d_loc = d_loc.data_ptr()
    _check(lib().kb_screen_ex(ctypes.byref(r), arr, n, float(atol), float(rtol), int(flags),
                              ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                              ctypes.c_void_p(d_stats.data_ptr()),
                              ctypes.byref(opts) if opts is not None else None, _stream_handle(stream)))
    _after_one_off(keep, stream)
    return d_stats, workspace


NOALLOC_SCRATCH_BYTES = 16 << 20


def kb_screen_noalloc(ref, cands, atol, rtol, flags=0, d_stats=None, stream=None):
    """Enqueue kb_screen_noalloc (the library's fixed scratch instead of a
    workspace; at most KB_INLINE_CANDS candidates).  Returns d_stats; read
    the records with kb_screen_stats."""
    n = len(cands)
    r = describe(ref)
    arr = (KbTensor * max(1, n))(*[describe(c) for c in cands])
    if d_stats is None:
        d_stats = alloc_stats(max(1, n), ref.device)
    _check(lib().kb_screen_noalloc(ctypes.byref(r), arr, n, float(atol), float(rtol), int(flags),
                                   ctypes.c_void_p(d_stats.data_ptr()), _stream_handle(stream)))
    return d_stats


def kb_screen_stats(d_stats, n_cands, stream=None):
    """Read back n_cands records (synchronizes the stream): (list of dicts
    with the library's verdict as "passed", summary dict)."""
    host = (KbStats * max(1, n_cands))()
    summ = KbSummary()
    passed = (ctypes.c_int32 * max(1, n_cands))()
    _check(lib().kb_screen_stats(ctypes.c_void_p(d_stats.data_ptr()), n_cands, host,
                                 ctypes.byref(summ), passed, _stream_handle(stream)))
    return [host[k].as_dict(passed[k]) for k in range(n_cands)], summ.as_dict()


def kb_screen_locate(ref, cands, atol, rtol, d_stats, flags=0, stream=None):
    """Positions of the first mismatch and of the maxima for each candidate
    (list of dicts, -1 where none).  d_stats holds the records kb_screen
    wrote for the same arguments on the same stream; synchronizes the
    stream to read the result."""
    torch = _torch()
    r = describe(ref)
    arr = (KbTensor * max(1, len(cands)))(*[describe(c) for c in cands])
    out = torch.empty(max(1, len(cands)) * ctypes.sizeof(KbLocate), dtype=torch.uint8,
                      device=ref.device)
    _check(lib().kb_screen_locate(ctypes.byref(r), arr, len(cands), float(atol), float(rtol),
                                  int(flags), ctypes.c_void_p(d_stats.data_ptr()),
                                  ctypes.c_void_p(out.data_ptr()), _stream_handle(stream)))
    _sync_stream(stream)
    return read_locate(out, len(cands))


class Locator:
    """Repeated kb_screen_locate calls over one fixed set of buffers and
    records, with the argument marshalling done once (as Screener does for
    kb_screen): launch() enqueues, read() copies the positions back."""

    def __init__(self, ref, cands, atol, rtol, d_stats, flags=0, stream=None):
        torch = _torch()
        self._keep = (ref, list(cands), d_stats)
        self.n = len(cands)
        self._ref = describe(ref)
        self._arr = (KbTensor * max(1, self.n))(*[describe(c) for c in cands])
        self.out = torch.empty(max(1, self.n) * ctypes.sizeof(KbLocate), dtype=torch.uint8, device=ref.device)
        self.atol, self.rtol, self.flags = float(atol), float(rtol), int(flags)
        self._stats = ctypes.c_void_p(d_stats.data_ptr())
        self._out = ctypes.c_void_p(self.out.data_ptr())
        self.stream = stream
        self._stream = _stream_handle(stream)
        self._L = lib()

    def launch(self):
        _check(self._L.kb_screen_locate(ctypes.byref(self._ref), self._arr, self.n, self.atol, self.rtol,
                                        self.flags, self._stats, self._out, self._stream))

    def read(self):
        """Wait for the launch stream, then copy the positions back."""
        _sync_stream(self.stream)
        return read_locate(self.out, self.n)


def locate(ref, cands, atol, rtol, flags=0, stream=None):
    """Screen, then locate (two passes): (records, positions)."""
    d_stats, _ = kb_screen(ref, cands, atol, rtol, flags, stream=stream)
    recs, _ = kb_screen_stats(d_stats, len(cands), stream=stream)
    return recs, kb_screen_locate(ref, cands, atol, rtol, d_stats, flags, stream=stream)


def screen_positions(ref, cands, atol, rtol, flags=0, stream=None):
    """Screen with the positions found in the same pass: (records, positions)."""
    d_loc = alloc_locate(max(1, len(cands)), ref.device)
    d_stats, _ = kb_screen(ref, cands, atol, rtol, flags, stream=stream, d_loc=d_loc)
    recs, _ = kb_screen_stats(d_stats, len(cands), stream=stream)
    return recs, read_locate(d_loc, len(cands))


RUNG_MAX_ITER = 4096
RUNG_ALPHA, RUNG_BETA = 0.02, 0.01


def kb_rung_stats(samples, base=0, rung=0, budget=0.0, alpha=RUNG_ALPHA, beta=RUNG_BETA,
                  rows=None, scores=None, stream=None):
    """Enqueue the rung statistics of samples, a contiguous float64 device
    tensor [n_cands][n_shapes][n_iter] of timing samples (us).  Returns the
    (rows, scores) device buffers; read them with rung_records."""
    torch = _torch()
    if samples.dtype != torch.float64 or samples.dim() != 3 or not samples.is_contiguous():
        raise ValueError("samples must be a contiguous float64 [n_cands][n_shapes][n_iter] tensor")
    C, S, N = samples.shape
    if rows is None:
        rows = torch.empty(max(1, C * S) * ctypes.sizeof(KbSampleStats), dtype=torch.uint8,
                           device=samples.device)
    if scores is None:
        scores = torch.empty(max(1, C) * ctypes.sizeof(KbRungScore), dtype=torch.uint8,
                             device=samples.device)
    _check(lib().kb_rung_stats(ctypes.c_void_p(samples.data_ptr()), C, S, N, int(base), int(rung),
                               float(budget), float(alpha), float(beta),
                               ctypes.c_void_p(rows.data_ptr()), ctypes.c_void_p(scores.data_ptr()),
                               _stream_handle(stream)))
    return rows, scores


def rung_records(rows, scores, n_cands, n_shapes):
    """Host copies: (rows as n_cands lists of n_shapes dicts, scores as a
    list of n_cands dicts).  Synchronizes with the device."""
    rb = rows.cpu().numpy().tobytes()
    sb = scores.cpu().numpy().tobytes()
    R = (KbSampleStats * (n_cands * n_shapes)).from_buffer_copy(rb[:n_cands * n_shapes * 80])
    Sc = (KbRungScore * n_cands).from_buffer_copy(sb[:n_cands * 32])
    return ([[R[c * n_shapes + s].as_dict() for s in range(n_shapes)] for c in range(n_cands)],
            [Sc[c].as_dict() for c in range(n_cands)])


def rung_stats(samples, base=0, rung=0, budget=0.0, alpha=RUNG_ALPHA, beta=RUNG_BETA, stream=None):
    """Enqueue, then read back: (rows, scores) as lists of dicts."""
    C, S, _ = samples.shape
    rows, scores = kb_rung_stats(samples, base, rung, budget, alpha, beta, stream=stream)
    return rung_records(rows, scores, C, S)


PROMOTE_MAX = 65536


def kb_rung_promote(scores, n_cands, base=0, frac_num=2, frac_den=5, stream=None):
    """Enqueue the promotion decision over a device buffer of n_cands
    kb_rung_score (e.g. the scores kb_rung_stats returned).  Returns device
    int32 tensors (rank, order, promoted)."""
    torch = _torch()
    dev = scores.device
    rank = torch.empty(n_cands, dtype=torch.int32, device=dev)
    order = torch.empty(n_cands, dtype=torch.int32, device=dev)
    promoted = torch.empty(n_cands, dtype=torch.int32, device=dev)
    _check(lib().kb_rung_promote(ctypes.c_void_p(scores.data_ptr()), int(n_cands), int(base),
                                 int(frac_num), int(frac_den), ctypes.c_void_p(rank.data_ptr()),
                                 ctypes.c_void_p(order.data_ptr()),
                                 ctypes.c_void_p(promoted.data_ptr()), _stream_handle(stream)))
    return rank, order, promoted


def kb_rung_survival(entering, failed, promoted, original):
    """Table A.1's Fail% and Promotion% per rung (host only): two lists."""
    n = len(entering)
    arr = lambda v: (ctypes.c_int32 * max(1, n))(*[int(x) for x in v])
    fp = (ctypes.c_double * max(1, n))()
    pp = (ctypes.c_double * max(1, n))()
    _check(lib().kb_rung_survival(arr(entering), arr(failed), arr(promoted), n, int(original), fp, pp))
    return list(fp)[:n], list(pp)[:n]


MAX_OUTPUTS = 64


def kb_screen_multi(refs, cands, atol, rtol, flags=0, workspace=None, d_stats=None, stream=None):
    """Enqueue the screen of multi-output candidates.  refs: list of
    n_outputs reference tensors; cands: list of n_cands lists of n_outputs
    tensors (or None); atol, rtol: per-output lists (or one value for all).
    Returns (d_stats, workspace); the records are output-major."""
    torch = _torch()
    n_out, n = len(refs), len(cands)
    if isinstance(atol, (int, float)):
        atol = [atol] * n_out
    if isinstance(rtol, (int, float)):
        rtol = [rtol] * n_out
    R = (KbTensor * max(1, n_out))(*[describe(r) for r in refs])
    C = (KbTensor * max(1, n * n_out))(*[describe(c) for row in cands for c in row])
    if workspace is None:
        nbytes = lib().kb_screen_multi_workspace_bytes(R, n_out, max(1, n))
        if nbytes == 0:
            raise KbError(KB_ERR_INVALID_ARG, "no multi-output workspace size for these arguments")
        workspace = torch.empty(nbytes, dtype=torch.uint8, device=refs[0].device)
        kb_screen_workspace_init(workspace, stream)
    if d_stats is None:
        d_stats = alloc_stats(max(1, n * n_out), refs[0].device)
    A = (ctypes.c_float * max(1, n_out))(*[float(x) for x in atol])
    T = (ctypes.c_float * max(1, n_out))(*[float(x) for x in rtol])
    opts, keep = _one_off_opts(lib().kb_screen_multi_host_table_bytes(n_out, max(1, n)), stream)
    _check(lib().kb_screen_multi(R, n_out, C, n, A, T, int(flags),
                                 ctypes.c_void_p(workspace.data_ptr()), workspace.numel(),
                                 ctypes.c_void_p(d_stats.data_ptr()),
                                 ctypes.byref(opts) if opts is not None else None, _stream_handle(stream)))
    _after_one_off(keep, stream)
    return d_stats, workspace


class MultiScreener:
    """Repeated kb_screen_multi calls over one fixed set of buffers, with the
    argument marshalling (descriptors, tolerances, workspace, records, stream
    handle) done once at construction, as Screener does for one output."""

    def __init__(self, refs, cands, atol, rtol, flags=0, stream=None):
        torch = _torch()
        self.n_out, self.n = len(refs), len(cands)
        if isinstance(atol, (int, float)):
            atol = [atol] * self.n_out
        if isinstance(rtol, (int, float)):
            rtol = [rtol] * self.n_out
        self._keep = (list(refs), [list(row) for row in cands])
        self._R = (KbTensor * max(1, self.n_out))(*[describe(r) for r in refs])
        self._C = (KbTensor * max(1, self.n * self.n_out))(*[describe(c) for row in cands for c in row])
        self._A = (ctypes.c_float * max(1, self.n_out))(*[float(x) for x in atol])
        self._T = (ctypes.c_float * max(1, self.n_out))(*[float(x) for x in rtol])
        self.flags = int(flags)
        self._L = lib()
        nbytes = self._L.kb_screen_multi_workspace_bytes(self._R, self.n_out, max(1, self.n))
        if nbytes == 0:
            raise KbError(KB_ERR_INVALID_ARG, "no multi-output workspace size for these arguments")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=refs[0].device)
        kb_screen_workspace_init(self.workspace, stream)
        self.d_stats = alloc_stats(max(1, self.n * self.n_out), refs[0].device)
        self._ws = ctypes.c_void_p(self.workspace.data_ptr())
        self._st = ctypes.c_void_p(self.d_stats.data_ptr())
        self._stream = _stream_handle(stream)
        self.stream = stream
        tb = self._L.kb_screen_multi_host_table_bytes(self.n_out, max(1, self.n))
        self._tables = HostTables(tb, count=4) if tb > 0 else None

    def launch(self):
        i, opts = self._tables.acquire() if self._tables else (None, None)
        _check(self._L.kb_screen_multi(self._R, self.n_out, self._C, self.n, self._A, self._T, self.flags,
                                       self._ws, self.workspace.numel(), self._st,
                                       ctypes.byref(opts) if opts is not None else None, self._stream))
        if self._tables:
            self._tables.release(i, self.stream)

    def records(self):
        """All n_out * n_cands records, output-major (synchronizes the stream)."""
        recs, _ = kb_screen_stats(self.d_stats, self.n * self.n_out, stream=self.stream)
        return recs


def screen_multi(refs, cands, atol, rtol, flags=0, stream=None):
    """Gate + screen + readback of multi-output candidates: (records[o][k]
    dicts, summary dict, passed list)."""
    n_out, n = len(refs), len(cands)
    d_stats, _ = kb_screen_multi(refs, cands, atol, rtol, flags, stream=stream)
    recs, _ = kb_screen_stats(d_stats, n * n_out, stream=stream)
    host = (KbStats * max(1, n * n_out))()
    for i, r in enumerate(recs):
        for name, _ in KbStats._fields_:
            setattr(host[i], name, r[name])
    summ = KbSummary()
    passed = (ctypes.c_int32 * max(1, n))()
    _check(lib().kb_summarize_multi(host, n_out, n, ctypes.byref(summ), passed))
    return ([recs[o * n:(o + 1) * n] for o in range(n_out)], summ.as_dict(), list(passed)[:n])


def kb_gen_inputs(dst, dist, p0=0.0, p1=1.0, seed=0, stream_id=0, sub=0, offset=0, stream=None):
    """Fill torch tensor dst (contiguous) with elements offset.. of the seeded stream."""
    if not dst.is_contiguous():
        raise ValueError("dst must be contiguous")
    _check(lib().kb_gen_inputs(ctypes.c_void_p(dst.data_ptr()), dtype_code(dst), dst.numel(),
                               int(dist), float(p0), float(p1), int(seed), int(stream_id),
                               int(sub), int(offset), _stream_handle(stream)))
    return dst


def kb_gen_softmax_rows(dst, sigma, seed=0, stream_id=0, sub=0, stream=None):
    """Fill a contiguous float32 [rows, cols] tensor with softmax rows of NORMAL(0, sigma) logits."""
    if not dst.is_contiguous() or dst.dim() != 2:
        raise ValueError("dst must be a contiguous 2-d tensor")
    _check(lib().kb_gen_softmax_rows(ctypes.c_void_p(dst.data_ptr()), dtype_code(dst), dst.shape[0],
                                     dst.shape[1], float(sigma), int(seed), int(stream_id), int(sub),
                                     _stream_handle(stream)))
    return dst


def kb_gen_indices(m, n, device, seed=0, stream_id=0, sub=0, stream=None):
    """m distinct indices in [0, n), in draw order: a device int64 tensor
    holding the library's uint64 values (all below 2^63)."""
    torch = _torch()
    out = torch.empty(max(1, m), dtype=torch.int64, device=device)
    _check(lib().kb_gen_indices(ctypes.c_void_p(out.data_ptr()), int(m), int(n), int(seed), int(stream_id),
                                int(sub), _stream_handle(stream)))
    return out[:m]


def kb_gen_perturb(dst, src, op, a=0.0, b=0.0, p=0.0, seed=0, stream_id=0, sub=0, offset=0, stream=None):
    """dst = op(src) elementwise (contiguous tensors of one dtype; dst may be src)."""
    if not (dst.is_contiguous() and src.is_contiguous()) or dst.numel() != src.numel() or dst.dtype != src.dtype:
        raise ValueError("dst and src must be contiguous tensors of one size and dtype")
    _check(lib().kb_gen_perturb(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(src.data_ptr()), dtype_code(dst),
                                dst.numel(), int(op), float(a), float(b), float(p), int(seed), int(stream_id),
                                int(sub), int(offset), _stream_handle(stream)))
    return dst


def kb_gen_scatter(dst, ref, idx, mode, stream=None):
    """dst[idx] = NaN (KB_SCATTER_NAN) or the infinity with ref's sign (KB_SCATTER_INF_SIGN_OF_REF)."""
    torch = _torch()
    if not (dst.is_contiguous() and ref.is_contiguous()) or dst.numel() != ref.numel() or dst.dtype != ref.dtype:
        raise ValueError("dst and ref must be contiguous tensors of one size and dtype")
    if idx.dtype != torch.int64 or not idx.is_contiguous():
        raise ValueError("idx must be a contiguous int64 tensor")
    _check(lib().kb_gen_scatter(ctypes.c_void_p(dst.data_ptr()), ctypes.c_void_p(ref.data_ptr()), dtype_code(dst),
                                dst.numel(), ctypes.c_void_p(idx.data_ptr()), idx.numel(), int(mode),
                                _stream_handle(stream)))
    return dst


def kb_summarize(records):
    """Verdict summary (dict) of a list of record dicts or a KbStats array."""
    if isinstance(records, list):
        arr = (KbStats * max(1, len(records)))()
        for k, r in enumerate(records):
            for name, _ in KbStats._fields_:
                setattr(arr[k], name, r[name])
        n = len(records)
    else:
        arr, n = records, len(records)
    summ = KbSummary()
    _check(lib().kb_summarize(arr, n, ctypes.byref(summ), None))
    return summ.as_dict()


def screen(ref, cands, atol, rtol, flags=0, stream=None):
    """Gate + screen + readback: (list of per-candidate dicts, summary dict)."""
    d_stats, _ = kb_screen(ref, cands, atol, rtol, flags, stream=stream)
    return kb_screen_stats(d_stats, len(cands), stream=stream)


class Screener:
    """Repeated screening of one fixed set of buffers with the argument
    marshalling done once: descriptors, workspace, record buffers and the
    stream handle are built at construction and reused by every launch.

    host_slots > 0 places the records in that many pinned host buffers that
    the kernel writes directly (a pipelined caller launches into one slot and
    summarizes another after an event); otherwise they go to device memory
    and read() copies them back.  positions=True also finds the positions in
    the same pass (positions() copies them back)."""

    def __init__(self, ref, cands, atol, rtol, flags=0, stream=None, host_slots=0, positions=False):
        torch = _torch()
        self.ref, self.cands = ref, list(cands)
        self.n = len(self.cands)
        self.atol, self.rtol, self.flags = float(atol), float(rtol), int(flags)
        self.stream = stream
        self._stream = _stream_handle(stream)
        self._ref = describe(ref)
        self._arr = (KbTensor * max(1, self.n))(*[describe(c) for c in self.cands])
        self.workspace = alloc_workspace(max(1, self.n), ref.numel(), self._ref.dtype, ref.device,
                                         stream, positions=positions)
        self.d_loc = alloc_locate(max(1, self.n), ref.device) if positions else None
        self._ws = ctypes.c_void_p(self.workspace.data_ptr())
        nbytes = max(1, self.n) * ctypes.sizeof(KbStats)
        if host_slots > 0:
            self.slots = [torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
                          for _ in range(host_slots)]
            self._views = [ctypes.cast(ctypes.c_void_p(t.data_ptr()), ctypes.POINTER(KbStats))
                           for t in self.slots]
        else:
            self.slots = [alloc_stats(max(1, self.n), ref.device)]
            self._views = None
        self._slot_ptr = [ctypes.c_void_p(t.data_ptr()) for t in self.slots]
        self._host = (KbStats * max(1, self.n))()
        self._passed = (ctypes.c_int32 * max(1, self.n))()
        self._summary = KbSummary()
        self._L = lib()
        # more than KB_INLINE_CANDS candidates: a ring of pinned launch
        # tables, one per record slot (at least two)
        tb = self._L.kb_screen_host_table_bytes(max(1, self.n))
        self._tables = HostTables(tb, count=max(2, len(self.slots))) if tb > 0 else None
        self._opts = None
        if self.d_loc is not None:
            if self._tables:
                for o in self._tables.opts:
                    o.d_loc = self.d_loc.data_ptr()
            else:
                self._opts = KbScreenOpts(None, 0, self.d_loc.data_ptr())

    @property
    def d_stats(self):
        return self.slots[0]

    def launch(self, slot=0):
        i, opts = self._tables.acquire() if self._tables else (None, self._opts)
        _check(self._L.kb_screen_ex(ctypes.byref(self._ref), self._arr, self.n, self.atol, self.rtol,
                                    self.flags, self._ws, self.workspace.numel(),
                                    self._slot_ptr[slot], ctypes.byref(opts) if opts is not None else None,
                                    self._stream))
        if self._tables:
            self._tables.release(i, self.stream)

    def read(self, slot=0):
        """Copy the records back (synchronizes the stream); returns the
        summary (the verdicts are kept for records())."""
        _check(self._L.kb_screen_stats(self._slot_ptr[slot], self.n, self._host,
                                       ctypes.byref(self._summary), self._passed, self._stream))
        return self._summary

    def summarize(self, slot):
        """Summary of a pinned host slot; the caller has synchronized past the launch."""
        _check(self._L.kb_summarize(self._views[slot], self.n, ctypes.byref(self._summary),
                                    self._passed))
        return self._summary

    def records(self, slot=None):
        """Record dicts of the last read() (slot None) or of a pinned slot,
        each with the library's verdict as "passed"."""
        if slot is None:
            src = self._host
        else:
            src = self._views[slot]
            _check(self._L.kb_summarize(src, self.n, None, self._passed))
        return [src[k].as_dict(self._passed[k]) for k in range(self.n)]

    def positions(self):
        """Wait for the launch stream, then copy the positions of the last
        launch back (positions=True only)."""
        _sync_stream(self.stream)
        return read_locate(self.d_loc, self.n)

    def launch_plan(self):
        return kb_screen_launch(max(1, self.n), self.ref.numel(), self._ref.dtype)
