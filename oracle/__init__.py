"""CPU oracle for the candidate-screening path (ctypes over oracle/libkbo.so).

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the
benchmark's CPU-baseline leg are its only users; the product package never
imports it.  See kbo.c for what each function computes and how it is pinned.

Arrays are numpy arrays holding raw storage: float32 for f32, and uint16 (or
float16) bit patterns for f16 and bf16.
"""
import ctypes
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from . import build as _build

F32, F16, BF16, U32 = 0, 1, 2, 3
DIST_U32, DIST_UNIFORM, DIST_NORMAL, DIST_STUDENT_T3 = 0, 1, 2, 3
(PERTURB_ADD_UNIFORM, PERTURB_REL_UNIFORM, PERTURB_ADD_NORMAL, PERTURB_SCALE_WHERE,
 PERTURB_FLIP_LSB_WHERE, PERTURB_SPECIALS, PERTURB_ZERO_SUBNORMAL_REL) = range(1, 8)
SCATTER_NAN, SCATTER_INF_SIGN_OF_REF = 1, 2
EQUAL_NAN = 1
DTYPES = {"f32": F32, "f16": F16, "bf16": BF16, "u32": U32}
NP_STORAGE = {F32: np.float32, F16: np.uint16, BF16: np.uint16, U32: np.uint32}


class Partial(ctypes.Structure):
    _fields_ = [("numel", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
                ("nan_count", ctypes.c_uint64), ("pos_inf_count", ctypes.c_uint64),
                ("neg_inf_count", ctypes.c_uint64),
                ("sum_sq_diff", ctypes.c_double), ("sum_sq_diff_comp", ctypes.c_double),
                ("sum_sq_ref", ctypes.c_double), ("sum_sq_ref_comp", ctypes.c_double),
                ("max_abs_err", ctypes.c_float), ("max_rel_err", ctypes.c_float),
                ("bitdiff", ctypes.c_uint32), ("_pad", ctypes.c_uint32)]


class Stats(ctypes.Structure):
    _fields_ = [("numel", ctypes.c_uint64), ("mismatches", ctypes.c_uint64),
                ("nan_count", ctypes.c_uint64), ("pos_inf_count", ctypes.c_uint64),
                ("neg_inf_count", ctypes.c_uint64),
                ("sum_sq_diff", ctypes.c_double), ("sum_sq_ref", ctypes.c_double),
                ("rel_l2", ctypes.c_double),
                ("max_abs_err", ctypes.c_float), ("max_rel_err", ctypes.c_float),
                ("bitwise_equal", ctypes.c_int32), ("passed", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class RowStats(ctypes.Structure):
    _fields_ = [("mean", ctypes.c_double), ("p50", ctypes.c_double), ("p90", ctypes.c_double),
                ("p95", ctypes.c_double), ("p99", ctypes.c_double), ("tail90", ctypes.c_double),
                ("tail95", ctypes.c_double), ("tail99", ctypes.c_double),
                ("speedup", ctypes.c_double), ("n", ctypes.c_int32), ("valid", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


class RungScore(ctypes.Structure):
    _fields_ = [("latency", ctypes.c_double), ("score", ctypes.c_double),
                ("speedup", ctypes.c_double), ("valid", ctypes.c_int32), ("_pad", ctypes.c_int32)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_ if name != "_pad"}


_lib = None


def lib():
    """Load oracle/libkbo.so, building it first if it is missing.  The
    environment variable KBO_LIB names another build of the same sources to
    load instead (the mutation test runs the pins against copies of the
    oracle with a planted mistake)."""
    global _lib
    if _lib is None:
        path = os.environ.get("KBO_LIB") or _build.LIB
        if path == _build.LIB and not os.path.exists(path):
            _build.build()
        L = ctypes.CDLL(path)
        u32, u64, f32, vp = ctypes.c_uint32, ctypes.c_uint64, ctypes.c_float, ctypes.c_void_p
        L.kbo_philox4x32_10.argtypes = [ctypes.POINTER(u32), ctypes.POINTER(u32),
                                        ctypes.POINTER(u32)]
        L.kbo_stream_block.argtypes = [u64, u32, u32, u64, ctypes.POINTER(u32)]
        L.kbo_u01.argtypes = [u32]
        L.kbo_u01.restype = f32
        L.kbo_uniform.argtypes = [u32, f32, f32]
        L.kbo_uniform.restype = f32
        L.kbo_normal01.argtypes = [u32, u32, ctypes.c_int]
        L.kbo_normal01.restype = f32
        L.kbo_f32_to_f16.argtypes = [f32]
        L.kbo_f32_to_f16.restype = ctypes.c_uint16
        L.kbo_f32_to_bf16.argtypes = [f32]
        L.kbo_f32_to_bf16.restype = ctypes.c_uint16
        L.kbo_f16_to_f32.argtypes = [ctypes.c_uint16]
        L.kbo_f16_to_f32.restype = f32
        L.kbo_bf16_to_f32.argtypes = [ctypes.c_uint16]
        L.kbo_bf16_to_f32.restype = f32
        L.kbo_gen.argtypes = [vp, ctypes.c_int, u64, ctypes.c_int, f32, f32, u64, u32, u32, u64]
        L.kbo_gen.restype = ctypes.c_int
        L.kbo_box_muller64.argtypes = [u32, u32, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(ctypes.c_double)]
        L.kbo_student_t3_64.argtypes = [ctypes.POINTER(u32)]
        L.kbo_student_t3_64.restype = ctypes.c_double
        L.kbo_student_t3.argtypes = [ctypes.POINTER(u32)]
        L.kbo_student_t3.restype = f32
        L.kbo_softmax_row.argtypes = [vp, u64, vp]
        L.kbo_gen_softmax_rows.argtypes = [vp, u64, u64, u64, f32, u64, u32, u32]
        L.kbo_gen_softmax_rows.restype = ctypes.c_int
        L.kbo_gen_indices.argtypes = [vp, u32, u64, u64, u32, u32]
        L.kbo_gen_indices.restype = ctypes.c_int
        L.kbo_perturb.argtypes = [vp, vp, ctypes.c_int, u64, ctypes.c_int, f32, f32, f32, u64, u32, u32, u64]
        L.kbo_perturb.restype = ctypes.c_int
        L.kbo_scatter.argtypes = [vp, vp, ctypes.c_int, u64, vp, u32, ctypes.c_int]
        L.kbo_scatter.restype = ctypes.c_int
        L.kbo_partial_init.argtypes = [ctypes.POINTER(Partial)]
        L.kbo_screen_range.argtypes = [ctypes.c_int, vp, vp, u64, u64, f32, f32, u32,
                                       ctypes.POINTER(Partial)]
        L.kbo_screen_range.restype = ctypes.c_int
        L.kbo_merge.argtypes = [ctypes.POINTER(Partial), ctypes.POINTER(Partial)]
        L.kbo_finalize.argtypes = [ctypes.POINTER(Partial), ctypes.POINTER(Stats)]
        L.kbo_screen.argtypes = [ctypes.c_int, vp, vp, u64, f32, f32, u32, ctypes.POINTER(Stats)]
        L.kbo_screen.restype = ctypes.c_int
        L.kbo_match.argtypes = [f32, f32, f32, f32, u32]
        L.kbo_match.restype = ctypes.c_int
        L.kbo_locate.argtypes = [ctypes.c_int, vp, vp, u64, f32, f32, u32, f32, f32,
                                 ctypes.POINTER(ctypes.c_int64 * 3)]
        L.kbo_locate.restype = ctypes.c_int
        for name in ("kbo_f32_to_f16_n", "kbo_f32_to_bf16_n", "kbo_f16_to_f32_n",
                     "kbo_bf16_to_f32_n"):
            getattr(L, name).argtypes = [vp, vp, u64]
        L.kbo_uniform_n.argtypes = [vp, f32, f32, vp, u64]
        L.kbo_match16_n.argtypes = [ctypes.c_int, vp, vp, f32, f32, u32, vp, u64]
        d, i = ctypes.c_double, ctypes.c_int
        L.kbo_quantile_sorted.argtypes = [vp, i, d]
        L.kbo_quantile_sorted.restype = d
        L.kbo_row_stats.argtypes = [vp, i, ctypes.POINTER(RowStats)]
        L.kbo_rung_score_of.argtypes = [d, i, d, d, d]
        L.kbo_rung_score_of.restype = d
        L.kbo_rung_stats.argtypes = [vp, i, i, i, i, i, d, d, d, ctypes.POINTER(RowStats),
                                     ctypes.POINTER(RungScore)]
        L.kbo_rung_stats.restype = ctypes.c_int
        L.kbo_rung_promote.argtypes = [vp, vp, i, i, i, i, vp, vp, vp]
        L.kbo_rung_promote.restype = ctypes.c_int
        L.kbo_rung_survival.argtypes = [vp, vp, vp, i, i, vp, vp]
        L.kbo_rung_survival.restype = ctypes.c_int
        _lib = L
    return _lib


def _code(dtype):
    return DTYPES[dtype] if isinstance(dtype, str) else int(dtype)


def philox4x32_10(counter, key):
    c = (ctypes.c_uint32 * 4)(*counter)
    k = (ctypes.c_uint32 * 2)(*key)
    o = (ctypes.c_uint32 * 4)()
    lib().kbo_philox4x32_10(c, k, o)
    return tuple(o)


def stream_block(seed, stream_id, sub, b):
    o = (ctypes.c_uint32 * 4)()
    lib().kbo_stream_block(seed, stream_id, sub, b, o)
    return tuple(o)


def u01(x):
    return lib().kbo_u01(x)


def uniform(x, a, b):
    return lib().kbo_uniform(x, a, b)


def normal01(xa, xb, odd):
    return lib().kbo_normal01(xa, xb, odd)


def gen(dtype, n, dist, p0=0.0, p1=1.0, seed=0, stream_id=0, sub=0, offset=0):
    """Elements offset..offset+n-1 of a stream, as a numpy storage array."""
    code = _code(dtype)
    out = np.empty(n, dtype=NP_STORAGE[code])
    rc = lib().kbo_gen(out.ctypes.data, code, n, dist, p0, p1, seed, stream_id, sub, offset)
    if rc != 0:
        raise ValueError("invalid (dtype, dist) pair")
    return out


def box_muller64(xa, xb):
    """(cosine, sine) branches in binary64, unrounded."""
    c, s_ = ctypes.c_double(), ctypes.c_double()
    lib().kbo_box_muller64(xa, xb, ctypes.byref(c), ctypes.byref(s_))
    return c.value, s_.value


def student_t3(words, exact=False):
    """Student-t (3) of one block's four words: binary32, or binary64 with exact=True."""
    w = (ctypes.c_uint32 * 4)(*words)
    return lib().kbo_student_t3_64(w) if exact else lib().kbo_student_t3(w)


def softmax_row(x):
    """Softmax of one row of binary32 logits (binary64 inside, rounded once)."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.empty_like(x)
    lib().kbo_softmax_row(x.ctypes.data, x.size, out.ctypes.data)
    return out


def gen_softmax_rows(rows, cols, sigma, seed=0, stream_id=0, sub=0, row0=0):
    """Rows row0..row0+rows-1 of the softmax tensor of NORMAL(0, sigma) logits, float32 [rows, cols]."""
    out = np.empty((rows, cols), dtype=np.float32)
    if lib().kbo_gen_softmax_rows(out.ctypes.data, row0, rows, cols, sigma, seed, stream_id, sub) != 0:
        raise ValueError("cols must be >= 1")
    return out


def gen_indices(m, n, seed=0, stream_id=0, sub=0):
    """m distinct indices in [0, n) in draw order (uint64 array)."""
    out = np.empty(max(1, m), dtype=np.uint64)
    if lib().kbo_gen_indices(out.ctypes.data, m, n, seed, stream_id, sub) != 0:
        raise ValueError("need 1 <= n and m <= n")
    return out[:m]


def perturb(src, dtype, op, a=0.0, b=0.0, p=0.0, seed=0, stream_id=0, sub=0, offset=0):
    """A new storage array: the planted change `op` applied to storage array src."""
    code = _code(dtype)
    src = _storage(src, code)
    out = np.empty_like(src)
    rc = lib().kbo_perturb(out.ctypes.data, src.ctypes.data, code, src.size, op, a, b, p, seed, stream_id,
                           sub, offset)
    if rc != 0:
        raise ValueError("op %d not defined for dtype code %d" % (op, code))
    return out


def scatter(dst, ref, dtype, idx, mode):
    """In place: dst[idx] = NaN (mode 1) or the infinity with ref's sign (mode 2)."""
    code = _code(dtype)
    dst = _storage(dst, code)
    ref = _storage(ref, code)
    idx = np.ascontiguousarray(idx, dtype=np.uint64)
    if lib().kbo_scatter(dst.ctypes.data, ref.ctypes.data, code, dst.size, idx.ctypes.data, idx.size,
                         mode) != 0:
        raise ValueError("bad mode or dtype")
    return dst


def _storage(a, code):
    a = np.ascontiguousarray(a)
    want = 4 if code == F32 else 2
    if a.dtype.itemsize != want:
        raise TypeError("storage itemsize %d does not fit dtype code %d" % (a.dtype.itemsize, code))
    return a


def screen_partial(ref, cand, dtype, atol, rtol, flags=0, lo=0, hi=None):
    code = _code(dtype)
    ref = _storage(ref, code)
    cand = _storage(cand, code)
    if hi is None:
        hi = ref.size
    p = Partial()
    lib().kbo_partial_init(ctypes.byref(p))
    rc = lib().kbo_screen_range(code, ref.ctypes.data, cand.ctypes.data, lo, hi, atol, rtol,
                                flags, ctypes.byref(p))
    if rc != 0:
        raise ValueError("bad dtype")
    return p


def merge(parts):
    acc = Partial()
    lib().kbo_partial_init(ctypes.byref(acc))
    for p in parts:
        lib().kbo_merge(ctypes.byref(acc), ctypes.byref(p))
    return acc


def finalize(p):
    s = Stats()
    lib().kbo_finalize(ctypes.byref(p), ctypes.byref(s))
    return s.as_dict()


def screen(ref, cand, dtype, atol, rtol, flags=0, chunk=None, threads=1):
    """Statistics of one candidate against the reference.

    With chunk set, [0, n) is cut into chunks screened independently (on up
    to `threads` host threads; ctypes releases the GIL) and merged in chunk
    order, which is the merge law applied to a partition of the elements.
    """
    code = _code(dtype)
    ref = _storage(ref, code)
    cand = _storage(cand, code)
    n = ref.size
    if cand.size != n:
        raise ValueError("size mismatch")
    if not chunk or chunk >= n:
        return finalize(screen_partial(ref, cand, code, atol, rtol, flags))
    bounds = [(lo, min(n, lo + chunk)) for lo in range(0, n, chunk)]
    if threads > 1:
        with ThreadPoolExecutor(threads) as ex:
            parts = list(ex.map(lambda b: screen_partial(ref, cand, code, atol, rtol, flags,
                                                          b[0], b[1]), bounds))
    else:
        parts = [screen_partial(ref, cand, code, atol, rtol, flags, lo, hi) for lo, hi in bounds]
    return finalize(merge(parts))


def locate(ref, cand, dtype, atol, rtol, max_abs, max_rel, flags=0):
    """(first_mismatch, max_abs_index, max_rel_index) of one candidate, -1
    where none; max_abs / max_rel are the candidate's maxima."""
    code = _code(dtype)
    ref = _storage(ref, code)
    cand = _storage(cand, code)
    if cand.size != ref.size:
        raise ValueError("size mismatch")
    out = (ctypes.c_int64 * 3)()
    rc = lib().kbo_locate(code, ref.ctypes.data, cand.ctypes.data, ref.size, atol, rtol, flags,
                          max_abs, max_rel, ctypes.byref(out))
    if rc:
        raise ValueError("bad dtype")
    return tuple(out)


# ---- rung benchmarker statistics (kbo_rung.c) ----

ALPHA, BETA = 0.02, 0.01  # Appendix A.2


def quantile_sorted(x, p):
    """p-quantile of a 1-D array sorted ascending (linear interpolation)."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    return lib().kbo_quantile_sorted(x.ctypes.data, x.size, float(p))


def row_stats(t):
    """Statistics of one row of timing samples (dict; speedup NaN)."""
    t = np.ascontiguousarray(t, dtype=np.float64)
    out = RowStats()
    lib().kbo_row_stats(t.ctypes.data, t.size, ctypes.byref(out))
    return out.as_dict()


def rung_score_of(latency, rung, budget, alpha=ALPHA, beta=BETA):
    return lib().kbo_rung_score_of(float(latency), int(rung), float(budget), float(alpha),
                                   float(beta))


def rung_stats(samples, base=0, rung=0, budget=0.0, alpha=ALPHA, beta=BETA):
    """samples: array [n_cands][n_shapes][n_iter] of timing samples (us).
    Returns (rows: list of n_cands lists of n_shapes dicts, scores: list of
    n_cands dicts)."""
    a = np.ascontiguousarray(samples, dtype=np.float64)
    if a.ndim != 3:
        raise ValueError("samples must be [n_cands][n_shapes][n_iter]")
    C, S, N = a.shape
    rows = (RowStats * (C * S))()
    scores = (RungScore * C)()
    rc = lib().kbo_rung_stats(a.ctypes.data, C, S, N, int(base), int(rung), float(budget),
                              float(alpha), float(beta), rows, scores)
    if rc:
        raise ValueError("bad sizes")
    return ([[rows[c * S + s].as_dict() for s in range(S)] for c in range(C)],
            [scores[c].as_dict() for c in range(C)])


def rung_promote(scores, valid, base=0, num=2, den=5):
    """The promotion decision over one rung's candidates: (rank, order,
    promoted) as int32 arrays."""
    sc = np.ascontiguousarray(scores, dtype=np.float64)
    va = np.ascontiguousarray(valid, dtype=np.int32)
    n = sc.size
    rank = np.empty(n, np.int32)
    order = np.empty(n, np.int32)
    prom = np.empty(n, np.int32)
    rc = lib().kbo_rung_promote(sc.ctypes.data, va.ctypes.data, n, int(base), int(num), int(den),
                                rank.ctypes.data, order.ctypes.data, prom.ctypes.data)
    if rc:
        raise ValueError("bad arguments")
    return rank, order, prom


def rung_survival(entering, failed, promoted, original):
    """Table A.1's Fail% and Promotion% per rung (two float64 arrays)."""
    e = np.ascontiguousarray(entering, dtype=np.int32)
    f = np.ascontiguousarray(failed, dtype=np.int32)
    p = np.ascontiguousarray(promoted, dtype=np.int32)
    fp = np.empty(e.size)
    pp = np.empty(e.size)
    rc = lib().kbo_rung_survival(e.ctypes.data, f.ctypes.data, p.ctypes.data, e.size, int(original),
                                 fp.ctypes.data, pp.ctypes.data)
    if rc:
        raise ValueError("bad arguments")
    return fp, pp


# ---- multi-output candidates ----

STATUS_OK, REJECT_NULL, REJECT_DTYPE, REJECT_SHAPE, REJECT_LAYOUT = 0, 1, 2, 3, 4


def gate_status(ref, cand):
    """The policy gate of one output (Section 3.2: the output's shape and
    dtype against the reference's), plus the two checks a tensor view needs
    before it can be read: data present, dense row-major layout.  ref and
    cand are dicts {"null": bool, "dtype": int, "shape": tuple, "strides":
    tuple} (cand may be None: a missing output).  The first failing check,
    in the order null, dtype, shape, layout."""
    if cand is None:
        return REJECT_NULL
    numel = 1
    for d in cand["shape"]:
        numel *= d
    if cand["null"] and numel != 0:
        return REJECT_NULL
    if cand["dtype"] != ref["dtype"]:
        return REJECT_DTYPE
    if tuple(cand["shape"]) != tuple(ref["shape"]):
        return REJECT_SHAPE
    if numel != 0:
        expect = 1
        for d, st in zip(reversed(cand["shape"]), reversed(cand["strides"])):
            if d != 1 and st != expect:
                return REJECT_LAYOUT
            expect *= d
    return STATUS_OK


def rejected_record(status):
    rec = {f: 0 for f in ("numel", "mismatches", "nan_count", "pos_inf_count", "neg_inf_count",
                          "bitwise_equal", "passed")}
    rec.update({"sum_sq_diff": 0.0, "sum_sq_ref": 0.0, "rel_l2": 0.0, "max_abs_err": 0.0,
                "max_rel_err": 0.0, "status": status})
    return rec


def screen_multi(refs, cands, atol, rtol, flags=0):
    """Multi-output screen.  refs: list of (meta, storage, dtype name);
    cands: list of per-candidate lists of (meta or None, storage or None);
    atol, rtol: per-output lists.  One gate over all outputs: a candidate is
    read only if every output passes; otherwise each of its records has the
    first failing status of the first failing output.  Returns (records as
    records[o][k], passed[k]: every output passes and matches)."""
    n_out = len(refs)
    status = []
    for row in cands:
        st = STATUS_OK
        for o in range(n_out):
            st = gate_status(refs[o][0], row[o][0])
            if st != STATUS_OK:
                break
        status.append(st)
    records = [[None] * len(cands) for _ in range(n_out)]
    for k, row in enumerate(cands):
        for o in range(n_out):
            if status[k] != STATUS_OK:
                records[o][k] = rejected_record(status[k])
            else:
                r = screen(refs[o][1], row[o][1], refs[o][2], atol[o], rtol[o], flags)
                r["status"] = STATUS_OK
                records[o][k] = r
    passed = [int(status[k] == STATUS_OK and all(records[o][k]["mismatches"] == 0
                                                  for o in range(n_out)))
              for k in range(len(cands))]
    return records, passed


def match(c, r, atol, rtol, flags=0):
    return bool(lib().kbo_match(c, r, atol, rtol, flags))


def f32_to_f16(x):
    return lib().kbo_f32_to_f16(x)


def f32_to_bf16(x):
    return lib().kbo_f32_to_bf16(x)


def f16_to_f32(h):
    return lib().kbo_f16_to_f32(h)


def bf16_to_f32(h):
    return lib().kbo_bf16_to_f32(h)


def _bulk(name, inp, out_dtype):
    inp = np.ascontiguousarray(inp)
    out = np.empty(inp.size, dtype=out_dtype)
    getattr(lib(), name)(inp.ctypes.data, out.ctypes.data, inp.size)
    return out


def f32_to_f16_n(x):
    return _bulk("kbo_f32_to_f16_n", np.asarray(x, dtype=np.float32), np.uint16)


def f32_to_bf16_n(x):
    return _bulk("kbo_f32_to_bf16_n", np.asarray(x, dtype=np.float32), np.uint16)


def f16_to_f32_n(h):
    return _bulk("kbo_f16_to_f32_n", np.asarray(h, dtype=np.uint16), np.float32)


def bf16_to_f32_n(h):
    return _bulk("kbo_bf16_to_f32_n", np.asarray(h, dtype=np.uint16), np.float32)


def uniform_n(x, a, b):
    x = np.ascontiguousarray(x, dtype=np.uint32)
    out = np.empty(x.size, dtype=np.float32)
    lib().kbo_uniform_n(x.ctypes.data, a, b, out.ctypes.data, x.size)
    return out


def match16_n(dtype, c, r, atol, rtol, flags=0):
    c = np.ascontiguousarray(c, dtype=np.uint16)
    r = np.ascontiguousarray(r, dtype=np.uint16)
    out = np.empty(c.size, dtype=np.uint8)
    lib().kbo_match16_n(_code(dtype), c.ctypes.data, r.ctypes.data, atol, rtol, flags,
                        out.ctypes.data, c.size)
    return out
