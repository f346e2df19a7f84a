"""ctypes binding of libsaki.so (include/saki.h).

Argument marshalling only: every step of the path runs in the HIP library.
Tensors are torch device tensors; the library sees their data pointers and the
current torch stream.  If the built library is missing the binding raises; it
has no fallback.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsaki.so")

SAKI_F32, SAKI_BF16 = 0, 1
SAKI_OP_COUPLE, SAKI_OP_ROUTE, SAKI_OP_VERIFY, SAKI_OP_SELECT = 0, 1, 2, 3
SAKI_TARGET_MODE, SAKI_TARGET_SAMPLE = 0, 1
SAKI_SELECT_RANDOM, SAKI_SELECT_TV_WEIGHTED = 0, 1
SAKI_MAX_VOCAB = 1 << 21
SAKI_STATIC_MAX_ROWS = 262144
SAKI_CHUNK = 1024
ROW_OK, ROW_NONFINITE, ROW_BAD_DRAFT, ROW_SKIPPED = 0, 1, 2, 3

STATUS = {0: "SAKI_OK", 1: "SAKI_E_NULLPTR", 2: "SAKI_E_SHAPE", 3: "SAKI_E_VALUE",
          4: "SAKI_E_DTYPE", 5: "SAKI_E_ALIGN", 6: "SAKI_E_WORKSPACE", 7: "SAKI_E_DEVICE",
          8: "SAKI_E_LAUNCH"}

EXPORTED = ["saki_workspace_bytes", "saki_couple", "saki_couple_static", "saki_route_loss", "saki_spec_verify",
            "saki_select_positions", "saki_probe_metrics", "saki_sample", "saki_commit",
            "saki_status_str", "saki_last_error"]
SEQ_RUNNING, SEQ_FINISHED, SEQ_STOPPED = 0, 1, 2
SAKI_MAX_PROBE_K = 64


class SakiRows(ctypes.Structure):
    _fields_ = [("student", ctypes.c_void_p), ("teacher", ctypes.c_void_p),
                ("dtype", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("n_rows", ctypes.c_int64), ("vocab", ctypes.c_int64),
                ("row_stride", ctypes.c_int64), ("row_offset", ctypes.c_int64)]


COUPLE_FLOAT_FIELDS = ["lambda", "kl", "tv", "accept_prob", "margin", "logp_token",
                       "logt_token", "logq_token"]
COUPLE_INT_FIELDS = ["proposal", "token", "teacher_argmax", "target"]
COUPLE_U8_FIELDS = ["corrected", "row_status"]
# struct order of saki_couple_out
COUPLE_FIELDS = COUPLE_FLOAT_FIELDS + ["proposal", "token", "teacher_argmax"] + COUPLE_U8_FIELDS + ["target"]


class SakiCoupleOut(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in COUPLE_FIELDS]


class SakiRouteArgs(ctypes.Structure):
    _fields_ = [("valid_mask", ctypes.c_void_p), ("grad_scale", ctypes.c_float),
                ("grad_dtype", ctypes.c_int32), ("row_loss", ctypes.c_void_p),
                ("loss_sum", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("grad_stride", ctypes.c_int64), ("correction_target", ctypes.c_int32)]


# struct order of saki_traj after (n_seq, max_len)
TRAJ_FIELDS = ["tokens", "corrected", "lambda", "kl", "tv", "logp_token", "logt_token",
               "teacher_argmax", "length", "done"]
TRAJ_DTYPES = dict(tokens=torch.int32, corrected=torch.uint8, teacher_argmax=torch.int32,
                   length=torch.int32, done=torch.uint8)


class SakiTraj(ctypes.Structure):
    _fields_ = [("n_seq", ctypes.c_int64), ("max_len", ctypes.c_int64)] + \
               [(n, ctypes.c_void_p) for n in TRAJ_FIELDS]


class SakiError(RuntimeError):
    def __init__(self, status, detail):
        super().__init__(f"{STATUS.get(status, status)}: {detail}")
        self.status = status


_lib = None


def load(path=LIB_PATH):
    """Load libsaki.so once and declare its C signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libsaki.so not built at {path}; run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    lib.saki_workspace_bytes.restype = ctypes.c_size_t
    lib.saki_workspace_bytes.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_int64]
    lib.saki_couple.restype = ctypes.c_int
    lib.saki_couple.argtypes = [ctypes.POINTER(SakiRows), ctypes.c_double, ctypes.c_uint64,
                                ctypes.POINTER(SakiCoupleOut), ctypes.POINTER(SakiRouteArgs),
                                ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.saki_couple_static.restype = ctypes.c_int
    lib.saki_couple_static.argtypes = [ctypes.POINTER(SakiRows), ctypes.c_double, ctypes.c_uint64,
                                       ctypes.POINTER(SakiCoupleOut), ctypes.POINTER(SakiRouteArgs),
                                       ctypes.c_void_p]
    lib.saki_route_loss.restype = ctypes.c_int
    lib.saki_route_loss.argtypes = [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.POINTER(SakiRouteArgs), ctypes.c_void_p,
                                    ctypes.c_size_t, ctypes.c_void_p]
    lib.saki_spec_verify.restype = ctypes.c_int
    lib.saki_spec_verify.argtypes = [ctypes.POINTER(SakiRows), ctypes.c_int32, ctypes.c_void_p,
                                     ctypes.c_double, ctypes.c_uint64, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_void_p,
                                     ctypes.POINTER(SakiCoupleOut), ctypes.c_void_p,
                                     ctypes.c_size_t, ctypes.c_void_p]
    lib.saki_select_positions.restype = ctypes.c_int
    lib.saki_select_positions.argtypes = [ctypes.c_int32, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_uint64, ctypes.c_int64,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                                          ctypes.c_void_p]
    lib.saki_probe_metrics.restype = ctypes.c_int
    lib.saki_probe_metrics.argtypes = [ctypes.POINTER(SakiRows), ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                       ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.saki_sample.restype = ctypes.c_int
    lib.saki_sample.argtypes = [ctypes.POINTER(SakiRows), ctypes.c_int64, ctypes.c_uint64,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    lib.saki_commit.restype = ctypes.c_int
    lib.saki_commit.argtypes = [ctypes.POINTER(SakiTraj), ctypes.c_int32, ctypes.c_int32,
                                ctypes.c_void_p, ctypes.c_void_p, ctypes.POINTER(SakiCoupleOut),
                                ctypes.c_void_p, ctypes.c_void_p]
    lib.saki_status_str.restype = ctypes.c_char_p
    lib.saki_status_str.argtypes = [ctypes.c_int]
    lib.saki_last_error.restype = ctypes.c_char_p
    lib.saki_last_error.argtypes = []
    _lib = lib
    return lib


def _check(status):
    if status != 0:
        raise SakiError(status, _lib.saki_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dense(*ts):
    """Per-row arrays are passed as bare pointers: they must be contiguous."""
    for t in ts:
        if t is not None and not t.is_contiguous():
            raise ValueError("per-row arrays must be contiguous tensors")


def _dtype_code(dt):
    if dt == torch.float32:
        return SAKI_F32
    if dt == torch.bfloat16:
        return SAKI_BF16
    raise ValueError(f"unsupported dtype {dt}")


def _stream(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _rows(student, teacher, row_offset):
    assert student.dim() == 2 and student.shape == teacher.shape
    assert student.dtype == teacher.dtype and student.stride() == teacher.stride()
    assert student.stride(1) == 1
    return SakiRows(_ptr(student), _ptr(teacher), _dtype_code(student.dtype), 0,
                    student.shape[0], student.shape[1], student.stride(0), row_offset)


def workspace_bytes(op, n_rows, vocab):
    load()
    return int(_lib.saki_workspace_bytes(op, n_rows, vocab))


def alloc_rows(n_rows, vocab, dtype, device):
    """[n_rows, vocab] tensor whose row pitch is a multiple of 16 bytes (the ABI's layout rule)."""
    per = 16 // torch.tensor([], dtype=dtype).element_size()
    pitch = (vocab + per - 1) // per * per
    return torch.empty(n_rows, pitch, dtype=dtype, device=device)[:, :vocab]


def alloc_couple_out(n_rows, device, fields=COUPLE_FIELDS):
    out = {}
    for f in fields:
        if f in COUPLE_FLOAT_FIELDS:
            out[f] = torch.empty(n_rows, dtype=torch.float32, device=device)
        elif f in COUPLE_INT_FIELDS:
            out[f] = torch.empty(n_rows, dtype=torch.int32, device=device)
        else:
            out[f] = torch.empty(n_rows, dtype=torch.uint8, device=device)
    return out


def _couple_struct(out):
    return SakiCoupleOut(*[_ptr(out.get(f)) for f in COUPLE_FIELDS])


def _route_struct(valid_mask, grad_scale, row_loss, loss_sum, grad, correction_target=SAKI_TARGET_MODE):
    gdt = _dtype_code(grad.dtype) if grad is not None else SAKI_F32
    gstride = grad.stride(0) if grad is not None else 0
    return SakiRouteArgs(_ptr(valid_mask), float(grad_scale), gdt, _ptr(row_loss),
                         _ptr(loss_sum), _ptr(grad), gstride, int(correction_target))


def saki_couple(student, teacher, eps, seed, row_offset=0, out=None, route=None,
                workspace=None, stream=None):
    """Call saki_couple on preallocated buffers.

    out:   dict field -> tensor (missing fields are not written)
    route: None, or dict with optional keys valid_mask, grad_scale, row_loss,
           loss_sum (float64 tensor of 1), grad (2-D float32/bfloat16 tensor),
           correction_target (SAKI_TARGET_MODE or SAKI_TARGET_SAMPLE).
    """
    load()
    rows = _rows(student, teacher, row_offset)
    co = _couple_struct(out or {})
    rt = None
    if route is not None:
        rt = _route_struct(route.get("valid_mask"), route.get("grad_scale", 1.0),
                           route.get("row_loss"), route.get("loss_sum"), route.get("grad"),
                           route.get("correction_target", SAKI_TARGET_MODE))
    ws_b = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.saki_couple(ctypes.byref(rows), float(eps), int(seed) & (2**64 - 1),
                          ctypes.byref(co), ctypes.byref(rt) if rt is not None else None,
                          _ptr(workspace), ws_b, _stream(stream))
    _check(st)


def saki_couple_static(student, teacher, eps, seed, row_offset=0, out=None, route=None, stream=None):
    """Call saki_couple_static (no workspace: the library's static scratch) on
    preallocated buffers; out and route as for saki_couple."""
    load()
    rows = _rows(student, teacher, row_offset)
    co = _couple_struct(out or {})
    rt = None
    if route is not None:
        rt = _route_struct(route.get("valid_mask"), route.get("grad_scale", 1.0),
                           route.get("row_loss"), route.get("loss_sum"), route.get("grad"),
                           route.get("correction_target", SAKI_TARGET_MODE))
    st = _lib.saki_couple_static(ctypes.byref(rows), float(eps), int(seed) & (2**64 - 1),
                                 ctypes.byref(co), ctypes.byref(rt) if rt is not None else None,
                                 _stream(stream))
    _check(st)


def saki_route_loss(student, token, corrected, teacher_argmax, advantage, valid_mask=None,
                    grad_scale=1.0, row_loss=None, loss_sum=None, grad=None, workspace=None,
                    stream=None):
    load()
    rt = _route_struct(valid_mask, grad_scale, row_loss, loss_sum, grad)
    ws_b = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.saki_route_loss(_ptr(student), _dtype_code(student.dtype), student.shape[0],
                              student.shape[1], student.stride(0), _ptr(token), _ptr(corrected),
                              _ptr(teacher_argmax), _ptr(advantage), ctypes.byref(rt),
                              _ptr(workspace), ws_b, _stream(stream))
    _check(st)


def saki_spec_verify(student, teacher, k, draft, eps, seed, row_offset=0, eos_id=-1,
                     accepted_len=None, correction=None, per_pos=None, workspace=None,
                     stream=None):
    load()
    rows = _rows(student, teacher, row_offset)
    pp = _couple_struct(per_pos) if per_pos is not None else None
    ws_b = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.saki_spec_verify(ctypes.byref(rows), int(k), _ptr(draft), float(eps),
                               int(seed) & (2**64 - 1), int(eos_id), _ptr(accepted_len),
                               _ptr(correction), ctypes.byref(pp) if pp is not None else None,
                               _ptr(workspace), ws_b, _stream(stream))
    _check(st)


# ---------------------------------------------------------------------------
# Convenience wrappers that allocate their outputs (tests, examples).
# ---------------------------------------------------------------------------
def couple(student, teacher, eps, seed, row_offset=0, route=False, grad_dtype=None,
           valid_mask=None, grad_scale=1.0, correction_target=SAKI_TARGET_MODE, stream=None):
    n, V = student.shape
    dev = student.device
    out = alloc_couple_out(n, dev)
    rargs = None
    if route:
        rargs = dict(valid_mask=valid_mask, grad_scale=grad_scale,
                     row_loss=torch.empty(n, dtype=torch.float32, device=dev),
                     loss_sum=torch.empty(1, dtype=torch.float64, device=dev),
                     correction_target=correction_target)
        if grad_dtype is not None:
            rargs["grad"] = alloc_rows(n, V, grad_dtype, dev)
    ws = torch.empty(max(workspace_bytes(SAKI_OP_COUPLE, n, V), 8), dtype=torch.uint8, device=dev)
    saki_couple(student, teacher, eps, seed, row_offset, out, rargs, ws, stream)
    if rargs is not None:
        out.update({k: v for k, v in rargs.items() if k in ("row_loss", "loss_sum", "grad")})
    return out


def route_loss(student, token, corrected, teacher_argmax, advantage, valid_mask=None,
               grad_scale=1.0, grad_dtype=torch.float32, stream=None):
    n, V = student.shape
    dev = student.device
    row_loss = torch.empty(n, dtype=torch.float32, device=dev)
    loss_sum = torch.empty(1, dtype=torch.float64, device=dev)
    grad = alloc_rows(n, V, grad_dtype, dev) if grad_dtype is not None else None
    ws = torch.empty(max(workspace_bytes(SAKI_OP_ROUTE, n, V), 8), dtype=torch.uint8, device=dev)
    saki_route_loss(student, token, corrected, teacher_argmax, advantage, valid_mask, grad_scale,
                    row_loss, loss_sum, grad, ws, stream)
    return dict(row_loss=row_loss, loss_sum=loss_sum, grad=grad)


def spec_verify(student, teacher, k, draft, eps, seed, row_offset=0, eos_id=-1, per_pos=True,
                stream=None):
    n, V = student.shape
    dev = student.device
    nb = n // k
    acc = torch.empty(nb, dtype=torch.int32, device=dev)
    corr = torch.empty(nb, dtype=torch.int32, device=dev)
    pp = alloc_couple_out(n, dev) if per_pos else None
    ws = torch.empty(max(workspace_bytes(SAKI_OP_VERIFY, n, V), 8), dtype=torch.uint8, device=dev)
    saki_spec_verify(student, teacher, k, draft, eps, seed, row_offset, eos_id, acc, corr, pp,
                     ws, stream)
    out = dict(accepted_len=acc, correction=corr)
    if pp is not None:
        out["per_pos"] = pp
    return out


def saki_select_positions(mode, traj_offsets, tv, corrected, selected, seed, valid_mask=None,
                          row_offset=0, workspace=None, stream=None):
    """Call saki_select_positions on preallocated buffers (traj_offsets: int64 [n_traj + 1])."""
    load()
    n_traj = traj_offsets.numel() - 1
    n_rows = tv.numel()
    ws_b = 0 if workspace is None else workspace.numel() * workspace.element_size()
    st = _lib.saki_select_positions(int(mode), n_traj, n_rows, _ptr(traj_offsets), _ptr(tv),
                                    _ptr(corrected), _ptr(valid_mask), int(seed) & (2**64 - 1),
                                    int(row_offset), _ptr(selected), _ptr(workspace), ws_b,
                                    _stream(stream))
    _check(st)


def select_positions(mode, traj_offsets, tv, corrected, seed, valid_mask=None, row_offset=0,
                     stream=None):
    """Placement-control selection mask (uint8 [n_rows]); allocates its output and workspace."""
    n = tv.numel()
    sel = torch.empty(n, dtype=torch.uint8, device=tv.device)
    ws = torch.empty(max(workspace_bytes(SAKI_OP_SELECT, n, 0), 8), dtype=torch.uint8,
                     device=tv.device)
    saki_select_positions(mode, traj_offsets, tv, corrected, sel, seed, valid_mask, row_offset, ws,
                          stream)
    return sel


def saki_probe_metrics(student, teacher, k, c1=None, ck=None, kl_ts=None, entropy=None, topk=None,
                       row_status=None, stream=None):
    """Call saki_probe_metrics on preallocated outputs (any may be None)."""
    load()
    rows = _rows(student, teacher, 0)
    st = _lib.saki_probe_metrics(ctypes.byref(rows), int(k), _ptr(c1), _ptr(ck), _ptr(kl_ts),
                                 _ptr(entropy), _ptr(topk), _ptr(row_status), _stream(stream))
    _check(st)


def probe_metrics(student, teacher, k=16, stream=None):
    """Probe metrics per row; allocates its outputs."""
    n = student.shape[0]
    dev = student.device
    out = dict(c1=torch.empty(n, dtype=torch.float32, device=dev),
               ck=torch.empty(n, dtype=torch.float32, device=dev),
               kl_ts=torch.empty(n, dtype=torch.float32, device=dev),
               entropy=torch.empty(n, dtype=torch.float32, device=dev),
               topk=torch.empty(n, k, dtype=torch.int32, device=dev),
               row_status=torch.empty(n, dtype=torch.uint8, device=dev))
    saki_probe_metrics(student, teacher, k, stream=stream, **out)
    return out


def saki_sample(student, token, seed, row_offset=0, row_step=1, row_status=None, stream=None):
    """Call saki_sample: token[r] ~ softmax(student[r]) keyed by row_offset + r * row_step.

    student is a [n_rows, V] tensor whose rows may be strided (stride(1) == 1)."""
    load()
    assert student.dim() == 2 and student.stride(1) == 1
    _dense(token, row_status)
    rows = SakiRows(_ptr(student), None, _dtype_code(student.dtype), 0, student.shape[0],
                    student.shape[1], student.stride(0), int(row_offset))
    st = _lib.saki_sample(ctypes.byref(rows), int(row_step), int(seed) & (2**64 - 1), _ptr(token),
                          _ptr(row_status), _stream(stream))
    _check(st)


def sample(student, seed, row_offset=0, row_step=1, stream=None):
    """Draws one token per row; allocates token (int32) and row_status (uint8)."""
    n = student.shape[0]
    tok = torch.empty(n, dtype=torch.int32, device=student.device)
    status = torch.empty(n, dtype=torch.uint8, device=student.device)
    saki_sample(student, tok, seed, row_offset, row_step, status, stream)
    return tok, status


def alloc_traj(n_seq, max_len, device, fields=TRAJ_FIELDS):
    """Trajectory buffers: tokens -1, float metadata NaN, length 0, done running."""
    out = {}
    for f in fields:
        dt = TRAJ_DTYPES.get(f, torch.float32)
        shape = (n_seq,) if f in ("length", "done") else (n_seq, max_len)
        if f == "tokens" or f == "teacher_argmax":
            out[f] = torch.full(shape, -1, dtype=dt, device=device)
        elif dt == torch.float32:
            out[f] = torch.full(shape, float("nan"), dtype=dt, device=device)
        else:
            out[f] = torch.zeros(shape, dtype=dt, device=device)
    return out


def saki_commit(traj, max_len, k, eos_id, accepted_len, correction, per_pos, n_commit=None,
                stream=None):
    """Call saki_commit on trajectory buffers `traj` (dict of TRAJ_FIELDS tensors)."""
    load()
    _dense(*traj.values(), accepted_len, correction, n_commit, *per_pos.values())
    n_seq = traj["length"].numel()
    tr = SakiTraj(n_seq, int(max_len), *[_ptr(traj.get(f)) for f in TRAJ_FIELDS])
    pp = _couple_struct(per_pos)
    st = _lib.saki_commit(ctypes.byref(tr), int(k), int(eos_id), _ptr(accepted_len),
                          _ptr(correction), ctypes.byref(pp), _ptr(n_commit), _stream(stream))
    _check(st)
