"""ctypes binding of libolive_score.so (the C ABI of include/olive_score.h).

Argument marshalling only: every function has the C name and forwards plain
pointers, sizes and the HIP stream. Torch tensors are accepted wherever the C
function takes a device pointer (their data_ptr() is passed); None maps to NULL.
The library must have been built (python -m paper_2609_36246_amd.build); loading
fails loudly otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libolive_score.so")

OLIVE_OK = 0
OLIVE_E_NULL = 1
OLIVE_E_SHAPE = 2
OLIVE_E_DTYPE = 3
OLIVE_E_RANGE = 4
OLIVE_E_HIP = 5
OLIVE_E_NOMEM = 6
OLIVE_E_UNSUPPORTED = 7
OLIVE_E_LIMIT = 8
STATUS_CODES = list(range(9))

OLIVE_F32 = 0
OLIVE_BF16 = 1
OLIVE_W_DV = 0
OLIVE_W_VD = 1
OLIVE_REGION_TEACHER = 0
OLIVE_REGION_STUDENT = 1
OLIVE_REGION_ALL = 2
OLIVE_REGION_SPANS = 3
OLIVE_FLAG_SIMPLE_KERNEL = 1
OLIVE_FLAG_KERNEL_TIMING = 2
OLIVE_FLAG_TOPK = 4
OLIVE_FLAG_BACKWARD = 8
OLIVE_FLAG_NARROW_TILE = 16
OLIVE_GRAD_REUSE_FORWARD = 1
OLIVE_TOPK = 16
OLIVE_OUT_REGION_ONLY = 1


class olive_score_desc(ctypes.Structure):
    _fields_ = [("vocab", ctypes.c_int64), ("d_student", ctypes.c_int32),
                ("d_teacher", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("w_layout", ctypes.c_int32), ("logit_scale_student", ctypes.c_float),
                ("logit_scale_teacher", ctypes.c_float), ("max_positions", ctypes.c_int64),
                ("max_seqs", ctypes.c_int32), ("flags", ctypes.c_int32)]


class olive_batch(ctypes.Structure):
    _fields_ = [("num_seqs", ctypes.c_int32), ("region", ctypes.c_int32),
                ("total_positions", ctypes.c_int64), ("cu_seqlens", ctypes.c_void_p),
                ("cut", ctypes.c_void_p), ("valid_len", ctypes.c_void_p),
                ("targets", ctypes.c_void_p), ("h_student", ctypes.c_void_p),
                ("h_teacher", ctypes.c_void_p)]


class olive_score_outputs(ctypes.Structure):
    _fields_ = [("size", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("kl", ctypes.c_void_p), ("kl_reverse", ctypes.c_void_p),
                ("counts", ctypes.c_void_p), ("logp_student", ctypes.c_void_p),
                ("logp_teacher", ctypes.c_void_p), ("argmax_student", ctypes.c_void_p),
                ("argmax_teacher", ctypes.c_void_p), ("ce_per_seq", ctypes.c_void_p),
                ("topk_overlap", ctypes.c_void_p), ("kl_topk", ctypes.c_void_p),
                ("topk_student", ctypes.c_void_p), ("topk_teacher", ctypes.c_void_p),
                ("jsd", ctypes.c_void_p)]


class olive_grad_outputs(ctypes.Structure):
    _fields_ = [("size", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("w_ce", ctypes.c_float), ("w_kl", ctypes.c_float),
                ("grad_h_student", ctypes.c_void_p), ("grad_w_student", ctypes.c_void_p),
                ("counts", ctypes.c_void_p)]


class olive_spans(ctypes.Structure):
    _fields_ = [("size", ctypes.c_int32), ("num_spans", ctypes.c_int32),
                ("span_offsets", ctypes.c_void_p), ("spans", ctypes.c_void_p)]


class OliveError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s" % (what, olive_status_string(status)))


_lib: Optional[ctypes.CDLL] = None


def load() -> ctypes.CDLL:
    """Load the built library (once) and declare its signatures."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError("libolive_score.so is not built (run: python -m "
                          "paper_2609_36246_amd.build); there is no fallback")
    # torch's HIP runtime must be resident first: the library's libamdhip64.so.7 then
    # resolves to it by soname.  Loaded the other way round, torch (which asks for the
    # file libamdhip64.so) brings a second runtime into the process and the library's
    # calls see no device and cannot use torch's streams or allocations.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    vp, i32p, i64p, f32p = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
    st = ctypes.c_int
    lib.olive_score_init.argtypes = [ctypes.POINTER(ctypes.c_void_p),
                                     ctypes.POINTER(olive_score_desc), vp, vp, vp]
    lib.olive_score_init.restype = st
    lib.olive_token_logprobs.argtypes = [vp, ctypes.POINTER(olive_batch), f32p, f32p, i32p, i32p,
                                         vp]
    lib.olive_token_logprobs.restype = st
    lib.olive_kl_masked.argtypes = [vp, ctypes.POINTER(olive_batch), f32p, i64p, f32p, f32p,
                                    i32p, i32p, f32p, vp]
    lib.olive_kl_masked.restype = st
    lib.olive_kl_masked_static.argtypes = [ctypes.POINTER(olive_score_desc), vp, vp,
                                           ctypes.POINTER(olive_batch), f32p, i64p, f32p, f32p,
                                           i32p, i32p, f32p, vp]
    lib.olive_kl_masked_static.restype = st
    lib.olive_score_batch.argtypes = [vp, ctypes.POINTER(olive_batch),
                                      ctypes.POINTER(olive_score_outputs), vp]
    lib.olive_score_batch.restype = st
    lib.olive_score_batch_spans.argtypes = [vp, ctypes.POINTER(olive_batch),
                                            ctypes.POINTER(olive_spans),
                                            ctypes.POINTER(olive_score_outputs), vp]
    lib.olive_score_batch_spans.restype = st
    lib.olive_score_backward.argtypes = [vp, ctypes.POINTER(olive_batch),
                                         ctypes.POINTER(olive_spans),
                                         ctypes.POINTER(olive_grad_outputs), vp]
    lib.olive_score_backward.restype = st
    lib.olive_score_free.argtypes = [vp]
    lib.olive_score_free.restype = st
    lib.olive_status_string.argtypes = [st]
    lib.olive_status_string.restype = ctypes.c_char_p
    lib.olive_score_last_error.argtypes = [vp, ctypes.POINTER(ctypes.c_int32)]
    lib.olive_score_last_error.restype = st
    lib.olive_score_last_stats.argtypes = [vp, ctypes.POINTER(ctypes.c_int64)]
    lib.olive_score_last_stats.restype = st
    lib.olive_score_kernel_times.argtypes = [vp, ctypes.POINTER(ctypes.c_float), ctypes.c_int]
    lib.olive_score_kernel_times.restype = st
    _lib = lib
    return lib


def _ptr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(status: int, what: str):
    if status != OLIVE_OK:
        raise OliveError(status, what)


def olive_status_string(status: int) -> str:
    return load().olive_status_string(status).decode()


def olive_score_init(desc: olive_score_desc, w_student, w_teacher=None, stream=None,
                     check: bool = True):
    """Returns an opaque context handle (int). Raises OliveError unless check=False,
    in which case (status, handle) is returned."""
    h = ctypes.c_void_p()
    s = load().olive_score_init(ctypes.byref(h), ctypes.byref(desc), _ptr(w_student),
                                _ptr(w_teacher), _stream(stream) if check else stream)
    if not check:
        return s, h.value
    _check(s, "olive_score_init")
    return h.value


def make_batch(cu_seqlens, cut, targets, h_student, h_teacher=None, valid_len=None,
               region: int = OLIVE_REGION_TEACHER, total_positions: Optional[int] = None,
               num_seqs: Optional[int] = None) -> olive_batch:
    """An olive_batch over device tensors (the caller keeps them alive)."""
    b = olive_batch()
    b.num_seqs = int(num_seqs if num_seqs is not None else cu_seqlens.shape[0] - 1)
    b.region = int(region)
    b.total_positions = int(total_positions if total_positions is not None
                            else targets.shape[0])
    b.cu_seqlens = _ptr(cu_seqlens)
    b.cut = _ptr(cut)
    b.valid_len = _ptr(valid_len)
    b.targets = _ptr(targets)
    b.h_student = _ptr(h_student)
    b.h_teacher = _ptr(h_teacher)
    return b


def olive_token_logprobs(ctx, batch: olive_batch, logp_student, logp_teacher=None,
                         argmax_student=None, argmax_teacher=None, stream=None,
                         check: bool = True) -> int:
    s = load().olive_token_logprobs(ctx, ctypes.byref(batch), _ptr(logp_student),
                                    _ptr(logp_teacher), _ptr(argmax_student),
                                    _ptr(argmax_teacher), _stream(stream))
    if check:
        _check(s, "olive_token_logprobs")
    return s


def olive_kl_masked(ctx, batch: olive_batch, kl, counts=None, logp_student=None,
                    logp_teacher=None, argmax_student=None, argmax_teacher=None,
                    ce_per_seq=None, stream=None, check: bool = True) -> int:
    s = load().olive_kl_masked(ctx, ctypes.byref(batch), _ptr(kl), _ptr(counts),
                               _ptr(logp_student), _ptr(logp_teacher), _ptr(argmax_student),
                               _ptr(argmax_teacher), _ptr(ce_per_seq), _stream(stream))
    if check:
        _check(s, "olive_kl_masked")
    return s


def olive_kl_masked_static(desc: olive_score_desc, w_student, w_teacher, batch: olive_batch,
                           kl, counts=None, logp_student=None, logp_teacher=None,
                           argmax_student=None, argmax_teacher=None, ce_per_seq=None,
                           stream=None, check: bool = True) -> int:
    """olive_kl_masked without a context ([V][d] weights read in place; nothing is
    allocated: the library's fixed per-GPU scratch array holds the workspace)."""
    s = load().olive_kl_masked_static(ctypes.byref(desc), _ptr(w_student), _ptr(w_teacher),
                                      ctypes.byref(batch), _ptr(kl), _ptr(counts),
                                      _ptr(logp_student), _ptr(logp_teacher),
                                      _ptr(argmax_student), _ptr(argmax_teacher),
                                      _ptr(ce_per_seq), _stream(stream))
    if check:
        _check(s, "olive_kl_masked_static")
    return s


def make_outputs(kl=None, kl_reverse=None, counts=None, logp_student=None, logp_teacher=None,
                 argmax_student=None, argmax_teacher=None, ce_per_seq=None,
                 topk_overlap=None, kl_topk=None, topk_student=None, topk_teacher=None,
                 jsd=None, flags: int = 0) -> olive_score_outputs:
    o = olive_score_outputs()
    o.size = ctypes.sizeof(olive_score_outputs)
    o.flags = int(flags)
    o.kl, o.kl_reverse, o.counts = _ptr(kl), _ptr(kl_reverse), _ptr(counts)
    o.logp_student, o.logp_teacher = _ptr(logp_student), _ptr(logp_teacher)
    o.argmax_student, o.argmax_teacher = _ptr(argmax_student), _ptr(argmax_teacher)
    o.ce_per_seq = _ptr(ce_per_seq)
    o.topk_overlap, o.kl_topk = _ptr(topk_overlap), _ptr(kl_topk)
    o.topk_student, o.topk_teacher = _ptr(topk_student), _ptr(topk_teacher)
    o.jsd = _ptr(jsd)
    return o


def olive_score_batch(ctx, batch: olive_batch, outputs: olive_score_outputs, stream=None,
                      check: bool = True) -> int:
    s = load().olive_score_batch(ctx, ctypes.byref(batch), ctypes.byref(outputs),
                                 _stream(stream))
    if check:
        _check(s, "olive_score_batch")
    return s


def make_spans(span_offsets, span_pairs, num_spans: Optional[int] = None) -> olive_spans:
    """An olive_spans over device tensors: offsets [B+1] int32, pairs [S, 2] int32."""
    sp = olive_spans()
    sp.size = ctypes.sizeof(olive_spans)
    sp.num_spans = int(num_spans if num_spans is not None else span_pairs.shape[0])
    sp.span_offsets = _ptr(span_offsets)
    sp.spans = _ptr(span_pairs) if sp.num_spans > 0 else None
    return sp


def make_grad_outputs(w_ce=1.0, w_kl=0.0, grad_h=None, grad_w=None,
                      counts=None, reuse_forward=False) -> olive_grad_outputs:
    o = olive_grad_outputs()
    o.size = ctypes.sizeof(olive_grad_outputs)
    o.flags = OLIVE_GRAD_REUSE_FORWARD if reuse_forward else 0
    o.w_ce, o.w_kl = float(w_ce), float(w_kl)
    o.grad_h_student, o.grad_w_student = _ptr(grad_h), _ptr(grad_w)
    o.counts = _ptr(counts)
    return o


def olive_score_backward(ctx, batch: olive_batch, grads: olive_grad_outputs, spans=None,
                         stream=None, check: bool = True) -> int:
    s = load().olive_score_backward(ctx, ctypes.byref(batch),
                                    ctypes.byref(spans) if spans is not None else None,
                                    ctypes.byref(grads), _stream(stream))
    if check:
        _check(s, "olive_score_backward")
    return s


def olive_score_batch_spans(ctx, batch: olive_batch, spans: olive_spans,
                            outputs: olive_score_outputs, stream=None, check: bool = True) -> int:
    s = load().olive_score_batch_spans(ctx, ctypes.byref(batch), ctypes.byref(spans),
                                       ctypes.byref(outputs), _stream(stream))
    if check:
        _check(s, "olive_score_batch_spans")
    return s


def olive_score_free(ctx) -> int:
    return load().olive_score_free(ctx)


def olive_score_last_error(ctx) -> int:
    v = ctypes.c_int32(0)
    _check(load().olive_score_last_error(ctx, ctypes.byref(v)), "olive_score_last_error")
    return v.value


def olive_score_last_stats(ctx) -> dict:
    out = (ctypes.c_int64 * 6)()
    _check(load().olive_score_last_stats(ctx, out), "olive_score_last_stats")
    kid = out[2]
    return dict(splits=out[0], flagged=out[1],
                kernel={0: "mfma", 1: "generic", 2: "mfma"}.get(kid),
                tile={0: "256x128", 2: "256x256"}.get(kid), grid=out[3],
                topk_filtered=out[4], topk_scanned=out[5])


def olive_score_kernel_times(ctx, n: int) -> list:
    """Durations (ms) of the scoring kernel in the last n calls (needs the timing flag)."""
    buf = (ctypes.c_float * n)()
    _check(load().olive_score_kernel_times(ctx, buf, n), "olive_score_kernel_times")
    return list(buf)


def make_desc(vocab, d_student, d_teacher, dtype=OLIVE_BF16, w_layout=OLIVE_W_DV,
              scale_student=1.0, scale_teacher=1.0, max_positions=1, max_seqs=1,
              flags=0) -> olive_score_desc:
    d = olive_score_desc()
    d.vocab = int(vocab)
    d.d_student = int(d_student)
    d.d_teacher = int(d_teacher)
    d.dtype = int(dtype)
    d.w_layout = int(w_layout)
    d.logit_scale_student = float(scale_student)
    d.logit_scale_teacher = float(scale_teacher)
    d.max_positions = int(max_positions)
    d.max_seqs = int(max_seqs)
    d.flags = int(flags)
    return d
