"""ctypes binding of libdavet.so (the C ABI declared in include/davet.h).

Argument marshalling only: tensors are passed as device pointers, host
arrays as ctypes arrays, and every non-zero status raises DavetError with the
library's own message.  There is no fallback: if the shared library is
missing the import of this module fails.
"""

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdavet.so")

DAVET_F32 = 0
DAVET_BF16 = 1
DAVET_F16 = 2
MAX_SEQS = 64


class DavetError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("davet status %d: %s" % (status, msg))
        self.status = status


class ViewGeom(C.Structure):
    _fields_ = [("n_crops", C.c_int32), ("grid", C.c_int32), ("d", C.c_int32),
                ("K", C.c_int32), ("dtype", C.c_int32),
                ("mixed_stride", C.c_int32), ("realizer", C.c_int32)]


DAVET_REALIZER_POOL = 0
DAVET_REALIZER_PRUNE = 1
DAVET_REALIZER_MERGE = 2
MAX_REALIZER_GRID = 64


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d", C.c_int32),
                ("n_heads", C.c_int32), ("head_dim", C.c_int32),
                ("ffn", C.c_int32), ("vocab", C.c_int32),
                ("mask_id", C.c_int32), ("rms_eps", C.c_float),
                ("rope_theta", C.c_float), ("dtype", C.c_int32)]


class LayerWeights(C.Structure):
    _fields_ = [("wqkv", C.c_void_p), ("wo", C.c_void_p), ("wg", C.c_void_p),
                ("wu", C.c_void_p), ("wd", C.c_void_p),
                ("attn_norm", C.c_void_p), ("ffn_norm", C.c_void_p)]


class WeightsT(C.Structure):
    _fields_ = [("embed", C.c_void_p), ("head", C.c_void_p),
                ("final_norm", C.c_void_p),
                ("layers", C.POINTER(LayerWeights)),
                ("head_layout", C.c_int32)]


DAVET_HEAD_ROWS = 0
DAVET_HEAD_TILED = 1


class Policy(C.Structure):
    _fields_ = [("B", C.c_double), ("rho", C.c_double), ("alpha", C.c_double),
                ("demand", C.c_double), ("early", C.c_int32), ("K", C.c_int32)]


if not os.path.exists(LIB_PATH):
    raise ImportError("libdavet.so is not built (%s); run "
                      "`python paper_2608_01821_amd/build.py`" % LIB_PATH)
_L = C.CDLL(LIB_PATH)

_vp = C.c_void_p
_i32 = C.c_int32
_P_i32 = C.POINTER(C.c_int32)
_P_f64 = C.POINTER(C.c_double)
_P_i64 = C.POINTER(C.c_int64)
_P_vp = C.POINTER(C.c_void_p)

_SIGS = {
    "davet_last_error": (C.c_char_p, []),
    "davet_version": (C.c_char_p, []),
    "davet_view_sizes": (C.c_int, [C.POINTER(ViewGeom), _P_i32]),
    "davet_view_map_sizes": (C.c_int, [C.POINTER(ViewGeom), _P_i32]),
    "davet_build_views": (C.c_int, [C.POINTER(ViewGeom), _vp, _P_vp, _P_vp,
                                    _P_vp, _vp, C.c_size_t, _vp]),
    "davet_build_views_static": (C.c_int, [C.POINTER(ViewGeom), _vp, _P_vp,
                                           _P_vp, _P_vp, _vp]),
    "davet_views_scratch_bytes": (C.c_int, [C.POINTER(ViewGeom),
                                            C.POINTER(C.c_size_t)]),
    "davet_realizer_key_count": (C.c_int, [C.POINTER(ViewGeom), _P_i32]),
    "davet_realizer_keys": (C.c_int, [C.POINTER(ViewGeom), _vp, _vp, _vp]),
    "davet_realizer_maps": (C.c_int, [C.POINTER(ViewGeom), _vp, _P_vp, _P_vp,
                                      _vp]),
    "davet_convert": (C.c_int, [_vp, _i32, _vp, _i32, C.c_size_t, _vp]),
    "davet_head_tiled_elems": (C.c_size_t, [_i32, _i32]),
    "davet_pack_head": (C.c_int, [_vp, _vp, _i32, _i32, _i32, _vp]),
    "davet_workspace_bytes": (C.c_int, [C.POINTER(ModelCfg), _i32, _i32, _i32,
                                        C.POINTER(C.c_size_t)]),
    "davet_denoise_step": (C.c_int, [C.POINTER(ModelCfg), C.POINTER(WeightsT),
                                     _i32, _P_vp, _P_i32, _vp, _P_i32, _vp,
                                     _vp, _i32, _vp, _vp, _vp, _vp, C.c_size_t,
                                     _vp]),
    "davet_fp16_overflow_count": (C.c_int, [_vp, _P_i32, _vp]),
    "davet_set_attention_split": (C.c_int, [_i32]),
    "davet_unmask": (C.c_int, [_i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp,
                               _vp]),
    "davet_demand_prior": (C.c_double, [_i32]),
    "davet_parse_operation": (C.c_int, [C.c_char_p, _P_i32]),
    "davet_policy_envelope": (C.c_int, [C.POINTER(Policy), _i32, _P_f64,
                                        _P_f64]),
    "davet_policy_step": (C.c_int, [C.POINTER(Policy), _i32, _i32, _P_f64,
                                    _P_f64, C.c_double, C.c_double, _P_f64,
                                    _P_i32, _P_f64]),
    "davet_step_stats": (C.c_int, [_i32, C.POINTER(C.c_float), _P_i32, _P_i32,
                                   C.POINTER(C.c_uint8), _P_f64, _P_f64]),
    "davet_policy_step_device": (C.c_int, [_i32, _i32, _i32, _i32,
                                           C.POINTER(Policy), _P_f64, _P_f64,
                                           _vp, _vp, _vp, _vp, _vp, _vp, _vp,
                                           _vp]),
    "davet_run_schedule": (C.c_int, [C.POINTER(ModelCfg), C.POINTER(WeightsT),
                                     _i32, C.POINTER(ViewGeom), _P_vp, _P_vp,
                                     _vp, _P_i32, _i32, _i32, _i32,
                                     C.POINTER(Policy), _P_i32, _vp, _vp,
                                     _P_i32, _P_f64, _vp, _vp, _vp, _vp,
                                     C.c_size_t, _vp]),
    "davet_mailbox_create": (C.c_int, [_P_vp]),
    "davet_mailbox_destroy": (C.c_int, [_vp]),
    "davet_set_wait_limit": (C.c_int, [C.c_double]),
    "davet_prof_enable": (C.c_int, [_i32]),
    "davet_prof_reset": (C.c_int, []),
    "davet_prof_only": (C.c_int, [_i32]),
    "davet_prof_read": (C.c_int, [_i32, _P_i64, _P_f64]),
    "davet_prof_class_name": (C.c_char_p, [_i32]),
}

for _name, (_res, _args) in _SIGS.items():
    _f = getattr(_L, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_SIGS)


def raw():
    """The loaded ctypes library."""
    return _L


def _check(status):
    if status != 0:
        raise DavetError(status, _L.davet_last_error().decode())
    return status


def _ptr(t):
    """Device (or host) address of a tensor, or None.  The library reads
    every buffer as dense, so a strided view is refused."""
    if t is None:
        return None
    if not t.is_contiguous():
        raise ValueError("davet: tensor arguments must be contiguous")
    return C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, int):
        return C.c_void_p(stream)
    return C.c_void_p(stream.cuda_stream)


def _addr(t):
    """Integer address of a dense tensor, or None."""
    p = _ptr(t)
    return None if p is None else p.value


def _ptr_array(items):
    arr = (C.c_void_p * max(1, len(items)))()
    for i, t in enumerate(items):
        if t is None or isinstance(t, int):
            arr[i] = t
        else:
            if not t.is_contiguous():
                raise ValueError("davet: tensor arguments must be contiguous")
            arr[i] = t.data_ptr()
    return arr


def _i32_array(vals):
    arr = (C.c_int32 * max(1, len(vals)))()
    for i, v in enumerate(vals):
        arr[i] = int(v)
    return arr


class Weights:
    """Holds the davet_weights struct and keeps the tensors it points to
    alive.  ``layers`` is a list of dicts with tensors wqkv, wo, wg, wu, wd
    and optional attn_norm / ffn_norm (float32).  ``head`` is row-major
    [vocab, d], or the output of davet_pack_head with
    head_layout=DAVET_HEAD_TILED."""

    def __init__(self, embed, head, layers, final_norm=None,
                 head_layout=DAVET_HEAD_ROWS):
        self._keep = [embed, head, final_norm, layers]
        self._layers = (LayerWeights * max(1, len(layers)))()
        for i, lw in enumerate(layers):
            self._layers[i] = LayerWeights(
                _addr(lw["wqkv"]), _addr(lw["wo"]), _addr(lw["wg"]),
                _addr(lw["wu"]), _addr(lw["wd"]), _addr(lw.get("attn_norm")),
                _addr(lw.get("ffn_norm")))
        self.struct = WeightsT(_addr(embed), _addr(head), _addr(final_norm),
                               self._layers, int(head_layout))


def davet_version():
    return _L.davet_version().decode()


def davet_view_sizes(geom: ViewGeom):
    out = (C.c_int32 * geom.K)()
    _check(_L.davet_view_sizes(C.byref(geom), out))
    return list(out)


def davet_view_map_sizes(geom: ViewGeom):
    out = (C.c_int32 * geom.K)()
    _check(_L.davet_view_map_sizes(C.byref(geom), out))
    return list(out)


def davet_views_scratch_bytes(geom):
    out = C.c_size_t(0)
    _check(_L.davet_views_scratch_bytes(C.byref(geom), C.byref(out)))
    return int(out.value)


def davet_build_views(geom, v, levels, offsets=None, members=None,
                      scratch=None, stream=None):
    """``scratch``: a device tensor of davet_views_scratch_bytes bytes; when
    None and the realizer needs one, a torch buffer on v's device."""
    K = geom.K
    lv = _ptr_array(list(levels) + [None] * (K - len(levels)))
    off = _ptr_array(offsets) if offsets is not None else None
    mem = _ptr_array(members) if members is not None else None
    if scratch is None:
        nb = davet_views_scratch_bytes(geom)
        if nb:
            import torch
            scratch = torch.empty(nb, dtype=torch.uint8, device=v.device)
    nbytes = 0 if scratch is None else scratch.numel() * scratch.element_size()
    _check(_L.davet_build_views(C.byref(geom), _ptr(v), lv, off, mem,
                                _ptr(scratch), nbytes, _stream(stream)))


STATIC_SCRATCH_BYTES = 4 << 20


def davet_build_views_static(geom, v, levels, offsets=None, members=None,
                             stream=None):
    """davet_build_views with the library's own device scratch (no
    allocation by the library or by this binding)."""
    K = geom.K
    lv = _ptr_array(list(levels) + [None] * (K - len(levels)))
    off = _ptr_array(offsets) if offsets is not None else None
    mem = _ptr_array(members) if members is not None else None
    _check(_L.davet_build_views_static(C.byref(geom), _ptr(v), lv, off, mem,
                                       _stream(stream)))


def davet_realizer_key_count(geom):
    out = C.c_int32(0)
    _check(_L.davet_realizer_key_count(C.byref(geom), C.byref(out)))
    return int(out.value)


def davet_realizer_keys(geom, v, keys, stream=None):
    _check(_L.davet_realizer_keys(C.byref(geom), _ptr(v), _ptr(keys),
                                  _stream(stream)))


def davet_realizer_maps(geom, keys, offsets=None, members=None, stream=None):
    K = geom.K
    off = _ptr_array(list(offsets) + [None] * (K - len(offsets))) \
        if offsets is not None else None
    mem = _ptr_array(list(members) + [None] * (K - len(members))) \
        if members is not None else None
    _check(_L.davet_realizer_maps(C.byref(geom), _ptr(keys), off, mem,
                                  _stream(stream)))


def davet_convert(src, src_dtype, dst, dst_dtype, n=None, stream=None):
    n = src.numel() if n is None else n
    _check(_L.davet_convert(_ptr(src), int(src_dtype), _ptr(dst),
                            int(dst_dtype), int(n), _stream(stream)))


def davet_head_tiled_elems(vocab, d):
    return int(_L.davet_head_tiled_elems(int(vocab), int(d)))


def davet_pack_head(src, dst, vocab, d, dtype, stream=None):
    _check(_L.davet_pack_head(_ptr(src), _ptr(dst), int(vocab), int(d),
                              int(dtype), _stream(stream)))


def davet_workspace_bytes(cfg, max_tokens, max_seqs, L):
    out = C.c_size_t(0)
    _check(_L.davet_workspace_bytes(C.byref(cfg), int(max_tokens),
                                    int(max_seqs), int(L), C.byref(out)))
    return out.value


def davet_denoise_step(cfg, weights: Weights, views, n_view, prompt_ids,
                       cu_prompt, resp_ids, resp_masked, L, conf_out,
                       argmax_out, logits_out, workspace, stream=None):
    n = len(views)
    _check(_L.davet_denoise_step(
        C.byref(cfg), C.byref(weights.struct), n, _ptr_array(views),
        _i32_array(n_view), _ptr(prompt_ids), _i32_array(cu_prompt),
        _ptr(resp_ids), _ptr(resp_masked), int(L), _ptr(conf_out),
        _ptr(argmax_out), _ptr(logits_out), _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))


def davet_fp16_overflow_count(workspace, stream=None) -> int:
    """Non-finite 16-bit projection outputs stored by the last step (or
    schedule) that ran on `workspace`; waits for `stream`."""
    out = C.c_int32(0)
    _check(_L.davet_fp16_overflow_count(_ptr(workspace), C.byref(out),
                                        _stream(stream)))
    return out.value


def davet_set_attention_split(mode):
    """Attention key-range split: 0 automatic, 1 off, 2..8 forced."""
    _check(_L.davet_set_attention_split(int(mode)))


def davet_unmask(n_seqs, L, k, conf, argmax, resp_ids, resp_masked,
                 selected=None, stream=None):
    _check(_L.davet_unmask(int(n_seqs), int(L), int(k), _ptr(conf),
                           _ptr(argmax), _ptr(resp_ids), _ptr(resp_masked),
                           _ptr(selected), _stream(stream)))


def davet_demand_prior(category):
    return _L.davet_demand_prior(int(category))


def davet_parse_operation(query: str) -> int:
    out = C.c_int32(-1)
    _check(_L.davet_parse_operation(query.encode("utf-8"), C.byref(out)))
    return out.value


def davet_policy_envelope(pol: Policy, T):
    lo = (C.c_double * T)()
    up = (C.c_double * T)()
    _check(_L.davet_policy_envelope(C.byref(pol), int(T), lo, up))
    return list(lo), list(up)


def davet_policy_step(pol: Policy, t, T, lower, upper, cbar_prev, churn_prev):
    lo = (C.c_double * T)(*lower)
    up = (C.c_double * T)(*upper)
    b = C.c_double(0)
    lv = C.c_int32(0)
    r = C.c_double(0)
    _check(_L.davet_policy_step(C.byref(pol), int(t), int(T), lo, up,
                                float(cbar_prev), float(churn_prev),
                                C.byref(b), C.byref(lv), C.byref(r)))
    return b.value, lv.value, r.value


def davet_step_stats(conf, argmax, argmax_prev, masked_after):
    conf = np.ascontiguousarray(conf, dtype=np.float32)
    am = np.ascontiguousarray(argmax, dtype=np.int32)
    m = np.ascontiguousarray(masked_after, dtype=np.uint8)
    prev = None if argmax_prev is None else \
        np.ascontiguousarray(argmax_prev, dtype=np.int32)
    cb = C.c_double(0)
    ch = C.c_double(0)
    _check(_L.davet_step_stats(
        len(conf), conf.ctypes.data_as(C.POINTER(C.c_float)),
        am.ctypes.data_as(_P_i32),
        None if prev is None else prev.ctypes.data_as(_P_i32),
        m.ctypes.data_as(C.POINTER(C.c_uint8)), C.byref(cb), C.byref(ch)))
    return cb.value, ch.value


def davet_policy_step_device(pols, t, T, lower, upper, conf, argmax,
                             argmax_prev, masked_after, level_out, budget_out,
                             r_out=None, stream=None):
    """lower/upper: host float64 [n_seqs * T]; the other arrays are device
    tensors ([n_seqs * L] inputs, [n_seqs] outputs)."""
    n = len(pols)
    L = conf.numel() // n
    p = (Policy * n)(*pols)
    lo = np.ascontiguousarray(lower, dtype=np.float64)
    up = np.ascontiguousarray(upper, dtype=np.float64)
    _check(_L.davet_policy_step_device(
        n, L, int(t), int(T), p, lo.ctypes.data_as(_P_f64),
        up.ctypes.data_as(_P_f64), _ptr(conf), _ptr(argmax), _ptr(argmax_prev),
        _ptr(masked_after), _ptr(level_out), _ptr(budget_out), _ptr(r_out),
        _stream(stream)))


class Mailbox:
    """A davet_mailbox (pinned host memory the policy-mode loop writes the
    next levels into), made once and freed by close() or at exit."""

    def __init__(self):
        h = C.c_void_p()
        _check(_L.davet_mailbox_create(C.byref(h)))
        self.handle = h

    def close(self):
        if self.handle is not None and self.handle.value:
            h, self.handle = self.handle, None
            _check(_L.davet_mailbox_destroy(h))

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


_MAILBOX = None


def default_mailbox():
    """The process's mailbox, made on first use (a set-up step, not part of
    a loop's steady state)."""
    global _MAILBOX
    if _MAILBOX is None:
        _MAILBOX = Mailbox()
    return _MAILBOX


def davet_set_wait_limit(seconds):
    _check(_L.davet_set_wait_limit(float(seconds)))


def davet_run_schedule(cfg, weights: Weights, geoms, visual, view_bufs,
                       prompt_ids, cu_prompt, L, T, k, pols, fixed_levels,
                       resp_ids, resp_masked, workspace, conf_trace=None,
                       argmax_trace=None, stream=None, mailbox=None):
    """Returns (levels [n_seqs*T], budgets [n_seqs*T]) as host lists.
    ``mailbox``: a Mailbox; in policy mode the process's default one when
    None."""
    n = len(visual)
    g = (ViewGeom * n)(*geoms)
    p = (Policy * n)(*pols) if pols is not None else None
    fl = _i32_array(np.asarray(fixed_levels).reshape(-1)) \
        if fixed_levels is not None else None
    lv = (C.c_int32 * (n * T))()
    bu = (C.c_double * (n * T))()
    if mailbox is None and pols is not None:
        mailbox = default_mailbox()
    mb = None if mailbox is None else mailbox.handle
    _check(_L.davet_run_schedule(
        C.byref(cfg), C.byref(weights.struct), n, g, _ptr_array(visual),
        _ptr_array(view_bufs), _ptr(prompt_ids), _i32_array(cu_prompt),
        int(L), int(T), int(k), p, fl, _ptr(resp_ids), _ptr(resp_masked),
        lv, bu, _ptr(conf_trace), _ptr(argmax_trace), mb, _ptr(workspace),
        workspace.numel() * workspace.element_size(), _stream(stream)))
    return list(lv), list(bu)


def prof_enable(max_launches):
    _check(_L.davet_prof_enable(int(max_launches)))


def prof_reset():
    _check(_L.davet_prof_reset())


def prof_only(cls_name=None):
    """Record only launches of the named kernel class (None: every class)."""
    idx = -1
    if cls_name is not None:
        i = 0
        while True:
            n = _L.davet_prof_class_name(i)
            if not n:
                raise DavetError(-1, "unknown kernel class %r" % cls_name)
            if n.decode() == cls_name:
                idx = i
                break
            i += 1
    _check(_L.davet_prof_only(idx))


def prof_read():
    """{kernel class name: (launches, total ms)}"""
    n = 32
    cnt = (C.c_int64 * n)()
    ms = (C.c_double * n)()
    k = _L.davet_prof_read(n, cnt, ms)
    if k < 0:
        _check(k)
    return {_L.davet_prof_class_name(i).decode(): (cnt[i], ms[i])
            for i in range(k)}
