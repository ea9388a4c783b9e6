"""ctypes binding of the LayerCheck HIP library (argument marshalling only).

Functions carry the C names of ``include/layercheck.h``; every step of the
decision path runs in the library's kernels.  Pointers are plain integers
(device addresses, e.g. ``tensor.data_ptr()``); the stream is a raw
``hipStream_t`` value (e.g. ``torch.cuda.current_stream().cuda_stream``).
The library is loaded on first use and a missing build raises immediately:
there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np

LIB_PATH = os.environ.get("LAYERCHECK_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                              "liblayercheck.so")

LC_OK, LC_ERR_INVALID_ARG, LC_ERR_BAD_STATE, LC_ERR_CAPACITY, LC_ERR_NO_VERSION, LC_ERR_HIP, LC_ERR_OOM, \
    LC_ERR_IO = range(8)
LC_DT_BF16, LC_DT_F32 = 1, 2
LC_MODE_ACCUM, LC_MODE_SNAPSHOT = 0, 1

EXPORTED = ("lc_query_build", "lc_query_layout", "lc_init_layout", "lc_score_layers", "lc_select", "lc_pack_selected",
            "lc_restore_composite", "lc_rebase", "lc_adamw_step_score", "lc_sgd_step_score", "lc_store_open",
            "lc_store_append", "lc_store_append_async", "lc_store_sync", "lc_store_count", "lc_store_entry",
            "lc_store_plan", "lc_store_restore", "lc_store_compact", "lc_store_discard_after", "lc_store_close",
            "lc_read_state", "lc_record_bytes", "lc_destroy", "lc_last_error", "lc_score_layers_static")


class lc_segment(C.Structure):
    _fields_ = [("layer", C.c_uint32), ("reserved", C.c_uint32), ("numel", C.c_uint64),
                ("weight", C.c_void_p), ("shadow", C.c_void_p), ("master", C.c_void_p),
                ("exp_avg", C.c_void_p), ("exp_avg_sq", C.c_void_p)]


class lc_build_info(C.Structure):
    _fields_ = [("chunk_bytes", C.c_uint32), ("piece_bytes", C.c_uint32), ("record_align", C.c_uint32),
                ("reserved", C.c_uint32)]


class lc_layout_desc(C.Structure):
    _fields_ = [("n_layers", C.c_uint32), ("n_segments", C.c_uint32),
                ("segments", C.POINTER(lc_segment)), ("weight_dtype", C.c_int32),
                ("has_master", C.c_int32), ("mode", C.c_int32), ("reserved", C.c_int32),
                ("k0", C.POINTER(C.c_double)), ("s_max", C.c_int64), ("eps_w", C.c_double),
                ("t_base", C.c_int64), ("stream", C.c_void_p)]


class lc_select_stats(C.Structure):
    _fields_ = [("n_selected", C.c_uint32), ("n_forced", C.c_uint32), ("payload_bytes", C.c_uint64),
                ("max_age", C.c_int64), ("weighted_age", C.c_double)]


class lc_pack_result(C.Structure):
    _fields_ = [("bytes_written", C.c_uint64), ("n_packed", C.c_uint32), ("next_rank", C.c_uint32),
                ("done", C.c_int32), ("reserved", C.c_int32)]


class lc_version(C.Structure):
    _fields_ = [("step", C.c_int64), ("mask", C.POINTER(C.c_uint8)), ("payload", C.c_void_p),
                ("payload_bytes", C.c_uint64)]


class lc_adamw_params(C.Structure):
    _fields_ = [("lr", C.c_double), ("beta1", C.c_double), ("beta2", C.c_double), ("eps", C.c_double),
                ("weight_decay", C.c_double), ("adam_step", C.c_int64)]


class lc_sgd_params(C.Structure):
    _fields_ = [("lr", C.c_double), ("weight_decay", C.c_double)]


class LCError(RuntimeError):
    def __init__(self, code: int, func: str, msg: str):
        super().__init__(f"{func} failed with status {code}: {msg}")
        self.code = code


_LIB = None


def load_library(path: str = LIB_PATH):
    global _LIB
    if _LIB is None:
        if not os.path.exists(path):
            raise RuntimeError(f"LayerCheck HIP library not built: {path} is missing "
                               "(run `python -m paper_2609_27193_amd.build_lib`)")
        lib = C.CDLL(path)
        P = C.POINTER
        sig = {
            "lc_query_build": (C.c_int, [P(lc_build_info)]),
            "lc_query_layout": (C.c_int, [P(lc_layout_desc), P(C.c_uint64), P(C.c_uint64)]),
            "lc_init_layout": (C.c_int, [P(lc_layout_desc), P(C.c_void_p)]),
            "lc_score_layers": (C.c_int, [C.c_void_p, C.c_int64]),
            "lc_score_layers_static": (C.c_int, [P(lc_segment), C.c_uint32, C.c_uint32, C.c_int32, C.c_double,
                                                 C.c_void_p, C.c_void_p]),
            "lc_select": (C.c_int, [C.c_void_p, C.c_int64, C.c_double, P(C.c_uint8), P(lc_select_stats)]),
            "lc_pack_selected": (C.c_int, [C.c_void_p, C.c_void_p, C.c_uint64, C.c_uint32, P(lc_pack_result)]),
            "lc_restore_composite": (C.c_int, [C.c_void_p, P(lc_version), C.c_uint32, C.c_int64, P(C.c_int64)]),
            "lc_rebase": (C.c_int, [C.c_void_p, C.c_int64]),
            "lc_adamw_step_score": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_void_p), C.c_int32, P(C.c_uint8),
                                              P(lc_adamw_params)]),
            "lc_sgd_step_score": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_void_p), C.c_int32, P(C.c_uint8),
                                            P(lc_sgd_params)]),
            "lc_store_open": (C.c_int, [C.c_char_p, C.c_uint32, P(C.c_uint64), C.c_uint64, P(C.c_void_p)]),
            "lc_store_append": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_uint8), C.c_void_p, C.c_uint64,
                                          C.c_void_p]),
            "lc_store_append_async": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_uint8), C.c_void_p, C.c_uint64,
                                                C.c_void_p, C.c_void_p]),
            "lc_store_sync": (C.c_int, [C.c_void_p]),
            "lc_store_count": (C.c_int, [C.c_void_p, P(C.c_uint32)]),
            "lc_store_entry": (C.c_int, [C.c_void_p, C.c_uint32, P(C.c_int64), P(C.c_uint8), P(C.c_uint64)]),
            "lc_store_plan": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_int64)]),
            "lc_store_restore": (C.c_int, [C.c_void_p, C.c_void_p, C.c_int64, P(C.c_int64)]),
            "lc_store_compact": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_uint32)]),
            "lc_store_discard_after": (C.c_int, [C.c_void_p, C.c_int64, P(C.c_uint32)]),
            "lc_store_close": (C.c_int, [C.c_void_p]),
            "lc_read_state": (C.c_int, [C.c_void_p, P(C.c_double), P(C.c_double), P(C.c_int64)]),
            "lc_record_bytes": (C.c_uint64, [C.c_void_p, C.c_uint32]),
            "lc_destroy": (C.c_int, [C.c_void_p]),
            "lc_last_error": (C.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(lib, name)
            f.restype = res
            f.argtypes = args
        _LIB = lib
    return _LIB


def _check(code: int, func: str):
    if code != LC_OK:
        raise LCError(code, func, load_library().lc_last_error().decode(errors="replace"))


@dataclass
class Segment:
    """One contiguous piece of one layer's tensor: device addresses as ints."""
    layer: int
    numel: int
    weight: int
    shadow: Optional[int]
    master: Optional[int]
    exp_avg: Optional[int]
    exp_avg_sq: Optional[int]


class LayoutDesc:
    """Owns the ctypes arrays behind an ``lc_layout_desc``."""

    def __init__(self, segments: Sequence[Segment], n_layers: int, weight_dtype: int, has_master: bool,
                 mode: int, k0: Sequence[float], s_max: int, eps_w: float = 1e-8, t_base: int = 0,
                 stream: int = 0):
        self._segs = (lc_segment * len(segments))()
        for i, s in enumerate(segments):
            self._segs[i] = lc_segment(s.layer, 0, s.numel, s.weight, s.shadow or None, s.master or None,
                                       s.exp_avg or None, s.exp_avg_sq or None)
        if len(k0) != n_layers:
            raise ValueError(f"k0 has {len(k0)} entries for {n_layers} layers")
        self._k0 = (C.c_double * n_layers)(*[float(x) for x in k0])
        self.n_layers = n_layers
        self.desc = lc_layout_desc(n_layers, len(segments), self._segs, weight_dtype, int(has_master),
                                   mode, 0, self._k0, s_max, eps_w, t_base, stream or None)


def lc_query_build() -> dict:
    info = lc_build_info()
    _check(load_library().lc_query_build(C.byref(info)), "lc_query_build")
    return {"chunk_bytes": info.chunk_bytes, "piece_bytes": info.piece_bytes, "record_align": info.record_align}


def lc_query_layout(layout: LayoutDesc):
    n = layout.n_layers
    numel = (C.c_uint64 * n)()
    rec = (C.c_uint64 * n)()
    _check(load_library().lc_query_layout(C.byref(layout.desc), numel, rec), "lc_query_layout")
    return list(numel), list(rec)


def lc_init_layout(layout: LayoutDesc) -> C.c_void_p:
    ctx = C.c_void_p()
    _check(load_library().lc_init_layout(C.byref(layout.desc), C.byref(ctx)), "lc_init_layout")
    return ctx


def lc_score_layers(ctx, step: int) -> None:
    _check(load_library().lc_score_layers(ctx, step), "lc_score_layers")


def lc_score_layers_static(segments: Sequence["Segment"], n_layers: int, weight_dtype: int, eps_w: float,
                           u_out: int, stream: int = 0) -> None:
    """u_out: device address of n_layers doubles."""
    arr = (lc_segment * len(segments))()
    for i, s in enumerate(segments):
        arr[i] = lc_segment(s.layer, 0, s.numel, s.weight, s.shadow or None, s.master or None,
                            s.exp_avg or None, s.exp_avg_sq or None)
    _check(load_library().lc_score_layers_static(arr, len(segments), n_layers, weight_dtype, eps_w,
                                                 u_out or None, stream or None), "lc_score_layers_static")


def lc_select(ctx, step: int, lr_scale: float, n_layers: Optional[int] = None):
    """With ``n_layers`` given, returns (mask uint8[N], stats dict) and
    synchronises; without it, the call is asynchronous and returns None."""
    if n_layers is None:
        _check(load_library().lc_select(ctx, step, lr_scale, None, None), "lc_select")
        return None
    mask = np.zeros(n_layers, dtype=np.uint8)
    st = lc_select_stats()
    _check(load_library().lc_select(ctx, step, lr_scale, mask.ctypes.data_as(C.POINTER(C.c_uint8)),
                                    C.byref(st)), "lc_select")
    return mask, {"n_selected": st.n_selected, "n_forced": st.n_forced, "payload_bytes": st.payload_bytes,
                  "max_age": st.max_age, "weighted_age": st.weighted_age}


def lc_pack_selected(ctx, staging: int, capacity: int, first_rank: int = 0) -> dict:
    r = lc_pack_result()
    _check(load_library().lc_pack_selected(ctx, staging or None, capacity, first_rank, C.byref(r)),
           "lc_pack_selected")
    return {"bytes_written": r.bytes_written, "n_packed": r.n_packed, "next_rank": r.next_rank,
            "done": r.done}


def lc_restore_composite(ctx, versions: Sequence[dict], t_fail: int, n_layers: int) -> np.ndarray:
    """versions: dicts with ``step``, ``mask`` (uint8[N] array), ``payload``
    (address int) and ``payload_bytes``."""
    arr = (lc_version * len(versions))()
    keep = []
    for i, v in enumerate(versions):
        m = np.ascontiguousarray(v["mask"], dtype=np.uint8)
        keep.append(m)
        arr[i] = lc_version(int(v["step"]), m.ctypes.data_as(C.POINTER(C.c_uint8)), v["payload"] or None,
                            int(v["payload_bytes"]))
    chosen = np.zeros(n_layers, dtype=np.int64)
    _check(load_library().lc_restore_composite(ctx, arr, len(versions), t_fail,
                                               chosen.ctypes.data_as(C.POINTER(C.c_int64))),
           "lc_restore_composite")
    return chosen


def lc_rebase(ctx, step: int) -> None:
    _check(load_library().lc_rebase(ctx, step), "lc_rebase")


def lc_adamw_step_score(ctx, step: int, grads: Sequence[int], grad_dtype: int, lr: float, beta1: float,
                        beta2: float, eps: float, weight_decay: float, adam_step: int,
                        decay_mask: Optional[Sequence[int]] = None) -> None:
    """grads: one device address per segment, in layout order."""
    g = (C.c_void_p * len(grads))(*[int(x) for x in grads])
    dm = None
    if decay_mask is not None:
        dm_arr = np.ascontiguousarray(decay_mask, dtype=np.uint8)
        dm = dm_arr.ctypes.data_as(C.POINTER(C.c_uint8))
    prm = lc_adamw_params(lr, beta1, beta2, eps, weight_decay, adam_step)
    _check(load_library().lc_adamw_step_score(ctx, step, g, grad_dtype, dm, C.byref(prm)), "lc_adamw_step_score")


def lc_sgd_step_score(ctx, step: int, grads: Sequence[int], grad_dtype: int, lr: float, weight_decay: float,
                      decay_mask: Optional[Sequence[int]] = None) -> None:
    """grads: one device address per segment, in layout order."""
    g = (C.c_void_p * len(grads))(*[int(x) for x in grads])
    dm = None
    if decay_mask is not None:
        dm_arr = np.ascontiguousarray(decay_mask, dtype=np.uint8)
        dm = dm_arr.ctypes.data_as(C.POINTER(C.c_uint8))
    prm = lc_sgd_params(lr, weight_decay)
    _check(load_library().lc_sgd_step_score(ctx, step, g, grad_dtype, dm, C.byref(prm)), "lc_sgd_step_score")


class Store:
    """Persistence store (a directory of version files and a manifest)."""

    def __init__(self, directory: str, record_bytes: Sequence[int], buffer_bytes: int = 0):
        self.n = len(record_bytes)
        rb = (C.c_uint64 * self.n)(*[int(x) for x in record_bytes])
        h = C.c_void_p()
        _check(load_library().lc_store_open(os.fsencode(directory), self.n, rb, buffer_bytes, C.byref(h)),
               "lc_store_open")
        self.h = h

    def append(self, step: int, mask, payload: int, payload_bytes: int, stream: int = 0) -> None:
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        _check(load_library().lc_store_append(self.h, step, m.ctypes.data_as(C.POINTER(C.c_uint8)), payload or None,
                                              payload_bytes, stream or None), "lc_store_append")

    def append_async(self, step: int, mask, payload: int, payload_bytes: int, stream: int = 0,
                     reuse_event: int = 0) -> None:
        """lc_store_append_async: ``stream`` runs on; ``reuse_event`` (a raw
        hipEvent_t, e.g. ``torch.cuda.Event().cuda_event`` once created) marks
        when the payload may be overwritten."""
        m = np.ascontiguousarray(mask, dtype=np.uint8)
        _check(load_library().lc_store_append_async(self.h, step, m.ctypes.data_as(C.POINTER(C.c_uint8)),
                                                    payload or None, payload_bytes, stream or None,
                                                    reuse_event or None), "lc_store_append_async")

    def sync(self) -> None:
        _check(load_library().lc_store_sync(self.h), "lc_store_sync")

    def entries(self):
        n = C.c_uint32()
        _check(load_library().lc_store_count(self.h, C.byref(n)), "lc_store_count")
        out = []
        for i in range(n.value):
            step, nbytes = C.c_int64(), C.c_uint64()
            mask = np.zeros(self.n, dtype=np.uint8)
            _check(load_library().lc_store_entry(self.h, i, C.byref(step), mask.ctypes.data_as(C.POINTER(C.c_uint8)),
                                                 C.byref(nbytes)), "lc_store_entry")
            out.append({"step": step.value, "mask": mask, "payload_bytes": nbytes.value})
        return out

    def plan(self, t_fail: int) -> np.ndarray:
        out = np.zeros(self.n, dtype=np.int64)
        _check(load_library().lc_store_plan(self.h, t_fail, out.ctypes.data_as(C.POINTER(C.c_int64))),
               "lc_store_plan")
        return out

    def restore(self, ctx, t_fail: int) -> np.ndarray:
        out = np.zeros(self.n, dtype=np.int64)
        _check(load_library().lc_store_restore(self.h, ctx, t_fail, out.ctypes.data_as(C.POINTER(C.c_int64))),
               "lc_store_restore")
        return out

    def compact(self, t_keep: int) -> int:
        """Removes versions no plan with t_fail >= t_keep can choose; returns
        the number of files removed."""
        n = C.c_uint32()
        _check(load_library().lc_store_compact(self.h, t_keep, C.byref(n)), "lc_store_compact")
        return n.value

    def discard_after(self, step: int) -> int:
        """Removes the versions newer than ``step`` (an abandoned timeline);
        returns the number of files removed."""
        n = C.c_uint32()
        _check(load_library().lc_store_discard_after(self.h, step, C.byref(n)), "lc_store_discard_after")
        return n.value

    def close(self) -> None:
        if self.h is not None:
            h, self.h = self.h, None
            _check(load_library().lc_store_close(h), "lc_store_close")

    def __enter__(self):
        return self

    def __exit__(self, *exc) -> None:
        self.close()

    def __del__(self):
        # a store dropped without close() still finishes its writes
        if getattr(self, "h", None) is not None and _LIB is not None:
            _LIB.lc_store_close(self.h)
            self.h = None


def lc_read_state(ctx, n_layers: int):
    u = np.zeros(n_layers, dtype=np.float64)
    d = np.zeros(n_layers, dtype=np.float64)
    t = np.zeros(n_layers, dtype=np.int64)
    _check(load_library().lc_read_state(ctx, u.ctypes.data_as(C.POINTER(C.c_double)),
                                        d.ctypes.data_as(C.POINTER(C.c_double)),
                                        t.ctypes.data_as(C.POINTER(C.c_int64))), "lc_read_state")
    return u, d, t


def lc_record_bytes(ctx, layer: int) -> int:
    return int(load_library().lc_record_bytes(ctx, layer))


def lc_destroy(ctx) -> None:
    _check(load_library().lc_destroy(ctx), "lc_destroy")


def segments_from_state(state) -> List[Segment]:
    """Segments of a :class:`paper_2609_27193_amd.inputs.SyntheticState`."""
    out = []
    for seg in state.segments:
        w, s, m, a, v = state.seg_views(seg)
        out.append(Segment(seg.layer, seg.numel, w.data_ptr(), None if s is None else s.data_ptr(),
                           None if m is None else m.data_ptr(), a.data_ptr(), v.data_ptr()))
    return out
