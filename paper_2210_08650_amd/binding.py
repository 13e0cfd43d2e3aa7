"""ctypes binding of libhapi.so, one function per C entry point (same names).

Argument marshalling only: every step of the feature-extraction pass runs in
the library's HIP kernels.  Device pointers are passed as integers or as
objects with a ``data_ptr()`` method (torch tensors); streams as integers or
objects with a ``cuda_stream`` attribute.  A negative status raises
``HapiError`` carrying the library's message.  The library must be built
(``python paper_2210_08650_amd/build.py``); importing without it fails.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhapi.so")

HAPI_OK, HAPI_E_INVAL, HAPI_E_UNSUPPORTED, HAPI_E_NOMEM, HAPI_E_DEVICE = 0, -1, -2, -3, -4
HAPI_F32, HAPI_BF16 = 0, 1
(HAPI_CONV, HAPI_MAXPOOL, HAPI_AVGPOOL, HAPI_BASIC_BLOCK, HAPI_BOTTLENECK, HAPI_PATCH_EMBED,
 HAPI_TOKENS, HAPI_VIT_BLOCK, HAPI_LAYERNORM, HAPI_DENSE_BLOCK, HAPI_PREACT_CONV,
 HAPI_BATCHNORM) = range(12)

__all__ = ["HapiError", "Desc", "hapi_layer", "hapi_model_desc", "hapi_kernel_stat",
           "HAPI_OK", "HAPI_E_INVAL", "HAPI_E_UNSUPPORTED", "HAPI_E_NOMEM", "HAPI_E_DEVICE",
           "HAPI_F32", "HAPI_BF16", "HAPI_CONV", "HAPI_MAXPOOL", "HAPI_AVGPOOL",
           "HAPI_BASIC_BLOCK", "HAPI_BOTTLENECK", "HAPI_PATCH_EMBED", "HAPI_TOKENS",
           "HAPI_VIT_BLOCK", "HAPI_LAYERNORM", "HAPI_DENSE_BLOCK", "HAPI_PREACT_CONV",
           "HAPI_BATCHNORM", "LIB_PATH", "EXPORTED",
           "hapi_raw_weight_count", "hapi_packed_weight_bytes", "hapi_pack_weights",
           "hapi_layer_shape", "hapi_workspace_bytes", "hapi_chunk_count", "hapi_extract",
           "hapi_workspace_guards", "HAPI_GUARD_BYTES", "hapi_extract_range",
           "hapi_extract_noalloc", "HAPI_NOALLOC_SCRATCH_BYTES", "hapi_profile_layers", "hapi_profile_memory",
           "hapi_stats_enable", "hapi_stats_collect", "hapi_last_error", "hapi_split_job", "hapi_split_estimate", "hapi_split_choice", "hapi_choose_split"]

_STATUS = {HAPI_E_INVAL: "HAPI_E_INVAL", HAPI_E_UNSUPPORTED: "HAPI_E_UNSUPPORTED",
           HAPI_E_NOMEM: "HAPI_E_NOMEM", HAPI_E_DEVICE: "HAPI_E_DEVICE"}


class HapiError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"{_STATUS.get(code, code)}: {message}")
        self.code = code


class hapi_layer(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("cin", ctypes.c_int32), ("cout", ctypes.c_int32),
                ("width", ctypes.c_int32), ("k", ctypes.c_int32), ("stride", ctypes.c_int32),
                ("pad", ctypes.c_int32), ("relu", ctypes.c_int32), ("has_bias", ctypes.c_int32),
                ("has_bn", ctypes.c_int32), ("heads", ctypes.c_int32), ("mlp_dim", ctypes.c_int32),
                ("reserved", ctypes.c_int32 * 4)]


class hapi_model_desc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("layers", ctypes.POINTER(hapi_layer)),
                ("dtype", ctypes.c_int32), ("in_c", ctypes.c_int32), ("in_h", ctypes.c_int32),
                ("in_w", ctypes.c_int32), ("stream", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p), ("workspace_bytes", ctypes.c_size_t),
                ("chunk", ctypes.c_int32), ("inflight", ctypes.c_int32),
                ("direct", ctypes.c_int32)]


class hapi_kernel_stat(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double), ("busy_ms", ctypes.c_double)]


class hapi_split_job(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("freeze_idx", ctypes.c_int32),
                ("train_batch", ctypes.c_int32), ("request_images", ctypes.c_int32),
                ("server_slots", ctypes.c_int32), ("reserved0", ctypes.c_int32),
                ("iterations", ctypes.c_int64),
                ("image_bytes", ctypes.POINTER(ctypes.c_int64)),
                ("srv_layer_s", ctypes.POINTER(ctypes.c_double)),
                ("cli_layer_s", ctypes.POINTER(ctypes.c_double)),
                ("srv_read_data_s", ctypes.c_double), ("srv_read_model_s", ctypes.c_double),
                ("srv_to_gpu_s", ctypes.c_double), ("cli_rest_s", ctypes.c_double),
                ("srv_from_gpu_s_per_byte", ctypes.c_double),
                ("srv_pickle_s_per_byte", ctypes.c_double),
                ("cli_unpickle_s_per_byte", ctypes.c_double),
                ("cli_loader_s_per_byte", ctypes.c_double),
                ("cli_to_gpu_s_per_byte", ctypes.c_double),
                ("net_bytes_per_s", ctypes.c_double),
                ("cli_mem_bytes", ctypes.c_int64), ("cli_fixed_mem_bytes", ctypes.c_int64),
                ("nosplit_iter_s", ctypes.c_double)]


class hapi_split_estimate(ctypes.Structure):
    _fields_ = [("rt_srv", ctypes.c_double), ("rt_nw", ctypes.c_double),
                ("rt_cli", ctypes.c_double), ("epoch_s", ctypes.c_double),
                ("sum_s", ctypes.c_double), ("cli_mem_bytes", ctypes.c_int64),
                ("oom", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class hapi_split_choice(ctypes.Structure):
    _fields_ = [("hapi", ctypes.c_int32), ("earliest", ctypes.c_int32),
                ("freeze", ctypes.c_int32), ("min_output", ctypes.c_int32),
                ("nosplit", ctypes.c_int32), ("nsg", ctypes.c_int32)]


def _hip_runtimes():
    try:
        with open("/proc/self/maps") as f:
            return {line.split()[-1] for line in f if "libamdhip64" in line}
    except OSError:
        return set()


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python paper_2210_08650_amd/build.py`")
    # libhapi must share torch's HIP runtime (streams and device pointers come
    # from torch).  Importing torch first maps torch's libamdhip64, whose soname
    # then satisfies libhapi's dependency; loading libhapi first would map a
    # second runtime that does not see torch's device state.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    if len(_hip_runtimes()) > 1:
        raise ImportError(f"two HIP runtimes are mapped: {sorted(_hip_runtimes())}")
    D = ctypes.POINTER(hapi_model_desc)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    sig = {
        "hapi_raw_weight_count": (i64, [D]),
        "hapi_packed_weight_bytes": (i64, [D]),
        "hapi_pack_weights": (ctypes.c_int, [D, vp, vp]),
        "hapi_layer_shape": (ctypes.c_int, [D, i32, ctypes.POINTER(i64), ctypes.POINTER(i32)]),
        "hapi_workspace_bytes": (i64, [D, i32, i32, i32]),
        "hapi_chunk_count": (i32, [D, i32]),
        "hapi_workspace_guards": (i32, [D, i32, i32, ctypes.POINTER(i64), i32]),
        "hapi_extract": (ctypes.c_int, [D, vp, vp, i32, i32, vp]),
        "hapi_extract_range": (ctypes.c_int, [D, vp, vp, i32, i32, i32, vp]),
        "hapi_extract_noalloc": (ctypes.c_int, [D, vp, vp, i32, i32, vp]),
        "hapi_profile_layers": (ctypes.c_int, [D, i32, ctypes.POINTER(i64),
                                               ctypes.POINTER(ctypes.c_float)]),
        "hapi_profile_memory": (ctypes.c_int, [D, i32, ctypes.POINTER(i64)]),
        "hapi_stats_enable": (ctypes.c_int, [i32]),
        "hapi_stats_collect": (ctypes.c_int, [ctypes.POINTER(hapi_kernel_stat), i32]),
        "hapi_last_error": (ctypes.c_char_p, []),
        "hapi_choose_split": (ctypes.c_int, [ctypes.POINTER(hapi_split_job),
                                             ctypes.POINTER(hapi_split_estimate),
                                             ctypes.POINTER(hapi_split_choice)]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype, f.argtypes = res, args
    return lib


_lib = _load()
EXPORTED = ("hapi_raw_weight_count", "hapi_packed_weight_bytes", "hapi_pack_weights",
            "hapi_layer_shape", "hapi_workspace_bytes", "hapi_chunk_count", "hapi_extract",
            "hapi_workspace_guards", "hapi_extract_range", "hapi_extract_noalloc", "hapi_profile_layers", "hapi_profile_memory",
            "hapi_stats_enable", "hapi_stats_collect", "hapi_last_error", "hapi_choose_split")


def _ptr(p):
    if p is None:
        return None
    if hasattr(p, "data_ptr"):
        return p.data_ptr()
    return int(p)


def _stream(s):
    if s is None:
        return None
    if hasattr(s, "cuda_stream"):
        return s.cuda_stream
    return int(s)


def _check(code):
    if code < 0:
        raise HapiError(int(code), hapi_last_error())
    return code


class Desc:
    """Owns a ``hapi_model_desc`` and the layer array it points to."""

    def __init__(self, layers, dtype, in_shape=(3, 224, 224), stream=None, workspace=None,
                 workspace_bytes=0, chunk=0, inflight=0, direct=0):
        self._layers = (hapi_layer * len(layers))()
        for i, spec in enumerate(layers):
            if isinstance(spec, hapi_layer):
                self._layers[i] = spec
            else:
                for key, val in spec.items():
                    setattr(self._layers[i], key, val)
        self.c = hapi_model_desc()
        self.c.n_layers = len(layers)
        self.c.layers = ctypes.cast(self._layers, ctypes.POINTER(hapi_layer))
        self.c.dtype = dtype
        self.c.in_c, self.c.in_h, self.c.in_w = in_shape
        self.set(stream=stream, workspace=workspace, workspace_bytes=workspace_bytes, chunk=chunk,
                 inflight=inflight, direct=direct)

    def set(self, stream=None, workspace=None, workspace_bytes=None, chunk=None, inflight=None,
            direct=None):
        if stream is not None:
            self.c.stream = _stream(stream)
        if workspace is not None:
            # Keep the owner alive while the descriptor points at its memory: a
            # temporary tensor would otherwise return to torch's caching
            # allocator and be reused under the library's feet.
            self._workspace = workspace
            self.c.workspace = _ptr(workspace)
        if workspace_bytes is not None:
            self.c.workspace_bytes = int(workspace_bytes)
        if chunk is not None:
            self.c.chunk = int(chunk)
        if inflight is not None:
            self.c.inflight = int(inflight)
        if direct is not None:
            self.c.direct = int(direct)
        return self

    @property
    def ref(self):
        return ctypes.byref(self.c)

    @property
    def n_layers(self):
        return self.c.n_layers


def hapi_raw_weight_count(desc: Desc) -> int:
    return _check(_lib.hapi_raw_weight_count(desc.ref))


def hapi_packed_weight_bytes(desc: Desc) -> int:
    return _check(_lib.hapi_packed_weight_bytes(desc.ref))


def hapi_pack_weights(desc: Desc, raw_weights, packed) -> None:
    _check(_lib.hapi_pack_weights(desc.ref, _ptr(raw_weights), _ptr(packed)))


def hapi_layer_shape(desc: Desc, layer: int) -> tuple:
    dims = (ctypes.c_int64 * 3)()
    nd = ctypes.c_int32()
    _check(_lib.hapi_layer_shape(desc.ref, int(layer), dims, ctypes.byref(nd)))
    return tuple(int(dims[i]) for i in range(nd.value))


def hapi_workspace_bytes(desc: Desc, batch: int, split_layer: int, profile: bool = False) -> int:
    return _check(_lib.hapi_workspace_bytes(desc.ref, int(batch), int(split_layer), int(profile)))


HAPI_GUARD_BYTES = 4096


def hapi_workspace_guards(desc: Desc, batch: int, split_layer: int) -> list:
    """Byte offsets (relative to the workspace) of the HAPI_GUARD_BYTES gaps no
    kernel writes."""
    n = _check(_lib.hapi_workspace_guards(desc.ref, int(batch), int(split_layer), None, 0))
    arr = (ctypes.c_int64 * max(n, 1))()
    _check(_lib.hapi_workspace_guards(desc.ref, int(batch), int(split_layer), arr, n))
    return [int(arr[i]) for i in range(n)]


def hapi_chunk_count(desc: Desc, batch: int) -> int:
    return _check(_lib.hapi_chunk_count(desc.ref, int(batch)))


def hapi_extract(desc: Desc, weights, images, batch: int, split_layer: int, out) -> None:
    _check(_lib.hapi_extract(desc.ref, _ptr(weights), _ptr(images), int(batch),
                             int(split_layer), _ptr(out)))


HAPI_NOALLOC_SCRATCH_BYTES = 256 << 20


def hapi_extract_noalloc(desc: Desc, weights, images, batch: int, split_layer: int, out) -> None:
    _check(_lib.hapi_extract_noalloc(desc.ref, _ptr(weights), _ptr(images), int(batch),
                                     int(split_layer), _ptr(out)))


def hapi_extract_range(desc: Desc, weights, input, batch: int, start_layer: int,
                       end_layer: int, out) -> None:
    _check(_lib.hapi_extract_range(desc.ref, _ptr(weights), _ptr(input), int(batch),
                                   int(start_layer), int(end_layer), _ptr(out)))


def hapi_profile_layers(desc: Desc, batch: int, time_layers: bool = False):
    """Returns (out_bytes[0..n], out_us[0..n] or None)."""
    n = desc.n_layers + 1
    b = (ctypes.c_int64 * n)()
    us = (ctypes.c_float * n)() if time_layers else None
    _check(_lib.hapi_profile_layers(desc.ref, int(batch), b, us))
    return [int(v) for v in b], ([float(v) for v in us] if us is not None else None)


def hapi_profile_memory(desc: Desc, batch: int) -> list:
    """Device bytes of an extraction to every split 0..n_layers."""
    b = (ctypes.c_int64 * (desc.n_layers + 1))()
    _check(_lib.hapi_profile_memory(desc.ref, int(batch), b))
    return [int(v) for v in b]


def hapi_stats_enable(enable: bool) -> None:
    _check(_lib.hapi_stats_enable(int(bool(enable))))


def hapi_stats_collect(max_entries: int = 16) -> list:
    arr = (hapi_kernel_stat * max_entries)()
    n = _check(_lib.hapi_stats_collect(arr, max_entries))
    return [dict(name=arr[i].name.decode(), launches=int(arr[i].launches),
                 total_ms=float(arr[i].total_ms), flops=float(arr[i].flops),
                 bytes=float(arr[i].bytes), busy_ms=float(arr[i].busy_ms))
            for i in range(min(n, max_entries))]


def hapi_last_error() -> str:
    msg = _lib.hapi_last_error()
    return msg.decode() if msg else ""


_SPLIT_ARRAYS = {"image_bytes": ctypes.c_int64, "srv_layer_s": ctypes.c_double,
                 "cli_layer_s": ctypes.c_double}


def hapi_choose_split(**job):
    """Fields of ``hapi_split_job`` as keywords (the three per-layer arrays as
    sequences of ``n_layers + 1`` values).  Returns ``(choice, estimates)``:
    a dict of the ``hapi_split_choice`` fields and one dict of
    ``hapi_split_estimate`` fields per split 0..freeze_idx."""
    j = hapi_split_job()
    keep = []
    for key, val in job.items():
        if key in _SPLIT_ARRAYS:
            if len(val) != int(job.get("n_layers", 0)) + 1:
                raise ValueError(f"{key} must hold n_layers + 1 values, got {len(val)}")
            arr = (_SPLIT_ARRAYS[key] * len(val))(*val)
            keep.append(arr)
            setattr(j, key, ctypes.cast(arr, ctypes.POINTER(_SPLIT_ARRAYS[key])))
        else:
            setattr(j, key, val)
    nf = max(int(j.freeze_idx), 0) + 1
    est = (hapi_split_estimate * nf)()
    ch = hapi_split_choice()
    _check(_lib.hapi_choose_split(ctypes.byref(j), est, ctypes.byref(ch)))
    choice = {name: int(getattr(ch, name)) for name, _ in hapi_split_choice._fields_}
    rows = [{name: (int(v) if isinstance(v, int) else float(v))
             for name, v in ((f, getattr(est[s], f)) for f, _ in hapi_split_estimate._fields_)
             if name != "reserved"} for s in range(nf)]
    return choice, rows
