"""Thin ctypes binding over libspecdec.so (argument marshalling only).

Every function named ``specdec_*`` here calls the C entry point of the same
name; torch tensors are passed as device pointers and torch only provides
device memory and streams.  The classes bundle the buffers a caller owns
(weights, workspace, KV storage) with their handles.

The library must be built (``paper_2608_10362_amd.build.build()``); loading
fails loudly otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspecdec.so")

SPECDEC_F32, SPECDEC_BF16 = 0, 1
ROLE_TARGET, ROLE_DRAFT = 0, 1
INPUT_PROBS, INPUT_LOGITS = 0, 1
PURPOSE_DRAFT, PURPOSE_ACCEPT, PURPOSE_RESAMPLE = 0, 1, 2

STATUS = {0: "ok", -1: "invalid argument", -2: "unsupported shape", -3: "KV capacity exceeded",
          -4: "non-finite probability or logit", -5: "HIP runtime error", -6: "unsupported request",
          -7: "token id out of range",
          -8: "request needs more scratch than the static no-allocation buffer holds",
          -9: "a kernel's bounded wait for other blocks ran out"}


# Size of the static scratch of specdec_accept_noalloc (SPECDEC_ACCEPT_NOALLOC_SCRATCH_BYTES).
ACCEPT_NOALLOC_SCRATCH_BYTES = 2 << 20


class SpecdecError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {STATUS.get(status, status)} ({status})")
        self.status = status


class ModelDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
                ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
                ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
                ("dtype", ctypes.c_int32)]


_PP = ctypes.POINTER(ctypes.c_void_p)


class Weights(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("lm_head", ctypes.c_void_p), ("final_norm", ctypes.c_void_p),
                ("attn_norm", _PP), ("wq", _PP), ("wk", _PP), ("wv", _PP), ("wo", _PP), ("ffn_norm", _PP),
                ("w_gate", _PP), ("w_up", _PP), ("w_down", _PP)]


class KV(ctypes.Structure):
    _fields_ = [("data", ctypes.c_void_p), ("state", ctypes.c_void_p), ("batch", ctypes.c_int32),
                ("capacity", ctypes.c_int32), ("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("len_upper", ctypes.c_int64)]


_lib = None

_SIGS = {
    "specdec_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(ModelDesc), ctypes.c_int32, ctypes.c_int32]),
    "specdec_packed_bytes": (ctypes.c_size_t, [ctypes.POINTER(ModelDesc), ctypes.c_int32]),
    "specdec_packed_bytes_fmt": (ctypes.c_size_t, [ctypes.POINTER(ModelDesc), ctypes.c_int32, ctypes.c_int32]),
    "specdec_pack_weights_fmt": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.c_int32,
                                                ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "specdec_model_create_fmt": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.c_int32,
                                                ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32,
                                                ctypes.c_int32, ctypes.c_void_p, ctypes.c_size_t,
                                                ctypes.POINTER(ctypes.c_void_p)]),
    "specdec_pack_weights": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.c_int32,
                                            ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]),
    "specdec_model_create": (ctypes.c_int, [ctypes.POINTER(ModelDesc), ctypes.POINTER(Weights), ctypes.c_int32,
                                            ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_void_p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_void_p)]),
    "specdec_model_destroy": (None, [ctypes.c_void_p]),
    "specdec_kv_bytes": (ctypes.c_size_t, [ctypes.POINTER(ModelDesc), ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "specdec_kv_state_count": (ctypes.c_int32, [ctypes.c_int32]),
    "specdec_kv_init": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                       ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_kv_write_context": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                                ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_kv_read_context": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                               ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_kv_set_state": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                            ctypes.c_void_p]),
    "specdec_kv_read_state": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                             ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_prefill": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(KV), ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.c_void_p]),
    "specdec_draft_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(KV), ctypes.c_int32, ctypes.c_int32,
                                          ctypes.c_float, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                          ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_verify": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(KV), ctypes.c_int32, ctypes.c_void_p,
                                      ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_accept": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_float,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32,
                                      ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_size_t, ctypes.c_void_p]),
    "specdec_accept_workspace_bytes": (ctypes.c_size_t, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]),
    "specdec_accept_noalloc": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                              ctypes.c_float, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_int32, ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64,
                                              ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                              ctypes.c_void_p]),
    "specdec_packed_range": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                                            ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t)]),
    "specdec_event_create": (ctypes.c_int, [ctypes.POINTER(ctypes.c_void_p)]),
    "specdec_event_destroy": (ctypes.c_int, [ctypes.c_void_p]),
    "specdec_load_async": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                                          ctypes.c_void_p]),
    "specdec_stream_wait_event": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_event_query": (ctypes.c_int, [ctypes.c_void_p, ctypes.POINTER(ctypes.c_int32)]),
    "specdec_kv_commit": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_kv_step_word": (ctypes.c_void_p, [ctypes.POINTER(KV)]),
    "specdec_sample": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_int64,
                                      ctypes.c_void_p, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32,
                                      ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_draw_u32": (ctypes.c_int, [ctypes.c_int32, ctypes.c_uint64, ctypes.c_uint64, ctypes.c_int32,
                                        ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_device_status": (ctypes.c_int, [ctypes.POINTER(KV), ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "specdec_last_hip_error": (ctypes.c_char_p, []),
    "specdec_stream_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_timing_enable": (ctypes.c_int, [ctypes.c_int32]),
    "specdec_timing_read": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_void_p]),
    "specdec_time_kernel": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p]),
}

KERNEL_KINDS = ("embed", "qkv", "rope_append", "attention", "o_proj", "gate_up", "down", "lm_head", "draft_finish",
                "accept", "commit")


def lib() -> ctypes.CDLL:
    """Load libspecdec.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2608_10362_amd.build.build()")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(l, name)
            f.restype = res
            f.argtypes = args
        _lib = l
    return _lib


def _check(status: int, what: str):
    if status != 0:
        if status == -5:  # name the HIP error behind it
            what = f"{what} [{lib().specdec_last_hip_error().decode()}]"
        raise SpecdecError(status, what)


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev(t, name: str, dtype=None, numel: int = 0, optional: bool = False):
    """Check that a tensor argument is a contiguous device tensor of the right type and size."""
    import torch
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name}: missing")
    if not isinstance(t, torch.Tensor) or t.device.type != "cuda":
        raise ValueError(f"{name}: expected a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if t.numel() < numel:
        raise ValueError(f"{name}: needs at least {numel} elements, has {t.numel()}")
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def make_desc(shape) -> ModelDesc:
    return ModelDesc(shape.n_layers, shape.d_model, shape.n_heads, shape.n_kv_heads, shape.head_dim, shape.ffn_dim,
                     shape.vocab, shape.rms_eps, shape.rope_base,
                     SPECDEC_BF16 if shape.dtype == "bf16" else SPECDEC_F32)


def workspace_bytes(shape, max_rows: int, max_ctx: int) -> int:
    d = make_desc(shape)
    return lib().specdec_workspace_bytes(ctypes.byref(d), max_rows, max_ctx)


def kv_bytes(shape, n_layers: int, batch: int, capacity: int) -> int:
    d = make_desc(shape)
    return lib().specdec_kv_bytes(ctypes.byref(d), n_layers, batch, capacity)


# ---------------------------------------------------------------- device weights
def _to_device(arr, dtype: str, device):
    import torch
    if isinstance(arr, torch.Tensor):
        return arr.to(device).contiguous()
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)).to(device)


class DeviceWeights:
    """Device copies of a model's weights (from synth's numpy dict, or torch tensors).

    For bf16 models the matrices are packed once (specdec_pack_weights) into
    ``self.packed``; the row-major matrices are then released unless
    ``keep_rowmajor`` is set (the embedding and RMSNorm gains stay).
    """

    KEYS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")
    MATS = ("wq", "wk", "wv", "wo", "w_gate", "w_up", "w_down")

    FORMATS = {"bf16": 0, "int4": 1}  # SPECDEC_WEIGHTS_*

    def __init__(self, shape, weights: Dict, device="cuda", keep_rowmajor: bool = False, stream=None,
                 weight_format: str = "bf16"):
        """``weight_format`` (bf16 models): "bf16", or "int4" for the INT4 image
        (layer matrices quantized on the device, see specdec_pack_weights_fmt)."""
        import torch
        if weight_format not in self.FORMATS or (weight_format != "bf16" and shape.dtype != "bf16"):
            raise ValueError(f"weight format {weight_format!r} for a {shape.dtype} model")
        self.weight_format = weight_format
        self.shape = shape
        self.t = {k: _to_device(weights[k], shape.dtype, device) for k in ("embed", "lm_head", "final_norm")}
        self.layers = [{k: _to_device(L[k], shape.dtype, device) for k in self.KEYS} for L in weights["layers"]]
        self.packed = None
        if shape.dtype == "bf16":
            desc = make_desc(shape.with_layers(self.n_layers))
            fmt = self.FORMATS[weight_format]
            nbytes = lib().specdec_packed_bytes_fmt(ctypes.byref(desc), self.n_layers, fmt)
            if nbytes == 0:
                raise SpecdecError(-2, "specdec_packed_bytes_fmt")
            self.packed = torch.empty(nbytes, dtype=torch.uint8, device=self.t["embed"].device)
            w, keep = self.c_struct(self.n_layers)
            _check(lib().specdec_pack_weights_fmt(ctypes.byref(desc), ctypes.byref(w), self.n_layers, fmt,
                                                  self.packed.data_ptr(), nbytes, _stream(stream)),
                   "specdec_pack_weights_fmt")
            torch.cuda.current_stream().synchronize() if stream is None else stream.synchronize()
            if not keep_rowmajor:
                self.t["lm_head"] = None
                for L in self.layers:
                    for k in self.MATS:
                        L[k] = None

    @property
    def n_layers(self):
        return len(self.layers)

    def c_struct(self, n_layers: int):
        arrays = {}
        for k in self.KEYS:
            arr = (ctypes.c_void_p * n_layers)(*[_ptr(self.layers[l][k]) for l in range(n_layers)])
            arrays[k] = arr
        w = Weights(self.t["embed"].data_ptr(), _ptr(self.t["lm_head"]), self.t["final_norm"].data_ptr(),
                    *[ctypes.cast(arrays[k], _PP) for k in self.KEYS])
        return w, arrays


class Model:
    """A model handle (target, or a draft = layer prefix) with its own workspace."""

    def __init__(self, dw: DeviceWeights, n_layers: int, max_rows: int, max_ctx: int, packed=None):
        """``packed``: a device image to run from instead of ``dw.packed`` (a
        draft slot, see DraftSlot); it must hold at least ``n_layers`` layers."""
        import torch
        self.dw = dw
        self.shape = dw.shape
        self.n_layers = n_layers
        self.desc = make_desc(dw.shape.with_layers(dw.n_layers))
        nbytes = lib().specdec_workspace_bytes(ctypes.byref(self.desc), max_rows, max_ctx)
        if nbytes == 0:
            raise SpecdecError(-2, "specdec_workspace_bytes")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=dw.t["embed"].device)
        w, self._arrays = dw.c_struct(n_layers)
        h = ctypes.c_void_p()
        pk = dw.packed if packed is None else packed
        if packed is not None:
            _dev(packed, "packed", torch.uint8, 1)
        self._packed = pk  # (kept alive with the handle)
        _check(lib().specdec_model_create_fmt(ctypes.byref(self.desc), ctypes.byref(w), n_layers,
                                              DeviceWeights.FORMATS[dw.weight_format], _ptr(pk),
                                              0 if pk is None else pk.numel(), max_rows, max_ctx,
                                              self.workspace.data_ptr(), nbytes, ctypes.byref(h)),
               "specdec_model_create_fmt")
        self.handle = h

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.specdec_model_destroy(self.handle)
            self.handle = None


class KVCache:
    """KV storage + sequence state of one model instance."""

    def __init__(self, model: Model, batch: int, capacity: int, stream=None):
        import torch
        self.model = model
        dev = model.workspace.device
        nbytes = lib().specdec_kv_bytes(ctypes.byref(model.desc), model.n_layers, batch, capacity)
        self.data = torch.empty(nbytes, dtype=torch.uint8, device=dev)
        self.state = torch.zeros(lib().specdec_kv_state_count(batch), dtype=torch.int32, device=dev)
        self.kv = KV()
        _check(lib().specdec_kv_init(ctypes.byref(self.kv), model.handle, batch, capacity, self.data.data_ptr(),
                                     nbytes, self.state.data_ptr(), _stream(stream)), "specdec_kv_init")

    @property
    def batch(self):
        return self.kv.batch

    def storage_dtype(self):
        import torch
        return torch.bfloat16 if self.kv.dtype == SPECDEC_BF16 else torch.float32

    def write_context(self, layer: int, b: int, pos0: int, k, v, stream=None):
        n = k.shape[0]
        _dev(k, "k", self.storage_dtype(), n * self.kv.n_kv_heads * self.kv.head_dim)
        _dev(v, "v", self.storage_dtype(), n * self.kv.n_kv_heads * self.kv.head_dim)
        _check(lib().specdec_kv_write_context(ctypes.byref(self.kv), layer, b, pos0, k.shape[0], k.data_ptr(),
                                              v.data_ptr(), _stream(stream)), "specdec_kv_write_context")

    def read_context(self, layer: int, b: int, pos0: int, n: int, stream=None):
        import torch
        shp = (n, self.kv.n_kv_heads, self.kv.head_dim)
        k = torch.empty(shp, dtype=self.storage_dtype(), device=self.data.device)
        v = torch.empty_like(k)
        _check(lib().specdec_kv_read_context(ctypes.byref(self.kv), layer, b, pos0, n, k.data_ptr(), v.data_ptr(),
                                             _stream(stream)), "specdec_kv_read_context")
        return k, v

    def set_state(self, length, pending, n_pending, stream=None):
        L = np.ascontiguousarray(length, dtype=np.int32)
        P = np.ascontiguousarray(pending, dtype=np.int32).reshape(-1)
        N = np.ascontiguousarray(n_pending, dtype=np.int32)
        _check(lib().specdec_kv_set_state(ctypes.byref(self.kv), L.ctypes.data, P.ctypes.data, N.ctypes.data,
                                          _stream(stream)), "specdec_kv_set_state")

    def read_state(self, stream=None):
        B = self.batch
        L = np.zeros(B, np.int32)
        P = np.zeros(2 * B, np.int32)
        N = np.zeros(B, np.int32)
        S = np.zeros(1, np.int32)
        _check(lib().specdec_kv_read_state(ctypes.byref(self.kv), L.ctypes.data, P.ctypes.data, N.ctypes.data,
                                           S.ctypes.data, _stream(stream)), "specdec_kv_read_state")
        return {"len": L, "pending": P.reshape(B, 2), "n_pending": N, "status": int(S[0])}

    def step_word(self) -> int:
        """Device address of the commit counter (the step_dev argument)."""
        return int(lib().specdec_kv_step_word(ctypes.byref(self.kv)))

    def read_step(self) -> int:
        """The commit counter's value (synchronizes the current stream)."""
        B = self.batch
        return int(self.state[4 * B + 2:4 * B + 4].cpu().numpy().view(np.uint64)[0])


# ---------------------------------------------------------------- draft reload
def packed_range(shape, first_layer: int, n_layers: int):
    """(offset, bytes) of layers [first_layer, first_layer + n_layers) in the packed image."""
    d = make_desc(shape)
    off, nb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().specdec_packed_range(ctypes.byref(d), first_layer, n_layers, ctypes.byref(off), ctypes.byref(nb)),
           "specdec_packed_range")
    return off.value, nb.value


class Event:
    """A completion event owned by the library (see specdec_event_create)."""

    def __init__(self):
        h = ctypes.c_void_p()
        _check(lib().specdec_event_create(ctypes.byref(h)), "specdec_event_create")
        self.handle = h

    def query(self) -> bool:
        done = ctypes.c_int32(0)
        _check(lib().specdec_event_query(self.handle, ctypes.byref(done)), "specdec_event_query")
        return bool(done.value)

    def wait(self, stream=None):
        """Make `stream` (default: the current one) wait for the event."""
        _check(lib().specdec_stream_wait_event(_stream(stream), self.handle), "specdec_stream_wait_event")

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.specdec_event_destroy(self.handle)
            self.handle = None


class DraftSlot:
    """One resident draft slot: a device buffer in the packed-image format for
    drafts of up to ``max_layers`` layers (drafts are layer prefixes of the
    target, so their images are prefixes of its image).  The backing storage
    is a pinned host copy of that image prefix.  The shared LM head is copied
    into the slot once; ``load_async`` then re-sends only the layers of the
    draft being made resident, on ``copy_stream``, and ``event`` completes when
    they have landed."""

    def __init__(self, dw: DeviceWeights, max_layers: int):
        import torch
        if dw.packed is None:
            raise ValueError("draft slots hold packed (bf16) images")
        self.shape = dw.shape.with_layers(dw.n_layers)
        self.max_layers = max_layers
        off0, nb = packed_range(self.shape, 0, max_layers)
        self.nbytes = off0 + nb
        dev = dw.packed.device
        self.slot = torch.empty(self.nbytes, dtype=torch.uint8, device=dev)
        self.host = torch.empty(self.nbytes, dtype=torch.uint8, pin_memory=True)
        self.host.copy_(dw.packed[:self.nbytes])
        self.slot[:off0].copy_(dw.packed[:off0])  # the shared LM head, once
        torch.cuda.current_stream().synchronize()
        self.event = Event()
        self.layers = 0  # layers whose load has been issued

    def load_async(self, n_layers: int, copy_stream=None) -> int:
        """Issue the H2D copy of layers [0, n_layers); returns the bytes sent."""
        if not 0 < n_layers <= self.max_layers:
            raise ValueError("n_layers outside the slot")
        off, nb = packed_range(self.shape, 0, n_layers)
        _check(lib().specdec_load_async(self.slot.data_ptr() + off, self.host.data_ptr() + off, nb,
                                        _stream(copy_stream), self.event.handle), "specdec_load_async")
        self.layers = n_layers
        return nb


# ---------------------------------------------------------------- entry points
def specdec_prefill(model: Model, kv: KVCache, tokens, stream=None):
    """tokens: device int32 [batch, n]."""
    import torch
    _dev(tokens, "tokens", torch.int32, kv.batch * tokens.shape[-1])
    if tokens.dim() != 2 or tokens.shape[0] != kv.batch:
        raise ValueError("tokens: expected [batch, n]")
    _check(lib().specdec_prefill(model.handle, ctypes.byref(kv.kv), tokens.shape[1], tokens.data_ptr(),
                                 _stream(stream)), "specdec_prefill")


def specdec_draft_step(draft: Model, kv: KVCache, gamma: int, slot: int, temperature: float, seed: int, step: int,
                       rand, q_out, d_out, ld_d: int, logits_out=None, stream=None, step_dev=None):
    """step_dev: a cache's KVCache.step_word() (device address of its commit
    counter) read in place of `step`, or None."""
    import torch
    B, V = kv.batch, draft.shape.vocab
    if rand is not None:
        _dev(rand, "rand", None, B)
        if rand.element_size() != 4:
            raise ValueError("rand: expected 32-bit words")
    _dev(q_out, "q_out", torch.float32, B * gamma * V, optional=temperature == 0)
    _dev(d_out, "d_out", torch.int32, (B - 1) * ld_d + gamma)
    _dev(logits_out, "logits_out", torch.float32, B * V, optional=True)
    _check(lib().specdec_draft_step(draft.handle, ctypes.byref(kv.kv), gamma, slot, temperature, seed, step,
                                    step_dev, _ptr(rand), _ptr(q_out), d_out.data_ptr(), ld_d, _ptr(logits_out),
                                    _stream(stream)), "specdec_draft_step")


def specdec_verify(target: Model, kv: KVCache, gamma: int, d, ld_d: int, logits_out, stream=None):
    import torch
    B, V = kv.batch, target.shape.vocab
    _dev(d, "d", torch.int32, (B - 1) * ld_d + gamma, optional=gamma == 0)
    _dev(logits_out, "logits_out", torch.float32, B * (gamma + 1) * V)
    _check(lib().specdec_verify(target.handle, ctypes.byref(kv.kv), gamma, _ptr(d), ld_d, logits_out.data_ptr(),
                                _stream(stream)), "specdec_verify")


def specdec_accept_workspace_bytes(batch: int, gamma: int, vocab: int) -> int:
    return int(lib().specdec_accept_workspace_bytes(batch, gamma, vocab))


def accept_workspace(batch: int, gamma: int, vocab: int, device="cuda"):
    """A device buffer large enough for specdec_accept's workspace."""
    import torch
    n = specdec_accept_workspace_bytes(batch, gamma, vocab)
    if n == 0:
        raise ValueError("specdec_accept does not support these sizes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def specdec_accept(batch: int, gamma: int, vocab: int, input_kind: int, temperature: float, p, q, d, ld_d: int,
                   rand, seed: int, step: int, n_accepted, next_token, status=None, workspace=None, stream=None,
                   step_dev=None):
    """Accept / resample.  `workspace` (uint8 device tensor) is allocated per
    call when not given; pass one from accept_workspace() in loops.  step_dev:
    as for specdec_draft_step."""
    import torch
    _dev(p, "p", torch.float32, batch * (gamma + 1) * vocab)
    _dev(q, "q", torch.float32, batch * gamma * vocab, optional=temperature == 0 or gamma == 0)
    _dev(d, "d", torch.int32, (batch - 1) * ld_d + gamma, optional=gamma == 0)
    if rand is not None:
        _dev(rand, "rand", rand.dtype, batch * (gamma + 1))
        if rand.dtype not in (torch.int32, torch.uint32):
            raise ValueError("rand: expected 32-bit words")
    _dev(n_accepted, "n_accepted", torch.int32, batch)
    _dev(next_token, "next_token", torch.int32, batch)
    _dev(status, "status", torch.int32, 1, optional=True)
    if workspace is None:
        workspace = accept_workspace(batch, gamma, vocab, p.device)
    _dev(workspace, "workspace", torch.uint8, 1)
    _check(lib().specdec_accept(batch, gamma, vocab, input_kind, temperature, p.data_ptr(), _ptr(q), _ptr(d), ld_d,
                                _ptr(rand), seed, step, step_dev, n_accepted.data_ptr(), next_token.data_ptr(),
                                _ptr(status), workspace.data_ptr(), workspace.numel(), _stream(stream)),
           "specdec_accept")


def specdec_accept_noalloc(batch: int, gamma: int, vocab: int, input_kind: int, temperature: float, p, q, d,
                           ld_d: int, rand, seed: int, step: int, n_accepted, next_token, status=None, stream=None,
                           step_dev=None):
    """specdec_accept with the library's static scratch (no workspace, no allocation)."""
    import torch
    _dev(p, "p", torch.float32, batch * (gamma + 1) * vocab)
    _dev(q, "q", torch.float32, batch * gamma * vocab, optional=temperature == 0 or gamma == 0)
    _dev(d, "d", torch.int32, (batch - 1) * ld_d + gamma, optional=gamma == 0)
    if rand is not None:
        _dev(rand, "rand", rand.dtype, batch * (gamma + 1))
        if rand.dtype not in (torch.int32, torch.uint32):
            raise ValueError("rand: expected 32-bit words")
    _dev(n_accepted, "n_accepted", torch.int32, batch)
    _dev(next_token, "next_token", torch.int32, batch)
    _dev(status, "status", torch.int32, 1, optional=True)
    _check(lib().specdec_accept_noalloc(batch, gamma, vocab, input_kind, temperature, p.data_ptr(), _ptr(q), _ptr(d),
                                        ld_d, _ptr(rand), seed, step, step_dev, n_accepted.data_ptr(),
                                        next_token.data_ptr(), _ptr(status), _stream(stream)),
           "specdec_accept_noalloc")


def specdec_kv_commit(kv: KVCache, gamma: int, role: int, n_accepted, d, ld_d: int, next_token, stream=None):
    import torch
    B = kv.batch
    _dev(n_accepted, "n_accepted", torch.int32, B)
    _dev(next_token, "next_token", torch.int32, B)
    _dev(d, "d", torch.int32, (B - 1) * ld_d + gamma, optional=role == ROLE_TARGET)
    _check(lib().specdec_kv_commit(ctypes.byref(kv.kv), gamma, role, n_accepted.data_ptr(), _ptr(d), ld_d,
                                   next_token.data_ptr(), _stream(stream)), "specdec_kv_commit")


def specdec_sample(probs, rand, seed: int, step: int, purpose: int, index: int, out, vocab=None, stream=None):
    import torch
    B, ld = probs.shape
    _dev(probs, "probs", torch.float32, B * ld)
    if rand is not None:
        _dev(rand, "rand", rand.dtype, B)
    _dev(out, "out", torch.int32, B)
    if vocab is not None and vocab > ld:
        raise ValueError("vocab > row length")
    _check(lib().specdec_sample(B, vocab or ld, probs.data_ptr(), ld, _ptr(rand), seed, step, purpose, index,
                                out.data_ptr(), _stream(stream)), "specdec_sample")


def specdec_draw_u32(batch: int, seed: int, step: int, purpose: int, index: int, out, stream=None):
    _dev(out, "out", out.dtype if out is not None else None, batch)
    if out.element_size() != 4:
        raise ValueError("out: expected 32-bit words")
    _check(lib().specdec_draw_u32(batch, seed, step, purpose, index, out.data_ptr(), _stream(stream)),
           "specdec_draw_u32")


def specdec_device_status(kv: KVCache, stream=None) -> int:
    out = ctypes.c_int32(0)
    lib().specdec_device_status(ctypes.byref(kv.kv), _stream(stream), ctypes.byref(out))
    return out.value


def specdec_stream_read(buf, sink, nbytes=None, stream=None):
    """Streaming-read ceiling probe over a device tensor (see the header)."""
    _dev(buf, "buf", None, 1)
    _dev(sink, "sink", None, 1)
    size = buf.numel() * buf.element_size()
    n = size if nbytes is None else int(nbytes)
    if not 0 <= n <= size:
        raise ValueError("nbytes: outside the buffer")
    _check(lib().specdec_stream_read(buf.data_ptr(), n, sink.data_ptr(), _stream(stream)), "specdec_stream_read")


def specdec_status_string(status: int) -> str:
    return lib().specdec_status_string(status).decode()


def specdec_timing_enable(enable: bool):
    _check(lib().specdec_timing_enable(1 if enable else 0), "specdec_timing_enable")


def specdec_time_kernel(model: "Model", kind: str, reps: int = 20, stream=None) -> float:
    """Average duration (us) of `kind` re-launched back to back, layer after layer (see the header)."""
    out = ctypes.c_double(0.0)
    _check(lib().specdec_time_kernel(model.handle, KERNEL_KINDS.index(kind), reps, _stream(stream),
                                     ctypes.byref(out)), "specdec_time_kernel")
    return out.value


def specdec_timing_read():
    """{kind: (total_ms, launches)} since the last read (synchronizes on the events)."""
    ms = np.zeros(len(KERNEL_KINDS), np.float64)
    n = np.zeros(len(KERNEL_KINDS), np.int64)
    _check(lib().specdec_timing_read(ms.ctypes.data, n.ctypes.data), "specdec_timing_read")
    return {k: (float(ms[i]), int(n[i])) for i, k in enumerate(KERNEL_KINDS)}


# ---------------------------------------------------------------- one iteration
class SpecDecoder:
    """Buffers and call sequence of one draft-and-verify iteration for a batch.

    The call order is the inner loop of the paper's runtime (Sec. 3.4, Alg. 3):
    gamma draft steps, one verify pass, accept / resample, commit of both
    caches.  Host code only sequences the calls; tokens and counts stay on
    the device.  With device_step the Philox step of every draw is the target
    cache's commit counter, read on the device (the `step` arguments below are
    then ignored), so a captured iteration draws fresh words on each replay.
    """

    def __init__(self, target: Model, draft: Model, kv_t: KVCache, kv_d: KVCache, gamma: int,
                 temperature: float, seed: int, device_step: bool = False):
        import torch
        self.target, self.draft, self.kv_t, self.kv_d = target, draft, kv_t, kv_d
        self.gamma, self.temperature, self.seed = gamma, temperature, seed
        self.step_dev = kv_t.step_word() if device_step else None
        B, V = kv_t.batch, target.shape.vocab
        dev = kv_t.data.device
        self.B, self.V = B, V
        self.d = torch.zeros((B, gamma), dtype=torch.int32, device=dev)
        self.q = torch.zeros((B, gamma, V), dtype=torch.float32, device=dev) if temperature > 0 else None
        self.logits = torch.empty((B, gamma + 1, V), dtype=torch.float32, device=dev)
        self.n_acc = torch.zeros(B, dtype=torch.int32, device=dev)
        self.next = torch.zeros(B, dtype=torch.int32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.accept_ws = accept_workspace(B, gamma, V, dev)

    def draft_phase(self, step: int, stream=None):
        for s in range(self.gamma):
            specdec_draft_step(self.draft, self.kv_d, self.gamma, s, self.temperature, self.seed, step, None, self.q,
                               self.d, self.gamma, None, stream, step_dev=self.step_dev)

    def verify_phase(self, step: int, stream=None):
        specdec_verify(self.target, self.kv_t, self.gamma, self.d, self.gamma, self.logits, stream)
        specdec_accept(self.B, self.gamma, self.V, INPUT_LOGITS, self.temperature, self.logits, self.q, self.d,
                       self.gamma, None, self.seed, step, self.n_acc, self.next, self.status, self.accept_ws, stream,
                       step_dev=self.step_dev)

    def commit_phase(self, stream=None):
        specdec_kv_commit(self.kv_t, self.gamma, ROLE_TARGET, self.n_acc, self.d, self.gamma, self.next, stream)
        specdec_kv_commit(self.kv_d, self.gamma, ROLE_DRAFT, self.n_acc, self.d, self.gamma, self.next, stream)

    def step(self, step: int, stream=None):
        self.draft_phase(step, stream)
        self.verify_phase(step, stream)
        self.commit_phase(stream)
