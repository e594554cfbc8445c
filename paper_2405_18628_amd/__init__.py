"""Python binding of libppd, the MI355X (gfx950) PPD tree-verification step.

Argument marshalling only: every step of the computation runs in the HIP
kernels of libppd.so.  Functions carry the names of the C ABI (include/ppd.h);
tensors are torch tensors used as device memory, streams are torch streams.
Importing works without a GPU (the host-side tree builder and the argument
checks run anywhere); device calls need the built library and a GPU, and
fail loudly otherwise -- there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# PPD_LIBRARY selects another build of the same library (the host-sanitizer
# build that the CPU tests load); by default the one next to this file
LIB_PATH = os.environ.get("PPD_LIBRARY") or os.path.join(_HERE, "libppd.so")

PPD_OK, PPD_EINVAL, PPD_ETREE, PPD_ECAPACITY, PPD_EDEVICE, PPD_EUNSUPPORTED, PPD_EWORKSPACE = range(7)
PPD_F32, PPD_BF16 = 0, 1
PPD_T_MAX = 128
PPD_MASK_WORDS = 2
PPD_DEV_BAD_TOKEN, PPD_DEV_BAD_PARENT, PPD_DEV_NAN_LOGIT = 1, 2, 4
PPD_W_QKV, PPD_W_O, PPD_W_GATE_UP, PPD_W_DOWN, PPD_W_LM_HEAD = range(5)

_STATUS_NAMES = {0: "PPD_OK", 1: "PPD_EINVAL", 2: "PPD_ETREE", 3: "PPD_ECAPACITY",
                 4: "PPD_EDEVICE", 5: "PPD_EUNSUPPORTED", 6: "PPD_EWORKSPACE"}


class PPDError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class ppd_model(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_heads", C.c_int32),
                ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32), ("ffn", C.c_int32),
                ("vocab", C.c_int32), ("n_prompt", C.c_int32), ("rms_eps", C.c_float),
                ("rope_base", C.c_float), ("dtype", C.c_int32),
                ("tok_emb", C.c_void_p), ("prompt_emb", C.c_void_p),
                ("attn_norm", C.POINTER(C.c_void_p)), ("w_qkv", C.POINTER(C.c_void_p)),
                ("w_o", C.POINTER(C.c_void_p)), ("mlp_norm", C.POINTER(C.c_void_p)),
                ("w_gate_up", C.POINTER(C.c_void_p)), ("w_down", C.POINTER(C.c_void_p)),
                ("final_norm", C.c_void_p), ("lm_head", C.c_void_p)]


class ppd_kv(C.Structure):
    _fields_ = [("k", C.c_void_p), ("v", C.c_void_p), ("capacity", C.c_int32),
                ("len_dev", C.c_void_p)]


_lib = None


def lib() -> C.CDLL:
    """The loaded libppd.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: run paper_2405_18628_amd.build.build()")
        L = C.CDLL(LIB_PATH)
        vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
        P = C.POINTER
        L.ppd_workspace_bytes.argtypes = [P(ppd_model), i32, i32]
        L.ppd_workspace_bytes.restype = sz
        L.ppd_workspace_init.argtypes = [vp, sz, vp]
        L.ppd_build_tree_mask.argtypes = [i32, vp, vp, vp]
        L.ppd_verify_step.argtypes = [P(ppd_model), P(ppd_kv), i32, i32, vp, vp, vp, vp, sz, vp,
                                      vp, vp]
        L.ppd_verify_batch.argtypes = [P(ppd_model), i32, vp, vp, vp, vp, vp, vp, vp, sz, vp, vp,
                                       vp]
        L.ppd_verify_step_static.argtypes = [P(ppd_model), P(ppd_kv), i32, i32, vp, vp, vp, vp, vp,
                                             vp, vp]
        L.ppd_accept.argtypes = [i32, vp, vp, vp, i32, vp, vp, vp, vp, sz, vp]
        L.ppd_kv_compact.argtypes = [P(ppd_model), P(ppd_kv), i32, vp, i32, vp, vp]
        L.ppd_device_status.argtypes = [vp, sz, P(C.c_uint32), i32, vp]
        L.ppd_set_kernel_timer.argtypes = [i32, vp, vp, i32]
        L.ppd_last_error.restype = C.c_char_p
        L.ppd_next_tree.argtypes = [i32, vp, vp, i32, i32, i32, vp, vp, vp, vp, i32, vp, vp, vp, vp,
                                    sz, vp]
        L.ppd_sparse_template.argtypes = [vp, i32, i32, i32, i32, i32, vp, vp, P(C.c_int32),
                                          P(C.c_double)]
        L.ppd_packed_weight_bytes.argtypes = [i32, i32, i32]
        L.ppd_packed_weight_bytes.restype = sz
        L.ppd_pack_weight.argtypes = [i32, i32, i32, vp, vp, vp]
        L.ppd_read_probe.argtypes = [vp, sz, vp, vp]
        for f in ("ppd_verify_step_static", "ppd_next_tree", "ppd_sparse_template", "ppd_verify_batch", "ppd_pack_weight", "ppd_workspace_init", "ppd_build_tree_mask", "ppd_verify_step", "ppd_accept",
                  "ppd_kv_compact", "ppd_device_status", "ppd_set_kernel_timer", "ppd_read_probe"):
            getattr(L, f).restype = C.c_int
        _lib = L
    return _lib


def ppd_last_error() -> str:
    return lib().ppd_last_error().decode()


def _check(status: int):
    if status != PPD_OK:
        raise PPDError(status, ppd_last_error())


def _ptr(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def _dev(t, dtype=None, name="tensor"):
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")


# ---------------------------------------------------------------------------


class Model:
    """A ppd_model description over device tensors (kept alive by this object).

    `w` follows the row-major layout of include/ppd.h (see
    synth.model.make_weights).  For bf16 models the five projection matrices
    are packed once here (ppd_pack_weight) and the description points at the
    packed copies; `w` itself is left unchanged."""

    _PACKED = {"w_qkv": PPD_W_QKV, "w_o": PPD_W_O, "w_gate_up": PPD_W_GATE_UP,
               "w_down": PPD_W_DOWN}

    def __init__(self, shape, w, stream=None):
        import torch
        dt = torch.bfloat16 if shape.dtype == "bf16" else torch.float32
        self.shape = shape
        self.w = w
        layers = w["layers"]
        n = shape.n_layers
        bf16 = shape.dtype == "bf16"
        self.packed = {k: [] for k in self._PACKED}

        def arr(key):
            ptrs = []
            for lay in layers:
                _dev(lay[key], dt, key)
                if bf16 and key in self._PACKED:
                    pk = ppd_pack_weight(self._PACKED[key], lay[key], stream)
                    self.packed[key].append(pk)
                    ptrs.append(_ptr(pk))
                else:
                    ptrs.append(_ptr(lay[key]))
            return (C.c_void_p * n)(*ptrs)

        for key in ("tok_emb", "prompt_emb", "final_norm", "lm_head"):
            _dev(w[key], dt, key)
        self._arrays = {k: arr(k) for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up",
                                            "w_down")}
        self.lm_head = ppd_pack_weight(PPD_W_LM_HEAD, w["lm_head"], stream) if bf16 else w["lm_head"]
        a = self._arrays
        self.desc = ppd_model(
            shape.n_layers, shape.hidden, shape.n_heads, shape.n_kv_heads, shape.head_dim,
            shape.ffn, shape.vocab, shape.n_prompt, shape.rms_eps, shape.rope_base,
            PPD_BF16 if bf16 else PPD_F32,
            _ptr(w["tok_emb"]), _ptr(w["prompt_emb"]),
            C.cast(a["attn_norm"], C.POINTER(C.c_void_p)), C.cast(a["w_qkv"], C.POINTER(C.c_void_p)),
            C.cast(a["w_o"], C.POINTER(C.c_void_p)), C.cast(a["mlp_norm"], C.POINTER(C.c_void_p)),
            C.cast(a["w_gate_up"], C.POINTER(C.c_void_p)), C.cast(a["w_down"], C.POINTER(C.c_void_p)),
            _ptr(w["final_norm"]), _ptr(self.lm_head))


    def first_layers(self, n: int) -> "Model":
        """The same model cut to its first n decoder layers (final norm and
        LM head unchanged), sharing this object's packed weights: no copy."""
        import copy
        if not 1 <= n <= self.shape.n_layers:
            raise ValueError(f"n={n} outside [1, {self.shape.n_layers}]")
        m = copy.copy(self)
        m.shape = self.shape.with_layers(n)
        m.desc = ppd_model.from_buffer_copy(self.desc)
        m.desc.n_layers = n
        m._parent = self
        return m


class KVCache:
    """K [layers][kv_heads][capacity][head_dim], V [layers][kv_heads][head_dim][capacity]."""

    def __init__(self, k, v, len_dev=None):
        self.k, self.v, self.len_dev = k, v, len_dev
        self.capacity = int(k.shape[2])
        self.desc = ppd_kv(_ptr(k), _ptr(v), self.capacity, _ptr(len_dev) or None)


# ---------------------------------------------------------------------------
# the C ABI, one Python function per entry point


def ppd_workspace_bytes(model: Model, t_max: int, max_len: int) -> int:
    n = lib().ppd_workspace_bytes(C.byref(model.desc), t_max, max_len)
    if n == 0:
        raise PPDError(PPD_EINVAL, ppd_last_error())
    return int(n)


def ppd_packed_weight_bytes(kind: int, rows: int, cols: int) -> int:
    n = lib().ppd_packed_weight_bytes(int(kind), int(rows), int(cols))
    if n == 0:
        raise PPDError(PPD_EINVAL, ppd_last_error())
    return int(n)


def ppd_pack_weight(kind: int, src, stream=None):
    """Packed copy (a new uint8 device tensor) of the row-major bf16 matrix
    `src` [rows][cols], in the layout the bf16 GEMMs read."""
    import torch
    _dev(src, torch.bfloat16, "weight")
    rows, cols = (int(x) for x in src.shape)
    dst = torch.empty(ppd_packed_weight_bytes(kind, rows, cols), dtype=torch.uint8,
                      device=src.device)
    _check(lib().ppd_pack_weight(int(kind), rows, cols, _ptr(src), _ptr(dst), _stream(stream)))
    return dst


def ppd_workspace_init(ws, stream=None):
    _dev(ws, None, "ws")
    _check(lib().ppd_workspace_init(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def ppd_build_tree_mask(parent: Sequence[int]):
    """Host: (depth int32[T], mask uint64[T][2]) of a topological parent array."""
    p = np.ascontiguousarray(np.asarray(parent, dtype=np.int32))
    T = int(p.shape[0])
    depth = np.zeros(T, np.int32)
    mask = np.zeros((T, PPD_MASK_WORDS), np.uint64)
    _check(lib().ppd_build_tree_mask(T, p.ctypes.data, depth.ctypes.data, mask.ctypes.data))
    return depth, mask


def ppd_verify_step(model: Model, kv: KVCache, L: int, T: int, ids, depth, mask, ws, logits,
                    pred, stream=None):
    import torch
    for t, n in ((ids, "ids"), (depth, "depth"), (pred, "pred")):
        _dev(t, torch.int32, n)
    _dev(mask, None, "mask")
    _dev(ws, None, "ws")
    _dev(logits, torch.float32, "logits")
    _check(lib().ppd_verify_step(C.byref(model.desc), C.byref(kv.desc), int(L), int(T), _ptr(ids),
                                 _ptr(depth), _ptr(mask), _ptr(ws),
                                 ws.numel() * ws.element_size(), _ptr(logits) or None,
                                 _ptr(pred), _stream(stream)))


def ppd_verify_step_static(model: Model, kv: KVCache, L: int, T: int, ids, depth, mask, logits,
                           pred, status_out=None, stream=None):
    """ppd_verify_step with the library's static workspace (no allocation)."""
    import torch
    for t, n in ((ids, "ids"), (depth, "depth"), (pred, "pred")):
        _dev(t, torch.int32, n)
    _dev(mask, None, "mask")
    _dev(logits, torch.float32, "logits")
    _dev(status_out, torch.int32, "status_out")
    _check(lib().ppd_verify_step_static(C.byref(model.desc), C.byref(kv.desc), int(L), int(T),
                                        _ptr(ids), _ptr(depth), _ptr(mask), _ptr(logits) or None,
                                        _ptr(pred), _ptr(status_out) or None, _stream(stream)))


def ppd_verify_batch(model: Model, kvs: Sequence[KVCache], L: Sequence[int], T: Sequence[int],
                     ids, depth, mask, ws, logits, pred, stream=None):
    """One step over len(kvs) sequences whose trees are packed in sequence
    order (device ids / depth / mask / logits / pred rows)."""
    import torch
    for t, n in ((ids, "ids"), (depth, "depth"), (pred, "pred")):
        _dev(t, torch.int32, n)
    _dev(mask, None, "mask")
    _dev(ws, None, "ws")
    _dev(logits, torch.float32, "logits")
    B = len(kvs)
    if len(L) != B or len(T) != B:
        raise ValueError("kvs, L and T differ in length")
    descs = (ppd_kv * max(B, 1))(*[kv.desc for kv in kvs])
    Ls = np.ascontiguousarray(np.asarray(L, dtype=np.int32))
    Ts = np.ascontiguousarray(np.asarray(T, dtype=np.int32))
    _check(lib().ppd_verify_batch(C.byref(model.desc), B, C.cast(descs, C.c_void_p),
                                  Ls.ctypes.data, Ts.ctypes.data, _ptr(ids), _ptr(depth),
                                  _ptr(mask), _ptr(ws), ws.numel() * ws.element_size(),
                                  _ptr(logits) or None, _ptr(pred), _stream(stream)))


def ppd_accept(T: int, parent, ids, pred, vocab: int, path, n_path, next_tok, ws, stream=None):
    import torch
    for t, n in ((parent, "parent"), (ids, "ids"), (pred, "pred"), (path, "path"),
                 (n_path, "n_path"), (next_tok, "next_tok")):
        _dev(t, torch.int32, n)
    _check(lib().ppd_accept(int(T), _ptr(parent), _ptr(ids), _ptr(pred), int(vocab), _ptr(path),
                            _ptr(n_path), _ptr(next_tok), _ptr(ws), ws.numel() * ws.element_size(),
                            _stream(stream)))


def ppd_next_tree(T: int, parent, ids, vocab: int, n_prompt: int, logits, path, n_path,
                  next_tok, tpl_parent: Sequence[int], tpl_kind: Sequence[int], next_ids, ws,
                  stream=None, n_ept: int = 1):
    """Token ids of the next step's tree (template tpl_parent / tpl_kind, host
    sequences) into the device tensor next_ids."""
    import torch
    for t, n in ((parent, "parent"), (ids, "ids"), (path, "path"), (n_path, "n_path"),
                 (next_tok, "next_tok"), (next_ids, "next_ids")):
        _dev(t, torch.int32, n)
    _dev(logits, torch.float32, "logits")
    tp = np.ascontiguousarray(np.asarray(tpl_parent, dtype=np.int32))
    tk = np.ascontiguousarray(np.asarray(tpl_kind, dtype=np.int32))
    if tp.shape != tk.shape:
        raise ValueError("tpl_parent and tpl_kind differ in length")
    _check(lib().ppd_next_tree(int(T), _ptr(parent), _ptr(ids), int(vocab), int(n_prompt),
                               int(n_ept), _ptr(logits), _ptr(path), _ptr(n_path), _ptr(next_tok),
                               int(tp.shape[0]), tp.ctypes.data, tk.ctypes.data, _ptr(next_ids),
                               _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def ppd_sparse_template(p_table, n_cand: int, n_prompt: int, n_ept: int = 1):
    """Template of the n_cand candidates that maximise Proposition 1's expected
    accepted length under the host table p_table[depth - 1][rank].  Returns
    (tpl_parent, tpl_kind, expected accepted candidates)."""
    p = np.ascontiguousarray(np.asarray(p_table, dtype=np.float64))
    if p.ndim != 2:
        raise ValueError("p_table must be 2-D [depth][rank]")
    par = np.zeros(PPD_T_MAX, np.int32)
    kind = np.zeros(PPD_T_MAX, np.int32)
    T = C.c_int32(0)
    f = C.c_double(0.0)
    _check(lib().ppd_sparse_template(p.ctypes.data, p.shape[0], p.shape[1], int(n_cand),
                                     int(n_prompt), int(n_ept), par.ctypes.data, kind.ctypes.data,
                                     C.byref(T), C.byref(f)))
    return par[:T.value].copy(), kind[:T.value].copy(), float(f.value)


def ppd_kv_compact(model: Model, kv: KVCache, L: int, path, n_path, stream=None,
                   path_len: Optional[int] = None):
    """path: device int32 tensor (its length is passed as path_len unless
    given); n_path: device int32 count, clamped on the device."""
    import torch
    _dev(path, torch.int32, "path")
    _dev(n_path, torch.int32, "n_path")
    n = int(path.numel()) if path_len is None else int(path_len)
    _check(lib().ppd_kv_compact(C.byref(model.desc), C.byref(kv.desc), int(L), _ptr(path), n,
                                _ptr(n_path), _stream(stream)))


def ppd_device_status(ws, clear: bool = False, stream=None) -> int:
    out = C.c_uint32(0)
    _check(lib().ppd_device_status(_ptr(ws), ws.numel() * ws.element_size(), C.byref(out),
                                   int(bool(clear)), _stream(stream)))
    return int(out.value)


def ppd_read_probe(buf, sink, stream=None):
    """One read of the whole device tensor buf by the HBM read probe; the XOR
    of what it read lands in the device uint32 tensor sink."""
    _dev(buf, None, "buf")
    _dev(sink, None, "sink")
    _check(lib().ppd_read_probe(_ptr(buf), buf.numel() * buf.element_size(), _ptr(sink), _stream(stream)))


KERNEL_KINDS = {"qkv": 0, "attention": 1, "o_proj": 2, "gate_up": 3, "down": 4, "lm_head": 5,
                "next_tree": 6}


def ppd_set_kernel_timer(kind, start_events=(), stop_events=()):
    """Record HIP events around every launch of one kernel kind in later
    ppd_verify_step calls of this thread (torch.cuda.Event objects);
    call with no events to disable.  Returns the ctypes arrays (keep them)."""
    n = len(start_events)
    if n == 0:
        _check(lib().ppd_set_kernel_timer(0, None, None, 0))
        return None
    k = KERNEL_KINDS.get(kind, kind)
    for e in list(start_events) + list(stop_events):
        if not e.cuda_event:      # torch creates the HIP event on first record
            e.record()
    st = (C.c_void_p * n)(*[e.cuda_event for e in start_events])
    sp = (C.c_void_p * n)(*[e.cuda_event for e in stop_events])
    _check(lib().ppd_set_kernel_timer(int(k), st, sp, n))
    return st, sp


__all__ = ["ppd_verify_step_static", "ppd_verify_batch", "ppd_next_tree", "ppd_sparse_template", "ppd_packed_weight_bytes", "ppd_pack_weight", "ppd_set_kernel_timer", "Model", "KVCache", "PPDError", "lib", "ppd_workspace_bytes", "ppd_workspace_init",
           "ppd_build_tree_mask", "ppd_verify_step", "ppd_accept", "ppd_kv_compact",
           "ppd_device_status", "ppd_last_error", "ppd_read_probe"]
