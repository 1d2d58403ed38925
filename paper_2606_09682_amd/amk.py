"""ctypes binding of libamk.so (include/amk.h): same names, argument marshalling only.

Every computation of the decode step runs in the HIP library; this module
only converts Python / torch arguments into the C structures and checks
status codes.  If the library is missing it raises: there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Mapping, Optional

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libamk.so")

# ---- constants (mirror include/amk.h) ---------------------------------------
AMK_ABI_VERSION = 5
AMK_OK = 0
AMK_ERR_INVALID_ARGUMENT = -1
AMK_ERR_UNSUPPORTED = -2
AMK_ERR_SCHEDULE_REJECTED = -3
AMK_ERR_OUT_OF_MEMORY = -4
AMK_ERR_DEVICE = -5
AMK_ERR_COOPERATIVE_UNSUPPORTED = -6
AMK_ERR_TIMEOUT = -7
AMK_ERR_BAD_STATE = -8
AMK_ERR_ABORTED = -9
AMK_ERR_NONFINITE = -10

AMK_WEIGHTS_BF16 = 0
AMK_WEIGHTS_W8A16 = 1
AMK_WEIGHTS_W4A16 = 2

AMK_SCHEDULE_SHORT, AMK_SCHEDULE_LONG, AMK_SCHEDULE_TINY = 0, 1, 2
AMK_ASSIGN_ROUND_ROBIN, AMK_ASSIGN_LPT = 0, 1
AMK_TINY_MAX = 8
AMK_OP_QKV, AMK_OP_ATTN, AMK_OP_COMBINE, AMK_OP_O, AMK_OP_GATEUP, AMK_OP_DOWN, AMK_OP_LMHEAD, AMK_OP_ARGMAX = range(1, 9)
AMK_MAX_WAITS = 4
AMK_CU_INLINE = -1
AMK_TRACE_FIELDS = 8
(AMK_TRACE_WAIT_BEGIN, AMK_TRACE_WAIT_END, AMK_TRACE_INPUT_READY, AMK_TRACE_COMPUTE_END,
 AMK_TRACE_SIGNALLED, AMK_TRACE_PUBLISHED, AMK_TRACE_CHAINED, AMK_TRACE_SATISFIED) = range(8)

(AMK_CHECK_OK, AMK_CHECK_WELL_FORMED, AMK_CHECK_CAPACITY, AMK_CHECK_WAIT_SATISFIABLE, AMK_CHECK_ALL_JOIN,
 AMK_CHECK_ACYCLIC, AMK_CHECK_QUEUE_ORDER, AMK_CHECK_RACE, AMK_CHECK_KV_ORDER, AMK_CHECK_OUTPUT,
 AMK_CHECK_INLINE) = range(11)


# ---- structures ---------------------------------------------------------------
class amk_config_t(ctypes.Structure):
    _fields_ = [("abi_version", ctypes.c_uint32), ("hidden", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("n_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("intermediate", ctypes.c_int32), ("vocab", ctypes.c_int32), ("max_seq", ctypes.c_int32),
                ("rope_theta", ctypes.c_float), ("rms_eps", ctypes.c_float), ("tied_embeddings", ctypes.c_int32),
                ("weight_format", ctypes.c_int32), ("device", ctypes.c_int32), ("group_size", ctypes.c_int32)]


class amk_linear_t(ctypes.Structure):
    _fields_ = [("w", ctypes.c_void_p), ("scale", ctypes.c_void_p)]


class amk_layer_weights_t(ctypes.Structure):
    _fields_ = [("attn_norm", ctypes.c_void_p), ("mlp_norm", ctypes.c_void_p)] + [
        (n, amk_linear_t) for n in ("q", "k", "v", "o", "gate", "up", "down")]


class amk_weights_t(ctypes.Structure):
    _fields_ = [("embed", ctypes.c_void_p), ("final_norm", ctypes.c_void_p), ("lm_head", amk_linear_t),
                ("layers", ctypes.POINTER(amk_layer_weights_t))]


class amk_tuning_t(ctypes.Structure):
    _fields_ = [("attn_splits", ctypes.c_int32), ("timeout_us", ctypes.c_int32),
                ("max_rows_per_task", ctypes.c_int32), ("trace", ctypes.c_int32), ("short_context", ctypes.c_int32),
                ("tiny_context", ctypes.c_int32), ("queue_assign", ctypes.c_int32)]


class amk_task_t(ctypes.Structure):
    _fields_ = [("op", ctypes.c_uint16), ("layer", ctypes.c_uint16), ("cu", ctypes.c_int32), ("seq", ctypes.c_int32),
                ("begin", ctypes.c_int32), ("end", ctypes.c_int32), ("aux", ctypes.c_int16),
                ("n_wait", ctypes.c_int16), ("wait_counter", ctypes.c_int32 * AMK_MAX_WAITS),
                ("wait_count", ctypes.c_int32 * AMK_MAX_WAITS), ("signal_counter", ctypes.c_int32),
                ("chain_counter", ctypes.c_int32)]


class amk_check_report_t(ctypes.Structure):
    _fields_ = [("ok", ctypes.c_int32), ("rule", ctypes.c_int32), ("task", ctypes.c_int32), ("other", ctypes.c_int32),
                ("n_tasks", ctypes.c_int32), ("n_counters", ctypes.c_int32), ("n_edges", ctypes.c_int32),
                ("message", ctypes.c_char * 256)]


class AmkError(RuntimeError):
    def __init__(self, status: int, what: str = ""):
        self.status = status
        super().__init__(f"{what}: {amk_status_string(status)} ({status})" if what else
                         f"{amk_status_string(status)} ({status})")


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libamk.so (built in-tree by paper_2606_09682_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: run `python -m paper_2606_09682_amd.build` first")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    sig = {
        "amk_create": (ctypes.c_int, [P(amk_config_t), P(amk_weights_t), P(amk_tuning_t), P(ctypes.c_void_p)]),
        "amk_decode_step": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                           ctypes.c_void_p, ctypes.c_void_p]),
        "amk_create_static": (ctypes.c_int, [P(amk_config_t), P(amk_weights_t), P(amk_tuning_t),
                                             P(ctypes.c_void_p)]),
        "amk_destroy": (ctypes.c_int, [ctypes.c_void_p]),
        "amk_kv_cache_bytes": (ctypes.c_size_t, [P(amk_config_t)]),
        "amk_next_token_ptr": (ctypes.c_void_p, [ctypes.c_void_p]),
        "amk_copy_next_token": (ctypes.c_int, [ctypes.c_void_p, P(ctypes.c_int32), ctypes.c_void_p]),
        "amk_get_status": (ctypes.c_int, [ctypes.c_void_p]),
        "amk_read_probe": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.c_void_p]),
        "amk_reset": (ctypes.c_int, [ctypes.c_void_p]),
        "amk_set_abort": (ctypes.c_int, [ctypes.c_void_p, ctypes.c_int32]),
        "amk_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "amk_schedule_size": (ctypes.c_int, [P(amk_config_t), P(amk_tuning_t), ctypes.c_int32, ctypes.c_int32,
                                             P(ctypes.c_int32), P(ctypes.c_int32)]),
        "amk_schedule_export": (ctypes.c_int, [P(amk_config_t), P(amk_tuning_t), ctypes.c_int32, ctypes.c_int32,
                                               P(amk_task_t), ctypes.c_int32, P(ctypes.c_int32), P(ctypes.c_int32)]),
        "amk_schedule_check": (ctypes.c_int, [P(amk_config_t), P(amk_tuning_t), ctypes.c_int32, P(amk_task_t),
                                              ctypes.c_int32, ctypes.c_int32, P(amk_check_report_t)]),
        "amk_check_config": (ctypes.c_int, [P(amk_config_t), ctypes.c_int32]),
        "amk_trace_copy": (ctypes.c_int, [ctypes.c_void_p, P(ctypes.c_uint64), ctypes.c_int64, P(ctypes.c_int32),
                                          P(ctypes.c_int32)]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(status: int, what: str) -> None:
    if status != AMK_OK:
        raise AmkError(status, what)


# ---- thin wrappers with the C names -------------------------------------------------
def amk_status_string(status: int) -> str:
    return load().amk_status_string(status).decode()


def amk_kv_cache_bytes(cfg: amk_config_t) -> int:
    return int(load().amk_kv_cache_bytes(ctypes.byref(cfg)))


def amk_create(cfg: amk_config_t, weights: amk_weights_t, tuning: Optional[amk_tuning_t] = None) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    _check(load().amk_create(ctypes.byref(cfg), ctypes.byref(weights), ctypes.byref(tuning) if tuning else None,
                             ctypes.byref(h)), "amk_create")
    return h


def amk_create_static(cfg: amk_config_t, weights: amk_weights_t,
                      tuning: Optional[amk_tuning_t] = None) -> ctypes.c_void_p:
    """amk_create whose device memory is the library's static array (see amk.h)."""
    h = ctypes.c_void_p()
    _check(load().amk_create_static(ctypes.byref(cfg), ctypes.byref(weights),
                                    ctypes.byref(tuning) if tuning else None, ctypes.byref(h)), "amk_create_static")
    return h


def amk_decode_step(h, token: int, pos: int, kv_cache_ptr: int, logits_ptr: int, stream: int = 0) -> None:
    _check(load().amk_decode_step(h, token, pos, kv_cache_ptr, logits_ptr, stream or None), "amk_decode_step")


def amk_destroy(h) -> None:
    _check(load().amk_destroy(h), "amk_destroy")


def amk_next_token_ptr(h) -> int:
    return int(load().amk_next_token_ptr(h) or 0)


def amk_copy_next_token(h, stream: int = 0) -> int:
    v = ctypes.c_int32(-1)
    _check(load().amk_copy_next_token(h, ctypes.byref(v), stream or None), "amk_copy_next_token")
    return int(v.value)


def amk_get_status(h) -> int:
    return int(load().amk_get_status(h))


def amk_read_probe(buf_ptr: int, nbytes: int, blocks: int, sink_ptr: int, stream: int) -> None:
    """Enqueue one streaming read of nbytes at device address buf_ptr (see amk.h)."""
    _check(load().amk_read_probe(buf_ptr, nbytes, blocks, sink_ptr, stream), "amk_read_probe")


def amk_reset(h) -> None:
    _check(load().amk_reset(h), "amk_reset")


def amk_set_abort(h, value: int) -> None:
    _check(load().amk_set_abort(h, int(value)), "amk_set_abort")


def amk_trace_copy(h, n_tasks: int):
    """(variant, per-task timestamps) of the last step: a list of
    AMK_TRACE_FIELDS-tuples in the order of that variant's export."""
    buf = (ctypes.c_uint64 * (n_tasks * AMK_TRACE_FIELDS))()
    n, v = ctypes.c_int32(), ctypes.c_int32()
    _check(load().amk_trace_copy(h, buf, len(buf), ctypes.byref(n), ctypes.byref(v)), "amk_trace_copy")
    return v.value, [tuple(buf[i * AMK_TRACE_FIELDS:(i + 1) * AMK_TRACE_FIELDS]) for i in range(n.value)]


def amk_check_config(cfg: amk_config_t, n_cu: int) -> int:
    return int(load().amk_check_config(ctypes.byref(cfg), n_cu))


def amk_schedule_export(cfg: amk_config_t, n_cu: int, tuning: Optional[amk_tuning_t] = None,
                        variant: int = AMK_SCHEDULE_LONG):
    """Returns (tasks array, n_counters) of the lowering of cfg onto n_cu queues."""
    lib = load()
    nt, nc = ctypes.c_int32(), ctypes.c_int32()
    tp = ctypes.byref(tuning) if tuning else None
    _check(lib.amk_schedule_size(ctypes.byref(cfg), tp, n_cu, variant, ctypes.byref(nt), ctypes.byref(nc)),
           "amk_schedule_size")
    arr = (amk_task_t * nt.value)()
    _check(lib.amk_schedule_export(ctypes.byref(cfg), tp, n_cu, variant, arr, nt.value, ctypes.byref(nt),
                                   ctypes.byref(nc)), "amk_schedule_export")
    return arr, nc.value


def amk_schedule_check(cfg: amk_config_t, n_cu: int, tasks, n_counters: int,
                       tuning: Optional[amk_tuning_t] = None) -> amk_check_report_t:
    rep = amk_check_report_t()
    _check(load().amk_schedule_check(ctypes.byref(cfg), ctypes.byref(tuning) if tuning else None, n_cu, tasks,
                                     len(tasks), n_counters, ctypes.byref(rep)), "amk_schedule_check")
    return rep


# ---- convenience: a decoder over torch device tensors ---------------------------------
def make_config(hidden: int, n_layers: int, n_heads: int, n_kv_heads: int, head_dim: int, intermediate: int,
                vocab: int, max_seq: int, rope_theta: float, rms_eps: float = 1e-5, tied_embeddings: bool = False,
                weight_format: str = "bf16", device: int = -1, group_size: int = 0) -> amk_config_t:
    fmt = {"bf16": AMK_WEIGHTS_BF16, "w8a16": AMK_WEIGHTS_W8A16, "w4a16": AMK_WEIGHTS_W4A16}[weight_format]
    return amk_config_t(AMK_ABI_VERSION, hidden, n_layers, n_heads, n_kv_heads, head_dim, intermediate, vocab,
                        max_seq, rope_theta, rms_eps, int(tied_embeddings), fmt, device, group_size)


_PROJ = (("q", "wq"), ("k", "wk"), ("v", "wv"), ("o", "wo"), ("gate", "wg"), ("up", "wu"), ("down", "wd"))


def expected_sizes(cfg: amk_config_t) -> Dict[str, int]:
    """Bytes every weight tensor must have for cfg.  The library receives bare
    pointers and reads these extents; a smaller tensor would be read past its
    end on the device, so the binding checks them before amk_create."""
    H, I, V = cfg.hidden, cfg.intermediate, cfg.vocab
    qd, kd = cfg.n_heads * cfg.head_dim, cfg.n_kv_heads * cfg.head_dim
    shapes = {"wq": (qd, H), "wk": (kd, H), "wv": (kd, H), "wo": (H, qd), "wg": (I, H), "wu": (I, H), "wd": (H, I)}
    group = cfg.group_size or 128

    def lin(out, inp):
        if cfg.weight_format == AMK_WEIGHTS_W8A16:
            return out * inp, 4 * out
        if cfg.weight_format == AMK_WEIGHTS_W4A16:
            return out * inp // 2, 2 * out * (inp // group)
        return 2 * out * inp, 0

    sizes = {"embed": 2 * V * H, "final_norm": 2 * H}
    names = [(f"layers.{l}.{n}", shapes[n]) for l in range(cfg.n_layers) for n in shapes]
    if not cfg.tied_embeddings:
        names.append(("lm_head", (V, H)))
    for l in range(cfg.n_layers):
        sizes[f"layers.{l}.attn_norm"] = sizes[f"layers.{l}.mlp_norm"] = 2 * H
    for name, (out, inp) in names:
        w, sc = lin(out, inp)
        sizes[name] = w
        if sc:
            sizes[name + ".scale"] = sc
    return sizes


def check_sizes(cfg: amk_config_t, tensors: Mapping[str, "object"]) -> None:
    """Raise ValueError unless every tensor amk_create will read is present with
    exactly the bytes cfg implies (device and layout are checked at create)."""
    for name, nbytes in expected_sizes(cfg).items():
        if name not in tensors:
            raise ValueError(f"missing tensor {name}")
        t = tensors[name]
        have = t.numel() * t.element_size()
        if have != nbytes:
            raise ValueError(f"{name} has {have} bytes, the config needs {nbytes}")


class Decoder:
    """One handle over weights that live in torch device tensors.

    ``tensors`` maps names to contiguous device tensors: 'embed' [V,H],
    'final_norm' [H], 'lm_head' [V,H] (untied), and per layer l
    'layers.{l}.attn_norm', 'layers.{l}.mlp_norm' (bf16 [H]) and the
    projections 'layers.{l}.w{q,k,v,o,g,u,d}' [out,in] -- bf16 (any 2-byte
    dtype holding bf16 bits) or, for W8A16, int8 with an fp32 scale tensor
    under the same name + '.scale', or, for W4A16, packed uint8 [out, in/2]
    with an fp16 [out, in/group] scale tensor under name + '.scale'.  The
    tensors are borrowed: they must
    outlive the decoder, which keeps references to them.  ``static=True``
    creates the handle with amk_create_static (no device allocation)."""

    def __init__(self, cfg: amk_config_t, tensors: Mapping[str, "object"], tuning: Optional[amk_tuning_t] = None,
                 static: bool = False):
        self.cfg = cfg
        check_sizes(cfg, tensors)
        self._keep: Dict[str, object] = dict(tensors)
        quant = cfg.weight_format in (AMK_WEIGHTS_W8A16, AMK_WEIGHTS_W4A16)
        fmt_name = "W8A16" if cfg.weight_format == AMK_WEIGHTS_W8A16 else "W4A16"
        scale_size = 4 if cfg.weight_format == AMK_WEIGHTS_W8A16 else 2

        def ptr(name):
            t = tensors[name]
            if not t.is_cuda or not t.is_contiguous():
                raise ValueError(f"{name} must be a contiguous device tensor")
            return t.data_ptr()

        def lin(name, quantized):
            if quantized:
                if tensors[name].element_size() != 1:
                    raise ValueError(f"{name} must be 1-byte elements under {fmt_name}")
                if tensors[name + ".scale"].element_size() != scale_size:
                    raise ValueError(f"{name}.scale must have {scale_size}-byte elements under {fmt_name}")
                return amk_linear_t(ptr(name), ptr(name + ".scale"))
            if tensors[name].element_size() != 2:
                raise ValueError(f"{name} must hold bf16 values")
            return amk_linear_t(ptr(name), None)

        L = cfg.n_layers
        self._layers = (amk_layer_weights_t * L)()
        for l in range(L):
            p = f"layers.{l}."
            lw = self._layers[l]
            lw.attn_norm = ptr(p + "attn_norm")
            lw.mlp_norm = ptr(p + "mlp_norm")
            for field, name in _PROJ:
                setattr(lw, field, lin(p + name, quant))
        lm = amk_linear_t(None, None) if cfg.tied_embeddings else lin("lm_head", quant)
        self._weights = amk_weights_t(ptr("embed"), ptr("final_norm"), lm, self._layers)
        import torch
        # the device amk_create resolved (-1 = the current device at creation)
        self._dev = cfg.device if cfg.device >= 0 else torch.cuda.current_device()
        self.handle = (amk_create_static if static else amk_create)(cfg, self._weights, tuning)

    def kv_cache_bytes(self) -> int:
        return amk_kv_cache_bytes(self.cfg)

    def step(self, token: int, pos: int, kv_cache, logits, stream: Optional[int] = None) -> None:
        """Enqueue one decode step; kv_cache / logits are contiguous device
        tensors of at least amk_kv_cache_bytes and 4 * vocab bytes."""
        if not hasattr(self, "_need"):
            self._need = (amk_kv_cache_bytes(self.cfg), 4 * self.cfg.vocab)
        dev = self._dev
        for t, need, what in ((kv_cache, self._need[0], "kv_cache"), (logits, self._need[1], "logits")):
            if not t.is_cuda or t.device.index != dev:
                raise ValueError(f"{what} must be a tensor on cuda:{dev}, the decoder's device")
            if not t.is_contiguous() or t.numel() * t.element_size() < need:
                raise ValueError(f"{what} must be contiguous with at least {need} bytes")
        if stream is None:
            import torch
            stream = torch.cuda.current_stream().cuda_stream
        amk_decode_step(self.handle, token, pos, kv_cache.data_ptr(), logits.data_ptr(), stream)

    def next_token(self, stream: Optional[int] = None) -> int:
        if stream is None:
            import torch
            stream = torch.cuda.current_stream().cuda_stream
        return amk_copy_next_token(self.handle, stream)

    def status(self) -> int:
        return amk_get_status(self.handle)

    def reset(self) -> None:
        amk_reset(self.handle)

    def set_abort(self, value: int) -> None:
        amk_set_abort(self.handle, value)

    def close(self) -> None:
        if getattr(self, "handle", None):
            amk_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
