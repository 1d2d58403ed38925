"""The C ABI library loads, exports every function include/amk.h declares, and
its ctypes mirror agrees with the header's layouts and constants (no GPU)."""
import ctypes
import os
import re
import subprocess

import pytest

import synth
from paper_2606_09682_amd import amk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "amk.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(amk.LIB_PATH):
        from paper_2606_09682_amd import build
        build.build()
    return amk.load()


def _declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(amk_\w+)\s*\(", text, re.M)))


def test_every_declared_symbol_is_exported(lib):
    names = _declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", amk.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (amk_\w+)", out))
    assert set(names) <= exported


def _c_layout():
    """Compile a C program against amk.h that prints sizes, offsets and enum values."""
    src = r'''
#include <stdio.h>
#include <stddef.h>
#include "amk.h"
#define S(t) printf("sizeof %s %zu\n", #t, sizeof(t));
#define O(t, f) printf("offsetof %s.%s %zu\n", #t, #f, offsetof(t, f));
#define E(v) printf("enum %s %d\n", #v, (int)(v));
int main(void) {
  S(amk_config_t) S(amk_linear_t) S(amk_layer_weights_t) S(amk_weights_t) S(amk_tuning_t) S(amk_task_t)
  S(amk_check_report_t)
  O(amk_config_t, rope_theta) O(amk_config_t, device) O(amk_config_t, group_size) O(amk_layer_weights_t, down)
  O(amk_weights_t, layers)
  O(amk_tuning_t, trace) O(amk_tuning_t, short_context) O(amk_tuning_t, tiny_context) O(amk_tuning_t, queue_assign)
  O(amk_task_t, aux) O(amk_task_t, n_wait) O(amk_task_t, wait_counter) O(amk_task_t, wait_count)
  O(amk_task_t, signal_counter) O(amk_task_t, chain_counter) O(amk_check_report_t, message)
  E(AMK_ABI_VERSION) E(AMK_OK) E(AMK_ERR_INVALID_ARGUMENT) E(AMK_ERR_UNSUPPORTED) E(AMK_ERR_SCHEDULE_REJECTED)
  E(AMK_ERR_OUT_OF_MEMORY) E(AMK_ERR_DEVICE) E(AMK_ERR_COOPERATIVE_UNSUPPORTED) E(AMK_ERR_TIMEOUT)
  E(AMK_ERR_BAD_STATE) E(AMK_ERR_ABORTED) E(AMK_ERR_NONFINITE) E(AMK_WEIGHTS_BF16) E(AMK_WEIGHTS_W8A16) E(AMK_WEIGHTS_W4A16)
  E(AMK_MAX_WAITS)
  E(AMK_OP_QKV) E(AMK_OP_ATTN) E(AMK_OP_COMBINE) E(AMK_OP_O) E(AMK_OP_GATEUP) E(AMK_OP_DOWN) E(AMK_OP_LMHEAD)
  E(AMK_OP_ARGMAX) E(AMK_CHECK_OK) E(AMK_CHECK_WELL_FORMED) E(AMK_CHECK_CAPACITY) E(AMK_CHECK_WAIT_SATISFIABLE)
  E(AMK_CHECK_ALL_JOIN) E(AMK_CHECK_ACYCLIC) E(AMK_CHECK_QUEUE_ORDER) E(AMK_CHECK_RACE) E(AMK_CHECK_KV_ORDER)
  E(AMK_CHECK_OUTPUT) E(AMK_CHECK_INLINE) E(AMK_CU_INLINE) E(AMK_TRACE_FIELDS) E(AMK_TRACE_WAIT_BEGIN) E(AMK_TRACE_WAIT_END) E(AMK_TRACE_INPUT_READY)
  E(AMK_TRACE_COMPUTE_END) E(AMK_TRACE_SIGNALLED) E(AMK_TRACE_PUBLISHED)
  E(AMK_TRACE_CHAINED) E(AMK_TRACE_SATISFIED) E(AMK_SCHEDULE_SHORT) E(AMK_SCHEDULE_LONG)
  E(AMK_SCHEDULE_TINY) E(AMK_TINY_MAX) E(AMK_ASSIGN_ROUND_ROBIN) E(AMK_ASSIGN_LPT)
  return 0;
}
'''
    import tempfile
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "layout.c")
        exe = os.path.join(d, "layout")
        open(c, "w").write(src)
        subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), c, "-o", exe],
                       check=True)
        out = subprocess.run([exe], capture_output=True, text=True, check=True).stdout
    res = {}
    for line in out.splitlines():
        kind, name, val = line.split()
        res[(kind, name)] = int(val)
    return res


def test_ctypes_mirror_matches_header():
    c = _c_layout()
    for t in ("amk_config_t", "amk_linear_t", "amk_layer_weights_t", "amk_weights_t", "amk_tuning_t", "amk_task_t",
              "amk_check_report_t"):
        assert ctypes.sizeof(getattr(amk, t)) == c[("sizeof", t)], t
    assert c[("sizeof", "amk_task_t")] == 64
    for key, val in c.items():
        kind, name = key
        if kind == "offsetof":
            t, f = name.split(".")
            assert getattr(getattr(amk, t), f).offset == val, name
        elif kind == "enum":
            assert getattr(amk, name) == val, name


def test_status_strings(lib):
    for code in range(0, -11, -1):
        assert amk.amk_status_string(code) not in ("", "unknown status")
    assert amk.amk_status_string(-99) == "unknown status"


def _cfg(name, fmt="bf16", **over):
    c = synth.get(name)
    kw = dict(hidden=c.hidden, n_layers=c.n_layers, n_heads=c.n_heads, n_kv_heads=c.n_kv_heads,
              head_dim=c.head_dim, intermediate=c.intermediate, vocab=c.vocab, max_seq=c.seq_capacity,
              rope_theta=c.rope_theta, rms_eps=c.rms_eps, tied_embeddings=c.tied_embeddings, weight_format=fmt)
    kw.update(over)
    return amk.make_config(**kw)


@pytest.mark.parametrize("name", list(synth.CONFIGS))
def test_kv_cache_bytes(lib, name):
    c = synth.get(name)
    want = c.n_layers * 2 * c.n_kv_heads * c.seq_capacity * c.head_dim * 2
    assert amk.amk_kv_cache_bytes(_cfg(name)) == want


@pytest.mark.parametrize("name", list(synth.CONFIGS))
@pytest.mark.parametrize("n_cu", [256, 80, 7, 1])
@pytest.mark.parametrize("fmt", ["bf16", "w8a16", "w4a16"])
def test_every_workload_schedule_is_accepted(lib, name, n_cu, fmt):
    c = synth.get(name)
    if fmt == "w4a16" and c.intermediate % 32:
        # int4 rows must be whole 16-byte vectors of 32 columns (tiny: SwiGLU 688)
        assert amk.amk_check_config(_cfg(name, fmt, group_size=32), n_cu) == amk.AMK_ERR_UNSUPPORTED
        return
    over = dict(group_size=c.int4_group) if fmt == "w4a16" else {}
    assert amk.amk_check_config(_cfg(name, fmt, **over), n_cu) == amk.AMK_OK


@pytest.mark.parametrize("over,status", [
    (dict(n_kv_heads=3), amk.AMK_ERR_UNSUPPORTED),            # 4 heads not a multiple of 3 KV heads
    (dict(head_dim=96), amk.AMK_ERR_UNSUPPORTED),             # not a power of two
    (dict(head_dim=32), amk.AMK_ERR_UNSUPPORTED),             # below the attention tiling minimum
    (dict(hidden=200), amk.AMK_ERR_UNSUPPORTED),              # rows not whole 16-byte vectors
    (dict(intermediate=690), amk.AMK_ERR_UNSUPPORTED),
    (dict(n_heads=32, n_kv_heads=2), amk.AMK_ERR_UNSUPPORTED),# group of 16 heads
    (dict(vocab=0), amk.AMK_ERR_INVALID_ARGUMENT),
    (dict(weight_format=7), amk.AMK_ERR_INVALID_ARGUMENT),
])
def test_unsupported_configs_are_rejected(lib, over, status):
    cfg = _cfg("tiny")
    for k, v in over.items():
        setattr(cfg, k, v)
    assert amk.amk_check_config(cfg, 256) == status


@pytest.mark.parametrize("over,status", [
    (dict(group_size=48), amk.AMK_ERR_INVALID_ARGUMENT),    # not a power of two
    (dict(group_size=16), amk.AMK_ERR_INVALID_ARGUMENT),    # below one lane's 32 columns
    (dict(group_size=2048), amk.AMK_ERR_INVALID_ARGUMENT),  # above the largest group
    (dict(group_size=512), amk.AMK_ERR_UNSUPPORTED),        # does not divide hidden 256
    (dict(intermediate=688, group_size=32), amk.AMK_ERR_UNSUPPORTED),  # 688 not a multiple of 32
    (dict(group_size=0), amk.AMK_OK),                       # default 128
    (dict(group_size=256), amk.AMK_OK),
])
def test_w4a16_config_rules(lib, over, status):
    cfg = _cfg("tiny", "w4a16", intermediate=768)
    for k, v in over.items():
        setattr(cfg, k, v)
    assert amk.amk_check_config(cfg, 256) == status


def test_bad_abi_version_rejected(lib):
    cfg = _cfg("tiny")
    cfg.abi_version = 99
    assert amk.amk_check_config(cfg, 256) == amk.AMK_ERR_INVALID_ARGUMENT


def test_null_arguments_fail_cleanly(lib):
    h = ctypes.c_void_p()
    assert lib.amk_create(None, None, None, ctypes.byref(h)) == amk.AMK_ERR_INVALID_ARGUMENT
    assert h.value is None
    assert lib.amk_create(None, None, None, None) == amk.AMK_ERR_INVALID_ARGUMENT
    assert lib.amk_decode_step(None, 0, 0, None, None, None) == amk.AMK_ERR_INVALID_ARGUMENT
    assert lib.amk_get_status(None) == amk.AMK_ERR_INVALID_ARGUMENT
    assert lib.amk_reset(None) == amk.AMK_ERR_INVALID_ARGUMENT
    assert lib.amk_destroy(None) == amk.AMK_OK
    assert amk.amk_kv_cache_bytes(amk.amk_config_t()) == 0


def test_kernels_use_no_scratch(lib):
    """Every decode-kernel instantiation keeps its state in registers: no
    scratch memory and no spilled VGPRs (the build records the compiler's
    resource-usage remarks)."""
    from paper_2606_09682_amd import build
    if not os.path.exists(build.RESOURCES):
        build.build()
    rows = [line.split() for line in open(build.RESOURCES) if "amk_decode_kernel" in line]
    # head_dim {64, 128} x group {4, 8} x {bf16, W8A16, W4A16} x {tiny schedule, the others}
    assert len(rows) == 24
    for name, *kv in rows:
        fields = dict(x.split("=") for x in kv)
        assert fields["scratch"] == "0" and fields["vgpr_spill"] == "0", (name, fields)
        assert int(fields["vgprs"]) <= 256, (name, fields)


def test_read_probe_rejects_bad_arguments(lib):
    # validated on the host before any device call
    dummy = ctypes.c_void_p(4096)
    for nbytes, blocks, buf in ((15, 4, dummy), (0, 4, dummy), (1024, 0, dummy), (1024, 70000, dummy),
                                (1024, 4, ctypes.c_void_p(4104)), (1024, 4, None)):
        assert lib.amk_read_probe(buf, nbytes, blocks, dummy, None) == amk.AMK_ERR_INVALID_ARGUMENT
    assert lib.amk_read_probe(dummy, 1024, 4, None, None) == amk.AMK_ERR_INVALID_ARGUMENT


@pytest.mark.parametrize("fmt", ["bf16", "w8a16", "w4a16"])
def test_binding_checks_tensor_sizes(fmt):
    """The binding refuses weight tensors whose byte size differs from what the
    config implies (the library itself only sees pointers); checked before any
    device call, so CPU tensors do."""
    import torch
    shape = synth.get("tiny").with_(intermediate=768) if fmt == "w4a16" else synth.get("tiny")
    w = synth.make_weights(shape, seed=0)
    if fmt == "w8a16":
        synth.add_w8a16(w)
    if fmt == "w4a16":
        synth.add_w4a16(w, group=64)
    from synth.device import config_kwargs, weights_to_device
    cfg = amk.make_config(**config_kwargs(shape, fmt, 8, 64 if fmt == "w4a16" else 0))
    tensors = weights_to_device(w, fmt, device="cpu")
    amk.check_sizes(cfg, tensors)  # the synthetic tensors fit exactly
    for victim in ("layers.1.wd", "embed", "layers.0.mlp_norm") + (("layers.2.wk.scale",) if fmt != "bf16" else ()):
        bad = dict(tensors)
        bad[victim] = tensors[victim].flatten()[:-1]
        with pytest.raises(ValueError, match=victim):
            amk.check_sizes(cfg, bad)
    bad = dict(tensors)
    del bad["layers.3.wu"]
    with pytest.raises(ValueError, match="missing"):
        amk.check_sizes(cfg, bad)
    if fmt == "w4a16":  # scales for a different group size have a different extent
        with pytest.raises(ValueError, match="scale"):
            amk.check_sizes(amk.make_config(**config_kwargs(shape, fmt, 8, 128)), tensors)
