"""Host side of the C ABI, on the CPU: the library loads, exports every function
include/tss.h declares, and its pure host checks (config, tree, mask, tree
metadata, size queries, argument validation before any device work) behave as
documented.  No compute call is made here."""
import ctypes
import os
import re

import numpy as np
import pytest

import synth
from oracle import tree_meta as oracle_tree_meta
from paper_2609_26100_amd import tss as abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "tss.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(tss_[a-z0-9_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = abi.lib()
    declared = _declared()
    assert len(declared) >= 20
    for name in declared:
        assert hasattr(lib, name), name
    assert sorted(abi.EXPORTS) == declared


@pytest.mark.parametrize("shape", [synth.TINY, synth.LLAMA_7B, synth.LLAMA_13B, synth.LLAMA_33B])
def test_cfg_accepts_workload_shapes(shape):
    cfg = abi.make_cfg(shape)
    assert abi.tss_cfg_check(cfg) == abi.TSS_OK
    wb = abi.tss_weights_bytes(cfg)
    es = 2 if shape.dtype == "bf16" else 4
    d, f, v, L = shape.d_model, shape.ffn_dim, shape.vocab, shape.n_layers
    params = 2 * v * d + L * (4 * d * d + 3 * d * f)
    assert params * es <= wb <= params * es + (L * 6 + 3) * 256 + (2 * L + 1) * d * 4
    assert abi.tss_workspace_bytes(cfg) > 0
    kb = abi.tss_kv_bytes(cfg, 1, 1030)
    assert kb >= L * 65 * 16 * 2 * d * es


def test_7b_sizes():
    cfg = abi.make_cfg(synth.LLAMA_7B)
    assert abs(abi.tss_weights_bytes(cfg) - 13.48e9) < 0.02e9


@pytest.mark.parametrize("field,val", [("head_dim", 96), ("d_model", 4000), ("vocab", 32001), ("max_nodes", 65),
                                       ("max_nodes", 0), ("n_layers", 0), ("dtype", 7), ("rms_eps", 0.0),
                                       ("ffn_dim", 11000), ("n_layers", 257), ("max_batch", 0), ("max_batch", 9)])
def test_cfg_rejects(field, val):
    cfg = abi.make_cfg(synth.LLAMA_7B)
    setattr(cfg, field, val)
    assert abi.tss_cfg_check(cfg) == abi.TSS_EINVAL
    assert abi.tss_weights_bytes(cfg) == 0


def test_cfg_batch_capacity():
    """The workspace holds the rows of a whole batch (up to 128 bf16 / 64 fp32 rows)."""
    one = abi.make_cfg(synth.LLAMA_13B, max_nodes=9, max_batch=1)
    eight = abi.make_cfg(synth.LLAMA_13B, max_nodes=9, max_batch=8)
    assert abi.tss_cfg_check(eight) == abi.TSS_OK
    assert abi.tss_workspace_bytes(eight) > abi.tss_workspace_bytes(one)
    big = abi.make_cfg(synth.LLAMA_13B, max_nodes=64, max_batch=8)   # capped at 128 rows
    assert abi.tss_workspace_bytes(big) < 2 * abi.tss_workspace_bytes(abi.make_cfg(synth.LLAMA_13B, 64, 2))
    wide = abi.make_cfg(synth.TINY)
    wide.d_model, wide.n_heads = 8192, 128     # the fp32 mode takes d <= 4096
    assert abi.tss_cfg_check(wide) == abi.TSS_EINVAL


def test_validate_tree():
    ok = [-1, 0, 0, 1, 3]
    assert abi.tss_validate_tree(ok, 5, 64) == abi.TSS_OK
    assert abi.tss_validate_tree(None, 6, 64) == abi.TSS_OK       # chain
    for bad, n in (([0, 0], 2), ([-1, 1], 2), ([-1, 0, 2], 3), ([-1, -1], 2), ([-1, 0, 5], 3)):
        assert abi.tss_validate_tree(bad, n, 64) == abi.TSS_EINVAL, bad
    assert abi.tss_validate_tree(None, 0, 64) == abi.TSS_EINVAL
    assert abi.tss_validate_tree(None, 65, 64) == abi.TSS_EINVAL
    assert abi.tss_validate_tree(None, 7, 6) == abi.TSS_EINVAL


def test_validate_mask():
    assert abi.tss_validate_mask(np.array([0, 1, 0, 1], np.uint8), 4) == abi.TSS_OK
    assert abi.tss_validate_mask(None, 4) == abi.TSS_OK
    assert abi.tss_validate_mask(np.array([0, 2, 0, 1], np.uint8), 4) == abi.TSS_EINVAL
    assert abi.tss_validate_mask(np.zeros(300, np.uint8), 300) == abi.TSS_EINVAL


@pytest.mark.parametrize("n,stream", [(1, 0), (8, 1), (33, 2), (64, 3)])
def test_tree_meta_matches_oracle(n, stream):
    parent = synth.random_tree(n, seed=5, stream=stream)
    st, depth, anc = abi.tss_tree_meta(parent, n)
    assert st == abi.TSS_OK
    od, vis = oracle_tree_meta(parent)
    np.testing.assert_array_equal(depth, od)
    for i in range(n):
        bits = {j for j in range(n) if (int(anc[i]) >> j) & 1}
        assert bits == vis[i]


def test_tree_meta_chain_default():
    st, depth, anc = abi.tss_tree_meta(None, 64)
    assert st == abi.TSS_OK
    assert list(depth) == list(range(64))
    assert int(anc[63]) == (1 << 64) - 1


def test_create_validates_before_device_work():
    cfg = abi.make_cfg(synth.TINY)
    L = abi.lib()
    out = ctypes.c_void_p()
    # null buffers
    assert L.tss_create(ctypes.byref(cfg), None, None, 0, None, 0, ctypes.byref(out)) == abi.TSS_EINVAL
    # buffers smaller than the size queries
    assert L.tss_create(ctypes.byref(cfg), None, 0x1000, 16, 0x2000, 16, ctypes.byref(out)) == abi.TSS_ENOSPACE
    assert out.value is None
    bad = abi.make_cfg(synth.TINY)
    bad.head_dim = 32
    assert L.tss_create(ctypes.byref(bad), None, 0x1000, 1 << 40, 0x2000, 1 << 40, ctypes.byref(out)) == abi.TSS_EINVAL


def test_null_context_calls_fail_cleanly():
    L = abi.lib()
    al, nt = ctypes.c_int32(), ctypes.c_int32()
    assert L.tss_verify(None, 0, None, None, 1, None, 0, ctypes.byref(al), ctypes.byref(nt)) == abi.TSS_EINVAL
    assert L.tss_prefill(None, 0, None, 0) == abi.TSS_EINVAL
    assert L.tss_verify_batch(None, 1, None, None, None, None, None, 0, None, None) == abi.TSS_EINVAL
    assert L.tss_verify_sweep(None, 0, None, None, 1, 1, None, None, None, None, None, 0) == abi.TSS_EINVAL
    assert L.tss_get_path(None, 0, None, None) == abi.TSS_EINVAL
    assert L.tss_set_skip_mask(None, 0, None) == abi.TSS_EINVAL
    assert L.tss_load_weights(None, 0, 1, None) == abi.TSS_EINVAL
    L.tss_destroy(None)


def test_status_strings():
    for s in (abi.TSS_OK, abi.TSS_EINVAL, abi.TSS_ENOSPACE, abi.TSS_ECAPACITY, abi.TSS_ESTATE, abi.TSS_EHIP):
        assert abi.tss_status_string(s) not in ("", "unknown status")


def test_sweep_prefix_bytes():
    cfg = abi.make_cfg(synth.LLAMA_7B, 64)
    assert abi.tss_sweep_prefix_bytes(cfg, 33) == 32 * 33 * 4096 * 4
    assert abi.tss_sweep_prefix_bytes(cfg, 0) == 0
    assert abi.tss_sweep_prefix_bytes(cfg, 65) == 0


def test_static_scratch_sizes():
    """tss_verify_static serves every workload shape's single-sequence steps
    (up to 64 nodes) from the 64 MiB static scratch; the size query follows
    the single-sequence layout whatever max_batch is, and a model with a
    d 8192, 64000-token vocabulary is reported as not fitting (its partial
    states, activations and logits exceed the scratch)."""
    for shape in (synth.TINY, synth.LLAMA_7B, synth.LLAMA_13B, synth.LLAMA_33B):
        one = abi.tss_static_workspace_bytes(abi.make_cfg(shape, 64, 1))
        assert 0 < one <= abi.TSS_STATIC_SCRATCH_BYTES
        assert abi.tss_static_workspace_bytes(abi.make_cfg(shape, 64, 8)) == one
        assert abi.tss_workspace_bytes(abi.make_cfg(shape, 64, 1)) == one
    big = synth.ModelShape("d8192-v64000", 90, n_layers=1, d_model=8192, n_heads=64, head_dim=128, ffn_dim=64,
                           vocab=64000)
    assert abi.tss_static_workspace_bytes(abi.make_cfg(big, 64, 1)) > abi.TSS_STATIC_SCRATCH_BYTES
    bad = abi.make_cfg(synth.TINY)
    bad.head_dim = 96
    assert abi.tss_static_workspace_bytes(bad) == 0


def test_bf16_to_f16_every_pattern():
    """The weight conversion of the bf16 mode, on all 65536 bf16 patterns:
    the fp16 value numpy's round-to-nearest-even float32 -> float16 cast gives
    (bf16 -> float32 is exact), NaN for NaN, and the count of finite values
    beyond fp16's range equal to the patterns of magnitude >= 65536."""
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got, over = abi.tss_bf16_to_f16(bits)
    f32 = (bits.astype(np.uint32) << 16).view(np.float32)
    with np.errstate(over="ignore"):
        want = f32.astype(np.float16)
    nan = np.isnan(f32)
    g = got.view(np.float16)
    assert np.isnan(g[nan]).all()
    np.testing.assert_array_equal(got[~nan], want.view(np.uint16)[~nan])
    assert over == int((np.isfinite(f32) & (np.abs(f32) >= 65536)).sum()) == 2 * (0x7f80 - 0x4780)
    # exact where fp16 has the value: every bf16 of magnitude 2^-14 .. 65280
    a = np.abs(f32)
    exact = (a >= 2.0 ** -14) & (a <= 65280)
    np.testing.assert_array_equal(g[exact].astype(np.float32), f32[exact])
    # the subnormal range rounds to the nearest multiple of 2^-24
    sub = (a > 0) & (a < 2.0 ** -14)
    assert (np.abs(g[sub].astype(np.float64) - f32[sub]) <= 2.0 ** -25).all()
    assert abi.tss_bf16_to_f16(np.zeros(0, np.uint16))[1] == 0
