"""Python binding of the C ABI in include/tss.h (ctypes; argument marshalling only).

Every function here has the name of the C function it calls and does no
computation of its own: all work of the verify step runs in libtss.so's HIP
kernels.  Loading fails loudly when the library has not been built; there is
no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtss.so")

TSS_OK, TSS_EINVAL, TSS_ENOSPACE, TSS_ECAPACITY, TSS_ESTATE, TSS_EHIP = 0, -1, -2, -3, -4, -5
TSS_F32, TSS_BF16 = 0, 1
TSS_COMMIT = 1
TSS_LAUNCH_DIRECT, TSS_LAUNCH_GRAPH = 0, 1
(TSS_K_EMBED, TSS_K_QKV, TSS_K_ATTN, TSS_K_OPROJ, TSS_K_GATEUP, TSS_K_DOWN, TSS_K_LMHEAD, TSS_K_ACCEPT,
 TSS_K_COMPACT) = range(9)

# every function include/tss.h declares
EXPORTS = (
    "tss_cfg_check", "tss_weights_bytes", "tss_workspace_bytes", "tss_kv_bytes", "tss_create",
    "tss_load_weights", "tss_kv_alloc", "tss_set_skip_mask", "tss_prefill", "tss_verify", "tss_get_logits",
    "tss_verify_batch", "tss_verify_sweep", "tss_sweep_prefix_bytes", "tss_get_greedy", "tss_get_path", "tss_seq_length", "tss_seq_truncate", "tss_validate_tree", "tss_validate_mask",
    "tss_tree_meta", "tss_set_launch_mode", "tss_profile_kernel", "tss_profile_read", "tss_last_error", "tss_status_string",
    "tss_destroy", "tss_get_logits_device", "tss_get_attn_split", "tss_check_kv", "tss_verify_static",
    "tss_static_workspace_bytes", "tss_bf16_to_f16",
)

TSS_STATIC_SCRATCH_BYTES = 64 << 20


class tss_model_cfg(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32), ("vocab", ctypes.c_int32),
        ("rope_base", ctypes.c_float), ("rms_eps", ctypes.c_float), ("dtype", ctypes.c_int32),
        ("max_nodes", ctypes.c_int32), ("max_batch", ctypes.c_int32),
    ]


class TSSError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{msg} (status {status})")
        self.status = status


_lib = None


def lib():
    """The loaded libtss.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with python -m paper_2609_26100_amd.build")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, U32, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint32, ctypes.c_size_t
        CFG = ctypes.POINTER(tss_model_cfg)
        sig = {
            "tss_cfg_check": (ctypes.c_int, [CFG]),
            "tss_weights_bytes": (SZ, [CFG]),
            "tss_workspace_bytes": (SZ, [CFG]),
            "tss_kv_bytes": (SZ, [CFG, I32, I32]),
            "tss_create": (ctypes.c_int, [CFG, P, P, SZ, P, SZ, ctypes.POINTER(P)]),
            "tss_load_weights": (ctypes.c_int, [P, I32, I32, ctypes.POINTER(P)]),
            "tss_kv_alloc": (ctypes.c_int, [P, I32, I32, P, SZ, P]),
            "tss_set_skip_mask": (ctypes.c_int, [P, I32, P]),
            "tss_prefill": (ctypes.c_int, [P, I32, P, I32]),
            "tss_verify": (ctypes.c_int, [P, I32, P, P, I32, P, U32, ctypes.POINTER(I32), ctypes.POINTER(I32)]),
            "tss_verify_batch": (ctypes.c_int, [P, I32, P, P, P, P, P, U32, P, P]),
            "tss_verify_sweep": (ctypes.c_int, [P, I32, P, P, I32, I32, P, P, P, P, P, SZ]),
            "tss_sweep_prefix_bytes": (SZ, [CFG, I32]),
            "tss_get_logits": (ctypes.c_int, [P, P, I32]),
            "tss_get_greedy": (ctypes.c_int, [P, P, I32]),
            "tss_get_logits_device": (ctypes.c_int, [P, P, I32]),
            "tss_get_attn_split": (ctypes.c_int, [P, ctypes.POINTER(I32), P, P]),
            "tss_check_kv": (ctypes.c_int, [P]),
            "tss_verify_static": (ctypes.c_int, [P, I32, P, P, I32, P, U32, ctypes.POINTER(I32),
                                                 ctypes.POINTER(I32)]),
            "tss_static_workspace_bytes": (SZ, [CFG]),
            "tss_bf16_to_f16": (ctypes.c_int64, [P, P, ctypes.c_int64]),
            "tss_get_path": (ctypes.c_int, [P, I32, P, ctypes.POINTER(I32)]),
            "tss_seq_length": (ctypes.c_int, [P, I32, ctypes.POINTER(I32)]),
            "tss_seq_truncate": (ctypes.c_int, [P, I32, I32]),
            "tss_validate_tree": (ctypes.c_int, [P, I32, I32]),
            "tss_validate_mask": (ctypes.c_int, [P, I32]),
            "tss_tree_meta": (ctypes.c_int, [P, I32, P, P]),
            "tss_set_launch_mode": (ctypes.c_int, [P, I32]),
            "tss_profile_kernel": (ctypes.c_int, [P, I32, I32]),
            "tss_profile_read": (ctypes.c_int, [P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_int64), I32]),
            "tss_last_error": (ctypes.c_char_p, [P]),
            "tss_status_string": (ctypes.c_char_p, [ctypes.c_int]),
            "tss_destroy": (None, [P]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _ptr(a):
    """Host pointer of a contiguous numpy array (or None)."""
    if a is None:
        return None
    if not a.flags["C_CONTIGUOUS"]:
        raise ValueError("array must be C-contiguous")
    return a.ctypes.data


def _check(status, ctx=None, what=""):
    if status != TSS_OK:
        msg = tss_last_error(ctx) if ctx else tss_status_string(status)
        raise TSSError(status, f"{what}: {msg}")


def make_cfg(shape, max_nodes=64, max_batch=1) -> tss_model_cfg:
    return tss_model_cfg(shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.ffn_dim, shape.vocab,
                         shape.rope_base, shape.rms_eps, TSS_BF16 if shape.dtype == "bf16" else TSS_F32, max_nodes,
                         max_batch)


def tss_cfg_check(cfg) -> int:
    return lib().tss_cfg_check(ctypes.byref(cfg))


def tss_weights_bytes(cfg) -> int:
    return lib().tss_weights_bytes(ctypes.byref(cfg))


def tss_workspace_bytes(cfg) -> int:
    return lib().tss_workspace_bytes(ctypes.byref(cfg))


def tss_kv_bytes(cfg, n_seqs, max_tokens_per_seq) -> int:
    return lib().tss_kv_bytes(ctypes.byref(cfg), n_seqs, max_tokens_per_seq)


def tss_create(cfg, hip_stream, dev_weights, weights_bytes, dev_workspace, workspace_bytes):
    out = ctypes.c_void_p()
    st = lib().tss_create(ctypes.byref(cfg), hip_stream, dev_weights, weights_bytes, dev_workspace, workspace_bytes,
                          ctypes.byref(out))
    if st != TSS_OK:
        raise TSSError(st, f"tss_create: {lib().tss_last_error(None).decode()}")
    return out.value


def tss_load_weights(ctx, first, host_arrays):
    arrs = [np.ascontiguousarray(a) for a in host_arrays]
    ptrs = (ctypes.c_void_p * len(arrs))(*[a.ctypes.data for a in arrs])
    _check(lib().tss_load_weights(ctx, first, len(arrs), ptrs), ctx, "tss_load_weights")


def tss_kv_alloc(ctx, n_seqs, max_tokens_per_seq, dev_pool, pool_bytes, page_order=None):
    po = None if page_order is None else np.ascontiguousarray(page_order, dtype=np.int32)
    _check(lib().tss_kv_alloc(ctx, n_seqs, max_tokens_per_seq, dev_pool, pool_bytes, _ptr(po)), ctx, "tss_kv_alloc")


def tss_set_skip_mask(ctx, seq, mask):
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    _check(lib().tss_set_skip_mask(ctx, seq, _ptr(m)), ctx, "tss_set_skip_mask")


def tss_prefill(ctx, seq, tokens):
    t = np.ascontiguousarray(tokens, dtype=np.int32)
    _check(lib().tss_prefill(ctx, seq, _ptr(t), len(t)), ctx, "tss_prefill")


def tss_verify(ctx, seq, draft_tokens, tree_parent=None, skip_mask=None, flags=0):
    """Returns (accept_len, next_token)."""
    t = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    p = None if tree_parent is None else np.ascontiguousarray(tree_parent, dtype=np.int32)
    m = None if skip_mask is None else np.ascontiguousarray(skip_mask, dtype=np.uint8)
    al, nt = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().tss_verify(ctx, seq, _ptr(t), _ptr(p), len(t), _ptr(m), flags, ctypes.byref(al), ctypes.byref(nt)),
           ctx, "tss_verify")
    return al.value, nt.value


def tss_verify_static(ctx, seq, draft_tokens, tree_parent=None, skip_mask=None, flags=0):
    """tss_verify with the step's workspace in the library's static device scratch (allocates nothing).
    Returns (accept_len, next_token)."""
    t = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    p = None if tree_parent is None else np.ascontiguousarray(tree_parent, dtype=np.int32)
    m = None if skip_mask is None else np.ascontiguousarray(skip_mask, dtype=np.uint8)
    al, nt = ctypes.c_int32(), ctypes.c_int32()
    _check(lib().tss_verify_static(ctx, seq, _ptr(t), _ptr(p), len(t), _ptr(m), flags, ctypes.byref(al),
                                   ctypes.byref(nt)), ctx, "tss_verify_static")
    return al.value, nt.value


def tss_static_workspace_bytes(cfg) -> int:
    return lib().tss_static_workspace_bytes(ctypes.byref(cfg))


def tss_bf16_to_f16(bits):
    """bf16 bit patterns (uint16) -> (fp16 bit patterns, count beyond fp16's range)."""
    src = np.ascontiguousarray(bits, dtype=np.uint16)
    dst = np.empty_like(src)
    over = lib().tss_bf16_to_f16(src.ctypes.data, dst.ctypes.data, src.size)
    if over < 0:
        raise TSSError(TSS_EINVAL, "tss_bf16_to_f16 refused its arguments")
    return dst, int(over)


def tss_verify_batch(ctx, seq_ids, draft_tokens, node_offsets, tree_parents=None, skip_masks=None, flags=0):
    """Returns (accept_len[n_seqs], next_token[n_seqs])."""
    ids = np.ascontiguousarray(seq_ids, dtype=np.int32)
    offs = np.ascontiguousarray(node_offsets, dtype=np.int32)
    t = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    p = None if tree_parents is None else np.ascontiguousarray(tree_parents, dtype=np.int32)
    m = None if skip_masks is None else np.ascontiguousarray(skip_masks, dtype=np.uint8)
    n = len(ids)
    if len(offs) != n + 1 or (p is not None and len(p) != len(t)) or (m is not None and m.size % max(n, 1)):
        raise ValueError("seq_ids, node_offsets, tree_parents and skip_masks do not describe one batch")
    if len(offs) and offs[-1] != len(t):
        raise ValueError("node_offsets[-1] must equal the number of draft tokens")
    al = np.zeros(n, dtype=np.int32)
    nt = np.zeros(n, dtype=np.int32)
    _check(lib().tss_verify_batch(ctx, n, _ptr(ids), _ptr(offs), _ptr(t), _ptr(p), _ptr(m), flags, _ptr(al), _ptr(nt)),
           ctx, "tss_verify_batch")
    return al, nt


def tss_sweep_prefix_bytes(cfg, n_nodes) -> int:
    return lib().tss_sweep_prefix_bytes(ctypes.byref(cfg), n_nodes)


def tss_verify_sweep(ctx, seq, draft_tokens, tree_parent, skip_masks, want_greedy=False, dev_prefix=None,
                     prefix_bytes=0):
    """Dry-run verifies of one draft tree under each row of skip_masks
    [n_masks][n_layers]; returns (accept_len[n_masks], next_token[n_masks]) and,
    with want_greedy, greedy[n_masks][n_nodes].  dev_prefix: device pointer of
    a prefix buffer (tss_sweep_prefix_bytes) or None."""
    t = np.ascontiguousarray(draft_tokens, dtype=np.int32)
    p = None if tree_parent is None else np.ascontiguousarray(tree_parent, dtype=np.int32)
    m = np.ascontiguousarray(skip_masks, dtype=np.uint8)
    if m.ndim != 2 or (p is not None and len(p) != len(t)):
        raise ValueError("skip_masks must be [n_masks][n_layers] and tree_parent as long as draft_tokens")
    k = m.shape[0]
    al = np.zeros(k, dtype=np.int32)
    nt = np.zeros(k, dtype=np.int32)
    g = np.zeros((k, len(t)), dtype=np.int32) if want_greedy else None
    _check(lib().tss_verify_sweep(ctx, seq, _ptr(t), _ptr(p), len(t), k, _ptr(m), _ptr(al), _ptr(nt), _ptr(g),
                                  dev_prefix, prefix_bytes), ctx, "tss_verify_sweep")
    return (al, nt, g) if want_greedy else (al, nt)


def tss_get_logits(ctx, n_nodes, vocab):
    out = np.empty((n_nodes, vocab), dtype=np.float32)
    _check(lib().tss_get_logits(ctx, _ptr(out), n_nodes), ctx, "tss_get_logits")
    return out


def tss_get_logits_device(ctx, dev_dst, n_nodes):
    """Enqueues a copy of the last verify's logits into device memory at dev_dst (an address)."""
    _check(lib().tss_get_logits_device(ctx, dev_dst, n_nodes), ctx, "tss_get_logits_device")


def tss_get_attn_split(ctx):
    """[(groups, rows)] per attention item of the last step's last attention launch."""
    n = ctypes.c_int32()
    groups = np.zeros(16, dtype=np.int32)
    rows = np.zeros(16, dtype=np.int32)
    _check(lib().tss_get_attn_split(ctx, ctypes.byref(n), _ptr(groups), _ptr(rows)), ctx, "tss_get_attn_split")
    return [(int(groups[i]), int(rows[i])) for i in range(n.value)]


def tss_check_kv(ctx):
    _check(lib().tss_check_kv(ctx), ctx, "tss_check_kv")


def tss_get_greedy(ctx, n_nodes):
    out = np.empty(n_nodes, dtype=np.int32)
    _check(lib().tss_get_greedy(ctx, _ptr(out), n_nodes), ctx, "tss_get_greedy")
    return out


def tss_get_path(ctx, index=0, max_nodes=64):
    """Local node ids of result `index`'s accepted path (root first)."""
    out = np.zeros(max_nodes, dtype=np.int32)
    n = ctypes.c_int32()
    _check(lib().tss_get_path(ctx, index, _ptr(out), ctypes.byref(n)), ctx, "tss_get_path")
    return out[: n.value].copy()


def tss_seq_length(ctx, seq) -> int:
    n = ctypes.c_int32()
    _check(lib().tss_seq_length(ctx, seq, ctypes.byref(n)), ctx, "tss_seq_length")
    return n.value


def tss_seq_truncate(ctx, seq, n_kv):
    _check(lib().tss_seq_truncate(ctx, seq, n_kv), ctx, "tss_seq_truncate")


def tss_validate_tree(parent, n_nodes, max_nodes) -> int:
    p = None if parent is None else np.ascontiguousarray(parent, dtype=np.int32)
    return lib().tss_validate_tree(_ptr(p), n_nodes, max_nodes)


def tss_validate_mask(mask, n_layers) -> int:
    m = None if mask is None else np.ascontiguousarray(mask, dtype=np.uint8)
    return lib().tss_validate_mask(_ptr(m), n_layers)


def tss_tree_meta(parent, n_nodes):
    p = None if parent is None else np.ascontiguousarray(parent, dtype=np.int32)
    depth = np.zeros(n_nodes, dtype=np.int32)
    anc = np.zeros(n_nodes, dtype=np.uint64)
    st = lib().tss_tree_meta(_ptr(p), n_nodes, _ptr(depth), _ptr(anc))
    return st, depth, anc


def tss_set_launch_mode(ctx, mode):
    _check(lib().tss_set_launch_mode(ctx, mode), ctx, "tss_set_launch_mode")


def tss_profile_kernel(ctx, kernel, layer=-1):
    _check(lib().tss_profile_kernel(ctx, kernel, layer), ctx, "tss_profile_kernel")


def tss_profile_read(ctx, reset=False):
    """Returns (total_ms, count) of the profiled launches' own execution time."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    _check(lib().tss_profile_read(ctx, ctypes.byref(ms), ctypes.byref(n), int(reset)), ctx, "tss_profile_read")
    return ms.value, n.value


def tss_last_error(ctx) -> str:
    r = lib().tss_last_error(ctx)
    return r.decode() if r else ""


def tss_status_string(status) -> str:
    return lib().tss_status_string(status).decode()


def tss_destroy(ctx):
    lib().tss_destroy(ctx)
