"""A TSS verifier bound to torch-owned device buffers.

PyTorch only provides the device memory (packed weights, workspace, KV pool)
and the HIP stream; every step of the verify path runs in libtss.so.
"""
from __future__ import annotations

import numpy as np

from . import tss as abi


class Verifier:
    def __init__(self, shape, n_seqs=1, max_tokens=2048, max_nodes=64, device="cuda:0", stream=None,
                 page_order=None, max_batch=1):
        import torch

        self.torch = torch
        self.shape = shape
        self.device = torch.device(device)
        self.cfg = abi.make_cfg(shape, max_nodes, max_batch)
        if abi.tss_cfg_check(self.cfg) != abi.TSS_OK:
            raise ValueError(f"unsupported shape {shape}")
        self.stream = stream if stream is not None else torch.cuda.current_stream(self.device)
        wb = abi.tss_weights_bytes(self.cfg)
        sb = abi.tss_workspace_bytes(self.cfg)
        kb = abi.tss_kv_bytes(self.cfg, n_seqs, max_tokens)
        self.weights = torch.empty(wb, dtype=torch.uint8, device=self.device)
        self.workspace = torch.zeros(sb, dtype=torch.uint8, device=self.device)
        self.kv_pool = torch.zeros(kb, dtype=torch.uint8, device=self.device)
        torch.cuda.synchronize(self.device)
        self.ctx = abi.tss_create(self.cfg, self.stream.cuda_stream, self.weights.data_ptr(), wb,
                                  self.workspace.data_ptr(), sb)
        abi.tss_kv_alloc(self.ctx, n_seqs, max_tokens, self.kv_pool.data_ptr(), kb, page_order)
        self.n_seqs, self.max_tokens = n_seqs, max_tokens
        self._mask = {i: np.zeros(shape.n_layers, np.uint8) for i in range(n_seqs)}
        self.prefix = None  # device buffer of the mask sweep's shared prefix

    def bind_kv(self, n_seqs, max_tokens, page_order=None):
        """Binds a new KV pool (a new device buffer) and resets every sequence to length 0 with a dense
        mask.  Returns the previous pool's tensor: the library no longer touches it."""
        kb = abi.tss_kv_bytes(self.cfg, n_seqs, max_tokens)
        old = self.kv_pool
        self.kv_pool = self.torch.zeros(kb, dtype=self.torch.uint8, device=self.device)
        self.torch.cuda.synchronize(self.device)
        abi.tss_kv_alloc(self.ctx, n_seqs, max_tokens, self.kv_pool.data_ptr(), kb, page_order)
        self.n_seqs, self.max_tokens = n_seqs, max_tokens
        self._mask = {i: np.zeros(self.shape.n_layers, np.uint8) for i in range(n_seqs)}
        return old

    def load(self, get_tensor):
        """Streams every tensor, in the ABI's tensor order, from get_tensor(index) -> host array in the
        shape's dtype (fp32, or bf16 bit patterns as uint16)."""
        for idx in range(3 + 9 * self.shape.n_layers):
            abi.tss_load_weights(self.ctx, idx, [get_tensor(idx)])

    def set_launch_mode(self, mode):
        abi.tss_set_launch_mode(self.ctx, mode)

    def set_mask(self, seq, mask):
        abi.tss_set_skip_mask(self.ctx, seq, mask)
        L = self.shape.n_layers
        self._mask[seq] = np.zeros(L, np.uint8) if mask is None else np.asarray(mask, dtype=np.uint8).copy()

    def prefill(self, seq, tokens):
        abi.tss_prefill(self.ctx, seq, tokens)

    def verify(self, seq, tokens, parent=None, mask=None, commit=False):
        return abi.tss_verify(self.ctx, seq, tokens, parent, mask, abi.TSS_COMMIT if commit else 0)

    def verify_batch(self, seqs, drafts, parents=None, masks=None, commit=False):
        """drafts: one token array per sequence (root first); parents: None or one parent array (or None for
        a chain) per sequence; masks: None or one mask (or None for the sequence's own) per sequence.
        Returns (accept_len[n], next_token[n])."""
        offs = np.concatenate([[0], np.cumsum([len(t) for t in drafts])]).astype(np.int32)
        tokens = np.concatenate([np.asarray(t, dtype=np.int32) for t in drafts])
        par = None
        if parents is not None and any(p is not None for p in parents):
            par = np.concatenate([np.arange(-1, len(t) - 1, dtype=np.int32) if p is None else np.asarray(p, np.int32)
                                  for t, p in zip(drafts, parents)])
        m = None
        if masks is not None:
            L = self.shape.n_layers
            rows = []
            for sq, mk in zip(seqs, masks):
                rows.append(self._mask[sq] if mk is None else np.asarray(mk, dtype=np.uint8))
            m = np.concatenate(rows).astype(np.uint8)
            assert m.size == L * len(seqs)
        return abi.tss_verify_batch(self.ctx, seqs, tokens, offs, par, m, abi.TSS_COMMIT if commit else 0)

    def verify_sweep(self, seq, tokens, masks, parent=None, want_greedy=False, reuse_prefix=True):
        """Dry runs of one draft tree under each mask (rows of masks); returns
        (accept_len[k], next_token[k]) and, with want_greedy, greedy[k][n].
        With reuse_prefix the masks share the dense prefix through a device
        buffer owned by this verifier (allocated on first use)."""
        m = np.asarray(masks, dtype=np.uint8).reshape(-1, self.shape.n_layers)
        ptr, nbytes = None, 0
        if reuse_prefix:
            nbytes = abi.tss_sweep_prefix_bytes(self.cfg, self.cfg.max_nodes)
            if self.prefix is None:
                self.prefix = self.torch.empty(nbytes, dtype=self.torch.uint8, device=self.device)
            ptr = self.prefix.data_ptr()
        return abi.tss_verify_sweep(self.ctx, seq, tokens, parent, m, want_greedy, ptr, nbytes)

    def logits(self, n_nodes):
        return abi.tss_get_logits(self.ctx, n_nodes, self.shape.vocab)

    def logits_device(self, n_nodes):
        """The last verify's logits copied into a new torch device tensor [n_nodes][vocab] on the verifier's stream."""
        out = self.torch.empty((n_nodes, self.shape.vocab), dtype=self.torch.float32, device=self.device)
        abi.tss_get_logits_device(self.ctx, out.data_ptr(), n_nodes)
        return out

    def check_kv(self):
        """Raises if the KV binding is inconsistent (page table, lengths)."""
        abi.tss_check_kv(self.ctx)

    def attn_split(self):
        """[(workgroups per head, rows)] per attention item of the last step's last attention launch."""
        return abi.tss_get_attn_split(self.ctx)

    def greedy(self, n_nodes):
        return abi.tss_get_greedy(self.ctx, n_nodes)

    def path(self, index=0):
        """Accepted path (local node ids, root first) of result `index` of the last verify."""
        return abi.tss_get_path(self.ctx, index, self.cfg.max_nodes)

    def length(self, seq):
        return abi.tss_seq_length(self.ctx, seq)

    def truncate(self, seq, n):
        abi.tss_seq_truncate(self.ctx, seq, n)

    def close(self):
        if self.ctx:
            abi.tss_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
