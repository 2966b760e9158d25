"""A verify session: the device buffers one instance needs (weights, KV pool,
workspace, outputs) and the flattening of per-sample trees into the C ABI's
arrays.  Marshalling only; the computation is the library's."""

from __future__ import annotations

import numpy as np
import torch

from . import binding as B


def flatten_trees(trees):
    """[(tokens, parents), ...] -> (tree_offsets, tokens, parents) int32 arrays."""
    sizes = [len(t[0]) for t in trees]
    offsets = np.zeros(len(trees) + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(sizes)
    tokens = np.fromiter((int(x) for t in trees for x in t[0]), dtype=np.int32, count=offsets[-1])
    parents = np.fromiter((int(x) for t in trees for x in t[1]), dtype=np.int32, count=offsets[-1])
    return offsets, tokens, parents


class Verifier:
    def __init__(self, cfg, W, capacity, max_batch, max_tokens, device="cuda", sampling=False):
        """sampling=True sizes the workspace for verify_sampled at temperature > 0."""
        self.cfg = cfg
        self.weights = B.Weights(W)
        self.kv = B.KVPool(cfg, capacity, device=device)
        nbytes = (B.spec_workspace_bytes_sampled if sampling else B.spec_workspace_bytes)(
            cfg, max_batch, max_tokens)
        if nbytes == 0:
            raise B.SpecError(-1, "invalid workspace request")
        self.workspace = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.max_batch, self.max_tokens = max_batch, max_tokens
        self.accepted_len = torch.empty(max_batch, dtype=torch.int32, device=device)
        self.next_token = torch.empty(max_batch, dtype=torch.int32, device=device)
        self.accepted_nodes = torch.empty(max_batch, B.SPEC_MAX_TREE, dtype=torch.int32,
                                          device=device)
        self.new_seq_lens = torch.empty(max_batch, dtype=torch.int32, device=device)

    def debug_buffers(self, n_tokens, logits=True):
        dev = self.workspace.device
        d = {"argmax": torch.empty(n_tokens, dtype=torch.int32, device=dev),
             "depth": torch.empty(n_tokens, dtype=torch.int32, device=dev),
             "pos": torch.empty(n_tokens, dtype=torch.int32, device=dev),
             "anc": torch.empty(n_tokens, B.SPEC_ANC_WORDS, dtype=torch.int64, device=dev)}
        if logits:
            d["logits"] = torch.empty(n_tokens, self.cfg.vocab, dtype=torch.float32, device=dev)
        return d

    def verify(self, sample_ids, trees, seq_lens, debug=None, stream=None, flat=None):
        """Enqueue one verify step; returns views of the device outputs."""
        offsets, tokens, parents = flat if flat is not None else flatten_trees(trees)
        b = len(sample_ids)
        B.spec_verify(self.cfg, self.weights, self.kv, sample_ids, offsets, tokens, parents,
                      seq_lens, self.workspace, self.accepted_len, self.next_token,
                      self.accepted_nodes, debug=debug, stream=stream)
        return self.accepted_len[:b], self.next_token[:b], self.accepted_nodes[:b]

    def verify_noalloc(self, sample_ids, trees, seq_lens, debug=None, stream=None, flat=None):
        """verify() on the library's static device scratch instead of this
        session's workspace (spec_verify_noalloc)."""
        offsets, tokens, parents = flat if flat is not None else flatten_trees(trees)
        b = len(sample_ids)
        B.spec_verify_noalloc(self.cfg, self.weights, self.kv, sample_ids, offsets, tokens,
                              parents, seq_lens, self.accepted_len, self.next_token,
                              self.accepted_nodes, debug=debug, stream=stream)
        return self.accepted_len[:b], self.next_token[:b], self.accepted_nodes[:b]

    def verify_sampled(self, sample_ids, trees, seq_lens, temperature, eos_token=-1,
                       draft_probs=None, uniforms=None, debug=None, stream=None, flat=None):
        """Enqueue one verify step with speculative-sampling acceptance."""
        offsets, tokens, parents = flat if flat is not None else flatten_trees(trees)
        b = len(sample_ids)
        B.spec_verify_sampled(self.cfg, self.weights, self.kv, sample_ids, offsets, tokens, parents,
                              seq_lens, self.workspace, self.accepted_len, self.next_token,
                              self.accepted_nodes, temperature, eos_token, draft_probs, uniforms,
                              debug=debug, stream=stream)
        return self.accepted_len[:b], self.next_token[:b], self.accepted_nodes[:b]

    def commit(self, sample_ids, seq_lens, stream=None):
        b = len(sample_ids)
        B.spec_kv_commit(self.kv, sample_ids, seq_lens, self.accepted_len, self.accepted_nodes,
                         self.new_seq_lens, stream=stream)
        return self.new_seq_lens[:b]
