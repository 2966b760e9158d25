"""Oracle for the KV transfer buffer of sample migration.

TEST INFRASTRUCTURE ONLY.  The plain statement of what packing and
unpacking a migration buffer compute; only the test suite may import it.
The product path never does, and shares no code with it.

Paper, Section 6.2 ("Two-stage Sample Migration"): a migration first copies
the K/V of the migrating samples out of the cache store into one
pre-allocated contiguous buffer (phase 1), so that the transfer between
instances is a single copy (phase 2), and the receiving instance parses the
buffer and appends the K/V to its own store (phase 3).  The buffer is
organised by model, then layer, then sample.  Verified K/V never changes
after it is verified (the Markov property of verification), so the transfer
can move any token range of a sample; stage 1 moves the verified prefix and
stage 2 the tokens verified while stage 1 ran.

Reading taken where the paper is silent:
* within a layer, K precedes V; within a sample's part, the KV heads follow
  each other and each holds its tokens in order, head_dim values per token
  (the order of the cache itself);
* the library holds one model (the target LLM); the draft model's part of
  the hierarchy is empty.

A sample's cache is given as two tensors ``k``, ``v`` of shape
[layers, kv_heads, capacity, head_dim] (any dtype; bytes are moved, not
values).
"""

import torch


def pack(ks, vs, tok_begin, tok_end):
    """Phase 1: the buffer, a 1-D tensor, for samples ``ks[j], vs[j]`` and token
    ranges [tok_begin[j], tok_end[j])."""
    layers = ks[0].shape[0]
    parts = []
    for layer in range(layers):
        for cache in (ks, vs):                     # K, then V
            for j, c in enumerate(cache):          # samples in call order
                run = c[layer, :, tok_begin[j]:tok_end[j], :]   # [kv_heads, tokens, head_dim]
                parts.append(run.reshape(-1))
    return torch.cat(parts) if parts else torch.empty(0, dtype=ks[0].dtype)


def unpack(buf, ks, vs, tok_begin, tok_end):
    """Phase 3: write the buffer's runs into the given caches (in place) at
    token ranges [tok_begin[j], tok_end[j]); returns the caches."""
    layers, heads, _, hd = ks[0].shape
    off = 0
    for layer in range(layers):
        for cache in (ks, vs):
            for j, c in enumerate(cache):
                n = tok_end[j] - tok_begin[j]
                size = heads * n * hd
                c[layer, :, tok_begin[j]:tok_end[j], :] = buf[off:off + size].reshape(heads, n, hd)
                off += size
    assert off == buf.numel(), "buffer size does not match the ranges"
    return ks, vs


def transfer_bytes(layers, kv_heads, head_dim, tok_begin, tok_end, elem_bytes=2):
    """Size of the buffer in bytes."""
    tokens = sum(e - b for b, e in zip(tok_begin, tok_end))
    return tokens * layers * 2 * kv_heads * head_dim * elem_bytes
