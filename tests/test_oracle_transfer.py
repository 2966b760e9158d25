"""Pins of the migration-buffer oracle (oracle.transfer), CPU only.

Every cache element carries a unique integer code (sample, layer, K/V,
head, position, dim), so the buffer's order is checked element by element
against a closed-form offset written independently of the oracle's
concatenation: layer, then K before V, then samples in call order, then
heads, then tokens, then head_dim (the paper's model -> layer -> sample
hierarchy of Section 6.2)."""

import itertools

import pytest
import torch

from oracle import transfer

L, H, D = 3, 2, 4


def coded_caches(caps):
    ks, vs = [], []
    for j, cap in enumerate(caps):
        idx = torch.arange(L * H * cap * D, dtype=torch.int64).reshape(L, H, cap, D)
        l_ = idx // (H * cap * D)
        h_ = (idx // (cap * D)) % H
        p_ = (idx // D) % cap
        d_ = idx % D
        code = lambda kv: ((((j * L + l_) * 2 + kv) * H + h_) * 1000 + p_) * D + d_
        ks.append(code(0))
        vs.append(code(1))
    return ks, vs


def closed_form_offset(layer, kv, j, head, t, d, begin, end):
    """Offset of element (layer, K/V, sample j, head, token t, dim d)."""
    n = [e - b for b, e in zip(begin, end)]
    total = sum(n)
    slab = total * H * D                      # one (layer, K/V)
    before = sum(n[:j])                       # tokens of earlier samples
    return (layer * 2 + kv) * slab + before * H * D + head * n[j] * D + (t - begin[j]) * D + d


@pytest.mark.parametrize("begin,end", [([0, 3, 5], [7, 3, 9]),      # an empty range in the middle
                                       ([2], [11]),
                                       ([0, 0], [1, 12])])
def test_buffer_order_matches_closed_form(begin, end):
    caps = [12] * len(begin)
    ks, vs = coded_caches(caps)
    buf = transfer.pack(ks, vs, begin, end)
    assert buf.numel() * 2 == transfer.transfer_bytes(L, H, D, begin, end)
    seen = 0
    for j in range(len(begin)):
        for layer, kv, head, t, d in itertools.product(range(L), range(2), range(H),
                                                       range(begin[j], end[j]), range(D)):
            src = (ks if kv == 0 else vs)[j][layer, head, t, d]
            assert buf[closed_form_offset(layer, kv, j, head, t, d, begin, end)] == src
            seen += 1
    assert seen == buf.numel()


def test_round_trip_moves_only_the_ranges():
    caps = [10, 6]
    ks, vs = coded_caches(caps)
    begin, end = [2, 0], [9, 6]
    buf = transfer.pack(ks, vs, begin, end)
    dk = [torch.full_like(k, -1) for k in ks]
    dv = [torch.full_like(v, -1) for v in vs]
    transfer.unpack(buf, dk, dv, begin, end)
    for j in range(2):
        assert torch.equal(dk[j][:, :, begin[j]:end[j]], ks[j][:, :, begin[j]:end[j]])
        assert torch.equal(dv[j][:, :, begin[j]:end[j]], vs[j][:, :, begin[j]:end[j]])
        outside = torch.ones(caps[j], dtype=torch.bool)
        outside[begin[j]:end[j]] = False
        assert (dk[j][:, :, outside] == -1).all() and (dv[j][:, :, outside] == -1).all()


def test_two_stage_migration_equals_one_copy():
    """Stage 1 moves the verified prefix, stage 2 the tokens verified since;
    together they deliver the same cache as moving everything at once."""
    ks, vs = coded_caches([20, 20])
    s1b, s1e = [0, 0], [11, 7]
    s2b, s2e = [11, 7], [15, 20]
    once = ([torch.zeros_like(k) for k in ks], [torch.zeros_like(v) for v in vs])
    transfer.unpack(transfer.pack(ks, vs, [0, 0], [15, 20]), *once, [0, 0], [15, 20])
    two = ([torch.zeros_like(k) for k in ks], [torch.zeros_like(v) for v in vs])
    transfer.unpack(transfer.pack(ks, vs, s1b, s1e), *two, s1b, s1e)
    transfer.unpack(transfer.pack(ks, vs, s2b, s2e), *two, s2b, s2e)
    for a, b in zip(once[0] + once[1], two[0] + two[1]):
        assert torch.equal(a, b)


def test_planted_mistakes_are_caught():
    """Plausible layout mistakes, planted in a copy of pack, fail the
    closed-form check."""
    caps = [8, 8]
    ks, vs = coded_caches(caps)
    begin, end = [1, 2], [6, 8]

    def v_before_k(ks, vs, b, e):
        return transfer.pack(vs, ks, b, e)

    def samples_outermost(ks, vs, b, e):
        parts = []
        for j in range(len(ks)):
            for layer in range(L):
                for c in (ks, vs):
                    parts.append(c[j][layer, :, b[j]:e[j], :].reshape(-1))
        return torch.cat(parts)

    def tokens_before_heads(ks, vs, b, e):
        parts = []
        for layer in range(L):
            for c in (ks, vs):
                for j in range(len(ks)):
                    parts.append(c[j][layer, :, b[j]:e[j], :].transpose(0, 1).reshape(-1))
        return torch.cat(parts)

    for bad in (v_before_k, samples_outermost, tokens_before_heads):
        buf = bad(ks, vs, begin, end)
        ok = all(buf[closed_form_offset(layer, kv, j, head, t, d, begin, end)] ==
                 (ks if kv == 0 else vs)[j][layer, head, t, d]
                 for j in range(2) for layer in range(L) for kv in range(2) for head in range(H)
                 for t in range(begin[j], end[j]) for d in range(D))
        assert not ok, bad.__name__
