"""GPU parity of the migration buffer (spec_kv_pack / spec_kv_unpack) against
the oracle, through the C ABI: the buffer must equal the oracle's bit for
bit, unpacking must write exactly the ranges, and a two-stage migration
(verified prefix first, then the tokens verified since) must deliver the
source's K/V bitwise."""

import dataclasses

import numpy as np
import pytest
import torch

import oracle
import paper_2512_04752_amd as sv
import workload as wl
from tests.gpu_util import say

pytestmark = pytest.mark.gpu


def random_pool(cfg, caps, seed):
    pool = sv.KVPool(cfg, caps)
    g = torch.Generator(device="cuda").manual_seed(seed)
    # random bit patterns, so that a misplaced element cannot match by accident
    pool.buf.copy_(torch.randint(0, 256, pool.buf.shape, generator=g, device="cuda",
                                 dtype=torch.uint8))
    torch.cuda.synchronize()
    return pool


def views(pool, ids):
    ks, vs = [], []
    for i in ids:
        k, v = pool.sample_view(i)
        ks.append(k.cpu().view(torch.int16))
        vs.append(v.cpu().view(torch.int16))
    return ks, vs


def gpu_pack(pool, ids, begin, end):
    n = sv.spec_kv_transfer_bytes(pool, begin, end)
    buf = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    sv.spec_kv_pack(pool, ids, begin, end, buf)
    torch.cuda.synchronize()
    return buf[:n]


CASES = {
    # samples in pool order 4, 0, 2, 3 (capacities 33, 40, 64, 1): a whole sample,
    # a middle range, and two empty ranges (at the end and of a 1-slot sample)
    "tiny": (wl.TINY, [40, 7, 64, 1, 33], [4, 0, 2, 3], [0, 3, 64, 1], [33, 40, 64, 1]),
    "tiny_ragged": (wl.TINY, [40, 7, 64, 1, 33], [2, 4, 1], [5, 0, 2], [60, 33, 7]),
    "llama1b_2layer": (dataclasses.replace(wl.LLAMA_1B, n_layers=2), [300, 1000, 77],
                       [1, 0, 2], [0, 123, 10], [1000, 300, 77]),
}


@pytest.mark.parametrize("name", sorted(CASES))
def test_pack_matches_oracle_bitwise(name):
    cfg, caps, ids, begin, end = CASES[name]
    say(f"pack parity {name}: samples {ids}, ranges {list(zip(begin, end))}")
    src = random_pool(cfg, caps, 11)
    buf = gpu_pack(src, ids, begin, end)
    ks, vs = views(src, ids)
    want = oracle.transfer.pack(ks, vs, begin, end)
    assert buf.numel() == want.numel() * 2 == oracle.transfer.transfer_bytes(
        cfg.n_layers, cfg.n_kv_heads, cfg.head_dim, begin, end)
    assert torch.equal(buf.cpu().view(torch.int16), want)


@pytest.mark.parametrize("name", sorted(CASES))
def test_unpack_writes_exactly_the_ranges(name):
    cfg, caps, ids, begin, end = CASES[name]
    say(f"unpack parity {name}")
    src = random_pool(cfg, caps, 12)
    buf = gpu_pack(src, ids, begin, end)
    # destination: another pool with other capacities, samples in another order
    dcaps = [max(caps) + 5] * len(caps)
    dst = random_pool(cfg, dcaps, 13)
    dids = [(i + 2) % len(dcaps) for i in ids]
    before_k, before_v = views(dst, dids)
    sv.spec_kv_unpack(dst, dids, begin, end, buf)
    torch.cuda.synchronize()
    got_k, got_v = views(dst, dids)
    want_k = [k.clone() for k in before_k]
    want_v = [v.clone() for v in before_v]
    oracle.transfer.unpack(buf.cpu().view(torch.int16), want_k, want_v, begin, end)
    for a, b in zip(got_k + got_v, want_k + want_v):
        assert torch.equal(a, b)


def test_two_stage_migration_llama8b():
    """The paper's migration of five samples between two instances' pools at
    the 8B shape: stage 1 moves the verified prefix, stage 2 the tokens
    verified meanwhile; the destination then holds the source's K/V."""
    cfg = wl.LLAMA_8B
    rng = np.random.default_rng(5)
    lens = [int(x) for x in np.clip(np.round(rng.lognormal(np.log(1024), 0.8, 5)), 128, 2048)]
    caps = [x + 16 for x in lens]
    say(f"two-stage migration, 8B shape, lengths {lens}")
    src = random_pool(cfg, caps, 21)
    dst = random_pool(cfg, [max(caps) + 100] * 6, 22)
    ids = list(range(5))
    dids = [5 - i for i in range(1, 6)]          # 4, 3, 2, 1, 0
    s1 = [x - 7 for x in lens]                   # verified when stage 1 starts
    zero = [0] * 5
    for b, e in ((zero, s1), (s1, lens)):
        n = sv.spec_kv_transfer_bytes(src, b, e)
        buf = torch.empty(n, dtype=torch.uint8, device="cuda")
        sv.spec_kv_pack(src, ids, b, e, buf)
        sv.spec_kv_unpack(dst, dids, b, e, buf)
    torch.cuda.synchronize()
    for i, d, S in zip(ids, dids, lens):
        ks, vs = src.sample_view(i)
        kd, vd = dst.sample_view(d)
        assert torch.equal(ks[:, :, :S].view(torch.int16), kd[:, :, :S].view(torch.int16))
        assert torch.equal(vs[:, :, :S].view(torch.int16), vd[:, :, :S].view(torch.int16))


def test_full_pack_matches_oracle_llama8b():
    """Every byte of an 8B-shape buffer (three samples, ~0.5 GB) against the
    oracle."""
    cfg = wl.LLAMA_8B
    caps = [1500, 2000, 640]
    ids, begin, end = [2, 0, 1], [0, 17, 5], [640, 1500, 1999]
    say("full 8B-shape pack parity")
    src = random_pool(cfg, caps, 31)
    buf = gpu_pack(src, ids, begin, end)
    ks, vs = views(src, ids)
    assert torch.equal(buf.cpu().view(torch.int16), oracle.transfer.pack(ks, vs, begin, end))
