"""Host-side checks of the C-ABI library that need no GPU: it loads, exports
every entry point the header declares, sizes KV pools and workspaces, carves
pools, and rejects malformed calls before touching the device."""

import ctypes
import os
import re

import numpy as np
import pytest

import paper_2512_04752_amd as sv
import workload as wl
from paper_2512_04752_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specverify.h")

# A plausible device address for pure host-side calls; never dereferenced,
# since every call below fails validation or touches no device memory.
FAKE_DEV = 0x7F0000000000


def header_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w]+\*?\s+\**(spec_\w+)\s*\(", text, re.M)))


def test_exports_every_declared_symbol():
    L = sv.lib()
    declared = header_functions()
    assert declared, "no declarations parsed"
    assert sorted(B.EXPORTS) == declared
    for name in declared:
        assert hasattr(L, name), name


def test_kv_bytes_arithmetic():
    cfg = wl.TINY
    caps = [100, 37, 1]
    per = lambda cap: (cfg.n_layers * 2 * cfg.n_kv_heads * cap * cfg.head_dim * 2 + 255) // 256 * 256
    ctl = (len(caps) * 32 + 255) // 256 * 256
    assert sv.spec_kv_bytes(cfg, caps) == sum(per(c) for c in caps) + ctl
    assert sv.spec_kv_bytes(cfg, [0]) == 0
    bad = wl.ModelConfig(2, 256, 4, 2, 32, 1024, 1024)          # head_dim 32 unsupported
    assert sv.spec_kv_bytes(bad, [10]) == 0


def test_kv_alloc_carves_contiguous_blocks():
    cfg = wl.LLAMA_8B
    caps = [1000, 17, 2048]
    need = sv.spec_kv_bytes(cfg, caps)
    L = sv.lib()
    c = B.make_config(cfg)
    arr = (ctypes.c_int32 * 3)(*caps)
    h = ctypes.c_void_p()
    assert L.spec_kv_alloc(ctypes.byref(c), 3, arr, ctypes.c_void_p(FAKE_DEV), need - 1,
                           ctypes.byref(h)) == -3
    assert L.spec_kv_alloc(ctypes.byref(c), 3, arr, ctypes.c_void_p(FAKE_DEV + 8), need,
                           ctypes.byref(h)) == -1          # misaligned
    assert L.spec_kv_alloc(ctypes.byref(c), 3, arr, ctypes.c_void_p(FAKE_DEV), need,
                           ctypes.byref(h)) == 0
    offs = [sv.spec_kv_sample_layout(h, i) for i in range(3)]
    assert offs[0] == (0, 1000)
    blk = lambda cap: cfg.n_layers * 2 * cfg.n_kv_heads * cap * cfg.head_dim * 2
    assert offs[1] == (blk(1000), 17)
    assert offs[2][0] == offs[1][0] + (blk(17) + 255) // 256 * 256
    with pytest.raises(sv.SpecError):
        sv.spec_kv_sample_layout(h, 3)
    sv.spec_kv_free(h)


def test_workspace_bytes_monotone():
    cfg = wl.LLAMA_8B
    a = sv.spec_workspace_bytes(cfg, 4, 256)
    b = sv.spec_workspace_bytes(cfg, 128, 1024)
    c = sv.spec_workspace_bytes(cfg, 256, 16384)
    assert 0 < a < b < c
    assert sv.spec_workspace_bytes(cfg, 0, 10) == 0
    assert sv.spec_workspace_bytes(cfg, 10, 5) == 0
    # the 16384-token sweep cell fits comfortably in one GPU's HBM
    assert c < 8 << 30


class FakeVerify:
    """spec_verify with fake device pointers: only for calls that must fail
    validation (the library checks everything before any device work)."""

    def __init__(self, cfg=wl.TINY, caps=(200, 200, 200)):
        self.cfg = cfg
        self.c = B.make_config(cfg)
        self.L = sv.lib()
        arr = (ctypes.c_int32 * len(caps))(*caps)
        need = sv.spec_kv_bytes(cfg, list(caps))
        self.kv = ctypes.c_void_p()
        assert self.L.spec_kv_alloc(ctypes.byref(self.c), len(caps), arr,
                                    ctypes.c_void_p(FAKE_DEV), need, ctypes.byref(self.kv)) == 0
        n = cfg.n_layers
        self.ptrs = {k: (ctypes.c_void_p * n)(*[FAKE_DEV] * n) for k in B.Weights.LAYER_FIELDS}
        self.w = B.spec_weights(FAKE_DEV, FAKE_DEV, FAKE_DEV,
                                *[ctypes.cast(self.ptrs[k], ctypes.POINTER(ctypes.c_void_p))
                                  for k in B.Weights.LAYER_FIELDS])

    def call(self, ids, trees, lens, ws_bytes=None):
        offs, toks, pars = sv.flatten_trees(trees)
        if ws_bytes is None:
            ws_bytes = sv.spec_workspace_bytes(self.cfg, len(ids), int(offs[-1]))
        i = lambda a: B._i32(a)
        (a1, p1), (a2, p2), (a3, p3), (a4, p4), (a5, p5) = (i(ids), i(offs), i(toks), i(pars),
                                                            i(lens))
        rc = self.L.spec_verify(ctypes.byref(self.c), ctypes.byref(self.w), self.kv, len(ids), p1,
                                p2, p3, p4, p5, ctypes.c_void_p(FAKE_DEV), ws_bytes, None,
                                ctypes.c_void_p(FAKE_DEV), ctypes.c_void_p(FAKE_DEV),
                                ctypes.c_void_p(FAKE_DEV), None)
        return rc, self.L.spec_last_error().decode()

    def close(self):
        self.L.spec_kv_free(self.kv)


@pytest.fixture
def fake():
    f = FakeVerify()
    yield f
    f.close()


GOOD = ([5, 6, 7], [-1, 0, 0])


@pytest.mark.parametrize("case,code", [
    ("root_parent", -2), ("parent_after", -2), ("parent_self", -2), ("token_range", -2),
    ("negative_token", -2), ("empty_tree", -2), ("too_big_tree", -6), ("capacity", -3),
    ("dup_sample", -1), ("bad_sample", -1), ("workspace", -5), ("neg_len", -1),
])
def test_validation_errors(fake, case, code):
    ids, trees, lens, ws = [0, 1], [GOOD, GOOD], [10, 10], None
    if case == "root_parent":
        trees = [GOOD, ([1, 2], [0, 0])]
    elif case == "parent_after":
        trees = [GOOD, ([1, 2, 3], [-1, 2, 0])]
    elif case == "parent_self":
        trees = [GOOD, ([1, 2, 3], [-1, 0, 2])]
    elif case == "token_range":
        trees = [GOOD, ([1, 1024], [-1, 0])]
    elif case == "negative_token":
        trees = [GOOD, ([1, -3], [-1, 0])]
    elif case == "empty_tree":
        trees = [GOOD, ([], [])]
    elif case == "too_big_tree":
        n = B.SPEC_MAX_TREE + 1
        trees = [GOOD, ([1] * n, wl.chain_tree(n))]
    elif case == "capacity":
        lens = [10, 198]
    elif case == "dup_sample":
        ids = [1, 1]
    elif case == "bad_sample":
        ids = [0, 3]
    elif case == "workspace":
        ws = 1000
    elif case == "neg_len":
        lens = [10, -1]
    rc, msg = fake.call(ids, trees, lens, ws)
    assert rc == code, msg
    assert msg


def test_unsupported_shape_rejected():
    L = sv.lib()
    bad = B.make_config(wl.ModelConfig(2, 200, 4, 2, 64, 1024, 1024))   # hidden % 128 != 0
    arr = (ctypes.c_int32 * 1)(10)
    h = ctypes.c_void_p()
    assert L.spec_kv_alloc(ctypes.byref(bad), 1, arr, ctypes.c_void_p(FAKE_DEV), 1 << 30,
                           ctypes.byref(h)) == -6
    assert b"hidden" in L.spec_last_error()


def test_commit_validation(fake):
    L = fake.L
    ids = (ctypes.c_int32 * 2)(0, 0)
    lens = (ctypes.c_int32 * 2)(5, 5)
    assert L.spec_kv_commit(fake.kv, 2, ids, lens, ctypes.c_void_p(FAKE_DEV),
                            ctypes.c_void_p(FAKE_DEV), ctypes.c_void_p(FAKE_DEV), None) == -1
    ids = (ctypes.c_int32 * 1)(0)
    lens = (ctypes.c_int32 * 1)(200)
    assert L.spec_kv_commit(fake.kv, 1, ids, lens, ctypes.c_void_p(FAKE_DEV),
                            ctypes.c_void_p(FAKE_DEV), ctypes.c_void_p(FAKE_DEV), None) == -3


def test_flatten_trees():
    offs, toks, pars = sv.flatten_trees([([1, 2], [-1, 0]), ([3], [-1])])
    assert offs.tolist() == [0, 2, 3] and toks.tolist() == [1, 2, 3] and pars.tolist() == [-1, 0, -1]


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="missing"):
        B.lib()


def test_transfer_bytes_and_validation(fake):
    """spec_kv_transfer_bytes arithmetic and the pack/unpack rejections, all
    before any device work (fake device pointers are never touched)."""
    L = fake.L
    cfg = fake.cfg
    i32 = lambda *v: (ctypes.c_int32 * len(v))(*v)
    per_tok = cfg.n_layers * 2 * cfg.n_kv_heads * cfg.head_dim * 2
    assert L.spec_kv_transfer_bytes(fake.kv, 2, i32(3, 0), i32(10, 0)) == 7 * per_tok
    assert L.spec_kv_transfer_bytes(fake.kv, 2, i32(3, 5), i32(10, 4)) == 0      # end < begin
    need = 12 * per_tok
    buf = ctypes.c_void_p(FAKE_DEV)
    for fn in (L.spec_kv_pack, L.spec_kv_unpack):
        # range past the capacity (200)
        assert fn(fake.kv, 2, i32(0, 1), i32(0, 195), i32(10, 202), buf, need, None) == -3
        # buffer too small
        assert fn(fake.kv, 2, i32(0, 1), i32(0, 0), i32(5, 7), buf, need - 1, None) == -3
        # misaligned buffer
        assert fn(fake.kv, 1, i32(0), i32(0), i32(5), ctypes.c_void_p(FAKE_DEV + 8), need,
                  None) == -1
        # duplicate and out-of-range sample ids
        assert fn(fake.kv, 2, i32(1, 1), i32(0, 0), i32(1, 1), buf, need, None) == -1
        assert fn(fake.kv, 1, i32(3), i32(0), i32(1), buf, need, None) == -1
        # negative begin
        assert fn(fake.kv, 1, i32(0), i32(-1), i32(1), buf, need, None) == -3
        assert L.spec_last_error()
    # nothing to move: accepted without device work
    assert L.spec_kv_pack(fake.kv, 1, i32(0), i32(4), i32(4), buf, 0, None) == 0


def test_sampled_workspace_adds_logits_and_residual():
    cfg = wl.LLAMA_8B
    for b, n in [(1, 1), (4, 256), (128, 1024)]:
        plain = sv.spec_workspace_bytes(cfg, b, n)
        samp = sv.spec_workspace_bytes_sampled(cfg, b, n)
        # fp32 logits, a 96-byte decision per node, an fp64 row per sample
        extra = n * cfg.vocab * 4 + n * 96 + b * cfg.vocab * 8
        assert extra <= samp - plain < extra + 1024
    assert sv.spec_workspace_bytes_sampled(cfg, 0, 8) == 0


def sampled_call(f, samp, ws_bytes=None, trees=None):
    ids, lens = [0, 1], [10, 10]
    trees = trees or [GOOD, GOOD]
    offs, toks, pars = sv.flatten_trees(trees)
    if ws_bytes is None:
        ws_bytes = sv.spec_workspace_bytes_sampled(f.cfg, len(ids), int(offs[-1]))
    (a1, p1), (a2, p2), (a3, p3), (a4, p4), (a5, p5) = (B._i32(ids), B._i32(offs), B._i32(toks),
                                                        B._i32(pars), B._i32(lens))
    rc = f.L.spec_verify_sampled(ctypes.byref(f.c), ctypes.byref(f.w), f.kv, len(ids), p1, p2, p3,
                                 p4, p5, ctypes.c_void_p(FAKE_DEV), ws_bytes, None,
                                 ctypes.byref(samp) if samp is not None else None,
                                 ctypes.c_void_p(FAKE_DEV), ctypes.c_void_p(FAKE_DEV),
                                 ctypes.c_void_p(FAKE_DEV), None)
    return rc, f.L.spec_last_error().decode()


@pytest.mark.parametrize("case", ["null", "neg_t", "nan_t", "inf_t", "eos_high", "eos_low",
                                  "no_q", "no_u", "plain_ws", "tree"])
def test_sampled_validation(fake, case):
    """Malformed sampled calls fail before any device work (fake device
    pointers are never dereferenced)."""
    samp = B.spec_sampling(0.8, -1, FAKE_DEV, FAKE_DEV)
    ws, trees, code = None, None, -1
    if case == "null":
        samp = None
    elif case == "neg_t":
        samp.temperature = -0.5
    elif case == "nan_t":
        samp.temperature = float("nan")
    elif case == "inf_t":
        samp.temperature = float("inf")
    elif case == "eos_high":
        samp.eos_token = fake.cfg.vocab
    elif case == "eos_low":
        samp.eos_token = -2
    elif case == "no_q":
        samp.draft_probs = None
    elif case == "no_u":
        samp.uniforms = None
    elif case == "plain_ws":
        ws, code = sv.spec_workspace_bytes(fake.cfg, 2, 6), -5
    elif case == "tree":
        trees, code = [GOOD, ([1, 2], [-1, 1])], -2
    rc, msg = sampled_call(fake, samp, ws, trees)
    assert rc == code, msg
    assert msg


def test_sampled_workspace_beyond_4gib():
    """Sizes are size_t end to end (a 16384-node sampled call needs over
    4 GiB for its fp32 logits alone)."""
    n = sv.spec_workspace_bytes_sampled(wl.LLAMA_8B, 512, 16384)
    assert n > 16384 * wl.LLAMA_8B.vocab * 4 > 1 << 32


def test_noalloc_rejects_calls_beyond_its_scratch():
    """spec_verify_noalloc refuses, before any device work, a call whose
    workspace would exceed the static scratch, and validates like
    spec_verify."""
    cfg = wl.LLAMA_8B
    caps = [4096] * 256
    f = FakeVerify(cfg, caps)
    try:
        def call(ids, trees, lens):
            offs, toks, pars = sv.flatten_trees(trees)
            i = lambda a: B._i32(a)   # noqa: E731
            (_, p1), (_, p2), (_, p3), (_, p4), (_, p5) = (i(ids), i(offs), i(toks), i(pars),
                                                          i(lens))
            rc = f.L.spec_verify_noalloc(ctypes.byref(f.c), ctypes.byref(f.w), f.kv, len(ids),
                                         p1, p2, p3, p4, p5, None, ctypes.c_void_p(FAKE_DEV),
                                         ctypes.c_void_p(FAKE_DEV), ctypes.c_void_p(FAKE_DEV),
                                         None)
            return rc, f.L.spec_last_error().decode()
        tree = (list(range(16)), [-1] + list(range(15)))
        assert sv.spec_workspace_bytes(cfg, 256, 4096) > B.SPEC_NOALLOC_SCRATCH_BYTES
        rc, msg = call(list(range(256)), [tree] * 256, [100] * 256)
        assert rc == -5 and "static scratch" in msg, msg
        rc, msg = call([0, 1], [tree, ([1, 2], [0, 0])], [10, 10])
        assert rc == -2, msg
    finally:
        f.close()
