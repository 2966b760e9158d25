"""ctypes binding of libspecverify.so: the C entry points under the same
names, marshalling torch tensors, numpy arrays and Python lists into
pointers.  Every step of the verify computation runs in the library's HIP
kernels; PyTorch only provides device memory and the stream.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_float, c_int32, c_int64, c_size_t, c_uint64, c_void_p

import numpy as np
import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspecverify.so")

SPEC_MAX_TREE = 256
SPEC_ANC_WORDS = SPEC_MAX_TREE // 64   # 64-bit words of one node's ancestor set
STATUS = {0: "SPEC_OK", -1: "SPEC_ERR_INVALID", -2: "SPEC_ERR_TREE", -3: "SPEC_ERR_CAPACITY",
          -5: "SPEC_ERR_WORKSPACE", -6: "SPEC_ERR_UNSUPPORTED", -7: "SPEC_ERR_HIP"}
KERNEL_CLASS = {"gemm_qkv": 0, "attention": 1, "gemm_o": 2, "gemm_gate_up": 3, "gemm_down": 4,
                "lm_head": 5, "commit": 6, "accept": 8}   # the kernel classes of one verify step
TRANSFER_CLASS = 7                                    # spec_kv_pack / spec_kv_unpack

# Every symbol the public header declares.
EXPORTS = ("spec_kv_bytes", "spec_kv_alloc", "spec_kv_free", "spec_kv_sample_layout",
           "spec_workspace_bytes", "spec_verify", "spec_kv_commit", "spec_last_error",
           "spec_profile_begin", "spec_profile_end", "spec_kv_transfer_bytes", "spec_kv_pack",
           "spec_kv_unpack", "spec_cost_model_create", "spec_cost_model_free", "spec_cost_predict",
           "spec_cost_model_stats", "spec_select_draft_count", "spec_workspace_bytes_sampled",
           "spec_verify_sampled", "spec_verify_noalloc")
SPEC_NOALLOC_SCRATCH_BYTES = 320 << 20


class SpecError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"{STATUS.get(code, code)}: {msg}")
        self.code = code


class spec_model_config(ctypes.Structure):
    _fields_ = [("n_layers", c_int32), ("hidden", c_int32), ("n_heads", c_int32),
                ("n_kv_heads", c_int32), ("head_dim", c_int32), ("ffn", c_int32),
                ("vocab", c_int32), ("rope_theta", c_float), ("rms_eps", c_float)]


class spec_weights(ctypes.Structure):
    _fields_ = [("tok_embed", c_void_p), ("final_norm", c_void_p), ("lm_head", c_void_p),
                ("attn_norm", POINTER(c_void_p)), ("wq", POINTER(c_void_p)),
                ("wk", POINTER(c_void_p)), ("wv", POINTER(c_void_p)), ("wo", POINTER(c_void_p)),
                ("ffn_norm", POINTER(c_void_p)), ("w_gate", POINTER(c_void_p)),
                ("w_up", POINTER(c_void_p)), ("w_down", POINTER(c_void_p))]


class spec_cost_coeffs(ctypes.Structure):
    _fields_ = [("c0", ctypes.c_double), ("c_seq", ctypes.c_double), ("c_draft", ctypes.c_double),
                ("c_tree", ctypes.c_double), ("bucket_ratio", ctypes.c_double)]


class spec_sampling(ctypes.Structure):
    _fields_ = [("temperature", c_float), ("eos_token", c_int32), ("draft_probs", c_void_p),
                ("uniforms", c_void_p)]


class spec_debug(ctypes.Structure):
    _fields_ = [("logits", c_void_p), ("argmax", c_void_p), ("depth", c_void_p),
                ("pos", c_void_p), ("anc", c_void_p)]


_lib = None


def lib():
    """Load the library; fails loudly when it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing; build it with "
                           "`python -m paper_2512_04752_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    i32p = POINTER(c_int32)
    L.spec_kv_bytes.argtypes = [POINTER(spec_model_config), c_int32, i32p]
    L.spec_kv_bytes.restype = c_size_t
    L.spec_kv_alloc.argtypes = [POINTER(spec_model_config), c_int32, i32p, c_void_p, c_size_t,
                                POINTER(c_void_p)]
    L.spec_kv_free.argtypes = [c_void_p]
    L.spec_kv_sample_layout.argtypes = [c_void_p, c_int32, POINTER(c_int64), i32p]
    L.spec_workspace_bytes.argtypes = [POINTER(spec_model_config), c_int32, c_int32]
    L.spec_workspace_bytes.restype = c_size_t
    L.spec_verify.argtypes = [POINTER(spec_model_config), POINTER(spec_weights), c_void_p,
                              c_int32, i32p, i32p, i32p, i32p, i32p, c_void_p, c_size_t,
                              c_void_p, c_void_p, c_void_p, c_void_p, POINTER(spec_debug)]
    L.spec_kv_commit.argtypes = [c_void_p, c_int32, i32p, i32p, c_void_p, c_void_p, c_void_p,
                                 c_void_p]
    L.spec_workspace_bytes_sampled.argtypes = [POINTER(spec_model_config), c_int32, c_int32]
    L.spec_workspace_bytes_sampled.restype = c_size_t
    L.spec_verify_sampled.argtypes = [POINTER(spec_model_config), POINTER(spec_weights), c_void_p,
                                      c_int32, i32p, i32p, i32p, i32p, i32p, c_void_p, c_size_t,
                                      c_void_p, POINTER(spec_sampling), c_void_p, c_void_p,
                                      c_void_p, POINTER(spec_debug)]
    L.spec_verify_noalloc.argtypes = [POINTER(spec_model_config), POINTER(spec_weights),
                                      c_void_p, c_int32, i32p, i32p, i32p, i32p, i32p, c_void_p,
                                      c_void_p, c_void_p, c_void_p, POINTER(spec_debug)]
    L.spec_kv_transfer_bytes.argtypes = [c_void_p, c_int32, i32p, i32p]
    L.spec_kv_transfer_bytes.restype = c_size_t
    L.spec_kv_pack.argtypes = [c_void_p, c_int32, i32p, i32p, i32p, c_void_p, c_size_t, c_void_p]
    L.spec_kv_unpack.argtypes = [c_void_p, c_int32, i32p, i32p, i32p, c_void_p, c_size_t, c_void_p]
    L.spec_cost_model_create.argtypes = [POINTER(spec_cost_coeffs), POINTER(c_void_p)]
    L.spec_cost_model_free.argtypes = [c_void_p]
    L.spec_cost_predict.argtypes = [c_void_p, c_int64, c_int64, c_int64]
    L.spec_cost_predict.restype = ctypes.c_double
    L.spec_cost_model_stats.argtypes = [c_void_p, POINTER(c_int64), POINTER(c_int64)]
    L.spec_select_draft_count.argtypes = [c_void_p, c_int32, i32p, i32p, i32p,
                                          POINTER(c_float), c_int32, c_int32, i32p, i32p,
                                          POINTER(ctypes.c_double)]
    L.spec_last_error.restype = ctypes.c_char_p
    L.spec_profile_begin.argtypes = [c_int32, c_int32]
    L.spec_profile_end.argtypes = [POINTER(c_float), i32p]
    for name in ("spec_kv_alloc", "spec_kv_free", "spec_kv_sample_layout", "spec_verify",
                 "spec_kv_commit", "spec_profile_begin", "spec_profile_end", "spec_kv_pack",
                 "spec_kv_unpack", "spec_cost_model_create", "spec_cost_model_free",
                 "spec_cost_model_stats", "spec_select_draft_count", "spec_verify_sampled",
                 "spec_verify_noalloc"):
        getattr(L, name).restype = c_int32
    _lib = L
    return L


def _check(rc):
    if rc != 0:
        raise SpecError(rc, lib().spec_last_error().decode())


def _i32(a):
    arr = np.ascontiguousarray(np.asarray(a, dtype=np.int32))
    return arr, arr.ctypes.data_as(POINTER(c_int32))


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return c_void_p(stream.cuda_stream)


def make_config(cfg) -> spec_model_config:
    return spec_model_config(cfg.n_layers, cfg.hidden, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim,
                             cfg.ffn, cfg.vocab, float(cfg.rope_theta), float(cfg.rms_eps))


class Weights:
    """Device bf16 weights plus the spec_weights struct pointing at them."""

    LAYER_FIELDS = ("attn_norm", "wq", "wk", "wv", "wo", "ffn_norm", "w_gate", "w_up", "w_down")

    def __init__(self, W):
        self.W = W
        for t in [W["tok_embed"], W["final_norm"], W["lm_head"]] + \
                [lw[k] for lw in W["layers"] for k in self.LAYER_FIELDS]:
            if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous():
                raise ValueError("weights must be contiguous bf16 device tensors")
        n = len(W["layers"])
        self._arrays = {}
        for k in self.LAYER_FIELDS:
            arr = (c_void_p * n)(*[lw[k].data_ptr() for lw in W["layers"]])
            self._arrays[k] = arr
        self.struct = spec_weights(W["tok_embed"].data_ptr(), W["final_norm"].data_ptr(),
                                   W["lm_head"].data_ptr(),
                                   *[ctypes.cast(self._arrays[k], POINTER(c_void_p))
                                     for k in self.LAYER_FIELDS])


def spec_kv_bytes(cfg, capacity) -> int:
    c = make_config(cfg)
    arr, p = _i32(capacity)
    return int(lib().spec_kv_bytes(ctypes.byref(c), len(arr), p))


class KVPool:
    """A KV pool over a torch-owned device buffer (spec_kv_alloc)."""

    def __init__(self, cfg, capacity, device="cuda"):
        self.cfg = cfg
        self.ccfg = make_config(cfg)
        self.capacity = [int(c) for c in capacity]
        nbytes = spec_kv_bytes(cfg, self.capacity)
        if nbytes == 0:
            raise SpecError(-1, "invalid KV pool request")
        self.buf = torch.empty(nbytes, dtype=torch.uint8, device=device)
        self.handle = spec_kv_alloc(cfg, self.capacity, self.buf)

    def sample_view(self, sample):
        """(K, V) views of one sample, each [n_layers, n_kv_heads, capacity, head_dim]."""
        off, cap = spec_kv_sample_layout(self.handle, sample)
        c = self.cfg
        n = c.n_layers * 2 * c.n_kv_heads * cap * c.head_dim
        blk = self.buf[off:off + 2 * n].view(torch.bfloat16)
        blk = blk.view(c.n_layers, 2, c.n_kv_heads, cap, c.head_dim)
        return blk[:, 0], blk[:, 1]

    def close(self):
        if self.handle is not None:
            spec_kv_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def spec_kv_alloc(cfg, capacity, buf):
    c = make_config(cfg)
    arr, p = _i32(capacity)
    h = c_void_p()
    _check(lib().spec_kv_alloc(ctypes.byref(c), len(arr), p, c_void_p(buf.data_ptr()),
                               buf.numel() * buf.element_size(), ctypes.byref(h)))
    return h


def spec_kv_free(handle):
    _check(lib().spec_kv_free(handle))


def spec_kv_sample_layout(handle, sample):
    off, cap = c_int64(), c_int32()
    _check(lib().spec_kv_sample_layout(handle, sample, ctypes.byref(off), ctypes.byref(cap)))
    return off.value, cap.value


def spec_workspace_bytes(cfg, max_batch, max_tokens) -> int:
    c = make_config(cfg)
    return int(lib().spec_workspace_bytes(ctypes.byref(c), max_batch, max_tokens))


def spec_verify(cfg, weights: Weights, kv: KVPool, sample_ids, tree_offsets, tree_tokens,
                tree_parents, seq_lens, workspace, accepted_len, next_token, accepted_nodes,
                debug=None, stream=None):
    """Enqueue one verify step.  Host arrays may be lists or numpy arrays;
    workspace and outputs are device tensors; ``debug`` is an optional dict
    with any of logits/argmax/depth/pos/anc device tensors."""
    c = make_config(cfg)
    ids, p_ids = _i32(sample_ids)
    offs, p_offs = _i32(tree_offsets)
    toks, p_toks = _i32(tree_tokens)
    pars, p_pars = _i32(tree_parents)
    lens, p_lens = _i32(seq_lens)
    dbg = None
    if debug:
        dbg = spec_debug(*[debug[k].data_ptr() if debug.get(k) is not None else None
                           for k in ("logits", "argmax", "depth", "pos", "anc")])
    _check(lib().spec_verify(ctypes.byref(c), ctypes.byref(weights.struct), kv.handle,
                             len(ids), p_ids, p_offs, p_toks, p_pars, p_lens,
                             _ptr(workspace), workspace.numel() * workspace.element_size(),
                             _stream(stream), _ptr(accepted_len), _ptr(next_token),
                             _ptr(accepted_nodes), ctypes.byref(dbg) if dbg else None))


def spec_verify_noalloc(cfg, weights: Weights, kv: KVPool, sample_ids, tree_offsets, tree_tokens,
                        tree_parents, seq_lens, accepted_len, next_token, accepted_nodes,
                        debug=None, stream=None):
    """spec_verify with the library's static device scratch as workspace."""
    c = make_config(cfg)
    ids, p_ids = _i32(sample_ids)
    offs, p_offs = _i32(tree_offsets)
    toks, p_toks = _i32(tree_tokens)
    pars, p_pars = _i32(tree_parents)
    lens, p_lens = _i32(seq_lens)
    dbg = None
    if debug:
        dbg = spec_debug(*[debug[k].data_ptr() if debug.get(k) is not None else None
                           for k in ("logits", "argmax", "depth", "pos", "anc")])
    _check(lib().spec_verify_noalloc(ctypes.byref(c), ctypes.byref(weights.struct), kv.handle,
                                     len(ids), p_ids, p_offs, p_toks, p_pars, p_lens,
                                     _stream(stream), _ptr(accepted_len), _ptr(next_token),
                                     _ptr(accepted_nodes), ctypes.byref(dbg) if dbg else None))


def spec_workspace_bytes_sampled(cfg, max_batch, max_tokens) -> int:
    c = make_config(cfg)
    return int(lib().spec_workspace_bytes_sampled(ctypes.byref(c), max_batch, max_tokens))


def spec_verify_sampled(cfg, weights: Weights, kv: KVPool, sample_ids, tree_offsets, tree_tokens,
                        tree_parents, seq_lens, workspace, accepted_len, next_token,
                        accepted_nodes, temperature, eos_token=-1, draft_probs=None,
                        uniforms=None, debug=None, stream=None):
    """spec_verify with speculative-sampling acceptance at ``temperature`` (0:
    greedy) and end-of-sequence truncation.  draft_probs: device fp32
    [N][vocab]; uniforms: device fp32 [N][2]."""
    c = make_config(cfg)
    ids, p_ids = _i32(sample_ids)
    offs, p_offs = _i32(tree_offsets)
    toks, p_toks = _i32(tree_tokens)
    pars, p_pars = _i32(tree_parents)
    lens, p_lens = _i32(seq_lens)
    n = int(offs[-1])
    if temperature > 0:
        for t, cols, what in ((draft_probs, cfg.vocab, "draft_probs"), (uniforms, 2, "uniforms")):
            if (t is None or t.dtype != torch.float32 or not t.is_contiguous()
                    or tuple(t.shape) != (n, cols)):
                raise ValueError(f"{what} must be a contiguous float32 [{n}, {cols}] tensor")
    samp = spec_sampling(float(temperature), int(eos_token), _ptr(draft_probs), _ptr(uniforms))
    dbg = None
    if debug:
        dbg = spec_debug(*[debug[k].data_ptr() if debug.get(k) is not None else None
                           for k in ("logits", "argmax", "depth", "pos", "anc")])
    _check(lib().spec_verify_sampled(ctypes.byref(c), ctypes.byref(weights.struct), kv.handle,
                                     len(ids), p_ids, p_offs, p_toks, p_pars, p_lens,
                                     _ptr(workspace), workspace.numel() * workspace.element_size(),
                                     _stream(stream), ctypes.byref(samp), _ptr(accepted_len),
                                     _ptr(next_token), _ptr(accepted_nodes),
                                     ctypes.byref(dbg) if dbg else None))


def spec_kv_commit(kv: KVPool, sample_ids, seq_lens, accepted_len, accepted_nodes, new_seq_lens,
                   stream=None):
    ids, p_ids = _i32(sample_ids)
    lens, p_lens = _i32(seq_lens)
    _check(lib().spec_kv_commit(kv.handle, len(ids), p_ids, p_lens, _ptr(accepted_len),
                                _ptr(accepted_nodes), _ptr(new_seq_lens), _stream(stream)))


def spec_kv_transfer_bytes(kv: KVPool, tok_begin, tok_end) -> int:
    b, p_b = _i32(tok_begin)
    e, p_e = _i32(tok_end)
    return int(lib().spec_kv_transfer_bytes(kv.handle, len(b), p_b, p_e))


def spec_kv_pack(kv: KVPool, sample_ids, tok_begin, tok_end, buf, stream=None):
    """Copy token ranges of the given samples into the transfer buffer ``buf``
    (a device tensor of at least spec_kv_transfer_bytes bytes)."""
    ids, p_ids = _i32(sample_ids)
    b, p_b = _i32(tok_begin)
    e, p_e = _i32(tok_end)
    _check(lib().spec_kv_pack(kv.handle, len(ids), p_ids, p_b, p_e, _ptr(buf),
                              buf.numel() * buf.element_size(), _stream(stream)))


def spec_kv_unpack(kv: KVPool, sample_ids, tok_begin, tok_end, buf, stream=None):
    """Write a transfer buffer's runs into token ranges of this pool's samples."""
    ids, p_ids = _i32(sample_ids)
    b, p_b = _i32(tok_begin)
    e, p_e = _i32(tok_end)
    _check(lib().spec_kv_unpack(kv.handle, len(ids), p_ids, p_b, p_e, _ptr(buf),
                                buf.numel() * buf.element_size(), _stream(stream)))


class CostModel:
    """The library's verification-cost predictor (spec_cost_model_*)."""

    def __init__(self, c0, c_seq, c_draft, c_tree, bucket_ratio=0.0):
        self.coeffs = spec_cost_coeffs(c0, c_seq, c_draft, c_tree, bucket_ratio)
        h = c_void_p()
        _check(lib().spec_cost_model_create(ctypes.byref(self.coeffs), ctypes.byref(h)))
        self.handle = h

    @classmethod
    def from_dict(cls, d, bucket_ratio=None):
        return cls(d["c0"], d["c_seq"], d["c_draft"], d["c_tree"],
                   d.get("bucket_ratio", 0.0) if bucket_ratio is None else bucket_ratio)

    def predict(self, n_seq, n_draft, tree_kv):
        t = lib().spec_cost_predict(self.handle, int(n_seq), int(n_draft), int(tree_kv))
        if t < 0:
            raise SpecError(-1, "negative feature")
        return t

    def stats(self):
        h, m = c_int64(), c_int64()
        _check(lib().spec_cost_model_stats(self.handle, ctypes.byref(h), ctypes.byref(m)))
        return h.value, m.value

    def close(self):
        if self.handle is not None:
            _check(lib().spec_cost_model_free(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def spec_select_draft_count(model: CostModel, seq_lens, tree_offsets, parents, weights, n_max,
                            patience=2):
    """Returns (n, selected [batch][n_max] int32 array, objective [n_max])."""
    lens, p_lens = _i32(seq_lens)
    offs, p_offs = _i32(tree_offsets)
    pars, p_pars = _i32(parents)
    w = np.ascontiguousarray(np.asarray(weights, dtype=np.float32))
    sel = np.empty((len(lens), n_max), dtype=np.int32)
    obj = np.empty(n_max, dtype=np.float64)
    n = c_int32()
    _check(lib().spec_select_draft_count(model.handle, len(lens), p_lens, p_offs, p_pars,
                                         w.ctypes.data_as(POINTER(c_float)), n_max, patience,
                                         ctypes.byref(n), sel.ctypes.data_as(POINTER(c_int32)),
                                         obj.ctypes.data_as(POINTER(ctypes.c_double))))
    return n.value, sel, obj


def spec_profile_begin(kernel_class, max_launches):
    if kernel_class == "transfer":
        k = TRANSFER_CLASS
    else:
        k = KERNEL_CLASS[kernel_class] if isinstance(kernel_class, str) else int(kernel_class)
    _check(lib().spec_profile_begin(k, max_launches))


def spec_profile_end():
    ms, n = c_float(), c_int32()
    _check(lib().spec_profile_end(ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
