// Host side of the specverify C ABI: argument validation, per-call planning
// (per-sample descriptors, split-KV attention work list), workspace carving,
// one staged host-to-device upload per call and the launch sequence of the
// verify step.  Every step of the computation itself runs in the HIP kernels.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <string>
#include <vector>

#include "common.h"
#include "specverify.h"

#define SPEC_API extern "C" __attribute__((visibility("default")))

using namespace spec;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(SPEC_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)               \
  do {                                    \
    hipError_t e_ = (expr);               \
    if (e_ != hipSuccess) return hip_fail(e_, what); \
  } while (0)

constexpr size_t kAlign = 256;
constexpr int kPartCap = 8192;          // split-KV partial tiles per call
constexpr int kTargetSlots = 512;       // attention CU slots aimed for (two rounds of 256 CUs)
constexpr int kMinChunk = 64;           // keys per split, lower bound
constexpr int kSmallChunk = 256;        // small calls: chunks of 64-key multiples up to this
constexpr int kMaxSplits = 64;          // key ranges per row tile (combine kernel's table)

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool config_ok(const spec_model_config* c, std::string* why) {
  char buf[256];
  auto bad = [&](const char* m) {
    snprintf(buf, sizeof buf, "unsupported model shape: %s", m);
    *why = buf;
    return false;
  };
  if (c->n_layers < 1 || c->hidden < 1 || c->n_heads < 1 || c->n_kv_heads < 1 || c->ffn < 1 ||
      c->vocab < 1 || c->head_dim < 1)
    return bad("non-positive dimension");
  if (c->head_dim != 64 && c->head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c->n_heads % c->n_kv_heads) return bad("n_heads must be a multiple of n_kv_heads");
  if (c->hidden % 128) return bad("hidden must be a multiple of 128");
  if ((c->n_heads * c->head_dim) % 128) return bad("n_heads*head_dim must be a multiple of 128");
  if ((c->n_kv_heads * c->head_dim) % 128)
    return bad("n_kv_heads*head_dim must be a multiple of 128");
  if (c->ffn % 128) return bad("ffn must be a multiple of 128");
  if (c->vocab % 128) return bad("vocab must be a multiple of 128");
  if (!(c->rope_theta > 0.f) || !(c->rms_eps >= 0.f)) return bad("rope_theta/rms_eps");
  return true;
}

bool same_config(const spec_model_config* a, const spec_model_config* b) {
  return a->n_layers == b->n_layers && a->hidden == b->hidden && a->n_heads == b->n_heads &&
         a->n_kv_heads == b->n_kv_heads && a->head_dim == b->head_dim && a->ffn == b->ffn &&
         a->vocab == b->vocab;
}

size_t sample_bytes(const spec_model_config* c, int32_t cap) {
  return align_up((size_t)c->n_layers * 2 * c->n_kv_heads * (size_t)cap * c->head_dim * 2);
}

// Workspace carving; every region 256-byte aligned.
struct WsLayout {
  size_t blob, toks, anc, rope, x, h, q, o, act, part_o, part_ml, lm_val, lm_idx, argmax, splitk,
      logits, resid, total;
  size_t blob_bytes;
};

int64_t max_row_tiles(const spec_model_config* c, int64_t max_batch, int64_t max_tokens) {
  const int64_t G = c->n_heads / c->n_kv_heads;
  return (int64_t)c->n_kv_heads * ((max_tokens * G + 31) / 32 + max_batch);
}

WsLayout ws_layout(const spec_model_config* c, int64_t max_batch, int64_t max_tokens,
                   bool sampling = false) {
  WsLayout L{};
  // attention items: one per row tile and split, then padded per XCD (at most 8x)
  const int64_t items = 8 * (max_row_tiles(c, max_batch, max_tokens) + kPartCap);
  L.blob_bytes = align_up(max_batch * sizeof(SampleInfo)) + 2 * align_up(max_tokens * 4) +
                 align_up(items * sizeof(AttnItem)) + 2 * kAlign +  // narrow + two wide lists
                 align_up(kPartCap * sizeof(CombineItem));
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off += align_up(bytes);
    return at;
  };
  const size_t nq_hd = (size_t)c->n_heads * c->head_dim;
  L.blob = take(L.blob_bytes);
  L.toks = take(max_tokens * sizeof(TokInfo));
  L.anc = take(max_tokens * 8 * kAncWords);
  L.rope = take(max_tokens * (size_t)(c->head_dim / 2) * 8);
  L.x = take(max_tokens * (size_t)c->hidden * 4);
  L.h = take(max_tokens * (size_t)c->hidden * 2);
  L.q = take(max_tokens * nq_hd * 2);
  L.o = take(max_tokens * nq_hd * 2);
  L.act = take(max_tokens * (size_t)c->ffn * 2);
  L.part_o = take((size_t)kPartCap * 32 * c->head_dim * 2);
  L.part_ml = take((size_t)kPartCap * 32 * 2 * 4);
  L.lm_val = take(max_tokens * (size_t)(c->vocab / 64) * 4);
  L.lm_idx = take(max_tokens * (size_t)(c->vocab / 64) * 4);
  L.argmax = take(max_tokens * 4);
  L.splitk = take(gemm_partial_bytes());
  if (sampling) {   // speculative sampling: fp32 logits, node decisions, fp64 residual rows
    L.logits = take(max_tokens * (size_t)c->vocab * 4);
    L.resid = take(sample_accept_scratch((int)max_batch, (int)max_tokens, c->vocab));
  }
  L.total = off;
  return L;
}

// Process-wide kernel timing state (measurement only).
struct Profiler {
  bool on = false;
  int kind = -1, max = 0, count = 0;
  std::vector<hipEvent_t> ev;
} g_prof;

template <class F>
hipError_t timed(int kind, hipStream_t s, F&& fn) {
  const bool rec = g_prof.on && g_prof.kind == kind && g_prof.count < g_prof.max;
  if (rec) {
    const hipError_t e = hipEventRecord(g_prof.ev[2 * g_prof.count], s);
    if (e != hipSuccess) return e;
  }
  const hipError_t e = fn();
  if (rec) {
    const hipError_t e2 = hipEventRecord(g_prof.ev[2 * g_prof.count + 1], s);
    ++g_prof.count;
    if (e2 != hipSuccess) return e2;
  }
  return e;
}

}  // namespace

// Library-owned part of a KV pool: capacities, block offsets and a two-slot
// pinned staging ring for the per-call host->device uploads.
struct spec_kv {
  spec_model_config cfg;
  int32_t n = 0;
  std::vector<int32_t> cap;
  std::vector<int64_t> base;     // element offsets of the sample blocks
  bf16* pool = nullptr;
  size_t bytes = 0;
  size_t ctl_off = 0;            // byte offset of the control area (commit descriptors)
  struct Slot {
    void* host = nullptr;
    size_t size = 0;
    hipEvent_t ev = nullptr;
    bool pending = false;
  } slots[2];
  int next = 0;
};

namespace {

// Copy `bytes` of `src` to device `dst` through the next pinned staging slot.
int stage_upload(spec_kv* kv, const void* src, size_t bytes, void* dst, hipStream_t s) {
  spec_kv::Slot& sl = kv->slots[kv->next];
  kv->next ^= 1;
  if (sl.pending) {
    HIP_TRY(hipEventSynchronize(sl.ev), "staging wait");
    sl.pending = false;
  }
  if (sl.ev == nullptr) HIP_TRY(hipEventCreateWithFlags(&sl.ev, hipEventDisableTiming), "event");
  if (sl.size < bytes) {
    if (sl.host) HIP_TRY(hipHostFree(sl.host), "free staging");
    sl.host = nullptr;
    sl.size = 0;
    const size_t want = std::max(bytes, (size_t)1 << 20);
    HIP_TRY(hipHostMalloc(&sl.host, want, hipHostMallocDefault), "pinned staging");
    sl.size = want;
  }
  memcpy(sl.host, src, bytes);
  HIP_TRY(hipMemcpyAsync(dst, sl.host, bytes, hipMemcpyHostToDevice, s), "upload");
  HIP_TRY(hipEventRecord(sl.ev, s), "staging event");
  sl.pending = true;
  return SPEC_OK;
}

int check_samples(const spec_kv* kv, int32_t batch, const int32_t* ids) {
  std::vector<char> seen(kv->n, 0);
  for (int b = 0; b < batch; ++b) {
    const int id = ids[b];
    if (id < 0 || id >= kv->n) return fail(SPEC_ERR_INVALID, "sample_ids[%d] = %d out of range", b, id);
    if (seen[id]) return fail(SPEC_ERR_INVALID, "sample id %d appears twice", id);
    seen[id] = 1;
  }
  return SPEC_OK;
}

}  // namespace

SPEC_API const char* spec_last_error(void) { return g_err.c_str(); }

namespace spec {
int set_error(int code, const char* msg) {
  g_err = msg;
  return code;
}
}  // namespace spec

SPEC_API size_t spec_kv_bytes(const spec_model_config* cfg, int32_t n_samples,
                              const int32_t* capacity) {
  std::string why;
  if (!cfg || !capacity || n_samples < 1 || !config_ok(cfg, &why)) return 0;
  size_t total = 0;
  for (int i = 0; i < n_samples; ++i) {
    if (capacity[i] < 1) return 0;
    total += sample_bytes(cfg, capacity[i]);
  }
  return total + align_up((size_t)n_samples * sizeof(SampleInfo));
}

SPEC_API int spec_kv_alloc(const spec_model_config* cfg, int32_t n_samples,
                           const int32_t* capacity, void* device_buf, size_t buf_bytes,
                           spec_kv** out) {
  g_err.clear();
  if (!cfg || !capacity || !device_buf || !out) return fail(SPEC_ERR_INVALID, "null argument");
  if (n_samples < 1) return fail(SPEC_ERR_INVALID, "n_samples must be >= 1");
  std::string why;
  if (!config_ok(cfg, &why)) return fail(SPEC_ERR_UNSUPPORTED, "%s", why.c_str());
  if ((uintptr_t)device_buf % kAlign) return fail(SPEC_ERR_INVALID, "device_buf not 256-byte aligned");
  for (int i = 0; i < n_samples; ++i)
    if (capacity[i] < 1) return fail(SPEC_ERR_INVALID, "capacity[%d] = %d", i, capacity[i]);
  const size_t need = spec_kv_bytes(cfg, n_samples, capacity);
  if (buf_bytes < need)
    return fail(SPEC_ERR_CAPACITY, "KV buffer holds %zu bytes, needs %zu", buf_bytes, need);
  spec_kv* kv = new spec_kv;
  kv->cfg = *cfg;
  kv->n = n_samples;
  kv->cap.assign(capacity, capacity + n_samples);
  kv->base.resize(n_samples);
  size_t off = 0;
  for (int i = 0; i < n_samples; ++i) {
    kv->base[i] = (int64_t)(off / 2);
    off += sample_bytes(cfg, capacity[i]);
  }
  kv->ctl_off = off;
  kv->pool = (bf16*)device_buf;
  kv->bytes = buf_bytes;
  *out = kv;
  return SPEC_OK;
}

SPEC_API int spec_kv_free(spec_kv* kv) {
  if (!kv) return fail(SPEC_ERR_INVALID, "null handle");
  int rc = SPEC_OK;
  for (auto& sl : kv->slots) {
    if (sl.pending && hipEventSynchronize(sl.ev) != hipSuccess) rc = SPEC_ERR_HIP;
    if (sl.ev) (void)hipEventDestroy(sl.ev);
    if (sl.host) (void)hipHostFree(sl.host);
  }
  delete kv;
  return rc;
}

SPEC_API int spec_kv_sample_layout(const spec_kv* kv, int32_t sample, int64_t* byte_offset,
                                   int32_t* capacity) {
  if (!kv || !byte_offset || !capacity) return fail(SPEC_ERR_INVALID, "null argument");
  if (sample < 0 || sample >= kv->n) return fail(SPEC_ERR_INVALID, "sample %d out of range", sample);
  *byte_offset = kv->base[sample] * 2;
  *capacity = kv->cap[sample];
  return SPEC_OK;
}

SPEC_API size_t spec_workspace_bytes(const spec_model_config* cfg, int32_t max_batch,
                                     int32_t max_tokens) {
  std::string why;
  if (!cfg || max_batch < 1 || max_tokens < max_batch || !config_ok(cfg, &why)) return 0;
  return ws_layout(cfg, max_batch, max_tokens).total;
}

namespace {

int verify_impl(const spec_model_config* cfg, const spec_weights* w, spec_kv* kv, int32_t batch,
                const int32_t* sample_ids, const int32_t* tree_offsets, const int32_t* tree_tokens,
                const int32_t* tree_parents, const int32_t* seq_lens, void* workspace,
                size_t ws_bytes, void* stream, const spec_sampling* samp, int32_t* accepted_len,
                int32_t* next_token, int32_t* accepted_nodes, const spec_debug* dbg,
                bool noalloc = false) {
  // ---- validation (no side effects) ----
  if (!cfg || !w || !kv || !sample_ids || !tree_offsets || !tree_tokens || !tree_parents ||
      !seq_lens || (!workspace && !noalloc) || !accepted_len || !next_token || !accepted_nodes)
    return fail(SPEC_ERR_INVALID, "null argument");
  std::string why;
  if (!config_ok(cfg, &why)) return fail(SPEC_ERR_UNSUPPORTED, "%s", why.c_str());
  if (!same_config(cfg, &kv->cfg)) return fail(SPEC_ERR_INVALID, "config differs from the KV pool's");
  if (batch < 1) return fail(SPEC_ERR_INVALID, "batch must be >= 1");
  if (!w->tok_embed || !w->final_norm || !w->lm_head || !w->attn_norm || !w->wq || !w->wk ||
      !w->wv || !w->wo || !w->ffn_norm || !w->w_gate || !w->w_up || !w->w_down)
    return fail(SPEC_ERR_INVALID, "null weight pointer");
  for (int l = 0; l < cfg->n_layers; ++l)
    if (!w->attn_norm[l] || !w->wq[l] || !w->wk[l] || !w->wv[l] || !w->wo[l] || !w->ffn_norm[l] ||
        !w->w_gate[l] || !w->w_up[l] || !w->w_down[l])
      return fail(SPEC_ERR_INVALID, "null weight pointer in layer %d", l);
  if (int rc = check_samples(kv, batch, sample_ids)) return rc;
  if (tree_offsets[0] != 0) return fail(SPEC_ERR_TREE, "tree_offsets[0] must be 0");
  for (int b = 0; b < batch; ++b) {
    const int T = tree_offsets[b + 1] - tree_offsets[b];
    if (T < 1 || T > SPEC_MAX_TREE)
      return fail(T < 1 ? SPEC_ERR_TREE : SPEC_ERR_UNSUPPORTED, "sample %d has %d tree nodes", b, T);
    const int S = seq_lens[b];
    if (S < 0) return fail(SPEC_ERR_INVALID, "seq_lens[%d] = %d", b, S);
    if ((int64_t)S + T > kv->cap[sample_ids[b]])
      return fail(SPEC_ERR_CAPACITY, "sample %d: %d committed + %d nodes exceed capacity %d", b, S,
                  T, kv->cap[sample_ids[b]]);
    const int t0 = tree_offsets[b];
    if (tree_parents[t0] != -1) return fail(SPEC_ERR_TREE, "sample %d: root parent must be -1", b);
    for (int i = 0; i < T; ++i) {
      const int tok = tree_tokens[t0 + i];
      if (tok < 0 || tok >= cfg->vocab)
        return fail(SPEC_ERR_TREE, "sample %d node %d: token %d out of range", b, i, tok);
      if (i > 0) {
        const int p = tree_parents[t0 + i];
        if (p < 0 || p >= i)
          return fail(SPEC_ERR_TREE, "sample %d node %d: parent %d not before the node", b, i, p);
      }
    }
  }
  const bool sampled = samp && samp->temperature > 0.f;
  if (samp) {
    if (!(samp->temperature >= 0.f) || !std::isfinite(samp->temperature))
      return fail(SPEC_ERR_INVALID, "temperature must be finite and >= 0");
    if (samp->eos_token < -1 || samp->eos_token >= cfg->vocab)
      return fail(SPEC_ERR_INVALID, "eos_token %d out of range", samp->eos_token);
    if (sampled && (!samp->draft_probs || !samp->uniforms))
      return fail(SPEC_ERR_INVALID, "sampling needs draft_probs and uniforms");
  }
  const int N = tree_offsets[batch];
  const size_t need = ws_layout(cfg, batch, N, sampled).total;
  if (noalloc && need > SPEC_NOALLOC_SCRATCH_BYTES)
    return fail(SPEC_ERR_WORKSPACE,
                "%d samples with %d tree nodes need %zu bytes of workspace, more than the %zu "
                "bytes of spec_verify_noalloc's static scratch",
                batch, N, need, (size_t)SPEC_NOALLOC_SCRATCH_BYTES);
  if (noalloc) {
    HIP_TRY(noalloc_scratch(&workspace), "static scratch lookup");
    ws_bytes = SPEC_NOALLOC_SCRATCH_BYTES;
  }
  if (ws_bytes < need) return fail(SPEC_ERR_WORKSPACE, "workspace %zu bytes, needs %zu", ws_bytes, need);

  // ---- planning ----
  const int L = cfg->n_layers, H = cfg->hidden, nq = cfg->n_heads, nkv = cfg->n_kv_heads;
  const int hd = cfg->head_dim, G = nq / nkv, F = cfg->ffn, V = cfg->vocab;
  const WsLayout ly = ws_layout(cfg, batch, N, sampled);
  char* ws = (char*)workspace;
  hipStream_t s = (hipStream_t)stream;

  std::vector<SampleInfo> si(batch);
  for (int b = 0; b < batch; ++b) {
    const int id = sample_ids[b];
    si[b] = SampleInfo{kv->base[id], kv->cap[id], seq_lens[b], tree_offsets[b],
                       tree_offsets[b + 1] - tree_offsets[b], 0, 0};
  }
  // Split-KV plan.  A row tile is 32 query rows of one (sample, kv head).  A
  // (sample, kv head) with one tile gets narrow items (2 waves dealing the
  // keys among themselves, two work-groups per CU); 2-4 tiles get one 4-wave
  // wide group (two per CU); more get 8-wave groups of 8 tiles (one per CU).
  // Every (sample, kv head) key range is cut into chunks of `chunk` keys,
  // sized so that the whole call is about kTargetSlots chunk-sized CU
  // occupancies (a few per CU, for balance), with at most kMaxSplits chunks
  // per range and at most kPartCap partial states.
  auto tiles_of = [&](int b) { return (si[b].ntok * G + 31) / 32; };
  auto keys_of = [&](int b) { return (int64_t)si[b].seq_len + si[b].ntok; };
  // Cost weight of one chunk's work-groups: their CU occupancy, except that a
  // narrow item counts as a whole CU (measured: sizing its chunks as half a
  // CU's worth, i.e. twice as many splits, is slower).
  auto cu_weight = [&](int tiles) {
    return tiles == 1 ? 1.0 : tiles <= 4 ? 0.5 : (double)((tiles + 7) / 8);
  };
  int64_t max_keys = 0;
  double work = 0.0;
  for (int b = 0; b < batch; ++b) {
    max_keys = std::max(max_keys, keys_of(b));
    work += (double)nkv * keys_of(b) * cu_weight(tiles_of(b));
  }
  auto part_slots = [&](int64_t c) {
    int64_t slots = 0;
    for (int b = 0; b < batch; ++b) {
      const int64_t ns = (keys_of(b) + c - 1) / c;
      if (ns > 1) slots += ns * nkv * tiles_of(b);
    }
    return slots;
  };
  // Chunk length: a multiple of 128 keys.  A small call (under kSmallChunk
  // keys of work per slot at that target) instead aims at one round of the
  // 256 CUs, in multiples of 64 keys between kMinChunk and kSmallChunk: a
  // single short sample gets more, shorter chunks (each work-group's block
  // chain is serial), and a few samples with multi-tile trees do not spill
  // into a second round.  Measured per 32-layer step against a 256-key floor:
  // batch 1, 1.1K keys, attention 0.50 -> 0.44 ms; against the two-round
  // target at 64-key granularity: batch 4 x 16 nodes 5.75 -> 5.48 ms.
  auto round128 = [](int64_t x) { return (x + 127) / 128 * 128; };
  auto round64 = [](int64_t x) { return (x + 63) / 64 * 64; };
  const int64_t min_split = (max_keys + kMaxSplits - 1) / kMaxSplits;
  const int64_t want = std::max<int64_t>(min_split, (int64_t)(work / kTargetSlots));
  int64_t chunk = round128(want);
  if (want < kSmallChunk)
    chunk = std::min<int64_t>(kSmallChunk, round64(std::max<int64_t>({kMinChunk, min_split, (int64_t)(work / 256)})));
  while (part_slots(chunk) > kPartCap) chunk += 128;    // terminates: one chunk per range has none
  // Work items.  Split key ranges write their partial states to per-tile
  // slots part + tile * ns + split.
  std::vector<AttnItem> items, wide4, wide8;
  std::vector<CombineItem> comb;
  int part = 0;
  for (int b = 0; b < batch; ++b) {
    const int keys = (int)keys_of(b);
    const int ns = (int)((keys + chunk - 1) / chunk);
    const int tiles = tiles_of(b);
    for (int g = 0; g < nkv; ++g) {
      for (int t = 0; t < tiles && ns > 1; ++t)
        comb.push_back(CombineItem{b, g, t * 32, ns, part + t * ns, 0, 0, 0});
      for (int k = 0; k < ns; ++k) {
        const int k0 = (int)(k * chunk), k1 = (int)std::min<int64_t>(keys, (k + 1) * chunk);
        const int p = ns > 1 ? part + k : 0;
        if (tiles == 1)
          items.push_back(AttnItem{b, g, 0, k0, k1, ns, p, 0});
        else if (tiles <= 4)
          wide4.push_back(AttnItem{b, g, 0, k0, k1, ns, p, 0});
        else
          for (int rg = 0; rg < (tiles + 7) / 8; ++rg)
            wide8.push_back(AttnItem{b, g, rg * 256, k0, k1, ns, ns > 1 ? p + rg * 8 * ns : 0, 0});
      }
      if (ns > 1) part += ns * tiles;
    }
  }
  // Longest-first per XCD: a kernel hands XCD x the items [x*per, (x+1)*per)
  // in order.  Deal the groups of items that share a key range (adjacent, so
  // they meet in one XCD's L2), longest first, to the XCD with the least work
  // so far; pad every XCD's list to `per` with empty items (sample -1).
  auto deal = [](std::vector<AttnItem>& list) {
    struct Group { size_t first, count; int64_t work; };
    std::vector<Group> groups;
    for (size_t i = 0; i < list.size();) {
      size_t j = i;
      while (j < list.size() && list[j].sample == list[i].sample && list[j].kvh == list[i].kvh &&
             list[j].key0 == list[i].key0)
        ++j;
      groups.push_back(Group{i, j - i, (int64_t)(list[i].key1 - list[i].key0) * (int64_t)(j - i)});
      i = j;
    }
    std::stable_sort(groups.begin(), groups.end(),
                     [](const Group& x, const Group& y) { return x.work > y.work; });
    std::vector<AttnItem> xcd[8];
    int64_t load[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    for (const Group& gp : groups) {
      const int x = (int)(std::min_element(load, load + 8) - load);
      load[x] += gp.work;
      xcd[x].insert(xcd[x].end(), list.begin() + gp.first, list.begin() + gp.first + gp.count);
    }
    size_t per = 0;
    for (auto& v : xcd) per = std::max(per, v.size());
    std::vector<AttnItem> dealt;
    dealt.reserve(per * 8);
    for (auto& v : xcd) {
      dealt.insert(dealt.end(), v.begin(), v.end());
      dealt.resize(dealt.size() + (per - v.size()), AttnItem{-1, 0, 0, 0, 0, 1, 0, 0});
    }
    list.swap(dealt);
  };
  deal(items);
  deal(wide4);
  deal(wide8);

  // ---- one upload of the per-call descriptors ----
  const size_t o_si = 0;
  const size_t o_tok = align_up(batch * sizeof(SampleInfo));
  const size_t o_par = o_tok + align_up((size_t)N * 4);
  const size_t o_items = o_par + align_up((size_t)N * 4);
  const size_t o_wide4 = o_items + align_up(items.size() * sizeof(AttnItem));
  const size_t o_wide8 = o_wide4 + align_up(wide4.size() * sizeof(AttnItem));
  const size_t o_comb = o_wide8 + align_up(wide8.size() * sizeof(AttnItem));
  const size_t blob_bytes = o_comb + comb.size() * sizeof(CombineItem);
  std::vector<char> blob(blob_bytes, 0);
  memcpy(blob.data() + o_si, si.data(), batch * sizeof(SampleInfo));
  memcpy(blob.data() + o_tok, tree_tokens, (size_t)N * 4);
  memcpy(blob.data() + o_par, tree_parents, (size_t)N * 4);
  memcpy(blob.data() + o_items, items.data(), items.size() * sizeof(AttnItem));
  if (!wide4.empty()) memcpy(blob.data() + o_wide4, wide4.data(), wide4.size() * sizeof(AttnItem));
  if (!wide8.empty()) memcpy(blob.data() + o_wide8, wide8.data(), wide8.size() * sizeof(AttnItem));
  if (!comb.empty()) memcpy(blob.data() + o_comb, comb.data(), comb.size() * sizeof(CombineItem));
  if (noalloc)   // no pinned staging: a copy from pageable memory, done before the call returns
    HIP_TRY(hipMemcpyAsync(ws + ly.blob, blob.data(), blob_bytes, hipMemcpyHostToDevice, s),
            "upload");
  else if (int rc = stage_upload(kv, blob.data(), blob_bytes, ws + ly.blob, s))
    return rc;

  const SampleInfo* d_si = (const SampleInfo*)(ws + ly.blob + o_si);
  const int32_t* d_tok = (const int32_t*)(ws + ly.blob + o_tok);
  const int32_t* d_par = (const int32_t*)(ws + ly.blob + o_par);
  const AttnItem* d_items = (const AttnItem*)(ws + ly.blob + o_items);
  const AttnItem* d_wide4 = (const AttnItem*)(ws + ly.blob + o_wide4);
  const AttnItem* d_wide8 = (const AttnItem*)(ws + ly.blob + o_wide8);
  const CombineItem* d_comb = (const CombineItem*)(ws + ly.blob + o_comb);
  TokInfo* d_toks = (TokInfo*)(ws + ly.toks);
  uint64_t* d_anc = (uint64_t*)(ws + ly.anc);
  float2* d_rope = (float2*)(ws + ly.rope);
  float* d_x = (float*)(ws + ly.x);
  bf16* d_h = (bf16*)(ws + ly.h);
  bf16* d_q = (bf16*)(ws + ly.q);
  bf16* d_o = (bf16*)(ws + ly.o);
  bf16* d_act = (bf16*)(ws + ly.act);
  float* d_lmv = (float*)(ws + ly.lm_val);
  int32_t* d_lmi = (int32_t*)(ws + ly.lm_idx);
  int32_t* d_arg = (int32_t*)(ws + ly.argmax);

  const spec_debug nodbg{};
  const spec_debug& D = dbg ? *dbg : nodbg;

  // ---- the step ----
  HIP_TRY(launch_tree_meta(d_si, batch, d_par, d_toks, d_anc, D.depth, D.pos, D.anc, s), "tree meta");
  HIP_TRY(launch_rope_table(d_toks, N, hd, cfg->rope_theta, d_rope, s), "rope table");
  HIP_TRY(launch_embed(d_tok, (const bf16*)w->tok_embed, d_x, N, H, s), "embed");

  GemmArgs ga{};
  ga.M = N;
  ga.samples = d_si;
  ga.toks = d_toks;
  ga.kv_pool = kv->pool;
  ga.n_kv_heads = nkv;
  ga.head_dim = hd;
  ga.rope_cs = d_rope;
  ga.partial = (float*)(ws + ly.splitk);
  AttnArgs aa{};
  aa.q = d_q;
  aa.kv_pool = kv->pool;
  aa.samples = d_si;
  aa.toks = d_toks;
  aa.anc = d_anc;
  aa.items = d_items;
  aa.n_items = (int)items.size();
  aa.wide = d_wide4;
  aa.n_wide = (int)wide4.size();
  aa.wide8 = d_wide8;
  aa.n_wide8 = (int)wide8.size();
  aa.part_o = (f16*)(ws + ly.part_o);
  aa.part_ml = (float*)(ws + ly.part_ml);
  aa.out = d_o;
  aa.n_heads = nq;
  aa.n_kv_heads = nkv;
  aa.head_dim = hd;
  aa.comb = d_comb;
  aa.n_comb = (int)comb.size();

  // Every RMSNorm after the first follows a residual product (O or down
  // projection); when that product is split over K the norm runs inside its
  // split-K reduction, otherwise on its own.
  auto resid_then_norm = [&](int kind, GemmArgs g, const void* gain, const char* what) -> int {
    bool fused = false;
    g.norm_gain = (const bf16*)gain;
    g.norm_out = d_h;
    g.norm_eps = cfg->rms_eps;
    g.norm_done = &fused;
    HIP_TRY(timed(kind, s, [&] { return launch_gemm(EPI_RESID, g, s); }), what);
    if (!fused) HIP_TRY(launch_rmsnorm(d_x, (const bf16*)gain, d_h, N, H, cfg->rms_eps, s), "rmsnorm");
    return SPEC_OK;
  };
  HIP_TRY(launch_rmsnorm(d_x, (const bf16*)w->attn_norm[0], d_h, N, H, cfg->rms_eps, s), "rmsnorm");
  for (int l = 0; l < L; ++l) {
    GemmArgs g = ga;
    g.A = d_h;
    g.K = H;
    g.B0 = (const bf16*)w->wq[l];
    g.B1 = (const bf16*)w->wk[l];
    g.B2 = (const bf16*)w->wv[l];
    g.n0 = nq * hd;
    g.n1 = g.n2 = nkv * hd;
    g.N = g.n0 + g.n1 + g.n2;
    g.q_out = d_q;
    g.layer = l;
    HIP_TRY(timed(SPEC_K_GEMM_QKV, s, [&] { return launch_gemm(EPI_QKV, g, s); }), "qkv gemm");
    aa.layer = l;
    HIP_TRY(timed(SPEC_K_ATTENTION, s, [&] { return launch_attention(aa, s); }), "attention");
    g = ga;
    g.A = d_o;
    g.K = nq * hd;
    g.B0 = (const bf16*)w->wo[l];
    g.n0 = g.N = H;
    g.x = d_x;
    if (int rc = resid_then_norm(SPEC_K_GEMM_O, g, w->ffn_norm[l], "o gemm")) return rc;
    g = ga;
    g.A = d_h;
    g.K = H;
    g.B0 = (const bf16*)w->w_gate[l];
    g.B1 = (const bf16*)w->w_up[l];
    g.n0 = g.n1 = F;
    g.N = 2 * F;
    g.act_out = d_act;
    HIP_TRY(timed(SPEC_K_GEMM_GATE_UP, s, [&] { return launch_gemm(EPI_GATE_UP, g, s); }), "gate/up gemm");
    g = ga;
    g.A = d_act;
    g.K = F;
    g.B0 = (const bf16*)w->w_down[l];
    g.n0 = g.N = H;
    g.x = d_x;
    const void* next_norm = l + 1 < L ? w->attn_norm[l + 1] : w->final_norm;
    if (int rc = resid_then_norm(SPEC_K_GEMM_DOWN, g, next_norm, "down gemm")) return rc;
  }
  {
    GemmArgs g = ga;
    g.A = d_h;
    g.K = H;
    g.B0 = (const bf16*)w->lm_head;
    g.n0 = g.N = V;
    g.part_val = d_lmv;
    g.part_idx = d_lmi;
    g.logits = D.logits ? D.logits : sampled ? (float*)(ws + ly.logits) : nullptr;
    HIP_TRY(timed(SPEC_K_LM_HEAD, s, [&] { return launch_gemm(EPI_ARGMAX, g, s); }), "lm head");
  }
  HIP_TRY(launch_argmax_reduce(d_lmv, d_lmi, N, gemm_parts(V, N, H), d_arg, D.argmax, s), "argmax");
  if (sampled) {
    const float* logits = D.logits ? D.logits : (const float*)(ws + ly.logits);
    HIP_TRY(timed(SPEC_K_ACCEPT, s, [&] {
              return launch_sample_accept(d_si, batch, N, d_toks, d_tok, d_par, logits,
                                          samp->draft_probs, samp->uniforms, V, samp->temperature,
                                          samp->eos_token, ws + ly.resid, accepted_len, next_token,
                                          accepted_nodes, s);
            }),
            "sampled accept");
  } else if (samp && samp->eos_token >= 0) {
    HIP_TRY(timed(SPEC_K_ACCEPT, s, [&] {
              return launch_accept_eos(d_si, batch, d_tok, d_par, d_toks, d_arg, samp->eos_token,
                                       accepted_len, next_token, accepted_nodes, s);
            }),
            "accept");
  } else {
    HIP_TRY(timed(SPEC_K_ACCEPT, s, [&] {
              return launch_accept(d_si, batch, d_tok, d_par, d_toks, d_arg, accepted_len,
                                   next_token, accepted_nodes, s);
            }),
            "accept");
  }
  return SPEC_OK;
}

}  // namespace

SPEC_API int spec_verify(const spec_model_config* cfg, const spec_weights* w, spec_kv* kv,
                         int32_t batch, const int32_t* sample_ids, const int32_t* tree_offsets,
                         const int32_t* tree_tokens, const int32_t* tree_parents,
                         const int32_t* seq_lens, void* workspace, size_t ws_bytes, void* stream,
                         int32_t* accepted_len, int32_t* next_token, int32_t* accepted_nodes,
                         const spec_debug* dbg) {
  g_err.clear();
  return verify_impl(cfg, w, kv, batch, sample_ids, tree_offsets, tree_tokens, tree_parents,
                     seq_lens, workspace, ws_bytes, stream, nullptr, accepted_len, next_token,
                     accepted_nodes, dbg);
}

SPEC_API size_t spec_workspace_bytes_sampled(const spec_model_config* cfg, int32_t max_batch,
                                             int32_t max_tokens) {
  std::string why;
  if (!cfg || max_batch < 1 || max_tokens < max_batch || !config_ok(cfg, &why)) return 0;
  return ws_layout(cfg, max_batch, max_tokens, true).total;
}

SPEC_API int spec_verify_sampled(const spec_model_config* cfg, const spec_weights* w,
                                 spec_kv* kv, int32_t batch, const int32_t* sample_ids,
                                 const int32_t* tree_offsets, const int32_t* tree_tokens,
                                 const int32_t* tree_parents, const int32_t* seq_lens,
                                 void* workspace, size_t ws_bytes, void* stream,
                                 const spec_sampling* samp, int32_t* accepted_len,
                                 int32_t* next_token, int32_t* accepted_nodes,
                                 const spec_debug* dbg) {
  g_err.clear();
  if (!samp) return fail(SPEC_ERR_INVALID, "null sampling parameters");
  return verify_impl(cfg, w, kv, batch, sample_ids, tree_offsets, tree_tokens, tree_parents,
                     seq_lens, workspace, ws_bytes, stream, samp, accepted_len, next_token,
                     accepted_nodes, dbg);
}

SPEC_API int spec_verify_noalloc(const spec_model_config* cfg, const spec_weights* w,
                                 spec_kv* kv, int32_t batch, const int32_t* sample_ids,
                                 const int32_t* tree_offsets, const int32_t* tree_tokens,
                                 const int32_t* tree_parents, const int32_t* seq_lens,
                                 void* stream, int32_t* accepted_len, int32_t* next_token,
                                 int32_t* accepted_nodes, const spec_debug* dbg) {
  g_err.clear();
  return verify_impl(cfg, w, kv, batch, sample_ids, tree_offsets, tree_tokens, tree_parents,
                     seq_lens, nullptr, 0, stream, nullptr, accepted_len, next_token,
                     accepted_nodes, dbg, true);
}

SPEC_API int spec_kv_commit(spec_kv* kv, int32_t batch, const int32_t* sample_ids,
                            const int32_t* seq_lens, const int32_t* accepted_len,
                            const int32_t* accepted_nodes, int32_t* new_seq_lens, void* stream) {
  g_err.clear();
  if (!kv || !sample_ids || !seq_lens || !accepted_len || !accepted_nodes || !new_seq_lens)
    return fail(SPEC_ERR_INVALID, "null argument");
  if (batch < 1 || batch > kv->n) return fail(SPEC_ERR_INVALID, "batch %d out of range", batch);
  if (int rc = check_samples(kv, batch, sample_ids)) return rc;
  std::vector<SampleInfo> si(batch);
  for (int b = 0; b < batch; ++b) {
    const int id = sample_ids[b];
    if (seq_lens[b] < 0 || seq_lens[b] >= kv->cap[id])
      return fail(SPEC_ERR_CAPACITY, "seq_lens[%d] = %d outside capacity %d", b, seq_lens[b], kv->cap[id]);
    si[b] = SampleInfo{kv->base[id], kv->cap[id], seq_lens[b], 0, SPEC_MAX_TREE, 0, 0};
  }
  hipStream_t s = (hipStream_t)stream;
  void* ctl = (char*)kv->pool + kv->ctl_off;
  if (int rc = stage_upload(kv, si.data(), batch * sizeof(SampleInfo), ctl, s)) return rc;
  const spec_model_config& c = kv->cfg;
  HIP_TRY(timed(SPEC_K_COMMIT, s, [&] {
            return launch_compact((const SampleInfo*)ctl, batch, kv->pool, c.n_layers,
                                  c.n_kv_heads, c.head_dim, accepted_len, accepted_nodes,
                                  new_seq_lens, s);
          }),
          "compact");
  return SPEC_OK;
}

namespace {

// Validate a transfer request and build its per-sample descriptors.
int transfer_plan(const spec_kv* kv, int32_t n, const int32_t* sample_ids, const int32_t* tok_begin,
                  const int32_t* tok_end, std::vector<MigrateInfo>* info, int64_t* wg_per_slab,
                  int64_t* tok_total) {
  if (!kv || !sample_ids || !tok_begin || !tok_end) return fail(SPEC_ERR_INVALID, "null argument");
  if (n < 1 || n > kv->n) return fail(SPEC_ERR_INVALID, "n %d out of range", n);
  if (int rc = check_samples(kv, n, sample_ids)) return rc;
  const spec_model_config& c = kv->cfg;
  info->resize(n);
  int64_t wg = 0, tok = 0;
  for (int j = 0; j < n; ++j) {
    const int id = sample_ids[j];
    if (tok_begin[j] < 0 || tok_end[j] < tok_begin[j] || tok_end[j] > kv->cap[id])
      return fail(SPEC_ERR_CAPACITY, "token range [%d, %d) of sample %d outside capacity %d",
                  tok_begin[j], tok_end[j], id, kv->cap[id]);
    const int count = tok_end[j] - tok_begin[j];
    const int64_t chunks = kv_transfer_chunks(count, c.head_dim);
    (*info)[j] = MigrateInfo{kv->base[id], kv->cap[id], tok_begin[j], count, (int32_t)tok,
                             (int32_t)wg, (int32_t)chunks};
    wg += chunks * c.n_kv_heads;
    tok += count;
    if (wg > 0x7fffffff || tok > 0x7fffffff) return fail(SPEC_ERR_INVALID, "transfer too large");
  }
  *wg_per_slab = wg;
  *tok_total = tok;
  return SPEC_OK;
}

int transfer(bool to_buffer, spec_kv* kv, int32_t n, const int32_t* sample_ids,
             const int32_t* tok_begin, const int32_t* tok_end, void* buf, size_t buf_bytes,
             void* stream) {
  g_err.clear();
  std::vector<MigrateInfo> info;
  int64_t wg = 0, tok = 0;
  if (int rc = transfer_plan(kv, n, sample_ids, tok_begin, tok_end, &info, &wg, &tok)) return rc;
  if (!buf) return fail(SPEC_ERR_INVALID, "null buffer");
  if ((uintptr_t)buf % 16) return fail(SPEC_ERR_INVALID, "buffer not 16-byte aligned");
  const spec_model_config& c = kv->cfg;
  const size_t need = (size_t)tok * c.n_layers * 2 * c.n_kv_heads * c.head_dim * 2;
  if (buf_bytes < need)
    return fail(SPEC_ERR_CAPACITY, "transfer buffer holds %zu bytes, needs %zu", buf_bytes, need);
  if (wg == 0) return SPEC_OK;
  hipStream_t s = (hipStream_t)stream;
  void* ctl = (char*)kv->pool + kv->ctl_off;
  if (int rc = stage_upload(kv, info.data(), n * sizeof(MigrateInfo), ctl, s)) return rc;
  HIP_TRY(timed(SPEC_K_TRANSFER, s, [&] {
            return launch_kv_transfer(to_buffer, (const MigrateInfo*)ctl, n, wg, (int)tok, kv->pool,
                                      (bf16*)buf, c.n_layers, c.n_kv_heads, c.head_dim, s);
          }),
          to_buffer ? "kv pack" : "kv unpack");
  return SPEC_OK;
}

}  // namespace

SPEC_API size_t spec_kv_transfer_bytes(const spec_kv* kv, int32_t n, const int32_t* tok_begin,
                                       const int32_t* tok_end) {
  if (!kv || !tok_begin || !tok_end || n < 1) return 0;
  size_t tok = 0;
  for (int j = 0; j < n; ++j) {
    if (tok_end[j] < tok_begin[j] || tok_begin[j] < 0) return 0;
    tok += (size_t)(tok_end[j] - tok_begin[j]);
  }
  const spec_model_config& c = kv->cfg;
  return tok * c.n_layers * 2 * c.n_kv_heads * c.head_dim * 2;
}

SPEC_API int spec_kv_pack(spec_kv* kv, int32_t n, const int32_t* sample_ids,
                          const int32_t* tok_begin, const int32_t* tok_end, void* buf,
                          size_t buf_bytes, void* stream) {
  return transfer(true, kv, n, sample_ids, tok_begin, tok_end, buf, buf_bytes, stream);
}

SPEC_API int spec_kv_unpack(spec_kv* kv, int32_t n, const int32_t* sample_ids,
                            const int32_t* tok_begin, const int32_t* tok_end, const void* buf,
                            size_t buf_bytes, void* stream) {
  return transfer(false, kv, n, sample_ids, tok_begin, tok_end, const_cast<void*>(buf), buf_bytes,
                  stream);
}

SPEC_API int spec_profile_begin(int32_t kernel_class, int32_t max_launches) {
  if (kernel_class < 0 || kernel_class >= SPEC_K_COUNT || max_launches < 1)
    return fail(SPEC_ERR_INVALID, "bad profile request");
  for (auto e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof.ev.assign(2 * (size_t)max_launches, nullptr);
  for (auto& e : g_prof.ev) HIP_TRY(hipEventCreate(&e), "profile event");
  g_prof.kind = kernel_class;
  g_prof.max = max_launches;
  g_prof.count = 0;
  g_prof.on = true;
  return SPEC_OK;
}

SPEC_API int spec_profile_end(float* total_ms, int32_t* launches) {
  if (!total_ms || !launches) return fail(SPEC_ERR_INVALID, "null argument");
  g_prof.on = false;
  float tot = 0.f;
  for (int i = 0; i < g_prof.count; ++i) {
    HIP_TRY(hipEventSynchronize(g_prof.ev[2 * i + 1]), "profile sync");
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, g_prof.ev[2 * i], g_prof.ev[2 * i + 1]), "profile elapsed");
    tot += ms;
  }
  *total_ms = tot;
  *launches = g_prof.count;
  for (auto e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof.ev.clear();
  g_prof.count = 0;
  return SPEC_OK;
}
