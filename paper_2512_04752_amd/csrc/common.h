// Shared device types, descriptors and launcher prototypes of the
// specverify library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "specverify.h"

namespace spec {

typedef __bf16 bf16;
typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(4))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) int i32x4;
typedef __attribute__((ext_vector_type(2))) int i32x2;
typedef _Float16 f16;
typedef __attribute__((ext_vector_type(4))) _Float16 f16x4;

constexpr int kMaxTree = SPEC_MAX_TREE;        // nodes per draft tree
constexpr int kAncWords = kMaxTree / 64;       // 64-bit words of a node's ancestor set
static_assert(kMaxTree % 64 == 0 && kAncWords == SPEC_ANC_WORDS, "ancestor words");

// A set of nodes of one tree held in registers: bit t % 64 of word t / 64.
// Four named words, picked by compare-and-select, so that the set never
// needs dynamic register indexing (which would put it in scratch memory).
struct NodeSet {
  uint64_t w0, w1, w2, w3;
  __device__ __forceinline__ void clear() { w0 = w1 = w2 = w3 = 0ull; }
  __device__ __forceinline__ void load(const uint64_t* p) { w0 = p[0]; w1 = p[1]; w2 = p[2]; w3 = p[3]; }
  __device__ __forceinline__ uint64_t word(int t) const {
    const int k = t >> 6;
    return k == 0 ? w0 : k == 1 ? w1 : k == 2 ? w2 : w3;
  }
  __device__ __forceinline__ bool has(int t) const { return (word(t) >> (t & 63)) & 1ull; }
  __device__ __forceinline__ void add(int t) {
    const int k = t >> 6;
    const uint64_t bit = 1ull << (t & 63);
    w0 |= k == 0 ? bit : 0ull;
    w1 |= k == 1 ? bit : 0ull;
    w2 |= k == 2 ? bit : 0ull;
    w3 |= k == 3 ? bit : 0ull;
  }
};
static_assert(kAncWords == 4, "NodeSet holds four words");
constexpr int kWave = 64;

// Per live sample, built on the host for every verify call.
struct SampleInfo {
  int64_t kv_base;   // element offset of the sample's block in the KV pool
  int32_t cap;       // positions per (layer, K/V, kv head)
  int32_t seq_len;   // committed length S_b
  int32_t tok0;      // first node row of the sample in the batch
  int32_t ntok;      // T_b
  int32_t pad0, pad1;
};
static_assert(sizeof(SampleInfo) == 32, "SampleInfo layout");

// Per node row, written by the metadata kernel.
struct TokInfo {
  int32_t sample;    // live-sample index b
  int32_t node;      // node index inside its tree
  int32_t pos;       // rotary position S_b + depth
  int32_t depth;
};
static_assert(sizeof(TokInfo) == 16, "TokInfo layout");

// One attention work item: a tile of up to 32 query rows of one
// (sample, kv head) against the key range [key0, key1) of its cache.
// Query row r of a (sample, kv head) is (node r / G, query head kvh*G + r % G).
struct AttnItem {
  int32_t sample, kvh, row0, key0, key1, nsplit, part, pad;
};
static_assert(sizeof(AttnItem) == 32, "AttnItem layout");

// One sample of a KV transfer (pack or unpack of a token range).
struct MigrateInfo {
  int64_t kv_base;      // element offset of the sample's block in the KV pool
  int32_t cap;          // positions per (layer, K/V, kv head)
  int32_t begin;        // first token of the range
  int32_t count;        // tokens in the range
  int32_t tok_prefix;   // tokens of the samples before this one in the call
  int32_t wg_prefix;    // work-groups of the samples before it, within one (layer, K/V)
  int32_t chunks;       // work-groups per (layer, K/V, kv head) run of this sample
};
static_assert(sizeof(MigrateInfo) == 32, "MigrateInfo layout");

// One split-combine job: nsplit partial tiles starting at slot part0.
struct CombineItem {
  int32_t sample, kvh, row0, nsplit, part0, pad0, pad1, pad2;
};

// Record `msg` as the calling thread's spec_last_error() and return `code`.
int set_error(int code, const char* msg);

// ---------------------------------------------------------------------------
// Launchers (each returns hipGetLastError() of its launch)
// ---------------------------------------------------------------------------

enum GemmEpilogue { EPI_QKV = 0, EPI_RESID = 1, EPI_GATE_UP = 2, EPI_ARGMAX = 3 };

struct GemmArgs {
  const bf16* A;          // [M][K] activations
  int M, K;
  // Weight segments (row-major [rows][K]); virtual columns run through them
  // in order.
  const bf16* B0; const bf16* B1; const bf16* B2;
  int n0, n1, n2;         // rows of each segment
  int N;                  // n0 + n1 + n2 (EPI_GATE_UP: 2 * ffn)
  // EPI_QKV
  bf16* q_out;            // [M][n_heads*head_dim]
  bf16* kv_pool;
  const SampleInfo* samples;
  const TokInfo* toks;
  int layer, n_kv_heads, head_dim;
  const float2* rope_cs;  // [M][head_dim/2] (cos, sin) of each row's angles
  // EPI_RESID
  float* x;               // [M][N] residual, x += A.B^T
  // EPI_GATE_UP
  bf16* act_out;          // [M][ffn]
  // EPI_ARGMAX
  float* part_val;        // [M][gemm_parts(N, M, K)]
  int32_t* part_idx;
  float* logits;          // optional [M][N]
  // Split-K scratch (gemm_partial_bytes() bytes; NULL disables splitting) and
  // the split count the launcher picked.
  float* partial;
  int ksplit;
  // EPI_RESID: the RMSNorm that follows the product (norm_out = bf16 of
  // x / rms(x) * norm_gain, row-major [M][N]); NULL: none.  When the product
  // is split over K, the launcher fuses the norm into the split-K reduction
  // and sets *norm_done; otherwise the caller runs the norm itself.
  const bf16* norm_gain;
  bf16* norm_out;
  float norm_eps;
  bool* norm_done;
};

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s);
// Number of (max, index) partials per row the EPI_ARGMAX launch for an
// [M x N] product with inner dimension K writes.
int gemm_parts(int N, int M, int K);
// Bytes of split-K partial storage launch_gemm may use through GemmArgs::partial.
size_t gemm_partial_bytes();
// Device address of the current device's static scratch (noalloc.hip).
hipError_t noalloc_scratch(void** out);

struct AttnArgs {
  const bf16* q;            // [N][n_heads*head_dim]
  const bf16* kv_pool;
  const SampleInfo* samples;
  const TokInfo* toks;
  const uint64_t* anc;      // [N][kAncWords] ancestor sets (NodeSet words)
  const AttnItem* items;    // 32-row items (tree_attention_kernel)
  int n_items;
  const AttnItem* wide;     // 128-row items (tree_attention_wide_kernel<HD, 4>)
  int n_wide;
  const AttnItem* wide8;    // 256-row items (tree_attention_wide_kernel<HD, 8>)
  int n_wide8;
  f16* part_o;              // [slots][32][head_dim], the split's output divided by its l
  float* part_ml;           // [slots][32][2]
  bf16* out;                // [N][n_heads*head_dim]
  int layer, n_heads, n_kv_heads, head_dim;
  const CombineItem* comb;
  int n_comb;
};

hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

hipError_t launch_tree_meta(const SampleInfo* samples, int batch, const int32_t* parents,
                            TokInfo* toks, uint64_t* anc, int32_t* dbg_depth, int32_t* dbg_pos,
                            uint64_t* dbg_anc, hipStream_t s);
hipError_t launch_rope_table(const TokInfo* toks, int n, int head_dim, float theta, float2* cs,
                             hipStream_t s);
hipError_t launch_embed(const int32_t* tokens, const bf16* table, float* x, int n, int hidden,
                        hipStream_t s);
hipError_t launch_rmsnorm(const float* x, const bf16* gain, bf16* out, int n, int hidden,
                          float eps, hipStream_t s);
hipError_t launch_argmax_reduce(const float* part_val, const int32_t* part_idx, int n, int parts,
                                int32_t* argmax, int32_t* dbg_argmax, hipStream_t s);
hipError_t launch_accept(const SampleInfo* samples, int batch, const int32_t* tokens,
                         const int32_t* parents, const TokInfo* toks, const int32_t* argmax,
                         int32_t* accepted_len, int32_t* next_token, int32_t* accepted_nodes,
                         hipStream_t s);
// Work-groups one (layer, K/V, kv head) run of `count` tokens takes.
int64_t kv_transfer_chunks(int count, int head_dim);
// Copy the runs described by info[0..n) between the pool and the transfer
// buffer (to_buffer: pool -> buffer, else buffer -> pool); wg_per_slab =
// sum over samples of n_kv_heads * chunks, tok_total = sum of counts.
hipError_t launch_kv_transfer(bool to_buffer, const MigrateInfo* info, int n, int64_t wg_per_slab,
                              int tok_total, bf16* pool, bf16* buf, int n_layers, int n_kv_heads,
                              int head_dim, hipStream_t s);
// Speculative sampling over the trees (temperature > 0): per-row log-sum-exp
// of logits / T, then one work-group per sample walks its tree.
// Scratch of launch_sample_accept: per-node decisions and one fp64 vocabulary
// row per sample.
size_t sample_accept_scratch(int batch, int n_tokens, int vocab);
hipError_t launch_sample_accept(const SampleInfo* samples, int batch, int n_tokens,
                                const TokInfo* toks, const int32_t* tokens,
                                const int32_t* parents, const float* logits,
                                const float* draft_probs, const float* uniforms, int vocab,
                                float temperature, int eos, void* scratch, int32_t* accepted_len,
                                int32_t* next_token, int32_t* accepted_nodes, hipStream_t s);
// Greedy acceptance with an end-of-sequence token.
hipError_t launch_accept_eos(const SampleInfo* samples, int batch, const int32_t* tokens,
                             const int32_t* parents, const TokInfo* toks, const int32_t* argmax,
                             int eos, int32_t* accepted_len, int32_t* next_token,
                             int32_t* accepted_nodes, hipStream_t s);
hipError_t launch_compact(const SampleInfo* samples, int batch, bf16* kv_pool, int n_layers,
                          int n_kv_heads, int head_dim, const int32_t* accepted_len,
                          const int32_t* accepted_nodes, int32_t* new_seq_lens, hipStream_t s);

}  // namespace spec
