/*
 * specverify: one batched speculative-decoding tree-verify step on an
 * AMD Instinct MI355X (gfx950).
 *
 * The operation (RLHFSpec, Section 2.2 "Speculative Decoding"; Section 5.2
 * names its two costs, attention over the KV cache and the FFN matrix
 * products; Section 6.2 fixes that a step never rewrites verified KV):
 *
 *   For every live sample b the caller hands in a committed KV length S_b
 *   and a draft token tree of T_b nodes (node 0 = root = the token decided
 *   by the previous step, whose K/V are not cached yet).  The target model,
 *   a Llama-style decoder, runs one forward pass over all N = sum T_b
 *   nodes: node i sits at position S_b + depth(i) and attends to the whole
 *   committed prefix plus its own ancestors in the tree (itself included).
 *   Greedy acceptance then takes g_i = argmax of node i's logits (lowest
 *   token id on ties), accepts a node when every edge on its branch carries
 *   the token its parent predicted (the root is always accepted), and
 *   picks the deepest accepted node (lowest node index on ties):
 *   accepted_len = its depth, next_token = its g.  Committing moves the K/V
 *   of the accepted branch to cache positions S_b .. S_b + accepted_len and
 *   the committed length becomes S_b + accepted_len + 1.
 *
 * Conventions for every entry point:
 *   - Return value: SPEC_OK (0) or a negative spec_status.  On a validation
 *     failure nothing has been enqueued and no output or KV byte has been
 *     written; spec_last_error() then describes the failure.
 *   - Work is enqueued on the caller's HIP stream (passed as void*; NULL is
 *     the null stream) and is asynchronous: device outputs are valid once
 *     the stream has been synchronised.
 *   - "host" / "device" below says where a pointer must point.  All device
 *     memory (weights, KV pool, workspace, outputs) is allocated and owned
 *     by the caller; the library never allocates device memory.  The only
 *     allocations it makes are its opaque handle and a small pinned host
 *     staging area inside it.
 *   - One spec_kv handle must not be used from two threads or two streams
 *     at once.
 *   - Numerics: bf16 weights, bf16 activations at GEMM inputs, bf16 KV
 *     cache; fp32 accumulation, softmax, norms and residual stream.
 *   - Supported shapes: head_dim 64 or 128; hidden, n_heads*head_dim and
 *     ffn multiples of 128; n_kv_heads*head_dim a multiple of 128; vocab a
 *     multiple of 128; n_heads a multiple of n_kv_heads; 1 <= T_b <=
 *     SPEC_MAX_TREE.  Anything else returns SPEC_ERR_UNSUPPORTED.
 */
#ifndef SPECVERIFY_H
#define SPECVERIFY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPEC_MAX_TREE 256
/* 64-bit words of one node's ancestor set (spec_debug.anc). */
#define SPEC_ANC_WORDS (SPEC_MAX_TREE / 64)

typedef enum {
  SPEC_OK = 0,
  SPEC_ERR_INVALID = -1,     /* null pointer, non-positive size, bad config or sample id */
  SPEC_ERR_TREE = -2,        /* parents[0] != -1, parent not before child, token out of range */
  SPEC_ERR_CAPACITY = -3,    /* S_b + T_b exceeds the sample's KV capacity, or buffer too small */
  SPEC_ERR_WORKSPACE = -5,   /* workspace smaller than the call needs */
  SPEC_ERR_UNSUPPORTED = -6, /* shape outside the supported set (see above) */
  SPEC_ERR_HIP = -7          /* a HIP runtime call or kernel launch failed */
} spec_status;

/* Llama-style decoder shape.  rope_theta: base of the rotary frequencies,
 * frequency j = rope_theta^(-2j/head_dim), half-split rotation (element j
 * pairs with j + head_dim/2).  rms_eps: RMSNorm epsilon. */
typedef struct {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
  float rope_theta, rms_eps;
} spec_model_config;

/* Weights: device pointers to row-major bf16 matrices in [out][in] layout
 * (a GEMM computes x . W^T), read-only, owned by the caller.  The per-layer
 * fields are HOST arrays of n_layers device pointers. */
typedef struct {
  const void* tok_embed;        /* [vocab][hidden] */
  const void* final_norm;       /* [hidden] RMSNorm gain */
  const void* lm_head;          /* [vocab][hidden] (untied) */
  const void* const* attn_norm; /* [hidden] */
  const void* const* wq;        /* [n_heads*head_dim][hidden] */
  const void* const* wk;        /* [n_kv_heads*head_dim][hidden] */
  const void* const* wv;        /* [n_kv_heads*head_dim][hidden] */
  const void* const* wo;        /* [hidden][n_heads*head_dim] */
  const void* const* ffn_norm;  /* [hidden] */
  const void* const* w_gate;    /* [ffn][hidden] */
  const void* const* w_up;      /* [ffn][hidden] */
  const void* const* w_down;    /* [hidden][ffn] */
} spec_weights;

/* Opaque KV-pool handle (host memory, owned by the library). */
typedef struct spec_kv spec_kv;

/* Optional device dumps for tests; any field may be NULL.  N = sum T_b,
 * rows in batch order (sample 0's nodes first, each tree in its own node
 * order). */
typedef struct {
  float* logits;      /* [N][vocab] fp32 */
  int32_t* argmax;    /* [N] greedy token after each node */
  int32_t* depth;     /* [N] depth of each node (root 0) */
  int32_t* pos;       /* [N] position S_b + depth */
  uint64_t* anc;      /* [N][SPEC_ANC_WORDS] ancestor set: bit t % 64 of word t / 64 is node t
                         of the same tree; own bit set, bits of nodes >= T_b clear */
} spec_debug;

/* ---- KV pool (Section 6.2: verified KV is never rewritten) -------------
 *
 * Layout: sample s owns one contiguous block of
 *   n_layers * 2 * n_kv_heads * capacity[s] * head_dim  bf16 values,
 * ordered [layer][K=0,V=1][kv_head][position][head_dim]; blocks follow each
 * other in sample order, each starting at a 256-byte aligned offset.
 * Positions [0, S_s) hold committed K/V (K already rotated). */

/* Bytes a pool for n_samples samples with the given host capacities needs,
 * or 0 if an argument is invalid. */
size_t spec_kv_bytes(const spec_model_config* cfg, int32_t n_samples, const int32_t* capacity);

/* Create a handle over caller memory device_buf (device, >= spec_kv_bytes,
 * 256-byte aligned).  capacity: host [n_samples].  *out receives the handle. */
int spec_kv_alloc(const spec_model_config* cfg, int32_t n_samples, const int32_t* capacity,
                  void* device_buf, size_t buf_bytes, spec_kv** out);

/* Release the handle (not device_buf).  Waits for the handle's pending
 * staging copies. */
int spec_kv_free(spec_kv* kv);

/* Byte offset of sample's block inside device_buf and its capacity. */
int spec_kv_sample_layout(const spec_kv* kv, int32_t sample, int64_t* byte_offset,
                          int32_t* capacity);

/* ---- The verify step ---------------------------------------------------- */

/* Workspace bytes spec_verify needs for up to max_batch samples and
 * max_tokens tree nodes in total; 0 if an argument is invalid. */
size_t spec_workspace_bytes(const spec_model_config* cfg, int32_t max_batch, int32_t max_tokens);

/* One tree-verify step over `batch` live samples.
 *   sample_ids   host [batch]   pool sample of each live sample (distinct)
 *   tree_offsets host [batch+1] tree_offsets[0] = 0, T_b = diff, 1..SPEC_MAX_TREE
 *   tree_tokens  host [N]       token of every node, in [0, vocab)
 *   tree_parents host [N]       parent node index within the same tree;
 *                               -1 for node 0, 0 <= parent < node otherwise
 *   seq_lens     host [batch]   committed length S_b, S_b + T_b <= capacity
 *   workspace    device, ws_bytes >= spec_workspace_bytes(cfg, batch, N)
 * Outputs (device, int32):
 *   accepted_len   [batch]                  depth of the deepest accepted node
 *   next_token     [batch]                  greedy token after that node
 *   accepted_nodes [batch][SPEC_MAX_TREE]   node ids of the accepted branch,
 *                                           root first, then -1
 * KV effect: writes the nodes' K/V to positions S_b + node of each sample
 * (never below S_b).  dbg may be NULL. */
int spec_verify(const spec_model_config* cfg, const spec_weights* w, spec_kv* kv,
                int32_t batch, const int32_t* sample_ids, const int32_t* tree_offsets,
                const int32_t* tree_tokens, const int32_t* tree_parents, const int32_t* seq_lens,
                void* workspace, size_t ws_bytes, void* stream,
                int32_t* accepted_len, int32_t* next_token, int32_t* accepted_nodes,
                const spec_debug* dbg);

/* ---- Acceptance at a sampling temperature, and end of sequence ---------
 *
 * Speculative decoding is lossless (Section 2.2): at temperature T > 0 the
 * verified tokens follow the target model's sampling distribution
 * p_u = softmax(z_u / T) (z_u: the logits after node u).  This assumes the
 * draft drew the children of every node u independently from its own
 * distribution q_u.  The acceptance walk (multi-draft speculative sampling):
 * at the current node u, with the unnormalised residual P = p_u (total R =
 * its fp64 sum), try u's children in node order; child c with token x is
 * accepted when uniforms[c][0] * q_u(x) * R < P(x); a rejected child sets
 * P = max(P - R q_u, 0) and R = sum P.  An accepted child becomes u.  When no
 * child of u is accepted (or u has none) the next token is the smallest y
 * with P(0) + ... + P(y) > uniforms[u][1] * R.  Residuals, sums and the CDF
 * are fp64.  accepted_len = depth of the final u, accepted_nodes = the path.
 *
 * End of sequence (eos_token >= 0, RLHF rollouts end at it): an accepted node
 * carrying the EOS token ends the branch, its children are not tried and
 * next_token = -1.  With temperature 0 the acceptance is spec_verify's greedy
 * rule with that truncation (an accepted EOS node accepts no children).
 *
 * spec_sampling:
 *   temperature  >= 0, finite
 *   eos_token    -1 (none) or a token id
 *   draft_probs  device [N][vocab] fp32, row i = q of node i (sums to 1;
 *                read for nodes with children); unused when temperature == 0
 *   uniforms     device [N][2] fp32 in [0, 1): column 0 = node i's
 *                acceptance draw as a child, column 1 = the draw that samples
 *                the next token if the walk ends at node i; unused at T == 0
 * The random draws are inputs so that the caller owns the randomness. */
typedef struct {
  float temperature;
  int32_t eos_token;
  const float* draft_probs;
  const float* uniforms;
} spec_sampling;

/* Workspace bytes spec_verify_sampled needs at temperature > 0 (the logits
 * [N][vocab] fp32, per-row log-sum-exp and a [batch][vocab] fp64 residual on
 * top of spec_workspace_bytes); 0 if an argument is invalid.  At temperature
 * 0 spec_workspace_bytes suffices. */
size_t spec_workspace_bytes_sampled(const spec_model_config* cfg, int32_t max_batch,
                                    int32_t max_tokens);

/* spec_verify with the acceptance above.  Same arguments and outputs; samp
 * must not be NULL.  dbg->logits, when given, receives the logits the
 * sampling reads. */
int spec_verify_sampled(const spec_model_config* cfg, const spec_weights* w, spec_kv* kv,
                        int32_t batch, const int32_t* sample_ids, const int32_t* tree_offsets,
                        const int32_t* tree_tokens, const int32_t* tree_parents,
                        const int32_t* seq_lens, void* workspace, size_t ws_bytes, void* stream,
                        const spec_sampling* samp, int32_t* accepted_len, int32_t* next_token,
                        int32_t* accepted_nodes, const spec_debug* dbg);

/* ---- Verify without a caller workspace ---------------------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation):
 * spec_verify with its workspace taken from a static device array of
 * SPEC_NOALLOC_SCRATCH_BYTES, one per device, held by the library from the
 * first call on that device until the process ends.  Arguments, outputs, KV
 * effect and results are spec_verify's (bitwise: the same plan and kernels),
 * without workspace and ws_bytes.  The call makes no device or pinned host
 * allocation; its per-call descriptors go to the device from pageable host
 * memory (hipMemcpyAsync, which may block the calling thread until the copy
 * is done).  Returns SPEC_ERR_WORKSPACE, before enqueueing anything, when
 * spec_workspace_bytes(cfg, batch, N) exceeds SPEC_NOALLOC_SCRATCH_BYTES (at
 * the Llama-3-8B shape, 128 samples with 1024 tree nodes in total fit).
 * Every call on one device shares that device's array and leaves its
 * contents behind: calls that overlap on one device (two streams, two
 * threads) race and must be serialised by the caller.  The calling thread's
 * current device must be the stream's; SPEC_ERR_HIP if the array's address
 * cannot be looked up on it. */
#define SPEC_NOALLOC_SCRATCH_BYTES ((size_t)320 << 20)

int spec_verify_noalloc(const spec_model_config* cfg, const spec_weights* w, spec_kv* kv,
                        int32_t batch, const int32_t* sample_ids, const int32_t* tree_offsets,
                        const int32_t* tree_tokens, const int32_t* tree_parents,
                        const int32_t* seq_lens, void* stream, int32_t* accepted_len,
                        int32_t* next_token, int32_t* accepted_nodes, const spec_debug* dbg);

/* Commit the accepted branches of the preceding spec_verify (same batch,
 * sample_ids and seq_lens, same stream): the K/V of node accepted_nodes[b][d]
 * moves to position S_b + d for d = 1..accepted_len[b] (all layers, K and
 * V), and new_seq_lens[b] = S_b + accepted_len[b] + 1.
 *   accepted_len, accepted_nodes: device, as written by spec_verify
 *   new_seq_lens: device [batch] int32 output */
int spec_kv_commit(spec_kv* kv, int32_t batch, const int32_t* sample_ids,
                   const int32_t* seq_lens, const int32_t* accepted_len,
                   const int32_t* accepted_nodes, int32_t* new_seq_lens, void* stream);

/* ---- KV transfer for sample migration ----------------------------------
 * (Section 6.2, "Two-stage Sample Migration": phase 1 copies the K/V of the
 * migrating samples out of the cache store into one contiguous buffer, so
 * that the transfer is a single copy; phase 3 parses such a buffer and
 * appends its K/V to the destination store.  Verified K/V never changes
 * (the Markov property the paper relies on), so stage 1 can move the
 * verified prefix [0, S) while the sample keeps running and stage 2 only the
 * tokens verified since: both are a token range [begin, end) per sample.)
 *
 * Buffer layout, the paper's model -> layer -> sample order (this library
 * holds one model, the LLM):
 *   [layer][K=0,V=1][sample j in call order][kv_head][token begin_j .. end_j-1][head_dim]
 * bf16, no padding; its size is spec_kv_transfer_bytes.
 *
 *   sample_ids host [n]  distinct pool samples, 1 <= n <= pool samples
 *   tok_begin  host [n]  first token of each range, 0 <= begin
 *   tok_end    host [n]  one past the last, begin <= end <= capacity
 *                        (empty ranges are allowed and contribute nothing)
 *   buf        device, 16-byte aligned, buf_bytes >= spec_kv_transfer_bytes
 * The buffer belongs to the caller.  Returns SPEC_ERR_CAPACITY for a range
 * outside a sample's capacity or a buffer that is too small; nothing is
 * enqueued then. */

/* Bytes of the transfer buffer for these ranges (0 if an argument is invalid). */
size_t spec_kv_transfer_bytes(const spec_kv* kv, int32_t n, const int32_t* tok_begin,
                              const int32_t* tok_end);

/* Phase 1: copy positions [begin_j, end_j) of every layer, K and V and KV
 * head of sample sample_ids[j] into buf.  Reads the pool only. */
int spec_kv_pack(spec_kv* kv, int32_t n, const int32_t* sample_ids, const int32_t* tok_begin,
                 const int32_t* tok_end, void* buf, size_t buf_bytes, void* stream);

/* Phase 3: the reverse: write buf's runs to positions [begin_j, end_j) of
 * sample sample_ids[j] of this pool (the destination of the migration; the
 * caller raises its committed lengths afterwards).  Reads buf only. */
int spec_kv_unpack(spec_kv* kv, int32_t n, const int32_t* sample_ids, const int32_t* tok_begin,
                   const int32_t* tok_end, const void* buf, size_t buf_bytes, void* stream);

/* ---- Drafting-strategy selection (Section 5) ----------------------------
 *
 * Verification-cost predictor (Section 5.2, "the execution time"): a
 * regression on the verification features, in milliseconds,
 *   t_sd = c0 + c_seq * N_seq + c_draft * N_draft + c_tree * TK
 * with N_seq = sum of committed lengths S_b (the KV the attention loads),
 * N_draft = sum of tree sizes T_b (the rows of the FFN products) and
 * TK = sum of T_b * S_b (the attention work that grows with both).  The
 * coefficients are fitted offline on measured steps of this library.
 * Bucket cache: with bucket_ratio r > 0, every feature x > 0 falls in bucket
 * floor(log(x) / log(1 + r)) (0 has its own bucket); all feature triples in
 * one bucket share the prediction at the buckets' geometric midpoints, which
 * is computed once and then read from the cache.  r = 0 disables it. */
typedef struct {
  double c0, c_seq, c_draft, c_tree;
  double bucket_ratio;
} spec_cost_coeffs;

typedef struct spec_cost_model spec_cost_model;   /* opaque, host, owned by the library */

int spec_cost_model_create(const spec_cost_coeffs* coeffs, spec_cost_model** out);
int spec_cost_model_free(spec_cost_model* model);
/* Predicted step time in ms, or a negative value for a negative feature. */
double spec_cost_predict(spec_cost_model* model, int64_t n_seq, int64_t n_draft, int64_t tree_kv);
/* Cache hits and misses since creation. */
int spec_cost_model_stats(const spec_cost_model* model, int64_t* hits, int64_t* misses);

/* Choose the draft token num n (tree nodes per sample, root included) of the
 * next step for a batch (Sections 5.1 and 5.3): n maximises
 * al(n) / t_sd(n), where al(n) = sum over samples of the weights of S_b(n)
 * and t_sd is the predictor above at the features of trees of min(n, |tree|)
 * nodes.  S_b(1) = {root}; S_b(n+1) adds the heaviest unselected node of the
 * sample's candidate tree, taken from a max-priority queue that receives the
 * nodes of layer m (depth m) when the search reaches layer m; equal weights
 * go to the shallower node, then the lower index.  Since weights never grow
 * from parent to child, S_b(n) is a connected tree.  The search over n stops
 * after `patience` consecutive falls of the objective.
 *   seq_lens      host [batch]    committed length S_b of each sample
 *   tree_offsets  host [batch+1]  candidate trees, offsets[0] = 0, sizes >= 1
 *   parents       host [total]    parent within the tree, -1 for node 0,
 *                                 0 <= parent < node otherwise
 *   weights       host [total]    w(u) = F(dl(u)) >= 0, w(child) <= w(parent)
 *   n_max         1 .. SPEC_MAX_TREE
 * Outputs (host): *n_out; selected [batch][n_max], sample b's nodes in the
 * order they joined S_b (the first n form S_b(n)), -1 past the tree's size;
 * objective [n_max] (may be NULL): al(n) / t_sd(n), 0 past the stop. */
int spec_select_draft_count(spec_cost_model* model, int32_t batch, const int32_t* seq_lens,
                            const int32_t* tree_offsets, const int32_t* parents,
                            const float* weights, int32_t n_max, int32_t patience, int32_t* n_out,
                            int32_t* selected, double* objective);

/* Message of the last failure on the calling thread ("" if none). */
const char* spec_last_error(void);

/* ---- Kernel timing (measurement only) ----------------------------------
 * While enabled, every launch of the named kernel class is bracketed by a
 * pair of HIP events on its stream.  spec_profile_end synchronises those
 * events, returns the summed duration in ms and the launch count, and
 * disables timing.  Kernel classes: */
enum {
  SPEC_K_GEMM_QKV = 0,
  SPEC_K_ATTENTION = 1,
  SPEC_K_GEMM_O = 2,
  SPEC_K_GEMM_GATE_UP = 3,
  SPEC_K_GEMM_DOWN = 4,
  SPEC_K_LM_HEAD = 5,
  SPEC_K_COMMIT = 6,
  SPEC_K_TRANSFER = 7,   /* spec_kv_pack / spec_kv_unpack */
  SPEC_K_ACCEPT = 8,     /* tree acceptance: greedy, greedy with EOS, or sampled */
  SPEC_K_COUNT = 9
};
int spec_profile_begin(int32_t kernel_class, int32_t max_launches);
int spec_profile_end(float* total_ms, int32_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* SPECVERIFY_H */
