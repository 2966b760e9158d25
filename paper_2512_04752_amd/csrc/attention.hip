// Tree attention for the verify step.
//
// Query row r of (sample b, kv head g) is node r / G with query head
// g*G + r % G (G = n_heads / n_kv_heads query heads share one KV head).  It
// sees every committed key [0, S_b) and, of the tree keys at cache slots
// S_b + t, exactly its ancestors t (itself included), given as a bitmask.
//
// Every kernel processes 32-key blocks per wave with the transposed products
//
//   S^T (32 keys x 32 rows) = K . Q^T   v_mfma_f32_32x32x16_bf16, A = K (LDS)
//   online softmax per row              each lane owns one row (16 of its keys,
//                                       the other 16 in lane ^ 32)
//   O^T (dims x 32 rows) += V^T . P^T   A = V^T read from row-major V in LDS
//                                       with ds_read_b64_tr_b16, B = P straight
//                                       from the S^T accumulator registers
//
// which keep a row's softmax state and its output column in one lane.  K and
// V rows are copied HBM -> LDS verbatim by global_load_lds_dwordx4 with their
// 16-byte chunks XOR-swizzled so that both the K reads (16 rows, one chunk)
// and the transposing V reads (4 rows x 4 columns of 8 bytes) are free of
// bank conflicts.
//
// The softmax runs in the base-2 domain (scores scaled by log2(e)/sqrt(d)
// inside one FMA, v_exp_f32 directly).  The running output is rescaled only
// when some row's maximum outgrew the reference maximum by more than
// kRescaleSlack (a wave-uniform test); the maximum settles within that slack
// after the first blocks, so the rescale of the accumulators is rare.
//
//   * tree_attention_kernel: one 32-row tile per work-group (at most 32 query
//     rows per KV head, e.g. 8-node trees with 4 query heads per KV head).  The
//     key range is dealt to the work-group's 2 waves in 32-key blocks; each
//     wave streams its blocks through a private 40 KB LDS ring of
//     half-stages (the K or the V rows of one block; the K of block t is
//     waited for before the V, and three half-stages stay in flight), with no
//     work-group barrier, and the partial softmax states are merged through
//     LDS at the end.  Two such work-groups share a CU, so one's start-up
//     (descriptor, query and first-block latency) and merge overlap the
//     other's streaming.
//   * tree_attention_wide_kernel<HD, NW>: 32*NW query rows per work-group
//     (NW = 4 or 8 waves; larger trees).  Wave w owns rows 32w..32w+31; all
//     waves share a ring of 64-key K/V stages loaded cooperatively, so the
//     key range is read once per 32*NW rows, and each wave ends with complete
//     rows (no merge).  Both score blocks of a stage are computed before the
//     first softmax, so the second block's MFMAs overlap the first softmax.
//
// Long key ranges are split into ranges processed in parallel and merged by
// attention_combine_kernel.
#include <math.h>

#include "common.h"

namespace spec {

namespace {

constexpr int KBLK = 32;

typedef __attribute__((address_space(3))) char lds_char;
typedef short v4i16 __attribute__((ext_vector_type(4)));

// Direct global -> LDS load: 16 bytes per lane, landing at the wave-uniform
// LDS address `lds` + 16 * lane.  Issued as inline assembly so that the
// compiler does not track an LDS write in flight: it cannot tell which ring
// stage a load targets, and would make every transposing V read wait for all
// outstanding loads (vmcnt(0)), which collapses the ring's lookahead.  The
// rings' own vmcnt waits and barriers order these loads.
// Every K/V row is read once per step, so the loads carry the non-temporal
// policy (nt): the stream passes through L2 without displacing what is
// re-read (queries, partial states).  Measured on the 8B shape: early-phase
// attention (batch 128, 8-node trees) 4.76 -> 3.87 ms per step, long-tail
// attention (batch 4, 64-node trees) 4.59 -> 4.49 ms.
__device__ __forceinline__ void load_lds16(const void* g, void* lds) {
  const uint32_t m0 = (uint32_t)(uintptr_t)(lds_char*)lds;
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt" ::"v"(g), "s"(m0) : "memory", "m0");
}

// Physical 16-byte chunk of logical chunk c in K row `key`: 16 consecutive
// rows reading one logical chunk hit 16 distinct 16-byte bank groups.
template <int HD>
__device__ __forceinline__ int kswz(int key) {
  return HD == 128 ? (key & 15) : ((key >> 1) & 7);
}
// V rows: the transposing read touches 4 consecutive rows x 32 bytes.
__device__ __forceinline__ int vswz(int key) { return (key & 3) << 1; }

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work-group barrier for a shared LDS ring: this wave's LDS reads are
// complete (the oldest slot may be refilled by any wave afterwards) while its
// direct-to-LDS loads of later stages stay in flight.  __syncthreads() would
// add a work-group fence, i.e. a wait for every outstanding global load,
// leaving one stage of lookahead however deep the ring.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// The running output is kept relative to a reference maximum m_run and
// rescaled only when some row's maximum exceeds it by more than this many
// binary orders; meanwhile probabilities up to 2^kRescaleSlack are formed,
// which fp32 sums and bf16 P^T operands hold with unchanged relative
// precision.  Softmax is invariant to the reference, so the result is the
// same up to rounding.
constexpr float kRescaleSlack = 8.f;

// max / sum of a value and its copy in lane ^ 32 (v_permlane32_swap: each
// lane ends with both halves' values in the two results).
__device__ __forceinline__ float max_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Scores of keys this lane's row may not see become -inf: committed keys
// (tree index tt < 0) are visible, tree key tt is visible when node tt is an
// ancestor, keys from key1 on never are.  The 32 keys of the block span at
// most two words of the ancestor set, picked once.
__device__ __forceinline__ void mask_block(f32x16& s, int kb, int key1, int seq_len, const NodeSet& anc,
                                           int h) {
  const int t0 = kb - seq_len;
  const uint64_t lo = anc.word(t0), hi = anc.word(t0 + 31);
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int key = kb + 8 * (e >> 2) + 4 * h + (e & 3);
    const int tt = key - seq_len;
    const uint64_t w = (tt >> 6) == (t0 >> 6) ? lo : hi;
    const bool anc_bit = (w >> (tt & 63)) & 1ull;
    const bool vis = (key < key1) & ((tt < 0) | anc_bit);
    s[e] = vis ? s[e] : -INFINITY;
  }
}

// Online-softmax update of one 64-key stage: raw scores sa (keys kb..kb+31)
// and sb (kb+32..kb+63), one running-maximum update and at most one rescale
// of the output for both.
template <int NB>
__device__ __forceinline__ void softmax_stage(bool mask_a, bool mask_b, f32x16& sa, f32x16& sb, int kb,
                                              int key1, int seq_len, const NodeSet& anc, int h, float sl2,
                                              float& m_run, float& l_run, f32x16 (&o)[NB],
                                              bf16x8 (&pa)[2], bf16x8 (&pb)[2]) {
  if (mask_a) mask_block(sa, kb, key1, seq_len, anc, h);
  if (mask_b) mask_block(sb, kb + 32, key1, seq_len, anc, h);
  float smax = fmaxf(sa[0], sb[0]);
#pragma unroll
  for (int e = 1; e < 16; ++e) smax = fmaxf(smax, fmaxf(sa[e], sb[e]));
  smax = max_xor32(smax);
  const float m_new = fmaxf(m_run, smax * sl2);
  if (__ballot(m_new > m_run + kRescaleSlack)) {
    const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < NB; ++i) o[i] *= alpha;
    m_run = m_new;
  }
  const float mb = m_run == -INFINITY ? 0.f : m_run;
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const float p0 = fast_exp2(fmaf(sa[e], sl2, -mb));
    const float p1 = fast_exp2(fmaf(sb[e], sl2, -mb));
    psum += p0 + p1;
    pa[e >> 3][e & 7] = (bf16)p0;
    pb[e >> 3][e & 7] = (bf16)p1;
  }
  l_run += psum;
}

// K fragment (A operand of S^T = K.Q^T) of k-step ks for key row `row` of a
// swizzled K block: 8 consecutive dims 16 ks + 8 h.
template <int HD>
__device__ __forceinline__ bf16x8 k_fragment(const char* k0, int row, int ks, int h) {
  return *(const bf16x8*)(k0 + row * (HD * 2) + (((2 * ks + h) ^ kswz<HD>(row)) << 4));
}

// V^T fragment (A operand) of k-step kst for output dims [32i, 32i+32) from
// a row-major, vswz-swizzled V block in LDS whose key 0 is `v0`.  Lane l
// (group q = l/16, L = l%16) ends with V[16 kst + 4(q/2) + {0..3, 8..11}]
// [32i + 16(q%2) + L]: register slot j carries key 16 kst + 8(j/4) + 4h + j%4
// with h = l/32, as the P^T operand expects.
template <int HD>
__device__ __forceinline__ bf16x8 vt_fragment(const char* v0, int kst, int i, int lane) {
  const int q = (lane >> 4) & 3, L = lane & 15;
  const int row = 16 * kst + 4 * (q >> 1) + (L >> 2);
  const int col = i * 32 + 16 * (q & 1) + 4 * (L & 3);           // element column
  const int chunk = col >> 3, within = (col & 7) * 2;
  const char* p0 = v0 + row * (HD * 2) + ((chunk ^ vswz(row)) << 4) + within;
  const char* p1 = v0 + (row + 8) * (HD * 2) + ((chunk ^ vswz(row + 8)) << 4) + within;
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)p0);
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16*)p1);
  const v4i16 both[2] = {lo, hi};
  bf16x8 f;
  __builtin_memcpy(&f, both, 16);
  return f;
}

// Online-softmax update of one 32-key block.  s holds the raw scores K.q of
// keys kb + 8(e/4) + 4h + e%4 of this lane's row; m_run is the running
// maximum of the scaled scores (base-2 domain).  Produces P^T in bf16 and
// accumulates the row sum of the unrounded probabilities.
template <bool MASK, int NB>
__device__ __forceinline__ void softmax_block(f32x16& s, int kb, int key1, int seq_len, const NodeSet& anc,
                                              int h, float sl2, float& m_run, float& l_run,
                                              f32x16 (&o)[NB], bf16x8 (&pb)[2]) {
  if constexpr (MASK) mask_block(s, kb, key1, seq_len, anc, h);
  float smax = s[0];
#pragma unroll
  for (int e = 1; e < 16; ++e) smax = fmaxf(smax, s[e]);
  smax = max_xor32(smax);
  const float m_new = fmaxf(m_run, smax * sl2);
  if (__ballot(m_new > m_run + kRescaleSlack)) {
    // exp2(m_run - m_new) is 0 for a first visible block (m_run = -inf);
    // rows with nothing visible yet keep alpha = 1.
    const float alpha = m_new == -INFINITY ? 1.f : fast_exp2(m_run - m_new);
    l_run *= alpha;
#pragma unroll
    for (int i = 0; i < NB; ++i) o[i] *= alpha;
    m_run = m_new;
  }
  const float mb = m_run == -INFINITY ? 0.f : m_run;
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const float pe = fast_exp2(fmaf(s[e], sl2, -mb));     // masked: exp2(-inf) = 0
    psum += pe;
    pb[e >> 3][e & 7] = (bf16)pe;
  }
  l_run += psum;
}

template <int NB>
__device__ __forceinline__ void softmax_any(bool mask, f32x16& s, int kb, int key1, int seq_len,
                                            const NodeSet& anc, int h, float sl2, float& m_run,
                                            float& l_run, f32x16 (&o)[NB], bf16x8 (&pb)[2]) {
  if (mask) softmax_block<true, NB>(s, kb, key1, seq_len, anc, h, sl2, m_run, l_run, o, pb);
  else softmax_block<false, NB>(s, kb, key1, seq_len, anc, h, sl2, m_run, l_run, o, pb);
}

// O^T += V^T . P^T for one 32-key block whose V rows start at v0.
template <int HD>
__device__ __forceinline__ void pv_block(const char* v0, const bf16x8 (&pb)[2], f32x16 (&o)[HD / 32],
                                         int lane) {
#pragma unroll
  for (int kst = 0; kst < 2; ++kst)
#pragma unroll
    for (int i = 0; i < HD / 32; ++i)
      o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vt_fragment<HD>(v0, kst, i, lane), pb[kst], o[i],
                                                    0, 0, 0);
}

template <int HD>
struct AttnCfg {
  static constexpr int ROW = HD * 2;                    // bytes per K or V row
  // narrow kernel: per-wave ring of half-stages (the K or the V rows of one
  // 32-key block), 40 KB per wave, so four waves fill the CU's 160 KB
  static constexpr int KV_BYTES = KBLK * ROW;
  static constexpr int WAVE_RING = 40 * 1024;
  static constexpr int NH = WAVE_RING / KV_BYTES;       // half-stage slots: 5 (HD 128), 10 (HD 64)
  static constexpr int LOADS = KV_BYTES / 1024;         // wave-loads for K (and for V)
  static constexpr int ROWS_PER_LOAD = 1024 / ROW;
  static constexpr int O_STRIDE = HD + 1;               // floats per merge row
  static constexpr int NWN = 2;                         // waves per work-group
  static constexpr int MERGE_BYTES = NWN * 32 * O_STRIDE * 4 + NWN * 32 * 2 * 4;
  static constexpr int SMEM = (NWN * WAVE_RING) > MERGE_BYTES ? (NWN * WAVE_RING) : MERGE_BYTES;
  // wide kernels: shared ring of 64-key stages
  static constexpr int WKEYS = 64;
  static constexpr int W_KV = WKEYS * ROW;              // K (or V) bytes per stage
  static constexpr int W_STAGE = 2 * W_KV;
};

// Wide-kernel ring depth: 8-wave groups own a CU (two waves per SIMD) and
// take four stages; 4-wave groups run two per CU within 160 KB of LDS.
template <int HD, int NW>
constexpr int wide_stages() {
  return (NW == 8 || HD == 64) ? 4 : 2;
}

// Wait until at most n (< N) of this wave's half-stage loads, L
// vector-memory operations each, are outstanding (n is wave-uniform).
template <int L, int N>
__device__ __forceinline__ void wait_halves(int n) {
  if constexpr (N <= 1) {
    wait_vm<0>();
  } else {
    if (n >= N - 1) wait_vm<(N - 1) * L>();
    else wait_halves<L, N - 1>(n);
  }
}

template <int HD>
__global__ __launch_bounds__(AttnCfg<HD>::NWN * 64, 2) void tree_attention_kernel(AttnArgs a) {
  using C = AttnCfg<HD>;
  constexpr int DC = HD / 8;                  // 16-byte chunks per row
  constexpr int NB = HD / 32;                 // 32-dim output blocks
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  // Items are dealt round-robin over the 8 XCDs; remap so that consecutive
  // items run on one XCD.
  const int per_xcd = gridDim.x >> 3;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= a.n_items) return;
  const AttnItem it = a.items[item];
  if (it.sample < 0) return;          // padding of a shorter per-XCD list
  const SampleInfo si = a.samples[it.sample];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int G = a.n_heads / a.n_kv_heads;
  const int nq_hd = a.n_heads * HD;

  // This lane's query row and its Q fragments (B operand of S^T = K.Q^T).
  const int grow = it.row0 + r;
  const int node = grow / G, head = it.kvh * G + grow % G;
  const bool row_ok = node < si.ntok;
  bf16x8 qf[HD / 16];
  const bf16* qrow = a.q + (size_t)(si.tok0 + (row_ok ? node : 0)) * nq_hd + head * HD;
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) {
    qf[ks] = *(const bf16x8*)(qrow + ks * 16 + h * 8);
    if (!row_ok) qf[ks] = bf16x8{};
  }
  // At most 32 rows per KV head: the tree has at most 32 nodes, all in word 0.
  NodeSet anc_row;
  anc_row.clear();
  anc_row.w0 = row_ok ? a.anc[(size_t)(si.tok0 + node) * kAncWords] : 1ull;

  const size_t head_stride = (size_t)si.cap * HD;
  const bf16* kbase = a.kv_pool + si.kv_base + ((size_t)a.layer * 2 * a.n_kv_heads + it.kvh) * head_stride;
  const bf16* vbase = kbase + (size_t)a.n_kv_heads * head_stride;
  char* ring = smem + w * C::WAVE_RING;

  // Blocks of this wave: w, w + NWN, w + 2 NWN, ... of the item's range.
  const int nblk = (it.key1 - it.key0 + KBLK - 1) / KBLK;
  const int mine = nblk > w ? (nblk - w + C::NWN - 1) / C::NWN : 0;
  const int mask_from = min(si.seq_len, it.key1);   // blocks ending past this need the mask

  // Half-stage h of this wave is the K rows (h even) or the V rows (h odd)
  // of its block h/2, in ring slot h % NH.  Lane l of wave-load j copies row
  // (j*ROWS_PER_LOAD + l / DC) into physical chunk l % DC; keys past the
  // range repeat the last key, whose scores are masked.
  const int lrow = lane / DC, lch = lane % DC;
  auto issue = [&](int hs) {
    const int kb = it.key0 + (w + C::NWN * (hs >> 1)) * KBLK;
    char* st = ring + (hs % C::NH) * C::KV_BYTES;
    const bool is_v = hs & 1;
    const bf16* src = is_v ? vbase : kbase;
#pragma unroll
    for (int j = 0; j < C::LOADS; ++j) {
      const int row = j * C::ROWS_PER_LOAD + lrow;
      int key = kb + row;
      key = key < it.key1 ? key : it.key1 - 1;
      const int sw = is_v ? vswz(row) : kswz<HD>(row);
      load_lds16(src + (size_t)key * HD + ((lch ^ sw) << 3), st + j * 1024);
    }
  };

  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e)/sqrt(d)
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x16{};

  // NH - 2 half-stages ahead of the block being read: while block t is
  // multiplied, the K and V of block t+1 and the K of block t+2 (at HD 128)
  // are in flight.
  const int nh = 2 * mine;
#pragma unroll
  for (int hs = 0; hs < C::NH - 2; ++hs)
    if (hs < nh) issue(hs);

  for (int t = 0; t < mine; ++t) {
    // The slots of block t-1 (consumed in the previous iteration) take
    // half-stages 2t+NH-2 and 2t+NH-1.
    if (2 * t + C::NH - 2 < nh) issue(2 * t + C::NH - 2);
    if (2 * t + C::NH - 1 < nh) issue(2 * t + C::NH - 1);
    const int newest = min(2 * t + C::NH - 1, nh - 1);
    wait_halves<C::LOADS, C::NH>(newest - 2 * t);          // K of block t has landed
    const char* st = ring + ((2 * t) % C::NH) * C::KV_BYTES;
    const char* sv = ring + ((2 * t + 1) % C::NH) * C::KV_BYTES;
    const int kb = it.key0 + (w + C::NWN * t) * KBLK;

    // S^T = K . Q^T for the 32 keys of this block (two independent chains).
    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int ks = 0; ks < HD / 16; ks += 2) {
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_fragment<HD>(st, r, ks, h), qf[ks], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k_fragment<HD>(st, r, ks + 1, h), qf[ks + 1], s1, 0,
                                                   0, 0);
    }
    f32x16 s = s0 + s1;
    bf16x8 pb[2];
    softmax_any<NB>(kb + KBLK > mask_from, s, kb, it.key1, si.seq_len, anc_row, h, sl2, m_run, l_run,
                    o, pb);
    wait_halves<C::LOADS, C::NH>(newest - 2 * t - 1);      // V of block t has landed
    pv_block<HD>(sv, pb, o, lane);
  }
  l_run += __shfl_xor(l_run, 32);

  // Merge the waves' (m, l, O) through LDS.
  __syncthreads();
  float* o_sh = (float*)smem;
  float* ml_sh = o_sh + C::NWN * 32 * C::O_STRIDE;
  if (h == 0) {
    ml_sh[(w * 32 + r) * 2] = m_run;
    ml_sh[(w * 32 + r) * 2 + 1] = l_run;
  }
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int d = i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      o_sh[(w * 32 + r) * C::O_STRIDE + d] = o[i][e];
    }
  __syncthreads();

  // Each thread merges 8 consecutive dimensions of a row and writes them as
  // one 16-byte store (bf16 output, or the fp16 partial of a split range).
  for (int idx = tid; idx < 32 * (HD / 8); idx += C::NWN * 64) {
    const int row = idx / (HD / 8), d0 = (idx % (HD / 8)) * 8;
    const int gr = it.row0 + row;
    const int nd = gr / G, hq = it.kvh * G + gr % G;
    if (nd >= si.ntok) continue;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < C::NWN; ++ww) M = fmaxf(M, ml_sh[(ww * 32 + row) * 2]);
    float O[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f}, L = 0.f;
#pragma unroll
    for (int ww = 0; ww < C::NWN; ++ww) {
      const float mw = ml_sh[(ww * 32 + row) * 2];
      const float f = (mw == -INFINITY) ? 0.f : fast_exp2(mw - M);
#pragma unroll
      for (int j = 0; j < 8; ++j) O[j] += f * o_sh[(ww * 32 + row) * C::O_STRIDE + d0 + j];
      L += f * ml_sh[(ww * 32 + row) * 2 + 1];
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    if (it.nsplit == 1) {
      bf16x8 v;
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = (bf16)(O[j] * inv);
      *(bf16x8*)(a.out + (size_t)(si.tok0 + nd) * nq_hd + hq * HD + d0) = v;
    } else {
      typedef __attribute__((ext_vector_type(8))) _Float16 f16x8;
      f16x8 v;
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = (f16)(O[j] * inv);
      *(f16x8*)(a.part_o + ((size_t)it.part * 32 + row) * HD + d0) = v;
      if (d0 == 0) {
        a.part_ml[((size_t)it.part * 32 + row) * 2] = M;
        a.part_ml[((size_t)it.part * 32 + row) * 2 + 1] = L;
      }
    }
  }
}

// 32*NW query rows per work-group: wave w owns rows it.row0 + 32w .. +31 and
// all keys of the range, streamed in shared 64-key stages through an NS-deep
// ring (one barrier per stage, NS-2 stages in flight behind the one being
// read).  With the range split, wave w's partial state goes to slot
// it.part + w * it.nsplit (its row tile's slot for this split).
template <int HD, int NW>
__global__ __launch_bounds__(64 * NW, NW == 4 ? 2 : 1) void tree_attention_wide_kernel(AttnArgs a,
                                                                       const AttnItem* items,
                                                                       int n_items) {
  using C = AttnCfg<HD>;
  constexpr int DC = HD / 8;
  constexpr int NB = HD / 32;
  constexpr int NS = wide_stages<HD, NW>();
  constexpr int W_LOADS = C::W_KV / 1024 / NW;   // per wave and stage, for K (and for V)
  constexpr int LPW = 2 * W_LOADS;                // vector-memory ops per wave and stage
  static_assert(W_LOADS >= 1, "stage too small for the work-group");
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int per_xcd = gridDim.x >> 3;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= n_items) return;
  const AttnItem it = items[item];
  if (it.sample < 0) return;
  const SampleInfo si = a.samples[it.sample];
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = lane & 31, h = lane >> 5;
  const int G = a.n_heads / a.n_kv_heads;
  const int nq_hd = a.n_heads * HD;

  const int grow = it.row0 + 32 * w + r;
  const int node = grow / G, head = it.kvh * G + grow % G;
  const bool row_ok = node < si.ntok;
  bf16x8 qf[HD / 16];
  const bf16* qrow = a.q + (size_t)(si.tok0 + (row_ok ? node : 0)) * nq_hd + (row_ok ? head : 0) * HD;
#pragma unroll
  for (int ks = 0; ks < HD / 16; ++ks) {
    qf[ks] = *(const bf16x8*)(qrow + ks * 16 + h * 8);
    if (!row_ok) qf[ks] = bf16x8{};
  }
  NodeSet anc_row;
  anc_row.clear();
  anc_row.w0 = 1ull;
  if (row_ok) anc_row.load(a.anc + (size_t)(si.tok0 + node) * kAncWords);

  const size_t head_stride = (size_t)si.cap * HD;
  const bf16* kbase = a.kv_pool + si.kv_base + ((size_t)a.layer * 2 * a.n_kv_heads + it.kvh) * head_stride;
  const bf16* vbase = kbase + (size_t)a.n_kv_heads * head_stride;

  const int nstage = (it.key1 - it.key0 + C::WKEYS - 1) / C::WKEYS;
  const int mask_from = min(si.seq_len, it.key1);
  // Wave w loads rows [W_LOADS*ROWS_PER_LOAD*w, +W_LOADS*ROWS_PER_LOAD) of
  // each stage's K and V.
  const int lrow = lane / DC, lch = lane % DC;
  auto issue = [&](int t, int slot) {
    const int kb = it.key0 + t * C::WKEYS;
    char* st = smem + slot * C::W_STAGE;
#pragma unroll
    for (int j = 0; j < W_LOADS; ++j) {
      const int row = (w * W_LOADS + j) * C::ROWS_PER_LOAD + lrow;
      int key = kb + row;
      key = key < it.key1 ? key : it.key1 - 1;
      load_lds16(kbase + (size_t)key * HD + ((lch ^ kswz<HD>(row)) << 3),
                 st + (w * W_LOADS + j) * 1024);
      load_lds16(vbase + (size_t)key * HD + ((lch ^ vswz(row)) << 3),
                 st + C::W_KV + (w * W_LOADS + j) * 1024);
    }
  };

  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x16{};

#pragma unroll
  for (int t = 0; t < NS - 1; ++t)
    if (t < nstage) issue(t, t);
  // Unrolled by the ring depth so that every LDS address is a per-lane base
  // plus an immediate.
  for (int t0 = 0; t0 < nstage; t0 += NS) {
#pragma unroll
    for (int u = 0; u < NS; ++u) {
      const int t = t0 + u;
      if (t >= nstage) break;
      // Stage t must have landed; stages t+1 .. t+NS-2 may stay in flight.
      const int pending = min(NS - 2, nstage - 1 - t);
      if constexpr (NS == 4) {
        if (pending >= 2) wait_vm<2 * LPW>();
        else if (pending == 1) wait_vm<LPW>();
        else wait_vm<0>();
      } else {
        wait_vm<0>();
      }
      ring_barrier();     // stage t visible to all waves; stage t-1 fully consumed
      if (t + NS - 1 < nstage) issue(t + NS - 1, (u + NS - 1) % NS);
      const char* st = smem + u * C::W_STAGE;
      const int kb = it.key0 + t * C::WKEYS;

      // Scores of both 32-key blocks (two independent MFMA chains), K
      // fragments read one k-step ahead.
      f32x16 sa = f32x16{}, sb = f32x16{};
      bf16x8 ka = k_fragment<HD>(st, r, 0, h), kb2 = k_fragment<HD>(st, KBLK + r, 0, h);
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        bf16x8 na, nb;
        if (ks + 1 < HD / 16) {
          na = k_fragment<HD>(st, r, ks + 1, h);
          nb = k_fragment<HD>(st, KBLK + r, ks + 1, h);
        }
        sa = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[ks], sa, 0, 0, 0);
        sb = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kb2, qf[ks], sb, 0, 0, 0);
        if (ks + 1 < HD / 16) {
          ka = na;
          kb2 = nb;
        }
      }
      bf16x8 pa[2], pb[2];
      softmax_stage<NB>(kb + KBLK > mask_from, kb + 2 * KBLK > mask_from, sa, sb, kb, it.key1,
                        si.seq_len, anc_row, h, sl2, m_run, l_run, o, pa, pb);
      pv_block<HD>(st + C::W_KV, pa, o, lane);
      pv_block<HD>(st + C::W_KV + KBLK * C::ROW, pb, o, lane);
    }
  }
  l_run = sum_xor32(l_run);

  // Finished rows go out through LDS so that every store writes 1 KB
  // contiguous: each wave stages its 32 rows (bf16 output or fp16 partial,
  // both 2 bytes per element) in a private region of the now idle ring,
  // then lane l of store k writes 16 bytes of row 4k + l/16.
  __syncthreads();            // every wave has finished reading the last stage
  constexpr int PITCH = HD * 2 + 16;                 // bytes per staged row
  char* stg = smem + w * 32 * PITCH;
  const float inv = l_run > 0.f ? 1.f / l_run : 0.f;
  const bool split = it.nsplit > 1;
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      char* dst = stg + r * PITCH + (32 * i + 8 * q + 4 * h) * 2;
      if (split) {
        f16x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = (f16)(o[i][4 * q + j] * inv);
        *(f16x4*)dst = v;
      } else {
        bf16x4 v;
#pragma unroll
        for (int j = 0; j < 4; ++j) v[j] = (bf16)(o[i][4 * q + j] * inv);
        *(bf16x4*)dst = v;
      }
    }
  const int slot = it.part + w * it.nsplit;
  if (split && h == 0 && row_ok) {
    a.part_ml[((size_t)slot * 32 + r) * 2] = m_run;
    a.part_ml[((size_t)slot * 32 + r) * 2 + 1] = l_run;
  }
  constexpr int CPR = HD / 8;                        // 16-byte chunks per row
  constexpr int RPS = 64 / CPR;                      // rows per 1 KB store
#pragma unroll
  for (int k = 0; k < 32 / RPS; ++k) {
    const int rr = k * RPS + lane / CPR, ch = lane % CPR;
    const i32x4 v = *(const i32x4*)(stg + rr * PITCH + ch * 16);
    const int gr = it.row0 + 32 * w + rr;
    const int nd = gr / G;
    if (nd >= si.ntok) continue;
    char* g = split ? (char*)(a.part_o + ((size_t)slot * 32 + rr) * HD)
                    : (char*)(a.out + (size_t)(si.tok0 + nd) * nq_hd + (it.kvh * G + gr % G) * HD);
    *(i32x4*)(g + ch * 16) = v;
  }
}

// Merge the partial states of a row tile's key ranges.  A 256-thread block
// takes RPB query rows of one item with HD/4 lanes per row, four consecutive
// dimensions per lane.  Split s holds its normalised output o_s / l_s and
// (m_s, l_s); its weight in the merged row is l_s 2^(m_s - M) with M the
// largest m_s.  A row's lanes share the weights, and every split's partial
// output is one 8-byte load per lane, four splits in flight at a time,
// accumulated in split order.
template <int HD>
__global__ __launch_bounds__(256) void attention_combine_kernel(AttnArgs a) {
  constexpr int LPR = HD / 4, RPB = 256 / LPR, MAXS = 64;
  __shared__ float wgt[RPB][MAXS];
  __shared__ float inv_l[RPB];
  const CombineItem ci = a.comb[blockIdx.x];
  const int lane = threadIdx.x % LPR, rr = threadIdx.x / LPR;
  const int row = blockIdx.y * RPB + rr;
  const SampleInfo si = a.samples[ci.sample];
  const int G = a.n_heads / a.n_kv_heads;
  const int gr = ci.row0 + row;
  const int nd = gr / G, hq = ci.kvh * G + gr % G;
  const bool live = nd < si.ntok;
  const int ns = live ? ci.nsplit : 0;
  float M = -INFINITY;
  for (int sp = lane; sp < ns; sp += LPR)
    M = fmaxf(M, a.part_ml[((size_t)(ci.part0 + sp) * 32 + row) * 2]);
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) M = fmaxf(M, __shfl_xor(M, m));
  float L = 0.f;
  for (int sp = lane; sp < ns; sp += LPR) {
    const size_t slot = (size_t)(ci.part0 + sp) * 32 + row;
    const float ms = a.part_ml[slot * 2];
    const float f = (ms == -INFINITY) ? 0.f : fast_exp2(ms - M) * a.part_ml[slot * 2 + 1];
    wgt[rr][sp] = f;
    L += f;
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) L += __shfl_xor(L, m);
  if (lane == 0) inv_l[rr] = 1.f / L;
  __syncthreads();
  if (!live) return;
  const f16* src = a.part_o + ((size_t)ci.part0 * 32 + row) * HD + 4 * lane;
  constexpr size_t STRIDE = (size_t)32 * HD;   // elements between consecutive splits
  f32x4 O = {0.f, 0.f, 0.f, 0.f};
  int sp = 0;
  for (; sp + 4 <= ns; sp += 4) {
    f16x4 p[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) p[u] = *(const f16x4*)(src + (sp + u) * STRIDE);
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int j = 0; j < 4; ++j) O[j] += wgt[rr][sp + u] * (float)p[u][j];
  }
  for (; sp < ns; ++sp) {
    const f16x4 p = *(const f16x4*)(src + sp * STRIDE);
#pragma unroll
    for (int j = 0; j < 4; ++j) O[j] += wgt[rr][sp] * (float)p[j];
  }
  bf16x4 v;
#pragma unroll
  for (int j = 0; j < 4; ++j) v[j] = (bf16)(O[j] * inv_l[rr]);
  *(bf16x4*)(a.out + (size_t)(si.tok0 + nd) * a.n_heads * HD + hq * HD + 4 * lane) = v;
}

template <int HD, int NW>
hipError_t launch_wide(const AttnArgs& a, const AttnItem* items, int n, hipStream_t s) {
  using C = AttnCfg<HD>;
  constexpr int SMEM = wide_stages<HD, NW>() * C::W_STAGE;
  static bool configured = false;
  if (!configured) {
    const hipError_t e = hipFuncSetAttribute((const void*)tree_attention_wide_kernel<HD, NW>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, SMEM);
    if (e != hipSuccess) return e;
    configured = true;
  }
  tree_attention_wide_kernel<HD, NW><<<(n + 7) / 8 * 8, 64 * NW, SMEM, s>>>(a, items, n);
  return hipSuccess;
}

template <int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t s) {
  using C = AttnCfg<HD>;
  static bool configured = false;
  if (!configured) {
    const hipError_t e = hipFuncSetAttribute((const void*)tree_attention_kernel<HD>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, C::SMEM);
    if (e != hipSuccess) return e;
    configured = true;
  }
  hipError_t e = hipSuccess;
  if (a.n_items) tree_attention_kernel<HD><<<(a.n_items + 7) / 8 * 8, C::NWN * 64, C::SMEM, s>>>(a);
  if (a.n_wide && e == hipSuccess) e = launch_wide<HD, 4>(a, a.wide, a.n_wide, s);
  if (a.n_wide8 && e == hipSuccess) e = launch_wide<HD, 8>(a, a.wide8, a.n_wide8, s);
  if (e != hipSuccess) return e;
  if (a.n_comb)
    attention_combine_kernel<HD><<<dim3(a.n_comb, 32 / (256 / (HD / 4))), 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_items == 0 && a.n_wide == 0 && a.n_wide8 == 0) return hipSuccess;
  if (a.head_dim == 128) return launch_hd<128>(a, s);
  if (a.head_dim == 64) return launch_hd<64>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace spec
