// Tree attention for the verify step.
//
// Query row r of (sample b, kv head g) is node r / G with query head
// g*G + r % G (G = n_heads / n_kv_heads query heads share one KV head).  It
// sees every committed key [0, S_b) and, of the tree keys at cache slots
// S_b + t, exactly its ancestors t (itself included), given as a bitmask.
//
// Both kernels process 32-key blocks per wave with the transposed products
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
//   * tree_attention_kernel: one 32-row tile per work-group (at most 32 query
//     rows per KV head, e.g. 8-node trees with 4 query heads per KV head).  The
//     key range is dealt to the 4 waves in 32-key blocks; each wave streams
//     its blocks through a private LDS ring (no work-group barrier), and the
//     four partial softmax states are merged through LDS at the end.
//   * tree_attention_wide_kernel: 128 query rows per work-group (larger
//     trees).  Wave w owns rows 32w..32w+31; all four waves share 64-key K/V
//     stages loaded cooperatively, so the range is read once per 128 rows, and
//     each wave ends with complete rows (no merge).
//
// Long key ranges are split into ranges processed in parallel and merged by
// attention_combine_kernel.
#include <math.h>

#include "common.h"

namespace spec {

namespace {

constexpr int NT = 256, KBLK = 32;

typedef __attribute__((address_space(3))) void lds_void;
typedef short v4i16 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void load_lds16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds, 16, 0, 0);
}

// Physical 16-byte chunk of logical chunk c in K row `key`: 16 consecutive
// rows reading one logical chunk hit 16 distinct 16-byte bank groups.
template <int HD>
__device__ __forceinline__ int kswz(int key) {
  return HD == 128 ? (key & 15) : ((key >> 1) & 7);
}
// V rows: the transposing read touches 4 consecutive rows x 32 bytes.
__device__ __forceinline__ int vswz(int key) { return (key & 3) << 1; }

template <int N>
__device__ __forceinline__ void wait_vm() {
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if constexpr (N == 16) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else if constexpr (N == 24) asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
  else static_assert(N < 0, "unsupported vmcnt");
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

// Online-softmax update of one 32-key block: masks, rescales o, returns P^T.
template <int NB>
__device__ __forceinline__ void softmax_block(f32x16& s, int kb, int key1, int seq_len, uint64_t anc,
                                              int h, float sl2, float& m_run, float& l_run,
                                              f32x16 (&o)[NB], bf16x8 (&pb)[2]) {
  float smax = -INFINITY;
  if (kb + KBLK <= seq_len && kb + KBLK <= key1) {       // wholly committed prefix: no mask
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      s[e] *= sl2;
      smax = fmaxf(smax, s[e]);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = kb + 8 * (e >> 2) + 4 * h + (e & 3);
      const int tt = key - seq_len;
      const bool anc_bit = (anc >> (tt & 63)) & 1ull;
      const bool vis = (key < key1) & ((tt < 0) | anc_bit);
      s[e] = vis ? s[e] * sl2 : -INFINITY;
      smax = fmaxf(smax, s[e]);
    }
  }
  smax = fmaxf(smax, __shfl_xor(smax, 32));
  const float m_new = fmaxf(m_run, smax);
  const bool none = (m_new == -INFINITY);
  const float alpha = none ? 1.f : exp2f(m_run - m_new);
  float psum = 0.f;
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const float pe = none ? 0.f : exp2f(s[e] - m_new);
    psum += pe;
    pb[e >> 3][e & 7] = (bf16)pe;
  }
  l_run = l_run * alpha + psum;
  m_run = m_new;
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] *= alpha;
}

template <int HD>
struct AttnCfg {
  static constexpr int ROW = HD * 2;                    // bytes per K or V row
  // narrow kernel: per-wave ring of 32-key blocks
  static constexpr int NST = HD == 128 ? 2 : 4;
  static constexpr int KV_BYTES = KBLK * ROW;
  static constexpr int STAGE = 2 * KV_BYTES;
  static constexpr int WAVE_RING = NST * STAGE;         // 32 KB per wave
  static constexpr int LOADS = KV_BYTES / 1024;         // wave-loads for K (and for V)
  static constexpr int ROWS_PER_LOAD = 1024 / ROW;
  static constexpr int O_STRIDE = HD + 1;               // floats per merge row
  static constexpr int MERGE_BYTES = 4 * 32 * O_STRIDE * 4 + 4 * 32 * 2 * 4;
  static constexpr int SMEM = (4 * WAVE_RING) > MERGE_BYTES ? (4 * WAVE_RING) : MERGE_BYTES;
  // wide kernel: shared 2-stage ring of 64-key stages
  static constexpr int WKEYS = 64;
  static constexpr int W_KV = WKEYS * ROW;              // K (or V) bytes per stage
  static constexpr int W_STAGE = 2 * W_KV;
  static constexpr int W_SMEM = 2 * W_STAGE;
  static constexpr int W_LOADS = W_KV / 1024 / 4;       // per wave, for K (and for V)
};

template <int HD>
__global__ __launch_bounds__(NT, 1) void tree_attention_kernel(AttnArgs a) {
  using C = AttnCfg<HD>;
  constexpr int DC = HD / 8;                  // 16-byte chunks per row
  constexpr int NB = HD / 32;                 // 32-dim output blocks
  constexpr int LPS = 2 * C::LOADS;           // wave-loads per stage
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  // Items are dealt round-robin over the 8 XCDs; remap so that consecutive
  // items run on one XCD.
  const int per_xcd = gridDim.x >> 3;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= a.n_items) return;
  const AttnItem it = a.items[item];
  if (it.sample < 0) return;          // padding of a shorter per-XCD list
  const SampleInfo si = a.samples[it.sample];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
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
  const uint64_t anc_row = row_ok ? a.anc[si.tok0 + node] : 1ull;

  const size_t head_stride = (size_t)si.cap * HD;
  const bf16* kbase = a.kv_pool + si.kv_base + ((size_t)a.layer * 2 * a.n_kv_heads + it.kvh) * head_stride;
  const bf16* vbase = kbase + (size_t)a.n_kv_heads * head_stride;
  char* ring = smem + w * C::WAVE_RING;

  // Blocks of this wave: w, w+4, w+8, ... of the item's range.
  const int nblk = (it.key1 - it.key0 + KBLK - 1) / KBLK;
  const int mine = nblk > w ? (nblk - w + 3) / 4 : 0;

  // Lane l of wave-load j copies row (j*ROWS_PER_LOAD + l / DC) of the block
  // into physical chunk l % DC; keys past the range repeat the last key,
  // whose scores are masked.
  const int lrow = lane / DC, lch = lane % DC;
  auto issue = [&](int t, int slot) {
    const int kb = it.key0 + (w + 4 * t) * KBLK;
    char* st = ring + slot * C::STAGE;
#pragma unroll
    for (int j = 0; j < C::LOADS; ++j) {
      const int row = j * C::ROWS_PER_LOAD + lrow;
      int key = kb + row;
      key = key < it.key1 ? key : it.key1 - 1;
      load_lds16(kbase + (size_t)key * HD + ((lch ^ kswz<HD>(row)) << 3), st + j * 1024);
      load_lds16(vbase + (size_t)key * HD + ((lch ^ vswz(row)) << 3), st + C::KV_BYTES + j * 1024);
    }
  };

  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e)/sqrt(d)
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x16{};

#pragma unroll
  for (int t = 0; t < C::NST - 1; ++t)
    if (t < mine) issue(t, t);

  for (int t = 0; t < mine; ++t) {
    // Keep NST-1 blocks in flight: issue block t+NST-1 into the slot of block
    // t-1 (consumed in the previous iteration), then wait for block t.
    if (t + C::NST - 1 < mine) {
      issue(t + C::NST - 1, (t + C::NST - 1) % C::NST);
      wait_vm<LPS * (C::NST - 1)>();
    } else {
      wait_vm<0>();
    }
    const char* st = ring + (t % C::NST) * C::STAGE;
    const int kb = it.key0 + (w + 4 * t) * KBLK;

    // S^T = K . Q^T for the 32 keys of this block (two independent chains).
    f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
    for (int ks = 0; ks < HD / 16; ks += 2) {
      const bf16x8 k0 = *(const bf16x8*)(st + r * C::ROW + (((2 * ks + h) ^ kswz<HD>(r)) << 4));
      const bf16x8 k1 = *(const bf16x8*)(st + r * C::ROW + (((2 * ks + 2 + h) ^ kswz<HD>(r)) << 4));
      s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[ks], s0, 0, 0, 0);
      s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[ks + 1], s1, 0, 0, 0);
    }
    f32x16 s = s0 + s1;
    bf16x8 pb[2];
    softmax_block<NB>(s, kb, it.key1, si.seq_len, anc_row, h, sl2, m_run, l_run, o, pb);

    // O^T += V^T . P^T
#pragma unroll
    for (int kst = 0; kst < 2; ++kst)
#pragma unroll
      for (int i = 0; i < NB; ++i)
        o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vt_fragment<HD>(st + C::KV_BYTES, kst, i, lane),
                                                      pb[kst], o[i], 0, 0, 0);
  }
  l_run += __shfl_xor(l_run, 32);

  // Merge the four waves' (m, l, O) through LDS.
  __syncthreads();
  float* o_sh = (float*)smem;
  float* ml_sh = o_sh + 4 * 32 * C::O_STRIDE;
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

  for (int idx = tid; idx < 32 * HD; idx += NT) {
    const int row = idx / HD, d = idx % HD;
    const int gr = it.row0 + row;
    const int nd = gr / G, hq = it.kvh * G + gr % G;
    if (nd >= si.ntok) continue;
    float M = -INFINITY;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) M = fmaxf(M, ml_sh[(ww * 32 + row) * 2]);
    float O = 0.f, L = 0.f;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) {
      const float mw = ml_sh[(ww * 32 + row) * 2];
      const float f = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
      O += f * o_sh[(ww * 32 + row) * C::O_STRIDE + d];
      L += f * ml_sh[(ww * 32 + row) * 2 + 1];
    }
    if (it.nsplit == 1) {
      a.out[(size_t)(si.tok0 + nd) * nq_hd + hq * HD + d] = (bf16)(O / L);
    } else {
      a.part_o[((size_t)it.part * 32 + row) * HD + d] = O;
      if (d == 0) {
        a.part_ml[((size_t)it.part * 32 + row) * 2] = M;
        a.part_ml[((size_t)it.part * 32 + row) * 2 + 1] = L;
      }
    }
  }
}

// 128 query rows per work-group: wave w owns rows it.row0 + 32w .. +31 and
// all keys of the range, streamed in shared 64-key stages (two-stage ring,
// one barrier per stage).  With the range split, wave w's partial state goes
// to slot it.part + w * it.nsplit (its row tile's slot for this split).
template <int HD>
__global__ __launch_bounds__(NT, 2) void tree_attention_wide_kernel(AttnArgs a) {
  using C = AttnCfg<HD>;
  constexpr int DC = HD / 8;
  constexpr int NB = HD / 32;
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  const int per_xcd = gridDim.x >> 3;
  const int item = (blockIdx.x & 7) * per_xcd + (blockIdx.x >> 3);
  if (item >= a.n_wide) return;
  const AttnItem it = a.wide[item];
  if (it.sample < 0) return;
  const SampleInfo si = a.samples[it.sample];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
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
  const uint64_t anc_row = row_ok ? a.anc[si.tok0 + node] : 1ull;

  const size_t head_stride = (size_t)si.cap * HD;
  const bf16* kbase = a.kv_pool + si.kv_base + ((size_t)a.layer * 2 * a.n_kv_heads + it.kvh) * head_stride;
  const bf16* vbase = kbase + (size_t)a.n_kv_heads * head_stride;

  const int nstage = (it.key1 - it.key0 + C::WKEYS - 1) / C::WKEYS;
  // Wave w loads rows [16w, 16w+16) of each stage's K and V.
  const int lrow = lane / DC, lch = lane % DC;
  auto issue = [&](int t, int slot) {
    const int kb = it.key0 + t * C::WKEYS;
    char* st = smem + slot * C::W_STAGE;
#pragma unroll
    for (int j = 0; j < C::W_LOADS; ++j) {
      const int row = (w * C::W_LOADS + j) * C::ROWS_PER_LOAD + lrow;
      int key = kb + row;
      key = key < it.key1 ? key : it.key1 - 1;
      load_lds16(kbase + (size_t)key * HD + ((lch ^ kswz<HD>(row)) << 3),
                 st + (w * C::W_LOADS + j) * 1024);
      load_lds16(vbase + (size_t)key * HD + ((lch ^ vswz(row)) << 3),
                 st + C::W_KV + (w * C::W_LOADS + j) * 1024);
    }
  };

  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x16{};

  if (nstage > 0) issue(0, 0);
  for (int t = 0; t < nstage; ++t) {
    wait_vm<0>();
    __syncthreads();      // stage t visible to all waves; stage t-1 fully consumed
    if (t + 1 < nstage) issue(t + 1, (t + 1) & 1);
    const char* st = smem + (t & 1) * C::W_STAGE;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const char* kblk = st + half * KBLK * C::ROW;
      const int kb = it.key0 + t * C::WKEYS + half * KBLK;
      f32x16 s0 = f32x16{}, s1 = f32x16{};
#pragma unroll
      for (int ks = 0; ks < HD / 16; ks += 2) {
        const int krow = half * KBLK + r;
        const bf16x8 k0 = *(const bf16x8*)(kblk + r * C::ROW + (((2 * ks + h) ^ kswz<HD>(krow)) << 4));
        const bf16x8 k1 = *(const bf16x8*)(kblk + r * C::ROW + (((2 * ks + 2 + h) ^ kswz<HD>(krow)) << 4));
        s0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0, qf[ks], s0, 0, 0, 0);
        s1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1, qf[ks + 1], s1, 0, 0, 0);
      }
      f32x16 s = s0 + s1;
      bf16x8 pb[2];
      softmax_block<NB>(s, kb, it.key1, si.seq_len, anc_row, h, sl2, m_run, l_run, o, pb);
      const char* vblk = st + C::W_KV + half * KBLK * C::ROW;
#pragma unroll
      for (int kst = 0; kst < 2; ++kst)
#pragma unroll
        for (int i = 0; i < NB; ++i)
          o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vt_fragment<HD>(vblk, kst, i, lane), pb[kst],
                                                        o[i], 0, 0, 0);
    }
  }
  l_run += __shfl_xor(l_run, 32);

  // Lane (r, h) holds dims 32i + 8(e/4) + 4h + e%4 of row r.
  if (!row_ok) return;
  const int slot = it.part + w * it.nsplit;
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int d = i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      if (it.nsplit == 1)
        a.out[(size_t)(si.tok0 + node) * nq_hd + head * HD + d] = (bf16)(o[i][e] / l_run);
      else
        a.part_o[((size_t)slot * 32 + r) * HD + d] = o[i][e];
    }
  if (it.nsplit > 1 && h == 0) {
    a.part_ml[((size_t)slot * 32 + r) * 2] = m_run;
    a.part_ml[((size_t)slot * 32 + r) * 2 + 1] = l_run;
  }
}

// Merge the partial states of a row tile's key ranges: one block per query
// row, one thread per head dimension; the per-split weights are computed once
// into LDS and every split's partial output is an independent load.
template <int HD>
__global__ __launch_bounds__(HD) void attention_combine_kernel(AttnArgs a) {
  constexpr int MAXS = 64;
  __shared__ float wgt[MAXS];
  __shared__ float inv_l;
  const CombineItem ci = a.comb[blockIdx.x];
  const int row = blockIdx.y;
  const SampleInfo si = a.samples[ci.sample];
  const int G = a.n_heads / a.n_kv_heads;
  const int gr = ci.row0 + row;
  const int nd = gr / G, hq = ci.kvh * G + gr % G;
  if (nd >= si.ntok) return;
  const int d = threadIdx.x;
  if (d < 64) {
    float M = -INFINITY;
    for (int sp = d; sp < ci.nsplit; sp += 64)
      M = fmaxf(M, a.part_ml[((size_t)(ci.part0 + sp) * 32 + row) * 2]);
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) M = fmaxf(M, __shfl_xor(M, m));
    float L = 0.f;
    for (int sp = d; sp < ci.nsplit; sp += 64) {
      const size_t slot = (size_t)(ci.part0 + sp) * 32 + row;
      const float ms = a.part_ml[slot * 2];
      const float f = (ms == -INFINITY) ? 0.f : exp2f(ms - M);
      if (sp < MAXS) wgt[sp] = f;
      L += f * a.part_ml[slot * 2 + 1];
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) L += __shfl_xor(L, m);
    if (d == 0) inv_l = 1.f / L;
  }
  __syncthreads();
  float O = 0.f;
  for (int sp = 0; sp < ci.nsplit; ++sp)
    O += wgt[sp] * a.part_o[((size_t)(ci.part0 + sp) * 32 + row) * HD + d];
  a.out[(size_t)(si.tok0 + nd) * a.n_heads * HD + hq * HD + d] = (bf16)(O * inv_l);
}

template <int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t s) {
  using C = AttnCfg<HD>;
  static bool configured = false;
  if (!configured) {
    hipError_t e = hipFuncSetAttribute((const void*)tree_attention_kernel<HD>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, C::SMEM);
    if (e != hipSuccess) return e;
    e = hipFuncSetAttribute((const void*)tree_attention_wide_kernel<HD>,
                            hipFuncAttributeMaxDynamicSharedMemorySize, C::W_SMEM);
    if (e != hipSuccess) return e;
    configured = true;
  }
  if (a.n_items) tree_attention_kernel<HD><<<(a.n_items + 7) / 8 * 8, NT, C::SMEM, s>>>(a);
  if (a.n_wide) tree_attention_wide_kernel<HD><<<(a.n_wide + 7) / 8 * 8, NT, C::W_SMEM, s>>>(a);
  if (a.n_comb) attention_combine_kernel<HD><<<dim3(a.n_comb, 32), HD, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_items == 0 && a.n_wide == 0) return hipSuccess;
  if (a.head_dim == 128) return launch_hd<128>(a, s);
  if (a.head_dim == 64) return launch_hd<64>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace spec
