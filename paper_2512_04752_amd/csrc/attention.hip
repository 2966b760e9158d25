// Tree attention for the verify step.
//
// Query row r of (sample b, kv head g) is node r / G with query head
// g*G + r % G (G = n_heads / n_kv_heads query heads share one KV head).  It
// sees every committed key [0, S_b) and, of the tree keys at cache slots
// S_b + t, exactly its ancestors t (itself included), given as a bitmask.
//
// One work-group takes a tile of 32 query rows and a key range [key0, key1)
// of their cache (split-KV: long caches are cut into ranges processed in
// parallel and merged by the combine kernel).  The range is cut into blocks of
// 32 keys dealt round-robin to the 4 waves; each wave is an independent
// streaming worker with a private LDS ring that it fills itself with
// global_load_lds_dwordx4 (K and V rows copied verbatim, K chunk-swizzled), so
// the key loop needs no work-group barrier, only the wave's own vmcnt waits.
// Per 32-key block:
//
//   S^T (32 keys x 32 rows) = K . Q^T   v_mfma_f32_32x32x16_bf16, A = K (LDS)
//   online softmax per row              each lane owns one row (16 of its keys,
//                                       the other 16 in lane ^ 32)
//   O^T (dims x 32 rows) += V^T . P^T   A = V^T gathered from the row-major V
//                                       rows in LDS, B = P straight from the
//                                       S^T accumulator registers
//
// Computing the transposed products keeps a row's softmax state and its
// output column in the same lane, so rescaling needs no data movement.  At the
// end the four waves' partial states are merged through LDS.
#include <math.h>

#include "common.h"

namespace spec {

namespace {

constexpr int NT = 256, KBLK = 32;

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void load_lds16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds, 16, 0, 0);
}

template <int HD>
struct AttnCfg {
  static constexpr int ROW = HD * 2;                    // bytes per K or V row
  static constexpr int NST = HD == 128 ? 2 : 4;         // ring stages per wave
  static constexpr int KV_BYTES = KBLK * ROW;           // one block of K (or V)
  static constexpr int STAGE = 2 * KV_BYTES;
  static constexpr int WAVE_RING = NST * STAGE;         // 32 KB per wave
  static constexpr int LOADS = KV_BYTES / 1024;         // wave-loads for K (and for V)
  static constexpr int ROWS_PER_LOAD = 1024 / ROW;
  static constexpr int O_STRIDE = HD + 1;               // floats per merge row
  static constexpr int MERGE_BYTES = 4 * 32 * O_STRIDE * 4 + 4 * 32 * 2 * 4;
  static constexpr int SMEM = (4 * WAVE_RING) > MERGE_BYTES ? (4 * WAVE_RING) : MERGE_BYTES;
};

// Physical 16-byte chunk of logical chunk c in K row `key`: 16 consecutive
// rows reading one logical chunk hit 16 distinct 16-byte bank groups.
template <int HD>
__device__ __forceinline__ int kswz(int key) {
  return HD == 128 ? (key & 15) : ((key >> 1) & 7);
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  if constexpr (N == 0) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if constexpr (N == 8) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  else if constexpr (N == 16) asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
  else if constexpr (N == 24) asm volatile("s_waitcnt vmcnt(24)" ::: "memory");
  else static_assert(N < 0, "unsupported vmcnt");
}

template <int HD>
__global__ __launch_bounds__(NT, 1) void tree_attention_kernel(AttnArgs a) {
  using C = AttnCfg<HD>;
  constexpr int DC = HD / 8;                  // 16-byte chunks per row
  constexpr int NB = HD / 32;                 // 32-dim output blocks
  constexpr int LPS = 2 * C::LOADS;           // wave-loads per stage
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  // Items are dealt round-robin over the 8 XCDs; remap so that consecutive
  // items (the row tiles sharing one key range) run on one XCD.
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

  // Lane l of wave-load j copies row (j*ROWS_PER_LOAD + l / DC) of the block,
  // 16-byte chunk l % DC (physical); keys past the range repeat the last key,
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
      load_lds16(vbase + (size_t)key * HD + (lch << 3), st + C::KV_BYTES + j * 1024);
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
    const bf16* vt = (const bf16*)(st + C::KV_BYTES);
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
    // Element e of this lane: key kb + 8*(e/4) + 4h + e%4 of row r.  Blocks
    // wholly inside the committed prefix need no mask.
    float smax = -INFINITY;
    if (kb + KBLK <= si.seq_len && kb + KBLK <= it.key1) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        s[e] *= sl2;
        smax = fmaxf(smax, s[e]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int key = kb + 8 * (e >> 2) + 4 * h + (e & 3);
        const int tt = key - si.seq_len;
        const bool anc_bit = (anc_row >> (tt & 63)) & 1ull;
        const bool vis = (key < it.key1) & ((tt < 0) | anc_bit);
        s[e] = vis ? s[e] * sl2 : -INFINITY;
        smax = fmaxf(smax, s[e]);
      }
    }
    smax = fmaxf(smax, __shfl_xor(smax, 32));
    const float m_new = fmaxf(m_run, smax);
    const bool none = (m_new == -INFINITY);
    const float alpha = none ? 1.f : exp2f(m_run - m_new);
    float psum = 0.f;
    bf16x8 pb[2];
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

    // O^T += V^T . P^T.  Register slot j of k-step st (this lane's half h)
    // carries key 16*st + 8*(j/4) + 4h + j%4, matching the S^T layout.
#pragma unroll
    for (int kst = 0; kst < 2; ++kst) {
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const bf16* vp = vt + (16 * kst + 4 * h) * HD + i * 32 + r;
        bf16x8 vf;
#pragma unroll
        for (int j = 0; j < 8; ++j) vf[j] = vp[((j >> 2) * 8 + (j & 3)) * HD];
        o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[kst], o[i], 0, 0, 0);
      }
    }
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
  constexpr int SMEM = AttnCfg<HD>::SMEM;
  static bool configured = false;
  if (!configured) {
    const hipError_t e = hipFuncSetAttribute((const void*)tree_attention_kernel<HD>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, SMEM);
    if (e != hipSuccess) return e;
    configured = true;
  }
  const int grid = (a.n_items + 7) / 8 * 8;
  tree_attention_kernel<HD><<<grid, NT, SMEM, s>>>(a);
  if (a.n_comb) attention_combine_kernel<HD><<<dim3(a.n_comb, 32), HD, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  if (a.head_dim == 128) return launch_hd<128>(a, s);
  if (a.head_dim == 64) return launch_hd<64>(a, s);
  return hipErrorInvalidValue;
}

}  // namespace spec
