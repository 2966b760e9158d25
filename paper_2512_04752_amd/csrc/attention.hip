// Tree attention for the verify step.
//
// Query row r of (sample b, kv head g) is node r / G with query head
// g*G + r % G (G = n_heads / n_kv_heads query heads share one KV head).  It
// sees every committed key [0, S_b) and, of the tree keys at cache slots
// S_b + t, exactly its ancestors t (itself included), given as a bitmask.
//
// One work-group takes a tile of 32 query rows and a key range [key0, key1)
// (split-KV: long caches are cut into ranges processed in parallel and merged
// by the combine kernel).  Per step it stages 128 keys of K (row-major,
// chunk-swizzled) and V (transposed, [dim][key]) in LDS with coalesced 16-byte
// loads; wave w handles keys [32w, 32w+32) of the step:
//
//   S^T (32 keys x 32 rows) = K . Q^T   v_mfma_f32_32x32x16_bf16, A = K from LDS
//   online softmax per row              each lane owns one row (16 of its keys,
//                                       the other 16 in lane ^ 32)
//   O^T (dims x 32 rows) += V^T . P^T   A = V^T from LDS, B = P straight from
//                                       the S^T accumulator registers
//
// Computing the transposed products keeps a row's softmax state and its
// output column in the same lane, so rescaling needs no data movement.  At the
// end the four waves' partial states are merged through LDS.
#include <math.h>

#include "common.h"

namespace spec {

namespace {

constexpr int KB = 128;       // keys per step
constexpr int NT = 256;

template <int HD>
struct AttnSmem {
  static constexpr int VT_STRIDE = KB + 4;                       // bf16 per V^T row
  static constexpr int K_BYTES = KB * HD * 2;
  static constexpr int VT_BYTES = HD * VT_STRIDE * 2;
  static constexpr int O_STRIDE = HD + 1;                        // floats per merge row
  static constexpr int MERGE_BYTES = 4 * 32 * O_STRIDE * 4 + 4 * 32 * 2 * 4;
  static constexpr int BYTES = (K_BYTES + VT_BYTES) > MERGE_BYTES ? (K_BYTES + VT_BYTES) : MERGE_BYTES;
};

template <int HD>
__global__ __launch_bounds__(NT, 2) void tree_attention_kernel(AttnArgs a) {
  using SM = AttnSmem<HD>;
  constexpr int DC = HD / 8;                  // 16-byte chunks per row
  constexpr int KLOADS = KB * DC / NT;        // K chunks per thread per step
  constexpr int VPAIRS = (KB / 4) * DC / NT;  // (4-key group, chunk) pairs per thread
  constexpr int NB = HD / 32;                 // 32-dim output blocks
  __shared__ __attribute__((aligned(16))) char smem[SM::BYTES];
  char* k_lds = smem;
  bf16* vt_lds = (bf16*)(smem + SM::K_BYTES);

  const AttnItem it = a.items[blockIdx.x];
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

  const float sl2 = 1.4426950408889634f / sqrtf((float)HD);   // log2(e)/sqrt(d)
  float m_run = -INFINITY, l_run = 0.f;
  f32x16 o[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) o[i] = f32x16{};

  i32x4 kreg[KLOADS];
  i32x4 vreg[VPAIRS][4];
  auto gload = [&](int kb) {
#pragma unroll
    for (int i = 0; i < KLOADS; ++i) {
      const int q = tid + NT * i, key = q / DC, c = q % DC;
      kreg[i] = (kb + key < it.key1) ? *(const i32x4*)(kbase + (size_t)(kb + key) * HD + c * 8)
                                     : i32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < VPAIRS; ++i) {
      const int p = tid + NT * i, kg = p / DC, c = p % DC;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int key = kb + kg * 4 + j;
        vreg[i][j] = (key < it.key1) ? *(const i32x4*)(vbase + (size_t)key * HD + c * 8)
                                     : i32x4{0, 0, 0, 0};
      }
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int i = 0; i < KLOADS; ++i) {
      const int q = tid + NT * i, key = q / DC, c = q % DC;
      *(i32x4*)(k_lds + key * HD * 2 + ((c ^ (key & 7)) << 4)) = kreg[i];
    }
#pragma unroll
    for (int i = 0; i < VPAIRS; ++i) {
      const int p = tid + NT * i, kg = p / DC, c = p % DC;
      const bf16x8 v0 = __builtin_bit_cast(bf16x8, vreg[i][0]);
      const bf16x8 v1 = __builtin_bit_cast(bf16x8, vreg[i][1]);
      const bf16x8 v2 = __builtin_bit_cast(bf16x8, vreg[i][2]);
      const bf16x8 v3 = __builtin_bit_cast(bf16x8, vreg[i][3]);
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        const bf16x4 t = {v0[dd], v1[dd], v2[dd], v3[dd]};
        *(bf16x4*)(vt_lds + (c * 8 + dd) * SM::VT_STRIDE + kg * 4) = t;
      }
    }
  };

  if (it.key0 < it.key1) gload(it.key0);
  for (int kb = it.key0; kb < it.key1; kb += KB) {
    __syncthreads();                       // previous step's LDS reads are done
    sstore();
    __syncthreads();
    if (kb + KB < it.key1) gload(kb + KB); // next step's loads overlap this step's math

    // S^T = K . Q^T for keys [32w, 32w+32) of this step.
    f32x16 s = f32x16{};
    const int krow = w * 32 + r;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks) {
      const bf16x8 kf = *(const bf16x8*)(k_lds + krow * HD * 2 + (((2 * ks + h) ^ (krow & 7)) << 4));
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s, 0, 0, 0);
    }
    // Element e of this lane: key kb + 32w + 8*(e/4) + 4h + e%4 of row r.
    float smax = -INFINITY;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int key = kb + w * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      const int t = key - si.seq_len;
      const bool vis = key < it.key1 && (t < 0 || ((anc_row >> t) & 1ull));
      s[e] = vis ? s[e] * sl2 : -INFINITY;
      smax = fmaxf(smax, s[e]);
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
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int i = 0; i < NB; ++i) {
        const bf16* vp = vt_lds + (i * 32 + r) * SM::VT_STRIDE + w * 32 + 16 * st + 4 * h;
        const bf16x4 lo = *(const bf16x4*)vp;
        const bf16x4 hi = *(const bf16x4*)(vp + 8);
        const bf16x8 vf = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        o[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pb[st], o[i], 0, 0, 0);
      }
    }
  }
  l_run += __shfl_xor(l_run, 32);

  // Merge the four waves' (m, l, O) through LDS.
  __syncthreads();
  float* o_sh = (float*)smem;
  float* ml_sh = o_sh + 4 * 32 * SM::O_STRIDE;
  if (h == 0) {
    ml_sh[(w * 32 + r) * 2] = m_run;
    ml_sh[(w * 32 + r) * 2 + 1] = l_run;
  }
#pragma unroll
  for (int i = 0; i < NB; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int d = i * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
      o_sh[(w * 32 + r) * SM::O_STRIDE + d] = o[i][e];
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
      O += f * o_sh[(ww * 32 + row) * SM::O_STRIDE + d];
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

}  // namespace

hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.n_items == 0) return hipSuccess;
  if (a.head_dim == 128) {
    tree_attention_kernel<128><<<a.n_items, NT, 0, s>>>(a);
    if (a.n_comb) attention_combine_kernel<128><<<dim3(a.n_comb, 32), 128, 0, s>>>(a);
  } else if (a.head_dim == 64) {
    tree_attention_kernel<64><<<a.n_items, NT, 0, s>>>(a);
    if (a.n_comb) attention_combine_kernel<64><<<dim3(a.n_comb, 32), 64, 0, s>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace spec
