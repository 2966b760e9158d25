// bf16 GEMM on gfx950 matrix cores: C[M][N] = A[M][K] . B[N][K]^T with fp32
// accumulation and a fused epilogue per use in the verify forward pass:
//
//   EPI_QKV      q/k/v projections; rotary embedding of q and k; q goes to a
//                workspace buffer, k and v straight into the KV cache at the
//                node's slot S_b + node
//   EPI_RESID    o-projection / down-projection, added into the fp32
//                residual stream
//   EPI_GATE_UP  gate and up projections of the same features side by side,
//                emitting silu(gate) * up in bf16
//   EPI_ARGMAX   LM head: per row, the (max, lowest index) over each 64
//                columns, optionally also the fp32 logits
//
// Tiling: 128 x 128 output tile per 256-thread work-group (4 waves, 2 x 2,
// 64 x 64 each), K step 64, two LDS buffers (64 KB) so that one barrier per
// K step suffices; the next K slice is fetched into registers while the
// current one feeds v_mfma_f32_32x32x16_bf16.  Both operands are K-major, so
// every lane reads 16 contiguous bytes per MFMA operand.  LDS rows are 128 B
// with the 16-byte chunk index XOR-swizzled by (row & 7).
//
// Work-groups are dispatched round-robin over the 8 XCDs; the tile order is
// remapped so that the M tiles sharing one weight tile run on the same XCD
// and hit its L2 instead of HBM.
#include "common.h"

namespace spec {

namespace {

constexpr int BM = 128, BN = 128, BK = 64, NT = 256;

__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * 128 + ((chunk ^ (row & 7)) << 4);
}

// Weight row feeding tile-local virtual column u of column tile tn.
template <int EPI>
__device__ __forceinline__ const bf16* weight_row(const GemmArgs& a, int tn, int u) {
  if constexpr (EPI == EPI_QKV) {
    // Virtual order: each wave's two 32-column MFMA blocks hold head dims j
    // and j + head_dim/2, so the rotary pairs meet in one lane.
    const int vs = tn * BN;
    const bf16* base;
    int local;
    if (vs < a.n0) { base = a.B0; local = vs; }
    else if (vs < a.n0 + a.n1) { base = a.B1; local = vs - a.n0; }
    else { base = a.B2; local = vs - a.n0 - a.n1; }
    const int hd = a.head_dim, qpd = hd / 64;
    const int wn = u >> 6, blk = (u >> 5) & 1, c = u & 31;
    const int head = wn / qpd;
    const int dim = (wn % qpd) * 32 + blk * (hd / 2) + c;
    return base + (size_t)(local + head * hd + dim) * a.K;
  } else if constexpr (EPI == EPI_GATE_UP) {
    const int f = tn * 64 + (u >> 6) * 32 + (u & 31);
    return (((u >> 5) & 1) ? a.B1 : a.B0) + (size_t)f * a.K;
  } else {
    return a.B0 + (size_t)(tn * BN + u) * a.K;
  }
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

template <int EPI>
__global__ __launch_bounds__(NT, 2) void gemm_bf16_kernel(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[2][2][BM * BK * 2];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int ntm = (a.M + BM - 1) / BM;
  const int total = gridDim.x;
  int bid = blockIdx.x;
  if ((total & 7) == 0) bid = (bid & 7) * (total >> 3) + (bid >> 3);
  const int tm = bid % ntm, tn = bid / ntm;

  // Global -> register loader: 4 rows x one 16-byte chunk of A and of B.
  const int lrow = tid >> 3, lchunk = tid & 7;
  const bf16* pa[4];
  const bf16* pb[4];
  bool oka[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int row = lrow + 32 * r;
    const int grow = tm * BM + row;
    oka[r] = grow < a.M;
    pa[r] = a.A + (size_t)(oka[r] ? grow : 0) * a.K + lchunk * 8;
    pb[r] = weight_row<EPI>(a, tn, row) + lchunk * 8;
  }
  i32x4 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      ra[r] = oka[r] ? *(const i32x4*)(pa[r] + k0) : i32x4{0, 0, 0, 0};
      rb[r] = *(const i32x4*)(pb[r] + k0);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int off = lds_off(lrow + 32 * r, lchunk);
      *(i32x4*)(smem[buf][0] + off) = ra[r];
      *(i32x4*)(smem[buf][1] + off) = rb[r];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  const int wm = wave >> 1, wn = wave & 1;
  const int KT = a.K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < KT) gload((kt + 1) * BK);
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      const int chunk = ks * 2 + (lane >> 5);
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        af[i] = *(const bf16x8*)(smem[cur][0] + lds_off(wm * 64 + i * 32 + (lane & 31), chunk));
        bfr[i] = *(const bf16x8*)(smem[cur][1] + lds_off(wn * 64 + i * 32 + (lane & 31), chunk));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < KT) sstore(cur ^ 1);
    __syncthreads();
  }

  // Accumulator layout of a 32x32 block: lane l, element e holds
  // row 8*(e/4) + 4*(l/32) + e%4, column l%32.
  const int c = lane & 31;
  const int rbase = tm * BM + wm * 64 + 4 * (lane >> 5);

  if constexpr (EPI == EPI_RESID) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          if (row < a.M) {
            float* px = a.x + (size_t)row * a.N + tn * BN + wn * 64 + j * 32 + c;
            *px += acc[i][j][e];
          }
        }
  } else if constexpr (EPI == EPI_GATE_UP) {
    const int F = a.N / 2;
    const int f = tn * 64 + wn * 32 + c;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
        if (row < a.M) a.act_out[(size_t)row * F + f] = (bf16)(silu(acc[i][0][e]) * acc[i][1][e]);
      }
  } else if constexpr (EPI == EPI_QKV) {
    const int vs = tn * BN;
    int seg, local;
    if (vs < a.n0) { seg = 0; local = vs; }
    else if (vs < a.n0 + a.n1) { seg = 1; local = vs - a.n0; }
    else { seg = 2; local = vs - a.n0 - a.n1; }
    const int hd = a.head_dim, qpd = hd / 64, half = hd / 2;
    const int head = local / hd + wn / qpd;
    const int fi = (wn % qpd) * 32 + c;             // rotary frequency index, < hd/2
    const int dim = fi;                             // first element of the pair
    const int nq_hd = a.n0;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
        if (row >= a.M) continue;
        float x1 = acc[i][0][e], x2 = acc[i][1][e];
        if (seg < 2) {
          const float2 cs = a.rope_cs[(size_t)row * half + fi];
          const float y1 = x1 * cs.x - x2 * cs.y;
          const float y2 = x2 * cs.x + x1 * cs.y;
          x1 = y1;
          x2 = y2;
        }
        if (seg == 0) {
          bf16* pq = a.q_out + (size_t)row * nq_hd + head * hd + dim;
          pq[0] = (bf16)x1;
          pq[half] = (bf16)x2;
        } else {
          const TokInfo t = a.toks[row];
          const SampleInfo s = a.samples[t.sample];
          const int slot = s.seq_len + t.node;
          bf16* p = a.kv_pool + s.kv_base +
                    ((((size_t)a.layer * 2 + (seg - 1)) * a.n_kv_heads + head) * s.cap + slot) * hd +
                    dim;
          p[0] = (bf16)x1;
          p[half] = (bf16)x2;
        }
      }
  } else {  // EPI_ARGMAX
    const int col0 = tn * BN + wn * 64 + c;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
        float v = acc[i][0][e];
        int idx = col0;
        const float v2 = acc[i][1][e];
        if (v2 > v) { v = v2; idx = col0 + 32; }
        if (a.logits != nullptr && row < a.M) {
          a.logits[(size_t)row * a.N + col0] = acc[i][0][e];
          a.logits[(size_t)row * a.N + col0 + 32] = v2;
        }
#pragma unroll
        for (int m = 16; m >= 1; m >>= 1) {
          const float ov = __shfl_xor(v, m);
          const int oi = __shfl_xor(idx, m);
          if (ov > v || (ov == v && oi < idx)) { v = ov; idx = oi; }
        }
        if (c == 0 && row < a.M) {
          const int parts = a.N / 64;
          a.part_val[(size_t)row * parts + tn * 2 + wn] = v;
          a.part_idx[(size_t)row * parts + tn * 2 + wn] = idx;
        }
      }
  }
}

}  // namespace

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s) {
  const int ntm = (a.M + BM - 1) / BM;
  const int ntn = a.N / BN;
  const dim3 grid(ntm * ntn), block(NT);
  switch (epi) {
    case EPI_QKV: gemm_bf16_kernel<EPI_QKV><<<grid, block, 0, s>>>(a); break;
    case EPI_RESID: gemm_bf16_kernel<EPI_RESID><<<grid, block, 0, s>>>(a); break;
    case EPI_GATE_UP: gemm_bf16_kernel<EPI_GATE_UP><<<grid, block, 0, s>>>(a); break;
    case EPI_ARGMAX: gemm_bf16_kernel<EPI_ARGMAX><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace spec
