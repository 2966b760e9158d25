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
//   EPI_ARGMAX   LM head: per row, the (max, lowest index) over each wave's
//                column slab, optionally also the fp32 logits
//
// Structure (one work-group = NW = 4 or 8 waves in a WM x WN grid, output
// tile BM x BN, each wave BM/WM x BN/WN built from 32 x 32
// v_mfma_f32_32x32x16_bf16 blocks; K step BK = 64 or 32):
//   * operand tiles move HBM/L2 -> LDS with global_load_lds_dwordx4 (no
//     register staging) into a ring of NS stages; the next NS-1 K steps are
//     in flight while the current one is multiplied, and one barrier per K
//     step both publishes the next stage and frees the oldest slot.  The
//     barrier waits only for this wave's LDS reads and for the loads of the
//     next stage (vmcnt counts the later stages out), never for the whole
//     ring.  A stage's wave-loads are issued in BK/16 parts between the MFMA
//     blocks, with their LDS destinations in scalar registers;
//   * each wave-load writes 1 KB = 8 tile rows of 128 bytes (16 of 64 bytes
//     for BK = 32); the 16-byte chunk index of row r is XOR-ed with
//     (r >> 1) & 7 ((r >> 2) & 3), which makes the MFMA operand reads (16
//     consecutive rows, one chunk) hit all 64 LDS banks once;
//   * fragments of the next 16-wide k-step are read from LDS into a second
//     register set while the current set feeds the MFMAs.
// Tile shapes (pick_tile): 256 x 256 (8 waves of 128 x 64, 4 stages of 32)
// and 256 x 128 (8 waves of 64 x 64, 3 stages of 64) for many rows: two
// waves per SIMD, so one wave's MFMAs cover the other's waits and barrier;
// 128 x 128 (4 waves, 4 stages) for up to 128 rows or narrow products, and
// 32 x 256 / 64 x 256 (4 waves, 3 stages) for few rows, where the weights
// are streamed.  Work-groups are
// dealt round-robin over the 8 XCDs; the tile order is remapped so that the
// M tiles sharing one weight tile run on one XCD and hit its L2.
//
// Products with too few output tiles to fill the CUs split K: each split
// writes its fp32 tile to a partial buffer and a second kernel sums the splits
// in a fixed order (bitwise reproducible) and applies the same epilogue.
#include <algorithm>

#include "common.h"

namespace spec {

namespace {

constexpr size_t kPartialCap = 64ull << 20;   // bytes of split-K partials (workspace)

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void load_lds16(const void* g, void* lds) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds, 16, 0, 0);
}

// 16-byte chunk swizzle of tile row `row` for K steps of BK elements (rows of
// 2*BK bytes): 16 consecutive rows reading one logical chunk hit 16
// distinct 16-byte bank groups.
template <int BK>
__device__ __forceinline__ int swz(int row) { return BK == 64 ? (row >> 1) & 7 : (row >> 2) & 3; }

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Work-group barrier for the LDS ring: this wave's LDS reads are complete
// (its slot may be refilled by any wave afterwards), but its direct-to-LDS
// loads of later stages stay in flight.  __syncthreads() would add a
// work-group fence, i.e. a wait for every outstanding global load, which
// would leave only one stage of lookahead however deep the ring.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Virtual-column mapping.  Column u of an output tile belongs to wave column
// wn = u / TN, MFMA block nb = (u % TN) / 32, lane column c = u % 32.  For
// EPI_QKV and EPI_GATE_UP, blocks (2p, 2p+1) of a wave column form pair
// P = (u % BN) / 64 of the tile: rotary partners (dims j, j + d/2) or
// (gate, up) of one feature.
template <int EPI, int BN>
__device__ __forceinline__ const bf16* weight_row(const GemmArgs& a, int tn, int u) {
  const int P = u >> 6, blk = (u >> 5) & 1, c = u & 31;
  if constexpr (EPI == EPI_QKV) {
    const int vs = tn * BN;
    const bf16* base;
    int local;
    if (vs < a.n0) { base = a.B0; local = vs; }
    else if (vs < a.n0 + a.n1) { base = a.B1; local = vs - a.n0; }
    else { base = a.B2; local = vs - a.n0 - a.n1; }
    const int hd = a.head_dim, qpd = hd / 64;
    const int head = P / qpd, dim = (P % qpd) * 32 + blk * (hd / 2) + c;
    return base + (size_t)(local + head * hd + dim) * a.K;
  } else if constexpr (EPI == EPI_GATE_UP) {
    const int f = tn * (BN / 2) + P * 32 + c;
    return (blk ? a.B1 : a.B0) + (size_t)f * a.K;
  } else {
    return a.B0 + (size_t)(tn * BN + u) * a.K;
  }
}

__device__ __forceinline__ float silu(float g) { return g / (1.0f + __expf(-g)); }

// Pair epilogues: (x1, x2) are the two members of pair P of tile tn, lane
// column c, output row `row`.
template <int BN>
__device__ __forceinline__ void epi_qkv(const GemmArgs& a, int row, int tn, int P, int c, float x1,
                                        float x2) {
  const int vs = tn * BN;
  int seg, local;
  if (vs < a.n0) { seg = 0; local = vs; }
  else if (vs < a.n0 + a.n1) { seg = 1; local = vs - a.n0; }
  else { seg = 2; local = vs - a.n0 - a.n1; }
  const int hd = a.head_dim, qpd = hd / 64, half = hd / 2;
  const int head = local / hd + P / qpd;
  const int fi = (P % qpd) * 32 + c;           // rotary frequency index = first dim of the pair
  if (seg < 2) {
    const float2 cs = a.rope_cs[(size_t)row * half + fi];
    const float y1 = x1 * cs.x - x2 * cs.y;
    const float y2 = x2 * cs.x + x1 * cs.y;
    x1 = y1;
    x2 = y2;
  }
  if (seg == 0) {
    bf16* pq = a.q_out + (size_t)row * a.n0 + head * hd + fi;
    pq[0] = (bf16)x1;
    pq[half] = (bf16)x2;
  } else {
    const TokInfo t = a.toks[row];
    const SampleInfo s = a.samples[t.sample];
    const int slot = s.seq_len + t.node;
    bf16* pk = a.kv_pool + s.kv_base +
               ((((size_t)a.layer * 2 + (seg - 1)) * a.n_kv_heads + head) * s.cap + slot) * hd + fi;
    pk[0] = (bf16)x1;
    pk[half] = (bf16)x2;
  }
}

template <int BN>
__device__ __forceinline__ void epi_gate_up(const GemmArgs& a, int row, int tn, int P, int c,
                                            float g, float u) {
  const int f = tn * (BN / 2) + P * 32 + c;
  a.act_out[(size_t)row * (a.N / 2) + f] = (bf16)(silu(g) * u);
}

// Work-groups per CU a tile configuration is compiled for: two when its ring
// leaves room for a second one in the 160 KB of LDS and its accumulators
// leave room for a second wave per SIMD, so that one wave's waits are
// covered by the other's MFMAs.
template <int BM, int BN, int NS, int BK>
constexpr int gemm_occupancy() {
  return (NS * (BM + BN) * BK * 2 <= 80 * 1024 && BM * BN <= 256 * 128) ? 2 : 1;
}

template <int EPI, int BM, int BN, int WM, int NS, int BK, int NW = 4>
__global__ __launch_bounds__(NW * 64, (gemm_occupancy<BM, BN, NS, BK>())) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int WN = NW / WM;
  constexpr int TM = BM / WM, TN = BN / WN, MB = TM / 32, NB = TN / 32;
  constexpr int ROWB = BK * 2, CPR = BK / 8, RPL = 1024 / ROWB;  // row bytes, chunks, rows per load
  constexpr int KS = BK / 16;                                     // MFMA k-steps per K step
  constexpr int A_BYTES = BM * ROWB, STAGE = (BM + BN) * ROWB;
  constexpr int A_LOADS = A_BYTES / 1024 / NW, B_LOADS = BN * ROWB / 1024 / NW;
  constexpr int LPW = A_LOADS + B_LOADS;    // wave-loads per wave and stage
  static_assert(BK == 32 || BK == 64, "K step");
  static_assert(MB >= 1 && NB >= 2 && A_LOADS >= 1 && B_LOADS >= 1, "tile shape");
  static_assert(A_BYTES % (1024 * NW) == 0 && BN * ROWB % (1024 * NW) == 0, "loads per wave");
  static_assert(NS >= 2 && (NS - 2) * LPW <= 63, "ring depth (vmcnt holds at most 63)");
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  // The wave index is made scalar so that every LDS destination (M0) of the
  // direct loads is computed in scalar registers.
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int ntm = (a.M + BM - 1) / BM;
  const int tiles = ntm * (a.N / BN);
  // Work-group b runs on XCD b % 8, which receives q + 1 work-groups (x < r)
  // or q (x >= r) for a grid of 8q + r.  Give each XCD a contiguous range of
  // logical ids, so that the M tiles sharing a weight tile (adjacent ids)
  // meet in one XCD's L2.
  const int total = gridDim.x;
  int bid = blockIdx.x;
  {
    const int q = total >> 3, r = total & 7, x = bid & 7, j = bid >> 3;
    bid = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + j;
  }
  const int tile = bid % tiles, split = bid / tiles;
  const int tm = tile % ntm, tn = tile / ntm;
  const int KT = a.K / BK / a.ksplit;            // K steps of this split
  const int k_off = split * KT * BK;

  // Wave-load j of this wave fills tile rows [(wave*LOADS + j)*RPL, +RPL);
  // lane l lands at row l/CPR, physical chunk l%CPR, so it fetches logical
  // chunk (l%CPR) ^ swz(row).
  const int lr = lane / CPR, lc = lane % CPR;
  const bf16* pa[A_LOADS];
  const bf16* pb[B_LOADS];
#pragma unroll
  for (int j = 0; j < A_LOADS; ++j) {
    const int trow = (wave * A_LOADS + j) * RPL + lr;
    int row = tm * BM + trow;
    row = row < a.M ? row : a.M - 1;      // rows past M repeat the last row; never stored
    pa[j] = a.A + (size_t)row * a.K + k_off + ((lc ^ swz<BK>(trow)) << 3);
  }
#pragma unroll
  for (int j = 0; j < B_LOADS; ++j) {
    const int trow = (wave * B_LOADS + j) * RPL + lr;
    pb[j] = weight_row<EPI, BN>(a, tn, trow) + k_off + ((lc ^ swz<BK>(trow)) << 3);
  }
  // Part q of stage kt's loads (every KS-th wave-load), so that a stage's
  // loads are spread between the MFMA blocks of a K step instead of issued
  // in one burst.
  auto issue_q = [&](int kt, int slot, int q) {
    char* base = smem + slot * STAGE;
#pragma unroll
    for (int j = 0; j < A_LOADS; ++j)
      if (j % KS == q) load_lds16(pa[j] + kt * BK, base + (wave * A_LOADS + j) * 1024);
#pragma unroll
    for (int j = 0; j < B_LOADS; ++j)
      if (j % KS == q) load_lds16(pb[j] + kt * BK, base + A_BYTES + (wave * B_LOADS + j) * 1024);
  };

  f32x16 acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < NB; ++j) acc[i][j] = f32x16{};

  const int wm = wave / WN, wn = wave % WN;
  int arow[MB], brow[NB];
#pragma unroll
  for (int i = 0; i < MB; ++i) arow[i] = wm * TM + i * 32 + (lane & 31);
#pragma unroll
  for (int j = 0; j < NB; ++j) brow[j] = wn * TN + j * 32 + (lane & 31);

  bf16x8 fa[2][MB], fb[2][NB];
  auto load_frags = [&](const char* st, int ks, int set) {
    const int chunk = ks * 2 + (lane >> 5);
#pragma unroll
    for (int i = 0; i < MB; ++i)
      fa[set][i] = *(const bf16x8*)(st + arow[i] * ROWB + ((chunk ^ swz<BK>(arow[i])) << 4));
#pragma unroll
    for (int j = 0; j < NB; ++j)
      fb[set][j] = *(const bf16x8*)(st + A_BYTES + brow[j] * ROWB + ((chunk ^ swz<BK>(brow[j])) << 4));
  };
  auto mfmas = [&](int set) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][i], fb[set][j], acc[i][j], 0, 0, 0);
  };

  // Prologue: stages 0 .. NS-2 in flight, wait for stage 0.
#pragma unroll
  for (int st = 0; st < NS - 1; ++st)
    if (st < KT) {
#pragma unroll
      for (int q = 0; q < KS; ++q) issue_q(st, st, q);
    }
  if (KT >= NS - 1) wait_vm<(NS - 2) * LPW>();
  else wait_vm<0>();
  ring_barrier();
  // Stage pk (slot ps) is issued part by part between the MFMA blocks of the
  // current step; -1 when none is left.
  int pk = NS - 1 < KT ? NS - 1 : -1, ps = NS - 1;
  if (pk >= 0) issue_q(pk, ps, 0);
  load_frags(smem, 0, 0);
  for (int kt = 0; kt < KT; ++kt) {
    const char* st = smem + (kt % NS) * STAGE;
#pragma unroll
    for (int ks = 0; ks + 1 < KS; ++ks) {
      load_frags(st, ks + 1, (ks + 1) & 1);
      if (pk >= 0) issue_q(pk, ps, ks + 1);
      mfmas(ks & 1);
    }
    pk = -1;
    if (kt + 1 < KT) {
      // Stage kt+1 has landed for every wave (stages kt+2 .. kt+NS-1 may
      // still be in flight), and every wave is done reading stage kt (its
      // last fragments are in registers): that slot takes stage kt+NS.
      if (kt + NS - 1 < KT) wait_vm<(NS - 2) * LPW>();
      else wait_vm<0>();
      ring_barrier();
      if (kt + NS < KT) {
        pk = kt + NS;
        ps = kt % NS;
        issue_q(pk, ps, 0);
      }
      load_frags(smem + ((kt + 1) % NS) * STAGE, 0, 0);
    }
    mfmas((KS - 1) & 1);
  }

  // Accumulator layout of a 32x32 block: lane l, element e holds
  // row 8*(e/4) + 4*(l/32) + e%4, column l%32.
  const int c = lane & 31;
  const int rbase = tm * BM + wm * TM + 4 * (lane >> 5);

  if (a.ksplit > 1) {
    // Raw fp32 tile of this split, virtual column order.
    float* out = a.partial + (size_t)split * a.M * a.N + tn * BN + wn * TN + c;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          if (row < a.M) out[(size_t)row * a.N + j * 32] = acc[i][j][e];
        }
    return;
  }

  if constexpr (EPI == EPI_RESID) {
    // Read a whole 32x32 block of the residual before writing any of it, so
    // the 16 loads per lane are in flight together.
    float* xcol = a.x + tn * BN + wn * TN + c;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        float xv[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          xv[e] = row < a.M ? xcol[(size_t)row * a.N + j * 32] : 0.f;
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          if (row < a.M) xcol[(size_t)row * a.N + j * 32] = xv[e] + acc[i][j][e];
        }
      }
  } else if constexpr (EPI == EPI_GATE_UP) {
#pragma unroll
    for (int p = 0; p < NB / 2; ++p)
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          if (row >= a.M) continue;
          epi_gate_up<BN>(a, row, tn, wn * (NB / 2) + p, c, acc[i][2 * p][e], acc[i][2 * p + 1][e]);
        }
  } else if constexpr (EPI == EPI_QKV) {
    // The same arithmetic as epi_qkv, with the segment and head taken once
    // per wave and, for each 32-row block, every row's rotary angles and
    // destination fetched before any is used, so those loads (and the
    // token -> sample -> cache slot chain of K and V rows) are in flight
    // together instead of one row after another.
    const int vs = tn * BN;
    const int seg = vs < a.n0 ? 0 : (vs < a.n0 + a.n1 ? 1 : 2);
    const int local = vs - (seg == 0 ? 0 : (seg == 1 ? a.n0 : a.n0 + a.n1));
    const int hd = a.head_dim, qpd = hd / 64, half = hd / 2;
#pragma unroll
    for (int p = 0; p < NB / 2; ++p) {
      const int P = wn * (NB / 2) + p;
      const int head = local / hd + P / qpd;
      const int fi = (P % qpd) * 32 + c;
#pragma unroll
      for (int i = 0; i < MB; ++i) {
        float2 cs[16];
        bf16* dst[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          row = row < a.M ? row : a.M - 1;        // loads only; stores are guarded below
          cs[e] = seg < 2 ? a.rope_cs[(size_t)row * half + fi] : float2{1.f, 0.f};
        }
        if (seg == 0) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
            dst[e] = a.q_out + (size_t)row * a.n0 + head * hd + fi;
          }
        } else {
          int smp[16], node[16];
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
            row = row < a.M ? row : a.M - 1;
            smp[e] = a.toks[row].sample;
            node[e] = a.toks[row].node;
          }
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const SampleInfo sv = a.samples[smp[e]];
            dst[e] = a.kv_pool + sv.kv_base +
                     ((((size_t)a.layer * 2 + (seg - 1)) * a.n_kv_heads + head) * sv.cap + sv.seq_len +
                      node[e]) * hd + fi;
          }
        }
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
          if (row >= a.M) continue;
          float x1 = acc[i][2 * p][e], x2 = acc[i][2 * p + 1][e];
          if (seg < 2) {
            const float y1 = x1 * cs[e].x - x2 * cs[e].y;
            const float y2 = x2 * cs[e].x + x1 * cs[e].y;
            x1 = y1;
            x2 = y2;
          }
          dst[e][0] = (bf16)x1;
          dst[e][half] = (bf16)x2;
        }
      }
    }
  } else {  // EPI_ARGMAX: one partial (max, lowest index) per row and wave slab of TN columns
    const int col0 = tn * BN + wn * TN + c;
    const int parts = a.N / TN;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = rbase + i * 32 + 8 * (e >> 2) + (e & 3);
        float v = acc[i][0][e];
        int idx = col0;
#pragma unroll
        for (int j = 1; j < NB; ++j)
          if (acc[i][j][e] > v) { v = acc[i][j][e]; idx = col0 + 32 * j; }
        if (a.logits != nullptr && row < a.M) {
#pragma unroll
          for (int j = 0; j < NB; ++j) a.logits[(size_t)row * a.N + col0 + 32 * j] = acc[i][j][e];
        }
#pragma unroll
        for (int m = 16; m >= 1; m >>= 1) {
          const float ov = __shfl_xor(v, m);
          const int oi = __shfl_xor(idx, m);
          if (ov > v || (ov == v && oi < idx)) { v = ov; idx = oi; }
        }
        if (c == 0 && row < a.M) {
          a.part_val[(size_t)row * parts + tn * WN + wn] = v;
          a.part_idx[(size_t)row * parts + tn * WN + wn] = idx;
        }
      }
  }
}

// ---- few rows: the product is a stream of the weight rows -----------------
//
// One work-group of 4 waves owns one unit of 16 weight rows and splits K into
// four quarters, one per wave.  A wave multiplies with
// v_mfma_f32_16x16x32_bf16: A = the activation rows (zero from row M on),
// B = its 16 weight rows; lane l loads 16 bytes of row l % 16 at k-offset
// 8 (l / 16), so a wave reads 512 contiguous bytes of each row per 256-wide
// step, and the next step's loads are in flight while the current one is
// multiplied.  The quarters' 16 x 16 tiles meet in LDS and wave 0 sums them
// in wave order (a fixed order: bitwise reproducible) and applies the
// epilogue; no K split leaves the work-group, so no reduction kernel follows
// (a residual product leaves its RMSNorm to the caller).  Units: QKV = 8
// rotary pairs (dims j, j + d/2) of one head, GATE_UP = 8 (gate, up)
// features, RESID = 16 output columns.  Every unit reads all M activation
// rows, so the activation bytes grow with M against a fixed weight stream;
// past skinny_max_rows() the tile kernel's 256-row weight tiles win, and the
// LM head always takes the tile kernel.  Accumulator layout of the 16 x 16
// block: lane l, element i holds activation row 4 (l / 16) + i and unit row
// l % 16.
constexpr int kSkinnyRows = 16;
// Rows up to which a product takes this path (measured on the 8B shape
// against the tile kernel with its K splits): q/k/v and gate/up up to 4 rows
// (at 8 rows the activation re-reads already cost more than the saved
// reductions); the residual products up to 8 (at 16 rows the RMSNorm that
// then runs on its own costs more than the fused split-K reduction it
// replaces).
template <int EPI>
constexpr int skinny_max_rows() { return EPI == EPI_RESID ? 8 : 4; }

template <int EPI>
__device__ __forceinline__ const bf16* skinny_row(const GemmArgs& a, int unit, int c) {
  if constexpr (EPI == EPI_QKV) {
    const int hd = a.head_dim, upd = hd / 16;       // units per head
    const int head_all = unit / upd, jb = unit % upd;
    const int nh0 = a.n0 / hd, nh1 = a.n1 / hd;
    const bf16* base;
    int head;
    if (head_all < nh0) { base = a.B0; head = head_all; }
    else if (head_all < nh0 + nh1) { base = a.B1; head = head_all - nh0; }
    else { base = a.B2; head = head_all - nh0 - nh1; }
    const int dim = c < 8 ? jb * 8 + c : hd / 2 + jb * 8 + (c - 8);
    return base + (size_t)(head * hd + dim) * a.K;
  } else if constexpr (EPI == EPI_GATE_UP) {
    const int f = unit * 8 + (c & 7);
    return (c < 8 ? a.B0 : a.B1) + (size_t)f * a.K;
  } else {
    return a.B0 + (size_t)(unit * kSkinnyRows + c) * a.K;
  }
}

template <int EPI>
__global__ __launch_bounds__(256) void skinny_gemm_kernel(GemmArgs a) {
  static_assert(EPI != EPI_ARGMAX, "the LM head streams its rows through the tile kernel");
  __shared__ f32x4 red[4][64];
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int c = lane & 15, kq = lane >> 4;
  const int unit = blockIdx.x;
  const int kw = a.K / 4;                            // K of this wave (a multiple of 32)
  const int k0 = wave * kw, k1 = k0 + kw;
  const bf16* wrow = skinny_row<EPI>(a, unit, c) + kq * 8;
  const bool arow_ok = c < a.M;
  const bf16* arow = a.A + (size_t)(arow_ok ? c : 0) * a.K + kq * 8;

  constexpr int KB = 8;                              // 32-wide k-blocks per step
  bf16x8 bw[2][KB], ba[2][KB];
  auto load = [&](int set, int k) {
#pragma unroll
    for (int j = 0; j < KB; ++j) {
      const int kk = k + j * 32;
      const bool in = kk < k1;
      bw[set][j] = in ? *(const bf16x8*)(wrow + kk) : bf16x8{};
      ba[set][j] = in && arow_ok ? *(const bf16x8*)(arow + kk) : bf16x8{};
    }
  };
  f32x4 acc = f32x4{};
  auto mfmas = [&](int set) {
#pragma unroll
    for (int j = 0; j < KB; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ba[set][j], bw[set][j], acc, 0, 0, 0);
  };
  load(0, k0);
  for (int k = k0; k < k1; k += 2 * KB * 32) {
    if (k + KB * 32 < k1) load(1, k + KB * 32);
    mfmas(0);
    if (k + KB * 32 >= k1) break;
    if (k + 2 * KB * 32 < k1) load(0, k + 2 * KB * 32);
    mfmas(1);
  }

  const int m0 = 4 * kq;                             // first activation row of this lane's elements
  {
    red[wave][lane] = acc;
    __syncthreads();
    if (wave != 0) return;
    f32x4 t = red[0][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) t += red[w][lane];
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int m = m0 + i;
        if (m < a.M) a.x[(size_t)m * a.N + unit * kSkinnyRows + c] += t[i];
      }
    } else if constexpr (EPI == EPI_GATE_UP) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float u = __shfl_xor(t[i], 8);         // lanes c and c + 8: gate and up of one feature
        const int m = m0 + i;
        if (c < 8 && m < a.M) a.act_out[(size_t)m * (a.N / 2) + unit * 8 + c] = (bf16)(silu(t[i]) * u);
      }
    } else {  // EPI_QKV: lanes c < 8 hold dims j, lanes c + 8 their partners j + d/2
      const int hd = a.head_dim, half = hd / 2, upd = hd / 16;
      const int head_all = unit / upd, jb = unit % upd;
      const int nh0 = a.n0 / hd, nh1 = a.n1 / hd;
      const int seg = head_all < nh0 ? 0 : (head_all < nh0 + nh1 ? 1 : 2);
      const int head = head_all - (seg == 0 ? 0 : (seg == 1 ? nh0 : nh0 + nh1));
      const int j = jb * 8 + (c & 7);               // rotary frequency index of the pair
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float other = __shfl_xor(t[i], 8);
        const int m = m0 + i;
        if (m >= a.M) continue;
        const float x1 = c < 8 ? t[i] : other, x2 = c < 8 ? other : t[i];
        float y = t[i];
        if (seg < 2) {
          const float2 cs = a.rope_cs[(size_t)m * half + j];
          y = c < 8 ? x1 * cs.x - x2 * cs.y : x2 * cs.x + x1 * cs.y;
        }
        const int dim = c < 8 ? j : j + half;
        if (seg == 0) {
          a.q_out[(size_t)m * a.n0 + head * hd + dim] = (bf16)y;
        } else {
          const TokInfo tk = a.toks[m];
          const SampleInfo sv = a.samples[tk.sample];
          a.kv_pool[sv.kv_base + ((((size_t)a.layer * 2 + (seg - 1)) * a.n_kv_heads + head) * sv.cap +
                                  sv.seq_len + tk.node) * hd + dim] = (bf16)y;
        }
      }
    }
  }
}

template <int EPI>
hipError_t launch_skinny(const GemmArgs& a, hipStream_t s) {
  long grid;
  if constexpr (EPI == EPI_QKV) grid = (long)(a.n0 + a.n1 + a.n2) / kSkinnyRows;
  else grid = (long)a.N / kSkinnyRows;
  if (a.norm_done) *a.norm_done = false;
  skinny_gemm_kernel<EPI><<<(unsigned)grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

// Sum the K splits in split order and apply the epilogue.  Thread (row,
// group g of 64 virtual columns, lane column c) owns virtual columns g*64 + c
// and g*64 + 32 + c: pair (g % (BN/64)) of tile g / (BN/64), or two residual
// columns.
template <int EPI, int BN>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int half_n = a.N / 2;
  if (idx >= (size_t)a.M * half_n) return;
  const int row = (int)(idx / half_n), rem = (int)(idx % half_n);
  const int g = rem >> 5, c = rem & 31;
  const size_t base = (size_t)row * a.N + g * 64 + c;
  float x1 = 0.f, x2 = 0.f;
  for (int s = 0; s < a.ksplit; ++s) {
    x1 += a.partial[(size_t)s * a.M * a.N + base];
    x2 += a.partial[(size_t)s * a.M * a.N + base + 32];
  }
  constexpr int PPT = BN / 64;     // pairs per tile
  if constexpr (EPI == EPI_RESID) {
    a.x[base] += x1;
    a.x[base + 32] += x2;
  } else if constexpr (EPI == EPI_QKV) {
    epi_qkv<BN>(a, row, g / PPT, g % PPT, c, x1, x2);
  } else if constexpr (EPI == EPI_GATE_UP) {
    epi_gate_up<BN>(a, row, g / PPT, g % PPT, c, x1, x2);
  }
}

// Split-K reduction of a residual product fused with the RMSNorm that
// follows it: x += (sum of the splits, in split order), then
// norm_out = bf16(x / sqrt(mean(x^2) + eps) * gain), one 256-thread block per
// row, CPT 4-float chunks of the row per thread (N <= 1024 * CPT).  Bitwise
// the same as splitk_reduce_kernel followed by the stand-alone RMSNorm (same
// summation orders), one pass over the row fewer.  Every chunk's split loads
// are issued together, four splits per round.  EAGER (few rows, so few blocks
// to hide latency with): the residual row is loaded before the splits and
// eight splits go per round, for fewer round trips at the price of registers
// (at 1024 rows the lost occupancy costs more: O 1.78 -> 1.88 ms per step).
template <int CPT, bool EAGER>
__global__ __launch_bounds__(256) void splitk_reduce_norm_kernel(GemmArgs a) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  float* xr = a.x + (size_t)row * a.N;
  const size_t plane = (size_t)a.M * a.N;
  const float* pr = a.partial + (size_t)row * a.N;
  f32x4 v[CPT], t[CPT], x0[CPT];
#pragma unroll
  for (int k = 0; k < CPT; ++k) {
    t[k] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int c = (threadIdx.x + 256 * k) * 4;
    if (EAGER && c < a.N) x0[k] = *(const f32x4*)(xr + c);   // in flight with the first splits
  }
  int s = 0;
  if constexpr (EAGER && CPT <= 4) {  // eight splits per round while the registers allow
    for (; s + 8 <= a.ksplit; s += 8) {
      f32x4 p[8][CPT];
#pragma unroll
      for (int q = 0; q < 8; ++q)
#pragma unroll
        for (int k = 0; k < CPT; ++k) {
          const int c = (threadIdx.x + 256 * k) * 4;
          p[q][k] = c < a.N ? *(const f32x4*)(pr + (s + q) * plane + c) : f32x4{0.f, 0.f, 0.f, 0.f};
        }
#pragma unroll
      for (int q = 0; q < 8; ++q)
#pragma unroll
        for (int k = 0; k < CPT; ++k) t[k] += p[q][k];
    }
  }
  for (; s + 4 <= a.ksplit; s += 4) {
    f32x4 p[4][CPT];
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int k = 0; k < CPT; ++k) {
        const int c = (threadIdx.x + 256 * k) * 4;
        p[q][k] = c < a.N ? *(const f32x4*)(pr + (s + q) * plane + c) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
    for (int q = 0; q < 4; ++q)
#pragma unroll
      for (int k = 0; k < CPT; ++k) t[k] += p[q][k];
  }
  for (; s < a.ksplit; ++s)
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int c = (threadIdx.x + 256 * k) * 4;
      if (c < a.N) t[k] += *(const f32x4*)(pr + s * plane + c);
    }
  float ss = 0.f;
#pragma unroll
  for (int k = 0; k < CPT; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < a.N) {
      v[k] = (EAGER ? x0[k] : *(const f32x4*)(xr + c)) + t[k];
      *(f32x4*)(xr + c) = v[k];
      ss += v[k][0] * v[k][0] + v[k][1] * v[k][1] + v[k][2] * v[k][2] + v[k][3] * v[k][3];
    }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float rstd = rsqrtf(tot / (float)a.N + a.norm_eps);
  bf16* orow = a.norm_out + (size_t)row * a.N;
#pragma unroll
  for (int k = 0; k < CPT; ++k) {
    const int c = (threadIdx.x + 256 * k) * 4;
    if (c < a.N) {
      const bf16x4 g = *(const bf16x4*)(a.norm_gain + c);
      bf16x4 y;
#pragma unroll
      for (int j = 0; j < 4; ++j) y[j] = (bf16)(v[k][j] * rstd * (float)g[j]);
      *(bf16x4*)(orow + c) = y;
    }
  }
}

// Launch the fused reduction + norm; false when the row is too long for it.
bool launch_reduce_norm(const GemmArgs& a, hipStream_t s) {
  const int cpt = (a.N + 1023) / 1024;
  const bool eager = a.M <= 512;       // at most two blocks per CU
  auto go = [&](auto kern) { kern<<<(unsigned)a.M, 256, 0, s>>>(a); return true; };
  switch (cpt) {
    case 1: return eager ? go(splitk_reduce_norm_kernel<1, true>) : go(splitk_reduce_norm_kernel<1, false>);
    case 2: return eager ? go(splitk_reduce_norm_kernel<2, true>) : go(splitk_reduce_norm_kernel<2, false>);
    case 3:
    case 4: return eager ? go(splitk_reduce_norm_kernel<4, true>) : go(splitk_reduce_norm_kernel<4, false>);
    case 5: case 6: case 7:
    case 8: return eager ? go(splitk_reduce_norm_kernel<8, true>) : go(splitk_reduce_norm_kernel<8, false>);
    default: return false;
  }
}

enum TileShape { TILE_256x256, TILE_256x128, TILE_128x128, TILE_64x256, TILE_32x256 };

// Shape choice (measured over the verify step's products at 32 to 1024 rows):
//   * few rows: 32- or 64-row tiles that stream 256 weight rows each;
//   * up to 128 rows: 128 x 128 tiles with a 4-stage ring (one work-group per
//     CU, deep lookahead for the weight stream);
//   * many rows and at least 384 256 x 256 tiles (gate/up, LM head): 256 x 256
//     tiles, which need the fewest operand bytes per flop, 8 waves, with
//     32-wide K steps in a 4-stage ring (128 KB; 3-5 % faster than 64-wide
//     steps in two stages);
//   * otherwise (the q/k/v projection from 512 rows on included) 256 x 128
//     tiles, 8 waves, 64-wide K steps in a 3-stage ring (144 KB), or, for
//     products too narrow to give 64 of them, 128 x 128 tiles with split K.
// 256-wide tiles need every weight segment (q/k/v) to be a multiple of 256 so
// no tile straddles two; 128-wide ones need multiples of 128.
TileShape pick_tile(int epi, int M, int N, int K, int n0, int n1) {
  const bool w256 = N % 256 == 0 && n0 % 256 == 0 && n1 % 256 == 0;
  if (w256 && M <= 32) return TILE_32x256;
  if (w256 && M <= 64) return TILE_64x256;
  if (M <= 128) return TILE_128x128;
  if (w256 && M > 128 && (long)((M + 255) / 256) * (N / 256) >= 384) return TILE_256x256;
  if ((long)((M + 255) / 256) * (N / 128) < 64 && K <= 4096) return TILE_128x128;
  return TILE_256x128;
}

// K splits: about one work-group per CU for the wide tiles (their ring holds
// a CU's LDS) and two for the skinny ones, at least 8 K steps per split, the
// splits dividing the K steps, partials within the workspace area.
int choose_splits(int epi, int BM, int BK, long tiles, int M, int N, int K) {
  if (epi == EPI_ARGMAX) return 1;
  const long target = BM <= 64 ? 512 : 256;
  int s = (int)std::max<long>(1, std::min<long>(16, target / tiles));
  const int kt = K / BK;
  while (s > 1 && (kt % s != 0 || kt / s < 8 || (size_t)s * M * N * 4 > kPartialCap)) --s;
  return s;
}

template <int EPI, int BM, int BN, int WM, int NS, int BK = 64, int NW = 4>
hipError_t launch_tile(GemmArgs a, hipStream_t s) {
  constexpr int SMEM = NS * (BM + BN) * BK * 2;
  static bool configured = false;
  if (!configured) {
    const hipError_t e = hipFuncSetAttribute((const void*)gemm_bf16_kernel<EPI, BM, BN, WM, NS, BK, NW>,
                                             hipFuncAttributeMaxDynamicSharedMemorySize, SMEM);
    if (e != hipSuccess) return e;
    configured = true;
  }
  const long tiles = (long)((a.M + BM - 1) / BM) * (a.N / BN);
  a.ksplit = a.partial ? choose_splits(EPI, BM, BK, tiles, a.M, a.N, a.K) : 1;
  gemm_bf16_kernel<EPI, BM, BN, WM, NS, BK, NW><<<(unsigned)(tiles * a.ksplit), NW * 64, SMEM, s>>>(a);
  if (a.ksplit > 1) {
    if (EPI == EPI_RESID && a.norm_out != nullptr && a.N % 4 == 0 && launch_reduce_norm(a, s)) {
      if (a.norm_done) *a.norm_done = true;
    } else {
      const size_t threads = (size_t)a.M * (a.N / 2);
      splitk_reduce_kernel<EPI, BN><<<(unsigned)((threads + 255) / 256), 256, 0, s>>>(a);
    }
  }
  return hipGetLastError();
}

template <int EPI>
hipError_t launch_epi(const GemmArgs& a, hipStream_t s) {
  // Few rows: every supported shape has K a multiple of 128 and head_dim 64
  // or 128, which the weight-row units assume.
  if constexpr (EPI != EPI_ARGMAX)
    if (a.M <= skinny_max_rows<EPI>() && a.K % 128 == 0) return launch_skinny<EPI>(a, s);
  switch (pick_tile(EPI, a.M, a.N, a.K, a.n0, a.n1)) {
    case TILE_256x256: return launch_tile<EPI, 256, 256, 2, 4, 32, 8>(a, s);
    case TILE_256x128: return launch_tile<EPI, 256, 128, 4, 3, 64, 8>(a, s);
    case TILE_32x256: return launch_tile<EPI, 32, 256, 1, 3>(a, s);
    case TILE_64x256: return launch_tile<EPI, 64, 256, 2, 3>(a, s);
    default: return launch_tile<EPI, 128, 128, 2, 4>(a, s);
  }
}

}  // namespace

int gemm_parts(int N, int M, int K) {
  switch (pick_tile(EPI_ARGMAX, M, N, K, N, 0)) {
    case TILE_64x256: return N / 128;
    default: return N / 64;       // 256x128, 128x128 and 32x256: wave slabs of 64 columns
  }
}

size_t gemm_partial_bytes() { return kPartialCap; }

hipError_t launch_gemm(int epi, const GemmArgs& a, hipStream_t s) {
  switch (epi) {
    case EPI_QKV: return launch_epi<EPI_QKV>(a, s);
    case EPI_RESID: return launch_epi<EPI_RESID>(a, s);
    case EPI_GATE_UP: return launch_epi<EPI_GATE_UP>(a, s);
    case EPI_ARGMAX: return launch_epi<EPI_ARGMAX>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace spec
