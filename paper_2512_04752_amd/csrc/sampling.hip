// Tree acceptance at a sampling temperature (speculative sampling over the
// draft tree), and greedy acceptance with an end-of-sequence token.
//
// Speculative decoding is lossless (RLHFSpec Section 2.2: the verified
// output follows the target model's distribution).  At temperature T > 0
// every node u has the target distribution p_u = softmax(z_u / T) of the
// token after it, and the draft drew u's children independently from its
// own distribution q_u.  The walk from the root (multi-draft speculative
// sampling) keeps an unnormalised residual P with total R, starting at
// P_0 = exp(z_u / T - max(z_u) / T) (so p_u = P_0 / R_0), and tries u's
// children in node order: child c with token x is accepted when
// a_c * q_u(x) * R < P(x) (probability min(1, p'(x) / q_u(x)) for the
// normalised residual p' = P / R); a rejected child turns P into
// max(P - R q_u, 0) (R times the textbook residual max(p' - q_u, 0)).  The
// walk moves to an accepted child; when no child is accepted (or u has none)
// the next token is drawn from P by inverse CDF with u's second uniform.
// a_c and the sampling draws are inputs.
//
// What happens at a node depends on that node's row alone (its logits, its
// draft row, its children's tokens and uniforms), not on the path to it.
// So the work splits in two launches:
//   * node_decide_kernel: one work-group per node with children decides, in
//     parallel over the whole batch, which child the walk would take from it
//     (or that none is accepted), keeping the residual totals R_0 .. R_k;
//   * sample_walk_kernel: one work-group per sample follows those decisions
//     from the root and draws the next token at the node where the walk
//     stops.
// The residual is never stored for the first kMaxRecompute rejections at a
// node: P_k(y) is recomputed from z(y) and q(y) with the k totals (reading
// 8 bytes per vocabulary entry instead of reading and writing 16).  A node
// with more rejected children continues in the walk kernel on a stored fp64
// row of the sample.
//
// Vocabulary-wide arithmetic is fp64 (exp, residuals, sums, the CDF), so the
// decisions are those of a float64 statement of the same procedure, up to
// about one ulp per exp; the logits are the forward pass's fp32 values.  Every reduction runs in a
// fixed order, so results are reproducible run to run.
//
// End of sequence: an accepted node carrying the EOS token ends the branch
// (its children are not tried, no next token: -1).
#include <math.h>

#include "common.h"

namespace spec {

namespace {

constexpr int kMaxRecompute = 8;   // rejections per node recomputed from z and q

enum : int32_t { NODE_LEAF = 0, NODE_CHILD = 1, NODE_DRAW = 2, NODE_MORE = 3, NODE_END = 4 };

// A node's decision (written by node_decide_kernel for every node).
struct NodeRec {
  int32_t kind;     // NODE_*
  int32_t arg;      // CHILD: accepted child (node index); MORE: position of the next child to try
  int32_t k;        // rejections done: R[0 .. k] valid
  int32_t pad;
  double base;      // max(z_u)
  double R[kMaxRecompute + 1];
};
static_assert(sizeof(NodeRec) == 96, "NodeRec layout");

// ---- exp for arguments <= 0 (fp64) ---------------------------------------
//
// Tang's table-driven method (P. T. P. Tang, ACM TOMS 15(2), 1989): write
// x = (64 m + j) ln2/64 + r with |r| <= ln2/128, so exp(x) = 2^m 2^(j/64) e^r;
// 2^(j/64) comes from a table of correctly rounded doubles and e^r - 1 from
// its degree-5 Taylor polynomial (truncation below 4e-17 relative).  The
// reduction uses ln2/64 split into a 21-bit high part (n * hi exact) and a
// low part.  Within about one ulp of exp over [-745, 0]; arguments are
// clamped at -800, where ldexp underflows to 0 (a NaN argument gives 0).

__constant__ double kExp2Frac[64] = {
    0x1.0000000000000p+0, 0x1.02c9a3e778061p+0, 0x1.059b0d3158574p+0,
    0x1.0874518759bc8p+0, 0x1.0b5586cf9890fp+0, 0x1.0e3ec32d3d1a2p+0,
    0x1.11301d0125b51p+0, 0x1.1429aaea92de0p+0, 0x1.172b83c7d517bp+0,
    0x1.1a35beb6fcb75p+0, 0x1.1d4873168b9aap+0, 0x1.2063b88628cd6p+0,
    0x1.2387a6e756238p+0, 0x1.26b4565e27cddp+0, 0x1.29e9df51fdee1p+0,
    0x1.2d285a6e4030bp+0, 0x1.306fe0a31b715p+0, 0x1.33c08b26416ffp+0,
    0x1.371a7373aa9cbp+0, 0x1.3a7db34e59ff7p+0, 0x1.3dea64c123422p+0,
    0x1.4160a21f72e2ap+0, 0x1.44e086061892dp+0, 0x1.486a2b5c13cd0p+0,
    0x1.4bfdad5362a27p+0, 0x1.4f9b2769d2ca7p+0, 0x1.5342b569d4f82p+0,
    0x1.56f4736b527dap+0, 0x1.5ab07dd485429p+0, 0x1.5e76f15ad2148p+0,
    0x1.6247eb03a5585p+0, 0x1.6623882552225p+0, 0x1.6a09e667f3bcdp+0,
    0x1.6dfb23c651a2fp+0, 0x1.71f75e8ec5f74p+0, 0x1.75feb564267c9p+0,
    0x1.7a11473eb0187p+0, 0x1.7e2f336cf4e62p+0, 0x1.82589994cce13p+0,
    0x1.868d99b4492edp+0, 0x1.8ace5422aa0dbp+0, 0x1.8f1ae99157736p+0,
    0x1.93737b0cdc5e5p+0, 0x1.97d829fde4e50p+0, 0x1.9c49182a3f090p+0,
    0x1.a0c667b5de565p+0, 0x1.a5503b23e255dp+0, 0x1.a9e6b5579fdbfp+0,
    0x1.ae89f995ad3adp+0, 0x1.b33a2b84f15fbp+0, 0x1.b7f76f2fb5e47p+0,
    0x1.bcc1e904bc1d2p+0, 0x1.c199bdd85529cp+0, 0x1.c67f12e57d14bp+0,
    0x1.cb720dcef9069p+0, 0x1.d072d4a07897cp+0, 0x1.d5818dcfba487p+0,
    0x1.da9e603db3285p+0, 0x1.dfc97337b9b5fp+0, 0x1.e502ee78b3ff6p+0,
    0x1.ea4afa2a490dap+0, 0x1.efa1bee615a27p+0, 0x1.f50765b6e4540p+0,
    0x1.fa7c1819e90d8p+0,
};

constexpr double kInvLn2x64 = 0x1.71547652b82fep+6;    // 64 / ln 2
constexpr double kLn2x64Hi = 0x1.62e42p-7;             // ln2/64, high 21 bits
constexpr double kLn2x64Lo = 0x1.fdf473de6af28p-28;    // ln2/64 - kLn2x64Hi
constexpr double kRoundShift = 0x1.8p52;               // adding it rounds to an integer

__shared__ double s_exp2_frac[64];   // kExp2Frac, staged per work-group

__device__ __forceinline__ void exp_table_init() {
  if (threadIdx.x < 64) s_exp2_frac[threadIdx.x] = kExp2Frac[threadIdx.x];
  __syncthreads();
}

__device__ __forceinline__ double exp_le0(double x) {
  x = fmax(x, -800.0);                                 // below -745.2 the result underflows to 0
  const double t = fma(x, kInvLn2x64, kRoundShift);
  const int n = __double2loint(t);                     // round(x * 64 / ln2)
  const double nd = t - kRoundShift;
  const double r = fma(-nd, kLn2x64Lo, fma(-nd, kLn2x64Hi, x));
  const double p = fma(r * r, fma(r, fma(r, fma(r, 1.0 / 120, 1.0 / 24), 1.0 / 6), 0.5), r);
  const double s = s_exp2_frac[n & 63];
  return ldexp(fma(s, p, s), n >> 6);
}

// ---- the residual, element-wise -------------------------------------------

// P_0(y) = exp((z(y) - max z) / T); the fp32 difference is exact in fp64.
__device__ __forceinline__ double target0(float z, double inv_t, double zmax) {
  return exp_le0(((double)z - zmax) * inv_t);
}
__device__ __forceinline__ double resid_step(double v, double R, float q) {
  return fmax(v - R * (double)q, 0.0);
}
// P_k(y) from z(y), q(y) and the totals R[0 .. k-1].
__device__ __forceinline__ double resid_k(float z, float q, int k, const double* R, double inv_t,
                                          double base) {
  double v = target0(z, inv_t, base);
  for (int i = 0; i < k; ++i) v = resid_step(v, R[i], q);
  return v;
}

// Where the residual comes from, fixed at compile time so that every load
// lands in registers:
//   RM_TARGET  P_0 = exp((z - base) / T), base = max z, recomputed (reads z);
//   RM_CHAIN   P_k recomputed from z, q and R[0 .. k-1] (reads z and q);
//   RM_STORED  a stored fp64 row (reads P, and q where a pass needs it).
// Four consecutive vocabulary entries are one group; fetch() issues a
// group's loads, eval() turns them into P values, so that a thread can put
// several groups' loads in flight before computing.
enum { RM_TARGET = 0, RM_CHAIN = 1, RM_STORED = 2 };

struct Raw {
  float4 a, b, c;   // TARGET/CHAIN: a = z, b = q; STORED: a, b = the four P bits, c = q
};

template <int MODE, bool NEED_Q>
struct Resid {
  const float* z;
  const float* q;
  const double* R;   // LDS, R[0 .. k]
  int k;
  double inv_t, base;
  const double* P;
  __device__ __forceinline__ void fetch(int g, Raw& w) const {
    if constexpr (MODE == RM_STORED) {
      w.a = reinterpret_cast<const float4*>(P)[2 * g];
      w.b = reinterpret_cast<const float4*>(P)[2 * g + 1];
      if constexpr (NEED_Q) w.c = reinterpret_cast<const float4*>(q)[g];
    } else {
      w.a = reinterpret_cast<const float4*>(z)[g];
      if constexpr (NEED_Q || MODE == RM_CHAIN) w.b = reinterpret_cast<const float4*>(q)[g];
    }
  }
  __device__ __forceinline__ float4 qof(const Raw& w) const {
    if constexpr (MODE == RM_STORED) return w.c;
    else return w.b;
  }
  __device__ __forceinline__ void eval(const Raw& w, double v[4]) const {
    if constexpr (MODE == RM_STORED) {
      const double2 lo = __builtin_bit_cast(double2, w.a);
      const double2 hi = __builtin_bit_cast(double2, w.b);
      v[0] = lo.x; v[1] = lo.y; v[2] = hi.x; v[3] = hi.y;
    } else {
      // the same operations, in the same order, as resid_k for each entry
      v[0] = target0(w.a.x, inv_t, base);
      v[1] = target0(w.a.y, inv_t, base);
      v[2] = target0(w.a.z, inv_t, base);
      v[3] = target0(w.a.w, inv_t, base);
      if constexpr (MODE == RM_CHAIN) {
        for (int i = 0; i < k; ++i) {
          const double Ri = R[i];
          v[0] = resid_step(v[0], Ri, w.b.x);
          v[1] = resid_step(v[1], Ri, w.b.y);
          v[2] = resid_step(v[2], Ri, w.b.z);
          v[3] = resid_step(v[3], Ri, w.b.w);
        }
      }
    }
  }
};

constexpr int kUnroll = 4;   // groups per thread in flight

// ---- work-group reductions (fixed order; every thread gets the same value) -

__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return __shfl(v, 0);
}

template <int NT>
__device__ __forceinline__ double block_sum(double v, double* red) {
  v = wave_sum(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double r = 0.0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) r += red[w];
  __syncthreads();
  return r;
}

// Merge two (max, sum of exp((z - max) / T)) pairs.
__device__ __forceinline__ void lse_merge(float& m, double& s, float m2, double s2, double inv_t) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) { m = m2; s = s2; return; }
  if (m2 > m) {
    s = s * exp_le0(((double)m - (double)m2) * inv_t) + s2;
    m = m2;
  } else {
    s += s2 * exp_le0(((double)m2 - (double)m) * inv_t);
  }
}

// One pass over z: base = max(z) and R_0 = sum exp((z - base) / T).  Each
// thread keeps a running (max, sum) over batches of 4 * kUnroll entries:
// the batch's max first (one rescale of the sum when it grows), then
// independent exps, so the exps of a batch do not wait on each other.
template <int NT>
__device__ __forceinline__ void target_pass(const float* z, int vocab, double inv_t, double* red,
                                            float* redm, double* base, double* R0) {
  float m = -INFINITY;
  double s = 0.0;
  const int G4 = vocab / 4;
  for (int gb = threadIdx.x; gb < G4; gb += NT * kUnroll) {
    float4 zz[kUnroll];
    float mb = -INFINITY;
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      zz[i] = gb + i * NT < G4 ? reinterpret_cast<const float4*>(z)[gb + i * NT]
                               : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
    }
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
      mb = fmaxf(mb, fmaxf(fmaxf(zz[i].x, zz[i].y), fmaxf(zz[i].z, zz[i].w)));
    if (mb > m) {
      if (m != -INFINITY) s *= exp_le0(((double)m - (double)mb) * inv_t);
      m = mb;
    }
    if (m == -INFINITY) continue;
    double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      acc[0] += exp_le0(((double)zz[i].x - (double)m) * inv_t);
      acc[1] += exp_le0(((double)zz[i].y - (double)m) * inv_t);
      acc[2] += exp_le0(((double)zz[i].z - (double)m) * inv_t);
      acc[3] += exp_le0(((double)zz[i].w - (double)m) * inv_t);
    }
    s += (acc[0] + acc[1]) + (acc[2] + acc[3]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(m, o);
    const double s2 = __shfl_xor(s, o);
    lse_merge(m, s, m2, s2, inv_t);
  }
  m = __shfl(m, 0);
  s = __shfl(s, 0);
  if ((threadIdx.x & 63) == 0) {
    redm[threadIdx.x >> 6] = m;
    red[threadIdx.x >> 6] = s;
  }
  __syncthreads();
  float M = -INFINITY;
  double S = 0.0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) lse_merge(M, S, redm[w], red[w], inv_t);
  __syncthreads();
  *base = (double)M;
  *R0 = S;
}

// The residual after one more rejection: returns sum max(P_k - R_k q, 0);
// with `out` set, also stores that residual there.
template <int NT, class RS>
__device__ __forceinline__ double reject_pass(const RS& r, int vocab, double Rk, double* out,
                                              double* red) {
  double part[4] = {0.0, 0.0, 0.0, 0.0};
  const int G4 = vocab / 4;
  for (int gb = threadIdx.x; gb < G4; gb += NT * kUnroll) {
    Raw w[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
      if (gb + i * NT < G4) r.fetch(gb + i * NT, w[i]);
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      const int g = gb + i * NT;
      if (g >= G4) break;
      double v[4];
      r.eval(w[i], v);
      const float4 qq = r.qof(w[i]);
      const float qs[4] = {qq.x, qq.y, qq.z, qq.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[e] = resid_step(v[e], Rk, qs[e]);
        part[e] += v[e];
      }
      if (out) {
        reinterpret_cast<double2*>(out)[2 * g] = make_double2(v[0], v[1]);
        reinterpret_cast<double2*>(out)[2 * g + 1] = make_double2(v[2], v[3]);
      }
    }
  }
  return block_sum<NT>((part[0] + part[1]) + (part[2] + part[3]), red);
}

// Stores P_k (recomputed) into `out`.
template <int NT, class RS>
__device__ __forceinline__ void store_pass(const RS& r, int vocab, double* out) {
  const int G4 = vocab / 4;
  for (int gb = threadIdx.x; gb < G4; gb += NT * kUnroll) {
    Raw w[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
      if (gb + i * NT < G4) r.fetch(gb + i * NT, w[i]);
#pragma unroll
    for (int i = 0; i < kUnroll; ++i) {
      const int g = gb + i * NT;
      if (g >= G4) break;
      double v[4];
      r.eval(w[i], v);
      reinterpret_cast<double2*>(out)[2 * g] = make_double2(v[0], v[1]);
      reinterpret_cast<double2*>(out)[2 * g + 1] = make_double2(v[2], v[3]);
    }
  }
  __syncthreads();
}

__device__ __forceinline__ double wave_incl_scan(double x, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const double t = __shfl_up(x, o);
    if (lane >= o) x += t;
  }
  return x;
}

// Inverse CDF of the residual: the smallest y whose running sum exceeds
// frac * (the residual's total); the last entry of positive mass when
// rounding leaves the target at or past the total; -1 only for non-finite
// logits.  Wave w owns a contiguous segment of the vocabulary, walked 256
// entries (64 lanes x 4) per step, steps grouped in blocks of kBlockSteps.
// Pass 1 sums each block (per-lane sums over its steps, then one wave
// reduction) into LDS; the total, the target, the owner wave and the owner
// block follow in order from those sums; pass 2 rescans the owner block's
// steps with an inclusive wave scan per step.  Returns the total as well.
constexpr int kBlockSteps = 8;
constexpr int kBlockCap = 32;        // blocks per wave held in LDS

template <int NT, class RS>
__device__ __forceinline__ int cdf_draw(const RS& r, int vocab, double frac, double* red,
                                       int* ired, double* blk_tot, double* total) {
  constexpr int W = NT / 64;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int G4 = vocab / 4;
  const int seg = (G4 + W - 1) / W;
  const int steps = (seg + 63) / 64;
  // steps per block: kBlockSteps, more when the segment is too long for the cap
  const int spb = max(kBlockSteps, (steps + kBlockCap - 1) / kBlockCap);
  const int nblk = (steps + spb - 1) / spb;
  const int g0 = min(G4, w * seg), g1 = min(G4, g0 + seg);
  double tot = 0.0;
  for (int b0 = 0; b0 < nblk; ++b0) {
    double ls = 0.0;                     // this lane's sum over the block's steps
    const int s_end = min(steps, (b0 + 1) * spb);
    for (int st0 = b0 * spb; st0 < s_end; st0 += kUnroll) {
      Raw raw[kUnroll];
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int g = g0 + 64 * (st0 + i) + lane;
        if (st0 + i < s_end && g < g1) r.fetch(g, raw[i]);
      }
#pragma unroll
      for (int i = 0; i < kUnroll; ++i) {
        const int g = g0 + 64 * (st0 + i) + lane;
        if (st0 + i < s_end && g < g1) {
          double v[4];
          r.eval(raw[i], v);
          ls += ((v[0] + v[1]) + v[2]) + v[3];
        }
      }
    }
    const double bt = wave_sum(ls);
    if (lane == 0) blk_tot[w * kBlockCap + b0] = bt;
    tot += bt;
  }
  if (lane == 0) red[w] = tot;
  __syncthreads();
  if (threadIdx.x == 0) {
    double all = 0.0;
    for (int i = 0; i < W; ++i) all += red[i];
    const double target = frac * all;
    double run = 0.0, off = 0.0, off_last = 0.0;
    int owner = -1, last = -1;
    for (int i = 0; i < W; ++i) {
      if (red[i] > 0.0) { last = i; off_last = run; }
      if (owner < 0 && run + red[i] > target) { owner = i; off = run; }
      run += red[i];
    }
    if (owner < 0) { owner = last; off = off_last; }
    int blk = -1;
    if (owner >= 0) {
      double acc = off, acc_last = off;
      int lastb = -1;
      for (int i = 0; i < nblk; ++i) {
        const double t = blk_tot[owner * kBlockCap + i];
        if (t > 0.0) { lastb = i; acc_last = acc; }
        if (blk < 0 && acc + t > target) { blk = i; off = acc; }
        acc += t;
      }
      if (blk < 0) { blk = lastb; off = acc_last; }
    }
    ired[0] = blk >= 0 ? owner : -1;
    ired[1] = -1;
    ired[2] = blk;
    red[W] = off;
    red[W + 1] = target;
    red[W + 2] = all;
  }
  __syncthreads();
  const double target = red[W + 1];
  *total = red[W + 2];
  if (w == ired[0]) {
    const int blk = ired[2];
    double acc = red[W];
    int pick = -1, lastpos = -1;
    for (int st = blk * spb; st < min(steps, (blk + 1) * spb) && pick < 0; ++st) {
      const int g = g0 + 64 * st + lane;
      double v[4] = {0.0, 0.0, 0.0, 0.0};
      if (g < g1) {
        Raw raw;
        r.fetch(g, raw);
        r.eval(raw, v);
      }
      const double sl = ((v[0] + v[1]) + v[2]) + v[3];
      const double incl = wave_incl_scan(sl, lane);
      int mylast = -1;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (v[e] > 0.0) mylast = 4 * g + e;
      const unsigned long long pos = __ballot(mylast >= 0);
      if (pos) lastpos = __shfl(mylast, 63 - __clzll(pos));
      double excl = __shfl_up(incl, 1);
      if (lane == 0) excl = 0.0;
      const unsigned long long hit = __ballot(g < g1 && acc + incl > target);
      if (hit) {
        // the first lane whose inclusive sum passes the target walks its four
        const int L = __ffsll(hit) - 1;
        int mine = -1;
        if (lane == L) {
          double run = acc + excl;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            run += v[e];
            if (mine < 0 && run > target) mine = 4 * g + e;
          }
          if (mine < 0) mine = mylast;
        }
        pick = __shfl(mine, L);
        if (pick < 0) pick = lastpos;
      }
      acc += __shfl(incl, 63);
    }
    if (pick < 0) pick = lastpos;
    if (lane == 0) ired[1] = pick;
  }
  __syncthreads();
  return ired[1];
}

// max over z (fp32, no exp).
template <int NT>
__device__ __forceinline__ float max_pass(const float* z, int vocab, float* redm) {
  float m = -INFINITY;
  const int G4 = vocab / 4;
  for (int gb = threadIdx.x; gb < G4; gb += NT * kUnroll) {
    float4 zz[kUnroll];
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
      zz[i] = gb + i * NT < G4 ? reinterpret_cast<const float4*>(z)[gb + i * NT]
                               : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
#pragma unroll
    for (int i = 0; i < kUnroll; ++i)
      m = fmaxf(m, fmaxf(fmaxf(zz[i].x, zz[i].y), fmaxf(zz[i].z, zz[i].w)));
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
  if ((threadIdx.x & 63) == 0) redm[threadIdx.x >> 6] = m;
  __syncthreads();
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) M = fmaxf(M, redm[w]);
  __syncthreads();
  return M;
}

// ---- launch 1: every node's decision ----------------------------------------

template <int NT>
__global__ __launch_bounds__(NT) void node_decide_kernel(
    const SampleInfo* samples, const TokInfo* toks, const int32_t* tokens, const int32_t* parents,
    const float* logits, const float* draft_probs, const float* uniforms, int vocab, double inv_t,
    int eos, NodeRec* recs) {
  __shared__ double red[NT / 64];
  __shared__ float redm[NT / 64];
  __shared__ double R[kMaxRecompute + 1];
  __shared__ int kids[kMaxTree];
  __shared__ int nkids;
  exp_table_init();
  const int row = blockIdx.x;
  const TokInfo ti = toks[row];
  const SampleInfo s = samples[ti.sample];
  const int u = ti.node;
  NodeRec* rec = recs + row;
  if (tokens[row] == eos) {
    if (threadIdx.x == 0) rec->kind = NODE_END;
    return;
  }
  if (threadIdx.x == 0) {
    int n = 0;
    for (int c = u + 1; c < s.ntok; ++c)
      if (parents[s.tok0 + c] == u) kids[n++] = c;
    nkids = n;
  }
  __syncthreads();
  const int nk = nkids;
  if (nk == 0) {
    if (threadIdx.x == 0) rec->kind = NODE_LEAF;
    return;
  }
  const float* z = logits + (size_t)row * vocab;
  const float* q = draft_probs + (size_t)row * vocab;
  double base, R0;
  target_pass<NT>(z, vocab, inv_t, red, redm, &base, &R0);
  if (threadIdx.x == 0) R[0] = R0;
  __syncthreads();
  int k = 0, kind = NODE_DRAW, arg = 0;
  for (int j = 0; j < nk; ++j) {
    if (k == kMaxRecompute) { kind = NODE_MORE; arg = j; break; }   // kids[j..] untested
    const int c = kids[j];
    const int x = tokens[s.tok0 + c];
    const double a = (double)uniforms[2 * (size_t)(s.tok0 + c)];
    const double px = resid_k(z[x], q[x], k, R, inv_t, base);
    if (a * (double)q[x] * R[k] < px) { kind = NODE_CHILD; arg = c; break; }
    double Rn;
    if (k == 0)
      Rn = reject_pass<NT>(Resid<RM_TARGET, true>{z, q, R, 0, inv_t, base, nullptr}, vocab, R[0],
                           nullptr, red);
    else
      Rn = reject_pass<NT>(Resid<RM_CHAIN, true>{z, q, R, k, inv_t, base, nullptr}, vocab, R[k],
                           nullptr, red);
    if (threadIdx.x == 0) R[k + 1] = Rn;
    __syncthreads();
    ++k;
  }
  if (threadIdx.x == 0) {
    rec->kind = kind;
    rec->arg = arg;
    rec->k = k;
    rec->base = base;
    for (int i = 0; i <= k; ++i) rec->R[i] = R[i];
  }
}

// ---- launch 2: the walk and the final draw ---------------------------------

template <int NT>
__global__ __launch_bounds__(NT) void sample_walk_kernel(
    const SampleInfo* samples, const int32_t* tokens, const int32_t* parents, const float* logits,
    const float* draft_probs, const float* uniforms, int vocab, double inv_t, int eos,
    const NodeRec* recs, double* resid, int32_t* accepted_len, int32_t* next_token,
    int32_t* accepted_nodes) {
  __shared__ double red[NT / 64 + 3];
  __shared__ float redm[NT / 64];
  __shared__ int ired[3];
  __shared__ double blk_tot[(NT / 64) * kBlockCap];
  __shared__ double R[kMaxTree + 1];
  __shared__ int path[kMaxTree];
  exp_table_init();
  const int b = blockIdx.x;
  const SampleInfo s = samples[b];
  double* Pst = resid + (size_t)b * vocab;

  int u = 0, depth = 0, next = -1;
  if (threadIdx.x == 0) path[0] = 0;
  bool ended = tokens[s.tok0] == eos;
  while (!ended) {
    const NodeRec& rec = recs[s.tok0 + u];
    const int kind = rec.kind;
    if (kind == NODE_END) {        // not reached: EOS nodes end the walk when entered
      ended = true;
      break;
    }
    if (kind == NODE_CHILD) {
      u = rec.arg;
      ++depth;
      if (threadIdx.x == 0) path[depth] = u;
      ended = tokens[s.tok0 + u] == eos;
      continue;
    }
    const float* z = logits + (size_t)(s.tok0 + u) * vocab;
    const float* q = draft_probs + (size_t)(s.tok0 + u) * vocab;
    double base;
    int k;
    if (kind == NODE_LEAF) {
      // no children: the draw from p_u needs only the max first (the draw's
      // own pass sums P_0)
      base = (double)max_pass<NT>(z, vocab, redm);
      if (threadIdx.x == 0) R[0] = 1.0;
      k = 0;
    } else {
      base = rec.base;
      k = min(max(rec.k, 0), kMaxRecompute);
      if (threadIdx.x <= k) R[threadIdx.x] = rec.R[threadIdx.x];
    }
    __syncthreads();
    bool stored = false;
    int moved = -1;
    if (kind == NODE_MORE) {
      // More rejected children than recomputation covers: store P_k once,
      // then try the untested children (positions rec.arg on) on the stored
      // row.
      store_pass<NT>(Resid<RM_CHAIN, false>{z, q, R, k, inv_t, base, nullptr}, vocab, Pst);
      stored = true;
      int pos = 0;
      for (int c = u + 1; c < s.ntok; ++c) {
        if (parents[s.tok0 + c] != u) continue;
        if (pos++ < rec.arg) continue;
        const int x = tokens[s.tok0 + c];
        const double a = (double)uniforms[2 * (size_t)(s.tok0 + c)];
        if (a * (double)q[x] * R[k] < Pst[x]) { moved = c; break; }
        const double Rn = reject_pass<NT>(Resid<RM_STORED, true>{z, q, R, 0, inv_t, base, Pst},
                                          vocab, R[k], Pst, red);
        if (threadIdx.x == 0) R[k + 1] = Rn;
        __syncthreads();
        ++k;
      }
    }
    if (moved >= 0) {
      u = moved;
      ++depth;
      if (threadIdx.x == 0) path[depth] = u;
      ended = tokens[s.tok0 + u] == eos;
      continue;
    }
    // Draw the next token from the residual.  A residual with no mass left
    // (only through rounding) falls back to p_u.
    if (!(R[k] > 0.0)) { k = 0; stored = false; }
    const double a2 = (double)uniforms[2 * (size_t)(s.tok0 + u) + 1];
    double total;
    if (stored)
      next = cdf_draw<NT>(Resid<RM_STORED, false>{z, q, R, 0, inv_t, base, Pst}, vocab, a2, red,
                          ired, blk_tot, &total);
    else if (k == 0)
      next = cdf_draw<NT>(Resid<RM_TARGET, false>{z, q, R, 0, inv_t, base, nullptr}, vocab, a2,
                          red, ired, blk_tot, &total);
    else
      next = cdf_draw<NT>(Resid<RM_CHAIN, false>{z, q, R, k, inv_t, base, nullptr}, vocab, a2,
                          red, ired, blk_tot, &total);
    break;
  }
  if (threadIdx.x == 0) {
    accepted_len[b] = depth;
    next_token[b] = ended ? -1 : next;
    int32_t* out = accepted_nodes + (size_t)b * kMaxTree;
    for (int d = 0; d < kMaxTree; ++d) out[d] = d <= depth ? path[d] : -1;
  }
}

// Greedy acceptance with an end-of-sequence token: as the plain greedy rule
// (a node is accepted when its parent is and its token is the parent's
// greedy successor; the deepest accepted node, lowest index on ties, ends
// the branch), except that an accepted EOS node accepts no children and, if
// it ends the branch, there is no next token.
__global__ void accept_eos_kernel(const SampleInfo* samples, int batch, const int32_t* tokens,
                                  const int32_t* parents, const TokInfo* toks, const int32_t* argmax,
                                  int eos, int32_t* accepted_len, int32_t* next_token,
                                  int32_t* accepted_nodes) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const SampleInfo s = samples[b];
  NodeSet open;                                   // accepted and not EOS: may have children
  open.clear();
  if (tokens[s.tok0] != eos) open.add(0);
  int best = 0, best_depth = 0;
  for (int i = 1; i < s.ntok; ++i) {
    const int row = s.tok0 + i;
    const int p = parents[row];
    if (open.has(p) && tokens[row] == argmax[s.tok0 + p]) {
      if (tokens[row] != eos) open.add(i);
      const int d = toks[row].depth;
      if (d > best_depth) { best_depth = d; best = i; }
    }
  }
  accepted_len[b] = best_depth;
  next_token[b] = tokens[s.tok0 + best] == eos ? -1 : argmax[s.tok0 + best];
  int32_t* out = accepted_nodes + (size_t)b * kMaxTree;
  for (int d = best_depth + 1; d < kMaxTree; ++d) out[d] = -1;
  int node = best;
  for (int d = best_depth; d >= 0; --d) {
    out[d] = node;
    node = (node > 0) ? parents[s.tok0 + node] : 0;
  }
}

}  // namespace

size_t sample_accept_scratch(int batch, int n_tokens, int vocab) {
  return (size_t)n_tokens * sizeof(NodeRec) + 256 + (size_t)batch * vocab * sizeof(double);
}

hipError_t launch_sample_accept(const SampleInfo* samples, int batch, int n_tokens,
                                const TokInfo* toks, const int32_t* tokens,
                                const int32_t* parents, const float* logits,
                                const float* draft_probs, const float* uniforms, int vocab,
                                float temperature, int eos, void* scratch, int32_t* accepted_len,
                                int32_t* next_token, int32_t* accepted_nodes, hipStream_t s) {
  const double inv_t = 1.0 / (double)temperature;
  NodeRec* recs = (NodeRec*)scratch;
  double* resid = (double*)((char*)scratch +
                            ((size_t)n_tokens * sizeof(NodeRec) + 255) / 256 * 256);
  node_decide_kernel<1024><<<n_tokens, 1024, 0, s>>>(samples, toks, tokens, parents, logits,
                                                   draft_probs, uniforms, vocab, inv_t, eos, recs);
  sample_walk_kernel<1024><<<batch, 1024, 0, s>>>(samples, tokens, parents, logits, draft_probs,
                                                  uniforms, vocab, inv_t, eos, recs, resid,
                                                  accepted_len, next_token, accepted_nodes);
  return hipGetLastError();
}

hipError_t launch_accept_eos(const SampleInfo* samples, int batch, const int32_t* tokens,
                             const int32_t* parents, const TokInfo* toks, const int32_t* argmax,
                             int eos, int32_t* accepted_len, int32_t* next_token,
                             int32_t* accepted_nodes, hipStream_t s) {
  accept_eos_kernel<<<(batch + 63) / 64, 64, 0, s>>>(samples, batch, tokens, parents, toks, argmax,
                                                     eos, accepted_len, next_token, accepted_nodes);
  return hipGetLastError();
}

}  // namespace spec
