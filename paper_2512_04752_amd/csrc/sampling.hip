// Tree acceptance at a sampling temperature (speculative sampling over the
// draft tree), and greedy acceptance with an end-of-sequence token.
//
// Speculative decoding is lossless (RLHFSpec Section 2.2: the verified
// output follows the target model's distribution).  At temperature T > 0
// every node u has the target distribution p_u = softmax(z_u / T) of the
// token after it, and the draft drew u's children independently from its
// own distribution q_u.  The walk from the root (multi-draft speculative
// sampling) keeps an unnormalised residual P with total R, starting at
// P = exp(z_u / T - max(z_u) / T) (so p_u = P / R), and tries u's children
// in node order: child c with token x is accepted when a_c * q_u(x) * R < P(x)
// (probability min(1, p'(x) / q_u(x)) for the normalised residual p' = P / R);
// a rejected child turns P into max(P - R q_u, 0) (R times the textbook
// residual max(p' - q_u, 0)).  The walk moves to an accepted child; when no child is
// accepted (or u has none) the next token is drawn from P by inverse CDF with
// u's second uniform.  a_c and the sampling draws are inputs.
//
// Vocabulary-wide work runs in fp64 (residuals, sums, the CDF) so that the
// decisions are those of a float64 statement of the same procedure; the
// logits themselves are the forward pass's fp32 values.
//
// End of sequence: an accepted node carrying the EOS token ends the branch
// (its children are not tried, no next token: -1).
#include <math.h>

#include "common.h"

namespace spec {

namespace {

constexpr int NT = 512;   // 8 waves: one work-group walks one sample's tree

// Sum of one fp64 value per thread across the work-group, in a fixed order.
__device__ double block_sum(double v, double* red) {
  red[threadIdx.x] = v;
  __syncthreads();
#pragma unroll
  for (int s = NT / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__device__ float block_max(float v, float* red) {
  red[threadIdx.x] = v;
  __syncthreads();
#pragma unroll
  for (int s = NT / 2; s > 0; s >>= 1) {
    if (threadIdx.x < s) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + s]);
    __syncthreads();
  }
  const float r = red[0];
  __syncthreads();
  return r;
}

// P[y] = exp(z[y] / T - max(z) / T) over the vocabulary (interleaved, so
// each wave reads and writes contiguous runs); returns the fp64 total.
// Unnormalised: p_u = P / total.
__device__ double fill_target(const float* z, int vocab, double inv_t, double* P, double* red,
                              float* redf) {
  float m = -INFINITY;
  for (int y = threadIdx.x; y < vocab; y += NT) m = fmaxf(m, z[y]);
  const double base = (double)block_max(m, redf) * inv_t;
  double part = 0.0;
  for (int y = threadIdx.x; y < vocab; y += NT) {
    const double v = exp((double)z[y] * inv_t - base);
    P[y] = v;
    part += v;
  }
  return block_sum(part, red);
}

// One work-group per sample.  P: this sample's [vocab] fp64 residual.  Every
// global write of P is followed by a work-group barrier (inside the block
// reductions) before another thread reads it.
__global__ __launch_bounds__(NT) void sample_accept_kernel(
    const SampleInfo* samples, const int32_t* tokens, const int32_t* parents, const float* logits,
    const float* draft_probs, const float* uniforms, int vocab, double inv_t, int eos,
    double* resid, int32_t* accepted_len, int32_t* next_token, int32_t* accepted_nodes) {
  __shared__ double red[NT];
  __shared__ double scan[NT];
  __shared__ float redf[NT];
  __shared__ int path[kMaxTree];
  const int b = blockIdx.x;
  const SampleInfo s = samples[b];
  double* P = resid + (size_t)b * vocab;

  int u = 0, depth = 0, next = -1;
  if (threadIdx.x == 0) path[0] = 0;
  bool ended = tokens[s.tok0] == eos;           // a root carrying EOS: nothing follows
  while (!ended) {
    const float* z = logits + (size_t)(s.tok0 + u) * vocab;
    double R = fill_target(z, vocab, inv_t, P, red, redf);
    const float* q = draft_probs + (size_t)(s.tok0 + u) * vocab;
    int moved = -1;
    for (int c = u + 1; c < s.ntok; ++c) {
      if (parents[s.tok0 + c] != u) continue;
      const int x = tokens[s.tok0 + c];
      // accept with probability min(1, (P[x] / R) / q[x])
      const double a = (double)uniforms[2 * (size_t)(s.tok0 + c)];
      if (a * (double)q[x] * R < P[x]) {
        moved = c;
        break;
      }
      double part = 0.0;
      for (int y = threadIdx.x; y < vocab; y += NT) {
        const double v = fmax(P[y] - R * (double)q[y], 0.0);
        P[y] = v;
        part += v;
      }
      R = block_sum(part, red);
    }
    if (moved >= 0) {
      u = moved;
      ++depth;
      if (threadIdx.x == 0) path[depth] = u;
      if (tokens[s.tok0 + u] == eos) ended = true;
      continue;
    }
    // No child accepted: draw the next token from P.  A residual with no
    // mass left (only through rounding) falls back to p_u.
    if (!(R > 0.0)) R = fill_target(z, vocab, inv_t, P, red, redf);
    // Inverse CDF: the smallest y whose running sum exceeds a * R.  Each
    // thread sums a contiguous chunk; thread 0 scans the chunk sums in order
    // and walks the chunk holding the target.
    const double target = (double)uniforms[2 * (size_t)(s.tok0 + u) + 1] * R;
    const int chunk = (vocab + NT - 1) / NT;
    const int y0 = threadIdx.x * chunk, y1 = min(vocab, y0 + chunk);
    double part = 0.0;
    for (int y = y0; y < y1; ++y) part += P[y];
    scan[threadIdx.x] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
      double run = 0.0;
      int owner = -1, last = -1;
      for (int t = 0; t < NT; ++t) {
        if (scan[t] > 0.0) last = t;
        if (owner < 0 && run + scan[t] > target) owner = t;
        const double before = run;
        run += scan[t];
        scan[t] = before;                      // exclusive prefix
      }
      if (owner < 0) owner = last;             // target at or past the total: last non-empty chunk
      int pick = -1;
      if (owner >= 0) {                        // < 0 only for non-finite logits
        int lastpos = -1;
        double acc = scan[owner];
        const int a0 = owner * chunk, a1 = min(vocab, a0 + chunk);
        for (int y = a0; y < a1; ++y) {
          if (P[y] > 0.0) lastpos = y;
          acc += P[y];
          if (acc > target) { pick = y; break; }
        }
        if (pick < 0) pick = lastpos;
      }
      red[0] = (double)pick;
    }
    __syncthreads();
    next = (int)red[0];
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
  uint64_t open = tokens[s.tok0] == eos ? 0ull : 1ull;   // accepted and not EOS: may have children
  int best = 0, best_depth = 0;
  for (int i = 1; i < s.ntok; ++i) {
    const int row = s.tok0 + i;
    const int p = parents[row];
    if (((open >> p) & 1ull) && tokens[row] == argmax[s.tok0 + p]) {
      if (tokens[row] != eos) open |= 1ull << i;
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

hipError_t launch_sample_accept(const SampleInfo* samples, int batch, const int32_t* tokens,
                                const int32_t* parents, const float* logits,
                                const float* draft_probs, const float* uniforms, int vocab,
                                float temperature, int eos, double* resid, int32_t* accepted_len,
                                int32_t* next_token, int32_t* accepted_nodes, hipStream_t s) {
  const double inv_t = 1.0 / (double)temperature;
  sample_accept_kernel<<<batch, NT, 0, s>>>(samples, tokens, parents, logits, draft_probs,
                                            uniforms, vocab, inv_t, eos, resid, accepted_len,
                                            next_token, accepted_nodes);
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
