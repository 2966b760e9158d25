// The small kernels of the verify step: tree metadata, rotary angle table,
// embedding gather, RMSNorm, the final argmax reduction, greedy tree
// acceptance and KV compaction.
#include <math.h>

#include "common.h"

namespace spec {

namespace {

// Depth, position and ancestor set of every node: one work-group per sample,
// thread i = node i (a tree has at most kMaxTree nodes).  The set is
// kAncWords 64-bit words, bit t % 64 of word t / 64 standing for node t.
// Pointer jumping: node i holds the set of its ancestors at distance < 2^r
// and its ancestor at distance 2^r (the root points at itself); each round
// publishes both in LDS and takes "set |= set of that ancestor, jump to its
// jump", so ceil(log2 T) rounds cover every depth below T.  Depth is the
// set's size minus one.
__global__ __launch_bounds__(kMaxTree) void tree_meta_kernel(const SampleInfo* samples,
                                                             const int32_t* parents, TokInfo* toks,
                                                             uint64_t* anc, int32_t* dbg_depth,
                                                             int32_t* dbg_pos, uint64_t* dbg_anc) {
  __shared__ uint64_t sset[kMaxTree][kAncWords];
  __shared__ int sjump[kMaxTree];
  const int b = blockIdx.x, i = threadIdx.x;
  const SampleInfo s = samples[b];
  const bool live = i < s.ntok;
  int jump = (live && i > 0) ? parents[s.tok0 + i] : i;
  uint64_t set[kAncWords];
#pragma unroll
  for (int w = 0; w < kAncWords; ++w) set[w] = w == (i >> 6) ? 1ull << (i & 63) : 0ull;
  for (int r = 0; (1 << r) < s.ntok; ++r) {     // same bound in every thread of the sample
#pragma unroll
    for (int w = 0; w < kAncWords; ++w) sset[i][w] = set[w];
    sjump[i] = jump;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kAncWords; ++w) set[w] |= sset[jump][w];
    jump = sjump[jump];
    __syncthreads();
  }
  if (!live) return;
  int size = 0;
#pragma unroll
  for (int w = 0; w < kAncWords; ++w) size += __popcll(set[w]);
  const int row = s.tok0 + i, depth = size - 1;
  toks[row] = TokInfo{b, i, s.seq_len + depth, depth};
#pragma unroll
  for (int w = 0; w < kAncWords; ++w) {
    anc[(size_t)row * kAncWords + w] = set[w];
    if (dbg_anc) dbg_anc[(size_t)row * kAncWords + w] = set[w];
  }
  if (dbg_depth) dbg_depth[row] = depth;
  if (dbg_pos) dbg_pos[row] = s.seq_len + depth;
}

// cos/sin of position * theta^(-2j/d), angles in double precision.
__global__ void rope_table_kernel(const TokInfo* toks, int n, int half, int head_dim, double theta,
                                  float2* cs) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= n * half) return;
  const int row = idx / half, j = idx % half;
  const double freq = pow(theta, -2.0 * (double)j / (double)head_dim);
  const double ang = (double)toks[row].pos * freq;
  double sn, cn;
  sincos(ang, &sn, &cn);
  cs[idx] = make_float2((float)cn, (float)sn);
}

__global__ void embed_kernel(const int32_t* tokens, const bf16* table, float* x, int hidden) {
  const int row = blockIdx.x;
  const bf16* src = table + (size_t)tokens[row] * hidden;
  float* dst = x + (size_t)row * hidden;
  for (int c = threadIdx.x * 8; c < hidden; c += blockDim.x * 8) {
    const bf16x8 v = *(const bf16x8*)(src + c);
    f32x4 lo = {(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
    f32x4 hi = {(float)v[4], (float)v[5], (float)v[6], (float)v[7]};
    *(f32x4*)(dst + c) = lo;
    *(f32x4*)(dst + c + 4) = hi;
  }
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
  return v;
}

// out = bf16(x / sqrt(mean(x^2) + eps) * gain), one 256-thread block per row.
// CPT > 0: the row is CPT 4-float chunks per thread (hidden <= 1024 * CPT),
// all loaded (with their gains) before any is used, so a short row costs one
// memory round trip (with few rows there are few blocks to hide latency);
// CPT = 0: any length, a strided loop.  Both sum each thread's chunks in
// column order, then the lanes, then the four waves: the same result.
template <int CPT>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const float* x, const bf16* gain, bf16* out,
                                                      int hidden, float eps) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const float* xr = x + (size_t)row * hidden;
  bf16* orow = out + (size_t)row * hidden;
  float ss = 0.f;
  if constexpr (CPT > 0) {
    f32x4 v[CPT];
    bf16x4 g[CPT];
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int c = (threadIdx.x + 256 * k) * 4;
      if (c < hidden) {
        v[k] = *(const f32x4*)(xr + c);
        g[k] = *(const bf16x4*)(gain + c);
      }
    }
#pragma unroll
    for (int k = 0; k < CPT; ++k)
      if ((threadIdx.x + 256 * k) * 4 < hidden)
        ss += v[k][0] * v[k][0] + v[k][1] * v[k][1] + v[k][2] * v[k][2] + v[k][3] * v[k][3];
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = red[0] + red[1] + red[2] + red[3];
    const float rstd = rsqrtf(tot / (float)hidden + eps);
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int c = (threadIdx.x + 256 * k) * 4;
      if (c < hidden) {
        bf16x4 y;
#pragma unroll
        for (int j = 0; j < 4; ++j) y[j] = (bf16)(v[k][j] * rstd * (float)g[k][j]);
        *(bf16x4*)(orow + c) = y;
      }
    }
  } else {
    for (int c = threadIdx.x * 4; c < hidden; c += 256 * 4) {
      const f32x4 v = *(const f32x4*)(xr + c);
      ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
    }
    ss = wave_sum(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    const float tot = red[0] + red[1] + red[2] + red[3];
    const float rstd = rsqrtf(tot / (float)hidden + eps);
    for (int c = threadIdx.x * 4; c < hidden; c += 256 * 4) {
      const f32x4 v = *(const f32x4*)(xr + c);
      const bf16x4 g = *(const bf16x4*)(gain + c);
      bf16x4 y;
#pragma unroll
      for (int k = 0; k < 4; ++k) y[k] = (bf16)(v[k] * rstd * (float)g[k]);
      *(bf16x4*)(orow + c) = y;
    }
  }
}

// Row maximum over the LM-head partials; ties go to the lowest token id.
__global__ __launch_bounds__(256) void argmax_reduce_kernel(const float* part_val,
                                                            const int32_t* part_idx, int parts,
                                                            int32_t* argmax, int32_t* dbg_argmax) {
  // (max, lowest index) is the same whatever order the partials are visited
  // in, so each thread loads eight of them before comparing any: one memory
  // round trip per 2048 partials instead of a dependent load per step.
  constexpr int U = 8;
  __shared__ float sv[4];
  __shared__ int si[4];
  const int row = blockIdx.x;
  const float* pvr = part_val + (size_t)row * parts;
  const int32_t* pir = part_idx + (size_t)row * parts;
  float v = -INFINITY;
  int idx = 0x7fffffff;
  for (int p0 = threadIdx.x; p0 < parts; p0 += 256 * U) {
    float pv[U];
    int pi[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int p = p0 + 256 * u;
      pv[u] = p < parts ? pvr[p] : -INFINITY;
      pi[u] = p < parts ? pir[p] : 0x7fffffff;
    }
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (pv[u] > v || (pv[u] == v && pi[u] < idx)) { v = pv[u]; idx = pi[u]; }
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(v, m);
    const int oi = __shfl_xor(idx, m);
    if (ov > v || (ov == v && oi < idx)) { v = ov; idx = oi; }
  }
  if ((threadIdx.x & 63) == 0) { sv[threadIdx.x >> 6] = v; si[threadIdx.x >> 6] = idx; }
  __syncthreads();
  if (threadIdx.x == 0) {
#pragma unroll
    for (int w = 1; w < 4; ++w)
      if (sv[w] > v || (sv[w] == v && si[w] < idx)) { v = sv[w]; idx = si[w]; }
    if (idx == 0x7fffffff) idx = 0;   // every logit NaN: report token 0
    argmax[row] = idx;
    if (dbg_argmax) dbg_argmax[row] = idx;
  }
}

// Greedy tree acceptance, one thread per sample: a node is accepted when its
// parent is and its token is the parent's greedy successor; the deepest
// accepted node (lowest index on ties) ends the accepted branch.
__global__ void accept_kernel(const SampleInfo* samples, int batch, const int32_t* tokens,
                              const int32_t* parents, const TokInfo* toks, const int32_t* argmax,
                              int32_t* accepted_len, int32_t* next_token,
                              int32_t* accepted_nodes) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const SampleInfo s = samples[b];
  NodeSet acc;
  acc.clear();
  acc.add(0);
  int best = 0, best_depth = 0;
  for (int i = 1; i < s.ntok; ++i) {
    const int row = s.tok0 + i;
    const int p = parents[row];
    if (acc.has(p) && tokens[row] == argmax[s.tok0 + p]) {
      acc.add(i);
      const int d = toks[row].depth;
      if (d > best_depth) { best_depth = d; best = i; }
    }
  }
  accepted_len[b] = best_depth;
  next_token[b] = argmax[s.tok0 + best];
  int32_t* out = accepted_nodes + (size_t)b * kMaxTree;
  for (int d = best_depth + 1; d < kMaxTree; ++d) out[d] = -1;
  int node = best;
  for (int d = best_depth; d >= 0; --d) {
    out[d] = node;
    node = (node > 0) ? parents[s.tok0 + node] : 0;
  }
}

// Move the accepted branch of one sample, for one layer and a group of K/V heads, to positions
// S_b + 1 .. S_b + accepted_len: row d takes the row of node path[d] > d (rows with path[d] == d
// stay).  Every row written before row d lies below d, and every source of row d or later lies
// above it, so the chunks go in passes of increasing d.  Within a pass a source can be the
// destination of a deeper row, so each pass reads all its chunks into registers, the work-group
// synchronises, and then the pass writes.
template <int HD>
__global__ __launch_bounds__(256) void compact_kernel(const SampleInfo* samples, bf16* kv_pool,
                                                      int n_kv_heads, int heads_per_wg,
                                                      const int32_t* accepted_len,
                                                      const int32_t* accepted_nodes,
                                                      int32_t* new_seq_lens) {
  constexpr int DC = HD / 8;  // 16-byte chunks per row of one head
  constexpr int PER = 8;      // chunks per thread and pass
  const int b = blockIdx.x, layer = blockIdx.y;
  const SampleInfo s = samples[b];
  int acc = accepted_len[b];
  if (acc < 0) acc = 0;
  if (acc > s.ntok - 1) acc = s.ntok - 1;
  if (s.seq_len + acc >= s.cap) acc = s.cap - 1 - s.seq_len;
  if (layer == 0 && blockIdx.z == 0 && threadIdx.x == 0) new_seq_lens[b] = s.seq_len + acc + 1;
  if (acc == 0) return;
  const size_t head_stride = (size_t)s.cap * HD;
  bf16* base = kv_pool + s.kv_base +
               ((size_t)layer * 2 * n_kv_heads + (size_t)blockIdx.z * heads_per_wg) * head_stride;
  const int32_t* nodes = accepted_nodes + (size_t)b * kMaxTree;
  const int per_row = heads_per_wg * DC, total = acc * per_row;
  for (int q0 = 0; q0 < total; q0 += 256 * PER) {
    i32x4 v[PER];
    int64_t dst[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int q = q0 + threadIdx.x + 256 * k;
      dst[k] = -1;
      if (q < total) {
        const int d = 1 + q / per_row, r = q % per_row;
        const int nd = nodes[d];
        if (nd > d && nd < s.ntok && s.seq_len + nd < s.cap) {
          const int64_t col = (int64_t)(r / DC) * head_stride + (r % DC) * 8;
          v[k] = *(const i32x4*)(base + col + (int64_t)(s.seq_len + nd) * HD);
          dst[k] = col + (int64_t)(s.seq_len + d) * HD;
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < PER; ++k)
      if (dst[k] >= 0) *(i32x4*)(base + dst[k]) = v[k];
  }
}

}  // namespace

hipError_t launch_tree_meta(const SampleInfo* samples, int batch, const int32_t* parents,
                            TokInfo* toks, uint64_t* anc, int32_t* dbg_depth, int32_t* dbg_pos,
                            uint64_t* dbg_anc, hipStream_t s) {
  tree_meta_kernel<<<batch, kMaxTree, 0, s>>>(samples, parents, toks, anc, dbg_depth, dbg_pos,
                                               dbg_anc);
  return hipGetLastError();
}

hipError_t launch_rope_table(const TokInfo* toks, int n, int head_dim, float theta, float2* cs,
                             hipStream_t s) {
  const int half = head_dim / 2;
  const int total = n * half;
  rope_table_kernel<<<(total + 255) / 256, 256, 0, s>>>(toks, n, half, head_dim, (double)theta, cs);
  return hipGetLastError();
}

hipError_t launch_embed(const int32_t* tokens, const bf16* table, float* x, int n, int hidden,
                        hipStream_t s) {
  embed_kernel<<<n, 256, 0, s>>>(tokens, table, x, hidden);
  return hipGetLastError();
}

hipError_t launch_rmsnorm(const float* x, const bf16* gain, bf16* out, int n, int hidden,
                          float eps, hipStream_t s) {
  switch ((hidden + 1023) / 1024) {
    case 1: rmsnorm_kernel<1><<<n, 256, 0, s>>>(x, gain, out, hidden, eps); break;
    case 2: rmsnorm_kernel<2><<<n, 256, 0, s>>>(x, gain, out, hidden, eps); break;
    case 3:
    case 4: rmsnorm_kernel<4><<<n, 256, 0, s>>>(x, gain, out, hidden, eps); break;
    case 5: case 6: case 7:
    case 8: rmsnorm_kernel<8><<<n, 256, 0, s>>>(x, gain, out, hidden, eps); break;
    default: rmsnorm_kernel<0><<<n, 256, 0, s>>>(x, gain, out, hidden, eps); break;
  }
  return hipGetLastError();
}

hipError_t launch_argmax_reduce(const float* part_val, const int32_t* part_idx, int n, int parts,
                                int32_t* argmax, int32_t* dbg_argmax, hipStream_t s) {
  argmax_reduce_kernel<<<n, 256, 0, s>>>(part_val, part_idx, parts, argmax, dbg_argmax);
  return hipGetLastError();
}

hipError_t launch_accept(const SampleInfo* samples, int batch, const int32_t* tokens,
                         const int32_t* parents, const TokInfo* toks, const int32_t* argmax,
                         int32_t* accepted_len, int32_t* next_token, int32_t* accepted_nodes,
                         hipStream_t s) {
  accept_kernel<<<(batch + 63) / 64, 64, 0, s>>>(samples, batch, tokens, parents, toks, argmax,
                                                 accepted_len, next_token, accepted_nodes);
  return hipGetLastError();
}

hipError_t launch_compact(const SampleInfo* samples, int batch, bf16* kv_pool, int n_layers,
                          int n_kv_heads, int head_dim, const int32_t* accepted_len,
                          const int32_t* accepted_nodes, int32_t* new_seq_lens, hipStream_t s) {
  // Head groups split each (sample, layer) only as far as it takes to give the launch about
  // a thousand work-groups: at large batch one work-group moves all K/V heads of a layer.
  const int heads = 2 * n_kv_heads;
  int groups = 1;
  while (groups < heads && (int64_t)batch * n_layers * groups < 1024) {
    ++groups;
    while (heads % groups) ++groups;
  }
  const dim3 grid(batch, n_layers, groups);
  const int hpw = heads / groups;
  if (head_dim == 128)
    compact_kernel<128><<<grid, 256, 0, s>>>(samples, kv_pool, n_kv_heads, hpw, accepted_len,
                                             accepted_nodes, new_seq_lens);
  else if (head_dim == 64)
    compact_kernel<64><<<grid, 256, 0, s>>>(samples, kv_pool, n_kv_heads, hpw, accepted_len,
                                            accepted_nodes, new_seq_lens);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace spec
