// Decisions of a step and the window bookkeeping, on the device.
//
// Per sequence b, positions p in [0, S_b) map to index off[b] + p of the
// token / decoded-flag arrays.  decoded0 is the decoded-flag snapshot taken at
// the phase start, so "decoded in this phase" = decoded && !decoded0.
#include <climits>

#include "common.h"
#include "kernels.h"

namespace wd {

// ---- confidence: argmax ([MASK] excluded, lowest id on ties) and its softmax probability ----
// Pass 1: block (row, chunk) reduces its slice of the vocabulary to
// (max, lowest argmax, sum exp(l - max)).  Pass 2: one wave per row merges the
// chunks in order.  Both passes use fixed reduction orders.
__device__ __forceinline__ void better(float& bv, int& bi, float ov, int oi) {
  if (ov > bv || (ov == bv && oi < bi)) {
    bv = ov;
    bi = oi;
  }
}

__global__ __launch_bounds__(256) void k_conf_partial(const float* __restrict__ logits, int V,
                                                      int mask_id, float* __restrict__ pmax,
                                                      int* __restrict__ pidx,
                                                      float* __restrict__ psum) {
  __shared__ float bv[4], ss[4];
  __shared__ int bi[4];
  const int row = blockIdx.x, ch = blockIdx.y;
  const int per = (V + kConfChunks - 1) / kConfChunks;
  const int lo = ch * per, hi = min(V, lo + per);
  const float* L = logits + (long)row * V;
  float best = -INFINITY;
  int idx = INT_MAX;
  for (int v = lo + threadIdx.x; v < hi; v += blockDim.x) {
    if (v == mask_id) continue;
    const float x = L[v];
    if (x > best) {
      best = x;
      idx = v;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) better(best, idx, __shfl_xor(best, o, 64), __shfl_xor(idx, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    bv[w] = best;
    bi[w] = idx;
  }
  __syncthreads();
  best = bv[0];
  idx = bi[0];
  for (int i = 1; i < 4; ++i) better(best, idx, bv[i], bi[i]);
  float s = 0.f;
  if (best > -INFINITY)
    for (int v = lo + threadIdx.x; v < hi; v += blockDim.x)
      if (v != mask_id) s += expf(L[v] - best);
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) ss[w] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    const int k = row * kConfChunks + ch;
    pmax[k] = best;
    pidx[k] = idx;
    psum[k] = ss[0] + ss[1] + ss[2] + ss[3];
  }
}

__global__ __launch_bounds__(64) void k_conf_final(const float* __restrict__ pmax,
                                                   const int* __restrict__ pidx,
                                                   const float* __restrict__ psum,
                                                   int32_t* __restrict__ tok,
                                                   float* __restrict__ conf) {
  const int row = blockIdx.x;
  if (threadIdx.x != 0) return;
  float best = -INFINITY;
  int idx = INT_MAX;
  for (int c = 0; c < kConfChunks; ++c)
    better(best, idx, pmax[row * kConfChunks + c], pidx[row * kConfChunks + c]);
  float s = 0.f;
  for (int c = 0; c < kConfChunks; ++c) {
    const float m = pmax[row * kConfChunks + c];
    if (m > -INFINITY) s += psum[row * kConfChunks + c] * expf(m - best);
  }
  tok[row] = idx;
  conf[row] = 1.0f / s;
}

hipError_t confidence(const float* logits, int n, int V, int mask_id, int32_t* tok, float* conf,
                      float* scratch, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  float* pmax = scratch;
  int* pidx = (int*)(scratch + (long)n * kConfChunks);
  float* psum = scratch + 2L * n * kConfChunks;
  hipLaunchKernelGGL(k_conf_partial, dim3(n, kConfChunks), dim3(256), 0, st, logits, V, mask_id,
                     pmax, pidx, psum);
  hipLaunchKernelGGL(k_conf_final, dim3(n), dim3(64), 0, st, pmax, pidx, psum, tok, conf);
  return hipGetLastError();
}

// Merge of the LM head's per-tile (max, argmax, sum exp) of one row: each
// thread takes tiles tid, tid + 256, ... in order, then a fixed tree over the
// block; the same rules (lowest id on ties, sums rescaled to the row max).
__global__ __launch_bounds__(256) void k_conf_tiles(const float* __restrict__ pmax,
                                                    const int* __restrict__ pidx,
                                                    const float* __restrict__ psum, int n_tiles,
                                                    int32_t* __restrict__ tok,
                                                    float* __restrict__ conf) {
  __shared__ float bv[4], ss[4];
  __shared__ int bi[4];
  const long base = (long)blockIdx.x * n_tiles;
  float best = -INFINITY;
  int idx = INT_MAX;
  for (int t = threadIdx.x; t < n_tiles; t += blockDim.x) better(best, idx, pmax[base + t], pidx[base + t]);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) better(best, idx, __shfl_xor(best, o, 64), __shfl_xor(idx, o, 64));
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    bv[w] = best;
    bi[w] = idx;
  }
  __syncthreads();
  best = bv[0];
  idx = bi[0];
  for (int i = 1; i < 4; ++i) better(best, idx, bv[i], bi[i]);
  float s = 0.f;
  if (best > -INFINITY)
    for (int t = threadIdx.x; t < n_tiles; t += blockDim.x) {
      const float m = pmax[base + t];
      if (m > -INFINITY) s += psum[base + t] * expf(m - best);
    }
  s = wave_sum(s);
  if ((threadIdx.x & 63) == 0) ss[w] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    tok[blockIdx.x] = idx;
    conf[blockIdx.x] = 1.0f / (ss[0] + ss[1] + ss[2] + ss[3]);
  }
}

hipError_t confidence_tiles(const float* pmax, const int* pidx, const float* psum, int n,
                            int n_tiles, int32_t* tok, float* conf, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_conf_tiles, dim3(n), dim3(256), 0, st, pmax, pidx, psum, n_tiles, tok, conf);
  return hipGetLastError();
}

// ---- block-wide exclusive prefix count of a flag (blockDim.x multiple of 64) ----------
__device__ __forceinline__ int block_prefix(bool f, int* wtot, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  const unsigned long long m = __ballot(f);
  const int in_wave = __popcll(m & ((1ull << lane) - 1ull));
  __syncthreads();
  if (lane == 0) wtot[w] = __popcll(m);
  __syncthreads();
  int before = 0;
  total = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) before += wtot[i];
    total += wtot[i];
  }
  return before + in_wave;
}

// ---- row set of a step ----------------------------------------------------------------------
// One workgroup per sequence walks positions [0, c) in order, so rows come
// out sorted by position.  Active positions are the first n_act undecoded
// ones (the internal window); rows, by the sequence's mode g.mode[b]:
//   0 (refresh): every position of [0, c), row = row0 + p
//   1 (normal):  active positions and positions decoded in the phase
//   2 (full):    every position of [0, c), every undecoded one active
//   3 (buffer-only refresh): undecoded positions of [0, c) and positions
//                decoded during the previous phase (dec0 set, decp clear)
//  -1:           none (a finished sequence)
// c = g.ctx[b].  Sequence b has g.nact[b] active positions, stored at
// compact indices b * n_act + rank (n_act = the stride, at least every
// g.nact[b]); unused slots get position -1.
// err bit 0: the row or active count differs from the host's schedule.
__device__ __forceinline__ bool compact_mode(int mode) { return mode == 1 || mode == 3; }

__global__ __launch_bounds__(1024) void k_build_rows(const uint8_t* __restrict__ dec,
                                                     const uint8_t* __restrict__ dec0,
                                                     const uint8_t* __restrict__ decp, int n_act,
                                                     WdStepGeom g, int32_t* __restrict__ row_tok,
                                                     int32_t* __restrict__ row_pos,
                                                     int32_t* __restrict__ row_seq,
                                                     int32_t* __restrict__ row_out,
                                                     int32_t* __restrict__ act_pos,
                                                     int32_t* __restrict__ err) {
  __shared__ int wtot[16];
  const int b = blockIdx.x;
  const int mode = g.mode[b], na = g.nact[b];
  const int off = g.off[b], c = mode < 0 ? 0 : g.ctx[b], row0 = g.row0[b], nrows = g.nrows[b];
  int carry_u = 0, carry_o = 0;
  for (int base = 0; base < c; base += blockDim.x) {
    const int p = base + threadIdx.x;
    const bool valid = p < c;
    const bool d = valid ? dec[off + p] != 0 : true;
    const bool und = valid && !d;
    int tot_u, tot_o;
    const int rank_u = carry_u + block_prefix(und, wtot, tot_u);
    const bool act = und && rank_u < na;
    bool online;
    if (mode == 1)
      online = act || (valid && d && dec0[off + p] == 0);
    else if (mode == 3)
      online = und || (valid && d && dec0[off + p] != 0 && decp[off + p] == 0);
    else
      online = valid;
    const int rank_o = carry_o + block_prefix(online, wtot, tot_o);
    const int ro = compact_mode(mode) ? rank_o : p;
    if (online && ro < nrows) {
      const int r = row0 + ro;
      row_tok[r] = off + p;
      row_pos[r] = p;
      row_seq[r] = b;
      row_out[r] = act ? b * n_act + rank_u : -1;
    }
    if (act) act_pos[b * n_act + rank_u] = p;
    carry_u += tot_u;
    carry_o += tot_o;
  }
  // A count that disagrees with the host's schedule is reported through err;
  // the slots it left unwritten get harmless values so later kernels stay in
  // bounds (position 0 of the sequence, no active row).
  const int wrote_o = compact_mode(mode) ? carry_o : c;
  for (int i = wrote_o + threadIdx.x; i < nrows; i += blockDim.x) {
    row_tok[row0 + i] = off;
    row_pos[row0 + i] = 0;
    row_seq[row0 + i] = b;
    row_out[row0 + i] = -1;
  }
  for (int i = min(carry_u, na) + threadIdx.x; i < n_act; i += blockDim.x) act_pos[b * n_act + i] = -1;
  if (threadIdx.x == 0) {
    if (wrote_o != nrows || carry_u < na || na > n_act) atomicOr(err, 1);
  }
}

hipError_t build_rows(const uint8_t* decoded, const uint8_t* decoded0, const uint8_t* decoded_prev,
                      int n_act, const WdStepGeom& g, int32_t* row_tok, int32_t* row_pos,
                      int32_t* row_seq, int32_t* row_out, int32_t* act_pos, int32_t* err,
                      hipStream_t st) {
  hipLaunchKernelGGL(k_build_rows, dim3(g.batch), dim3(1024), 0, st, decoded, decoded0,
                     decoded_prev, n_act, g, row_tok, row_pos, row_seq, row_out, act_pos, err);
  return hipGetLastError();
}

// ---- phase start ------------------------------------------------------------------------------
// Sequences with g.mode[b] == 0 start a phase: their decoded flags are
// snapshot (D_p is measured against it; the previous snapshot moves to
// decp) and their window is checked.
__global__ void k_snapshot(const uint8_t* __restrict__ dec, uint8_t* __restrict__ dec0,
                           uint8_t* __restrict__ decp, WdStepGeom g,
                           const int32_t* __restrict__ seq_len) {
  const int b = blockIdx.y;
  if (g.mode[b] != 0) return;
  const long off = g.off[b];
  for (int p = blockIdx.x * blockDim.x + threadIdx.x; p < seq_len[b]; p += gridDim.x * blockDim.x) {
    decp[off + p] = dec0[off + p];
    dec0[off + p] = dec[off + p];
  }
}

// err bit 1: c is not (E-th undecoded position below end + 1), or end when
// fewer remain.
__global__ __launch_bounds__(1024) void k_check_window(const uint8_t* __restrict__ dec, int E,
                                                       WdStepGeom g,
                                                       int32_t* __restrict__ err) {
  __shared__ int red[16];
  const int b = blockIdx.x;
  if (g.mode[b] != 0) return;
  const int off = g.off[b], c = g.ctx[b], S = g.end[b];
  int below = 0, all = 0;
  for (int p = threadIdx.x; p < S; p += blockDim.x) {
    const int u = dec[off + p] == 0;
    all += u;
    if (p < c) below += u;
  }
  int t;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int o = 32; o > 0; o >>= 1) {
    below += __shfl_xor(below, o, 64);
    all += __shfl_xor(all, o, 64);
  }
  if (lane == 0) red[w] = below;
  __syncthreads();
  t = 0;
  for (int i = 0; i < nw; ++i) t += red[i];
  below = t;
  __syncthreads();
  if (lane == 0) red[w] = all;
  __syncthreads();
  t = 0;
  for (int i = 0; i < nw; ++i) t += red[i];
  all = t;
  if (threadIdx.x == 0) {
    bool ok;
    if (all >= E)
      ok = below == E && c >= 1 && c <= S && dec[off + c - 1] == 0;
    else
      ok = c == S;
    if (!ok) atomicOr(err, 2);
  }
}

hipError_t slide(const uint8_t* decoded, uint8_t* decoded0, uint8_t* decoded_prev, int Smax, int E,
                 const WdStepGeom& g, const int32_t* seq_len, int32_t* err, hipStream_t st) {
  const int chunks = std::max(1, std::min(64, (Smax + 255) / 256));
  hipLaunchKernelGGL(k_snapshot, dim3(chunks, g.batch), dim3(256), 0, st, decoded, decoded0,
                     decoded_prev, g, seq_len);
  hipLaunchKernelGGL(k_check_window, dim3(g.batch), dim3(1024), 0, st, decoded, E, g, err);
  return hipGetLastError();
}

// ---- top-k decode -------------------------------------------------------------------------------
// Candidate i of sequence b (index b * n_act + i) ranks by (conf desc,
// position asc); the k best are decoded.
// err bit 2: sequence b decoded other than min(k, g.nact[b]) positions, or a
// candidate was already decoded (the host's schedule assumes neither).
__global__ __launch_bounds__(256) void k_select_update(const int32_t* __restrict__ act_pos,
                                                       const int32_t* __restrict__ act_tok,
                                                       const float* __restrict__ act_conf,
                                                       int n_act, int k, WdStepGeom g,
                                                       const int32_t* __restrict__ seq_len,
                                                       int32_t* __restrict__ x,
                                                       uint8_t* __restrict__ dec,
                                                       int32_t* __restrict__ sel_pos,
                                                       int32_t* __restrict__ sel_tok,
                                                       float* __restrict__ sel_conf,
                                                       int32_t* __restrict__ err) {
  __shared__ int n_sel, bad;
  const int b = blockIdx.x;
  const long base = (long)b * n_act;
  for (int i = threadIdx.x; i < k; i += blockDim.x) {
    sel_pos[b * k + i] = -1;
    sel_tok[b * k + i] = -1;
    sel_conf[b * k + i] = 0.f;
  }
  if (threadIdx.x == 0) n_sel = bad = 0;
  __syncthreads();
  const int S = seq_len[b];
  for (int i = threadIdx.x; i < n_act; i += blockDim.x) {
    const float ci = act_conf[base + i];
    const int pi = act_pos[base + i];
    if (pi < 0 || pi >= S) continue;  // a slot the bookkeeping flagged as missing
    int rank = 0;
    for (int j = 0; j < n_act; ++j) {
      const float cj = act_conf[base + j];
      const int pj = act_pos[base + j];
      if (pj < 0 || pj >= S) continue;
      rank += (cj > ci) || (cj == ci && pj < pi);
    }
    if (rank < k) {
      // each thread reads and writes only its own candidate's flag
      if (dec[g.off[b] + pi]) atomicOr(&bad, 1);
      const int t = act_tok[base + i];
      sel_pos[b * k + rank] = pi;
      sel_tok[b * k + rank] = t;
      sel_conf[b * k + rank] = ci;
      x[g.off[b] + pi] = t;
      dec[g.off[b] + pi] = 1;
      atomicAdd(&n_sel, 1);
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int want = g.mode[b] < 0 ? 0 : min(k, g.nact[b]);
    if (bad || n_sel != want) atomicOr(err, 4);
  }
}

hipError_t select_update(const int32_t* act_pos, const int32_t* act_tok, const float* act_conf,
                         int n_act, int k, const WdStepGeom& g, const int32_t* seq_len, int32_t* x,
                         uint8_t* decoded, int32_t* sel_pos, int32_t* sel_tok, float* sel_conf,
                         int32_t* err, hipStream_t st) {
  hipLaunchKernelGGL(k_select_update, dim3(g.batch), dim3(256), 0, st, act_pos, act_tok, act_conf,
                     n_act, k, g, seq_len, x, decoded, sel_pos, sel_tok, sel_conf, err);
  return hipGetLastError();
}

}  // namespace wd
