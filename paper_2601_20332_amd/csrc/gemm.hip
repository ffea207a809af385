// Projection GEMMs of the decoder layers and the LM head:
//   C[s][m][n] = sum_{k in split s} X[m][k] * W[n][k]
// X is the activation block (rows of the step's row set), W a weight matrix
// in [out_features, in_features] layout.  Callers reduce the S split-K
// partials in their fused epilogues.
//
// bf16 path: weights are streamed once from HBM as pre-packed 16x32 MFMA
// fragments (1 KB per fragment, one fully coalesced 16-byte load per lane),
// activations are read from L2, products run on v_mfma_f32_16x16x32_bf16.
// At the row counts of a normal step (tens of rows) the kernel is bound by
// HBM bandwidth on the weight stream; the split-K factor is chosen so that a
// launch has enough workgroups to keep every CU's memory pipeline full.
#include <hip/hip_ext.h>

#include <algorithm>
#include <climits>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace wd {

// ---- weight packing -------------------------------------------------------------
// Fragment (nt, kt) holds packed rows nt*16..nt*16+15 and columns
// kt*32..kt*32+31; lane l stores packed row nt*16 + l%16, columns
// kt*32 + (l/16)*8 .. +7 (the MFMA A-operand layout).  Fragments of one
// 16-row group are contiguous along K, so a wave streams each group as one
// contiguous run.
//
// Row order of the packed matrix (which output feature each packed row is):
//   kPackPlain:    as given.
//   kPackRopePair: within each 128-row head, group gi (packed rows
//                  gi*16..gi*16+15) holds dims gi*8..gi*8+7, then their RoPE
//                  partners 64+gi*8..64+gi*8+7, so that in the MFMA output a
//                  value and its partner sit in lanes l and l ^ 32.
//   kPackGateUp:   W (gate, F rows) and W2 (up, F rows) interleaved: group g
//                  holds gate features g*8..g*8+7, then the same up features.
__device__ __forceinline__ long packed_source_row(int perm, long row, int N, int& which) {
  which = 0;
  if (perm == kPackRopePair) {
    const long head = row >> 7;
    const int r = (int)(row & 127), gi = r >> 4, rr = r & 15;
    return head * 128 + (rr < 8 ? gi * 8 + rr : 64 + gi * 8 + rr - 8);
  }
  if (perm == kPackGateUp) {
    const int rr = (int)(row & 15);
    which = rr >= 8;
    return (row >> 4) * 8 + (rr & 7);
  }
  return row;
}

__global__ void k_pack_frags(const uint16_t* __restrict__ W, const uint16_t* __restrict__ W2, int N,
                             int K, int perm, u32x4* __restrict__ out) {
  const int KT = K >> 5;
  const long total = (long)(N >> 4) * KT * 64;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const long f = i >> 6;
    const int kt = (int)(f % KT);
    const long nt = f / KT;
    int which;
    const long row = packed_source_row(perm, nt * 16 + (lane & 15), N, which);
    const int col = kt * 32 + (lane >> 4) * 8;
    out[i] = *(const u32x4*)((which ? W2 : W) + row * K + col);
  }
}

hipError_t pack_frags(const uint16_t* W, int N, int K, void* out, hipStream_t st, int perm,
                      const uint16_t* W2) {
  if (N % 16 || K % 32) return hipErrorInvalidValue;
  if (perm == kPackRopePair && N % 128) return hipErrorInvalidValue;
  if (perm == kPackGateUp && !W2) return hipErrorInvalidValue;
  const long total = (long)(N / 16) * (K / 32) * 64;
  const int blocks = (int)std::min<long>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_pack_frags, dim3(blocks), dim3(256), 0, st, W, W2, N, K, perm, (u32x4*)out);
  return hipGetLastError();
}

// ---- FP8 (e4m3) weights: per-row scales, packing, decode ----------------------------
// The FP8-weight variant stores each projection matrix as e4m3 codes with one
// float32 scale per output row: s_n = max_k |W[n][k]| / 448 (1 for a zero
// row), code = the e4m3 value nearest to W[n][k] / s_n (float32 quotient,
// ties to the even code, saturating at 448).  A packed fp8 fragment (nt, kt2)
// holds packed rows nt*16..+15 and K columns kt2*64..+63: lane l holds row
// nt*16 + l%16, K columns kt2*64 + (l/16)*8 .. +7 (bytes 0-7) and
// kt2*64 + 32 + (l/16)*8 .. +7 (bytes 8-15), i.e. the A operands of K steps
// 2 kt2 and 2 kt2 + 1 once decoded to bf16 (e4m3 values are exact in bf16).
// The GEMMs multiply each output feature's fp32 sum by its scale.
__device__ __forceinline__ uint32_t e4m3_code(float x) {
  const uint32_t sign = (__float_as_uint(x) >> 31) << 7;
  const float a = fabsf(x);
  if (!(a < 448.f)) return sign | 0x7Eu;
  if (a < 0x1p-6f) return sign | (uint32_t)rintf(a * 512.f);  // m * 2^-9; m = 8 is 2^-6
  int e;
  const float mant = frexpf(a, &e) * 2.f;                       // a = mant * 2^(e-1)
  float q = rintf((mant - 1.f) * 8.f);
  int E = e - 1 + 7;
  if (q == 8.f) {
    q = 0.f;
    ++E;
  }
  const uint32_t code = min((uint32_t)(E << 3) | (uint32_t)q, 0x7Eu);
  return sign | code;
}

__global__ __launch_bounds__(256) void k_row_scale(const uint16_t* __restrict__ W,
                                                   const uint16_t* __restrict__ W2, int N, int K,
                                                   int perm, float* __restrict__ scale) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  int which;
  const long src = packed_source_row(perm, row, N, which);
  const uint16_t* w = (which ? W2 : W) + src * K;
  float m = 0.f;
  for (int k = threadIdx.x; k < K; k += blockDim.x) m = fmaxf(m, fabsf(bf2f(w[k])));
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    const float a = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    scale[row] = a > 0.f ? __fdiv_rn(a, 448.f) : 1.f;
  }
}

__global__ void k_pack_fp8(const uint16_t* __restrict__ W, const uint16_t* __restrict__ W2, int N,
                           int K, int perm, const float* __restrict__ scale,
                           u32x4* __restrict__ out) {
  const int KT2 = K >> 6;
  const long total = (long)(N >> 4) * KT2 * 64;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const long f = i >> 6;
    const int kt2 = (int)(f % KT2);
    const long nt = f / KT2;
    const long prow = nt * 16 + (lane & 15);
    int which;
    const long row = packed_source_row(perm, prow, N, which);
    const uint16_t* w = (which ? W2 : W) + row * K + kt2 * 64 + (lane >> 4) * 8;
    const float s = scale[prow];
    uint32_t b[16];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      b[j] = e4m3_code(__fdiv_rn(bf2f(w[j]), s));
      b[8 + j] = e4m3_code(__fdiv_rn(bf2f(w[32 + j]), s));
    }
    u32x4 v;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      v[q] = b[4 * q] | (b[4 * q + 1] << 8) | (b[4 * q + 2] << 16) | (b[4 * q + 3] << 24);
    out[i] = v;
  }
}

hipError_t pack_fp8(const uint16_t* W, int N, int K, void* out, float* scale, hipStream_t st,
                    int perm, const uint16_t* W2) {
  if (N % 16 || K % 64) return hipErrorInvalidValue;
  if (perm == kPackRopePair && N % 128) return hipErrorInvalidValue;
  if (perm == kPackGateUp && !W2) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_row_scale, dim3(N), dim3(256), 0, st, W, W2, N, K, perm, scale);
  const long total = (long)(N / 16) * (K / 64) * 64;
  const int blocks = (int)std::min<long>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_pack_fp8, dim3(blocks), dim3(256), 0, st, W, W2, N, K, perm, scale,
                     (u32x4*)out);
  return hipGetLastError();
}

// 4 e4m3 codes -> 4 bf16 (2 words): hardware conversion to f32, which is exact,
// then the top 16 bits of each value.
__device__ __forceinline__ u32x2 bf16x4_of_fp8x4(uint32_t w) {
  const auto a = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, false);
  const auto b = __builtin_amdgcn_cvt_pk_f32_fp8((int)w, true);
  u32x2 r;
  r.x = (__float_as_uint(a[0]) >> 16) | (__float_as_uint(a[1]) & 0xFFFF0000u);
  r.y = (__float_as_uint(b[0]) >> 16) | (__float_as_uint(b[1]) & 0xFFFF0000u);
  return r;
}

// A packed fp8 fragment -> the bf16 A operands of its two K steps.
__device__ __forceinline__ void fp8_frag_to_bf16(const u32x4 raw, u32x4& k0, u32x4& k1) {
  const u32x2 p = bf16x4_of_fp8x4(raw.x), q = bf16x4_of_fp8x4(raw.y);
  const u32x2 r = bf16x4_of_fp8x4(raw.z), t = bf16x4_of_fp8x4(raw.w);
  k0 = u32x4{p.x, p.y, q.x, q.y};
  k1 = u32x4{r.x, r.y, t.x, t.y};
}

// ---- bf16 weight-streaming GEMM ----------------------------------------------------
// Workgroup = 4 waves; wave w owns NF 16-row weight groups (the workgroup
// covers 64*NF output features), all four waves walk the same K range.  The
// activation rows of the tile (16*MF rows) are staged through LDS in chunks
// of CK 32-wide K steps, so each activation fragment is fetched from L2 once
// per workgroup and read by all four waves; the next chunk is prefetched
// into registers while the current one is consumed.  Weights go straight
// from HBM to registers (non-temporal), U K steps ahead of the MFMAs.
// Grid = NB (weight groups / (4 NF)) x MT (row tiles) x S (K splits),
// remapped so that each XCD receives a contiguous range of tiles (the row
// tiles and splits of one weight group share an L2).
constexpr int kWaves = 4;

// With a start/stop event pair, the launch records them from its own dispatch
// (the kernel's execution time, as a kernel trace reports it).
template <typename F, typename... A>
static void launch_timed_block(F kernel, dim3 grid, dim3 block, hipStream_t st, hipEvent_t e0,
                               hipEvent_t e1, A... args) {
  if (e0)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
}

template <typename F, typename... A>
static void launch_timed(F kernel, dim3 grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                         A... args) {
  launch_timed_block(kernel, grid, dim3(256), st, e0, e1, args...);
}


// W8: fp8 weights (packed fp8 fragments, one per two K steps) with per-row
// scales wsc; the fp32 results are multiplied by the scale of their feature.
template <int NF, int MF, int U, int kCK, bool W8>
__global__ __launch_bounds__(256) void k_gemm_bf16(const uint16_t* __restrict__ X, int ldx,
                                                   const u32x4* __restrict__ Wp,
                                                   float* __restrict__ C, int M, int N, int K,
                                                   int NB, int MT, int S, int ks_per_split,
                                                   const float* __restrict__ wsc) {
  constexpr int ROWS = 16 * MF;
  constexpr int PITCH = kCK * 32 + 8;   // bf16 per LDS row; the 16-byte pad spreads banks
  constexpr int CHUNK16 = ROWS * kCK * 4;
  constexpr int PER_T = (CHUNK16 + 255) / 256;
  __shared__ __attribute__((aligned(16))) uint16_t xs[ROWS * PITCH];
  const int G = NB * MT * S;
  int id = blockIdx.x;
  if ((G & 7) == 0) id = (id & 7) * (G >> 3) + (id >> 3);
  const int mt = id % MT;
  const int rest = id / MT;
  const int nb = rest % NB;
  const int s = rest / NB;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int KT = K >> 5;
  const int kt0 = s * ks_per_split;
  const int kt1 = min(KT, kt0 + ks_per_split);
  const int m0 = mt * ROWS;
  const int f0 = (nb * kWaves + wave) * NF;
  const int frags = W8 ? KT / 2 : KT;  // packed fragments per 16-row group
  const u32x4* wp[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) wp[f] = Wp + ((long)(f0 + f) * frags) * 64 + lane;
  f32x4 acc[NF][MF];
#pragma unroll
  for (int a = 0; a < NF; ++a)
#pragma unroll
    for (int b = 0; b < MF; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const int nchunk = (kt1 - kt0 + kCK - 1) / kCK;
  u32x4 pre[PER_T];
  // chunk c of the tile's activations: rows m0.., K steps kt0 + c*kCK ..; rows >= M
  // and K steps >= kt1 read as zero
  auto gload = [&](int c) {
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int e = tid + i * 256;
      pre[i] = zero;
      if (e < CHUNK16) {
        const int r = e / (kCK * 4), cc = e % (kCK * 4);
        const int kt = kt0 + c * kCK + cc / 4;
        if (m0 + r < M && kt < kt1) pre[i] = *(const u32x4*)(X + (long)(m0 + r) * ldx + kt * 32 + (cc & 3) * 8);
      }
    }
  };
  auto lstore = [&](int c) {
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int e = tid + i * 256;
      if (e < CHUNK16) {
        const int r = e / (kCK * 4), cc = e % (kCK * 4);
        *(u32x4*)(&xs[r * PITCH + cc * 8]) = pre[i];
      }
    }
  };
  gload(0);
  lstore(0);
  __syncthreads();
  for (int c = 0; c < nchunk; ++c) {
    if (c + 1 < nchunk) gload(c + 1);
    const int kbase = kt0 + c * kCK;
    const int nk = min(kCK, kt1 - kbase);
    for (int k = 0; k < nk; k += U) {
      u32x4 a[U][NF];
      if constexpr (W8) {
        // K steps come in pairs (split and chunk starts are even)
        u32x4 raw[U / 2][NF];
#pragma unroll
        for (int u = 0; u < U; u += 2)
#pragma unroll
          for (int f = 0; f < NF; ++f)
            raw[u / 2][f] = (k + u < nk)
                                ? __builtin_nontemporal_load(wp[f] + (long)((kbase + k + u) >> 1) * 64)
                                : zero;
#pragma unroll
        for (int u = 0; u < U; u += 2)
#pragma unroll
          for (int f = 0; f < NF; ++f) fp8_frag_to_bf16(raw[u / 2][f], a[u][f], a[u + 1][f]);
      } else {
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
          for (int f = 0; f < NF; ++f)
            a[u][f] = (k + u < nk) ? __builtin_nontemporal_load(wp[f] + (long)(kbase + k + u) * 64) : zero;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        u32x4 b[MF];
#pragma unroll
        for (int f = 0; f < MF; ++f)
          b[f] = *(const u32x4*)(&xs[(f * 16 + (lane & 15)) * PITCH + (k + u) * 32 + (lane >> 4) * 8]);
#pragma unroll
        for (int i = 0; i < NF; ++i)
#pragma unroll
          for (int j = 0; j < MF; ++j) acc[i][j] = mfma16(a[u][i], b[j], acc[i][j]);
      }
    }
    if (c + 1 < nchunk) {
      __syncthreads();
      lstore(c + 1);
      __syncthreads();
    }
  }
#pragma unroll
  for (int i = 0; i < NF; ++i) {
    const int n0 = (f0 + i) * 16 + (lane >> 4) * 4;
    const f32x4 sc = W8 ? *(const f32x4*)(wsc + n0) : f32x4{1.f, 1.f, 1.f, 1.f};
#pragma unroll
    for (int j = 0; j < MF; ++j) {
      const int m = m0 + j * 16 + (lane & 15);
      if (m < M) *(f32x4*)(C + ((long)s * M + m) * N + n0) = W8 ? acc[i][j] * sc : acc[i][j];
    }
  }
}


// ---- few-row GEMM with its epilogue, no K split ----------------------------------------
// For the wide products of a normal step (Q/K/V, gate/up, LM head) the whole
// K range of a tile of GW 16-feature weight groups is one workgroup (one wave
// per group), so its sums are final and the epilogue runs in the kernel: no
// split-K partials and no epilogue launch.  Activations are staged through
// LDS and shared by the waves.  Every iteration waits on loads issued several
// iterations earlier: the weights of iteration it + 3 are loaded while it is
// computed (a ring of four register buffers), the activations of it + 2 go to
// registers and those of it + 1 to the other half of a double-buffered LDS
// tile, so neither stream pays a full memory round trip per iteration.
// Loads read clamped addresses, so they are never predicated; K steps past
// the end are zeroed when stored to LDS and their products add nothing.
//
// EPI == kEpiQkv: weights packed kPackRopePair.  Adds the bias, rotates q/k
// heads (RoPE pairs meet in lanes l and l ^ 32), rounds to T, stores q rows and
// scatters k/v rows into the cache at row_tok.
// EPI == kEpiSwiGlu: weights packed kPackGateUp.  out[m][f] = silu(g) * u.
// EPI == kEpiConf (LM head): reduces the tile's 64 vocabulary entries of each
// row to (max logit, lowest id reaching it, sum exp(l - max)), [MASK]
// excluded, into pmax / pidx / psum[m][tile]; writes the logits themselves
// only when ep.logits is set.
struct FusedEpi {
  // Q/K/V
  const uint16_t* bias;     // [(nh + 2 nkv) * 128] or null
  const float* rope_cs;     // [pos][64][cos, sin]
  const int32_t* row_pos;
  const int32_t* row_tok;
  int nh, nkv;
  uint16_t *q, *kc, *vc;
  long cache_rows;
  // SwiGLU
  uint16_t* out;
  int F;
  // LM head + confidence
  int mask_id, n_tiles;
  float* logits;            // [M][V] fp32, or null
  float *pmax, *psum;       // [M][n_tiles]
  int* pidx;
  // K-split partials: split s of `splits` covers K steps [s ks, s ks + ks)
  float* C;                 // [splits][M][N] fp32
  int splits, ks;
};

template <int V>
using ic = std::integral_constant<int, V>;

// f(ic<I>{}), f(ic<I + 1>{}), ..., f(ic<N - 1>{})
template <int I, int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(ic<I>{});
    static_for<I + 1, N>(f);
  }
}

// R: depth of the weight ring (loads run R - 1 iterations ahead); XD: the
// activations are loaded XD iterations ahead and staged in LDS one ahead.
template <int EPI, int MF, int U, bool W8, int GW, int R, int XD>
__global__ __launch_bounds__(64 * GW) void k_gemm_bf16_fused(const uint16_t* __restrict__ X, int ldx,
                                                             const u32x4* __restrict__ Wp, int M,
                                                             int N, int K, FusedEpi ep,
                                                             const float* __restrict__ wsc) {
  static_assert(EPI != kEpiConf || GW == kWaves, "the confidence epilogue reduces 64-entry tiles");
  static_assert(R % XD == 0 && XD % 2 == 0, "ring slots and activation buffers repeat together");
  constexpr int NT = 64 * GW;
  constexpr int ROWS = 16 * MF;
  constexpr int PITCH = U * 32 + 8;
  constexpr int CHUNK16 = ROWS * U * 4;
  constexpr int PER_T = (CHUNK16 + NT - 1) / NT;
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][ROWS * PITCH];
  const int G = gridDim.x;
  int id = blockIdx.x;
  if ((G & 7) == 0) id = (id & 7) * (G >> 3) + (id >> 3);
  // with a K split, workgroup id takes group block id % nblk over split id / nblk
  const int nblk = EPI == kEpiPartial ? G / ep.splits : G;
  const int nb = id % nblk, sp = id / nblk;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int KT = K >> 5;
  const int kt_begin = EPI == kEpiPartial ? sp * ep.ks : 0;
  const int KTs = EPI == kEpiPartial ? min(KT, kt_begin + ep.ks) - kt_begin : KT;  // this split's
  const int grp = nb * GW + wave;  // this wave's 16-row weight group
  // without a K split the last workgroup may hold fewer than GW groups: its
  // spare waves stream the last group again (every wave takes part in the
  // loop's barriers) and store nothing
  const int ngroups = N >> 4;
  const bool live = grp < ngroups;
  const int grp_ld = min(grp, ngroups - 1);
  // W8: the ring holds raw fp8 fragments (one per two K steps), decoded when used
  constexpr int UW = W8 ? U / 2 : U;
  const int frags = W8 ? KTs / 2 : KTs;
  const u32x4* wp =
      Wp + ((long)grp_ld * (W8 ? KT / 2 : KT) + (W8 ? kt_begin / 2 : kt_begin)) * 64 + lane;
  f32x4 acc[MF];
#pragma unroll
  for (int b = 0; b < MF; ++b) acc[b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const int n_it = (KTs + U - 1) / U;
  u32x4 pre[XD][PER_T];
  u32x4 a[R][UW];
  // EV (the split's K steps a multiple of U, as at every shipped shape): one
  // clamped iteration index per load group, the per-thread activation offsets
  // computed once, and no zero masks when staging (rows past M repeat row
  // M - 1, whose products are never stored).  Otherwise every load clamps its
  // own K step and the staging zeroes rows past M and K steps past the end.
  // Both give the same sums.
  const u32x4* xrow[PER_T];
#pragma unroll
  for (int i = 0; i < PER_T; ++i) {
    const int e = min(tid + i * NT, CHUNK16 - 1);
    const int r = e / (U * 4), cc = e % (U * 4);
    xrow[i] = (const u32x4*)(X + (long)min(r, M - 1) * ldx + (kt_begin + cc / 4) * 32 + (cc & 3) * 8);
  }
  auto wload = [&](auto B, int it, auto EV) {
    constexpr int b = decltype(B)::value;
    if constexpr (decltype(EV)::value) {
      const u32x4* base = wp + (long)min(it, n_it - 1) * (UW * 64);
#pragma unroll
      for (int u = 0; u < UW; ++u) a[b][u] = __builtin_nontemporal_load(base + u * 64);
    } else {
#pragma unroll
      for (int u = 0; u < UW; ++u)
        a[b][u] = __builtin_nontemporal_load(wp + (long)min(it * UW + u, frags - 1) * 64);
    }
  };
  auto xload = [&](auto P, int it, auto EV) {
    constexpr int p = decltype(P)::value;
    if constexpr (decltype(EV)::value) {
      const long step = (long)min(it, n_it - 1) * (U * 4);  // u32x4 per iteration of a row
#pragma unroll
      for (int i = 0; i < PER_T; ++i) pre[p][i] = xrow[i][step];
    } else {
#pragma unroll
      for (int i = 0; i < PER_T; ++i) {
        const int e = min(tid + i * NT, CHUNK16 - 1);
        const int r = e / (U * 4), cc = e % (U * 4);
        const long row = min(r, M - 1);
        const int kc = kt_begin + min(it * U + cc / 4, KTs - 1);
        pre[p][i] = *(const u32x4*)(X + row * ldx + kc * 32 + (cc & 3) * 8);
      }
    }
  };
  auto xstore = [&](auto P, int buf, int it, auto EV) {
    constexpr int p = decltype(P)::value;
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int e = tid + i * NT;
      if (CHUNK16 % NT == 0 || e < CHUNK16) {
        const int r = e / (U * 4), cc = e % (U * 4);
        if constexpr (decltype(EV)::value) {
          *(u32x4*)(&xs[buf][r * PITCH + cc * 8]) = pre[p][i];
        } else {
          const bool ok = r < M && it * U + cc / 4 < KTs;
          *(u32x4*)(&xs[buf][r * PITCH + cc * 8]) = ok ? pre[p][i] : zero;
        }
      }
    }
  };
  auto compute = [&](auto B, int buf) {
    constexpr int bsel = decltype(B)::value;
    const uint16_t* xb = xs[buf];
    constexpr int PAIR = W8 ? 2 : 1;  // K steps per weight register of the ring
#pragma unroll
    for (int uw = 0; uw < UW; ++uw) {
      u32x4 w[PAIR];
      if constexpr (W8)
        fp8_frag_to_bf16(a[bsel][uw], w[0], w[1]);
      else
        w[0] = a[bsel][uw];
#pragma unroll
      for (int h = 0; h < PAIR; ++h) {
        const int u = uw * PAIR + h;
        u32x4 b[MF];
#pragma unroll
        for (int j = 0; j < MF; ++j)
          b[j] = *(const u32x4*)(&xb[(j * 16 + (lane & 15)) * PITCH + u * 32 + (lane >> 4) * 8]);
#pragma unroll
        for (int j = 0; j < MF; ++j) acc[j] = mfma16(w[h], b[j], acc[j]);
      }
    }
  };
  // iteration it = base + J with base a multiple of R (and of XD): buffers are static
  auto body = [&](auto J, int it, auto EV) {
    constexpr int j = decltype(J)::value;
    xload(ic<j % XD>{}, it + XD, EV);
    wload(ic<(j + R - 1) % R>{}, it + R - 1, EV);
    if (it < n_it) compute(ic<j % R>{}, j & 1);
    xstore(ic<(j + 1) % XD>{}, (j + 1) & 1, it + 1, EV);
    __syncthreads();
  };
  // Q/K/V epilogue inputs, loaded before the K loop so that their latency
  // (the cos/sin address depends on the row's position) hides behind it
  [[maybe_unused]] float qkv_bias[4];
  [[maybe_unused]] f32x4 qkv_cs[MF][2];
  [[maybe_unused]] int qkv_tok[MF];
  if constexpr (EPI == kEpiQkv) {
    const int head = grp_ld >> 3, i0 = (grp_ld & 7) * 8 + ((lane >> 4) & 1) * 4;
    const int dim0 = (lane >> 5) * 64 + i0;
#pragma unroll
    for (int j = 0; j < 4; ++j) qkv_bias[j] = ep.bias ? bf2f(ep.bias[head * 128 + dim0 + j]) : 0.f;
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) {
      const int m = min(jf * 16 + (lane & 15), M - 1);
      qkv_tok[jf] = ep.row_tok[m];
      const f32x4* cs = (const f32x4*)(ep.rope_cs + ((long)ep.row_pos[m] * 64 + i0) * 2);
      qkv_cs[jf][0] = cs[0];
      qkv_cs[jf][1] = cs[1];
    }
  }
  auto run = [&](auto EV) {
    static_for<0, XD>([&](auto J) { xload(J, decltype(J)::value, EV); });
    static_for<0, R - 1>([&](auto J) { wload(J, decltype(J)::value, EV); });
    xstore(ic<0>{}, 0, 0, EV);
    __syncthreads();
    for (int it = 0; it < n_it; it += R)
      static_for<0, R>([&](auto J) { body(J, it + decltype(J)::value, EV); });
  };
  if (KTs % U == 0)  // uniform over the grid
    run(std::true_type{});
  else
    run(std::false_type{});

  // the confidence epilogue has barriers; its launches divide the groups evenly
  if constexpr (EPI != kEpiConf)
    if (!live) return;
  // lane l holds packed rows grp*16 + (l/16)*4 + j (j < 4) of activation rows
  // j*16 + l%16; packed rows 0..7 of a group pair with rows 8..15 (lane l ^ 32)
  const int hi = lane >> 5;               // 0: rows 0..7 of the group, 1: rows 8..15
  const int sub = ((lane >> 4) & 1) * 4;  // first of this lane's 4 rows within its half
  if constexpr (W8) {
    const f32x4 sc = *(const f32x4*)(wsc + grp * 16 + (lane >> 4) * 4);
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) acc[jf] *= sc;
  }
  if constexpr (EPI == kEpiQkv) {
    const int head = grp >> 3, gi = grp & 7;
    const int i0 = gi * 8 + sub;          // rotation index of j = 0 (< 64)
    const int dim0 = hi * 64 + i0;        // this lane's dims dim0 .. dim0 + 3
    const bool rot = head < ep.nh + ep.nkv;
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) {
      float x[4], p[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = acc[jf][j] + qkv_bias[j];
        p[j] = __shfl_xor(x[j], 32, 64);
      }
      const int m = jf * 16 + (lane & 15);
      if (m >= M) continue;
      if (rot) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const float c = qkv_cs[jf][j >> 1][(j & 1) * 2], sn = qkv_cs[jf][j >> 1][(j & 1) * 2 + 1];
          x[j] = hi ? x[j] * c + p[j] * sn : x[j] * c - p[j] * sn;
        }
      }
      uint16_t* dst;
      if (head < ep.nh)
        dst = ep.q + ((long)m * ep.nh + head) * 128;
      else if (head < ep.nh + ep.nkv)
        dst = ep.kc + ((long)(head - ep.nh) * ep.cache_rows + qkv_tok[jf]) * 128;
      else
        dst = ep.vc + ((long)(head - ep.nh - ep.nkv) * ep.cache_rows + qkv_tok[jf]) * 128;
      u32x2 w;
      w.x = (uint32_t)f2bf(x[0]) | ((uint32_t)f2bf(x[1]) << 16);
      w.y = (uint32_t)f2bf(x[2]) | ((uint32_t)f2bf(x[3]) << 16);
      *(u32x2*)(dst + dim0) = w;
    }
  } else if constexpr (EPI == kEpiPartial) {
    // lane: features grp * 16 + (lane / 16) * 4 .. + 3 of rows jf * 16 + lane % 16
    const int n0 = grp * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) {
      const int m = jf * 16 + (lane & 15);
      if (m < M) *(f32x4*)(ep.C + ((long)sp * M + m) * N + n0) = acc[jf];
    }
  } else if constexpr (EPI == kEpiConf) {
    // lane: vocabulary ids v0 .. v0 + 3 of rows jf * 16 + lane % 16
    __shared__ float cm[kWaves][16 * MF], cs[kWaves][16 * MF];
    __shared__ int ci[kWaves][16 * MF];
    const int v0 = grp * 16 + (lane >> 4) * 4;
    const int N4 = N;
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) {
      const int m = jf * 16 + (lane & 15);
      if (ep.logits && m < M) *(f32x4*)(ep.logits + (long)m * N4 + v0) = acc[jf];
      float bm = -INFINITY;
      int bi = INT_MAX;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        if (v0 + j != ep.mask_id && acc[jf][j] > bm) {
          bm = acc[jf][j];
          bi = v0 + j;
        }
#pragma unroll
      for (int o = 16; o < 64; o <<= 1) {
        const float om = __shfl_xor(bm, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (om > bm || (om == bm && oi < bi)) {
          bm = om;
          bi = oi;
        }
      }
      if (lane < 16) {
        cm[wave][jf * 16 + lane] = bm;
        ci[wave][jf * 16 + lane] = bi;
      }
    }
    __syncthreads();
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) {
      const int r = jf * 16 + (lane & 15);
      float mx = cm[0][r];
#pragma unroll
      for (int w = 1; w < kWaves; ++w) mx = fmaxf(mx, cm[w][r]);
      float sum = 0.f;
      if (mx > -INFINITY)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (v0 + j != ep.mask_id) sum += expf(acc[jf][j] - mx);
      sum += __shfl_xor(sum, 16, 64);
      sum += __shfl_xor(sum, 32, 64);
      if (lane < 16) cs[wave][r] = sum;
    }
    __syncthreads();
    if (tid < 16 * MF && tid < M) {
      const int r = tid;
      float bm = cm[0][r];
      int bi = ci[0][r];
#pragma unroll
      for (int w = 1; w < kWaves; ++w)
        if (cm[w][r] > bm || (cm[w][r] == bm && ci[w][r] < bi)) {
          bm = cm[w][r];
          bi = ci[w][r];
        }
      const long o = (long)r * ep.n_tiles + nb;
      ep.pmax[o] = bm;
      ep.pidx[o] = bi;
      ep.psum[o] = cs[0][r] + cs[1][r] + cs[2][r] + cs[3][r];
    }
  } else {
    const int f0 = grp * 8 + sub;         // this lane's features f0 .. f0 + 3
#pragma unroll
    for (int jf = 0; jf < MF; ++jf) {
      float x[4], p[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = acc[jf][j];
        p[j] = __shfl_xor(x[j], 32, 64);
      }
      const int m = jf * 16 + (lane & 15);
      if (hi || m >= M) continue;
      u32x2 w;
      float y[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) y[j] = x[j] / (1.0f + expf(-x[j])) * p[j];
      w.x = (uint32_t)f2bf(y[0]) | ((uint32_t)f2bf(y[1]) << 16);
      w.y = (uint32_t)f2bf(y[2]) | ((uint32_t)f2bf(y[3]) << 16);
      *(u32x2*)(ep.out + (long)m * ep.F + f0) = w;
    }
  }
}

bool fused_rows_ok(int M, int N, int K, int max_rows) {
  return M >= 1 && M <= max_rows && max_rows <= 96 && N % 64 == 0 && K % 32 == 0 && N / 64 >= 192;
}

template <int EPI, int U, bool W8, int GW, int R, int XD = 2>
static void launch_fused_mf(dim3 grid, int M, const uint16_t* X, int ldx, const u32x4* W, int N,
                            int K, const FusedEpi& ep, const float* wsc, hipStream_t st,
                            hipEvent_t e0, hipEvent_t e1) {
  const dim3 block(64 * GW);
  // 65 to 96 rows (gate/up, O and down only): activations two iterations ahead,
  // which keeps the larger staging within the register file
  switch ((M + 15) / 16) {
    case 1: launch_timed_block(k_gemm_bf16_fused<EPI, 1, U, W8, GW, R, XD>, grid, block, st, e0, e1, X, ldx, W, M, N, K, ep, wsc); break;
    case 2: launch_timed_block(k_gemm_bf16_fused<EPI, 2, U, W8, GW, R, XD>, grid, block, st, e0, e1, X, ldx, W, M, N, K, ep, wsc); break;
    case 3: launch_timed_block(k_gemm_bf16_fused<EPI, 3, U, W8, GW, R, XD>, grid, block, st, e0, e1, X, ldx, W, M, N, K, ep, wsc); break;
    case 4: launch_timed_block(k_gemm_bf16_fused<EPI, 4, U, W8, GW, R, XD>, grid, block, st, e0, e1, X, ldx, W, M, N, K, ep, wsc); break;
    case 5:
      if constexpr (EPI == kEpiSwiGlu || EPI == kEpiPartial)
        launch_timed_block(k_gemm_bf16_fused<EPI, 5, U, W8, GW, R, 2>, grid, block, st, e0, e1, X, ldx, W, M, N, K, ep, wsc);
      break;
    default:
      if constexpr (EPI == kEpiSwiGlu || EPI == kEpiPartial)
        launch_timed_block(k_gemm_bf16_fused<EPI, 6, U, W8, GW, R, 2>, grid, block, st, e0, e1, X, ldx, W, M, N, K, ep, wsc);
      break;
  }
}

// GW weight groups (16 features each) per workgroup, one wave each.  A wave
// streams at a bounded rate (its loop is latency-bound), so a launch is
// fastest when its workgroups fill the 256 CUs in as few rounds as possible:
// the least rounds x GW, ties to more groups per workgroup (every workgroup
// stages all activation rows).  Two groups only when that is still one
// round.  GW need not divide the groups: the last workgroup's spare waves
// store nothing.  Measured (33-39 rows): Q/K/V 4096 x 12288 20.1 us with GW 3
// against 21.2 with GW 4; 3584 x 4608 15.5 with GW 2 against 17.1; gate/up
// 4096 x 24576 33.7 with GW 6 against 38.9 with GW 4.  The LM head's
// confidence epilogue needs GW 4.
static int fused_groups_per_wg(int groups) {
  int best = 4;
  long best_key = LONG_MAX;
  for (int gw : {10, 8, 6, 4, 3, 2}) {
    const long wgs = (groups + gw - 1) / gw, rounds = (wgs + 255) / 256;
    if (gw == 2 && rounds > 1) continue;
    const long key = rounds * gw * 16 + (16 - gw);
    if (key < best_key) {
      best_key = key;
      best = gw;
    }
  }
  return best;
}

template <int EPI, int U, bool W8>
static void launch_fused_gw(int gw, const uint16_t* X, int ldx, const u32x4* W, int M, int N,
                            int K, const FusedEpi& ep, const float* wsc, hipStream_t st,
                            hipEvent_t e0, hipEvent_t e1) {
  const dim3 grid((N / 16 + gw - 1) / gw);
  if constexpr (EPI == kEpiConf) {
    launch_fused_mf<EPI, U, W8, 4, 4, 2>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1);
  } else {
    switch (gw) {
      case 10: launch_fused_mf<EPI, U, W8, 10, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1); break;
      case 8: launch_fused_mf<EPI, U, W8, 8, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1); break;
      case 6: launch_fused_mf<EPI, U, W8, 6, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1); break;
      case 3: launch_fused_mf<EPI, U, W8, 3, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1); break;
      case 2: launch_fused_mf<EPI, U, W8, 2, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1); break;
      default: launch_fused_mf<EPI, U, W8, 4, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, e0, e1); break;
    }
  }
}

template <int EPI, int U>
static hipError_t launch_fused(const uint16_t* X, int ldx, const void* Wp, int M, int N, int K,
                               const FusedEpi& ep, const float* wsc, hipStream_t st, hipEvent_t e0,
                               hipEvent_t e1) {
  if (!fused_rows_ok(M, N, K, fused_max_rows(EPI)) || (wsc && K % 64)) return hipErrorInvalidValue;
  const u32x4* W = (const u32x4*)Wp;
  const int gw = EPI == kEpiConf ? 4 : fused_groups_per_wg(N / 16);
  if (EPI == kEpiConf && (N / 16) % gw) return hipErrorInvalidValue;
  if (wsc)
    launch_fused_gw<EPI, U, true>(gw, X, ldx, W, M, N, K, ep, wsc, st, e0, e1);
  else
    launch_fused_gw<EPI, U, false>(gw, X, ldx, W, M, N, K, ep, wsc, st, e0, e1);
  return hipGetLastError();
}

hipError_t gemm_bf16_qkv_fused(const uint16_t* X, int ldx, const void* Wp, int M, int N, int K,
                               const uint16_t* bias, const float* rope_cs, const int32_t* row_pos,
                               const int32_t* row_tok, int nh, int nkv, uint16_t* q, uint16_t* kc,
                               uint16_t* vc, long cache_rows, hipStream_t st, hipEvent_t e0,
                               hipEvent_t e1, const float* wsc) {
  if (N != (nh + 2 * nkv) * 128) return hipErrorInvalidValue;
  FusedEpi ep{};
  ep.bias = bias;
  ep.rope_cs = rope_cs;
  ep.row_pos = row_pos;
  ep.row_tok = row_tok;
  ep.nh = nh;
  ep.nkv = nkv;
  ep.q = q;
  ep.kc = kc;
  ep.vc = vc;
  ep.cache_rows = cache_rows;
  return launch_fused<kEpiQkv, 4>(X, ldx, Wp, M, N, K, ep, wsc, st, e0, e1);
}

hipError_t gemm_bf16_lmhead_conf(const uint16_t* X, int ldx, const void* Wp, int M, int V, int K,
                                 int mask_id, float* logits, float* pmax, int* pidx, float* psum,
                                 hipStream_t st, hipEvent_t e0, hipEvent_t e1, const float* wsc) {
  FusedEpi ep{};
  ep.mask_id = mask_id;
  ep.n_tiles = V / 64;
  ep.logits = logits;
  ep.pmax = pmax;
  ep.pidx = pidx;
  ep.psum = psum;
  return launch_fused<kEpiConf, 4>(X, ldx, Wp, M, V, K, ep, wsc, st, e0, e1);
}

hipError_t gemm_bf16_swiglu_fused(const uint16_t* X, int ldx, const void* Wp, int M, int F, int K,
                                  uint16_t* out, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                                  const float* wsc) {
  FusedEpi ep{};
  ep.out = out;
  ep.F = F;
  return launch_fused<kEpiSwiGlu, 4>(X, ldx, Wp, M, 2 * F, K, ep, wsc, st, e0, e1);
}

hipError_t gemm_bf16_split_fused(const uint16_t* X, int ldx, const void* Wp, float* C, int M,
                                 int N, int K, int gw, int splits, int ks, hipStream_t st,
                                 hipEvent_t e0, hipEvent_t e1, const float* wsc) {
  const int KT = K / 32;
  if (M < 1 || M > 96 || N % 16 || K % 32 || ks <= 0 || splits <= 0 ||
      (long)splits * ks < KT || (long)(splits - 1) * ks >= KT || (N / 16) % gw ||
      (wsc && (K % 64 || ks % 2)))
    return hipErrorInvalidValue;
  FusedEpi ep{};
  ep.C = C;
  ep.splits = splits;
  ep.ks = ks;
  const dim3 grid(N / 16 / gw * splits);
  const u32x4* W = (const u32x4*)Wp;
#define WD_SPLIT_GW(GWV)                                                                       \
  case GWV:                                                                                    \
    if (wsc)                                                                                   \
      launch_fused_mf<kEpiPartial, 4, true, GWV, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st,  \
                                                       e0, e1);                                \
    else                                                                                       \
      launch_fused_mf<kEpiPartial, 4, false, GWV, 4, 4>(grid, M, X, ldx, W, N, K, ep, wsc, st, \
                                                        e0, e1);                               \
    break;
  switch (gw) {
    WD_SPLIT_GW(2)
    WD_SPLIT_GW(3)
    WD_SPLIT_GW(4)
    WD_SPLIT_GW(6)
    WD_SPLIT_GW(7)
    default: return hipErrorInvalidValue;
  }
#undef WD_SPLIT_GW
  return hipGetLastError();
}

// ---- bf16 GEMM for many rows (refresh steps, the full-sequence path, batches) ----------
// Same operands and tile order as above, with 128-row activation tiles and
// NF weight groups per wave (16*NF*8 MFMAs per 4 K steps).  With few waves per
// CU, load latency must be covered by loads in flight: weights are fetched
// two iterations (8 K steps) ahead through a ring of three register buffers,
// the next activation chunk one iteration ahead into the other half of a
// double-buffered LDS tile; one barrier per iteration.
template <int NF, bool W8>
__global__ __launch_bounds__(256, 2) void k_gemm_bf16_big(const uint16_t* __restrict__ X, int ldx,
                                                          const u32x4* __restrict__ Wp,
                                                          float* __restrict__ C, int M, int N,
                                                          int K, int NB, int MT, int S,
                                                          int ks_per_split,
                                                          const float* __restrict__ wsc) {
  constexpr int MF = 8, U = 4;
  constexpr int ROWS = 16 * MF;
  constexpr int PITCH = U * 32 + 8;
  constexpr int CHUNK16 = ROWS * U * 4;
  constexpr int PER_T = CHUNK16 / 256;
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][ROWS * PITCH];
  const int G = NB * MT * S;
  int id = blockIdx.x;
  if ((G & 7) == 0) id = (id & 7) * (G >> 3) + (id >> 3);
  const int mt = id % MT;
  const int rest = id / MT;
  const int nb = rest % NB;
  const int s = rest / NB;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int KT = K >> 5;
  const int kt0 = s * ks_per_split;
  const int kt1 = min(KT, kt0 + ks_per_split);
  const int m0 = mt * ROWS;
  const int f0 = (nb * kWaves + wave) * NF;
  // W8: the ring holds raw fp8 fragments (one per two K steps), decoded when used
  constexpr int UW = W8 ? U / 2 : U;
  const int frags = W8 ? KT / 2 : KT;
  const u32x4* wp[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) wp[f] = Wp + ((long)(f0 + f) * frags) * 64 + lane;
  f32x4 acc[NF][MF];
#pragma unroll
  for (int a = 0; a < NF; ++a)
#pragma unroll
    for (int b = 0; b < MF; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};
  const u32x4 zero = {0u, 0u, 0u, 0u};
  const int n_it = (kt1 - kt0 + U - 1) / U;
  u32x4 pre[PER_T];
  u32x4 a0[UW][NF], a1[UW][NF], a2[UW][NF];

  // Loads are branch-free and never waited on early: an out-of-range K step
  // reads the weights of the last valid step (finite values, multiplied by
  // the zero activations stored for that step), and out-of-range activation
  // elements read a clamped address and are zeroed only when they are
  // stored to LDS.
  auto wload = [&](u32x4 (&a)[UW][NF], int it) {
    const int kb = kt0 + it * U;
#pragma unroll
    for (int u = 0; u < UW; ++u) {
      // W8: split starts and U are even, so fragment (kb + 2u) / 2 holds steps kb + 2u, + 1
      const int kk = W8 ? min((kb >> 1) + u, (kt1 >> 1) - 1) : min(kb + u, kt1 - 1);
#pragma unroll
      for (int f = 0; f < NF; ++f) a[u][f] = __builtin_nontemporal_load(wp[f] + (long)kk * 64);
    }
  };
  auto xload = [&](int it) {
    const int kb = kt0 + it * U;
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int e = tid + i * 256;
      const int r = e / (U * 4), cc = e % (U * 4);
      const long row = min(m0 + r, M - 1);
      const int kc = min(kb + cc / 4, kt1 - 1);
      pre[i] = *(const u32x4*)(X + row * ldx + kc * 32 + (cc & 3) * 8);
    }
  };
  auto xstore = [&](int buf, int it) {
    const int kb = kt0 + it * U;
#pragma unroll
    for (int i = 0; i < PER_T; ++i) {
      const int e = tid + i * 256;
      const int r = e / (U * 4), cc = e % (U * 4);
      const bool ok = m0 + r < M && kb + cc / 4 < kt1;
      *(u32x4*)(&xs[buf][r * PITCH + cc * 8]) = ok ? pre[i] : zero;
    }
  };
  auto compute = [&](const u32x4 (&a)[UW][NF], int buf) {
    const uint16_t* xb = xs[buf];
    constexpr int PAIR = W8 ? 2 : 1;
#pragma unroll
    for (int uw = 0; uw < UW; ++uw) {
      u32x4 w[PAIR][NF];
#pragma unroll
      for (int i = 0; i < NF; ++i) {
        if constexpr (W8)
          fp8_frag_to_bf16(a[uw][i], w[0][i], w[1][i]);
        else
          w[0][i] = a[uw][i];
      }
#pragma unroll
      for (int h = 0; h < PAIR; ++h) {
        const int u = uw * PAIR + h;
        u32x4 b[MF];
#pragma unroll
        for (int j = 0; j < MF; ++j)
          b[j] = *(const u32x4*)(&xb[(j * 16 + (lane & 15)) * PITCH + u * 32 + (lane >> 4) * 8]);
#pragma unroll
        for (int j = 0; j < MF; ++j)
#pragma unroll
          for (int i = 0; i < NF; ++i) acc[i][j] = mfma16(w[h][i], b[j], acc[i][j]);
      }
    }
  };
  // iteration it: weights of it come from `cur`, weights of it + 2 go to `ld`
  // The activation loads go first: the load counter is in order, so waiting
  // for them before the LDS store must not also wait for the weight prefetch.
  auto body = [&](u32x4 (&cur)[UW][NF], u32x4 (&ld)[UW][NF], int it) {
    const bool more = it + 1 < n_it;
    if (more) xload(it + 1);
    if (it + 2 < n_it) wload(ld, it + 2);
    compute(cur, it & 1);
    if (more) xstore((it + 1) & 1, it + 1);
    __syncthreads();
  };

  xload(0);
  wload(a0, 0);
  if (n_it > 1) wload(a1, 1);
  xstore(0, 0);
  __syncthreads();
  for (int it = 0; it < n_it; it += 3) {
    body(a0, a2, it);
    if (it + 1 < n_it) body(a1, a0, it + 1);
    if (it + 2 < n_it) body(a2, a1, it + 2);
  }
#pragma unroll
  for (int i = 0; i < NF; ++i) {
    const int n0 = (f0 + i) * 16 + (lane >> 4) * 4;
    const f32x4 sc = W8 ? *(const f32x4*)(wsc + n0) : f32x4{1.f, 1.f, 1.f, 1.f};
#pragma unroll
    for (int j = 0; j < MF; ++j) {
      const int m = m0 + j * 16 + (lane & 15);
      if (m < M) *(f32x4*)(C + ((long)s * M + m) * N + n0) = W8 ? acc[i][j] * sc : acc[i][j];
    }
  }
}

// Launch shape, from the measured behaviour of the kernel on MI355X.
// Up to 64 rows (normal steps, weight-streaming bound): one row tile of
// 16*MF rows; wide matrices (N >= 16384) stream best with 2 weight groups
// per wave and as few K splits as give >= 384 workgroups, narrower ones with
// 1 group per wave and >= 512 workgroups.  Above 64 rows (refresh steps, the
// full-sequence path, batches): 128-row tiles, 2 weight groups per wave,
// software-pipelined, K splits until 256 workgroups run (split-K partials
// cost rows*N*4 bytes each).


GemmPlan plan_gemm_bf16(int M, int N, int K, bool w8, int max_splits) {
  GemmPlan p;
  const int KT = K / 32;
  if (M <= 96 && !w8 && (K >= N || (N / 64 < 192 && M <= 64)) && N % 64 == 0) {
    // K at least N (O, down): the pipelined kernel with partials, 4 groups
    // per workgroup and the most power-of-two splits that keep one round of
    // workgroups, each split at least 16 K steps (measured with weights read
    // from HBM, 33-39 rows: 4096 x 12288 18.5 us against 19.5 for the kernel
    // below, 18944 x 3584 25.5 against 26.3, 4096 x 4096 9.2 against 9.2
    // with 4 splits instead of 8, which halves what the residual norm reads)
    // Up to 96 rows: at 66-94 rows (weights from HBM) O takes 11.0-12.4 us and
    // down 23.1-25.8 against 14.6-15.4 and 30.2-33.8 on 128-row tiles.
    // Where 4 groups per workgroup cannot fill the CUs (Dream-7B's 3584-wide
    // O and down: 224 workgroups), 7 groups with twice the splits may: the
    // fullest one-round grid wins, ties to fewer splits.
    // Products too narrow for the fused kernel (N / 64 < 192) take this one
    // too up to 64 rows, whatever K: Dream-7B's Q/K/V (4608 x 3584) with 3 groups per
    // workgroup and 2 splits runs 10.2-10.8 us against 10.3-10.9 for the
    // kernel below with 8 splits, and the Q/K/V epilogue reads 2 partials
    // instead of 8.
    const int groups = N / 16;
    int best_gw = 4, best_S = 1;
    long best_grid = -1;
    for (int gw : {4, 7, 3}) {
      if (groups % gw) continue;
      int S = 1;
      while (2 * S <= max_splits && (long)(groups / gw) * 2 * S <= 256 && KT / (2 * S) >= 16) S *= 2;
      const long grid = (long)(groups / gw) * S;
      if (grid > best_grid || (grid == best_grid && S < best_S)) {
        best_grid = grid;
        best_gw = gw;
        best_S = S;
      }
    }
    p.fused_gw = best_gw;
    p.ks_per_split = (KT + best_S - 1) / best_S;
    p.splits = (KT + p.ks_per_split - 1) / p.ks_per_split;
    p.grid = groups / best_gw * p.splits;
    p.mf = (M + 15) / 16;
    return p;
  }
  if (M > 64 && !w8 && N % 256 == 0) {
    // k_gemm_bf16_dma: 64 * mfw-row x (32 * tnb)-feature tiles, S K splits.
    // Measured on the projection shapes (224 to 600 rows): a grid that fits
    // one round of one workgroup per CU (128 to 256 workgroups) beats more,
    // smaller workgroups, and partials cost their epilogue a read each.  So: a
    // one-round grid if there is one, else no K split if the tiles alone give
    // 256 workgroups; then least work per CU (rounds x rows x features x K
    // steps), at least 32 K steps per split, taller tiles, fewer splits, wider
    // tiles.  192-feature tiles (N a multiple of 192 too) fill all 256 CUs
    // where 256-feature ones leave a quarter idle (weights from HBM): Q/K/V
    // 12288 x 4096 at 66-384 rows 23-48 us against 25-52, at 1024 rows 96
    // against 114; gate/up 24576 x 4096 at 66-384 rows 41-89 against 43-96.
    // Beyond two rounds of workgroups they lose (gate/up at 8000 rows: 1610
    // against 1440 us), so they are not offered there.
    struct Cand {
      int mfw, tnb, splits, ks;
      long grid, key[6];
    };
    //
    // 128-feature tiles are offered only when the pick among the wider ones
    // splits K into steps shorter than 32: they reach the same grid with half
    // the splits, so half the partials for the residual norm to read.  O
    // 4096 x 4096 at 224-384 rows: 17.0-22.8 us with 4 splits against
    // 18.7-23.1 with 8 (down, with 48-step splits, would lose: 38.5-56.2
    // against 35.2-45.7).
    Cand c[36];
    int n = 0;
    bool one_round = false, unsplit_fills = false;
    auto add = [&](int tnb) {
      if (N % (32 * tnb)) return;
      for (int mfw : {4, 3, 2})
        for (int S = 1; S <= 8 && S <= max_splits; S *= 2) {
          const int ks = (KT + S - 1) / S;
          if (S > 1 && ks < 8) break;
          const int splits = (KT + ks - 1) / ks;
          const int MT = (M + 64 * mfw - 1) / (64 * mfw);
          const long grid = (long)(N / (32 * tnb)) * MT * splits;
          const long rounds = (grid + 255) / 256;
          if (tnb < 8 && rounds > 2) continue;  // many rounds: wider tiles move fewer bytes
          const bool single = grid >= 128 && rounds == 1;
          one_round |= single;
          unsplit_fills |= splits == 1 && grid >= 256;
          c[n++] = {mfw, tnb, splits, ks, grid,
                    {single ? 0 : 1, rounds * mfw * tnb * ks, ks >= 32 ? 0 : 1, -mfw, splits, -tnb}};
        }
    };
    auto best = [&]() {
      const Cand* b = nullptr;
      for (int i = 0; i < n; ++i) {
        if (!one_round && unsplit_fills && c[i].splits != 1) continue;
        if (!b || std::lexicographical_compare(c[i].key, c[i].key + 6, b->key, b->key + 6)) b = &c[i];
      }
      return b;
    };
    add(8);
    add(6);
    const Cand* pick = best();
    if (pick->ks < 32) {
      add(4);
      pick = best();
    }
    // From four rounds of unsplit 256 x 256 tiles on (batched refresh steps),
    // those tiles on the pinned 4-wave schedule beat the finer tiles the work
    // count prefers, though they round up more rows: Q/K/V and gate/up at
    // 3000-11000 rows 2-9% faster (gate/up at 5000 rows 922 against 1014 us,
    // 192- or 128-row tiles); O and down reach four rounds only past 16000
    // rows.  Every output sums K in the same order on either tile.
    for (int i = 0; i < n; ++i)
      if (c[i].mfw == 4 && c[i].tnb == 8 && c[i].splits == 1 && c[i].grid >= 1024) pick = &c[i];
    p.dma_mfw = pick->mfw;
    p.dma_tnb = pick->tnb;
    p.splits = pick->splits;
    p.ks_per_split = pick->ks;
    p.grid = (int)pick->grid;
    p.dma_nw = pick->tnb == 6 ? 12 : 8;
    p.dma_gm = 0;
    if (p.grid > 512 && pick->mfw == 4 && pick->tnb == 8) {
      // several rounds of 256 x 256 tiles (batches, long full-sequence
      // steps): one wave per SIMD with the pinned schedule, in bands of 8
      // row tiles (measured at 12000 rows; gemm_tiles.hip)
      p.dma_nw = 4;
      p.dma_gm = 8;
    }
    p.mf = 8;
    p.nf = 4;
    p.ck = 1;
    return p;
  }
  if (M <= 64) {
    p.nf = (N >= 16384 && N % 128 == 0) ? 2 : 1;
    p.mf = M <= 16 ? 1 : M <= 32 ? 2 : M <= 48 ? 3 : 4;
    p.ck = 8;
  } else {
    p.mf = 8;
    p.ck = 4;
    p.nf = N % 128 == 0 ? 2 : 1;
  }
  const int NB = N / (16 * kWaves * p.nf);
  const int MT = (M + 16 * p.mf - 1) / (16 * p.mf);
  const long target = M > 64 ? 256 : p.nf == 2 ? 384 : 512;
  int S = 1;
  while ((long)NB * MT * S < target && KT / (2 * S) >= p.ck && 2 * S <= max_splits) S *= 2;
  p.ks_per_split = (KT + S - 1) / S;
  if (w8) p.ks_per_split += p.ks_per_split & 1;  // fp8 fragments hold K steps in pairs
  p.splits = (KT + p.ks_per_split - 1) / p.ks_per_split;
  p.grid = NB * MT * p.splits;
  return p;
}

template <int NF, int MF, bool W8>
static void launch_mf(dim3 grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1, const uint16_t* X,
                      int ldx, const void* Wp, float* C, int M, int N, int K, int NB, int MT,
                      int S, int ks, const float* wsc) {
  if constexpr (MF == 8) {
    launch_timed(k_gemm_bf16_big<NF, W8>, grid, st, e0, e1, X, ldx, (const u32x4*)Wp, C, M, N, K,
                 NB, MT, S, ks, wsc);
  } else if constexpr (W8) {
    // fp8 fragments carry two K steps; with one weight group per wave, twice
    // the steps per batch (the same bytes in flight) measured faster, with
    // two groups (LM head) the bf16 batch did
    launch_timed(k_gemm_bf16<NF, MF, NF == 1 ? 16 : 4, NF == 1 ? 16 : 8, true>, grid, st, e0, e1,
                 X, ldx, (const u32x4*)Wp, C, M, N, K, NB, MT, S, ks, wsc);
  } else {
    launch_timed(k_gemm_bf16<NF, MF, NF == 1 ? 8 : 4, 8, false>, grid, st, e0, e1, X, ldx,
                 (const u32x4*)Wp, C, M, N, K, NB, MT, S, ks, wsc);
  }
}

bool gemm_plan_ok(const GemmPlan& p, int M, int N, int K, bool w8, bool swiglu) {
  if (M <= 0 || N <= 0 || K <= 0 || K % 32) return false;
  const int KT = K / 32;
  if (p.splits < 1 || p.ks_per_split < 1 || (long)p.ks_per_split * p.splits < KT ||
      (long)p.ks_per_split * (p.splits - 1) >= KT)
    return false;
  const bool fp8_steps = K % 64 == 0 && p.ks_per_split % 2 == 0;  // fp8 fragments pair K steps
  if (p.fused_gw) {
    const int gw = p.fused_gw;
    return !swiglu && M <= 96 && N % 16 == 0 && (gw == 2 || gw == 3 || gw == 4 || gw == 6 || gw == 7) &&
           (N / 16) % gw == 0 && (long)(N / 16 / gw) * p.splits == p.grid && (!w8 || fp8_steps);
  }
  if (p.dma_mfw) {
    const int TN = 32 * p.dma_tnb;
    if (w8 || p.dma_mfw < 2 || p.dma_mfw > 4 ||
        (p.dma_tnb != 8 && p.dma_tnb != 6 && p.dma_tnb != 4) || N % TN)
      return false;
    // the instances the launcher has: 12 waves with 192-feature tiles, 8
    // with the others, 4 only with 256 x 256 tiles; bands of 0 or 8 row tiles
    const bool waves_ok = p.dma_tnb == 6 ? p.dma_nw == 12
                                         : p.dma_nw == 8 || (p.dma_nw == 4 && p.dma_tnb == 8 &&
                                                             p.dma_mfw == 4);
    if (!waves_ok || (p.dma_gm != 0 && p.dma_gm != 8)) return false;
    const long MT = (M + 64L * p.dma_mfw - 1) / (64L * p.dma_mfw);
    return (long)(N / TN) * MT * p.splits == p.grid && (!swiglu || p.splits == 1);
  }
  if (swiglu || (p.nf != 1 && p.nf != 2) ||
      (p.mf != 1 && p.mf != 2 && p.mf != 3 && p.mf != 4 && p.mf != 8) ||
      N % (16 * kWaves * p.nf))
    return false;
  const long NB = N / (16 * kWaves * p.nf), MT = (M + 16L * p.mf - 1) / (16L * p.mf);
  return NB * MT * p.splits == p.grid && (!w8 || fp8_steps);
}

void gemm_plan_tile(const GemmPlan& p, int* kernel, int* rows, int* features, int* waves) {
  if (p.fused_gw) {
    *kernel = 1;
    *rows = 16 * p.mf;
    *features = 16 * p.fused_gw;
    *waves = p.fused_gw;
  } else if (p.dma_mfw) {
    *kernel = 2;
    *rows = 64 * p.dma_mfw;
    *features = 32 * p.dma_tnb;
    *waves = p.dma_nw;
  } else {
    *kernel = 3;
    *rows = 16 * p.mf;
    *features = 16 * kWaves * p.nf;
    *waves = kWaves;
  }
}

hipError_t gemm_bf16(const uint16_t* X, int ldx, const void* Wp, float* C, int M, int N, int K,
                     const GemmPlan& p, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop,
                     const float* wsc) {
  if (M <= 0) return hipSuccess;
  if (!gemm_plan_ok(p, M, N, K, wsc != nullptr, false)) return hipErrorInvalidValue;
  if (p.fused_gw) {
    return gemm_bf16_split_fused(X, ldx, Wp, C, M, N, K, p.fused_gw, p.splits, p.ks_per_split, st,
                                 ev_start, ev_stop, wsc);
  }
  if (p.dma_mfw) {
    if (!launch_gemm_tiles(p, X, ldx, Wp, C, M, N, K, nullptr, st, ev_start, ev_stop))
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
  const int NB = N / (16 * kWaves * p.nf);
  const int MT = (M + 16 * p.mf - 1) / (16 * p.mf);
  const dim3 grid(p.grid);
  bool launched = false;
#define WD_GEMM_CASE(NF, MF)                                                                  \
  if (p.nf == NF && p.mf == MF) {                                                             \
    if (wsc)                                                                                  \
      launch_mf<NF, MF, true>(grid, st, ev_start, ev_stop, X, ldx, Wp, C, M, N, K, NB, MT,    \
                              p.splits, p.ks_per_split, wsc);                                 \
    else                                                                                      \
      launch_mf<NF, MF, false>(grid, st, ev_start, ev_stop, X, ldx, Wp, C, M, N, K, NB, MT,   \
                               p.splits, p.ks_per_split, wsc);                                \
    launched = true;                                                                          \
  }
  WD_GEMM_CASE(1, 1) WD_GEMM_CASE(1, 2) WD_GEMM_CASE(1, 3) WD_GEMM_CASE(1, 4)
  WD_GEMM_CASE(2, 1) WD_GEMM_CASE(2, 2) WD_GEMM_CASE(2, 3) WD_GEMM_CASE(2, 4)
  WD_GEMM_CASE(1, 8) WD_GEMM_CASE(2, 8)
#undef WD_GEMM_CASE
  if (!launched) return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t gemm_bf16_qkv_tiles(const uint16_t* X, int ldx, const void* Wp, int M, int N, int K,
                               const GemmPlan& p, const QkvOut& qo, hipStream_t st, hipEvent_t e0,
                               hipEvent_t e1) {
  if (M <= 0) return hipSuccess;
  if (!p.dma_mfw || p.splits != 1 || N != (qo.nh + 2 * qo.nkv) * 128 ||
      !gemm_plan_ok(p, M, N, K, false, true))
    return hipErrorInvalidValue;
  if (!launch_gemm_tiles(p, X, ldx, Wp, nullptr, M, N, K, nullptr, st, e0, e1, &qo))
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t gemm_bf16_swiglu_dma(const uint16_t* X, int ldx, const void* Wp, uint16_t* out, int M,
                                int F, int K, const GemmPlan& p, hipStream_t st,
                                hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int N = 2 * F;
  if (M <= 0) return hipSuccess;
  if (!p.dma_mfw || !gemm_plan_ok(p, M, N, K, false, true)) return hipErrorInvalidValue;
  if (!launch_gemm_tiles(p, X, ldx, Wp, nullptr, M, N, K, out, st, ev_start, ev_stop))
    return hipErrorInvalidValue;
  return hipGetLastError();
}

// ---- fp32 GEMM (small fp32 models) -------------------------------------------------
// 64x64 output tile per 256-thread block, 4x4 outputs per thread, K in
// chunks of 16 staged through LDS.  N and K must be multiples of 64 and 16.
__global__ __launch_bounds__(256) void k_gemm_f32(const float* __restrict__ X, int ldx,
                                                  const float* __restrict__ W,
                                                  float* __restrict__ C, int M, int N, int K) {
  __shared__ float xs[16][65];
  __shared__ float ws[16][65];
  const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4] = {};
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int e = threadIdx.x; e < 64 * 16; e += 256) {
      const int r = e >> 4, kk = e & 15;
      xs[kk][r] = (m0 + r < M) ? X[(long)(m0 + r) * ldx + k0 + kk] : 0.f;
      ws[kk][r] = W[(long)(n0 + r) * K + k0 + kk];
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float xr[4], wr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) xr[i] = xs[kk][ty * 4 + i];
#pragma unroll
      for (int j = 0; j < 4; ++j) wr[j] = ws[kk][tx * 4 + j];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(xr[i], wr[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; ++j) C[(long)m * N + n0 + tx * 4 + j] = acc[i][j];
  }
}

hipError_t gemm_f32(const float* X, int ldx, const float* W, float* C, int M, int N, int K,
                    hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
  if (M <= 0) return hipSuccess;
  dim3 grid(N / 64, (M + 63) / 64);
  launch_timed(k_gemm_f32, grid, st, ev_start, ev_stop, X, ldx, W, C, M, N, K);
  return hipGetLastError();
}

}  // namespace wd
