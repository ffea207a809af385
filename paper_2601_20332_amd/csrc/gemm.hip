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
#include "common.h"
#include "kernels.h"

namespace wd {

// ---- weight packing -------------------------------------------------------------
// Fragment (nt, kt) holds W rows nt*16..nt*16+15 and columns kt*32..kt*32+31;
// lane l stores row nt*16 + l%16, columns kt*32 + (l/16)*8 .. +7 (the MFMA
// A-operand layout).  Fragments of one 16-row group are contiguous along K,
// so a wave streams each group as one contiguous run.
__global__ void k_pack_frags(const uint16_t* __restrict__ W, int N, int K, u32x4* __restrict__ out) {
  const int KT = K >> 5;
  const long total = (long)(N >> 4) * KT * 64;
  for (long i = (long)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (long)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const long f = i >> 6;
    const int kt = (int)(f % KT);
    const long nt = f / KT;
    const long row = nt * 16 + (lane & 15);
    const int col = kt * 32 + (lane >> 4) * 8;
    out[i] = *(const u32x4*)(W + row * K + col);
  }
}

hipError_t pack_frags(const uint16_t* W, int N, int K, void* out, hipStream_t st) {
  const long total = (long)(N / 16) * (K / 32) * 64;
  const int blocks = (int)std::min<long>((total + 255) / 256, 65536);
  hipLaunchKernelGGL(k_pack_frags, dim3(blocks), dim3(256), 0, st, W, N, K, (u32x4*)out);
  return hipGetLastError();
}

// ---- bf16 weight-streaming GEMM ----------------------------------------------------
// Workgroup = 4 waves on the same NF 16-row weight groups and the same
// 16*MF activation rows; the waves take every 4th 32-wide K step of the
// workgroup's split and are summed through LDS at the end.
// Grid = NB (weight groups / NF) x MT (row tiles) x S (K splits), remapped so
// that each XCD receives a contiguous range of tiles (row tiles of one weight
// group share an L2).
template <int NF, int MF>
__global__ __launch_bounds__(256) void k_gemm_bf16(const uint16_t* __restrict__ X, int ldx,
                                                   const u32x4* __restrict__ Wp,
                                                   float* __restrict__ C, int M, int N, int K,
                                                   int NB, int MT, int S, int ks_per_split) {
  const int G = NB * MT * S;
  int id = blockIdx.x;
  if ((G & 7) == 0) id = (id & 7) * (G >> 3) + (id >> 3);
  const int mt = id % MT;
  const int rest = id / MT;
  const int nb = rest % NB;
  const int s = rest / NB;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int KT = K >> 5;
  const int kt0 = s * ks_per_split;
  const int kt1 = min(KT, kt0 + ks_per_split);
  const int m0 = mt * 16 * MF;

  const u32x4* wp[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f) wp[f] = Wp + ((long)(nb * NF + f) * KT) * 64 + lane;
  const uint16_t* xp[MF];
  bool xv[MF];
#pragma unroll
  for (int f = 0; f < MF; ++f) {
    const int row = m0 + f * 16 + (lane & 15);
    xv[f] = row < M;
    xp[f] = X + (long)(xv[f] ? row : 0) * ldx + (lane >> 4) * 8;
  }

  f32x4 acc[NF][MF];
#pragma unroll
  for (int a = 0; a < NF; ++a)
#pragma unroll
    for (int b = 0; b < MF; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  const u32x4 zero = {0u, 0u, 0u, 0u};
  int kt = kt0 + wave;
  // Four K steps per iteration: all loads first, so each wave keeps
  // 4 * (NF + MF) 16-byte loads in flight.
  for (; kt + 12 < kt1; kt += 16) {
    u32x4 a[4][NF], b[4][MF];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
#pragma unroll
      for (int f = 0; f < NF; ++f) a[u][f] = __builtin_nontemporal_load(wp[f] + (long)(kt + 4 * u) * 64);
#pragma unroll
      for (int f = 0; f < MF; ++f)
        b[u][f] = xv[f] ? *(const u32x4*)(xp[f] + (kt + 4 * u) * 32) : zero;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
      for (int i = 0; i < NF; ++i)
#pragma unroll
        for (int j = 0; j < MF; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, a[u][i]), __builtin_bit_cast(bf16x8, b[u][j]), acc[i][j],
              0, 0, 0);
  }
  for (; kt < kt1; kt += 4) {
    u32x4 a[NF], b[MF];
#pragma unroll
    for (int f = 0; f < NF; ++f) a[f] = __builtin_nontemporal_load(wp[f] + (long)kt * 64);
#pragma unroll
    for (int f = 0; f < MF; ++f) b[f] = xv[f] ? *(const u32x4*)(xp[f] + kt * 32) : zero;
#pragma unroll
    for (int i = 0; i < NF; ++i)
#pragma unroll
      for (int j = 0; j < MF; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, a[i]), __builtin_bit_cast(bf16x8, b[j]), acc[i][j], 0, 0, 0);
  }

  __shared__ f32x4 red[4][NF * MF][64];
#pragma unroll
  for (int i = 0; i < NF; ++i)
#pragma unroll
    for (int j = 0; j < MF; ++j) red[wave][i * MF + j][lane] = acc[i][j];
  __syncthreads();
  for (int o = threadIdx.x; o < NF * MF * 64; o += 256) {
    const int f = o >> 6, l = o & 63;
    const int i = f / MF, j = f % MF;
    const int m = m0 + j * 16 + (l & 15);
    if (m >= M) continue;
    f32x4 v = red[0][f][l];
    v += red[1][f][l];
    v += red[2][f][l];
    v += red[3][f][l];
    const int n = (nb * NF + i) * 16 + (l >> 4) * 4;
    *(f32x4*)(C + ((long)s * M + m) * N + n) = v;
  }
}

constexpr int kNF = 2;
constexpr int kMF = 4;

GemmPlan plan_gemm_bf16(int M, int N, int K) {
  GemmPlan p;
  const int NB = N / (16 * kNF);
  const int MT = (M + 16 * kMF - 1) / (16 * kMF);
  const int KT = K / 32;
  int S = 1;
  // enough workgroups to cover every CU twice, while each wave keeps >= 4 K steps
  while ((long)NB * MT * S < 512 && KT / (2 * S) >= 16) S *= 2;
  p.splits = S;
  p.ks_per_split = (KT + S - 1) / S;
  p.splits = (KT + p.ks_per_split - 1) / p.ks_per_split;
  p.grid = NB * MT * p.splits;
  return p;
}

hipError_t gemm_bf16(const uint16_t* X, int ldx, const void* Wp, float* C, int M, int N, int K,
                     const GemmPlan& p, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  const int NB = N / (16 * kNF);
  const int MT = (M + 16 * kMF - 1) / (16 * kMF);
  hipLaunchKernelGGL((k_gemm_bf16<kNF, kMF>), dim3(p.grid), dim3(256), 0, st, X, ldx,
                     (const u32x4*)Wp, C, M, N, K, NB, MT, p.splits, p.ks_per_split);
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
                    hipStream_t st) {
  if (M <= 0) return hipSuccess;
  dim3 grid(N / 64, (M + 63) / 64);
  hipLaunchKernelGGL(k_gemm_f32, grid, dim3(256), 0, st, X, ldx, W, C, M, N, K);
  return hipGetLastError();
}

}  // namespace wd
