// The many-row projection GEMM (refresh steps, the full-sequence path,
// batches): C[s][m][n] = sum over split s of K of X[m][k] W[n][k] on
// 32x32x16 bf16 MFMAs, both operands staged through LDS by direct-to-LDS
// loads, or with the SwiGLU epilogue out[m][f] = silu(gate) * up.  The
// launch plan (tile, waves, K splits, raster) comes from plan_gemm_bf16.
#include <hip/hip_ext.h>

#include <cmath>
#include <type_traits>

#include "common.h"
#include "kernels.h"

namespace wd {

namespace {

template <int V>
using ic = std::integral_constant<int, V>;

// With a start/stop event pair, the launch records them from its own dispatch
// (the kernel's execution time, as a kernel trace reports it).
template <typename F, typename... A>
void launch_timed_block(F kernel, dim3 grid, dim3 block, hipStream_t st, hipEvent_t e0,
                        hipEvent_t e1, A... args) {
  if (e0)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, st, e0, e1, 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, st, args...);
}

}  // namespace

// ---- bf16 GEMM for many rows: multi-stage LDS pipeline fed by direct-to-LDS loads -------
// Workgroup tile: 64 * MFW rows x 32 * TNB features (256, 192 or 128); wave
// (wm, wn) computes 32 * MFW rows x 32 * TNB / (NW / 2) features (256: 128
// with 4 waves, 64 with 8; 192: 32 with 12; 128: 32 with 8) on
// v_mfma_f32_32x32x16_bf16 (weights as the A operand, activations as B).
// Each 32-wide K step
// is one stage in LDS, filled by 16-byte direct-to-LDS loads (lane l of a
// load lands at +16 l) ST - 1 stages ahead of the step being computed; one
// barrier per stage, with the waits issued by hand so that the compiler does
// not drain every load at the barrier.
// Stage layout (1 KB blocks after a 1 KB pad that keeps every load target off
// LDS address 0):
//   activation blocks 0 .. 4 MFW - 1: tile rows 16 b .. 16 b + 15, 64 bytes
//     each; the 16-byte chunk c of row r sits in slot c ^ swz(r), with
//     swz(r) = ((r >> 1) ^ (r >> 2)) & 3, so the 32-row operand reads hit
//     distinct banks;
//   weight blocks 4 MFW + 2 i + h: the A operand of feature block i (packed
//     groups 2 i, 2 i + 1 of the tile) for K half h, assembled by the loads
//     themselves from the two packed 16x32 fragments: rows of 16 lanes
//     [g0 h0 g1 h1] (h = 0) and [g2 h2 g3 h3] (h = 1).
typedef float f32x16 __attribute__((ext_vector_type(16)));
__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                  __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
// at most N vector-memory operations of this wave outstanding (vmcnt in bits
// 3:0 and 15:14; expcnt and lgkmcnt left unconstrained)
#define WD_WAIT_VM(N) __builtin_amdgcn_s_waitcnt(((N) & 15) | 0x70 | 0xF00 | ((((N) >> 4) & 3) << 14))
// every LDS operation of this wave complete (lgkmcnt 0; vmcnt, expcnt free)
#define WD_WAIT_LGKM0() __builtin_amdgcn_s_waitcnt(0xC07F)

// Epilogues (EPI; the last two need all of K in one workgroup, S = 1):
//   kTileEpiPartial: fp32 split-K partials C[s][m][n].
//   kTileEpiSwiGlu (weights packed kPackGateUp): lane values of packed groups
//     2 i + h come as gate (e / 4 = 2 h) and up (e / 4 = 2 h + 1) of the same
//     features, so the epilogue writes out[m][f] = silu(gate) * up (bf16, F =
//     N / 2 per row) instead of the fp32 products.
//   kTileEpiQkv (weights packed kPackRopePair, head_dim 128): likewise a lane
//     holds four dims of a head (e / 4 = 2 h) and their rotation partners 64
//     dims on (e / 4 = 2 h + 1), so it adds the bias, rotates q and k at the
//     row's position and stores q, k and v as bf16 (q to its row, k and v to
//     the row's K/V cache row), as k_qkv_epilogue does from the partials.
// TNB: 32-feature blocks per tile (8: 256 features, 6: 192, 4: 128).  NW: waves per
// workgroup, in two row halves; the NW / 2 waves of a half split the TNB
// blocks evenly (8 waves and 256 features: two waves per SIMD, 64 features
// each; 4 waves: one per SIMD, 128 x 128 each).  SCH 1: each K step's operand
// reads pinned under the MFMAs of the step before (for one wave per SIMD).  gm > 0:
// workgroups in bands of gm row tiles (for grids of several rounds).
constexpr int kTileEpiPartial = 0, kTileEpiSwiGlu = 1, kTileEpiQkv = 2;

template <int MFW, int ST, int EPI, int NW, int TNB, int SCH>
__global__ __launch_bounds__(64 * NW, 1) void k_gemm_bf16_dma(const uint16_t* __restrict__ X, int ldx,
                                                          const u32x4* __restrict__ Wp,
                                                          float* __restrict__ C, int M, int N,
                                                          int K, int NB, int MT, int S, int ks,
                                                          int gm, uint16_t* __restrict__ out,
                                                          QkvOut qo) {
  // the host pass only needs the kernel's signature
#if defined(__HIP_DEVICE_COMPILE__)
  static_assert(NW % 2 == 0 && TNB % (NW / 2) == 0, "waves split the feature blocks evenly");
  constexpr int NFW = TNB / (NW / 2);    // 32-feature blocks of each wave
  constexpr int F = 4 * MFW + 2 * TNB;   // 1 KB blocks per stage
  constexpr int FW = (F + NW - 1) / NW;  // blocks wave w loads: w, w + NW, ... below F
  constexpr int FWMIN = F / NW;          // blocks every wave loads
  constexpr int STAGE16 = (F + 1) * 64;  // u32x4 per stage buffer, pad included
  static_assert(ST >= 3 && ST <= 4, "stages");
  static_assert(SCH == 0 || SCH == 1, "schedules");
  static_assert((ST - 2) * FW < 64, "outstanding loads fit the wait counter");
  __shared__ __attribute__((aligned(16))) u32x4 st0[STAGE16], st1[STAGE16], st2[STAGE16],
      st3[ST > 3 ? STAGE16 : 1];
  const int G = NB * MT * S;
  int id = blockIdx.x;
  if ((G & 7) == 0) id = (id & 7) * (G >> 3) + (id >> 3);
  int mt, nb, sp;
  if (gm <= 0) {
    // row tiles of one weight slice next to each other (one XCD shares the slice)
    mt = id % MT;
    nb = (id / MT) % NB;
    sp = id / (MT * NB);
  } else {
    // bands of gm row tiles: within a band the row tile varies fastest, so
    // the workgroups an XCD runs at once cover gm row tiles x a few weight
    // slices and each operand tile it loads serves several of them
    sp = id / (MT * NB);
    const int t = id % (MT * NB), band = t / (gm * NB), first = band * gm;
    const int rows = min(MT - first, gm), w = t % (gm * NB);
    mt = first + w % rows;
    nb = w / rows;
  }
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int wm = wave & 1, wn = wave >> 1;
  const int KT = K >> 5;
  const int kt0 = sp * ks, nkt = min(KT, kt0 + ks) - kt0;
  const int m0 = mt * 64 * MFW;
  // per-lane source of every block this wave loads, at K step kt0
  const u32x4* src[FW];
  int step16[FW];  // u32x4 between consecutive K steps
#pragma unroll
  for (int q = 0; q < FW; ++q) {
    const int f = min(wave + NW * q, F - 1);  // a wave past F never issues this slot
    if (f < 4 * MFW) {
      const int r = f * 16 + (lane >> 2);
      const int c = (lane & 3) ^ (((r >> 1) ^ (r >> 2)) & 3);
      const long row = min(m0 + r, M - 1);
      src[q] = (const u32x4*)(X + row * ldx + kt0 * 32 + c * 8);
      step16[q] = 4;
    } else {
      const int i = (f - 4 * MFW) >> 1, h = f & 1;
      const int g = 2 * (nb * TNB + i) + ((lane >> 4) & 1);
      const int sl = (lane & 15) + 16 * (2 * h + (lane >> 5));
      src[q] = Wp + ((long)g * KT + kt0) * 64 + sl;
      step16[q] = 64;
    }
  }
  auto stage = [&](auto B) -> u32x4* {
    constexpr int b = decltype(B)::value;
    if constexpr (b == 0) return st0 + 64;
    else if constexpr (b == 1) return st1 + 64;
    else if constexpr (b == 2) return st2 + 64;
    else return st3 + 64;
  };
  auto issue = [&](auto B, int it) {
    const int k = min(it, nkt - 1);  // steps past the split reload its last one, unused
    u32x4* dst = stage(B);
#pragma unroll
    for (int q = 0; q < FW; ++q)
      if (q < FWMIN || wave + NW * q < F)  // uniform over the wave
        __builtin_amdgcn_global_load_lds(src[q] + (long)k * step16[q], dst + (wave + NW * q) * 64,
                                         16, 0, 0);
  };
  f32x16 acc[NFW][MFW];
#pragma unroll
  for (int a = 0; a < NFW; ++a)
#pragma unroll
    for (int b = 0; b < MFW; ++b)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
  // Per-lane offsets (u32x4) of this wave's operands inside a stage: weight
  // block 4 MFW + 2 (wn NFW + ii) + h, and activation row (wm MFW + jj) 32 +
  // l % 32 in slot (2 h + l / 32) ^ swz(l) (swz only sees the row's low bits).
  // They are kept opaque so that each operand read is its stage buffer plus
  // one offset and a constant: the LDS lowering tags an access with its buffer
  // only a few address steps deep, and for an untagged read the compiler
  // waits for every direct-to-LDS load in flight.
  int a_off = (4 * MFW + 2 * wn * NFW) * 64 + lane;
  int x_off0 = wm * MFW * 128 + (lane & 31) * 4 + (((lane >> 5) ^ (lane >> 1) ^ (lane >> 2)) & 3);
  int x_off1 = wm * MFW * 128 + (lane & 31) * 4 + ((2 + (lane >> 5)) ^ (((lane >> 1) ^ (lane >> 2)) & 3));
  asm volatile("" : "+v"(a_off), "+v"(x_off0), "+v"(x_off1));
  // SCH 0: step it reads and multiplies its own operands.  SCH 1 (one wave
  // per SIMD): the operands of step it + 1's first K half are read under step
  // it's second-half MFMAs, and step it's second half under its first, so
  // the wave hides its own LDS latency across steps; the barrier at step it
  // therefore certifies stage it + 1 as well (one stage fewer in flight).
  // The schedule is pinned with scheduling barriers (the compiler would
  // otherwise wait for each small group of reads before the MFMAs that use
  // them).  Measured at 5000-12000 rows against reads within the step only:
  // 2-7% faster on the four projections.
  u32x4 a[2][NFW], bx[2][MFW];
  auto rd = [&](const u32x4* sb, int h) {
#pragma unroll
    for (int ii = 0; ii < NFW; ++ii) a[h][ii] = sb[a_off + ii * 128 + h * 64];
#pragma unroll
    for (int jj = 0; jj < MFW; ++jj) bx[h][jj] = sb[(h ? x_off1 : x_off0) + jj * 128];
  };
  auto mm = [&](int h) {
#pragma unroll
    for (int jj = 0; jj < MFW; ++jj)
#pragma unroll
      for (int ii = 0; ii < NFW; ++ii) acc[ii][jj] = mfma32(a[h][ii], bx[h][jj], acc[ii][jj]);
  };
  auto interleave = [&]() {
#pragma unroll
    for (int i = 0; i < NFW + MFW; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // two MFMAs
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one LDS read
    }
  };
  // step it: its stage has landed (this wave: at most the later stages' loads
  // outstanding; every wave: the barrier), every wave has finished reading the
  // buffer of step it - 1, which is refilled with step it + ST - 1
  auto body = [&](auto J, int it) {
    constexpr int j = decltype(J)::value;
    // a wave that loads more than FWMIN blocks per stage waits for more than it must
    WD_WAIT_VM((ST - 2 - SCH) * FWMIN);
    WD_WAIT_LGKM0();
    __builtin_amdgcn_s_barrier();
    issue(ic<(j + ST - 1) % ST>{}, it + ST - 1);
    if (it < nkt) {
      const u32x4* sb = stage(ic<j % ST>{});
      if constexpr (SCH == 0) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          u32x4 a0[NFW], b0[MFW];
#pragma unroll
          for (int ii = 0; ii < NFW; ++ii) a0[ii] = sb[a_off + ii * 128 + h * 64];
#pragma unroll
          for (int jj = 0; jj < MFW; ++jj) b0[jj] = sb[(h ? x_off1 : x_off0) + jj * 128];
#pragma unroll
          for (int jj = 0; jj < MFW; ++jj)
#pragma unroll
            for (int ii = 0; ii < NFW; ++ii) acc[ii][jj] = mfma32(a0[ii], b0[jj], acc[ii][jj]);
        }
      } else {
        // a[0] / bx[0] hold step it's first half (read in step it - 1)
        rd(sb, 1);
        mm(0);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
        rd(stage(ic<(j + 1) % ST>{}), 0);  // at the last step a valid read, unused
        mm(1);
        interleave();
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };
  issue(ic<0>{}, 0);
  issue(ic<1>{}, 1);
  if constexpr (ST > 3) issue(ic<2>{}, 2);
  if constexpr (SCH == 1) {
    // stages 0 and 1 landed for every wave; step 0's first half
    WD_WAIT_VM((ST - 3) * FWMIN);
    __builtin_amdgcn_s_barrier();
    rd(stage(ic<0>{}), 0);
  }
  for (int it = 0; it < nkt; it += ST) {
    body(ic<0>{}, it);
    body(ic<1>{}, it + 1);
    body(ic<2>{}, it + 2);
    if constexpr (ST > 3) body(ic<3>{}, it + 3);
  }
  WD_WAIT_VM(0);  // no load may land in LDS after the workgroup ends
  // D of (feature block i, row block j): lane l holds row j * 32 + l % 32,
  // features i * 32 + (e / 4) * 8 + (l / 32) * 4 + e % 4
#pragma unroll
  for (int ii = 0; ii < NFW; ++ii)
#pragma unroll
    for (int jj = 0; jj < MFW; ++jj) {
      const int m = m0 + (wm * MFW + jj) * 32 + (lane & 31);
      if (m >= M) continue;
      if constexpr (EPI == kTileEpiQkv) {
        const int i = nb * TNB + wn * NFW + ii;
#pragma unroll
        for (int hg = 0; hg < 2; ++hg) {
          const int grp = 2 * i + hg, head = grp >> 3;
          const int d0 = (grp & 7) * 8 + (lane >> 5) * 4;  // dims d0 .. d0 + 3, partners + 64
          float x0[4], x1[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            x0[j] = acc[ii][jj][8 * hg + j];
            x1[j] = acc[ii][jj][8 * hg + 4 + j];
          }
          if (qo.bias) {
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              x0[j] += bf2f(qo.bias[head * 128 + d0 + j]);
              x1[j] += bf2f(qo.bias[head * 128 + d0 + 64 + j]);
            }
          }
          if (head < qo.nh + qo.nkv) {
            const f32x4* cs = (const f32x4*)(qo.rope + ((long)qo.row_pos[m] * 64 + d0) * 2);
            const f32x4 a = cs[0], b = cs[1];  // (cos, sin) of dims d0, d0 + 1 and d0 + 2, d0 + 3
            const float c[4] = {a[0], a[2], b[0], b[2]}, sn[4] = {a[1], a[3], b[1], b[3]};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const float y0 = x0[j] * c[j] - x1[j] * sn[j];
              const float y1 = x1[j] * c[j] + x0[j] * sn[j];
              x0[j] = y0;
              x1[j] = y1;
            }
          }
          uint16_t* dst;
          if (head < qo.nh)
            dst = qo.q + ((long)m * qo.nh + head) * 128;
          else if (head < qo.nh + qo.nkv)
            dst = qo.kc + ((long)(head - qo.nh) * qo.cache_rows + qo.row_tok[m]) * 128;
          else
            dst = qo.vc + ((long)(head - qo.nh - qo.nkv) * qo.cache_rows + qo.row_tok[m]) * 128;
          u32x2 w0, w1;
          w0.x = (uint32_t)f2bf(x0[0]) | ((uint32_t)f2bf(x0[1]) << 16);
          w0.y = (uint32_t)f2bf(x0[2]) | ((uint32_t)f2bf(x0[3]) << 16);
          w1.x = (uint32_t)f2bf(x1[0]) | ((uint32_t)f2bf(x1[1]) << 16);
          w1.y = (uint32_t)f2bf(x1[2]) | ((uint32_t)f2bf(x1[3]) << 16);
          *(u32x2*)(dst + d0) = w0;
          *(u32x2*)(dst + d0 + 64) = w1;
        }
        continue;
      }
      if constexpr (EPI == kTileEpiSwiGlu) {
        const int F = N >> 1;
        const int i = nb * TNB + wn * NFW + ii;
#pragma unroll
        for (int hg = 0; hg < 2; ++hg) {
          const int f0 = (2 * i + hg) * 8 + (lane >> 5) * 4;
          float y[4];
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            const float x = acc[ii][jj][8 * hg + j], u = acc[ii][jj][8 * hg + 4 + j];
            y[j] = x / (1.0f + expf(-x)) * u;
          }
          u32x2 w;
          w.x = (uint32_t)f2bf(y[0]) | ((uint32_t)f2bf(y[1]) << 16);
          w.y = (uint32_t)f2bf(y[2]) | ((uint32_t)f2bf(y[3]) << 16);
          *(u32x2*)(out + (long)m * F + f0) = w;
        }
        continue;
      }
      const int n0 = (nb * TNB + wn * NFW + ii) * 32 + (lane >> 5) * 4;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 v = {acc[ii][jj][g * 4], acc[ii][jj][g * 4 + 1], acc[ii][jj][g * 4 + 2],
                         acc[ii][jj][g * 4 + 3]};
        *(f32x4*)(C + ((long)sp * M + m) * N + n0 + g * 8) = v;
      }
    }
#endif
}

// Waves of the many-row kernel: with 256-feature tiles 8 (two per SIMD, 64
// features each) measured 2-8% faster than 4 with the plain schedule on the
// refresh shapes (224-384 rows, weights from HBM): Q/K/V at 384 rows 51.7 us
// against 54.8, gate/up 91.9 against 94.1, down 47.0 against 50.7.  With
// 192-feature tiles 12 (three per SIMD, 32 features each) beat 6 by up to
// 10%.  At 12000 rows (several rounds of 256 x 256 tiles) 4 waves of 128 x
// 128 with the pinned schedule and 4 stages, in bands of 8 row tiles, beat 8
// waves without bands: Q/K/V (12288 x 4096) 1042-1046 us against 1155, O
// 325 against 323-428, down 997 against 1004-1172.
template <int EPI>
static bool launch_dma(const GemmPlan& p, hipStream_t st, hipEvent_t e0, hipEvent_t e1,
                       const uint16_t* X, int ldx, const u32x4* Wp, float* C, int M, int N,
                       int K, int NB, int MT, int S, int ks, uint16_t* out, const QkvOut& qo) {
  const dim3 grid(p.grid), b(64 * p.dma_nw);
#define WD_DMA(MFW, ST, NW, TNB, SCH)                                                          \
  launch_timed_block(k_gemm_bf16_dma<MFW, ST, EPI, NW, TNB, SCH>, grid, b, st, e0, e1, X, ldx,  \
                     Wp, C, M, N, K, NB, MT, S, ks, p.dma_gm, out, qo)
  if (p.dma_nw == 4 && p.dma_tnb == 8 && p.dma_mfw == 4) {
    WD_DMA(4, 4, 4, 8, 1);
    return true;
  }
  if (p.dma_nw == 8 && p.dma_tnb == 8) {
    switch (p.dma_mfw) {
      case 4: WD_DMA(4, 3, 8, 8, 0); return true;
      case 3: WD_DMA(3, 4, 8, 8, 0); return true;
      case 2: WD_DMA(2, 4, 8, 8, 0); return true;
      default: return false;
    }
  }
  if (p.dma_nw == 12 && p.dma_tnb == 6) {
    switch (p.dma_mfw) {
      case 4: WD_DMA(4, 3, 12, 6, 0); return true;
      case 3: WD_DMA(3, 4, 12, 6, 0); return true;
      case 2: WD_DMA(2, 4, 12, 6, 0); return true;
      default: return false;
    }
  }
  if (p.dma_nw == 8 && p.dma_tnb == 4) {
    switch (p.dma_mfw) {
      case 4: WD_DMA(4, 3, 8, 4, 0); return true;
      case 3: WD_DMA(3, 4, 8, 4, 0); return true;
      case 2: WD_DMA(2, 4, 8, 4, 0); return true;
      default: return false;
    }
  }
#undef WD_DMA
  return false;
}

bool launch_gemm_tiles(const GemmPlan& p, const uint16_t* X, int ldx, const void* Wp, float* C,
                       int M, int N, int K, uint16_t* swiglu_out, hipStream_t st, hipEvent_t e0,
                       hipEvent_t e1, const QkvOut* qkv) {
  const int TN = 32 * p.dma_tnb;
  const int NB = N / TN, MT = (M + 64 * p.dma_mfw - 1) / (64 * p.dma_mfw);
  const QkvOut none{};
  if (qkv)
    return p.splits == 1 &&
           launch_dma<kTileEpiQkv>(p, st, e0, e1, X, ldx, (const u32x4*)Wp, nullptr, M, N, K, NB,
                                   MT, 1, K / 32, nullptr, *qkv);
  if (swiglu_out)
    return launch_dma<kTileEpiSwiGlu>(p, st, e0, e1, X, ldx, (const u32x4*)Wp, nullptr, M, N, K,
                                      NB, MT, 1, K / 32, swiglu_out, none);
  return launch_dma<kTileEpiPartial>(p, st, e0, e1, X, ldx, (const u32x4*)Wp, C, M, N, K, NB, MT,
                                     p.splits, p.ks_per_split, nullptr, none);
}

}  // namespace wd
