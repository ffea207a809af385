// Row-wise pieces of a decoder layer and the windowed attention.
//
// Row set: every kernel works on the step's rows r = 0..M-1.  Row r is
// position row_pos[r] of sequence row_seq[r]; its token and its K/V cache row
// are at index row_tok[r] of the concatenated token / cache arrays.
// K/V cache of one layer: [n_kv][cache_rows][head_dim], cache_rows = total
// positions of the batch.
#include <hip/hip_ext.h>

#include "common.h"
#include "kernels.h"

namespace wd {

// four consecutive outputs of a normalized row: one 8-byte store for bf16
template <typename T>
__device__ __forceinline__ void store4(T* dst, float x0, float x1, float x2, float x3) {
  if constexpr (sizeof(T) == 2) {
    u32x2 w;
    w.x = (uint32_t)Elem<T>::from_f(x0) | ((uint32_t)Elem<T>::from_f(x1) << 16);
    w.y = (uint32_t)Elem<T>::from_f(x2) | ((uint32_t)Elem<T>::from_f(x3) << 16);
    *(u32x2*)dst = w;
  } else {
    *(f32x4*)dst = f32x4{x0, x1, x2, x3};
  }
}

// ---- embedding gather + first RMSNorm ------------------------------------------------
// One block per row, 1024 threads; H must be a multiple of 4 and at most 16384.
template <typename T>
__global__ __launch_bounds__(1024) void k_embed_norm(const int32_t* __restrict__ x,
                                                     const int32_t* __restrict__ row_tok,
                                                     const T* __restrict__ emb,
                                                     const T* __restrict__ gamma, float eps,
                                                     float* __restrict__ h, T* __restrict__ a, int H) {
  __shared__ float red[16];
  const long r = blockIdx.x;
  const T* e = emb + (long)x[row_tok[r]] * H;
  float* hr = h + r * H;
  float v[4][4], g[4][4];
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int i = (threadIdx.x + it * 1024) * 4;
    if (i < H) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        g[it][q] = Elem<T>::load(gamma + i + q);
        v[it][q] = Elem<T>::load(e + i + q);
        ss += v[it][q] * v[it][q];
      }
      *(f32x4*)(hr + i) = f32x4{v[it][0], v[it][1], v[it][2], v[it][3]};
    }
  }
  const float inv = 1.0f / sqrtf(block_sum(ss, red) / (float)H + eps);
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int i = (threadIdx.x + it * 1024) * 4;
    if (i < H)
      store4(a + r * H + i, v[it][0] * inv * g[it][0], v[it][1] * inv * g[it][1],
             v[it][2] * inv * g[it][2], v[it][3] * inv * g[it][3]);
  }
}

template <typename T>
hipError_t embed_norm(const int32_t* x, const int32_t* row_tok, const T* emb, const T* gamma,
                      float eps, float* h, T* a, int M, int H, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (H % 4 || H > 16384) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_embed_norm<T>, dim3(M), dim3(1024), 0, st, x, row_tok, emb, gamma, eps, h, a, H);
  return hipGetLastError();
}

// ---- residual add of split-K partials + RMSNorm -----------------------------------------
// One block per row, 1024 threads, 4 consecutive features per thread and pass,
// so every partial of the row is in flight at once.
template <typename T>
__global__ __launch_bounds__(1024) void k_residual_norm(float* __restrict__ h,
                                                        const float* __restrict__ C, int S, int M,
                                                        int H, const T* __restrict__ gamma,
                                                        float eps, T* __restrict__ a,
                                                        const int32_t* __restrict__ row_out) {
  __shared__ float red[16];
  const long r = blockIdx.x;
  float* hr = h + r * H;
  f32x4 v[4];
  float g[4][4];  // gains, loaded with the partials rather than after the reduction
  float ss = 0.f;
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int i = (threadIdx.x + it * 1024) * 4;
    if (i < H) {
#pragma unroll
      for (int q = 0; q < 4; ++q) g[it][q] = Elem<T>::load(gamma + i + q);
      const f32x4 acc = split_sum((const f32x4*)(C + r * H + i), (long)M * H / 4, S);
      v[it] = *(const f32x4*)(hr + i) + acc;
      *(f32x4*)(hr + i) = v[it];
      ss += v[it][0] * v[it][0] + v[it][1] * v[it][1] + v[it][2] * v[it][2] + v[it][3] * v[it][3];
    }
  }
  const int dst = row_out ? row_out[r] : (int)r;
  if (dst < 0) return;  // uniform over the block
  const float inv = 1.0f / sqrtf(block_sum(ss, red) / (float)H + eps);
#pragma unroll
  for (int it = 0; it < 4; ++it) {
    const int i = (threadIdx.x + it * 1024) * 4;
    if (i < H)
      store4(a + (long)dst * H + i, v[it][0] * inv * g[it][0], v[it][1] * inv * g[it][1],
             v[it][2] * inv * g[it][2], v[it][3] * inv * g[it][3]);
  }
}

template <typename T>
hipError_t residual_norm(float* h, const float* C, int S, int M, int H, const T* gamma, float eps,
                         T* a, const int32_t* row_out, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (H % 4 || H > 16384) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_residual_norm<T>, dim3(M), dim3(1024), 0, st, h, C, S, M, H, gamma, eps, a,
                     row_out);
  return hipGetLastError();
}

// ---- QKV epilogue: split-K sum, bias, RoPE, q store, K/V cache scatter ------------------
// Head slots: hs < n_heads is a query head, then n_kv key heads, then n_kv
// value heads.  RoPE rotates the pair (i, i + d/2) of a head.
// bf16 weights are packed with RoPE pairs adjacent (kPackRopePair), so the
// GEMM's columns of dim i and i + 64 of a head are at group i/8, rows i%8
// and 8 + i%8; fp32 weights are in plain order.
template <typename T>
__device__ __forceinline__ int qkv_col(int head, int i, int d, int partner) {
  if constexpr (sizeof(T) == 2)
    return head * 128 + (i >> 3) * 16 + partner * 8 + (i & 7);
  else
    return head * d + i + partner * (d >> 1);
}

template <typename T>
__global__ __launch_bounds__(64) void k_qkv_epilogue(const float* __restrict__ C, int S, int M,
                                                     int N, const T* __restrict__ bias,
                                                     const float* __restrict__ rope_cs,
                                                     const int32_t* __restrict__ row_pos,
                                                     const int32_t* __restrict__ row_tok, int nh,
                                                     int nkv, int d, T* __restrict__ q,
                                                     T* __restrict__ kc, T* __restrict__ vc,
                                                     long cache_rows) {
  // a thread takes dims i .. i + 3 of one head and their rotation partners
  // i + d / 2 .. (16-byte partial loads, 8-byte bf16 stores); a 64-thread
  // block covers 512 / d heads of row r
  const int tph = d >> 3, half = d >> 1;
  const int r = blockIdx.x, hs = blockIdx.y * (64 / tph) + threadIdx.x / tph;
  if (hs >= nh + 2 * nkv) return;
  const int i = (threadIdx.x % tph) * 4;
  const int col = hs * d + i;  // feature index of dim i (bias, outputs)
  f32x4 x0, x1;
  split_sum2((const f32x4*)(C + (long)r * N + qkv_col<T>(hs, i, d, 0)),
             (const f32x4*)(C + (long)r * N + qkv_col<T>(hs, i, d, 1)), (long)M * N / 4, S, x0, x1);
  if (bias) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x0[j] += Elem<T>::load(bias + col + j);
      x1[j] += Elem<T>::load(bias + col + half + j);
    }
  }
  if (hs < nh + nkv) {
    const f32x4* cs = (const f32x4*)(rope_cs + ((long)row_pos[r] * half + i) * 2);
    const f32x4 a = cs[0], b = cs[1];  // (cos, sin) of dims i, i + 1 and i + 2, i + 3
    const float c[4] = {a[0], a[2], b[0], b[2]}, sn[4] = {a[1], a[3], b[1], b[3]};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float y0 = x0[j] * c[j] - x1[j] * sn[j];
      const float y1 = x1[j] * c[j] + x0[j] * sn[j];
      x0[j] = y0;
      x1[j] = y1;
    }
  }
  T* dst;
  if (hs < nh) {
    dst = q + (long)r * nh * d + hs * d;
  } else if (hs < nh + nkv) {
    dst = kc + ((long)(hs - nh) * cache_rows + row_tok[r]) * d;
  } else {
    dst = vc + ((long)(hs - nh - nkv) * cache_rows + row_tok[r]) * d;
  }
  store4(dst + i, x0[0], x0[1], x0[2], x0[3]);
  store4(dst + i + half, x1[0], x1[1], x1[2], x1[3]);
}

template <typename T>
hipError_t qkv_epilogue(const float* C, int S, int M, const T* bias, const float* rope_cs,
                        const int32_t* row_pos, const int32_t* row_tok, int n_heads, int n_kv,
                        int head_dim, T* q, T* kcache, T* vcache, long cache_rows, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (head_dim != 64 && head_dim != 128) return hipErrorInvalidValue;
  const int N = (n_heads + 2 * n_kv) * head_dim, per_block = 512 / head_dim;
  const int hblocks = (n_heads + 2 * n_kv + per_block - 1) / per_block;
  hipLaunchKernelGGL(k_qkv_epilogue<T>, dim3(M, hblocks), dim3(64), 0, st, C, S, M, N, bias,
                     rope_cs, row_pos, row_tok, n_heads, n_kv, head_dim, q, kcache, vcache,
                     cache_rows);
  return hipGetLastError();
}

// ---- SwiGLU -----------------------------------------------------------------------------
// Four consecutive features per thread; F is a multiple of 4 (of 8 for bf16).
// bf16 weights are packed with gate and up interleaved by 8 rows
// (kPackGateUp): gate feature f is GEMM column (f/8)*16 + f%8, up feature f
// is 8 columns later; fp32 weights are gate then up.
template <typename T>
__global__ void k_swiglu(const float* __restrict__ C, int S, int M, int F, T* __restrict__ out) {
  const long total = (long)M * F / 4;
  for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long)gridDim.x * blockDim.x) {
    const long r = e / (F / 4);
    const int f = (int)(e - r * (F / 4)) * 4;
    const int gcol = sizeof(T) == 2 ? (f >> 3) * 16 + (f & 7) : f;
    const int ucol = sizeof(T) == 2 ? gcol + 8 : F + f;
    const float* cr = C + r * (2L * F);
    f32x4 g, u;
    split_sum2((const f32x4*)(cr + gcol), (const f32x4*)(cr + ucol), (long)M * F / 2, S, g, u);
#pragma unroll
    for (int q = 0; q < 4; ++q) out[r * F + f + q] = Elem<T>::from_f(g[q] / (1.0f + expf(-g[q])) * u[q]);
  }
}

template <typename T>
hipError_t swiglu(const float* C, int S, int M, int F, T* out, hipStream_t st) {
  if (M <= 0) return hipSuccess;
  if (F % (sizeof(T) == 2 ? 8 : 4)) return hipErrorInvalidValue;
  const long total = (long)M * F / 4;
  const int blocks = (int)std::min<long>((total + 255) / 256, 8192);
  hipLaunchKernelGGL(k_swiglu<T>, dim3(blocks), dim3(256), 0, st, C, S, M, F, out);
  return hipGetLastError();
}

// ---- attention, fp32 models: one wave per (row, head) ------------------------------------
// Scores for keys lane, lane + 64, ... are kept in LDS (dynamic, ctx floats).
__global__ __launch_bounds__(64) void k_attn_f32(const float* __restrict__ q,
                                                 const float* __restrict__ kc,
                                                 const float* __restrict__ vc, long cache_rows,
                                                 float* __restrict__ o,
                                                 const int32_t* __restrict__ row_seq,
                                                 WdStepGeom g, int nh, int nkv, int d) {
  extern __shared__ float p[];
  __shared__ float qs[128];
  const int r = blockIdx.x, h = blockIdx.y, lane = threadIdx.x;
  const int b = row_seq[r];
  const int c = g.ctx[b];
  const long off = g.off[b];
  const int kvh = h / (nh / nkv);
  const float* kb = kc + ((long)kvh * cache_rows + off) * d;
  const float* vb = vc + ((long)kvh * cache_rows + off) * d;
  for (int i = lane; i < d; i += 64) qs[i] = q[(long)r * nh * d + h * d + i];
  __syncthreads();
  const float scale = 1.0f / sqrtf((float)d);
  float mx = -INFINITY;
  for (int j = lane; j < c; j += 64) {
    const float* kr = kb + (long)j * d;
    float s = 0.f;
    for (int i = 0; i < d; ++i) s = fmaf(qs[i], kr[i], s);
    s *= scale;
    p[j] = s;
    mx = fmaxf(mx, s);
  }
  mx = wave_max(mx);
  float sum = 0.f;
  for (int j = lane; j < c; j += 64) {
    const float e = expf(p[j] - mx);
    p[j] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  __syncthreads();
  for (int i = lane; i < d; i += 64) {
    float acc = 0.f;
    for (int j = 0; j < c; ++j) acc = fmaf(p[j], vb[(long)j * d + i], acc);
    o[(long)r * nh * d + h * d + i] = acc / sum;
  }
}

// ---- attention, bf16 models: flash-style with MFMA (head_dim 128) ----------------------------
// Workgroup = (query head, sequence, block of 64 query rows); wave w owns 16
// query rows.  Keys go in tiles of 64 through LDS: K row-major (A operand of
// S^T = K Q^T) and V transposed (A operand of O^T = V^T P^T), so the scores
// stay in registers in exactly the layout the second product needs.  Softmax
// runs online in fp32; P enters the bf16 MFMA as hi + lo bf16 parts, which
// keeps P V at fp32-level accuracy.
//
// Key order inside a tile: key = 16 kq + k16 sits at V^T position 4 k16 + kq,
// so a thread that loaded keys t, t + 16, t + 32, t + 48 writes each of its
// dims as one 8-byte store.  Row r of score subtile st is key
// pi(st, r) = 16 (r % 4) + 8 (st / 2) + 2 (r / 4) + st % 2 (K is stored at that
// row), which puts in each lane exactly the scores its P operand needs for the
// V^T positions it multiplies.  V^T rows are 64 keys (8 chunks of 16 bytes);
// chunk j of dim d is stored at chunk j ^ ((d / 8) % 8), which spreads both
// the stores and the 16-byte operand reads over the banks.
constexpr int kAttD = 128;
constexpr int kKT = 64;              // keys per tile
constexpr int kKPitch = kAttD + 8;   // bf16 elements per K row in LDS
constexpr int kVPitch = kKT;         // bf16 elements per V^T row in LDS (swizzled chunks)
constexpr int kMaxSplit = 16;        // most key splits of one attention launch

// Split-KV: blockIdx.z = query block * nsplit + split; split s covers keys
// [s * keys_per_split, (s + 1) * keys_per_split) of [0, c).  With nsplit == 1
// the normalized output is written as bf16; otherwise the unnormalized fp32
// output and the running max / sum go to part / ml for k_attn_combine.
__global__ __launch_bounds__(256) void k_attn_bf16(const uint16_t* __restrict__ q,
                                                   const uint16_t* __restrict__ kc,
                                                   const uint16_t* __restrict__ vc,
                                                   long cache_rows, uint16_t* __restrict__ o,
                                                   WdStepGeom g, int nh, int nkv, int nsplit,
                                                   int keys_per_split, int M,
                                                   float* __restrict__ part,
                                                   float* __restrict__ ml) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKT * kKPitch];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kAttD * kVPitch];
  const int h = blockIdx.x, b = blockIdx.y;
  const int qb = blockIdx.z / nsplit, split = blockIdx.z % nsplit;
  const int nq = g.nrows[b];
  if (qb * 64 >= nq) return;
  const int key_lo = split * keys_per_split;
  const int c = min(g.ctx[b], key_lo + keys_per_split);
  const long off = g.off[b];
  const int row0 = g.row0[b];
  const int kvh = h / (nh / nkv);
  const uint16_t* kb = kc + ((long)kvh * cache_rows + off) * kAttD;
  const uint16_t* vb = vc + ((long)kvh * cache_rows + off) * kAttD;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l16 = lane & 15, grp = lane >> 4;
  const int qi = qb * 64 + wave * 16 + l16;  // this lane's query (column of S^T / O^T)
  const bool qvalid = qi < nq;
  const bool wave_active = qb * 64 + wave * 16 < nq;
  const long ldq = (long)nh * kAttD;

  u32x4 qf[4];
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int cc = 0; cc < 4; ++cc)
    qf[cc] = qvalid ? *(const u32x4*)(q + (long)(row0 + qi) * ldq + h * kAttD + cc * 32 + grp * 8)
                    : zero4;

  f32x4 oacc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) oacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)

  // K/V tile of 64 keys x 256 B each: thread tid covers keys (tid >> 4) + 16 i,
  // 16-byte chunk tid & 15 (dims 8 (tid & 15) ..).  The next tile's loads are
  // issued before the current tile is computed; addresses are clamped to the
  // last key and the keys past c are zeroed when the tile is stored.
  const int tkey = tid >> 4, tch = tid & 15;
  u32x4 kr[4], vr[4];
  auto load_tile = [&](int j0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const long kk = min(j0 + tkey + 16 * i, c - 1);
      kr[i] = *(const u32x4*)(kb + kk * kAttD + tch * 8);
      vr[i] = *(const u32x4*)(vb + kk * kAttD + tch * 8);
    }
  };
  if (key_lo < c) load_tile(key_lo);
  for (int j0 = key_lo; j0 < c; j0 += kKT) {
    __syncthreads();
    // K rows at the score row that holds them; V^T dims as 4-key runs
    u32x4 vv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = tkey + 16 * i;  // k16 = tkey, kq = i
      const bool ok = j0 + key < c;
      const u32x4 kv = ok ? kr[i] : zero4;
      vv[i] = ok ? vr[i] : zero4;
      const int st = 2 * (tkey >> 3) + (tkey & 1), r = 4 * ((tkey >> 1) & 3) + i;
      *(u32x4*)(Ks + (st * 16 + r) * kKPitch + tch * 8) = kv;
    }
    {
      const int chunk = (tkey >> 1) ^ (tch & 7);  // dims tch * 8 .. have d / 8 = tch
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int sh = 16 * (e & 1);
        u32x2 w;
        w.x = ((vv[0][e >> 1] >> sh) & 0xffffu) | (((vv[1][e >> 1] >> sh) & 0xffffu) << 16);
        w.y = ((vv[2][e >> 1] >> sh) & 0xffffu) | (((vv[3][e >> 1] >> sh) & 0xffffu) << 16);
        *(u32x2*)(Vt + (tch * 8 + e) * kVPitch + chunk * 8 + (tkey & 1) * 4) = w;
      }
    }
    __syncthreads();
    load_tile(min(j0 + kKT, c - 1));
    if (!wave_active) continue;

    // S^T[key][query] for 4 subtiles of 16 keys
    f32x4 sacc[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      sacc[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        const u32x4 ka = *(const u32x4*)(Ks + (st * 16 + l16) * kKPitch + cc * 32 + grp * 8);
        sacc[st] = mfma16(ka, qf[cc], sacc[st]);
      }
    }
    // this lane holds keys pi(st, grp * 4 + jj) for query l16
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int key = j0 + 16 * jj + 8 * (st >> 1) + 2 * grp + (st & 1);
        const float s = key < c ? sacc[st][jj] * scale : -INFINITY;
        sacc[st][jj] = s;
        tmax = fmaxf(tmax, s);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float corr = expf(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const float pv = expf(sacc[st][jj] - m_new);
        sacc[st][jj] = pv;
        psum += pv;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * corr + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[i] *= corr;

    // O^T += V^T P^T over two 32-position chunks (subtiles 2pc, 2pc+1)
#pragma unroll
    for (int pc = 0; pc < 2; ++pc) {
      // element e of lane grp's fragment is V^T position 32 pc + 8 grp + e, the key
      // of score subtile 2 pc + e / 4, row grp * 4 + e % 4
      u32x4 bhi, blo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4& sp = sacc[2 * pc + (i >> 1)];
        const float p0 = sp[(2 * i) & 3], p1 = sp[(2 * i + 1) & 3];
        const uint16_t h0 = f2bf(p0), h1 = f2bf(p1);
        bhi[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        blo[i] = (uint32_t)f2bf(p0 - bf2f(h0)) | ((uint32_t)f2bf(p1 - bf2f(h1)) << 16);
      }
#pragma unroll
      for (int df = 0; df < 8; ++df) {
        const int d = df * 16 + l16;
        const u32x4 va = *(const u32x4*)(Vt + d * kVPitch + (((4 * pc + grp) ^ ((d >> 3) & 7)) * 8));
        oacc[df] = mfma16(va, bhi, oacc[df]);
        oacc[df] = mfma16(va, blo, oacc[df]);
      }
    }
  }
  if (!qvalid) return;
  if (nsplit > 1) {
    const long pr = ((long)split * M + row0 + qi) * nh + h;
    float* prow = part + pr * kAttD;
#pragma unroll
    for (int df = 0; df < 8; ++df) *(f32x4*)(prow + df * 16 + grp * 4) = oacc[df];
    if (grp == 0) {
      ml[pr * 2] = m_run;
      ml[pr * 2 + 1] = l_run;
    }
    return;
  }
  const float inv = 1.0f / l_run;
  uint16_t* orow = o + (long)(row0 + qi) * ldq + h * kAttD;
#pragma unroll
  for (int df = 0; df < 8; ++df) {
    u32x2 w;
    w.x = (uint32_t)f2bf(oacc[df][0] * inv) | ((uint32_t)f2bf(oacc[df][1] * inv) << 16);
    w.y = (uint32_t)f2bf(oacc[df][2] * inv) | ((uint32_t)f2bf(oacc[df][3] * inv) << 16);
    *(u32x2*)(orow + df * 16 + grp * 4) = w;
  }
}

// Grouped K/V heads (n_kv < n_heads) with many rows per sequence (refresh
// steps): the same computation with one workgroup per (K/V head, block of
// 16 NWQ columns), a column being a (query head of the group, row) pair, so
// that every K/V tile a workgroup stages serves all the query heads that
// read it.  The first 256 threads stage the tiles as above.  Measured at the
// Dream-7B shape (28 query / 4 K/V heads), isolated: 600 rows x 600 keys
// 40.5 us (8 waves, no key split) against 51.5 us per query head; at
// normal-step shapes (34-46 rows x 416-768 keys, 0.85-1.6 MB of K/V per
// layer) grouping does not pay (0.95-1.01x at every split count tried): the
// kernel is bound by the latency of its few tile steps there, not by loads.
template <int NWQ>
__global__ __launch_bounds__(64 * NWQ) void k_attn_bf16_grouped(const uint16_t* __restrict__ q,
                                                   const uint16_t* __restrict__ kc,
                                                   const uint16_t* __restrict__ vc,
                                                   long cache_rows, uint16_t* __restrict__ o,
                                                   WdStepGeom g, int nh, int nkv, int nsplit,
                                                   int keys_per_split, int M,
                                                   float* __restrict__ part,
                                                   float* __restrict__ ml) {
  __shared__ __attribute__((aligned(16))) uint16_t Ks[kKT * kKPitch];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[kAttD * kVPitch];
  // blockIdx.x = K/V head; the columns of a workgroup are (query head of the
  // group, row) pairs, head-major: column i is head kvh * G + i / nq, row i % nq
  const int kvh = blockIdx.x, b = blockIdx.y;
  const int qb = blockIdx.z / nsplit, split = blockIdx.z % nsplit;
  const int nq = g.nrows[b];
  const int G = nh / nkv, ncol = G * nq;
  constexpr int QB = 16 * NWQ;
  if (qb * QB >= ncol) return;
  const int key_lo = split * keys_per_split;
  const int c = min(g.ctx[b], key_lo + keys_per_split);
  const long off = g.off[b];
  const int row0 = g.row0[b];
  const uint16_t* kb = kc + ((long)kvh * cache_rows + off) * kAttD;
  const uint16_t* vb = vc + ((long)kvh * cache_rows + off) * kAttD;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l16 = lane & 15, grp = lane >> 4;
  const int col = qb * QB + wave * 16 + l16;  // this lane's column of S^T / O^T
  const bool qvalid = col < ncol;
  const int h = kvh * G + (qvalid ? col / nq : 0), qi = qvalid ? col % nq : 0;
  const bool wave_active = qb * QB + wave * 16 < ncol;
  const bool loader = tid < 256;  // the first 256 threads stage the K/V tiles
  const long ldq = (long)nh * kAttD;

  u32x4 qf[4];
  const u32x4 zero4 = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int cc = 0; cc < 4; ++cc)
    qf[cc] = qvalid ? *(const u32x4*)(q + (long)(row0 + qi) * ldq + h * kAttD + cc * 32 + grp * 8)
                    : zero4;

  f32x4 oacc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) oacc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;
  const float scale = 0.08838834764831845f;  // 1/sqrt(128)

  // K/V tile of 64 keys x 256 B each: thread tid covers keys (tid >> 4) + 16 i,
  // 16-byte chunk tid & 15 (dims 8 (tid & 15) ..).  The next tile's loads are
  // issued before the current tile is computed; addresses are clamped to the
  // last key and the keys past c are zeroed when the tile is stored.
  const int tkey = tid >> 4, tch = tid & 15;
  u32x4 kr[4], vr[4];
  auto load_tile = [&](int j0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const long kk = min(j0 + tkey + 16 * i, c - 1);
      kr[i] = *(const u32x4*)(kb + kk * kAttD + tch * 8);
      vr[i] = *(const u32x4*)(vb + kk * kAttD + tch * 8);
    }
  };
  if (loader && key_lo < c) load_tile(key_lo);
  for (int j0 = key_lo; j0 < c; j0 += kKT) {
    __syncthreads();
    if (loader) {
    // K rows at the score row that holds them; V^T dims as 4-key runs
    u32x4 vv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int key = tkey + 16 * i;  // k16 = tkey, kq = i
      const bool ok = j0 + key < c;
      const u32x4 kv = ok ? kr[i] : zero4;
      vv[i] = ok ? vr[i] : zero4;
      const int st = 2 * (tkey >> 3) + (tkey & 1), r = 4 * ((tkey >> 1) & 3) + i;
      *(u32x4*)(Ks + (st * 16 + r) * kKPitch + tch * 8) = kv;
    }
    {
      const int chunk = (tkey >> 1) ^ (tch & 7);  // dims tch * 8 .. have d / 8 = tch
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int sh = 16 * (e & 1);
        u32x2 w;
        w.x = ((vv[0][e >> 1] >> sh) & 0xffffu) | (((vv[1][e >> 1] >> sh) & 0xffffu) << 16);
        w.y = ((vv[2][e >> 1] >> sh) & 0xffffu) | (((vv[3][e >> 1] >> sh) & 0xffffu) << 16);
        *(u32x2*)(Vt + (tch * 8 + e) * kVPitch + chunk * 8 + (tkey & 1) * 4) = w;
      }
    }
    }
    __syncthreads();
    if (loader) load_tile(min(j0 + kKT, c - 1));
    if (!wave_active) continue;

    // S^T[key][query] for 4 subtiles of 16 keys
    f32x4 sacc[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) {
      sacc[st] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int cc = 0; cc < 4; ++cc) {
        const u32x4 ka = *(const u32x4*)(Ks + (st * 16 + l16) * kKPitch + cc * 32 + grp * 8);
        sacc[st] = mfma16(ka, qf[cc], sacc[st]);
      }
    }
    // this lane holds keys pi(st, grp * 4 + jj) for query l16
    float tmax = -INFINITY;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const int key = j0 + 16 * jj + 8 * (st >> 1) + 2 * grp + (st & 1);
        const float s = key < c ? sacc[st][jj] * scale : -INFINITY;
        sacc[st][jj] = s;
        tmax = fmaxf(tmax, s);
      }
    tmax = fmaxf(tmax, __shfl_xor(tmax, 16, 64));
    tmax = fmaxf(tmax, __shfl_xor(tmax, 32, 64));
    const float m_new = fmaxf(m_run, tmax);
    const float corr = expf(m_run - m_new);
    float psum = 0.f;
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const float pv = expf(sacc[st][jj] - m_new);
        sacc[st][jj] = pv;
        psum += pv;
      }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    l_run = l_run * corr + psum;
    m_run = m_new;
#pragma unroll
    for (int i = 0; i < 8; ++i) oacc[i] *= corr;

    // O^T += V^T P^T over two 32-position chunks (subtiles 2pc, 2pc+1)
#pragma unroll
    for (int pc = 0; pc < 2; ++pc) {
      // element e of lane grp's fragment is V^T position 32 pc + 8 grp + e, the key
      // of score subtile 2 pc + e / 4, row grp * 4 + e % 4
      u32x4 bhi, blo;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4& sp = sacc[2 * pc + (i >> 1)];
        const float p0 = sp[(2 * i) & 3], p1 = sp[(2 * i + 1) & 3];
        const uint16_t h0 = f2bf(p0), h1 = f2bf(p1);
        bhi[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
        blo[i] = (uint32_t)f2bf(p0 - bf2f(h0)) | ((uint32_t)f2bf(p1 - bf2f(h1)) << 16);
      }
#pragma unroll
      for (int df = 0; df < 8; ++df) {
        const int d = df * 16 + l16;
        const u32x4 va = *(const u32x4*)(Vt + d * kVPitch + (((4 * pc + grp) ^ ((d >> 3) & 7)) * 8));
        oacc[df] = mfma16(va, bhi, oacc[df]);
        oacc[df] = mfma16(va, blo, oacc[df]);
      }
    }
  }
  if (!qvalid) return;
  if (nsplit > 1) {
    const long pr = ((long)split * M + row0 + qi) * nh + h;
    float* prow = part + pr * kAttD;
#pragma unroll
    for (int df = 0; df < 8; ++df) *(f32x4*)(prow + df * 16 + grp * 4) = oacc[df];
    if (grp == 0) {
      ml[pr * 2] = m_run;
      ml[pr * 2 + 1] = l_run;
    }
    return;
  }
  const float inv = 1.0f / l_run;
  uint16_t* orow = o + (long)(row0 + qi) * ldq + h * kAttD;
#pragma unroll
  for (int df = 0; df < 8; ++df) {
    u32x2 w;
    w.x = (uint32_t)f2bf(oacc[df][0] * inv) | ((uint32_t)f2bf(oacc[df][1] * inv) << 16);
    w.y = (uint32_t)f2bf(oacc[df][2] * inv) | ((uint32_t)f2bf(oacc[df][3] * inv) << 16);
    *(u32x2*)(orow + df * 16 + grp * 4) = w;
  }
}

// out = sum_s exp(m_s - m) O_s / sum_s exp(m_s - m) l_s, m = max_s m_s.
// Workgroup (h, r) of the (nh, M) grid runs on the XCD (linear id mod 8) that
// ran every split of head h when nh is a multiple of 8, so the partials it
// reads were written through its own L2.
__global__ __launch_bounds__(128) void k_attn_combine(const float* __restrict__ part,
                                                      const float* __restrict__ ml, int nsplit,
                                                      int M, int nh, uint16_t* __restrict__ o) {
  const int h = blockIdx.x, r = blockIdx.y, dd = threadIdx.x;
  // every split's (m, l, O) in flight at once; nsplit <= kMaxSplit, and only
  // the splits that exist are loaded (nsplit is uniform, so are the branches)
  float ms[kMaxSplit], ls[kMaxSplit], os[kMaxSplit];
#pragma unroll
  for (int s = 0; s < kMaxSplit; ++s) {
    ms[s] = -INFINITY;
    ls[s] = os[s] = 0.f;
    if (s < nsplit) {
      const long pr = ((long)s * M + r) * nh + h;
      ms[s] = ml[pr * 2];
      ls[s] = ml[pr * 2 + 1];
      os[s] = part[pr * kAttD + dd];
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int s = 0; s < kMaxSplit; ++s)
    if (s < nsplit) mx = fmaxf(mx, ms[s]);
  float l = 0.f, acc = 0.f;
#pragma unroll
  for (int s = 0; s < kMaxSplit; ++s)
    if (s < nsplit) {
      const float w = expf(ms[s] - mx);
      l += w * ls[s];
      acc += w * os[s];
    }
  o[((long)r * nh + h) * kAttD + dd] = f2bf(acc / l);
}

hipError_t attention_bf16(const uint16_t* q, const uint16_t* kcache, const uint16_t* vcache,
                          long cache_rows, uint16_t* o, const WdStepGeom& g, int n_heads, int n_kv,
                          int head_dim, float* part, long part_floats, hipStream_t st,
                          hipEvent_t e0, hipEvent_t e1) {
  if (head_dim != kAttD) return hipErrorInvalidValue;
  int nqmax = 0, cmax = 0, M = 0;
  long qblocks = 0;
  for (int b = 0; b < g.batch; ++b) {
    nqmax = std::max(nqmax, g.nrows[b]);
    cmax = std::max(cmax, g.ctx[b]);
    M = std::max(M, g.row0[b] + g.nrows[b]);
    qblocks += (g.nrows[b] + 63) / 64;
  }
  if (nqmax <= 0) return hipSuccess;
  if (n_kv < n_heads && nqmax >= 256) {
    // refresh-step rows with grouped K/V heads: each staged tile serves the
    // group's query heads; no key split (so no merge)
    constexpr int NWQ = 8;
    const int G = n_heads / n_kv;
    const int blocks = (G * nqmax + 16 * NWQ - 1) / (16 * NWQ);
    const int tiles = (cmax + kKT - 1) / kKT;
    dim3 grid(n_kv, g.batch, blocks);
    if (e0)
      hipExtLaunchKernelGGL(k_attn_bf16_grouped<NWQ>, grid, dim3(64 * NWQ), 0, st, e0, e1, 0, q,
                            kcache, vcache, cache_rows, o, g, n_heads, n_kv, 1, tiles * kKT, M,
                            part, part);
    else
      hipLaunchKernelGGL(k_attn_bf16_grouped<NWQ>, grid, dim3(64 * NWQ), 0, st, q, kcache, vcache,
                         cache_rows, o, g, n_heads, n_kv, 1, tiles * kKT, M, part, part);
    return hipGetLastError();
  }
  // split the keys until about 512 workgroups run, into at most 8 splits, if
  // the partial buffer allows.  Measured (isolated, 32 heads): 16 one-tile
  // splits cost more than 8 two-tile ones (1024 keys: 20.8 against 17.4 us at
  // 64 rows, 16.1 against 14.8 at 34), the combine reading every split.  But
  // once the unsplit grid has 128 workgroups (refresh-step rows), splitting
  // costs more than it parallelizes: 32 heads, rows x keys 224 x 224 17.1 us
  // unsplit against 21.7, 384 x 384 23.1 against 33.4, 832 x 832 55.4
  // against 72.2 (2 splits).
  const int tiles = (cmax + kKT - 1) / kKT;
  int nsplit = n_heads * qblocks >= 128
                   ? 1
                   : std::min<long>(tiles, std::max<long>(1, (512 + n_heads * qblocks - 1) /
                                                                 (n_heads * qblocks)));
  nsplit = std::min(nsplit, std::min(kMaxSplit, 8));
  while (nsplit > 1 && (long)nsplit * M * n_heads * (kAttD + 2) > part_floats) --nsplit;
  const int tps = (tiles + nsplit - 1) / nsplit;
  nsplit = (tiles + tps - 1) / tps;
  float* ml = part + (long)nsplit * M * n_heads * kAttD;
  dim3 grid(n_heads, g.batch, ((nqmax + 63) / 64) * nsplit);
  // with events, e0 is recorded by the first launch's dispatch and e1 by the last one's
  if (e0) {
    hipExtLaunchKernelGGL(k_attn_bf16, grid, dim3(256), 0, st, e0, nsplit > 1 ? nullptr : e1, 0, q,
                          kcache, vcache, cache_rows, o, g, n_heads, n_kv, nsplit, tps * kKT, M,
                          part, ml);
    if (nsplit > 1)
      hipExtLaunchKernelGGL(k_attn_combine, dim3(n_heads, M), dim3(kAttD), 0, st, nullptr, e1, 0,
                            (const float*)part, (const float*)ml, nsplit, M, n_heads, o);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_attn_bf16, grid, dim3(256), 0, st, q, kcache, vcache, cache_rows, o, g,
                     n_heads, n_kv, nsplit, tps * kKT, M, part, ml);
  if (nsplit > 1)
    hipLaunchKernelGGL(k_attn_combine, dim3(n_heads, M), dim3(kAttD), 0, st, part, ml, nsplit, M,
                       n_heads, o);
  return hipGetLastError();
}

hipError_t attention_f32(const float* q, const float* kcache, const float* vcache, long cache_rows,
                         float* o, const int32_t* row_seq, int M, const WdStepGeom& g, int n_heads,
                         int n_kv, int head_dim, hipStream_t st) {
  int cmax = 0;
  for (int b = 0; b < g.batch; ++b) cmax = std::max(cmax, g.ctx[b]);
  if (M <= 0) return hipSuccess;
  if (head_dim > 128 || cmax > 16384) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_attn_f32, dim3(M, n_heads), dim3(64), cmax * sizeof(float), st, q, kcache,
                     vcache, cache_rows, o, row_seq, g, n_heads, n_kv, head_dim);
  return hipGetLastError();
}

// ---- fp32 copies for debugging --------------------------------------------------------------
template <typename T>
__global__ void k_widen(const T* __restrict__ src, long stride, float* __restrict__ dst, int rows,
                        int cols) {
  const long total = (long)rows * cols;
  for (long e = (long)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (long)gridDim.x * blockDim.x) {
    const long r = e / cols;
    dst[e] = Elem<T>::to_f(src[r * stride + (e - r * cols)]);
  }
}

template <typename T>
hipError_t widen_rows(const T* src, long src_stride, float* dst, int rows, int cols,
                      hipStream_t st) {
  const long total = (long)rows * cols;
  if (total <= 0) return hipSuccess;
  const int blocks = (int)std::min<long>((total + 255) / 256, 4096);
  hipLaunchKernelGGL(k_widen<T>, dim3(blocks), dim3(256), 0, st, src, src_stride, dst, rows, cols);
  return hipGetLastError();
}

#define WD_INSTANTIATE(T)                                                                       \
  template hipError_t embed_norm<T>(const int32_t*, const int32_t*, const T*, const T*, float,   \
                                    float*, T*, int, int, hipStream_t);                          \
  template hipError_t residual_norm<T>(float*, const float*, int, int, int, const T*, float, T*, \
                                       const int32_t*, hipStream_t);                             \
  template hipError_t qkv_epilogue<T>(const float*, int, int, const T*, const float*,            \
                                      const int32_t*, const int32_t*, int, int, int, T*, T*, T*, \
                                      long, hipStream_t);                                        \
  template hipError_t swiglu<T>(const float*, int, int, int, T*, hipStream_t);                   \
  template hipError_t widen_rows<T>(const T*, long, float*, int, int, hipStream_t);
WD_INSTANTIATE(float)
WD_INSTANTIATE(uint16_t)

}  // namespace wd
