// Host-side launch wrappers of the libwd kernels.  Every wrapper enqueues
// on the given stream and returns the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "common.h"

namespace wd {

// ---- GEMM (gemm.hip) -------------------------------------------------------------
struct GemmPlan {
  int nf = 1;            // 16-row weight groups per wave
  int mf = 4;            // 16-row activation fragments per row tile
  int ck = 8;            // 32-wide K steps per LDS activation chunk
  int splits = 1;        // K splits = number of partial outputs
  int ks_per_split = 0;  // 32-wide K steps per split
  int grid = 0;
  int dma_mfw = 0;       // > 0: k_gemm_bf16_dma with 64 * dma_mfw-row tiles
  int dma_tnb = 8;       // its 32-feature blocks per tile: 8, 6 or 4 (256, 192, 128 features)
  int dma_nw = 0;        // its waves per workgroup: 12 (192 features), 8, or 4 (256 x 256 tiles,
                         // operand reads pinned ahead of the MFMAs)
  int dma_gm = 0;        // > 0: its workgroups in bands of dma_gm row tiles
  int fused_gw = 0;      // > 0: gemm_bf16_split_fused with fused_gw groups per workgroup
};
// Launch plan for C = X W^T; at most max_splits K splits.
GemmPlan plan_gemm_bf16(int M, int N, int K, bool w8 = false, int max_splits = 1 << 20);
// Whether plan p can run C = X W^T (M x K by K x N; w8: fp8 weights; swiglu:
// the many-row kernel's SwiGLU epilogue, which needs all of K in one
// workgroup).  gemm_bf16 and gemm_bf16_swiglu_dma reject plans for which
// this is false.
bool gemm_plan_ok(const GemmPlan& p, int M, int N, int K, bool w8, bool swiglu);
// Where the Q/K/V projection's epilogue in the many-row kernel puts its
// results (bf16 models, head_dim 128, weights packed kPackRopePair): bias
// (null without), the RoPE table [position][64][cos, sin], each row's
// position and K/V cache row, q [M][nh][128], and this layer's K and V cache
// [nkv][cache_rows][128].
struct QkvOut {
  const uint16_t* bias;
  const float* rope;
  const int32_t* row_pos;
  const int32_t* row_tok;
  uint16_t* q;
  uint16_t* kc;
  uint16_t* vc;
  long cache_rows;
  int nh, nkv;
};
// The many-row kernel (gemm_tiles.hip) for plan p (p.dma_mfw > 0, checked by
// gemm_plan_ok): split-K partials into C; with swiglu_out the SwiGLU
// epilogue; with qkv the Q/K/V epilogue (both need p.splits == 1).  False if
// the plan names no instance or does not fit the epilogue.
bool launch_gemm_tiles(const GemmPlan& p, const uint16_t* X, int ldx, const void* Wp, float* C,
                       int M, int N, int K, uint16_t* swiglu_out, hipStream_t st, hipEvent_t e0,
                       hipEvent_t e1, const QkvOut* qkv = nullptr);
// Many-row Q/K/V product with its epilogue in the kernel: p must be a
// k_gemm_bf16_dma plan without a K split for (M, N, K), N = (nh + 2 nkv) 128.
hipError_t gemm_bf16_qkv_tiles(const uint16_t* X, int ldx, const void* Wp, int M, int N, int K,
                               const GemmPlan& p, const QkvOut& qo, hipStream_t st,
                               hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
// The kernel plan p launches (1 pipelined few-row kernel with K-split
// partials, 2 the many-row LDS-pipelined kernel, 3 the split-K tiled kernel)
// and its workgroup tile and waves.
void gemm_plan_tile(const GemmPlan& p, int* kernel, int* rows, int* features, int* waves);
// Row orders of packed weights (gemm.hip): plain; RoPE pairs adjacent within
// each 128-row head (Q/K/V); gate and up interleaved by 8 rows (W2 = up).
constexpr int kPackPlain = 0, kPackRopePair = 1, kPackGateUp = 2;
hipError_t pack_frags(const uint16_t* W, int N, int K, void* out, hipStream_t st,
                      int perm = kPackPlain, const uint16_t* W2 = nullptr);
// FP8-weight variant: per-row scales (in packed row order) and e4m3 fragments
// of 16 rows x 64 K columns (N x K bytes); K a multiple of 64.
hipError_t pack_fp8(const uint16_t* W, int N, int K, void* out, float* scale, hipStream_t st,
                    int perm = kPackPlain, const uint16_t* W2 = nullptr);
// Few-row products with their epilogue in the kernel (no K split), for
// M <= fused_max_rows rows when N / 64 >= 192 (fused_rows_ok).  Q/K/V: weights packed
// kPackRopePair, head_dim 128; writes q [M][nh][128] and the k/v cache rows
// row_tok of each head.  SwiGLU: weights packed kPackGateUp (N = 2F);
// writes out [M][F] = silu(gate) * up.
constexpr int kEpiQkv = 1, kEpiSwiGlu = 2, kEpiConf = 3, kEpiPartial = 4;
// Most rows of the fused products: 96 for gate/up (at 66-94 rows it beats the
// 128-row tiles: 38.7-47.0 us against 44.0-47.4), 64 for Q/K/V and the LM head
// (the 128-row tiles win there above 64 rows: Q/K/V 26-29 us against 29-40).
constexpr int fused_max_rows(int epi) { return epi == kEpiSwiGlu ? 96 : 64; }
bool fused_rows_ok(int M, int N, int K, int max_rows = 64);
// Many-row gate/up with SwiGLU in the epilogue: p must be a k_gemm_bf16_dma
// plan without a K split for (M, 2F, K); weights packed kPackGateUp; writes
// out [M][F] = silu(gate) * up.
hipError_t gemm_bf16_swiglu_dma(const uint16_t* X, int ldx, const void* Wp, uint16_t* out, int M,
                                int F, int K, const GemmPlan& p, hipStream_t st,
                                hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);
// The same pipelined few-row kernel over K splits (1 <= M <= 64): gw 16-row
// weight groups per workgroup (2, 3, 4 or 6; N / 16 a multiple of it), split
// s covering K steps [s ks, s ks + ks); writes C[s][m][n] fp32 like gemm_bf16.
hipError_t gemm_bf16_split_fused(const uint16_t* X, int ldx, const void* Wp, float* C, int M,
                                 int N, int K, int gw, int splits, int ks, hipStream_t st,
                                 hipEvent_t e0, hipEvent_t e1, const float* wsc);
hipError_t gemm_bf16_qkv_fused(const uint16_t* X, int ldx, const void* Wp, int M, int N, int K,
                               const uint16_t* bias, const float* rope_cs, const int32_t* row_pos,
                               const int32_t* row_tok, int nh, int nkv, uint16_t* q, uint16_t* kc,
                               uint16_t* vc, long cache_rows, hipStream_t st,
                               hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr,
                               const float* wsc = nullptr);
// LM head with the confidence reduction in the kernel: per row and 64-entry
// vocabulary tile, (max logit, lowest id reaching it, sum exp(l - max)),
// [MASK] excluded, at [row][tile] of pmax / pidx / psum (V / 64 tiles);
// logits [M][V] are written only if non-null.  confidence_tiles merges them.
hipError_t gemm_bf16_lmhead_conf(const uint16_t* X, int ldx, const void* Wp, int M, int V, int K,
                                 int mask_id, float* logits, float* pmax, int* pidx, float* psum,
                                 hipStream_t st, hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr,
                                 const float* wsc = nullptr);
hipError_t gemm_bf16_swiglu_fused(const uint16_t* X, int ldx, const void* Wp, int M, int F, int K,
                                  uint16_t* out, hipStream_t st, hipEvent_t e0 = nullptr,
                                  hipEvent_t e1 = nullptr, const float* wsc = nullptr);
// ev_start / ev_stop (optional, both or neither): recorded by the launch itself.
// wsc: per-row scales of fp8 weights (packed by pack_fp8), null for bf16.
hipError_t gemm_bf16(const uint16_t* X, int ldx, const void* Wp, float* C, int M, int N, int K,
                     const GemmPlan& p, hipStream_t st, hipEvent_t ev_start = nullptr,
                     hipEvent_t ev_stop = nullptr, const float* wsc = nullptr);
hipError_t gemm_f32(const float* X, int ldx, const float* W, float* C, int M, int N, int K,
                    hipStream_t st, hipEvent_t ev_start = nullptr, hipEvent_t ev_stop = nullptr);

// ---- row-wise layer pieces (layer.hip) -------------------------------------------------
// h[r] = emb[x[row_tok[r]]]; a[r] = RMSNorm(h[r]) * gamma
template <typename T>
hipError_t embed_norm(const int32_t* x, const int32_t* row_tok, const T* emb, const T* gamma,
                      float eps, float* h, T* a, int M, int H, hipStream_t st);
// h[r] += sum_s C[s][r]; a[dst(r)] = RMSNorm(h[r]) * gamma, dst(r) = row_out ? row_out[r] : r
// (rows with dst < 0 are not normalized)
template <typename T>
hipError_t residual_norm(float* h, const float* C, int S, int M, int H, const T* gamma, float eps,
                         T* a, const int32_t* row_out, hipStream_t st);
// q/k/v from the QKV partials: bias, RoPE on q and k, store q; k and v go to
// the cache rows row_tok[r] of this layer.
template <typename T>
hipError_t qkv_epilogue(const float* C, int S, int M, const T* bias, const float* rope_cs,
                        const int32_t* row_pos, const int32_t* row_tok, int n_heads, int n_kv,
                        int head_dim, T* q, T* kcache, T* vcache, long cache_rows, hipStream_t st);
// out[r][f] = silu(g) * u with g = sum_s C[s][r][f], u = sum_s C[s][r][F + f]
template <typename T>
hipError_t swiglu(const float* C, int S, int M, int F, T* out, hipStream_t st);
// Non-causal attention of the step's rows over cache rows [0, c) of their
// sequence (rows of sequence b are g.row0[b] .. g.row0[b] + g.nrows[b] - 1).
// `part` (part_floats floats) holds split-KV partials; fewer splits are used
// when it is too small.
hipError_t attention_bf16(const uint16_t* q, const uint16_t* kcache, const uint16_t* vcache,
                          long cache_rows, uint16_t* o, const WdStepGeom& g, int n_heads, int n_kv,
                          int head_dim, float* part, long part_floats, hipStream_t st,
                          hipEvent_t e0 = nullptr, hipEvent_t e1 = nullptr);
hipError_t attention_f32(const float* q, const float* kcache, const float* vcache, long cache_rows,
                         float* o, const int32_t* row_seq, int M, const WdStepGeom& g, int n_heads,
                         int n_kv, int head_dim, hipStream_t st);

// ---- decisions and bookkeeping (decide.hip) -------------------------------------------
// Two passes: kConfChunks vocabulary chunks per row into `scratch`
// (3 * n * kConfChunks floats), then a per-row combine.
constexpr int kConfChunks = 16;
// Achievable dense bf16 MFMA TFLOP/s and HBM read GB/s (4 GiB allocated and
// freed here); synchronizes the stream.
hipError_t measure_peaks(hipStream_t st, double* mfma_tflops, double* read_gbs);

// Merges the per-tile reductions of gemm_bf16_lmhead_conf in tile order.
hipError_t confidence_tiles(const float* pmax, const int* pidx, const float* psum, int n,
                            int n_tiles, int32_t* tok, float* conf, hipStream_t st);
hipError_t confidence(const float* logits, int n, int V, int mask_id, int32_t* tok, float* conf,
                      float* scratch, hipStream_t st);
// Row set of a step, per sequence by g.mode[b]: 0 = refresh ([0, c)),
// 1 = normal (active + phase-decoded positions), 2 = full ([0, c), every
// undecoded position active), 3 = buffer-only refresh (undecoded positions
// of [0, c) + positions decoded in the previous phase), -1 = no rows.  The
// g.nact[b] active rows of sequence b get compact indices b * n_act + rank.
hipError_t build_rows(const uint8_t* decoded, const uint8_t* decoded0, const uint8_t* decoded_prev,
                      int n_act, const WdStepGeom& g, int32_t* row_tok, int32_t* row_pos,
                      int32_t* row_seq, int32_t* row_out, int32_t* act_pos, int32_t* err,
                      hipStream_t st);
// Phase start of the sequences with g.mode[b] == 0: decoded_prev = decoded0,
// decoded0 = decoded over their positions; checks their c against the flags
// below g.end[b].
hipError_t slide(const uint8_t* decoded, uint8_t* decoded0, uint8_t* decoded_prev, int Smax, int E,
                 const WdStepGeom& g, const int32_t* seq_len, int32_t* err, hipStream_t st);
// Top-k decode of each sequence among its n_act candidates; writes tokens,
// decoded flags and the step's selection (b * k + rank).  Sets err bit 2
// when sequence b (g.mode[b] >= 0) decodes other than min(k, g.nact[b])
// positions or a candidate that is already decoded.
hipError_t select_update(const int32_t* act_pos, const int32_t* act_tok, const float* act_conf,
                         int n_act, int k, const WdStepGeom& g, const int32_t* seq_len, int32_t* x,
                         uint8_t* decoded, int32_t* sel_pos, int32_t* sel_tok, float* sel_conf,
                         int32_t* err, hipStream_t st);
// Utility: widen n dtype elements (strided rows) to fp32.
template <typename T>
hipError_t widen_rows(const T* src, long src_stride, float* dst, int rows, int cols, hipStream_t st);

}  // namespace wd
