// Internal declarations shared by the HIP kernels and the host driver of
// libppd.  Device helpers: bfloat16 bit conversions (round to nearest even),
// MFMA operand types, wavefront reductions.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/ppd.h"

typedef uint16_t bf16_t;  // raw bfloat16 storage word
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

#define PPD_WAVE 64

__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// float -> bfloat16, round to nearest, ties to even (NaN stays NaN): the
// gfx950 conversion instruction (v_cvt_pk_bf16_f32) in the default rounding
// mode
typedef __bf16 hw_bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const hw_bf16x2 v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ floatx4 mfma16x16x32(bf16x8 a, bf16x8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, PPD_WAVE);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, PPD_WAVE));
  return v;
}

// ---------------------------------------------------------------------------
// workspace layout (computed on the host, passed to kernels as pointers)

// the first 256 bytes of the workspace hold the status word (offset 0) and a
// 64-byte line of zeros (offset PPD_WS_ZEROS) that is never written
#define PPD_WS_ZEROS 64

struct WsLayout {
  size_t status;      // uint32 [4]
  size_t x;           // float  [T_pad][H]        residual stream
  size_t xg;          // act    [T_pad][H]        x * gain (next norm's operand)
  size_t ss;          // float  [max_ss][T_pad]   sum-of-squares partials
  size_t q;           // act    [T_pad][nh][d]    queries after RoPE
  size_t attn_o;      // act    [T_pad][nh d]     attention output
  size_t act;         // act    [T_pad][F]        SwiGLU output
  size_t tmp;         // float  [T_pad][max(qkv_rows, 2F, V)]  (fp32 path only)
  size_t attn_part;   // float  [nh][max_splits][T_pad][d + 2]
  size_t gemm_part;   // float  [max_part_floats]
  size_t amax;        // float2 [max_amax_tiles][T_pad]
  size_t rope;        // float2 [T_pad][d/2]      (cos, sin)
  size_t total;
  int max_ss, max_splits, max_amax_tiles;
  size_t max_part_floats;
};

#define PPD_ATTN_MAX_SPLITS 64

// ---------------------------------------------------------------------------
// kernel launchers (defined in the .hip files, called by the host driver)

// Skinny GEMM partition.  Tiles of ns row groups of 16 (QKV) or 32 rows
// (ns = 4: 128 rows, QKV 64, half a head; ns = 3 for whole-tile QKV and
// gate/up where that spreads them over more CUs, see gemm_ns_of);
// each tile's K is cut in 64-column chunks, padded with zero chunks to
// kc_pad, a multiple of PPD_GEMM_RING; a group is PPD_GEMM_RING consecutive
// chunks of one tile.
// Unit u = tile * kc_pad + chunk.  Workgroup w of G owns the contiguous
// groups [Ng w / G, Ng (w + 1) / G), Ng = n_tiles * kc_pad / PPD_GEMM_RING,
// so every workgroup streams an equal share and tile boundaries fall between
// groups.  G = n_tiles: one whole tile per workgroup, finished in place;
// otherwise (split) every workgroup stores the partial sums of its tile
// segments and a finish kernel adds them in workgroup order.
#ifndef PPD_GEMM_RING
#define PPD_GEMM_RING 4
#endif
#define PPD_GEMM_BN 128
__host__ __device__ inline long gemm_group_lo(long Ng, int G, int w) { return Ng * w / G; }
// workgroup owning group x
__host__ __device__ inline int gemm_group_owner(long Ng, int G, long x) {
  return (int)(((x + 1) * G - 1) / Ng);
}

// The sequences of one (batched) step: their tree tokens are packed in
// sequence order, sequence s owning tokens [t0[s], t0[s + 1]); each has its
// own cache and cached length.
struct SeqBatch {
  int B;
  int t0[PPD_BATCH_MAX + 1];  // t0[B]: all tokens
  int L[PPD_BATCH_MAX];       // tokens already in the sequence's cache
  int cap[PPD_BATCH_MAX];     // its capacity
  bf16_t *k[PPD_BATCH_MAX];   // this layer's keys [nkv][cap][128]
  bf16_t *v[PPD_BATCH_MAX];   // this layer's values [nkv][128][cap]
};

struct GemmLaunch {
  // operands
  const bf16_t *W;      // packed weight (ppd_pack_weight)
  const bf16_t *A;      // [T_pad][K]
  const bf16_t *zeros;  // 16 zero bytes in global memory
  int N, K, T, MT;      // N = output rows (SwiGLU: F), MT = T_pad / 16
  int kind;             // GemmKind
  int n_tiles, kc_pad, G, maxc;  // partition (see above); maxc: max workgroups per tile
  int ns;               // row groups (waves with rows) per tile: 4, or 3 (whole QKV / gate/up)
  int split;            // G != n_tiles: partial sums + finish kernel
  float *part;          // split: [n_tiles][maxc][8 MT 64][4] partial sums
  // epilogue inputs
  const float *ss;  // norm partials for row scaling (QKV, SwiGLU, LOGITS)
  int n_ss;
  float inv_h, eps;
  const float2 *rope;  // [T_pad][64]
  // QKV outputs
  bf16_t *q;           // [T_pad][nh][128]
  int nh, nkv;
  SeqBatch sb;         // caches, positions: token t of sequence s goes to L[s] + t - t0[s]
  // RESID
  float *x;
  bf16_t *xg;
  const bf16_t *gain;  // next norm's gain [N]
  float *ss_out;       // [n_tiles][T_pad]
  // SWIGLU
  bf16_t *act;         // [T_pad][N]
  // LOGITS
  float *logits;       // [T][N] or null
  float2 *amax;        // [n_tiles][T_pad]
  uint32_t *status;
  void *ev_start, *ev_stop;  // optional events at the first dispatch's start / last one's end
};

enum GemmKind { GEMM_QKV = 0, GEMM_RESID = 1, GEMM_SWIGLU = 2, GEMM_LOGITS = 3 };

// packed layout of a weight for GEMM kind `kind` with N output rows (SwiGLU:
// F features, 2F rows) and K columns
// with ns row groups per tile
int gemm_tiles_of(int kind, int N, int ns);
int gemm_tile_rows_of(int kind, int ns);  // 16 ns (QKV), 32 ns (gate/up) or 128
int gemm_kc_pad_of(int K);
hipError_t launch_pack_weight(int kind, int N, int K, int ns, const bf16_t *src, bf16_t *dst,
                              hipStream_t s);
hipError_t launch_gemm_bf16(const GemmLaunch &g, hipStream_t s);

#define PPD_ATTN_OROW 132  // floats per partial row: 128 dims, m, l, padding

struct AttnLaunch {
  const bf16_t *q;      // [T_pad][nh][d]
  const uint64_t *mask; // [T][2], bits over the token's own tree
  bf16_t *out;          // [T_pad][nh d]
  float *part;          // [nh][max_splits][T_pad][PPD_ATTN_OROW] (splits > 1)
  const bf16_t *zeros;  // >= 16 zero bytes
  int T_pad, nh, nkv, max_splits;
  int MT;               // largest query-tile count of a sequence
  SeqBatch sb;
  // sequence s: workgroups [wg0[s], wg0[s + 1]) = nh x splits[s], chunk[s]
  // 32-key blocks per split
  int wg0[PPD_BATCH_MAX + 1], splits[PPD_BATCH_MAX], chunk[PPD_BATCH_MAX];
  float scale_log2;     // log2(e) / sqrt(d)
  void *ev_start, *ev_stop;  // optional events at the first dispatch's start / last one's end
};
hipError_t launch_attn_bf16(const AttnLaunch &a, hipStream_t s);

// next-step candidate generation (k_next.hip)
#define PPD_NEXT_MAX_DEPTH 15
struct NextTreeLaunch {
  const int32_t *parent, *ids;  // this step's tree
  int T, vocab;
  int n_ept;                    // EPT groups per prompt token (1: plain chains)
  const float *logits;          // [T][vocab]
  const int32_t *path, *n_path, *next_tok;
  int32_t *next_ids;            // [tpl_T]
  uint32_t *status;
  int tpl_T;
  int8_t tpl_depth[PPD_T_MAX];  // template node depth (root 0)
  int16_t tpl_kind[PPD_T_MAX];  // rank of a candidate, or -1 - prompt id
  int k_of_depth[PPD_NEXT_MAX_DEPTH + 1];  // ranks needed at each depth (0: none)
  void *ev_start, *ev_stop;     // optional events on the dispatch (profiling)
};
hipError_t launch_next_tree(const NextTreeLaunch &p, int n_depths, hipStream_t s);

// records the thread's error message (ppd_last_error) and returns s
ppd_status ppd_fail(ppd_status s, const char *fmt, ...);

hipError_t launch_embed(int dtype, const void *tok_emb, const void *prompt_emb, const int32_t *ids,
                        int T, int vocab, int n_prompt, int H, const void *gain, float *x,
                        void *xg, float *ss, uint32_t *status, hipStream_t s);
hipError_t launch_rope_table(const int32_t *depth, const SeqBatch &sb, int d, float base, float2 *rope,
                             hipStream_t s);
hipError_t launch_argmax_final(const float2 *amax, int n_tiles, int T, int T_pad, int32_t *pred,
                               uint32_t *status, hipStream_t s);
hipError_t launch_accept(int T, const int32_t *parent, const int32_t *ids, const int32_t *pred,
                         int vocab, int32_t *path, int32_t *n_path, int32_t *next_tok,
                         uint32_t *status, hipStream_t s);
hipError_t launch_kv_compact(int dtype, void *k, void *v, int n_layers, int nkv, int cap, int d,
                             int L, const int32_t *path, int path_len, const int32_t *n_path,
                             int32_t *len_dev, hipStream_t s);
hipError_t launch_ws_init(void *ws, size_t n_words, hipStream_t s);

// fp32 path (simple kernels for float32 models)
// xg = x * gain and r[t] = 1/sqrt(mean(x^2)+eps); r is stored after xg's T_pad rows
hipError_t launch_f32_rownorm(const float *x, const float *gain, int T, int H, float eps,
                              float *xg, hipStream_t s);
hipError_t launch_f32_matmul(const float *A, const float *W, int T, int N, int K, float *out,
                             hipStream_t s);
hipError_t launch_f32_matmul_scaled(const float *A, const float *W, int T, int N, int K,
                                    const float *r, float *out, hipStream_t s);
hipError_t launch_f32_qkv_post(const float *qkv, const float2 *rope, int T, int nh, int nkv, int d,
                               float *q, float *kc, float *vc, int cap, int L, hipStream_t s);
hipError_t launch_f32_attention(const float *q, const float *kc, const float *vc,
                                const uint64_t *mask, int T, int L, int cap, int nh, int nkv,
                                int d, float *out, hipStream_t s);
hipError_t launch_f32_add(float *x, const float *y, int n, hipStream_t s);
hipError_t launch_f32_swiglu(const float *gu, int T, int F, float *act, hipStream_t s);
hipError_t launch_f32_argmax(const float *logits, int T, int V, int32_t *pred, uint32_t *status,
                             hipStream_t s);
