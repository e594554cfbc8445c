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

// buffer resource over a whole workspace region (raw, untyped loads)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc_of(const void *p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}
// 16-byte load that misses L1 (sc0): data written by another compute unit of
// this XCD is read from the shared L2 (each address is read once per
// dispatch, after the writers' arrival)
__device__ __forceinline__ floatx4 load_l2(__amdgpu_buffer_rsrc_t r, uint32_t byte_off) {
  return __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(r, (int)byte_off, 0, 1));
}

// the XCD this wave runs on
__device__ __forceinline__ unsigned xcc_id() {
  unsigned v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xf;
}

// Arrival at an XCD-local counter shared by n workgroups of one dispatch
// (one thread per workgroup, after its results have reached L2), then a
// bounded wait for the other n - 1.  Workgroup b runs on XCD (b + o) % 8, o
// being the dispatcher's offset (round-robin from wherever the previous
// dispatch left it: the same for every workgroup of this one), so each
// arrival adds 1 + 256 o, o = (this XCD - set) mod 8; a final count whose
// high part is not n o means the workgroups did not share an XCD.  Agent
// scope: a workgroup-scope load may be served by this compute unit's L1,
// which keeps the line of the first poll.
__device__ __forceinline__ void xcd_arrive_wait(uint32_t *ctr, int set, uint32_t n, int spin_limit,
                                                uint32_t *status) {
  const uint32_t o = (xcc_id() - (unsigned)set) & 7u;
  __hip_atomic_fetch_add(ctr, 1u + (o << 8), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  int it = 0;
  uint32_t v;
  while (((v = __hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) & 0xffu) < n) {
    if (++it > spin_limit) {
      atomicOr(status, PPD_DEV_SYNC_TIMEOUT);
      break;
    }
    __builtin_amdgcn_s_sleep(2);
  }
  if ((v >> 8) != o * n) atomicOr(status, PPD_DEV_XCD_PLACEMENT);
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
  size_t xg;          // fp32 path: float [T_pad][H] x * gain, then [T_pad] row scales
  size_t ss;          // float  [max_ss][T_pad]   sum-of-squares partials
  size_t q;           // float  [T_pad][nh][d]    queries after RoPE
  size_t attn_o;      // float  [T_pad][nh d]     attention output
  size_t act;         // float  [T_pad][F]        SwiGLU output
  size_t tmp;         // float  [T_pad][max(qkv_rows, 2F, V)]  (fp32 path only)
  size_t attn_part;   // float  [nh][max_splits][T_pad][d + 2]
  size_t gemm_part;   // float  [max_part_floats]
  size_t amax;        // float2 [max_amax_tiles][T_pad]
  size_t rope;        // float2 [T_pad][d/2]      (cos, sin)
  size_t ctr;         // uint32 [n_ctr]           tile / head counters (zeroed per step)
  size_t n_ctr;
  size_t total;
  int max_ss, max_splits, max_amax_tiles;
  size_t max_part_floats;
};

#define PPD_ATTN_MAX_SPLITS 64

// ---------------------------------------------------------------------------
// kernel launchers (defined in the .hip files, called by the host driver)

// Skinny GEMM partition (k_gemm.hip).  Weights are packed group-major: a
// group is 16 output rows (gate/up: 16 features, i.e. 16 gate and 16 up
// rows), each of its K / 64 chunks a run of 1 KB MFMA fragments.  The groups
// are dealt to the 8 XCDs (XCD x: groups [xg0[x], xg0[x + 1])); on each XCD,
// TX tiles (consecutive groups, at most 4 gw) x s K-slices take its TX s
// workgroups (workgroup b runs on XCD b % 8, slot b / 8 = tile s + slice).
// A tile split over s > 1 slices is finished inside the kernel: partial sums
// to L2, an XCD-local counter, each slice finishing token blocks ks, ks + s,
// ...  Grid = 8 TX s <= 256, one workgroup per compute unit.
#define PPD_GEMM_BN 128

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
  const float *A;       // [T_pad][K] fp32 activations (norm consumers: the residual x)
  const bf16_t *gain;   // norm consumers (QKV, gate/up, LM head): the norm gain [K]
  int N, K, T, MT;      // N = output rows (SwiGLU: F), MT = T_pad / 16
  int kind;             // GemmKind
  // partition (see above)
  int kc;               // K / 64
  int gw;               // groups per wave (a tile holds at most 4 gw groups)
  int TX, s;            // tiles per XCD, K slices per tile
  int xg0[9];
  float *part;          // s > 1: [8 TX][s][4 gw S MT][64] floatx4 partial sums
  uint32_t *ctr;        // s > 1: tile counters, XCD x's at ctr + 32 x (zeroed per step)
  int spin_limit;       // bounded wait for a tile's other slices
  // epilogue inputs
  const float *ss;      // norm partials for row scaling (QKV, SwiGLU, LOGITS)
  int n_ss;
  float inv_h, eps;
  const float2 *rope;   // [T_pad][64]
  // QKV outputs
  float *q;             // [T_pad][nh][128] fp32
  int nh, nkv;
  SeqBatch sb;          // caches, positions: token t of sequence s goes to L[s] + t - t0[s]
  // RESID
  float *x;
  float *ss_out;        // [8 TX][T_pad]
  // SWIGLU
  float *act;           // [T_pad][N] fp32
  // LOGITS
  float *logits;        // [T][N] or null
  float2 *amax;         // [8 TX][T_pad]
  uint32_t *status;
  void *ev_start, *ev_stop;  // optional events at the dispatch's start / end
};

enum GemmKind { GEMM_QKV = 0, GEMM_RESID = 1, GEMM_SWIGLU = 2, GEMM_LOGITS = 3 };

int gemm_groups_of(int kind, int N);  // groups of a GEMM with N output rows (gate/up: features)
int gemm_sub_of(int kind);            // 16-row sub-tiles per group (2 for gate/up)
int gemm_gw_max(int kind, int MT);    // largest groups-per-wave instantiated for MT token tiles
hipError_t launch_pack_weight(int kind, int N, int K, const bf16_t *src, bf16_t *dst, hipStream_t s);
hipError_t launch_gemm_bf16(const GemmLaunch &g, hipStream_t s);

#define PPD_ATTN_OROW 132  // floats per partial row: 128 dims, m, l, padding

struct AttnLaunch {
  const float *q;       // [T_pad][nh][d] fp32
  const uint64_t *mask; // [T][2], bits over the token's own tree
  float *out;           // [T_pad][nh d] fp32
  float *part;          // [nh][max_splits][T_pad][PPD_ATTN_OROW] (splits > 1)
  const bf16_t *zeros;  // >= 16 zero bytes
  int T_pad, nh, nkv, max_splits;
  int MT;               // largest query-tile count of a sequence
  SeqBatch sb;
  // sequence s: workgroups [wg0[s], wg0[s + 1]) = nh x splits[s], chunk[s]
  // 32-key blocks per split
  int wg0[PPD_BATCH_MAX + 1], splits[PPD_BATCH_MAX], chunk[PPD_BATCH_MAX];
  // xcd_merge (one sequence): the heads are dealt to the 8 XCDs (XCD x:
  // heads [nh x / 8, nh (x + 1) / 8), workgroup b runs on XCD b % 8, slot
  // b / 8 = local head splits + split), and each head's splits merge inside
  // the kernel through L2 behind the head's counter, ctr + 32 x + local head
  // (zeroed per step); otherwise a merge kernel adds them
  int xcd_merge;
  uint32_t *ctr;
  int spin_limit;
  uint32_t *status;
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

// embedding rows into x (fp32), rows T..T_pad-1 zero, and the rotary
// table [T_pad][d / 2] (cos, sin); bf16 models also write each row's sum of
// squares to ss and zero the n_ctr tile / head counters
hipError_t launch_embed(int dtype, const void *tok_emb, const void *prompt_emb, const int32_t *ids,
                        const int32_t *depth, const SeqBatch &sb, int d, float base, float2 *rope,
                        int vocab, int n_prompt, int H, float *x, float *ss, uint32_t *ctr,
                        size_t n_ctr, uint32_t *status, hipStream_t s);
hipError_t launch_argmax_final(const float2 *amax, int n_tiles, int T, int T_pad, int32_t *pred,
                               uint32_t *status, hipStream_t s);
hipError_t launch_accept(int T, const int32_t *parent, const int32_t *ids, const int32_t *pred,
                         int vocab, int32_t *path, int32_t *n_path, int32_t *next_tok,
                         uint32_t *status, hipStream_t s);
hipError_t launch_kv_compact(int dtype, void *k, void *v, int n_layers, int nkv, int cap, int d,
                             int L, const int32_t *path, int path_len, const int32_t *n_path,
                             int32_t *len_dev, hipStream_t s);
hipError_t launch_ws_init(void *ws, size_t n_words, hipStream_t s);
hipError_t launch_read_probe(const void *buf, size_t bytes, uint32_t *sink, hipStream_t s);

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
