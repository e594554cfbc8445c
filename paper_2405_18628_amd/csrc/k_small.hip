// Small kernels of the verification step: embedding gather, rotary tables,
// final greedy argmax, acceptance, KV compaction and workspace reset.
#include <algorithm>

#include "ppd_internal.h"

// ---------------------------------------------------------------------------
// Embedding and rotary tables, one launch.  Row t of the residual stream x
// is the embedding of ids[t] (Section 3: prompt tokens are trained
// embeddings appended to the input); for bf16 models the kernel also writes
// the row's sum of squares (the first RMSNorm's one partial per row; its
// x * gain is formed by the consumer GEMM) and, spread over the blocks,
// zeroes the step's tile and head counters.  Rows T..T_pad-1 are zero.
// Rotary table row t: node t sits at position L + depth[t] (Section 3.1);
// the angle of frequency i is pos * base^(-2i/d), evaluated in double
// precision and rounded to float; padding rows get position 0.  Rows of a
// width that is a multiple of 16 bytes are read 16 bytes at a time.

template <typename WT>
__global__ __launch_bounds__(256) void embed_kernel(const WT *__restrict__ tok_emb,
                                                    const WT *__restrict__ prompt_emb,
                                                    const int32_t *__restrict__ ids,
                                                    const int32_t *__restrict__ depth, SeqBatch sb,
                                                    int d, float base, float2 *__restrict__ rope,
                                                    int vocab, int n_prompt, int H,
                                                    float *__restrict__ x, float *__restrict__ ss,
                                                    uint32_t *__restrict__ ctr, size_t n_ctr,
                                                    uint32_t *status) {
  const int t = blockIdx.x, T = sb.t0[sb.B];
  for (size_t i = (size_t)t * blockDim.x + threadIdx.x; i < n_ctr; i += (size_t)gridDim.x * blockDim.x)
    ctr[i] = 0u;
  // rotary row t
  {
    int L = sb.L[0];  // the cached length of token t's sequence
    for (int j = 1; j < sb.B; ++j) L = t >= sb.t0[j] ? sb.L[j] : L;
    for (int i = threadIdx.x; i < d / 2; i += blockDim.x) {
      const double pos = t < T ? (double)L + (double)depth[t] : 0.0;
      const double inv = exp(-(2.0 * i / d) * log((double)base));
      double sn, c;
      sincos(pos * inv, &sn, &c);
      rope[(size_t)t * (d / 2) + i] = make_float2((float)c, (float)sn);
    }
  }
  float *xr = x + (size_t)t * H;
  if (t >= T) {
    for (int k = threadIdx.x; k < H; k += blockDim.x) xr[k] = 0.f;
    if (ss && threadIdx.x == 0) ss[t] = 0.f;
    return;
  }
  int id = ids[t];
  if (id < 0 || id >= vocab + n_prompt) {
    if (threadIdx.x == 0) atomicOr(status, PPD_DEV_BAD_TOKEN);
    id = 0;
  }
  const WT *src = id < vocab ? tok_emb + (size_t)id * H : prompt_emb + (size_t)(id - vocab) * H;
  // 16-byte pieces, several in flight per thread (rows of any other width:
  // one element at a time)
  constexpr int E = 16 / sizeof(WT);
  float acc = 0.f;
  if (H % E) {
    for (int k = threadIdx.x; k < H; k += blockDim.x) {
      float v;
      if constexpr (sizeof(WT) == 2) {
        v = bf16_to_f32(src[k]);
      } else {
        v = src[k];
      }
      xr[k] = v;
      acc += v * v;
    }
  }
#pragma unroll 4
  for (int c = threadIdx.x; H % E == 0 && c < H / E; c += blockDim.x) {
    const u32x4 w = *(const u32x4 *)(src + (size_t)c * E);
    float v[E];
    if constexpr (sizeof(WT) == 2) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] = bf16_to_f32(w[e] & 0xffffu);
        v[2 * e + 1] = bf16_to_f32(w[e] >> 16);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = __uint_as_float(w[e]);
    }
#pragma unroll
    for (int e = 0; e < E; e += 4) {
      *(floatx4 *)(xr + (size_t)c * E + e) = floatx4{v[e], v[e + 1], v[e + 2], v[e + 3]};
      acc += (v[e] * v[e] + v[e + 1] * v[e + 1]) + (v[e + 2] * v[e + 2] + v[e + 3] * v[e + 3]);
    }
  }
  if (ss) {
    __shared__ float red[4];
    acc = wave_sum(acc);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) ss[t] = (red[0] + red[1]) + (red[2] + red[3]);
  }
}

hipError_t launch_embed(int dtype, const void *tok_emb, const void *prompt_emb, const int32_t *ids,
                        const int32_t *depth, const SeqBatch &sb, int d, float base, float2 *rope,
                        int vocab, int n_prompt, int H, float *x, float *ss, uint32_t *ctr,
                        size_t n_ctr, uint32_t *status, hipStream_t s) {
  const int T_pad = (sb.t0[sb.B] + 15) & ~15;
  if (dtype == PPD_BF16) {
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(T_pad), dim3(256), 0, s, (const bf16_t *)tok_emb,
                       (const bf16_t *)prompt_emb, ids, depth, sb, d, base, rope, vocab, n_prompt, H, x,
                       ss, ctr, n_ctr, status);
  } else {
    hipLaunchKernelGGL(embed_kernel<float>, dim3(T_pad), dim3(256), 0, s, (const float *)tok_emb,
                       (const float *)prompt_emb, ids, depth, sb, d, base, rope, vocab, n_prompt, H, x,
                       (float *)nullptr, (uint32_t *)nullptr, (size_t)0, status);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Greedy token (Section 3, exact matching compares against it): per row, the
// smallest vocabulary index attaining the maximum logit.  Combines per-tile
// partials (value, index) written by the LM-head epilogue.  The combining
// operator (larger value, then smaller index) is associative and commutative,
// so the result does not depend on reduction order.

__device__ __forceinline__ void amax_merge(float &v, int &i, float v2, int i2) {
  if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
    v = v2;
    i = i2;
  }
}

__global__ __launch_bounds__(256) void argmax_final_kernel(const float2 *__restrict__ amax,
                                                           int n_tiles, int T_pad,
                                                           int32_t *__restrict__ pred) {
  const int t = blockIdx.x;
  float v = 0.f;
  int idx = -1;
  for (int j = threadIdx.x; j < n_tiles; j += blockDim.x) {
    float2 p = amax[(size_t)j * T_pad + t];
    amax_merge(v, idx, p.x, __float_as_int(p.y));
  }
  for (int o = 32; o > 0; o >>= 1) {
    float v2 = __shfl_xor(v, o, 64);
    int i2 = __shfl_xor(idx, o, 64);
    amax_merge(v, idx, v2, i2);
  }
  __shared__ float sv[4];
  __shared__ int si[4];
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = v;
    si[threadIdx.x >> 6] = idx;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) amax_merge(v, idx, sv[w], si[w]);
    pred[t] = idx < 0 ? 0 : idx;
  }
}

hipError_t launch_argmax_final(const float2 *amax, int n_tiles, int T, int T_pad, int32_t *pred,
                               uint32_t *status, hipStream_t s) {
  (void)status;
  hipLaunchKernelGGL(argmax_final_kernel, dim3(T), dim3(256), 0, s, amax, n_tiles, T_pad, pred);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Acceptance (Section 3, exact matching): node i > 0 is verified iff every
// node on its root path (root excluded) holds a vocabulary token equal to the
// greedy token of its parent.  The accepted node is the deepest verified
// node, ties to the smallest index; n_path = its depth + 1 tokens are emitted
// (accepted candidates plus the bonus token pred[best]).  One thread per node
// checks its own root path; a block reduction picks the best node.

__global__ __launch_bounds__(128) void accept_kernel(int T, const int32_t *__restrict__ parent,
                                                     const int32_t *__restrict__ ids,
                                                     const int32_t *__restrict__ pred, int vocab,
                                                     int32_t *__restrict__ path,
                                                     int32_t *__restrict__ n_path,
                                                     int32_t *__restrict__ next_tok,
                                                     uint32_t *status) {
  __shared__ int sp[PPD_T_MAX], sid[PPD_T_MAX], spr[PPD_T_MAX];
  __shared__ int bad;
  __shared__ int key_s[2];
  const int i = threadIdx.x;
  if (i == 0) bad = 0;
  __syncthreads();
  if (i < T) {
    int p = parent[i];
    bool okp = (i == 0) ? (p == -1) : (p >= 0 && p < i);
    if (!okp) {
      bad = 1;
      p = i == 0 ? -1 : 0;
    }
    sp[i] = p;
    sid[i] = ids[i];
    spr[i] = pred[i];
  }
  __syncthreads();
  if (bad && i == 0) atomicOr(status, PPD_DEV_BAD_PARENT);
  // verified?  walk the root path (parents are earlier nodes: it terminates)
  int key = -1;  // depth * 256 + (255 - i) for verified nodes
  if (i < T) {
    bool ok = true;
    int depth = 0;
    int u = i;
    while (u > 0) {
      int p = sp[u];
      int tok = sid[u];
      ok = ok && tok >= 0 && tok < vocab && tok == spr[p];
      u = p;
      ++depth;
    }
    if (ok) key = depth * 256 + (255 - i);
  }
  // block max of key (deepest first, then smallest index)
  for (int o = 32; o > 0; o >>= 1) key = max(key, __shfl_xor(key, o, 64));
  if ((i & 63) == 0) key_s[i >> 6] = key;
  __syncthreads();
  if (i == 0) {
    int k = max(key_s[0], key_s[1]);
    int best = 255 - (k & 255);
    int depth = k >> 8;
    int u = best;
    for (int j = depth; j >= 0; --j) {
      path[j] = u;
      u = sp[u];
    }
    *n_path = depth + 1;
    *next_tok = spr[best];
  }
}

hipError_t launch_accept(int T, const int32_t *parent, const int32_t *ids, const int32_t *pred,
                         int vocab, int32_t *path, int32_t *n_path, int32_t *next_tok,
                         uint32_t *status, hipStream_t s) {
  hipLaunchKernelGGL(accept_kernel, dim3(1), dim3(128), 0, s, T, parent, ids, pred, vocab, path,
                     n_path, next_tok, status);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// KV compaction (Section 5.3: one cache; only accepted tokens are committed):
// cache[L + k] <- cache[L + path[k]], k < n.  Sources are read into LDS before
// any destination is written, so overlapping moves are safe.  One block per
// (layer, kv head).  n = *n_path clamped to the path's length and to the
// cache's room past L, path entries clamped to that room.

template <typename ET>
__global__ __launch_bounds__(256) void kv_compact_kernel(ET *__restrict__ k, ET *__restrict__ v,
                                                         int cap, int d, int L,
                                                         const int32_t *__restrict__ path,
                                                         int path_len,
                                                         const int32_t *__restrict__ n_path,
                                                         int32_t *len_dev) {
  __shared__ ET buf[PPD_T_MAX * 128];
  __shared__ int sp[PPD_T_MAX];
  int n = *n_path;
  const int room = min(cap - L, PPD_T_MAX);
  n = max(0, min(n, min(room, path_len)));
  for (int j = threadIdx.x; j < n; j += blockDim.x) {
    int p = path[j];
    sp[j] = max(0, min(p, room - 1));
  }
  __syncthreads();
  const size_t lh = blockIdx.x;
  ET *kb = k + lh * (size_t)cap * d;
  ET *vb = v + lh * (size_t)d * cap;
  // keys: rows of d elements
  for (int e = threadIdx.x; e < n * d; e += blockDim.x) {
    int r = e / d, c = e % d;
    buf[e] = kb[(size_t)(L + sp[r]) * d + c];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < n * d; e += blockDim.x) {
    int r = e / d, c = e % d;
    kb[(size_t)(L + r) * d + c] = buf[e];
  }
  __syncthreads();
  // values: [d][cap]
  for (int e = threadIdx.x; e < n * d; e += blockDim.x) {
    int c = e / n, r = e % n;
    buf[e] = vb[(size_t)c * cap + L + sp[r]];
  }
  __syncthreads();
  for (int e = threadIdx.x; e < n * d; e += blockDim.x) {
    int c = e / n, r = e % n;
    vb[(size_t)c * cap + L + r] = buf[e];
  }
  if (len_dev && blockIdx.x == 0 && threadIdx.x == 0) *len_dev = L + n;
}

hipError_t launch_kv_compact(int dtype, void *k, void *v, int n_layers, int nkv, int cap, int d,
                             int L, const int32_t *path, int path_len, const int32_t *n_path,
                             int32_t *len_dev, hipStream_t s) {
  dim3 grid(n_layers * nkv);
  if (dtype == PPD_BF16)
    hipLaunchKernelGGL(kv_compact_kernel<bf16_t>, grid, dim3(256), 0, s, (bf16_t *)k, (bf16_t *)v,
                       cap, d, L, path, path_len, n_path, len_dev);
  else
    hipLaunchKernelGGL(kv_compact_kernel<float>, grid, dim3(256), 0, s, (float *)k, (float *)v, cap,
                       d, L, path, path_len, n_path, len_dev);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------

// ---------------------------------------------------------------------------
// HBM read probe: workgroup b reads the b-th of 256 contiguous pieces of the
// buffer (16-byte non-temporal loads, RP per thread in flight), XORs them,
// and adds its XOR into the sink with an atomic.
constexpr int RP = 8;
__global__ __launch_bounds__(256, 1) void read_probe_kernel(const u32x4 *__restrict__ buf, size_t n16,
                                                            uint32_t *sink) {
  const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const size_t b0 = min(n16, blockIdx.x * per), b1 = min(n16, b0 + per);
  u32x4 acc = u32x4{0u, 0u, 0u, 0u};
  for (size_t i = b0 + threadIdx.x; i < b1; i += (size_t)RP * blockDim.x) {
    u32x4 r[RP];
#pragma unroll
    for (int j = 0; j < RP; ++j) {
      const size_t k = i + (size_t)j * blockDim.x;
      r[j] = __builtin_nontemporal_load(buf + (k < b1 ? k : b0));
    }
#pragma unroll
    for (int j = 0; j < RP; ++j)
      if (i + (size_t)j * blockDim.x < b1) acc ^= r[j];  // the clamped repeats are not added
  }
  const uint32_t v = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (v) atomicXor(sink, v);
}

hipError_t launch_read_probe(const void *buf, size_t bytes, uint32_t *sink, hipStream_t s) {
  hipLaunchKernelGGL(read_probe_kernel, dim3(256), dim3(256), 0, s, (const u32x4 *)buf, bytes / 16, sink);
  return hipGetLastError();
}

__global__ void ws_init_kernel(uint32_t *w, size_t n) {
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < n;
       i += (size_t)gridDim.x * blockDim.x)
    w[i] = 0u;
}

hipError_t launch_ws_init(void *ws, size_t n_words, hipStream_t s) {
  hipLaunchKernelGGL(ws_init_kernel, dim3(64), dim3(256), 0, s, (uint32_t *)ws, n_words);
  return hipGetLastError();
}
