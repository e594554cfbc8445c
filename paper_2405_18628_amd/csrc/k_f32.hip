// Straightforward float32 kernels of the verification step, used for float32
// models (small models where the step is cache-resident and latency, not
// bandwidth, matters).  One thread per output for matrix products, one block
// per (node, head) for tree attention.  Same semantics as the bfloat16 path:
// RMSNorm is applied as (x * gain) followed by a per-row scale of the product.
#include "ppd_internal.h"

__global__ __launch_bounds__(256) void f32_norm_prep_kernel(const float *__restrict__ x,
                                                            const float *__restrict__ gain, int H,
                                                            float eps, float *__restrict__ xg,
                                                            float *__restrict__ r) {
  const int t = blockIdx.x;
  float acc = 0.f;
  for (int k = threadIdx.x; k < H; k += blockDim.x) {
    const float v = x[(size_t)t * H + k];
    acc += v * v;
    xg[(size_t)t * H + k] = v * gain[k];
  }
  __shared__ float red[4];
  acc = wave_sum(acc);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) r[t] = rsqrtf(((red[0] + red[1]) + (red[2] + red[3])) / (float)H + eps);
}

hipError_t launch_f32_rownorm(const float *x, const float *gain, int T, int H, float eps,
                              float *xg, hipStream_t s) {
  // r is stored right after xg's T_pad rows
  const int T_pad = (T + 15) & ~15;
  hipLaunchKernelGGL(f32_norm_prep_kernel, dim3(T), dim3(256), 0, s, x, gain, H, eps, xg,
                     xg + (size_t)T_pad * H);
  return hipGetLastError();
}

// out[t][n] = (r ? r[t] : 1) * sum_k A[t][k] W[n][k]; r follows A's T_pad rows when
// scale_rows is set (see launch_f32_rownorm)
// (grid: (N / 256, T) -- one row of blocks per token)
__global__ __launch_bounds__(256) void f32_matmul_kernel(const float *__restrict__ A,
                                                         const float *__restrict__ W, int N,
                                                         int K, const float *__restrict__ r,
                                                         float *__restrict__ out) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  const int t = blockIdx.y;
  if (n >= N) return;
  const float *a = A + (size_t)t * K;
  const float *w = W + (size_t)n * K;
  float acc = 0.f;
  for (int k = 0; k < K; ++k) acc = fmaf(a[k], w[k], acc);
  out[(size_t)t * N + n] = r ? acc * r[t] : acc;
}

hipError_t launch_f32_matmul(const float *A, const float *W, int T, int N, int K, float *out,
                             hipStream_t s) {
  hipLaunchKernelGGL(f32_matmul_kernel, dim3((N + 255) / 256, T), dim3(256), 0, s, A, W, N, K,
                     (const float *)nullptr, out);
  return hipGetLastError();
}

hipError_t launch_f32_matmul_scaled(const float *A, const float *W, int T, int N, int K,
                                    const float *r, float *out, hipStream_t s) {
  hipLaunchKernelGGL(f32_matmul_kernel, dim3((N + 255) / 256, T), dim3(256), 0, s, A, W, N, K,
                     r, out);
  return hipGetLastError();
}

// RoPE (rotate-half) on queries and keys; q -> workspace, k and v -> cache
// position L + t.
__global__ void f32_qkv_post_kernel(const float *__restrict__ qkv, const float2 *__restrict__ rope,
                                    int nh, int nkv, int d, float *__restrict__ q,
                                    float *__restrict__ kc, float *__restrict__ vc, int cap, int L) {
  const int t = blockIdx.x;
  const int half = d / 2;
  const int rows = (nh + 2 * nkv) * d;
  const float *src = qkv + (size_t)t * rows;
  for (int e = threadIdx.x; e < (nh + 2 * nkv) * half; e += blockDim.x) {
    const int hp = e / half, i = e % half;
    float a = src[hp * d + i], b = src[hp * d + i + half];
    if (hp < nh + nkv) {
      const float2 cs = rope[(size_t)t * half + i];
      const float a2 = a * cs.x - b * cs.y, b2 = b * cs.x + a * cs.y;
      a = a2;
      b = b2;
    }
    if (hp < nh) {
      q[((size_t)t * nh + hp) * d + i] = a;
      q[((size_t)t * nh + hp) * d + i + half] = b;
    } else if (hp < nh + nkv) {
      float *kr = kc + ((size_t)(hp - nh) * cap + L + t) * d;
      kr[i] = a;
      kr[i + half] = b;
    } else {
      float *vb = vc + (size_t)(hp - nh - nkv) * d * cap + L + t;
      vb[(size_t)i * cap] = a;
      vb[(size_t)(i + half) * cap] = b;
    }
  }
}

hipError_t launch_f32_qkv_post(const float *qkv, const float2 *rope, int T, int nh, int nkv, int d,
                               float *q, float *kc, float *vc, int cap, int L, hipStream_t s) {
  hipLaunchKernelGGL(f32_qkv_post_kernel, dim3(T), dim3(256), 0, s, qkv, rope, nh, nkv, d, q, kc,
                     vc, cap, L);
  return hipGetLastError();
}

// Tree attention, one block of 128 threads per (node t, head h): keys in chunks
// of 128 (one per thread), online softmax; thread i accumulates output dim i.
__global__ __launch_bounds__(128) void f32_attention_kernel(
    const float *__restrict__ q, const float *__restrict__ kc, const float *__restrict__ vc,
    const uint64_t *__restrict__ mask, int T, int L, int cap, int nh, int nkv, int d,
    float *__restrict__ out) {
  const int t = blockIdx.x, h = blockIdx.y;
  const int kvh = h / (nh / nkv);
  const float *qr = q + ((size_t)t * nh + h) * d;
  const float *kb = kc + (size_t)kvh * cap * d;
  const float *vb = vc + (size_t)kvh * d * cap;
  const uint64_t m0 = mask[2 * t], m1 = mask[2 * t + 1];
  const float scale = rsqrtf((float)d);
  __shared__ float p_s[128];
  __shared__ float red[2];
  float m_run = -INFINITY, l_run = 0.f, acc = 0.f;
  const int n_keys = L + T;
  for (int c0 = 0; c0 < n_keys; c0 += 128) {
    const int j = c0 + threadIdx.x;
    float sc = -INFINITY;
    bool vis = j < L;
    if (!vis && j < n_keys) {
      const int jj = j - L;
      vis = ((jj < 64 ? (m0 >> jj) : (m1 >> (jj - 64))) & 1ull) != 0;
    }
    if (vis) {
      float dot = 0.f;
      for (int i = 0; i < d; ++i) dot = fmaf(qr[i], kb[(size_t)j * d + i], dot);
      sc = dot * scale;
    }
    float bm = wave_max(sc);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = bm;
    __syncthreads();
    bm = fmaxf(red[0], red[1]);
    __syncthreads();
    const float m_new = fmaxf(m_run, bm);
    const float m_ref = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = expf(m_run - m_ref);
    const float pj = expf(sc - m_ref);
    p_s[threadIdx.x] = pj;
    float ps = wave_sum(pj);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ps;
    __syncthreads();
    ps = red[0] + red[1];
    l_run = l_run * alpha + ps;
    m_run = m_new;
    if ((int)threadIdx.x < d) {
      acc *= alpha;
      const int cn = min(128, n_keys - c0);
      for (int jj = 0; jj < cn; ++jj) {
        const float pv = p_s[jj];
        if (pv != 0.f) acc = fmaf(pv, vb[(size_t)threadIdx.x * cap + c0 + jj], acc);
      }
    }
    __syncthreads();
  }
  if ((int)threadIdx.x < d) out[(size_t)t * nh * d + h * d + threadIdx.x] = acc / l_run;
}

hipError_t launch_f32_attention(const float *q, const float *kc, const float *vc,
                                const uint64_t *mask, int T, int L, int cap, int nh, int nkv,
                                int d, float *out, hipStream_t s) {
  hipLaunchKernelGGL(f32_attention_kernel, dim3(T, nh), dim3(128), 0, s, q, kc, vc, mask, T, L,
                     cap, nh, nkv, d, out);
  return hipGetLastError();
}

__global__ void f32_add_kernel(float *__restrict__ x, const float *__restrict__ y, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) x[i] += y[i];
}

hipError_t launch_f32_add(float *x, const float *y, int n, hipStream_t s) {
  hipLaunchKernelGGL(f32_add_kernel, dim3((n + 255) / 256), dim3(256), 0, s, x, y, n);
  return hipGetLastError();
}

__global__ void f32_swiglu_kernel(const float *__restrict__ gu, int F, float *__restrict__ act) {
  const int t = blockIdx.y;
  const int f = blockIdx.x * blockDim.x + threadIdx.x;
  if (f >= F) return;
  const float g = gu[(size_t)t * 2 * F + f], u = gu[(size_t)t * 2 * F + F + f];
  act[(size_t)t * F + f] = g / (1.f + expf(-g)) * u;
}

hipError_t launch_f32_swiglu(const float *gu, int T, int F, float *act, hipStream_t s) {
  hipLaunchKernelGGL(f32_swiglu_kernel, dim3((F + 255) / 256, T), dim3(256), 0, s, gu, F, act);
  return hipGetLastError();
}

// greedy token per row: smallest index of the maximum; NaN logits are skipped
// and flagged
__global__ __launch_bounds__(256) void f32_argmax_kernel(const float *__restrict__ logits, int V,
                                                         int32_t *__restrict__ pred,
                                                         uint32_t *status) {
  const int t = blockIdx.x;
  const float *row = logits + (size_t)t * V;
  float bv = 0.f;
  int bi = -1;
  bool nan = false;
  for (int n = threadIdx.x; n < V; n += blockDim.x) {
    const float v = row[n];
    if (v != v) {
      nan = true;
      continue;
    }
    if (bi < 0 || v > bv) {
      bv = v;
      bi = n;
    }
  }
  if (nan) atomicOr(status, PPD_DEV_NAN_LOGIT);
  for (int o = 32; o > 0; o >>= 1) {
    const float v2 = __shfl_xor(bv, o, 64);
    const int i2 = __shfl_xor(bi, o, 64);
    if (i2 >= 0 && (bi < 0 || v2 > bv || (v2 == bv && i2 < bi))) {
      bv = v2;
      bi = i2;
    }
  }
  __shared__ float sv[4];
  __shared__ int si[4];
  if ((threadIdx.x & 63) == 0) {
    sv[threadIdx.x >> 6] = bv;
    si[threadIdx.x >> 6] = bi;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w)
      if (si[w] >= 0 && (bi < 0 || sv[w] > bv || (sv[w] == bv && si[w] < bi))) {
        bv = sv[w];
        bi = si[w];
      }
    pred[t] = bi < 0 ? 0 : bi;
  }
}

hipError_t launch_f32_argmax(const float *logits, int T, int V, int32_t *pred, uint32_t *status,
                             hipStream_t s) {
  hipLaunchKernelGGL(f32_argmax_kernel, dim3(T), dim3(256), 0, s, logits, V, pred, status);
  return hipGetLastError();
}
