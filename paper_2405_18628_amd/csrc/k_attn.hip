// Split-KV tree attention on the gfx950 matrix cores (Section 4.1: every tree
// node attends to the cached prefix, to its ancestors and to itself).
//
// Keys of one kv head occupy cache positions [0, L + T): the accepted prefix
// [0, L) -- visible to every node -- followed by the tree nodes' own keys
// (written at L + i by the QKV epilogue), visible to node t iff bit i of its
// ancestor mask is set.  The key range is cut into 32-key blocks; workgroup
// (head, split) streams a contiguous run of blocks through LDS and keeps an
// online softmax per query; the last split of a head to finish (atomic
// ticket) combines the splits in split order.
//
// Per 32-key block, on the matrix cores (v_mfma_f32_16x16x32_bf16):
//   S^T[key][query] = K Q^T      keys are the 16-row A operand (from LDS),
//                                queries the B operand (registers)
//   O^T[d][query]  += V^T P^T    values (stored position-minor, so V^T rows
//                                are contiguous) are the A operand from LDS;
//                                P^T comes straight from S^T's accumulator
//                                layout: the key order inside a 16-key tile is
//                                permuted so each lane's 8 probabilities are 8
//                                consecutive keys, i.e. a valid B operand.
// Softmax runs in fp32 in the log2 domain; P is rounded to bf16 for the PV
// product.
#include "ppd_internal.h"

namespace {

constexpr int KROW = 136;  // LDS row of 128 keys dims + 8 pad (bf16 elements)
constexpr int VROW = 40;   // LDS row of 32 keys + 8 pad

// MFMA row m of key tile kt holds key 8 (m / 4) + 4 kt + (m % 4); LDS row of a key
__device__ __forceinline__ int key_lds_row(int j) {  // j in [0, 32)
  const int a = j >> 3, kt = (j >> 2) & 1, e = j & 3;
  return kt * 16 + a * 4 + e;
}

template <int NQ>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnLaunch p) {
  __shared__ __attribute__((aligned(16))) bf16_t k_lds[32 * KROW];
  __shared__ __attribute__((aligned(16))) bf16_t v_lds[128 * VROW];
  __shared__ int last_s;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int h = blockIdx.x / p.splits;
  const int split = blockIdx.x % p.splits;
  const int kvh = h / (p.nh / p.nkv);
  const int n_keys = p.L + p.T;
  const int nblk = (n_keys + 31) >> 5;
  const int b0 = split * p.chunk, b1 = min(nblk, b0 + p.chunk);
  const bf16_t *kbase = p.kc + (size_t)kvh * p.cap * 128;
  const bf16_t *vbase = p.vc + (size_t)kvh * 128 * p.cap;

  // queries of this wave's tiles (B operand), ancestor masks, softmax state
  u32x4 qf[NQ][4];
  uint64_t mk0[NQ], mk1[NQ];
  floatx4 o[NQ][8];
  float m_run[NQ], l_run[NQ];
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int qt = wave + 4 * q;
    const int t = qt * 16 + lr;
    const bool live = qt < p.MT && t < p.T;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) {
      qf[q][ds] = live ? *(const u32x4 *)(p.q + ((size_t)t * p.nh + h) * 128 + ds * 32 + lg * 8)
                       : u32x4{0u, 0u, 0u, 0u};
    }
    mk0[q] = live ? p.mask[2 * t] : 0ull;
    mk1[q] = live ? p.mask[2 * t + 1] : 0ull;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[q][dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    m_run[q] = -INFINITY;
    l_run[q] = 0.f;
  }

  // global -> register staging of one block: 2 K chunks + 2 V chunks per thread
  u32x4 kst[2], vst[2];
  auto fetch = [&](int b) {
    const int key0 = b * 32;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int c = threadIdx.x + 256 * r;  // 0..511
      // K: key c / 16, 16-byte chunk c % 16 of its 128 dims
      const int j = c >> 4, ch = c & 15;
      const int key = key0 + j;
      kst[r] = key < n_keys ? *(const u32x4 *)(kbase + (size_t)key * 128 + ch * 8)
                            : u32x4{0u, 0u, 0u, 0u};
      // V^T: dim row c / 4, keys 8 (c % 4) .. + 7
      const int d = c >> 2, kc8 = (c & 3) * 8;
      const int kk = key0 + kc8;
      u32x4 v = u32x4{0u, 0u, 0u, 0u};
      if (kk < n_keys) {
        v = *(const u32x4 *)(vbase + (size_t)d * p.cap + kk);
        const int nv = n_keys - kk;  // valid keys in this chunk (may be < 8)
        if (nv < 8) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const int k0 = 2 * w;
            uint32_t keep = (k0 < nv ? 0xffffu : 0u) | (k0 + 1 < nv ? 0xffff0000u : 0u);
            v[w] &= keep;
          }
        }
      }
      vst[r] = v;
    }
  };
  auto stash = [&]() {
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int c = threadIdx.x + 256 * r;
      const int j = c >> 4, ch = c & 15;
      *(u32x4 *)(k_lds + key_lds_row(j) * KROW + ch * 8) = kst[r];
      const int d = c >> 2, kc8 = (c & 3) * 8;
      *(u32x4 *)(v_lds + d * VROW + kc8) = vst[r];
    }
  };

  if (b0 < b1) fetch(b0);
  for (int b = b0; b < b1; ++b) {
    __syncthreads();
    stash();
    __syncthreads();
    if (b + 1 < b1) fetch(b + 1);
    const int key0 = b * 32;
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int qt = wave + 4 * q;
      if (qt >= p.MT) continue;
      // S^T for 2 key tiles
      floatx4 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        s[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) {
          const u32x4 ka = *(const u32x4 *)(k_lds + (kt * 16 + lr) * KROW + ds * 32 + lg * 8);
          s[kt] = mfma16x16x32(as_bf16x8(ka), as_bf16x8(qf[q][ds]), s[kt]);
        }
      }
      // scale, mask, block max
      float sv[8];
      float bmax = -INFINITY;
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = key0 + lg * 8 + kt * 4 + e;
          bool vis;
          if (j < p.L) {
            vis = true;
          } else if (j < n_keys) {
            const int jj = j - p.L;
            vis = ((jj < 64 ? (mk0[q] >> jj) : (mk1[q] >> (jj - 64))) & 1ull) != 0;
          } else {
            vis = false;
          }
          const float x = vis ? s[kt][e] * p.scale_log2 : -INFINITY;
          sv[kt * 4 + e] = x;
          bmax = fmaxf(bmax, x);
        }
      bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
      bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
      // no divergence around the MFMAs: a query with nothing visible yet uses
      // a finite reference so that every probability and alpha is exactly 0
      const float m_new = fmaxf(m_run[q], bmax);
      const float m_ref = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_run[q] - m_ref);
      m_run[q] = m_new;
      float pv[8];
      float psum = 0.f;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        pv[i] = exp2f(sv[i] - m_ref);
        psum += pv[i];
      }
      l_run[q] = l_run[q] * alpha + psum;
      const u32x4 pb = u32x4{pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                             pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const u32x4 va = *(const u32x4 *)(v_lds + (dt * 16 + lr) * VROW + lg * 8);
        o[q][dt] = mfma16x16x32(as_bf16x8(va), as_bf16x8(pb), o[q][dt] * alpha);
      }
    }
  }

  // per-query totals: l over the 4 lane groups (m is already uniform)
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    l_run[q] += __shfl_xor(l_run[q], 16, 64);
    l_run[q] += __shfl_xor(l_run[q], 32, 64);
  }

  const int T_pad = p.MT * 16;
  if (p.splits == 1) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int qt = wave + 4 * q;
      const int t = qt * 16 + lr;
      if (qt >= p.MT || t >= p.T) continue;
      const float inv = 1.f / l_run[q];
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const floatx4 v = o[q][dt] * inv;
        *(u32x2 *)(p.out + (size_t)t * p.nh * 128 + h * 128 + dt * 16 + lg * 4) =
            u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      }
    }
    return;
  }

  // Publish this split's (O, m, l), row stride 132 floats, with agent-scope
  // relaxed atomic stores: they write through to memory that every XCD sees,
  // without the L2 write-back and invalidate that a device fence costs.  The
  // ticket is taken only after the stores have completed (s_waitcnt), and
  // the last split reads the partials back with agent-scope atomic loads,
  // which bypass any stale copy in its own L2.
  uint64_t *mypart = (uint64_t *)(p.part + ((size_t)h * p.splits + split) * T_pad * 132);
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const int qt = wave + 4 * q;
    if (qt >= p.MT) continue;
    const int t = qt * 16 + lr;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) {
      uint64_t *d = mypart + ((size_t)t * 132 + dt * 16 + lg * 4) / 2;
      const floatx4 v = o[q][dt];
      __hip_atomic_store(d, __builtin_bit_cast(uint64_t, float2{v[0], v[1]}), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(d + 1, __builtin_bit_cast(uint64_t, float2{v[2], v[3]}), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    if (lg == 0)
      __hip_atomic_store(mypart + ((size_t)t * 132 + 128) / 2,
                         __builtin_bit_cast(uint64_t, float2{m_run[q], l_run[q]}), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev =
        __hip_atomic_fetch_add(&p.counters[h], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = prev == (unsigned)(p.splits - 1);
    if (last) __hip_atomic_store(&p.counters[h], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last_s = last;
  }
  __syncthreads();
  if (!last_s) return;

  // combine the splits of head h in split order: thread -> (t, 4 dims)
  const uint64_t *hp = (const uint64_t *)(p.part + (size_t)h * p.splits * T_pad * 132);
  auto ld2 = [](const uint64_t *a) {
    return __builtin_bit_cast(float2, __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  };
  for (int w = threadIdx.x; w < p.T * 32; w += 256) {
    const int t = w >> 5, d4 = (w & 31) * 4;
    float M = -INFINITY;
    for (int s = 0; s < p.splits; ++s) M = fmaxf(M, ld2(hp + (((size_t)s * T_pad + t) * 132 + 128) / 2).x);
    floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
    float lsum = 0.f;
    for (int s = 0; s < p.splits; ++s) {
      const uint64_t *row = hp + ((size_t)s * T_pad + t) * 132 / 2;
      const float2 ml = ld2(row + 64);
      const float sc = ml.x == -INFINITY ? 0.f : exp2f(ml.x - M);
      lsum += sc * ml.y;
      const float2 a = ld2(row + d4 / 2), b = ld2(row + d4 / 2 + 1);
      acc += sc * floatx4{a.x, a.y, b.x, b.y};
    }
    const float inv = 1.f / lsum;
    *(u32x2 *)(p.out + (size_t)t * p.nh * 128 + h * 128 + d4) =
        u32x2{pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
  }
}

}  // namespace

hipError_t launch_attn_bf16(const AttnLaunch &a, hipStream_t s) {
  dim3 grid(a.nh * a.splits), block(256);
  if (a.MT <= 4)
    hipLaunchKernelGGL(attn_bf16_kernel<1>, grid, block, 0, s, a);
  else
    hipLaunchKernelGGL(attn_bf16_kernel<2>, grid, block, 0, s, a);
  return hipGetLastError();
}
