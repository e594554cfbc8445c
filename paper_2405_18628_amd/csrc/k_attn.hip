// Split-KV tree attention on the gfx950 matrix cores (Section 4.1: every tree
// node attends to the cached prefix, to its ancestors and to itself).
//
// Keys of one kv head occupy cache positions [0, L + T): the accepted prefix
// [0, L) -- visible to every node -- followed by the tree nodes' own keys
// (written at L + i by the QKV epilogue), visible to node t iff bit i of its
// ancestor mask is set.  The key range is cut into 32-key blocks.
//
// Work decomposition.  A workgroup owns one head h, one tile of 16 queries
// and one of KS contiguous key splits; its four waves cut that split again
// into four contiguous runs and each keeps its own online softmax.  A wave
// streams its run through a private two-slot LDS ring with direct-to-LDS
// transfers (global_load_lds_dwordx4), so waves never wait on each other
// inside the loop: block i+1 is requested before block i is waited for.
// At the end the four waves are merged through LDS; with KS > 1 the merged
// (O, m, l) of each split is published and the last split of the (head,
// query tile) to finish (atomic ticket) merges the splits in split order.
// The query tiles of one (head, split) get workgroup ids congruent mod 8,
// which the dispatcher places on one XCD, so they share its L2 and the
// keys/values cross HBM about once.
//
// Per 32-key block, on the matrix cores (v_mfma_f32_16x16x32_bf16):
//   S^T[key][query] = K Q^T      keys are the 16-row A operand (LDS),
//                                queries the B operand (registers)
//   O^T[d][query]  += V^T P^T    values (stored position-minor, so V^T rows
//                                are contiguous) are the A operand (LDS);
//                                P^T comes straight from S^T's accumulator
//                                layout: LDS row m of key tile kt holds key
//                                8 (m / 4) + 4 kt + (m % 4), so each lane's 8
//                                probabilities are 8 consecutive keys, i.e. a
//                                valid B operand.
// Softmax runs in fp32 in the log2 domain; P enters the PV product as the sum
// of two bf16 parts (hi, lo), i.e. to about 16 significant bits.
#include "ppd_internal.h"

namespace {

constexpr int KSLOT = 8192;               // 32 keys x 256 bytes
constexpr int VSLOT = 8192;               // 128 dims x 64 bytes (32 keys)
constexpr int SLOT = KSLOT + VSLOT;       // one block in LDS
constexpr int WAVE_LDS = SLOT;            // per wave (also holds its merge rows)
constexpr int OROW = 132;                 // merge row: 128 dims + padding (floats)
#ifndef PPD_ATTN_RING
#define PPD_ATTN_RING 2
#endif
constexpr int RING = PPD_ATTN_RING;       // blocks in flight per wave (registers)

// LDS row of the K slot holding key j (j < 32) of a block: MFMA row m of key
// tile kt holds key 8 (m / 4) + 4 kt + (m % 4)
__device__ __forceinline__ int row_of_key(int j) {
  const int a = j >> 3, kt = (j >> 2) & 1, e = j & 3;
  return kt * 16 + a * 4 + e;
}

__global__ __launch_bounds__(256, 1) void attn_bf16_kernel(AttnLaunch p) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[4 * WAVE_LDS];
  __shared__ float ml_s[4][16][2];
  __shared__ int last_s;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int KS = p.splits;
  const int G = p.nh * KS;
  // workgroup id -> (group g = (head, split), query tile qt)
  const int x8 = blockIdx.x & 7, rr = blockIdx.x >> 3;
  const int qt = rr % p.MT;
  const int g = (rr / p.MT) * 8 + x8;
  if (g >= G) return;
  const int h = g / KS, ks = g % KS;
  const int kvh = h / (p.nh / p.nkv);
  const int n_keys = p.L + p.T;
  const int nblk = (n_keys + 31) >> 5;
  const int b0 = min(nblk, ks * p.chunk), b1 = min(nblk, b0 + p.chunk);
  const int cpw = (b1 - b0 + 3) >> 2;
  const int wvs = __builtin_amdgcn_readfirstlane(wave);  // wave index as a scalar
  const int wb0 = min(b1, b0 + wvs * cpw), wb1 = min(b1, wb0 + cpw);
  const int nw = wb1 - wb0;
  const bf16_t *kbase = p.kc + (size_t)kvh * p.cap * 128;
  const bf16_t *vbase = p.vc + (size_t)kvh * 128 * p.cap;
  const u32x4 *zp = (const u32x4 *)p.zeros;
  unsigned char *wl = lds + wave * WAVE_LDS;

  // ---- this lane's queries (B operand) and ancestor masks
  const int tq_l = qt * 16 + lr;
  const bool qlive = tq_l < p.T;
  u32x4 qf[4];
#pragma unroll
  for (int ds = 0; ds < 4; ++ds)
    qf[ds] = *(qlive ? (const u32x4 *)(p.q + ((size_t)tq_l * p.nh + h) * 128 + ds * 32 + lg * 8) : zp);
  const uint64_t mk0 = qlive ? p.mask[2 * tq_l] : 0ull;
  const uint64_t mk1 = qlive ? p.mask[2 * tq_l + 1] : 0ull;

  // ---- register ring.  A block is loaded with 16-byte non-temporal loads:
  // K rows are contiguous (8 KB per block), lane + 64 i covers 16-byte chunk
  // c of it (key c / 16, column c % 16); V^T chunk c is dim row c / 4, keys
  // 8 (c % 4) .. + 7 of the block.
  u32x4 kr[RING][8], vr[RING][8];
  // Past its run a wave re-reads its last block (any in-bounds block does:
  // the data is never staged), so every iteration issues the same loads.
  const int b_last = wb1 > 0 ? wb1 - 1 : 0;
  auto load = [&](int b, u32x4 (&kd)[8], u32x4 (&vd)[8]) {
    const int bb = min(b, b_last);
    const u32x4 *kb = (const u32x4 *)(kbase + (size_t)bb * 32 * 128);
#pragma unroll
    for (int i = 0; i < 8; ++i) kd[i] = __builtin_nontemporal_load(kb + lane + 64 * i);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int c = lane + 64 * i;
      vd[i] = __builtin_nontemporal_load(
          (const u32x4 *)(vbase + (size_t)(c >> 2) * p.cap + bb * 32 + (c & 3) * 8));
    }
  };
  // Block b -> this wave's LDS slot, swizzled (K: physical 16-byte column =
  // logical ^ (row % 16); V^T: logical ^ ((row / 4) % 4)); keys past the
  // last valid one are cleared (value groups; key rows are masked anyway)
  // LDS byte offsets of this lane's chunks (the same for every block)
  int kofs[8], vofs[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int c = lane + 64 * i;
    const int R = row_of_key(c >> 4);
    kofs[i] = R * 256 + (((c & 15) ^ (R & 15)) * 16);
    const int r = c >> 2, cv = c & 3;
    vofs[i] = KSLOT + r * 64 + ((cv ^ ((r >> 2) & 3)) * 16);
  }
  const int vkey = (lane & 3) * 8;  // first key of this lane's value chunks
  auto stage = [&](int b, const u32x4 (&kd)[8], const u32x4 (&vd)[8]) {
#pragma unroll
    for (int i = 0; i < 8; ++i) *(u32x4 *)(wl + kofs[i]) = kd[i];
    const int nv = n_keys - b * 32;  // valid keys in this block (may exceed 32)
    if (nv >= 32) {
#pragma unroll
      for (int i = 0; i < 8; ++i) *(u32x4 *)(wl + vofs[i]) = vd[i];
    } else {
      const int keep_n = nv - vkey;
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        u32x4 v = vd[i];
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          const uint32_t keep = (2 * w < keep_n ? 0xffffu : 0u) | (2 * w + 1 < keep_n ? 0xffff0000u : 0u);
          v[w] &= keep;
        }
        *(u32x4 *)(wl + vofs[i]) = v;
      }
    }
  };

  floatx4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

#pragma unroll
  for (int j = 0; j < RING; ++j) load(wb0 + j, kr[j], vr[j]);
  __builtin_amdgcn_sched_barrier(0);

  for (int c0 = 0; c0 < nw; c0 += RING) {
#pragma unroll
    for (int j = 0; j < RING; ++j) {
      const int i = c0 + j;
      const bool live = i < nw;
      // stage block i (its loads were issued RING blocks ago), then reuse
      // the registers for block i + RING; the wave's own LDS operations run
      // in order, so block i-1's reads precede these writes
      if (live) stage(wb0 + i, kr[j], vr[j]);
      __builtin_amdgcn_sched_barrier(0);
      load(wb0 + i + RING, kr[j], vr[j]);
      __builtin_amdgcn_sched_barrier(0);
      if (!live) continue;
      const unsigned char *ks_l = wl;
      const unsigned char *vs_l = wl + KSLOT;
      const int key0 = (wb0 + i) * 32;
      // S^T for the two 16-key tiles
      floatx4 s[2];
#pragma unroll
      for (int kt = 0; kt < 2; ++kt) {
        s[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ds = 0; ds < 4; ++ds) {
          const u32x4 ka = *(const u32x4 *)(ks_l + (kt * 16 + lr) * 256 + (((ds * 4 + lg) ^ lr) * 16));
          s[kt] = mfma16x16x32(as_bf16x8(ka), as_bf16x8(qf[ds]), s[kt]);
        }
      }
      // scale, mask, block max: this lane holds keys key0 + 8 lg + 4 kt + e
      float sv[8];
      float bmax = -INFINITY;
      if (key0 + 32 <= p.L) {
        // the whole block is cached prefix: visible to every node
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float x = s[kt][e] * p.scale_log2;
            sv[kt * 4 + e] = x;
            bmax = fmaxf(bmax, x);
          }
      } else {
        // this lane's 8 keys key0 + 8 lg .. + 7: visibility bits from the
        // prefix bound and the ancestor mask (bit j - L for tree keys)
        const int j0 = key0 + lg * 8;
        uint32_t visb = 0;
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const int j = j0 + u;
          const int jj = j - p.L;
          const uint64_t word = jj < 64 ? mk0 : mk1;
          const uint32_t anc = (uint32_t)((word >> (jj & 63)) & 1ull);
          visb |= ((uint32_t)(j < p.L) | ((uint32_t)(j < n_keys) & anc)) << u;
        }
#pragma unroll
        for (int kt = 0; kt < 2; ++kt)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const float x = (visb >> (kt * 4 + e)) & 1u ? s[kt][e] * p.scale_log2 : -INFINITY;
            sv[kt * 4 + e] = x;
            bmax = fmaxf(bmax, x);
          }
      }
      bmax = fmaxf(bmax, __shfl_xor(bmax, 16, 64));
      bmax = fmaxf(bmax, __shfl_xor(bmax, 32, 64));
      // no divergence around the MFMAs: a query with nothing visible yet uses
      // a finite reference so that every probability and alpha is exactly 0
      const float m_new = fmaxf(m_run, bmax);
      const float m_ref = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_run - m_ref);
      m_run = m_new;
      float pv[8];
      float psum = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pv[e] = exp2f(sv[e] - m_ref);
        psum += pv[e];
      }
      l_run = l_run * alpha + psum;
      // P = hi + lo, both bf16: the PV product then carries P to ~16
      // significant bits (two MFMAs per tile; the kernel is bound by HBM)
      float plo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) plo[e] = pv[e] - bf16_to_f32(f32_to_bf16(pv[e]));
      const u32x4 pb = u32x4{pack_bf16x2(pv[0], pv[1]), pack_bf16x2(pv[2], pv[3]),
                             pack_bf16x2(pv[4], pv[5]), pack_bf16x2(pv[6], pv[7])};
      const u32x4 pl = u32x4{pack_bf16x2(plo[0], plo[1]), pack_bf16x2(plo[2], plo[3]),
                             pack_bf16x2(plo[4], plo[5]), pack_bf16x2(plo[6], plo[7])};
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) {
        const int r = dt * 16 + lr;
        const u32x4 va = *(const u32x4 *)(vs_l + r * 64 + ((lg ^ ((lr >> 2) & 3)) * 16));
        o[dt] = mfma16x16x32(as_bf16x8(va), as_bf16x8(pb), o[dt] * alpha);
        o[dt] = mfma16x16x32(as_bf16x8(va), as_bf16x8(pl), o[dt]);
      }
    }
  }
  // per-query l over the 4 lane groups (m is already uniform)
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);

  // ---- merge the four waves through LDS (this wave's ring is free now)
  float *ow = (float *)wl;  // [16][OROW]
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) *(floatx4 *)(ow + lr * OROW + dt * 16 + lg * 4) = o[dt];
  if (lg == 0) {
    ml_s[wave][lr][0] = m_run;
    ml_s[wave][lr][1] = l_run;
  }
  __syncthreads();
  // thread -> query tq = tid / 16, dims 8 (tid % 16) .. + 7
  const int tq = threadIdx.x >> 4, d8 = (threadIdx.x & 15) * 8;
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < 4; ++w) M = fmaxf(M, ml_s[w][tq][0]);
  floatx4 acc0 = floatx4{0.f, 0.f, 0.f, 0.f}, acc1 = acc0;
  float lsum = 0.f;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const float mw = ml_s[w][tq][0];
    const float sc = mw == -INFINITY ? 0.f : exp2f(mw - M);
    lsum += sc * ml_s[w][tq][1];
    const float *src = (const float *)(lds + w * WAVE_LDS) + tq * OROW + d8;
    acc0 += sc * *(const floatx4 *)src;
    acc1 += sc * *(const floatx4 *)(src + 4);
  }
  const int t = qt * 16 + tq;
  auto store_out = [&](floatx4 v0, floatx4 v1) {
    bf16_t *dst = p.out + (size_t)t * p.nh * 128 + h * 128 + d8;
    *(u32x4 *)dst = u32x4{pack_bf16x2(v0[0], v0[1]), pack_bf16x2(v0[2], v0[3]),
                          pack_bf16x2(v1[0], v1[1]), pack_bf16x2(v1[2], v1[3])};
  };
  if (KS == 1) {
    if (t < p.T) {
      const float inv = 1.f / lsum;
      store_out(acc0 * inv, acc1 * inv);
    }
    return;
  }

  // ---- publish this split's (O, m, l), rows of OROW floats.  Agent-scope
  // relaxed atomic stores write through to memory that every XCD sees,
  // without the L2 write-back and invalidate that a device fence costs; the
  // ticket is taken only after they have completed, and the last split
  // reads them back with agent-scope atomic loads (never a stale L2 copy).
  const int tile = h * p.MT + qt;
  uint64_t *part = (uint64_t *)(p.part + (size_t)tile * KS * 16 * OROW);
  {
    uint64_t *row = part + ((size_t)ks * 16 + tq) * (OROW / 2);
    const floatx4 v0 = acc0, v1 = acc1;
    __hip_atomic_store(row + d8 / 2, __builtin_bit_cast(uint64_t, float2{v0[0], v0[1]}),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(row + d8 / 2 + 1, __builtin_bit_cast(uint64_t, float2{v0[2], v0[3]}),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(row + d8 / 2 + 2, __builtin_bit_cast(uint64_t, float2{v1[0], v1[1]}),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(row + d8 / 2 + 3, __builtin_bit_cast(uint64_t, float2{v1[2], v1[3]}),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (d8 == 0)
      __hip_atomic_store(row + 64, __builtin_bit_cast(uint64_t, float2{M, lsum}), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev =
        __hip_atomic_fetch_add(&p.counters[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const int last = prev == (unsigned)(KS - 1);
    if (last) __hip_atomic_store(&p.counters[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    last_s = last;
  }
  __syncthreads();
  if (!last_s || t >= p.T) return;

  auto ld2 = [](const uint64_t *a) {
    return __builtin_bit_cast(float2, __hip_atomic_load(a, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
  };
  float Mt = -INFINITY;
  for (int s2 = 0; s2 < KS; ++s2) Mt = fmaxf(Mt, ld2(part + ((size_t)s2 * 16 + tq) * (OROW / 2) + 64).x);
  acc0 = floatx4{0.f, 0.f, 0.f, 0.f};
  acc1 = acc0;
  lsum = 0.f;
  for (int s2 = 0; s2 < KS; ++s2) {
    const uint64_t *row = part + ((size_t)s2 * 16 + tq) * (OROW / 2);
    const float2 ml = ld2(row + 64);
    const float2 a = ld2(row + d8 / 2), b = ld2(row + d8 / 2 + 1);
    const float2 c = ld2(row + d8 / 2 + 2), d = ld2(row + d8 / 2 + 3);
    const float sc = ml.x == -INFINITY ? 0.f : exp2f(ml.x - Mt);
    lsum += sc * ml.y;
    acc0 += sc * floatx4{a.x, a.y, b.x, b.y};
    acc1 += sc * floatx4{c.x, c.y, d.x, d.y};
  }
  const float inv = 1.f / lsum;
  store_out(acc0 * inv, acc1 * inv);
}

}  // namespace

int attn_grid_size(int nh, int splits, int MT) { return ((nh * splits + 7) / 8) * 8 * MT; }

hipError_t launch_attn_bf16(const AttnLaunch &a, hipStream_t s) {
  dim3 grid(attn_grid_size(a.nh, a.splits, a.MT)), block(256);
  if (a.ev_start)
    hipExtLaunchKernelGGL(attn_bf16_kernel, grid, block, 0, s, (hipEvent_t)a.ev_start,
                          (hipEvent_t)a.ev_stop, 0, a);
  else
    hipLaunchKernelGGL(attn_bf16_kernel, grid, block, 0, s, a);
  return hipGetLastError();
}
