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
constexpr int SLOT = KSLOT + VSLOT;       // one ring slot
constexpr int QBYTES = 4096;              // 16 queries x 256 bytes
constexpr int MBYTES = 1024;              // ancestor masks (16 x 16 bytes used)
constexpr int WAVE_LDS = 2 * SLOT + QBYTES + MBYTES;
constexpr int OROW = 132;                 // merge row: 128 dims + padding (floats)

typedef __attribute__((address_space(3))) void lds_void_t;

// One 16-byte-per-lane global -> LDS transfer: lane l's bytes land at LDS
// byte lds_addr + 16 l.  Inline assembly, so that the compiler does not
// track the LDS write (the kernel waits on vmcnt explicitly).
__device__ __forceinline__ void dma16(const void *g, unsigned lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_addr)
               : "memory", "m0");
}

// key (within its 32-key block) held by LDS row R of the block's K slot
__device__ __forceinline__ int key_of_row(int R) {
  const int kt = R >> 4, m = R & 15;
  return 8 * (m >> 2) + 4 * kt + (m & 3);
}

__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnLaunch p) {
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
  const int wb0 = min(b1, b0 + wave * cpw), wb1 = min(b1, wb0 + cpw);
  const int nw = wb1 - wb0;
  const bf16_t *kbase = p.kc + (size_t)kvh * p.cap * 128;
  const bf16_t *vbase = p.vc + (size_t)kvh * 128 * p.cap;
  const bf16_t *zp = p.zeros;

  const int wv = __builtin_amdgcn_readfirstlane(wave);
  const unsigned wbase = (unsigned)(size_t)(lds_void_t *)lds + (unsigned)(wv * WAVE_LDS);
  unsigned char *wl = lds + wave * WAVE_LDS;

  // ---- queries and masks of the tile -> this wave's LDS
  {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row = 4 * i + (lane >> 4);
      const int t = qt * 16 + row;
      dma16(t < p.T ? (const void *)(p.q + ((size_t)t * p.nh + h) * 128 + (lane & 15) * 8) : zp,
            wbase + 2 * SLOT + i * 1024);
    }
    const int t = qt * 16 + lane;
    dma16(lane < 16 && t < p.T ? (const void *)(p.mask + 2 * t) : zp, wbase + 2 * SLOT + QBYTES);
  }

  // ---- per-lane transfer offsets of a block (elements from the block start)
  int koff[8], voff[8], vkey[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    // K: LDS row R = 4 i + lane / 16 (256 bytes), physical 16-byte column
    // lane % 16 holds logical column c = phys ^ (R % 16)
    const int R = 4 * i + (lane >> 4);
    const int c = (lane & 15) ^ (R & 15);
    koff[i] = key_of_row(R) * 128 + c * 8;
    // V^T: LDS row r = 16 i + lane / 4 (64 bytes), physical column lane % 4
    // holds logical column (8 keys) c = phys ^ ((r / 4) % 4)
    const int r = 16 * i + (lane >> 2);
    const int cv = (lane & 3) ^ ((r >> 2) & 3);
    voff[i] = r * p.cap + cv * 8;
    vkey[i] = cv * 8;
  }
  int kkey[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) kkey[i] = key_of_row(4 * i + (lane >> 4));

  // Block b (of this wave's run; past the run: zero lines) -> ring slot s.
  // Keys past the end read zeros, except the tail of a partly valid
  // 8-key value group, which is cleared in LDS after arrival.
  auto issue = [&](int b, int s) {
    const bool in_run = b < wb1;
    const int key0 = b * 32;
    const unsigned slot = wbase + (unsigned)(s * SLOT);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      dma16(in_run && key0 + kkey[i] < n_keys ? (const void *)(kbase + (size_t)key0 * 128 + koff[i]) : zp,
            slot + i * 1024);
#pragma unroll
    for (int i = 0; i < 8; ++i)
      dma16(in_run && key0 + vkey[i] < n_keys ? (const void *)(vbase + key0 + voff[i]) : zp,
            slot + KSLOT + i * 1024);
  };

  floatx4 o[8];
#pragma unroll
  for (int dt = 0; dt < 8; ++dt) o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  issue(wb0, 0);
  issue(wb0 + 1, 1);
  asm volatile("s_waitcnt vmcnt(16)" ::: "memory");  // queries, masks, block 0

  if (nw > 0) {
    u32x4 qf[4];
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) qf[ds] = *(const u32x4 *)(wl + 2 * SLOT + lr * 256 + (ds * 4 + lg) * 16);
    const uint64_t mk0 = *(const uint64_t *)(wl + 2 * SLOT + QBYTES + lr * 16);
    const uint64_t mk1 = *(const uint64_t *)(wl + 2 * SLOT + QBYTES + lr * 16 + 8);

    for (int i = 0; i < nw; ++i) {
      if (i > 0) {
        issue(wb0 + i + 1, (i + 1) & 1);  // into the slot block i-1 used
        asm volatile("s_waitcnt vmcnt(16)" ::: "memory");  // block i arrived
      }
      const unsigned char *ks_l = wl + (i & 1) * SLOT;
      const unsigned char *vs_l = ks_l + KSLOT;
      const int key0 = (wb0 + i) * 32;
      const int nv = n_keys - key0;  // valid keys in this block (may exceed 32)
      if (nv < 32 && (nv & 7)) {
        // clear the invalid tail of the partly valid 8-key group, rows lane, lane + 64
        const int c = nv >> 3;
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const int r = lane + 64 * hh;
          u32x4 *ptr = (u32x4 *)(wl + (i & 1) * SLOT + KSLOT + r * 64 + ((c ^ ((r >> 2) & 3)) * 16));
          u32x4 v = *ptr;
          const int keep_n = nv & 7;
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t keep = (2 * w < keep_n ? 0xffffu : 0u) | (2 * w + 1 < keep_n ? 0xffff0000u : 0u);
            v[w] &= keep;
          }
          *ptr = v;
        }
      }
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
#pragma unroll
      for (int kt = 0; kt < 2; ++kt)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int j = key0 + lg * 8 + kt * 4 + e;
          const int jj = j - p.L;  // tree node index of key j (if j >= L)
          const uint64_t word = jj < 64 ? mk0 : mk1;
          const int anc = (int)((word >> (jj & 63)) & 1ull);
          const int vis = (j < p.L) | ((j < n_keys) & anc);
          const float x = vis ? s[kt][e] * p.scale_log2 : -INFINITY;
          sv[kt * 4 + e] = x;
          bmax = fmaxf(bmax, x);
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
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // trailing zero-line transfers

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
