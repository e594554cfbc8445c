// Split-KV tree attention on the gfx950 matrix cores (Section 4.1: every tree
// node attends to the cached prefix, to its ancestors and to itself).
//
// Keys of one kv head occupy cache positions [0, L + T): the accepted prefix
// [0, L) -- visible to every node -- followed by the tree nodes' own keys
// (written at L + i by the QKV epilogue), visible to node t iff bit i of its
// ancestor mask is set.  The key range is cut into 32-key blocks.
//
// Work decomposition.  The step is bound by reading the keys and values, and
// a compute unit's load path sustains only ~35 GB/s, so the kernel reads
// each key/value block once per compute unit and spreads the blocks over all
// CUs: a workgroup owns one sequence (a batched step packs several, each
// with its own cache and tree), one head h and one of KS contiguous key
// splits (at most one round of workgroups on the CUs), and all of that
// sequence's T queries.  Its eight waves load the split's 64-key block pairs
// cooperatively (16-byte non-temporal loads of whole 128-byte lines into
// registers, the next pair requested while the current one is multiplied),
// stage each pair in a double-buffered LDS slot, and multiply:
// wave w takes the pair's block w / 4 with its 16-query tiles w % 4 (and
// w % 4 + 4), keeping one online softmax per query; the two blocks' waves
// are merged through LDS at the end.  With KS > 1 each query's (O, m, l) is
// stored and the splits are added in split order: for a single sequence
// inside the kernel (a head's splits share an XCD, so they meet in its L2:
// each split, once all have arrived at the head's counter, merges 1 / KS of
// the queries), for a batch by a merge kernel; with KS = 1 the workgroup
// writes the output itself.
//
// Per 32-key block and query tile, on the matrix cores
// (v_mfma_f32_16x16x32_bf16):
//   S^T[key][query] = K Q^T      keys are the 16-row A operand (LDS),
//                                queries the B operand (registers), as two
//                                bf16 parts (hi, lo) of the fp32 queries
//   O^T[d][query]  += V^T P^T    values (stored position-minor, so V^T rows
//                                are contiguous) are the A operand (LDS);
//                                P^T comes straight from S^T's accumulator
//                                layout: LDS row m of key tile kt holds key
//                                8 (m / 4) + 4 kt + (m % 4), so each lane's 8
//                                probabilities are 8 consecutive keys, i.e. a
//                                valid B operand.
// Softmax runs in fp32 in the log2 domain against a lazily moved reference
// (rescaling only when a block's maximum exceeds it by more than 2^8); P
// enters the PV product as the sum of two bf16 parts (hi, lo), i.e. to about
// 16 significant bits.
#include <algorithm>

#include "ppd_internal.h"

namespace {

constexpr int KSLOT = 8192;          // 32 keys x 256 bytes
constexpr int VSLOT = 8192;          // 128 dims x 64 bytes (32 keys)
constexpr int SLOT = KSLOT + VSLOT;  // one block in LDS
constexpr int OROW = PPD_ATTN_OROW;  // partial row: 128 dims, m, l, padding (floats)

// LDS row of the K slot holding key j (j < 32) of a block: MFMA row m of key
// tile kt holds key 8 (m / 4) + 4 kt + (m % 4)
__device__ __forceinline__ int row_of_key(int j) {
  const int a = j >> 3, kt = (j >> 2) & 1, e = j & 3;
  return kt * 16 + a * 4 + e;
}

// s_waitcnt immediate for "at most n vector-memory operations outstanding"
// (expcnt and lgkmcnt left at their maxima, i.e. not waited on)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Reductions over the four 16-lane groups of a wave (lanes l, l ^ 16,
// l ^ 32, l ^ 48) with the gfx950 lane-swap instructions: swapping a value
// with itself across 16-lane (32-lane) halves gives each lane its partner's
// value in one of the two results and its own in the other.
__device__ __forceinline__ float quad_max(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float quad_sum(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// one wave's state for one 16-query tile
struct QTile {
  u32x4 qh[4], ql[4];  // queries (B operand, hi and lo parts), dims 32 ds + 8 (lane / 16) .. + 7
  uint64_t mk0, mk1;
  floatx4 o[8];  // O^T tiles: dims 16 dt + 4 (lane / 16) + e, query lane % 16
  float m_run;   // reference of the exponentials (log2 domain, scaled)
  float l_run;
};

// Merge of one query's KS split rows, 4 dims of a row: the rows are read 8
// at a time (one round trip per batch) and added in split order, scaled to
// the running maximum.  rows(s0, ml, r) loads splits s0 .. s0 + 7 (those
// below KS): ml[v] = (m, l, -, -), r[v] = the 4 dims.
constexpr int MERGE_B = 8;
template <typename ROWS>
__device__ __forceinline__ floatx4 merge_splits(int KS, ROWS rows) {
  constexpr int B = MERGE_B;
  float M = -INFINITY, lsum = 0.f;
  floatx4 acc = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < KS; s0 += B) {
    floatx4 ml[B], r[B];
    rows(s0, ml, r);
    float mb = -INFINITY;
#pragma unroll
    for (int v = 0; v < B; ++v)
      if (s0 + v < KS) mb = fmaxf(mb, ml[v][0]);
    if (mb > M) {
      const float f = exp2f(M - mb);  // 0 while M = -inf (nothing accumulated)
      acc *= f;
      lsum *= f;
      M = mb;
    }
#pragma unroll
    for (int v = 0; v < B; ++v) {
      if (s0 + v < KS) {
        const float sc = ml[v][0] == -INFINITY ? 0.f : exp2f(ml[v][0] - M);
        lsum += sc * ml[v][1];
        acc += sc * r[v];
      }
    }
  }
  return acc * (1.f / lsum);
}

// Eight waves: wave w works on query tiles (w % 4) + 4 i (i < NQ) and on the
// blocks of parity w / 4, so two waves share each SIMD and hide each other's
// latencies; the two parities are merged at the end.  RING: block pairs
// requested ahead.  XM: one sequence, heads dealt to the XCDs, splits merged
// in the kernel.
template <int NQ, int RING, bool XM>
__global__ __launch_bounds__(512, 1) void attn_bf16_kernel(AttnLaunch p) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[4 * SLOT];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int qw = wave & 3, par = wave >> 2;
  const int lr = lane & 15, lg = lane >> 4;
  // this workgroup's sequence (uniform), head and key split
  int sq = 0, h, ks;
  [[maybe_unused]] int xs = 0, h0 = 0;  // XM: the XCD set and its first head
  if constexpr (XM) {
    const int KS = p.splits[0];
    xs = blockIdx.x & 7;
    const int j = blockIdx.x >> 3;
    h0 = p.nh * xs / 8;
    h = h0 + j / KS;
    ks = j % KS;
    if (h >= p.nh * (xs + 1) / 8) return;  // a slot past the XCD's heads
  } else {
    for (int j = 1; j < p.sb.B; ++j) sq = (int)blockIdx.x >= p.wg0[j] ? j : sq;
    const int KS = p.splits[sq];
    const int wl = blockIdx.x - p.wg0[sq];
    h = wl / KS;
    ks = wl % KS;
  }
  const int KS = p.splits[sq];
  const int kvh = h / (p.nh / p.nkv);
  const int t0 = p.sb.t0[sq], T = p.sb.t0[sq + 1] - t0, L = p.sb.L[sq], cap = p.sb.cap[sq];
  const int n_keys = L + T;
  const int nblk = (n_keys + 31) >> 5;
  const int b0 = min(nblk, ks * p.chunk[sq]), b1 = min(nblk, b0 + p.chunk[sq]);
  const int nb = b1 - b0;
  const int nsteps = (nb + 1) >> 1;  // block pairs
  const bf16_t *kbase = p.sb.k[sq] + (size_t)kvh * cap * 128;
  const bf16_t *vbase = p.sb.v[sq] + (size_t)kvh * 128 * cap;
  const u32x4 *zp = (const u32x4 *)p.zeros;

  // ---- this wave's query tiles that exist (tokens t0 + tile 16 + lr)
  const int n_live = min(NQ, ((T + 15) / 16 - qw + 3) / 4);
  QTile qt[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int tl = (qw + 4 * i) * 16 + lr;
    const int tq = t0 + tl;
    const bool qlive = tl < T;
#pragma unroll
    for (int ds = 0; ds < 4; ++ds) {
      const floatx4 *src = qlive ? (const floatx4 *)(p.q + ((size_t)tq * p.nh + h) * 128 + ds * 32 + lg * 8)
                                 : (const floatx4 *)zp;
      const floatx4 a = src[0], b = src[1];
      const float v[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
      float lo[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) lo[e] = v[e] - bf16_to_f32(f32_to_bf16(v[e]));
      qt[i].qh[ds] = u32x4{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                           pack_bf16x2(v[6], v[7])};
      qt[i].ql[ds] = u32x4{pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]), pack_bf16x2(lo[4], lo[5]),
                           pack_bf16x2(lo[6], lo[7])};
    }
    qt[i].mk0 = qlive ? p.mask[2 * tq] : 0ull;
    qt[i].mk1 = qlive ? p.mask[2 * tq + 1] : 0ull;
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) qt[i].o[dt] = floatx4{0.f, 0.f, 0.f, 0.f};
    qt[i].m_run = -INFINITY;
    qt[i].l_run = 0.f;
  }
  __builtin_amdgcn_sched_barrier(0);

  // ---- cooperative loads of a block pair (64 keys), whole 128-byte lines:
  // K chunk c = tid + 512 i (i < 2) of the pair's 16 KB is key c / 16,
  // column c % 16; V^T chunk c is dim row c / 8, keys 8 (c % 8) .. + 7 of the
  // pair.  Key rows past the cache capacity are clamped into it (such keys
  // are never visible, and their values are cleared when staged).  Past the
  // split every lane reads the head's first 16 bytes (offsets masked to 0:
  // one line per load), so every iteration issues the same loads.
  const int b_last = nb > 0 ? b1 - 1 : 0;
  u32x4 kr[RING][2], vr[RING][2];
  auto request = [&](int st, u32x4(&kd)[2], u32x4(&vd)[2]) {
    const int kp0 = min(b0 + 2 * st, b_last) * 32;
    // opaque to the compiler, so that it issues the same loads on every path
    int keep = __builtin_amdgcn_readfirstlane(st < nsteps ? -1 : 0);
    asm volatile("" : "+s"(keep));
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = tid + 512 * i;
      const int key = min(kp0 + (c >> 4), cap - 1);
      kd[i] = __builtin_nontemporal_load((const u32x4 *)(kbase + ((key * 128 + (c & 15) * 8) & keep)));
      const int g0 = min(kp0 + (c & 7) * 8, cap - 8);
      vd[i] = __builtin_nontemporal_load((const u32x4 *)(vbase + (((c >> 3) * cap + g0) & keep)));
    }
  };
  // LDS destinations of this thread's chunks: block parity and byte offset
  // within the block slot.  K row R = row_of_key(key % 32), physical 16-byte
  // column = logical ^ (R % 16); V^T row = dim, physical column = logical ^
  // ((dim / 4) % 4)
  int kofs[2], vofs[2], kpar[2], vpar[2], vgrp[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int c = tid + 512 * i;
    const int k = c >> 4, R = row_of_key(k & 31);
    kpar[i] = k >> 5;
    kofs[i] = R * 256 + (((c & 15) ^ (R & 15)) * 16);
    const int d = c >> 3, g = c & 7;
    vpar[i] = g >> 2;
    vgrp[i] = g & 3;
    // the odd block's V^T rows are stored as row d ^ 2, so that the two
    // blocks' stores from one 16-lane group fall into different banks
    vofs[i] = KSLOT + (d ^ (vpar[i] << 1)) * 64 + (((g & 3) ^ ((d >> 2) & 3)) * 16);
  }
  // block index of pair st, parity q (past the split: beyond the last key)
  auto block_of = [&](int st, int q) { return 2 * st + q < nb ? b0 + 2 * st + q : nblk + 1; };
  auto stage = [&](int st, const u32x4(&kd)[2], const u32x4(&vd)[2]) {
    unsigned char *base = lds + (st & 1) * 2 * SLOT;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *(u32x4 *)(base + kpar[i] * SLOT + kofs[i]) = kd[i];
      *(u32x4 *)(base + vpar[i] * SLOT + vofs[i]) = vd[i];
    }
    // a pair reaching past the last key: clear the values of keys >= n_keys
    // in LDS (their probabilities are 0, but the cache there may hold
    // anything); each thread rewrites only its own chunks
    if (n_keys - block_of(st, 0) * 32 < 64) {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int keep_n = n_keys - block_of(st, vpar[i]) * 32 - vgrp[i] * 8;
        if (keep_n < 8) {
          u32x4 v = vd[i];
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t keep =
                (2 * w < keep_n ? 0xffffu : 0u) | (2 * w + 1 < keep_n ? 0xffff0000u : 0u);
            v[w] &= keep;
          }
          *(u32x4 *)(base + vpar[i] * SLOT + vofs[i]) = v;
        }
      }
    }
  };

#pragma unroll
  for (int j = 0; j < RING; ++j) request(j, kr[j], vr[j]);
  __builtin_amdgcn_sched_barrier(0);
  // the query loads (issued first) have landed; the ring may still fly
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(4 * RING));

  // one block for one query tile
  auto compute = [&](QTile &Q, const unsigned char *sl, int key0) {
    const unsigned char *ks_l = sl;
    const unsigned char *vs_l = sl + KSLOT;
    // S^T for the two 16-key tiles
    floatx4 s[2];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt) {
      s[kt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < 4; ++ds) {
        const u32x4 ka = *(const u32x4 *)(ks_l + (kt * 16 + lr) * 256 + (((ds * 4 + lg) ^ lr) * 16));
        s[kt] = mfma16x16x32(as_bf16x8(ka), as_bf16x8(Q.ql[ds]), s[kt]);
        s[kt] = mfma16x16x32(as_bf16x8(ka), as_bf16x8(Q.qh[ds]), s[kt]);
      }
    }
    // mask and block max: this lane holds keys key0 + 8 lg + 4 kt + e of its
    // query; scores stay unscaled here (the scale c > 0 keeps the order)
    float sv[8];
#pragma unroll
    for (int kt = 0; kt < 2; ++kt)
#pragma unroll
      for (int e = 0; e < 4; ++e) sv[kt * 4 + e] = s[kt][e];
    if (key0 + 32 > L) {
      // this lane's 8 keys key0 + 8 lg .. + 7 (bit u = key j0 + u): visible
      // if in the cached prefix, or a tree key (j - L < T) whose bit j - L of
      // the ancestor mask is set; blocks wholly in the prefix skip this
      const int j0 = key0 + lg * 8;
      const int sh = j0 - L;  // ancestor-mask bit of key j0
      const uint32_t pre = (1u << min(8, max(0, -sh))) - 1u;
      const uint32_t valid = (1u << min(8, max(0, n_keys - j0))) - 1u;
      uint64_t win;  // mask bits sh .. sh + 7 in its low byte (0 below bit 0)
      if (sh >= 128)
        win = 0ull;
      else if (sh >= 64)
        win = Q.mk1 >> (sh - 64);
      else if (sh >= 0)
        win = (Q.mk0 >> sh) | (sh > 56 ? Q.mk1 << (64 - sh) : 0ull);
      else
        win = sh > -8 ? Q.mk0 << -sh : 0ull;
      const uint32_t vis = pre | ((uint32_t)win & valid & 0xffu);
#pragma unroll
      for (int u = 0; u < 8; ++u) sv[u] = (vis >> u) & 1u ? sv[u] : -INFINITY;
    }
    // this lane's maximum over its 8 keys (scaled; the scale c > 0 keeps
    // the order)
    const float c = p.scale_log2;
    const float lmax = c * fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                                 fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
    // Lazy rescaling: the exponentials are taken against a reference (m_run)
    // that moves only when a block's maximum exceeds it by more than 8 (log2
    // units), so probabilities stay below 2^8 and the accumulators are
    // rescaled only then.  The common case needs no exchange between lanes:
    // only when some lane's own maximum exceeds the reference does the wave
    // (all together) reduce the block maximum over each query's four lane
    // groups and move the reference of the queries that need it.
    if (__ballot(lmax > Q.m_run + 8.f)) {
      const float bmax = quad_max(lmax);
      const bool need = bmax > Q.m_run + 8.f;  // the same in a query's four lanes
      // 0 when leaving -inf (nothing accumulated yet), 1 where kept
      const float alpha = need ? __builtin_amdgcn_exp2f(Q.m_run - bmax) : 1.f;
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) Q.o[dt] *= alpha;
      Q.l_run *= alpha;
      Q.m_run = need ? bmax : Q.m_run;
    }
    // a query with nothing visible yet keeps reference -inf: use 0 so that
    // its probabilities are exactly 0
    const float m_eff = Q.m_run == -INFINITY ? 0.f : Q.m_run;
    float pv[8];
    float psum = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pv[e] = __builtin_amdgcn_exp2f(fmaf(sv[e], c, -m_eff));
      psum += pv[e];
    }
    Q.l_run += psum;
    // P = hi + lo, both bf16 (lo the rounding of what hi leaves): the PV
    // product carries P to ~16 significant bits, as the activations are
    // carried (two MFMAs per tile, the smaller part first)
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
      const u32x4 va = *(const u32x4 *)(vs_l + (r ^ (par << 1)) * 64 + ((lg ^ ((lr >> 2) & 3)) * 16));
      Q.o[dt] = mfma16x16x32(as_bf16x8(va), as_bf16x8(pl), Q.o[dt]);
      Q.o[dt] = mfma16x16x32(as_bf16x8(va), as_bf16x8(pb), Q.o[dt]);
    }
  };

  // ---- main loop, RING pairs per trip.  Pair st: stage it (requested RING
  // pairs ago) into LDS slots 2 (st & 1) + parity and request pair st + RING
  // into the freed registers; barrier; every wave multiplies its query tiles
  // with the block of its parity.  The slots staged here were last read for
  // pair st - 2, which every wave finished before pair st - 1's barrier.  The
  // last trip runs whole: its blocks past the split lie beyond the last key
  // (values cleared, nothing visible), so the loop body has no branch around
  // its loads.
  for (int c0 = 0; c0 < nsteps; c0 += RING) {
#pragma unroll
    for (int j = 0; j < RING; ++j) {
      const int st = c0 + j;
      stage(st, kr[j], vr[j]);
      __builtin_amdgcn_sched_barrier(0);
      request(st + RING, kr[j], vr[j]);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      const unsigned char *sl = lds + ((st & 1) * 2 + par) * SLOT;
      const int kb = block_of(st, par);
#pragma unroll
      for (int qi = 0; qi < NQ; ++qi)
        if (qi < n_live) compute(qt[qi], sl, kb * 32);
    }
  }

  // ---- merge the two parities (waves w and w + 4) through LDS, one query
  // tile slot at a time, then the output (KS = 1) or this split's partial
  // row [16 queries][OROW]
  float *mrow = (float *)lds + (size_t)qw * 16 * OROW + lr * OROW;
#pragma unroll
  for (int qi = 0; qi < NQ; ++qi) {
    __syncthreads();  // the LDS ring (or the previous round) is free
    QTile &Q = qt[qi];
    float l = quad_sum(Q.l_run);
    const bool live = qi < n_live;
    if (par == 1 && live) {
#pragma unroll
      for (int dt = 0; dt < 8; ++dt) *(floatx4 *)(mrow + dt * 16 + lg * 4) = Q.o[dt];
      if (lg == 0) *(float2 *)(mrow + 128) = float2{Q.m_run, l};
    }
    __syncthreads();
    if (par == 1 || !live) continue;
    const float2 ml1 = *(const float2 *)(mrow + 128);
    const float M = fmaxf(Q.m_run, ml1.x);
    const float s0 = Q.m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(Q.m_run - M);
    const float s1 = ml1.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml1.x - M);
    floatx4 o[8];
#pragma unroll
    for (int dt = 0; dt < 8; ++dt) o[dt] = Q.o[dt] * s0 + *(const floatx4 *)(mrow + dt * 16 + lg * 4) * s1;
    l = l * s0 + ml1.y * s1;
    const int tile = qw + 4 * qi;
    const int tl = tile * 16 + lr;  // query within the sequence
    if (tl < T) {
      const size_t t = (size_t)t0 + tl;
      if (KS == 1) {
        const float inv = 1.f / l;
        float *dst = p.out + t * p.nh * 128 + h * 128 + lg * 4;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) *(floatx4 *)(dst + dt * 16) = o[dt] * inv;
      } else {
        float *row = p.part + (((size_t)h * p.max_splits + ks) * p.T_pad + t) * OROW;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) *(floatx4 *)(row + dt * 16 + lg * 4) = o[dt];
        if (lg == 0) *(float2 *)(row + 128) = float2{M, l};
      }
    }
  }
  if constexpr (XM) {
    if (KS == 1) return;
    // every split of the head stores its rows (in this XCD's L2) and arrives
    // at the head's counter; then each merges queries [T ks / KS,
    // T (ks + 1) / KS), thread -> query tid / 32, dims 4 (tid % 32) .. + 3
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0);  // this thread's row stores have reached L2
    __syncthreads();
    if (tid == 0) xcd_arrive_wait(p.ctr + xs * 32 + (h - h0), xs, (uint32_t)KS, p.spin_limit, p.status);
    __syncthreads();
    const size_t split_floats = (size_t)p.T_pad * OROW;
    const float *hp = p.part + (size_t)h * p.max_splits * split_floats;
    const __amdgpu_buffer_rsrc_t rp = rsrc_of(hp, (uint32_t)(KS * split_floats * 4));
    const int d4 = (tid & 31) * 4;
    for (int tl = T * ks / KS + (tid >> 5); tl < T * (ks + 1) / KS; tl += 16) {
      const floatx4 o = merge_splits(KS, [&](int s0, floatx4(&ml)[MERGE_B], floatx4(&r)[MERGE_B]) {
#pragma unroll
        for (int v = 0; v < MERGE_B; ++v) {
          const size_t row = (size_t)min(s0 + v, KS - 1) * split_floats + (size_t)tl * OROW;
          ml[v] = load_l2(rp, (uint32_t)((row + 128) * 4));
          r[v] = load_l2(rp, (uint32_t)((row + d4) * 4));
        }
      });
      *(floatx4 *)(p.out + (size_t)(t0 + tl) * p.nh * 128 + h * 128 + d4) = o;
    }
  }
}

// ---- merge of the KS splits of a batch (after the attention kernel):
// workgroup (sequence s and head h, query tile qt); thread -> query
// tq = tid / 32, dims 4 (tid % 32) .. + 3.
__global__ __launch_bounds__(512) void attn_merge_kernel(AttnLaunch p) {
  const int sq = blockIdx.x / p.nh, h = blockIdx.x % p.nh, qt = blockIdx.y;
  const int tq = threadIdx.x >> 5, d4 = (threadIdx.x & 31) * 4;
  const int KS = p.splits[sq];
  const int tl = qt * 16 + tq;
  if (KS == 1 || tl >= p.sb.t0[sq + 1] - p.sb.t0[sq]) return;  // one split: already final
  const size_t t = (size_t)p.sb.t0[sq] + tl;
  const floatx4 o = merge_splits(KS, [&](int s0, floatx4(&ml)[MERGE_B], floatx4(&r)[MERGE_B]) {
#pragma unroll
    for (int v = 0; v < MERGE_B; ++v) {
      const float *row = p.part + (((size_t)h * p.max_splits + min(s0 + v, KS - 1)) * p.T_pad + t) * OROW;
      ml[v] = *(const floatx4 *)(row + 128);
      r[v] = *(const floatx4 *)(row + d4);
    }
  });
  *(floatx4 *)(p.out + t * p.nh * 128 + h * 128 + d4) = o;
}

}  // namespace

hipError_t launch_attn_bf16(const AttnLaunch &a, hipStream_t s) {
  const dim3 grid(a.wg0[a.sb.B]), block(512), mblock(512);
  hipEvent_t ev0 = (hipEvent_t)a.ev_start, ev1 = (hipEvent_t)a.ev_stop;
  int max_ks = 1;
  for (int j = 0; j < a.sb.B; ++j) max_ks = std::max(max_ks, a.splits[j]);
  const bool merge_kernel = max_ks > 1 && !a.xcd_merge;
  hipEvent_t main_stop = merge_kernel ? nullptr : ev1;
  // one pair requested ahead: deeper rings put every workgroup's whole split
  // in flight at once, and the first pairs then arrive later (measured at
  // 7B: 19.2 us per layer with one pair ahead, 22.5 with five)
  auto kernel = a.xcd_merge ? (a.MT > 4 ? attn_bf16_kernel<2, 1, true> : attn_bf16_kernel<1, 1, true>)
                            : (a.MT > 4 ? attn_bf16_kernel<2, 1, false> : attn_bf16_kernel<1, 1, false>);
  if (ev0)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, ev0, main_stop, 0, a);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !merge_kernel) return e;
  const dim3 mgrid(a.nh * a.sb.B, a.MT, 1);
  if (ev1)
    hipExtLaunchKernelGGL(attn_merge_kernel, mgrid, mblock, 0, s, nullptr, ev1, 0, a);
  else
    hipLaunchKernelGGL(attn_merge_kernel, mgrid, mblock, 0, s, a);
  return hipGetLastError();
}
