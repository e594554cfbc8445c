// Skinny-M bfloat16 GEMMs of the verification forward pass, with fused
// epilogues.  out[row][t] = sum_k W[row][k] * A[t][k] for the T <= 128 tree
// tokens t, fp32 accumulation on the gfx950 matrix cores
// (v_mfma_f32_16x16x32_bf16: weight rows are the 16-row A operand, tokens the
// 16-column B operand).
//
// The step is bound by streaming the weights from HBM once (arithmetic
// intensity ~T flop/byte, far below the MI355X ridge), so the kernel is built
// around the weight stream:
//  * a workgroup owns a tile of BN weight rows (128, or 64 for the residual
//    projections) and one slice of K (split-K across workgroups where N alone
//    gives too few tiles);
//  * K is walked in 64-wide chunks.  Each chunk of weights and activations
//    is fetched cooperatively with 16-byte direct-to-LDS transfers
//    (global_load_lds_dwordx4) in which 8 consecutive lanes cover one row's
//    full 128-byte line (the pattern that streams at full HBM rate).  An
//    NS-slot LDS ring keeps NS-1 chunks in flight; 16-byte columns are
//    XOR-swizzled per row pair, so the MFMA operand reads are conflict-free;
//  * each workgroup starts its K walk at its own chunk offset, which spreads
//    the lockstep workgroups over the HBM channels;
//  * each wave owns whole 16-row sub-tiles (two of them, 64 rows apart, for
//    128-row tiles: the RoPE and SwiGLU partners), so no reduction between
//    waves is needed;
//  * split-K partials go to the workspace with agent-scope relaxed atomic
//    stores (coherent across the XCDs without L2 write-back/invalidate); the
//    last workgroup of a tile (atomic ticket) adds them in split order, so
//    results never depend on timing;
//  * the epilogue is fused: RMSNorm row scale, RoPE + query/key/value stores
//    into the cache (QKV), residual add + next norm operand + sum of squares
//    (output / down projection), SwiGLU (gate/up), logits + argmax partials
//    (LM head).
#include "ppd_internal.h"

namespace {

#ifndef PPD_GEMM_NS
#define PPD_GEMM_NS 3
#endif
constexpr int NS = PPD_GEMM_NS;  // LDS ring slots (chunks requested ahead + 1)
constexpr int KC = 64;           // K per chunk: two MFMA k-steps, one 128-byte line per row

template <int KIND>
constexpr int kSub = (KIND == GEMM_RESID) ? 1 : 2;  // 16-row sub-tiles per wave
template <int KIND>
constexpr int kBN = 64 * kSub<KIND>;                 // rows per tile

// weight row of tile row r (0 <= r < BN)
template <int KIND>
__device__ __forceinline__ int tile_row(int tile, int r, int F) {
  if constexpr (KIND == GEMM_SWIGLU) {
    // 64 features: gate rows f0..f0+63, then the matching up rows
    return r < 64 ? tile * 64 + r : F + tile * 64 + (r - 64);
  } else {
    // QKV: tile = one head's 128 rows (dims 0..127); others: consecutive rows
    return tile * kBN<KIND> + r;
  }
}

__device__ __forceinline__ void amax_merge(float &v, int &i, float v2, int i2) {
  if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
    v = v2;
    i = i2;
  }
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(1))) void glb_void_t;

// 16-byte column swizzle of a 128-byte LDS row: logical column c of row r is
// stored at physical column c ^ ((r >> 1) & 7).  Sixteen consecutive rows
// read at one logical column then cover all 64 banks exactly once.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r >> 1) & 7); }

// One 16-byte-per-lane global -> LDS transfer (global_load_lds_dwordx4): lane
// l's 16 bytes land at LDS byte lds_addr + 16 l.  Issued as inline assembly so
// that the compiler does not track the LDS write: its waitcnt pass would
// otherwise drain every transfer in flight before each LDS read; the kernel
// waits explicitly (s_waitcnt vmcnt + barrier) instead.
__device__ __forceinline__ void dma16(const void *g, unsigned lds_addr) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_addr)
               : "memory", "m0");
}

// s_waitcnt immediate for "at most n vector-memory operations outstanding"
// (expcnt and lgkmcnt left at their maxima, i.e. not waited on)
constexpr int vmcnt_imm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }
// s_waitcnt immediate for "no LDS operation outstanding" (vmcnt, expcnt at maxima)
constexpr int lgkmcnt0_imm = 15 | (3 << 14) | (7 << 4);

template <int MT, int KIND>
__global__ __launch_bounds__(256, 2) void gemm_bf16_kernel(GemmLaunch g) {
  constexpr int SUB = kSub<KIND>;
  constexpr int BN = kBN<KIND>;
  constexpr int T_pad = MT * 16;
  constexpr int WBLK = BN / 8;                // 8-row blocks of weights per chunk
  constexpr int ABLK = T_pad / 8;             // 8-row blocks of activations per chunk
  constexpr int NW = WBLK / 4;                // per wave (BN is a multiple of 32)
  constexpr int NA = (ABLK + 3) / 4;          // per wave (excess loads hit a dummy block)
  constexpr int LPC = NW + NA;                // vector loads per wave per chunk
  constexpr int SLOT = (BN + T_pad) * 128;    // bytes of one ring slot
  __shared__ __attribute__((aligned(1024))) unsigned char lds[NS * SLOT + 1024];
  __shared__ float rs_s[128];
  __shared__ float red_s[4][128][2];
  __shared__ int last_s;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15;         // MFMA row (weights) / column (tokens) within a 16-tile
  const int lg = lane >> 4;         // this lane's 16-byte k group within a 32-step
  const int split = blockIdx.x % g.sk;
  const int tile = blockIdx.x / g.sk;
  const int K = g.K;
  const int nks = K >> 5;
  const int k_begin = (int)((long)nks * split / g.sk) * 32;
  const int k_end = (int)((long)nks * (split + 1) / g.sk) * 32;
  const int n_chunks = (k_end - k_begin + KC - 1) / KC;
  const int rows_total = KIND == GEMM_SWIGLU ? 2 * g.N : g.N;

  // ---- load slots.  A wave instruction moves one 8-row block: lane l lands
  // at LDS byte 16 l of the block, i.e. row (l >> 3), physical column l & 7,
  // so it fetches logical column swz(row, l & 7) of that row from memory.
  const int wv = __builtin_amdgcn_readfirstlane(wave);  // wave index as a scalar
  const unsigned lds_base = (unsigned)(size_t)(lds_void_t *)lds;
  const int brow = lane >> 3;
  const bf16_t *wsrc[NW];
  int wcol[NW];
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const int r = (wave + 4 * i) * 8 + brow;
    const int c = swz(r, lane & 7);
    int row = tile_row<KIND>(tile, r, g.N);
    row = row < rows_total ? row : rows_total - 1;
    wsrc[i] = g.W + (size_t)row * K + c * 8;
    wcol[i] = c * 8;
  }
  const bf16_t *asrc[NA];
  int acol[NA];
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int blk = wave + 4 * i;
    const int r = (blk < ABLK ? blk : 0) * 8 + brow;
    const int c = swz(r, lane & 7);
    asrc[i] = g.A + (size_t)r * K + c * 8;
    acol[i] = c * 8;
  }

  floatx4 acc[SUB][MT];
#pragma unroll
  for (int q = 0; q < SUB; ++q)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[q][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Chunk C goes to ring slot C % NS; columns past the slice end (and the
  // padding transfers of waves without an activation block) read 16 zero
  // bytes of the workspace.
  const bf16_t *zp = g.zeros;
  // Each workgroup walks its slice starting at its own chunk offset: all
  // workgroups start together, and rows 8 KB apart otherwise hit the same
  // HBM channels in lockstep.
  const int rot = n_chunks > 0 ? (int)(blockIdx.x % (unsigned)n_chunks) : 0;
  auto issue = [&](int C) {
    const int cc = C < n_chunks ? (C + rot) % n_chunks : C;
    const int k0 = k_begin + cc * KC;
    const unsigned slot = lds_base + (unsigned)((C % NS) * SLOT);
#pragma unroll
    for (int i = 0; i < NW; ++i)
      dma16(k0 + wcol[i] < k_end ? wsrc[i] + k0 : zp, slot + (unsigned)((wv + 4 * i) * 1024));
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int blk = wv + 4 * i;  // scalar
      if (blk < ABLK)
        dma16(k0 + acol[i] < k_end ? asrc[i] + k0 : zp, slot + (unsigned)(BN * 128 + blk * 1024));
      else
        dma16(zp, lds_base + (unsigned)(NS * SLOT));
    }
  };

  for (int c = 0; c < NS - 1 && c < n_chunks; ++c) issue(c);

  // ---- RMSNorm row scale r[t] = 1/sqrt(mean(x^2) + eps) from the
  // producer's sum-of-squares partials, fetched while the first chunks are in
  // flight: group j of the J = 256 / T_pad thread groups sums partials j,
  // j + J, ..., then the group sums are added in group order.
  if constexpr (KIND != GEMM_RESID) {
    constexpr int J = 256 / T_pad;
    float *gs = &red_s[0][0][0];
    if (tid < J * T_pad) {
      const int t = tid % T_pad, j = tid / T_pad;
      float s = 0.f;
      for (int p0 = j; p0 < g.n_ss; p0 += 16 * J) {
        float v[16];
#pragma unroll
        for (int u = 0; u < 16; ++u) {
          const int pp = p0 + u * J;
          const float x = g.ss[(size_t)(pp < g.n_ss ? pp : 0) * T_pad + t];  // a valid row
          v[u] = pp < g.n_ss ? x : 0.f;
        }
#pragma unroll
        for (int u = 0; u < 16; ++u) s += v[u];
      }
      gs[tid] = s;
    }
    __syncthreads();
    if (tid < T_pad) {
      float s = 0.f;
      for (int j = 0; j < J; ++j) s += gs[j * T_pad + tid];
      rs_s[tid] = rsqrtf(s * g.inv_h + g.eps);
    }
    // rs_s is read after the main loop; its write completes before the
    // loop's first barrier
    __builtin_amdgcn_s_waitcnt(lgkmcnt0_imm);
  }

  auto compute = [&](int c) {
    const unsigned char *wl = lds + (c % NS) * SLOT;
    const unsigned char *al = wl + BN * 128;
#pragma unroll
    for (int s = 0; s < KC / 32; ++s) {
      u32x4 wf[SUB], af[MT];
#pragma unroll
      for (int q = 0; q < SUB; ++q) {
        const int r = (wave + 4 * q) * 16 + lr;
        wf[q] = *(const u32x4 *)(wl + r * 128 + swz(r, s * 4 + lg) * 16);
      }
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int r = mt * 16 + lr;
        af[mt] = *(const u32x4 *)(al + r * 128 + swz(r, s * 4 + lg) * 16);
      }
#pragma unroll
      for (int q = 0; q < SUB; ++q)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
          acc[q][mt] = mfma16x16x32(as_bf16x8(wf[q]), as_bf16x8(af[mt]), acc[q][mt]);
    }
  };

  // Steady state: each iteration requests the chunk NS-1 ahead.
  const int n_main = n_chunks - (NS - 1);
  for (int c = 0; c < n_main; ++c) {
    // own transfers of chunk c done (chunks c+1 .. c+NS-2 may still fly),
    // then every wave's; the barrier also retires all reads of chunk c-1,
    // whose slot the next request overwrites.  (A bare s_barrier: a fence
    // would wait for every transfer in flight.)
    __builtin_amdgcn_s_waitcnt(vmcnt_imm((NS - 2) * LPC));
    asm volatile("s_barrier" ::: "memory");
    issue(c + NS - 1);
    compute(c);
  }

  // Epilogue operands, requested now so that their latency overlaps the
  // last chunks' (RoPE factors for QKV; residual stream and next norm gain
  // for the residual projections).
  const int r4 = (lane >> 4) * 4;  // accumulator rows 4 (lane / 16) + e
  [[maybe_unused]] floatx4 rope_r[MT][2];
  [[maybe_unused]] floatx4 x_r[MT];
  [[maybe_unused]] uint2 gain_r;
  if constexpr (KIND == GEMM_QKV) {
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const floatx4 *rp = (const floatx4 *)(g.rope + (size_t)(mt * 16 + lr) * 64 + wave * 16 + r4);
      rope_r[mt][0] = rp[0];
      rope_r[mt][1] = rp[1];
    }
  } else if constexpr (KIND == GEMM_RESID) {
    const int n = tile * 64 + wave * 16 + r4;
    gain_r = *(const uint2 *)(g.gain + n);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) x_r[mt] = *(const floatx4 *)(g.x + (size_t)(mt * 16 + lr) * g.N + n);
  }

  // Tail: the last chunks are all requested already; wait for them once
  // (no padding transfers whose latency every workgroup would wait out).
  __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
  asm volatile("s_barrier" ::: "memory");
  for (int c = n_main > 0 ? n_main : 0; c < n_chunks; ++c) compute(c);

  // ---- split-K: publish the partial tile; the last workgroup sums all.
  // Partials are written and read with agent-scope relaxed atomics (coherent
  // across the XCDs without writing back or invalidating whole L2 caches);
  // every store has completed (vmcnt 0) before the ticket is taken.
  if (g.sk > 1) {
    constexpr size_t tile_u64 = (size_t)4 * SUB * MT * 64 * 2;
    {
      uint64_t *dst = (uint64_t *)g.part + (size_t)blockIdx.x * tile_u64;
#pragma unroll
      for (int q = 0; q < SUB; ++q)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
          const size_t o = (size_t)(((wave * SUB + q) * MT + mt) * 64 + lane) * 2;
          const floatx4 r = acc[q][mt];
          __hip_atomic_store(dst + o, __builtin_bit_cast(uint64_t, float2{r[0], r[1]}),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(dst + o + 1, __builtin_bit_cast(uint64_t, float2{r[2], r[3]}),
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
      const unsigned prev =
          __hip_atomic_fetch_add(&g.counters[tile], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int last = prev == (unsigned)(g.sk - 1);
      if (last) __hip_atomic_store(&g.counters[tile], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_s = last;
    }
    __syncthreads();
    if (!last_s) return;
#pragma unroll
    for (int q = 0; q < SUB; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[q][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    // U splits' partials are requested together, then added in split order
    constexpr int U = SUB * MT <= 4 ? 4 : (SUB * MT <= 8 ? 2 : 1);
    for (int s0 = 0; s0 < g.sk; s0 += U) {
      float2 buf[U][SUB][MT][2];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int s = s0 + u < g.sk ? s0 + u : s0;
        const uint64_t *src = (const uint64_t *)g.part + (size_t)(tile * g.sk + s) * tile_u64;
#pragma unroll
        for (int q = 0; q < SUB; ++q)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const size_t o = (size_t)(((wave * SUB + q) * MT + mt) * 64 + lane) * 2;
            buf[u][q][mt][0] = __builtin_bit_cast(
                float2, __hip_atomic_load(src + o, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
            buf[u][q][mt][1] = __builtin_bit_cast(
                float2, __hip_atomic_load(src + o + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
          }
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (s0 + u < g.sk)
#pragma unroll
          for (int q = 0; q < SUB; ++q)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[q][mt] += floatx4{buf[u][q][mt][0].x, buf[u][q][mt][0].y, buf[u][q][mt][1].x,
                                    buf[u][q][mt][1].y};
    }
  }

  // accumulator layout: lane holds rows 4 (lane / 16) + e of its sub-tile,
  // token column lane % 16 of token tile mt
  const int T = g.T;

  if constexpr (KIND == GEMM_QKV) {
    const int hp = tile;                // head part: q heads, then k, then v
    const int i0 = wave * 16 + r4;      // dims i0..i0+3 and their partners +64
    const int nh = g.nh, nkv = g.nkv;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      if (t >= T) continue;
      const float rs = rs_s[t];
      float lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = acc[0][mt][e] * rs;
        hi[e] = acc[1][mt][e] * rs;
      }
      if (hp < nh + nkv) {
        const float cs_all[8] = {rope_r[mt][0][0], rope_r[mt][0][1], rope_r[mt][0][2], rope_r[mt][0][3],
                                 rope_r[mt][1][0], rope_r[mt][1][1], rope_r[mt][1][2], rope_r[mt][1][3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float2 cs = float2{cs_all[2 * e], cs_all[2 * e + 1]};
          const float a = lo[e], b = hi[e];
          lo[e] = a * cs.x - b * cs.y;
          hi[e] = b * cs.x + a * cs.y;
        }
        const u32x2 plo = u32x2{pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3])};
        const u32x2 phi = u32x2{pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3])};
        bf16_t *dst = hp < nh ? g.q + ((size_t)t * nh + hp) * 128
                              : g.kc + ((size_t)(hp - nh) * g.cap + g.L + t) * 128;
        *(u32x2 *)(dst + i0) = plo;
        *(u32x2 *)(dst + i0 + 64) = phi;
      } else {
        bf16_t *vb = g.vc + (size_t)(hp - nh - nkv) * 128 * g.cap + g.L + t;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          vb[(size_t)(i0 + e) * g.cap] = f32_to_bf16(lo[e]);
          vb[(size_t)(i0 + e + 64) * g.cap] = f32_to_bf16(hi[e]);
        }
      }
    }
  } else if constexpr (KIND == GEMM_SWIGLU) {
    const int f0 = tile * 64 + wave * 16 + r4;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      if (t >= T) continue;
      const float rs = rs_s[t];
      float a[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float gt = acc[0][mt][e] * rs, up = acc[1][mt][e] * rs;
        a[e] = gt / (1.f + expf(-gt)) * up;
      }
      *(u32x2 *)(g.act + (size_t)t * g.N + f0) =
          u32x2{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3])};
    }
  } else if constexpr (KIND == GEMM_RESID) {
    const int n = tile * 64 + wave * 16 + r4;
    const uint2 gw = gain_r;
    const float g0 = bf16_to_f32(gw.x & 0xffff), g1 = bf16_to_f32(gw.x >> 16);
    const float g2 = bf16_to_f32(gw.y & 0xffff), g3 = bf16_to_f32(gw.y >> 16);
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      float sq = 0.f;
      if (t < T) {
        float *xp = g.x + (size_t)t * g.N + n;
        floatx4 xv = x_r[mt];
        xv += acc[0][mt];
        *(floatx4 *)xp = xv;
        *(u32x2 *)(g.xg + (size_t)t * g.N + n) =
            u32x2{pack_bf16x2(xv[0] * g0, xv[1] * g1), pack_bf16x2(xv[2] * g2, xv[3] * g3)};
        sq = (xv[0] * xv[0] + xv[1] * xv[1]) + (xv[2] * xv[2] + xv[3] * xv[3]);
      }
      // sum over the 4 lane groups (rows) of this wave
      sq += __shfl_xor(sq, 16, 64);
      sq += __shfl_xor(sq, 32, 64);
      if (lane < 16) red_s[wave][t][0] = sq;
    }
    __syncthreads();
    if (tid < T_pad) {
      const float v = tid < T ? ((red_s[0][tid][0] + red_s[1][tid][0]) +
                                 (red_s[2][tid][0] + red_s[3][tid][0]))
                              : 0.f;
      g.ss_out[(size_t)tile * T_pad + tid] = v;
    }
  } else {  // GEMM_LOGITS
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      const float rs = t < T ? rs_s[t] : 0.f;
      float bv = 0.f;
      int bi = -1;
#pragma unroll
      for (int q = 0; q < SUB; ++q) {
        const int n = tile * BN + (wave + 4 * q) * 16 + r4;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[q][mt][e] * rs;
        if (t < T) {
          if (g.logits) {
            if ((g.N & 3) == 0 && n + 3 < g.N) {
              *(floatx4 *)(g.logits + (size_t)t * g.N + n) = floatx4{v[0], v[1], v[2], v[3]};
            } else {
              for (int e = 0; e < 4; ++e)
                if (n + e < g.N) g.logits[(size_t)t * g.N + n + e] = v[e];
            }
          }
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (n + e < g.N) {
              if (v[e] != v[e]) {
                atomicOr(g.status, PPD_DEV_NAN_LOGIT);
              } else if (bi < 0 || v[e] > bv) {
                bv = v[e];
                bi = n + e;
              }
            }
          }
        }
      }
      // merge over the 4 lane groups: larger value, then smaller index
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float v2 = __shfl_xor(bv, o, 64);
        const int i2 = __shfl_xor(bi, o, 64);
        amax_merge(bv, bi, v2, i2);
      }
      if (lane < 16) {
        red_s[wave][t][0] = bv;
        red_s[wave][t][1] = __int_as_float(bi);
      }
    }
    __syncthreads();
    if (tid < T_pad) {
      float v = red_s[0][tid][0];
      int i = __float_as_int(red_s[0][tid][1]);
      for (int w = 1; w < 4; ++w) amax_merge(v, i, red_s[w][tid][0], __float_as_int(red_s[w][tid][1]));
      g.amax[(size_t)tile * T_pad + tid] = make_float2(v, __int_as_float(i));
    }
  }
}

template <int KIND>
hipError_t launch_kind(const GemmLaunch &g, int n_tiles, hipStream_t s) {
  dim3 grid(n_tiles * g.sk), block(256);
  switch (g.MT) {
#define PPD_CASE(M) \
  case M:                                                                                   \
    if (g.ev_start)                                                                         \
      hipExtLaunchKernelGGL((gemm_bf16_kernel<M, KIND>), grid, block, 0, s,                 \
                            (hipEvent_t)g.ev_start, (hipEvent_t)g.ev_stop, 0, g);           \
    else                                                                                    \
      hipLaunchKernelGGL((gemm_bf16_kernel<M, KIND>), grid, block, 0, s, g);                \
    break;
    PPD_CASE(1) PPD_CASE(2) PPD_CASE(3) PPD_CASE(4) PPD_CASE(5) PPD_CASE(6) PPD_CASE(7) PPD_CASE(8)
#undef PPD_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

int gemm_tile_rows(int kind) { return kind == GEMM_RESID ? 64 : 128; }

hipError_t launch_gemm_bf16(const GemmLaunch &g, int n_tiles, hipStream_t s) {
  switch (g.kind) {
    case GEMM_QKV: return launch_kind<GEMM_QKV>(g, n_tiles, s);
    case GEMM_RESID: return launch_kind<GEMM_RESID>(g, n_tiles, s);
    case GEMM_SWIGLU: return launch_kind<GEMM_SWIGLU>(g, n_tiles, s);
    case GEMM_LOGITS: return launch_kind<GEMM_LOGITS>(g, n_tiles, s);
  }
  return hipErrorInvalidValue;
}
