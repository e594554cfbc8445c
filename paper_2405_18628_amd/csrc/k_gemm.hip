// Skinny-M GEMMs of the verification forward pass with fused epilogues.
// out[row][t] = sum_k W[row][k] * A[t][k] for the T <= 128 tree tokens t, on
// the gfx950 matrix cores (v_mfma_f32_16x16x32_bf16: weight rows are the
// 16-row A operand, tokens the 16-column B operand), fp32 accumulation.
//
// Precision.  Weights are bf16.  Activations are kept in fp32 in memory and
// enter the matrix cores as the sum of two bf16 parts (hi = bf16(a),
// lo = bf16(a - hi): about 16 significant bits), two products per weight
// fragment.  A bf16 rounding of every activation between layers would make
// two correct implementations drift apart layer after layer (each rounding
// flip is a full bf16 ulp); with the pair the drift stays near fp32 noise at
// any depth.
//
// The step is bound by streaming the weights from HBM once (~T flop per byte
// at bf16, far below the MI355X ridge), so the kernel is organised around
// the weight stream and around what else each compute unit must load:
//  * weights are pre-packed group-major (launch_pack_weight): a group is 16
//    output rows (gate/up: 16 gate rows and the matching 16 up rows), and
//    each 64-column chunk of a group is a run of 1 KB fragments in the lane
//    order of the instruction's A operand; a wave loads them straight into a
//    register ring with 16-byte non-temporal loads (no LDS on this path);
//  * the groups are dealt to eight workgroup sets b % 8 (each runs on one
//    XCD: the dispatcher deals workgroups round-robin over the XCDs) and,
//    within a set, to TX tiles x s K-slices over its 32 workgroups: a
//    tall tile over a slice of K keeps each workgroup's per-chunk work
//    (loading and staging the T x 64 activation chunk as two bf16 planes,
//    two products per fragment, one wave per SIMD) small next to the weight
//    bytes it streams; a whole-K tile of few groups is bound by that work,
//    not by HBM;
//  * the activation chunk (fp32, the same for all of a slice's workgroups,
//    an L2 hit) is staged per chunk in a double-buffered, XOR-swizzled LDS
//    slot as the two bf16 parts; norm consumers form RMSNorm's x * gain here
//    (the row scale is applied to the output rows in the epilogue);
//  * a tile's s slices finish in the same kernel: each stores its partial
//    sums (to L2: all of a tile's workgroups share one XCD), arrives at the
//    tile's counter (an atomic), waits for the others (bounded spin) and
//    finishes its share of the tile (QKV, gate/up: (group, token block)
//    items dealt in turn; the others: whole token blocks), adding the
//    partials in slice order (deterministic);
//  * epilogues: RMSNorm row scale, RoPE + query / key / value stores into the
//    cache (QKV), residual add + per-tile sum of squares (output / down
//    projections), SwiGLU (gate/up), logits + per-tile argmax (LM head).
#include <algorithm>

#include "ppd_internal.h"

namespace {

constexpr int KC = 64;    // K per chunk: two MFMA k-steps
constexpr int FRAG = 64;  // u32x4 per packed operand fragment (1 KB)

template <int KIND>
constexpr int SUB = KIND == GEMM_SWIGLU ? 2 : 1;  // 16-row sub-tiles per group

__device__ __forceinline__ void amax_merge(float &v, int &i, float v2, int i2) {
  if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
    v = v2;
    i = i2;
  }
}

// 16-byte column swizzle of a 128-byte LDS row: logical column c of row r is
// stored at physical column c ^ ((r >> 1) & 7); sixteen consecutive rows read
// at one logical column cover all banks once.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r >> 1) & 7); }

// weight row held by row r (< 16) of sub-tile q of group grp; rows past the
// matrix are padding (zero weights, no output)
template <int KIND>
__device__ __forceinline__ int group_row(int grp, int q, int r, int N) {
  if constexpr (KIND == GEMM_SWIGLU) {
    const int f = grp * 16 + r;  // feature
    return f >= N ? 2 * N : q == 0 ? f : N + f;
  } else if constexpr (KIND == GEMM_QKV) {
    // group gs: dims 8 (gs % 8) .. + 7 of head part gs / 8 in rows 0..7 and
    // their RoPE partners (+ 64) in rows 8..15, so a pair lies in lanes l
    // and l + 32 of the accumulator
    return (grp >> 3) * 128 + (r < 8 ? 0 : 64) + 8 * (grp & 7) + (r & 7);
  } else {
    return grp * 16 + r;
  }
}

// ---- RMSNorm row scale r[t] = 1/sqrt(mean(x^2) + eps) of tokens
// tok0 .. tok0 + NT - 1 from the producer's per-tile sums of squares
// ss[p][T_pad]: two threads per token, thread j adding partials j, j + 2, ...
// in order, then the two sums are added -- the same order whatever NT or the
// other tokens of the step (a batched step gives each sequence its own
// step's bits).
template <int NT>
__device__ __forceinline__ void rs_request(const GemmLaunch &g, int tok0, float (&ssv)[16]) {
  static_assert(2 * NT <= 256, "two threads per token");
  const int tid = threadIdx.x, t = tid % NT, j = tid / NT;
  const int T_pad = g.MT * 16;
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const int pp = j + 2 * i;
    const bool use = tid < 2 * NT && pp < g.n_ss;
    const float v = g.ss[(size_t)(use ? pp : 0) * T_pad + tok0 + t];  // always a valid row
    ssv[i] = use ? v : 0.f;
  }
}

template <int NT>
__device__ __forceinline__ void rs_finish(const GemmLaunch &g, int tok0, const float (&ssv)[16],
                                          float *gs, float *rs_s) {
  const int tid = threadIdx.x;
  const int T_pad = g.MT * 16;
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += ssv[i];
  if (tid < 2 * NT) {
    const int t = tid % NT, j = tid / NT;
    for (int pp = j + 32; pp < g.n_ss; pp += 2) s += g.ss[(size_t)pp * T_pad + tok0 + t];
    gs[tid] = s;
  }
  __syncthreads();
  if (tid < NT) rs_s[tok0 + tid] = rsqrtf((gs[tid] + gs[NT + tid]) * g.inv_h + g.eps);
}

// ---- inputs of an epilogue that come from memory, requested ahead of it
// (one round trip, overlapped with the wait for the partial sums): the
// residual rows (output / down projections) and the RoPE angles (QKV) of the
// lane's rows and token
template <int KIND, int GW>
struct EpiIn {};
template <int GW>
struct EpiIn<GEMM_QKV, GW> {
  floatx4 cs[GW][2];  // (cos, sin) of dims i0 .. i0 + 3
};
template <int GW>
struct EpiIn<GEMM_RESID, GW> {
  floatx4 x[GW];
};

template <int KIND, int GW>
__device__ __forceinline__ void epi_load(const GemmLaunch &g, int ga, int gb, int mt, EpiIn<KIND, GW> &in,
                                         unsigned gmask = ~0u) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int tk = mt * 16 + (lane & 15);
  if constexpr (KIND == GEMM_QKV) {
#pragma unroll
    for (int i = 0; i < GW; ++i) {
      const int gs = ga + wave + 4 * i;
      const int i0 = 8 * (gs & 7) + 4 * ((lane >> 4) & 1);
      const bool use = ((gmask >> i) & 1u) && gs < gb && (gs >> 3) < g.nh + g.nkv;
      const floatx4 *rp = (const floatx4 *)(g.rope + (size_t)(use ? tk : 0) * 64 + (use ? i0 : 0));
      in.cs[i][0] = rp[0];
      in.cs[i][1] = rp[1];
    }
  } else if constexpr (KIND == GEMM_RESID) {
#pragma unroll
    for (int i = 0; i < GW; ++i) {
      const int grp = ga + wave + 4 * i;
      const int n = grp * 16 + (lane >> 4) * 4;
      const bool use = grp < gb && n < g.N && tk < g.T;
      in.x[i] = use ? *(const floatx4 *)(g.x + (size_t)tk * g.N + n) : floatx4{0.f, 0.f, 0.f, 0.f};
    }
  }
}

// ---- epilogue of token block mt of tile gt (groups [ga, gb)), from the
// complete sums a[i][q]: the lane holds rows 4 (lane / 16) + e of sub-tile q
// of its wave's group i (group ga + wave + 4 i), token mt 16 + lane % 16.
// Called by all threads (it has barriers); rs_s holds the row scales, in the
// inputs epi_load requested.
template <int KIND, int GW>
__device__ __forceinline__ void epilogue(const GemmLaunch &g, int gt, int ga, int gb, int mt,
                                         const floatx4 (&a)[GW][SUB<KIND>], const float *rs_s,
                                         float (*red_s)[128][2], const EpiIn<KIND, GW> &in,
                                         unsigned gmask = ~0u) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, r4 = (lane >> 4) * 4;
  const int T = g.T, T_pad = g.MT * 16;
  const int tk = mt * 16 + lr;
  if constexpr (KIND == GEMM_QKV) {
    const int nh = g.nh, nkv = g.nkv;
    const bool upper = lane >= 32;  // rows 8..15: the RoPE partner dims (+64)
    // this token's sequence: its cache and the position L + local index
    bf16_t *kc = g.sb.k[0], *vc = g.sb.v[0];
    int cap = g.sb.cap[0], pos = g.sb.L[0] + tk;
    for (int j = 1; j < g.sb.B; ++j)
      if (tk >= g.sb.t0[j]) {
        kc = g.sb.k[j];
        vc = g.sb.v[j];
        cap = g.sb.cap[j];
        pos = g.sb.L[j] + tk - g.sb.t0[j];
      }
    const float rs = rs_s[tk];  // finite for padding tokens too
#pragma unroll
    for (int i = 0; i < GW; ++i) {
      const int gs = ga + wave + 4 * i;  // uniform in the wave
      if (!((gmask >> i) & 1u) || gs >= gb || gs >= (nh + 2 * nkv) * 8) continue;
      const int hp = gs >> 3;  // head part: q heads, then k, then v
      const int i0 = 8 * (gs & 7) + 4 * ((lane >> 4) & 1);
      const int d0 = i0 + (upper ? 64 : 0);  // this lane's dims d0 .. d0 + 3
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = a[i][0][e] * rs;
      if (hp < nh + nkv) {
        const floatx4 c0 = in.cs[i][0], c1 = in.cs[i][1];  // (cos, sin) of dims i0 .. i0 + 3
        const float cs[8] = {c0[0], c0[1], c0[2], c0[3], c1[0], c1[1], c1[2], c1[3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // [0]: lane l % 32's value (dim i), [1]: lane l % 32 + 32's (dim i + 64)
          const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[e]), __float_as_uint(v[e]),
                                                           false, false);
          const float x0 = __uint_as_float(pr[0]), x1 = __uint_as_float(pr[1]);
          const float c = cs[2 * e], sn = cs[2 * e + 1];
          v[e] = upper ? x1 * c + x0 * sn : x0 * c - x1 * sn;
        }
      }
      if (tk >= T) continue;
      if (hp < nh) {
        *(floatx4 *)(g.q + ((size_t)tk * nh + hp) * 128 + d0) = floatx4{v[0], v[1], v[2], v[3]};
      } else if (hp < nh + nkv) {
        bf16_t *dst = kc + ((size_t)(hp - nh) * cap + pos) * 128;
        *(u32x2 *)(dst + d0) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      } else {
        bf16_t *vb = vc + (size_t)(hp - nh - nkv) * 128 * cap + pos;
#pragma unroll
        for (int e = 0; e < 4; ++e) vb[(size_t)(d0 + e) * cap] = f32_to_bf16(v[e]);
      }
    }
  } else if constexpr (KIND == GEMM_SWIGLU) {
    if (tk < T) {
      const float rs = rs_s[tk];
#pragma unroll
      for (int i = 0; i < GW; ++i) {
        const int grp = ga + wave + 4 * i;
        const int f0 = grp * 16 + r4;
        if (!((gmask >> i) & 1u) || grp >= gb || f0 >= g.N) continue;
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float gt_ = a[i][0][e] * rs, up = a[i][1][e] * rs;
          o[e] = gt_ / (1.f + expf(-gt_)) * up;
        }
        *(floatx4 *)(g.act + (size_t)tk * g.N + f0) = floatx4{o[0], o[1], o[2], o[3]};
      }
    }
  } else if constexpr (KIND == GEMM_RESID) {
    float sq = 0.f;
    if (tk < T) {
#pragma unroll
      for (int i = 0; i < GW; ++i) {
        const int grp = ga + wave + 4 * i;
        const int n = grp * 16 + r4;
        if (grp >= gb || n >= g.N) continue;
        floatx4 xv = in.x[i];
        xv += a[i][0];
        *(floatx4 *)(g.x + (size_t)tk * g.N + n) = xv;
        sq += (xv[0] * xv[0] + xv[1] * xv[1]) + (xv[2] * xv[2] + xv[3] * xv[3]);
      }
    }
    // sum over the 4 lane groups (rows) of this wave, then over the waves
    sq += __shfl_xor(sq, 16, 64);
    sq += __shfl_xor(sq, 32, 64);
    if (lane < 16) red_s[wave][lane][0] = sq;
    __syncthreads();
    if (tid < 16) {
      const int tok = mt * 16 + tid;
      const float v = tok < T ? ((red_s[0][tid][0] + red_s[1][tid][0]) + (red_s[2][tid][0] + red_s[3][tid][0]))
                              : 0.f;
      g.ss_out[(size_t)gt * T_pad + tok] = v;
    }
    __syncthreads();
  } else {  // GEMM_LOGITS
    const float rs = tk < T ? rs_s[tk] : 0.f;
    float bv = 0.f;
    int bi = -1;
#pragma unroll
    for (int i = 0; i < GW; ++i) {
      const int grp = ga + wave + 4 * i;
      const int n = grp * 16 + r4;
      if (grp >= gb || tk >= T) continue;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = a[i][0][e] * rs;
      if (g.logits) {
        if ((g.N & 3) == 0 && n + 3 < g.N) {
          *(floatx4 *)(g.logits + (size_t)tk * g.N + n) = floatx4{v[0], v[1], v[2], v[3]};
        } else {
          for (int e = 0; e < 4; ++e)
            if (n + e < g.N) g.logits[(size_t)tk * g.N + n + e] = v[e];
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
    // merge over the 4 lane groups: larger value, then smaller index
#pragma unroll
    for (int off = 16; off <= 32; off <<= 1) {
      const float v2 = __shfl_xor(bv, off, 64);
      const int i2 = __shfl_xor(bi, off, 64);
      amax_merge(bv, bi, v2, i2);
    }
    if (lane < 16) {
      red_s[wave][lane][0] = bv;
      red_s[wave][lane][1] = __int_as_float(bi);
    }
    __syncthreads();
    if (tid < 16) {
      float v = red_s[0][tid][0];
      int i = __float_as_int(red_s[0][tid][1]);
      for (int w = 1; w < 4; ++w) amax_merge(v, i, red_s[w][tid][0], __float_as_int(red_s[w][tid][1]));
      g.amax[(size_t)gt * T_pad + mt * 16 + tid] = make_float2(v, __int_as_float(i));
    }
    __syncthreads();
  }
}

// tile gt of an XCD holding no group: the outputs other kernels sum over
// every tile are written neutral (sum of squares 0, no argmax candidate)
template <int KIND>
__device__ __forceinline__ void empty_tile(const GemmLaunch &g, int gt) {
  const int T_pad = g.MT * 16;
  for (int tk = threadIdx.x; tk < T_pad; tk += blockDim.x) {
    if constexpr (KIND == GEMM_RESID) g.ss_out[(size_t)gt * T_pad + tk] = 0.f;
    if constexpr (KIND == GEMM_LOGITS) g.amax[(size_t)gt * T_pad + tk] = make_float2(0.f, __int_as_float(-1));
  }
}

// ---- the GEMM.  Workgroup b: XCD x = b % 8, slot j = b / 8 -> tile
// t = j / s (groups [ga, gb) of the XCD's range), K slice ks = j % s (chunks
// [c0, c1)).  Wave w owns groups ga + w + 4 i, i < GW.  RING: weight chunks
// requested ahead.
template <int MT, int KIND, int GW, int RING>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(GemmLaunch g) {
  // activation chunks requested ahead (L2 hits, but ~1 us away under the
  // weight stream): 4, or 2 where 4 chunks of MT tiles would not fit the
  // registers
  constexpr int RA = MT <= 4 ? 4 : 2;
  constexpr int T_pad = MT * 16;
  constexpr int S = SUB<KIND>;
  constexpr int PLANE = T_pad * 128;          // bytes of one bf16 plane of a chunk
  constexpr bool kNorm = KIND != GEMM_RESID;  // A operand = x * gain, rows scaled in the epilogue
  constexpr int UNR = RING > RA ? RING : RA;  // chunks per unrolled trip (both rings wrap)
  static_assert(UNR % RING == 0 && UNR % RA == 0 && UNR % 2 == 0, "ring depths");
  __shared__ __attribute__((aligned(16))) unsigned char lds_a[2][2 * PLANE];
  __shared__ float rs_s[128];
  __shared__ float red_s[4][128][2];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
  const int s = g.s;
  const int t = __builtin_amdgcn_readfirstlane(j / s), ks = __builtin_amdgcn_readfirstlane(j % s);
  const int gt = x * g.TX + t;  // global tile index (sum-of-squares / argmax partial rows)
  const int nx = g.xg0[x + 1] - g.xg0[x];
  const int ga = __builtin_amdgcn_readfirstlane(g.xg0[x] + nx * t / g.TX);
  const int gb = __builtin_amdgcn_readfirstlane(g.xg0[x] + nx * (t + 1) / g.TX);
  const int K = g.K, kc = g.kc;
  const int c0 = __builtin_amdgcn_readfirstlane(kc * ks / s);
  const int c1 = __builtin_amdgcn_readfirstlane(kc * (ks + 1) / s);
  if (ga >= gb) {  // no groups on this tile
    if (ks == 0) empty_tile<KIND>(g, gt);
    return;
  }
  // groups of this wave that exist (uniform in the wave)
  const int live = __builtin_amdgcn_readfirstlane(min(GW, max(0, (gb - ga - wave + 3) / 4)));

  [[maybe_unused]] float ssv[16];
  if constexpr (kNorm) rs_request<T_pad>(g, 0, ssv);

  // ---- register rings.  Weight chunk c of this wave: fragments (group i,
  // sub-tile q, k-step s) for i < GW, read through a buffer resource with
  // the non-temporal hint (offsets from the weight's base; a packed weight
  // is below 2 GB).  Past the slice, and for groups the wave does not own,
  // every lane reads the tile's first 16 bytes (one line), so every
  // iteration issues the same loads.
  const u32x4 *wp = (const u32x4 *)g.W;
  const __amdgpu_buffer_rsrc_t wrs = rsrc_of(g.W, 0x7ffffff0u);
  u32x4 wr[RING][GW * S * 2];
  auto request_w = [&](int c, u32x4(&dw)[GW * S * 2]) {
    const bool cin = c < c1;
#pragma unroll
    for (int i = 0; i < GW; ++i) {
      const bool use = cin && i < live;
      const int grp = use ? ga + wave + 4 * i : ga;
      const int cc = use ? c : c0;
      const u32x4 *gp = wp + (((size_t)grp * kc + cc) * S) * 2 * FRAG + (use ? lane : 0);
#pragma unroll
      for (int q = 0; q < S; ++q)
#pragma unroll
        for (int st = 0; st < 2; ++st)
          dw[(i * S + q) * 2 + st] =
              __builtin_amdgcn_raw_buffer_load_b128(wrs, (int)((gp + (q * 2 + st) * FRAG - wp) * 16), 0, 2);
    }
  };
  // activation pieces of a chunk: thread tid loads 16 bytes (4 columns
  // 4 (tid % 16) ..) of rows tid / 16 + 16 r, r < MT; norm kinds also the 4
  // gains of those columns
  const int acol = (tid & 15) * 4, arow = tid >> 4;
  u32x4 ar[RA][MT];
  [[maybe_unused]] uint2 agn[RA];
  auto request_a = [&](int c, u32x4(&da)[MT], uint2 &gn) {
    const bool cin = c < c1;
    const int k0 = (cin ? c : c0) * KC + acol;
#pragma unroll
    for (int r = 0; r < MT; ++r) da[r] = *(const u32x4 *)(g.A + (size_t)(arow + 16 * r) * K + k0);
    if constexpr (kNorm) gn = *(const uint2 *)(g.gain + k0);
  };
  // stage as the two bf16 parts: plane 0 = hi, plane 1 = lo
  auto stage = [&](const u32x4(&da)[MT], const uint2 &gn, int slot) {
    float gv[4] = {1.f, 1.f, 1.f, 1.f};
    if constexpr (kNorm) {
      gv[0] = bf16_to_f32(gn.x & 0xffff);
      gv[1] = bf16_to_f32(gn.x >> 16);
      gv[2] = bf16_to_f32(gn.y & 0xffff);
      gv[3] = bf16_to_f32(gn.y >> 16);
    }
#pragma unroll
    for (int r = 0; r < MT; ++r) {
      const int row = arow + 16 * r;
      float v[4], lo[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        // padding tokens (rows past T, whatever the workspace holds there)
        // enter as zeros, so their sums are finite
        v[e] = row < g.T ? __uint_as_float(da[r][e]) * gv[e] : 0.f;
        lo[e] = v[e] - bf16_to_f32(f32_to_bf16(v[e]));
      }
      const int off = row * 128 + swz(row, acol >> 3) * 16 + (acol & 7) * 2;
      *(uint2 *)(&lds_a[slot][off]) = uint2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      *(uint2 *)(&lds_a[slot][PLANE + off]) = uint2{pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3])};
    }
  };

  floatx4 acc[GW][S][MT];
#pragma unroll
  for (int i = 0; i < GW; ++i)
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int m = 0; m < MT; ++m) acc[i][q][m] = floatx4{0.f, 0.f, 0.f, 0.f};

#pragma unroll
  for (int r = 0; r < RING; ++r) request_w(c0 + r, wr[r]);
#pragma unroll
  for (int r = 0; r < RA; ++r) request_a(c0 + r, ar[r], agn[r]);
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (kNorm) rs_finish<T_pad>(g, 0, ssv, &red_s[0][0][0], rs_s);
  // rs_s is read after the main loop's barriers; red_s is next written by an
  // epilogue, after them as well

  // ---- main loop, RING chunks per trip.  Chunk c: stage its activations
  // (requested RA chunks ago) into LDS slot (c - c0) & 1, request chunk
  // c + RA's into the freed registers; barrier; multiply with the weight
  // fragments requested RING chunks ago, then request chunk c + RING's into
  // them.  The slot staged here was last read for chunk c - 2, which every
  // wave finished before chunk c - 1's barrier.  Chunks past the slice
  // (the last trip) only stage and load one line.
  for (int cb = c0; cb < c1; cb += UNR) {
#pragma unroll
    for (int r = 0; r < UNR; ++r) {
      const int c = cb + r;
      const int slot = r & 1;  // (c - c0) & 1: UNR is even
      stage(ar[r % RA], agn[r % RA], slot);
      __builtin_amdgcn_sched_barrier(0);
      request_a(c + RA, ar[r % RA], agn[r % RA]);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      if (c < c1) {
        const unsigned char *al = lds_a[slot];
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          u32x4 bh[MT], bl[MT];
#pragma unroll
          for (int m = 0; m < MT; ++m) {
            const int row = m * 16 + lr;
            const int off = row * 128 + swz(row, st * 4 + lg) * 16;
            bh[m] = *(const u32x4 *)(al + off);
            bl[m] = *(const u32x4 *)(al + PLANE + off);
          }
#pragma unroll
          for (int i = 0; i < GW; ++i) {
            if (i >= live) break;
#pragma unroll
            for (int q = 0; q < S; ++q)
#pragma unroll
              for (int m = 0; m < MT; ++m) {
                const bf16x8 w = as_bf16x8(wr[r % RING][(i * S + q) * 2 + st]);
                acc[i][q][m] = mfma16x16x32(w, as_bf16x8(bl[m]), acc[i][q][m]);
                acc[i][q][m] = mfma16x16x32(w, as_bf16x8(bh[m]), acc[i][q][m]);
              }
          }
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      request_w(c + RING, wr[r % RING]);
      __builtin_amdgcn_sched_barrier(0);
    }
  }

  if (s == 1) {  // whole tile: finish in place
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      floatx4 am[GW][S];
#pragma unroll
      for (int i = 0; i < GW; ++i)
#pragma unroll
        for (int q = 0; q < S; ++q) am[i][q] = acc[i][q][m];
      EpiIn<KIND, GW> in;
      epi_load<KIND, GW>(g, ga, gb, m, in);
      epilogue<KIND, GW>(g, gt, ga, gb, m, am, rs_s, red_s, in);
    }
    return;
  }

  // ---- split tile: partials to L2, arrive, wait for the tile's other
  // slices, finish this slice's items.  Item (group i, token block m) is
  // finished by slice fin(i, m): QKV and gate/up deal the tile's items to the
  // slices in turn ((i MT + m) % s); the others keep whole token blocks
  // together (their epilogues reduce over the tile's rows): m % s.  A slice
  // stores the partial sums of the items other slices finish and keeps its
  // own in registers.  Partial (tile gt, slice sl): [wave][i][q][m][lane]
  // floatx4.
  constexpr int PW = GW * S * MT;  // floatx4 per lane per wave
  constexpr bool kItems = KIND == GEMM_QKV || KIND == GEMM_SWIGLU;
  auto fin = [&](int i, int m) { return kItems ? (i * MT + m) % s : m % s; };
  float *part = g.part + ((size_t)gt * s + ks) * (4 * PW * 64 * 4);
#pragma unroll
  for (int i = 0; i < GW; ++i) {
    if (i >= live) break;
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int m = 0; m < MT; ++m)
        if (fin(i, m) != ks)
          *(floatx4 *)(part + ((size_t)((wave * GW + i) * S + q) * MT + m) * 256 + lane * 4) = acc[i][q][m];
  }
  // the items of token block m this slice finishes
  auto mine = [&](int m) {
    unsigned gm = 0;
#pragma unroll
    for (int i = 0; i < GW; ++i) gm |= fin(i, m) == ks ? 1u << i : 0u;
    return gm;
  };
  // the epilogue inputs of this slice's first token block, requested now:
  // they arrive while the partial sums are stored and the slices meet
  int m0 = -1;
  unsigned gm0 = 0;
#pragma unroll
  for (int m = 0; m < MT; ++m)
    if (m0 < 0 && mine(m)) {
      m0 = m;
      gm0 = mine(m);
    }
  EpiIn<KIND, GW> in0;
  if (m0 >= 0) epi_load<KIND, GW>(g, ga, gb, m0, in0, gm0);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0);  // this thread's partial stores have reached L2
  __syncthreads();
  // one 128-byte line of counters per group of XCD slots
  if (tid == 0) xcd_arrive_wait(g.ctr + x * 32 + t, x, (uint32_t)s, g.spin_limit, g.status);
  __syncthreads();
  const float *tile_part = g.part + (size_t)gt * s * (4 * PW * 64 * 4);
  const __amdgpu_buffer_rsrc_t rp = rsrc_of(tile_part, (uint32_t)s * 4 * PW * 64 * 16);
  // the other slices' partials are requested SB at a time (one round trip
  // per batch; past the last slice nothing is loaded) and added in slice
  // order, this slice's own from its registers
  constexpr int SB = GW * S <= 2 ? 8 : 4;
  auto finish_block = [&](int m, unsigned gmask) {
    floatx4 am[GW][S];
#pragma unroll
    for (int i = 0; i < GW; ++i)
#pragma unroll
      for (int q = 0; q < S; ++q) am[i][q] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (int sb = 0; sb < s; sb += SB) {
      floatx4 buf[SB][GW][S];
#pragma unroll
      for (int b = 0; b < SB; ++b) {
        const int sl = sb + b;
#pragma unroll
        for (int i = 0; i < GW; ++i)
#pragma unroll
          for (int q = 0; q < S; ++q) {
            const uint32_t off =
                (uint32_t)((((size_t)sl * 4 * PW + ((wave * GW + i) * S + q) * MT + m) * 64 + lane) * 16);
            buf[b][i][q] = sl < s && sl != ks && i < live && ((gmask >> i) & 1u) ? load_l2(rp, off)
                                                                                 : floatx4{0.f, 0.f, 0.f, 0.f};
          }
      }
#pragma unroll
      for (int b = 0; b < SB; ++b)
        if (sb + b < s) {
#pragma unroll
          for (int i = 0; i < GW; ++i)
#pragma unroll
            for (int q = 0; q < S; ++q) am[i][q] += sb + b == ks ? acc[i][q][m] : buf[b][i][q];
        }
    }
    EpiIn<KIND, GW> in;
    if (m == m0)
      in = in0;
    else
      epi_load<KIND, GW>(g, ga, gb, m, in, gmask);
    epilogue<KIND, GW>(g, gt, ga, gb, m, am, rs_s, red_s, in, gmask);
  };
  if constexpr (kItems) {
#pragma unroll
    for (int m = 0; m < MT; ++m) {
      const unsigned gmask = mine(m);
      if (gmask) finish_block(m, gmask);  // uniform: no barriers in these epilogues
    }
  } else {
#pragma unroll
    for (int m = 0; m < MT; ++m)
      if (m % s == ks) finish_block(m, ~0u);  // uniform in the workgroup
  }
}

template <int MT, int KIND, int GW>
hipError_t launch_mt_gw(const GemmLaunch &g, hipStream_t s) {
  constexpr int WS = GW * SUB<KIND>;  // weight fragment pairs per wave and chunk
  constexpr int RING = WS >= 4 ? 2 : WS >= 2 ? 4 : 8;
  const dim3 grid(8 * g.TX * g.s), block(256);
  hipEvent_t ev0 = (hipEvent_t)g.ev_start, ev1 = (hipEvent_t)g.ev_stop;
  if (ev0)
    hipExtLaunchKernelGGL((gemm_bf16_kernel<MT, KIND, GW, RING>), grid, block, 0, s, ev0, ev1, 0, g);
  else
    hipLaunchKernelGGL((gemm_bf16_kernel<MT, KIND, GW, RING>), grid, block, 0, s, g);
  return hipGetLastError();
}

// groups per wave instantiated for S sub-tiles and MT token tiles: the
// accumulators (GW S MT floatx4) and one chunk's weight fragments (GW S
// pairs) must leave room in one wave's registers
constexpr int gw_limit(int S, int MT) {
  return S == 1 ? (MT <= 4 ? 6 : MT <= 6 ? 4 : 3) : (MT <= 4 ? 3 : MT <= 6 ? 2 : 1);
}

template <int MT, int KIND>
hipError_t launch_mt(const GemmLaunch &g, hipStream_t s) {
  constexpr int LIM = gw_limit(SUB<KIND>, MT);
  switch (g.gw) {
    case 1: return launch_mt_gw<MT, KIND, 1>(g, s);
    case 2:
      if constexpr (LIM >= 2) return launch_mt_gw<MT, KIND, 2>(g, s);
      break;
    case 3:
      if constexpr (LIM >= 3) return launch_mt_gw<MT, KIND, 3>(g, s);
      break;
    case 4:
      if constexpr (LIM >= 4) return launch_mt_gw<MT, KIND, 4>(g, s);
      break;
    case 6:
      if constexpr (LIM >= 6) return launch_mt_gw<MT, KIND, 6>(g, s);
      break;
  }
  return hipErrorInvalidValue;
}

template <int KIND>
hipError_t launch_kind(const GemmLaunch &g, hipStream_t s) {
  switch (g.MT) {
    case 1: return launch_mt<1, KIND>(g, s);
    case 2: return launch_mt<2, KIND>(g, s);
    case 3: return launch_mt<3, KIND>(g, s);
    case 4: return launch_mt<4, KIND>(g, s);
    case 5: return launch_mt<5, KIND>(g, s);
    case 6: return launch_mt<6, KIND>(g, s);
    case 7: return launch_mt<7, KIND>(g, s);
    case 8: return launch_mt<8, KIND>(g, s);
  }
  return hipErrorInvalidValue;
}

// ---- weight packing.  Packed 16-byte item (group, chunk, sub-tile q < S,
// k-step s < 2, lane l < 64) holds the 8 bf16 of weight row
// group_row(group, q, l % 16) at columns 64 chunk + 32 s + 8 (l / 16) .. + 7;
// rows past the matrix are zero.
template <int KIND>
__global__ __launch_bounds__(256) void pack_kernel(const bf16_t *__restrict__ src, u32x4 *__restrict__ dst,
                                                   int N, int K, int rows_total, int kc, long n_items) {
  constexpr int S = SUB<KIND>;
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_items;
       i += (long)gridDim.x * blockDim.x) {
    const int l = (int)(i & 63);
    const long f = i >> 6;  // fragment ((group kc + chunk) S + q) 2 + s
    const int st = (int)(f & 1), q = (int)((f >> 1) % S);
    const long gc = f / (2 * S);
    const int chunk = (int)(gc % kc), grp = (int)(gc / kc);
    const int row = group_row<KIND>(grp, q, l & 15, N);
    const int col = chunk * KC + 32 * st + 8 * (l >> 4);
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row < rows_total && col < K) v = *(const u32x4 *)(src + (size_t)row * K + col);
    dst[i] = v;
  }
}

template <int KIND>
hipError_t launch_pack_kind(int N, int K, const bf16_t *src, bf16_t *dst, hipStream_t s) {
  const int G = gemm_groups_of(KIND, N), kc = K / KC;
  const long n_items = (long)G * kc * SUB<KIND> * 2 * FRAG;
  const int rows_total = KIND == GEMM_SWIGLU ? 2 * N : N;
  const dim3 grid((unsigned)std::min<long>(8192, (n_items + 255) / 256)), block(256);
  hipLaunchKernelGGL((pack_kernel<KIND>), grid, block, 0, s, src, (u32x4 *)dst, N, K, rows_total, kc,
                     n_items);
  return hipGetLastError();
}

}  // namespace

int gemm_groups_of(int kind, int N) {
  // QKV: N / 16 (head_dim 128); gate/up: 16 features per group; others 16 rows
  return (N + 15) / 16;
}

int gemm_sub_of(int kind) { return kind == GEMM_SWIGLU ? 2 : 1; }

int gemm_gw_max(int kind, int MT) { return gw_limit(gemm_sub_of(kind), MT); }

hipError_t launch_pack_weight(int kind, int N, int K, const bf16_t *src, bf16_t *dst, hipStream_t s) {
  if (K % KC) return hipErrorInvalidValue;
  switch (kind) {
    case GEMM_QKV: return launch_pack_kind<GEMM_QKV>(N, K, src, dst, s);
    case GEMM_RESID: return launch_pack_kind<GEMM_RESID>(N, K, src, dst, s);
    case GEMM_SWIGLU: return launch_pack_kind<GEMM_SWIGLU>(N, K, src, dst, s);
    case GEMM_LOGITS: return launch_pack_kind<GEMM_LOGITS>(N, K, src, dst, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_bf16(const GemmLaunch &g, hipStream_t s) {
  switch (g.kind) {
    case GEMM_QKV: return launch_kind<GEMM_QKV>(g, s);
    case GEMM_RESID: return launch_kind<GEMM_RESID>(g, s);
    case GEMM_SWIGLU: return launch_kind<GEMM_SWIGLU>(g, s);
    case GEMM_LOGITS: return launch_kind<GEMM_LOGITS>(g, s);
  }
  return hipErrorInvalidValue;
}
