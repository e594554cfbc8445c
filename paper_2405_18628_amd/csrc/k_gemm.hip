// Skinny-M bfloat16 GEMMs of the verification forward pass, with fused
// epilogues.  out[row][t] = sum_k W[row][k] * A[t][k] for the T <= 128 tree
// tokens t, fp32 accumulation on the gfx950 matrix cores
// (v_mfma_f32_16x16x32_bf16: weight rows are the 16-row A operand, tokens the
// 16-column B operand).
//
// The step is bound by streaming the weights from HBM once (arithmetic
// intensity ~T flop/byte, far below the MI355X ridge), so the kernel is built
// around the weight stream:
//  * weights are pre-packed (launch_pack_weight) so that every MFMA operand
//    fragment -- 16 rows x 32 columns, in the lane order the instruction
//    reads it -- is one contiguous 1 KB; a wave loads its fragments straight
//    into registers with 16-byte non-temporal loads, PPD_GEMM_RING chunks
//    ahead, with no LDS on the weight path (weights are not shared between
//    waves);
//  * the activations (the same for every workgroup, served from L2) follow
//    the same register ring and are staged per chunk in a double-buffered,
//    XOR-swizzled LDS slot read by the four waves;
//  * a compute unit's load path sustains only ~35 GB/s, so a GEMM needs
//    (nearly) every CU streaming to approach the HBM rate.  GEMMs with enough
//    tiles (128 rows; QKV: 64, half a head) run one whole tile per workgroup
//    and finish it in place (fused epilogue).  The others are cut Stream-K
//    style: the (tile, chunk) units are split into equal contiguous ranges,
//    one per compute unit; a workgroup streams across tile boundaries and
//    stores the partial sums of each tile segment, and a small finish kernel
//    (one workgroup per tile and 16-token block) adds a tile's partials in
//    workgroup order and runs the epilogue -- the kernel boundary orders the
//    two, so no cross-workgroup synchronisation is needed and results never
//    depend on timing;
//  * the epilogue: RMSNorm row scale, RoPE + query/key/value stores into the
//    cache (QKV), residual add + next norm operand + sum of squares (output /
//    down projection), SwiGLU (gate/up), logits + argmax partials (LM head).
#include <algorithm>

#include "ppd_internal.h"

namespace {

constexpr int KC = 64;            // K per chunk: two MFMA k-steps
constexpr int BN = PPD_GEMM_BN;   // rows of a 128-row tile: 8 sub-tiles of 16
constexpr int R = PPD_GEMM_RING;  // chunks requested ahead
constexpr int FRAG = 64;          // u32x4 per packed operand fragment (1 KB)
// Ring depth of 3- and 2-group whole tiles (needs K % 512 == 0).  Measured at 7B:
// with 3 of 4 waves streaming weights a 4-chunk ring keeps too few bytes in
// flight (QKV 30.0, gate/up 40.1 us against 28.9 / 37.5 with 4-group tiles);
// 8 chunks give 28.1 / 35.9 us.  4-group tiles and split GEMMs are slower
// with 8 (gate/up 38.5, output / down projection 18.9 / 28.2 against 17.3 /
// 26.2 us).
constexpr int kRing3 = 8;

// A tile holds NS row groups, each of SUBS sub-tiles of 16 rows: wave w
// owns group w, i.e. sub-tiles w (QKV: 16 rows, 8 dims of a head and their
// RoPE partners) or w and w + NS (SwiGLU: 16 gate rows and the matching 16
// up rows; others: 16 + 16 consecutive rows).  NS = 4 gives 64-row QKV tiles
// (half a head), 64 features per gate/up tile and 128-row tiles elsewhere.
// Whole-tile QKV and gate/up GEMMs may take smaller tiles where that spreads
// them over more CUs: NS = 3 (waves 0-2 own the groups, wave 3 only stages
// activations; 7B: 256 QKV tiles instead of 192, 230 gate/up tiles instead
// of 172) or NS = 2 (waves w and w + 2 share group w, each multiplying one of
// the two k-steps of every chunk, and add their sums through LDS at the end;
// 1.4B: 176 whole gate/up tiles instead of a split GEMM).
template <int KIND>
constexpr int SUBS = KIND == GEMM_QKV ? 1 : 2;
// u32x4 per packed (tile, chunk): NS SUBS sub-tiles x 2 k-steps
template <int KIND, int NS>
constexpr int UNIT = 2 * NS * SUBS<KIND> * FRAG;

// weight row of tile row r (0 <= r < 16 NS SUBS); rows >= the matrix's are
// padding (zero weights, no output)
template <int KIND, int NS>
__device__ __forceinline__ int tile_row(int tile, int r, int N) {
  if constexpr (KIND == GEMM_SWIGLU) {
    // 16 NS features: gate rows f0 .. f0 + 16 NS - 1, then the matching up rows
    constexpr int FT = 16 * NS;
    const int f = tile * FT + (r < FT ? r : r - FT);
    return f >= N ? 2 * N : r < FT ? f : N + f;  // features past F: padding
  } else if constexpr (KIND == GEMM_QKV) {
    // global sub-tile gs: sub-tile gs % 8 of head part gs / 8; its rows 0..7
    // are dims 8 (gs % 8) .. + 7, rows 8..15 their RoPE partners 64 + those
    // dims, so a pair lies in lanes l and l + 32 of the accumulator
    const int gs = tile * NS + (r >> 4), rr = r & 15;
    return (gs >> 3) * 128 + (rr < 8 ? 0 : 64) + 8 * (gs & 7) + (rr & 7);
  } else {
    return tile * BN + r;  // consecutive rows
  }
}

__device__ __forceinline__ void amax_merge(float &v, int &i, float v2, int i2) {
  if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
    v = v2;
    i = i2;
  }
}

// 16-byte column swizzle of a 128-byte LDS row: logical column c of row r is
// stored at physical column c ^ ((r >> 1) & 7).  Sixteen consecutive rows
// read at one logical column then cover all 64 banks exactly once.
__device__ __forceinline__ int swz(int r, int c) { return c ^ ((r >> 1) & 7); }

// ---- RMSNorm row scale r[t] = 1/sqrt(mean(x^2) + eps) of tokens
// tok0 .. tok0 + NT - 1 from the producer's sum-of-squares partials
// ss[p][T_pad]: two threads per token, thread j adding partials j, j + 2,
// j + 4, ... in order (the first 16 requested by rs_request, so that a caller
// can overlap their latency), then the two sums are added.  The order is the
// same whatever NT, so a token's scale does not depend on the other tokens
// of the step (a batched step gives each sequence its own step's bits).
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

// ---- epilogue operands
template <int KIND, int MTE>
struct EpiOperands {
  floatx4 rope[MTE][2];  // QKV: (cos, sin) of dims i0..i0+3 for each token tile
  floatx4 x[2][MTE];     // RESID: residual stream of the lane's rows
  uint2 gain[2];         // RESID: next norm gain of the lane's rows
};

template <int KIND, int MTE, int NS = 4>
__device__ __forceinline__ void epi_request(const GemmLaunch &g, int t, int mt0,
                                            EpiOperands<KIND, MTE> &o) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int lr = lane & 15, r4 = (lane >> 4) * 4;
  if constexpr (KIND == GEMM_QKV) {
    // pair indices 8 (gs % 8) + 4 (lane / 16 % 2) + e, e < 4, of the wave's
    // global sub-tile gs (waves >= NS read a valid pair and do not use it)
    const int i0 = 8 * ((t * NS + wave) & 7) + 4 * ((lane >> 4) & 1);
#pragma unroll
    for (int mt = 0; mt < MTE; ++mt) {
      const floatx4 *rp = (const floatx4 *)(g.rope + (size_t)((mt0 + mt) * 16 + lr) * 64 + i0);
      o.rope[mt][0] = rp[0];
      o.rope[mt][1] = rp[1];
    }
  } else if constexpr (KIND == GEMM_RESID) {
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int n = t * BN + (wave + 4 * q) * 16 + r4;
      o.gain[q] = *(const uint2 *)(g.gain + n);
#pragma unroll
      for (int mt = 0; mt < MTE; ++mt)
        o.x[q][mt] = *(const floatx4 *)(g.x + (size_t)((mt0 + mt) * 16 + lr) * g.N + n);
    }
  }
}

// Epilogue of tile t for token tiles mt0 .. mt0 + MTE - 1 from the complete
// sums in acc.  Accumulator layout: the lane holds rows 4 (lane / 16) + e of
// sub-tiles wave (and wave + 4), token (mt0 + mt) 16 + lane % 16.  Called by
// all 256 threads (it has barriers); rs_s holds the row scales by token.
template <int KIND, int MTE, int NS = 4>
__device__ __forceinline__ void epilogue(const GemmLaunch &g, int t, int mt0,
                                         const floatx4 (&acc)[SUBS<KIND>][MTE],
                                         const EpiOperands<KIND, MTE> &o, const float *rs_s,
                                         float (*red_s)[128][2]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, r4 = (lane >> 4) * 4;
  const int T = g.T, T_pad = g.MT * 16;
  if constexpr (KIND == GEMM_QKV) {
    const int gs = t * NS + wave;   // the wave's global sub-tile
    const int nh = g.nh, nkv = g.nkv;
    if (wave >= NS || gs >= (nh + 2 * nkv) * 8) return;  // no rows (no barriers below)
    const int hp = gs >> 3;         // head part: q heads, then k, then v
    const bool upper = lane >= 32;  // rows 8..15: the partner dims (+64)
    const int i0 = 8 * (gs & 7) + 4 * ((lane >> 4) & 1);
    const int d0 = i0 + (upper ? 64 : 0);  // this lane's dims d0 .. d0 + 3
#pragma unroll
    for (int mt = 0; mt < MTE; ++mt) {
      // padding tokens have a finite row scale too: the pair exchange below
      // runs on all lanes (lanes l and l + 32 hold the same token)
      const int tk = (mt0 + mt) * 16 + lr;
      const float rs = rs_s[tk];
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = acc[0][mt][e] * rs;
      if (hp < nh + nkv) {
        const float cs[8] = {o.rope[mt][0][0], o.rope[mt][0][1], o.rope[mt][0][2], o.rope[mt][0][3],
                             o.rope[mt][1][0], o.rope[mt][1][1], o.rope[mt][1][2], o.rope[mt][1][3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          // [0]: lane l % 32's value (dim i), [1]: lane l % 32 + 32's (dim i + 64)
          const auto pr = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[e]), __float_as_uint(v[e]),
                                                           false, false);
          const float a = __uint_as_float(pr[0]), b = __uint_as_float(pr[1]);
          const float c = cs[2 * e], sn = cs[2 * e + 1];
          v[e] = upper ? b * c + a * sn : a * c - b * sn;
        }
      }
      if (tk >= T) continue;
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
      if (hp < nh + nkv) {
        bf16_t *dst = hp < nh ? g.q + ((size_t)tk * nh + hp) * 128
                              : kc + ((size_t)(hp - nh) * cap + pos) * 128;
        *(u32x2 *)(dst + d0) = u32x2{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
      } else {
        bf16_t *vb = vc + (size_t)(hp - nh - nkv) * 128 * cap + pos;
#pragma unroll
        for (int e = 0; e < 4; ++e) vb[(size_t)(d0 + e) * cap] = f32_to_bf16(v[e]);
      }
    }
  } else if constexpr (KIND == GEMM_SWIGLU) {
    const int f0 = t * 16 * NS + wave * 16 + r4;
    if (wave >= NS || f0 >= g.N) return;  // no features (no barriers below)
#pragma unroll
    for (int mt = 0; mt < MTE; ++mt) {
      const int tk = (mt0 + mt) * 16 + lr;
      if (tk >= T) continue;
      const float rs = rs_s[tk];
      float a[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float gt = acc[0][mt][e] * rs, up = acc[1][mt][e] * rs;
        a[e] = gt / (1.f + expf(-gt)) * up;
      }
      *(u32x2 *)(g.act + (size_t)tk * g.N + f0) =
          u32x2{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3])};
    }
  } else if constexpr (KIND == GEMM_RESID) {
#pragma unroll
    for (int mt = 0; mt < MTE; ++mt) {
      const int tk = (mt0 + mt) * 16 + lr;
      float sq = 0.f;
      if (tk < T) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int n = t * BN + (wave + 4 * q) * 16 + r4;
          const uint2 gw = o.gain[q];
          const float g0 = bf16_to_f32(gw.x & 0xffff), g1 = bf16_to_f32(gw.x >> 16);
          const float g2 = bf16_to_f32(gw.y & 0xffff), g3 = bf16_to_f32(gw.y >> 16);
          floatx4 xv = o.x[q][mt];
          xv += acc[q][mt];
          *(floatx4 *)(g.x + (size_t)tk * g.N + n) = xv;
          *(u32x2 *)(g.xg + (size_t)tk * g.N + n) =
              u32x2{pack_bf16x2(xv[0] * g0, xv[1] * g1), pack_bf16x2(xv[2] * g2, xv[3] * g3)};
          sq += (xv[0] * xv[0] + xv[1] * xv[1]) + (xv[2] * xv[2] + xv[3] * xv[3]);
        }
      }
      // sum over the 4 lane groups (rows) of this wave
      sq += __shfl_xor(sq, 16, 64);
      sq += __shfl_xor(sq, 32, 64);
      if (lane < 16) red_s[wave][tk][0] = sq;
    }
    __syncthreads();
    if (tid < MTE * 16) {
      const int tk = mt0 * 16 + tid;
      const float v = tk < T ? ((red_s[0][tk][0] + red_s[1][tk][0]) + (red_s[2][tk][0] + red_s[3][tk][0]))
                             : 0.f;
      g.ss_out[(size_t)t * T_pad + tk] = v;
    }
  } else {  // GEMM_LOGITS
#pragma unroll
    for (int mt = 0; mt < MTE; ++mt) {
      const int tk = (mt0 + mt) * 16 + lr;
      const float rs = tk < T ? rs_s[tk] : 0.f;
      float bv = 0.f;
      int bi = -1;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const int n = t * BN + (wave + 4 * q) * 16 + r4;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = acc[q][mt][e] * rs;
        if (tk < T) {
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
      }
      // merge over the 4 lane groups: larger value, then smaller index
#pragma unroll
      for (int off = 16; off <= 32; off <<= 1) {
        const float v2 = __shfl_xor(bv, off, 64);
        const int i2 = __shfl_xor(bi, off, 64);
        amax_merge(bv, bi, v2, i2);
      }
      if (lane < 16) {
        red_s[wave][tk][0] = bv;
        red_s[wave][tk][1] = __int_as_float(bi);
      }
    }
    __syncthreads();
    if (tid < MTE * 16) {
      const int tk = mt0 * 16 + tid;
      float v = red_s[0][tk][0];
      int i = __float_as_int(red_s[0][tk][1]);
      for (int w = 1; w < 4; ++w) amax_merge(v, i, red_s[w][tk][0], __float_as_int(red_s[w][tk][1]));
      g.amax[(size_t)t * T_pad + tk] = make_float2(v, __int_as_float(i));
    }
  }
}

// partial sums of tile t by its contributor `slot`: [8 sub-tile pairs x MT][64
// lanes] floatx4, sub-tile pair index (wave 2 + q) MT + mt
__device__ __forceinline__ floatx4 *partial_of(const GemmLaunch &g, int t, int slot) {
  return (floatx4 *)g.part + ((size_t)t * g.maxc + slot) * (size_t)(8 * g.MT * 64);
}

// ---- the GEMM.  Workgroup w of G owns the units [u0, u1) (see
// PPD_GEMM_RING); SPLIT: store the partial of every tile segment, else every
// segment is a whole tile and is finished in place.
template <int MT, int KIND, bool SPLIT, int NS, int RING>
__global__ __launch_bounds__(256, 1) void gemm_bf16_kernel(GemmLaunch g) {
  static_assert(NS == 4 || (!SPLIT && (KIND == GEMM_QKV || KIND == GEMM_SWIGLU)),
                "3- and 2-group tiles: whole-tile QKV and gate/up only");
  static_assert(RING == R || (!SPLIT && RING % R == 0), "whole tiles only take a deeper ring");
  constexpr int T_pad = MT * 16;
  constexpr int NAP = (T_pad * 8 + 255) / 256;  // 16-byte activation pieces per thread per chunk
  __shared__ __attribute__((aligned(16))) unsigned char lds_a[2][T_pad * 128];
  __shared__ float rs_s[128];
  __shared__ float red_s[4][128][2];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15;  // MFMA row (weights) / column (tokens) within a 16-tile
  const int lg = lane >> 4;  // this lane's 16-byte k group within a 32-step
  // NS = 3: wave 3 owns no rows (it stages activations, skips the weights);
  // NS = 2: wave w multiplies k-step w / 2 of group w % 2
  const bool owns = NS != 3 || __builtin_amdgcn_readfirstlane(wave) < NS;
  const int kst = __builtin_amdgcn_readfirstlane(wave >> 1);  // NS = 2: this wave's k-step
  const int K = g.K, kc = g.kc_pad, G = g.G;
  const long Ng = (long)g.n_tiles * kc / RING;
  // this workgroup's units [u0, u1) (uniform: kept in scalar registers)
  const int u0 = __builtin_amdgcn_readfirstlane((int)gemm_group_lo(Ng, G, blockIdx.x) * RING);
  const int u1 = __builtin_amdgcn_readfirstlane((int)gemm_group_lo(Ng, G, blockIdx.x + 1) * RING);

  // norm row scales, requested before the weight stream starts
  constexpr bool kScale = !SPLIT && KIND != GEMM_RESID;
  [[maybe_unused]] float ssv[16];
  if constexpr (kScale) rs_request<T_pad>(g, 0, ssv);

  // ---- register rings.  Unit u's weight fragments for this wave: sub-tiles
  // wave (and wave + NS), k-steps 0 and 1.  Its activation pieces: 16-byte piece
  // e = tid + 256 i of the [T_pad][64] chunk (row e / 8, column e % 8).
  // Requests past the range read one 16-byte line (lane offsets masked to 0),
  // so every iteration issues the same loads.
  constexpr int S = SUBS<KIND>;
  const u32x4 *wp = (const u32x4 *)g.W;
  u32x4 wr[RING][2 * S], ar[RING][NAP];
  auto request_w = [&](int u, u32x4(&dw)[2 * S]) {
    if (!owns) return;
    const int live = u < u1 ? 63 : 0;
    const int uu = u < u1 ? u : u1 - 1;
    const u32x4 *wu = wp + (size_t)uu * UNIT<KIND, NS> + (lane & live);
    if constexpr (NS == 2) {
      // group wave % 2, k-step kst only (held in slot q * 2)
#pragma unroll
      for (int q = 0; q < S; ++q)
        dw[q * 2] = __builtin_nontemporal_load(wu + (((wave & 1) + 2 * q) * 2 + kst) * FRAG);
    } else {
#pragma unroll
      for (int q = 0; q < S; ++q)
#pragma unroll
        for (int s = 0; s < 2; ++s)
          dw[q * 2 + s] = __builtin_nontemporal_load(wu + ((wave + NS * q) * 2 + s) * FRAG);
    }
  };
  // per-lane element offsets of the activation pieces within a chunk;
  // pieces e >= T_pad * 8 (odd MT) load row 0 and are not staged
  int aoff[NAP];
#pragma unroll
  for (int i = 0; i < NAP; ++i) {
    int e = tid + 256 * i;
    if constexpr (T_pad * 8 % 256 != 0) e = e < T_pad * 8 ? e : 0;
    aoff[i] = (e >> 3) * K + (e & 7) * 8;
  }
  // u: unit to request; cu: its chunk within its tile
  auto request_a = [&](int u, int cu, u32x4(&da)[NAP]) {
    const int k0 = cu * KC;
    const bool kin = k0 < K;  // padding chunks read zeros
    const bf16_t *base = kin ? g.A + k0 : g.zeros;
    // past the range and in padding chunks every lane reads the base line.
    // The mask is opaque to the compiler, so that it issues the same loads
    // on every path instead of branching on it.
    int keep = __builtin_amdgcn_readfirstlane((u < u1 && kin) ? -1 : 0);
    asm volatile("" : "+s"(keep));
#pragma unroll
    for (int i = 0; i < NAP; ++i) da[i] = *(const u32x4 *)(base + (aoff[i] & keep));
  };
  auto stage = [&](const u32x4(&da)[NAP], int slot) {
#pragma unroll
    for (int i = 0; i < NAP; ++i) {
      const int e = tid + 256 * i;
      if (T_pad * 8 % 256 == 0 || e < T_pad * 8) {
        const int r = e >> 3, c = e & 7;
        *(u32x4 *)(&lds_a[slot][r * 128 + swz(r, c) * 16]) = da[i];
      }
    }
  };

  floatx4 acc[S][MT];
  int tile = u0 / kc;
  [[maybe_unused]] EpiOperands<KIND, MT> eo;
  if constexpr (!SPLIT) epi_request<KIND, MT, NS>(g, tile, 0, eo);
  const int c0 = u0 - tile * kc;  // first unit's chunk (a multiple of RING)
#pragma unroll
  for (int j = 0; j < RING; ++j) {
    request_w(u0 + j, wr[j]);
    request_a(u0 + j, c0 + j, ar[j]);
  }
  __builtin_amdgcn_sched_barrier(0);
  if constexpr (kScale) rs_finish<T_pad>(g, 0, ssv, &red_s[0][0][0], rs_s);
  // rs_s is read by epilogues after the main loop's barriers; red_s is next
  // written by an epilogue, after them as well

  // ---- main loop over segments (the units of one tile within [u0, u1)),
  // RING units per trip.  Unit u: stage its activations (requested RING units ago)
  // into LDS slot (u - u0) & 1 and request unit u + RING's into the freed
  // registers; barrier; multiply with the weight fragments requested RING units
  // ago, then request unit u + RING's weights into them.  The slot staged here
  // was last read for unit u - 2, which every wave finished before unit
  // u - 1's barrier.  The accumulators are zeroed per segment, so the inner
  // loop carries them unchanged.
  int gc = c0;  // chunk of unit gu within its tile
  for (int gu = u0; gu < u1;) {
    const int ue = min(u1, (tile + 1) * kc);
#pragma unroll
    for (int q = 0; q < S; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[q][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
    for (; gu < ue; gu += RING) {
      // chunk of unit gu + RING + j: gc + RING + j, wrapped into the next tile
      const int nc = gc + RING < kc ? gc + RING : gc + RING - kc;
#pragma unroll
      for (int j = 0; j < RING; ++j) {
        const int u = gu + j;
        const int slot = (u - u0) & 1;
        stage(ar[j], slot);
        __builtin_amdgcn_sched_barrier(0);
        request_a(u + RING, nc + j, ar[j]);
        __builtin_amdgcn_sched_barrier(0);
        __syncthreads();
        const unsigned char *al = lds_a[slot];
        if constexpr (NS == 2) {
          u32x4 af[MT];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int r = mt * 16 + lr;
            af[mt] = *(const u32x4 *)(al + r * 128 + swz(r, kst * 4 + lg) * 16);
          }
#pragma unroll
          for (int q = 0; q < S; ++q)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[q][mt] = mfma16x16x32(as_bf16x8(wr[j][q * 2]), as_bf16x8(af[mt]), acc[q][mt]);
        }
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          if (NS == 2 || !owns) break;
          u32x4 af[MT];
#pragma unroll
          for (int mt = 0; mt < MT; ++mt) {
            const int r = mt * 16 + lr;
            af[mt] = *(const u32x4 *)(al + r * 128 + swz(r, s * 4 + lg) * 16);
          }
#pragma unroll
          for (int q = 0; q < S; ++q)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
              acc[q][mt] = mfma16x16x32(as_bf16x8(wr[j][q * 2 + s]), as_bf16x8(af[mt]), acc[q][mt]);
        }
        __builtin_amdgcn_sched_barrier(0);
        request_w(u + RING, wr[j]);
        __builtin_amdgcn_sched_barrier(0);
      }
      gc = nc;
    }
    if constexpr (SPLIT) {
      // this segment's partial, in slot (this workgroup - the tile's first
      // contributor); plain stores: the finish kernel runs after this grid
      const int first = gemm_group_owner(Ng, G, (long)tile * kc / RING);
      floatx4 *dst = partial_of(g, tile, blockIdx.x - first);
#pragma unroll
      for (int q = 0; q < S; ++q)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) dst[((wave * S + q) * MT + mt) * 64 + lane] = acc[q][mt];
      ++tile;
    } else {
      if constexpr (NS == 2) {
        // wave w + 2 adds its k-step's sums into wave w's through the
        // activation slots (2 S MT KB <= their 4 MT KB), once every wave is
        // done reading them
        floatx4 *red = (floatx4 *)&lds_a[0][0];
        __syncthreads();
        if (wave >= 2) {
#pragma unroll
          for (int q = 0; q < S; ++q)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) red[(((wave - 2) * S + q) * MT + mt) * 64 + lane] = acc[q][mt];
        }
        __syncthreads();
        if (wave < 2) {
#pragma unroll
          for (int q = 0; q < S; ++q)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) acc[q][mt] += red[((wave * S + q) * MT + mt) * 64 + lane];
        }
      }
      epilogue<KIND, MT, NS>(g, tile, 0, acc, eo, rs_s, red_s);
      if (ue < u1) {
        __syncthreads();  // red_s is written again by the next tile's epilogue
        epi_request<KIND, MT, NS>(g, ++tile, 0, eo);
      }
    }
  }
}

// ---- finish of a split GEMM: workgroup (tile, 16-token block mt) adds the
// tile's partials in contributor (workgroup) order and runs the epilogue for
// the block's tokens.  The waves and lanes keep the GEMM's accumulator layout.
template <int KIND>
__global__ __launch_bounds__(256) void gemm_finish_kernel(GemmLaunch g) {
  __shared__ float rs_s[128];
  __shared__ float red_s[4][128][2];
  const int t = blockIdx.x, mt = blockIdx.y;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long Ng = (long)g.n_tiles * g.kc_pad / R;
  const int first = gemm_group_owner(Ng, g.G, (long)t * g.kc_pad / R);
  const int n_c = gemm_group_owner(Ng, g.G, (long)(t + 1) * g.kc_pad / R - 1) - first + 1;

  [[maybe_unused]] float ssv[16];
  if constexpr (KIND != GEMM_RESID) rs_request<16>(g, mt * 16, ssv);
  EpiOperands<KIND, 1> eo;
  epi_request<KIND, 1>(g, t, mt, eo);

  // U contributors' partials are requested together (one round trip), then
  // added in order
  constexpr int U = 8, S = SUBS<KIND>;
  floatx4 acc[S][1];
#pragma unroll
  for (int q = 0; q < S; ++q) acc[q][0] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < n_c; c0 += U) {
    floatx4 buf[U][S];
#pragma unroll
    for (int v = 0; v < U; ++v) {
      const floatx4 *src = partial_of(g, t, min(c0 + v, n_c - 1));
#pragma unroll
      for (int q = 0; q < S; ++q) buf[v][q] = src[((wave * S + q) * g.MT + mt) * 64 + lane];
    }
#pragma unroll
    for (int v = 0; v < U; ++v)
      if (c0 + v < n_c) {
#pragma unroll
        for (int q = 0; q < S; ++q) acc[q][0] += buf[v][q];
      }
  }
  if constexpr (KIND != GEMM_RESID) rs_finish<16>(g, mt * 16, ssv, &red_s[0][0][0], rs_s);
  __syncthreads();  // red_s (used by rs_finish) is reused by the epilogue
  epilogue<KIND, 1>(g, t, mt, acc, eo, rs_s, red_s);
}

template <int KIND>
hipError_t launch_kind(const GemmLaunch &g, hipStream_t s) {
  const dim3 grid(g.G), block(256);
  hipEvent_t ev0 = (hipEvent_t)g.ev_start, ev1 = (hipEvent_t)g.ev_stop;
  // timed: from the GEMM dispatch's start to the last dispatch's end
  hipEvent_t gemm_stop = g.split ? nullptr : ev1;
  constexpr bool kNs3 = KIND == GEMM_QKV || KIND == GEMM_SWIGLU;
  if (g.ns != 4 && !(kNs3 && (g.ns == 3 || g.ns == 2) && !g.split && g.kc_pad % kRing3 == 0))
    return hipErrorInvalidValue;
  switch (g.MT) {
#define PPD_LAUNCH(M, SP, NS, RG)                                                            \
  if (ev0)                                                                                   \
    hipExtLaunchKernelGGL((gemm_bf16_kernel<M, KIND, SP, NS, RG>), grid, block, 0, s, ev0,   \
                          gemm_stop, 0, g);                                                  \
  else                                                                                       \
    hipLaunchKernelGGL((gemm_bf16_kernel<M, KIND, SP, NS, RG>), grid, block, 0, s, g);
#define PPD_CASE(M)                                                                          \
  case M:                                                                                    \
    if (g.split) {                                                                           \
      PPD_LAUNCH(M, true, 4, R)                                                              \
    } else if (g.ns == 3) {                                                                  \
      if constexpr (kNs3) { PPD_LAUNCH(M, false, (kNs3 ? 3 : 4), kRing3) }                   \
    } else if (g.ns == 2) {                                                                  \
      if constexpr (kNs3) { PPD_LAUNCH(M, false, (kNs3 ? 2 : 4), kRing3) }                   \
    } else {                                                                                 \
      PPD_LAUNCH(M, false, 4, R)                                                             \
    }                                                                                        \
    break;
    PPD_CASE(1) PPD_CASE(2) PPD_CASE(3) PPD_CASE(4) PPD_CASE(5) PPD_CASE(6) PPD_CASE(7) PPD_CASE(8)
#undef PPD_CASE
#undef PPD_LAUNCH
    default: return hipErrorInvalidValue;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !g.split) return e;
  const dim3 fgrid(g.n_tiles, g.MT);
  if (ev1)
    hipExtLaunchKernelGGL(gemm_finish_kernel<KIND>, fgrid, block, 0, s, nullptr, ev1, 0, g);
  else
    hipLaunchKernelGGL(gemm_finish_kernel<KIND>, fgrid, block, 0, s, g);
  return hipGetLastError();
}

// ---- weight packing.  Packed 16-byte item (tile, chunk, sub-tile q < 4 SUBS,
// k-step s < 2, lane l < 64) holds the 8 bf16 of weight row
// tile_row(tile, 16 q + l % 16) at columns 64 chunk + 32 s + 8 (l / 16) ..
// + 7; rows and columns past the matrix (padding) are zero.
template <int KIND, int NS>
__global__ __launch_bounds__(256) void pack_kernel(const bf16_t *__restrict__ src, u32x4 *__restrict__ dst,
                                                   int N, int K, int rows_total, int kc_pad, long n_items) {
  for (long i = blockIdx.x * (long)blockDim.x + threadIdx.x; i < n_items;
       i += (long)gridDim.x * blockDim.x) {
    constexpr int NQ = NS * SUBS<KIND>;  // sub-tiles per tile
    const int l = (int)(i & 63);
    const long f = i >> 6;  // fragment ((tile kc_pad + chunk) NQ + q) 2 + s
    const int s = (int)(f & 1), q = (int)((f >> 1) % NQ);
    const long tc = f / (2 * NQ);
    const int chunk = (int)(tc % kc_pad), tile = (int)(tc / kc_pad);
    const int row = tile_row<KIND, NS>(tile, 16 * q + (l & 15), N);
    const int col = chunk * KC + 32 * s + 8 * (l >> 4);
    u32x4 v = u32x4{0u, 0u, 0u, 0u};
    if (row < rows_total && col < K) v = *(const u32x4 *)(src + (size_t)row * K + col);
    dst[i] = v;
  }
}

template <int KIND, int NS>
hipError_t launch_pack_kind(int N, int K, const bf16_t *src, bf16_t *dst, hipStream_t s) {
  const int n_tiles = gemm_tiles_of(KIND, N, NS), kc_pad = gemm_kc_pad_of(K);
  const long n_items = (long)n_tiles * kc_pad * UNIT<KIND, NS>;
  const int rows_total = KIND == GEMM_SWIGLU ? 2 * N : N;
  const dim3 grid((unsigned)std::min<long>(8192, (n_items + 255) / 256)), block(256);
  hipLaunchKernelGGL((pack_kernel<KIND, NS>), grid, block, 0, s, src, (u32x4 *)dst, N, K, rows_total,
                     kc_pad, n_items);
  return hipGetLastError();
}

}  // namespace

int gemm_tiles_of(int kind, int N, int ns) {
  // QKV: N / 16 sub-tiles; gate/up: N / 16 blocks of 16 features
  return kind == GEMM_SWIGLU || kind == GEMM_QKV ? (N / 16 + ns - 1) / ns : (N + BN - 1) / BN;
}

int gemm_tile_rows_of(int kind, int ns) {
  return kind == GEMM_QKV ? 16 * ns : kind == GEMM_SWIGLU ? 32 * ns : BN;
}

int gemm_kc_pad_of(int K) { return ((K / KC + R - 1) / R) * R; }

hipError_t launch_pack_weight(int kind, int N, int K, int ns, const bf16_t *src, bf16_t *dst,
                              hipStream_t s) {
  if (ns == 3) {
    if (kind == GEMM_QKV) return launch_pack_kind<GEMM_QKV, 3>(N, K, src, dst, s);
    if (kind == GEMM_SWIGLU) return launch_pack_kind<GEMM_SWIGLU, 3>(N, K, src, dst, s);
    return hipErrorInvalidValue;
  }
  if (ns == 2) {
    if (kind == GEMM_QKV) return launch_pack_kind<GEMM_QKV, 2>(N, K, src, dst, s);
    if (kind == GEMM_SWIGLU) return launch_pack_kind<GEMM_SWIGLU, 2>(N, K, src, dst, s);
    return hipErrorInvalidValue;
  }
  if (ns != 4) return hipErrorInvalidValue;
  switch (kind) {
    case GEMM_QKV: return launch_pack_kind<GEMM_QKV, 4>(N, K, src, dst, s);
    case GEMM_RESID: return launch_pack_kind<GEMM_RESID, 4>(N, K, src, dst, s);
    case GEMM_SWIGLU: return launch_pack_kind<GEMM_SWIGLU, 4>(N, K, src, dst, s);
    case GEMM_LOGITS: return launch_pack_kind<GEMM_LOGITS, 4>(N, K, src, dst, s);
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
