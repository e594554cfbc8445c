// Skinny-M bfloat16 GEMMs of the verification forward pass, with fused
// epilogues.  out[row][t] = sum_k W[row][k] * A[t][k] for the T <= 128 tree
// tokens t, fp32 accumulation on the gfx950 matrix cores
// (v_mfma_f32_16x16x32_bf16: weights are the 16-row A operand, tokens the
// 16-column B operand).
//
// The step is bound by streaming the weights from HBM once (arithmetic
// intensity ~T flop/byte, far below the MI355X ridge), so the kernel is built
// around the weight stream:
//  * a workgroup owns a 64-row tile of W and one slice of K (split-K across
//    workgroups when N alone gives too few tiles); its 4 waves split the
//    slice's K range, so every weight and activation byte is loaded by
//    exactly one lane, straight from global memory into MFMA operand
//    registers (16 bytes per lane, no LDS staging);
//  * loads are double-buffered in registers, weights with a non-temporal hint
//    (streamed once), activations through L2 (shared by every workgroup);
//  * the 4 waves' partial tiles are summed in LDS in a fixed order; split-K
//    partials go to the workspace and the last workgroup of a tile (atomic
//    ticket) adds them in split order, so results never depend on timing;
//  * the epilogue is fused: RMSNorm row scale, RoPE + query/key/value stores
//    into the cache (QKV), residual add + next norm operand + sum of squares
//    (O / down projection), SwiGLU (gate/up), logits + argmax partials (LM
//    head).
#include "ppd_internal.h"

namespace {

constexpr int BN = PPD_GEMM_BN;  // 64 rows = 4 sub-tiles of 16
constexpr int U = 2;             // k-steps (32 each) per pipeline stage

__device__ __forceinline__ u32x4 ldg_nt(const bf16_t *p) {
  return __builtin_nontemporal_load((const u32x4 *)p);
}
__device__ __forceinline__ u32x4 ldg(const bf16_t *p) { return *(const u32x4 *)p; }

// first W row of sub-tile j (0..3) of `tile`
template <int KIND>
__device__ __forceinline__ int subtile_row(int tile, int j, int F) {
  if constexpr (KIND == GEMM_QKV) {
    // tile = (head part hp, half hh): sub-tiles 0,1 hold dims 32hh..32hh+31,
    // sub-tiles 2,3 the RoPE partners 64 + 32hh ..
    return (tile >> 1) * 128 + (tile & 1) * 32 + (j & 1) * 16 + (j >> 1) * 64;
  } else if constexpr (KIND == GEMM_SWIGLU) {
    // features 32 tile .. 32 tile + 31: sub-tiles 0,1 gate rows, 2,3 up rows
    return (j >> 1) * F + tile * 32 + (j & 1) * 16;
  } else {
    return tile * BN + j * 16;
  }
}

template <int MT, int KIND>
__global__ __launch_bounds__(256, (MT <= 4 ? 2 : 1)) void gemm_bf16_kernel(GemmLaunch g) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int split = blockIdx.x % g.sk;
  const int tile = blockIdx.x / g.sk;
  const int K = g.K;
  const int rows_total = (KIND == GEMM_SWIGLU) ? 2 * g.N : (KIND == GEMM_QKV ? g.N : g.N);
  const int lr = lane & 15;         // row within sub-tile (A operand) / token within tile (B)
  const int kg = (lane >> 4) * 8;   // this lane's 8-element k group within a 32-step

  // k-steps of this split, then of this wave
  const int nks = K >> 5;
  const int s0 = (int)((long)nks * split / g.sk), s1 = (int)((long)nks * (split + 1) / g.sk);
  const int w0 = s0 + (s1 - s0) * wave / 4, w1 = s0 + (s1 - s0) * (wave + 1) / 4;

  const bf16_t *wrow[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int r = subtile_row<KIND>(tile, j, g.N) + lr;
    r = r < rows_total ? r : rows_total - 1;
    wrow[j] = g.W + (size_t)r * K + kg;
  }
  const bf16_t *arow[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) arow[mt] = g.A + (size_t)(mt * 16 + lr) * K + kg;

  floatx4 acc[4][MT];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[j][mt] = floatx4{0.f, 0.f, 0.f, 0.f};

  u32x4 wb0[U][4], ab0[U][MT], wb1[U][4], ab1[U][MT];
  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};

#define PPD_LOAD(WB, AB, KS)                                              \
  _Pragma("unroll") for (int u = 0; u < U; ++u) {                         \
    const int ks_ = (KS) + u;                                             \
    if (ks_ < w1) {                                                       \
      _Pragma("unroll") for (int j = 0; j < 4; ++j) WB[u][j] = ldg_nt(wrow[j] + ks_ * 32); \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) AB[u][mt] = ldg(arow[mt] + ks_ * 32); \
    } else {                                                              \
      _Pragma("unroll") for (int j = 0; j < 4; ++j) WB[u][j] = zero;      \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt) AB[u][mt] = zero; \
    }                                                                     \
  }
#define PPD_COMPUTE(WB, AB)                                               \
  _Pragma("unroll") for (int u = 0; u < U; ++u)                           \
    _Pragma("unroll") for (int j = 0; j < 4; ++j)                         \
      _Pragma("unroll") for (int mt = 0; mt < MT; ++mt)                   \
        acc[j][mt] = mfma16x16x32(as_bf16x8(WB[u][j]), as_bf16x8(AB[u][mt]), acc[j][mt]);

  PPD_LOAD(wb0, ab0, w0);
  for (int ks = w0; ks < w1; ks += 2 * U) {
    PPD_LOAD(wb1, ab1, ks + U);
    PPD_COMPUTE(wb0, ab0);
    PPD_LOAD(wb0, ab0, ks + 2 * U);
    PPD_COMPUTE(wb1, ab1);
  }
#undef PPD_LOAD
#undef PPD_COMPUTE

  // ---- sum the 4 waves' partial tiles (fixed order); waves 0 and 1 keep
  // sub-tiles (w, w + 2) -- the RoPE / SwiGLU partner pairs.
  __shared__ floatx4 red[4][4][64];
  __shared__ float rs_s[128];
  __shared__ float pair_s[2][128][2];
  __shared__ int last_s;
  floatx4 res[2][MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
    for (int j = 0; j < 4; ++j) red[wave][j][lane] = acc[j][mt];
    __syncthreads();
    if (wave < 2) {
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int j = wave + 2 * p;
        res[p][mt] = ((red[0][j][lane] + red[1][j][lane]) + red[2][j][lane]) + red[3][j][lane];
      }
    }
    __syncthreads();
  }

  // ---- split-K: publish the partial tile; the last workgroup sums all
  if (g.sk > 1) {
    const size_t tile_floats = (size_t)4 * MT * 64 * 4;
    if (wave < 2) {
      floatx4 *dst = (floatx4 *)(g.part + (size_t)blockIdx.x * tile_floats);
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) dst[((wave * 2 + p) * MT + mt) * 64 + lane] = res[p][mt];
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned prev = atomicAdd(&g.counters[tile], 1u);
      int last = prev == (unsigned)(g.sk - 1);
      if (last) g.counters[tile] = 0u;
      last_s = last;
    }
    __syncthreads();
    if (!last_s) return;
    __threadfence();
    if (wave < 2) {
#pragma unroll
      for (int p = 0; p < 2; ++p)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) res[p][mt] = floatx4{0.f, 0.f, 0.f, 0.f};
      for (int s = 0; s < g.sk; ++s) {
        const floatx4 *src = (const floatx4 *)(g.part + (size_t)(tile * g.sk + s) * tile_floats);
#pragma unroll
        for (int p = 0; p < 2; ++p)
#pragma unroll
          for (int mt = 0; mt < MT; ++mt)
            res[p][mt] += src[((wave * 2 + p) * MT + mt) * 64 + lane];
      }
    }
  }

  // ---- RMSNorm row scale r[t] = 1/sqrt(mean(x^2) + eps) from the
  // producer's sum-of-squares partials (summed in partial order)
  if constexpr (KIND != GEMM_RESID) {
    if (threadIdx.x < MT * 16) {
      const int t = threadIdx.x;
      const int T_pad = MT * 16;
      float s = 0.f;
      for (int p = 0; p < g.n_ss; ++p) s += g.ss[(size_t)p * T_pad + t];
      rs_s[t] = rsqrtf(s * g.inv_h + g.eps);
    }
    __syncthreads();
  }
  if (wave >= 2) {
    if constexpr (KIND == GEMM_RESID || KIND == GEMM_LOGITS) {
      __syncthreads();  // matches the pair exchange below
    }
    return;
  }

  const int r4 = (lane >> 4) * 4;  // first of this lane's 4 rows within a sub-tile
  const int T = g.T;
  const int T_pad = MT * 16;

  if constexpr (KIND == GEMM_QKV) {
    const int hp = tile >> 1;
    const int i0 = (tile & 1) * 32 + wave * 16 + r4;  // dims i0..i0+3 and +64
    const int nh = g.nh, nkv = g.nkv;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      if (t >= T) continue;
      const float rs = rs_s[t];
      float lo[4], hi[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = res[0][mt][e] * rs;
        hi[e] = res[1][mt][e] * rs;
      }
      if (hp < nh + nkv) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float2 cs = g.rope[(size_t)t * 64 + i0 + e];
          const float a = lo[e], b = hi[e];
          lo[e] = a * cs.x - b * cs.y;
          hi[e] = b * cs.x + a * cs.y;
        }
        u32x2 plo = u32x2{pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3])};
        u32x2 phi = u32x2{pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3])};
        bf16_t *dst;
        if (hp < nh) {
          dst = g.q + ((size_t)t * nh + hp) * 128;
        } else {
          dst = g.kc + ((size_t)(hp - nh) * g.cap + g.L + t) * 128;
        }
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
    const int f0 = tile * 32 + wave * 16 + r4;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      if (t >= T) continue;
      const float rs = rs_s[t];
      float a[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float gt = res[0][mt][e] * rs, up = res[1][mt][e] * rs;
        a[e] = gt / (1.f + expf(-gt)) * up;
      }
      *(u32x2 *)(g.act + (size_t)t * g.N + f0) =
          u32x2{pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3])};
    }
  } else if constexpr (KIND == GEMM_RESID) {
    float sq[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      sq[mt] = 0.f;
      if (t >= T) continue;
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int n = tile * BN + (wave + 2 * p) * 16 + r4;
        float *xp = g.x + (size_t)t * g.N + n;
        floatx4 xv = *(floatx4 *)xp;
        xv += res[p][mt];
        *(floatx4 *)xp = xv;
        const uint2 gw = *(const uint2 *)(g.gain + n);
        const float g0 = bf16_to_f32(gw.x & 0xffff), g1 = bf16_to_f32(gw.x >> 16);
        const float g2 = bf16_to_f32(gw.y & 0xffff), g3 = bf16_to_f32(gw.y >> 16);
        *(u32x2 *)(g.xg + (size_t)t * g.N + n) =
            u32x2{pack_bf16x2(xv[0] * g0, xv[1] * g1), pack_bf16x2(xv[2] * g2, xv[3] * g3)};
        sq[mt] += (xv[0] * xv[0] + xv[1] * xv[1]) + (xv[2] * xv[2] + xv[3] * xv[3]);
      }
    }
    // reduce over the 4 lane groups (rows), then over the two waves
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v = sq[mt];
      v += __shfl_xor(v, 16, 64);
      v += __shfl_xor(v, 32, 64);
      if (lane < 16) pair_s[wave][mt * 16 + lane][0] = v;
    }
    __syncthreads();
    if (wave == 0) {
      for (int t = lane; t < T_pad; t += 64) {
        const float v = t < T ? pair_s[0][t][0] + pair_s[1][t][0] : 0.f;
        g.ss_out[(size_t)tile * T_pad + t] = v;
      }
    }
  } else {  // GEMM_LOGITS
    float bv[MT];
    int bi[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const int t = mt * 16 + lr;
      bv[mt] = 0.f;
      bi[mt] = -1;
      const float rs = t < T ? rs_s[t] : 0.f;
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        const int n = tile * BN + (wave + 2 * p) * 16 + r4;
        float v[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = res[p][mt][e] * rs;
          if (t < T && n + e < g.N && v[e] != v[e]) atomicOr(g.status, PPD_DEV_NAN_LOGIT);
        }
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
            if (n + e < g.N && v[e] == v[e] && (bi[mt] < 0 || v[e] > bv[mt])) {
              bv[mt] = v[e];
              bi[mt] = n + e;
            }
          }
        }
      }
    }
    // merge across lane groups, then the two waves: larger value, smaller index
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      float v = bv[mt];
      int i = bi[mt];
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float v2 = __shfl_xor(v, o, 64);
        const int i2 = __shfl_xor(i, o, 64);
        if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
          v = v2;
          i = i2;
        }
      }
      if (lane < 16) {
        pair_s[wave][mt * 16 + lane][0] = v;
        pair_s[wave][mt * 16 + lane][1] = __int_as_float(i);
      }
    }
    __syncthreads();
    if (wave == 0) {
      for (int t = lane; t < T_pad; t += 64) {
        float v = pair_s[0][t][0];
        int i = __float_as_int(pair_s[0][t][1]);
        const float v2 = pair_s[1][t][0];
        const int i2 = __float_as_int(pair_s[1][t][1]);
        if (i2 >= 0 && (i < 0 || v2 > v || (v2 == v && i2 < i))) {
          v = v2;
          i = i2;
        }
        g.amax[(size_t)tile * T_pad + t] = make_float2(v, __int_as_float(i));
      }
    }
  }
}

template <int KIND>
hipError_t launch_kind(const GemmLaunch &g, int n_tiles, hipStream_t s) {
  dim3 grid(n_tiles * g.sk), block(256);
  switch (g.MT) {
#define PPD_CASE(M) \
  case M: hipLaunchKernelGGL((gemm_bf16_kernel<M, KIND>), grid, block, 0, s, g); break;
    PPD_CASE(1) PPD_CASE(2) PPD_CASE(3) PPD_CASE(4) PPD_CASE(5) PPD_CASE(6) PPD_CASE(7) PPD_CASE(8)
#undef PPD_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_bf16(const GemmLaunch &g, int n_tiles, hipStream_t s) {
  switch (g.kind) {
    case GEMM_QKV: return launch_kind<GEMM_QKV>(g, n_tiles, s);
    case GEMM_RESID: return launch_kind<GEMM_RESID>(g, n_tiles, s);
    case GEMM_SWIGLU: return launch_kind<GEMM_SWIGLU>(g, n_tiles, s);
    case GEMM_LOGITS: return launch_kind<GEMM_LOGITS>(g, n_tiles, s);
  }
  return hipErrorInvalidValue;
}
