// Candidate generation for the next step (Section 3, step (1): candidates are
// the model's predictions at the prompt tokens; Section 3.1: the prompt token
// at token distance j stands at the position of the j-th token after the last
// accepted one; Section 4 and the tree-construction appendix: the tree is a
// sparse tree of top-k candidates with prompt tokens appended).
//
// The next tree is a fixed template whose ids are filled on the device from
// this step's outputs, so the decode loop needs no host round trip: the root
// is the bonus token, a candidate at depth d with rank r takes the r-th best
// token of the logits of the accepted node's d-th prompt token (past the end
// of that chain: its deepest node, or the accepted node itself), and prompt
// nodes carry fixed prompt ids.  Ranks order larger logits first, equal ones
// by smaller index, NaN last.
//
// One workgroup of 1024 threads per candidate depth.  It walks the accepted
// node's prompt chain, then selects the top kd of one logits row:
//   1. every thread holds 32 strided elements of the row in registers (all
//      loads in flight at once) and takes its best one;
//   2. the kd-th best of the 16 wave maxima (kd <= 16) is reached by at
//      least kd elements, so every element of the top kd reaches it;
//   3. the elements that reach it (only threads whose best does) go to a
//      list in LDS, and each is ranked by counting the list entries that
//      beat it.
// Comparisons use one 64-bit key per element that orders (value, index) as
// the ranks do, so selection is integer max / compare without branches.
// If the list would overflow, kd rounds of a workgroup-wide maximum over the
// elements below the previous pick select the ranks instead.
#include <type_traits>

#include "ppd_internal.h"

namespace {

constexpr int kThreads = 1024;
constexpr int kPer = 32;                    // row elements per thread per chunk
constexpr int kChunk = kThreads * kPer;     // row elements per chunk
constexpr int kListCap = 2048;              // candidate list capacity

// Rank key of (value, index): a larger key ranks first.  The high word maps
// the float monotonically onto unsigned order (-0 as +0, every NaN to 0,
// below all numbers), the low word is ~index, so equal values rank the
// smaller index first.  Key 0 is "no element": every element's low word
// is at least 2^31.
__device__ __forceinline__ uint32_t value_word(float v) {
  uint32_t b = __float_as_uint(v);
  const uint32_t mag = b & 0x7fffffffu;
  b = mag == 0 ? 0u : b;
  const uint32_t k = b ^ ((uint32_t)((int32_t)b >> 31) | 0x80000000u);
  return mag > 0x7f800000u ? 0u : k;
}
__device__ __forceinline__ uint64_t make_key(uint32_t hi, int idx) {
  return ((uint64_t)hi << 32) | (uint32_t)~idx;
}
__device__ __forceinline__ int key_index(uint64_t key) { return (int)~(uint32_t)key; }
__device__ __forceinline__ bool key_is_nan(uint64_t key) { return (uint32_t)(key >> 32) == 0; }

__device__ __forceinline__ uint64_t lane_key(uint64_t k, int j) {
  const uint32_t lo = __builtin_amdgcn_readlane((uint32_t)k, j);
  const uint32_t hi = __builtin_amdgcn_readlane((uint32_t)(k >> 32), j);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }

template <int CTRL>
__device__ __forceinline__ uint64_t dpp_key(uint64_t k) {
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)k, CTRL, 0xf, 0xf, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(k >> 32), CTRL, 0xf, 0xf, false);
  return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

// maximum key over the wave, in every lane: lane pairs within quads (DPP
// quad permutations), 8-lane halves (half-row mirror), 16-lane rows (row
// mirror), row pairs and wave halves (permlane swaps)
__device__ __forceinline__ uint64_t wave_max_key(uint64_t k) {
  k = umax64(k, dpp_key<0xb1>(k));   // quad_perm [1,0,3,2]
  k = umax64(k, dpp_key<0x4e>(k));   // quad_perm [2,3,0,1]
  k = umax64(k, dpp_key<0x141>(k));  // row_half_mirror
  k = umax64(k, dpp_key<0x140>(k));  // row_mirror
  uint32_t lo = (uint32_t)k, hi = (uint32_t)(k >> 32);
  auto l16 = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
  auto h16 = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
  k = umax64(((uint64_t)h16[0] << 32) | l16[0], ((uint64_t)h16[1] << 32) | l16[1]);
  lo = (uint32_t)k;
  hi = (uint32_t)(k >> 32);
  auto l32 = __builtin_amdgcn_permlane32_swap(lo, lo, false, false);
  auto h32 = __builtin_amdgcn_permlane32_swap(hi, hi, false, false);
  return umax64(((uint64_t)h32[0] << 32) | l32[0], ((uint64_t)h32[1] << 32) | l32[1]);
}

// MULTI: the row spans several register chunks (reloaded in each pass);
// VEC: rows are 16-byte aligned, read in float4 (a thread's elements are
// then runs of 4); EPT: several EPT groups, whose rows are averaged
template <bool MULTI, bool VEC, bool EPT>
__global__ __launch_bounds__(kThreads) void next_tree_kernel(NextTreeLaunch p) {
  // per EPT group: the chain node reached so far (-2 - node once the chain
  // has ended at that node), the next level's node, the logits row used
  __shared__ int cur_s[PPD_EPT_MAX], find_s[PPD_EPT_MAX], src_s[PPD_EPT_MAX];
  __shared__ int acc_s, count_s, nan_s;
  __shared__ uint64_t wave_s[kThreads / 64];
  __shared__ uint64_t list_s[kListCap];
  __shared__ int top_s[PPD_TOPK_MAX];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = blockIdx.x + 1;  // candidate depth handled here
  const int kd = p.k_of_depth[d];
  const int V = p.vocab;
  const int G = EPT ? p.n_ept : 1;

  // this step's tree and accepted path, one node per thread
  int my_par = INT_MIN, my_id = -1, my_path = 0;
  if (tid < p.T) {
    my_par = p.parent[tid];
    my_id = p.ids[tid];
    my_path = p.path[tid];
  }

  // ---- root and prompt nodes (workgroup 0)
  if (blockIdx.x == 0) {
    for (int i = tid; i < p.tpl_T; i += kThreads) {
      const int kind = p.tpl_kind[i];
      if (i == 0)
        p.next_ids[0] = *p.next_tok;
      else if (kind < 0)
        p.next_ids[i] = V + (-kind - 1);
    }
  }
  if (kd == 0) return;  // no candidate at this depth

  // ---- the accepted node and its prompt chains (one per EPT group), up to
  // depth d; a chain stops at its first missing level
  if (tid == 0) {
    acc_s = min(max(*p.n_path, 1), p.T) - 1;  // the accepted node's place on the path
    nan_s = 0;
    count_s = 0;
  }
  __syncthreads();
  if (tid == acc_s)
    for (int g = 0; g < G; ++g) cur_s[g] = min(max(my_path, 0), p.T - 1);
  for (int j = 0; j < d; ++j) {
    if (tid < G) find_s[tid] = INT_MAX;
    __syncthreads();
    const int g = my_id - V - j * G;  // my node's group if it is a level-j EPT
    if (g >= 0 && g < G && my_par == cur_s[g]) atomicMin(&find_s[g], tid);
    __syncthreads();
    bool any = false;
    for (int q = 0; q < G; ++q) any |= find_s[q] != INT_MAX;
    if (!any) break;  // uniform: every chain ends here
    if (tid < G) {
      const int c = cur_s[tid];
      if (c >= 0) cur_s[tid] = find_s[tid] != INT_MAX ? find_s[tid] : -2 - c;
    }
    __syncthreads();  // find_s is reset next
  }
  __syncthreads();
  if (tid < G) {
    const int c = cur_s[tid];
    src_s[tid] = c >= 0 ? c : -2 - c;
  }
  __syncthreads();

  // ---- 1. the row in registers (as value words), each thread's best; with
  // EPT groups the row is their mean: added in group order, then divided
  const int n_chunks = MULTI ? (V + kChunk - 1) / kChunk : 1;
  // row index of this thread's element e of chunk c (grows with e)
  auto eidx = [&](int c, int e) {
    return VEC ? c * kChunk + 4 * ((e >> 2) * kThreads + tid) + (e & 3)
               : c * kChunk + e * kThreads + tid;
  };
  // elements [E0, E0 + N) of this thread's chunk c of a row into x
  auto load_part = [&](auto e0_tag, auto n_tag, const float *row, int c, float *x) {
    constexpr int E0 = decltype(e0_tag)::value, N = decltype(n_tag)::value;
    if (VEC) {
      const float4 *row4 = (const float4 *)row;
      const int V4 = V >> 2;
#pragma unroll
      for (int j = 0; j < N / 4; ++j) {
        const float4 v = row4[min(c * (kChunk / 4) + (E0 / 4 + j) * kThreads + tid, V4 - 1)];
        x[4 * j] = v.x;
        x[4 * j + 1] = v.y;
        x[4 * j + 2] = v.z;
        x[4 * j + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int e = 0; e < N; ++e) x[e] = row[min(eidx(c, E0 + e), V - 1)];
    }
    __builtin_amdgcn_sched_barrier(0);  // all loads in flight before the first use
  };
  using Z = std::integral_constant<int, 0>;
  using Half = std::integral_constant<int, kPer / 2>;
  using Full = std::integral_constant<int, kPer>;
  uint32_t h[kPer];
  auto load = [&](int c) {
    float x[kPer];
    // row bases are wave-uniform: scalar base + 32-bit lane offsets
    load_part(Z(), Full(), p.logits + (size_t)__builtin_amdgcn_readfirstlane(src_s[0]) * V, c, x);
    if (EPT) {
      for (int g = 1; g < G; ++g) {
        const float *row = p.logits + (size_t)__builtin_amdgcn_readfirstlane(src_s[g]) * V;
        float y[kPer / 2];  // half a chunk at a time keeps the registers in bounds
        load_part(Z(), Half(), row, c, y);
#pragma unroll
        for (int e = 0; e < kPer / 2; ++e) x[e] += y[e];
        load_part(Half(), Half(), row, c, y);
#pragma unroll
        for (int e = 0; e < kPer / 2; ++e) x[kPer / 2 + e] += y[e];
      }
      const float n = (float)G;
#pragma unroll
      for (int e = 0; e < kPer; ++e) x[e] = x[e] / n;
    }
#pragma unroll
    for (int e = 0; e < kPer; ++e) h[e] = value_word(x[e]);
  };
  auto key_of = [&](int c, int e) -> uint64_t {
    const int idx = eidx(c, e);
    return idx < V ? make_key(h[e], idx) : 0;
  };
  uint64_t best = 0;
  for (int c = 0; c < n_chunks; ++c) {
    load(c);
    // indices grow with e: the first maximal word has the smallest index
    uint32_t bh = h[0];
    int be = 0;
#pragma unroll
    for (int e = 1; e < kPer; ++e) {
      const bool take = (h[e] > bh) & (eidx(c, e) < V);
      bh = take ? h[e] : bh;
      be = take ? e : be;
    }
    const int bi = eidx(c, be);
    best = umax64(best, bi < V ? make_key(bh, bi) : 0);
  }

  // ---- 2. threshold: the kd-th best of the 16 wave maxima (kd <= 16)
  const uint64_t wmax = wave_max_key(best);
  if (lane == 0) wave_s[wave] = wmax;
  __syncthreads();
  uint64_t tau = 0;
  {
    const uint64_t mine = lane < kThreads / 64 ? wave_s[lane] : 0;
    int rank = 0;
#pragma unroll
    for (int q = 0; q < kThreads / 64; ++q) rank += wave_s[q] > mine ? 1 : 0;
    const unsigned long long sel = __ballot(lane < kThreads / 64 && rank == kd - 1 && mine != 0);
    if (sel) tau = lane_key(mine, __builtin_ctzll(sel));
  }
  // tau == 0 (no threshold) only when fewer than kd waves hold elements,
  // so the row is shorter than the list

  // ---- 3. the elements reaching the threshold, ranked by counting
  const uint64_t t1 = tau == 0 ? 1 : tau;  // empty keys (0) never reach it
  if (best >= t1) {
    for (int c = 0; c < n_chunks; ++c) {
      if (MULTI) load(c);
#pragma unroll
      for (int e = 0; e < kPer; ++e) {
        const uint64_t k = key_of(c, e);
        if (k >= t1) {
          const int slot = atomicAdd(&count_s, 1);
          if (slot < kListCap) list_s[slot] = k;
        }
      }
    }
  }
  __syncthreads();
  const int n = count_s;
  if (n <= kListCap) {
    for (int i = tid; i < n; i += kThreads) {
      const uint64_t c = list_s[i];
      int r = 0;
      for (int j = 0; j < n; ++j) r += list_s[j] > c ? 1 : 0;
      if (r < kd) {
        top_s[r] = key_index(c);
        if (key_is_nan(c)) nan_s = 1;
      }
    }
  } else {
    // kd rounds of a workgroup maximum over the keys below the previous
    // pick (the row has more than kListCap > kd elements)
    uint64_t last = ~0ull;
    for (int r = 0; r < kd; ++r) {
      uint64_t b = 0;
      for (int c = 0; c < n_chunks; ++c) {
        if (MULTI) load(c);
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
          const uint64_t k = key_of(c, e);
          b = umax64(b, k < last ? k : 0);
        }
      }
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) {
        const uint32_t lo = __shfl_xor((uint32_t)b, off, 64);
        const uint32_t hi = __shfl_xor((uint32_t)(b >> 32), off, 64);
        b = umax64(b, ((uint64_t)hi << 32) | lo);
      }
      __syncthreads();  // wave_s is still read above / in the last round
      if (lane == 0) wave_s[wave] = b;
      __syncthreads();
      uint64_t w = 0;
#pragma unroll
      for (int q = 0; q < kThreads / 64; ++q) w = umax64(w, wave_s[q]);
      if (tid == 0) {
        top_s[r] = key_index(w);
        if (key_is_nan(w)) nan_s = 1;
      }
      last = w;
    }
  }
  __syncthreads();

  // ---- the template's candidates at depth d
  for (int i = tid; i < p.tpl_T; i += kThreads)
    if (i > 0 && p.tpl_depth[i] == d && p.tpl_kind[i] >= 0) p.next_ids[i] = top_s[p.tpl_kind[i]];
  if (tid == 0 && nan_s) atomicOr(p.status, PPD_DEV_NAN_LOGIT);
}

}  // namespace

hipError_t launch_next_tree(const NextTreeLaunch &p, int n_depths, hipStream_t s) {
  const dim3 grid(max(1, n_depths)), block(kThreads);
  const bool vec = p.vocab % 4 == 0 && (uintptr_t)p.logits % 16 == 0;
  const bool multi = p.vocab > kChunk, ept = p.n_ept > 1;
  void (*kernel)(NextTreeLaunch);
  if (ept)
    kernel = multi ? (vec ? next_tree_kernel<true, true, true> : next_tree_kernel<true, false, true>)
                   : (vec ? next_tree_kernel<false, true, true> : next_tree_kernel<false, false, true>);
  else
    kernel = multi ? (vec ? next_tree_kernel<true, true, false> : next_tree_kernel<true, false, false>)
                   : (vec ? next_tree_kernel<false, true, false> : next_tree_kernel<false, false, false>);
  if (p.ev_start)
    hipExtLaunchKernelGGL(kernel, grid, block, 0, s, (hipEvent_t)p.ev_start,
                          (hipEvent_t)p.ev_stop, 0, p);
  else
    hipLaunchKernelGGL(kernel, grid, block, 0, s, p);
  return hipGetLastError();
}
