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
// One workgroup per candidate depth: it walks the accepted node's prompt
// chain, selects the top kd of one logits row (each thread keeps a sorted
// list of the K best of its strided elements, K >= kd; kd rounds of a
// workgroup-wide maximum over the lists' heads then emit the ranks in
// order), and writes the template's candidates at its depth.  Workgroup 0 also writes the root and the prompt
// nodes.
#include "ppd_internal.h"

namespace {

// (value, index) ordered as in the rank definition: a NaN loses to every
// number, numbers compare by value, then by smaller index
struct Cand {
  float v;
  int i;  // INT_MAX: empty
};

__device__ __forceinline__ bool beats(const Cand &a, const Cand &b) {
  if (a.i == INT_MAX) return false;
  if (b.i == INT_MAX) return true;
  const bool an = a.v != a.v, bn = b.v != b.v;
  if (an != bn) return bn;
  if (an) return a.i < b.i;
  return a.v > b.v || (a.v == b.v && a.i < b.i);
}

// K: list length, a power of two >= every depth's rank count kd
template <int K>
__global__ __launch_bounds__(256) void next_tree_kernel(NextTreeLaunch p) {
  __shared__ int chain_s[PPD_NEXT_MAX_DEPTH + 1];
  __shared__ int found_s;
  __shared__ Cand wave_best[4];
  __shared__ int top_s[PPD_TOPK_MAX];
  __shared__ int nan_s;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int d = blockIdx.x + 1;  // candidate depth handled here
  const int kd = p.k_of_depth[d];

  // ---- root and prompt nodes (workgroup 0)
  if (blockIdx.x == 0) {
    for (int i = tid; i < p.tpl_T; i += blockDim.x) {
      const int kind = p.tpl_kind[i];
      if (i == 0)
        p.next_ids[0] = *p.next_tok;
      else if (kind < 0)
        p.next_ids[i] = p.vocab + (-kind - 1);
    }
  }
  if (kd == 0) return;  // no candidate at this depth

  // ---- the accepted node and its prompt chain, up to depth d
  if (tid == 0) {
    const int n = min(max(*p.n_path, 1), p.T);
    int a = p.path[n - 1];
    a = min(max(a, 0), p.T - 1);
    chain_s[0] = a;
    nan_s = 0;
  }
  __syncthreads();
  int src = chain_s[0];
  for (int j = 0; j < d; ++j) {
    const int cur = chain_s[j];
    if (tid == 0) found_s = INT_MAX;
    __syncthreads();
    for (int i = tid; i < p.T; i += blockDim.x)
      if (p.parent[i] == cur && p.ids[i] == p.vocab + j) atomicMin(&found_s, i);
    __syncthreads();
    const int f = found_s;
    if (f == INT_MAX) break;  // uniform: the chain ends here
    if (tid == 0) chain_s[j + 1] = f;
    src = f;
    __syncthreads();
  }

  // ---- per-thread sorted lists of the kd best strided elements of the row
  const float *row = p.logits + (size_t)src * p.vocab;
  Cand lst[K];
#pragma unroll
  for (int k = 0; k < K; ++k) lst[k] = Cand{0.f, INT_MAX};
  for (int v = tid; v < p.vocab; v += blockDim.x) {
    Cand c{row[v], v};
    if (!beats(c, lst[K - 1])) continue;
    // sorted insertion: walking from the best, c takes the first slot it
    // beats and the displaced entry moves on (the worst falls off)
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (beats(c, lst[k])) {
        const Cand t = lst[k];
        lst[k] = c;
        c = t;
      }
    }
  }

  // ---- kd rounds: the workgroup's best head is rank r; its owner pops it
  for (int r = 0; r < kd; ++r) {
    Cand b = lst[0];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      Cand o{__shfl_xor(b.v, off, 64), __shfl_xor(b.i, off, 64)};
      if (beats(o, b)) b = o;
    }
    if (lane == 0) wave_best[wave] = b;
    __syncthreads();
    Cand w = wave_best[0];
    for (int q = 1; q < 4; ++q)
      if (beats(wave_best[q], w)) w = wave_best[q];
    if (tid == 0) {
      top_s[r] = w.i == INT_MAX ? 0 : w.i;
      if (w.i == INT_MAX || w.v != w.v) nan_s = 1;
    }
    if (lst[0].i == w.i && w.i != INT_MAX) {  // the owner: drop its head
#pragma unroll
      for (int k = 0; k < K - 1; ++k) lst[k] = lst[k + 1];
      lst[K - 1] = Cand{0.f, INT_MAX};
    }
    __syncthreads();  // wave_best is rewritten next round
  }

  // ---- the template's candidates at depth d
  for (int i = tid; i < p.tpl_T; i += blockDim.x)
    if (i > 0 && p.tpl_depth[i] == d && p.tpl_kind[i] >= 0) p.next_ids[i] = top_s[p.tpl_kind[i]];
  if (tid == 0 && nan_s) atomicOr(p.status, PPD_DEV_NAN_LOGIT);
}

}  // namespace

hipError_t launch_next_tree(const NextTreeLaunch &p, int n_depths, hipStream_t s) {
  int kmax = 1;
  for (int d = 1; d <= PPD_NEXT_MAX_DEPTH; ++d) kmax = max(kmax, p.k_of_depth[d]);
  const dim3 grid(max(1, n_depths)), block(256);
  if (kmax <= 1)
    hipLaunchKernelGGL(next_tree_kernel<1>, grid, block, 0, s, p);
  else if (kmax <= 2)
    hipLaunchKernelGGL(next_tree_kernel<2>, grid, block, 0, s, p);
  else if (kmax <= 4)
    hipLaunchKernelGGL(next_tree_kernel<4>, grid, block, 0, s, p);
  else if (kmax <= 8)
    hipLaunchKernelGGL(next_tree_kernel<8>, grid, block, 0, s, p);
  else
    hipLaunchKernelGGL(next_tree_kernel<16>, grid, block, 0, s, p);
  return hipGetLastError();
}
