// Hardware-aware tree sizing support (Section 4.2; Proposition 1 of the
// tree-construction appendix): the sparse-tree template of n candidates
// that maximises the expected number of accepted candidates, given an
// acceptance probability per (depth, rank).
//
// Under Proposition 1 a candidate contributes the product of the
// probabilities along its root path, and a product never exceeds its
// prefix's (probabilities are at most 1).  The best tree of n candidates is
// therefore the n rank paths of largest product, taken here by best-first
// expansion from the root: a max-heap of frontier paths ordered by product,
// then depth, then the rank path (lexicographically), popped n times; a
// popped path's children join the frontier.  Every path outside the
// frontier has an unpopped ancestor that orders before it, so the pops come
// out in the global order of all paths.  Host code; nothing runs on the GPU.
#include <algorithm>
#include <queue>
#include <vector>

#include "ppd_internal.h"

namespace {

struct Frontier {
  double v;               // product of the probabilities along the path
  std::vector<int> path;  // ranks, root first
  int parent;             // template index of the path's prefix
};

// true when a orders after b (so the heap's top is the first in order)
struct After {
  bool operator()(const Frontier &a, const Frontier &b) const {
    if (a.v != b.v) return a.v < b.v;
    if (a.path.size() != b.path.size()) return a.path.size() > b.path.size();
    return a.path > b.path;
  }
};

}  // namespace

extern "C" ppd_status ppd_sparse_template(const double *p_table, int32_t depth_max, int32_t k_max,
                                          int32_t n_cand, int32_t n_prompt, int32_t n_ept,
                                          int32_t *tpl_parent, int32_t *tpl_kind, int32_t *tpl_T,
                                          double *expected_accepted) {
  if (!p_table || !tpl_parent || !tpl_kind || !tpl_T)
    return ppd_fail(PPD_EINVAL, "NULL argument");
  if (depth_max < 1 || depth_max > PPD_NEXT_MAX_DEPTH || k_max < 1 || k_max > PPD_TOPK_MAX)
    return ppd_fail(PPD_EINVAL, "table of %d x %d outside [1, %d] x [1, %d]", depth_max, k_max,
                    PPD_NEXT_MAX_DEPTH, PPD_TOPK_MAX);
  for (int i = 0; i < depth_max * k_max; ++i)
    if (!(p_table[i] >= 0.0 && p_table[i] <= 1.0))
      return ppd_fail(PPD_EINVAL, "p_table[%d] is not a probability", i);
  if (n_cand < 0 || n_prompt < 0 || n_ept < 1 || n_ept > PPD_EPT_MAX ||
      (int64_t)n_prompt * n_ept > 32767)
    return ppd_fail(PPD_EINVAL, "n_cand, n_prompt >= 0 and 1 <= n_ept <= %d required",
                    PPD_EPT_MAX);
  const int64_t T = 1 + (int64_t)n_cand + (1 + (int64_t)n_cand) * n_prompt * n_ept;
  if (T > PPD_T_MAX) return ppd_fail(PPD_EINVAL, "template of %lld nodes > %d", (long long)T,
                                     PPD_T_MAX);
  int64_t n_paths = 0, level = 1;  // paths available up to depth_max (saturated)
  for (int d = 1; d <= depth_max && n_paths < n_cand; ++d) {
    level = std::min<int64_t>(level * k_max, 1 << 20);
    n_paths += level;
  }
  if (n_paths < n_cand) return ppd_fail(PPD_EINVAL, "only %lld rank paths", (long long)n_paths);

  std::priority_queue<Frontier, std::vector<Frontier>, After> heap;
  for (int r = 0; r < k_max; ++r) heap.push(Frontier{p_table[r], {r}, 0});
  tpl_parent[0] = -1;
  tpl_kind[0] = 0;
  double f = 0.0;
  for (int c = 1; c <= n_cand; ++c) {
    const Frontier top = heap.top();
    heap.pop();
    tpl_parent[c] = top.parent;
    tpl_kind[c] = top.path.back();
    f += top.v;
    const int d = (int)top.path.size();
    if (d < depth_max)
      for (int r = 0; r < k_max; ++r) {
        Frontier ch{top.v * p_table[d * k_max + r], top.path, c};
        ch.path.push_back(r);
        heap.push(std::move(ch));
      }
  }
  // one chain of n_prompt prompt tokens per EPT group under every node
  int t = n_cand + 1;
  for (int c = 0; c <= n_cand; ++c)
    for (int g = 0; g < n_ept; ++g) {
      int prev = c;
      for (int j = 0; j < n_prompt; ++j) {
        tpl_parent[t] = prev;
        tpl_kind[t] = -1 - (j * n_ept + g);
        prev = t++;
      }
    }
  *tpl_T = t;
  if (expected_accepted) *expected_accepted = f;
  return PPD_OK;
}
