/*
 * ppd.h -- C ABI of the Parallel Prompt Decoding (PPD) tree-verification step
 * for AMD Instinct MI355X (gfx950).
 *
 * One decode step of PPD (Section 3 of the paper: candidate generation,
 * verification and acceptance merged into a single forward pass) is, on the
 * verification side:
 *
 *   ppd_build_tree_mask  host: depths and ancestor bitmask of the candidate
 *                        tree with its prompt-token chains (Section 4.1)
 *   ppd_verify_step      device: one forward pass of the frozen decoder over
 *                        all T tree nodes against the KV cache under the tree
 *                        mask; per-node logits and greedy tokens
 *   ppd_accept           device: exact-matching verification, longest
 *                        accepted root path, bonus token (Section 3)
 *   ppd_kv_compact       device: commit the accepted nodes' keys/values to
 *                        the single shared KV cache (Section 5.3)
 *   ppd_next_tree        device: the next step's candidate tree from this
 *                        step's outputs (Section 3, step (1))
 *
 * Conventions shared by every call
 * --------------------------------
 * Tree.  Nodes 0..T-1 in topological order: parent[0] = -1 (node 0 is the
 *   root: the last verified token, whose keys/values are not cached yet) and
 *   0 <= parent[i] < i.  ids[i] < vocab is a vocabulary token; ids[i] >= vocab
 *   is prompt token ids[i] - vocab (< n_prompt).  Node i sits at position
 *   L + depth[i] (Section 3.1: a prompt token takes the position of the token
 *   it predicts) and attends to cache positions [0, L), to its tree ancestors
 *   and to itself (Section 4.1).  1 <= T <= PPD_T_MAX.
 * Mask.  uint64 mask[T][PPD_MASK_WORDS]; bit (j % 64) of word j / 64 of row i
 *   is set iff node j is node i or one of its ancestors.
 * Memory.  Every pointer marked "device" is HIP device memory owned by the
 *   caller and must stay valid until the enqueued work completes.  The
 *   library allocates nothing and keeps no state besides the thread-local
 *   error string and the optional thread-local kernel timer.  Weights and
 *   caches of PPD_BF16 models are bfloat16 (raw 16-bit words), their
 *   activations fp32; PPD_F32 models use float32 throughout.
 * Streams.  Device calls enqueue on `stream` (a hipStream_t; NULL = default
 *   stream) and return without waiting.  verify -> accept -> compact must be
 *   enqueued in that order on one stream; no host synchronisation is needed
 *   between them.  Calls never allocate, synchronise or memset, so a caller may
 *   capture them into a HIP graph.
 * Errors.  Host-checkable conditions are rejected before anything is
 *   enqueued, with a non-zero ppd_status and a message from ppd_last_error().
 *   Invalid data that only the device sees (a token id out of range, a parent
 *   index out of range in ppd_accept, a NaN logit) sets a bit in the
 *   workspace's status word (read with ppd_device_status); kernels clamp the
 *   offending index so that no access leaves its buffer.
 */
#ifndef PPD_H
#define PPD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  PPD_OK = 0,
  PPD_EINVAL = 1,       /* null pointer, bad size or model description     */
  PPD_ETREE = 2,        /* parent array is not a topological tree          */
  PPD_ECAPACITY = 3,    /* L + T exceeds the cache capacity                */
  PPD_EDEVICE = 4,      /* a HIP launch or runtime call failed             */
  PPD_EUNSUPPORTED = 5, /* shape outside what the kernels implement        */
  PPD_EWORKSPACE = 6    /* workspace missing or smaller than required      */
} ppd_status;

typedef enum { PPD_F32 = 0, PPD_BF16 = 1 } ppd_dtype;

#define PPD_T_MAX 128
#define PPD_BATCH_MAX 16  /* sequences in one ppd_verify_batch call */
#define PPD_CAPACITY_MAX (1 << 24) /* KV positions per head */
#define PPD_MASK_WORDS 2

/* device status bits (ppd_device_status) */
#define PPD_DEV_BAD_TOKEN 1u   /* an id >= vocab + n_prompt was clamped      */
#define PPD_DEV_BAD_PARENT 2u  /* ppd_accept saw parent[i] outside [0, i)    */
#define PPD_DEV_NAN_LOGIT 4u   /* a NaN logit was seen by the greedy argmax  */
#define PPD_DEV_XCD_PLACEMENT 8u /* workgroups that hand partial sums over
                                    through one XCD's L2 ran on different
                                    XCDs (the dispatch was not round-robin
                                    over the 8 XCDs); outputs are invalid    */
#define PPD_DEV_SYNC_TIMEOUT 16u /* a workgroup gave up waiting for the other
                                    workgroups of its tile (bounded wait); the
                                    step's outputs are then invalid          */

/*
 * Llama-style decoder (the paper's MobileLLaMA / Vicuna family): pre-RMSNorm
 * (eps rms_eps), rotary embedding with rotate-half pairing (dimension i pairs
 * with i + head_dim/2, frequency rope_base^(-2i/head_dim)), multi-head
 * attention with n_kv_heads dividing n_heads, SwiGLU MLP, untied LM head.
 * All weight pointers are device pointers; per-layer tensors are given as
 * HOST arrays of n_layers device pointers.  For PPD_BF16 models the five
 * projection matrices (w_qkv, w_o, w_gate_up, w_down, lm_head) are passed in
 * the packed form written by ppd_pack_weight from the row-major matrices
 * below; every other tensor, and every tensor of PPD_F32 models, is passed
 * row-major as listed.  Row-major layouts:
 *   tok_emb     [vocab][hidden]
 *   prompt_emb  [n_prompt][hidden]       trained prompt-token embeddings
 *   attn_norm   [hidden]     per layer
 *   w_qkv       [(n_heads + 2 n_kv_heads) head_dim][hidden]  rows q | k | v
 *   w_o         [hidden][n_heads head_dim]
 *   mlp_norm    [hidden]
 *   w_gate_up   [2 ffn][hidden]           rows gate | up
 *   w_down      [hidden][ffn]
 *   final_norm  [hidden]
 *   lm_head     [vocab][hidden]
 */
typedef struct {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab, n_prompt;
  float rms_eps, rope_base;
  int32_t dtype; /* ppd_dtype */
  const void *tok_emb, *prompt_emb;
  const void *const *attn_norm, *const *w_qkv, *const *w_o;
  const void *const *mlp_norm, *const *w_gate_up, *const *w_down;
  const void *final_norm, *lm_head;
} ppd_model;

/*
 * Weight packing for PPD_BF16 models.  The verification step streams every
 * projection weight from HBM once per step (its cost is that stream), so the
 * library keeps them in the order its matrix-core GEMMs consume them,
 * group-major: a group is 16 output rows -- 16 QKV rows (dims 8j .. 8j + 7
 * of a head and their RoPE partners + 64), 16 gate/up features (their 16
 * gate rows, then their 16 up rows), or 16 consecutive rows of the other
 * matrices -- and group g's 64-column chunks follow one another, each a run
 * of 1 KB operand fragments of 16 rows x 32 columns in the lane order of the
 * gfx950 bf16 MFMA instruction: 16-byte item (g, chunk, sub-tile q, k-step s,
 * lane l) holds row r(g, q, l % 16), columns 64 chunk + 32 s + 8 (l / 16) ..
 * + 7.  The layout fixes no tiling: how many groups a workgroup streams and
 * over which columns is chosen per step (from T).  Rows past the matrix
 * (the LM head's last group when vocab % 16 != 0) are zero.  The packed form
 * depends only on the matrix, not on T or L; pack once at load time.
 *   kind  which matrix (ppd_weight_kind); rows, cols: its row-major shape,
 *         i.e. PPD_W_QKV [(n_heads + 2 n_kv_heads) 128][hidden],
 *         PPD_W_O [hidden][n_heads 128], PPD_W_GATE_UP [2 ffn][hidden],
 *         PPD_W_DOWN [hidden][ffn], PPD_W_LM_HEAD [vocab][hidden].
 *         cols % 64 == 0; rows % 128 == 0 except for the LM head.
 *         Size: (rows rounded up to 16) x cols x 2 bytes.
 *   src   device bfloat16 [rows][cols], row-major (not modified)
 *   dst   device buffer of ppd_packed_weight_bytes(kind, rows, cols) bytes,
 *         caller-owned, must not overlap src
 * ppd_packed_weight_bytes returns 0 for invalid arguments (message in
 * ppd_last_error).  ppd_pack_weight enqueues one kernel on `stream`;
 * PPD_EINVAL / PPD_EUNSUPPORTED for bad arguments, nothing enqueued.
 */
typedef enum {
  PPD_W_QKV = 0,
  PPD_W_O = 1,
  PPD_W_GATE_UP = 2,
  PPD_W_DOWN = 3,
  PPD_W_LM_HEAD = 4
} ppd_weight_kind;

size_t ppd_packed_weight_bytes(int32_t kind, int32_t rows, int32_t cols);
ppd_status ppd_pack_weight(int32_t kind, int32_t rows, int32_t cols, const void *src, void *dst,
                           void *stream);

/*
 * The single KV cache of the accepted sequence (device memory, caller-owned).
 *   k  [n_layers][n_kv_heads][capacity][head_dim]   keys after RoPE
 *   v  [n_layers][n_kv_heads][head_dim][capacity]   values, position-minor
 * Positions [0, L) hold the accepted prefix.  ppd_verify_step writes the keys
 * and values of tree node i to position L + i (scratch beyond the prefix);
 * ppd_kv_compact moves the accepted ones down to L, L+1, ...
 * len_dev (optional, device int32) receives L + n_path from ppd_kv_compact.
 */
typedef struct {
  void *k, *v;
  int32_t capacity;   /* positions per head, 1 .. PPD_CAPACITY_MAX */
  int32_t *len_dev;
} ppd_kv;

/* Bytes of device workspace ppd_verify_step needs for trees of up to t_max
 * nodes and caches of up to max_len positions.  0 on invalid input. */
size_t ppd_workspace_bytes(const ppd_model *model, int32_t t_max, int32_t max_len);

/* Zero the workspace's header -- the status word and a line of zeros the
 * kernels read in place of padding (enqueued on `stream`).  Call once after
 * allocating a workspace; later calls never write the header except for
 * status bits. */
ppd_status ppd_workspace_init(void *ws, size_t ws_bytes, void *stream);

/*
 * Host-side tree preparation (Section 4.1).  parent: host int32[T].
 * depth_out: host int32[T], root depth 0.  mask_out: host uint64[T][2] as
 * described above.  Returns PPD_ETREE if parent is not a topological tree,
 * PPD_EINVAL for T outside [1, PPD_T_MAX] or null pointers.
 */
ppd_status ppd_build_tree_mask(int32_t T, const int32_t *parent, int32_t *depth_out,
                               uint64_t *mask_out);

/*
 * One forward pass over the T tree nodes (Sections 3 and 4.1).
 *   L       tokens already in the cache (host value); needs L + T <= capacity
 *   ids     device int32[T]
 *   depth   device int32[T] (from ppd_build_tree_mask)
 *   mask    device uint64[T][2]
 *   ws      device workspace of ws_bytes >= ppd_workspace_bytes(model, T, L)
 *   logits  device float32[T][vocab], or NULL to skip storing logits
 *   pred    device int32[T]: greedy token of every node (smallest index among
 *           equal maxima)
 * Also writes the nodes' keys/values to cache positions L .. L+T-1.
 */
ppd_status ppd_verify_step(const ppd_model *model, const ppd_kv *kv, int32_t L, int32_t T,
                           const int32_t *ids, const int32_t *depth, const uint64_t *mask,
                           void *ws, size_t ws_bytes, float *logits, int32_t *pred,
                           void *stream);

/*
 * Several sequences in one step, sharing the weight stream (batch > 1; the
 * paper's batch-size experiment, Section "Effect of Batch Size on
 * Speedup"): sequence s has its own cache kvs[s], cached length L[s] and
 * tree of T[s] nodes, and the sequences are independent -- each sequence's
 * logits, greedy tokens and cache rows are those ppd_verify_step gives for
 * it alone.  The trees are packed in sequence order: sequence s owns rows
 * [t0_s, t0_s + T[s]) of ids, depth, mask, logits and pred, t0_s = T[0] + ..
 * + T[s - 1]; its depth and mask rows refer to its own tree (node indices
 * local to the sequence, as ppd_build_tree_mask gives them).
 *   B          1 .. PPD_BATCH_MAX sequences; T[0] + .. + T[B - 1] <= PPD_T_MAX
 *   kvs        host array of B cache descriptors (all of the model's dtype)
 *   L, T       host int32[B]
 *   ws         as for ppd_verify_step with t_max = the total token count
 * B > 1 needs a bf16 model (PPD_EUNSUPPORTED otherwise).  Acceptance and
 * compaction stay per sequence: ppd_accept(T[s], parent + t0_s, ids + t0_s,
 * pred + t0_s, ...) and ppd_kv_compact(model, &kvs[s], L[s], ...).
 */
ppd_status ppd_verify_batch(const ppd_model *model, int32_t B, const ppd_kv *kvs,
                            const int32_t *L, const int32_t *T, const int32_t *ids,
                            const int32_t *depth, const uint64_t *mask, void *ws, size_t ws_bytes,
                            float *logits, int32_t *pred, void *stream);

/*
 * Exact-matching verification and acceptance (Section 3).  Node i > 0 is
 * verified iff its parent is verified (the root always is), ids[i] < vocab
 * and ids[i] == pred[parent[i]]; prompt nodes never are.  The accepted node
 * is the deepest verified one (ties: smallest index).  Outputs (device):
 *   path      int32[T]: accepted node indices root first (path[0] = 0)
 *   n_path    int32: depth of the accepted node + 1 = tokens emitted this
 *             step (accepted candidates plus the bonus token)
 *   next_tok  int32: pred[accepted node], the bonus token and next root
 * parent, ids, pred: device int32[T].  ws: the workspace (status word).
 */
ppd_status ppd_accept(int32_t T, const int32_t *parent, const int32_t *ids,
                      const int32_t *pred, int32_t vocab, int32_t *path, int32_t *n_path,
                      int32_t *next_tok, void *ws, size_t ws_bytes, void *stream);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture that forbids allocation, serving loops that must not allocate,
 * harnesses that forbid it): ppd_verify_step with the workspace taken from a
 * static device array of the library, PPD_STATIC_WS_BYTES (64 MiB) on each
 * GPU it runs on, held until the process ends; the call allocates nothing.
 * Arguments as ppd_verify_step, without ws / ws_bytes; status_out (optional
 * device uint32) receives the step's device status word (ppd_device_status
 * bits), the header of the array being cleared at the start of every call.
 * PPD_EWORKSPACE when the step needs more than PPD_STATIC_WS_BYTES
 * (ppd_workspace_bytes(model, T, capacity); a Vicuna-13B-shaped step needs
 * about 15 MiB with a 64-node tree, 30 MiB with 128), nothing enqueued.  All
 * calls on one GPU share the array: calls that may overlap on one GPU
 * (unordered streams, several threads) race and must not be made.
 */
#define PPD_STATIC_WS_BYTES (64u << 20)
ppd_status ppd_verify_step_static(const ppd_model *model, const ppd_kv *kv, int32_t L, int32_t T,
                                  const int32_t *ids, const int32_t *depth, const uint64_t *mask,
                                  float *logits, int32_t *pred, uint32_t *status_out, void *stream);

/*
 * Commit accepted keys/values (Section 5.3: one cache shared by guessing and
 * verification; prompt-token entries are never committed):
 * cache[L + k] <- cache[L + path[k]] for k < *n_path, every layer and kv head.
 * path: device int32[path_len] and n_path: device int32 (as written by
 * ppd_accept, whose path holds T entries: pass path_len = T).  L: host value
 * used by the matching ppd_verify_step.  *n_path is read on the device and
 * clamped to [0, min(path_len, capacity - L)], so a stale or foreign count
 * never reads past the path or writes past the cache; path entries are
 * clamped the same way.  1 <= path_len <= PPD_T_MAX, else PPD_EINVAL.
 */
ppd_status ppd_kv_compact(const ppd_model *model, const ppd_kv *kv, int32_t L,
                          const int32_t *path, int32_t path_len, const int32_t *n_path,
                          void *stream);

/*
 * Candidate generation for the next step (Section 3, step (1); Section 3.1;
 * Section 4 with the tree-construction appendix), so that the decode loop
 * verify -> accept -> compact -> next tree runs without a host round trip.
 * The next tree has the fixed shape of a template (tpl_parent, a topological
 * parent array with tpl_parent[0] = -1) whose token ids are written to
 * next_ids:
 *   node 0 (root)           *next_tok, the bonus token from ppd_accept;
 *   tpl_kind[i] = r >= 0     a candidate of rank r: the r-th best token of the
 *                            logits of the accepted node's d-th prompt token,
 *                            d = the node's depth in the template (the
 *                            accepted node's prompt chain: its child with id
 *                            vocab + 0, that node's child with id vocab + 1,
 *                            ...; past the chain's end its deepest node, or
 *                            the accepted node itself when it has none);
 *   tpl_kind[i] = -1 - q     prompt embedding q (id vocab + q).
 * Ensemble prompt tokens (Section 3.2, the EPT appendix): with n_ept EPTs per
 * prompt token, prompt embedding q is the EPT of group q % n_ept at token
 * distance q / n_ept + 1; a node carries one chain per group (group g: ids
 * vocab + g, vocab + n_ept + g, ...), which under the ancestor mask is the
 * ensemble mask, and the logits row behind a depth-d candidate is the mean of
 * the groups' d-th chain nodes' rows (float32: added in group order, then
 * divided by n_ept).  n_ept = 1 is the plain single chain (prompt id j at
 * distance j + 1).
 * Ranks order larger logits first, equal logits by smaller index, NaN last
 * (a NaN among the selected ranks sets PPD_DEV_NAN_LOGIT).  One workgroup
 * per candidate depth reads one logits row.  The template's
 * parent/depth/mask are the caller's (ppd_build_tree_mask on tpl_parent).
 *   T, parent, ids    this step's tree (device int32[T])
 *   n_prompt, n_ept   token distances per chain, EPT groups (1 <= n_ept <=
 *                     PPD_EPT_MAX); prompt embeddings n_prompt * n_ept
 *   logits            device float32[T][vocab] written by ppd_verify_step
 *   path, n_path, next_tok   device, as written by ppd_accept (path holds
 *                     T entries, all read)
 *   tpl_T, tpl_parent, tpl_kind   HOST arrays of tpl_T entries (copied into
 *                     the launch; the call keeps no pointer to them)
 *   next_ids          device int32[tpl_T] (output)
 *   ws                the workspace (status word)
 * Template rules (else PPD_EINVAL, nothing enqueued): 1 <= tpl_T <= PPD_T_MAX;
 * a candidate's parent is the root or a candidate, rank < PPD_TOPK_MAX and <
 * vocab, depth <= 15; a distance-1 EPT hangs under the root or a candidate,
 * a distance-(j+1) EPT of group g under the distance-j EPT of group g, and
 * j < n_prompt.
 */
#define PPD_TOPK_MAX 16
#define PPD_EPT_MAX 64
ppd_status ppd_next_tree(int32_t T, const int32_t *parent, const int32_t *ids, int32_t vocab,
                         int32_t n_prompt, int32_t n_ept, const float *logits, const int32_t *path,
                         const int32_t *n_path, const int32_t *next_tok, int32_t tpl_T,
                         const int32_t *tpl_parent, const int32_t *tpl_kind, int32_t *next_ids,
                         void *ws, size_t ws_bytes, void *stream);

/*
 * Tree sizing (Section 4.2, the hardware-aware tree size; Proposition 1 of
 * the tree-construction appendix).  Host only: enqueues nothing.
 * Builds the template (for ppd_next_tree) of the n_cand candidates that
 * maximise the expected number of accepted candidates when the rank-r guess
 * at depth d is accepted, given its parent is, with probability
 * p_table[(d - 1) * k_max + r], independently (Proposition 1: the sum over
 * candidates of the product of the probabilities along their root paths).
 * The best tree holds the n_cand rank paths of largest product (ties:
 * shallower, then lexicographically smaller rank path); its layout is the
 * root, the candidates in that order, then under the root and every
 * candidate, in node order, one chain of n_prompt prompt tokens per EPT group
 * (kinds as in ppd_next_tree).  The caller picks n_cand by measuring the
 * forward latency of the resulting T (Speedup = (1 + expected) / latency).
 *   p_table           host double[depth_max][k_max], entries in [0, 1]
 *   depth_max, k_max  1..15, 1..PPD_TOPK_MAX
 *   tpl_parent, tpl_kind   host int32[PPD_T_MAX] (outputs), tpl_T their length
 *   expected_accepted host double (output, may be NULL): Proposition 1's sum
 * PPD_EINVAL if T = 1 + n_cand + (1 + n_cand) n_prompt n_ept > PPD_T_MAX, the
 * table holds fewer than n_cand rank paths, or an argument is out of range.
 */
ppd_status ppd_sparse_template(const double *p_table, int32_t depth_max, int32_t k_max,
                               int32_t n_cand, int32_t n_prompt, int32_t n_ept,
                               int32_t *tpl_parent, int32_t *tpl_kind, int32_t *tpl_T,
                               double *expected_accepted);

/*
 * Profiling aid, not needed for correctness.  While set, every
 * ppd_verify_step issued from this thread launches the i-th kernel of kind
 * `kind` in the step (i < n_events) with start_events[i] / stop_events[i]
 * attached to the dispatch itself (hipExtLaunchKernelGGL), so they take the
 * kernel's own start and end times on the step's stream.  kind: 0 QKV GEMM, 1 tree attention, 2 output
 * projection, 3 gate/up GEMM, 4 down projection, 5 LM head; kind 6 times
 * the one kernel of each ppd_next_tree call instead (with the first events).  The arrays are
 * host arrays of hipEvent_t and must stay valid while set; n_events = 0
 * disables.  Thread-local setting.
 */
ppd_status ppd_set_kernel_timer(int32_t kind, void *const *start_events, void *const *stop_events,
                                int32_t n_events);

/*
 * Measurement aid, not needed for correctness: the practical HBM read rate
 * the step's weight streams are compared with.  One launch of 256
 * workgroups (one per compute unit, 16-byte non-temporal loads, several in
 * flight per thread) reads `bytes` bytes of device buffer `buf` once
 * (`bytes` a multiple of 16, buf 16-byte aligned) and writes a 32-bit XOR of
 * everything read to device `sink` (so the loads cannot be dropped).
 * Enqueued on `stream`; PPD_EINVAL for a null pointer or a misaligned size.
 */
ppd_status ppd_read_probe(const void *buf, size_t bytes, uint32_t *sink, void *stream);

/* Synchronously read (and optionally clear) the workspace status word. */
ppd_status ppd_device_status(void *ws, size_t ws_bytes, uint32_t *status_out, int32_t clear,
                             void *stream);

/* Message for the last non-OK status returned on this thread. */
const char *ppd_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* PPD_H */
