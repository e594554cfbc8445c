"""CPU oracle for the Parallel Prompt Decoding (PPD) tree-verification step.

TEST INFRASTRUCTURE.  Only the test-suite, the smoke check and the benchmark's
CPU-baseline leg may import this module.  The GPU library never calls it and
shares no code with it.

Plain, slow, float64 numpy.  Each function restates what the paper computes:

* Section 3 (guess-and-verify in one step): the tree of candidate tokens, with
  prompt tokens appended, goes through one forward pass of the frozen decoder;
  candidates are verified by exact matching against the model's greedy token;
  the accepted candidates enter the sequence and the KV cache.
* Section 3.1: a prompt token stands at the position of the future token it
  approximates, so a node at depth k of the tree sits at position L + k.
* Section 4.1 (customised sparse tree attention, after SpecInfer): every node
  attends to the cached prefix, to its own ancestors and to itself, and to
  nothing else, so many candidates are scored without growing the batch.
* Section 5.3 (memory efficiency): a single KV cache is shared by guessing and
  verification; only accepted tokens are committed to it.

The decoder is Llama-style (the paper's MobileLLaMA / Vicuna family):
pre-RMSNorm, rotary position embedding with rotate-half pairing, multi-head
(optionally grouped) attention, SwiGLU MLP, tied nothing.

Precision.  Every sum is taken in float64.  `store` is the storage type of the
model: its weights and embeddings (already rounded on input) and its KV cache.
The keys and values a step writes to the cache are rounded to it; the
activations between matrix products (queries, the normalised operands, the
attention and SwiGLU outputs) are rounded only for a float32 model, whose GPU
path stores them in float32 -- a bf16 model's GPU path keeps them in float32
too and feeds the bf16 matrix cores their two-part (hi + lo) bf16 sum, so they
are left unrounded here.  The residual stream, softmax and logits are never
rounded.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

# ----------------------------------------------------------------------------
# storage rounding


def round_store(x: np.ndarray, store: Optional[str]) -> np.ndarray:
    """Round float64 values to the storage type and return them as float64.

    "bf16": round to nearest even on the bfloat16 grid (via float32, whose
    rounding is also to nearest even).  "f32": float32.  None: unchanged."""
    if store is None:
        return x
    x32 = np.asarray(x, dtype=np.float32)
    if store == "f32":
        return x32.astype(np.float64)
    if store == "bf16":
        b = x32.view(np.uint32).astype(np.uint64)
        nan = np.isnan(x32)
        b = (b + 0x7FFF + ((b >> 16) & 1)) & 0xFFFF0000
        out = b.astype(np.uint32).view(np.float32).astype(np.float64)
        out[nan] = np.nan
        return out
    raise ValueError(store)


def to_f64(t) -> np.ndarray:
    """torch tensor (any float dtype, any device) or array -> float64 numpy."""
    if hasattr(t, "detach"):
        t = t.detach()
        if t.dtype.is_floating_point and t.element_size() < 4:
            t = t.float()
        return t.cpu().numpy().astype(np.float64)
    return np.asarray(t, dtype=np.float64)


# ----------------------------------------------------------------------------
# model container


class Model:
    """Weights of one decoder, converted to float64 on access.

    `w` is the dict produced by `synth.model.make_weights` (torch tensors) or
    an equivalent dict of arrays.  Layers are converted lazily and not kept,
    so a 7B-shaped model fits in host memory as its bf16 original."""

    def __init__(self, shape, w: Dict, keep_layers: bool = True):
        self.shape = shape
        self._w = w
        self._keep = keep_layers
        self._cache: Dict[int, Dict[str, np.ndarray]] = {}
        self.tok_emb_src = w["tok_emb"]
        self.prompt_emb = to_f64(w["prompt_emb"])
        self.final_norm = to_f64(w["final_norm"])
        self._lm_head = None

    @property
    def lm_head(self) -> np.ndarray:
        if self._lm_head is None:
            self._lm_head = to_f64(self._w["lm_head"])
        return self._lm_head

    def embed_row(self, token: int) -> np.ndarray:
        return to_f64(self.tok_emb_src[int(token)])

    def layer(self, l: int) -> Dict[str, np.ndarray]:
        if l in self._cache:
            return self._cache[l]
        src = self._w["layers"][l]
        lay = {k: to_f64(v) for k, v in src.items()}
        if self._keep:
            self._cache[l] = lay
        return lay


# ----------------------------------------------------------------------------
# tree structure (Section 4.1)


def validate_tree(parent: Sequence[int]) -> None:
    """Topologically ordered tree: parent[0] = -1 (root), 0 <= parent[i] < i."""
    p = np.asarray(parent)
    if p.ndim != 1 or p.size < 1 or p[0] != -1:
        raise ValueError("parent[0] must be -1")
    for i in range(1, p.size):
        if not (0 <= p[i] < i):
            raise ValueError(f"parent[{i}]={p[i]} is not an earlier node")


def build_mask(parent: Sequence[int]) -> Tuple[np.ndarray, np.ndarray]:
    """depth[i] (root = 0) and the tree attention mask.

    anc[i, j] is True iff node j lies on the root-to-i path (j == i included):
    the only tree nodes i may attend to (Section 4.1)."""
    validate_tree(parent)
    T = len(parent)
    depth = np.zeros(T, np.int64)
    anc = np.zeros((T, T), bool)
    for i in range(T):
        j = i
        while j != -1:
            anc[i, j] = True
            j = int(parent[j])
        depth[i] = anc[i].sum() - 1
    return depth, anc


def pack_mask(anc: np.ndarray, words: int = 2) -> np.ndarray:
    """Bit-packed mask rows: bit (j mod 64) of word j // 64 is anc[i, j]."""
    T = anc.shape[0]
    out = np.zeros((T, words), np.uint64)
    for i in range(T):
        for j in range(T):
            if anc[i, j]:
                out[i, j // 64] |= np.uint64(1) << np.uint64(j % 64)
    return out


# ----------------------------------------------------------------------------
# decoder building blocks


def rms_scale(x: np.ndarray, eps: float) -> np.ndarray:
    """Per-row RMSNorm factor 1 / sqrt(mean(x^2) + eps)."""
    return 1.0 / np.sqrt(np.mean(x * x, axis=-1) + eps)


def round_act(x: np.ndarray, store: Optional[str]) -> np.ndarray:
    """An activation between matrix products: float32 models store it in
    float32; bf16 models keep it unrounded (see the module header)."""
    return round_store(x, "f32") if store == "f32" else x


def normed_rows(x: np.ndarray, g: np.ndarray, eps: float, store) -> Tuple[np.ndarray, np.ndarray]:
    """RMSNorm(x) * g, split as (operand, row scale).

    RMSNorm(x)_k * g_k = r * (x_k * g_k) with r = 1/sqrt(mean(x^2) + eps), so
    (RMSNorm(x) * g) W = r * ((x * g) W) exactly; the operand x * g is
    rounded as an activation (round_act).  Returns (x * g, r)."""
    return round_act(x * g, store), rms_scale(x, eps)


def rope_tables(pos: np.ndarray, d: int, base: float) -> Tuple[np.ndarray, np.ndarray]:
    """cos/sin of pos * base^(-2i/d), i < d/2 (rotary embedding)."""
    i = np.arange(d // 2, dtype=np.float64)
    inv = base ** (-2.0 * i / d)
    ang = np.asarray(pos, np.float64)[:, None] * inv[None, :]
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half rotary embedding; x [n, heads, d], cos/sin [n, d/2].

    Pairs (i, i + d/2) rotate by the angle of frequency i."""
    h = x.shape[-1] // 2
    a, b = x[..., :h], x[..., h:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def embed(model: Model, ids: Sequence[int]) -> np.ndarray:
    """Token embedding for ids < vocab; prompt-token embedding ids - vocab else
    (prompt tokens are trained embeddings appended to the input, Section 3)."""
    V = model.shape.vocab
    rows = []
    for t in ids:
        t = int(t)
        if 0 <= t < V:
            rows.append(model.embed_row(t))
        elif V <= t < V + model.shape.n_prompt:
            rows.append(model.prompt_emb[t - V])
        else:
            raise ValueError(f"token id {t} out of range")
    return np.stack(rows)


# ----------------------------------------------------------------------------
# the verification forward pass (Sections 3 and 4.1)


def _matmul(a: np.ndarray, b: np.ndarray, acc: str) -> np.ndarray:
    """a @ b summed in float64 ("f64") or, for a second, independently
    rounded computation of the same values, in float32 ("f32": operands and
    products in float32, as a float32-accumulating matrix unit sums them)."""
    if acc == "f64":
        return a @ b
    if acc == "f32":
        return (a.astype(np.float32) @ b.astype(np.float32)).astype(np.float64)
    raise ValueError(acc)


def verify_forward(model: Model, k_cache: Sequence[np.ndarray], v_cache: Sequence[np.ndarray],
                   L: int, ids: Sequence[int], parent: Sequence[int],
                   store: Optional[str], acc: str = "f64", taps: Sequence[int] = ()) -> Dict:
    """One forward pass over all T tree nodes.

    k_cache[l] / v_cache[l]: [n_kv_heads, >=L, d] float64 keys (after RoPE) and
    values of the accepted prefix.  Node i sits at position L + depth[i] and
    attends to cache positions [0, L) and to its tree ancestors and itself.

    acc: "f64" (the oracle) or "f32" -- every matrix product summed in
    float32 and the residual stream kept in float32, the same values rounded
    differently; two such computations bound how closely any two correct
    implementations with the same storage roundings can agree.
    taps: decoder depths n (1 <= n <= n_layers) at which the final norm and
    LM head are also applied to the residual stream after n layers, i.e. the
    logits of the same model cut to its first n layers ("tap_logits").

    Returns logits [T, vocab], the tree keys/values per layer
    ([n_kv_heads, T, d], rounded to the storage type) and depth."""
    sh = model.shape
    mm = lambda a, b: _matmul(a, b, acc)
    resid = (lambda v: v) if acc == "f64" else (lambda v: round_store(v, "f32"))

    def head(xr):
        a_, r_ = normed_rows(xr, model.final_norm, sh.rms_eps, store)
        return r_[:, None] * mm(a_, model.lm_head.T)

    tap_logits = {}
    T = len(ids)
    depth, anc = build_mask(parent)
    pos = L + depth
    cos, sin = rope_tables(pos, sh.head_dim, sh.rope_base)
    nh, nkv, d = sh.n_heads, sh.n_kv_heads, sh.head_dim
    grp = nh // nkv
    x = embed(model, ids)                                   # residual stream
    tree_k, tree_v = [], []
    for l in range(sh.n_layers):
        lay = model.layer(l)
        a, r = normed_rows(x, lay["attn_norm"], sh.rms_eps, store)
        qkv = r[:, None] * mm(a, lay["w_qkv"].T)
        q = qkv[:, :nh * d].reshape(T, nh, d)
        k = qkv[:, nh * d:(nh + nkv) * d].reshape(T, nkv, d)
        v = qkv[:, (nh + nkv) * d:].reshape(T, nkv, d)
        q = round_act(apply_rope(q, cos, sin), store)
        k = round_store(apply_rope(k, cos, sin), store)     # the cache's type
        v = round_store(v, store)
        kt = k.transpose(1, 0, 2)                           # [nkv, T, d]
        vt = v.transpose(1, 0, 2)
        tree_k.append(kt)
        tree_v.append(vt)
        o = np.zeros((T, nh, d))
        kcl, vcl = k_cache[l], v_cache[l]
        for h in range(nh):
            kh = np.concatenate([kcl[h // grp][:L], kt[h // grp]], axis=0)
            vh = np.concatenate([vcl[h // grp][:L], vt[h // grp]], axis=0)
            s = mm(q[:, h, :], kh.T) / np.sqrt(d)           # [T, L+T]
            s[:, L:][~anc] = -np.inf                        # tree part: ancestors only
            o[:, h, :] = mm(softmax_rows(s), vh)
        o = round_act(o.reshape(T, nh * d), store)
        x = resid(x + mm(o, lay["w_o"].T))
        a, r = normed_rows(x, lay["mlp_norm"], sh.rms_eps, store)
        gu = r[:, None] * mm(a, lay["w_gate_up"].T)
        act = round_act(silu(gu[:, :sh.ffn]) * gu[:, sh.ffn:], store)
        x = resid(x + mm(act, lay["w_down"].T))
        if l + 1 in taps and l + 1 < sh.n_layers:
            tap_logits[l + 1] = head(x)
    logits = head(x)
    if sh.n_layers in taps:
        tap_logits[sh.n_layers] = logits
    return {"logits": logits, "tree_k": tree_k, "tree_v": tree_v, "depth": depth,
            "tap_logits": tap_logits}


def argmax_first(logits: np.ndarray) -> np.ndarray:
    """Greedy token per row: the smallest index attaining the maximum."""
    return np.argmax(logits, axis=-1).astype(np.int64)


# ----------------------------------------------------------------------------
# verification and acceptance (Section 3: exact matching)


def accept(parent: Sequence[int], ids: Sequence[int], pred: Sequence[int], vocab: int):
    """Exact-matching verification and acceptance.

    A candidate is verified when its token equals the greedy prediction at its
    parent and its parent is verified (the root always is).  Prompt nodes are
    never verified.  The accepted path is the deepest verified node's root
    path (ties: smallest node index).  Tokens emitted this step are the
    accepted candidates plus the bonus token pred[best]: n_path of them, so a
    root-only tree emits exactly one token, as vanilla decoding does.

    Returns (path root-first, n_path, next_tok)."""
    T = len(parent)
    depth, _ = build_mask(parent)
    ok = np.zeros(T, bool)
    ok[0] = True
    for i in range(1, T):
        p = int(parent[i])
        ok[i] = ok[p] and 0 <= int(ids[i]) < vocab and int(ids[i]) == int(pred[p])
    best = 0
    for i in range(1, T):
        if ok[i] and depth[i] > depth[best]:
            best = i
    path = []
    j = best
    while j != -1:
        path.append(j)
        j = int(parent[j])
    path = path[::-1]
    return np.asarray(path, np.int64), len(path), int(pred[best])


def kv_compact(k_cache: List[np.ndarray], v_cache: List[np.ndarray], tree_k, tree_v,
               L: int, path: Sequence[int]):
    """Commit the accepted nodes' keys/values: cache[L + k] = tree[path[k]].

    Prompt-token keys/values are never committed: one shared cache (Section
    5.3).  Returns the new cache length L + len(path)."""
    for l in range(len(k_cache)):
        for kk, node in enumerate(path):
            k_cache[l][:, L + kk, :] = tree_k[l][:, node, :]
            v_cache[l][:, L + kk, :] = tree_v[l][:, node, :]
    return L + len(path)


# ----------------------------------------------------------------------------
# plain causal decoding (the reference behaviour the tree step must reproduce)


def decode_token(model: Model, k_cache: List[np.ndarray], v_cache: List[np.ndarray],
                 L: int, token: int, store: Optional[str]) -> np.ndarray:
    """Ordinary one-token decode at position L with a growing KV cache.

    Appends the token's keys/values at position L of every layer (caches must
    have room) and returns its logits.  No tree, no mask: the token sees
    positions [0, L] only."""
    sh = model.shape
    nh, nkv, d = sh.n_heads, sh.n_kv_heads, sh.head_dim
    grp = nh // nkv
    cos, sin = rope_tables(np.array([L]), d, sh.rope_base)
    x = embed(model, [token])
    for l in range(sh.n_layers):
        lay = model.layer(l)
        a, r = normed_rows(x, lay["attn_norm"], sh.rms_eps, store)
        qkv = r[:, None] * (a @ lay["w_qkv"].T)
        q = round_act(apply_rope(qkv[:, :nh * d].reshape(1, nh, d), cos, sin), store)
        k = round_store(apply_rope(qkv[:, nh * d:(nh + nkv) * d].reshape(1, nkv, d), cos, sin), store)
        v = round_store(qkv[:, (nh + nkv) * d:].reshape(1, nkv, d), store)
        k_cache[l][:, L, :] = k[0]
        v_cache[l][:, L, :] = v[0]
        o = np.zeros((nh, d))
        for h in range(nh):
            kh = k_cache[l][h // grp][:L + 1]
            vh = v_cache[l][h // grp][:L + 1]
            s = kh @ q[0, h] / np.sqrt(d)
            p = np.exp(s - s.max())
            o[h] = (p / p.sum()) @ vh
        o = round_act(o.reshape(1, nh * d), store)
        x = x + o @ lay["w_o"].T
        a, r = normed_rows(x, lay["mlp_norm"], sh.rms_eps, store)
        gu = r[:, None] * (a @ lay["w_gate_up"].T)
        act = round_act(silu(gu[:, :sh.ffn]) * gu[:, sh.ffn:], store)
        x = x + act @ lay["w_down"].T
    a, r = normed_rows(x, model.final_norm, sh.rms_eps, store)
    return (r[:, None] * (a @ model.lm_head.T))[0]


def new_cache(model: Model, capacity: int):
    sh = model.shape
    k = [np.zeros((sh.n_kv_heads, capacity, sh.head_dim)) for _ in range(sh.n_layers)]
    v = [np.zeros((sh.n_kv_heads, capacity, sh.head_dim)) for _ in range(sh.n_layers)]
    return k, v


def copy_cache(k_cache, v_cache):
    return [a.copy() for a in k_cache], [a.copy() for a in v_cache]


def causal_logits(model: Model, k_cache, v_cache, L: int, tokens: Sequence[int],
                  store: Optional[str]) -> np.ndarray:
    """Logits after each of `tokens` fed one by one at positions L, L+1, ...

    Works on copies, so the given caches are unchanged (brute-force check of
    one tree path)."""
    kc, vc = copy_cache(k_cache, v_cache)
    out = []
    for j, t in enumerate(tokens):
        out.append(decode_token(model, kc, vc, L + j, t, store))
    return np.stack(out)


def prefill(model: Model, tokens: Sequence[int], capacity: int, store: Optional[str]):
    """KV cache of a prompt, built by plain one-token decoding."""
    kc, vc = new_cache(model, capacity)
    last = None
    for j, t in enumerate(tokens):
        last = decode_token(model, kc, vc, j, t, store)
    return kc, vc, last


def greedy_decode(model: Model, k_cache, v_cache, L: int, first_token: int, n: int,
                  store: Optional[str]) -> List[int]:
    """Vanilla greedy continuation: feed first_token at L, then n-1 more tokens.

    Returns the n tokens emitted after first_token (works on copies)."""
    kc, vc = copy_cache(k_cache, v_cache)
    out, tok = [], int(first_token)
    for j in range(n):
        logits = decode_token(model, kc, vc, L + j, tok, store)
        tok = int(np.argmax(logits))
        out.append(tok)
    return out


def path_tokens(parent: Sequence[int], ids: Sequence[int], node: int) -> List[int]:
    """Token ids on the root-to-node path, root first."""
    seq = []
    j = int(node)
    while j != -1:
        seq.append(int(ids[j]))
        j = int(parent[j])
    return seq[::-1]


# ----------------------------------------------------------------------------
# candidate generation for the next step (Section 3, step (1); Section 3.1;
# Section 4 and the tree-construction appendix)
#
# The next step's tree is a fixed sparse-tree template whose token ids are
# filled from this step's outputs: its root is the bonus token (the accepted
# node's greedy token) and a candidate at depth d with rank r takes the r-th
# best token of the logits of the d-th prompt token attached to the accepted
# node -- that prompt token stands d positions past the accepted node, i.e.
# at the position of the bonus token's (d-1)-th successor, so its output
# predicts the token at depth d of the next tree (Section 3.1).  Prompt nodes
# of the template carry fixed prompt ids.
#
# Ensemble prompt tokens (Section 3.2; the EPT appendix on masks and
# aggregation): with n_ept EPTs per prompt token, the EPTs form n_ept
# disjoint groups, and an EPT of group g sees, besides the input tokens, only
# the EPTs of group g at earlier positions.  In a tree that is n_ept parallel
# prompt chains under a node, chain g holding the group-g EPTs of token
# distances 1, 2, ...; the ancestor mask is then exactly the ensemble mask.
# The EPT of token distance j (1-based) in group g is prompt embedding
# (j - 1) * n_ept + g.  The guess for a token distance averages the logits of
# its n_ept EPTs (the text's "averaging the logits"; the printed formula
# averages probabilities -- the text's reading is taken).

TOPK_MAX = 16  # largest rank + 1 a template may use per depth


def ept_prompt_id(j: int, g: int, n_ept: int) -> int:
    """Prompt embedding of the EPT of group g at token distance j + 1."""
    return j * n_ept + g


def prompt_chain(parent: Sequence[int], ids: Sequence[int], vocab: int, node: int,
                 n_ept: int = 1, group: int = 0) -> List[int]:
    """The prompt tokens of EPT group `group` attached to `node`: p_1 is its
    child with prompt id ept_prompt_id(0, group), p_j the child of p_{j-1}
    with prompt id ept_prompt_id(j - 1, group) (with one EPT: prompt id j - 1).
    Returns [p_1, p_2, ...] (empty if the node carries none); the first such
    child is taken if several match."""
    T = len(parent)
    chain = []
    cur = int(node)
    while True:
        want = vocab + ept_prompt_id(len(chain), group, n_ept)
        nxt = -1
        for i in range(T):
            if int(parent[i]) == cur and int(ids[i]) == want:
                nxt = i
                break
        if nxt < 0:
            return chain
        chain.append(nxt)
        cur = nxt


def ept_mean_row(rows: Sequence[np.ndarray]) -> np.ndarray:
    """Average of the EPT groups' logits rows, in float32 as the logits are
    stored: the rows added in group order, then divided by their count (a
    single row is returned unchanged).  The ranks taken from it are integer
    decisions, so both implementations take them on this same float32
    value."""
    acc = np.asarray(rows[0], np.float32).copy()
    for r in rows[1:]:
        acc = (acc + np.asarray(r, np.float32)).astype(np.float32)
    if len(rows) > 1:
        acc = (acc / np.float32(len(rows))).astype(np.float32)
    return acc


def rank_order(row: np.ndarray) -> np.ndarray:
    """Vocabulary indices of one logits row from best to worst: larger value
    first, equal values by smaller index; NaN ranks below every number."""
    v = np.asarray(row, np.float64)
    key = np.where(np.isnan(v), -np.inf, v)
    nan_last = np.isnan(v).astype(np.int64)
    # lexsort sorts by the last key first
    return np.lexsort((np.arange(v.shape[0]), -key, nan_last)).astype(np.int64)


def template_depths(tpl_parent: Sequence[int]) -> np.ndarray:
    depth, _ = build_mask(tpl_parent)
    return depth


def validate_template(tpl_parent: Sequence[int], tpl_kind: Sequence[int], n_prompt: int,
                      n_ept: int = 1) -> None:
    """A template is a topological tree (tpl_parent) with a kind per node:
    kind >= 0 is a candidate of that rank (< TOPK_MAX) whose parent is the root
    or a candidate; kind < 0 is prompt embedding q = -kind - 1, the EPT of
    group q mod n_ept at token distance q // n_ept + 1 (< n_prompt token
    distances), attached to a candidate (token distance 1) or to the same
    group's EPT one token distance lower.  Node 0 is the root (its kind is
    ignored)."""
    validate_tree(tpl_parent)
    T = len(tpl_parent)
    for i in range(1, T):
        k, p = int(tpl_kind[i]), int(tpl_parent[i])
        pk = int(tpl_kind[p]) if p > 0 else 0
        if k >= 0:
            if k >= TOPK_MAX or (p > 0 and pk < 0):
                raise ValueError(f"template node {i}: bad candidate")
        else:
            j, g = divmod(-k - 1, n_ept)
            if j >= n_prompt:
                raise ValueError(f"template node {i}: token distance {j + 1} > {n_prompt}")
            if j == 0:
                if p > 0 and pk < 0:
                    raise ValueError(f"template node {i}: prompt chain out of order")
            elif p == 0 or pk != -1 - ept_prompt_id(j - 1, g, n_ept):
                raise ValueError(f"template node {i}: prompt chain out of order")


def next_tree_ids(parent: Sequence[int], ids: Sequence[int], vocab: int, path: Sequence[int],
                  next_tok: int, logits: np.ndarray, tpl_parent: Sequence[int],
                  tpl_kind: Sequence[int], n_ept: int = 1) -> np.ndarray:
    """Token ids of the next step's tree (template tpl_parent / tpl_kind).

    Root: next_tok, the bonus token.  Candidate at template depth d with rank
    r: rank_order(row)[r], where row is the logits of the accepted node's d-th
    prompt token -- with n_ept > 1, ept_mean_row over the d-th EPT of every
    group's chain.  For d beyond a chain, that chain's deepest node (or the
    accepted node itself when it carries none) -- a reading of this build:
    the template stays fixed, and exact-match verification keeps the output
    lossless whatever the guesses.  Prompt nodes: vocab + prompt id."""
    a = int(path[-1])
    chains = [prompt_chain(parent, ids, vocab, a, n_ept, g) for g in range(n_ept)]
    depth = template_depths(tpl_parent)
    T = len(tpl_parent)
    out = np.zeros(T, np.int64)
    out[0] = int(next_tok)
    order_of = {}
    for i in range(1, T):
        k = int(tpl_kind[i])
        if k < 0:
            out[i] = vocab + (-k - 1)
            continue
        d = int(depth[i])
        srcs = tuple(ch[d - 1] if d <= len(ch) else (ch[-1] if ch else a) for ch in chains)
        if srcs not in order_of:
            row = logits[srcs[0]] if n_ept == 1 else ept_mean_row([logits[s] for s in srcs])
            order_of[srcs] = rank_order(row)
        out[i] = int(order_of[srcs][k])
    return out


# ----------------------------------------------------------------------------
# tree sizing (Section 4.2, hardware-aware tree size; Proposition 1 of the
# tree-construction appendix)
#
# Proposition 1: with an acceptance probability per tree position, the
# expected number of accepted candidates of a tree is the sum over its
# candidates of the product of the probabilities along the candidate's root
# path.  Here a candidate at depth d with rank r (the r-th best guess at that
# distance) is accepted, given its parent is, with probability p[d - 1][r],
# independently of other depths.  The tree of n candidates that maximises
# that sum takes the n rank paths of largest product (every product is at
# most its prefix's, so those paths contain their prefixes).  The hardware-
# aware size is then the n that maximises tokens per step over forward
# latency, Speedup(n) = tau(n) / L_fp(n), with tau(n) = 1 + the expected
# accepted candidates (the bonus token always comes).


def prop1_expected_accepted(tpl_parent: Sequence[int], tpl_kind: Sequence[int],
                            p_table) -> float:
    """Proposition 1's sum for a template: candidates (kind >= 0) at depth d,
    rank r contribute the product of p[depth - 1][rank] along their path."""
    depth = template_depths(tpl_parent)
    val = {0: 1.0}
    total = 0.0
    for i in range(1, len(tpl_parent)):
        k = int(tpl_kind[i])
        if k < 0:
            continue
        val[i] = val[int(tpl_parent[i])] * float(p_table[int(depth[i]) - 1][k])
        total += val[i]
    return total


def best_candidate_paths(p_table, n_cand: int) -> List[Tuple[int, ...]]:
    """The n_cand rank paths (depth <= len(p_table), ranks < len(p_table[0]))
    of largest product, in order: larger product first, then shallower, then
    the lexicographically smaller path.  Found by listing every path."""
    import itertools
    D, K = len(p_table), len(p_table[0])
    scored = []
    for d in range(1, D + 1):
        for path in itertools.product(range(K), repeat=d):
            v = 1.0
            for j, r in enumerate(path):
                v *= float(p_table[j][r])
            scored.append((-v, d, path))
    scored.sort()
    return [s[2] for s in scored[:n_cand]]


def sparse_template(p_table, n_cand: int, n_prompt: int, n_ept: int = 1):
    """Template of the best n_cand candidates: root, the candidates in the
    order of best_candidate_paths, then under the root and every candidate,
    in node order, one chain of n_prompt prompt tokens per EPT group.
    Returns (tpl_parent, tpl_kind, expected accepted candidates)."""
    paths = best_candidate_paths(p_table, n_cand)
    parent, kind = [-1], [0]
    node_of = {(): 0}
    for path in paths:
        parent.append(node_of[path[:-1]])
        kind.append(path[-1])
        node_of[path] = len(parent) - 1
    for c in range(len(parent)):
        for g in range(n_ept):
            prev = c
            for j in range(n_prompt):
                parent.append(prev)
                kind.append(-1 - ept_prompt_id(j, g, n_ept))
                prev = len(parent) - 1
    return (np.asarray(parent, np.int64), np.asarray(kind, np.int64),
            prop1_expected_accepted(parent, kind, p_table))
