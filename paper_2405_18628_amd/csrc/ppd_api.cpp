// Host side of libppd: argument validation, workspace layout and the launch
// sequence of the verification step.  Everything is enqueued on the caller's
// stream; nothing is allocated, copied or synchronised (except in
// ppd_device_status, which is documented as synchronous).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>

#include "ppd_internal.h"

namespace {

thread_local std::string g_err;

// optional per-thread kernel timer (ppd_set_kernel_timer)
struct KernelTimer {
  int kind = -1;
  void *const *start = nullptr;
  void *const *stop = nullptr;
  int n = 0;
  int next = 0;  // launches of `kind` seen in the current step
};
thread_local KernelTimer g_timer;

enum TimedKind { TK_QKV = 0, TK_ATTN = 1, TK_O = 2, TK_GATEUP = 3, TK_DOWN = 4, TK_LM = 5, TK_NEXT = 6 };

// Events of the next timed launch of `kind` (both null when not timed).  The
// kernel is then launched with hipExtLaunchKernelGGL, which records them at
// the dispatch's own start and end, so they measure the kernel alone.
void timer_events(int kind, void **start, void **stop) {
  *start = *stop = nullptr;
  if (g_timer.kind != kind || g_timer.next >= g_timer.n) return;
  *start = g_timer.start[g_timer.next];
  *stop = g_timer.stop[g_timer.next];
  ++g_timer.next;
}

ppd_status fail(ppd_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

}  // namespace

// the same for the library's other translation units
ppd_status ppd_fail(ppd_status s, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

namespace {

#define PPD_TRY_HIP(call)                                                               \
  do {                                                                                  \
    hipError_t e_ = (call);                                                             \
    if (e_ != hipSuccess) return fail(PPD_EDEVICE, "%s: %s", #call, hipGetErrorString(e_)); \
  } while (0)

constexpr int kCUs = 256;          // MI355X compute units
constexpr size_t kAlign = 256;
constexpr size_t kMaxPackedBytes = 0x7ffffff0u;  // one buffer resource per packed weight

size_t align_up(size_t v) { return (v + kAlign - 1) & ~(kAlign - 1); }
int t_pad_of(int T) { return (T + 15) & ~15; }

ppd_status pack_args(int kind, int rows, int cols, int *gk, int *N);

ppd_status check_model(const ppd_model *m) {
  if (!m) return fail(PPD_EINVAL, "model is NULL");
  if (m->n_layers < 1 || m->hidden < 1 || m->n_heads < 1 || m->n_kv_heads < 1 ||
      m->head_dim < 2 || m->ffn < 1 || m->vocab < 1 || m->n_prompt < 0)
    return fail(PPD_EINVAL, "model sizes must be positive");
  if (m->n_heads % m->n_kv_heads) return fail(PPD_EINVAL, "n_kv_heads must divide n_heads");
  if (m->head_dim % 2 || m->head_dim > 128)
    return fail(PPD_EUNSUPPORTED, "head_dim must be even and <= 128");
  if (!(m->rms_eps >= 0.f) || !(m->rope_base > 0.f))
    return fail(PPD_EINVAL, "rms_eps must be >= 0 and rope_base > 0");
  if (m->dtype != PPD_F32 && m->dtype != PPD_BF16) return fail(PPD_EINVAL, "unknown dtype");
  if (m->dtype == PPD_BF16) {
    if (m->head_dim != 128) return fail(PPD_EUNSUPPORTED, "bf16 kernels need head_dim 128");
    if (m->hidden % 128) return fail(PPD_EUNSUPPORTED, "bf16 kernels need hidden %% 128 == 0");
    if (m->ffn % 64) return fail(PPD_EUNSUPPORTED, "bf16 kernels need ffn %% 64 == 0");
    const int shapes[5][3] = {{PPD_W_QKV, (m->n_heads + 2 * m->n_kv_heads) * 128, m->hidden},
                              {PPD_W_O, m->hidden, m->n_heads * 128},
                              {PPD_W_GATE_UP, 2 * m->ffn, m->hidden},
                              {PPD_W_DOWN, m->hidden, m->ffn},
                              {PPD_W_LM_HEAD, m->vocab, m->hidden}};
    for (const auto &w : shapes) {
      int gk, N;
      const ppd_status st = pack_args(w[0], w[1], w[2], &gk, &N);
      if (st != PPD_OK) return st;
    }
  }
  if (!m->tok_emb || !m->lm_head || !m->final_norm || (m->n_prompt > 0 && !m->prompt_emb))
    return fail(PPD_EINVAL, "embedding, LM head and final norm pointers must be set");
  const void *const *arrs[6] = {m->attn_norm, m->w_qkv, m->w_o, m->mlp_norm, m->w_gate_up,
                                m->w_down};
  for (int a = 0; a < 6; ++a) {
    if (!arrs[a]) return fail(PPD_EINVAL, "per-layer pointer array %d is NULL", a);
    for (int l = 0; l < m->n_layers; ++l)
      if (!arrs[a][l]) return fail(PPD_EINVAL, "per-layer pointer %d of layer %d is NULL", a, l);
  }
  return PPD_OK;
}

int qkv_rows(const ppd_model *m) { return (m->n_heads + 2 * m->n_kv_heads) * m->head_dim; }

// ---- launch shapes (also used to size the workspace)

// Compute units of the current device (one workgroup per compute unit; the
// XCD-local tile finish needs the MI355X layout of 8 XCDs x 32 CUs with
// round-robin dispatch, else every tile is finished whole, without waits).
int device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return n;
}

struct GemmShape {
  int kind, N, K;
};

// Partition of one GEMM for MT token tiles (see GemmLaunch): for each
// candidate number s of K slices (the XCD's 32 workgroups then take 32 / s
// tiles of h groups), a model of the slowest workgroup's time, taken from
// measurements on MI355X: its weight bytes plus 0.4 x its fp32 activation
// bytes (L2 hits, read while the weights stream) at a compute unit's ~35
// GB/s, or its matrix-core time at 70 % of peak if larger; with s > 1 a
// tail that does not overlap the stream -- ~1.5 us of hand-off plus writing
// and reading its partial sums at ~25 GB/s.  The cheapest is taken.  Groups
// per wave come from the instantiated set {1, 2, 3, 4, 6} (bounded by the
// registers).
struct GemmPlan {
  int gw = 1, TX = 32, s = 1;
  int xg0[9] = {0};
};

GemmPlan plan_gemm(const GemmShape &sh, int MT, bool xcd_sync) {
  GemmPlan best;
  const int G = gemm_groups_of(sh.kind, sh.N), S = gemm_sub_of(sh.kind), kc = sh.K / 64;
  for (int x = 0; x <= 8; ++x) best.xg0[x] = (int)((long)G * x / 8);
  const int nx = (G + 7) / 8;
  const int gmax = gemm_gw_max(sh.kind, MT);
  double best_t = 1e30;
  for (int s = 1; s <= 16; s *= 2) {
    if (s > kc || (s > 1 && !xcd_sync)) break;
    const int TX = 32 / s;
    const int h = std::max(1, (nx + TX - 1) / TX);
    int gw = (h + 3) / 4;
    if (gw == 5) gw = 6;
    if (gw > gmax) continue;
    const double kch = (double)((kc + s - 1) / s);
    const double wb = (double)h * 16 * S * kch * 64 * 2;
    const double ab = (double)MT * 16 * kch * 64 * 4;
    const double pb = (double)h * 16 * S * MT * 16 * 4;
    const double flops = 4.0 * MT * 16 * h * 16 * S * kch * 64;
    const double t = std::max((wb + 0.4 * ab) / 35e9, flops / (0.7 * 2.5e15 / 256)) +
                     (s > 1 ? 1.5e-6 + 2 * pb / 25e9 : 0.0);
    if (t < best_t) {
      best_t = t;
      best.gw = gw;
      best.TX = TX;
      best.s = s;
    }
  }
  return best;
}

enum { SH_QKV = 0, SH_O = 1, SH_GATE_UP = 2, SH_DOWN = 3, SH_LM = 4 };

void gemm_shapes(const ppd_model *m, GemmShape out[5]) {
  out[SH_QKV] = {GEMM_QKV, qkv_rows(m), m->hidden};
  out[SH_O] = {GEMM_RESID, m->hidden, m->n_heads * 128};
  out[SH_GATE_UP] = {GEMM_SWIGLU, m->ffn, m->hidden};
  out[SH_DOWN] = {GEMM_RESID, m->hidden, m->ffn};
  out[SH_LM] = {GEMM_LOGITS, m->vocab, m->hidden};
}

// bytes of the partial sums of a plan (0 when every tile is whole)
size_t plan_part_bytes(const GemmShape &sh, const GemmPlan &p, int MT) {
  if (p.s == 1) return 0;
  return (size_t)8 * p.TX * p.s * 4 * p.gw * gemm_sub_of(sh.kind) * MT * 64 * 16;
}

constexpr int kSpinLimit = 1 << 14;  // bounded wait of a tile's slices (~10-20 ms)

// Key splits of the attention: a workgroup per (head, split) reads each
// key/value block once, so the splits spread the cache over the compute
// units -- about one workgroup per CU, each keeping at least 4 of the
// 32-key blocks.
// key splits per head: nh x splits workgroups must fit one round on the CUs
// (one attention workgroup per CU), or the last ones run alone afterwards
int attn_max_splits(int nh) { return std::max(1, std::min(PPD_ATTN_MAX_SPLITS, kCUs / nh)); }

void attn_splits(const ppd_model *m, int L, int T, int *splits, int *chunk) {
  const int nblk = (L + T + 31) / 32;
  const int ks = std::max(1, std::min(attn_max_splits(m->n_heads), nblk / 4));
  const int c = ((nblk + ks - 1) / ks + 1) & ~1;  // even: splits start on 64-key pairs
  *splits = (nblk + c - 1) / c;
  *chunk = c;
}

// One sequence on 256 CUs: the heads are dealt to the 8 XCDs (at most
// ceil(nh / 8) per XCD) and each head's splits take that XCD's 32 CUs
// together (they merge through its L2), so a head gets up to
// 32 / ceil(nh / 8) splits.  Returns the workgroup count (8 x heads per XCD
// x splits).
int attn_splits_xcd(const ppd_model *m, int L, int T, int *splits, int *chunk) {
  const int nblk = (L + T + 31) / 32, hpx = (m->n_heads + 7) / 8;
  const int ks = std::max(1, std::min(std::min(PPD_ATTN_MAX_SPLITS, 32 / hpx), nblk / 4));
  const int c = ((nblk + ks - 1) / ks + 1) & ~1;  // even: splits start on 64-key pairs
  *splits = (nblk + c - 1) / c;
  *chunk = c;
  return 8 * hpx * *splits;
}

WsLayout layout_of(const ppd_model *m, int T) {
  WsLayout w{};
  const int Tp = t_pad_of(T);
  const bool bf16 = m->dtype == PPD_BF16;
  const int H = m->hidden, F = m->ffn, nh = m->n_heads, d = m->head_dim;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  w.status = take(16);
  w.x = take(sizeof(float) * Tp * H);
  // activations are fp32 on both paths; the fp32 path also keeps x * gain
  // and the row scales (the bf16 GEMMs form x * gain while staging)
  w.xg = take(bf16 ? 0 : sizeof(float) * (Tp * H + Tp));
  w.max_ss = 1;
  w.max_amax_tiles = 1;
  size_t part = 0;
  if (bf16) {
    GemmShape gs[5];
    gemm_shapes(m, gs);
    const bool sync = device_cus() == 256;
    for (int mt = 1; mt <= Tp / 16; ++mt)
      for (int i = 0; i < 5; ++i) {
        const GemmPlan p = plan_gemm(gs[i], mt, sync);
        part = std::max(part, plan_part_bytes(gs[i], p, mt));
        if (gs[i].kind == GEMM_RESID) w.max_ss = std::max(w.max_ss, 8 * p.TX);
        if (gs[i].kind == GEMM_LOGITS) w.max_amax_tiles = std::max(w.max_amax_tiles, 8 * p.TX);
      }
  }
  w.ss = take(sizeof(float) * w.max_ss * Tp);
  w.q = take(sizeof(float) * Tp * nh * d);
  w.attn_o = take(sizeof(float) * Tp * nh * d);
  w.act = take(sizeof(float) * Tp * F);
  if (!bf16) {
    const size_t wide = std::max({(size_t)qkv_rows(m), (size_t)2 * F, (size_t)H, (size_t)m->vocab});
    w.tmp = take(sizeof(float) * Tp * wide);
  } else {
    w.tmp = take(0);
  }
  w.max_splits = bf16 ? attn_max_splits(nh) : 0;
  w.attn_part = take(sizeof(float) * (size_t)nh * w.max_splits * Tp * PPD_ATTN_OROW);
  w.max_part_floats = part / sizeof(float);
  w.gemm_part = take(part);
  w.amax = take(sizeof(float2) * w.max_amax_tiles * Tp);
  w.rope = take(sizeof(float2) * Tp * (d / 2));
  // counters: one 1 KB block (8 XCDs x one 128-byte line) per GEMM launch
  // (tiles) and per attention launch (heads)
  w.n_ctr = bf16 ? (size_t)(5 * m->n_layers + 1) * 256 : 0;
  w.ctr = take(sizeof(uint32_t) * w.n_ctr);
  w.total = off;
  return w;
}

template <typename P>
P *at(void *ws, size_t off) {
  return (P *)((char *)ws + off);
}

ppd_status check_kv(const ppd_model *m, const ppd_kv *kv) {
  if (!kv || !kv->k || !kv->v) return fail(PPD_EINVAL, "kv cache pointers must be set");
  if (kv->capacity < 1) return fail(PPD_EINVAL, "kv capacity must be positive");
  if (m->dtype == PPD_BF16 && kv->capacity % 8)
    return fail(PPD_EUNSUPPORTED, "bf16 caches need capacity %% 8 == 0");
  if (kv->capacity > PPD_CAPACITY_MAX)  // per-head offsets are 32-bit in the kernels
    return fail(PPD_EUNSUPPORTED, "capacity %d > %d", kv->capacity, PPD_CAPACITY_MAX);
  return PPD_OK;
}

// the sequences of a step, with this layer's cache slices
SeqBatch seq_batch(const ppd_model *m, int B, const ppd_kv *kvs, const int32_t *Ls,
                   const int32_t *Ts, int layer) {
  SeqBatch sb{};
  sb.B = B;
  for (int j = 0; j < B; ++j) {
    sb.t0[j + 1] = sb.t0[j] + Ts[j];
    sb.L[j] = Ls[j];
    sb.cap[j] = kvs[j].capacity;
    const size_t per_layer = (size_t)m->n_kv_heads * kvs[j].capacity * m->head_dim;
    sb.k[j] = (bf16_t *)kvs[j].k + (size_t)layer * per_layer;
    sb.v[j] = (bf16_t *)kvs[j].v + (size_t)layer * per_layer;
  }
  return sb;
}

ppd_status step_bf16(const ppd_model *m, int B, const ppd_kv *kvs, const int32_t *Ls,
                     const int32_t *Ts, const int32_t *ids, const int32_t *depth,
                     const uint64_t *mask, void *ws, const WsLayout &w, float *logits,
                     int32_t *pred, hipStream_t s) {
  const int H = m->hidden, nh = m->n_heads, nkv = m->n_kv_heads;
  int T = 0, MT_seq = 1;
  for (int j = 0; j < B; ++j) {
    T += Ts[j];
    MT_seq = std::max(MT_seq, (Ts[j] + 15) / 16);
  }
  const int Tp = t_pad_of(T), MT = Tp / 16;
  uint32_t *status = at<uint32_t>(ws, w.status);
  float *x = at<float>(ws, w.x);
  float *ss = at<float>(ws, w.ss);
  float *q = at<float>(ws, w.q);
  float *attn_o = at<float>(ws, w.attn_o);
  float *act = at<float>(ws, w.act);
  float *part = at<float>(ws, w.gemm_part);
  float2 *amax = at<float2>(ws, w.amax);
  float2 *rope = at<float2>(ws, w.rope);
  uint32_t *ctr = at<uint32_t>(ws, w.ctr);
  GemmShape gs[5];
  gemm_shapes(m, gs);
  const bool sync = device_cus() == 256;
  GemmPlan plan[5];
  for (int i = 0; i < 5; ++i) plan[i] = plan_gemm(gs[i], MT, sync);
  int launch = 0;  // GEMM launches of this step: counter block `launch`
  auto setup = [&](GemmLaunch &g, int i) {
    g.kind = gs[i].kind;
    g.N = gs[i].N;
    g.K = gs[i].K;
    g.kc = gs[i].K / 64;
    g.gw = plan[i].gw;
    g.TX = plan[i].TX;
    g.s = plan[i].s;
    for (int xx = 0; xx <= 8; ++xx) g.xg0[xx] = plan[i].xg0[xx];
    g.ctr = ctr + (size_t)launch++ * 256;
  };

  // embedding, its sum of squares (one partial per row), rotary table,
  // zeroed counters
  PPD_TRY_HIP(launch_embed(PPD_BF16, m->tok_emb, m->prompt_emb, ids, depth,
                           seq_batch(m, B, kvs, Ls, Ts, 0), m->head_dim, m->rope_base, rope,
                           m->vocab, m->n_prompt, H, x, ss, ctr, w.n_ctr, status, s));
  int n_ss = 1;
  // attention work per sequence: nh x splits workgroups
  // (one sequence on 256 CUs: heads dealt to the XCDs, splits merged in the
  // kernel; a batch: a merge kernel)
  int splits[PPD_BATCH_MAX], chunk[PPD_BATCH_MAX], wg0[PPD_BATCH_MAX + 1] = {0};
  const bool xcd_merge = B == 1 && sync && nh <= 256;
  uint32_t *attn_ctr = ctr + (size_t)(4 * m->n_layers + 1) * 256;
  if (xcd_merge) {
    wg0[1] = attn_splits_xcd(m, Ls[0], Ts[0], &splits[0], &chunk[0]);
  } else {
    for (int j = 0; j < B; ++j) {
      attn_splits(m, Ls[j], Ts[j], &splits[j], &chunk[j]);
      wg0[j + 1] = wg0[j] + nh * splits[j];
    }
  }
  const float inv_h = 1.0f / (float)H;

  for (int l = 0; l < m->n_layers; ++l) {
    const SeqBatch sb = seq_batch(m, B, kvs, Ls, Ts, l);
    GemmLaunch g{};
    g.T = T;
    g.MT = MT;
    g.part = part;
    g.inv_h = inv_h;
    g.eps = m->rms_eps;
    g.status = status;
    g.spin_limit = kSpinLimit;
    // QKV + RoPE + cache stores; A = x * attn_norm
    GemmLaunch qg = g;
    setup(qg, SH_QKV);
    qg.W = (const bf16_t *)m->w_qkv[l];
    qg.A = x;
    qg.gain = (const bf16_t *)m->attn_norm[l];
    qg.ss = ss;
    qg.n_ss = n_ss;
    qg.rope = rope;
    qg.q = q;
    qg.nh = nh;
    qg.nkv = nkv;
    qg.sb = sb;
    timer_events(TK_QKV, &qg.ev_start, &qg.ev_stop);
    PPD_TRY_HIP(launch_gemm_bf16(qg, s));
    // tree attention
    AttnLaunch a{};
    a.q = q;
    a.mask = mask;
    a.out = attn_o;
    a.part = at<float>(ws, w.attn_part);
    a.zeros = (const bf16_t *)((const char *)ws + PPD_WS_ZEROS);
    a.T_pad = Tp;
    a.nh = nh;
    a.nkv = nkv;
    a.max_splits = w.max_splits;
    a.MT = MT_seq;
    a.sb = sb;
    for (int j = 0; j < B; ++j) {
      a.splits[j] = splits[j];
      a.chunk[j] = chunk[j];
    }
    for (int j = 0; j <= B; ++j) a.wg0[j] = wg0[j];
    a.xcd_merge = xcd_merge;
    a.ctr = attn_ctr + (size_t)l * 256;
    a.spin_limit = kSpinLimit;
    a.status = status;
    a.scale_log2 = (float)(1.4426950408889634 / std::sqrt(128.0));
    timer_events(TK_ATTN, &a.ev_start, &a.ev_stop);
    PPD_TRY_HIP(launch_attn_bf16(a, s));
    // O projection + residual; sums of squares for the MLP norm
    GemmLaunch o = g;
    setup(o, SH_O);
    o.W = (const bf16_t *)m->w_o[l];
    o.A = attn_o;
    o.x = x;
    o.ss_out = ss;
    timer_events(TK_O, &o.ev_start, &o.ev_stop);
    PPD_TRY_HIP(launch_gemm_bf16(o, s));
    n_ss = 8 * plan[SH_O].TX;
    // gate/up + SwiGLU; A = x * mlp_norm
    GemmLaunch u = g;
    setup(u, SH_GATE_UP);
    u.W = (const bf16_t *)m->w_gate_up[l];
    u.A = x;
    u.gain = (const bf16_t *)m->mlp_norm[l];
    u.ss = ss;
    u.n_ss = n_ss;
    u.act = act;
    timer_events(TK_GATEUP, &u.ev_start, &u.ev_stop);
    PPD_TRY_HIP(launch_gemm_bf16(u, s));
    // down projection + residual; sums of squares for the next norm
    GemmLaunch dn = g;
    setup(dn, SH_DOWN);
    dn.W = (const bf16_t *)m->w_down[l];
    dn.A = act;
    dn.x = x;
    dn.ss_out = ss;
    timer_events(TK_DOWN, &dn.ev_start, &dn.ev_stop);
    PPD_TRY_HIP(launch_gemm_bf16(dn, s));
    n_ss = 8 * plan[SH_DOWN].TX;
  }
  // final norm + LM head + greedy partials; A = x * final_norm
  GemmLaunch lm{};
  setup(lm, SH_LM);
  lm.W = (const bf16_t *)m->lm_head;
  lm.A = x;
  lm.gain = (const bf16_t *)m->final_norm;
  lm.T = T;
  lm.MT = MT;
  lm.part = part;
  lm.ss = ss;
  lm.n_ss = n_ss;
  lm.inv_h = inv_h;
  lm.eps = m->rms_eps;
  lm.logits = logits;
  lm.amax = amax;
  lm.status = status;
  lm.spin_limit = kSpinLimit;
  timer_events(TK_LM, &lm.ev_start, &lm.ev_stop);
  PPD_TRY_HIP(launch_gemm_bf16(lm, s));
  PPD_TRY_HIP(launch_argmax_final(amax, 8 * plan[SH_LM].TX, T, Tp, pred, status, s));
  return PPD_OK;
}

ppd_status step_f32(const ppd_model *m, const ppd_kv *kv, int L, int T, const int32_t *ids,
                    const int32_t *depth, const uint64_t *mask, void *ws, const WsLayout &w,
                    float *logits, int32_t *pred, hipStream_t s) {
  const int H = m->hidden, F = m->ffn, nh = m->n_heads, nkv = m->n_kv_heads, d = m->head_dim;
  const int Tp = t_pad_of(T);
  const int cap = kv->capacity;
  uint32_t *status = at<uint32_t>(ws, w.status);
  float *x = at<float>(ws, w.x);
  float *xg = at<float>(ws, w.xg);
  float *r = xg + (size_t)Tp * H;
  float *q = at<float>(ws, w.q);
  float *attn_o = at<float>(ws, w.attn_o);
  float *act = at<float>(ws, w.act);
  float *tmp = at<float>(ws, w.tmp);
  float2 *rope = at<float2>(ws, w.rope);

  SeqBatch one{};
  one.B = 1;
  one.t0[1] = T;
  one.L[0] = L;
  PPD_TRY_HIP(launch_embed(PPD_F32, m->tok_emb, m->prompt_emb, ids, depth, one, d, m->rope_base, rope,
                           m->vocab, m->n_prompt, H, x, nullptr, nullptr, 0, status, s));
  for (int l = 0; l < m->n_layers; ++l) {
    float *kc = (float *)kv->k + (size_t)l * nkv * cap * d;
    float *vc = (float *)kv->v + (size_t)l * nkv * d * cap;
    PPD_TRY_HIP(launch_f32_rownorm(x, (const float *)m->attn_norm[l], T, H, m->rms_eps, xg, s));
    PPD_TRY_HIP(launch_f32_matmul_scaled(xg, (const float *)m->w_qkv[l], T, qkv_rows(m), H, r,
                                         tmp, s));
    PPD_TRY_HIP(launch_f32_qkv_post(tmp, rope, T, nh, nkv, d, q, kc, vc, cap, L, s));
    PPD_TRY_HIP(launch_f32_attention(q, kc, vc, mask, T, L, cap, nh, nkv, d, attn_o, s));
    PPD_TRY_HIP(launch_f32_matmul(attn_o, (const float *)m->w_o[l], T, H, nh * d, tmp, s));
    PPD_TRY_HIP(launch_f32_add(x, tmp, T * H, s));
    PPD_TRY_HIP(launch_f32_rownorm(x, (const float *)m->mlp_norm[l], T, H, m->rms_eps, xg, s));
    PPD_TRY_HIP(launch_f32_matmul_scaled(xg, (const float *)m->w_gate_up[l], T, 2 * F, H, r, tmp,
                                         s));
    PPD_TRY_HIP(launch_f32_swiglu(tmp, T, F, act, s));
    PPD_TRY_HIP(launch_f32_matmul(act, (const float *)m->w_down[l], T, H, F, tmp, s));
    PPD_TRY_HIP(launch_f32_add(x, tmp, T * H, s));
  }
  PPD_TRY_HIP(launch_f32_rownorm(x, (const float *)m->final_norm, T, H, m->rms_eps, xg, s));
  float *lg = logits ? logits : tmp;
  PPD_TRY_HIP(launch_f32_matmul_scaled(xg, (const float *)m->lm_head, T, m->vocab, H, r, lg, s));
  PPD_TRY_HIP(launch_f32_argmax(lg, T, m->vocab, pred, status, s));
  return PPD_OK;
}

// GEMM kind and output-row count of a weight given as a row-major
// [rows][cols] matrix
ppd_status pack_args(int kind, int rows, int cols, int *gk, int *N) {
  if (rows < 1 || cols < 1) return fail(PPD_EINVAL, "weight sizes must be positive");
  if (cols % 64) return fail(PPD_EUNSUPPORTED, "packed weights need cols %% 64 == 0");
  switch (kind) {
    case PPD_W_QKV:
      if (rows % 128) return fail(PPD_EUNSUPPORTED, "w_qkv needs rows %% 128 == 0 (head_dim 128)");
      *gk = GEMM_QKV, *N = rows;
      break;
    case PPD_W_O:
    case PPD_W_DOWN:
      if (rows % 128) return fail(PPD_EUNSUPPORTED, "w_o / w_down need rows (hidden) %% 128 == 0");
      *gk = GEMM_RESID, *N = rows;
      break;
    case PPD_W_GATE_UP:
      if (rows % 128) return fail(PPD_EUNSUPPORTED, "w_gate_up needs rows (2 ffn) %% 128 == 0");
      *gk = GEMM_SWIGLU, *N = rows / 2;
      break;
    case PPD_W_LM_HEAD:
      *gk = GEMM_LOGITS, *N = rows;
      break;
    default:
      return fail(PPD_EINVAL, "unknown weight kind %d", kind);
  }
  // the GEMM reads a packed weight through one buffer resource: < 2 GB
  const size_t bytes = (size_t)gemm_groups_of(*gk, *N) * gemm_sub_of(*gk) * 16 * cols * sizeof(bf16_t);
  if (bytes > kMaxPackedBytes)
    return fail(PPD_EUNSUPPORTED, "a packed weight of %zu bytes exceeds %zu", bytes, kMaxPackedBytes);
  return PPD_OK;
}

}  // namespace

extern "C" {

size_t ppd_workspace_bytes(const ppd_model *model, int32_t t_max, int32_t max_len) {
  if (check_model(model) != PPD_OK) return 0;
  if (t_max < 1 || t_max > PPD_T_MAX || max_len < 0) {
    fail(PPD_EINVAL, "t_max must be in [1, %d] and max_len >= 0", PPD_T_MAX);
    return 0;
  }
  return layout_of(model, t_max).total;
}

ppd_status ppd_workspace_init(void *ws, size_t ws_bytes, void *stream) {
  const size_t need = align_up(16);  // status word and the line of zeros
  if (!ws || ws_bytes < need) return fail(PPD_EWORKSPACE, "workspace needs at least %zu bytes", need);
  PPD_TRY_HIP(launch_ws_init(ws, need / 4, (hipStream_t)stream));
  return PPD_OK;
}

ppd_status ppd_build_tree_mask(int32_t T, const int32_t *parent, int32_t *depth_out,
                               uint64_t *mask_out) {
  if (T < 1 || T > PPD_T_MAX) return fail(PPD_EINVAL, "T=%d outside [1, %d]", T, PPD_T_MAX);
  if (!parent || !depth_out || !mask_out) return fail(PPD_EINVAL, "NULL argument");
  if (parent[0] != -1) return fail(PPD_ETREE, "parent[0] must be -1 (root)");
  for (int i = 1; i < T; ++i)
    if (parent[i] < 0 || parent[i] >= i)
      return fail(PPD_ETREE, "parent[%d]=%d is not an earlier node", i, parent[i]);
  for (int i = 0; i < T; ++i) {
    uint64_t row[PPD_MASK_WORDS] = {0, 0};
    int dep = -1;
    for (int j = i; j != -1; j = parent[j]) {
      row[j >> 6] |= 1ull << (j & 63);
      ++dep;
    }
    depth_out[i] = dep;
    mask_out[i * PPD_MASK_WORDS + 0] = row[0];
    mask_out[i * PPD_MASK_WORDS + 1] = row[1];
  }
  return PPD_OK;
}

ppd_status ppd_verify_batch(const ppd_model *model, int32_t B, const ppd_kv *kvs,
                            const int32_t *L, const int32_t *T, const int32_t *ids,
                            const int32_t *depth, const uint64_t *mask, void *ws, size_t ws_bytes,
                            float *logits, int32_t *pred, void *stream) {
  ppd_status st = check_model(model);
  if (st != PPD_OK) return st;
  if (B < 1 || B > PPD_BATCH_MAX)
    return fail(PPD_EINVAL, "B=%d outside [1, %d]", B, PPD_BATCH_MAX);
  if (!kvs || !L || !T) return fail(PPD_EINVAL, "NULL sequence arrays");
  if (B > 1 && model->dtype != PPD_BF16)
    return fail(PPD_EUNSUPPORTED, "batched steps need a bf16 model");
  int64_t total = 0;
  for (int j = 0; j < B; ++j) {
    if ((st = check_kv(model, &kvs[j])) != PPD_OK) return st;
    if (T[j] < 1) return fail(PPD_EINVAL, "T[%d]=%d must be >= 1", j, T[j]);
    if (L[j] < 0) return fail(PPD_EINVAL, "L[%d] must be >= 0", j);
    if ((int64_t)L[j] + T[j] > kvs[j].capacity)
      return fail(PPD_ECAPACITY, "sequence %d: L + T = %lld exceeds capacity %d", j,
                  (long long)L[j] + T[j], kvs[j].capacity);
    total += T[j];
  }
  if (total > PPD_T_MAX)
    return fail(PPD_EINVAL, "%lld tree tokens in all > %d", (long long)total, PPD_T_MAX);
  if (!ids || !depth || !mask || !pred) return fail(PPD_EINVAL, "NULL tree or output pointer");
  const WsLayout w = layout_of(model, (int)total);
  if (!ws || ws_bytes < w.total)
    return fail(PPD_EWORKSPACE, "workspace of %zu bytes is smaller than the %zu required", ws_bytes,
                w.total);
  hipStream_t s = (hipStream_t)stream;
  g_timer.next = 0;
  if (model->dtype == PPD_BF16)
    return step_bf16(model, B, kvs, L, T, ids, depth, mask, ws, w, logits, pred, s);
  return step_f32(model, &kvs[0], L[0], T[0], ids, depth, mask, ws, w, logits, pred, s);
}

ppd_status ppd_verify_step(const ppd_model *model, const ppd_kv *kv, int32_t L, int32_t T,
                           const int32_t *ids, const int32_t *depth, const uint64_t *mask,
                           void *ws, size_t ws_bytes, float *logits, int32_t *pred,
                           void *stream) {
  if (!kv) return fail(PPD_EINVAL, "kv cache pointers must be set");
  if (T < 1 || T > PPD_T_MAX) return fail(PPD_EINVAL, "T=%d outside [1, %d]", T, PPD_T_MAX);
  return ppd_verify_batch(model, 1, kv, &L, &T, ids, depth, mask, ws, ws_bytes, logits, pred,
                          stream);
}

ppd_status ppd_accept(int32_t T, const int32_t *parent, const int32_t *ids, const int32_t *pred,
                      int32_t vocab, int32_t *path, int32_t *n_path, int32_t *next_tok, void *ws,
                      size_t ws_bytes, void *stream) {
  if (T < 1 || T > PPD_T_MAX) return fail(PPD_EINVAL, "T=%d outside [1, %d]", T, PPD_T_MAX);
  if (vocab < 1) return fail(PPD_EINVAL, "vocab must be positive");
  if (!parent || !ids || !pred || !path || !n_path || !next_tok)
    return fail(PPD_EINVAL, "NULL argument");
  if (!ws || ws_bytes < 16) return fail(PPD_EWORKSPACE, "workspace (status word) required");
  PPD_TRY_HIP(launch_accept(T, parent, ids, pred, vocab, path, n_path, next_tok, (uint32_t *)ws,
                            (hipStream_t)stream));
  return PPD_OK;
}

ppd_status ppd_kv_compact(const ppd_model *model, const ppd_kv *kv, int32_t L,
                          const int32_t *path, int32_t path_len, const int32_t *n_path,
                          void *stream) {
  ppd_status st = check_model(model);
  if (st != PPD_OK) return st;
  if ((st = check_kv(model, kv)) != PPD_OK) return st;
  if (L < 0 || L >= kv->capacity)
    return fail(PPD_ECAPACITY, "L=%d must be in [0, capacity=%d)", L, kv->capacity);
  if (!path || !n_path) return fail(PPD_EINVAL, "NULL path");
  if (path_len < 1 || path_len > PPD_T_MAX)
    return fail(PPD_EINVAL, "path_len=%d outside [1, %d]", path_len, PPD_T_MAX);
  PPD_TRY_HIP(launch_kv_compact(model->dtype, kv->k, kv->v, model->n_layers, model->n_kv_heads,
                                kv->capacity, model->head_dim, L, path, path_len, n_path,
                                kv->len_dev, (hipStream_t)stream));
  return PPD_OK;
}

ppd_status ppd_next_tree(int32_t T, const int32_t *parent, const int32_t *ids, int32_t vocab,
                         int32_t n_prompt, int32_t n_ept, const float *logits, const int32_t *path,
                         const int32_t *n_path, const int32_t *next_tok, int32_t tpl_T,
                         const int32_t *tpl_parent, const int32_t *tpl_kind, int32_t *next_ids,
                         void *ws, size_t ws_bytes, void *stream) {
  if (T < 1 || T > PPD_T_MAX) return fail(PPD_EINVAL, "T=%d outside [1, %d]", T, PPD_T_MAX);
  if (tpl_T < 1 || tpl_T > PPD_T_MAX)
    return fail(PPD_EINVAL, "template size %d outside [1, %d]", tpl_T, PPD_T_MAX);
  if (vocab < 1 || n_prompt < 0) return fail(PPD_EINVAL, "vocab must be positive, n_prompt >= 0");
  if (n_ept < 1 || n_ept > PPD_EPT_MAX || (int64_t)n_prompt * n_ept > 32767)
    return fail(PPD_EINVAL, "n_ept=%d outside [1, %d] or too many prompt ids", n_ept, PPD_EPT_MAX);
  if (!parent || !ids || !logits || !path || !n_path || !next_tok || !tpl_parent || !tpl_kind ||
      !next_ids)
    return fail(PPD_EINVAL, "NULL argument");
  if (!ws || ws_bytes < 16) return fail(PPD_EWORKSPACE, "workspace (status word) required");
  NextTreeLaunch p{};
  p.parent = parent;
  p.ids = ids;
  p.T = T;
  p.vocab = vocab;
  p.n_ept = n_ept;
  p.logits = logits;
  p.path = path;
  p.n_path = n_path;
  p.next_tok = next_tok;
  p.next_ids = next_ids;
  p.status = (uint32_t *)ws;
  p.tpl_T = tpl_T;
  // the template: topological, candidates under the root or candidates,
  // one prompt chain per EPT group under candidates, in token-distance order
  if (tpl_parent[0] != -1) return fail(PPD_EINVAL, "template: tpl_parent[0] must be -1");
  int n_depths = 0;
  for (int i = 0; i < tpl_T; ++i) {
    const int par = tpl_parent[i], kind = tpl_kind[i];
    int depth = 0;
    if (i > 0) {
      if (par < 0 || par >= i)
        return fail(PPD_EINVAL, "template: tpl_parent[%d]=%d is not an earlier node", i, par);
      const int pk = par > 0 ? tpl_kind[par] : 0;  // the root counts as a candidate
      depth = p.tpl_depth[par] + 1;
      if (kind >= 0) {
        if (pk < 0) return fail(PPD_EINVAL, "template: candidate %d under a prompt token", i);
        if (kind >= PPD_TOPK_MAX || kind >= vocab)
          return fail(PPD_EINVAL, "template: rank %d of node %d too large", kind, i);
        if (depth > PPD_NEXT_MAX_DEPTH)
          return fail(PPD_EINVAL, "template: candidate depth %d > %d", depth, PPD_NEXT_MAX_DEPTH);
        p.k_of_depth[depth] = std::max(p.k_of_depth[depth], kind + 1);
        n_depths = std::max(n_depths, depth);
      } else {
        const int q = -kind - 1;  // prompt embedding: token distance j + 1, EPT group g
        const int j = q / n_ept, g = q % n_ept;
        if (kind < -32767 || j >= n_prompt)
          return fail(PPD_EINVAL, "template: prompt id %d beyond %d token distances", q, n_prompt);
        if (j == 0 ? pk < 0 : pk != -1 - ((j - 1) * n_ept + g))
          return fail(PPD_EINVAL, "template: prompt token %d of node %d out of chain order", q, i);
      }
    }
    if (depth > 127) return fail(PPD_EINVAL, "template too deep");
    p.tpl_depth[i] = (int8_t)depth;
    p.tpl_kind[i] = (int16_t)(i == 0 ? 0 : std::max(kind, -32768));
  }
  if (g_timer.kind == TK_NEXT) g_timer.next = 0;  // one timed launch per call
  timer_events(TK_NEXT, &p.ev_start, &p.ev_stop);
  PPD_TRY_HIP(launch_next_tree(p, n_depths, (hipStream_t)stream));
  return PPD_OK;
}

ppd_status ppd_read_probe(const void *buf, size_t bytes, uint32_t *sink, void *stream) {
  if (!buf || !sink) return fail(PPD_EINVAL, "NULL argument");
  if (bytes % 16 || ((uintptr_t)buf & 15)) return fail(PPD_EINVAL, "buf and bytes must be 16-byte aligned");
  PPD_TRY_HIP(launch_read_probe(buf, bytes, sink, (hipStream_t)stream));
  return PPD_OK;
}

ppd_status ppd_device_status(void *ws, size_t ws_bytes, uint32_t *status_out, int32_t clear,
                             void *stream) {
  if (!ws || ws_bytes < 16 || !status_out) return fail(PPD_EINVAL, "NULL or short workspace");
  hipStream_t s = (hipStream_t)stream;
  PPD_TRY_HIP(hipMemcpyAsync(status_out, ws, sizeof(uint32_t), hipMemcpyDeviceToHost, s));
  PPD_TRY_HIP(hipStreamSynchronize(s));
  if (clear) PPD_TRY_HIP(launch_ws_init(ws, 4, s));
  return PPD_OK;
}

ppd_status ppd_set_kernel_timer(int32_t kind, void *const *start_events, void *const *stop_events,
                                int32_t n_events) {
  if (n_events <= 0) {
    g_timer = KernelTimer{};
    return PPD_OK;
  }
  if (kind < TK_QKV || kind > TK_NEXT || !start_events || !stop_events)
    return fail(PPD_EINVAL, "bad kernel timer arguments");
  g_timer.kind = kind;
  g_timer.start = start_events;
  g_timer.stop = stop_events;
  g_timer.n = n_events;
  g_timer.next = 0;
  return PPD_OK;
}

const char *ppd_last_error(void) { return g_err.c_str(); }

size_t ppd_packed_weight_bytes(int32_t kind, int32_t rows, int32_t cols) {
  int gk, N;
  if (pack_args(kind, rows, cols, &gk, &N) != PPD_OK) return 0;
  return (size_t)gemm_groups_of(gk, N) * gemm_sub_of(gk) * 16 * cols * sizeof(bf16_t);
}

ppd_status ppd_pack_weight(int32_t kind, int32_t rows, int32_t cols, const void *src, void *dst,
                           void *stream) {
  int gk, N;
  ppd_status st = pack_args(kind, rows, cols, &gk, &N);
  if (st != PPD_OK) return st;
  if (!src || !dst) return fail(PPD_EINVAL, "NULL weight pointer");
  PPD_TRY_HIP(launch_pack_weight(gk, N, cols, (const bf16_t *)src, (bf16_t *)dst, (hipStream_t)stream));
  return PPD_OK;
}

}  // extern "C"
