// Host runtime behind the C ABI: model and KV-cache objects, the launch plan
// of one target forward over a batch of window rows, and the verification /
// prefill / rollback entry points.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/dsi.h"
#include "internal.h"

using namespace dsi;

namespace {

thread_local std::string g_err;

dsi_status fail(dsi_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return st;
}

#define HIP_TRY(expr)                                                              \
  do {                                                                             \
    hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess)                                                          \
      return fail(DSI_EHIP, "%s failed: %s", #expr, hipGetErrorString(e_));        \
  } while (0)

#define DSI_TRY(expr)               \
  do {                              \
    dsi_status s_ = (expr);         \
    if (s_ != DSI_OK) return s_;    \
  } while (0)

size_t round_up(size_t x, size_t m) { return (x + m - 1) / m * m; }
int cdiv(int a, int b) { return (a + b - 1) / b; }

struct DevBuf {
  void* p = nullptr;
  size_t bytes = 0;
};

dsi_status ensure(DevBuf& b, size_t bytes) {
  if (b.bytes >= bytes) return DSI_OK;
  if (b.p) {
    hipError_t e = hipFree(b.p);
    b.p = nullptr;
    b.bytes = 0;
    if (e != hipSuccess) return fail(DSI_EHIP, "hipFree: %s", hipGetErrorString(e));
  }
  hipError_t e = hipMalloc(&b.p, bytes);
  if (e != hipSuccess) {
    hipGetLastError();
    b.p = nullptr;
    return fail(DSI_ENOMEM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
  }
  b.bytes = bytes;
  return DSI_OK;
}

}  // namespace

struct LayerW {
  float* attn_norm = nullptr;
  float* ffn_norm = nullptr;
  void* wqkv = nullptr;
  void* wo = nullptr;
  void* wgu = nullptr;
  void* wdown = nullptr;
  // the same matrices in the ring layout of their role (nullable)
  void* wqkv_s = nullptr;
  void* wo_s = nullptr;
  void* wgu_s = nullptr;
  void* wdown_s = nullptr;
};

struct dsi_model {
  dsi_config cfg;
  hipStream_t stream = nullptr;
  int wtype = 0, kvb = 0, esz = 4, kvesz = 4;
  int d = 0, hq = 0, hkv = 0, hd = 0, qdim = 0, kvdim = 0, ff = 0, V = 0, L = 0;
  int Kb_d = 0, Kb_q = 0, Kb_ff = 0;
  int Nb_qkv = 0, Nb_o = 0, Nb_gu = 0, Nb_down = 0, Nb_head = 0;
  int G_gu = 1, G_head = 1;   // n-block groups of the packed gate/up and LM head
  // ring layouts of the four layer GEMMs (nbw == 0: the role has none) and
  // whether one-row-tile forwards on single-window caches use them
  RingCfg rc_qkv, rc_o, rc_gu, rc_down, rc_head;
  bool use_ring = true;
  void* embed = nullptr;
  float* final_norm = nullptr;
  void* lm_head = nullptr;
  void* lm_head_s = nullptr;   // the LM head in the ring layout (nullable)
  std::vector<LayerW> layers;
  std::vector<unsigned> set_mask;   // [L+1]: bit per tensor id (index 0: globals)
  std::vector<void*> allocs;
  // forward workspace for up to kMaxRows rows
  float* x = nullptr;
  float* delta = nullptr;       // [kMaxSplits][kMaxRows][d] K-split partial outputs
  float* ssq = nullptr;         // [kMaxRows][Nb_o] per-n-block sums of x^2 (EPI_RESID)
  float* ssq2 = nullptr;        // [kMaxRows][Nb_down] the same after the down projection
  int* gcnt = nullptr;          // EPI_PARTRES arrival counters
  PackRef pk_d{}, pk_q{}, pk_ff{};
  float* qbuf = nullptr;
  float2* rope = nullptr;
  float* logits = nullptr;
  void* vws = nullptr;
  void* dws = nullptr;          // drafter-sampling workspace
  // token trees: per-row depth and ancestor mask, per-window flags/decisions
  int* tdepth = nullptr;
  unsigned long long* tanc = nullptr;
  int* tbad = nullptr;
  int4* tdec = nullptr;
  int* err = nullptr;
  DevBuf attn_o, attn_ml;
  int live_kv = 0;
  // diagnostics: event pairs around one kernel class
  int prof_class = 0;
  std::vector<hipEvent_t> prof_ev;
  size_t prof_used = 0;
  // shape of the most recent verification forward (for dsi_profile_kernel)
  int last_window0 = -1, last_B = 0, last_R = 0;
  // captured verification steps, keyed by every value their launches use
  bool use_graphs = true;
  struct Graph {
    std::vector<uint64_t> key;
    hipGraphExec_t exec = nullptr;
    uint64_t used = 0;
  };
  std::vector<Graph> graphs;
  uint64_t graph_clock = 0;
};

struct dsi_kv {
  dsi_model* m = nullptr;
  int n_windows = 0, max_len = 0, maxlen_pad = 0;
  void* k = nullptr;
  void* v = nullptr;
  int* lens = nullptr;
  std::vector<long long> hi, lo;   // host bounds on each window's length
  size_t win_elems = 0;            // elements of one (layer, window) of K (= of V)
};

namespace {

dsi_status dev_alloc(std::vector<void*>& list, void** p, size_t bytes) {
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    hipGetLastError();
    *p = nullptr;
    return fail(DSI_ENOMEM, "hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
  }
  list.push_back(*p);
  e = hipMemset(*p, 0, bytes);
  if (e != hipSuccess) return fail(DSI_EHIP, "hipMemset failed: %s", hipGetErrorString(e));
  return DSI_OK;
}

void free_list(std::vector<void*>& list) {
  for (void* p : list) hipFree(p);
  list.clear();
}

bool all_set(const dsi_model* m) {
  const unsigned glob = (1u << DSI_T_EMBED) | (1u << DSI_T_FINAL_NORM) | (1u << DSI_T_LM_HEAD);
  const unsigned lay = 0xFF8u;   // ids 3..11
  if ((m->set_mask[0] & glob) != glob) return false;
  for (int l = 0; l < m->L; ++l)
    if ((m->set_mask[l + 1] & lay) != lay) return false;
  return true;
}

void* kv_ptr(const dsi_kv* kv, void* base, int layer, int window) {
  const size_t off = ((size_t)layer * kv->n_windows + window) * kv->win_elems;
  return (char*)base + off * kv->m->kvesz;
}

PackRef make_pack(dsi_model* m, int Kb, dsi_status* st) {
  PackRef p{};
  p.Kb = Kb;
  const size_t elems = (size_t)kMaxMt * Kb * 512;
  *st = dev_alloc(m->allocs, &p.hi, elems * m->esz);
  if (*st == DSI_OK && m->wtype == W_BF16) *st = dev_alloc(m->allocs, &p.lo, elems * 2);
  return p;
}

// event pair around the launches of one kernel class (diagnostics only)
struct Prof {
  dsi_model* m;
  int idx = -1;
  Prof(dsi_model* mm, int cls) : m(mm) {
    if (m->prof_class != cls) return;
    if (m->prof_used + 2 > m->prof_ev.size()) {
      hipEvent_t a, b;
      if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) return;
      m->prof_ev.push_back(a);
      m->prof_ev.push_back(b);
    }
    idx = (int)m->prof_used;
    m->prof_used += 2;
    hipEventRecord(m->prof_ev[idx], m->stream);
  }
  ~Prof() {
    if (idx >= 0) hipEventRecord(m->prof_ev[idx + 1], m->stream);
  }
};

// ------------------------------------------------------------- forward plan
//
// GEMM arguments of each kernel class of layer l over M rows, shared by the
// forward and the profiling replay.
//   QKV     attn-normed pack pk_d -> q, K/V cache (RoPE, append)
//   O       attention pack pk_q -> x += o W_o^T (in place), pk_d = x * g_ffn,
//           per-n-block sums of x^2 (EPI_RESID)
//   gate/up pk_d scaled by the RMSNorm of x (ssq) -> SwiGLU pack pk_ff
//   down    pk_ff -> K-split partials; below the last layer the last split
//           to finish folds them into x and writes the next layer's
//           attention-norm input pk_d = x * g_attn and ssq2 (EPI_PARTRES);
//           after the last layer the final RMSNorm folds them
//   QKV     (layers >= 1) scaled by the RMSNorm of x from ssq2
//   head    final-normed pack pk_d -> logits
// Ring layout of one role for a launch (a one-row-tile forward on a
// single-window cache): see ring_forward.
void set_ring(GemmArgs& g, const RingCfg& c, const void* ws, bool ring) {
  if (ring && c.nbw && ws) {
    g.Ws = ws;
    g.ring_nk = c.nk;
    g.ring_nbw = c.nbw;
  }
}

GemmArgs qkv_args(dsi_model* m, dsi_kv* kv, int l, int M, RowMap rows, bool ring = false) {
  GemmArgs g{};
  g.M = M;
  g.S = 1;
  g.W = m->layers[l].wqkv;
  set_ring(g, m->rc_qkv, m->layers[l].wqkv_s, ring);
  g.Xhi = m->pk_d.hi;
  g.Xlo = m->pk_d.lo;
  g.Nb = m->Nb_qkv;
  g.Kb = m->Kb_d;
  g.epi.kind = EPI_QKV;
  g.epi.q_out = m->qbuf;
  g.epi.kcache = kv_ptr(kv, kv->k, l, 0);
  g.epi.vcache = kv_ptr(kv, kv->v, l, 0);
  g.epi.kv_bf16 = m->kvb;
  g.epi.n_heads = m->hq;
  g.epi.n_kv = m->hkv;
  g.epi.hd = m->hd;
  g.epi.maxlen = kv->maxlen_pad;
  g.epi.rope = m->rope;
  g.epi.rows = rows;
  if (l > 0) {   // the previous layer's down projection left x * g_attn and ssq2
    g.ssq = m->ssq2;
    g.ssq_n = m->Nb_down;
    g.norm_d = m->d;
    g.eps = m->cfg.rms_eps;
  }
  return g;
}

GemmArgs oproj_args(dsi_model* m, int l, int M, bool ring = false) {
  GemmArgs g{};
  g.M = M;
  g.S = 1;
  g.W = m->layers[l].wo;
  set_ring(g, m->rc_o, m->layers[l].wo_s, ring);
  g.Xhi = m->pk_q.hi;
  g.Xlo = m->pk_q.lo;
  g.Nb = m->Nb_o;
  g.Kb = m->Kb_q;
  g.epi.kind = EPI_RESID;
  g.epi.x = m->x;
  g.epi.ld = m->d;
  g.epi.n_valid = m->d;
  g.epi.gain = m->layers[l].ffn_norm;
  g.epi.pack = m->pk_d;
  g.epi.ssq = m->ssq;
  return g;
}

GemmArgs gateup_args(dsi_model* m, int l, int M, bool ring = false) {
  GemmArgs g{};
  g.M = M;
  g.S = 1;
  g.W = m->layers[l].wgu;
  set_ring(g, m->rc_gu, m->layers[l].wgu_s, ring);
  g.Xhi = m->pk_d.hi;
  g.Xlo = m->pk_d.lo;
  g.Nb = m->Nb_gu;
  g.Kb = m->Kb_d;
  g.G = m->G_gu;
  g.epi.kind = EPI_SILU;
  g.epi.pack = m->pk_ff;
  g.epi.ff = m->ff;
  g.ssq = m->ssq;
  g.ssq_n = m->Nb_o;
  g.norm_d = m->d;
  g.eps = m->cfg.rms_eps;
  return g;
}

GemmArgs down_args(dsi_model* m, int l, int M, int mt, float* hidden_next = nullptr, bool ring = false) {
  GemmArgs g{};
  g.M = M;
  g.W = m->layers[l].wdown;
  set_ring(g, m->rc_down, m->layers[l].wdown_s, ring);
  g.Xhi = m->pk_ff.hi;
  g.Xlo = m->pk_ff.lo;
  g.Nb = m->Nb_down;
  g.Kb = m->Kb_ff;
  g.S = gemm_part_splits(m->wtype, m->Nb_down, m->Kb_ff, mt);
  if (g.Ws && g.S != m->rc_down.S) {   // the ring layout was built for another split
    g.Ws = nullptr;
    g.ring_nk = 0;
    g.ring_nbw = 0;
  }
  g.epi.kind = EPI_PART;
  g.epi.out = m->delta;
  g.epi.ld = m->d;
  g.epi.part_stride = (size_t)kMaxRows * m->d;
  g.epi.n_valid = m->d;
  if (l + 1 < m->L) {
    g.epi.kind = EPI_PARTRES;
    g.epi.x = m->x;
    g.epi.gain = m->layers[l + 1].attn_norm;
    g.epi.pack = m->pk_d;
    g.epi.ssq = m->ssq2;
    g.epi.cnt = m->gcnt;
    g.epi.copy = hidden_next;
  }
  return g;
}

GemmArgs head_args(dsi_model* m, float* logits, int M, bool ring = false) {
  GemmArgs g{};
  g.M = M;
  g.S = 1;
  g.W = m->lm_head;
  set_ring(g, m->rc_head, m->lm_head_s, ring);
  g.Xhi = m->pk_d.hi;
  g.Xlo = m->pk_d.lo;
  g.Nb = m->Nb_head;
  g.Kb = m->Kb_d;
  g.G = m->G_head;
  g.epi.kind = EPI_STORE;
  g.epi.out = logits;
  g.epi.ld = m->V;
  g.epi.n_valid = m->V;
  return g;
}

//
// One target forward over M = B * R rows: R consecutive rows of each of the
// B windows window0..window0+B-1, appended after each window's cached
// length.  Writes the rows' K/V into the cache (the window length itself is
// advanced by the caller).  logits: nullptr (no head), else [M][V]
// (head_last_only: only the last row, into logits[0..V)).
// Attention partition of a forward: query tiles and key chunks.  Sized from
// the host bound on lengths; allocates the chunk-partial buffers (so no
// allocation happens while launches are being captured).
struct AttnPlan {
  int n_qtiles = 0, chunk = 0, n_chunks = 0, waves = kAttnWaves;
};

dsi_status plan_attention(dsi_model* m, dsi_kv* kv, int window0, int B, int R, AttnPlan* p) {
  long long kmax = 0;
  for (int b = 0; b < B; ++b) kmax = std::max(kmax, kv->hi[window0 + b] + R);
  // The chunk size depends only on the model, R and the cache capacity --
  // never on B or the current lengths -- so a window's partial sums and
  // therefore its results are identical alone or inside a batch.
  const int G = m->hq / m->hkv;
  p->n_qtiles = cdiv(G * R, 16);
  // about two workgroups per CU for one window (a full second round, not a
  // short tail): at most 512 / (KV heads x query tiles) chunks, when every
  // wave takes a single 32-key step (latency-bound); when that still leaves
  // several steps per wave (long prefixes, bandwidth-bound), at most 256 /
  // (KV heads x query tiles) chunks: one round of workgroups streams faster
  // than two
  const int units = m->hkv * p->n_qtiles;
  int want = std::max(1, 512 / units);
  auto chunk_of = [&](int w, int q) {
    const int c = (int)round_up((size_t)cdiv(kv->max_len, w), (size_t)q);
    return std::min(std::max(c, q), 16384);
  };
  // A cache with many windows (verification tasks batched together) whose
  // 8-wave plan gives every wave a single 32-key step (latency-bound) would
  // need several rounds of 8-wave workgroups when all its windows are
  // verified at once: there, 4-wave workgroups with twice the chunks, three
  // per CU, finish sooner.  Multi-step waves (long prefixes) stay at 8 waves.
  // The choice depends on the cache's capacity (windows, max_len), never on
  // the call's batch or lengths.
  const int q8 = kAttnWaves * 32;
  int chunk8 = chunk_of(want, q8);
  if (chunk8 > q8) {
    want = std::max(1, 256 / units);
    chunk8 = chunk_of(want, q8);
  }
  const long long full8 = (long long)kv->n_windows * m->hkv * p->n_qtiles * cdiv(kv->max_len, chunk8);
  p->waves = (chunk8 == q8 && full8 > 256) ? 4 : kAttnWaves;
  p->chunk = p->waves == 4 ? chunk_of(2 * want, 4 * 32) : chunk_of(want, q8);
  // A short cache is read in one chunk per (window, KV head, query tile):
  // the kernel then normalises its own output and the combine launch (~4-5
  // us) is saved, at the price of a few dependent steps per wave -- up to
  // three, or five when there are at least 64 such workgroups (many
  // windows).  Measured per step: 1B at 518 positions 0.797 -> 0.771 ms,
  // 8B at 523 3.243 -> 3.217 ms, the 7-window 8B batch at 1036 (112
  // workgroups) 4.615 -> 4.545 ms; a single 8B or 13B window at 1035
  // positions (five steps, 24 and 40 workgroups) was 2 % slower, at 2059
  // (nine steps) 10 %.
  const int steps1 = cdiv(kv->max_len, q8);
  const long long wg1 = (long long)kv->n_windows * m->hkv * p->n_qtiles;
  if (steps1 <= 3 || (steps1 <= 5 && wg1 >= 64)) {
    p->waves = kAttnWaves;
    p->chunk = chunk_of(1, q8);
  }
  p->n_chunks = (int)((kmax + p->chunk - 1) / p->chunk);
  const size_t nparts = (size_t)B * m->hkv * p->n_qtiles * p->n_chunks * 16;
  DSI_TRY(ensure(m->attn_o, nparts * m->hd * sizeof(float)));
  DSI_TRY(ensure(m->attn_ml, nparts * sizeof(float2)));
  return DSI_OK;
}

// Whether a forward runs its layer GEMMs on the ring layouts: every bf16
// forward of a model built with them (one to four row tiles, any number of
// windows).  The ring kernels form each row's sums in the same order for
// every row count, so a window's results are the same alone or inside a
// batch.
bool ring_forward(const dsi_model* m, const dsi_kv* kv, int mt) {
  (void)kv;
  return m->use_ring && m->wtype == W_BF16 && mt >= 1 && mt <= kMaxMt;
}

// Stream-ordered launches only (capturable into a graph).  depth / anc
// (nullable, device [M]): token-tree rows (RowMap::depth, AttnArgs::anc).
dsi_status run_forward(dsi_model* m, dsi_kv* kv, const AttnPlan& ap, int window0, int B, int R,
                       const int* d_tokens, float* logits, int head_last_only, float* hidden,
                       const int* depth = nullptr, const unsigned long long* anc = nullptr) {
  hipStream_t s = m->stream;
  const int M = B * R;
  const int mt = cdiv(M, 16);
  RowMap rows{kv->lens, window0, R, depth};
  const size_t Md = (size_t)M * m->d;
  const bool ring = ring_forward(m, kv, mt);

  EmbedArgs ea{};
  ea.tokens = d_tokens;
  ea.E = m->embed;
  ea.wtype = m->wtype;
  ea.V = m->V;
  ea.d = m->d;
  ea.M = M;
  ea.x = m->x;
  ea.gain = m->layers[0].attn_norm;
  ea.eps = m->cfg.rms_eps;
  ea.pack = m->pk_d;
  ea.rope = m->rope;
  ea.hd = m->hd;
  ea.log2_base = log2((double)m->cfg.rope_base);
  ea.rows = rows;
  ea.err = m->err;
  ea.hidden0 = hidden;
  HIP_TRY(launch_embed_norm(ea, s));

  int last_splits = 0;
  const size_t dstride = (size_t)kMaxRows * m->d;
  for (int l = 0; l < m->L; ++l) {
    // fused QKV + RoPE + KV append
    {
      Prof p(m, DSI_K_QKV);
      HIP_TRY(launch_gemm(m->wtype, mt, qkv_args(m, kv, l, M, rows, ring), s));
    }

    AttnArgs aa{};
    aa.q = m->qbuf;
    aa.kc = kv_ptr(kv, kv->k, l, 0);
    aa.vc = kv_ptr(kv, kv->v, l, 0);
    aa.rows = rows;
    aa.n_windows = B;
    aa.n_heads = m->hq;
    aa.n_kv = m->hkv;
    aa.maxlen = kv->maxlen_pad;
    aa.n_qtiles = ap.n_qtiles;
    aa.chunk = ap.chunk;
    aa.n_chunks = ap.n_chunks;
    aa.scale = (float)(1.0 / sqrt((double)m->hd));
    aa.part_o = (float*)m->attn_o.p;
    aa.part_ml = (float2*)m->attn_ml.p;
    aa.out = m->pk_q;
    aa.wtype = m->wtype;
    aa.anc = anc;
    aa.waves = ap.waves;
    {
      Prof p(m, DSI_K_ATTN);
      HIP_TRY(launch_attention(m->kvb, m->hd, aa, s));
    }

    // O projection: residual update in place, FFN-norm input for gate/up
    {
      Prof p(m, DSI_K_OPROJ);
      HIP_TRY(launch_gemm(m->wtype, mt, oproj_args(m, l, M, ring), s));
    }
    // gate/up (RMSNorm scale applied to the accumulators) + SwiGLU
    {
      Prof p(m, DSI_K_GATEUP);
      HIP_TRY(launch_gemm(m->wtype, mt, gateup_args(m, l, M, ring), s));
    }
    // down projection into K-split partials
    // down projection; below the last layer it also folds the residual and
    // prepares the next layer's normed input (EPI_PARTRES)
    const GemmArgs gd = down_args(m, l, M, mt, hidden ? hidden + (size_t)(l + 1) * Md : nullptr, ring);
    {
      Prof p(m, DSI_K_DOWN);
      HIP_TRY(launch_gemm(m->wtype, mt, gd, s));
    }
    last_splits = gd.S;
  }
  if (!logits) {
    // fold the last residual update only when the caller wants hidden states
    if (hidden)
      HIP_TRY(launch_rmsnorm_pack(m->x, m->delta, last_splits, dstride, M, m->d, m->final_norm,
                                  m->cfg.rms_eps, m->wtype, m->pk_d, hidden + (size_t)m->L * Md, s));
    return DSI_OK;
  }

  GemmArgs gh = head_args(m, logits, M, ring);
  Prof ph(m, DSI_K_HEAD);
  if (head_last_only) {
    const size_t off = (size_t)(M - 1) * m->d;
    HIP_TRY(launch_rmsnorm_pack(m->x + off, m->delta + off, last_splits, dstride, 1, m->d, m->final_norm,
                                m->cfg.rms_eps, m->wtype, m->pk_d, nullptr, s));
    gh.M = 1;
    HIP_TRY(launch_gemm(m->wtype, 1, gh, s));
  } else {
    HIP_TRY(launch_rmsnorm_pack(m->x, m->delta, last_splits, dstride, M, m->d, m->final_norm,
                                m->cfg.rms_eps, m->wtype, m->pk_d,
                                hidden ? hidden + (size_t)m->L * Md : nullptr, s));
    gh.M = M;
    HIP_TRY(launch_gemm(m->wtype, mt, gh, s));
  }
  return DSI_OK;
}

// library workspace for dsi_accept, one per device
struct AcceptWs {
  DevBuf ws;
  int* err = nullptr;
};
std::mutex g_accept_mu;
std::map<int, AcceptWs> g_accept;

dsi_status check_err_word(int* err, hipStream_t s) {
  HIP_TRY(hipStreamSynchronize(s));
  int h = 0;
  HIP_TRY(hipMemcpy(&h, err, sizeof(int), hipMemcpyDeviceToHost));
  if (h) {
    HIP_TRY(hipMemset(err, 0, sizeof(int)));
    std::string what;
    if (h & 1) what += " token id outside [0, vocab);";
    if (h & 2) what += " verification input invalid (token id or q(d) <= 0);";
    if (h & 4) what += " rollback above the current length;";
    if (h & 8) what += " token-tree parent array invalid;";
    return fail(DSI_EINVAL, "device-detected input error:%s", what.c_str());
  }
  return DSI_OK;
}

dsi_status verify_args_ok(int B, int k, int V, const int* tokens, const float* q, const float* u,
                          float T, int mode, const int* n_out, const int* tok_out) {
  if (B < 1) return fail(DSI_EINVAL, "n_windows must be >= 1");
  if (k < 0) return fail(DSI_EINVAL, "k must be >= 0");
  if ((long long)B * (k + 1) > DSI_MAX_ROWS)
    return fail(DSI_EINVAL, "n_windows*(k+1) = %lld exceeds %d", (long long)B * (k + 1), DSI_MAX_ROWS);
  if (!tokens || !n_out || !tok_out) return fail(DSI_EINVAL, "null tokens or output pointer");
  if (mode != DSI_SAMPLE && mode != DSI_GREEDY) return fail(DSI_EINVAL, "bad mode %d", mode);
  if (mode == DSI_SAMPLE) {
    if (!u) return fail(DSI_EINVAL, "sample mode needs d_u");
    if (k > 0 && !q) return fail(DSI_EINVAL, "sample mode needs d_q");
    if (!(T > 0.f) || !isfinite(T)) return fail(DSI_EINVAL, "temperature must be positive");
  }
  if (V < 1) return fail(DSI_EINVAL, "vocab must be >= 1");
  return DSI_OK;
}

// Launch a verification step through a cached graph: captured from the
// stream on first use of a key, replayed afterwards (one submission instead
// of a few hundred kernel launches).  At most kMaxGraphs are kept (least
// recently used evicted).
constexpr size_t kMaxGraphs = 16;

template <typename F>
dsi_status replay_or_capture(dsi_model* m, const std::vector<uint64_t>& key, F&& launches) {
  ++m->graph_clock;
  for (auto& g : m->graphs)
    if (g.key == key) {
      g.used = m->graph_clock;
      HIP_TRY(hipGraphLaunch(g.exec, m->stream));
      return DSI_OK;
    }
  HIP_TRY(hipStreamBeginCapture(m->stream, hipStreamCaptureModeThreadLocal));
  const dsi_status st = launches();
  hipGraph_t graph = nullptr;
  const hipError_t e = hipStreamEndCapture(m->stream, &graph);
  if (st != DSI_OK) {
    if (graph) hipGraphDestroy(graph);
    return st;
  }
  if (e != hipSuccess) return fail(DSI_EHIP, "graph capture: %s", hipGetErrorString(e));
  hipGraphExec_t exec = nullptr;
  const hipError_t ei = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  hipGraphDestroy(graph);
  if (ei != hipSuccess) return fail(DSI_EHIP, "graph instantiate: %s", hipGetErrorString(ei));
  if (m->graphs.size() >= kMaxGraphs) {
    auto old = std::min_element(m->graphs.begin(), m->graphs.end(),
                                [](const dsi_model::Graph& x, const dsi_model::Graph& y) {
                                  return x.used < y.used;
                                });
    hipGraphExecDestroy(old->exec);
    m->graphs.erase(old);
  }
  m->graphs.push_back(dsi_model::Graph{key, exec, m->graph_clock});
  HIP_TRY(hipGraphLaunch(exec, m->stream));
  return DSI_OK;
}

// ---------------------------------------------------------------- no-alloc accept
// Fixed device array holding the accept/reject workspace of
// dsi_accept_noalloc: the first 256 bytes are the device error word, the
// rest the verification workspace.  Each device holds its own copy at its own
// address until the process ends.  In host code `scratch` names a host-side
// stand-in, so kernels and fills only ever see the device address taken by
// hipGetSymbolAddress below.
constexpr size_t kScratchHead = 256;
static __device__ __align__(256) unsigned char scratch[DSI_ACCEPT_NOALLOC_BYTES];
std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_dev;   // device -> device address of its `scratch`

dsi_status scratch_address(int dev, void** out) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_dev.find(dev);
  if (it != g_scratch_dev.end()) {
    *out = it->second;
    return DSI_OK;
  }
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !p) {
    hipGetLastError();
    return fail(DSI_EHIP, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
  }
  g_scratch_dev[dev] = p;
  *out = p;
  return DSI_OK;
}

}  // namespace

extern "C" {

const char* dsi_last_error(void) { return g_err.c_str(); }

dsi_status dsi_model_create(const dsi_config* cfg, void* stream, dsi_model** out) {
  if (!cfg || !out) return fail(DSI_EINVAL, "null argument");
  const dsi_config c = *cfg;
  if (c.n_layers < 1 || c.d_model < 32 || c.d_model % 32 || c.n_heads < 1 || c.n_kv_heads < 1 ||
      c.n_heads % c.n_kv_heads || c.d_ff < 1 || c.vocab < 1)
    return fail(DSI_EINVAL, "invalid shape (d_model must be a multiple of 32)");
  if (c.d_model > 8192) return fail(DSI_EINVAL, "d_model must be at most 8192");
  if (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 96 && c.head_dim != 128)
    return fail(DSI_EINVAL, "head_dim must be 32, 64, 96 or 128");
  if ((c.wdtype != DSI_F32 && c.wdtype != DSI_BF16) || (c.kvdtype != DSI_F32 && c.kvdtype != DSI_BF16))
    return fail(DSI_EINVAL, "bad dtype");
  if (!(c.rms_eps >= 0.f) || !(c.rope_base > 0.f)) return fail(DSI_EINVAL, "bad eps / rope_base");
  dsi_model* m = new (std::nothrow) dsi_model();
  if (!m) return fail(DSI_ENOMEM, "host allocation failed");
  m->cfg = c;
  m->stream = (hipStream_t)stream;
  // graph replay needs a capturable stream (not the null stream)
  const char* g = getenv("DSI_GRAPHS");
  m->use_graphs = stream != nullptr && !(g && g[0] == '0');
  m->wtype = c.wdtype == DSI_BF16 ? W_BF16 : W_F32;
  m->kvb = c.kvdtype == DSI_BF16 ? 1 : 0;
  m->esz = m->wtype == W_BF16 ? 2 : 4;
  m->kvesz = m->kvb ? 2 : 4;
  m->d = c.d_model;
  m->hq = c.n_heads;
  m->hkv = c.n_kv_heads;
  m->hd = c.head_dim;
  m->qdim = c.n_heads * c.head_dim;
  m->kvdim = c.n_kv_heads * c.head_dim;
  m->ff = c.d_ff;
  m->V = c.vocab;
  m->L = c.n_layers;
  m->Kb_d = m->d / 32;
  m->Kb_q = m->qdim / 32;
  m->Kb_ff = cdiv(m->ff, 32);
  m->Nb_qkv = (m->qdim + 2 * m->kvdim) / 16;
  m->Nb_o = m->d / 16;
  m->Nb_gu = cdiv(m->ff, 8);
  m->Nb_down = m->d / 16;
  m->Nb_head = cdiv(m->V, 16);
  m->G_gu = gemm_wgroup(m->wtype, EPI_SILU, m->Nb_gu);
  m->G_head = gemm_wgroup(m->wtype, EPI_STORE, m->Nb_head);
  const char* rg = getenv("DSI_RING");
  m->use_ring = !(rg && rg[0] == '0');
  ring_config(m->wtype, EPI_QKV, m->Nb_qkv, m->Kb_d, 1, &m->rc_qkv);
  ring_config(m->wtype, EPI_RESID, m->Nb_o, m->Kb_q, 1, &m->rc_o);
  ring_config(m->wtype, EPI_SILU, m->Nb_gu, m->Kb_d, 1, &m->rc_gu);
  ring_config(m->wtype, EPI_STORE, m->Nb_head, m->Kb_d, 1, &m->rc_head);
  ring_config(m->wtype, EPI_PARTRES, m->Nb_down, m->Kb_ff,
              gemm_part_splits(m->wtype, m->Nb_down, m->Kb_ff, 1), &m->rc_down);
  m->layers.resize(m->L);
  m->set_mask.assign(m->L + 1, 0u);

  dsi_status st = DSI_OK;
  auto A = [&](void** p, size_t bytes) {
    if (st == DSI_OK) st = dev_alloc(m->allocs, p, bytes);
  };
  const size_t tile = 512;
  A(&m->embed, (size_t)m->V * m->d * m->esz);
  A((void**)&m->final_norm, (size_t)m->d * 4);
  A(&m->lm_head, (size_t)m->Nb_head * m->Kb_d * tile * m->esz);
  if (m->use_ring && m->rc_head.nbw) A(&m->lm_head_s, m->rc_head.tiles() * tile * m->esz);
  for (int l = 0; l < m->L && st == DSI_OK; ++l) {
    LayerW& w = m->layers[l];
    A((void**)&w.attn_norm, (size_t)m->d * 4);
    A((void**)&w.ffn_norm, (size_t)m->d * 4);
    A(&w.wqkv, (size_t)m->Nb_qkv * m->Kb_d * tile * m->esz);
    A(&w.wo, (size_t)m->Nb_o * m->Kb_q * tile * m->esz);
    A(&w.wgu, (size_t)m->Nb_gu * m->Kb_d * tile * m->esz);
    A(&w.wdown, (size_t)m->Nb_down * m->Kb_ff * tile * m->esz);
    if (m->use_ring) {
      if (m->rc_qkv.nbw) A(&w.wqkv_s, m->rc_qkv.tiles() * tile * m->esz);
      if (m->rc_o.nbw) A(&w.wo_s, m->rc_o.tiles() * tile * m->esz);
      if (m->rc_gu.nbw) A(&w.wgu_s, m->rc_gu.tiles() * tile * m->esz);
      if (m->rc_down.nbw) A(&w.wdown_s, m->rc_down.tiles() * tile * m->esz);
    }
  }
  A((void**)&m->x, (size_t)kMaxRows * m->d * 4);
  A((void**)&m->delta, (size_t)kMaxSplits * kMaxRows * m->d * 4);
  A((void**)&m->ssq, (size_t)m->Nb_o * kMaxRows * 4);
  A((void**)&m->ssq2, (size_t)m->Nb_down * kMaxRows * 4);
  A((void**)&m->gcnt, (size_t)(m->Nb_down + 64) * sizeof(int));
  if (st == DSI_OK) m->pk_d = make_pack(m, m->Kb_d, &st);
  if (st == DSI_OK) m->pk_q = make_pack(m, m->Kb_q, &st);
  if (st == DSI_OK) m->pk_ff = make_pack(m, m->Kb_ff, &st);
  A((void**)&m->qbuf, (size_t)kMaxRows * m->qdim * 4);
  A((void**)&m->rope, (size_t)kMaxRows * (m->hd / 2) * sizeof(float2));
  A((void**)&m->logits, (size_t)kMaxRows * m->V * 4);
  A(&m->vws, verify_workspace_bytes(kMaxRows, kMaxRows, m->V));
  A(&m->dws, draft_workspace_bytes(m->V));
  A((void**)&m->tdepth, (size_t)kMaxRows * sizeof(int));
  A((void**)&m->tanc, (size_t)kMaxRows * sizeof(unsigned long long));
  A((void**)&m->tbad, (size_t)kMaxRows * sizeof(int));
  A((void**)&m->tdec, (size_t)kMaxRows * sizeof(int4));

  A((void**)&m->err, 64);
  if (st != DSI_OK) {
    free_list(m->allocs);
    delete m;
    return st;
  }
  *out = m;
  return DSI_OK;
}

dsi_status dsi_model_destroy(dsi_model* m) {
  if (!m) return DSI_OK;
  if (m->live_kv) return fail(DSI_ESTATE, "destroy the model's KV caches first");
  hipStreamSynchronize(m->stream);
  for (auto& g : m->graphs) hipGraphExecDestroy(g.exec);
  for (hipEvent_t e : m->prof_ev) hipEventDestroy(e);
  free_list(m->allocs);
  if (m->attn_o.p) hipFree(m->attn_o.p);
  if (m->attn_ml.p) hipFree(m->attn_ml.p);
  delete m;
  return DSI_OK;
}

dsi_status dsi_model_set_tensor(dsi_model* m, int32_t layer, int32_t id, const void* src, size_t nbytes,
                                int32_t src_on_device) {
  if (!m || !src) return fail(DSI_EINVAL, "null argument");
  const bool global = id == DSI_T_EMBED || id == DSI_T_FINAL_NORM || id == DSI_T_LM_HEAD;
  if (id < 0 || id > DSI_T_W_DOWN) return fail(DSI_EINVAL, "bad tensor id %d", id);
  if (global ? layer != -1 : (layer < 0 || layer >= m->L))
    return fail(DSI_EINVAL, "bad layer %d for tensor %d", layer, id);
  size_t rows = 1, cols = 1;
  switch (id) {
    case DSI_T_EMBED: case DSI_T_LM_HEAD: rows = m->V; cols = m->d; break;
    case DSI_T_FINAL_NORM: case DSI_T_ATTN_NORM: case DSI_T_FFN_NORM: rows = 1; cols = m->d; break;
    case DSI_T_WQ: rows = m->qdim; cols = m->d; break;
    case DSI_T_WK: case DSI_T_WV: rows = m->kvdim; cols = m->d; break;
    case DSI_T_WO: rows = m->d; cols = m->qdim; break;
    case DSI_T_W_GATE: case DSI_T_W_UP: rows = m->ff; cols = m->d; break;
    case DSI_T_W_DOWN: rows = m->d; cols = m->ff; break;
  }
  if (nbytes != rows * cols * m->esz)
    return fail(DSI_EINVAL, "tensor %d: expected %zu bytes, got %zu", id, rows * cols * m->esz, nbytes);
  const hipMemcpyKind kind = src_on_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;

  if (id == DSI_T_FINAL_NORM || id == DSI_T_ATTN_NORM || id == DSI_T_FFN_NORM) {
    std::vector<unsigned char> hbuf(nbytes);
    if (src_on_device) HIP_TRY(hipMemcpy(hbuf.data(), src, nbytes, hipMemcpyDeviceToHost));
    else memcpy(hbuf.data(), src, nbytes);
    std::vector<float> g(m->d);
    for (int i = 0; i < m->d; ++i) {
      if (m->wtype == W_BF16) {
        uint16_t b;
        memcpy(&b, hbuf.data() + 2 * i, 2);
        uint32_t u = (uint32_t)b << 16;
        memcpy(&g[i], &u, 4);
      } else {
        memcpy(&g[i], hbuf.data() + 4 * i, 4);
      }
    }
    float* dst = id == DSI_T_FINAL_NORM ? m->final_norm
                 : id == DSI_T_ATTN_NORM ? m->layers[layer].attn_norm : m->layers[layer].ffn_norm;
    HIP_TRY(hipMemcpy(dst, g.data(), (size_t)m->d * 4, hipMemcpyHostToDevice));
  } else if (id == DSI_T_EMBED) {
    HIP_TRY(hipMemcpy(m->embed, src, nbytes, kind));
  } else {
    const void* dsrc = src;
    void* staging = nullptr;
    if (!src_on_device) {
      hipError_t e = hipMalloc(&staging, nbytes);
      if (e != hipSuccess) {
        hipGetLastError();
        return fail(DSI_ENOMEM, "staging hipMalloc(%zu) failed", nbytes);
      }
      e = hipMemcpy(staging, src, nbytes, hipMemcpyHostToDevice);
      if (e != hipSuccess) {
        hipFree(staging);
        return fail(DSI_EHIP, "hipMemcpy: %s", hipGetErrorString(e));
      }
      dsrc = staging;
    }
    hipError_t e = hipSuccess;
    LayerW* lw = global ? nullptr : &m->layers[layer];
    const int nq = m->qdim / 16, nk = m->kvdim / 16;
    switch (id) {
      case DSI_T_LM_HEAD:
        e = launch_prepack(m->wtype, dsrc, m->V, m->d, m->lm_head, m->Kb_d, 0, 0, m->hd, 0, m->Nb_head, m->G_head,
                           nullptr);
        break;
      case DSI_T_WQ:
        e = launch_prepack(m->wtype, dsrc, m->qdim, m->d, lw->wqkv, m->Kb_d, 0, 1, m->hd, 0, m->Nb_qkv, 1, nullptr);
        break;
      case DSI_T_WK:
        e = launch_prepack(m->wtype, dsrc, m->kvdim, m->d, lw->wqkv, m->Kb_d, nq, 1, m->hd, 0, m->Nb_qkv, 1, nullptr);
        break;
      case DSI_T_WV:
        e = launch_prepack(m->wtype, dsrc, m->kvdim, m->d, lw->wqkv, m->Kb_d, nq + nk, 0, m->hd, 0, m->Nb_qkv, 1,
                           nullptr);
        break;
      case DSI_T_WO:
        e = launch_prepack(m->wtype, dsrc, m->d, m->qdim, lw->wo, m->Kb_q, 0, 0, m->hd, 0, m->Nb_o, 1, nullptr);
        break;
      case DSI_T_W_GATE:
        e = launch_prepack(m->wtype, dsrc, m->ff, m->d, lw->wgu, m->Kb_d, 0, 2, m->hd, 0, m->Nb_gu, m->G_gu, nullptr);
        break;
      case DSI_T_W_UP:
        e = launch_prepack(m->wtype, dsrc, m->ff, m->d, lw->wgu, m->Kb_d, 0, 2, m->hd, 1, m->Nb_gu, m->G_gu, nullptr);
        break;
      case DSI_T_W_DOWN:
        e = launch_prepack(m->wtype, dsrc, m->d, m->ff, lw->wdown, m->Kb_ff, 0, 0, m->hd, 0, m->Nb_down, 1, nullptr);
        break;
    }
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (staging) hipFree(staging);
    if (e != hipSuccess) return fail(DSI_EHIP, "prepack: %s", hipGetErrorString(e));
  }
  m->set_mask[global ? 0 : layer + 1] |= 1u << id;
  if (id == DSI_T_LM_HEAD && m->lm_head_s) {
    hipError_t e = launch_restream(m->lm_head, m->Nb_head, m->Kb_d, m->G_head, m->rc_head, m->lm_head_s, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail(DSI_EHIP, "ring layout: %s", hipGetErrorString(e));
  }
  if (!global) {
    // once every part of a role's matrix is packed, lay it out for the ring
    // kernel as well
    const unsigned have = m->set_mask[layer + 1];
    LayerW& lw = m->layers[layer];
    hipError_t e = hipSuccess;
    const unsigned qkv = (1u << DSI_T_WQ) | (1u << DSI_T_WK) | (1u << DSI_T_WV);
    const unsigned gu = (1u << DSI_T_W_GATE) | (1u << DSI_T_W_UP);
    if ((id == DSI_T_WQ || id == DSI_T_WK || id == DSI_T_WV) && (have & qkv) == qkv && lw.wqkv_s)
      e = launch_restream(lw.wqkv, m->Nb_qkv, m->Kb_d, 1, m->rc_qkv, lw.wqkv_s, nullptr);
    else if (id == DSI_T_WO && lw.wo_s)
      e = launch_restream(lw.wo, m->Nb_o, m->Kb_q, 1, m->rc_o, lw.wo_s, nullptr);
    else if ((id == DSI_T_W_GATE || id == DSI_T_W_UP) && (have & gu) == gu && lw.wgu_s)
      e = launch_restream(lw.wgu, m->Nb_gu, m->Kb_d, m->G_gu, m->rc_gu, lw.wgu_s, nullptr);
    else if (id == DSI_T_W_DOWN && lw.wdown_s)
      e = launch_restream(lw.wdown, m->Nb_down, m->Kb_ff, 1, m->rc_down, lw.wdown_s, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return fail(DSI_EHIP, "ring layout: %s", hipGetErrorString(e));
  }
  return DSI_OK;
}

dsi_status dsi_kv_create(dsi_model* m, int32_t n_windows, int32_t max_len, dsi_kv** out) {
  if (!m || !out) return fail(DSI_EINVAL, "null argument");
  if (n_windows < 1 || max_len < 1) return fail(DSI_EINVAL, "n_windows and max_len must be >= 1");
  dsi_kv* kv = new (std::nothrow) dsi_kv();
  if (!kv) return fail(DSI_ENOMEM, "host allocation failed");
  kv->m = m;
  kv->n_windows = n_windows;
  kv->max_len = max_len;
  kv->maxlen_pad = (int)round_up((size_t)max_len, 64);
  kv->win_elems = (size_t)m->hkv * kv->maxlen_pad * m->hd;
  kv->hi.assign(n_windows, 0);
  kv->lo.assign(n_windows, 0);
  const size_t bytes = (size_t)m->L * n_windows * kv->win_elems * m->kvesz;
  std::vector<void*> list;
  dsi_status st = dev_alloc(list, &kv->k, bytes);
  if (st == DSI_OK) st = dev_alloc(list, &kv->v, bytes);
  if (st == DSI_OK) st = dev_alloc(list, (void**)&kv->lens, (size_t)n_windows * sizeof(int));
  if (st != DSI_OK) {
    free_list(list);
    delete kv;
    return st;
  }
  m->live_kv++;
  *out = kv;
  return DSI_OK;
}

dsi_status dsi_kv_destroy(dsi_kv* kv) {
  if (!kv) return DSI_OK;
  hipStreamSynchronize(kv->m->stream);
  hipFree(kv->k);
  hipFree(kv->v);
  hipFree(kv->lens);
  kv->m->live_kv--;
  delete kv;
  return DSI_OK;
}

dsi_status dsi_prefill(dsi_model* m, dsi_kv* kv, int32_t window, const int32_t* d_tokens, int32_t n,
                       float* d_last_logits) {
  if (!m || !kv || kv->m != m) return fail(DSI_EINVAL, "model / kv mismatch");
  if (window < 0 || window >= kv->n_windows) return fail(DSI_EINVAL, "bad window %d", window);
  if (n < 0 || (n > 0 && !d_tokens)) return fail(DSI_EINVAL, "bad token count / pointer");
  if (!all_set(m)) return fail(DSI_ESTATE, "not every model tensor has been set");
  if (kv->hi[window] + n > kv->max_len)
    return fail(DSI_ECAPACITY, "window %d: length (<= %lld) + %d exceeds max_len %d", window,
                kv->hi[window], n, kv->max_len);
  for (int off = 0; off < n; off += kMaxRows) {
    const int rows = std::min(kMaxRows, n - off);
    const bool last = off + rows == n;
    AttnPlan ap;
    DSI_TRY(plan_attention(m, kv, window, 1, rows, &ap));
    DSI_TRY(run_forward(m, kv, ap, window, 1, rows, d_tokens + off, last ? d_last_logits : nullptr, 1,
                        nullptr));
    HIP_TRY(launch_kv_add_checked(kv->lens, window, d_tokens + off, rows, m->V, m->err, m->stream));
    kv->hi[window] += rows;
  }
  return DSI_OK;
}

dsi_status dsi_verify(dsi_model* m, dsi_kv* kv, const dsi_verify_args* a, int32_t* d_n_accepted,
                      int32_t* d_next_token) {
  if (!m || !kv || !a || kv->m != m) return fail(DSI_EINVAL, "null argument or model / kv mismatch");
  const int B = a->n_windows, k = a->k;
  DSI_TRY(verify_args_ok(B, k, m->V, a->d_tokens, a->d_q, a->d_u, a->temperature, a->mode,
                         d_n_accepted, d_next_token));
  if (a->window0 < 0 || a->window0 + B > kv->n_windows)
    return fail(DSI_EINVAL, "windows [%d, %d) outside the cache's %d", a->window0, a->window0 + B,
                kv->n_windows);
  if (!all_set(m)) return fail(DSI_ESTATE, "not every model tensor has been set");
  for (int b = 0; b < B; ++b)
    if (kv->hi[a->window0 + b] + k + 1 > kv->max_len)
      return fail(DSI_ECAPACITY, "window %d: length (<= %lld) + %d exceeds max_len %d", a->window0 + b,
                  kv->hi[a->window0 + b], k + 1, kv->max_len);
  float* logits = a->d_logits_out ? a->d_logits_out : m->logits;
  AttnPlan ap;
  DSI_TRY(plan_attention(m, kv, a->window0, B, k + 1, &ap));
  m->last_window0 = a->window0;
  m->last_B = B;
  m->last_R = k + 1;
  VerifyArgs va{};
  va.B = B;
  va.k = k;
  va.V = m->V;
  va.logits = logits;
  va.tokens = a->d_tokens;
  va.q = a->d_q;
  va.u = a->d_u;
  va.temperature = (double)a->temperature;
  va.greedy = a->mode == DSI_GREEDY;
  va.commit = a->commit;
  va.lens = kv->lens;
  va.window0 = a->window0;
  va.n_out = d_n_accepted;
  va.tok_out = d_next_token;
  va.err = m->err;
  verify_bind_workspace(va, m->vws, B * (k + 1), B, m->V);
  auto launches = [&]() -> dsi_status {
    DSI_TRY(run_forward(m, kv, ap, a->window0, B, k + 1, a->d_tokens, logits, 0, a->d_hidden_out));
    Prof p(m, DSI_K_VERIFY);
    HIP_TRY(launch_verify(va, m->stream));
    return DSI_OK;
  };
  if (m->use_graphs && m->prof_class == 0) {
    // every value the launches depend on (model-owned buffers are fixed for
    // the model's lifetime except the attention partials, which are keyed)
    uint32_t tbits;
    memcpy(&tbits, &a->temperature, 4);
    const std::vector<uint64_t> key = {
        1u, (uint64_t)a->window0, (uint64_t)B, (uint64_t)k, (uint64_t)(uintptr_t)a->d_tokens,
        (uint64_t)(uintptr_t)a->d_q, (uint64_t)(uintptr_t)a->d_u, tbits, (uint64_t)a->mode,
        (uint64_t)a->commit, (uint64_t)(uintptr_t)logits, (uint64_t)(uintptr_t)a->d_hidden_out,
        (uint64_t)(uintptr_t)d_n_accepted, (uint64_t)(uintptr_t)d_next_token,
        (uint64_t)(uintptr_t)kv->k, (uint64_t)(uintptr_t)kv->v, (uint64_t)(uintptr_t)kv->lens,
        (uint64_t)kv->n_windows, (uint64_t)kv->max_len, (uint64_t)kv->maxlen_pad,
        (uint64_t)ap.n_qtiles, (uint64_t)ap.chunk, (uint64_t)ap.n_chunks, (uint64_t)ap.waves,
        (uint64_t)(uintptr_t)m->attn_o.p, (uint64_t)(uintptr_t)m->attn_ml.p};
    DSI_TRY(replay_or_capture(m, key, launches));
  } else {
    DSI_TRY(launches());
  }
  if (a->commit)
    for (int b = 0; b < B; ++b) kv->hi[a->window0 + b] += k + 1;
  return DSI_OK;
}

dsi_status dsi_verify_tree(dsi_model* m, dsi_kv* kv, const dsi_tree_args* a, int32_t* d_path,
                           int32_t* d_n_accepted, int32_t* d_next_token) {
  if (!m || !kv || !a || kv->m != m) return fail(DSI_EINVAL, "null argument or model / kv mismatch");
  const int B = a->n_windows, R = a->n_nodes;
  if (B < 1) return fail(DSI_EINVAL, "n_windows must be >= 1");
  if (R < 1) return fail(DSI_EINVAL, "n_nodes must be >= 1");
  if ((long long)B * R > DSI_MAX_ROWS)
    return fail(DSI_EINVAL, "n_windows*n_nodes = %lld exceeds %d", (long long)B * R, DSI_MAX_ROWS);
  if (!a->d_tokens || !a->d_parent || !d_path || !d_n_accepted || !d_next_token)
    return fail(DSI_EINVAL, "null tokens, parents or output pointer");
  if (a->window0 < 0 || a->window0 + B > kv->n_windows)
    return fail(DSI_EINVAL, "windows [%d, %d) outside the cache's %d", a->window0, a->window0 + B,
                kv->n_windows);
  if (!all_set(m)) return fail(DSI_ESTATE, "not every model tensor has been set");
  for (int b = 0; b < B; ++b)
    if (kv->hi[a->window0 + b] + R > kv->max_len)
      return fail(DSI_ECAPACITY, "window %d: length (<= %lld) + %d exceeds max_len %d", a->window0 + b,
                  kv->hi[a->window0 + b], R, kv->max_len);
  float* logits = a->d_logits_out ? a->d_logits_out : m->logits;
  AttnPlan ap;
  DSI_TRY(plan_attention(m, kv, a->window0, B, R, &ap));
  m->last_window0 = a->window0;
  m->last_B = B;
  m->last_R = R;
  // row statistics of the greedy rule over all B*R node rows
  VerifyArgs va{};
  va.B = B;
  va.k = R - 1;
  va.V = m->V;
  va.logits = logits;
  va.temperature = 1.0;
  va.greedy = 1;
  verify_bind_workspace(va, m->vws, B * R, B, m->V);
  TreeArgs ta{};
  ta.B = B;
  ta.R = R;
  ta.V = m->V;
  ta.C = va.C;
  ta.tokens = a->d_tokens;
  ta.parent = a->d_parent;
  ta.depth = m->tdepth;
  ta.anc = m->tanc;
  ta.bad = m->tbad;
  ta.part_arg = va.part_arg;
  ta.path = d_path;
  ta.n_out = d_n_accepted;
  ta.tok_out = d_next_token;
  ta.commit = a->commit;
  ta.lens = kv->lens;
  ta.window0 = a->window0;
  ta.err = m->err;
  ta.decision = m->tdec;
  const size_t layer_elems = (size_t)kv->n_windows * kv->win_elems;
  auto launches = [&]() -> dsi_status {
    HIP_TRY(launch_tree_prep(ta, m->stream));
    DSI_TRY(run_forward(m, kv, ap, a->window0, B, R, a->d_tokens, logits, 0, nullptr, m->tdepth, m->tanc));
    Prof p(m, DSI_K_VERIFY);
    HIP_TRY(launch_verify_rowstats(va, m->stream));
    HIP_TRY(launch_tree_decide(ta, m->stream));
    if (a->commit)
      HIP_TRY(launch_tree_compact(ta, m->kvb, kv->k, kv->v, m->L, layer_elems, kv->win_elems, m->hkv, m->hd,
                                  kv->maxlen_pad, m->stream));
    return DSI_OK;
  };
  if (m->use_graphs && m->prof_class == 0) {
    const std::vector<uint64_t> key = {
        2u, (uint64_t)a->window0, (uint64_t)B, (uint64_t)R, (uint64_t)(uintptr_t)a->d_tokens,
        (uint64_t)(uintptr_t)a->d_parent, (uint64_t)a->commit, (uint64_t)(uintptr_t)logits,
        (uint64_t)(uintptr_t)d_path, (uint64_t)(uintptr_t)d_n_accepted, (uint64_t)(uintptr_t)d_next_token,
        (uint64_t)(uintptr_t)kv->k, (uint64_t)(uintptr_t)kv->v, (uint64_t)(uintptr_t)kv->lens,
        (uint64_t)kv->n_windows, (uint64_t)kv->max_len, (uint64_t)kv->maxlen_pad,
        (uint64_t)ap.n_qtiles, (uint64_t)ap.chunk, (uint64_t)ap.n_chunks, (uint64_t)ap.waves,
        (uint64_t)(uintptr_t)m->attn_o.p, (uint64_t)(uintptr_t)m->attn_ml.p};
    DSI_TRY(replay_or_capture(m, key, launches));
  } else {
    DSI_TRY(launches());
  }
  if (a->commit)
    for (int b = 0; b < B; ++b) kv->hi[a->window0 + b] += R;
  return DSI_OK;
}

dsi_status dsi_draft(dsi_model* m, dsi_kv* kv, int32_t window, const int32_t* d_feed, int32_t n_feed,
                     int32_t k, const float* d_u, float temperature, int32_t* d_tokens, float* d_q) {
  if (!m || !kv || kv->m != m) return fail(DSI_EINVAL, "model / kv mismatch");
  if (window < 0 || window >= kv->n_windows) return fail(DSI_EINVAL, "bad window %d", window);
  if (n_feed < 1 || n_feed > kMaxRows || !d_feed)
    return fail(DSI_EINVAL, "feed 1..%d tokens (got %d)", kMaxRows, n_feed);
  if (k < 1) return fail(DSI_EINVAL, "k must be >= 1");
  if (!d_u || !d_tokens || !d_q) return fail(DSI_EINVAL, "null uniforms / output pointer");
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return fail(DSI_EINVAL, "temperature must be > 0");
  if (!all_set(m)) return fail(DSI_ESTATE, "not every model tensor has been set");
  if (kv->hi[window] + n_feed + k - 1 > kv->max_len)
    return fail(DSI_ECAPACITY, "window %d: length (<= %lld) + %d exceeds max_len %d", window, kv->hi[window],
                n_feed + k - 1, kv->max_len);
  hipStream_t s = m->stream;
  // w0, the last fed token, opens the verification window
  HIP_TRY(hipMemcpyAsync(d_tokens, d_feed + n_feed - 1, sizeof(int32_t), hipMemcpyDeviceToDevice, s));
  for (int i = 0; i < k; ++i) {
    // step i forwards the unseen feed (i = 0) or the previous draft, whose
    // last row's logits give q_{i+1} and d_{i+1}
    const int* rows = i == 0 ? d_feed : d_tokens + i;
    const int R = i == 0 ? n_feed : 1;
    AttnPlan ap;
    DSI_TRY(plan_attention(m, kv, window, 1, R, &ap));
    DSI_TRY(run_forward(m, kv, ap, window, 1, R, rows, m->logits, 1, nullptr));
    HIP_TRY(launch_kv_add_checked(kv->lens, window, rows, R, m->V, m->err, s));
    kv->hi[window] += R;
    DraftArgs da{};
    da.logits = m->logits;
    da.V = m->V;
    da.temperature = (double)temperature;
    da.u = d_u + i;
    da.q_out = d_q + (size_t)i * m->V;
    da.tok_out = d_tokens + i + 1;
    HIP_TRY(launch_draft_sample(da, m->dws, s));
  }
  return DSI_OK;
}

dsi_status dsi_accept(void* stream, int32_t B, int32_t k, int32_t V, const float* d_logits,
                      const int32_t* d_tokens, const float* d_q, const float* d_u, float temperature,
                      int32_t mode, int32_t* d_n_accepted, int32_t* d_next_token) {
  DSI_TRY(verify_args_ok(B, k, V, d_tokens, d_q, d_u, temperature, mode, d_n_accepted, d_next_token));
  if (!d_logits) return fail(DSI_EINVAL, "null logits");
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  std::lock_guard<std::mutex> lk(g_accept_mu);
  AcceptWs& w = g_accept[dev];
  if (!w.err) {
    hipError_t e = hipMalloc((void**)&w.err, 64);
    if (e != hipSuccess) {
      hipGetLastError();
      w.err = nullptr;
      return fail(DSI_ENOMEM, "hipMalloc failed");
    }
    HIP_TRY(hipMemset(w.err, 0, 64));
  }
  DSI_TRY(ensure(w.ws, verify_workspace_bytes(B * (k + 1), B, V)));
  VerifyArgs va{};
  va.B = B;
  va.k = k;
  va.V = V;
  va.logits = d_logits;
  va.tokens = d_tokens;
  va.q = d_q;
  va.u = d_u;
  va.temperature = (double)temperature;
  va.greedy = mode == DSI_GREEDY;
  va.commit = 0;
  va.lens = nullptr;
  va.window0 = 0;
  va.n_out = d_n_accepted;
  va.tok_out = d_next_token;
  va.err = w.err;
  verify_bind_workspace(va, w.ws.p, B * (k + 1), B, V);
  HIP_TRY(launch_verify(va, (hipStream_t)stream));
  return DSI_OK;
}


dsi_status dsi_accept_noalloc(void* stream, int32_t B, int32_t k, int32_t V, const float* d_logits,
                              const int32_t* d_tokens, const float* d_q, const float* d_u,
                              float temperature, int32_t mode, int32_t* d_n_accepted,
                              int32_t* d_next_token) {
  DSI_TRY(verify_args_ok(B, k, V, d_tokens, d_q, d_u, temperature, mode, d_n_accepted, d_next_token));
  if (!d_logits) return fail(DSI_EINVAL, "null logits");
  const size_t need = verify_workspace_bytes(B * (k + 1), B, V);
  if (need > DSI_ACCEPT_NOALLOC_BYTES - kScratchHead)
    return fail(DSI_ECAPACITY,
                "dsi_accept_noalloc: %d rows over a vocabulary of %d need %zu workspace bytes; the "
                "fixed array holds %zu",
                B * (k + 1), V, need, (size_t)DSI_ACCEPT_NOALLOC_BYTES - kScratchHead);
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  void* base = nullptr;
  DSI_TRY(scratch_address(dev, &base));
  hipStream_t s = (hipStream_t)stream;
  // the error word accumulates with atomics: clear it (a fill kernel, so the
  // call stays capturable)
  HIP_TRY(launch_fill_zero(base, sizeof(int), s));
  VerifyArgs va{};
  va.B = B;
  va.k = k;
  va.V = V;
  va.logits = d_logits;
  va.tokens = d_tokens;
  va.q = d_q;
  va.u = d_u;
  va.temperature = (double)temperature;
  va.greedy = mode == DSI_GREEDY;
  va.commit = 0;
  va.lens = nullptr;
  va.window0 = 0;
  va.n_out = d_n_accepted;
  va.tok_out = d_next_token;
  va.err = (int*)base;
  verify_bind_workspace(va, (char*)base + kScratchHead, B * (k + 1), B, V);
  HIP_TRY(launch_verify(va, s));
  return DSI_OK;
}

dsi_status dsi_kv_rollback(dsi_kv* kv, int32_t window, int32_t new_len) {
  if (!kv) return fail(DSI_EINVAL, "null kv");
  if (window < 0 || window >= kv->n_windows) return fail(DSI_EINVAL, "bad window %d", window);
  if (new_len < 0 || new_len > kv->hi[window])
    return fail(DSI_EINVAL, "rollback to %d above the window's length (<= %lld)", new_len, kv->hi[window]);
  HIP_TRY(launch_kv_rollback(kv->lens, window, new_len, kv->m->err, kv->m->stream));
  kv->hi[window] = new_len;
  kv->lo[window] = std::min(kv->lo[window], (long long)new_len);
  return DSI_OK;
}

dsi_status dsi_kv_poison(dsi_kv* kv, int32_t window) {
  if (!kv) return fail(DSI_EINVAL, "null kv");
  if (window < 0 || window >= kv->n_windows) return fail(DSI_EINVAL, "bad window %d", window);
  dsi_model* m = kv->m;
  HIP_TRY(launch_kv_poison(m->kvb, kv_ptr(kv, kv->k, 0, window), kv_ptr(kv, kv->v, 0, window),
                           (size_t)kv->n_windows * kv->win_elems, m->L, m->hkv, m->hd, kv->maxlen_pad, kv->lens,
                           window, m->stream));
  return DSI_OK;
}

dsi_status dsi_kv_length(dsi_kv* kv, int32_t window, int32_t* len) {
  if (!kv || !len) return fail(DSI_EINVAL, "null argument");
  if (window < 0 || window >= kv->n_windows) return fail(DSI_EINVAL, "bad window %d", window);
  HIP_TRY(hipStreamSynchronize(kv->m->stream));
  int h = 0;
  HIP_TRY(hipMemcpy(&h, kv->lens + window, sizeof(int), hipMemcpyDeviceToHost));
  *len = h;
  kv->hi[window] = kv->lo[window] = h;
  return check_err_word(kv->m->err, kv->m->stream);
}

dsi_status dsi_profile_begin(dsi_model* m, int32_t kernel_class) {
  if (!m) return fail(DSI_EINVAL, "null model");
  if (kernel_class < DSI_K_QKV || kernel_class > DSI_K_VERIFY) return fail(DSI_EINVAL, "bad kernel class");
  HIP_TRY(hipStreamSynchronize(m->stream));
  m->prof_class = kernel_class;
  m->prof_used = 0;
  return DSI_OK;
}

dsi_status dsi_profile_end(dsi_model* m, int32_t* launches, double* total_ms) {
  if (!m || !launches || !total_ms) return fail(DSI_EINVAL, "null argument");
  HIP_TRY(hipStreamSynchronize(m->stream));
  double tot = 0.0;
  for (size_t i = 0; i + 1 < m->prof_used; i += 2) {
    float ms = 0.f;
    HIP_TRY(hipEventElapsedTime(&ms, m->prof_ev[i], m->prof_ev[i + 1]));
    tot += ms;
  }
  *launches = (int32_t)(m->prof_used / 2);
  *total_ms = tot;
  m->prof_class = 0;
  m->prof_used = 0;
  return DSI_OK;
}

dsi_status dsi_profile_stream(const void* d_buf, uint64_t bytes, int32_t slices, int32_t nontemporal,
                              int32_t workgroups, int32_t rounds, void* d_sink, uint64_t* bytes_per_launch,
                              double* avg_ms) {
  if (!d_buf || !d_sink || !bytes_per_launch || !avg_ms || rounds < 1 || slices < 1)
    return fail(DSI_EINVAL, "bad argument");
  if (workgroups < 0 || workgroups > kStreamMaxWorkgroups)
    return fail(DSI_EINVAL, "workgroups must be 0 (default %d) or 1..%d", kStreamWorkgroups, kStreamMaxWorkgroups);
  if (((uintptr_t)d_buf & 15) != 0) return fail(DSI_EINVAL, "buffer not 16-byte aligned");
  const int wgs = workgroups ? workgroups : kStreamWorkgroups;
  const uint64_t slice = bytes / (uint64_t)slices;
  const uint64_t waves = (uint64_t)wgs * 8;
  const uint64_t run = slice / waves / 8192 * 8192;   // bytes per wave: whole rings of 8 x 1 KB
  if (run < 8192 || slice < (16ull << 20)) return fail(DSI_EINVAL, "slices must hold at least 16 MiB");
  const size_t per_wave_vec = (size_t)(run / 16);
  hipEvent_t e0, e1;
  HIP_TRY(hipEventCreate(&e0));
  HIP_TRY(hipEventCreate(&e1));
  dsi_status st = DSI_OK;
  auto go = [&](int r) -> hipError_t {
    return launch_stream_read((const char*)d_buf + (size_t)(r % slices) * slice, per_wave_vec, wgs, nontemporal,
                              d_sink, nullptr);
  };
  hipError_t e = go(0);   // warm-up
  if (e == hipSuccess) e = hipEventRecord(e0, nullptr);
  for (int r = 1; r <= rounds && e == hipSuccess; ++r) e = go(r);
  if (e == hipSuccess) e = hipEventRecord(e1, nullptr);
  if (e == hipSuccess) e = hipEventSynchronize(e1);
  float ms = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&ms, e0, e1);
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  if (e != hipSuccess) st = fail(DSI_EHIP, "HIP error: %s", hipGetErrorString(e));
  if (st != DSI_OK) return st;
  *bytes_per_launch = run * waves;
  *avg_ms = (double)ms / rounds;
  return DSI_OK;
}

dsi_status dsi_profile_kernel(dsi_model* m, dsi_kv* kv, int32_t cls, int32_t rounds, int32_t* launches,
                              double* avg_ms) {
  if (!m || !kv || kv->m != m || !launches || !avg_ms || rounds < 1)
    return fail(DSI_EINVAL, "bad argument");
  if (m->last_B < 1 || m->last_window0 + m->last_B > kv->n_windows)
    return fail(DSI_ESTATE, "run dsi_verify on this cache first");
  if (cls != DSI_K_QKV && cls != DSI_K_OPROJ && cls != DSI_K_GATEUP && cls != DSI_K_DOWN && cls != DSI_K_HEAD)
    return fail(DSI_EINVAL, "kernel class %d is not a GEMM class", cls);
  const int M = m->last_B * m->last_R, mt = cdiv(M, 16);
  const size_t dstride = (size_t)kMaxRows * m->d;
  hipStream_t s = m->stream;
  const RowMap rows{kv->lens, m->last_window0, m->last_R};
  const bool ring = ring_forward(m, kv, mt);
  auto one = [&](int l) -> dsi_status {
    GemmArgs g;
    switch (cls) {
      case DSI_K_QKV: g = qkv_args(m, kv, l, M, rows, ring); break;
      case DSI_K_OPROJ: g = oproj_args(m, l, M, ring); break;
      case DSI_K_GATEUP: g = gateup_args(m, l, M, ring); break;
      case DSI_K_DOWN: g = down_args(m, l, M, mt, nullptr, ring); break;
      default: g = head_args(m, m->logits, M, ring); break;
    }
    HIP_TRY(launch_gemm(m->wtype, mt, g, s));
    return DSI_OK;
  };
  const int per_round = cls == DSI_K_HEAD ? 1 : m->L;
  DSI_TRY(one(cls == DSI_K_HEAD ? -1 : 0));   // warm-up launch
  hipEvent_t e0, e1;
  HIP_TRY(hipEventCreate(&e0));
  HIP_TRY(hipEventCreate(&e1));
  HIP_TRY(hipEventRecord(e0, s));
  for (int r = 0; r < rounds; ++r)
    for (int l = 0; l < per_round; ++l) DSI_TRY(one(cls == DSI_K_HEAD ? -1 : l));
  HIP_TRY(hipEventRecord(e1, s));
  HIP_TRY(hipEventSynchronize(e1));
  float ms = 0.f;
  HIP_TRY(hipEventElapsedTime(&ms, e0, e1));
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  *launches = rounds * per_round;
  *avg_ms = (double)ms / (rounds * per_round);
  return DSI_OK;
}

dsi_status dsi_sync(dsi_model* m) {
  if (!m) return fail(DSI_EINVAL, "null model");
  return check_err_word(m->err, m->stream);
}

static dsi_status kv_copy(dsi_kv* kv, int32_t window, int32_t layer, int32_t len, void* dk, void* dv,
                          int to_cache) {
  if (!kv || !dk || !dv) return fail(DSI_EINVAL, "null argument");
  dsi_model* m = kv->m;
  if (window < 0 || window >= kv->n_windows || layer < 0 || layer >= m->L || len < 0 || len > kv->max_len)
    return fail(DSI_EINVAL, "bad window / layer / len");
  HIP_TRY(launch_kv_copy(to_cache, m->kvb, kv_ptr(kv, kv->k, layer, window), kv_ptr(kv, kv->v, layer, window),
                         m->hkv, m->hd, kv->maxlen_pad, len, dk, dv, m->stream));
  return DSI_OK;
}

dsi_status dsi_kv_export(dsi_kv* kv, int32_t window, int32_t layer, int32_t len, void* d_k, void* d_v) {
  return kv_copy(kv, window, layer, len, d_k, d_v, 0);
}

dsi_status dsi_kv_import(dsi_kv* kv, int32_t window, int32_t layer, int32_t len, const void* d_k,
                         const void* d_v) {
  return kv_copy(kv, window, layer, len, (void*)d_k, (void*)d_v, 1);
}

dsi_status dsi_kv_set_length(dsi_kv* kv, int32_t window, int32_t len) {
  if (!kv) return fail(DSI_EINVAL, "null kv");
  if (window < 0 || window >= kv->n_windows || len < 0 || len > kv->max_len)
    return fail(DSI_EINVAL, "bad window / len");
  HIP_TRY(launch_kv_set(kv->lens, window, len, kv->m->stream));
  kv->hi[window] = kv->lo[window] = len;
  return DSI_OK;
}

}  // extern "C"
