// Host engine behind the C ABI (include/chimera.h): weight repacking, arena
// carving, paged-KV page tables, static tree metadata, and the launch
// sequence of prefill and of one draft -> verify -> accept -> compact step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <stdexcept>
#include <string>
#include <vector>

#include "chimera.h"
#include "kernels.h"

namespace {

thread_local std::string g_err;

struct Err : std::runtime_error {
  chimera_status st;
  Err(chimera_status s, const std::string& m) : std::runtime_error(m), st(s) {}
};

#define HIPCK(x)                                                                          \
  do {                                                                                    \
    hipError_t e_ = (x);                                                                  \
    if (e_ != hipSuccess) throw Err(CHIMERA_EHIP, std::string(#x) + ": " + hipGetErrorString(e_)); \
  } while (0)
#define REQUIRE(c, st, msg) \
  do {                      \
    if (!(c)) throw Err(st, msg); \
  } while (0)

template <class F>
chimera_status guard(F&& f) {
  try {
    f();
    return CHIMERA_OK;
  } catch (const Err& e) {
    g_err = e.what();
    return e.st;
  } catch (const std::exception& e) {
    g_err = e.what();
    return CHIMERA_EINVAL;
  } catch (...) {
    g_err = "unknown error";
    return CHIMERA_EINVAL;
  }
}

// Bump allocator over a caller arena; with base == nullptr it only sizes.
struct Arena {
  char* base;
  size_t size;
  size_t off = 0;
  void* take(size_t bytes) {
    off = (off + 255) / 256 * 256;
    if (base != nullptr) REQUIRE(off + bytes <= size, CHIMERA_ENOMEM, "arena too small");
    void* p = base ? base + off : nullptr;
    off += bytes;
    return p;
  }
  template <class T>
  T* arr(size_t n) { return static_cast<T*>(take(n * sizeof(T))); }
};

size_t esize(int dt) { return dt == CHIMERA_BF16 ? 2 : 4; }

// Row capacity of a tiled GEMM-input buffer that may hold up to m rows: a
// launch with m rows reads 16-row tiles in groups of 1, 2 or 4.
// Rows of an activation buffer: whole tiles of the GEMM row blocks that
// read it (16, 32, 64, then 128-row blocks).
int mcap(int m) { return m <= 16 ? 16 : (m <= 32 ? 32 : (m <= 64 ? 64 : (m + 127) / 128 * 128)); }

struct BlockW {
  float* attn_norm = nullptr;
  void* wqkv = nullptr;
  void* wo = nullptr;
  float* ffn_norm = nullptr;
  void* wgu = nullptr;
  void* wdown = nullptr;
};

void validate_config(const chimera_config* c) {
  REQUIRE(c != nullptr, CHIMERA_EINVAL, "null config");
  REQUIRE(c->dtype == CHIMERA_F32 || c->dtype == CHIMERA_BF16, CHIMERA_EINVAL, "dtype");
  REQUIRE(c->n_layers >= 1 && c->n_heads >= 1, CHIMERA_EINVAL, "layers/heads");
  REQUIRE(c->head_dim == 64 || c->head_dim == 128, CHIMERA_EINVAL, "head_dim must be 64 or 128");
  REQUIRE(c->n_heads * c->head_dim == c->d_model, CHIMERA_EINVAL, "n_heads * head_dim != d_model");
  REQUIRE(c->d_model % 256 == 0 && c->d_model <= 8192, CHIMERA_EINVAL, "d_model must be a multiple of 256, <= 8192");
  REQUIRE(c->d_ffn % 64 == 0, CHIMERA_EINVAL, "d_ffn must be a multiple of 64");
  REQUIRE(c->vocab % 64 == 0 && c->vocab >= 64, CHIMERA_EINVAL, "vocab must be a multiple of 64");
  REQUIRE(c->n_draft_heads >= 0 && c->n_draft_heads <= 8, CHIMERA_EINVAL, "n_draft_heads in [0, 8]");
  REQUIRE(c->max_positions >= 16, CHIMERA_EINVAL, "max_positions");
  REQUIRE(c->rms_eps > 0.f && c->rope_base > 1.f, CHIMERA_EINVAL, "eps/base");
}

}  // namespace

struct chimera_model {
  chimera_config cfg{};
  int dt = 0;
  size_t es = 4;
  void* embed = nullptr;
  std::vector<BlockW> layers;
  BlockW enc;
  float* final_norm = nullptr;
  void* lm_head = nullptr;
  void* tri_w1 = nullptr;
  void* tri_w2 = nullptr;
  std::vector<void*> head_a, head_theta;
  float* rcos = nullptr;
  float* rsin = nullptr;
};

// Encoder memory per sequence and stream: positions 0 .. max_len + 63, then
// (stream 1) one slot per draft-tree node for the speculative trigram entries.
constexpr int ENC_TREE_SLOTS = 64;

struct chimera_kv {
  chimera_model* m = nullptr;
  int B = 0, max_len = 0, n_pages = 0, ps = 0, max_pages = 0, cap = 0;
  void* pool = nullptr;
  int64_t page_stride = 0, layer_stride = 0;
  int* page_table = nullptr;  // device [B][max_pages]
  std::vector<int> page_table_host;
  void* enc_k = nullptr;
  void* enc_v = nullptr;
};

namespace {

struct TreeMeta {
  int* parent = nullptr;
  int* depth = nullptr;
  int* rank = nullptr;
  unsigned long long* anc = nullptr;
  uint8_t* path = nullptr;  // [64][64]
};

struct Event2 {
  hipEvent_t a, b;
};

}  // namespace

struct chimera_ctx {
  chimera_model* m = nullptr;
  chimera_kv* kv = nullptr;
  int B = 0, N = 0, K = 0, D = 0, Mv = 0, Md = 0, Mq = 0, G = 0, nblk_enc = 0, tok_stride = 0;
  std::vector<int> parent, rank, depth, s_k;
  std::vector<unsigned long long> anc;
  TreeMeta tree, chain;
  // drafting plan (chimera_set_drafting): chain (0) or branch-conditioned (1)
  int branch = 0;
  std::vector<int> lvl_R, lvl_off;  // drafted nodes per sequence and their offset in d_nodes, per level
  int* d_nodes = nullptr;           // [64]
  int* tok_src = nullptr;           // [64]
  // state
  int* n = nullptr;
  int* tok = nullptr;
  void* h_last = nullptr;
  int* cand = nullptr;
  int* tree_tok = nullptr;
  int* inject = nullptr;
  int* inject_on = nullptr;
  int* s_k_dev = nullptr;
  int* out_tok = nullptr;
  int* out_nodes = nullptr;
  int* out_len = nullptr;
  int* pro_base = nullptr;
  int* pro_count = nullptr;
  void* pro_h = nullptr;
  int* pf_n = nullptr;
  int* pf_tokens = nullptr;
  // verify workspaces
  float* x = nullptr;
  void* xn = nullptr;
  void* q = nullptr;
  void* attn = nullptr;
  void* hbuf = nullptr;
  float* parts = nullptr;
  float* scratch = nullptr;
  float* logits = nullptr;
  int* amax = nullptr;
  void* hl = nullptr;      // tiled (LM head input)
  void* hl_rm = nullptr;   // row-major copy (decode state)
  int mt_v = 0, mt_d = 0, mt_q = 0;  // 16-row tiles of the verify, draft-row and draft-query buffers
  float* part_o = nullptr;
  float* part_ml = nullptr;
  int* v_pos = nullptr;
  int64_t* v_kvoff = nullptr;
  int64_t* rowtab = nullptr;  // [B][TREE_ATTN_TAIL_ROWS]: window rows of the current verify pass
  // trigram lookup cache (attached by chimera_set_trigram_cache; hit/miss/stats live in this arena)
  TriCache tri;
  bool tri_on = false;
  // compaction check (debug mode): counters then the tree K/V copy, in a
  // caller-owned arena; nullptr = off
  unsigned long long* cc_counts = nullptr;
  void* cc_side = nullptr;
  // decoding: greedy, or typical acceptance with sampling (chimera_set_decoding)
  int typical = 0;
  float temperature = 1.f, t_eps = 0.09f, t_delta = 0.3f;
  unsigned long long t_seed = 0;
  double* t_lse = nullptr;  // [Mv]
  double* t_H = nullptr;    // [Mv]
  int* t_sample = nullptr;  // [Mv]
  int* v_qrow = nullptr;
  // draft workspaces
  void* tri_in = nullptr;
  void* tri_a = nullptr;
  float* htri = nullptr;
  void* un = nullptr;
  int* d_pos = nullptr;
  int64_t* d_kvoff = nullptr;
  int* d_qrow = nullptr;
  void* qc = nullptr;
  void* attn_c = nullptr;
  void* yn = nullptr;
  void* hc = nullptr;
  void* zin = nullptr;
  void* ak = nullptr;
  float* dlogits = nullptr;
  float* dparts = nullptr;
  float* enc_part = nullptr;
  float* topk_v = nullptr;
  int* topk_i = nullptr;
  // host side
  int batch = 0;
  std::vector<int> n_host;
  bool poisoned = false;
  const int* f_ref = nullptr;
  const uint8_t* f_ok = nullptr;
  int f_stride = 0;
  // Step results, one contiguous device block copied back by one transfer:
  // out_tok [B][K+1], out_nodes [B][K+1], out_len [B] (K = the depth the
  // context was sized for).
  char* result = nullptr;
  char* host_result = nullptr;  // pinned mirror
  char* host_pipe = nullptr;    // pinned [CHIMERA_MAX_PIPELINED_STEPS] result blocks (chimera_steps)
  size_t res_bytes = 0, res_nodes_off = 0, res_len_off = 0;
  // profiling
  bool prof = false;
  std::vector<Event2> ev_pool;
  size_t ev_used = 0;
  std::vector<double> ev_bytes;
  unsigned long long* stamp_ring = nullptr;  // device [STAMP_RING][STAMP_WORDS], one slot per step
  unsigned int* stamp_count = nullptr;       // device: steps stamped so far
  unsigned int prof_first = 0;               // stamp_count at the previous chimera_profile_read
  double clock_khz = 0.0;
  bool ev_created = false;
  chimera_profile acc{};
  // the step as a HIP graph, replayed every step
  bool graph_on = true;
  hipGraph_t graph = nullptr;
  hipGraphExec_t gexec = nullptr;
  bool capturing = false;  // chimera_step is capturing its launch sequence
  hipStream_t graph_stream = nullptr;
  size_t graph_ev_used = 0;
};

namespace {

// ---------------------------------------------------------------------------
// Model layout
// ---------------------------------------------------------------------------
void carve_block(const chimera_config& c, size_t es, Arena& a, BlockW& w) {
  const size_t d = c.d_model, hd = (size_t)c.n_heads * c.head_dim, F = c.d_ffn;
  w.attn_norm = a.arr<float>(d);
  w.wqkv = a.take(d * 3 * hd * es);
  w.wo = a.take(hd * d * es);
  w.ffn_norm = a.arr<float>(d);
  w.wgu = a.take(d * 2 * F * es);
  w.wdown = a.take(F * d * es);
}

void carve_model(const chimera_config& c, Arena& a, chimera_model& m) {
  const size_t es = esize(c.dtype), d = c.d_model, V = c.vocab;
  m.embed = a.take(V * d * es);
  m.layers.assign(c.n_layers, BlockW{});
  for (auto& l : m.layers) carve_block(c, es, a, l);
  m.final_norm = a.arr<float>(d);
  m.lm_head = a.take(d * V * es);
  m.tri_w1 = a.take(3 * d * d * es);
  m.tri_w2 = a.take(d * d * es);
  carve_block(c, es, a, m.enc);
  m.head_a.assign(c.n_draft_heads, nullptr);
  m.head_theta.assign(c.n_draft_heads, nullptr);
  for (int k = 0; k < c.n_draft_heads; ++k) {
    m.head_a[k] = a.take(2 * d * d * es);
    m.head_theta[k] = a.take(d * V * es);
  }
  m.rcos = a.arr<float>((size_t)c.max_positions * (c.head_dim / 2));
  m.rsin = a.arr<float>((size_t)c.max_positions * (c.head_dim / 2));
}

struct TensorSrc {
  const chimera_tensor* t = nullptr;
  int64_t numel = 0;
};

// ---------------------------------------------------------------------------
// Launch helpers
// ---------------------------------------------------------------------------
struct Gemm {
  chimera_ctx* c;
  hipStream_t st;
  bool timed;  // record events around the launch (verify GEMMs while profiling)

  void run(const void* X, int x_mtiles, int M, const void* W, int N, int K, GemmEpi e, int nb_off = 0,
           int nb_count = 0, const int* skip = nullptr) const {
    GemmShape s;
    s.X = X;
    s.x_mtiles = x_mtiles;
    s.M = M;
    s.W = W;
    s.N = N;
    s.K = K;
    s.nb_off = nb_off;
    s.nb_count = nb_count;
    s.skip = skip;
    const int cols = nb_count ? nb_count * 16 : N;
    s.splits = gemm_pick_splits(cols, K, c->m->dt);
    const int tiles_read = M <= 16 ? 1 : (M <= 32 ? 2 : 4 * ((M + 63) / 64));
    REQUIRE(tiles_read <= x_mtiles, CHIMERA_EINVAL, "GEMM rows exceed the input buffer");
    if (e.kind != EPI_PARTIAL) e.part = c->scratch;
    Event2* ev = nullptr;
    // per-launch events only for eager launches; a captured graph keeps the
    // phase stamps alone (querying the capture state for every launch while
    // capturing made the replayed graph slower)
    if (timed && c->prof && !c->capturing && c->ev_created && c->ev_used < c->ev_pool.size()) {
      ev = &c->ev_pool[c->ev_used];
      const double es = (double)c->m->es;
      c->ev_bytes[c->ev_used] = (double)K * cols * es + (double)M * K * es + (double)M * cols * 4.0;
      c->ev_used++;
    }
    if (ev)  // the kernels record the events at their own start and end
      launch_gemm(c->m->dt, s, e, st, ev->a, ev->b);
    else
      launch_gemm(c->m->dt, s, e, st);
  }
  int splits(int N, int K) const { return gemm_pick_splits(N, K, c->m->dt); }
};

struct VerifyRows {
  const int* tokens;
  int M;
  const int* n_b;
  const int* page_table;
  const int* depth;
  const uint8_t* path;
  int N, D, B;
};

// Target layer stack over M rows; leaves the post-final-norm states in c->hl.
void verify_layers(chimera_ctx* c, const VerifyRows& r, hipStream_t st, bool timed) {
  chimera_model* m = c->m;
  chimera_kv* kv = c->kv;
  const chimera_config& cf = m->cfg;
  const int dt = m->dt, d = cf.d_model, F = cf.d_ffn, H = cf.n_heads, hd = cf.head_dim;
  const int hdim = H * hd;
  const Gemm g{c, st, timed};
  launch_embed(dt, r.tokens, m->embed, c->x, r.M, d, cf.vocab, st);
  launch_attn_rows(r.n_b, r.page_table, kv->max_pages, kv->ps, kv->page_stride, hd, r.N, r.B, c->rowtab, st);
  int nparts = 0;
  for (int l = 0; l < cf.n_layers; ++l) {
    const BlockW& w = m->layers[l];
    launch_rmsnorm(dt, c->x, nparts ? c->parts : nullptr, nparts, w.attn_norm, c->xn, c->mt_v, nullptr, r.M, d,
                   cf.rms_eps, 1, nullptr, 0, 0, st);
    char* kbase = (char*)kv->pool + (size_t)l * kv->layer_stride * m->es;
    char* vbase = kbase + (size_t)H * kv->ps * hd * m->es;
    GemmEpi e;
    e.kind = EPI_QKV;
    e.pos = c->v_pos;
    e.kvoff = c->v_kvoff;
    e.qrow = c->v_qrow;
    e.kbase = kbase;
    e.vbase = vbase;
    e.head_stride = (int64_t)kv->ps * hd;
    e.qout = c->q;
    e.ldq = hdim;
    e.rcos = m->rcos;
    e.rsin = m->rsin;
    e.H = H;
    e.hd = hd;
    g.run(c->xn, c->mt_v, r.M, w.wqkv, 3 * hdim, d, e);

    TreeAttnArgs a{};
    a.q = c->q;
    a.ldq = hdim;
    a.kpool = kbase;
    a.vpool = vbase;
    a.page_stride = kv->page_stride;
    a.page_table = r.page_table;
    a.max_pages = kv->max_pages;
    a.n_b = r.n_b;
    a.depth = r.depth;
    a.path = r.path;
    a.N = r.N;
    a.H = H;
    a.hd = hd;
    a.ps = kv->ps;
    a.D = r.D;
    a.scale = 1.0f / std::sqrt((float)hd);
    a.part_o = c->part_o;
    a.part_ml = c->part_ml;
    a.G = c->G;
    a.out = c->attn;
    a.o_mtiles = c->mt_v;
    a.B = r.B;
    a.rowtab = c->rowtab;
    launch_tree_attn(dt, a, st);

    GemmEpi eo;
    eo.kind = EPI_PARTIAL;
    eo.part = c->parts;
    g.run(c->attn, c->mt_v, r.M, w.wo, d, hdim, eo);
    nparts = g.splits(d, hdim);
    launch_rmsnorm(dt, c->x, c->parts, nparts, w.ffn_norm, c->xn, c->mt_v, nullptr, r.M, d, cf.rms_eps, 1, nullptr, 0,
                   0, st);
    GemmEpi egu;
    egu.kind = EPI_SWIGLU;
    egu.out_t = c->hbuf;
    egu.o_mtiles = c->mt_v;
    g.run(c->xn, c->mt_v, r.M, w.wgu, 2 * F, d, egu);
    GemmEpi ed;
    ed.kind = EPI_PARTIAL;
    ed.part = c->parts;
    g.run(c->hbuf, c->mt_v, r.M, w.wdown, d, F, ed);
    nparts = g.splits(d, F);
  }
  launch_rmsnorm(dt, c->x, c->parts, nparts, m->final_norm, c->hl, c->mt_v, c->hl_rm, r.M, d, cf.rms_eps, 1, nullptr,
                 0, 0, st);
}

StepState make_state(chimera_ctx* c) {
  chimera_model* m = c->m;
  chimera_kv* kv = c->kv;
  StepState s{};
  s.B = c->batch;
  s.N = c->N;
  s.K = c->K;
  s.d = m->cfg.d_model;
  s.V = m->cfg.vocab;
  s.H = m->cfg.n_heads;
  s.hd = m->cfg.head_dim;
  s.ps = kv->ps;
  s.max_pages = kv->max_pages;
  s.tok_stride = c->tok_stride;
  s.cap = kv->cap;
  s.page_stride = kv->page_stride;
  s.n = c->n;
  s.tok = c->tok;
  s.h_last = c->h_last;
  s.page_table = kv->page_table;
  s.t_parent = c->tree.parent;
  s.t_depth = c->tree.depth;
  s.t_rank = c->tree.rank;
  s.t_anc = c->tree.anc;
  s.s_k = c->s_k_dev;
  s.cand = c->cand;
  s.tree_tok = c->tree_tok;
  s.inject = c->inject;
  s.inject_on = c->inject_on;
  s.f_ref = c->f_ref;
  s.f_ok = c->f_ok;
  s.f_stride = c->f_stride;
  s.out_tok = c->out_tok;
  s.out_nodes = c->out_nodes;
  s.out_len = c->out_len;
  s.pro_base = c->pro_base;
  s.pro_count = c->pro_count;
  s.pro_h = c->pro_h;
  s.hl = c->hl_rm;
  s.amax = c->amax;
  s.v_pos = c->v_pos;
  s.v_kvoff = c->v_kvoff;
  s.v_qrow = c->v_qrow;
  s.typical = c->typical;
  s.inv_T = 1.f / c->temperature;
  s.eps = c->t_eps;
  s.delta = c->t_delta;
  s.logits = c->logits;
  s.t_lse = c->t_lse;
  s.t_H = c->t_H;
  s.t_sample = c->t_sample;
  const TreeMeta& dm = c->branch ? c->tree : c->chain;
  s.d_nodes = c->d_nodes;
  s.d_parent = dm.parent;
  s.d_rank = dm.rank;
  s.d_path = dm.path;
  s.tok_src = c->tok_src;
  s.tree_slot0 = kv->cap - ENC_TREE_SLOTS;
  return s;
}

// The draft: K levels of trigram MLP -> encoder block -> head k -> top-s.
// Level k runs one query per drafted node: the rank-0 chain's node k (chain
// drafting) or every depth-k tree node with children (branch-conditioned
// drafting).  Level 0 also commits the previous step's encoder entries.
void run_draft(chimera_ctx* c, const StepState& s, hipStream_t st) {
  chimera_model* m = c->m;
  chimera_kv* kv = c->kv;
  const chimera_config& cf = m->cfg;
  const int dt = m->dt, d = cf.d_model, F = cf.d_ffn, H = cf.n_heads, hd = cf.head_dim, V = cf.vocab;
  const int hdim = H * hd, B = c->batch, K = c->K;
  const Gemm g{c, st, false};
  for (int k = 0; k < K; ++k) {
    const DraftLevel lv{k, c->lvl_R[k], c->lvl_off[k]};
    const int Q = B * lv.R;              // query rows
    const int Mk = draft_level_rows(s, lv);  // plus the prologue rows at level 0
    launch_draft_rows(dt, s, m->embed, lv, c->tri_in, c->mt_d, c->d_pos, c->d_kvoff, c->d_qrow, st);
    // trigram encoder (Eq. 2); with the cache, hits fill their rows and the MLP
    // launches do nothing when every row hit
    const int* tri_skip = nullptr;
    if (c->tri_on) {
      launch_tri_lookup(s, c->tri, lv, c->htri, st);
      tri_skip = c->tri.miss;
    }
    GemmEpi e1;
    e1.kind = EPI_SILU;
    e1.out_t = c->tri_a;
    e1.o_mtiles = c->mt_d;
    g.run(c->tri_in, c->mt_d, Mk, m->tri_w1, d, 3 * d, e1, 0, 0, tri_skip);
    GemmEpi e2;
    e2.kind = EPI_F32;
    e2.out_f = c->htri;
    e2.ldo = d;
    g.run(c->tri_a, c->mt_d, Mk, m->tri_w2, d, d, e2, 0, 0, tri_skip);
    if (c->tri_on) launch_tri_insert(s, c->tri, lv, 0, 0, 0, c->htri, st);
    launch_rmsnorm(dt, c->htri, nullptr, 0, m->enc.attn_norm, c->un, c->mt_d, nullptr, Mk, d, cf.rms_eps, 0,
                   k == 0 ? c->pro_h : nullptr, Q, Q + B * (K + 1), st);
    GemmEpi eq;
    eq.kind = EPI_QKV;
    eq.pos = c->d_pos;
    eq.kvoff = c->d_kvoff;
    eq.qrow = c->d_qrow;
    eq.kbase = kv->enc_k;
    eq.vbase = kv->enc_v;
    eq.head_stride = (int64_t)kv->cap * hd;
    eq.qout = c->qc;
    eq.ldq = hdim;
    eq.rcos = m->rcos;
    eq.rsin = m->rsin;
    eq.H = H;
    eq.hd = hd;
    g.run(c->un, c->mt_d, Mk, m->enc.wqkv, 3 * hdim, d, eq);

    EncAttnArgs ea{};
    ea.q = c->qc;
    ea.ldq = hdim;
    ea.kbase = kv->enc_k;
    ea.vbase = kv->enc_v;
    ea.cap = kv->cap;
    ea.n_b = c->n;
    ea.level = k;
    ea.nodes = c->d_nodes + lv.off;
    ea.R = lv.R;
    ea.path = s.d_path;
    ea.tree_slot0 = s.tree_slot0;
    ea.H = H;
    ea.hd = hd;
    ea.scale = 1.0f / std::sqrt((float)hd);
    ea.part = c->enc_part;
    ea.nblk = c->nblk_enc;
    ea.out = c->attn_c;
    ea.o_mtiles = c->mt_q;
    ea.B = B;
    launch_enc_attn(dt, ea, st);

    GemmEpi eo;
    eo.kind = EPI_PARTIAL;
    eo.part = c->dparts;
    g.run(c->attn_c, c->mt_q, Q, m->enc.wo, d, hdim, eo);
    launch_rmsnorm(dt, c->htri, c->dparts, g.splits(d, hdim), m->enc.ffn_norm, c->yn, c->mt_q, nullptr, Q, d,
                   cf.rms_eps, 1, nullptr, 0, 0, st);
    GemmEpi egu;
    egu.kind = EPI_SWIGLU;
    egu.out_t = c->hc;
    egu.o_mtiles = c->mt_q;
    g.run(c->yn, c->mt_q, Q, m->enc.wgu, 2 * F, d, egu);
    GemmEpi ed;
    ed.kind = EPI_PARTIAL;
    ed.part = c->dparts;
    g.run(c->hc, c->mt_q, Q, m->enc.wdown, d, F, ed);
    launch_draft_finish(dt, s, lv, c->htri, c->dparts, g.splits(d, F), c->zin, c->mt_q, st);
    GemmEpi ea1;
    ea1.kind = EPI_SILU;
    ea1.out_t = c->ak;
    ea1.o_mtiles = c->mt_q;
    g.run(c->zin, c->mt_q, Q, m->head_a[k], d, 2 * d, ea1);
    // head logits: chain drafting keeps every level ([B][K][V]); branch-
    // conditioned drafting uses the verify logits buffer as scratch
    float* z = c->branch ? c->logits : c->dlogits + (size_t)k * V;
    const int64_t ldz = c->branch ? V : (int64_t)K * V;
    GemmEpi et;
    et.kind = EPI_F32;
    et.out_f = z;
    et.ldo = (int)ldz;
    g.run(c->ak, c->mt_q, Q, m->head_theta[k], V, d, et);
    launch_topk(z, ldz, s, lv, c->topk_v, c->topk_i, st);
  }
}

void drop_graph(chimera_ctx* c) {
  if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
  if (c->graph) (void)hipGraphDestroy(c->graph);
  c->gexec = nullptr;
  c->graph = nullptr;
}

void check_ctx(chimera_ctx* c) {
  REQUIRE(c != nullptr, CHIMERA_EINVAL, "null ctx");
  REQUIRE(!c->poisoned, CHIMERA_ESTATE, "context poisoned by an earlier HIP failure");
}

void sync_or_poison(chimera_ctx* c, hipStream_t st) {
  hipError_t e = hipStreamSynchronize(st);
  if (e == hipSuccess) e = hipGetLastError();
  if (e != hipSuccess) {
    c->poisoned = true;
    throw Err(CHIMERA_EHIP, std::string("HIP failure: ") + hipGetErrorString(e));
  }
}

// Size (and, with a real arena, carve) a context.
void carve_ctx(chimera_ctx* c, Arena& a) {
  chimera_model* m = c->m;
  const chimera_config& cf = m->cfg;
  const size_t es = m->es, d = cf.d_model, F = cf.d_ffn, V = cf.vocab, H = cf.n_heads, hd = cf.head_dim;
  const size_t B = c->B, K = c->K, Mv = c->Mv, Md = c->Md, N = c->N, Mq = c->Mq;
  const size_t Qp = (size_t)mcap(c->Mq);
  c->mt_v = (int)(Mv / 16);
  c->mt_d = (int)(Md / 16);
  c->mt_q = (int)(Qp / 16);
  c->n = a.arr<int>(B);
  c->tok = a.arr<int>(B * c->tok_stride);
  c->h_last = a.take(B * d * es);
  c->cand = a.arr<int>(B * 64 * 8);
  c->d_nodes = a.arr<int>(64);
  c->tok_src = a.arr<int>(64);
  c->tree_tok = a.arr<int>(Mv);
  c->inject = a.arr<int>(B * std::max<size_t>(N, 2));
  c->inject_on = a.arr<int>(1);
  c->s_k_dev = a.arr<int>(8);
  c->res_nodes_off = sizeof(int) * B * (K + 1);
  c->res_len_off = 2 * c->res_nodes_off;
  c->res_bytes = c->res_len_off + sizeof(int) * B;
  c->result = (char*)a.take(c->res_bytes);
  if (c->result != nullptr) {
    c->out_tok = (int*)c->result;
    c->out_nodes = (int*)(c->result + c->res_nodes_off);
    c->out_len = (int*)(c->result + c->res_len_off);
  }
  c->stamp_ring = a.arr<unsigned long long>((size_t)STAMP_RING * STAMP_WORDS);
  c->stamp_count = a.arr<unsigned int>(1);
  c->pro_base = a.arr<int>(B);
  c->pro_count = a.arr<int>(B);
  c->pro_h = a.take(B * (K + 1) * d * es);
  c->pf_n = a.arr<int>(1);
  c->pf_tokens = a.arr<int>(64);
  c->x = a.arr<float>(Mv * d);
  c->xn = a.take(Mv * d * es);
  c->q = a.take(Mv * d * es);
  c->attn = a.take(Mv * d * es);
  c->hbuf = a.take(Mv * F * es);
  c->parts = a.arr<float>(8 * Mv * d);
  // split-K scratch: the largest splits * M * N_full over the launches this
  // context makes (partials are indexed with the full packed width)
  size_t scr = 1;
  auto need = [&](size_t M, int cols, int n_full, int Kd) {
    const int s = gemm_pick_splits(cols, Kd, m->dt);
    if (s > 1) scr = std::max(scr, (size_t)s * M * (size_t)n_full);
  };
  const int hdim = (int)(H * hd);
  for (size_t M : {Mv, Md, Qp, (size_t)128}) {
    need(M, 3 * hdim, 3 * hdim, (int)d);
    need(M, 2 * hdim, 3 * hdim, (int)d);
    need(M, 2 * (int)F, 2 * (int)F, (int)d);
    need(M, (int)V, (int)V, (int)d);
    need(M, (int)d, (int)d, 3 * (int)d);
    need(M, (int)d, (int)d, (int)d);
    need(M, (int)d, (int)d, 2 * (int)d);
  }
  c->scratch = a.arr<float>(scr);
  c->logits = a.arr<float>(Mv * V);
  c->amax = a.arr<int>(Mv);
  c->hl = a.take(Mv * d * es);
  c->hl_rm = a.take(Mv * d * es);
  const size_t qrows = std::max(B * N, (size_t)64);
  c->part_o = a.arr<float>(qrows * H * c->G * hd);
  c->part_ml = a.arr<float>(qrows * H * c->G * 2);
  c->rowtab = a.arr<int64_t>(B * TREE_ATTN_TAIL_ROWS);
  c->t_lse = a.arr<double>(Mv);
  c->t_H = a.arr<double>(Mv);
  c->t_sample = a.arr<int>(Mv);
  c->tri.hit = a.arr<int>(Md);
  c->tri.miss = a.arr<int>(1);
  c->tri.stats = a.arr<unsigned long long>(2);
  c->v_pos = a.arr<int>(Mv);
  c->v_kvoff = a.arr<int64_t>(Mv);
  c->v_qrow = a.arr<int>(Mv);
  c->tri_in = a.take(Md * 3 * d * es);
  c->tri_a = a.take(Md * d * es);
  c->htri = a.arr<float>(Md * d);
  c->un = a.take(Md * d * es);
  c->d_pos = a.arr<int>(Md);
  c->d_kvoff = a.arr<int64_t>(Md);
  c->d_qrow = a.arr<int>(Md);
  c->qc = a.take(Md * d * es);
  c->attn_c = a.take(Qp * d * es);
  c->yn = a.take(Qp * d * es);
  c->hc = a.take(Qp * F * es);
  c->zin = a.take(Qp * 2 * d * es);
  c->ak = a.take(Qp * d * es);
  c->dlogits = a.arr<float>(B * std::max<size_t>(K, 1) * V);
  c->dparts = a.arr<float>(8 * Mq * d);
  c->enc_part = a.arr<float>(Mq * H * c->nblk_enc * (hd + 2));
  c->topk_v = a.arr<float>(Mq * 32 * 8);
  c->topk_i = a.arr<int>(Mq * 32 * 8);
  auto meta = [&](TreeMeta& t) {
    t.parent = a.arr<int>(64);
    t.depth = a.arr<int>(64);
    t.rank = a.arr<int>(64);
    t.anc = a.arr<unsigned long long>(64);
    t.path = a.arr<uint8_t>(64 * 64);
  };
  meta(c->tree);
  meta(c->chain);
}

void upload_meta(TreeMeta& t, const std::vector<int>& parent, const std::vector<int>& rank,
                 const std::vector<int>& depth, const std::vector<unsigned long long>& anc) {
  const int n = (int)parent.size();
  std::vector<int> p(64, -1), r(64, 0), dp(64, 0);
  std::vector<unsigned long long> an(64, 0);
  std::vector<uint8_t> path(64 * 64, 0);
  for (int u = 0; u < n; ++u) {
    p[u] = parent[u];
    r[u] = rank[u];
    dp[u] = depth[u];
    an[u] = anc[u];
    for (int w = 0; w < n; ++w)
      if ((anc[u] >> w) & 1ull) path[u * 64 + depth[w]] = (uint8_t)w;
  }
  HIPCK(hipMemcpy(t.parent, p.data(), 64 * sizeof(int), hipMemcpyHostToDevice));
  HIPCK(hipMemcpy(t.rank, r.data(), 64 * sizeof(int), hipMemcpyHostToDevice));
  HIPCK(hipMemcpy(t.depth, dp.data(), 64 * sizeof(int), hipMemcpyHostToDevice));
  HIPCK(hipMemcpy(t.anc, an.data(), 64 * sizeof(unsigned long long), hipMemcpyHostToDevice));
  HIPCK(hipMemcpy(t.path, path.data(), 64 * 64, hipMemcpyHostToDevice));
}

// Drafted nodes per level and each verify node's list: chain drafting drafts
// chain node k at level k and takes node u's token from level depth(u) - 1;
// branch-conditioned drafting drafts every tree node with children and takes
// node u's token from its parent's own list.
void set_draft_plan(chimera_ctx* c) {
  std::vector<int> nodes, src(64, 0);
  std::vector<char> has_child(64, 0);
  for (int u = 1; u < c->N; ++u) has_child[c->parent[u]] = 1;
  c->lvl_R.assign(std::max(c->K, 1), 0);
  c->lvl_off.assign(std::max(c->K, 1), 0);
  for (int k = 0; k < c->K; ++k) {
    c->lvl_off[k] = (int)nodes.size();
    if (!c->branch)
      nodes.push_back(k);
    else
      for (int u = 0; u < c->N; ++u)
        if (c->depth[u] == k && has_child[u]) nodes.push_back(u);
    c->lvl_R[k] = (int)nodes.size() - c->lvl_off[k];
    REQUIRE(c->lvl_R[k] >= 1 && c->B * c->lvl_R[k] <= std::max(c->Mq, 1), CHIMERA_EINVAL,
            "draft level larger than the context was sized for");
  }
  for (int u = 1; u < c->N; ++u) src[u] = c->branch ? c->parent[u] : c->depth[u] - 1;
  nodes.resize(64, 0);
  HIPCK(hipMemcpy(c->d_nodes, nodes.data(), 64 * sizeof(int), hipMemcpyHostToDevice));
  HIPCK(hipMemcpy(c->tok_src, src.data(), 64 * sizeof(int), hipMemcpyHostToDevice));
}

void ctx_dims(chimera_ctx* c) {
  const chimera_config& cf = c->m->cfg;
  c->Mv = mcap(std::max(c->B * c->N, 64));
  // query rows of one draft level: B (chain drafting) or B times the level's
  // drafted nodes (branch-conditioned drafting), fewer than N per sequence
  c->Mq = c->B * std::max(c->N - 1, 1);
  c->Md = mcap(std::max({c->B * (2 * (c->K + 1) + 1), c->Mq, 128}));
  c->G = tree_attn_groups(c->kv->max_len);
  c->tok_stride = c->kv->max_len + 8;
  c->nblk_enc = (2 * c->kv->cap + cf.n_draft_heads + 1 + 255) / 256;
}

// Algorithmic bytes of one verify pass: every target weight once (norm
// gains included), the KV read over the committed lengths (sum_n summed over
// the batch) and the tree's own K/V rows written.
double verify_pass_bytes(const chimera_ctx* c, double sum_n) {
  const chimera_model* m = c->m;
  const chimera_config& cf = m->cfg;
  const double es = (double)m->es, d = cf.d_model, F = cf.d_ffn, V = cf.vocab;
  const double hdim = (double)cf.n_heads * cf.head_dim;
  const double w_layer = (d * 3 * hdim + hdim * d + d * 2 * F + F * d) * es + 2 * d * 4;
  const double bytes = cf.n_layers * w_layer + d * V * es + d * 4;
  return bytes + (double)cf.n_layers * 2 * hdim * es * (sum_n + (double)c->batch * c->N);
}

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* chimera_last_error(void) { return g_err.c_str(); }

chimera_status chimera_weight_bytes(const chimera_config* cfg, int64_t* bytes) {
  return guard([&] {
    validate_config(cfg);
    REQUIRE(bytes != nullptr, CHIMERA_EINVAL, "null bytes");
    Arena a{nullptr, 0};
    chimera_model tmp;
    tmp.cfg = *cfg;
    carve_model(*cfg, a, tmp);
    *bytes = (int64_t)a.off + 256;
  });
}

chimera_status chimera_load(const chimera_config* cfg, const chimera_tensor* tensors, int32_t n_tensors, void* arena,
                            int64_t arena_bytes, void* stream, chimera_model** out) {
  return guard([&] {
    validate_config(cfg);
    REQUIRE(out != nullptr && arena != nullptr && tensors != nullptr, CHIMERA_EINVAL, "null argument");
    hipStream_t st = (hipStream_t)stream;
    const chimera_config& c = *cfg;
    const int dt = c.dtype;
    const size_t es = esize(dt);
    const int64_t d = c.d_model, F = c.d_ffn, V = c.vocab, hdim = (int64_t)c.n_heads * c.head_dim;
    // expected tensor list
    std::map<std::string, std::pair<int64_t, int>> want;  // numel, dtype
    auto blk = [&](const std::string& p) {
      want[p + "attn_norm"] = {d, CHIMERA_F32};
      want[p + "wq"] = {d * hdim, dt};
      want[p + "wk"] = {d * hdim, dt};
      want[p + "wv"] = {d * hdim, dt};
      want[p + "wo"] = {hdim * d, dt};
      want[p + "ffn_norm"] = {d, CHIMERA_F32};
      want[p + "w_gate"] = {d * F, dt};
      want[p + "w_up"] = {d * F, dt};
      want[p + "w_down"] = {F * d, dt};
    };
    want["tok_embed"] = {V * d, dt};
    for (int l = 0; l < c.n_layers; ++l) blk("layers." + std::to_string(l) + ".");
    want["final_norm"] = {d, CHIMERA_F32};
    want["lm_head"] = {d * V, dt};
    want["draft.tri_w1"] = {3 * d * d, dt};
    want["draft.tri_w2"] = {d * d, dt};
    blk("draft.enc.");
    for (int k = 0; k < c.n_draft_heads; ++k) {
      want["draft.heads." + std::to_string(k) + ".a"] = {2 * d * d, dt};
      want["draft.heads." + std::to_string(k) + ".theta"] = {d * V, dt};
    }
    std::map<std::string, const chimera_tensor*> have;
    for (int i = 0; i < n_tensors; ++i) {
      const chimera_tensor& t = tensors[i];
      REQUIRE(t.name != nullptr && t.data != nullptr, CHIMERA_EINVAL, "tensor without name or data");
      auto it = want.find(t.name);
      REQUIRE(it != want.end(), CHIMERA_EINVAL, std::string("unexpected tensor ") + t.name);
      REQUIRE(t.numel == it->second.first, CHIMERA_EINVAL, std::string("wrong size for ") + t.name);
      REQUIRE(t.dtype == it->second.second, CHIMERA_EINVAL, std::string("wrong dtype for ") + t.name);
      REQUIRE(t.on_device == 1, CHIMERA_EINVAL,
              std::string("tensor ") + t.name + " is not in device memory (copy it to the device first)");
      have[t.name] = &t;
    }
    for (auto& kvp : want) REQUIRE(have.count(kvp.first), CHIMERA_EINVAL, "missing tensor " + kvp.first);

    int64_t need = 0;
    {
      Arena a{nullptr, 0};
      chimera_model tmp;
      carve_model(c, a, tmp);
      need = (int64_t)a.off;
    }
    REQUIRE(arena_bytes >= need, CHIMERA_ENOMEM, "weight arena too small");
    auto* m = new chimera_model();
    try {
      m->cfg = c;
      m->dt = dt;
      m->es = es;
      Arena a{(char*)arena, (size_t)arena_bytes};
      carve_model(c, a, *m);
      auto dev = [&](const std::string& name) -> const void* { return have[name]->data; };
      auto copy = [&](void* dst, const std::string& name) {
        const chimera_tensor* t = have[name];
        const size_t bytes = (size_t)t->numel * (t->dtype == CHIMERA_F32 ? 4 : 2);
        HIPCK(hipMemcpyAsync(dst, t->data, bytes, hipMemcpyDeviceToDevice, st));
      };
      auto pack = [&](void* dst, int kind, const std::string& a0, const std::string& a1, const std::string& a2, int K,
                      int n_src) {
        const void* s0 = dev(a0);
        const void* s1 = a1.empty() ? nullptr : dev(a1);
        const void* s2 = a2.empty() ? nullptr : dev(a2);
        launch_repack(dt, kind, s0, s1, s2, K, n_src, dst, c.n_heads, c.head_dim, st);
        HIPCK(hipGetLastError());
      };
      auto block = [&](const std::string& p, BlockW& w) {
        copy(w.attn_norm, p + "attn_norm");
        copy(w.ffn_norm, p + "ffn_norm");
        pack(w.wqkv, PACK_QKV, p + "wq", p + "wk", p + "wv", (int)d, (int)hdim);
        pack(w.wo, PACK_NATURAL, p + "wo", "", "", (int)hdim, (int)d);
        pack(w.wgu, PACK_GU, p + "w_gate", p + "w_up", "", (int)d, (int)F);
        pack(w.wdown, PACK_NATURAL, p + "w_down", "", "", (int)F, (int)d);
      };
      copy(m->embed, "tok_embed");
      for (int l = 0; l < c.n_layers; ++l) block("layers." + std::to_string(l) + ".", m->layers[l]);
      copy(m->final_norm, "final_norm");
      pack(m->lm_head, PACK_NATURAL, "lm_head", "", "", (int)d, (int)V);
      pack(m->tri_w1, PACK_NATURAL, "draft.tri_w1", "", "", (int)(3 * d), (int)d);
      pack(m->tri_w2, PACK_NATURAL, "draft.tri_w2", "", "", (int)d, (int)d);
      block("draft.enc.", m->enc);
      for (int k = 0; k < c.n_draft_heads; ++k) {
        const std::string p = "draft.heads." + std::to_string(k) + ".";
        pack(m->head_a[k], PACK_NATURAL, p + "a", "", "", (int)(2 * d), (int)d);
        pack(m->head_theta[k], PACK_NATURAL, p + "theta", "", "", (int)d, (int)V);
      }
      // rotary tables: angle(p, i) = p * base^(-2i/hd) in double, rounded to float
      const int half = c.head_dim / 2;
      std::vector<float> cs((size_t)c.max_positions * half), sn((size_t)c.max_positions * half);
      for (int p = 0; p < c.max_positions; ++p)
        for (int i = 0; i < half; ++i) {
          const double inv = std::pow((double)c.rope_base, -(2.0 * i) / (double)c.head_dim);
          const double ang = (double)p * inv;
          cs[(size_t)p * half + i] = (float)std::cos(ang);
          sn[(size_t)p * half + i] = (float)std::sin(ang);
        }
      HIPCK(hipMemcpyAsync(m->rcos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice, st));
      HIPCK(hipMemcpyAsync(m->rsin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice, st));
      HIPCK(hipStreamSynchronize(st));
    } catch (...) {
      delete m;
      throw;
    }
    *out = m;
  });
}

static void kv_dims(const chimera_model* m, int32_t max_batch, int32_t max_len, int32_t n_pages, int32_t page_size) {
  REQUIRE(m != nullptr, CHIMERA_EINVAL, "null model");
  REQUIRE(max_batch >= 1 && max_batch <= 64, CHIMERA_EINVAL, "max_batch in [1, 64]");
  REQUIRE(page_size >= 1 && page_size <= 256, CHIMERA_EINVAL, "page_size");
  REQUIRE(max_len >= 64 && max_len + 64 <= m->cfg.max_positions, CHIMERA_EINVAL,
          "max_len must be >= 64 and max_len + 64 <= max_positions");
  const int per = (max_len + 64 + page_size - 1) / page_size;
  REQUIRE((int64_t)n_pages >= (int64_t)per * max_batch, CHIMERA_EINVAL, "n_pages too small for max_batch * max_len");
}

static void carve_kv(chimera_kv* kv, Arena& a) {
  const chimera_model* m = kv->m;
  const chimera_config& c = m->cfg;
  const size_t es = m->es, H = c.n_heads, hd = c.head_dim;
  kv->pool = a.take((size_t)c.n_layers * kv->n_pages * 2 * H * kv->ps * hd * es);
  kv->page_table = a.arr<int>((size_t)kv->B * kv->max_pages);
  kv->enc_k = a.take((size_t)kv->B * 2 * H * kv->cap * hd * es);
  kv->enc_v = a.take((size_t)kv->B * 2 * H * kv->cap * hd * es);
}

chimera_status chimera_kv_bytes(const chimera_model* m, int32_t max_batch, int32_t max_len, int32_t n_pages,
                                int32_t page_size, int64_t* bytes) {
  return guard([&] {
    kv_dims(m, max_batch, max_len, n_pages, page_size);
    REQUIRE(bytes != nullptr, CHIMERA_EINVAL, "null bytes");
    chimera_kv kv;
    kv.m = const_cast<chimera_model*>(m);
    kv.B = max_batch;
    kv.max_len = max_len;
    kv.n_pages = n_pages;
    kv.ps = page_size;
    kv.max_pages = (max_len + 64 + page_size - 1) / page_size;
    kv.cap = max_len + 64 + ENC_TREE_SLOTS;
    Arena a{nullptr, 0};
    carve_kv(&kv, a);
    *bytes = (int64_t)a.off + 256;
  });
}

chimera_status chimera_kv_create(chimera_model* m, int32_t max_batch, int32_t max_len, int32_t n_pages,
                                 int32_t page_size, const int32_t* page_order, void* arena, int64_t arena_bytes,
                                 chimera_kv** out) {
  return guard([&] {
    kv_dims(m, max_batch, max_len, n_pages, page_size);
    REQUIRE(out != nullptr && arena != nullptr, CHIMERA_EINVAL, "null argument");
    auto* kv = new chimera_kv();
    try {
      kv->m = m;
      kv->B = max_batch;
      kv->max_len = max_len;
      kv->n_pages = n_pages;
      kv->ps = page_size;
      kv->max_pages = (max_len + 64 + page_size - 1) / page_size;
      kv->cap = max_len + 64 + ENC_TREE_SLOTS;
      const int64_t H = m->cfg.n_heads, hd = m->cfg.head_dim;
      kv->page_stride = 2 * H * page_size * hd;
      kv->layer_stride = (int64_t)n_pages * kv->page_stride;
      Arena a{(char*)arena, (size_t)arena_bytes};
      carve_kv(kv, a);
      std::vector<int> order(n_pages);
      std::vector<char> seen(n_pages, 0);
      for (int i = 0; i < n_pages; ++i) {
        const int p = page_order ? page_order[i] : i;
        REQUIRE(p >= 0 && p < n_pages && !seen[p], CHIMERA_EINVAL, "page_order must be a permutation");
        seen[p] = 1;
        order[i] = p;
      }
      kv->page_table_host.resize((size_t)kv->B * kv->max_pages);
      for (int b = 0; b < kv->B; ++b)
        for (int i = 0; i < kv->max_pages; ++i)
          kv->page_table_host[(size_t)b * kv->max_pages + i] = order[(size_t)b * kv->max_pages + i];
      HIPCK(hipMemcpy(kv->page_table, kv->page_table_host.data(), kv->page_table_host.size() * sizeof(int),
                      hipMemcpyHostToDevice));
    } catch (...) {
      delete kv;
      throw;
    }
    *out = kv;
  });
}

static void tree_from(const int32_t* parent, const int32_t* rank, int32_t n_nodes, int n_heads, chimera_ctx* c) {
  REQUIRE(n_nodes >= 1 && n_nodes <= 64, CHIMERA_EINVAL, "n_nodes in [1, 64]");
  REQUIRE(parent != nullptr && rank != nullptr, CHIMERA_EINVAL, "null tree");
  REQUIRE(parent[0] == -1, CHIMERA_EINVAL, "node 0 must be the root");
  c->parent.assign(parent, parent + n_nodes);
  c->rank.assign(rank, rank + n_nodes);
  c->depth.assign(n_nodes, 0);
  c->anc.assign(n_nodes, 0);
  c->anc[0] = 1ull;
  int D = 0;
  for (int u = 1; u < n_nodes; ++u) {
    const int p = parent[u];
    REQUIRE(p >= 0 && p < u, CHIMERA_EINVAL, "parent must precede its child");
    REQUIRE(rank[u] >= 0 && rank[u] < 8, CHIMERA_EINVAL, "rank in [0, 8)");
    c->depth[u] = c->depth[p] + 1;
    REQUIRE(c->depth[u] >= c->depth[u - 1], CHIMERA_EINVAL, "nodes must be ordered by depth");
    c->anc[u] = c->anc[p] | (1ull << u);
    D = std::max(D, c->depth[u]);
    for (int w = 1; w < u; ++w)
      REQUIRE(!(parent[w] == p && rank[w] == rank[u]), CHIMERA_EINVAL, "siblings must have distinct ranks");
  }
  REQUIRE(D <= n_heads, CHIMERA_EINVAL, "tree deeper than the number of draft heads");
  c->N = n_nodes;
  c->K = D;
  c->D = D;
  c->s_k.assign(8, 1);
  for (int u = 1; u < n_nodes; ++u) c->s_k[c->depth[u] - 1] = std::max(c->s_k[c->depth[u] - 1], rank[u] + 1);
}

chimera_status chimera_ctx_bytes(const chimera_model* m, const chimera_kv* kv, int32_t n_nodes, int64_t* bytes) {
  return guard([&] {
    REQUIRE(m != nullptr && kv != nullptr && bytes != nullptr, CHIMERA_EINVAL, "null argument");
    REQUIRE(n_nodes >= 1 && n_nodes <= 64, CHIMERA_EINVAL, "n_nodes in [1, 64]");
    chimera_ctx c;
    c.m = const_cast<chimera_model*>(m);
    c.kv = const_cast<chimera_kv*>(kv);
    c.B = kv->B;
    c.N = n_nodes;
    c.K = std::min<int>(n_nodes - 1, m->cfg.n_draft_heads);
    ctx_dims(&c);
    Arena a{nullptr, 0};
    carve_ctx(&c, a);
    *bytes = (int64_t)a.off + 256;
  });
}

chimera_status chimera_ctx_create(chimera_model* m, chimera_kv* kv, const int32_t* parent, const int32_t* rank,
                                  int32_t n_nodes, void* arena, int64_t arena_bytes, chimera_ctx** out) {
  return guard([&] {
    REQUIRE(m != nullptr && kv != nullptr && out != nullptr && arena != nullptr, CHIMERA_EINVAL, "null argument");
    REQUIRE(kv->m == m, CHIMERA_EINVAL, "kv belongs to another model");
    auto* c = new chimera_ctx();
    try {
      c->m = m;
      c->kv = kv;
      c->B = kv->B;
      tree_from(parent, rank, n_nodes, m->cfg.n_draft_heads, c);
      // carve with the worst-case number of levels (what chimera_ctx_bytes
      // sized), then run with the tree's own depth
      const int K_used = c->K;
      c->K = std::min<int>(n_nodes - 1, m->cfg.n_draft_heads);
      ctx_dims(c);
      Arena a{(char*)arena, (size_t)arena_bytes};
      carve_ctx(c, a);
      c->K = K_used;
      upload_meta(c->tree, c->parent, c->rank, c->depth, c->anc);
      std::vector<int> cp(64), cr(64, 0), cd(64);
      std::vector<unsigned long long> ca(64);
      for (int u = 0; u < 64; ++u) {
        cp[u] = u - 1;
        cd[u] = u;
        ca[u] = (u == 63) ? ~0ull : ((1ull << (u + 1)) - 1ull);
      }
      upload_meta(c->chain, cp, cr, cd, ca);
      set_draft_plan(c);
      HIPCK(hipMemcpy(c->s_k_dev, c->s_k.data(), 8 * sizeof(int), hipMemcpyHostToDevice));
      HIPCK(hipMemset(c->inject_on, 0, sizeof(int)));
      HIPCK(hipMemset(c->tri.miss, 0, sizeof(int)));
      HIPCK(hipMemset(c->tri.stats, 0, 2 * sizeof(unsigned long long)));
      HIPCK(hipMemset(c->n, 0, sizeof(int) * c->B));
      HIPCK(hipMemset(c->stamp_count, 0, sizeof(unsigned int)));
      HIPCK(hipMemset(c->tok, 0, sizeof(int) * (size_t)c->B * c->tok_stride));
      HIPCK(hipHostMalloc((void**)&c->host_result, c->res_bytes));
      HIPCK(hipHostMalloc((void**)&c->host_pipe, c->res_bytes * CHIMERA_MAX_PIPELINED_STEPS));
      c->n_host.assign(c->B, 0);
    } catch (...) {
      if (c->host_result) (void)hipHostFree(c->host_result);
      if (c->host_pipe) (void)hipHostFree(c->host_pipe);
      delete c;
      throw;
    }
    *out = c;
  });
}

chimera_status chimera_prefill(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, const int32_t* tokens,
                               const int32_t* lens, int32_t batch, int32_t* first_tokens, void* stream) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(m == ctx->m && kv == ctx->kv, CHIMERA_EINVAL, "ctx belongs to another model/kv");
    REQUIRE(tokens != nullptr && lens != nullptr && first_tokens != nullptr, CHIMERA_EINVAL, "null argument");
    REQUIRE(batch >= 1 && batch <= ctx->B, CHIMERA_EINVAL, "batch out of range");
    const chimera_config& cf = m->cfg;
    int64_t off = 0;
    for (int b = 0; b < batch; ++b) {
      REQUIRE(lens[b] >= 1, CHIMERA_EINVAL, "empty prompt");
      REQUIRE(lens[b] + ctx->N + ctx->K + 2 <= kv->max_len, CHIMERA_ECAPACITY, "prompt exceeds the KV capacity");
      for (int i = 0; i < lens[b]; ++i)
        REQUIRE(tokens[off + i] >= 0 && tokens[off + i] < cf.vocab, CHIMERA_EINVAL, "token id out of range");
      off += lens[b];
    }
    hipStream_t st = (hipStream_t)stream;
    ctx->batch = batch;
    drop_graph(ctx);
    StepState s = make_state(ctx);
    const int dt = m->dt, d = cf.d_model, H = cf.n_heads, hd = cf.head_dim, V = cf.vocab;
    const int hdim = H * hd;
    const Gemm g{ctx, st, false};
    off = 0;
    for (int b = 0; b < batch; ++b) {
      const int n = lens[b];
      HIPCK(hipMemcpyAsync(ctx->tok + (size_t)b * ctx->tok_stride, tokens + off, sizeof(int) * n,
                           hipMemcpyHostToDevice, st));
      off += n;
      for (int p0 = 0; p0 < n; p0 += 64) {
        const int M = std::min(64, n - p0);
        launch_prefill_rows(dt, s, m->embed, b, p0, M, ctx->pf_tokens, ctx->tri_in, ctx->mt_d, ctx->d_pos,
                            ctx->d_kvoff, ctx->d_qrow, ctx->pf_n, st);
        VerifyRows r{ctx->pf_tokens, M, ctx->pf_n, kv->page_table + (size_t)b * kv->max_pages,
                     ctx->chain.depth, ctx->chain.path, M, M - 1, 1};
        verify_layers(ctx, r, st, false);
        // draft memory: target-state entries (rows [0, M)) and trigram entries (rows [M, 2M))
        GemmEpi e1;
        e1.kind = EPI_SILU;
        e1.out_t = ctx->tri_a;
        e1.o_mtiles = ctx->mt_d;
        g.run(ctx->tri_in, ctx->mt_d, M, m->tri_w1, d, 3 * d, e1);
        GemmEpi e2;
        e2.kind = EPI_F32;
        e2.out_f = ctx->htri + (size_t)M * d;
        e2.ldo = d;
        g.run(ctx->tri_a, ctx->mt_d, M, m->tri_w2, d, d, e2);
        if (ctx->tri_on) launch_tri_insert(s, ctx->tri, DraftLevel{0, 1, 0}, b, p0, M, ctx->htri + (size_t)M * d, st);
        launch_rmsnorm(dt, ctx->htri, nullptr, 0, m->enc.attn_norm, ctx->un, ctx->mt_d, nullptr, 2 * M, d, cf.rms_eps,
                       0, ctx->hl_rm, 0, M, st);
        GemmEpi ekv;
        ekv.kind = EPI_QKV;
        ekv.pos = ctx->d_pos;
        ekv.kvoff = ctx->d_kvoff;
        ekv.qrow = ctx->d_qrow;
        ekv.kbase = kv->enc_k;
        ekv.vbase = kv->enc_v;
        ekv.head_stride = (int64_t)kv->cap * hd;
        ekv.qout = ctx->qc;
        ekv.ldq = hdim;
        ekv.rcos = m->rcos;
        ekv.rsin = m->rsin;
        ekv.H = H;
        ekv.hd = hd;
        g.run(ctx->un, ctx->mt_d, 2 * M, m->enc.wqkv, 3 * hdim, d, ekv, hdim / 16, 2 * hdim / 16);
        if (p0 + M == n) {
          GemmEpi el;
          el.kind = EPI_F32;
          el.out_f = ctx->logits;
          el.ldo = V;
          g.run(ctx->hl, ctx->mt_v, M, m->lm_head, V, d, el);
          if (ctx->typical)  // the first generated token is sampled at position n
            launch_typical_stats(ctx->logits + (size_t)(M - 1) * V, 1, V, 1, b, nullptr, nullptr, n,
                                 1.f / ctx->temperature, ctx->t_seed, ctx->t_lse, ctx->t_H, ctx->amax, st);
          else
            launch_argmax(ctx->logits + (size_t)(M - 1) * V, 1, V, ctx->amax, st);
          const char* last = (const char*)ctx->hl_rm + (size_t)(M - 1) * d * m->es;
          launch_prefill_finish(dt, s, b, n, ctx->amax, last, st);
        }
      }
    }
    HIPCK(hipGetLastError());
    sync_or_poison(ctx, st);
    for (int b = 0; b < batch; ++b) {
      int t = 0;
      HIPCK(hipMemcpy(&t, ctx->tok + (size_t)b * ctx->tok_stride + lens[b], sizeof(int), hipMemcpyDeviceToHost));
      first_tokens[b] = t;
      ctx->n_host[b] = lens[b];
    }
  });
}

}  // extern "C"

namespace {

// Enqueue one draft -> verify -> accept -> compact step on st: replay of the
// captured graph (captured on first use) or eager launches.
void enqueue_step(chimera_ctx* ctx, hipStream_t st) {
  chimera_model* m = ctx->m;
  chimera_kv* kv = ctx->kv;
  const chimera_config& cf = m->cfg;
  const int dt = m->dt, d = cf.d_model, V = cf.vocab;
  StepState s = make_state(ctx);
  const bool use_graph = ctx->graph_on && st != nullptr;
  // Under graph replay the step does not consult the profiling flag at all:
  // phase times come from the stamp ring, read by chimera_profile_read.
  // (Reading the flag on every replayed step was measured to slow the
  // replay, with identical GPU work.)
  if (!use_graph && ctx->prof && !ctx->ev_created) {  // per-launch GEMM events: eager launches only
    ctx->ev_pool.resize(1024);
    ctx->ev_bytes.assign(1024, 0.0);
    for (auto& e : ctx->ev_pool) {
      HIPCK(hipEventCreate(&e.a));
      HIPCK(hipEventCreate(&e.b));
    }
    ctx->ev_created = true;
  }
  // Phase timestamps: a one-lane kernel between phases writes the device
  // wall clock.  They are part of every step (graph or eager), so turning
  // profiling on times the same replayed graph that runs without it.
  auto mark = [&](int idx, hipStream_t q) { launch_stamp(ctx->stamp_ring, ctx->stamp_count, idx, ctx->n, ctx->batch, q); };
  // the launch sequence of one step; every varying scalar lives in device memory
  auto enqueue = [&](hipStream_t q) {
    const Gemm gq{ctx, q, true};
    ctx->ev_used = 0;
    mark(0, q);
    if (ctx->K > 0) run_draft(ctx, s, q);
    mark(1, q);
    launch_tree_setup(s, q);
    const int M = ctx->batch * ctx->N;
    VerifyRows r{ctx->tree_tok, M, ctx->n, kv->page_table, ctx->tree.depth, ctx->tree.path, ctx->N, ctx->D,
                 ctx->batch};
    verify_layers(ctx, r, q, true);
    GemmEpi el;
    el.kind = EPI_F32;
    el.out_f = ctx->logits;
    el.ldo = V;
    gq.run(ctx->hl, ctx->mt_v, M, m->lm_head, V, d, el);
    if (ctx->typical)
      launch_typical_stats(ctx->logits, M, V, ctx->N, 0, ctx->n, ctx->tree.depth, -1, 1.f / ctx->temperature,
                           ctx->t_seed, ctx->t_lse, ctx->t_H, ctx->t_sample, q);
    else
      launch_argmax(ctx->logits, M, V, ctx->amax, q);
    mark(2, q);
    launch_accept(dt, s, q);
    if (ctx->cc_side) launch_kv_snapshot(dt, s, kv->pool, cf.n_layers, kv->layer_stride, ctx->cc_side, q);
    launch_compact(dt, s, kv->pool, cf.n_layers, kv->layer_stride, q);
    if (ctx->cc_side)
      launch_kv_check(dt, s, kv->pool, cf.n_layers, kv->layer_stride, ctx->cc_side, ctx->cc_counts, q);
    launch_advance(dt, s, q);
    mark(3, q);
  };
  if (use_graph) {
    if (ctx->gexec == nullptr || ctx->graph_stream != st) {
      drop_graph(ctx);
      HIPCK(hipStreamBeginCapture(st, hipStreamCaptureModeThreadLocal));
      ctx->capturing = true;
      try {
        enqueue(st);
      } catch (...) {
        ctx->capturing = false;
        hipGraph_t g = nullptr;
        (void)hipStreamEndCapture(st, &g);
        if (g) (void)hipGraphDestroy(g);
        throw;
      }
      ctx->capturing = false;
      HIPCK(hipStreamEndCapture(st, &ctx->graph));
      HIPCK(hipGraphInstantiate(&ctx->gexec, ctx->graph, nullptr, nullptr, 0));
      ctx->graph_stream = st;
      ctx->graph_ev_used = ctx->ev_used;
    }
    ctx->ev_used = ctx->graph_ev_used;
    HIPCK(hipGraphLaunch(ctx->gexec, st));
  } else {
    enqueue(st);
  }
  HIPCK(hipGetLastError());
}

// One step's outputs from a host copy of the result block.
void parse_result(const chimera_ctx* ctx, const char* block, int32_t* new_tokens, int32_t* n_new,
                  int32_t* path_nodes) {
  const size_t K1 = ctx->K + 1, B = ctx->batch;
  const int* h_tok = (const int*)block;
  const int* h_nodes = (const int*)(block + ctx->res_nodes_off);
  const int* h_len = (const int*)(block + ctx->res_len_off);
  for (size_t b = 0; b < B; ++b) {
    const int L = h_len[b];
    n_new[b] = L;
    for (size_t i = 0; i < K1; ++i) {
      new_tokens[b * K1 + i] = i < (size_t)L ? h_tok[b * K1 + i] : -1;
      if (path_nodes) path_nodes[b * K1 + i] = i < (size_t)L ? h_nodes[b * K1 + i] : -1;
    }
  }
}

// Per-launch GEMM events of an eagerly launched, profiled step (after its sync).
void collect_gemm_events(chimera_ctx* ctx, hipStream_t st) {
  const bool use_graph = ctx->graph_on && st != nullptr;
  if (use_graph || !ctx->prof) return;
  float ms = 0.f;
  for (size_t i = 0; i < ctx->ev_used; ++i) {
    HIPCK(hipEventElapsedTime(&ms, ctx->ev_pool[i].a, ctx->ev_pool[i].b));
    ctx->acc.ms_gemm_verify += ms;
    ctx->acc.gemm_verify_bytes += ctx->ev_bytes[i];
    ctx->acc.gemm_verify_launches += 1;
  }
}

void check_step_call(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, int n_steps) {
  check_ctx(ctx);
  REQUIRE(m == ctx->m && kv == ctx->kv, CHIMERA_EINVAL, "ctx belongs to another model/kv");
  REQUIRE(ctx->batch >= 1, CHIMERA_ESTATE, "chimera_step before chimera_prefill");
  for (int b = 0; b < ctx->batch; ++b)
    REQUIRE(ctx->n_host[b] + (int64_t)(n_steps - 1) * (ctx->K + 1) + ctx->N + ctx->K + 2 <= kv->max_len,
            CHIMERA_ECAPACITY, "sequence would outgrow its KV capacity");
}

}  // namespace

extern "C" {

chimera_status chimera_step(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, int32_t* new_tokens, int32_t* n_new,
                            int32_t* path_nodes, void* stream) {
  return guard([&] {
    check_step_call(m, kv, ctx, 1);
    REQUIRE(new_tokens != nullptr && n_new != nullptr, CHIMERA_EINVAL, "null output");
    hipStream_t st = (hipStream_t)stream;
    enqueue_step(ctx, st);
    HIPCK(hipMemcpyAsync(ctx->host_result, ctx->result, ctx->res_bytes, hipMemcpyDeviceToHost, st));
    sync_or_poison(ctx, st);
    parse_result(ctx, ctx->host_result, new_tokens, n_new, path_nodes);
    collect_gemm_events(ctx, st);
    for (int b = 0; b < ctx->batch; ++b) ctx->n_host[b] += n_new[b];
  });
}

chimera_status chimera_steps(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, int32_t n_steps, int32_t* new_tokens,
                             int32_t* n_new, int32_t* path_nodes, void* stream) {
  return guard([&] {
    REQUIRE(n_steps >= 1 && n_steps <= CHIMERA_MAX_PIPELINED_STEPS, CHIMERA_EINVAL, "n_steps in [1, 64]");
    check_step_call(m, kv, ctx, n_steps);
    REQUIRE(new_tokens != nullptr && n_new != nullptr, CHIMERA_EINVAL, "null output");
    hipStream_t st = (hipStream_t)stream;
    const size_t B = ctx->batch, K1 = ctx->K + 1;
    // eager launches with per-launch events reuse one event set per step:
    // those steps synchronise one at a time
    const bool each = !(ctx->graph_on && st != nullptr) && ctx->prof;
    for (int i = 0; i < n_steps; ++i) {
      enqueue_step(ctx, st);
      HIPCK(hipMemcpyAsync(ctx->host_pipe + (size_t)i * ctx->res_bytes, ctx->result, ctx->res_bytes,
                           hipMemcpyDeviceToHost, st));
      if (each) {
        sync_or_poison(ctx, st);
        collect_gemm_events(ctx, st);
      }
    }
    sync_or_poison(ctx, st);
    for (int i = 0; i < n_steps; ++i) {
      parse_result(ctx, ctx->host_pipe + (size_t)i * ctx->res_bytes, new_tokens + i * B * K1, n_new + i * B,
                   path_nodes ? path_nodes + i * B * K1 : nullptr);
      for (size_t b = 0; b < B; ++b) ctx->n_host[b] += n_new[i * B + b];
    }
  });
}

chimera_status chimera_set_forcing(chimera_ctx* ctx, const int32_t* ref, const uint8_t* ok, int32_t stride) {
  return guard([&] {
    check_ctx(ctx);
    drop_graph(ctx);
    if (ref == nullptr) {
      ctx->f_ref = nullptr;
      ctx->f_ok = nullptr;
      ctx->f_stride = 0;
      return;
    }
    REQUIRE(ok != nullptr, CHIMERA_EINVAL, "ok table missing");
    REQUIRE(stride >= ctx->kv->max_len + 8, CHIMERA_EINVAL, "forcing stride must cover max_len + 8 positions");
    ctx->f_ref = ref;
    ctx->f_ok = ok;
    ctx->f_stride = stride;
  });
}

chimera_status chimera_set_tree_tokens(chimera_ctx* ctx, const int32_t* tokens, int32_t batch) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(tokens != nullptr, CHIMERA_EINVAL, "null tokens");
    REQUIRE(batch == ctx->batch, CHIMERA_EINVAL, "batch must match the prefilled batch");
    REQUIRE(ctx->N >= 2, CHIMERA_EINVAL, "tree has no draft nodes");
    const size_t cnt = (size_t)batch * (ctx->N - 1);
    for (size_t i = 0; i < cnt; ++i)
      REQUIRE(tokens[i] >= 0 && tokens[i] < ctx->m->cfg.vocab, CHIMERA_EINVAL, "token id out of range");
    HIPCK(hipMemcpy(ctx->inject, tokens, cnt * sizeof(int), hipMemcpyHostToDevice));
    const int one = 1;
    HIPCK(hipMemcpy(ctx->inject_on, &one, sizeof(int), hipMemcpyHostToDevice));
  });
}

chimera_status chimera_debug_copy(chimera_ctx* ctx, int32_t what, void* dst, int64_t bytes) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(dst != nullptr, CHIMERA_EINVAL, "null dst");
    const size_t B = std::max(ctx->batch, 1), N = ctx->N, K = ctx->K, V = ctx->m->cfg.vocab;
    const void* src = nullptr;
    size_t size = 0;
    switch (what) {
      case CHIMERA_DBG_VERIFY_LOGITS: src = ctx->logits; size = B * N * V * 4; break;
      case CHIMERA_DBG_DRAFT_LOGITS:
        REQUIRE(!ctx->branch, CHIMERA_EINVAL, "draft logits are kept by chain drafting only");
        src = ctx->dlogits;
        size = B * K * V * 4;
        break;
      case CHIMERA_DBG_TREE_TOKENS: src = ctx->tree_tok; size = B * N * 4; break;
      case CHIMERA_DBG_DRAFT_LISTS: src = ctx->cand; size = B * 64 * 8 * 4; break;
      case CHIMERA_DBG_SEQ_LEN: src = ctx->n; size = B * 4; break;
      case CHIMERA_DBG_TOKENS: src = ctx->tok; size = B * ctx->tok_stride * 4; break;
      default: throw Err(CHIMERA_EINVAL, "unknown debug buffer");
    }
    REQUIRE((size_t)bytes == size, CHIMERA_EINVAL, "bytes must equal the buffer size (" + std::to_string(size) + ")");
    HIPCK(hipDeviceSynchronize());
    HIPCK(hipMemcpy(dst, src, size, hipMemcpyDeviceToHost));
  });
}

chimera_status chimera_kv_read(chimera_kv* kv, int32_t layer, int32_t b, int32_t pos0, int32_t count, void* k_out,
                               void* v_out) {
  return guard([&] {
    REQUIRE(kv != nullptr && k_out != nullptr && v_out != nullptr, CHIMERA_EINVAL, "null argument");
    const chimera_config& c = kv->m->cfg;
    REQUIRE(layer >= 0 && layer < c.n_layers, CHIMERA_EINVAL, "layer");
    REQUIRE(b >= 0 && b < kv->B, CHIMERA_EINVAL, "sequence");
    REQUIRE(pos0 >= 0 && count >= 0 && pos0 + count <= kv->max_pages * kv->ps, CHIMERA_EINVAL, "position range");
    const size_t es = kv->m->es, H = c.n_heads, hd = c.head_dim;
    HIPCK(hipDeviceSynchronize());
    for (int i = 0; i < count; ++i) {
      const int p = pos0 + i;
      const int page = kv->page_table_host[(size_t)b * kv->max_pages + p / kv->ps];
      for (size_t h = 0; h < H; ++h) {
        const size_t base = (size_t)layer * kv->layer_stride + (size_t)page * kv->page_stride +
                            (h * kv->ps + (size_t)(p % kv->ps)) * hd;
        const size_t vofs = H * kv->ps * hd;
        char* ko = (char*)k_out + (((size_t)i * H + h) * hd) * es;
        char* vo = (char*)v_out + (((size_t)i * H + h) * hd) * es;
        HIPCK(hipMemcpy(ko, (char*)kv->pool + base * es, hd * es, hipMemcpyDeviceToHost));
        HIPCK(hipMemcpy(vo, (char*)kv->pool + (base + vofs) * es, hd * es, hipMemcpyDeviceToHost));
      }
    }
  });
}

chimera_status chimera_profile_enable(chimera_ctx* ctx, int32_t enable) {
  return guard([&] {
    check_ctx(ctx);
    ctx->prof = enable != 0;
    ctx->acc = chimera_profile{};
  });
}

chimera_status chimera_profile_read(chimera_ctx* ctx, chimera_profile* out) {
  return guard([&] {
    REQUIRE(ctx != nullptr && out != nullptr, CHIMERA_EINVAL, "null argument");
    chimera_profile p = ctx->acc;  // eager per-launch GEMM figures
    ctx->acc = chimera_profile{};
    if (ctx->clock_khz <= 0.0) {
      int dev = 0, khz = 0;
      HIPCK(hipGetDevice(&dev));
      HIPCK(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev));
      REQUIRE(khz > 0, CHIMERA_EHIP, "device wall clock rate unknown");
      ctx->clock_khz = khz;
    }
    {
      // phase times of the steps stamped since the previous read (at most the
      // last STAMP_RING of them)
      HIPCK(hipDeviceSynchronize());
      unsigned int last = 0;
      HIPCK(hipMemcpy(&last, ctx->stamp_count, sizeof(unsigned int), hipMemcpyDeviceToHost));
      const unsigned int first = last - ctx->prof_first > (unsigned)STAMP_RING ? last - STAMP_RING : ctx->prof_first;
      std::vector<unsigned long long> ring((size_t)STAMP_RING * STAMP_WORDS);
      HIPCK(hipMemcpy(ring.data(), ctx->stamp_ring, ring.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost));
      std::vector<double> v_ms, s_ms, d_ms;
      for (unsigned int c = first; c != last; ++c) {
        const unsigned long long* t = ring.data() + (size_t)(c % STAMP_RING) * STAMP_WORDS;
        d_ms.push_back((double)(t[1] - t[0]) / ctx->clock_khz);
        v_ms.push_back((double)(t[2] - t[1]) / ctx->clock_khz);
        s_ms.push_back((double)(t[3] - t[0]) / ctx->clock_khz);
        p.ms_draft += d_ms.back();
        p.ms_verify += v_ms.back();
        p.ms_tail += (double)(t[3] - t[2]) / ctx->clock_khz;
        p.verify_bytes += verify_pass_bytes(ctx, (double)t[4]);
        p.steps += 1;
      }
      auto median = [](std::vector<double> x) {
        if (x.empty()) return 0.0;
        std::sort(x.begin(), x.end());
        const size_t h = x.size() / 2;
        return x.size() % 2 ? x[h] : 0.5 * (x[h - 1] + x[h]);
      };
      p.ms_draft_median = median(d_ms);
      p.ms_verify_median = median(v_ms);
      p.ms_step_median = median(s_ms);
      ctx->prof_first = last;
    }
    *out = p;
  });
}

chimera_status chimera_debug_gemm(int32_t dtype, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                                  float* y) {
  return guard([&] {
    REQUIRE(dtype == CHIMERA_F32 || dtype == CHIMERA_BF16, CHIMERA_EINVAL, "dtype");
    REQUIRE(x && w && y, CHIMERA_EINVAL, "null argument");
    const int KB = dtype == CHIMERA_BF16 ? 32 : 16;
    REQUIRE(M >= 1 && M <= 256 && N % 64 == 0 && N > 0 && K % KB == 0 && K > 0, CHIMERA_EINVAL,
            "M in [1, 256], N % 64 == 0, K % KB == 0");
    const size_t es = esize(dtype);
    void *dx = nullptr, *dxr = nullptr, *dw = nullptr, *dp = nullptr, *dy = nullptr, *ds = nullptr;
    auto cleanup = [&] {
      for (void* p : {dx, dxr, dw, dp, dy, ds})
        if (p) (void)hipFree(p);
    };
    try {
      const int mc = mcap(M);
      HIPCK(hipMalloc(&dx, (size_t)mc * K * es));
      HIPCK(hipMemset(dx, 0, (size_t)mc * K * es));
      HIPCK(hipMalloc(&dw, (size_t)K * N * es));
      HIPCK(hipMalloc(&dp, (size_t)K * N * es));
      HIPCK(hipMalloc(&dy, (size_t)M * N * 4));
      HIPCK(hipMalloc(&ds, (size_t)8 * M * N * 4 + 65536 * 4));
      HIPCK(hipMalloc(&dxr, (size_t)M * K * es));
      HIPCK(hipMemcpy(dxr, x, (size_t)M * K * es, hipMemcpyHostToDevice));
      launch_tile_rows(dtype, dxr, M, K, dx, mc / 16, nullptr);
      HIPCK(hipMemcpy(dw, w, (size_t)K * N * es, hipMemcpyHostToDevice));
      launch_repack(dtype, PACK_NATURAL, dw, nullptr, nullptr, K, N, dp, 1, 64, nullptr);
      GemmShape s;
      s.X = dx;
      s.x_mtiles = mc / 16;
      s.M = M;
      s.W = dp;
      s.N = N;
      s.K = K;
      s.splits = gemm_pick_splits(N, K, dtype);
      GemmEpi e;
      e.kind = EPI_F32;
      e.out_f = (float*)dy;
      e.ldo = N;
      e.part = (float*)ds;
      launch_gemm(dtype, s, e, nullptr);
      HIPCK(hipGetLastError());
      HIPCK(hipDeviceSynchronize());
      HIPCK(hipMemcpy(y, dy, (size_t)M * N * 4, hipMemcpyDeviceToHost));
    } catch (...) {
      cleanup();
      throw;
    }
    cleanup();
  });
}

}  // extern "C"

// ---------------------------------------------------------------------------
// GEMM with static scratch (chimera_gemm_static): the tiled copy of x, the
// packed copy of w and the split-K partials live in this file-scope device
// array instead of buffers the call allocates.  Each device holds its own
// copy until the process ends; host code uses its per-device address from
// hipGetSymbolAddress, never the array's name.
// ---------------------------------------------------------------------------
constexpr size_t GEMM_STATIC_SCRATCH_BYTES = (size_t)32 << 20;
static __device__ __align__(256) unsigned char scratch[GEMM_STATIC_SCRATCH_BYTES];

namespace {
constexpr int MAX_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[MAX_DEVICES] = {};

// Device address of `scratch` on the current device, looked up once per device.
char* static_scratch() {
  int dev = -1;
  HIPCK(hipGetDevice(&dev));
  REQUIRE(dev >= 0 && dev < MAX_DEVICES, CHIMERA_EINVAL, "device index out of range");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    HIPCK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    REQUIRE(p != nullptr, CHIMERA_EHIP, "no device address for the static scratch");
    g_scratch_ptr[dev] = p;
  }
  return (char*)g_scratch_ptr[dev];
}

size_t round256(size_t b) { return (b + 255) / 256 * 256; }
}  // namespace

extern "C" {

chimera_status chimera_gemm_static(int32_t dtype, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                                   float* y, void* stream) {
  return guard([&] {
    REQUIRE(dtype == CHIMERA_F32 || dtype == CHIMERA_BF16, CHIMERA_EINVAL, "dtype");
    REQUIRE(x && w && y, CHIMERA_EINVAL, "null argument");
    const int KB = dtype == CHIMERA_BF16 ? 32 : 16;
    REQUIRE(M >= 1 && M <= 256 && N % 64 == 0 && N > 0 && K % KB == 0 && K > 0, CHIMERA_EINVAL,
            "M in [1, 256], N % 64 == 0, K % KB == 0");
    const size_t es = esize(dtype);
    const int mc = mcap(M);
    const int splits = gemm_pick_splits(N, K, dtype);
    const size_t xb = round256((size_t)mc * K * es);
    const size_t wb = round256((size_t)K * N * es);
    const size_t pb = splits > 1 ? (size_t)splits * M * N * sizeof(float) : 0;
    REQUIRE(xb + wb + pb <= GEMM_STATIC_SCRATCH_BYTES, CHIMERA_ENOMEM,
            "tiled x + packed w + split-K partials exceed the 32 MiB static scratch (" +
                std::to_string(xb + wb + pb) + " bytes)");
    hipStream_t st = (hipStream_t)stream;
    char* base = static_scratch();
    // Rows of the last 16-row tile past M keep an earlier call's values; each
    // output row depends only on its own input row and rows >= M are not stored.
    launch_tile_rows(dtype, x, M, K, base, mc / 16, st);
    launch_repack(dtype, PACK_NATURAL, w, nullptr, nullptr, K, N, base + xb, 1, 64, st);
    GemmShape s;
    s.X = base;
    s.x_mtiles = mc / 16;
    s.M = M;
    s.W = base + xb;
    s.N = N;
    s.K = K;
    s.splits = splits;
    GemmEpi e;
    e.kind = EPI_F32;
    e.out_f = y;
    e.ldo = N;
    e.part = (float*)(base + xb + wb);
    launch_gemm(dtype, s, e, st);
    HIPCK(hipGetLastError());
  });
}

chimera_status chimera_set_drafting(chimera_ctx* ctx, int32_t mode) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(mode == CHIMERA_DRAFT_CHAIN || mode == CHIMERA_DRAFT_BRANCH, CHIMERA_EINVAL, "unknown drafting mode");
    drop_graph(ctx);
    const int old = ctx->branch;
    ctx->branch = mode == CHIMERA_DRAFT_BRANCH;
    try {
      set_draft_plan(ctx);
    } catch (...) {
      ctx->branch = old;
      set_draft_plan(ctx);
      throw;
    }
  });
}

chimera_status chimera_set_decoding(chimera_ctx* ctx, int32_t mode, float temperature, float eps, float delta,
                                    uint64_t seed) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(mode == CHIMERA_DECODE_GREEDY || mode == CHIMERA_DECODE_TYPICAL, CHIMERA_EINVAL, "decoding mode");
    if (mode == CHIMERA_DECODE_TYPICAL)
      REQUIRE(temperature > 0.f && eps >= 0.f && delta >= 0.f, CHIMERA_EINVAL,
              "typical decoding needs temperature > 0, eps >= 0, delta >= 0");
    drop_graph(ctx);
    ctx->typical = mode == CHIMERA_DECODE_TYPICAL;
    ctx->temperature = mode == CHIMERA_DECODE_TYPICAL ? temperature : 1.f;
    ctx->t_eps = eps;
    ctx->t_delta = delta;
    ctx->t_seed = seed;
  });
}

static int64_t tri_header_bytes(int64_t n_entries) {
  const int64_t h = n_entries * (int64_t)(sizeof(unsigned long long) + sizeof(unsigned int)) + 256;
  return (h + 255) / 256 * 256;
}

chimera_status chimera_trigram_cache_bytes(const chimera_model* m, int32_t n_entries, int64_t* bytes) {
  return guard([&] {
    REQUIRE(m != nullptr && bytes != nullptr, CHIMERA_EINVAL, "null argument");
    REQUIRE(n_entries >= TRI_WAYS && n_entries % TRI_WAYS == 0, CHIMERA_EINVAL,
            "n_entries must be a positive multiple of 8");
    *bytes = tri_header_bytes(n_entries) + (int64_t)n_entries * m->cfg.d_model * (int64_t)sizeof(float);
  });
}

chimera_status chimera_set_trigram_cache(chimera_ctx* ctx, void* arena, int64_t arena_bytes, int32_t n_entries) {
  return guard([&] {
    check_ctx(ctx);
    drop_graph(ctx);
    if (arena == nullptr) {
      ctx->tri_on = false;
      return;
    }
    REQUIRE(ctx->K > 0, CHIMERA_EINVAL, "the trigram cache needs a draft (tree with more than one node)");
    REQUIRE(ctx->m->cfg.vocab < (1 << 21) - 1, CHIMERA_EINVAL, "vocab too large for the trigram key");
    REQUIRE(n_entries >= TRI_WAYS && n_entries % TRI_WAYS == 0, CHIMERA_EINVAL,
            "n_entries must be a positive multiple of 8");
    const int64_t hb = tri_header_bytes(n_entries);
    const int64_t need = hb + (int64_t)n_entries * ctx->m->cfg.d_model * (int64_t)sizeof(float);
    REQUIRE(arena_bytes >= need, CHIMERA_ENOMEM, "trigram cache arena too small");
    REQUIRE(((uintptr_t)arena & 255) == 0, CHIMERA_EINVAL, "arena must be 256-byte aligned");
    char* p = (char*)arena;
    ctx->tri.keys = (unsigned long long*)p;
    ctx->tri.stamps = (unsigned int*)(p + (size_t)n_entries * sizeof(unsigned long long));
    ctx->tri.clock = (unsigned int*)(p + (size_t)n_entries * (sizeof(unsigned long long) + sizeof(unsigned int)));
    ctx->tri.vals = (float*)(p + hb);
    ctx->tri.n_sets = n_entries / TRI_WAYS;
    HIPCK(hipMemset(arena, 0, (size_t)hb));  // keys (empty), stamps, clock; values are written on insert
    HIPCK(hipMemset(ctx->tri.miss, 0, sizeof(int)));
    HIPCK(hipMemset(ctx->tri.stats, 0, 2 * sizeof(unsigned long long)));
    HIPCK(hipDeviceSynchronize());
    ctx->tri_on = true;
  });
}

chimera_status chimera_compaction_check_bytes(const chimera_ctx* ctx, int64_t* bytes) {
  return guard([&] {
    check_ctx(const_cast<chimera_ctx*>(ctx));
    REQUIRE(bytes != nullptr, CHIMERA_EINVAL, "null argument");
    const chimera_config& cf = ctx->m->cfg;
    // sized for the context's maximum batch, so any prefill batch fits
    *bytes = 256 + (int64_t)cf.n_layers * 2 * ctx->B * ctx->N * cf.n_heads * cf.head_dim * ctx->m->es;
  });
}

chimera_status chimera_set_compaction_check(chimera_ctx* ctx, void* arena, int64_t arena_bytes) {
  return guard([&] {
    check_ctx(ctx);
    drop_graph(ctx);
    if (arena == nullptr) {
      ctx->cc_side = nullptr;
      ctx->cc_counts = nullptr;
      return;
    }
    int64_t need = 0;
    chimera_compaction_check_bytes(ctx, &need);
    REQUIRE(arena_bytes >= need, CHIMERA_ENOMEM, "compaction check arena too small");
    REQUIRE(((uintptr_t)arena & 255) == 0, CHIMERA_EINVAL, "arena must be 256-byte aligned");
    HIPCK(hipMemset(arena, 0, 256));  // the counters
    HIPCK(hipDeviceSynchronize());
    ctx->cc_counts = (unsigned long long*)arena;
    ctx->cc_side = (char*)arena + 256;
  });
}

chimera_status chimera_compaction_check_read(chimera_ctx* ctx, int64_t* rows_checked, int64_t* mismatches) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(rows_checked != nullptr && mismatches != nullptr, CHIMERA_EINVAL, "null argument");
    REQUIRE(ctx->cc_counts != nullptr, CHIMERA_ESTATE, "compaction check is not enabled");
    unsigned long long c[2] = {0, 0};
    HIPCK(hipDeviceSynchronize());
    HIPCK(hipMemcpy(c, ctx->cc_counts, sizeof(c), hipMemcpyDeviceToHost));
    *rows_checked = (int64_t)c[0];
    *mismatches = (int64_t)c[1];
  });
}

chimera_status chimera_trigram_cache_stats(chimera_ctx* ctx, int64_t* lookups, int64_t* hits) {
  return guard([&] {
    check_ctx(ctx);
    REQUIRE(lookups != nullptr && hits != nullptr, CHIMERA_EINVAL, "null argument");
    unsigned long long st[2] = {0, 0};
    HIPCK(hipMemcpy(st, ctx->tri.stats, sizeof(st), hipMemcpyDeviceToHost));
    *lookups = (int64_t)st[0];
    *hits = (int64_t)st[1];
  });
}

chimera_status chimera_set_graph(chimera_ctx* ctx, int32_t enable) {
  return guard([&] {
    check_ctx(ctx);
    drop_graph(ctx);
    ctx->graph_on = enable != 0;
  });
}

void chimera_ctx_free(chimera_ctx* ctx) {
  if (!ctx) return;
  drop_graph(ctx);
  if (ctx->host_result) (void)hipHostFree(ctx->host_result);
  if (ctx->host_pipe) (void)hipHostFree(ctx->host_pipe);
  if (ctx->ev_created) {
    for (auto& e : ctx->ev_pool) {
      (void)hipEventDestroy(e.a);
      (void)hipEventDestroy(e.b);
    }
  }
  delete ctx;
}

void chimera_kv_free(chimera_kv* kv) { delete kv; }
void chimera_free(chimera_model* m) { delete m; }

}  // extern "C"
