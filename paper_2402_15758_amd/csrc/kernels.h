// Launch interface of the gfx950 kernels used by the host engine.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

enum { DT_F32 = 0, DT_BF16 = 1 };

// ---- GEMM ------------------------------------------------------------------
// Y = X[M][K] @ W[K][N] with W repacked into 1 KiB tiles: tile (nb, kb) holds
// columns [16 nb, 16 nb + 16) and reduction indices [kb KB, kb KB + KB),
// KB = 4 * VEC (32 for bf16, 16 for f32); lane l's 16 bytes are
// W[kb KB + (l >> 4) VEC + e][16 nb + (l & 15)], e < VEC.  Tiles of one
// column block are contiguous along kb, so a workgroup streams them linearly.
enum { PACK_NATURAL = 0, PACK_QKV = 1, PACK_GU = 2 };
// PACK_QKV puts both halves of 8 rotary pairs in one 16-column block: for
// Q and K, block q of a head holds dims 8q + l (lane column l < 8) and
// hd/2 + 8q + l - 8 (l >= 8); V keeps its natural order.  PACK_GU puts gate
// columns 8c + l (l < 8) and up columns 8c + l - 8 (l >= 8) in block c.  The
// epilogue pairs lane columns l and l ^ 8.

enum { EPI_F32 = 0, EPI_T = 1, EPI_SILU = 2, EPI_SWIGLU = 3, EPI_QKV = 4, EPI_PARTIAL = 5 };

struct GemmEpi {
  int kind = EPI_F32;
  float* out_f = nullptr;  // EPI_F32: row-major [M][ldo]
  int ldo = 0;
  void* out_t = nullptr;   // EPI_T / EPI_SILU / EPI_SWIGLU: tiled storage-type output
  int o_mtiles = 0;        //   with this many 16-row tiles
  float* part = nullptr;   // EPI_PARTIAL: [splits][M][N] (packed column order); other
                           // epilogues with split-K: scratch of the same shape
  // EPI_QKV: per-row rotary position, KV element offset (-1: skip) and
  // Q output row (-1: skip); K/V go to kbase/vbase + kvoff + h*head_stride.
  const int* pos = nullptr;
  const int64_t* kvoff = nullptr;
  const int* qrow = nullptr;
  void* kbase = nullptr;
  void* vbase = nullptr;
  int64_t head_stride = 0;
  void* qout = nullptr;    // row-major [rows][ldq]
  int ldq = 0;
  const float* rcos = nullptr;  // [max_pos][hd/2]
  const float* rsin = nullptr;
  int H = 0, hd = 0;
};

struct GemmShape {
  const int* skip = nullptr;  // optional: the launch does nothing when *skip == 0 (device int)
  const void* X = nullptr;  // tiled activations
  int x_mtiles = 0;         // 16-row tiles of X's buffer
  int M = 0;
  const void* W = nullptr;  // packed
  int N = 0;                // packed columns of the whole matrix
  int K = 0;
  int nb_off = 0;           // first 16-column block to compute
  int nb_count = 0;         // number of 16-column blocks to compute; 0 = all
  int splits = 1;           // split of the reduction across workgroups
};

// Splits chosen from (N, K) only, never from M; at most GEMM_MAX_SPLITS (the
// consumers of split-K partials load them all at once).
constexpr int GEMM_MAX_SPLITS = 8;
int gemm_pick_splits(int n_cols, int K, int dtype);
// ev_start / ev_stop (optional): recorded by the dispatch of the GEMM's
// first and last kernel (hipExtLaunchKernel), i.e. the kernel execution span.
void launch_gemm(int dtype, const GemmShape& s, const GemmEpi& e, hipStream_t st, hipEvent_t ev_start = nullptr,
                 hipEvent_t ev_stop = nullptr);
void launch_repack(int dtype, int kind, const void* src0, const void* src1, const void* src2, int K, int n_src,
                   void* dst, int H, int hd, hipStream_t st);
// Row-major [M][K] -> tiled (test hook and one-off conversions).
void launch_tile_rows(int dtype, const void* src, int M, int K, void* dst, int mtiles, hipStream_t st);

// ---- elementwise / norms ------------------------------------------------------
void launch_embed(int dtype, const int* tokens, const void* E, float* x, int M, int d, int V, hipStream_t st);
// x[r] += sum_s parts[s][r] (if parts), optionally written back; out (tiled,
// o_mtiles tiles) row r = T(rmsnorm(x[r]) * gamma), and the same values
// row-major into out_rm if given.  Rows r in [alt_begin, alt_end) read their
// input from row-major alt[(r - alt_begin)] (storage type) instead of x.
void launch_rmsnorm(int dtype, float* x, const float* parts, int n_parts, const float* gamma, void* out, int o_mtiles,
                    void* out_rm, int M, int d, float eps, int write_back, const void* alt, int alt_begin,
                    int alt_end, hipStream_t st);

// ---- attention ---------------------------------------------------------------
// The shared pass of the tree attention writes one partial per group of
// 64-position chunks.  Groups are fixed by absolute chunk index: chunks
// 0 .. TREE_ATTN_NEAR_CHUNKS-1 form pairs; later chunks form groups of
// TREE_ATTN_FAR_GROUP (fewer partials where contexts are long).
constexpr int TREE_ATTN_NEAR_CHUNKS = 16;
constexpr int TREE_ATTN_FAR_GROUP = 4;
// Group slots covering positions 0 .. max_len - 1.
inline int tree_attn_groups(int max_len) {
  const int chunks = (max_len + 63) / 64;
  if (chunks <= TREE_ATTN_NEAR_CHUNKS) return (chunks + 1) / 2;
  return TREE_ATTN_NEAR_CHUNKS / 2 + (chunks - TREE_ATTN_NEAR_CHUNKS + TREE_ATTN_FAR_GROUP - 1) / TREE_ATTN_FAR_GROUP;
}
struct TreeAttnArgs {
  const void* q;            // [B*N][ldq] rotated queries
  int ldq;
  const void* kpool;        // layer base of K in the paged pool
  const void* vpool;        // layer base of V
  int64_t page_stride;      // elements between consecutive pages
  const int* page_table;    // [B][max_pages]
  int max_pages;
  const int* n_b;           // [B] committed length
  const int* depth;         // [N]
  const uint8_t* path;      // [N][64]: node at each depth on the root->u path
  int N, H, hd, ps, D;      // D = deepest node depth of the tree
  float scale;
  float* part_o;            // [B][H][G][N][hd]
  float* part_ml;           // [B][H][G][N][2]
  int G;                    // group slots (tree_attn_groups)
  void* out;                // tiled [B*N][H*hd] with o_mtiles tiles
  int o_mtiles;
  int B;
  const int64_t* rowtab;    // [B][TREE_ATTN_TAIL_ROWS] from launch_attn_rows
};
void launch_tree_attn(int dtype, const TreeAttnArgs& a, hipStream_t st);
// Each query reduces the keys at positions P_u - W + 1 .. P_u (W = this
// window) itself; the keys before them go through the shared MFMA pass.  W
// exceeds the depth of every tree (at most 8 levels), so the shared keys of a
// tree query are committed ones; a prefill chain (node j at position n + j)
// keeps its own positions in place and may be deeper.
constexpr int TREE_ATTN_WINDOW = 16;
// Window row table per sequence: entry k < W is position n - W + k, entry
// W + j the slot of tree node j.
constexpr int TREE_ATTN_TAIL_ROWS = TREE_ATTN_WINDOW + 64;
// rowtab[b][rr] = page-resolved element offset (head and layer excluded) of
// window row rr, written once per verify pass for all layers.
void launch_attn_rows(const int* n_b, const int* page_table, int max_pages, int ps, int64_t page_stride, int hd,
                      int N, int B, int64_t* rowtab, hipStream_t st);

// Query row r = b * R + i of draft level `level` is draft-tree node
// nodes[i] of sequence b, at trigram position n_b + level.  Its keys, in
// order: target-state entries 0..n-1, trigram entries 0..n (stream 1), then
// the trigram entries of its ancestors-or-self at depths 1..level, kept in
// stream-1 slots tree_slot0 + node.
struct EncAttnArgs {
  const void* q;            // [B*R][ldq]
  int ldq;
  const void* kbase;        // encoder memory K [B][2][H][cap][hd]
  const void* vbase;
  int cap;
  const int* n_b;           // [B]
  int level;
  const int* nodes;         // [R] drafted draft-tree nodes of this level
  int R;
  const uint8_t* path;      // [64][64] draft-tree node at each depth on the root->u path
  int tree_slot0;
  int H, hd;
  float scale;
  float* part;              // [B*R][H][nblk][hd + 2]
  int nblk;
  void* out;                // tiled [B*R][H*hd] with o_mtiles tiles
  int o_mtiles;
  int B;
};
void launch_enc_attn(int dtype, const EncAttnArgs& a, hipStream_t st);

// ---- decode-state kernels ------------------------------------------------------
struct StepState {
  int B, N, K, d, V, H, hd, ps, max_pages, tok_stride, cap;
  int64_t page_stride;      // elements between pages in the target pool
  int* n;                   // [B]
  int* tok;                 // [B][tok_stride]: committed tokens, pending, chain tokens
  void* h_last;             // [B][d]
  const int* page_table;    // [B][max_pages]
  const int* t_parent;      // [N]
  const int* t_depth;       // [N]
  const int* t_rank;        // [N]
  const unsigned long long* t_anc;  // [N]
  int* s_k;                 // [K] candidates per head
  int* cand;                // [B][64][8]: top-s list of each drafted draft-tree node
  int* tree_tok;            // [B*N]
  const int* inject;        // [B][N-1] injected tree tokens
  int* inject_on;           // [1]
  const int* f_ref;         // forcing reference [B][f_stride] (nullable)
  const uint8_t* f_ok;
  int f_stride;
  int* out_tok;             // [B][K+1]
  int* out_nodes;           // [B][K+1]
  int* out_len;             // [B]
  int* pro_base;            // [B]
  int* pro_count;           // [B]
  void* pro_h;              // [B][K+1][d]
  const void* hl;           // [B*N][d] post-final-norm verify states (row-major)
  const int* amax;          // [B*N]
  // verify row descriptors
  int* v_pos;               // [B*N]
  int64_t* v_kvoff;         // [B*N]
  int* v_qrow;              // [B*N]
  // typical decoding (typical != 0): the verify logits, their per-row
  // log-sum-exp and entropy at temperature 1 / inv_T, and each row's sample
  int typical;
  float inv_T, eps, delta;
  const float* logits;      // [B*N][V]
  const double* t_lse;      // [B*N]
  const double* t_H;        // [B*N]
  const int* t_sample;      // [B*N]
  // drafting plan.  The draft tree is the rank-0 chain (chain drafting: node
  // k at depth k) or the verify tree itself (branch-conditioned drafting).
  // Level k drafts the depth-k draft-tree nodes that have children.
  const int* d_nodes;       // [64] drafted draft-tree nodes, level by level
  const int* d_parent;      // [64] draft-tree parent
  const int* d_rank;        // [64] draft-tree rank
  const uint8_t* d_path;    // [64][64] draft-tree node at each depth on the root->u path
  const int* tok_src;       // [N] verify node -> the cand row holding its token (rank t_rank)
  int tree_slot0;           // stream-1 slot of draft-tree node 0 in the encoder memory
};
// One draft level: R drafted nodes per sequence, s.d_nodes[off .. off + R).
// Query rows r = b * R + i; at level 0 (R = 1) the prologue rows follow.
struct DraftLevel {
  int level, R, off;
};
// Per row r of logits [rows][V]: at temperature 1 / inv_T, lse = log sum_v
// exp(z_v), H = the entropy of softmax(z), and sample = the Gumbel-max sample
// (argmax_v z_v - log(-log(u_v)), u_v from the SplitMix64 chain keyed by
// (seed, sequence, position, v)) for sequence b0 + r / N at position
// n_b[b] + depth[r % N] + 1, or at fixed_pos when fixed_pos >= 0.
void launch_typical_stats(const float* logits, int rows, int V, int N, int b0, const int* n_b, const int* depth,
                          int fixed_pos, float inv_T, unsigned long long seed, double* lse, double* H, int* sample,
                          hipStream_t st);
void launch_argmax(const float* logits, int M, int V, int* amax, hipStream_t st);
// Per query row r of level lv: the top-s list of z = logits + r * ld into
// cand[b][node] (forced as set up in s).  scratch: [B*R][32][8] values and ids.
void launch_topk(const float* logits, int64_t ld, const StepState& s, const DraftLevel& lv, float* scratch_v,
                 int* scratch_i, hipStream_t st);
void launch_tree_setup(const StepState& s, hipStream_t st);
void launch_accept(int dtype, const StepState& s, hipStream_t st);
void launch_compact(int dtype, const StepState& s, void* pool, int n_layers, int64_t layer_stride, hipStream_t st);
// Compaction check: the tree's K/V rows of every layer copied to side
// [layer][kv][B][N][H*hd] before compaction, compared with the accepted
// path's slots after it (counts[0] += rows, counts[1] += differing chunks).
void launch_kv_snapshot(int dtype, const StepState& s, const void* pool, int n_layers, int64_t layer_stride,
                        void* side, hipStream_t st);
void launch_kv_check(int dtype, const StepState& s, const void* pool, int n_layers, int64_t layer_stride,
                     const void* side, unsigned long long* counts, hipStream_t st);
void launch_advance(int dtype, const StepState& s, hipStream_t st);

// Rows of draft level lv.  Rows [0, B R) are the queries (trigram position
// n + level along each drafted node's path).  At level 0 rows
// [B, B + B(K+1)) are the previous step's committed target-state entries
// and rows [B + B(K+1), B + 2B(K+1)) their trigram entries.  Writes the
// trigram inputs [rows][3d], rotary positions, encoder-memory offsets and Q rows.
int draft_level_rows(const StepState& s, const DraftLevel& lv);
void launch_draft_rows(int dtype, const StepState& s, const void* E, const DraftLevel& lv, void* tri_in,
                       int tri_mtiles, int* pos, int64_t* kvoff, int* qrow, hipStream_t st);
// zin[r] (tiled) = [h_last[b]; T(x[r] + sum_s parts[s][r])], r = b R + i,
// parts [n_parts][B R][d]
void launch_draft_finish(int dtype, const StepState& s, const DraftLevel& lv, const float* x, const float* parts,
                         int n_parts, void* zin, int z_mtiles, hipStream_t st);
// Prefill chunk rows: positions p0 .. p0+M-1 of sequence b; writes verify
// descriptors (pos, kvoff through the page table, qrow), the token list,
// trigram inputs for the same positions and the encoder descriptors of the
// target-state rows [0, M) and trigram rows [M, 2M).
void launch_prefill_rows(int dtype, const StepState& s, const void* E, int b, int p0, int M, int* tokens_out,
                         void* tri_in, int tri_mtiles, int* enc_pos, int64_t* enc_kvoff, int* enc_qrow, int* pf_n,
                         hipStream_t st);
// Prefill end: pending token, h_last, committed length and tokens.
// ---- trigram lookup cache (exact memoization of the trigram encoder) -------
// Set-associative with TRI_WAYS ways and least-recently-used replacement.
// Key of the trigram ending at position p: token ids + 1 of positions p-2,
// p-1, p (0 before the sequence start) packed into 21 bits each.
constexpr int TRI_WAYS = 8;
struct TriCache {
  unsigned long long* keys = nullptr;   // [n_sets][TRI_WAYS], 0 = empty
  unsigned int* stamps = nullptr;       // [n_sets][TRI_WAYS], last use
  float* vals = nullptr;                // [n_sets][TRI_WAYS][d]: trigram encoder outputs
  unsigned int* clock = nullptr;        // [1]
  int n_sets = 0;
  int* hit = nullptr;                   // [rows]: 1 = row filled from the cache or needs no trigram
  int* miss = nullptr;                  // [1]: rows left for the trigram MLP (0 skips it)
  unsigned long long* stats = nullptr;  // [2]: lookups, hits
};
// Draft level lv: look up the trigram rows of draft_rows (query rows and
// committed trigram rows), copy hits into htri rows [r][d].
void launch_tri_lookup(const StepState& s, const TriCache& c, const DraftLevel& lv, float* htri, hipStream_t st);
// Insert the rows the MLP computed: draft level (prefill_M = 0, rows as in
// draft_rows, values htri[r]) or a prefill chunk of sequence b at positions
// p0 .. p0+prefill_M-1 (values vals[i]).  Resets the miss count.
void launch_tri_insert(const StepState& s, const TriCache& c, const DraftLevel& lv, int b, int p0, int prefill_M,
                       const float* vals, hipStream_t st);

void launch_prefill_finish(int dtype, const StepState& s, int b, int n, const int* amax_row, const void* hl_row,
                           hipStream_t st);

// ---- phase timestamps -------------------------------------------------------
// Every step writes one ring slot of STAMP_WORDS words: the device wall clock
// (hipDeviceAttributeWallClockRate kHz) at step start (0), draft end (1),
// verify end (2) and step end (3), and the step's summed committed length
// (4).  A stamp runs after every earlier kernel of the stream has finished;
// stamp 3 advances the step counter.
constexpr int STAMP_RING = 4096;
constexpr int STAMP_WORDS = 8;
void launch_stamp(unsigned long long* ring, unsigned int* counter, int idx, const int* n_b, int B, hipStream_t st);
