/*
 * chimera.h -- C ABI of an MI355X (gfx950) implementation of one Chimera
 * decode step (Zeng et al., arXiv 2402.15758).
 *
 * One step is the paper's draft-then-verify iteration (Sec. 3.1, "Drafting"
 * and "Verification"): the lightweight draft (Sec. 4.1: trigram encoder,
 * Eq. 2; full-context encoder, Eq. 3; residual decoding heads, Eq. 4)
 * proposes per-head top-k candidates that form a static token tree
 * (Sec. 4.4); the target model scores the whole tree in one forward pass
 * with tree-structured attention (Sec. 4.3); the longest path whose tokens
 * equal the target's greedy choices is accepted (Sec. 4.3, greedy decoding)
 * and its keys/values are compacted in place in the paged KV cache.
 *
 * Conventions for every call:
 *  - All device memory is allocated by the caller (arena pointers) and only
 *    borrowed by the library until the matching *_free call; the library
 *    never frees caller memory.  Arena sizes come from the *_bytes queries.
 *  - Streams are hipStream_t passed as void*; NULL means the null stream.
 *  - Every call returns a chimera_status; nothing aborts or throws across the
 *    ABI.  chimera_last_error() returns a thread-local message for the last
 *    failure on the calling thread.
 *  - Inputs are validated before any launch; on a validation error no state
 *    changes.  An asynchronous HIP error surfaces as CHIMERA_EHIP at the
 *    call's final synchronisation and poisons the context (later calls on it
 *    return CHIMERA_ESTATE).
 *  - A context is used by one host thread at a time.
 */
#ifndef CHIMERA_H
#define CHIMERA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct chimera_model chimera_model; /* weights; read-only after load */
typedef struct chimera_kv chimera_kv;       /* paged target KV + draft-encoder memory */
typedef struct chimera_ctx chimera_ctx;     /* per-batch decode state and workspaces */

typedef enum {
  CHIMERA_OK = 0,
  CHIMERA_EINVAL = -1,    /* bad argument, shape, token id or tree */
  CHIMERA_ENOMEM = -2,    /* arena too small */
  CHIMERA_ECAPACITY = -3, /* a sequence would outgrow its KV capacity */
  CHIMERA_EHIP = -4,      /* a HIP runtime call or kernel failed */
  CHIMERA_ESTATE = -5     /* context poisoned by an earlier HIP failure, or call out of order */
} chimera_status;

typedef enum { CHIMERA_F32 = 0, CHIMERA_BF16 = 1 } chimera_dtype;

/* Shapes.  The target is a Llama-style decoder (the paper's backbones,
 * Table 1): pre-RMSNorm blocks with multi-head attention and rotary
 * positions (rotate-half pairs (i, i + head_dim/2), angle p * base^(-2i/hd)),
 * SwiGLU feed-forward, final RMSNorm and an untied LM head.  The draft is the
 * trigram MLP (Eq. 2), one encoder block of the same shape (Eq. 3) and
 * n_draft_heads heads A_k (2d -> d), SiLU, Theta_k (d -> V) (Eq. 4). */
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab, n_draft_heads;
  float rope_base; /* 10000 */
  float rms_eps;   /* 1e-5 */
  int32_t dtype;   /* chimera_dtype of weights and stored activations */
  int32_t max_positions; /* size of the rotary tables: positions 0..max_positions-1 */
} chimera_config;

/* One weight tensor.  Names and shapes follow the canonical list:
 *   tok_embed [V, d];
 *   layers.{l}.{attn_norm [d], wq|wk|wv [d, H*hd], wo [H*hd, d], ffn_norm [d],
 *               w_gate|w_up [d, F], w_down [F, d]};
 *   final_norm [d]; lm_head [d, V];
 *   draft.tri_w1 [3d, d]; draft.tri_w2 [d, d];
 *   draft.enc.{same nine tensors as a layer};
 *   draft.heads.{k}.a [2d, d]; draft.heads.{k}.theta [d, V].
 * Matrices are row-major [d_in, d_out] (y = x @ W).  Norm gains are always
 * float32; every other tensor has the config's dtype. */
typedef struct {
  const char* name;
  const void* data;
  int64_t numel;
  int32_t dtype;     /* chimera_dtype */
  int32_t on_device; /* must be 1: data is device memory (host tensors give CHIMERA_EINVAL) */
} chimera_tensor;

/* Bytes of the weight arena for this config (repacked weights + rotary
 * tables). */
chimera_status chimera_weight_bytes(const chimera_config* cfg, int64_t* bytes);

/* Validate the tensor list and repack every tensor into `arena` (device
 * memory of at least chimera_weight_bytes) in the order the GEMM kernels
 * stream it.  Every tensor must already be in device memory; the call reads
 * each once, allocates nothing, and the caller may free them after it
 * returns.  Synchronises `stream`. */
chimera_status chimera_load(const chimera_config* cfg, const chimera_tensor* tensors, int32_t n_tensors,
                            void* arena, int64_t arena_bytes, void* stream, chimera_model** out);

/* Paged target KV (page_size tokens per page, all layers, K and V) for up to
 * max_batch sequences of at most max_len positions each, plus the draft
 * encoder's memory.  n_pages must cover max_batch * ceil(max_len/page_size). */
chimera_status chimera_kv_bytes(const chimera_model* m, int32_t max_batch, int32_t max_len, int32_t n_pages,
                                int32_t page_size, int64_t* bytes);
/* page_order (host, n_pages entries, nullable): the order in which physical
 * pages are handed to sequences; NULL means 0, 1, 2, ... */
chimera_status chimera_kv_create(chimera_model* m, int32_t max_batch, int32_t max_len, int32_t n_pages,
                                 int32_t page_size, const int32_t* page_order, void* arena, int64_t arena_bytes,
                                 chimera_kv** out);

/* Decode context for a static candidate tree of n_nodes nodes (root
 * included, n_nodes <= 64).  Node i has parent parent[i] (< i; -1 for the
 * root, node 0) and takes the rank[i]-th candidate (rank < 8) of draft head
 * depth(i)-1; siblings must have distinct ranks and depth(i) <=
 * n_draft_heads.  n_nodes == 1 gives plain greedy autoregressive decoding
 * (no draft). */
chimera_status chimera_ctx_bytes(const chimera_model* m, const chimera_kv* kv, int32_t n_nodes, int64_t* bytes);
chimera_status chimera_ctx_create(chimera_model* m, chimera_kv* kv, const int32_t* parent, const int32_t* rank,
                                  int32_t n_nodes, void* arena, int64_t arena_bytes, chimera_ctx** out);

/* Prefill (the prefix X, Sec. 4.1.1): run the target over each prompt,
 * fill its KV pages and the draft encoder's memory, and return the first
 * generated token of every sequence.  tokens (host) holds the prompts
 * back to back; lens (host) their lengths (>= 1); batch <= max_batch.
 * Synchronises `stream`. */
chimera_status chimera_prefill(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, const int32_t* tokens,
                               const int32_t* lens, int32_t batch, int32_t* first_tokens, void* stream);

/* One draft -> verify -> accept -> compact iteration for every sequence.
 * Outputs (host): new_tokens [batch][K+1] -- the accepted draft tokens in
 * depth order followed by the bonus token (the target's argmax after the
 * accepted path); n_new [batch] -- their count L, 1 <= L <= K+1; path_nodes
 * [batch][K+1] (nullable) -- the accepted tree node ids from the root in
 * depth order (L entries), i.e. the tree KV slots that were compacted.  The
 * generated stream is the prefill token followed by every step's
 * new_tokens; with greedy verification it equals greedy autoregressive
 * decoding.  K = tree depth.  Synchronises `stream`. */
chimera_status chimera_step(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, int32_t* new_tokens,
                            int32_t* n_new, int32_t* path_nodes, void* stream);

/* Pipelined decoding: n_steps consecutive chimera_step iterations enqueued
 * back to back on `stream`, each step's results copied asynchronously to
 * its own host slot, with one synchronisation at the end.  Every input a
 * step needs lives in device memory, so no step waits for the host.
 * Outputs (host): new_tokens [n_steps][batch][K+1], n_new [n_steps][batch],
 * path_nodes [n_steps][batch][K+1] (nullable), each step as chimera_step
 * reports it.  n_steps in [1, CHIMERA_MAX_PIPELINED_STEPS]; the capacity
 * check assumes every step accepts K+1 tokens (CHIMERA_ECAPACITY before
 * any launch otherwise).  Results are identical to n_steps chimera_step
 * calls.  Synchronises `stream`. */
#define CHIMERA_MAX_PIPELINED_STEPS 64
chimera_status chimera_steps(chimera_model* m, chimera_kv* kv, chimera_ctx* ctx, int32_t n_steps, int32_t* new_tokens,
                             int32_t* n_new, int32_t* path_nodes, void* stream);

/* ---- benchmarking and parity hooks --------------------------------------
 * Forced acceptance (synthetic workloads): at draft level k of a step with
 * committed length n the predicted position is j = n+1+k; if ok[b*stride+j]
 * the level's candidate list becomes ref[b*stride+j] followed by the best
 * remaining ids, otherwise the best ids excluding ref[b*stride+j].  ref and
 * ok are caller-owned device arrays [batch][stride] that must stay valid
 * while forcing is set.  ref == NULL disables forcing. */
chimera_status chimera_set_forcing(chimera_ctx* ctx, const int32_t* ref, const uint8_t* ok, int32_t stride);

/* Replace the draft's tree tokens for nodes 1..n_nodes-1 of the next step
 * only (host array [batch][n_nodes-1]); the root stays the pending token. */
chimera_status chimera_set_tree_tokens(chimera_ctx* ctx, const int32_t* tokens, int32_t batch);

enum {
  CHIMERA_DBG_VERIFY_LOGITS = 0, /* float32 [batch*n_nodes][V], last step */
  CHIMERA_DBG_DRAFT_LOGITS = 1,  /* float32 [batch][K][V], last step */
  CHIMERA_DBG_TREE_TOKENS = 2,   /* int32 [batch][n_nodes], last step */
  CHIMERA_DBG_DRAFT_LISTS = 3,   /* int32 [batch][64][8], last step's top-s list of each drafted node
                                    (chain drafting: row k = head k; branch: row u = tree node u) */
  CHIMERA_DBG_SEQ_LEN = 4,       /* int32 [batch], committed length n */
  CHIMERA_DBG_TOKENS = 5         /* int32 [batch][max_len + 8], committed tokens then pending */
};
/* Copy a debug buffer to host memory (bytes must equal its size). */
chimera_status chimera_debug_copy(chimera_ctx* ctx, int32_t what, void* dst, int64_t bytes);

/* Read the target K and V of `count` positions starting at pos0 of
 * sequence b in layer `layer` through the page table, into host arrays
 * [count][H][hd] of the model dtype. */
chimera_status chimera_kv_read(chimera_kv* kv, int32_t layer, int32_t b, int32_t pos0, int32_t count, void* k_out,
                               void* v_out);

/* Per-phase timing of steps.  Phases: draft, verify (tree pass + LM head +
 * argmax), tail (accept, compact, advance).  Every step (graph replay or
 * eager launches) runs a one-lane kernel at each phase boundary that
 * records the device wall clock into a ring of the last 4096 steps, so a
 * replayed graph is timed as it runs.  chimera_profile_read synchronises the
 * device and reports the steps stamped since its previous call (or since
 * the context was created; at most the last 4096), then starts a new window.
 * chimera_profile_enable(ctx, 1) only adds per-launch HIP events to every
 * verify-pass GEMM launched eagerly (chimera_set_graph(ctx, 0)): the
 * ms_gemm_verify, gemm_verify_launches and gemm_verify_bytes fields, summed
 * since the previous read (zero under graph replay). */
typedef struct {
  int64_t steps;
  double ms_draft, ms_verify, ms_tail, ms_gemm_verify;  /* sums over the steps */
  int64_t gemm_verify_launches;
  double gemm_verify_bytes; /* algorithmic bytes of those launches: weights + activations in/out */
  double verify_bytes;      /* algorithmic bytes of the verify passes: weights, KV read and write */
  double ms_draft_median, ms_verify_median, ms_step_median; /* per-step medians (step: first to last stamp) */
} chimera_profile;
chimera_status chimera_profile_enable(chimera_ctx* ctx, int32_t enable);
chimera_status chimera_profile_read(chimera_ctx* ctx, chimera_profile* out);

/* Launch mode of chimera_step: 1 (default) captures the step's launch
 * sequence once into a HIP graph and replays it every step (recaptured after
 * prefill, set_forcing, set_drafting, set_decoding, set_trigram_cache or a
 * stream change; needs a non-null stream); 0 launches every kernel
 * individually.  Results are identical. */
chimera_status chimera_set_graph(chimera_ctx* ctx, int32_t enable);

/* Verification rule (Sec. 4.3; Sec. 5.1 tests greedy and typical decoding at
 * T = 1).  CHIMERA_DECODE_GREEDY (the default) accepts the longest path of
 * target argmax tokens and is lossless against greedy decoding.
 * CHIMERA_DECODE_TYPICAL selects candidates by their probability under the
 * target at the given temperature:
 *  - a draft node passes when p_parent(token) > min(eps, delta * exp(-H)),
 *    H the entropy of the parent's distribution (the rule the paper takes
 *    from Medusa, which it does not spell out; 0.09 and 0.3 are the usual
 *    values);
 *  - the deepest node whose whole path passes is accepted (ties: higher path
 *    log-probability, then lower node id);
 *  - the bonus token, and the first token after a prompt, are sampled by the
 *    Gumbel-max trick.  u_v uses the top 53 bits of
 *    SplitMix64(SplitMix64(SplitMix64(SplitMix64(seed) ^ b) ^ position) ^ v),
 *    b the sequence, position the token's position, v the token id.
 * Not lossless: the stream is a sample, reproducible from the seed.
 * Takes effect from the next prefill or step. */
enum { CHIMERA_DECODE_GREEDY = 0, CHIMERA_DECODE_TYPICAL = 1 };
chimera_status chimera_set_decoding(chimera_ctx* ctx, int32_t mode, float temperature, float eps, float delta,
                                    uint64_t seed);

/* Drafting (Sec. 4.1, Sec. 4.4).  CHIMERA_DRAFT_CHAIN (the default) runs the
 * K draft levels along the rank-0 chain: head k reads the encoder output at
 * the position the rank-0 tokens of heads 0..k-1 reach, and its top-s list
 * fills every tree node at depth k + 1 (rank r: the list's rank-r token).
 * CHIMERA_DRAFT_BRANCH (branch-conditioned drafting) runs level k once for
 * every depth-k tree node that has children, along that node's own tokens:
 * its trigram uses its path tokens, its encoder query sees the target-state
 * entries 0..n-1, the trigram entries 0..n and its ancestors' speculative
 * trigram entries (the tree mask of Sec. 4.3 applied to the encoder), and a
 * child of rank r takes the rank-r token of its parent's own list.  Both are
 * lossless under greedy verification; on a chain-shaped tree they are the
 * same computation.  Branch-conditioned levels run B times the level's
 * drafted nodes as GEMM rows, so the weight bytes per level stay those of
 * the chain.  Forcing (chimera_set_forcing) biases every drafted node's
 * list of a level alike.  CHIMERA_DBG_DRAFT_LOGITS is kept by chain
 * drafting only.
 * CHIMERA_EINVAL for an unknown mode.  Takes effect from the next step. */
enum { CHIMERA_DRAFT_CHAIN = 0, CHIMERA_DRAFT_BRANCH = 1 };
chimera_status chimera_set_drafting(chimera_ctx* ctx, int32_t mode);

/* Trigram lookup cache (Sec. 4.1.1: a fixed-size dictionary of trigram
 * encoder outputs with least-recently-used replacement).  The cache holds
 * n_entries outputs of Eq. 2 (float32, d_model each) in 8-way sets keyed by
 * the trigram's three token ids.  While attached:
 *  - prefill inserts the prompt's trigrams;
 *  - every draft level looks its trigram rows up first, and the trigram MLP
 *    is skipped when every row hits;
 *  - the rows it does compute are inserted, evicting a set's least recently
 *    used entry.
 * It is exact memoization: tokens, trees and logits are bit-identical with
 * and without it.  Evicted entries are dropped; a later miss recomputes
 * them.  The arena (device memory of chimera_trigram_cache_bytes, 256-byte
 * aligned) is owned by the caller and borrowed until it is detached
 * (arena == NULL) or the context is freed.  n_entries: a positive multiple of
 * 8.  Needs a draft (n_nodes > 1) and vocab < 2^21 - 1; CHIMERA_EINVAL
 * otherwise, CHIMERA_ENOMEM if the arena is too small.  Attaching empties the
 * cache and synchronises the device. */
chimera_status chimera_trigram_cache_bytes(const chimera_model* m, int32_t n_entries, int64_t* bytes);
chimera_status chimera_set_trigram_cache(chimera_ctx* ctx, void* arena, int64_t arena_bytes, int32_t n_entries);
/* Cumulative draft-level trigram lookups and hits since the cache was attached. */
chimera_status chimera_trigram_cache_stats(chimera_ctx* ctx, int64_t* lookups, int64_t* hits);

/* DEBUG MODE -- compaction check (race detection for the in-place KV
 * compaction after acceptance, Sec. 4.3).  While a side arena is attached,
 * every step copies the K and V rows of all tree nodes (slots n..n+N-1,
 * every layer and head) into the arena after the verify pass, and after the
 * compaction compares slot n+d of every sequence and layer with the copy of
 * the accepted path's node path[d], d = 0..L-1.  The arena (device memory of
 * chimera_compaction_check_bytes: 256 bytes of counters, then
 * [layer][K|V][batch][node][heads * head_dim] in the storage type for the
 * context's maximum batch; 256-byte aligned) is owned by the caller and borrowed until it is detached
 * (arena == NULL) or the context is freed.  Attaching zeroes the counters
 * and synchronises the device; attaching or detaching re-captures the step
 * graph.  CHIMERA_ENOMEM if the arena is too small, CHIMERA_EINVAL if it is
 * misaligned.  The step's tokens and cache are the same with and without it. */
chimera_status chimera_compaction_check_bytes(const chimera_ctx* ctx, int64_t* bytes);
chimera_status chimera_set_compaction_check(chimera_ctx* ctx, void* arena, int64_t arena_bytes);
/* Rows compared and 16-byte chunks found different since the arena was
 * attached (synchronises the device).  CHIMERA_ESTATE when no arena is attached. */
chimera_status chimera_compaction_check_read(chimera_ctx* ctx, int64_t* rows_checked, int64_t* mismatches);

/* TEST HOOK -- allocates.  y[M][N] (float32, host) = x[M][K] @ w[K][N]
 * through the repack and GEMM kernels of `dtype`, on device buffers the call
 * allocates (hipMalloc) and frees itself; synchronises the device.  x and w
 * are host arrays of that dtype.  M in [1, 256], N % 64 == 0, K a multiple
 * of 32 (bf16) or 16 (f32); CHIMERA_EINVAL otherwise. */
chimera_status chimera_debug_gemm(int32_t dtype, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                                  float* y);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * product as chimera_debug_gemm with every buffer in device memory and no
 * allocation, no free and no synchronisation.
 *   x: device [M][K] row-major, w: device [K][N] row-major, both of `dtype`
 *   (caller-owned, only read); y: device float32 [M][N] row-major
 *   (caller-owned, written); stream: hipStream_t or NULL.
 * The call only enqueues its kernels on `stream`.  Its scratch -- the tiled
 * copy of x, the repacked copy of w and the split-K partials -- is a 32 MiB
 * static device array that every device holds until the process ends:
 *   round256(mcap(M) K es) + round256(K N es) + splits M N 4 <= 32 MiB,
 * with es the dtype size, mcap(M) M rounded up to 16, 32, 64 or a multiple
 * of 128, and splits the reduction split the library picks for (N, K)
 * (at most 8).  Larger shapes return CHIMERA_ENOMEM before any launch; the
 * shape rules of chimera_debug_gemm give CHIMERA_EINVAL.  Every call on a
 * device shares that device's scratch: calls that overlap on one device
 * (other streams, other threads) race and must be serialised by the
 * caller. */
chimera_status chimera_gemm_static(int32_t dtype, const void* x, const void* w, int32_t M, int32_t N, int32_t K,
                                   float* y, void* stream);

const char* chimera_last_error(void);
void chimera_ctx_free(chimera_ctx* ctx);
void chimera_kv_free(chimera_kv* kv);
void chimera_free(chimera_model* m);

#ifdef __cplusplus
}
#endif
#endif /* CHIMERA_H */
