// Attention kernels of the decode step.
//
// Tree-masked paged attention (verify pass, Sec. 4.3).  Query u of a tree
// sits at position P_u = n + depth(u); it sees cache positions 0..n-1 and
// the tree slots of its ancestors, i.e. the logical key sequence 0..P_u in
// which position n + e maps to the tree slot of u's depth-e ancestor.  The
// keys are reduced with the online softmax in two parts, folded in order:
//   * positions 0 .. P_u - W (W = TREE_ATTN_WINDOW, deeper than any tree)
//     are committed keys, shared by every query of the tree: an MFMA pass
//     over 64-position chunks aligned to position 0, in groups fixed by
//     chunk index (pairs, then groups of four past the first 16 chunks),
//     writes one partial (m, l, O) per group, each query masking the keys
//     past its own bound;
//   * the window P_u - W + 1 .. P_u, which holds every tree position, is
//     reduced per query (one wave per query and head) after folding the
//     group partials in group order.
// The decomposition depends on P_u alone, so a query gets bit-identical
// results whether it is a node of a 64-node tree or the single query of a
// plain autoregressive step at the same position.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int CHUNK = 64;   // positions per chunk
constexpr int NEAR = TREE_ATTN_NEAR_CHUNKS;
constexpr int FAR = TREE_ATTN_FAR_GROUP;
constexpr int GMAX = FAR > 2 ? FAR : 2;  // chunks per group, upper bound
static_assert(NEAR % 2 == 0, "near chunks form pairs");
// Group of chunk c, and the first chunk and chunk count of group g.
__device__ __forceinline__ int group_of_chunk(int c) { return c < NEAR ? c / 2 : NEAR / 2 + (c - NEAR) / FAR; }
__device__ __forceinline__ int group_first_chunk(int g) { return g < NEAR / 2 ? 2 * g : NEAR + (g - NEAR / 2) * FAR; }
__device__ __forceinline__ int group_chunks(int g) { return g < NEAR / 2 ? 2 : FAR; }
constexpr int WIN = TREE_ATTN_WINDOW;  // window positions reduced per query
// The tree attention's softmax runs in base 2 on scores pre-scaled by
// log2(e) (exp(x) = 2^(x log2 e)), with gfx950's v_exp_f32; partials keep
// their maxima in that scale.
constexpr float LOG2E = 1.44269504088896340736f;
// Two floats -> two bf16 (round to nearest even) in one v_cvt_pk_bf16_f32;
// a in the low half.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b) {
  typedef float f2 __attribute__((ext_vector_type(2)));
  typedef __bf16 b2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f2{a, b}, b2));
}
// gfx950's transposed LDS read of four 16-bit elements (layout described at
// its use in the shared pass)
__device__ __forceinline__ int2 ld_tr16(const void* p) {
  typedef short s4 __attribute__((ext_vector_type(4)));
  const s4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4*)p);
  return __builtin_bit_cast(int2, v);
}
__device__ __forceinline__ float exp2_diff(float a, float b) {
  return a == -CH_INF ? 0.0f : __builtin_amdgcn_exp2f(a - b);
}
constexpr int MAX_NODES = 64;
static_assert(WIN + MAX_NODES == TREE_ATTN_TAIL_ROWS, "window rows");
static_assert(WIN == 16, "the window pass maps four lanes to each window key");

// Page-resolved offsets of the window rows: entry k < WIN is position
// n - WIN + k (committed), entry WIN + j the slot of tree node j (position
// n + j); entries before position 0 or past the tree are zero.
__global__ void attn_rows_kernel(const int* __restrict__ n_b, const int* __restrict__ page_table, int max_pages,
                                 int ps, int64_t page_stride, int hd, int N, int64_t* __restrict__ rowtab) {
  const int b = blockIdx.x;
  const int n = n_b[b];
  for (int rr = threadIdx.x; rr < TREE_ATTN_TAIL_ROWS; rr += blockDim.x) {
    const int p = rr < WIN ? n - WIN + rr : n + rr - WIN;
    int64_t off = 0;
    if (p >= 0 && (rr < WIN || rr - WIN < N))
      off = (int64_t)page_table[(int64_t)b * max_pages + p / ps] * page_stride + (int64_t)(p % ps) * hd;
    rowtab[(int64_t)b * TREE_ATTN_TAIL_ROWS + rr] = off;
  }
}

// ---------------------------------------------------------------------------
// Shared pass: grid (group slots, H, B), 4 waves; wave w owns queries
// 16w .. 16w+15 as MFMA columns.  S^T = K Q^T, then O^T += V^T P^T.
// ---------------------------------------------------------------------------
template <typename T, int HD>
// Three waves per SIMD (168 VGPRs or fewer): the pass is bound by the issue
// of its per-chunk VALU and MFMA chains, so occupancy is what hides them.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(3, 8))) void tree_attn_shared(const TreeAttnArgs a) {
  constexpr int VEC = ET<T>::VEC, KB = 4 * VEC;
  constexpr bool B16 = sizeof(T) == 2;
  constexpr int KP = HD + VEC;         // K row pitch (elements)
  // 16-bit V is staged as it lies in the cache, one key per row, and read
  // back transposed by ds_read_b64_tr_b16; the 16-element pad puts the 16
  // rows of one transposed read on distinct banks.  fp32 V is staged as V^T.
  constexpr int VRP = HD + 16;         // V row pitch (16-bit elements)
  constexpr int VP = CHUNK + VEC;      // V^T row pitch (fp32 elements)
  __shared__ __attribute__((aligned(16))) T Ks[CHUNK * KP];
  __shared__ __attribute__((aligned(16))) T Vt[B16 ? CHUNK * VRP : HD * VP];

  __shared__ int64_t pbase[GMAX * CHUNK];  // element offset of each staged key's row
  const int grp = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  // wave-uniform wave index: the MFMAs below sit under wave-level branches only
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int u = 16 * wave + c16;
  const bool wave_on = 16 * wave < a.N;
  const bool valid_u = u < a.N;
  const int uu = valid_u ? u : 0;
  // independent loads first: the queries' fragments, their depth, n
  int4 qf[HD / KB];
  if (wave_on) {
    const T* qrow = (const T*)a.q + (int64_t)(b * a.N + uu) * a.ldq + h * HD + g * VEC;
#pragma unroll
    for (int ks = 0; ks < HD / KB; ++ks) qf[ks] = ld16(qrow + ks * KB);
  }
  const int dep_u = a.depth[uu];
  const int n = a.n_b[b];
  // the group's page ids need no n: load them with it
  const int c_begin = group_first_chunk(grp);
  const int nch = group_chunks(grp);
  constexpr int PB = (GMAX * CHUNK + 255) / 256;
  int pg[PB];
#pragma unroll
  for (int t = 0; t < PB; ++t) {
    const int i = tid + 256 * t;
    const int pi = (c_begin * CHUNK + i) / a.ps;
    pg[t] = (i < nch * CHUNK && pi < a.max_pages) ? a.page_table[(int64_t)b * a.max_pages + pi] : 0;
  }
  const int maxk = n + a.D - WIN;        // last position any query treats as shared
  if (maxk < 0 || c_begin > maxk / CHUNK) return;
  const int c_end = min(c_begin + nch - 1, maxk / CHUNK);
  const int lim_u = n + dep_u - WIN;    // query u's last shared position
  // rows past the ones written so far (positions >= n + N) may hold
  // anything: they are staged as zeros, so masked keys add exact zeros
  const int wlim = n + a.N;
#pragma unroll
  for (int t = 0; t < PB; ++t) {
    const int i = tid + 256 * t;
    const int p = c_begin * CHUNK + i;
    if (i < nch * CHUNK) pbase[i] = (int64_t)pg[t] * a.page_stride + ((int64_t)h * a.ps + p % a.ps) * HD;
  }
  __syncthreads();
  float m = -CH_INF, l = 0.f;
  const float scale2 = a.scale * LOG2E;
  f32x4 o[HD / 16];
#pragma unroll
  for (int db = 0; db < HD / 16; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  const T* kpool = (const T*)a.kpool;
  const T* vpool = (const T*)a.vpool;
  // K and V rows of one chunk pass through registers: the global loads of
  // chunk c+1 are issued before chunk c is reduced.
  constexpr int PER = CHUNK * (HD / VEC) / 256;
  int4 kreg[PER], vreg[PER];
  // Consecutive lanes read consecutive 16-byte parts of a row (whole rows
  // per instruction), except fp32 V: there consecutive lanes read the same
  // part of consecutive rows, the order its transposed LDS writes need.
  constexpr int PARTS = HD / VEC;
  auto v_key = [](int idx) { return B16 ? idx / PARTS : idx % CHUNK; };
  auto v_part = [](int idx) { return B16 ? idx % PARTS : idx / CHUNK; };
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int idx = tid + 256 * t;
      const int kk = idx / PARTS, kp = idx % PARTS;
      kreg[t] = ld16(kpool + pbase[(c - c_begin) * CHUNK + kk] + kp * VEC);
      vreg[t] = ld16(vpool + pbase[(c - c_begin) * CHUNK + v_key(idx)] + v_part(idx) * VEC);
    }
  };
  load_chunk(c_begin);
  for (int c = c_begin; c <= c_end; ++c) {
    __syncthreads();
    // every row of the chunk written so far: no zero staging (uniform)
    const bool whole = (c + 1) * CHUNK <= wlim;
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int idx = tid + 256 * t;
      const int4 zero = int4{0, 0, 0, 0};
      st16(&Ks[(idx / PARTS) * KP + (idx % PARTS) * VEC], whole || c * CHUNK + idx / PARTS < wlim ? kreg[t] : zero);
      const int key = v_key(idx), part = v_part(idx);
      const int4 vk = whole || c * CHUNK + key < wlim ? vreg[t] : zero;
      if constexpr (B16) {
        st16(&Vt[key * VRP + part * VEC], vk);
      } else {
        const T* ve = reinterpret_cast<const T*>(&vk);
#pragma unroll
        for (int e = 0; e < VEC; ++e) Vt[(part * VEC + e) * VP + key] = ve[e];
      }
    }
    __syncthreads();
    if (c < c_end) load_chunk(c + 1);
    if (!wave_on) continue;

    f32x4 s[4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
      s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < HD / KB; ++ks)
        s[kb] = mfma_kb<T>(ld16(&Ks[(16 * kb + c16) * KP + ks * KB + g * VEC]), qf[ks], s[kb]);
    }
    // When every key of the chunk is visible to every valid query of the
    // wave (the wave-uniform common case), the masks and the -inf guards
    // are skipped: the values are the same ones the masked path computes.
    const bool open = __builtin_amdgcn_ballot_w64(valid_u && c * CHUNK + CHUNK - 1 > lim_u) == 0;
    float mc = -CH_INF;
    float alpha = 1.f, ls = 0.f, mn;
    if (open) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v = s[kb][r] * scale2;
          s[kb][r] = v;
          mc = fmaxf(mc, v);
        }
      mc = rows_max(mc);
      mn = fmaxf(m, mc);
      alpha = exp2_diff(m, mn);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = __builtin_amdgcn_exp2f(s[kb][r] - mn);
          s[kb][r] = p;
          ls = ls + p;
        }
    } else {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool act = valid_u && c * CHUNK + 16 * kb + 4 * g + r <= lim_u;  // S^T row = key
          const float v = act ? s[kb][r] * scale2 : -CH_INF;
          s[kb][r] = v;
          mc = fmaxf(mc, v);
        }
      mc = rows_max(mc);
      mn = fmaxf(m, mc);
      if (mn != -CH_INF) {
        alpha = exp2_diff(m, mn);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float p = exp2_diff(s[kb][r], mn);
            s[kb][r] = p;
            ls = ls + p;
          }
      } else {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    ls = rows_sum(ls);
    l = l * alpha + ls;
    m = mn;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) o[db] = o[db] * alpha;

    if constexpr (sizeof(T) == 2) {
      // P enters the bf16 MFMA as three bf16 terms, P = hi + mid + lo with
      // hi = bf16(P), mid = bf16(P - hi), lo = bf16(P - hi - mid): all 24
      // bits of the float P, so every product with a bf16 V is exact and PV
      // is as precise as a float dot product
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        // fragment element e is s[2 kp + e / 4][e % 4]; two elements per
        // conversion, element 2q in the low half of word q
        uint32_t ph[4], pm[4], pl[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const float a0 = s[2 * kp + q / 2][2 * (q % 2)], a1 = s[2 * kp + q / 2][2 * (q % 2) + 1];
          ph[q] = cvt_pk_bf16(a0, a1);
          const float r0 = a0 - __uint_as_float(ph[q] << 16), r1 = a1 - __uint_as_float(ph[q] & 0xffff0000u);
          pm[q] = cvt_pk_bf16(r0, r1);
          pl[q] = cvt_pk_bf16(r0 - __uint_as_float(pm[q] << 16), r1 - __uint_as_float(pm[q] & 0xffff0000u));
        }
        const int4 hfrag = int4{(int)ph[0], (int)ph[1], (int)ph[2], (int)ph[3]};
        const int4 mfrag = int4{(int)pm[0], (int)pm[1], (int)pm[2], (int)pm[3]};
        const int4 lfrag = int4{(int)pl[0], (int)pl[1], (int)pl[2], (int)pl[3]};
        // V^T fragments two output blocks at a time; within a pair the terms
        // alternate between the two accumulators.  Lane (g, c16) needs dim
        // 16 db + c16 of keys 32 kp + 4 g + {0..3} and 32 kp + 16 + 4 g +
        // {0..3}, the key order of the P fragment.  A transposed read hands
        // lane i of each 16-lane group element i % 4 of the 8-byte blocks
        // addressed by lanes i / 4 + 4 e (e = 0..3), so lane (g, c16)
        // addresses row 32 kp + 4 g + c16 / 4 (plus 16 for the second half),
        // dims 16 db + 4 (c16 % 4) .. + 3.
        const T* vrow = &Vt[(32 * kp + 4 * g + (c16 >> 2)) * VRP + 4 * (c16 & 3)];
#pragma unroll
        for (int d2 = 0; d2 < HD / 16; d2 += 2) {
          int4 vf[2];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const int2 lo = ld_tr16(vrow + 16 * (d2 + j));
            const int2 hi = ld_tr16(vrow + 16 * VRP + 16 * (d2 + j));
            vf[j] = int4{lo.x, lo.y, hi.x, hi.y};
          }
          o[d2] = mfma_kb<T>(vf[0], hfrag, o[d2]);
          o[d2 + 1] = mfma_kb<T>(vf[1], hfrag, o[d2 + 1]);
          o[d2] = mfma_kb<T>(vf[0], mfrag, o[d2]);
          o[d2 + 1] = mfma_kb<T>(vf[1], mfrag, o[d2 + 1]);
          o[d2] = mfma_kb<T>(vf[0], lfrag, o[d2]);
          o[d2 + 1] = mfma_kb<T>(vf[1], lfrag, o[d2 + 1]);
        }
      }
    } else {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int4 bfrag = int4{__float_as_int(s[kb][0]), __float_as_int(s[kb][1]), __float_as_int(s[kb][2]),
                                __float_as_int(s[kb][3])};
#pragma unroll
        for (int db = 0; db < HD / 16; ++db)
          o[db] = mfma_kb<T>(ld16(&Vt[(16 * db + c16) * VP + 16 * kb + 4 * g]), bfrag, o[db]);
      }
    }
  }
  if (!valid_u) return;
  const int64_t slot = (((int64_t)b * a.H + h) * a.G + grp) * a.N + u;
  float* po = a.part_o + slot * HD;
#pragma unroll
  for (int db = 0; db < HD / 16; ++db)
#pragma unroll
    for (int r = 0; r < 4; ++r) po[16 * db + 4 * g + r] = o[db][r];
  if (g == 0) {
    a.part_ml[slot * 2] = m;
    a.part_ml[slot * 2 + 1] = l;
  }
}

// ---------------------------------------------------------------------------
// Window pass: grid (ceil(H / 4), N, B), one wave per (query u, head h):
//   1. loads that need nothing: n, u's depth and path, the window rows'
//      page-resolved offsets (written once per pass), the query, the first
//      batch of group partials;
//   2. the window's K and V rows are requested (for the scores lane
//      4 k + j holds dims [j HD/4, (j+1) HD/4) of window key k; for PV each
//      lane reads its own output dims of every row); while they are in
//      flight the group partials are folded in group order;
//   3. scores, the window's softmax step and PV in window order.
// Window key k is position P_u - W + 1 + k: a committed row below n, the
// slot of u's ancestor at depth p - n from n on.  Keys before position 0
// read u's own slot and add exact zeros.
// ---------------------------------------------------------------------------
template <typename T, int HD>
__global__ __launch_bounds__(256) void tree_attn_window(const TreeAttnArgs a) {
  constexpr int VEC = ET<T>::VEC;
  constexpr int DPL = HD / 64;   // output dims per lane
  constexpr int LPK = 64 / WIN;  // lanes per window key
  constexpr int DPK = HD / LPK;  // score dims per lane
  constexpr int NQ = DPK / VEC;  // 16-byte loads per lane and row
  constexpr int BATCH = 8;       // group partials loaded per round trip
  static_assert(NQ >= 1 && DPK % VEC == 0, "window layout");
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int h = 4 * blockIdx.x + wave, u = blockIdx.y, b = blockIdx.z;
  if (h >= a.H) return;  // wave-uniform
  const int kw = lane / LPK, sub = lane % LPK;
  // 1. loads that need nothing
  const int n = a.n_b[b];
  const int dep = a.depth[u];
  const int pth = a.path[u * 64 + lane];  // node at depth `lane` on u's path
  const int64_t* rt = a.rowtab + (int64_t)b * TREE_ATTN_TAIL_ROWS;
  const long long r_lo = rt[lane];                           // entries 0 .. 63
  const long long r_hi = rt[64 + (lane & (TREE_ATTN_TAIL_ROWS - 64 - 1))];  // entries 64 ..
  int4 qv[NQ];
  {
    const T* qrow = (const T*)a.q + (int64_t)(b * a.N + u) * a.ldq + h * HD + sub * DPK;
#pragma unroll
    for (int i = 0; i < NQ; ++i) qv[i] = ld16(qrow + i * VEC);
  }
  float bm[BATCH], bl[BATCH], bo[BATCH][DPL];
  // this (sequence, head, query)'s partials: group g at slot base + g * N
  const int64_t slot0 = ((int64_t)b * a.H + h) * a.G * a.N + u;
  const float* pml = a.part_ml + slot0 * 2;
  const float* po = a.part_o + slot0 * HD + DPL * lane;
  auto load_batch = [&](int g0, int lim_g) {
#pragma unroll
    for (int t = 0; t < BATCH; ++t) {
      bm[t] = -CH_INF;
      bl[t] = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) bo[t][e] = 0.f;
      if (g0 + t < lim_g) {
        const int gs = (g0 + t) * a.N;  // group offset in slots
        bm[t] = pml[gs * 2];
        bl[t] = pml[gs * 2 + 1];
#pragma unroll
        for (int e = 0; e < DPL; ++e) bo[t][e] = po[gs * HD + e];
      }
    }
  };
  // slots past this step's groups are read but never folded
  load_batch(0, a.G);

  // 2. the window rows
  const int Pu = n + dep;
  const int p = Pu - WIN + 1 + kw;
  const int jn = __shfl(pth, min(max(p - n, 0), 63));
  int e = p < n ? p - (n - WIN) : WIN + jn;  // row-table entry of window key kw
  if (p < 0) e = WIN + u;                    // u's own slot
  const long long olo = __shfl(r_lo, e & 63);
  const long long ohi = __shfl(r_hi, e & (TREE_ATTN_TAIL_ROWS - 64 - 1));
  const int64_t hoff = (int64_t)h * a.ps * HD;
  const int64_t roff = (e < 64 ? olo : ohi) + hoff;
  const T* kpool = (const T*)a.kpool;
  const T* vpool = (const T*)a.vpool;
  int4 kv[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) kv[i] = ld16(kpool + roff + sub * DPK + i * VEC);
  T vv[WIN][DPL];
#pragma unroll
  for (int k = 0; k < WIN; ++k) {
    const uint32_t ro_lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)roff, k * LPK);
    const int64_t ro = (int64_t)(((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(roff >> 32), k * LPK) << 32) |
                                 (uint64_t)ro_lo);
#pragma unroll
    for (int d = 0; d < DPL; ++d) vv[k][d] = vpool[ro + DPL * lane + d];
  }
  // while they are in flight: fold the group partials in group order
  const int lim = Pu - WIN;
  const int ngrp = lim >= 0 ? group_of_chunk(lim / CHUNK) + 1 : 0;
  float m = -CH_INF, l = 0.f, o[DPL];
#pragma unroll
  for (int d = 0; d < DPL; ++d) o[d] = 0.f;
  for (int g0 = 0; g0 < ngrp; g0 += BATCH) {
    if (g0 > 0) load_batch(g0, ngrp);
#pragma unroll
    for (int t = 0; t < BATCH; ++t) {
      if (g0 + t >= ngrp || bm[t] == -CH_INF) continue;
      const float mn = fmaxf(m, bm[t]);
      const float a1 = exp2_diff(m, mn), a2 = __builtin_amdgcn_exp2f(bm[t] - mn);
      l = l * a1 + bl[t] * a2;
#pragma unroll
      for (int d = 0; d < DPL; ++d) o[d] = o[d] * a1 + bo[t][d] * a2;
      m = mn;
    }
  }

  // 3. the window: each score is a fixed-order dot product over the four
  // lanes of its key
  float acc = 0.f;
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const T* qe = reinterpret_cast<const T*>(&qv[i]);
    const T* ke = reinterpret_cast<const T*>(&kv[i]);
#pragma unroll
    for (int j = 0; j < VEC; ++j) acc = fmaf(ET<T>::to_f(qe[j]), ET<T>::to_f(ke[j]), acc);
  }
  static_assert(LPK == 4, "four lanes per window key");
  acc = acc + dpp_mov<DPP_XOR1>(acc);
  acc = acc + dpp_mov<DPP_XOR2>(acc);
  const bool valid = p >= 0;
  const float s = valid ? acc * (a.scale * LOG2E) : -CH_INF;
  const float mc = wave_max(s);
  const float mn = fmaxf(m, mc);
  const float alpha = exp2_diff(m, mn);
  const float pe = valid ? __builtin_amdgcn_exp2f(s - mn) : 0.f;
  l = l * alpha + wave_sum(sub == 0 ? pe : 0.f);
#pragma unroll
  for (int d = 0; d < DPL; ++d) o[d] = o[d] * alpha;
#pragma unroll
  for (int k = 0; k < WIN; ++k) {
    const float pk = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pe), k * LPK));
#pragma unroll
    for (int d = 0; d < DPL; ++d) o[d] = fmaf(pk, ET<T>::to_f(vv[k][d]), o[d]);
  }
#pragma unroll
  for (int d = 0; d < DPL; ++d) store_tiled<T>((T*)a.out, a.o_mtiles, b * a.N + u, h * HD + DPL * lane + d, o[d] / l);
}

template <typename T, int HD>
void tree_attn_go(const TreeAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((tree_attn_shared<T, HD>), dim3(a.G, a.H, a.B), dim3(256), 0, st, a);
  hipLaunchKernelGGL((tree_attn_window<T, HD>), dim3((a.H + 3) / 4, a.N, a.B), dim3(256), 0, st, a);
}

// ---------------------------------------------------------------------------
// Draft encoder attention: one query per drafted node (trigram position
// n+k) over the target-state entries 0..n-1, the trigram entries 0..n and
// the node's ancestors-or-self at depths 1..k, in that order.
// grid (key blocks of 256, H, B*R); each wave reduces 64 keys, four at a
// time: lane group sub = lane >> 4 takes key 4*kg + sub and lane c =
// lane & 15 the head-dim slice [c*HD/16, (c+1)*HD/16).
// ---------------------------------------------------------------------------
// DS consecutive elements of a row, loaded as one vector.
template <typename T, int DS>
struct alignas(DS * sizeof(T) >= 16 ? 16 : DS * sizeof(T)) Frag {
  T v[DS];
};

template <typename T, int HD>
__global__ __launch_bounds__(256) void enc_attn_partial(const EncAttnArgs a) {
  constexpr int DS = HD / 16;            // dims per lane
  constexpr int VEC = ET<T>::VEC;
  static_assert(DS % VEC == 0 || VEC % DS == 0, "slice");
  __shared__ float wm[4], wl[4];
  __shared__ float wo[4][HD];
  const int blk = blockIdx.x, h = blockIdx.y, row = blockIdx.z, b = row / a.R;
  const int node = a.nodes[row % a.R];
  const int n = a.n_b[b];
  const int nkeys = 2 * n + a.level + 1;
  const int nblk_used = (nkeys + 255) / 256;
  if (blk >= nblk_used) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane >> 4, c = lane & 15;
  float q[DS];
  {
    const T* qrow = (const T*)a.q + (int64_t)row * a.ldq + h * HD + c * DS;
#pragma unroll
    for (int e = 0; e < DS; ++e) q[e] = ET<T>::to_f(qrow[e]);
  }
  const int key0 = blk * 256 + wave * 64;
  // the node's path (draft-tree node at each depth), one entry per lane
  const int pth = a.path[node * 64 + lane];
  // every K and V slice of the wave's 64 keys is requested before any is
  // used; keys past the last one read the last key's row and are masked
  Frag<T, DS> kf[16], vf[16];
#pragma unroll
  for (int kg = 0; kg < 16; ++kg) {
    const int key = min(key0 + 4 * kg + sub, nkeys - 1);
    const int tn = __shfl(pth, max(key - 2 * n, 0));
    const int stream = key < n ? 0 : 1;
    const int pos = key < n ? key : (key <= 2 * n ? key - n : a.tree_slot0 + tn);
    const int64_t off = ((((int64_t)b * 2 + stream) * a.H + h) * a.cap + pos) * HD + c * DS;
    kf[kg] = *reinterpret_cast<const Frag<T, DS>*>((const T*)a.kbase + off);
    vf[kg] = *reinterpret_cast<const Frag<T, DS>*>((const T*)a.vbase + off);
  }
  float sc[16];
  float mloc = -CH_INF;
#pragma unroll
  for (int kg = 0; kg < 16; ++kg) {
    const int key = key0 + 4 * kg + sub;
    float d = 0.f;
#pragma unroll
    for (int e = 0; e < DS; ++e) d = fmaf(q[e], ET<T>::to_f(kf[kg].v[e]), d);
    d = row16_sum(d);
    sc[kg] = key < nkeys ? d * a.scale : -CH_INF;
    mloc = fmaxf(mloc, sc[kg]);
  }
  const float mw = rows_max(mloc);
  float lsum = 0.f, o[DS];
#pragma unroll
  for (int e = 0; e < DS; ++e) o[e] = 0.f;
#pragma unroll
  for (int kg = 0; kg < 16; ++kg) {
    const int key = key0 + 4 * kg + sub;
    const float p = (key < nkeys && mw != -CH_INF) ? expf(sc[kg] - mw) : 0.f;
    lsum = lsum + p;
#pragma unroll
    for (int e = 0; e < DS; ++e) o[e] = fmaf(p, ET<T>::to_f(vf[kg].v[e]), o[e]);
  }
  lsum = rows_sum(lsum);
#pragma unroll
  for (int e = 0; e < DS; ++e) {
    o[e] = rows_sum(o[e]);
  }
  if (lane == 0) {
    wm[wave] = mw;
    wl[wave] = lsum;
  }
  if (sub == 0) {
#pragma unroll
    for (int e = 0; e < DS; ++e) wo[wave][c * DS + e] = o[e];
  }
  __syncthreads();
  if (wave != 0) return;
  float m = -CH_INF;
  for (int w = 0; w < 4; ++w) m = fmaxf(m, wm[w]);
  float l = 0.f;
  float* dst = a.part + (((int64_t)row * a.H + h) * a.nblk + blk) * (HD + 2);
  for (int i = lane; i < HD; i += 64) {
    float acc = 0.f;
    for (int w = 0; w < 4; ++w) acc = acc + wo[w][i] * exp_diff(wm[w], m);
    dst[i] = acc;
  }
  for (int w = 0; w < 4; ++w) l = l + wl[w] * exp_diff(wm[w], m);
  if (lane == 0) {
    dst[HD] = m;
    dst[HD + 1] = l;
  }
}

template <typename T, int HD>
__global__ void enc_attn_combine(const EncAttnArgs a) {
  constexpr int DPL = HD / 64;
  const int h = blockIdx.x, row = blockIdx.y, lane = threadIdx.x;
  const int n = a.n_b[row / a.R];
  const int nkeys = 2 * n + a.level + 1;
  const int used = (nkeys + 255) / 256;
  float m = -CH_INF, l = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;
  // block partials are requested CB at a time, then folded in block order
  constexpr int CB = 8;
  for (int b0 = 0; b0 < used; b0 += CB) {
    float bm[CB], bl[CB], bo[CB][DPL];
#pragma unroll
    for (int t = 0; t < CB; ++t) {
      bm[t] = -CH_INF;
      bl[t] = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) bo[t][e] = 0.f;
      if (b0 + t < used) {
        const float* src = a.part + (((int64_t)row * a.H + h) * a.nblk + b0 + t) * (HD + 2);
        bm[t] = src[HD];
        bl[t] = src[HD + 1];
#pragma unroll
        for (int e = 0; e < DPL; ++e) bo[t][e] = src[DPL * lane + e];
      }
    }
#pragma unroll
    for (int t = 0; t < CB; ++t) {
      if (b0 + t >= used || bm[t] == -CH_INF) continue;
      const float mn = fmaxf(m, bm[t]);
      const float a1 = exp_diff(m, mn), a2 = expf(bm[t] - mn);
      l = l * a1 + bl[t] * a2;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[e] = o[e] * a1 + bo[t][e] * a2;
      m = mn;
    }
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) store_tiled<T>((T*)a.out, a.o_mtiles, row, h * HD + DPL * lane + e, o[e] / l);
}

template <typename T, int HD>
void enc_attn_go(const EncAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((enc_attn_partial<T, HD>), dim3(a.nblk, a.H, a.B * a.R), dim3(256), 0, st, a);
  hipLaunchKernelGGL((enc_attn_combine<T, HD>), dim3(a.H, a.B * a.R), dim3(64), 0, st, a);
}

}  // namespace

void launch_attn_rows(const int* n_b, const int* page_table, int max_pages, int ps, int64_t page_stride, int hd,
                      int N, int B, int64_t* rowtab, hipStream_t st) {
  hipLaunchKernelGGL(attn_rows_kernel, dim3(B), dim3(TREE_ATTN_TAIL_ROWS), 0, st, n_b, page_table, max_pages, ps,
                     page_stride, hd, N, rowtab);
}

void launch_tree_attn(int dtype, const TreeAttnArgs& a, hipStream_t st) {
  if (dtype == DT_BF16 && a.hd == 128)
    tree_attn_go<bf16_t, 128>(a, st);
  else if (dtype == DT_BF16 && a.hd == 64)
    tree_attn_go<bf16_t, 64>(a, st);
  else if (dtype == DT_F32 && a.hd == 64)
    tree_attn_go<float, 64>(a, st);
  else
    tree_attn_go<float, 128>(a, st);
}

void launch_enc_attn(int dtype, const EncAttnArgs& a, hipStream_t st) {
  if (dtype == DT_BF16 && a.hd == 128)
    enc_attn_go<bf16_t, 128>(a, st);
  else if (dtype == DT_BF16 && a.hd == 64)
    enc_attn_go<bf16_t, 64>(a, st);
  else if (dtype == DT_F32 && a.hd == 64)
    enc_attn_go<float, 64>(a, st);
  else
    enc_attn_go<float, 128>(a, st);
}
