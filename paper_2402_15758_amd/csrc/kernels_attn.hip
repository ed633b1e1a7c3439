// Attention kernels of the decode step.
//
// Tree-masked paged attention (verify pass, Sec. 4.3).  Query u of a tree
// sits at position P_u = n + depth(u); it sees cache positions 0..n-1 and
// the tree slots of its ancestors, i.e. the logical key sequence 0..P_u in
// which position n + e maps to the tree slot of u's depth-e ancestor.  The
// keys are reduced in 64-position chunks aligned to position 0, in chunk
// order, with the online softmax:
//   * chunks 0 .. c_u - 2 (c_u = P_u / 64) hold committed keys only and are
//     shared by every query of the tree: an MFMA pass over groups of two
//     chunks writes one partial (m, l, O) per group;
//   * the last two chunks c_u - 1 and c_u, which contain every tree
//     position, are reduced per query (scores by MFMA over the staged rows,
//     softmax and PV on the VALU in logical key order) after folding the
//     group partials in group order.
// The decomposition depends on P_u alone, so a query gets bit-identical
// results whether it is a node of a 64-node tree or the single query of a
// plain autoregressive step at the same position.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int CHUNK = 64;   // positions per chunk
constexpr int GROUP = TREE_ATTN_GROUP_POSITIONS / CHUNK;  // chunks per shared-pass workgroup
constexpr int TAIL_ROWS = 2 * CHUNK;  // committed rows staged by the tail pass
constexpr int MAX_NODES = 64;
// queries (one wave each) per tail-pass workgroup: 8 (one workgroup per CU
// at a 64-node tree and 32 heads), or 16 when the 8-query grid would need
// more than two rounds of workgroups (large batches of small trees)
constexpr int TAIL_QPW = 8;
constexpr int TAIL_QPW_WIDE = 16;
static_assert(TAIL_ROWS + MAX_NODES == TREE_ATTN_TAIL_ROWS, "tail rows");

// Page-resolved offsets of the tail pass's staged rows (positions lo .. n+N-1
// with lo = 64 * max(n / 64 - 1, 0)); entries past them are zero.
__global__ void attn_rows_kernel(const int* __restrict__ n_b, const int* __restrict__ page_table, int max_pages,
                                 int ps, int64_t page_stride, int hd, int N, int64_t* __restrict__ rowtab) {
  const int b = blockIdx.x;
  const int n = n_b[b];
  const int cmin = n / CHUNK;
  const int lo = (cmin >= 1 ? cmin - 1 : 0) * CHUNK;
  const int nrows = n - lo + N;
  for (int rr = threadIdx.x; rr < TREE_ATTN_TAIL_ROWS; rr += blockDim.x) {
    int64_t off = 0;
    if (rr < nrows) {
      const int p = lo + rr;
      off = (int64_t)page_table[(int64_t)b * max_pages + p / ps] * page_stride + (int64_t)(p % ps) * hd;
    }
    rowtab[(int64_t)b * TREE_ATTN_TAIL_ROWS + rr] = off;
  }
}

// ---------------------------------------------------------------------------
// Shared pass: grid (group slots, H, B), 4 waves; wave w owns queries
// 16w .. 16w+15 as MFMA columns.  S^T = K Q^T, then O^T += V^T P^T.
// ---------------------------------------------------------------------------
template <typename T, int HD>
__global__ __launch_bounds__(256) void tree_attn_shared(const TreeAttnArgs a) {
  constexpr int VEC = ET<T>::VEC, KB = 4 * VEC;
  constexpr int KP = HD + VEC;         // K row pitch (elements)
  constexpr int VP = CHUNK + VEC;      // V^T row pitch (elements)
  __shared__ __attribute__((aligned(16))) T Ks[CHUNK * KP];
  __shared__ __attribute__((aligned(16))) T Vt[HD * VP];

  __shared__ int64_t pbase[GROUP * CHUNK];  // element offset of each staged key's row
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
  const int c_begin = grp * GROUP;
  constexpr int PB = (GROUP * CHUNK + 255) / 256;
  int pg[PB];
#pragma unroll
  for (int t = 0; t < PB; ++t) {
    const int i = tid + 256 * t;
    const int pi = (c_begin * CHUNK + i) / a.ps;
    pg[t] = (i < GROUP * CHUNK && pi < a.max_pages) ? a.page_table[(int64_t)b * a.max_pages + pi] : 0;
  }
  const int cmax = (n + a.D) / CHUNK;
  const int last = cmax - 2;            // last chunk any query treats as shared
  if (c_begin > last) return;
  const int c_end = min(c_begin + GROUP - 1, last);
  const int lim_u = (n + dep_u) / CHUNK - 2;
#pragma unroll
  for (int t = 0; t < PB; ++t) {
    const int i = tid + 256 * t;
    const int p = c_begin * CHUNK + i;
    if (i < GROUP * CHUNK) pbase[i] = (int64_t)pg[t] * a.page_stride + ((int64_t)h * a.ps + p % a.ps) * HD;
  }
  __syncthreads();
  float m = -CH_INF, l = 0.f;
  f32x4 o[HD / 16];
#pragma unroll
  for (int db = 0; db < HD / 16; ++db) o[db] = f32x4{0.f, 0.f, 0.f, 0.f};

  const T* kpool = (const T*)a.kpool;
  const T* vpool = (const T*)a.vpool;
  // K rows and V^T of one chunk pass through registers: the global loads of
  // chunk c+1 are issued before chunk c is reduced.
  constexpr int PER = CHUNK * (HD / VEC) / 256;
  int4 kreg[PER], vreg[PER];
  // K: consecutive lanes read consecutive 16-byte parts of a row (whole
  // rows per instruction); V: consecutive lanes read the same part of
  // consecutive rows, the order its transposed LDS writes need
  constexpr int PARTS = HD / VEC;
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int idx = tid + 256 * t;
      const int kk = idx / PARTS, kp = idx % PARTS;
      kreg[t] = ld16(kpool + pbase[(c - c_begin) * CHUNK + kk] + kp * VEC);
      const int key = idx % CHUNK, part = idx / CHUNK;
      vreg[t] = ld16(vpool + pbase[(c - c_begin) * CHUNK + key] + part * VEC);
    }
  };
  load_chunk(c_begin);
  for (int c = c_begin; c <= c_end; ++c) {
    __syncthreads();
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int idx = tid + 256 * t;
      st16(&Ks[(idx / PARTS) * KP + (idx % PARTS) * VEC], kreg[t]);
      const int key = idx % CHUNK, part = idx / CHUNK;
      const T* ve = reinterpret_cast<const T*>(&vreg[t]);
#pragma unroll
      for (int e = 0; e < VEC; ++e) Vt[(part * VEC + e) * VP + key] = ve[e];
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
    const bool act = valid_u && c <= lim_u;
    float mc = -CH_INF;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float v = act ? s[kb][r] * a.scale : -CH_INF;
        s[kb][r] = v;
        mc = fmaxf(mc, v);
      }
    mc = rows_max(mc);
    const float mn = fmaxf(m, mc);
    float alpha = 1.f, ls = 0.f;
    if (mn != -CH_INF) {
      alpha = exp_diff(m, mn);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float p = exp_diff(s[kb][r], mn);
          s[kb][r] = p;
          ls = ls + p;
        }
    } else {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    ls = rows_sum(ls);
    l = l * alpha + ls;
    m = mn;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) o[db] = o[db] * alpha;

    if constexpr (sizeof(T) == 2) {
      // P enters the bf16 MFMA as two bf16 terms, P = hi + lo with
      // hi = bf16(P) and lo = bf16(P - hi), which keeps 16 of its bits
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        bf16_t pb[8], pl[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pb[r] = f2bf(s[2 * kp][r]);
          pb[4 + r] = f2bf(s[2 * kp + 1][r]);
          pl[r] = f2bf(s[2 * kp][r] - bf2f(pb[r]));
          pl[4 + r] = f2bf(s[2 * kp + 1][r] - bf2f(pb[4 + r]));
        }
        const int4 bfrag = *reinterpret_cast<const int4*>(pb);
        const int4 lfrag = *reinterpret_cast<const int4*>(pl);
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) {
          const T* vr = &Vt[(16 * db + c16) * VP];
          const int2 lo = *reinterpret_cast<const int2*>(vr + 32 * kp + 4 * g);
          const int2 hi = *reinterpret_cast<const int2*>(vr + 32 * kp + 16 + 4 * g);
          const int4 vf = int4{lo.x, lo.y, hi.x, hi.y};
          o[db] = mfma_kb<T>(vf, bfrag, o[db]);
          o[db] = mfma_kb<T>(vf, lfrag, o[db]);
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
// Tail pass: grid (ceil(N/QPW), H, B), QPW waves; wave w reduces query
// u = QPW * blockIdx.x + w, with arithmetic that does not depend on QPW.
// The workgroup stages the committed positions lo .. n-1 of the last chunks
// followed by every tree slot (rows 0 .. nrows-1):
//   1. loads that need nothing: n, the staged rows' page-resolved offsets
//      (written once per pass), the queries' MFMA fragments, tree paths and
//      depths, the first batch of shared-pass partials;
//   2. K fragments and V rows are requested; while they are in flight each
//      wave folds its query's partials in group order; then S = Q K^T over
//      every staged row by MFMA -> LDS, and V -> LDS as float;
//   3. per query: the last two chunks in logical-position order (lane = key);
//      PV on the VALU.
// Each score is one MFMA dot product whose value does not depend on where
// the query or key sits in the tile, so a query's scores are the same in a
// tree and in a single-query step.
// ---------------------------------------------------------------------------
template <typename T, int HD, int QPW>
__global__ __launch_bounds__(64 * QPW) void tree_attn_tail(const TreeAttnArgs a) {
  constexpr int NT = 64 * QPW;
  constexpr int VEC = ET<T>::VEC;
  constexpr int KB = 4 * VEC;                 // reduction indices per MFMA k-block
  constexpr int ROWS = TAIL_ROWS + MAX_NODES;  // staged rows, upper bound
  constexpr int DPL = HD / 64;                 // output dims per lane
  constexpr int PARTS = HD / VEC;
  constexpr int BATCH = 8;                     // shared-pass partials loaded per round trip
  constexpr int PV_BATCH = 16;                 // keys whose V rows are read per round
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  float* Vl = reinterpret_cast<float*>(smem);  // [ROWS][HD]
  float* Sl = Vl + ROWS * HD;                  // [QPW][ROWS]
  __shared__ int64_t rowbase[ROWS];
  __shared__ uint8_t spath[QPW][64];
  __shared__ int sdepth[QPW];

  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g = lane >> 4, c16 = lane & 15;
  const int u0 = QPW * blockIdx.x;
  const int u = u0 + wave;
  const bool active = u < a.N;
  // 1. loads that need nothing
  const int n = a.n_b[b];
  int4 qf[HD / KB];  // MFMA A operand: row c16 = query u0 + c16 (zero beyond the workgroup's queries)
  {
    const int uq = u0 + c16;
    const bool qok = c16 < QPW && uq < a.N;
    const T* qrow = (const T*)a.q + (int64_t)(b * a.N + (qok ? uq : 0)) * a.ldq + h * HD + g * VEC;
#pragma unroll
    for (int ks = 0; ks < HD / KB; ++ks) qf[ks] = qok ? ld16(qrow + ks * KB) : int4{0, 0, 0, 0};
  }
  for (int i = tid; i < QPW * 64; i += NT) {
    const int uu = u0 + i / 64;
    spath[i / 64][i % 64] = uu < a.N ? a.path[uu * 64 + i % 64] : 0;
  }
  if (tid < QPW) sdepth[tid] = (u0 + tid) < a.N ? a.depth[u0 + tid] : 0;
  float bm[BATCH], bl[BATCH], bo[BATCH][DPL];
  auto load_batch = [&](int g0) {
#pragma unroll
    for (int t = 0; t < BATCH; ++t) {
      bm[t] = -CH_INF;
      bl[t] = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) bo[t][e] = 0.f;
      if (active && g0 + t < a.G) {  // slots past this step's groups are read but never folded
        const int64_t slot = (((int64_t)b * a.H + h) * a.G + g0 + t) * a.N + u;
        bm[t] = a.part_ml[slot * 2];
        bl[t] = a.part_ml[slot * 2 + 1];
#pragma unroll
        for (int e = 0; e < DPL; ++e) bo[t][e] = a.part_o[slot * HD + DPL * lane + e];
      }
    }
  };
  load_batch(0);
  const int64_t hoff = (int64_t)h * a.ps * HD;
  for (int rr = tid; rr < ROWS; rr += NT) rowbase[rr] = a.rowtab[(int64_t)b * ROWS + rr] + hoff;
  const int cmin = n / CHUNK;
  const int lo = (cmin >= 1 ? cmin - 1 : 0) * CHUNK;  // first staged committed position
  const int nc = n - lo;                               // committed rows staged (<= 127)
  const int nrows = nc + a.N;
  __syncthreads();
  // 2. V rows -> LDS (float); scores by MFMA -> LDS
  const T* kpool = (const T*)a.kpool;
  const T* vpool = (const T*)a.vpool;
  // every load of this phase is issued before any is used: K fragments of
  // the wave's row tiles (wave w takes tiles w and w + QPW), then V rows
  constexpr int RT_PER_WAVE = (ROWS / 16 + QPW - 1) / QPW;
  int4 kf[RT_PER_WAVE][HD / KB];
#pragma unroll
  for (int j = 0; j < RT_PER_WAVE; ++j) {
    const int rr = 16 * (wave + QPW * j) + c16;  // MFMA B column: staged row
    const T* kr = kpool + rowbase[rr < nrows ? rr : 0] + g * VEC;
#pragma unroll
    for (int ks = 0; ks < HD / KB; ++ks) kf[j][ks] = ld16(kr + ks * KB);
  }
  constexpr int UNR = (ROWS * PARTS + NT - 1) / NT;
  int4 vbuf[UNR];
#pragma unroll
  for (int t = 0; t < UNR; ++t) {  // unpredicated: slots past the staged rows re-read row 0
    const int idx = tid + NT * t;
    const int rr = idx < nrows * PARTS ? idx / PARTS : 0;
    vbuf[t] = ld16(vpool + rowbase[rr] + (idx % PARTS) * VEC);
  }
  // while those loads are in flight: fold the shared-pass partials of this
  // wave's query in group order
  const int Pu = n + sdepth[wave];
  const int cu = Pu / CHUNK;
  float m = -CH_INF, l = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;
  const int lim = cu - 2;
  const int ngrp = (active && lim >= 0) ? lim / GROUP + 1 : 0;
  auto fold_batch = [&](int g0) {
#pragma unroll
    for (int t = 0; t < BATCH; ++t) {
      if (g0 + t >= ngrp || bm[t] == -CH_INF) continue;
      const float mn = fmaxf(m, bm[t]);
      const float a1 = exp_diff(m, mn), a2 = expf(bm[t] - mn);
      l = l * a1 + bl[t] * a2;
#pragma unroll
      for (int e = 0; e < DPL; ++e) o[e] = o[e] * a1 + bo[t][e] * a2;
      m = mn;
    }
  };
  // the first batch was loaded before the K/V requests: straight-line code
  // here lets its wait leave those in flight
  fold_batch(0);
  for (int g0 = BATCH; g0 < ngrp; g0 += BATCH) {
    load_batch(g0);
    fold_batch(g0);
  }
#pragma unroll
  for (int j = 0; j < RT_PER_WAVE; ++j) {
    const int rt = wave + QPW * j;
    if (16 * rt >= nrows) break;  // wave-uniform
    const int rr = 16 * rt + c16;
    f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < HD / KB; ++ks) acc = mfma_kb<T>(qf[ks], kf[j][ks], acc);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int qi = 4 * g + r;  // output row = query
      if (qi < QPW && rr < nrows) Sl[qi * ROWS + rr] = acc[r];
    }
  }
#pragma unroll
  for (int t = 0; t < UNR; ++t) {
    const int idx = tid + NT * t;
    if (idx < nrows * PARTS) {
      const T* ve = reinterpret_cast<const T*>(&vbuf[t]);
      float* dst = &Vl[(idx / PARTS) * HD + (idx % PARTS) * VEC];
#pragma unroll
      for (int e = 0; e < VEC; e += 4)
        *reinterpret_cast<float4*>(dst + e) =
            float4{ET<T>::to_f(ve[e]), ET<T>::to_f(ve[e + 1]), ET<T>::to_f(ve[e + 2]), ET<T>::to_f(ve[e + 3])};
    }
  }
  __syncthreads();
  if (!active) return;

  // 3. per query: the last two chunks, keys in logical-position order
  const float* srow = Sl + wave * ROWS;
  // the last two chunks, keys in logical-position order
  for (int c = (cu >= 1 ? cu - 1 : 0); c <= cu; ++c) {
    const int p = c * CHUNK + lane;
    const bool valid = p <= Pu;
    int row = 0;
    float s = -CH_INF;
    if (valid) {
      row = p < n ? p - lo : nc + (int)spath[wave][p - n];
      s = srow[row] * a.scale;
    }
    // lane 0 holds the chunk's first key, always one of the query's keys
    const int row0 = __builtin_amdgcn_readlane(row, 0);
    if (!valid) row = row0;
    const float mc = wave_max(s);
    const float mn = fmaxf(m, mc);
    const float alpha = exp_diff(m, mn);
    const float pe = valid ? expf(s - mn) : 0.f;
    l = l * alpha + wave_sum(pe);
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[e] = o[e] * alpha;
    // keys in order, 16 per round: the 16 V rows are read before any is used.
    // Keys past the query's last one in a round have pe = 0 and the staged
    // row of the chunk's first key, so they add exact zeros.
    const int cnt = __builtin_amdgcn_readfirstlane(min(CHUNK, Pu - c * CHUNK + 1));
    for (int i0 = 0; i0 < cnt; i0 += PV_BATCH) {
      float pis[PV_BATCH];
      float vv[PV_BATCH][DPL];
#pragma unroll
      for (int j = 0; j < PV_BATCH; ++j) {
        pis[j] = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pe), i0 + j));
        const int ri = __builtin_amdgcn_readlane(row, i0 + j);
        const float* vr = &Vl[ri * HD + DPL * lane];
#pragma unroll
        for (int e = 0; e < DPL; ++e) vv[j][e] = vr[e];
      }
#pragma unroll
      for (int j = 0; j < PV_BATCH; ++j)
#pragma unroll
        for (int e = 0; e < DPL; ++e) o[e] = fmaf(pis[j], vv[j][e], o[e]);
    }
    m = mn;
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) store_tiled<T>((T*)a.out, a.o_mtiles, b * a.N + u, h * HD + DPL * lane + e, o[e] / l);
}

template <typename T, int HD, int QPW>
void tail_go(const TreeAttnArgs& a, hipStream_t st) {
  const size_t smem = (size_t)(TAIL_ROWS + MAX_NODES) * (HD + QPW) * sizeof(float);
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)tree_attn_tail<T, HD, QPW>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)smem);
    attr_set = true;
  }
  hipLaunchKernelGGL((tree_attn_tail<T, HD, QPW>), dim3((a.N + QPW - 1) / QPW, a.H, a.B), dim3(64 * QPW), smem, st,
                     a);
}

template <typename T, int HD>
void tree_attn_go(const TreeAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((tree_attn_shared<T, HD>), dim3(a.G, a.H, a.B), dim3(256), 0, st, a);
  const int64_t wgs8 = (int64_t)((a.N + TAIL_QPW - 1) / TAIL_QPW) * a.H * a.B;
  if (wgs8 > 512)
    tail_go<T, HD, TAIL_QPW_WIDE>(a, st);
  else
    tail_go<T, HD, TAIL_QPW>(a, st);
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
  for (int blk = 0; blk < used; ++blk) {
    const float* src = a.part + (((int64_t)row * a.H + h) * a.nblk + blk) * (HD + 2);
    const float mg = src[HD], lg = src[HD + 1];
    if (mg == -CH_INF) continue;
    const float mn = fmaxf(m, mg);
    const float a1 = exp_diff(m, mn), a2 = expf(mg - mn);
    l = l * a1 + lg * a2;
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[e] = o[e] * a1 + src[DPL * lane + e] * a2;
    m = mn;
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
