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
//     position, are reduced per query by a VALU pass that first folds the
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
  const int cmax = (n + a.D) / CHUNK;
  const int last = cmax - 2;            // last chunk any query treats as shared
  const int c_begin = grp * GROUP;
  if (c_begin > last) return;
  const int c_end = min(c_begin + GROUP - 1, last);
  const int lim_u = (n + dep_u) / CHUNK - 2;
  for (int i = tid; i < (c_end - c_begin + 1) * CHUNK; i += 256) {
    const int p = c_begin * CHUNK + i;
    pbase[i] = (int64_t)a.page_table[(int64_t)b * a.max_pages + p / a.ps] * a.page_stride +
               ((int64_t)h * a.ps + p % a.ps) * HD;
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
  auto load_chunk = [&](int c) {
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int idx = tid + 256 * t;
      const int key = idx % CHUNK, part = idx / CHUNK;
      const int64_t base = pbase[(c - c_begin) * CHUNK + key] + part * VEC;
      kreg[t] = ld16(kpool + base);
      vreg[t] = ld16(vpool + base);
    }
  };
  load_chunk(c_begin);
  for (int c = c_begin; c <= c_end; ++c) {
    __syncthreads();
#pragma unroll
    for (int t = 0; t < PER; ++t) {
      const int idx = tid + 256 * t;
      const int key = idx % CHUNK, part = idx / CHUNK;
      st16(&Ks[key * KP + part * VEC], kreg[t]);
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
    mc = fmaxf(mc, __shfl_xor(mc, 16));
    mc = fmaxf(mc, __shfl_xor(mc, 32));
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
    ls = ls + __shfl_xor(ls, 16);
    ls = ls + __shfl_xor(ls, 32);
    l = l * alpha + ls;
    m = mn;
#pragma unroll
    for (int db = 0; db < HD / 16; ++db) o[db] = o[db] * alpha;

    if constexpr (sizeof(T) == 2) {
#pragma unroll
      for (int kp = 0; kp < 2; ++kp) {
        bf16_t pb[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pb[r] = f2bf(s[2 * kp][r]);
          pb[4 + r] = f2bf(s[2 * kp + 1][r]);
        }
        const int4 bfrag = *reinterpret_cast<const int4*>(pb);
#pragma unroll
        for (int db = 0; db < HD / 16; ++db) {
          const T* vr = &Vt[(16 * db + c16) * VP];
          const int2 lo = *reinterpret_cast<const int2*>(vr + 32 * kp + 4 * g);
          const int2 hi = *reinterpret_cast<const int2*>(vr + 32 * kp + 16 + 4 * g);
          o[db] = mfma_kb<T>(int4{lo.x, lo.y, hi.x, hi.y}, bfrag, o[db]);
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
// Tail pass: grid (ceil(N/16), H, B), 16 waves; wave w reduces query
// 16*blockIdx.x + w.  The committed rows of the last chunks and every tree
// slot are staged in LDS once per workgroup.  Loads that do not depend on
// each other are issued together: (query, n) -> (page offsets, tree paths,
// first batch of shared-pass partials) -> staged rows.
// ---------------------------------------------------------------------------
template <typename T, int HD>
__global__ __launch_bounds__(1024) void tree_attn_tail(const TreeAttnArgs a) {
  constexpr int VEC = ET<T>::VEC;
  constexpr int KP = HD + VEC;
  constexpr int ROWS = TAIL_ROWS + MAX_NODES;
  constexpr int DPL = HD / 64;  // output dims per lane
  constexpr int PARTS = HD / VEC;
  constexpr int BATCH = 8;      // shared-pass partials loaded per round trip
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  T* Kl = reinterpret_cast<T*>(smem);
  T* Vl = Kl + ROWS * KP;
  float* qs = reinterpret_cast<float*>(Vl + ROWS * HD);
  __shared__ int64_t rowbase[ROWS];
  __shared__ uint8_t spath[16][64];
  __shared__ int sdepth[16];

  const int h = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int u = 16 * blockIdx.x + wave;
  const bool active = u < a.N;
  // round trip 1: the query row, n, tree metadata of this workgroup's queries
  T qv[DPL];
  if (active) {
    const T* qrow = (const T*)a.q + (int64_t)(b * a.N + u) * a.ldq + h * HD + DPL * lane;
#pragma unroll
    for (int e = 0; e < DPL; ++e) qv[e] = qrow[e];
  }
  for (int i = tid; i < 16 * 64; i += 1024) {
    const int uu = 16 * blockIdx.x + i / 64;
    spath[i / 64][i % 64] = uu < a.N ? a.path[uu * 64 + i % 64] : 0;
  }
  if (tid < 16) sdepth[tid] = (16 * blockIdx.x + tid) < a.N ? a.depth[16 * blockIdx.x + tid] : 0;
  const int n = a.n_b[b];
  const int cmin = n / CHUNK;
  const int lo = (cmin >= 1 ? cmin - 1 : 0) * CHUNK;  // first staged committed position
  const int nc = n - lo;                               // committed rows staged (<= 127)
  const T* kpool = (const T*)a.kpool;
  const T* vpool = (const T*)a.vpool;
  const int* ptab = a.page_table + (int64_t)b * a.max_pages;
  const int nrows_total = nc + a.N;
  // round trip 2: page offsets of the staged rows, first batch of partials
  for (int rr = tid; rr < nrows_total; rr += 1024) {
    const int p = rr < nc ? lo + rr : n + (rr - nc);
    rowbase[rr] = (int64_t)ptab[p / a.ps] * a.page_stride + ((int64_t)h * a.ps + p % a.ps) * HD;
  }
  // groups every query of the tree folds are bounded by those of the deepest node
  const int ngrp_max = ((n + a.D) / CHUNK - 2) >= 0 ? ((n + a.D) / CHUNK - 2) / GROUP + 1 : 0;
  float bm[BATCH], bl[BATCH], bo[BATCH][DPL];
  auto load_batch = [&](int g0) {
#pragma unroll
    for (int t = 0; t < BATCH; ++t) {
      bm[t] = -CH_INF;
      bl[t] = 0.f;
#pragma unroll
      for (int e = 0; e < DPL; ++e) bo[t][e] = 0.f;
      if (active && g0 + t < ngrp_max) {
        const int64_t slot = (((int64_t)b * a.H + h) * a.G + g0 + t) * a.N + u;
        bm[t] = a.part_ml[slot * 2];
        bl[t] = a.part_ml[slot * 2 + 1];
#pragma unroll
        for (int e = 0; e < DPL; ++e) bo[t][e] = a.part_o[slot * HD + DPL * lane + e];
      }
    }
  };
  load_batch(0);
  if (active) {
#pragma unroll
    for (int e = 0; e < DPL; ++e) qs[wave * HD + DPL * lane + e] = ET<T>::to_f(qv[e]);
  }
  __syncthreads();
  // round trip 3: the staged rows
  {
    constexpr int UNR = (ROWS * PARTS + 1023) / 1024;
    int4 kbuf[UNR], vbuf[UNR];
#pragma unroll
    for (int t = 0; t < UNR; ++t) {
      const int idx = tid + 1024 * t;
      if (idx < nrows_total * PARTS) {
        const int64_t base = rowbase[idx / PARTS] + (idx % PARTS) * VEC;
        kbuf[t] = ld16(kpool + base);
        vbuf[t] = ld16(vpool + base);
      }
    }
#pragma unroll
    for (int t = 0; t < UNR; ++t) {
      const int idx = tid + 1024 * t;
      if (idx < nrows_total * PARTS) {
        const int rr = idx / PARTS, part = idx % PARTS;
        const int dst = rr < nc ? rr : TAIL_ROWS + (rr - nc);
        st16(&Kl[dst * KP + part * VEC], kbuf[t]);
        st16(&Vl[dst * HD + part * VEC], vbuf[t]);
      }
    }
  }
  __syncthreads();
  if (!active) return;

  const float* q = qs + wave * HD;
  const int Pu = n + sdepth[wave];
  const int cu = Pu / CHUNK;
  // fold the shared-pass partials in group order
  float m = -CH_INF, l = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;
  const int lim = cu - 2;
  const int ngrp = lim >= 0 ? lim / GROUP + 1 : 0;
  for (int g0 = 0; g0 < ngrp; g0 += BATCH) {
    if (g0 > 0) load_batch(g0);
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
  }
  // the last two chunks, keys in logical-position order
  for (int c = (cu >= 1 ? cu - 1 : 0); c <= cu; ++c) {
    const int p = c * CHUNK + lane;
    const bool valid = p <= Pu;
    int row = 0;
    float s = -CH_INF;
    if (valid) {
      row = p < n ? p - lo : TAIL_ROWS + (int)spath[wave][p - n];
      const T* kr = &Kl[row * KP];
      float acc = 0.f;
#pragma unroll
      for (int part = 0; part < PARTS; ++part) {
        const int4 kv = ld16(kr + part * VEC);
        const T* ke = reinterpret_cast<const T*>(&kv);
#pragma unroll
        for (int e4 = 0; e4 < VEC; e4 += 4) {
          const float4 qq = *reinterpret_cast<const float4*>(q + part * VEC + e4);
          acc = fmaf(qq.x, ET<T>::to_f(ke[e4 + 0]), acc);
          acc = fmaf(qq.y, ET<T>::to_f(ke[e4 + 1]), acc);
          acc = fmaf(qq.z, ET<T>::to_f(ke[e4 + 2]), acc);
          acc = fmaf(qq.w, ET<T>::to_f(ke[e4 + 3]), acc);
        }
      }
      s = acc * a.scale;
    }
    const float mc = wave_max(s);
    const float mn = fmaxf(m, mc);
    const float alpha = exp_diff(m, mn);
    const float pe = valid ? expf(s - mn) : 0.f;
    l = l * alpha + wave_sum(pe);
#pragma unroll
    for (int e = 0; e < DPL; ++e) o[e] = o[e] * alpha;
    const int cnt = min(CHUNK, Pu - c * CHUNK + 1);
#pragma unroll
    for (int i = 0; i < CHUNK; ++i) {
      if (i < cnt) {
        const float pi = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pe), i));
        const int ri = __builtin_amdgcn_readlane(row, i);
        const T* vr = &Vl[ri * HD + DPL * lane];
        if constexpr (sizeof(T) == 2 && DPL == 2) {
          const uint32_t u2 = *reinterpret_cast<const uint32_t*>(vr);
          o[0] = fmaf(pi, __uint_as_float(u2 << 16), o[0]);
          o[1] = fmaf(pi, __uint_as_float(u2 & 0xffff0000u), o[1]);
        } else {
#pragma unroll
          for (int e = 0; e < DPL; ++e) o[e] = fmaf(pi, ET<T>::to_f(vr[e]), o[e]);
        }
      }
    }
    m = mn;
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) store_tiled<T>((T*)a.out, a.o_mtiles, b * a.N + u, h * HD + DPL * lane + e, o[e] / l);
}

template <typename T, int HD>
void tree_attn_go(const TreeAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((tree_attn_shared<T, HD>), dim3(a.G, a.H, a.B), dim3(256), 0, st, a);
  constexpr int VEC = ET<T>::VEC;
  const size_t smem = (size_t)(TAIL_ROWS + MAX_NODES) * ((HD + VEC) + HD) * sizeof(T) + 16 * HD * sizeof(float);
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute((const void*)tree_attn_tail<T, HD>, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)smem);
    attr_set = true;
  }
  hipLaunchKernelGGL((tree_attn_tail<T, HD>), dim3((a.N + 15) / 16, a.H, a.B), dim3(1024), smem, st, a);
}

// ---------------------------------------------------------------------------
// Draft encoder attention: one query per sequence (trigram position n+k)
// over the target-state entries 0..n-1 and trigram entries 0..n+k.
// grid (key blocks of 256, H, B); each wave reduces 64 keys, four at a
// time: lane group sub = lane >> 4 takes key 4*kg + sub and lane c =
// lane & 15 the head-dim slice [c*HD/16, (c+1)*HD/16).
// ---------------------------------------------------------------------------
template <typename T, int HD>
__global__ __launch_bounds__(256) void enc_attn_partial(const EncAttnArgs a) {
  constexpr int DS = HD / 16;            // dims per lane
  constexpr int VEC = ET<T>::VEC;
  static_assert(DS % VEC == 0 || VEC % DS == 0, "slice");
  __shared__ float wm[4], wl[4];
  __shared__ float wo[4][HD];
  const int blk = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
  const int n = a.n_b[b];
  const int nkeys = 2 * n + a.step + 1;
  const int nblk_used = (nkeys + 255) / 256;
  if (blk >= nblk_used) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane >> 4, c = lane & 15;
  float q[DS];
  {
    const T* qrow = (const T*)a.q + (int64_t)b * a.ldq + h * HD + c * DS;
#pragma unroll
    for (int e = 0; e < DS; ++e) q[e] = ET<T>::to_f(qrow[e]);
  }
  const int key0 = blk * 256 + wave * 64;
  auto row_ptr = [&](const void* base, int k) -> const T* {
    const int stream = k < n ? 0 : 1;
    const int pos = k < n ? k : k - n;
    return (const T*)base + ((((int64_t)b * 2 + stream) * a.H + h) * a.cap + pos) * HD + c * DS;
  };
  float sc[16];
  float mloc = -CH_INF;
#pragma unroll
  for (int kg = 0; kg < 16; ++kg) {
    const int key = key0 + 4 * kg + sub;
    float d = 0.f;
    if (key < nkeys) {
      const T* kr = row_ptr(a.kbase, key);
#pragma unroll
      for (int e = 0; e < DS; ++e) d = fmaf(q[e], ET<T>::to_f(kr[e]), d);
    }
    d = d + __shfl_xor(d, 1);
    d = d + __shfl_xor(d, 2);
    d = d + __shfl_xor(d, 4);
    d = d + __shfl_xor(d, 8);
    sc[kg] = key < nkeys ? d * a.scale : -CH_INF;
    mloc = fmaxf(mloc, sc[kg]);
  }
  mloc = fmaxf(mloc, __shfl_xor(mloc, 16));
  const float mw = fmaxf(mloc, __shfl_xor(mloc, 32));
  float lsum = 0.f, o[DS];
#pragma unroll
  for (int e = 0; e < DS; ++e) o[e] = 0.f;
#pragma unroll
  for (int kg = 0; kg < 16; ++kg) {
    const int key = key0 + 4 * kg + sub;
    const float p = (key < nkeys && mw != -CH_INF) ? expf(sc[kg] - mw) : 0.f;
    lsum = lsum + p;
    if (key < nkeys) {
      const T* vr = row_ptr(a.vbase, key);
#pragma unroll
      for (int e = 0; e < DS; ++e) o[e] = fmaf(p, ET<T>::to_f(vr[e]), o[e]);
    }
  }
  lsum = lsum + __shfl_xor(lsum, 16);
  lsum = lsum + __shfl_xor(lsum, 32);
#pragma unroll
  for (int e = 0; e < DS; ++e) {
    o[e] = o[e] + __shfl_xor(o[e], 16);
    o[e] = o[e] + __shfl_xor(o[e], 32);
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
  float* dst = a.part + (((int64_t)b * a.H + h) * a.nblk + blk) * (HD + 2);
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
  const int h = blockIdx.x, b = blockIdx.y, lane = threadIdx.x;
  const int n = a.n_b[b];
  const int nkeys = 2 * n + a.step + 1;
  const int used = (nkeys + 255) / 256;
  float m = -CH_INF, l = 0.f, o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) o[e] = 0.f;
  for (int blk = 0; blk < used; ++blk) {
    const float* src = a.part + (((int64_t)b * a.H + h) * a.nblk + blk) * (HD + 2);
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
  for (int e = 0; e < DPL; ++e) store_tiled<T>((T*)a.out, a.o_mtiles, b, h * HD + DPL * lane + e, o[e] / l);
}

template <typename T, int HD>
void enc_attn_go(const EncAttnArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((enc_attn_partial<T, HD>), dim3(a.nblk, a.H, a.B), dim3(256), 0, st, a);
  hipLaunchKernelGGL((enc_attn_combine<T, HD>), dim3(a.H, a.B), dim3(64), 0, st, a);
}

}  // namespace

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
