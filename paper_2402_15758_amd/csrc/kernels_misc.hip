// Decode-state kernels: embedding gather, RMSNorm with fused residual add,
// argmax and top-s selection, tree assembly, greedy acceptance, in-place KV
// compaction, state advance, and the row setup of the draft and prefill.
#include "common.h"
#include "kernels.h"

namespace {


template <typename T>
__global__ void embed_kernel(const int* __restrict__ tokens, const T* __restrict__ E, float* __restrict__ x, int d,
                             int V) {
  const int r = blockIdx.x;
  const int t = min(max(tokens[r], 0), V - 1);
  const T* e = E + (int64_t)t * d;
  float* xr = x + (int64_t)r * d;
  constexpr int VEC = ET<T>::VEC, U = 4;  // 16-byte pieces, U per thread requested at once
  const int pieces = d / VEC;
  for (int p0 = threadIdx.x; p0 < pieces; p0 += U * 256) {
    int4 buf[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (p0 + 256 * u < pieces) buf[u] = ld16(e + (int64_t)(p0 + 256 * u) * VEC);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (p0 + 256 * u >= pieces) break;
      const T* v = reinterpret_cast<const T*>(&buf[u]);
#pragma unroll
      for (int k = 0; k < VEC; ++k) xr[(p0 + 256 * u) * VEC + k] = ET<T>::to_f(v[k]);
    }
  }
  for (int i = pieces * VEC + threadIdx.x; i < d; i += 256) xr[i] = ET<T>::to_f(e[i]);  // d % VEC tail
}

// Fixed-order block sum: wave butterflies, then the waves in order.
template <int NW>
__device__ __forceinline__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  float t = sh[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) t = t + sh[w];
  return t;
}

// 4 consecutive elements of the storage type as floats / back.
template <typename T>
__device__ __forceinline__ float4 ld4f(const T* p);
template <>
__device__ __forceinline__ float4 ld4f<float>(const float* p) { return *reinterpret_cast<const float4*>(p); }
template <>
__device__ __forceinline__ float4 ld4f<bf16_t>(const bf16_t* p) {
  const uint2 u = *reinterpret_cast<const uint2*>(p);
  return float4{__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                __uint_as_float(u.y & 0xffff0000u)};
}
template <typename T>
__device__ __forceinline__ void st4f(T* p, float4 v);
template <>
__device__ __forceinline__ void st4f<float>(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
template <>
__device__ __forceinline__ void st4f<bf16_t>(bf16_t* p, float4 v) {
  uint2 u;
  u.x = (uint32_t)f2bf(v.x) | ((uint32_t)f2bf(v.y) << 16);
  u.y = (uint32_t)f2bf(v.z) | ((uint32_t)f2bf(v.w) << 16);
  *reinterpret_cast<uint2*>(p) = u;
}

// One workgroup of 1024 threads per row; thread t owns the float4 groups
// t, t+1024, ... (NV of them).  Fixed-order sum of squares.
template <typename T, int NV>
__global__ __launch_bounds__(1024) void rmsnorm_kernel(float* __restrict__ x, const float* __restrict__ parts,
                                                      int n_parts, const float* __restrict__ gamma, T* __restrict__ out,
                                                      int o_mtiles, T* __restrict__ out_rm, int M, int d, float eps,
                                                      int write_back, const T* __restrict__ alt, int alt_begin,
                                                      int alt_end) {
  __shared__ float sh[16];
  const int r = blockIdx.x;
  const bool use_alt = alt != nullptr && r >= alt_begin && r < alt_end;
  float4 v[NV], gm[NV];
  float ss = 0.f;
  // every load is issued before any is used: the gains, the row, and all of
  // its split-K partials (then summed in slice order)
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = 4 * (threadIdx.x + 1024 * j);
    gm[j] = i < d ? *reinterpret_cast<const float4*>(gamma + i) : float4{0.f, 0.f, 0.f, 0.f};
  }
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = 4 * (threadIdx.x + 1024 * j);
    float4 val = float4{0.f, 0.f, 0.f, 0.f};
    if (i < d) {
      if (use_alt) {
        val = ld4f<T>(alt + (int64_t)(r - alt_begin) * d + i);
      } else {
        val = *reinterpret_cast<const float4*>(x + (int64_t)r * d + i);
        float4 pq[GEMM_MAX_SPLITS];
#pragma unroll
        for (int q = 0; q < GEMM_MAX_SPLITS; ++q)
          if (q < n_parts) pq[q] = *reinterpret_cast<const float4*>(parts + ((int64_t)q * M + r) * d + i);
        if (n_parts > 0) {
          float4 f = pq[0];
#pragma unroll
          for (int q = 1; q < GEMM_MAX_SPLITS; ++q) {
            if (q < n_parts) {
              f.x = f.x + pq[q].x;
              f.y = f.y + pq[q].y;
              f.z = f.z + pq[q].z;
              f.w = f.w + pq[q].w;
            }
          }
          val.x = val.x + f.x;
          val.y = val.y + f.y;
          val.z = val.z + f.z;
          val.w = val.w + f.w;
          if (write_back) *reinterpret_cast<float4*>(x + (int64_t)r * d + i) = val;
        }
      }
    }
    v[j] = val;
    ss = fmaf(val.x, val.x, ss);
    ss = fmaf(val.y, val.y, ss);
    ss = fmaf(val.z, val.z, ss);
    ss = fmaf(val.w, val.w, ss);
  }
  ss = block_sum<16>(ss, sh);
  const float rinv = 1.0f / sqrtf(ss / (float)d + eps);
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int i = 4 * (threadIdx.x + 1024 * j);
    if (i < d) {
      float4 o;
      o.x = (v[j].x * rinv) * gm[j].x;
      o.y = (v[j].y * rinv) * gm[j].y;
      o.z = (v[j].z * rinv) * gm[j].z;
      o.w = (v[j].w * rinv) * gm[j].w;
      // 4 consecutive columns stay inside one lane's fragment chunk
      st4f<T>(out + tiled_index<T>(o_mtiles, r, i), o);
      if (out_rm != nullptr) st4f<T>(out_rm + (int64_t)r * d + i, o);
    }
  }
}

// (value, id) order: larger value first, then lower id.
__device__ __forceinline__ bool better(float v, int i, float bv, int bi) { return v > bv || (v == bv && i < bi); }

__device__ __forceinline__ void block_best(float& v, int& i, float* shv, int* shi) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(v, m);
    const int oi = __shfl_xor(i, m);
    if (better(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) {
    shv[wave] = v;
    shi[wave] = i;
  }
  __syncthreads();
  v = shv[0];
  i = shi[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w)
    if (better(shv[w], shi[w], v, i)) {
      v = shv[w];
      i = shi[w];
    }
}

// Best (value, id) over the 64 lanes of a wave, on every lane.
__device__ __forceinline__ void wave_best(float& v, int& i) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const float ov = __shfl_xor(v, m);
    const int oi = __shfl_xor(i, m);
    if (better(ov, oi, v, i)) {
      v = ov;
      i = oi;
    }
  }
}

__global__ __launch_bounds__(1024) void argmax_kernel(const float* __restrict__ logits, int V, int* __restrict__ amax) {
  __shared__ float shv[16];
  __shared__ int shi[16];
  const int r = blockIdx.x;
  const float* z = logits + (int64_t)r * V;
  float bv = -CH_INF;
  int bi = 0x7fffffff;
  constexpr int U = 8;  // float4 pieces per thread requested at once
  for (int b4 = threadIdx.x; 4 * b4 < V; b4 += U * 1024) {
    float4 q[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (4 * (b4 + 1024 * u) < V) q[u] = *reinterpret_cast<const float4*>(z + 4 * (b4 + 1024 * u));
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int i4 = b4 + 1024 * u;
      if (4 * i4 >= V) break;
      const float e[4] = {q[u].x, q[u].y, q[u].z, q[u].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const float v = (e[k] != e[k]) ? -CH_INF : e[k];
        if (better(v, 4 * i4 + k, bv, bi)) {
          bv = v;
          bi = 4 * i4 + k;
        }
      }
    }
  }
  block_best(bv, bi, shv, shi);
  if (threadIdx.x == 0) amax[r] = bi < V ? bi : 0;
}

// Top-s of draft head `level` for every sequence, with the forced-acceptance
// rule; the rank-0 entry becomes the chain token at position n + 1 + level.
// Stage 1: TOPK_SPLIT workgroups per sequence keep the best S ids of their
// slice (excluding the reference id); stage 2 merges them.
constexpr int TOPK_SPLIT = 32;
constexpr int SMAX = 8;

__device__ __forceinline__ int forced_ref(const StepState& s, int b, int level, int V, bool* ok) {
  *ok = false;
  if (s.f_ref == nullptr) return -1;
  const int j = s.n[b] + 1 + level;
  int g = s.f_ref[(int64_t)b * s.f_stride + j];
  if (g < 0 || g >= V) return -1;
  *ok = s.f_ok[(int64_t)b * s.f_stride + j] != 0;
  return g;
}

__global__ __launch_bounds__(256) void topk_partial_kernel(const float* __restrict__ logits, int64_t ld, StepState s,
                                                           DraftLevel dl, float* __restrict__ pv,
                                                           int* __restrict__ pi) {
  __shared__ float shv[4 * SMAX];
  __shared__ int shi[4 * SMAX];
  const int split = blockIdx.x, r = blockIdx.y, b = r / dl.R;
  const int V = s.V, level = dl.level;
  const int S = s.s_k[level];
  bool ok;
  const int excl = forced_ref(s, b, level, V, &ok);
  const float* z = logits + (int64_t)r * ld;
  const int lo = (int)((int64_t)V * split / TOPK_SPLIT), hi = (int)((int64_t)V * (split + 1) / TOPK_SPLIT);
  float lv[SMAX];
  int li[SMAX];
#pragma unroll
  for (int q = 0; q < SMAX; ++q) {
    lv[q] = -CH_INF;
    li[q] = 0x7fffffff;
  }
  // PT values per thread are requested before any is compared
  constexpr int PT = 4;
  for (int base = lo + threadIdx.x; base < hi; base += 256 * PT) {
    float zv[PT];
#pragma unroll
    for (int t = 0; t < PT; ++t) zv[t] = base + 256 * t < hi ? z[base + 256 * t] : -CH_INF;
#pragma unroll
    for (int t = 0; t < PT; ++t) {
      const int i = base + 256 * t;
      if (i >= hi || i == excl) continue;
      float v = zv[t];
      v = (v != v) ? -CH_INF : v;
      if (!better(v, i, lv[SMAX - 1], li[SMAX - 1])) continue;
      // insert into the sorted local list
      float cv = v;
      int ci = i;
#pragma unroll
      for (int q = 0; q < SMAX; ++q) {
        if (better(cv, ci, lv[q], li[q])) {
          const float tv = lv[q];
          const int ti = li[q];
          lv[q] = cv;
          li[q] = ci;
          cv = tv;
          ci = ti;
        }
      }
    }
  }
  // each wave's best S from its lanes' sorted lists, then the workgroup's
  // best S from the waves' 4 S candidates (one barrier)
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int head = 0;
  for (int q = 0; q < S; ++q) {
    float hv = -CH_INF;
    int hi_ = 0x7fffffff;
#pragma unroll
    for (int e = 0; e < SMAX; ++e)
      if (e == head) {
        hv = lv[e];
        hi_ = li[e];
      }
    float bv = hv;
    int bi = hi_;
    wave_best(bv, bi);
    if (bi == hi_ && hi_ != 0x7fffffff) ++head;
    if (lane == 0) {
      shv[wave * SMAX + q] = bv;
      shi[wave * SMAX + q] = bi;
    }
  }
  __syncthreads();
  if (wave != 0) return;
  float cv = -CH_INF;
  int ci = 0x7fffffff;
  if (lane < 4 * S) {
    cv = shv[(lane / S) * SMAX + lane % S];
    ci = shi[(lane / S) * SMAX + lane % S];
  }
  for (int q = 0; q < S; ++q) {
    float bv = cv;
    int bi = ci;
    wave_best(bv, bi);
    if (bi == ci && ci != 0x7fffffff) {
      cv = -CH_INF;
      ci = 0x7fffffff;
    }
    if (lane == 0) {
      pv[((int64_t)r * TOPK_SPLIT + split) * SMAX + q] = bv;
      pi[((int64_t)r * TOPK_SPLIT + split) * SMAX + q] = bi;
    }
  }
}

__global__ __launch_bounds__(64) void topk_merge_kernel(StepState s, DraftLevel lv, const float* __restrict__ pv,
                                                        const int* __restrict__ pi) {
  const int row = blockIdx.x, lane = threadIdx.x;
  const int b = row / lv.R, node = s.d_nodes[lv.off + row % lv.R];
  const int V = s.V, level = lv.level;
  const int S = s.s_k[level];
  bool ok;
  const int g = forced_ref(s, b, level, V, &ok);
  // lane holds candidates lane, lane+64, ... of the TOPK_SPLIT*S list
  constexpr int PER = (TOPK_SPLIT * SMAX + 63) / 64;
  float cv[PER];
  int ci[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int idx = lane + 64 * q;
    const int sp = idx / SMAX, r = idx % SMAX;
    const bool valid = sp < TOPK_SPLIT && r < S;
    cv[q] = valid ? pv[((int64_t)row * TOPK_SPLIT + sp) * SMAX + r] : -CH_INF;
    ci[q] = valid ? pi[((int64_t)row * TOPK_SPLIT + sp) * SMAX + r] : 0x7fffffff;
  }
  int* out = s.cand + ((int64_t)b * 64 + node) * 8;
  int first = 0;
  if (ok) {
    if (lane == 0) out[0] = g;
    first = 1;
  }
  for (int r = first; r < S; ++r) {
    float bv = -CH_INF;
    int bi = 0x7fffffff;
    int bq = -1;
#pragma unroll
    for (int q = 0; q < PER; ++q)
      if (better(cv[q], ci[q], bv, bi)) {
        bv = cv[q];
        bi = ci[q];
        bq = q;
      }
    float wv = bv;
    int wi = bi;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = __shfl_xor(wv, m);
      const int oi = __shfl_xor(wi, m);
      if (better(ov, oi, wv, wi)) {
        wv = ov;
        wi = oi;
      }
    }
    if (bq >= 0 && bi == wi) {
#pragma unroll
      for (int q = 0; q < PER; ++q)
        if (q == bq) cv[q] = -CH_INF, ci[q] = 0x7fffffff;
    }
    const int id = wi < V ? wi : 0;
    if (lane == 0) out[r] = id;
  }
}

__global__ void tree_setup_kernel(StepState s) {
  const int b = blockIdx.x, u = threadIdx.x;
  if (u >= s.N) return;
  const int n = s.n[b];
  const int dep = s.t_depth[u];
  int t;
  if (u == 0)
    t = s.tok[(int64_t)b * s.tok_stride + n];
  else if (s.inject_on[0])
    t = s.inject[(int64_t)b * (s.N - 1) + u - 1];
  else
    t = s.cand[((int64_t)b * 64 + s.tok_src[u]) * 8 + s.t_rank[u]];
  const int row = b * s.N + u;
  s.tree_tok[row] = t;
  const int slot = n + u;
  s.v_pos[row] = n + dep;
  s.v_qrow[row] = row;
  s.v_kvoff[row] =
      (int64_t)s.page_table[(int64_t)b * s.max_pages + slot / s.ps] * s.page_stride + (int64_t)(slot % s.ps) * s.hd;
}

// Greedy acceptance, one wave per sequence, lane = tree node.
__device__ __forceinline__ double readlane_f64(double x, int lane) {
  const unsigned long long u = (unsigned long long)__double_as_longlong(x);
  const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)u, lane);
  const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(u >> 32), lane);
  return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

__global__ void accept_kernel(StepState s) {
  const int b = blockIdx.x, u = threadIdx.x;
  const bool valid = u < s.N;
  const int row = b * s.N + (valid ? u : 0);
  const int tok_u = s.tree_tok[row];
  const int par = valid ? s.t_parent[u] : -1;
  const unsigned long long anc = valid ? s.t_anc[u] : 0ull;
  const int dep = s.t_depth[valid ? u : 0];
  int v, bonus;
  if (!s.typical) {
    // greedy: every non-root token equals the target argmax at its parent;
    // the deepest such node (unique: siblings are distinct)
    const int a_u = s.amax[row];
    const int a_par = par >= 0 ? s.amax[b * s.N + par] : -1;
    const bool good = valid && (u == 0 || tok_u == a_par);
    const unsigned long long goodmask = __ballot(good);
    const bool acc = valid && ((anc & ~goodmask) == 0ull);
    int key = acc ? dep : -1;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) key = max(key, __shfl_xor(key, m));
    const unsigned long long vmask = __ballot(acc && dep == key);
    v = __ffsll((long long)vmask) - 1;
    bonus = __shfl(a_u, v);
  } else {
    // typical: a node passes when p_parent(tok) > min(eps, delta exp(-H_parent));
    // the deepest node whose root path passes, then the highest path
    // log-probability, then the lowest index
    double lp = 0.0;
    bool ok = true;
    if (valid && u > 0) {
      const int pr = b * s.N + par;
      lp = (double)(s.logits[(int64_t)pr * s.V + tok_u] * s.inv_T) - s.t_lse[pr];
      const double thr = fmin((double)s.eps, (double)s.delta * exp(-s.t_H[pr]));
      ok = thr <= 0.0 || lp > log(thr);
    }
    const unsigned long long okmask = __ballot(valid && ok);
    const bool acc = valid && ((anc & ~okmask) == 0ull);
    double plp = 0.0;  // path log-probability, ancestors in id (= depth) order
    for (int x = 0; x < s.N; ++x) {
      const double lx = readlane_f64(lp, x);
      if ((anc >> x) & 1ull) plp += lx;
    }
    const unsigned long long accmask = __ballot(acc);
    int best = 0, bd = -1;
    double bp = 0.0;
    for (int x = 0; x < s.N; ++x) {
      const int dx = __builtin_amdgcn_readlane(dep, x);
      const double px = readlane_f64(plp, x);
      if (((accmask >> x) & 1ull) && (dx > bd || (dx == bd && px > bp))) {
        best = x;
        bd = dx;
        bp = px;
      }
    }
    v = best;
    bonus = s.t_sample[b * s.N + v];
  }
  const unsigned long long path = __shfl(anc, v);
  const int L = __popcll(path);
  const int K1 = s.K + 1;
  if (valid && ((path >> u) & 1ull)) {
    const int idx = __popcll(path & ((1ull << u) - 1ull));
    s.out_nodes[b * K1 + idx] = u;
    if (idx >= 1) s.out_tok[b * K1 + idx - 1] = tok_u;
  }
  if (u == 0) {
    s.out_tok[b * K1 + L - 1] = bonus;
    s.out_len[b] = L;
  }
}

__device__ __forceinline__ unsigned long long splitmix64_d(unsigned long long x) {
  unsigned long long z = x + 0x9e3779b97f4a7c15ull;
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

// One workgroup per logits row; fp64 accumulation, fixed reduction order.
__global__ __launch_bounds__(1024) void typical_stats_kernel(const float* __restrict__ logits, int V, int N, int b0,
                                                             const int* __restrict__ n_b, const int* __restrict__ depth,
                                                             int fixed_pos, float inv_T, unsigned long long seed,
                                                             double* lse, double* Hout, int* sample) {
  const int r = blockIdx.x, tid = threadIdx.x;
  const int b = b0 + r / N;
  const int pos = fixed_pos >= 0 ? fixed_pos : n_b[b] + depth[r % N] + 1;
  const float* l = logits + (int64_t)r * V;
  __shared__ double red_a[1024], red_b[1024];
  __shared__ int red_i[1024];
  __shared__ float red_m[1024];
  float m = -CH_INF;
  for (int v = tid; v < V; v += 1024) m = fmaxf(m, l[v] * inv_T);
  red_m[tid] = m;
  __syncthreads();
  for (int w = 512; w >= 1; w >>= 1) {
    if (tid < w) red_m[tid] = fmaxf(red_m[tid], red_m[tid + w]);
    __syncthreads();
  }
  const double mx = (double)red_m[0];
  const unsigned long long base = splitmix64_d(splitmix64_d(splitmix64_d(seed) ^ (unsigned long long)b) ^
                                               (unsigned long long)pos);
  double S = 0.0, E = 0.0, best = -HUGE_VAL;
  int bi = 0x7fffffff;
  for (int v = tid; v < V; v += 1024) {
    const double z = (double)(l[v] * inv_T);
    const double e = exp(z - mx);
    S += e;
    E += e * (z - mx);
    const double uu = ((double)(splitmix64_d(base ^ (unsigned long long)v) >> 11) + 0.5) * 0x1p-53;
    const double sc = z - log(-log(uu));
    if (sc > best) {  // ascending v per thread: ties keep the lower id
      best = sc;
      bi = v;
    }
  }
  __syncthreads();
  red_a[tid] = S;
  red_b[tid] = E;
  __syncthreads();
  for (int w = 512; w >= 1; w >>= 1) {
    if (tid < w) {
      red_a[tid] = red_a[tid] + red_a[tid + w];
      red_b[tid] = red_b[tid] + red_b[tid + w];
    }
    __syncthreads();
  }
  const double Ssum = red_a[0], Esum = red_b[0];
  __syncthreads();
  red_a[tid] = best;
  red_i[tid] = bi;
  __syncthreads();
  for (int w = 512; w >= 1; w >>= 1) {
    if (tid < w) {
      const double o = red_a[tid + w];
      const int oi = red_i[tid + w];
      if (o > red_a[tid] || (o == red_a[tid] && oi < red_i[tid])) {
        red_a[tid] = o;
        red_i[tid] = oi;
      }
    }
    __syncthreads();
  }
  if (tid == 0) {
    const double ls = log(Ssum);
    lse[r] = mx + ls;
    Hout[r] = ls - Esum / Ssum;
    sample[r] = red_i[0];
  }
}

// In-place compaction of the accepted path: slot n+d <- slot n+path[d], for
// d = 1..L-1 in increasing order (sources are never below their
// destination, so no source is overwritten before it is read).
template <typename T>
__global__ __launch_bounds__(256) void compact_kernel(StepState s, T* pool, int64_t layer_stride) {
  const int layer = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int L = s.out_len[b];
  const int n = s.n[b];
  const int K1 = s.K + 1;
  constexpr int VEC = ET<T>::VEC;
  T* base = pool + (int64_t)layer * layer_stride + (int64_t)kv * s.H * s.ps * s.hd;
  const int* ptab = s.page_table + (int64_t)b * s.max_pages;
  const int nvec = s.H * s.hd / VEC;
  for (int dd = 1; dd < L; ++dd) {
    const int src = n + s.out_nodes[b * K1 + dd];
    const int dst = n + dd;
    if (src == dst) continue;
    const int64_t sb = (int64_t)ptab[src / s.ps] * s.page_stride + (int64_t)(src % s.ps) * s.hd;
    const int64_t db = (int64_t)ptab[dst / s.ps] * s.page_stride + (int64_t)(dst % s.ps) * s.hd;
    for (int e = threadIdx.x; e < nvec; e += 256) {
      const int h = (e * VEC) / s.hd, dim = (e * VEC) % s.hd;
      const int64_t ho = (int64_t)h * s.ps * s.hd + dim;
      st16(base + db + ho, ld16(base + sb + ho));
    }
  }
}

// Compaction check (debug mode).  Before compaction: node u's K or V row of
// every layer (slot n+u, all heads) is copied to
// side[((layer * 2 + kv) * B + b) * N + u][H * hd].  After compaction: slot
// n+d must hold the copy of node path[d] for d = 0..L-1; counts[0] gains the
// rows compared and counts[1] the 16-byte chunks that differ.
template <typename T>
__global__ __launch_bounds__(256) void kv_snapshot_kernel(StepState s, const T* pool, int64_t layer_stride,
                                                          T* side) {
  const int layer = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int n = s.n[b];
  constexpr int VEC = ET<T>::VEC;
  const T* base = pool + (int64_t)layer * layer_stride + (int64_t)kv * s.H * s.ps * s.hd;
  const int* ptab = s.page_table + (int64_t)b * s.max_pages;
  const int nvec = s.H * s.hd / VEC;
  T* dst = side + (((int64_t)layer * 2 + kv) * s.B + b) * s.N * s.H * s.hd;
  for (int u = 0; u < s.N; ++u) {
    const int slot = n + u;
    const int64_t sb = (int64_t)ptab[slot / s.ps] * s.page_stride + (int64_t)(slot % s.ps) * s.hd;
    for (int e = threadIdx.x; e < nvec; e += 256) {
      const int h = (e * VEC) / s.hd, dim = (e * VEC) % s.hd;
      st16(dst + (int64_t)u * s.H * s.hd + e * VEC, ld16(base + sb + (int64_t)h * s.ps * s.hd + dim));
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void kv_check_kernel(StepState s, const T* pool, int64_t layer_stride,
                                                       const T* side, unsigned long long* counts) {
  __shared__ unsigned int bad;
  const int layer = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int L = s.out_len[b];
  const int n = s.n[b];
  const int K1 = s.K + 1;
  constexpr int VEC = ET<T>::VEC;
  const T* base = pool + (int64_t)layer * layer_stride + (int64_t)kv * s.H * s.ps * s.hd;
  const int* ptab = s.page_table + (int64_t)b * s.max_pages;
  const int nvec = s.H * s.hd / VEC;
  const T* snap = side + (((int64_t)layer * 2 + kv) * s.B + b) * s.N * s.H * s.hd;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  unsigned int mine = 0;
  for (int dd = 0; dd < L; ++dd) {
    const int u = s.out_nodes[b * K1 + dd];
    const int slot = n + dd;
    const int64_t db = (int64_t)ptab[slot / s.ps] * s.page_stride + (int64_t)(slot % s.ps) * s.hd;
    for (int e = threadIdx.x; e < nvec; e += 256) {
      const int h = (e * VEC) / s.hd, dim = (e * VEC) % s.hd;
      const int4 got = ld16(base + db + (int64_t)h * s.ps * s.hd + dim);
      const int4 want = ld16(snap + (int64_t)u * s.H * s.hd + e * VEC);
      mine += (got.x != want.x || got.y != want.y || got.z != want.z || got.w != want.w) ? 1u : 0u;
    }
  }
  if (mine) atomicAdd(&bad, mine);
  __syncthreads();
  if (threadIdx.x == 0) {
    atomicAdd(&counts[0], (unsigned long long)L);
    if (bad) atomicAdd(&counts[1], (unsigned long long)bad);
  }
}

// Workgroup (b, idx) moves accepted row idx of sequence b into the encoder
// prologue rows (and h_last for the last one); workgroup (b, 0) also commits
// the tokens and advances n.
template <typename T>
__global__ __launch_bounds__(256) void advance_kernel(StepState s) {
  const int b = blockIdx.x, idx = blockIdx.y;
  const int L = s.out_len[b];
  const int K1 = s.K + 1;
  const int d = s.d;
  if (idx < L) {
    const int node = s.out_nodes[b * K1 + idx];
    const T* src = (const T*)s.hl + (int64_t)(b * s.N + node) * d;
    T* dst = (T*)s.pro_h + ((int64_t)b * K1 + idx) * d;
    T* hl = idx == L - 1 ? (T*)s.h_last + (int64_t)b * d : nullptr;
    for (int i = threadIdx.x; i < d; i += 256) {
      const T v = src[i];
      dst[i] = v;
      if (hl) hl[i] = v;
    }
  }
  if (idx != 0) return;
  const int n = s.n[b];
  if (threadIdx.x < L) s.tok[(int64_t)b * s.tok_stride + n + 1 + threadIdx.x] = s.out_tok[b * K1 + threadIdx.x];
  __syncthreads();
  if (threadIdx.x == 0) {
    s.pro_base[b] = n;
    s.pro_count[b] = L;
    s.n[b] = n + L;
    if (b == 0) s.inject_on[0] = 0;  // injected tree tokens apply to one step only
  }
}

// Token at position q >= 0 of sequence b along draft-tree node `node`'s
// path: committed tokens and the pending one (q <= n) from tok, the draft
// positions n + depth from the drafted lists of the node's ancestors.
// node < 0: committed tokens only (prefill and the prologue rows).
__device__ __forceinline__ int path_token(const StepState& s, int b, int node, int q) {
  if (node < 0) return s.tok[(int64_t)b * s.tok_stride + q];
  const int n = s.n[b];
  if (q <= n) return s.tok[(int64_t)b * s.tok_stride + q];
  const int a = s.d_path[node * 64 + (q - n)];
  return s.cand[((int64_t)b * 64 + s.d_parent[a]) * 8 + s.d_rank[a]];
}

// Trigram input t = [e(pos-2); e(pos-1); e(pos)] of one row, zero vectors
// before the sequence start, written tiled.
template <typename T>
__device__ __forceinline__ void trigram_row(const StepState& s, const T* E, int b, int node, int pos, T* dst,
                                            int mtiles, int row) {
  const int d = s.d;
  int tk[3];
#pragma unroll
  for (int part = 0; part < 3; ++part) tk[part] = pos - 2 + part >= 0 ? path_token(s, b, node, pos - 2 + part) : -1;
  for (int i = blockIdx.y * blockDim.x + threadIdx.x; i < 3 * d; i += gridDim.y * blockDim.x) {
    const int part = i / d, col = i % d;
    T v = ET<T>::from_f(0.f);
    if (tk[part] >= 0) v = E[(int64_t)tk[part] * d + col];
    copy_tiled<T>(dst, mtiles, row, i, v);
  }
}

__device__ __forceinline__ int64_t enc_off(const StepState& s, int b, int stream, int pos) {
  return ((((int64_t)b * 2 + stream) * s.H) * s.cap + pos) * s.hd;
}

template <typename T>
__global__ void draft_rows_kernel(StepState s, const T* E, DraftLevel lv, T* tri_in, int tri_mtiles, int* pos,
                                  int64_t* kvoff, int* qrow) {
  const int r = blockIdx.x;
  const int B = s.B, K1 = s.K + 1, Q = B * lv.R;
  int b, p, node = -1, q = -1;
  int64_t off;
  bool valid = true, want_tri = true;
  if (r < Q) {
    // query: the root's trigram entry lives at stream-1 position n, a deeper
    // node's in its own slot
    b = r / lv.R;
    node = s.d_nodes[lv.off + r % lv.R];
    p = s.n[b] + lv.level;
    q = r;
    off = enc_off(s, b, 1, lv.level == 0 ? p : s.tree_slot0 + node);
  } else if (r < Q + B * K1) {
    const int i = r - Q;
    b = i / K1;
    const int e = i % K1;
    valid = e < s.pro_count[b];
    p = s.pro_base[b] + e;
    off = enc_off(s, b, 0, p);
    want_tri = false;
  } else {
    const int i = r - Q - B * K1;
    b = i / K1;
    const int e = i % K1;
    valid = e < s.pro_count[b];
    p = s.pro_base[b] + e;
    off = enc_off(s, b, 1, p);
  }
  if (threadIdx.x == 0 && blockIdx.y == 0) {
    pos[r] = valid ? p : 0;
    kvoff[r] = valid ? off : -1;
    qrow[r] = q;
  }
  if (want_tri && valid) {
    trigram_row<T>(s, E, b, node, p, tri_in, tri_mtiles, r);
  } else {
    for (int i = blockIdx.y * blockDim.x + threadIdx.x; i < 3 * s.d; i += gridDim.y * blockDim.x)
      copy_tiled<T>(tri_in, tri_mtiles, r, i, ET<T>::from_f(0.f));
  }
}

template <typename T>
__global__ __launch_bounds__(256) void draft_finish_kernel(StepState s, DraftLevel lv, const float* x,
                                                           const float* parts, int n_parts, T* zin, int z_mtiles) {
  const int r = blockIdx.x, b = r / lv.R, d = s.d, M = s.B * lv.R;
  const T* hl = (const T*)s.h_last + (int64_t)b * d;
  for (int i = blockIdx.y * 256 + threadIdx.x; i < d; i += gridDim.y * 256) {
    copy_tiled<T>(zin, z_mtiles, r, i, hl[i]);
    float pq[GEMM_MAX_SPLITS];  // every slice requested before the first is added
#pragma unroll
    for (int q = 0; q < GEMM_MAX_SPLITS; ++q)
      if (q < n_parts) pq[q] = parts[((int64_t)q * M + r) * d + i];
    float f = pq[0];
#pragma unroll
    for (int q = 1; q < GEMM_MAX_SPLITS; ++q)
      if (q < n_parts) f = f + pq[q];
    store_tiled<T>(zin, z_mtiles, r, d + i, x[(int64_t)r * d + i] + f);
  }
}

template <typename T>
__global__ void prefill_rows_kernel(StepState s, const T* E, int b, int p0, int M, int* tokens_out, T* tri_in,
                                    int tri_mtiles, int* enc_pos, int64_t* enc_kvoff, int* enc_qrow, int* pf_n) {
  const int i = blockIdx.x;
  const int p = p0 + i;
  if (threadIdx.x == 0) {
    const int* ptab = s.page_table + (int64_t)b * s.max_pages;
    s.v_pos[i] = p;
    s.v_qrow[i] = i;
    s.v_kvoff[i] = (int64_t)ptab[p / s.ps] * s.page_stride + (int64_t)(p % s.ps) * s.hd;
    tokens_out[i] = s.tok[(int64_t)b * s.tok_stride + p];
    enc_pos[i] = p;
    enc_kvoff[i] = enc_off(s, b, 0, p);
    enc_qrow[i] = -1;
    enc_pos[M + i] = p;
    enc_kvoff[M + i] = enc_off(s, b, 1, p);
    enc_qrow[M + i] = -1;
    if (i == 0) pf_n[0] = p0;  // committed length seen by the chunk's attention
  }
  trigram_row<T>(s, E, b, -1, p, tri_in, tri_mtiles, i);
}

// ---------------------------------------------------------------------------
// Trigram lookup cache
// ---------------------------------------------------------------------------
__device__ __forceinline__ unsigned long long tri_key(const StepState& s, int b, int node, int p) {
  auto t = [&](int q) -> unsigned long long {
    return q >= 0 ? (unsigned long long)(path_token(s, b, node, q) + 1) : 0ull;
  };
  return (t(p - 2) << 42) | (t(p - 1) << 21) | t(p);
}

__device__ __forceinline__ int tri_set(unsigned long long key, int n_sets) {
  unsigned long long z = key + 0x9e3779b97f4a7c15ull;  // SplitMix64 finalizer as the set hash
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  z = z ^ (z >> 31);
  return (int)(z % (unsigned long long)n_sets);
}

// Row r of a draft level (the row order of draft_rows_kernel): the trigram's
// sequence, draft-tree node (-1: committed tokens) and end position, or
// false for rows without a trigram.
__device__ __forceinline__ bool draft_tri_row(const StepState& s, const DraftLevel& lv, int r, int& b, int& node,
                                              int& p) {
  const int B = s.B, K1 = s.K + 1, Q = B * lv.R;
  if (r < Q) {
    b = r / lv.R;
    node = s.d_nodes[lv.off + r % lv.R];
    p = s.n[b] + lv.level;
    return true;
  }
  if (r < Q + B * K1) return false;  // target-state entries
  const int i = r - Q - B * K1;
  b = i / K1;
  const int e = i % K1;
  if (e >= s.pro_count[b]) return false;
  p = s.pro_base[b] + e;
  node = -1;
  return true;
}

__global__ __launch_bounds__(256) void tri_lookup_kernel(StepState s, TriCache c, DraftLevel lv,
                                                         float* __restrict__ htri) {
  const int r = blockIdx.x, d = s.d;
  __shared__ int way;
  int b = 0, node = -1, p = 0;
  if (!draft_tri_row(s, lv, r, b, node, p)) {
    if (threadIdx.x == 0) c.hit[r] = 1;
    return;
  }
  const unsigned long long key = tri_key(s, b, node, p);
  const int set = tri_set(key, c.n_sets);
  if (threadIdx.x == 0) way = -1;
  __syncthreads();
  if (threadIdx.x < TRI_WAYS && c.keys[(int64_t)set * TRI_WAYS + threadIdx.x] == key) way = threadIdx.x;
  __syncthreads();
  const int w = way;
  if (w < 0) {
    if (threadIdx.x == 0) {
      c.hit[r] = 0;
      atomicAdd(c.miss, 1);
      atomicAdd(&c.stats[0], 1ull);
    }
    return;
  }
  const float* src = c.vals + ((int64_t)set * TRI_WAYS + w) * d;
  for (int i = threadIdx.x; i < d; i += 256) htri[(int64_t)r * d + i] = src[i];
  if (threadIdx.x == 0) {
    c.hit[r] = 1;
    c.stamps[(int64_t)set * TRI_WAYS + w] = atomicAdd(c.clock, 1u) + 1u;
    atomicAdd(&c.stats[0], 1ull);
    atomicAdd(&c.stats[1], 1ull);
  }
}

// One workgroup per row.  Only the first missing row of a set inserts in a
// launch (rows of one set never race); a key already present is left alone.
__global__ __launch_bounds__(256) void tri_insert_kernel(StepState s, TriCache c, DraftLevel lv, int pb, int p0,
                                                         int prefill_M, const float* __restrict__ vals) {
  const int r = blockIdx.x, d = s.d;
  __shared__ int victim;
  __shared__ int present;
  if (r == 0 && threadIdx.x == 0) *c.miss = 0;  // consumed by this level's MLP launches
  auto row_of = [&](int rr, int& b, int& node, int& p) -> bool {
    if (prefill_M > 0) {
      b = pb;
      node = -1;
      p = p0 + rr;
      return true;
    }
    return draft_tri_row(s, lv, rr, b, node, p) && c.hit[rr] == 0;
  };
  int b = 0, node = -1, p = 0;
  if (!row_of(r, b, node, p)) return;
  const unsigned long long key = tri_key(s, b, node, p);
  const int set = tri_set(key, c.n_sets);
  for (int r2 = 0; r2 < r; ++r2) {  // an earlier row of this launch owns the set
    int b2, n2, p2;
    if (row_of(r2, b2, n2, p2) && tri_set(tri_key(s, b2, n2, p2), c.n_sets) == set) return;
  }
  if (threadIdx.x == 0) {
    int v = 0, hitw = -1;
    unsigned int best = 0xffffffffu;
    for (int w = 0; w < TRI_WAYS; ++w) {
      const unsigned long long k = c.keys[(int64_t)set * TRI_WAYS + w];
      const unsigned int st = k == 0 ? 0u : c.stamps[(int64_t)set * TRI_WAYS + w];
      if (k == key) hitw = w;
      if (st < best) {
        best = st;
        v = w;
      }
    }
    victim = v;
    present = hitw >= 0;
  }
  __syncthreads();
  if (present) return;
  const int64_t slot = (int64_t)set * TRI_WAYS + victim;
  const float* src = vals + (int64_t)r * d;
  for (int i = threadIdx.x; i < d; i += 256) c.vals[slot * d + i] = src[i];
  if (threadIdx.x == 0) {
    c.keys[slot] = key;
    c.stamps[slot] = atomicAdd(c.clock, 1u) + 1u;
  }
}

template <typename T>
__global__ void prefill_finish_kernel(StepState s, int b, int n, const int* amax_row, const T* hl_row) {
  const int d = s.d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) ((T*)s.h_last)[(int64_t)b * d + i] = hl_row[i];
  if (threadIdx.x == 0) {
    s.tok[(int64_t)b * s.tok_stride + n] = amax_row[0];
    s.n[b] = n;
    s.pro_base[b] = n;
    s.pro_count[b] = 0;
  }
}

}  // namespace

void launch_embed(int dtype, const int* tokens, const void* E, float* x, int M, int d, int V, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(embed_kernel<bf16_t>, dim3(M), dim3(256), 0, st, tokens, (const bf16_t*)E, x, d, V);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, st, tokens, (const float*)E, x, d, V);
}

template <typename T, int NV>
static void norm_go(float* x, const float* parts, int n_parts, const float* gamma, void* out, int ldo, void* out_rm,
                    int M, int d, float eps, int write_back, const void* alt, int alt_begin, int alt_end,
                    hipStream_t st) {
  hipLaunchKernelGGL((rmsnorm_kernel<T, NV>), dim3(M), dim3(1024), 0, st, x, parts, n_parts, gamma, (T*)out, ldo,
                     (T*)out_rm, M, d, eps, write_back, (const T*)alt, alt_begin, alt_end);
}

template <typename T>
static void norm_t(float* x, const float* parts, int n_parts, const float* gamma, void* out, int ldo, void* out_rm,
                   int M, int d, float eps, int write_back, const void* alt, int alt_begin, int alt_end,
                   hipStream_t st) {
  switch ((d + 4095) / 4096) {
    case 1: norm_go<T, 1>(x, parts, n_parts, gamma, out, ldo, out_rm, M, d, eps, write_back, alt, alt_begin, alt_end, st); break;
    default: norm_go<T, 2>(x, parts, n_parts, gamma, out, ldo, out_rm, M, d, eps, write_back, alt, alt_begin, alt_end, st); break;
  }
}

void launch_rmsnorm(int dtype, float* x, const float* parts, int n_parts, const float* gamma, void* out, int ldo,
                    void* out_rm, int M, int d, float eps, int write_back, const void* alt, int alt_begin, int alt_end,
                    hipStream_t st) {
  if (M <= 0) return;
  if (dtype == DT_BF16)
    norm_t<bf16_t>(x, parts, n_parts, gamma, out, ldo, out_rm, M, d, eps, write_back, alt, alt_begin, alt_end, st);
  else
    norm_t<float>(x, parts, n_parts, gamma, out, ldo, out_rm, M, d, eps, write_back, alt, alt_begin, alt_end, st);
}

void launch_argmax(const float* logits, int M, int V, int* amax, hipStream_t st) {
  hipLaunchKernelGGL(argmax_kernel, dim3(M), dim3(1024), 0, st, logits, V, amax);
}

void launch_topk(const float* logits, int64_t ld, const StepState& s, const DraftLevel& lv, float* scratch_v,
                 int* scratch_i, hipStream_t st) {
  const int Q = s.B * lv.R;
  hipLaunchKernelGGL(topk_partial_kernel, dim3(TOPK_SPLIT, Q), dim3(256), 0, st, logits, ld, s, lv, scratch_v,
                     scratch_i);
  hipLaunchKernelGGL(topk_merge_kernel, dim3(Q), dim3(64), 0, st, s, lv, (const float*)scratch_v,
                     (const int*)scratch_i);
}

void launch_tree_setup(const StepState& s, hipStream_t st) {
  hipLaunchKernelGGL(tree_setup_kernel, dim3(s.B), dim3(64), 0, st, s);
}

void launch_typical_stats(const float* logits, int rows, int V, int N, int b0, const int* n_b, const int* depth,
                          int fixed_pos, float inv_T, unsigned long long seed, double* lse, double* H, int* sample,
                          hipStream_t st) {
  hipLaunchKernelGGL(typical_stats_kernel, dim3(rows), dim3(1024), 0, st, logits, V, N, b0, n_b, depth, fixed_pos,
                     inv_T, seed, lse, H, sample);
}

void launch_accept(int, const StepState& s, hipStream_t st) {
  hipLaunchKernelGGL(accept_kernel, dim3(s.B), dim3(64), 0, st, s);
}

void launch_compact(int dtype, const StepState& s, void* pool, int n_layers, int64_t layer_stride, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(compact_kernel<bf16_t>, dim3(n_layers, 2, s.B), dim3(256), 0, st, s, (bf16_t*)pool,
                       layer_stride);
  else
    hipLaunchKernelGGL(compact_kernel<float>, dim3(n_layers, 2, s.B), dim3(256), 0, st, s, (float*)pool,
                       layer_stride);
}

void launch_kv_snapshot(int dtype, const StepState& s, const void* pool, int n_layers, int64_t layer_stride,
                        void* side, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(kv_snapshot_kernel<bf16_t>, dim3(n_layers, 2, s.B), dim3(256), 0, st, s, (const bf16_t*)pool,
                       layer_stride, (bf16_t*)side);
  else
    hipLaunchKernelGGL(kv_snapshot_kernel<float>, dim3(n_layers, 2, s.B), dim3(256), 0, st, s, (const float*)pool,
                       layer_stride, (float*)side);
}

void launch_kv_check(int dtype, const StepState& s, const void* pool, int n_layers, int64_t layer_stride,
                     const void* side, unsigned long long* counts, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(kv_check_kernel<bf16_t>, dim3(n_layers, 2, s.B), dim3(256), 0, st, s, (const bf16_t*)pool,
                       layer_stride, (const bf16_t*)side, counts);
  else
    hipLaunchKernelGGL(kv_check_kernel<float>, dim3(n_layers, 2, s.B), dim3(256), 0, st, s, (const float*)pool,
                       layer_stride, (const float*)side, counts);
}

void launch_advance(int dtype, const StepState& s, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(advance_kernel<bf16_t>, dim3(s.B, s.K + 1), dim3(256), 0, st, s);
  else
    hipLaunchKernelGGL(advance_kernel<float>, dim3(s.B, s.K + 1), dim3(256), 0, st, s);
}

int draft_level_rows(const StepState& s, const DraftLevel& lv) {
  return s.B * lv.R + (lv.level == 0 ? 2 * s.B * (s.K + 1) : 0);
}

void launch_draft_rows(int dtype, const StepState& s, const void* E, const DraftLevel& lv, void* tri_in,
                       int tri_mtiles, int* pos, int64_t* kvoff, int* qrow, hipStream_t st) {
  const dim3 grid(draft_level_rows(s, lv), (3 * s.d + 255) / 256);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(draft_rows_kernel<bf16_t>, grid, dim3(256), 0, st, s, (const bf16_t*)E, lv,
                       (bf16_t*)tri_in, tri_mtiles, pos, kvoff, qrow);
  else
    hipLaunchKernelGGL(draft_rows_kernel<float>, grid, dim3(256), 0, st, s, (const float*)E, lv,
                       (float*)tri_in, tri_mtiles, pos, kvoff, qrow);
}

void launch_draft_finish(int dtype, const StepState& s, const DraftLevel& lv, const float* x, const float* parts,
                         int n_parts, void* zin, int z_mtiles, hipStream_t st) {
  const dim3 grid(s.B * lv.R, (s.d + 255) / 256);
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(draft_finish_kernel<bf16_t>, grid, dim3(256), 0, st, s, lv, x, parts, n_parts,
                       (bf16_t*)zin, z_mtiles);
  else
    hipLaunchKernelGGL(draft_finish_kernel<float>, grid, dim3(256), 0, st, s, lv, x, parts, n_parts,
                       (float*)zin, z_mtiles);
}

void launch_prefill_rows(int dtype, const StepState& s, const void* E, int b, int p0, int M, int* tokens_out,
                         void* tri_in, int tri_mtiles, int* enc_pos, int64_t* enc_kvoff, int* enc_qrow, int* pf_n,
                         hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(prefill_rows_kernel<bf16_t>, dim3(M), dim3(256), 0, st, s, (const bf16_t*)E, b, p0, M,
                       tokens_out, (bf16_t*)tri_in, tri_mtiles, enc_pos, enc_kvoff, enc_qrow, pf_n);
  else
    hipLaunchKernelGGL(prefill_rows_kernel<float>, dim3(M), dim3(256), 0, st, s, (const float*)E, b, p0, M, tokens_out,
                       (float*)tri_in, tri_mtiles, enc_pos, enc_kvoff, enc_qrow, pf_n);
}

void launch_tri_lookup(const StepState& s, const TriCache& c, const DraftLevel& lv, float* htri, hipStream_t st) {
  hipLaunchKernelGGL(tri_lookup_kernel, dim3(draft_level_rows(s, lv)), dim3(256), 0, st, s, c, lv, htri);
}

void launch_tri_insert(const StepState& s, const TriCache& c, const DraftLevel& lv, int b, int p0, int prefill_M,
                       const float* vals, hipStream_t st) {
  const int rows = prefill_M > 0 ? prefill_M : draft_level_rows(s, lv);
  hipLaunchKernelGGL(tri_insert_kernel, dim3(rows), dim3(256), 0, st, s, c, lv, b, p0, prefill_M, vals);
}

void launch_prefill_finish(int dtype, const StepState& s, int b, int n, const int* amax_row, const void* hl_row,
                           hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(prefill_finish_kernel<bf16_t>, dim3(1), dim3(256), 0, st, s, b, n, amax_row,
                       (const bf16_t*)hl_row);
  else
    hipLaunchKernelGGL(prefill_finish_kernel<float>, dim3(1), dim3(256), 0, st, s, b, n, amax_row,
                       (const float*)hl_row);
}

// ---- phase timestamps ---------------------------------------------------------
// One lane reads the GPU's constant-rate wall clock and stores it in the
// current step's ring slot.  Kernels of a stream run one after another, so a
// stamp launched between two phases records when the first phase's last
// kernel has finished, and the four stamps of a step see the same counter.
__global__ void stamp_kernel(unsigned long long* ring, unsigned int* counter, int idx, const int* n_b, int B) {
  if (threadIdx.x != 0) return;
  const unsigned int c = *counter;
  unsigned long long* slot = ring + (size_t)(c % STAMP_RING) * STAMP_WORDS;
  slot[idx] = __builtin_amdgcn_s_memrealtime();
  if (idx == 0) {
    unsigned long long sum = 0;
    for (int b = 0; b < B; ++b) sum += (unsigned long long)n_b[b];
    slot[4] = sum;
  }
  if (idx == 3) *counter = c + 1;
}

void launch_stamp(unsigned long long* ring, unsigned int* counter, int idx, const int* n_b, int B, hipStream_t st) {
  hipLaunchKernelGGL(stamp_kernel, dim3(1), dim3(64), 0, st, ring, counter, idx, n_b, B);
}
