// Decode-state kernels: embedding gather, RMSNorm with fused residual add,
// argmax and top-s selection, tree assembly, greedy acceptance, in-place KV
// compaction, state advance, and the row setup of the draft and prefill.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int MAX_PER_THREAD = 32;  // d <= 8192 with 256 threads

template <typename T>
__global__ void embed_kernel(const int* __restrict__ tokens, const T* __restrict__ E, float* __restrict__ x, int d,
                             int V) {
  const int r = blockIdx.x;
  const int t = min(max(tokens[r], 0), V - 1);
  const T* e = E + (int64_t)t * d;
  for (int i = threadIdx.x; i < d; i += blockDim.x) x[(int64_t)r * d + i] = ET<T>::to_f(e[i]);
}

// Fixed-order block sum (256 threads): wave butterflies, then waves in order.
__device__ __forceinline__ float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wave] = v;
  __syncthreads();
  return ((sh[0] + sh[1]) + sh[2]) + sh[3];
}

template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(float* __restrict__ x, const float* __restrict__ parts,
                                                      int n_parts, const float* __restrict__ gamma, T* __restrict__ out,
                                                      int ldo, int M, int d, float eps, int write_back,
                                                      const T* __restrict__ alt, int alt_begin, int alt_end) {
  __shared__ float sh[4];
  const int r = blockIdx.x;
  const bool use_alt = alt != nullptr && r >= alt_begin && r < alt_end;
  float v[MAX_PER_THREAD];
  float ss = 0.f;
  int c = 0;
  for (int i = threadIdx.x; i < d; i += 256, ++c) {
    float val;
    if (use_alt) {
      val = ET<T>::to_f(alt[(int64_t)(r - alt_begin) * d + i]);
    } else {
      val = x[(int64_t)r * d + i];
      if (n_parts > 0) {
        float f = parts[(int64_t)r * d + i];
        for (int s = 1; s < n_parts; ++s) f = f + parts[((int64_t)s * M + r) * d + i];
        val = val + f;
        if (write_back) x[(int64_t)r * d + i] = val;
      }
    }
    v[c] = val;
    ss = fmaf(val, val, ss);
  }
  ss = block_sum(ss, sh);
  const float rinv = 1.0f / sqrtf(ss / (float)d + eps);
  c = 0;
  for (int i = threadIdx.x; i < d; i += 256, ++c) out[(int64_t)r * ldo + i] = ET<T>::from_f((v[c] * rinv) * gamma[i]);
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

__global__ __launch_bounds__(256) void argmax_kernel(const float* __restrict__ logits, int V, int* __restrict__ amax) {
  __shared__ float shv[4];
  __shared__ int shi[4];
  const int r = blockIdx.x;
  const float* z = logits + (int64_t)r * V;
  float bv = -CH_INF;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < V; i += 256) {
    float v = z[i];
    v = (v != v) ? -CH_INF : v;
    if (better(v, i, bv, bi)) {
      bv = v;
      bi = i;
    }
  }
  block_best(bv, bi, shv, shi);
  if (threadIdx.x == 0) amax[r] = bi < V ? bi : 0;
}

// Top-s of draft head `level` for every sequence, with the forced-acceptance
// rule; the rank-0 entry becomes the chain token at position n + 1 + level.
__global__ __launch_bounds__(256) void topk_kernel(const float* __restrict__ logits, StepState s, int level) {
  __shared__ float shv[4];
  __shared__ int shi[4];
  __shared__ int chosen[8];
  const int b = blockIdx.x;
  const int K = s.K, V = s.V;
  const int S = s.s_k[level];
  const float* z = logits + ((int64_t)b * K + level) * V;
  const int n = s.n[b];
  const int j = n + 1 + level;
  int excl = -1, first = 0;
  if (s.f_ref != nullptr) {
    excl = s.f_ref[(int64_t)b * s.f_stride + j];
    if (excl < 0 || excl >= V) excl = -1;  // no usable reference at this position
    if (excl >= 0 && s.f_ok[(int64_t)b * s.f_stride + j]) {
      if (threadIdx.x == 0) chosen[0] = excl;
      first = 1;
    }
  }
  for (int r = first; r < S; ++r) {
    __syncthreads();
    float bv = -CH_INF;
    int bi = 0x7fffffff;
    for (int i = threadIdx.x; i < V; i += 256) {
      bool skip = i == excl;
      for (int q = 0; q < r; ++q) skip |= (chosen[q] == i);
      if (skip) continue;
      float v = z[i];
      v = (v != v) ? -CH_INF : v;
      if (better(v, i, bv, bi)) {
        bv = v;
        bi = i;
      }
    }
    block_best(bv, bi, shv, shi);
    if (threadIdx.x == 0) chosen[r] = bi < V ? bi : 0;
  }
  __syncthreads();
  if (threadIdx.x < S) s.cand[((int64_t)b * K + level) * 8 + threadIdx.x] = chosen[threadIdx.x];
  if (threadIdx.x == 0) s.tok[(int64_t)b * s.tok_stride + j] = chosen[0];
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
    t = s.cand[((int64_t)b * s.K + dep - 1) * 8 + s.t_rank[u]];
  const int row = b * s.N + u;
  s.tree_tok[row] = t;
  const int slot = n + u;
  s.v_pos[row] = n + dep;
  s.v_qrow[row] = row;
  s.v_kvoff[row] =
      (int64_t)s.page_table[(int64_t)b * s.max_pages + slot / s.ps] * s.page_stride + (int64_t)(slot % s.ps) * s.hd;
}

// Greedy acceptance, one wave per sequence, lane = tree node.
__global__ void accept_kernel(StepState s) {
  const int b = blockIdx.x, u = threadIdx.x;
  const bool valid = u < s.N;
  const int row = b * s.N + (valid ? u : 0);
  const int a_u = s.amax[row];
  const int tok_u = s.tree_tok[row];
  const int par = valid ? s.t_parent[u] : -1;
  const int a_par = par >= 0 ? s.amax[b * s.N + par] : -1;
  const bool good = valid && (u == 0 || tok_u == a_par);
  const unsigned long long goodmask = __ballot(good);
  const unsigned long long anc = valid ? s.t_anc[u] : 0ull;
  const bool acc = valid && ((anc & ~goodmask) == 0ull);
  int key = acc ? s.t_depth[u] : -1;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) key = max(key, __shfl_xor(key, m));
  const unsigned long long vmask = __ballot(acc && s.t_depth[valid ? u : 0] == key);
  const int v = __ffsll((long long)vmask) - 1;
  const unsigned long long path = __shfl(anc, v);
  const int L = __popcll(path);
  const int bonus = __shfl(a_u, v);
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

template <typename T>
__global__ __launch_bounds__(256) void advance_kernel(StepState s) {
  const int b = blockIdx.x;
  const int L = s.out_len[b];
  const int n = s.n[b];
  const int K1 = s.K + 1;
  const int d = s.d;
  if (threadIdx.x < L) s.tok[(int64_t)b * s.tok_stride + n + 1 + threadIdx.x] = s.out_tok[b * K1 + threadIdx.x];
  const T* hl = (const T*)s.hl;
  T* proh = (T*)s.pro_h;
  for (int idx = 0; idx < L; ++idx) {
    const int node = s.out_nodes[b * K1 + idx];
    const T* src = hl + (int64_t)(b * s.N + node) * d;
    T* dst = proh + ((int64_t)b * K1 + idx) * d;
    for (int i = threadIdx.x; i < d; i += 256) dst[i] = src[i];
    if (idx == L - 1)
      for (int i = threadIdx.x; i < d; i += 256) ((T*)s.h_last)[(int64_t)b * d + i] = src[i];
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    s.pro_base[b] = n;
    s.pro_count[b] = L;
    s.n[b] = n + L;
  }
}

template <typename T>
__device__ __forceinline__ void trigram_row(const StepState& s, const T* E, int b, int pos, T* dst) {
  const int d = s.d;
  for (int i = threadIdx.x; i < 3 * d; i += blockDim.x) {
    const int part = i / d, col = i % d;
    const int p = pos - 2 + part;
    T v = ET<T>::from_f(0.f);
    if (p >= 0) v = E[(int64_t)s.tok[(int64_t)b * s.tok_stride + p] * d + col];
    dst[i] = v;
  }
}

__device__ __forceinline__ int64_t enc_off(const StepState& s, int b, int stream, int pos) {
  return ((((int64_t)b * 2 + stream) * s.H) * s.cap + pos) * s.hd;
}

template <typename T>
__global__ void draft_rows_kernel(StepState s, const T* E, int level, T* tri_in, int* pos, int64_t* kvoff,
                                  int* qrow) {
  const int r = blockIdx.x;
  const int B = s.B, K1 = s.K + 1;
  int b, p, stream, q = -1;
  bool valid = true, want_tri = true;
  if (r < B) {
    b = r;
    p = s.n[b] + level;
    stream = 1;
    q = b;
  } else if (r < B + B * K1) {
    const int i = r - B;
    b = i / K1;
    const int e = i % K1;
    valid = e < s.pro_count[b];
    p = s.pro_base[b] + e;
    stream = 0;
    want_tri = false;
  } else {
    const int i = r - B - B * K1;
    b = i / K1;
    const int e = i % K1;
    valid = e < s.pro_count[b];
    p = s.pro_base[b] + e;
    stream = 1;
  }
  if (threadIdx.x == 0) {
    pos[r] = valid ? p : 0;
    kvoff[r] = valid ? enc_off(s, b, stream, p) : -1;
    qrow[r] = q;
  }
  T* dst = tri_in + (int64_t)r * 3 * s.d;
  if (want_tri && valid) {
    trigram_row<T>(s, E, b, p, dst);
  } else {
    for (int i = threadIdx.x; i < 3 * s.d; i += blockDim.x) dst[i] = ET<T>::from_f(0.f);
  }
}

template <typename T>
__global__ __launch_bounds__(256) void draft_finish_kernel(StepState s, const float* x, const float* parts,
                                                           int n_parts, T* zin) {
  const int b = blockIdx.x, d = s.d;
  const T* hl = (const T*)s.h_last + (int64_t)b * d;
  T* z = zin + (int64_t)b * 2 * d;
  for (int i = threadIdx.x; i < d; i += 256) {
    z[i] = hl[i];
    float f = parts[(int64_t)b * d + i];
    for (int q = 1; q < n_parts; ++q) f = f + parts[((int64_t)q * s.B + b) * d + i];
    z[d + i] = ET<T>::from_f(x[(int64_t)b * d + i] + f);
  }
}

template <typename T>
__global__ void prefill_rows_kernel(StepState s, const T* E, int b, int p0, int M, int* tokens_out, T* tri_in,
                                    int* enc_pos, int64_t* enc_kvoff, int* enc_qrow, int* pf_n) {
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
  trigram_row<T>(s, E, b, p, tri_in + (int64_t)i * 3 * s.d);
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

void launch_rmsnorm(int dtype, float* x, const float* parts, int n_parts, const float* gamma, void* out, int ldo, int M,
                    int d, float eps, int write_back, const void* alt, int alt_begin, int alt_end, hipStream_t st) {
  if (M <= 0) return;
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16_t>, dim3(M), dim3(256), 0, st, x, parts, n_parts, gamma, (bf16_t*)out, ldo,
                       M, d, eps, write_back, (const bf16_t*)alt, alt_begin, alt_end);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(M), dim3(256), 0, st, x, parts, n_parts, gamma, (float*)out, ldo, M,
                       d, eps, write_back, (const float*)alt, alt_begin, alt_end);
}

void launch_argmax(const float* logits, int M, int V, int* amax, hipStream_t st) {
  hipLaunchKernelGGL(argmax_kernel, dim3(M), dim3(256), 0, st, logits, V, amax);
}

void launch_topk(const float* logits, const StepState& s, int level, hipStream_t st) {
  hipLaunchKernelGGL(topk_kernel, dim3(s.B), dim3(256), 0, st, logits, s, level);
}

void launch_tree_setup(const StepState& s, hipStream_t st) {
  hipLaunchKernelGGL(tree_setup_kernel, dim3(s.B), dim3(64), 0, st, s);
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

void launch_advance(int dtype, const StepState& s, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(advance_kernel<bf16_t>, dim3(s.B), dim3(256), 0, st, s);
  else
    hipLaunchKernelGGL(advance_kernel<float>, dim3(s.B), dim3(256), 0, st, s);
}

void launch_draft_rows(int dtype, const StepState& s, const void* E, int level, void* tri_in, int* pos,
                       int64_t* kvoff, int* qrow, hipStream_t st) {
  const int rows = level == 0 ? s.B * (2 * (s.K + 1) + 1) : s.B;
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(draft_rows_kernel<bf16_t>, dim3(rows), dim3(256), 0, st, s, (const bf16_t*)E, level,
                       (bf16_t*)tri_in, pos, kvoff, qrow);
  else
    hipLaunchKernelGGL(draft_rows_kernel<float>, dim3(rows), dim3(256), 0, st, s, (const float*)E, level,
                       (float*)tri_in, pos, kvoff, qrow);
}

void launch_draft_finish(int dtype, const StepState& s, const float* x, const float* parts, int n_parts, void* zin,
                         hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(draft_finish_kernel<bf16_t>, dim3(s.B), dim3(256), 0, st, s, x, parts, n_parts, (bf16_t*)zin);
  else
    hipLaunchKernelGGL(draft_finish_kernel<float>, dim3(s.B), dim3(256), 0, st, s, x, parts, n_parts, (float*)zin);
}

void launch_prefill_rows(int dtype, const StepState& s, const void* E, int b, int p0, int M, int* tokens_out,
                         void* tri_in, int* enc_pos, int64_t* enc_kvoff, int* enc_qrow, int* pf_n, hipStream_t st) {
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(prefill_rows_kernel<bf16_t>, dim3(M), dim3(256), 0, st, s, (const bf16_t*)E, b, p0, M,
                       tokens_out, (bf16_t*)tri_in, enc_pos, enc_kvoff, enc_qrow, pf_n);
  else
    hipLaunchKernelGGL(prefill_rows_kernel<float>, dim3(M), dim3(256), 0, st, s, (const float*)E, b, p0, M, tokens_out,
                       (float*)tri_in, enc_pos, enc_kvoff, enc_qrow, pf_n);
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
