// Skinny GEMMs on MFMA for the decode step: Y = X[M][K] @ W[K][N] with M the
// number of tree nodes (or draft rows) and W streamed from HBM exactly once.
//
// Both operands are stored in MFMA fragment order, so every operand load of
// a wave is one contiguous 1 KiB (64 lanes x 16 bytes):
//   * W (repacked at load): workgroup column group g (4 blocks of 16
//     columns) stores its tiles as [g][kb][4][1 KiB];
//   * X (written tiled by the kernel that produces it): tile (kb, mb) of
//     16 rows x KB reduction indices at ((kb * mtiles + mb) * 64 + lane).
// A workgroup = 4 wave64s owns CB column blocks (64 columns; 32 for
// single-tile launches) and one slice of the reduction (split-K across
// workgroups); its waves take interleaved k-blocks and are summed through
// LDS in wave order.  Split-K slices are written as partials and summed in
// slice order by their consumer (the next norm) or by a finishing pass that
// applies the epilogue.  Every row's arithmetic depends only on (N, K): the
// same row gives identical bits whether a launch carries 1 or 64 rows.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int NB = 4;  // 16-column blocks per weight-layout group
constexpr int PF = 2;  // k-blocks in flight per wave
// Matrices at least this wide run unsplit (their epilogue needs whole sums and
// they already have >= 128 column groups); narrower ones split the reduction
// until a launch has at least SPLIT_TARGET_WGS workgroups.
constexpr int SPLIT_MIN_COLS_NO = 8192;
constexpr int SPLIT_TARGET_WGS = 256;

// ---------------------------------------------------------------------------
// Weight repacking (load time)
// ---------------------------------------------------------------------------
template <typename T>
__global__ void repack_kernel(const T* __restrict__ s0, const T* __restrict__ s1, const T* __restrict__ s2, int K,
                              int n_src, int kind, int H, int hd, T* __restrict__ dst, int nblocks) {
  constexpr int VEC = ET<T>::VEC, KB = 4 * VEC;
  const int kblocks = K / KB;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)nblocks * kblocks * 64;
  if (tid >= total) return;
  const int lane = (int)(tid & 63);
  const int64_t tile = tid >> 6;
  const int kb = (int)(tile % kblocks);
  const int c = (int)(tile / kblocks);
  const int cl = lane & 15;
  const T* src = s0;
  int col;
  if (kind == PACK_QKV) {
    const int per_sec = H * hd / 16;
    const int sec = c / per_sec, within = c % per_sec;
    const int h = within / (hd / 16), blk = within % (hd / 16);
    const int dim = sec < 2 ? (blk & 1) * (hd / 2) + 16 * (blk >> 1) + cl : 16 * blk + cl;
    src = sec == 0 ? s0 : (sec == 1 ? s1 : s2);
    col = h * hd + dim;
  } else if (kind == PACK_GU) {
    src = (c & 1) ? s1 : s0;
    col = 16 * (c >> 1) + cl;
  } else {
    col = 16 * c + cl;
  }
  const int k0 = kb * KB + (lane >> 4) * VEC;
  T* d = dst + ((((int64_t)(c / NB) * kblocks + kb) * NB + c % NB) * 64 + lane) * VEC;
#pragma unroll
  for (int e = 0; e < VEC; ++e) d[e] = src[(int64_t)(k0 + e) * n_src + col];
}

// ---------------------------------------------------------------------------
// Epilogue on one column pair: (v0, v1) are the values of packed column
// blocks 2*pair and 2*pair+1 at column offset c16 of row `row`.
// ---------------------------------------------------------------------------
template <typename T, int EPI>
__device__ __forceinline__ void epi_pair(const GemmEpi& e, int N, int M, int split, int row, int pair, int c16,
                                         float v0, float v1) {
  if constexpr (EPI == EPI_PARTIAL) {
    float* p = e.part + ((int64_t)split * M + row) * N + 32 * pair + c16;
    p[0] = v0;
    p[16] = v1;
  } else if constexpr (EPI == EPI_F32) {
    float* p = e.out_f + (int64_t)row * e.ldo + 32 * pair + c16;
    p[0] = v0;
    p[16] = v1;
  } else if constexpr (EPI == EPI_T) {
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, 32 * pair + c16, v0);
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, 32 * pair + 16 + c16, v1);
  } else if constexpr (EPI == EPI_SILU) {
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, 32 * pair + c16, silu_f(v0));
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, 32 * pair + 16 + c16, silu_f(v1));
  } else if constexpr (EPI == EPI_SWIGLU) {
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, 16 * pair + c16, silu_f(v0) * v1);
  } else if constexpr (EPI == EPI_QKV) {
    const int hd = e.hd;
    const int pairs_head = hd / 32;
    const int sec_pairs = e.H * pairs_head;
    const int sec = pair / sec_pairs, rem = pair % sec_pairs;
    const int h = rem / pairs_head, pp = rem % pairs_head;
    if (sec < 2) {
      const int i = 16 * pp + c16;
      const int pos = e.pos[row];
      const float c = e.rcos[(int64_t)pos * (hd / 2) + i];
      const float s = e.rsin[(int64_t)pos * (hd / 2) + i];
      const float o0 = v0 * c - v1 * s;
      const float o1 = v1 * c + v0 * s;
      if (sec == 0) {
        const int qr = e.qrow[row];
        if (qr >= 0) {
          T* q = (T*)e.qout + (int64_t)qr * e.ldq + h * hd;
          q[i] = ET<T>::from_f(o0);
          q[i + hd / 2] = ET<T>::from_f(o1);
        }
      } else {
        const int64_t off = e.kvoff[row];
        if (off >= 0) {
          T* k = (T*)e.kbase + off + h * e.head_stride;
          k[i] = ET<T>::from_f(o0);
          k[i + hd / 2] = ET<T>::from_f(o1);
        }
      }
    } else {
      const int64_t off = e.kvoff[row];
      if (off >= 0) {
        T* v = (T*)e.vbase + off + h * e.head_stride;
        v[32 * pp + c16] = ET<T>::from_f(v0);
        v[32 * pp + 16 + c16] = ET<T>::from_f(v1);
      }
    }
  }
}

template <typename T>
__device__ __forceinline__ int4 ldw(const T* p) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  const i32x4 v = __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(p));
  return int4{v.x, v.y, v.z, v.w};
}

// ---------------------------------------------------------------------------
// The GEMM.  grid = (column groups of 16*CB, row blocks of 16*MB, splits).
// ---------------------------------------------------------------------------
template <typename T, int MB, int CB, int EPI>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmShape sh, const GemmEpi e) {
  constexpr int VEC = ET<T>::VEC, KB = 4 * VEC;
  __shared__ f32x4 red[4][MB][CB][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4, c16 = lane & 15;
  const int kblocks = sh.K / KB;
  const int cb0 = sh.nb_off + blockIdx.x * CB;      // first 16-column block
  const int grp = cb0 / NB, sub = cb0 % NB;          // layout group, offset inside it
  const int mb0 = blockIdx.y * MB;
  const int kps = kblocks / sh.splits;
  const int kbeg = blockIdx.z * kps;
  const int kend = kbeg + kps;
  const T* X = (const T*)sh.X + (int64_t)lane * VEC;
  const T* W = (const T*)sh.W + (((int64_t)grp * kblocks * NB + sub) * 64 + lane) * VEC;

  f32x4 acc[MB][CB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  int4 bw[PF][CB], bx[PF][MB];
  auto load = [&](int s, int kb) {
#pragma unroll
    for (int j = 0; j < CB; ++j) bw[s][j] = ldw(W + ((int64_t)kb * NB + j) * 64 * VEC);
#pragma unroll
    for (int i = 0; i < MB; ++i) bx[s][i] = ld16(X + ((int64_t)kb * sh.x_mtiles + mb0 + i) * 64 * VEC);
  };
  const int kfirst = kbeg + wave;
#pragma unroll
  for (int s = 0; s < PF; ++s)
    if (kfirst + 4 * s < kend) load(s, kfirst + 4 * s);
  for (int it = 0;; it += PF) {
    bool done = false;
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      const int kb = kfirst + 4 * (it + s);
      if (kb >= kend) {
        done = true;
        break;
      }
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < CB; ++j) acc[i][j] = mfma_kb<T>(bx[s][i], bw[s][j], acc[i][j]);
      const int kn = kb + 4 * PF;
      if (kn < kend) load(s, kn);
    }
    if (done) break;
  }

#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) red[wave][i][j][lane] = acc[i][j];
  __syncthreads();
  constexpr int ITEMS = MB * (CB / 2);
  for (int it = wave; it < ITEMS; it += 4) {
    const int i = it / (CB / 2), jp = it % (CB / 2);
    f32x4 v0 = red[0][i][2 * jp][lane];
    f32x4 v1 = red[0][i][2 * jp + 1][lane];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      v0 = v0 + red[w][i][2 * jp][lane];
      v1 = v1 + red[w][i][2 * jp + 1][lane];
    }
    const int pair = cb0 / 2 + jp;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * (mb0 + i) + 4 * g + r;
      if (row < sh.M) epi_pair<T, EPI>(e, sh.N, sh.M, blockIdx.z, row, pair, c16, v0[r], v1[r]);
    }
  }
}

// Sum split-K partials in split order and apply the epilogue.
template <typename T, int EPI>
__global__ void gemm_finish_kernel(const GemmShape sh, const GemmEpi e, const float* __restrict__ part) {
  const int npairs = (sh.nb_count ? sh.nb_count : sh.N / 16) / 2;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)sh.M * npairs * 16;
  if (tid >= total) return;
  const int c16 = (int)(tid & 15);
  const int pr = (int)((tid >> 4) % npairs);
  const int row = (int)((tid >> 4) / npairs);
  const int pair = (sh.nb_off >> 1) + pr;
  float v0 = 0.f, v1 = 0.f;
  for (int s = 0; s < sh.splits; ++s) {
    const float* p = part + ((int64_t)s * sh.M + row) * sh.N + 32 * pair + c16;
    v0 = (s == 0) ? p[0] : v0 + p[0];
    v1 = (s == 0) ? p[16] : v1 + p[16];
  }
  epi_pair<T, EPI>(e, sh.N, sh.M, 0, row, pair, c16, v0, v1);
}

template <typename T, int MB, int EPI>
void gemm_go(const GemmShape& s, const GemmEpi& e, hipStream_t st) {
  constexpr int CB = MB == 1 ? 2 : 4;
  const int nbc = s.nb_count ? s.nb_count : s.N / 16;
  dim3 grid(nbc / CB, (s.M + 16 * MB - 1) / (16 * MB), s.splits);
  if (s.splits == 1 || EPI == EPI_PARTIAL) {
    hipLaunchKernelGGL((gemm_kernel<T, MB, CB, EPI>), grid, dim3(256), 0, st, s, e);
  } else {
    GemmEpi pe = e;  // e.part is the partial scratch
    hipLaunchKernelGGL((gemm_kernel<T, MB, CB, EPI_PARTIAL>), grid, dim3(256), 0, st, s, pe);
    const int64_t total = (int64_t)s.M * (nbc / 2) * 16;
    hipLaunchKernelGGL((gemm_finish_kernel<T, EPI>), dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, s, e,
                       (const float*)e.part);
  }
}

template <typename T, int MB>
void gemm_epi(const GemmShape& s, const GemmEpi& e, hipStream_t st) {
  switch (e.kind) {
    case EPI_F32: gemm_go<T, MB, EPI_F32>(s, e, st); break;
    case EPI_T: gemm_go<T, MB, EPI_T>(s, e, st); break;
    case EPI_SILU: gemm_go<T, MB, EPI_SILU>(s, e, st); break;
    case EPI_SWIGLU: gemm_go<T, MB, EPI_SWIGLU>(s, e, st); break;
    case EPI_QKV: gemm_go<T, MB, EPI_QKV>(s, e, st); break;
    default: gemm_go<T, MB, EPI_PARTIAL>(s, e, st); break;
  }
}

template <typename T>
void gemm_t(const GemmShape& s, const GemmEpi& e, hipStream_t st) {
  if (s.M <= 16)
    gemm_epi<T, 1>(s, e, st);
  else if (s.M <= 32)
    gemm_epi<T, 2>(s, e, st);
  else
    gemm_epi<T, 4>(s, e, st);
}

template <typename T>
__global__ void tile_rows_kernel(const T* __restrict__ src, int M, int K, T* __restrict__ dst, int mtiles) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= (int64_t)M * K) return;
  const int r = (int)(tid / K), c = (int)(tid % K);
  copy_tiled<T>(dst, mtiles, r, c, src[tid]);
}

}  // namespace

void launch_tile_rows(int dtype, const void* src, int M, int K, void* dst, int mtiles, hipStream_t st) {
  const int64_t total = (int64_t)M * K;
  dim3 grid((unsigned)((total + 255) / 256));
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(tile_rows_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)src, M, K, (bf16_t*)dst, mtiles);
  else
    hipLaunchKernelGGL(tile_rows_kernel<float>, grid, dim3(256), 0, st, (const float*)src, M, K, (float*)dst, mtiles);
}

int gemm_pick_splits(int n_cols, int K, int dtype) {
  // Wide matrices have enough 64-column groups to fill the GPU on their own;
  // narrow ones split the reduction so that >= 256 workgroups stream weights.
  const int KB = dtype == DT_BF16 ? 32 : 16;
  const int kblocks = K / KB;
  if (n_cols >= SPLIT_MIN_COLS_NO) return 1;
  const int groups = n_cols / 64;
  int s = 1;
  while (groups * s < SPLIT_TARGET_WGS && s < 8 && kblocks % (2 * s) == 0 && kblocks / (2 * s) >= 16) s *= 2;
  return s;
}

void launch_gemm(int dtype, const GemmShape& s, const GemmEpi& e, hipStream_t st) {
  if (s.M <= 0) return;
  if (dtype == DT_BF16)
    gemm_t<bf16_t>(s, e, st);
  else
    gemm_t<float>(s, e, st);
}

void launch_repack(int dtype, int kind, const void* src0, const void* src1, const void* src2, int K, int n_src,
                   void* dst, int H, int hd, hipStream_t st) {
  const int n_packed = kind == PACK_QKV ? 3 * n_src : (kind == PACK_GU ? 2 * n_src : n_src);
  const int nblocks = n_packed / 16;
  const int KB = dtype == DT_BF16 ? 32 : 16;
  const int64_t total = (int64_t)nblocks * (K / KB) * 64;
  dim3 grid((unsigned)((total + 255) / 256));
  if (dtype == DT_BF16)
    hipLaunchKernelGGL(repack_kernel<bf16_t>, grid, dim3(256), 0, st, (const bf16_t*)src0, (const bf16_t*)src1,
                       (const bf16_t*)src2, K, n_src, kind, H, hd, (bf16_t*)dst, nblocks);
  else
    hipLaunchKernelGGL(repack_kernel<float>, grid, dim3(256), 0, st, (const float*)src0, (const float*)src1,
                       (const float*)src2, K, n_src, kind, H, hd, (float*)dst, nblocks);
}
