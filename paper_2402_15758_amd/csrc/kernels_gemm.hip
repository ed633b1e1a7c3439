// Skinny GEMMs on MFMA for the decode step: Y = X[M][K] @ W[K][N] with M the
// number of tree nodes (or draft rows) and W streamed from HBM exactly once.
//
// Both operands are stored in MFMA fragment order, so every operand load of
// a wave is one contiguous 1 KiB (64 lanes x 16 bytes):
//   * W (repacked at load): layout group g of 4 column blocks stores its
//     tiles as [g][kb][4][1 KiB];
//   * X (written tiled by the kernel that produces it): tile (kb, mb) of
//     16 rows x KB reduction indices at ((kb * mtiles + mb) * 64 + lane).
//
// Work split.  A launch runs GEMM_WGS / splits workgroups per reduction slice
// (more only when a matrix has over CB_MAX column blocks per workgroup), and
// the 16-column blocks are dealt out in contiguous runs whose lengths differ
// by at most one, so every CU streams the same number of weight bytes and
// the activation tiles a workgroup reads are reused across its whole run.
// A workgroup = 4 wave64s; its waves take interleaved k-blocks and are summed
// through LDS in wave order.  The steady-state loop issues the loads of
// stage s + PF unconditionally, so the wait before stage s only covers that
// stage's own loads.  Split-K slices are written as partials and summed in
// slice order by their consumer (the next norm) or by a finishing pass that
// applies the epilogue.  Every row's arithmetic depends only on (N, K): the
// same row gives identical bits whether a launch carries 1 or 256 rows.
#include <hip/hip_ext.h>

#include <algorithm>

#include "common.h"
#include "kernels.h"

// The GEMM kernels take GemmShape and GemmEpi by value: a plain block of
// pointers and integers well inside the kernel-argument limit.
static_assert(sizeof(GemmShape) + sizeof(GemmEpi) + 4 * sizeof(int) <= 512, "GEMM kernel-argument block");
static_assert(alignof(GemmShape) <= 8 && alignof(GemmEpi) <= 8, "GEMM kernel-argument alignment");

namespace {

constexpr int NB = 4;        // 16-column blocks per weight-layout group
constexpr int CB_MAX = 8;    // column blocks per workgroup, upper bound
constexpr int RED_TILES = 32;  // 16x16 output tiles per wave in one LDS reduction round (4 x 32 KiB)
constexpr int GEMM_WGS = 256;  // one workgroup per CU per reduction slice
constexpr int GEMM_XCDS = 8;   // accelerator dies; workgroups are dealt to them round-robin
// Matrices at least this wide run unsplit (their epilogue needs whole sums and
// they fill the GPU on their own); narrower ones split the reduction until a
// launch has at least SPLIT_TARGET_WGS 64-column groups' worth of work.
constexpr int SPLIT_MIN_COLS_NO = 8192;
constexpr int SPLIT_TARGET_WGS = 256;

// ---------------------------------------------------------------------------
// Weight repacking (load time).  Packed column block c, lane column cl:
//   PACK_NATURAL: column 16 c + cl.
//   PACK_QKV: sections Q, K, V of H * hd / 16 blocks each; block q of head h
//     holds, for Q and K, rotary dims 8q + cl (cl < 8) and hd/2 + 8q + cl - 8
//     (cl >= 8), so both halves of a rotary pair sit in lanes cl and cl ^ 8;
//     V keeps dims 16q + cl.
//   PACK_GU: gate column 8c + cl (cl < 8) and up column 8c + cl - 8 (cl >= 8).
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
    const int h = within / (hd / 16), q = within % (hd / 16);
    const int dim = sec < 2 ? (cl < 8 ? 8 * q + cl : hd / 2 + 8 * q + cl - 8) : 16 * q + cl;
    src = sec == 0 ? s0 : (sec == 1 ? s1 : s2);
    col = h * hd + dim;
  } else if (kind == PACK_GU) {
    src = cl < 8 ? s0 : s1;
    col = 8 * c + (cl & 7);
  } else {
    col = 16 * c + cl;
  }
  const int k0 = kb * KB + (lane >> 4) * VEC;
  T* d = dst + ((((int64_t)(c / NB) * kblocks + kb) * NB + c % NB) * 64 + lane) * VEC;
#pragma unroll
  for (int e = 0; e < VEC; ++e) d[e] = src[(int64_t)(k0 + e) * n_src + col];
}

// ---------------------------------------------------------------------------
// Epilogue of one output element: v is packed column 16 blk + c16 of `row`,
// vp the same row's value at lane column c16 ^ 8 (the other half of a rotary
// or gate/up pair).
// ---------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ void epi_elem(const GemmEpi& e, int kind, int N, int M, int split, int row, int blk,
                                         int c16, float v, float vp) {
  const int col = 16 * blk + c16;
  if (kind == EPI_PARTIAL) {
    e.part[((int64_t)split * M + row) * N + col] = v;
  } else if (kind == EPI_F32) {
    e.out_f[(int64_t)row * e.ldo + col] = v;
  } else if (kind == EPI_T) {
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, col, v);
  } else if (kind == EPI_SILU) {
    store_tiled<T>((T*)e.out_t, e.o_mtiles, row, col, silu_f(v));
  } else if (kind == EPI_SWIGLU) {
    if (c16 < 8) store_tiled<T>((T*)e.out_t, e.o_mtiles, row, 8 * blk + c16, silu_f(v) * vp);
  } else if (kind == EPI_QKV) {
    const int hd = e.hd;
    const int blk_head = hd / 16;
    const int sec_blks = e.H * blk_head;
    const int sec = blk / sec_blks, rem = blk % sec_blks;
    const int h = rem / blk_head, q = rem % blk_head;
    if (sec < 2) {
      const bool first = c16 < 8;
      const int i = 8 * q + (c16 & 7);
      const int pos = e.pos[row];
      const float c = e.rcos[(int64_t)pos * (hd / 2) + i];
      const float s = e.rsin[(int64_t)pos * (hd / 2) + i];
      // first half: x1 cos - x2 sin; second half: x2 cos + x1 sin
      const float o = first ? v * c - vp * s : v * c + vp * s;
      const int dim = first ? i : i + hd / 2;
      if (sec == 0) {
        const int qr = e.qrow[row];
        if (qr >= 0) ((T*)e.qout)[(int64_t)qr * e.ldq + h * hd + dim] = ET<T>::from_f(o);
      } else {
        const int64_t off = e.kvoff[row];
        if (off >= 0) ((T*)e.kbase)[off + h * e.head_stride + dim] = ET<T>::from_f(o);
      }
    } else {
      const int64_t off = e.kvoff[row];
      if (off >= 0) ((T*)e.vbase)[off + h * e.head_stride + 16 * q + c16] = ET<T>::from_f(v);
    }
  }
}

// Per-row targets of the QKV epilogue, staged in LDS before the k-loop.
struct RowMeta {
  int64_t kvoff;  // K/V element offset (-1: skip)
  int pos;        // rotary position
  int qrow;       // Q output row (-1: skip)
};

// QKV epilogue of one element with its rotary cos/sin already loaded (the
// same arithmetic as epi_elem's EPI_QKV branch).
template <typename T>
__device__ __forceinline__ void qkv_store(const GemmEpi& e, const RowMeta& rm, int blk, int c16, float v, float vp,
                                          float c, float s) {
  const int hd = e.hd;
  const int blk_head = hd / 16;
  const int sec_blks = e.H * blk_head;
  const int sec = blk / sec_blks, rem = blk % sec_blks;
  const int h = rem / blk_head, q = rem % blk_head;
  if (sec < 2) {
    const bool first = c16 < 8;
    const int i = 8 * q + (c16 & 7);
    const float o = first ? v * c - vp * s : v * c + vp * s;
    const int dim = first ? i : i + hd / 2;
    if (sec == 0) {
      if (rm.qrow >= 0) ((T*)e.qout)[(int64_t)rm.qrow * e.ldq + h * hd + dim] = ET<T>::from_f(o);
    } else if (rm.kvoff >= 0) {
      ((T*)e.kbase)[rm.kvoff + h * e.head_stride + dim] = ET<T>::from_f(o);
    }
  } else if (rm.kvoff >= 0) {
    ((T*)e.vbase)[rm.kvoff + h * e.head_stride + 16 * q + c16] = ET<T>::from_f(v);
  }
}

// The same element's value before the store: rotated Q/K or plain V.
__device__ __forceinline__ float qkv_value(const GemmEpi& e, int blk, int c16, float v, float vp, float c, float s) {
  const int sec = blk / (e.H * (e.hd / 16));
  if (sec == 2) return v;
  return c16 < 8 ? v * c - vp * s : v * c + vp * s;
}

// 8 consecutive outputs of one row of a QKV tile as one 16-byte store: half 0
// holds lane columns 0..7 of block blk, half 1 columns 8..15.
template <typename T>
__device__ __forceinline__ void qkv_store16(const GemmEpi& e, const RowMeta& rm, int blk, int half, int4 v) {
  const int hd = e.hd;
  const int blk_head = hd / 16;
  const int sec_blks = e.H * blk_head;
  const int sec = blk / sec_blks, rem = blk % sec_blks;
  const int h = rem / blk_head, q = rem % blk_head;
  const int dim = sec < 2 ? (half ? hd / 2 : 0) + 8 * q : 16 * q + 8 * half;
  if (sec == 0) {
    if (rm.qrow >= 0) *reinterpret_cast<int4*>((T*)e.qout + (int64_t)rm.qrow * e.ldq + h * hd + dim) = v;
  } else if (rm.kvoff >= 0) {
    T* base = (T*)(sec == 1 ? e.kbase : e.vbase);
    *reinterpret_cast<int4*>(base + rm.kvoff + h * e.head_stride + dim) = v;
  }
}

template <typename T>
__device__ __forceinline__ int4 ldw(const T* p) {
  typedef int i32x4 __attribute__((ext_vector_type(4)));
  const i32x4 v = __builtin_nontemporal_load(reinterpret_cast<const i32x4*>(p));
  return int4{v.x, v.y, v.z, v.w};
}

// One workgroup's run of CB column blocks starting at block cb0, rows
// [16 mb0, 16 (mb0 + MB)), reduction slice [kbeg, kend).  red: LDS of
// [4][MB][CB][64] f32x4.
// Epilogue of gemm_run for column blocks [J0, J0 + JN) of the run: the waves'
// partial sums are added in wave order through LDS, then stored.
template <typename T, int MB, int CB, int J0, int JN>
__device__ __forceinline__ void gemm_epilogue(const GemmShape& sh, const GemmEpi& e, int kind, int cb0, int mb0,
                                              const f32x4 (&acc)[MB][CB], f32x4* red, const RowMeta* rm,
                                              float* stage, int wave, int lane, int split) {
  const int g = lane >> 4, c16 = lane & 15;
  // this wave's output tiles: items it = wave, wave + 4, ... of MB * JN
  constexpr int ITEMS = (MB * JN + 3) / 4;
  // QKV: the rotary table entries of every element are requested first, so
  // that their round trip overlaps the reduction below
  float cs[ITEMS][4], sn[ITEMS][4];
  if (kind == EPI_QKV) {
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
      const int it = wave + 4 * k;
      const int i = it / JN, j = J0 + it % JN;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        cs[k][r] = 1.f;
        sn[k][r] = 0.f;
        const int lr = 16 * i + 4 * g + r;
        const int row = 16 * mb0 + lr;
        const int q = (cb0 + j) % (e.hd / 16);
        const bool rot = (cb0 + j) < 2 * e.H * (e.hd / 16);
        if (it < MB * JN && row < sh.M && rot) {
          const int64_t ti = (int64_t)rm[lr].pos * (e.hd / 2) + 8 * q + (c16 & 7);
          cs[k][r] = e.rcos[ti];
          sn[k][r] = e.rsin[ti];
        }
      }
    }
  }
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int jj = 0; jj < JN; ++jj) red[((wave * MB + i) * JN + jj) * 64 + lane] = acc[i][J0 + jj];
  __syncthreads();
  f32x4 vv[ITEMS], vpp[ITEMS];
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const int it = wave + 4 * k;
    if (it < MB * JN) {  // wave-uniform
      const int i = it / JN, j = it % JN;
      f32x4 v = red[((0 * MB + i) * JN + j) * 64 + lane];
#pragma unroll
      for (int w = 1; w < 4; ++w) v = v + red[((w * MB + i) * JN + j) * 64 + lane];
      vv[k] = v;
#pragma unroll
      for (int r = 0; r < 4; ++r) vpp[k][r] = dpp_mov<DPP_ROR8>(v[r]);  // lane column c16 ^ 8
    }
  }
  if (kind == EPI_QKV) {
    if constexpr (sizeof(T) == 2) {
      // each 16x16 tile goes through the wave's LDS tile, then 32 lanes store
      // 8 consecutive outputs of one row each
      T* tw = reinterpret_cast<T*>(stage + wave * 256);
#pragma unroll
      for (int k = 0; k < ITEMS; ++k) {
        const int it = wave + 4 * k;
        if (it >= MB * JN) break;  // wave-uniform
        const int i = it / JN, blk = cb0 + J0 + it % JN;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          tw[(4 * g + r) * 16 + c16] = ET<T>::from_f(qkv_value(e, blk, c16, vv[k][r], vpp[k][r], cs[k][r], sn[k][r]));
        __builtin_amdgcn_wave_barrier();
        if (lane < 32) {
          const int lr = 16 * i + (lane & 15);
          const int4 v = *reinterpret_cast<const int4*>(tw + (lane & 15) * 16 + 8 * (lane >> 4));
          if (16 * mb0 + lr < sh.M) qkv_store16<T>(e, rm[lr], blk, lane >> 4, v);
        }
        __builtin_amdgcn_wave_barrier();
      }
      return;
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
      const int it = wave + 4 * k;
      const int i = it / JN, j = J0 + it % JN;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int lr = 16 * i + 4 * g + r;
        const int row = 16 * mb0 + lr;
        if (it < MB * JN && row < sh.M) qkv_store<T>(e, rm[lr], cb0 + j, c16, vv[k][r], vpp[k][r], cs[k][r], sn[k][r]);
      }
    }
    return;
  }
  if (kind == EPI_F32 || kind == EPI_PARTIAL) {
    // float outputs: the tile goes through the wave's LDS tile, then each lane
    // stores 4 consecutive columns of one row (16 rows x 64 bytes)
    float* tw = stage + wave * 256;
    float* base;
    int64_t ld;
    if (kind == EPI_F32) {
      base = e.out_f;
      ld = e.ldo;
    } else {
      base = e.part + (int64_t)split * sh.M * sh.N;
      ld = sh.N;
    }
#pragma unroll
    for (int k = 0; k < ITEMS; ++k) {
      const int it = wave + 4 * k;
      if (it >= MB * JN) break;  // wave-uniform
      const int i = it / JN, blk = cb0 + J0 + it % JN;
#pragma unroll
      for (int r = 0; r < 4; ++r) tw[(4 * g + r) * 16 + c16] = vv[k][r];
      __builtin_amdgcn_wave_barrier();
      const int row = 16 * (mb0 + i) + (lane >> 2);
      const float4 v = *reinterpret_cast<const float4*>(tw + (lane >> 2) * 16 + 4 * (lane & 3));
      if (row < sh.M) *reinterpret_cast<float4*>(base + (int64_t)row * ld + 16 * blk + 4 * (lane & 3)) = v;
      __builtin_amdgcn_wave_barrier();
    }
    return;
  }
  if constexpr (sizeof(T) == 2) {
    if (kind == EPI_SWIGLU) {
      // the 16 x 8 outputs of a tile (gate columns c16 < 8 times their up
      // partners) are 16 rows of 8 consecutive tiled elements: one 16-byte
      // store per row
      T* tw = reinterpret_cast<T*>(stage + wave * 256);
#pragma unroll
      for (int k = 0; k < ITEMS; ++k) {
        const int it = wave + 4 * k;
        if (it >= MB * JN) break;  // wave-uniform
        const int i = it / JN, blk = cb0 + J0 + it % JN;
        if (c16 < 8) {
#pragma unroll
          for (int r = 0; r < 4; ++r) tw[(4 * g + r) * 8 + c16] = ET<T>::from_f(silu_f(vv[k][r]) * vpp[k][r]);
        }
        __builtin_amdgcn_wave_barrier();
        if (lane < 16) {
          const int row = 16 * (mb0 + i) + lane;
          const int4 v = *reinterpret_cast<const int4*>(tw + lane * 8);
          if (row < sh.M) *reinterpret_cast<int4*>((T*)e.out_t + tiled_index<T>(e.o_mtiles, row, 8 * blk)) = v;
        }
        __builtin_amdgcn_wave_barrier();
      }
      return;
    }
  }
#pragma unroll
  for (int k = 0; k < ITEMS; ++k) {
    const int it = wave + 4 * k;
    const int i = it / JN, j = J0 + it % JN;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = 16 * (mb0 + i) + 4 * g + r;
      if (it < MB * JN && row < sh.M)
        epi_elem<T>(e, kind, sh.N, sh.M, split, row, cb0 + j, c16, vv[k][r], vpp[k][r]);
    }
  }
}

template <typename T, int MB, int CB, int PF>
__device__ __forceinline__ void gemm_run(const GemmShape& sh, const GemmEpi& e, int kind, int cb0, int mb0, int kbeg,
                                         int kend, f32x4* red, const RowMeta* rm, float* stage, int split) {
  constexpr int VEC = ET<T>::VEC;
  // The wave index is made provably wave-uniform so that every branch of the
  // k-loop below is a scalar branch: an MFMA ignores EXEC, so it must never
  // sit in a lane-predicated region.
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int kblocks = sh.K / (4 * VEC);
  const T* X = (const T*)sh.X + (int64_t)lane * VEC;
  const T* Wl = (const T*)sh.W + (int64_t)lane * VEC;
  int64_t wofs[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    const int c = cb0 + j;
    wofs[j] = ((int64_t)(c / NB) * kblocks * NB + c % NB) * 64 * VEC;
  }

  f32x4 acc[MB][CB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < CB; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  int4 bw[PF][CB], bx[PF][MB];
  auto load = [&](int s, int kb) {
#pragma unroll
    for (int j = 0; j < CB; ++j) bw[s][j] = ldw(Wl + wofs[j] + (int64_t)kb * NB * 64 * VEC);
#pragma unroll
    for (int i = 0; i < MB; ++i) bx[s][i] = ld16(X + ((int64_t)kb * sh.x_mtiles + mb0 + i) * 64 * VEC);
  };
  auto mma = [&](int s) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int j = 0; j < CB; ++j) acc[i][j] = mfma_kb<T>(bx[s][i], bw[s][j], acc[i][j]);
  };
  // wave w takes k-blocks kbeg + w, kbeg + w + 4, ... (nk of them)
  const int kfirst = kbeg + wave;
  const int nk = kfirst < kend ? (kend - kfirst + 3) / 4 : 0;
  if (nk >= PF) {
#pragma unroll
    for (int s = 0; s < PF; ++s) load(s, kfirst + 4 * s);
    int it = 0;
    for (; it + 2 * PF <= nk; it += PF) {
#pragma unroll
      for (int s = 0; s < PF; ++s) {
        mma(s);
        load(s, kfirst + 4 * (it + PF + s));
      }
    }
    // stages it .. it+PF-1 are loaded; rem (< PF) k-blocks remain after them
    const int rem = nk - it - PF;
#pragma unroll
    for (int s = 0; s < PF; ++s) {
      mma(s);
      if (s < rem) load(s, kfirst + 4 * (it + PF + s));
    }
#pragma unroll
    for (int s = 0; s < PF - 1; ++s)
      if (s < rem) mma(s);
  } else {
    for (int t = 0; t < nk; ++t) {
      load(0, kfirst + 4 * t);
      mma(0);
    }
  }

  // the four waves' partial sums meet in LDS, JR column blocks at a time
  constexpr int JR = CB < RED_TILES / MB ? CB : RED_TILES / MB;
  gemm_epilogue<T, MB, CB, 0, JR>(sh, e, kind, cb0, mb0, acc, red, rm, stage, wave, lane, split);
  if constexpr (CB > JR) {
    __syncthreads();  // the first round's reads of red are done
    gemm_epilogue<T, MB, CB, JR, CB - JR>(sh, e, kind, cb0, mb0, acc, red, rm, stage, wave, lane, split);
  }
}

// Workgroup -> (row block, column run, split).  Workgroups are dealt to the
// 8 XCDs round-robin by linear id.  When a launch has several row blocks and
// its (run, split) count is a multiple of 8, consecutive workgroups of one
// XCD take the row blocks of one weight run, so every run's weight tiles are
// fetched from HBM once into that XCD's L2 and re-read from there; otherwise
// the linear order is used.  The mapping moves no arithmetic.
struct GemmTile {
  int rb, run, split;
};
// X, Y: grid.x and grid.y (X > 1 and grid.y * grid.z a multiple of 8).
__device__ __forceinline__ GemmTile gemm_tile_xcd(int X, int Y) {
  const int L = blockIdx.x + X * (blockIdx.y + Y * blockIdx.z);  // linear dispatch id
  const int xcd = L % GEMM_XCDS, k = L / GEMM_XCDS;
  const int r = (k / X) * GEMM_XCDS + xcd;
  return GemmTile{k % X, r % Y, r / Y};
}

// grid = (row blocks of 16 MB, workgroups per slice, splits).  Workgroups
// [0, nbig) own CBA column blocks, the others CBA - 1.
template <typename T, int MB, int CBA, bool XCD_MAP>
__global__ __launch_bounds__(256) void gemm_kernel(const GemmShape sh, const GemmEpi e, int kind, int nbig, int gx,
                                                   int gy) {
  constexpr int PF = MB == 1 ? 4 : (MB >= 8 ? 2 : 3);
  constexpr int JR = CBA < RED_TILES / MB ? CBA : RED_TILES / MB;
  if (sh.skip && *sh.skip == 0) return;
  __shared__ f32x4 red[4 * MB * JR * 64];
  const int kblocks = sh.K / (4 * ET<T>::VEC);
  const int kps = kblocks / sh.splits;
  const GemmTile tl = XCD_MAP ? gemm_tile_xcd(gx, gy) : GemmTile{(int)blockIdx.x, (int)blockIdx.y, (int)blockIdx.z};
  const int kbeg = tl.split * kps;
  const int kend = kbeg + kps;
  const int b = tl.run;
  const int mb0 = tl.rb * MB;
  // QKV epilogue targets of this workgroup's rows (visible after the k-loop's
  // barrier)
  __shared__ RowMeta rm[16 * MB];
  __shared__ __attribute__((aligned(16))) float stage[4 * 256];  // a 16x16 output tile per wave
  if (kind == EPI_QKV && threadIdx.x < 16 * MB) {
    const int row = 16 * mb0 + threadIdx.x;
    RowMeta t{-1, 0, -1};
    if (row < sh.M) t = RowMeta{e.kvoff[row], e.pos[row], e.qrow[row]};
    rm[threadIdx.x] = t;
  }
  if (b < nbig) {
    gemm_run<T, MB, CBA, PF>(sh, e, kind, sh.nb_off + b * CBA, mb0, kbeg, kend, red, rm, stage, tl.split);
  } else {
    if constexpr (CBA > 1)
      gemm_run<T, MB, CBA - 1, PF>(sh, e, kind, sh.nb_off + nbig * CBA + (b - nbig) * (CBA - 1), mb0, kbeg, kend,
                                   red, rm, stage, tl.split);
  }
}

// Sum split-K partials in split order and apply the epilogue (one thread
// per output element of the launch's column blocks).
template <typename T>
__global__ void gemm_finish_kernel(const GemmShape sh, const GemmEpi e, int kind, const float* __restrict__ part) {
  if (sh.skip && *sh.skip == 0) return;
  const int nbc = sh.nb_count ? sh.nb_count : sh.N / 16;
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)sh.M * nbc * 16;
  if (tid >= total) return;
  const int c16 = (int)(tid & 15);
  const int blk = sh.nb_off + (int)((tid >> 4) % nbc);
  const int row = (int)((tid >> 4) / nbc);
  // every slice is requested before the first is added
  float pv[GEMM_MAX_SPLITS], pp[GEMM_MAX_SPLITS];
#pragma unroll
  for (int s = 0; s < GEMM_MAX_SPLITS; ++s) {
    if (s < sh.splits) {
      const float* p = part + ((int64_t)s * sh.M + row) * sh.N + 16 * blk;
      pv[s] = p[c16];
      pp[s] = p[c16 ^ 8];
    }
  }
  float v = pv[0], vp = pp[0];
#pragma unroll
  for (int s = 1; s < GEMM_MAX_SPLITS; ++s) {
    if (s < sh.splits) {
      v = v + pv[s];
      vp = vp + pp[s];
    }
  }
  epi_elem<T>(e, kind, sh.N, sh.M, 0, row, blk, c16, v, vp);
}

template <typename T, int MB, int CBA>
void gemm_launch(const GemmShape& s, const GemmEpi& e, int kind, int nwg, int nbig, hipStream_t st, hipEvent_t ea,
                 hipEvent_t eb) {
  dim3 grid((s.M + 16 * MB - 1) / (16 * MB), nwg, s.splits);
  const int gx = (int)grid.x, gy = (int)grid.y;
  if (gx > 1 && (gy * s.splits) % GEMM_XCDS == 0) {
    if constexpr (MB > 1) {
      if (ea || eb)
        hipExtLaunchKernelGGL((gemm_kernel<T, MB, CBA, true>), grid, dim3(256), 0, st, ea, eb, 0, s, e, kind, nbig, gx,
                              gy);
      else
        hipLaunchKernelGGL((gemm_kernel<T, MB, CBA, true>), grid, dim3(256), 0, st, s, e, kind, nbig, gx, gy);
      return;
    }
  }
  if (ea || eb)
    hipExtLaunchKernelGGL((gemm_kernel<T, MB, CBA, false>), grid, dim3(256), 0, st, ea, eb, 0, s, e, kind, nbig, gx,
                          gy);
  else
    hipLaunchKernelGGL((gemm_kernel<T, MB, CBA, false>), grid, dim3(256), 0, st, s, e, kind, nbig, gx, gy);
}

template <typename T, int MB>
void gemm_mb(const GemmShape& s, const GemmEpi& e, int kind, int nwg, int cba, int nbig, hipStream_t st,
             hipEvent_t ea, hipEvent_t eb) {
  switch (cba) {
    case 1: gemm_launch<T, MB, 1>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 2: gemm_launch<T, MB, 2>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 3: gemm_launch<T, MB, 3>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 4: gemm_launch<T, MB, 4>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 5: gemm_launch<T, MB, 5>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 6: gemm_launch<T, MB, 6>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 7: gemm_launch<T, MB, 7>(s, e, kind, nwg, nbig, st, ea, eb); break;
    default: gemm_launch<T, MB, 8>(s, e, kind, nwg, nbig, st, ea, eb); break;
  }
}

// 128-row tiles; runs of up to 6 blocks fit the registers without spills.
constexpr int CB_MAX_MB8 = 6;
template <typename T>
void gemm_mb8(const GemmShape& s, const GemmEpi& e, int kind, int nwg, int cba, int nbig, hipStream_t st,
              hipEvent_t ea, hipEvent_t eb) {
  switch (cba) {
    case 1: gemm_launch<T, 8, 1>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 2: gemm_launch<T, 8, 2>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 3: gemm_launch<T, 8, 3>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 4: gemm_launch<T, 8, 4>(s, e, kind, nwg, nbig, st, ea, eb); break;
    case 5: gemm_launch<T, 8, 5>(s, e, kind, nwg, nbig, st, ea, eb); break;
    default: gemm_launch<T, 8, 6>(s, e, kind, nwg, nbig, st, ea, eb); break;
  }
}

template <typename T>
void gemm_t(const GemmShape& s, const GemmEpi& e, hipStream_t st, hipEvent_t ev_start, hipEvent_t ev_stop) {
  const int nbc = s.nb_count ? s.nb_count : s.N / 16;
  // workgroups per slice: GEMM_WGS / splits, at least ceil(nbc / CB_MAX),
  // at most one per column block; runs of cba or cba - 1 blocks
  int nwg = (GEMM_WGS + s.splits - 1) / s.splits;
  nwg = std::max(nwg, (nbc + CB_MAX - 1) / CB_MAX);
  nwg = std::min(nwg, nbc);
  const int cba = (nbc + nwg - 1) / nwg;
  const int nbig = nbc - nwg * (cba - 1);
  const bool finish = s.splits > 1 && e.kind != EPI_PARTIAL;
  const int kind = finish ? EPI_PARTIAL : e.kind;
  hipEvent_t eb = finish ? nullptr : ev_stop;
  // Rows per workgroup: every output element's arithmetic is the same for
  // any MB (the waves split the reduction, not the rows), so the choice only
  // trades weight re-reads against activation traffic.  Above 64 rows a
  // 128-row tile halves the weight re-reads when the buffer holds whole tiles.
  if (s.M <= 16)
    gemm_mb<T, 1>(s, e, kind, nwg, cba, nbig, st, ev_start, eb);
  else if (s.M <= 32)
    gemm_mb<T, 2>(s, e, kind, nwg, cba, nbig, st, ev_start, eb);
  else if (s.M > 64 && cba <= CB_MAX_MB8 && (s.M + 127) / 128 * 8 <= s.x_mtiles) {
    // A 128-row workgroup holds one CU on its own.  When runs of up to
    // CB_MAX_MB8 blocks let the whole launch (row blocks x runs x splits) fit
    // one workgroup per CU, deal the columns that way: a single round beats
    // two rounds of shorter runs, each re-reading the activation tiles.
    const int gx = (s.M + 127) / 128;
    const int nwg1 = std::max((nbc + CB_MAX_MB8 - 1) / CB_MAX_MB8, GEMM_WGS / (gx * s.splits));
    if (nwg1 < nwg && gx * nwg1 * s.splits <= GEMM_WGS) {
      const int cba1 = (nbc + nwg1 - 1) / nwg1;
      gemm_mb8<T>(s, e, kind, nwg1, cba1, nbc - nwg1 * (cba1 - 1), st, ev_start, eb);
    } else {
      gemm_mb8<T>(s, e, kind, nwg, cba, nbig, st, ev_start, eb);
    }
  } else
    gemm_mb<T, 4>(s, e, kind, nwg, cba, nbig, st, ev_start, eb);
  if (finish) {
    const int64_t total = (int64_t)s.M * nbc * 16;
    const dim3 grid((unsigned)((total + 255) / 256));
    if (ev_stop)
      hipExtLaunchKernelGGL((gemm_finish_kernel<T>), grid, dim3(256), 0, st, nullptr, ev_stop, 0, s, e, e.kind,
                            (const float*)e.part);
    else
      hipLaunchKernelGGL((gemm_finish_kernel<T>), grid, dim3(256), 0, st, s, e, e.kind, (const float*)e.part);
  }
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
  // Wide matrices have enough column blocks to fill the GPU on their own;
  // narrow ones split the reduction so that >= 256 workgroups stream weights.
  const int KB = dtype == DT_BF16 ? 32 : 16;
  const int kblocks = K / KB;
  if (n_cols >= SPLIT_MIN_COLS_NO) return 1;
  const int groups = n_cols / 64;
  int s = 1;
  while (groups * s < SPLIT_TARGET_WGS && s < GEMM_MAX_SPLITS && kblocks % (2 * s) == 0 && kblocks / (2 * s) >= 16) s *= 2;
  return s;
}

void launch_gemm(int dtype, const GemmShape& s, const GemmEpi& e, hipStream_t st, hipEvent_t ev_start,
                 hipEvent_t ev_stop) {
  if (s.M <= 0) return;
  if (dtype == DT_BF16)
    gemm_t<bf16_t>(s, e, st, ev_start, ev_stop);
  else
    gemm_t<float>(s, e, st, ev_start, ev_stop);
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
