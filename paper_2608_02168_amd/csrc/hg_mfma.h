// MFMA building blocks for gfx950 (fp32 path: v_mfma_f32_16x16x4_f32).
//
// Lane layouts (64-lane wave, g = lane / 16, c = lane % 16):
//   A operand (16 x 4):  lane holds A[c][g]
//   B operand (4 x 16):  lane holds B[g][c]
//   C/D (16 x 16):       lane holds D[4 g + v][c] in accumulator register v
//
// Two kernels are built on it:
//   gemm_rows   C[rows] = epi(A[rows] . op(W))   with W (d x d) staged in LDS,
//               rows gathered through a row map; a 16-wide K block is split
//               so each lane reads 4 consecutive A elements (one float4),
//               matched by the same K permutation of W inside LDS;
//   gemm_tn     partial[chunk] = A[rows]^T B[rows] over a chunk of rows,
//               a deterministic split-K for weight gradients and Gram matrices.
#pragma once

#include "hg_internal.h"

namespace hg {

typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4 mfma4(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ int lane64() { return threadIdx.x & 63; }

// Row map: row(i) = (list ? list[i] : first + i) * mul + add.
struct RowMap {
  const int32_t* list;
  int64_t first;
  int32_t mul;
  int32_t add;
  __device__ __forceinline__ int64_t operator()(int64_t i) const {
    const int64_t b = list ? (int64_t)list[i] : first + i;
    return b * mul + add;
  }
};

inline RowMap rows_contig(int64_t first) { return RowMap{nullptr, first, 1, 0}; }
inline RowMap rows_list(const int32_t* list, int32_t mul = 1, int32_t add = 0) {
  return RowMap{list, 0, mul, add};
}

// ---- A loaders: return 4 consecutive columns [c, c+4) of segment row i ----
template <int D>
struct LoadRows {
  const float* base;
  RowMap map;
  __device__ __forceinline__ f32x4 row4(int64_t i, int c) const {
    return *reinterpret_cast<const f32x4*>(base + map(i) * D + c);
  }
  __device__ __forceinline__ float at(int64_t i, int c) const { return base[map(i) * D + c]; }
};

// (x - mu[c]) * sc[c]: the per-column standardisation of the alignment loss.
template <int D>
struct LoadStd {
  const float* base;
  RowMap map;
  const float* mu;
  const float* sc;
  __device__ __forceinline__ f32x4 row4(int64_t i, int c) const {
    f32x4 x = *reinterpret_cast<const f32x4*>(base + map(i) * D + c);
    f32x4 m = *reinterpret_cast<const f32x4*>(mu + c);
    f32x4 s = *reinterpret_cast<const f32x4*>(sc + c);
    return (x - m) * s;
  }
  __device__ __forceinline__ float at(int64_t i, int c) const {
    return (base[map(i) * D + c] - mu[c]) * sc[c];
  }
};

// ---- epilogue: out[row] = acc + bias + addend[row] --------------------------
template <int D>
struct StoreRows {
  float* out;
  RowMap map;
  const float* bias;    // [D] or null
  const float* addend;  // rows through the same map, or null (may equal out)
  __device__ __forceinline__ void operator()(int64_t i, int c, float v) const {
    const int64_t o = map(i) * D + c;
    if (bias) v += bias[c];
    if (addend) v += addend[o];
    out[o] = v;
  }
};

// ---- gemm_rows --------------------------------------------------------------
// Block = 4 waves, tile = 64 rows (16 per wave); persistent over tiles.
// LDS holds op(W) in fragment order: element ((kb*NB + nb)*64 + lane)*4 + s is
// op(W)[16 kb + 4 (lane/16) + s][16 nb + lane%16].
template <int D, bool kTransW, class ALoad, class Epi>
__global__ void __launch_bounds__(256) k_gemm_rows(int64_t n_rows, const float* __restrict__ W,
                                                   ALoad aload, Epi epi) {
  constexpr int NB = D / 16;
  extern __shared__ f32x4 wl[];
  const int tid = threadIdx.x;
  for (int e = tid; e < NB * NB * 64; e += 256) {
    const int l = e & 63;
    const int nb = (e >> 6) % NB;
    const int kb = (e >> 6) / NB;
    const int j = 16 * nb + (l & 15);
    const int k0 = 16 * kb + 4 * (l >> 4);
    f32x4 v;
    if (kTransW) {
      v = *reinterpret_cast<const f32x4*>(W + (int64_t)j * D + k0);
    } else {
      v[0] = W[(int64_t)(k0 + 0) * D + j];
      v[1] = W[(int64_t)(k0 + 1) * D + j];
      v[2] = W[(int64_t)(k0 + 2) * D + j];
      v[3] = W[(int64_t)(k0 + 3) * D + j];
    }
    wl[e] = v;
  }
  __syncthreads();
  const int w = tid >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  const int64_t ntiles = (n_rows + 63) / 64;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t r0 = t * 64 + 16 * w;
    const int64_t ia = r0 + c;
    f32x4 a[NB];
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) {
      if (ia < n_rows) {
        a[kb] = aload.row4(ia, 16 * kb + 4 * g);
      } else {
        a[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
    }
    f32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < NB; ++kb) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const f32x4 b = wl[(kb * NB + nb) * 64 + l];
        acc[nb] = mfma4(a[kb][0], b[0], acc[nb]);
        acc[nb] = mfma4(a[kb][1], b[1], acc[nb]);
        acc[nb] = mfma4(a[kb][2], b[2], acc[nb]);
        acc[nb] = mfma4(a[kb][3], b[3], acc[nb]);
      }
    }
#pragma unroll
    for (int v = 0; v < 4; ++v) {
      const int64_t i = r0 + 4 * g + v;
      if (i < n_rows) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) epi(i, 16 * nb + c, acc[nb][v]);
      }
    }
  }
}

template <int D, bool kTransW, class ALoad, class Epi>
int launch_gemm_rows(const char* name, int64_t n_rows, const float* W, ALoad aload, Epi epi,
                     hipStream_t s) {
  if (n_rows <= 0) return HG_OK;
  const int64_t tiles = cdiv(n_rows, 64);
  const int64_t cap = (int64_t)num_cus() * 2;
  const int64_t grid = tiles < cap ? tiles : cap;
  const size_t lds = sizeof(float) * D * D;
  HG_LAUNCH(name, (k_gemm_rows<D, kTransW, ALoad, Epi>), dim3((unsigned)grid), dim3(256), lds, s,
            n_rows, W, aload, epi);
  return HG_OK;
}

// ---- gemm_tn split-K ----------------------------------------------------------
// partial[chunk][i][j] = sum_{rows k of the chunk} A[k][i] * B[k][j]
// colsum[chunk][j]    = sum_{rows k of the chunk} B[k][j]        (if colsum)
// D = 128: wave w owns the 64 x 64 quadrant (w/2, w%2) over all rows of the
// chunk.  D = 64: every wave owns the whole 64 x 64 output over every fourth
// group of 4 rows; the four waves are summed in LDS in wave order.
template <int D, class LA, class LB>
__global__ void __launch_bounds__(256) k_gemm_tn(int64_t n_rows, int64_t kc, LA la, LB lb,
                                                 float* __restrict__ partial,
                                                 float* __restrict__ colsum) {
  static_assert(D == 64 || D == 128, "gemm_tn: d must be 64 or 128");
  constexpr bool kQuad = (D == 128);
  const int w = threadIdx.x >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  const int64_t chunk = blockIdx.x;
  const int64_t k_beg = chunk * kc;
  const int64_t k_end = (k_beg + kc < n_rows) ? k_beg + kc : n_rows;
  const int qi = kQuad ? (w >> 1) : 0;
  const int qj = kQuad ? (w & 1) : 0;
  const int64_t step0 = kQuad ? 0 : 4 * w;
  const int64_t stride = kQuad ? 4 : 16;
  f32x4 acc[4][4];
  float bs[4];
#pragma unroll
  for (int bi = 0; bi < 4; ++bi) {
    bs[bi] = 0.f;
#pragma unroll
    for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  for (int64_t k0 = k_beg + step0; k0 < k_end; k0 += stride) {
    const int64_t row = k0 + g;
    float a[4], b[4];
    if (row < k_end) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        a[q] = la.at(row, 64 * qi + 16 * q + c);
        b[q] = lb.at(row, 64 * qj + 16 * q + c);
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = b[q] = 0.f;
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) bs[q] += b[q];
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = mfma4(a[bi], b[bj], acc[bi][bj]);
  }
  // column sums: reduce the 4 row groups of the wave
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    bs[q] += __shfl_xor(bs[q], 16, 64);
    bs[q] += __shfl_xor(bs[q], 32, 64);
  }
  float* out = partial + chunk * (int64_t)D * D;
  if (kQuad) {
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int bj = 0; bj < 4; ++bj)
#pragma unroll
        for (int v = 0; v < 4; ++v)
          out[(int64_t)(64 * qi + 16 * bi + 4 * g + v) * D + 64 * qj + 16 * bj + c] = acc[bi][bj][v];
    if (colsum && qi == 0 && g == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) colsum[chunk * D + 64 * qj + 16 * q + c] = bs[q];
    }
  } else {
    __shared__ float red[64 * 64];
    __shared__ float cred[64];
    for (int ww = 0; ww < 4; ++ww) {
      if (w == ww) {
#pragma unroll
        for (int bi = 0; bi < 4; ++bi)
#pragma unroll
          for (int bj = 0; bj < 4; ++bj)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int idx = (16 * bi + 4 * g + v) * 64 + 16 * bj + c;
              red[idx] = (ww == 0 ? 0.f : red[idx]) + acc[bi][bj][v];
            }
        if (g == 0) {
#pragma unroll
          for (int q = 0; q < 4; ++q) cred[16 * q + c] = (ww == 0 ? 0.f : cred[16 * q + c]) + bs[q];
        }
      }
      __syncthreads();
    }
    for (int e = threadIdx.x; e < 64 * 64; e += 256) out[e] = red[e];
    if (colsum && threadIdx.x < 64) colsum[chunk * D + threadIdx.x] = cred[threadIdx.x];
  }
}

// out[i] (+)= sum_{c < nchunks} partial[c][i]   (fixed order)
static __global__ void k_sum_partials(const float* __restrict__ partial, int64_t nchunks, int64_t n,
                                      float* __restrict__ out, int accumulate) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  float s = accumulate ? out[i] : 0.f;
  for (int64_t c = 0; c < nchunks; ++c) s += partial[c * n + i];
  out[i] = s;
}

// Chunking of a K-reduction of n rows (deterministic in n).
inline int64_t splitk_chunk(int64_t n) {
  int64_t chunks = cdiv(n, 512);
  const int64_t cap = (int64_t)num_cus() * 4;
  if (chunks > cap) chunks = cap;
  if (chunks < 1) chunks = 1;
  int64_t kc = cdiv(n, chunks);
  kc = cdiv(kc, 16) * 16;
  return kc > 16 ? kc : 16;
}
inline int64_t splitk_max_chunks() { return (int64_t)num_cus() * 4 + 1; }

template <int D, class LA, class LB>
int launch_gemm_tn(const char* name, int64_t n_rows, LA la, LB lb, float* partial, float* colsum,
                   float* out, float* out_colsum, int accumulate, hipStream_t s) {
  if (n_rows <= 0) {
    if (!accumulate) {
      HG_TRY(fill_f32(out, 0.f, (int64_t)D * D, s));
      if (out_colsum) HG_TRY(fill_f32(out_colsum, 0.f, D, s));
    }
    return HG_OK;
  }
  const int64_t kc = splitk_chunk(n_rows);
  const int64_t chunks = cdiv(n_rows, kc);
  HG_LAUNCH(name, (k_gemm_tn<D, LA, LB>), dim3((unsigned)chunks), dim3(256), 0, s, n_rows, kc, la,
            lb, partial, out_colsum ? colsum : nullptr);
  HG_LAUNCH("splitk_reduce", k_sum_partials, dim3((unsigned)cdiv((int64_t)D * D, 256)), dim3(256), 0, s,
            (const float*)partial, chunks, (int64_t)D * D, out, accumulate);
  if (out_colsum)
    HG_LAUNCH("splitk_reduce", k_sum_partials, dim3(1), dim3(256), 0, s, (const float*)colsum, chunks,
              (int64_t)D, out_colsum, accumulate);
  return HG_OK;
}

}  // namespace hg
