// Rows of several overlapping subgraphs of one graph on one device
// (Algorithm 1 over K workers).  Every node is a base node of exactly one
// subgraph (its own partition block) and an overlap node of every other
// subgraph that selected it.
//
//   MeanAgg (the inference step of Algorithm 1; averaging of the overlap
//   nodes' representations in "Prediction and Optimization"):
//     H[v] = (1/cnt[v]) sum_{k : v in subgraph k} H_k[g2l_k[v]]
//   its backward for one subgraph:  dH_k[i] = dH[l2g_k[i]] / cnt[l2g_k[i]]
//   the home copies (the CCA target of an overlap node: its row in the
//   subgraph of its own partition block):
//     Y[i] = H_home[g2l_home[l2g_k[overlap_k[i]]]],  home = part of that node
//
// All three are row gathers: one thread moves one 16-byte chunk of a row, so
// a row is a run of consecutive lanes and each load instruction of a wave
// covers whole 64-byte segments.  The MeanAgg forward walks the subgraphs in
// k order for every node (fixed summation order, no atomics, no zeroing);
// local ids follow global ids within a node type, so consecutive nodes read
// nearly consecutive rows of every subgraph.
#include <cmath>

#include "hg_mfma.h"

namespace hg {
namespace {

constexpr int kMaxParts = HG_MAX_PARTS;
constexpr int kRowThreads = 256;

// The K subgraphs' row arrays and global2local maps, passed by value in the
// kernel arguments (no device-side table to keep in sync).
struct PartTables {
  const void* h[kMaxParts];
  const int32_t* g2l[kMaxParts];
};

inline unsigned row_grid(int64_t rows, int chunks_per_row) {
  return (unsigned)cdiv(rows * chunks_per_row, kRowThreads);
}

template <int D, class T>
__global__ void __launch_bounds__(kRowThreads)
    k_mean_agg_fwd(int64_t n, int K, PartTables p, T* __restrict__ H, int32_t* __restrict__ cnt) {
  constexpr int EL = Elt<T>::EL, CPR = D / EL;
  const int64_t t = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  const int64_t v = t / CPR;
  if (v >= n) return;
  const int c = (int)(t % CPR) * EL;
  float acc[EL];
#pragma unroll
  for (int q = 0; q < EL; ++q) acc[q] = 0.f;
  int m = 0;
  // the maps of four subgraphs are read before their rows, so the row loads
  // of a group are in flight together
  for (int k0 = 0; k0 < K; k0 += 4) {
    int32_t r[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) r[u] = (k0 + u < K) ? p.g2l[k0 + u][v] : -1;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (r[u] < 0) continue;
      float x[EL];
      Elt<T>::load(static_cast<const T*>(p.h[k0 + u]) + (int64_t)r[u] * D + c, x);
#pragma unroll
      for (int q = 0; q < EL; ++q) acc[q] += x[q];
      ++m;
    }
  }
  if (m > 1) {
    const float fm = (float)m;
#pragma unroll
    for (int q = 0; q < EL; ++q) acc[q] = acc[q] / fm;
  }
  Elt<T>::store(H + v * D + c, acc);
  if (cnt && c == 0) cnt[v] = m;
}

template <int D, class T>
__global__ void __launch_bounds__(kRowThreads)
    k_mean_agg_bwd(int64_t n_sub, const int32_t* __restrict__ l2g, const int32_t* __restrict__ cnt,
                   const T* __restrict__ dH, T* __restrict__ dHk, int accumulate) {
  constexpr int EL = Elt<T>::EL, CPR = D / EL;
  const int64_t t = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  const int64_t i = t / CPR;
  if (i >= n_sub) return;
  const int c = (int)(t % CPR) * EL;
  const int64_t v = l2g[i];
  const int m = cnt[v];
  float x[EL];
  Elt<T>::load(dH + v * D + c, x);
  // a node that no subgraph holds cannot be a row of one: poison it
  const float fm = m > 0 ? (float)m : __builtin_nanf("");
#pragma unroll
  for (int q = 0; q < EL; ++q) x[q] = m == 1 ? x[q] : x[q] / fm;
  if (accumulate) {
    float y[EL];
    Elt<T>::load(dHk + i * D + c, y);
#pragma unroll
    for (int q = 0; q < EL; ++q) x[q] = y[q] + x[q];
  }
  Elt<T>::store(dHk + i * D + c, x);
}

template <int D, class T>
__global__ void __launch_bounds__(kRowThreads)
    k_home_gather(int64_t m, int K, PartTables p, const int32_t* __restrict__ overlap,
                  const int32_t* __restrict__ l2g, const int32_t* __restrict__ home, T* __restrict__ Y) {
  constexpr int EL = Elt<T>::EL, CPR = D / EL;
  const int64_t t = (int64_t)blockIdx.x * kRowThreads + threadIdx.x;
  const int64_t i = t / CPR;
  if (i >= m) return;
  const int c = (int)(t % CPR) * EL;
  const int64_t v = l2g[overlap[i]];
  const int h = home[i];
  const int32_t r = (h >= 0 && h < K) ? p.g2l[h][v] : -1;
  float x[EL];
  if (r >= 0) {
    Elt<T>::load(static_cast<const T*>(p.h[h]) + (int64_t)r * D + c, x);
  } else {
#pragma unroll
    for (int q = 0; q < EL; ++q) x[q] = __builtin_nanf("");
  }
  Elt<T>::store(Y + i * D + c, x);
}

int check_rows(int32_t d, int32_t dtype) {
  if (dtype != HG_DTYPE_F32 && dtype != HG_DTYPE_BF16) return fail(HG_ERR_ARG, "dtype must be f32 or bf16");
  if (d != 64 && d != 128 && d != 256) return fail(HG_ERR_UNSUPPORTED, "d must be 64, 128 or 256");
  return HG_OK;
}

int fill_tables(int32_t K, const int32_t* const* g2l, const void* const* h_parts, PartTables& p) {
  if (K < 1 || K > kMaxParts) return fail(HG_ERR_ARG, "K must be in [1, %d]", kMaxParts);
  if (!g2l || !h_parts) return fail(HG_ERR_ARG, "null table");
  for (int k = 0; k < kMaxParts; ++k) {
    p.h[k] = k < K ? h_parts[k] : nullptr;
    p.g2l[k] = k < K ? g2l[k] : nullptr;
    if (k < K && (!p.h[k] || !p.g2l[k])) return fail(HG_ERR_ARG, "null pointer for subgraph %d", k);
  }
  return HG_OK;
}

template <class T>
constexpr int chunks_per_row(int D) {
  return D / Elt<T>::EL;
}

template <int D, class T>
int launch_mean_agg_fwd(int64_t n, int K, const PartTables& p, void* H, int32_t* cnt, hipStream_t st) {
  HG_LAUNCH("mean_agg_fwd", (k_mean_agg_fwd<D, T>), dim3(row_grid(n, chunks_per_row<T>(D))), dim3(kRowThreads), 0,
            st, n, K, p, static_cast<T*>(H), cnt);
  return HG_OK;
}

template <int D, class T>
int launch_mean_agg_bwd(int64_t n, const int32_t* l2g, const int32_t* cnt, const void* dH, void* dh, int acc,
                        hipStream_t st) {
  HG_LAUNCH("mean_agg_bwd", (k_mean_agg_bwd<D, T>), dim3(row_grid(n, chunks_per_row<T>(D))), dim3(kRowThreads), 0,
            st, n, l2g, cnt, static_cast<const T*>(dH), static_cast<T*>(dh), acc);
  return HG_OK;
}

template <int D, class T>
int launch_home_gather(int64_t m, int K, const PartTables& p, const int32_t* overlap, const int32_t* l2g,
                       const int32_t* home, void* Y, hipStream_t st) {
  HG_LAUNCH("home_gather", (k_home_gather<D, T>), dim3(row_grid(m, chunks_per_row<T>(D))), dim3(kRowThreads), 0,
            st, m, K, p, overlap, l2g, home, static_cast<T*>(Y));
  return HG_OK;
}

// (d, dtype) -> the instantiation of a launcher: F<D, T>(args...)
#define HG_ROWS_DISPATCH(d, dtype, F, ...)                                   \
  ((dtype) == HG_DTYPE_BF16                                                  \
       ? ((d) == 64    ? F<64, bf16_t>(__VA_ARGS__)                          \
          : (d) == 128 ? F<128, bf16_t>(__VA_ARGS__)                         \
                       : F<256, bf16_t>(__VA_ARGS__))                        \
       : ((d) == 64    ? F<64, float>(__VA_ARGS__)                           \
          : (d) == 128 ? F<128, float>(__VA_ARGS__)                          \
                       : F<256, float>(__VA_ARGS__)))

}  // namespace
}  // namespace hg

using namespace hg;

extern "C" {

int hg_mean_agg_fwd(int64_t n_nodes, int32_t d, int32_t dtype, int32_t K, const int32_t* const* g2l,
                    const void* const* h_parts, void* H, int32_t* cnt, void* stream) {
  HG_TRY(check_rows(d, dtype));
  if (n_nodes < 0) return fail(HG_ERR_ARG, "n_nodes < 0");
  PartTables p;
  HG_TRY(fill_tables(K, g2l, h_parts, p));
  if (n_nodes == 0) return HG_OK;
  if (!H) return fail(HG_ERR_ARG, "null H");
  return HG_ROWS_DISPATCH(d, dtype, launch_mean_agg_fwd, n_nodes, K, p, H, cnt, static_cast<hipStream_t>(stream));
}

int hg_mean_agg_bwd(int64_t n_sub, int32_t d, int32_t dtype, const int32_t* l2g, const int32_t* cnt,
                    const void* dH, void* dh_part, int32_t accumulate, void* stream) {
  HG_TRY(check_rows(d, dtype));
  if (n_sub < 0) return fail(HG_ERR_ARG, "n_sub < 0");
  if (accumulate != 0 && accumulate != 1) return fail(HG_ERR_ARG, "accumulate must be 0 or 1");
  if (n_sub == 0) return HG_OK;
  if (!l2g || !cnt || !dH || !dh_part) return fail(HG_ERR_ARG, "null pointer");
  if (dH == dh_part) return fail(HG_ERR_ARG, "dh_part must not alias dH");
  return HG_ROWS_DISPATCH(d, dtype, launch_mean_agg_bwd, n_sub, l2g, cnt, dH, dh_part, accumulate,
                          static_cast<hipStream_t>(stream));
}

int hg_home_gather(int64_t m, int32_t d, int32_t dtype, int32_t K, const int32_t* overlap, const int32_t* l2g,
                   const int32_t* home, const int32_t* const* g2l, const void* const* h_parts, void* Y,
                   void* stream) {
  HG_TRY(check_rows(d, dtype));
  if (m < 0) return fail(HG_ERR_ARG, "m < 0");
  PartTables p;
  HG_TRY(fill_tables(K, g2l, h_parts, p));
  if (m == 0) return HG_OK;
  if (!overlap || !l2g || !home || !Y) return fail(HG_ERR_ARG, "null pointer");
  return HG_ROWS_DISPATCH(d, dtype, launch_home_gather, m, K, p, overlap, l2g, home, Y,
                          static_cast<hipStream_t>(stream));
}

}  // extern "C"
