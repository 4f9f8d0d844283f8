// hg_layer_fwd / hg_layer_bwd: one relation-typed mean-aggregation layer.
//
// Forward (message, aggregation and update equations of the "Heterogeneous
// Graph Transformer" paragraph in relation-typed mean form):
//   (c) MFMA transforms  Y_self = H W_self[t] + b[t]   per contiguous type range
//                        Y[slot(i,r)] = H_i W_r         for i in S_r (active sources)
//   (b) SpMM             z_j = Y_self[j] + sum_{edges i->j of relation r} w_ij Y[slot(i,r)] / deg_r(j)
//                        (w_ij = 1 without edge weights)
//                        h'_j = ReLU(z_j) + h_j, ReLU mask saved as bits
// Y holds one row per active (source, relation) pair, A rows in all (slots
// numbered in CSC row order; the plan gives the slot of every CSR entry), or
// is indexed by the CSC row q = i R + r when that costs at most a few times
// more (the plan's row-indexed layout).
// Backward:
//   dZ = G * mask, formed while the dX self-transform loads G (and written out)
//   (b) transposed SpMM  dY[slot(i,r)] = sum_{edges i->j of r} csc_scale * dZ_j  (no atomics;
//                        rows longer than the chunk size are split, then summed in order)
//   (c) MFMA             dH = G + dZ W_self^T, then dH[S_r] += dY_r W_r^T for r = 0..R-1
//                        dW_self[t] = H_t^T dZ_t, db[t] = colsum dZ_t, dW_r = H[S_r]^T dY_r
//                        (split-K with a fixed-order reduction)
#include <vector>

#include "hg_internal.h"
#include "hg_mfma.h"

namespace hg {

namespace {

// ---- forward SpMM + epilogue --------------------------------------------------
// One wave per destination row.  A row of D elements of T is read as LPR
// 16-byte chunks (EL elements each); lanes form EPW = 64/LPR slots, a slot
// gathers one source row, so one wave step covers EPW edges.  Neighbour ids
// and weights of up to 64 entries sit one per lane and are broadcast with
// ds_bpermute.  Accumulation is float32.
// fp32 rows: 8 waves per SIMD (<= 64 VGPRs) keep the most gathers in flight.
// Rows of more than kFwdChunk entries (destination hubs) are left to the
// plan's chunks: k_spmm_fwd_part sums one chunk each, k_spmm_fwd_merge adds
// a row's chunks in order and applies the epilogue.

// acc (lane's slot share, columns c0..c0+EL) += weighted Y rows of the CSR
// entries [beg, end) of destination row rb / R, whose entries over all
// relations are [p0, pe).  Y row of an entry: its slot, or src * R + r in
// the row-indexed layout (csr_slot null).
template <int D, class T>
__device__ __forceinline__ void fwd_gather(int64_t rb, int32_t R, int32_t p0, int32_t pe, int32_t beg, int32_t end,
                                           const int32_t* __restrict__ csr_ptr, const int32_t* __restrict__ csr_col,
                                           const int32_t* __restrict__ csr_slot, const float* __restrict__ csr_w,
                                           const T* __restrict__ Y, int l, int slot, int c0,
                                           float (&acc)[Elt<T>::EL]) {
  constexpr int EL = Elt<T>::EL;
  constexpr int EPW = 64 / (D / EL);
  constexpr int U = 4;
  for (int32_t base = beg; base < end; base += 64) {
    const int32_t pos = base + l;
    int32_t rowi = 0;
    float wgt = 0.f;
    if (pos < end) {
      int32_t lo = p0, hi = pe, r = 0;
      for (int t = 1; t < R; ++t) {
        const int32_t pt = csr_ptr[rb + t];
        if (pt <= pos) {
          lo = pt;
          r = t;
        } else if (pt < hi) {
          hi = pt;
        }
      }
      rowi = csr_slot ? csr_slot[pos] : csr_col[pos] * R + r;
      wgt = (csr_w ? csr_w[pos] : 1.0f) / (float)(hi - lo);
    }
    const int cnt = (end - base) < 64 ? (end - base) : 64;
    for (int e = 0; e < cnt; e += EPW * U) {
      typename Elt<T>::rawv_t v[U];
      float ww[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int my = e + u * EPW + slot;
        const int32_t q = __shfl(rowi, my & 63, 64);
        const float wq = __shfl(wgt, my & 63, 64);
        ww[u] = (my < cnt) ? wq : 0.f;
        v[u] = (my < cnt) ? Elt<T>::rawv(Y + (int64_t)q * D + c0) : Elt<T>::rawv_zero();
      }
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < EL; ++k) acc[k] += ww[u] * Elt<T>::rawv_get(v[u], k);
    }
  }
}

// z = acc + Y_self[j]; h' = ReLU(z) + h; the mask bits.  acc is reduced over
// the slots; every lane of the wave calls it (the mask word is gathered with
// shuffles), slot 0 stores.
template <int D, class T>
__device__ __forceinline__ void fwd_epilogue(int64_t j, const float (&acc)[Elt<T>::EL], int slot, int c0,
                                             const T* __restrict__ Yself, const T* __restrict__ Hin,
                                             T* __restrict__ Hout, uint32_t* __restrict__ mask, int relu,
                                             int residual) {
  constexpr int EL = Elt<T>::EL;
  const int64_t off = j * D + c0;
  uint32_t word = 0;
  if (slot == 0) {
    float ys[EL], h[EL], z[EL];
    Elt<T>::load(Yself + off, ys);
    float hin[EL];
    if (residual) Elt<T>::load(Hin + off, hin);
    uint32_t bits = 0;
#pragma unroll
    for (int k = 0; k < EL; ++k) {
      z[k] = acc[k] + ys[k];
      h[k] = (relu && !(z[k] > 0.f)) ? 0.f : z[k];
      if (residual) h[k] += hin[k];
      bits |= ((!relu || z[k] > 0.f) ? 1u : 0u) << k;
    }
    Elt<T>::store(Hout + off, h);
    word = bits << (c0 & 31);
  }
  // OR the EL-bit groups of the 32/EL lanes that share a mask word
#pragma unroll
  for (int o = 1; o < 32 / EL; o <<= 1) word |= __shfl_xor(word, o, 64);
  if (slot == 0 && (c0 & 31) == 0) mask[j * (D / 32) + (c0 >> 5)] = word;
}

template <int D, class T>
__global__ void __launch_bounds__(256, (sizeof(T) == 2 || D <= 128) ? 8 : 4) k_spmm_fwd(int64_t n_sub, int32_t R, const int32_t* __restrict__ csr_ptr,
                                                  const int32_t* __restrict__ csr_col,
                                                  const int32_t* __restrict__ csr_slot,
                                                  const float* __restrict__ csr_w,
                                                  const T* __restrict__ Y, const T* __restrict__ Yself,
                                                  const T* __restrict__ Hin, T* __restrict__ Hout,
                                                  uint32_t* __restrict__ mask, int relu, int residual) {
  constexpr int EL = Elt<T>::EL;
  constexpr int LPR = D / EL;
  constexpr int EPW = 64 / LPR;
  static_assert(LPR <= 64 && EPW * LPR == 64, "row must span a power-of-two number of lanes");
  const int l = threadIdx.x & 63;
  const int slot = l / LPR;
  const int c0 = (l % LPR) * EL;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t j = wave0; j < n_sub; j += nwaves) {
    const int64_t rb = j * R;
    const int32_t p0 = csr_ptr[rb];
    const int32_t pe = csr_ptr[rb + R];
    if (pe - p0 > kFwdChunk) continue;  // a chunked row
    float acc[EL];
#pragma unroll
    for (int q = 0; q < EL; ++q) acc[q] = 0.f;
    fwd_gather<D, T>(rb, R, p0, pe, p0, pe, csr_ptr, csr_col, csr_slot, csr_w, Y, l, slot, c0, acc);
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
      for (int k = 0; k < EL; ++k) acc[k] += __shfl_xor(acc[k], o, 64);
    fwd_epilogue<D, T>(j, acc, slot, c0, Yself, Hin, Hout, mask, relu, residual);
  }
}

// One wave per chunk (j, begin, end, partial slot) of a long destination
// row: the chunk's weighted sum, float32, into its partial row.
template <int D, class T>
__global__ void __launch_bounds__(256) k_spmm_fwd_part(int64_t n_items, const int4* __restrict__ items, int32_t R,
                                                       const int32_t* __restrict__ csr_ptr,
                                                       const int32_t* __restrict__ csr_col,
                                                       const int32_t* __restrict__ csr_slot,
                                                       const float* __restrict__ csr_w, const T* __restrict__ Y,
                                                       float* __restrict__ part) {
  constexpr int EL = Elt<T>::EL;
  constexpr int LPR = D / EL;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR;
  const int c0 = (l % LPR) * EL;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t it = wave0; it < n_items; it += nwaves) {
    const int4 item = items[it];
    const int64_t rb = (int64_t)item.x * R;
    float acc[EL];
#pragma unroll
    for (int q = 0; q < EL; ++q) acc[q] = 0.f;
    fwd_gather<D, T>(rb, R, csr_ptr[rb], csr_ptr[rb + R], item.y, item.z, csr_ptr, csr_col, csr_slot, csr_w, Y, l,
                     slot, c0, acc);
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
      for (int k = 0; k < EL; ++k) acc[k] += __shfl_xor(acc[k], o, 64);
    if (slot == 0) {
      float* p = part + (int64_t)item.w * D + c0;
#pragma unroll
      for (int k = 0; k < EL; k += 4) *reinterpret_cast<f32x4*>(p + k) = f32x4{acc[k], acc[k + 1], acc[k + 2], acc[k + 3]};
    }
  }
}

// One wave per long row (j, first partial, count): the partial rows added in
// float64 (slot s takes partials s, s + EPW, ...; the slots then add in a
// fixed tree), then the epilogue.
template <int D, class T>
__global__ void __launch_bounds__(256) k_spmm_fwd_merge(int64_t n_heavy, const int4* __restrict__ heavy,
                                                        const float* __restrict__ part, const T* __restrict__ Yself,
                                                        const T* __restrict__ Hin, T* __restrict__ Hout,
                                                        uint32_t* __restrict__ mask, int relu, int residual) {
  constexpr int EL = Elt<T>::EL;
  constexpr int LPR = D / EL;
  constexpr int EPW = 64 / LPR;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR;
  const int c0 = (l % LPR) * EL;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t h = wave0; h < n_heavy; h += nwaves) {
    const int4 hv = heavy[h];
    double sd[EL];
#pragma unroll
    for (int k = 0; k < EL; ++k) sd[k] = 0.0;
    for (int32_t c = slot; c < hv.z; c += EPW) {
      const float* p = part + (int64_t)(hv.y + c) * D + c0;
#pragma unroll
      for (int k = 0; k < EL; k += 4) {
        const f32x4 x = *reinterpret_cast<const f32x4*>(p + k);
        sd[k] += x[0]; sd[k + 1] += x[1]; sd[k + 2] += x[2]; sd[k + 3] += x[3];
      }
    }
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
      for (int k = 0; k < EL; ++k) sd[k] += __shfl_xor(sd[k], o, 64);
    float acc[EL];
#pragma unroll
    for (int k = 0; k < EL; ++k) acc[k] = (float)sd[k];
    fwd_epilogue<D, T>(hv.x, acc, slot, c0, Yself, Hin, Hout, mask, relu, residual);
  }
}

// ---- backward transposed SpMM over the CSC work items ---------------------------
// CSC rows of hub sources hold up to millions of entries, so each lane
// accumulates in float64 (the kernel is bound by the gathers, not the adds);
// split rows keep float64 partial rows.
template <int D, class T, class TO>
__global__ void __launch_bounds__(256, (sizeof(T) == 2 || D <= 128) ? 8 : 4) k_spmm_bwd(int64_t n_items, const int4* __restrict__ items,
                                                  const int32_t* __restrict__ csc_row,
                                                  const float* __restrict__ csc_scale,
                                                  const T* __restrict__ dZ,
                                                  TO* __restrict__ dY, double* __restrict__ partial) {
  constexpr int EL = Elt<T>::EL;
  constexpr int LPR = D / EL;
  constexpr int EPW = 64 / LPR;
  constexpr int U = 4;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR;
  const int c0 = (l % LPR) * EL;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  if constexpr (sizeof(T) == 4) {
    // float32 rows: one float4 per lane, float64 accumulators (54 VGPRs)
    for (int64_t it = wave0; it < n_items; it += nwaves) {
      const int4 item = items[it];
      const int32_t beg = item.y, end = item.z;
      f64x4 acc = {0.0, 0.0, 0.0, 0.0};
      for (int32_t base = beg; base < end; base += 64) {
        const int32_t pos = base + l;
        int32_t dst = 0;
        float sc = 0.f;
        if (pos < end) {
          dst = csc_row[pos];
          sc = csc_scale[pos];
        }
        const int cnt = (end - base) < 64 ? (end - base) : 64;
        for (int e = 0; e < cnt; e += EPW * U) {
          f32x4 v[U];
          float ww[U];
#pragma unroll
          for (int u = 0; u < U; ++u) {
            const int my = e + u * EPW + slot;
            const int32_t q = __shfl(dst, my & 63, 64);
            const float wq = __shfl(sc, my & 63, 64);
            ww[u] = (my < cnt) ? wq : 0.f;
            if (my < cnt) {
              v[u] = *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(dZ) + (int64_t)q * D + c0);
            } else {
              v[u] = f32x4{0.f, 0.f, 0.f, 0.f};
            }
          }
#pragma unroll
          for (int u = 0; u < U; ++u)
#pragma unroll
            for (int q = 0; q < 4; ++q) acc[q] += (double)ww[u] * (double)v[u][q];
        }
      }
#pragma unroll
      for (int o = LPR; o < 64; o <<= 1) {
        acc[0] += __shfl_xor(acc[0], o, 64);
        acc[1] += __shfl_xor(acc[1], o, 64);
        acc[2] += __shfl_xor(acc[2], o, 64);
        acc[3] += __shfl_xor(acc[3], o, 64);
      }
      if (slot == 0) {
        if (item.w < 0) {
          f32x4 o;
#pragma unroll
          for (int q = 0; q < 4; ++q) o[q] = (float)acc[q];
          *reinterpret_cast<f32x4*>(dY + (int64_t)item.x * D + c0) = o;
        } else {
          *reinterpret_cast<f64x4*>(partial + (int64_t)item.w * D + c0) = acc;
        }
      }
    }
  } else {
    // bf16 rows: the gathered chunks stay packed until the float64 adds
    // (<= 64 VGPRs, 8 waves per SIMD as for float32 rows)
    for (int64_t it = wave0; it < n_items; it += nwaves) {
      const int4 item = items[it];
      const int32_t beg = item.y, end = item.z;
      double acc[EL];
#pragma unroll
      for (int k = 0; k < EL; ++k) acc[k] = 0.0;
      for (int32_t base = beg; base < end; base += 64) {
        const int32_t pos = base + l;
        int32_t dst = 0;
        float sc = 0.f;
        if (pos < end) {
          dst = csc_row[pos];
          sc = csc_scale[pos];
        }
        const int cnt = (end - base) < 64 ? (end - base) : 64;
        for (int e = 0; e < cnt; e += EPW * U) {
          typename Elt<T>::rawv_t v[U];
          float ww[U];
  #pragma unroll
          for (int u = 0; u < U; ++u) {
            const int my = e + u * EPW + slot;
            const int32_t q = __shfl(dst, my & 63, 64);
            const float wq = __shfl(sc, my & 63, 64);
            ww[u] = (my < cnt) ? wq : 0.f;
            v[u] = (my < cnt) ? Elt<T>::rawv(dZ + (int64_t)q * D + c0) : Elt<T>::rawv_zero();
          }
  #pragma unroll
          for (int u = 0; u < U; ++u) {
            const double w = (double)ww[u];
  #pragma unroll
            for (int k = 0; k < EL; ++k) acc[k] += (double)Elt<T>::rawv_get(v[u], k) * w;
          }
        }
      }
  #pragma unroll
      for (int o = LPR; o < 64; o <<= 1)
  #pragma unroll
        for (int k = 0; k < EL; ++k) acc[k] += __shfl_xor(acc[k], o, 64);
      if (slot == 0) {
        if (item.w < 0) {
          static_assert(sizeof(TO) == 4, "dY is float32");
          float* o = dY + (int64_t)item.x * D + c0;
  #pragma unroll
          for (int k = 0; k < EL; k += 4)
            *reinterpret_cast<f32x4*>(o + k) =
                f32x4{(float)acc[k], (float)acc[k + 1], (float)acc[k + 2], (float)acc[k + 3]};
        } else {
          double* p = partial + (int64_t)item.w * D + c0;
  #pragma unroll
          for (int k = 0; k < EL; k += 4)
            *reinterpret_cast<f64x4*>(p + k) = f64x4{acc[k], acc[k + 1], acc[k + 2], acc[k + 3]};
        }
      }
    }
  }
}

// Split rows: dY[q] = sum of its partial rows (float64), in a fixed order:
// the 64 / (D/4) lane groups of the wave take interleaved partials, each
// group with four accumulators for partials i, i + G, i + 2G, i + 3G (G the
// group count) so that eight or more rows are in flight per wave, then the
// accumulators and the groups are added in a fixed tree.  A hub's row of
// millions of entries (thousands of partials) no longer waits on one load
// at a time.
template <int D, class T>
__global__ void k_heavy_reduce(int64_t n_heavy, const int4* __restrict__ heavy,
                               const double* __restrict__ partial, T* __restrict__ dY) {
  constexpr int EL = 4;
  constexpr int LPR = D / EL;
  constexpr int NG = 64 / LPR;  // lane groups per wave
  constexpr int U = 4;
  const int l = threadIdx.x & 63;
  const int grp = l / LPR, lr = l % LPR;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t h = wave0; h < n_heavy; h += nwaves) {
    const int4 hv = heavy[h];
    double s[U][EL];
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int k = 0; k < EL; ++k) s[u][k] = 0.0;
    const double* base = partial + (int64_t)hv.y * D + lr * EL;
    int32_t i = grp;
    for (; i + (U - 1) * NG < hv.z; i += U * NG) {
      double x[U][EL];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < EL; ++k) x[u][k] = base[(int64_t)(i + u * NG) * D + k];
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int k = 0; k < EL; ++k) s[u][k] += x[u][k];
    }
    for (; i < hv.z; i += NG) {
#pragma unroll
      for (int k = 0; k < EL; ++k) s[0][k] += base[(int64_t)i * D + k];
    }
    double t[EL];
#pragma unroll
    for (int k = 0; k < EL; ++k) t[k] = (s[0][k] + s[1][k]) + (s[2][k] + s[3][k]);
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
      for (int k = 0; k < EL; ++k) t[k] += __shfl_xor(t[k], o, 64);
    if (grp == 0)
      *reinterpret_cast<f32x4*>(dY + (int64_t)hv.x * D + lr * EL) =
          f32x4{(float)t[0], (float)t[1], (float)t[2], (float)t[3]};
  }
}

inline unsigned wave_grid(int64_t n_waves) {
  int64_t blocks = cdiv(n_waves, 4);
  const int64_t cap = (int64_t)num_cus() * 64;
  if (blocks > cap) blocks = cap;
  return (unsigned)(blocks > 0 ? blocks : 1);
}

int validate_layer(const hg_subgraph* s, const hg_layer_desc* L) {
  if (!s || !L) return fail(HG_ERR_ARG, "null subgraph or layer descriptor");
  if (L->d_in != L->d_out) return fail(HG_ERR_UNSUPPORTED, "d_in %d != d_out %d", L->d_in, L->d_out);
  if (L->dtype != HG_DTYPE_F32 && L->dtype != HG_DTYPE_BF16)
    return fail(HG_ERR_ARG, "dtype %d", L->dtype);
  if (L->d_in != 64 && L->d_in != 128 && L->d_in != 256)
    return fail(HG_ERR_UNSUPPORTED, "layers support d in {64, 128, 256}, got %d", L->d_in);
  if ((L->relu != 0 && L->relu != 1) || (L->residual != 0 && L->residual != 1))
    return fail(HG_ERR_ARG, "relu/residual must be 0 or 1");
  if (s->n_sub < 0 || s->n_rel < 1 || s->n_ntype < 1 || !s->csr_ptr || !s->csc_ptr || !s->plan)
    return fail(HG_ERR_ARG, "subgraph not built");
  return HG_OK;
}

template <int D, class T>
struct FwdWs {
  T *Y, *Yself;
  float* part;  // partial rows of the chunks of long destination rows
  template <class A>
  void layout(A& a, const hg_subgraph* s) {
    Y = a.template take<T>(n_slots(s) * (int64_t)D);
    Yself = a.template take<T>(s->n_sub * (int64_t)D);
    part = a.template take<float>(s->plan_fwd_parts * (int64_t)D);
  }
};

// dZ keeps the feature type (it is G times a 0/1 mask, exact); dY and, for
// bfloat16 features, the dH accumulator are float32 so hub rows keep full
// precision until the single final rounding.
template <int D, class T>
struct BwdWs {
  T* dZ;
  float *dY, *dhacc, *splitk, *colsum;
  double* part;
  template <class A>
  void layout(A& a, const hg_subgraph* s) {
    dZ = a.template take<T>(s->n_sub * (int64_t)D);
    dY = a.template take<float>(n_slots(s) * (int64_t)D);
    dhacc = a.template take<float>(sizeof(T) == 2 ? s->n_sub * (int64_t)D : 0);
    part = a.template take<double>(s->plan_partials * (int64_t)D);
    splitk = a.template take<float>(splitk_max_chunks() * (int64_t)D * D);
    colsum = a.template take<float>(splitk_max_chunks() * (int64_t)D);
  }
};

// Row transform with float32 operands and results (split-fp16 MFMA products).
template <int D, bool kTransW, class ALoad, class Epi>
int rows_f32(const char* name, int64_t n, const float* W, ALoad la, Epi ep, hipStream_t st) {
  return launch_gemm_rows_pp<D, kTransW>(name, n, W, la, ep, st);
}

// fp32 features use the fp32 MFMA transform, bf16 features the bf16 one.
template <int D, class T, bool kTransW, class ALoad, class Epi>
int transform(const char* name, int64_t n, const float* W, ALoad la, Epi ep, hipStream_t st) {
  if constexpr (sizeof(T) == 4) {
    return rows_f32<D, kTransW>(name, n, W, la, ep, st);
  } else {
    return launch_gemm_rows_bf16<D, kTransW>(name, n, W, la, ep, st);
  }
}

template <int D, class T>
int layer_fwd_impl(const hg_subgraph* s, const hg_layer_desc* L, const T* Hin, const float* W_rel,
                   const float* W_self, const float* bias, T* Hout, uint32_t* mask, void* ws,
                   size_t ws_bytes, hipStream_t st) {
  Arena a(ws, ws_bytes);
  FwdWs<D, T> w;
  w.layout(a, s);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "forward workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  const int32_t R = s->n_rel;
  const PlanView pv = plan_view(s);
  // (c) self transform per node type, bias folded in
  for (int t = 0; t < s->n_ntype; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    LoadRows<D, T> la{Hin, rows_contig(lo)};
    StoreRows<D, T> ep{w.Yself, rows_contig(lo), bias ? bias + (int64_t)t * D : nullptr, nullptr};
    HG_TRY((transform<D, T, false>("gemm_fwd_self", hi - lo, W_self + (int64_t)t * D * D, la, ep, st)));
  }
  // (c) relation transforms over the active sources
  int64_t off = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t n = s->n_active[r];
    LoadRows<D, T> la{Hin, rows_list(pv.active + off)};
    StoreRows<D, T> ep{w.Y, rows_list(pv.act_slot + off), nullptr, nullptr};
    HG_TRY((transform<D, T, false>("gemm_fwd_rel", n, W_rel + (int64_t)r * D * D, la, ep, st)));
    off += n;
  }
  // (b) aggregation + epilogue; long destination rows by chunks; the edge
  // weights of a weighted graph multiply the messages
  const float* csr_w = s->weighted ? s->csr_w : nullptr;
  if (s->n_sub > 0)
    HG_LAUNCH("spmm_fwd", (k_spmm_fwd<D, T>), dim3(wave_grid(s->n_sub)), dim3(256), 0, st, s->n_sub, R,
              (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col, pv.csr_slot, csr_w, (const T*)w.Y, (const T*)w.Yself, Hin,
              Hout, mask, L->relu, L->residual);
  if (s->plan_fwd_heavy > 0) {
    HG_LAUNCH("spmm_fwd_part", (k_spmm_fwd_part<D, T>), dim3(wave_grid(s->plan_fwd_parts)), dim3(256), 0, st,
              (int64_t)s->plan_fwd_parts, pv.fwd_items, R, (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col,
              pv.csr_slot, csr_w, (const T*)w.Y, w.part);
    HG_LAUNCH("spmm_fwd_merge", (k_spmm_fwd_merge<D, T>), dim3(wave_grid(s->plan_fwd_heavy)), dim3(256), 0, st,
              (int64_t)s->plan_fwd_heavy, pv.fwd_heavy, (const float*)w.part, (const T*)w.Yself, Hin, Hout, mask,
              L->relu, L->residual);
  }
  return HG_OK;
}

template <int D, class T>
int layer_bwd_impl(const hg_subgraph* s, const hg_layer_desc* L, const T* Hin, const float* W_rel,
                   const float* W_self, const uint32_t* mask, const T* G, T* dHin, float* dW_rel,
                   float* dW_self, float* dbias, int acc, void* ws, size_t ws_bytes, hipStream_t st) {
  Arena a(ws, ws_bytes);
  BwdWs<D, T> w;
  w.layout(a, s);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "backward workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  const int32_t R = s->n_rel;
  const PlanView pv = plan_view(s);
  // float32 rows: dH accumulates in place; bfloat16 rows: in a float32
  // accumulator, each row written once in bf16 by the last pass reaching it
  constexpr bool kBf = sizeof(T) == 2;
  float* dacc = kBf ? w.dhacc : reinterpret_cast<float*>(dHin);
  const int32_t* cptr = (const int32_t*)s->csc_ptr;
  // (c) dH = G (residual) + dZ W_self^T per type, float32 MFMA; the A-operand
  // load forms dZ = G * mask and also writes it out for the SpMM and dW_self
  for (int t = 0; t < s->n_ntype; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    LoadMasked<D, T> la{G, mask, rows_contig(lo), w.dZ};
    // the residual addend G is A's own rows before masking (float32 rows of
    // d = 128 hold them with 256 VGPRs, one block per compute unit)
    constexpr bool kFromA = true;
    if constexpr (kBf) {
      StoreLast<D, T, kFromA> ep{reinterpret_cast<bf16_t*>(dHin), dacc, rows_contig(lo), nullptr,
                                 L->residual ? G : nullptr, cptr, R, -1};
      HG_TRY((rows_f32<D, true>("gemm_bwd_dx_self", hi - lo, W_self + (int64_t)t * D * D, la, ep, st)));
    } else {
      StoreRows<D, float, T, kFromA> ep{dacc, rows_contig(lo), nullptr, L->residual ? G : nullptr};
      HG_TRY((rows_f32<D, true>("gemm_bwd_dx_self", hi - lo, W_self + (int64_t)t * D * D, la, ep, st)));
    }
  }
  // (b) transposed SpMM into float32 dY
  if (s->plan_items > 0)
    HG_LAUNCH("spmm_bwd", (k_spmm_bwd<D, T, float>), dim3(wave_grid(s->plan_items)), dim3(256), 0, st,
              (int64_t)s->plan_items, pv.items, (const int32_t*)s->csc_row, (const float*)s->csc_scale,
              (const T*)w.dZ, w.dY, w.part);
  if (s->plan_heavy > 0)
    HG_LAUNCH("spmm_bwd_reduce", (k_heavy_reduce<D, float>), dim3(wave_grid(s->plan_heavy)), dim3(256), 0, st,
              (int64_t)s->plan_heavy, pv.heavy, (const double*)w.part, w.dY);
  // (c) dH += dY_r W_r^T per relation, in relation order
  std::vector<int64_t> act_off(R + 1, 0);
  for (int r = 0; r < R; ++r) act_off[r + 1] = act_off[r] + s->n_active[r];
  for (int r = 0; r < R; ++r) {
    const int64_t n = s->n_active[r], off = act_off[r];
    LoadRows<D, float> la{w.dY, rows_list(pv.act_slot + off)};
    if constexpr (kBf) {
      StoreLast<D, float> ep{reinterpret_cast<bf16_t*>(dHin), dacc, rows_list(pv.active + off), nullptr, dacc, cptr,
                             R, r};
      HG_TRY((rows_f32<D, true>("gemm_bwd_dx_rel", n, W_rel + (int64_t)r * D * D, la, ep, st)));
    } else {
      StoreRows<D, float, float> ep{dacc, rows_list(pv.active + off), nullptr, dacc};
      HG_TRY((rows_f32<D, true>("gemm_bwd_dx_rel", n, W_rel + (int64_t)r * D * D, la, ep, st)));
    }
  }
  // (c) weight gradients, split-K
  for (int t = 0; t < s->n_ntype; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    LoadRows<D, T> la{Hin, rows_contig(lo)};
    LoadRows<D, T> lb{w.dZ, rows_contig(lo)};
    HG_TRY((launch_gemm_tn<D>("gemm_bwd_dw_self", hi - lo, la, lb, w.splitk, w.colsum,
                              dW_self + (int64_t)t * D * D, dbias ? dbias + (int64_t)t * D : nullptr, acc, st)));
  }
  for (int r = 0; r < R; ++r) {
    const int64_t n = s->n_active[r], off = act_off[r];
    LoadRows<D, T> la{Hin, rows_list(pv.active + off)};
    LoadRows<D, float> lb{w.dY, rows_list(pv.act_slot + off)};
    HG_TRY((launch_gemm_tn<D>("gemm_bwd_dw_rel", n, la, lb, w.splitk, w.colsum, dW_rel + (int64_t)r * D * D,
                              nullptr, acc, st)));
  }
  return HG_OK;
}

template <template <int, class> class WS>
size_t ws_size(const hg_subgraph* s, const hg_layer_desc* L) {
  Sizer z;
  const bool bf = L->dtype == HG_DTYPE_BF16;
  switch (L->d_in) {
    case 64: if (bf) { WS<64, bf16_t> w; w.layout(z, s); } else { WS<64, float> w; w.layout(z, s); } break;
    case 128: if (bf) { WS<128, bf16_t> w; w.layout(z, s); } else { WS<128, float> w; w.layout(z, s); } break;
    default: if (bf) { WS<256, bf16_t> w; w.layout(z, s); } else { WS<256, float> w; w.layout(z, s); } break;
  }
  return z.used + 256;
}

}  // namespace

}  // namespace hg

using namespace hg;

extern "C" size_t hg_layer_saved_size(const hg_subgraph* s, const hg_layer_desc* L) {
  if (!s || !L || L->d_out <= 0) return 0;
  return sizeof(uint32_t) * (size_t)s->n_sub * (size_t)((L->d_out + 31) / 32);
}

extern "C" size_t hg_layer_fwd_workspace_size(const hg_subgraph* s, const hg_layer_desc* L) {
  if (validate_layer(s, L) != HG_OK) return 0;
  return ws_size<FwdWs>(s, L);
}

extern "C" size_t hg_layer_bwd_workspace_size(const hg_subgraph* s, const hg_layer_desc* L) {
  if (validate_layer(s, L) != HG_OK) return 0;
  return ws_size<BwdWs>(s, L);
}

extern "C" int hg_layer_fwd(const hg_subgraph* s, const hg_layer_desc* L, const void* H_in,
                            const float* W_rel, const float* W_self, const float* bias, void* H_out,
                            void* saved, void* ws, size_t ws_bytes, void* stream) {
  HG_TRY(validate_layer(s, L));
  if (s->n_sub > 0 && (!H_in || !H_out || !saved || !W_rel || !W_self))
    return fail(HG_ERR_ARG, "null layer argument");
  if (H_in == H_out && s->n_sub > 0) return fail(HG_ERR_ARG, "H_out must not alias H_in");
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t* m = (uint32_t*)saved;
  if (L->dtype == HG_DTYPE_BF16) {
    const bf16_t* hi = (const bf16_t*)H_in;
    bf16_t* ho = (bf16_t*)H_out;
    if (L->d_in == 64) return layer_fwd_impl<64, bf16_t>(s, L, hi, W_rel, W_self, bias, ho, m, ws, ws_bytes, st);
    if (L->d_in == 128) return layer_fwd_impl<128, bf16_t>(s, L, hi, W_rel, W_self, bias, ho, m, ws, ws_bytes, st);
    return layer_fwd_impl<256, bf16_t>(s, L, hi, W_rel, W_self, bias, ho, m, ws, ws_bytes, st);
  }
  const float* hi = (const float*)H_in;
  float* ho = (float*)H_out;
  if (L->d_in == 64) return layer_fwd_impl<64, float>(s, L, hi, W_rel, W_self, bias, ho, m, ws, ws_bytes, st);
  if (L->d_in == 128) return layer_fwd_impl<128, float>(s, L, hi, W_rel, W_self, bias, ho, m, ws, ws_bytes, st);
  return layer_fwd_impl<256, float>(s, L, hi, W_rel, W_self, bias, ho, m, ws, ws_bytes, st);
}

extern "C" int hg_layer_bwd(const hg_subgraph* s, const hg_layer_desc* L, const void* H_in,
                            const float* W_rel, const float* W_self, const void* saved,
                            const void* dH_out, void* dH_in, float* dW_rel, float* dW_self,
                            float* dbias, int32_t accumulate, void* ws, size_t ws_bytes, void* stream) {
  HG_TRY(validate_layer(s, L));
  if (accumulate != 0 && accumulate != 1) return fail(HG_ERR_ARG, "accumulate must be 0 or 1");
  if (!W_rel || !W_self || !dW_rel || !dW_self) return fail(HG_ERR_ARG, "null weight argument");
  if (s->n_sub > 0 && (!H_in || !saved || !dH_out || !dH_in)) return fail(HG_ERR_ARG, "null layer argument");
  if (dH_in == dH_out && s->n_sub > 0) return fail(HG_ERR_ARG, "dH_in must not alias dH_out");
  hipStream_t st = static_cast<hipStream_t>(stream);
  const uint32_t* m = (const uint32_t*)saved;
  if (L->dtype == HG_DTYPE_BF16) {
    const bf16_t* hi = (const bf16_t*)H_in;
    const bf16_t* g = (const bf16_t*)dH_out;
    bf16_t* dh = (bf16_t*)dH_in;
    if (L->d_in == 64)
      return layer_bwd_impl<64, bf16_t>(s, L, hi, W_rel, W_self, m, g, dh, dW_rel, dW_self, dbias, accumulate, ws, ws_bytes, st);
    if (L->d_in == 128)
      return layer_bwd_impl<128, bf16_t>(s, L, hi, W_rel, W_self, m, g, dh, dW_rel, dW_self, dbias, accumulate, ws, ws_bytes, st);
    return layer_bwd_impl<256, bf16_t>(s, L, hi, W_rel, W_self, m, g, dh, dW_rel, dW_self, dbias, accumulate, ws, ws_bytes, st);
  }
  const float* hi = (const float*)H_in;
  const float* g = (const float*)dH_out;
  float* dh = (float*)dH_in;
  if (L->d_in == 64)
    return layer_bwd_impl<64, float>(s, L, hi, W_rel, W_self, m, g, dh, dW_rel, dW_self, dbias, accumulate, ws, ws_bytes, st);
  if (L->d_in == 128)
    return layer_bwd_impl<128, float>(s, L, hi, W_rel, W_self, m, g, dh, dW_rel, dW_self, dbias, accumulate, ws, ws_bytes, st);
  return layer_bwd_impl<256, float>(s, L, hi, W_rel, W_self, m, g, dh, dW_rel, dW_self, dbias, accumulate, ws, ws_bytes, st);
}
