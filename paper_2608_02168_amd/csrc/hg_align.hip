// hg_align_loss_fwd_bwd: CCA consistency-alignment loss on the overlap batch
// (Section "Cross-Subgraph Consistency Alignment": standardisation,
// invariance, decorrelation and CCA-loss equations) and its gradient.
//
//   (d1) column statistics of X = H[overlap] and Y = H_ref: sums of x and x^2
//        in float64 in one pass per view (the float64 sums keep the
//        difference Sxx - S^2/M exact to far below float32 rounding),
//        fixed-order chunk reduction
//   (d2) Grams Xh^T Xh and Yh^T Yh on MFMA (split-K over the batch, the
//        standardisation applied while loading), L_inv partials, loss scalars
//   (d3) G_Xh = 2 w (Xh - Yh) + 4 lambda_n Xh (Xh^T Xh - I) on MFMA, the
//        standardisation backward, and dH[overlap] += scale * dX (rows are
//        distinct, so no atomics)
#include "hg_internal.h"
#include "hg_mfma.h"

namespace hg {

namespace {

// Per-column sums over batch rows in float64, one partial row set per chunk.
// A row is D/4 lanes that each read 16 bytes (columns c..c+3); four rows per
// lane are in flight before their values are added; the functor gives NS
// float4 values of row b (NS sums per column).  Partials [chunk][NS][D].
// acc += v in float64; with F::kSquare the second sum takes the float64
// square of the first value (exact for a float32 x).
template <class F, int NS>
__device__ __forceinline__ void add_sums(double (&acc)[NS][4], const f32x4 (&v)[NS]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const double x = (double)v[0][k];
    acc[0][k] += x;
    if constexpr (F::kSquare) {
      acc[1][k] += x * x;
    } else {
#pragma unroll
      for (int q = 1; q < NS; ++q) acc[q][k] += (double)v[q][k];
    }
  }
}

template <int D, int NS, class F>
__global__ void __launch_bounds__(256) k_colsum(int64_t m, int64_t rows_per_chunk, F f,
                                                double* __restrict__ partial) {
  auto add = [](double (&a)[NS][4], const f32x4 (&v)[NS]) { add_sums<F, NS>(a, v); };
  constexpr int TPR = D / 4, RPI = 256 / TPR, U = 4;
  __shared__ double red[NS * 4][256];
  const int t = threadIdx.x;
  const int c = (t % TPR) * 4, ph = t / TPR;
  const int64_t b0 = (int64_t)blockIdx.x * rows_per_chunk;
  const int64_t b1 = (b0 + rows_per_chunk < m) ? b0 + rows_per_chunk : m;
  double acc[NS][4];
#pragma unroll
  for (int q = 0; q < NS; ++q)
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[q][k] = 0.0;
  int64_t b = b0 + ph;
  for (; b + (U - 1) * RPI < b1; b += U * RPI) {
    f32x4 v[U][NS];
#pragma unroll
    for (int u = 0; u < U; ++u) f.at4(b + u * RPI, c, v[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) add(acc, v[u]);
  }
  for (; b < b1; b += RPI) {
    f32x4 v[NS];
    f.at4(b, c, v);
    add(acc, v);
  }
#pragma unroll
  for (int q = 0; q < NS; ++q)
#pragma unroll
    for (int k = 0; k < 4; ++k) red[q * 4 + k][t] = acc[q][k];
  __syncthreads();
  if (t < TPR) {
#pragma unroll
    for (int q = 0; q < NS; ++q)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        double tot = 0.0;
        for (int p = 0; p < RPI; ++p) tot += red[q * 4 + k][p * TPR + t];
        partial[((int64_t)blockIdx.x * NS + q) * D + c + k] = tot;
      }
  }
}

// out[j] = sum of partial[chunk][j] over the chunks in fixed order, j < nj;
// 64 values per block, each of its 4 waves sums a quarter of the chunks.
__global__ void __launch_bounds__(256) k_colsum_total(const double* __restrict__ partial, int64_t nch, int nj,
                                                      double* __restrict__ out) {
  __shared__ double red[4][64];
  const int l = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int j = blockIdx.x * 64 + l;
  const int64_t per = (nch + 3) / 4, lo = q * per, hi = (lo + per < nch) ? lo + per : nch;
  double s = 0.0;
  if (j < nj)
    for (int64_t k = lo; k < hi; ++k) s += partial[k * nj + j];
  red[q][l] = s;
  __syncthreads();
  if (q == 0 && j < nj) out[j] = ((red[0][l] + red[1][l]) + red[2][l]) + red[3][l];
}

template <int D, class T>
struct FMoments {  // x and x^2 of a gathered / contiguous row
  static constexpr int NS = 2;
  static constexpr bool kSquare = true;
  const T* base;
  RowMap map;
  __device__ __forceinline__ void at4(int64_t b, int c, f32x4 (&v)[2]) const {
    v[0] = Elt<T>::load4(base + map(b) * D + c);
    v[1] = v[0];
  }
};

template <int D, class T>
struct FInv {  // w_b (xh - yh)^2
  static constexpr int NS = 1;
  static constexpr bool kSquare = false;
  LoadStd<D, T> x, y;
  const float* w;
  __device__ __forceinline__ void at4(int64_t b, int c, f32x4 (&v)[1]) const {
    const f32x4 d = x.load4(x.rowp(b), c) - y.load4(y.rowp(b), c);
    v[0] = (w ? w[b] : 1.f) * (d * d);
  }
};

template <int D, class T>
struct FGradStats {  // g' = G / sqrt(M) and g' * xt, xt = (x - mu) / sigma
  static constexpr int NS = 2;
  static constexpr bool kSquare = false;
  const float* G;
  float inv_sqrt_m;
  LoadStd<D, T> xt;
  __device__ __forceinline__ void at4(int64_t b, int c, f32x4 (&v)[2]) const {
    const f32x4 g = *reinterpret_cast<const f32x4*>(G + b * D + c) * inv_sqrt_m;
    v[0] = g;
    v[1] = g * xt.load4(xt.rowp(b), c);
  }
};

// mean, 1/sigma and the standardisation scale from the float64 sums S = sum x
// and Q = sum x^2 of each column: var = (Q - S^2/M) / (M - ddof).
template <int D>
__global__ void k_stats(const double* __restrict__ sums, int64_t m, int32_t ddof, float eps, float* __restrict__ mu,
                        float* __restrict__ inv_sig, float* __restrict__ sc_hat) {
  const int c = threadIdx.x;
  if (c < D) {
    const double S = sums[c], Q = sums[D + c];
    const double mean = S / (double)m;
    double var = (Q - S * mean) / (double)(m - ddof);
    var = var > 0.0 ? var : 0.0;
    const float sig = sqrtf((float)var + eps);
    mu[c] = (float)mean;
    inv_sig[c] = 1.0f / sig;
    sc_hat[c] = 1.0f / (sig * sqrtf((float)m));
  }
}

// Fixed-order block sum of n values (one block of 256 threads).
__device__ float block_sum_fixed(float v) {
  __shared__ float red[256];
  red[threadIdx.x] = v;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  const float r = red[0];
  __syncthreads();
  return r;
}

// loss3 and C - I (in place).  inv_cols: per-column L_inv totals [D].
template <int D>
__global__ void k_loss_final(const double* __restrict__ inv_cols, float* __restrict__ cx,
                             float* __restrict__ cy, float lambda_n, float* __restrict__ loss3) {
  const int t = threadIdx.x;
  float li = 0.f;
  for (int c = t; c < D; c += 256) li += (float)inv_cols[c];
  float ld = 0.f;
  for (int e = t; e < D * D; e += 256) {
    const float id = ((e / D) == (e % D)) ? 1.f : 0.f;
    const float a = cx[e] - id, b = cy[e] - id;
    cx[e] = a;
    cy[e] = b;
    ld += a * a + b * b;
  }
  const float L_inv = block_sum_fixed(li);
  const float L_dec = block_sum_fixed(ld);
  if (t == 0) {
    loss3[0] = L_inv;
    loss3[1] = L_dec;
    loss3[2] = L_inv + lambda_n * L_dec;
  }
}

// Epilogue of the gradient GEMM: G[b][c] = 4 lambda_n acc + sign * 2 w_b (xh - yh).
template <int D, class T>
struct GradEpi {
  float* G;
  LoadStd<D, T> self, other;
  const float* w;
  float four_lambda;
  float two_sign;
  __device__ __forceinline__ int64_t row(int64_t b) const { return b; }
  __device__ __forceinline__ float pre(int64_t b, int64_t, int c) const {
    const float diff = self.at(b, c) - other.at(b, c);
    return two_sign * (w ? w[b] : 1.f) * diff;
  }
  __device__ __forceinline__ void store(int64_t b, int64_t, int c, float acc, float pre) const {
    G[b * D + c] = four_lambda * acc + pre;
  }
  __device__ __forceinline__ f32x4 pre4(int64_t b, int64_t, int c) const {
    const auto ps = self.rowp(b);
    const auto po = other.rowp(b);
    const f32x4 diff = self.load4(ps, c) - other.load4(po, c);
    return (two_sign * (w ? w[b] : 1.f)) * diff;
  }
  __device__ __forceinline__ void store4(int64_t b, int64_t, int c, f32x4 acc, f32x4 pre) const {
    *reinterpret_cast<f32x4*>(G + b * D + c) = four_lambda * acc + pre;
  }
};

// dX = (1/sigma)(g' - S1/M - xt * S2/(M - ddof)); dst[row] = scale * dX,
// plus base[row] when accumulate (base may be dst itself).
template <int D, class T>
__global__ void k_std_backward(int64_t m, const float* __restrict__ G, float inv_sqrt_m, LoadStd<D, T> xt,
                               const float* __restrict__ inv_sig, const double* __restrict__ S12, int32_t ddof,
                               float scale, const T* base, T* dst, RowMap dmap, int accumulate) {
  const int64_t total = m * D;
  const float inv_m = 1.0f / (float)m;
  const float inv_md = 1.0f / (float)(m - ddof);
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = e / D;
    const int c = (int)(e % D);
    const float g = G[e] * inv_sqrt_m;
    const float dx = inv_sig[c] * (g - (float)S12[c] * inv_m - xt.at(b, c) * (float)S12[D + c] * inv_md);
    const int64_t o = dmap(b) * D + c;
    const float v = (accumulate ? Elt<T>::get(base + o) : 0.f) + scale * dx;
    if constexpr (sizeof(T) == 4) {
      dst[o] = v;
    } else {
      dst[o] = f2bf(v);
    }
  }
}

template <int D>
struct AlignWs {
  float *mux, *muy, *isx, *isy, *shx, *shy, *cx, *cy, *gpart, *gx;
  double *cpart, *sums;
  template <class A>
  void layout(A& a, int64_t m, int64_t nchunks) {
    cpart = a.template take<double>(nchunks * 2 * D);
    sums = a.template take<double>(2 * D);
    mux = a.template take<float>(D);
    muy = a.template take<float>(D);
    isx = a.template take<float>(D);
    isy = a.template take<float>(D);
    shx = a.template take<float>(D);
    shy = a.template take<float>(D);
    cx = a.template take<float>(D * D);
    cy = a.template take<float>(D * D);
    gpart = a.template take<float>(splitk_max_chunks() * (int64_t)D * D);
    gx = a.template take<float>(m * D);
  }
};

inline int64_t align_chunks(int64_t m) {
  int64_t n = cdiv(m, 256);
  return n < 1024 ? (n > 0 ? n : 1) : 1024;
}

// out [F::NS][D] (float64) = column sums of f over the m batch rows.
template <int D, class F>
int colsum(const char* name, int64_t m, F f, double* part, double* out, hipStream_t s) {
  const int64_t nch = align_chunks(m);
  const int64_t rpc = cdiv(m, nch);
  constexpr int NJ = F::NS * D;
  HG_LAUNCH(name, (k_colsum<D, F::NS, F>), dim3((unsigned)nch), dim3(256), 0, s, m, rpc, f, part);
  HG_LAUNCH(name, k_colsum_total, dim3((unsigned)cdiv(NJ, 64)), dim3(256), 0, s, (const double*)part, nch, NJ, out);
  return HG_OK;
}

template <int D, class T, class ALoad, class Epi>
int grad_gemm(int64_t m, const float* W, ALoad la, Epi ep, hipStream_t s) {
  return launch_gemm_rows<D, false>("align_grad_gemm", m, W, la, ep, s);
}

template <int D, class T>
int align_impl(int64_t m, const T* H, const int32_t* overlap, const T* Href, const float* w, float lambda_n,
               float scale, float eps, int32_t ddof, float* loss3, T* dH, const T* dHbase, T* dHref, void* ws,
               size_t ws_bytes, hipStream_t s) {
  Arena a(ws, ws_bytes);
  AlignWs<D> q;
  q.layout(a, m, align_chunks(m));
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "alignment workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  const RowMap mx = rows_list(overlap), my = rows_contig(0);
  // (d1) statistics
  HG_TRY((colsum<D>("align_stats", m, FMoments<D, T>{H, mx}, q.cpart, q.sums, s)));
  HG_LAUNCH("align_sigma", k_stats<D>, dim3(1), dim3(256), 0, s, (const double*)q.sums, m, ddof, eps, q.mux, q.isx,
            q.shx);
  HG_TRY((colsum<D>("align_stats", m, FMoments<D, T>{Href, my}, q.cpart, q.sums, s)));
  HG_LAUNCH("align_sigma", k_stats<D>, dim3(1), dim3(256), 0, s, (const double*)q.sums, m, ddof, eps, q.muy, q.isy,
            q.shy);
  const LoadStd<D, T> xh{H, mx, q.mux, q.shx}, yh{Href, my, q.muy, q.shy};
  // (d2) Grams and loss
  HG_TRY((launch_gemm_tn<D>("align_gram", m, xh, xh, q.gpart, nullptr, q.cx, nullptr, 0, s)));
  HG_TRY((launch_gemm_tn<D>("align_gram", m, yh, yh, q.gpart, nullptr, q.cy, nullptr, 0, s)));
  HG_TRY((colsum<D>("align_inv", m, FInv<D, T>{xh, yh, w}, q.cpart, q.sums, s)));
  HG_LAUNCH("align_loss", k_loss_final<D>, dim3(1), dim3(256), 0, s, (const double*)q.sums, q.cx, q.cy,
            lambda_n, loss3);
  // (d3) gradient of the local view
  const float inv_sqrt_m = 1.0f / sqrtf((float)m);
  const unsigned ge = (unsigned)(cdiv(m * D, 256) < 65536 ? cdiv(m * D, 256) : 65536);
  {
    GradEpi<D, T> ep{q.gx, xh, yh, w, 4.0f * lambda_n, 2.0f};
    HG_TRY((grad_gemm<D, T>(m, q.cx, xh, ep, s)));
    const LoadStd<D, T> xt{H, mx, q.mux, q.isx};
    HG_TRY((colsum<D>("align_grad_stats", m, FGradStats<D, T>{q.gx, inv_sqrt_m, xt}, q.cpart, q.sums, s)));
    HG_LAUNCH("align_std_backward", (k_std_backward<D, T>), dim3(ge), dim3(256), 0, s, m, (const float*)q.gx,
              inv_sqrt_m, xt, (const float*)q.isx, (const double*)q.sums, ddof, scale,
              dHbase ? dHbase : (const T*)dH, dH, mx, 1);
  }
  if (dHref) {
    GradEpi<D, T> ep{q.gx, yh, xh, w, 4.0f * lambda_n, 2.0f};
    HG_TRY((grad_gemm<D, T>(m, q.cy, yh, ep, s)));
    const LoadStd<D, T> yt{Href, my, q.muy, q.isy};
    HG_TRY((colsum<D>("align_grad_stats", m, FGradStats<D, T>{q.gx, inv_sqrt_m, yt}, q.cpart, q.sums, s)));
    HG_LAUNCH("align_std_backward", (k_std_backward<D, T>), dim3(ge), dim3(256), 0, s, m, (const float*)q.gx,
              inv_sqrt_m, yt, (const float*)q.isy, (const double*)q.sums, ddof, scale, (const T*)dHref, dHref, my,
              0);
  }
  return HG_OK;
}

}  // namespace

}  // namespace hg

using namespace hg;

extern "C" size_t hg_align_workspace_size(int64_t M, int32_t d) {
  if (M < 0) return 0;
  Sizer z;
  if (d == 64) {
    AlignWs<64> w;
    w.layout(z, M, align_chunks(M));
  } else if (d == 128) {
    AlignWs<128> w;
    w.layout(z, M, align_chunks(M));
  } else if (d == 256) {
    AlignWs<256> w;
    w.layout(z, M, align_chunks(M));
  } else {
    return 0;
  }
  return z.used + 256;
}

extern "C" int hg_align_loss_fwd_bwd(int64_t M, int32_t d, int32_t dtype, int64_t n_rows, const void* H,
                                     const int32_t* overlap, const void* H_ref, const float* w,
                                     float lambda_n, float scale, float eps, int32_t ddof, float* loss3,
                                     void* dH, const void* dH_base, void* dH_ref, void* ws, size_t ws_bytes,
                                     void* stream) {
  if (M < 0 || n_rows < 0) return fail(HG_ERR_ARG, "negative size");
  if (!loss3) return fail(HG_ERR_ARG, "null loss3");
  if (dtype != HG_DTYPE_F32 && dtype != HG_DTYPE_BF16) return fail(HG_ERR_ARG, "dtype %d", dtype);
  if (d != 64 && d != 128 && d != 256)
    return fail(HG_ERR_UNSUPPORTED, "alignment supports d in {64, 128, 256}, got %d", d);
  if (ddof < 0) return fail(HG_ERR_ARG, "ddof < 0");
  if (!(eps >= 0.f)) return fail(HG_ERR_ARG, "eps must be >= 0");
  if (M > n_rows) return fail(HG_ERR_ARG, "M %lld > n_rows %lld", (long long)M, (long long)n_rows);
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (M == 0) return fill_f32(loss3, 0.f, 3, s);
  if (M <= ddof) return fail(HG_ERR_ARG, "M %lld <= ddof %d", (long long)M, ddof);
  if (!H || !overlap || !H_ref || !dH) return fail(HG_ERR_ARG, "null alignment argument");
  if (dtype == HG_DTYPE_BF16) {
    const bf16_t *h = (const bf16_t*)H, *r = (const bf16_t*)H_ref;
    bf16_t *dh = (bf16_t*)dH, *dr = (bf16_t*)dH_ref;
    const bf16_t* db = (const bf16_t*)dH_base;
    if (d == 64) return align_impl<64, bf16_t>(M, h, overlap, r, w, lambda_n, scale, eps, ddof, loss3, dh, db, dr, ws, ws_bytes, s);
    if (d == 128) return align_impl<128, bf16_t>(M, h, overlap, r, w, lambda_n, scale, eps, ddof, loss3, dh, db, dr, ws, ws_bytes, s);
    return align_impl<256, bf16_t>(M, h, overlap, r, w, lambda_n, scale, eps, ddof, loss3, dh, db, dr, ws, ws_bytes, s);
  }
  const float *h = (const float*)H, *r = (const float*)H_ref;
  float *dh = (float*)dH, *dr = (float*)dH_ref;
  const float* db = (const float*)dH_base;
  if (d == 64) return align_impl<64, float>(M, h, overlap, r, w, lambda_n, scale, eps, ddof, loss3, dh, db, dr, ws, ws_bytes, s);
  if (d == 128) return align_impl<128, float>(M, h, overlap, r, w, lambda_n, scale, eps, ddof, loss3, dh, db, dr, ws, ws_bytes, s);
  return align_impl<256, float>(M, h, overlap, r, w, lambda_n, scale, eps, ddof, loss3, dh, db, dr, ws, ws_bytes, s);
}
