// hg_align_loss_fwd_bwd: CCA consistency-alignment loss on the overlap batch
// (Section "Cross-Subgraph Consistency Alignment": standardisation,
// invariance, decorrelation and CCA-loss equations) and its gradient.
//
//   (d1) column statistics of X = H[overlap] and Y = H_ref: two-pass mean and
//        variance, fixed-order chunk reduction
//   (d2) Grams Xh^T Xh and Yh^T Yh on MFMA (split-K over the batch, the
//        standardisation applied while loading), L_inv partials, loss scalars
//   (d3) G_Xh = 2 w (Xh - Yh) + 4 lambda_n Xh (Xh^T Xh - I) on MFMA, the
//        standardisation backward, and dH[overlap] += scale * dX (rows are
//        distinct, so no atomics)
#include "hg_internal.h"
#include "hg_mfma.h"

namespace hg {

namespace {

// Per-column sums of f(b, c) over batch rows, one partial row per chunk.
template <int D, class F>
__global__ void __launch_bounds__(256) k_colsum(int64_t m, int64_t rows_per_chunk, F f,
                                                float* __restrict__ partial) {
  constexpr int RPB = 256 / D;
  __shared__ float red[256];
  const int t = threadIdx.x;
  const int c = t % D, ph = t / D;
  const int64_t b0 = (int64_t)blockIdx.x * rows_per_chunk;
  const int64_t b1 = (b0 + rows_per_chunk < m) ? b0 + rows_per_chunk : m;
  float s = 0.f;
  for (int64_t b = b0 + ph; b < b1; b += RPB) s += f(b, c);
  red[t] = s;
  __syncthreads();
  if (t < D) {
    float tot = 0.f;
#pragma unroll
    for (int p = 0; p < RPB; ++p) tot += red[p * D + t];
    partial[(int64_t)blockIdx.x * D + t] = tot;
  }
}

template <int D, class T>
struct FRow {  // value of a gathered / contiguous row
  const T* base;
  RowMap map;
  __device__ __forceinline__ float operator()(int64_t b, int c) const { return Elt<T>::get(base + map(b) * D + c); }
};

template <int D, class T>
struct FCentredSq {
  const T* base;
  RowMap map;
  const float* mu;
  __device__ __forceinline__ float operator()(int64_t b, int c) const {
    const float x = Elt<T>::get(base + map(b) * D + c) - mu[c];
    return x * x;
  }
};

template <int D, class T>
struct FInv {  // w_b (xh - yh)^2
  LoadStd<D, T> x, y;
  const float* w;
  __device__ __forceinline__ float operator()(int64_t b, int c) const {
    const float d = x.at(b, c) - y.at(b, c);
    return (w ? w[b] : 1.f) * d * d;
  }
};

template <int D>
struct FGrad {  // g' = G / sqrt(M)  (gradient w.r.t. the centred, 1/sigma-scaled view)
  const float* G;
  float inv_sqrt_m;
  __device__ __forceinline__ float operator()(int64_t b, int c) const { return G[b * D + c] * inv_sqrt_m; }
};

template <int D, class T>
struct FGradX {  // g' * xt, xt = (x - mu) / sigma
  const float* G;
  float inv_sqrt_m;
  LoadStd<D, T> xt;
  __device__ __forceinline__ float operator()(int64_t b, int c) const {
    return G[b * D + c] * inv_sqrt_m * xt.at(b, c);
  }
};

// mean / sigma / scales from the column sums.
template <int D>
__global__ void k_stats_mean(const float* __restrict__ sum, int64_t m, float* __restrict__ mu) {
  const int c = threadIdx.x;
  if (c < D) mu[c] = sum[c] / (float)m;
}

template <int D>
__global__ void k_stats_sigma(const float* __restrict__ sq, int64_t m, int32_t ddof, float eps,
                              float* __restrict__ inv_sig, float* __restrict__ sc_hat) {
  const int c = threadIdx.x;
  if (c < D) {
    const float var = sq[c] / (float)(m - ddof);
    const float sig = sqrtf(var + eps);
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
__global__ void k_loss_final(const float* __restrict__ inv_cols, float* __restrict__ cx,
                             float* __restrict__ cy, float lambda_n, float* __restrict__ loss3) {
  const int t = threadIdx.x;
  float li = 0.f;
  for (int c = t; c < D; c += 256) li += inv_cols[c];
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
                               const float* __restrict__ inv_sig, const float* __restrict__ S1,
                               const float* __restrict__ S2, int32_t ddof, float scale, const T* base,
                               T* dst, RowMap dmap, int accumulate) {
  const int64_t total = m * D;
  const float inv_m = 1.0f / (float)m;
  const float inv_md = 1.0f / (float)(m - ddof);
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = e / D;
    const int c = (int)(e % D);
    const float g = G[e] * inv_sqrt_m;
    const float dx = inv_sig[c] * (g - S1[c] * inv_m - xt.at(b, c) * S2[c] * inv_md);
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
  float *sum, *mux, *muy, *isx, *isy, *shx, *shy, *cx, *cy, *cpart, *gpart, *invc, *s1, *s2, *gx;
  template <class A>
  void layout(A& a, int64_t m, int64_t nchunks) {
    sum = a.template take<float>(D);
    mux = a.template take<float>(D);
    muy = a.template take<float>(D);
    isx = a.template take<float>(D);
    isy = a.template take<float>(D);
    shx = a.template take<float>(D);
    shy = a.template take<float>(D);
    cx = a.template take<float>(D * D);
    cy = a.template take<float>(D * D);
    cpart = a.template take<float>((nchunks + kSplitGroups + 1) * D);
    gpart = a.template take<float>(splitk_max_chunks() * (int64_t)D * D);
    invc = a.template take<float>(D);
    s1 = a.template take<float>(D);
    s2 = a.template take<float>(D);
    gx = a.template take<float>(m * D);
  }
};

inline int64_t align_chunks(int64_t m) {
  int64_t n = cdiv(m, 256);
  return n < 1024 ? (n > 0 ? n : 1) : 1024;
}

template <int D, class F>
int colsum(const char* name, int64_t m, F f, float* part, float* out, hipStream_t s) {
  const int64_t nch = align_chunks(m);
  const int64_t rpc = cdiv(m, nch);
  HG_LAUNCH(name, (k_colsum<D, F>), dim3((unsigned)nch), dim3(256), 0, s, m, rpc, f, part);
  HG_TRY(reduce_partials(part, nch, (int64_t)D, part + nch * D, out, 0, s));
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
  HG_TRY((colsum<D>("align_stats", m, FRow<D, T>{H, mx}, q.cpart, q.sum, s)));
  HG_LAUNCH("align_mean", k_stats_mean<D>, dim3(1), dim3(256), 0, s, (const float*)q.sum, m, q.mux);
  HG_TRY((colsum<D>("align_stats", m, FCentredSq<D, T>{H, mx, q.mux}, q.cpart, q.sum, s)));
  HG_LAUNCH("align_sigma", k_stats_sigma<D>, dim3(1), dim3(256), 0, s, (const float*)q.sum, m, ddof, eps,
            q.isx, q.shx);
  HG_TRY((colsum<D>("align_stats", m, FRow<D, T>{Href, my}, q.cpart, q.sum, s)));
  HG_LAUNCH("align_mean", k_stats_mean<D>, dim3(1), dim3(256), 0, s, (const float*)q.sum, m, q.muy);
  HG_TRY((colsum<D>("align_stats", m, FCentredSq<D, T>{Href, my, q.muy}, q.cpart, q.sum, s)));
  HG_LAUNCH("align_sigma", k_stats_sigma<D>, dim3(1), dim3(256), 0, s, (const float*)q.sum, m, ddof, eps,
            q.isy, q.shy);
  const LoadStd<D, T> xh{H, mx, q.mux, q.shx}, yh{Href, my, q.muy, q.shy};
  // (d2) Grams and loss
  HG_TRY((launch_gemm_tn<D>("align_gram", m, xh, xh, q.gpart, nullptr, q.cx, nullptr, 0, s)));
  HG_TRY((launch_gemm_tn<D>("align_gram", m, yh, yh, q.gpart, nullptr, q.cy, nullptr, 0, s)));
  HG_TRY((colsum<D>("align_inv", m, FInv<D, T>{xh, yh, w}, q.cpart, q.invc, s)));
  HG_LAUNCH("align_loss", k_loss_final<D>, dim3(1), dim3(256), 0, s, (const float*)q.invc, q.cx, q.cy,
            lambda_n, loss3);
  // (d3) gradient of the local view
  const float inv_sqrt_m = 1.0f / sqrtf((float)m);
  const unsigned ge = (unsigned)(cdiv(m * D, 256) < 65536 ? cdiv(m * D, 256) : 65536);
  {
    GradEpi<D, T> ep{q.gx, xh, yh, w, 4.0f * lambda_n, 2.0f};
    HG_TRY((grad_gemm<D, T>(m, q.cx, xh, ep, s)));
    const LoadStd<D, T> xt{H, mx, q.mux, q.isx};
    HG_TRY((colsum<D>("align_grad_stats", m, FGrad<D>{q.gx, inv_sqrt_m}, q.cpart, q.s1, s)));
    HG_TRY((colsum<D>("align_grad_stats", m, FGradX<D, T>{q.gx, inv_sqrt_m, xt}, q.cpart, q.s2, s)));
    HG_LAUNCH("align_std_backward", (k_std_backward<D, T>), dim3(ge), dim3(256), 0, s, m, (const float*)q.gx,
              inv_sqrt_m, xt, (const float*)q.isx, (const float*)q.s1, (const float*)q.s2, ddof, scale,
              dHbase ? dHbase : (const T*)dH, dH, mx, 1);
  }
  if (dHref) {
    GradEpi<D, T> ep{q.gx, yh, xh, w, 4.0f * lambda_n, 2.0f};
    HG_TRY((grad_gemm<D, T>(m, q.cy, yh, ep, s)));
    const LoadStd<D, T> yt{Href, my, q.muy, q.isy};
    HG_TRY((colsum<D>("align_grad_stats", m, FGrad<D>{q.gx, inv_sqrt_m}, q.cpart, q.s1, s)));
    HG_TRY((colsum<D>("align_grad_stats", m, FGradX<D, T>{q.gx, inv_sqrt_m, yt}, q.cpart, q.s2, s)));
    HG_LAUNCH("align_std_backward", (k_std_backward<D, T>), dim3(ge), dim3(256), 0, s, m, (const float*)q.gx,
              inv_sqrt_m, yt, (const float*)q.isy, (const float*)q.s1, (const float*)q.s2, ddof, scale,
              (const T*)dHref, dHref, my, 0);
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
