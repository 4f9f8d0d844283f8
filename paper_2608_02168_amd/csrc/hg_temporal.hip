// The temporal module of the encoder ("Temporal Graph Learning"): attention
// over the w previous states of a node (E12) and the GRU update (E13).
//
//   u_k = tanh(c_k Q^T), s_k = r . u_k, a = softmax_k(s), Ht = sum_k a_k c_k
//   g_r = sigmoid(h Wi0 + bi0 + Ht Wh0 + bh0), g_z = sigmoid(h Wi1 + bi1 + Ht Wh1 + bh1)
//   g_n = tanh(h Wi2 + bi2 + g_r * (Ht Wh2 + bh2)),  H = (1 - g_z) g_n + g_z Ht
//
// One wave owns 16 rows at a time.  Every row-sized quantity stays in
// registers in the MFMA output layout (lane (c, g) holds row c, columns
// 16 b + 4 g .. + 3 of column block b), which is also the layout the MFMA
// takes its row operand in, so one product feeds the next without a trip
// through LDS.  The seven 64 x 64 weights sit in LDS row-major with a row
// pitch of 68 floats: a lane reads a fragment of W as four 4-byte words
// (op(W) = W) and a fragment of W^T as one 16-byte word (op(W) = W^T), both
// without bank conflicts, so one copy serves products with W and with W^T.
//
// The backward recomputes the forward in registers (nothing is saved between
// the two calls), forms dh, dHt and dC_k in the same pass and writes the gate
// and score gradients it needs for the weight gradients, which are
// deterministic split-K reductions (gemm_tn) over the rows.
#include "hg_mfma.h"

namespace hg {
namespace {

constexpr int kTD = 64;          // state width d
constexpr int kTP = 68;          // LDS row pitch (floats) of a staged 64 x 64 matrix
constexpr int kTMaxW = 4;        // longest context
constexpr int kTThreads = 512;
constexpr int kTWaves = kTThreads / 64;
constexpr int kTMat = kTD * kTP;
constexpr int kTVec = 7 * kTMat;  // then r, bi0 + bh0, bi1 + bh1, bi2, bh2
constexpr int kTUnscale = kTVec + 5 * kTD;  // then the 7 matrices' unscale factors
constexpr size_t kTLds = sizeof(float) * (7 * kTMat + 5 * kTD + 8);

struct TParams {
  const float *Q, *r, *Wi, *bi, *Wh, *bh;
};
template <class T>
struct TCtx {
  const T* c[kTMaxW];
};
template <class T>
struct TCtxOut {
  T* c[kTMaxW];
};

// LDS: Q, Wi[0..2], Wh[0..2] (row-major, pitch kTP), each scaled by the
// power of two that brings its largest magnitude into [2^14, 2^15) and held
// as split-fp16 pairs (one 32-bit word per weight: the fp16 high part, then
// the fp16 remainder; see t_gemm), then the vectors, then the 7 factors that
// undo the scalings.
__device__ __forceinline__ void t_stage(float* lds, const TParams& p) {
  constexpr int kDD = kTD * kTD;
  __shared__ float wmax[kTWaves][7];
  auto src_of = [&](int m) { return m == 0 ? p.Q : (m < 4 ? p.Wi + (m - 1) * kDD : p.Wh + (m - 4) * kDD); };
  {
    // largest |w| of each matrix: wave w reduces matrix m over its lanes,
    // the block over its waves
    const int wv = threadIdx.x >> 6, l = threadIdx.x & 63;
    for (int m = 0; m < 7; ++m) {
      const float* src = src_of(m);
      float mx = 0.f;
      for (int e = wv * 64 + l; e < kDD; e += kTThreads) mx = fmaxf(mx, fabsf(src[e]));
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
      if (l == 0) wmax[wv][m] = mx;
    }
  }
  __syncthreads();
  uint32_t* wl = reinterpret_cast<uint32_t*>(lds);
  for (int e = threadIdx.x; e < 7 * kDD; e += kTThreads) {
    const int m = e / kDD, ij = e - m * kDD;
    float mx = wmax[0][m];
#pragma unroll
    for (int q = 1; q < kTWaves; ++q) mx = fmaxf(mx, wmax[q][m]);
    // the scaled weight as its fp16 high part (low half) and the fp16
    // remainder (high half), as split8 forms them
    const float v = src_of(m)[ij] * split_scale(split_exp(mx));
    const auto hp = __builtin_amdgcn_cvt_pkrtz(v, 0.f);
    const auto lp = __builtin_amdgcn_cvt_pkrtz(v - (float)hp[0], 0.f);
    wl[m * kTMat + (ij / kTD) * kTP + (ij % kTD)] =
        (__builtin_bit_cast(uint32_t, hp) & 0xFFFFu) | (__builtin_bit_cast(uint32_t, lp) << 16);
  }
  if (threadIdx.x < 7) {
    float mx = wmax[0][threadIdx.x];
#pragma unroll
    for (int q = 1; q < kTWaves; ++q) mx = fmaxf(mx, wmax[q][threadIdx.x]);
    lds[kTUnscale + threadIdx.x] = split_unscale(split_exp(mx));
  }
  float* v = lds + kTVec;
  for (int c = threadIdx.x; c < kTD; c += kTThreads) {
    const float bi0 = p.bi ? p.bi[c] : 0.f, bi1 = p.bi ? p.bi[kTD + c] : 0.f, bi2 = p.bi ? p.bi[2 * kTD + c] : 0.f;
    const float bh0 = p.bh ? p.bh[c] : 0.f, bh1 = p.bh ? p.bh[kTD + c] : 0.f, bh2 = p.bh ? p.bh[2 * kTD + c] : 0.f;
    v[c] = p.r[c];
    v[kTD + c] = bi0 + bh0;
    v[2 * kTD + c] = bi1 + bh1;
    v[3 * kTD + c] = bi2;
    v[4 * kTD + c] = bh2;
  }
  __syncthreads();
}

__device__ __forceinline__ f32x4 t_vec4(const float* v, int col) { return *reinterpret_cast<const f32x4*>(v + col); }

// acc += x . op(M) for the 64 x 64 matrix M = matrix mat in LDS (scaled, see
// t_stage; its factor undoes the scaling) on the split-fp16 MFMA (v_mfma_f32_16x16x32_f16,
// three products per K block: the high parts of both factors and each
// factor's remainder against the other's high part, as in the row GEMMs).
// The row is scaled by the power of two of its largest magnitude (the four
// lanes of row c agree by two xor shuffles).  K block kb2 of 32 takes the
// lane's columns 16 (2 kb2) + 4 g .. + 3 (slots 0-3) and 16 (2 kb2 + 1) +
// 4 g .. + 3 (slots 4-7); lane (c, g) supplies op(M)[k][16 nb + c] for the
// same k and receives row c, columns 16 nb + 4 g .. + 3, the layout x is
// held in, so one product feeds the next.  op(M) = M is read as 8 words
// down a column, op(M) = M^T as two 16-byte words along a row (pitch 68:
// neither conflicts); each word holds a weight's two fp16 parts, which are
// regrouped into the MFMA's high-part and remainder operands.
template <bool kTrans>
__device__ __forceinline__ void t_gemm(const float* lds, int mat, const f32x4 (&x)[4], f32x4 (&acc)[4], int g,
                                       int c) {
  const uint32_t* M = reinterpret_cast<const uint32_t*>(lds) + mat * kTMat;
  const float uw = lds[kTUnscale + mat];
  float mx = 0.f;
#pragma unroll
  for (int b = 0; b < 4; ++b)
#pragma unroll
    for (int v = 0; v < 4; ++v) mx = fmaxf(mx, fabsf(x[b][v]));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  const uint32_t ex = split_exp(mx);
  const float sx = split_scale(ex), ux = split_unscale(ex);
  uint4 xh[2], xl[2];
#pragma unroll
  for (int kb2 = 0; kb2 < 2; ++kb2) {
    float v[8];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      v[q] = x[2 * kb2][q] * sx;
      v[4 + q] = x[2 * kb2 + 1][q] * sx;
    }
    split8(v, xh[kb2], xl[kb2]);
  }
  f32x4 t[4];
#pragma unroll
  for (int nb = 0; nb < 4; ++nb) t[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      // each fragment is read and split right before its MFMAs (hoisting
      // them all would exhaust the registers)
      __builtin_amdgcn_sched_barrier(0);
      uint32_t w[8];
      if constexpr (kTrans) {
        const uint32_t* q = M + (16 * nb + c) * kTP + 32 * kb2 + 4 * g;
        const uint4 a = *reinterpret_cast<const uint4*>(q), b = *reinterpret_cast<const uint4*>(q + 16);
        w[0] = a.x; w[1] = a.y; w[2] = a.z; w[3] = a.w;
        w[4] = b.x; w[5] = b.y; w[6] = b.z; w[7] = b.w;
      } else {
        const uint32_t* q = M + (32 * kb2 + 4 * g) * kTP + 16 * nb + c;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
          w[s] = q[s * kTP];
          w[4 + s] = q[(16 + s) * kTP];
        }
      }
      uint32_t h[4], r[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        h[q] = (w[2 * q] & 0xFFFFu) | (w[2 * q + 1] << 16);
        r[q] = (w[2 * q] >> 16) | (w[2 * q + 1] & 0xFFFF0000u);
      }
      const uint4 wh{h[0], h[1], h[2], h[3]}, wl{r[0], r[1], r[2], r[3]};
      t[nb] = mfma_f16(wh, xh[kb2], t[nb]);
      t[nb] = mfma_f16(wh, xl[kb2], t[nb]);
      t[nb] = mfma_f16(wl, xh[kb2], t[nb]);
    }
  }
#pragma unroll
  for (int nb = 0; nb < 4; ++nb)
#pragma unroll
    for (int v = 0; v < 4; ++v) acc[nb][v] += (t[nb][v] * ux) * uw;
}

template <class T>
__device__ __forceinline__ void t_load(const T* base, int64_t row, int g, f32x4 (&x)[4]) {
  const T* p = base + row * kTD + 4 * g;
#pragma unroll
  for (int b = 0; b < 4; ++b) x[b] = Elt<T>::load4(p + 16 * b);
}

template <class T>
__device__ __forceinline__ void t_store(T* base, int64_t row, int g, const f32x4 (&x)[4]) {
  T* p = base + row * kTD + 4 * g;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    if constexpr (sizeof(T) == 4) {
      *reinterpret_cast<f32x4*>(p + 16 * b) = x[b];
    } else {
      *reinterpret_cast<uint2*>(p + 16 * b) = uint2{pack2bf(x[b][0], x[b][1]), pack2bf(x[b][2], x[b][3])};
    }
  }
}

__device__ __forceinline__ void t_zero(f32x4 (&x)[4]) {
#pragma unroll
  for (int b = 0; b < 4; ++b) x[b] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// The sum over the four lanes (c, 0..3) that share row c.
__device__ __forceinline__ float t_rowsum(float v) {
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

__device__ __forceinline__ float t_sigmoid(float x) { return __builtin_amdgcn_rcpf(1.f + __expf(-x)); }

// tanh x = sign(x) (1 - 2 / (exp(2|x|) + 1)); exp overflows to inf for large
// |x|, which gives exactly +-1.
__device__ __forceinline__ float t_tanh(float x) {
  const float e = __expf(2.f * fabsf(x));
  return copysignf(1.f - 2.f * __builtin_amdgcn_rcpf(e + 1.f), x);
}

// E12 for the lane's row: u_k = tanh(c_k Q^T), a = softmax(r . u_k), Ht.
template <int W, int WA>
__device__ __forceinline__ void t_attend(const float* lds, const float* rv, const f32x4 (&cx)[WA][4], float (&a)[WA],
                                         f32x4 (&ht)[4], int g, int c) {
  t_zero(ht);
  if constexpr (W > 0) {
    float s[WA];
#pragma unroll
    for (int k = 0; k < W; ++k) {
      f32x4 acc[4];
      t_zero(acc);
      t_gemm<true>(lds, 0, cx[k], acc, g, c);
      float part = 0.f;
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const f32x4 r4 = t_vec4(rv, 16 * b + 4 * g);
#pragma unroll
        for (int v = 0; v < 4; ++v) part += r4[v] * t_tanh(acc[b][v]);
      }
      s[k] = t_rowsum(part);
    }
    float m = s[0];
#pragma unroll
    for (int k = 1; k < W; ++k) m = fmaxf(m, s[k]);
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < W; ++k) {
      a[k] = __expf(s[k] - m);
      sum += a[k];
    }
    const float inv = 1.f / sum;
#pragma unroll
    for (int k = 0; k < W; ++k) {
      a[k] *= inv;
#pragma unroll
      for (int b = 0; b < 4; ++b) ht[b] += a[k] * cx[k][b];
    }
  }
}

// The gate pre-activations without biases: ar = h Wi0 + Ht Wh0,
// az = h Wi1 + Ht Wh1, ain = h Wi2, ahn = Ht Wh2.
template <int W>
__device__ __forceinline__ void t_gates(const float* lds, const f32x4 (&x)[4], const f32x4 (&ht)[4],
                                        f32x4 (&ar)[4], f32x4 (&az)[4], f32x4 (&ain)[4], f32x4 (&ahn)[4], int g,
                                        int c) {
  t_zero(ar);
  t_zero(az);
  t_zero(ain);
  t_zero(ahn);
  t_gemm<false>(lds, 1, x, ar, g, c);
  t_gemm<false>(lds, 2, x, az, g, c);
  t_gemm<false>(lds, 3, x, ain, g, c);
  if constexpr (W > 0) {
    t_gemm<false>(lds, 4, ht, ar, g, c);
    t_gemm<false>(lds, 5, ht, az, g, c);
    t_gemm<false>(lds, 6, ht, ahn, g, c);
  }
}

template <int W, class T>
__global__ void __launch_bounds__(kTThreads) k_temporal_fwd(int64_t n, const T* __restrict__ h, TCtx<T> C,
                                                            TParams p, T* __restrict__ H) {
  constexpr int WA = W > 0 ? W : 1;
  extern __shared__ float lds[];
  t_stage(lds, p);
  const float* vec = lds + kTVec;
  const int l = lane64(), g = l >> 4, c = l & 15;
  const int64_t ntiles = (n + 15) / 16;
  const int64_t nw = (int64_t)gridDim.x * kTWaves;
  for (int64_t t = (int64_t)blockIdx.x * kTWaves + (threadIdx.x >> 6); t < ntiles; t += nw) {
    const int64_t i = 16 * t + c;
    const bool live = i < n;
    const int64_t ri = live ? i : n - 1;  // a row past the end reads the last row and stores nothing
    f32x4 x[4], cx[WA][4], ht[4];
    float a[WA];
    t_load(h, ri, g, x);
#pragma unroll
    for (int k = 0; k < W; ++k) t_load(C.c[k], ri, g, cx[k]);
    t_attend<W, WA>(lds, vec, cx, a, ht, g, c);
    f32x4 ar[4], az[4], ain[4], ahn[4];
    t_gates<W>(lds, x, ht, ar, az, ain, ahn, g, c);
    f32x4 out[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int col = 16 * b + 4 * g;
      const f32x4 br = t_vec4(vec + kTD, col), bz = t_vec4(vec + 2 * kTD, col);
      const f32x4 bin = t_vec4(vec + 3 * kTD, col), bhn = t_vec4(vec + 4 * kTD, col);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float rg = t_sigmoid(ar[b][v] + br[v]);
        const float zg = t_sigmoid(az[b][v] + bz[v]);
        const float ng = t_tanh(ain[b][v] + bin[v] + rg * (ahn[b][v] + bhn[v]));
        out[b][v] = (1.f - zg) * ng + zg * ht[b][v];
      }
    }
    if (live) t_store(H, i, g, out);
  }
}

// Backward.  Per row: the gate gradients dG = [d g_r-pre | d g_z-pre |
// d g_n-pre (input side) | d (Ht Wh2 + bh2)] (fp32 [n, 4, 64]), Ht (fp32
// [n, 64]), dpre_k = ds_k r (1 - u_k^2) (fp32 [w, n, 64]); dh = sum of the
// input-side gate gradients times Wi^T; dC_k += a_k dHt + dpre_k Q; per block
// the partial sums of dr = sum ds_k u_k (fp32 [gridDim.x, 64]).
template <int W, class T>
__global__ void __launch_bounds__(kTThreads) k_temporal_bwd(int64_t n, const T* __restrict__ h, TCtx<T> C,
                                                            TParams p, const T* __restrict__ dH,
                                                            T* __restrict__ dh, TCtxOut<T> dC,
                                                            float* __restrict__ Ht_out, float* __restrict__ dG,
                                                            float* __restrict__ dpre, float* __restrict__ dr_part) {
  constexpr int WA = W > 0 ? W : 1;
  extern __shared__ float lds[];
  __shared__ f32x4 red[kTWaves][16];
  t_stage(lds, p);
  const float* vec = lds + kTVec;
  const int l = lane64(), g = l >> 4, c = l & 15;
  const int wv = threadIdx.x >> 6;
  const int64_t ntiles = (n + 15) / 16;
  const int64_t nw = (int64_t)gridDim.x * kTWaves;
  f32x4 drp[4];
  t_zero(drp);
  for (int64_t t = (int64_t)blockIdx.x * kTWaves + wv; t < ntiles; t += nw) {
    const int64_t i = 16 * t + c;
    const bool live = i < n;
    const int64_t ri = live ? i : n - 1;
    f32x4 x[4], cx[WA][4], ht[4], dy[4];
    float a[WA];
    t_load(h, ri, g, x);
#pragma unroll
    for (int k = 0; k < W; ++k) t_load(C.c[k], ri, g, cx[k]);
    t_load(dH, ri, g, dy);
    t_attend<W, WA>(lds, vec, cx, a, ht, g, c);
    f32x4 ar[4], az[4], ain[4], ahn[4];
    t_gates<W>(lds, x, ht, ar, az, ain, ahn, g, c);
    // gate gradients, in place of the pre-activations
    f32x4 dht[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int col = 16 * b + 4 * g;
      const f32x4 br = t_vec4(vec + kTD, col), bz = t_vec4(vec + 2 * kTD, col);
      const f32x4 bin = t_vec4(vec + 3 * kTD, col), bhn = t_vec4(vec + 4 * kTD, col);
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        const float rg = t_sigmoid(ar[b][v] + br[v]);
        const float zg = t_sigmoid(az[b][v] + bz[v]);
        const float ghn = ahn[b][v] + bhn[v];
        const float ng = t_tanh(ain[b][v] + bin[v] + rg * ghn);
        const float dyv = dy[b][v];
        const float dpn = dyv * (1.f - zg) * (1.f - ng * ng);
        const float dpz = dyv * (ht[b][v] - ng) * zg * (1.f - zg);
        const float dpr = dpn * ghn * rg * (1.f - rg);
        dht[b][v] = dyv * zg;
        ar[b][v] = dpr;
        az[b][v] = dpz;
        ain[b][v] = dpn;
        ahn[b][v] = dpn * rg;
      }
    }
    if (live) {
      t_store(Ht_out, i, g, ht);
      t_store(dG, 4 * i + 0, g, ar);
      t_store(dG, 4 * i + 1, g, az);
      t_store(dG, 4 * i + 2, g, ain);
      t_store(dG, 4 * i + 3, g, ahn);
    }
    f32x4 acc[4];
    t_zero(acc);
    t_gemm<true>(lds, 1, ar, acc, g, c);
    t_gemm<true>(lds, 2, az, acc, g, c);
    t_gemm<true>(lds, 3, ain, acc, g, c);
    if (live) t_store(dh, i, g, acc);
    if constexpr (W > 0) {
      t_gemm<true>(lds, 4, ar, dht, g, c);
      t_gemm<true>(lds, 5, az, dht, g, c);
      t_gemm<true>(lds, 6, ahn, dht, g, c);
      // softmax backward: da_k = dHt . c_k, ds_k = a_k (da_k - sum_j a_j da_j).
      // The context rows are read again here and u_k = tanh(c_k Q^T) is
      // recomputed, rather than both kept live through the products above
      // (the rows were read moments ago and are likely still cached; keeping
      // them and u costs more registers than the wave has).
#pragma unroll
      for (int k = 0; k < W; ++k) t_load(C.c[k], ri, g, cx[k]);
      float da[WA];
      float sad = 0.f;
#pragma unroll
      for (int k = 0; k < W; ++k) {
        float part = 0.f;
#pragma unroll
        for (int b = 0; b < 4; ++b)
#pragma unroll
          for (int v = 0; v < 4; ++v) part += dht[b][v] * cx[k][b][v];
        da[k] = t_rowsum(part);
        sad += a[k] * da[k];
      }
#pragma unroll
      for (int k = 0; k < W; ++k) {
        const float ds = a[k] * (da[k] - sad);
        const float dsl = live ? ds : 0.f;
        f32x4 dp[4];
        t_zero(dp);
        t_gemm<true>(lds, 0, cx[k], dp, g, c);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const f32x4 r4 = t_vec4(vec, 16 * b + 4 * g);
#pragma unroll
          for (int v = 0; v < 4; ++v) {
            const float u = t_tanh(dp[b][v]);
            drp[b][v] += dsl * u;
            dp[b][v] = ds * r4[v] * (1.f - u * u);
          }
        }
        if (live) t_store(dpre + (int64_t)k * n * kTD, i, g, dp);
        if (dC.c[k]) {
          f32x4 o[4];
          t_load(dC.c[k], ri, g, o);
#pragma unroll
          for (int b = 0; b < 4; ++b) o[b] += a[k] * dht[b];
          t_gemm<false>(lds, 0, dp, o, g, c);
          if (live) t_store(dC.c[k], i, g, o);
        }
      }
    }
  }
  if constexpr (W > 0) {
    // dr: over the rows of the wave (lanes c = 0..15), then the waves in order
#pragma unroll
    for (int b = 0; b < 4; ++b)
#pragma unroll
      for (int v = 0; v < 4; ++v)
#pragma unroll
        for (int o = 1; o < 16; o <<= 1) drp[b][v] += __shfl_xor(drp[b][v], o, 64);
  }
  if (c == 0) {
#pragma unroll
    for (int b = 0; b < 4; ++b) red[wv][4 * b + g] = drp[b];
  }
  __syncthreads();
  if (threadIdx.x < 16) {
    f32x4 s = red[0][threadIdx.x];
    for (int q = 1; q < kTWaves; ++q) s += red[q][threadIdx.x];
    *reinterpret_cast<f32x4*>(dr_part + (int64_t)blockIdx.x * kTD + 4 * threadIdx.x) = s;
  }
}

// dr (+)= sum over blocks of the partials, in block order.
__global__ void k_temporal_dr(const float* __restrict__ part, int64_t blocks, float* __restrict__ dr, int accumulate) {
  const int c = threadIdx.x;
  if (c >= kTD) return;
  float s = accumulate ? dr[c] : 0.f;
  for (int64_t b = 0; b < blocks; ++b) s += part[b * kTD + c];
  dr[c] = s;
}

int64_t t_grid(int64_t n) {
  const int64_t blocks = cdiv(cdiv(n, 16), kTWaves);
  const int64_t cap = num_cus();
  return blocks < cap ? blocks : cap;
}

struct TempWs {
  float *Ht, *dG, *dpre, *dr_part, *splitk, *colsum;
  template <class A>
  void layout(A& a, int64_t n, int w) {
    Ht = a.template take<float>(n * kTD);
    dG = a.template take<float>(4 * n * kTD);
    dpre = a.template take<float>((int64_t)w * n * kTD);
    dr_part = a.template take<float>((t_grid(n) > 0 ? t_grid(n) : 1) * kTD);
    splitk = a.template take<float>(splitk_max_chunks() * (int64_t)kTD * kTD);
    colsum = a.template take<float>(splitk_max_chunks() * (int64_t)kTD);
  }
};

template <class K>
int t_set_lds(K kern) {
  HG_HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                 (int)kTLds));
  return HG_OK;
}

template <int W, class T>
int temporal_fwd_launch(int64_t n, const T* h, const void* const* C, const TParams& p, T* H, hipStream_t st) {
  TCtx<T> ctx{};
  for (int k = 0; k < W; ++k) ctx.c[k] = static_cast<const T*>(C[k]);
  auto kern = k_temporal_fwd<W, T>;
  static bool attr = false;
  if (!attr) {
    HG_TRY(t_set_lds(kern));
    attr = true;
  }
  HG_LAUNCH("temporal_fwd", kern, dim3((unsigned)t_grid(n)), dim3(kTThreads), kTLds, st, n, h, ctx, p, H);
  return HG_OK;
}

template <int W, class T>
int temporal_bwd_launch(int64_t n, const T* h, const void* const* C, const TParams& p, const T* dH, T* dh,
                        void* const* dC, const TempWs& w, hipStream_t st) {
  TCtx<T> ctx{};
  TCtxOut<T> dctx{};
  for (int k = 0; k < W; ++k) {
    ctx.c[k] = static_cast<const T*>(C[k]);
    dctx.c[k] = dC ? static_cast<T*>(dC[k]) : nullptr;
  }
  auto kern = k_temporal_bwd<W, T>;
  static bool attr = false;
  if (!attr) {
    HG_TRY(t_set_lds(kern));
    attr = true;
  }
  HG_LAUNCH("temporal_bwd", kern, dim3((unsigned)t_grid(n)), dim3(kTThreads), kTLds, st, n, h, ctx, p, dH, dh, dctx,
            w.Ht, w.dG, w.dpre, w.dr_part);
  return HG_OK;
}

template <class T>
int temporal_fwd_impl(int64_t n, int w, const T* h, const void* const* C, const TParams& p, T* H, hipStream_t st) {
  switch (w) {
    case 0: return temporal_fwd_launch<0, T>(n, h, C, p, H, st);
    case 1: return temporal_fwd_launch<1, T>(n, h, C, p, H, st);
    case 2: return temporal_fwd_launch<2, T>(n, h, C, p, H, st);
    case 3: return temporal_fwd_launch<3, T>(n, h, C, p, H, st);
    default: return temporal_fwd_launch<4, T>(n, h, C, p, H, st);
  }
}

template <class T>
int temporal_bwd_impl(int64_t n, int w, const T* h, const void* const* C, const TParams& p, const T* dH, T* dh,
                      void* const* dC, int accumulate, const hg_temporal_grads* G, void* ws, size_t ws_bytes,
                      hipStream_t st) {
  Arena a(ws, ws_bytes);
  TempWs wk;
  wk.layout(a, n, w);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "temporal backward workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  if (n > 0) {
    int s = HG_OK;
    switch (w) {
      case 0: s = temporal_bwd_launch<0, T>(n, h, C, p, dH, dh, dC, wk, st); break;
      case 1: s = temporal_bwd_launch<1, T>(n, h, C, p, dH, dh, dC, wk, st); break;
      case 2: s = temporal_bwd_launch<2, T>(n, h, C, p, dH, dh, dC, wk, st); break;
      case 3: s = temporal_bwd_launch<3, T>(n, h, C, p, dH, dh, dC, wk, st); break;
      default: s = temporal_bwd_launch<4, T>(n, h, C, p, dH, dh, dC, wk, st); break;
    }
    HG_TRY(s);
  }
  constexpr int64_t kDD = (int64_t)kTD * kTD;
  // dWi[k] = h^T dG[:, k], dbi[k] = column sums of dG[:, k]
  for (int k = 0; k < 3; ++k) {
    HG_TRY((launch_gemm_tn<kTD>("temporal_dWi", n, LoadRows<kTD, T>{h, rows_contig(0)},
                                LoadRows<kTD, float>{wk.dG, RowMap{nullptr, 0, 4, k}}, wk.splitk, wk.colsum,
                                G->Wi + k * kDD, G->bi ? G->bi + k * kTD : nullptr, accumulate, st)));
  }
  // dWh[k] = Ht^T dG[:, k'] with k' = 0, 1, 3 (the new gate's hidden side is gated by r)
  for (int k = 0; k < 3; ++k) {
    const int q = k < 2 ? k : 3;
    HG_TRY((launch_gemm_tn<kTD>("temporal_dWh", n, LoadRows<kTD, float>{wk.Ht, rows_contig(0)},
                                LoadRows<kTD, float>{wk.dG, RowMap{nullptr, 0, 4, q}}, wk.splitk, wk.colsum,
                                G->Wh + k * kDD, G->bh ? G->bh + k * kTD : nullptr, accumulate, st)));
  }
  // dQ = sum_k dpre_k^T C_k
  if (w == 0 || n == 0) {
    if (!accumulate) HG_TRY(fill_f32(G->Q, 0.f, kDD, st));
  }
  if (n > 0) {
    for (int k = 0; k < w; ++k) {
      HG_TRY((launch_gemm_tn<kTD>("temporal_dQ", n, LoadRows<kTD, float>{wk.dpre + (int64_t)k * n * kTD,
                                                                         rows_contig(0)},
                                  LoadRows<kTD, T>{static_cast<const T*>(C[k]), rows_contig(0)}, wk.splitk,
                                  wk.colsum, G->Q, nullptr, (k > 0 || accumulate) ? 1 : 0, st)));
    }
  }
  const int64_t blocks = n > 0 ? t_grid(n) : 0;
  HG_LAUNCH("temporal_dr", k_temporal_dr, dim3(1), dim3(kTD), 0, st, (const float*)wk.dr_part, blocks, G->r,
            accumulate);
  return HG_OK;
}

bool t_alias(const void* x, const void* y) { return x && y && x == y; }

int t_check(int64_t n, int32_t d, int32_t w, int32_t dtype, const void* h, const void* const* C,
            const hg_temporal_weights* W, const void* out) {
  if (n < 0 || w < 0) return fail(HG_ERR_ARG, "n < 0 or w < 0");
  if (d != kTD) return fail(HG_ERR_UNSUPPORTED, "temporal module: d = 64 only (d=%d)", d);
  if (w > kTMaxW) return fail(HG_ERR_UNSUPPORTED, "temporal module: w <= %d (w=%d)", kTMaxW, w);
  if (dtype != HG_DTYPE_F32 && dtype != HG_DTYPE_BF16) return fail(HG_ERR_UNSUPPORTED, "dtype %d", dtype);
  if (!W || !W->Q || !W->r || !W->Wi || !W->Wh) return fail(HG_ERR_ARG, "null weight (only bi, bh may be NULL)");
  if (n > 0) {
    if (!h || !out) return fail(HG_ERR_ARG, "null row array");
    if (w > 0 && !C) return fail(HG_ERR_ARG, "null context array");
    for (int k = 0; k < w; ++k) {
      if (!C[k]) return fail(HG_ERR_ARG, "null context state %d", k);
      if (t_alias(C[k], out)) return fail(HG_ERR_ARG, "the output must not alias context state %d", k);
    }
    if (t_alias(h, out)) return fail(HG_ERR_ARG, "the output must not alias h");
  }
  return HG_OK;
}

TParams t_params(const hg_temporal_weights* W) { return TParams{W->Q, W->r, W->Wi, W->bi, W->Wh, W->bh}; }

}  // namespace
}  // namespace hg

using namespace hg;

extern "C" {

size_t hg_temporal_bwd_workspace_size(int64_t n, int32_t d, int32_t w) {
  if (n < 0 || d != kTD || w < 0 || w > kTMaxW) return 0;
  Sizer z;
  TempWs t;
  t.layout(z, n, w);
  return z.used;
}

int hg_temporal_fwd(int64_t n, int32_t d, int32_t w, int32_t dtype, const void* h, const void* const* C,
                    const hg_temporal_weights* W, void* H, void* stream) {
  HG_TRY(t_check(n, d, w, dtype, h, C, W, H));
  if (n == 0) return HG_OK;
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const TParams p = t_params(W);
  if (dtype == HG_DTYPE_F32)
    return temporal_fwd_impl<float>(n, w, static_cast<const float*>(h), C, p, static_cast<float*>(H), st);
  return temporal_fwd_impl<bf16_t>(n, w, static_cast<const bf16_t*>(h), C, p, static_cast<bf16_t*>(H), st);
}

int hg_temporal_bwd(int64_t n, int32_t d, int32_t w, int32_t dtype, const void* h, const void* const* C,
                    const hg_temporal_weights* W, const void* dH, void* dh, void* const* dC, int32_t accumulate,
                    const hg_temporal_grads* G, void* ws, size_t ws_bytes, void* stream) {
  HG_TRY(t_check(n, d, w, dtype, h, C, W, dh));
  if (!G || !G->Q || !G->r || !G->Wi || !G->Wh) return fail(HG_ERR_ARG, "null gradient (only bi, bh may be NULL)");
  if (accumulate != 0 && accumulate != 1) return fail(HG_ERR_ARG, "accumulate must be 0 or 1");
  if (n > 0) {
    if (!dH) return fail(HG_ERR_ARG, "null dH");
    if (t_alias(dh, dH)) return fail(HG_ERR_ARG, "dh must not alias dH");
    if (dC) {
      for (int k = 0; k < w; ++k) {
        if (!dC[k]) continue;
        if (t_alias(dC[k], dh) || t_alias(dC[k], dH) || t_alias(dC[k], h))
          return fail(HG_ERR_ARG, "dC[%d] must not alias h, dH or dh", k);
        for (int j = 0; j < w; ++j) {
          if (t_alias(dC[k], C[j])) return fail(HG_ERR_ARG, "dC[%d] must not alias a context state", k);
          if (j != k && t_alias(dC[k], dC[j])) return fail(HG_ERR_ARG, "dC[%d] and dC[%d] alias", k, j);
        }
      }
    }
  }
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const TParams p = t_params(W);
  if (dtype == HG_DTYPE_F32)
    return temporal_bwd_impl<float>(n, w, static_cast<const float*>(h), C, p, static_cast<const float*>(dH),
                                     static_cast<float*>(dh), dC, accumulate, G, ws, ws_bytes, st);
  return temporal_bwd_impl<bf16_t>(n, w, static_cast<const bf16_t*>(h), C, p, static_cast<const bf16_t*>(dH),
                                   static_cast<bf16_t*>(dh), dC, accumulate, G, ws, ws_bytes, st);
}

}  // extern "C"
