// Prediction head, masked BCE and the Adam update ("Prediction and
// Optimization": the two-layer MLP E18, the BCE loss E19 over the labelled
// nodes, the joint objective E20, the Adam optimiser with weight decay).
//
//   a = H W1 + b1, hid = ReLU(a), o = hid W2 + b2, p = sigmoid(o)
//   L_BCE = (1/N_m) sum_labelled softplus(o) - y o
//   dL/do = (p - y)/N_m on labelled rows; da = mask * (dL/do W2^T);
//   dH = da W1^T, dW1 = H^T da, db1 = sum da, dW2 = hid^T dL/do, db2 = sum dL/do
//
// da is rank one per row, so it is never stored: LoadRank1Masked forms it in
// the MFMA loaders of the dH and dW1 GEMMs from dL/do, W2 and the ReLU mask.
#include <cmath>

#include "hg_mfma.h"

namespace hg {
namespace {

constexpr int kHeadBlocks = 1024;
constexpr int kHeadThreads = 256;

// Row i, column c: (bit c of mask row i) ? u[i] * w[c] : 0.
template <int D>
struct LoadRank1Masked {
  const float* u;
  const float* w;
  const uint32_t* mask;
  RowMap map;
  // split-K (gemm_tn) form
  struct Raw {
    float u;
    uint32_t word;
  };
  struct Prep {
    f32x4 w;
    int shift;
  };
  __device__ __forceinline__ Raw raw4b(int64_t b, int c) const { return Raw{u[b], mask[b * (D / 32) + (c >> 5)]}; }
  __device__ __forceinline__ Prep prep(int c) const { return Prep{*reinterpret_cast<const f32x4*>(w + c), c & 31}; }
  __device__ __forceinline__ f32x4 cook4(const Raw& r, const Prep& p) const {
    const uint32_t nib = r.word >> p.shift;
    f32x4 x;
#pragma unroll
    for (int k = 0; k < 4; ++k) x[k] = ((nib >> k) & 1u) ? r.u * p.w[k] : 0.f;
    return x;
  }
  // whole-row (gemm_rows_pp) form: lane group g holds columns 16 kb + 4 g
  struct RowRaw {
    float u;
    uint32_t m[D / 32];
  };
  __device__ __forceinline__ void fetch_row(int64_t b, int, RowRaw& r) const {
    r.u = u[b];
#pragma unroll
    for (int q = 0; q < D / 32; ++q) r.m[q] = mask[b * (D / 32) + q];
  }
  __device__ __forceinline__ f32x4 operand4(const RowRaw& r, int kb, int g) const {
    const f32x4 wv = *reinterpret_cast<const f32x4*>(w + 16 * kb + 4 * g);
    const uint32_t nib = r.m[kb >> 1] >> (16 * (kb & 1) + 4 * g);
    f32x4 x;
#pragma unroll
    for (int k = 0; k < 4; ++k) x[k] = ((nib >> k) & 1u) ? r.u * wv[k] : 0.f;
    return x;
  }
  __device__ __forceinline__ f32x4 stored4(const RowRaw& r, int kb) const { return operand4(r, kb, 0); }
  static constexpr bool kTee = false;
  static constexpr bool kBoundByStored = false;
  __device__ __forceinline__ void tee4(int64_t, int, int, f32x4) const {}
};

// Same epilogue as the attention layer's: hid = relu(acc + b1), mask bits.
template <int D>
struct StoreHidden {
  static constexpr bool kAddA = false;
  static constexpr bool kMask = true;
  float* out;
  RowMap map;
  const float* bias;
  uint32_t* mask;
  __device__ __forceinline__ f32x4 pre4(int64_t, int64_t, int) const { return f32x4{0.f, 0.f, 0.f, 0.f}; }
  __device__ __forceinline__ uint32_t store4(int64_t, int64_t ro, int c, f32x4 acc, f32x4) const {
    const f32x4 a = acc + (bias ? *reinterpret_cast<const f32x4*>(bias + c) : f32x4{0.f, 0.f, 0.f, 0.f});
    uint32_t bits = 0;
    f32x4 h;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      bits |= (a[k] > 0.f ? 1u : 0u) << k;
      h[k] = fmaxf(a[k], 0.f);
    }
    *reinterpret_cast<f32x4*>(out + ro * D + c) = h;
    return bits;
  }
  __device__ __forceinline__ void mask_word(int64_t ro, int wi, uint32_t word) const { mask[ro * (D / 32) + wi] = word; }
};

__device__ __forceinline__ float block_sum_256(float v, float* red) {
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

// Number of labelled rows, as per-block partial counts (row i of the head is
// row rows[i] of the labels when a row list is given).
__global__ void __launch_bounds__(kHeadThreads) k_count_labels(const int8_t* __restrict__ labels,
                                                               const int32_t* __restrict__ rows, int64_t n,
                                                               int32_t* __restrict__ part) {
  __shared__ float red[kHeadThreads];
  float c = 0.f;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    c += labels[rows ? (int64_t)rows[i] : i] >= 0 ? 1.f : 0.f;
  const float s = block_sum_256(c, red);
  if (threadIdx.x == 0) part[blockIdx.x] = (int32_t)s;
}

// One wave holds 64 / (D/4) rows; per row the logit, the probability, the
// loss term and dL/do; per block the partial sums of dW2 (D), db2, loss.
template <int D>
__global__ void __launch_bounds__(kHeadThreads) k_mlp_head(int64_t n, const float* __restrict__ hid,
                                                           const float* __restrict__ W2, const float* __restrict__ b2,
                                                           const int8_t* __restrict__ labels,
                                                           const int32_t* __restrict__ rows,
                                                           const int32_t* __restrict__ cnt_part,
                                                           float* __restrict__ dout, float* __restrict__ prob,
                                                           float* __restrict__ part) {
  constexpr int LPR = D / 4, RPW = 64 / LPR, NW = kHeadThreads / 64;
  __shared__ float red[kHeadThreads];
  __shared__ f32x4 wred[NW][LPR];
  __shared__ int nm_s;
  if (threadIdx.x == 0) {
    int64_t c = 0;
    for (int k = 0; k < kHeadBlocks; ++k) c += cnt_part[k];
    nm_s = (int)c;
  }
  __syncthreads();
  const float inv_nm = nm_s > 0 ? 1.0f / (float)nm_s : 0.f;
  const int l = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4;
  const f32x4 w4 = *reinterpret_cast<const f32x4*>(W2 + c0);
  const float bb = b2 ? b2[0] : 0.f;
  const int64_t gw = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  f32x4 aw = {0.f, 0.f, 0.f, 0.f};
  float ab = 0.f, al = 0.f;
  for (int64_t i0 = gw * RPW; i0 < n; i0 += nwaves * RPW) {
    const int64_t i = i0 + slot;
    const bool live = i < n;
    const f32x4 h = live ? *reinterpret_cast<const f32x4*>(hid + i * D + c0) : f32x4{0.f, 0.f, 0.f, 0.f};
    float o = h[0] * w4[0] + h[1] * w4[1] + h[2] * w4[2] + h[3] * w4[3];
#pragma unroll
    for (int q = 1; q < LPR; q <<= 1) o += __shfl_xor(o, q, 64);
    o += bb;
    const int lab = live ? (int)labels[rows ? (int64_t)rows[i] : i] : -1;
    float d_o = 0.f, term = 0.f;
    const float p = 1.0f / (1.0f + __expf(-o));
    if (lab >= 0) {
      const float y = (float)lab;
      d_o = (p - y) * inv_nm;
      term = fmaxf(o, 0.f) + log1pf(__expf(-fabsf(o))) - y * o;
    }
    if (live && lr == 0) {
      dout[i] = d_o;
      if (prob) prob[i] = p;
      ab += d_o;
      al += term;
    }
    aw += d_o * h;
  }
  // dW2: over the rows of the wave, then the waves of the block in order
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) aw[k] += __shfl_xor(aw[k], o, 64);
  if (slot == 0) wred[wv][lr] = aw;
  const float sb = block_sum_256(ab, red);
  const float sl = block_sum_256(al, red);
  if (threadIdx.x < LPR) {
    f32x4 s = wred[0][threadIdx.x];
    for (int q = 1; q < NW; ++q) s += wred[q][threadIdx.x];
    *reinterpret_cast<f32x4*>(part + (int64_t)blockIdx.x * (D + 2) + 4 * threadIdx.x) = s;
  }
  if (threadIdx.x == 0) {
    part[(int64_t)blockIdx.x * (D + 2) + D] = sb;
    part[(int64_t)blockIdx.x * (D + 2) + D + 1] = sl * inv_nm;
  }
}

// Sums the block partials in block order: dW2 [D], db2, loss.
template <int D>
__global__ void k_head_final(const float* __restrict__ part, float* __restrict__ dW2, float* __restrict__ db2,
                             float* __restrict__ loss) {
  const int c = threadIdx.x;
  if (c >= D + 2) return;
  float s = 0.f;
  for (int b = 0; b < kHeadBlocks; ++b) s += part[(int64_t)b * (D + 2) + c];
  if (c < D) {
    dW2[c] = s;
  } else if (c == D) {
    if (db2) db2[0] = s;
  } else {
    loss[0] = s;
  }
}

__global__ void k_adam(int64_t n, float* __restrict__ theta, const float* __restrict__ grad, float* __restrict__ m,
                       float* __restrict__ v, float lr, float beta1, float beta2, float eps, float wd, float bc1,
                       float bc2) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const float th = theta[i];
    const float g = grad[i] + wd * th;
    const float mi = beta1 * m[i] + (1.f - beta1) * g;
    const float vi = beta2 * v[i] + (1.f - beta2) * g * g;
    m[i] = mi;
    v[i] = vi;
    theta[i] = th - lr * (mi / bc1) / (sqrtf(vi / bc2) + eps);
  }
}

struct HeadWs {
  float* hid;       // [n, d]
  uint32_t* mask;   // [n, d / 32]
  float* dout;      // [n]
  int32_t* cnt;     // [kHeadBlocks]
  float* part;      // [kHeadBlocks, d + 2]
  float *splitk, *colsum;
  template <class A>
  void layout(A& a, int64_t n, int d) {
    hid = a.template take<float>(n * d);
    mask = a.template take<uint32_t>(n * (d / 32));
    dout = a.template take<float>(n);
    cnt = a.template take<int32_t>(kHeadBlocks);
    part = a.template take<float>((int64_t)kHeadBlocks * (d + 2));
    splitk = a.template take<float>(splitk_max_chunks() * (int64_t)d * d);
    colsum = a.template take<float>(splitk_max_chunks() * (int64_t)d);
  }
};

// With a row list only the listed rows (a superset of the labelled ones) go
// through the head: the hidden rows, logits and dL/do are kept compactly in
// list order, H is read and dH written through the list, and the other rows
// of dH are zero.
template <int D>
int head_impl(int64_t n, const float* H, const float* W1, const float* b1, const float* W2, const float* b2,
              const int8_t* labels, const int32_t* rows, int64_t n_list, float* loss, float* prob, float* dH,
              float* dW1, float* db1, float* dW2, float* db2, void* ws, size_t ws_bytes, hipStream_t st) {
  Arena a(ws, ws_bytes);
  HeadWs w;
  w.layout(a, n, D);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "prediction-head workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  const int64_t m = rows ? n_list : n;
  const RowMap hm = rows ? rows_list(rows) : rows_contig(0);
  // hidden layer and its ReLU mask
  HG_TRY((launch_gemm_rows_pp<D, false>("head_hidden", m, W1, LoadRows<D, float>{H, hm},
                                        StoreHidden<D>{w.hid, rows_contig(0), b1, w.mask}, st)));
  HG_LAUNCH("head_count", k_count_labels, dim3(kHeadBlocks), dim3(kHeadThreads), 0, st, labels, rows, m, w.cnt);
  HG_LAUNCH("head_logit", k_mlp_head<D>, dim3(kHeadBlocks), dim3(kHeadThreads), 0, st, m, (const float*)w.hid, W2, b2,
            labels, rows, (const int32_t*)w.cnt, w.dout, prob, w.part);
  HG_LAUNCH("head_final", k_head_final<D>, dim3(1), dim3(256), 0, st, (const float*)w.part, dW2, db2, loss);
  // dH = da W1^T and dW1 = H^T da with da = mask * (dL/do W2^T) formed in the loaders
  if (rows && n > 0) HG_TRY(fill_f32(dH, 0.f, n * D, st));
  const LoadRank1Masked<D> da{w.dout, W2, w.mask, rows_contig(0)};
  HG_TRY((launch_gemm_rows_pp<D, true>("head_dx", m, W1, da, StoreRows<D, float>{dH, hm, nullptr, nullptr}, st)));
  HG_TRY((launch_gemm_tn<D>("head_dw", m, LoadRows<D, float>{H, hm}, da, w.splitk, w.colsum, dW1, db1, 0, st)));
  return HG_OK;
}

}  // namespace
}  // namespace hg

using namespace hg;

extern "C" {

size_t hg_mlp_bce_workspace_size(int64_t n_rows, int32_t d, int32_t d_hidden) {
  if (n_rows < 0 || d != d_hidden || (d != 64 && d != 128)) return 0;
  Sizer z;
  HeadWs w;
  w.layout(z, n_rows, d);
  return z.used;
}

int hg_mlp_bce_fwd_bwd(int64_t n_rows, int32_t d, int32_t d_hidden, const float* H, const float* W1, const float* b1,
                       const float* W2, const float* b2, const int8_t* labels, const int32_t* rows, int64_t n_list,
                       float* loss, float* prob, float* dH, float* dW1, float* db1, float* dW2, float* db2, void* ws,
                       size_t ws_bytes, void* stream) {
  if (n_rows < 0) return fail(HG_ERR_ARG, "n_rows < 0");
  if (rows && (n_list < 0 || n_list > n_rows)) return fail(HG_ERR_ARG, "n_list outside [0, n_rows]");
  if (rows && prob) return fail(HG_ERR_ARG, "prob needs every row: it must be NULL with a row list");
  if (d != d_hidden || (d != 64 && d != 128))
    return fail(HG_ERR_UNSUPPORTED, "prediction head: d_hidden == d in {64, 128} (d=%d, d_hidden=%d)", d, d_hidden);
  if (!W1 || !W2 || !loss || !dW1 || !dW2 || (n_rows > 0 && (!H || !labels || !dH)))
    return fail(HG_ERR_ARG, "null pointer (only b1, b2, prob, db1, db2 may be NULL; H, labels, dH when n_rows = 0)");
  if (n_rows > 0 && dH == H) return fail(HG_ERR_ARG, "dH must not alias H");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (d == 64)
    return head_impl<64>(n_rows, H, W1, b1, W2, b2, labels, rows, n_list, loss, prob, dH, dW1, db1, dW2, db2, ws,
                         ws_bytes, st);
  return head_impl<128>(n_rows, H, W1, b1, W2, b2, labels, rows, n_list, loss, prob, dH, dW1, db1, dW2, db2, ws,
                        ws_bytes, st);
}

int hg_adam_step(int64_t n, float* param, const float* grad, float* m, float* v, int64_t step, float lr, float beta1,
                 float beta2, float eps, float weight_decay, void* stream) {
  if (n < 0 || step < 1) return fail(HG_ERR_ARG, "n < 0 or step < 1");
  if (n == 0) return HG_OK;
  if (!param || !grad || !m || !v) return fail(HG_ERR_ARG, "null pointer");
  if (!(beta1 >= 0.f && beta1 < 1.f) || !(beta2 >= 0.f && beta2 < 1.f) || !(eps > 0.f))
    return fail(HG_ERR_ARG, "beta1, beta2 in [0, 1) and eps > 0 required");
  const float bc1 = (float)(1.0 - std::pow((double)beta1, (double)step));
  const float bc2 = (float)(1.0 - std::pow((double)beta2, (double)step));
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t blocks = cdiv(n, 256) < 4096 ? cdiv(n, 256) : 4096;
  HG_LAUNCH("adam", k_adam, dim3((unsigned)blocks), dim3(256), 0, st, n, param, grad, m, v, lr, beta1, beta2, eps,
            weight_decay, bc1, bc2);
  return HG_OK;
}

}  // extern "C"
