// Heterogeneous graph transformer layer (the attention, message, softmax,
// aggregation and update equations E6-E11 of the "Heterogeneous Graph
// Transformer" paragraph), float32.
//
// Forward:
//   1. K, Q, V: per-type projections with bias (pipelined fp32 MFMA GEMM);
//   2. Kt = K W_att[r], Vt = V W_msg[r] for the active sources of each
//      relation (the per-head dk x dk blocks expanded to one block-diagonal
//      d x d matrix per relation), stored at row src * R + r like the mean
//      layer's relation transforms;
//   3. k_hgt_attn_fwd: one wave per destination j streams its CSR row,
//      gathers Kt and Vt of every in-edge, and keeps an online softmax per
//      head (running max, running sum, running weighted sum), so the scores
//      never go to memory; writes h~_j and the per-head log-sum-exp;
//   4. z = h~ W_agg[type] + b_agg, h' = ReLU(z) + h, with the ReLU mask
//      written by the GEMM epilogue.
#include <cmath>

#include "hg_mfma.h"

namespace hg {
namespace {

constexpr int kAttnThreads = 256;

bool hgt_shape_ok(int d, int heads) {
  if (d != 64 && d != 128) return false;
  if (heads < 1 || d % heads) return false;
  const int dk = d / heads;
  return dk >= 4 && (dk & (dk - 1)) == 0;
}

int validate_hgt(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L) return fail(HG_ERR_ARG, "null subgraph or layer descriptor");
  if (L->dtype != HG_DTYPE_F32) return fail(HG_ERR_UNSUPPORTED, "attention layer: float32 features only");
  if (!hgt_shape_ok(L->d, L->heads))
    return fail(HG_ERR_UNSUPPORTED, "attention layer: d in {64, 128} and d / heads a power of two >= 4 (d=%d, heads=%d)",
                L->d, L->heads);
  if ((L->relu != 0 && L->relu != 1) || (L->residual != 0 && L->residual != 1))
    return fail(HG_ERR_ARG, "relu and residual must be 0 or 1");
  if (s->n_rel < 1 || s->n_ntype < 1) return fail(HG_ERR_ARG, "subgraph has no relations or node types");
  if (s->n_sub < 0 || s->e_sub < 0) return fail(HG_ERR_ARG, "subgraph sizes are negative");
  return HG_OK;
}

// Layout of `saved` (float32 unless noted).
struct HgtSaved {
  float *K, *Q, *V;   // [n_sub, d]
  float *Kt, *Vt;     // [n_sub * R, d], rows src * R + r of active (src, r)
  float* ht;          // [n_sub, d]
  float* lse;         // [n_sub, S]
  template <class A>
  void layout(A& a, const hg_subgraph* s, int d, int S) {
    const int64_t n = s->n_sub, nr = s->n_sub * (int64_t)s->n_rel;
    K = a.template take<float>(n * d);
    Q = a.template take<float>(n * d);
    V = a.template take<float>(n * d);
    Kt = a.template take<float>(nr * d);
    Vt = a.template take<float>(nr * d);
    ht = a.template take<float>(n * d);
    lse = a.template take<float>(n * S);
  }
};

struct HgtFwdWs {
  float *Watt, *Wmsg;  // [R, d, d] block-diagonal expansions
  template <class A>
  void layout(A& a, const hg_subgraph* s, int d) {
    Watt = a.template take<float>((int64_t)s->n_rel * d * d);
    Wmsg = a.template take<float>((int64_t)s->n_rel * d * d);
  }
};

// [R, S, dk, dk] -> [R, d, d] with zero off-diagonal blocks.
__global__ void k_blockdiag(const float* __restrict__ w, int64_t R, int d, int S, float* __restrict__ out) {
  const int dk = d / S;
  const int64_t total = R * d * d;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / ((int64_t)d * d);
    const int row = (int)((e / d) % d), col = (int)(e % d);
    const int sr = row / dk, sc = col / dk;
    out[e] = (sr == sc) ? w[((r * S + sr) * dk + row % dk) * dk + col % dk] : 0.f;
  }
}

__device__ __forceinline__ int type_of(int64_t v, int T, const int32_t* __restrict__ type_off) {
  int t = 0;
  for (int k = 1; k < T; ++k) t += (v >= (int64_t)type_off[k]) ? 1 : 0;
  return t;
}

// One wave per destination row; the row's lanes form 64 / (D/4) slots that
// take alternate in-edges, each slot with its own online-softmax state per
// head (lanes of one head hold its dk columns); the slot states are merged at
// the end.  U in-edges per slot are in flight (two row gathers each).
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_attn_fwd(
    int64_t n_sub, int32_t R, int32_t T, const int32_t* __restrict__ type_off, const int32_t* __restrict__ csr_ptr,
    const int32_t* __restrict__ csr_col, const float* __restrict__ Q, const float* __restrict__ Kt,
    const float* __restrict__ Vt, const float* __restrict__ mu, float inv_sqrt_dk, float* __restrict__ ht,
    float* __restrict__ lse) {
  constexpr int LPR = D / 4, EPW = 64 / LPR, DK = D / S, LPH = DK / 4, U = 2;
  static_assert(LPH >= 1 && (LPH & (LPH - 1)) == 0, "head width must be a power of two >= 4");
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t j = wave0; j < n_sub; j += nwaves) {
    const int tj = type_of(j, T, type_off);
    const f32x4 q = *reinterpret_cast<const f32x4*>(Q + j * D + c0);
    const int64_t rb = j * R;
    const int32_t p0 = csr_ptr[rb], pe = csr_ptr[rb + R];
    float m = -INFINITY, ls = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int32_t base = p0; base < pe; base += 64) {
      const int32_t pos = base + l;
      int32_t rowi = 0;
      float cf = 0.f;
      if (pos < pe) {
        const int32_t src = csr_col[pos];
        int r = 0;
        for (int t = 1; t < R; ++t) r += (csr_ptr[rb + t] <= pos) ? 1 : 0;
        rowi = src * R + r;
        cf = mu[((int64_t)type_of(src, T, type_off) * R + r) * T + tj] * inv_sqrt_dk;
      }
      const int cnt = (pe - base) < 64 ? (pe - base) : 64;
      for (int e = 0; e < cnt; e += EPW * U) {
        f32x4 kv[U], vv[U];
        float cc[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int my = e + u * EPW + slot;
          const int32_t qi = __shfl(rowi, my & 63, 64);
          cc[u] = __shfl(cf, my & 63, 64);
          ok[u] = my < cnt;
          if (ok[u]) {
            kv[u] = *reinterpret_cast<const f32x4*>(Kt + (int64_t)qi * D + c0);
            vv[u] = *reinterpret_cast<const f32x4*>(Vt + (int64_t)qi * D + c0);
          } else {
            kv[u] = vv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          float dot = kv[u][0] * q[0] + kv[u][1] * q[1] + kv[u][2] * q[2] + kv[u][3] * q[3];
#pragma unroll
          for (int o = 1; o < LPH; o <<= 1) dot += __shfl_xor(dot, o, 64);
          if (ok[u]) {
            const float sc = dot * cc[u];
            const float mn = fmaxf(m, sc);
            const float a = __expf(m - mn), p = __expf(sc - mn);
            ls = ls * a + p;
            acc = acc * a + p * vv[u];
            m = mn;
          }
        }
      }
    }
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1) {
      const float m2 = __shfl_xor(m, o, 64), l2 = __shfl_xor(ls, o, 64);
      f32x4 a2;
#pragma unroll
      for (int k = 0; k < 4; ++k) a2[k] = __shfl_xor(acc[k], o, 64);
      const float mn = fmaxf(m, m2);
      const float s1 = (m == -INFINITY) ? 0.f : __expf(m - mn);
      const float s2 = (m2 == -INFINITY) ? 0.f : __expf(m2 - mn);
      ls = ls * s1 + l2 * s2;
      acc = acc * s1 + a2 * s2;
      m = mn;
    }
    if (slot == 0) {
      const float inv = ls > 0.f ? 1.0f / ls : 0.f;
      *reinterpret_cast<f32x4*>(ht + j * D + c0) = acc * inv;
      if (lr % LPH == 0) lse[j * S + head] = ls > 0.f ? m + logf(ls) : -INFINITY;
    }
  }
}

// Epilogue of the aggregation GEMM: h' = relu(acc + b) + h (residual), with
// the decision bits 1[acc + b > 0] (all ones without ReLU) returned for the
// mask word.
template <int D>
struct StoreReluMask {
  static constexpr bool kAddA = false;
  static constexpr bool kMask = true;
  float* out;
  RowMap map;
  const float* bias;   // [D] or null
  const float* resid;  // rows through the same map, or null
  uint32_t* mask;      // [rows, D / 32]
  int relu;
  __device__ __forceinline__ f32x4 pre4(int64_t, int64_t ro, int c) const {
    return resid ? *reinterpret_cast<const f32x4*>(resid + ro * D + c) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  __device__ __forceinline__ uint32_t store4(int64_t, int64_t ro, int c, f32x4 acc, f32x4 pre) const {
    const f32x4 z = acc + (bias ? *reinterpret_cast<const f32x4*>(bias + c) : f32x4{0.f, 0.f, 0.f, 0.f});
    uint32_t bits = 0;
    f32x4 h;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      bits |= ((!relu || z[k] > 0.f) ? 1u : 0u) << k;
      h[k] = (relu ? fmaxf(z[k], 0.f) : z[k]) + pre[k];
    }
    *reinterpret_cast<f32x4*>(out + ro * D + c) = h;
    return bits;
  }
  __device__ __forceinline__ void mask_word(int64_t ro, int w, uint32_t word) const {
    mask[ro * (D / 32) + w] = word;
  }
};

inline unsigned attn_grid(int64_t rows) {
  int64_t blocks = cdiv(rows, kAttnThreads / 64);
  const int64_t cap = (int64_t)num_cus() * 32;
  if (blocks > cap) blocks = cap;
  return (unsigned)(blocks > 0 ? blocks : 1);
}

template <int D>
int hgt_fwd_impl(const hg_subgraph* s, const hg_hgt_desc* L, const float* Hin, const hg_hgt_weights* W,
                 float* Hout, uint32_t* mask, void* saved, void* ws, size_t ws_bytes, hipStream_t st) {
  const int S = L->heads;
  const int32_t R = s->n_rel, T = s->n_ntype;
  Arena as(saved, (size_t)-1);
  HgtSaved sv;
  sv.layout(as, s, D, S);
  Arena a(ws, ws_bytes);
  HgtFwdWs w;
  w.layout(a, s, D);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "attention forward workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  const PlanView pv = plan_view(s);
  // block-diagonal relation matrices
  {
    const int64_t n = (int64_t)R * D * D;
    const unsigned g = (unsigned)(cdiv(n, 256) < 4096 ? cdiv(n, 256) : 4096);
    HG_LAUNCH("hgt_blockdiag", k_blockdiag, dim3(g), dim3(256), 0, st, W->W_att, (int64_t)R, D, S, w.Watt);
    HG_LAUNCH("hgt_blockdiag", k_blockdiag, dim3(g), dim3(256), 0, st, W->W_msg, (int64_t)R, D, S, w.Wmsg);
  }
  // (1) per-type projections
  for (int t = 0; t < T; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    const int64_t wo = (int64_t)t * D * D, bo = (int64_t)t * D;
    LoadRows<D, float> la{Hin, rows_contig(lo)};
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_proj", hi - lo, W->W_K + wo, la,
                                          StoreRows<D, float>{sv.K, rows_contig(lo), W->b_K ? W->b_K + bo : nullptr, nullptr},
                                          st)));
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_proj", hi - lo, W->W_Q + wo, la,
                                          StoreRows<D, float>{sv.Q, rows_contig(lo), W->b_Q ? W->b_Q + bo : nullptr, nullptr},
                                          st)));
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_proj", hi - lo, W->W_V + wo, la,
                                          StoreRows<D, float>{sv.V, rows_contig(lo), W->b_V ? W->b_V + bo : nullptr, nullptr},
                                          st)));
  }
  // (2) relation transforms of the keys and values of each relation's active sources
  int64_t off = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t n = s->n_active[r];
    const float* wa = w.Watt + (int64_t)r * D * D;
    const float* wm = w.Wmsg + (int64_t)r * D * D;
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_rel", n, wa, LoadRows<D, float>{sv.K, rows_list(pv.active + off)},
                                          StoreRows<D, float>{sv.Kt, rows_list(pv.active + off, R, r), nullptr, nullptr},
                                          st)));
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_rel", n, wm, LoadRows<D, float>{sv.V, rows_list(pv.active + off)},
                                          StoreRows<D, float>{sv.Vt, rows_list(pv.active + off, R, r), nullptr, nullptr},
                                          st)));
    off += n;
  }
  // (3) attention-weighted aggregation
  const float inv_sqrt_dk = 1.0f / std::sqrt((float)(D / S));
  if (s->n_sub > 0) {
#define HG_ATTN_FWD(S_)                                                                                         \
  HG_LAUNCH("hgt_attn_fwd", (k_hgt_attn_fwd<D, S_>), dim3(attn_grid(s->n_sub)), dim3(kAttnThreads), 0, st,     \
            s->n_sub, R, T, (const int32_t*)s->type_off, (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col, \
            (const float*)sv.Q, (const float*)sv.Kt, (const float*)sv.Vt, W->mu, inv_sqrt_dk, sv.ht, sv.lse)
    switch (D / S) {
      case 4: HG_ATTN_FWD(D / 4); break;
      case 8: HG_ATTN_FWD(D / 8); break;
      case 16: HG_ATTN_FWD(D / 16); break;
      case 32: HG_ATTN_FWD(D / 32); break;
      case 64: HG_ATTN_FWD(D / 64); break;
      case 128: if constexpr (D >= 128) { HG_ATTN_FWD(D / 128); } break;
      default: return fail(HG_ERR_UNSUPPORTED, "attention layer: head width %d", D / S);
    }
#undef HG_ATTN_FWD
  }
  // (4) aggregation transform, ReLU, residual, mask
  for (int t = 0; t < T; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    StoreReluMask<D> ep{Hout, rows_contig(lo), W->b_agg ? W->b_agg + (int64_t)t * D : nullptr,
                        L->residual ? Hin : nullptr, mask, L->relu};
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_agg", hi - lo, W->W_agg + (int64_t)t * D * D,
                                          LoadRows<D, float>{sv.ht, rows_contig(lo)}, ep, st)));
  }
  return HG_OK;
}

size_t saved_size(const hg_subgraph* s, int d, int S) {
  Sizer z;
  HgtSaved sv;
  sv.layout(z, s, d, S);
  return z.used;
}

}  // namespace
}  // namespace hg

using namespace hg;

extern "C" {

size_t hg_hgt_saved_size(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L || !hgt_shape_ok(L->d, L->heads)) return 0;
  return saved_size(s, L->d, L->heads);
}

size_t hg_hgt_fwd_workspace_size(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L || !hgt_shape_ok(L->d, L->heads)) return 0;
  Sizer z;
  HgtFwdWs w;
  w.layout(z, s, L->d);
  return z.used;
}

size_t hg_hgt_bwd_workspace_size(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L || !hgt_shape_ok(L->d, L->heads)) return 0;
  return 0;
}

int hg_hgt_fwd(const hg_subgraph* s, const hg_hgt_desc* L, const void* H_in, const hg_hgt_weights* W, void* H_out,
               void* mask, void* saved, void* ws, size_t ws_bytes, void* stream) {
  HG_TRY(validate_hgt(s, L));
  if (!H_in || !H_out || !mask || !saved || !W)
    return fail(HG_ERR_ARG, "null input, output, mask, saved or weights pointer");
  if (!W->W_K || !W->W_Q || !W->W_V || !W->W_att || !W->W_msg || !W->mu || !W->W_agg)
    return fail(HG_ERR_ARG, "null weight pointer (only biases may be NULL)");
  if (H_in == H_out) return fail(HG_ERR_ARG, "H_out must not alias H_in");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  if (L->d == 64)
    return hgt_fwd_impl<64>(s, L, static_cast<const float*>(H_in), W, static_cast<float*>(H_out),
                            static_cast<uint32_t*>(mask), saved, ws, ws_bytes, st);
  return hgt_fwd_impl<128>(s, L, static_cast<const float*>(H_in), W, static_cast<float*>(H_out),
                           static_cast<uint32_t*>(mask), saved, ws, ws_bytes, st);
}

int hg_hgt_bwd(const hg_subgraph* s, const hg_hgt_desc* L, const void*, const hg_hgt_weights*, const void*,
               const void*, const void*, void*, const hg_hgt_grads*, void*, size_t, void*) {
  HG_TRY(validate_hgt(s, L));
  return fail(HG_ERR_UNSUPPORTED, "attention-layer backward is not built yet");
}

}  // extern "C"
