// Heterogeneous graph transformer layer (the attention, message, softmax,
// aggregation and update equations E6-E11 of the "Heterogeneous Graph
// Transformer" paragraph), float32.
//
// Forward:
//   1. K, Q, V: per-type projections with bias (pipelined fp32 MFMA GEMM);
//   2. Kt = K W_att[r], Vt = V W_msg[r] for the active sources of each
//      relation (the per-head dk x dk blocks expanded to one block-diagonal
//      d x d matrix per relation), one row per active (source, relation)
//      slot like the mean layer's relation transforms;
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
  if ((L->relu != 0 && L->relu != 1) || (L->residual != 0 && L->residual != 1) || (L->lean != 0 && L->lean != 1))
    return fail(HG_ERR_ARG, "relu, residual and lean must be 0 or 1");
  if (s->n_rel < 1 || s->n_ntype < 1) return fail(HG_ERR_ARG, "subgraph has no relations or node types");
  if (s->n_sub < 0 || s->e_sub < 0) return fail(HG_ERR_ARG, "subgraph sizes are negative");
  if (s->weighted) return fail(HG_ERR_UNSUPPORTED, "attention layer: edge weights are not supported");
  return HG_OK;
}

// Layout of `saved` (float32 unless noted).
// The forward's intermediates for the backward.  A lean layer keeps Kt and
// Vt out of them (they are 5/7 of the bytes at R = 5): the forward writes them
// to its workspace and the backward computes them again from K and V, two row
// transforms instead of a whole forward, so that a caller holding the layers
// of several snapshots at once keeps 2/7 of the bytes per layer.
struct HgtSaved {
  float *K, *Q, *V;   // [n_sub, d]
  float *Kt, *Vt;     // [A, d], one row per active (source, relation) slot; absent when lean
  float* ht;          // [n_sub, d]
  float* lse;         // [n_sub, S]
  template <class A>
  void layout(A& a, const hg_subgraph* s, int d, int S, bool lean) {
    const int64_t n = s->n_sub, nr = lean ? 0 : n_slots(s);
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
  float *Kt, *Vt;      // lean layers: [A, d]
  float *pacc, *pml;   // chunks of long destination rows: [parts, d], [parts, 2 S] (2 S <= d / 2)
  template <class A>
  void layout(A& a, const hg_subgraph* s, int d, bool lean) {
    const int64_t nr = lean ? n_slots(s) : 0;
    Watt = a.template take<float>((int64_t)s->n_rel * d * d);
    Wmsg = a.template take<float>((int64_t)s->n_rel * d * d);
    Kt = a.template take<float>(nr * d);
    Vt = a.template take<float>(nr * d);
    pacc = a.template take<float>(s->plan_fwd_parts * d);
    pml = a.template take<float>(s->plan_fwd_parts * (d / 2));
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

// Online softmax over the CSR entries [beg, end) of destination row j
// (entries [p0, pe) over all relations): per lane the running max m, sum ls
// and weighted value sum acc of its slot and head, merged over the slots at
// the end (every lane then holds its head's state of the whole range).
template <int D, int S>
__device__ __forceinline__ void attn_fwd_range(int64_t j, int tj, int32_t R, int32_t T,
                                               const int32_t* __restrict__ type_off,
                                               const int32_t* __restrict__ csr_ptr,
                                               const int32_t* __restrict__ csr_col,
                                               const int32_t* __restrict__ csr_slot, const float* __restrict__ Kt,
                                               const float* __restrict__ Vt, const float* __restrict__ mu,
                                               float inv_sqrt_dk, int32_t beg, int32_t end, f32x4 q, int l,
                                               float& m, float& ls, f32x4& acc) {
  constexpr int LPR = D / 4, EPW = 64 / LPR, DK = D / S, LPH = DK / 4, U = 2;
  const int slot = l / LPR, c0 = (l % LPR) * 4;
  const int64_t rb = j * R;
  m = -INFINITY;
  ls = 0.f;
  acc = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int32_t base = beg; base < end; base += 64) {
    const int32_t pos = base + l;
    int32_t rowi = 0;
    float cf = 0.f;
    if (pos < end) {
      const int32_t src = csr_col[pos];
      int r = 0;
      for (int t = 1; t < R; ++t) r += (csr_ptr[rb + t] <= pos) ? 1 : 0;
      rowi = csr_slot ? csr_slot[pos] : src * R + r;
      cf = mu[((int64_t)type_of(src, T, type_off) * R + r) * T + tj] * inv_sqrt_dk;
    }
    const int cnt = (end - base) < 64 ? (end - base) : 64;
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
}

// One wave per destination row; the row's lanes form 64 / (D/4) slots that
// take alternate in-edges, each slot with its own online-softmax state per
// head (lanes of one head hold its dk columns); the slot states are merged at
// the end.  U in-edges per slot are in flight (two row gathers each).  Rows
// of more than kFwdChunk entries are left to the plan's chunks
// (k_hgt_attn_fwd_part, k_hgt_attn_fwd_merge).
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_attn_fwd(
    int64_t n_sub, int32_t R, int32_t T, const int32_t* __restrict__ type_off, const int32_t* __restrict__ csr_ptr,
    const int32_t* __restrict__ csr_col, const int32_t* __restrict__ csr_slot, const float* __restrict__ Q,
    const float* __restrict__ Kt, const float* __restrict__ Vt, const float* __restrict__ mu, float inv_sqrt_dk,
    float* __restrict__ ht, float* __restrict__ lse) {
  constexpr int LPR = D / 4, DK = D / S, LPH = DK / 4;
  static_assert(LPH >= 1 && (LPH & (LPH - 1)) == 0, "head width must be a power of two >= 4");
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t j = wave0; j < n_sub; j += nwaves) {
    const int64_t rb = j * R;
    const int32_t p0 = csr_ptr[rb], pe = csr_ptr[rb + R];
    if (pe - p0 > kFwdChunk) continue;  // a chunked row
    const int tj = type_of(j, T, type_off);
    const f32x4 q = *reinterpret_cast<const f32x4*>(Q + j * D + c0);
    float m, ls;
    f32x4 acc;
    attn_fwd_range<D, S>(j, tj, R, T, type_off, csr_ptr, csr_col, csr_slot, Kt, Vt, mu, inv_sqrt_dk, p0, pe, q, l,
                         m, ls, acc);
    if (slot == 0) {
      const float inv = ls > 0.f ? 1.0f / ls : 0.f;
      *reinterpret_cast<f32x4*>(ht + j * D + c0) = acc * inv;
      if (lr % LPH == 0) lse[j * S + head] = ls > 0.f ? m + logf(ls) : -INFINITY;
    }
  }
}

// One wave per chunk (j, begin, end, partial slot) of a long destination row:
// the chunk's softmax state, acc into pacc [part, D] and (m, ls) per head
// into pml [part, 2 S].
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_attn_fwd_part(
    int64_t n_items, const int4* __restrict__ items, int32_t R, int32_t T, const int32_t* __restrict__ type_off,
    const int32_t* __restrict__ csr_ptr, const int32_t* __restrict__ csr_col, const int32_t* __restrict__ csr_slot,
    const float* __restrict__ Q, const float* __restrict__ Kt, const float* __restrict__ Vt,
    const float* __restrict__ mu, float inv_sqrt_dk, float* __restrict__ pacc, float* __restrict__ pml) {
  constexpr int LPR = D / 4, DK = D / S, LPH = DK / 4;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t it = wave0; it < n_items; it += nwaves) {
    const int4 item = items[it];
    const int64_t j = item.x;
    const int tj = type_of(j, T, type_off);
    const f32x4 q = *reinterpret_cast<const f32x4*>(Q + j * D + c0);
    float m, ls;
    f32x4 acc;
    attn_fwd_range<D, S>(j, tj, R, T, type_off, csr_ptr, csr_col, csr_slot, Kt, Vt, mu, inv_sqrt_dk, item.y,
                         item.z, q, l, m, ls, acc);
    if (slot == 0) {
      *reinterpret_cast<f32x4*>(pacc + (int64_t)item.w * D + c0) = acc;
      if (lr % LPH == 0) {
        pml[(int64_t)item.w * 2 * S + head] = m;
        pml[(int64_t)item.w * 2 * S + S + head] = ls;
      }
    }
  }
}

// One wave per long row (j, first partial, count): the chunks' softmax states
// combined in chunk order, then h~_j and the log-sum-exps.  Every chunk holds
// at least one entry, so every m is finite.
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_attn_fwd_merge(int64_t n_heavy, const int4* __restrict__ heavy,
                                                                     const float* __restrict__ pacc,
                                                                     const float* __restrict__ pml,
                                                                     float* __restrict__ ht, float* __restrict__ lse) {
  constexpr int LPR = D / 4, DK = D / S, LPH = DK / 4;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t h = wave0; h < n_heavy; h += nwaves) {
    const int4 hv = heavy[h];
    if (slot != 0) continue;
    float m = -INFINITY, ls = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int32_t c = 0; c < hv.z; ++c) {
      const int64_t pi = hv.y + c;
      const float m2 = pml[pi * 2 * S + head], l2 = pml[pi * 2 * S + S + head];
      const f32x4 a2 = *reinterpret_cast<const f32x4*>(pacc + pi * D + c0);
      const float mn = fmaxf(m, m2);
      const float s1 = (m == -INFINITY) ? 0.f : __expf(m - mn);
      const float s2 = __expf(m2 - mn);
      ls = ls * s1 + l2 * s2;
      acc = acc * s1 + a2 * s2;
      m = mn;
    }
    const int64_t j = hv.x;
    const float inv = ls > 0.f ? 1.0f / ls : 0.f;
    *reinterpret_cast<f32x4*>(ht + j * D + c0) = acc * inv;
    if (lr % LPH == 0) lse[j * S + head] = ls > 0.f ? m + logf(ls) : -INFINITY;
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

// Kt = K W_att[r] and Vt = V W_msg[r] for the active sources of each
// relation, at the rows of their slots (Watt, Wmsg: the block-diagonal
// expansions).
template <int D>
int rel_transforms(const hg_subgraph* s, const PlanView& pv, const float* Watt, const float* Wmsg, const float* K,
                   const float* V, float* Kt, float* Vt, hipStream_t st) {
  const int32_t R = s->n_rel;
  int64_t off = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t n = s->n_active[r];
    const float* wa = Watt + (int64_t)r * D * D;
    const float* wm = Wmsg + (int64_t)r * D * D;
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_rel", n, wa, LoadRows<D, float>{K, rows_list(pv.active + off)},
                                          StoreRows<D, float>{Kt, rows_list(pv.act_slot + off), nullptr, nullptr},
                                          st)));
    HG_TRY((launch_gemm_rows_pp<D, false>("hgt_rel", n, wm, LoadRows<D, float>{V, rows_list(pv.active + off)},
                                          StoreRows<D, float>{Vt, rows_list(pv.act_slot + off), nullptr, nullptr},
                                          st)));
    off += n;
  }
  return HG_OK;
}

template <int D>
int hgt_fwd_impl(const hg_subgraph* s, const hg_hgt_desc* L, const float* Hin, const hg_hgt_weights* W,
                 float* Hout, uint32_t* mask, void* saved, void* ws, size_t ws_bytes, hipStream_t st) {
  const int S = L->heads;
  const int32_t R = s->n_rel, T = s->n_ntype;
  const bool lean = L->lean != 0;
  Arena as(saved, (size_t)-1);
  HgtSaved sv;
  sv.layout(as, s, D, S, lean);
  Arena a(ws, ws_bytes);
  HgtFwdWs w;
  w.layout(a, s, D, lean);
  float* Kt = lean ? w.Kt : sv.Kt;
  float* Vt = lean ? w.Vt : sv.Vt;
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
  HG_TRY(rel_transforms<D>(s, pv, w.Watt, w.Wmsg, sv.K, sv.V, Kt, Vt, st));
  // (3) attention-weighted aggregation
  const float inv_sqrt_dk = 1.0f / std::sqrt((float)(D / S));
  if (s->n_sub > 0) {
#define HG_ATTN_FWD(S_)                                                                                         \
  do {                                                                                                          \
    HG_LAUNCH("hgt_attn_fwd", (k_hgt_attn_fwd<D, S_>), dim3(attn_grid(s->n_sub)), dim3(kAttnThreads), 0, st,   \
              s->n_sub, R, T, (const int32_t*)s->type_off, (const int32_t*)s->csr_ptr,                          \
              (const int32_t*)s->csr_col, pv.csr_slot, (const float*)sv.Q, (const float*)Kt, (const float*)Vt,  \
              W->mu, inv_sqrt_dk, sv.ht, sv.lse);                                                               \
    if (s->plan_fwd_heavy > 0) {                                                                                \
      HG_LAUNCH("hgt_attn_fwd_part", (k_hgt_attn_fwd_part<D, S_>), dim3(attn_grid(s->plan_fwd_parts)),          \
                dim3(kAttnThreads), 0, st, (int64_t)s->plan_fwd_parts, pv.fwd_items, R, T,                      \
                (const int32_t*)s->type_off, (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col,            \
                pv.csr_slot, (const float*)sv.Q, (const float*)Kt, (const float*)Vt, W->mu, inv_sqrt_dk,        \
                w.pacc, w.pml);                                                                                 \
      HG_LAUNCH("hgt_attn_fwd_merge", (k_hgt_attn_fwd_merge<D, S_>), dim3(attn_grid(s->plan_fwd_heavy)),        \
                dim3(kAttnThreads), 0, st, (int64_t)s->plan_fwd_heavy, pv.fwd_heavy, (const float*)w.pacc,      \
                (const float*)w.pml, sv.ht, sv.lse);                                                            \
    }                                                                                                           \
  } while (0)
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


// ---- backward ------------------------------------------------------------------
// With alpha^s(e) recomputed from the saved log-sum-exp, dalpha = dh~_j . msg
// and D_j^s = dh~_j^s . h~_j^s (= sum_e alpha dalpha):
//   dscore^s(e) = alpha (dalpha - D_j^s)
//   dQ_j   += dscore c Kt(e),  dKt(e) += dscore c Q_j,  dVt(e) += alpha dh~_j
//   dmu    += dscore (Kt(e) . Q_j) / sqrt(dk)
// The destination pass (CSR rows) produces dQ, D and per-row sums for dmu;
// the source pass (CSC work items of the plan) produces dKt and dVt.
constexpr int kMaxTypesBwd = 4;

struct HgtBwdWs {
  float *dZ, *dht, *dQ, *dK, *dV;  // [n_sub, d]
  float* ld;                       // [n_sub, 2S]: per head the log-sum-exp, then per head D_j
  float* contrib;                  // [e_sub]: each CSR entry's term of the mu gradient (summed over heads)
  float *dKt, *dVt;                // [A, d]
  double *pk, *pv;                 // [plan_partials, d]
  float* rowpart;                  // [n_sub * R * T]: dmu sums of each CSR row, by source type
  float* mupart;                   // [T * R * T, kMuChunks]
  float *Watt, *Wmsg;              // [R, d, d] block-diagonal expansions
  float *gatt, *gmsg;              // [R, d, d] full gradients before the block extraction
  float *splitk, *colsum;          // split-K partials
  float *Kt, *Vt;                  // lean layers: Kt and Vt computed again, [A, d]
  float* pdq;                      // [fwd parts, d]: dQ shares of the chunks of long destination rows
  template <class A>
  void layout(A& a, const hg_subgraph* s, int d, int S, bool lean);
};
constexpr int kMuChunks = 64;

template <class A>
void HgtBwdWs::layout(A& a, const hg_subgraph* s, int d, int S, bool lean) {
  const int64_t n = s->n_sub, R = s->n_rel, T = s->n_ntype;
  dZ = a.template take<float>(n * d);
  dht = a.template take<float>(n * d);
  dQ = a.template take<float>(n * d);
  dK = a.template take<float>(n * d);
  dV = a.template take<float>(n * d);
  ld = a.template take<float>(n * 2 * S);
  contrib = a.template take<float>(s->e_sub);
  dKt = a.template take<float>(n_slots(s) * d);
  dVt = a.template take<float>(n_slots(s) * d);
  pk = a.template take<double>(s->plan_partials * d);
  pv = a.template take<double>(s->plan_partials * d);
  rowpart = a.template take<float>(n * R * T);
  mupart = a.template take<float>(T * R * T * kMuChunks);
  Watt = a.template take<float>(R * d * d);
  Wmsg = a.template take<float>(R * d * d);
  gatt = a.template take<float>(R * d * d);
  gmsg = a.template take<float>(R * d * d);
  splitk = a.template take<float>(splitk_max_chunks() * (int64_t)d * d);
  colsum = a.template take<float>(splitk_max_chunks() * (int64_t)d);
  const int64_t nr = lean ? n_slots(s) : 0;
  Kt = a.template take<float>(nr * d);
  Vt = a.template take<float>(nr * d);
  pdq = a.template take<float>(s->plan_fwd_parts * d);
}

template <int LPH>
__device__ __forceinline__ float head_sum(float v) {
#pragma unroll
  for (int o = 1; o < LPH; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// dq (lane's slot share) += the destination-side terms of the CSR entries
// [beg, end) of row j, and each entry's mu-gradient term (summed over the
// heads) into contrib.  q, g: Q_j and dh~_j columns of the lane; lj, dsum:
// its head's log-sum-exp and D_j.
template <int D, int S>
__device__ __forceinline__ void attn_bwd_dst_range(int64_t j, int tj, int32_t R, int32_t T,
                                                   const int32_t* __restrict__ type_off,
                                                   const int32_t* __restrict__ csr_ptr,
                                                   const int32_t* __restrict__ csr_col,
                                                   const int32_t* __restrict__ csr_slot,
                                                   const float* __restrict__ Kt, const float* __restrict__ Vt,
                                                   const float* __restrict__ mu, float inv_sqrt_dk, int32_t beg,
                                                   int32_t end, f32x4 q, f32x4 g, float lj, float dsum, int l,
                                                   f32x4& dq, float* __restrict__ contrib) {
  constexpr int LPR = D / 4, EPW = 64 / LPR, DK = D / S, LPH = DK / 4, U = 2;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4;
  const bool head_lead = (lr % LPH) == 0;
  const int64_t rb = j * R;
  for (int32_t base = beg; base < end; base += 64) {
    const int32_t pos = base + l;
    int32_t rowi = 0;
    float cf = 0.f;
    if (pos < end) {
      const int32_t src = csr_col[pos];
      int r = 0;
      for (int t = 1; t < R; ++t) r += (csr_ptr[rb + t] <= pos) ? 1 : 0;
      rowi = csr_slot ? csr_slot[pos] : src * R + r;
      cf = mu[((int64_t)type_of(src, T, type_off) * R + r) * T + tj] * inv_sqrt_dk;
    }
    const int cnt = (end - base) < 64 ? (end - base) : 64;
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
        const float dot = head_sum<LPH>(kv[u][0] * q[0] + kv[u][1] * q[1] + kv[u][2] * q[2] + kv[u][3] * q[3]);
        const float dal = head_sum<LPH>(vv[u][0] * g[0] + vv[u][1] * g[1] + vv[u][2] * g[2] + vv[u][3] * g[3]);
        float cm = 0.f;
        if (ok[u]) {
          const float a = __expf(dot * cc[u] - lj);
          const float ds = a * (dal - dsum);
          dq += (ds * cc[u]) * kv[u];
          cm = head_lead ? ds * dot * inv_sqrt_dk : 0.f;
        }
        // the mu term of this entry: sum over the heads of the slot
#pragma unroll
        for (int o = LPH; o < LPR; o <<= 1) cm += __shfl_xor(cm, o, 64);
        if (ok[u] && lr == 0) contrib[base + e + u * EPW + slot] = cm;
      }
    }
  }
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) dq[k] += __shfl_xor(dq[k], o, 64);
}

// Destination pass: one wave per node j over all its in-edges (the relation
// of each entry is found from the row pointers, as in the forward).  Writes
// dQ_j, the packed per-head (log-sum-exp, D_j) record of j, and each CSR
// entry's mu-gradient term (summed over the heads) for k_dmu_rows.  The
// in-edges of rows longer than kFwdChunk are left to the plan's chunks
// (k_hgt_attn_bwd_dst_part, k_hgt_dq_merge); their record is written here.
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_attn_bwd_dst(
    int64_t n_sub, int32_t R, int32_t T, const int32_t* __restrict__ type_off, const int32_t* __restrict__ csr_ptr,
    const int32_t* __restrict__ csr_col, const int32_t* __restrict__ csr_slot, const float* __restrict__ Q,
    const float* __restrict__ Kt, const float* __restrict__ Vt, const float* __restrict__ ht, const float* __restrict__ dht,
    const float* __restrict__ lse, const float* __restrict__ mu, float inv_sqrt_dk, float* __restrict__ dQ,
    float* __restrict__ ld, float* __restrict__ contrib) {
  constexpr int LPR = D / 4, DK = D / S, LPH = DK / 4;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const bool head_lead = (lr % LPH) == 0;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t j = wave0; j < n_sub; j += nwaves) {
    const f32x4 g = *reinterpret_cast<const f32x4*>(dht + j * D + c0);
    const f32x4 h = *reinterpret_cast<const f32x4*>(ht + j * D + c0);
    const float dsum = head_sum<LPH>(g[0] * h[0] + g[1] * h[1] + g[2] * h[2] + g[3] * h[3]);
    const float lj = lse[j * S + head];
    if (slot == 0 && head_lead) {
      ld[j * 2 * S + head] = lj;
      ld[j * 2 * S + S + head] = dsum;
    }
    const int64_t rb = j * R;
    const int32_t p0 = csr_ptr[rb], pe = csr_ptr[rb + R];
    if (pe - p0 > kFwdChunk) continue;  // a chunked row
    const int tj = type_of(j, T, type_off);
    const f32x4 q = *reinterpret_cast<const f32x4*>(Q + j * D + c0);
    f32x4 dq = {0.f, 0.f, 0.f, 0.f};
    attn_bwd_dst_range<D, S>(j, tj, R, T, type_off, csr_ptr, csr_col, csr_slot, Kt, Vt, mu, inv_sqrt_dk, p0, pe, q,
                             g, lj, dsum, l, dq, contrib);
    if (slot == 0) *reinterpret_cast<f32x4*>(dQ + j * D + c0) = dq;
  }
}

// One wave per chunk (j, begin, end, partial slot) of a long destination row:
// the chunk's share of dQ_j into pdq [part, D], and its entries' mu terms.
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_attn_bwd_dst_part(
    int64_t n_items, const int4* __restrict__ items, int32_t R, int32_t T, const int32_t* __restrict__ type_off,
    const int32_t* __restrict__ csr_ptr, const int32_t* __restrict__ csr_col, const int32_t* __restrict__ csr_slot,
    const float* __restrict__ Q, const float* __restrict__ Kt, const float* __restrict__ Vt,
    const float* __restrict__ ht, const float* __restrict__ dht, const float* __restrict__ lse,
    const float* __restrict__ mu, float inv_sqrt_dk, float* __restrict__ pdq, float* __restrict__ contrib) {
  constexpr int LPR = D / 4, DK = D / S, LPH = DK / 4;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t it = wave0; it < n_items; it += nwaves) {
    const int4 item = items[it];
    const int64_t j = item.x;
    const f32x4 g = *reinterpret_cast<const f32x4*>(dht + j * D + c0);
    const f32x4 h = *reinterpret_cast<const f32x4*>(ht + j * D + c0);
    const float dsum = head_sum<LPH>(g[0] * h[0] + g[1] * h[1] + g[2] * h[2] + g[3] * h[3]);
    const float lj = lse[j * S + head];
    const int tj = type_of(j, T, type_off);
    const f32x4 q = *reinterpret_cast<const f32x4*>(Q + j * D + c0);
    f32x4 dq = {0.f, 0.f, 0.f, 0.f};
    attn_bwd_dst_range<D, S>(j, tj, R, T, type_off, csr_ptr, csr_col, csr_slot, Kt, Vt, mu, inv_sqrt_dk, item.y,
                             item.z, q, g, lj, dsum, l, dq, contrib);
    if (slot == 0) *reinterpret_cast<f32x4*>(pdq + (int64_t)item.w * D + c0) = dq;
  }
}

// One wave per long row (j, first partial, count): dQ_j = the chunks' shares
// added in float64 (lane group s takes chunks s, s + G, ...; the groups then
// add in a fixed tree).
template <int D>
__global__ void __launch_bounds__(kAttnThreads) k_hgt_dq_merge(int64_t n_heavy, const int4* __restrict__ heavy,
                                                               const float* __restrict__ pdq, float* __restrict__ dQ) {
  constexpr int LPR = D / 4, EPW = 64 / LPR;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, c0 = (l % LPR) * 4;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t h = wave0; h < n_heavy; h += nwaves) {
    const int4 hv = heavy[h];
    f64x4 sd = {0.0, 0.0, 0.0, 0.0};
    for (int32_t c = slot; c < hv.z; c += EPW) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(pdq + (int64_t)(hv.y + c) * D + c0);
#pragma unroll
      for (int k = 0; k < 4; ++k) sd[k] += (double)x[k];
    }
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
      for (int k = 0; k < 4; ++k) sd[k] += __shfl_xor(sd[k], o, 64);
    if (slot == 0)
      *reinterpret_cast<f32x4*>(dQ + (int64_t)hv.x * D + c0) =
          f32x4{(float)sd[0], (float)sd[1], (float)sd[2], (float)sd[3]};
  }
}

// rowpart[(j R + r) T + ti] = sum of the mu terms of CSR row (j, r) whose
// source has type ti (one thread per row, entries in order).
// Rows of destinations whose in-edges are chunked (more than kFwdChunk over
// all relations) are left to k_dmu_heavy.
__global__ void k_dmu_rows(int64_t n_rows, int32_t R, int32_t T, const int32_t* __restrict__ type_off,
                           const int32_t* __restrict__ csr_ptr, const int32_t* __restrict__ csr_col,
                           const float* __restrict__ contrib, float* __restrict__ rowpart) {
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n_rows; q += (int64_t)gridDim.x * blockDim.x) {
    const int64_t rb = q - q % R;
    if (csr_ptr[rb + R] - csr_ptr[rb] > kFwdChunk) continue;
    float acc[kMaxTypesBwd] = {0.f, 0.f, 0.f, 0.f};
    for (int32_t p = csr_ptr[q]; p < csr_ptr[q + 1]; ++p) {
      const int ti = type_of(csr_col[p], T, type_off);
      const float v = contrib[p];
#pragma unroll
      for (int t = 0; t < kMaxTypesBwd; ++t) acc[t] += (ti == t) ? v : 0.f;
    }
    for (int t = 0; t < T; ++t) rowpart[q * T + t] = acc[t];
  }
}

// Source pass: one wave per work item (CSC row q = i * R + r or a chunk of
// it, at slot item.x); Kt and Vt of the row are read once, Q and dh~
// gathered per out-edge.
// At most 128 VGPRs from four heads on: four waves per SIMD for the gathers
// in flight (130 registers, three waves, made the pass 7% slower); one or
// two heads would spill there.
template <int D, int S>
__global__ void __launch_bounds__(kAttnThreads, S >= 4 ? 4 : 1) k_hgt_attn_bwd_src(
    int64_t n_items, const int4* __restrict__ items, const int32_t* __restrict__ slot_q, int32_t R, int32_t T,
    const int32_t* __restrict__ type_off,
    const int32_t* __restrict__ csc_row, const float* __restrict__ Q, const float* __restrict__ Kt,
    const float* __restrict__ Vt, const float* __restrict__ dht, const float* __restrict__ ld,
    const float* __restrict__ mu, float inv_sqrt_dk, float* __restrict__ dKt,
    float* __restrict__ dVt, double* __restrict__ pk, double* __restrict__ pv) {
  constexpr int LPR = D / 4, EPW = 64 / LPR, DK = D / S, LPH = DK / 4, U = 4;
  const int l = threadIdx.x & 63;
  const int slot = l / LPR, lr = l % LPR, c0 = lr * 4, head = lr / LPH;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t it = wave0; it < n_items; it += nwaves) {
    const int4 item = items[it];
    const int64_t srow = item.x;
    const int32_t qrow = slot_q ? slot_q[srow] : (int32_t)srow;
    const int32_t i = qrow / R, r = qrow % R;
    const int ti = type_of(i, T, type_off);
    const f32x4 kt = *reinterpret_cast<const f32x4*>(Kt + srow * D + c0);
    const f32x4 vt = *reinterpret_cast<const f32x4*>(Vt + srow * D + c0);
    f64x4 dk = {0.0, 0.0, 0.0, 0.0}, dv = {0.0, 0.0, 0.0, 0.0};
    for (int32_t base = item.y; base < item.z; base += 64) {
      const int32_t pos = base + l;
      int32_t jj = 0;
      float cf = 0.f;
      if (pos < item.z) {
        jj = csc_row[pos];
        cf = mu[((int64_t)ti * R + r) * T + type_of(jj, T, type_off)] * inv_sqrt_dk;
      }
      const int cnt = (item.z - base) < 64 ? (item.z - base) : 64;
      for (int e = 0; e < cnt; e += EPW * U) {
        f32x4 qv[U], gv[U];
        float cc[U], lj[U], dj[U];
        bool ok[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int my = e + u * EPW + slot;
          const int64_t j = __shfl(jj, my & 63, 64);
          cc[u] = __shfl(cf, my & 63, 64);
          ok[u] = my < cnt;
          if (ok[u]) {
            qv[u] = *reinterpret_cast<const f32x4*>(Q + j * D + c0);
            gv[u] = *reinterpret_cast<const f32x4*>(dht + j * D + c0);
            lj[u] = ld[j * 2 * S + head];
            dj[u] = ld[j * 2 * S + S + head];
          } else {
            qv[u] = gv[u] = f32x4{0.f, 0.f, 0.f, 0.f};
            lj[u] = dj[u] = 0.f;
          }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const float dot = head_sum<LPH>(kt[0] * qv[u][0] + kt[1] * qv[u][1] + kt[2] * qv[u][2] + kt[3] * qv[u][3]);
          const float dal = head_sum<LPH>(vt[0] * gv[u][0] + vt[1] * gv[u][1] + vt[2] * gv[u][2] + vt[3] * gv[u][3]);
          if (ok[u]) {
            const float a = __expf(dot * cc[u] - lj[u]);
            const float ds = a * (dal - dj[u]);
            const double wk = (double)(ds * cc[u]), wv = (double)a;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              dk[k] += wk * (double)qv[u][k];
              dv[k] += wv * (double)gv[u][k];
            }
          }
        }
      }
    }
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        dk[k] += __shfl_xor(dk[k], o, 64);
        dv[k] += __shfl_xor(dv[k], o, 64);
      }
    if (slot == 0) {
      if (item.w < 0) {
        *reinterpret_cast<f32x4*>(dKt + srow * D + c0) = f32x4{(float)dk[0], (float)dk[1], (float)dk[2], (float)dk[3]};
        *reinterpret_cast<f32x4*>(dVt + srow * D + c0) = f32x4{(float)dv[0], (float)dv[1], (float)dv[2], (float)dv[3]};
      } else {
        *reinterpret_cast<f64x4*>(pk + (int64_t)item.w * D + c0) = dk;
        *reinterpret_cast<f64x4*>(pv + (int64_t)item.w * D + c0) = dv;
      }
    }
  }
}

// Split rows: sum their float64 partial rows in chunk order.
template <int D>
__global__ void k_hgt_heavy_reduce(int64_t n_heavy, const int4* __restrict__ heavy, const double* __restrict__ pk,
                                   const double* __restrict__ pv, float* __restrict__ dKt, float* __restrict__ dVt) {
  // as the mean layer's split-row reduction: the lane groups of the wave take
  // interleaved partials, two per group in flight, fixed-order combination
  constexpr int LPR = D / 4, NG = 64 / LPR;
  const int l = threadIdx.x & 63;
  const int grp = l / LPR, lr = l % LPR;
  const int64_t wave0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nwaves = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t h = wave0; h < n_heavy; h += nwaves) {
    const int4 hv = heavy[h];
    f64x4 a0 = {0.0, 0.0, 0.0, 0.0}, b0 = a0, a1 = a0, b1 = a0;
    const int64_t o = (int64_t)hv.y * D + 4 * lr;
    int32_t c = grp;
    for (; c + NG < hv.z; c += 2 * NG) {
      const f64x4 x0 = *reinterpret_cast<const f64x4*>(pk + o + (int64_t)c * D);
      const f64x4 y0 = *reinterpret_cast<const f64x4*>(pv + o + (int64_t)c * D);
      const f64x4 x1 = *reinterpret_cast<const f64x4*>(pk + o + (int64_t)(c + NG) * D);
      const f64x4 y1 = *reinterpret_cast<const f64x4*>(pv + o + (int64_t)(c + NG) * D);
      a0 += x0;
      b0 += y0;
      a1 += x1;
      b1 += y1;
    }
    if (c < hv.z) {
      a0 += *reinterpret_cast<const f64x4*>(pk + o + (int64_t)c * D);
      b0 += *reinterpret_cast<const f64x4*>(pv + o + (int64_t)c * D);
    }
    f64x4 a = a0 + a1, b = b0 + b1;
#pragma unroll
    for (int m = LPR; m < 64; m <<= 1)
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        a[k] += __shfl_xor(a[k], m, 64);
        b[k] += __shfl_xor(b[k], m, 64);
      }
    if (grp == 0) {
      *reinterpret_cast<f32x4*>(dKt + (int64_t)hv.x * D + 4 * lr) = f32x4{(float)a[0], (float)a[1], (float)a[2], (float)a[3]};
      *reinterpret_cast<f32x4*>(dVt + (int64_t)hv.x * D + 4 * lr) = f32x4{(float)b[0], (float)b[1], (float)b[2], (float)b[3]};
    }
  }
}

// [R, d, d] -> its diagonal blocks [R, S, dk, dk] (added into out when accumulate).
__global__ void k_diagblocks(const float* __restrict__ full, int64_t R, int d, int S, float* __restrict__ out,
                             int accumulate) {
  const int dk = d / S;
  const int64_t total = R * S * dk * dk;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t r = e / ((int64_t)S * dk * dk);
    const int s = (int)((e / ((int64_t)dk * dk)) % S);
    const int a = (int)((e / dk) % dk), b = (int)(e % dk);
    const float v = full[(r * d + s * dk + a) * d + s * dk + b];
    out[e] = accumulate ? out[e] + v : v;
  }
}

// The rows (j, r) of one long destination row j per block: each thread sums
// the entries t, t + 256, ... by source type, then a fixed tree over the
// threads.
constexpr int kDmuThreads = 256;
__global__ void __launch_bounds__(kDmuThreads) k_dmu_heavy(int64_t n_heavy, const int4* __restrict__ heavy, int32_t R,
                                                          int32_t T, const int32_t* __restrict__ type_off,
                                                          const int32_t* __restrict__ csr_ptr,
                                                          const int32_t* __restrict__ csr_col,
                                                          const float* __restrict__ contrib,
                                                          float* __restrict__ rowpart) {
  __shared__ float red[kMaxTypesBwd][kDmuThreads];
  const int tid = threadIdx.x;
  for (int64_t h = blockIdx.x; h < n_heavy; h += gridDim.x) {
    const int64_t j = heavy[h].x;
    for (int32_t r = 0; r < R; ++r) {
      const int64_t q = j * R + r;
      float acc[kMaxTypesBwd] = {0.f, 0.f, 0.f, 0.f};
      for (int32_t p = csr_ptr[q] + tid; p < csr_ptr[q + 1]; p += kDmuThreads) {
        const int ti = type_of(csr_col[p], T, type_off);
        const float v = contrib[p];
#pragma unroll
        for (int t = 0; t < kMaxTypesBwd; ++t) acc[t] += (ti == t) ? v : 0.f;
      }
#pragma unroll
      for (int t = 0; t < kMaxTypesBwd; ++t) red[t][tid] = acc[t];
      __syncthreads();
      for (int o = kDmuThreads / 2; o > 0; o >>= 1) {
        if (tid < o)
#pragma unroll
          for (int t = 0; t < kMaxTypesBwd; ++t) red[t][tid] += red[t][tid + o];
        __syncthreads();
      }
      if (tid < T) rowpart[q * T + tid] = red[tid][0];
      __syncthreads();
    }
  }
}

// dmu[ti][r][tj] = sum over destinations j of type tj of rowpart[(j R + r) T + ti]:
// block (c, m) sums chunk c of the type range in a fixed tree order.
__global__ void __launch_bounds__(256) k_dmu_partial(const float* __restrict__ rowpart, const int32_t* __restrict__ type_off,
                                                    int32_t R, int32_t T, float* __restrict__ mupart) {
  __shared__ float red[256];
  const int m = blockIdx.y;  // (ti * R + r) * T + tj
  const int tj = m % T, r = (m / T) % R, ti = m / (T * R);
  const int64_t lo = type_off[tj], hi = type_off[tj + 1];
  const int64_t per = (hi - lo + kMuChunks - 1) / kMuChunks;
  const int64_t c0 = lo + per * blockIdx.x, c1 = (c0 + per < hi) ? c0 + per : hi;
  float acc = 0.f;
  for (int64_t j = c0 + threadIdx.x; j < c1; j += blockDim.x) acc += rowpart[(j * R + r) * T + ti];
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if (threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) mupart[(int64_t)m * kMuChunks + blockIdx.x] = red[0];
}

__global__ void k_dmu_final(const float* __restrict__ mupart, int M, float* __restrict__ dmu, int accumulate) {
  const int m = blockIdx.x * blockDim.x + threadIdx.x;
  if (m >= M) return;
  float s = 0.f;
  for (int c = 0; c < kMuChunks; ++c) s += mupart[(int64_t)m * kMuChunks + c];
  dmu[m] = accumulate ? dmu[m] + s : s;
}

// out[row0 + i] = addend[row0 + i] + sum_m A_m[row0 + i] W_m^T over three
// row sets of the same rows (dH = G + dK W_K^T + dQ W_Q^T + dV W_V^T): the
// three d x d matrices stay in LDS together (48 KB at d = 64, split-fp16
// fragments as in k_gemm_rows), and each output row is written once instead
// of being read and written again for every product.  Each product is
// unscaled on its own (the rows of A_m have their own scales) and the three
// are added in the order m = 0, 1, 2.
constexpr int kSum3 = 3;
template <int D>
__global__ void __launch_bounds__(kGemmThreads) k_gemm_rows_sum3(int64_t n_rows, int64_t row0,
                                                                 const float* __restrict__ W0,
                                                                 const float* __restrict__ W1,
                                                                 const float* __restrict__ W2,
                                                                 const float* __restrict__ A0,
                                                                 const float* __restrict__ A1,
                                                                 const float* __restrict__ A2,
                                                                 const float* __restrict__ addend,
                                                                 float* __restrict__ out) {
  static_assert(D == 64, "three 64 x 64 matrices in LDS");
  constexpr int KB = D / 16, KB2 = D / 32, NB = D / 16;
  constexpr int kWaves = kGemmThreads / 64;
  constexpr int kRowsPerTile = 16 * kWaves;
  constexpr int kFrag = KB2 * NB * 64;
  __shared__ uint4 wsl[kSum3][2 * kFrag];  // per matrix: high parts, then remainders
  __shared__ float wmax[kWaves];
  __shared__ float uws[kSum3];
  const int tid = threadIdx.x;
  const float* Ws[kSum3] = {W0, W1, W2};
  const float* As[kSum3] = {A0, A1, A2};
#pragma unroll
  for (int mi = 0; mi < kSum3; ++mi) {
    const float* W = Ws[mi];
    float m = 0.f;
    for (int e = tid; e < D * D / 4; e += kGemmThreads) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(W + 4 * e);
      m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if ((tid & 63) == 0) wmax[tid >> 6] = m;
    __syncthreads();
    m = wmax[0];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) m = fmaxf(m, wmax[q]);
    const uint32_t ew = split_exp(m);
    const float sw = split_scale(ew);
    for (int e = tid; e < kFrag; e += kGemmThreads) {
      const int l = e & 63;
      const int nb = (e >> 6) % NB;
      const int kb2 = (e >> 6) / NB;
      const int j = 16 * nb + (l & 15);
      float v[8];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // op(W) = W^T: element (k, j) is W[j][k]
        const f32x4 x = *reinterpret_cast<const f32x4*>(W + (int64_t)j * D + 16 * (2 * kb2 + h) + 4 * (l >> 4));
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * h + q] = x[q] * sw;
      }
      split8(v, wsl[mi][e], wsl[mi][kFrag + e]);
    }
    if (tid == 0) uws[mi] = split_unscale(ew);
    __syncthreads();
  }
  const int w = tid >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  const int64_t ntiles = (n_rows + kRowsPerTile - 1) / kRowsPerTile;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t i = t * kRowsPerTile + 16 * w + c;
    const bool live = i < n_rows;
    const int64_t row = row0 + (live ? i : 0);
    f32x4 tot[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) tot[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // the next operand's row is loaded while the current one is multiplied
    f32x4 nxt[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      nxt[kb] = live ? *reinterpret_cast<const f32x4*>(As[0] + row * D + 16 * kb + 4 * g) : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int mi = 0; mi < kSum3; ++mi) {
      __builtin_amdgcn_sched_barrier(0);
      f32x4 a[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) a[kb] = nxt[kb];
      if (mi + 1 < kSum3) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          nxt[kb] = live ? *reinterpret_cast<const f32x4*>(As[mi + 1] + row * D + 16 * kb + 4 * g)
                         : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      float m = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        m = fmaxf(m, fmaxf(fmaxf(fabsf(a[kb][0]), fabsf(a[kb][1])), fmaxf(fabsf(a[kb][2]), fabsf(a[kb][3]))));
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      const uint32_t ex = split_exp(m);
      const float sx = split_scale(ex), ux = split_unscale(ex);
      uint4 xh[KB2], xlo[KB2];
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = a[2 * kb2][q] * sx;
          v[4 + q] = a[2 * kb2 + 1][q] * sx;
        }
        split8(v, xh[kb2], xlo[kb2]);
      }
      f32x4 acc[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
        // each K block's fragments are read right before its MFMAs
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int e = (kb2 * NB + nb) * 64 + l;
          const uint4 bh = wsl[mi][e], bl = wsl[mi][kFrag + e];
          acc[nb] = mfma_f16(bh, xh[kb2], acc[nb]);
          acc[nb] = mfma_f16(bh, xlo[kb2], acc[nb]);
          acc[nb] = mfma_f16(bl, xh[kb2], acc[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) tot[nb] += split_unscale4(acc[nb], ux, uws[mi]);
    }
    if (live) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = 16 * nb + 4 * g;
        const f32x4 pre = addend ? *reinterpret_cast<const f32x4*>(addend + row * D + col)
                                 : f32x4{0.f, 0.f, 0.f, 0.f};
        *reinterpret_cast<f32x4*>(out + row * D + col) = pre + tot[nb];
      }
    }
  }
}

// out[i] = sum over the relations r with (i, r) active (CSC row i R + r not
// empty, i.e. i in S_r) of A[i R + r] op(W_r), op(W_r) = W_r^T, for every row
// i < n_rows: dK = sum_r dKt_r W_att[r]^T and dV likewise, each row written
// once (no zero fill, no read-modify-write per relation).  The R split-fp16
// matrices sit in LDS together (16 KB each at d = 64, R <= kSumRMax); each
// product is unscaled on its own and added in relation order; a relation no
// row of a wave's 16 is active in costs no MFMA; the next relation's rows are
// loaded while the current ones are multiplied.
constexpr int kSumRMax = 8;
// one block of 16 waves per compute unit: R = 5 matrices take 80 KB, so two
// blocks would need a few bytes more than the 160 KB of LDS
constexpr int kSumRThreads = 1024;
template <int D>
__global__ void __launch_bounds__(kSumRThreads) k_gemm_rows_sumr(int64_t n_rows, int32_t R,
                                                                 const float* __restrict__ W,
                                                                 const float* __restrict__ A,
                                                                 const int32_t* __restrict__ csc_ptr,
                                                                 const SlotEnt* __restrict__ slot_tab,
                                                                 float* __restrict__ out) {
  static_assert(D == 64, "R matrices of 64 x 64 in LDS");
  constexpr int KB = D / 16, KB2 = D / 32, NB = D / 16;
  constexpr int kWaves = kSumRThreads / 64;
  constexpr int kRowsPerTile = 16 * kWaves;
  constexpr int kFrag = KB2 * NB * 64;
  extern __shared__ uint4 wsr[];  // per relation: [kFrag] high parts, then [kFrag] remainders
  __shared__ float wmax[kWaves];
  __shared__ float uws[kSumRMax];
  const int tid = threadIdx.x;
  for (int r = 0; r < R; ++r) {
    const float* Wr = W + (int64_t)r * D * D;
    float m = 0.f;
    for (int e = tid; e < D * D / 4; e += kSumRThreads) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(Wr + 4 * e);
      m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    if ((tid & 63) == 0) wmax[tid >> 6] = m;
    __syncthreads();
    m = wmax[0];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) m = fmaxf(m, wmax[q]);
    const uint32_t ew = split_exp(m);
    const float sw = split_scale(ew);
    uint4* wl = wsr + (int64_t)r * 2 * kFrag;
    for (int e = tid; e < kFrag; e += kSumRThreads) {
      const int l = e & 63;
      const int nb = (e >> 6) % NB;
      const int kb2 = (e >> 6) / NB;
      const int j = 16 * nb + (l & 15);
      float v[8];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // op(W) = W^T: element (k, j) is W[j][k]
        const f32x4 x = *reinterpret_cast<const f32x4*>(Wr + (int64_t)j * D + 16 * (2 * kb2 + h) + 4 * (l >> 4));
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * h + q] = x[q] * sw;
      }
      split8(v, wl[e], wl[kFrag + e]);
    }
    if (tid == 0) uws[r] = split_unscale(ew);
    __syncthreads();
  }
  const int w = tid >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  const int64_t ntiles = (n_rows + kRowsPerTile - 1) / kRowsPerTile;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t i = t * kRowsPerTile + 16 * w + c;
    const bool live = i < n_rows;
    // the row's CSC pointers i R .. i R + R: relation r is active iff its row
    // is not empty; the active relations of row i hold consecutive slots
    // from slot(i R) (row-indexed layout, slot_tab null: rows i R + r)
    int32_t p[kSumRMax + 1];
#pragma unroll
    for (int q = 0; q <= kSumRMax; ++q) p[q] = (live && q <= R) ? csc_ptr[i * R + q] : 0;
    int64_t sl = (live && slot_tab) ? slot_of(slot_tab, i * R) : 0;
    f32x4 tot[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) tot[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 nxt[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
      nxt[kb] = (live && R > 0 && p[1] > p[0])
                    ? *reinterpret_cast<const f32x4*>(A + (slot_tab ? sl : i * R) * D + 16 * kb + 4 * g)
                    : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < kSumRMax; ++r) {
      if (r >= R) break;
      __builtin_amdgcn_sched_barrier(0);
      const bool act = live && p[r + 1] > p[r];
      if (act) ++sl;  // sl: slot of the next active relation of row i
      f32x4 a[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) a[kb] = nxt[kb];
      if (r + 1 < R && r + 1 < kSumRMax) {
        const bool act1 = live && p[r + 2] > p[r + 1];
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
          nxt[kb] = act1 ? *reinterpret_cast<const f32x4*>(A + (slot_tab ? sl : i * R + r + 1) * D + 16 * kb + 4 * g)
                         : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      if (__ballot(act) == 0) continue;  // wave-uniform: no row of the 16 is in S_r
      float m = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
        m = fmaxf(m, fmaxf(fmaxf(fabsf(a[kb][0]), fabsf(a[kb][1])), fmaxf(fabsf(a[kb][2]), fabsf(a[kb][3]))));
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      const uint32_t ex = split_exp(m);
      const float sx = split_scale(ex), ux = split_unscale(ex);
      uint4 xh[KB2], xlo[KB2];
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
        float v[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = a[2 * kb2][q] * sx;
          v[4 + q] = a[2 * kb2 + 1][q] * sx;
        }
        split8(v, xh[kb2], xlo[kb2]);
      }
      const uint4* wl = wsr + (int64_t)r * 2 * kFrag;
      f32x4 acc[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          const int e = (kb2 * NB + nb) * 64 + l;
          const uint4 bh = wl[e], bl = wl[kFrag + e];
          acc[nb] = mfma_f16(bh, xh[kb2], acc[nb]);
          acc[nb] = mfma_f16(bh, xlo[kb2], acc[nb]);
          acc[nb] = mfma_f16(bl, xh[kb2], acc[nb]);
        }
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) tot[nb] += split_unscale4(acc[nb], ux, uws[r]);
    }
    if (live) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        *reinterpret_cast<f32x4*>(out + i * D + 16 * nb + 4 * g) = tot[nb];
    }
  }
}

template <int D>
int launch_gemm_rows_sumr(const char* name, int64_t n_rows, int32_t R, const float* W, const float* A,
                          const int32_t* csc_ptr, const SlotEnt* slot_tab, float* out, hipStream_t st) {
  if (n_rows <= 0) return HG_OK;
  if (R < 1 || R > kSumRMax) return fail(HG_ERR_ARG, "%s: R = %d outside [1, %d]", name, R, kSumRMax);
  const size_t lds = sizeof(uint4) * 2 * ((D / 32) * (D / 16) * 64) * (size_t)R;
  auto kern = k_gemm_rows_sumr<D>;
  if (lds > 65536) {
    static bool attr_set = false;
    if (!attr_set) {
      HG_HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)(sizeof(uint4) * 2 * ((D / 32) * (D / 16) * 64) * kSumRMax)));
      attr_set = true;
    }
  }
  const int64_t tiles = cdiv(n_rows, 16 * (kSumRThreads / 64));
  const int64_t cap = (int64_t)num_cus();
  HG_LAUNCH(name, kern, dim3((unsigned)(tiles < cap ? tiles : cap)), dim3(kSumRThreads), lds, st, n_rows, R, W, A,
            csc_ptr, slot_tab, out);
  return HG_OK;
}

template <int D>
int hgt_bwd_impl(const hg_subgraph* s, const hg_hgt_desc* L, const float* Hin, const hg_hgt_weights* W,
                 const uint32_t* mask, const void* saved, const float* G, float* dHin, const hg_hgt_grads* dW,
                 int acc, void* ws, size_t ws_bytes, hipStream_t st) {
  const int S = L->heads;
  const int32_t R = s->n_rel, T = s->n_ntype;
  const bool lean = L->lean != 0;
  Arena as(const_cast<void*>(saved), (size_t)-1);
  HgtSaved sv;
  sv.layout(as, s, D, S, lean);
  Arena a(ws, ws_bytes);
  HgtBwdWs w;
  w.layout(a, s, D, S, lean);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "attention backward workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  const PlanView pv = plan_view(s);
  const float inv_sqrt_dk = 1.0f / std::sqrt((float)(D / S));
  {
    const int64_t n = (int64_t)R * D * D;
    const unsigned g = (unsigned)(cdiv(n, 256) < 4096 ? cdiv(n, 256) : 4096);
    HG_LAUNCH("hgt_blockdiag", k_blockdiag, dim3(g), dim3(256), 0, st, W->W_att, (int64_t)R, D, S, w.Watt);
    HG_LAUNCH("hgt_blockdiag", k_blockdiag, dim3(g), dim3(256), 0, st, W->W_msg, (int64_t)R, D, S, w.Wmsg);
  }
  // a lean layer's Kt and Vt, from the saved K and V
  if (lean) HG_TRY(rel_transforms<D>(s, pv, w.Watt, w.Wmsg, sv.K, sv.V, w.Kt, w.Vt, st));
  const float* Kt = lean ? w.Kt : sv.Kt;
  const float* Vt = lean ? w.Vt : sv.Vt;
  // (1) dZ = G * mask (written by the A load), dh~ = dZ W_agg^T; dW_agg, db_agg
  for (int t = 0; t < T; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    LoadMasked<D, float> la{G, mask, rows_contig(lo), w.dZ};
    HG_TRY((launch_gemm_rows_pp<D, true>("hgt_bwd_dht", hi - lo, W->W_agg + (int64_t)t * D * D, la,
                                         StoreRows<D, float>{w.dht, rows_contig(lo), nullptr, nullptr}, st)));
    HG_TRY((launch_gemm_tn<D>("hgt_bwd_dw", hi - lo, LoadRows<D, float>{sv.ht, rows_contig(lo)},
                              LoadRows<D, float>{w.dZ, rows_contig(lo)}, w.splitk, w.colsum,
                              dW->W_agg + (int64_t)t * D * D, dW->b_agg ? dW->b_agg + (int64_t)t * D : nullptr, acc, st)));
  }
  // (2) destination pass, (3) source pass
  if (s->n_sub > 0) {
#define HG_ATTN_BWD(S_)                                                                                               \
  do {                                                                                                                \
    HG_LAUNCH("hgt_attn_bwd_dst", (k_hgt_attn_bwd_dst<D, S_>), dim3(attn_grid(s->n_sub)), dim3(kAttnThreads), 0, st, \
              s->n_sub, R, T, (const int32_t*)s->type_off, (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col,   \
              pv.csr_slot, (const float*)sv.Q, Kt, Vt, (const float*)sv.ht,                                           \
              (const float*)w.dht, (const float*)sv.lse, W->mu, inv_sqrt_dk, w.dQ, w.ld, w.contrib);                 \
    if (s->plan_fwd_heavy > 0) {                                                                                      \
      HG_LAUNCH("hgt_attn_bwd_dst_part", (k_hgt_attn_bwd_dst_part<D, S_>), dim3(attn_grid(s->plan_fwd_parts)),        \
                dim3(kAttnThreads), 0, st, (int64_t)s->plan_fwd_parts, pv.fwd_items, R, T,                            \
                (const int32_t*)s->type_off, (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col, pv.csr_slot,    \
                (const float*)sv.Q, Kt, Vt, (const float*)sv.ht, (const float*)w.dht, (const float*)sv.lse, W->mu,   \
                inv_sqrt_dk, w.pdq, w.contrib);                                                                       \
      HG_LAUNCH("hgt_dq_merge", k_hgt_dq_merge<D>, dim3(attn_grid(s->plan_fwd_heavy)), dim3(kAttnThreads), 0, st,     \
                (int64_t)s->plan_fwd_heavy, pv.fwd_heavy, (const float*)w.pdq, w.dQ);                                 \
    }                                                                                                                 \
    if (s->plan_items > 0)                                                                                            \
      HG_LAUNCH("hgt_attn_bwd_src", (k_hgt_attn_bwd_src<D, S_>), dim3(attn_grid(s->plan_items)), dim3(kAttnThreads),  \
                0, st, (int64_t)s->plan_items, pv.items, pv.slot_q, R, T, (const int32_t*)s->type_off,                \
                (const int32_t*)s->csc_row, (const float*)sv.Q, Kt, Vt,                                               \
                (const float*)w.dht, (const float*)w.ld, W->mu, inv_sqrt_dk, w.dKt, w.dVt,                            \
                w.pk, w.pv);                                                                                          \
  } while (0)
    switch (D / S) {
      case 4: HG_ATTN_BWD(D / 4); break;
      case 8: HG_ATTN_BWD(D / 8); break;
      case 16: HG_ATTN_BWD(D / 16); break;
      case 32: HG_ATTN_BWD(D / 32); break;
      case 64: HG_ATTN_BWD(D / 64); break;
      case 128: if constexpr (D >= 128) { HG_ATTN_BWD(D / 128); } break;
      default: return fail(HG_ERR_UNSUPPORTED, "attention layer: head width %d", D / S);
    }
#undef HG_ATTN_BWD
    if (s->plan_heavy > 0)
      HG_LAUNCH("hgt_bwd_heavy", k_hgt_heavy_reduce<D>, dim3(attn_grid(s->plan_heavy)), dim3(kAttnThreads), 0, st,
                (int64_t)s->plan_heavy, pv.heavy, (const double*)w.pk, (const double*)w.pv, w.dKt, w.dVt);
  }
  // (4) dK = sum_r dKt_r W_att[r]^T, dV = sum_r dVt_r W_msg[r]^T over the rows
  // of S_r; full dW_att, dW_msg
  const bool fused_rel = D == 64 && R <= kSumRMax;
  if (fused_rel) {
    if constexpr (D == 64) {
      HG_TRY(launch_gemm_rows_sumr<D>("hgt_bwd_dx_rel", s->n_sub, R, w.Watt, w.dKt, (const int32_t*)s->csc_ptr, pv.slot_tab,
                                      w.dK, st));
      HG_TRY(launch_gemm_rows_sumr<D>("hgt_bwd_dx_rel", s->n_sub, R, w.Wmsg, w.dVt, (const int32_t*)s->csc_ptr, pv.slot_tab,
                                      w.dV, st));
    }
  } else {
    HG_TRY(fill_f32(w.dK, 0.f, s->n_sub * (int64_t)D, st));
    HG_TRY(fill_f32(w.dV, 0.f, s->n_sub * (int64_t)D, st));
  }
  int64_t off = 0;
  for (int r = 0; r < R; ++r) {
    const int64_t n = s->n_active[r];
    const int64_t wo = (int64_t)r * D * D;
    if (!fused_rel) {
      HG_TRY((launch_gemm_rows_pp<D, true>("hgt_bwd_dx_rel", n, w.Watt + wo,
                                           LoadRows<D, float>{w.dKt, rows_list(pv.act_slot + off)},
                                           StoreRows<D, float>{w.dK, rows_list(pv.active + off), nullptr, w.dK}, st)));
      HG_TRY((launch_gemm_rows_pp<D, true>("hgt_bwd_dx_rel", n, w.Wmsg + wo,
                                           LoadRows<D, float>{w.dVt, rows_list(pv.act_slot + off)},
                                           StoreRows<D, float>{w.dV, rows_list(pv.active + off), nullptr, w.dV}, st)));
    }
    HG_TRY((launch_gemm_tn<D>("hgt_bwd_dw", n, LoadRows<D, float>{sv.K, rows_list(pv.active + off)},
                              LoadRows<D, float>{w.dKt, rows_list(pv.act_slot + off)}, w.splitk, w.colsum,
                              w.gatt + wo, nullptr, 0, st)));
    HG_TRY((launch_gemm_tn<D>("hgt_bwd_dw", n, LoadRows<D, float>{sv.V, rows_list(pv.active + off)},
                              LoadRows<D, float>{w.dVt, rows_list(pv.act_slot + off)}, w.splitk, w.colsum,
                              w.gmsg + wo, nullptr, 0, st)));
    off += n;
  }
  {
    const int64_t n = (int64_t)R * D * D / S;
    const unsigned g = (unsigned)(cdiv(n, 256) < 4096 ? cdiv(n, 256) : 4096);
    HG_LAUNCH("hgt_diagblocks", k_diagblocks, dim3(g), dim3(256), 0, st, (const float*)w.gatt, (int64_t)R, D, S, dW->W_att,
              acc);
    HG_LAUNCH("hgt_diagblocks", k_diagblocks, dim3(g), dim3(256), 0, st, (const float*)w.gmsg, (int64_t)R, D, S, dW->W_msg,
              acc);
  }
  // (5) dH = G (residual) + dK W_K^T + dQ W_Q^T + dV W_V^T per type; projection gradients
  for (int t = 0; t < T; ++t) {
    const int64_t lo = s->type_off_host[t], hi = s->type_off_host[t + 1];
    const int64_t wo = (int64_t)t * D * D, bo = (int64_t)t * D;
    const float* srcs[3] = {w.dK, w.dQ, w.dV};
    const float* Ws[3] = {W->W_K, W->W_Q, W->W_V};
    float* dWs[3] = {dW->W_K, dW->W_Q, dW->W_V};
    float* dbs[3] = {dW->b_K, dW->b_Q, dW->b_V};
    if constexpr (D == 64) {
      // the three products in one pass (their matrices fit LDS together)
      const int64_t n = hi - lo;
      if (n > 0) {
        const int64_t tiles = cdiv(n, 16 * (kGemmThreads / 64));
        const int64_t cap = (int64_t)num_cus() * 3;
        HG_LAUNCH("hgt_bwd_dx", k_gemm_rows_sum3<D>, dim3((unsigned)(tiles < cap ? tiles : cap)), dim3(kGemmThreads),
                  0, st, n, lo, W->W_K + wo, W->W_Q + wo, W->W_V + wo, (const float*)w.dK, (const float*)w.dQ,
                  (const float*)w.dV, L->residual ? G : nullptr, dHin);
      }
    } else {
      for (int k = 0; k < 3; ++k) {
        const float* addend = (k == 0) ? (L->residual ? G : nullptr) : dHin;
        HG_TRY((launch_gemm_rows_pp<D, true>("hgt_bwd_dx", hi - lo, Ws[k] + wo,
                                             LoadRows<D, float>{srcs[k], rows_contig(lo)},
                                             StoreRows<D, float>{dHin, rows_contig(lo), nullptr, addend}, st)));
      }
    }
    for (int k = 0; k < 3; ++k)
      HG_TRY((launch_gemm_tn<D>("hgt_bwd_dw", hi - lo, LoadRows<D, float>{Hin, rows_contig(lo)},
                                LoadRows<D, float>{srcs[k], rows_contig(lo)}, w.splitk, w.colsum, dWs[k] + wo,
                                dbs[k] ? dbs[k] + bo : nullptr, acc, st)));
  }
  // (6) dmu: per CSR row by source type, then per meta relation over each type range
  {
    const int64_t nq = s->n_sub * (int64_t)R;
    if (nq > 0)
      HG_LAUNCH("hgt_bwd_dmu", k_dmu_rows, dim3((unsigned)(cdiv(nq, 256) < 65536 ? cdiv(nq, 256) : 65536)), dim3(256), 0,
                st, nq, R, T, (const int32_t*)s->type_off, (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col,
                (const float*)w.contrib, w.rowpart);
    if (s->plan_fwd_heavy > 0)
      HG_LAUNCH("hgt_bwd_dmu", k_dmu_heavy, dim3((unsigned)(s->plan_fwd_heavy < 65536 ? s->plan_fwd_heavy : 65536)),
                dim3(kDmuThreads), 0, st, (int64_t)s->plan_fwd_heavy, pv.fwd_heavy, R, T, (const int32_t*)s->type_off,
                (const int32_t*)s->csr_ptr, (const int32_t*)s->csr_col, (const float*)w.contrib, w.rowpart);
    const int M = T * R * T;
    HG_LAUNCH("hgt_bwd_dmu", k_dmu_partial, dim3(kMuChunks, M), dim3(256), 0, st, (const float*)w.rowpart,
              (const int32_t*)s->type_off, R, T, w.mupart);
    HG_LAUNCH("hgt_bwd_dmu", k_dmu_final, dim3((unsigned)cdiv(M, 256)), dim3(256), 0, st, (const float*)w.mupart, M,
              dW->mu, acc);
  }
  return HG_OK;
}

size_t saved_size(const hg_subgraph* s, int d, int S, bool lean) {
  Sizer z;
  HgtSaved sv;
  sv.layout(z, s, d, S, lean);
  return z.used;
}

}  // namespace
}  // namespace hg

using namespace hg;

extern "C" {

size_t hg_hgt_saved_size(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L || !hgt_shape_ok(L->d, L->heads)) return 0;
  return saved_size(s, L->d, L->heads, L->lean != 0);
}

size_t hg_hgt_fwd_workspace_size(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L || !hgt_shape_ok(L->d, L->heads)) return 0;
  Sizer z;
  HgtFwdWs w;
  w.layout(z, s, L->d, L->lean != 0);
  return z.used;
}

size_t hg_hgt_bwd_workspace_size(const hg_subgraph* s, const hg_hgt_desc* L) {
  if (!s || !L || !hgt_shape_ok(L->d, L->heads)) return 0;
  Sizer z;
  HgtBwdWs w;
  w.layout(z, s, L->d, L->heads, L->lean != 0);
  return z.used;
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

int hg_hgt_bwd(const hg_subgraph* s, const hg_hgt_desc* L, const void* H_in, const hg_hgt_weights* W,
               const void* mask, const void* saved, const void* dH_out, void* dH_in, const hg_hgt_grads* dW,
               int32_t accumulate, void* ws, size_t ws_bytes, void* stream) {
  HG_TRY(validate_hgt(s, L));
  if (accumulate != 0 && accumulate != 1) return fail(HG_ERR_ARG, "accumulate must be 0 or 1");
  if (s->n_ntype > kMaxTypesBwd)
    return fail(HG_ERR_UNSUPPORTED, "attention-layer backward: at most %d node types (got %d)", kMaxTypesBwd,
                s->n_ntype);
  if (!H_in || !mask || !saved || !dH_out || !dH_in || !W || !dW)
    return fail(HG_ERR_ARG, "null input, mask, saved, gradient or weights pointer");
  if (!W->W_K || !W->W_Q || !W->W_V || !W->W_att || !W->W_msg || !W->mu || !W->W_agg)
    return fail(HG_ERR_ARG, "null weight pointer (only biases may be NULL)");
  if (!dW->W_K || !dW->W_Q || !dW->W_V || !dW->W_att || !dW->W_msg || !dW->mu || !dW->W_agg)
    return fail(HG_ERR_ARG, "null weight-gradient pointer (only bias gradients may be NULL)");
  if (dH_in == dH_out || dH_in == H_in) return fail(HG_ERR_ARG, "dH_in must not alias dH_out or H_in");
  const hipStream_t st = static_cast<hipStream_t>(stream);
  const float* Hin = static_cast<const float*>(H_in);
  const uint32_t* m = static_cast<const uint32_t*>(mask);
  const float* G = static_cast<const float*>(dH_out);
  float* dH = static_cast<float*>(dH_in);
  if (L->d == 64) return hgt_bwd_impl<64>(s, L, Hin, W, m, saved, G, dH, dW, accumulate, ws, ws_bytes, st);
  return hgt_bwd_impl<128>(s, L, Hin, W, m, saved, G, dH, dW, accumulate, ws, ws_bytes, st);
}

}  // extern "C"
