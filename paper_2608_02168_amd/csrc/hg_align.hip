// hg_align_loss_fwd_bwd: CCA consistency-alignment loss on the overlap batch
// (Section "Cross-Subgraph Consistency Alignment": standardisation,
// invariance, decorrelation and CCA-loss equations) and its gradient, in
// three passes over the two views X = H[overlap] and Y = H_ref:
//
//   (d1) k_align_stats: per-column float64 sums of x and x^2 of both views,
//        one partial row set per chunk of rows;
//   (d2) k_align_gram: every block first reduces (d1) in a fixed order, so
//        all blocks hold the same mean, 1/sigma and standardisation scale;
//        then over its chunk of rows the Gram matrices Xh^T Xh and Yh^T Yh
//        on the split-fp16 MFMA (only the blocks on and above the diagonal)
//        and, in float64, the column sums the gradient and the loss need:
//          v = sum Xh, w = sum Yh, u = sum o (Xh - Yh),
//          p = sum o (Xh - Yh) Xh, q = sum o (Yh - Xh) Yh, l = sum o (Xh - Yh)^2
//        (o the row weight).  The last block of every group of 16 chunks
//        sums the group's partials in chunk order, and the last group to
//        finish sums the groups in order, mirrors the Grams, and writes
//        C' = Xh^T Xh - I (and of Y), the loss and the two column vectors of
//        the standardisation backward: with G = 2 o (Xh - Yh) + 4 lambda Xh C'
//        and g' = G / sqrt(M),
//          S1 = sum_b g'_b = (2 u + 4 lambda v C') / sqrt(M),
//          S2 = sum_b g'_b xt_b = 2 p + 4 lambda diag(C C')
//        (xt = (x - mu) / sigma = Xh sqrt(M)), so G never reaches memory;
//   (d3) the gradient row GEMM Xh C' on the split-fp16 MFMA whose epilogue
//        forms G, the standardisation backward
//          dX = (1/sigma) (g' - S1 / M - xt S2 / (M - ddof))
//        and writes dH[overlap] = base + scale * dX (rows are distinct: no
//        atomics); the same for Y into dH_ref when it is requested.
//
// The counters of (d2) are zeroed by (d1), which runs first on the stream.
// Every reduction has a fixed order: results are bitwise reproducible.
#include <mutex>

#include "hg_internal.h"
#include "hg_mfma.h"

namespace hg {

namespace {

constexpr int kAlignGroup = 16;       // chunks per first-level group of (d2)
constexpr int kStatChunksMax = 128;   // chunks per view of (d1)
constexpr float kGramScale = 16384.f;                      // 2^14
constexpr float kGramUnscale = 1.0f / (16384.f * 16384.f);  // 2^-28

// |Xh| <= 1 for every element: (x - mu)^2 is one term of the column's sum of
// squares, which is (M - ddof) var <= M (var + eps) = M sigma^2.  Scaled by
// 2^14 every value is below 2^15, so the split-fp16 parts cannot overflow.

template <int D>
struct AShape {
  static constexpr int QN = D / 64;                  // 64-feature quadrants per side
  static constexpr int NQ = QN * (QN + 1) / 2;       // quadrants with qi <= qj
  static constexpr int BPC = D == 256 ? 2 : 1;       // blocks per chunk (one view each at d = 256)
  static constexpr int GW = 2 * NQ / BPC;            // Gram waves per block
  static constexpr int SW = 2;                       // column-sum waves
  static constexpr int kThreads = 64 * (GW + SW);
  static constexpr int kChunkCap = D == 64 ? 512 : (D == 128 ? 256 : 128);
  static constexpr int kGramFloats = 2 * NQ * 64 * 64;  // one chunk's partial Grams, both views
};

struct AlignPlan {
  int64_t m, nch1, rpc1, nchg, rpc2, ngroups, grid2;
};

template <int D>
AlignPlan align_plan(int64_t m) {
  AlignPlan p{};
  p.m = m;
  p.nch1 = m > 0 ? (cdiv(m, 512) < kStatChunksMax ? cdiv(m, 512) : kStatChunksMax) : 1;
  p.rpc1 = m > 0 ? cdiv(m, p.nch1) : 1;
  int64_t n = m > 0 ? cdiv(m, 128) : 1;
  n = n < AShape<D>::kChunkCap ? n : AShape<D>::kChunkCap;
  p.rpc2 = cdiv(cdiv(m > 0 ? m : 1, n), 64) * 64;
  p.nchg = m > 0 ? cdiv(m, p.rpc2) : 1;
  p.ngroups = cdiv(p.nchg, kAlignGroup);
  p.grid2 = AShape<D>::BPC == 1 ? p.nchg : 16 * cdiv(p.nchg, 8);
  return p;
}

// finals: C' of both views, then per view mu, 1/sigma, the standardisation
// scale 1/(sigma sqrt(M)), S1 and S2 ([2][D] each)
template <int D>
struct AlignFin {
  float* base;
  __host__ __device__ float* cp(int v) const { return base + (int64_t)v * D * D; }
  __host__ __device__ float* mu(int v) const { return base + 2 * D * D + v * D; }
  __host__ __device__ float* is(int v) const { return base + 2 * D * D + 2 * D + v * D; }
  __host__ __device__ float* sh(int v) const { return base + 2 * D * D + 4 * D + v * D; }
  __host__ __device__ float* s1(int v) const { return base + 2 * D * D + 6 * D + v * D; }
  __host__ __device__ float* s2(int v) const { return base + 2 * D * D + 8 * D + v * D; }
  static constexpr int64_t kFloats = 2 * D * D + 10 * D;
};

template <int D>
struct AlignWs {
  double* stat;   // [nch1][2 views][2][D]
  float* gpart;   // [nchg][2 views][NQ][64 x 64]
  double* spart;  // [nchg][6][D]
  int32_t* cnt;   // [ngroups + 1]
  float* fin;     // AlignFin
  template <class A>
  void layout(A& a, const AlignPlan& p) {
    stat = a.template take<double>(p.nch1 * 4 * D);
    gpart = a.template take<float>(p.nchg * (int64_t)AShape<D>::kGramFloats);
    spart = a.template take<double>(p.nchg * 6 * D);
    cnt = a.template take<int32_t>(p.ngroups + 1);
    fin = a.template take<float>(AlignFin<D>::kFloats);
  }
};

// ---- (d1) column sums of x and x^2 ----------------------------------------------
// grid (chunks, 2 views), 16 waves; a row is D/4 lanes reading 16 bytes
// (columns c..c+3), four rows per lane in flight (their overlap entries first).
// Lanes of one column are combined by xor shuffles inside the wave, then the
// waves in order.  Block (0, 0) zeroes the counters of (d2).
constexpr int kStatThreads = 1024;
template <int D, class T>
__global__ void __launch_bounds__(kStatThreads) k_align_stats(int64_t m, int64_t rpc, const T* __restrict__ H,
                                                              const int32_t* __restrict__ ov,
                                                              const T* __restrict__ Href, double* __restrict__ stat,
                                                              int32_t* __restrict__ cnt, int ncnt) {
  constexpr int TPR = D / 4, RPI = kStatThreads / TPR, U = 4, NW = kStatThreads / 64;
  __shared__ double red[NW][8][TPR < 64 ? TPR : 64];
  const int t = threadIdx.x;
  const int view = blockIdx.y;
  if (blockIdx.x == 0 && view == 0 && t < ncnt) cnt[t] = 0;
  const int c = (t % TPR) * 4, ph = t / TPR;
  const int64_t b0 = (int64_t)blockIdx.x * rpc;
  const int64_t b1 = (b0 + rpc < m) ? b0 + rpc : m;
  const T* base = view ? Href : H;
  double s[4] = {0.0, 0.0, 0.0, 0.0}, q[4] = {0.0, 0.0, 0.0, 0.0};
  auto add = [&](const f32x4& v) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const double x = (double)v[k];
      s[k] += x;
      q[k] += x * x;
    }
  };
  int64_t b = b0 + ph;
  for (; b + (U - 1) * RPI < b1; b += U * RPI) {
    int64_t r[U];
#pragma unroll
    for (int u = 0; u < U; ++u) r[u] = view ? b + u * RPI : (int64_t)ov[b + u * RPI];
    f32x4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = Elt<T>::load4(base + r[u] * D + c);
#pragma unroll
    for (int u = 0; u < U; ++u) add(v[u]);
  }
  for (; b < b1; b += RPI) add(Elt<T>::load4(base + (view ? b : (int64_t)ov[b]) * D + c));
  // lanes of the same columns inside the wave (rows ph differ in the lane bits above TPR)
#pragma unroll
  for (int o = TPR; o < 64; o <<= 1)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      s[k] += __shfl_xor(s[k], o, 64);
      q[k] += __shfl_xor(q[k], o, 64);
    }
  const int wv = t >> 6, l = t & 63;
  constexpr int LW = TPR < 64 ? TPR : 64;  // distinct column groups per wave
  if (l < LW)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      red[wv][k][l] = s[k];
      red[wv][4 + k][l] = q[k];
    }
  __syncthreads();
  // column group cg is held by lane cg % 64 of the waves whose lanes cover it
  if (t < TPR) {
    double* out = stat + ((int64_t)blockIdx.x * 2 + view) * 2 * D;
    constexpr int WPR = TPR / LW;  // waves per row (D = 256: a row spans one wave)
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      double ts = 0.0, tq = 0.0;
      for (int ww = t / LW; ww < NW; ww += WPR) {
        ts += red[ww][k][t % LW];
        tq += red[ww][4 + k][t % LW];
      }
      out[c + k] = ts;
      out[D + c + k] = tq;
    }
  }
}

// Fixed-order sum over the threads of a block (NT <= 1024).
template <int NT>
__device__ double block_sum_d(double v, double* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o && (int)threadIdx.x + o < NT) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

// quadrant index q (qi <= qj, row-major over the upper triangle) -> (qi, qj)
template <int QN>
__device__ __forceinline__ void quad_of(int q, int& qi, int& qj) {
  qi = 0;
  qj = 0;
#pragma unroll
  for (int i = 0; i < QN; ++i) {
    if (q >= 0 && q < QN - i) {
      qi = i;
      qj = i + q;
    }
    q -= QN - i;
  }
}

// ---- (d2) Grams, column sums, last-block reductions, loss and finals -----------
// The rows of a step (64 rows of both views, 32 at d = 256 in float32) are
// staged in LDS: every thread
// loads its share of step s + 1 from HBM while step s is multiplied, and all
// waves read their operands from LDS (each row leaves HBM once).  LDS: two
// step buffers [2 views][32][D] of the storage type, then the stat arrays;
// the end-of-chunk arrays reuse the step buffers.
template <int D, class T>
struct GramLds {
  // steps of 64 rows up to 512-byte rows (128 KB of LDS at most), except at
  // d = 256, whose ten Gram waves per view spill with two 32-row blocks per
  // step (32-row steps: 1.6 against 3.3 ms per bf16 step)
  static constexpr int kStepRows = (D * sizeof(T) <= 512 && D < 256) ? 64 : 32;
  static constexpr int kStep = 2 * kStepRows * D;               // elements of one step buffer
  static constexpr size_t kRows = 2 * (size_t)kStep * sizeof(T);  // both step buffers, bytes
  static constexpr size_t kTail = sizeof(double) * (128 * 25 + 1024 + 6 * D);
  static constexpr size_t kBytes = (kRows > kTail ? kRows : kTail);
};

template <int D, class T>
__global__ void __launch_bounds__(AShape<D>::kThreads) k_align_gram(
    int64_t m, int64_t nch1, int64_t rpc, int64_t nchg, int32_t ddof, float eps, float lambda_n,
    const T* __restrict__ H, const int32_t* __restrict__ ov, const T* __restrict__ Href, const float* __restrict__ w,
    const double* __restrict__ stat, float* __restrict__ gpart, double* __restrict__ spart, int32_t* __restrict__ cnt,
    float* __restrict__ finp, float* __restrict__ loss3) {
  typedef AShape<D> S;
  typedef GramLds<D, T> LY;
  constexpr int NT = S::kThreads, QN = S::QN, NQ = S::NQ, GW = S::GW;
  constexpr int TPR = D / 4, RPS = 128 / TPR;  // column-sum waves: lanes per row, rows per sweep
  constexpr int CPR = D * (int)sizeof(T) / 16;  // 16-byte chunks per row
  constexpr int SR = LY::kStepRows;
  constexpr int ITEMS = 2 * SR * CPR;           // chunks per step, both views
  constexpr int PER = (ITEMS + NT - 1) / NT;    // chunks per thread and step
  extern __shared__ __align__(16) unsigned char lds[];
  T* rows = reinterpret_cast<T*>(lds);  // [2 buffers][2 views][SR][D]
  double* sred = reinterpret_cast<double*>(lds);           // [128][25]   (after the walk)
  double* red = sred + 128 * 25;                           // [1024]
  double* sums = red + 1024;                               // [6][D]
  __shared__ float st_mu[2][D], st_sh[2][D], st_is[2][D];
  __shared__ int s_last;
  const int tid = threadIdx.x;
  int64_t chunk;
  int y;
  if (S::BPC == 1) {
    chunk = blockIdx.x;
    y = 0;
  } else {
    // the two blocks of a chunk are 8 apart: same XCD, so the second read of a row hits its L2
    y = (blockIdx.x >> 3) & 1;
    chunk = (int64_t)(((blockIdx.x >> 4) << 3) | (blockIdx.x & 7));
  }
  if (chunk >= nchg) return;  // padding block: no part in the counts
  const AlignFin<D> fin{finp};
  // mean, 1/sigma and scale of both views from the (d1) partials, fixed order
  for (int e = tid; e < 2 * D; e += NT) {
    const int v = e / D, c = e % D;
    double s = 0.0, q = 0.0;
#pragma unroll 16
    for (int64_t k = 0; k < nch1; ++k) {
      s += stat[(k * 2 + v) * 2 * D + c];
      q += stat[(k * 2 + v) * 2 * D + D + c];
    }
    const double mean = s / (double)m;
    double var = (q - s * mean) / (double)(m - ddof);
    var = var > 0.0 ? var : 0.0;
    const float sig = sqrtf((float)var + eps);
    st_mu[v][c] = (float)mean;
    st_is[v][c] = 1.0f / sig;
    st_sh[v][c] = 1.0f / (sig * sqrtf((float)m));
  }
  const int64_t r_beg = chunk * rpc;
  const int64_t r_end = (r_beg + rpc < m) ? r_beg + rpc : m;
  // loader: chunk j of a step is (view, row, 16-byte piece); its HBM row id
  // comes from the overlap list for view 0
  auto row_id = [&](int64_t r0, int j) -> int64_t {
    const int v = j / (SR * CPR), r = (j / CPR) % SR;
    const int64_t rr = r0 + r;
    if (rr >= r_end) return -1;
    return v ? rr : (int64_t)ov[rr];
  };
  auto fetch = [&](int64_t r0, const int64_t (&id)[PER], uint4 (&x)[PER]) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int j = tid + k * NT;
      x[k] = uint4{0u, 0u, 0u, 0u};
      if (j < ITEMS && id[k] >= 0) {
        const T* base = (j / (SR * CPR)) ? Href : H;
        x[k] = *reinterpret_cast<const uint4*>(base + id[k] * D + (j % CPR) * (16 / (int)sizeof(T)));
      }
    }
  };
  auto park = [&](int buf, const uint4 (&x)[PER]) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int j = tid + k * NT;
      if (j < ITEMS) reinterpret_cast<uint4*>(rows + (int64_t)buf * LY::kStep)[j] = x[k];
    }
  };
  auto ids = [&](int64_t r0, int64_t (&id)[PER]) {
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int j = tid + k * NT;
      id[k] = (j < ITEMS && r0 < r_end) ? row_id(r0, j) : -1;
    }
  };
  const int wv = tid >> 6, l = lane64();
  const int g = l >> 4, c = l & 15;
  // Gram wave
  const int tile = y * GW + wv;
  const int gview = tile / NQ, gq = tile % NQ;
  int qi, qj;
  quad_of<QN>(gq, qi, qj);
  const bool gram = wv < GW, diag = qi == qj;
  const int ca = 64 * qi + 4 * c, cb = 64 * qj + 4 * c;
  // column-sum waves (block y = 0 only)
  const bool csum = !gram && y == 0;
  const int sl = tid - 64 * GW;  // 0..127 on the column-sum waves
  const int scol = (sl % TPR) * 4, soff = sl / TPR;
  int64_t idn[PER];
  uint4 xr[PER];
  ids(r_beg, idn);
  fetch(r_beg, idn, xr);
  ids(r_beg + SR, idn);
  park(0, xr);
  __syncthreads();  // stats and step 0 in LDS
  // every wave walks the chunk's steps with the same loads, parks and
  // barriers; body(sv, r0) works on step r0 staged at sv ([2 views][SR][D])
  auto walk = [&](auto&& body) {
    int buf = 0;
    for (int64_t r0 = r_beg; r0 < r_end; r0 += SR, buf ^= 1) {
      const bool more = r0 + SR < r_end;
      if (more) fetch(r0 + SR, idn, xr);  // step s + 1 in flight while step s is used
      if (more) ids(r0 + 2 * SR, idn);
      body((const T*)(rows + (int64_t)buf * LY::kStep), r0);
      if (more) park(buf ^ 1, xr);
      __syncthreads();
    }
  };
  if (gram) {
    f32x4 acc[4][4];
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int bj = 0; bj < 4; ++bj) acc[bi][bj] = f32x4{0.f, 0.f, 0.f, 0.f};
    walk([&](const T* sv, int64_t r0) {
      const T* src = sv + gview * SR * D;
      // operand rows: 8 rows x 4 columns per lane, standardised and scaled by 2^14
      auto rows8 = [&](int kb, int col, f32x4 (&x)[8]) {
        f32x4 mu4, sc4;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          mu4[k] = st_mu[gview][col + k];
          sc4[k] = st_sh[gview][col + k] * kGramScale;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int r = 32 * kb + 8 * g + e;
          const f32x4 v = Elt<T>::load4(src + r * D + col);
          x[e] = (r0 + r < r_end) ? (v - mu4) * sc4 : f32x4{0.f, 0.f, 0.f, 0.f};
        }
      };
      for (int kb = 0; kb < SR / 32; ++kb) {
        uint4 hb[4], lb[4];
        {
          f32x4 xb[8];
          rows8(kb, cb, xb);
#pragma unroll
          for (int bj = 0; bj < 4; ++bj) {
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = xb[e][bj];
            split8(v, hb[bj], lb[bj]);
          }
        }
        if (diag) {
#pragma unroll
          for (int bi = 0; bi < 4; ++bi)
#pragma unroll
            for (int bj = 0; bj < 4; ++bj) {
              acc[bi][bj] = mfma_f16(hb[bi], hb[bj], acc[bi][bj]);
              acc[bi][bj] = mfma_f16(hb[bi], lb[bj], acc[bi][bj]);
              acc[bi][bj] = mfma_f16(lb[bi], hb[bj], acc[bi][bj]);
            }
        } else {
          f32x4 xa[8];
          rows8(kb, ca, xa);
#pragma unroll
          for (int bi = 0; bi < 4; ++bi) {
            uint4 ha, la;
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = xa[e][bi];
            split8(v, ha, la);
#pragma unroll
            for (int bj = 0; bj < 4; ++bj) {
              acc[bi][bj] = mfma_f16(ha, hb[bj], acc[bi][bj]);
              acc[bi][bj] = mfma_f16(ha, lb[bj], acc[bi][bj]);
              acc[bi][bj] = mfma_f16(la, hb[bj], acc[bi][bj]);
            }
          }
        }
      }
    });
    // partial Grams of this chunk: lane (c, g), register v of block (bi, bj)
    // is element [4 (4 g + v) + bi][4 c + bj] of the quadrant
    float* out = gpart + (chunk * (int64_t)S::kGramFloats) + (int64_t)(gview * NQ + gq) * 4096;
#pragma unroll
    for (int bi = 0; bi < 4; ++bi)
#pragma unroll
      for (int v = 0; v < 4; ++v) {
        f32x4 row4;
#pragma unroll
        for (int bj = 0; bj < 4; ++bj) row4[bj] = acc[bi][bj][v] * kGramUnscale;
        *reinterpret_cast<f32x4*>(out + (4 * (4 * g + v) + bi) * 64 + 4 * c) = row4;
      }
  } else {
    double cs[6][4];
#pragma unroll
    for (int k = 0; k < 6; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) cs[k][q] = 0.0;
    walk([&](const T* sv, int64_t r0) {
      if (!csum) return;
      f32x4 smx, ssx, smy, ssy;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        smx[k] = st_mu[0][scol + k];
        ssx[k] = st_sh[0][scol + k];
        smy[k] = st_mu[1][scol + k];
        ssy[k] = st_sh[1][scol + k];
      }
#pragma unroll
      for (int k = 0; k < SR / RPS; ++k) {
        const int r = soff + k * RPS;
        const int64_t rg = r0 + r;
        if (rg < r_end) {
          const f32x4 xh = (Elt<T>::load4(sv + r * D + scol) - smx) * ssx;
          const f32x4 yh = (Elt<T>::load4(sv + SR * D + r * D + scol) - smy) * ssy;
          const double om = w ? (double)w[rg] : 1.0;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const double xv = (double)xh[q], yv = (double)yh[q], dl = xv - yv, od = om * dl;
            cs[0][q] += xv;
            cs[1][q] += yv;
            cs[2][q] += od;
            cs[3][q] += od * xv;
            cs[4][q] -= od * yv;
            cs[5][q] += od * dl;
          }
        }
      }
    });
    if (csum) {
#pragma unroll
      for (int k = 0; k < 6; ++k)
#pragma unroll
        for (int q = 0; q < 4; ++q) sred[sl * 25 + 4 * k + q] = cs[k][q];
    }
  }
  __syncthreads();
  if (y == 0 && tid < TPR) {
    double* out = spart + chunk * 6 * D;
#pragma unroll
    for (int k = 0; k < 6; ++k)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        double s = 0.0;
        for (int p = 0; p < RPS; ++p) s += sred[(p * TPR + tid) * 25 + 4 * k + q];
        out[k * D + 4 * tid + q] = s;
      }
  }
  // ---- first level: the last block of the group sums its chunks in order ----
  __threadfence();
  __syncthreads();
  const int64_t grp = chunk / kAlignGroup;
  const int64_t c0 = grp * kAlignGroup, c1 = (c0 + kAlignGroup < nchg) ? c0 + kAlignGroup : nchg;
  if (tid == 0) s_last = atomicAdd(&cnt[grp], 1) == S::BPC * (int)(c1 - c0) - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  // all chunk loads of an element are issued before the in-order sum
  for (int e4 = tid; e4 < S::kGramFloats / 4; e4 += NT) {
    f32x4 v[kAlignGroup];
#pragma unroll
    for (int k = 0; k < kAlignGroup; ++k)
      v[k] = c0 + k < c1 ? *reinterpret_cast<const f32x4*>(gpart + (c0 + k) * S::kGramFloats + 4 * e4)
                         : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 sum = v[0];
#pragma unroll
    for (int k = 1; k < kAlignGroup; ++k) sum += v[k];
    *reinterpret_cast<f32x4*>(gpart + c0 * S::kGramFloats + 4 * e4) = sum;
  }
  for (int e = tid; e < 6 * D; e += NT) {
    double v[kAlignGroup];
#pragma unroll
    for (int k = 0; k < kAlignGroup; ++k) v[k] = c0 + k < c1 ? spart[(c0 + k) * 6 * D + e] : 0.0;
    double sum = v[0];
#pragma unroll
    for (int k = 1; k < kAlignGroup; ++k) sum += v[k];
    spart[c0 * 6 * D + e] = sum;
  }
  __threadfence();
  __syncthreads();
  const int64_t ngroups = (nchg + kAlignGroup - 1) / kAlignGroup;
  if (tid == 0) s_last = atomicAdd(&cnt[ngroups], 1) == (int)ngroups - 1;
  __syncthreads();
  if (!s_last) return;
  __threadfence();
  // ---- second level (one block): groups in order, then the finals ----------
  constexpr int kMaxGroups = (S::kChunkCap + kAlignGroup - 1) / kAlignGroup;
  double ldec = 0.0;
  for (int e4 = tid; e4 < S::kGramFloats / 4; e4 += NT) {
    f32x4 v[kMaxGroups];
#pragma unroll
    for (int k = 0; k < kMaxGroups; ++k)
      v[k] = k < ngroups ? *reinterpret_cast<const f32x4*>(gpart + (int64_t)k * kAlignGroup * S::kGramFloats + 4 * e4)
                         : f32x4{0.f, 0.f, 0.f, 0.f};
    f32x4 sum = v[0];
#pragma unroll
    for (int k = 1; k < kMaxGroups; ++k) sum += v[k];
    const int e = 4 * e4;
    const int vw = e / (NQ * 4096), q = (e / 4096) % NQ, i = (e % 4096) / 64, j0 = e % 64;
    int a, b;
    quad_of<QN>(q, a, b);
    const int gi = 64 * a + i;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int gj = 64 * b + j0 + k;
      const float cp = sum[k] - (gi == gj ? 1.f : 0.f);
      fin.cp(vw)[gi * D + gj] = cp;
      if (a != b) fin.cp(vw)[gj * D + gi] = cp;
      ldec += (a != b ? 2.0 : 1.0) * (double)cp * (double)cp;
    }
  }
  for (int e = tid; e < 6 * D; e += NT) {
    double v[kMaxGroups];
#pragma unroll
    for (int k = 0; k < kMaxGroups; ++k) v[k] = k < ngroups ? spart[(int64_t)k * kAlignGroup * 6 * D + e] : 0.0;
    double sum = v[0];
#pragma unroll
    for (int k = 1; k < kMaxGroups; ++k) sum += v[k];
    sums[e] = sum;
  }
  for (int e = tid; e < 2 * D; e += NT) {
    const int v = e / D, cc = e % D;
    fin.mu(v)[cc] = st_mu[v][cc];
    fin.is(v)[cc] = st_is[v][cc];
    fin.sh(v)[cc] = st_sh[v][cc];
  }
  __threadfence();
  __syncthreads();
  const double L_dec = block_sum_d<NT>(ldec, red);
  double linv = 0.0;
  for (int cc = tid; cc < D; cc += NT) linv += sums[5 * D + cc];
  const double L_inv = block_sum_d<NT>(linv, red);
  const double inv_sqrt_m = 1.0 / sqrt((double)m);
  for (int e = tid; e < 2 * D; e += NT) {
    const int v = e / D, cc = e % D;
    const float* P = fin.cp(v);
    // column cc of C' (read by consecutive threads: coalesced), 16 loads in
    // flight; C' is symmetric, so (C' C')_cc is the column's sum of squares
    double t1 = 0.0, t2 = 0.0;
    for (int k0 = 0; k0 < D; k0 += 16) {
      float pk[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) pk[k] = P[(k0 + k) * D + cc];
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        t1 += sums[v * D + k0 + k] * (double)pk[k];  // v C' (view X) or w C' (view Y)
        t2 += (double)pk[k] * (double)pk[k];
      }
    }
    const double u = v == 0 ? sums[2 * D + cc] : -sums[2 * D + cc];
    const double pq = v == 0 ? sums[3 * D + cc] : sums[4 * D + cc];
    fin.s1(v)[cc] = (float)((2.0 * u + 4.0 * (double)lambda_n * t1) * inv_sqrt_m);
    fin.s2(v)[cc] = (float)(2.0 * pq + 4.0 * (double)lambda_n * (t2 + (double)P[cc * D + cc]));
  }
  if (tid == 0) {
    loss3[0] = (float)L_inv;
    loss3[1] = (float)L_dec;
    loss3[2] = (float)(L_inv + (double)lambda_n * L_dec);
  }
}

// ---- (d3) the gradient pass ---------------------------------------------------
// Row GEMM acc = Xh C' on the split-fp16 MFMA (C' staged once per block in
// LDS in fragment order, as in k_gemm_rows: the W fragments are the A
// operand, the rows the B operand, so lane (c, g) of wave w ends with row
// 16 w + c of a 128-row tile, columns col0 + 16 nb + 4 g .. + 3), with the
// standardisation backward in the epilogue:
//   out = base + o kx (Xh - Yh) - kc - ke (x - mu) + ka acc,
//   kx = scale (1/sigma) 2 / sqrt(M),  kc = scale (1/sigma) S1 / M,
//   ke = scale (1/sigma)^2 S2 / (M - ddof),  ka = scale (1/sigma) 4 lambda / sqrt(M)
// (the file comment's dX times scale).  The lane's x columns of every output
// block are among the A-operand columns it holds, so only the other view's
// row and the base row are read in the epilogue.  blockIdx.y picks the
// 128-column slice at d = 256.
template <int D, class T>
__global__ void __launch_bounds__(kGemmThreads) k_align_grad(int64_t m, const T* __restrict__ self, RowMap smap,
                                                             const T* __restrict__ other, RowMap omap,
                                                             const float* __restrict__ finp, int view,
                                                             const float* __restrict__ w, const T* base, T* out,
                                                             float scale, float lambda_n, int32_t ddof) {
  constexpr int DN = F32Slice<D>::DN;
  constexpr int KB = D / 16, KB2 = D / 32, NB = DN / 16;
  constexpr int kWaves = kGemmThreads / 64;
  constexpr int kRowsPerTile = 16 * kWaves;
  constexpr int kFrag = KB2 * NB * 64;
  extern __shared__ uint4 wsl[];  // [kFrag] high parts, then [kFrag] remainders
  __shared__ float wmax[kWaves + 1];
  __shared__ float k_mu[D], k_sh[D], k_muo[D], k_sho[D], k_x[D], k_c[D], k_e[D], k_a[D];
  const AlignFin<D> fin{const_cast<float*>(finp)};
  const float* W = fin.cp(view);
  const int tid = threadIdx.x;
  const int col0 = DN * blockIdx.y;
  {
    const float rs = 1.0f / sqrtf((float)m);
    for (int c = tid; c < D; c += kGemmThreads) {
      const float isg = fin.is(view)[c];
      k_mu[c] = fin.mu(view)[c];
      k_sh[c] = fin.sh(view)[c];
      k_muo[c] = fin.mu(1 - view)[c];
      k_sho[c] = fin.sh(1 - view)[c];
      k_x[c] = scale * isg * 2.0f * rs;
      k_c[c] = scale * isg * fin.s1(view)[c] / (float)m;
      k_e[c] = scale * isg * isg * fin.s2(view)[c] / (float)(m - ddof);
      k_a[c] = scale * isg * 4.0f * lambda_n * rs;
    }
    float mx = 0.f;
    for (int e = tid; e < D * D / 4; e += kGemmThreads) {
      const f32x4 v = *reinterpret_cast<const f32x4*>(W + 4 * e);
      mx = fmaxf(mx, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
    if ((tid & 63) == 0) wmax[tid >> 6] = mx;
    __syncthreads();
    mx = wmax[0];
#pragma unroll
    for (int q = 1; q < kWaves; ++q) mx = fmaxf(mx, wmax[q]);
    const uint32_t ew = split_exp(mx);
    const float sw = split_scale(ew);
    for (int e = tid; e < kFrag; e += kGemmThreads) {
      const int l = e & 63;
      const int nb = (e >> 6) % NB;
      const int kb2 = (e >> 6) / NB;
      const int j = col0 + 16 * nb + (l & 15);
      float v[8];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int k0 = 16 * (2 * kb2 + h) + 4 * (l >> 4);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[4 * h + q] = W[(int64_t)(k0 + q) * D + j] * sw;
      }
      split8(v, wsl[e], wsl[kFrag + e]);
    }
    if (tid == 0) wmax[kWaves] = split_unscale(ew);
    __syncthreads();
  }
  const float uw = wmax[kWaves];
  const int wv = tid >> 6;
  const int l = lane64();
  const int g = l >> 4, c = l & 15;
  const int64_t ntiles = (m + kRowsPerTile - 1) / kRowsPerTile;
  for (int64_t t = blockIdx.x; t < ntiles; t += gridDim.x) {
    const int64_t i = t * kRowsPerTile + 16 * wv + c;
    const bool live = i < m;
    const int64_t rs_ = live ? smap(i) : 0;
    typename Elt<T>::raw4_t xr[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) xr[kb] = Elt<T>::raw4(self + rs_ * D + 16 * kb + 4 * g);
    uint4 xh[KB2], xlo[KB2];
    float ux;
    {
      auto xhat = [&](int kb) -> f32x4 {
        const int col = 16 * kb + 4 * g;
        const f32x4 x = Elt<T>::cook4(xr[kb]);
        f32x4 r;
#pragma unroll
        for (int q = 0; q < 4; ++q) r[q] = live ? (x[q] - k_mu[col + q]) * k_sh[col + q] : 0.f;
        return r;
      };
      float mx = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const f32x4 a = xhat(kb);
        mx = fmaxf(mx, fmaxf(fmaxf(fabsf(a[0]), fabsf(a[1])), fmaxf(fabsf(a[2]), fabsf(a[3]))));
      }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const uint32_t ex = split_exp(mx);
      const float sx = split_scale(ex);
      ux = split_unscale(ex);
#pragma unroll
      for (int kb2 = 0; kb2 < KB2; ++kb2) {
        const f32x4 a0 = xhat(2 * kb2), a1 = xhat(2 * kb2 + 1);
        float v[8];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          v[q] = a0[q] * sx;
          v[4 + q] = a1[q] * sx;
        }
        split8(v, xh[kb2], xlo[kb2]);
      }
    }
    f32x4 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) acc[nb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb2 = 0; kb2 < KB2; ++kb2) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int e = (kb2 * NB + nb) * 64 + l;
        const uint4 bh = wsl[e], bl = wsl[kFrag + e];
        acc[nb] = mfma_f16(bh, xh[kb2], acc[nb]);
        acc[nb] = mfma_f16(bh, xlo[kb2], acc[nb]);
        acc[nb] = mfma_f16(bl, xh[kb2], acc[nb]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    if (live) {
      const int64_t ro = omap(i);
      const float om = w ? w[i] : 1.f;
      f32x4 yv[NB], bv[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = col0 + 16 * nb + 4 * g;
        yv[nb] = Elt<T>::load4(other + ro * D + col);
        bv[nb] = base ? Elt<T>::load4(base + rs_ * D + col) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int col = col0 + 16 * nb + 4 * g;
        // the lane's A chunk of these columns (both candidates named at
        // compile time: a run-time index would put the row in scratch)
        f32x4 x;
        if constexpr (D == DN) {
          x = Elt<T>::cook4(xr[nb]);
        } else {
          x = blockIdx.y == 0 ? Elt<T>::cook4(xr[nb]) : Elt<T>::cook4(xr[NB + nb]);
        }
        const f32x4 a = split_unscale4(acc[nb], ux, uw);
        f32x4 r;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int cc = col + q;
          const float dxm = x[q] - k_mu[cc];
          const float xhv = dxm * k_sh[cc];
          const float yhv = (yv[nb][q] - k_muo[cc]) * k_sho[cc];
          r[q] = bv[nb][q] + om * k_x[cc] * (xhv - yhv) - k_c[cc] - k_e[cc] * dxm + k_a[cc] * a[q];
        }
        if constexpr (sizeof(T) == 4) {
          *reinterpret_cast<f32x4*>(out + rs_ * D + col) = r;
        } else {
          *reinterpret_cast<uint2*>(out + rs_ * D + col) = uint2{pack2bf(r[0], r[1]), pack2bf(r[2], r[3])};
        }
      }
    }
  }
}

template <int D, class T>
int launch_align_grad(int64_t m, const T* self, RowMap smap, const T* other, RowMap omap, const float* fin,
                      int view, const float* w, const T* base, T* out, float scale, float lambda_n, int32_t ddof,
                      hipStream_t s) {
  constexpr int DN = F32Slice<D>::DN;
  const int64_t tiles = cdiv(m, 16 * (kGemmThreads / 64));
  const int64_t cap = (int64_t)num_cus() * (D > 128 ? 1 : 2);
  const int64_t grid = tiles < cap ? tiles : cap;
  const size_t lds = sizeof(float) * D * DN;
  auto kern = k_align_grad<D, T>;
  if (lds > 65536) {
    static bool attr_set = false;
    if (!attr_set) {
      HG_HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                     (int)lds));
      attr_set = true;
    }
  }
  HG_LAUNCH("align_grad", kern, dim3((unsigned)grid, D / DN), dim3(kGemmThreads), lds, s, m, self, smap, other,
            omap, fin, view, w, base, out, scale, lambda_n, ddof);
  return HG_OK;
}

template <int D, class T>
int align_impl(int64_t m, const T* H, const int32_t* overlap, const T* Href, const float* w, float lambda_n,
               float scale, float eps, int32_t ddof, float* loss3, T* dH, const T* dHbase, T* dHref, void* ws,
               size_t ws_bytes, hipStream_t s) {
  const AlignPlan p = align_plan<D>(m);
  Arena a(ws, ws_bytes);
  AlignWs<D> q;
  q.layout(a, p);
  if (!a.ok()) return fail(HG_ERR_CAPACITY, "alignment workspace needs %zu bytes, got %zu", a.used, ws_bytes);
  // (d1)
  HG_LAUNCH("align_stats", (k_align_stats<D, T>), dim3((unsigned)p.nch1, 2), dim3(kStatThreads), 0, s, m, p.rpc1, H,
            overlap, Href, q.stat, q.cnt, (int)(p.ngroups + 1));
  // (d2)
  {
    auto kern = k_align_gram<D, T>;
    const size_t lds = GramLds<D, T>::kBytes;
    if (lds > 65536) {
      static bool attr_set = false;
      if (!attr_set) {
        HG_HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
        attr_set = true;
      }
    }
    HG_LAUNCH("align_gram", kern, dim3((unsigned)p.grid2), dim3(AShape<D>::kThreads), lds, s, m, p.nch1, p.rpc2,
              p.nchg, ddof, eps, lambda_n, H, overlap, Href, w, (const double*)q.stat, q.gpart, q.spart, q.cnt,
              q.fin, loss3);
  }
  // (d3)
  HG_TRY((launch_align_grad<D, T>(m, H, rows_list(overlap), Href, rows_contig(0), q.fin, 0, w,
                                  dHbase ? dHbase : (const T*)dH, dH, scale, lambda_n, ddof, s)));
  if (dHref)
    HG_TRY((launch_align_grad<D, T>(m, Href, rows_contig(0), H, rows_list(overlap), q.fin, 1, w, nullptr, dHref,
                                    scale, lambda_n, ddof, s)));
  return HG_OK;
}

template <int D>
size_t align_ws_bytes(int64_t m) {
  Sizer z;
  AlignWs<D> w;
  w.layout(z, align_plan<D>(m));
  return z.used + 256;
}

}  // namespace

}  // namespace hg

using namespace hg;

extern "C" size_t hg_align_workspace_size(int64_t M, int32_t d) {
  if (M < 0) return 0;
  if (d == 64) return align_ws_bytes<64>(M);
  if (d == 128) return align_ws_bytes<128>(M);
  if (d == 256) return align_ws_bytes<256>(M);
  return 0;
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

// ---- no-allocation variant -------------------------------------------------------
// The same passes with the workspace in a file-scope device array.  In host
// code `scratch` names a host-side stand-in, not device memory: its device
// address is taken with hipGetSymbolAddress once per device (each device
// holds its own copy) and only that address is passed to the kernels.  The
// counters of the Gram pass are zeroed by the statistics pass of the same
// call, so nothing has to be cleared between calls.
namespace hg {
namespace {
constexpr size_t kAlignScratchBytes = size_t(48) << 20;
constexpr int kMaxDevices = 64;
__device__ __align__(256) unsigned char scratch[kAlignScratchBytes];
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

int scratch_address(void** out) {
  int dev = 0;
  HG_HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(HG_ERR_UNSUPPORTED, "device %d beyond %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(HG_ERR_HIP, "hipGetSymbolAddress(scratch) on device %d failed: %s", dev, hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return HG_OK;
}
}  // namespace
}  // namespace hg

extern "C" size_t hg_align_noalloc_scratch_size(void) { return kAlignScratchBytes; }

extern "C" int hg_align_loss_fwd_bwd_noalloc(int64_t M, int32_t d, int32_t dtype, int64_t n_rows, const void* H,
                                             const int32_t* overlap, const void* H_ref, const float* w,
                                             float lambda_n, float scale, float eps, int32_t ddof, float* loss3,
                                             void* dH, const void* dH_base, void* dH_ref, void* stream) {
  if (d != 64 && d != 128 && d != 256)
    return fail(HG_ERR_UNSUPPORTED, "alignment supports d in {64, 128, 256}, got %d", d);
  const size_t need = hg_align_workspace_size(M, d);
  if (need > kAlignScratchBytes)
    return fail(HG_ERR_CAPACITY, "alignment needs %zu bytes of scratch, the static scratch holds %zu", need,
                kAlignScratchBytes);
  void* ws = nullptr;
  HG_TRY(scratch_address(&ws));
  return hg_align_loss_fwd_bwd(M, d, dtype, n_rows, H, overlap, H_ref, w, lambda_n, scale, eps, ddof, loss3, dH,
                               dH_base, dH_ref, ws, kAlignScratchBytes, stream);
}
