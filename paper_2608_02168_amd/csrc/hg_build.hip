// hg_build_csr: risk-aware overlapping-subgraph construction on the GPU.
//
// Steps (Methodology, "Risk-Aware Subgraph Construction"; Algorithm 1,
// construction loop):
//   1. one pass over the edges: range checks, out-degrees, and for every node
//      outside V_k the smallest index of an edge joining it to V_k (either
//      direction) -- a node is a candidate of C_k iff that index exists;
//   2. node keys: out-degree, or the h-index of the out-neighbour multiset;
//   3. C'_k = candidates with key <= theta, compacted in gid order;
//   4. TopM: an exact radix select of the min(M, |C'_k|) smallest 128-bit
//      composites (key, splitmix64(seed ^ gid), gid) -- unique by gid, so the
//      selected set is unique;
//   5. local ids in (node type, gid) order by a stable bucket partition;
//   6. induced-subgraph edge compaction in original edge order (local ids
//      from a 32-byte-per-64-nodes rank table, per-tile counts, ballots);
//   7. stable LSD radix sorts by (dst, r) and (src, r) give the CSR and CSC;
//      row pointers from run-length counts; csc_scale = 1/deg_r(dst);
//   8. the execution plan: per-relation active-source lists and the chunked
//      work list of the atomic-free transposed SpMM.
#include <vector>

#include "hg_internal.h"

namespace hg {

namespace {

constexpr int kBT = 256;  // threads per block for the elementwise passes
constexpr int kChunk = 1024;  // max CSC entries handled by one backward work item

inline unsigned grid_for(int64_t n, int64_t cap = 16384) {
  int64_t b = cdiv(n > 0 ? n : 1, kBT);
  return (unsigned)(b < cap ? b : cap);
}

__device__ __forceinline__ int64_t cdiv_dev(int64_t a, int64_t b) { return (a + b - 1) / b; }

#define GRID_STRIDE(i, n)                                                        \
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < (n);     \
       i += (int64_t)gridDim.x * blockDim.x)

// Device counters written by the build.
enum : int { C_ERR = 0, C_NSUB, C_ESUB, C_MSEL, C_ITEMS, C_HEAVY, C_PARTS, C_CPRIME, C_BASE, C_FHEAVY, C_FPARTS,
             C_ASLOTS, C_COUNT };

// The row-indexed layout of the relation transforms is kept when nq rows cost
// at most kRowLayoutMaxSpread times the a active ones.
__host__ __device__ inline bool row_layout(int64_t nq, int64_t a) { return nq <= kRowLayoutMaxSpread * a; }

// A subgraph that holds three quarters of the graph's nodes or more (|V_k|
// plus the budget) is built the "dense" way: the base edge of every candidate
// is found in the first edge pass, whose LDS tables absorb the hub nodes'
// many edges.  Otherwise the first pass only marks candidates and the base
// edges of the few selected nodes are found with the induced edges.  Both
// give the same outputs.
__host__ __device__ inline bool dense_build(int64_t n_base, int64_t budget, int64_t n_nodes) {
  const int64_t b = budget < n_nodes ? budget : n_nodes;
  return 4 * (n_base + b) >= 3 * n_nodes;
}

struct SelectState {
  uint32_t k_rem;   // how many more to take from the current prefix bucket
  uint32_t mode;    // 0 = searching, 1 = done (take composite prefix <= digits), 2 = take none
  uint32_t npass;   // number of fixed leading digits
  uint32_t pad;
  uint32_t digits[16];
  int32_t hist[256];
};

__device__ __forceinline__ uint64_t splitmix64_first(uint64_t state) {
  // SplitMix64 (Steele, Lea, Flood 2014): advance by the golden gamma, then
  // the variant-13 finaliser.
  uint64_t z = state + 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Byte p (0 = most significant) of the 128-bit composite (key, hash, gid).
__device__ __forceinline__ uint32_t composite_digit(uint32_t key, uint64_t h, uint32_t gid, int p) {
  uint32_t w;
  switch (p >> 2) {
    case 0: w = key; break;
    case 1: w = (uint32_t)(h >> 32); break;
    case 2: w = (uint32_t)h; break;
    default: w = gid; break;
  }
  return (w >> (8 * (3 - (p & 3)))) & 0xFFu;
}

// bits[v / 32] bit v % 32 = pred(v); one wave covers 64 nodes (two words).
// Also |V_k|, as one partial count per block (summed by k_sum_counts).
__global__ void __launch_bounds__(kBT) k_base_bits(const int32_t* __restrict__ part, int32_t k, int64_t n,
                                                   uint32_t* __restrict__ bits, int32_t* __restrict__ block_cnt) {
  __shared__ int32_t wc[kBT / 64];
  int32_t c = 0;  // the same in every lane of a wave
  GRID_STRIDE(v0, cdiv_dev(n, 64) * 64) {
    const bool in = v0 < n && part[v0] == k;
    const uint64_t m = __ballot(in);
    c += (int32_t)__popcll(m);
    if ((threadIdx.x & 63) == 0) {
      const int64_t wd = v0 >> 5;
      bits[wd] = (uint32_t)m;
      if ((v0 + 32) < n) bits[wd + 1] = (uint32_t)(m >> 32);
    }
  }
  if ((threadIdx.x & 63) == 0) wc[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0;
    for (int q = 0; q < kBT / 64; ++q) t += wc[q];
    block_cnt[blockIdx.x] = t;
  }
}

// out[0] = sum of the nb block counts (one block, fixed order).
__global__ void __launch_bounds__(256) k_sum_counts(const int32_t* __restrict__ block_cnt, int nb,
                                                    int32_t* __restrict__ out) {
  __shared__ int32_t red[256];
  int32_t t = 0;
  for (int i = threadIdx.x; i < nb; i += 256) t += block_cnt[i];
  red[threadIdx.x] = t;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = red[0];
}

// Membership of the subgraph's node set: base nodes and selected overlap nodes.
__global__ void k_member_bits(const int32_t* __restrict__ part, int32_t k, const uint8_t* __restrict__ sel,
                              int64_t n, uint32_t* __restrict__ bits) {
  GRID_STRIDE(v0, cdiv_dev(n, 64) * 64) {
    const bool in = v0 < n && (part[v0] == k || sel[v0]);
    const uint64_t m = __ballot(in);
    if ((threadIdx.x & 63) == 0) {
      const int64_t wd = v0 >> 5;
      bits[wd] = (uint32_t)m;
      if ((v0 + 32) < n) bits[wd + 1] = (uint32_t)(m >> 32);
    }
  }
}

__device__ __forceinline__ bool bit_of(const uint32_t* __restrict__ bits, int32_t v) {
  return (bits[v >> 5] >> (v & 31)) & 1u;
}

// ---- block-aggregated atomics -----------------------------------------------
// A heavy-tailed graph sends a large share of all edges to a few hub nodes and
// many edges to each of the next thousand or so: one global atomic per edge
// on such a counter serialises (a 1M-node graph whose top source holds 19% of
// 20M edges spent ~18 ms in one such pass).  Each block therefore combines its
// updates in an LDS hash table first (open addressing, 4 probes; integer add or
// min, whose result does not depend on the order) and sends one global
// atomic per table entry when it is done; a key that finds no free slot goes
// straight to the global atomic.  Hot keys arrive early and keep their slots.
constexpr int kAggBits = 11, kAggSlots = 1 << kAggBits;
constexpr uint32_t kAggEmpty = 0xFFFFFFFFu;

template <bool kMin, int kBits = kAggBits>
struct LdsAgg {
  static constexpr int kSlots = 1 << kBits;
  uint32_t* key;  // [kSlots] in LDS
  int32_t* val;
  __device__ __forceinline__ void init() {
    for (int q = threadIdx.x; q < kSlots; q += blockDim.x) {
      key[q] = kAggEmpty;
      val[q] = kMin ? INT32_MAX : 0;
    }
  }
  __device__ __forceinline__ void put(uint32_t k, int32_t v, int32_t* __restrict__ tgt) {
    uint32_t h = (k * 0x9E3779B1u) >> (32 - kBits);
#pragma unroll
    for (int probe = 0; probe < 4; ++probe) {
      // a plain read first: a full table costs loads, not compare-and-swaps
      uint32_t cur = __atomic_load_n(&key[h], __ATOMIC_RELAXED);
      if (cur == kAggEmpty) cur = atomicCAS(&key[h], kAggEmpty, k);
      if (cur == kAggEmpty || cur == k) {
        if (kMin) {
          atomicMin(&val[h], v);
        } else {
          atomicAdd(&val[h], v);
        }
        return;
      }
      h = (h + 1) & (kSlots - 1);
    }
    if (kMin) {
      atomicMin(&tgt[k], v);
    } else {
      atomicAdd(&tgt[k], v);
    }
  }
  // after a __syncthreads: one global atomic per filled slot
  __device__ __forceinline__ void flush(int32_t* __restrict__ tgt) {
    for (int q = threadIdx.x; q < kSlots; q += blockDim.x) {
      const uint32_t k = key[q];
      if (k != kAggEmpty) {
        if (kMin) {
          atomicMin(&tgt[k], val[q]);
        } else {
          atomicAdd(&tgt[k], val[q]);
        }
      }
    }
  }
};

// Launch shape of the aggregation passes: blocks of 512 threads, three per
// compute unit (the edge pass's three tables take 48 KB of LDS), each working
// through a long stretch of edges before it flushes its table.
constexpr int kAggBT = 512;
inline unsigned agg_grid(int64_t n, int per_cu = 3) {
  const int64_t b = cdiv(n > 0 ? n : 1, kAggBT), cap = (int64_t)num_cus() * per_cu;
  return (unsigned)(b < cap ? b : cap);
}

// The out-degree counts: every edge adds 1 to its source, and with Zipf
// sources a few thousand hubs take most of the edges.  A table of 2^13 slots
// (64 KB, two blocks per compute unit) keeps far more of them than the
// 2^11-slot tables of the passes that hold several tables at once.
constexpr int kDegBits = 13, kDegSlots = 1 << kDegBits, kDegPerCu = 2;
constexpr int kEpItems = 4;

// Range checks and the candidates C_k: every node outside V_k joined to V_k
// by an edge gets first[v] < n_edges -- in a dense build the smallest index of
// such an edge (block-aggregated atomic minimum), otherwise 0 (a plain store:
// every writer stores the same value, and a node already marked is only
// read).  Out-degrees: of every node when count_all (the h-index needs them),
// else of the nodes outside V_k when count_out (the out-degree key of the
// candidates, all of which lie outside V_k), else none (keys given by the
// caller).
__global__ void __launch_bounds__(kAggBT) k_edges_pass(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                                   const uint8_t* __restrict__ rel,
                                                   const uint32_t* __restrict__ base_bits, int64_t n_nodes,
                                                   int64_t n_edges, int32_t n_rel, int count_all, int count_out,
                                                   int64_t budget, int32_t* __restrict__ outdeg,
                                                   int32_t* __restrict__ first, int32_t* __restrict__ cnt) {
  __shared__ uint32_t lk[3][kAggSlots];
  __shared__ int32_t lv[3][kAggSlots];
  LdsAgg<false> deg{lk[0], lv[0]};
  LdsAgg<true> fs{lk[1], lv[1]}, fd{lk[2], lv[2]};
  const bool exact = dense_build(cnt[C_BASE], budget, n_nodes);
  const bool counting = count_all || count_out;
  if (counting) deg.init();
  if (exact) {
    fs.init();
    fd.init();
  }
  __syncthreads();
  // kEpItems edges per thread and round (strided by the grid), every load of
  // a round issued before the lookups that depend on it
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e0 < n_edges; e0 += kEpItems * stride) {
    int32_t sv[kEpItems], dv[kEpItems];
    uint32_t rv[kEpItems], ws[kEpItems], wd[kEpItems];
    bool ok[kEpItems], ps[kEpItems], pd[kEpItems];
    // loads without branches (an index past the end reads the last edge and
    // counts for nothing; an endpoint out of range reads word 0), so the
    // loads of all items are in flight together
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      const int64_t e = e0 + j * stride;
      const int64_t ec = e < n_edges ? e : n_edges - 1;
      sv[j] = src[ec];
      dv[j] = dst[ec];
      rv[j] = rel[ec];
    }
    uint32_t is[kEpItems], id[kEpItems];
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      const bool in_range = sv[j] >= 0 && sv[j] < n_nodes && dv[j] >= 0 && dv[j] < n_nodes;
      is[j] = in_range ? (uint32_t)sv[j] >> 5 : 0u;
      id[j] = in_range ? (uint32_t)dv[j] >> 5 : 0u;
    }
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      ws[j] = base_bits[is[j]];
      wd[j] = base_bits[id[j]];
    }
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      const int64_t e = e0 + j * stride;
      const bool in_range = sv[j] >= 0 && sv[j] < n_nodes && dv[j] >= 0 && dv[j] < n_nodes;
      ok[j] = e < n_edges && in_range && rv[j] < (uint32_t)n_rel;
      if (e < n_edges && !ok[j]) atomicOr(&cnt[C_ERR], 1);
      ps[j] = ok[j] && ((ws[j] >> (sv[j] & 31)) & 1u);
      pd[j] = ok[j] && ((wd[j] >> (dv[j] & 31)) & 1u);
    }
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      if (!ok[j]) continue;
      const int64_t e = e0 + j * stride;
      const int32_t s = sv[j], d = dv[j];
      if (count_all || (count_out && !ps[j])) deg.put((uint32_t)s, 1, outdeg);
      if (exact) {
        if (pd[j] && !ps[j]) fs.put((uint32_t)s, (int32_t)e, first);
        if (ps[j] && !pd[j]) fd.put((uint32_t)d, (int32_t)e, first);
      } else {
        if (pd[j] && !ps[j] && first[s] != 0) first[s] = 0;
        if (ps[j] && !pd[j] && first[d] != 0) first[d] = 0;
      }
    }
  }
  __syncthreads();
  if (counting) deg.flush(outdeg);
  if (exact) {
    fs.flush(first);
    fd.flush(first);
  }
}

// Out-degrees of every node, with the range checks of the edge arrays.
__global__ void __launch_bounds__(kAggBT) k_all_outdeg(const int32_t* __restrict__ src,
                                                   const int32_t* __restrict__ dst,
                                                   const uint8_t* __restrict__ rel, int64_t n_nodes,
                                                   int64_t n_edges, int32_t n_rel, int32_t* __restrict__ outdeg,
                                                   int32_t* __restrict__ cnt) {
  __shared__ uint32_t lk[kDegSlots];
  __shared__ int32_t lv[kDegSlots];
  LdsAgg<false, kDegBits> deg{lk, lv};
  deg.init();
  __syncthreads();
  // kEpItems edges per thread and round, all their loads issued first
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t e0 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e0 < n_edges; e0 += kEpItems * stride) {
    int32_t sv[kEpItems], dv[kEpItems];
    uint32_t rv[kEpItems];
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      const int64_t e = e0 + j * stride;
      const int64_t ec = e < n_edges ? e : n_edges - 1;
      sv[j] = src[ec];
      dv[j] = dst[ec];
      rv[j] = rel[ec];
    }
#pragma unroll
    for (int j = 0; j < kEpItems; ++j) {
      if (e0 + j * stride >= n_edges) continue;
      if (sv[j] < 0 || sv[j] >= n_nodes || dv[j] < 0 || dv[j] >= n_nodes || rv[j] >= (uint32_t)n_rel) {
        atomicOr(&cnt[C_ERR], 1);
        continue;
      }
      deg.put((uint32_t)sv[j], 1, outdeg);
    }
  }
  __syncthreads();
  deg.flush(outdeg);
}

__global__ void k_check_ntype(const uint8_t* __restrict__ ntype, int64_t n, int32_t n_ntype,
                              int32_t* __restrict__ cnt) {
  GRID_STRIDE(v, n) {
    if (ntype[v] >= n_ntype) atomicOr(&cnt[C_ERR], 2);
  }
}

// h-index histogram sizes: D+1 bins for every candidate of out-degree D.
__global__ void k_hindex_sizes(const int32_t* __restrict__ outdeg, const int32_t* __restrict__ first,
                               int64_t n, int32_t n_edges, int32_t* __restrict__ sz) {
  GRID_STRIDE(v, n) { sz[v] = (first[v] < n_edges) ? outdeg[v] + 1 : 0; }
}

__global__ void __launch_bounds__(kAggBT) k_hindex_hist(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                                    int64_t n_edges, const int32_t* __restrict__ outdeg,
                                                    const int32_t* __restrict__ first,
                                                    const int32_t* __restrict__ hoff, int32_t* __restrict__ hist) {
  __shared__ uint32_t lk[kAggSlots];
  __shared__ int32_t lv[kAggSlots];
  LdsAgg<false> agg{lk, lv};
  agg.init();
  __syncthreads();
  GRID_STRIDE(e, n_edges) {
    const int32_t s = src[e];
    if (first[s] < (int32_t)n_edges) {
      const int32_t ds = outdeg[s];
      const int32_t c = min(outdeg[dst[e]], ds);
      agg.put((uint32_t)(hoff[s] + c), 1, hist);  // hoff[s] + c < E + N < 2^31
    }
  }
  __syncthreads();
  agg.flush(hist);
}

// key[v] = max h with #{neighbour degrees >= h} >= h, scanning h upwards.
__global__ void k_hindex_final(const int32_t* __restrict__ outdeg, const int32_t* __restrict__ first,
                               const int32_t* __restrict__ hoff, const int32_t* __restrict__ hist,
                               int64_t n, int32_t n_edges, int32_t* __restrict__ key) {
  GRID_STRIDE(v, n) {
    if (first[v] >= n_edges) continue;
    const int32_t D = outdeg[v];
    const int32_t* hv = hist + hoff[v];
    int32_t h = 0, ge = D;  // ge = #{values >= h}
    while (h < D) {
      const int32_t nxt = ge - hv[h];
      if (nxt >= h + 1) {
        ++h;
        ge = nxt;
      } else {
        break;
      }
    }
    key[v] = h;
  }
}

__global__ void k_copy_key(const int32_t* __restrict__ outdeg, int64_t n, int32_t* __restrict__ key) {
  GRID_STRIDE(v, n) { key[v] = outdeg[v]; }
}

__global__ void k_filter_flags(const int32_t* __restrict__ first, const int32_t* __restrict__ key,
                               int64_t n, int32_t n_edges, int32_t theta, int32_t* __restrict__ flag) {
  GRID_STRIDE(v, n) { flag[v] = (first[v] < n_edges && key[v] <= theta) ? 1 : 0; }
}

__global__ void k_compact_nodes(const int32_t* __restrict__ first, const int32_t* __restrict__ key,
                                const int32_t* __restrict__ pos, int64_t n, int32_t n_edges,
                                int32_t theta, int32_t* __restrict__ list) {
  GRID_STRIDE(v, n) {
    if (first[v] < n_edges && key[v] <= theta) list[pos[v]] = (int32_t)v;
  }
}

__global__ void k_select_init(SelectState* st, const int32_t* __restrict__ cprime, int64_t budget) {
  const int t = threadIdx.x;
  st->hist[t] = 0;
  if (t == 0) {
    const int64_t c = *cprime;
    const int64_t take = budget < c ? budget : c;
    st->k_rem = (uint32_t)take;
    st->npass = 0;
    st->mode = (take == 0) ? 2u : ((take == c) ? 1u : 0u);
  }
  if (t < 16) st->digits[t] = 0;
}

__device__ __forceinline__ bool prefix_match(const SelectState* st, uint32_t key, uint64_t h,
                                             uint32_t gid, int npass) {
  for (int p = 0; p < npass; ++p)
    if (composite_digit(key, h, gid, p) != st->digits[p]) return false;
  return true;
}

__global__ void k_select_hist(SelectState* st, const int32_t* __restrict__ list,
                              const int32_t* __restrict__ cprime, const int32_t* __restrict__ key,
                              uint64_t seed) {
  __shared__ int lh[256];
  if (st->mode != 0) return;
  lh[threadIdx.x] = 0;
  __syncthreads();
  const int npass = (int)st->npass;
  const int64_t c = *cprime;
  GRID_STRIDE(i, c) {
    const uint32_t gid = (uint32_t)list[i];
    const uint32_t kv = (uint32_t)key[gid];
    const uint64_t h = splitmix64_first(seed ^ (uint64_t)gid);
    if (prefix_match(st, kv, h, gid, npass)) atomicAdd(&lh[composite_digit(kv, h, gid, npass)], 1);
  }
  __syncthreads();
  if (lh[threadIdx.x]) atomicAdd(&st->hist[threadIdx.x], lh[threadIdx.x]);
}

// One block of 256 threads: pick the bucket holding the k_rem-th smallest.
__global__ void k_select_pick(SelectState* st) {
  __shared__ int cnt[256];
  __shared__ int pre[256];
  if (st->mode != 0) return;
  const int t = threadIdx.x;
  cnt[t] = st->hist[t];
  __syncthreads();
  if (t == 0) {
    int run = 0;
    for (int b = 0; b < 256; ++b) {
      pre[b] = run;
      run += cnt[b];
    }
  }
  __syncthreads();
  const uint32_t k = st->k_rem;
  const uint32_t lo = (uint32_t)pre[t], c = (uint32_t)cnt[t];
  __syncthreads();
  if (c > 0 && lo < k && k <= lo + c) {
    const uint32_t p = st->npass;
    st->digits[p] = (uint32_t)t;
    st->npass = p + 1;
    st->k_rem = k - lo;
    if (k - lo == c) st->mode = 1;
  }
  st->hist[t] = 0;
}

__global__ void k_select_mark(const SelectState* st, const int32_t* __restrict__ list,
                              const int32_t* __restrict__ cprime, const int32_t* __restrict__ key,
                              uint64_t seed, uint8_t* __restrict__ sel) {
  const uint32_t mode = st->mode;
  if (mode == 2) return;
  const int npass = (int)st->npass;
  const int64_t c = *cprime;
  GRID_STRIDE(i, c) {
    const uint32_t gid = (uint32_t)list[i];
    const uint32_t kv = (uint32_t)key[gid];
    const uint64_t h = splitmix64_first(seed ^ (uint64_t)gid);
    bool le = true;
    for (int p = 0; p < npass; ++p) {
      const uint32_t dg = composite_digit(kv, h, gid, p);
      if (dg != st->digits[p]) {
        le = dg < st->digits[p];
        break;
      }
    }
    if (le) sel[gid] = 1;
  }
}

// Node-set digits for the relabel; in a sparse build the selected nodes'
// first[] goes back to n_edges for the base-edge minimum of the induced-edge
// pass.
__global__ void k_member_digit(const int32_t* __restrict__ part, int32_t k,
                               const uint8_t* __restrict__ sel, const uint8_t* __restrict__ ntype,
                               int64_t n, int64_t n_edges, int64_t budget, const int32_t* __restrict__ cnt,
                               uint8_t* __restrict__ digit, int32_t* __restrict__ iota, int32_t* __restrict__ first) {
  const bool exact = dense_build(cnt[C_BASE], budget, n);
  GRID_STRIDE(v, n) {
    digit[v] = (part[v] == k || sel[v]) ? ntype[v] : (uint8_t)255;
    iota[v] = (int32_t)v;
    if (!exact && sel[v]) first[v] = (int32_t)n_edges;
  }
}

__global__ void k_global2local(const int32_t* __restrict__ l2g, const int32_t* __restrict__ type_off,
                               int32_t n_ntype, int32_t* __restrict__ g2l, int32_t* __restrict__ cnt) {
  const int64_t ns = type_off[n_ntype];
  if (blockIdx.x == 0 && threadIdx.x == 0) cnt[C_NSUB] = (int32_t)ns;
  GRID_STRIDE(i, ns) { g2l[l2g[i]] = (int32_t)i; }
}

__global__ void k_overlap_flags(const int32_t* __restrict__ l2g, const uint8_t* __restrict__ sel,
                                const int32_t* __restrict__ cnt, int64_t n, int32_t* __restrict__ flag) {
  const int64_t ns = cnt[C_NSUB];
  GRID_STRIDE(i, n) { flag[i] = (i < ns && sel[l2g[i]]) ? 1 : 0; }
}

__global__ void k_overlap_fill(const int32_t* __restrict__ l2g, const int32_t* __restrict__ flag,
                               const int32_t* __restrict__ pos, const int32_t* __restrict__ cnt,
                               const int32_t* __restrict__ part, const int32_t* __restrict__ first,
                               const uint8_t* __restrict__ rel, int32_t* __restrict__ overlap,
                               int32_t* __restrict__ home, uint8_t* __restrict__ orel) {
  const int64_t ns = cnt[C_NSUB];
  GRID_STRIDE(i, ns) {
    if (flag[i]) {
      const int32_t p = pos[i];
      const int32_t g = l2g[i];
      overlap[p] = (int32_t)i;
      home[p] = part[g];
      orel[p] = rel[first[g]];
    }
  }
}

// ---- induced edges from a rank table (node types 0 and 1) ------------------
// Local ids order the node set by (type, gid).  For 32 consecutive gids an
// entry holds the masks of their type-0 and type-1 members and the number of
// type-0 and type-1 members before them (16 bytes per 32 nodes, 5 MB for 10M
// nodes, where global2local takes 40 MB), so
//   local(v) = pre0 + popc(mem0 below v)                          (type 0)
//   local(v) = type_off[1] + pre1 + popc(mem1 below v)            (type 1)
// and -1 outside the node set: one 16-byte load per endpoint.
struct __align__(16) RankEnt {
  uint32_t mem0, mem1, pre0, pre1;
};
constexpr int kRankGroup = 32;

// Masks and member counts of every 32-node group (one wave per two groups).
__global__ void __launch_bounds__(kBT) k_rank_bits(const int32_t* __restrict__ part, int32_t k,
                                                   const uint8_t* __restrict__ sel, const uint8_t* __restrict__ ntype,
                                                   int64_t n, RankEnt* __restrict__ rt, int32_t* __restrict__ c0,
                                                   int32_t* __restrict__ c1) {
  GRID_STRIDE(v, cdiv_dev(n, 64) * 64) {
    const bool in = v < n && (part[v] == k || sel[v]);
    const bool t1 = in && ntype[v] == 1;
    const uint64_t m = __ballot(in), m1 = __ballot(t1), m0 = m & ~m1;
    const int l = threadIdx.x & 63;
    if (l < 2) {  // lane h writes group 2 (v / 64) + h, the half h of the wave's 64 nodes
      const int64_t b = (v >> 6) * 2 + l;
      const uint32_t g0 = (uint32_t)(m0 >> (32 * l)), g1 = (uint32_t)(m1 >> (32 * l));
      rt[b].mem0 = g0;
      rt[b].mem1 = g1;
      c0[b] = __popc(g0);
      c1[b] = __popc(g1);
    }
  }
}

__global__ void k_rank_pack(const int32_t* __restrict__ pre0, const int32_t* __restrict__ pre1, int64_t nb,
                            RankEnt* __restrict__ rt) {
  GRID_STRIDE(b, nb) {
    rt[b].pre0 = (uint32_t)pre0[b];
    rt[b].pre1 = (uint32_t)pre1[b];
  }
}

// The local id of v from its group's entry (already loaded), -1 outside.
__device__ __forceinline__ int32_t rank_of(uint4 a, int32_t off1, int32_t v) {
  const uint32_t bit = 1u << (v & 31), below = bit - 1u;
  const int32_t r0 = (int32_t)a.z + __popc(a.x & below);
  const int32_t r1 = off1 + (int32_t)a.w + __popc(a.y & below);
  return (a.x & bit) ? r0 : ((a.y & bit) ? r1 : -1);
}

// Edges in tiles of kETile = 16 rounds of kBT consecutive edges (round j of a
// tile: edges base + kBT j .. + kBT - 1, one per thread, coalesced).
constexpr int kERounds = 16;
constexpr int kETile = kBT * kERounds;

// The CSR entry of every kept edge at its edge index: key dst_local * R + r
// and the source's local id (and the edge id or weight when the sort
// carries one); a bit per edge, set when the edge is kept (both endpoints in
// the node set, not after the snapshot cut: keep[e / 64] bit e % 64, one
// ballot per wave and round); and the number of kept edges per tile.  When
// every edge is kept the entries are the sort's input as they stand;
// otherwise k_edge_emit compacts them.  In a sparse build also the base edge
// of every selected node: the smallest index of an edge of the node set
// joining it to V_k (atomic minimum; the selected nodes are few and of small
// key).
template <bool kTs, bool kW>
__global__ void __launch_bounds__(kBT) k_edge_ids(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                                                  const uint8_t* __restrict__ rel, int32_t n_rel,
                                                  const RankEnt* __restrict__ rt, const int32_t* __restrict__ type_off,
                                                  const uint32_t* __restrict__ base_bits, const int32_t* __restrict__ ts,
                                                  int32_t t_cut, int64_t n_edges, int sparse,
                                                  uint32_t* __restrict__ kcsr, int32_t* __restrict__ vsrc,
                                                  int32_t* __restrict__ veid, const float* __restrict__ edge_w,
                                                  int32_t* __restrict__ vw, uint64_t* __restrict__ keep_bits,
                                                  int32_t* __restrict__ tile_cnt, int32_t* __restrict__ first) {
  __shared__ int32_t wsum[kBT / 64];
  const int64_t base = (int64_t)blockIdx.x * kETile;
  const int32_t off1 = type_off[1];
  int32_t c = 0;
  // kEiItems rounds at a time, each phase's loads issued for all of them
  // before any is used: the endpoints (with relation, weight and timestamp),
  // then the sources' rank entries, then the destinations' (looked up only
  // for an edge whose source is in the node set -- in a sparse build most
  // are not -- and neither for an edge after the snapshot cut in a dense
  // build; a sparse build still needs such an edge for the base edges)
  constexpr int kEiItems = 4;
  for (int j0 = 0; j0 < kERounds; j0 += kEiItems) {
    int32_t sv[kEiItems], dv[kEiItems], wv[kEiItems];
    uint32_t rv[kEiItems];
    bool in[kEiItems], late[kEiItems];
#pragma unroll
    for (int u = 0; u < kEiItems; ++u) {
      // past the end: the last edge's loads, and nothing kept
      const int64_t e = base + (int64_t)(j0 + u) * kBT + threadIdx.x;
      in[u] = e < n_edges;
      const int64_t ec = in[u] ? e : n_edges - 1;
      sv[u] = src[ec];
      dv[u] = dst[ec];
      rv[u] = rel[ec];
      wv[u] = kW ? __float_as_int(edge_w[ec]) : 0;
      late[u] = kTs ? ts[ec] > t_cut : false;
    }
    uint4 ra[kEiItems];
#pragma unroll
    for (int u = 0; u < kEiItems; ++u) {
      ra[u] = uint4{0u, 0u, 0u, 0u};
      if (in[u] && !(late[u] && !sparse)) ra[u] = *reinterpret_cast<const uint4*>(rt + (sv[u] >> 5));
    }
    int32_t a[kEiItems];
#pragma unroll
    for (int u = 0; u < kEiItems; ++u) a[u] = rank_of(ra[u], off1, sv[u]);
    uint4 rb[kEiItems];
#pragma unroll
    for (int u = 0; u < kEiItems; ++u) {
      rb[u] = uint4{0u, 0u, 0u, 0u};
      if (a[u] >= 0) rb[u] = *reinterpret_cast<const uint4*>(rt + (dv[u] >> 5));
    }
#pragma unroll
    for (int u = 0; u < kEiItems; ++u) {
      const int64_t e = base + (int64_t)(j0 + u) * kBT + threadIdx.x;
      const int32_t b = a[u] >= 0 ? rank_of(rb[u], off1, dv[u]) : -1;
      if (sparse && a[u] >= 0 && b >= 0) {
        const bool ps = bit_of(base_bits, sv[u]), pd = bit_of(base_bits, dv[u]);
        if (pd && !ps) atomicMin(&first[sv[u]], (int32_t)e);
        if (ps && !pd) atomicMin(&first[dv[u]], (int32_t)e);
      }
      const bool keep = !late[u] && a[u] >= 0 && b >= 0;
      if (keep) {
        kcsr[e] = (uint32_t)b * (uint32_t)n_rel + rv[u];
        vsrc[e] = a[u];
        if (veid) veid[e] = (int32_t)e;
        if (kW) vw[e] = wv[u];
      }
      const uint64_t kb = __ballot(keep);
      // the wave's 64 edges start at a multiple of 64 (tiles of kETile)
      if ((threadIdx.x & 63) == 0 && base + (int64_t)(j0 + u) * kBT + (threadIdx.x & ~63) < n_edges)
        keep_bits[(base + (int64_t)(j0 + u) * kBT + threadIdx.x) >> 6] = kb;
      c += __popcll(kb);
    }
  }
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t t = 0;
#pragma unroll
    for (int q = 0; q < kBT / 64; ++q) t += wsum[q];
    tile_cnt[blockIdx.x] = t;
  }
}

// Stable compaction of the kept CSR entries of a tile at tile_off[tile]
// (exclusive scan of the tile counts): the rank of a kept entry is the
// number of kept entries before it in (round, wave, lane) order, i.e. in
// edge order.  v2 / o2: the second sort value (edge id or weight), or null.
__global__ void __launch_bounds__(kBT) k_edge_emit(const uint32_t* __restrict__ kin, const int32_t* __restrict__ v1,
                                                   const int32_t* __restrict__ v2,
                                                   const uint64_t* __restrict__ keep_bits, int64_t n_edges,
                                                   const int32_t* __restrict__ tile_off, uint32_t* __restrict__ kout,
                                                   int32_t* __restrict__ o1, int32_t* __restrict__ o2) {
  constexpr int NW = kBT / 64;
  __shared__ int32_t cnt[kERounds * NW];
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  const uint64_t lt = (l == 0) ? 0ull : (~0ull >> (64 - l));
  const int64_t base = (int64_t)blockIdx.x * kETile;
  uint64_t bal[kERounds];
#pragma unroll
  for (int j = 0; j < kERounds; ++j) {
    const int64_t e0 = base + (int64_t)j * kBT + 64 * w;
    bal[j] = e0 < n_edges ? keep_bits[e0 >> 6] : 0ull;
    if (l == 0) cnt[j * NW + w] = (int32_t)__popcll(bal[j]);
  }
  __syncthreads();
  if (threadIdx.x == 0) {  // exclusive prefix in (round, wave) order
    int32_t run = 0;
    for (int q = 0; q < kERounds * NW; ++q) {
      const int32_t c = cnt[q];
      cnt[q] = run;
      run += c;
    }
  }
  __syncthreads();
  const int32_t t0 = tile_off[blockIdx.x];
#pragma unroll
  for (int j = 0; j < kERounds; ++j) {
    if ((bal[j] >> l) & 1ull) {
      const int64_t e = base + (int64_t)j * kBT + threadIdx.x;
      const int32_t p = t0 + cnt[j * NW + w] + (int32_t)__popcll(bal[j] & lt);
      kout[p] = kin[e];
      o1[p] = v1[e];
      if (v2) o2[p] = v2[e];
    }
  }
}

// Keep flag of every edge: both endpoints in the node set (two lookups in the
// membership bitmap, N/8 bytes, which stays in the L2 cache).  With
// timestamps, an edge after the cut is dropped like an edge that leaves the
// node set.
// An edge of the node set (timestamps aside) between a selected node and a
// base node is a candidate edge of the selected node: the smallest such index
// is its base edge (atomic minimum; selected nodes are few and of small key).
__global__ void k_edge_keep(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                            const uint32_t* __restrict__ member, const uint32_t* __restrict__ base_bits,
                            const int32_t* __restrict__ ts, int32_t t_cut, int64_t n_edges,
                            int32_t* __restrict__ keep, int32_t* __restrict__ first) {
  GRID_STRIDE(e, n_edges) {
    const int32_t s = src[e], d = dst[e];
    const bool in = bit_of(member, s) && bit_of(member, d);
    if (in) {
      const bool ps = bit_of(base_bits, s), pd = bit_of(base_bits, d);
      if (pd && !ps) atomicMin(&first[s], (int32_t)e);
      if (ps && !pd) atomicMin(&first[d], (int32_t)e);
    }
    keep[e] = (in && !(ts && ts[e] > t_cut)) ? 1 : 0;
  }
}

// Stable compaction of the kept edges (pos = exclusive scan of keep,
// pos[n_edges] = their count); the local ids of a kept edge's endpoints are
// gathered here, so an edge that leaves the node set costs no lookup.
__global__ void k_edge_compact(const int32_t* __restrict__ src, const int32_t* __restrict__ dst,
                               const int32_t* __restrict__ g2l, const uint8_t* __restrict__ rel,
                               const int32_t* __restrict__ pos, int64_t n_edges, int32_t n_rel,
                               uint32_t* __restrict__ kcsr, int32_t* __restrict__ vsrc, int32_t* __restrict__ veid,
                               const float* __restrict__ edge_w, int32_t* __restrict__ vw) {
  GRID_STRIDE(e, n_edges) {
    const int32_t p = pos[e];
    if (pos[e + 1] != p) {
      kcsr[p] = (uint32_t)g2l[dst[e]] * (uint32_t)n_rel + (uint32_t)rel[e];
      vsrc[p] = g2l[src[e]];
      if (veid) veid[p] = (int32_t)e;
      if (vw) vw[p] = __float_as_int(edge_w[e]);
    }
  }
}

// Row lengths of sorted keys.  A block takes kRCChunk consecutive keys (16
// contiguous ones per thread); a run of equal keys that lies inside the chunk
// is counted by a plain store (no other block sees that key), the chunk's
// first and last runs, which may continue into a neighbour, by an atomic
// add.  A row of any length then costs at most one atomic per chunk it
// touches (a hub's row of millions of entries no longer serialises one
// atomic per wave on one counter).  cnt must be zero on entry.
constexpr int kRCItems = 16;
constexpr int kRCChunk = kBT * kRCItems;
__global__ void __launch_bounds__(kBT) k_row_count(const uint32_t* __restrict__ keys, int64_t n,
                                                   int32_t* __restrict__ cnt) {
  __shared__ int32_t starts[kRCChunk + 1];
  __shared__ int32_t wsum[kBT / 64];
  const int t = threadIdx.x;
  const int64_t base = (int64_t)blockIdx.x * kRCChunk;
  const int m = (int)((n - base) < kRCChunk ? (n - base) : kRCChunk);
  const int p0 = t * kRCItems;
  uint32_t k[kRCItems];
  if (p0 + kRCItems <= m) {
    // 16 consecutive keys as four 16-byte loads (chunks start 64-byte aligned)
    const uint4* kp = reinterpret_cast<const uint4*>(keys + base + p0);
#pragma unroll
    for (int j = 0; j < kRCItems / 4; ++j) {
      const uint4 v = kp[j];
      k[4 * j] = v.x;
      k[4 * j + 1] = v.y;
      k[4 * j + 2] = v.z;
      k[4 * j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < kRCItems; ++j) k[j] = (p0 + j < m) ? keys[base + p0 + j] : 0u;
  }
  uint32_t prev = (p0 > 0 && p0 - 1 < m) ? keys[base + p0 - 1] : ~k[0];
  int nf = 0;
#pragma unroll
  for (int j = 0; j < kRCItems; ++j) {
    nf += (p0 + j < m && (j == 0 ? k[0] != prev : k[j] != k[j - 1])) ? 1 : 0;
  }
  // exclusive scan of the run-start counts over the block
  int inc = nf;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(inc, o, 64);
    if ((t & 63) >= o) inc += v;
  }
  if ((t & 63) == 63) wsum[t >> 6] = inc;
  __syncthreads();
  int off = 0, total = 0;
#pragma unroll
  for (int q = 0; q < kBT / 64; ++q) {
    off += (q < (t >> 6)) ? wsum[q] : 0;
    total += wsum[q];
  }
  int idx = off + inc - nf;
#pragma unroll
  for (int j = 0; j < kRCItems; ++j) {
    if (p0 + j < m && (j == 0 ? k[0] != prev : k[j] != k[j - 1])) starts[idx++] = p0 + j;
  }
  if (t == 0) starts[total] = m;
  __syncthreads();
  const bool cont_in = base > 0 && m > 0 && keys[base - 1] == keys[base];
  const bool cont_out = m > 0 && base + m < n && keys[base + m] == keys[base + m - 1];
  for (int r = t; r < total; r += kBT) {
    const int s0 = starts[r], len = starts[r + 1] - s0;
    const uint32_t key = keys[base + s0];
    if ((r == 0 && cont_in) || (r == total - 1 && cont_out)) {
      atomicAdd(&cnt[key], len);
    } else {
      cnt[key] = len;
    }
  }
}

// The CSC sort's input, taken from the CSR in its order: the key (source, r)
// = csr_col[p] * R + r and, as the value, the destination with the in-degree
// of its row, read from csr_ptr while the row is at hand (rows arrive in
// order).  packed: value = destination | min(deg, 255) << 24 (destinations
// below 2^24), which the sort's last pass unpacks into csc_row and the scale;
// else the destination and, as a second value, the scale w / deg itself (a
// correctly rounded float32 quotient; w = the entry's weight, or 1).  A
// stable sort of this input by its key lists a CSC row by (destination,
// original edge index).  Each thread takes kCiItems entries, one per round of
// the block, all loads of a round issued before any store.
constexpr int kCiItems = 4;
__global__ void __launch_bounds__(kBT) k_csc_input(const uint32_t* __restrict__ kcsr,
                                                   const int32_t* __restrict__ csr_col,
                                                   const int32_t* __restrict__ csr_ptr,
                                                   const float* __restrict__ csr_w, int64_t n, int32_t n_rel,
                                                   int packed, uint32_t* __restrict__ kcsc, int32_t* __restrict__ v1,
                                                   int32_t* __restrict__ v2) {
  const int64_t base = (int64_t)blockIdx.x * (kBT * kCiItems) + threadIdx.x;
  uint32_t key[kCiItems];
  int32_t col[kCiItems], lo[kCiItems], hi[kCiItems];
#pragma unroll
  for (int j = 0; j < kCiItems; ++j) {
    const int64_t p = base + (int64_t)j * kBT;
    key[j] = p < n ? kcsr[p] : 0u;
    col[j] = p < n ? csr_col[p] : 0;
  }
#pragma unroll
  for (int j = 0; j < kCiItems; ++j) {
    const int64_t p = base + (int64_t)j * kBT;
    lo[j] = p < n ? csr_ptr[key[j]] : 0;
    hi[j] = p < n ? csr_ptr[key[j] + 1] : 1;
  }
#pragma unroll
  for (int j = 0; j < kCiItems; ++j) {
    const int64_t p = base + (int64_t)j * kBT;
    if (p < n) {
      const uint32_t dst = key[j] / (uint32_t)n_rel, r = key[j] - dst * (uint32_t)n_rel;
      const int32_t deg = hi[j] - lo[j];
      kcsc[p] = (uint32_t)col[j] * (uint32_t)n_rel + r;
      if (packed) {
        v1[p] = (int32_t)(dst | ((uint32_t)(deg < 255 ? deg : 255) << 24));
      } else {
        v1[p] = (int32_t)dst;
        v2[p] = __float_as_int((csr_w ? csr_w[p] : 1.0f) / (float)deg);
      }
    }
  }
}

__global__ void k_gather_w(const int32_t* __restrict__ eid, const float* __restrict__ edge_w, int64_t n,
                           float* __restrict__ out) {
  GRID_STRIDE(p, n) out[p] = edge_w[eid[p]];
}

// Per CSC row q: relation digit for the active-source partition, work-item
// counts, and the slot table's active mask and count of each 64 rows (one
// wave covers 64 consecutive rows: the grid stride is a multiple of 64).
__global__ void __launch_bounds__(kBT) k_active_digit(const int32_t* __restrict__ csc_ptr, int64_t nq, int32_t n_rel,
                                                      uint8_t* __restrict__ digit, int32_t* __restrict__ srcid,
                                                      int32_t* __restrict__ n_items, int32_t* __restrict__ n_heavy,
                                                      int32_t* __restrict__ n_parts, SlotEnt* __restrict__ tab,
                                                      int32_t* __restrict__ tab_cnt) {
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q - lane < nq; q += stride) {
    const bool live = q < nq;
    const int32_t len = live ? csc_ptr[q + 1] - csc_ptr[q] : 0;
    if (live) {
      digit[q] = len > 0 ? (uint8_t)(q % n_rel) : (uint8_t)255;
      srcid[q] = (int32_t)(q / n_rel);
      const int32_t nch = (len + kChunk - 1) / kChunk;
      n_items[q] = nch;
      n_heavy[q] = nch > 1 ? 1 : 0;
      n_parts[q] = nch > 1 ? nch : 0;
    }
    const uint64_t m = __ballot(len > 0);
    if (lane == 0) {
      tab[q >> 6].mask = m;
      tab_cnt[q >> 6] = (int32_t)__popcll(m);
    }
  }
}

// The count before each 64 rows; for the row-indexed layout the identity
// (all rows marked, 64 b before block b), so that slot(q) = q.
__global__ void k_slot_pack(const int32_t* __restrict__ pre, int64_t nb, int64_t nq,
                            const int32_t* __restrict__ a_total, SlotEnt* __restrict__ tab) {
  const bool by_row = row_layout(nq, *a_total);
  GRID_STRIDE(b, nb) {
    if (by_row) tab[b].mask = ~0ull;
    tab[b].pre = by_row ? (int32_t)(64 * b) : pre[b];
    tab[b].pad = 0;
  }
}

// Work items of the CSC rows (first field: the row's slot) and the slot ->
// row map.
__global__ void k_plan_items(const int32_t* __restrict__ csc_ptr, int64_t nq,
                             const int32_t* __restrict__ item_off, const int32_t* __restrict__ heavy_off,
                             const int32_t* __restrict__ part_off, const SlotEnt* __restrict__ tab,
                             const int32_t* __restrict__ a_total, int4* __restrict__ items, int4* __restrict__ heavy,
                             int32_t* __restrict__ slot_q) {
  const bool by_row = row_layout(nq, *a_total);
  GRID_STRIDE(q, nq) {
    const int32_t beg = csc_ptr[q], end = csc_ptr[q + 1];
    const int32_t len = end - beg;
    if (len <= 0) continue;
    const int32_t sl = slot_of(tab, q);
    if (!by_row) slot_q[sl] = (int32_t)q;
    const int32_t nch = (len + kChunk - 1) / kChunk;
    const int32_t io = item_off[q];
    if (nch == 1) {
      items[io] = make_int4(sl, beg, end, -1);
    } else {
      const int32_t so = part_off[q];
      for (int32_t c = 0; c < nch; ++c) {
        const int32_t b = beg + c * kChunk;
        const int32_t e2 = min(end, b + kChunk);
        items[io + c] = make_int4(sl, b, e2, so + c);
      }
      heavy[heavy_off[q]] = make_int4(sl, so, nch, 0);
    }
  }
}

// Destination rows longer than kFwdChunk entries: per node j a 0/1 flag
// and its number of chunks (0 for the rows one wave walks).
__global__ void k_fwd_counts(const int32_t* __restrict__ csr_ptr, int64_t ns, int32_t n_rel,
                             int32_t* __restrict__ heavy_flag, int32_t* __restrict__ n_parts) {
  GRID_STRIDE(j, ns) {
    const int32_t len = csr_ptr[(j + 1) * n_rel] - csr_ptr[j * n_rel];
    const int32_t nch = len > kFwdChunk ? (len + kFwdChunk - 1) / kFwdChunk : 0;
    heavy_flag[j] = nch > 0 ? 1 : 0;
    n_parts[j] = nch;
  }
}

// The chunks of the long destination rows (each chunk is one partial slot)
// and one entry per long row.
__global__ void k_fwd_items(const int32_t* __restrict__ csr_ptr, int64_t ns, int32_t n_rel,
                            const int32_t* __restrict__ heavy_off, const int32_t* __restrict__ part_off,
                            int4* __restrict__ items, int4* __restrict__ heavy) {
  GRID_STRIDE(j, ns) {
    const int32_t beg = csr_ptr[j * n_rel], end = csr_ptr[(j + 1) * n_rel];
    const int32_t len = end - beg;
    if (len <= kFwdChunk) continue;
    const int32_t nch = (len + kFwdChunk - 1) / kFwdChunk;
    const int32_t so = part_off[j];
    for (int32_t c = 0; c < nch; ++c) {
      const int32_t b = beg + c * kFwdChunk;
      items[so + c] = make_int4((int32_t)j, b, min(end, b + kFwdChunk), so + c);
    }
    heavy[heavy_off[j]] = make_int4((int32_t)j, so, nch, 0);
  }
}

// Slot of each entry of the per-relation active-source lists.
__global__ void k_act_slot(const int32_t* __restrict__ act, const int32_t* __restrict__ act_off, int32_t n_rel,
                           int64_t cap, const SlotEnt* __restrict__ tab, int32_t* __restrict__ act_slot) {
  const int64_t n = act_off[n_rel];
  GRID_STRIDE(k, cap) {
    if (k >= n) break;
    int32_t lo = 0, hi = n_rel;  // act_off[lo] <= k < act_off[hi]
    while (hi - lo > 1) {
      const int32_t mid = (lo + hi) >> 1;
      if (act_off[mid] <= k) lo = mid; else hi = mid;
    }
    act_slot[k] = slot_of(tab, (int64_t)act[k] * n_rel + lo);
  }
}

// Slot of the (source, relation) row of each CSR entry; the relation is the
// low part of the entry's sorted CSR key dst * R + r.
__global__ void k_csr_slot(const int32_t* __restrict__ csr_col, const uint32_t* __restrict__ kcsr, int64_t n,
                           int32_t n_rel, int64_t nq, const int32_t* __restrict__ a_total,
                           const SlotEnt* __restrict__ tab, int32_t* __restrict__ csr_slot) {
  if (row_layout(nq, *a_total)) return;  // the kernels index by q
  GRID_STRIDE(p, n) {
    const int64_t q = (int64_t)csr_col[p] * n_rel + (int64_t)(kcsr[p] % (uint32_t)n_rel);
    csr_slot[p] = slot_of(tab, q);
  }
}

// The CSC sort packs destination and row degree into one value while the
// destinations fit in 24 bits.
constexpr int64_t kPackedMaxNodes = (int64_t)1 << 24;

int bits_for(int64_t nvals) {
  int b = 0;
  while (b < 32 && ((int64_t)1 << b) < nvals) ++b;
  return b;
}

// Workspace layout, shared by the sizing and the run.
template <class A>
struct BuildWs {
  int32_t *cnt, *outdeg, *first, *key, *flag, *pos, *list, *iota, *hoff, *hist;
  uint8_t *sel, *digit;
  SelectState* st;
  int32_t *keep, *vsrc, *vdst, *veid, *alt1, *alt2, *alt3, *rowcnt, *q_items, *q_heavy, *q_parts,
      *q_src, *scratch, *bcnt;
  int32_t* vw;                // weighted graphs: edge weights (float bits) of the kept edges in edge order
  int32_t *vsc, *vsc_alt;     // unpacked CSC sort: the scales (float bits) and their ping-pong buffer
  uint32_t *kcsr, *kcsc, *kalt, *bbits, *mbits;
  RankEnt* rt;
  int32_t *rc0, *rc1, *tile_cnt;
  void layout(A& a, int64_t N, int64_t E, int64_t R, bool hindex, bool weighted) {
    const int64_t NQ = N * R + 1;
    cnt = a.template take<int32_t>(C_COUNT + 8);
    bcnt = a.template take<int32_t>(16384);  // block counts of k_base_bits (grid_for caps it there)
    outdeg = a.template take<int32_t>(N);
    first = a.template take<int32_t>(N);
    key = a.template take<int32_t>(N);
    flag = a.template take<int32_t>(N + 1);
    pos = a.template take<int32_t>(N + 1);
    list = a.template take<int32_t>(N);
    iota = a.template take<int32_t>(N);
    hoff = a.template take<int32_t>(hindex ? N + 1 : 0);
    hist = a.template take<int32_t>(hindex ? E + N : 0);
    sel = a.template take<uint8_t>(N);
    bbits = a.template take<uint32_t>(N / 32 + 2);
    mbits = a.template take<uint32_t>(2 * (N / 64 + 1));
    // rank groups: cdiv(N, 64) * 2 <= N / 32 + 2
    rt = a.template take<RankEnt>(N / kRankGroup + 2);
    rc0 = a.template take<int32_t>(N / kRankGroup + 2);
    rc1 = a.template take<int32_t>(N / kRankGroup + 2);
    tile_cnt = a.template take<int32_t>(E / kETile + 2);
    digit = a.template take<uint8_t>(NQ > N ? NQ : N);
    st = a.template take<SelectState>(1);
    keep = a.template take<int32_t>(E + 1);
    kcsr = a.template take<uint32_t>(E);
    kcsc = a.template take<uint32_t>(E);
    kalt = a.template take<uint32_t>(E);
    vsrc = a.template take<int32_t>(E);
    vdst = a.template take<int32_t>(E);
    veid = a.template take<int32_t>(E);
    alt1 = a.template take<int32_t>(E);
    alt2 = a.template take<int32_t>(E);
    alt3 = a.template take<int32_t>(E);
    rowcnt = a.template take<int32_t>(NQ);
    q_items = a.template take<int32_t>(NQ);
    q_heavy = a.template take<int32_t>(NQ);
    q_parts = a.template take<int32_t>(NQ);
    q_src = a.template take<int32_t>(NQ);
    vw = a.template take<int32_t>(weighted ? E : 0);
    const bool unpacked = weighted || N >= kPackedMaxNodes;
    vsc = a.template take<int32_t>(unpacked ? E : 0);
    vsc_alt = a.template take<int32_t>(unpacked ? E : 0);
    int64_t sc = scan_scratch_elems(E + N + NQ + 1);
    int64_t rs = radix_scratch_elems(E > NQ ? E : NQ);
    scratch = a.template take<int32_t>(sc > rs ? sc : rs);
  }
};

struct PlanLayout {
  size_t s_off, soff_off, aslot_off, slotq_off, cslot_off, tab_off, items_off, heavy_off, fitems_off, fheavy_off,
      total;
  int64_t cap_s, cap_items, cap_heavy, cap_tab, cap_fitems, cap_fheavy;
  PlanLayout(int64_t N, int64_t E, int64_t R) {
    const int64_t nq = N * R;
    cap_s = nq < E ? nq : E;
    cap_heavy = E / kChunk + 1;
    cap_items = cap_s + cap_heavy;
    cap_tab = nq / 64 + 1;
    // a row of L > kFwdChunk entries has ceil(L / kFwdChunk) < 2 L / kFwdChunk chunks
    cap_fheavy = E / kFwdChunk + 1;
    cap_fitems = 2 * (E / kFwdChunk) + 2;
    const size_t ns = (size_t)(cap_s > 0 ? cap_s : 1);
    size_t o = 0;
    s_off = o; o = align_up(o + sizeof(int32_t) * ns);
    soff_off = o; o = align_up(o + sizeof(int32_t) * (size_t)(R + 1));
    aslot_off = o; o = align_up(o + sizeof(int32_t) * ns);
    slotq_off = o; o = align_up(o + sizeof(int32_t) * ns);
    cslot_off = o; o = align_up(o + sizeof(int32_t) * (size_t)(E > 0 ? E : 1));
    tab_off = o; o = align_up(o + sizeof(SlotEnt) * (size_t)cap_tab);
    items_off = o; o = align_up(o + sizeof(int4) * (size_t)cap_items);
    heavy_off = o; o = align_up(o + sizeof(int4) * (size_t)cap_heavy);
    fitems_off = o; o = align_up(o + sizeof(int4) * (size_t)cap_fitems);
    fheavy_off = o; o = align_up(o + sizeof(int4) * (size_t)cap_fheavy);
    total = o;
  }
};

}  // namespace

PlanView plan_view(const hg_subgraph* s) {
  PlanLayout pl(s->n_nodes, s->n_edges, s->n_rel);
  const char* b = static_cast<const char*>(s->plan);
  PlanView v;
  v.active = reinterpret_cast<const int32_t*>(b + pl.s_off);
  v.act_slot = reinterpret_cast<const int32_t*>(b + pl.aslot_off);
  const bool by_row = s->plan_slot_rows == s->n_sub * (int64_t)s->n_rel;
  v.slot_q = by_row ? nullptr : reinterpret_cast<const int32_t*>(b + pl.slotq_off);
  v.csr_slot = by_row ? nullptr : reinterpret_cast<const int32_t*>(b + pl.cslot_off);
  v.slot_tab = by_row ? nullptr : reinterpret_cast<const SlotEnt*>(b + pl.tab_off);
  v.items = reinterpret_cast<const int4*>(b + pl.items_off);
  v.heavy = reinterpret_cast<const int4*>(b + pl.heavy_off);
  v.fwd_items = reinterpret_cast<const int4*>(b + pl.fitems_off);
  v.fwd_heavy = reinterpret_cast<const int4*>(b + pl.fheavy_off);
  return v;
}

}  // namespace hg

using namespace hg;

extern "C" size_t hg_plan_size(int64_t n_nodes, int64_t n_edges, int32_t n_rel) {
  if (n_nodes < 0 || n_edges < 0 || n_rel < 1) return 0;
  return PlanLayout(n_nodes, n_edges, n_rel).total;
}

static int validate_build(const hg_graph_desc* g, const hg_overlap_desc* o) {
  if (!g || !o) return fail(HG_ERR_ARG, "null descriptor");
  if (g->n_nodes < 1 || g->n_nodes >= ((int64_t)1 << 31))
    return fail(HG_ERR_ARG, "n_nodes %lld outside [1, 2^31)", (long long)g->n_nodes);
  if (g->n_edges < 0) return fail(HG_ERR_ARG, "n_edges %lld < 0", (long long)g->n_edges);
  if (g->n_edges >= ((int64_t)1 << 31))
    return fail(HG_ERR_UNSUPPORTED, "n_edges %lld >= 2^31", (long long)g->n_edges);
  if (g->n_rel < 1 || g->n_rel > HG_MAX_REL) return fail(HG_ERR_UNSUPPORTED, "n_rel %d", g->n_rel);
  if (g->n_ntype < 1 || g->n_ntype > HG_MAX_NTYPE)
    return fail(HG_ERR_UNSUPPORTED, "n_ntype %d", g->n_ntype);
  if (g->n_nodes * (int64_t)g->n_rel >= ((int64_t)1 << 31) - 1)
    return fail(HG_ERR_UNSUPPORTED, "n_nodes * n_rel >= 2^31");
  if (g->n_edges > 0 && (!g->src || !g->dst || !g->rel))
    return fail(HG_ERR_ARG, "null edge array");
  if (!g->ntype || !g->part) return fail(HG_ERR_ARG, "null node array");
  if (o->budget_M < 0) return fail(HG_ERR_ARG, "budget_M < 0");
  if (o->key != HG_KEY_OUTDEG && o->key != HG_KEY_HINDEX) return fail(HG_ERR_ARG, "key %d", o->key);
  if (o->key_dir != HG_KEYDIR_OUT) return fail(HG_ERR_UNSUPPORTED, "key_dir %d", o->key_dir);
  if (o->theta < 0) return fail(HG_ERR_ARG, "theta < 0");
  return HG_OK;
}

// ---- node keys of the whole graph (the same for every partition block) ----

namespace {

struct KeyWs {
  int32_t *cnt, *outdeg, *first, *hoff, *hist, *flag, *scratch;
  template <class A>
  void layout(A& a, int64_t N, int64_t E, bool hindex) {
    cnt = a.template take<int32_t>(C_COUNT + 8);
    outdeg = a.template take<int32_t>(hindex ? N : 0);
    first = a.template take<int32_t>(hindex ? N : 0);
    hoff = a.template take<int32_t>(hindex ? N + 1 : 0);
    hist = a.template take<int32_t>(hindex ? E + N : 0);
    flag = a.template take<int32_t>(hindex ? N + 1 : 0);
    scratch = a.template take<int32_t>(hindex ? scan_scratch_elems(N + 1) : 0);
  }
};

int validate_keys(const hg_graph_desc* g, int32_t key) {
  if (!g) return fail(HG_ERR_ARG, "null descriptor");
  if (g->n_nodes < 1 || g->n_nodes >= ((int64_t)1 << 31))
    return fail(HG_ERR_ARG, "n_nodes %lld outside [1, 2^31)", (long long)g->n_nodes);
  if (g->n_edges < 0) return fail(HG_ERR_ARG, "n_edges %lld < 0", (long long)g->n_edges);
  if (g->n_edges + g->n_nodes >= ((int64_t)1 << 31))
    return fail(HG_ERR_UNSUPPORTED, "n_edges + n_nodes >= 2^31");
  if (g->n_rel < 1 || g->n_rel > HG_MAX_REL) return fail(HG_ERR_UNSUPPORTED, "n_rel %d", g->n_rel);
  if (g->n_edges > 0 && (!g->src || !g->dst || !g->rel)) return fail(HG_ERR_ARG, "null edge array");
  if (key != HG_KEY_OUTDEG && key != HG_KEY_HINDEX) return fail(HG_ERR_ARG, "key %d", key);
  return HG_OK;
}

}  // namespace

extern "C" size_t hg_node_keys_workspace_size(const hg_graph_desc* g, int32_t key) {
  if (validate_keys(g, key) != HG_OK) return 0;
  Sizer sz;
  KeyWs w;
  w.layout(sz, g->n_nodes, g->n_edges, key == HG_KEY_HINDEX);
  return sz.used + 256;
}

extern "C" int hg_node_keys(const hg_graph_desc* g, int32_t key, int32_t* keys, void* ws, size_t ws_bytes,
                            void* stream) {
  HG_TRY(validate_keys(g, key));
  if (!keys) return fail(HG_ERR_ARG, "null keys");
  const size_t need = hg_node_keys_workspace_size(g, key);
  if (!ws || ws_bytes < need) return fail(HG_ERR_CAPACITY, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  const int64_t N = g->n_nodes, E = g->n_edges;
  const bool hindex = key == HG_KEY_HINDEX;
  hipStream_t s = static_cast<hipStream_t>(stream);
  Arena arena(ws, ws_bytes);
  KeyWs w;
  w.layout(arena, N, E, hindex);
  if (!arena.ok()) return fail(HG_ERR_CAPACITY, "workspace layout overflow");
  const unsigned gN = grid_for(N);
  int32_t* deg = hindex ? w.outdeg : keys;
  HG_TRY(fill_i32(w.cnt, 0, C_COUNT + 8, s));
  HG_TRY(fill_i32(keys, 0, N, s));
  if (hindex) HG_TRY(fill_i32(deg, 0, N, s));
  if (E > 0)
    HG_LAUNCH("keys_outdeg", k_all_outdeg, dim3(agg_grid(E, kDegPerCu)), dim3(kAggBT), 0, s, g->src, g->dst, g->rel, N, E,
              g->n_rel, deg, w.cnt);
  int32_t herr = 0;
  HG_HIP_TRY(hipMemcpyAsync(&herr, w.cnt + C_ERR, sizeof(int32_t), hipMemcpyDeviceToHost, s));
  HG_HIP_TRY(hipStreamSynchronize(s));
  if (herr) return fail(HG_ERR_RANGE, "input ids out of range (flags 0x%x)", herr);
  if (hindex && E > 0) {
    // every node is treated as a candidate: first[v] = 0 < E
    HG_TRY(fill_i32(w.first, 0, N, s));
    HG_LAUNCH("keys_hindex_sizes", k_hindex_sizes, dim3(gN), dim3(kBT), 0, s, (const int32_t*)deg,
              (const int32_t*)w.first, N, (int32_t)E, w.flag);
    HG_TRY(fill_i32(w.flag + N, 0, 1, s));
    HG_TRY(scan_exclusive_i32(w.flag, w.hoff, N + 1, nullptr, w.scratch, s));
    HG_TRY(fill_i32(w.hist, 0, E + N, s));
    HG_LAUNCH("keys_hindex_hist", k_hindex_hist, dim3(agg_grid(E)), dim3(kAggBT), 0, s, g->src, g->dst, E,
              (const int32_t*)deg, (const int32_t*)w.first, (const int32_t*)w.hoff, w.hist);
    HG_LAUNCH("keys_hindex_final", k_hindex_final, dim3(gN), dim3(kBT), 0, s, (const int32_t*)deg,
              (const int32_t*)w.first, (const int32_t*)w.hoff, (const int32_t*)w.hist, N, (int32_t)E, keys);
  }
  return HG_OK;
}

extern "C" size_t hg_build_csr_workspace_size(const hg_graph_desc* g, const hg_overlap_desc* o) {
  if (validate_build(g, o) != HG_OK) return 0;
  Sizer sz;
  BuildWs<Sizer> w;
  w.layout(sz, g->n_nodes, g->n_edges, g->n_rel, o->key == HG_KEY_HINDEX, g->edge_w != nullptr);
  return sz.used + 256;
}

extern "C" int hg_build_csr(const hg_graph_desc* g, const hg_overlap_desc* o, hg_subgraph* out,
                            void* ws, size_t ws_bytes, void* stream) {
  HG_TRY(validate_build(g, o));
  if (!out) return fail(HG_ERR_ARG, "null output");
  if (!out->local2global || !out->global2local || !out->type_off || !out->csr_ptr ||
      !out->csc_ptr || !out->plan || (!out->overlap && o->budget_M > 0) ||
      (!out->overlap_home && o->budget_M > 0) || (!out->overlap_rel && o->budget_M > 0) ||
      (g->n_edges > 0 && (!out->csr_col || !out->csc_row || !out->csc_scale)))
    return fail(HG_ERR_ARG, "null output array");
  const bool weighted = g->edge_w != nullptr;
  const bool want_eid = out->csr_eid != nullptr;
  if (weighted && g->n_edges > 0 && !out->csr_w) return fail(HG_ERR_ARG, "a weighted graph needs the csr_w output");
  const int64_t N = g->n_nodes, E = g->n_edges, R = g->n_rel, T = g->n_ntype;
  const size_t need_plan = hg_plan_size(N, E, (int32_t)R);
  if (out->plan_bytes < need_plan)
    return fail(HG_ERR_CAPACITY, "plan needs %zu bytes, got %zu", need_plan, out->plan_bytes);
  const size_t need = hg_build_csr_workspace_size(g, o);
  if (!ws || ws_bytes < need) return fail(HG_ERR_CAPACITY, "workspace needs %zu bytes, got %zu", need, ws_bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const bool hindex = o->key == HG_KEY_HINDEX;

  Arena arena(ws, ws_bytes);
  BuildWs<Arena> w;
  w.layout(arena, N, E, R, hindex, g->edge_w != nullptr);
  if (!arena.ok()) return fail(HG_ERR_CAPACITY, "workspace layout overflow");

  const unsigned gN = grid_for(N), gE = grid_for(E);
  // 1. degrees, base-edge index, range checks
  HG_TRY(fill_i32(w.cnt, 0, C_COUNT + 8, s));
  HG_TRY(fill_i32(w.outdeg, 0, N, s));
  HG_TRY(fill_i32(w.first, (int32_t)E, N, s));
  HG_TRY(fill_u8(w.sel, 0, N, s));
  const unsigned gB = grid_for(cdiv(N, 64) * 64);
  HG_LAUNCH("build_base_bits", k_base_bits, dim3(gB), dim3(kBT), 0, s, g->part, g->k, N, w.bbits, w.bcnt);
  HG_LAUNCH("build_base_count", k_sum_counts, dim3(1), dim3(256), 0, s, (const int32_t*)w.bcnt, (int)gB,
            w.cnt + C_BASE);
  if (E > 0)
    HG_LAUNCH("build_edges_pass", k_edges_pass, dim3(agg_grid(E, kDegPerCu)), dim3(kAggBT), 0, s, g->src, g->dst,
              g->rel, (const uint32_t*)w.bbits, N, E, (int32_t)R, (hindex && !o->node_key) ? 1 : 0,
              (!hindex && !o->node_key) ? 1 : 0, o->budget_M, w.outdeg, w.first, w.cnt);
  HG_LAUNCH("build_check_ntype", k_check_ntype, dim3(gN), dim3(kBT), 0, s, g->ntype, N, (int32_t)T, w.cnt);
  {
    int32_t herr = 0;
    HG_HIP_TRY(hipMemcpyAsync(&herr, w.cnt + C_ERR, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    HG_HIP_TRY(hipStreamSynchronize(s));
    if (herr) return fail(HG_ERR_RANGE, "input ids out of range (flags 0x%x)", herr);
  }
  // 2. keys (the caller's, when given: they do not depend on k)
  const int32_t* key = o->node_key ? o->node_key : w.key;
  if (hindex && !o->node_key) {
    HG_LAUNCH("build_hindex_sizes", k_hindex_sizes, dim3(gN), dim3(kBT), 0, s,
              (const int32_t*)w.outdeg, (const int32_t*)w.first, N, (int32_t)E, w.flag);
    HG_TRY(fill_i32(w.flag + N, 0, 1, s));
    HG_TRY(scan_exclusive_i32(w.flag, w.hoff, N + 1, nullptr, w.scratch, s));
    HG_TRY(fill_i32(w.hist, 0, E + N, s));
    if (E > 0)
      HG_LAUNCH("build_hindex_hist", k_hindex_hist, dim3(agg_grid(E)), dim3(kAggBT), 0, s, g->src, g->dst, E,
                (const int32_t*)w.outdeg, (const int32_t*)w.first, (const int32_t*)w.hoff, w.hist);
    HG_LAUNCH("build_hindex_final", k_hindex_final, dim3(gN), dim3(kBT), 0, s,
              (const int32_t*)w.outdeg, (const int32_t*)w.first, (const int32_t*)w.hoff,
              (const int32_t*)w.hist, N, (int32_t)E, w.key);
  } else if (!o->node_key) {
    // the out-degrees of the nodes outside V_k (every candidate among them)
    HG_LAUNCH("build_copy_key", k_copy_key, dim3(gN), dim3(kBT), 0, s, (const int32_t*)w.outdeg, N, w.key);
  }
  // 3. filtered candidates, compacted in gid order
  HG_LAUNCH("build_filter_flags", k_filter_flags, dim3(gN), dim3(kBT), 0, s, (const int32_t*)w.first,
            key, N, (int32_t)E, o->theta, w.flag);
  HG_TRY(scan_exclusive_i32(w.flag, w.pos, N, w.cnt + C_CPRIME, w.scratch, s));
  HG_LAUNCH("build_compact_nodes", k_compact_nodes, dim3(gN), dim3(kBT), 0, s, (const int32_t*)w.first,
            key, (const int32_t*)w.pos, N, (int32_t)E, o->theta, w.list);
  // 4. TopM by exact radix select over the 128-bit composite
  {
    const int64_t budget = o->budget_M;
    HG_LAUNCH("build_select_init", k_select_init, dim3(1), dim3(256), 0, s, w.st,
              (const int32_t*)(w.cnt + C_CPRIME), budget);
    for (int p = 0; p < 16; ++p) {
      HG_LAUNCH("build_select_hist", k_select_hist, dim3(grid_for(N, 2048)), dim3(256), 0, s, w.st,
                (const int32_t*)w.list, (const int32_t*)(w.cnt + C_CPRIME), key,
                o->seed);
      HG_LAUNCH("build_select_pick", k_select_pick, dim3(1), dim3(256), 0, s, w.st);
    }
    HG_LAUNCH("build_select_mark", k_select_mark, dim3(grid_for(N, 2048)), dim3(256), 0, s,
              (const SelectState*)w.st, (const int32_t*)w.list, (const int32_t*)(w.cnt + C_CPRIME),
              key, o->seed, w.sel);
  }
  // 5. local ids in (ntype, gid) order
  HG_LAUNCH("build_member_digit", k_member_digit, dim3(gN), dim3(kBT), 0, s, g->part, g->k,
            (const uint8_t*)w.sel, g->ntype, N, E, o->budget_M, (const int32_t*)w.cnt, w.digit, w.iota, w.first);
  HG_TRY(bucket_partition(w.digit, w.iota, N, (int)T, out->local2global, out->type_off, w.scratch, s));
  HG_TRY(fill_i32(out->global2local, -1, N, s));
  HG_LAUNCH("build_global2local", k_global2local, dim3(gN), dim3(kBT), 0, s,
            (const int32_t*)out->local2global, (const int32_t*)out->type_off, (int32_t)T,
            out->global2local, w.cnt);
  // 6. induced-subgraph edges in original order, and the base edges of the
  // selected nodes
  // the CSR sort carries the edge id if asked for, else a weighted graph's weight
  const bool emit_w = weighted && !want_eid;
  // with at most two node types the CSR entries are formed in edge order and
  // compacted only if some edge was dropped (below, once the count is known)
  bool rank_path = false;
  const int64_t ntiles = cdiv(E, kETile);
  if (E > 0) {
    int32_t nb_host = 0;
    HG_HIP_TRY(hipMemcpyAsync(&nb_host, w.cnt + C_BASE, sizeof(int32_t), hipMemcpyDeviceToHost, s));
    HG_HIP_TRY(hipStreamSynchronize(s));
    const bool dense = dense_build(nb_host, o->budget_M, N);
    if (T <= 2) {
      rank_path = true;
      const int64_t nb = cdiv(N, 64) * 2;
      HG_LAUNCH("build_rank_bits", k_rank_bits, dim3(grid_for(nb * kRankGroup)), dim3(kBT), 0, s, g->part, g->k,
                (const uint8_t*)w.sel, g->ntype, N, w.rt, w.rc0, w.rc1);
      HG_TRY(scan_exclusive_i32(w.rc0, w.rc0, nb, nullptr, w.scratch, s));
      HG_TRY(scan_exclusive_i32(w.rc1, w.rc1, nb, nullptr, w.scratch, s));
      HG_LAUNCH("build_rank_pack", k_rank_pack, dim3(grid_for(nb)), dim3(kBT), 0, s, (const int32_t*)w.rc0,
                (const int32_t*)w.rc1, nb, w.rt);
#define HG_EDGE_IDS(TS_, W_)                                                                                   \
  HG_LAUNCH("build_edge_ids", (k_edge_ids<TS_, W_>), dim3((unsigned)ntiles), dim3(kBT), 0, s, g->src, g->dst,     \
            g->rel, (int32_t)R, (const RankEnt*)w.rt, (const int32_t*)out->type_off, (const uint32_t*)w.bbits,    \
            g->edge_ts, g->t_cut, E, dense ? 0 : 1, w.kcsr, w.vsrc, want_eid ? w.veid : nullptr, g->edge_w,       \
            emit_w ? w.vw : nullptr, reinterpret_cast<uint64_t*>(w.keep), w.tile_cnt, w.first)
      if (g->edge_ts) {
        if (emit_w) HG_EDGE_IDS(true, true); else HG_EDGE_IDS(true, false);
      } else {
        if (emit_w) HG_EDGE_IDS(false, true); else HG_EDGE_IDS(false, false);
      }
#undef HG_EDGE_IDS
      HG_TRY(scan_exclusive_i32(w.tile_cnt, w.tile_cnt, ntiles, w.cnt + C_ESUB, w.scratch, s));
    } else {
      // more than two node types: local ids from global2local, membership from a bitmap
      HG_LAUNCH("build_member_bits", k_member_bits, dim3(gB), dim3(kBT), 0, s, g->part, g->k,
                (const uint8_t*)w.sel, N, w.mbits);
      HG_LAUNCH("build_edge_keep", k_edge_keep, dim3(gE), dim3(kBT), 0, s, g->src, g->dst,
                (const uint32_t*)w.mbits, (const uint32_t*)w.bbits, g->edge_ts, g->t_cut, E, w.keep, w.first);
      // keep[E] = 0, so the scan's entry E is the number of kept edges
      HG_TRY(fill_i32(w.keep + E, 0, 1, s));
      HG_TRY(scan_exclusive_i32(w.keep, w.keep, E + 1, w.cnt + C_ESUB, w.scratch, s));
      HG_LAUNCH("build_edge_compact", k_edge_compact, dim3(gE), dim3(kBT), 0, s, g->src, g->dst,
                (const int32_t*)out->global2local, g->rel, (const int32_t*)w.keep, E, (int32_t)R, w.kcsr, w.vsrc,
                want_eid ? w.veid : nullptr, g->edge_w, emit_w ? w.vw : nullptr);
    }
  } else {
    HG_TRY(fill_i32(w.cnt + C_ESUB, 0, 1, s));
  }
  // overlap list (local ids ascending) with each node's home block and the
  // relation of its base edge
  HG_LAUNCH("build_overlap_flags", k_overlap_flags, dim3(gN), dim3(kBT), 0, s,
            (const int32_t*)out->local2global, (const uint8_t*)w.sel, (const int32_t*)w.cnt, N, w.flag);
  HG_TRY(scan_exclusive_i32(w.flag, w.pos, N, w.cnt + C_MSEL, w.scratch, s));
  if (o->budget_M > 0)
    HG_LAUNCH("build_overlap_fill", k_overlap_fill, dim3(gN), dim3(kBT), 0, s,
              (const int32_t*)out->local2global, (const int32_t*)w.flag, (const int32_t*)w.pos,
              (const int32_t*)w.cnt, g->part, (const int32_t*)w.first, g->rel, out->overlap,
              out->overlap_home, out->overlap_rel);
  // counts needed to size the sorts
  int32_t hc[C_COUNT];
  HG_HIP_TRY(hipMemcpyAsync(hc, w.cnt, sizeof(hc), hipMemcpyDeviceToHost, s));
  HG_HIP_TRY(hipStreamSynchronize(s));
  const int64_t NS = hc[C_NSUB], ES = hc[C_ESUB];
  const int64_t NQ = NS * R;
  // 7. CSR: stable sort by dst*R + r; CSC: stable sort of the CSR-ordered entries by src*R + r
  const int bits = bits_for(NQ);
  uint32_t* csr_keys = w.kcsr;  // the CSR's sorted keys, kept for the slots of its entries
  {
    uint32_t* ko;
    int32_t *v1o, *v2o;
    // second value: the edge id if asked for, else the weight of a weighted graph
    int32_t* v2 = want_eid ? w.veid : (weighted ? w.vw : nullptr);
    int32_t* v2_final = want_eid ? out->csr_eid : (weighted ? reinterpret_cast<int32_t*>(out->csr_w) : nullptr);
    uint32_t *sk = w.kcsr, *sk_alt = w.kalt;
    int32_t *s1 = w.vsrc, *s1_alt = w.alt1, *s2 = v2, *s2_alt = v2 ? w.alt2 : nullptr;
    if (rank_path && ES < E) {
      // some edges were dropped: compact the entries into the ping-pong buffers
      HG_LAUNCH("build_edge_compact", k_edge_emit, dim3((unsigned)ntiles), dim3(kBT), 0, s, (const uint32_t*)w.kcsr,
                (const int32_t*)w.vsrc, (const int32_t*)v2, (const uint64_t*)w.keep, E, (const int32_t*)w.tile_cnt,
                w.kalt, w.alt1, v2 ? w.alt2 : nullptr);
      std::swap(sk, sk_alt);
      std::swap(s1, s1_alt);
      std::swap(s2, s2_alt);
    }
    HG_TRY(radix_sort_pairs(sk, sk_alt, s1, s1_alt, s2, s2_alt, ES, bits, w.scratch, s, &ko, &v1o, &v2o,
                            out->csr_col, v2_final));
    csr_keys = ko;
    if (ES > 0 && v1o != out->csr_col) {  // no pass ran (a single key value)
      HG_HIP_TRY(hipMemcpyAsync(out->csr_col, v1o, sizeof(int32_t) * ES, hipMemcpyDeviceToDevice, s));
      if (v2)
        HG_HIP_TRY(hipMemcpyAsync(v2_final, v2o, sizeof(int32_t) * ES, hipMemcpyDeviceToDevice, s));
    }
    // both edge ids and weights asked for: the weights through the edge ids
    if (want_eid && weighted && ES > 0)
      HG_LAUNCH("build_csr_w", k_gather_w, dim3(grid_for(ES)), dim3(kBT), 0, s, (const int32_t*)out->csr_eid,
                g->edge_w, ES, out->csr_w);
    HG_TRY(fill_i32(w.rowcnt, 0, NQ + 1, s));
    if (ES > 0)
      HG_LAUNCH("build_row_count", k_row_count, dim3((unsigned)cdiv(ES, kRCChunk)), dim3(kBT), 0, s,
                (const uint32_t*)ko, ES, w.rowcnt);
    HG_TRY(scan_exclusive_i32(w.rowcnt, out->csr_ptr, NQ + 1, nullptr, w.scratch, s));
  }
  {
    // the CSC sort's input from the CSR in its order (the CSR keys stay
    // where the CSR sort left them, for the slots of its entries)
    uint32_t* ko;
    int32_t *v1o, *v2o;
    const bool packed = !weighted && NS < kPackedMaxNodes;
    if (ES > 0)
      HG_LAUNCH("build_csc_input", k_csc_input, dim3((unsigned)cdiv(ES, kBT * kCiItems)), dim3(kBT), 0, s,
                (const uint32_t*)csr_keys, (const int32_t*)out->csr_col, (const int32_t*)out->csr_ptr,
                weighted ? (const float*)out->csr_w : nullptr, ES, (int32_t)R, packed ? 1 : 0, w.kcsc, w.vdst,
                packed ? nullptr : w.vsc);
    int32_t* scale_bits = reinterpret_cast<int32_t*>(out->csc_scale);
    const SortUnpack up{out->csr_ptr, (int32_t)R, out->csc_scale};
    HG_TRY(radix_sort_pairs(w.kcsc, csr_keys == w.kalt ? w.kcsr : w.kalt, w.vdst, w.alt3, packed ? nullptr : w.vsc,
                            packed ? nullptr : w.vsc_alt, ES, bits, w.scratch, s, &ko, &v1o, &v2o, out->csc_row,
                            packed ? nullptr : scale_bits, packed ? &up : nullptr));
    if (ES > 0 && v1o != out->csc_row) {  // no pass ran (unpacked, a single key value)
      HG_HIP_TRY(hipMemcpyAsync(out->csc_row, v1o, sizeof(int32_t) * ES, hipMemcpyDeviceToDevice, s));
      HG_HIP_TRY(hipMemcpyAsync(scale_bits, v2o, sizeof(int32_t) * ES, hipMemcpyDeviceToDevice, s));
    }
    HG_TRY(fill_i32(w.rowcnt, 0, NQ + 1, s));
    if (ES > 0)
      HG_LAUNCH("build_row_count", k_row_count, dim3((unsigned)cdiv(ES, kRCChunk)), dim3(kBT), 0, s,
                (const uint32_t*)ko, ES, w.rowcnt);
    HG_TRY(scan_exclusive_i32(w.rowcnt, out->csc_ptr, NQ + 1, nullptr, w.scratch, s));
  }
  // 8. plan: active-source lists and backward work items
  PlanLayout pl(N, E, R);
  char* pb = static_cast<char*>(out->plan);
  int32_t* act = reinterpret_cast<int32_t*>(pb + pl.s_off);
  int32_t* act_off = reinterpret_cast<int32_t*>(pb + pl.soff_off);
  int4* items = reinterpret_cast<int4*>(pb + pl.items_off);
  int4* heavy = reinterpret_cast<int4*>(pb + pl.heavy_off);
  int32_t* act_slot = reinterpret_cast<int32_t*>(pb + pl.aslot_off);
  int32_t* slot_q = reinterpret_cast<int32_t*>(pb + pl.slotq_off);
  int32_t* csr_slot = reinterpret_cast<int32_t*>(pb + pl.cslot_off);
  SlotEnt* tab = reinterpret_cast<SlotEnt*>(pb + pl.tab_off);
  if (NQ > 0) {
    const int64_t nb = NQ / 64 + 1;  // w.rowcnt (NQ + 1 entries) is free: it holds the slot counts
    HG_TRY(fill_i32(w.rowcnt, 0, nb, s));
    HG_LAUNCH("build_active_digit", k_active_digit, dim3(grid_for(NQ)), dim3(kBT), 0, s,
              (const int32_t*)out->csc_ptr, NQ, (int32_t)R, w.digit, w.q_src, w.q_items, w.q_heavy,
              w.q_parts, tab, w.rowcnt);
    HG_TRY(scan_exclusive_i32(w.rowcnt, w.rowcnt, nb, w.cnt + C_ASLOTS, w.scratch, s));
    HG_LAUNCH("build_slot_pack", k_slot_pack, dim3(grid_for(nb)), dim3(kBT), 0, s, (const int32_t*)w.rowcnt, nb,
              NQ, (const int32_t*)(w.cnt + C_ASLOTS), tab);
    HG_TRY(bucket_partition(w.digit, w.q_src, NQ, (int)R, act, act_off, w.scratch, s));
    HG_TRY(scan_exclusive_i32(w.q_items, w.q_items, NQ, w.cnt + C_ITEMS, w.scratch, s));
    HG_TRY(scan_exclusive_i32(w.q_heavy, w.q_heavy, NQ, w.cnt + C_HEAVY, w.scratch, s));
    HG_TRY(scan_exclusive_i32(w.q_parts, w.q_parts, NQ, w.cnt + C_PARTS, w.scratch, s));
    HG_LAUNCH("build_plan_items", k_plan_items, dim3(grid_for(NQ)), dim3(kBT), 0, s,
              (const int32_t*)out->csc_ptr, NQ, (const int32_t*)w.q_items, (const int32_t*)w.q_heavy,
              (const int32_t*)w.q_parts, (const SlotEnt*)tab, (const int32_t*)(w.cnt + C_ASLOTS), items, heavy,
              slot_q);
    const int64_t cap_a = NQ < ES ? NQ : ES;
    if (cap_a > 0)
      HG_LAUNCH("build_act_slot", k_act_slot, dim3(grid_for(cap_a)), dim3(kBT), 0, s, (const int32_t*)act,
                (const int32_t*)act_off, (int32_t)R, cap_a, (const SlotEnt*)tab, act_slot);
    if (ES > 0)
      HG_LAUNCH("build_csr_slot", k_csr_slot, dim3(grid_for(ES)), dim3(kBT), 0, s, (const int32_t*)out->csr_col,
                (const uint32_t*)csr_keys, ES, (int32_t)R, NQ, (const int32_t*)(w.cnt + C_ASLOTS),
                (const SlotEnt*)tab, csr_slot);
    // long destination rows and their chunks (w.q_items, w.q_heavy are free again)
    int4* fitems = reinterpret_cast<int4*>(pb + pl.fitems_off);
    int4* fheavy = reinterpret_cast<int4*>(pb + pl.fheavy_off);
    HG_LAUNCH("build_fwd_counts", k_fwd_counts, dim3(grid_for(NS)), dim3(kBT), 0, s, (const int32_t*)out->csr_ptr,
              NS, (int32_t)R, w.q_heavy, w.q_items);
    HG_TRY(scan_exclusive_i32(w.q_heavy, w.q_heavy, NS, w.cnt + C_FHEAVY, w.scratch, s));
    HG_TRY(scan_exclusive_i32(w.q_items, w.q_items, NS, w.cnt + C_FPARTS, w.scratch, s));
    HG_LAUNCH("build_fwd_items", k_fwd_items, dim3(grid_for(NS)), dim3(kBT), 0, s, (const int32_t*)out->csr_ptr, NS,
              (int32_t)R, (const int32_t*)w.q_heavy, (const int32_t*)w.q_items, fitems, fheavy);
  } else {
    HG_TRY(fill_i32(act_off, 0, R + 1, s));
    HG_TRY(fill_i32(w.cnt + C_ITEMS, 0, 3, s));
    HG_TRY(fill_i32(w.cnt + C_FHEAVY, 0, 3, s));
  }
  // final sync: host counts
  std::vector<int32_t> tof(T + 1), aof(R + 1);
  HG_HIP_TRY(hipMemcpyAsync(hc, w.cnt, sizeof(hc), hipMemcpyDeviceToHost, s));
  HG_HIP_TRY(hipMemcpyAsync(tof.data(), out->type_off, sizeof(int32_t) * (T + 1), hipMemcpyDeviceToHost, s));
  HG_HIP_TRY(hipMemcpyAsync(aof.data(), act_off, sizeof(int32_t) * (R + 1), hipMemcpyDeviceToHost, s));
  HG_HIP_TRY(hipStreamSynchronize(s));
  out->n_nodes = N;
  out->n_edges = E;
  out->n_sub = NS;
  out->e_sub = ES;
  out->m_sel = hc[C_MSEL];
  out->n_rel = (int32_t)R;
  out->n_ntype = (int32_t)T;
  for (int t = 0; t <= HG_MAX_NTYPE; ++t) out->type_off_host[t] = t <= T ? tof[t] : 0;
  for (int r = 0; r < HG_MAX_REL; ++r) out->n_active[r] = r < R ? (int64_t)aof[r + 1] - aof[r] : 0;
  out->plan_items = hc[C_ITEMS];
  out->plan_heavy = hc[C_HEAVY];
  out->plan_partials = hc[C_PARTS];
  out->plan_fwd_heavy = hc[C_FHEAVY];
  out->plan_fwd_parts = hc[C_FPARTS];
  out->plan_slot_rows = row_layout(NQ, hc[C_ASLOTS]) ? NQ : hc[C_ASLOTS];
  out->weighted = weighted ? 1 : 0;
  return HG_OK;
}
