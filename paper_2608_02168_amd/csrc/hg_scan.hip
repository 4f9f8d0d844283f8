// Device-wide primitives: exclusive scan, stable LSD radix sort, stable
// bucket partition and fills.  All of them are deterministic: counts use
// integer atomics only where the result does not depend on their order.
#include "hg_internal.h"

namespace hg {

namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;  // 4096
constexpr int kWaves = kThreads / kWave;

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }

// Inclusive wave scan of one int per lane.
__device__ __forceinline__ int wave_incl_scan(int v) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    int t = __shfl_up(v, o, kWave);
    if (l >= o) v += t;
  }
  return v;
}

// Exclusive block scan of one int per thread (a block of kT threads); returns
// the block total in *total.
template <int kT = kThreads>
__device__ __forceinline__ int block_excl_scan(int v, int* total) {
  constexpr int kW = kT / kWave;
  __shared__ int wsum[kW];
  const int w = threadIdx.x / kWave;
  int inc = wave_incl_scan(v);
  if (lane_id() == kWave - 1) wsum[w] = inc;
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int i = 0; i < kW; ++i) {
    int x = wsum[i];
    off += (i < w) ? x : 0;
    tot += x;
  }
  __syncthreads();
  *total = tot;
  return off + inc - v;
}

__global__ void k_tile_sums(const int32_t* __restrict__ in, int64_t n, int32_t* __restrict__ sums) {
  const int64_t base = (int64_t)blockIdx.x * kTile;
  int s = 0;
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    int64_t i = base + (int64_t)j * kThreads + threadIdx.x;
    s += (i < n) ? in[i] : 0;
  }
  int tot;
  (void)block_excl_scan(s, &tot);
  if (threadIdx.x == 0) sums[blockIdx.x] = tot;
}

// Single block: exclusive scan of sums[0..m) in place, carrying across chunks.
__global__ void k_scan_sums(int32_t* __restrict__ sums, int64_t m, int32_t* __restrict__ total) {
  int carry = 0;
  for (int64_t base = 0; base < m; base += kThreads) {
    int64_t i = base + threadIdx.x;
    int v = (i < m) ? sums[i] : 0;
    int tot;
    int ex = block_excl_scan(v, &tot);
    if (i < m) sums[i] = carry + ex;
    carry += tot;
  }
  if (threadIdx.x == 0 && total) *total = carry;
}

// Per tile: 16 rounds of 256 consecutive items (coalesced loads and stores),
// each an exclusive block scan carried over from the previous round.
__global__ void k_scan_tiles(const int32_t* __restrict__ in, int32_t* __restrict__ out, int64_t n,
                             const int32_t* __restrict__ tile_off) {
  const int64_t base = (int64_t)blockIdx.x * kTile;
  int carry = tile_off[blockIdx.x];
  int v[kItems];
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + (int64_t)j * kThreads + threadIdx.x;
    v[j] = (i < n) ? in[i] : 0;
  }
#pragma unroll
  for (int j = 0; j < kItems; ++j) {
    const int64_t i = base + (int64_t)j * kThreads + threadIdx.x;
    int tot;
    const int ex = block_excl_scan(v[j], &tot);
    if (i < n) out[i] = carry + ex;
    carry += tot;
  }
}

// ---- radix sort -------------------------------------------------------------
// Tiles of 8192 items: a run of an 8-bit digit inside a tile then averages
// 32 items (128 bytes of keys), of a 9-bit digit 16; runs that continue in
// the next tile are completed in the same L2 (see xcd_tile).
constexpr int kRItems = 32;
constexpr int kRTile = kThreads * kRItems;
// Key sorts take 512 threads per scatter block (16 items each): with one
// value per key two blocks fit a compute unit's LDS, 16 waves in flight.
constexpr int kKeyThreads = 512;

// Tile of a block: blocks go round-robin over the 8 XCDs, so block b runs on
// XCD b mod 8; XCD x takes the x-th eighth of the tiles in order.  The
// histogram pass writes digit d of tile t next to that of tile t + 1, and in
// the scatter pass a digit's run of tile t continues in tile t + 1, so
// consecutive tiles on one XCD complete each other's partly written lines in
// that XCD's L2 before they are written back (tiles on different XCDs leave
// two partial lines).
__device__ __forceinline__ int64_t xcd_tile(int64_t b, int64_t ntiles) {
  const int64_t q = ntiles >> 3, r = ntiles & 7, x = b & 7, i = b >> 3;
  return x * q + (x < r ? x : r) + i;
}

// Digit histogram of one tile of kTN items: hist[d * ntiles + tile].  Keys
// of a whole tile are read as 16-byte vectors (4 consecutive keys per thread
// and load).  Sorted runs of one key (a hub's entries once the lower digits
// are sorted) would send all 64 lanes of an LDS atomic to one counter, which
// serialises it: a wave whose 256 keys of a load all carry the wave's first
// digit adds them with one atomic, and a thread adds equal neighbours among
// its 4 keys together.
template <bool kDigitArray, int kTN = kRTile, int kBins = 256>
__global__ void k_radix_upsweep(const uint32_t* __restrict__ keys, const uint8_t* __restrict__ digits,
                                int64_t n, int shift, uint32_t dmask, int32_t* __restrict__ hist,
                                int64_t ntiles) {
  static_assert(kBins % kThreads == 0, "bins in whole rounds of the block");
  __shared__ int cnt[kBins];
#pragma unroll
  for (int q = 0; q < kBins; q += kThreads) cnt[q + threadIdx.x] = 0;
  __syncthreads();
  const int64_t tile = xcd_tile(blockIdx.x, ntiles);
  const int64_t base = tile * kTN;
  const bool vec = !kDigitArray && base + kTN <= n && (reinterpret_cast<uintptr_t>(keys) & 15u) == 0;
  if (vec) {
    constexpr int kV = kTN / (4 * kThreads);
    const uint4* kp = reinterpret_cast<const uint4*>(keys + base);
    uint4 v[kV];
#pragma unroll
    for (int j = 0; j < kV; ++j) v[j] = kp[j * kThreads + threadIdx.x];
#pragma unroll
    for (int j = 0; j < kV; ++j) {
      const uint32_t d0 = (v[j].x >> shift) & dmask, d1 = (v[j].y >> shift) & dmask;
      const uint32_t d2 = (v[j].z >> shift) & dmask, d3 = (v[j].w >> shift) & dmask;
      const uint32_t lead = (uint32_t)__builtin_amdgcn_readfirstlane((int)d0);
      if (__ballot(d0 == lead && d1 == lead && d2 == lead && d3 == lead) == ~0ull) {
        if ((threadIdx.x & (kWave - 1)) == 0) atomicAdd(&cnt[lead], 4 * kWave);
      } else {
        uint32_t pd = d0;
        int pc = 1;
        const uint32_t dn[3] = {d1, d2, d3};
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          if (dn[q] == pd) {
            ++pc;
          } else {
            atomicAdd(&cnt[pd], pc);
            pd = dn[q];
            pc = 1;
          }
        }
        atomicAdd(&cnt[pd], pc);
      }
    }
  } else {
#pragma unroll 4
    for (int j = 0; j < kTN / kThreads; ++j) {
      int64_t i = base + (int64_t)j * kThreads + threadIdx.x;
      if (i < n) {
        uint32_t d = kDigitArray ? (uint32_t)digits[i] : ((keys[i] >> shift) & dmask);
        if (!kDigitArray || d != 255u) atomicAdd(&cnt[d], 1);
      }
    }
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < kBins; q += kThreads) hist[(int64_t)(q + threadIdx.x) * ntiles + tile] = cnt[q + threadIdx.x];
}

// Stable scatter of one tile, staged through LDS.  Wave w owns the 2048
// consecutive items [2048 w, 2048 w + 2048) of the tile and visits them in 32
// rounds of 64 (lane order), so the tile order is (wave, round, lane).  An
// item's rank among equal digits inside its wave comes from wave-private LDS
// counters (no block barrier per round); one barrier later the per-digit
// offsets of the waves are known, each item is written to its slot of an LDS
// copy of the tile sorted by digit, and that copy is written out in slot
// order, so every digit's run lands in consecutive global addresses.
// offs is the digit-major exclusive scan of the per-tile counts with the
// grand total at offs[256 * ntiles].
// kUnpack: the CSC sort's last pass (SortUnpack): v1 packs the destination
// and its row's in-degree; v1_out gets the destination, scale_out 1 / deg.
// kT threads per block (a multiple of 256), tiles of kTN items, kTN / kT
// items per thread.
template <bool kDigitArray, bool kHasV2, bool kUnpack = false, int kT = kThreads, int kTN = kRTile, int kBins = 256>
__global__ void __launch_bounds__(kT) k_radix_downsweep(
    const uint32_t* __restrict__ keys, const uint8_t* __restrict__ digits,
    const int32_t* __restrict__ v1, const int32_t* __restrict__ v2, int64_t n, int shift, uint32_t dmask,
    const int32_t* __restrict__ offs, int64_t ntiles, uint32_t* __restrict__ keys_out,
    int32_t* __restrict__ v1_out, int32_t* __restrict__ v2_out, SortUnpack up = SortUnpack{nullptr, 1, nullptr}) {
  constexpr int kW = kT / kWave, kI = kTN / kT;
  constexpr int kBits = kBins == 512 ? 9 : 8;
  static_assert(kBins == 256 || (kBins == 512 && !kDigitArray), "8- or 9-bit key digits");
  static_assert(kT >= kBins, "one thread per digit");
  __shared__ int gbase[kBins];
  __shared__ int loff[kBins];
  __shared__ uint16_t wcnt[kW][kBins];  // counts, then offsets, below kTN
  __shared__ uint32_t sk[kDigitArray ? 1 : kTN];
  __shared__ int32_t sv1[kTN];
  __shared__ int32_t sv2[kHasV2 ? kTN : 1];
  __shared__ uint8_t sd[kDigitArray ? kTN : 1];  // a key's digit is read off sk
  const int t = threadIdx.x;
  const int w = t / kWave;
  const int l = lane_id();
  const int64_t tile = xcd_tile(blockIdx.x, ntiles);
  int cnt = 0;
  if (t < kBins) {
    const int64_t fi = (int64_t)t * ntiles + tile;
    const int base = offs[fi];
    cnt = offs[fi + 1] - base;
    gbase[t] = base;
  }
  for (int q = t; q < kW * kBins; q += kT) (&wcnt[0][0])[q] = 0;
  const uint64_t lt_mask = (l == 0) ? 0ull : (~0ull >> (kWave - l));
  const int64_t wbase = tile * kTN + (int64_t)w * (kI * kWave);
  // all loads of the wave's slice first
  uint32_t kd[kI];  // key, or digit
  int32_t a1[kI], a2[kHasV2 ? kI : 1];
#pragma unroll
  for (int j = 0; j < kI; ++j) {
    const int64_t i = wbase + (int64_t)j * kWave + l;
    if (i < n) {
      kd[j] = kDigitArray ? (uint32_t)digits[i] : keys[i];
      a1[j] = v1[i];
      if (kHasV2) a2[j] = v2[i];
    } else {
      kd[j] = kDigitArray ? 255u : 0u;
      a1[j] = 0;
      if (kHasV2) a2[j] = 0;
    }
  }
  int lo = 0, kept = 0;
  lo = block_excl_scan<kT>(cnt, &kept);  // includes a barrier: wcnt zeroing is visible after it
  if (t < kBins) loff[t] = lo;
  // ranks inside the wave
  uint16_t rk[kI];
#pragma unroll
  for (int j = 0; j < kI; ++j) {
    const int64_t i = wbase + (int64_t)j * kWave + l;
    const uint32_t d = kDigitArray ? kd[j] : ((kd[j] >> shift) & dmask);
    const bool valid = i < n && (!kDigitArray || d != 255u);
    uint64_t m = __ballot(valid);
#pragma unroll
    for (int b = 0; b < kBits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bal = __ballot(bit);
      m &= bit ? bal : ~bal;
    }
    int r = 0;
    if (valid) r = wcnt[w][d] + __popcll(m & lt_mask);
    // every lane has read the counter before the group's leader advances it
    __builtin_amdgcn_wave_barrier();
    if (valid && (m & lt_mask) == 0) wcnt[w][d] = (uint16_t)(wcnt[w][d] + __popcll(m));
    __builtin_amdgcn_wave_barrier();
    rk[j] = valid ? (uint16_t)r : (uint16_t)0xFFFFu;
  }
  __syncthreads();
  // per digit: exclusive prefix over the waves, added to the tile-local offset
  if (t < kBins) {
    int run = loff[t];
#pragma unroll
    for (int q = 0; q < kW; ++q) {
      const int c = wcnt[q][t];
      wcnt[q][t] = (uint16_t)run;
      run += c;
    }
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < kI; ++j) {
    if (rk[j] != 0xFFFFu) {
      const uint32_t d = kDigitArray ? kd[j] : ((kd[j] >> shift) & dmask);
      const int lpos = wcnt[w][d] + rk[j];
      if (!kDigitArray) sk[lpos] = kd[j];
      sv1[lpos] = a1[j];
      if (kHasV2) sv2[lpos] = a2[j];
      if (kDigitArray) sd[lpos] = (uint8_t)d;
    }
  }
  __syncthreads();
  for (int idx = t; idx < kept; idx += kT) {
    const int d = kDigitArray ? (int)sd[idx] : (int)((sk[idx] >> shift) & dmask);
    const int pos = gbase[d] + (idx - loff[d]);
    if (!kDigitArray) keys_out[pos] = sk[idx];
    if (kUnpack) {
      const uint32_t v = (uint32_t)sv1[idx];
      const int32_t dst = (int32_t)(v & 0xFFFFFFu);
      int32_t deg = (int32_t)(v >> 24);
      if (deg == 255) {
        const int64_t row = (int64_t)dst * up.n_rel + (int64_t)(sk[idx] % (uint32_t)up.n_rel);
        deg = up.csr_ptr[row + 1] - up.csr_ptr[row];
      }
      v1_out[pos] = dst;
      up.scale[pos] = 1.0f / (float)deg;
    } else {
      v1_out[pos] = sv1[idx];
    }
    if (kHasV2) v2_out[pos] = sv2[idx];
  }
}

__global__ void k_bin_offsets(const int32_t* __restrict__ offs, int64_t ntiles, int nbins,
                              const int32_t* __restrict__ total, int32_t* __restrict__ bin_off) {
  int b = threadIdx.x;
  if (b < nbins) bin_off[b] = offs[(int64_t)b * ntiles];
  if (b == nbins) bin_off[b] = *total;
}

template <class T>
__global__ void k_fill(T* __restrict__ p, T v, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (; i < n; i += stride) p[i] = v;
}

template <class T>
int fill_impl(T* p, T v, int64_t n, hipStream_t s) {
  if (n <= 0) return HG_OK;
  int64_t blocks = cdiv(n, 256);
  if (blocks > 65536) blocks = 65536;
  HG_LAUNCH("fill", (k_fill<T>), dim3((unsigned)blocks), dim3(256), 0, s, p, v, n);
  return HG_OK;
}

}  // namespace

int64_t scan_scratch_elems(int64_t n) { return cdiv(n > 0 ? n : 1, kTile) + 64; }

int scan_exclusive_i32(const int32_t* in, int32_t* out, int64_t n, int32_t* total_dev,
                       int32_t* scratch, hipStream_t s) {
  if (n <= 0) {
    if (total_dev) HG_TRY(fill_i32(total_dev, 0, 1, s));
    return HG_OK;
  }
  const int64_t tiles = cdiv(n, kTile);
  HG_LAUNCH("scan_tile_sums", k_tile_sums, dim3((unsigned)tiles), dim3(kThreads), 0, s, in, n, scratch);
  HG_LAUNCH("scan_sums", k_scan_sums, dim3(1), dim3(kThreads), 0, s, scratch, tiles, total_dev);
  HG_LAUNCH("scan_tiles", k_scan_tiles, dim3((unsigned)tiles), dim3(kThreads), 0, s, in, out, n,
            (const int32_t*)scratch);
  return HG_OK;
}

int64_t radix_scratch_elems(int64_t n) {
  const int64_t tiles = cdiv(n > 0 ? n : 1, kRTile);
  const int64_t h = 512 * tiles;
  return h + 1 + scan_scratch_elems(h) + 64;
}

namespace {

// One LSD pass over the digit of nb (<= 9) bits at shift: tile histograms,
// their digit-major scan, the stable scatter.
template <int kBins>
int radix_pass(const uint32_t* ka, uint32_t* kb, const int32_t* a1, int32_t* b1, const int32_t* a2, int32_t* b2,
               int64_t n, int shift, uint32_t dmask, int32_t* scratch, hipStream_t s, const SortUnpack* unpack) {
  const int64_t tiles = cdiv(n, kRTile);
  int32_t* hist = scratch;
  int32_t* sscr = scratch + kBins * tiles + 1;
  HG_LAUNCH("radix_upsweep", (k_radix_upsweep<false, kRTile, kBins>), dim3((unsigned)tiles), dim3(kThreads), 0, s,
            ka, (const uint8_t*)nullptr, n, shift, dmask, hist, tiles);
  HG_TRY(scan_exclusive_i32(hist, hist, kBins * tiles, hist + kBins * tiles, sscr, s));
  if (unpack) {
    HG_LAUNCH("radix_downsweep", (k_radix_downsweep<false, false, true, kKeyThreads, kRTile, kBins>),
              dim3((unsigned)tiles), dim3(kKeyThreads), 0, s, ka, (const uint8_t*)nullptr, a1,
              (const int32_t*)nullptr, n, shift, dmask, (const int32_t*)hist, tiles, kb, b1, (int32_t*)nullptr,
              *unpack);
  } else if (a2) {
    HG_LAUNCH("radix_downsweep", (k_radix_downsweep<false, true, false, kKeyThreads, kRTile, kBins>),
              dim3((unsigned)tiles), dim3(kKeyThreads), 0, s, ka, (const uint8_t*)nullptr, a1, a2, n, shift, dmask,
              (const int32_t*)hist, tiles, kb, b1, b2);
  } else {
    HG_LAUNCH("radix_downsweep", (k_radix_downsweep<false, false, false, kKeyThreads, kRTile, kBins>),
              dim3((unsigned)tiles), dim3(kKeyThreads), 0, s, ka, (const uint8_t*)nullptr, a1,
              (const int32_t*)nullptr, n, shift, dmask, (const int32_t*)hist, tiles, kb, b1, (int32_t*)nullptr);
  }
  return HG_OK;
}

}  // namespace

int radix_sort_pairs(uint32_t* keys, uint32_t* keys_alt, int32_t* v1, int32_t* v1_alt,
                     int32_t* v2, int32_t* v2_alt, int64_t n, int bits, int32_t* scratch,
                     hipStream_t s, uint32_t** keys_out, int32_t** v1_out, int32_t** v2_out,
                     int32_t* v1_final, int32_t* v2_final, const SortUnpack* unpack) {
  *keys_out = keys;
  *v1_out = v1;
  if (v2_out) *v2_out = v2;
  if (unpack) {
    if (v2 || !v1_final) return fail(HG_ERR_ARG, "radix_sort_pairs: unpack needs v1_final and no v2");
    if (bits < 1) bits = 1;  // a single key value still takes the unpacking pass
  }
  if (n <= 0 || bits <= 0) return HG_OK;
  // Digits of 8 or 9 bits, as few passes as 9-bit digits allow: P passes
  // take P * 8 bits with 8-bit digits and the first bits - 8 P of them one
  // bit more (26 bits: 9, 9, 8 in three passes instead of four).
  const int passes = (bits + 8) / 9;
  const int wide = bits > 8 * passes ? bits - 8 * passes : 0;
  uint32_t *ka = keys, *kb = keys_alt;
  int32_t *a1 = v1, *b1 = v1_alt, *a2 = v2, *b2 = v2_alt;
  int shift = 0;
  for (int p = 0; p < passes; ++p) {
    const int nb = p < wide ? 9 : (bits - shift < 8 ? bits - shift : 8);
    const uint32_t dmask = (1u << nb) - 1u;
    const bool last = p == passes - 1;
    // the last pass writes the values straight into their final arrays
    if (last) {
      if (v1_final) b1 = v1_final;
      if (v2_final && v2) b2 = v2_final;
    }
    const SortUnpack* up = (unpack && last) ? unpack : nullptr;
    if (nb > 8) {
      HG_TRY(radix_pass<512>(ka, kb, a1, b1, a2, b2, n, shift, dmask, scratch, s, up));
    } else {
      HG_TRY(radix_pass<256>(ka, kb, a1, b1, a2, b2, n, shift, dmask, scratch, s, up));
    }
    shift += nb;
    uint32_t* tk = ka; ka = kb; kb = tk;
    int32_t* t1 = a1; a1 = b1; b1 = t1;
    int32_t* t2 = a2; a2 = b2; b2 = t2;
  }
  *keys_out = ka;
  *v1_out = a1;
  if (v2_out) *v2_out = a2;
  return HG_OK;
}

int bucket_partition(const uint8_t* digit, const int32_t* val, int64_t n, int nbins, int32_t* out,
                     int32_t* bin_off, int32_t* scratch, hipStream_t s) {
  if (nbins < 1 || nbins > 255) return fail(HG_ERR_ARG, "bucket_partition: nbins %d", nbins);
  if (n <= 0) return fill_i32(bin_off, 0, nbins + 1, s);
  const int64_t tiles = cdiv(n, kRTile);
  int32_t* hist = scratch;
  int32_t* sscr = scratch + 256 * tiles + 1;
  int32_t* total = hist + 256 * tiles;
  HG_LAUNCH("partition_upsweep", (k_radix_upsweep<true>), dim3((unsigned)tiles), dim3(kThreads), 0, s,
            (const uint32_t*)nullptr, digit, n, 0, 0xFFu, hist, tiles);
  HG_TRY(scan_exclusive_i32(hist, hist, 256 * tiles, total, sscr, s));
  HG_LAUNCH("partition_downsweep", (k_radix_downsweep<true, false>), dim3((unsigned)tiles),
            dim3(kThreads), 0, s, (const uint32_t*)nullptr, digit, val, (const int32_t*)nullptr, n,
            0, 0xFFu, (const int32_t*)hist, tiles, (uint32_t*)nullptr, out, (int32_t*)nullptr);
  HG_LAUNCH("partition_offsets", k_bin_offsets, dim3(1), dim3(256), 0, s, (const int32_t*)hist,
            tiles, nbins, (const int32_t*)total, bin_off);
  return HG_OK;
}

int fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s) { return fill_impl(p, v, n, s); }
int fill_u8(uint8_t* p, uint8_t v, int64_t n, hipStream_t s) { return fill_impl(p, v, n, s); }
int fill_f32(float* p, float v, int64_t n, hipStream_t s) { return fill_impl(p, v, n, s); }

}  // namespace hg
