// Memory-system ceiling for the random-row gather pattern of the sparse
// products: rows of a float32 table fetched through uniformly random row ids,
// summed in groups of G consecutive ids, with or without one output row
// written per group.  This is a hardware characterisation used by the
// benchmark to place the SpMM kernels against what the memory system delivers
// for this access pattern; it is a separate library (libhg_ceiling.so) and not
// part of libhg.so.
#include <hip/hip_runtime.h>

#include <cstdint>

namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

// splitmix64 finaliser over (seed + i * golden gamma): uniform ids in [0, n_rows)
__global__ void k_random_rows(int32_t* __restrict__ idx, int64_t n, int64_t n_rows, uint64_t seed) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    uint64_t z = seed + (uint64_t)(i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    idx[i] = (int32_t)(z % (uint64_t)n_rows);
  }
}

// One wave per group; LPR lanes hold one row (a float4 each), so a load
// instruction fetches 64 / LPR rows; U instructions are in flight per wave.
template <int D>
__global__ void __launch_bounds__(256) k_gather(const float* __restrict__ table, const int32_t* __restrict__ idx,
                                                int64_t n_groups, int group, float* __restrict__ out, int write) {
  constexpr int LPR = D / 4, EPW = 64 / LPR, U = 4;
  const int l = threadIdx.x & 63, slot = l / LPR, c0 = (l % LPR) * 4;
  const int64_t w0 = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  const int64_t nw = ((int64_t)gridDim.x * blockDim.x) >> 6;
  for (int64_t gi = w0; gi < n_groups; gi += nw) {
    const int32_t my = idx[gi * group + (l < group ? l : group - 1)];
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    for (int e = 0; e < group; e += EPW * U) {
      f32x4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int me = e + u * EPW + slot;
        const int32_t q = __shfl(my, me & 63, 64);
        if (me < group) {
          v[u] = *reinterpret_cast<const f32x4*>(table + (int64_t)q * D + c0);
        } else {
          v[u] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) acc += v[u];
    }
#pragma unroll
    for (int o = LPR; o < 64; o <<= 1) {
#pragma unroll
      for (int k = 0; k < 4; ++k) acc[k] += __shfl_xor(acc[k], o, 64);
    }
    // without writes, the sum is stored only if it is not finite (never, for
    // a finite table), which keeps the loads from being optimised away
    const bool store = write ? true : !(acc[0] - acc[0] == 0.f);
    if (slot == 0 && store) *reinterpret_cast<f32x4*>(out + (write ? gi : 0) * D + c0) = acc;
  }
}

}  // namespace

extern "C" {

// idx[0..n) = uniform random row ids in [0, n_rows).  Returns 0, or -1 on bad
// arguments, -4 on a HIP error.
int hgc_random_rows(int32_t* idx, int64_t n, int64_t n_rows, uint64_t seed, hipStream_t s) {
  if (!idx || n < 0 || n_rows <= 0 || n_rows > INT32_MAX) return -1;
  if (n == 0) return 0;
  hipLaunchKernelGGL(k_random_rows, dim3(4096), dim3(256), 0, s, idx, n, n_rows, seed);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// For g in [0, n_idx / group): sum of table rows idx[g*group .. g*group+group),
// written to out row g when write != 0 (out holds n_idx / group rows of d
// floats); when write == 0 out needs one row and is written only for a
// non-finite sum.  idx values must lie in [0, n_rows) (the caller's contract:
// hgc_random_rows produces such ids).  d in {64, 128, 256}, 1 <= group <= 64.
// Returns 0, -1 on bad arguments, -5 for an unsupported d, -4 on a HIP error.
int hgc_gather(const float* table, int64_t n_rows, int32_t d, const int32_t* idx, int64_t n_idx, int32_t group,
               float* out, int32_t write, hipStream_t s) {
  if (!table || !idx || !out || n_rows <= 0 || n_idx < 0 || group < 1 || group > 64) return -1;
  const int64_t n_groups = n_idx / group;
  if (n_groups == 0) return 0;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -4;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return -4;
  int64_t blocks = (n_groups + 3) / 4;
  if (blocks > (int64_t)cus * 8) blocks = (int64_t)cus * 8;
  switch (d) {
    case 64:
      hipLaunchKernelGGL(k_gather<64>, dim3((unsigned)blocks), dim3(256), 0, s, table, idx, n_groups, group, out, write);
      break;
    case 128:
      hipLaunchKernelGGL(k_gather<128>, dim3((unsigned)blocks), dim3(256), 0, s, table, idx, n_groups, group, out, write);
      break;
    case 256:
      hipLaunchKernelGGL(k_gather<256>, dim3((unsigned)blocks), dim3(256), 0, s, table, idx, n_groups, group, out, write);
      break;
    default:
      return -5;
  }
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
