// Internal declarations shared by the libhg.so translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>

#include "../../include/hg.h"

namespace hg {

constexpr int kWave = 64;

// ---- host-side error reporting -----------------------------------------
void set_detail(const char* fmt, ...);
int fail(int code, const char* fmt, ...);

#define HG_HIP_TRY(expr)                                                     \
  do {                                                                       \
    hipError_t e_ = (expr);                                                  \
    if (e_ != hipSuccess)                                                    \
      return ::hg::fail(HG_ERR_HIP, "%s failed: %s (%s:%d)", #expr,          \
                        hipGetErrorString(e_), __FILE__, __LINE__);          \
  } while (0)

#define HG_TRY(expr)              \
  do {                            \
    int s_ = (expr);              \
    if (s_ != HG_OK) return s_;   \
  } while (0)

// ---- kernel timing log ----------------------------------------------------
bool timing_on();
void timing_begin(const char* name, hipStream_t s, void** tok);
void timing_end(void* tok, hipStream_t s);

// Launch a kernel, optionally bracketed by timing events; returns HG status.
#define HG_LAUNCH(name, kernel, grid, block, shmem, stream, ...)             \
  do {                                                                       \
    void* tok_ = nullptr;                                                    \
    if (::hg::timing_on()) ::hg::timing_begin(name, stream, &tok_);          \
    hipLaunchKernelGGL(kernel, grid, block, shmem, stream, __VA_ARGS__);     \
    if (tok_) ::hg::timing_end(tok_, stream);                                \
    hipError_t le_ = hipGetLastError();                                      \
    if (le_ != hipSuccess)                                                   \
      return ::hg::fail(HG_ERR_HIP, "launch of %s failed: %s", name,        \
                        hipGetErrorString(le_));                             \
  } while (0)

inline int64_t cdiv(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

// Bump allocator over a caller-provided workspace.
struct Arena {
  char* base;
  size_t cap;
  size_t used = 0;
  Arena(void* p, size_t c) : base(static_cast<char*>(p)), cap(c) {}
  template <class T>
  T* take(int64_t n) {
    size_t off = align_up(used);
    used = off + align_up(sizeof(T) * (size_t)(n > 0 ? n : 0));
    return (used <= cap && base) ? reinterpret_cast<T*>(base + off) : nullptr;
  }
  bool ok() const { return used <= cap; }
};

// Sizing pass: same sequence of takes without memory.
struct Sizer {
  size_t used = 0;
  template <class T>
  T* take(int64_t n) {
    used = align_up(used) + align_up(sizeof(T) * (size_t)(n > 0 ? n : 0));
    return nullptr;
  }
};

int num_cus();

// Slots of the relation transforms.  The active (source, relation) pairs --
// the CSC rows q = i * R + r that hold at least one entry -- are numbered
// 0 .. A-1 in q order, so the transforms Y_r[slot] take A rows instead of
// n_sub * R, and the active relations of one source have consecutive slots.
// slot(q) = the number of active rows before q, from one 16-byte entry per
// 64 rows: the active-row mask of the 64 and the count before them.
//
// When the row-indexed layout (slot = q, n_sub * R rows) costs at most
// kRowLayoutMaxSpread times the compact one, the build keeps it instead: the
// gathers and row writes of the SpMMs run 5-7% faster over rows spread at
// the pitch of R rows per node than over packed rows (measured at R = 5,
// 3.6x spread), and the memory is there.  The plan then has no slot arrays
// (PlanView's csr_slot, slot_q and slot_tab are null) and the kernels index
// the transforms by q.
constexpr int64_t kRowLayoutMaxSpread = 4;
struct alignas(16) SlotEnt {
  uint64_t mask;
  int32_t pre;
  int32_t pad;
};

__device__ __forceinline__ int32_t slot_of(const SlotEnt* __restrict__ tab, int64_t q) {
  const int4 e = *reinterpret_cast<const int4*>(tab + (q >> 6));
  const uint64_t m = ((uint64_t)(uint32_t)e.y << 32) | (uint32_t)e.x;
  return e.z + (int32_t)__popcll(m & ((1ull << (q & 63)) - 1ull));
}

// Execution plan written by hg_build_csr (laid out for the input capacities).
struct PlanView {
  const int32_t* active;    // concatenated S_r lists: sources with >= 1 out-edge of relation r, ascending
  const int32_t* act_slot;  // slot of each entry of `active` (same order)
  const int32_t* slot_q;    // [A]: the CSC row q = i * R + r of each slot (null: row-indexed, slot = q)
  const int32_t* csr_slot;  // [e_sub]: slot of the (source, relation) of each CSR entry (null: row-indexed)
  const SlotEnt* slot_tab;  // [n_sub * R / 64 + 1] (null: row-indexed)
  const int4* items;        // backward work items (slot, begin, end, partial slot or -1)
  const int4* heavy;        // split rows (slot, first partial slot, number of slots, 0)
  const int4* fwd_items;    // chunks of long destination rows (j, begin, end, partial slot)
  const int4* fwd_heavy;    // long destination rows (j, first partial slot, number of slots, 0)
};

// Destination rows (all relations of one node j in the CSR) longer than
// this are not walked by one wave: the plan cuts them into chunks of this
// many entries whose partial results are merged in chunk order.
constexpr int32_t kFwdChunk = 2048;
PlanView plan_view(const hg_subgraph* s);

// Rows of the relation transforms: A (compact) or n_sub * R (row-indexed).
inline int64_t n_slots(const hg_subgraph* s) { return s->plan_slot_rows; }

// ---- primitives (hg_scan.hip) -------------------------------------------
// Exclusive prefix sum of n int32 values into out (out may equal in).
// Writes the total into *total_dev (device int32) if non-null.  Scratch:
// scan_scratch_elems(n) int32.
int64_t scan_scratch_elems(int64_t n);
int scan_exclusive_i32(const int32_t* in, int32_t* out, int64_t n, int32_t* total_dev,
                       int32_t* scratch, hipStream_t s);

// Last pass of the CSC sort: its value packs a destination (low 24 bits)
// and the in-degree of the destination's row (high 8 bits, 255 = "255 or
// more": read from csr_ptr); the pass writes the destination to v1_final and
// the mean weight 1 / deg, a correctly rounded float32 quotient, to scale.
// The row of an entry is destination * n_rel + key % n_rel.
struct SortUnpack {
  const int32_t* csr_ptr;
  int32_t n_rel;
  float* scale;
};

// Stable LSD radix sort of (key, value[, value2]) by the low `bits` bits of
// key (uint32).  Ping-pong buffers must hold n elements; the result ends in
// the *_out buffers.  v1_final / v2_final (may be NULL; n elements, distinct
// from every other buffer) receive the values of the last pass directly, so
// *v1_out == v1_final whenever at least one pass ran.  With unpack (no v2,
// v1_final given) at least one pass runs and its last pass unpacks v1 as
// SortUnpack states.  Scratch: radix_scratch_elems(n).
int64_t radix_scratch_elems(int64_t n);
int radix_sort_pairs(uint32_t* keys, uint32_t* keys_alt, int32_t* v1, int32_t* v1_alt,
                     int32_t* v2, int32_t* v2_alt, int64_t n, int bits,
                     int32_t* scratch, hipStream_t s, uint32_t** keys_out,
                     int32_t** v1_out, int32_t** v2_out, int32_t* v1_final = nullptr,
                     int32_t* v2_final = nullptr, const SortUnpack* unpack = nullptr);

// Stable partition of n items into `nbins` (<= 256) buckets by a digit array
// (uint8, 255 = drop).  Writes out[off[bin] + rank] = val[i] and bin_off[0..nbins]
// (device int32).  Scratch: radix_scratch_elems(n).
int bucket_partition(const uint8_t* digit, const int32_t* val, int64_t n, int nbins,
                     int32_t* out, int32_t* bin_off, int32_t* scratch, hipStream_t s);

// Fill helpers (used instead of hipMemsetAsync so the kernels can be captured).
int fill_i32(int32_t* p, int32_t v, int64_t n, hipStream_t s);
int fill_u8(uint8_t* p, uint8_t v, int64_t n, hipStream_t s);
int fill_f32(float* p, float v, int64_t n, hipStream_t s);

}  // namespace hg
