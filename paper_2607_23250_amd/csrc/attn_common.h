// Shared device helpers and workspace layout for the attention kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "libra.h"

namespace libra {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Keys per forward KV block; keys per backward KV block; rows per wave.
constexpr int kFwdBN = 64;
constexpr int kBwdBK = 128;
constexpr int kRows = 32;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

// Buckets of the longest-first ordering of work items.
constexpr int kBuckets = 8192;
constexpr int kPrepThreads = 1024;

// Workspace header (int32 slots).
enum HdrSlot {
  kFwdQueue = 0,   // next forward item to take
  kFwdItems = 1,   // number of forward items
  kBwdQueue = 2,
  kBwdItems = 3,
  kBadTiles = 4,   // tiles skipped because they were out of range
  kHdrSlots = 64
};

// One forward work item: up to 4 query heads of one KV group x up to
// 32 * (4 / heads) consecutive rows of one sample fragment of one tile.
struct FwdItem {
  int32_t q_row0;   // Q/O row of the first row
  int32_t q_loc0;   // sample-local position of the first row
  int32_t sample;   // sample index j
  int32_t head0;    // first query head
  int32_t nh;       // heads (1..4)
  int32_t nrows;    // rows (1..128)
  int32_t g;        // KV head
  int32_t pad;
};

// One backward work item: 128 keys (block kb, anchored at the sample start)
// of KV head g of sample j.
struct BwdItem {
  int32_t sample;
  int32_t kb;
  int32_t g;
  int32_t pad;
};

// Offset of sample j in the padded, transposed V copy: sample j starts at a
// multiple of kFwdBN and owns ceil(len/kFwdBN)*kFwdBN zero-padded slots.
// ceil64(cu[j] + 128 j) keeps consecutive samples apart without a prefix sum.
__host__ __device__ inline int64_t vt_offset(int64_t cu_j, int64_t j) {
  return (cu_j + 128 * j + 63) / 64 * 64;
}
__host__ __device__ inline int64_t vt_pitch(int64_t n_kv, int64_t n_samples) {
  return n_kv + 128 * n_samples + 64;
}

// Swap bits 2 and 3 of a row index: reading MFMA operand rows in this order
// makes the 16 accumulator registers of a lane hold 8 + 8 contiguous rows.
__device__ __forceinline__ int perm32(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// First index i in [0, n] with a[i] > x (a sorted ascending, n+1 entries read at most n).
__device__ __forceinline__ int64_t upper_bound64(const int64_t *a, int64_t n, int64_t x) {
  int64_t lo = 0, hi = n;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

// A tile is usable when it lies inside the buffers the call describes.
__device__ __forceinline__ bool tile_ok(const libra_tile_t &t, int64_t n_q, int64_t n_kv,
                                        int h_q) {
  return t.q_begin >= 0 && t.q_end <= n_kv && t.q_begin < t.q_end && t.q_row >= 0 &&
         t.q_row + (t.q_end - t.q_begin) <= n_q && t.head_begin >= 0 &&
         t.head_end <= h_q && t.head_begin < t.head_end;
}

// ---------------------------------------------------------------------------
// Host-side workspace layouts and launchers (defined in attn_fwd.hip / attn_bwd.hip).
struct FwdLayout {
  size_t hdr = 0, items = 0, vt = 0, total = 0;
  int64_t max_items = 0, pitch = 0;
};
struct BwdLayout {
  size_t hdr = 0, ext = 0, gmask = 0, items = 0, dvec = 0, qt = 0, dot = 0, dqacc = 0, total = 0;
  int64_t max_items = 0, nq_pad = 0;
};

FwdLayout fwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d);
BwdLayout bwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d);

// Optional HIP events recorded around a main kernel (see libra_timing_*).
struct KernelTimer {
  hipEvent_t begin = nullptr, end = nullptr;
};

int launch_fwd(const void *q, const void *k, const void *v, const int64_t *cu, int64_t n,
               const libra_tile_t *tiles, int64_t T, int64_t n_q, int64_t n_kv, int h_q,
               int h_kv, int d, float scale, void *o, float *lse, void *ws,
               const FwdLayout &L, hipStream_t st, const KernelTimer *tm);
int launch_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
               const void *dout, const int64_t *cu, int64_t n, const libra_tile_t *tiles,
               int64_t T, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d, float scale,
               void *dq, void *dk, void *dv, bool accumulate, void *ws, const BwdLayout &L,
               hipStream_t st, const KernelTimer *tm);

}  // namespace libra
