// Shared device helpers and workspace layout for the attention kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "libra.h"

namespace libra {

typedef __bf16 bf16;
typedef bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16;
typedef f16 f16x8 __attribute__((ext_vector_type(8)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Keys per forward KV block; keys per backward KV block; rows per wave.
constexpr int kFwdBN = 64;
constexpr int kBwdBK = 128;
constexpr int kRows = 32;
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

// Work items are ordered longest-first in one queue per XCD (8 XCDs of 32
// CUs, each with its own L2): items that stream the same K/V (forward, dQ) or
// the same query blocks (dK/dV) share a queue, so the CUs of one XCD read the
// same blocks at about the same time.  A workgroup serves the queue of its XCD
// (workgroups are dispatched round-robin over the XCDs) and moves on to the
// other queues when it runs dry.
constexpr int kXcds = 8;
constexpr int kQBuckets = 1024;      // cost buckets per queue
constexpr int kPrepThreads = 1024;

// Workspace header (int32 slots).  A queue set at `base` keeps the queue
// heads at [base, base+8), item counts at [base+8, base+16) and segment
// starts at [base+16, base+24).
enum HdrSlot {
  kBadTiles = 4,   // tiles skipped because they were out of range (+1 on item overflow)
  kFwdQ = 8,       // forward / dQ work items
  kBwdQ = 32,      // dK/dV work items
  kMaxAbs = 56,    // backward: max |x| (fp32 bits) of Q, dO, K, V in slots 56..59
  kFwdSplits = 60, // forward: split items (FwdSplit records), then partial slots used (61)
  kHdrSlots = 64
};
static_assert(kBadTiles * 4 == LIBRA_WS_SKIPPED_OFFSET, "documented offset of the skip count");

// Cost bucket, 0 = longest: exact below 512, then 32 units per bucket.
__device__ __forceinline__ int cost_bucket(int64_t c) {
  const int64_t b = c < 512 ? c : 512 + (c - 512) / 32;
  return kQBuckets - 1 - (int)(b < kQBuckets - 1 ? b : kQBuckets - 1);
}

// One workgroup of kPrepThreads: counts items per (queue, bucket), scans, and
// scatters them so that each queue's segment is longest-first.
// `each(f, scatter)` must call f(item, cost, queue) once per item, the same
// items with the same costs and queues in both passes (scatter = false:
// counting, then true: placing).
template <typename Item, typename Each>
__device__ void build_queues(Each &&each, int32_t *hist, int32_t *part, int32_t *hdr, int base,
                             Item *out, int64_t max_items) {
  const int tid = threadIdx.x;
  for (int i = tid; i < kXcds * kQBuckets; i += kPrepThreads) hist[i] = 0;
  __syncthreads();
  each([&](const Item &, int64_t cost, int x) {
    atomicAdd(&hist[x * kQBuckets + cost_bucket(cost)], 1);
  }, false);
  __syncthreads();
  constexpr int per = kXcds * kQBuckets / kPrepThreads;
  int32_t s = 0;
  for (int i = 0; i < per; ++i) s += hist[tid * per + i];
  part[tid] = s;
  __syncthreads();
  for (int o = 1; o < kPrepThreads; o <<= 1) {
    const int32_t v = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int32_t pos = part[tid] - s;
  constexpr int threads_per_queue = kPrepThreads / kXcds;
  if (tid % threads_per_queue == 0) {
    const int x = tid / threads_per_queue;
    const int32_t start = pos;
    const int32_t end = part[tid + threads_per_queue - 1];
    const int32_t lim = (int32_t)(max_items < INT32_MAX ? max_items : INT32_MAX);
    hdr[base + x] = 0;
    hdr[base + kXcds + x] = (end < lim ? end : lim) - (start < lim ? start : lim);
    hdr[base + 2 * kXcds + x] = start;
    if (x == kXcds - 1 && end > lim) atomicAdd(&hdr[kBadTiles], 1);
  }
  __syncthreads();
  for (int i = 0; i < per; ++i) {
    const int32_t cnt = hist[tid * per + i];
    hist[tid * per + i] = pos;
    pos += cnt;
  }
  __syncthreads();
  each([&](const Item &it, int64_t cost, int x) {
    const int32_t p = atomicAdd(&hist[x * kQBuckets + cost_bucket(cost)], 1);
    if (p < max_items) out[p] = it;
  }, true);
}

// The XCD this workgroup runs on, read from the hardware (XCC_ID, bits 3:0).
// Workgroups are dispatched round-robin over the XCDs, so this equals
// blockIdx.x % 8 on a device in single-partition mode.
__device__ __forceinline__ int xcd_of_workgroup() {
  return __builtin_amdgcn_s_getreg(20 | (3 << 11)) & (kXcds - 1);   // hwreg(XCC_ID, 0, 4)
}

// Thread 0 of a persistent workgroup: index of the next item to run, or -1.
// `q` is the queue being served (starts at the workgroup's XCD), `left` the
// number of queues not yet found empty.
__device__ __forceinline__ int take_item(int32_t *hdr, int base, int &q, int &left) {
  while (left > 0) {
    const int got = atomicAdd(&hdr[base + q], 1);
    if (got < hdr[base + kXcds + q]) return hdr[base + 2 * kXcds + q] + got;
    q = (q + 1) % kXcds;
    --left;
  }
  return -1;
}

// One forward work item: up to 4 query heads of one KV group x up to
// 32 * (4 / heads) consecutive rows of one sample fragment of one tile.
// An item walks the 64-key blocks [kb0, kb1) of its rows' sample; a whole
// item has kb0 = 0 and kb1 = the blocks its last row attends.  A forward item
// split into key ranges (split K) has one item per range, each writing its
// unnormalised partial result to partial slot `slot` (-1: a whole item,
// which writes O and LSE itself).
struct FwdItem {
  int32_t q_row0;   // Q/O row of the first row
  int32_t q_loc0;   // sample-local position of the first row
  int32_t sample;   // sample index j
  int32_t head0;    // first query head
  int32_t nh;       // heads (1..4)
  int32_t nrows;    // rows (1..128)
  int32_t g;        // KV head
  int32_t kb0;      // first key block
  int32_t kb1;      // end of the key blocks
  int32_t slot;     // partial slot of a split part, or -1
  int32_t pad0, pad1;
};
static_assert(sizeof(FwdItem) == 48, "item layout");

// A split forward item: the whole item (kb0 = 0, slot = -1) and the partial
// slots [base, base + parts) of its parts, in key order.
struct FwdSplit {
  FwdItem item;
  int32_t base;
  int32_t parts;
  int32_t pad0, pad1;
};

// Partial slots of split forward items: per slot, the unnormalised O of the
// item's 4 waves x 32 rows (fp32, D per row), then the running max (log2
// units) and the row sum of P of each of the 128 rows.
constexpr int kFwdPartRows = 4 * 32;
constexpr int kFwdSplitMinBlocks = 32;   // a part walks at least 32 key blocks (2048 keys)
constexpr int kFwdSplitSlots = 3072;     // partial slots of one forward call
__host__ __device__ constexpr size_t fwd_part_floats(int d) {
  return (size_t)kFwdPartRows * (size_t)(d + 2);
}

// One backward work item: 128 keys (block kb, anchored at the sample start)
// of KV head g of sample j.
struct BwdItem {
  int32_t sample;
  int32_t kb;
  int32_t g;
  int32_t pad;
};

// Swap bits 2 and 3 of a row index: reading MFMA operand rows in this order
// makes the 16 accumulator registers of a lane hold 8 + 8 contiguous rows.
__device__ __forceinline__ int perm32(int m) {
  return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1);
}

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 mfma32h(f16x8 a, f16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Lanes l and l ^ 32 hold the two halves of a query's row: v_permlane32_swap
// on two copies of x pairs them up in every lane (lanes 0-31 get
// (x[l], x[l + 32]), lanes 32-63 (x[l - 32], x[l])) without a round trip
// through LDS; max and sum of the pair are symmetric, so both lanes of a row
// get the same bits.
__device__ __forceinline__ float row_max2(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float row_sum2(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// Backward "aug" records: per 32-row block and query head, two MFMA
// A-operands of 64 lanes x 8 fp16 (-LSE / scale, then -D; see bwd_pre_kernel).
constexpr int kAugEl = 2 * 64 * 8;


// Swizzle of row-major Q / dO / K / V tiles that are read both by rows
// (16-byte reads, 16 consecutive rows per pass) and by the LDS transpose
// reads below (8-byte reads of 4 rows x 64 bytes per pass, rows 4j..4j+3).
// The chunk is XORed with a bit rotation of the row that spreads either
// pattern over all 64 banks.  C = 16-byte columns per row (8 or 16).
template <int C>
__host__ __device__ __forceinline__ int swt(int row, int col) {
  static_assert(C == 8 || C == 16, "tiles of 64 or 128 bf16 per row");
  if constexpr (C == 16) {
    const int x = row & 15;
    return col ^ (((x & 3) << 2) | (x >> 2));
  } else {
    const int x = (row >> 1) & 7;
    return col ^ (((x & 1) << 2) | (x >> 1));
  }
}

// gfx950 LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16
// lanes, lane 4r + e receives as element i the 16-bit element e of the
// 8 bytes addressed by lane 4i + r of the same group: 16 lanes that address
// 4 consecutive elements of 4 rows each come back holding one column of 4
// rows each, i.e. a 4 x 16 block read transposed.
__device__ __forceinline__ bf16x4 lds_tr16(const bf16 *p) {
  const i16x4 r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4 *)(p));
  return __builtin_bit_cast(bf16x4, r);
}
// An MFMA operand of 8 consecutive rows at one column from two transpose reads.
__device__ __forceinline__ bf16x8 lds_tr16x2(const bf16 *p0, const bf16 *p1) {
  const bf16x4 a = lds_tr16(p0), b = lds_tr16(p1);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// The same two transpose reads for an fp16 tile.
__device__ __forceinline__ f16x8 lds_tr16x2h(const f16 *p0, const f16 *p1) {
  const i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4 *)(p0));
  const i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4 *)(p1));
  return __builtin_bit_cast(f16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Asynchronous 16-byte global -> LDS copy by one wave: lane i's bytes land at
// lds + 16 * i; `lds` must be the same for every lane of the wave.
//
// Written as inline asm on purpose: for the builtin the compiler tracks the
// asynchronous LDS write and, unable to tell ring stages apart, waits for
// every outstanding global -> LDS load (vmcnt(0)) before the first LDS read
// that follows, which defeats a multi-stage ring.  Callers wait for their own
// stages (s_waitcnt vmcnt(N)) before reading them.  M0 (the LDS destination
// of the instruction) is saved and restored around it.
__device__ __forceinline__ void g2l16(const void *g, bf16 *lds) {
  const uint32_t a = __builtin_amdgcn_readfirstlane(
      (uint32_t)(size_t)(__attribute__((address_space(3))) bf16 *)lds);
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(g), "s"(a)
      : "memory");
}
// LDS byte address of a shared-memory pointer, as a wave-uniform value.
__device__ __forceinline__ uint32_t lds_addr(const bf16 *lds) {
  return __builtin_amdgcn_readfirstlane(
      (uint32_t)(size_t)(__attribute__((address_space(3))) const bf16 *)lds);
}
// Four 16-byte-per-lane global -> LDS copies in one statement (one M0 save and
// restore): rows at byte offsets o0, o1 (per lane) from the wave-uniform bases
// ga and gb land at LDS addresses la0, la1 (from ga) and lb0, lb1 (from gb).
__device__ __forceinline__ void g2l16x4(const void *ga, const void *gb, uint32_t o0, uint32_t o1,
                                        uint32_t la0, uint32_t la1, uint32_t lb0, uint32_t lb1) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %7\n\t"
      "s_mov_b32 m0, %4\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %7\n\t"
      "s_mov_b32 m0, %5\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %8\n\t"
      "s_mov_b32 m0, %6\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %8\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(o0), "v"(o1), "s"(la0), "s"(la1), "s"(lb0), "s"(lb1), "s"(ga), "s"(gb)
      : "memory");
}
// Four such copies from one base: rows at byte offsets o0 .. o3 from g land at
// la0 .. la3.
__device__ __forceinline__ void g2l16x4r(const void *g, uint32_t o0, uint32_t o1, uint32_t o2,
                                         uint32_t o3, uint32_t la0, uint32_t la1, uint32_t la2,
                                         uint32_t la3) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %5\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %9\n\t"
      "s_mov_b32 m0, %6\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %2, %9\n\t"
      "s_mov_b32 m0, %7\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %3, %9\n\t"
      "s_mov_b32 m0, %8\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %4, %9\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(o0), "v"(o1), "v"(o2), "v"(o3), "s"(la0), "s"(la1), "s"(la2), "s"(la3), "s"(g)
      : "memory");
}
// One such copy: lane bytes at byte offset o from the wave-uniform base g land
// at LDS address la.
__device__ __forceinline__ void g2l16s(const void *g, uint32_t o, uint32_t la) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %3\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(o), "s"(la), "s"(g)
      : "memory");
}
// Two such copies: the row at o0 from ga to la0 and from gb to lb0.
__device__ __forceinline__ void g2l16x2(const void *ga, const void *gb, uint32_t o0,
                                        uint32_t la0, uint32_t lb0) {
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %2\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %4\n\t"
      "s_mov_b32 m0, %3\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, %5\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "v"(o0), "s"(la0), "s"(lb0), "s"(ga), "s"(gb)
      : "memory");
}
// Workgroup barrier without the memory fence of __syncthreads(): the fence
// would wait for every outstanding global load of the wave, including the
// global -> LDS prefetches of later pipeline stages.  Callers make the data
// they publish complete first (s_waitcnt on the loads that filled it).
__device__ __forceinline__ void barrier_nofence() { __builtin_amdgcn_s_barrier(); }


// s_waitcnt vmcnt(0) that the compiler's wait-count pass sees (unlike an
// inline-asm wait): after it, registers loaded from global memory count as
// ready, so no wait for them is placed inside a loop that follows, where it
// would also wait for the loop's own global -> LDS prefetches.
__device__ __forceinline__ void wait_vm_known() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Wait for this wave's outstanding global loads (including global -> LDS).
__device__ __forceinline__ void wait_vm() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Scheduling hint for a run of N MFMAs that each consume one 16-byte LDS
// read: issue AHEAD reads first, then alternate one MFMA with one read, so
// that every read is in flight while earlier MFMAs execute.
template <int N, int AHEAD>
__device__ __forceinline__ void sched_pipeline() {
  __builtin_amdgcn_sched_group_barrier(0x100, AHEAD, 0);   // DS reads
#pragma unroll
  for (int i = 0; i < N - AHEAD; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);      // MFMA
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);      // DS read
  }
  __builtin_amdgcn_sched_group_barrier(0x008, AHEAD, 0);
}

// Compile-time loop: f(std::integral_constant<int, i>{}) for i in [0, N).  Register
// arrays indexed this way are kept in registers (a runtime-indexed or
// captured array can end up in scratch memory).
template <int I, int N, typename F>
__device__ __forceinline__ void static_for_impl(F &&f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for_impl<I + 1, N>(f);
  }
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl<0, N>(f);
}

// x as hi + mid + lo, three bf16 values in elements 0..2 of r, the rest zero
// (exact to about 2^-24 |x|).  Against a k-block of ones in k = 0, 1, 2 an
// MFMA adds x itself to every accumulator of the row (or column).
__device__ __forceinline__ void split3(float x, bf16x8 &r) {
  const bf16 a = static_cast<bf16>(x);
  const float x1 = x - static_cast<float>(a);
  const bf16 b = static_cast<bf16>(x1);
  const bf16 c = static_cast<bf16>(x1 - static_cast<float>(b));
  static_for<8>([&](auto i) { r[int(i)] = bf16(0.f); });
  r[0] = a;
  r[1] = b;
  r[2] = c;
}

// The same split in fp16: hi + mid + lo carry about 33 significant bits.
__device__ __forceinline__ void split3h(float x, f16x8 &r) {
  const f16 a = static_cast<f16>(x);
  const float x1 = x - static_cast<float>(a);
  const f16 b = static_cast<f16>(x1);
  const f16 c = static_cast<f16>(x1 - static_cast<float>(b));
  static_for<8>([&](auto i) { r[int(i)] = f16(0.f); });
  r[0] = a;
  r[1] = b;
  r[2] = c;
}

// Power-of-two scale of a tensor whose max |x| has fp32 bits `mx`, for its
// fp16 copy.  Gradient-side operands (dO, V) are brought to max |x s| in
// [1, 2), up or down; score-side operands (Q, K) only down, to max |x s| in
// [4, 8), so that the augmented -LSE operand of the dK / dV kernel stays
// inside the fp16 range.  A zero or non-finite max gives s = 1.
__host__ __device__ __forceinline__ float fp16_scale(uint32_t mx, bool up) {
  const int e = (int)((mx >> 23) & 0xff) - 127;   // floor(log2 max) for a normal max
  if (mx == 0 || e == 128 || e == -127) return 1.f;
  int k = up ? -e : (e > 2 ? -(e - 2) : 0);
  k = k < -126 ? -126 : (k > 126 ? 126 : k);
  return __builtin_bit_cast(float, (uint32_t)(k + 127) << 23);
}

// s_waitcnt vmcnt(N) for a compile-time N.
template <int N>
__device__ __forceinline__ void wait_vm_n() {
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Wait until at most k * L vector-memory operations are outstanding
// (k in [0, KMAX]; larger k wait for KMAX * L).
template <int L, int KMAX>
__device__ __forceinline__ void wait_stages(int k) {
  bool done = false;
  static_for<KMAX>([&](auto i) {
    if (!done && k == int(i)) {
      wait_vm_n<int(i) * L>();
      done = true;
    }
  });
  if (!done) wait_vm_n<KMAX * L>();
}

// A zero accumulator produced by an MFMA: in kernels whose MFMAs write
// AGPRs this keeps long-lived accumulators in AGPRs from their first
// definition (a VALU zero-fill would be a VGPR definition and make the
// register allocator copy the accumulators between the two files).
__device__ __forceinline__ f32x16 mfma_zero() {
  bf16x8 z;
  static_for<8>([&](auto i) { z[int(i)] = bf16(0.f); });
  f32x16 c;
  static_for<16>([&](auto i) { c[int(i)] = 0.f; });
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(z, z, c, 0, 0, 0);
}

// A zero accumulator as a plain constant (the first MFMA of a chain reads it
// as the inline constant 0).
__device__ __forceinline__ f32x16 mfma_zero_c() {
  f32x16 c;
  static_for<16>([&](auto i) { c[int(i)] = 0.f; });
  return c;
}

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
  size_t hdr = 0, items = 0, splits = 0, parts = 0, total = 0;
  int64_t max_items = 0;
  int32_t max_parts = 0;   // 0: items are never split
};
struct BwdLayout {
  size_t hdr = 0, ext = 0, gmask = 0, items = 0, qitems = 0, q16 = 0, do16 = 0, k16 = 0,
         v16 = 0, stats = 0, aug = 0, splits = 0, parts = 0, total = 0;
  int32_t max_parts = 0;   // split-K partial slots of the dQ kernel
  int64_t max_items = 0, max_qitems = 0, nq_pad = 0;
};

// `split`: room for split-K partial results (libra_attn_fwd); without it the
// forward never splits an item (the allocation-free entry point).
FwdLayout fwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d,
                     bool split = true);
BwdLayout bwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d);

// Optional HIP events recorded around a main kernel (see libra_timing_*).
struct KernelTimer {
  hipEvent_t begin = nullptr, end = nullptr;
};

// Shared preparation pass (attn_fwd.hip): forward-style work items, also
// used by the dQ kernel.
// Forward-style items for the dQ kernel's `grid` workgroups, split K as in
// the forward when max_parts > 0 (split records into `splits`), but only when
// whole rounds of items would leave workgroups idle: measured on calls of one
// tile, splitting items that already fill the grid cost dQ 2-4%, while the
// forward gained 3-5% from it.
void enqueue_fwd_items(const int64_t *cu, int64_t n, const libra_tile_t *tiles, int64_t T,
                       int h_q, int h_kv, int64_t n_q, int64_t n_kv, int32_t *hdr,
                       FwdItem *items, int64_t max_items, bool count_bad, int grid,
                       int max_parts, FwdSplit *splits, hipStream_t st);
int64_t fwd_max_items(int64_t T, int64_t n, int64_t n_q, int h_q, int h_kv);

int launch_fwd(const void *q, const void *k, const void *v, const int64_t *cu, int64_t n,
               const libra_tile_t *tiles, int64_t T, int64_t n_q, int64_t n_kv, int h_q,
               int h_kv, int d, float scale, void *o, float *lse, void *ws,
               const FwdLayout &L, hipStream_t st, const KernelTimer *tm);
// The dQ kernel of the backward pass (attn_bwd_dq.hip), on `blocks`
// persistent workgroups over the forward-style work items.
int launch_bwd_dq(int d, const bf16 *q, const bf16 *dout, const bf16 *k, const bf16 *v,
                  const float *stats, const int64_t *cu, const FwdItem *items, int32_t *hdr,
                  int h_q, int h_kv, int64_t n_q, int64_t n_kv, int64_t nq_pad, float scale,
                  bf16 *dq, f16 *aug, const FwdSplit *splits, float *parts, int max_parts,
                  int blocks, hipStream_t st, const KernelTimer *tm);
int launch_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
               const void *dout, const int64_t *cu, int64_t n, const libra_tile_t *tiles,
               int64_t T, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d, float scale,
               void *dq, void *dk, void *dv, bool accumulate, void *ws, const BwdLayout &L,
               hipStream_t st, const KernelTimer *tm_kv, const KernelTimer *tm_q);

}  // namespace libra
