// Backward pass of document-masked causal attention over SH-Tiles (gfx950).
//
// Textbook attention gradients (the paper's backward reuses the forward
// assignment with reversed transfers, Sec. 4.3.3, so it computes exactly
// these): P = exp(S - LSE), D = rowsum(dO * O), dV = P^T dO,
// dS = P * (dO V^T - D), dQ = scale dS K, dK = scale dS^T Q.
//
// Two persistent kernels, no atomics (every output element has one writer):
//   * dK / dV (here), KV-stationary: a work item is 128 keys of one KV head of
//     one sample (anchored at the sample start); each of the 4 waves keeps 32
//     keys of K and V in registers plus fp32 dK^T / dV^T accumulators and
//     loops over the 32-row query blocks of the tiles that attend them, two
//     query heads of the KV group per step.  S and dP are computed with
//     queries on M (lane = key), exactly the operand layout that dV^T = dO^T P
//     and dK^T = Q^T dS need; the dO^T / Q^T operands come from the same
//     row-major LDS tiles through the LDS transpose reads.  LSE and D enter
//     the S and dP products as one extra k-block (see bwd_pre_kernel), so the
//     VALU only exponentiates and multiplies.  Steps are staged in a 4-deep
//     LDS ring, two ahead of the one computed.
//   * dQ (attn_bwd_dq.hip), query-stationary, shaped like the forward.  It
//     recomputes S and dP instead of accumulating dQ across key blocks with
//     atomics: on long samples that accumulation is read-modify-write traffic
//     of 4 bytes x d per (32 queries x 128 keys) per head, which would bound
//     the whole backward by HBM.
// Preparation: D = rowsum(dO * O), the augmented operands and the two
// work-item lists, longest first.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "attn_common.h"
#include "errors.h"

namespace libra {

__device__ __forceinline__ int32_t ld_agent(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_agent(const unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bit set of the KV heads whose query groups intersect [hb, he).
__device__ __forceinline__ unsigned long long group_bits(int hb, int he, int G) {
  unsigned long long m = 0;
  for (int g = hb / G; g * G < he; ++g) m |= 1ull << g;
  return m;
}

// ---------------------------------------------------------------------------
// One workgroup: per sample, the key extent attended by covered rows and the
// KV heads involved; then items (sample, 128-key block, KV head) ordered by
// the number of attending rows, longest first, one queue per XCD keyed by
// (KV head, key block) so that an XCD streams the query blocks of few heads.
__global__ __launch_bounds__(kPrepThreads) void prep_bwd_kernel(
    const int64_t *__restrict__ cu, int64_t n, const libra_tile_t *__restrict__ tiles, int64_t T,
    int h_q, int h_kv, int64_t n_q, int64_t n_kv, int32_t *__restrict__ hdr,
    int32_t *__restrict__ ext, unsigned long long *__restrict__ gmask,
    BwdItem *__restrict__ items, int64_t max_items) {
  __shared__ int32_t hist[kXcds * kQBuckets];
  __shared__ int32_t part[kPrepThreads];
  const int tid = threadIdx.x;
  const int G = h_q / h_kv;
  const int R = h_kv >= kXcds ? 1 : kXcds / h_kv;
  for (int64_t j = tid; j < n; j += kPrepThreads) {
    __hip_atomic_store(&ext[j], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&gmask[j], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  if (tid < 5) {
    // the skipped-tile count (counted here for the backward) and the max |x| slots
    __hip_atomic_store(&hdr[tid == 0 ? (int)kBadTiles : kMaxAbs + tid - 1], 0, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  }
  __threadfence();
  __syncthreads();
  int bad = 0;
  for (int64_t t = tid; t < T; t += kPrepThreads) {
    const libra_tile_t tl = tiles[t];
    if (!tile_ok(tl, n_q, n_kv, h_q)) {
      ++bad;
      continue;
    }
    const unsigned long long bits = group_bits(tl.head_begin, tl.head_end, G);
    for (int64_t j = upper_bound64(cu, n, tl.q_begin) - 1; j < n && cu[j] < tl.q_end; ++j) {
      const int64_t pe = tl.q_end < cu[j + 1] ? tl.q_end : cu[j + 1];
      atomicMax(&ext[j], (int32_t)(pe - cu[j]));
      atomicOr(&gmask[j], bits);
    }
  }
  if (bad) atomicAdd(&hdr[kBadTiles], bad);
  __threadfence();
  __syncthreads();
  // Samples with more than kCoopBlocks key blocks are enumerated by the
  // whole workgroup (key blocks across the threads), the others by one
  // thread each; if the list of long samples overflows, every sample goes the
  // per-thread way.  Both enumerations below see the same items.
  constexpr int kCoopBlocks = 64, kMaxLong = 256;
  __shared__ int32_t longs[kMaxLong];
  __shared__ int32_t n_long;
  if (tid == 0) n_long = 0;
  __syncthreads();
  for (int64_t j = tid; j < n; j += kPrepThreads) {
    const int32_t e = ld_agent(&ext[j]);
    if ((e + kBwdBK - 1) / kBwdBK > kCoopBlocks) {
      const int32_t slot = atomicAdd(&n_long, 1);
      if (slot < kMaxLong) longs[slot] = (int32_t)j;
    }
  }
  __syncthreads();
  const bool coop = n_long <= kMaxLong;
  auto emit = [&](auto &&f, int64_t j, int32_t e, int g, int kb) {
    f(BwdItem{(int32_t)j, kb, g, 0}, (int64_t)(e - kb * kBwdBK + kRows - 1) / kRows,
      (g * R + kb % R) % kXcds);
  };
  auto each = [&](auto &&f, bool) {
    for (int64_t j = tid; j < n; j += kPrepThreads) {
      const int32_t e = ld_agent(&ext[j]);
      if (e == 0) continue;
      const int nkb = (e + kBwdBK - 1) / kBwdBK;
      if (coop && nkb > kCoopBlocks) continue;
      const unsigned long long mk = ld_agent(&gmask[j]);
      for (int g = 0; g < h_kv; ++g)
        if (mk >> g & 1ull)
          for (int kb = 0; kb < nkb; ++kb) emit(f, j, e, g, kb);
    }
    if (!coop) return;
    for (int i = 0; i < n_long; ++i) {
      const int64_t j = longs[i];
      const int32_t e = ld_agent(&ext[j]);
      const int nkb = (e + kBwdBK - 1) / kBwdBK;
      const unsigned long long mk = ld_agent(&gmask[j]);
      for (int g = 0; g < h_kv; ++g)
        if (mk >> g & 1ull)
          for (int kb = tid; kb < nkb; kb += kPrepThreads) emit(f, j, e, g, kb);
    }
  };
  build_queues<BwdItem>(each, hist, part, hdr, kBwdQ, items, max_items);
}

// ---------------------------------------------------------------------------
// fp16 operands of the dK / dV kernel.  Its products run on fp16 copies of
// Q, dO, K and V (same matrix-core rate as bf16, three more significant bits
// for the rounded P and dS operands), each scaled by a power of two chosen
// from the tensor's max |x| over what the kernel reads (fp16_scale), so that
// the copies stay inside the fp16 range whatever the inputs' magnitude.
// Two passes find the maxima (fp32 bits, atomicMax on the header slots
// kMaxAbs + 0..3): Q and dO over the covered (row, head) pairs, K and V over
// the keys of the dK / dV work items.

// Workgroup-wide max of two non-negative floats (256 threads), then at most
// one atomic per slot and workgroup, skipped when the slot already holds as
// much (fp32 bits of non-negative floats order like unsigned integers).  Per
// wave atomics on the same two slots serialise: thousands of them took
// longer than the pass's loads.
__device__ __forceinline__ void block_max2_to(float a, float b, int32_t *slot_a,
                                              int32_t *slot_b) {
  __shared__ float red[2][4];
  for (int o = 32; o > 0; o >>= 1) {
    a = fmaxf(a, __shfl_xor(a, o));
    b = fmaxf(b, __shfl_xor(b, o));
  }
  const int tid = threadIdx.x;
  if ((tid & 63) == 0) {
    red[0][tid >> 6] = a;
    red[1][tid >> 6] = b;
  }
  __syncthreads();
  if (tid == 0) {
    a = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    b = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));
    const unsigned ua = __float_as_uint(a), ub = __float_as_uint(b);
    if (a > 0.f && ua > (unsigned)ld_agent(slot_a))
      atomicMax(reinterpret_cast<unsigned int *>(slot_a), ua);
    if (b > 0.f && ub > (unsigned)ld_agent(slot_b))
      atomicMax(reinterpret_cast<unsigned int *>(slot_b), ub);
  }
}

__device__ __forceinline__ float absmax8(const bf16x8 &x) {
  float m = 0.f;
  static_for<8>([&](auto i) { m = fmaxf(m, fabsf(static_cast<float>(x[int(i)]))); });
  return m;
}

constexpr int kTileSplit = 64;

// Per tile (kTileSplit workgroups each): max |Q| and max |dO| over the
// covered (row, head) pairs; and, in the fp16 copies, zeros for the rows of
// the tile's first and last 32-row blocks that lie outside the tile (the
// dK / dV kernel stages whole blocks; rows no tile covers must hold finite
// values, since they meet P = dS = 0 in its products).
template <int D>
__global__ __launch_bounds__(256) void bwd_absmax_q_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ dout,
    const libra_tile_t *__restrict__ tiles, int h_q, int64_t n_q, int64_t n_kv,
    int32_t *__restrict__ hdr, f16 *__restrict__ q16, f16 *__restrict__ do16) {
  const int tid = threadIdx.x;
  const libra_tile_t tl = tiles[blockIdx.x / kTileSplit];
  if (!tile_ok(tl, n_q, n_kv, h_q)) return;
  const int64_t ra = tl.q_row, rb = tl.q_row + (tl.q_end - tl.q_begin);
  const int r = tid >> 3, part = tid & 7;   // 8 threads per row, 32 rows per pass
  float mq = 0.f, mo = 0.f;
  for (int64_t m = ra / kRows + blockIdx.x % kTileSplit; m * kRows < rb; m += kTileSplit) {
    const int64_t row = m * kRows + r;
    const bool ok = row >= ra && row < rb;
    if (!ok && row >= n_q) continue;
    for (int h = tl.head_begin; h < tl.head_end; ++h) {
      const size_t off = ((size_t)row * h_q + h) * D + part * (D / 8);
      static_for<D / 64>([&](auto c) {
        if (ok) {
          mq = fmaxf(mq, absmax8(*reinterpret_cast<const bf16x8 *>(q + off + 8 * c)));
          mo = fmaxf(mo, absmax8(*reinterpret_cast<const bf16x8 *>(dout + off + 8 * c)));
        } else {
          f16x8 z;
          static_for<8>([&](auto i) { z[int(i)] = f16(0.f); });
          *reinterpret_cast<f16x8 *>(q16 + off + 8 * c) = z;
          *reinterpret_cast<f16x8 *>(do16 + off + 8 * c) = z;
        }
      });
    }
  }
  block_max2_to(mq, mo, &hdr[kMaxAbs + 0], &hdr[kMaxAbs + 1]);
}

// The keys the dK / dV kernel loads: for every sample with covered rows,
// its keys up to the end of the last 128-key block that those rows attend
// (all KV heads).  One wave per key row.  CONVERT = false: max |K| and
// max |V| over them; CONVERT = true: their scaled fp16 copies.
template <int D, bool CONVERT>
__global__ __launch_bounds__(256) void bwd_kv_pass_kernel(
    const bf16 *__restrict__ k, const bf16 *__restrict__ v, const int64_t *__restrict__ cu,
    int64_t n, const int32_t *__restrict__ ext, int h_kv, int64_t n_kv,
    int32_t *__restrict__ hdr, f16 *__restrict__ k16, f16 *__restrict__ v16) {
  const int l = threadIdx.x & 63;
  const int64_t wave = ((int64_t)blockIdx.x * 256 + threadIdx.x) >> 6;
  const int64_t waves = (int64_t)gridDim.x * 4;
  const int chunks = h_kv * D / 8;   // 16-byte chunks of a row
  float mk = 0.f, mv = 0.f, s_k = 1.f, s_v = 1.f;
  if constexpr (CONVERT) {
    s_k = fp16_scale((uint32_t)hdr[kMaxAbs + 2], false);
    s_v = fp16_scale((uint32_t)hdr[kMaxAbs + 3], true);
  }
  int64_t lo = 0, hi = 0, end = 0;   // rows [lo, hi) of the current sample; loaded keys end at `end`
  for (int64_t row = wave; row < n_kv; row += waves) {
    if (row < lo || row >= hi) {
      const int64_t j = upper_bound64(cu, n, row) - 1;
      lo = cu[j];
      hi = cu[j + 1];
      const int64_t e = (int64_t)ext[j];
      const int64_t lim = (e + kBwdBK - 1) / kBwdBK * kBwdBK;
      end = lo + (e > 0 ? (lim < hi - lo ? lim : hi - lo) : 0);
    }
    if (row >= end) continue;
    for (int c = l; c < chunks; c += 64) {
      const size_t off = (size_t)row * h_kv * D + 8 * (size_t)c;
      const bf16x8 kx = *reinterpret_cast<const bf16x8 *>(k + off);
      const bf16x8 vx = *reinterpret_cast<const bf16x8 *>(v + off);
      if constexpr (CONVERT) {
        f16x8 kh, vh;
        static_for<8>([&](auto i) {
          kh[int(i)] = static_cast<f16>(static_cast<float>(kx[int(i)]) * s_k);
          vh[int(i)] = static_cast<f16>(static_cast<float>(vx[int(i)]) * s_v);
        });
        *reinterpret_cast<f16x8 *>(k16 + off) = kh;
        *reinterpret_cast<f16x8 *>(v16 + off) = vh;
      } else {
        mk = fmaxf(mk, absmax8(kx));
        mv = fmaxf(mv, absmax8(vx));
      }
    }
  }
  if constexpr (!CONVERT) {
    block_max2_to(mk, mv, &hdr[kMaxAbs + 2], &hdr[kMaxAbs + 3]);
  }
}

// Pre-pass over the covered (row, head) pairs, 32 rows at a time:
//   * the fp16 copies of Q and dO (scaled, see above);
//   * per 32-row block of each head, the 32 values LSE * log2(e) followed by
//     the 32 values D = rowsum(dO * O) for the dQ kernel ("stats",
//     [h_q][nq_pad / 32][64] floats, so one 256-byte load fetches both);
//   * for the dK / dV kernel the first of the two records of its extra
//     16-deep k-block ("aug", [h_q][nq_pad / 32][2][64 lanes][8] fp16): MFMA
//     A-operand lane l < 32 holds three fp16 terms summing to -LSE / scale
//     (first record) or -D (second, written by the dQ kernel from the exact
//     row sums) of the block's row perm32(l), in the scaled units of the
//     copies, then zeros; lanes 32..63 hold zeros.  Against a B operand of
//     ones in k = 0, 1, 2 the products then come out as S - LSE / scale and
//     dP - D directly.
template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ o, const bf16 *__restrict__ dout,
    const float *__restrict__ lse, const libra_tile_t *__restrict__ tiles, int h_q,
    int64_t n_q, int64_t n_kv, int64_t nq_pad, float scale, const int32_t *__restrict__ hdr,
    f16 *__restrict__ q16, f16 *__restrict__ do16, float *__restrict__ stats,
    f16 *__restrict__ aug) {
  const int tid = threadIdx.x;
  const libra_tile_t tl = tiles[blockIdx.x / kTileSplit];
  if (!tile_ok(tl, n_q, n_kv, h_q)) return;
  const float s_q = fp16_scale((uint32_t)hdr[kMaxAbs + 0], false);
  const float s_o = fp16_scale((uint32_t)hdr[kMaxAbs + 1], true);
  const float s_k = fp16_scale((uint32_t)hdr[kMaxAbs + 2], false);
  const int64_t ra = tl.q_row, rb = tl.q_row + (tl.q_end - tl.q_begin);
  // 8 threads per row, 32 rows per pass
  const int r = tid >> 3, part = tid & 7;
  for (int64_t m = ra / kRows + blockIdx.x % kTileSplit; m * kRows < rb; m += kTileSplit) {
    const int64_t row = m * kRows + r;
    const bool ok = row >= ra && row < rb;
    for (int h = tl.head_begin; h < tl.head_end; ++h) {
      float acc = 0.f;
      if (ok) {
        const size_t off = ((size_t)row * h_q + h) * D + part * (D / 8);
        static_for<D / 64>([&](auto c) {
          const bf16x8 qv = *reinterpret_cast<const bf16x8 *>(q + off + 8 * c);
          const bf16x8 ov = *reinterpret_cast<const bf16x8 *>(o + off + 8 * c);
          const bf16x8 dv = *reinterpret_cast<const bf16x8 *>(dout + off + 8 * c);
          f16x8 qh, dh;
          static_for<8>([&](auto i) {
            const float dx = static_cast<float>(dv[int(i)]);
            acc += static_cast<float>(ov[int(i)]) * dx;
            qh[int(i)] = static_cast<f16>(static_cast<float>(qv[int(i)]) * s_q);
            dh[int(i)] = static_cast<f16>(dx * s_o);
          });
          *reinterpret_cast<f16x8 *>(q16 + off + 8 * c) = qh;
          *reinterpret_cast<f16x8 *>(do16 + off + 8 * c) = dh;
        });
      }
      acc += __shfl_xor(acc, 1);
      acc += __shfl_xor(acc, 2);
      acc += __shfl_xor(acc, 4);
      if (part == 0 && ok) {
        float *st = stats + ((size_t)h * (nq_pad / kRows) + m) * 2 * kRows;
        const float lv = lse[(size_t)h * n_q + row];
        st[r] = lv * kLog2e;
        st[kRows + r] = acc;
        f16 *ag = aug + ((size_t)h * (nq_pad / kRows) + m) * kAugEl + 8 * perm32(r);
        f16x8 sv;
        split3h(-lv / scale * (s_q * s_k), sv);
        *reinterpret_cast<f16x8 *>(ag) = sv;
      }
    }
  }
}

__global__ __launch_bounds__(256) void zero_kernel(uint4 *__restrict__ p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * 256)
    p[i] = make_uint4(0, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// dK / dV kernel.
template <int D>
struct KvShape {
  static constexpr int QC = D / 8;          // 16-byte columns of a Q / dO row
  static constexpr int Q_EL = kRows * D;
  static constexpr int F_EL = kAugEl;                         // the two augmented operands
  static constexpr int HEAD_EL = 2 * Q_EL + F_EL;             // Q, dO, aug of one head
  static constexpr int STAGE_EL = 2 * HEAD_EL;                // a step is two query heads
  static constexpr int NSTAGE = 4;                            // LDS ring of steps
  static_assert((NSTAGE & (NSTAGE - 1)) == 0, "ring index by mask");
  static constexpr int NQ = kRows * QC / 64 / kWaves;   // wave loads per Q (dO) tile
  static constexpr int LOADS = 4 * NQ + 1;              // per wave per step
  static constexpr size_t SMEM = NSTAGE * STAGE_EL * sizeof(bf16);
  static_assert((NSTAGE - 2) * LOADS <= 63, "vmcnt range");
};

// Walks the steps (32-row query block x query head) that attend one KV block:
// tiles in list order, query blocks in row order, heads in order.  Per
// fragment (one tile's rows of the sample) everything a step needs is
// precomputed, so that advancing is a few 32-bit scalar operations plus two
// running 64-bit offsets (the Q / dO element offset and the aug offset).
struct StepIter {
  const libra_tile_t *tiles;
  int64_t T, n_q, n_kv, key0, len;
  int h_q, g, G, kloc0, D;
  int64_t nblk;
  // fragment
  int64_t t, row0;          // tile index; buffer row of the fragment's first 32-row block
  int nm, lo0, hin, qb0;    // blocks; lo of block 0; hi of the last block; q_loc of row0
  int h0, h1;
  bool clamp_last;          // the last block runs past the end of the buffer
  // position
  int mi, h;
  int64_t qoff, soff;       // element offset of (row0 + 32 mi, h) in Q / dO; in aug
  bool valid;

  __device__ bool seek() {
    for (; t < T; ++t) {
      const libra_tile_t tl = tiles[t];
      if (!tile_ok(tl, n_q, n_kv, h_q)) continue;
      const int64_t pb = tl.q_begin > key0 ? tl.q_begin : key0;
      const int64_t pe = tl.q_end < key0 + len ? tl.q_end : key0 + len;
      if (pb >= pe) continue;
      h0 = max(tl.head_begin, g * G);
      h1 = min(tl.head_end, (g + 1) * G);
      if (h0 >= h1) continue;
      const int64_t fra = tl.q_row + (pb - tl.q_begin);
      const int64_t frb = fra + (pe - pb);
      const int64_t qla = pb - key0;
      const int64_t first = fra + (kloc0 > qla ? kloc0 - qla : 0);
      if (first >= frb) continue;
      const int64_t mf = first / kRows, ml = (frb - 1) / kRows;
      row0 = mf * kRows;
      nm = (int)(ml - mf + 1);
      lo0 = (int)(fra > row0 ? fra - row0 : 0);
      hin = (int)(frb - ml * kRows);
      qb0 = (int)(qla - (fra - row0));
      clamp_last = ml * kRows + kRows > n_q;
      mi = 0;
      h = h0;
      qoff = (row0 * h_q + h0) * D;
      soff = ((int64_t)h0 * nblk + mf) * kAugEl;
      return true;
    }
    return false;
  }
  __device__ void start() { t = 0; valid = seek(); }
  // steps are pairs of query heads (h, h + 1); two() is false for the last
  // step of an odd head count
  __device__ void next() {
    if ((h += 2) < h1) {
      qoff += 2 * D;
      soff += 2 * nblk * kAugEl;
      return;
    }
    const int back = h - 2 - h0;                 // heads advanced within this block
    h = h0;
    if (++mi < nm) {
      qoff += (int64_t)(kRows * h_q - back) * D;
      soff -= (int64_t)back * nblk * kAugEl - kAugEl;
      return;
    }
    ++t;
    valid = seek();
  }
  __device__ bool two() const { return h + 1 < h1; }
  __device__ int lo() const { return mi == 0 ? lo0 : 0; }
  __device__ int hi() const { return mi == nm - 1 ? hin : kRows; }
  __device__ int qb() const { return qb0 + kRows * mi; }        // q_loc of the block's row 0
  __device__ bool clamp() const { return clamp_last && mi == nm - 1; }
  __device__ int64_t m0() const { return row0 + (int64_t)kRows * mi; }
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) __attribute__((amdgpu_waves_per_eu(1, 1))) void attn_bwd_dkdv_kernel(
    const f16 *__restrict__ k, const f16 *__restrict__ v, const f16 *__restrict__ q,
    const f16 *__restrict__ dout, const f16 *__restrict__ aug,
    const int64_t *__restrict__ cu, const libra_tile_t *__restrict__ tiles, int64_t T,
    const BwdItem *__restrict__ items, int32_t *__restrict__ hdr, int h_q, int h_kv,
    int64_t n_q, int64_t n_kv, int64_t nq_pad, float scale, float c2,
    void *__restrict__ dk_out, void *__restrict__ dv_out, int accumulate) {
  using S = KvShape<D>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  __shared__ int32_t s_item;

  const int tid = threadIdx.x, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  const int G = h_q / h_kv;
  const int64_t nblk = nq_pad / kRows;
  int q_serve = xcd_of_workgroup(), q_left = kXcds;
  // per-lane LDS offsets (elements) of the operand reads: rows of Q / dO for
  // S and dP (row perm32(ln), 8 columns), and the transpose reads that give
  // dO^T / Q^T for dV^T and dK^T: this lane addresses 4 columns of row
  // 8 kg + 4 half + i of the block (i = (l % 16) / 4), the columns whose
  // 16-lane group hands them to the lanes that need column perm32(ln)
  const int prow = perm32(ln);
  int qoff[D / 16], troff[D / 32][2];
  static_for<D / 16>([&](auto c) { qoff[c] = prow * D + 8 * swt<S::QC>(prow, 2 * c + kg); });
  {
    const int grp = l >> 4, i = (l & 15) >> 2, r = l & 3;
    static_for<D / 32>([&](auto dt) {
      static_for<2>([&](auto hf) {
        const int row = 8 * (grp >> 1) + 4 * hf + i;
        const int chunk = 4 * dt + 2 * (grp & 1) + (r & 1);
        troff[dt][hf] = row * D + 8 * swt<S::QC>(row, chunk) + 4 * (r >> 1);
      });
    });
  }
  // per-lane parts of the staging addresses (bytes), fixed for the kernel
  static_assert(S::NQ == 1 || S::NQ == 2, "two or four staging copies per head");
  uint32_t q_lane[S::NQ];
  static_for<S::NQ>([&](auto u) {
    const int r = (w + kWaves * u) * (64 / S::QC) + l / S::QC;
    q_lane[u] = 2u * (uint32_t)(r * h_q * D + 8 * swt<S::QC>(r, l % S::QC));
  });
  // B operand of the augmented k-block: ones in k = 0, 1, 2 (lanes of kg 0)
  f16x8 ones3;
  static_for<8>([&](auto i) { ones3[int(i)] = f16(kg == 0 && i < 3 ? 1.f : 0.f); });
  // Every operand is an fp16 copy scaled by a power of two (fp16_scale): the
  // scores come out multiplied by s_q s_k, dP and D by s_o s_v, so the
  // exponent takes c2 / (s_q s_k) and the outputs are scaled back at the end
  // (exactly: all factors are powers of two).
  const float s_q = fp16_scale((uint32_t)hdr[kMaxAbs + 0], false);
  const float s_o = fp16_scale((uint32_t)hdr[kMaxAbs + 1], true);
  const float s_k = fp16_scale((uint32_t)hdr[kMaxAbs + 2], false);
  const float s_v = fp16_scale((uint32_t)hdr[kMaxAbs + 3], true);
  const float c2s = c2 / (s_q * s_k);
  const float dk_mul = scale / (s_q * s_o * s_v), dv_mul = 1.f / s_o;

  for (;;) {
    if (tid == 0) s_item = take_item(hdr, kBwdQ, q_serve, q_left);
    __syncthreads();
    const int idx = __builtin_amdgcn_readfirstlane(s_item);
    if (idx < 0) break;
    const BwdItem item = items[idx];
    const int64_t key0 = cu[item.sample];
    const int64_t len = cu[item.sample + 1] - key0;
    const int g = item.g;
    const int kloc0 = item.kb * kBwdBK;
    const int kw0 = kloc0 + 32 * w;                   // first key of this wave
    const int kl = kw0 + ln;                          // this lane's key (sample-local)
    const bool key_ok = kl < len;
    const bool wave_keys_ok = kw0 + 31 < len;
    const int64_t krow = key0 + kl;

    f16x8 kf[D / 16], vf[D / 16];
    static_for<D / 16>([&](auto c) {
      if (key_ok) {
        const size_t off = ((size_t)krow * h_kv + g) * D + 16 * c + 8 * kg;
        kf[c] = *reinterpret_cast<const f16x8 *>(k + off);
        vf[c] = *reinterpret_cast<const f16x8 *>(v + off);
      } else {
        static_for<8>([&](auto i) { kf[c][int(i)] = f16(0.f); vf[c][int(i)] = f16(0.f); });
      }
    });
    wait_vm_known();
    f32x16 dva[D / 32], dka[D / 32];
    static_for<D / 32>([&](auto dt) {
      dva[dt] = mfma_zero();
      dka[dt] = mfma_zero();
    });

    // ---- one step = (32-row query block, head); its Q, dO rows and aug go
    // global -> LDS into ring stage `sg` (rows of the block outside the
    // fragment are real rows of other fragments or the clamped last row;
    // their P and dS are masked to zero)
    auto issue = [&](const StepIter &st, int sg) {
      // head h into the first half of the stage, head h + 1 (or h again when
      // the step has one head; it is then not computed) into the second
      const int64_t dq2 = st.two() ? D : 0, ds2 = st.two() ? nblk * kAugEl : 0;
      static_for<2>([&](auto hb) {
        bf16 *Qs = smem + sg * S::STAGE_EL + hb * S::HEAD_EL;
        bf16 *dOs = Qs + S::Q_EL;
        const int64_t qo = st.qoff + (hb ? dq2 : 0);
        if (!st.clamp()) {
          // wave w stages rows w * 64 / QC ... of each 16-byte column group;
          // wave loads u = 0, 1 land 1 KiB x (w + 4 u) into the tile
          const uint32_t lq = lds_addr(Qs) + 1024u * w, ld = lds_addr(dOs) + 1024u * w;
          if constexpr (S::NQ == 2)
            g2l16x4(q + qo, dout + qo, q_lane[0], q_lane[1], lq, lq + 4096u, ld, ld + 4096u);
          else
            g2l16x2(q + qo, dout + qo, q_lane[0], lq, ld);
        } else {
          // the last block of the buffer: rows past it read the last row (masked)
          const int64_t m0 = st.m0();
          const int hh = st.h + (hb && st.two() ? 1 : 0);
          static_for<S::NQ>([&](auto u) {
            const int wl = w + kWaves * u;
            const int r = wl * (64 / S::QC) + l / S::QC;
            const int64_t row = m0 + r < n_q ? m0 + r : n_q - 1;
            const size_t off = ((size_t)row * h_q + hh) * D + 8 * swt<S::QC>(r, l % S::QC);
            g2l16(q + off, Qs + wl * 512);
            g2l16(dout + off, dOs + wl * 512);
          });
        }
      });
      // one augmented record per wave: head w / 2, record w % 2
      const int64_t ao = st.soff + (w >= 2 ? ds2 : 0) + (w & 1) * (kAugEl / 2);
      g2l16s(aug + ao, 16u * l,
             lds_addr(smem + sg * S::STAGE_EL + (w >> 1) * S::HEAD_EL + 2 * S::Q_EL +
                      (w & 1) * (kAugEl / 2)));
    };

    // ---- compute one step from the LDS stage at Qs.  Rows of the block are
    // m0 + iq, iq in [0, 32); with MASK, row iq counts for this lane's key
    // only when lower <= iq < upper (inside the fragment and causal).
    auto step = [&](bool full, const bf16 *Qs, int lower, int upper) {
      constexpr int NC = D / 16, NT = D / 32;
      const bf16 *dOs = Qs + S::Q_EL;
      const bf16 *Ag = dOs + S::Q_EL;     // -LSE / scale record, then the -D record
      // (1) Q rows and this lane's part of the -LSE / scale operand
      f16x8 qa[NC], oa[NC], sag, dag;
      sag = *reinterpret_cast<const f16x8 *>(Ag + 8 * l);
      static_for<NC>([&](auto c) { qa[c] = *reinterpret_cast<const f16x8 *>(Qs + qoff[c]); });
      __builtin_amdgcn_sched_barrier(0);
      // (2) S - LSE / scale = [Q | aug] [K | ones]^T (queries on M, this
      // lane's key on N) while the dO rows and the -D operand load
      f32x16 sa = mfma32h(sag, ones3, mfma_zero_c()), pa;
      static_for<NC>([&](auto c) { sa = mfma32h(qa[c], kf[c], sa); });
      dag = *reinterpret_cast<const f16x8 *>(Ag + kAugEl / 2 + 8 * l);
      static_for<NC>([&](auto c) { oa[c] = *reinterpret_cast<const f16x8 *>(dOs + qoff[c]); });
      static_for<NC + 1>([&](auto i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, i < NC / 2 + 1 ? 2 : 0, 0);
      });
      __builtin_amdgcn_sched_barrier(0);
      // (3) dP - D = [dO | aug] [V | ones]^T with P = exp2((S - LSE / scale) c2)
      // on the VALU and the transpose reads of dO^T; register 8 hh + i of S
      // holds row 16 hh + 8 kg + i
      f16x8 ta[NT][2];
      float pf[16];
      f16x8 pb16[2], db16[2];
      auto phase3 = [&](auto mask_t) {
      constexpr bool MASK = decltype(mask_t)::value;
      pa = mfma32h(dag, ones3, mfma_zero_c());
      static_for<NC>([&](auto c) { pa = mfma32h(oa[c], vf[c], pa); });
      static_for<2>([&](auto hh) {
        static_for<8>([&](auto i) {
          constexpr int r = 8 * hh + i;
          float p = fast_exp2(sa[r] * c2s);
          if constexpr (MASK) {
            const int iq = 16 * hh + 8 * kg + i;
            p = (iq >= lower && iq < upper) ? p : 0.f;
          }
          pf[r] = p;
          pb16[hh][int(i)] = static_cast<f16>(p);
        });
      });
      static_for<NT>([&](auto dt) {
        static_for<2>([&](auto c) {
          const f16 *base = reinterpret_cast<const f16 *>(dOs) + 16 * c * D;
          ta[dt][c] = lds_tr16x2h(base + troff[dt][0], base + troff[dt][1]);
        });
      });
      static_for<NC + 1>([&](auto i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, MASK ? 9 : 5, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, i < NC ? 2 : 0, 0);
      });
      };
      if (full) phase3(std::false_type{});
      else phase3(std::true_type{});
      __builtin_amdgcn_sched_barrier(0);
      // (4) dV^T += dO^T P with dS = P (dP - D) on the VALU and the transpose
      // reads of Q^T
      f16x8 tq[NT][2];
      static_for<NT>([&](auto dt) {
        static_for<2>([&](auto c) { dva[dt] = mfma32h(ta[dt][c], pb16[c], dva[dt]); });
      });
      static_for<2>([&](auto hh) {
        static_for<8>([&](auto i) {
          constexpr int r = 8 * hh + i;
          db16[hh][int(i)] = static_cast<f16>(pf[r] * pa[r]);
        });
      });
      static_for<NT>([&](auto dt) {
        static_for<2>([&](auto c) {
          const f16 *base = reinterpret_cast<const f16 *>(Qs) + 16 * c * D;
          tq[dt][c] = lds_tr16x2h(base + troff[dt][0], base + troff[dt][1]);
        });
      });
      static_for<2 * NT>([&](auto i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 7, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
      });
      __builtin_amdgcn_sched_barrier(0);
      // (5) dK^T += Q^T dS
      static_for<NT>([&](auto dt) {
        static_for<2>([&](auto c) { dka[dt] = mfma32h(tq[dt][c], db16[c], dka[dt]); });
      });
    };

    // Steps are walked once, at issue; what the compute side needs of the step
    // in ring stage j (lo | hi << 8 | two << 16, and the q_loc of the block's
    // row 0) waits in lane j of desc / desc_qb.
    StepIter iss{tiles, T, n_q, n_kv, key0, len, h_q, g, G, kloc0, D, nblk};
    iss.start();
    int desc = 0, desc_qb = 0;
    int issued = 0, computed = 0;
    auto issue_next = [&]() {
      const int sg = issued & (S::NSTAGE - 1);
      issue(iss, sg);
      if (l == sg) {
        desc = iss.lo() | iss.hi() << 8 | (iss.two() ? 1 << 16 : 0);
        desc_qb = iss.qb();
      }
      iss.next();
      ++issued;
    };
    while (iss.valid && issued < S::NSTAGE - 1) issue_next();
    while (computed < issued) {
      // keep up to NSTAGE - 1 steps in flight, the one computed now included
      if (iss.valid && issued < computed + S::NSTAGE - 1) issue_next();
      // wait for this step's loads: in steady state NSTAGE - 2 later steps
      // stay in flight; near the end of an item, wait for everything
      if (issued - 1 - computed >= S::NSTAGE - 2) {
        wait_vm_n<(S::NSTAGE - 2) * S::LOADS>();
      } else {
        wait_vm_n<0>();
      }
      barrier_nofence();

      const int sg = computed & (S::NSTAGE - 1);
      const int dsc = __builtin_amdgcn_readlane(desc, sg);
      const int lo_l = dsc & 0xff, hi_l = (dsc >> 8) & 0xff;
      const bool two = (dsc >> 16) != 0;
      const int qb = __builtin_amdgcn_readlane(desc_qb, sg);   // q_loc of the block's row 0
      if (kw0 <= qb + hi_l - 1) {
        const bf16 *Qs = smem + sg * S::STAGE_EL;
        // interior blocks: every row inside the fragment and at or after every key
        const bool full = lo_l == 0 && hi_l == kRows && wave_keys_ok && kw0 + 31 <= qb;
        const int need = kl - qb;                               // first iq with q_loc >= kl
        const int lower = need > lo_l ? (need < kRows ? need : kRows) : lo_l;
        const int upper = key_ok ? hi_l : 0;
        step(full, Qs, lower, upper);
        if (two) step(full, Qs + S::HEAD_EL, lower, upper);
      }
      ++computed;
    }

    // ---- write dK, dV for this wave's 32 keys
    if (key_ok) {
      const size_t base = ((size_t)krow * h_kv + g) * D + 8 * kg;
      static_for<D / 32>([&](auto dt) {
        static_for<2>([&](auto hh) {
          const size_t off = base + 32 * dt + 16 * hh;
          if (accumulate) {
            float4 *dkp = reinterpret_cast<float4 *>(static_cast<float *>(dk_out) + off);
            float4 *dvp = reinterpret_cast<float4 *>(static_cast<float *>(dv_out) + off);
            static_for<2>([&](auto e) {
              constexpr int r0 = 8 * hh + 4 * e;
              float4 a = dkp[e], bb = dvp[e];
              a.x += dka[dt][r0 + 0] * dk_mul; bb.x += dva[dt][r0 + 0] * dv_mul;
              a.y += dka[dt][r0 + 1] * dk_mul; bb.y += dva[dt][r0 + 1] * dv_mul;
              a.z += dka[dt][r0 + 2] * dk_mul; bb.z += dva[dt][r0 + 2] * dv_mul;
              a.w += dka[dt][r0 + 3] * dk_mul; bb.w += dva[dt][r0 + 3] * dv_mul;
              dkp[e] = a;
              dvp[e] = bb;
            });
          } else {
            bf16x8 a, bb;
            static_for<8>([&](auto i) {
              a[int(i)] = static_cast<bf16>(dka[dt][8 * hh + i] * dk_mul);
              bb[int(i)] = static_cast<bf16>(dva[dt][8 * hh + i] * dv_mul);
            });
            *reinterpret_cast<bf16x8 *>(static_cast<bf16 *>(dk_out) + off) = a;
            *reinterpret_cast<bf16x8 *>(static_cast<bf16 *>(dv_out) + off) = bb;
          }
        });
      });
    }
    wait_vm_n<0>();
    __syncthreads();   // the ring is reused by the next item
  }
}

// ---------------------------------------------------------------------------
static size_t align256b(size_t x) { return (x + 255) / 256 * 256; }

BwdLayout bwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d) {
  BwdLayout L;
  L.max_items = (n_kv / kBwdBK + n + 1) * (int64_t)h_kv;
  L.max_qitems = fwd_max_items(T, n, n_q, h_q, h_kv);
  L.nq_pad = (n_q + kRows - 1) / kRows * kRows;
  L.hdr = 0;
  L.ext = align256b(kHdrSlots * sizeof(int32_t));
  L.gmask = align256b(L.ext + (size_t)n * sizeof(int32_t));
  L.items = align256b(L.gmask + (size_t)n * sizeof(unsigned long long));
  L.qitems = align256b(L.items + (size_t)L.max_items * sizeof(BwdItem));
  L.q16 = align256b(L.qitems + (size_t)L.max_qitems * sizeof(FwdItem));
  L.do16 = align256b(L.q16 + (size_t)n_q * h_q * d * sizeof(f16));
  L.k16 = align256b(L.do16 + (size_t)n_q * h_q * d * sizeof(f16));
  L.v16 = align256b(L.k16 + (size_t)n_kv * h_kv * d * sizeof(f16));
  L.stats = align256b(L.v16 + (size_t)n_kv * h_kv * d * sizeof(f16));
  L.aug = align256b(L.stats + (size_t)h_q * L.nq_pad * 2 * sizeof(float));
  L.splits = align256b(L.aug + (size_t)h_q * (L.nq_pad / kRows) * kAugEl * sizeof(f16));
  L.max_parts = kFwdSplitSlots;
  L.parts = align256b(L.splits + (size_t)(L.max_parts / 2) * sizeof(FwdSplit));
  L.total = align256b(L.parts + (size_t)L.max_parts * fwd_part_floats(d) * sizeof(float));
  return L;
}

template <int D>
static int launch_bwd_d(const bf16 *q, const bf16 *k, const bf16 *v, const bf16 *o,
                        const float *lse, const bf16 *dout, const int64_t *cu, int64_t n,
                        const libra_tile_t *tiles, int64_t T, int64_t n_q, int64_t n_kv, int h_q,
                        int h_kv, float scale, bf16 *dq, void *dk, void *dv, bool accumulate,
                        char *ws, const BwdLayout &L, hipStream_t st, const KernelTimer *tm_kv,
                        const KernelTimer *tm_q) {
  int32_t *hdr = reinterpret_cast<int32_t *>(ws + L.hdr);
  int32_t *ext = reinterpret_cast<int32_t *>(ws + L.ext);
  auto *gmask = reinterpret_cast<unsigned long long *>(ws + L.gmask);
  BwdItem *items = reinterpret_cast<BwdItem *>(ws + L.items);
  FwdItem *qitems = reinterpret_cast<FwdItem *>(ws + L.qitems);
  f16 *q16 = reinterpret_cast<f16 *>(ws + L.q16);
  f16 *do16 = reinterpret_cast<f16 *>(ws + L.do16);
  f16 *k16 = reinterpret_cast<f16 *>(ws + L.k16);
  f16 *v16 = reinterpret_cast<f16 *>(ws + L.v16);
  float *stats = reinterpret_cast<float *>(ws + L.stats);
  f16 *aug = reinterpret_cast<f16 *>(ws + L.aug);
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&attn_bwd_dkdv_kernel<D>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)KvShape<D>::SMEM) != hipSuccess)
      return fail(LIBRA_EHIP, "hipFuncSetAttribute failed");
    attr_set = true;
  }
  if (!accumulate) {
    const int64_t n16 = n_kv * h_kv * D * (int64_t)sizeof(bf16) / 16;
    const unsigned blocks = (unsigned)std::min<int64_t>((n16 + 255) / 256, 4096);
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, st, static_cast<uint4 *>(dk), n16);
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, st, static_cast<uint4 *>(dv), n16);
  }
  if (T > 0) {
    hipLaunchKernelGGL(prep_bwd_kernel, dim3(1), dim3(kPrepThreads), 0, st, cu, n, tiles, T, h_q,
                       h_kv, n_q, n_kv, hdr, ext, gmask, items, L.max_items);
    int dev = 0, cus = 256;
    hipGetDevice(&dev);
    hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    // the dQ kernel runs one workgroup per CU; its items split K like the
    // forward's when there are few of them
    auto *splits = reinterpret_cast<FwdSplit *>(ws + L.splits);
    float *parts = reinterpret_cast<float *>(ws + L.parts);
    enqueue_fwd_items(cu, n, tiles, T, h_q, h_kv, n_q, n_kv, hdr, qitems, L.max_qitems, false,
                      cus, L.max_parts, splits, st);
    {
      // stats and aug of rows outside the covered ones stay zero (finite):
      // they are only read for masked rows; lanes 32..63 of aug stay zero
      const int64_t s16 = (int64_t)(L.splits - L.stats) / 16;
      hipLaunchKernelGGL(zero_kernel, dim3((unsigned)std::min<int64_t>((s16 + 255) / 256, 4096)),
                         dim3(256), 0, st, reinterpret_cast<uint4 *>(stats), s16);
    }
    hipLaunchKernelGGL(bwd_absmax_q_kernel<D>, dim3((unsigned)(T * kTileSplit)), dim3(256), 0, st,
                       q, dout, tiles, h_q, n_q, n_kv, hdr, q16, do16);
    hipLaunchKernelGGL((bwd_kv_pass_kernel<D, false>), dim3((unsigned)cus * 8), dim3(256), 0, st,
                       k, v, cu, n, ext, h_kv, n_kv, hdr, k16, v16);
    hipLaunchKernelGGL((bwd_kv_pass_kernel<D, true>), dim3((unsigned)cus * 8), dim3(256), 0, st,
                       k, v, cu, n, ext, h_kv, n_kv, hdr, k16, v16);
    hipLaunchKernelGGL(bwd_pre_kernel<D>, dim3((unsigned)(T * kTileSplit)), dim3(256), 0, st, q,
                       o, dout, lse, tiles, h_q, n_q, n_kv, L.nq_pad, scale, hdr, q16, do16,
                       stats, aug);
    // dQ first: it writes the -D records the dK / dV kernel reads
    const int rc = launch_bwd_dq(D, q, dout, k, v, stats, cu, qitems, hdr, h_q, h_kv, n_q, n_kv,
                                 L.nq_pad, scale, dq, aug, splits, parts, L.max_parts, cus,
                                 st, tm_q);
    if (rc != LIBRA_OK) return rc;
    if (tm_kv) hipEventRecord(tm_kv->begin, st);
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<D>, dim3(cus), dim3(kThreads), KvShape<D>::SMEM, st,
                       k16, v16, q16, do16, aug, cu, tiles, T, items, hdr, h_q, h_kv, n_q, n_kv,
                       L.nq_pad, scale, scale * kLog2e, dk, dv, accumulate ? 1 : 0);
    if (tm_kv) hipEventRecord(tm_kv->end, st);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(LIBRA_EHIP, "backward launch failed: %s", hipGetErrorString(e));
  return LIBRA_OK;
}

int launch_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
               const void *dout, const int64_t *cu, int64_t n, const libra_tile_t *tiles,
               int64_t T, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d, float scale,
               void *dq, void *dk, void *dv, bool accumulate, void *ws, const BwdLayout &L,
               hipStream_t st, const KernelTimer *tm_kv, const KernelTimer *tm_q) {
  auto Q = static_cast<const bf16 *>(q);
  auto K = static_cast<const bf16 *>(k);
  auto V = static_cast<const bf16 *>(v);
  auto O = static_cast<const bf16 *>(o);
  auto dO = static_cast<const bf16 *>(dout);
  auto dQ = static_cast<bf16 *>(dq);
  char *W = static_cast<char *>(ws);
  if (d == 128)
    return launch_bwd_d<128>(Q, K, V, O, lse, dO, cu, n, tiles, T, n_q, n_kv, h_q, h_kv, scale,
                             dQ, dk, dv, accumulate, W, L, st, tm_kv, tm_q);
  return launch_bwd_d<64>(Q, K, V, O, lse, dO, cu, n, tiles, T, n_q, n_kv, h_q, h_kv, scale, dQ,
                          dk, dv, accumulate, W, L, st, tm_kv, tm_q);
}

}  // namespace libra
